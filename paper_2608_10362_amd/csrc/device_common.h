// Device-side helpers shared by the gfx950 kernels: storage types, Philox,
// wavefront / block reductions, and the layout of the per-row descriptors.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace specdec {

constexpr int kWave = 64;

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float floatx4;
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// ------------------------------------------------------------------ storage types
__device__ __forceinline__ float bf16_bits_to_f32(uint16_t b) {
  return __uint_as_float(((uint32_t)b) << 16);
}
// round-to-nearest-even float -> bf16 bits (finite inputs; NaN kept as a quiet NaN)
__device__ __forceinline__ uint16_t f32_to_bf16_bits(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu)) return (uint16_t)((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

// Stacked bf16 operand of at most 16 activation rows, the x operand of the
// skinny GEMMs written by the kernels that produce x: per 32-column k-step,
// stt fragments of 1 KB in MFMA operand order (lane 16*(k%32/8) + row,
// element k%8).  stt = 1 (at most 8 rows): row m's hi part in fragment row m
// and its lo part in row 8 + m, so one product gives both; stt = 2 (at most
// 16 rows): the hi parts in fragment 0, the lo parts in fragment 1.  hi =
// bf16(v), lo = bf16(v - hi) (round to nearest even, as the GEMMs' own split).
__device__ __forceinline__ void put_stacked(uint16_t* xs, int stt, int m, int k, float v) {
  const __bf16 h = (__bf16)v;
  const __bf16 l = (__bf16)(v - (float)h);
  const size_t at = (size_t)(k >> 5) * stt * 512 + (size_t)(16 * ((k & 31) >> 3) + m) * 8 + (k & 7);
  xs[at] = __builtin_bit_cast(uint16_t, h);
  xs[at + (stt == 1 ? 64 : 512)] = __builtin_bit_cast(uint16_t, l);
}

template <typename T> struct Storage;
template <> struct Storage<float> {
  __device__ __forceinline__ static float load(const float* p) { return *p; }
  __device__ __forceinline__ static void store(float* p, float v) { *p = v; }
};
template <> struct Storage<uint16_t> {
  __device__ __forceinline__ static float load(const uint16_t* p) { return bf16_bits_to_f32(*p); }
  __device__ __forceinline__ static void store(uint16_t* p, float v) { *p = f32_to_bf16_bits(v); }
};

// ------------------------------------------------------------------ Philox4x32-10
// Salmon et al., SC'11.  key = (seed_lo, seed_hi); counter (c0..c3); 10 rounds,
// multipliers 0xD2511F53 / 0xCD9E8D57, key increments 0x9E3779B9 / 0xBB67AE85.
__device__ __forceinline__ uint32_t philox_word0(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3,
                                                 uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    uint32_t lo0 = 0xD2511F53u * c0, hi0 = __umulhi(0xD2511F53u, c0);
    uint32_t lo1 = 0xCD9E8D57u * c2, hi1 = __umulhi(0xCD9E8D57u, c2);
    uint32_t n0 = hi1 ^ c1 ^ k0, n2 = hi0 ^ c3 ^ k1;
    c0 = n0; c1 = lo1; c2 = n2; c3 = lo0;
    k0 += 0x9E3779B9u; k1 += 0xBB67AE85u;
  }
  return c0;
}
__device__ __forceinline__ uint32_t draw_word(uint64_t seed, int b, uint64_t step, int purpose, int index) {
  return philox_word0((uint32_t)b, (uint32_t)step, (uint32_t)(step >> 32),
                      ((uint32_t)(purpose & 0xffff) << 16) | (uint32_t)(index & 0xffff),
                      (uint32_t)seed, (uint32_t)(seed >> 32));
}
// u = (x >> 8) * 2^-24, exact in float32
__device__ __forceinline__ float word_to_uniform(uint32_t x) { return (float)(x >> 8) * 5.9604644775390625e-08f; }

// ------------------------------------------------------------------ reductions
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}
// wave_sum of N values at once: the same butterfly per value (bit-identical
// results), each level's N shuffles issued before any of their sums, so the
// N reductions share one shuffle round trip per level instead of taking N.
template <int N>
__device__ __forceinline__ void wave_sum_n(float (&v)[N]) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    float s[N];
#pragma unroll
    for (int i = 0; i < N; ++i) s[i] = __shfl_xor(v[i], o, kWave);
#pragma unroll
    for (int i = 0; i < N; ++i) v[i] += s[i];
  }
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
  return v;
}
__device__ __forceinline__ uint64_t wave_sum_u64(uint64_t v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}
// (value, index) max with the lowest index on ties
__device__ __forceinline__ void wave_argmax(float& v, int& i) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    float ov = __shfl_xor(v, o, kWave);
    int oi = __shfl_xor(i, o, kWave);
    if (ov > v || (ov == v && oi < i)) { v = ov; i = oi; }
  }
}

// Block-wide sum / max of float (blockDim.x a multiple of 64, <= 1024).
// `red` is __shared__ float[16]; the result is returned to every thread.
__device__ __forceinline__ float block_sum(float v, float* red) {
  v = wave_sum(v);
  int w = threadIdx.x / kWave, l = threadIdx.x % kWave, nw = blockDim.x / kWave;
  __syncthreads();
  if (l == 0) red[w] = v;
  __syncthreads();
  float t = 0.f;
  for (int i = 0; i < nw; ++i) t += red[i];  // fixed order: deterministic
  return t;
}
__device__ __forceinline__ float block_max(float v, float* red) {
  v = wave_max(v);
  int w = threadIdx.x / kWave, l = threadIdx.x % kWave, nw = blockDim.x / kWave;
  __syncthreads();
  if (l == 0) red[w] = v;
  __syncthreads();
  float t = red[0];
  for (int i = 1; i < nw; ++i) t = fmaxf(t, red[i]);
  return t;
}
__device__ __forceinline__ void block_argmax(float& v, int& idx, float* redv, int* redi) {
  wave_argmax(v, idx);
  int w = threadIdx.x / kWave, l = threadIdx.x % kWave, nw = blockDim.x / kWave;
  __syncthreads();
  if (l == 0) { redv[w] = v; redi[w] = idx; }
  __syncthreads();
  v = redv[0]; idx = redi[0];
  for (int i = 1; i < nw; ++i)
    if (redv[i] > v || (redv[i] == v && redi[i] < idx)) { v = redv[i]; idx = redi[i]; }
}

// ------------------------------------------------------------------ row descriptors
// Every forward call works on M rows; row r belongs to sequence rows[r].b at
// absolute position rows[r].pos with token rows[r].tok; invalid rows (padding
// of the draft's first slot) compute garbage that is never stored in a cache.
struct RowDesc {
  int32_t b, pos, tok, valid;
};

// Device status codes (match specdec_status).
constexpr int32_t kStatusKvCapacity = -3;
constexpr int32_t kStatusNonFinite = -4;
constexpr int32_t kStatusBadToken = -7;
constexpr int32_t kStatusWaitExpired = -9;

__device__ __forceinline__ void set_status(int32_t* status, int32_t code) {
  if (status) atomicCAS(status, 0, code);
}

}  // namespace specdec
