// Skinny-M weight-streaming GEMMs of the verify and draft passes:
//   y[m, n] = s_m * sum_k W[n, k] * (x[m, k] * g[k])
// with M = rows of the pass (gamma+1 per sequence for verify, 1-2 for a draft
// step) and W streamed once from HBM.  Epilogues: store (Q|K|V projections,
// LM head), residual add (O and down projections, also emitting the partial
// sums of squares the next RMSNorm needs), and SwiGLU (gate|up).
//
// bf16 weights run on MFMA (v_mfma_f32_16x16x32_bf16).  The float32
// activations are split into hi + lo bf16 parts (x = hi + lo + O(2^-17 |x|)),
// so two MFMAs per weight fragment reproduce a float32-accuracy product while
// the weight fragment is read from HBM once; the padding of M up to 16 is
// free because the pass is bandwidth-bound (about M flops per weight byte).
// float32 weights (the tiny configuration) run on a plain vector kernel.
#include "device_common.h"
#include "internal.h"

namespace specdec {

namespace {

constexpr int kMfmaThreads = 1024;  // 16 waves split K
constexpr int kMfmaWaves = kMfmaThreads / kWave;

__device__ __forceinline__ float silu_f(float z) { return z / (1.0f + expf(-z)); }

__device__ __forceinline__ float load_gain(const void* g, int bf16, int n) {
  return bf16 ? bf16_bits_to_f32(((const uint16_t*)g)[n]) : ((const float*)g)[n];
}

// ---------------------------------------------------------------- shared pieces
// Row scale s_m = 1/sqrt(sum_p ss[p][m] / K + eps): one wave per row, lanes
// stride over the partial sums, fixed shuffle tree (deterministic).
template <int MP>
__device__ __forceinline__ void row_scale(const GemmArgs& a, float* scale) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
  for (int m = wave; m < MP; m += nw) {
    float t = 0.f;
    if (a.ss_in && m < a.M)
      for (int p = lane; p < a.n_ss; p += kWave) t += a.ss_in[(size_t)p * a.ss_ld + m];
    t = wave_sum(t);
    if (lane == 0) scale[m] = (a.ss_in && m < a.M) ? 1.0f / sqrtf(t / (float)a.K + a.eps) : 1.0f;
  }
}

// Epilogue over this block's final sums yfin[m][c], c < NC columns.
template <int NC, int KIND>
__device__ __forceinline__ void epilogue(const GemmArgs& a, int blk, float (*yfin)[NC + 1], const float* scale) {
  const int M = a.M;
  if (KIND == EPI_STORE) {
    for (int i = threadIdx.x; i < M * NC; i += blockDim.x) {
      int m = i / NC, c = i % NC;
      int n = blk * NC + c;
      if (n < a.n_rows) a.out[(size_t)m * a.ldo + n] = yfin[m][c] * scale[m];
    }
  } else if (KIND == EPI_RESID) {
    for (int i = threadIdx.x; i < M * NC; i += blockDim.x) {
      int m = i / NC, c = i % NC;
      int n = blk * NC + c;
      float hv = 0.f;
      if (n < a.n_rows) {
        float* hp = a.out + (size_t)m * a.ldo + n;
        hv = *hp + yfin[m][c];
        *hp = hv;
        a.xg_out[(size_t)m * a.ldo + n] = hv * load_gain(a.gain_out, a.gain_bf16, n);
      }
      yfin[m][c] = hv;
    }
    __syncthreads();
    for (int m = threadIdx.x; m < M; m += blockDim.x) {
      float t = 0.f;
      for (int c = 0; c < NC; ++c) t += yfin[m][c] * yfin[m][c];
      a.ss_out[(size_t)blk * a.ss_ld + m] = t;
    }
  } else {  // EPI_SWIGLU: columns [0, NC/2) gate, [NC/2, NC) up
    constexpr int H = NC / 2;
    for (int i = threadIdx.x; i < M * H; i += blockDim.x) {
      int m = i / H, c = i % H;
      int n = blk * H + c;
      if (n < a.n_rows) {
        float g = yfin[m][c] * scale[m];
        float u = yfin[m][H + c] * scale[m];
        a.out[(size_t)m * a.ldo + n] = silu_f(g) * u;
      }
    }
  }
}

// Row pointer of weight row `r` of the block's concatenated row space.
template <typename WT>
__device__ __forceinline__ const WT* weight_row(const GemmArgs& a, int kind, int blk, int NC, int c, bool& ok) {
  if (kind == EPI_SWIGLU) {
    const int H = NC / 2;
    int seg = c >= H;
    int n = blk * H + (c - seg * H);
    ok = n < a.n_rows;
    if (!ok) n = 0;
    return (const WT*)a.w[seg] + (size_t)n * a.K;
  }
  int n = blk * NC + c;
  ok = n < a.n_rows;
  if (!ok) n = 0;
  int b1 = a.n_seg[0], b2 = b1 + a.n_seg[1];
  if (n < b1) return (const WT*)a.w[0] + (size_t)n * a.K;
  if (n < b2) return (const WT*)a.w[1] + (size_t)(n - b1) * a.K;
  return (const WT*)a.w[2] + (size_t)(n - b2) * a.K;
}

// Base of the packed 16-row tile `t` (t < NC/16) of block `blk`.  Packed
// matrices are sequences of 16-row tiles of ceil(K/32) 1 KB fragments.
__device__ __forceinline__ const uint16_t* weight_tile(const GemmArgs& a, int kind, int blk, int NC, int t,
                                                       int KS, bool& ok) {
  int seg, n;
  if (kind == EPI_SWIGLU) {
    const int H = NC / 2;
    seg = 16 * t >= H;
    n = blk * H + 16 * t - seg * H;
    ok = n < a.n_rows;
    if (!ok) n = 0;
  } else {
    n = blk * NC + 16 * t;
    ok = n < a.n_rows;
    if (!ok) n = 0;
    const int b1 = a.n_seg[0], b2 = b1 + a.n_seg[1];
    seg = n < b1 ? 0 : (n < b2 ? 1 : 2);
    n -= seg == 0 ? 0 : (seg == 1 ? b1 : b2);
  }
  return (const uint16_t*)a.w[seg] + (size_t)(n / 16) * KS * 512;
}

// ---------------------------------------------------------------- MFMA kernel (bf16 weights)
// Persistent: one 16-wave block per CU loops over row tiles of NC = 16*T
// weight rows (tile = blockIdx.x + i*gridDim.x).  Within a tile, wave w
// reduces k-steps [w*KS/16, (w+1)*KS/16) of 32 columns each, UB k-steps per
// register buffer; the next buffer -- including the first one of the next
// tile -- is loaded while the current one is multiplied, so the weight
// stream keeps going through the cross-wave reduction and the epilogue.
// MFMA operand layout (16x16x32): lane l holds A[l%16][8(l/16)+j] (x rows),
// B[8(l/16)+j][l%16] (= W[n0 + l%16][k0 + 8(l/16) + j]: 16 bytes at lane*16 of
// the packed 1 KB fragment), D[4(l/16)+r][l%16].
template <int T, int MT, int UB, bool PIPE, int KIND>
__global__ __launch_bounds__(kMfmaThreads) void gemm_bf16_mfma(GemmArgs a, int n_tiles) {
  constexpr int NC = 16 * T;
  constexpr int MP = 16 * MT;
  constexpr int NF = T * MT;              // accumulator fragments per wave
  constexpr int RR = NF <= 2 ? NF : 2;    // fragments reduced per LDS round
  __shared__ float red[RR][kMfmaWaves][kWave][4];
  __shared__ float yfin[MP][NC + 1];
  __shared__ float scale[MP];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int kg = lane >> 4, mrow = lane & 15;
  const int K = a.K;
  const int KS = (K + 31) / 32;
#ifdef SPECDEC_KSTEP_CONTIGUOUS
  const int ks0 = (wave * KS) / kMfmaWaves, ks1 = ((wave + 1) * KS) / kMfmaWaves;
  const int kstride = 1;
#else
  // k-steps interleaved across waves (wave w: w, w+16, ...): at any moment the
  // block reads 16 consecutive k-steps = 1 KB contiguous of each of its rows.
  const int ks0 = wave, ks1 = KS;
  const int kstride = kMfmaWaves;
#endif
  const int my_ks = ks1 > ks0 ? (ks1 - ks0 + kstride - 1) / kstride : 0;
  const int nbat = max(1, (my_ks + UB - 1) / UB);
  const int my_tiles = (n_tiles - (int)blockIdx.x + (int)gridDim.x - 1) / (int)gridDim.x;
  const int total = my_tiles * nbat;

  floatx4 acc[T][MT];
#pragma unroll
  for (int t = 0; t < T; ++t)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) acc[t][mt] = floatx4{0.f, 0.f, 0.f, 0.f};

  u32x4 wA[UB][T], wB[UB][T];
  f32x4 xA[UB][MT][2], xB[UB][MT][2];
  // load the q-th batch of this wave's work list (tile q / nbat, k-steps from (q % nbat) * UB)
  auto load = [&](int q, u32x4 (&wv)[UB][T], f32x4 (&xv)[UB][MT][2]) {
    const int tile = blockIdx.x + (q / nbat) * gridDim.x;
    const int kb = (q % nbat) * UB;  // index into this wave's k-step list
    const uint16_t* wtile[T];
    bool rok[T];
#pragma unroll
    for (int t = 0; t < T; ++t) wtile[t] = weight_tile(a, KIND, tile, NC, t, KS, rok[t]) + lane * 8;
#pragma unroll
    for (int u = 0; u < UB; ++u) {
      const int ks = ks0 + (kb + u) * kstride;
      const int k = ks * 32 + kg * 8;
      const bool kok = (kb + u) < my_ks && ks < KS;
#pragma unroll
      for (int t = 0; t < T; ++t) {
        if (kok && rok[t]) wv[u][t] = __builtin_nontemporal_load((const u32x4*)(wtile[t] + (size_t)ks * 512));
        else wv[u][t] = u32x4{0u, 0u, 0u, 0u};
      }
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        const int m = mt * 16 + mrow;
        if (kok && k < K && m < a.M) {
          const f32x4* xp = (const f32x4*)(a.x + (size_t)m * a.ldx + k);
          xv[u][mt][0] = xp[0];
          xv[u][mt][1] = xp[1];
        } else {
          xv[u][mt][0] = f32x4{0.f, 0.f, 0.f, 0.f};
          xv[u][mt][1] = f32x4{0.f, 0.f, 0.f, 0.f};
        }
      }
    }
  };
  auto compute = [&](u32x4 (&wv)[UB][T], f32x4 (&xv)[UB][MT][2]) {
#pragma unroll
    for (int u = 0; u < UB; ++u) {
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        bf16x8 hi, lo;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const float v = xv[u][mt][j >> 2][j & 3];
          const __bf16 h = (__bf16)v;
          hi[j] = h;
          lo[j] = (__bf16)(v - (float)h);
        }
#pragma unroll
        for (int t = 0; t < T; ++t) {
          const bf16x8 b = __builtin_bit_cast(bf16x8, wv[u][t]);
          acc[t][mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(hi, b, acc[t][mt], 0, 0, 0);
          acc[t][mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(lo, b, acc[t][mt], 0, 0, 0);
        }
      }
    }
  };
  // After the last batch of a tile: cross-wave reduction (fixed wave order) and epilogue.
  auto finish = [&](int q) {
    if (q % nbat != nbat - 1) return;
    const int tile = blockIdx.x + (q / nbat) * gridDim.x;
#pragma unroll
    for (int f0 = 0; f0 < NF; f0 += RR) {
#pragma unroll
      for (int f = 0; f < RR; ++f) {
        if (f0 + f < NF) {
          const int t = (f0 + f) / MT, mt = (f0 + f) % MT;
#pragma unroll
          for (int r = 0; r < 4; ++r) red[f][wave][lane][r] = acc[t][mt][r];
        }
      }
      __syncthreads();
      if (tid < 256 * RR && f0 + (tid >> 8) < NF) {
        const int f = tid >> 8, l = tid & 63, r = (tid >> 6) & 3;
        const int t = (f0 + f) / MT, mt = (f0 + f) % MT;
        float s = 0.f;
#pragma unroll
        for (int w = 0; w < kMfmaWaves; ++w) s += red[f][w][l][r];
        yfin[mt * 16 + 4 * (l >> 4) + r][t * 16 + (l & 15)] = s;
      }
      __syncthreads();
    }
#pragma unroll
    for (int t = 0; t < T; ++t)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) acc[t][mt] = floatx4{0.f, 0.f, 0.f, 0.f};
    epilogue<NC, KIND>(a, tile, yfin, scale);
    __syncthreads();  // yfin is reused by the next tile
  };

  int q = 0;
  if (total > 0) load(0, wA, xA);
  // The row scale is only needed by the epilogue: computed while the first loads fly.
  row_scale<MP>(a, scale);
  if (PIPE) {
    while (q < total) {
      if (q + 1 < total) load(q + 1, wB, xB);
      compute(wA, xA);
      finish(q);
      if (++q >= total) break;
      if (q + 1 < total) load(q + 1, wA, xA);
      compute(wB, xB);
      finish(q);
      ++q;
    }
  } else {
    for (; q < total; ++q) {
      if (q > 0) load(q, wA, xA);
      compute(wA, xA);
      finish(q);
    }
  }
}

// ---------------------------------------------------------------- vector kernel (float32 weights)
// Block = 4 waves over NC weight rows; each wave takes NC/4 rows, lanes stride
// over K; M processed 8 rows at a time.
template <int NC, int KIND>
__global__ __launch_bounds__(256) void gemm_f32_vector(GemmArgs a) {
  constexpr int MPMAX = kMaxGemmRows;
  __shared__ float yfin[MPMAX][NC + 1];
  __shared__ float scale[MPMAX];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int blk = blockIdx.x;
  row_scale<MPMAX>(a, scale);
  for (int c = wave; c < NC; c += 4) {
    bool ok;
    const float* wr = weight_row<float>(a, KIND, blk, NC, c, ok);
    for (int m0 = 0; m0 < a.M; m0 += 8) {
      float acc[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) acc[i] = 0.f;
      if (ok) {
        for (int k = lane; k < a.K; k += kWave) {
          float w = wr[k];
#pragma unroll
          for (int i = 0; i < 8; ++i)
            if (m0 + i < a.M) acc[i] += w * a.x[(size_t)(m0 + i) * a.ldx + k];
        }
      }
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        float s = wave_sum(acc[i]);
        if (lane == 0 && m0 + i < a.M) yfin[m0 + i][c] = s;
      }
    }
  }
  __syncthreads();
  epilogue<NC, KIND>(a, blk, yfin, scale);
}

// k-steps per register buffer and whether two buffers are kept (the next
// batch's loads in flight while the current one is multiplied): chosen so W
// and x fragments stay within the 128 VGPRs a wave of a 16-wave block may use.
template <int T, int MT> struct Batch;
template <> struct Batch<1, 1> { static constexpr int UB = 3; static constexpr bool PIPE = true; };
template <> struct Batch<1, 2> { static constexpr int UB = 2; static constexpr bool PIPE = true; };
template <> struct Batch<1, 4> { static constexpr int UB = 2; static constexpr bool PIPE = false; };
template <> struct Batch<2, 1> { static constexpr int UB = 2; static constexpr bool PIPE = true; };
template <> struct Batch<2, 2> { static constexpr int UB = 1; static constexpr bool PIPE = true; };
template <> struct Batch<2, 4> { static constexpr int UB = 1; static constexpr bool PIPE = false; };
template <> struct Batch<3, 1> { static constexpr int UB = 1; static constexpr bool PIPE = true; };
template <> struct Batch<3, 2> { static constexpr int UB = 1; static constexpr bool PIPE = true; };
template <> struct Batch<3, 4> { static constexpr int UB = 1; static constexpr bool PIPE = false; };

int compute_units() {
  static int cus = [] {
    int dev = 0, n = 0;
    if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) !=
                                                 hipSuccess || n <= 0)
      n = 256;
    return n;
  }();
  return cus;
}

template <int T, int MT, int KIND>
void launch_mfma_mt(const GemmArgs& a, int tiles, hipStream_t s) {
  const int grid = tiles < compute_units() ? tiles : compute_units();
  hipLaunchKernelGGL((gemm_bf16_mfma<T, MT, Batch<T, MT>::UB, Batch<T, MT>::PIPE, KIND>), dim3(grid),
                     dim3(kMfmaThreads), 0, s, a, tiles);
}

template <int T, int KIND>
hipError_t launch_mfma_t(const GemmArgs& a, int blocks, hipStream_t s) {
  const int MT = (a.M + 15) / 16;
  if (MT <= 1) launch_mfma_mt<T, 1, KIND>(a, blocks, s);
  else if (MT <= 2) launch_mfma_mt<T, 2, KIND>(a, blocks, s);
  else if (MT <= 4) launch_mfma_mt<T, 4, KIND>(a, blocks, s);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

// 16-row tiles per work unit of the bf16 kernel.  More tiles per unit mean
// fewer activation loads per weight byte; the choice balances the units over
// the CUs of the persistent grid (ties go to the larger unit).  SwiGLU pairs
// a gate tile with an up tile.
int mfma_tiles(int kind, int n_rows) {
  if (kind == EPI_SWIGLU) return 2;
  const int cus = compute_units();
  int best = 1;
  double best_eff = 0.0;
  for (int T = 3; T >= 1; --T) {
    const int units = (n_rows + 16 * T - 1) / (16 * T);
    const int rounds = (units + cus - 1) / cus;
    const double eff = (double)units / ((double)rounds * cus);
    if (eff > best_eff + 1e-9) {
      best_eff = eff;
      best = T;
    }
  }
  return best;
}

// One thread per 16-byte piece of the packed image of W [N, K] (row-major).
__global__ void pack_kernel(const uint16_t* __restrict__ src, uint16_t* __restrict__ dst, int N, int K, int KS) {
  const size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x;
  const size_t pieces = (size_t)(N / 16) * KS * 64;
  if (i >= pieces) return;
  const int lane = (int)(i % 64);
  const size_t frag = i / 64;
  const int ks = (int)(frag % KS), t = (int)(frag / KS);
  const int row = 16 * t + (lane & 15), k = 32 * ks + 8 * (lane >> 4);
  u32x4 v = u32x4{0u, 0u, 0u, 0u};
  if (k + 8 <= K) {
    v = *(const u32x4*)(src + (size_t)row * K + k);
  } else {
    uint16_t e[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) e[j] = k + j < K ? src[(size_t)row * K + k + j] : 0;
    v = u32x4{e[0] | (uint32_t)e[1] << 16, e[2] | (uint32_t)e[3] << 16, e[4] | (uint32_t)e[5] << 16,
              e[6] | (uint32_t)e[7] << 16};
  }
  *(u32x4*)(dst + i * 8) = v;
}

}  // namespace

size_t packed_elems(int N, int K) { return (size_t)(N / 16) * ((K + 31) / 32) * 512; }

hipError_t launch_pack(const void* src, void* dst, int N, int K, hipStream_t s) {
  if (N % 16 || K % 8) return hipErrorInvalidValue;
  const int KS = (K + 31) / 32;
  const size_t pieces = (size_t)(N / 16) * KS * 64;
  hipLaunchKernelGGL(pack_kernel, dim3((unsigned)((pieces + 255) / 256)), dim3(256), 0, s, (const uint16_t*)src,
                     (uint16_t*)dst, N, K, KS);
  return hipGetLastError();
}

int gemm_row_blocks(int dtype, int kind, int n_rows, int M) {
  (void)M;
  if (dtype == SPECDEC_BF16) {
    int nc = 16 * mfma_tiles(kind, n_rows);
    int per = kind == EPI_SWIGLU ? nc / 2 : nc;
    return (n_rows + per - 1) / per;
  }
  int per = kind == EPI_SWIGLU ? 16 : 16;
  return (n_rows + per - 1) / per;
}

hipError_t launch_gemm(int dtype, const GemmArgs& a, hipStream_t s) {
  if (a.M <= 0 || a.M > kMaxGemmRows || (a.K % 8) != 0 || (a.ldx % 4) != 0) return hipErrorInvalidValue;
  const int blocks = gemm_row_blocks(dtype, a.kind, a.n_rows, a.M);
  if (dtype == SPECDEC_BF16) {
    const int T = mfma_tiles(a.kind, a.n_rows);
    switch (a.kind) {
      case EPI_STORE:
        return T == 1 ? launch_mfma_t<1, EPI_STORE>(a, blocks, s)
                      : (T == 2 ? launch_mfma_t<2, EPI_STORE>(a, blocks, s) : launch_mfma_t<3, EPI_STORE>(a, blocks, s));
      case EPI_RESID:
        return T == 1 ? launch_mfma_t<1, EPI_RESID>(a, blocks, s)
                      : (T == 2 ? launch_mfma_t<2, EPI_RESID>(a, blocks, s) : launch_mfma_t<3, EPI_RESID>(a, blocks, s));
      case EPI_SWIGLU: return launch_mfma_t<2, EPI_SWIGLU>(a, blocks, s);
    }
    return hipErrorInvalidValue;
  }
  switch (a.kind) {
    case EPI_STORE: hipLaunchKernelGGL((gemm_f32_vector<16, EPI_STORE>), dim3(blocks), dim3(256), 0, s, a); break;
    case EPI_RESID: hipLaunchKernelGGL((gemm_f32_vector<16, EPI_RESID>), dim3(blocks), dim3(256), 0, s, a); break;
    case EPI_SWIGLU: hipLaunchKernelGGL((gemm_f32_vector<32, EPI_SWIGLU>), dim3(blocks), dim3(256), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace specdec
