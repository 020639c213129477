// RoPE + KV append and GQA attention of the verify / draft passes against the
// resident KV cache.
//
// KV layout (per layer l, sequence b, kv head g), storage type KT:
//   K block [capacity][head_dim]  (row = position)
//   V block [head_dim][capacity]  (transposed: a row = one dimension over positions)
// at element offset ((l*B + b)*h_kv + g) * 2*capacity*head_dim (V after K).
// The transposed V makes both operands of softmax(QK^T)V read contiguous
// position runs.
//
// Attention is split over key chunks (flash-decoding style): one block per
// (chunk, kv head, sequence) computes, for every query row of the sequence
// and every query head of the kv group, the chunk's max, exp-sum and
// unnormalised P V; a combine kernel merges the chunks per (row, head).  Query
// i of a sequence at position pos_i sees keys 0..pos_i (causal inside the
// verify block).
#include "device_common.h"
#include "internal.h"

namespace specdec {

namespace {

template <typename KT>
__device__ __forceinline__ KT* k_block(const KvLayout& kv, int layer, int b, int g) {
  size_t off = (((size_t)layer * kv.batch + b) * kv.n_kv_heads + g) * 2 * (size_t)kv.capacity * kv.head_dim;
  return (KT*)kv.data + off;
}

// ---------------------------------------------------------------- RoPE + append
template <typename KT>
__global__ __launch_bounds__(256) void rope_append_kernel(AttnArgs a) {
  const int r = blockIdx.x;
  const RowDesc rd = a.rows[r];
  const int hd = a.head_dim, half = hd / 2, H = a.n_heads, G = a.n_kv_heads;
  const float* cs = a.rope_cs + (size_t)r * hd;
  const float* src = a.qkv + (size_t)r * (H + 2 * G) * hd;
  float* qr = a.qr + (size_t)r * H * hd;
  for (int i = threadIdx.x; i < H * half; i += blockDim.x) {
    const int head = i / half, j = i % half;
    const float x1 = src[head * hd + j], x2 = src[head * hd + j + half];
    const float c = cs[j], s = cs[half + j];
    qr[head * hd + j] = x1 * c - x2 * s;
    qr[head * hd + j + half] = x2 * c + x1 * s;
  }
  if (!rd.valid) return;
  for (int i = threadIdx.x; i < G * half; i += blockDim.x) {
    const int g = i / half, j = i % half;
    const float* kp = src + (H + g) * hd;
    const float x1 = kp[j], x2 = kp[j + half];
    const float c = cs[j], s = cs[half + j];
    KT* kb = k_block<KT>(a.kv, a.layer, rd.b, g) + (size_t)rd.pos * hd;
    Storage<KT>::store(kb + j, x1 * c - x2 * s);
    Storage<KT>::store(kb + j + half, x2 * c + x1 * s);
  }
  for (int i = threadIdx.x; i < G * hd; i += blockDim.x) {
    const int g = i / hd, dd = i % hd;
    KT* vb = k_block<KT>(a.kv, a.layer, rd.b, g) + (size_t)a.kv.capacity * hd;
    Storage<KT>::store(vb + (size_t)dd * a.kv.capacity + rd.pos, src[(H + G + g) * hd + dd]);
  }
}

// ---------------------------------------------------------------- split-KV partials
constexpr int kQB = 16;  // queries per pass

template <typename KT>
__global__ __launch_bounds__(256) void attn_partial_kernel(AttnArgs a) {
  extern __shared__ float smem[];
  const int c = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
  const int hd = a.head_dim, H = a.n_heads, G = a.n_kv_heads, group = H / G;
  const int rps = a.rps, r0 = b * rps, chunk = a.chunk;
  int nk = 0;
  for (int i = 0; i < rps; ++i) {
    const RowDesc rd = a.rows[r0 + i];
    if (rd.valid) nk = max(nk, rd.pos + 1);
  }
  const int kbeg = c * chunk;
  if (kbeg >= nk) return;
  const int nkeys = min(chunk, nk - kbeg);

  float* Ks = smem;                           // [chunk][hd+1]
  float* Vs = Ks + chunk * (hd + 1);          // [hd][chunk+1]
  float* qs = Vs + hd * (chunk + 1);          // [kQB][hd]
  float* S = qs + kQB * hd;                   // [kQB][chunk]
  float* ml = S + kQB * chunk;                // [kQB][2]

  const KT* kb = k_block<KT>(a.kv, a.layer, b, g);
  const KT* vb = kb + (size_t)a.kv.capacity * hd;
  for (int i = threadIdx.x; i < nkeys * hd; i += blockDim.x) {
    const int key = i / hd, dd = i % hd;
    Ks[key * (hd + 1) + dd] = Storage<KT>::load(kb + (size_t)(kbeg + key) * hd + dd);
  }
  for (int i = threadIdx.x; i < hd * nkeys; i += blockDim.x) {
    const int dd = i / nkeys, key = i % nkeys;
    Vs[dd * (chunk + 1) + key] = Storage<KT>::load(vb + (size_t)dd * a.kv.capacity + kbeg + key);
  }
  const float scale = 1.0f / sqrtf((float)hd);
  const int nq = rps * group;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;

  for (int qb = 0; qb < nq; qb += kQB) {
    __syncthreads();  // tiles loaded / previous pass done with qs, S
    for (int i = threadIdx.x; i < kQB * hd; i += blockDim.x) {
      const int ql = i / hd, dd = i % hd, qi = qb + ql;
      float v = 0.f;
      if (qi < nq) {
        const int row = r0 + qi / group, head = g * group + qi % group;
        v = a.qr[((size_t)row * H + head) * hd + dd];
      }
      qs[i] = v;
    }
    __syncthreads();
    for (int p = threadIdx.x; p < kQB * chunk; p += blockDim.x) {
      const int ql = p / chunk, key = p % chunk, qi = qb + ql;
      float s = -INFINITY;
      if (qi < nq && key < nkeys) {
        const RowDesc rd = a.rows[r0 + qi / group];
        if (rd.valid && kbeg + key <= rd.pos) {
          const float* qv = qs + ql * hd;
          const float* kv = Ks + key * (hd + 1);
          float t = 0.f;
          for (int dd = 0; dd < hd; ++dd) t += qv[dd] * kv[dd];
          s = t * scale;
        }
      }
      S[p] = s;
    }
    __syncthreads();
    for (int ql = wave; ql < kQB; ql += 4) {
      float mx = -INFINITY;
      for (int key = lane; key < chunk; key += kWave) mx = fmaxf(mx, S[ql * chunk + key]);
      mx = wave_max(mx);
      float sum = 0.f;
      for (int key = lane; key < chunk; key += kWave) {
        const float s = S[ql * chunk + key];
        const float e = (mx == -INFINITY) ? 0.f : expf(s - mx);
        S[ql * chunk + key] = e;
        sum += e;
      }
      sum = wave_sum(sum);
      if (lane == 0) { ml[2 * ql] = mx; ml[2 * ql + 1] = sum; }
    }
    __syncthreads();
    for (int p = threadIdx.x; p < kQB * hd; p += blockDim.x) {
      const int ql = p / hd, dd = p % hd, qi = qb + ql;
      if (qi >= nq || ml[2 * ql] == -INFINITY) continue;
      const float* pr = S + ql * chunk;
      const float* vr = Vs + dd * (chunk + 1);
      float o = 0.f;
      for (int key = 0; key < nkeys; ++key) o += pr[key] * vr[key];
      const int row = r0 + qi / group, head = g * group + qi % group;
      const size_t slot = ((size_t)row * H + head) * a.n_split + c;
      a.o_part[slot * hd + dd] = o;
      if (dd == 0) { a.ml_part[2 * slot] = ml[2 * ql]; a.ml_part[2 * slot + 1] = ml[2 * ql + 1]; }
    }
  }
}

// ---------------------------------------------------------------- combine
__global__ __launch_bounds__(128) void attn_combine_kernel(AttnArgs a) {
  const int head = blockIdx.x, r = blockIdx.y;
  const int hd = a.head_dim, H = a.n_heads;
  const RowDesc rd = a.rows[r];
  float* o = a.o + ((size_t)r * H + head) * hd;
  if (!rd.valid) {
    for (int dd = threadIdx.x; dd < hd; dd += blockDim.x) o[dd] = 0.f;
    return;
  }
  int nch = (rd.pos + 1 + a.chunk - 1) / a.chunk;
  if (nch > a.n_split) {  // the host's bound on the context was wrong: report, stay in bounds
    if (threadIdx.x == 0) set_status(a.status, kStatusKvCapacity);
    nch = a.n_split;
  }
  const size_t base = ((size_t)r * H + head) * a.n_split;
  float mx = -INFINITY;
  for (int c = 0; c < nch; ++c) mx = fmaxf(mx, a.ml_part[2 * (base + c)]);
  float L = 0.f;
  for (int c = 0; c < nch; ++c) L += expf(a.ml_part[2 * (base + c)] - mx) * a.ml_part[2 * (base + c) + 1];
  const float inv = 1.0f / L;
  for (int dd = threadIdx.x; dd < hd; dd += blockDim.x) {
    float acc = 0.f;
    for (int c = 0; c < nch; ++c) acc += expf(a.ml_part[2 * (base + c)] - mx) * a.o_part[(base + c) * hd + dd];
    o[dd] = acc * inv;
  }
}

// ---------------------------------------------------------------- KV context copy
template <typename KT>
__global__ __launch_bounds__(256) void kv_copy_kernel(KvLayout kv, int layer, int b, int pos0, const KT* k,
                                                      const KT* v, KT* k_out, KT* v_out) {
  const int p = blockIdx.x;
  const int hd = kv.head_dim, G = kv.n_kv_heads;
  for (int i = threadIdx.x; i < G * hd; i += blockDim.x) {
    const int g = i / hd, dd = i % hd;
    KT* kb = k_block<KT>(kv, layer, b, g);
    KT* vb = kb + (size_t)kv.capacity * hd;
    KT* kc = kb + (size_t)(pos0 + p) * hd + dd;
    KT* vc = vb + (size_t)dd * kv.capacity + pos0 + p;
    const size_t src = ((size_t)p * G + g) * hd + dd;
    if (k) *kc = k[src];
    if (v) *vc = v[src];
    if (k_out) k_out[src] = *kc;
    if (v_out) v_out[src] = *vc;
  }
}

size_t attn_smem_bytes(int chunk, int hd) {
  return sizeof(float) * ((size_t)chunk * (hd + 1) + (size_t)hd * (chunk + 1) + kQB * hd + kQB * chunk + 2 * kQB);
}

}  // namespace

int attention_chunk(int head_dim) { return head_dim >= 128 ? 32 : (head_dim >= 64 ? 64 : 128); }

hipError_t launch_rope_append(const AttnArgs& a, hipStream_t s) {
  if (a.kv.dtype == SPECDEC_BF16)
    hipLaunchKernelGGL((rope_append_kernel<uint16_t>), dim3(a.M), dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL((rope_append_kernel<float>), dim3(a.M), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_attention(const AttnArgs& a, hipStream_t s) {
  const int B = a.M / a.rps;
  const size_t smem = attn_smem_bytes(a.chunk, a.head_dim);
  dim3 grid(a.n_split, a.n_kv_heads, B);
  if (a.kv.dtype == SPECDEC_BF16)
    hipLaunchKernelGGL((attn_partial_kernel<uint16_t>), grid, dim3(256), smem, s, a);
  else
    hipLaunchKernelGGL((attn_partial_kernel<float>), grid, dim3(256), smem, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(attn_combine_kernel, dim3(a.n_heads, a.M), dim3(128), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_kv_copy(const KvLayout& kv, int layer, int b, int pos0, int n, const void* k, const void* v,
                          void* k_out, void* v_out, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  if (kv.dtype == SPECDEC_BF16)
    hipLaunchKernelGGL((kv_copy_kernel<uint16_t>), dim3(n), dim3(256), 0, s, kv, layer, b, pos0,
                       (const uint16_t*)k, (const uint16_t*)v, (uint16_t*)k_out, (uint16_t*)v_out);
  else
    hipLaunchKernelGGL((kv_copy_kernel<float>), dim3(n), dim3(256), 0, s, kv, layer, b, pos0, (const float*)k,
                       (const float*)v, (float*)k_out, (float*)v_out);
  return hipGetLastError();
}

}  // namespace specdec
