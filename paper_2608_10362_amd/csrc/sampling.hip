// Row set-up + embedding gather, the draft's sampling step, the speculative
// accept / resample decision, the fixed-point sampler, Philox draws and the
// KV commit.
//
// Sampling reading (shared with the host documentation in specdec.h): a draw
// from non-negative weights r_j uses R_j = floor(r_j * 2^40) as uint64,
// S = sum R_j, t = floor(x * S / 2^32) for a 32-bit word x, and returns the
// smallest j with R_0 + ... + R_j > t.  Every sum is an integer sum, so the
// result does not depend on how the block splits and orders the reduction.
#include "device_common.h"
#include "internal.h"

namespace specdec {

namespace {

constexpr int kSampThreads = 1024;
constexpr int kMaxGamma = 31;

__device__ __forceinline__ uint64_t fp_weight(float r) {
  return r > 0.f ? (uint64_t)(r * 1099511627776.0f) : 0ull;  // exact: r * 2^40, truncation = floor
}
// floor(x * S / 2^32) without a 128-bit product (S < 2^56, x < 2^32).
__device__ __forceinline__ uint64_t scale_word(uint32_t x, uint64_t S) {
  return (uint64_t)x * (S >> 32) + (((uint64_t)x * (S & 0xffffffffull)) >> 32);
}

__device__ __forceinline__ uint64_t shfl_up_u64(uint64_t v, int o) {
  uint32_t lo = __shfl_up((uint32_t)v, o, kWave), hi = __shfl_up((uint32_t)(v >> 32), o, kWave);
  return ((uint64_t)hi << 32) | lo;
}

struct SampShared {
  uint64_t wave_tot[kSampThreads / kWave];
  int token;
};

// Block-wide fixed-point draw over j < V with weights rf(j) (floats >= 0).
// Wave w owns the contiguous segment [w*seg, (w+1)*seg) (seg a multiple of
// 64); lanes read it with unit stride.  Pass 1 sums the integer weights per
// wave; the wave whose range of the running sum holds t then scans its
// segment 64 entries at a time.  Returns the token (same value in every
// thread), or -1 when all weights are zero.
template <typename RF>
__device__ int block_draw(RF rf, int V, uint32_t x, SampShared& sh) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, nw = blockDim.x / kWave;
  const int seg = ((V + nw - 1) / nw + kWave - 1) / kWave * kWave;
  const int j0 = min(V, wave * seg), j1 = min(V, j0 + seg);
  uint64_t mine = 0;
  for (int j = j0 + lane; j < j1; j += kWave) mine += fp_weight(rf(j));
  mine = wave_sum_u64(mine);
  __syncthreads();
  if (lane == 0) sh.wave_tot[wave] = mine;
  if (tid == 0) sh.token = -1;
  __syncthreads();
  uint64_t before = 0, total = 0;
  for (int w = 0; w < nw; ++w) {
    if (w < wave) before += sh.wave_tot[w];
    total += sh.wave_tot[w];
  }
  if (total != 0) {
    const uint64_t t = scale_word(x, total);
    if (mine != 0 && before <= t && t < before + mine) {
      uint64_t cum0 = before;
      for (int c = j0; c < j1; c += kWave) {
        const int j = c + lane;
        uint64_t incl = j < j1 ? fp_weight(rf(j)) : 0ull;
#pragma unroll
        for (int o = 1; o < kWave; o <<= 1) {
          const uint64_t n = shfl_up_u64(incl, o);
          if (lane >= o) incl += n;
        }
        const unsigned long long hit = __ballot(cum0 + incl > t);
        if (hit) {
          const int first = __ffsll(hit) - 1;
          if (lane == 0) sh.token = c + first;
          break;
        }
        cum0 += __shfl(incl, kWave - 1, kWave);
      }
    }
  }
  __syncthreads();
  return sh.token;
}

// Online (max, sum exp) of z_j = row[j] / T over a row, block-wide, one pass.
// Elements are read four at a time when the row is 16-byte aligned.  The
// per-thread states are merged in a fixed order (deterministic).
struct MaxSum {
  float m, s;
};
__device__ __forceinline__ void ms_add(MaxSum& a, float z) {
  if (z > a.m) {
    a.s = a.s * expf(a.m - z) + 1.0f;
    a.m = z;
  } else {
    a.s += expf(z - a.m);
  }
}
__device__ __forceinline__ MaxSum ms_merge(MaxSum a, MaxSum b) {
  if (b.m == -INFINITY) return a;
  if (a.m == -INFINITY) return b;
  const float m = fmaxf(a.m, b.m);
  return MaxSum{m, a.s * expf(a.m - m) + b.s * expf(b.m - m)};
}
__device__ MaxSum block_max_sum(const float* row, int V, float T, float* red2) {
  const int tid = threadIdx.x, nt = blockDim.x, lane = tid & 63, wave = tid >> 6, nw = nt / kWave;
  MaxSum st{-INFINITY, 0.f};
  if ((V & 3) == 0 && ((uintptr_t)row & 15) == 0) {
    const f32x4* r4 = (const f32x4*)row;
    const int V4 = V >> 2;
    int j = tid;
    for (; j + 3 * nt < V4; j += 4 * nt) {
      f32x4 v[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) v[u] = r4[j + u * nt];
#pragma unroll
      for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int e = 0; e < 4; ++e) ms_add(st, v[u][e] / T);
    }
    for (; j < V4; j += nt) {
      const f32x4 v = r4[j];
#pragma unroll
      for (int e = 0; e < 4; ++e) ms_add(st, v[e] / T);
    }
  } else {
    for (int j = tid; j < V; j += nt) ms_add(st, row[j] / T);
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    MaxSum other{__shfl_xor(st.m, o, kWave), __shfl_xor(st.s, o, kWave)};
    st = ms_merge(st, other);
  }
  __syncthreads();
  if (lane == 0) { red2[2 * wave] = st.m; red2[2 * wave + 1] = st.s; }
  __syncthreads();
  MaxSum tot{red2[0], red2[1]};
  for (int w = 1; w < nw; ++w) tot = ms_merge(tot, MaxSum{red2[2 * w], red2[2 * w + 1]});
  return tot;
}

// ---------------------------------------------------------------- rows + embedding
template <typename ET>
__global__ __launch_bounds__(256) void rows_embed_kernel(RowsArgs a) {
  __shared__ float red[16];
  const int r = blockIdx.x, b = r / a.rps, i = r % a.rps;
  int pos = 0, tok = 0, valid = 1;
  switch (a.mode) {
    case ROWS_VERIFY:
      pos = a.len[b] + i;
      tok = i == 0 ? a.pending[2 * b + 1] : a.tok_src[(size_t)b * a.ld_tok + i - 1];
      break;
    case ROWS_DRAFT_FIRST: {
      const int np = a.n_pending[b];
      valid = i >= 2 - np;
      pos = a.len[b] + i - (2 - np);
      tok = a.pending[2 * b + i];
      break;
    }
    case ROWS_DRAFT_NEXT:
      pos = a.len[b] + a.n_pending[b] + a.slot - 1;
      tok = a.tok_src[(size_t)b * a.ld_tok + a.slot - 1];
      break;
    default:  // ROWS_PREFILL
      pos = a.len[b] + a.c0 + i;
      tok = a.tok_src[(size_t)b * a.ld_tok + a.c0 + i];
      break;
  }
  if (valid) {
    if (tok < 0 || tok >= a.vocab) {
      if (threadIdx.x == 0) set_status(a.status, kStatusBadToken);
      valid = 0;
    }
    if (pos < 0 || pos >= a.capacity) {
      if (threadIdx.x == 0) set_status(a.status, kStatusKvCapacity);
      valid = 0;
    }
  }
  if (!valid) {
    tok = 0;
    pos = 0;
  }
  if (threadIdx.x == 0) a.rows[r] = RowDesc{b, pos, tok, valid};
  const int hd = a.head_dim, half = hd / 2;
  for (int j = threadIdx.x; j < half; j += blockDim.x) {
    const double inv_freq = pow(a.rope_base, -2.0 * (double)j / (double)hd);
    const double ang = (double)pos * inv_freq;
    a.rope_cs[(size_t)r * hd + j] = (float)cos(ang);
    a.rope_cs[(size_t)r * hd + half + j] = (float)sin(ang);
  }
  const ET* e = (const ET*)a.embed + (size_t)tok * a.d_model;
  const ET* gn = (const ET*)a.gain;
  float* h = a.h + (size_t)r * a.d_model;
  float* xg = a.xg + (size_t)r * a.d_model;
  float ss = 0.f;
  for (int k = threadIdx.x; k < a.d_model; k += blockDim.x) {
    const float v = Storage<ET>::load(e + k);
    h[k] = v;
    xg[k] = v * Storage<ET>::load(gn + k);
    ss += v * v;
  }
  ss = block_sum(ss, red);
  if (threadIdx.x == 0) a.ss[r] = ss;
}

// ---------------------------------------------------------------- draft finish
__global__ __launch_bounds__(kSampThreads) void draft_finish_kernel(DraftFinishArgs a) {
  __shared__ float redf[16];
  __shared__ float red2[32];
  __shared__ int redi[16];
  __shared__ SampShared sh;
  const int b = blockIdx.x, V = a.V, tid = threadIdx.x, nt = blockDim.x;
  const float* lg = a.logits + ((size_t)b * a.rps + a.rps - 1) * V;
  bool bad = false;
  for (int j = tid; j < V; j += nt) {
    const float v = lg[j];
    bad |= !isfinite(v);
    if (a.logits_out) a.logits_out[(size_t)b * V + j] = v;
  }
  if (__syncthreads_or(bad)) {
    if (tid == 0) {
      set_status(a.status, kStatusNonFinite);
      a.d_out[(size_t)b * a.ld_d + a.slot] = 0;
    }
    return;
  }
  int tok;
  if (a.temperature == 0.f) {
    float bv = -INFINITY;
    int bi = 0x7fffffff;
    for (int j = tid; j < V; j += nt)
      if (lg[j] > bv) { bv = lg[j]; bi = j; }
    block_argmax(bv, bi, redf, redi);
    tok = bi;
  } else {
    const float T = a.temperature;
    const MaxSum st = block_max_sum(lg, V, T, red2);
    const float mx = st.m, s = st.s;
    auto qf = [&](int j) { return expf(lg[j] / T - mx) / s; };
    if (a.q_out) {
      float* qo = a.q_out + ((size_t)b * a.gamma + a.slot) * V;
      for (int j = tid; j < V; j += nt) qo[j] = qf(j);
    }
    const uint32_t x = a.rand ? a.rand[b] : draw_word(a.seed, b, a.step, SPECDEC_PURPOSE_DRAFT, a.slot);
    tok = block_draw(qf, V, x, sh);
  }
  if (tid == 0) a.d_out[(size_t)b * a.ld_d + a.slot] = tok;
}

// ---------------------------------------------------------------- accept / resample
__global__ __launch_bounds__(kSampThreads) void accept_kernel(AcceptArgs a) {
  __shared__ float redf[16];
  __shared__ float red2[32];
  __shared__ int redi[16];
  __shared__ float rmax[kMaxGamma + 1], rsum[kMaxGamma + 1];
  __shared__ SampShared sh;
  const int b = blockIdx.x, g = a.gamma, V = a.V, tid = threadIdx.x, nt = blockDim.x;
  const float* P = a.p + (size_t)b * (g + 1) * V;
  const float* Q = a.q ? a.q + (size_t)b * g * V : nullptr;
  const int32_t* d = a.d + (size_t)b * a.ld_d;
  auto word = [&](int i) -> uint32_t {
    if (a.rand) return a.rand[(size_t)b * (g + 1) + i];
    return i < g ? draw_word(a.seed, b, a.step, SPECDEC_PURPOSE_ACCEPT, i)
                 : draw_word(a.seed, b, a.step, SPECDEC_PURPOSE_RESAMPLE, 0);
  };
  bool bad = false;
  int A = g, next = -1;
  if (a.temperature == 0.f) {
    for (int i = 0; i <= g; ++i) {
      float bv = -INFINITY;
      int bi = 0x7fffffff;
      for (int j = tid; j < V; j += nt) {
        const float v = P[(size_t)i * V + j];
        bad |= !isfinite(v);
        if (v > bv) { bv = v; bi = j; }
      }
      block_argmax(bv, bi, redf, redi);
      if (i < g && bi != d[i]) { A = i; next = bi; break; }
      if (i == g) next = bi;
    }
    bad = __syncthreads_or(bad);
  } else {
    const float T = a.temperature;
    const bool logits = a.input_kind == SPECDEC_INPUT_LOGITS;
    for (int i = 0; i <= g; ++i) {
      const float* row = P + (size_t)i * V;
      if (logits) {
        const MaxSum st = block_max_sum(row, V, T, red2);
        // a NaN/Inf logit makes the row's max or sum non-finite
        bad |= !isfinite(st.m) || !isfinite(st.s);
        if (tid == 0) { rmax[i] = st.m; rsum[i] = st.s; }
      } else {
        for (int j = tid; j < V; j += nt) bad |= !isfinite(row[j]);
      }
    }
    bad = __syncthreads_or(bad);
    auto pf = [&](int i, int j) -> float {
      const float v = P[(size_t)i * V + j];
      return logits ? expf(v / T - rmax[i]) / rsum[i] : v;
    };
    if (!bad) {
      for (int i = 0; i < g; ++i) {
        const int di = d[i];
        if (di < 0 || di >= V) { bad = true; break; }
        const float pd = pf(i, di), qd = Q[(size_t)i * V + di];
        if (!isfinite(qd)) { bad = true; break; }
        const float u = word_to_uniform(word(i));
        if (!(__fmul_rn(u, qd) < pd)) { A = i; break; }
      }
    }
    if (!bad && A < g) {
      bool badq = false;
      for (int j = tid; j < V; j += nt) badq |= !isfinite(Q[(size_t)A * V + j]);
      bad = __syncthreads_or(badq);
    }
    if (!bad) {
      const uint32_t x = word(g);
      if (A < g) {
        const float* qr = Q + (size_t)A * V;
        next = block_draw([&](int j) { return fmaxf(0.f, __fsub_rn(pf(A, j), qr[j])); }, V, x, sh);
        if (next < 0) next = block_draw([&](int j) { return pf(A, j); }, V, x, sh);
      } else {
        next = block_draw([&](int j) { return pf(g, j); }, V, x, sh);
      }
    }
  }
  if (tid == 0) {
    if (bad) {
      set_status(a.status, kStatusNonFinite);
      a.n_accepted[b] = -1;
      a.next_token[b] = -1;
    } else {
      a.n_accepted[b] = A;
      a.next_token[b] = next;
    }
  }
}

// ---------------------------------------------------------------- sampler / philox
__global__ __launch_bounds__(kSampThreads) void sample_kernel(int V, const float* probs, int64_t ld,
                                                              const uint32_t* rand, uint64_t seed, uint64_t step,
                                                              int purpose, int index, int32_t* out) {
  __shared__ SampShared sh;
  const int b = blockIdx.x;
  const float* row = probs + (size_t)b * ld;
  const uint32_t x = rand ? rand[b] : draw_word(seed, b, step, purpose, index);
  const int tok = block_draw([&](int j) { return row[j]; }, V, x, sh);
  if (threadIdx.x == 0) out[b] = tok;
}

__global__ void draw_kernel(int B, uint64_t seed, uint64_t step, int purpose, int index, uint32_t* out) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b < B) out[b] = draw_word(seed, b, step, purpose, index);
}

// ---------------------------------------------------------------- commit
__global__ void commit_kernel(CommitArgs a) {
  for (int b = threadIdx.x; b < a.B; b += blockDim.x) {
    const int A = a.n_accepted[b], g = a.gamma;
    if (A < 0 || A > g) continue;
    const int nxt = a.next_token[b];
    if (a.role == SPECDEC_ROLE_TARGET) {
      a.len[b] += A + 1;
      a.pending[2 * b] = 0;
      a.pending[2 * b + 1] = nxt;
      a.n_pending[b] = 1;
    } else {
      const int np = a.n_pending[b];
      a.len[b] += np + min(A, g - 1);
      if (A == g) {
        a.pending[2 * b] = a.d[(size_t)b * a.ld_d + g - 1];
        a.n_pending[b] = 2;
      } else {
        a.pending[2 * b] = 0;
        a.n_pending[b] = 1;
      }
      a.pending[2 * b + 1] = nxt;
    }
  }
}

}  // namespace

hipError_t launch_rows_embed(int dtype, const RowsArgs& a, hipStream_t s) {
  if (dtype == SPECDEC_BF16)
    hipLaunchKernelGGL((rows_embed_kernel<uint16_t>), dim3(a.M), dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL((rows_embed_kernel<float>), dim3(a.M), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_draft_finish(const DraftFinishArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(draft_finish_kernel, dim3(a.B), dim3(kSampThreads), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_accept(const AcceptArgs& a, hipStream_t s) {
  if (a.gamma > kMaxGamma) return hipErrorInvalidValue;
  hipLaunchKernelGGL(accept_kernel, dim3(a.B), dim3(kSampThreads), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_sample(int B, int V, const float* probs, int64_t ld, const uint32_t* rand, uint64_t seed,
                         uint64_t step, int purpose, int index, int32_t* out, hipStream_t s) {
  hipLaunchKernelGGL(sample_kernel, dim3(B), dim3(kSampThreads), 0, s, V, probs, ld, rand, seed, step, purpose,
                     index, out);
  return hipGetLastError();
}

hipError_t launch_draw(int B, uint64_t seed, uint64_t step, int purpose, int index, uint32_t* out, hipStream_t s) {
  hipLaunchKernelGGL(draw_kernel, dim3((B + 255) / 256), dim3(256), 0, s, B, seed, step, purpose, index, out);
  return hipGetLastError();
}

hipError_t launch_commit(const CommitArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(commit_kernel, dim3(1), dim3(64), 0, s, a);
  return hipGetLastError();
}

}  // namespace specdec
