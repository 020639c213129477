// Row set-up + embedding gather, the draft's sampling step, the speculative
// accept / resample decision, the fixed-point sampler, Philox draws and the
// KV commit.
//
// Sampling reading (shared with the host documentation in specdec.h): a draw
// from non-negative weights r_j uses R_j = floor(r_j * 2^40) as uint64,
// S = sum R_j, t = floor(x * S / 2^32) for a 32-bit word x, and returns the
// smallest j with R_0 + ... + R_j > t.  Every sum is an integer sum, so the
// result does not depend on how the block splits and orders the reduction.
#include <mutex>

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
    const float xv = v * Storage<ET>::load(gn + k);
    xg[k] = xv;
    if (a.xs) put_stacked(a.xs, a.stt, r, k, xv);
    ss += v * v;
  }
  ss = block_sum(ss, red);
  if (threadIdx.x == 0) a.ss[r] = ss;
}

// ---------------------------------------------------------------- multi-block softmax / accept / draw
// A vocabulary row is cut into NC chunks so that a single decision uses many
// CUs, in two launches:
//   stats         per (chunk, row): online (max, sum exp) of z = x / T, argmax, finiteness
//   decide-draw   per (chunk, sequence): every block merges the chunk statistics
//                 (fixed order) and takes the decision; each sums the integer
//                 weights of its chunk of the row to draw from (the draft's q is
//                 also written here); the last block of the sequence finds the
//                 chunk holding t, scans it and emits the token
constexpr int kChunkThreads = 256;

__host__ __device__ __forceinline__ int n_chunks(int V) {
  int nc = (V + 511) / 512;  // (512-entry chunks: 63 blocks per 32000-entry row; 1024 and 2048 were slower)
  return nc < 1 ? 1 : (nc > 64 ? 64 : nc);
}
__host__ __device__ __forceinline__ int chunk_size(int V) { return (V + n_chunks(V) - 1) / n_chunks(V); }

struct StatPart {
  float m, s, amax_v;
  int amax_i, bad, pad0, pad1, pad2;
};
struct DrawPart {
  unsigned long long res, prob;
};
// A sequence's decision, kept in LDS by every block of the decide-and-draw launch.
struct SeqState {
  int A;            // accepted count (-1 error, -2 no draw needed)
  int pad;
  float2 ms[kMaxGamma + 1];  // merged (max, sum) per row
};

struct Scratch {
  StatPart* stats;  // [rows_total][NC]
  DrawPart* draw;   // [B][NC]
  uint32_t* count;  // [B] blocks of the decide-and-draw launch done (zeroed by the stats launch)
};
__host__ __device__ inline size_t align256(size_t x) { return (x + 255) / 256 * 256; }
__host__ __device__ inline Scratch carve(void* base, int B, int rows, int V) {
  const int NC = n_chunks(V);
  char* p = (char*)base;
  Scratch s;
  s.stats = (StatPart*)p;
  p += align256(sizeof(StatPart) * (size_t)B * rows * NC);
  s.draw = (DrawPart*)p;
  p += align256(sizeof(DrawPart) * (size_t)B * NC);
  s.count = (uint32_t*)p;
  return s;
}

// p_i(j) of row i: softmax(l/T) from merged statistics, or the probability itself.
__device__ __forceinline__ float prob_of(const float* row, int j, bool logits, float T, float2 ms) {
  const float v = row[j];
  return logits ? expf(v / T - ms.x) / ms.y : v;
}

// stats: grid (NC, B * rows_per_seq), block 256.  Row i of sequence b is
// x + (b * row_stride + row_off + i) * V.
// Every value of the row, and of the row `chk` pairs with it (the draft's q
// row i of an accept, rows i < chk_rows), must be finite.
// It also zeroes the sequence's counter of the decide-and-draw launch that follows.
__global__ __launch_bounds__(kChunkThreads) void stats_kernel(const float* x, int V, int rows_per_seq, int row_stride,
                                                              int row_off, float T, const float* chk, int chk_rows,
                                                              StatPart* out, uint32_t* count) {
  __shared__ float sm_m[4], sm_s[4], sm_v[4];
  __shared__ int sm_i[4], sm_b[4];
  const int c = blockIdx.x, r = blockIdx.y, NC = gridDim.x;
  const int b = r / rows_per_seq, i = r % rows_per_seq;
  if (c == 0 && i == 0 && threadIdx.x == 0) count[b] = 0u;
  const float* row = x + ((size_t)b * row_stride + row_off + i) * V;
  const int cs = chunk_size(V), j0 = c * cs, j1 = min(V, j0 + cs);
  MaxSum st{-INFINITY, 0.f};
  float bv = -INFINITY;
  int bi = 0x7fffffff, bad = 0;
  for (int j = j0 + threadIdx.x; j < j1; j += kChunkThreads) {
    const float v = row[j];
    bad |= !isfinite(v);
    if (v > bv) { bv = v; bi = j; }
    if (T > 0.f) ms_add(st, v / T);
  }
  if (chk && i < chk_rows) {
    const float* crow = chk + ((size_t)b * chk_rows + i) * V;
    for (int j = j0 + threadIdx.x; j < j1; j += kChunkThreads) bad |= !isfinite(crow[j]);
  }
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    st = ms_merge(st, MaxSum{__shfl_xor(st.m, o, kWave), __shfl_xor(st.s, o, kWave)});
    const float ov = __shfl_xor(bv, o, kWave);
    const int oi = __shfl_xor(bi, o, kWave);
    if (ov > bv || (ov == bv && oi < bi)) { bv = ov; bi = oi; }
    bad |= __shfl_xor(bad, o, kWave);
  }
  if (lane == 0) { sm_m[w] = st.m; sm_s[w] = st.s; sm_v[w] = bv; sm_i[w] = bi; sm_b[w] = bad; }
  __syncthreads();
  if (threadIdx.x == 0) {
    MaxSum t{sm_m[0], sm_s[0]};
    float tv = sm_v[0];
    int ti = sm_i[0], tb = sm_b[0];
    for (int k = 1; k < kChunkThreads / kWave; ++k) {
      t = ms_merge(t, MaxSum{sm_m[k], sm_s[k]});
      if (sm_v[k] > tv || (sm_v[k] == tv && sm_i[k] < ti)) { tv = sm_v[k]; ti = sm_i[k]; }
      tb |= sm_b[k];
    }
    out[(size_t)r * NC + c] = StatPart{t.m, t.s, tv, ti, tb, 0, 0, 0};
  }
}

// Merge the chunk statistics of one row across a wave: lane k holds chunk k
// (NC <= 64), xor butterfly (every lane ends with the same, deterministic
// result: each merge is symmetric in its operands).
__device__ StatPart wave_merge_stats(const StatPart* parts, int NC) {
  const int lane = threadIdx.x & 63;
  StatPart p{-INFINITY, 0.f, -INFINITY, 0x7fffffff, 0, 0, 0, 0};
  if (lane < NC) p = parts[lane];
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    const MaxSum t = ms_merge(MaxSum{p.m, p.s}, MaxSum{__shfl_xor(p.m, o, kWave), __shfl_xor(p.s, o, kWave)});
    const float ov = __shfl_xor(p.amax_v, o, kWave);
    const int oi = __shfl_xor(p.amax_i, o, kWave);
    if (ov > p.amax_v || (ov == p.amax_v && oi < p.amax_i)) {
      p.amax_v = ov;
      p.amax_i = oi;
    }
    p.bad |= __shfl_xor(p.bad, o, kWave);
    p.m = t.m;
    p.s = t.s;
  }
  return p;
}

// Weight sources of a draw.
enum { W_ACCEPT = 0, W_DRAFT = 1 };

struct DrawArgs {
  int mode, B, V, gamma;
  float T;
  // accept: p rows [B, gamma+1, V] (probabilities or logits), q rows [B, gamma, V], drafts
  const float* p;
  const float* q;
  int logits;
  const int32_t* d;
  int ld_d;
  // draft: logits of the proposing rows (the last of rps per sequence), q output
  const float* lg;
  int rps, slot;
  float* q_out;
  void* scratch;
  int rows;  // rows per sequence in the scratch statistics
  // the words of the draws, the outputs
  const uint32_t* rand;   // accept: [B, gamma+1] (accept words, then the resample word); draft: [B]
  uint64_t seed, step;
  const uint64_t* step_dev;  // or null: read in place of step
  int32_t* n_accepted;    // accept only
  int32_t* out;           // accept: next_token[B]; draft: d_out + slot (stride ld_out)
  int ld_out;
  int32_t* status;
};

// R_j weights of sequence b at column j, for the residual (res) and the plain row (prob).
__device__ __forceinline__ void weights_at(const DrawArgs& a, const SeqState& st, int b, int j, float& res, float& prob) {
  if (a.mode == W_ACCEPT) {
    const int A = st.A, g = a.gamma;
    const float* P = a.p + ((size_t)b * (g + 1) + A) * a.V;
    const float pj = prob_of(P, j, a.logits, a.T, st.ms[A]);
    prob = pj;
    res = A < g ? fmaxf(0.f, __fsub_rn(pj, a.q[((size_t)b * g + A) * a.V + j])) : 0.f;
  } else {
    const float* lg = a.lg + ((size_t)b * a.rps + a.rps - 1) * a.V;
    prob = expf(lg[j] / a.T - st.ms[0].x) / st.ms[0].y;
    res = 0.f;
  }
}

// decide-and-draw: grid (NC, B), block 256.  Every block of sequence b first
// takes the sequence's decision itself, from the chunk statistics of the stats
// launch (merged in a fixed order: every block reaches the same result):
//   accept: the row statistics, then the gamma accept tests in parallel lanes,
//           the first event (rejection or error) in draft order wins;
//   draft:  the proposing row's statistics.
// Greedy decisions and errors are written by block 0 and end there.  Otherwise
// block c sums the integer weights of its chunk of the row to draw from (the
// residual and the plain row; the draft's q chunk is written here), publishes
// them with agent-scope stores and counts itself; the last block of the
// sequence finds the chunk holding t (a wave prefix sum over the chunk sums)
// and scans that chunk for the token.  Integer sums: exact in any order.
__global__ __launch_bounds__(kChunkThreads) void decide_draw_kernel(DrawArgs a) {
  __shared__ SeqState st;
  __shared__ int amax[kMaxGamma + 1];
  __shared__ int bad_rows;
  __shared__ unsigned long long sr[4], sp[4], wtot[4];
  __shared__ int last, chunk_sel, use_res, done;
  __shared__ unsigned long long t_in_chunk;
  const int c = blockIdx.x, b = blockIdx.y, V = a.V, NC = gridDim.x, cs = chunk_size(V);
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  Scratch sc = carve(a.scratch, a.B, a.rows, V);
  const bool accept = a.mode == W_ACCEPT;
  const int g = accept ? a.gamma : 0;
  const float T = a.T;
  const uint64_t step = a.step_dev ? *a.step_dev : a.step;
  if (threadIdx.x == 0) bad_rows = 0;
  __syncthreads();
  // row statistics (wave w: rows w, w + 4, ...)
  for (int r = w; r <= g; r += kChunkThreads / kWave) {
    const StatPart p = wave_merge_stats(sc.stats + ((size_t)b * a.rows + r) * NC, NC);
    if (lane == 0) {
      amax[r] = p.amax_i;
      st.ms[r] = make_float2(p.m, p.s);
      const bool softmax = accept ? (a.logits && T > 0.f) : T > 0.f;
      if (p.bad || (softmax && (!isfinite(p.m) || !isfinite(p.s)))) atomicOr(&bad_rows, 1);
    }
  }
  __syncthreads();
  if (w == 0) {
    int bad = bad_rows, A = g;
    if (accept && !bad) {
      // lane i < g: event of draft position i (1 = rejection, 2 = error)
      const int32_t* d = a.d + (size_t)b * a.ld_d;
      int ev = 0;
      if (lane < g) {
        const int di = d[lane];
        if (T == 0.f) {
          ev = amax[lane] != di ? 1 : 0;
        } else if (di < 0 || di >= V) {
          ev = 2;
        } else {
          const float pd = prob_of(a.p + ((size_t)b * (g + 1) + lane) * V, di, a.logits, T, st.ms[lane]);
          const float qd = a.q[((size_t)b * g + lane) * V + di];
          const uint32_t wd = a.rand ? a.rand[(size_t)b * (g + 1) + lane]
                                     : draw_word(a.seed, b, step, SPECDEC_PURPOSE_ACCEPT, lane);
          ev = !isfinite(qd) ? 2 : (!(__fmul_rn(word_to_uniform(wd), qd) < pd) ? 1 : 0);
        }
      }
      const unsigned long long hit = __ballot(ev != 0);
      if (hit) {
        const int first = __ffsll(hit) - 1;
        if (__shfl(ev, first, kWave) == 2) bad = 1;
        else A = first;
      }
    }
    if (lane == 0) {
      const bool greedy = T == 0.f;
      if (c == 0) {  // (one block writes the decision)
        if (bad) set_status(a.status, kStatusNonFinite);
        if (accept) {
          a.n_accepted[b] = bad ? -1 : A;
          if (bad) a.out[b] = -1;
          else if (greedy) a.out[b] = amax[A];
        } else if (bad || greedy) {
          a.out[(size_t)b * a.ld_out] = bad ? 0 : amax[0];
        }
      }
      st.A = bad ? -1 : (greedy ? -2 : (accept ? A : 0));
    }
  }
  __syncthreads();
  if (st.A < 0) return;  // (block-uniform: an error, or a greedy decision already written)

  // this chunk's integer weight sums
  {
    const int j0 = c * cs, j1 = min(V, j0 + cs);
    unsigned long long r_sum = 0, p_sum = 0;
    float* qo = !accept && a.q_out ? a.q_out + ((size_t)b * a.gamma + a.slot) * V : nullptr;
    for (int j = j0 + threadIdx.x; j < j1; j += kChunkThreads) {
      float res, prob;
      weights_at(a, st, b, j, res, prob);
      if (qo) qo[j] = prob;
      r_sum += fp_weight(res);
      p_sum += fp_weight(prob);
    }
    r_sum = wave_sum_u64(r_sum);
    p_sum = wave_sum_u64(p_sum);
    if (lane == 0) { sr[w] = r_sum; sp[w] = p_sum; }
    __syncthreads();
    if (threadIdx.x == 0) {
      unsigned long long dr = 0ull, dp = 0ull;
      for (int k = 0; k < kChunkThreads / kWave; ++k) { dr += sr[k]; dp += sp[k]; }
      DrawPart* dst = sc.draw + (size_t)b * NC + c;
      __hip_atomic_store(&dst->res, dr, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(&dst->prob, dp, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      // (the stores have completed before the count: the last block reads them with agent-scope loads)
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      const uint32_t old = __hip_atomic_fetch_add(sc.count + b, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      last = old == (uint32_t)(NC - 1);
      if (last) __hip_atomic_store(sc.count + b, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    __syncthreads();
    if (!last) return;
  }

  // the last block: the chunk holding t, then the token inside it
  if (w == 0) {  // lane k holds chunk k
    DrawPart pk{0ull, 0ull};
    if (lane < NC) {
      const DrawPart* src = sc.draw + (size_t)b * NC + lane;
      pk.res = __hip_atomic_load(&src->res, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      pk.prob = __hip_atomic_load(&src->prob, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    const unsigned long long tr = wave_sum_u64(pk.res), tp = wave_sum_u64(pk.prob);
    const bool res = accept && st.A < g && tr != 0;
    const unsigned long long S = res ? tr : tp;
    uint32_t x;
    if (accept)
      x = a.rand ? a.rand[(size_t)b * (g + 1) + g] : draw_word(a.seed, b, step, SPECDEC_PURPOSE_RESAMPLE, 0);
    else
      x = a.rand ? a.rand[b] : draw_word(a.seed, b, step, SPECDEC_PURPOSE_DRAFT, a.slot);
    if (S == 0) {
      if (lane == 0) {
        a.out[(size_t)b * a.ld_out] = -1;
        done = 1;
      }
    } else {
      const unsigned long long t = scale_word(x, S);
      const unsigned long long wk = res ? pk.res : pk.prob;
      unsigned long long incl = wk;
#pragma unroll
      for (int o = 1; o < kWave; o <<= 1) {
        const unsigned long long n = shfl_up_u64(incl, o);
        if (lane >= o) incl += n;
      }
      // the chunk whose share [incl - wk, incl) of the running sum holds t
      const unsigned long long hit = __ballot(t < incl && t >= incl - wk);
      const int csel = __ffsll(hit) - 1;
      if (lane == csel) {
        chunk_sel = csel;
        use_res = res;
        t_in_chunk = t - (incl - wk);
        done = 0;
      }
      if (hit == 0 && lane == 0) {  // (t < S: unreachable)
        a.out[(size_t)b * a.ld_out] = -1;
        done = 1;
      }
    }
  }
  __syncthreads();
  if (done) return;
  // scan the selected chunk: thread k owns 4 consecutive columns
  const int j0 = chunk_sel * cs, j1 = min(V, j0 + cs);
  unsigned long long mine[4], tot = 0;
  for (int base = j0; base < j1; base += 4 * kChunkThreads) {
    const int jj = base + 4 * threadIdx.x;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      float res = 0.f, prob = 0.f;
      if (jj + e < j1) weights_at(a, st, b, jj + e, res, prob);
      mine[e] = jj + e < j1 ? fp_weight(use_res ? res : prob) : 0ull;
    }
    const unsigned long long sum4 = mine[0] + mine[1] + mine[2] + mine[3];
    unsigned long long incl = sum4;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
      const unsigned long long n = shfl_up_u64(incl, o);
      if (lane >= o) incl += n;
    }
    __syncthreads();
    if (lane == kWave - 1) wtot[w] = incl;
    __syncthreads();
    unsigned long long wbefore = 0, round_tot = 0;
    for (int k = 0; k < kChunkThreads / kWave; ++k) {
      if (k < w) wbefore += wtot[k];
      round_tot += wtot[k];
    }
    const unsigned long long t = t_in_chunk - tot;  // position inside this round
    unsigned long long cum = wbefore + incl - sum4;
    if (t < round_tot && cum <= t && t < cum + sum4) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        cum += mine[e];
        if (cum > t) { a.out[(size_t)b * a.ld_out] = jj + e; break; }
      }
    }
    if (t < round_tot) break;  // uniform: every thread sees the same totals
    tot += round_tot;
  }
}

__global__ void copy_logits_kernel(const float* lg, int rps, int V, float* out) {
  const int b = blockIdx.y;
  const float* src = lg + ((size_t)b * rps + rps - 1) * V;
  for (int j = blockIdx.x * blockDim.x + threadIdx.x; j < V; j += gridDim.x * blockDim.x) out[(size_t)b * V + j] = src[j];
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
  if (threadIdx.x == 0) *a.counter += 1;
}

}  // namespace

hipError_t launch_rows_embed(int dtype, const RowsArgs& a, hipStream_t s) {
  if (dtype == SPECDEC_BF16)
    hipLaunchKernelGGL((rows_embed_kernel<uint16_t>), dim3(a.M), dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL((rows_embed_kernel<float>), dim3(a.M), dim3(256), 0, s, a);
  return hipGetLastError();
}

size_t sampling_scratch_bytes(int B, int rows, int V) {
  const int NC = n_chunks(V);
  return align256(sizeof(StatPart) * (size_t)B * rows * NC) + align256(sizeof(DrawPart) * (size_t)B * NC) +
         align256(sizeof(uint32_t) * (size_t)B);
}

// Two launches: the chunk statistics, then decide-and-draw.
hipError_t launch_draft_finish(const DraftFinishArgs& a, hipStream_t s) {
  const int NC = n_chunks(a.V);
  if (a.logits_out) {
    hipLaunchKernelGGL(copy_logits_kernel, dim3((a.V + 255) / 256, a.B), dim3(256), 0, s, a.logits, a.rps, a.V,
                       a.logits_out);
  }
  Scratch sc = carve(a.scratch, a.B, 1, a.V);
  hipLaunchKernelGGL(stats_kernel, dim3(NC, a.B), dim3(kChunkThreads), 0, s, a.logits, a.V, 1, a.rps, a.rps - 1,
                     a.temperature, nullptr, 0, sc.stats, sc.count);
  DrawArgs d{};
  d.mode = W_DRAFT;
  d.B = a.B;
  d.V = a.V;
  d.gamma = a.gamma;
  d.T = a.temperature;
  d.lg = a.logits;
  d.rps = a.rps;
  d.slot = a.slot;
  d.q_out = a.q_out;
  d.scratch = a.scratch;
  d.rows = 1;
  d.rand = a.rand;
  d.seed = a.seed;
  d.step = a.step;
  d.step_dev = a.step_dev;
  d.out = a.d_out + a.slot;
  d.ld_out = a.ld_d;
  d.status = a.status;
  hipLaunchKernelGGL(decide_draw_kernel, dim3(NC, a.B), dim3(kChunkThreads), 0, s, d);
  return hipGetLastError();
}

// ---------------------------------------------------------------- static scratch of the no-allocation accept
// Device scratch of specdec_accept_noalloc: a file-scope array each GPU the
// library runs on holds until the process ends.  In host code the array's name
// is not a device address; its address on the current device comes from
// hipGetSymbolAddress, looked up once per device (on that device's first call)
// and kept.  Every call on a GPU shares the array.
static __device__ __align__(256) unsigned char scratch[kStaticAcceptScratchBytes];

hipError_t static_accept_scratch(void** out) {
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static void* ptr[kMaxDevices] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (!ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    ptr[dev] = p;
  }
  *out = ptr[dev];
  return hipSuccess;
}

// Two launches: the chunk statistics of every row, then decide-and-draw.
hipError_t launch_accept(const AcceptArgs& a, hipStream_t s) {
  if (a.gamma > kMaxGamma) return hipErrorInvalidValue;
  const int NC = n_chunks(a.V);
  Scratch sc = carve(a.scratch, a.B, a.gamma + 1, a.V);
  const bool logits = a.input_kind == SPECDEC_INPUT_LOGITS;
  hipLaunchKernelGGL(stats_kernel, dim3(NC, a.B * (a.gamma + 1)), dim3(kChunkThreads), 0, s, a.p, a.V, a.gamma + 1,
                     a.gamma + 1, 0, logits ? a.temperature : 0.f, a.temperature > 0.f ? a.q : nullptr, a.gamma,
                     sc.stats, sc.count);
  DrawArgs d{};
  d.mode = W_ACCEPT;
  d.B = a.B;
  d.V = a.V;
  d.gamma = a.gamma;
  d.T = a.temperature;
  d.p = a.p;
  d.q = a.q;
  d.logits = logits;
  d.d = a.d;
  d.ld_d = a.ld_d;
  d.scratch = a.scratch;
  d.rows = a.gamma + 1;
  d.rand = a.rand;
  d.seed = a.seed;
  d.step = a.step;
  d.step_dev = a.step_dev;
  d.n_accepted = a.n_accepted;
  d.out = a.next_token;
  d.ld_out = 1;
  d.status = a.status;
  hipLaunchKernelGGL(decide_draw_kernel, dim3(NC, a.B), dim3(kChunkThreads), 0, s, d);
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
