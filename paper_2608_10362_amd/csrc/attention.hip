// RoPE + KV append and GQA attention of the verify / draft passes against the
// resident KV cache.
//
// The KV layout (internal.h) stores bf16 caches in MFMA operand order, so
// that every wavefront load of the attention kernel reads 1 KB contiguously.
//
// Attention is split over key chunks (flash-decoding style): one wave per
// (16-query tile, 64-key split, kv head, sequence) computes, for every query
// row of the sequence and every query head of the kv group, the chunk's max,
// exp-sum and unnormalised P V; a combine kernel merges the chunks per (row,
// head).  Query i of a sequence at position pos_i sees keys 0..pos_i (causal
// inside the verify block).
#include <algorithm>

#include "device_common.h"
#include "internal.h"

namespace specdec {

namespace {

// ---------------------------------------------------------------- RoPE + append
// Block (head slot, row): slots [0, H) rotate a query head into qr, [H, H+G)
// rotate a key head and store it at the row's position, [H+G, H+2G) store a
// value head (transposed).  Thread j handles the pair (j, j + hd/2).
template <typename KT>
__global__ __launch_bounds__(64) void rope_append_kernel(AttnArgs a) {
  const int hs = blockIdx.x, r = blockIdx.y, j = threadIdx.x;
  const int hd = a.head_dim, half = hd / 2, H = a.n_heads, G = a.n_kv_heads;
  if (j >= half) return;
  const RowDesc rd = a.rows[r];
  const float* src = a.qkv + (size_t)r * (H + 2 * G) * hd + (size_t)hs * hd;
  const float x1 = src[j], x2 = src[j + half];
  const int cap = a.kv.capacity;
  if (hs >= H + G) {  // value head
    if (!rd.valid) return;
    KT* blk = k_block<KT>(a.kv, a.layer, rd.b, hs - H - G);
    Storage<KT>::store(blk + KvIndex<KT>::v(rd.pos, j, hd, cap), x1);
    Storage<KT>::store(blk + KvIndex<KT>::v(rd.pos, j + half, hd, cap), x2);
    return;
  }
  const float* cs = a.rope_cs + (size_t)r * hd;
  const float c = cs[j], s = cs[half + j];
  const float y1 = x1 * c - x2 * s, y2 = x2 * c + x1 * s;
  if (hs < H) {
    float* q = a.qr + ((size_t)r * H + hs) * hd;
    q[j] = y1;
    q[j + half] = y2;
  } else if (rd.valid) {
    KT* blk = k_block<KT>(a.kv, a.layer, rd.b, hs - H);
    Storage<KT>::store(blk + KvIndex<KT>::k(rd.pos, j, hd, cap), y1);
    Storage<KT>::store(blk + KvIndex<KT>::k(rd.pos, j + half, hd, cap), y2);
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

// ---------------------------------------------------------------- MFMA attention partials (bf16 cache)
// The keys [0, 32 n_sub) of each (kv head, sequence) are cut into n_part parts
// of S sub-chunks of 32 keys; the last part also takes the remainder (fewer
// than 2S sub-chunks).  One block per (part, 16-query tile, kv head,
// sequence) and one wave per sub-chunk.  S is chosen on the host so that the
// blocks about fill the CUs once: every CU then streams about the same number
// of K/V bytes.  Per wave, S = Q K^T and O = P V run on
// v_mfma_f32_16x16x32_bf16 with the float32 operands (Q, P) split into hi + lo
// bf16 parts; lane l holds rows 4(l/16)+r of S and O, so the per-row max and
// sum live in the same lanes.  The block merges its waves' (max, sum, O) in
// LDS (fixed wave order) and writes one partial per part.
constexpr int kSubKeys = 32;

__device__ __forceinline__ void split_hilo(const float* v, bf16x8& hi, bf16x8& lo) {
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const __bf16 h = (__bf16)v[j];
    hi[j] = h;
    lo[j] = (__bf16)(v[j] - (float)h);
  }
}

// One element of the attention output o[row][head * hd + d], also into the
// stacked operand of the O projection when the pass hands x over stacked.
__device__ __forceinline__ void put_o(const AttnArgs& a, float* o, int row, int head, int d, float v) {
  o[d] = v;
  if (a.xs) put_stacked(a.xs, a.stt, row, head * a.head_dim + d, v);
}

// Reductions over the 16 lanes of a row of the wave (lanes 16k .. 16k+15)
// with DPP moves: swaps within quads, then the half-row and row mirrors.
// Every lane ends with the same value (each step combines two equal-order
// partial results, and both operations commute).
template <int CTRL>
__device__ __forceinline__ float dpp_mov(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, 0xF, 0xF, false));
}
__device__ __forceinline__ float group16_max(float v) {
  v = fmaxf(v, dpp_mov<0xB1>(v));   // quad_perm [1,0,3,2]
  v = fmaxf(v, dpp_mov<0x4E>(v));   // quad_perm [2,3,0,1]
  v = fmaxf(v, dpp_mov<0x141>(v));  // row_half_mirror
  return fmaxf(v, dpp_mov<0x140>(v));  // row_mirror
}
__device__ __forceinline__ float group16_sum(float v) {
  v += dpp_mov<0xB1>(v);
  v += dpp_mov<0x4E>(v);
  v += dpp_mov<0x141>(v);
  return v + dpp_mov<0x140>(v);
}

// Dynamic LDS: per wave a P tile [16][36] (the transposed read of P V), then,
// reused once every wave is past P V, the merge buffers [NW][RS][HD + 4] of
// O (rows padded against bank conflicts) and [NW][RS][2] of (max, sum), RS =
// query rows of the tile.  With the in-kernel combine (own), the combining
// block's own part [RS][HD + 2] (O, max, sum) follows them.
__host__ __device__ inline size_t attn_block_shared(int NW, int RS, int HD) {
  const size_t p = (size_t)NW * 16 * (kSubKeys + 4);
  const size_t m = (size_t)NW * RS * (HD + 6);
  return p > m ? p : m;
}
__host__ __device__ inline size_t attn_block_lds(int NW, int RS, int HD, bool own = false) {
  return (attn_block_shared(NW, RS, HD) + (own ? (size_t)RS * (HD + 2) : 0)) * sizeof(float);
}

// Flagged partial words of the in-kernel combine: the float in the low half,
// the launch's tag in the high half, written and read as single 64-bit
// agent-scope accesses (a reader sees a whole word, old or new).
__device__ __forceinline__ void ll_put(uint64_t* p, float v, uint32_t tag) {
  __hip_atomic_store(p, ((uint64_t)tag << 32) | (uint64_t)__float_as_uint(v), __ATOMIC_RELAXED,
                     __HIP_MEMORY_SCOPE_AGENT);
}
// Cache-policy bits of a load served by the coherent level (sc1), not by a
// possibly stale line of this XCD's L2.
constexpr int kCoherentLoad = 16;
// Polls of the combining block before it gives up (each takes a memory round
// trip, about a microsecond: a quarter of a second or so in all).
constexpr int kLlMaxPolls = 1 << 18;

constexpr int kMaxPartWaves = 12;  // 3 waves per SIMD: up to 170 VGPRs per lane
constexpr int kLoopWaves = 4;      // waves per block when waves loop over several sub-chunks

// LOOP: wave w takes sub-chunks w, w + NW, ... of its part (online softmax
// across them), so long contexts keep every wave streaming K/V instead of
// ending the block after one sub-chunk (4-wave blocks, up to 256 registers);
// otherwise each wave takes one sub-chunk (up to 12-wave blocks).
template <int HD, bool LOOP>
__global__ __launch_bounds__(LOOP ? 64 * kLoopWaves : 64 * kMaxPartWaves, LOOP ? 2 : 1) void attn_block_kernel(
    AttnArgs a, int S, int n_sub, int NW) {
  constexpr int KST = HD / 32;  // k-steps of Q K^T
  constexpr int DT = HD / 16;   // 16-wide dimension tiles of P V
  constexpr int NT = kSubKeys / 16;
  extern __shared__ float smem[];
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int g = blockIdx.y, b = blockIdx.z;
  const int H = a.n_heads, G = a.n_kv_heads, group = H / G;
  const int rps = a.rps, r0 = b * rps, nq = rps * group;
  const int n_part = a.n_split;
  const int part = blockIdx.x % n_part, mt = blockIdx.x / n_part;
  const int RS = min(16, nq - mt * 16);  // query rows of this tile (> 0 by the grid)
  const int c16 = lane & 15, grp = lane >> 4;
  int sub_here = part == n_part - 1 ? n_sub - part * S : S;
  if (a.seq_bound) {
    // Keys past this sequence's own context are never loaded: within a sequence
    // positions grow with the row index, so its last row (when valid) bounds
    // them.  (Scalar loads; one wait before the K/V loads are issued.)
    const RowDesc last = a.rows[r0 + rps - 1];
    if (last.valid) {
      const int first = part * S * kSubKeys;
      if (first > last.pos) sub_here = 0;  // (block-uniform) no key of this part is visible
      const int need = (last.pos + 1 - first + kSubKeys - 1) / kSubKeys;
      sub_here = need < 0 ? 0 : (need < sub_here ? need : sub_here);
    }
  }
  const uint16_t* kb = k_block<uint16_t>(a.kv, a.layer, b, g);
  const uint16_t* vb = kb + (size_t)a.kv.capacity * HD;

  floatx4 of[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) of[dt] = floatx4{0.f, 0.f, 0.f, 0.f};
  float mx[4] = {-INFINITY, -INFINITY, -INFINITY, -INFINITY}, sm[4] = {0.f, 0.f, 0.f, 0.f};
  int qpos[4] = {-1, -1, -1, -1};
  float* pbuf = smem + (size_t)wave * 16 * (kSubKeys + 4);

  // Every load of the first sub-chunk is issued before anything waits,
  // smallest first (loads complete in order, so waiting for an early one never
  // waits for a later one): the row descriptors (every wave: the combining
  // block reads them from its lanes too), the K fragments, Q, then the V
  // fragments.  Row descriptors and Q go through range-checked buffer loads.
  // Lane l < 16 holds the descriptor of the row of query l of the tile
  // (queries qa = mt*16 + l; rows r0 + qa / group).  (Only the two fields
  // used: a wider load leaves dead destination registers the allocator
  // reuses, which forces a wait for the load.)
  const int ql = mt * 16 + lane;
  int rd_pos, rd_valid;
  {
    const __amdgpu_buffer_rsrc_t rr = __builtin_amdgcn_make_buffer_rsrc(const_cast<RowDesc*>(a.rows), (short)0,
                                                                         a.M * (int)sizeof(RowDesc), 0x00020000);
    const uint32_t roff = ((uint32_t)(r0 + min(ql, nq - 1) / group) * (uint32_t)sizeof(RowDesc)) |
                          ((uint32_t)(lane >= 16 || ql >= nq) << 31);
    rd_pos = (int)__builtin_amdgcn_raw_buffer_load_b32(rr, roff + offsetof(RowDesc, pos), 0, 0);
    rd_valid = (int)__builtin_amdgcn_raw_buffer_load_b32(rr, roff + offsetof(RowDesc, valid), 0, 0);
  }
  // In-kernel combine of looping launches: the epoch of the sequence, tile
  // and kv head (this launch tags its words with epoch + 1), read through the
  // coherent level (sc1) and used only once the partials are out.
  const bool ll_mode = LOOP && a.ll != nullptr;
  const uint32_t ep_idx = (uint32_t)(((size_t)b * (gridDim.x / n_part) + mt) * G + g);
  uint32_t ep_raw = 0;
  if constexpr (LOOP)  // (unconditional load, range 0 without the combine: a branch here made the key loads wait for it)
    ep_raw = __builtin_amdgcn_raw_buffer_load_b32(
        __builtin_amdgcn_make_buffer_rsrc(a.epochs, (short)0, ll_mode ? (ep_idx + 1u) * 4u : 0u, 0x00020000),
        ep_idx * 4u, 0, kCoherentLoad);
  float* const sown = smem + attn_block_shared(NW, RS, HD);  // (combiner: its own part per row)
  if (wave < sub_here) {  // (wave-uniform) a wave past the part's sub-chunks only joins the merge
    // K fragments of a sub-chunk: 2 x KST contiguous 1 KB fragments (k0 + 32 <= capacity);
    // V fragments: DT contiguous 1 KB fragments (32 positions x 16 dims each).
    u32x4 kf[NT][KST], vf[DT];
    auto load_k = [&](int k0) {
      const uint16_t* kfrag = kb + (size_t)(k0 / 16) * KST * 512 + lane * 8;
#pragma unroll
      for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int c = 0; c < KST; ++c) kf[t][c] = *(const u32x4*)(kfrag + (size_t)(t * KST + c) * 512);
    };
    auto load_v = [&](int k0) {
      const uint16_t* vfrag = vb + (size_t)(k0 / 32) * DT * 512 + lane * 8;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) vf[dt] = *(const u32x4*)(vfrag + (size_t)dt * 512);
    };
    int k0 = (part * S + wave) * kSubKeys;
    load_k(k0);
    // Q fragments (A operand): query qa = mt*16 + l%16 (zeros past nq).
    f32x4 qv4[KST][2];
    {
      const int qa = mt * 16 + c16;
      const int row = r0 + qa / group, head = g * group + qa % group;
      const __amdgpu_buffer_rsrc_t qrs =
          __builtin_amdgcn_make_buffer_rsrc(a.qr, (short)0, a.M * H * HD * 4, 0x00020000);
      const uint32_t qoff = ((((uint32_t)row * H + head) * HD + 8 * grp) * 4u) | ((uint32_t)(qa >= nq) << 31);
#pragma unroll
      for (int c = 0; c < KST; ++c) {
        qv4[c][0] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(qrs, qoff + 128u * c, 0, 0));
        qv4[c][1] =
            __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(qrs, qoff + 128u * c + 16u, 0, 0));
      }
    }
    load_v(k0);
    // (compiler barrier: keeps what follows from being hoisted above the loads)
    asm volatile("" ::: "memory");

    // nk = max(pos) + 1 over the tile's valid query rows: no key past it is read.
    // (Lane reads rather than shuffles: the compiler then waits for the row
    // descriptors alone, with the K, Q and V loads above still in flight; with
    // shuffles it held the Q and V loads back until the descriptors arrived.)
    const int mypos = (lane < 16 && ql < nq && rd_valid) ? rd_pos : -1;
    int lp[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) lp[i] = __builtin_amdgcn_readlane(mypos, i);
    int nk = lp[0] + 1;
#pragma unroll
    for (int i = 1; i < 16; ++i) nk = max(nk, lp[i] + 1);
    // positions of the 4 query rows this lane holds in the C layout (-1: none)
#pragma unroll
    for (int r = 0; r < 4; ++r)
      qpos[r] = grp == 0 ? lp[r] : (grp == 1 ? lp[4 + r] : (grp == 2 ? lp[8 + r] : lp[12 + r]));
    const float scale = 1.0f / sqrtf((float)HD);
    bf16x8 qhi[KST], qlo[KST];
#pragma unroll
    for (int c = 0; c < KST; ++c) {
      float v[8];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        v[j] = qv4[c][0][j] * scale;
        v[4 + j] = qv4[c][1][j] * scale;
      }
      split_hilo(v, qhi[c], qlo[c]);
    }

    for (int j = wave; j < sub_here && k0 < nk; j += NW) {  // (wave-uniform)
      if (j != wave) {  // the first sub-chunk's fragments were loaded above
        load_k(k0);
        load_v(k0);
      }
      // keys past the context: zero their V entries (never multiply stale memory)
      const int nvalid = nk - (k0 + 8 * grp);
      if (nvalid < 8) {
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            if (2 * q >= nvalid) vf[dt][q] = 0u;
            else if (2 * q + 1 >= nvalid) vf[dt][q] &= 0xffffu;
          }
      }
      floatx4 sf[NT];
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        floatx4 acc = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int c = 0; c < KST; ++c) {
          const bf16x8 kk = __builtin_bit_cast(bf16x8, kf[t][c]);
          acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qhi[c], kk, acc, 0, 0, 0);
          acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qlo[c], kk, acc, 0, 0, 0);
        }
        const int key = k0 + 16 * t + c16;
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (key > qpos[r]) acc[r] = -INFINITY;
        sf[t] = acc;
      }
      // Online softmax: the running (max, sum, O) of each row is rescaled by
      // exp(old max - new max) when this sub-chunk raises the max.
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        float m = -INFINITY;
#pragma unroll
        for (int t = 0; t < NT; ++t) m = fmaxf(m, sf[t][r]);
        const float mnew = fmaxf(mx[r], group16_max(m));
        const float alpha = mx[r] == -INFINITY ? 0.f : expf(mx[r] - mnew);
        float sum = 0.f;
#pragma unroll
        for (int t = 0; t < NT; ++t) {
          const float p = mnew == -INFINITY || sf[t][r] == -INFINITY ? 0.f : expf(sf[t][r] - mnew);
          pbuf[(4 * grp + r) * (kSubKeys + 4) + 16 * t + c16] = p;
          sum += p;
        }
        sm[r] = sm[r] * alpha + group16_sum(sum);
        mx[r] = mnew;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) of[dt][r] *= alpha;
      }
      __builtin_amdgcn_wave_barrier();  // P written by all lanes of the wave before the transposed reads
      float pv[8];
#pragma unroll
      for (int q = 0; q < 8; ++q) pv[q] = pbuf[c16 * (kSubKeys + 4) + 8 * grp + q];
      bf16x8 phi, plo;
      split_hilo(pv, phi, plo);
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        const bf16x8 vv = __builtin_bit_cast(bf16x8, vf[dt]);
        of[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(phi, vv, of[dt], 0, 0, 0);
        of[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(plo, vv, of[dt], 0, 0, 0);
      }
      if constexpr (!LOOP) break;
      __builtin_amdgcn_wave_barrier();  // the transposed reads of P done before the next sub-chunk writes it
      k0 += NW * kSubKeys;
    }
  }

  constexpr int DPL = HD >= 64 ? HD / 64 : 1;
  // The combining block.  Looping launches (several rounds of blocks per
  // CU): the block of the last part holding a key some valid row of the tile
  // sees (the parts after it hold none); every part it waits for has a lower
  // block index, so it was dispatched before it, and no other block waits for
  // anything; its own part stays in LDS.  The other blocks end without
  // waiting for their stores, which frees their CU for the next round sooner.
  // One-round launches: the last block to count itself, after its partial
  // stores are acknowledged (faster there than a fixed combining block that
  // polls: all blocks run at once, and polling started before the other
  // parts' words had landed).  (Lane reads of the descriptors, long arrived.)
  // (The descriptor values pass through an empty asm here so that the
  // compiler does not share this test with the one before the key loads and
  // wait for the descriptors before issuing them.)
  int last_part = n_part - 1;
  uint32_t tag = 0;
  if (ll_mode) {
    int rp = rd_pos, rv = rd_valid;
    asm volatile("" : "+v"(rp), "+v"(rv));
    const int vpos = (lane < 16 && ql < nq && rv) ? rp : -1;
    int mpos = -1;
#pragma unroll
    for (int i = 0; i < 16; ++i) mpos = max(mpos, __builtin_amdgcn_readlane(vpos, i));
    if (mpos >= 0) last_part = min(mpos / a.chunk, n_part - 1);
    tag = ep_raw + 1u == 0u ? 1u : ep_raw + 1u;
  }
  const bool combiner = LOOP && ll_mode && part == last_part;
  uint32_t* const epoch = a.epochs + ep_idx;  // (combiner: the next launch's epoch goes here)
  if (NW == 1) {  // (block-uniform) the wave's own (max, sum, O) rows are the part's partials
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int row = 4 * grp + r;
      if (row >= RS || qpos[r] < 0 || mx[r] == -INFINITY) continue;
      const int qc = mt * 16 + row;
      const size_t slot = ((size_t)(r0 + qc / group) * H + g * group + qc % group) * n_part + part;
      if (combiner) {
        float* own = sown + (size_t)row * (HD + 2);
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) own[dt * 16 + c16] = of[dt][r];
        if (c16 == 0) {
          own[HD] = mx[r];
          own[HD + 1] = sm[r];
        }
      } else if (ll_mode) {
        uint64_t* w = a.ll + slot * (HD + 2);
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) ll_put(w + dt * 16 + c16, of[dt][r], tag);
        if (c16 == 0) {
          ll_put(w + HD, mx[r], tag);
          ll_put(w + HD + 1, sm[r], tag);
        }
      } else if (a.counters) {
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
          __hip_atomic_store(&a.o_part[slot * HD + dt * 16 + c16], of[dt][r], __ATOMIC_RELAXED,
                             __HIP_MEMORY_SCOPE_AGENT);
        if (c16 == 0) {
          __hip_atomic_store(&a.ml_part[2 * slot], mx[r], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          __hip_atomic_store(&a.ml_part[2 * slot + 1], sm[r], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
      } else {
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) a.o_part[slot * HD + dt * 16 + c16] = of[dt][r];
        if (c16 == 0) {
          a.ml_part[2 * slot] = mx[r];
          a.ml_part[2 * slot + 1] = sm[r];
        }
      }
    }
  } else {
  // Merge the waves' partials of this part (LDS reused: every wave is past P V).
  __syncthreads();
  constexpr int OS = HD + 4;                   // row stride of the O partials
  float* so = smem;                            // [NW][RS][OS]
  float* sml = smem + (size_t)NW * RS * OS;    // [NW][RS][2]
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int row = 4 * grp + r;
    if (row >= RS) continue;
    const bool live = qpos[r] >= 0 && mx[r] != -INFINITY;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) so[((size_t)wave * RS + row) * OS + dt * 16 + c16] = live ? of[dt][r] : 0.f;
    if (c16 == 0) {
      sml[((size_t)wave * RS + row) * 2] = live ? mx[r] : -INFINITY;
      sml[((size_t)wave * RS + row) * 2 + 1] = live ? sm[r] : 0.f;
    }
  }
  __syncthreads();
  // One wave per row: the waves' weights exp(m_w - M) are uniform across the
  // wave, each lane sums HD / 64 dims over the waves in fixed order.
  constexpr int MAXW = LOOP ? kLoopWaves : kMaxPartWaves;
  for (int row = wave; row < RS; row += NW) {  // (wave-uniform)
    // The waves' partials in groups of 4: every read of a group first, then
    // the arithmetic (a wave past NW or without keys gets weight 0, and adding
    // 0 * a finite partial changes no sum).
    constexpr int WG = 4;
    float M = -INFINITY;
#pragma unroll
    for (int w0 = 0; w0 < MAXW; w0 += WG) {
      if (w0 >= NW) break;
#pragma unroll
      for (int w = w0; w < w0 + WG; ++w)
        if (w < NW) M = fmaxf(M, sml[((size_t)w * RS + row) * 2]);
    }
    if (M == -INFINITY) continue;  // no key of this part is visible to the row
    float L = 0.f, O[DPL];
#pragma unroll
    for (int j = 0; j < DPL; ++j) O[j] = 0.f;
#pragma unroll
    for (int w0 = 0; w0 < MAXW; w0 += WG) {
      if (w0 >= NW) break;
      float mw[WG], lw[WG], ow[WG][DPL];
#pragma unroll
      for (int i = 0; i < WG; ++i) {
        const size_t wr = (size_t)min(w0 + i, NW - 1) * RS + row;
        mw[i] = sml[wr * 2];
        lw[i] = sml[wr * 2 + 1];
#pragma unroll
        for (int j = 0; j < DPL; ++j) ow[i][j] = lane + 64 * j < HD ? so[wr * OS + lane + 64 * j] : 0.f;
      }
#pragma unroll
      for (int i = 0; i < WG; ++i) {
        const float e = w0 + i < NW && mw[i] != -INFINITY ? expf(mw[i] - M) : 0.f;
        L += e * lw[i];
#pragma unroll
        for (int j = 0; j < DPL; ++j) O[j] += e * ow[i][j];
      }
    }
    const int qc = mt * 16 + row;
    const int qrow = r0 + qc / group, head = g * group + qc % group;
    const size_t slot = ((size_t)qrow * H + head) * n_part + part;
    if (combiner) {  // (kept in LDS for its own combine)
      float* own = sown + (size_t)row * (HD + 2);
#pragma unroll
      for (int j = 0; j < DPL; ++j)
        if (lane + 64 * j < HD) own[lane + 64 * j] = O[j];
      if (lane == 0) {
        own[HD] = M;
        own[HD + 1] = L;
      }
    } else if (ll_mode) {  // (tagged words: the combining block polls them)
      uint64_t* w = a.ll + slot * (HD + 2);
#pragma unroll
      for (int j = 0; j < DPL; ++j)
        if (lane + 64 * j < HD) ll_put(w + lane + 64 * j, O[j], tag);
      if (lane == 0) {
        ll_put(w + HD, M, tag);
        ll_put(w + HD + 1, L, tag);
      }
    } else if (a.counters) {  // (agent-scope stores: visible to the combining block on any XCD once completed)
#pragma unroll
      for (int j = 0; j < DPL; ++j)
        if (lane + 64 * j < HD)
          __hip_atomic_store(&a.o_part[slot * HD + lane + 64 * j], O[j], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      if (lane == 0) {
        __hip_atomic_store(&a.ml_part[2 * slot], M, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(&a.ml_part[2 * slot + 1], L, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
    } else {  // (read by the combine kernel after this launch)
#pragma unroll
      for (int j = 0; j < DPL; ++j)
        if (lane + 64 * j < HD) a.o_part[slot * HD + lane + 64 * j] = O[j];
      if (lane == 0) {
        a.ml_part[2 * slot] = M;
        a.ml_part[2 * slot + 1] = L;
      }
    }
  }
  }
  // The memory system is idle while the combining blocks finish: blocks that
  // do not combine read their share of the next launch's weights into the
  // last-level cache before they end.
  auto read_ahead = [&]() {
    // (Block i of n: the first kNextWeightsPerBlock bytes of slice i of n.)
    // The loaded words are only kept live to the end (no store), so the loads
    // are issued and waited for and nothing else.
    if (a.next_w) {
      const uint32_t nblk = gridDim.x * gridDim.y * gridDim.z;
      const uint32_t lb = blockIdx.x + gridDim.x * (blockIdx.y + gridDim.y * blockIdx.z);
      const uint32_t slice = (a.next_w_bytes / nblk + 1023u) & ~1023u;
      const __amdgpu_buffer_rsrc_t nr = __builtin_amdgcn_make_buffer_rsrc(const_cast<unsigned char*>(a.next_w),
                                                                          (short)0, a.next_w_bytes, 0x00020000);
      // Wave w reads KB-chunks w, w + NW, ... (at most kNextLoads of them), all
      // issued before the one wait; a dword per lane at a 16-byte stride touches
      // every line of the chunk.  (Offsets past the share or next_w_bytes read
      // nothing: the out-of-range bit and the descriptor's range.)
      constexpr int kNextLoads = 6;
      const uint32_t lim = min(kNextWeightsPerBlock, slice);
      uint32_t v[kNextLoads];
#pragma unroll
      for (int i = 0; i < kNextLoads; ++i) {
        const uint32_t c = ((uint32_t)wave + (uint32_t)i * NW) * 1024u;
        v[i] = __builtin_amdgcn_raw_buffer_load_b32(nr, (lb * slice + c + lane * 16u) | ((uint32_t)(c >= lim) << 31),
                                                    0, 0);
      }
      uint32_t keep = 0;
#pragma unroll
      for (int i = 0; i < kNextLoads; ++i) keep ^= v[i];
      asm volatile("" ::"v"(keep));
    }
  };
  if constexpr (LOOP) {
    if (!ll_mode) return;
    if (!combiner) {
      read_ahead();
      return;
    }
    // The combining block: one wave per query row of the tile.  Its own part
    // comes from LDS; the other parts' words are polled until every one read
    // carries this launch's tag (each write and read is a whole 64-bit word),
    // in batches of PB parts; the parts are added in part order.
    __syncthreads();  // (the block's own part in LDS)
    for (int row = wave; row < RS; row += NW) {  // (wave-uniform)
      const int qc = mt * 16 + row;
      const int qrow = r0 + qc / group, head = g * group + qc % group;
      RowDesc rd;
      rd.pos = __shfl(rd_pos, row, kWave);  // (lane `row` loaded this query's row descriptor)
      rd.valid = __shfl(rd_valid, row, kWave);
      float* o = a.o + ((size_t)qrow * H + head) * HD;
      if (!rd.valid) {
#pragma unroll
        for (int j = 0; j < DPL; ++j)
          if (lane + 64 * j < HD) put_o(a, o, qrow, head, lane + 64 * j, 0.f);
        continue;
      }
      // parts holding keys <= pos (the last part also holds the remainder); the
      // last one, when among them, is this block's own (nch <= last_part + 1)
      const int nch = min(rd.pos / a.chunk + 1, n_part);
      if (rd.pos + 1 > a.max_ctx && lane == 0) set_status(a.status, kStatusKvCapacity);  // the host's bound was wrong
      const bool own_row = nch == last_part + 1;
      const int npoll = own_row ? last_part : nch;  // parts read from memory
      const float* own = sown + (size_t)row * (HD + 2);
      const uint64_t* w = a.ll + ((size_t)qrow * H + head) * n_part * (HD + 2);
      constexpr int PB = 8;
      // lane p < nch: part p's (max, sum)
      float mp = -INFINITY, lp = 0.f;
      if (lane == last_part && own_row) {
        mp = own[HD];
        lp = own[HD + 1];
      }
      float acc[DPL];
#pragma unroll
      for (int j = 0; j < DPL; ++j) acc[j] = 0.f;
      float mx = 0.f, wgt = 0.f;
      bool expired = false;
      const int pl = min(lane, max(npoll - 1, 0));  // (clamped: every load below reads a polled slot)
      for (int p0 = 0; p0 < nch; p0 += PB) {  // (wave-uniform)
        float ov[PB][DPL];
        for (int poll = 0;; ++poll) {  // (wave-uniform)
          // Every load first (branch-free, addresses clamped to polled slots),
          // then the tag tests and the selection of own and absent parts.
          uint64_t wm = 0, wl = 0, wo[PB][DPL];
          if (npoll > 0) {  // (wave-uniform)
            if (p0 == 0) {
              wm = __hip_atomic_load(const_cast<uint64_t*>(w) + (size_t)pl * (HD + 2) + HD, __ATOMIC_RELAXED,
                                     __HIP_MEMORY_SCOPE_AGENT);
              wl = __hip_atomic_load(const_cast<uint64_t*>(w) + (size_t)pl * (HD + 2) + HD + 1, __ATOMIC_RELAXED,
                                     __HIP_MEMORY_SCOPE_AGENT);
            }
#pragma unroll
            for (int pp = 0; pp < PB; ++pp) {
              const int pc = min(p0 + pp, npoll - 1);
#pragma unroll
              for (int j = 0; j < DPL; ++j)
                wo[pp][j] = __hip_atomic_load(const_cast<uint64_t*>(w) + (size_t)pc * (HD + 2) + min(lane + 64 * j, HD - 1),
                                              __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
          }
          bool ok = true;
          if (p0 == 0 && lane < npoll) {
            ok = (uint32_t)(wm >> 32) == tag && (uint32_t)(wl >> 32) == tag;
            mp = __uint_as_float((uint32_t)wm);
            lp = __uint_as_float((uint32_t)wl);
          }
#pragma unroll
          for (int pp = 0; pp < PB; ++pp) {
            const int p = p0 + pp;
#pragma unroll
            for (int j = 0; j < DPL; ++j) {
              const int dd = lane + 64 * j;
              const bool polled = p < npoll && dd < HD;
              ok = ok && (!polled || (uint32_t)(wo[pp][j] >> 32) == tag);
              ov[pp][j] = polled ? __uint_as_float((uint32_t)wo[pp][j])
                                 : (p < nch && dd < HD ? own[min(dd, HD - 1)] : 0.f);
            }
          }
          if (__all(ok)) break;
          if (poll >= kLlMaxPolls) {
            expired = true;
            break;
          }
        }
        if (expired) break;
        if (p0 == 0) {
          mx = wave_max(lane < nch ? mp : -INFINITY);
          wgt = lane < nch ? expf(mp - mx) : 0.f;
        }
#pragma unroll
        for (int pp = 0; pp < PB; ++pp) {
          const float wp = __shfl(wgt, (p0 + pp) & 63, kWave);
          const float wv = p0 + pp < nch ? wp : 0.f;
#pragma unroll
          for (int j = 0; j < DPL; ++j) acc[j] += wv * ov[pp][j];
        }
      }
      if (expired) {  // (a part never arrived: report it, write zeros)
        if (lane == 0) set_status(a.status, kStatusWaitExpired);
#pragma unroll
        for (int j = 0; j < DPL; ++j)
          if (lane + 64 * j < HD) put_o(a, o, qrow, head, lane + 64 * j, 0.f);
        continue;
      }
      const float L = wave_sum(wgt * lp);
      const float inv = 1.0f / L;
#pragma unroll
      for (int j = 0; j < DPL; ++j)
        if (lane + 64 * j < HD) put_o(a, o, qrow, head, lane + 64 * j, acc[j] * inv);
    }
    // Every part of this launch has been read (so every block of it has read
    // the epoch): the next launch's tag.
    __syncthreads();
    if (threadIdx.x == 0) __hip_atomic_store(epoch, tag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  } else {
    if (!a.counters) return;

    // The last block of this (sequence, tile, kv head) to finish combines the
    // parts: every wave's partial stores have completed before the block's
    // single counter increment, and the combining block reads the partials
    // with agent-scope loads.  The counter goes back to zero for the next launch.
    __shared__ int s_last;
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    if (threadIdx.x == 0) {
      uint32_t* ctr = a.counters + ep_idx;
      const uint32_t old = __hip_atomic_fetch_add(ctr, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      const int last = old == (uint32_t)(n_part - 1);
      if (last) __hip_atomic_store(ctr, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      s_last = last;
    }
    __syncthreads();
    if (!s_last) {
      read_ahead();
      return;
    }
    for (int row = wave; row < RS; row += NW) {  // (wave-uniform) one wave per query row of the tile
      const int qc = mt * 16 + row;
      const int qrow = r0 + qc / group, head = g * group + qc % group;
      RowDesc rd;
      rd.pos = __shfl(rd_pos, row, kWave);  // (lane `row` loaded this query's row descriptor)
      rd.valid = __shfl(rd_valid, row, kWave);
      float* o = a.o + ((size_t)qrow * H + head) * HD;
      if (!rd.valid) {
#pragma unroll
        for (int j = 0; j < DPL; ++j)
          if (lane + 64 * j < HD) put_o(a, o, qrow, head, lane + 64 * j, 0.f);
        continue;
      }
      // parts holding keys <= pos (the last part also holds the remainder)
      const int nch = min(rd.pos / a.chunk + 1, n_part);
      if (rd.pos + 1 > a.max_ctx && lane == 0) set_status(a.status, kStatusKvCapacity);  // the host's bound was wrong
      const size_t base = ((size_t)qrow * H + head) * n_part;
      // lane p < nch: part p's (max, sum); the first parts' outputs in the same round trip
      constexpr int PB = 8;
      const int pl = min(lane, nch - 1);
      const float mp = __hip_atomic_load(&a.ml_part[2 * (base + pl)], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      const float lp = __hip_atomic_load(&a.ml_part[2 * (base + pl) + 1], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      float acc[DPL];
#pragma unroll
      for (int j = 0; j < DPL; ++j) acc[j] = 0.f;
      float mx = 0.f, wgt = 0.f;
      for (int p0 = 0; p0 < nch; p0 += PB) {  // (wave-uniform)
        float ov[PB][DPL];
#pragma unroll
        for (int pp = 0; pp < PB; ++pp) {
          const int p = min(p0 + pp, nch - 1);  // (parts past nch get weight 0 below)
#pragma unroll
          for (int j = 0; j < DPL; ++j)
            ov[pp][j] = lane + 64 * j < HD ? __hip_atomic_load(&a.o_part[(base + p) * HD + lane + 64 * j],
                                                               __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)
                                           : 0.f;
        }
        if (p0 == 0) {
          mx = wave_max(lane < nch ? mp : -INFINITY);
          wgt = lane < nch ? expf(mp - mx) : 0.f;
        }
#pragma unroll
        for (int pp = 0; pp < PB; ++pp) {
          const float w = __shfl(wgt, (p0 + pp) & 63, kWave);
          const float wv = p0 + pp < nch ? w : 0.f;
#pragma unroll
          for (int j = 0; j < DPL; ++j) acc[j] += wv * ov[pp][j];
        }
      }
      const float L = wave_sum(wgt * lp);
      const float inv = 1.0f / L;
#pragma unroll
      for (int j = 0; j < DPL; ++j)
        if (lane + 64 * j < HD) put_o(a, o, qrow, head, lane + 64 * j, acc[j] * inv);
    }
  }
}

// ---------------------------------------------------------------- combine
// Block (head, row): weights w_c = exp(m_c - max_c m_c) of the row's chunks
// in LDS (fixed-order reductions), then o = sum_c w_c o_c / sum_c w_c l_c with
// the chunk loop unrolled so the partial loads overlap.
__global__ __launch_bounds__(128) void attn_combine_kernel(AttnArgs a) {
  extern __shared__ float wsh[];  // [n_split]
  __shared__ float red[16];
  const int head = blockIdx.x, r = blockIdx.y;
  const int hd = a.head_dim, H = a.n_heads;
  const RowDesc rd = a.rows[r];
  float* o = a.o + ((size_t)r * H + head) * hd;
  if (!rd.valid) {
    for (int dd = threadIdx.x; dd < hd; dd += blockDim.x) put_o(a, o, r, head, dd, 0.f);
    return;
  }
  // splits holding keys <= pos (with parts, the last one also holds the remainder)
  const int nch = min(rd.pos / a.chunk + 1, a.n_split);
  if (rd.pos + 1 > a.max_ctx && threadIdx.x == 0) set_status(a.status, kStatusKvCapacity);  // the host's bound was wrong
  const size_t base = ((size_t)r * H + head) * a.n_split;
  float mx = -INFINITY;
  for (int c = threadIdx.x; c < nch; c += blockDim.x) mx = fmaxf(mx, a.ml_part[2 * (base + c)]);
  mx = block_max(mx, red);
  float L = 0.f;
  for (int c = threadIdx.x; c < nch; c += blockDim.x) {
    const float w = expf(a.ml_part[2 * (base + c)] - mx);
    wsh[c] = w;
    L += w * a.ml_part[2 * (base + c) + 1];
  }
  L = block_sum(L, red);  // its barrier also publishes wsh
  const float inv = 1.0f / L;
  const float* op = a.o_part + base * hd;
  for (int dd = threadIdx.x; dd < hd; dd += blockDim.x) {
    float acc0 = 0.f, acc1 = 0.f, acc2 = 0.f, acc3 = 0.f;
    int c = 0;
    for (; c + 4 <= nch; c += 4) {
      acc0 += wsh[c] * op[(size_t)c * hd + dd];
      acc1 += wsh[c + 1] * op[(size_t)(c + 1) * hd + dd];
      acc2 += wsh[c + 2] * op[(size_t)(c + 2) * hd + dd];
      acc3 += wsh[c + 3] * op[(size_t)(c + 3) * hd + dd];
    }
    for (; c < nch; ++c) acc0 += wsh[c] * op[(size_t)c * hd + dd];
    put_o(a, o, r, head, dd, ((acc0 + acc1) + (acc2 + acc3)) * inv);
  }
}

// ---------------------------------------------------------------- combine (bf16 path)
// One wave per (row, head).  Every load is issued before the first wait: the
// row's (max, sum) pairs (lane c holds splits c, c+64, ...) and the first 16
// splits' partial outputs (lane holds dims lane, lane+64); each later chunk is
// requested before the current one is accumulated.  o = sum_c w_c o_c /
// sum_c w_c l_c with w_c = exp(m_c - max_c m_c), summed over c in order in four
// interleaved accumulators.
constexpr int kCombineMaxSplits = 256;  // 4 per lane

template <int HD>
__global__ __launch_bounds__(64) void attn_combine_wave_kernel(AttnArgs a) {
  constexpr int DPL = HD >= 64 ? HD / 64 : 1;  // dims per lane
  constexpr int CH = 16;                        // splits per chunk of partial outputs
  const int head = blockIdx.x, r = blockIdx.y, lane = threadIdx.x, H = a.n_heads, ns = a.n_split;
  const size_t base = ((size_t)r * H + head) * ns;
  const __amdgpu_buffer_rsrc_t mlr =
      __builtin_amdgcn_make_buffer_rsrc(a.ml_part + 2 * base, (short)0, ns * 8, 0x00020000);
  const __amdgpu_buffer_rsrc_t opr =
      __builtin_amdgcn_make_buffer_rsrc(a.o_part + base * HD, (short)0, ns * HD * 4, 0x00020000);
  // (two 4-byte loads per pair: this toolchain's 8-byte raw buffer load returns
  // the low word in both elements)
  float mv[4], lv[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const uint32_t c = lane + 64 * j;
    mv[j] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(mlr, c * 8u, 0, 0));
    lv[j] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(mlr, c * 8u + 4u, 0, 0));
  }
  auto load_chunk = [&](int c0, float (&ov)[CH][DPL]) {
#pragma unroll
    for (int cc = 0; cc < CH; ++cc)
#pragma unroll
      for (int d = 0; d < DPL; ++d) {
        const uint32_t dim = lane + 64 * d;
        const uint32_t off = (((uint32_t)(c0 + cc) * HD + dim) * 4u) | ((uint32_t)(dim >= (uint32_t)HD) << 31);
        ov[cc][d] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(opr, off, 0, 0));
      }
  };
  // Partial outputs of NG chunks (64 splits) are requested at once: one memory
  // round trip for contexts up to 64 splits, one more per further 64.
  constexpr int NG = 4;
  float ov[NG][CH][DPL];
#pragma unroll
  for (int g = 0; g < NG; ++g) load_chunk(g * CH, ov[g]);
  asm volatile("" ::: "memory");  // (keep the loads above the exits below)

  const RowDesc rd = a.rows[r];
  float* o = a.o + ((size_t)r * H + head) * HD;
  if (!rd.valid) {
#pragma unroll
    for (int d = 0; d < DPL; ++d)
      if (lane + 64 * d < HD) put_o(a, o, r, head, lane + 64 * d, 0.f);
    return;
  }
  // parts holding keys <= pos (the last part also holds the remainder)
  const int nch = min(rd.pos / a.chunk + 1, ns);
  if (rd.pos + 1 > a.max_ctx && lane == 0) set_status(a.status, kStatusKvCapacity);  // the host's bound was wrong
  float mx = -INFINITY;
#pragma unroll
  for (int j = 0; j < 4; ++j)
    if (lane + 64 * j < nch) mx = fmaxf(mx, mv[j]);
  mx = wave_max(mx);
  float wv[4], L = 0.f;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    wv[j] = lane + 64 * j < nch ? expf(mv[j] - mx) : 0.f;
    L += wv[j] * lv[j];
  }
  L = wave_sum(L);
  float acc[4][DPL];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int d = 0; d < DPL; ++d) acc[i][d] = 0.f;
  for (int g0 = 0; g0 < nch; g0 += NG * CH) {
    if (g0 > 0) {
#pragma unroll
      for (int g = 0; g < NG; ++g) load_chunk(g0 + g * CH, ov[g]);
    }
#pragma unroll
    for (int g = 0; g < NG; ++g)
#pragma unroll
      for (int cc = 0; cc < CH; ++cc) {
        const int c = g0 + g * CH + cc;
        if (c < nch) {
          const float wj = c < 64 ? wv[0] : (c < 128 ? wv[1] : (c < 192 ? wv[2] : wv[3]));
          const float w = __shfl(wj, c & 63, kWave);
#pragma unroll
          for (int d = 0; d < DPL; ++d) acc[cc & 3][d] += w * ov[g][cc][d];
        }
      }
  }
  const float inv = 1.0f / L;
#pragma unroll
  for (int d = 0; d < DPL; ++d)
    if (lane + 64 * d < HD) put_o(a, o, r, head, lane + 64 * d, ((acc[0][d] + acc[1][d]) + (acc[2][d] + acc[3][d])) * inv);
}

// ---------------------------------------------------------------- KV context copy
template <typename KT>
__global__ __launch_bounds__(256) void kv_copy_kernel(KvLayout kv, int layer, int b, int pos0, const KT* k,
                                                      const KT* v, KT* k_out, KT* v_out) {
  const int p = blockIdx.x;
  const int hd = kv.head_dim, G = kv.n_kv_heads;
  for (int i = threadIdx.x; i < G * hd; i += blockDim.x) {
    const int g = i / hd, dd = i % hd;
    KT* blk = k_block<KT>(kv, layer, b, g);
    KT* kc = blk + KvIndex<KT>::k(pos0 + p, dd, hd, kv.capacity);
    KT* vc = blk + KvIndex<KT>::v(pos0 + p, dd, hd, kv.capacity);
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

int attention_chunk(int dtype, int head_dim) {
  if (dtype == SPECDEC_BF16) return kSubKeys;  // (parts are whole numbers of sub-chunks: at most one split each)
  return head_dim >= 128 ? 32 : (head_dim >= 64 ? 64 : 128);
}

hipError_t launch_rope_append(const AttnArgs& a, hipStream_t s) {
  dim3 grid(a.n_heads + 2 * a.n_kv_heads, a.M);
  if (a.kv.dtype == SPECDEC_BF16)
    hipLaunchKernelGGL((rope_append_kernel<uint16_t>), grid, dim3(64), 0, s, a);
  else
    hipLaunchKernelGGL((rope_append_kernel<float>), grid, dim3(64), 0, s, a);
  return hipGetLastError();
}

__global__ void fill_u32_kernel(uint32_t* p, size_t n, uint32_t v) {
  const size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

hipError_t launch_fill_u32(uint32_t* p, size_t n, uint32_t v, hipStream_t s) {
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(fill_u32_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, p, n, v);
  return hipGetLastError();
}

size_t attention_counter_count(int n_heads, int n_kv_heads, int max_rows) {
  // sequences x query tiles <= max_rows * group / 16 + max_rows
  const size_t group = (size_t)(n_heads / n_kv_heads);
  return (size_t)n_kv_heads * ((size_t)max_rows * group / 16 + (size_t)max_rows + 1);
}

size_t attention_ll_words(int n_heads, int head_dim, int max_rows, int n_split_max) {
  // slots (row, head, part) for up to min(kLlMaxParts, n_split_max) parts: a
  // launch's parts never outnumber its sub-chunks, ceil(max_ctx / 32)
  const size_t parts = (size_t)std::min(kLlMaxParts, n_split_max);
  return (size_t)max_rows * n_heads * parts * (head_dim + 2);
}

hipError_t launch_attention(const AttnArgs& a, hipStream_t s) {
  const int B = a.M / a.rps;
  AttnArgs ab = a;  // the bf16 path chooses its own parts
  if (a.kv.dtype == SPECDEC_BF16) {
    const int nq = a.rps * (a.n_heads / a.n_kv_heads), n_mt = (nq + 15) / 16, RS = nq < 16 ? nq : 16;
    const int n_sub = (a.max_ctx + kSubKeys - 1) / kSubKeys;
    if (n_sub * kSubKeys > a.kv.capacity || n_sub > a.n_split * (a.chunk / kSubKeys)) return hipErrorInvalidValue;
    const long units = (long)a.n_kv_heads * B * n_mt;
    const int cus = device_compute_units();
    int S = 0, n_part = 0, NW = 0;
    if (n_sub * units <= (long)cus * kMaxPartWaves) {
      // One sub-chunk per wave, one round: parts of S sub-chunks (the last one
      // takes the remainder), the blocks about filling the CUs once.
      S = (int)((n_sub * units + cus / 2) / cus);
      S = S < 1 ? 1 : (S > kMaxPartWaves ? kMaxPartWaves : S);  // (reduced below while the last part is too big)
      // (more units than CUs: a part never holds more sub-chunks than the keys
      // have, so its waves take one sub-chunk each and never loop)
      S = std::max(1, std::min(S, n_sub));
      for (;; --S) {
        n_part = n_sub / S > 0 ? n_sub / S : 1;
        NW = n_sub - (n_part - 1) * S;
        if (S == 1 || (NW <= kMaxPartWaves && attn_block_lds(NW, RS, a.head_dim) <= 65536)) break;
      }
    } else {
      // Long contexts: 4-wave blocks whose waves loop over the sub-chunks of
      // their part; parts sized for about 12 blocks per CU (two resident per
      // CU, six rounds: short tails when sequences differ in length; measured
      // on 16 sequences of 1024-8192 keys: 4, 8, 10, 12, 16 and 24 blocks per
      // CU, 12 the fastest).
      NW = kLoopWaves;
      const long parts = std::max(1L, (12L * cus + units - 1) / units);
      S = (int)((n_sub + parts - 1) / parts);
      S = (S + NW - 1) / NW * NW;
      n_part = (n_sub + S - 1) / S;
    }
    if (NW > kMaxPartWaves || attn_block_lds(NW, RS, a.head_dim) > 65536) return hipErrorInvalidValue;
    ab.n_split = n_part;
    ab.chunk = S * kSubKeys;
    // In-kernel combine: one part per lane, at most two query rows per wave of
    // the combining block (its rows go one after another), and its own part's
    // rows fit in LDS next to the merge buffers; otherwise the separate
    // combine kernel (one wave per row and head).
    // (Looping launches combine through the tagged words and keep the
    // combining block's own part in LDS; one-round launches count arrivals.)
    const bool loop = S > NW;
    if (loop) ab.counters = nullptr;
    else {
      ab.ll = nullptr;
      ab.epochs = nullptr;
    }
    if (n_part > kLlMaxParts || (RS + NW - 1) / NW > 2 || attn_block_lds(NW, RS, a.head_dim, loop) > 65536 ||
        (loop ? !ab.ll || !ab.epochs : !ab.counters)) {
      ab.epochs = nullptr;
      ab.counters = nullptr;
      ab.ll = nullptr;
    }
    dim3 grid(n_part * n_mt, a.n_kv_heads, B);
    const size_t lds = attn_block_lds(NW, RS, a.head_dim, ab.ll != nullptr);
    if (loop && NW > kLoopWaves) return hipErrorInvalidValue;  // (the looping kernel's block bound)
#define SD_ATTN(HDV)                                                                                       \
  if (loop) hipLaunchKernelGGL((attn_block_kernel<HDV, true>), grid, dim3(64 * NW), lds, s, ab, S, n_sub, NW); \
  else hipLaunchKernelGGL((attn_block_kernel<HDV, false>), grid, dim3(64 * NW), lds, s, ab, S, n_sub, NW);
    switch (a.head_dim) {
      case 32: SD_ATTN(32) break;
      case 64: SD_ATTN(64) break;
      case 128: SD_ATTN(128) break;
      default: return hipErrorInvalidValue;
    }
#undef SD_ATTN
  } else {
    const size_t smem = attn_smem_bytes(a.chunk, a.head_dim);
    dim3 grid(a.n_split, a.n_kv_heads, B);
    hipLaunchKernelGGL((attn_partial_kernel<float>), grid, dim3(256), smem, s, a);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (ab.kv.dtype == SPECDEC_BF16 && (ab.ll || ab.counters)) return hipSuccess;  // combined by the blocks
  if (ab.kv.dtype == SPECDEC_BF16 && ab.n_split <= kCombineMaxSplits) {
    switch (ab.head_dim) {
      case 32: hipLaunchKernelGGL((attn_combine_wave_kernel<32>), dim3(ab.n_heads, ab.M), dim3(64), 0, s, ab); break;
      case 64: hipLaunchKernelGGL((attn_combine_wave_kernel<64>), dim3(ab.n_heads, ab.M), dim3(64), 0, s, ab); break;
      default: hipLaunchKernelGGL((attn_combine_wave_kernel<128>), dim3(ab.n_heads, ab.M), dim3(64), 0, s, ab); break;
    }
  } else {
    hipLaunchKernelGGL(attn_combine_kernel, dim3(ab.n_heads, ab.M), dim3(128), sizeof(float) * ab.n_split, s, ab);
  }
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
