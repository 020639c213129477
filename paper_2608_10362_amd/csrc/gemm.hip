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
#include <algorithm>
#include <type_traits>

#include "device_common.h"
#include "internal.h"

namespace specdec {

namespace {

constexpr int kMfmaThreads = 1024;  // 16 waves split K
constexpr int kMfmaWaves = kMfmaThreads / kWave;

__device__ __forceinline__ float silu_f(float z) { return z / (1.0f + expf(-z)); }

// Raw buffer descriptor over `bytes` bytes at `base` (dword 3: the gfx9 raw
// buffer format); loads past `bytes` return zeros.
constexpr uint32_t kOutOfRange = 0x80000000u;
constexpr int kNonTemporal = 2;  // cache-policy bit of a streamed (read-once) load
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}

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

// Epilogue over this block's final sums yfin[m][c], c < NC columns (store,
// residual, SwiGLU; the MFMA kernel has its own residual and QKV epilogues
// that take their inputs from registers and LDS).
template <int NC, int KIND, int NTH>
__device__ __forceinline__ void epilogue(const GemmArgs& a, int blk, float (*yfin)[NC + 1], const float* scale) {
  const int M = a.M;  // (NTH = threads of the block: a constant, not a read of the dispatch packet)
  if (KIND == EPI_STORE) {
    for (int i = threadIdx.x; i < M * NC; i += NTH) {
      int m = i / NC, c = i % NC;
      int n = blk * NC + c;
      if (n < a.n_rows) a.out[(size_t)m * a.ldo + n] = yfin[m][c] * scale[m];
    }
  } else if (KIND == EPI_RESID) {
    for (int i = threadIdx.x; i < M * NC; i += NTH) {
      int m = i / NC, c = i % NC;
      int n = blk * NC + c;
      float hv = 0.f;
      if (n < a.n_rows) {
        float* hp = a.out + (size_t)m * a.ldo + n;
        hv = *hp + yfin[m][c];
        *hp = hv;
        const float xv = hv * load_gain(a.gain_out, a.gain_bf16, n);
        a.xg_out[(size_t)m * a.ldo + n] = xv;
        if (a.xs_out) put_stacked(a.xs_out, a.stt, m, n, xv);
      }
      yfin[m][c] = hv;
    }
    __syncthreads();
    for (int m = threadIdx.x; m < M; m += NTH) {
      float t = 0.f;
      for (int c = 0; c < NC; ++c) t += yfin[m][c] * yfin[m][c];
      a.ss_out[(size_t)blk * a.ss_ld + m] = t;
    }
  } else {  // EPI_SWIGLU: columns [0, NC/2) gate, [NC/2, NC) up
    constexpr int H = NC / 2;
    for (int i = threadIdx.x; i < M * H; i += NTH) {
      int m = i / H, c = i % H;
      int n = blk * H + c;
      if (n < a.n_rows) {
        float g = yfin[m][c] * scale[m];
        float u = yfin[m][H + c] * scale[m];
        const float y = silu_f(g) * u;
        a.out[(size_t)m * a.ldo + n] = y;
        if (a.xs_out) put_stacked(a.xs_out, a.stt, m, n, y);
      }
    }
  }
}

// Q|K|V epilogue over this block's final sums yfin[m][c], c < NC columns of
// the concatenated Q|K|V rows (bf16 cache).  Columns of the Q and K segments
// come in RoPE pairs: column c (c % 16 < 8) is dim j = 8 * (tile within the
// head) + c % 8 of its head, column c ^ 8 is dim j + hd/2; x1' = x1 cos - x2
// sin, x2' = x2 cos + x1 sin.  Rotated queries go to qr, K and V into the
// cache at each valid row's position.  s_rows / s_cs: the rows' descriptors
// and cos | sin tables.
template <int NC, int NTH>
__device__ __forceinline__ void qkv_epilogue(const GemmArgs& a, int blk, const float (*yfin)[NC + 1],
                                             const float* scale, const RowDesc* s_rows, const float (*s_cs)[128]) {
  const int M = a.M, hd = a.head_dim, half = hd >> 1, H = a.n_heads;
  const int nq = a.n_seg[0], nqk = nq + a.n_seg[1], cap = a.kv.capacity;
#pragma unroll 1
  for (int i = threadIdx.x; i < M * NC; i += NTH) {
    const int m = i / NC, c = i % NC, n = blk * NC + c;
    if (n >= a.n_rows) continue;
    const float x = yfin[m][c] * scale[m];
    const RowDesc rd = s_rows[m];
    if (n < nqk) {
      const bool is_k = n >= nq;
      const int r = is_k ? n - nq : n;
      const int head = r / hd, w = r % hd, ec = w & 15;
      const int j = 8 * (w >> 4) + (ec & 7);
      const float y = yfin[m][c ^ 8] * scale[m];
      const float cs = s_cs[m][j], sn = s_cs[m][half + j];
      const float out = ec < 8 ? x * cs - y * sn : x * cs + y * sn;
      const int d = ec < 8 ? j : half + j;
      if (!is_k) {
        a.qr[((size_t)m * H + head) * hd + d] = out;
      } else if (rd.valid) {
        uint16_t* kvb = k_block<uint16_t>(a.kv, a.layer, rd.b, head);
        Storage<uint16_t>::store(kvb + KvIndex<uint16_t>::k(rd.pos, d, hd, cap), out);
      }
    } else if (rd.valid) {
      const int r = n - nqk, head = r / hd, d = r % hd;
      uint16_t* kvb = k_block<uint16_t>(a.kv, a.layer, rd.b, head);
      Storage<uint16_t>::store(kvb + KvIndex<uint16_t>::v(rd.pos, d, hd, cap), x);
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

// Segment and local row of row tile t of block blk (as weight_tile).
__device__ __forceinline__ void tile_segment(const GemmArgs& a, int kind, int blk, int NC, int t, int& seg, int& n,
                                             bool& ok) {
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
}

// INT4 image of W [N, K]: per 16-row tile and group of 128 columns a 1 KB
// block in which lane l = 16*(k%32/8) + n%16 holds 16 bytes, the words of
// the group's four k-steps; word j holds the 8 codes of row n at columns
// 128g + 32j + 8*(l/16) .. +7, low nibble first.  Then the group scales
// [N/16][KG][16] (bf16).
struct Q4Frag {
  uint32_t codes;
  uint32_t scale;  // bf16 bits of the group scale of the lane's row (lane % 16)
};

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
template <int T, int MT, int UB, bool PIPE, int KIND, bool Q4 = false, int XS = 0>
__global__ __launch_bounds__(kMfmaThreads) void gemm_bf16_mfma(GemmArgs a, int n_tiles) {
  // Q4: INT4 weights (Q4Frag).  A code q is fed to the MFMA as the bf16 value
  // 136 + q (bits 0x4300 | (q + 8): two byte permutes and an OR per four
  // codes), and the bias is cancelled inside the accumulator by a product of
  // the same x with the constant -136, shared by the unit's tiles; each
  // k-step's product is then multiplied by the lane's row scale in float32,
  // so the effective weights are code * scale.
  // XS > 0: x comes as the stacked operand a.xs (put_stacked, XS fragments
  // per k-step, at most 8 rows when XS = 1, 16 when XS = 2) in place of the
  // float32 rows: one 16-byte load per fragment and one product per fragment
  // and tile.  The hi and lo parts accumulate apart (accumulator tiles 0 and
  // 1, or rows m and 8 + m of tile 0) and are added once per tile before the
  // cross-wave sums, the same arithmetic for either count of fragments.
  // XS = 3: XS = 1 with each wave's x fragments (at most 8 k-steps, K <= 4096)
  // fetched once into LDS and read from there for every unit of the block.
  static_assert(XS == 0 || (MT == 1 && !Q4), "stacked x: bf16 weights, one row tile");
  using WReg = std::conditional_t<Q4, Q4Frag, u32x4>;
  constexpr bool XL = XS == 3;
  constexpr int XF = XL ? 1 : XS;   // stacked fragments per k-step
  constexpr int MA = XS ? XF : MT;  // accumulator row tiles
  constexpr int NC = 16 * T;
  constexpr int MP = 16 * MT;
  constexpr int NF = T * MT;              // accumulator fragments per wave
  constexpr int RR = XL ? 1 : (NF <= 2 ? NF : 2);  // fragments reduced per LDS round (XL: LDS goes to x)
  constexpr bool QKV = KIND == EPI_QKV;
  constexpr int E = (MP * NC + kMfmaThreads - 1) / kMfmaThreads;  // epilogue elements per thread
  __shared__ float red[RR][kMfmaWaves][kWave][4];
  __shared__ u32x4 s_xl[XL ? kMfmaWaves : 1][XL ? 8 : 1][kWave];  // XL: wave w's x fragments, k-steps w + 16j
  __shared__ float yfin[MP][NC + 1];
  __shared__ float scale[MP];
  __shared__ RowDesc s_rows[QKV ? MP : 1];
  __shared__ float s_cs[QKV ? MP : 1][QKV ? 128 : 1];  // RoPE cos | sin of each row (head_dim <= 128)

  // The wave index is uniform across the wave; saying so keeps every per-wave
  // quantity derived from it (k-step list, tile, weight segment, buffer
  // descriptors) in scalar registers.
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int kg = lane >> 4, mrow = lane & 15;
  // Stacked x: the lanes of a fragment's padding rows (rows >= M of its hi and
  // lo halves) read nothing, which keeps them zero; only rows < M reach an
  // output (5 rows: 10 of the 16 fragment rows fetched, 1 row: 2).
  const uint32_t xrbad = XS ? (uint32_t)(((XS == 2 ? mrow : (mrow & 7)) >= a.M)) << 31 : 0u;
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

  floatx4 acc[T][MA];
#pragma unroll
  for (int t = 0; t < T; ++t)
#pragma unroll
    for (int mt = 0; mt < MA; ++mt) acc[t][mt] = floatx4{0.f, 0.f, 0.f, 0.f};

  WReg wA[UB][T], wB[UB][T];
  f32x4 xA[UB][MA][2], xB[UB][MA][2];  // (stacked x: [u][fragment][0] holds the fragment's 16 bytes)
  // Residual epilogue inputs (old h and the next RMSNorm gain) of the tile whose
  // last batch sits in the matching register buffer, fetched with that batch.
  // (Only when every thread has at most one epilogue element; larger row
  // counts read them in the epilogue, keeping the registers for the loads.)
  constexpr bool PRE = KIND == EPI_RESID && E == 1;
  struct Pre {
    float h[E];
    uint32_t g[E];  // bf16 bits of the gain (bf16 models only run this kernel)
  } pA, pB;
  auto epi_fetch = [&](int q, Pre& p) {
    if constexpr (PRE) {
      // (every batch fetches its tile's inputs: no branch; the copy fetched with
      // the tile's last batch is the one its epilogue uses)
      const int tile = blockIdx.x + (q / nbat) * gridDim.x;
      const __amdgpu_buffer_rsrc_t hr = make_rsrc(a.out, (uint32_t)a.M * a.ldo * 4u);
      const __amdgpu_buffer_rsrc_t gr = make_rsrc(a.gain_out, (uint32_t)a.n_rows * 2u);
#pragma unroll
      for (int e = 0; e < E; ++e) {
        const int i = tid + e * kMfmaThreads, m = i / NC, n = tile * NC + i % NC;
        const uint32_t bad = (uint32_t)(n >= a.n_rows) << 31;  // (rows m >= M fall outside hr)
        p.h[e] = __builtin_bit_cast(
            float, __builtin_amdgcn_raw_buffer_load_b32(hr, (((uint32_t)m * a.ldo + n) * 4u) | bad, 0, 0));
        p.g[e] = __builtin_amdgcn_raw_buffer_load_b16(gr, ((uint32_t)n * 2u) | bad, 0, 0);
      }
    }
  };
  // Loads go through buffer descriptors: an offset past the descriptor's range
  // reads zeros without touching memory, so rows beyond M, tiles beyond N and
  // k-steps beyond the wave's list need no branches (a branch around a load
  // makes the compiler wait for the data where the paths join).
  const __amdgpu_buffer_rsrc_t xr = XS ? make_rsrc(a.xs, (uint32_t)KS * XF * 1024u)
                                       : make_rsrc(a.x, (uint32_t)a.M * a.ldx * 4u);
  // load the q-th batch of this wave's work list (tile q / nbat, k-steps from (q % nbat) * UB)
  auto load = [&](int q, WReg (&wv)[UB][T], f32x4 (&xv)[UB][MA][2]) {
    const int tile = blockIdx.x + (q / nbat) * gridDim.x;
    const int kb = (q % nbat) * UB;  // index into this wave's k-step list
    __amdgpu_buffer_rsrc_t wr[T], sr[T];
#pragma unroll
    for (int t = 0; t < T; ++t) {
      bool rok;
      if constexpr (Q4) {
        int seg, n;
        tile_segment(a, KIND, tile, NC, t, seg, n, rok);
        const int KG = (K + 127) / 128;
        wr[t] = make_rsrc((const char*)a.w[seg] + (size_t)(n / 16) * KG * 1024, rok ? (uint32_t)KG * 1024u : 0u);
        sr[t] = make_rsrc(a.wscale[seg] + (size_t)(n / 16) * KG * 16, rok ? (uint32_t)KG * 32u : 0u);
      } else {
        const uint16_t* base = weight_tile(a, KIND, tile, NC, t, KS, rok);
        wr[t] = make_rsrc(base, rok ? (uint32_t)KS * 1024u : 0u);
      }
    }
#pragma unroll
    for (int u = 0; u < UB; ++u) {
      const int ks = ks0 + (kb + u) * kstride;
      const int k = ks * 32 + kg * 8;
      // (out-of-range flags are OR-ed into the offsets: a select on a wave-uniform
      // flag would become a branch)
      const uint32_t wbad = (uint32_t)((kb + u) >= my_ks || ks >= KS) << 31;
      const uint32_t woff = ((uint32_t)ks * 1024u + lane * 16u) | wbad;
#pragma unroll
      for (int t = 0; t < T; ++t) {
        if constexpr (Q4) {
          const uint32_t qoff = ((uint32_t)(ks >> 2) * 1024u + lane * 16u + (uint32_t)(ks & 3) * 4u) | wbad;
          const uint32_t soff = ((uint32_t)(ks >> 2) * 32u + (lane & 15) * 2u) | wbad;
          wv[u][t].codes = __builtin_amdgcn_raw_buffer_load_b32(wr[t], qoff, 0, kNonTemporal);
          wv[u][t].scale = __builtin_amdgcn_raw_buffer_load_b16(sr[t], soff, 0, 0);
        } else {
          wv[u][t] = __builtin_amdgcn_raw_buffer_load_b128(wr[t], woff, 0, kNonTemporal);
        }
      }
      if constexpr (XL) {
        // (x comes from LDS)
      } else if constexpr (XS) {
#pragma unroll
        for (int f = 0; f < XS; ++f) {
          const uint32_t xoff = (((uint32_t)ks * XS + f) * 1024u + lane * 16u) | wbad | xrbad;
          xv[u][f][0] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(xr, xoff, 0, 0));
        }
      } else {
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
          const int m = mt * 16 + mrow;
          const uint32_t xoff = (((uint32_t)m * a.ldx + k) * 4u) | wbad | ((uint32_t)(k >= K) << 31);
          xv[u][mt][0] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(xr, xoff, 0, 0));
          xv[u][mt][1] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(xr, xoff + 16u, 0, 0));
        }
      }
    }
  };
  auto compute = [&](WReg (&wv)[UB][T], f32x4 (&xv)[UB][MA][2], int q) {
    if constexpr (XL) {
      const int kb = (q % nbat) * UB;  // (past the wave's k-steps the weights read zeros)
#pragma unroll
      for (int u = 0; u < UB; ++u) {
        const bf16x8 xf = __builtin_bit_cast(bf16x8, s_xl[wave][min(kb + u, 7)][lane]);
#pragma unroll
        for (int t = 0; t < T; ++t)
          acc[t][0] =
              __builtin_amdgcn_mfma_f32_16x16x32_bf16(xf, __builtin_bit_cast(bf16x8, wv[u][t]), acc[t][0], 0, 0, 0);
      }
      return;
    }
    if constexpr (XS) {
#pragma unroll
      for (int u = 0; u < UB; ++u)
#pragma unroll
        for (int f = 0; f < XS; ++f) {
          const bf16x8 xf = __builtin_bit_cast(bf16x8, xv[u][f][0]);
#pragma unroll
          for (int t = 0; t < T; ++t)
            acc[t][f] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xf, __builtin_bit_cast(bf16x8, wv[u][t]), acc[t][f],
                                                                0, 0, 0);
        }
      return;
    }
#pragma unroll
    for (int u = 0; u < UB; ++u) {
      // Q4: the codes of each tile as biased bf16 operands and the row scales
      bf16x8 bq[Q4 ? T : 1];
      float sc[Q4 ? T : 1];
      if constexpr (Q4) {
#pragma unroll
        for (int t = 0; t < T; ++t) {
          const uint32_t c = wv[u][t].codes ^ 0x88888888u;  // q + 8 in each nibble
          const uint32_t even = c & 0x0F0F0F0Fu, odd = (c >> 4) & 0x0F0F0F0Fu;  // codes 0,2,4,6 / 1,3,5,7
          u32x4 v;
          // dword j/2 of the operand: code j in its low half, code j+1 in its high half
          v[0] = __builtin_amdgcn_perm(odd, even, 0x0c040c00u) | 0x43004300u;
          v[1] = __builtin_amdgcn_perm(odd, even, 0x0c050c01u) | 0x43004300u;
          v[2] = __builtin_amdgcn_perm(odd, even, 0x0c060c02u) | 0x43004300u;
          v[3] = __builtin_amdgcn_perm(odd, even, 0x0c070c03u) | 0x43004300u;
          bq[t] = __builtin_bit_cast(bf16x8, v);
          sc[t] = bf16_bits_to_f32((uint16_t)wv[u][t].scale);
        }
      }
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
        floatx4 bias = floatx4{0.f, 0.f, 0.f, 0.f};
        if constexpr (Q4) {  // -136 * sum_k x[m][k] in every column
          const u32x4 m136 = u32x4{0xC308C308u, 0xC308C308u, 0xC308C308u, 0xC308C308u};
          bias = __builtin_amdgcn_mfma_f32_16x16x32_bf16(hi, __builtin_bit_cast(bf16x8, m136), bias, 0, 0, 0);
          bias = __builtin_amdgcn_mfma_f32_16x16x32_bf16(lo, __builtin_bit_cast(bf16x8, m136), bias, 0, 0, 0);
        }
#pragma unroll
        for (int t = 0; t < T; ++t) {
          if constexpr (Q4) {
            floatx4 p = __builtin_amdgcn_mfma_f32_16x16x32_bf16(hi, bq[t], bias, 0, 0, 0);
            p = __builtin_amdgcn_mfma_f32_16x16x32_bf16(lo, bq[t], p, 0, 0, 0);
#pragma unroll
            for (int r = 0; r < 4; ++r) acc[t][mt][r] = fmaf(sc[t], p[r], acc[t][mt][r]);
          } else {
            const bf16x8 b = __builtin_bit_cast(bf16x8, wv[u][t]);
            acc[t][mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(hi, b, acc[t][mt], 0, 0, 0);
            acc[t][mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(lo, b, acc[t][mt], 0, 0, 0);
          }
        }
      }
    }
  };
  auto mfma_epilogue = [&](int blk, const Pre& p) {
    const int M = a.M;
    if constexpr (PRE) {
      const int m = tid / NC, c = tid % NC, n = blk * NC + c;
      if (m < M) {
        float hv = 0.f;
        if (n < a.n_rows) {
          hv = p.h[0] + yfin[m][c];
          a.out[(size_t)m * a.ldo + n] = hv;
          const float xv = hv * bf16_bits_to_f32((uint16_t)p.g[0]);
          a.xg_out[(size_t)m * a.ldo + n] = xv;
          if (a.xs_out) put_stacked(a.xs_out, a.stt, m, n, xv);
        }
        yfin[m][c] = hv;
      }
      __syncthreads();
      for (int m = tid; m < M; m += kMfmaThreads) {
        float t = 0.f;
        for (int c = 0; c < NC; ++c) t += yfin[m][c] * yfin[m][c];
        a.ss_out[(size_t)blk * a.ss_ld + m] = t;
      }
    } else if constexpr (KIND == EPI_QKV) {
      qkv_epilogue<NC, kMfmaThreads>(a, blk, yfin, scale, s_rows, s_cs);
    } else {
      epilogue<NC, KIND, kMfmaThreads>(a, blk, yfin, scale);
    }
  };
  // After the last batch of a tile: cross-wave reduction (fixed wave order) and epilogue.
  auto finish = [&](int q, const Pre& p) {
    if (q % nbat != nbat - 1) return;
    const int tile = blockIdx.x + (q / nbat) * gridDim.x;
    if constexpr (XF == 1) {  // hi (rows 0-7, lanes 0-31) + lo (rows 8-15, lanes 32-63)
#pragma unroll
      for (int t = 0; t < T; ++t)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float v = acc[t][0][r], o = __shfl_xor(v, 32, kWave);
          acc[t][0][r] = lane < 32 ? v + o : 0.f;
        }
    } else if constexpr (XF == 2) {  // hi (tile 0) + lo (tile 1)
#pragma unroll
      for (int t = 0; t < T; ++t) acc[t][0] += acc[t][1];
    }
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
      for (int mt = 0; mt < MA; ++mt) acc[t][mt] = floatx4{0.f, 0.f, 0.f, 0.f};
    mfma_epilogue(tile, p);
    __syncthreads();  // yfin is reused by the next tile
  };

  // Prologue.  The small operands only the epilogue needs (row-scale partial
  // sums, the QKV tables) are requested first, then both register buffers'
  // weight batches; storing the small ones then waits for them alone (loads
  // complete in order), so no wave waits for a weight batch before its first
  // multiply.
  constexpr int RS_ROWS = (MP + kMfmaWaves - 1) / kMfmaWaves;  // scale rows per wave
  constexpr int RS_P = 4;                                      // partial sums per lane held
  float rs_v[RS_ROWS][RS_P];
  {
    const __amdgpu_buffer_rsrc_t sr = make_rsrc(a.ss_in, a.ss_in ? (uint32_t)a.n_ss * a.ss_ld * 4u : 0u);
#pragma unroll
    for (int r = 0; r < RS_ROWS; ++r) {
      const int m = wave + r * kMfmaWaves;
#pragma unroll
      for (int i = 0; i < RS_P; ++i) {
        const int p = lane + i * kWave;
        const uint32_t off = (m < a.M && p < a.n_ss) ? ((uint32_t)p * a.ss_ld + m) * 4u : kOutOfRange;
        rs_v[r][i] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(sr, off, 0, 0));
      }
    }
  }
  constexpr bool HOIST = QKV && MT <= 2;  // (the 64-row tables would cost spills)
  constexpr int CS_E = HOIST ? MP * 128 / kMfmaThreads : 1;  // table entries per thread
  float cs_v[CS_E];
  RowDesc rd_v{0, 0, 0, 0};
  if constexpr (HOIST) {
    const __amdgpu_buffer_rsrc_t cr = make_rsrc(a.rope_cs, (uint32_t)a.M * a.head_dim * 4u);
#pragma unroll
    for (int e = 0; e < CS_E; ++e) {
      const int i = tid + e * kMfmaThreads, m = i / 128, j = i % 128;
      const uint32_t off = j < a.head_dim ? ((uint32_t)m * a.head_dim + j) * 4u : kOutOfRange;
      cs_v[e] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(cr, off, 0, 0));
    }
    const __amdgpu_buffer_rsrc_t rr = make_rsrc(a.rows, (uint32_t)a.M * (uint32_t)sizeof(RowDesc));
    rd_v = __builtin_bit_cast(RowDesc, __builtin_amdgcn_raw_buffer_load_b128(
                                           rr, tid < MP ? (uint32_t)tid * (uint32_t)sizeof(RowDesc) : kOutOfRange, 0, 0));
  }
  int q = 0;
  u32x4 xl[XL ? 8 : 1];
  if constexpr (XL) {  // this wave's x fragments, requested before the weights
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int ks = ks0 + j * kstride;
      xl[j] = __builtin_amdgcn_raw_buffer_load_b128(
          xr, ((uint32_t)ks * 1024u + lane * 16u) | ((uint32_t)(j >= my_ks || ks >= KS) << 31) | xrbad, 0, 0);
    }
  }
  if (total > 0) {
    load(0, wA, xA);
    epi_fetch(0, pA);
  }
  if (PIPE && total > 1) {
    load(1, wB, xB);
    epi_fetch(1, pB);
  }
  if constexpr (XL) {  // (read back by this wave only)
#pragma unroll
    for (int j = 0; j < 8; ++j) s_xl[wave][j][lane] = xl[j];
  }
  // s_m = 1/sqrt(sum_p ss[p][m] / K + eps): lanes sum their partials in p order
  // (held ones first, then any beyond 64*RS_P), fixed shuffle tree.
  {
    float t[RS_ROWS];
#pragma unroll
    for (int r = 0; r < RS_ROWS; ++r) {
      const int m = wave + r * kMfmaWaves;
      t[r] = 0.f;
#pragma unroll
      for (int i = 0; i < RS_P; ++i) t[r] += rs_v[r][i];
      if (a.ss_in && m < a.M)
        for (int p = lane + RS_P * kWave; p < a.n_ss; p += kWave) t[r] += a.ss_in[(size_t)p * a.ss_ld + m];
    }
    wave_sum_n(t);
#pragma unroll
    for (int r = 0; r < RS_ROWS; ++r) {
      const int m = wave + r * kMfmaWaves;
      if (lane == 0 && m < MP) scale[m] = (a.ss_in && m < a.M) ? 1.0f / sqrtf(t[r] / (float)a.K + a.eps) : 1.0f;
    }
  }
  if constexpr (HOIST) {
#pragma unroll
    for (int e = 0; e < CS_E; ++e) {
      const int i = tid + e * kMfmaThreads;
      s_cs[i / 128][i % 128] = cs_v[e];
    }
    if (tid < MP) s_rows[tid] = rd_v;
  } else if constexpr (QKV) {
    for (int i = tid; i < MP; i += kMfmaThreads) s_rows[i] = i < a.M ? a.rows[i] : RowDesc{0, 0, 0, 0};
    for (int i = tid; i < MP * 128; i += kMfmaThreads) {
      const int m = i / 128, j = i % 128;
      s_cs[m][j] = (m < a.M && j < a.head_dim) ? a.rope_cs[(size_t)m * a.head_dim + j] : 0.f;
    }
  }
  if (PIPE) {
    // A buffer is refilled as soon as its batch has been multiplied, before the
    // tile's reduction and epilogue (which use only the accumulators, LDS and
    // the epilogue inputs fetched with that batch): two batches stay in flight
    // across tile boundaries.
    // (Not for the INT4 three-tile kernels over more than 16 rows: the longer
    // live ranges there cost spills.)
    constexpr bool EARLY = !(Q4 && MT >= 2);
    while (q < total) {
      compute(wA, xA, q);
      if (EARLY && q + 2 < total) load(q + 2, wA, xA);
      finish(q, pA);
      if (!EARLY && q + 2 < total) load(q + 2, wA, xA);
      if (q + 2 < total) epi_fetch(q + 2, pA);
      if (++q >= total) break;
      compute(wB, xB, q);
      if (EARLY && q + 2 < total) load(q + 2, wB, xB);
      finish(q, pB);
      if (!EARLY && q + 2 < total) load(q + 2, wB, xB);
      if (q + 2 < total) epi_fetch(q + 2, pB);
      ++q;
    }
  } else {
    for (; q < total; ++q) {
      if (q > 0) {
        load(q, wA, xA);
        epi_fetch(q, pA);
      }
      compute(wA, xA, q);
      finish(q, pA);
    }
  }
}

// ---------------------------------------------------------------- INT4 kernel for passes of at most 16 rows
// A block (one per CU, 8 waves) owns U units of TU 16-row tiles (unit
// blockIdx.x + i*gridDim.x; a SwiGLU unit pairs a gate tile with an up tile)
// and wave w reduces groups [w*gw, (w+1)*gw) of 128 columns of all of them.
// Every code block (16 bytes per lane, tile and group) and group scale of the
// wave is requested in the prologue, so the block's whole weight share is in
// flight before the first multiply; the activations go through LDS instead
// of registers.  Per window of GPW groups per wave, the block turns its x
// chunks (8 columns of one row) into hi + lo bf16 operands, ordered as the
// code unpacking orders columns; a group's sum over its four k-steps is
// multiplied by the group's scale in float32.
constexpr int kQ4Threads = 512;
constexpr int kQ4Waves = kQ4Threads / kWave;
constexpr int kQ4Rows = 16;                    // rows per launch
constexpr int kQ4RowBlock = 16 * 32 + 16;      // window bytes of one (group, row): 16 chunks, padding
constexpr int kQ4WindowBytes = 128 * 1024;
constexpr int kQ4WindowRows = kQ4WindowBytes / kQ4RowBlock / kQ4Waves;  // GPW * M per window <= this (31)
constexpr int kQ4Chunks = (kQ4Waves * kQ4WindowRows * 16 + kQ4Threads - 1) / kQ4Threads;  // per thread

typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// One k-step's code word (8 columns of the lane's row) as biased bf16 MFMA
// operands 136 + q (bits 0x4300 | (q + 8)): element 2d is column d, element
// 2d + 1 column d + 4.  (The nibble's two's-complement sign bit flipped gives
// q + 8; both that flip and the 0x4300 exponent bits are one XOR after the
// mask, since the mask leaves those bits zero.)
__device__ __forceinline__ bf16x8 q4_operand(uint32_t w) {
  u32x4 v;
  v[0] = (w & 0x000F000Fu) ^ 0x43084308u;
  v[1] = ((w >> 4) & 0x000F000Fu) ^ 0x43084308u;
  v[2] = ((w >> 8) & 0x000F000Fu) ^ 0x43084308u;
  v[3] = ((w >> 12) & 0x000F000Fu) ^ 0x43084308u;
  return __builtin_bit_cast(bf16x8, v);
}

template <int U, int TU, int GW, int GPW, int KIND>
__global__ __launch_bounds__(kQ4Threads) void gemm_q4_lds(GemmArgs a, int n_units, int gw) {
  // GPW: groups per wave per window (GPW * M <= kQ4WindowRows); the windows
  // are a compile-time sequence, so no branch joins paths with different
  // loads in flight (which would force waits for every outstanding load).
  constexpr int F = U * TU, NC = 16 * TU, NWIN = (GW + GPW - 1) / GPW;
  constexpr bool QKV = KIND == EPI_QKV;
  __shared__ __align__(16) unsigned char s_win[kQ4WindowBytes];    // x window, then the cross-wave sums
  __shared__ float yfin[U][kQ4Rows][NC + 1];
  __shared__ float scale[kQ4Rows];
  __shared__ RowDesc s_rows[QKV ? kQ4Rows : 1];
  __shared__ float s_cs[QKV ? kQ4Rows : 1][QKV ? 128 : 1];

  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int M = a.M, K = a.K, G = (K + 127) / 128;
  const int my_g = max(0, min(G - wave * gw, gw));  // groups of this wave
  const int n_chunks = kQ4Waves * GPW * M * 16;      // x chunks per window
  const int chr = (n_chunks + kQ4Threads - 1) / kQ4Threads;  // of them per thread (<= kQ4Chunks)

  // Window wi: chunk c = (slot*M + m)*16 + 4j + kq, slot = wave'*GPW + lgw,
  // holds x[m][128*grp + 32j + 8kq .. +7] of group grp = wave'*gw + wi*GPW + lgw.
  f32x4 xw[kQ4Chunks][2];
  auto load_window = [&](int wi) {
    const __amdgpu_buffer_rsrc_t xr = make_rsrc(a.x, (uint32_t)M * a.ldx * 4u);
#pragma unroll
    for (int i = 0; i < kQ4Chunks; ++i) {
      // (block-uniform: pieces past the window's rows are not requested at all;
      // an out-of-range load still takes its issue slot in the texture unit)
      if (i >= chr) break;
      const int c = tid + i * kQ4Threads, jq = c & 15, r = c >> 4;
      const int m = r % M, slot = r / M, lg = wi * GPW + slot % GPW;
      const int grp = (slot / GPW) * gw + lg;
      const int col = grp * 128 + (jq >> 2) * 32 + (jq & 3) * 8;
      const uint32_t bad = (uint32_t)(c >= n_chunks || lg >= gw || grp >= G || col >= K) << 31;
      const uint32_t off = (((uint32_t)m * a.ldx + col) * 4u) | bad;
      xw[i][0] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(xr, off, 0, 0));
      xw[i][1] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(xr, off + 16u, 0, 0));
    }
  };
  auto store_window = [&]() {
#pragma unroll
    for (int i = 0; i < kQ4Chunks; ++i) {
      const int c = tid + i * kQ4Threads, jq = c & 15, r = c >> 4;
      if (c < n_chunks) {
        // columns 0, 4, 1, 5, 2, 6, 3, 7 (the order of the unpacked codes)
        const f32x2 p0 = {xw[i][0][0], xw[i][1][0]}, p1 = {xw[i][0][1], xw[i][1][1]};
        const f32x2 p2 = {xw[i][0][2], xw[i][1][2]}, p3 = {xw[i][0][3], xw[i][1][3]};
        const bf16x2 h0 = __builtin_convertvector(p0, bf16x2), h1 = __builtin_convertvector(p1, bf16x2);
        const bf16x2 h2 = __builtin_convertvector(p2, bf16x2), h3 = __builtin_convertvector(p3, bf16x2);
        const f32x2 r0 = p0 - __builtin_convertvector(h0, f32x2), r1 = p1 - __builtin_convertvector(h1, f32x2);
        const f32x2 r2 = p2 - __builtin_convertvector(h2, f32x2), r3 = p3 - __builtin_convertvector(h3, f32x2);
        const u32x4 hv = {__builtin_bit_cast(uint32_t, h0), __builtin_bit_cast(uint32_t, h1),
                          __builtin_bit_cast(uint32_t, h2), __builtin_bit_cast(uint32_t, h3)};
        const u32x4 lv = {__builtin_bit_cast(uint32_t, __builtin_convertvector(r0, bf16x2)),
                          __builtin_bit_cast(uint32_t, __builtin_convertvector(r1, bf16x2)),
                          __builtin_bit_cast(uint32_t, __builtin_convertvector(r2, bf16x2)),
                          __builtin_bit_cast(uint32_t, __builtin_convertvector(r3, bf16x2))};
        unsigned char* dst = s_win + r * kQ4RowBlock + jq * 32;
        *(u32x4*)dst = hv;
        *(u32x4*)(dst + 16) = lv;
      }
    }
  };

  // Prologue: the first window's x, the row-scale partials and the QKV
  // tables are requested before the scales and codes (loads complete in
  // order, so the conversions below wait for them alone).
  load_window(0);
  constexpr int RS_ROWS = kQ4Rows / kQ4Waves, RS_P = 4;
  float rs_v[RS_ROWS][RS_P];
  {
    const __amdgpu_buffer_rsrc_t sr = make_rsrc(a.ss_in, a.ss_in ? (uint32_t)a.n_ss * a.ss_ld * 4u : 0u);
#pragma unroll
    for (int r = 0; r < RS_ROWS; ++r) {
      const int m = wave + r * kQ4Waves;
#pragma unroll
      for (int i = 0; i < RS_P; ++i) {
        const int p = lane + i * kWave;
        const uint32_t off = (m < M && p < a.n_ss) ? ((uint32_t)p * a.ss_ld + m) * 4u : kOutOfRange;
        rs_v[r][i] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(sr, off, 0, 0));
      }
    }
  }
  constexpr int CS_E = QKV ? kQ4Rows * 128 / kQ4Threads : 1;
  float cs_v[CS_E];
  RowDesc rd_v{0, 0, 0, 0};
  if constexpr (QKV) {
    const __amdgpu_buffer_rsrc_t cr = make_rsrc(a.rope_cs, (uint32_t)M * a.head_dim * 4u);
#pragma unroll
    for (int e = 0; e < CS_E; ++e) {
      const int i = tid + e * kQ4Threads, m = i / 128, j = i % 128;
      const uint32_t off = j < a.head_dim ? ((uint32_t)m * a.head_dim + j) * 4u : kOutOfRange;
      cs_v[e] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(cr, off, 0, 0));
    }
    const __amdgpu_buffer_rsrc_t rr = make_rsrc(a.rows, (uint32_t)M * (uint32_t)sizeof(RowDesc));
    rd_v = __builtin_bit_cast(RowDesc, __builtin_amdgcn_raw_buffer_load_b128(
                                           rr, tid < kQ4Rows ? (uint32_t)tid * (uint32_t)sizeof(RowDesc) : kOutOfRange,
                                           0, 0));
  }
  // Residual GEMMs (one 16-column unit): the old h and the next RMSNorm gain of
  // this thread's output element.
  constexpr bool PRE = KIND == EPI_RESID && U == 1;
  float pre_h = 0.f;
  uint32_t pre_g = 0u;
  if constexpr (PRE) {
    const int m = tid / 16, n = blockIdx.x * 16 + tid % 16;
    const uint32_t bad = (uint32_t)(m >= M || n >= a.n_rows) << 31;
    const __amdgpu_buffer_rsrc_t hr = make_rsrc(a.out, (uint32_t)M * a.ldo * 4u);
    const __amdgpu_buffer_rsrc_t gr = make_rsrc(a.gain_out, (uint32_t)a.n_rows * 2u);
    pre_h = __builtin_bit_cast(
        float, __builtin_amdgcn_raw_buffer_load_b32(hr, (((uint32_t)m * a.ldo + n) * 4u) | bad, 0, 0));
    pre_g = __builtin_amdgcn_raw_buffer_load_b16(gr, ((uint32_t)n * 2u) | bad, 0, 0);
  }
  // The wave's code blocks and scales, group-major.  All scales come first
  // (a group's products wait for its scales, and loads complete in issue
  // order); the codes of D groups are requested here and each later group's
  // D groups ahead of its products.  A shallow depth keeps the prologue's
  // vector-memory issue short, so it does not hold up the x conversion:
  // deeper requests (up to 8 groups, about 64 KB per CU in flight) measured
  // 2% slower over a 7B verify, and one group is too few below six.
  constexpr int D = F >= 6 ? 1 : 2;
  u32x4 cw[F][GW];
  uint32_t sw[F][GW];
  __amdgpu_buffer_rsrc_t crs[F], srs[F];
#pragma unroll
  for (int f = 0; f < F; ++f) {
    const int unit = blockIdx.x + (f / TU) * gridDim.x;
    int seg, n;
    bool ok;
    tile_segment(a, KIND, unit, NC, f % TU, seg, n, ok);
    ok = ok && unit < n_units;
    crs[f] = make_rsrc((const char*)a.w[seg] + (size_t)(n / 16) * G * 1024, ok ? (uint32_t)G * 1024u : 0u);
    srs[f] = make_rsrc(a.wscale[seg] + (size_t)(n / 16) * G * 16, ok ? (uint32_t)G * 32u : 0u);
  }
#pragma unroll
  for (int lg = 0; lg < GW; ++lg) {
    const uint32_t bad = (uint32_t)(lg >= my_g) << 31;
#pragma unroll
    for (int f = 0; f < F; ++f)
      sw[f][lg] = __builtin_amdgcn_raw_buffer_load_b16(
          srs[f], ((uint32_t)(wave * gw + lg) * 32u + (lane & 15) * 2u) | bad, 0, 0);
  }
  __builtin_amdgcn_sched_barrier(0);
  auto issue_codes = [&](int lg) {
    const uint32_t bad = (uint32_t)(lg >= my_g) << 31;
#pragma unroll
    for (int f = 0; f < F; ++f)
      cw[f][lg] = __builtin_amdgcn_raw_buffer_load_b128(
          crs[f], ((uint32_t)(wave * gw + lg) * 1024u + lane * 16u) | bad, 0, kNonTemporal);
    __builtin_amdgcn_sched_barrier(0);
  };
#pragma unroll
  for (int lg = 0; lg < D && lg < GW; ++lg) issue_codes(lg);

  {
    float t[RS_ROWS];
#pragma unroll
    for (int r = 0; r < RS_ROWS; ++r) {
      const int m = wave + r * kQ4Waves;
      t[r] = 0.f;
#pragma unroll
      for (int i = 0; i < RS_P; ++i) t[r] += rs_v[r][i];
      if (a.ss_in && m < M)
        for (int p = lane + RS_P * kWave; p < a.n_ss; p += kWave) t[r] += a.ss_in[(size_t)p * a.ss_ld + m];
    }
    wave_sum_n(t);
#pragma unroll
    for (int r = 0; r < RS_ROWS; ++r) {
      const int m = wave + r * kQ4Waves;
      if (lane == 0) scale[m] = (a.ss_in && m < M) ? 1.0f / sqrtf(t[r] / (float)K + a.eps) : 1.0f;
    }
  }
  if constexpr (QKV) {
#pragma unroll
    for (int e = 0; e < CS_E; ++e) {
      const int i = tid + e * kQ4Threads;
      s_cs[i / 128][i % 128] = cs_v[e];
    }
    if (tid < kQ4Rows) s_rows[tid] = rd_v;
  }
  store_window();
  __syncthreads();

  floatx4 acc[F];
#pragma unroll
  for (int f = 0; f < F; ++f) acc[f] = floatx4{0.f, 0.f, 0.f, 0.f};
  const int kq = lane >> 4;
  // STACK (at most 8 rows, GPW > 1 implies M <= 7): the hi parts of the rows
  // go to A rows 0..7 and the lo parts to rows 8..15, so one product per
  // k-step covers both; output rows m and m + 8 are added after the
  // cross-wave sums.  Otherwise hi and lo are two products.
  constexpr bool STACK = GPW > 1;
  // The +136 bias of the code operands is cancelled by the product of the same
  // x with -136 (bf16 0xC308), shared by the block's tiles and added to each
  // tile's group sum before the scale.
  const bf16x8 m136 = __builtin_bit_cast(bf16x8, u32x4{0xC308C308u, 0xC308C308u, 0xC308C308u, 0xC308C308u});
  auto compute_group = [&](int lg) {
    const int slot = wave * GPW + lg % GPW;
    floatx4 pb = floatx4{0.f, 0.f, 0.f, 0.f};
    if constexpr (STACK) {
      const unsigned char* xa =
          s_win + (slot * M + min(lane & 7, M - 1)) * kQ4RowBlock + kq * 32 + ((lane >> 3) & 1) * 16;
      floatx4 p[F];
#pragma unroll
      for (int f = 0; f < F; ++f) p[f] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const bf16x8 xv = *(const bf16x8*)(xa + j * 128);
        pb = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xv, m136, pb, 0, 0, 0);
#pragma unroll
        for (int f = 0; f < F; ++f)
          p[f] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xv, q4_operand(cw[f][lg][j]), p[f], 0, 0, 0);
      }
#pragma unroll
      for (int f = 0; f < F; ++f) {
        const float sc = bf16_bits_to_f32((uint16_t)sw[f][lg]);
#pragma unroll
        for (int r = 0; r < 4; ++r) acc[f][r] = fmaf(sc, p[f][r] + pb[r], acc[f][r]);
      }
    } else {
      const unsigned char* xb = s_win + (slot * M + min(lane & 15, M - 1)) * kQ4RowBlock + kq * 32;
      floatx4 ph[F], pl[F];
#pragma unroll
      for (int f = 0; f < F; ++f) {
        ph[f] = floatx4{0.f, 0.f, 0.f, 0.f};
        pl[f] = floatx4{0.f, 0.f, 0.f, 0.f};
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const bf16x8 hi = *(const bf16x8*)(xb + j * 128), lo = *(const bf16x8*)(xb + j * 128 + 16);
        pb = __builtin_amdgcn_mfma_f32_16x16x32_bf16(hi, m136, pb, 0, 0, 0);
        pb = __builtin_amdgcn_mfma_f32_16x16x32_bf16(lo, m136, pb, 0, 0, 0);
#pragma unroll
        for (int f = 0; f < F; ++f) {
          const bf16x8 b = q4_operand(cw[f][lg][j]);
          ph[f] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(hi, b, ph[f], 0, 0, 0);
          pl[f] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(lo, b, pl[f], 0, 0, 0);
        }
      }
#pragma unroll
      for (int f = 0; f < F; ++f) {
        const float sc = bf16_bits_to_f32((uint16_t)sw[f][lg]);
#pragma unroll
        for (int r = 0; r < 4; ++r) acc[f][r] = fmaf(sc, (ph[f][r] + pl[f][r]) + pb[r], acc[f][r]);
      }
    }
  };
  // (blocks of one tile have the registers to fetch the next window's x while
  // the current one is multiplied; a window past the wave's groups loads
  // nothing and converts zeros)
  constexpr bool PREFETCH = F == 1;
#pragma unroll
  for (int w = 0; w < NWIN; ++w) {
    if (w > 0) {
      __syncthreads();
      if constexpr (!PREFETCH) load_window(w);
      store_window();
      __syncthreads();
    }
    if constexpr (PREFETCH) {
      if (w + 1 < NWIN) load_window(w + 1);
    }
#pragma unroll
    for (int i = 0; i < GPW; ++i) {
      const int lg = w * GPW + i;
      if (lg + D < GW) issue_codes(lg + D);
      if (lg < GW && lg < my_g) compute_group(lg);
    }
  }

  // Cross-wave sums in fixed wave order: red[f][wave][lane][r] -> yfin.
  __syncthreads();
  float* red = (float*)s_win;
#pragma unroll
  for (int f = 0; f < F; ++f) *(floatx4*)&red[((f * kQ4Waves + wave) * kWave + lane) * 4] = acc[f];
  __syncthreads();
  for (int i = tid; i < F * kWave * 4; i += kQ4Threads) {
    const int f = i / (kWave * 4), l = (i / 4) % kWave, r = i % 4;
    float s = 0.f;
#pragma unroll
    for (int w = 0; w < kQ4Waves; ++w) s += red[((f * kQ4Waves + w) * kWave + l) * 4 + r];
    yfin[f / TU][4 * (l >> 4) + r][(f % TU) * 16 + (l & 15)] = s;
  }
  __syncthreads();
  if constexpr (STACK) {  // rows m (hi parts) + m + 8 (lo parts)
    for (int i = tid; i < U * 8 * NC; i += kQ4Threads) {
      const int u = i / (8 * NC), m = (i / NC) % 8, c = i % NC;
      yfin[u][m][c] += yfin[u][m + 8][c];
    }
    __syncthreads();
  }
  if constexpr (PRE) {  // h += y; xg = h * gain; sum of squares of the unit's new h
    const int m = tid / 16, c = tid % 16, n = blockIdx.x * 16 + c;
    if (m < M) {
      float hv = 0.f;
      if (n < a.n_rows) {
        hv = pre_h + yfin[0][m][c];
        a.out[(size_t)m * a.ldo + n] = hv;
        a.xg_out[(size_t)m * a.ldo + n] = hv * bf16_bits_to_f32((uint16_t)pre_g);
      }
      yfin[0][m][c] = hv;
    }
    __syncthreads();
    if (tid < M) {
      float t = 0.f;
      for (int c2 = 0; c2 < 16; ++c2) t += yfin[0][tid][c2] * yfin[0][tid][c2];
      a.ss_out[(size_t)blockIdx.x * a.ss_ld + tid] = t;
    }
    return;
  }
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int unit = blockIdx.x + u * gridDim.x;
    if (unit >= n_units) break;  // (block-uniform)
    if constexpr (QKV) qkv_epilogue<NC, kQ4Threads>(a, unit, yfin[u], scale, s_rows, s_cs);
    else epilogue<NC, KIND, kQ4Threads>(a, unit, yfin[u], scale);
  }
}

// ---------------------------------------------------------------- wide-M MFMA kernel (bf16 weights)
// Passes of more than 64 rows (the verify blocks of many sequences, prefill
// and catch-up chunks) in launches of up to 128 rows.  A block covers NC =
// 64*T weight rows and a range of k-steps with G k-groups of 4 waves: group g
// takes every G-th k-step of the range and wave w of a group owns tiles
// wT..wT+T-1.  Each k-step's x slab (MP rows x 32 columns) is converted once
// by its group into hi + lo bf16 A fragments in LDS (two buffers per group)
// and shared by the group's four waves, so activation traffic per weight
// byte falls by the 4T tiles sharing it.  Grids are about one block per CU,
// so the G groups are what keeps more than one wave per SIMD busy; each wave
// also keeps x slabs XR = 4 k-steps ahead and weight fragments D k-steps ahead
// in register rings.  The groups' sums are added in group order in LDS; the
// epilogues (store, SwiGLU, QKV with RoPE) then read the accumulators in
// place.  Residual GEMMs (O, down: few row tiles) split K over the grid and
// write partial sums, which resid_reduce_kernel adds in a fixed order; Q|K|V
// and gate|up do the same with three tiles per wave, their partial sums added
// by qkv_reduce_kernel (with RoPE, the query store and the KV append) and
// swiglu_reduce_kernel.  (With three tiles per wave the x ring holds two slabs,
// and the groups' sums go through the slab buffers one tile at a time.)
constexpr int kWideGroups = 2;
constexpr int kWideThreads = 256 * kWideGroups;
constexpr int kWideRows = 128;  // rows per launch of the wide kernel
constexpr int kWideCols = 128;  // columns per block of the split-K reduction (and per ss partial)
constexpr int kWideMaxSs = 64;  // ss partials a wide launch sums (one per lane)
constexpr int kWideSplitMax = 12;  // K splits of a wide launch's partial sums

template <int MT, int T, int KIND>
__global__ __launch_bounds__(kWideThreads) void gemm_bf16_wide(GemmArgs a, int ks_per_split, int n_split) {
  constexpr int G = kWideGroups;
  constexpr int MP = 16 * MT, NC = 64 * T;
  constexpr int D = T == 1 ? 8 : 4;                  // weight k-steps in flight per wave
  constexpr int XR = T >= 3 ? 2 : 4;                 // x slabs in flight per group (registers: T >= 3)
  constexpr int PJ = (MP * 4 + 255) / 256;           // 32-byte x pieces per thread per slab
  constexpr int MTP = PJ * 256 / 64;                 // m tiles the pieces cover (>= MT; extra rows read zeros)
  constexpr bool QKV = KIND == EPI_QKV, SCALE = KIND != EPI_RESID;
  constexpr int RSR = MP / (4 * G);                  // row-scale rows per wave
  constexpr int CSL = QKV ? MP / 16 : 1;             // 16-byte cos/sin pieces per lane (8 columns x MP rows x 2)
  static_assert(KIND != EPI_SWIGLU || T == 2, "SwiGLU pairs one gate and one up tile per wave");
  static_assert(!QKV || T == 1, "the QKV epilogue tables cover one tile per wave");
  static_assert(D % XR == 0, "the unrolled step loop indexes both rings statically");
  static_assert(MP % (4 * G) == 0, "row-scale rows split evenly over the waves");
  static_assert(4 * MT <= G * 2 * MTP * 2, "one tile's group sums fit in the slab buffers");
  __shared__ u32x4 s_a[G][2][MTP][2][kWave];  // [group][buffer][m tile][hi, lo][lane]
  __shared__ float scale[MP];
  __shared__ f32x4 s_cs[QKV ? 4 : 1][QKV ? MP : 1][4];  // per tile wave, per row: cos of its 8 dims, then sin
  __shared__ RowDesc s_rows[QKV ? MP : 1];

  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int grp = wave >> 2, wl = wave & 3, gtid = tid & 255;  // k-group, wave in group, thread in group
  const int K = a.K, KS = (K + 31) / 32;
  const int split = (int)blockIdx.x % n_split, blk = (int)blockIdx.x / n_split;
  const int ks_begin = split * ks_per_split;
  const int ks_end = min(KS, ks_begin + ks_per_split);
  const int n_k = ks_end - ks_begin;
  const int n_steps = (n_k + G - 1) / G;  // steps of every group (a group's last ones may be past the range)

  // Weight tiles of this wave (SwiGLU: gate tile w and the up tile of the same columns).
  __amdgpu_buffer_rsrc_t wr[T];
#pragma unroll
  for (int t = 0; t < T; ++t) {
    const int lt = KIND == EPI_SWIGLU ? (t == 0 ? wl : 4 + wl) : wl * T + t;
    bool ok;
    const uint16_t* base = weight_tile(a, KIND, blk, NC, lt, KS, ok);
    wr[t] = make_rsrc(base, ok ? (uint32_t)KS * 1024u : 0u);
  }
  const __amdgpu_buffer_rsrc_t xr = make_rsrc(a.x, (uint32_t)a.M * a.ldx * 4u);

  floatx4 acc[T][MT];
#pragma unroll
  for (int t = 0; t < T; ++t)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) acc[t][mt] = floatx4{0.f, 0.f, 0.f, 0.f};
  u32x4 wv[D][T];
  f32x4 xv[XR][PJ][2];

  // Step j of group g is k-step ks_begin + j*G + g.
  auto load_w = [&](int j, u32x4 (&w)[T]) {
    const int i = j * G + grp;
    const uint32_t bad = (uint32_t)(i >= n_k) << 31;
    const uint32_t off = ((uint32_t)(ks_begin + i) * 1024u + lane * 16u) | bad;
#pragma unroll
    for (int t = 0; t < T; ++t) w[t] = __builtin_amdgcn_raw_buffer_load_b128(wr[t], off, 0, kNonTemporal);
  };
  // Piece p = lane p%64 of the A fragment of m tile p/64: 8 consecutive floats
  // of row 16*(p/64) + p%16 at column 8*(p%64/16) of the k-step (a wave moves
  // whole fragments: contiguous LDS stores, 16 rows x 128 bytes per load).
  auto load_x = [&](int j, f32x4 (&xs)[PJ][2]) {
    const int i = j * G + grp;
    const uint32_t bad = (uint32_t)(i >= n_k) << 31;
#pragma unroll
    for (int q = 0; q < PJ; ++q) {
      const int p = gtid + q * 256, m = (p >> 6) * 16 + (p & 15), k = (ks_begin + i) * 32 + ((p >> 4) & 3) * 8;
      const uint32_t off = (((uint32_t)m * a.ldx + k) * 4u) | bad | ((uint32_t)(k >= K) << 31);
      xs[q][0] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(xr, off, 0, 0));
      xs[q][1] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(xr, off + 16u, 0, 0));
    }
  };
  // A fragment lane 16*(k/8) + m%16 holds row m, columns 8*(k/8)..+7
  auto store_x = [&](int buf, const f32x4 (&xs)[PJ][2]) {
#pragma unroll
    for (int q = 0; q < PJ; ++q) {
      const int p = gtid + q * 256;
      const int mt = p >> 6, ln = p & 63;
      bf16x8 hi, lo;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float v = xs[q][e >> 2][e & 3];
        const __bf16 h = (__bf16)v;
        hi[e] = h;
        lo[e] = (__bf16)(v - (float)h);
      }
      s_a[grp][buf][mt][0][ln] = __builtin_bit_cast(u32x4, hi);
      s_a[grp][buf][mt][1][ln] = __builtin_bit_cast(u32x4, lo);
    }
  };
  // All fragment reads first, then the hi products of every tile, then the lo
  // ones (a product's accumulator is not the previous product's).
  auto compute = [&](int buf, const u32x4 (&w)[T]) {
    bf16x8 av[MT][2];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      av[mt][0] = __builtin_bit_cast(bf16x8, s_a[grp][buf][mt][0][lane]);
      av[mt][1] = __builtin_bit_cast(bf16x8, s_a[grp][buf][mt][1][lane]);
    }
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int t = 0; t < T; ++t)
          acc[t][mt] =
              __builtin_amdgcn_mfma_f32_16x16x32_bf16(av[mt][h], __builtin_bit_cast(bf16x8, w[t]), acc[t][mt], 0, 0, 0);
    __builtin_amdgcn_sched_group_barrier(0x100, 2 * MT, 0);     // LDS reads
    __builtin_amdgcn_sched_group_barrier(0x008, 2 * MT * T, 0);  // then MFMAs
  };

  // QKV epilogue geometry of this wave's tile: rotation dims 8*tq + e (e < 8)
  // of its head for Q and K columns.
  const int hd = a.head_dim, half = hd >> 1;
  const int nq = a.n_seg[0], nqk = nq + a.n_seg[1];
  const int n0 = blk * NC + wl * 16;  // (QKV: T == 1)
  const int r0 = n0 >= nqk ? n0 - nqk : (n0 >= nq ? n0 - nq : n0);
  const int tq = (r0 % hd) >> 4;

  // Prologue.  Loads in order: the epilogue's small operands (row-scale
  // partial sums; QKV: cos/sin of the tile's 8 dims and the row descriptors,
  // fetched by group 0), XR x slabs, D weight k-steps.  Loads complete in
  // order, so storing the small operands waits for them alone.
  float rsv[SCALE ? RSR : 1];
  if constexpr (SCALE) {
    const __amdgpu_buffer_rsrc_t sr = make_rsrc(a.ss_in, a.ss_in ? (uint32_t)a.n_ss * a.ss_ld * 4u : 0u);
#pragma unroll
    for (int i = 0; i < RSR; ++i) {
      const int m = wave + 4 * G * i;
      const uint32_t off = ((uint32_t)lane * a.ss_ld + m) * 4u | ((uint32_t)(m >= a.M || lane >= a.n_ss) << 31);
      rsv[i] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(sr, off, 0, 0));
    }
  }
  f32x4 csv[CSL];
  u32x4 rdv = u32x4{0u, 0u, 0u, 0u};
  if constexpr (QKV) {
    const __amdgpu_buffer_rsrc_t cr = make_rsrc(a.rope_cs, (uint32_t)a.M * hd * 4u);
#pragma unroll
    for (int q = 0; q < CSL; ++q) {  // piece v = lane + 64q: row v/4, (cos, sin) = (v/2)%2, half (v%2)
      const int v = lane + 64 * q, m = v >> 2, sn = (v >> 1) & 1, hf = v & 1;
      const uint32_t off = ((uint32_t)m * hd + sn * half + 8 * tq + 4 * hf) * 4u |
                           ((uint32_t)(n0 >= nqk || grp != 0) << 31);
      csv[q] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(cr, off, 0, 0));
    }
    const __amdgpu_buffer_rsrc_t rr = make_rsrc(a.rows, (uint32_t)a.M * (uint32_t)sizeof(RowDesc));
    rdv = __builtin_amdgcn_raw_buffer_load_b128(
        rr, (uint32_t)tid * (uint32_t)sizeof(RowDesc) | ((uint32_t)(tid >= MP) << 31), 0, 0);
  }
#pragma unroll
  for (int r = 0; r < XR; ++r) load_x(r, xv[r]);
#pragma unroll
  for (int u = 0; u < D; ++u) load_w(u, wv[u]);
  if constexpr (SCALE) {
    // s_m = 1/sqrt(sum_p ss[p][m] / K + eps): partial p in lane p, fixed shuffle tree
    wave_sum_n(rsv);  // (n_ss <= 64: checked by the launcher)
#pragma unroll
    for (int i = 0; i < RSR; ++i) {
      const int m = wave + 4 * G * i;
      if (lane == 0) scale[m] = (a.ss_in && m < a.M) ? 1.0f / sqrtf(rsv[i] / (float)a.K + a.eps) : 1.0f;
    }
  }
  if constexpr (QKV) {
    if (grp == 0) {
#pragma unroll
      for (int q = 0; q < CSL; ++q) {
        const int v = lane + 64 * q;
        s_cs[wl][v >> 2][v & 3] = csv[q];
      }
    }
    if (tid < MP) s_rows[tid] = __builtin_bit_cast(RowDesc, rdv);
  }
  store_x(0, xv[0]);
  load_x(XR, xv[0]);
  __syncthreads();

  // Step j: multiply the group's slab j (LDS buffer j%2) by weight slot j%D,
  // refill the slot with step j+D, move slab j+1 (register slot (j+1)%XR) into
  // the other buffer and fetch slab j+1+XR into its slot.  The step count is
  // rounded up to a multiple of D: steps past the range multiply zeros (their
  // loads are out of range), which keeps the loop free of early exits (an exit
  // edge into the loop makes the compiler wait for every load in flight at the
  // top of the loop).  (Scheduling barriers keep each step's conversions after
  // its multiplies: hoisted above them, the conversions of a later slab would
  // wait for the weight loads issued after it.)
  for (int j0 = 0; j0 < n_steps; j0 += D) {
#pragma unroll
    for (int u = 0; u < D; ++u) {
      const int j = j0 + u;
      __builtin_amdgcn_sched_barrier(0);
      compute(u & 1, wv[u]);
      __builtin_amdgcn_sched_barrier(0);
      load_w(j + D, wv[u]);
      store_x((u + 1) & 1, xv[(u + 1) % XR]);
      load_x(j + 1 + XR, xv[(u + 1) % XR]);
      __syncthreads();
    }
  }

  // Group sums: groups 1.. park theirs in the (now free) slab buffers, group 0
  // adds them in group order and runs the epilogue.
  if constexpr (G > 1 && (G - 1) * 4 * T * MT > G * 2 * MTP * 2) {
    // (too many for the slab buffers at once: one tile at a time)
    static_assert(G == 2, "tile-at-a-time group sums: two groups");
    floatx4* park = reinterpret_cast<floatx4*>(&s_a[0][0][0][0][0]);
#pragma unroll
    for (int t = 0; t < T; ++t) {
      if (grp > 0) {
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) park[(wl * MT + mt) * kWave + lane] = acc[t][mt];
      }
      __syncthreads();
      if (grp == 0) {
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) acc[t][mt] += park[(wl * MT + mt) * kWave + lane];
      }
      __syncthreads();
    }
    if (grp > 0) return;
  } else if constexpr (G > 1) {
    floatx4* park = reinterpret_cast<floatx4*>(&s_a[0][0][0][0][0]);
    if (grp > 0) {
#pragma unroll
      for (int t = 0; t < T; ++t)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) park[(((grp - 1) * 4 + wl) * T * MT + t * MT + mt) * kWave + lane] = acc[t][mt];
    }
    __syncthreads();
    if (grp > 0) return;
#pragma unroll
    for (int g = 1; g < G; ++g)
#pragma unroll
      for (int t = 0; t < T; ++t)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) acc[t][mt] += park[(((g - 1) * 4 + wl) * T * MT + t * MT + mt) * kWave + lane];
  }

  // Epilogue (group 0).  acc[t][mt][r] is row mt*16 + 4*(lane/16) + r, column lane%16 of tile t.
  const int M = a.M, cl = lane & 15, rg = lane >> 4;
  if constexpr (KIND == EPI_RESID) {
    // Each 16 x 16 accumulator tile goes through a wave-private LDS square
    // (inside the wave's own part of the group-sum area, which it has read):
    // lane l then holds 4 consecutive columns of row l/4 and stores them as
    // one 16-byte write, a quarter of the store instructions of writing each
    // lane's 4 rows of one column.  (LDS operations of a wave complete in
    // order; the wave barriers keep the compiler from reordering them.)
    float* yp = a.ypart + (size_t)split * M * a.n_rows;
    constexpr int PSTRIDE = ((G - 1) * 4 * T * MT > G * 2 * MTP * 2 ? MT : T * MT) * 256;  // floats per wave
    float* sq = reinterpret_cast<float*>(&s_a[0][0][0][0][0]) + (size_t)wl * PSTRIDE;  // [16][17]
    const int rr = lane >> 2, c4 = 4 * (lane & 3);
#pragma unroll
    for (int t = 0; t < T; ++t) {
      const int n0 = blk * NC + (wl * T + t) * 16;
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
#pragma unroll
        for (int r = 0; r < 4; ++r) sq[(4 * rg + r) * 17 + cl] = acc[t][mt][r];
        __builtin_amdgcn_wave_barrier();
        const f32x4 v = f32x4{sq[rr * 17 + c4], sq[rr * 17 + c4 + 1], sq[rr * 17 + c4 + 2], sq[rr * 17 + c4 + 3]};
        __builtin_amdgcn_wave_barrier();
        const int m = mt * 16 + rr;
        if (m < M && n0 + c4 < a.n_rows) *(f32x4*)(yp + (size_t)m * a.n_rows + n0 + c4) = v;
      }
    }
  } else if constexpr (KIND == EPI_STORE) {
#pragma unroll
    for (int t = 0; t < T; ++t) {
      const int n = blk * NC + (wl * T + t) * 16 + cl;
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int m = mt * 16 + 4 * rg + r;
          if (m < M && n < a.n_rows) a.out[(size_t)m * a.ldo + n] = acc[t][mt][r] * scale[m];
        }
    }
  } else if constexpr (KIND == EPI_SWIGLU) {
    const int f = blk * (NC / 2) + wl * 16 + cl;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = mt * 16 + 4 * rg + r;
        if (m < M && f < a.n_rows)
          a.out[(size_t)m * a.ldo + f] = silu_f(acc[0][mt][r] * scale[m]) * (acc[1][mt][r] * scale[m]);
      }
  } else {  // EPI_QKV: the RoPE partner of column c is column c ^ 8 of the same tile, i.e. lane ^ 8
    const int H = a.n_heads, cap = a.kv.capacity;
    const int n = n0 + cl;
    const bool is_q = n < nq, is_v = n >= nqk;
    const int head = r0 / hd, w = r0 % hd + cl, ec = cl, e = cl & 7;
    const int j = 8 * tq + e, d = ec < 8 ? j : half + j;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = mt * 16 + 4 * rg + r;
        const float x = acc[0][mt][r] * scale[m];
        const float y = __shfl_xor(x, 8, kWave);
        if (m >= M || n >= a.n_rows) continue;
        const RowDesc rd = s_rows[m];
        if (is_v) {
          if (rd.valid) {
            uint16_t* kvb = k_block<uint16_t>(a.kv, a.layer, rd.b, head);
            Storage<uint16_t>::store(kvb + KvIndex<uint16_t>::v(rd.pos, w, hd, cap), x);
          }
          continue;
        }
        const f32x4 c4 = s_cs[wl][m][e >> 2], s4 = s_cs[wl][m][2 + (e >> 2)];
        const float cs = c4[e & 3], sn = s4[e & 3];
        const float out = ec < 8 ? x * cs - y * sn : x * cs + y * sn;
        if (is_q) {
          a.qr[((size_t)m * H + head) * hd + d] = out;
        } else if (rd.valid) {
          uint16_t* kvb = k_block<uint16_t>(a.kv, a.layer, rd.b, head);
          Storage<uint16_t>::store(kvb + KvIndex<uint16_t>::k(rd.pos, d, hd, cap), out);
        }
      }
  }
}

// Split-K partial sums of 4 columns of one row, added in split order; every
// split's load is issued before the first add (the split index is clamped, so
// loads past n_split re-read the last split and are not added).
template <int NS>
__device__ __forceinline__ f32x4 sum_splits_n(const float* yp, size_t split_stride, int n_split) {
  f32x4 v[NS];
#pragma unroll
  for (int s = 0; s < NS; ++s) v[s] = *(const f32x4*)(yp + (size_t)min(s, n_split - 1) * split_stride);
  f32x4 y = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int s = 0; s < NS; ++s)
    if (s < n_split) y += v[s];
  return y;
}
__device__ __forceinline__ f32x4 sum_splits(const float* yp, size_t split_stride, int n_split) {
  if (n_split <= 4) return sum_splits_n<4>(yp, split_stride, n_split);  // (block-uniform)
  if (n_split <= 8) return sum_splits_n<8>(yp, split_stride, n_split);
  return sum_splits_n<kWideSplitMax>(yp, split_stride, n_split);
}

// RMSNorm scales of rows m0 .. m0+7 into s_scale: the block loads every
// partial sum of squares at once (two per thread), then thread r < 8 adds its
// row's in partial order.
__device__ __forceinline__ void row_scales8(const GemmArgs& a, int m0, float* s_scale, float (*s_ss)[kWideMaxSs]) {
  const int tid = threadIdx.x;
  float v[2];
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    const int i = tid + 256 * k, r = i / kWideMaxSs, p = i % kWideMaxSs, m = m0 + r;
    v[k] = a.ss_in && p < a.n_ss && m < a.M ? a.ss_in[(size_t)p * a.ss_ld + m] : 0.f;
  }
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    const int i = tid + 256 * k;
    s_ss[i / kWideMaxSs][i % kWideMaxSs] = v[k];
  }
  __syncthreads();
  if (tid < 8) {
    float ss = 0.f;
    for (int p = 0; p < a.n_ss; ++p) ss += s_ss[tid][p];
    s_scale[tid] = a.ss_in ? 1.0f / sqrtf(ss / (float)a.K + a.eps) : 1.0f;
  }
  __syncthreads();
}
static_assert(8 * kWideMaxSs == 512, "row_scales8: two partials per thread of a 256-thread block");

// Sum of the split-K partials of a residual GEMM in split order, residual
// add, next RMSNorm input and its sums of squares.  Block = 128 columns x 8
// rows; thread = 4 columns of one row; ss partial p = column block p.
__global__ __launch_bounds__(256) void resid_reduce_kernel(GemmArgs a, int n_split) {
  const int tid = threadIdx.x, m = (int)blockIdx.y * 8 + (tid >> 5);
  const int n = (int)blockIdx.x * kWideCols + 4 * (tid & 31);
  const int M = a.M;
  float t = 0.f;
  if (m < M && n < a.n_rows) {
    const f32x4 y = sum_splits(a.ypart + (size_t)m * a.n_rows + n, (size_t)M * a.n_rows, n_split);
    float* hp = a.out + (size_t)m * a.ldo + n;
    const f32x4 h = *(const f32x4*)hp + y;
    *(f32x4*)hp = h;
    const uint16_t* g = (const uint16_t*)a.gain_out + n;
    *(f32x4*)(a.xg_out + (size_t)m * a.ldo + n) =
        f32x4{h[0] * bf16_bits_to_f32(g[0]), h[1] * bf16_bits_to_f32(g[1]), h[2] * bf16_bits_to_f32(g[2]),
              h[3] * bf16_bits_to_f32(g[3])};
    t = h[0] * h[0] + h[1] * h[1] + h[2] * h[2] + h[3] * h[3];
  }
#pragma unroll
  for (int o = 16; o > 0; o >>= 1) t += __shfl_xor(t, o, kWave);
  if ((tid & 31) == 0 && m < M) a.ss_out[(size_t)blockIdx.x * a.ss_ld + m] = t;
}

// Sum of the split-K partial sums of a wide pass's gate and up projections
// (rows [0, F) and [F, 2F) of the partials) in split order, times the row's
// RMSNorm scale, then SwiGLU.  Block = 128 columns x 8 rows; thread = 4 columns of one row.
__global__ __launch_bounds__(256) void swiglu_reduce_kernel(GemmArgs a, int n_split) {
  __shared__ float s_scale[8];
  __shared__ float s_ss[8][kWideMaxSs];
  const int tid = threadIdx.x, m = (int)blockIdx.y * 8 + (tid >> 5);
  const int f = (int)blockIdx.x * kWideCols + 4 * (tid & 31);
  const int M = a.M, F = a.n_rows, W = 2 * F;
  row_scales8(a, (int)blockIdx.y * 8, s_scale, s_ss);
  if (m >= M || f >= F) return;
  const float* yp = a.ypart + (size_t)m * W;
  const f32x4 gs = sum_splits(yp + f, (size_t)M * W, n_split), us = sum_splits(yp + F + f, (size_t)M * W, n_split);
  const float sc = s_scale[tid >> 5];
  f32x4 o;
#pragma unroll
  for (int e = 0; e < 4; ++e) o[e] = silu_f(gs[e] * sc) * (us[e] * sc);
  *(f32x4*)(a.out + (size_t)m * a.ldo + f) = o;
}

// Sum of the split-K partial sums of a wide pass's Q|K|V projections in split
// order, times the row's RMSNorm scale, then RoPE on the Q and K columns and
// the stores: rotated queries to qr, rotated keys and the values appended to
// the KV cache (valid rows).  Q and K columns come in the packed RoPE order:
// column c of a head's 16-column tile tq is dim 8tq + c for c < 8, hd/2 + 8tq
// + c - 8 otherwise, so each column's rotation partner (c ^ 8) is 8 columns
// away, in the lane ^ 2 of the row's 32 threads.  Block = 128 columns x 8
// rows; thread = 4 columns of one row.
__global__ __launch_bounds__(256) void qkv_reduce_kernel(GemmArgs a, int n_split) {
  __shared__ float s_scale[8];
  __shared__ float s_ss[8][kWideMaxSs];
  const int tid = threadIdx.x, m = (int)blockIdx.y * 8 + (tid >> 5);
  const int n = (int)blockIdx.x * kWideCols + 4 * (tid & 31);
  const int M = a.M;
  row_scales8(a, (int)blockIdx.y * 8, s_scale, s_ss);
  const bool live = m < M && n < a.n_rows;
  f32x4 y = f32x4{0.f, 0.f, 0.f, 0.f};
  if (live) y = sum_splits(a.ypart + (size_t)m * a.n_rows + n, (size_t)M * a.n_rows, n_split);
  const float sc = s_scale[tid >> 5];
  f32x4 z;  // (every lane takes part in the shuffles)
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    y[e] *= sc;
    z[e] = __shfl_xor(y[e], 2, kWave);
  }
  if (!live) return;
  const int H = a.n_heads, hd = a.head_dim, half = hd >> 1, cap = a.kv.capacity;
  const int nq = a.n_seg[0], nqk = nq + a.n_seg[1];
  const RowDesc rd = a.rows[m];
  if (n >= nqk) {  // values: natural order
    if (!rd.valid) return;
    const int r = n - nqk, head = r / hd, w = r % hd;
    uint16_t* kvb = k_block<uint16_t>(a.kv, a.layer, rd.b, head);
#pragma unroll
    for (int e = 0; e < 4; ++e) Storage<uint16_t>::store(kvb + KvIndex<uint16_t>::v(rd.pos, w + e, hd, cap), y[e]);
    return;
  }
  const bool is_q = n < nq;
  const int r = n - (is_q ? 0 : nq), head = r / hd, w = r % hd, tq = w >> 4;
  const float* cs = a.rope_cs + (size_t)m * hd;
  uint16_t* kvb = is_q || !rd.valid ? nullptr : k_block<uint16_t>(a.kv, a.layer, rd.b, head);
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const int ec = (w & 15) + e, j = 8 * tq + (ec & 7), d = ec < 8 ? j : half + j;
    const float c = cs[j], sn = cs[half + j];
    const float out = ec < 8 ? y[e] * c - z[e] * sn : y[e] * c + z[e] * sn;
    if (is_q) a.qr[((size_t)m * H + head) * hd + d] = out;
    else if (kvb) Storage<uint16_t>::store(kvb + KvIndex<uint16_t>::k(rd.pos, d, hd, cap), out);
  }
}

// ---------------------------------------------------------------- tile MFMA kernel (bf16 weights, 129+ rows)
// Launches of more than 128 rows (prefill chunks, up to 4 row tiles of 256 per
// launch, row tiles adjacent in the grid so the blocks sharing a weight
// column tile run together): compute-bound.  A block
// covers 256 rows x 128 weight rows (SwiGLU: 64 gate and the 64 matching up
// rows) with 8 waves in a 4 x 2 grid, each owning 64 x 64 = 4 x 4 MFMA tiles.
// Per k-step the block stages in LDS the x slab (256 rows x 32 columns, split
// into hi + lo bf16 A fragments; each wave moves whole fragments) and its 8
// weight fragments (wave w moves fragment w); each wave then reads 8 A and
// 4 B fragments for its 32 products (384 bytes of LDS per product, against
// 1 KB when a wave owns one column tile).  x and weights are fetched two
// k-steps ahead.  Epilogues in place: store (Q|K|V columns written back in
// natural order, RoPE and the KV append then run in rope_append_kernel),
// SwiGLU, and residual partial sums over n_split k ranges for
// resid_reduce_kernel.
constexpr int kTileThreads = 512;
constexpr int kTileRows = 256, kTileCols = 128;
constexpr int kTileSplitMax = 8;
constexpr int kTileLaunchRows = 1024;  // rows per launch: up to 4 row tiles share each weight column tile
constexpr int kTilePartialRows = 2048; // split-K partials held: n_split * launch rows <= this

template <int KIND>  // EPI_STORE (also Q|K|V), EPI_SWIGLU, EPI_RESID (partials)
__global__ __launch_bounds__(kTileThreads) void gemm_bf16_tile(GemmArgs a, int n_ctiles, int ks_per_split,
                                                               int n_split) {
  constexpr int MTB = kTileRows / 16, NTB = kTileCols / 16;
  constexpr int PJ = kTileRows * 4 / kTileThreads;  // 32-byte x pieces per thread per slab
  constexpr int RSR = kTileRows / (kTileThreads / kWave);
  constexpr bool SCALE = KIND != EPI_RESID, SWIGLU = KIND == EPI_SWIGLU;
  __shared__ u32x4 s_a[2][MTB][2][kWave];  // [buffer][m tile][hi, lo][lane]
  __shared__ u32x4 s_b[2][NTB][kWave];     // [buffer][weight tile][lane]
  __shared__ float scale[kTileRows];

  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 1, wn = wave & 1;
  const int K = a.K, KS = (K + 31) / 32;
  const int n_rt = (a.M + kTileRows - 1) / kTileRows;
  const int rt = (int)blockIdx.x % n_rt, ct = ((int)blockIdx.x / n_rt) % n_ctiles;
  const int split = (int)blockIdx.x / (n_rt * n_ctiles);
  const int ks_begin = split * ks_per_split, ks_end = min(KS, ks_begin + ks_per_split);
  const int n_k = ks_end - ks_begin, n_steps = (n_k + 1) & ~1;
  const int m0 = rt * kTileRows, rows = min(a.M - m0, kTileRows);
  // weight tile j of the block: SwiGLU tiles 0..3 gate, 4..7 up (same columns)
  auto btile = [&](int j) { return SWIGLU ? (j < 2 ? wn * 2 + j : 4 + wn * 2 + (j - 2)) : wn * 4 + j; };

  bool ok;
  const uint16_t* wbase = weight_tile(a, KIND, ct, kTileCols, wave, KS, ok);  // (the tile this wave stages)
  const __amdgpu_buffer_rsrc_t wr = make_rsrc(wbase, ok ? (uint32_t)KS * 1024u : 0u);
  const __amdgpu_buffer_rsrc_t xr = make_rsrc(a.x + (size_t)m0 * a.ldx, (uint32_t)rows * a.ldx * 4u);

  floatx4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};
  f32x4 xv[2][PJ][2];
  u32x4 bv[2];

  auto load = [&](int i, f32x4 (&xs)[PJ][2], u32x4& b) {
    const uint32_t bad = (uint32_t)(i >= n_k) << 31;
    b = __builtin_amdgcn_raw_buffer_load_b128(wr, ((uint32_t)(ks_begin + i) * 1024u + lane * 16u) | bad, 0,
                                              kNonTemporal);
#pragma unroll
    for (int q = 0; q < PJ; ++q) {
      const int p = tid + q * kTileThreads, m = (p >> 6) * 16 + (p & 15);
      const int k = (ks_begin + i) * 32 + ((p >> 4) & 3) * 8;
      const uint32_t off = (((uint32_t)m * a.ldx + k) * 4u) | bad | ((uint32_t)(k >= K) << 31);
      xs[q][0] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(xr, off, 0, 0));
      xs[q][1] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(xr, off + 16u, 0, 0));
    }
  };
  auto store = [&](int buf, const f32x4 (&xs)[PJ][2], const u32x4& b) {
#pragma unroll
    for (int q = 0; q < PJ; ++q) {
      const int p = tid + q * kTileThreads, mt = p >> 6, ln = p & 63;
      bf16x8 hi, lo;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float v = xs[q][e >> 2][e & 3];
        const __bf16 h = (__bf16)v;
        hi[e] = h;
        lo[e] = (__bf16)(v - (float)h);
      }
      s_a[buf][mt][0][ln] = __builtin_bit_cast(u32x4, hi);
      s_a[buf][mt][1][ln] = __builtin_bit_cast(u32x4, lo);
    }
    s_b[buf][wave][lane] = b;
  };
  auto compute = [&](int buf) {
    bf16x8 av[4][2], bw[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      av[i][0] = __builtin_bit_cast(bf16x8, s_a[buf][wm * 4 + i][0][lane]);
      av[i][1] = __builtin_bit_cast(bf16x8, s_a[buf][wm * 4 + i][1][lane]);
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) bw[j] = __builtin_bit_cast(bf16x8, s_b[buf][btile(j)][lane]);
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av[i][h], bw[j], acc[i][j], 0, 0, 0);
    __builtin_amdgcn_sched_group_barrier(0x100, 12, 0);  // LDS reads
    __builtin_amdgcn_sched_group_barrier(0x008, 32, 0);  // then MFMAs
  };

  // Prologue: row-scale partial sums first, then slabs 0 and 1; slab 0 to LDS.
  float rsv[SCALE ? RSR : 1];
  if constexpr (SCALE) {
    const __amdgpu_buffer_rsrc_t sr = make_rsrc(a.ss_in, a.ss_in ? (uint32_t)a.n_ss * a.ss_ld * 4u : 0u);
#pragma unroll
    for (int i = 0; i < RSR; ++i) {
      const int m = m0 + wave + (kTileThreads / kWave) * i;
      const uint32_t off = ((uint32_t)lane * a.ss_ld + m) * 4u | ((uint32_t)(m >= a.M || lane >= a.n_ss) << 31);
      rsv[i] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(sr, off, 0, 0));
    }
  }
  load(0, xv[0], bv[0]);
  load(1, xv[1], bv[1]);
  if constexpr (SCALE) {
    wave_sum_n(rsv);  // (n_ss <= 64: checked by the launcher)
#pragma unroll
    for (int i = 0; i < RSR; ++i) {
      const int r = wave + (kTileThreads / kWave) * i, m = m0 + r;
      if (lane == 0) scale[r] = (a.ss_in && m < a.M) ? 1.0f / sqrtf(rsv[i] / (float)a.K + a.eps) : 1.0f;
    }
  }
  store(0, xv[0], bv[0]);
  load(2, xv[0], bv[0]);
  __syncthreads();

  // Step i: multiply buffer i%2, move slab i+1 (register slot (i+1)%2) into the
  // other buffer, fetch slab i+3 into that slot.  (Steps rounded up to even:
  // the last one multiplies zeros when n_k is odd.)
  for (int i0 = 0; i0 < n_steps; i0 += 2) {
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int i = i0 + u;
      __builtin_amdgcn_sched_barrier(0);
      compute(u);
      __builtin_amdgcn_sched_barrier(0);
      store(u ^ 1, xv[u ^ 1], bv[u ^ 1]);
      load(i + 3, xv[u ^ 1], bv[u ^ 1]);
      __syncthreads();
    }
  }

  // Epilogue.  acc[i][j][r]: row m0 + (wm*4 + i)*16 + 4*(lane/16) + r, column lane%16 of weight tile btile(j).
  const int cl = lane & 15, rg = lane >> 4;
  if constexpr (KIND == EPI_SWIGLU) {
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int f = ct * (kTileCols / 2) + (wn * 2 + j) * 16 + cl;
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int mr = (wm * 4 + i) * 16 + 4 * rg + r;
          if (mr < rows && f < a.n_rows)
            a.out[(size_t)(m0 + mr) * a.ldo + f] =
                silu_f(acc[i][j][r] * scale[mr]) * (acc[i][j + 2][r] * scale[mr]);
        }
    }
  } else if constexpr (KIND == EPI_RESID) {
    float* yp = a.ypart + (size_t)split * a.M * a.n_rows;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int n = ct * kTileCols + btile(j) * 16 + cl;
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int mr = (wm * 4 + i) * 16 + 4 * rg + r;
          if (mr < rows && n < a.n_rows) yp[(size_t)(m0 + mr) * a.n_rows + n] = acc[i][j][r];
        }
    }
  } else {
    // store; Q|K|V: Q and K columns come in the packed RoPE order (column c of
    // a head's tile tq is dim 8*tq + c for c < 8, hd/2 + 8*tq + c - 8 otherwise)
    const int hd = a.head_dim, nqk = a.n_seg[0] + a.n_seg[1];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int n = ct * kTileCols + btile(j) * 16 + cl;
      int col = n;
      if (a.kind == EPI_QKV && n < nqk) {
        const int base = n >= a.n_seg[0] ? a.n_seg[0] : 0, r = n - base, w = r % hd, tq = w >> 4, ec = w & 15;
        col = base + (r / hd) * hd + (ec < 8 ? 8 * tq + ec : hd / 2 + 8 * tq + ec - 8);
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int mr = (wm * 4 + i) * 16 + 4 * rg + r;
          if (mr < rows && n < a.n_rows) a.out[(size_t)(m0 + mr) * a.ldo + col] = acc[i][j][r] * scale[mr];
        }
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
  epilogue<NC, KIND, 256>(a, blk, yfin, scale);
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

// The residual and QKV epilogues keep more live registers: one k-step per
// buffer for single-tile units over more than 16 rows.
template <int T, int MT, int KIND> struct BatchK {
  static constexpr bool tight = (KIND == EPI_RESID || KIND == EPI_QKV) && T == 1 && MT >= 2;
  static constexpr int UB = tight ? 1 : Batch<T, MT>::UB;
  static constexpr bool PIPE = Batch<T, MT>::PIPE;
};

// (INT4 weights: a k-step's fragment is a quarter of the bf16 one, so a buffer
// holds more k-steps to keep as many weight bytes in flight.)
template <int T, int MT, int KIND, bool Q4> struct BatchQ {
  static constexpr int UB = Q4 ? (MT == 1 ? (T == 1 ? 3 : (T == 2 ? 2 : 1)) : 1) : BatchK<T, MT, KIND>::UB;
  static constexpr bool PIPE_Q = !(Q4 && T == 3 && MT == 4);
  static constexpr bool PIPE = BatchK<T, MT, KIND>::PIPE && PIPE_Q;
};

// (Single-tile units reading one stacked x fragment per k-step, from memory or
// LDS, have the registers for four k-steps per buffer: measured 9.9 -> 9.2 us
// for the 7B O projection.  Two fragments per k-step or float32 x would spill.)
template <int T, int MT, int KIND, bool Q4, int XS> struct BatchX {
  static constexpr int UB = (!Q4 && T == 1 && MT == 1 && (XS == 1 || XS == 3)) ? 4 : BatchQ<T, MT, KIND, Q4>::UB;
  static constexpr bool PIPE = BatchQ<T, MT, KIND, Q4>::PIPE;
};

template <int T, int MT, int KIND, bool Q4 = false, int XS = 0>
void launch_mfma_mt(const GemmArgs& a, int tiles, hipStream_t s) {
  const int grid = tiles < compute_units() ? tiles : compute_units();
  hipLaunchKernelGGL(
      (gemm_bf16_mfma<T, MT, BatchX<T, MT, KIND, Q4, XS>::UB, BatchX<T, MT, KIND, Q4, XS>::PIPE, KIND, Q4, XS>),
      dim3(grid), dim3(kMfmaThreads), 0, s, a, tiles);
}

template <int T, int KIND, bool Q4 = false>
hipError_t launch_mfma_t(const GemmArgs& a, int blocks, hipStream_t s) {
  const int MT = (a.M + 15) / 16;
  if constexpr (!Q4) {
    if (a.xs) {  // stacked x (passes of at most 16 rows)
      if (a.stt != (a.M <= 8 ? 1 : 2) || a.M > 16) return hipErrorInvalidValue;
      // (x held in LDS: measured faster for the store, SwiGLU and residual GEMMs, slower for Q|K|V, whose
      // epilogue tables then leave room for one reduction fragment per round only)
      if (KIND != EPI_QKV && a.stt == 1 && (a.K + 31) / 32 <= 8 * kMfmaWaves)
        launch_mfma_mt<T, 1, KIND, false, 3>(a, blocks, s);
      else if (a.stt == 1) launch_mfma_mt<T, 1, KIND, false, 1>(a, blocks, s);
      else launch_mfma_mt<T, 1, KIND, false, 2>(a, blocks, s);
      return hipGetLastError();
    }
  }
  if (MT <= 1) launch_mfma_mt<T, 1, KIND, Q4>(a, blocks, s);
  else if (MT <= 2) launch_mfma_mt<T, 2, KIND, Q4>(a, blocks, s);
  else if (MT <= 4) launch_mfma_mt<T, 4, KIND, Q4>(a, blocks, s);
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
__global__ void pack_kernel(const uint16_t* __restrict__ src, uint16_t* __restrict__ dst, int N, int K, int KS,
                            int rope_hd) {
  const size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x;
  const size_t pieces = (size_t)(N / 16) * KS * 64;
  if (i >= pieces) return;
  const int lane = (int)(i % 64);
  const size_t frag = i / 64;
  const int ks = (int)(frag % KS), t = (int)(frag / KS);
  int row = 16 * t + (lane & 15);
  if (rope_hd > 0) {  // tile t of its head: rows 8t' + e and hd/2 + 8t' + e, e < 8
    const int head = (16 * t) / rope_hd, tq = (16 * t) % rope_hd / 16, e = lane & 15;
    row = head * rope_hd + (e < 8 ? 8 * tq + e : rope_hd / 2 + 8 * tq + (e - 8));
  }
  const int k = 32 * ks + 8 * (lane >> 4);
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

// INT4 quantization and packing, one thread per (packed row n, group of 128
// columns): s = bf16(max|w| / 7) (IEEE division), q = clamp(rint(w / s), -8, 7)
// (q = 0 where s = 0); the thread writes its row's 16 code words of the
// group and the row's scale.  Rows follow the bf16 image's order (rope_hd).
__global__ void pack_int4_kernel(const uint16_t* __restrict__ src, uint32_t* __restrict__ frag,
                                 uint16_t* __restrict__ scale, int N, int K, int KS, int KG, int rope_hd) {
  const size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x;
  if (i >= (size_t)N * KG) return;
  const int n = (int)(i / KG), g = (int)(i % KG);
  int row = n;
  if (rope_hd > 0) {
    const int t = n / 16, head = (16 * t) / rope_hd, tq = (16 * t) % rope_hd / 16, e = n & 15;
    row = head * rope_hd + (e < 8 ? 8 * tq + e : rope_hd / 2 + 8 * tq + (e - 8));
  }
  const uint16_t* w = src + (size_t)row * K;
  const int k0 = g * 128, k1 = min(K, k0 + 128);
  float amax = 0.f;
  for (int k = k0; k < k1; ++k) amax = fmaxf(amax, fabsf(bf16_bits_to_f32(w[k])));
  const __bf16 sb = (__bf16)__fdiv_rn(amax, 7.0f);
  const float sf = (float)sb;
  scale[((size_t)(n / 16) * KG + g) * 16 + (n & 15)] = __builtin_bit_cast(uint16_t, sb);
  // (the group's four k-steps: a k-step past K keeps zero codes)
  for (int j = 0; j < 4; ++j)
    for (int kg = 0; kg < 4; ++kg) {
      const int ks = 4 * g + j;
      uint32_t word = 0u;
      for (int e = 0; e < 8; ++e) {
        const int k = ks * 32 + kg * 8 + e;
        int q = 0;
        if (ks < KS && k < K && sf != 0.f)
          q = (int)fminf(fmaxf(rintf(__fdiv_rn(bf16_bits_to_f32(w[k]), sf)), -8.f), 7.f);
        word |= ((uint32_t)q & 0xFu) << (4 * e);
      }
      frag[(((size_t)(n / 16) * KG + g) * 64 + kg * 16 + (n & 15)) * 4 + j] = word;
    }
}

}  // namespace

int device_compute_units() { return compute_units(); }

size_t packed_int4_frag_bytes(int N, int K) { return (size_t)(N / 16) * ((K + 127) / 128) * 1024; }
size_t packed_int4_scale_bytes(int N, int K) { return (size_t)(N / 16) * ((K + 127) / 128) * 32; }

hipError_t launch_pack_int4(const void* src, void* frag, void* scale, int N, int K, int rope_hd, hipStream_t s) {
  if (N % 16 || K % 32) return hipErrorInvalidValue;
  if (rope_hd < 0 || (rope_hd > 0 && (rope_hd % 16 || N % rope_hd))) return hipErrorInvalidValue;
  const int KS = K / 32, KG = (K + 127) / 128;
  const size_t n = (size_t)N * KG;
  hipLaunchKernelGGL(pack_int4_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, (const uint16_t*)src,
                     (uint32_t*)frag, (uint16_t*)scale, N, K, KS, KG, rope_hd);
  return hipGetLastError();
}

size_t packed_elems(int N, int K) { return (size_t)(N / 16) * ((K + 31) / 32) * 512; }

hipError_t launch_pack(const void* src, void* dst, int N, int K, int rope_hd, hipStream_t s) {
  if (N % 16 || K % 8) return hipErrorInvalidValue;
  if (rope_hd < 0 || (rope_hd > 0 && (rope_hd % 16 || N % rope_hd))) return hipErrorInvalidValue;
  const int KS = (K + 31) / 32;
  const size_t pieces = (size_t)(N / 16) * KS * 64;
  hipLaunchKernelGGL(pack_kernel, dim3((unsigned)((pieces + 255) / 256)), dim3(256), 0, s, (const uint16_t*)src,
                     (uint16_t*)dst, N, K, KS, rope_hd);
  return hipGetLastError();
}

bool gemm_wide(int dtype, int M) { return dtype == SPECDEC_BF16 && M > kMaxGemmRows; }
int gemm_launch_rows(int dtype, int M) {
  return !gemm_wide(dtype, M) ? kMaxGemmRows : (M > kWideRows ? kTileLaunchRows : kWideRows);
}
size_t wide_ypart_floats(int n_rows) {
  return (size_t)std::max(kWideSplitMax * kWideRows, kTilePartialRows) * n_rows;
}

int gemm_row_blocks(int dtype, int kind, int n_rows, int M) {
  if (gemm_wide(dtype, M) && kind == EPI_RESID) return (n_rows + kWideCols - 1) / kWideCols;
  if (dtype == SPECDEC_BF16) {
    int nc = 16 * mfma_tiles(kind, n_rows);
    int per = kind == EPI_SWIGLU ? nc / 2 : nc;
    return (n_rows + per - 1) / per;
  }
  int per = kind == EPI_SWIGLU ? 16 : 16;
  return (n_rows + per - 1) / per;
}

namespace {
template <int MT, int T, int KIND>
void launch_wide_mt(const GemmArgs& a, int blocks, int ks_per_split, int n_split, hipStream_t s) {
  hipLaunchKernelGGL((gemm_bf16_wide<MT, T, KIND>), dim3(blocks * n_split), dim3(kWideThreads), 0, s, a,
                     ks_per_split, n_split);
}
template <int T, int KIND>
void launch_wide_t(const GemmArgs& a, int blocks, int ks_per_split, int n_split, hipStream_t s) {
  const int MT = (a.M + 15) / 16;
  if (MT <= 4) launch_wide_mt<4, T, KIND>(a, blocks, ks_per_split, n_split, s);
  else if (MT <= 7) launch_wide_mt<7, T, KIND>(a, blocks, ks_per_split, n_split, s);
  else launch_wide_mt<8, T, KIND>(a, blocks, ks_per_split, n_split, s);
}

// Launches of 129..1024 rows on the tile kernel (Q|K|V: a store of the
// projections in natural column order, then rope_append_kernel).
hipError_t launch_tile(const GemmArgs& a, hipStream_t s) {
  if (a.M > kTileLaunchRows || (a.ss_in && a.n_ss > kWideMaxSs)) return hipErrorInvalidValue;
  const int KS = (a.K + 31) / 32, n_rt = (a.M + kTileRows - 1) / kTileRows;
  switch (a.kind) {
    case EPI_STORE:
    case EPI_QKV: {
      if (a.kind == EPI_QKV && (!a.out || a.ldo < a.n_rows || a.head_dim % 16 || a.n_seg[0] % a.head_dim ||
                                a.n_seg[1] % a.head_dim))
        return hipErrorInvalidValue;
      const int nct = (a.n_rows + kTileCols - 1) / kTileCols;
      hipLaunchKernelGGL(gemm_bf16_tile<EPI_STORE>, dim3(n_rt * nct), dim3(kTileThreads), 0, s, a, nct, KS, 1);
      if (a.kind == EPI_QKV) {
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        AttnArgs r{};
        r.rows = a.rows; r.M = a.M; r.rps = a.M; r.n_heads = a.n_heads; r.n_kv_heads = a.n_kv_heads;
        r.head_dim = a.head_dim; r.qkv = a.out; r.rope_cs = a.rope_cs; r.qr = a.qr; r.kv = a.kv; r.layer = a.layer;
        return launch_rope_append(r, s);
      }
      break;
    }
    case EPI_SWIGLU: {
      const int nct = (a.n_rows + kTileCols / 2 - 1) / (kTileCols / 2);
      hipLaunchKernelGGL(gemm_bf16_tile<EPI_SWIGLU>, dim3(n_rt * nct), dim3(kTileThreads), 0, s, a, nct, KS, 1);
      break;
    }
    case EPI_RESID: {
      if (!a.ypart || a.n_rows % 4) return hipErrorInvalidValue;
      const int nct = (a.n_rows + kTileCols - 1) / kTileCols, blocks = n_rt * nct;
      int n_split = std::min(kTileSplitMax, std::max(1, (compute_units() + blocks - 1) / blocks));
      n_split = std::min({n_split, KS, kTilePartialRows / a.M});
      const int per = (KS + n_split - 1) / n_split;
      n_split = (KS + per - 1) / per;
      hipLaunchKernelGGL(gemm_bf16_tile<EPI_RESID>, dim3(blocks * n_split), dim3(kTileThreads), 0, s, a, nct, per,
                         n_split);
      hipLaunchKernelGGL(resid_reduce_kernel, dim3((a.n_rows + kWideCols - 1) / kWideCols, (a.M + 7) / 8),
                         dim3(256), 0, s, a, n_split);
      break;
    }
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_wide(const GemmArgs& a, hipStream_t s) {
  if (a.M > kWideRows) return launch_tile(a, s);
  if (a.ss_in && a.n_ss > kWideMaxSs) return hipErrorInvalidValue;
  const int KS = (a.K + 31) / 32, cus = compute_units();
  switch (a.kind) {
    case EPI_STORE: {
      const int T = (a.n_rows + 127) / 128 * 10 >= cus * 9 ? 2 : 1;
      const int blocks = (a.n_rows + 64 * T - 1) / (64 * T);
      if (T == 2) launch_wide_t<2, EPI_STORE>(a, blocks, KS, 1, s);
      else launch_wide_t<1, EPI_STORE>(a, blocks, KS, 1, s);
      break;
    }
    case EPI_QKV: {
      if (a.kv.dtype != SPECDEC_BF16 || a.head_dim % 16 || a.n_seg[0] % a.head_dim || a.n_seg[1] % a.head_dim)
        return hipErrorInvalidValue;
      // Three tiles per wave over a K split that keeps the grid within the
      // CUs (the 7B shape: 64 column blocks x 4 splits): raw partial sums,
      // then qkv_reduce_kernel (row scale, RoPE, the query store and the KV
      // append).  The wide kernel's time follows its k-steps per
      // block more than its products per k-step, so fewer k-steps per block
      // pay for the extra launches (16 long-context 7B sequences, 112 rows per
      // verify: 16.53 -> 15.16 ms on one box together with the SwiGLU split,
      // one tile per wave and no split before).
      const int blocks = (a.n_rows + 191) / 192;
      int n_split = std::min({kWideSplitMax, KS, std::max(1, cus / blocks)});
      const int ks_per_split = (KS + n_split - 1) / n_split;
      n_split = (KS + ks_per_split - 1) / ks_per_split;
      if (!a.ypart || a.n_rows % 16 || (size_t)n_split * a.M * a.n_rows > wide_ypart_floats(a.K)) {
        launch_wide_t<1, EPI_QKV>(a, (a.n_rows + 63) / 64, KS, 1, s);
        break;
      }
      GemmArgs p = a;
      p.kind = EPI_RESID;
      launch_wide_t<3, EPI_RESID>(p, blocks, ks_per_split, n_split, s);
      hipLaunchKernelGGL(qkv_reduce_kernel, dim3((a.n_rows + kWideCols - 1) / kWideCols, (a.M + 7) / 8), dim3(256), 0,
                         s, a, n_split);
      break;
    }
    case EPI_SWIGLU: {
      // The gate and up rows as one 2F-row matrix, three tiles per wave, K
      // split within the CUs: raw partial sums, then swiglu_reduce_kernel.
      const int W = 2 * a.n_rows, blocks = (W + 191) / 192;
      int n_split = std::min({kWideSplitMax, KS, std::max(1, cus / blocks)});
      const int ks_per_split = (KS + n_split - 1) / n_split;
      n_split = (KS + ks_per_split - 1) / ks_per_split;
      if (n_split < 2 || !a.ypart || a.n_rows % 16 || a.ldo % 4 || (size_t)n_split * a.M * W > wide_ypart_floats(a.K)) {
        launch_wide_t<2, EPI_SWIGLU>(a, (a.n_rows + 63) / 64, KS, 1, s);
        break;
      }
      GemmArgs p = a;
      p.kind = EPI_RESID;
      p.n_rows = W;
      p.n_seg[0] = a.n_rows;
      p.n_seg[1] = a.n_rows;
      p.n_seg[2] = 0;
      launch_wide_t<3, EPI_RESID>(p, blocks, ks_per_split, n_split, s);
      hipLaunchKernelGGL(swiglu_reduce_kernel, dim3((a.n_rows + kWideCols - 1) / kWideCols, (a.M + 7) / 8), dim3(256),
                         0, s, a, n_split);
      break;
    }
    case EPI_RESID: {
      if (!a.ypart || a.n_rows % 16) return hipErrorInvalidValue;
      // Three tiles per wave (each x slab serves 192 columns) and K split as far
      // as the grid stays within the CUs (each split at least one k-step): the
      // 7B O and down projections over 112 rows run 22 column blocks x 11
      // splits.  (One tile per wave and 4 splits, then two tiles and 8 splits:
      // the 16-sequence long-context verify 17.10 -> 16.50 ms, then
      // 15.46-15.71 -> 15.11-15.25 ms, each on one box.)
      const int blocks = (a.n_rows + 191) / 192;
      int n_split = std::min(kWideSplitMax, std::max(1, cus / blocks));
      n_split = std::min(n_split, KS);
      const int ks_per_split = (KS + n_split - 1) / n_split;
      n_split = (KS + ks_per_split - 1) / ks_per_split;
      launch_wide_t<3, EPI_RESID>(a, blocks, ks_per_split, n_split, s);
      hipLaunchKernelGGL(resid_reduce_kernel, dim3((a.n_rows + kWideCols - 1) / kWideCols, (a.M + 7) / 8),
                         dim3(256), 0, s, a, n_split);
      break;
    }
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}
}  // namespace

// INT4 passes of at most 16 rows on gemm_q4_lds: hipErrorNotSupported where
// its register budget does not cover the shape (the caller then runs the
// skinny kernel's INT4 path).  Groups per wave and window: all of them (one
// window) while the rows allow, else one.
template <int U, int TU, int GW, int KIND>
static void launch_q4_w(const GemmArgs& a, int n_units, int gw, hipStream_t s) {
  const int grid = std::min(n_units, compute_units());
  constexpr int G1 = GW == 4 ? 4 : 6;  // (12 groups: two windows of 6 for up to 5 rows)
  if (G1 * a.M <= kQ4WindowRows)
    hipLaunchKernelGGL((gemm_q4_lds<U, TU, GW, G1, KIND>), dim3(grid), dim3(kQ4Threads), 0, s, a, n_units, gw);
  else
    hipLaunchKernelGGL((gemm_q4_lds<U, TU, GW, 1, KIND>), dim3(grid), dim3(kQ4Threads), 0, s, a, n_units, gw);
}

template <int U, int TU, int KIND>
static hipError_t launch_q4_u(const GemmArgs& a, int n_units, int gw, hipStream_t s) {
  if (gw <= 4) {
    launch_q4_w<U, TU, 4, KIND>(a, n_units, gw, s);
  } else if constexpr (U * TU == 1) {  // (12 groups per wave: single-tile units only)
    if (gw > 12) return hipErrorNotSupported;
    launch_q4_w<U, TU, 12, KIND>(a, n_units, gw, s);
  } else {
    return hipErrorNotSupported;
  }
  return hipGetLastError();
}

static hipError_t launch_q4_lds(const GemmArgs& a, hipStream_t s) {
  if (a.M > kQ4Rows || a.n_rows % 16 || (a.kind == EPI_QKV && a.head_dim > 128)) return hipErrorNotSupported;
  // (residual GEMMs: one tile per unit, as the RMSNorm partials of the consumer expect)
  if (a.kind == EPI_RESID && mfma_tiles(EPI_RESID, a.n_rows) != 1) return hipErrorNotSupported;
  const int n_units = a.n_rows / 16, cus = compute_units();
  const int U = (n_units + cus - 1) / cus;
  const int G = (a.K + 127) / 128, gw = (G + kQ4Waves - 1) / kQ4Waves;
  switch (a.kind) {
    case EPI_QKV:
      if (U == 1) return launch_q4_u<1, 1, EPI_QKV>(a, n_units, gw, s);
      if (U == 2) return launch_q4_u<2, 1, EPI_QKV>(a, n_units, gw, s);
      if (U == 3) return launch_q4_u<3, 1, EPI_QKV>(a, n_units, gw, s);
      break;
    case EPI_SWIGLU:
      if (U == 1) return launch_q4_u<1, 2, EPI_SWIGLU>(a, n_units, gw, s);
      if (U == 2) return launch_q4_u<2, 2, EPI_SWIGLU>(a, n_units, gw, s);
      if (U == 3) return launch_q4_u<3, 2, EPI_SWIGLU>(a, n_units, gw, s);
      break;
    case EPI_RESID:
      if (U == 1) return launch_q4_u<1, 1, EPI_RESID>(a, n_units, gw, s);
      if (U == 2) return launch_q4_u<2, 1, EPI_RESID>(a, n_units, gw, s);
      break;
    default: break;
  }
  return hipErrorNotSupported;
}

hipError_t launch_gemm(int dtype, const GemmArgs& a, hipStream_t s) {
  if (a.M <= 0 || (a.K % 8) != 0 || (a.ldx % 4) != 0) return hipErrorInvalidValue;
  if (a.wide) {
    if (a.q4) return hipErrorInvalidValue;  // (INT4 weights run passes of at most 64 rows)
    if (dtype != SPECDEC_BF16 || (a.kind == EPI_RESID && (!a.gain_bf16 || a.n_rows % 4))) return hipErrorInvalidValue;
    return launch_wide(a, s);
  }
  if (a.M > kMaxGemmRows) return hipErrorInvalidValue;
  const int blocks = gemm_row_blocks(dtype, a.kind, a.n_rows, a.M);
  if (a.q4) {  // INT4 layer weights (passes of at most 64 rows)
    if (dtype != SPECDEC_BF16 || (a.K % 32) != 0) return hipErrorInvalidValue;
    if (a.kind == EPI_RESID && !a.gain_bf16) return hipErrorInvalidValue;
    if (a.kind == EPI_QKV && (a.kv.dtype != SPECDEC_BF16 || a.head_dim % 16 || a.n_seg[0] % a.head_dim ||
                              a.n_seg[1] % a.head_dim))
      return hipErrorInvalidValue;
    const hipError_t e = launch_q4_lds(a, s);
    if (e != hipErrorNotSupported) return e;
    // (Q|K|V over more than 32 rows: one tile per unit, the registers going to
    // the row tiles; the residual GEMMs keep mfma_tiles' count, which their
    // RMSNorm partials follow)
    const int T = a.M > 32 && a.kind == EPI_QKV ? 1 : mfma_tiles(a.kind, a.n_rows);
    const int units = a.kind == EPI_QKV ? (a.n_rows + 16 * T - 1) / (16 * T) : blocks;
    switch (a.kind) {
      case EPI_RESID:
        if (!a.gain_bf16) return hipErrorInvalidValue;
        return T == 1 ? launch_mfma_t<1, EPI_RESID, true>(a, blocks, s)
                      : (T == 2 ? launch_mfma_t<2, EPI_RESID, true>(a, blocks, s)
                                : launch_mfma_t<3, EPI_RESID, true>(a, blocks, s));
      case EPI_SWIGLU: return launch_mfma_t<2, EPI_SWIGLU, true>(a, blocks, s);
      case EPI_QKV:
        if (a.kv.dtype != SPECDEC_BF16 || a.head_dim % 16 || a.n_seg[0] % a.head_dim || a.n_seg[1] % a.head_dim)
          return hipErrorInvalidValue;
        return T == 1 ? launch_mfma_t<1, EPI_QKV, true>(a, units, s)
                      : (T == 2 ? launch_mfma_t<2, EPI_QKV, true>(a, units, s)
                                : launch_mfma_t<3, EPI_QKV, true>(a, units, s));
      default: return hipErrorInvalidValue;
    }
  }
  if (dtype == SPECDEC_BF16) {
    if (a.kind == EPI_RESID && !a.gain_bf16) return hipErrorInvalidValue;
    const int T = mfma_tiles(a.kind, a.n_rows);
    switch (a.kind) {
      case EPI_STORE: {
        // (x as the stacked operand: single-tile units, which hold four k-steps
        // per register buffer, where they balance over the CUs as well; the 7B
        // LM head over 5 rows took 43.3 us in 2000 units against 45.3 us in 1000.
        // With float32 x the larger unit stays: 46 against 59 us.)
        const int cus = compute_units(), u1 = (a.n_rows + 15) / 16;
        const double e1 = (double)u1 / ((double)((u1 + cus - 1) / cus) * cus);
        const double eT = (double)blocks / ((double)((blocks + cus - 1) / cus) * cus);
        if (a.xs && T > 1 && e1 >= eT - 1e-9) return launch_mfma_t<1, EPI_STORE>(a, u1, s);
        return T == 1 ? launch_mfma_t<1, EPI_STORE>(a, blocks, s)
                      : (T == 2 ? launch_mfma_t<2, EPI_STORE>(a, blocks, s) : launch_mfma_t<3, EPI_STORE>(a, blocks, s));
      }
      case EPI_RESID:
        return T == 1 ? launch_mfma_t<1, EPI_RESID>(a, blocks, s)
                      : (T == 2 ? launch_mfma_t<2, EPI_RESID>(a, blocks, s) : launch_mfma_t<3, EPI_RESID>(a, blocks, s));
      case EPI_SWIGLU: return launch_mfma_t<2, EPI_SWIGLU>(a, blocks, s);
      case EPI_QKV:
        if (a.kv.dtype != SPECDEC_BF16 || a.head_dim % 16 || a.n_seg[0] % a.head_dim || a.n_seg[1] % a.head_dim)
          return hipErrorInvalidValue;
        return T == 1 ? launch_mfma_t<1, EPI_QKV>(a, blocks, s)
                      : (T == 2 ? launch_mfma_t<2, EPI_QKV>(a, blocks, s) : launch_mfma_t<3, EPI_QKV>(a, blocks, s));
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
