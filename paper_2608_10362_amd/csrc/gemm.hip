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

// ---------------------------------------------------------------- MFMA kernel (bf16 weights)
// Block = 16 waves; the block owns NC = 16*T weight rows and all M rows of x;
// wave w reduces k-steps [w*KS/16, (w+1)*KS/16) of 32 columns each, UB k-steps
// per batch of loads.  MFMA operand layout (16x16x32): lane l holds
// A[l%16][8(l/16)+j] (x rows), B[8(l/16)+j][l%16] (= W[n0 + l%16][k0 + 8(l/16) + j]),
// D[4(l/16)+r][l%16].
template <int T, int MT, int UB, bool PIPE, int KIND>
__global__ __launch_bounds__(kMfmaThreads) void gemm_bf16_mfma(GemmArgs a) {
  constexpr int NC = 16 * T;
  constexpr int MP = 16 * MT;
  __shared__ float red[kMfmaWaves][kWave][4];
  __shared__ float yfin[MP][NC + 1];
  __shared__ float scale[MP];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int blk = blockIdx.x;
  const int kg = lane >> 4, mrow = lane & 15;

  const uint16_t* wrow[T];
  bool rok[T];
#pragma unroll
  for (int t = 0; t < T; ++t) wrow[t] = weight_row<uint16_t>(a, KIND, blk, NC, t * 16 + mrow, rok[t]);

  const int K = a.K;
  const int KS = (K + 31) / 32;
  const int ks0 = (wave * KS) / kMfmaWaves, ks1 = ((wave + 1) * KS) / kMfmaWaves;

  floatx4 acc[T][MT];
#pragma unroll
  for (int t = 0; t < T; ++t)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) acc[t][mt] = floatx4{0.f, 0.f, 0.f, 0.f};

  // Two register buffers of UB k-steps: the loads of batch i+1 are in flight
  // while batch i is multiplied.
  u32x4 wA[UB][T], wB[UB][T];
  f32x4 xA[UB][MT][2], xB[UB][MT][2];
  auto load = [&](int kb, u32x4 (&wv)[UB][T], f32x4 (&xv)[UB][MT][2]) {
#pragma unroll
    for (int u = 0; u < UB; ++u) {
      const int k = (kb + u) * 32 + kg * 8;
      const bool kok = (kb + u) < ks1 && k < K;
#pragma unroll
      for (int t = 0; t < T; ++t) {
        if (kok && rok[t]) wv[u][t] = __builtin_nontemporal_load((const u32x4*)(wrow[t] + k));
        else wv[u][t] = u32x4{0u, 0u, 0u, 0u};
      }
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        const int m = mt * 16 + mrow;
        if (kok && m < a.M) {
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
  int kb = ks0;
  if (PIPE) {
    if (kb < ks1) load(kb, wA, xA);
    while (kb < ks1) {
      if (kb + UB < ks1) load(kb + UB, wB, xB);
      compute(wA, xA);
      kb += UB;
      if (kb >= ks1) break;
      if (kb + UB < ks1) load(kb + UB, wA, xA);
      compute(wB, xB);
      kb += UB;
    }
  } else {
    for (; kb < ks1; kb += UB) {
      load(kb, wA, xA);
      compute(wA, xA);
    }
  }

  // The row scale is only needed by the epilogue: computed after the weight stream.
  row_scale<MP>(a, scale);

  // Cross-wave reduction, fragment by fragment, in a fixed wave order.
#pragma unroll
  for (int t = 0; t < T; ++t) {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
#pragma unroll
      for (int r = 0; r < 4; ++r) red[wave][lane][r] = acc[t][mt][r];
      __syncthreads();
      if (tid < 256) {
        const int l = tid & 63, r = tid >> 6;
        float s = 0.f;
#pragma unroll
        for (int w = 0; w < kMfmaWaves; ++w) s += red[w][l][r];
        yfin[mt * 16 + 4 * (l >> 4) + r][t * 16 + (l & 15)] = s;
      }
      __syncthreads();
    }
  }
  epilogue<NC, KIND>(a, blk, yfin, scale);
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
template <> struct Batch<1, 1> { static constexpr int UB = 4; static constexpr bool PIPE = true; };
template <> struct Batch<1, 2> { static constexpr int UB = 2; static constexpr bool PIPE = true; };
template <> struct Batch<1, 4> { static constexpr int UB = 2; static constexpr bool PIPE = false; };
template <> struct Batch<2, 1> { static constexpr int UB = 2; static constexpr bool PIPE = true; };
template <> struct Batch<2, 2> { static constexpr int UB = 1; static constexpr bool PIPE = true; };
template <> struct Batch<2, 4> { static constexpr int UB = 1; static constexpr bool PIPE = false; };

template <int T, int MT, int KIND>
void launch_mfma_mt(const GemmArgs& a, int blocks, hipStream_t s) {
  hipLaunchKernelGGL((gemm_bf16_mfma<T, MT, Batch<T, MT>::UB, Batch<T, MT>::PIPE, KIND>), dim3(blocks),
                     dim3(kMfmaThreads), 0, s, a);
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

// Tiles (of 16 weight rows) per block for the bf16 kernel.
int mfma_tiles(int kind, int n_rows) {
  if (kind == EPI_SWIGLU) return 2;
  return n_rows >= 16384 ? 2 : 1;
}

}  // namespace

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
      case EPI_STORE: return T == 1 ? launch_mfma_t<1, EPI_STORE>(a, blocks, s) : launch_mfma_t<2, EPI_STORE>(a, blocks, s);
      case EPI_RESID: return T == 1 ? launch_mfma_t<1, EPI_RESID>(a, blocks, s) : launch_mfma_t<2, EPI_RESID>(a, blocks, s);
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
