// Host-side interfaces between the C ABI (api.hip) and the kernel files.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "specdec.h"
#include "device_common.h"

namespace specdec {

// ------------------------------------------------------------------ KV cache layout
// Per layer l, sequence b, kv head g: a K block then a V block of
// capacity*head_dim elements each, at element offset
// ((l*B + b)*h_kv + g) * 2*capacity*head_dim.
//  * bf16 caches store both in MFMA operand order, in 1 KB fragments:
//    K fragment (16 positions x 32 dims): lane 16*(d%32/8) + p%16, element d%8;
//    V fragment (32 positions x 16 dims): lane 16*(p%32/8) + d%16, element p%8.
//  * float32 caches: K row-major [position][dim], V transposed [dim][position].
struct KvLayout {
  void* data;
  int batch, capacity, n_kv_heads, head_dim, dtype;
  size_t layer_elems() const { return (size_t)batch * n_kv_heads * 2 * (size_t)capacity * head_dim; }
};

template <typename KT>
__device__ __forceinline__ KT* k_block(const KvLayout& kv, int layer, int b, int g) {
  size_t off = (((size_t)layer * kv.batch + b) * kv.n_kv_heads + g) * 2 * (size_t)kv.capacity * kv.head_dim;
  return (KT*)kv.data + off;
}

// Element offsets of K[p][d] and V[p][d] inside a (layer, sequence, kv head) block.
template <typename KT> struct KvIndex;
template <> struct KvIndex<float> {
  __device__ static size_t k(int p, int d, int hd, int cap) { return (size_t)p * hd + d; }
  __device__ static size_t v(int p, int d, int hd, int cap) { return (size_t)cap * hd + (size_t)d * cap + p; }
};
template <> struct KvIndex<uint16_t> {
  __device__ static size_t k(int p, int d, int hd, int cap) {
    const int kst = hd / 32;
    return ((size_t)((p >> 4) * kst + (d >> 5)) * 64 + ((d & 31) >> 3) * 16 + (p & 15)) * 8 + (d & 7);
  }
  __device__ static size_t v(int p, int d, int hd, int cap) {
    const int dt = hd / 16;
    return (size_t)cap * hd + ((size_t)((p >> 5) * dt + (d >> 4)) * 64 + ((p & 31) >> 3) * 16 + (d & 15)) * 8 +
           (p & 7);
  }
};

// ------------------------------------------------------------------ GEMM
// y = (x (.) gain) W^T, optional per-row scale s_m = 1/sqrt(mean_k h_mk^2 + eps)
// taken from partial sums of squares, W bf16 or f32 row-major [N, K] split in
// up to three row segments (Wq|Wk|Wv, or gate|up for SwiGLU).
// EPI_QKV (bf16 only): Q|K|V projections whose epilogue applies RoPE to the
// query and key rows, writes the rotated queries to qr and appends K and V
// to the cache.  It needs the rotation pairs (j, j + hd/2) of a head in the
// same 16-row tile, which the packed image provides (see launch_pack).
enum EpiKind { EPI_STORE = 0, EPI_RESID = 1, EPI_SWIGLU = 2, EPI_QKV = 3 };
constexpr int kMaxGemmRows = 64;  // rows of x per launch of the skinny kernels (callers split larger M)
// Passes of more than kMaxGemmRows bf16 rows run the wide kernel in launches of
// up to gemm_launch_rows() rows; residual GEMMs there split K over the grid
// and need ypart = wide_ypart_floats(n_rows) floats.
bool gemm_wide(int dtype, int M);
int gemm_launch_rows(int dtype, int M);
size_t wide_ypart_floats(int n_rows);

struct GemmArgs {
  const float* x;      // [M, ldx] (for normalised inputs: h * gain, the producer applies the gain)
  int ldx;
  const float* ss_in;  // [n_ss, ss_ld] partial sums of squares of the h rows, or null (no row scale)
  int n_ss, ss_ld;
  float eps;
  int M, K;
  const void* w[3];    // bf16: packed images of the segments; f32: row-major [n_seg, K]
  int n_seg[3];
  int n_rows;          // total rows over segments (STORE/RESID); F for SWIGLU
  int kind;
  float* out;          // STORE: [M, ldo] ; SWIGLU: [M, ldo] ; RESID: residual [M, ldo] updated in place
  int ldo;
  float* ss_out;       // RESID: [n_blocks, ss_ld] sums of squares of the new residual rows
  float* xg_out;       // RESID: [M, ldo] new residual times gain_out (input of the next RMSNorm'd GEMM)
  const void* gain_out;
  int gain_bf16;
  // EPI_QKV
  const RowDesc* rows;    // [M]
  const float* rope_cs;   // [M, hd]: cos (j < hd/2) then sin
  float* qr;              // [M, H, hd] rotated queries
  KvLayout kv;
  int layer, n_heads, n_kv_heads, head_dim;
  // wide passes
  int wide;               // 1: the whole pass has more than kMaxGemmRows rows (set by the caller for every launch)
  float* ypart;           // RESID: split-K partial sums, wide_ypart_floats(n_rows) floats
  // Passes of at most 16 rows, bf16 weights: x also as a stacked operand
  // (put_stacked, stt fragments per k-step), read instead of x when xs is set;
  // RESID and SwiGLU epilogues also write their output stacked into xs_out.
  const uint16_t* xs;
  uint16_t* xs_out;
  int stt;
  // INT4 weights: w[] are INT4 images (packed_int4_*), wscale[] their group scales
  int q4;
  const uint16_t* wscale[3];
};
// Packed bf16 weight image (16-row x 32-column 1 KB fragments in MFMA operand
// order).  rope_hd > 0 reorders the rows of each head of rope_hd rows so that
// tile t of the head holds rows 8t..8t+7 then rope_hd/2 + 8t .. +7 (the
// rotation pairs of RoPE side by side, 8 columns apart); 0 keeps the order.
size_t packed_elems(int N, int K);
hipError_t launch_pack(const void* src, void* dst, int N, int K, int rope_hd, hipStream_t s);
// INT4 image of a bf16 W [N, K] (K % 32 == 0): code blocks of 1 KB per 16-row
// tile and group of 128 columns (lane l of the bf16 fragment's lane order holds
// the 32-bit code words of the group's four k-steps, 4 bits per code, low
// nibble first) and bf16 scales [N/16][ceil(K/128)][16]; the quantizer runs on
// the device (groups of 128 columns, s = bf16(max|w| / 7), q = clamp(rint(w/s),
// -8, 7)).  rope_hd as for launch_pack.
size_t packed_int4_frag_bytes(int N, int K);
size_t packed_int4_scale_bytes(int N, int K);
hipError_t launch_pack_int4(const void* src, void* frag, void* scale, int N, int K, int rope_hd, hipStream_t s);
// Number of row blocks the launcher uses for this GEMM (for ss partial counts)
// in a pass of M rows.
int gemm_row_blocks(int dtype, int kind, int n_rows, int M);
hipError_t launch_gemm(int dtype, const GemmArgs& a, hipStream_t s);

// ------------------------------------------------------------------ rows / embedding
enum RowMode { ROWS_VERIFY = 0, ROWS_DRAFT_FIRST = 1, ROWS_DRAFT_NEXT = 2, ROWS_PREFILL = 3 };
struct RowsArgs {
  int mode, M, rps;       // rows, rows per sequence
  const int32_t* len;     // [B]
  const int32_t* pending; // [2B]
  const int32_t* n_pending;
  int32_t* status;
  const int32_t* tok_src; // VERIFY/DRAFT_NEXT: drafts (ld_tok); PREFILL: tokens [B, ld_tok]
  int ld_tok;
  int slot;               // DRAFT_NEXT
  int c0;                 // PREFILL: first token index of this chunk
  int capacity, vocab, d_model, head_dim;
  double rope_base;
  const void* embed;      // [V, d] storage type
  const void* gain;       // [d] first layer's attention RMSNorm gain
  RowDesc* rows;          // out [M]
  float* rope_cs;         // out [M, head_dim]: cos j<hd/2 then sin
  float* h;               // out [M, d]
  float* xg;              // out [M, d] h * gain
  float* ss;              // out [M] sum of squares of h rows
  uint16_t* xs;           // out (or null): xg as a stacked operand (put_stacked), stt fragments per k-step
  int stt;
};
hipError_t launch_rows_embed(int dtype, const RowsArgs& a, hipStream_t s);

// ------------------------------------------------------------------ attention
struct AttnArgs {
  const RowDesc* rows;
  int M, rps, n_heads, n_kv_heads, head_dim;
  const float* qkv;      // [M, (h + 2 h_kv) hd] pre-RoPE projections
  const float* rope_cs;  // [M, hd]
  float* qr;             // [M, h hd] RoPE'd queries (workspace)
  KvLayout kv;
  int layer;
  int max_ctx;           // host upper bound of (pos + 1) over rows
  int chunk;             // keys per split
  int n_split;           // splits = ceil(max_ctx / chunk)
  float* o_part;         // [M, h, n_split, hd]
  float* ml_part;        // [M, h, n_split, 2]
  float* o;              // [M, h hd]
  uint16_t* xs;          // or null: o also as a stacked operand (put_stacked), stt fragments per k-step
  int stt;
  int32_t* status;
  int seq_bound;         // 1: bound each sequence's keys by its own last row (batches of several sequences)
  // bf16 in-kernel combine (all null: a separate combine kernel adds the
  // parts).  epochs: one word per (sequence, query tile, kv head), zero at
  // first use; a launch reads e and tags every partial word it writes with
  // e + 1 (never 0), and the combining block stores e + 1 once it has read
  // every part.  ll: [M, h, parts <= kLlMaxParts, hd + 2] tagged words, zero
  // at first use: low half the float (hd O values, then max and sum), high
  // half the tag.  counters (one-round launches): one word per (sequence,
  // query tile, kv head), zero between launches; the last block to count
  // combines.
  uint32_t* epochs;
  uint64_t* ll;
  uint32_t* counters;
  // Or null: the weights the next launch streams (the O projection's image,
  // next_w_bytes long).  With the in-kernel combine, every block that does not
  // combine reads up to kNextWeightsPerBlock bytes of its share of them after
  // its partials are out, while the combining blocks finish: the next launch
  // then starts on data already in the last-level cache.
  const unsigned char* next_w;
  uint32_t next_w_bytes;
};
constexpr uint32_t kNextWeightsPerBlock = 48u << 10;
constexpr int kLlMaxParts = 64;  // parts of one head the in-kernel combine takes (one per lane)
// Epoch words a model workspace holds for the attention's in-kernel combine.
size_t attention_counter_count(int n_heads, int n_kv_heads, int max_rows);
// Flagged partial words (uint64) of the in-kernel combine for max_rows rows.
size_t attention_ll_words(int n_heads, int head_dim, int max_rows, int n_split_max);
hipError_t launch_fill_u32(uint32_t* p, size_t n, uint32_t v, hipStream_t s);
int attention_chunk(int dtype, int head_dim);  // keys per split of the attention kernel
int device_compute_units();                    // CUs of the current device (cached)
hipError_t launch_rope_append(const AttnArgs& a, hipStream_t s);
hipError_t launch_attention(const AttnArgs& a, hipStream_t s);

// ------------------------------------------------------------------ sampling / bookkeeping
struct DraftFinishArgs {
  int B, rps, V;
  const float* logits;   // [M, V]
  float temperature;
  uint64_t seed, step;
  const uint64_t* step_dev;  // or null: the step read on the device in place of `step`
  const uint32_t* rand;  // [B] or null
  int slot, gamma;
  float* q_out;          // [B, gamma, V] or null
  int32_t* d_out;
  int ld_d;
  float* logits_out;     // [B, V] or null
  int32_t* status;
  void* scratch;         // sampling_scratch_bytes(B, 1, V) bytes
};
hipError_t launch_draft_finish(const DraftFinishArgs& a, hipStream_t s);

// Scratch of the multi-block softmax / accept / draw kernels for B sequences
// with `rows` distribution rows each over a vocabulary of V.
size_t sampling_scratch_bytes(int B, int rows, int V);

struct AcceptArgs {
  int B, gamma, V, input_kind;
  float temperature;
  const float* p;
  const float* q;
  const int32_t* d;
  int ld_d;
  const uint32_t* rand;
  uint64_t seed, step;
  const uint64_t* step_dev;  // or null: the step read on the device in place of `step`
  int32_t* n_accepted;
  int32_t* next_token;
  int32_t* status;
  void* scratch;         // sampling_scratch_bytes(B, gamma + 1, V) bytes
};
hipError_t launch_accept(const AcceptArgs& a, hipStream_t s);
// The no-allocation accept's static scratch: its size, and its address on the
// current device (looked up on the device's first call).
constexpr size_t kStaticAcceptScratchBytes = SPECDEC_ACCEPT_NOALLOC_SCRATCH_BYTES;
hipError_t static_accept_scratch(void** out);

hipError_t launch_sample(int B, int V, const float* probs, int64_t ld, const uint32_t* rand, uint64_t seed,
                         uint64_t step, int purpose, int index, int32_t* out, hipStream_t s);
hipError_t launch_draw(int B, uint64_t seed, uint64_t step, int purpose, int index, uint32_t* out, hipStream_t s);

struct CommitArgs {
  int B, gamma, role;
  int32_t* len;
  int32_t* pending;
  int32_t* n_pending;
  const int32_t* n_accepted;
  const int32_t* d;
  int ld_d;
  const int32_t* next_token;
  uint64_t* counter;  // the cache's commit counter, +1 per launch
};
hipError_t launch_commit(const CommitArgs& a, hipStream_t s);

// Streaming-read ceiling probe (stream.hip): reads bytes / 1024 KB-chunks of buf.
hipError_t launch_stream_read(const void* buf, size_t bytes, uint32_t* sink, hipStream_t s);

hipError_t launch_kv_copy(const KvLayout& kv, int layer, int b, int pos0, int n, const void* k, const void* v,
                          void* k_out, void* v_out, hipStream_t s);

}  // namespace specdec
