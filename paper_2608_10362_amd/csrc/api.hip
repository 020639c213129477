// C ABI of the speculative-decoding hot path: argument validation, workspace
// carving, and the launch sequence of one forward pass (verify or draft step).
#include <algorithm>
#include <cstring>
#include <vector>

#include "device_common.h"
#include "internal.h"
#include "specdec.h"

using namespace specdec;


struct specdec_model {
  specdec_model_desc desc;
  int n_layers;  // layers this handle runs
  int max_rows, max_ctx;
  const void* embed;
  const void* lm_head;
  const void* final_norm;
  std::vector<const void*> attn_norm, wq, wk, wv, wo, ffn_norm, w_gate, w_up, w_down;
  int wfmt = SPECDEC_WEIGHTS_BF16;  // SPECDEC_WEIGHTS_INT4: the layer matrices above are INT4 code images
  std::vector<const uint16_t*> sq, sk, sv, so, sg, su, sd;  // ... and these their group scales
  // workspace carve
  RowDesc* rows;
  float* rope_cs;
  float* h;
  float* xg;
  float* ss;
  int ss_ld, ss_parts_max;
  float* qkv;
  float* qr;
  float* o_part;
  float* ml_part;
  float* o;
  float* u;
  float* logits;
  void* samp;  // scratch of the draft's softmax / draw kernels
  uint16_t* xs_d = nullptr;  // bf16: the stacked x operand of the d_model-column GEMMs (passes of <= 16 rows)
  uint16_t* xs_f = nullptr;  // bf16: the stacked attention output (the O projection's x), then SwiGLU output
  float* ypart = nullptr;  // split-K partials of the wide residual GEMMs (passes of more than 64 rows)
  uint32_t* attn_ctr = nullptr;           // bf16: the attention combine's epochs
  uint32_t* attn_cnt = nullptr;           // bf16: the one-round attention combine's arrival counters
  uint64_t* attn_ll = nullptr;            // bf16: the attention combine's tagged partial words
  size_t attn_ll_words = 0;
  mutable bool attn_ctr_ready = false;    // set once all three have been zeroed on a stream
  int chunk, n_split_max;
  // per-layer launches of the last forward pass, for specdec_time_kernel
  // (entry l: layer l; the head and the embedding have one)
  mutable bool rec_valid[SPECDEC_KERNEL_KINDS] = {};
  mutable std::vector<GemmArgs> rec_gemm[SPECDEC_KERNEL_KINDS];
  mutable int rec_rows[SPECDEC_KERNEL_KINDS];
  mutable std::vector<AttnArgs> rec_attn;
  mutable RowsArgs rec_embed;
};

namespace {

// ---------------------------------------------------------------- kernel timing hook
struct Timing {
  bool enabled = false;
  std::vector<hipEvent_t> pool;
  struct Rec { int kind; hipEvent_t b, e; };
  std::vector<Rec> recs;
  hipEvent_t get() {
    if (!pool.empty()) { hipEvent_t ev = pool.back(); pool.pop_back(); return ev; }
    hipEvent_t ev = nullptr;
    if (hipEventCreate(&ev) != hipSuccess) return nullptr;
    return ev;
  }
};
Timing g_timing;

// Brackets the launches of one kernel kind with events when timing is on.
struct Timed {
  int kind;
  hipStream_t s;
  hipEvent_t b = nullptr;
  Timed(int k, hipStream_t st) : kind(k), s(st) {
    if (g_timing.enabled && (b = g_timing.get()) && hipEventRecord(b, s) != hipSuccess) {
      g_timing.pool.push_back(b);
      b = nullptr;
    }
  }
  ~Timed() {
    if (!b) return;
    hipEvent_t e = g_timing.get();
    if (!e) { g_timing.pool.push_back(b); return; }
    if (hipEventRecord(e, s) != hipSuccess) {
      g_timing.pool.push_back(b);
      g_timing.pool.push_back(e);
      return;
    }
    g_timing.recs.push_back({kind, b, e});
  }
};

constexpr size_t kAlign = 256;
size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

int elem_bytes(int dtype) { return dtype == SPECDEC_BF16 ? 2 : 4; }

// Workspace layout (in order); shared by specdec_workspace_bytes and create.
struct WsLayout {
  size_t rows, rope, h, xg, ss, qkv, qr, o_part, ml_part, o, u, logits, samp, xs_d, xs_f, ypart, ctr, cnt, ll, total;
  int ss_parts, chunk, n_split;
};

WsLayout ws_layout(const specdec_model_desc* d, int max_rows, int max_ctx) {
  WsLayout w{};
  const size_t R = (size_t)max_rows;
  const int hd = d->head_dim, H = d->n_heads, G = d->n_kv_heads;
  // (passes of up to max_rows rows: the skinny and, above kMaxGemmRows, the wide partial counts)
  w.ss_parts = std::max(1, gemm_row_blocks(d->dtype, EPI_RESID, d->d_model, std::min(max_rows, kMaxGemmRows)));
  const bool wide = gemm_wide(d->dtype, max_rows);
  if (wide) w.ss_parts = std::max(w.ss_parts, gemm_row_blocks(d->dtype, EPI_RESID, d->d_model, max_rows));
  w.chunk = attention_chunk(d->dtype, hd);
  w.n_split = (max_ctx + w.chunk - 1) / w.chunk;
  size_t off = 0;
  auto take = [&](size_t bytes) { size_t at = off; off = align_up(off + bytes); return at; };
  w.rows = take(R * sizeof(RowDesc));
  w.rope = take(R * hd * 4);
  w.h = take(R * d->d_model * 4);
  w.xg = take(R * d->d_model * 4);
  w.ss = take((size_t)w.ss_parts * R * 4);
  w.qkv = take(R * (H + 2 * G) * hd * 4);
  w.qr = take(R * H * hd * 4);
  w.o_part = take(R * H * (size_t)w.n_split * hd * 4);
  w.ml_part = take(R * H * (size_t)w.n_split * 2 * 4);
  w.o = take(R * H * hd * 4);
  w.u = take(R * d->ffn_dim * 4);
  w.logits = take(R * d->vocab * 4);
  w.samp = take(sampling_scratch_bytes(max_rows, 1, d->vocab));
  // (stacked operands: two 1 KB fragments per 32 columns)
  w.xs_d = take(d->dtype == SPECDEC_BF16 ? (size_t)(d->d_model + 31) / 32 * 2048 : 0);
  w.xs_f = take(d->dtype == SPECDEC_BF16 ? (size_t)(std::max(d->ffn_dim, H * hd) + 31) / 32 * 2048 : 0);
  w.ypart = take(wide ? wide_ypart_floats(d->d_model) * 4 : 0);
  w.ctr = take(d->dtype == SPECDEC_BF16 ? attention_counter_count(H, G, max_rows) * 4 : 0);
  w.cnt = take(d->dtype == SPECDEC_BF16 ? attention_counter_count(H, G, max_rows) * 4 : 0);
  w.ll = take(d->dtype == SPECDEC_BF16 ? attention_ll_words(H, hd, max_rows, w.n_split) * 8 : 0);
  w.total = off;
  return w;
}

specdec_status check_desc(const specdec_model_desc* d) {
  if (!d) return SPECDEC_ERR_INVALID_ARG;
  if (d->dtype != SPECDEC_F32 && d->dtype != SPECDEC_BF16) return SPECDEC_ERR_INVALID_ARG;
  if (d->n_layers <= 0 || d->d_model <= 0 || d->n_heads <= 0 || d->n_kv_heads <= 0 || d->head_dim <= 0 ||
      d->ffn_dim <= 0 || d->vocab <= 0 || !(d->rms_eps >= 0.f) || !(d->rope_base > 0.f))
    return SPECDEC_ERR_INVALID_ARG;
  if (d->d_model % 64 || d->ffn_dim % 32 || d->vocab % 16 || d->n_heads % d->n_kv_heads) return SPECDEC_ERR_SHAPE;
  if (d->head_dim != 32 && d->head_dim != 64 && d->head_dim != 128) return SPECDEC_ERR_SHAPE;
  if ((d->n_heads * d->head_dim) % 64 || (d->n_kv_heads * d->head_dim) % 32) return SPECDEC_ERR_SHAPE;
  return SPECDEC_OK;
}

// The last HIP error a call of this thread returned SPECDEC_ERR_HIP for.
thread_local hipError_t g_last_hip_error = hipSuccess;

specdec_status hip_status(hipError_t e) {
  if (e == hipSuccess) return SPECDEC_OK;
  g_last_hip_error = e;
  return SPECDEC_ERR_HIP;
}

// Packed image: LM head, then per layer Wq, Wk, Wv, Wo, W_gate, W_up, W_down,
// each 256-byte aligned.  Returns the bytes and the (N, K, byte offset) list.
struct PackedMat {
  int N, K;
  size_t off;
  size_t soff = 0;  // INT4 matrices: byte offset of the group scales
};
size_t image_layout(const specdec_model_desc* d, int n_layers, std::vector<PackedMat>* mats) {
  const int q = d->n_heads * d->head_dim, kv = d->n_kv_heads * d->head_dim;
  size_t off = 0;
  auto add = [&](int N, int K) {
    if (mats) mats->push_back(PackedMat{N, K, off});
    off = align_up(off + packed_elems(N, K) * 2);
  };
  add(d->vocab, d->d_model);
  for (int l = 0; l < n_layers; ++l) {
    add(q, d->d_model);
    add(kv, d->d_model);
    add(kv, d->d_model);
    add(d->d_model, q);
    add(d->ffn_dim, d->d_model);
    add(d->ffn_dim, d->d_model);
    add(d->d_model, d->ffn_dim);
  }
  return off;
}

// INT4 image: the LM head in bf16 (as above), then per layer the same seven
// matrices as INT4 code fragments followed by their group scales.
size_t image_layout_int4(const specdec_model_desc* d, int n_layers, std::vector<PackedMat>* mats) {
  const int q = d->n_heads * d->head_dim, kv = d->n_kv_heads * d->head_dim;
  size_t off = 0;
  if (mats) mats->push_back(PackedMat{d->vocab, d->d_model, off});
  off = align_up(off + packed_elems(d->vocab, d->d_model) * 2);
  auto add = [&](int N, int K) {
    PackedMat m{N, K, off};
    off = align_up(off + packed_int4_frag_bytes(N, K));
    m.soff = off;
    off = align_up(off + packed_int4_scale_bytes(N, K));
    if (mats) mats->push_back(m);
  };
  for (int l = 0; l < n_layers; ++l) {
    add(q, d->d_model);
    add(kv, d->d_model);
    add(kv, d->d_model);
    add(d->d_model, q);
    add(d->ffn_dim, d->d_model);
    add(d->ffn_dim, d->d_model);
    add(d->d_model, d->ffn_dim);
  }
  return off;
}

size_t image_bytes(const specdec_model_desc* d, int n_layers, int fmt, std::vector<PackedMat>* mats) {
  return fmt == SPECDEC_WEIGHTS_INT4 ? image_layout_int4(d, n_layers, mats) : image_layout(d, n_layers, mats);
}

#define SD_TRY(expr)                                   \
  do {                                                 \
    hipError_t _e = (expr);                            \
    if (_e != hipSuccess) return hip_status(_e);       \
  } while (0)

int32_t* kv_len(const specdec_kv* kv) { return kv->state; }
int32_t* kv_pending(const specdec_kv* kv) { return kv->state + kv->batch; }
int32_t* kv_npending(const specdec_kv* kv) { return kv->state + 3 * kv->batch; }
int32_t* kv_status(const specdec_kv* kv) { return kv->state + 4 * kv->batch; }
uint64_t* kv_counter(const specdec_kv* kv) { return reinterpret_cast<uint64_t*>(kv->state + 4 * kv->batch + 2); }
bool misaligned8(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 7u) != 0; }

KvLayout kv_layout(const specdec_kv* kv) {
  return KvLayout{kv->data, kv->batch, kv->capacity, kv->n_kv_heads, kv->head_dim, kv->dtype};
}

specdec_status check_kv(const specdec_model* m, const specdec_kv* kv) {
  if (!m || !kv || !kv->data || !kv->state) return SPECDEC_ERR_INVALID_ARG;
  if (kv->n_layers < m->n_layers || kv->n_kv_heads != m->desc.n_kv_heads || kv->head_dim != m->desc.head_dim ||
      kv->dtype != m->desc.dtype)
    return SPECDEC_ERR_SHAPE;
  return SPECDEC_OK;
}

// Runs GEMM `g` over the rows [0, M) in launches of at most gemm_launch_rows rows
// (the kernel family is chosen by the whole pass's M, so every launch of a pass
// writes the same number of ss partials).
hipError_t gemm_rows(int dtype, GemmArgs g, int M, hipStream_t s) {
  const int step = gemm_launch_rows(dtype, M);
  g.wide = gemm_wide(dtype, M);
  for (int m0 = 0; m0 < M; m0 += step) {
    GemmArgs c = g;
    c.M = std::min(step, M - m0);
    c.x = g.x + (size_t)m0 * g.ldx;
    if (g.out) c.out = g.out + (size_t)m0 * g.ldo;
    if (g.rows) c.rows = g.rows + m0;
    if (g.rope_cs) c.rope_cs = g.rope_cs + (size_t)m0 * g.head_dim;
    if (g.qr) c.qr = g.qr + (size_t)m0 * g.n_heads * g.head_dim;
    if (g.ss_in) c.ss_in = g.ss_in + m0;
    if (g.ss_out) c.ss_out = g.ss_out + m0;
    if (g.xg_out) c.xg_out = g.xg_out + (size_t)m0 * g.ldo;
    hipError_t e = launch_gemm(dtype, c, s);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

// One forward pass over M = B*rps rows described by `ra` (mode, token source),
// writing logits [M, V] to `logits`.  ctx_bound: host upper bound of pos+1.
specdec_status forward(const specdec_model* m, specdec_kv* kv, RowsArgs ra, int ctx_bound, float* logits,
                       hipStream_t s) {
  const specdec_model_desc& d = m->desc;
  const int M = ra.M, dt = d.dtype;
  const int H = d.n_heads, G = d.n_kv_heads, hd = d.head_dim;
  if (M > m->max_rows) return SPECDEC_ERR_SHAPE;
  ctx_bound = std::min(ctx_bound, kv->capacity);
  const int n_split = (ctx_bound + m->chunk - 1) / m->chunk;
  if (n_split > m->n_split_max) return SPECDEC_ERR_SHAPE;

  ra.len = kv_len(kv);
  ra.pending = kv_pending(kv);
  ra.n_pending = kv_npending(kv);
  ra.status = kv_status(kv);
  ra.capacity = kv->capacity;
  ra.vocab = d.vocab;
  ra.d_model = d.d_model;
  ra.head_dim = hd;
  ra.rope_base = d.rope_base;
  ra.embed = m->embed;
  ra.gain = m->attn_norm[0];
  ra.xg = m->xg;
  ra.rows = m->rows;
  ra.rope_cs = m->rope_cs;
  ra.h = m->h;
  ra.ss = m->ss;
  // Passes of at most 16 rows on bf16 weights hand x from kernel to kernel also
  // as a stacked operand (put_stacked): the skinny GEMMs then read one 16-byte
  // fragment per k-step (two when M > 8) instead of two float32 loads per row
  // tile.
  const bool stk = dt == SPECDEC_BF16 && m->wfmt != SPECDEC_WEIGHTS_INT4 && M <= 16 && m->xs_d;
  const int stt = M <= 8 ? 1 : 2;
  ra.xs = stk ? m->xs_d : nullptr;
  ra.stt = stt;
  {
    Timed t(SPECDEC_KERNEL_EMBED, s);
    SD_TRY(launch_rows_embed(dt, ra, s));
  }
  m->rec_embed = ra;
  m->rec_valid[SPECDEC_KERNEL_EMBED] = true;
  auto rec = [&](int kind, int layer, const GemmArgs& g) {
    std::vector<GemmArgs>& v = m->rec_gemm[kind];
    v.resize((size_t)layer + 1);
    v[(size_t)layer] = g;
    m->rec_rows[kind] = M;
    m->rec_valid[kind] = true;
  };

  GemmArgs base{};
  base.eps = d.rms_eps;
  base.ss_ld = m->ss_ld;
  base.gain_bf16 = dt == SPECDEC_BF16;
  base.ypart = m->ypart;
  base.stt = stt;
  int n_ss = 1;
  const int n_resid_blocks = gemm_row_blocks(dt, EPI_RESID, d.d_model, M);

  AttnArgs at{};
  at.rows = m->rows;
  at.M = M;
  at.rps = ra.rps;
  at.n_heads = H;
  at.n_kv_heads = G;
  at.head_dim = hd;
  at.qkv = m->qkv;
  at.rope_cs = m->rope_cs;
  at.qr = m->qr;
  at.kv = kv_layout(kv);
  at.max_ctx = ctx_bound;
  at.chunk = m->chunk;
  at.n_split = n_split;
  at.o_part = m->o_part;
  at.ml_part = m->ml_part;
  at.o = m->o;
  at.status = kv_status(kv);
  at.seq_bound = M / ra.rps > 1;
  if (m->attn_ctr && !m->attn_ctr_ready) {  // (fill kernels: a capturing caller may record them)
    SD_TRY(launch_fill_u32(m->attn_ctr, attention_counter_count(H, G, m->max_rows), 0u, s));
    SD_TRY(launch_fill_u32(m->attn_cnt, attention_counter_count(H, G, m->max_rows), 0u, s));
    SD_TRY(launch_fill_u32((uint32_t*)m->attn_ll, 2 * m->attn_ll_words, 0u, s));
    m->attn_ctr_ready = true;
  }
  at.epochs = m->attn_ctr;
  at.counters = m->attn_cnt;
  at.ll = m->attn_ll;
  at.xs = stk ? m->xs_f : nullptr;
  at.stt = stt;

  for (int l = 0; l < m->n_layers; ++l) {
    GemmArgs q = base;  // RMSNorm + Q|K|V projections
    q.x = m->xg; q.ldx = d.d_model; q.ss_in = m->ss; q.n_ss = n_ss;
    q.K = d.d_model;
    q.w[0] = m->wq[l]; q.w[1] = m->wk[l]; q.w[2] = m->wv[l];
    q.n_seg[0] = H * hd; q.n_seg[1] = G * hd; q.n_seg[2] = G * hd;
    q.n_rows = (H + 2 * G) * hd; q.kind = EPI_STORE; q.out = m->qkv; q.ldo = (H + 2 * G) * hd;
    if (dt == SPECDEC_BF16) {  // RoPE, the query store and the KV append run in the GEMM epilogue
      q.kind = EPI_QKV;  // (q.out stays the qkv scratch: passes of more than 128 rows store the projections there
                         // and apply RoPE and the KV append in rope_append_kernel)
      q.rows = m->rows; q.rope_cs = m->rope_cs; q.qr = m->qr; q.kv = kv_layout(kv); q.layer = l;
      q.n_heads = H; q.n_kv_heads = G; q.head_dim = hd;
    }
    const bool q4 = m->wfmt == SPECDEC_WEIGHTS_INT4;
    if (q4) { q.q4 = 1; q.wscale[0] = m->sq[l]; q.wscale[1] = m->sk[l]; q.wscale[2] = m->sv[l]; }
    if (stk) q.xs = m->xs_d;
    {
      Timed t(SPECDEC_KERNEL_QKV, s);
      SD_TRY(gemm_rows(dt, q, M, s));
    }
    rec(SPECDEC_KERNEL_QKV, l, q);

    at.layer = l;
    // (the O projection's image follows the attention: bf16 fragments, or the INT4 code blocks)
    at.next_w = dt == SPECDEC_BF16 ? (const unsigned char*)m->wo[l] : nullptr;
    at.next_w_bytes = (uint32_t)(m->wfmt == SPECDEC_WEIGHTS_INT4 ? packed_int4_frag_bytes(d.d_model, H * hd)
                                                                   : packed_elems(d.d_model, H * hd) * 2);
    if (dt != SPECDEC_BF16) {
      Timed t(SPECDEC_KERNEL_ROPE_APPEND, s);
      SD_TRY(launch_rope_append(at, s));
    }
    {
      Timed t(SPECDEC_KERNEL_ATTENTION, s);
      SD_TRY(launch_attention(at, s));
    }
    m->rec_attn.resize((size_t)l + 1);
    m->rec_attn[(size_t)l] = at;
    if (l == 0) {
      m->rec_valid[SPECDEC_KERNEL_ATTENTION] = true;
      m->rec_valid[SPECDEC_KERNEL_ROPE_APPEND] = dt != SPECDEC_BF16;
    }

    GemmArgs o = base;  // O projection + residual
    o.x = m->o; o.ldx = H * hd; o.K = H * hd;
    o.w[0] = m->wo[l]; o.n_seg[0] = d.d_model; o.n_rows = d.d_model; o.kind = EPI_RESID;
    o.out = m->h; o.ldo = d.d_model; o.ss_out = m->ss; o.xg_out = m->xg; o.gain_out = m->ffn_norm[l];
    if (q4) { o.q4 = 1; o.wscale[0] = m->so[l]; }
    if (stk) { o.xs = m->xs_f; o.xs_out = m->xs_d; }
    {
      Timed t(SPECDEC_KERNEL_O_PROJ, s);
      SD_TRY(gemm_rows(dt, o, M, s));
    }
    rec(SPECDEC_KERNEL_O_PROJ, l, o);
    n_ss = n_resid_blocks;

    GemmArgs gu = base;  // RMSNorm + gate|up + SwiGLU
    gu.x = m->xg; gu.ldx = d.d_model; gu.ss_in = m->ss; gu.n_ss = n_ss;
    gu.K = d.d_model;
    gu.w[0] = m->w_gate[l]; gu.w[1] = m->w_up[l]; gu.n_seg[0] = d.ffn_dim; gu.n_seg[1] = d.ffn_dim;
    gu.n_rows = d.ffn_dim; gu.kind = EPI_SWIGLU; gu.out = m->u; gu.ldo = d.ffn_dim;
    if (q4) { gu.q4 = 1; gu.wscale[0] = m->sg[l]; gu.wscale[1] = m->su[l]; }
    if (stk) { gu.xs = m->xs_d; gu.xs_out = m->xs_f; }
    {
      Timed t(SPECDEC_KERNEL_GATE_UP, s);
      SD_TRY(gemm_rows(dt, gu, M, s));
    }
    rec(SPECDEC_KERNEL_GATE_UP, l, gu);

    GemmArgs dn = base;  // down projection + residual
    dn.x = m->u; dn.ldx = d.ffn_dim; dn.K = d.ffn_dim;
    dn.w[0] = m->w_down[l]; dn.n_seg[0] = d.d_model; dn.n_rows = d.d_model; dn.kind = EPI_RESID;
    dn.out = m->h; dn.ldo = d.d_model; dn.ss_out = m->ss; dn.xg_out = m->xg;
    dn.gain_out = l + 1 < m->n_layers ? m->attn_norm[l + 1] : m->final_norm;
    if (q4) { dn.q4 = 1; dn.wscale[0] = m->sd[l]; }
    if (stk) { dn.xs = m->xs_f; dn.xs_out = m->xs_d; }
    {
      Timed t(SPECDEC_KERNEL_DOWN, s);
      SD_TRY(gemm_rows(dt, dn, M, s));
    }
    rec(SPECDEC_KERNEL_DOWN, l, dn);
  }

  GemmArgs hd_ = base;  // final RMSNorm + LM head
  hd_.x = m->xg; hd_.ldx = d.d_model; hd_.ss_in = m->ss; hd_.n_ss = n_ss;
  hd_.K = d.d_model; hd_.w[0] = m->lm_head; hd_.n_seg[0] = d.vocab; hd_.n_rows = d.vocab;
  hd_.kind = EPI_STORE; hd_.out = logits; hd_.ldo = d.vocab;
  if (stk) hd_.xs = m->xs_d;
  {
    Timed t(SPECDEC_KERNEL_LM_HEAD, s);
    SD_TRY(gemm_rows(dt, hd_, M, s));
  }
  rec(SPECDEC_KERNEL_LM_HEAD, 0, hd_);
  return SPECDEC_OK;
}

__global__ void prefill_finish_kernel(int B, int n, const int32_t* tokens, int32_t* len, int32_t* pending,
                                      int32_t* n_pending) {
  for (int b = threadIdx.x; b < B; b += blockDim.x) {
    len[b] += n - 1;
    pending[2 * b] = 0;
    pending[2 * b + 1] = tokens[(size_t)b * n + n - 1];
    n_pending[b] = 1;
  }
}

}  // namespace

extern "C" {

size_t specdec_workspace_bytes(const specdec_model_desc* desc, int32_t max_rows, int32_t max_ctx) {
  if (check_desc(desc) != SPECDEC_OK || max_rows <= 0 || max_ctx <= 0) return 0;
  return ws_layout(desc, max_rows, max_ctx).total;
}

size_t specdec_packed_bytes_fmt(const specdec_model_desc* desc, int32_t n_layers_used, int32_t format) {
  if (check_desc(desc) != SPECDEC_OK || n_layers_used <= 0 || n_layers_used > desc->n_layers) return 0;
  if (desc->dtype != SPECDEC_BF16) return 0;
  if (format != SPECDEC_WEIGHTS_BF16 && format != SPECDEC_WEIGHTS_INT4) return 0;
  return image_bytes(desc, n_layers_used, format, nullptr);
}

size_t specdec_packed_bytes(const specdec_model_desc* desc, int32_t n_layers_used) {
  return specdec_packed_bytes_fmt(desc, n_layers_used, SPECDEC_WEIGHTS_BF16);
}

specdec_status specdec_pack_weights_fmt(const specdec_model_desc* desc, const specdec_weights* w,
                                        int32_t n_layers_used, int32_t format, void* packed, size_t packed_bytes,
                                        void* stream) {
  specdec_status st = check_desc(desc);
  if (st != SPECDEC_OK) return st;
  if (desc->dtype != SPECDEC_BF16) return SPECDEC_ERR_UNSUPPORTED;
  if (format != SPECDEC_WEIGHTS_BF16 && format != SPECDEC_WEIGHTS_INT4) return SPECDEC_ERR_INVALID_ARG;
  if (!w || !packed || n_layers_used <= 0 || n_layers_used > desc->n_layers) return SPECDEC_ERR_INVALID_ARG;
  if ((uintptr_t)packed % kAlign) return SPECDEC_ERR_INVALID_ARG;
  std::vector<PackedMat> mats;
  if (packed_bytes < image_bytes(desc, n_layers_used, format, &mats)) return SPECDEC_ERR_INVALID_ARG;
  if (!w->lm_head || !w->wq || !w->wk || !w->wv || !w->wo || !w->w_gate || !w->w_up || !w->w_down)
    return SPECDEC_ERR_INVALID_ARG;
  std::vector<const void*> src;
  src.push_back(w->lm_head);
  for (int l = 0; l < n_layers_used; ++l) {
    const void* m[7] = {w->wq[l], w->wk[l], w->wv[l], w->wo[l], w->w_gate[l], w->w_up[l], w->w_down[l]};
    for (const void* p : m) {
      if (!p) return SPECDEC_ERR_INVALID_ARG;
      src.push_back(p);
    }
  }
  hipStream_t s = (hipStream_t)stream;
  for (size_t i = 0; i < mats.size(); ++i) {
    // Wq and Wk (matrices 1 and 2 of each layer's seven) carry the RoPE pair order
    const int in_layer = i == 0 ? -1 : (int)((i - 1) % 7);
    const int rope_hd = in_layer == 0 || in_layer == 1 ? desc->head_dim : 0;
    if (format == SPECDEC_WEIGHTS_INT4 && i > 0)
      SD_TRY(launch_pack_int4(src[i], (char*)packed + mats[i].off, (char*)packed + mats[i].soff, mats[i].N, mats[i].K,
                              rope_hd, s));
    else
      SD_TRY(launch_pack(src[i], (char*)packed + mats[i].off, mats[i].N, mats[i].K, rope_hd, s));
  }
  return SPECDEC_OK;
}

specdec_status specdec_pack_weights(const specdec_model_desc* desc, const specdec_weights* w, int32_t n_layers_used,
                                    void* packed, size_t packed_bytes, void* stream) {
  return specdec_pack_weights_fmt(desc, w, n_layers_used, SPECDEC_WEIGHTS_BF16, packed, packed_bytes, stream);
}

specdec_status specdec_model_create(const specdec_model_desc* desc, const specdec_weights* w, int32_t n_layers_used,
                                    const void* packed, size_t packed_bytes, int32_t max_rows, int32_t max_ctx,
                                    void* workspace, size_t workspace_bytes, specdec_model** out) {
  return specdec_model_create_fmt(desc, w, n_layers_used, SPECDEC_WEIGHTS_BF16, packed, packed_bytes, max_rows,
                                  max_ctx, workspace, workspace_bytes, out);
}

specdec_status specdec_model_create_fmt(const specdec_model_desc* desc, const specdec_weights* w,
                                        int32_t n_layers_used, int32_t format, const void* packed,
                                        size_t packed_bytes, int32_t max_rows, int32_t max_ctx, void* workspace,
                                        size_t workspace_bytes, specdec_model** out) {
  if (!out) return SPECDEC_ERR_INVALID_ARG;
  *out = nullptr;
  specdec_status st = check_desc(desc);
  if (st != SPECDEC_OK) return st;
  if (!w || !workspace || max_rows <= 0 || max_ctx <= 0) return SPECDEC_ERR_INVALID_ARG;
  if (n_layers_used <= 0 || n_layers_used > desc->n_layers) return SPECDEC_ERR_INVALID_ARG;
  if ((uintptr_t)workspace % kAlign) return SPECDEC_ERR_INVALID_ARG;
  // passes of more than 64 rows sum one RMSNorm partial per 128 columns in a wave: d_model <= 8192
  if (gemm_wide(desc->dtype, max_rows) && desc->d_model > 8192) return SPECDEC_ERR_SHAPE;
  const WsLayout L = ws_layout(desc, max_rows, max_ctx);
  if (workspace_bytes < L.total) return SPECDEC_ERR_INVALID_ARG;
  const bool bf16 = desc->dtype == SPECDEC_BF16;
  if (format != SPECDEC_WEIGHTS_BF16 && format != SPECDEC_WEIGHTS_INT4) return SPECDEC_ERR_INVALID_ARG;
  // INT4 layer weights run the skinny GEMMs only: passes of at most 64 rows
  if (format == SPECDEC_WEIGHTS_INT4 && (!bf16 || max_rows > kMaxGemmRows)) return SPECDEC_ERR_UNSUPPORTED;
  std::vector<PackedMat> mats;
  if (bf16) {
    if (!packed || (uintptr_t)packed % kAlign) return SPECDEC_ERR_INVALID_ARG;
    if (packed_bytes < image_bytes(desc, n_layers_used, format, &mats)) return SPECDEC_ERR_INVALID_ARG;
  } else if (packed) {
    return SPECDEC_ERR_INVALID_ARG;
  }
  if (!w->embed || !w->final_norm || !w->attn_norm || !w->ffn_norm) return SPECDEC_ERR_INVALID_ARG;
  if (!bf16 && (!w->lm_head || !w->wq || !w->wk || !w->wv || !w->wo || !w->w_gate || !w->w_up || !w->w_down))
    return SPECDEC_ERR_INVALID_ARG;
  for (int l = 0; l < n_layers_used; ++l) {
    if (!w->attn_norm[l] || !w->ffn_norm[l]) return SPECDEC_ERR_INVALID_ARG;
    if (!bf16 && (!w->wq[l] || !w->wk[l] || !w->wv[l] || !w->wo[l] || !w->w_gate[l] || !w->w_up[l] ||
                  !w->w_down[l]))
      return SPECDEC_ERR_INVALID_ARG;
  }

  specdec_model* m = new specdec_model();
  m->desc = *desc;
  m->n_layers = n_layers_used;
  m->max_rows = max_rows;
  m->max_ctx = max_ctx;
  m->embed = w->embed;
  m->final_norm = w->final_norm;
  m->attn_norm.assign(w->attn_norm, w->attn_norm + n_layers_used);
  m->ffn_norm.assign(w->ffn_norm, w->ffn_norm + n_layers_used);
  if (bf16) {  // matrices from the packed image
    const char* img = (const char*)packed;
    m->lm_head = img + mats[0].off;
    for (int l = 0; l < n_layers_used; ++l) {
      const PackedMat* p = &mats[1 + 7 * l];
      m->wq.push_back(img + p[0].off);
      m->wk.push_back(img + p[1].off);
      m->wv.push_back(img + p[2].off);
      m->wo.push_back(img + p[3].off);
      m->w_gate.push_back(img + p[4].off);
      m->w_up.push_back(img + p[5].off);
      m->w_down.push_back(img + p[6].off);
      if (format == SPECDEC_WEIGHTS_INT4) {
        auto sc = [&](int j) { return (const uint16_t*)(img + p[j].soff); };
        m->sq.push_back(sc(0)); m->sk.push_back(sc(1)); m->sv.push_back(sc(2)); m->so.push_back(sc(3));
        m->sg.push_back(sc(4)); m->su.push_back(sc(5)); m->sd.push_back(sc(6));
      }
    }
    m->wfmt = format;
  } else {
    m->lm_head = w->lm_head;
    m->wq.assign(w->wq, w->wq + n_layers_used);
    m->wk.assign(w->wk, w->wk + n_layers_used);
    m->wv.assign(w->wv, w->wv + n_layers_used);
    m->wo.assign(w->wo, w->wo + n_layers_used);
    m->w_gate.assign(w->w_gate, w->w_gate + n_layers_used);
    m->w_up.assign(w->w_up, w->w_up + n_layers_used);
    m->w_down.assign(w->w_down, w->w_down + n_layers_used);
  }
  char* base = (char*)workspace;
  m->rows = (RowDesc*)(base + L.rows);
  m->rope_cs = (float*)(base + L.rope);
  m->h = (float*)(base + L.h);
  m->xg = (float*)(base + L.xg);
  m->ss = (float*)(base + L.ss);
  m->ss_ld = max_rows;
  m->ss_parts_max = L.ss_parts;
  m->qkv = (float*)(base + L.qkv);
  m->qr = (float*)(base + L.qr);
  m->o_part = (float*)(base + L.o_part);
  m->ml_part = (float*)(base + L.ml_part);
  m->o = (float*)(base + L.o);
  m->u = (float*)(base + L.u);
  m->logits = (float*)(base + L.logits);
  m->samp = base + L.samp;
  m->xs_d = desc->dtype == SPECDEC_BF16 ? (uint16_t*)(base + L.xs_d) : nullptr;
  m->xs_f = desc->dtype == SPECDEC_BF16 ? (uint16_t*)(base + L.xs_f) : nullptr;
  m->ypart = gemm_wide(desc->dtype, max_rows) ? (float*)(base + L.ypart) : nullptr;
  m->attn_ctr = desc->dtype == SPECDEC_BF16 ? (uint32_t*)(base + L.ctr) : nullptr;
  m->attn_cnt = desc->dtype == SPECDEC_BF16 ? (uint32_t*)(base + L.cnt) : nullptr;
  m->attn_ll = desc->dtype == SPECDEC_BF16 ? (uint64_t*)(base + L.ll) : nullptr;
  m->attn_ll_words = desc->dtype == SPECDEC_BF16 ? attention_ll_words(desc->n_heads, desc->head_dim, max_rows, L.n_split) : 0;
  m->chunk = L.chunk;
  m->n_split_max = L.n_split;
  *out = m;
  return SPECDEC_OK;
}

void specdec_model_destroy(specdec_model* model) { delete model; }

size_t specdec_kv_bytes(const specdec_model_desc* desc, int32_t n_layers_used, int32_t batch, int32_t capacity) {
  if (check_desc(desc) != SPECDEC_OK || n_layers_used <= 0 || batch <= 0 || capacity <= 0) return 0;
  return (size_t)n_layers_used * batch * desc->n_kv_heads * 2 * (size_t)capacity * desc->head_dim *
         elem_bytes(desc->dtype);
}

int32_t specdec_kv_state_count(int32_t batch) { return batch > 0 ? 4 * batch + 4 : 0; }

specdec_status specdec_kv_init(specdec_kv* kv, const specdec_model* model, int32_t batch, int32_t capacity,
                               void* data, size_t data_bytes, int32_t* state, void* stream) {
  if (!kv || !model || !data || !state || batch <= 0 || capacity <= 0 || misaligned8(state))
    return SPECDEC_ERR_INVALID_ARG;
  if (capacity % 64) return SPECDEC_ERR_SHAPE;
  if (data_bytes < specdec_kv_bytes(&model->desc, model->n_layers, batch, capacity)) return SPECDEC_ERR_INVALID_ARG;
  kv->data = data;
  kv->state = state;
  kv->batch = batch;
  kv->capacity = capacity;
  kv->n_layers = model->n_layers;
  kv->n_kv_heads = model->desc.n_kv_heads;
  kv->head_dim = model->desc.head_dim;
  kv->dtype = model->desc.dtype;
  kv->len_upper = 0;
  return hip_status(hipMemsetAsync(state, 0, sizeof(int32_t) * specdec_kv_state_count(batch), (hipStream_t)stream));
}

specdec_status specdec_kv_write_context(specdec_kv* kv, int32_t layer, int32_t b, int32_t pos0, int32_t n,
                                        const void* k, const void* v, void* stream) {
  if (!kv || !kv->data || !k || !v || layer < 0 || layer >= kv->n_layers || b < 0 || b >= kv->batch || pos0 < 0 ||
      n < 0)
    return SPECDEC_ERR_INVALID_ARG;
  if (pos0 + n > kv->capacity) return SPECDEC_ERR_KV_CAPACITY;
  return hip_status(launch_kv_copy(kv_layout(kv), layer, b, pos0, n, k, v, nullptr, nullptr, (hipStream_t)stream));
}

specdec_status specdec_kv_read_context(const specdec_kv* kv, int32_t layer, int32_t b, int32_t pos0, int32_t n,
                                       void* k, void* v, void* stream) {
  if (!kv || !kv->data || !k || !v || layer < 0 || layer >= kv->n_layers || b < 0 || b >= kv->batch || pos0 < 0 ||
      n < 0)
    return SPECDEC_ERR_INVALID_ARG;
  if (pos0 + n > kv->capacity) return SPECDEC_ERR_KV_CAPACITY;
  return hip_status(launch_kv_copy(kv_layout(kv), layer, b, pos0, n, nullptr, nullptr, k, v, (hipStream_t)stream));
}

specdec_status specdec_kv_set_state(specdec_kv* kv, const int32_t* len, const int32_t* pending,
                                    const int32_t* n_pending, void* stream) {
  if (!kv || !kv->state || !len || !pending || !n_pending) return SPECDEC_ERR_INVALID_ARG;
  const int B = kv->batch;
  std::vector<int32_t> host(specdec_kv_state_count(B), 0);
  int64_t mx = 0;
  for (int b = 0; b < B; ++b) {
    if (len[b] < 0 || len[b] > kv->capacity || n_pending[b] < 1 || n_pending[b] > 2) return SPECDEC_ERR_INVALID_ARG;
    host[b] = len[b];
    host[B + 2 * b] = pending[2 * b];
    host[B + 2 * b + 1] = pending[2 * b + 1];
    host[3 * B + b] = n_pending[b];
    mx = std::max<int64_t>(mx, len[b]);
  }
  hipStream_t s = (hipStream_t)stream;
  // lengths, pending tokens and the status word; the commit counter is kept
  SD_TRY(hipMemcpyAsync(kv->state, host.data(), (4 * (size_t)B + 1) * 4, hipMemcpyHostToDevice, s));
  SD_TRY(hipStreamSynchronize(s));
  kv->len_upper = mx;
  return SPECDEC_OK;
}

specdec_status specdec_kv_read_state(specdec_kv* kv, int32_t* len, int32_t* pending, int32_t* n_pending,
                                     int32_t* status, void* stream) {
  if (!kv || !kv->state) return SPECDEC_ERR_INVALID_ARG;
  const int B = kv->batch;
  std::vector<int32_t> host(specdec_kv_state_count(B), 0);
  hipStream_t s = (hipStream_t)stream;
  SD_TRY(hipMemcpyAsync(host.data(), kv->state, host.size() * 4, hipMemcpyDeviceToHost, s));
  SD_TRY(hipStreamSynchronize(s));
  int64_t mx = 0;
  for (int b = 0; b < B; ++b) {
    if (len) len[b] = host[b];
    if (pending) { pending[2 * b] = host[B + 2 * b]; pending[2 * b + 1] = host[B + 2 * b + 1]; }
    if (n_pending) n_pending[b] = host[3 * B + b];
    mx = std::max<int64_t>(mx, host[b]);
  }
  if (status) *status = host[4 * B];
  kv->len_upper = mx;
  return SPECDEC_OK;
}

specdec_status specdec_prefill(const specdec_model* model, specdec_kv* kv, int32_t n, const int32_t* tokens,
                               void* stream) {
  specdec_status st = check_kv(model, kv);
  if (st != SPECDEC_OK) return st;
  if (!tokens || n < 1) return SPECDEC_ERR_INVALID_ARG;
  const int B = kv->batch;
  if (kv->len_upper + n - 1 > kv->capacity) return SPECDEC_ERR_KV_CAPACITY;
  hipStream_t s = (hipStream_t)stream;
  // Chunks of as many tokens per sequence as the handle's rows allow (bf16: passes
  // of more than 64 rows run the wide GEMM; float32 models keep 64-row chunks).
  const int per = model->max_rows / B;
  const int C = std::max(1, model->desc.dtype == SPECDEC_BF16 ? per : std::min(per, 64));
  if (model->max_rows < B) return SPECDEC_ERR_SHAPE;
  for (int c0 = 0; c0 < n - 1; c0 += C) {
    const int rps = std::min(C, n - 1 - c0);
    RowsArgs ra{};
    ra.mode = ROWS_PREFILL;
    ra.M = B * rps;
    ra.rps = rps;
    ra.tok_src = tokens;
    ra.ld_tok = n;
    ra.c0 = c0;
    st = forward(model, kv, ra, (int)std::min<int64_t>(kv->len_upper + c0 + rps, kv->capacity), model->logits, s);
    if (st != SPECDEC_OK) return st;
  }
  hipLaunchKernelGGL(prefill_finish_kernel, dim3(1), dim3(64), 0, s, B, n, tokens, kv_len(kv), kv_pending(kv),
                     kv_npending(kv));
  SD_TRY(hipGetLastError());
  kv->len_upper += n - 1;
  return SPECDEC_OK;
}

specdec_status specdec_draft_step(const specdec_model* draft, specdec_kv* kv, int32_t gamma, int32_t slot,
                                  float temperature, uint64_t seed, uint64_t step, const uint64_t* step_dev,
                                  const uint32_t* rand, float* q_out, int32_t* d_out, int32_t ld_d,
                                  float* logits_out, void* stream) {
  specdec_status st = check_kv(draft, kv);
  if (st != SPECDEC_OK) return st;
  if (!d_out || gamma < 1 || slot < 0 || slot >= gamma || ld_d < gamma || !(temperature >= 0.f) ||
      misaligned8(step_dev))
    return SPECDEC_ERR_INVALID_ARG;
  if (temperature > 0.f && !q_out) return SPECDEC_ERR_INVALID_ARG;
  const int B = kv->batch;
  if (kv->len_upper + slot + 2 > kv->capacity) return SPECDEC_ERR_KV_CAPACITY;
  hipStream_t s = (hipStream_t)stream;
  RowsArgs ra{};
  if (slot == 0) {
    ra.mode = ROWS_DRAFT_FIRST;
    ra.rps = 2;
  } else {
    ra.mode = ROWS_DRAFT_NEXT;
    ra.rps = 1;
    ra.tok_src = d_out;
    ra.ld_tok = ld_d;
    ra.slot = slot;
  }
  ra.M = B * ra.rps;
  if (ra.M > draft->max_rows) return SPECDEC_ERR_SHAPE;
  st = forward(draft, kv, ra, (int)(kv->len_upper + slot + 2), draft->logits, s);
  if (st != SPECDEC_OK) return st;
  DraftFinishArgs f{};
  f.B = B;
  f.rps = ra.rps;
  f.V = draft->desc.vocab;
  f.logits = draft->logits;
  f.temperature = temperature;
  f.seed = seed;
  f.step = step;
  f.step_dev = step_dev;
  f.rand = rand;
  f.slot = slot;
  f.gamma = gamma;
  f.q_out = q_out;
  f.d_out = d_out;
  f.ld_d = ld_d;
  f.logits_out = logits_out;
  f.status = kv_status(kv);
  f.scratch = draft->samp;
  Timed t(SPECDEC_KERNEL_DRAFT_FINISH, s);
  return hip_status(launch_draft_finish(f, s));
}

specdec_status specdec_verify(const specdec_model* target, specdec_kv* kv, int32_t gamma, const int32_t* d,
                              int32_t ld_d, float* logits_out, void* stream) {
  specdec_status st = check_kv(target, kv);
  if (st != SPECDEC_OK) return st;
  if (!logits_out || gamma < 0 || (gamma > 0 && (!d || ld_d < gamma))) return SPECDEC_ERR_INVALID_ARG;
  const int B = kv->batch;
  if (kv->len_upper + gamma + 1 > kv->capacity) return SPECDEC_ERR_KV_CAPACITY;
  RowsArgs ra{};
  ra.mode = ROWS_VERIFY;
  ra.rps = gamma + 1;
  ra.M = B * ra.rps;
  ra.tok_src = d;
  ra.ld_tok = ld_d;
  if (ra.M > target->max_rows) return SPECDEC_ERR_SHAPE;
  return forward(target, kv, ra, (int)(kv->len_upper + gamma + 1), logits_out, (hipStream_t)stream);
}

specdec_status specdec_packed_range(const specdec_model_desc* desc, int32_t first_layer, int32_t n_layers,
                                    size_t* offset, size_t* bytes) {
  specdec_status st = check_desc(desc);
  if (st != SPECDEC_OK) return st;
  if (desc->dtype != SPECDEC_BF16) return SPECDEC_ERR_UNSUPPORTED;
  if (!offset || !bytes || first_layer < 0 || n_layers <= 0 || first_layer + n_layers > desc->n_layers)
    return SPECDEC_ERR_INVALID_ARG;
  std::vector<PackedMat> mats;
  const size_t total = image_layout(desc, first_layer + n_layers, &mats);
  // matrices: [0] LM head, then 7 per layer
  *offset = mats[1 + 7 * (size_t)first_layer].off;
  *bytes = total - *offset;
  return SPECDEC_OK;
}

specdec_status specdec_event_create(void** event) {
  if (!event) return SPECDEC_ERR_INVALID_ARG;
  *event = nullptr;
  hipEvent_t e = nullptr;
  SD_TRY(hipEventCreateWithFlags(&e, hipEventDisableTiming));
  *event = (void*)e;
  return SPECDEC_OK;
}

specdec_status specdec_event_destroy(void* event) {
  if (!event) return SPECDEC_ERR_INVALID_ARG;
  SD_TRY(hipEventDestroy((hipEvent_t)event));
  return SPECDEC_OK;
}

specdec_status specdec_load_async(void* dst, const void* host_src, size_t bytes, void* copy_stream, void* done_event) {
  if (!dst || !host_src || !bytes || !done_event) return SPECDEC_ERR_INVALID_ARG;
  hipStream_t s = (hipStream_t)copy_stream;
  SD_TRY(hipMemcpyAsync(dst, host_src, bytes, hipMemcpyHostToDevice, s));
  SD_TRY(hipEventRecord((hipEvent_t)done_event, s));
  return SPECDEC_OK;
}

specdec_status specdec_stream_wait_event(void* stream, void* event) {
  if (!event) return SPECDEC_ERR_INVALID_ARG;
  SD_TRY(hipStreamWaitEvent((hipStream_t)stream, (hipEvent_t)event, 0));
  return SPECDEC_OK;
}

specdec_status specdec_event_query(void* event, int32_t* done) {
  if (!event || !done) return SPECDEC_ERR_INVALID_ARG;
  const hipError_t e = hipEventQuery((hipEvent_t)event);
  if (e == hipSuccess) {
    *done = 1;
    return SPECDEC_OK;
  }
  if (e == hipErrorNotReady) {
    (void)hipGetLastError();  // clear the not-ready code
    *done = 0;
    return SPECDEC_OK;
  }
  return SPECDEC_ERR_HIP;
}

size_t specdec_accept_workspace_bytes(int32_t batch, int32_t gamma, int32_t vocab) {
  if (batch <= 0 || gamma < 0 || gamma > 31 || vocab <= 0) return 0;
  return sampling_scratch_bytes(batch, gamma + 1, vocab);
}

}  // extern "C"

namespace {
// Argument checks shared by specdec_accept and specdec_accept_noalloc.
specdec_status check_accept(int32_t batch, int32_t gamma, int32_t vocab, int32_t input_kind, float temperature,
                            const float* p, const float* q, const int32_t* d, int32_t ld_d,
                            const int32_t* n_accepted, const int32_t* next_token) {
  if (batch <= 0 || gamma < 0 || vocab <= 0 || !p || !n_accepted || !next_token || !(temperature >= 0.f))
    return SPECDEC_ERR_INVALID_ARG;
  if (gamma > 31) return SPECDEC_ERR_UNSUPPORTED;
  if (input_kind != SPECDEC_INPUT_PROBS && input_kind != SPECDEC_INPUT_LOGITS) return SPECDEC_ERR_INVALID_ARG;
  if (gamma > 0 && (!d || ld_d < gamma)) return SPECDEC_ERR_INVALID_ARG;
  if (temperature > 0.f && gamma > 0 && !q) return SPECDEC_ERR_INVALID_ARG;
  return SPECDEC_OK;
}
}  // namespace

extern "C" {

specdec_status specdec_accept(int32_t batch, int32_t gamma, int32_t vocab, int32_t input_kind, float temperature,
                              const float* p, const float* q, const int32_t* d, int32_t ld_d, const uint32_t* rand,
                              uint64_t seed, uint64_t step, const uint64_t* step_dev, int32_t* n_accepted,
                              int32_t* next_token, int32_t* status, void* workspace, size_t workspace_bytes,
                              void* stream) {
  const specdec_status st = check_accept(batch, gamma, vocab, input_kind, temperature, p, q, d, ld_d, n_accepted,
                                         next_token);
  if (st != SPECDEC_OK) return st;
  if (misaligned8(step_dev)) return SPECDEC_ERR_INVALID_ARG;
  if (!workspace || workspace_bytes < sampling_scratch_bytes(batch, gamma + 1, vocab)) return SPECDEC_ERR_INVALID_ARG;
  AcceptArgs a{};
  a.B = batch;
  a.gamma = gamma;
  a.V = vocab;
  a.input_kind = input_kind;
  a.temperature = temperature;
  a.p = p;
  a.q = q;
  a.d = d;
  a.ld_d = ld_d;
  a.rand = rand;
  a.seed = seed;
  a.step = step;
  a.step_dev = step_dev;
  a.n_accepted = n_accepted;
  a.next_token = next_token;
  a.status = status;
  a.scratch = workspace;
  Timed t(SPECDEC_KERNEL_ACCEPT, (hipStream_t)stream);
  return hip_status(launch_accept(a, (hipStream_t)stream));
}

specdec_status specdec_accept_noalloc(int32_t batch, int32_t gamma, int32_t vocab, int32_t input_kind,
                                      float temperature, const float* p, const float* q, const int32_t* d,
                                      int32_t ld_d, const uint32_t* rand, uint64_t seed, uint64_t step,
                                      const uint64_t* step_dev, int32_t* n_accepted, int32_t* next_token,
                                      int32_t* status, void* stream) {
  const specdec_status st = check_accept(batch, gamma, vocab, input_kind, temperature, p, q, d, ld_d, n_accepted,
                                         next_token);
  if (st != SPECDEC_OK) return st;
  if (misaligned8(step_dev)) return SPECDEC_ERR_INVALID_ARG;
  if (sampling_scratch_bytes(batch, gamma + 1, vocab) > kStaticAcceptScratchBytes) return SPECDEC_ERR_SCRATCH_LIMIT;
  void* scratch = nullptr;
  if (static_accept_scratch(&scratch) != hipSuccess) return SPECDEC_ERR_HIP;
  AcceptArgs a{};
  a.B = batch;
  a.gamma = gamma;
  a.V = vocab;
  a.input_kind = input_kind;
  a.temperature = temperature;
  a.p = p;
  a.q = q;
  a.d = d;
  a.ld_d = ld_d;
  a.rand = rand;
  a.seed = seed;
  a.step = step;
  a.step_dev = step_dev;
  a.n_accepted = n_accepted;
  a.next_token = next_token;
  a.status = status;
  a.scratch = scratch;  // (the device address of the static array, never the array's host-side name)
  Timed t(SPECDEC_KERNEL_ACCEPT, (hipStream_t)stream);
  return hip_status(launch_accept(a, (hipStream_t)stream));
}

const uint64_t* specdec_kv_step_word(const specdec_kv* kv) {
  return kv && kv->state ? kv_counter(kv) : nullptr;
}

specdec_status specdec_kv_commit(specdec_kv* kv, int32_t gamma, int32_t role, const int32_t* n_accepted,
                                 const int32_t* d, int32_t ld_d, const int32_t* next_token, void* stream) {
  if (!kv || !kv->state || !n_accepted || !next_token || gamma < 1) return SPECDEC_ERR_INVALID_ARG;
  if (role != SPECDEC_ROLE_TARGET && role != SPECDEC_ROLE_DRAFT) return SPECDEC_ERR_INVALID_ARG;
  if (role == SPECDEC_ROLE_DRAFT && (!d || ld_d < gamma)) return SPECDEC_ERR_INVALID_ARG;
  CommitArgs c{};
  c.B = kv->batch;
  c.gamma = gamma;
  c.role = role;
  c.len = kv_len(kv);
  c.pending = kv_pending(kv);
  c.n_pending = kv_npending(kv);
  c.n_accepted = n_accepted;
  c.d = d;
  c.ld_d = ld_d;
  c.next_token = next_token;
  c.counter = kv_counter(kv);
  specdec_status st;
  {
    Timed t(SPECDEC_KERNEL_COMMIT, (hipStream_t)stream);
    st = hip_status(launch_commit(c, (hipStream_t)stream));
  }
  if (st == SPECDEC_OK) kv->len_upper += gamma + 1;
  return st;
}

specdec_status specdec_sample(int32_t batch, int32_t vocab, const float* probs, int64_t ld, const uint32_t* rand,
                              uint64_t seed, uint64_t step, int32_t purpose, int32_t index, int32_t* out,
                              void* stream) {
  if (batch <= 0 || vocab <= 0 || !probs || !out || ld < vocab) return SPECDEC_ERR_INVALID_ARG;
  return hip_status(launch_sample(batch, vocab, probs, ld, rand, seed, step, purpose, index, out, (hipStream_t)stream));
}

specdec_status specdec_draw_u32(int32_t batch, uint64_t seed, uint64_t step, int32_t purpose, int32_t index,
                                uint32_t* out, void* stream) {
  if (batch <= 0 || !out || purpose < 0 || purpose > 0xffff || index < 0 || index > 0xffff)
    return SPECDEC_ERR_INVALID_ARG;
  return hip_status(launch_draw(batch, seed, step, purpose, index, out, (hipStream_t)stream));
}

specdec_status specdec_device_status(specdec_kv* kv, void* stream, int32_t* host_out) {
  if (!kv || !kv->state) return SPECDEC_ERR_INVALID_ARG;
  int32_t v = 0;
  hipStream_t s = (hipStream_t)stream;
  SD_TRY(hipMemcpyAsync(&v, kv_status(kv), 4, hipMemcpyDeviceToHost, s));
  SD_TRY(hipStreamSynchronize(s));
  if (host_out) *host_out = v;
  return (specdec_status)v;
}

specdec_status specdec_timing_enable(int32_t enable) {
  g_timing.enabled = enable != 0;
  return SPECDEC_OK;
}

specdec_status specdec_timing_read(double* total_ms, int64_t* launches) {
  double ms[SPECDEC_KERNEL_KINDS] = {0};
  int64_t n[SPECDEC_KERNEL_KINDS] = {0};
  specdec_status st = SPECDEC_OK;
  for (auto& r : g_timing.recs) {
    float t = 0.f;
    if (hipEventSynchronize(r.e) != hipSuccess || hipEventElapsedTime(&t, r.b, r.e) != hipSuccess) st = SPECDEC_ERR_HIP;
    ms[r.kind] += t;
    n[r.kind] += 1;
    g_timing.pool.push_back(r.b);
    g_timing.pool.push_back(r.e);
  }
  g_timing.recs.clear();
  for (int k = 0; k < SPECDEC_KERNEL_KINDS; ++k) {
    if (total_ms) total_ms[k] = ms[k];
    if (launches) launches[k] = n[k];
  }
  return st;
}

specdec_status specdec_time_kernel(const specdec_model* m, int32_t kind, int32_t reps, void* stream,
                                   double* avg_us) {
  if (!m || !avg_us || reps <= 0 || kind < 0 || kind >= SPECDEC_KERNEL_KINDS) return SPECDEC_ERR_INVALID_ARG;
  if (!m->rec_valid[kind]) return SPECDEC_ERR_UNSUPPORTED;
  hipStream_t s = (hipStream_t)stream;
  const int dt = m->desc.dtype;
  // Launch i re-runs layer i mod L: each launch streams weights (and keys and
  // values) that the launches just before it did not touch, as in the pass.
  auto launch = [&](int i) -> hipError_t {
    switch (kind) {
      case SPECDEC_KERNEL_EMBED: return launch_rows_embed(dt, m->rec_embed, s);
      case SPECDEC_KERNEL_ROPE_APPEND: return launch_rope_append(m->rec_attn[(size_t)i % m->rec_attn.size()], s);
      case SPECDEC_KERNEL_ATTENTION: return launch_attention(m->rec_attn[(size_t)i % m->rec_attn.size()], s);
      default: {
        const std::vector<GemmArgs>& v = m->rec_gemm[kind];
        return gemm_rows(dt, v[(size_t)i % v.size()], m->rec_rows[kind], s);
      }
    }
  };
  hipEvent_t e0 = nullptr, e1 = nullptr;
  SD_TRY(hipEventCreate(&e0));
  if (hipEventCreate(&e1) != hipSuccess) {
    (void)hipEventDestroy(e0);
    return SPECDEC_ERR_HIP;
  }
  hipError_t err = launch(0);  // warm-up
  if (err == hipSuccess) err = hipEventRecord(e0, s);
  for (int i = 1; i <= reps && err == hipSuccess; ++i) err = launch(i);
  if (err == hipSuccess) err = hipEventRecord(e1, s);
  if (err == hipSuccess) err = hipEventSynchronize(e1);
  float ms = 0.f;
  if (err == hipSuccess) err = hipEventElapsedTime(&ms, e0, e1);
  (void)hipEventDestroy(e0);
  (void)hipEventDestroy(e1);
  if (err != hipSuccess) return SPECDEC_ERR_HIP;
  *avg_us = 1e3 * (double)ms / reps;
  return SPECDEC_OK;
}

specdec_status specdec_stream_read(const void* buf, size_t bytes, uint32_t* sink, void* stream) {
  if (!buf || !sink || ((uintptr_t)buf & 15)) return SPECDEC_ERR_INVALID_ARG;
  return hip_status(launch_stream_read(buf, bytes, sink, (hipStream_t)stream));
}

const char* specdec_last_hip_error(void) {
  const hipError_t e = g_last_hip_error;
  g_last_hip_error = hipSuccess;
  return e == hipSuccess ? "" : hipGetErrorName(e);
}

const char* specdec_status_string(specdec_status s) {
  switch (s) {
    case SPECDEC_OK: return "ok";
    case SPECDEC_ERR_INVALID_ARG: return "invalid argument";
    case SPECDEC_ERR_SHAPE: return "unsupported shape";
    case SPECDEC_ERR_KV_CAPACITY: return "KV capacity exceeded";
    case SPECDEC_ERR_NONFINITE: return "non-finite probability or logit";
    case SPECDEC_ERR_HIP: return "HIP runtime error";
    case SPECDEC_ERR_UNSUPPORTED: return "unsupported request";
    case SPECDEC_ERR_BAD_TOKEN: return "token id out of range";
    case SPECDEC_ERR_SCRATCH_LIMIT: return "request needs more scratch than the static no-allocation buffer holds";
    case SPECDEC_ERR_WAIT_EXPIRED: return "a kernel's bounded wait for other blocks ran out";
  }
  return "unknown status";
}

}  // extern "C"
