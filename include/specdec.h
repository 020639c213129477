/*
 * specdec.h -- C ABI of the MI355X (gfx950) speculative-decoding hot path.
 *
 * One draft-and-verify iteration (the inner loop of the MemSpec runtime,
 * Sec. 3.4, Alg. 3: the active draft proposes, then the target verifies):
 *
 *   for s in 0..gamma-1: specdec_draft_step(draft, draft_kv, ..., slot = s)
 *   specdec_verify(target, target_kv, ...)      -- one target pass over gamma+1 tokens
 *   specdec_accept(...)                         -- speculative accept / resample
 *   specdec_kv_commit(target_kv, TARGET, ...);  specdec_kv_commit(draft_kv, DRAFT, ...)
 *
 * Throughput of the loop is E[A] / L_iter (Sec. 2.1, Eq. (1)); A is the number
 * of drafted tokens the target accepts.  The verification rule (accept with
 * probability min(1, p/q), else resample from norm(max(0, p - q)), bonus
 * token from p_{gamma+1} when all are accepted) is the one of the
 * speculative-decoding works the paper builds on; the paper itself runs the
 * greedy special case (Sec. 4.1, "Runtime configuration").
 *
 * Conventions for every function below:
 *  - Pointers are DEVICE pointers unless marked "host".  The caller owns every
 *    buffer (weights, KV, workspace, outputs); the library never allocates
 *    device memory, so calls can be captured into a HIP graph.
 *  - `stream` is a hipStream_t passed as void* (NULL = the default stream).
 *    Calls are asynchronous on it unless documented as synchronizing.
 *  - Argument and shape errors are returned synchronously and nothing is
 *    launched.  Errors only a kernel can see (token id out of range, KV
 *    capacity overflow, NaN/Inf probabilities) set a sticky device status
 *    word (specdec_kv.state, or the `status` argument of specdec_accept);
 *    the kernel then skips the offending writes.  Read it with
 *    specdec_kv_read_state or specdec_device_status.
 *  - Handles are not thread-safe; calls on one KV cache must be
 *    stream-ordered.
 *  - Graph capture: every launch of an iteration reads lengths, pending
 *    tokens and (with step_dev) the Philox step from the device, so one
 *    captured iteration can be replayed R times with no host work between
 *    replays.  Its grids are sized from the host bound kv->len_upper at
 *    capture: set that field of each cache to the bound the R-th replay will
 *    reach (current bound + R * (gamma+1)) before capturing, within capacity.
 *  - Storage types: SPECDEC_F32 (weights and KV float32) or SPECDEC_BF16
 *    (weights and KV bfloat16).  Activations, logits and probabilities are
 *    always float32.
 */
#ifndef SPECDEC_H
#define SPECDEC_H

#include <stddef.h>
#include <stdint.h>

#if defined(__GNUC__)
#define SPECDEC_API __attribute__((visibility("default")))
#else
#define SPECDEC_API
#endif

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  SPECDEC_OK = 0,
  SPECDEC_ERR_INVALID_ARG = -1, /* null pointer, negative size, bad enum */
  SPECDEC_ERR_SHAPE = -2,       /* dimensions the kernels do not support */
  SPECDEC_ERR_KV_CAPACITY = -3, /* the call could write past the KV capacity */
  SPECDEC_ERR_NONFINITE = -4,   /* NaN/Inf probability or logit (device status) */
  SPECDEC_ERR_HIP = -5,         /* a HIP runtime call failed */
  SPECDEC_ERR_UNSUPPORTED = -6, /* valid request outside what is implemented */
  SPECDEC_ERR_BAD_TOKEN = -7,   /* token id outside [0, vocab) (device status) */
  SPECDEC_ERR_SCRATCH_LIMIT = -8, /* needs more than the static scratch of specdec_accept_noalloc */
  SPECDEC_ERR_WAIT_EXPIRED = -9   /* a kernel's bounded wait for other blocks ran out (device status) */
} specdec_status;

enum { SPECDEC_F32 = 0, SPECDEC_BF16 = 1 };
/* Weight image formats of bf16 models (activations, KV and the LM head stay
 * bf16 in both): BF16 stores every matrix in bf16; INT4 stores the layer
 * matrices as 4-bit codes with one bf16 scale per row and group of 128
 * input columns (the paper's models are INT4, Sec. 4.1; round-to-nearest
 * groups stand in for GPTQ, which needs calibration data). */
enum { SPECDEC_WEIGHTS_BF16 = 0, SPECDEC_WEIGHTS_INT4 = 1 };
enum { SPECDEC_ROLE_TARGET = 0, SPECDEC_ROLE_DRAFT = 1 };
enum { SPECDEC_INPUT_PROBS = 0, SPECDEC_INPUT_LOGITS = 1 };
/* Philox counter purposes (see specdec_draw_u32). */
enum { SPECDEC_PURPOSE_DRAFT = 0, SPECDEC_PURPOSE_ACCEPT = 1, SPECDEC_PURPOSE_RESAMPLE = 2 };

/* Llama-style decoder shape.  The paper's targets are LLaMA-2 7B and
 * Qwen2.5 7B with 400M/0.5B drafts (Sec. 4.1, "Models"); a draft here is a
 * prefix of the target's layers sharing its embedding, final norm and LM head. */
typedef struct {
  int32_t n_layers;   /* layers held by the weight arrays */
  int32_t d_model;    /* d: multiple of 64 */
  int32_t n_heads;    /* query heads h; h*hd a multiple of 64 */
  int32_t n_kv_heads; /* kv heads; n_heads % n_kv_heads == 0 (GQA: kv head = q head / (h / h_kv)) */
  int32_t head_dim;   /* hd: 32, 64 or 128 */
  int32_t ffn_dim;    /* SwiGLU hidden size F: multiple of 32 */
  int32_t vocab;      /* V: multiple of 16 */
  float rms_eps;      /* RMSNorm epsilon */
  float rope_base;    /* RoPE base (rotate-half pairs (j, j + hd/2), theta_j = base^(-2j/hd)) */
  int32_t dtype;      /* SPECDEC_F32 or SPECDEC_BF16 */
} specdec_model_desc;

/* Device pointers to weights, all row-major [out, in] of the storage type.
 * Per-layer arrays are HOST arrays of n_layers device pointers. */
typedef struct {
  const void* embed;      /* [V, d] */
  const void* lm_head;    /* [V, d] (not tied to embed) */
  const void* final_norm; /* [d] */
  const void* const* attn_norm; /* L x [d] */
  const void* const* wq;        /* L x [h*hd, d] */
  const void* const* wk;        /* L x [h_kv*hd, d] */
  const void* const* wv;        /* L x [h_kv*hd, d] */
  const void* const* wo;        /* L x [d, h*hd] */
  const void* const* ffn_norm;  /* L x [d] */
  const void* const* w_gate;    /* L x [F, d] */
  const void* const* w_up;      /* L x [F, d] */
  const void* const* w_down;    /* L x [d, F] */
} specdec_weights;

typedef struct specdec_model specdec_model; /* opaque host handle */

/* Per-model-instance KV cache and sequence state.  A POD the caller allocates
 * (host memory); specdec_kv_init fills it.  Fields are read-only for the caller
 * except len_upper (see graph capture above). */
typedef struct {
  void* data;          /* device: K and V of every layer (layout private to the library) */
  int32_t* state;      /* device: int32 [4*batch + 4], 8-byte aligned: len[B], pending[2B],
                          n_pending[B], status, one unused word, then the commit counter
                          (uint64 over the last two words, see specdec_kv_step_word) */
  int32_t batch;       /* sequences */
  int32_t capacity;    /* positions per sequence (multiple of 64) */
  int32_t n_layers;    /* layers this cache serves */
  int32_t n_kv_heads, head_dim, dtype;
  int64_t len_upper;   /* host-side upper bound of max_b len[b] (kept by the library; a
                          caller may raise it before a graph capture) */
} specdec_kv;

/* ---------------------------------------------------------------- set-up */

/* Bytes of workspace a model handle needs for calls with up to `max_rows`
 * rows (rows = batch*(gamma+1) for verify, 2*batch for the draft's first
 * slot, batch*chunk for prefill) and contexts of up to `max_ctx` positions. */
SPECDEC_API size_t specdec_workspace_bytes(const specdec_model_desc* desc, int32_t max_rows, int32_t max_ctx);

/* Bytes of the packed weight image of a bf16 model's first n_layers_used
 * layers (0 for float32 models, which run on the row-major weights).
 * Image layout: the LM head, then per layer Wq, Wk, Wv, Wo, W_gate, W_up,
 * W_down; each [N, K] matrix is stored as 16-row x 32-column fragments of
 * 1 KB (fragment (t, s) at byte 1024*(t*ceil(K/32) + s); inside it, lane
 * l = 16*g + i holds row 16t + i, columns 32s + 8g .. 32s + 8g + 7, zero past
 * K), the operand order of v_mfma_f32_16x16x32_bf16, so that each wavefront
 * load of the GEMMs reads 1 KB of contiguous memory.  A prefix of the image
 * is the image of a layer prefix: a draft can use its target's image. */
SPECDEC_API size_t specdec_packed_bytes(const specdec_model_desc* desc, int32_t n_layers_used);

/* Write the packed image of the row-major `weights` (first n_layers_used
 * layers) into `packed` (device, >= specdec_packed_bytes, 256-byte aligned).
 * Asynchronous on stream; the row-major matrices may be freed once it has
 * completed.  Errors: INVALID_ARG, SHAPE, UNSUPPORTED (float32 model). */
SPECDEC_API specdec_status specdec_pack_weights(const specdec_model_desc* desc, const specdec_weights* weights,
                                                int32_t n_layers_used, void* packed, size_t packed_bytes,
                                                void* stream);

/* The same in a chosen weight format (SPECDEC_WEIGHTS_*).  INT4 image: the
 * LM head as in the bf16 image, then per layer the seven matrices, each as
 * INT4 code fragments followed by its scales (256-byte aligned):
 *  - codes: per 16-row tile t and group G of 128 columns a 1 KB block at
 *    byte 1024*(t*ceil(K/128) + G); lane l = 16*c + i holds 16 bytes at
 *    16*l, four 32-bit words, word j holding the 8 codes of row 16t + i at
 *    columns 128G + 32j + 8c .. +7, code e in bits 4e..4e+3 (two's
 *    complement, -8..7; columns past K hold 0);
 *  - scales: bf16 [N/16][ceil(K/128)][16] (tile, group, row in tile).
 * Quantization (on the device, from the bf16 matrices): per row and group of
 * 128 columns, s = bf16(max|w| / 7) (float32 division, then rounding to
 * nearest even), q = clamp(rint(w / s), -8, 7) (float32; q = 0 where s = 0).
 * The model then computes with the effective weights q * s exactly.
 * Requires K % 32 == 0 for every layer matrix.  Errors as specdec_pack_weights,
 * INVALID_ARG for an unknown format. */
SPECDEC_API size_t specdec_packed_bytes_fmt(const specdec_model_desc* desc, int32_t n_layers_used, int32_t format);
SPECDEC_API specdec_status specdec_pack_weights_fmt(const specdec_model_desc* desc, const specdec_weights* weights,
                                                    int32_t n_layers_used, int32_t format, void* packed,
                                                    size_t packed_bytes, void* stream);

/* Create a handle over caller-owned weights.  n_layers_used <= desc->n_layers
 * selects a layer prefix (a draft).  bf16 models take their matrices from
 * `packed` (an image written by specdec_pack_weights covering at least
 * n_layers_used layers, e.g. the target's image for a draft) and only the
 * embedding and RMSNorm gains from `weights`; float32 models pass
 * packed = NULL and use the row-major matrices of `weights`.
 * `workspace` (device, >= specdec_workspace_bytes, 256-byte aligned) belongs
 * to the handle until specdec_model_destroy; two handles may share one
 * workspace only if their calls never overlap.  Launches nothing (the
 * handle's first forward pass clears a region of the workspace, the bf16
 * attention's combine counters, with a small kernel on its stream; the
 * counters are back at zero after every attention launch).
 * Errors: INVALID_ARG (nulls), SHAPE (unsupported dims), HIP. */
SPECDEC_API specdec_status specdec_model_create(const specdec_model_desc* desc, const specdec_weights* weights,
                                    int32_t n_layers_used, const void* packed, size_t packed_bytes,
                                    int32_t max_rows, int32_t max_ctx,
                                    void* workspace, size_t workspace_bytes, specdec_model** out);
/* The same over an image of a chosen weight format.  INT4 handles run passes
 * of at most 64 rows (max_rows <= 64: verify and draft steps, prefill in
 * 64-row chunks); UNSUPPORTED otherwise or for float32 models. */
SPECDEC_API specdec_status specdec_model_create_fmt(const specdec_model_desc* desc, const specdec_weights* weights,
                                                    int32_t n_layers_used, int32_t format, const void* packed,
                                                    size_t packed_bytes, int32_t max_rows, int32_t max_ctx,
                                                    void* workspace, size_t workspace_bytes, specdec_model** out);
SPECDEC_API void specdec_model_destroy(specdec_model* model);

/* Bytes of KV storage for `batch` sequences of `capacity` positions over the
 * first `n_layers_used` layers of the model shape. */
SPECDEC_API size_t specdec_kv_bytes(const specdec_model_desc* desc, int32_t n_layers_used, int32_t batch, int32_t capacity);
/* Number of int32 entries of the KV state array (4*batch + 4). */
SPECDEC_API int32_t specdec_kv_state_count(int32_t batch);

/* Fill `kv` (host POD) over caller-owned device buffers and zero the state
 * (all lengths 0, no pending tokens, status OK, commit counter 0).
 * Asynchronous on stream.  Errors: INVALID_ARG (nulls, a state array that is
 * not 8-byte aligned, data_bytes below specdec_kv_bytes), SHAPE (capacity not
 * a multiple of 64). */
SPECDEC_API specdec_status specdec_kv_init(specdec_kv* kv, const specdec_model* model, int32_t batch, int32_t capacity,
                               void* data, size_t data_bytes, int32_t* state, void* stream);

/* Install K and V rows for sequence b, layer `layer`, positions [pos0, pos0+n):
 * k, v are device arrays [n, n_kv_heads, head_dim] of the storage type (K
 * after RoPE, as a forward pass would have stored it).  Used to set up a
 * resident context without prefill.  Asynchronous. */
SPECDEC_API specdec_status specdec_kv_write_context(specdec_kv* kv, int32_t layer, int32_t b, int32_t pos0, int32_t n,
                                        const void* k, const void* v, void* stream);
/* Copy K and V rows back out (same layout as specdec_kv_write_context). */
SPECDEC_API specdec_status specdec_kv_read_context(const specdec_kv* kv, int32_t layer, int32_t b, int32_t pos0, int32_t n,
                                       void* k, void* v, void* stream);

/* Set lengths and pending tokens from HOST arrays: len[B], pending[2B]
 * (right-aligned: pending[2b+1] is the newest token), n_pending[B] in {1,2}.
 * Clears the status word and leaves the commit counter as it is.
 * Synchronizes the stream. */
SPECDEC_API specdec_status specdec_kv_set_state(specdec_kv* kv, const int32_t* len, const int32_t* pending,
                                    const int32_t* n_pending, void* stream);
/* Read lengths, pending tokens and the status word into HOST arrays (any may
 * be NULL).  Synchronizes the stream and refreshes kv->len_upper. */
SPECDEC_API specdec_status specdec_kv_read_state(specdec_kv* kv, int32_t* len, int32_t* pending, int32_t* n_pending,
                                     int32_t* status, void* stream);

/* Commit a prompt: run the model over tokens[b, 0..n-2] (device int32 [batch, n])
 * in chunks of max_rows / batch tokens per sequence (float32 models: at most
 * 64), appending their K/V from position len[b], then len[b] += n-1 and the
 * pending token becomes tokens[b, n-1].  Also the catch-up forward of a draft
 * that missed committed tokens.  Not on the timed verify path (the paper
 * excludes prompt encoding from throughput, Sec. 4.1). */
SPECDEC_API specdec_status specdec_prefill(const specdec_model* model, specdec_kv* kv, int32_t n, const int32_t* tokens,
                               void* stream);

/* ---------------------------------------------------------------- hot path */

/* Draft single-token decode step at draft slot `slot` (0 <= slot < gamma):
 * the draft model proposing one candidate token per sequence, the first half
 * of a draft-and-verify iteration (Sec. 2.1; Alg. 3, the active draft's
 * proposal step, run gamma times per iteration).
 *
 *  slot 0 processes the cache's 1 or 2 pending tokens (2 after an iteration
 *  that accepted every draft), slot s > 0 processes d_out[b*ld_d + s-1].
 *  It appends their K/V speculatively (len is unchanged until commit), runs
 *  the LM head, and proposes d_out[b*ld_d + slot]:
 *    temperature == 0: argmax of the logits (lowest index on ties);
 *    temperature >  0: q = softmax(logits / T) written to q_out[b, slot, :]
 *      (q_out is [batch, gamma, V] float32) and the token drawn from q with
 *      the fixed-point inverse-CDF sampler (see specdec_sample) using the
 *      32-bit word rand[b] if rand != NULL, else Philox(seed, b, step,
 *      SPECDEC_PURPOSE_DRAFT, slot).
 *  step_dev (optional): a device uint64 read by the kernel in place of `step`
 *      (e.g. specdec_kv_step_word of the target cache), so that a captured
 *      HIP graph of an iteration draws fresh words on every replay.
 *  logits_out (optional, [batch, V]) receives the proposing row's logits.
 * Errors: INVALID_ARG, SHAPE (batch/gamma beyond the handle's max_rows),
 * KV_CAPACITY (len_upper + 2 + gamma > capacity). */
SPECDEC_API specdec_status specdec_draft_step(const specdec_model* draft, specdec_kv* kv, int32_t gamma, int32_t slot,
                                  float temperature, uint64_t seed, uint64_t step, const uint64_t* step_dev,
                                  const uint32_t* rand, float* q_out, int32_t* d_out, int32_t ld_d,
                                  float* logits_out, void* stream);

/* Target verify pass (Sec. 2.1: the target model checks the drafted
 * candidates; Alg. 3, the verification step): one forward over the
 * gamma+1 tokens
 * [pending token, d[b*ld_d + 0 .. gamma-1]] at positions len[b] .. len[b]+gamma,
 * causal inside the block, against the resident cache (the drafted tokens'
 * K/V are appended speculatively).  logits_out: [batch, gamma+1, V] float32,
 * row i = next-token logits after token i. */
SPECDEC_API specdec_status specdec_verify(const specdec_model* target, specdec_kv* kv, int32_t gamma, const int32_t* d,
                              int32_t ld_d, float* logits_out, void* stream);

/* Accept / resample for every sequence b (one draft-and-verify decision; it
 * yields the accepted count A of Sec. 2.1, Eq. 1):
 *  p:  [batch, gamma+1, V] float32 -- target probabilities (input_kind PROBS)
 *      or logits (input_kind LOGITS: p = softmax(logits / temperature));
 *  q:  [batch, gamma, V] float32 draft probabilities (unused when greedy);
 *  d:  drafted tokens d[b*ld_d + i];
 *  rand: [batch, gamma+1] 32-bit words ([0, gamma) accept tests, [gamma] the
 *      resample / bonus draw) or NULL => Philox(seed, b, step, purpose, index);
 *  step_dev: as for specdec_draft_step (NULL => `step`).
 * Sampling (temperature > 0): accept d_i iff fl32(u_i * q_i(d_i)) < p_i(d_i)
 * with u_i = (word >> 8) * 2^-24; at the first rejection emit a draw from
 * max(0, fl32(p_i - q_i)) (from p_i if that is all zero); if all accepted emit
 * a draw from p_{gamma+1}.  Greedy (temperature == 0): A = length of the
 * prefix where d_i equals argmax p_i; emit argmax p_{A+1}.
 * Outputs n_accepted[b] = A in [0, gamma], next_token[b].  A NaN or Inf
 * anywhere in p (either kind) or, when sampling, in q, or a drafted token
 * outside [0, V) when sampling, sets *status = SPECDEC_ERR_NONFINITE (device
 * int32, sticky, may be NULL) and writes A = -1, next_token = -1.
 * workspace: device scratch of at least specdec_accept_workspace_bytes(batch,
 * gamma, vocab) bytes, 256-byte aligned, owned by the caller; its contents
 * need no initialisation and are dead after the call.  Calls that share a
 * workspace must be ordered on one stream.
 * Errors: INVALID_ARG (also for a missing or short workspace), UNSUPPORTED
 * (gamma > 31). */
SPECDEC_API specdec_status specdec_accept(int32_t batch, int32_t gamma, int32_t vocab, int32_t input_kind, float temperature,
                              const float* p, const float* q, const int32_t* d, int32_t ld_d, const uint32_t* rand,
                              uint64_t seed, uint64_t step, const uint64_t* step_dev, int32_t* n_accepted,
                              int32_t* next_token, int32_t* status, void* workspace, size_t workspace_bytes,
                              void* stream);

/* Bytes of the accept workspace for `batch` sequences of gamma+1 rows over a
 * vocabulary of `vocab` (0 for arguments specdec_accept rejects). */
SPECDEC_API size_t specdec_accept_workspace_bytes(int32_t batch, int32_t gamma, int32_t vocab);

/* For callers that cannot allocate device memory: code under HIP graph
 * capture that may not call hipMalloc, tight serving loops, harnesses that
 * forbid allocation.  specdec_accept without the workspace argument; every
 * other argument, the result and the device status are those of
 * specdec_accept, and the kernels are the same.
 * Scratch: a static device array of SPECDEC_ACCEPT_NOALLOC_SCRATCH_BYTES in the
 * library, held by each GPU the library runs on until the process ends; no
 * call allocates or frees memory.  A request needing more scratch than the
 * array (specdec_accept_workspace_bytes(batch, gamma, vocab) bytes, e.g. up to
 * 64 sequences at gamma 8 over a 32000-token vocabulary) returns
 * SPECDEC_ERR_SCRATCH_LIMIT and launches nothing.  Every call on one GPU
 * shares the array and nothing in it needs to start at zero; calls that
 * overlap on one GPU (unordered streams, or threads) race on it and must not
 * be issued. */
#define SPECDEC_ACCEPT_NOALLOC_SCRATCH_BYTES ((size_t)2 << 20)
SPECDEC_API specdec_status specdec_accept_noalloc(int32_t batch, int32_t gamma, int32_t vocab, int32_t input_kind,
                                                  float temperature, const float* p, const float* q, const int32_t* d,
                                                  int32_t ld_d, const uint32_t* rand, uint64_t seed, uint64_t step,
                                                  const uint64_t* step_dev, int32_t* n_accepted, int32_t* next_token,
                                                  int32_t* status, void* stream);

/* KV commit / rollback after specdec_accept (device-side, graph friendly):
 * the A accepted drafts and the emitted token become committed text, the
 * rejected drafts are dropped (Sec. 2.1: A tokens accepted per iteration; the
 * end of one pass of Alg. 3's inner loop).
 *  TARGET: len += A+1; pending = [next]                       (n_pending = 1)
 *  DRAFT:  len += n_pending + min(A, gamma-1);
 *          pending = [d_gamma, next] if A == gamma else [next]
 * Entries at or beyond the new length are speculative and get overwritten.
 * A < 0 (an accept error) leaves that sequence untouched.  Every call adds 1
 * to the cache's commit counter (specdec_kv_step_word).  The host bound
 * kv->len_upper grows by gamma+1. */
SPECDEC_API specdec_status specdec_kv_commit(specdec_kv* kv, int32_t gamma, int32_t role, const int32_t* n_accepted,
                                 const int32_t* d, int32_t ld_d, const int32_t* next_token, void* stream);

/* Device address of the cache's commit counter: a uint64 in the state array,
 * 0 after specdec_kv_init, +1 per specdec_kv_commit, kept by
 * specdec_kv_set_state.  Passed as step_dev to the draft steps and the accept
 * of an iteration (all before its commits), it numbers the iteration's Philox
 * draws from the device, which is what a graph replayed without host work
 * needs.  NULL if kv or its state is NULL. */
SPECDEC_API const uint64_t* specdec_kv_step_word(const specdec_kv* kv);

/* ---------------------------------------------------------------- draft reload
 * Only K drafts stay resident; the others live in backing storage and are
 * loaded asynchronously, overlapped with decoding, and the runtime never
 * waits for a draft that is still loading (Sec. 3.3, Alg. 2, its background
 * prefetch of a predicted draft; Sec. 3.4, Alg. 3).  On one GPU: the backing storage is pinned
 * host memory holding a packed image, a resident slot is a device buffer in
 * the packed-image format, and a load is an H2D copy on a side stream whose
 * completion an event records.  A draft model created over the slot may run
 * on another stream once that stream waits for the event (or once
 * specdec_event_query reports it done).  Keeping the shared LM head in the
 * slot and reloading only a layer range avoids re-sending it. */

/* Byte range [*offset, *offset + *bytes) of layers [first_layer, first_layer +
 * n_layers) in the packed image of `desc` (the LM head occupies [0, offset of
 * layer 0)).  Errors: INVALID_ARG (null pointers, range outside
 * [0, desc->n_layers)), UNSUPPORTED (float32 desc: no packed image). */
SPECDEC_API specdec_status specdec_packed_range(const specdec_model_desc* desc, int32_t first_layer, int32_t n_layers,
                                                size_t* offset, size_t* bytes);

/* Create / destroy a completion event (a HIP event without timing; host
 * object, no device memory).  *event receives the handle. */
SPECDEC_API specdec_status specdec_event_create(void** event);
SPECDEC_API specdec_status specdec_event_destroy(void* event);

/* Copy `bytes` bytes from host `host_src` to device `dst` on `copy_stream`
 * (asynchronous: host_src must be pinned memory, e.g. from hipHostMalloc or a
 * pinned torch tensor, and must stay valid until the event completes), then
 * record `done_event` on `copy_stream`.  Returns at once.  Errors: INVALID_ARG
 * (null pointers, bytes == 0), HIP. */
SPECDEC_API specdec_status specdec_load_async(void* dst, const void* host_src, size_t bytes, void* copy_stream,
                                              void* done_event);

/* Make later work on `stream` wait for `event` (device-side; the host does
 * not block). */
SPECDEC_API specdec_status specdec_stream_wait_event(void* stream, void* event);

/* Non-blocking completion test: *done = 1 when all work recorded before
 * `event` has finished, else 0. */
SPECDEC_API specdec_status specdec_event_query(void* event, int32_t* done);

/* ---------------------------------------------------------------- building blocks */

/* Fixed-point inverse-CDF draw for each row b of probs [batch, ld] (first
 * `vocab` entries used): R_j = floor(r_j * 2^40) (uint64), S = sum R_j,
 * t = floor(x * S / 2^32), out[b] = smallest j with R_0 + ... + R_j > t,
 * where x = rand[b] if rand != NULL else Philox(seed, b, step, purpose, index).
 * All-zero rows give out[b] = -1.  Integer sums make it independent of the
 * reduction order, so it is bit-exact with any correct implementation. */
SPECDEC_API specdec_status specdec_sample(int32_t batch, int32_t vocab, const float* probs, int64_t ld, const uint32_t* rand,
                              uint64_t seed, uint64_t step, int32_t purpose, int32_t index, int32_t* out,
                              void* stream);

/* Philox4x32-10 (Salmon et al., SC'11) word 0 for each b in [0, batch):
 * key = (seed & 0xffffffff, seed >> 32),
 * counter = (b, step & 0xffffffff, step >> 32, (purpose << 16) | index). */
SPECDEC_API specdec_status specdec_draw_u32(int32_t batch, uint64_t seed, uint64_t step, int32_t purpose, int32_t index,
                                uint32_t* out, void* stream);

/* ---------------------------------------------------------------- measurement */

/* Kernel kinds for specdec_timing_read. */
enum {
  SPECDEC_KERNEL_EMBED = 0,        /* row set-up + embedding gather */
  SPECDEC_KERNEL_QKV = 1,          /* RMSNorm + Q|K|V projection GEMM */
  SPECDEC_KERNEL_ROPE_APPEND = 2,  /* RoPE + KV append */
  SPECDEC_KERNEL_ATTENTION = 3,    /* split-KV attention + combine */
  SPECDEC_KERNEL_O_PROJ = 4,       /* O projection GEMM + residual */
  SPECDEC_KERNEL_GATE_UP = 5,      /* RMSNorm + gate|up GEMM + SwiGLU */
  SPECDEC_KERNEL_DOWN = 6,         /* down projection GEMM + residual */
  SPECDEC_KERNEL_LM_HEAD = 7,      /* final RMSNorm + LM head GEMM */
  SPECDEC_KERNEL_DRAFT_FINISH = 8, /* draft softmax + sample */
  SPECDEC_KERNEL_ACCEPT = 9,       /* accept / resample */
  SPECDEC_KERNEL_COMMIT = 10,      /* KV commit */
  SPECDEC_KERNEL_KINDS = 11
};

/* Measurement hook (process-wide, off by default, never used inside graph
 * capture): while enabled, every kernel launch of the hot path is bracketed by
 * a pair of HIP events recorded on the launch's own stream. */
SPECDEC_API specdec_status specdec_timing_enable(int32_t enable);
/* Synchronize on the recorded events and return, per kernel kind, the summed
 * duration in milliseconds and the number of launches since the last read
 * (host arrays of SPECDEC_KERNEL_KINDS entries; either may be NULL); resets
 * the accumulators. */
SPECDEC_API specdec_status specdec_timing_read(double* total_ms, int64_t* launches);

/* Time one kernel in isolation: re-launch the launches of kernel kind `kind`
 * recorded by the last forward pass (verify, draft step or prefill chunk) of
 * `model`, `reps` times back to back between two HIP events on `stream`, the
 * i-th launch being layer i mod L's (the head GEMM and the embedding have one
 * launch each), after one untimed launch of layer 0; return the average
 * duration in microseconds.  Consecutive launches thus stream different
 * layers' weights (and keys and values), as the pass does, rather than
 * re-reading data a cache may still hold.  Measurement only: the re-launched
 * kernels write the model's workspace, K/V at that pass's cache positions of
 * the layers they run (from the workspace's current contents) and (residual
 * and head kinds) the hidden state and logits, so the pass's outputs must be
 * consumed, and those cache entries rewritten, before the model is used again.
 * Synchronizes the stream.
 * Errors: INVALID_ARG, UNSUPPORTED (kind not recorded yet), HIP. */
SPECDEC_API specdec_status specdec_time_kernel(const specdec_model* model, int32_t kind, int32_t reps, void* stream,
                                               double* avg_us);

/* Synchronize the stream and return the sticky status word of `kv` (also
 * written to *host_out if non-NULL). */
SPECDEC_API specdec_status specdec_device_status(specdec_kv* kv, void* stream, int32_t* host_out);

/* Streaming-read ceiling (measurement): reads the first floor(bytes / 1024) KB
 * at buf (device, 16-byte aligned) with the weight stream's access pattern:
 * one 16-wave block per CU, each wave reading 1 KB per load, two batches of
 * four loads per wave in flight, nontemporal.  The loaded data is XOR-ed into
 * a value that is stored to *sink (device, 4 bytes) only in a case that does
 * not occur for real data.  Asynchronous on `stream`; time it with events on
 * that stream to get the device's read rate for this pattern.
 * Errors: INVALID_ARG (null or misaligned pointer), HIP (a block's range above
 * 4 GiB). */
SPECDEC_API specdec_status specdec_stream_read(const void* buf, size_t bytes, uint32_t* sink, void* stream);

SPECDEC_API const char* specdec_status_string(specdec_status s);
/* Name of the HIP error behind this thread's last SPECDEC_ERR_HIP (e.g.
 * "hipErrorInvalidValue"), or "" if none; reading it clears it.  The string
 * is static. */
SPECDEC_API const char* specdec_last_hip_error(void);

#ifdef __cplusplus
}
#endif
#endif /* SPECDEC_H */
