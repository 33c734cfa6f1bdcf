/*
 * onela.h -- C ABI of the MI355X (gfx950) large-beam Gated DeltaNet decode.
 *
 * The method is OneLA (arXiv 2609.12399): every live beam of a generative-
 * recommendation beam search is represented by one shared post-prefill state
 * S_ctx (Sec. 3.1) plus a short append-only chain of per-step transition
 * records, found through a parent-pointer ancestry index (Sec. 3.3, Eq. 5).
 * A decode step computes o_b = S_{t,b} q_b for every live beam b (Sec. 2.2,
 * Eq. 1) without materialising any per-beam d_v x d_k state.
 *
 * Records.  This library stores the record of step t and beam slot b as the
 * step's own inputs (k, v, alpha, beta) rather than the paper's
 * (alpha, delta, k) of Sec. 3.2: with A_j = alpha_j (I - beta_j k_j k_j^T),
 * Eq. 1 reads S_j = S_{j-1} A_j + beta_j v_j k_j^T, so the read-out
 * S_t q_t can be evaluated by folding the query newest-to-oldest through the
 * A_j, collecting the beta_j v_j k_j^T terms on the way, and applying S_ctx
 * once at the end.  In exact arithmetic this is the same o_t as the paper's
 * projection replay (Eqs. 3-4).
 *
 * Conventions for every entry point:
 *   - Tensors are device pointers owned by the caller, dense, row-major, and
 *     16-byte aligned.  The library allocates no device memory: all of its
 *     device state lives in a caller-provided workspace.
 *   - S is d_v x d_k (Sec. 2.2), stored [d_v][d_k].
 *   - Value head hv uses query/key head hv / (H_V / H_K) (grouped heads).
 *   - alpha, beta are fp32, one per (beam, value head).  q/k/v use the
 *     context's io dtype (bf16 bits or fp32).  Outputs are fp32.
 *   - Eq. 1 has no 1/sqrt(d_k) query scaling and none is applied.
 *   - All device work is enqueued asynchronously on the context's stream;
 *     no call synchronises except onela_get_device_status.  A context is
 *     bound to one stream and is not thread-safe.
 *   - An entry point that returns an error other than ONELA_EHIP has
 *     enqueued nothing and left the context unchanged.
 */
#ifndef ONELA_H
#define ONELA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct onela_ctx_s* onela_ctx_t;

typedef enum {
  ONELA_OK = 0,
  ONELA_EINVAL = 1,    /* NULL or misaligned pointer, unsupported dimension */
  ONELA_ESTEP = 2,     /* call out of the per-step protocol order */
  ONELA_EPARENT = 3,   /* device-detected: a parent index was out of range */
  ONELA_ECAPACITY = 4, /* width > max_beams, step >= max_steps, or a
                          workspace smaller than required */
  ONELA_EHIP = 5,      /* a HIP runtime call or kernel launch failed */
  ONELA_ENOMEM = 6     /* host allocation of the context failed */
} onela_status_t;

typedef enum { ONELA_F32 = 0, ONELA_BF16 = 1 } onela_dtype_t;

/* What one record of the arena holds.
 * ONELA_RECORD_INPUTS: the step's own inputs (k, v, alpha, beta); the decode
 *   folds the query newest-to-oldest and applies S_ctx once (see above).
 * ONELA_RECORD_DELTA: the paper's GDN transition record (alpha, delta, k) of
 *   Sec. 3.2 (Eq. 2), delta_t = beta_t (v_t - alpha_t S_{t-1} k_t), computed
 *   and appended by the decode step, which replays the ancestral records on
 *   the two projections S_ctx q_t and S_ctx k_t (Eqs. 3-4).  delta is stored
 *   in fp16 for bf16 io, scaled per row slice by a power of two that puts
 *   the row's largest magnitude at 2^14 (so neither fp16 overflow nor its
 *   subnormal range limits the inputs' magnitude), and in fp32 for fp32 io. */
typedef enum { ONELA_RECORD_INPUTS = 0, ONELA_RECORD_DELTA = 1 } onela_record_kind_t;

/* Where ONELA_RECORD_INPUTS records live (Sec. 3.3: a step's records are
 * written once, into the current step's physical slots, and never moved).
 * ONELA_RECORDS_COPY: the library copies each step's (k, v, alpha, beta) into
 *   its workspace arena; the caller may reuse its buffers once the step's
 *   launch has run.
 * ONELA_RECORDS_BORROW: the caller's step-t buffers ARE the slab of step t
 *   (zero copy): appending only registers their addresses.  The caller keeps
 *   k, v, alpha and beta of every step of the current beam search allocated
 *   and unmodified until onela_reset or onela_destroy.  The workspace then has
 *   no record arena.  Not available with ONELA_RECORD_DELTA (delta records are
 *   computed by the library and must be stored). */
typedef enum { ONELA_RECORDS_COPY = 0, ONELA_RECORDS_BORROW = 1 } onela_record_storage_t;

/* Shape of one decode context.  Supported (d_k, d_v): (32, 32), (64, 64),
 * (128, 128) with io_dtype ONELA_BF16 or ONELA_F32, and (128, 256), (128, 512),
 * (256, 256), (256, 512) with ONELA_BF16; num_v_heads a multiple of num_qk_heads;
 * 1 <= max_beams <= 65536; 1 <= max_steps <= 8 (the record chain of step t
 * has t + 1 records). */
typedef struct {
  int32_t num_requests; /* R: independent requests, one S_ctx each */
  int32_t num_qk_heads; /* H_K */
  int32_t num_v_heads;  /* H_V */
  int32_t d_k;
  int32_t d_v;
  int32_t max_beams;    /* W_max: upper bound on every W_t */
  int32_t max_steps;    /* T_max: decode steps 0 .. T_max - 1 */
  int32_t io_dtype;     /* onela_dtype_t of q, k, v */
  int32_t record_kind;  /* onela_record_kind_t */
  int32_t record_storage; /* onela_record_storage_t */
} onela_config_t;

/* Human-readable name of a status code (static string). */
const char* onela_status_str(onela_status_t status);

/* Checks a configuration on the host (no HIP call).  ONELA_OK or
 * ONELA_EINVAL. */
onela_status_t onela_check_config(const onela_config_t* cfg);

/* Bytes of device workspace onela_init needs for cfg (0 if cfg is invalid).
 * Layout (each part 256-byte aligned): status word, double-buffered ancestry
 * index [2][R][W_max][T_max] int32, S_ctx split into bf16 high/low halves
 * (written by the step-0 launch, read by later steps), and, unless records
 * are borrowed, the record arena: k [R][T_max][H_K][W_max][d_k],
 * v [R][T_max][H_V][W_max][d_v] in the io dtype, (alpha, beta)
 * [R][T_max][H_V][W_max] fp32 pairs and, for ONELA_RECORD_DELTA,
 * delta [R][T_max][H_V][W_max][d_v] (fp16 / fp32) and, per delta row, a
 * 32-bit word of int8 scale exponents [R][T_max][H_V][W_max]. */
size_t onela_workspace_bytes(const onela_config_t* cfg);

/* Creates a decode context and binds the shared post-prefill state
 * (Sec. 3.1: S_ctx is stored once per request and shared by all beams).
 * Host bookkeeping only: nothing is enqueued.  The current device's
 * compute-unit count is read once per device (a host attribute query) and
 * chooses the decode tiling of launches that would leave most units idle.
 *   s0        device, fp32 [R][H_V][d_v][d_k]; borrowed until onela_destroy
 *             (read by the step-0 launch of every beam search), owned by the
 *             caller
 *   workspace device, >= onela_workspace_bytes(cfg), 256-byte aligned;
 *             borrowed until onela_destroy, owned by the caller
 *   stream    a hipStream_t (NULL: the default stream)
 *   out       receives the context handle
 * Errors: ONELA_EINVAL (bad cfg or pointers), ONELA_ECAPACITY (workspace too
 * small), ONELA_ENOMEM, ONELA_EHIP. */
onela_status_t onela_init(const onela_config_t* cfg, const float* s0,
                          void* workspace, size_t workspace_bytes, void* stream,
                          onela_ctx_t* out);

/* Starts a new beam search on the same S_ctx: forgets all records and the
 * ancestry (host bookkeeping only; nothing is enqueued). */
onela_status_t onela_reset(onela_ctx_t ctx);

/* Ancestry index update of Sec. 3.3, Eq. 5, for decode step `step`:
 *   h_t(b, j) = h_{t-1}(pi_t(b), j) for 0 <= j < t-1,  h_t(b, t-1) = pi_t(b).
 * Global beam selection may reorder, duplicate or drop beams; only these
 * integer indices change, never the stored records.
 *   step       t; must be the next step (0 after init/reset)
 *   width      W_t, 1 <= W_t <= max_beams
 *   parents    device int32 [R][W_t], pi_t(b) in [0, W_{t-1}) indexing the
 *              previous step's beams of the same request; must be NULL at
 *              step 0 (every beam starts from S_ctx)
 *   gather_out optional device int32 [R][W_t][t]: receives h_t (the record
 *              slot of each beam's ancestor at steps 0..t-1); may be NULL
 * A parent out of range is detected on the device: that beam's indices
 * become -1 (its later outputs are unspecified but no out-of-bounds access
 * happens) and onela_get_device_status reports ONELA_EPARENT.
 * Host errors: ONELA_EINVAL, ONELA_ESTEP, ONELA_ECAPACITY, ONELA_EHIP. */
onela_status_t onela_resolve_ancestry(onela_ctx_t ctx, int32_t step,
                                      int32_t width, const int32_t* parents,
                                      int32_t* gather_out);

/* Appends the records of step `step` into the arena (Sec. 3.3: records are
 * written once to the physical slots of the current step and never
 * relocated).  Slot b of step t holds beam b's (k, v, alpha, beta).  With
 * ONELA_RECORDS_BORROW nothing is enqueued: the four buffers become step t's
 * slab and must stay valid for the rest of the beam search.
 *   k     device [R][W_t][H_K][d_k] io dtype
 *   v     device [R][W_t][H_V][d_v] io dtype
 *   alpha device fp32 [R][W_t][H_V]   (decay, Eq. 1)
 *   beta  device fp32 [R][W_t][H_V]   (correction strength, Eq. 1)
 * Must follow onela_resolve_ancestry(step) (which fixed W_t).  The inputs
 * may be reused by the caller once the enqueued copy has run.
 * Errors: ONELA_EINVAL, ONELA_ESTEP, ONELA_EHIP. */
onela_status_t onela_append_records(onela_ctx_t ctx, int32_t step,
                                    const void* k, const void* v,
                                    const float* alpha, const float* beta);

/* Decode step t: for every request r, live beam b < W_t and value head hv,
 *   o[r][b][hv] = S_{t,b} q_b   (Eq. 1 read-out after the step-t update),
 * where S_{t,b} is the state reached from S_ctx through the records at
 * slots h_t(b, 0), ..., h_t(b, t-1) and the beam's own step-t record.
 *   q device [R][W_t][H_K][d_k] io dtype
 *   o device fp32 [R][W_t][H_V][d_v], written completely
 * Must follow onela_append_records(step); may be repeated for the same
 * step (it reads the context and writes only o).
 * Errors: ONELA_EINVAL, ONELA_ESTEP, ONELA_EHIP. */
onela_status_t onela_decode_step(onela_ctx_t ctx, int32_t step, const void* q,
                                 float* o);

/* One whole decode step in a single launch: the ancestry update of
 * onela_resolve_ancestry, the record append of onela_append_records and the
 * read-out of onela_decode_step (Sec. 3.4 describes fusing the context
 * projection, ancestry replay, current update and record append into one
 * kernel).  Arguments have the meaning, layout and ownership given for those
 * three calls; on success the context is in the same state as after them,
 * so the two forms may be mixed from step to step.  Must be called for the
 * next step (0 after init/reset).  A bad parent is handled as in
 * onela_resolve_ancestry.
 * Errors: ONELA_EINVAL, ONELA_ESTEP, ONELA_ECAPACITY, ONELA_EHIP. */
onela_status_t onela_decode_step_fused(onela_ctx_t ctx, int32_t step, int32_t width,
                                       const int32_t* parents, const void* k,
                                       const void* v, const float* alpha,
                                       const float* beta, const void* q, float* o,
                                       int32_t* gather_out);

/* Synchronises the context's stream, returns and clears the sticky device
 * error (ONELA_OK or ONELA_EPARENT), or ONELA_EHIP.  The error covers the
 * current beam search: the step-0 decode launch of each search zeroes it,
 * and when a search resolves step 1 without having decoded step 0, the
 * resolve call zeroes it first (one extra launch). */
onela_status_t onela_get_device_status(onela_ctx_t ctx);

/* Frees the host-side context (the workspace stays the caller's). */
void onela_destroy(onela_ctx_t ctx);

/* ---- Setup helper: the post-prefill state S_ctx (Sec. 3.1) -------------
 * Eq. 1 over a prompt of P tokens from S = 0, for every request and value
 * head, fp32 state in registers.  Inputs [R][P][H_K][d_k] (k),
 * [R][P][H_V][d_v] (v), fp32 [R][P][H_V] (alpha, beta); output fp32
 * [R][H_V][d_v][d_k].  cfg supplies R, H_K, H_V, d_k, d_v and io_dtype.
 * Errors: ONELA_EINVAL, ONELA_EHIP. */
onela_status_t onela_prefill_state(const onela_config_t* cfg, int32_t prompt_len,
                                   const void* k, const void* v,
                                   const float* alpha, const float* beta,
                                   float* s0_out, void* stream);

/* ---- Chunked prefill of S_ctx (Sec. 3.1; Eq. 1 over the prompt) ----------
 * Same result as onela_prefill_state (Eq. 1 from S = 0 over the prompt, fp32
 * state), computed in chunks of 64 tokens: per chunk, the correction terms
 * delta_t of Eq. 2 solve a unit lower-triangular 64 x 64 system whose
 * matrices depend only on the chunk's own tokens (formed for all chunks in
 * parallel); a second launch then carries the state across the chunks in
 * order, on the matrix cores (fp32 products, and for bf16 keys exact products
 * of bf16 parts).  Inputs and output as for onela_prefill_state.
 * Workspace: onela_prefill_workspace_bytes(cfg, prompt_len) bytes (0 for an
 * empty prompt, or for an invalid cfg), 256-byte aligned, owned by the caller
 * and used only by the enqueued work: per (request, value head, chunk) the
 * fp32 matrices W [64][d_k], Kt^T [d_k][64], U^T [d_v][64] (in the order the
 * scan loads them) and the chunk's decay (16 copies).
 * Errors: ONELA_EINVAL, ONELA_ECAPACITY (workspace too small), ONELA_EHIP. */
size_t onela_prefill_workspace_bytes(const onela_config_t* cfg, int32_t prompt_len);
onela_status_t onela_prefill_state_chunked(const onela_config_t* cfg, int32_t prompt_len,
                                           const void* k, const void* v,
                                           const float* alpha, const float* beta,
                                           float* s0_out, void* workspace,
                                           size_t workspace_bytes, void* stream);

/* ---- Baseline: per-beam materialised states ("FullState", Sec. 2.3) ----
 * Every live beam keeps a full fp32 d_v x d_k state per value head.  One
 * call performs step t for all beams: copy the parent's state (S_ctx at
 * t = 0), apply Eq. 1, store the child's state, read out o = S q.
 * Workspace: [2][R][W_max][H_V][d_v][d_k] fp32 (double-buffered), see
 * onela_fullstate_workspace_bytes.  parents as in onela_resolve_ancestry
 * (NULL at step 0), prev_width = W_{t-1}.  Parents out of range are clamped
 * to 0 on the device and reported through *status_word (device int32, set
 * to nonzero; may be NULL).  Errors: ONELA_EINVAL, ONELA_ECAPACITY,
 * ONELA_EHIP. */
size_t onela_fullstate_workspace_bytes(const onela_config_t* cfg);
onela_status_t onela_fullstate_step(const onela_config_t* cfg, int32_t step,
                                    int32_t width, int32_t prev_width,
                                    const int32_t* parents, const float* s0,
                                    const void* q, const void* k, const void* v,
                                    const float* alpha, const float* beta,
                                    float* o, void* workspace,
                                    size_t workspace_bytes, int32_t* status_word,
                                    void* stream);

/* ---- Global beam selection (Sec. 2.1) ------------------------------------
 * After a decode step every live beam p < W_prev of a request is expanded
 * over the V entries of the SID codebook, and the global top-W candidates
 * become the next step's beams: candidate (p, v) has flat index p * V + v and
 * score beam_scores[p] + logp[p][v] (one fp32 addition; logp[p][v] alone when
 * beam_scores is NULL).  Order: higher score first, equal scores by lower
 * flat index, -0.0 below +0.0, every NaN below every number (NaNs among
 * themselves by flat index).  The result is unique.
 *   logp         device fp32 [R][W_prev][V]
 *   beam_scores  device fp32 [R][W_prev], or NULL
 *   parents_out  device int32 [R][W]: p of the b-th best candidate, i.e. the
 *                pi(b) that onela_resolve_ancestry takes for the next step
 *   tokens_out   device int32 [R][W]: its codebook entry v
 *   scores_out   device fp32 [R][W]: its candidate score (bit-exact)
 *   workspace    device, >= the size from onela_select_workspace_bytes,
 *                256-byte aligned; owned by the caller.  It must be
 *                zero-filled before its first use (e.g. one hipMemsetAsync
 *                when it is allocated): its first 129 KiB hold what the
 *                workgroups of one launch use to exchange a bound (a call
 *                counter, per-request bound words, wave summaries tagged
 *                with the call), and every call leaves them ready for the
 *                next, so a workspace may serve any number of calls of any
 *                shape, one at a time
 *   stream       hipStream_t (NULL: the default stream)
 * Limits: 1 <= R <= 65536, 1 <= W <= min(4096, W_prev * V),
 * W_prev * V <= 2^29.  All pointers 4-byte aligned.  Enqueued asynchronously;
 * the inputs must stay valid until the work has run.  Calls sharing one
 * workspace must not overlap (one stream, or the caller serialises them).
 * Errors: ONELA_EINVAL (limits, pointers), ONELA_ECAPACITY (workspace too
 * small), ONELA_EHIP. */
onela_status_t onela_select_workspace_bytes(int32_t num_requests, int32_t prev_width,
                                            int32_t vocab, int32_t width, size_t* bytes);
onela_status_t onela_select_beams(int32_t num_requests, int32_t prev_width, int32_t vocab,
                                  int32_t width, const float* logp,
                                  const float* beam_scores, int32_t* parents_out,
                                  int32_t* tokens_out, float* scores_out, void* workspace,
                                  size_t workspace_bytes, void* stream);

/* ---- Beam selection without a workspace ---------------------------------
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * selection, arguments, order and result as onela_select_beams, with the
 * workspace taken from a device array of the library instead of an argument.
 * Each GPU the library runs on holds its own 32 MiB array until the process
 * ends (its address is looked up once per device, on the first call with
 * that device current).  Calls whose workspace (onela_select_workspace_bytes)
 * would exceed 32 MiB return ONELA_ECAPACITY and enqueue nothing.  Nothing
 * is allocated by this call.  Every call on one GPU shares that GPU's array:
 * calls that overlap on one GPU (different streams, or host threads) race
 * and must be serialised by the caller; consecutive calls on one stream are
 * safe.  Errors: ONELA_EINVAL, ONELA_ECAPACITY, ONELA_EHIP. */
onela_status_t onela_select_beams_noalloc(int32_t num_requests, int32_t prev_width,
                                          int32_t vocab, int32_t width, const float* logp,
                                          const float* beam_scores, int32_t* parents_out,
                                          int32_t* tokens_out, float* scores_out,
                                          void* stream);

/* ---- Capacity model (host only) -----------------------------------------
 * Persistent recurrent-state bytes after `steps` decode steps for one GDN
 * layer (Sec. 4.4): one S_ctx per request and value head (state_bytes per
 * element) plus one record per (step, beam, value head).  record_bytes is
 * the size of one record; the paper's (alpha fp32, delta 16-bit, k 16-bit)
 * record at d_k = d_v = 128 is 516 bytes.  The FullState equivalent is
 * onela_fullstate_capacity_bytes.  Return 0 on invalid arguments. */
uint64_t onela_capacity_bytes(int32_t num_requests, int32_t num_v_heads,
                              int32_t d_k, int32_t d_v, int32_t beams,
                              int32_t steps, int32_t state_bytes,
                              int32_t record_bytes);
uint64_t onela_fullstate_capacity_bytes(int32_t num_requests,
                                        int32_t num_v_heads, int32_t d_k,
                                        int32_t d_v, int32_t beams,
                                        int32_t state_bytes);

#ifdef __cplusplus
}
#endif

#endif /* ONELA_H */
