/*
 * hybrid_attn.h -- C ABI of libhybattn, the MI355X (gfx950) block-hybrid
 * attention library.
 *
 * Method: "Retrofitting Linear Attention into Diffusion Language Models",
 * Section 3.1.  For a query q of the active block, with a per-query-head
 * feature map phi(x) = [softmax(xW), softmax(-xW)] (W in R^{d x F}, so phi has
 * f = 2F entries) and a committed-context state S (f x d), Z (f):
 *   sm_num  = sum_j exp(q.k_j/sqrt(d)) v_j,   sm_den = sum_j exp(q.k_j/sqrt(d))
 *             (j over all L tokens of the active block, no mask)
 *   lin_num = phi(q)^T S,                     lin_den = phi(q)^T Z
 *   out     = (w sm_num + lin_num) / (w sm_den + lin_den),  w = sigmoid(alpha)
 * and committing a block adds sum_t phi(k_t) v_t^T to S and sum_t phi(k_t)
 * to Z.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Memory.  Every pointer argument is a device pointer (hipMalloc'ed or
 *   equivalent), owned by the caller.  The library never allocates or frees
 *   device memory; a scratch buffer, where one is needed, is the caller's
 *   workspace of at least hybrid_workspace_bytes() bytes.
 * Alignment.  Every pointer must be 16-byte aligned.
 * Layouts.  Row-major, contiguous, outermost index first:
 *   q, out        [B][L][Hq][d]        (prefill: [B][T][Hq][d])
 *   k, v          [B][L][Hkv][d]       (prefill: [B][T][Hkv][d])
 *   W             [Hq][F][d]           row j of head h is column j of W_h;
 *                                      this is the weight layout of a linear
 *                                      layer d -> F
 *   alpha         [Hq] float           gate logits; the library forms sigmoid
 *   S             [n_slots][Hq][d][f] float   S_h stored transposed:
 *                                      entry (feature r, value dim c) of S_h
 *                                      is at c*f + r, so the f features of
 *                                      one value dim are contiguous
 *   z             [n_slots][Hq][f] float
 *   slots         [B] int32 or NULL    state slot of request b; NULL means
 *                                      slot b.  A slot outside [0, n_slots)
 *                                      makes that request's outputs NaN and
 *                                      leaves every state untouched.
 *   block_len     [B] int32 or NULL    active tokens of request b's block,
 *                                      clamped to [0, L]; NULL means L for
 *                                      every request.  Request b then acts
 *                                      as a call with L = block_len[b] on
 *                                      its first block_len[b] rows: its
 *                                      later rows of q, k and v play no part
 *                                      (their values may be anything, NaN
 *                                      included) and its later rows of out
 *                                      are not written.  0 makes the request
 *                                      a no-op.  This serves a batch whose
 *                                      requests sit in blocks of different
 *                                      lengths, e.g. a prompt's last,
 *                                      partial block.
 *   k_cache, v_cache [B][max_prefix][Hkv][d]; request b uses rows
 *                                      0 .. prefix_len[b]-1.
 *   Query head h reads KV head h / (Hq / Hkv).
 * Types.  q, k, v, W and the KV cache share dims->dtype (fp32 or bf16), and so
 *   does out unless dims->flags has HYB_OUT_F32; alpha, S and z are always
 *   fp32.  All accumulation is fp32.  On the bf16 path the matrix-core
 *   operands are bf16: phi(q) and the state read by a step are rounded to
 *   bf16 (round to nearest even), while the block softmax weights and phi(k)
 *   in a state update are carried as a bf16 pair hi + lo (about 16 bits).
 *   A bf16 out is the rounded fp32 result.
 * Execution.  Work is enqueued on `stream` (a hipStream_t; NULL = the null
 *   stream) and the call returns without synchronising.  Results are
 *   bitwise reproducible from run to run (no atomics).
 * Validation.  Every check below runs on the host before anything is
 *   enqueued.  On failure the call returns the status, enqueues nothing,
 *   touches no output and sets a message readable with hybrid_last_error().
 *   Values that live in device memory (slots, block_len, prefix_len) cannot be checked
 *   on the host; the kernels clamp or mask them as documented per call.
 * Errors after launch.  HYB_ELAUNCH reports a failed kernel launch; outputs,
 *   and for commit/prefill the state, are then undefined.
 * Threading.  Calls are reentrant; the error message is thread-local.
 */
#ifndef HYBRID_ATTN_H
#define HYBRID_ATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  HYB_OK = 0,
  HYB_ENULL = 1,        /* a required pointer is NULL                       */
  HYB_EINVAL = 2,       /* a size is out of range or inconsistent           */
  HYB_EALIGN = 3,       /* a pointer is not 16-byte aligned                 */
  HYB_EDTYPE = 4,       /* dims->dtype is not a hyb_dtype_t                 */
  HYB_EUNSUPPORTED = 5, /* no kernel for this (dtype, head_dim, feat_dim)   */
  HYB_EWORKSPACE = 6,   /* workspace missing or smaller than required       */
  HYB_ELAUNCH = 7       /* the HIP runtime rejected a launch                */
} hyb_status_t;

typedef enum { HYB_F32 = 0, HYB_BF16 = 1 } hyb_dtype_t;

typedef enum {
  HYB_OP_STEP = 0,
  HYB_OP_COMMIT = 1,
  HYB_OP_PREFILL = 2,
  HYB_OP_SOFTMAX_PREFIX = 3,
  HYB_OP_BACKWARD = 4,
  HYB_OP_BACKWARD_FULL = 5
} hyb_op_t;

typedef struct {
  int32_t batch;      /* B, requests in this call, >= 0 (0: nothing to do)   */
  int32_t n_q_heads;  /* Hq, >= 1                                            */
  int32_t n_kv_heads; /* Hkv, >= 1, divides Hq                               */
  int32_t head_dim;   /* d: 64 or 128                                        */
  int32_t block;      /* L, active-block tokens: 1..32                       */
  int32_t feat_dim;   /* f = 2F, rows of S: 64, 128 or 256                   */
  int32_t dtype;      /* hyb_dtype_t                                         */
  int32_t n_slots;    /* rows of the state pool S, z; >= 1 when batch > 0   */
  int32_t flags;      /* HYB_OUT_F32 and, for the step only, HYB_STEP_SPLIT
                         or HYB_STEP_WHOLE; any other bit is rejected      */
} hyb_dims_t;

/* flags: out is fp32 whatever dtype is (default: out has dtype).  The bf16
 * output of a call equals the round-to-nearest-even bf16 of its fp32 output
 * bit for bit. */
#define HYB_OUT_F32 1
/* flags of hybrid_attn_step only (any other entry point rejects them): which
 * of its three kernels runs.  HYB_STEP_SPLIT: one wave per (request, query
 * head, 32-column slice of d), for batches too small to fill the chip with
 * HYB_STEP_WHOLE: one workgroup per group of query heads sharing a KV head,
 * each streaming its heads' whole states.  HYB_STEP_HALVES: two workgroups
 * per group of four query heads, each streaming half of every head's state
 * columns and writing half of its output columns (bf16, feat_dim <= 128,
 * n_q_heads / n_kv_heads a multiple of 4; otherwise HYB_EUNSUPPORTED).  None:
 * the library picks by the batch (HALVES where it is supported and its
 * workgroups fill 128 to 256 compute units; else SPLIT while its
 * B * Hq * d/32 waves fit on the chip at once, 1024 of them; else HALVES
 * while its workgroups fit on the 256 compute units; else WHOLE).  More than
 * one: rejected.
 * Results agree to the same bound against the definition; they need not
 * agree bit for bit. */
#define HYB_STEP_SPLIT 2
#define HYB_STEP_WHOLE 4
#define HYB_STEP_HALVES 8

/* One denoising step of the active block (Section 3.1: within-block
 * softmax branch, linear readout of the committed state, gated merge with a
 * shared normaliser).  Reads S and z, writes out.  q, k, v, W, alpha, S, z
 * and out are required; slots and block_len may be NULL.  out must not
 * overlap an input.  Empty context (z = 0) gives plain block softmax. */
int hybrid_attn_step(const hyb_dims_t* dims, const void* q, const void* k,
                     const void* v, const void* W, const float* alpha,
                     const float* S, const float* z, const int32_t* slots,
                     const int32_t* block_len, void* out, void* stream);

/* The last denoising step of a block fused with its commit, in one launch
 * (the single kernel of Section 3.3: within-block softmax, readout, gated
 * merge and the causal state update).  out is exactly what hybrid_attn_step
 * gives on the state as it was; then, as hybrid_state_commit,
 * S_h += sum_t phi_h(k_t) v_t^T and z_h += sum_t phi_h(k_t), in place.
 * Arguments as for hybrid_attn_step, with S and z writable.  out, S and z
 * must not overlap each other or any input; two requests of one call must
 * not share a slot.  A request whose slot is out of range gets NaN outputs
 * and leaves the state untouched. */
int hybrid_attn_step_commit(const hyb_dims_t* dims, const void* q,
                            const void* k, const void* v, const void* W,
                            const float* alpha, float* S, float* z,
                            const int32_t* slots, const int32_t* block_len,
                            void* out, void* stream);

/* Commit of a finished block (Section 3.1 state update):
 * S_h += sum_t phi_h(k_t) v_t^T and z_h += sum_t phi_h(k_t) over the block
 * tokens (the first block_len[b] of request b; all L when block_len is
 * NULL), in place, for every request and query head.  Two requests of one
 * call must not share a slot. */
int hybrid_state_commit(const hyb_dims_t* dims, const void* k, const void* v,
                        const void* W, float* S, float* z,
                        const int32_t* slots, const int32_t* block_len,
                        void* stream);

/* Block-causal prefill of seq_len tokens (Figure 2 pattern): the tokens are
 * cut into seq_len / L blocks; block c is answered against the state of the
 * blocks before it (as hybrid_attn_step) and then committed.  The state
 * starts from what S, z hold, so successive calls continue one prompt.
 * seq_len must be a positive multiple of L.  out may be NULL (state only; q
 * is then ignored and may be NULL).  ws/ws_bytes: workspace of at least
 * hybrid_workspace_bytes(dims, HYB_OP_PREFILL, seq_len) bytes (may be NULL
 * when that is 0); the prompt is processed in sequence segments whose state
 * increments (and a snapshot of the incoming state, which the segments start
 * from) pass through it, so results equal the block-by-block ones up to the
 * order of fp32 additions.  It must not overlap any other argument.  Two
 * requests of one call must not share a slot. */
int hybrid_state_prefill(const hyb_dims_t* dims, int32_t seq_len,
                         const void* q, const void* k, const void* v,
                         const void* W, const float* alpha, float* S, float* z,
                         const int32_t* slots, void* out, void* ws,
                         size_t ws_bytes, void* stream);

/* Bytes of the library-held scratch buffer of hybrid_state_prefill_noalloc,
 * per GPU. */
#define HYB_NOALLOC_SCRATCH_BYTES (64u << 20)

/* hybrid_state_prefill for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): the same computation and results, bit for bit, with the
 * workspace taken from a scratch buffer the library holds on each GPU
 * (HYB_NOALLOC_SCRATCH_BYTES, kept from the first call on a device until
 * the process ends).  The call itself allocates nothing; the caller still
 * passes inputs, outputs and the state.  A call whose workspace
 * (hybrid_workspace_bytes(dims, HYB_OP_PREFILL, seq_len)) exceeds the
 * scratch size returns HYB_EWORKSPACE and enqueues nothing.  Every call on
 * one GPU shares that GPU's buffer, which keeps the last call's contents
 * (nothing in it needs to start at zero): calls whose executions overlap on
 * one GPU, e.g. on two streams, race and must not be issued. */
int hybrid_state_prefill_noalloc(const hyb_dims_t* dims, int32_t seq_len,
                                 const void* q, const void* k, const void* v,
                                 const void* W, const float* alpha, float* S,
                                 float* z, const int32_t* slots, void* out,
                                 void* stream);

/* Exact softmax attention of the active block's queries over each request's
 * cached prefix plus the block itself (the softmax teacher the hybrid layer
 * replaces; Section 2.2, without a mask inside the block).  prefix_len is a
 * device array [B]; values are clamped to [0, max_prefix].  ws/ws_bytes: at
 * least hybrid_workspace_bytes(dims, HYB_OP_SOFTMAX_PREFIX, max_prefix)
 * bytes, not overlapping any argument; when that is 0 (the prefix is not
 * split across workgroups) ws may be NULL. */
int softmax_prefix_step(const hyb_dims_t* dims, const void* q, const void* k,
                        const void* v, const void* k_cache,
                        const void* v_cache, const int32_t* prefix_len,
                        int32_t max_prefix, void* out, void* ws,
                        size_t ws_bytes, void* stream);

/* softmax_prefix_step over a paged KV cache, as a serving engine keeps it
 * (Section 3.3 keeps the hybrid state beside such a cache; the softmax
 * layers it replaces read it).  k_pages, v_pages: page pools
 * [n_pages][page_size][Hkv][d] in dims->dtype; page_table: device
 * [B][max_pages] int32, entry i of request b naming the page that holds its
 * cached tokens i*page_size .. (i+1)*page_size - 1 (token j at row
 * j % page_size).  prefix_len (device [B]) is clamped to
 * [0, max_pages * page_size]; only the first ceil(prefix_len[b] / page_size)
 * entries of a row are read, and a page number outside [0, n_pages) is
 * clamped into it (device values cannot be checked on the host).  page_size
 * is a power of two from 32 to 65536 (HYB_EUNSUPPORTED otherwise); n_pages
 * >= 1 and the page table are required when max_pages > 0.  Pages may be
 * shared by requests and appear in any order.  The result equals
 * softmax_prefix_step on the gathered contiguous cache, bit for bit.
 * ws/ws_bytes: at least hybrid_workspace_bytes(dims, HYB_OP_SOFTMAX_PREFIX,
 * max_pages * page_size) bytes (NULL when that is 0), not overlapping any
 * argument.  out must not overlap an input. */
int softmax_prefix_step_paged(const hyb_dims_t* dims, const void* q,
                              const void* k, const void* v,
                              const void* k_pages, const void* v_pages,
                              int32_t n_pages, int32_t page_size,
                              const int32_t* page_table, int32_t max_pages,
                              const int32_t* prefix_len, void* out, void* ws,
                              size_t ws_bytes, void* stream);

/* Gradient of the block-hybrid layer over a training sequence with respect
 * to its feature-map weights W and gate logits alpha: the attention transfer
 * of Section 3.2 (Stage 1), which trains only {W, alpha} with the backbone
 * frozen.  The forward is the block-causal pattern of Figure 2 from an empty
 * state (hybrid_state_prefill's outputs for a fresh request): q [B][T][Hq][d],
 * k, v [B][T][Hkv][d], W, alpha as for hybrid_attn_step, T = seq_len.
 * Objective, exactly one of:
 *   dout   [B][T][Hq][d] (dims->dtype): L = sum <dout, out>, i.e. the
 *          gradient for an upstream gradient dout; loss must be NULL;
 *   target [B][T][Hq][d] (dims->dtype): the frozen softmax teacher's output;
 *          L = sum |out - target|^2, the attention-transfer loss, formed
 *          without writing out; loss (fp32 [Hq], may be NULL) receives L per
 *          query head.
 * Outputs (fp32, overwritten, summed over the batch): dW [Hq][F][d] in W's
 * layout, dalpha [Hq].  seq_len must be a positive multiple of L.  feat_dim
 * must be 64 or 128 (HYB_EUNSUPPORTED otherwise); dims->flags must be 0;
 * n_slots is not used.  ws/ws_bytes: at least hybrid_workspace_bytes(dims,
 * HYB_OP_BACKWARD, seq_len) bytes, not overlapping any argument; outputs
 * must not overlap each other or an input.  batch 0 writes nothing.
 * Deterministic: partial sums are added in a fixed order. */
int hybrid_attn_backward(const hyb_dims_t* dims, int32_t seq_len,
                         const void* q, const void* k, const void* v,
                         const void* W, const float* alpha, const void* dout,
                         const void* target, float* dW, float* dalpha,
                         float* loss, void* ws, size_t ws_bytes, void* stream);

/* hybrid_attn_backward that also returns the gradients with respect to the
 * layer's inputs q, k and v, which end-to-end training through the hybrid
 * layers needs (Stage 2 of Section 3.2 adapts the attention projections
 * around them).  Arguments and the objective as for hybrid_attn_backward;
 * dq [B][T][Hq][d], dk and dv [B][T][Hkv][d] are fp32 whatever dims->dtype
 * is (dk and dv sum over the query heads that share each KV head), all
 * three required and overwritten.  ws/ws_bytes: at least
 * hybrid_workspace_bytes(dims, HYB_OP_BACKWARD_FULL, seq_len) bytes.  No
 * output may overlap another output, an input or the workspace.  The
 * in-block softmax weights are formed as exp(log w + q.k/sqrt(d)), so the
 * scaled scores must stay well below 80 (the W, alpha gradients share this
 * range through 1/D).  Deterministic. */
int hybrid_attn_backward_full(const hyb_dims_t* dims, int32_t seq_len,
                              const void* q, const void* k, const void* v,
                              const void* W, const float* alpha,
                              const void* dout, const void* target, float* dq,
                              float* dk, float* dv, float* dW, float* dalpha,
                              float* loss, void* ws, size_t ws_bytes,
                              void* stream);

/* Workspace bytes the given op needs for these dims; `extent` is seq_len for
 * HYB_OP_PREFILL, HYB_OP_BACKWARD and HYB_OP_BACKWARD_FULL, max_prefix for
 * HYB_OP_SOFTMAX_PREFIX, ignored otherwise.  Returns 0 for invalid dims. */
size_t hybrid_workspace_bytes(const hyb_dims_t* dims, int32_t op,
                              int32_t extent);

/* Message of the last failed call on this thread ("" if none). */
const char* hybrid_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* HYBRID_ATTN_H */
