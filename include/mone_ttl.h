/*
 * mone_ttl.h -- C ABI of the MI355X (gfx950) MoNe test-time-learning library.
 *
 * MoNe (Modular Neural Memory) attaches a fast-weight memory network to every layer of a
 * frozen Transformer.  A long context is consumed in segments of T tokens (Sec. 3.1); for each
 * segment, every layer's memory takes one gradient step on an associative loss computed from
 * that layer's own hidden states only (Sec. 3.3, Sec. 3.4), and after the last segment the
 * memory is read on query tokens without being updated (Eq. read).
 *
 * The memory, loss and optimiser implemented here are a fully specified variant of the paper's:
 *   memory   M(x) = W2 . SiLU(W1 . x), a 2-layer MLP d -> h -> D (D = 2*d_kv), no biases,
 *            output [K | V] (the SwiGLU memory of Eq. swiglu without its gate branch);
 *   targets  t = [W_k x ; W_v x] from the frozen projections (Eq. proj), no preprocessing;
 *   loss     L_s = (1/n) sum_j ||M(x_j) - t_j||^2 over the n tokens of the segment
 *            (segment-level average of Sec. 3.3; MONE_LOSS_MSE_MEAN also divides by D), or
 *            the paper's negative inner product L_s = -(1/n) sum_j t_j . M(x_j)
 *            (Eq. mem_loss; MONE_LOSS_NIP);
 *   update   W <- W - lr * dL_s/dW for W1 and W2, both gradients taken at W_{s-1}
 *            (Eq. update with a plain SGD step),
 *            or, with MONE_OPT_PAPER (mone_ttl_init_paper), the paper's own optimiser: a
 *            softplus per-token learning rate, momentum with a sigmoid decay predicted from
 *            the segment, and a channel-wise L2 renormalisation after each update (the
 *            exact form is stated at mone_ttl_init_paper).
 *
 * Conventions for every call:
 *   - Matrices are row-major.  W1 is [h][d] (acts on column vectors: z = W1 x), W2 is [D][h],
 *     W_kv is [D][d] = [W_k ; W_v] (rows [0, d_kv) give K, rows [d_kv, D) give V).  A tensor
 *     "[L][...]" holds the L layers back to back with no padding.
 *   - Device pointers are HIP device addresses, 16-byte aligned, owned by the caller; the
 *     library never allocates device memory.  Host pointers are marked "host".
 *   - `stream` is a hipStream_t (NULL = the null stream).  Calls only enqueue work on it,
 *     except where a call says it synchronises.  A handle must not be used from two threads
 *     at once.
 *   - Every call returns a mone_status.  Arguments are validated on the host before any HIP
 *     call; a failing call enqueues nothing and leaves the state untouched.
 *     mone_ttl_last_error() returns a message for the last failure of the calling thread.
 *   - GPU-path limits: d_model, d_hidden and d_kv must be multiples of 64 (MONE_EUNSUPPORTED
 *     otherwise); seg_len is at most 65536.
 */
#ifndef MONE_TTL_H
#define MONE_TTL_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  MONE_OK = 0,
  MONE_EINVAL = -1,       /* bad argument: null/misaligned pointer, bad size, bad enum */
  MONE_EUNSUPPORTED = -2, /* valid but outside the GPU path's limits */
  MONE_EHIP = -3,         /* a HIP runtime call or kernel launch failed */
  MONE_ESTATE = -4        /* the handle is not usable for this call */
} mone_status;

typedef enum { MONE_F32 = 0, MONE_BF16 = 1 } mone_dtype;

typedef enum {
  MONE_LOSS_MSE_SUM = 0,  /* l_j = ||y_j - t_j||^2; dL_s/dY = (2/n)(Y - T) */
  MONE_LOSS_MSE_MEAN = 1, /* l_j = ||y_j - t_j||^2 / D; dL_s/dY = (2/(n D))(Y - T) */
  MONE_LOSS_NIP = 2       /* the paper's negative inner product (Eq. mem_loss) with the whole
                             target row: l_j = -t_j . y_j; dL_s/dY = -(1/n) T, which does not
                             involve Y, so the forward of the memory's output layer is skipped */
} mone_loss;

typedef enum {
  MONE_OPT_SGD = 0,   /* W -= lr * grad (mone_ttl_init) */
  MONE_OPT_PAPER = 1  /* per-token rates, momentum, renormalisation (mone_ttl_init_paper) */
} mone_optimizer;

typedef struct {
  int32_t n_layers;  /* L >= 1: layers with a memory */
  int32_t d_model;   /* d: width of the hidden states x (memory input) */
  int32_t d_hidden;  /* h: memory hidden width */
  int32_t d_kv;      /* width of K and of V; the memory output is D = 2*d_kv */
  int32_t seg_len;   /* T: maximum tokens per segment */
  int32_t act_dtype; /* mone_dtype of x, x_q, W_kv and stored intermediates; the fast weights
                        are always fp32 */
  int32_t loss;      /* mone_loss */
  float lr;          /* learning rate (finite, may be 0); with MONE_OPT_PAPER it scales the
                        per-token rates */
  int32_t optimizer; /* mone_optimizer */
  int32_t block_tokens; /* block form of mone_ttl_segments: tokens per block.  0 chooses:
                           8 segments, at most 1024 tokens (512 at seg_len 64, 1024 at 128 and
                           256), when the block form applies (plain SGD, a squared-error loss,
                           seg_len a multiple of 64 of at most 256) and the fast weights of all
                           layers hold at least 2^24 elements, else none.  Negative: none.
                           Positive: a multiple of seg_len, from 2 * seg_len to 4096, where the
                           block form applies (else MONE_EUNSUPPORTED). */
} mone_ttl_config;

typedef struct mone_ttl mone_ttl; /* opaque host object */

/* Number of workspace bytes a handle for `cfg` needs.  It depends on L, d, h, d_kv, T, the
 * activation dtype and the optimiser only -- never on the context length N, which is not an
 * argument anywhere: the memory's footprint is constant in N (Sec. 4.3).  It includes a fixed
 * 16 MiB area for split-contraction partial sums (short segments and query batches).  Returns 0
 * if `cfg` is invalid or unsupported (mone_ttl_last_error() says why). */
size_t mone_ttl_workspace_bytes(const mone_ttl_config* cfg);

/* Create a handle over caller-owned state (the initial state W_0, s = 0 in Sec. 3.1).
 *   wkv        [L][D][d] act_dtype, frozen; borrowed, must stay valid and unchanged while the
 *              handle lives.
 *   w1         [L][h][d] fp32 fast weights W1; borrowed and updated in place by
 *              mone_ttl_segment.
 *   w2         [L][D][h] fp32 fast weights W2; as w1.
 *   workspace  device buffer of at least mone_ttl_workspace_bytes(cfg) bytes, owned by the
 *              handle until mone_ttl_destroy; 256-byte aligned.
 * Enqueues on `stream` the clearing of the workspace and the construction of the handle's
 * internal copies of w1/w2 (activation-dtype and transposed copies).  Writing w1/w2 from
 * outside while the handle lives makes those copies stale: create a new handle instead (a
 * checkpoint is a copy of w1/w2; resuming is mone_ttl_init on the copy).
 * On success *out receives the handle; on failure *out is left NULL. */
int mone_ttl_init(mone_ttl** out, const mone_ttl_config* cfg, const void* wkv, float* w1,
                  float* w2, void* workspace, size_t workspace_bytes, void* stream);

/* The paper's optimiser (Sec. 3.3, Eq. update; implementation details, App. A.2), whose
 * exact form the paper leaves open; the reading implemented, per layer and segment of n tokens:
 *   eta_j  = lr * softplus(u . x_j + b_u)            per-token learning rate
 *   beta   = sigmoid(v . mean_j(x_j) + b_v)          momentum decay, one per layer and segment
 *   g      = gradient of (1/n) sum_j eta_j l_j at W_{s-1}
 *   mu     = beta * mu + g;   W = W - mu             (for W1 and W2; mu starts as given)
 *   W      = W with each row (output channel) rescaled to the L2 norm it had in the weights
 *            the handle was created from (a row of norm 0 stays as it is).
 * Since the rescaling keeps every row norm, resuming from a checkpoint (a copy of w1, w2, mom1,
 * mom2) restores the same targets.  Pointers (device, fp32, 16-byte aligned, borrowed for the
 * handle's lifetime; u and v are read, mom1 and mom2 are state updated in place): */
typedef struct {
  const float* rate_w;   /* u   [L][d] */
  const float* rate_b;   /* b_u [L] */
  const float* decay_w;  /* v   [L][d] */
  const float* decay_b;  /* b_v [L] */
  float* mom1;           /* mu of W1 [L][h][d]; zero for a fresh state */
  float* mom2;           /* mu of W2 [L][D][h]; zero for a fresh state */
} mone_paper_optimizer;

/* mone_ttl_init for cfg->optimizer == MONE_OPT_PAPER (mone_ttl_init rejects that value, this
 * call rejects any other).  Also enqueues the computation of the row norms of w1 and w2 (the
 * renormalisation targets).  Errors as mone_ttl_init; opt and every pointer in it must be
 * non-NULL. */
int mone_ttl_init_paper(mone_ttl** out, const mone_ttl_config* cfg, const void* wkv, float* w1,
                        float* w2, const mone_paper_optimizer* opt, void* workspace,
                        size_t workspace_bytes, void* stream);

/* One test-time-learning step of every layer on one segment (Eq. update; Sec. 3.4).
 *   x         [L][n_tokens][d] act_dtype: the segment's hidden states at each layer.
 *   n_tokens  0 <= n_tokens <= seg_len.  The loss averages over the n_tokens tokens present
 *             (a short final segment); n_tokens = 0 is a no-op (an empty segment has no
 *             gradient).
 * For each layer l independently: Z = X W1^T, A = SiLU(Z), R = A W2^T - X W_kv^T,
 * G = c R, W2 -= lr G^T A, W1 -= lr ((G W2) * SiLU'(Z))^T X, both gradients at the weights
 * the call started from.  All L layers run as one grouped launch per stage.  Segments must be
 * enqueued in context order (Sec. 3.4: W_0 -> W_1 -> ... -> W_S); `x` may be reused or freed
 * once the enqueued work has completed on `stream`.
 * Graph capture: the call enqueues kernels only (no allocation, memset or synchronisation), so
 * it may be captured in a HIP graph, with the timing hooks off.  Consecutive calls alternate
 * between two internal copies of W2^T (the backward reads the previous one while the update
 * writes the next), so a graph must capture an even number of consecutive calls with the same
 * n_tokens; replaying it then continues the handle's sequence, and eager calls may follow. */
int mone_ttl_segment(mone_ttl* h, const void* x, int32_t n_tokens, void* stream);

/* For callers that cannot allocate device memory (code under stream capture, tight serving
 * loops, hosts that forbid hipMalloc): one SGD step of every layer on one segment, exactly the
 * step of mone_ttl_init followed by mone_ttl_segment, with no handle and no caller workspace.
 *   cfg, wkv, w1, w2, x, n_tokens, stream: as for mone_ttl_init and mone_ttl_segment; w1 and
 *            w2 are updated in place.  cfg->optimizer must be MONE_OPT_SGD.
 * The workspace is a static device array of 64 MiB inside the library, one per device, held
 * until the process ends; its address is taken once per device, on the first call with that
 * device current.  Every call clears it and rebuilds the weight copies from w1 and w2, so
 * consecutive calls continue the TTL chain W_0 -> W_1 -> ... like consecutive
 * mone_ttl_segment calls.  All calls on one device share the array: calls that overlap on one
 * device (other streams, other threads) race and must not be issued.
 * No hipMalloc, hipFree or other allocation, host or device.  Returns MONE_EUNSUPPORTED, before
 * any HIP call, for a configuration whose workspace (mone_ttl_workspace_bytes) exceeds 64 MiB,
 * and for MONE_OPT_PAPER. */
int mone_ttl_step_noalloc(const mone_ttl_config* cfg, const void* wkv, float* w1, float* w2,
                          const void* x, int32_t n_tokens, void* stream);

/* Several consecutive segments of seg_len tokens in one call (Sec. 3.1: the context read
 * segment after segment; Sec. 3.4: each layer's chain W_0 -> W_1 -> ... in context order):
 * the same as n_segments calls of mone_ttl_segment with n_tokens = seg_len, up to rounding.
 *   x             the segments' hidden states: token t of segment s of layer l at
 *                 x + l * layer_stride + (s * seg_len + t) * d_model (elements of act_dtype),
 *                 i.e. each layer's part of the context in one piece.
 *   layer_stride  elements between layers, >= n_segments * seg_len * d_model; x and
 *                 layer_stride * element size 16-byte aligned.
 *   n_segments    >= 0 (0 is a no-op).
 * With a block form (cfg->block_tokens; by default for short segments of large memories,
 * whose steps are bound by rewriting every fast weight for few tokens), the segments run in
 * blocks of block_tokens / seg_len: a block computes each segment's step at the weights it
 * started from plus the earlier segments' updates, which enter through T x T products of the
 * segments' tokens, hidden activations and loss gradients (exact algebra of the sequential
 * chain, summed in another order), and writes the fast weights once per block (a last
 * block may hold fewer segments; a single one runs alone).  Otherwise the segments run one by
 * one.  The workspace of such configurations includes the block's buffers
 * (mone_ttl_workspace_bytes).  With the paper's optimiser the row renormalisations of W1
 * and W2 are carried between the call's segments as pending row scales (applied to the
 * forward products, the stored loss gradient and the next updates) and written into w1, w2
 * and their copies after the last segment, so w1 and w2 hold the renormalised weights when
 * the call's work completes, equal to those of one call per segment up to rounding.
 * mone_ttl_loss then reports the last segment's loss. */
int mone_ttl_segments(mone_ttl* h, const void* x, int64_t layer_stride, int32_t n_segments,
                      void* stream);

/* Read of the current state on query-side inputs, without any update (Eq. read; Sec. 3.4):
 *   KV = W2 SiLU(W1 x_q) for every query row of every layer.
 *   xq       [L][q][d] act_dtype.
 *   q        >= 0 query rows (q = 0 is a no-op).
 *   kv       [L][q][D] of kv_dtype (MONE_F32 or MONE_BF16); columns [0, d_kv) are K,
 *            [d_kv, D) are V.
 * The fast weights are not modified, so the call may be repeated (with identical results)
 * and further segments may follow it (incremental extension, multi-query reuse).  It uses the
 * handle's scratch space, so it must not overlap with another call on the same handle. */
int mone_memory_kv(mone_ttl* h, const void* xq, int32_t q, void* kv, int32_t kv_dtype,
                   void* stream);

/* Memory injection into attention at read time (Eq. attn, with the scaled softmax attention of
 * Eq. std_attn).  The memory's K/V rows for the query tokens (mone_memory_kv's output) join the
 * keys and values of those tokens in one softmax, per layer l and query head a:
 *   out_i = softmax over j <= i of [ q_i.k_j / sqrt(dh) , q_i.km_j / sqrt(dh) ]
 *           applied to [ v_j , vm_j ]
 * where head a reads key/value head a / (n_heads / n_kv_heads) (grouped-query attention) and
 * the memory row j = [km_j | vm_j] is the memory's output on query token j.  In this form the
 * memory's output is already in key/value space (it is trained against [W_k x ; W_v x]), so it
 * is used as it is.
 *   qh      [L][q][n_heads*dh] act_dtype: the query tokens' attention queries
 *   kh, vh  [L][q][n_kv_heads*dh] act_dtype: their keys and values; dh = d_kv / n_kv_heads,
 *           at most 256
 *   kv_mem  [L][q][D] of kv_dtype (MONE_F32 or MONE_BF16), K columns [0, d_kv), V [d_kv, D)
 *   out     [L][q][n_heads*dh] of out_dtype
 * n_heads must be a multiple of n_kv_heads and n_kv_heads must divide d_kv.  Uses nothing of
 * the handle but its shape (L, d_kv, act_dtype); q = 0 is a no-op.  The work is O(q^2) per
 * head (16 query rows per workgroup, keys in chunks of 32 of each set): it is meant for query
 * batches, not for long prefills. */
int mone_memory_attention(mone_ttl* h, const void* qh, const void* kh, const void* vh,
                          const void* kv_mem, int32_t kv_dtype, int32_t q, int32_t n_heads,
                          int32_t n_kv_heads, void* out, int32_t out_dtype, void* stream);

/* The segment loss L_s of the last mone_ttl_segment call, per layer, evaluated at the weights
 * that step started from (the loss of Sec. 3.3 for that segment).  out_host: host float[L].
 * Synchronises `stream`.  MONE_ESTATE if no non-empty segment has been processed yet;
 * MONE_EUNSUPPORTED for MONE_LOSS_NIP with MONE_OPT_PAPER (the step there only forms the
 * rate-weighted gradient, not the plain loss). */
int mone_ttl_loss(mone_ttl* h, float* out_host, void* stream);

/* Destroy a handle (host memory only; the caller frees its device buffers afterwards, once
 * the enqueued work has completed).  NULL is accepted. */
int mone_ttl_destroy(mone_ttl* h);

/* Message of the last failing call on this thread ("" if none).  Valid until the next call. */
const char* mone_ttl_last_error(void);

/* ---- measurement hooks ---------------------------------------------------------------- */

/* Stages of one segment and of one read, in launch order. */
#define MONE_STAGE_XT 0    /* X -> X^T staging copy (operand of the W1 gradient) */
#define MONE_STAGE_FWD1 1  /* Z = X W1^T; A = SiLU(Z) */
#define MONE_STAGE_FWD2 2  /* R = A W2^T - X W_kv^T; G = c R (times the rates); loss partials */
#define MONE_STAGE_BWD 3   /* dZ = (G W2) * SiLU'(Z), and the W2 update (one grouped launch) */
#define MONE_STAGE_UPD 4   /* the W1 update (dZ^T X) */
#define MONE_STAGE_KV1 5   /* read: A_q = SiLU(X_q W1^T) */
#define MONE_STAGE_KV2 6   /* read: KV = A_q W2^T */
#define MONE_STAGE_RATE 7  /* MONE_OPT_PAPER: per-token rates and the momentum decay */
#define MONE_STAGE_RENORM 8 /* MONE_OPT_PAPER: row renormalisation of W1, W2 and their copies */
#define MONE_STAGE_ATTN 9  /* mone_memory_attention */
#define MONE_STAGE_BFWD 10 /* block form: X W1^T, the targets and the token Gram X X^T */
#define MONE_STAGE_BSEQ 11 /* block form: one segment's corrected forward, loss gradient and
                              backward (five launches) */
#define MONE_STAGE_BUPD 12 /* block form: the block's W2 and W1 updates */
#define MONE_N_STAGES 13

/* Enable (max_records > 0) or disable (0) per-stage timing: each subsequent launch of a stage
 * whose bit is set in stage_mask (bit i = stage i; MONE_ALL_STAGES for every stage) is
 * bracketed by a pair of HIP events recorded on the call's stream, up to max_records pairs
 * (further launches are not timed).  The events are created on the current device without a
 * system-scope fence (timing only: recording them does not write back or invalidate caches
 * between the timed kernels).  Host call, no device allocation.  Enabling again discards
 * earlier records. */
#define MONE_ALL_STAGES 0xffffffffu
int mone_ttl_set_stage_timing(mone_ttl* h, int32_t max_records, uint32_t stage_mask);

/* Synchronise on the recorded events and report, per stage, the summed elapsed milliseconds
 * (ms_sum, host double[MONE_N_STAGES]) and the number of timed launches (count, host
 * int32[MONE_N_STAGES]); then clear the records. */
int mone_ttl_stage_times(mone_ttl* h, double* ms_sum, int32_t* count);

#ifdef __cplusplus
}
#endif

#endif /* MONE_TTL_H */
