/*
 * mone_swiglu.h -- C ABI of the paper-form MoNe memory on MI355X (gfx950): a SwiGLU MLP per
 * fast-weight head (Sec. 3.2, Eq. swiglu; App. A.2), trained at test time with the negative
 * inner product loss (Sec. 3.3, Eq. mem_loss) on preprocessed keys and values.
 *
 * Per layer and segment of n tokens with hidden states x_j (j = 0 .. n-1, the token's index in
 * its segment), for every head e of width d_h (the memory's width H d_h equals d_model):
 *   keys     k_j = RoPE_j( L2( SiLU( s * (P_k x_j) + b ) ) )   per head: L2 divides by
 *            max(||k_{j,e}||, 1e-12); RoPE_j turns the channel pairs (c, c + d_h/2) of each
 *            head by the angle j * base^(-2c/d_h) (segment-local positions, Sec. 3.3)
 *   values   v_j = SiLU(P_v x_j)                                 (Eq. proj with App. A.2)
 *   memory   y_{j,e} = W_out^T ( SiLU(W_in k_{j,e}) * (W_gate k_{j,e}) )   (Eq. swiglu)
 *   loss     L_s = -(1/n) sum_j sum_e v_{j,e} . y_{j,e}                       (Eq. mem_loss)
 *   update   SGD: W <- W - lr dL_s/dW for the 3 H matrices of the layer (Eq. update), or the
 *            paper's optimiser (MONE_OPT_PAPER): eta_j = lr softplus(u . x_j + b_u) weights
 *            token j's gradient, mu = beta mu + g with beta = sigmoid(v . mean_j x_j + b_v),
 *            W = W - mu, then every row of every matrix is rescaled to the L2 norm it had in
 *            the weights the handle was created from (a row of norm 0 stays as it is).
 * The gradient at the memory's output, -eta_j v_j / n, does not involve the output, so the
 * memory's forward output is never formed during learning; the loss is summed from the hidden
 * activations against their gradient.
 *
 * Conventions are those of mone_ttl.h (row-major, caller-owned 16-byte-aligned device buffers,
 * host-side validation, mone_status return codes, mone_ttl_last_error()).
 * GPU-path limits: d_model a multiple of 64, d_head a multiple of 16 in [16, 256], seg_len at
 * most 65536 (MONE_EUNSUPPORTED otherwise).
 */
#ifndef MONE_SWIGLU_H
#define MONE_SWIGLU_H

#include <stddef.h>
#include <stdint.h>

#include "mone_ttl.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct {
  int32_t n_layers;  /* L >= 1 */
  int32_t d_model;   /* d: width of the hidden states x, = n_heads * d_head */
  int32_t n_heads;   /* H: fast-weight heads per layer */
  int32_t d_head;    /* d_h: head width (even) */
  int32_t seg_len;   /* T: maximum tokens per segment */
  int32_t act_dtype; /* mone_dtype of x, the projections and the stored intermediates; the
                        fast weights are always fp32 */
  int32_t optimizer; /* mone_optimizer */
  float lr;          /* learning rate (finite, may be 0); scales the paper optimiser's rates */
  float rope_base;   /* RoPE base (> 0; the usual value is 10000) */
  int32_t prep_segments; /* segments whose weight-independent preprocessing (rates, projections,
                            key normalisation and RoPE) mone_swiglu_segments computes in one
                            batch, in [0, 16]: 0 chooses 8 when seg_len is a multiple of 64
                            (else 1); above 1 needs seg_len a multiple of 64.  The workspace
                            holds that many copies of the preprocessing buffers, and above 1
                            two sets of the copies the memory steps read. */
} mone_swiglu_config;

/* Frozen parameters (borrowed for the handle's lifetime, read only). */
typedef struct {
  const void* proj;      /* [L][2d][d] act_dtype: rows [0, d) are P_k, rows [d, 2d) are P_v */
  const float* k_scale;  /* [L][d] fp32: per-channel scale s of the keys' affine step */
  const float* k_shift;  /* [L][d] fp32: per-channel shift b */
} mone_swiglu_frozen;

/* Fast weights: fp32 [L][H][d_h][d_h] each, borrowed and updated in place.  Head e of layer l
 * maps a key row k to (SiLU(k W_in^T) * k W_gate^T) W_out. */
typedef struct {
  float* w_in;
  float* w_gate;
  float* w_out;
} mone_swiglu_weights;

/* State of the paper's optimiser (fp32, borrowed; u and v read, the momenta updated in place,
 * zero for a fresh state). */
typedef struct {
  const float* rate_w;   /* u   [L][d] */
  const float* rate_b;   /* b_u [L] */
  const float* decay_w;  /* v   [L][d] */
  const float* decay_b;  /* b_v [L] */
  float* mom_in;         /* [L][H][d_h][d_h] */
  float* mom_gate;
  float* mom_out;
} mone_swiglu_optimizer;

typedef struct mone_swiglu mone_swiglu; /* opaque host object */

/* Workspace bytes for `cfg` (0 if invalid or unsupported).  Independent of the context
 * length. */
size_t mone_swiglu_workspace_bytes(const mone_swiglu_config* cfg);

/* Create a handle over caller-owned state.  `opt` must be NULL for MONE_OPT_SGD and non-NULL
 * (every pointer set) for MONE_OPT_PAPER.  The workspace (256-byte aligned, at least
 * mone_swiglu_workspace_bytes(cfg) bytes) is owned by the handle until mone_swiglu_destroy.
 * Enqueues on `stream` the clearing of the workspace, the construction of the handle's MFMA
 * copies of the fast weights, the RoPE table and, for MONE_OPT_PAPER, the row norms of the
 * weights (the renormalisation targets).  As with mone_ttl_init, writing the fast weights from
 * outside while the handle lives makes its copies stale; a checkpoint is a copy of the weights
 * (and momenta), and resuming is a new handle on the copy. */
int mone_swiglu_init(mone_swiglu** out, const mone_swiglu_config* cfg,
                     const mone_swiglu_frozen* frozen, const mone_swiglu_weights* weights,
                     const mone_swiglu_optimizer* opt, void* workspace, size_t workspace_bytes,
                     void* stream);

/* One test-time-learning step of every layer on one segment.
 *   x         [L][n_tokens][d] act_dtype.
 *   n_tokens  0 <= n_tokens <= seg_len; 0 is a no-op.  Positions restart at 0 in every
 *             segment.
 * Segments must be enqueued in context order.  The call enqueues kernels only (no allocation,
 * memset or synchronisation) and keeps no state that alternates between calls, so one call may
 * be captured in a HIP graph (timing hooks off) and replayed once per segment. */
int mone_swiglu_segment(mone_swiglu* h, const void* x, int32_t n_tokens, void* stream);

/* Several consecutive whole segments of seg_len tokens in one call (Sec. 3.1; each layer's
 * chain in context order, Sec. 3.4): the same as n_segments calls of mone_swiglu_segment.
 *   x             token t of segment s of layer l at x + l * layer_stride + (s * seg_len + t)
 *                 * d_model (elements of act_dtype): each layer's part of the context in one
 *                 piece.
 *   layer_stride  elements between layers, >= n_segments * seg_len * d_model; x and
 *                 layer_stride * element size 16-byte aligned.
 *   n_segments    >= 0 (0 is a no-op).
 * The preprocessing that does not depend on the fast weights (the paper optimiser's rates and
 * decay, the key/value projections with their affine step and SiLU, the keys' normalisation
 * and segment-local RoPE) runs once for up to prep_segments segments at a time, as larger
 * launches; each segment's memory step (DA, FWD, UPD) then follows in order.  With more than
 * one such batch, the preprocessing of the next batch runs on an internal stream of the handle
 * (default priority) beside the memory steps of the current one; the internal stream starts
 * after the work queued on `stream` before the call and `stream` waits for it before the call's
 * end, so the call orders like one stream and can be captured in a HIP graph.  Calls on one
 * handle must not overlap. */
int mone_swiglu_segments(mone_swiglu* h, const void* x, int64_t layer_stride, int32_t n_segments,
                         void* stream);

/* The segment loss L_s of the last non-empty segment, per layer, at the weights that step
 * started from (unweighted by the rates).  out_host: host float[L].  Synchronises `stream`.
 * MONE_ESTATE before the first non-empty segment. */
int mone_swiglu_loss(mone_swiglu* h, float* out_host, void* stream);

/* Frozen parameters of the read (borrowed for the duration of a call, read only). */
typedef struct {
  const void* proj_q;    /* [L][d][d] act_dtype: the query projection P_q */
  const float* q_scale;  /* [L][d] fp32: per-channel scale of the queries' affine step */
  const float* q_shift;  /* [L][d] fp32: per-channel shift */
  const float* rms_w;    /* [L][d] fp32: per-channel weight of the memory tokens' RMSNorm */
  const float* gate_w;   /* [L][H][d] fp32: per-head gate vectors a_e */
  const float* gate_b;   /* [L][H] fp32: per-head gate biases c_e */
  const void* w_kv;      /* [L][2 d_kv][d] act_dtype: the backbone's [W_k ; W_v] */
  int32_t d_kv;          /* width of K and of V (a multiple of 64) */
} mone_swiglu_reader;

/* Read of the current fast weights on query-side inputs, without any update (Eq. read, with the
 * per-head RMSNorm and gate of Sec. 3.2 and the projection of Eq. attn), per layer and query
 * token j (positions j = 0 .. q-1):
 *   q_j   = RoPE_j( L2( SiLU( s_q * (P_q x_j) + b_q ) ) )        per head, as the keys
 *   o_j,e = M_e(q_j,e)                                              the memory, head e
 *   h_j,e = o_j,e / sqrt(mean(o_j,e^2) + 1e-6) * w_rms,e * SiLU(a_e . x_j + c_e)
 *   kv_j  = [ h_j W_k^T | h_j W_v^T ]                               the memory token's K and V
 *   xq       [L][q][d] act_dtype.
 *   q        0 <= q <= seg_len rounded up to a multiple of 256; q = 0 is a no-op.
 *   kv       [L][q][2 d_kv] of kv_dtype (MONE_F32 or MONE_BF16): K columns [0, d_kv), V after.
 * The fast weights are not modified.  The call uses the handle's scratch space, so it must not
 * overlap with another call on the same handle. */
int mone_swiglu_read(mone_swiglu* h, const mone_swiglu_reader* rd, const void* xq, int32_t q,
                     void* kv, int32_t kv_dtype, void* stream);

/* Memory injection into attention for the paper-form memory: exactly mone_memory_attention
 * (Eq. attn, Eq. std_attn; grouped heads, causal over the query keys and the memory rows) with
 * the memory rows kv_mem of mone_swiglu_read, for the handle's L layers and activation dtype and
 * the given d_kv. */
int mone_swiglu_attention(mone_swiglu* h, int32_t d_kv, const void* qh, const void* kh,
                          const void* vh, const void* kv_mem, int32_t kv_dtype, int32_t q,
                          int32_t n_heads, int32_t n_kv_heads, void* out, int32_t out_dtype,
                          void* stream);

/* Destroy a handle (host memory only).  NULL is accepted. */
int mone_swiglu_destroy(mone_swiglu* h);

/* ---- measurement hooks (as mone_ttl_set_stage_timing / mone_ttl_stage_times) ------------ */
#define MONE_SW_STAGE_RATE 0   /* MONE_OPT_PAPER: per-token rates and the momentum decay */
#define MONE_SW_STAGE_PROJ 1   /* [P_k x ; P_v x] for every token (one grouped GEMM) with the
                                  keys' affine step and SiLU and the values' SiLU fused */
#define MONE_SW_STAGE_KEYS 2   /* keys: per-token L2 norm per head and RoPE; K and K^T */
#define MONE_SW_STAGE_DA 3     /* dA^T = W_out dY^T per head: the hidden activations' gradient */
#define MONE_SW_STAGE_FWD 4    /* [Z | G]^T = [W_in ; W_gate] K^T per head; epilogue: A^T,
                                  dZ^T, dG^T and the loss partials */
#define MONE_SW_STAGE_UPD 5    /* the three weight gradients and the update (one launch; with
                                  MONE_OPT_PAPER also the momentum and the row renormalisation) */
#define MONE_SW_STAGE_QPROJ 6  /* read: P_q x_q with the affine step and SiLU; the gates */
#define MONE_SW_STAGE_QKEYS 7  /* read: L2 norm and RoPE of the queries */
#define MONE_SW_STAGE_QFWD 8   /* read: A = SiLU(Z) * G per head */
#define MONE_SW_STAGE_QOUT 9   /* read: O = A W_out per head, RMSNorm and gate -> h */
#define MONE_SW_STAGE_QKV 10   /* read: [h W_k^T | h W_v^T] */
#define MONE_SW_STAGE_ATTN 11  /* mone_swiglu_attention */
#define MONE_SW_N_STAGES 12

int mone_swiglu_set_stage_timing(mone_swiglu* h, int32_t max_records, uint32_t stage_mask);
int mone_swiglu_stage_times(mone_swiglu* h, double* ms_sum, int32_t* count);

#ifdef __cplusplus
}
#endif

#endif /* MONE_SWIGLU_H */
