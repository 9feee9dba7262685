// Host side of the paper-form memory (SwiGLU per fast-weight head): argument validation,
// workspace layout and the per-stage launches of a segment step.  The C ABI is declared in
// include/mone_swiglu.h.
//
// Data layout in HBM (row-major; B = L * H head operands, b = l * H + e; Tp = seg_len rounded
// up to 256; d_hp = d_h rounded up to 64, padding columns zero):
//   caller state   W_in, W_gate, W_out [L][H][d_h][d_h] fp32; P [L][2d][d] act; s, b [L][d]
//   workspace      K'   [L][Tp][d] act     keys after the affine step and SiLU
//                  K    [B][Tp][d_hp]      preprocessed keys (B operand of FWD)
//                  K^T  [B][d_h][Tp]       (B operand of the W_in / W_gate gradients)
//                  dY0  [B][Tp][d_hp]      -v / n (B operand of DA)
//                  dY^T [B][d_h][Tp]       -eta v / n (B operand of the W_out gradient)
//                  dA0^T [B][d_h][Tp]      DA's output, read by FWD's epilogue
//                  A^T  [B][d_h][Tp]       (A operand of the W_out gradient)
//                  [dZ|dG]^T [B][2 d_h][Tp] interleaved rows (A operand of the W_in/W_gate
//                                          gradients)
//                  W_ig [B][2 d_h][d_hp], W_out copy [B][d_h][d_hp]  MFMA copies
//                  RoPE table [Tp][d_h/2] (cos, sin); read gates [L][Tp][H]; loss partials;
//                  loss [L]
// The read reuses the step's scratch: K' holds the pre-normalisation queries and then the memory
// tokens h, K the queries, dY0 the hidden activations A (row-major, zero padding) and dA0^T's
// space the transposed W_out copy.
//                  paper optimiser (fp32): rates [L][Tp], decay block sums
//                  [L][Tp/kRateTokens], decay [L],
//                  initial row norms
// The preprocessing buffers (K', K, K^T, dY0, dY^T, rates, decay) have G copies, so that
// mone_swiglu_segments runs RATE, PROJ and KEYS once for G consecutive segments.
// A segment step, each stage one launch grouped over all layers (PROJ) or all B heads:
//   [RATE]  per-token rates and momentum decay (paper optimiser)
//   PROJ    [raw K | raw V] = X [P_k ; P_v]^T   epilogue: keys: affine, SiLU -> K';
//                                               values: SiLU -> dY0, dY^T
//   KEYS    K': per-token L2 norm per head, RoPE -> K, K^T
//   DA      dA0^T = W_out dY0^T
//   FWD     [Z | G]^T = W_ig K^T     epilogue: A^T, [dZ | dG]^T, loss partials
//   UPD     A^T dY and [dZ | dG]^T K  (2 problems)  epilogue: update of the masters + copies
//           (paper optimiser: momentum, and each row rescaled to its initial norm in the same
//           epilogue, 64 x 256 tiles holding whole rows)
#include <hip/hip_runtime.h>

#include <cmath>
#include <new>

#include "../../include/mone_swiglu.h"
#include "host_common.hpp"
#include "swiglu_kernels.hpp"

using namespace mone;

namespace {

struct SwLayout {
  int Tp, dhp, parts_max;
  // G copies of the weight-independent preprocessing outputs (K, K^T, dY0, dY^T, the rates and
  // the decay), so that mone_swiglu_segments can compute them for G segments in one batch;
  // their element strides between copies.  With G > 1 there are two sets of G copies: one
  // batch's preprocessing fills one set while the segments of the batch before it read the
  // other (the raw keys and the rates' partial sums, used only inside the preprocessing, keep
  // one set).
  int G, sets;
  long long kh_ss, kt_ss, dy_ss, dyt_ss, rate_ss, vpart_ss, beta_ss;
  size_t kpre, kh, kt, dy, dyt, dat, at, dzgt, wig, woc, rope, gate, loss_part, loss_out;
  size_t rate, vpart, beta, n_ig, n_out;  // paper optimiser
  size_t total;
};

constexpr int kMaxPrepSegments = 16;

// Segments per preprocessing batch: cfg->prep_segments, or by default 8 when segments are a
// multiple of 64 tokens (1 otherwise: the batch maps GEMM rows to segments in 64-row steps).
int prep_segments(const mone_swiglu_config* c) {
  if (c->prep_segments > 0) return c->prep_segments;
  return c->seg_len % 64 == 0 ? 8 : 1;
}

int check_sw_config(const mone_swiglu_config* c) {
  if (!c) return fail(MONE_EINVAL, "config is NULL");
  if (c->n_layers < 1 || c->d_model < 1 || c->n_heads < 1 || c->d_head < 1 || c->seg_len < 1)
    return fail(MONE_EINVAL, "config sizes must be >= 1 (L=%d d=%d H=%d d_h=%d T=%d)",
                c->n_layers, c->d_model, c->n_heads, c->d_head, c->seg_len);
  if ((long long)c->n_heads * c->d_head != c->d_model)
    return fail(MONE_EINVAL, "d_model %d is not n_heads %d x d_head %d", c->d_model, c->n_heads,
                c->d_head);
  if (c->d_head % 2) return fail(MONE_EINVAL, "d_head %d is odd (RoPE pairs channels)", c->d_head);
  if (c->act_dtype != MONE_F32 && c->act_dtype != MONE_BF16)
    return fail(MONE_EINVAL, "act_dtype %d is not MONE_F32 or MONE_BF16", c->act_dtype);
  if (c->optimizer != MONE_OPT_SGD && c->optimizer != MONE_OPT_PAPER)
    return fail(MONE_EINVAL, "optimizer %d is not a mone_optimizer", c->optimizer);
  if (!std::isfinite(c->lr)) return fail(MONE_EINVAL, "lr is not finite");
  if (!std::isfinite(c->rope_base) || !(c->rope_base > 0.0f))
    return fail(MONE_EINVAL, "rope_base must be finite and positive");
  if (c->d_model % 64) return fail(MONE_EUNSUPPORTED, "d_model must be a multiple of 64");
  if (c->d_head % 16 || c->d_head > 256)
    return fail(MONE_EUNSUPPORTED, "d_head must be a multiple of 16 in [16, 256]");
  if (c->seg_len > 65536) return fail(MONE_EUNSUPPORTED, "seg_len above 65536");
  if (c->prep_segments < 0 || c->prep_segments > kMaxPrepSegments)
    return fail(MONE_EINVAL, "prep_segments %d outside [0, %d]", c->prep_segments,
                kMaxPrepSegments);
  if (c->prep_segments > 1 && c->seg_len % 64)
    return fail(MONE_EUNSUPPORTED, "prep_segments > 1 needs seg_len a multiple of 64");
  const long long Tp = round_up(c->seg_len, 256), d = c->d_model;
  const long long E = c->act_dtype == MONE_BF16 ? 2 : 4;
  // per-layer and per-head operand slices are addressed with 32-bit byte offsets
  if (Tp * d * E * prep_segments(c) >= (1LL << 31) || 2 * d * d * E >= (1LL << 31))
    return fail(MONE_EUNSUPPORTED, "a per-layer matrix exceeds 2^31 bytes");
  return MONE_OK;
}

SwLayout make_sw_layout(const mone_swiglu_config* c) {
  SwLayout L{};
  const size_t E = c->act_dtype == MONE_BF16 ? 2 : 4;
  const size_t nl = (size_t)c->n_layers, d = c->d_model, dh = c->d_head;
  const size_t B = nl * (size_t)c->n_heads;
  L.Tp = (int)round_up(c->seg_len, 256);
  L.dhp = (int)round_up(c->d_head, 64);
  // 4 wave partials per FWD tile; no tile shape is smaller than 64 in either direction
  L.parts_max = 4 * ((2 * c->d_head + 63) / 64) * (L.Tp / 64);
  const size_t Tp = L.Tp, dhp = L.dhp;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off = align_up(off + bytes, kAlign);
    return o;
  };
  const size_t G = (size_t)prep_segments(c);
  const size_t NS = G > 1 ? 2 : 1;
  L.G = (int)G;
  L.sets = (int)NS;
  L.kh_ss = L.dy_ss = (long long)(B * Tp * dhp);
  L.kt_ss = L.dyt_ss = (long long)(B * dh * Tp);
  L.rate_ss = (long long)(nl * Tp);
  L.vpart_ss = (long long)(nl * (Tp / kRateTokens));
  L.beta_ss = (long long)nl;
  L.kpre = take(nl * G * Tp * d * E);
  L.kh = take(NS * G * B * Tp * dhp * E);
  L.kt = take(NS * G * B * dh * Tp * E);
  L.dy = take(NS * G * B * Tp * dhp * E);
  L.dyt = take(NS * G * B * dh * Tp * E);
  L.dat = take(B * dh * Tp * E);
  L.at = take(B * dh * Tp * E);
  L.dzgt = take(B * 2 * dh * Tp * E);
  L.wig = take(B * 2 * dh * dhp * E);
  L.woc = take(B * dh * dhp * E);
  L.rope = take(Tp * (dh / 2) * 8);
  L.gate = take(nl * Tp * (size_t)c->n_heads * 4);
  L.loss_part = take(B * (size_t)L.parts_max * 4);
  L.loss_out = take(nl * 4);
  if (c->optimizer == MONE_OPT_PAPER) {
    L.rate = take(NS * G * nl * Tp * 4);
    L.vpart = take(G * nl * (Tp / kRateTokens) * 4);
    L.beta = take(NS * G * nl * 4);
    L.n_ig = take(B * 2 * dh * 4);
    L.n_out = take(B * dh * 4);
  }
  L.total = off;
  return L;
}

// Tile shape of the per-head GEMMs: their K extent (d_hp or a segment's tokens) is short, and
// 128 x 128 tiles give several workgroups per CU even for a few layers.
constexpr TileShape kHeadTile = TILE_128x128;

template <typename E, class Epi>
hipError_t launch_head_gemm(const Spec* specs, int nspec, int heads, const Epi& epi,
                            hipStream_t s) {
  return launch_tiled<E, 128, 128, 2>(specs, nspec, heads, epi, s, nullptr);
}

}  // namespace

struct mone_swiglu {
  mone_swiglu_config cfg;
  SwLayout lay;
  mone_swiglu_frozen fz;
  mone_swiglu_weights w;
  mone_swiglu_optimizer opt;  // MONE_OPT_PAPER only
  unsigned char* ws;
  int last_n;      // tokens of the last non-empty segment (0: none yet)
  int last_parts;  // loss partials per head written by that segment
  StageTimer timer;
  // With two sets of preprocessing copies: the internal stream that runs the preprocessing of
  // a multi-segment call beside its memory steps (default priority), and its events
  hipStream_t side;
  hipEvent_t ev_fork, ev_join, ev_prep[2], ev_chain[2];

  template <typename T>
  T* at(size_t off) const { return reinterpret_cast<T*>(ws + off); }
};

namespace {

// Weight-independent preprocessing of g consecutive segments of n tokens each (g > 1: whole
// segments of seg_len tokens, seg_len a multiple of 64), into copies c0 .. c0+g-1: RATE (paper
// optimiser), PROJ and KEYS, each one launch over all g segments.  x [L][g*n][d], layer
// stride lsx.
template <typename E, bool PAPER>
int run_sw_prep(mone_swiglu* H, const void* x, long long lsx, int n, int g, int c0,
                hipStream_t s) {
  const mone_swiglu_config& c = H->cfg;
  const SwLayout& Ly = H->lay;
  const int L = c.n_layers, d = c.d_model, NH = c.n_heads, dh = c.d_head;
  const int Tp = Ly.Tp, dhp = Ly.dhp;
  // rows of a segment in the batched launches; one segment keeps its padded extent
  const int seg_rows = g > 1 ? n : Tp, kpre_rows = Ly.G * Tp;
  const int nz = g > 1 ? g * n : (int)round_up(n, 64);  // token rows KEYS writes
  float* rate = PAPER ? H->at<float>(Ly.rate) + c0 * Ly.rate_ss : nullptr;
  hipError_t e;

  if constexpr (PAPER) {
    H->timer.begin(MONE_SW_STAGE_RATE, s);
    rate_kernel<E><<<dim3(Tp / kRateTokens, L, g), dim3(256), 0, s>>>(
        reinterpret_cast<const E*>(x), lsx, d, n, H->opt.rate_w, H->opt.rate_b, H->opt.decay_w,
        c.lr, rate, Tp, H->at<float>(Ly.vpart), (long long)n * d, Ly.rate_ss, Ly.vpart_ss);
    decay_kernel<<<dim3((L + 63) / 64, g), dim3(64), 0, s>>>(H->at<float>(Ly.vpart),
                                                             Tp / kRateTokens, n,
                                                             H->opt.decay_b,
                                                             H->at<float>(Ly.beta) + c0 * Ly.beta_ss,
                                                             L);
    if ((e = hipGetLastError()) != hipSuccess) return hip_fail(e, "launch RATE");
    H->timer.end(MONE_SW_STAGE_RATE, s);
  }
  // PROJ: [raw K | raw V] = X [P_k ; P_v]^T; epilogue: K', dY0, dY^T
  {
    Spec sp{};
    sp.part[0].a = opnd(x, lsx, d, g * n);
    sp.part[0].b = opnd(H->fz.proj, 2LL * d * d, d, 2 * d);
    sp.part[0].k_len = d;
    sp.nparts = 1;
    sp.m_extent = g * n;
    sp.n = 2 * d;
    sp.m_store = g > 1 ? g * n : -1;
    sp.n_store = 2 * d;
    EpiSwProj<E> epi;
    epi.kpre = H->at<E>(Ly.kpre);
    epi.dy = H->at<E>(Ly.dy) + c0 * Ly.dy_ss;
    epi.dyt = H->at<E>(Ly.dyt) + c0 * Ly.dyt_ss;
    epi.kscale = H->fz.k_scale; epi.kshift = H->fz.k_shift; epi.rate = rate;
    epi.lr = c.lr; epi.inv_n = 1.0f / (float)n;
    epi.d = d; epi.dh = dh; epi.dhp = dhp; epi.H = NH; epi.Tp = Tp; epi.n = n;
    epi.seg_rows = seg_rows; epi.kpre_rows = kpre_rows;
    epi.dy_ss = Ly.dy_ss; epi.dyt_ss = Ly.dyt_ss; epi.rate_ss = Ly.rate_ss;
    H->timer.begin(MONE_SW_STAGE_PROJ, s);
    // 128 x 128 tiles (measured faster here than 256 x 256, which leave most CUs idle in
    // their second round); 64-row tiles for short segments
    const TileShape tp = g * n <= 64 ? TILE_64x256 : TILE_128x128;
    if ((e = launch_gemm<E>(tp, &sp, 1, L, epi, s)) != hipSuccess)
      return hip_fail(e, "launch PROJ");
    H->timer.end(MONE_SW_STAGE_PROJ, s);
  }
  // KEYS: per-token L2 norm per head and RoPE -> K, K^T
  {
    H->timer.begin(MONE_SW_STAGE_KEYS, s);
    sw_keys_kernel<E><<<dim3(nz / 64, NH, L), dim3(256), 0, s>>>(
        H->at<E>(Ly.kpre), d, NH, dh, dhp, Tp, H->at<float2>(Ly.rope),
        H->at<E>(Ly.kh) + c0 * Ly.kh_ss, H->at<E>(Ly.kt) + c0 * Ly.kt_ss, seg_rows, kpre_rows,
        Ly.kh_ss, Ly.kt_ss);
    if ((e = hipGetLastError()) != hipSuccess) return hip_fail(e, "launch KEYS");
    H->timer.end(MONE_SW_STAGE_KEYS, s);
  }
  return MONE_OK;
}

// The weight-dependent part of the step of one segment of n tokens whose preprocessing is in
// copy `cp`: DA, FWD and UPD.
template <typename E, bool PAPER>
int run_sw_update(mone_swiglu* H, int n, int cp, hipStream_t s) {
  const mone_swiglu_config& c = H->cfg;
  const SwLayout& Ly = H->lay;
  const int L = c.n_layers, NH = c.n_heads, dh = c.d_head, B = L * NH;
  const int Tp = Ly.Tp, dhp = Ly.dhp;
  constexpr int BK = 8 * (16 / (int)sizeof(E));
  const int kt = (int)round_up(n, BK);   // token extent of the UPD contractions
  E* kh = H->at<E>(Ly.kh) + cp * Ly.kh_ss;
  E* ktr = H->at<E>(Ly.kt) + cp * Ly.kt_ss;
  E* dy = H->at<E>(Ly.dy) + cp * Ly.dy_ss;
  E* dyt = H->at<E>(Ly.dyt) + cp * Ly.dyt_ss;
  E* dat = H->at<E>(Ly.dat);
  E* At = H->at<E>(Ly.at);
  E* dzgt = H->at<E>(Ly.dzgt);
  E* wig = H->at<E>(Ly.wig);
  E* woc = H->at<E>(Ly.woc);
  float* rate = PAPER ? H->at<float>(Ly.rate) + cp * Ly.rate_ss : nullptr;
  float* beta = PAPER ? H->at<float>(Ly.beta) + cp * Ly.beta_ss : nullptr;
  const long long lhT = (long long)dh * Tp, lhP = (long long)Tp * dhp;
  hipError_t e;
  // DA: dA0^T = W_out dY0^T (A operand W_out [d_h][d_hp], B operand dY0 [tokens][d_hp])
  {
    Spec sp{};
    sp.part[0].a = opnd(woc, (long long)dh * dhp, dhp, dh);
    sp.part[0].b = opnd(dy, lhP, dhp, n);
    sp.part[0].k_len = dhp;
    sp.nparts = 1;
    sp.m_extent = dh;
    sp.n = n;
    sp.m_store = dh;
    sp.n_store = -1;
    EpiSwDa<E> epi;
    epi.dat = dat; epi.ls = lhT; epi.Tp = Tp;
    H->timer.begin(MONE_SW_STAGE_DA, s);
    if ((e = launch_head_gemm<E>(&sp, 1, B, epi, s)) != hipSuccess)
      return hip_fail(e, "launch DA");
    H->timer.end(MONE_SW_STAGE_DA, s);
  }
  // FWD: [Z | G]^T = W_ig K^T (A operand W_ig [2 d_h][d_hp], B operand K [tokens][d_hp])
  {
    Spec sp{};
    sp.part[0].a = opnd(wig, 2LL * dh * dhp, dhp, 2 * dh);
    sp.part[0].b = opnd(kh, lhP, dhp, n);
    sp.part[0].k_len = dhp;
    sp.nparts = 1;
    sp.m_extent = 2 * dh;
    sp.n = n;
    sp.m_store = 2 * dh;
    sp.n_store = -1;
    EpiSwFwd<E> epi;
    epi.dat = dat; epi.rate = rate; epi.at = At; epi.dzgt = dzgt;
    epi.loss_part = H->at<float>(Ly.loss_part); epi.ls = lhT; epi.Tp = Tp; epi.n = n; epi.H = NH;
    epi.parts = 4 * tiles_for(kHeadTile, 2 * dh, n);
    epi.lr = c.lr;
    H->timer.begin(MONE_SW_STAGE_FWD, s);
    if ((e = launch_head_gemm<E>(&sp, 1, B, epi, s)) != hipSuccess)
      return hip_fail(e, "launch FWD");
    H->timer.end(MONE_SW_STAGE_FWD, s);
    H->last_parts = epi.parts;
  }
  // UPD: problem 0 = A^T dY (W_out's gradient), problem 1 = [dZ | dG]^T K (W_in's and W_gate's)
  {
    Spec sp[2] = {};
    sp[0].part[0].a = opnd(At, lhT, Tp, dh);
    sp[0].part[0].b = opnd(dyt, lhT, Tp, dh);
    sp[0].part[0].k_len = kt;
    sp[0].nparts = 1;
    sp[0].m_extent = dh;
    sp[0].n = dh;
    sp[0].m_store = dh;
    sp[0].n_store = dh;
    sp[1].part[0].a = opnd(dzgt, 2 * lhT, Tp, 2 * dh);
    sp[1].part[0].b = opnd(ktr, lhT, Tp, dh);
    sp[1].part[0].k_len = kt;
    sp[1].nparts = 1;
    sp[1].m_extent = 2 * dh;
    sp[1].n = dh;
    sp[1].m_store = 2 * dh;
    sp[1].n_store = dh;
    EpiSwUpd<E, PAPER> epi;
    epi.w_in = H->w.w_in; epi.w_gate = H->w.w_gate; epi.w_out = H->w.w_out;
    epi.m_in = PAPER ? H->opt.mom_in : nullptr;
    epi.m_gate = PAPER ? H->opt.mom_gate : nullptr;
    epi.m_out = PAPER ? H->opt.mom_out : nullptr;
    epi.wig = wig; epi.woc = woc;
    epi.beta = beta;
    epi.n_ig = PAPER ? H->at<float>(Ly.n_ig) : nullptr;
    epi.n_out = PAPER ? H->at<float>(Ly.n_out) : nullptr;
    epi.lsw = (long long)dh * dh; epi.dh = dh; epi.dhp = dhp; epi.H = NH;
    H->timer.begin(MONE_SW_STAGE_UPD, s);
    // the paper's optimiser renormalises whole rows in the epilogue: 64 x 256 tiles, one
    // workgroup per 64 rows of a head's matrix (d_h <= 256 columns)
    if constexpr (PAPER)
      e = launch_tiled<E, 64, 256, 1>(sp, 2, B, epi, s, nullptr);
    else
      e = launch_head_gemm<E>(sp, 2, B, epi, s);
    if (e != hipSuccess) return hip_fail(e, "launch UPD");
    H->timer.end(MONE_SW_STAGE_UPD, s);
  }
  H->last_n = n;
  return MONE_OK;
}

// One segment of n tokens: its preprocessing into copy 0, then its update.  x [L][n][d], layer
// stride lsx.
template <typename E, bool PAPER>
int run_sw_segment(mone_swiglu* H, const void* x, long long lsx, int n, hipStream_t s) {
  const int rc = run_sw_prep<E, PAPER>(H, x, lsx, n, 1, 0, s);
  return rc != MONE_OK ? rc : run_sw_update<E, PAPER>(H, n, 0, s);
}

// S whole segments from x [L][S*T][d] (layer stride lsx): preprocessing in batches of up to G
// segments, then each segment's update in order.  With two or more batches the preprocessing
// runs on the handle's internal stream, one batch ahead, into alternating sets of copies: batch
// k+1's preprocessing (which reads only x and the frozen parameters) overlaps batch k's memory
// steps on `s`.  Batch k's steps wait for its preprocessing; batch k+2's preprocessing waits for
// batch k's steps (the last readers of that set); the internal stream starts after the work
// queued on `s` before the call and `s` waits for it at the end, so the call keeps the ordering
// of a single stream (and can be captured in a graph).
template <typename E, bool PAPER>
int run_sw_segments(mone_swiglu* H, const void* x, long long lsx, int S, hipStream_t s) {
  const int T = H->cfg.seg_len, G = H->lay.G;
  const long long d = H->cfg.d_model;
  const int nb = (S + G - 1) / G;
  auto xs = [&](int b) { return reinterpret_cast<const E*>(x) + (long long)b * G * T * d; };
  auto gsz = [&](int b) { return S - b * G < G ? S - b * G : G; };
  auto steps = [&](int b, int c0) {
    int rc = MONE_OK;
    for (int cp = 0; cp < gsz(b) && rc == MONE_OK; ++cp)
      rc = run_sw_update<E, PAPER>(H, T, c0 + cp, s);
    return rc;
  };
  if (nb < 2 || H->lay.sets < 2) {
    for (int b = 0; b < nb; ++b) {
      int rc = run_sw_prep<E, PAPER>(H, xs(b), lsx, T, gsz(b), 0, s);
      if (rc == MONE_OK) rc = steps(b, 0);
      if (rc != MONE_OK) return rc;
    }
    return MONE_OK;
  }
  hipStream_t q = H->side;
  hipError_t e = hipEventRecord(H->ev_fork, s);
  if (e == hipSuccess) e = hipStreamWaitEvent(q, H->ev_fork, 0);
  if (e != hipSuccess) return hip_fail(e, "fork the preprocessing stream");
  auto prep = [&](int b) {
    int rc = run_sw_prep<E, PAPER>(H, xs(b), lsx, T, gsz(b), (b & 1) * G, q);
    if (rc != MONE_OK) return rc;
    const hipError_t er = hipEventRecord(H->ev_prep[b & 1], q);
    return er == hipSuccess ? MONE_OK : hip_fail(er, "record the preprocessing event");
  };
  int rc = prep(0);
  for (int b = 0; b < nb && rc == MONE_OK; ++b) {
    if (b + 1 < nb) {
      // set (b+1)&1 was last read by batch b-1's steps
      if (b >= 1 && (e = hipStreamWaitEvent(q, H->ev_chain[(b + 1) & 1], 0)) != hipSuccess) {
        rc = hip_fail(e, "wait for the steps");
        break;
      }
      if ((rc = prep(b + 1)) != MONE_OK) break;
    }
    if ((e = hipStreamWaitEvent(s, H->ev_prep[b & 1], 0)) != hipSuccess) {
      rc = hip_fail(e, "wait for the preprocessing");
      break;
    }
    if ((rc = steps(b, (b & 1) * G)) != MONE_OK) break;
    if ((e = hipEventRecord(H->ev_chain[b & 1], s)) != hipSuccess)
      rc = hip_fail(e, "record the steps event");
  }
  // join, also after an error, so that no work of the call is left outside `s`
  e = hipEventRecord(H->ev_join, q);
  if (e == hipSuccess) e = hipStreamWaitEvent(s, H->ev_join, 0);
  if (rc == MONE_OK && e != hipSuccess) rc = hip_fail(e, "join the preprocessing stream");
  return rc;
}

template <typename E>
int run_sw_read(mone_swiglu* H, const mone_swiglu_reader* rd, const void* xq, int q, void* kv,
                int kv_bf16, hipStream_t s) {
  const mone_swiglu_config& c = H->cfg;
  const SwLayout& Ly = H->lay;
  const int L = c.n_layers, d = c.d_model, NH = c.n_heads, dh = c.d_head, B = L * NH;
  const int Tp = Ly.Tp, dhp = Ly.dhp, D = 2 * rd->d_kv;
  const int qz = (int)round_up(q, 64);
  E* qpre = H->at<E>(Ly.kpre);  // the queries before normalisation, then the memory tokens h
  E* kq = H->at<E>(Ly.kh);
  E* abuf = H->at<E>(Ly.dy);    // A [B][Tp][d_hp]; its padding columns are always zero
  E* wot = H->at<E>(Ly.dat);    // W_out^T [B][d_h][d_hp]
  float* gate = H->at<float>(Ly.gate);
  const TileShape tq = q <= 64 ? TILE_64x256 : TILE_128x128;
  hipError_t e;
  // QPROJ: Q' = SiLU(s_q (X_q P_q^T) + b_q); the gates
  {
    Spec sp{};
    sp.part[0].a = opnd(xq, (long long)q * d, d, q);
    sp.part[0].b = opnd(rd->proj_q, (long long)d * d, d, d);
    sp.part[0].k_len = d;
    sp.nparts = 1;
    sp.m_extent = q;
    sp.n = d;
    sp.m_store = -1;
    sp.n_store = d;
    EpiSwQproj<E> epi;
    epi.qpre = qpre; epi.scale = rd->q_scale; epi.shift = rd->q_shift;
    epi.d = d; epi.Tp = Tp; epi.q = q;
    H->timer.begin(MONE_SW_STAGE_QPROJ, s);
    if ((e = launch_gemm<E>(tq, &sp, 1, L, epi, s)) != hipSuccess)
      return hip_fail(e, "launch QPROJ");
    sw_gate_kernel<E><<<dim3((q + 3) / 4, L), dim3(256), 0, s>>>(
        reinterpret_cast<const E*>(xq), q, d, NH, rd->gate_w, rd->gate_b, Tp, gate);
    if ((e = hipGetLastError()) != hipSuccess) return hip_fail(e, "launch gates");
    H->timer.end(MONE_SW_STAGE_QPROJ, s);
  }
  // QKEYS: per-head L2 norm and RoPE at positions 0 .. q-1
  H->timer.begin(MONE_SW_STAGE_QKEYS, s);
  sw_keys_kernel<E><<<dim3(qz / 64, NH, L), dim3(256), 0, s>>>(
      qpre, d, NH, dh, dhp, Tp, H->at<float2>(Ly.rope), kq, H->at<E>(Ly.kt), Tp, Tp, 0LL, 0LL);
  if ((e = hipGetLastError()) != hipSuccess) return hip_fail(e, "launch QKEYS");
  H->timer.end(MONE_SW_STAGE_QKEYS, s);
  // QFWD: A = SiLU(Z) * G with [Z | G] = K_q W_ig^T; and the W_out^T copy for QOUT
  {
    transpose_kernel<float, E><<<dim3((dh + 63) / 64, (dhp + 63) / 64, B), dim3(256), 0, s>>>(
        H->w.w_out, (long long)dh * dh, dh, dh, dh, wot, (long long)dh * dhp, dhp, dhp);
    if ((e = hipGetLastError()) != hipSuccess) return hip_fail(e, "launch W_out^T");
    Spec sp{};
    sp.part[0].a = opnd(kq, (long long)Tp * dhp, dhp, q);
    sp.part[0].b = opnd(H->at<E>(Ly.wig), 2LL * dh * dhp, dhp, 2 * dh);
    sp.part[0].k_len = dhp;
    sp.nparts = 1;
    sp.m_extent = q;
    sp.n = 2 * dh;
    sp.m_store = -1;
    sp.n_store = 2 * dh;
    EpiSwQfwd<E> epi;
    epi.a = abuf; epi.ls = (long long)Tp * dhp; epi.dhp = dhp;
    H->timer.begin(MONE_SW_STAGE_QFWD, s);
    if ((e = launch_gemm<E>(tq, &sp, 1, B, epi, s)) != hipSuccess)
      return hip_fail(e, "launch QFWD");
    H->timer.end(MONE_SW_STAGE_QFWD, s);
  }
  // QOUT: O = A W_out per head (64 x 256 tiles: whole rows), RMSNorm and gate -> h
  {
    Spec sp{};
    sp.part[0].a = opnd(abuf, (long long)Tp * dhp, dhp, q);
    sp.part[0].b = opnd(wot, (long long)dh * dhp, dhp, dh);
    sp.part[0].k_len = dhp;
    sp.nparts = 1;
    sp.m_extent = q;
    sp.n = dh;
    sp.m_store = q;
    sp.n_store = dh;
    EpiSwQout<E> epi;
    epi.hout = qpre; epi.rms_w = rd->rms_w; epi.gate = gate;
    epi.d = d; epi.dh = dh; epi.H = NH; epi.Tp = Tp;
    H->timer.begin(MONE_SW_STAGE_QOUT, s);
    if ((e = launch_tiled<E, 64, 256, 1>(&sp, 1, B, epi, s, nullptr)) != hipSuccess)
      return hip_fail(e, "launch QOUT");
    H->timer.end(MONE_SW_STAGE_QOUT, s);
  }
  // QKV: [h W_k^T | h W_v^T] into the caller's buffer
  {
    Spec sp{};
    sp.part[0].a = opnd(qpre, (long long)Tp * d, d, q);
    sp.part[0].b = opnd(rd->w_kv, (long long)D * d, d, D);
    sp.part[0].k_len = d;
    sp.nparts = 1;
    sp.m_extent = q;
    sp.n = D;
    sp.m_store = q;
    sp.n_store = D;
    EpiSwKv epi;
    epi.kv = kv; epi.ls = (long long)q * D; epi.D = D; epi.bf16_out = kv_bf16;
    H->timer.begin(MONE_SW_STAGE_QKV, s);
    if ((e = launch_gemm<E>(tq, &sp, 1, L, epi, s)) != hipSuccess)
      return hip_fail(e, "launch QKV");
    H->timer.end(MONE_SW_STAGE_QKV, s);
  }
  return MONE_OK;
}

// The internal stream and events (those created so far); the stream is drained first.
void release_side(mone_swiglu* H) {
  if (H->side) {
    (void)hipStreamSynchronize(H->side);
    (void)hipStreamDestroy(H->side);
    H->side = nullptr;
  }
  hipEvent_t* evs[6] = {&H->ev_fork, &H->ev_join, &H->ev_prep[0], &H->ev_prep[1],
                        &H->ev_chain[0], &H->ev_chain[1]};
  for (hipEvent_t* ev : evs)
    if (*ev) {
      (void)hipEventDestroy(*ev);
      *ev = nullptr;
    }
}

template <typename E>
hipError_t build_copies(mone_swiglu* H, hipStream_t s) {
  const mone_swiglu_config& c = H->cfg;
  const SwLayout& Ly = H->lay;
  const int dh = c.d_head, B = c.n_layers * c.n_heads;
  const long long per = 3LL * dh * Ly.dhp;
  sw_pack_kernel<E><<<dim3((unsigned)((per + 255) / 256), B), dim3(256), 0, s>>>(
      H->w.w_in, H->w.w_gate, H->w.w_out, dh, Ly.dhp, H->at<E>(Ly.wig), H->at<E>(Ly.woc));
  return hipGetLastError();
}

}  // namespace

extern "C" {

size_t mone_swiglu_workspace_bytes(const mone_swiglu_config* cfg) {
  g_err[0] = 0;
  if (check_sw_config(cfg) != MONE_OK) return 0;
  return make_sw_layout(cfg).total;
}

int mone_swiglu_init(mone_swiglu** out, const mone_swiglu_config* cfg,
                     const mone_swiglu_frozen* frozen, const mone_swiglu_weights* weights,
                     const mone_swiglu_optimizer* opt, void* workspace, size_t workspace_bytes,
                     void* stream) {
  g_err[0] = 0;
  if (!out) return fail(MONE_EINVAL, "out is NULL");
  *out = nullptr;
  int rc = check_sw_config(cfg);
  if (rc != MONE_OK) return rc;
  if (!frozen || !weights) return fail(MONE_EINVAL, "frozen and weights must be non-NULL");
  if (!frozen->proj || !frozen->k_scale || !frozen->k_shift || !weights->w_in ||
      !weights->w_gate || !weights->w_out || !workspace)
    return fail(MONE_EINVAL, "every frozen and weight pointer and the workspace must be non-NULL");
  if (!aligned16(frozen->proj) || !aligned16(frozen->k_scale) || !aligned16(frozen->k_shift) ||
      !aligned16(weights->w_in) || !aligned16(weights->w_gate) || !aligned16(weights->w_out))
    return fail(MONE_EINVAL, "frozen and weight pointers must be 16-byte aligned");
  const bool paper = cfg->optimizer == MONE_OPT_PAPER;
  if (paper != (opt != nullptr))
    return fail(MONE_EINVAL, paper ? "MONE_OPT_PAPER needs the optimiser state (opt)"
                                   : "opt must be NULL for MONE_OPT_SGD");
  if (paper) {
    if (!opt->rate_w || !opt->rate_b || !opt->decay_w || !opt->decay_b || !opt->mom_in ||
        !opt->mom_gate || !opt->mom_out)
      return fail(MONE_EINVAL, "every pointer of the optimiser state must be non-NULL");
    if (!aligned16(opt->rate_w) || !aligned16(opt->decay_w) || !aligned16(opt->mom_in) ||
        !aligned16(opt->mom_gate) || !aligned16(opt->mom_out))
      return fail(MONE_EINVAL, "rate_w, decay_w and the momenta must be 16-byte aligned");
  }
  if (((uintptr_t)workspace & (kAlign - 1)) != 0)
    return fail(MONE_EINVAL, "workspace must be 256-byte aligned");
  const SwLayout Ly = make_sw_layout(cfg);
  if (workspace_bytes < Ly.total)
    return fail(MONE_EINVAL, "workspace has %zu bytes, %zu needed", workspace_bytes, Ly.total);

  mone_swiglu* H = new (std::nothrow) mone_swiglu();
  if (!H) return fail(MONE_EINVAL, "host allocation failed");
  H->cfg = *cfg;
  H->lay = Ly;
  H->fz = *frozen;
  H->w = *weights;
  if (opt) H->opt = *opt;
  H->ws = reinterpret_cast<unsigned char*>(workspace);
  H->last_n = 0;
  H->last_parts = 0;

  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  hipError_t e = hipMemsetAsync(workspace, 0, Ly.total, s);
  if (e == hipSuccess)
    e = cfg->act_dtype == MONE_BF16 ? build_copies<bf16_t>(H, s) : build_copies<float>(H, s);
  if (e == hipSuccess) {
    const long long nt = (long long)Ly.Tp * (cfg->d_head / 2);
    sw_rope_table_kernel<<<dim3((unsigned)((nt + 255) / 256)), dim3(256), 0, s>>>(
        H->at<float2>(Ly.rope), Ly.Tp, cfg->d_head, (double)cfg->rope_base);
    e = hipGetLastError();
  }
  if (e == hipSuccess && paper) {
    const int B = cfg->n_layers * cfg->n_heads, dh = cfg->d_head;
    sw_row_norm_kernel<<<dim3((3 * dh + 3) / 4, B), dim3(256), 0, s>>>(
        weights->w_in, weights->w_gate, weights->w_out, dh, H->at<float>(Ly.n_ig),
        H->at<float>(Ly.n_out));
    e = hipGetLastError();
  }
  if (e != hipSuccess) {
    delete H;
    return hip_fail(e, "building the handle's copies");
  }
  if (Ly.sets > 1) {
    e = hipStreamCreateWithFlags(&H->side, hipStreamNonBlocking);
    hipEvent_t* evs[6] = {&H->ev_fork, &H->ev_join, &H->ev_prep[0], &H->ev_prep[1],
                          &H->ev_chain[0], &H->ev_chain[1]};
    for (int i = 0; i < 6 && e == hipSuccess; ++i)
      e = hipEventCreateWithFlags(evs[i], hipEventDisableTiming);
    if (e != hipSuccess) {
      release_side(H);
      delete H;
      return hip_fail(e, "creating the preprocessing stream and its events");
    }
  }
  *out = H;
  return MONE_OK;
}

int mone_swiglu_segment(mone_swiglu* H, const void* x, int32_t n_tokens, void* stream) {
  g_err[0] = 0;
  if (!H) return fail(MONE_EINVAL, "handle is NULL");
  if (n_tokens < 0 || n_tokens > H->cfg.seg_len)
    return fail(MONE_EINVAL, "n_tokens %d outside [0, seg_len=%d]", n_tokens, H->cfg.seg_len);
  if (n_tokens == 0) return MONE_OK;
  if (!x) return fail(MONE_EINVAL, "x is NULL");
  if (!aligned16(x)) return fail(MONE_EINVAL, "x must be 16-byte aligned");
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const bool paper = H->cfg.optimizer == MONE_OPT_PAPER;
  const long long lsx = (long long)n_tokens * H->cfg.d_model;
  if (H->cfg.act_dtype == MONE_BF16)
    return paper ? run_sw_segment<bf16_t, true>(H, x, lsx, n_tokens, s)
                 : run_sw_segment<bf16_t, false>(H, x, lsx, n_tokens, s);
  return paper ? run_sw_segment<float, true>(H, x, lsx, n_tokens, s)
               : run_sw_segment<float, false>(H, x, lsx, n_tokens, s);
}

int mone_swiglu_segments(mone_swiglu* H, const void* x, int64_t layer_stride,
                         int32_t n_segments, void* stream) {
  g_err[0] = 0;
  if (!H) return fail(MONE_EINVAL, "handle is NULL");
  if (n_segments < 0) return fail(MONE_EINVAL, "n_segments = %d is negative", n_segments);
  if (n_segments == 0) return MONE_OK;
  const mone_swiglu_config& c = H->cfg;
  const long long T = c.seg_len, d = c.d_model, E = c.act_dtype == MONE_BF16 ? 2 : 4;
  if (layer_stride < (long long)n_segments * T * d)
    return fail(MONE_EINVAL, "layer_stride %lld below n_segments * seg_len * d_model = %lld",
                (long long)layer_stride, (long long)n_segments * T * d);
  if (!x) return fail(MONE_EINVAL, "x is NULL");
  if (!aligned16(x) || (layer_stride * E) % 16 != 0)
    return fail(MONE_EINVAL, "x and layer_stride * element size must be 16-byte aligned");
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const bool paper = c.optimizer == MONE_OPT_PAPER;
  if (c.act_dtype == MONE_BF16)
    return paper ? run_sw_segments<bf16_t, true>(H, x, layer_stride, n_segments, s)
                 : run_sw_segments<bf16_t, false>(H, x, layer_stride, n_segments, s);
  return paper ? run_sw_segments<float, true>(H, x, layer_stride, n_segments, s)
               : run_sw_segments<float, false>(H, x, layer_stride, n_segments, s);
}

int mone_swiglu_loss(mone_swiglu* H, float* out_host, void* stream) {
  g_err[0] = 0;
  if (!H || !out_host) return fail(MONE_EINVAL, "handle and out_host must be non-NULL");
  if (H->last_n == 0) return fail(MONE_ESTATE, "no non-empty segment has been processed");
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const int L = H->cfg.n_layers, per = H->cfg.n_heads * H->last_parts;
  float* dev_out = H->at<float>(H->lay.loss_out);
  loss_finalize_kernel<<<dim3(L), dim3(256), 0, s>>>(H->at<float>(H->lay.loss_part), per, per,
                                                      1.0f, dev_out);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_fail(e, "launch loss");
  if ((e = hipMemcpyAsync(out_host, dev_out, sizeof(float) * L, hipMemcpyDeviceToHost, s)) !=
      hipSuccess)
    return hip_fail(e, "copy loss");
  if ((e = hipStreamSynchronize(s)) != hipSuccess) return hip_fail(e, "synchronise");
  return MONE_OK;
}

int mone_swiglu_read(mone_swiglu* H, const mone_swiglu_reader* rd, const void* xq, int32_t q,
                     void* kv, int32_t kv_dtype, void* stream) {
  g_err[0] = 0;
  if (!H) return fail(MONE_EINVAL, "handle is NULL");
  if (!rd) return fail(MONE_EINVAL, "reader is NULL");
  if (q < 0) return fail(MONE_EINVAL, "q = %d is negative", q);
  if (kv_dtype != MONE_F32 && kv_dtype != MONE_BF16)
    return fail(MONE_EINVAL, "kv_dtype %d is not MONE_F32 or MONE_BF16", kv_dtype);
  if (rd->d_kv < 1) return fail(MONE_EINVAL, "d_kv = %d must be >= 1", rd->d_kv);
  if (rd->d_kv % 64) return fail(MONE_EUNSUPPORTED, "d_kv must be a multiple of 64");
  if (2LL * rd->d_kv * H->cfg.d_model * (H->cfg.act_dtype == MONE_BF16 ? 2 : 4) >= (1LL << 31))
    return fail(MONE_EUNSUPPORTED, "a per-layer matrix exceeds 2^31 bytes");
  if (q > H->lay.Tp)
    return fail(MONE_EUNSUPPORTED, "q = %d above %d (seg_len rounded up to 256)", q, H->lay.Tp);
  if (!rd->proj_q || !rd->q_scale || !rd->q_shift || !rd->rms_w || !rd->gate_w || !rd->gate_b ||
      !rd->w_kv)
    return fail(MONE_EINVAL, "every pointer of the reader must be non-NULL");
  if (!aligned16(rd->proj_q) || !aligned16(rd->q_scale) || !aligned16(rd->q_shift) ||
      !aligned16(rd->rms_w) || !aligned16(rd->gate_w) || !aligned16(rd->w_kv))
    return fail(MONE_EINVAL, "proj_q, q_scale, q_shift, rms_w, gate_w and w_kv must be "
                "16-byte aligned");
  if (q == 0) return MONE_OK;
  if (!xq || !kv) return fail(MONE_EINVAL, "xq and kv must be non-NULL");
  if (!aligned16(xq) || !aligned16(kv)) return fail(MONE_EINVAL, "xq and kv must be 16-byte aligned");
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const int kvb = kv_dtype == MONE_BF16 ? 1 : 0;
  return H->cfg.act_dtype == MONE_BF16 ? run_sw_read<bf16_t>(H, rd, xq, q, kv, kvb, s)
                                       : run_sw_read<float>(H, rd, xq, q, kv, kvb, s);
}

int mone_swiglu_attention(mone_swiglu* H, int32_t d_kv, const void* qh, const void* kh,
                          const void* vh, const void* kv_mem, int32_t kv_dtype, int32_t q,
                          int32_t n_heads, int32_t n_kv_heads, void* out, int32_t out_dtype,
                          void* stream) {
  g_err[0] = 0;
  if (!H) return fail(MONE_EINVAL, "handle is NULL");
  if (d_kv < 1) return fail(MONE_EINVAL, "d_kv = %d must be >= 1", d_kv);
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const bool timed = q > 0;
  if (timed) H->timer.begin(MONE_SW_STAGE_ATTN, s);
  const int rc = launch_attention(H->cfg.n_layers, d_kv, H->cfg.act_dtype == MONE_BF16, qh, kh,
                                  vh, kv_mem, kv_dtype, q, n_heads, n_kv_heads, out, out_dtype, s);
  if (rc == MONE_OK && timed) H->timer.end(MONE_SW_STAGE_ATTN, s);
  return rc;
}

int mone_swiglu_destroy(mone_swiglu* H) {
  g_err[0] = 0;
  if (!H) return MONE_OK;
  H->timer.destroy();
  release_side(H);
  delete H;
  return MONE_OK;
}

int mone_swiglu_set_stage_timing(mone_swiglu* H, int32_t max_records, uint32_t stage_mask) {
  g_err[0] = 0;
  if (!H) return fail(MONE_EINVAL, "handle is NULL");
  return H->timer.enable(max_records, stage_mask);
}

int mone_swiglu_stage_times(mone_swiglu* H, double* ms_sum, int32_t* count) {
  g_err[0] = 0;
  if (!H || !ms_sum || !count) return fail(MONE_EINVAL, "NULL argument");
  return H->timer.report(ms_sum, count, MONE_SW_N_STAGES);
}

}  // extern "C"
