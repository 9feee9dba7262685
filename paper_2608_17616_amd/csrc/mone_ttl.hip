// Host side of the MoNe test-time-learning library: argument validation, workspace layout and
// the per-stage launches of a segment step and of the read.  The C ABI is declared in
// include/mone_ttl.h.
//
// Data layout in HBM (row-major; "[L]" = the L layers back to back):
//   caller state   W1 [L][h][d] fp32, W2 [L][D][h] fp32, W_kv [L][D][d] act
//   workspace      W1c [L][h][d] act   (bf16 mode only: MFMA copy of W1; fp32 mode reads W1)
//                  W2n [L][D][h] act   -W2 (forward 2 and the read: the residual Y - targets
//                                      becomes one K-concatenated sum, negated in the epilogue)
//                  W2t [2][L][h][D] act  W2 transposed (A operand of the backward GEMM), a
//                                      ping-pong pair: the backward of a step reads one copy
//                                      while the W2 update of the same launch writes the other
//                  A   [L][Tp][h], A^T [L][h][Tp], SiLU'(Z)^T [L][h][Tp]
//                  G   [L][Tp][D], G^T [L][D][Tp]
//                  dZ^T [L][h][Tp], X^T [L][d][Tp]
//                  loss partials [L][P], loss [L] fp32
//                  paper optimiser only (fp32): rates [L][Tp], decay block sums
//                  [L][Tp/kRateTokens] (one per 16-token block),
//                  decay [L], initial row norms [L][h] and [L][D], row-segment sums of
//                  squares [L][h][d/64] and [L][D][h/64], row scales [L][h] and [L][D]
// Tp = seg_len rounded up to 256; rows and columns beyond the segment's n tokens are zero, so
// the token-contracting GEMMs run over n rounded up to their K step with no masking.
//
// A segment step is five launches on the caller's stream, each grouped over all L layers:
//   XT   X -> X^T
//   FWD1 Z = X W1^T                      epilogue: A, A^T, SiLU'(Z)^T
//   FWD2 -R = [A | X] [-W2 | W_kv]^T     epilogue: G = c R, G^T, sum R^2 partials
//   BWD  dA^T = W2^T G^T  and  G^T A     epilogues: dZ^T = dA^T * SiLU'(Z)^T; fp32 SGD
//        (2 problems)                    read-modify-write of W2 + its copies
//   UPD  dZ^T X                          epilogue: fp32 SGD read-modify-write of W1 + copy
// With the paper's optimiser: RATE (per-token rates, momentum decay) after XT; FWD2 scales G by
// the rates; the BWD and UPD epilogues update momentum and masters and write row sums of
// squares; RENORM rescales the rows of W1 and W2 and writes their copies.
// The W2 update shares the backward's launch: it needs only G and A, and writes the W2^T copy
// the backward does not read, so CUs in its memory-bound epilogue overlap CUs computing the
// backward's MFMAs.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <new>
#include <vector>

#include "../../include/mone_ttl.h"
#include "host_common.hpp"

thread_local char g_err[512] = "";

using namespace mone;

namespace {

struct Layout {
  int Tp;
  int loss_per_layer;
  size_t w1c, w2c, w2t, a, at, dst, g, gt, dzt, xt, loss_part, loss_out, split;
  size_t rate, vpart, beta, norm1, norm2, ss1, ss2, scale1, scale2;  // paper optimiser
  // block form of consecutive segments (mone_ttl_segments): blk segments per block (0: none),
  // block rows padded to Btp; fp32 pre-update products and activation-dtype block operands
  int blk, Btp;
  size_t bz0, btgt, bgram, ba, bat, bsd, bg, bgt, bdzt, bxt, brr, bp, bda0, bq;
  size_t total;
};

// Block form of consecutive segments.  Short segments rewrite every fast weight for few
// tokens; a block of segments reads and writes them once, at the cost of the T x T token
// products of its segments' corrections (which grow with T and with the block).  It covers
// plain SGD on the squared-error losses with segments of a multiple of 64 tokens (whole K
// steps of the token products).  By default, for segments of at most 256 tokens when the fast
// weights of all layers hold at least 2^24 elements (below that, the weight traffic a block
// saves is small next to the latency of its extra launches): 8 segments per block, at most
// 1024 tokens (measured at 16 layers of 2048 -> 2048 -> 1024: T = 64 in 512-token blocks,
// T = 128 and 256 in 1024-token blocks; 512 segments of T = 512 ran faster one by one).
constexpr int kBlockMaxSeg = 256, kBlockSegs = 8, kBlockMaxDefault = 1024;
constexpr int kMaxBlockTokens = 4096;
constexpr long long kBlockMinWeights = 1LL << 24;

bool block_form_applies(const mone_ttl_config* c) {
  return c->optimizer == MONE_OPT_SGD &&
         (c->loss == MONE_LOSS_MSE_SUM || c->loss == MONE_LOSS_MSE_MEAN) && c->seg_len % 64 == 0;
}

// Tokens per block (0: no block form); the config has passed check_config.
int block_tokens(const mone_ttl_config* c) {
  if (c->block_tokens < 0 || !block_form_applies(c)) return 0;
  if (c->block_tokens > 0) return c->block_tokens;
  const long long w = (long long)c->n_layers * c->d_hidden * (c->d_model + 2LL * c->d_kv);
  if (c->seg_len > kBlockMaxSeg || w < kBlockMinWeights) return 0;
  const int segs = kBlockMaxDefault / c->seg_len < kBlockSegs ? kBlockMaxDefault / c->seg_len
                                                              : kBlockSegs;
  return segs * c->seg_len;  // at least 4 segments: seg_len <= 256
}

int check_config(const mone_ttl_config* c) {
  if (!c) return fail(MONE_EINVAL, "config is NULL");
  if (c->n_layers < 1 || c->d_model < 1 || c->d_hidden < 1 || c->d_kv < 1 || c->seg_len < 1)
    return fail(MONE_EINVAL, "config sizes must be >= 1 (L=%d d=%d h=%d d_kv=%d T=%d)",
                c->n_layers, c->d_model, c->d_hidden, c->d_kv, c->seg_len);
  if (c->act_dtype != MONE_F32 && c->act_dtype != MONE_BF16)
    return fail(MONE_EINVAL, "act_dtype %d is not MONE_F32 or MONE_BF16", c->act_dtype);
  if (c->loss != MONE_LOSS_MSE_SUM && c->loss != MONE_LOSS_MSE_MEAN && c->loss != MONE_LOSS_NIP)
    return fail(MONE_EINVAL, "loss %d is not a mone_loss", c->loss);
  if (!std::isfinite(c->lr)) return fail(MONE_EINVAL, "lr is not finite");
  if (c->optimizer != MONE_OPT_SGD && c->optimizer != MONE_OPT_PAPER)
    return fail(MONE_EINVAL, "optimizer %d is not a mone_optimizer", c->optimizer);
  if (c->d_model % 64 || c->d_hidden % 64 || c->d_kv % 64)
    return fail(MONE_EUNSUPPORTED, "d_model, d_hidden and d_kv must be multiples of 64");
  if (c->seg_len > 65536) return fail(MONE_EUNSUPPORTED, "seg_len above 65536");
  if (c->block_tokens > 0) {
    if (!block_form_applies(c))
      return fail(MONE_EUNSUPPORTED, "block_tokens needs plain SGD, a squared-error loss and "
                  "seg_len a multiple of 64");
    if (c->block_tokens % c->seg_len || c->block_tokens < 2 * c->seg_len ||
        c->block_tokens > kMaxBlockTokens)
      return fail(MONE_EINVAL, "block_tokens %d must be a multiple of seg_len %d from 2 * "
                  "seg_len to %d", c->block_tokens, c->seg_len, kMaxBlockTokens);
  }
  const long long Tp = round_up(c->seg_len, 256);
  const long long d = c->d_model, h = c->d_hidden, D = 2LL * c->d_kv;
  const long long mx = d > h ? (d > D ? d : D) : (h > D ? h : D);
  const long long E = c->act_dtype == MONE_BF16 ? 2 : 4;
  // per-layer operand slices are addressed with 32-bit byte offsets; fp32 masters are 4 bytes
  if (h * d * 4 >= (1LL << 31) || D * h * 4 >= (1LL << 31) || D * d * E >= (1LL << 31) ||
      Tp * mx * E >= (1LL << 31))
    return fail(MONE_EUNSUPPORTED, "a per-layer matrix exceeds 2^31 bytes");
  return MONE_OK;
}

// Tile of a weight-gradient launch (BWD, UPD), whose contraction runs over the k tokens of the
// segment.  Below 2048 tokens a 256 x 256 tile spends most of its time in the fp32
// read-modify-write epilogue with one workgroup per CU; 128 x 128 tiles keep two workgroups per
// CU, so one's epilogue overlaps the other's main loop (measured faster at k = 64 .. 1024, slower
// at k = 2048).
TileShape upd_tile(int m, int n_cols, int k, int layers) {
  if (k < 2048 && m > 64 && n_cols > 64) return TILE_128x128;
  return pick_tile(m, n_cols, layers);
}

Layout make_layout(const mone_ttl_config* c) {
  Layout L{};
  const size_t E = c->act_dtype == MONE_BF16 ? 2 : 4;
  const size_t nl = (size_t)c->n_layers;
  const size_t d = c->d_model, h = c->d_hidden, D = 2 * (size_t)c->d_kv;
  L.Tp = (int)round_up(c->seg_len, 256);
  const size_t Tp = L.Tp;
  // 4 wave partials per tile of the smallest tile shapes: forward 2's tiles over [Tp][D] and,
  // for the negative inner product, the W2 update's tiles over [D][h]
  const size_t lp_fwd2 = (Tp / 64) * ((D + 127) / 128), lp_w2 = ((D + 63) / 64) * ((h + 63) / 64);
  L.loss_per_layer = (int)(4 * (lp_fwd2 > lp_w2 ? lp_fwd2 : lp_w2));
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off = align_up(off + bytes, kAlign);
    return o;
  };
  const bool bf = c->act_dtype == MONE_BF16;
  L.w1c = bf ? take(nl * h * d * E) : 0;
  L.w2c = take(nl * D * h * E);
  L.w2t = take(2 * nl * h * D * E);
  L.a = take(nl * Tp * h * E);
  L.at = take(nl * h * Tp * E);
  L.dst = take(nl * h * Tp * E);
  L.g = take(nl * Tp * D * E);
  L.gt = take(nl * D * Tp * E);
  L.dzt = take(nl * h * Tp * E);
  L.xt = take(nl * d * Tp * E);
  L.loss_part = take(nl * (size_t)L.loss_per_layer * 4);
  L.loss_out = take(nl * 4);
  L.split = take(kSplitFloats * 4);  // split-K partial accumulators (short segments, reads)
  if (const int bt = block_tokens(c)) {
    L.blk = bt / c->seg_len;
    L.Btp = (int)round_up((long long)L.blk * c->seg_len, 256);
    const size_t Bp = L.Btp;
    L.bz0 = take(nl * Bp * h * 4);
    L.btgt = take(nl * Bp * D * 4);
    L.bgram = take(nl * Bp * Bp * E);
    L.ba = take(nl * Bp * h * E);
    L.bat = take(nl * h * Bp * E);
    L.bsd = take(nl * Bp * h * E);
    L.bg = take(nl * Bp * D * E);
    L.bgt = take(nl * D * Bp * E);
    L.bdzt = take(nl * h * Bp * E);
    L.bxt = take(nl * d * Bp * E);
    L.brr = take(nl * Tp * D * 4);
    L.bp = take(nl * Tp * Bp * E);
    L.bda0 = take(nl * Tp * h * 4);
    L.bq = take(nl * Tp * Bp * E);
  }
  if (c->optimizer == MONE_OPT_PAPER) {
    L.rate = take(nl * Tp * 4);
    L.vpart = take(nl * (Tp / kRateTokens) * 4);
    L.beta = take(nl * 4);
    L.norm1 = take(nl * h * 4);
    L.norm2 = take(nl * D * 4);
    L.ss1 = take(nl * h * (d / 64) * 4);
    L.ss2 = take(nl * D * (h / 64) * 4);
    L.scale1 = take(nl * h * 4);
    L.scale2 = take(nl * D * 4);
  }
  L.total = off;
  return L;
}

}  // namespace

struct mone_ttl {
  mone_ttl_config cfg;
  Layout lay;
  const void* wkv;
  float* w1;
  float* w2;
  unsigned char* ws;
  mone_paper_optimizer opt;  // MONE_OPT_PAPER only
  int last_n;           // tokens of the last non-empty segment (0: none yet)
  int w2t_cur;          // which copy of the W2^T ping-pong pair holds the current weights
  int last_loss_count;  // loss partials per layer written by that segment
  StageTimer timer;

  template <typename T>
  T* at(size_t off) const { return reinterpret_cast<T*>(ws + off); }

  void timing_begin(int stage, hipStream_t s) { timer.begin(stage, s); }
  void timing_end(int stage, hipStream_t s) { timer.end(stage, s); }
};

namespace {

// One segment step of all layers; x [L][n][d] with layer stride lsx elements.
// One segment step.  With the paper's optimiser, a multi-segment call defers the row
// renormalisations between its segments: pending says that the stored masters (and their
// copies) are diag(1/scale1) and diag(1/scale2) times the weights, so FWD1 scales Z's columns
// by scale1, FWD2 scales the A W2^T part of its product by scale2 and stores G diag(scale2)
// for the backward, and the updates read the scale times the master; finish applies this
// segment's renormalisations to the masters and their copies (the last segment of a call),
// otherwise the updates write the copies of their results and the scales are left pending.
// The weights equal those of one call per segment up to rounding.
template <typename E, bool PAPER>
int run_segment(mone_ttl* H, const void* x, long long lsx, int n, hipStream_t s,
                bool pending = false, bool finish = true) {
  const mone_ttl_config& c = H->cfg;
  const Layout& Ly = H->lay;
  const int Lc = c.n_layers, d = c.d_model, h = c.d_hidden, D = 2 * c.d_kv, Tp = Ly.Tp;
  constexpr int BK = 8 * (16 / (int)sizeof(E));
  const bool bf = sizeof(E) == 2;
  const E* w1op = bf ? H->at<E>(Ly.w1c) : reinterpret_cast<const E*>(H->w1);
  const E* w2neg = H->at<E>(Ly.w2c);
  const size_t w2t_bytes = (size_t)Lc * h * D * sizeof(E);
  E* w2t_old = H->at<E>(Ly.w2t + (size_t)H->w2t_cur * w2t_bytes);
  E* w2t_new = H->at<E>(Ly.w2t + (size_t)(H->w2t_cur ^ 1) * w2t_bytes);
  E* A = H->at<E>(Ly.a);
  E* At = H->at<E>(Ly.at);
  E* dSt = H->at<E>(Ly.dst);
  E* Gm = H->at<E>(Ly.g);
  E* Gt = H->at<E>(Ly.gt);
  E* dZt = H->at<E>(Ly.dzt);
  E* Xt = H->at<E>(Ly.xt);
  const long long lth = (long long)Tp * h, ltd = (long long)Tp * D, ltx = (long long)Tp * d;
  const int nz = (int)round_up(n, 64);  // zero-filled token extent of the transposed copies
  hipError_t e;

  // XT: X^T, the B operand of the W1 gradient (tokens become the contraction axis)
  H->timing_begin(MONE_STAGE_XT, s);
  transpose_vec_kernel<E><<<dim3((d + 63) / 64, nz / 64, Lc), dim3(256), 0, s>>>(
      reinterpret_cast<const E*>(x), lsx, d, n, d, Xt, ltx, Tp, nz);
  if ((e = hipGetLastError()) != hipSuccess) return hip_fail(e, "launch XT");
  H->timing_end(MONE_STAGE_XT, s);

  // RATE (paper optimiser): per-token rates and the momentum decay of this segment
  if constexpr (PAPER) {
    H->timing_begin(MONE_STAGE_RATE, s);
    rate_kernel<E><<<dim3(Tp / kRateTokens, Lc), dim3(256), 0, s>>>(
        reinterpret_cast<const E*>(x), lsx, d, n, H->opt.rate_w, H->opt.rate_b, H->opt.decay_w,
        c.lr, H->at<float>(Ly.rate), Tp, H->at<float>(Ly.vpart));
    decay_kernel<<<dim3((Lc + 63) / 64), dim3(64), 0, s>>>(H->at<float>(Ly.vpart),
                                                           Tp / kRateTokens, n,
                                                           H->opt.decay_b, H->at<float>(Ly.beta), Lc);
    if ((e = hipGetLastError()) != hipSuccess) return hip_fail(e, "launch RATE");
    H->timing_end(MONE_STAGE_RATE, s);
  }

  // FWD1: Z = X W1^T  ->  A, A^T, SiLU'(Z)^T
  {
    Spec sp{};
    sp.part[0].a = opnd(x, lsx, d, n);
    sp.part[0].b = opnd(w1op, (long long)h * d, d, h);
    sp.part[0].k_len = d;
    sp.nparts = 1;
    sp.m_extent = n;
    sp.n = h;
    sp.m_store = -1;
    sp.n_store = h;
    EpiFwd1<E> epi;
    epi.a = A; epi.at = At; epi.dst = dSt; epi.ls = lth; epi.h = h; epi.Tp = Tp; epi.n = n;
    epi.cs = PAPER && pending ? H->at<float>(Ly.scale1) : nullptr;
    H->timing_begin(MONE_STAGE_FWD1, s);
    if ((e = launch_gemm<E>(pick_tile(n, h, Lc), &sp, 1, Lc, epi, s, nullptr,
                            H->at<float>(Ly.split))) != hipSuccess)
      return hip_fail(e, "launch FWD1");
    H->timing_end(MONE_STAGE_FWD1, s);
  }
  // FWD2: -R = A (-W2)^T + X W_kv^T  ->  G = c R, G^T, loss partials
  {
    Spec sp{};
    const bool nip = c.loss == MONE_LOSS_NIP;
    if (nip) {  // dL/dY = -T/n needs only the targets T = X W_kv^T
      sp.part[0].a = opnd(x, lsx, d, n);
      sp.part[0].b = opnd(H->wkv, (long long)D * d, d, D);
      sp.part[0].k_len = d;
      sp.nparts = 1;
    } else {
      sp.part[0].a = opnd(A, lth, h, n);
      sp.part[0].b = opnd(w2neg, (long long)D * h, h, D);
      sp.part[0].k_len = h;
      sp.part[1].a = opnd(x, lsx, d, n);
      sp.part[1].b = opnd(H->wkv, (long long)D * d, d, D);
      sp.part[1].k_len = d;
      sp.nparts = 2;
    }
    sp.m_extent = n;
    sp.n = D;
    sp.m_store = -1;
    sp.n_store = D;
    EpiFwd2<E, PAPER> epi;
    epi.g = Gm; epi.gt = Gt; epi.loss_part = H->at<float>(Ly.loss_part); epi.ls = ltd;
    epi.D = D; epi.Tp = Tp; epi.n = n; epi.parts_per_layer = Ly.loss_per_layer;
    epi.c = c.loss == MONE_LOSS_MSE_SUM   ? 2.0f / (float)n
            : c.loss == MONE_LOSS_MSE_MEAN ? 2.0f / ((float)n * (float)D)
                                           : 1.0f / (float)n;
    epi.sq = nip ? 0 : 1;
    epi.rate = PAPER ? H->at<float>(Ly.rate) : nullptr;
    epi.gs = PAPER && pending ? H->at<float>(Ly.scale2) : nullptr;
    epi.ps = nip ? nullptr : epi.gs;
    int tiles = 0;
    H->timing_begin(MONE_STAGE_FWD2, s);
    if ((e = launch_gemm<E>(pick_tile(n, D, Lc), &sp, 1, Lc, epi, s, &tiles,
                            H->at<float>(Ly.split))) != hipSuccess)
      return hip_fail(e, "launch FWD2");
    H->timing_end(MONE_STAGE_FWD2, s);
    if (!nip) H->last_loss_count = 4 * tiles;
  }
  // BWD: dA^T = W2^T G^T (A operand W2^T [h][D], B operand G [tokens][D])  ->  dZ^T, and in
  // the same launch W2 -= lr G^T A (A operand G^T [D][tokens], B operand A^T [h][tokens])
  {
    const int kt = (int)round_up(n, BK);
    Spec sp[2] = {};
    sp[0].part[0].a = opnd(w2t_old, (long long)h * D, D, h);
    sp[0].part[0].b = opnd(Gm, ltd, D, n);
    sp[0].part[0].k_len = D;
    sp[0].nparts = 1;
    sp[0].m_extent = h;
    sp[0].n = n;
    sp[0].m_store = h;
    sp[0].n_store = -1;
    sp[1].part[0].a = opnd(Gt, ltd, Tp, D);
    sp[1].part[0].b = opnd(At, lth, Tp, h);
    sp[1].part[0].k_len = kt;
    sp[1].nparts = 1;
    sp[1].m_extent = D;
    sp[1].n = h;
    sp[1].m_store = D;
    sp[1].n_store = h;
    EpiBwdW2<E, PAPER> epi;
    epi.dst = dSt; epi.dzt = dZt; epi.lst = lth; epi.Tp = Tp; epi.n = n;
    epi.w2 = H->w2; epi.w2n = H->at<E>(Ly.w2c); epi.w2t = w2t_new;
    epi.ls2 = (long long)D * h; epi.h = h; epi.D = D; epi.lr = c.lr;
    epi.mom2 = PAPER ? H->opt.mom2 : nullptr;
    epi.beta = PAPER ? H->at<float>(Ly.beta) : nullptr;
    epi.ss2 = PAPER ? H->at<float>(Ly.ss2) : nullptr;
    epi.rs = PAPER && pending ? H->at<float>(Ly.scale2) : nullptr;
    epi.copy_pending = PAPER && !finish ? 1 : 0;
    epi.loss_part = H->at<float>(Ly.loss_part);
    epi.parts_per_layer = Ly.loss_per_layer;
    epi.nip = c.loss == MONE_LOSS_NIP ? 1 : 0;
    int tiles[2] = {0, 0};
    H->timing_begin(MONE_STAGE_BWD, s);
    if ((e = launch_gemm<E>(upd_tile(h, n, n, Lc), sp, 2, Lc, epi, s, tiles)) != hipSuccess)
      return hip_fail(e, "launch BWD");
    H->timing_end(MONE_STAGE_BWD, s);
    if (c.loss == MONE_LOSS_NIP) H->last_loss_count = 4 * tiles[1];
  }
  // UPD: W1 -= lr dZ^T X (A operand dZ^T [h][tokens], B operand X^T [d][tokens])
  {
    const int kt = (int)round_up(n, BK);
    Spec sp{};
    sp.part[0].a = opnd(dZt, lth, Tp, h);
    sp.part[0].b = opnd(Xt, ltx, Tp, d);
    sp.part[0].k_len = kt;
    sp.nparts = 1;
    sp.m_extent = h;
    sp.n = d;
    sp.m_store = h;
    sp.n_store = d;
    EpiW1<E, PAPER> epi;
    epi.w1 = H->w1; epi.w1s = bf ? H->at<E>(Ly.w1c) : nullptr;
    epi.ls1 = (long long)h * d; epi.d = d; epi.w1_copy = bf ? 1 : 0; epi.lr = c.lr;
    epi.mom1 = PAPER ? H->opt.mom1 : nullptr;
    epi.beta = PAPER ? H->at<float>(Ly.beta) : nullptr;
    epi.ss1 = PAPER ? H->at<float>(Ly.ss1) : nullptr;
    epi.h = h;
    epi.rs = PAPER && pending ? H->at<float>(Ly.scale1) : nullptr;
    epi.copy_pending = PAPER && bf && !finish ? 1 : 0;
    H->timing_begin(MONE_STAGE_UPD, s);
    if ((e = launch_gemm<E>(upd_tile(h, d, n, Lc), &sp, 1, Lc, epi, s)) != hipSuccess)
      return hip_fail(e, "launch UPD");
    H->timing_end(MONE_STAGE_UPD, s);
  }
  // RENORM (paper optimiser): the row scales that bring W1 and W2 back to their initial norms;
  // on finish, the rows rescaled and the copies the next segment reads (W1 in bf16 mode, -W2,
  // and W2^T into the other ping-pong copy)
  if constexpr (PAPER) {
    H->timing_begin(MONE_STAGE_RENORM, s);
    const long long r1 = (long long)Lc * h, r2 = (long long)Lc * D;
    row_scale_kernel<<<dim3((unsigned)((r1 + 255) / 256)), dim3(256), 0, s>>>(
        H->at<float>(Ly.ss1), d / 64, H->at<float>(Ly.norm1), H->at<float>(Ly.scale1), r1);
    row_scale_kernel<<<dim3((unsigned)((r2 + 255) / 256)), dim3(256), 0, s>>>(
        H->at<float>(Ly.ss2), h / 64, H->at<float>(Ly.norm2), H->at<float>(Ly.scale2), r2);
    const long long hd = (long long)h * d;
    if (finish) {
      renorm_w1_kernel<E><<<dim3((unsigned)((hd + 2047) / 2048), Lc), dim3(256), 0, s>>>(
          H->w1, bf ? H->at<E>(Ly.w1c) : nullptr, H->at<float>(Ly.scale1), h, d);
      renorm_w2_kernel<E><<<dim3(h / 64, D / 64, Lc), dim3(256), 0, s>>>(
          H->w2, H->at<E>(Ly.w2c), w2t_new, H->at<float>(Ly.scale2), D, h);
    }
    if ((e = hipGetLastError()) != hipSuccess) return hip_fail(e, "launch RENORM");
    H->timing_end(MONE_STAGE_RENORM, s);
  }
  H->w2t_cur ^= 1;
  H->last_n = n;
  return MONE_OK;
}

// Block form: nb consecutive segments of T tokens (nb <= blk) from x [L][nb*T][d], layer stride
// lsx, as one block.  Results equal nb run_segment calls up to the summation order.
template <typename E>
int run_block(mone_ttl* H, const E* x, long long lsx, int nb, hipStream_t s) {
  const mone_ttl_config& c = H->cfg;
  const Layout& Ly = H->lay;
  const int Lc = c.n_layers, d = c.d_model, h = c.d_hidden, D = 2 * c.d_kv, Tp = Ly.Tp;
  const int T = c.seg_len, Bt = nb * T, Bp = Ly.Btp;
  const bool bf = sizeof(E) == 2;
  const E* w1op = bf ? H->at<E>(Ly.w1c) : reinterpret_cast<const E*>(H->w1);
  const E* w2neg = H->at<E>(Ly.w2c);
  const size_t w2t_bytes = (size_t)Lc * h * D * sizeof(E);
  E* w2t_old = H->at<E>(Ly.w2t + (size_t)H->w2t_cur * w2t_bytes);
  E* w2t_new = H->at<E>(Ly.w2t + (size_t)(H->w2t_cur ^ 1) * w2t_bytes);
  float* z0 = H->at<float>(Ly.bz0);
  float* tgt = H->at<float>(Ly.btgt);
  E* gram = H->at<E>(Ly.bgram);
  E* ab = H->at<E>(Ly.ba);
  E* abt = H->at<E>(Ly.bat);
  E* sdb = H->at<E>(Ly.bsd);
  E* gb = H->at<E>(Ly.bg);
  E* gbt = H->at<E>(Ly.bgt);
  E* dzt = H->at<E>(Ly.bdzt);
  E* xt = H->at<E>(Ly.bxt);
  float* rr = H->at<float>(Ly.brr);
  E* pg = H->at<E>(Ly.bp);
  float* da0 = H->at<float>(Ly.bda0);
  E* qg = H->at<E>(Ly.bq);
  const long long lbh = (long long)Bp * h, lbd = (long long)Bp * D, lbb = (long long)Bp * Bp;
  const long long lbx = (long long)Bp * d, lth = (long long)Tp * h, ltd = (long long)Tp * D;
  const long long ltb = (long long)Tp * Bp;
  const float cmse = c.loss == MONE_LOSS_MSE_SUM ? 2.0f / (float)T
                                                 : 2.0f / ((float)T * (float)D);
  hipError_t e;

  // X^T of the block: the B operand of the block's W1 gradient
  H->timing_begin(MONE_STAGE_XT, s);
  transpose_vec_kernel<E><<<dim3((d + 63) / 64, (unsigned)(Bt / 64), Lc), dim3(256), 0, s>>>(
      x, lsx, d, Bt, d, xt, lbx, Bp, Bt);
  if ((e = hipGetLastError()) != hipSuccess) return hip_fail(e, "launch block XT");
  H->timing_end(MONE_STAGE_XT, s);

  // Block products at the block's starting weights: Z0 = X W1_0^T and the targets X W_kv^T
  // (two problems), and the token Gram matrix X X^T
  H->timing_begin(MONE_STAGE_BFWD, s);
  {
    Spec sp[2] = {};
    sp[0].part[0].a = opnd(x, lsx, d, Bt);
    sp[0].part[0].b = opnd(w1op, (long long)h * d, d, h);
    sp[0].part[0].k_len = d;
    sp[0].nparts = 1;
    sp[0].m_extent = Bt; sp[0].n = h; sp[0].m_store = -1; sp[0].n_store = h;
    sp[1] = sp[0];
    sp[1].part[0].b = opnd(H->wkv, (long long)D * d, d, D);
    sp[1].n = D; sp[1].n_store = D;
    EpiStore<float, float> epi;
    epi.p0 = z0; epi.ls0 = lbh; epi.ld0 = h; epi.s0 = 1.0f;
    epi.p1 = tgt; epi.ls1 = lbd; epi.ld1 = D; epi.s1 = 1.0f;
    if ((e = launch_gemm<E>(pick_tile(Bt, h, Lc), sp, 2, Lc, epi, s)) != hipSuccess)
      return hip_fail(e, "launch block forward");
  }
  {
    Spec sp{};
    sp.part[0].a = opnd(x, lsx, d, Bt);
    sp.part[0].b = opnd(x, lsx, d, Bt);
    sp.part[0].k_len = d;
    sp.nparts = 1;
    sp.m_extent = Bt; sp.n = Bt; sp.m_store = -1; sp.n_store = Bt;
    EpiStore<E, E> epi{};
    epi.p0 = gram; epi.ls0 = lbb; epi.ld0 = Bp; epi.s0 = 1.0f;
    if ((e = launch_gemm<E>(pick_tile(Bt, Bt, Lc), &sp, 1, Lc, epi, s)) != hipSuccess)
      return hip_fail(e, "launch token Gram");
  }
  H->timing_end(MONE_STAGE_BFWD, s);

  for (int j = 0; j < nb; ++j) {
    const int r0 = j * T, kp = j * T;  // block rows of segment j; tokens of the earlier ones
    H->timing_begin(MONE_STAGE_BSEQ, s);
    // Z_j = Z0_j - lr (X_j X_<j^T) dZ_<j  ->  A, A^T, SiLU'
    {
      Spec sp{};
      sp.part[0].a = opnd(gram + (long long)r0 * Bp, lbb, Bp, T);
      sp.part[0].b = opnd(dzt, lbh, Bp, h);
      sp.part[0].k_len = kp;
      sp.nparts = 1;
      sp.m_extent = T; sp.n = h; sp.m_store = T; sp.n_store = h;
      EpiBlkZ<E> epi;
      epi.z0 = z0; epi.a = ab; epi.at = abt; epi.sd = sdb; epi.ls = lbh;
      epi.h = h; epi.Btp = Bp; epi.r0 = r0; epi.lr = c.lr;
      if ((e = launch_gemm<E>(pick_tile(T, h, Lc), &sp, 1, Lc, epi, s, nullptr,
                              H->at<float>(Ly.split))) != hipSuccess)
        return hip_fail(e, "launch block Z");
    }
    // R0 = A_j W2_0^T - targets_j, and P = A_j A_<j^T
    {
      Spec sp[2] = {};
      sp[0].part[0].a = opnd(ab + (long long)r0 * h, lbh, h, T);
      sp[0].part[0].b = opnd(w2neg, (long long)D * h, h, D);
      sp[0].part[0].k_len = h;
      sp[0].nparts = 1;
      sp[0].m_extent = T; sp[0].n = D; sp[0].m_store = T; sp[0].n_store = D;
      sp[1] = sp[0];
      sp[1].part[0].b = opnd(ab, lbh, h, kp);
      sp[1].n = kp; sp[1].n_store = kp;
      EpiBlkY0<E> epi;
      epi.tgt = tgt; epi.lst = lbd; epi.rr = rr; epi.lsr = ltd; epi.pg = pg; epi.lsp = ltb;
      epi.D = D; epi.Btp = Bp; epi.r0 = r0;
      if ((e = launch_gemm<E>(pick_tile(T, D, Lc), sp, j > 0 ? 2 : 1, Lc, epi, s)) !=
          hipSuccess)
        return hip_fail(e, "launch block Y");
    }
    // R = R0 - lr P G_<j  ->  G = c R, G^T, loss partials
    {
      Spec sp{};
      sp.part[0].a = opnd(pg, ltb, Bp, T);
      sp.part[0].b = opnd(gbt, lbd, Bp, D);
      sp.part[0].k_len = kp;
      sp.nparts = 1;
      sp.m_extent = T; sp.n = D; sp.m_store = T; sp.n_store = D;
      EpiBlkG<E> epi;
      epi.rr = rr; epi.lsr = ltd; epi.g = gb; epi.gt = gbt; epi.lsg = lbd;
      epi.loss_part = H->at<float>(Ly.loss_part); epi.D = D; epi.Btp = Bp; epi.r0 = r0;
      epi.parts_per_layer = Ly.loss_per_layer; epi.lr = c.lr; epi.c = cmse;
      int tiles = 0;
      if ((e = launch_gemm<E>(pick_tile(T, D, Lc), &sp, 1, Lc, epi, s, &tiles,
                              H->at<float>(Ly.split))) != hipSuccess)
        return hip_fail(e, "launch block G");
      H->last_loss_count = 4 * tiles;
    }
    // dA0 = G_j W2_0 (the W2^T copy), and Q = G_j G_<j^T
    {
      Spec sp[2] = {};
      sp[0].part[0].a = opnd(gb + (long long)r0 * D, lbd, D, T);
      sp[0].part[0].b = opnd(w2t_old, (long long)h * D, D, h);
      sp[0].part[0].k_len = D;
      sp[0].nparts = 1;
      sp[0].m_extent = T; sp[0].n = h; sp[0].m_store = T; sp[0].n_store = h;
      sp[1] = sp[0];
      sp[1].part[0].b = opnd(gb, lbd, D, kp);
      sp[1].n = kp; sp[1].n_store = kp;
      EpiStore<float, E> epi;
      epi.p0 = da0; epi.ls0 = lth; epi.ld0 = h; epi.s0 = 1.0f;
      epi.p1 = qg; epi.ls1 = ltb; epi.ld1 = Bp; epi.s1 = 1.0f;
      if ((e = launch_gemm<E>(pick_tile(T, h, Lc), sp, j > 0 ? 2 : 1, Lc, epi, s)) !=
          hipSuccess)
        return hip_fail(e, "launch block dA");
    }
    // dA = dA0 - lr Q A_<j  ->  dZ^T = (dA * SiLU')^T
    {
      Spec sp{};
      sp.part[0].a = opnd(qg, ltb, Bp, T);
      sp.part[0].b = opnd(abt, lbh, Bp, h);
      sp.part[0].k_len = kp;
      sp.nparts = 1;
      sp.m_extent = T; sp.n = h; sp.m_store = T; sp.n_store = h;
      EpiBlkDZ<E> epi;
      epi.da0 = da0; epi.lsa = lth; epi.sd = sdb; epi.dzt = dzt; epi.ls = lbh;
      epi.h = h; epi.Btp = Bp; epi.r0 = r0; epi.lr = c.lr;
      if ((e = launch_gemm<E>(pick_tile(T, h, Lc), &sp, 1, Lc, epi, s, nullptr,
                              H->at<float>(Ly.split))) != hipSuccess)
        return hip_fail(e, "launch block dZ");
    }
    H->timing_end(MONE_STAGE_BSEQ, s);
  }

  // The block's updates in one launch: W2 -= lr G^T A (writing -W2 and the other W2^T copy)
  // and W1 -= lr dZ^T X (writing its copy)
  H->timing_begin(MONE_STAGE_BUPD, s);
  {
    Spec sp[2] = {};
    sp[0].part[0].a = opnd(gbt, lbd, Bp, D);
    sp[0].part[0].b = opnd(abt, lbh, Bp, h);
    sp[0].part[0].k_len = Bt;
    sp[0].nparts = 1;
    sp[0].m_extent = D; sp[0].n = h; sp[0].m_store = D; sp[0].n_store = h;
    sp[1].part[0].a = opnd(dzt, lbh, Bp, h);
    sp[1].part[0].b = opnd(xt, lbx, Bp, d);
    sp[1].part[0].k_len = Bt;
    sp[1].nparts = 1;
    sp[1].m_extent = h; sp[1].n = d; sp[1].m_store = h; sp[1].n_store = d;
    EpiBlkUpd<E> epi{};
    epi.w2.w2 = H->w2; epi.w2.w2n = H->at<E>(Ly.w2c); epi.w2.w2t = w2t_new;
    epi.w2.ls2 = (long long)D * h; epi.w2.h = h; epi.w2.D = D; epi.w2.lr = c.lr;
    epi.w1.w1 = H->w1; epi.w1.w1s = bf ? H->at<E>(Ly.w1c) : nullptr;
    epi.w1.ls1 = (long long)h * d; epi.w1.d = d; epi.w1.w1_copy = bf ? 1 : 0;
    epi.w1.lr = c.lr; epi.w1.h = h;
    if ((e = launch_gemm<E>(upd_tile(h, d, Bt, Lc), sp, 2, Lc, epi, s)) != hipSuccess)
      return hip_fail(e, "launch block updates");
  }
  H->timing_end(MONE_STAGE_BUPD, s);
  H->w2t_cur ^= 1;
  H->last_n = T;
  return MONE_OK;
}

template <typename E>
int run_kv(mone_ttl* H, const void* xq, int q, void* kv, int kv_bf16, hipStream_t s) {
  const mone_ttl_config& c = H->cfg;
  const Layout& Ly = H->lay;
  const int Lc = c.n_layers, d = c.d_model, h = c.d_hidden, D = 2 * c.d_kv, Tp = Ly.Tp;
  const bool bf = sizeof(E) == 2;
  const E* w1op = bf ? H->at<E>(Ly.w1c) : reinterpret_cast<const E*>(H->w1);
  const E* w2neg = H->at<E>(Ly.w2c);
  E* A = H->at<E>(Ly.a);  // scratch for A_q (the TTL intermediates are dead between calls)
  const long long lth = (long long)Tp * h;
  const size_t kvE = kv_bf16 ? 2 : 4;
  hipError_t e;
  for (int q0 = 0; q0 < q; q0 += Tp) {
    const int qc = q - q0 < Tp ? q - q0 : Tp;
    const E* xc = reinterpret_cast<const E*>(xq) + (long long)q0 * d;
    void* kvc = reinterpret_cast<unsigned char*>(kv) + (size_t)q0 * D * kvE;
    {
      Spec sp{};
      sp.part[0].a = opnd(xc, (long long)q * d, d, qc);
      sp.part[0].b = opnd(w1op, (long long)h * d, d, h);
      sp.part[0].k_len = d;
      sp.nparts = 1;
      sp.m_extent = qc;
      sp.n = h;
      sp.m_store = -1;
      sp.n_store = h;
      EpiKv1<E> epi;
      epi.a = A; epi.ls = lth; epi.h = h;
      H->timing_begin(MONE_STAGE_KV1, s);
      if ((e = launch_gemm<E>(pick_tile(qc, h, Lc), &sp, 1, Lc, epi, s, nullptr,
                              H->at<float>(Ly.split))) != hipSuccess)
        return hip_fail(e, "launch KV1");
      H->timing_end(MONE_STAGE_KV1, s);
    }
    {
      Spec sp{};
      sp.part[0].a = opnd(A, lth, h, qc);
      sp.part[0].b = opnd(w2neg, (long long)D * h, h, D);
      sp.part[0].k_len = h;
      sp.nparts = 1;
      sp.m_extent = qc;
      sp.n = D;
      sp.m_store = qc;
      sp.n_store = D;
      EpiKv2 epi;
      epi.kv = kvc; epi.ls = (long long)q * D; epi.D = D; epi.bf16_out = kv_bf16;
      H->timing_begin(MONE_STAGE_KV2, s);
      if ((e = launch_gemm<E>(pick_tile(qc, D, Lc), &sp, 1, Lc, epi, s, nullptr,
                              H->at<float>(Ly.split))) != hipSuccess)
        return hip_fail(e, "launch KV2");
      H->timing_end(MONE_STAGE_KV2, s);
    }
  }
  return MONE_OK;
}

}  // namespace

namespace {

// Pointer checks shared by the handle and the no-allocation step.
int check_state(const void* wkv, const float* w1, const float* w2) {
  if (!wkv || !w1 || !w2) return fail(MONE_EINVAL, "wkv, w1 and w2 must be non-NULL");
  if (!aligned16(wkv) || !aligned16(w1) || !aligned16(w2))
    return fail(MONE_EINVAL, "wkv, w1 and w2 must be 16-byte aligned");
  return MONE_OK;
}

// Fills a handle over the workspace ws (the layout's total bytes): clears the workspace and
// builds the weight copies from the fp32 masters (and, with the paper's optimiser, the row-norm
// targets).  No host or device allocation.
int init_state(mone_ttl* H, const mone_ttl_config* cfg, const Layout& Ly, const void* wkv,
               float* w1, float* w2, const mone_paper_optimizer* opt, unsigned char* ws,
               hipStream_t s) {
  H->cfg = *cfg;
  H->lay = Ly;
  H->wkv = wkv;
  H->w1 = w1;
  H->w2 = w2;
  H->ws = ws;
  H->last_n = 0;
  H->last_loss_count = 0;
  H->w2t_cur = 0;
  if (opt) H->opt = *opt;
  const int Lc = cfg->n_layers, d = cfg->d_model, h = cfg->d_hidden, D = 2 * cfg->d_kv;
  hipError_t e = hipMemsetAsync(ws, 0, Ly.total, s);
  if (e != hipSuccess) return hip_fail(e, "clearing the workspace");
  const long long n1 = (long long)Lc * h * d, n2 = (long long)Lc * D * h;
  if (cfg->act_dtype == MONE_BF16) {
    convert_kernel<bf16_t><<<dim3(2048), dim3(256), 0, s>>>(w1, H->at<bf16_t>(Ly.w1c), n1, 1.0f);
    convert_kernel<bf16_t><<<dim3(2048), dim3(256), 0, s>>>(w2, H->at<bf16_t>(Ly.w2c), n2, -1.0f);
    transpose_kernel<float, bf16_t><<<dim3((h + 63) / 64, (D + 63) / 64, Lc), dim3(256), 0, s>>>(
        w2, (long long)D * h, h, D, h, H->at<bf16_t>(Ly.w2t), (long long)h * D, D, D);
  } else {
    convert_kernel<float><<<dim3(2048), dim3(256), 0, s>>>(w2, H->at<float>(Ly.w2c), n2, -1.0f);
    transpose_kernel<float, float><<<dim3((h + 63) / 64, (D + 63) / 64, Lc), dim3(256), 0, s>>>(
        w2, (long long)D * h, h, D, h, H->at<float>(Ly.w2t), (long long)h * D, D, D);
  }
  if (opt) {  // the renormalisation targets: row norms of the initial weights
    row_norm_kernel<<<dim3((h + 3) / 4, Lc), dim3(256), 0, s>>>(w1, h, d, H->at<float>(Ly.norm1));
    row_norm_kernel<<<dim3((D + 3) / 4, Lc), dim3(256), 0, s>>>(w2, D, h, H->at<float>(Ly.norm2));
  }
  if ((e = hipGetLastError()) != hipSuccess) return hip_fail(e, "building the weight copies");
  return MONE_OK;
}

int create_handle(mone_ttl** out, const mone_ttl_config* cfg, const void* wkv, float* w1,
                  float* w2, const mone_paper_optimizer* opt, void* workspace,
                  size_t workspace_bytes, void* stream) {
  if (!out) return fail(MONE_EINVAL, "out is NULL");
  *out = nullptr;
  int rc = check_config(cfg);
  if (rc != MONE_OK) return rc;
  if ((rc = check_state(wkv, w1, w2)) != MONE_OK) return rc;
  if (!workspace) return fail(MONE_EINVAL, "workspace must be non-NULL");
  if (((uintptr_t)workspace & (kAlign - 1)) != 0)
    return fail(MONE_EINVAL, "workspace must be 256-byte aligned");
  const Layout Ly = make_layout(cfg);
  if (workspace_bytes < Ly.total)
    return fail(MONE_EINVAL, "workspace has %zu bytes, %zu needed", workspace_bytes, Ly.total);

  mone_ttl* H = new (std::nothrow) mone_ttl();
  if (!H) return fail(MONE_EINVAL, "host allocation failed");
  rc = init_state(H, cfg, Ly, wkv, w1, w2, opt, reinterpret_cast<unsigned char*>(workspace),
                  reinterpret_cast<hipStream_t>(stream));
  if (rc != MONE_OK) {
    delete H;
    return rc;
  }
  *out = H;
  return MONE_OK;
}

// Workspace of mone_ttl_step_noalloc: a static device array, one copy per device for the life
// of the process.  In host code `scratch` names a host-side stand-in, never the device memory:
// its device address comes from hipGetSymbolAddress, once per device, and only that address
// is passed to kernels and to hipMemsetAsync.
constexpr size_t kScratchBytes = (size_t)64 << 20;
__device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
unsigned char* g_scratch_dev[kMaxDevices] = {};

int scratch_address(unsigned char** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices) return fail(MONE_EUNSUPPORTED, "device %d", dev);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_dev[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
    if (!p || ((uintptr_t)p & (kAlign - 1)) != 0)
      return fail(MONE_EHIP, "static scratch at %p is not 256-byte aligned", p);
    g_scratch_dev[dev] = reinterpret_cast<unsigned char*>(p);
  }
  *out = g_scratch_dev[dev];
  return MONE_OK;
}

}  // namespace

extern "C" {

size_t mone_ttl_workspace_bytes(const mone_ttl_config* cfg) {
  g_err[0] = 0;
  if (check_config(cfg) != MONE_OK) return 0;
  return make_layout(cfg).total;
}

int mone_ttl_init(mone_ttl** out, const mone_ttl_config* cfg, const void* wkv, float* w1,
                  float* w2, void* workspace, size_t workspace_bytes, void* stream) {
  g_err[0] = 0;
  if (cfg && cfg->optimizer != MONE_OPT_SGD) {
    if (out) *out = nullptr;
    return fail(MONE_EINVAL, "optimizer %d needs mone_ttl_init_paper", cfg->optimizer);
  }
  return create_handle(out, cfg, wkv, w1, w2, nullptr, workspace, workspace_bytes, stream);
}

int mone_ttl_init_paper(mone_ttl** out, const mone_ttl_config* cfg, const void* wkv, float* w1,
                        float* w2, const mone_paper_optimizer* opt, void* workspace,
                        size_t workspace_bytes, void* stream) {
  g_err[0] = 0;
  if (out) *out = nullptr;
  if (cfg && cfg->optimizer != MONE_OPT_PAPER)
    return fail(MONE_EINVAL, "mone_ttl_init_paper needs optimizer MONE_OPT_PAPER");
  if (!opt) return fail(MONE_EINVAL, "opt is NULL");
  if (!opt->rate_w || !opt->rate_b || !opt->decay_w || !opt->decay_b || !opt->mom1 || !opt->mom2)
    return fail(MONE_EINVAL, "every pointer of the optimiser state must be non-NULL");
  if (!aligned16(opt->rate_w) || !aligned16(opt->decay_w) || !aligned16(opt->mom1) ||
      !aligned16(opt->mom2))
    return fail(MONE_EINVAL, "rate_w, decay_w, mom1 and mom2 must be 16-byte aligned");
  return create_handle(out, cfg, wkv, w1, w2, opt, workspace, workspace_bytes, stream);
}

int mone_ttl_segment(mone_ttl* H, const void* x, int32_t n_tokens, void* stream) {
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
    return paper ? run_segment<bf16_t, true>(H, x, lsx, n_tokens, s)
                 : run_segment<bf16_t, false>(H, x, lsx, n_tokens, s);
  return paper ? run_segment<float, true>(H, x, lsx, n_tokens, s)
               : run_segment<float, false>(H, x, lsx, n_tokens, s);
}

int mone_ttl_segments(mone_ttl* H, const void* x, int64_t layer_stride, int32_t n_segments,
                      void* stream) {
  g_err[0] = 0;
  if (!H) return fail(MONE_EINVAL, "handle is NULL");
  if (n_segments < 0) return fail(MONE_EINVAL, "n_segments = %d is negative", n_segments);
  if (n_segments == 0) return MONE_OK;
  const mone_ttl_config& c = H->cfg;
  const long long T = c.seg_len, d = c.d_model;
  if (layer_stride < (long long)n_segments * T * d)
    return fail(MONE_EINVAL, "layer_stride %lld below n_segments * seg_len * d_model = %lld",
                (long long)layer_stride, (long long)n_segments * T * d);
  if (!x) return fail(MONE_EINVAL, "x is NULL");
  const long long E = c.act_dtype == MONE_BF16 ? 2 : 4;
  if (!aligned16(x) || (layer_stride * E) % 16 != 0)
    return fail(MONE_EINVAL, "x and layer_stride * element size must be 16-byte aligned");
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const bool bf = c.act_dtype == MONE_BF16, paper = c.optimizer == MONE_OPT_PAPER;
  const int blk = H->lay.blk;
  int done = 0, rc = MONE_OK;
  while (done < n_segments && rc == MONE_OK) {
    const int nb = blk > 1 ? (n_segments - done < blk ? n_segments - done : blk) : 1;
    const unsigned char* xs = reinterpret_cast<const unsigned char*>(x) + done * T * d * E;
    if (nb > 1) {
      rc = bf ? run_block<bf16_t>(H, reinterpret_cast<const bf16_t*>(xs), layer_stride, nb, s)
              : run_block<float>(H, reinterpret_cast<const float*>(xs), layer_stride, nb, s);
    } else {
      // paper's optimiser: the row renormalisations deferred to the call's last segment
      const bool pending = done > 0, finish = done + 1 == n_segments;
      if (bf)
        rc = paper ? run_segment<bf16_t, true>(H, xs, layer_stride, (int)T, s, pending, finish)
                   : run_segment<bf16_t, false>(H, xs, layer_stride, (int)T, s);
      else
        rc = paper ? run_segment<float, true>(H, xs, layer_stride, (int)T, s, pending, finish)
                   : run_segment<float, false>(H, xs, layer_stride, (int)T, s);
    }
    done += nb;
  }
  return rc;
}

int mone_ttl_step_noalloc(const mone_ttl_config* cfg, const void* wkv, float* w1, float* w2,
                          const void* x, int32_t n_tokens, void* stream) {
  g_err[0] = 0;
  int rc = check_config(cfg);
  if (rc != MONE_OK) return rc;
  if (cfg->optimizer != MONE_OPT_SGD)
    return fail(MONE_EUNSUPPORTED, "mone_ttl_step_noalloc takes plain SGD only (the paper's "
                "optimiser keeps state across segments: use a handle)");
  if ((rc = check_state(wkv, w1, w2)) != MONE_OK) return rc;
  if (n_tokens < 0 || n_tokens > cfg->seg_len)
    return fail(MONE_EINVAL, "n_tokens %d outside [0, seg_len=%d]", n_tokens, cfg->seg_len);
  const Layout Ly = make_layout(cfg);
  if (Ly.total > kScratchBytes)
    return fail(MONE_EUNSUPPORTED, "this configuration needs %zu bytes of workspace; the static "
                "scratch of mone_ttl_step_noalloc holds %zu (use mone_ttl_init with a workspace)",
                Ly.total, kScratchBytes);
  if (n_tokens == 0) return MONE_OK;
  if (!x) return fail(MONE_EINVAL, "x is NULL");
  if (!aligned16(x)) return fail(MONE_EINVAL, "x must be 16-byte aligned");
  unsigned char* ws = nullptr;
  if ((rc = scratch_address(&ws)) != MONE_OK) return rc;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  mone_ttl H;  // on the stack: the handle's state for this one step
  if ((rc = init_state(&H, cfg, Ly, wkv, w1, w2, nullptr, ws, s)) != MONE_OK) return rc;
  const long long lsx = (long long)n_tokens * cfg->d_model;
  return cfg->act_dtype == MONE_BF16 ? run_segment<bf16_t, false>(&H, x, lsx, n_tokens, s)
                                     : run_segment<float, false>(&H, x, lsx, n_tokens, s);
}

int mone_memory_kv(mone_ttl* H, const void* xq, int32_t q, void* kv, int32_t kv_dtype,
                   void* stream) {
  g_err[0] = 0;
  if (!H) return fail(MONE_EINVAL, "handle is NULL");
  if (q < 0) return fail(MONE_EINVAL, "q = %d is negative", q);
  if (kv_dtype != MONE_F32 && kv_dtype != MONE_BF16)
    return fail(MONE_EINVAL, "kv_dtype %d is not MONE_F32 or MONE_BF16", kv_dtype);
  if (q == 0) return MONE_OK;
  if (!xq || !kv) return fail(MONE_EINVAL, "xq and kv must be non-NULL");
  if (!aligned16(xq) || !aligned16(kv)) return fail(MONE_EINVAL, "xq and kv must be 16-byte aligned");
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const int kvb = kv_dtype == MONE_BF16 ? 1 : 0;
  return H->cfg.act_dtype == MONE_BF16 ? run_kv<bf16_t>(H, xq, q, kv, kvb, s)
                                       : run_kv<float>(H, xq, q, kv, kvb, s);
}

int mone_memory_attention(mone_ttl* H, const void* qh, const void* kh, const void* vh,
                          const void* kv_mem, int32_t kv_dtype, int32_t q, int32_t n_heads,
                          int32_t n_kv_heads, void* out, int32_t out_dtype, void* stream) {
  g_err[0] = 0;
  if (!H) return fail(MONE_EINVAL, "handle is NULL");
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const bool timed = q > 0;
  if (timed) H->timing_begin(MONE_STAGE_ATTN, s);
  const int rc = launch_attention(H->cfg.n_layers, H->cfg.d_kv, H->cfg.act_dtype == MONE_BF16,
                                  qh, kh, vh, kv_mem, kv_dtype, q, n_heads, n_kv_heads, out,
                                  out_dtype, s);
  if (rc == MONE_OK && timed) H->timing_end(MONE_STAGE_ATTN, s);
  return rc;
}

int mone_ttl_loss(mone_ttl* H, float* out_host, void* stream) {
  g_err[0] = 0;
  if (!H || !out_host) return fail(MONE_EINVAL, "handle and out_host must be non-NULL");
  if (H->last_n == 0) return fail(MONE_ESTATE, "no non-empty segment has been processed");
  if (H->cfg.loss == MONE_LOSS_NIP && H->cfg.optimizer == MONE_OPT_PAPER)
    return fail(MONE_EUNSUPPORTED, "the negative inner product's loss is not formed with the "
                "paper optimiser (only its rate-weighted gradient is)");
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const mone_ttl_config& c = H->cfg;
  const float n = (float)H->last_n;
  // sum-of-squares partials for the squared errors; for the negative inner product the
  // partials already sum to L_s
  const float scale = c.loss == MONE_LOSS_MSE_SUM    ? 1.0f / n
                      : c.loss == MONE_LOSS_MSE_MEAN ? 1.0f / (n * 2.0f * c.d_kv)
                                                     : 1.0f;
  float* dev_out = H->at<float>(H->lay.loss_out);
  loss_finalize_kernel<<<dim3(c.n_layers), dim3(256), 0, s>>>(
      H->at<float>(H->lay.loss_part), H->lay.loss_per_layer, H->last_loss_count, scale, dev_out);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_fail(e, "launch loss");
  if ((e = hipMemcpyAsync(out_host, dev_out, sizeof(float) * c.n_layers, hipMemcpyDeviceToHost,
                          s)) != hipSuccess)
    return hip_fail(e, "copy loss");
  if ((e = hipStreamSynchronize(s)) != hipSuccess) return hip_fail(e, "synchronise");
  return MONE_OK;
}

int mone_ttl_destroy(mone_ttl* H) {
  g_err[0] = 0;
  if (!H) return MONE_OK;
  H->timer.destroy();
  delete H;
  return MONE_OK;
}

const char* mone_ttl_last_error(void) { return g_err; }

int mone_ttl_set_stage_timing(mone_ttl* H, int32_t max_records, uint32_t stage_mask) {
  g_err[0] = 0;
  if (!H) return fail(MONE_EINVAL, "handle is NULL");
  return H->timer.enable(max_records, stage_mask);
}

int mone_ttl_stage_times(mone_ttl* H, double* ms_sum, int32_t* count) {
  g_err[0] = 0;
  if (!H || !ms_sum || !count) return fail(MONE_EINVAL, "NULL argument");
  return H->timer.report(ms_sum, count, MONE_N_STAGES);
}

}  // extern "C"
