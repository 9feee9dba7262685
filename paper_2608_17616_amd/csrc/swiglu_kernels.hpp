// Device code of the paper-form memory (SwiGLU per fast-weight head, Eq. swiglu) for gfx950:
// the epilogues of its grouped GEMMs and its memory-bound kernels.
//
// Heads are the batch axis of every per-head GEMM: operand b = l * H + e is head e of layer l,
// stored head-major so that one layer stride addresses it.  Contractions over a head's d_h
// channels run over d_hp = d_h rounded up to 64 columns, the padding held at zero by every
// writer.  Token axes have Tp = seg_len rounded up to 256 entries; tokens at or past the
// segment's n are zero in every operand that a later GEMM contracts over.
#pragma once

#include "kernels.hpp"

namespace mone {
namespace {

// PROJ: tile of X [P_k ; P_v]^T = [raw keys | raw values] [tokens][2d], stored in fp32.
struct EpiSwProj : EpiBase {
  float* raw;
  long long ls;  // Tp * 2d
  int ld;        // 2d
  __device__ __forceinline__ float rows8(int, int layer, int row, int col, int, int,
                                         float (&v)[8], const float (&)[8]) const {
    store8(raw + (long long)layer * ls + (long long)row * ld + col, v);
    return 0.0f;
  }
};

// DA: tile of dA0^T = W_out dY0^T [d_h][tokens] for one head, with dY0 = -V / n the output
// gradient at unit rates: the gradient of the loss with respect to the hidden activations A.
template <typename E>
struct EpiSwDa : EpiBase {
  E* dat;
  long long ls;  // d_h * Tp
  int Tp;
  __device__ __forceinline__ float rows8(int, int b, int row, int col, int, int,
                                         float (&v)[8], const float (&)[8]) const {
    store8(dat + (long long)b * ls + (long long)row * Tp + col, v);
    return 0.0f;
  }
};

// FWD: tile of [Z | G]^T = W_ig K^T [2 d_h][tokens], whose rows interleave the two branches of
// Eq. swiglu: row 2i is z_i = W_in[i] . k, row 2i + 1 is g_i = W_gate[i] . k.  Rows come in
// pairs; for hidden unit i and 8 tokens the epilogue forms
//   a = SiLU(z) g                        -> A^T row i
//   dZ = eta dA0 g SiLU'(z)              -> row 2i of [dZ | dG]^T
//   dG = eta dA0 SiLU(z)                 -> row 2i + 1
// with dA0 from the DA stage and eta the token's rate (lr for SGD), and sums a * dA0 into the
// loss partials: the loss is A against its unit-rate gradient.  Tokens >= n are stored as 0.
template <typename E>
struct EpiSwFwd : EpiBase {
  static constexpr bool kPre = true;
  static constexpr int kAux = 16;
  static constexpr bool kPairRows = true;
  const E* dat;        // [B][d_h][Tp]
  const float* rate;   // [L][Tp] per-token rates, or null (constant lr)
  E* at;               // [B][d_h][Tp]
  E* dzgt;             // [B][2 d_h][Tp]
  float* loss_part;    // [B][parts]
  long long ls;        // d_h * Tp
  int Tp, n, H, parts;
  float lr;
  __device__ __forceinline__ void pre8(int, int b, int row, int col, int, int,
                                       float (&w)[kAux]) const {
    load8(dat + (long long)b * ls + (long long)(row >> 1) * Tp + col,
          *reinterpret_cast<float(*)[8]>(&w[0]));
    if (rate) load8(rate + (long long)(b / H) * Tp + col, *reinterpret_cast<float(*)[8]>(&w[8]));
  }
  __device__ __forceinline__ float rows8p(int, int b, int row, int col, int, int,
                                          const float (&z)[8], const float (&g)[8],
                                          const float (&w)[kAux]) const {
    float av[8], dz[8], dg[8], loss = 0.0f;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const bool ok = col + e < n;
      const float s = sigmoidf_(z[e]);
      const float si = z[e] * s;
      const float a = si * g[e];
      const float da = w[e];
      const float eda = (rate ? w[8 + e] : lr) * da;
      av[e] = ok ? a : 0.0f;
      dz[e] = ok ? eda * g[e] * (s * (1.0f + z[e] * (1.0f - s))) : 0.0f;
      dg[e] = ok ? eda * si : 0.0f;
      loss += ok ? a * da : 0.0f;
    }
    store8(at + (long long)b * ls + (long long)(row >> 1) * Tp + col, av);
    E* o = dzgt + (long long)b * 2 * ls + (long long)row * Tp + col;
    store8(o, dz);
    store8(o + Tp, dg);
    return loss;
  }
  __device__ __forceinline__ void finish(int, int b, int tile, int wave, int lane,
                                         float s) const {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off, 64);
    if (lane == 0) loss_part[(long long)b * parts + tile * 4 + wave] = s;
  }
};

// UPD: problem 0 is the tile of A^T dY [d_h][d_h] (the gradient of W_out, rows = hidden
// units), problem 1 the tile of [dZ | dG]^T K [2 d_h][d_h] (the gradients of W_in and W_gate,
// rows interleaved as in FWD).  The rates are already inside dY and dZ, dG, so the SGD update is
// W - acc.  fp32 read-modify-write of the masters, then the MFMA copies the next segment reads:
// W_ig (interleaved rows) and W_out, d_hp columns each.  With the paper's optimiser (PAPER):
// mu = beta mu + acc, W - mu, and each row chunk's sum of squares for the renormalisation,
// which writes the copies afterwards.
template <typename E, bool PAPER>
struct EpiSwUpd : EpiBase {
  static constexpr bool kPre = true;
  static constexpr int kAux = PAPER ? 16 : 8;
  static constexpr bool kRowNorm = PAPER;
  float* w_in; float* w_gate; float* w_out;   // masters [B][d_h][d_h]
  float* m_in; float* m_gate; float* m_out;   // PAPER: momenta, same layout
  E* wig; E* woc;                             // copies [B][2 d_h][d_hp], [B][d_h][d_hp]
  const float* beta;                          // PAPER: [L]
  float* ss_ig; float* ss_out;                // PAPER: [B][2 d_h][nseg], [B][d_h][nseg]
  long long lsw;                              // d_h * d_h
  int dh, dhp, H, nseg;
  __device__ __forceinline__ long long off(int pi, int b, int row, int col) const {
    return (long long)b * lsw + (long long)(pi ? row >> 1 : row) * dh + col;
  }
  __device__ __forceinline__ float* master(int pi, int row) const {
    return pi == 0 ? w_out : (row & 1) ? w_gate : w_in;
  }
  __device__ __forceinline__ float* mom(int pi, int row) const {
    return pi == 0 ? m_out : (row & 1) ? m_gate : m_in;
  }
  __device__ __forceinline__ void pre8(int pi, int b, int row, int col, int, int,
                                       float (&w)[kAux]) const {
    const long long o = off(pi, b, row, col);
    load8(master(pi, row) + o, *reinterpret_cast<float(*)[8]>(&w[0]));
    if constexpr (PAPER) load8(mom(pi, row) + o, *reinterpret_cast<float(*)[8]>(&w[8]));
  }
  __device__ __forceinline__ float rows8(int pi, int b, int row, int col, int, int,
                                         float (&v)[8], const float (&w)[kAux]) const {
    const long long o = off(pi, b, row, col);
    float nw[8];
    if constexpr (PAPER) {
      const float bt = beta[b / H];
      float m[8], ss = 0.0f;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        m[e] = bt * w[8 + e] + v[e];
        nw[e] = w[e] - m[e];
        ss += nw[e] * nw[e];
      }
      store8(mom(pi, row) + o, m);
      store8(master(pi, row) + o, nw);
      return ss;
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) nw[e] = w[e] - v[e];
      store8(master(pi, row) + o, nw);
      E* cp = pi == 0 ? woc + ((long long)b * dh + row) * dhp + col
                      : wig + ((long long)b * 2 * dh + row) * dhp + col;
      store8(cp, nw);
      return 0.0f;
    }
  }
  __device__ __forceinline__ void row_partial(int pi, int b, int row, int cb, float ss) const {
    if (PAPER) {
      if (pi == 0)
        ss_out[((long long)b * dh + row) * nseg + cb] = ss;
      else
        ss_ig[((long long)b * 2 * dh + row) * nseg + cb] = ss;
    }
  }
};

// RoPE table: tab[p][c] = (cos, sin) of p * base^(-2c/d_h) for positions p < Tp and channel
// pairs c < d_h / 2, evaluated in double precision.
__global__ void sw_rope_table_kernel(float2* __restrict__ tab, int Tp, int dh, double base) {
  const int half = dh / 2;
  const long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (long long)Tp * half) return;
  const int p = (int)(i / half), c = (int)(i - (long long)p * half);
  const double ang = (double)p * pow(base, -2.0 * (double)c / (double)dh);
  double sn, cs;
  sincos(ang, &sn, &cs);
  tab[i] = make_float2((float)cs, (float)sn);
}

// PREP: one workgroup per (TB tokens, head e, layer l).  From the fp32 raw projections:
//   keys   SiLU(s r + b) per channel, divided by max(norm, 1e-12) per token, then rotated by
//          RoPE at the token's position; written as K [B][Tp][d_hp] (zero padding columns) and
//          K^T [B][d_h][Tp];
//   values SiLU(r); written as dY0 = -v / n [B][Tp][d_hp] (unit rates, zero padding) and
//          dY^T = -eta v / n [B][d_h][Tp] (eta the token's rate, or lr).
// Tokens n <= j < j0 + TB are written as 0.  Dynamic LDS: TB * (d_h + 1) + TB floats.
template <typename E>
__global__ __launch_bounds__(256) void sw_prep_kernel(
    const float* __restrict__ raw, long long raw_ls, int d, int n, int H, int dh, int dhp,
    int Tp, int TB, const float* __restrict__ kscale, const float* __restrict__ kshift,
    const float2* __restrict__ rope, const float* __restrict__ rate, float lr, float inv_n,
    E* __restrict__ kh, E* __restrict__ kt, E* __restrict__ dy, E* __restrict__ dyt) {
  extern __shared__ float sm[];
  const int LD = dh + 1;
  float* sk = sm;
  float* sinv = sm + TB * LD;
  const int j0 = blockIdx.x * TB, e = blockIdx.y, l = blockIdx.z, b = l * H + e;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int d2 = 2 * d, half = dh / 2;
  const float* rk = raw + (long long)l * raw_ls + (long long)e * dh;
  const float* sc = kscale + (long long)l * d + (long long)e * dh;
  const float* sh = kshift + (long long)l * d + (long long)e * dh;
  const long long okh = (long long)b * Tp * dhp, okt = (long long)b * dh * Tp;

  // keys: affine, SiLU
  for (int i = tid; i < TB * dh; i += 256) {
    const int t = i / dh, c = i - t * dh, j = j0 + t;
    float kv = 0.0f;
    if (j < n) {
      const float u = sc[c] * rk[(long long)j * d2 + c] + sh[c];
      kv = u * sigmoidf_(u);
    }
    sk[t * LD + c] = kv;
  }
  __syncthreads();
  // per-token inverse norms (one wave per token, fixed-order reduction)
  for (int t = wave; t < TB; t += 4) {
    float ss = 0.0f;
    for (int c = lane; c < dh; c += 64) {
      const float x = sk[t * LD + c];
      ss += x * x;
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) ss += __shfl_xor(ss, off, 64);
    if (lane == 0) sinv[t] = 1.0f / fmaxf(sqrtf(ss), 1e-12f);
  }
  __syncthreads();
  // normalise and rotate in place; row-major copy with zero padding
  for (int i = tid; i < TB * half; i += 256) {
    const int t = i / half, c = i - t * half, j = j0 + t;
    const float inv = sinv[t];
    const float x1 = sk[t * LD + c] * inv, x2 = sk[t * LD + c + half] * inv;
    const float2 cs = rope[(long long)j * half + c];
    const float o1 = x1 * cs.x - x2 * cs.y, o2 = x1 * cs.y + x2 * cs.x;
    sk[t * LD + c] = o1;
    sk[t * LD + c + half] = o2;
    E* kr = kh + okh + (long long)j * dhp;
    kr[c] = from_f32<E>(o1);
    kr[c + half] = from_f32<E>(o2);
  }
  const int pad = dhp - dh;
  for (int i = tid; i < TB * pad; i += 256) {
    const int t = i / pad, c = dh + i - t * pad;
    kh[okh + (long long)(j0 + t) * dhp + c] = from_f32<E>(0.0f);
  }
  __syncthreads();
  for (int i = tid; i < dh * TB; i += 256) {
    const int c = i / TB, t = i - c * TB;
    kt[okt + (long long)c * Tp + j0 + t] = from_f32<E>(sk[t * LD + c]);
  }
  __syncthreads();
  // values: SiLU
  const float* rv = rk + d;
  for (int i = tid; i < TB * dh; i += 256) {
    const int t = i / dh, c = i - t * dh, j = j0 + t;
    float vv = 0.0f;
    if (j < n) {
      const float r = rv[(long long)j * d2 + c];
      vv = r * sigmoidf_(r);
    }
    sk[t * LD + c] = vv;
  }
  __syncthreads();
  for (int i = tid; i < TB * dhp; i += 256) {
    const int t = i / dhp, c = i - t * dhp;
    const float val = c < dh ? -sk[t * LD + c] * inv_n : 0.0f;
    dy[okh + (long long)(j0 + t) * dhp + c] = from_f32<E>(val);
  }
  for (int i = tid; i < dh * TB; i += 256) {
    const int c = i / TB, t = i - c * TB, j = j0 + t;
    const float eta = rate ? rate[(long long)l * Tp + j] : lr;
    dyt[okt + (long long)c * Tp + j] = from_f32<E>(-eta * sk[t * LD + c] * inv_n);
  }
}

// The MFMA copies of the fast weights: W_ig [B][2 d_h][d_hp] (row 2i = W_in row i, row 2i + 1
// = W_gate row i) and W_out [B][d_h][d_hp], zero in the padding columns.
// Grid (ceil(3 d_h d_hp / 256), B).
template <typename E>
__global__ __launch_bounds__(256) void sw_pack_kernel(const float* __restrict__ w_in,
                                                      const float* __restrict__ w_gate,
                                                      const float* __restrict__ w_out, int dh,
                                                      int dhp, E* __restrict__ wig,
                                                      E* __restrict__ woc) {
  const int b = blockIdx.y;
  const long long i = (long long)blockIdx.x * 256 + threadIdx.x;
  if (i >= 3LL * dh * dhp) return;
  const int r = (int)(i / dhp), c = (int)(i - (long long)r * dhp);
  const long long wb = (long long)b * dh * dh;
  float v = 0.0f;
  if (c < dh)
    v = r < 2 * dh ? ((r & 1) ? w_gate : w_in)[wb + (long long)(r >> 1) * dh + c]
                   : w_out[wb + (long long)(r - 2 * dh) * dh + c];
  if (r < 2 * dh)
    wig[((long long)b * 2 * dh + r) * dhp + c] = from_f32<E>(v);
  else
    woc[((long long)b * dh + r - 2 * dh) * dhp + c] = from_f32<E>(v);
}

// Row r of the three masters of head b in the interleaved order: r < 2 d_h is row r/2 of W_in
// (r even) or W_gate (r odd); r >= 2 d_h is row r - 2 d_h of W_out.
__device__ __forceinline__ float* sw_row(float* w_in, float* w_gate, float* w_out, int b, int r,
                                         int dh) {
  const long long wb = (long long)b * dh * dh;
  return r < 2 * dh ? ((r & 1) ? w_gate : w_in) + wb + (long long)(r >> 1) * dh
                    : w_out + wb + (long long)(r - 2 * dh) * dh;
}

// Row norms of the initial fast weights (the renormalisation targets), n_ig [B][2 d_h] in the
// interleaved order and n_out [B][d_h].  One wave per row; grid (ceil(3 d_h / 4), B).
__global__ __launch_bounds__(256) void sw_row_norm_kernel(float* w_in, float* w_gate, float* w_out,
                                                          int dh, float* __restrict__ n_ig,
                                                          float* __restrict__ n_out) {
  const int b = blockIdx.y, r = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (r >= 3 * dh) return;
  const float* row = sw_row(w_in, w_gate, w_out, b, r, dh);
  float s = 0.0f;
  for (int c = lane; c < dh; c += 64) s += row[c] * row[c];
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off, 64);
  if (lane == 0) {
    if (r < 2 * dh)
      n_ig[(long long)b * 2 * dh + r] = sqrtf(s);
    else
      n_out[(long long)b * dh + r - 2 * dh] = sqrtf(s);
  }
}

// Renormalisation of the paper's optimiser: every master row is rescaled to its initial norm,
// scale = norm0 / sqrt(sum of the row's nseg segment sums of squares, fixed order), 1 for a row
// of norm 0; the MFMA copy of the row is written from the rescaled values.
// One wave per row; grid (ceil(3 d_h / 4), B).
template <typename E>
__global__ __launch_bounds__(256) void sw_renorm_kernel(
    float* w_in, float* w_gate, float* w_out, int dh, int dhp, int nseg,
    const float* __restrict__ ss_ig, const float* __restrict__ ss_out,
    const float* __restrict__ n_ig, const float* __restrict__ n_out, E* __restrict__ wig,
    E* __restrict__ woc) {
  const int b = blockIdx.y, r = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (r >= 3 * dh) return;
  float* row = sw_row(w_in, w_gate, w_out, b, r, dh);
  const bool ig = r < 2 * dh;
  const long long ri = ig ? (long long)b * 2 * dh + r : (long long)b * dh + r - 2 * dh;
  const float* ss = (ig ? ss_ig : ss_out) + ri * nseg;
  float s = 0.0f;
  for (int k = 0; k < nseg; ++k) s += ss[k];
  const float scale = s > 0.0f ? (ig ? n_ig : n_out)[ri] * rsqrtf(s) : 1.0f;
  E* cp = (ig ? wig : woc) + ri * dhp;
  for (int c = lane; c < dh; c += 64) {
    const float v = row[c] * scale;
    row[c] = v;
    cp[c] = from_f32<E>(v);
  }
}

}  // namespace
}  // namespace mone
