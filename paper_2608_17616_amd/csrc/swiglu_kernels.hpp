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

// PROJ: tile of X [P_k ; P_v]^T = [raw keys | raw values] [tokens][2d], with the elementwise
// part of the preprocessing fused:
//   key columns    SiLU(s r + b) per channel  -> K' [L][Tp][d] (normalised and rotated by the
//                  KEYS kernel)
//   value columns  v = SiLU(r)                -> dY0 = -v / n [B][Tp][d_hp] (row pass) and
//                  dY^T = -eta v / n [B][d_h][Tp] (column pass, from v left in the staging)
// Tokens >= n are stored as 0.  d and d_h are multiples of 8, so a chunk never straddles the
// key/value boundary or a head.
// Several consecutive segments in one launch: GEMM row r is token t = r % seg_rows of segment
// s = r / seg_rows (seg_rows a multiple of 64, so a chunk of 8 rows stays in one segment);
// segment s's outputs go to its own copies (K' rows s * Tp + t of kpre_rows per layer; dY0,
// dY^T and the rates at strides dy_ss, dyt_ss, rate_ss).  One segment: seg_rows = Tp.
template <typename E>
struct EpiSwProj : EpiBase {
  static constexpr bool kCols = true;
  static constexpr bool kWriteback = true;
  E* kpre; E* dy; E* dyt;
  const float* kscale; const float* kshift;  // [L][d]
  const float* rate;                          // [L][Tp] per-token rates, or null (lr)
  float lr, inv_n;
  int d, dh, dhp, H, Tp, n;
  int seg_rows, kpre_rows;
  long long dy_ss, dyt_ss, rate_ss;
  __device__ __forceinline__ bool has_cols(int) const { return true; }
  __device__ __forceinline__ float rows8(int, int l, int row, int col, int, int, float (&v)[8],
                                         const float (&)[8]) const {
    const int sg = row / seg_rows, t = row - sg * seg_rows;
    float o[8];
    if (col < d) {
      const float* sc = kscale + (long long)l * d + col;
      const float* sh = kshift + (long long)l * d + col;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float u = sc[e] * v[e] + sh[e];
        o[e] = t < n ? u * sigmoidf_(u) : 0.0f;
      }
      store8(kpre + ((long long)l * kpre_rows + (long long)sg * Tp + t) * d + col, o);
    } else {
      const int c = col - d, e = c / dh, ch = c - e * dh;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const float sv = t < n ? v[i] * sigmoidf_(v[i]) : 0.0f;
        v[i] = sv;
        o[i] = -sv * inv_n;
      }
      store8(dy + sg * dy_ss + (((long long)l * H + e) * Tp + t) * dhp + ch, o);
    }
    return 0.0f;
  }
  __device__ __forceinline__ void cols8(int, int l, int row, int col, int, int,
                                        const float (&v)[8]) const {
    if (col < d) return;
    const int sg = row / seg_rows, t = row - sg * seg_rows;
    const int c = col - d, e = c / dh, ch = c - e * dh;
    const float* rt = rate ? rate + sg * rate_ss + (long long)l * Tp + t : nullptr;
    float o[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const float eta = rt ? rt[i] : lr;
      o[i] = -eta * v[i] * inv_n;
    }
    store8(dyt + sg * dyt_ss + (((long long)l * H + e) * dh + ch) * Tp + t, o);
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
// W - acc: fp32 read-modify-write of the masters, then the MFMA copies the next segment reads
// (W_ig with interleaved rows, and W_out; d_hp columns each).
// With the paper's optimiser (PAPER) the launch uses 64 x 256 tiles, so each workgroup holds
// whole rows (d_h <= 256): the row pass updates the momentum, mu = beta mu + acc, and leaves
// W - mu in the staging; after the workgroup has summed each row's squares, the scale pass
// rescales the row to its initial norm (norm0 / norm; 1 for a row of norm 0) and stores the
// master and its copy.
template <typename E, bool PAPER>
struct EpiSwUpd : EpiBase {
  static constexpr bool kPre = true;
  static constexpr int kAux = PAPER ? 16 : 8;
  static constexpr bool kWriteback = PAPER;
  static constexpr bool kRowScale = PAPER;
  float* w_in; float* w_gate; float* w_out;   // masters [B][d_h][d_h]
  float* m_in; float* m_gate; float* m_out;   // PAPER: momenta, same layout
  E* wig; E* woc;                             // copies [B][2 d_h][d_hp], [B][d_h][d_hp]
  const float* beta;                          // PAPER: [L]
  const float* n_ig; const float* n_out;      // PAPER: initial row norms [B][2 d_h], [B][d_h]
  long long lsw;                              // d_h * d_h
  int dh, dhp, H;
  __device__ __forceinline__ long long off(int pi, int b, int row, int col) const {
    return (long long)b * lsw + (long long)(pi ? row >> 1 : row) * dh + col;
  }
  __device__ __forceinline__ float* master(int pi, int row) const {
    return pi == 0 ? w_out : (row & 1) ? w_gate : w_in;
  }
  __device__ __forceinline__ float* mom(int pi, int row) const {
    return pi == 0 ? m_out : (row & 1) ? m_gate : m_in;
  }
  __device__ __forceinline__ E* copy(int pi, int b, int row, int col) const {
    return pi == 0 ? woc + ((long long)b * dh + row) * dhp + col
                   : wig + ((long long)b * 2 * dh + row) * dhp + col;
  }
  // SGD: split row chunks (columns col..col+3 and col+32..col+35), so the 16-byte master
  // accesses are contiguous across lanes (UPD 0.098 -> 0.095 ms at the paper's shape).  A
  // second half at or beyond d_h (the last 64-column segment of a row when d_h is not a
  // multiple of 64) is neither read nor stored; it enters the arithmetic as zeros, which the
  // accumulators also hold there.  The paper's optimiser keeps whole chunks: split, its launch
  // took 0.153 ms against 0.136.
  static constexpr bool kSplitCols = !PAPER;
  __device__ __forceinline__ bool split_cols(int) const { return !PAPER; }
  __device__ __forceinline__ void ld8(const float* p, float (&v)[8], bool hi) const {
    if constexpr (kSplitCols) load8_split(p, v, hi);
    else load8(p, v);
  }
  template <typename T>
  __device__ __forceinline__ void st8(T* p, const float (&v)[8], bool hi) const {
    if constexpr (kSplitCols) store8_split(p, v, hi);
    else store8(p, v);
  }
  __device__ __forceinline__ void pre8(int pi, int b, int row, int col, int, int N,
                                       float (&w)[kAux]) const {
    const long long o = off(pi, b, row, col);
    const bool hi = col + 32 < N;
    ld8(master(pi, row) + o, *reinterpret_cast<float(*)[8]>(&w[0]), hi);
    if constexpr (PAPER) ld8(mom(pi, row) + o, *reinterpret_cast<float(*)[8]>(&w[8]), hi);
  }
  __device__ __forceinline__ float rows8(int pi, int b, int row, int col, int, int N,
                                         float (&v)[8], const float (&w)[kAux]) const {
    const long long o = off(pi, b, row, col);
    const bool hi = col + 32 < N;
    if constexpr (PAPER) {
      const float bt = beta[b / H];
      float m[8], ss = 0.0f;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        m[e] = bt * w[8 + e] + v[e];
        v[e] = w[e] - m[e];
        ss += v[e] * v[e];
      }
      st8(mom(pi, row) + o, m, hi);
      return ss;
    } else {
      float nw[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) nw[e] = w[e] - v[e];
      st8(master(pi, row) + o, nw, hi);
      st8(copy(pi, b, row, col), nw, hi);
      return 0.0f;
    }
  }
  __device__ __forceinline__ void scale8(int pi, int b, int row, int col, int N, float ss,
                                         const float (&v)[8]) const {
    const float n0 = pi == 0 ? n_out[(long long)b * dh + row] : n_ig[(long long)b * 2 * dh + row];
    const float sc = ss > 0.0f ? n0 * rsqrtf(ss) : 1.0f;
    const bool hi = col + 32 < N;
    float nw[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) nw[e] = v[e] * sc;
    st8(master(pi, row) + off(pi, b, row, col), nw, hi);
    st8(copy(pi, b, row, col), nw, hi);
  }
};

// ---- the read (Eq. read, Eq. attn) --------------------------------------------------------

// Four consecutive elements (p 8-byte aligned for bf16, 16-byte for fp32).
__device__ __forceinline__ void store4(float* p, const float (&v)[4]) {
  *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
}
__device__ __forceinline__ void store4(bf16_t* p, const float (&v)[4]) {
  uint2 w;
  w.x = pack_bf16(v[0], v[1]);
  w.y = pack_bf16(v[2], v[3]);
  *reinterpret_cast<uint2*>(p) = w;
}

// QPROJ: tile of X_q P_q^T [q][d]: SiLU(s_q r + b_q) per channel -> Q' [L][Tp][d] (rows >= q
// stored as 0), which the KEYS kernel normalises and rotates like the keys.
template <typename E>
struct EpiSwQproj : EpiBase {
  E* qpre;
  const float* scale; const float* shift;  // [L][d]
  int d, Tp, q;
  __device__ __forceinline__ float rows8(int, int l, int row, int col, int, int, float (&v)[8],
                                         const float (&)[8]) const {
    const float* sc = scale + (long long)l * d + col;
    const float* sh = shift + (long long)l * d + col;
    float o[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float u = sc[e] * v[e] + sh[e];
      o[e] = row < q ? u * sigmoidf_(u) : 0.0f;
    }
    store8(qpre + ((long long)l * Tp + row) * d + col, o);
    return 0.0f;
  }
};

// QFWD: tile of [Z | G] = K_q W_ig^T [q][2 d_h] for one head; z_i and g_i are adjacent columns
// (W_ig interleaves the rows of W_in and W_gate), so a row chunk holds 4 hidden units:
// A = SiLU(z) g -> A [B][Tp][d_hp] (columns < d_h).
template <typename E>
struct EpiSwQfwd : EpiBase {
  E* a;
  long long ls;  // Tp * d_hp
  int dhp;
  __device__ __forceinline__ float rows8(int, int b, int row, int col, int, int, float (&v)[8],
                                         const float (&)[8]) const {
    float av[4];
#pragma unroll
    for (int p = 0; p < 4; ++p) av[p] = v[2 * p] * sigmoidf_(v[2 * p]) * v[2 * p + 1];
    store4(a + (long long)b * ls + (long long)row * dhp + col / 2, av);
    return 0.0f;
  }
};

// QOUT: tile of Y = A W_out [q][d_h] for one head, on 64 x 256 tiles so that a workgroup holds
// whole rows: the scale pass forms the memory token h = y / sqrt(mean(y^2) + 1e-6) * w_rms *
// gate -> H [L][Tp][d] at the head's columns.
template <typename E>
struct EpiSwQout : EpiBase {
  static constexpr bool kWriteback = true;
  static constexpr bool kRowScale = true;
  E* hout;
  const float* rms_w;  // [L][d]
  const float* gate;   // [L][Tp][H]
  int d, dh, H, Tp;
  __device__ __forceinline__ float rows8(int, int, int, int, int, int, float (&v)[8],
                                         const float (&)[8]) const {
    float ss = 0.0f;
#pragma unroll
    for (int e = 0; e < 8; ++e) ss += v[e] * v[e];
    return ss;
  }
  __device__ __forceinline__ void scale8(int, int b, int row, int col, int, float ss,
                                         const float (&v)[8]) const {
    const int l = b / H, e = b - l * H;
    const float r = rsqrtf(ss / (float)dh + 1e-6f);
    const float g = gate[((long long)l * Tp + row) * H + e];
    const float* w = rms_w + (long long)l * d + (long long)e * dh + col;
    float o[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) o[i] = v[i] * r * w[i] * g;
    store8(hout + ((long long)l * Tp + row) * d + (long long)e * dh + col, o);
  }
};

// QKV: tile of H [W_k ; W_v]^T [q][2 d_kv]: the memory tokens in the backbone's key/value space,
// stored into the caller's [L][q][2 d_kv] (fp32 or bf16), rows < q.
struct EpiSwKv : EpiBase {
  void* kv;
  long long ls;  // q * 2 d_kv
  int D;
  int bf16_out;
  __device__ __forceinline__ float rows8(int, int l, int row, int col, int M, int,
                                         float (&v)[8], const float (&)[8]) const {
    if (row >= M) return 0.0f;
    const long long o = (long long)l * ls + (long long)row * D + col;
    if (bf16_out)
      store8(reinterpret_cast<bf16_t*>(kv) + o, v);
    else
      store8(reinterpret_cast<float*>(kv) + o, v);
    return 0.0f;
  }
};

// Gates of the memory tokens: gate[l][j][e] = SiLU(a_{l,e} . x_j + c_{l,e}).  One wave per
// token (fixed-order reduction); grid (ceil(q / 4), L), 256 threads.
template <typename E>
__global__ __launch_bounds__(256) void sw_gate_kernel(const E* __restrict__ xq, int q, int d,
                                                      int H, const float* __restrict__ gw,
                                                      const float* __restrict__ gb, int Tp,
                                                      float* __restrict__ gate) {
  const int l = blockIdx.y, j = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (j >= q) return;
  const E* row = xq + ((long long)l * q + j) * d;
  for (int e = 0; e < H; ++e) {
    const float* w = gw + ((long long)l * H + e) * d;
    float s = 0.0f;
    for (int c = lane * 8; c < d; c += 64 * 8) {
      float x[8], u[8];
      load8(row + c, x);
#pragma unroll
      for (int i = 0; i < 8; ++i) u[i] = w[c + i];
#pragma unroll
      for (int i = 0; i < 8; ++i) s += x[i] * u[i];
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off, 64);
    if (lane == 0) {
      const float z = s + gb[(long long)l * H + e];
      gate[((long long)l * Tp + j) * H + e] = z * sigmoidf_(z);
    }
  }
}

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

// KEYS: one workgroup per (64 tokens, head e, layer l).  From the post-SiLU keys K' of the head,
// each token's keys are divided by max(norm, 1e-12) and rotated by RoPE at the token's position
// (the table holds cos and sin per position and channel pair); written as K [B][Tp][d_hp] (zero
// padding columns) and, through LDS, K^T [B][d_h][Tp].  Each half-wave (32 lanes) takes one
// token, lane i of it the 8 channels [8i, 8i + 8) as one 16-byte vector; the partner channels
// of vector i (RoPE pairs c and c + d_h/2) are vector i +- d_h/16, fetched by shuffle (d_h is a
// multiple of 16 and at most 256).  Tokens >= n hold zeros in K' and stay zero.
template <typename E>
__global__ __launch_bounds__(256) void sw_keys_kernel(const E* __restrict__ kpre, int d, int H,
                                                      int dh, int dhp, int Tp,
                                                      const float2* __restrict__ rope,
                                                      E* __restrict__ kh, E* __restrict__ kt,
                                                      int seg_rows, int kpre_rows,
                                                      long long kh_ss, long long kt_ss) {
  // [token][channel] in the output dtype (the values K^T stores), odd row stride in 32-bit words
  constexpr int TS = sizeof(E) == 2 ? 258 : 257;
  __shared__ E tile[64][TS];
  // several consecutive segments: block x covers tokens j0.. of segment sg (seg_rows a multiple
  // of 64); K' rows sg * Tp + j of kpre_rows per layer, and segment sg's copies of K and K^T
  const int gx = blockIdx.x * 64, sg = gx / seg_rows, j0 = gx - sg * seg_rows;
  const int e = blockIdx.y, l = blockIdx.z, b = l * H + e;
  const E* kl = kpre + ((long long)l * kpre_rows + (long long)sg * Tp) * d;
  kh += sg * kh_ss;
  kt += sg * kt_ss;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int li = lane & 31, hw = lane >> 5;  // vector index, half-wave
  const int nv = dh / 8, hv = dh / 16, half = dh / 2, c = 8 * li;
  const bool act = li < nv, lo = li < hv;
  const int src = (lane & 32) + (act ? (lo ? li + hv : li - hv) : li);
  // the 8 tokens of this half-wave: all loads issued first, then the arithmetic
  constexpr int IT = 8;
  float xs[IT][8];
#pragma unroll
  for (int it = 0; it < IT; ++it) {
    if (act) {
      load8(kl + (long long)(j0 + 2 * wave + hw + 8 * it) * d + (long long)e * dh + c, xs[it]);
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i) xs[it][i] = 0.0f;
    }
  }
#pragma unroll
  for (int it = 0; it < IT; ++it) {
    const int t = 2 * wave + hw + 8 * it, j = j0 + t;
    const float (&x)[8] = xs[it];
    float ss = 0.0f;
#pragma unroll
    for (int i = 0; i < 8; ++i) ss += x[i] * x[i];
#pragma unroll
    for (int off = 16; off > 0; off >>= 1) ss += __shfl_xor(ss, off, 64);  // within the half
    const float inv = 1.0f / fmaxf(sqrtf(ss), 1e-12f);
    float y[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) y[i] = __shfl(x[i], src, 64);
    float o[8] = {0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f};
    if (act) {
      const float4* cs = reinterpret_cast<const float4*>(rope + (long long)j * half +
                                                         (lo ? c : c - half));
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float4 r = cs[i];  // (cos, sin) of channel pairs 2i and 2i + 1 of the vector
        const float c0 = r.x, s0 = r.y, c1 = r.z, s1 = r.w;
        // c < d_h/2: x cos - partner sin; c >= d_h/2: partner sin + x cos
        o[2 * i] = (lo ? x[2 * i] * c0 - y[2 * i] * s0 : y[2 * i] * s0 + x[2 * i] * c0) * inv;
        o[2 * i + 1] = (lo ? x[2 * i + 1] * c1 - y[2 * i + 1] * s1
                           : y[2 * i + 1] * s1 + x[2 * i + 1] * c1) * inv;
      }
#pragma unroll
      for (int i = 0; i < 8; ++i) tile[t][c + i] = from_f32<E>(o[i]);
    }
    if (c < dhp) store8(kh + ((long long)b * Tp + j) * dhp + c, o);
  }
  __syncthreads();
  // K^T: 8 threads per channel row, 8 tokens (one vector) each
  for (int i = threadIdx.x; i < dh * 8; i += 256) {
    const int ch = i >> 3, t0 = (i & 7) * 8;
    float v[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) v[k] = to_f32(tile[t0 + k][ch]);
    store8(kt + ((long long)b * dh + ch) * Tp + j0 + t0, v);
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

}  // namespace
}  // namespace mone
