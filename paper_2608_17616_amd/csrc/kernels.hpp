// Device kernels of the MoNe test-time-learning path for gfx950 (CDNA4).
//
// One grouped GEMM kernel family does all the matrix work of a TTL step and of the read:
//   C[m][n] = sum_k A[m][k] * B[n][k]        ("NT": both operands K-contiguous in memory)
// with all L layers (and, for the update stage, two different problems) in one launch, and a
// fused epilogue per stage that applies the elementwise part of the step (SiLU and its
// derivative, the loss gradient and loss partials, the SiLU-gradient product, the SGD update).
//
// Every operand a GEMM reads is stored K-contiguous: the producers of intermediates write a
// transposed copy next to the plain one where a later stage contracts over tokens, so every
// tile load is a coalesced 16-byte-per-lane row load and every fragment read is one
// ds_read_b128.
//
// Tiles: BM x BN output per 256-thread workgroup (4 waves as 2 x 2), K step of 128 bytes per
// row (64 bf16 or 32 fp32).  A and B tiles are staged in LDS in double buffers with an XOR
// swizzle of the 16-byte column index by (row / 2) % 8, so both the row stores and the
// 32-row fragment reads are free of bank conflicts.  Global loads for tile k+1 are issued
// before the MFMAs of tile k.
//
// MFMA: bf16 uses v_mfma_f32_32x32x16_bf16 (one 16-byte fragment per lane = 8 k-values), fp32
// uses four v_mfma_f32_32x32x2_f32 on the four floats of the same 16-byte fragment.  Within a
// 32x32 block lane l supplies row (l % 32) of A and column (l % 32) of B; A and B take their
// k-values from the same fragment positions, so the k order inside an instruction does not
// matter.  Accumulator register r of lane l holds C[8*(r/4) + 4*(l/32) + r%4][l % 32].
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mone {

typedef uint16_t bf16_t;  // raw bf16 storage (same bits as torch.bfloat16)
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float to_f32(float v) { return v; }
__device__ __forceinline__ float to_f32(bf16_t v) { return __uint_as_float((uint32_t)v << 16); }

template <typename E> __device__ __forceinline__ E from_f32(float v);
template <> __device__ __forceinline__ float from_f32<float>(float v) { return v; }
// Round to nearest even (v_cvt_pk_bf16_f32 on gfx950).
template <> __device__ __forceinline__ bf16_t from_f32<bf16_t>(float v) {
  return __builtin_bit_cast(bf16_t, (__bf16)v);
}

// Four consecutive elements (16 bytes of fp32 or 8 bytes of bf16), p aligned accordingly.
__device__ __forceinline__ void store4(float* p, float a, float b, float c, float d) {
  *reinterpret_cast<float4*>(p) = make_float4(a, b, c, d);
}
__device__ __forceinline__ void store4(bf16_t* p, float a, float b, float c, float d) {
  u32x2 v;
  v[0] = (uint32_t)from_f32<bf16_t>(a) | ((uint32_t)from_f32<bf16_t>(b) << 16);
  v[1] = (uint32_t)from_f32<bf16_t>(c) | ((uint32_t)from_f32<bf16_t>(d) << 16);
  *reinterpret_cast<u32x2*>(p) = v;
}

__device__ __forceinline__ float sigmoidf_(float z) { return 1.0f / (1.0f + __expf(-z)); }

// ------------------------------------------------------------------------------------------
// Problem descriptors

struct Opnd {              // K-contiguous operand: element (r, k) of layer l at
  const void* p;           //   p + l*lstride + r*ld + k
  long long lstride;
  int ld;
  int rows;                // rows >= `rows` read as zero (ragged segments, short query batches)
};

struct Part {              // one K-range of the contraction: sum_k a(m, k) b(n, k), k < k_len
  Opnd a, b;
  int k_len;               // multiple of the tile K step
};

struct Problem {
  Part part[2];            // K-concatenated parts: the result is their sum
  int nparts;
  int M, N;                // output rows/cols that are stored (bounds of the epilogue)
  int tiles_m, tiles_n;    // tiles per layer
  int tile_begin;          // first workgroup of this problem in the launch
};

template <class Epi>
struct GemmLaunch {
  Problem prob[2];
  int nprob;
  Epi epi;
};

// ------------------------------------------------------------------------------------------
// The grouped GEMM kernel

typedef int32_t i32x4 __attribute__((ext_vector_type(4)));

// Buffer load of 4 bytes x size/4 per lane straight into LDS (no VGPR staging): lane l's data
// lands at M0 + 16*l for 16-byte loads; offsets at or beyond the descriptor's byte count read 0.
__device__ void raw_buffer_load_lds(i32x4 rsrc, __attribute__((address_space(3))) uint32_t* lds,
                                    int size, int voffset, int soffset, int offset,
                                    int aux) __asm("llvm.amdgcn.raw.buffer.load.lds");

// Raw buffer descriptor over [p, p + bytes): stride 0, range-checked by byte offset.
__device__ __forceinline__ i32x4 make_rsrc(const void* p, uint32_t bytes) {
  const uint64_t a = reinterpret_cast<uint64_t>(p);
  i32x4 r;
  r[0] = (int32_t)(uint32_t)(a & 0xffffffffu);
  r[1] = (int32_t)(uint32_t)((a >> 32) & 0xffffu);
  r[2] = (int32_t)bytes;
  r[3] = 0x00020000;
  return r;
}

// Workgroup -> tile.  Workgroups are dispatched round-robin over the 8 XCDs (bid % 8), each
// with its own L2: the bids of one XCD get one contiguous run of the problem's (layer, tile)
// sequence, so a layer's tiles share an L2.  Within a layer, tiles go in groups of GM tile
// rows, column-major inside a group, so concurrently running tiles reuse A and B panels.
__device__ __forceinline__ void map_tile(int local, int total, int tiles_m, int tiles_n,
                                         int* layer, int* tm, int* tn) {
  constexpr int NXCD = 8, GM = 4;
  const int full = total - total % NXCD;
  int v = local;
  if (local < full) v = (local % NXCD) * (full / NXCD) + local / NXCD;
  const int per_layer = tiles_m * tiles_n;
  *layer = v / per_layer;
  const int t = v - *layer * per_layer;
  const int group = t / (GM * tiles_n);
  const int first = group * GM;
  const int gm = tiles_m - first < GM ? tiles_m - first : GM;
  const int r = t - group * GM * tiles_n;
  *tm = first + r % gm;
  *tn = r / gm;
}

template <typename E, int BM, int BN, int WAVES_M, class Epi>
__global__ __launch_bounds__(256) void gemm_nt_kernel(GemmLaunch<Epi> G) {
  constexpr int VEC = 16 / (int)sizeof(E);   // elements per 16-byte vector
  constexpr int BK = 8 * VEC;                // K per tile: 8 vectors = 128 bytes per row
  constexpr int WAVES_N = 4 / WAVES_M;
  constexpr int WM = BM / WAVES_M, WN = BN / WAVES_N;  // wave tile
  constexpr int FM = WM / 32, FN = WN / 32;  // 32x32 MFMA blocks per wave
  constexpr int LA = BM / 32, LB = BN / 32;  // 1 KiB load instructions per wave per stage
  constexpr int STAGE = (BM + BN) * 128;     // bytes of one LDS stage (A rows, then B rows)
  static_assert(FM >= 1 && FN >= 1 && WAVES_M * WAVES_N == 4, "tile shape");
  __shared__ __attribute__((aligned(1024))) unsigned char smem[2 * STAGE];

  const int bid = blockIdx.x;
  const int pi = (G.nprob > 1 && bid >= G.prob[1].tile_begin) ? 1 : 0;
  const Problem& P = G.prob[pi];
  const int total = G.nprob > 1 && pi == 0 ? G.prob[1].tile_begin : (int)gridDim.x - P.tile_begin;
  int layer, tm, tn;
  map_tile(bid - P.tile_begin, total, P.tiles_m, P.tiles_n, &layer, &tm, &tn);
  const int t = tm * P.tiles_n + tn;
  const int m0 = tm * BM, n0 = tn * BN;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WAVES_N, wn = wave % WAVES_N;

  f32x16 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  const int nk0 = P.part[0].k_len / BK;
  const int nk = nk0 + (P.nparts > 1 ? P.part[1].k_len / BK : 0);

  // Per part: buffer descriptors over this layer's operand slices and each lane's byte offset
  // of its first load.  Lane l of load instruction i fills LDS row 8*(4*i + wave) + l/8, slot
  // l%8, and fetches the 16-byte vector (slot ^ swizzle(row)) of that row.
  i32x4 ra[2], rb[2];
  int oa[2], ob[2];
  const int lrow = lane >> 3, lslot = lane & 7;
#pragma unroll
  for (int pp = 0; pp < 2; ++pp) {
    const Part& Pt = P.part[pp < P.nparts ? pp : 0];
    const E* A = reinterpret_cast<const E*>(Pt.a.p) + (long long)layer * Pt.a.lstride;
    const E* B = reinterpret_cast<const E*>(Pt.b.p) + (long long)layer * Pt.b.lstride;
    ra[pp] = make_rsrc(A, (uint32_t)((long long)Pt.a.rows * Pt.a.ld * (int)sizeof(E)));
    rb[pp] = make_rsrc(B, (uint32_t)((long long)Pt.b.rows * Pt.b.ld * (int)sizeof(E)));
    const int r = 8 * wave + lrow;  // row of load 0; load i adds 32 rows (same swizzle)
    const int v = lslot ^ ((r >> 1) & 7);
    oa[pp] = ((m0 + r) * Pt.a.ld + v * VEC) * (int)sizeof(E);
    ob[pp] = ((n0 + r) * Pt.b.ld + v * VEC) * (int)sizeof(E);
  }

  auto issue_loads = [&](int kt, int stage) {
    const int pp = kt < nk0 ? 0 : 1;
    const int k0 = (kt - (pp ? nk0 : 0)) * BK * (int)sizeof(E);
    const Part& Pt = P.part[pp];
    unsigned char* sa = smem + stage * STAGE;
    unsigned char* sb = sa + BM * 128;
#pragma unroll
    for (int i = 0; i < LA; ++i) {
      auto* dst = reinterpret_cast<__attribute__((address_space(3))) uint32_t*>(
          reinterpret_cast<uintptr_t>(sa + (4 * i + wave) * 1024));
      raw_buffer_load_lds(ra[pp], dst, 16, oa[pp] + 32 * i * Pt.a.ld * (int)sizeof(E) + k0, 0,
                          0, 0);
    }
#pragma unroll
    for (int i = 0; i < LB; ++i) {
      auto* dst = reinterpret_cast<__attribute__((address_space(3))) uint32_t*>(
          reinterpret_cast<uintptr_t>(sb + (4 * i + wave) * 1024));
      raw_buffer_load_lds(rb[pp], dst, 16, ob[pp] + 32 * i * Pt.b.ld * (int)sizeof(E) + k0, 0,
                          0, 0);
    }
  };

  auto compute = [&](int stage) {
    const unsigned char* sa = smem + stage * STAGE;
    const unsigned char* sb = sa + BM * 128;
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      const int v = kk * 2 + (lane >> 5);
      u32x4 fa[FM], fb[FN];
#pragma unroll
      for (int i = 0; i < FM; ++i) {
        const int r = wm * WM + i * 32 + (lane & 31);
        fa[i] = *reinterpret_cast<const u32x4*>(sa + r * 128 + ((v ^ ((r >> 1) & 7)) << 4));
      }
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        const int r = wn * WN + j * 32 + (lane & 31);
        fb[j] = *reinterpret_cast<const u32x4*>(sb + r * 128 + ((v ^ ((r >> 1) & 7)) << 4));
      }
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) {
          if constexpr (sizeof(E) == 2) {
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                __builtin_bit_cast(bf16x8, fa[i]), __builtin_bit_cast(bf16x8, fb[j]),
                acc[i][j], 0, 0, 0);
          } else {
#pragma unroll
            for (int e = 0; e < 4; ++e)
              acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(
                  __uint_as_float(fa[i][e]), __uint_as_float(fb[j][e]), acc[i][j], 0, 0, 0);
          }
        }
    }
  };

  if (nk > 0) {
    issue_loads(0, 0);
    __builtin_amdgcn_s_waitcnt(0);  // all counters 0: this wave's loads have reached LDS
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
      if (kt + 1 < nk) issue_loads(kt + 1, (kt + 1) & 1);
      compute(kt & 1);
      __builtin_amdgcn_s_waitcnt(0);
      __syncthreads();
    }
  }

  float partial = 0.0f;
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const int col = n0 + wn * WN + j * 32 + (lane & 31);
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int row = m0 + wm * WM + i * 32 + g * 8 + (lane >> 5) * 4;
        partial += G.epi.apply(pi, layer, row, col, P.M, P.N, acc[i][j][4 * g + 0],
                               acc[i][j][4 * g + 1], acc[i][j][4 * g + 2], acc[i][j][4 * g + 3]);
      }
    }
  G.epi.finish(layer, t, wave, lane, partial);
}

// ------------------------------------------------------------------------------------------
// Epilogues.  apply() receives four vertically adjacent results C[row..row+3][col] (row is a
// multiple of 4) and returns a value summed per lane and handed to finish() (the loss
// partials; 0 elsewhere).  Intermediate buffers have Tp >= every stored row (a multiple of
// 256) rows, so tiles store whole 4-row groups; only caller-owned outputs check rows.

struct NoFinish {
  __device__ __forceinline__ void finish(int, int, int, int, float) const {}
};

// Forward 1: Z = X W1^T  ->  A = SiLU(Z) in [Tp][h] and [h][Tp], SiLU'(Z) in [Tp][h].
template <typename E>
struct EpiFwd1 : NoFinish {
  E* a; E* ds; E* at;
  long long ls;  // layer stride of a, ds and at (Tp*h)
  int h, Tp, n;
  __device__ __forceinline__ float apply(int, int layer, int row, int col, int, int N, float z0,
                                         float z1, float z2, float z3) const {
    if (col >= N) return 0.0f;
    const float z[4] = {z0, z1, z2, z3};
    float av[4], dv[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      if (row + i < n) {
        const float s = sigmoidf_(z[i]);
        av[i] = z[i] * s;
        dv[i] = s * (1.0f + z[i] * (1.0f - s));
      } else {
        av[i] = 0.0f;
        dv[i] = 0.0f;
      }
    }
    const long long base = (long long)layer * ls;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      a[base + (long long)(row + i) * h + col] = from_f32<E>(av[i]);
      ds[base + (long long)(row + i) * h + col] = from_f32<E>(dv[i]);
    }
    store4(at + base + (long long)col * Tp + row, av[0], av[1], av[2], av[3]);
    return 0.0f;
  }
};

// Forward 2 and loss gradient.  The GEMM computes -R = A (-W2)^T + X W_kv^T (K-concatenated,
// from the negated copy of W2), so R = Y - targets is the negated result.  Stores G = c R in
// [Tp][D] and [D][Tp]; sums R^2 per wave into the loss partials.
template <typename E>
struct EpiFwd2 {
  E* g; E* gt;
  float* loss_part;       // [L][parts_per_layer]
  long long ls;           // Tp*D
  int D, Tp, n, parts_per_layer;
  float c;
  __device__ __forceinline__ float apply(int, int layer, int row, int col, int, int N, float r0,
                                         float r1, float r2, float r3) const {
    if (col >= N) return 0.0f;
    float r[4] = {-r0, -r1, -r2, -r3};
#pragma unroll
    for (int i = 0; i < 4; ++i)
      if (row + i >= n) r[i] = 0.0f;
    const long long base = (long long)layer * ls;
#pragma unroll
    for (int i = 0; i < 4; ++i) g[base + (long long)(row + i) * D + col] = from_f32<E>(c * r[i]);
    store4(gt + base + (long long)col * Tp + row, c * r[0], c * r[1], c * r[2], c * r[3]);
    return r[0] * r[0] + r[1] * r[1] + r[2] * r[2] + r[3] * r[3];
  }
  __device__ __forceinline__ void finish(int layer, int tile, int wave, int lane, float s) const {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off, 64);
    if (lane == 0) loss_part[(long long)layer * parts_per_layer + tile * 4 + wave] = s;
  }
};

// Backward to the hidden layer: dA = G W2  ->  dZ = dA * SiLU'(Z), stored [h][Tp].
template <typename E>
struct EpiBwd : NoFinish {
  const E* ds; E* dzt;
  long long ls;  // Tp*h
  int h, Tp, n;
  __device__ __forceinline__ float apply(int, int layer, int row, int col, int, int N, float d0,
                                         float d1, float d2, float d3) const {
    if (col >= N) return 0.0f;
    const float dv[4] = {d0, d1, d2, d3};
    float dz[4];
    const long long base = (long long)layer * ls;
#pragma unroll
    for (int i = 0; i < 4; ++i)
      dz[i] = row + i < n ? dv[i] * to_f32(ds[base + (long long)(row + i) * h + col]) : 0.0f;
    store4(dzt + base + (long long)col * Tp + row, dz[0], dz[1], dz[2], dz[3]);
    return 0.0f;
  }
};

// SGD update of both matrices in one launch.  Problem 0: G^T A = dL/dW2 tile of W2 [D][h];
// problem 1: dZ^T X = dL/dW1 tile of W1 [h][d].  fp32 read-modify-write of the masters, then
// the activation-dtype copies the next segment's GEMMs read: -W2 [D][h] (forward 2 and the
// read) and W2^T [h][D] (backward) in both modes, W1 [h][d] in bf16 mode (fp32 mode reads the
// master).
template <typename E>
struct EpiUpdate : NoFinish {
  float* w2; E* w2n; E* w2t;
  float* w1; E* w1s;
  long long ls2, ls1;  // D*h, h*d
  int h, d, D;
  int w1_copy;         // write w1s (bf16 mode)
  float lr;
  __device__ __forceinline__ float apply(int pi, int layer, int row, int col, int M, int N,
                                         float g0, float g1, float g2, float g3) const {
    if (col >= N || row >= M) return 0.0f;
    const float gv[4] = {g0, g1, g2, g3};
    if (pi == 0) {
      const long long base = (long long)layer * ls2;
      float nw[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const long long idx = base + (long long)(row + i) * h + col;
        nw[i] = w2[idx] - lr * gv[i];
        w2[idx] = nw[i];
        w2n[idx] = from_f32<E>(-nw[i]);
      }
      store4(w2t + base + (long long)col * D + row, nw[0], nw[1], nw[2], nw[3]);
    } else {
      const long long base = (long long)layer * ls1;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const long long idx = base + (long long)(row + i) * d + col;
        const float w = w1[idx] - lr * gv[i];
        w1[idx] = w;
        if (w1_copy) w1s[idx] = from_f32<E>(w);
      }
    }
    return 0.0f;
  }
};

// Read, first layer: A_q = SiLU(X_q W1^T), stored [Tp][h] (rows >= q hold SiLU(0) = 0).
template <typename E>
struct EpiKv1 : NoFinish {
  E* a;
  long long ls;
  int h;
  __device__ __forceinline__ float apply(int, int layer, int row, int col, int, int N, float z0,
                                         float z1, float z2, float z3) const {
    if (col >= N) return 0.0f;
    const float z[4] = {z0, z1, z2, z3};
    const long long base = (long long)layer * ls;
#pragma unroll
    for (int i = 0; i < 4; ++i)
      a[base + (long long)(row + i) * h + col] = from_f32<E>(z[i] * sigmoidf_(z[i]));
    return 0.0f;
  }
};

// Read, second layer: the GEMM computes A_q (-W2)^T = -KV; stores KV into the caller's
// [L][q][D] output (fp32 or bf16).
struct EpiKv2 : NoFinish {
  void* kv;
  long long ls;  // q*D
  int D;
  int bf16_out;
  __device__ __forceinline__ float apply(int, int layer, int row, int col, int M, int N, float y0,
                                         float y1, float y2, float y3) const {
    if (col >= N) return 0.0f;
    const float y[4] = {-y0, -y1, -y2, -y3};
    const long long base = (long long)layer * ls + col;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      if (row + i >= M) break;
      const long long idx = base + (long long)(row + i) * D;
      if (bf16_out)
        reinterpret_cast<bf16_t*>(kv)[idx] = from_f32<bf16_t>(y[i]);
      else
        reinterpret_cast<float*>(kv)[idx] = y[i];
    }
    return 0.0f;
  }
};

// ------------------------------------------------------------------------------------------
// Data-movement helpers

// dst[l][c][r] = src[l][r][c] for r < R, 0 for R <= r < Rz; 64x64 tiles through LDS.
template <typename Ein, typename Eout>
__global__ __launch_bounds__(256) void transpose_kernel(const Ein* __restrict__ src,
                                                        long long src_ls, int src_ld, int R,
                                                        int C, Eout* __restrict__ dst,
                                                        long long dst_ls, int dst_ld, int Rz) {
  __shared__ float tile[64][65];
  const int c0 = blockIdx.x * 64, r0 = blockIdx.y * 64, l = blockIdx.z;
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  const Ein* s = src + (long long)l * src_ls;
  for (int r = ty; r < 64; r += 4) {
    const int gr = r0 + r, gc = c0 + tx;
    tile[r][tx] = (gr < R && gc < C) ? to_f32(s[(long long)gr * src_ld + gc]) : 0.0f;
  }
  __syncthreads();
  Eout* o = dst + (long long)l * dst_ls;
  for (int c = ty; c < 64; c += 4) {
    const int gc = c0 + c, gr = r0 + tx;
    if (gc < C && gr < Rz) o[(long long)gc * dst_ld + gr] = from_f32<Eout>(tile[tx][c]);
  }
}

// dst[i] = sign * src[i] in the destination dtype (fp32 -> bf16: nearest even).
template <typename Eout>
__global__ void convert_kernel(const float* __restrict__ src, Eout* __restrict__ dst, long long n,
                               float sign) {
  for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (long long)gridDim.x * blockDim.x)
    dst[i] = from_f32<Eout>(sign * src[i]);
}

// out[l] = scale * sum of the loss partials of layer l (fixed order: deterministic).
__global__ void loss_finalize_kernel(const float* __restrict__ part, int per_layer, int count,
                                     float scale, float* __restrict__ out) {
  const int l = blockIdx.x;
  __shared__ float red[256];
  float s = 0.0f;
  for (int i = threadIdx.x; i < count; i += blockDim.x) s += part[(long long)l * per_layer + i];
  red[threadIdx.x] = s;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) out[l] = red[0] * scale;
}

}  // namespace mone
