// Host helpers shared by the library's front ends (the configuration-form memory and the
// paper-form SwiGLU memory): error reporting, the grouped-GEMM launch helpers and per-stage
// timing with HIP events.
#pragma once

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <vector>

#include "../../include/mone_ttl.h"
#include "kernels.hpp"

// Message of the last failing call on this thread (defined once, in mone_ttl.hip).
extern thread_local char g_err[512];

namespace mone {
namespace {

inline int fail(int code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof g_err, fmt, ap);
  va_end(ap);
  return code;
}

inline int hip_fail(hipError_t e, const char* what) {
  return fail(MONE_EHIP, "%s: %s", what, hipGetErrorString(e));
}

constexpr size_t kAlign = 256;

inline size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }
inline long long round_up(long long v, long long a) { return (v + a - 1) / a * a; }
inline bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

// TILE_64x256_DEEP: 64 x 256 tiles with a 4-slot ring per operand (one workgroup per CU).
enum TileShape {
  TILE_256x256 = 0, TILE_128x128 = 1, TILE_64x256 = 2, TILE_256x64 = 3, TILE_64x256_DEEP = 4
};

constexpr int kNumCUs = 256;

// 64-row tiles for short row extents (short segments, query batches), with the deep ring when
// the launch has at most one tile per CU; 64-column tiles for short column extents (the token
// axis of the transposed backward); 256 x 256 when the grouped problem still has at least one
// such tile per CU; 128 x 128 otherwise.
inline TileShape pick_tile(int m, int n, int layers) {
  if (m <= 64)
    return (long long)((n + 255) / 256) * layers <= kNumCUs ? TILE_64x256_DEEP : TILE_64x256;
  if (n <= 64) return TILE_256x64;
  const long long big = (long long)((m + 255) / 256) * ((n + 255) / 256) * layers;
  if (m >= 256 && n >= 256 && big >= kNumCUs) return TILE_256x256;
  return TILE_128x128;
}

// Host description of one grouped problem before the tile shape fixes its tiling.
struct Spec {
  Part part[2];
  int nparts;
  int m_extent;   // rows that are computed (tiles cover them)
  int n;          // columns that are computed
  int m_store;    // rows stored by the epilogue; -1 = every computed tile row
  int n_store;    // columns stored by the epilogue; -1 = every computed tile column
};

inline Opnd opnd(const void* p, long long lstride, int ld, int rows) {
  Opnd o;
  o.p = p;
  o.lstride = lstride;
  o.ld = ld;
  o.rows = rows;
  return o;
}

template <typename E, int BM, int BN, int WAVES_M, int DEPTH = 0, class Epi>
hipError_t launch_tiled(const Spec* specs, int nspec, int layers, const Epi& epi,
                        hipStream_t s, int* tiles_per_layer) {
  GemmLaunch<Epi> G;
  std::memset(&G, 0, sizeof G);
  int begin = 0;
  for (int i = 0; i < nspec; ++i) {
    // the kernel reads as many operand parts as the epilogue type declares
    if (specs[i].nparts < 1 || specs[i].nparts > Epi::kParts) return hipErrorInvalidValue;
    Problem& P = G.prob[i];
    P.part[0] = specs[i].part[0];
    P.part[1] = specs[i].part[1];
    P.nparts = specs[i].nparts;
    P.tiles_m = (specs[i].m_extent + BM - 1) / BM;
    P.tiles_n = (specs[i].n + BN - 1) / BN;
    P.M = specs[i].m_store >= 0 ? specs[i].m_store : P.tiles_m * BM;
    P.N = specs[i].n_store >= 0 ? specs[i].n_store : P.tiles_n * BN;
    P.tile_begin = begin;
    begin += P.tiles_m * P.tiles_n * layers;
  }
  G.nprob = nspec;
  G.epi = epi;
  if (tiles_per_layer)  // tiles per layer of each problem
    for (int i = 0; i < nspec; ++i) tiles_per_layer[i] = G.prob[i].tiles_m * G.prob[i].tiles_n;
  if (begin == 0) return hipSuccess;
  gemm_nt_kernel<E, BM, BN, WAVES_M, Epi, DEPTH><<<dim3(begin), dim3(256), 0, s>>>(G);
  return hipGetLastError();
}

// Split-K of short-row launches with few tiles: the raw accumulators of at most one 64 x 256
// tile per CU.
constexpr size_t kSplitFloats = (size_t)kNumCUs * 64 * 256;

// Splits per tile for a single-problem 64 x 256 launch of `tiles` tiles (all layers) over
// `nsteps` K steps: doubled up to 4 while the launch keeps at most one workgroup per CU and
// every split at least 8 K steps.
inline int split_for(long long tiles, int nsteps) {
  int sp = 1;
  while (sp < 4 && tiles * sp * 2 <= kNumCUs && nsteps / (sp * 2) >= 8) sp *= 2;
  return sp;
}

// The two passes of a split-K launch (64 x 256 tiles, one problem): `split` workgroups per tile
// on the deep ring, each over a range of K steps, store their accumulators to `part`; then one
// workgroup per tile sums them in split order and runs the epilogue.
template <typename E, class Epi>
hipError_t launch_split(const Spec& spec, int layers, const Epi& epi, float* part, int split,
                        hipStream_t s, int* tiles_per_layer) {
  constexpr int BK = 8 * (16 / (int)sizeof(E));
  if (spec.nparts < 1 || spec.nparts > Epi::kParts) return hipErrorInvalidValue;
  GemmLaunch<Epi> G;
  std::memset(&G, 0, sizeof G);
  Problem& P = G.prob[0];
  P.part[0] = spec.part[0];
  P.part[1] = spec.part[1];
  P.nparts = spec.nparts;
  P.tiles_m = (spec.m_extent + 63) / 64;
  P.tiles_n = (spec.n + 255) / 256;
  P.M = spec.m_store >= 0 ? spec.m_store : P.tiles_m * 64;
  P.N = spec.n_store >= 0 ? spec.n_store : P.tiles_n * 256;
  P.tile_begin = 0;
  const int tiles = P.tiles_m * P.tiles_n * layers;
  if (tiles_per_layer) *tiles_per_layer = P.tiles_m * P.tiles_n;
  if (tiles == 0) return hipSuccess;
  if ((size_t)tiles * split * 64 * 256 > kSplitFloats) return hipErrorInvalidValue;
  const int nsteps = (spec.part[0].k_len + (spec.nparts > 1 ? spec.part[1].k_len : 0)) / BK;
  G.nprob = 1;
  G.epi = epi;
  G.part = part;
  G.split = split;
  G.split_steps = (nsteps + split - 1) / split;
  gemm_nt_kernel<E, 64, 256, 1, Epi, 4, kSplitPartial>
      <<<dim3(tiles * split), dim3(256), 0, s>>>(G);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  gemm_nt_kernel<E, 64, 256, 1, Epi, 0, kSplitReduce><<<dim3(tiles), dim3(256), 0, s>>>(G);
  return hipGetLastError();
}

// Tiles per layer of a problem of m x n under tile shape t (what launch_gemm will use).
inline int tiles_for(TileShape t, int m, int n) {
  const int bm = t == TILE_256x256 || t == TILE_256x64 ? 256 : t == TILE_128x128 ? 128 : 64;
  const int bn = t == TILE_256x64 ? 64 : t == TILE_128x128 ? 128 : 256;
  return ((m + bm - 1) / bm) * ((n + bn - 1) / bn);
}

// `split_part` (kSplitFloats floats, or null): single-problem deep-ring launches whose tiles
// leave CUs idle split their contraction (launch_split).
template <typename E, class Epi>
hipError_t launch_gemm(TileShape t, const Spec* specs, int nspec, int layers, const Epi& epi,
                       hipStream_t s, int* tiles_per_layer = nullptr,
                       float* split_part = nullptr) {
  if (t == TILE_64x256_DEEP && split_part && nspec == 1) {
    constexpr int BK = 8 * (16 / (int)sizeof(E));
    const long long tiles =
        (long long)((specs[0].m_extent + 63) / 64) * ((specs[0].n + 255) / 256) * layers;
    const int nsteps =
        (specs[0].part[0].k_len + (specs[0].nparts > 1 ? specs[0].part[1].k_len : 0)) / BK;
    const int sp = split_for(tiles, nsteps);
    if (sp > 1) return launch_split<E>(specs[0], layers, epi, split_part, sp, s, tiles_per_layer);
  }
  switch (t) {
    case TILE_256x256:
      return launch_tiled<E, 256, 256, 2>(specs, nspec, layers, epi, s, tiles_per_layer);
    case TILE_128x128:
      return launch_tiled<E, 128, 128, 2>(specs, nspec, layers, epi, s, tiles_per_layer);
    case TILE_256x64:
      return launch_tiled<E, 256, 64, 4>(specs, nspec, layers, epi, s, tiles_per_layer);
    case TILE_64x256_DEEP:
      return launch_tiled<E, 64, 256, 1, 4>(specs, nspec, layers, epi, s, tiles_per_layer);
    default:
      return launch_tiled<E, 64, 256, 1>(specs, nspec, layers, epi, s, tiles_per_layer);
  }
}

// Memory injection into attention (Eq. attn with Eq. std_attn): validation and the launch of
// memory_attention_kernel for L layers of K/V width d_kv; 16 query rows per workgroup.  With
// q = 0 nothing is launched.
inline int launch_attention(int L, int d_kv, bool act_bf16, const void* qh, const void* kh,
                            const void* vh, const void* kv_mem, int kv_dtype, int q, int n_heads,
                            int n_kv_heads, void* out, int out_dtype, hipStream_t s) {
  if (q < 0) return fail(MONE_EINVAL, "q = %d is negative", q);
  if ((kv_dtype != MONE_F32 && kv_dtype != MONE_BF16) ||
      (out_dtype != MONE_F32 && out_dtype != MONE_BF16))
    return fail(MONE_EINVAL, "kv_dtype and out_dtype must be MONE_F32 or MONE_BF16");
  if (n_heads < 1 || n_kv_heads < 1 || n_heads % n_kv_heads || d_kv % n_kv_heads)
    return fail(MONE_EINVAL, "heads: n_heads=%d must be a multiple of n_kv_heads=%d, which "
                "must divide d_kv=%d", n_heads, n_kv_heads, d_kv);
  const int dh = d_kv / n_kv_heads;
  if (dh > 256) return fail(MONE_EUNSUPPORTED, "head width %d above 256", dh);
  if (q == 0) return MONE_OK;
  if (!qh || !kh || !vh || !kv_mem || !out)
    return fail(MONE_EINVAL, "qh, kh, vh, kv_mem and out must be non-NULL");
  if (!aligned16(qh) || !aligned16(kh) || !aligned16(vh) || !aligned16(kv_mem) || !aligned16(out))
    return fail(MONE_EINVAL, "qh, kh, vh, kv_mem and out must be 16-byte aligned");
  const dim3 grid((q + 15) / 16, n_heads, L), block(256);
  const float scale = 1.0f / std::sqrt((float)dh);
  const bool kbf = kv_dtype == MONE_BF16, obf = out_dtype == MONE_BF16;
  // the eight dtype combinations of (activations, memory K/V, output), for heads of up to 128
  // columns or up to 256
#define MONE_ATTN_W(EA, EK, EO, DHM)                                                            \
  memory_attention_kernel<EA, EK, EO, DHM><<<grid, block, 0, s>>>(                             \
      reinterpret_cast<const EA*>(qh), reinterpret_cast<const EA*>(kh),                         \
      reinterpret_cast<const EA*>(vh), reinterpret_cast<const EK*>(kv_mem),                     \
      reinterpret_cast<EO*>(out), q, n_heads, n_kv_heads, dh, d_kv, scale)
#define MONE_ATTN(EA, EK, EO)                                                                   \
  do {                                                                                          \
    if (dh <= 128) MONE_ATTN_W(EA, EK, EO, 128);                                                \
    else MONE_ATTN_W(EA, EK, EO, 256);                                                          \
  } while (0)
  if (act_bf16) {
    if (kbf) { if (obf) MONE_ATTN(bf16_t, bf16_t, bf16_t); else MONE_ATTN(bf16_t, bf16_t, float); }
    else { if (obf) MONE_ATTN(bf16_t, float, bf16_t); else MONE_ATTN(bf16_t, float, float); }
  } else {
    if (kbf) { if (obf) MONE_ATTN(float, bf16_t, bf16_t); else MONE_ATTN(float, bf16_t, float); }
    else { if (obf) MONE_ATTN(float, float, bf16_t); else MONE_ATTN(float, float, float); }
  }
#undef MONE_ATTN
#undef MONE_ATTN_W
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_fail(e, "launch ATTN");
  return MONE_OK;
}

// Per-stage timing: each timed launch is bracketed by two HIP events on the launch's stream.
// Only the stages whose bit is set in `mask` are timed (stage i is bit i).
struct StageTimer {
  std::vector<hipEvent_t> ev;
  std::vector<int> stage;
  int cap = 0, used = 0;
  uint32_t mask = 0xffffffffu;

  bool on(int st) const { return used < cap && ((mask >> st) & 1u); }
  void begin(int st, hipStream_t s) {
    if (on(st)) (void)hipEventRecord(ev[2 * used], s);
  }
  void end(int st, hipStream_t s) {
    if (on(st)) {
      (void)hipEventRecord(ev[2 * used + 1], s);
      stage[used] = st;
      ++used;
    }
  }
  void destroy() {
    for (hipEvent_t e : ev) (void)hipEventDestroy(e);
    ev.clear();
    stage.clear();
    cap = used = 0;
  }
  int enable(int max_records, uint32_t stage_mask) {
    if (max_records < 0) return fail(MONE_EINVAL, "max_records is negative");
    destroy();
    mask = stage_mask;
    if (max_records == 0) return MONE_OK;
    ev.assign(2 * (size_t)max_records, nullptr);
    stage.assign((size_t)max_records, 0);
    for (size_t i = 0; i < ev.size(); ++i) {
      // timing only: no system-scope fence at each record (no cache writeback and
      // invalidation between the timed kernels, which would slow the work being timed)
      hipError_t e = hipEventCreateWithFlags(&ev[i], hipEventDisableSystemFence);
      if (e != hipSuccess) {
        ev.resize(i);
        destroy();
        return hip_fail(e, "hipEventCreate");
      }
    }
    cap = max_records;
    used = 0;
    return MONE_OK;
  }
  int report(double* ms_sum, int32_t* count, int n_stages) {
    for (int i = 0; i < n_stages; ++i) {
      ms_sum[i] = 0.0;
      count[i] = 0;
    }
    for (int i = 0; i < used; ++i) {
      hipError_t e = hipEventSynchronize(ev[2 * i + 1]);
      if (e != hipSuccess) return hip_fail(e, "hipEventSynchronize");
      float ms = 0.0f;
      if ((e = hipEventElapsedTime(&ms, ev[2 * i], ev[2 * i + 1])) != hipSuccess)
        return hip_fail(e, "hipEventElapsedTime");
      ms_sum[stage[i]] += ms;
      count[stage[i]] += 1;
    }
    used = 0;
    return MONE_OK;
  }
};

}  // namespace
}  // namespace mone
