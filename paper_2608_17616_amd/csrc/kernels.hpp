// Device kernels of the MoNe test-time-learning path for gfx950 (CDNA4).
//
// One grouped GEMM kernel family does all the matrix work of a TTL step and of the read:
//   C[m][n] = sum_k A[m][k] * B[n][k]        ("NT": both operands K-contiguous in memory)
// with all L layers (and, for the update stage, two different problems) in one launch, and a
// fused epilogue per stage that applies the elementwise part of the step (SiLU and its
// derivative, the loss gradient and loss partials, the SiLU-gradient product, the SGD update).
//
// Every operand a GEMM reads is stored K-contiguous: where a later stage contracts over
// tokens, the producing epilogue also writes a transposed copy, so every tile load is a
// coalesced row load and every fragment read is one ds_read_b128.
//
// Main loop.  BM x BN output per 256-thread workgroup (4 waves), K step of 128 bytes per row
// (64 bf16 or 32 fp32).  Operand tiles go from memory straight into LDS (buffer_load ... lds,
// no register staging) into rings of K-step slots (A two steps ahead for square tiles, B one);
// the 16-byte column slot of row r is XOR-swizzled by (r / 2) % 8, which each lane applies by
// choosing its source address, so fragment reads of 32 consecutive rows are free of bank
// conflicts.  The loads of later K steps are spread over the MFMAs of the current one, and each
// wave reads its fragments one sub-step ahead of the MFMAs that use them.  Launches with at most
// one tile per CU use a deep ring instead (4 slots per operand, both 3 steps ahead), and may
// split each tile's K steps over several workgroups: a partial pass stores raw accumulators,
// and a reduce pass sums them in split order before the epilogue.
//
// MFMA: bf16 uses v_mfma_f32_32x32x16_bf16 (one 16-byte fragment per lane = 8 k-values), fp32
// uses four v_mfma_f32_32x32x2_f32 on the four floats of the same 16-byte fragment.  Within a
// 32x32 block lane l supplies row (l % 32) of A and column (l % 32) of B; A and B take their
// k-values from the same fragment positions, so the k order inside an instruction does not
// matter.  Accumulator register r of lane l holds C[8*(r/4) + 4*(l/32) + r%4][l % 32].
//
// Epilogue.  Each wave stages its own accumulators through a private LDS region, one 64 x 64
// sub-block at a time, then processes them in chunks of 8 consecutive elements: a row pass (8
// columns of one row: 16- or 32-byte vector accesses) and, where a transposed copy is stored, a
// column pass (8 rows of one column).  An epilogue may also take its rows in pairs (rows 2i and
// 2i + 1 of a sub-block reach the same lane), for results that combine two interleaved output
// rows, or, on 64 x 256 tiles, scale whole rows after a workgroup-wide sum of their squares.
// The fp32 read-modify-write epilogues take split row chunks (columns 4q..4q+3 and 32+4q..
// 32+4q+3 of a 64-column segment for lane q), so that each 16-byte fp32 access instruction
// covers whole lines across its lanes.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <utility>

namespace mone {

typedef uint16_t bf16_t;  // raw bf16 storage (same bits as torch.bfloat16)
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef int32_t i32x4 __attribute__((ext_vector_type(4)));

// Buffer load of size bytes per lane straight into LDS (no VGPR staging): lane l's data lands
// at M0 + 16*l for 16-byte loads; offsets at or beyond the descriptor's byte count read 0.
__device__ void raw_buffer_load_lds(i32x4 rsrc, __attribute__((address_space(3))) uint32_t* lds,
                                    int size, int voffset, int soffset, int offset,
                                    int aux) __asm("llvm.amdgcn.raw.buffer.load.lds");

// Internal linkage: every library source file that includes this header has its own copies.
namespace {

__device__ __forceinline__ float to_f32(float v) { return v; }
__device__ __forceinline__ float to_f32(bf16_t v) { return __uint_as_float((uint32_t)v << 16); }

template <typename E> __device__ __forceinline__ E from_f32(float v);
template <> __device__ __forceinline__ float from_f32<float>(float v) { return v; }
// Round to nearest even (v_cvt_pk_bf16_f32 on gfx950).
template <> __device__ __forceinline__ bf16_t from_f32<bf16_t>(float v) {
  return __builtin_bit_cast(bf16_t, (__bf16)v);
}

__device__ __forceinline__ uint32_t pack_bf16(float a, float b) {
  return (uint32_t)from_f32<bf16_t>(a) | ((uint32_t)from_f32<bf16_t>(b) << 16);
}

typedef float f32x4v __attribute__((ext_vector_type(4)));
// Eight consecutive elements; p is 16-byte aligned.  Stores and fp32 loads are non-temporal:
// epilogue outputs are read by a later kernel, and the fp32 masters are read once per step, so
// neither should displace the operand panels other tiles are streaming through L2.
__device__ __forceinline__ void store8(float* p, const float (&v)[8]) {
  f32x4v a, b;
  a[0] = v[0]; a[1] = v[1]; a[2] = v[2]; a[3] = v[3];
  b[0] = v[4]; b[1] = v[5]; b[2] = v[6]; b[3] = v[7];
  __builtin_nontemporal_store(a, reinterpret_cast<f32x4v*>(p));
  __builtin_nontemporal_store(b, reinterpret_cast<f32x4v*>(p) + 1);
}
__device__ __forceinline__ void store8(bf16_t* p, const float (&v)[8]) {
  u32x4 w;
  w[0] = pack_bf16(v[0], v[1]);
  w[1] = pack_bf16(v[2], v[3]);
  w[2] = pack_bf16(v[4], v[5]);
  w[3] = pack_bf16(v[6], v[7]);
  __builtin_nontemporal_store(w, reinterpret_cast<u32x4*>(p));
}
__device__ __forceinline__ void load8(const float* p, float (&v)[8]) {
  const f32x4v a = __builtin_nontemporal_load(reinterpret_cast<const f32x4v*>(p));
  const f32x4v b = __builtin_nontemporal_load(reinterpret_cast<const f32x4v*>(p) + 1);
  v[0] = a[0]; v[1] = a[1]; v[2] = a[2]; v[3] = a[3];
  v[4] = b[0]; v[5] = b[1]; v[6] = b[2]; v[7] = b[3];
}
__device__ __forceinline__ void load8(const bf16_t* p, float (&v)[8]) {
  const u32x4 w = *reinterpret_cast<const u32x4*>(p);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    v[2 * i] = __uint_as_float(w[i] << 16);
    v[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
  }
}

// Split row chunks.  Lane q (0..7) of the 8 lanes covering a 64-column row segment holds
// columns 4q..4q+3 (v[0..3]) and 32+4q..32+4q+3 (v[4..7]); p points at column 4q.  Each 16-byte
// fp32 access instruction then covers 128 contiguous bytes across the 8 lanes: a non-temporal
// store of two 16-byte halves per lane 32 bytes apart (the unsplit chunk) leaves every line
// half written by each instruction, and measured 2.1 TB/s on its own against 5.4 TB/s.
// hi: the second half lies inside the row (false where a row ends within the segment; the row
// length is then a multiple of 8, so both lanes of a pair below are inside or both outside).
__device__ __forceinline__ void load8_split(const float* p, float (&v)[8], bool hi = true) {
  const f32x4v a = __builtin_nontemporal_load(reinterpret_cast<const f32x4v*>(p));
  f32x4v b = {0.0f, 0.0f, 0.0f, 0.0f};
  if (hi) b = __builtin_nontemporal_load(reinterpret_cast<const f32x4v*>(p + 32));
  v[0] = a[0]; v[1] = a[1]; v[2] = a[2]; v[3] = a[3];
  v[4] = b[0]; v[5] = b[1]; v[6] = b[2]; v[7] = b[3];
}
__device__ __forceinline__ void store8_split(float* p, const float (&v)[8], bool hi = true) {
  f32x4v a, b;
  a[0] = v[0]; a[1] = v[1]; a[2] = v[2]; a[3] = v[3];
  b[0] = v[4]; b[1] = v[5]; b[2] = v[6]; b[3] = v[7];
  __builtin_nontemporal_store(a, reinterpret_cast<f32x4v*>(p));
  if (hi) __builtin_nontemporal_store(b, reinterpret_cast<f32x4v*>(p + 32));
}
// bf16: lanes 2m and 2m+1 exchange halves (a DPP move within each pair of lanes), then lane 2m
// stores columns 8m..8m+7 and lane 2m+1 columns 32+8m..32+8m+7 (if hi), 16 bytes each.  Both
// lanes of a pair must execute this together (they always share a row, hence its bounds checks).
__device__ __forceinline__ void store8_split(bf16_t* p, const float (&v)[8], bool hi = true) {
  const uint32_t a0 = pack_bf16(v[0], v[1]), a1 = pack_bf16(v[2], v[3]);
  const uint32_t b0 = pack_bf16(v[4], v[5]), b1 = pack_bf16(v[6], v[7]);
  const bool odd = (__lane_id() & 1) != 0;
  // the half the partner keeps: the even lane sends columns 32+, the odd lane columns 0..3
  constexpr int kSwapPairs = 0xB1;  // quad_perm [1, 0, 3, 2]
  const uint32_t r0 = (uint32_t)__builtin_amdgcn_mov_dpp((int)(odd ? a0 : b0), kSwapPairs, 0xF,
                                                         0xF, false);
  const uint32_t r1 = (uint32_t)__builtin_amdgcn_mov_dpp((int)(odd ? a1 : b1), kSwapPairs, 0xF,
                                                         0xF, false);
  u32x4 w;
  if (odd) { w[0] = r0; w[1] = r1; w[2] = b0; w[3] = b1; }
  else { w[0] = a0; w[1] = a1; w[2] = r0; w[3] = r1; }
  if (!odd || hi) __builtin_nontemporal_store(w, reinterpret_cast<u32x4*>(odd ? p + 28 : p));
}

// Logistic function with the hardware exponential and reciprocal (about 1 ulp each; an IEEE
// division would cost ten instructions per element in the epilogues).
__device__ __forceinline__ float sigmoidf_(float z) {
  return __builtin_amdgcn_rcpf(1.0f + __expf(-z));
}

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
  int M, N;                // output rows/cols the epilogue may store
  int tiles_m, tiles_n;    // tiles per layer
  int tile_begin;          // first workgroup of this problem in the launch
};

// Split-K passes of a single-problem launch (mode 0: the whole contraction, then the epilogue).
enum SplitMode { kSplitNone = 0, kSplitPartial = 1, kSplitReduce = 2 };

template <class Epi>
struct GemmLaunch {
  Problem prob[2];
  int nprob;
  Epi epi;
  // Split-K (kernels instantiated with MODE != kSplitNone): in the partial pass workgroup b
  // takes split b / tiles of tile b % tiles, runs its split_steps K steps and stores its raw
  // accumulators to part; in the reduce pass each tile sums its splits' accumulators in split
  // order and runs the epilogue.
  float* part;
  int split, split_steps;
};

// ------------------------------------------------------------------------------------------
// The grouped GEMM kernel


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

template <int BM, int BN, int DEPTH = 0>
struct TileCfg {
  // Main loop: A and B panels of 128-byte rows in separate LDS rings.  The 256 x 256 and
  // 128 x 128 tiles keep A two K steps ahead (3 slots) and B one step ahead (2 slots), which
  // fills the 160 KiB of LDS for one 256 x 256 workgroup per CU or two 128 x 128 ones.  A deep
  // ring (DEPTH slots for both operands, both DEPTH - 1 steps ahead) is for launches with at
  // most one workgroup per CU, whose K steps would otherwise each wait a full memory latency.
  static constexpr int NA = DEPTH > 0 ? DEPTH : BM == BN ? 3 : 2;
  static constexpr int NB = DEPTH > 0 ? DEPTH : 2;
  static constexpr int ASLOT = BM * 128, BSLOT = BN * 128;
  static constexpr int RING = NA * ASLOT + NB * BSLOT;
  static constexpr int EPI_BYTES = 4 * 64 * 64 * 4;  // per-wave 64 x 64 fp32 staging
  static constexpr int SMEM = RING > EPI_BYTES ? RING : EPI_BYTES;
};

// Spread NR LDS reads and NV buffer loads evenly over NM MFMAs in the scheduler's order:
// after MFMA i come the reads and loads whose share falls there.
template <int NM, int NR, int NV, int I>
__device__ __forceinline__ void interleave_step() {
  constexpr int r = (NR * (I + 1)) / NM - (NR * I) / NM;
  constexpr int v = (NV * (I + 1)) / NM - (NV * I) / NM;
  __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);                   // MFMA
  if constexpr (r > 0) __builtin_amdgcn_sched_group_barrier(0x100, r, 0);  // DS read
  if constexpr (v > 0) __builtin_amdgcn_sched_group_barrier(0x020, v, 0);  // VMEM read
}
template <int NM, int NR, int NV, int... I>
__device__ __forceinline__ void interleave_seq(std::integer_sequence<int, I...>) {
  (interleave_step<NM, NR, NV, I>(), ...);
}
template <int NM, int NR, int NV>
__device__ __forceinline__ void interleave() {
  interleave_seq<NM, NR, NV>(std::make_integer_sequence<int, NM>{});
}
// The LDS reads of the next sub-step's fragments (NRL of them) go first: four before the
// first MFMA, then one after each MFMA until none is left (measured better than issuing all
// of them at once or spreading them evenly); the NV buffer loads are spread evenly.
template <int NM, int NR, int NV, int I>
__device__ __forceinline__ void front_step() {
  constexpr int r = I < NR ? 1 : 0;
  constexpr int v = (NV * (I + 1)) / NM - (NV * I) / NM;
  __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);                   // MFMA
  if constexpr (r > 0) __builtin_amdgcn_sched_group_barrier(0x100, r, 0);  // DS read
  if constexpr (v > 0) __builtin_amdgcn_sched_group_barrier(0x020, v, 0);  // VMEM read
}
template <int NM, int NR, int NV, int... I>
__device__ __forceinline__ void front_seq(std::integer_sequence<int, I...>) {
  (front_step<NM, NR, NV, I>(), ...);
}
template <int NRL, int NM, int NV>
__device__ __forceinline__ void reads_then_interleave() {
  constexpr int lead = NRL < 4 ? NRL : 4;
  __builtin_amdgcn_sched_group_barrier(0x100, lead, 0);
  front_seq<NM, NRL - lead, NV>(std::make_integer_sequence<int, NM>{});
}

template <typename E, int BM, int BN, int WAVES_M, class Epi, int DEPTH = 0,
          int MODE = kSplitNone>
__global__ __launch_bounds__(256) void gemm_nt_kernel(GemmLaunch<Epi> G) {
  using TC = TileCfg<BM, BN, DEPTH>;
  constexpr int VEC = 16 / (int)sizeof(E);   // elements per 16-byte vector
  constexpr int BK = 8 * VEC;                // K per step: 8 vectors = 128 bytes per row
  constexpr int WAVES_N = 4 / WAVES_M;
  constexpr int WM = BM / WAVES_M, WN = BN / WAVES_N;  // wave tile
  constexpr int FM = WM / 32, FN = WN / 32;  // 32x32 MFMA blocks per wave
  constexpr int LA = BM / 32, LB = BN / 32;  // 1 KiB load instructions per wave per panel
  constexpr int NA = TC::NA, NB = TC::NB, ASLOT = TC::ASLOT, BSLOT = TC::BSLOT;
  constexpr int MPF = sizeof(E) == 2 ? 1 : 4;  // MFMA instructions per fragment pair
  constexpr int NM = FM * FN * MPF;            // MFMA instructions per sub-step
  static_assert(FM >= 1 && FN >= 1 && WAVES_M * WAVES_N == 4, "tile shape");
  __shared__ __attribute__((aligned(1024))) unsigned char smem[TC::SMEM];

  // Problem of this workgroup: problem 0's tiles come first.  (Alternating the two problems'
  // tiles across the launch was measured slower: each XCD's L2 then serves both working sets.)
  int bid = blockIdx.x, gx = (int)gridDim.x, split_i = 0;
  if constexpr (MODE == kSplitPartial) {  // single problem: gridDim.x = split * tiles
    gx /= G.split;
    split_i = bid / gx;
    bid -= split_i * gx;
  }
  const int first1 = G.nprob > 1 ? G.prob[1].tile_begin : gx;
  const int pi = bid >= first1 ? 1 : 0;
  const int local = bid - (pi ? first1 : 0);
  const int total = pi ? gx - first1 : first1;
  const Problem& P = G.prob[pi];
  int layer, tm, tn;
  map_tile(local, total, P.tiles_m, P.tiles_n, &layer, &tm, &tn);
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
  constexpr int NP = Epi::kParts;
  // K steps [kbeg, nk) of this workgroup; loads of steps at or past nk read zeros.
  int kbeg = 0, nk = nk0 + (NP > 1 && P.nparts > 1 ? P.part[1].k_len / BK : 0);
  if constexpr (MODE == kSplitPartial) {
    kbeg = split_i * G.split_steps;
    nk = nk < kbeg + G.split_steps ? nk : kbeg + G.split_steps;
  } else if constexpr (MODE == kSplitReduce) {
    nk = 0;
  }

  // Per part: buffer descriptors over this layer's operand slices, and each lane's byte offset
  // for each of its load instructions.  Lane l of load instruction i fills LDS row
  // 8*(4*i + wave) + l/8, 16-byte slot l%8, and fetches the vector (slot ^ swizzle(row)) of that
  // row; the swizzle does not depend on i.  The K position of a step goes into the
  // instruction's scalar offset, so the per-lane offsets stay fixed for the whole loop.
  const int wave_u = __builtin_amdgcn_readfirstlane(wave);  // uniform: LDS addresses in SGPRs
  i32x4 ra[NP], rb[NP];
  int vofa[NP][LA], vofb[NP][LB];
  const int lrow = lane >> 3, lslot = lane & 7;
#pragma unroll
  for (int pp = 0; pp < NP; ++pp) {
    const Part& Pt = P.part[pp < P.nparts ? pp : 0];
    const E* A = reinterpret_cast<const E*>(Pt.a.p) + (long long)layer * Pt.a.lstride;
    const E* B = reinterpret_cast<const E*>(Pt.b.p) + (long long)layer * Pt.b.lstride;
    ra[pp] = make_rsrc(A, (uint32_t)((long long)Pt.a.rows * Pt.a.ld * (int)sizeof(E)));
    rb[pp] = make_rsrc(B, (uint32_t)((long long)Pt.b.rows * Pt.b.ld * (int)sizeof(E)));
    const unsigned r = 8u * wave + lrow;
    const unsigned v = lslot ^ ((r >> 1) & 7u);
    const unsigned lda = (unsigned)Pt.a.ld * sizeof(E), ldb = (unsigned)Pt.b.ld * sizeof(E);
    // Rows past the operand's end give offsets at or beyond the descriptor's range (read as
    // zero); the range is below 2^31, so the unsigned offsets cannot wrap.
#pragma unroll
    for (int i = 0; i < LA; ++i) vofa[pp][i] = (int)((m0 + r + 32u * i) * lda + v * 16u);
#pragma unroll
    for (int i = 0; i < LB; ++i) vofb[pp][i] = (int)((n0 + r + 32u * i) * ldb + v * 16u);
  }
  const i32x4 rnone = make_rsrc(P.part[0].a.p, 0u);  // zero range: every load reads 0

  // Loads of K step kt (of part PP, whose steps start at kbase) into an LDS slot, instructions
  // [i0, i1) of the panel.  Steps at or past the end use the zero-range descriptor: they move
  // no data and fill an already consumed slot with zeros, so every step issues the same
  // instructions.
  constexpr int KB = BK * (int)sizeof(E);  // bytes of one K step of one row
  auto load_a = [&](auto part, int kt, int slot, int i0, int i1) {
    constexpr int PP = decltype(part)::value < NP ? decltype(part)::value : 0;
    const i32x4 rs = kt < nk ? ra[PP] : rnone;
    const int so = (kt - (PP ? nk0 : 0)) * KB;
    unsigned char* sa = smem + slot * ASLOT;
#pragma unroll
    for (int i = 0; i < LA; ++i) {
      if (i < i0 || i >= i1) continue;
      auto* dst = reinterpret_cast<__attribute__((address_space(3))) uint32_t*>(
          reinterpret_cast<uintptr_t>(sa + (4 * i + wave_u) * 1024));
      raw_buffer_load_lds(rs, dst, 16, vofa[PP][i], so, 0, 0);
    }
  };
  auto load_b = [&](auto part, int kt, int slot, int i0, int i1) {
    constexpr int PP = decltype(part)::value < NP ? decltype(part)::value : 0;
    const i32x4 rs = kt < nk ? rb[PP] : rnone;
    const int so = (kt - (PP ? nk0 : 0)) * KB;
    unsigned char* sb = smem + NA * ASLOT + slot * BSLOT;
#pragma unroll
    for (int i = 0; i < LB; ++i) {
      if (i < i0 || i >= i1) continue;
      auto* dst = reinterpret_cast<__attribute__((address_space(3))) uint32_t*>(
          reinterpret_cast<uintptr_t>(sb + (4 * i + wave_u) * 1024));
      raw_buffer_load_lds(rs, dst, 16, vofb[PP][i], so, 0, 0);
    }
  };
  using Part0 = std::integral_constant<int, 0>;
  using Part1 = std::integral_constant<int, 1>;

  // Fragments of one K sub-step (16 bf16 / 8 fp32 k-values per lane).
  auto read_frags = [&](int sla, int slb, int kk, u32x4 (&fa)[FM], u32x4 (&fb)[FN]) {
    const unsigned char* sa = smem + sla * ASLOT;
    const unsigned char* sb = smem + NA * ASLOT + slb * BSLOT;
    const int v = kk * 2 + (lane >> 5);
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
  };
  auto mfmas = [&](const u32x4 (&fa)[FM], const u32x4 (&fb)[FN]) {
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        if constexpr (sizeof(E) == 2) {
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
              __builtin_bit_cast(bf16x8, fa[i]), __builtin_bit_cast(bf16x8, fb[j]), acc[i][j],
              0, 0, 0);
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(
                __uint_as_float(fa[i][e]), __uint_as_float(fb[j][e]), acc[i][j], 0, 0, 0);
        }
      }
  };

  // Part 0's contribution times a per-column factor (kPart0Scale): applied once, after the
  // last K step of part 0 this workgroup computes.  Lane l's accumulators of MFMA block j all
  // lie in column n0 + wn*WN + 32j + l%32.
  auto part0_scale = [&] {
    if constexpr (Epi::kPart0Scale) {
      if (G.epi.has_part0_scale()) {
#pragma unroll
        for (int j = 0; j < FN; ++j) {
          const int col = n0 + wn * WN + 32 * j + (lane & 31);
          const float f = col < P.N ? G.epi.part0_scale(layer, col) : 1.0f;
#pragma unroll
          for (int i = 0; i < FM; ++i)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] *= f;
        }
      }
    }
  };

  // Pipeline.  K step kt reads A slot kt % NA and B slot kt % NB in four sub-steps.  The
  // fragments of each sub-step are read while the MFMAs of the previous one run: sub-step 0 of
  // step kt+1 is read right after the synchronisation that ends step kt, and sub-step 3 of
  // step kt is multiplied after it.  With an A ring of 3 (A two steps ahead, B one), each of
  // the four MFMA blocks between two synchronisations carries a quarter of the next loads:
  // the second half of B's step kt+1, both halves of A's step kt+2, and (after the
  // synchronisation, into the B slot step kt has just released) the first half of B's step
  // kt+2.  With an A ring of 2, B's and A's step kt+1 go with sub-steps 0 and 1.  Before the
  // synchronisation each wave waits until its loads of step kt+1 have landed (A loads of step
  // kt+2 may stay in flight) and its LDS reads of step kt are done; the workgroup then
  // synchronises, so step kt+1 is complete in LDS and no wave reads the slots of step kt any
  // more (later loads may overwrite them).
  constexpr int VMC = NA > 2 ? LA : 0;  // loads allowed in flight at the synchronisation
  constexpr int WAIT_STEP = (VMC & 15) | ((VMC >> 4) << 14) | (7 << 4);
  if constexpr (DEPTH > 0) {
    // Deep ring: step kt reads slot kt % DEPTH; during its first three sub-steps each wave
    // loads step kt + DEPTH - 1 into the slot of step kt - 1, which the synchronisation ending
    // step kt - 1 released.  Before the synchronisation that ends step kt each wave waits until
    // its loads of step kt + 1 have landed; those of the DEPTH - 2 later steps stay in flight.
    static_assert(DEPTH >= 3 && NA == DEPTH && NB == DEPTH, "deep ring");
    constexpr int VMD = (DEPTH - 2) * (LA + LB);
    static_assert(VMD < 64, "vmcnt range");
    constexpr int WAIT_D = (VMD & 15) | ((VMD >> 4) << 14) | (7 << 4);
    if (nk > kbeg) {
      u32x4 fa0[FM], fb0[FN], fa1[FM], fb1[FN];
      // Prologue: steps kbeg .. kbeg + DEPTH - 2 into slots 0 .. DEPTH - 2 (the part of each
      // step chosen at run time here only).
#pragma unroll
      for (int j = 0; j < DEPTH - 1; ++j) {
        const int kj = kbeg + j;
        if (kj < nk0) { load_a(Part0{}, kj, j, 0, LA); load_b(Part0{}, kj, j, 0, LB); }
        else { load_a(Part1{}, kj, j, 0, LA); load_b(Part1{}, kj, j, 0, LB); }
      }
      __builtin_amdgcn_s_waitcnt(WAIT_D);
      asm volatile("" ::: "memory");
      __builtin_amdgcn_s_barrier();
      asm volatile("" ::: "memory");
      int sl = 0;
      read_frags(sl, sl, 0, fa0, fb0);
      auto dstep = [&](int kt, auto pl) {
        const int sl_load = sl == 0 ? DEPTH - 1 : sl - 1;  // slot of step kt - 1: free
        const int kl = kt + DEPTH - 1;
        constexpr int NF = FM + FN;
        read_frags(sl, sl, 1, fa1, fb1);
        load_b(pl, kl, sl_load, 0, LB / 2);
        mfmas(fa0, fb0);
        reads_then_interleave<NF, NM, LB / 2>();
        read_frags(sl, sl, 2, fa0, fb0);
        load_b(pl, kl, sl_load, LB / 2, LB);
        mfmas(fa1, fb1);
        reads_then_interleave<NF, NM, LB - LB / 2>();
        read_frags(sl, sl, 3, fa1, fb1);
        load_a(pl, kl, sl_load, 0, LA);
        mfmas(fa0, fb0);
        reads_then_interleave<NF, NM, LA>();
        __builtin_amdgcn_s_waitcnt(WAIT_D);
        asm volatile("" ::: "memory");
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
        sl = sl + 1 == DEPTH ? 0 : sl + 1;
        read_frags(sl, sl, 0, fa0, fb0);  // after the last step: a consumed slot, never used
        mfmas(fa1, fb1);
        reads_then_interleave<NF, NM, 0>();
      };
      if constexpr (NP == 1) {
        for (int kt = kbeg; kt < nk; ++kt) dstep(kt, Part0{});
      } else {
        // both operands switch part when the loaded step reaches nk0; part 0's computed steps
        // end at c
        const int sw = nk0 - (DEPTH - 1);
        const int e1 = sw < kbeg ? kbeg : (sw > nk ? nk : sw);
        const int c = nk0 < kbeg ? kbeg : (nk0 > nk ? nk : nk0);
        int kt = kbeg;
        for (; kt < e1; ++kt) dstep(kt, Part0{});
        if constexpr (Epi::kPart0Scale) {
          for (; kt < c; ++kt) dstep(kt, Part1{});
          if (kbeg < c) part0_scale();
        }
        for (; kt < nk; ++kt) dstep(kt, Part1{});
      }
      __builtin_amdgcn_s_waitcnt(0);  // the last (out-of-range) loads have retired
      __syncthreads();                // the epilogue reuses the LDS of the rings
    }
  } else if (nk > 0) {
    u32x4 fa0[FM], fb0[FN], fa1[FM], fb1[FN];
    // Prologue: step 0 first, then (ring of 3) A's step 1 and the first half of B's step 1,
    // which may still be in flight when step 0 starts.
    if (nk0 > 0) { load_a(Part0{}, 0, 0, 0, LA); load_b(Part0{}, 0, 0, 0, LB); }
    else { load_a(Part1{}, 0, 0, 0, LA); load_b(Part1{}, 0, 0, 0, LB); }
    if constexpr (NA > 2) {
      if (nk0 > 1) { load_a(Part0{}, 1, 1, 0, LA); load_b(Part0{}, 1, 1, 0, LB / 2); }
      else { load_a(Part1{}, 1, 1, 0, LA); load_b(Part1{}, 1, 1, 0, LB / 2); }
    }
    constexpr int VPRO = NA > 2 ? LA + LB / 2 : 0;  // prologue loads allowed in flight
    __builtin_amdgcn_s_waitcnt((VPRO & 15) | ((VPRO >> 4) << 14) | (7 << 4));
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
    int sa = 0, sb = 0;
    read_frags(sa, sb, 0, fa0, fb0);
    auto step = [&](int kt, auto pa, auto pb) {
      const int sa_next = sa + 1 == NA ? 0 : sa + 1;
      const int sa_load = sa == 0 ? NA - 1 : sa - 1;  // slot of step kt-1: free
      const int sb_next = sb ^ 1;
      constexpr int NF = FM + FN;  // LDS reads per sub-step
      read_frags(sa, sb, 1, fa1, fb1);
      if constexpr (NA > 2) {
        load_b(pb, kt + 1, sb_next, LB / 2, LB);
        mfmas(fa0, fb0);
        reads_then_interleave<NF, NM, LB - LB / 2>();
        read_frags(sa, sb, 2, fa0, fb0);
        load_a(pa, kt + NA - 1, sa_load, 0, LA / 2);
        mfmas(fa1, fb1);
        reads_then_interleave<NF, NM, LA / 2>();
        read_frags(sa, sb, 3, fa1, fb1);
        load_a(pa, kt + NA - 1, sa_load, LA / 2, LA);
        mfmas(fa0, fb0);
        reads_then_interleave<NF, NM, LA - LA / 2>();
      } else {
        load_b(pb, kt + 1, sb_next, 0, LB);
        mfmas(fa0, fb0);
        reads_then_interleave<NF, NM, LB>();
        read_frags(sa, sb, 2, fa0, fb0);
        load_a(pa, kt + NA - 1, sa_load, 0, LA);
        mfmas(fa1, fb1);
        reads_then_interleave<NF, NM, LA>();
        read_frags(sa, sb, 3, fa1, fb1);
        mfmas(fa0, fb0);
        reads_then_interleave<NF, NM, 0>();
      }
      // Explicit wait, then a bare barrier: a fenced barrier would also wait for the A loads
      // that may stay in flight.  The empty asm statements keep the compiler from moving LDS
      // accesses across the barrier.
      __builtin_amdgcn_s_waitcnt(WAIT_STEP);
      asm volatile("" ::: "memory");
      __builtin_amdgcn_s_barrier();
      asm volatile("" ::: "memory");
      const int sb_free = sb;  // B slot of step kt: read completely, free for step kt+2
      sa = sa_next;
      sb = sb_next;
      read_frags(sa, sb, 0, fa0, fb0);  // after the last step: a consumed slot, never used
      if constexpr (NA > 2) load_b(pa, kt + 2, sb_free, 0, LB / 2);  // step kt+2: A's part
      mfmas(fa1, fb1);
      reads_then_interleave<FM + FN, NM, (NA > 2 ? LB / 2 : 0)>();
    };
    if constexpr (NP == 1) {
      for (int kt = 0; kt < nk; ++kt) step(kt, Part0{}, Part0{});
    } else {
      // The loads' operand part changes at step nk0; running the steps in three ranges keeps
      // the part a compile-time choice (no per-step selects of offsets).
      const int e1 = nk0 - (NA - 1) < 0 ? 0 : (nk0 - (NA - 1) > nk ? nk : nk0 - (NA - 1));
      const int e2 = nk0 - 1 < e1 ? e1 : (nk0 - 1 > nk ? nk : nk0 - 1);
      const int c = nk0 < e2 ? e2 : (nk0 > nk ? nk : nk0);  // part 0's computed steps end
      int kt = 0;
      for (; kt < e1; ++kt) step(kt, Part0{}, Part0{});  // A and B loads in part 0
      for (; kt < e2; ++kt) step(kt, Part1{}, Part0{});  // A loads reach part 1 first
      if constexpr (Epi::kPart0Scale) {
        for (; kt < c; ++kt) step(kt, Part1{}, Part1{});
        if (c > 0) part0_scale();
      }
      for (; kt < nk; ++kt) step(kt, Part1{}, Part1{});
    }
    __builtin_amdgcn_s_waitcnt(0);  // the last (out-of-range) loads have retired
    __syncthreads();                // the epilogue reuses the LDS of the rings
  }

  // Split-K: accumulators in their register layout, lane-contiguous, per (split, tile, wave).
  if constexpr (MODE != kSplitNone) {
    constexpr int NACC = FM * FN * 16;
    const long long tile_off = ((long long)local * 4 + wave) * NACC * 64 + lane;
    const long long split_stride = (long long)total * 4 * NACC * 64;
    if constexpr (MODE == kSplitPartial) {
      float* dst = G.part + split_i * split_stride + tile_off;
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
          for (int r = 0; r < 16; ++r)
            __builtin_nontemporal_store(acc[i][j][r], dst + ((i * FN + j) * 16 + r) * 64);
      return;
    }
    for (int sp = 0; sp < G.split; ++sp) {  // reduce: splits summed in order
      const float* src = G.part + sp * split_stride + tile_off;
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
          for (int r = 0; r < 16; ++r)
            acc[i][j][r] += __builtin_nontemporal_load(src + ((i * FN + j) * 16 + r) * 64);
    }
  }

  // ---- epilogue: each wave stages its own accumulators through LDS, 64 x 64 at a time
  // A wave's tile is processed in 64 x 64 sub-blocks (2 x 2 MFMA blocks) in a private 16 KiB
  // LDS region, so the epilogue needs no workgroup synchronisation.  Per sub-block: stage the
  // accumulators; row pass: each lane takes row chunks (8 consecutive columns of one row;
  // 8 lanes cover a 64-column row segment); column pass, if the epilogue has one: column
  // chunks (8 consecutive rows of one column; 8 lanes cover the 64 rows of a column).  The
  // memory reads an epilogue needs per row chunk (pre8: the fp32 master, SiLU') are issued one
  // sub-block ahead (after the staging of the current one, or with kPreLate after its row
  // pass), the first before the first staging; 16-bit inputs (kPackAll) all at once.  Staging
  // layout: row r, column c at
  // r*64 + (c ^ sw(r)) with sw(r) = ((r ^ r/8) & 7) * 4, which keeps 4-column groups intact
  // (16-byte reads) and spreads the 8 rows of a column chunk over distinct banks.
  constexpr int SB = 64;                        // sub-block edge
  constexpr int NSM = WM / SB, NSN = WN / SB;   // sub-blocks per wave
  constexpr int NSB = NSM * NSN;
  constexpr int CPL = SB * SB / 8 / 64;         // row (and column) chunks per lane: 8
  static_assert(WM % SB == 0 && WN % SB == 0, "wave tile");
  float* stw = reinterpret_cast<float*>(smem) + wave * (SB * SB);
  // kRowScale: per-wave partial sums of squares of the tile's rows, after the 4 staging areas
  float* rss = reinterpret_cast<float*>(smem) + 4 * SB * SB;
  static_assert(!Epi::kRowScale || (NSB == 1 && WAVES_M == 1 &&
                                    TC::SMEM >= (4 * SB * SB + 4 * SB) * 4),
                "row scale: one 64 x 64 sub-block per wave, the 4 waves side by side");
  auto sidx = [](int r, int c) { return r * SB + (c ^ (((r ^ (r >> 3)) & 7) << 2)); };
  auto wave_sync = [] {  // this wave's LDS writes are visible to all its lanes
    __builtin_amdgcn_s_waitcnt((63 & 15) | ((63 >> 4) << 14) | (7 << 4));  // lgkmcnt(0)
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  };
  float partial = 0.0f;
  constexpr int NAUX = Epi::kAux;
  // Row chunks per lane: 8, or 4 pairs of rows (2i, 2i + 1) when the epilogue pairs rows.
  constexpr int RS = Epi::kPairRows ? 2 : 1;
  constexpr int NCH = CPL / RS;
  static_assert(!Epi::kPairRows || (!Epi::kRowNorm && !Epi::kCols && !Epi::kWriteback &&
                                     !Epi::kRowScale),
                "paired rows: row pass only");
  static_assert(!Epi::kRowScale || (Epi::kWriteback && !Epi::kRowNorm && !Epi::kCols),
                "row scale: row pass with write-back, then the scale pass");
  static_assert(!Epi::kSplitCols || !Epi::kPairRows, "split row chunks: no paired rows");
  float aux[2][NCH][NAUX];
  const int rl = lane >> 3, ql = lane & 7;      // row-chunk lane coordinates
  // Split row chunks (split_cols(pi)): lane ql's chunk is columns 4ql..4ql+3 and
  // 32+4ql..32+4ql+3 of its 64-column row segment, passed as the chunk's first column.  The
  // problem's N is then a multiple of 8, the chunk is handled when its first half is inside N,
  // and the epilogue masks a second half at or beyond N.
  const bool split = Epi::kSplitCols && G.epi.split_cols(pi);
  const int cq = split ? 4 * ql : 8 * ql;        // first column of this lane's chunks
  const int cq2 = split ? 4 * ql + 32 : 8 * ql + 4;  // first column of their second half
  // staging halves in the other order on odd rows (256 x 256 tiles; measured slower with the
  // two workgroups per CU of 128 x 128 tiles)
  const bool sflip = BM == 256 && BN == 256 && split && (rl & 1);
  auto issue_pre = [&](int sb, float (&ax)[NCH][NAUX]) {
    const int grow = m0 + wm * WM + (sb / NSN) * SB, gcol = n0 + wn * WN + (sb % NSN) * SB;
#pragma unroll
    for (int b = 0; b < NCH; ++b) {
      const int row = grow + RS * (rl + 8 * b), col = gcol + cq;
      if (row + RS - 1 < P.M && col < P.N) G.epi.pre8(pi, layer, row, col, P.M, P.N, ax[b]);
    }
  };
  // packed problems: sub-block q's chunk b in dwords 4(q&1)..4(q&1)+3 of aux[q>>1][b]
  const bool pack_all = Epi::kPackAll && G.epi.pack_all(pi);
  static_assert(!Epi::kPackAll || (NSB <= 4 && NAUX == 8), "packed aux: 4 sub-blocks");
  auto issue_pre_packed = [&](int q) {
    const int grow = m0 + wm * WM + (q / NSN) * SB, gcol = n0 + wn * WN + (q % NSN) * SB;
#pragma unroll
    for (int b = 0; b < NCH; ++b) {
      const int row = grow + RS * (rl + 8 * b), col = gcol + cq;
      float (&w)[4] = *reinterpret_cast<float(*)[4]>(&aux[q >> 1][b][4 * (q & 1)]);
      if (row + RS - 1 < P.M && col < P.N) G.epi.pre4p(pi, layer, row, col, w);
    }
  };
  if constexpr (Epi::kPre) {
    if constexpr (Epi::kPackAll) {
      if (pack_all) {
#pragma unroll
        for (int q = 0; q < NSB; ++q) issue_pre_packed(q);
      } else {
        issue_pre(0, aux[0]);
      }
    } else {
      issue_pre(0, aux[0]);
    }
  }
#pragma unroll
  for (int sb = 0; sb < NSB; ++sb) {
    const int sm = sb / NSN, sn = sb % NSN;
    const int grow = m0 + wm * WM + sm * SB, gcol = n0 + wn * WN + sn * SB;
    if (sb > 0) wave_sync();  // the previous sub-block's reads are done
#pragma unroll
    for (int ii = 0; ii < 2; ++ii)
#pragma unroll
      for (int jj = 0; jj < 2; ++jj)
#pragma unroll
        for (int g = 0; g < 4; ++g)
#pragma unroll
          for (int e = 0; e < 4; ++e)
            stw[sidx(ii * 32 + g * 8 + (lane >> 5) * 4 + e, jj * 32 + (lane & 31))] =
                acc[2 * sm + ii][2 * sn + jj][4 * g + e];
    wave_sync();
    if constexpr (Epi::kPre && !Epi::kPreLate) {
      if (sb + 1 < NSB && !pack_all) issue_pre(sb + 1, aux[(sb + 1) & 1]);
    }
#pragma unroll
    for (int b = 0; b < NCH; ++b) {
      const int r = RS * (rl + 8 * b), c = cq;
      float* s0 = stw + sidx(r, c);
      float* s1 = stw + sidx(r, cq2);
      // Split chunks put each half of a row's 8 lanes on 32 of the staging's banks, the same
      // 32 for every row: with sflip, odd rows access their halves in the other order, so that
      // each 16-byte access instruction of two adjacent rows covers all banks (as unsplit
      // chunks do).
      float* sa = sflip ? s1 : s0;
      float* sb2 = sflip ? s0 : s1;
      float v[8];
      const float4 xa = *reinterpret_cast<const float4*>(sa);
      const float4 xb = *reinterpret_cast<const float4*>(sb2);
      v[0] = sflip ? xb.x : xa.x; v[1] = sflip ? xb.y : xa.y;
      v[2] = sflip ? xb.z : xa.z; v[3] = sflip ? xb.w : xa.w;
      v[4] = sflip ? xa.x : xb.x; v[5] = sflip ? xa.y : xb.y;
      v[6] = sflip ? xa.z : xb.z; v[7] = sflip ? xa.w : xb.w;
      const bool ok = grow + r + RS - 1 < P.M && gcol + c < P.N;
      float val = 0.0f;
      if constexpr (Epi::kPairRows) {
        // the partner row r + 1 (r is even: sub-blocks start at even rows)
        const float4 y0 = *reinterpret_cast<const float4*>(stw + sidx(r + 1, c));
        const float4 y1 = *reinterpret_cast<const float4*>(stw + sidx(r + 1, cq2));
        const float w[8] = {y0.x, y0.y, y0.z, y0.w, y1.x, y1.y, y1.z, y1.w};
        if (ok) val = G.epi.rows8p(pi, layer, grow + r, gcol + c, P.M, P.N, v, w, aux[sb & 1][b]);
        partial += val;
      } else if (ok) {
        if (pack_all) {
          float x[NAUX];
          const float* w = &aux[sb >> 1][b][4 * (sb & 1)];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const uint32_t u = __float_as_uint(w[e]);
            x[2 * e] = __uint_as_float(u << 16);
            x[2 * e + 1] = __uint_as_float(u & 0xffff0000u);
          }
          val = G.epi.rows8(pi, layer, grow + r, gcol + c, P.M, P.N, v, x);
        } else {
          val = G.epi.rows8(pi, layer, grow + r, gcol + c, P.M, P.N, v, aux[sb & 1][b]);
        }
        if constexpr (Epi::kWriteback) {
          *reinterpret_cast<float4*>(sa) =
              make_float4(sflip ? v[4] : v[0], sflip ? v[5] : v[1], sflip ? v[6] : v[2],
                          sflip ? v[7] : v[3]);
          *reinterpret_cast<float4*>(sb2) =
              make_float4(sflip ? v[0] : v[4], sflip ? v[1] : v[5], sflip ? v[2] : v[6],
                          sflip ? v[3] : v[7]);
        }
      }
      if constexpr (Epi::kRowScale) {
        // this wave's 64-column part of the row's sum of squares, for the scale pass
        val += __shfl_xor(val, 1, 64);
        val += __shfl_xor(val, 2, 64);
        val += __shfl_xor(val, 4, 64);
        if (ql == 0) rss[wave * SB + r] = val;
      } else if constexpr (!Epi::kPairRows) {
        if constexpr (Epi::kRowNorm) {
          // the 8 lanes of a row segment are lanes 8*rl .. 8*rl+7: a fixed-order tree sum
          val += __shfl_xor(val, 1, 64);
          val += __shfl_xor(val, 2, 64);
          val += __shfl_xor(val, 4, 64);
          if (ok && ql == 0) G.epi.row_partial(pi, layer, grow + r, gcol / SB, val);
        } else {
          partial += val;
        }
      }
    }
    if constexpr (Epi::kPre && Epi::kPreLate) {
      if (sb + 1 < NSB && !pack_all) issue_pre(sb + 1, aux[(sb + 1) & 1]);
    }
    if constexpr (Epi::kCols) {
      if (G.epi.has_cols(pi)) {
        if constexpr (Epi::kWriteback) wave_sync();
        const int kc = lane & 7;  // row group of this lane's column chunks
#pragma unroll
        for (int b = 0; b < CPL; ++b) {
          const int c = (lane >> 3) + 8 * b;
          if (grow + 8 * kc + 8 > P.M || gcol + c >= P.N) continue;
          float v[8];
#pragma unroll
          for (int e = 0; e < 8; ++e) v[e] = stw[sidx(8 * kc + e, c)];
          G.epi.cols8(pi, layer, grow + 8 * kc, gcol + c, P.M, P.N, v);
        }
      }
    }
  }
  if constexpr (Epi::kRowScale) {
    // Scale pass: every row of the tile is whole in this workgroup (4 waves x 64 columns); its
    // sum of squares is the 4 waves' parts in a fixed order.  The row pass left the unscaled
    // values in each wave's staging.
    __syncthreads();
    const int grow = m0, gcol = n0 + wave * SB;
#pragma unroll
    for (int b = 0; b < CPL; ++b) {
      const int r = rl + 8 * b, c = cq;
      if (grow + r >= P.M || gcol + c >= P.N) continue;
      const float tot = ((rss[r] + rss[SB + r]) + rss[2 * SB + r]) + rss[3 * SB + r];
      const float4 xa = *reinterpret_cast<const float4*>(stw + sidx(r, sflip ? cq2 : c));
      const float4 xb = *reinterpret_cast<const float4*>(stw + sidx(r, sflip ? c : cq2));
      const float v[8] = {sflip ? xb.x : xa.x, sflip ? xb.y : xa.y, sflip ? xb.z : xa.z,
                          sflip ? xb.w : xa.w, sflip ? xa.x : xb.x, sflip ? xa.y : xb.y,
                          sflip ? xa.z : xb.z, sflip ? xa.w : xb.w};
      G.epi.scale8(pi, layer, grow + r, gcol + c, P.N, tot, v);
    }
  }
  G.epi.finish(pi, layer, t, wave, lane, partial);
}

// ------------------------------------------------------------------------------------------
// Epilogues.  pre8() may read memory for a row chunk (batched before the arithmetic); rows8()
// handles 8 consecutive columns C[row][col..col+7] and returns a value summed per lane and
// handed to finish() (the loss partials; 0 elsewhere); with kWriteback its updated values feed
// the column pass; cols8() handles 8 consecutive rows C[row..row+7][col].  Intermediate
// buffers have Tp rows (seg_len rounded up to 256), so tiles store whole chunks; bounds are
// checked in the kernel: a chunk is handled only if its rows are below M and its columns below
// N (M and N are multiples of 8 wherever a column pass runs).

struct EpiBase {
  static constexpr int kParts = 1;  // K-concatenated operand parts the problems may have
  static constexpr bool kPre = false;  // pre8 reads memory (loads are issued a batch ahead)
  static constexpr bool kPreLate = false;  // ... after this sub-block's row pass rather than
                                           // before it (shorter lead, fewer live registers)
  static constexpr int kAux = 8;       // floats pre8 reads per row chunk
  static constexpr bool kRowNorm = false;  // rows8 returns the chunk's sum of squares, which
                                           // is reduced per 64-column row segment
  static constexpr bool kPairRows = false; // rows8p(v = row r, w = row r + 1) for even r
                                           // replaces rows8 (row pass only)
  static constexpr bool kRowScale = false; // rows8 writes its results back and returns their
                                           // sum of squares; after a workgroup barrier
                                           // scale8 gets each whole row's sum (64 x 256 tiles)
  __device__ __forceinline__ void scale8(int, int, int, int, int, float,
                                         const float (&)[8]) const {}
  __device__ __forceinline__ void row_partial(int, int, int, int, float) const {}
  static constexpr bool kCols = false;
  static constexpr bool kWriteback = false;
  __device__ __forceinline__ bool has_cols(int) const { return false; }
  // part 0 of a K-concatenated contraction contributes part0_scale(layer, col) times its
  // product to column col (when has_part0_scale())
  static constexpr bool kPart0Scale = false;
  __device__ __forceinline__ bool has_part0_scale() const { return false; }
  __device__ __forceinline__ float part0_scale(int, int) const { return 1.0f; }
  // pre8/rows8 (and scale8) of problem pi take split row chunks (columns c..c+3 and
  // c+32..c+35; N a multiple of 8; the second half may lie at or beyond N): the fp32
  // read-modify-write epilogues, whose 16-byte accesses then coalesce
  static constexpr bool kSplitCols = false;
  __device__ __forceinline__ bool split_cols(int) const { return false; }
  __device__ __forceinline__ void pre8(int, int, int, int, int, int, float (&)[8]) const {}
  // kPackAll: problem pi with pack_all(pi) reads 16-bit values (pre4p: 8 of them, packed in 4
  // dwords held as float bits, widened by the kernel before rows8), and the loads of all of a
  // wave's sub-blocks (at most 4) are issued before its first staging, in the registers of the
  // two buffers: more loads in flight than one sub-block ahead
  static constexpr bool kPackAll = false;
  __device__ __forceinline__ bool pack_all(int) const { return false; }
  __device__ __forceinline__ void pre4p(int, int, int, int, float (&)[4]) const {}
  __device__ __forceinline__ void cols8(int, int, int, int, int, int, const float (&)[8]) const {}
  __device__ __forceinline__ void finish(int, int, int, int, int, float) const {}
};

// Forward 1: tile of Z = X W1^T [tokens][h].  Stores A = SiLU(Z) [Tp][h] (rows) and A^T,
// SiLU'(Z)^T [h][Tp] (columns); token rows >= n are stored as 0.  With bf16 outputs the row
// pass evaluates the logistic once per element and leaves (A, SiLU') packed as two bf16 in the
// staging slot for the column pass; with fp32 outputs the column pass recomputes them.
template <typename E>
struct EpiFwd1 : EpiBase {
  static constexpr bool kCols = true;
  static constexpr bool kWriteback = sizeof(E) == 2;
  E* a; E* at; E* dst;
  long long ls;  // layer stride of a, at and dst (Tp*h)
  int h, Tp, n;
  // [L][h] or null: the W1 operand holds diag(1/cs) times the weights (a row renormalisation
  // of W1 not yet applied to it), so column j of Z is the accumulator times cs[j]
  const float* cs;
  __device__ __forceinline__ bool has_cols(int) const { return true; }
  __device__ __forceinline__ float rows8(int, int layer, int row, int col, int, int,
                                         float (&z)[8], const float (&)[8]) const {
    if (cs) {
      const float* c = cs + (long long)layer * h + col;
#pragma unroll
      for (int e = 0; e < 8; ++e) z[e] *= c[e];
    }
    float av[8], dv[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float s = sigmoidf_(z[e]);
      av[e] = row < n ? z[e] * s : 0.0f;
      dv[e] = row < n ? s * (1.0f + z[e] * (1.0f - s)) : 0.0f;
    }
    store8(a + (long long)layer * ls + (long long)row * h + col, av);
    if constexpr (kWriteback) {
#pragma unroll
      for (int e = 0; e < 8; ++e) z[e] = __uint_as_float(pack_bf16(av[e], dv[e]));
    }
    return 0.0f;
  }
  __device__ __forceinline__ void cols8(int, int layer, int row, int col, int, int,
                                        const float (&z)[8]) const {
    float av[8], dv[8];
    // fp32 (no write-back): the column pass recomputes from the staged accumulators
    const float c = !kWriteback && cs ? cs[(long long)layer * h + col] : 1.0f;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      if constexpr (kWriteback) {
        const uint32_t w = __float_as_uint(z[e]);
        av[e] = __uint_as_float(w << 16);
        dv[e] = __uint_as_float(w & 0xffff0000u);
      } else {
        const float zc = z[e] * c;
        const float s = sigmoidf_(zc);
        const bool ok = row + e < n;
        av[e] = ok ? zc * s : 0.0f;
        dv[e] = ok ? s * (1.0f + zc * (1.0f - s)) : 0.0f;
      }
    }
    const long long o = (long long)layer * ls + (long long)col * Tp + row;
    store8(at + o, av);
    store8(dst + o, dv);
  }
};

// Forward 2 and loss gradient: tile of -R [tokens][D], where the GEMM computes
// A (-W2)^T + X W_kv^T (K-concatenated, from the negated copy of W2), so R = Y - targets.
// Stores G = c R [Tp][D] (rows) and G^T [D][Tp] (columns); sums R^2 per wave into the loss
// partials (sq).  For the negative inner product the GEMM is X W_kv^T alone (the targets T)
// and the same formula gives G = -c T; its loss comes from the W2 update's epilogue instead.
// PSCALE: a row renormalisation of W2 not yet applied to its copy (ps, gs: [L][D], or null):
// the copy is diag(1/s) times -W2, so part 0's product is scaled by column (ps), and the
// stored G, which the backward contracts with the unscaled W2^T copy, is G diag(s) (gs); G^T
// is not.  (A separate instantiation: the scale between the parts costs the 256 x 256 tile
// some spilled registers around it.)
template <typename E, bool PSCALE = false>
struct EpiFwd2 : EpiBase {
  static constexpr int kParts = 2;
  static constexpr bool kCols = true;
  static constexpr bool kPart0Scale = PSCALE;
  E* g; E* gt;
  float* loss_part;       // [L][parts_per_layer]
  const float* rate;      // [L][Tp] per-token rates (the paper's optimiser), or null
  const float* ps;
  const float* gs;
  long long ls;           // Tp*D
  int D, Tp, n, parts_per_layer;
  int sq;                 // write the sum-of-squares loss partials
  float c;
  __device__ __forceinline__ bool has_cols(int) const { return true; }
  __device__ __forceinline__ bool has_part0_scale() const { return PSCALE && ps != nullptr; }
  __device__ __forceinline__ float part0_scale(int layer, int col) const {
    return ps[(long long)layer * D + col];
  }
  __device__ __forceinline__ float rows8(int, int layer, int row, int col, int, int,
                                         float (&v)[8], const float (&)[8]) const {
    const float cr = rate ? c * rate[(long long)layer * Tp + row] : c;
    float gv[8], s = 0.0f;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float r = row < n ? -v[e] : 0.0f;
      s += r * r;
      gv[e] = cr * r;
    }
    if (PSCALE && gs) {
      const float* f = gs + (long long)layer * D + col;
#pragma unroll
      for (int e = 0; e < 8; ++e) gv[e] *= f[e];
    }
    store8(g + (long long)layer * ls + (long long)row * D + col, gv);
    return s;
  }
  __device__ __forceinline__ void cols8(int, int layer, int row, int col, int, int,
                                        const float (&v)[8]) const {
    float gv[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float cr = rate ? c * rate[(long long)layer * Tp + row + e] : c;
      gv[e] = row + e < n ? -cr * v[e] : 0.0f;
    }
    store8(gt + (long long)layer * ls + (long long)col * Tp + row, gv);
  }
  __device__ __forceinline__ void finish(int, int layer, int tile, int wave, int lane,
                                        float s) const {
    if (!sq) return;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off, 64);
    if (lane == 0) loss_part[(long long)layer * parts_per_layer + tile * 4 + wave] = s;
  }
};

// Backward and W2 update in one launch (both need only G, A and the previous W2).
// Problem 0: tile of dA^T = W2^T G^T [h][tokens]; stores dZ^T = dA^T * SiLU'(Z)^T [h][Tp]
// (rows; token columns >= n are stored as 0).  Problem 1: tile of G^T A = dL/dW2 of W2
// [D][h]; fp32 read-modify-write of the master (rows), then the copies the next segment reads:
// -W2 [D][h] (rows) and W2^T [h][D] (columns).  The backward reads the W2^T copy of the
// weights the step started from; the update writes the other copy of a ping-pong pair.
// With the paper's optimiser (PAPER), problem 1 updates the momentum, mu2 = beta mu2 + G^T A
// (the rates are already in G), and the master, W2 - mu2, both fp32; it returns each row
// chunk's sum of squares for the renormalisation, which writes the copies afterwards.  With a
// renormalisation pending (rs: [L][D], or null) the stored master is diag(1/rs) times the
// weights, so the update reads rs[row] times it; with copy_pending it writes the copies of its
// (not yet renormalised) result itself.
// For the negative inner product (nip, SGD only) problem 1 also sums <W2_{s-1}, G^T A> per
// wave into the loss partials: with G = -T/n that is -(1/n) sum_j t_j . y_j = L_s.
template <typename E, bool PAPER = false>
struct EpiBwdW2 : EpiBase {
  static constexpr bool kPre = true;
  static constexpr bool kPreLate = true;  // measured faster on 256 x 256 tiles (fewer spills)
  static constexpr int kAux = 8;  // the master (PAPER: the momentum is read in the row pass,
                                  // which keeps the 256 x 256 tile within its registers)
  static constexpr bool kRowNorm = PAPER;
  static constexpr bool kCols = true;
  static constexpr bool kWriteback = true;
  const E* dst; E* dzt;
  long long lst;       // Tp*h
  int Tp, n;
  float* w2; E* w2n; E* w2t;
  long long ls2;       // D*h
  int h, D;
  float lr;
  float* mom2;         // PAPER: [L][D][h] momentum
  const float* beta;   // PAPER: [L] momentum decay of this segment
  float* ss2;          // PAPER: [L][D][h/64] row-segment sums of squares
  const float* rs;     // PAPER: pending row scale of the master, or null
  int copy_pending;    // PAPER: write the copies of the result
  float* loss_part;    // nip: [L][parts_per_layer]
  int parts_per_layer;
  int nip;
  __device__ __forceinline__ bool has_cols(int pi) const {
    return pi == 1 && (!PAPER || copy_pending);
  }
  static constexpr bool kSplitCols = true;  // problem 1: split row chunks (h is a multiple of 64)
  __device__ __forceinline__ bool split_cols(int pi) const { return pi == 1; }
  // problem 0 (bf16): SiLU' of all sub-blocks loaded at once, packed
  static constexpr bool kPackAll = sizeof(E) == 2;
  __device__ __forceinline__ bool pack_all(int pi) const { return sizeof(E) == 2 && pi == 0; }
  __device__ __forceinline__ void pre4p(int, int layer, int row, int col, float (&w)[4]) const {
    const u32x4 u =
        *reinterpret_cast<const u32x4*>(dst + (long long)layer * lst + (long long)row * Tp + col);
#pragma unroll
    for (int e = 0; e < 4; ++e) w[e] = __uint_as_float(u[e]);
  }
  __device__ __forceinline__ void pre8(int pi, int layer, int row, int col, int, int,
                                       float (&x)[kAux]) const {
    float (&x0)[8] = *reinterpret_cast<float(*)[8]>(&x[0]);
    if (pi == 0) {
      load8(dst + (long long)layer * lst + (long long)row * Tp + col, x0);
    } else {
      const long long o = (long long)layer * ls2 + (long long)row * h + col;
      load8_split(w2 + o, x0);
    }
  }
  __device__ __forceinline__ float rows8(int pi, int layer, int row, int col, int, int,
                                         float (&v)[8], const float (&x)[kAux]) const {
    if (pi == 0) {
      float dz[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) dz[e] = col + e < n ? v[e] * x[e] : 0.0f;
      store8(dzt + (long long)layer * lst + (long long)row * Tp + col, dz);
      return 0.0f;
    }
    const long long o = (long long)layer * ls2 + (long long)row * h + col;
    if constexpr (PAPER) {
      const float b = beta[layer];
      const float sr = rs ? rs[(long long)layer * D + row] : 1.0f;
      float m[8], nw[8], ss = 0.0f;
      load8_split(mom2 + o, m);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        m[e] = b * m[e] + v[e];
        nw[e] = sr * x[e] - m[e];
        ss += nw[e] * nw[e];
      }
      store8_split(mom2 + o, m);
      store8_split(w2 + o, nw);
      if (copy_pending) {
        float cp[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) cp[e] = -nw[e];
        store8_split(w2n + o, cp);
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = nw[e];
      return ss;
    } else {
      float nw[8], cp[8], ip = 0.0f;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        ip += x[e] * v[e];
        nw[e] = x[e] - lr * v[e];
        cp[e] = -nw[e];
      }
      store8_split(w2 + o, nw);
      store8_split(w2n + o, cp);
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = nw[e];
      return nip ? ip : 0.0f;
    }
  }
  __device__ __forceinline__ void finish(int pi, int layer, int tile, int wave, int lane,
                                        float s) const {
    if (PAPER || !nip || pi != 1) return;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off, 64);
    if (lane == 0) loss_part[(long long)layer * parts_per_layer + tile * 4 + wave] = s;
  }
  __device__ __forceinline__ void row_partial(int pi, int layer, int row, int cb, float ss) const {
    if (PAPER && pi == 1) ss2[((long long)layer * D + row) * (h / 64) + cb] = ss;
  }
  __device__ __forceinline__ void cols8(int, int layer, int row, int col, int, int,
                                        const float (&v)[8]) const {
    store8(w2t + (long long)layer * ls2 + (long long)col * D + row, v);
  }
};

// W1 update: tile of dZ^T X = dL/dW1 of W1 [h][d]; fp32 read-modify-write of the master, and
// in bf16 mode the rounded copy the next segment's forward reads (fp32 mode reads the master).
// With the paper's optimiser (PAPER): mu1 = beta mu1 + dZ^T X, W1 - mu1 (fp32), and each row
// chunk's sum of squares for the renormalisation, which writes the copy afterwards.
template <typename E, bool PAPER = false>
struct EpiW1 : EpiBase {
  static constexpr bool kPre = true;
  static constexpr int kAux = 8;  // the master (PAPER: the momentum is read in the row pass)
  static constexpr bool kRowNorm = PAPER;
  float* w1; E* w1s;
  long long ls1;  // h*d
  int d;
  int w1_copy;
  float lr;
  float* mom1;         // PAPER: [L][h][d] momentum
  const float* beta;   // PAPER: [L]
  float* ss1;          // PAPER: [L][h][d/64] row-segment sums of squares
  int h;
  // PAPER: [L][h] or null: the stored master is diag(1/rs) times the weights (a row
  // renormalisation not yet applied to it), so the update reads rs[row] times the master; with
  // copy_pending the update also writes the copy of its (not yet renormalised) result
  const float* rs;
  int copy_pending;
  static constexpr bool kSplitCols = true;  // split row chunks (d is a multiple of 64)
  __device__ __forceinline__ bool split_cols(int) const { return true; }
  __device__ __forceinline__ void pre8(int, int layer, int row, int col, int, int,
                                       float (&w)[kAux]) const {
    const long long o = (long long)layer * ls1 + (long long)row * d + col;
    load8_split(w1 + o, w);
  }
  __device__ __forceinline__ float rows8(int, int layer, int row, int col, int, int,
                                         float (&v)[8], const float (&w)[kAux]) const {
    const long long o = (long long)layer * ls1 + (long long)row * d + col;
    if constexpr (PAPER) {
      const float b = beta[layer];
      const float sr = rs ? rs[(long long)layer * h + row] : 1.0f;
      float m[8], nw[8], ss = 0.0f;
      load8_split(mom1 + o, m);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        m[e] = b * m[e] + v[e];
        nw[e] = sr * w[e] - m[e];
        ss += nw[e] * nw[e];
      }
      store8_split(mom1 + o, m);
      store8_split(w1 + o, nw);
      if (copy_pending) store8_split(w1s + o, nw);
      return ss;
    } else {
      float nw[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) nw[e] = w[e] - lr * v[e];
      store8_split(w1 + o, nw);
      if (w1_copy) store8_split(w1s + o, nw);
      return 0.0f;
    }
  }
  __device__ __forceinline__ void row_partial(int, int layer, int row, int cb, float ss) const {
    if (PAPER) ss1[((long long)layer * h + row) * (d / 64) + cb] = ss;
  }
};

// Read, first layer: tile of X_q W1^T [q][h]; stores A_q = SiLU(.) [Tp][h] (rows >= q hold
// SiLU(0) = 0).
template <typename E>
struct EpiKv1 : EpiBase {
  E* a;
  long long ls;
  int h;
  __device__ __forceinline__ float rows8(int, int layer, int row, int col, int, int,
                                         float (&z)[8], const float (&)[8]) const {
    float av[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) av[e] = z[e] * sigmoidf_(z[e]);
    store8(a + (long long)layer * ls + (long long)row * h + col, av);
    return 0.0f;
  }
};

// Read, second layer: tile of A_q (-W2)^T = -KV [q][D]; stores KV into the caller's [L][q][D]
// output (fp32 or bf16), rows < q only.
struct EpiKv2 : EpiBase {
  void* kv;
  long long ls;  // q*D
  int D;
  int bf16_out;
  __device__ __forceinline__ float rows8(int, int layer, int row, int col, int M, int,
                                         float (&v)[8], const float (&)[8]) const {
    if (row >= M) return 0.0f;
    float y[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) y[e] = -v[e];
    const long long o = (long long)layer * ls + (long long)row * D + col;
    if (bf16_out)
      store8(reinterpret_cast<bf16_t*>(kv) + o, y);
    else
      store8(reinterpret_cast<float*>(kv) + o, y);
    return 0.0f;
  }
};

// ------------------------------------------------------------------------------------------
// Epilogues of the block form of consecutive segments (mone_ttl_segments).  A block of B
// segments j = 0..B-1 of T tokens each (block rows jT .. jT + T - 1) starts from the weights
// W_0 it finds.  Each segment's step uses W_{j-1} = W_0 minus the updates of the block's
// earlier segments, and those enter as products with T x T token blocks (exact algebra, the
// summation order aside):
//   Z_j  = X_j W1_{j-1}^T = X_j W1_0^T - lr sum_{i<j} (X_j X_i^T) dZ_i
//   Y_j  = A_j W2_{j-1}^T = A_j W2_0^T - lr sum_{i<j} (A_j A_i^T) G_i
//   dA_j = G_j W2_{j-1}   = G_j W2_0   - lr sum_{i<j} (G_j G_i^T) A_i
// The weights are read and written once per block: W -= lr sum_j (gradient of segment j).

// Plain stores of the accumulators times a per-problem scale: problem 0 as T0 [rows][ld0],
// problem 1 as T1 [rows][ld1] (the token-block products and the pre-update GEMMs).  Split row
// chunks (every column count here is a multiple of 64), so the fp32 outputs are stored with
// 16-byte accesses contiguous across lanes.
template <typename T0, typename T1>
struct EpiStore : EpiBase {
  static constexpr bool kSplitCols = true;
  __device__ __forceinline__ bool split_cols(int) const { return true; }
  T0* p0; long long ls0; int ld0; float s0;
  T1* p1; long long ls1; int ld1; float s1;
  __device__ __forceinline__ float rows8(int pi, int layer, int row, int col, int, int,
                                         float (&v)[8], const float (&)[8]) const {
    float o[8];
    const float sc = pi == 0 ? s0 : s1;
#pragma unroll
    for (int e = 0; e < 8; ++e) o[e] = sc * v[e];
    if (pi == 0) store8_split(p0 + (long long)layer * ls0 + (long long)row * ld0 + col, o);
    else store8_split(p1 + (long long)layer * ls1 + (long long)row * ld1 + col, o);
    return 0.0f;
  }
};

// Block form, pre-activations of segment j: Z = Z0 - lr acc with acc = (X_j X_<j^T) dZ_<j and
// Z0 = X_j W1_0^T; stores A = SiLU(Z) (block rows r0 + row, and A^T by columns) and SiLU'(Z).
template <typename E>
struct EpiBlkZ : EpiBase {
  static constexpr bool kPre = true;
  static constexpr bool kCols = true;
  static constexpr bool kWriteback = true;
  const float* z0;     // [L][Btp][h]
  E* a; E* at; E* sd;  // A [Btp][h], A^T [h][Btp], SiLU'(Z) [Btp][h]
  long long ls;        // Btp*h
  int h, Btp, r0;
  float lr;
  __device__ __forceinline__ bool has_cols(int) const { return true; }
  __device__ __forceinline__ void pre8(int, int layer, int row, int col, int, int,
                                       float (&x)[8]) const {
    load8(z0 + (long long)layer * ls + (long long)(r0 + row) * h + col, x);
  }
  __device__ __forceinline__ float rows8(int, int layer, int row, int col, int, int,
                                         float (&v)[8], const float (&x)[8]) const {
    float av[8], dv[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float z = x[e] - lr * v[e];
      const float sg = sigmoidf_(z);
      av[e] = z * sg;
      dv[e] = sg * (1.0f + z * (1.0f - sg));
    }
    const long long o = (long long)layer * ls + (long long)(r0 + row) * h + col;
    store8(a + o, av);
    store8(sd + o, dv);
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = av[e];
    return 0.0f;
  }
  __device__ __forceinline__ void cols8(int, int layer, int row, int col, int, int,
                                        const float (&v)[8]) const {
    store8(at + (long long)layer * ls + (long long)col * Btp + r0 + row, v);
  }
};

// Block form, output layer of segment j at W2_0: problem 0 is A_j (-W2_0)^T = -Y0, stored as
// the pre-update residual R0 = Y0 - targets (fp32); problem 1 is the token block
// P = A_j A_<j^T.
template <typename E>
struct EpiBlkY0 : EpiBase {
  static constexpr bool kPre = true;
  const float* tgt; long long lst;  // targets [L][Btp][D] (block rows)
  float* rr; long long lsr;         // R0 [L][Tp][D]
  E* pg; long long lsp;             // P [L][Tp][Btp]
  int D, Btp, r0;
  __device__ __forceinline__ void pre8(int pi, int layer, int row, int col, int, int,
                                       float (&x)[8]) const {
    if (pi == 0) {
      load8(tgt + (long long)layer * lst + (long long)(r0 + row) * D + col, x);
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) x[e] = 0.0f;
    }
  }
  __device__ __forceinline__ float rows8(int pi, int layer, int row, int col, int, int,
                                         float (&v)[8], const float (&x)[8]) const {
    if (pi == 0) {
      float o[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) o[e] = -v[e] - x[e];
      store8(rr + (long long)layer * lsr + (long long)row * D + col, o);
    } else {
      store8(pg + (long long)layer * lsp + (long long)row * Btp + col, v);
    }
    return 0.0f;
  }
};

// Block form, loss gradient of segment j: R = R0 - lr acc with acc = P G_<j; stores G = c R
// (block rows, and G^T by columns) and sums R^2 per wave into the loss partials.
template <typename E>
struct EpiBlkG : EpiBase {
  static constexpr bool kPre = true;
  static constexpr bool kCols = true;
  static constexpr bool kWriteback = true;
  const float* rr; long long lsr;  // R0 [L][Tp][D]
  E* g; E* gt; long long lsg;      // G [L][Btp][D], G^T [L][D][Btp]
  float* loss_part;
  int D, Btp, r0, parts_per_layer;
  float lr, c;
  __device__ __forceinline__ bool has_cols(int) const { return true; }
  __device__ __forceinline__ void pre8(int, int layer, int row, int col, int, int,
                                       float (&x)[8]) const {
    load8(rr + (long long)layer * lsr + (long long)row * D + col, x);
  }
  __device__ __forceinline__ float rows8(int, int layer, int row, int col, int, int,
                                         float (&v)[8], const float (&x)[8]) const {
    float gv[8], sq = 0.0f;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float r = x[e] - lr * v[e];
      sq += r * r;
      gv[e] = c * r;
    }
    store8(g + (long long)layer * lsg + (long long)(r0 + row) * D + col, gv);
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = gv[e];
    return sq;
  }
  __device__ __forceinline__ void cols8(int, int layer, int row, int col, int, int,
                                        const float (&v)[8]) const {
    store8(gt + (long long)layer * lsg + (long long)col * Btp + r0 + row, v);
  }
  __device__ __forceinline__ void finish(int, int layer, int tile, int wave, int lane,
                                        float sq) const {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) sq += __shfl_xor(sq, off, 64);
    if (lane == 0) loss_part[(long long)layer * parts_per_layer + tile * 4 + wave] = sq;
  }
};

// Block form, backward of segment j: dA = dA0 - lr acc with acc = Q A_<j (Q = G_j G_<j^T) and
// dA0 = G_j W2_0; stores dZ = dA * SiLU'(Z) by columns into dZ^T (block token columns).
template <typename E>
struct EpiBlkDZ : EpiBase {
  static constexpr bool kPre = true;
  static constexpr bool kCols = true;
  static constexpr bool kWriteback = true;
  const float* da0; long long lsa;  // dA0 [L][Tp][h]
  const E* sd; E* dzt; long long ls;  // SiLU'(Z) [L][Btp][h], dZ^T [L][h][Btp]
  int h, Btp, r0;
  float lr;
  __device__ __forceinline__ bool has_cols(int) const { return true; }
  __device__ __forceinline__ void pre8(int, int layer, int row, int col, int, int,
                                       float (&x)[8]) const {
    load8(da0 + (long long)layer * lsa + (long long)row * h + col, x);
  }
  __device__ __forceinline__ float rows8(int, int layer, int row, int col, int, int,
                                         float (&v)[8], const float (&x)[8]) const {
    float sv[8];
    load8(sd + (long long)layer * ls + (long long)(r0 + row) * h + col, sv);
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = (x[e] - lr * v[e]) * sv[e];
    return 0.0f;
  }
  __device__ __forceinline__ void cols8(int, int layer, int row, int col, int, int,
                                        const float (&v)[8]) const {
    store8(dzt + (long long)layer * ls + (long long)col * Btp + r0 + row, v);
  }
};

// Block form, the block's updates in one launch: problem 0 is the W2 update (G^T A: the W2
// update problem of EpiBwdW2, writing -W2 and the next W2^T copy), problem 1 the W1 update
// (dZ^T X: EpiW1).  Both read-modify-write epilogues stream their masters in one grid.
template <typename E>
struct EpiBlkUpd : EpiBase {
  static constexpr bool kPre = true;
  static constexpr bool kCols = true;
  static constexpr bool kWriteback = true;
  EpiBwdW2<E, false> w2;
  EpiW1<E, false> w1;
  __device__ __forceinline__ bool has_cols(int pi) const { return pi == 0; }
  static constexpr bool kSplitCols = true;  // both problems: as w2's problem 1 and w1
  __device__ __forceinline__ bool split_cols(int) const { return true; }
  __device__ __forceinline__ void pre8(int pi, int layer, int row, int col, int M, int N,
                                       float (&x)[8]) const {
    if (pi == 0) w2.pre8(1, layer, row, col, M, N, x);
    else w1.pre8(0, layer, row, col, M, N, x);
  }
  __device__ __forceinline__ float rows8(int pi, int layer, int row, int col, int M, int N,
                                         float (&v)[8], const float (&x)[8]) const {
    return pi == 0 ? w2.rows8(1, layer, row, col, M, N, v, x)
                   : w1.rows8(0, layer, row, col, M, N, v, x);
  }
  __device__ __forceinline__ void cols8(int, int layer, int row, int col, int M, int N,
                                        const float (&v)[8]) const {
    w2.cols8(1, layer, row, col, M, N, v);
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

// X^T staging: dst[l][c][r] = src[l][r][c] for r < R, 0 for R <= r < Rz (Rz a multiple of 64).
// 64 x 64 tiles through LDS with 16-byte vector loads (along c) and stores (along r).
template <typename E>
__global__ __launch_bounds__(256) void transpose_vec_kernel(const E* __restrict__ src,
                                                            long long src_ls, int src_ld, int R,
                                                            int C, E* __restrict__ dst,
                                                            long long dst_ls, int dst_ld,
                                                            int Rz) {
  constexpr int VEC = 16 / (int)sizeof(E);
  constexpr int VPR = 64 / VEC;          // vectors per 64-element row
  constexpr int NV = 64 * VPR / 256;     // vectors per thread
  __shared__ float tile[64][65];
  const int c0 = blockIdx.x * 64, r0 = blockIdx.y * 64, l = blockIdx.z;
  const E* s = src + (long long)l * src_ls;
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    const int idx = threadIdx.x + 256 * i, r = idx / VPR, cv = idx % VPR;
    const int gr = r0 + r, gc = c0 + cv * VEC;
    float v[8];
    if (gr < R && gc < C) {
      if constexpr (VEC == 8) {
        load8(reinterpret_cast<const bf16_t*>(s) + (long long)gr * src_ld + gc, v);
      } else {
        const float4 x = *reinterpret_cast<const float4*>(s + (long long)gr * src_ld + gc);
        v[0] = x.x; v[1] = x.y; v[2] = x.z; v[3] = x.w;
      }
    } else {
#pragma unroll
      for (int e = 0; e < VEC; ++e) v[e] = 0.0f;
    }
#pragma unroll
    for (int e = 0; e < VEC; ++e) tile[r][cv * VEC + e] = v[e];
  }
  __syncthreads();
  E* o = dst + (long long)l * dst_ls;
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    const int idx = threadIdx.x + 256 * i, c = idx / VPR, u = idx % VPR;
    const int gc = c0 + c, gr = r0 + u * VEC;
    if (gc >= C || gr >= Rz) continue;
    float v[8];
#pragma unroll
    for (int e = 0; e < VEC; ++e) v[e] = tile[u * VEC + e][c];
    if constexpr (VEC == 8) {
      store8(reinterpret_cast<bf16_t*>(o) + (long long)gc * dst_ld + gr, v);
    } else {
      *reinterpret_cast<float4*>(o + (long long)gc * dst_ld + gr) = make_float4(v[0], v[1], v[2], v[3]);
    }
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

// ------------------------------------------------------------------------------------------
// The paper's optimiser: per-token rates, momentum decay, row renormalisation

__device__ __forceinline__ float softplusf_(float z) {
  return fmaxf(z, 0.0f) + log1pf(__expf(-fabsf(z)));
}

// Per-token rates rate[l][j] = lr * softplus(u_l . x_j + b_u[l]) for j < n (0 for n <= j < Tp),
// and per-block sums of v_l . x_j over the block's kRateTokens tokens (summed in token order),
// from which decay_kernel forms the momentum decay.  Grid (Tp / kRateTokens, L, segments), 256
// threads: each wave takes kRateTokens / 4 consecutive tokens.  Segment z reads x + z * x_ss
// and writes rate + z * rate_ss and vpart + z * vpart_ss.
constexpr int kRateTokens = 16;
template <typename E>
__global__ __launch_bounds__(256) void rate_kernel(const E* __restrict__ x, long long x_ls, int d,
                                                   int n, const float* __restrict__ u,
                                                   const float* __restrict__ bu,
                                                   const float* __restrict__ v, float lr,
                                                   float* __restrict__ rate, int Tp,
                                                   float* __restrict__ vpart, long long x_ss = 0,
                                                   long long rate_ss = 0,
                                                   long long vpart_ss = 0) {
  constexpr int TW = kRateTokens / 4;
  const int l = blockIdx.y, j0 = blockIdx.x * kRateTokens, wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  __shared__ float wsum[4];
  x += blockIdx.z * x_ss;
  rate += blockIdx.z * rate_ss;
  vpart += blockIdx.z * vpart_ss;
  // This wave's TW tokens side by side: per 8-element chunk of the lane, u and v are read once
  // and the TW tokens' loads are issued together (each token's sums keep the chunk order).
  const E* xl = x + (long long)l * x_ls;
  const float* ul = u + (long long)l * d;
  const float* vl = v + (long long)l * d;
  const int jw = j0 + wave * TW;
  float su[TW], sv[TW];
#pragma unroll
  for (int t = 0; t < TW; ++t) su[t] = sv[t] = 0.0f;
  for (int c = lane * 8; c < d; c += 64 * 8) {
    float uu[8], vv[8], xv[TW][8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      uu[e] = ul[c + e];
      vv[e] = vl[c + e];
    }
#pragma unroll
    for (int t = 0; t < TW; ++t) {
      if (jw + t < n) {
        load8(xl + (long long)(jw + t) * d + c, xv[t]);
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) xv[t][e] = 0.0f;
      }
    }
#pragma unroll
    for (int t = 0; t < TW; ++t)
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        su[t] += xv[t][e] * uu[e];
        sv[t] += xv[t][e] * vv[e];
      }
  }
  float acc = 0.0f;
#pragma unroll
  for (int t = 0; t < TW; ++t) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
      su[t] += __shfl_xor(su[t], off, 64);
      sv[t] += __shfl_xor(sv[t], off, 64);
    }
    const int j = jw + t;
    if (lane == 0) {
      rate[(long long)l * Tp + j] = j < n ? lr * softplusf_(su[t] + bu[l]) : 0.0f;
      acc += j < n ? sv[t] : 0.0f;
    }
  }
  if (lane == 0) wsum[wave] = acc;
  __syncthreads();
  if (threadIdx.x == 0)
    vpart[(long long)l * (Tp / kRateTokens) + blockIdx.x] =
        ((wsum[0] + wsum[1]) + wsum[2]) + wsum[3];
}

// beta[l] = sigmoid(mean_j (v_l . x_j) + b_v[l]) = sigmoid(v_l . xbar + b_v[l]).  Grid
// (ceil(L / blockDim), segments): segment y reads vpart + y * L * nblk, writes beta + y * L.
__global__ void decay_kernel(const float* __restrict__ vpart, int nblk, int n,
                             const float* __restrict__ bv, float* __restrict__ beta, int L) {
  const int l = blockIdx.x * blockDim.x + threadIdx.x;
  if (l >= L) return;
  vpart += (long long)blockIdx.y * L * nblk;
  beta += (long long)blockIdx.y * L;
  float s = 0.0f;
  for (int b = 0; b < nblk; ++b) s += vpart[(long long)l * nblk + b];
  beta[l] = sigmoidf_(s / (float)n + bv[l]);
}

// L2 norm of every row of w [L][R][C] (fp32): one wave per row.  Grid (ceil(R / 4), L).
__global__ __launch_bounds__(256) void row_norm_kernel(const float* __restrict__ w, int R, int C,
                                                       float* __restrict__ norms) {
  const int l = blockIdx.y, r = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (r >= R) return;
  const float* row = w + ((long long)l * R + r) * C;
  float s = 0.0f;
  for (int c = lane * 4; c < C; c += 256) {
    const float4 a = *reinterpret_cast<const float4*>(row + c);
    s += a.x * a.x + a.y * a.y + a.z * a.z + a.w * a.w;
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off, 64);
  if (lane == 0) norms[(long long)l * R + r] = sqrtf(s);
}

// Row scales of the renormalisation: scale[l][r] = norm0[l][r] / ||row||, with ||row||^2 the
// sum of the row's nseg segment sums (fixed order); a row of norm 0 keeps scale 1.
__global__ void row_scale_kernel(const float* __restrict__ ss, int nseg, const float* __restrict__ norm0,
                                 float* __restrict__ scale, long long rows) {
  const long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= rows) return;
  float s = 0.0f;
  for (int b = 0; b < nseg; ++b) s += ss[i * nseg + b];
  scale[i] = s > 0.0f ? norm0[i] * rsqrtf(s) : 1.0f;
}

// W1 renormalisation: w1[l][r][:] *= scale[l][r]; in bf16 mode also the rounded copy w1s.
// Grid (ceil(h * d / 2048), L), 256 threads, 8 elements per thread.
template <typename E>
__global__ __launch_bounds__(256) void renorm_w1_kernel(float* __restrict__ w1, E* __restrict__ w1s,
                                                        const float* __restrict__ scale, int h, int d) {
  const int l = blockIdx.y;
  const long long i = ((long long)blockIdx.x * 256 + threadIdx.x) * 8;
  if (i >= (long long)h * d) return;
  const long long o = (long long)l * h * d + i;
  const float sc = scale[(long long)l * h + i / d];
  float v[8];
  load8(w1 + o, v);
#pragma unroll
  for (int e = 0; e < 8; ++e) v[e] *= sc;
  store8(w1 + o, v);
  if (w1s) store8(w1s + o, v);
}

// W2 renormalisation: w2[l][r][c] *= scale[l][r]; writes the copies the next segment reads,
// -W2 [D][h] and W2^T [h][D].  64 x 64 tiles through LDS; grid (h / 64, D / 64, L).
template <typename E>
__global__ __launch_bounds__(256) void renorm_w2_kernel(float* __restrict__ w2, E* __restrict__ w2n,
                                                        E* __restrict__ w2t,
                                                        const float* __restrict__ scale, int D, int h) {
  __shared__ float tile[64][65];
  const int c0 = blockIdx.x * 64, r0 = blockIdx.y * 64, l = blockIdx.z;
  const long long base = (long long)l * D * h;
#pragma unroll
  for (int i = 0; i < 2; ++i) {  // 64 rows x 8 chunks of 8 columns
    const int idx = threadIdx.x + 256 * i, r = idx >> 3, cc = (idx & 7) * 8;
    const long long o = base + (long long)(r0 + r) * h + c0 + cc;
    const float sc = scale[(long long)l * D + r0 + r];
    float v[8], nv[8];
    load8(w2 + o, v);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      v[e] *= sc;
      nv[e] = -v[e];
      tile[r][cc + e] = v[e];
    }
    store8(w2 + o, v);
    store8(w2n + o, nv);
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < 2; ++i) {  // 64 columns x 8 chunks of 8 rows, transposed
    const int idx = threadIdx.x + 256 * i, c = idx >> 3, rr = (idx & 7) * 8;
    float v[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = tile[rr + e][c];
    store8(w2t + base + (long long)(c0 + c) * D + r0 + rr, v);
  }
}

// ------------------------------------------------------------------------------------------
// Memory injection into attention (read time)

// out[l][i][a] = softmax over the keys j <= i of both sets (the query-side keys k_j and the
// memory keys km_j, one softmax) of the scaled scores q_i . k, applied to [v_j ; vm_j].  Head a
// of Q reads key/value head a / (n_heads / n_kv_heads); head width dh <= DHM.
// Workgroup: 16 query rows of one head and layer, 4 rows per wave.  Keys and values pass
// through LDS in chunks of 32 of each set, as fp32.  Score pass: lane L takes key L of the chunk
// (query-side keys on lanes 0-31, memory keys on lanes 32-63) over key rows of odd stride, so the
// 64 lanes read 64 distinct banks while the query rows are broadcast.  The softmax is online
// over the chunks in order (deterministic); the weighted sum has lanes over the head's columns.
// Grid (ceil(q / 16), n_heads, L), 256 threads.
template <typename E, typename EK, typename EO, int DHM>
__global__ __launch_bounds__(256) void memory_attention_kernel(
    const E* __restrict__ qh, const E* __restrict__ kh, const E* __restrict__ vh,
    const EK* __restrict__ kvm, EO* __restrict__ out, int q, int n_heads, int n_kv_heads, int dh,
    int d_kv, float scale) {
  constexpr int KC = 32;       // keys of each set per chunk
  constexpr int RW = 4;        // query rows per wave
  constexpr int QB = 4 * RW;   // query rows per workgroup
  constexpr int KS = DHM + 1;  // key row stride in LDS (odd)
  constexpr int NT = DHM / 64; // head columns per lane in the weighted sum
  __shared__ float ks[2 * KC * KS];   // [query-side keys ; memory keys] of the chunk
  __shared__ __attribute__((aligned(16))) float vs[2 * KC * DHM];  // [query-side ; memory values]
  __shared__ __attribute__((aligned(16))) float qs[QB * DHM];  // the block's query rows, scaled
  const int l = blockIdx.z, a = blockIdx.y, i0 = blockIdx.x * QB;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = a / (n_heads / n_kv_heads);
  const int dh4 = (dh + 3) & ~3;  // columns the score pass runs over (zero beyond dh)
  const long long qw = (long long)n_heads * dh, kw = (long long)n_kv_heads * dh;
  const E* ql = qh + (long long)l * q * qw + (long long)a * dh;
  const E* kl = kh + (long long)l * q * kw + (long long)g * dh;
  const E* vl = vh + (long long)l * q * kw + (long long)g * dh;
  const EK* ml = kvm + (long long)l * q * 2 * d_kv + (long long)g * dh;
  const int last = (i0 + QB < q ? i0 + QB : q) - 1;  // the block's last query row

  // Operand rows are moved in groups of 8 columns with 16-byte loads when dh is a multiple of
  // 8 (every row then starts 16-byte aligned), all of a thread's loads before its LDS writes;
  // element by element otherwise.
  const bool vec = (dh & 7) == 0;
  const int g8 = dh >> 3;
  if (vec) {
    constexpr int UQ = (QB * (DHM / 8) + 255) / 256;
    float x8[UQ][8];
#pragma unroll
    for (int u = 0; u < UQ; ++u) {
      const int x = tid + 256 * u, r = x / g8;
#pragma unroll
      for (int e = 0; e < 8; ++e) x8[u][e] = 0.0f;
      if (x < QB * g8 && i0 + r < q) load8(ql + (long long)(i0 + r) * qw + (x - r * g8) * 8, x8[u]);
    }
#pragma unroll
    for (int u = 0; u < UQ; ++u) {
      const int x = tid + 256 * u, r = x / g8, c = (x - r * g8) * 8;
      if (x >= QB * g8) continue;
      float* dst = qs + r * DHM + c;
      *reinterpret_cast<float4*>(dst) = make_float4(x8[u][0] * scale, x8[u][1] * scale,
                                                    x8[u][2] * scale, x8[u][3] * scale);
      *reinterpret_cast<float4*>(dst + 4) = make_float4(x8[u][4] * scale, x8[u][5] * scale,
                                                        x8[u][6] * scale, x8[u][7] * scale);
    }
  } else {
    for (int x = tid; x < QB * dh4; x += 256) {
      const int r = x / dh4, d = x - r * dh4;
      float v = 0.0f;
      if (i0 + r < q && d < dh) v = to_f32(ql[(long long)(i0 + r) * qw + d]) * scale;
      qs[r * DHM + d] = v;
    }
  }
  float m[RW], lsum[RW], acc[RW][NT];
#pragma unroll
  for (int r = 0; r < RW; ++r) {
    m[r] = -INFINITY;
    lsum[r] = 0.0f;
#pragma unroll
    for (int t = 0; t < NT; ++t) acc[r][t] = 0.0f;
  }
  // rows past q repeat the last row (finite, never stored)
  int row[RW];
#pragma unroll
  for (int r = 0; r < RW; ++r) {
    const int i = i0 + wave * RW + r;
    row[r] = i < last ? i : last;
  }

  for (int j0 = 0; j0 <= last; j0 += KC) {
    __syncthreads();  // the previous chunk is consumed (and the query rows are in place)
    // chunk row rr < KC: query-side key/value j0 + rr; rr >= KC: memory key/value j0 + rr - KC
    if (vec) {
      constexpr int UK = (2 * KC * (DHM / 8) + 255) / 256;
      float k8[UK][8], v8[UK][8];
#pragma unroll
      for (int u = 0; u < UK; ++u) {
        const int x = tid + 256 * u, rr = x / g8, c = (x - rr * g8) * 8;
        const int j = j0 + (rr & (KC - 1));
#pragma unroll
        for (int e = 0; e < 8; ++e) k8[u][e] = v8[u][e] = 0.0f;
        if (x < 2 * KC * g8 && j < q) {
          if (rr < KC) {
            load8(kl + (long long)j * kw + c, k8[u]);
            load8(vl + (long long)j * kw + c, v8[u]);
          } else {
            const EK* mj = ml + (long long)j * 2 * d_kv;
            load8(mj + c, k8[u]);
            load8(mj + d_kv + c, v8[u]);
          }
        }
      }
#pragma unroll
      for (int u = 0; u < UK; ++u) {
        const int x = tid + 256 * u, rr = x / g8, c = (x - rr * g8) * 8;
        if (x >= 2 * KC * g8) continue;
#pragma unroll
        for (int e = 0; e < 8; ++e) ks[rr * KS + c + e] = k8[u][e];
        float* vd = vs + rr * DHM + c;
        *reinterpret_cast<float4*>(vd) = make_float4(v8[u][0], v8[u][1], v8[u][2], v8[u][3]);
        *reinterpret_cast<float4*>(vd + 4) = make_float4(v8[u][4], v8[u][5], v8[u][6], v8[u][7]);
      }
    } else {
      for (int x = tid; x < 2 * KC * dh4; x += 256) {
        const int rr = x / dh4, d = x - rr * dh4;
        const int j = j0 + (rr & (KC - 1));
        float kv = 0.0f, vv = 0.0f;
        if (j < q && d < dh) {
          if (rr < KC) {
            kv = to_f32(kl[(long long)j * kw + d]);
            vv = to_f32(vl[(long long)j * kw + d]);
          } else {
            const EK* mj = ml + (long long)j * 2 * d_kv;
            kv = to_f32(mj[d]);
            vv = to_f32(mj[d_kv + d]);
          }
        }
        ks[rr * KS + d] = kv;
        vs[rr * DHM + d] = vv;
      }
    }
    __syncthreads();

    // scores of this wave's rows against key `lane` of the chunk
    float s[RW];
#pragma unroll
    for (int r = 0; r < RW; ++r) s[r] = 0.0f;
    const float* kr = ks + lane * KS;
    const float* qr = qs + wave * RW * DHM;
    for (int d = 0; d < dh4; d += 4) {
      const float k0 = kr[d], k1 = kr[d + 1], k2 = kr[d + 2], k3 = kr[d + 3];
#pragma unroll
      for (int r = 0; r < RW; ++r) {
        const float4 qv = *reinterpret_cast<const float4*>(qr + r * DHM + d);
        s[r] += qv.x * k0 + qv.y * k1 + qv.z * k2 + qv.w * k3;
      }
    }
    const int j = j0 + (lane & (KC - 1));
    float p[RW];
#pragma unroll
    for (int r = 0; r < RW; ++r) {
      const float sv = j <= row[r] ? s[r] : -INFINITY;
      float mx = sv;
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) mx = fmaxf(mx, __shfl_xor(mx, off, 64));
      const float mn = fmaxf(m[r], mx);  // finite: key 0 is in every row's first chunk
      const float c = __expf(m[r] - mn);
      p[r] = __expf(sv - mn);
      float ps = p[r];
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) ps += __shfl_xor(ps, off, 64);
      lsum[r] = lsum[r] * c + ps;
#pragma unroll
      for (int t = 0; t < NT; ++t) acc[r][t] *= c;
      m[r] = mn;
    }
    // weighted sum: value row L of the chunk (the key of lane L) with weight p of lane L
    for (int L = 0; L < 2 * KC; ++L) {
      float pb[RW];
#pragma unroll
      for (int r = 0; r < RW; ++r)
        pb[r] = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(p[r]), L));
      const float* vr = vs + L * DHM;
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        const int d = lane + 64 * t;
        if (d < dh) {
          const float vv = vr[d];
#pragma unroll
          for (int r = 0; r < RW; ++r) acc[r][t] += pb[r] * vv;
        }
      }
    }
  }
#pragma unroll
  for (int r = 0; r < RW; ++r) {
    const int i = i0 + wave * RW + r;
    if (i >= q) continue;
    EO* oi = out + ((long long)l * q + i) * qw + (long long)a * dh;
    const float inv = 1.0f / lsum[r];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const int d = lane + 64 * t;
      if (d < dh) oi[d] = from_f32<EO>(acc[r][t] * inv);
    }
  }
}

}  // namespace
}  // namespace mone
