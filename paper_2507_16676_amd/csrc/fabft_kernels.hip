// Flash-ABFT attention forward for gfx950 (MI355X).
//
// One pass over the keys per query tile (FlashAttention-2, Algorithm 2 of
// arXiv 2507.16676) with the online checksum of Algorithm 3 fused in:
//   s = scale * q.k; m_new = max(m, s); alpha = exp(m - m_new)
//   l = l*alpha + sum exp(s - m_new); o = o*alpha + sum exp(s - m_new) v
//   c = c*alpha + sum exp(s - m_new) sumrow(V)            (Alg. 3, Eq. 9)
// then O = o / l, pred = c / l (Eq. 8) and the per-row check against
// actual = sum_j O_ij.
//
// Dataflow. One workgroup = 8 waves = 256 query rows (one workgroup per CU,
// two waves per SIMD; at d = 256, 4 waves and one); one wave = 32 rows; key
// tiles of 64 keys.
//  * The 32x32x16 bf16 MFMA computes S^T = K Q^T (keys on the M side, the
//    wave's 32 queries on the N side) and O^T = V^T P^T. With this
//    orientation a lane holds values of a single query row, so the row max,
//    the sums l and c, the alpha rescale and the final row sum are in-lane
//    work plus one exchange between lane i and lane i+32 (permlane32 swap).
//  * Q stays in VGPRs as MFMA B operands for the whole pass.
//  * K and V tiles go from global memory straight into a 4-stage LDS ring
//    (buffer_load_dwordx4 ... lds: lane l of a load lands at base + 16 l), three
//    tiles ahead of use, with no register staging. Both tiles are stored
//    row-major with their 16-byte chunks XOR-swizzled by row: the K
//    swizzle makes the MFMA operand reads conflict-free, the V swizzle makes
//    the transposed reads conflict-free.
//  * The V^T operand of the P V MFMA comes from row-major V through the
//    transposing LDS read ds_read_b64_tr_b16: in a 16-lane group, lane r
//    receives element r%4 of the 8-byte loads of lanes 4e + r/4 (e = 0..3);
//    when lane 4e+q loads V[key0+e][col0+4q .. +3], lane r gets column
//    col0+r of keys key0..key0+3, i.e. 4 k-slots of the MFMA A operand.
//  * The K rows feeding MFMA row r are permuted (bits 2 and 3 of r swapped)
//    so that the S^T accumulator of a lane already holds, for each 16-key
//    step of P V, the 8 consecutive keys its B operand needs.
//  * sumrow(V) of a key tile is computed from LDS by the workgroup (four
//    threads per key on waves 0-3, one per SIMD; fp32 via v_dot2 and a DPP
//    reduction) while the tile before it is processed,
//    and stored as a bf16 pair
//    hi + lo (hi = bf16(vs), lo = bf16(vs - hi); |vs - hi - lo| <=
//    2^-17|vs|) in an 8-row operand [sumrow hi; sumrow lo; ones; 0; weighted
//    hi; weighted lo; 0; 0]: one sum per key and tile shared by all query rows
//    of the workgroup, the paper's shared adder.
//  * The weights p~ = bf16(p) feed the P V MFMA; l and the checksum c use
//    exactly those p~, so that the rounding of P cancels between pred and
//    actual. They come from two 4x4x4 MFMAs (16 blocks) per 16-key step on
//    the same P^T register as B operand: lane 4b+j is column j of block b
//    with its own query, and lanes 4b..4b+3 supply the rows [sumrow hi;
//    sumrow lo; ones; 0] of A, so element i of a lane accumulates c_hi,
//    c_lo and l of its query over its half of the keys (4 registers;
//    lanes l and l+32 add up at the end), rescaled like o (Eq. 10 carries c
//    as an extra row of V^T). Each output column is one query, so a
//    non-finite p~ in one row cannot reach the sums of another (a 16x16x32
//    on the same register would mix the two 16-query halves of the block).
//    With the weighted check two more 4x4x4 products per 8 keys carry the
//    weighted sums (rows [weighted hi; weighted lo; 0; 0]) in 4 more
//    registers; c and l come out the same either way.
//  * Masking (causal diagonal tiles, the ragged last tile) sets a score to
//    -inf, whose exponential is exactly 0.
//  * Persistent launch (optional): one workgroup per CU runs a
//    list of (head, query tile) items; when an item has a multiple of four
//    key tiles, the next item's first tiles load into the ring during its
//    last steps and its Q during the epilogue.
//  * Lazy rescaling: the running max used for the exponentials is moved only
//    when a tile's max exceeds it by more than 8 in the exp2 domain, so
//    p <= 256 and o, l, c are rescaled (alpha != 1) rarely; o*alpha is
//    skipped when no lane of the wave moved its max. o/l and c/l are
//    unchanged in exact arithmetic (the shift cancels).
//  * Algorithm 1 as the host of the checksum (optional): a first pass loads
//    K only and takes each row's max score over all its keys; the second is
//    the loop above with the running max preset to that value, so alpha
//    stays 1 and nothing is rescaled.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <atomic>
#include <climits>

#include "fabft_kernels.h"

// This file is compiled twice. Part 0 holds everything except the d = 128
// forward kernels without the weighted check; part 1 holds only those and
// is built with LLVM's iterative ILP scheduler, measured 2-3% faster for
// them (and 2-4% slower at d = 64, which therefore stays in part 0). A
// kernel is instantiated in one part only.
#ifndef FABFT_PART
#define FABFT_PART 0
#endif

namespace fabft {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

// Workgroup shape per row width D: WAVES waves of 32 query rows, an LDS ring
// of STAGES key tiles, AHEAD of them loading while one is in use. D = 256
// runs one wave per SIMD (512 registers for its 256-wide Q and o fragments)
// and a 2-stage ring (64 KiB per stage). D = 64 runs 8 waves like D = 128
// with a 4-stage ring of 69 KiB; sumrow there is taken once per key tile for
// 256 query rows rather than twice for two 4-wave workgroups of 128 rows
// each (7-8% faster with the checksum on 2,048- and 4,096-key rows; on
// 512-key rows the persistent launch makes up for the longer start-up).
template <int D>
struct Cfg {
  static constexpr int WAVES = (D == 256) ? 4 : 8;
  static constexpr int THREADS = 64 * WAVES;
  static constexpr int BR = 32 * WAVES;
  static constexpr int STAGES = D == 256 ? 2 : 4;
  static constexpr int AHEAD = STAGES - 1;
  static_assert(BR == query_tile_for(D), "query rows per workgroup");
};
constexpr int kBc = 64;                  // keys per tile
#ifndef FABFT_CAUSAL_BAND
#define FABFT_CAUSAL_BAND 4
#endif
constexpr int kCausalBand = FABFT_CAUSAL_BAND;  // heads per XCD in flight at once (causal)
constexpr float kLazy = 8.0f;            // max drift (exp2 domain) before a rescale
constexpr uint32_t kOnes = 0x3f803f80u;  // bf16 pair (1.0, 1.0)
constexpr uint32_t kAlt = 0xbf803f80u;   // bf16 pair (1.0, -1.0): weights (-1)^j

__device__ __forceinline__ f32x16 mfma32(u32x4 a, u32x4 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(
      __builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

// 16 independent 4x4x4 bf16 products: block b = lane / 4 takes A row i from
// lane 4b + i and B column j from lane 4b + j (4 k values each) and leaves
// D[i][j] in element i of lane 4b + j (checked with a probe on gfx950)
__device__ __forceinline__ f32x4 mfma4(u32x2 a, u32x2 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_4x4x4bf16_1k(__builtin_bit_cast(s16x4, a),
                                               __builtin_bit_cast(s16x4, b), c, 0, 0, 0);
}

// a.lo*b.lo + a.hi*b.hi + c on packed bf16 pairs, fp32 accumulate
__device__ __forceinline__ float dot2(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, a),
                                         __builtin_bit_cast(bf16x2, b), c, false);
}

// DPP lane permutations (update_dpp with every row and bank enabled)
template <int CTRL>
__device__ __forceinline__ float dpp(float x) {
  return __int_as_float(
      __builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, false));
}

// Sum over aligned groups of N (4 or 8) consecutive lanes; every lane of
// the group receives the same value.
template <int N>
__device__ __forceinline__ float group_sum(float x) {
  static_assert(N == 4 || N == 8, "group size");
  x += dpp<0xB1>(x);   // quad_perm [1,0,3,2]
  x += dpp<0x4E>(x);   // quad_perm [2,3,0,1]
  if constexpr (N == 8) x += dpp<0x141>(x);  // row_half_mirror
  return x;
}

// Combine the values of lanes i and i ^ 32 with a symmetric operation:
// v_permlane32_swap leaves (own, partner) in the two results of every lane.
__device__ __forceinline__ float sum_xor32(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float max_xor32(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __builtin_fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  f32x2 f = {a, b};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, bf16x2));
}

// The bits of x, opaque to the optimiser. This file is built with relaxed
// NaN rules, under which the compiler may fold an exponent-bits test of a
// float into "is infinite" and drop the NaN case; the asm keeps the test on
// the actual bits.
__device__ __forceinline__ uint32_t opaque_bits(float x) {
  uint32_t b = __float_as_uint(x);
  asm volatile("" : "+v"(b));
  return b;
}
__device__ __forceinline__ bool nonfinite_bits(float x) {
  return (opaque_bits(x) & 0x7f800000u) == 0x7f800000u;
}

// Row r of an MFMA 32-row block reads key 16*(r>>4) + 8*((r>>2)&1) + 4*((r>>3)&1) + (r&3)
__device__ __forceinline__ int swap_bits23(int r) {
  return (r & ~12) | ((r & 4) << 1) | ((r & 8) >> 1);
}

// s_waitcnt vmcnt(n) (expcnt and lgkmcnt left unconstrained), n < 16
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 16, "vmcnt range");
  __builtin_amdgcn_s_waitcnt(N | (0x7 << 4) | (0xF << 8));
}

// buffer_load_dwordx4 ... lds through a buffer resource (base, size in
// bytes): the 16 bytes at byte offset voff + soff of lane l land at LDS
// address lds + 16 l (lds is wave-uniform and goes through m0), and a load at
// or past the size reads zeros. The per-lane offsets stay fixed while the
// tile moves in the scalar soff, so issuing a tile costs no vector
// instruction, and rows past the end of K and V need no clamping.
// Inline asm: the compiler does not see this load, so it adds no wait of its
// own before LDS reads (its tracking of the builtin form makes every
// transposed V read wait for all outstanding loads, the prefetched tiles
// included); wait_vmcnt and the workgroup barrier order these loads before
// their readers. For the same reason it inserts no hazard wait states before
// the asm: a vector instruction that writes an SGPR (v_readfirstlane, or
// v_readlane restoring a spilled descriptor) needs 5 wait states before a
// memory instruction reads that SGPR, so the asm starts with s_nop 4 (which
// also covers the write of m0 before an LDS transfer).
typedef int i32x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ i32x4 buffer_rsrc(const void* base, uint32_t bytes) {
  const uint64_t a = (uint64_t)(uintptr_t)base;
  i32x4 r;
  r[0] = __builtin_amdgcn_readfirstlane((int)(uint32_t)a);
  r[1] = __builtin_amdgcn_readfirstlane((int)((a >> 32) & 0xffffu));   // stride 0
  r[2] = __builtin_amdgcn_readfirstlane((int)bytes);
  r[3] = 0x00020000;   // 32-bit data format, raw (offset) addressing
  return r;
}
__device__ __forceinline__ void buffer_load_lds16(i32x4 rsrc, uint32_t voff, uint32_t soff,
                                                  uint32_t lds) {
  const uint32_t base = __builtin_amdgcn_readfirstlane(lds);
  const uint32_t so = __builtin_amdgcn_readfirstlane(soff);
  asm volatile("s_nop 4\n\tbuffer_load_dwordx4 %0, %1, %2 offen lds"
               : : "v"(voff), "s"(rsrc), "s"(so), "{m0}"(base) : "memory");
}

// Tile layouts in LDS. A tile row (one key) holds D bf16 = CPR 16-byte
// chunks; logical chunk c of row r is stored at chunk c ^ swz(r).
template <int D>
struct Tile {
  static constexpr int CPR = D / 8;
  // K: 16 lanes read 16 different rows at one logical chunk
  static __device__ __forceinline__ int kswz(int r) { return D == 128 ? (r & 15) : ((r >> 1) & 7); }
  // V: 32 lanes read 4 consecutive rows x 4 consecutive chunks
  static __device__ __forceinline__ int vswz(int r) { return D == 128 ? 4 * (r & 3) : 4 * ((r >> 1) & 1); }
  static __device__ __forceinline__ int kidx(int r, int c) { return r * D + 8 * (c ^ kswz(r)); }
  static __device__ __forceinline__ int vidx(int r, int c) { return r * D + 8 * (c ^ vswz(r)); }
};

// Rows of the small A operand that yields c and l: sumrow(V) as bf16 hi and
// lo parts, ones, zeros, and the weighted row sums sum_j (-1)^j V_kj as hi
// and lo parts, padded to 8 rows. Lane 4b + i of a 4x4x4 product reads row i
// (VsHi, VsLo, Ones, Zero), for the weighted sums WHi, WLo, Zero, Zero: one
// wave-wide 16-byte load per 16 keys. Below d = 256 a row holds the tile's 64
// keys plus 8 unused ones: with 144-byte rows, rows 0-3 start 36 banks apart
// and one read touches no bank twice (128-byte rows put rows 0 and 2, and 1
// and 3, on the same banks). At d = 256 (one wave per SIMD, LDS for two
// 64 KiB stages) the rows stay 128 bytes.
enum { kRowVsHi = 0, kRowVsLo = 1, kRowOnes = 2, kRowZero = 3, kRowWHi = 4, kRowWLo = 5,
       kVsmRows = 8 };

// The ring's K tiles, then its V tiles, then the small operands: with the
// stage a compile-time constant, every operand read of a tile is a per-lane
// base register plus an immediate offset (K and V stages each span 64 KiB at
// d = 128, the reach of the LDS offset field).
template <int D>
struct Ring {
  static constexpr int VS = D == 256 ? kBc : kBc + 8;   // vsm row stride (keys)
  uint16_t k[Cfg<D>::STAGES][kBc * D];
  uint16_t v[Cfg<D>::STAGES][kBc * D];
  uint16_t vsm[Cfg<D>::STAGES][kVsmRows][VS];
};

// ---- work items: (head bh, query tile qt) pairs, p.n_items of them.
// Item of block vb when each workgroup runs one item. Workgroups go to the 8
// XCDs round robin (XCD = id mod 8). Without a mask every item costs the
// same: each XCD takes a contiguous range of heads, so that a head's K and V
// stay in one L2. With the causal mask the work of a query tile grows with
// its index: the heaviest tiles go first (longest job first), a band of
// heads at a time, and with a head count divisible by 8 a head stays on one
// XCD.
template <bool CAUSAL>
__device__ __forceinline__ void item_of_block(const FwdParams& p, int vb, int& bh, int& qt) {
  const int G = p.n_items;
  if (CAUSAL) {
    const int BH = G / p.n_qt;
    if ((BH & 7) == 0) {
      // XCD x owns heads x, x + 8, ...; it runs them a band of heads at a
      // time, each band longest tile first. The query tiles of a band stream
      // the same few K/V tiles at about the same time, so one HBM read
      // serves several of them from L2. A band holds as few heads as still
      // give the XCD's 32 CUs at least 64 query tiles (at most kCausalBand):
      // with long rows one head suffices, and all of an XCD's tiles then
      // share one head's K/V.
      const int bandw = min(kCausalBand, max(1, (64 + p.n_qt - 1) / p.n_qt));
      const int xcd = vb & 7, slot = vb >> 3;
      const int band = slot / (bandw * p.n_qt);
      const int h0 = band * bandw;
      const int nb = min(bandw, (BH >> 3) - h0);
      const int w = slot - h0 * p.n_qt;
      const int qr = w / nb;
      bh = (h0 + w - qr * nb) * 8 + xcd;
      qt = p.n_qt - 1 - qr;
    } else {
      const int qr = vb / BH;
      bh = vb - qr * BH;
      qt = p.n_qt - 1 - qr;
    }
  } else {
    const int xcd = vb & 7;
    const int per = G >> 3, rem = G & 7;
    const int slot = vb >> 3;
    const int logical = (xcd < rem) ? xcd * (per + 1) + slot
                                    : rem * (per + 1) + (xcd - rem) * per + slot;
    bh = logical / p.n_qt;
    qt = logical - bh * p.n_qt;
  }
}

// Item k of workgroup b when p.grid workgroups (a multiple of 8, one or two
// per CU) each run a list of items; false past the end of b's list.
// Workgroup b runs on XCD b mod 8 and takes only that XCD's items, in the
// one-item order (slot by slot): the XCD's G/8 workgroups deal its slots in
// rounds of G/8, every other round in reverse order. With the mask the slots
// of a band come heaviest first, so a workgroup's heavy tile of one round
// meets a light one in the next and the workgroups get about the same number
// of key tiles; the band's heads are still the ones in flight (the host takes
// this path with the mask only for a head count divisible by 8).
template <bool CAUSAL>
__device__ __forceinline__ bool persistent_item(const FwdParams& p, int b, int k, int& bh,
                                                int& qt) {
  const int G = p.grid;
  if (!CAUSAL) {
    const long long vb = (long long)b + (long long)k * G;
    if (vb >= p.n_items) return false;
    item_of_block<false>(p, (int)vb, bh, qt);
    return true;
  }
  const int nw = G >> 3, wx = b >> 3;
  const long long slot = (long long)k * nw + ((k & 1) ? nw - 1 - wx : wx);
  if (slot >= (p.n_items >> 3)) return false;
  item_of_block<true>(p, (int)(slot * 8 + (b & 7)), bh, qt);
  return true;
}

template <int S>
struct StageId {
  static constexpr int value = S;
};

// WCHK: the weighted second checksum is compiled in (only with CHECK).
// SPLIT: the workgroup runs one key split and writes partial row states.
// SCHK: the score check is compiled in (only with CHECK, not with SPLIT).
// TWOPASS: Algorithm 1 hosts the checksum: a first pass over K takes each
// row's max, the second runs the loop with that max fixed (only with CHECK).
template <int D, bool CAUSAL, bool CHECK, bool INJECT, bool WCHK, bool SPLIT, bool SCHK = false,
          bool TWOPASS = false>
__global__ __launch_bounds__(Cfg<D>::THREADS, 1) void fwd_kernel(FwdParams p) {
  constexpr int kWaves = Cfg<D>::WAVES;
  constexpr int kThreads = Cfg<D>::THREADS;
  constexpr int kBr = Cfg<D>::BR;
  constexpr int kStages = Cfg<D>::STAGES;
  constexpr int AHEAD = Cfg<D>::AHEAD;
  constexpr int BC = kBc;
  constexpr int CPR = Tile<D>::CPR;
  constexpr int NKB = BC / 32;    // 32-key blocks per tile
  constexpr int NDB = D / 32;     // 32-column blocks of the output
  constexpr int NDS = D / 16;     // 16-wide steps over d in Q K^T
  constexpr int NLD = BC * CPR / kThreads;   // 16-byte loads per thread per tensor and tile
  static_assert(NLD >= 1 && BC * CPR == NLD * kThreads, "loads cover the tile");
  // a workgroup may run a list of items (p.persist), handing the LDS ring
  // from one item to the next: the next item's Q and first key tiles load
  // while the current item's last tiles and epilogue run
  constexpr bool kPersist = !INJECT && !SPLIT && !SCHK && !TWOPASS && Cfg<D>::AHEAD >= 3;

  __shared__ __attribute__((aligned(16))) Ring<D> ring;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
  const int mrow = lane & 31;   // MFMA row / column index of this lane
  const int grp = lane >> 5;    // which 8-wide k slice this lane holds

  // ---- this workgroup's first item
  const int bid = blockIdx.x;
  int bh = 0, qt = 0, split = 0;
  if constexpr (SPLIT) {
    // the splits of one (head, query tile) are neighbours
    split = bid % p.nsplit;
    const int lg = bid / p.nsplit;
    bh = lg / p.n_qt;
    qt = lg - bh * p.n_qt;
  } else if (kPersist && p.persist) {
    if (!persistent_item<CAUSAL>(p, bid, 0, bh, qt)) return;   // nothing to do
  } else {
    item_of_block<CAUSAL>(p, bid, bh, qt);
  }
  // wave-uniform (for the compiler's divergence analysis: scalar registers)
  bh = __builtin_amdgcn_readfirstlane(bh);
  qt = __builtin_amdgcn_readfirstlane(qt);

  const int Lq = p.Lq, Lk = p.Lk;
  const int off = Lk - Lq;
  // q, k, v, o rows hold DIO <= D columns in memory; on chip the rows are D
  // wide and columns DIO.. are zero (zero scores, zero outputs)
  const int DIO = p.dio;
  const int CIO = DIO / 8;   // 16-byte chunks per row in memory
  const uint32_t kv_bytes = (uint32_t)Lk * DIO * 2;
  // key tiles of query tile qt_ (keys [0, kend)); wave-uniform (the
  // division runs on the vector ALU): scalar branches
  auto tiles_of = [&](int qt_) {
    int kend = Lk;
    if (CAUSAL) kend = min(Lk, qt_ * kBr + kBr + off);
    return __builtin_amdgcn_readfirstlane(kend > 0 ? (kend + BC - 1) / BC : 0);
  };

  // ---- the current item: key tiles [t_lo, t_end), this wave's first query
  // row wq_lo, the lane's row qrow, and the head's K / V buffer resources
  int t_lo = 0, t_end = 0, wq_lo = 0, qrow = 0;
  size_t qbase = 0;
  i32x4 krs, vrs;
  auto set_item = [&]() {
    const int ntiles = tiles_of(qt);
    t_lo = 0;
    t_end = ntiles;
    if (SPLIT) {
      t_lo = min(ntiles, split * p.split_tiles);
      t_end = min(ntiles, t_lo + p.split_tiles);
    }
    wq_lo = qt * kBr + 32 * wave;
    qrow = wq_lo + mrow;
    qbase = (size_t)bh * (size_t)Lq * DIO;
    const size_t kbase = (size_t)bh * (size_t)Lk * DIO;
    krs = buffer_rsrc(p.k + kbase, kv_bytes);
    vrs = buffer_rsrc(p.v + kbase, kv_bytes);
  };
  set_item();
  // ---- the next item of a persistent workgroup: head, query tile, key
  // tiles, K / V resources; cont: its first AHEAD tiles go into the ring
  // during the current item's last tiles (the current item has a multiple of
  // kStages tiles, so the next one starts in stage 0); te_v: the end of the
  // tiles in flight, for the waits
  int nbh = 0, nqt = 0, n_tend = 0, te_v = 0;
  bool cont = false;
  i32x4 krsN = {}, vrsN = {};

  // ---- Q fragments (B operand): lane holds query qrow, d slice 8*grp
  u32x4 qf[NDS];
  auto load_q = [&](int bh_, int qt_) __attribute__((always_inline)) {
    const int r = qt_ * kBr + 32 * wave + mrow;
    const uint16_t* qr = p.q + (size_t)bh_ * (size_t)Lq * DIO + (size_t)r * DIO;
#pragma unroll
    for (int s = 0; s < NDS; ++s) {
      qf[s] = u32x4{0, 0, 0, 0};
      if (r < Lq && 2 * s + grp < CIO) qf[s] = *reinterpret_cast<const u32x4*>(qr + 16 * s + 8 * grp);
    }
  };
  load_q(bh, qt);

  f32x16 oacc[NDB];
  // c / l accumulator of this lane's query: [0] c_hi, [1] c_lo, [2] l over
  // the lane's half of the keys (4x4x4 products; the two halves add up at
  // the end); with the weighted check, auxw [0] c_w hi, [1] c_w lo alike
  f32x4 aux, auxw;
  float s_lhs;    // score check: sum of this lane's scores in full tiles
  // score check on masked tiles (the diagonal and ragged ones): this lane's
  // sum of its visible scores, and the same sum from a second Q K^T product
  float d_lhs, d_rhs;
  float m2_run;   // running max, exp2 domain (s * scale * log2 e)
  // Algorithm 1 (TWOPASS): pass 0 streams K only and takes each row's max
  // over all its keys (m_acc, score units); pass 1 is the loop below with the
  // running max fixed at that value, so no rescale ever happens (alpha = 1).
  // One-pass kernels run pass 1 only.
  int pass = 1;
  float m_acc = -__builtin_inff();
  const float sl2 = p.sl2;

  // constant rows of the c / l operand in every stage (visible after the
  // first barrier)
  for (int e = tid; e < kStages * 2 * BC; e += kThreads) {
    const int st_i = e / (2 * BC), row = kRowOnes + (e / BC) % 2, key = e % BC;
    ring.vsm[st_i][row][key] = row == kRowOnes ? (uint16_t)0x3f80 : (uint16_t)0;
  }
  // row of the c / l operand that MFMA row mrow reads (rows 0, 1 only with
  // the checksum, rows 8, 9 only with the weighted one)
  // 4x4x4 form: lane 4b + i supplies row i of block b's A: sumrow hi, lo,
  // ones, zeros (the c rows read zeros without the checksum); for the
  // weighted sums, weighted hi, lo, zeros, zeros
  const int vsm_row4 = (lane & 3) == 2 ? (int)kRowOnes
                       : (!CHECK || (lane & 3) == 3) ? (int)kRowZero
                                                     : (lane & 3);
  const int vsm_roww = (lane & 3) < 2 ? (int)kRowWHi + (lane & 3) : (int)kRowZero;

  // ---- loader: 16-byte slot j*512 + tid of a tile holds row slot/CPR, stored
  // chunk slot%CPR (logical chunk = stored ^ swz(row)); rows past Lk read as
  // zeros (the mask gives them weight 0)
  uint32_t kvo[NLD], vvo[NLD];
#pragma unroll
  for (int j = 0; j < NLD; ++j) {
    const int slot = j * kThreads + tid;
    const int row = slot / CPR, sc = slot % CPR;
    // a chunk past the row's DIO columns reads from offset kv_bytes + soff,
    // past the end of the buffer: zeros
    const int kc = sc ^ Tile<D>::kswz(row), vc = sc ^ Tile<D>::vswz(row);
    kvo[j] = kc < CIO ? (uint32_t)(row * DIO + 8 * kc) * 2 : kv_bytes;
    vvo[j] = vc < CIO ? (uint32_t)(row * DIO + 8 * vc) * 2 : kv_bytes;
  }
  // LDS byte address of the ring and of this wave's 1 KiB slot in a tile
  const uint32_t ring_lds = (uint32_t)(uintptr_t)(lds_void*)&ring;
  const uint32_t wave_lds = __builtin_amdgcn_readfirstlane(ring_lds + 1024u * wave);
  auto issue = [&](auto S_, int t) {
    constexpr int S = decltype(S_)::value;
    i32x4 kr = krs, vr = vrs;
    if (t >= t_end) {
      if constexpr (!kPersist) {
        return;
      } else {
        // tile t - t_end of the next item (into the stage it starts in)
        t -= t_end;
        if (!cont || t >= n_tend) return;
        kr = krsN;
        vr = vrsN;
      }
    }
    const uint32_t soff = (uint32_t)t * BC * DIO * 2;
    // opaque copy: the destination addresses are formed here from one SGPR
    // (scalar adds) rather than hoisted as one live SGPR per stage and load
    uint32_t wl = wave_lds;
    asm volatile("" : "+s"(wl));
#pragma unroll
    for (int j = 0; j < NLD; ++j) {
      // each wave writes its own contiguous 1 KiB of the stage
      constexpr uint32_t kOff = offsetof(Ring<D>, k) + S * sizeof(Ring<D>::k[0]);
      constexpr uint32_t vOff = offsetof(Ring<D>, v) + S * sizeof(Ring<D>::v[0]);
      buffer_load_lds16(kr, kvo[j], soff, wl + kOff + j * kThreads * 16);
      if (!TWOPASS || pass != 0) buffer_load_lds16(vr, vvo[j], soff, wl + vOff + j * kThreads * 16);
    }
  };

  // ---- sumrow(V) of the tile in stage S (Eq. 4): TPK threads per key on
  // the first SW waves. Only waves 0-3 (one per SIMD) take it, four threads
  // per key: with 8 waves every SIMD spends one wave's vector instructions
  // on it rather than two (the sums are the same work either way; the
  // per-key reduction and the hi / lo split are paid once per four lanes
  // instead of eight).
  auto sumrow = [&](auto S_) __attribute__((always_inline)) {
    constexpr int S = decltype(S_)::value;
    constexpr int SW = 4;                         // waves taking part
    constexpr int TPK = 64 * SW / BC;             // threads per key
    constexpr int CPT = CPR / TPK;                // 16-byte chunks per thread
    static_assert(TPK * BC == 64 * SW && CPT * TPK == CPR, "sumrow covers the tile");
    if constexpr (SW < kWaves) {
      if (wave >= SW) return;                     // wave-uniform
    }
    const uint16_t* const sv = ring.v[S];
    uint16_t(*const svsm)[Ring<D>::VS] = ring.vsm[S];
    const int key = tid / TPK, part = tid % TPK;
    float a = 0.f, aw = 0.f;
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
      // at d = 128: chunk part + 4 i. A 16-lane read pass covers keys
      // 4m .. 4m+3 (parts 0-3 each); the V swizzle stores logical chunk c of
      // key r at c ^ 4(r mod 4), so the pass reads 16 distinct chunks of the
      // 256-byte rows: no bank conflict. At d = 64: chunk part + 4 j,
      // j = i ^ (key mod 2), so that the keys of one pass take opposite
      // halves of the row, whose banks the V swizzle keeps apart. d = 256
      // reads CPT consecutive chunks.
      const int c = D == 128 ? part + TPK * i
                  : CPT == 2 ? part + TPK * (i ^ (key & 1)) : CPT * part + i;
      const u32x4 ch = *reinterpret_cast<const u32x4*>(&sv[Tile<D>::vidx(key, c)]);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        a = dot2(ch[e], kOnes, a);
        // a chunk starts at an even column: pair weights (1, -1)
        if constexpr (WCHK) aw = dot2(ch[e], kAlt, aw);
      }
    }
    const float vs = group_sum<TPK>(a);
    const float vw = WCHK ? group_sum<TPK>(aw) : 0.f;
    if (part == 0) {
      const uint32_t hi = pack_bf16x2(vs, 0.f) & 0xffffu;
      const uint32_t lo = pack_bf16x2(vs - __uint_as_float(hi << 16), 0.f) & 0xffffu;
      svsm[kRowVsHi][key] = (uint16_t)hi;
      svsm[kRowVsLo][key] = (uint16_t)lo;
      if constexpr (WCHK) {
        const uint32_t whi = pack_bf16x2(vw, 0.f) & 0xffffu;
        const uint32_t wlo = pack_bf16x2(vw - __uint_as_float(whi << 16), 0.f) & 0xffffu;
        svsm[kRowWHi][key] = (uint16_t)whi;
        svsm[kRowWLo][key] = (uint16_t)wlo;
      }
    }
  };

  // ---- one key tile for this wave (steps A1-A5)
  auto compute = [&](auto S_, int t) {
    constexpr int S = decltype(S_)::value;
    const uint16_t* const sk = ring.k[S];
    const uint16_t* const sv = ring.v[S];
    const uint16_t(*const svsm)[Ring<D>::VS] = ring.vsm[S];
    const int kv0 = t * BC;
    const bool need_mask = (kv0 + BC > Lk) || (CAUSAL && kv0 + BC - 1 > wq_lo + off);

    if constexpr (INJECT) {
      // Q site: bit of q_ij in the registers of row i, flipped before the
      // Q K^T of tile f_tile; the flipped value stays for the later tiles
      // (lane grp holds columns 16s + 8grp .. +7 of its row)
      for (int fi = 0; fi < p.nf; ++fi) {
        const FaultDesc fd = p.f[fi];
        if (fd.site == 8 && pass == 1 && bh == fd.bh && qrow == fd.row && t == fd.tile &&
            ((fd.col >> 3) & 1) == grp) {
          const int sj = fd.col >> 4, e = (fd.col & 7) >> 1;
          const uint32_t mask = (1u << fd.bit) << (16 * (fd.col & 1));
#pragma unroll
          for (int s2 = 0; s2 < NDS; ++s2)
#pragma unroll
            for (int ee = 0; ee < 4; ++ee)
              if (s2 == sj && ee == e) qf[s2][ee] ^= mask;
        }
      }
    }
    // S^T = K Q^T (Alg. 3: s_i = q . k_i)
    f32x16 sacc[NKB];
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb) sacc[kb] = f32x16{};
    const int krow = swap_bits23(mrow);
    // operand reads run KAHEAD MFMAs ahead of their use (the scheduling
    // barriers keep the compiler from pulling them back next to the MFMA)
    constexpr int NQK = NDS * NKB, KAHEAD = 6;
    auto kread = [&](int i) {
      return *reinterpret_cast<const u32x4*>(
          &sk[Tile<D>::kidx((i % NKB) * 32 + krow, 2 * (i / NKB) + grp)]);
    };
    u32x4 kop[NQK];
#pragma unroll
    for (int i = 0; i < KAHEAD; ++i) kop[i] = kread(i);
#pragma unroll
    for (int i = 0; i < NQK; ++i) {
      __builtin_amdgcn_sched_barrier(0);
      if (i + KAHEAD < NQK) kop[i + KAHEAD] = kread(i + KAHEAD);
      sacc[i % NKB] = mfma32(kop[i], qf[i / NKB], sacc[i % NKB]);
    }
    __builtin_amdgcn_sched_barrier(0);
    // accumulator element i of block kb holds key kv0 + 32kb + 16(i/8) + 8grp + (i%8)
    if constexpr (INJECT) {
      for (int fi = 0; fi < p.nf; ++fi) {
        const FaultDesc fd = p.f[fi];
        if (fd.site == 1 && pass == 1 && bh == fd.bh && qrow == fd.row) {
          const int kl = fd.col - kv0;
          if (kl >= 0 && kl < BC && ((kl >> 3) & 1) == grp) {
            const int kb = kl >> 5, i = ((kl >> 4) & 1) * 8 + (kl & 7);
#pragma unroll
            for (int b = 0; b < NKB; ++b)
#pragma unroll
              for (int e = 0; e < 16; ++e)
                if (b == kb && e == i)
                  sacc[b][e] = __uint_as_float(__float_as_uint(sacc[b][e]) ^ (1u << fd.bit));
          }
        }
      }
    }

    if constexpr (SCHK) {
      // score check: sum of the scores of full (unmasked) tiles as they
      // enter the softmax (Section II's row checksum of a matrix product,
      // applied to S = Q K^T)
      if (!need_mask) {
#pragma unroll
        for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
          for (int i = 0; i < 16; ++i) s_lhs += sacc[kb][i];
      }
    }
    // mask, tile max (Alg. 3: m_i = max(m_{i-1}, s_i)). A masked score is
    // -inf, so its exponential below is exactly 0.
    if (need_mask) {
      // last visible key of the row (past Lk, or past the diagonal), relative
      // to this lane's first key of the tile
      int lim = Lk - 1;
      if (CAUSAL) lim = min(lim, qrow + off);
      const int rel = lim - (kv0 + 8 * grp);
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const bool hidden = 32 * kb + 16 * (i >> 3) + (i & 7) > rel;
          if constexpr (SCHK) d_lhs += hidden ? 0.f : sacc[kb][i];
          if (hidden) sacc[kb][i] = -__builtin_inff();
        }
    }
    // one chain of three-input maxima (v_max3): one instruction per two scores
    float mx = __builtin_fmaxf(sacc[0][0], sacc[0][1]);
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
      for (int i = (kb == 0 ? 2 : 0); i < 16; i += 2)
        mx = __builtin_fmaxf(__builtin_fmaxf(mx, sacc[kb][i]), sacc[kb][i + 1]);
    mx = max_xor32(mx);
    if constexpr (TWOPASS) {
      if (pass == 0) {
        m_acc = __builtin_fmaxf(m_acc, mx);
        return;
      }
    }
    // lazy running max in the exp2 domain
    const float mt2 = (mx == -__builtin_inff()) ? -__builtin_inff() : mx * sl2;
    const float m2_new = (mt2 > m2_run + kLazy) ? mt2 : m2_run;
    const float alpha = (m2_new == m2_run) ? 1.f : __builtin_amdgcn_exp2f(m2_run - m2_new);
    m2_run = m2_new;
    const float nm2 = (m2_new == -__builtin_inff()) ? 0.f : -m2_new;

    // p = exp(s - m) and p~ = bf16(p), the B operands of P V. With kLateP
    // (d = 64, where the vector ALU sets the pace) only the first 32-key
    // block is taken here; the second block's exponentials, packs and c / l
    // products run between the first block's P V products below, so that a
    // wave's matrix and vector work overlap (measured 1% faster at 512 keys,
    // and 1-2% slower at d = 128). The same operations on the same values
    // either way: the results are bitwise the same.
    constexpr bool kLateP = D == 64 && !INJECT && !WCHK && !SCHK;
    constexpr int NKB0 = kLateP ? 1 : NKB;   // key blocks taken here
#pragma unroll
    for (int kb = 0; kb < NKB0; ++kb)
#pragma unroll
      for (int i = 0; i < 16; ++i)
        sacc[kb][i] = __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[kb][i], sl2, nm2));
    u32x4 pb[NKB][2];
#pragma unroll
    for (int kb = 0; kb < NKB0; ++kb)
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int e = 0; e < 4; ++e)
          pb[kb][h][e] = pack_bf16x2(sacc[kb][8 * h + 2 * e], sacc[kb][8 * h + 2 * e + 1]);
    if constexpr (INJECT) {
      // M site (checker state): the running max of the lane holding the
      // row's first key half, after this tile's exponentials
      for (int fi = 0; fi < p.nf; ++fi) {
        const FaultDesc fd = p.f[fi];
        if (fd.site == 7 && bh == fd.bh && qrow == fd.row && t == fd.tile && grp == 0)
          m2_run = __uint_as_float(__float_as_uint(m2_run) ^ (1u << fd.bit));
      }
    }

    // c = c*alpha + sumrow(V) p~ and l = l*alpha + sum p~ (Alg. 3): the
    // c / l products read p~ before the P site and the P V product
    if (__ballot(alpha != 1.f)) {
#pragma unroll
      for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int i = 0; i < 16; ++i) oacc[db][i] *= alpha;
#pragma unroll
      for (int i = 0; i < 4; ++i) aux[i] *= alpha;
      if constexpr (WCHK) {
#pragma unroll
        for (int i = 0; i < 4; ++i) auxw[i] *= alpha;
      }
    }
    // each 8-key slice of p~ in two 4x4x4 products: the lane's own query
    // is its column, so rows never mix (a non-finite p~ stays in its row)
#pragma unroll
    for (int kb = 0; kb < NKB0; ++kb)
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const u32x4 a =
            *reinterpret_cast<const u32x4*>(&svsm[vsm_row4][32 * kb + 16 * h + 8 * grp]);
        aux = mfma4(u32x2{a[0], a[1]}, u32x2{pb[kb][h][0], pb[kb][h][1]}, aux);
        aux = mfma4(u32x2{a[2], a[3]}, u32x2{pb[kb][h][2], pb[kb][h][3]}, aux);
        if constexpr (WCHK) {
          const u32x4 aw4 =
              *reinterpret_cast<const u32x4*>(&svsm[vsm_roww][32 * kb + 16 * h + 8 * grp]);
          auxw = mfma4(u32x2{aw4[0], aw4[1]}, u32x2{pb[kb][h][0], pb[kb][h][1]}, auxw);
          auxw = mfma4(u32x2{aw4[2], aw4[3]}, u32x2{pb[kb][h][2], pb[kb][h][3]}, auxw);
        }
      }
    if constexpr (INJECT) {
      // C and L sites (checker state): a part of the fp32 accumulator pair
      // c = c_hi + c_lo, or l, of the row after this tile's update
      for (int fi = 0; fi < p.nf; ++fi) {
        const FaultDesc fd = p.f[fi];
        if ((fd.site == 5 || fd.site == 6) && bh == fd.bh && qrow == fd.row && t == fd.tile &&
            grp == 0) {
          const int el = fd.site == 5 ? fd.col : 2;   // c: hi (0) or lo (1) part
#pragma unroll
          for (int i = 0; i < 4; ++i)
            if (i == el) aux[i] = __uint_as_float(__float_as_uint(aux[i]) ^ (1u << fd.bit));
        }
      }
    }
    if constexpr (INJECT) {
      for (int fi = 0; fi < p.nf; ++fi) {
        const FaultDesc fd = p.f[fi];
        if (!(fd.site == 2 && bh == fd.bh && qrow == fd.row)) continue;
        const int kl = fd.col - kv0;
        if (kl >= 0 && kl < BC && ((kl >> 3) & 1) == grp) {
          const int kb = kl >> 5, h = (kl >> 4) & 1, e = (kl & 7) >> 1;
          const uint32_t mask = (1u << fd.bit) << (16 * (kl & 1));
#pragma unroll
          for (int b = 0; b < NKB; ++b)
#pragma unroll
            for (int hh = 0; hh < 2; ++hh)
#pragma unroll
              for (int ee = 0; ee < 4; ++ee)
                if (b == kb && hh == h && ee == e) pb[b][hh][ee] ^= mask;
        }
      }
    }

    // O^T = alpha O^T + V^T P^T (Alg. 3: o = o*alpha + v * p); o was
    // rescaled above
    // transposed reads: 16-lane group G = lane/16, lane L = 4e + q in it reads
    // V[32kb + 16h + 8(G>>1) + 4t + e][32db + 16(G&1) + 4q .. +3]
    const int gq = lane >> 4, ll = lane & 15;
    const int tr_key = 8 * (gq >> 1) + (ll >> 2);
    const int tr_col = 16 * (gq & 1) + 4 * (ll & 3);
    // step i = (kb, h, db); its two transposed reads run VAHEAD steps ahead
    constexpr int NPV = NKB * 2 * NDB, VAHEAD = 4;
    auto vread = [&](int i) {
      const int kb = i / (2 * NDB), h = (i / NDB) % 2, db = i % NDB;
      u32x2 part[2];
#pragma unroll
      for (int t2 = 0; t2 < 2; ++t2) {
        const int key = 32 * kb + 16 * h + 4 * t2 + tr_key;
        const int col = 32 * db + tr_col;
        const int idx = Tile<D>::vidx(key, col >> 3) + (col & 7);
        const s16x4 r = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(sv + idx));
        part[t2] = __builtin_bit_cast(u32x2, r);
      }
      return u32x4{part[0][0], part[0][1], part[1][0], part[1][1]};
    };
    u32x4 vop[NPV];
#pragma unroll
    for (int i = 0; i < VAHEAD; ++i) vop[i] = vread(i);
#pragma unroll
    for (int i = 0; i < NPV; ++i) {
      __builtin_amdgcn_sched_barrier(0);
      if (i + VAHEAD < NPV) vop[i + VAHEAD] = vread(i + VAHEAD);
      const int kb = i / (2 * NDB), h = (i / NDB) % 2, db = i % NDB;
      oacc[db] = mfma32(vop[i], pb[kb][h], oacc[db]);
      if constexpr (kLateP) {
        // the second key block, EPM exponentials and EPM / 2 packs after
        // each P V product of the first, then its c / l products
        constexpr int HALF = NPV / NKB, EPM = 16 / HALF;
        static_assert(NKB == 2 && EPM % 2 == 0, "late p~ in pairs per product");
        if (i < HALF) {
          __builtin_amdgcn_sched_barrier(0);
#pragma unroll
          for (int j = 0; j < EPM; ++j)
            sacc[1][EPM * i + j] =
                __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[1][EPM * i + j], sl2, nm2));
#pragma unroll
          for (int j = 0; j < EPM / 2; ++j) {
            const int e2 = EPM / 2 * i + j;   // pair e2: keys 2 e2, 2 e2 + 1
            pb[1][e2 >> 2][e2 & 3] = pack_bf16x2(sacc[1][2 * e2], sacc[1][2 * e2 + 1]);
          }
          if (i == HALF - 1) {
#pragma unroll
            for (int h2 = 0; h2 < 2; ++h2) {
              const u32x4 a =
                  *reinterpret_cast<const u32x4*>(&svsm[vsm_row4][32 + 16 * h2 + 8 * grp]);
              aux = mfma4(u32x2{a[0], a[1]}, u32x2{pb[1][h2][0], pb[1][h2][1]}, aux);
              aux = mfma4(u32x2{a[2], a[3]}, u32x2{pb[1][h2][2], pb[1][h2][3]}, aux);
            }
          }
        }
      }
    }
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (INJECT) {
      // O site: accumulator element (row, col) after the P V of tile f_tile
      for (int fi = 0; fi < p.nf; ++fi) {
        const FaultDesc fd = p.f[fi];
        if (!(fd.site == 3 && bh == fd.bh && qrow == fd.row && t == fd.tile)) continue;
        const int j = fd.col;
        // output column j = 32db + 8a + 4grp + (i%4), element i = 4a + (i%4)
        if (((j >> 2) & 1) == grp) {
          const int db = j >> 5, i = 4 * ((j >> 3) & 3) + (j & 3);
#pragma unroll
          for (int b = 0; b < NDB; ++b)
#pragma unroll
            for (int e = 0; e < 16; ++e)
              if (b == db && e == i)
                oacc[b][e] = __uint_as_float(__float_as_uint(oacc[b][e]) ^ (1u << fd.bit));
        }
      }
    }
    if constexpr (SCHK) {
      // a masked tile has no per-row prefix of the K column sums, so its
      // scores are checked by a second Q K^T product (same operands and
      // instructions, summed over the same visible keys; the two sums agree
      // bit for bit unless a stored score changed). The accumulators start
      // from an opaque zero, so that the compiler keeps the second product.
      if (need_mask) {
        f32x16 r[NKB];
#pragma unroll
        for (int kb = 0; kb < NKB; ++kb) {
          r[kb] = f32x16{};
          asm volatile("" : "+v"(r[kb]));
        }
#pragma unroll
        for (int i = 0; i < NQK; ++i) r[i % NKB] = mfma32(kread(i), qf[i / NKB], r[i % NKB]);
        int lim = Lk - 1;
        if (CAUSAL) lim = min(lim, qrow + off);
        const int rel = lim - (kv0 + 8 * grp);
#pragma unroll
        for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
          for (int i = 0; i < 16; ++i)
            d_rhs += (32 * kb + 16 * (i >> 3) + (i & 7) > rel) ? 0.f : r[kb][i];
      }
    }
  };

  // ---- pipeline: AHEAD tiles loading while tile t is processed
  constexpr int LPT = 2 * NLD;   // loads per thread per tile (K and V)
  // wait until at most n (0 .. AHEAD-1) tiles of this wave's loads are in flight
  auto wait_tiles = [&](int n) __attribute__((always_inline)) {
    if constexpr (TWOPASS) {
      if (pass == 0) {   // K loads only: NLD per tile
        if constexpr (AHEAD >= 3) {
          if (n >= 2) {
            wait_vmcnt<2 * NLD>();
            return;
          }
        }
        if constexpr (AHEAD >= 2) {
          if (n == 1) {
            wait_vmcnt<NLD>();
            return;
          }
        }
        wait_vmcnt<0>();
        return;
      }
    }
    if constexpr (AHEAD >= 3) {
      if (n >= 2) {
        wait_vmcnt<2 * LPT>();
        return;
      }
    }
    if constexpr (AHEAD >= 2) {
      if (n == 1) {
        wait_vmcnt<LPT>();
        return;
      }
    }
    wait_vmcnt<0>();
  };
  // ---- the items of this workgroup (one unless p.persist)
  bool primed = false;   // the item's first tiles are already in the ring
  for (int k = 0;; ++k) {
    // tile t sits in stage (t - t_lo) % kStages; the loop below is unrolled
    // kStages times so that each copy knows its stages at compile time. With
    // three tiles ahead, sumrow of tile t+1 is taken at the end of step t
    // (its loads are waited for at the top of step t); with one tile ahead,
    // sumrow of tile t is taken in step t before the compute, behind a second
    // barrier.
    // the next item, and whether the ring passes to it
    bool has_next = false;
    cont = false;
    te_v = t_end;
    if constexpr (kPersist) {
      if (p.persist) {
        has_next = __builtin_amdgcn_readfirstlane(
                       (int)persistent_item<CAUSAL>(p, bid, k + 1, nbh, nqt)) != 0;
      }
      if (has_next) {
        nbh = __builtin_amdgcn_readfirstlane(nbh);
        nqt = __builtin_amdgcn_readfirstlane(nqt);
        n_tend = tiles_of(nqt);
        cont = t_end > t_lo && (t_end - t_lo) % kStages == 0;
        if (cont) {
          te_v = t_end + min(AHEAD, n_tend);
          const size_t kb = (size_t)nbh * (size_t)Lk * DIO;
          krsN = buffer_rsrc(p.k + kb, kv_bytes);
          vrsN = buffer_rsrc(p.v + kb, kv_bytes);
        }
      }
    }
#pragma unroll
    for (int b = 0; b < NDB; ++b) oacc[b] = f32x16{};
    aux = f32x4{};
    auxw = f32x4{};
    s_lhs = 0.f;
    d_lhs = 0.f;
    d_rhs = 0.f;
    m2_run = -__builtin_inff();
    m_acc = -__builtin_inff();
    // (unrolled: each pass is compiled with its own constant pass number)
#pragma unroll
    for (pass = TWOPASS ? 0 : 1; pass < 2; ++pass) {
      if (TWOPASS && pass == 1) m2_run = (m_acc == -__builtin_inff()) ? m_acc : m_acc * sl2;
      if (!primed && t_end > t_lo) {
        // after a previous item whose ring drained (or the first pass of
        // Algorithm 1), every wave must be done with its stages before they
        // take new tiles
        if ((kPersist && k > 0) || (TWOPASS && pass == 1)) __syncthreads();
        issue(StageId<0>(), t_lo);
        if constexpr (AHEAD >= 2) issue(StageId<1>(), t_lo + 1);
        if constexpr (AHEAD >= 3) {
          issue(StageId<2>(), t_lo + 2);
          // first tile complete; the next two may be outstanding
          wait_tiles(min(2, t_end - 1 - t_lo));
          __syncthreads();
          if constexpr (CHECK) {
            if (pass == 1) sumrow(StageId<0>());
          }
        }
      }
      // A use of Q here, on every path into the loop, puts the compiler's own
      // wait for the Q loads (vmcnt(0): it does not count the tile loads, so it
      // also waits for the first tiles) before the loop rather than inside it.
#pragma unroll
      for (int s = 0; s < NDS; ++s) asm volatile("" : : "v"(qf[s]));
      static_assert(kStages == 4 || kStages == 2, "the loop below is unrolled over the stages");
      static_assert(AHEAD == kStages - 1, "the stage of tile t-1 takes tile t+AHEAD");
      auto step = [&](auto S_, int t) __attribute__((always_inline)) {
        constexpr int S = decltype(S_)::value;
        if constexpr (AHEAD >= 3) {
          // tile t+1 complete (tile t+2 may still be in flight); after the
          // barrier every wave is done with tile t-1, whose stage takes tile t+3
          wait_tiles(min(1, te_v - 2 - t));
          __syncthreads();
        } else {
          // tile t complete; after the barrier every wave is done with tile t-1,
          // whose stage takes tile t+1, loading while tile t is processed
          wait_tiles(0);
          __syncthreads();
          issue(StageId<(S + 1) % kStages>(), t + 1);
          if constexpr (CHECK) {
            if (pass == 1) {
              sumrow(S_);
              __syncthreads();
            }
          }
        }
        if constexpr (INJECT) {
          // V site: flip a bit of V[row][col] in this workgroup's copy of the
          // tile, after its sumrow was taken and before any wave reads it; VS
          // site (checker state): the same for the tile's sumrow operand (col 0:
          // hi part, col 1: lo part). The condition is uniform over the
          // workgroup; faults apply one after another.
          bool hit = false;
          for (int fi = 0; fi < p.nf; ++fi) {
            const FaultDesc fd = p.f[fi];
            if ((fd.site == 4 || fd.site == 9) && pass == 1 && bh == fd.bh && qt == fd.tile) {
              const int key = fd.row - t * BC;
              if (key >= 0 && key < BC) {
                hit = true;
                if (tid == 0) {
                  uint16_t* e = fd.site == 4
                                    ? ring.v[S] + Tile<D>::vidx(key, fd.col >> 3) + (fd.col & 7)
                                    : &ring.vsm[S][kRowVsHi + fd.col][key];
                  *e = (uint16_t)(*e ^ (1u << fd.bit));
                }
              }
            }
          }
          if (hit) __syncthreads();
        }
        // waves whose rows see none of this tile's keys, or that hold no row
        // below Lq, skip it (they still load and take sumrow for the others)
        if (wq_lo < Lq && (!CAUSAL || t * BC <= wq_lo + 31 + off)) compute(S_, t);
        if constexpr (AHEAD >= 3) {
          issue(StageId<(S + 3) % kStages>(), t + 3);
          if constexpr (CHECK) {
            if (t + 1 < te_v && pass == 1) sumrow(StageId<(S + 1) % kStages>());
          }
        }
      };
      for (int t = t_lo; t < t_end; t += kStages) {
        step(StageId<0>(), t);
        if (t + 1 >= t_end) break;
        step(StageId<1>(), t + 1);
        if constexpr (kStages == 4) {
          if (t + 2 >= t_end) break;
          step(StageId<2 % kStages>(), t + 2);
          if (t + 3 >= t_end) break;
          step(StageId<3 % kStages>(), t + 3);
        }
      }
    }
    // the next item's Q loads while this item's epilogue runs (q is not read
    // after the last Q K^T)
    if constexpr (kPersist) {
      if (cont) load_q(nbh, nqt);
    }

    if constexpr (SPLIT) {
      // ---- partial state of each row for this key split (merged by
      // merge_kernel): m, l, c, c_w and the unnormalised o, in the same
      // exponent reference m (exp2 domain)
      const float l_p = sum_xor32(aux[2]);
      const float c_p = sum_xor32(aux[0] + aux[1]);
      const float cw_p = WCHK ? sum_xor32(auxw[0] + auxw[1]) : 0.f;
      if (qrow < Lq) {
        float* rec = p.ws + (((size_t)bh * Lq + qrow) * p.nsplit + split) * (D + 4);
        if (grp == 0) *reinterpret_cast<f32x4*>(rec) = f32x4{m2_run, l_p, c_p, cw_p};
#pragma unroll
        for (int db = 0; db < NDB; ++db)
#pragma unroll
          for (int a = 0; a < 4; ++a)
            *reinterpret_cast<f32x4*>(rec + 4 + 32 * db + 8 * a + 4 * grp) =
                f32x4{oacc[db][4 * a], oacc[db][4 * a + 1], oacc[db][4 * a + 2], oacc[db][4 * a + 3]};
      }
      return;
    }

    // ---- epilogue: O = o / l (Alg. 3), pred = c / l (Eq. 8), check
    const float l_tot = sum_xor32(aux[2]);
    const float inv = l_tot > 0.f ? 1.0f / l_tot : 0.f;
    float act = 0.f, absum = 0.f, act_w = 0.f;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const float x = oacc[db][i] * inv;
        oacc[db][i] = x;
        act += x;
        absum += __builtin_fabsf(x);
        // column 32db + 8(i/4) + 4grp + i%4 is even iff i is even
        act_w += (i & 1) ? -x : x;
      }
    if (qrow < Lq) {
      uint16_t* orow = p.o + qbase + (size_t)qrow * DIO;
#pragma unroll
      for (int db = 0; db < NDB; ++db) {
        if (32 * db >= DIO) break;   // DIO is a multiple of 32
#pragma unroll
        for (int a = 0; a < 4; ++a) {
          const u32x2 w = {pack_bf16x2(oacc[db][4 * a], oacc[db][4 * a + 1]),
                           pack_bf16x2(oacc[db][4 * a + 2], oacc[db][4 * a + 3])};
          *reinterpret_cast<u32x2*>(orow + 32 * db + 8 * a + 4 * grp) = w;
        }
      }
    }
    if constexpr (CHECK) {
      act = sum_xor32(act);
      absum = sum_xor32(absum);
      const float c_tot = sum_xor32(aux[0] + aux[1]);
      const float pred = c_tot * inv;
      const float r = pred - act;
      const float M = absum + __builtin_fabsf(pred);
      // non-finite test on the bits (this file is built with relaxed NaN rules);
      // a non-finite residual also fails the threshold comparison. An overflow
      // of sum_j |O_ij| (a huge but finite row) would make the threshold
      // infinite and pass any residual, so it counts as non-finite as well.
      bool nonfinite = nonfinite_bits(r) || nonfinite_bits(absum);
      uint8_t f = (__builtin_fabsf(r) <= p.tau_rel * M + p.tau_abs) ? 0 : 1;
      // weighted check: pred_w = c_w / l against sum_j (-1)^j O_ij (the same
      // threshold rule; |w_j| = 1 keeps M)
      float pred_w = 0.f;
      float sc_lhs = 0.f, sc_rhs = 0.f, sc_bound = 0.f;   // score check (debug outputs)
      if constexpr (WCHK) {
        act_w = sum_xor32(act_w);
        pred_w = sum_xor32(auxw[0] + auxw[1]) * inv;
        const float rw = pred_w - act_w;
        nonfinite = nonfinite || nonfinite_bits(rw);
        if (!(__builtin_fabsf(rw) <= p.tau_rel * (absum + __builtin_fabsf(pred_w)) + p.tau_abs)) f |= 4;
      }
      if constexpr (SCHK) {
        // score check: sum over the full key tiles of s_ij against
        // q_i . sum_k K_k over the same keys (the prefix of the K column sums
        // up to the wave's first masked tile), within tau_s * |q_i| . sum_k |K_k|
        int tw = Lk / BC;   // tiles without the key-range mask
        if (CAUSAL) {
          const int lim = wq_lo + off + 1;   // tiles wholly below the wave's diagonal
          tw = min(tw, lim <= 0 ? 0 : lim / BC);
        }
        const size_t kro = ((size_t)bh * (p.ntk + 1) + tw) * D;
        float rhs = 0.f, ms = 0.f;
#pragma unroll
        for (int s2 = 0; s2 < NDS; ++s2) {
          const int c0 = 16 * s2 + 8 * grp;   // the lane's 8 columns of q
          const f32x4 kp0 = *reinterpret_cast<const f32x4*>(p.kpre + kro + c0);
          const f32x4 kp1 = *reinterpret_cast<const f32x4*>(p.kpre + kro + c0 + 4);
          const f32x4 ka0 = *reinterpret_cast<const f32x4*>(p.kabs + kro + c0);
          const f32x4 ka1 = *reinterpret_cast<const f32x4*>(p.kabs + kro + c0 + 4);
          const float kp[8] = {kp0[0], kp0[1], kp0[2], kp0[3], kp1[0], kp1[1], kp1[2], kp1[3]};
          const float ka[8] = {ka0[0], ka0[1], ka0[2], ka0[3], ka1[0], ka1[1], ka1[2], ka1[3]};
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float qa = __uint_as_float(qf[s2][e] << 16);
            const float qb = __uint_as_float(qf[s2][e] & 0xffff0000u);
            rhs = __builtin_fmaf(qa, kp[2 * e], __builtin_fmaf(qb, kp[2 * e + 1], rhs));
            ms = __builtin_fmaf(__builtin_fabsf(qa), ka[2 * e],
                                __builtin_fmaf(__builtin_fabsf(qb), ka[2 * e + 1], ms));
          }
        }
        // scores carry the softmax scale only in the exponent (exp2 of s * sl2):
        // the sums compare raw q . k
        const float lhs = sum_xor32(s_lhs);
        rhs = sum_xor32(rhs);
        ms = sum_xor32(ms);
        const float rs = lhs - rhs;
        nonfinite = nonfinite || nonfinite_bits(rs);
        if (!(__builtin_fabsf(rs) <= p.tau_s * ms + p.tau_abs)) f |= 8;
        // masked tiles: the two products' sums must agree bit for bit
        if (opaque_bits(sum_xor32(d_lhs)) != opaque_bits(sum_xor32(d_rhs))) f |= 8;
        sc_lhs = lhs;
        sc_rhs = rhs;
        sc_bound = ms;
      }
      if (nonfinite) f |= 3;
      if (grp == 0 && qrow < Lq) {
        const size_t ri = (size_t)bh * Lq + qrow;
        p.resid[ri] = r;
        p.flags[ri] = f;
        if constexpr (INJECT) {
          if (p.pred) p.pred[ri] = pred;
          if (p.actual) p.actual[ri] = act;
          if (p.pred_w) p.pred_w[ri] = pred_w;
          if (p.actual_w) p.actual_w[ri] = WCHK ? act_w : 0.f;
          if (p.s_lhs) p.s_lhs[ri] = sc_lhs;
          if (p.s_rhs) p.s_rhs[ri] = sc_rhs;
          if (p.s_bound) p.s_bound[ri] = sc_bound;
        }
      }
    }

    if (!has_next) break;
    // on to the next item: its first tiles are in the ring (cont), else it
    // starts like a first item
    bh = nbh;
    qt = nqt;
    set_item();
    primed = cont;
    if (!cont) load_q(bh, qt);
  }
}

// ---- persistent launches: how many workgroups the device holds at once
#if FABFT_PART == 0
std::atomic<int> g_persist{kPersistAuto};
void set_persistent(int mode) { g_persist.store(mode); }
int get_persistent() { return g_persist.load(); }
#else
extern std::atomic<int> g_persist;
#endif

// Compute units of the stream's device (0 if unknown), cached per device.
static int device_cus(hipStream_t stream) {
  constexpr int kMaxDev = 64;
  static std::atomic<int> cus[kMaxDev];
  int dev = -1;
  if (hipStreamGetDevice(stream, &dev) != hipSuccess || dev < 0 || dev >= kMaxDev) {
    (void)hipGetLastError();
    return 0;
  }
  int n = cus[dev].load();
  if (n == 0) {
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) {
      (void)hipGetLastError();
      return 0;
    }
    cus[dev].store(n);
  }
  return n;
}

template <int D, bool CAUSAL, bool CHECK, bool INJECT, bool WCHK, bool SPLIT, bool SCHK = false,
          bool TWOPASS = false>
static int launch_t(const FwdParams& p0, hipStream_t stream) {
  FwdParams p = p0;
  p.persist = 0;
  if constexpr (!INJECT && !SPLIT && !SCHK && !TWOPASS && Cfg<D>::AHEAD >= 3) {
    // one workgroup per CU (the occupancy the launch bounds give), a
    // multiple of 8 so that workgroup b stays on XCD b mod 8; with the mask
    // only for a head count divisible by 8 (the banded schedule). Automatic
    // only for short rows (at most 16 key tiles), where a workgroup's
    // start-up is a large part of its work; measured neutral on long rows.
    const int g = device_cus(stream) & ~7;
    const int heads = p.n_items / p.n_qt;
    const int mode = g_persist.load();
    const bool want = mode == kPersistAlways ||
                      (mode == kPersistAuto && (p.Lk + kBc - 1) / kBc <= 16);
    if (want && g >= 8 && p.n_items > g && (!CAUSAL || (heads & 7) == 0)) {
      p.persist = 1;
      p.grid = g;
    }
  }
  // the thread's last-error slot may hold an error of an unrelated earlier
  // HIP call (made by the caller); clear it so that only this launch counts
  (void)hipGetLastError();
  hipLaunchKernelGGL((fwd_kernel<D, CAUSAL, CHECK, INJECT, WCHK, SPLIT, SCHK, TWOPASS>), dim3(p.grid),
                     dim3(Cfg<D>::THREADS), 0, stream, p);
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

// mode 0: no checksum, 1: checksum, 2: checksum + injection/debug,
// 3: checksum, key split, 4: checksum, two passes (Algorithm 1), 5: the
// same with injection/debug; the weighted check (p.wcheck) in its own
// instantiations, below
template <int D, bool CAUSAL>
static int launch_c(const FwdParams& p, int mode, hipStream_t s) {
  if (mode == 0) return launch_t<D, CAUSAL, false, false, false, false>(p, s);
  if (mode == 4) return launch_t<D, CAUSAL, true, false, false, false, false, true>(p, s);
  if (mode == 5) return launch_t<D, CAUSAL, true, true, false, false, false, true>(p, s);
  if constexpr (D != 256) {
    // the score check (not built for the one-wave-per-SIMD width 256)
    if (p.kpre && (mode == 1 || mode == 2)) {
      if (mode == 1) return launch_t<D, CAUSAL, true, false, false, false, true>(p, s);
      return launch_t<D, CAUSAL, true, true, false, false, true>(p, s);
    }
  }
  if (mode == 1) return launch_t<D, CAUSAL, true, false, false, false>(p, s);
  if (mode == 3) return launch_t<D, CAUSAL, true, false, false, true>(p, s);
  return launch_t<D, CAUSAL, true, true, false, false>(p, s);
}

template <int D, bool CAUSAL>
static int launch_c_weighted(const FwdParams& p, int mode, hipStream_t s) {
  if (mode == 4) return launch_t<D, CAUSAL, true, false, true, false, false, true>(p, s);
  if (mode == 5) return launch_t<D, CAUSAL, true, true, true, false, false, true>(p, s);
  if constexpr (D != 256) {
    if (p.kpre && (mode == 1 || mode == 2)) {
      if (mode == 1) return launch_t<D, CAUSAL, true, false, true, false, true>(p, s);
      return launch_t<D, CAUSAL, true, true, true, false, true>(p, s);
    }
  }
  if (mode == 1) return launch_t<D, CAUSAL, true, false, true, false>(p, s);
  if (mode == 3) return launch_t<D, CAUSAL, true, false, true, true>(p, s);
  return launch_t<D, CAUSAL, true, true, true, false>(p, s);
}

template <int D>
static int launch_d_plain(const FwdParams& p, bool causal, int mode, hipStream_t s) {
  return causal ? launch_c<D, true>(p, mode, s) : launch_c<D, false>(p, mode, s);
}
template <int D>
static int launch_d_weighted(const FwdParams& p, bool causal, int mode, hipStream_t s) {
  return causal ? launch_c_weighted<D, true>(p, mode, s)
                : launch_c_weighted<D, false>(p, mode, s);
}

// the d = 128 forward kernels without the weighted check (part 1)
int launch_d128_plain(const FwdParams& p, bool causal, int mode, hipStream_t s);
#if FABFT_PART == 1
int launch_d128_plain(const FwdParams& p, bool causal, int mode, hipStream_t s) {
  return launch_d_plain<128>(p, causal, mode, s);
}
#else
template <int D>
static int launch_d(const FwdParams& p, bool causal, int mode, hipStream_t s) {
  const bool weighted = p.wcheck && mode != 0;
  if constexpr (D == 128) {
    if (!weighted) return launch_d128_plain(p, causal, mode, s);
  } else {
    if (!weighted) return launch_d_plain<D>(p, causal, mode, s);
  }
  return launch_d_weighted<D>(p, causal, mode, s);
}

// ---- merge of the key splits: one wave per query row. With m = max_s m_s
// and w_s = 2^(m_s - m): l = sum_s w_s l_s, o = sum_s w_s o_s, and c (and
// c_w) merge exactly like one more column of o (Eq. 10); then O = o / l,
// pred = c / l, actual = sum_j O_ij and the row's check as in the main
// kernel. Splits that saw no key have m_s = -inf and weight 0.
constexpr int kMergeWaves = 4;

__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x = __builtin_fmaxf(x, __shfl_xor(x, o));
  return x;
}
__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o);
  return x;
}

template <int D, bool WCHK>
__global__ __launch_bounds__(64 * kMergeWaves) void merge_kernel(FwdParams p, int rows_per_head) {
  constexpr int R = D + 4;
  constexpr int CPL = D / 64;   // output columns per lane
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int nrb = (rows_per_head + kMergeWaves - 1) / kMergeWaves;
  const int bh = blockIdx.x / nrb;
  const int row = (blockIdx.x - bh * nrb) * kMergeWaves + wave;
  if (row >= rows_per_head) return;   // wave-uniform; no barriers below
  const int ns = p.nsplit;
  const float* rec = p.ws + ((size_t)bh * rows_per_head + row) * ns * R;
  const float ms = lane < ns ? rec[(size_t)lane * R] : -__builtin_inff();
  const float m = wave_max(ms);
  const float w = (ms == -__builtin_inff()) ? 0.f : __builtin_amdgcn_exp2f(ms - m);
  const float l = wave_sum(lane < ns ? w * rec[(size_t)lane * R + 1] : 0.f);
  const float c = wave_sum(lane < ns ? w * rec[(size_t)lane * R + 2] : 0.f);
  const float cw = WCHK ? wave_sum(lane < ns ? w * rec[(size_t)lane * R + 3] : 0.f) : 0.f;
  float o[CPL];
#pragma unroll
  for (int u = 0; u < CPL; ++u) o[u] = 0.f;
  for (int s = 0; s < ns; ++s) {
    const float ws_ = __shfl(w, s);
#pragma unroll
    for (int u = 0; u < CPL; ++u) o[u] = __builtin_fmaf(ws_, rec[(size_t)s * R + 4 + lane + 64 * u], o[u]);
  }
  const float inv = l > 0.f ? 1.0f / l : 0.f;
  float act = 0.f, absum = 0.f, act_w = 0.f;
  uint16_t* orow = p.o + ((size_t)bh * rows_per_head + row) * p.dio;
#pragma unroll
  for (int u = 0; u < CPL; ++u) {
    const float x = o[u] * inv;   // 0 for columns past dio
    act += x;
    absum += __builtin_fabsf(x);
    act_w += (lane & 1) ? -x : x;   // column lane + 64u has the parity of lane
    if (lane + 64 * u < p.dio) orow[lane + 64 * u] = (uint16_t)(pack_bf16x2(x, 0.f) & 0xffffu);
  }
  act = wave_sum(act);
  absum = wave_sum(absum);
  const float pred = c * inv;
  const float r = pred - act;
  // as in the forward epilogue: an overflowed sum_j |O_ij| counts as non-finite
  bool nonfinite = nonfinite_bits(r) || nonfinite_bits(absum);
  uint8_t f = (__builtin_fabsf(r) <= p.tau_rel * (absum + __builtin_fabsf(pred)) + p.tau_abs) ? 0 : 1;
  if constexpr (WCHK) {
    act_w = wave_sum(act_w);
    const float pred_w = cw * inv;
    const float rw = pred_w - act_w;
    nonfinite = nonfinite || nonfinite_bits(rw);
    if (!(__builtin_fabsf(rw) <= p.tau_rel * (absum + __builtin_fabsf(pred_w)) + p.tau_abs)) f |= 4;
  }
  if (nonfinite) f |= 3;
  if (lane == 0) {
    const size_t ri = (size_t)bh * rows_per_head + row;
    p.resid[ri] = r;
    p.flags[ri] = f;
  }
}

int launch_merge(const FwdParams& p, int d, int nheads, hipStream_t stream) {
  const int nrb = (p.Lq + kMergeWaves - 1) / kMergeWaves;
  const long long g = (long long)nheads * nrb;
  if (g > INT_MAX) return -1;
  (void)hipGetLastError();
  const dim3 grid((unsigned)g), block(64 * kMergeWaves);
  if (compute_width(d) == 256) {
    if (p.wcheck) hipLaunchKernelGGL((merge_kernel<256, true>), grid, block, 0, stream, p, p.Lq);
    else hipLaunchKernelGGL((merge_kernel<256, false>), grid, block, 0, stream, p, p.Lq);
  } else if (compute_width(d) == 128) {
    if (p.wcheck) hipLaunchKernelGGL((merge_kernel<128, true>), grid, block, 0, stream, p, p.Lq);
    else hipLaunchKernelGGL((merge_kernel<128, false>), grid, block, 0, stream, p, p.Lq);
  } else {
    if (p.wcheck) hipLaunchKernelGGL((merge_kernel<64, true>), grid, block, 0, stream, p, p.Lq);
    else hipLaunchKernelGGL((merge_kernel<64, false>), grid, block, 0, stream, p, p.Lq);
  }
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

// ---- key split for a few query rows (Lq <= 4, decode): the MFMA kernel
// keeps one wave of its workgroup busy on a 32-row block whose other rows
// are empty, and that wave's tile work, not HBM, then sets the pace. Here
// every wave streams its own keys from HBM into registers and takes the
// products on the vector ALU: lane (g, c) of a load holds the 16-byte chunk
// c of key g's row (LPK = D / 8 lanes per key), so q . k is four dot2 per
// lane and a sum over the key's LPK lanes, and the P V update is eight FMAs
// per lane into the lane's own eight columns. Per row and wave: a running
// max (lazily moved, as in the forward kernel), l, c = sum p sumrow(V) (and
// c_w) and o, all in fp32 on the same p (Alg. 3); the waves' states are
// merged through LDS into the split's partial-state record, which
// merge_kernel combines across splits and checks as for the MFMA kernel.
constexpr int kDecWaves = 8;
constexpr int kDecLoads = 4;   // loads of K (and of V) per wave step
constexpr int kDecMaxRows = 4; // query rows per head up to which a split takes this kernel

// sum / max over aligned groups of N (8, 16, 32 or 64) lanes
template <int N>
__device__ __forceinline__ float span_sum(float x) {
  static_assert(N == 8 || N == 16 || N == 32 || N == 64, "span");
  x = group_sum<8>(x);
  if constexpr (N >= 16) x += dpp<0x140>(x);   // row_mirror: lanes i and 15 - i
  if constexpr (N >= 32) x += __shfl_xor(x, 16);
  if constexpr (N == 64) x = sum_xor32(x);
  return x;
}
// combine over the lanes that differ only in bits log2(G) .. 5 (the groups)
template <int G>
__device__ __forceinline__ float groups_sum(float x) {
#pragma unroll
  for (int o = G; o < 64; o <<= 1) x += __shfl_xor(x, o);
  return x;
}
template <int G>
__device__ __forceinline__ float groups_max(float x) {
#pragma unroll
  for (int o = G; o < 64; o <<= 1) x = __builtin_fmaxf(x, __shfl_xor(x, o));
  return x;
}

template <int D, int NQ, bool CAUSAL, bool WCHK>
__global__ __launch_bounds__(64 * kDecWaves) void decode_kernel(FwdParams p) {
  constexpr int LPK = D / 8;                // lanes per key
  constexpr int KPL = 64 / LPK;             // keys per load
  constexpr int NL = kDecLoads;
  constexpr int KS = NL * KPL;              // keys per wave step
  constexpr int R = D + 4;                  // record floats
  __shared__ float red[kDecWaves][NQ][R];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int split = blockIdx.x % p.nsplit;
  const int bh = blockIdx.x / p.nsplit;     // one query tile per head (Lq <= 4)
  const int Lq = p.Lq, Lk = p.Lk, off = Lk - Lq;
  const int DIO = p.dio, CIO = DIO / 8;
  const int c = lane % LPK, kg = lane / LPK;
  const float sl2 = p.sl2;
  // the split's keys: whole key tiles, as in the MFMA split kernel
  const int ntiles = (Lk + kBc - 1) / kBc;
  const int t_lo = min(ntiles, split * p.split_tiles);
  const int k_lo = t_lo * kBc;
  const int k_hi = min(Lk, min(ntiles, t_lo + p.split_tiles) * kBc);
  const int nsteps = (k_hi - k_lo + KS - 1) / KS;
  const bool col_ok = c < CIO;
  const uint16_t* kh = p.k + (size_t)bh * Lk * DIO + 8 * c;
  const uint16_t* vh = p.v + (size_t)bh * Lk * DIO + 8 * c;

  u32x4 q[NQ];
#pragma unroll
  for (int r = 0; r < NQ; ++r) {
    q[r] = u32x4{0, 0, 0, 0};
    if (r < Lq && col_ok)
      q[r] = *reinterpret_cast<const u32x4*>(p.q + ((size_t)bh * Lq + r) * DIO + 8 * c);
  }
  float m2[NQ], l[NQ], cs[NQ], cw[NQ], o[NQ][8];
#pragma unroll
  for (int r = 0; r < NQ; ++r) {
    m2[r] = -__builtin_inff();
    l[r] = cs[r] = cw[r] = 0.f;
#pragma unroll
    for (int j = 0; j < 8; ++j) o[r][j] = 0.f;
  }

  // keys of step j: k_lo + j*KS + n*KPL + kg (n < NL); rows past k_hi and
  // chunks past the row's DIO columns load as zeros
  auto load = [&](int j, u32x4 (&kk)[NL], u32x4 (&vv)[NL]) __attribute__((always_inline)) {
#pragma unroll
    for (int n = 0; n < NL; ++n) {
      const int key = k_lo + j * KS + n * KPL + kg;
      kk[n] = u32x4{0, 0, 0, 0};
      vv[n] = u32x4{0, 0, 0, 0};
      if (j < nsteps && key < k_hi && col_ok) {
        kk[n] = *reinterpret_cast<const u32x4*>(kh + (size_t)key * DIO);
        vv[n] = *reinterpret_cast<const u32x4*>(vh + (size_t)key * DIO);
      }
    }
  };
  auto step = [&](int j, const u32x4 (&kk)[NL], const u32x4 (&vv)[NL]) __attribute__((always_inline)) {
    if (j >= nsteps) return;   // wave-uniform
    // sumrow(V) (and the weighted sum) of each key of the step (Eq. 4)
    float vs[NL], vw[NL];
#pragma unroll
    for (int n = 0; n < NL; ++n) {
      float a = 0.f, b = 0.f;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        a = dot2(vv[n][e], kOnes, a);
        if constexpr (WCHK) b = dot2(vv[n][e], kAlt, b);
      }
      vs[n] = span_sum<LPK>(a);
      vw[n] = WCHK ? span_sum<LPK>(b) : 0.f;
    }
    float vf[NL][8];
#pragma unroll
    for (int n = 0; n < NL; ++n)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        vf[n][2 * e] = __uint_as_float(vv[n][e] << 16);
        vf[n][2 * e + 1] = __uint_as_float(vv[n][e] & 0xffff0000u);
      }
#pragma unroll
    for (int r = 0; r < NQ; ++r) {
      // s = q . k (Alg. 3), -inf where the key is not visible to row r
      float sc[NL];
      float mx = -__builtin_inff();
#pragma unroll
      for (int n = 0; n < NL; ++n) {
        float a = 0.f;
#pragma unroll
        for (int e = 0; e < 4; ++e) a = dot2(q[r][e], kk[n][e], a);
        a = span_sum<LPK>(a);
        const int key = k_lo + j * KS + n * KPL + kg;
        const bool vis = key < k_hi && r < Lq && (!CAUSAL || key <= r + off);
        sc[n] = vis ? a : -__builtin_inff();
        mx = __builtin_fmaxf(mx, sc[n]);
      }
      mx = groups_max<LPK>(mx);
      // lazy running max in the exp2 domain
      const float mt2 = (mx == -__builtin_inff()) ? -__builtin_inff() : mx * sl2;
      const float m2n = (mt2 > m2[r] + kLazy) ? mt2 : m2[r];
      if (m2n != m2[r]) {   // wave-uniform
        const float alpha = __builtin_amdgcn_exp2f(m2[r] - m2n);
        l[r] *= alpha;
        cs[r] *= alpha;
        cw[r] *= alpha;
#pragma unroll
        for (int jj = 0; jj < 8; ++jj) o[r][jj] *= alpha;
        m2[r] = m2n;
      }
      const float nm2 = (m2n == -__builtin_inff()) ? 0.f : -m2n;
#pragma unroll
      for (int n = 0; n < NL; ++n) {
        const float pr = __builtin_amdgcn_exp2f(__builtin_fmaf(sc[n], sl2, nm2));
        l[r] += pr;
        cs[r] = __builtin_fmaf(pr, vs[n], cs[r]);
        if constexpr (WCHK) cw[r] = __builtin_fmaf(pr, vw[n], cw[r]);
#pragma unroll
        for (int jj = 0; jj < 8; ++jj) o[r][jj] = __builtin_fmaf(pr, vf[n][jj], o[r][jj]);
      }
    }
  };

  // three steps in flight per wave: this wave's steps are wave, wave + W, ...
  u32x4 k0[NL], v0[NL], k1[NL], v1[NL], k2[NL], v2[NL];
  constexpr int W = kDecWaves;
  load(wave, k0, v0);
  load(wave + W, k1, v1);
  for (int j = wave; j < nsteps; j += 3 * W) {
    load(j + 2 * W, k2, v2);
    step(j, k0, v0);
    load(j + 3 * W, k0, v0);
    step(j + W, k1, v1);
    load(j + 4 * W, k1, v1);
    step(j + 2 * W, k2, v2);
  }

  // the wave's state per row: l, c, c_w and o summed over its key groups
  // (every lane of a group holds its group's sums), then through LDS
#pragma unroll
  for (int r = 0; r < NQ; ++r) {
    l[r] = groups_sum<LPK>(l[r]);
    cs[r] = groups_sum<LPK>(cs[r]);
    cw[r] = groups_sum<LPK>(cw[r]);
#pragma unroll
    for (int jj = 0; jj < 8; ++jj) o[r][jj] = groups_sum<LPK>(o[r][jj]);
    if (kg == 0) {
#pragma unroll
      for (int jj = 0; jj < 8; ++jj) red[wave][r][4 + 8 * c + jj] = o[r][jj];
    }
    if (lane == 0) {
      red[wave][r][0] = m2[r];
      red[wave][r][1] = l[r];
      red[wave][r][2] = cs[r];
      red[wave][r][3] = cw[r];
    }
  }
  __syncthreads();
  // merge of the waves (m = max_w m_w, x = sum_w x_w 2^(m_w - m)) into the
  // split's record; a split without a visible key keeps m = -inf, weight 0
  for (int e = tid; e < NQ * R; e += 64 * kDecWaves) {
    const int r = e / R, idx = e - r * R;
    if (r >= Lq) continue;
    float mm = -__builtin_inff();
#pragma unroll
    for (int w = 0; w < kDecWaves; ++w) mm = __builtin_fmaxf(mm, red[w][r][0]);
    float x = mm;
    if (idx > 0) {
      x = 0.f;
      if (mm != -__builtin_inff()) {
#pragma unroll
        for (int w = 0; w < kDecWaves; ++w)
          x = __builtin_fmaf(__builtin_amdgcn_exp2f(red[w][r][0] - mm), red[w][r][idx], x);
      }
    }
    p.ws[(((size_t)bh * Lq + r) * p.nsplit + split) * R + idx] = x;
  }
}

template <int D, bool CAUSAL>
static int launch_decode_c(const FwdParams& p, hipStream_t s) {
  const dim3 grid(p.grid), block(64 * kDecWaves);
  (void)hipGetLastError();
  const bool w = p.wcheck != 0;
  if (p.Lq == 1) {
    if (w) hipLaunchKernelGGL((decode_kernel<D, 1, CAUSAL, true>), grid, block, 0, s, p);
    else hipLaunchKernelGGL((decode_kernel<D, 1, CAUSAL, false>), grid, block, 0, s, p);
  } else if (p.Lq == 2) {
    if (w) hipLaunchKernelGGL((decode_kernel<D, 2, CAUSAL, true>), grid, block, 0, s, p);
    else hipLaunchKernelGGL((decode_kernel<D, 2, CAUSAL, false>), grid, block, 0, s, p);
  } else {
    if (w) hipLaunchKernelGGL((decode_kernel<D, 4, CAUSAL, true>), grid, block, 0, s, p);
    else hipLaunchKernelGGL((decode_kernel<D, 4, CAUSAL, false>), grid, block, 0, s, p);
  }
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

template <int D>
static int launch_decode(const FwdParams& p, bool causal, hipStream_t s) {
  return causal ? launch_decode_c<D, true>(p, s) : launch_decode_c<D, false>(p, s);
}

int launch_fwd(const FwdParams& p, int d, bool causal, int mode, hipStream_t stream) {
  const int dc = compute_width(d);
  if (mode == 3 && p.Lq <= kDecMaxRows && p.n_qt == 1) {
    // a key split of at most four query rows: the vector-ALU decode kernel
    if (dc == 256) return launch_decode<256>(p, causal, stream);
    if (dc == 128) return launch_decode<128>(p, causal, stream);
    return launch_decode<64>(p, causal, stream);
  }
  if (dc == 256) return launch_d<256>(p, causal, mode, stream);
  if (dc == 128) return launch_d<128>(p, causal, mode, stream);
  return launch_d<64>(p, causal, mode, stream);
}

int key_tile(int d) { return (d == 64 || d == 96 || d == 128 || d == 256) ? kBc : 0; }

// ---- global check of one head (Alg. 3, the check accumulated over all
// queries; Eq. 5 in its per-query form, Eq. 6-7): R = sum_i (pred_i -
// actual_i) = sum_i resid_i and A = sum_i sum_j |O_ij|, in fp64, one
// workgroup per (b, h), with a fixed reduction order (deterministic).
constexpr int kGThreads = 256;

__global__ __launch_bounds__(kGThreads) void global_check_kernel(
    const uint16_t* __restrict__ o, const float* __restrict__ resid, int Lq, int d,
    float tau_rel, float tau_abs, double* __restrict__ gsum, uint8_t* __restrict__ gflag) {
  __shared__ double red_r[kGThreads];
  __shared__ double red_a[kGThreads];
  const int bh = blockIdx.x;
  const int tid = threadIdx.x;
  const float* r = resid + (size_t)bh * Lq;
  const uint16_t* ob = o + (size_t)bh * Lq * d;
  double sr = 0.0, sa = 0.0;
  for (int i = tid; i < Lq; i += kGThreads) sr += (double)r[i];
  // O as 8-element chunks (rows are 16-byte aligned: d is 64, 96, 128 or 256)
  const size_t nchunk = (size_t)Lq * d / 8;
  for (size_t c = tid; c < nchunk; c += kGThreads) {
    const u32x4 w = *reinterpret_cast<const u32x4*>(ob + 8 * c);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      sa += (double)__builtin_fabsf(__uint_as_float(w[e] << 16));
      sa += (double)__builtin_fabsf(__uint_as_float(w[e] & 0xffff0000u));
    }
  }
  red_r[tid] = sr;
  red_a[tid] = sa;
  __syncthreads();
  for (int s = kGThreads / 2; s > 0; s >>= 1) {
    if (tid < s) {
      red_r[tid] += red_r[tid + s];
      red_a[tid] += red_a[tid + s];
    }
    __syncthreads();
  }
  if (tid == 0) {
    const double R = red_r[0], A = red_a[0];
    const uint64_t bits = __double_as_longlong(R);
    const bool nonfinite = ((bits >> 52) & 0x7ff) == 0x7ff;
    uint8_t f = (__builtin_fabs(R) <= (double)tau_rel * A + (double)tau_abs) ? 0 : 1;
    if (nonfinite) f = 3;
    gsum[bh] = R;
    gflag[bh] = f;
  }
}

// ---- score check operands: column sums of K and |K| per key tile (one
// workgroup of 256 threads per (head, tile): 16-byte loads of 8 columns of
// 4 rows per thread, partial sums reduced through LDS), then per head the
// exclusive prefix over the tiles in place (one thread per column): row t
// holds the sums over tiles 0 .. t-1, row ntk the sums over all keys.
// Columns past dio (d = 96) stay zero.
constexpr int kSumThreads = 256;
template <int D>
__global__ __launch_bounds__(kSumThreads) void ksum_kernel(const uint16_t* __restrict__ k, int Lk,
                                                           int ntk, int dio,
                                                           float* __restrict__ kpre,
                                                           float* __restrict__ kabs) {
  constexpr int CPR = D / 8;                 // 16-byte chunks per row
  constexpr int RG = kSumThreads / CPR;      // row groups
  constexpr int RPG = kBc / RG;              // rows per group
  static_assert(RG * CPR == kSumThreads && RPG * RG == kBc, "ksum layout");
  __shared__ float part_a[RG][D];
  __shared__ float part_b[RG][D];
  const int g = blockIdx.x;
  const int bh = g / ntk, t = g - bh * ntk;
  const int c = threadIdx.x % CPR, rg = threadIdx.x / CPR;
  float a[8] = {}, b[8] = {};
  if (8 * c < dio) {
    u32x4 ch[RPG];
#pragma unroll
    for (int r = 0; r < RPG; ++r) {
      const int row = t * kBc + rg * RPG + r;
      ch[r] = u32x4{0, 0, 0, 0};
      if (row < Lk)
        ch[r] = *reinterpret_cast<const u32x4*>(k + ((size_t)bh * Lk + row) * dio + 8 * c);
    }
#pragma unroll
    for (int r = 0; r < RPG; ++r)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float x0 = __uint_as_float(ch[r][e] << 16);
        const float x1 = __uint_as_float(ch[r][e] & 0xffff0000u);
        a[2 * e] += x0;
        a[2 * e + 1] += x1;
        b[2 * e] += __builtin_fabsf(x0);
        b[2 * e + 1] += __builtin_fabsf(x1);
      }
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    part_a[rg][8 * c + e] = a[e];
    part_b[rg][8 * c + e] = b[e];
  }
  __syncthreads();
  for (int j = threadIdx.x; j < D; j += kSumThreads) {
    float sa = 0.f, sb = 0.f;
#pragma unroll
    for (int r = 0; r < RG; ++r) {
      sa += part_a[r][j];
      sb += part_b[r][j];
    }
    const size_t o = ((size_t)bh * (ntk + 1) + t) * D + j;
    kpre[o] = sa;
    kabs[o] = sb;
  }
}

template <int D>
__global__ __launch_bounds__(D) void kscan_kernel(int ntk, float* __restrict__ kpre,
                                                  float* __restrict__ kabs) {
  const int bh = blockIdx.x, j = threadIdx.x;
  float* pa = kpre + (size_t)bh * (ntk + 1) * D + j;
  float* pb = kabs + (size_t)bh * (ntk + 1) * D + j;
  float ra = 0.f, rb = 0.f;
  // blocks of 8 tiles: the loads of a block are issued before its sums
  constexpr int U = 8;
  int t = 0;
  for (; t + U <= ntk; t += U) {
    float va[U], vb[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      va[u] = pa[(size_t)(t + u) * D];
      vb[u] = pb[(size_t)(t + u) * D];
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      pa[(size_t)(t + u) * D] = ra;
      pb[(size_t)(t + u) * D] = rb;
      ra += va[u];
      rb += vb[u];
    }
  }
  for (; t < ntk; ++t) {
    const float a = pa[(size_t)t * D], b = pb[(size_t)t * D];
    pa[(size_t)t * D] = ra;
    pb[(size_t)t * D] = rb;
    ra += a;
    rb += b;
  }
  pa[(size_t)ntk * D] = ra;
  pb[(size_t)ntk * D] = rb;
}

int launch_kpre(const uint16_t* k, int BH, int Lk, int d, float* kpre, float* kabs,
                hipStream_t stream) {
  const int ntk = (Lk + kBc - 1) / kBc;
  const long long g = (long long)BH * ntk;
  if (g < 1 || g > INT_MAX) return -1;
  (void)hipGetLastError();
  if (compute_width(d) == 128) {
    hipLaunchKernelGGL(ksum_kernel<128>, dim3((unsigned)g), dim3(kSumThreads), 0, stream, k, Lk,
                       ntk, d, kpre, kabs);
    hipLaunchKernelGGL(kscan_kernel<128>, dim3(BH), dim3(128), 0, stream, ntk, kpre, kabs);
  } else if (compute_width(d) == 64) {
    hipLaunchKernelGGL(ksum_kernel<64>, dim3((unsigned)g), dim3(kSumThreads), 0, stream, k, Lk,
                       ntk, d, kpre, kabs);
    hipLaunchKernelGGL(kscan_kernel<64>, dim3(BH), dim3(64), 0, stream, ntk, kpre, kabs);
  } else {
    return -1;
  }
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

// ---- per-head OR of the row flags (one workgroup per head)
__global__ __launch_bounds__(kGThreads) void head_flags_kernel(const uint8_t* __restrict__ flags,
                                                             int Lq, uint8_t* __restrict__ hflags) {
  __shared__ uint32_t red[kGThreads];
  const int bh = blockIdx.x;
  const uint8_t* f = flags + (size_t)bh * Lq;
  uint32_t acc = 0;
  for (int i = threadIdx.x; i < Lq; i += kGThreads) acc |= f[i];
  red[threadIdx.x] = acc;
  __syncthreads();
  for (int s = kGThreads / 2; s > 0; s >>= 1) {
    if ((int)threadIdx.x < s) red[threadIdx.x] |= red[threadIdx.x + s];
    __syncthreads();
  }
  if (threadIdx.x == 0) hflags[bh] = (uint8_t)red[0];
}

int launch_head_flags(const uint8_t* flags, int BH, int Lq, uint8_t* hflags, hipStream_t stream) {
  (void)hipGetLastError();
  hipLaunchKernelGGL(head_flags_kernel, dim3(BH), dim3(kGThreads), 0, stream, flags, Lq, hflags);
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

int launch_global(const uint16_t* o, const float* resid, int BH, int Lq, int d, float tau_rel,
                  float tau_abs, double* gsum, uint8_t* gflag, hipStream_t stream) {
  (void)hipGetLastError();
  hipLaunchKernelGGL(global_check_kernel, dim3(BH), dim3(kGThreads), 0, stream, o, resid, Lq, d,
                     tau_rel, tau_abs, gsum, gflag);
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

#endif  // FABFT_PART == 0

}  // namespace fabft
