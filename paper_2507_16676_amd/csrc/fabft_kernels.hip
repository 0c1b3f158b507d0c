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
// Dataflow (one workgroup = 4 waves = 128 query rows; one wave = 32 rows):
//  * The 32x32x16 bf16 MFMA computes S^T = K Q^T (keys on the M side, the
//    wave's 32 queries on the N side) and O^T = V^T P^T. With this
//    orientation a lane holds values of a single query row, so the row max,
//    the sums l and c, the alpha rescale and the final row sum are in-lane
//    work plus one exchange between lane i and lane i+32.
//  * Q stays in VGPRs as MFMA B operands for the whole pass.
//  * K and V tiles are loaded with 16-byte global loads into registers two
//    tiles ahead of use and written to a double-buffered LDS stage one tile
//    ahead: K row-major (padded rows), V transposed (V^T, padded rows), so
//    every MFMA A operand is one 16-byte LDS read. One barrier per tile.
//  * The K rows feeding MFMA row r are permuted (bits 2 and 3 of r swapped)
//    so that the S^T accumulator of a lane already holds, for each 16-key
//    step of P V, the 8 consecutive keys its B operand needs.
//  * sumrow(V) of the tile is summed in fp32 from the loader's registers
//    before V is written to LDS (the shared adder of the paper's checker),
//    reduced across lanes with DPP, and stored for the tile as a bf16 pair
//    hi + lo (hi = bf16(vs), lo = bf16(vs - hi); |vs - hi - lo| <= 2^-17|vs|)
//    so that the checksum can use the packed bf16 dot product.
//  * The weights p~ = bf16(p) feed the P V MFMA; l and the checksum c use
//    exactly those p~ (v_dot2_f32_bf16 on the packed pairs), so that the
//    rounding of P cancels between pred and actual. Every per-tile dot2
//    chain starts from zero and is folded into the running l and c with an
//    ordinary fp32 multiply-add.
//  * Lazy rescaling: the running max used for the exponentials is moved only
//    when a tile's max exceeds it by more than 8 in the exp2 domain, so
//    p <= 256 and o, l, c are rescaled (alpha != 1) rarely; o*alpha is
//    skipped when no lane of the wave moved its max. o/l and c/l are
//    unchanged in exact arithmetic (the shift cancels).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fabft_kernels.h"

namespace fabft {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;
constexpr int kBr = 32 * kWaves;
constexpr float kLazy = 8.0f;            // max drift (exp2 domain) before a rescale
constexpr uint32_t kOnes = 0x3f803f80u;  // bf16 pair (1.0, 1.0)

// BC keys per tile; the loader gives each thread KPT consecutive keys of one
// 16-byte column chunk, so that it can write KPT-key runs of V^T.
template <int D> struct TileCfg;
template <> struct TileCfg<128> { static constexpr int BC = 64, KPT = 4; };
template <> struct TileCfg<64> { static constexpr int BC = 64, KPT = 2; };

__device__ __forceinline__ f32x16 mfma32(u32x4 a, u32x4 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(
      __builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
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

// Sum over aligned groups of N consecutive lanes (N = 8 or 16); every lane
// of the group receives the same value.
template <int N>
__device__ __forceinline__ float group_sum(float x) {
  x += dpp<0xB1>(x);   // quad_perm [1,0,3,2]
  x += dpp<0x4E>(x);   // quad_perm [2,3,0,1]
  x += dpp<0x141>(x);  // row_half_mirror
  if constexpr (N == 16) x += dpp<0x140>(x);  // row_mirror
  return x;
}

// Combine the values of lanes i and i ^ 32 with a symmetric operation:
// v_permlane32_swap leaves (own, partner) in the two results of every lane.
__device__ __forceinline__ float sum_xor32(float x) {
#ifdef FABFT_SHFL_XOR32
  return x + __shfl_xor(x, 32);
#else
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
#endif
}
__device__ __forceinline__ float max_xor32(float x) {
#ifdef FABFT_SHFL_XOR32
  return __builtin_fmaxf(x, __shfl_xor(x, 32));
#else
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __builtin_fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
#endif
}

__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  f32x2 f = {a, b};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, bf16x2));
}
__device__ __forceinline__ float bf16_lo(uint32_t u) { return __uint_as_float(u << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t u) { return __uint_as_float(u & 0xffff0000u); }

// Row r of an MFMA 32-row block reads key 16*(r>>4) + 8*((r>>2)&1) + 4*((r>>3)&1) + (r&3)
__device__ __forceinline__ int swap_bits23(int r) {
  return (r & ~12) | ((r & 4) << 1) | ((r & 8) >> 1);
}

// V^T row r keeps its 8-key (16-byte) chunks in the order c ^ ((r >> 4) & 7):
// the loader's 8-byte writes (16 lanes on rows 8 apart) and the MFMA operand
// reads (16 lanes on consecutive rows) then fall in distinct LDS banks.
__device__ __forceinline__ int vt_chunk(int row, int c) { return c ^ ((row >> 4) & 7); }

// One LDS stage: a K tile, its V^T and sumrow(V) as bf16 hi/lo key pairs.
template <int D>
struct Stage {
  static constexpr int BC = TileCfg<D>::BC;
  static constexpr int KST = D + 8;   // LDS row stride of K (elements)
  static constexpr int VST = BC + 8;  // LDS row stride of V^T (elements)
  uint16_t k[BC * KST];
  uint16_t vt[D * VST];
  uint32_t vs_hi[BC / 2];
  uint32_t vs_lo[BC / 2];
};

template <int D, bool CAUSAL, bool CHECK, bool INJECT>
#ifndef FABFT_MIN_BLOCKS
#define FABFT_MIN_BLOCKS 2
#endif
__global__ __launch_bounds__(kThreads, FABFT_MIN_BLOCKS) void fwd_kernel(FwdParams p) {
  constexpr int BC = TileCfg<D>::BC;
  constexpr int KPT = TileCfg<D>::KPT;
  constexpr int KST = Stage<D>::KST;
  constexpr int VST = Stage<D>::VST;
  constexpr int CPR = D / 8;      // 16-byte chunks per K/V row
  constexpr int NKB = BC / 32;    // 32-key blocks per tile
  constexpr int NDB = D / 32;     // 32-column blocks of the output
  constexpr int NDS = D / 16;     // 16-wide steps over d in Q K^T
  static_assert(kThreads == (BC / KPT) * CPR, "loader covers the tile");

  __shared__ __attribute__((aligned(16))) Stage<D> stage[2];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
  const int mrow = lane & 31;   // MFMA row / column index of this lane
  const int grp = lane >> 5;    // which 8-wide k slice this lane holds

  // ---- workgroup -> (head, query tile): keep each head on one XCD, the
  // heaviest causal tiles first
  const int G = p.grid;
  const int bid = blockIdx.x;
  const int xcd = bid & 7;
  const int per = G >> 3, rem = G & 7;
  const int slot = bid >> 3;
  const int logical = (xcd < rem) ? xcd * (per + 1) + slot
                                  : rem * (per + 1) + (xcd - rem) * per + slot;
  const int bh = logical / p.n_qt;
  int qt = logical - bh * p.n_qt;
  if (CAUSAL) qt = p.n_qt - 1 - qt;

  const int Lq = p.Lq, Lk = p.Lk;
  const int q0 = qt * kBr;
  const int off = Lk - Lq;
  const size_t qbase = (size_t)bh * (size_t)Lq * D;
  const size_t kbase = (size_t)bh * (size_t)Lk * D;

  int kend = Lk;
  if (CAUSAL) kend = min(Lk, q0 + kBr + off);
  const int ntiles = kend > 0 ? (kend + BC - 1) / BC : 0;

  // ---- Q fragments (B operand): lane holds query q0+32w+mrow, d slice 8*grp
  const int qrow = q0 + 32 * wave + mrow;
  u32x4 qf[NDS];
#pragma unroll
  for (int s = 0; s < NDS; ++s) {
    qf[s] = u32x4{0, 0, 0, 0};
    if (qrow < Lq)
      qf[s] = *reinterpret_cast<const u32x4*>(p.q + qbase + (size_t)qrow * D + 16 * s + 8 * grp);
  }

  f32x16 oacc[NDB];
#pragma unroll
  for (int b = 0; b < NDB; ++b) oacc[b] = f32x16{};
  float m2_run = -__builtin_inff();   // running max, exp2 domain (s * scale * log2 e)
  float l_run = 0.f;
  float c_run = 0.f;
  const float sl2 = p.sl2;

  // ---- loader: thread -> (16-byte chunk lc, group of KPT keys lkg)
  const int lc = tid % CPR;
  const int lkg = tid / CPR;
  u32x4 kreg[KPT], vreg[KPT];
  const size_t ld_off = kbase + (size_t)(KPT * lkg) * D + 8 * lc;
  const uint16_t* kld = p.k + ld_off;   // this thread's first element of tile 0
  const uint16_t* vld = p.v + ld_off;
  auto gload = [&](int kv0) {
    const size_t o = (size_t)kv0 * D;
    if (kv0 + BC <= Lk) {   // whole tile in range (uniform)
#pragma unroll
      for (int r = 0; r < KPT; ++r) {
        kreg[r] = *reinterpret_cast<const u32x4*>(kld + o + r * D);
        vreg[r] = *reinterpret_cast<const u32x4*>(vld + o + r * D);
      }
    } else {
#pragma unroll
      for (int r = 0; r < KPT; ++r) {
        kreg[r] = u32x4{0, 0, 0, 0};
        vreg[r] = u32x4{0, 0, 0, 0};
        if (kv0 + KPT * lkg + r < Lk) {
          kreg[r] = *reinterpret_cast<const u32x4*>(kld + o + r * D);
          vreg[r] = *reinterpret_cast<const u32x4*>(vld + o + r * D);
        }
      }
    }
  };

  // registers -> LDS stage `buf` for the tile starting at key kv0
  auto stage_write = [&](int buf, int kv0) {
    Stage<D>& st = stage[buf];
    if constexpr (CHECK) {
      // sumrow(V) of this thread's KPT keys (Eq. 4): its 8 values, then the
      // CPR threads that share the keys
      float vsum[KPT];
#pragma unroll
      for (int r = 0; r < KPT; ++r) {
        float a = dot2(vreg[r][0], kOnes, 0.f);
        a = dot2(vreg[r][1], kOnes, a);
        a = dot2(vreg[r][2], kOnes, a);
        a = dot2(vreg[r][3], kOnes, a);
        vsum[r] = group_sum<CPR>(a);
      }
      if (lc == 0) {
        uint32_t hi[KPT / 2], lo[KPT / 2];
#pragma unroll
        for (int r = 0; r < KPT / 2; ++r) {
          hi[r] = pack_bf16x2(vsum[2 * r], vsum[2 * r + 1]);
          lo[r] = pack_bf16x2(vsum[2 * r] - bf16_lo(hi[r]), vsum[2 * r + 1] - bf16_hi(hi[r]));
        }
        if constexpr (KPT == 4) {
          *reinterpret_cast<u32x2*>(&st.vs_hi[2 * lkg]) = u32x2{hi[0], hi[1]};
          *reinterpret_cast<u32x2*>(&st.vs_lo[2 * lkg]) = u32x2{lo[0], lo[1]};
        } else {
          st.vs_hi[lkg] = hi[0];
          st.vs_lo[lkg] = lo[0];
        }
      }
    }
    if constexpr (INJECT) {
      // V site: flip a bit of V[key][col] after sumrow was taken
      if (p.f_site == 4 && bh == p.f_bh && qt == p.f_tile) {
        const int fk = p.f_row - kv0 - KPT * lkg;
        const int fc = p.f_col - 8 * lc;
        if (fk >= 0 && fk < KPT && fc >= 0 && fc < 8) {
          const uint32_t mask = (1u << p.f_bit) << (16 * (fc & 1));
#pragma unroll
          for (int r = 0; r < KPT; ++r)
            if (r == fk) {
#pragma unroll
              for (int e = 0; e < 4; ++e)
                if (e == (fc >> 1)) vreg[r][e] ^= mask;
            }
        }
      }
    }
#pragma unroll
    for (int r = 0; r < KPT; ++r)
      *reinterpret_cast<u32x4*>(&st.k[(KPT * lkg + r) * KST + 8 * lc]) = kreg[r];
    // V^T row 8lc+j, keys KPT*lkg .. +KPT-1: pairs of keys packed per dword
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int e = j >> 1;
      uint32_t w[KPT / 2];
#pragma unroll
      for (int r = 0; r < KPT / 2; ++r)
        w[r] = (j & 1) == 0 ? (vreg[2 * r][e] & 0xffffu) | (vreg[2 * r + 1][e] << 16)
                            : (vreg[2 * r][e] >> 16) | (vreg[2 * r + 1][e] & 0xffff0000u);
      const int row = 8 * lc + j, key = KPT * lkg;
      uint16_t* dst = &st.vt[row * VST + 8 * vt_chunk(row, key >> 3) + (key & 7)];
      if constexpr (KPT == 4)
        *reinterpret_cast<u32x2*>(dst) = u32x2{w[0], w[1]};
      else
        *reinterpret_cast<uint32_t*>(dst) = w[0];
    }
  };

  if (ntiles > 0) {
    gload(0);
    stage_write(0, 0);
    if (ntiles > 1) gload(BC);
  }

  const int wq_lo = q0 + 32 * wave;  // first query row of this wave

  for (int t = 0; t < ntiles; ++t) {
    const int kv0 = t * BC;
    // tile t sits in stage t&1; every wave is done with tile t-1, whose
    // stage (t+1)&1 is refilled with tile t+1
    __syncthreads();
    if (t + 1 < ntiles) {
      stage_write((t + 1) & 1, kv0 + BC);
      if (t + 2 < ntiles) gload(kv0 + 2 * BC);
    }
    const Stage<D>& st = stage[t & 1];

    // waves whose rows see none of this tile's keys skip it
    if (CAUSAL && kv0 > wq_lo + 31 + off) continue;
    const bool need_mask = (kv0 + BC > Lk) || (CAUSAL && kv0 + BC - 1 > wq_lo + off);

    // ---- S^T = K Q^T (Alg. 3: s_i = q . k_i)
    f32x16 sacc[NKB];
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb) sacc[kb] = f32x16{};
#pragma unroll
    for (int s = 0; s < NDS; ++s) {
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb) {
        const u32x4 a = *reinterpret_cast<const u32x4*>(
            &st.k[(kb * 32 + swap_bits23(mrow)) * KST + 16 * s + 8 * grp]);
        sacc[kb] = mfma32(a, qf[s], sacc[kb]);
      }
    }
    // accumulator element i of block kb holds key kv0 + 32kb + 16(i/8) + 8grp + (i%8)
    if constexpr (INJECT) {
      if (p.f_site == 1 && bh == p.f_bh && qrow == p.f_row) {
        const int kl = p.f_col - kv0;
        if (kl >= 0 && kl < BC && ((kl >> 3) & 1) == grp) {
          const int kb = kl >> 5, i = ((kl >> 4) & 1) * 8 + (kl & 7);
#pragma unroll
          for (int b = 0; b < NKB; ++b)
#pragma unroll
            for (int e = 0; e < 16; ++e)
              if (b == kb && e == i)
                sacc[b][e] = __uint_as_float(__float_as_uint(sacc[b][e]) ^ (1u << p.f_bit));
        }
      }
    }

    // ---- mask, tile max (Alg. 3: m_i = max(m_{i-1}, s_i))
    if (need_mask) {
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int key = kv0 + 32 * kb + 16 * (i >> 3) + 8 * grp + (i & 7);
          const bool ok = key < Lk && (!CAUSAL || key <= qrow + off);
          if (!ok) sacc[kb][i] = -__builtin_inff();
        }
    }
    float mx = -__builtin_inff();
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
      for (int i = 0; i < 16; i += 2)
        mx = __builtin_fmaxf(mx, __builtin_fmaxf(sacc[kb][i], sacc[kb][i + 1]));
    mx = max_xor32(mx);
    // lazy running max in the exp2 domain
    const float mt2 = (mx == -__builtin_inff()) ? -__builtin_inff() : mx * sl2;
    const float m2_new = (mt2 > m2_run + kLazy) ? mt2 : m2_run;
    const float alpha = (m2_new == m2_run) ? 1.f : __builtin_amdgcn_exp2f(m2_run - m2_new);
    m2_run = m2_new;
    const float nm2 = (m2_new == -__builtin_inff()) ? 0.f : -m2_new;

    // ---- p = exp(s - m) and p~ = bf16(p), the B operands of P V
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
      for (int i = 0; i < 16; ++i)
        sacc[kb][i] = __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[kb][i], sl2, nm2));
    if (need_mask) {
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int key = kv0 + 32 * kb + 16 * (i >> 3) + 8 * grp + (i & 7);
          const bool ok = key < Lk && (!CAUSAL || key <= qrow + off);
          if (!ok) sacc[kb][i] = 0.f;
        }
    }
    u32x4 pb[NKB][2];
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int e = 0; e < 4; ++e)
          pb[kb][h][e] = pack_bf16x2(sacc[kb][8 * h + 2 * e], sacc[kb][8 * h + 2 * e + 1]);

    // ---- l = l*alpha + sum p~ (Alg. 3)
    float lsum = 0.f;
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int e = 0; e < 4; ++e) lsum = dot2(pb[kb][h][e], kOnes, lsum);
    l_run = __builtin_fmaf(l_run, alpha, lsum);

    // ---- online checksum (Alg. 3: c = c*alpha + sumrow(V) * p~)
    if constexpr (CHECK) {
      float csum = 0.f;
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int pi = 16 * kb + 8 * h + 4 * grp;  // first key pair of this lane
          const u32x4 vh = *reinterpret_cast<const u32x4*>(&st.vs_hi[pi]);
          const u32x4 vl = *reinterpret_cast<const u32x4*>(&st.vs_lo[pi]);
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            csum = dot2(pb[kb][h][e], vh[e], csum);
            csum = dot2(pb[kb][h][e], vl[e], csum);
          }
        }
      c_run = __builtin_fmaf(c_run, alpha, csum);
    }
    if constexpr (INJECT) {
      if (p.f_site == 2 && bh == p.f_bh && qrow == p.f_row) {
        const int kl = p.f_col - kv0;
        if (kl >= 0 && kl < BC && ((kl >> 3) & 1) == grp) {
          const int kb = kl >> 5, h = (kl >> 4) & 1, e = (kl & 7) >> 1;
          const uint32_t mask = (1u << p.f_bit) << (16 * (kl & 1));
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

    // ---- O^T = alpha O^T + V^T P^T (Alg. 3: o = o*alpha + v * p)
    if (__ballot(alpha != 1.f)) {
#pragma unroll
      for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int i = 0; i < 16; ++i) oacc[db][i] *= alpha;
    }
    // (output blocks innermost: consecutive MFMAs accumulate independently)
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int db = 0; db < NDB; ++db) {
          const int row = 32 * db + mrow;
          const u32x4 a = *reinterpret_cast<const u32x4*>(
              &st.vt[row * VST + 8 * vt_chunk(row, 4 * kb + 2 * h + grp)]);
          oacc[db] = mfma32(a, pb[kb][h], oacc[db]);
        }
    if constexpr (INJECT) {
      // O site: accumulator element (row, col) after the P V of tile f_tile
      if (p.f_site == 3 && bh == p.f_bh && qrow == p.f_row && t == p.f_tile) {
        const int j = p.f_col;
        // output column j = 32db + 8a + 4grp + (i%4), element i = 4a + (i%4)
        if (((j >> 2) & 1) == grp) {
          const int db = j >> 5, i = 4 * ((j >> 3) & 3) + (j & 3);
#pragma unroll
          for (int b = 0; b < NDB; ++b)
#pragma unroll
            for (int e = 0; e < 16; ++e)
              if (b == db && e == i)
                oacc[b][e] = __uint_as_float(__float_as_uint(oacc[b][e]) ^ (1u << p.f_bit));
        }
      }
    }
  }

  // ---- epilogue: O = o / l (Alg. 3), pred = c / l (Eq. 8), check
  const float l_tot = sum_xor32(l_run);
  const float inv = l_tot > 0.f ? 1.0f / l_tot : 0.f;
  float act = 0.f, absum = 0.f;
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const float x = oacc[db][i] * inv;
      oacc[db][i] = x;
      act += x;
      absum += __builtin_fabsf(x);
    }
  if (qrow < Lq) {
    uint16_t* orow = p.o + qbase + (size_t)qrow * D;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int a = 0; a < 4; ++a) {
        const u32x2 w = {pack_bf16x2(oacc[db][4 * a], oacc[db][4 * a + 1]),
                         pack_bf16x2(oacc[db][4 * a + 2], oacc[db][4 * a + 3])};
        *reinterpret_cast<u32x2*>(orow + 32 * db + 8 * a + 4 * grp) = w;
      }
  }
  if constexpr (CHECK) {
    act = sum_xor32(act);
    absum = sum_xor32(absum);
    const float c_tot = sum_xor32(c_run);
    const float pred = c_tot * inv;
    const float r = pred - act;
    const float M = absum + __builtin_fabsf(pred);
    // non-finite test on the bits (this file is built with relaxed NaN rules);
    // a non-finite residual also fails the threshold comparison
    const bool nonfinite = (__float_as_uint(r) & 0x7f800000u) == 0x7f800000u;
    const uint8_t f = nonfinite ? 3 : (__builtin_fabsf(r) <= p.tau_rel * M + p.tau_abs ? 0 : 1);
    if (grp == 0 && qrow < Lq) {
      const size_t ri = (size_t)bh * Lq + qrow;
      p.resid[ri] = r;
      p.flags[ri] = f;
      if constexpr (INJECT) {
        if (p.pred) p.pred[ri] = pred;
        if (p.actual) p.actual[ri] = act;
      }
    }
  }
}

template <int D, bool CAUSAL, bool CHECK, bool INJECT>
static int launch_t(const FwdParams& p, hipStream_t stream) {
  hipLaunchKernelGGL((fwd_kernel<D, CAUSAL, CHECK, INJECT>), dim3(p.grid), dim3(kThreads), 0,
                     stream, p);
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

template <int D>
static int launch_d(const FwdParams& p, bool causal, int mode, hipStream_t s) {
  // mode 0: no checksum, 1: checksum, 2: checksum + injection/debug
  if (causal) {
    if (mode == 0) return launch_t<D, true, false, false>(p, s);
    if (mode == 1) return launch_t<D, true, true, false>(p, s);
    return launch_t<D, true, true, true>(p, s);
  }
  if (mode == 0) return launch_t<D, false, false, false>(p, s);
  if (mode == 1) return launch_t<D, false, true, false>(p, s);
  return launch_t<D, false, true, true>(p, s);
}

int launch_fwd(const FwdParams& p, int d, bool causal, int mode, hipStream_t stream) {
  if (d == 128) return launch_d<128>(p, causal, mode, stream);
  return launch_d<64>(p, causal, mode, stream);
}

int key_tile(int d) { return d == 128 ? TileCfg<128>::BC : TileCfg<64>::BC; }

}  // namespace fabft
