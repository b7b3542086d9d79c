// Block-sparse attention under a reused block mask (Sec. 3.3, historical
// sparse-connectivity reuse; Appendix C.3): the target's Q, K, V are
// recomputed and only the key blocks listed for a query block are visited.
//
// One workgroup per query block (BS queries, BS/32 waves of 32 queries).  The
// workgroup walks its compacted key-block list in stages of BS/2 keys (half a
// key block).  K and V stages are copied from HBM straight into LDS
// (global_load_lds, no register staging) into two slots each: the K tile of a
// stage is issued two stages before its scores are computed, the V tile one
// stage before its P.V product.  S^T = K Q^T and O^T += V^T P^T run on bf16
// MFMA 32x32x16 with fp32 accumulation; the online softmax runs in fp32 in
// the exp2 domain.
//
// Computing S^T (keys as MFMA rows, queries as columns) puts every score of a
// query in one lane pair (lane q and lane q+32), so the row max is one
// v_permlane32_swap and the row sum stays lane-local until the end.  The key
// order inside a 32-key MFMA tile is permuted (bits 2 and 3 of the row index
// swapped) so that the S^T accumulators are directly the B operand of the P.V
// product; its V^T operand comes from the row-major V stage through the LDS
// transpose read (ds_read_b64_tr_b16), so V never needs a transposed copy.
// K and V rows are XOR-swizzled in 16-byte chunks so both operand reads are
// free of bank conflicts.
#include "internal.h"

#include <math.h>

#include <type_traits>

namespace carnator {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

// s_waitcnt immediate: vmcnt(0) with expcnt and lgkmcnt left at their maxima.
constexpr int kWaitVm0 = 0x0F70;

// The tile loads are driven by hand: the direct loads, the wait and the
// barrier are written as inline assembly.  Issued through the compiler
// builtin, a direct load makes every later LDS read look like it may alias
// the transfer, and the compiler then drains all outstanding loads
// (vmcnt(0)) before each operand read, which removes the prefetch.  The
// asm writes M0 and declares it clobbered, so the compiler keeps no value of
// its own in M0 across a load.
//
// 16 bytes per lane from base + voff to LDS offset lds_off + 16 * lane; base
// and lds_off are the same in every lane.
__device__ inline void dma16(const void *base, unsigned voff, unsigned lds_off) {
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(voff), "s"(base),
               "s"(__builtin_amdgcn_readfirstlane(lds_off))
               : "memory", "m0");
}
// Wait until every direct load and LDS read of this wave has completed, then
// meet the other waves.
__device__ inline void wait_all_then_barrier() {
  asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// An empty use of x at this point of the instruction stream: keeps the
// compiler from sinking the computation of x into a later basic block.
__device__ inline void anchor(float x) { asm volatile("" ::"v"(x)); }

// MFMA row -> key inside a 32-key tile: swap bits 2 and 3.
__device__ inline int perm32(int rr) { return (rr & ~12) | ((rr & 4) << 1) | ((rr & 8) >> 1); }

// Lane l and lane l^32 hold the two halves of one query's keys.  One
// v_permlane32_swap exchanges the halves without going through LDS; both
// lanes then combine (x_lo, x_hi) in the same order.
__device__ inline float2 halves(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return make_float2(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

// Running-max growth (log2 units) below which O and l keep their old scale:
// P may then reach 2^8, harmless in fp32 and bf16, and most stages skip the
// rescale of the output accumulators.
constexpr float kRescaleSlack = 8.f;

// Chunk swizzles (16-byte chunk c of row r sits in slot c ^ swz(r)).
// K: the 16 lanes of a bank cycle read rows 0..15 (permuted) at one chunk.
template <int CPR>
__device__ inline int swz_k(int r) {
  if constexpr (CPR == 16) return r & 15;
  else return (r >> 1) & 7;
}
// V: the 32 lanes of a transpose read cover 4 consecutive rows x 64 bytes.
template <int CPR>
__device__ inline int swz_v(int r) {
  if constexpr (CPR == 16) return 4 * (r & 3);
  else return 4 * ((r >> 1) & 1);
}

// Longest key-block list a row can have (the number of key blocks is
// limited to this by the entry points).
constexpr int kMaxListBlocks = 2048;

template <int D, int BS>
struct Cfg {
  static constexpr int KT = BS / 2;               // keys per stage (two stages per block)
  static constexpr int MT = KT / 32;              // 32-key MFMA tiles per stage
  static constexpr int WAVES = BS / 32;
  static constexpr int NT = 64 * WAVES;
  static constexpr int RB = D * 2;                // bytes per K or V row
  static constexpr int CPR = D / 8;               // 16-byte chunks per row
  static constexpr int RPL = 1024 / RB;           // rows per 1-KiB direct load
  static constexpr int TB = KT * RB;              // one K or V tile
  static constexpr int LIST = 4 * TB;             // the row's key-block list follows the tiles
  static constexpr int LDS = LIST + 4 * (kMaxListBlocks + 2);  // K slots 0, 1; V slots 0, 1; list
  static constexpr int LI = TB / 1024 / WAVES;    // direct loads per wave per tile
  static_assert(TB % (1024 * WAVES) == 0, "tile split");
};

// One workgroup per query block, 32 queries per wave, two waves per SIMD.
//
// A wave issues vector instructions while its own MFMAs execute, but two
// waves sharing a SIMD overlap their MFMA and vector work far less, so the
// overlap is built into each wave's instruction stream.  Iteration j:
//   part A: O += V(j-1)^T P(j-1)^T on the matrix cores, interleaved with the
//           softmax of S(j) (row max, and P for the first 32 keys);
//   part B: S(j+1) = K(j+1) Q^T, first for keys 0..31 of the stage while P
//           for keys 32..63 of S(j) is formed, then for keys 32..63 once
//           those scores have been consumed.
// Only P is double-buffered in registers (the scores are reused in place).
//
// K and V have two LDS slots each.  Iteration j waits for V(j-1) and K(j+1),
// meets the other waves (after which K(j) and V(j-2) are no longer read) and
// issues V(j) and K(j+2) into those slots.
//
// A grown running max only records alpha: the output accumulators are
// rescaled at the start of the next iteration, since the P.V in flight in
// this one still belongs to the old max.  This keeps the softmax free of
// branches, so it shares one scheduling region with the MFMAs.
// At d = 64 the non-LSE kernel is held to 168 registers (a few spills), so
// three workgroups share a CU (their LDS, 3 x 40 KB, fits): with half the
// MFMAs per score of d = 128 it is bound by its vector work, which a third
// wave per SIMD overlaps better (2-3 % on the CogVideoX shape).
template <int D, int BS, bool WITH_LSE>
__global__ void __launch_bounds__(2 * BS, (D == 64 && !WITH_LSE) ? 3 : 2)
bsattn_kernel(View q, View k, View v, uint16_t *__restrict__ out, int64_t osb, int64_t osh,
              int64_t osn, int H, int N, int nB, const int32_t *__restrict__ row_ptr,
              const int32_t *__restrict__ col_idx, const int32_t *__restrict__ order,
              const int32_t *__restrict__ n_rows, float c2, float *__restrict__ lse) {
  using C = Cfg<D, BS>;
  constexpr int KT = C::KT, MT = C::MT;
  extern __shared__ __attribute__((aligned(1024))) unsigned char lds[];
  // a row subset: only order[0 .. *n_rows) (the whole workgroup, before any
  // barrier)
  if (n_rows != nullptr && (int)blockIdx.x >= *n_rows) return;

  // rows, list extents and block indices are clamped into range, so that
  // malformed lists cannot reach outside the tensors
  const int R = (int)gridDim.x;
  const int row = min(max(order[blockIdx.x], 0), R - 1);
  const int bh = row / nB;
  const int qb = row - bh * nB;
  const int b = bh / H, h = bh - b * H;
  const int Lr = min(max(row_ptr[row + 1] - row_ptr[row], 0), nB);
  const int e0 = min(max(row_ptr[row], 0), R * nB - Lr), e1 = e0 + Lr;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int l32 = lane & 31, hh = lane >> 5;
  const int qtok = qb * BS + wave * 32 + l32;

  // ---- Q fragment (B operand of S^T = K Q^T): query l32, channels 16t+8hh..+8
  bf16x8 qreg[D / 16];
  {
    const uint16_t *qp = q.data + (int64_t)b * q.sb + (int64_t)h * q.sh + (int64_t)qtok * q.sn + 8 * hh;
#pragma unroll
    for (int t = 0; t < D / 16; ++t) {
      uint4 w = make_uint4(0, 0, 0, 0);
      if (qtok < N) w = *reinterpret_cast<const uint4 *>(qp + 16 * t);
      qreg[t] = __builtin_bit_cast(bf16x8, w);
    }
  }
  // the Q fragment is in registers before any tile load is issued
  __builtin_amdgcn_s_waitcnt(kWaitVm0);

  f32x16 oacc[D / 32];
#pragma unroll
  for (int mo = 0; mo < D / 32; ++mo)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[mo][r] = 0.f;
  float mrun = -INFINITY, lrun = 0.f, lexact = 0.f, alpha = 1.f;

  const uint16_t *kbase = k.data + (int64_t)b * k.sb + (int64_t)h * k.sh;
  const uint16_t *vbase = v.data + (int64_t)b * v.sb + (int64_t)h * v.sh;

  // ---- direct loads: the i-th 1-KiB load of this wave fills rows
  // RPL (wave LI + i) .. + RPL of a tile; lane l writes 16 bytes at 16 l,
  // i.e. row +lrow, slot `slot`, which holds chunk slot ^ swz(row).
  // A tile always covers KT rows inside the tensor: a stage reaching past N
  // loads the KT rows ending at N instead (and masks the keys outside the
  // stage), and when N < KT the rows past N re-read row N - 1.  So one set
  // of lane offsets serves every tile.
  const int lrow = lane / (C::RB / 16), slot = lane % (C::RB / 16);
  unsigned koff[C::LI], voff[C::LI];  // lane offsets of a tile, bytes
#pragma unroll
  for (int i = 0; i < C::LI; ++i) {
    const int r = C::RPL * (wave * C::LI + i) + lrow;
    const int rr = min(r, N - 1);
    koff[i] = (unsigned)(((int64_t)rr * k.sn + (slot ^ swz_k<C::CPR>(r)) * 8) * 2);
    voff[i] = (unsigned)(((int64_t)rr * v.sn + (slot ^ swz_v<C::CPR>(r)) * 8) * 2);
  }
  const int kmax = max(N - KT, 0);  // first row of the last full tile

  // ---- operand-read lane offsets inside a tile
  // K (A of S^T): row perm32(l32), chunk 2t + hh
  int kread[D / 16];
  {
    const int kr = perm32(l32);
#pragma unroll
    for (int t = 0; t < D / 16; ++t) kread[t] = kr * C::RB + (((2 * t + hh) ^ swz_k<C::CPR>(kr)) << 4);
  }
  // V (A of O^T, via the transpose read): in each 16-lane group g, lane i
  // supplies row 8 hh + 4 rd + (i >> 2) (+16 t'), 4 columns at
  // 32 mo + 16 (g & 1) + 4 (i & 3); it receives V[key0 + 0..3][dv0 + i].
  int vread[D / 32];
  {
    const int g = lane >> 4, i = lane & 15;
    const int qr = i >> 2, p = i & 3;
    const int sw = swz_v<C::CPR>(qr);  // rows differ from qr only above bit 1
#pragma unroll
    for (int mo = 0; mo < D / 32; ++mo) {
      const int col = 32 * mo + 16 * (g & 1) + 4 * p;
      vread[mo] = 2 * C::TB + (8 * hh + qr) * C::RB + (((col >> 3) ^ sw) << 4) + ((col & 7) << 1);
    }
  }

  const unsigned lds_base = (unsigned)(size_t)(__attribute__((address_space(3))) unsigned char *)lds;
  const unsigned wdst = lds_base + wave * C::LI * 1024;
  // the direct loads of one tile: first row k0t (<= N - KT), LDS offset dst
  auto tile_base = [&](const uint16_t *base, int64_t sn, int k0t) __attribute__((always_inline)) { return base + (int64_t)k0t * sn; };
  auto issue_tile = [&](const uint16_t *tp, const unsigned (&off)[C::LI], unsigned dst) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < C::LI; ++i) dma16(tp, off[i], dst + i * 1024);
  };

  // Stage of keys [k0, k0 + KT) reaching past N: its tile starts at
  // k0t = min(k0, N - KT); keys of the tile before k0 (they belong to the
  // previous stage) or at N and beyond are masked.
  auto mask_tail = [&](f32x16 (&sacc)[MT], int k0) __attribute__((always_inline)) {
    const int k0t = min(k0, kmax);
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int g = r >> 2, i = r & 3;
        const int key = k0t + 32 * mt + 16 * (g >> 1) + 8 * hh + 4 * (g & 1) + i;
        if (key < k0 || key >= N) sacc[mt][r] = -INFINITY;
      }
  };
  auto rescale_o = [&]() __attribute__((always_inline)) {
    if (__ballot(alpha != 1.f)) {
#pragma unroll
      for (int mo = 0; mo < D / 32; ++mo)
#pragma unroll
        for (int r = 0; r < 16; ++r) oacc[mo][r] *= alpha;
      alpha = 1.f;
    }
  };

  // ---- the softmax of one stage, in chunks that the iteration spreads over
  // its MFMA slots (exp2 domain, c2 = scale * log2 e).  P is rounded to bf16
  // for the P.V product, and the row sum adds up the same rounded values (two
  // at a time with v_dot2 against (1, 1)), so each output is an exact convex
  // combination of V rows up to fp32 accumulation.
  constexpr int SC = MT * 16;               // scores per lane per stage
  constexpr int XA = MT == 1 ? SC : SC / 2;  // scores turned into P in part A
  const bf16x2 ones = {(__bf16)1.f, (__bf16)1.f};
  struct Soft {
    float m0, m1, msub, ps0, ps1, es0, es1;
  };
  // max over scores [x, x + 4)
  auto sm_max = [&](Soft &st, const f32x16 (&sc)[MT], int x) __attribute__((always_inline)) {
    st.m0 = __builtin_fmaxf(__builtin_fmaxf(st.m0, sc[x >> 4][x & 15]), sc[(x + 1) >> 4][(x + 1) & 15]);
    st.m1 = __builtin_fmaxf(__builtin_fmaxf(st.m1, sc[(x + 2) >> 4][(x + 2) & 15]), sc[(x + 3) >> 4][(x + 3) & 15]);
    anchor(st.m0);
    anchor(st.m1);
  };
  auto sm_alpha = [&](Soft &st) __attribute__((always_inline)) {
    const float2 hv = halves(__builtin_fmaxf(st.m0, st.m1));
    const float mtile = __builtin_fmaxf(hv.x, hv.y) * c2;
    const bool grow = mtile > mrun + kRescaleSlack;
    const float mnew = grow ? mtile : mrun;
    // exp2(mrun - mnew): 1 without growth, 0 from an empty start
    const float a = __builtin_amdgcn_exp2f(mnew == -INFINITY ? 0.f : mrun - mnew);
    alpha *= a;
    mrun = mnew;
    lrun *= a;
    if constexpr (WITH_LSE) lexact *= a;
    st.msub = (mnew == -INFINITY) ? 0.f : mnew;
    anchor(st.msub);
    anchor(a);
  };
  // P for scores x, x + 1
  auto sm_exp = [&](Soft &st, const f32x16 (&sc)[MT], bf16x8 (&pc)[KT / 16], int x) __attribute__((always_inline)) {
    const float v0 = __builtin_amdgcn_exp2f(fmaf(sc[x >> 4][x & 15], c2, -st.msub));
    const float v1 = __builtin_amdgcn_exp2f(fmaf(sc[(x + 1) >> 4][(x + 1) & 15], c2, -st.msub));
    const bf16x2 pp = {(__bf16)v0, (__bf16)v1};
    anchor(__builtin_bit_cast(float, pp));
    pc[x >> 3][x & 7] = pp[0];
    pc[x >> 3][(x & 7) + 1] = pp[1];
    if (((x >> 1) & 1) == 0) st.ps0 = __builtin_amdgcn_fdot2_f32_bf16(pp, ones, st.ps0, false);
    else st.ps1 = __builtin_amdgcn_fdot2_f32_bf16(pp, ones, st.ps1, false);
    if constexpr (WITH_LSE) {
      if (((x >> 1) & 1) == 0) st.es0 += v0 + v1;
      else st.es1 += v0 + v1;
    }
  };
  auto sm_done = [&](Soft &st) __attribute__((always_inline)) {
    lrun += st.ps0 + st.ps1;
    if constexpr (WITH_LSE) lexact += st.es0 + st.es1;
    anchor(lrun);
  };

  constexpr int PF = 4;  // operand reads run this many MFMA slots ahead
  // plain S^T = K Q^T into sacc from K slot KS (prologue)
  auto qk_plain = [&](f32x16 (&sacc)[MT]) __attribute__((always_inline)) {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
#pragma unroll
      for (int t = 0; t < D / 16; ++t) {
        const bf16x8 a = *reinterpret_cast<const bf16x8 *>(lds + kread[t] + mt * 32 * C::RB);
        if (t == 0) sacc[mt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qreg[t], f32x16{}, 0, 0, 0);
        else sacc[mt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qreg[t], sacc[mt], 0, 0, 0);
      }
    }
  };

  // ---- one iteration (VS: V slot of stage j-1, KS: K slot of stage j+1;
  // HAS_PV false for j = 0).  The direct loads of V(j) (tile vtp into LDS
  // vdst) and of K(j+2) (ktp, kdst) go one per MFMA slot at the start of
  // part A: issued in one burst they stall the wave behind the vector memory
  // queue, and issued late they are not there at the next iteration.
  auto iterate = [&](auto has_pv, auto vs_c, auto ks_c, f32x16 (&sc)[MT], const bf16x8 (&pprev)[KT / 16],
                     bf16x8 (&pcur)[KT / 16], const uint16_t *vtp, unsigned vdst, const uint16_t *ktp,
                     unsigned kdst) __attribute__((always_inline)) {
    constexpr bool HP = decltype(has_pv)::value;
    constexpr int VS = decltype(vs_c)::value, KS = decltype(ks_c)::value;
    constexpr int NPV = (KT / 16) * (D / 32);  // PV MFMAs
    constexpr int NQK = MT * (D / 16);         // QK MFMAs
    static_assert(NPV >= 2 * C::LI, "load slots");
    Soft st{-INFINITY, -INFINITY, 0.f, 0.f, 0.f, 0.f, 0.f};
    // part A: PV(j-1) | max, alpha, P for the first half of the scores
    {
      bf16x8 vf[NPV];
      auto vrd = [&](int i) __attribute__((always_inline)) {
        const int tp = i / (D / 32), mo = i % (D / 32);
        const int base = vread[mo] + VS * C::TB + 16 * tp * C::RB;
        const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)(lds + base));
        const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)(lds + base + 4 * C::RB));
        vf[i] = __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
      };
      // chunk plan over NPV slots: SC/4 max chunks, the alpha chunk and the
      // exp pairs of part A (all of them when a stage is one 32-key tile,
      // whose scores part B overwrites at once; else the first half)
      constexpr int NCA = SC / 4 + 1 + XA / 2 + (MT == 1 ? 1 : 0);
      if constexpr (HP) {
#pragma unroll
        for (int i = 0; i < PF; ++i) vrd(i);
      }
#pragma unroll
      for (int sl = 0; sl < NPV; ++sl) {
        if constexpr (HP) {
          if (sl + PF < NPV) vrd(sl + PF);
          const int tp = sl / (D / 32), mo = sl % (D / 32);
          oacc[mo] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[sl], pprev[tp], oacc[mo], 0, 0, 0);
        }
        if (sl < C::LI) dma16(vtp, voff[sl], vdst + sl * 1024);
        else if (sl < 2 * C::LI) dma16(ktp, koff[sl - C::LI], kdst + (sl - C::LI) * 1024);
#pragma unroll
        for (int c = 0; c < NCA; ++c) {
          if (c * NPV / NCA != sl) continue;
          if (c < SC / 4) sm_max(st, sc, 4 * c);
          else if (c == SC / 4) sm_alpha(st);
          else if (c < SC / 4 + 1 + XA / 2) sm_exp(st, sc, pcur, 2 * (c - SC / 4 - 1));
          else sm_done(st);
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    // part B: S(j+1) | P for the second half
    {
      bf16x8 kf[NQK];
      auto krd = [&](int i) __attribute__((always_inline)) {
        const int mt = i / (D / 16), t = i % (D / 16);
        kf[i] = *reinterpret_cast<const bf16x8 *>(lds + kread[t] + KS * C::TB + mt * 32 * C::RB);
      };
#pragma unroll
      for (int i = 0; i < PF; ++i) krd(i);
      // the second half of the scores is consumed during the first QK tile
      constexpr int NCB = MT == 1 ? 0 : (SC - XA) / 2 + 1;
#pragma unroll
      for (int sl = 0; sl < NQK; ++sl) {
        if (sl + PF < NQK) krd(sl + PF);

        const int mt = sl / (D / 16), t = sl % (D / 16);
        if (t == 0) sc[mt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[sl], qreg[t], f32x16{}, 0, 0, 0);
        else sc[mt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[sl], qreg[t], sc[mt], 0, 0, 0);
        constexpr int SB = (MT == 1 ? NQK : NQK / MT);  // slots before the last tile
#pragma unroll
        for (int c = 0; c < NCB; ++c) {
          if (c * SB / NCB != sl) continue;
          if (c < (SC - XA) / 2) sm_exp(st, sc, pcur, XA + 2 * c);
          else sm_done(st);
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  };

  if (e1 > e0) {
    f32x16 sc[MT];
    bf16x8 pa[KT / 16], pb[KT / 16];
    using T = std::true_type;
    using F = std::false_type;
    using I0 = std::integral_constant<int, 0>;
    using I1 = std::integral_constant<int, 1>;
    const int L = e1 - e0;  // key blocks of the row; stages 2b and 2b+1 are block b
    int *list = reinterpret_cast<int *>(lds + C::LIST);
    // prologue: K(0), K(1) (both halves of block 0), the row's list into LDS;
    // S(0)
    int blk0 = min(max(col_idx[e0], 0), nB - 1);
    int blk1 = L > 1 ? min(max(col_idx[e0 + 1], 0), nB - 1) : 0;
    {
      const int k0 = blk0 * BS;
      issue_tile(tile_base(kbase, k.sn, min(k0, kmax)), koff, wdst);
      issue_tile(tile_base(kbase, k.sn, min(k0 + KT, kmax)), koff, wdst + C::TB);
    }
    for (int i = threadIdx.x; i < L; i += C::NT) list[i] = min(max(col_idx[e0 + i], 0), nB - 1);
    asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");
    qk_plain(sc);
    if (blk0 * BS + KT > N) mask_tail(sc, blk0 * BS);

    // Stages come in pairs (both halves of block b): iteration 2b loads V(2b)
    // (first half of block b) and K(2b+2) (first half of block b+1),
    // iteration 2b+1 the second halves.  blk0 / blk1 hold blocks b and b+1;
    // block b+2 is read from the LDS list one pair ahead.
    auto pair = [&](auto first, int b) __attribute__((always_inline)) {
      const int nxt = list[min(b + 2, L - 1)];
      const bool more = b + 1 < L;
      // even stage j = 2b
      wait_all_then_barrier();
      if constexpr (!decltype(first)::value) rescale_o();
      {
        const int kv = blk0 * BS;
        const int kk = more ? blk1 * BS : 0;
        iterate(std::integral_constant<bool, !decltype(first)::value>{}, I1{}, I1{}, sc, pb, pa,
                tile_base(vbase, v.sn, min(kv, kmax)), wdst + 2 * C::TB,
                tile_base(kbase, k.sn, min(kk, kmax)), wdst);
        if (blk0 * BS + 2 * KT > N) mask_tail(sc, blk0 * BS + KT);  // S(2b+1)
      }
      // odd stage j = 2b+1
      wait_all_then_barrier();
      rescale_o();
      {
        const int kv = blk0 * BS + KT;
        const int kk = more ? blk1 * BS + KT : 0;
        iterate(T{}, I0{}, I0{}, sc, pa, pb, tile_base(vbase, v.sn, min(kv, kmax)), wdst + 3 * C::TB,
                tile_base(kbase, k.sn, min(kk, kmax)), wdst + C::TB);
        if (more && blk1 * BS + KT > N) mask_tail(sc, blk1 * BS);  // S(2b+2)
      }
      blk0 = blk1;
      blk1 = __builtin_amdgcn_readfirstlane(nxt);
    };
    pair(T{}, 0);
    for (int b = 1; b < L; ++b) pair(F{}, b);
    // P.V of the last stage (odd: V slot 1, P in pb)
    wait_all_then_barrier();
    rescale_o();
    auto pv_last = [&](auto vs_c, const bf16x8 (&pl)[KT / 16]) __attribute__((always_inline)) {
#pragma unroll
      for (int tp = 0; tp < KT / 16; ++tp)
#pragma unroll
        for (int mo = 0; mo < D / 32; ++mo) {
          const int base = vread[mo] + decltype(vs_c)::value * C::TB + 16 * tp * C::RB;
          const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)(lds + base));
          const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)(lds + base + 4 * C::RB));
          const bf16x8 av = __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
          oacc[mo] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, pl[tp], oacc[mo], 0, 0, 0);
        }
    };
    pv_last(I1{}, pb);
  }

  // ---- epilogue: normalise, store bf16 O (and the LSE)
  const float2 lh = halves(lrun);
  const float ltot = lh.x + lh.y;
  const float inv = ltot > 0.f ? 1.f / ltot : 0.f;
  if (qtok < N) {
    uint16_t *op = out + (int64_t)b * osb + (int64_t)h * osh + (int64_t)qtok * osn + 4 * hh;
#pragma unroll
    for (int mo = 0; mo < D / 32; ++mo)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        bf16x4 o4;
#pragma unroll
        for (int i = 0; i < 4; ++i) o4[i] = (__bf16)(oacc[mo][4 * g + i] * inv);
        *reinterpret_cast<bf16x4 *>(op + 32 * mo + 8 * g) = o4;
      }
    if constexpr (WITH_LSE) {
      const float2 eh = halves(lexact);
      const float etot = eh.x + eh.y;
      if (hh == 0)
        lse[(int64_t)bh * N + qtok] = etot > 0.f ? (mrun + __log2f(etot)) * 0.69314718055994531f : -INFINITY;
    }
  }
}

}  // namespace

hipError_t launch_bsattn(View q, View k, View v, uint16_t *out, int64_t osb, int64_t osh,
                         int64_t osn, int B, int H, int N, int d, int bs, const int32_t *row_ptr,
                         const int32_t *col_idx, const int32_t *order, const int32_t *n_rows,
                         float scale, float *lse, hipStream_t s) {
  const int nB = (N + bs - 1) / bs;
  const unsigned R = (unsigned)B * H * nB;
  const float c2 = scale * 1.4426950408889634f;
  hipError_t e = hipSuccess;
#define CARNATOR_BSATTN_L(DD, BB, LL)                                                             \
  do {                                                                                            \
    using C = Cfg<DD, BB>;                                                                        \
    e = hipFuncSetAttribute(reinterpret_cast<const void *>(&bsattn_kernel<DD, BB, LL>),           \
                            hipFuncAttributeMaxDynamicSharedMemorySize, C::LDS);                  \
    if (e != hipSuccess) return e;                                                                \
    hipLaunchKernelGGL((bsattn_kernel<DD, BB, LL>), dim3(R), dim3(C::NT), C::LDS, s, q, k, v,     \
                       out, osb, osh, osn, H, N, nB, row_ptr, col_idx, order, n_rows, c2, lse);   \
  } while (0)
#define CARNATOR_BSATTN(DD, BB)                  \
  do {                                           \
    if (lse) CARNATOR_BSATTN_L(DD, BB, true);    \
    else CARNATOR_BSATTN_L(DD, BB, false);       \
  } while (0)
  if (d == 128 && bs == 128) CARNATOR_BSATTN(128, 128);
  else if (d == 128 && bs == 64) CARNATOR_BSATTN(128, 64);
  else if (d == 64 && bs == 128) CARNATOR_BSATTN(64, 128);
  else CARNATOR_BSATTN(64, 64);
#undef CARNATOR_BSATTN
#undef CARNATOR_BSATTN_L
  return hipGetLastError();
}

}  // namespace carnator
