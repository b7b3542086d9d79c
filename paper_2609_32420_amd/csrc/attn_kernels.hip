// Block-sparse attention under a reused block mask (Sec. 3.3, historical
// sparse-connectivity reuse; Appendix C.3): the target's Q, K, V are
// recomputed and only the key blocks listed for a query block are visited.
//
// One workgroup per query block (BS queries, BS/32 waves of 32 queries).  The
// workgroup walks its compacted key-block list in stages of 32 keys.  K and V
// stages are copied from HBM straight into LDS (global_load_lds, no register
// staging) through a ring of four buffers, three stages ahead of the one being
// computed, so a load has three stages of MFMA work to land.  S^T = K Q^T and
// O^T += V^T P^T run on bf16 MFMA 32x32x16 with fp32 accumulation; the online
// softmax runs in fp32 in the exp2 domain.
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

namespace carnator {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

// Keys per stage and ring depth (see Cfg).
constexpr int kStageKeys = 64;
constexpr int kRing = 2;

// s_waitcnt immediate: vmcnt(0) with expcnt and lgkmcnt left at their maxima.
constexpr int kWaitVm0 = 0x0F70;

// The stage ring is driven by hand: the direct loads, the wait for the oldest
// stage and the barrier are written as inline assembly.  Issued through the
// compiler builtin, a direct load makes every later LDS read look like it may
// alias the transfer, and the compiler then drains all outstanding stages
// (vmcnt(0)) before each barrier and each operand read, which removes the
// prefetch.  Nothing else in this kernel uses M0.
//
// 16 bytes per lane from `g` to LDS offset lds_off + 16 * lane (lds_off is
// the same in every lane).
__device__ inline void dma16(const void *g, unsigned lds_off) {
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(g),
               "s"(__builtin_amdgcn_readfirstlane(lds_off))
               : "memory");
}
// Wait until at most N direct loads of this wave are in flight and every LDS
// read of this wave has returned, then meet the other waves.
template <int N>
__device__ inline void wait_then_barrier() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(N) : "memory");
}

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

template <int D, int BS, int KT_ = kStageKeys, int NST_ = kRing>
struct Cfg {
  static constexpr int KT = KT_;              // keys per stage
  static constexpr int NST = NST_;            // stages in the LDS ring
  static constexpr int MT = KT / 32;          // 32-key MFMA tiles per stage
  static constexpr int WAVES = BS / 32;
  static constexpr int NT = 64 * WAVES;       // == 2 * BS
  static constexpr int RB = D * 2;            // bytes per K or V row
  static constexpr int CPR = D / 8;           // 16-byte chunks per row
  static constexpr int TB = KT * RB;          // bytes of one K (or V) stage
  static constexpr int STAGE = 2 * TB;
  static constexpr int LDS = NST * STAGE;
  static constexpr int LI = TB / 1024 / WAVES;  // 1-KiB direct loads per wave for K (and for V)
  static constexpr int LIW = 2 * LI;            // direct loads per wave per stage
  static_assert(TB % (1024 * WAVES) == 0, "stage split");
  static_assert(NST >= 2 && NST <= 4, "ring depth");
};

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

// Two waves per SIMD (two workgroups per CU).  WITH_LSE adds the exact fp32
// row sum the log-sum-exp output needs.
template <int D, int BS, bool WITH_LSE>
__global__ void __launch_bounds__(2 * BS, 2)
bsattn_kernel(View q, View k, View v, uint16_t *__restrict__ out, int64_t osb, int64_t osh,
              int64_t osn, int H, int N, int nB, const int32_t *__restrict__ row_ptr,
              const int32_t *__restrict__ col_idx, const int32_t *__restrict__ order, float c2,
              float *__restrict__ lse) {
  using C = Cfg<D, BS>;
  constexpr int KT = C::KT, NST = C::NST, MT = C::MT;
  extern __shared__ __attribute__((aligned(1024))) unsigned char lds[];

  const int row = order[blockIdx.x];
  const int bh = row / nB;
  const int qb = row - bh * nB;
  const int b = bh / H, h = bh - b * H;
  const int e0 = row_ptr[row], e1 = row_ptr[row + 1];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int l32 = lane & 31, hh = lane >> 5;
  const int qtok = qb * BS + wave * 32 + l32;
  const int tail = N - (nB - 1) * BS;
  const int tail_st = (tail + KT - 1) / KT;

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
  // the Q fragment is in registers before any stage load is issued
  __builtin_amdgcn_s_waitcnt(kWaitVm0);

  f32x16 oacc[D / 32];
#pragma unroll
  for (int mo = 0; mo < D / 32; ++mo)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[mo][r] = 0.f;
  float mrun = -INFINITY, lrun = 0.f, lexact = 0.f;

  const uint16_t *kbase = k.data + (int64_t)b * k.sb + (int64_t)h * k.sh;
  const uint16_t *vbase = v.data + (int64_t)b * v.sb + (int64_t)h * v.sh;

  // ---- direct-load descriptors: the i-th 1-KiB load of this wave fills
  // bytes [1024 n, 1024 n + 1024) of the K (V) stage, n = wave * LI + i; lane
  // l writes 16 bytes at 1024 n + 16 l, i.e. row r, slot s, which holds chunk
  // s ^ swz(r) of that key row.
  int ldrow[C::LI];
  int64_t koff[C::LI], voff[C::LI];
#pragma unroll
  for (int i = 0; i < C::LI; ++i) {
    const int byte = (wave * C::LI + i) * 1024 + lane * 16;
    const int r = byte / C::RB, s = (byte % C::RB) / 16;
    ldrow[i] = r;
    koff[i] = (int64_t)r * k.sn + (s ^ swz_k<C::CPR>(r)) * 8;
    voff[i] = (int64_t)r * v.sn + (s ^ swz_v<C::CPR>(r)) * 8;
  }

  // ---- operand-read lane offsets inside a stage
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
  int vrow_base;
  {
    const int g = lane >> 4, i = lane & 15;
    const int qr = i >> 2, p = i & 3;
    vrow_base = (8 * hh + qr) * C::RB + C::TB;
    const int sw = swz_v<C::CPR>(qr);  // rows differ from qr only above bit 1
#pragma unroll
    for (int mo = 0; mo < D / 32; ++mo) {
      const int col = 32 * mo + 16 * (g & 1) + 4 * p;
      vread[mo] = (((col >> 3) ^ sw) << 4) + ((col & 7) << 1);
    }
  }

  auto nst = [&](int j) { return j == nB - 1 ? tail_st : BS / KT; };

  // issue the direct loads of stage (ee, ss) into ring buffer `buf`
  const unsigned lds_base = (unsigned)(size_t)(__attribute__((address_space(3))) unsigned char *)lds;
  auto issue = [&](int ee, int ss, int buf) {
    const int k0 = col_idx[ee] * BS + ss * KT;
    const unsigned kdst = lds_base + buf * C::STAGE + wave * C::LI * 1024;
    const unsigned vdst = kdst + C::TB;
    if (k0 + KT <= N) {
      const uint16_t *kt = kbase + (int64_t)k0 * k.sn;
      const uint16_t *vt = vbase + (int64_t)k0 * v.sn;
#pragma unroll
      for (int i = 0; i < C::LI; ++i) {
        dma16(kt + koff[i], kdst + i * 1024);
        dma16(vt + voff[i], vdst + i * 1024);
      }
    } else {
      // partial last block: rows past N re-read row N-1 (finite values whose
      // scores are masked below)
#pragma unroll
      for (int i = 0; i < C::LI; ++i) {
        const int r = min(k0 + ldrow[i], N - 1) - ldrow[i];
        dma16(kbase + (int64_t)r * k.sn + koff[i], kdst + i * 1024);
        dma16(vbase + (int64_t)r * v.sn + voff[i], vdst + i * 1024);
      }
    }
  };

  // ---- prologue: the first NST-1 stages
  int el = e0, sl = 0, pend = 0, lbuf = 0;
  auto advance = [&](int &ee, int &ss) {
    if (++ss >= nst(col_idx[ee])) {
      ++ee;
      ss = 0;
    }
  };
#pragma unroll
  for (int p = 0; p < NST - 1; ++p) {
    if (el < e1) {
      issue(el, sl, lbuf);
      advance(el, sl);
      ++pend;
      lbuf = (lbuf + 1) % NST;
    }
  }

  int ec = e0, sc = 0, cbuf = 0;
  while (ec < e1) {
    // stage (ec, sc) has landed when at most (pend - 1) newer stages are in
    // flight; after the barrier every wave's part of it is in LDS and the
    // buffer computed last (the oldest) is free for the next load
    if constexpr (NST >= 4) {
      if (pend >= 3) wait_then_barrier<2 * C::LIW>();
      else if (pend == 2) wait_then_barrier<C::LIW>();
      else wait_then_barrier<0>();
    } else if constexpr (NST == 3) {
      if (pend >= 2) wait_then_barrier<C::LIW>();
      else wait_then_barrier<0>();
    } else {
      wait_then_barrier<0>();
    }
    --pend;
    if (el < e1) {
      issue(el, sl, lbuf);
      advance(el, sl);
      ++pend;
      lbuf = (lbuf + 1) % NST;
    }

    const int k0 = col_idx[ec] * BS + sc * KT;
    const unsigned char *stage = lds + cbuf * C::STAGE;

    // ---- S^T = K Q^T for KT keys x 32 queries (MT 32-key MFMA tiles)
    f32x16 sacc[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
#pragma unroll
      for (int r = 0; r < 16; ++r) sacc[mt][r] = 0.f;
#pragma unroll
      for (int t = 0; t < D / 16; ++t) {
        const bf16x8 a = *reinterpret_cast<const bf16x8 *>(stage + kread[t] + mt * 32 * C::RB);
        sacc[mt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qreg[t], sacc[mt], 0, 0, 0);
      }
    }
    // keys past N (only in the partial last block)
    if (k0 + KT > N) {
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int g = r >> 2, i = r & 3;
          const int key = 32 * mt + 16 * (g >> 1) + 8 * hh + 4 * (g & 1) + i;
          if (k0 + key >= N) sacc[mt][r] = -INFINITY;
        }
    }

    // ---- online softmax (exp2 domain, c2 = scale * log2 e)
    float mloc = sacc[0][0];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int r = 0; r < 16; ++r) mloc = fmaxf(mloc, sacc[mt][r]);
    {
      const float2 hv = halves(mloc);
      mloc = fmaxf(hv.x, hv.y);
    }
    const float mtile = mloc * c2;
    if (__ballot(mtile > mrun + kRescaleSlack)) {
      const float mnew = fmaxf(mrun, mtile);
      const float alpha = (mnew == -INFINITY) ? 1.f : __builtin_amdgcn_exp2f(mrun - mnew);
#pragma unroll
      for (int mo = 0; mo < D / 32; ++mo)
#pragma unroll
        for (int r = 0; r < 16; ++r) oacc[mo][r] *= alpha;
      lrun *= alpha;
      if constexpr (WITH_LSE) lexact *= alpha;
      mrun = mnew;
    }
    const float msub = (mrun == -INFINITY) ? 0.f : mrun;
    // P is rounded to bf16 for the P.V product, and the row sum adds up the
    // same rounded values (two at a time with v_dot2 against (1, 1)), so each
    // output is an exact convex combination of V rows up to fp32
    // accumulation: the rounding of P does not bias it.
    bf16x8 pb[KT / 16];
    float psum[2] = {0.f, 0.f}, esum[4] = {0.f, 0.f, 0.f, 0.f};
    const bf16x2 ones = {(__bf16)1.f, (__bf16)1.f};
#pragma unroll
    for (int tp = 0; tp < KT / 16; ++tp) {
#pragma unroll
      for (int jj = 0; jj < 8; jj += 2) {
        const float p0 = __builtin_amdgcn_exp2f(fmaf(sacc[tp >> 1][8 * (tp & 1) + jj], c2, -msub));
        const float p1 = __builtin_amdgcn_exp2f(fmaf(sacc[tp >> 1][8 * (tp & 1) + jj + 1], c2, -msub));
        const bf16x2 pp = {(__bf16)p0, (__bf16)p1};
        pb[tp][jj] = pp[0];
        pb[tp][jj + 1] = pp[1];
        psum[(jj >> 1) & 1] = __builtin_amdgcn_fdot2_f32_bf16(pp, ones, psum[(jj >> 1) & 1], false);
        if constexpr (WITH_LSE) {
          esum[jj >> 1] += p0;
          esum[jj >> 1] += p1;
        }
      }
    }
    lrun += psum[0] + psum[1];
    if constexpr (WITH_LSE) lexact += (esum[0] + esum[1]) + (esum[2] + esum[3]);

    // ---- O^T += V^T P^T over KT/16 key steps of 16
#pragma unroll
    for (int tp = 0; tp < KT / 16; ++tp) {
      const unsigned char *vrow = stage + vrow_base + 16 * tp * C::RB;
#pragma unroll
      for (int mo = 0; mo < D / 32; ++mo) {
        const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)(vrow + vread[mo]));
        const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)(vrow + 4 * C::RB + vread[mo]));
        const bf16x8 av = __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
        oacc[mo] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, pb[tp], oacc[mo], 0, 0, 0);
      }
    }

    advance(ec, sc);
    cbuf = (cbuf + 1) % NST;
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
                         const int32_t *col_idx, const int32_t *order, float scale, float *lse,
                         hipStream_t s) {
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
                       out, osb, osh, osn, H, N, nB, row_ptr, col_idx, order, c2, lse);           \
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
