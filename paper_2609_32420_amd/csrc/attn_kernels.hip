// Block-sparse attention under a reused block mask (Sec. 3.3, historical
// sparse-connectivity reuse; Appendix C.3): the target's Q, K, V are
// recomputed and only the key blocks listed for a query block are visited.
//
// One workgroup per query block (BS queries, BS/32 waves of 32 queries).  The
// workgroup walks its compacted key-block list in sub-tiles of 64 keys:
// K and V^T sub-tiles are staged into LDS (double-buffered: the global loads
// of sub-tile s+1 are in flight while sub-tile s is computed), S^T = K Q^T and
// O^T += V^T P^T run on bf16 MFMA 32x32x16 with fp32 accumulation, and the
// online softmax runs in fp32 in the exp2 domain.
//
// Computing S^T (keys as MFMA rows, queries as columns) puts every score of a
// query in one lane pair (lane q and lane q+32), so the row max is one
// cross-lane swap and the row sum stays lane-local until the end.  The key
// order inside a 32-key MFMA tile is permuted (bits 2 and 3 of the row index
// swapped) so that the accumulator registers of S^T are directly the B operand
// of the P.V product, and the matching V^T operand is one contiguous 16-byte
// LDS read.
#include "internal.h"

#include <math.h>

namespace carnator {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int KT = 64;  // keys per sub-tile
// s_waitcnt immediate: vmcnt(0), expcnt and lgkmcnt left at their maxima.
constexpr int kWaitVm0 = 0x0F70;

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
// P may then reach 2^8, harmless in fp32 and bf16, and most sub-tiles skip the
// rescale of the 64 output accumulators.
constexpr float kRescaleSlack = 8.f;

// LDS rows are padded by 16 bytes.  For the 16 lanes that share a bank cycle
// of a 16-byte read (rows 32*mt + perm32(0..15) of K, rows 0..15 of V^T) the
// padding puts the 16-byte slots on distinct banks, and every operand read is
// a lane base plus a compile-time offset.
template <int D, int BS>
struct Cfg {
  static constexpr int WAVES = BS / 32;
  static constexpr int NT = 64 * WAVES;          // == 2 * BS
  static constexpr int KCH = D / 8;              // 16-B chunks per K row
  static constexpr int KROW = D * 2 + 16;        // bytes per K row (padded)
  static constexpr int VROW = KT * 2 + 16;       // bytes per V^T row (padded)
  static constexpr int KBYTES = KT * KROW;
  static constexpr int VBYTES = D * VROW;
  static constexpr int STAGE = KBYTES + VBYTES;
  static constexpr int LDS = 2 * STAGE;
  static constexpr int KCHUNKS = KT * KCH;       // K chunks per stage
  static constexpr int NCHUNK = (KCHUNKS + D * 8) / NT;  // chunks per thread
  static constexpr int KPT = KCHUNKS / NT;       // of which K
  static_assert(KCHUNKS % NT == 0 && (D * 8) % NT == 0, "stage split");
};

// Two waves per SIMD (two workgroups per CU); the d=128 / block-64 variant
// keeps its 16 staging chunks in registers at one wave per SIMD.
template <int D, int BS>
__global__ void __launch_bounds__(2 * BS, (D == 128 && BS == 64) ? 1 : 2)
bsattn_kernel(View q, View k, const uint16_t *__restrict__ vt, uint16_t *__restrict__ out,
              int64_t osb, int64_t osh, int64_t osn, int H, int N, int nB,
              const int32_t *__restrict__ row_ptr, const int32_t *__restrict__ col_idx,
              const int32_t *__restrict__ order, float c2, float *__restrict__ lse) {
  using C = Cfg<D, BS>;
  extern __shared__ __attribute__((aligned(16))) unsigned char lds[];

  const int row = order[blockIdx.x];
  const int bh = row / nB;
  const int qb = row - bh * nB;
  const int b = bh / H, h = bh - b * H;
  const int e0 = row_ptr[row], e1 = row_ptr[row + 1];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int l32 = lane & 31, hh = lane >> 5;
  const int qtok = qb * BS + wave * 32 + l32;
  const int64_t Npad = (int64_t)nB * BS;
  const int tail = N - (nB - 1) * BS;
  const int tail_sub = (tail + KT - 1) / KT;

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

  f32x16 oacc[D / 32];
#pragma unroll
  for (int mo = 0; mo < D / 32; ++mo)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[mo][r] = 0.f;
  float mrun = -INFINITY, lrun = 0.f;

  const uint16_t *kbase = k.data + (int64_t)b * k.sb + (int64_t)h * k.sh;
  const uint16_t *vbase = vt + (int64_t)bh * D * Npad;

  // per-lane staging offsets (bytes): global (relative to the sub-tile's first
  // key) and LDS (relative to the stage)
  int goff[C::NCHUNK], soff[C::NCHUNK], krow[C::KPT];
#pragma unroll
  for (int c = 0; c < C::NCHUNK; ++c) {
    const int f = threadIdx.x + C::NT * c;
    if (c < C::KPT) {
      const int r = f / C::KCH, cc = f % C::KCH;
      krow[c] = r;
      goff[c] = (int)(r * k.sn + cc * 8) * 2;
      soff[c] = r * C::KROW + cc * 16;
    } else {
      const int fv = f - C::KCHUNKS;
      const int dv = fv >> 3, cc = fv & 7;
      goff[c] = (int)(dv * Npad + cc * 8) * 2;
      soff[c] = C::KBYTES + dv * C::VROW + cc * 16;
    }
  }
  // operand-read lane bases inside a stage
  const int kread = perm32(l32) * C::KROW + hh * 16;
  const int vread = C::KBYTES + l32 * C::VROW + hh * 16;

  int e = e0, s = 0;
  auto nsub = [&](int j) { return j == nB - 1 ? tail_sub : BS / KT; };
  uint4 stg[C::NCHUNK];
  auto gload = [&](int ee, int ss) {
    const int k0 = col_idx[ee] * BS + ss * KT;
    const char *kt = reinterpret_cast<const char *>(kbase + (int64_t)k0 * k.sn);
    const char *vtp = reinterpret_cast<const char *>(vbase + k0);
    if (k0 + KT <= N) {
#pragma unroll
      for (int c = 0; c < C::NCHUNK; ++c)
        stg[c] = *reinterpret_cast<const uint4 *>((c < C::KPT ? kt : vtp) + goff[c]);
    } else {
      // partial last block: K rows past N read as zero (V^T is zero-padded)
#pragma unroll
      for (int c = 0; c < C::NCHUNK; ++c) {
        if (c < C::KPT) {
          uint4 w = make_uint4(0, 0, 0, 0);
          if (k0 + krow[c] < N) w = *reinterpret_cast<const uint4 *>(kt + goff[c]);
          stg[c] = w;
        } else {
          stg[c] = *reinterpret_cast<const uint4 *>(vtp + goff[c]);
        }
      }
    }
  };
  auto sstore = [&](int buf) {
    unsigned char *base = lds + buf * C::STAGE;
#pragma unroll
    for (int c = 0; c < C::NCHUNK; ++c) *reinterpret_cast<uint4 *>(base + soff[c]) = stg[c];
  };

  int buf = 0;
  if (e < e1) {
    gload(e, s);
    sstore(0);
  }
  // Every global load issued so far (Q fragment, first sub-tile) has landed
  // here; saying so explicitly lets the loop below keep the next sub-tile's
  // loads in flight across the MFMAs instead of draining them each iteration.
  __builtin_amdgcn_s_waitcnt(kWaitVm0);
  __syncthreads();

  while (e < e1) {
    const int j = col_idx[e];
    const int k0 = j * BS + s * KT;
    int en = e, sn = s + 1;
    if (sn >= nsub(j)) {
      en = e + 1;
      sn = 0;
    }
    const bool has_next = en < e1;
    if (has_next) gload(en, sn);

    const unsigned char *stage = lds + buf * C::STAGE;

    // ---- S^T = K Q^T for 64 keys x 32 queries (two 32-key MFMA tiles)
    f32x16 sacc[2];
#pragma unroll
    for (int mt = 0; mt < 2; ++mt) {
#pragma unroll
      for (int r = 0; r < 16; ++r) sacc[mt][r] = 0.f;
#pragma unroll
      for (int t = 0; t < D / 16; ++t) {
        const bf16x8 a = *reinterpret_cast<const bf16x8 *>(stage + kread + mt * 32 * C::KROW + t * 32);
        sacc[mt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qreg[t], sacc[mt], 0, 0, 0);
      }
    }
    // keys past N (only in the partial last block)
    if (k0 + KT > N) {
#pragma unroll
      for (int mt = 0; mt < 2; ++mt)
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
    for (int mt = 0; mt < 2; ++mt)
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
      mrun = mnew;
    }
    const float msub = (mrun == -INFINITY) ? 0.f : mrun;
    float psum[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int mt = 0; mt < 2; ++mt)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float p = __builtin_amdgcn_exp2f(fmaf(sacc[mt][r], c2, -msub));
        sacc[mt][r] = p;
        psum[r & 3] += p;
      }
    lrun += (psum[0] + psum[1]) + (psum[2] + psum[3]);

    // ---- O^T += V^T P^T over 4 key steps of 16
#pragma unroll
    for (int tp = 0; tp < KT / 16; ++tp) {
      const int mt = tp >> 1, a = tp & 1;
      bf16x8 pb;
#pragma unroll
      for (int jj = 0; jj < 8; ++jj) pb[jj] = (__bf16)sacc[mt][8 * a + jj];
#pragma unroll
      for (int mo = 0; mo < D / 32; ++mo) {
        const bf16x8 av = *reinterpret_cast<const bf16x8 *>(stage + vread + mo * 32 * C::VROW + tp * 32);
        oacc[mo] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, pb, oacc[mo], 0, 0, 0);
      }
    }

    if (has_next) sstore(buf ^ 1);
    __syncthreads();
    buf ^= 1;
    e = en;
    s = sn;
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
    if (lse != nullptr && hh == 0)
      lse[(int64_t)bh * N + qtok] = ltot > 0.f ? (mrun + __log2f(ltot)) * 0.69314718055994531f : -INFINITY;
  }
}

// V [B,H,N,d] -> V^T [BH][d][nB*bs], keys contiguous, zero past N.
template <int D>
__global__ void __launch_bounds__(256) transpose_v_kernel(View v, int H, int N, int64_t Npad,
                                                          uint16_t *__restrict__ vt) {
  __shared__ uint16_t tile[64][D + 8];
  const int bh = blockIdx.y;
  const int b = bh / H, h = bh - b * H;
  const int k0 = blockIdx.x * 64;
  const uint16_t *base = v.data + (int64_t)b * v.sb + (int64_t)h * v.sh;
  for (int f = threadIdx.x; f < 64 * D / 8; f += 256) {
    const int r = f / (D / 8), c = f % (D / 8);
    uint4 w = make_uint4(0, 0, 0, 0);
    if (k0 + r < N) w = *reinterpret_cast<const uint4 *>(base + (int64_t)(k0 + r) * v.sn + c * 8);
    *reinterpret_cast<uint4 *>(&tile[r][c * 8]) = w;
  }
  __syncthreads();
  uint16_t *dst = vt + (int64_t)bh * D * Npad + k0;
  for (int f = threadIdx.x; f < D * 8; f += 256) {
    const int dv = f >> 3, c = f & 7;
    uint16_t x[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) x[e] = tile[c * 8 + e][dv];
    uint4 w;
    w.x = x[0] | ((uint32_t)x[1] << 16);
    w.y = x[2] | ((uint32_t)x[3] << 16);
    w.z = x[4] | ((uint32_t)x[5] << 16);
    w.w = x[6] | ((uint32_t)x[7] << 16);
    *reinterpret_cast<uint4 *>(dst + (int64_t)dv * Npad + c * 8) = w;
  }
}

}  // namespace

hipError_t launch_transpose_v(View v, int B, int H, int N, int d, int bs, uint16_t *vt,
                              hipStream_t s) {
  const int nB = (N + bs - 1) / bs;
  const int64_t Npad = (int64_t)nB * bs;
  dim3 grid((unsigned)(Npad / 64), B * H);
  if (d == 128)
    hipLaunchKernelGGL(transpose_v_kernel<128>, grid, dim3(256), 0, s, v, H, N, Npad, vt);
  else
    hipLaunchKernelGGL(transpose_v_kernel<64>, grid, dim3(256), 0, s, v, H, N, Npad, vt);
  return hipGetLastError();
}

hipError_t launch_bsattn(View q, View k, const uint16_t *vt, uint16_t *out, int64_t osb,
                         int64_t osh, int64_t osn, int B, int H, int N, int d, int bs,
                         const int32_t *row_ptr, const int32_t *col_idx, const int32_t *order,
                         float scale, float *lse, hipStream_t s) {
  const int nB = (N + bs - 1) / bs;
  const unsigned R = (unsigned)B * H * nB;
  const float c2 = scale * 1.4426950408889634f;
  hipError_t e = hipSuccess;
#define CARNATOR_BSATTN(DD, BB)                                                                   \
  do {                                                                                            \
    using C = Cfg<DD, BB>;                                                                        \
    e = hipFuncSetAttribute(reinterpret_cast<const void *>(&bsattn_kernel<DD, BB>),               \
                            hipFuncAttributeMaxDynamicSharedMemorySize, C::LDS);                  \
    if (e != hipSuccess) return e;                                                                \
    hipLaunchKernelGGL((bsattn_kernel<DD, BB>), dim3(R), dim3(C::NT), C::LDS, s, q, k, vt, out,   \
                       osb, osh, osn, H, N, nB, row_ptr, col_idx, order, c2, lse);                \
  } while (0)
  if (d == 128 && bs == 128) CARNATOR_BSATTN(128, 128);
  else if (d == 128 && bs == 64) CARNATOR_BSATTN(128, 64);
  else if (d == 64 && bs == 128) CARNATOR_BSATTN(64, 128);
  else CARNATOR_BSATTN(64, 64);
#undef CARNATOR_BSATTN
  return hipGetLastError();
}

}  // namespace carnator
