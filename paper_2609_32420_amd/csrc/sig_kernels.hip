// Early-signature cosine scoring against a bank of cached signatures
// (Sec. 3.1: the target is compared against a bank built from completed
// requests; Sec. 4.1, candidate recall: rank by similarity, keep the top K).
//
// One pass over the bank per group of up to four queries: the queries are
// staged in LDS, one wave per bank row streams the row with 16-byte loads,
// <q, b> and |b|^2 accumulate in fp64 and a fixed-order wave reduction (so the
// result does not depend on scheduling) finishes each row.  Then a per-query
// top-k with the lower-row rule for near ties.
#include "internal.h"

#include <math.h>

#include <mutex>

// Scratch of the no-allocation entry point (carnator_signature_sim_noalloc):
// the fp64 cosines.  Each GPU the library runs on holds one copy until the
// process ends.  Host code never uses this name as an address: it asks the
// runtime for the array's device address (once per device).
static __device__ __align__(256) unsigned char scratch[carnator::kSigStaticScratchBytes];

namespace carnator {
namespace {

constexpr double kTieEps = 1e-6;
constexpr int kQChunk = 4;  // queries scored per pass over the bank

// One wave per bank row (grid-stride).  Scores queries [q0, q0 + nqc).  The
// wave streams its bank row and the query rows kU float4 per lane at a time,
// so the loads of a row are in flight together.  |q|^2 is accumulated in the
// same pass (every wave computes it in the same order, so every wave gets
// the same value) and no separate norm pass is needed.
constexpr int kU = 4;
__global__ void __launch_bounds__(256) scan_kernel(const float *__restrict__ query, int64_t q0,
                                                   int nqc, const float *__restrict__ bank,
                                                   int64_t m, int64_t dim, int64_t ld,
                                                   double *__restrict__ sims,
                                                   float *__restrict__ all_sim) {
  const int lane = threadIdx.x & 63;
  const int64_t nwaves = (int64_t)gridDim.x * 4;
  const int64_t d4 = dim / 4;
  const float *qbase = query + q0 * dim;
  for (int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); r < m; r += nwaves) {
    const float4 *bp = reinterpret_cast<const float4 *>(bank + r * ld);
    double bb = 0.0;
    double dot[kQChunk], qq2[kQChunk];
#pragma unroll
    for (int qq = 0; qq < kQChunk; ++qq) dot[qq] = qq2[qq] = 0.0;
    for (int64_t c0 = lane; c0 < d4; c0 += 64 * kU) {
      float4 x[kU];
#pragma unroll
      for (int u = 0; u < kU; ++u) {
        const int64_t c = c0 + 64 * u;
        x[u] = c < d4 ? bp[c] : make_float4(0.f, 0.f, 0.f, 0.f);
      }
#pragma unroll
      for (int qq = 0; qq < kQChunk; ++qq) {
        if (qq < nqc) {
          const float4 *qp = reinterpret_cast<const float4 *>(qbase + qq * dim);
          float4 y[kU];
#pragma unroll
          for (int u = 0; u < kU; ++u) {
            const int64_t c = c0 + 64 * u;
            y[u] = c < d4 ? qp[c] : make_float4(0.f, 0.f, 0.f, 0.f);
          }
          double d = dot[qq], n2 = qq2[qq];
#pragma unroll
          for (int u = 0; u < kU; ++u) {
            d = fma((double)x[u].x, (double)y[u].x, d);
            d = fma((double)x[u].y, (double)y[u].y, d);
            d = fma((double)x[u].z, (double)y[u].z, d);
            d = fma((double)x[u].w, (double)y[u].w, d);
            n2 = fma((double)y[u].x, (double)y[u].x, n2);
            n2 = fma((double)y[u].y, (double)y[u].y, n2);
            n2 = fma((double)y[u].z, (double)y[u].z, n2);
            n2 = fma((double)y[u].w, (double)y[u].w, n2);
          }
          dot[qq] = d;
          qq2[qq] = n2;
        }
      }
#pragma unroll
      for (int u = 0; u < kU; ++u) {
        bb = fma((double)x[u].x, (double)x[u].x, bb);
        bb = fma((double)x[u].y, (double)x[u].y, bb);
        bb = fma((double)x[u].z, (double)x[u].z, bb);
        bb = fma((double)x[u].w, (double)x[u].w, bb);
      }
    }
    const double bn = sqrt(wave_sum(bb));
#pragma unroll
    for (int qq = 0; qq < kQChunk; ++qq) {
      if (qq < nqc) {
        const double d = wave_sum(dot[qq]);
        const double den = sqrt(wave_sum(qq2[qq])) * bn;
        const double sv = den > 0.0 ? d / den : 0.0;
        if (lane == qq) {
          sims[(q0 + qq) * m + r] = sv;
          if (all_sim) all_sim[(q0 + qq) * m + r] = (float)sv;
        }
      }
    }
  }
}

// (value, index) ordered by descending value, lower index first.
__device__ inline bool better(double va, int ia, double vb, int ib) {
  return va > vb || (va == vb && ia < ib);
}

// ---- block-wide top-k --------------------------------------------------------
// One workgroup of 1024 threads per query; thread t owns rows t + 1024 u.
// Values are compared through an order-preserving map onto uint64 keys, and
// (key, row) pairs are ordered by descending key, lower row first.  Round r
// takes the best pair that comes after round r-1's pick in that order: every
// thread scans its rows, a wave reduction and an exchange of the 16 wave
// winners through LDS (one barrier) give every thread the same pick.  Rows of
// banks up to 8192 rows stay in registers; larger banks are re-read per
// round.
constexpr int kTkThreads = 1024;
constexpr int kTkWaves = kTkThreads / 64;
constexpr int kTkRegs = 8;

__device__ inline uint64_t okey(double v) {
  const uint64_t b = (uint64_t)__double_as_longlong(v);
  return (b >> 63) ? ~b : (b | 0x8000000000000000ull);
}
__device__ inline double okey_value(uint64_t k) {
  return __longlong_as_double((long long)((k >> 63) ? (k & 0x7fffffffffffffffull) : ~k));
}
__device__ inline bool kbetter(uint64_t ka, int xa, uint64_t kb, int xb) {
  return ka > kb || (ka == kb && xa < xb);
}

struct TkShared {
  uint64_t wk[2][kTkWaves];
  int wx[2][kTkWaves];
  uint64_t rk[64];
  int rx[64];
  int cnt[kTkWaves];
  double tv[64];
  int tx[64];
  uint64_t gmax[kTkThreads / 16];
  uint64_t ck[64];
  int cx[64];
  uint64_t theta;
  int ncand;
};

// Key of row x in the given mode: 0 ranks by value, 1 ranks rows within eps
// of cut above all others (so rounds then take the lowest such rows).
template <int MODE>
__device__ inline uint64_t mode_key(double v, double cut) {
  if (MODE == 0) return okey(v);
  return fabs(v - cut) <= kTieEps ? 1ull : 0ull;
}

template <int MODE>
__device__ inline void tk_rounds(const double (&vals)[kTkRegs], bool in_regs, const double *sv,
                                 int64_t m, int nsel, double cut, TkShared &sh, int round0) {
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  uint64_t pk = ~0ull;
  int px = -1;
  for (int r = 0; r < nsel; ++r) {
    uint64_t bk = 0;
    int bx = 0x7fffffff;
    if (in_regs) {
#pragma unroll
      for (int u = 0; u < kTkRegs; ++u) {
        const int x = t + kTkThreads * u;
        const uint64_t k = mode_key<MODE>(vals[u], cut);
        const bool ok = x < m && (k < pk || (k == pk && x > px)) && kbetter(k, x, bk, bx);
        bk = ok ? k : bk;
        bx = ok ? x : bx;
      }
    } else {
      for (int64_t x = t; x < m; x += kTkThreads) {
        const uint64_t k = mode_key<MODE>(sv[x], cut);
        const bool ok = (k < pk || (k == pk && (int)x > px)) && kbetter(k, (int)x, bk, bx);
        bk = ok ? k : bk;
        bx = ok ? (int)x : bx;
      }
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      const uint64_t ok = (uint64_t)__shfl_xor((long long)bk, o);
      const int ox = __shfl_xor(bx, o);
      const bool b = kbetter(ok, ox, bk, bx);
      bk = b ? ok : bk;
      bx = b ? ox : bx;
    }
    const int buf = (round0 + r) & 1;
    if (lane == 0) {
      sh.wk[buf][w] = bk;
      sh.wx[buf][w] = bx;
    }
    __syncthreads();
    bk = sh.wk[buf][0];
    bx = sh.wx[buf][0];
#pragma unroll
    for (int q = 1; q < kTkWaves; ++q) {
      const uint64_t ok = sh.wk[buf][q];
      const int ox = sh.wx[buf][q];
      const bool b = kbetter(ok, ox, bk, bx);
      bk = b ? ok : bk;
      bx = b ? ox : bx;
    }
    pk = bk;
    px = bx;
    if (t == 0) {
      sh.rk[r] = bk;
      sh.rx[r] = bx;
    }
  }
}


// Top-k with a candidate filter.  The rows are split into 64 groups (16
// lanes of a wave, all their rows); the topk-th largest group maximum theta
// is a lower bound of the topk-th largest value, since topk groups each hold
// a row at or above it.  Every row at or above theta - eps is a candidate:
// that set holds the top k and every row within eps of the k-th value, so
// when it has at most 64 rows one wave finishes the selection from it, tie
// rule included.  With more candidates, or a bank too large for registers,
// the rounds above give the ordered top k and the tie rule counts over all
// rows: when the rows within eps of the cut are exactly the picks at or below
// cut + eps the picks are the answer, otherwise further rounds take the
// lowest tied rows.
__global__ void __launch_bounds__(kTkThreads) topk_kernel(const double *__restrict__ sims, int64_t m,
                                                           int topk, int32_t *__restrict__ idx_out,
                                                           float *__restrict__ sim_out) {
  __shared__ TkShared sh;
  const double *sv = sims + (int64_t)blockIdx.x * m;
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  const bool in_regs = m <= (int64_t)kTkThreads * kTkRegs;
  int32_t *io = idx_out + (int64_t)blockIdx.x * topk;
  float *so = sim_out + (int64_t)blockIdx.x * topk;
  double vals[kTkRegs];
  if (in_regs) {
#pragma unroll
    for (int u = 0; u < kTkRegs; ++u) {
      const int64_t x = t + (int64_t)kTkThreads * u;
      vals[u] = x < m ? sv[x] : 0.0;
    }
  }
  if (in_regs) {
    uint64_t g = 0;
#pragma unroll
    for (int u = 0; u < kTkRegs; ++u) {
      const int64_t x = t + (int64_t)kTkThreads * u;
      const uint64_t k = okey(vals[u]);
      g = (x < m && k > g) ? k : g;
    }
    // maximum over the 16 lanes of a row (lane ^ 1, lane ^ 2, half-row and
    // row mirrors: every lane ends with the row's value)
    {
      uint64_t o = dpp64<0xB1, 0xF>(g);
      g = o > g ? o : g;
      o = dpp64<0x4E, 0xF>(g);
      g = o > g ? o : g;
      o = dpp64<0x141, 0xF>(g);
      g = o > g ? o : g;
      o = dpp64<0x140, 0xF>(g);
      g = o > g ? o : g;
    }
    if ((lane & 15) == 0) sh.gmax[w * 4 + (lane >> 4)] = g;
    if (t == 0) sh.ncand = 0;
    __syncthreads();
    if (w == 0) {
      const uint64_t mine = sh.gmax[lane];
      int greater = 0, geq = 0;
      for (int j = 0; j < 64; ++j) {
        const uint64_t gj = sh.gmax[j];
        greater += gj > mine ? 1 : 0;
        geq += gj >= mine ? 1 : 0;
      }
      const unsigned long long hit = __ballot(greater < topk && topk <= geq);
      if (lane == __ffsll((long long)hit) - 1) sh.theta = mine;
    }
    __syncthreads();
    // (theta = 0 when it comes from a group without rows: every row qualifies)
    const uint64_t th = sh.theta;
    const double low = th == 0 ? -INFINITY : okey_value(th) - kTieEps;
#pragma unroll
    for (int u = 0; u < kTkRegs; ++u) {
      const int64_t x = t + (int64_t)kTkThreads * u;
      const bool c = x < m && vals[u] >= low;
      const unsigned long long bits = __ballot(c);
      if (bits) {
        int base = 0;
        if (lane == 0) base = atomicAdd(&sh.ncand, __popcll(bits));
        base = __shfl(base, 0);
        const int pos = base + __popcll(bits & ((1ull << lane) - 1ull));
        if (c && pos < 64) {
          sh.ck[pos] = okey(vals[u]);
          sh.cx[pos] = (int)x;
        }
      }
    }
    __syncthreads();
    const int nc = sh.ncand;
    if (nc <= 64) {
      if (w != 0) return;
      // one wave: lane l < nc holds candidate l
      const bool on = lane < nc;
      uint64_t k = 0;
      int x = 0x7fffffff;
      if (on) {
        k = sh.ck[lane];
        x = sh.cx[lane];
      }
      int rank = 0;
      for (int j = 0; j < nc; ++j) rank += kbetter(sh.ck[j], sh.cx[j], k, x) ? 1 : 0;
      const double v = okey_value(k);
      const unsigned long long at_cut = __ballot(on && rank == topk - 1);
      const double cut = __shfl(v, __ffsll((long long)at_cut) - 1);
      const bool above = on && v > cut + kTieEps;
      const bool tie = on && fabs(v - cut) <= kTieEps;
      const int need = topk - __popcll(__ballot(above));
      // a tied row's place among the tied rows by row index
      const unsigned long long tied = __ballot(tie);
      int trank = 0;
      for (unsigned long long b = tied; b; b &= b - 1ull) trank += sh.cx[__ffsll((long long)b) - 1] < x ? 1 : 0;
      const bool pick = above || (tie && trank < need);
      // output slot: picks in descending value, lower row first
      const unsigned long long picks = __ballot(pick);
      int slot = 0;
      for (unsigned long long b = picks; b; b &= b - 1ull) {
        const int j = __ffsll((long long)b) - 1;
        slot += kbetter(sh.ck[j], sh.cx[j], k, x) ? 1 : 0;
      }
      if (pick) {
        io[slot] = x;
        so[slot] = (float)v;
      }
      return;
    }
  }
  tk_rounds<0>(vals, in_regs, sv, m, topk, 0.0, sh, 0);
  __syncthreads();
  const double cut = okey_value(sh.rk[topk - 1]);
  int nplus = 0;
  for (int r = 0; r < topk; ++r) nplus += okey_value(sh.rk[r]) > cut + kTieEps ? 1 : 0;
  const int need = topk - nplus;
  int mine = 0;
  if (in_regs) {
#pragma unroll
    for (int u = 0; u < kTkRegs; ++u) {
      const int64_t x = t + (int64_t)kTkThreads * u;
      mine += __popcll(__ballot(x < m && fabs(vals[u] - cut) <= kTieEps));
    }
  } else {
    for (int64_t x0 = 0; x0 < m; x0 += kTkThreads) {
      const int64_t x = x0 + t;
      mine += __popcll(__ballot(x < m && fabs(sv[x < m ? x : 0] - cut) <= kTieEps));
    }
  }
  if (lane == 0) sh.cnt[w] = mine;
  __syncthreads();
  int tied = 0;
#pragma unroll
  for (int q = 0; q < kTkWaves; ++q) tied += sh.cnt[q];
  if (tied == need) {
    if (t < topk) {
      io[t] = sh.rx[t];
      so[t] = (float)okey_value(sh.rk[t]);
    }
    return;
  }
  if (t < nplus) {
    sh.tv[t] = okey_value(sh.rk[t]);
    sh.tx[t] = sh.rx[t];
  }
  __syncthreads();
  if (t < nplus) {
    io[t] = sh.tx[t];
    so[t] = (float)sh.tv[t];
  }
  tk_rounds<1>(vals, in_regs, sv, m, need, cut, sh, topk);
  __syncthreads();
  if (w == 0) {
    double v = 0.0;
    int x = 0;
    if (lane < need) {
      x = sh.rx[lane];
      v = sv[x];
    }
    int rank = 0;
    for (int j = 0; j < need; ++j) {
      const int xj = sh.rx[j];
      const double vj = sv[xj];
      rank += (lane < need && better(vj, xj, v, x)) ? 1 : 0;
    }
    if (lane < need) {
      io[nplus + rank] = x;
      so[nplus + rank] = (float)v;
    }
  }
}

// Scan with the queries staged in LDS once per workgroup (16 waves, one bank
// row per wave per pass).  The row's loads are issued before the staging so
// both are in flight together; |q|^2 is computed once per workgroup (wave q
// for query q) instead of by every wave.  Column indices past the row end are
// clamped and their bank values zeroed, so the loads need no branches.
template <int KU, int NQ>
__global__ void __launch_bounds__(1024) scan_staged_kernel(const float *__restrict__ query, int64_t q0,
                                                     const float *__restrict__ bank, int64_t m,
                                                     int64_t dim, int64_t ld,
                                                     double *__restrict__ sims,
                                                     float *__restrict__ all_sim) {
  extern __shared__ float4 qs[];
  __shared__ double qn[NQ];
  const int t = threadIdx.x, lane = t & 63;
  const int w = __builtin_amdgcn_readfirstlane(t >> 6);
  const int d4 = (int)(dim / 4);
  const int64_t per_pass = (int64_t)gridDim.x * 16;
  const int npass = (int)((m + per_pass - 1) / per_pass);
  const float4 *qg = reinterpret_cast<const float4 *>(query + q0 * dim);
  for (int p = 0; p < npass; ++p) {
    const int64_t r = p * per_pass + (int64_t)blockIdx.x * 16 + w;
    const int64_t row = r < m ? r : m - 1;
    const float4 *bp = reinterpret_cast<const float4 *>(bank + row * ld);
    double bb = 0.0;
    double dot[NQ];
#pragma unroll
    for (int qq = 0; qq < NQ; ++qq) dot[qq] = 0.0;
    for (int cb = 0; cb < d4; cb += 64 * KU) {
      float4 x[KU];
#pragma unroll
      for (int u = 0; u < KU; ++u) {
        const int c = cb + lane + 64 * u;
        x[u] = bp[c < d4 ? c : d4 - 1];
      }
      if (p == 0 && cb == 0) {
        for (int i = t; i < NQ * d4; i += 1024) qs[i] = qg[i];
        __syncthreads();
        if (w < NQ) {
          double n2 = 0.0;
          for (int c = lane; c < d4; c += 64) {
            const float4 y = qs[w * d4 + c];
            n2 = fma((double)y.x, (double)y.x, n2);
            n2 = fma((double)y.y, (double)y.y, n2);
            n2 = fma((double)y.z, (double)y.z, n2);
            n2 = fma((double)y.w, (double)y.w, n2);
          }
          n2 = wave_sum(n2);
          if (lane == 0) qn[w] = n2;
        }
      }
#pragma unroll
      for (int u = 0; u < KU; ++u) {
        const int c = cb + lane + 64 * u;
        const bool in = c < d4;
        const int cc = in ? c : d4 - 1;
        const double x0 = in ? x[u].x : 0.f, x1 = in ? x[u].y : 0.f;
        const double x2 = in ? x[u].z : 0.f, x3 = in ? x[u].w : 0.f;
        bb = fma(x0, x0, bb);
        bb = fma(x1, x1, bb);
        bb = fma(x2, x2, bb);
        bb = fma(x3, x3, bb);
#pragma unroll
        for (int qq = 0; qq < NQ; ++qq) {
          const float4 y = qs[qq * d4 + cc];
          double d = dot[qq];
          d = fma(x0, (double)y.x, d);
          d = fma(x1, (double)y.y, d);
          d = fma(x2, (double)y.z, d);
          d = fma(x3, (double)y.w, d);
          dot[qq] = d;
        }
      }
    }
    if (p == 0) __syncthreads();
    const double bn = sqrt(wave_sum(bb));
#pragma unroll
    for (int qq = 0; qq < NQ; ++qq) {
      const double d = wave_sum(dot[qq]);
      const double den = sqrt(qn[qq]) * bn;
      const double sv = den > 0.0 ? d / den : 0.0;
      if (lane == qq && r < m) {
        sims[(q0 + qq) * m + r] = sv;
        if (all_sim) all_sim[(q0 + qq) * m + r] = (float)sv;
      }
    }
  }
}

// LDS budget for the staged queries of one pass.
constexpr int64_t kStageBytes = 144 * 1024;

template <int NQ>
hipError_t launch_staged(const float *query, int64_t q0, const float *bank, int64_t m, int64_t dim,
                         int64_t ld, double *sims, float *all_sim, hipStream_t s) {
  const size_t lds = (size_t)(NQ * dim * 4);
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(&scan_staged_kernel<4, NQ>),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  const int64_t blocks = (m + 15) / 16;
  const unsigned grid = (unsigned)(blocks < 2048 ? blocks : 2048);
  hipLaunchKernelGGL((scan_staged_kernel<4, NQ>), dim3(grid), dim3(1024), lds, s,
                     query, q0, bank, m, dim, ld, sims, all_sim);
  return hipGetLastError();
}

}  // namespace

hipError_t sig_static_scratch(void **ptr) {
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static void *addr[kMaxDevices] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void *p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    addr[dev] = p;
  }
  *ptr = addr[dev];
  return hipSuccess;
}

hipError_t launch_sig(const float *query, int64_t nq, const float *bank, int64_t m, int64_t dim,
                      int64_t ld, int topk, int32_t *idx, float *sim, float *all_sim,
                      double *sims, hipStream_t s) {
  const int64_t per_query = dim * 4;
  int64_t fit = kStageBytes / per_query;
  if (fit > kQChunk) fit = kQChunk;
  for (int64_t q0 = 0; q0 < nq; q0 += (fit > 0 ? fit : kQChunk)) {
    hipError_t e = hipSuccess;
    if (fit > 0) {
      const int nqc = (int)((nq - q0) < fit ? (nq - q0) : fit);
      switch (nqc) {
        case 1: e = launch_staged<1>(query, q0, bank, m, dim, ld, sims, all_sim, s); break;
        case 2: e = launch_staged<2>(query, q0, bank, m, dim, ld, sims, all_sim, s); break;
        case 3: e = launch_staged<3>(query, q0, bank, m, dim, ld, sims, all_sim, s); break;
        default: e = launch_staged<4>(query, q0, bank, m, dim, ld, sims, all_sim, s); break;
      }
    } else {
      // a query row too long for LDS: read the queries from global memory
      const int nqc = (int)((nq - q0) < kQChunk ? (nq - q0) : kQChunk);
      const int64_t blocks = (m + 3) / 4;
      const unsigned grid = (unsigned)(blocks < 8192 ? blocks : 8192);
      hipLaunchKernelGGL(scan_kernel, dim3(grid), dim3(256), 0, s, query, q0, nqc, bank, m, dim, ld,
                         sims, all_sim);
      e = hipGetLastError();
    }
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(topk_kernel, dim3((unsigned)nq), dim3(kTkThreads), 0, s, sims, m, topk, idx, sim);
  return hipGetLastError();
}

}  // namespace carnator
