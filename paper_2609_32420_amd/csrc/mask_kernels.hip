// Historical block-connectivity mask (Appendix C.3): block pooling of the
// historical Q/K, pooled logits, softmax over key blocks and the smallest
// prefix of key blocks (descending logit) whose mass reaches the threshold,
// with logits within 1e-6 of the cut handed to the lower block indices.
// Everything here runs in fp64.
#include "internal.h"

#include <math.h>

namespace carnator {
namespace {

constexpr double kTieEps = 1e-6;

__device__ inline double bf16_to_f64(uint32_t bits16) {
  return (double)__uint_as_float(bits16 << 16);
}

// One workgroup per (tensor, bh, block).  Thread t owns 8 consecutive
// channels (one 16-byte chunk) of every G-th token of the block.  The G
// partial sums are combined in a fixed order (first across the lanes of a
// wave that share a chunk, then across waves), so the result does not depend
// on timing.
template <int D>
__global__ void __launch_bounds__(256) pool_kernel(View q, View k, int H, int N, int bs, int nB,
                                                   double *__restrict__ qbar,
                                                   double *__restrict__ kbarT) {
  constexpr int CPR = D / 8;         // 16-byte chunks per token
  constexpr int G = 256 / CPR;       // token groups
  __shared__ double part[4][D];      // one partial per wave
  const int blk = blockIdx.x;
  const int bh = blockIdx.y;
  const int which = blockIdx.z;  // 0: Q_hist, 1: K_hist
  const View v = which ? k : q;
  const int b = bh / H, h = bh - b * H;
  const int t0 = blk * bs;
  const int n = min(bs, N - t0);
  const int c = threadIdx.x % CPR;
  const int g = threadIdx.x / CPR;
  const uint16_t *base = v.data + (int64_t)b * v.sb + (int64_t)h * v.sh + (int64_t)t0 * v.sn + c * 8;
  double acc[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) acc[e] = 0.0;
  // All of this thread's tokens (at most RPT) are loaded before any is added,
  // so a wave keeps RPT 16-byte loads in flight instead of one.
  constexpr int RPT = 128 / G;
  uint4 w[RPT];
#pragma unroll
  for (int u = 0; u < RPT; ++u) {
    const int r = g + u * G;
    w[u] = r < n ? *reinterpret_cast<const uint4 *>(base + (int64_t)r * v.sn) : make_uint4(0, 0, 0, 0);
  }
#pragma unroll
  for (int u = 0; u < RPT; ++u) {
    const uint32_t ww[4] = {w[u].x, w[u].y, w[u].z, w[u].w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      acc[2 * e] += bf16_to_f64(ww[e] & 0xffffu);
      acc[2 * e + 1] += bf16_to_f64(ww[e] >> 16);
    }
  }
  // lanes l, l + CPR, l + 2 CPR, ... of a wave hold the same channels
#pragma unroll
  for (int o = CPR; o < 64; o <<= 1)
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] += __shfl_xor(acc[e], o);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane < CPR) {
#pragma unroll
    for (int e = 0; e < 8; ++e) part[wave][c * 8 + e] = acc[e];
  }
  __syncthreads();
  for (int ch = threadIdx.x; ch < D; ch += 256) {
    const double s = ((part[0][ch] + part[1][ch]) + part[2][ch]) + part[3][ch];
    const double mean = s / (double)n;
    if (which == 0)
      qbar[((int64_t)bh * nB + blk) * D + ch] = mean;
    else
      kbarT[((int64_t)bh * D + ch) * nB + blk] = mean;
  }
}

// Descending logit, lower block index first on equality.
__device__ inline bool before(double sa, int ja, double sb, int jb) {
  return sa > sb || (sa == sb && ja < jb);
}

// One in-register compare-exchange stage (pair distance ST < E elements).
template <int E, int ST>
__device__ inline void bitonic_inreg(double (&s)[E], int (&j)[E], int lane, int size) {
#pragma unroll
  for (int u = 0; u < E; ++u) {
    if ((u & ST) == 0) {
      const int u2 = u | ST;
      const int p = lane * E + u;
      const bool dir = (p & size) == 0;
      const bool sw = dir ? before(s[u2], j[u2], s[u], j[u]) : before(s[u], j[u], s[u2], j[u2]);
      if (sw) {
        const double ts = s[u];
        s[u] = s[u2];
        s[u2] = ts;
        const int tj = j[u];
        j[u] = j[u2];
        j[u2] = tj;
      }
    }
  }
}

// Wave-level bitonic sort of P = 64*E (score, index) pairs held lane-major:
// lane L holds sorted positions L*E .. L*E+E-1.  Pairs closer than E
// positions are exchanged inside a lane, farther pairs across lanes.
template <int E>
__device__ inline void wave_bitonic(double (&s)[E], int (&j)[E], int lane) {
  constexpr int P = 64 * E;
#pragma unroll 1
  for (int size = 2; size <= P; size <<= 1) {
#pragma unroll 1
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      if (stride < E) {
        if constexpr (E > 1) if (stride == 1) bitonic_inreg<E, 1>(s, j, lane, size);
        if constexpr (E > 2) if (stride == 2) bitonic_inreg<E, 2>(s, j, lane, size);
        if constexpr (E > 4) if (stride == 4) bitonic_inreg<E, 4>(s, j, lane, size);
        if constexpr (E > 8) if (stride == 8) bitonic_inreg<E, 8>(s, j, lane, size);
        if constexpr (E > 16) if (stride == 16) bitonic_inreg<E, 16>(s, j, lane, size);
      } else {
        const int lx = stride / E;
#pragma unroll
        for (int u = 0; u < E; ++u) {
          const int p = lane * E + u;
          const double os = __shfl_xor(s[u], lx);
          const int oj = __shfl_xor(j[u], lx);
          const bool dir = (p & size) == 0;
          const bool lower = (p & stride) == 0;
          const bool mine_first = before(s[u], j[u], os, oj);
          const bool want_first = (lower == dir);
          if (mine_first != want_first) {
            s[u] = os;
            j[u] = oj;
          }
        }
      }
    }
  }
}

__device__ inline double wave_sum(double x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o);
  return x;
}

// One workgroup of 8 waves per (bh, R = 8 consecutive query blocks).
// Phase 1 computes the R x nB pooled logits into LDS; phase 2 gives each wave
// one row to select.
constexpr int kSelThreads = 512;
template <int D, int E, int R>
__global__ void __launch_bounds__(kSelThreads) select_kernel(const double *__restrict__ qbar,
                                                             const double *__restrict__ kbarT, int nB,
                                                             double sigma, double tau,
                                                             uint8_t *__restrict__ mask) {
  static_assert(R == 8, "one row per wave");
  extern __shared__ double sc[];  // [R][nB] logits, then [R][D] pooled queries
  const int bh = blockIdx.y;
  const int r0 = blockIdx.x * R;
  const int nr = min(R, nB - r0);
  const double *qb = qbar + ((int64_t)bh * nB + r0) * D;
  const double *kt = kbarT + (int64_t)bh * D * nB;

  // ---- phase 1: s_ij = sigma * <qbar_i, kbar_j>.  The R pooled query rows
  // sit in LDS; thread t owns rows 4 (t / 256) .. +4 of key blocks
  // t % 256 + 256 u, and streams kbar^T[c][j] (coalesced across lanes) 16
  // channels at a time so the loads overlap.
  double *qs = sc + R * nB;
  for (int x = threadIdx.x; x < R * D; x += kSelThreads) {
    const int r = x / D;
    qs[x] = qb[min(r, nr - 1) * D + (x - r * D)];
  }
  __syncthreads();
  const int rg = (threadIdx.x >> 8) * 4;
  for (int jj = threadIdx.x & 255; jj < nB; jj += 256) {
    double acc[4] = {0.0, 0.0, 0.0, 0.0};
    for (int c0 = 0; c0 < D; c0 += 16) {
      double kv[16];
#pragma unroll
      for (int u = 0; u < 16; ++u) kv[u] = kt[(int64_t)(c0 + u) * nB + jj];
#pragma unroll
      for (int u = 0; u < 16; u += 2)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const double2 qv = *reinterpret_cast<const double2 *>(qs + (rg + r) * D + c0 + u);
          acc[r] = fma(qv.x, kv[u], acc[r]);
          acc[r] = fma(qv.y, kv[u + 1], acc[r]);
        }
    }
#pragma unroll
    for (int r = 0; r < 4; ++r)
      if (rg + r < nr) sc[(rg + r) * nB + jj] = sigma * acc[r];
  }
  __syncthreads();

  // ---- phase 2: selection, one row per wave
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  for (int r = wave; r < nr; r += kSelThreads / 64) {
    const double *row = sc + r * nB;
    uint8_t *out = mask + ((int64_t)bh * nB + r0 + r) * nB;
    double s[E];
    int j[E];
#pragma unroll
    for (int u = 0; u < E; ++u) {
      const int p = lane * E + u;
      j[u] = p;
      s[u] = p < nB ? row[p] : -INFINITY;
    }
    wave_bitonic<E>(s, j, lane);

    // softmax over the sorted row; positions >= nB carry -inf and weigh 0
    const double smax = __shfl(s[0], 0);
    double e[E];
    double lsum = 0.0;
#pragma unroll
    for (int u = 0; u < E; ++u) {
      e[u] = (lane * E + u < nB) ? exp(s[u] - smax) : 0.0;
      lsum += e[u];
    }
    const double Z = wave_sum(lsum);
    // inclusive prefix of p = e / Z in sorted order
    double pl[E];
    double run = 0.0;
#pragma unroll
    for (int u = 0; u < E; ++u) {
      pl[u] = e[u] / Z;
      run += pl[u];
    }
    double incl = run;  // inclusive scan of the lane totals
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const double y = __shfl_up(incl, o);
      if (lane >= o) incl += y;
    }
    double excl = __shfl_up(incl, 1);
    if (lane == 0) excl = 0.0;
    int first = E;
    double cum = excl;
#pragma unroll
    for (int u = 0; u < E; ++u) {
      cum += pl[u];
      if (first == E && lane * E + u < nB && cum >= tau) first = u;
    }
    const unsigned long long hit = __ballot(first < E);
    int k;
    if (hit) {
      const int hl = __ffsll((long long)hit) - 1;
      k = hl * E + __shfl(first, hl) + 1;
    } else {
      k = nB;
    }
    // cut score = sorted position k-1
    const int cl = (k - 1) / E, cu = (k - 1) % E;
    double mine = 0.0;
#pragma unroll
    for (int u = 0; u < E; ++u)
      if (u == cu) mine = s[u];
    const double cut = __shfl(mine, cl);
    const double hiT = cut + kTieEps;

    // |S+| : blocks strictly above the tie band
    int nplus = 0;
    for (int base = 0; base < nB; base += 64) {
      const int jj = base + lane;
      const bool above = jj < nB && row[jj] > hiT;
      nplus += __popcll(__ballot(above));
    }
    const int need = k - nplus;
    // write the row in index order; the first `need` tied blocks are kept
    int tied_before = 0;
    for (int base = 0; base < nB; base += 64) {
      const int jj = base + lane;
      double sv = jj < nB ? row[jj] : -INFINITY;
      const bool above = jj < nB && sv > hiT;
      const bool tie = jj < nB && fabs(sv - cut) <= kTieEps;
      const unsigned long long tb = __ballot(tie);
      const int rank = tied_before + __popcll(tb & ((1ull << lane) - 1ull));
      if (jj < nB) out[jj] = (above || (tie && rank < need)) ? 1 : 0;
      tied_before += __popcll(tb);
    }
  }
}

__global__ void fill_ones_kernel(uint8_t *p, size_t n) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 1;
}

}  // namespace

hipError_t launch_pool(View q, View k, int B, int H, int N, int d, int bs, double *qbar,
                       double *kbarT, hipStream_t s) {
  const int nB = (N + bs - 1) / bs;
  dim3 grid(nB, B * H, 2);
  if (d == 128)
    hipLaunchKernelGGL(pool_kernel<128>, grid, dim3(256), 0, s, q, k, H, N, bs, nB, qbar, kbarT);
  else
    hipLaunchKernelGGL(pool_kernel<64>, grid, dim3(256), 0, s, q, k, H, N, bs, nB, qbar, kbarT);
  return hipGetLastError();
}

template <int D, int R>
static hipError_t launch_select_dr(const double *qbar, const double *kbarT, int BH, int nB,
                                   double sigma, double tau, uint8_t *mask, hipStream_t s) {
  dim3 grid((nB + R - 1) / R, BH);
  const size_t lds = (size_t)R * (nB + D) * sizeof(double);
  const int P = nB <= 64 ? 64 : (1 << (32 - __builtin_clz((unsigned)(nB - 1))));
#define CARNATOR_LDS_ATTR(EE)                                                                     \
  do {                                                                                            \
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(&select_kernel<D, EE, R>),  \
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);     \
    if (e != hipSuccess) return e;                                                                \
  } while (0)
  switch (P / 64) {
    case 1: CARNATOR_LDS_ATTR(1); break;
    case 2: CARNATOR_LDS_ATTR(2); break;
    case 4: CARNATOR_LDS_ATTR(4); break;
    case 8: CARNATOR_LDS_ATTR(8); break;
    case 16: CARNATOR_LDS_ATTR(16); break;
    case 32: CARNATOR_LDS_ATTR(32); break;
    default: return hipErrorInvalidValue;
  }
#undef CARNATOR_LDS_ATTR
  switch (P / 64) {
    case 1: hipLaunchKernelGGL((select_kernel<D, 1, R>), grid, dim3(kSelThreads), lds, s, qbar, kbarT, nB, sigma, tau, mask); break;
    case 2: hipLaunchKernelGGL((select_kernel<D, 2, R>), grid, dim3(kSelThreads), lds, s, qbar, kbarT, nB, sigma, tau, mask); break;
    case 4: hipLaunchKernelGGL((select_kernel<D, 4, R>), grid, dim3(kSelThreads), lds, s, qbar, kbarT, nB, sigma, tau, mask); break;
    case 8: hipLaunchKernelGGL((select_kernel<D, 8, R>), grid, dim3(kSelThreads), lds, s, qbar, kbarT, nB, sigma, tau, mask); break;
    case 16: hipLaunchKernelGGL((select_kernel<D, 16, R>), grid, dim3(kSelThreads), lds, s, qbar, kbarT, nB, sigma, tau, mask); break;
    case 32: hipLaunchKernelGGL((select_kernel<D, 32, R>), grid, dim3(kSelThreads), lds, s, qbar, kbarT, nB, sigma, tau, mask); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// 8 query blocks per workgroup: their logits and pooled rows take
// 64 * (nB + d) bytes of LDS (at most 139 KiB for nB = 2048, d = 128).
template <int D>
static hipError_t launch_select_d(const double *qbar, const double *kbarT, int BH, int nB,
                                  double sigma, double tau, uint8_t *mask, hipStream_t s) {
  return launch_select_dr<D, 8>(qbar, kbarT, BH, nB, sigma, tau, mask, s);
}

hipError_t launch_select(const double *qbar, const double *kbarT, int BH, int nB, int d,
                         double sigma, double tau, uint8_t *mask, hipStream_t s) {
  if (d == 128) return launch_select_d<128>(qbar, kbarT, BH, nB, sigma, tau, mask, s);
  return launch_select_d<64>(qbar, kbarT, BH, nB, sigma, tau, mask, s);
}

hipError_t launch_fill_ones(uint8_t *p, size_t n, hipStream_t s) {
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(fill_ones_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, p, n);
  return hipGetLastError();
}

}  // namespace carnator
