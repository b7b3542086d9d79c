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

// ---- selection --------------------------------------------------------------
//
// Sort keys: an order-preserving map of the fp64 logit onto uint64 whose low
// 11 bits are replaced by (2047 - block index).  Sorting the keys in
// descending order is sorting by logit with the lower index first among
// logits equal in their top 53 bits; logits closer than that (2^-42
// relative) lie deep inside the 1e-6 tie band, where the final choice is made
// by block index anyway.  The exact logit of each sorted entry is read back
// by its index.
__device__ inline uint64_t sel_key(double s, int j) {
  const uint64_t b = (uint64_t)__double_as_longlong(s);
  const uint64_t m = (b >> 63) ? ~b : (b | 0x8000000000000000ull);
  return (m & ~0x7ffull) | (uint64_t)(2047 - j);
}
__device__ inline int sel_index(uint64_t k) { return 2047 - (int)(k & 0x7ff); }

// Lane exchange with lane ^ o (o a power of two below 64) without LDS
// round trips: DPP quad permutes for 1 and 2, ds_swizzle for 4 and 8,
// v_permlane16/32_swap for 16 and 32.
template <int O>
__device__ inline uint32_t xchg32(uint32_t x, int lane) {
  if constexpr (O == 1) return __builtin_amdgcn_update_dpp(0u, x, 0xB1, 0xF, 0xF, false);
  else if constexpr (O == 2) return __builtin_amdgcn_update_dpp(0u, x, 0x4E, 0xF, 0xF, false);
  else if constexpr (O == 4 || O == 8) return __builtin_amdgcn_ds_swizzle(x, (O << 10) | 0x1f);
  else if constexpr (O == 16) {
    const auto r = __builtin_amdgcn_permlane16_swap(x, x, false, false);
    return (lane & 16) ? r[0] : r[1];
  } else {
    const auto r = __builtin_amdgcn_permlane32_swap(x, x, false, false);
    return (lane & 32) ? r[0] : r[1];
  }
}
template <int O>
__device__ inline uint64_t xchg64(uint64_t x, int lane) {
  const uint32_t lo = xchg32<O>((uint32_t)x, lane);
  const uint32_t hi = xchg32<O>((uint32_t)(x >> 32), lane);
  return ((uint64_t)hi << 32) | lo;
}

// One compare-exchange stage of a descending bitonic sort of P = 64 E keys
// held lane-major (lane L holds positions L E .. L E + E - 1).
template <int E, int ST>
__device__ inline void bitonic_stage(uint64_t (&k)[E], int lane, int size) {
  if constexpr (ST < E) {
#pragma unroll
    for (int u = 0; u < E; ++u) {
      if ((u & ST) == 0) {
        const int u2 = u | ST;
        const int p = lane * E + u;
        const bool desc = (p & size) == 0;  // this run sorts descending
        const uint64_t a = k[u], c = k[u2];
        const bool sw = desc ? (c > a) : (a > c);
        k[u] = sw ? c : a;
        k[u2] = sw ? a : c;
      }
    }
  } else {
    constexpr int LX = ST / E;
#pragma unroll
    for (int u = 0; u < E; ++u) {
      const int p = lane * E + u;
      const uint64_t o = xchg64<LX>(k[u], lane);
      const bool desc = (p & size) == 0;
      const bool lower = (p & ST) == 0;
      // the lower position of a pair keeps the larger key in a descending run
      const bool keep_big = lower == desc;
      const uint64_t a = k[u];
      k[u] = keep_big ? (a > o ? a : o) : (a < o ? a : o);
    }
  }
}
template <int E, int ST>
__device__ inline void bitonic_merge(uint64_t (&k)[E], int lane, int size) {
  bitonic_stage<E, ST>(k, lane, size);
  if constexpr (ST > 1) bitonic_merge<E, ST / 2>(k, lane, size);
}
template <int E, int SIZE>
__device__ inline void bitonic_sort(uint64_t (&k)[E], int lane) {
  if constexpr (SIZE > 2) bitonic_sort<E, SIZE / 2>(k, lane);
  bitonic_merge<E, SIZE / 2>(k, lane, SIZE);
}

__device__ inline double wave_sum(double x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o);
  return x;
}

// One workgroup of R waves per (bh, R consecutive query blocks).
//
// Phase 1, s_ij = sigma <qbar_i, kbar_j>: the R pooled query rows sit in LDS;
// a wave takes 16 key blocks at a time and forms the 16 x 16 tile of dot
// products on the fp64 matrix cores (16x16x4 steps over the channels, kbar^T
// read as 128-byte runs).  With R = 8 the upper half of the tile repeats row
// R - 1 and is not stored.  Phase 2 gives each wave one row.
template <int D, int E, int R>
__global__ void __launch_bounds__(64 * R) select_kernel(const double *__restrict__ qbar,
                                                        const double *__restrict__ kbarT, int nB,
                                                        double sigma, double tau,
                                                        uint8_t *__restrict__ mask) {
  extern __shared__ double sc[];  // [R][nB] logits, then [R][D] pooled queries
  const int bh = blockIdx.y;
  const int r0 = blockIdx.x * R;
  const int nr = min(R, nB - r0);
  const double *qb = qbar + ((int64_t)bh * nB + r0) * D;
  const double *kt = kbarT + (int64_t)bh * D * nB;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;

  double *qs = sc + R * nB;
  for (int x = threadIdx.x; x < R * D; x += 64 * R) {
    const int r = x / D;
    qs[x] = qb[min(r, nr - 1) * D + (x - r * D)];
  }
  __syncthreads();
  {
    // fp64 MFMA 16x16x4: wave w owns key blocks 16 w .. 16 w + 15 (then
    // + 16 R ...); lane l supplies qbar[row l % 16][4 c + l / 16] and
    // kbar[key l % 16][4 c + l / 16] and receives S[l / 16 + 4 v][l % 16].
    const int li = lane & 15, lk = lane >> 4;
    for (int j0 = wave * 16; j0 < nB; j0 += 16 * R) {
      const int jc = min(j0 + li, nB - 1);
      typedef double f64x4 __attribute__((ext_vector_type(4)));
      f64x4 acc = {0.0, 0.0, 0.0, 0.0};
      const double *kc = kt + (int64_t)lk * nB + jc;
      const double *qr = qs + min(li, R - 1) * D + lk;
#pragma unroll
      for (int c0 = 0; c0 < D / 4; c0 += 8) {
        double kv[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) kv[u] = kc[(int64_t)(4 * (c0 + u)) * nB];
#pragma unroll
        for (int u = 0; u < 8; ++u) acc = __builtin_amdgcn_mfma_f64_16x16x4f64(qr[4 * (c0 + u)], kv[u], acc, 0, 0, 0);
      }
      const int j = j0 + li;
      if (j < nB) {
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int r = lk + 4 * v;
          if (r < nr) sc[r * nB + j] = sigma * acc[v];
        }
      }
    }
  }
  __syncthreads();

  // ---- phase 2: selection, one row per wave
  for (int r = wave; r < nr; r += R) {
    const double *row = sc + r * nB;
    uint8_t *out = mask + ((int64_t)bh * nB + r0 + r) * nB;
    uint64_t key[E];
#pragma unroll
    for (int u = 0; u < E; ++u) {
      const int p = lane * E + u;
      key[u] = p < nB ? sel_key(row[p], p) : 0ull;  // 0 sorts last
    }
    bitonic_sort<E, 64 * E>(key, lane);
    double s[E];
#pragma unroll
    for (int u = 0; u < E; ++u) s[u] = lane * E + u < nB ? row[sel_index(key[u])] : -INFINITY;

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
#define CARNATOR_SEL(EE)                                                                          \
  do {                                                                                            \
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(&select_kernel<D, EE, R>),  \
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);     \
    if (e != hipSuccess) return e;                                                                \
    hipLaunchKernelGGL((select_kernel<D, EE, R>), grid, dim3(64 * R), lds, s, qbar, kbarT, nB,    \
                       sigma, tau, mask);                                                         \
  } while (0)
  switch (P / 64) {
    case 1: CARNATOR_SEL(1); break;
    case 2: CARNATOR_SEL(2); break;
    case 4: CARNATOR_SEL(4); break;
    case 8: CARNATOR_SEL(8); break;
    case 16: CARNATOR_SEL(16); break;
    case 32:
      if constexpr (R <= 8) CARNATOR_SEL(32);
      else return hipErrorInvalidValue;
      break;
    default: return hipErrorInvalidValue;
  }
#undef CARNATOR_SEL
  return hipGetLastError();
}

// R query blocks per workgroup (one wave each): their logits and pooled rows
// take 8 R (nB + d) bytes of LDS, which stays within 160 KiB with R = 16 up
// to nB = 1024 and with R = 8 up to nB = 2048.
template <int D>
static hipError_t launch_select_d(const double *qbar, const double *kbarT, int BH, int nB,
                                  double sigma, double tau, uint8_t *mask, hipStream_t s) {
  if (nB <= 1024) return launch_select_dr<D, 16>(qbar, kbarT, BH, nB, sigma, tau, mask, s);
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
