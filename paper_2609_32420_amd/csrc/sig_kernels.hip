// Early-signature cosine scoring against a bank of cached signatures
// (Sec. 3.1: the target is compared against a bank built from completed
// requests; Sec. 4.1, candidate recall: rank by similarity, keep the top K).
//
// One pass over the bank: one wave per bank row, 16-byte loads, fp64
// accumulation of <q, b> and |b|^2, a fixed-order wave reduction (so the
// result does not depend on scheduling), then a per-query top-k with the
// lower-row rule for near ties.
#include "internal.h"

#include <math.h>

namespace carnator {
namespace {

constexpr double kTieEps = 1e-6;
constexpr int kQChunk = 4;  // queries scored per pass over the bank

__device__ inline double wave_sum(double x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o);
  return x;
}

// One wave per bank row (grid-stride).  Scores queries [q0, q0 + nqc).  The
// wave streams the bank row and the query rows U float4 at a time per lane,
// so the loads of a row are in flight together.  |q|^2 is accumulated in the
// same pass (every wave computes it in the same order, so every wave gets the
// same value) and no separate norm pass is needed.
constexpr int kU = 4;
__global__ void __launch_bounds__(256) scan_kernel(const float *__restrict__ query, int64_t q0,
                                                   int nqc, const float *__restrict__ bank,
                                                   int64_t m, int64_t dim, int64_t ld,
                                                   double *__restrict__ sims,
                                                   float *__restrict__ all_sim) {
  const int lane = threadIdx.x & 63;
  const int64_t nwaves = (int64_t)gridDim.x * 4;
  const int64_t d4 = dim / 4;
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
          const float4 *qp = reinterpret_cast<const float4 *>(query + (q0 + qq) * dim);
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

// One workgroup per query: k rounds of block-wide argmax (each round takes
// the best element after the previous pick in that order), then the tie rule.
// The query's similarities are first copied to LDS when they fit
// (m <= kTopkLds), so the rounds read LDS instead of re-reading memory.
constexpr int kTopkLds = 8192;
__global__ void __launch_bounds__(1024) topk_kernel(const double *__restrict__ sims, int64_t m,
                                                    int topk, int32_t *__restrict__ idx_out,
                                                    float *__restrict__ sim_out) {
  extern __shared__ double vals[];  // [min(m, kTopkLds)]
  __shared__ double topv[64];
  __shared__ int topi[64];
  __shared__ double wv[16];
  __shared__ int wi[16];
  __shared__ int tsel[64];
  constexpr int NT = 1024;
  const double *gsv = sims + (int64_t)blockIdx.x * m;
  const bool in_lds = m <= kTopkLds;
  if (in_lds) {
    for (int64_t x = threadIdx.x; x < m; x += NT) vals[x] = gsv[x];
    __syncthreads();
  }
  const double *sv = in_lds ? vals : gsv;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  double pv = INFINITY;
  int pi = -1;
  for (int r = 0; r < topk; ++r) {
    double bv = -INFINITY;
    int bi = 0x7fffffff;
    for (int64_t x = threadIdx.x; x < m; x += NT) {
      const double v = sv[x];
      const int i = (int)x;
      const bool after = v < pv || (v == pv && i > pi);
      if (after && better(v, i, bv, bi)) {
        bv = v;
        bi = i;
      }
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      const double ov = __shfl_xor(bv, o);
      const int oi = __shfl_xor(bi, o);
      if (better(ov, oi, bv, bi)) {
        bv = ov;
        bi = oi;
      }
    }
    if (lane == 0) {
      wv[w] = bv;
      wi[w] = bi;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
      double cv = wv[0];
      int ci = wi[0];
      for (int q = 1; q < NT / 64; ++q)
        if (better(wv[q], wi[q], cv, ci)) {
          cv = wv[q];
          ci = wi[q];
        }
      topv[r] = cv;
      topi[r] = ci;
    }
    __syncthreads();
    pv = topv[r];
    pi = topi[r];
  }
  // tie rule: keep everything above cut + eps, fill the rest with the lowest
  // rows within eps of the cut
  const double cut = topv[topk - 1];
  int nplus = 0;
  for (int r = 0; r < topk; ++r) nplus += topv[r] > cut + kTieEps ? 1 : 0;
  const int need = topk - nplus;
  if (w == 0) {
    int got = 0;
    for (int64_t base = 0; base < m && got < need; base += 64) {
      const int64_t x = base + lane;
      const bool tie = x < m && fabs(sv[x] - cut) <= kTieEps;
      const unsigned long long bits = __ballot(tie);
      const int rank = got + __popcll(bits & ((1ull << lane) - 1ull));
      if (tie && rank < need) tsel[rank] = (int)x;
      got += __popcll(bits);
    }
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    // order the chosen tied rows by descending value, lower row first
    for (int a = 1; a < need; ++a) {
      const int ia = tsel[a];
      int b = a - 1;
      while (b >= 0 && better(sv[ia], ia, sv[tsel[b]], tsel[b])) {
        tsel[b + 1] = tsel[b];
        --b;
      }
      tsel[b + 1] = ia;
    }
    int32_t *io = idx_out + (int64_t)blockIdx.x * topk;
    float *so = sim_out + (int64_t)blockIdx.x * topk;
    for (int r = 0; r < nplus; ++r) {
      io[r] = topi[r];
      so[r] = (float)topv[r];
    }
    for (int r = 0; r < need; ++r) {
      io[nplus + r] = tsel[r];
      so[nplus + r] = (float)sv[tsel[r]];
    }
  }
}

}  // namespace

hipError_t launch_sig(const float *query, int64_t nq, const float *bank, int64_t m, int64_t dim,
                      int64_t ld, int topk, int32_t *idx, float *sim, float *all_sim,
                      double *sims, hipStream_t s) {
  const int64_t waves = (m + 3) / 4;
  const unsigned grid = (unsigned)(waves < 8192 ? waves : 8192);
  for (int64_t q0 = 0; q0 < nq; q0 += kQChunk) {
    const int nqc = (int)((nq - q0) < kQChunk ? (nq - q0) : kQChunk);
    hipLaunchKernelGGL(scan_kernel, dim3(grid), dim3(256), 0, s, query, q0, nqc, bank, m, dim, ld,
                       sims, all_sim);
  }
  const size_t lds = (size_t)(m <= kTopkLds ? m : 0) * sizeof(double);
  hipLaunchKernelGGL(topk_kernel, dim3((unsigned)nq), dim3(1024), lds, s, sims, m, topk, idx, sim);
  return hipGetLastError();
}

}  // namespace carnator
