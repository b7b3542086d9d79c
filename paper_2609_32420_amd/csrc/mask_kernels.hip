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
                                                   double *__restrict__ kbar) {
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
    (which ? kbar : qbar)[((int64_t)bh * nB + blk) * D + ch] = mean;
  }
}

// ---- selection --------------------------------------------------------------
//
// Selection keys: an order-preserving map of the fp64 logit onto uint64 whose
// low 11 bits are replaced by (2047 - block index).  Descending key order is
// descending logit with the lower index first among logits equal in their
// top 53 bits; logits closer than that (2^-42 relative) lie deep inside the
// 1e-6 tie band, where the final choice is made by block index anyway.  The
// keys are unique; the selection finds the k-th largest by bisection and
// reads back the exact logit of its block.
__device__ inline uint64_t sel_key(double s, int j) {
  const uint64_t b = (uint64_t)__double_as_longlong(s);
  const uint64_t m = (b >> 63) ? ~b : (b | 0x8000000000000000ull);
  return (m & ~0x7ffull) | (uint64_t)(2047 - j);
}
__device__ inline int sel_index(uint64_t k) { return 2047 - (int)(k & 0x7ff); }
// The logit a selection key stands for, up to its low 11 bits (used only to pick
// bisection points).
__device__ inline double key_value(uint64_t k) {
  const uint64_t b = (k >> 63) ? (k & 0x7fffffffffffffffull) : ~k;
  return __longlong_as_double((long long)b);
}

// Bisection state of one row (the same in every lane): mass(key >= lo) >=
// tau Z > mass(key >= hi), cnt_* the numbers of keys >= lo and >= hi.
struct Bisect {
  uint64_t lo, hi;
  int cnt_lo, cnt_hi;
  double m_hi;  // mass of the keys >= hi
  bool trie;
  int it;
};

// Bisection steps over EE positions per lane until at most `until` keys lie
// in [lo, hi).  The keys counted are those of the positions plus c_off, the
// mass their weights plus m_off (the keys above the positions' range).
// Split at the midpoint of the values while that separates keys; once it
// does not (a run of equal logits), split at the highest bit in which the
// interval's smallest and largest keys differ, which leaves keys on both
// sides and resolves equal logits by their index bits.
template <int EE>
__device__ inline void bisect_steps(const uint64_t (&key)[EE], const double (&pl)[EE], int c_off,
                                    double m_off, double tauZ, int until, Bisect &b) {
  for (; b.it < 192 && b.cnt_lo - b.cnt_hi > until; ++b.it) {
    uint64_t K = 0;
    if (!b.trie) {
      const double lv = key_value(b.lo), hv = key_value(b.hi - 1);
      K = sel_key(uniform(lv + 0.5 * (hv - lv)), 2047);
      b.trie = !(K > b.lo && K < b.hi);
    }
    if (b.trie) {
      uint64_t a = ~0ull, z = 0ull;
#pragma unroll
      for (int u = 0; u < EE; ++u) {
        const bool in = key[u] >= b.lo && key[u] < b.hi;
        a = in && key[u] < a ? key[u] : a;
        z = in && key[u] > z ? key[u] : z;
      }
      a = wave_min_u64(a);
      z = wave_max_u64(z);
      // a < z: the interval holds at least two (distinct) keys
      K = z & ~((1ull << (63 - __clzll((long long)(a ^ z)))) - 1ull);
    }
    double m = 0.0;
    int c = c_off;
#pragma unroll
    for (int u = 0; u < EE; ++u) {
      const bool ge = key[u] >= K;
      m += ge ? pl[u] : 0.0;
      c += __popcll(__ballot(ge));
    }
    m = m_off + wave_sum(m);
    const int before = b.cnt_lo - b.cnt_hi;
    if (m >= tauZ) {
      b.lo = K;
      b.cnt_lo = c;
    } else {
      b.hi = K;
      b.cnt_hi = c;
      b.m_hi = m;
    }
    if (b.cnt_lo - b.cnt_hi == before) b.trie = true;
  }
}

// The k-th largest key once the bisection has ended: the one key in [lo, hi)
// (k = cnt_lo), or, if the step cap was hit, the largest key in [lo, hi) and
// the number of keys at or above it.
template <int EE>
__device__ inline uint64_t bisect_result(const uint64_t (&key)[EE], int c_off, const Bisect &b,
                                         int &k) {
  uint64_t kstar = 0ull;
  if (b.cnt_lo - b.cnt_hi == 1) {
#pragma unroll
    for (int u = 0; u < EE; ++u) {
      const unsigned long long hit = __ballot(key[u] >= b.lo && key[u] < b.hi);
      if (hit) kstar = read_lane(key[u], __ffsll((long long)hit) - 1);
    }
    k = b.cnt_lo;
  } else {
    uint64_t kl = 0ull;
#pragma unroll
    for (int u = 0; u < EE; ++u)
      if (key[u] >= b.lo && key[u] < b.hi && key[u] > kl) kl = key[u];
    kstar = wave_max_u64(kl);
    k = c_off;
#pragma unroll
    for (int u = 0; u < EE; ++u) k += __popcll(__ballot(key[u] >= kstar));
  }
  return kstar;
}

// One workgroup of W waves per (bh, R consecutive query blocks), W = R or
// R / 2 (then each wave selects two rows).
//
// Phase 1, s_ij = sigma <qbar_i, kbar_j>: the R pooled query rows sit in LDS;
// a wave takes 16 key blocks at a time and forms the 16 x 16 tile of dot
// products on the fp64 matrix cores (16x16x4 steps over the channels).  The
// contraction visits the channels in an order that suits the loads: in
// 16-channel group g, lane (i, k) = (lane & 15, lane >> 4) holds channels
// 16 g + 4 k .. 16 g + 4 k + 3 of key block i (one 32-byte piece of its kbar
// row) and feeds channel 16 g + 4 k + t to step t, and the query side takes
// its channels in the same order.  With R = 8 the upper half of the tile
// repeats row R - 1 and is not stored.  Phase 2: wave w selects rows w,
// w + W, ... of the workgroup (E = positions per lane, 64 E >= nB).
// MASS: the rows are given, as block masses [BH][nB][nB] at qbar (kbar and
// sigma unused): phase 1 copies the workgroup's rows into LDS and phase 2
// selects on the masses themselves instead of the softmax of logits.
template <int D, int E, int R, int W, bool MASS>
__global__ void __launch_bounds__(64 * W) select_kernel(const double *__restrict__ qbar,
                                                        const double *__restrict__ kbar, int nB,
                                                        double sigma, double tau,
                                                        uint8_t *__restrict__ mask,
                                                        uint64_t *__restrict__ bits, int BH) {
  // LDS: [R][nB] logits, then the R pooled query rows, QS doubles apart (a
  // 16-byte pad spreads the 16 rows read by one MFMA step over the banks),
  // at least W * 128 doubles
  constexpr int QS = D + 2;
  extern __shared__ double sc[];
  // Workgroups are dealt to the 8 XCDs in turn.  Logical workgroup
  // (L mod 8) ceil(G / 8) + L / 8 gives each XCD a contiguous run of
  // (head, row block) pairs, so an XCD's L2 fetches the kbar of about
  // BH / 8 heads instead of all of them.
  const int nbx = (nB + R - 1) / R;
  const int G = nbx * BH;
  const int per = (G + 7) / 8;
  const int T = (int)(blockIdx.x & 7) * per + (int)(blockIdx.x >> 3);
  if (T >= G) return;  // the whole workgroup, before any barrier
  const int bh = T / nbx;
  const int r0 = (T - bh * nbx) * R;
  const int nr = min(R, nB - r0);
  const double *qb = qbar + ((int64_t)bh * nB + r0) * D;
  const double *kb = kbar + (int64_t)bh * nB * D;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  // phase 2's candidate buffers (64 keys and weights per wave) reuse the
  // pooled-row area, which phase 1's last barrier frees
  uint64_t *cbuf = reinterpret_cast<uint64_t *>(sc + R * nB);

  if constexpr (MASS) {
    const double *src = qbar + ((int64_t)bh * nB + r0) * nB;
    for (int x = threadIdx.x; x < nr * nB; x += 64 * W) sc[x] = src[x];
    __syncthreads();
  } else {
    double *qs = sc + R * nB;
    {
      constexpr int SPT = R * D / (64 * W);  // staged values per thread (all loads in flight)
      double sv[SPT];
  #pragma unroll
      for (int i = 0; i < SPT; ++i) {
        const int x = threadIdx.x + i * 64 * W, r = x / D, c = x - r * D;
        sv[i] = qb[min(r, nr - 1) * D + c];
      }
  #pragma unroll
      for (int i = 0; i < SPT; ++i) {
        const int x = threadIdx.x + i * 64 * W, r = x / D, c = x - r * D;
        qs[r * QS + c] = sv[i];
      }
    }
    __syncthreads();
    {
      typedef double f64x4 __attribute__((ext_vector_type(4)));
      constexpr int NG = D / 16;  // 16-channel groups
      const int li = lane & 15, lk = lane >> 4;
      const double *qr = qs + min(li, R - 1) * QS + 4 * lk;
      // The groups start at a different place in every wave: walking them in
      // lockstep sends every wave of the chip to the same few L2 channels.
      const int rot = (wave * 5 + T * 3) & (NG - 1);
      for (int j0 = wave * 16; j0 < nB; j0 += 16 * W) {
        const double *kr = kb + (int64_t)min(j0 + li, nB - 1) * D + 4 * lk;
        f64x4 acc = {0.0, 0.0, 0.0, 0.0};
        // All of the tile's loads are issued before the first product: left to
        // itself the compiler keeps two in flight, and the tile then costs
        // D / 8 L2 round trips instead of one.
        double2 kv[NG][2];
  #pragma unroll
        for (int g = 0; g < NG; ++g) {
          const int gr = (g + rot) & (NG - 1);
          kv[g][0] = *reinterpret_cast<const double2 *>(kr + 16 * gr);
          kv[g][1] = *reinterpret_cast<const double2 *>(kr + 16 * gr + 2);
        }
        __builtin_amdgcn_sched_barrier(0);
  #pragma unroll
        for (int g = 0; g < NG; ++g) {
          const int gr = (g + rot) & (NG - 1);
          acc = __builtin_amdgcn_mfma_f64_16x16x4f64(qr[16 * gr + 0], kv[g][0].x, acc, 0, 0, 0);
          acc = __builtin_amdgcn_mfma_f64_16x16x4f64(qr[16 * gr + 1], kv[g][0].y, acc, 0, 0, 0);
          acc = __builtin_amdgcn_mfma_f64_16x16x4f64(qr[16 * gr + 2], kv[g][1].x, acc, 0, 0, 0);
          acc = __builtin_amdgcn_mfma_f64_16x16x4f64(qr[16 * gr + 3], kv[g][1].y, acc, 0, 0, 0);
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
  }

  // ---- phase 2: selection, one row per wave.  Lane l holds positions
  // u 64 + l.  The k-th largest selection key K* (k the shortest prefix whose
  // mass reaches tau) is found by bisection over the keys, keeping
  // mass(key >= lo) >= tau > mass(key >= hi) until [lo, hi) holds one key.
  // The bisection state is the same in every lane and lives in scalar
  // registers; the vector work per step is one compare and add per position
  // and one wave sum.
  for (int r = wave; r < nr; r += W) {
    const double *row = sc + r * nB;
    const int64_t grow = (int64_t)bh * nB + r0 + r;
    double pl[E];
    uint64_t key[E];
    double smax = -INFINITY, smin = INFINITY;
#pragma unroll
    for (int u = 0; u < E; ++u) {
      const int p = u * 64 + lane;
      const bool ok = p < nB;
      const double s = row[min(p, nB - 1)];
      pl[u] = ok ? s : -INFINITY;  // the logit until the softmax below
      key[u] = ok ? sel_key(s, p) : 0ull;  // valid keys are > 2047
      smax = fmax(smax, pl[u]);
      smin = ok ? fmin(smin, s) : smin;
    }
    smax = wave_max(smax);
    smin = wave_min(smin);
    // softmax weights exp(s - max): a set's mass p = weight / Z reaches tau
    // when its weight reaches tau Z (Z the sum of all weights)
    double lsum = 0.0;
#pragma unroll
    for (int u = 0; u < E; ++u) {
      if constexpr (MASS) pl[u] = (u * 64 + lane < nB) ? pl[u] : 0.0;
      else pl[u] = (u * 64 + lane < nB) ? exp(pl[u] - smax) : 0.0;
      lsum += pl[u];
    }
    const double tauZ = tau * wave_sum(lsum);

    // every key lies in [smallest key of value smin, largest key of smax]
    Bisect bs{sel_key(smin, 2047), sel_key(smax, 0) + 1, 0, 0, 0.0, false, 0};
    bool reach;
    {
      double m = 0.0;
      int c = 0;
#pragma unroll
      for (int u = 0; u < E; ++u) {
        const bool ge = key[u] >= bs.lo;
        m += ge ? pl[u] : 0.0;
        c += __popcll(__ballot(ge));
      }
      bs.cnt_lo = c;
      reach = wave_sum(m) >= tauZ;
    }
    int k;
    double cut;
    if (!reach) {
      k = bs.cnt_lo;  // the whole row falls short of tau: keep every block
      cut = smin;
    } else {
      uint64_t kstar;
      if constexpr (E == 1) {
        bisect_steps<1>(key, pl, 0, 0.0, tauZ, 1, bs);
        kstar = bisect_result<1>(key, 0, bs, k);
      } else {
        // all positions until at most 64 keys are left in [lo, hi); those
        // keys and weights then go one per lane (through this wave's LDS
        // area), and the remaining steps touch one position per lane
        bisect_steps<E>(key, pl, 0, 0.0, tauZ, 64, bs);
        if (bs.cnt_lo - bs.cnt_hi > 64) {
          kstar = bisect_result<E>(key, 0, bs, k);  // the step cap was hit
        } else {
          uint64_t *ck = cbuf + wave * 128;
          double *cw = reinterpret_cast<double *>(ck + 64);
          int base = 0;
#pragma unroll
          for (int u = 0; u < E; ++u) {
            const bool in = key[u] >= bs.lo && key[u] < bs.hi;
            const unsigned long long hit = __ballot(in);
            if (in) {
              const int x = base + __popcll(hit & ((1ull << lane) - 1ull));
              ck[x] = key[u];
              cw[x] = pl[u];
            }
            base += __popcll(hit);
          }
          __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
          __builtin_amdgcn_wave_barrier();
          __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
          // empty lanes hold key 0, below every valid key (> 2047)
          uint64_t k1[1] = {lane < base ? ck[lane] : 0ull};
          double p1[1] = {lane < base ? cw[lane] : 0.0};
          const int c_off = bs.cnt_hi;
          const double m_off = bs.m_hi;
          bisect_steps<1>(k1, p1, c_off, m_off, tauZ, 1, bs);
          kstar = bisect_result<1>(k1, c_off, bs, k);
          __builtin_amdgcn_wave_barrier();  // the next row's compaction writes the same area
        }
      }
      cut = row[sel_index(kstar)];
    }
    const double hiT = cut + kTieEps;

    // |S+| : blocks strictly above the tie band
    int nplus = 0;
#pragma unroll
    for (int u = 0; u < E; ++u) nplus += __popcll(__ballot(u * 64 + lane < nB && row[min(u * 64 + lane, nB - 1)] > hiT));
    const int need = k - nplus;
    // write the row in index order; the first `need` tied blocks are kept.
    // As bits, the ballot of chunk u is word u of the row, stored by lane u.
    int tied_before = 0;
    uint64_t word = 0;
#pragma unroll
    for (int u = 0; u < E; ++u) {
      const int jj = u * 64 + lane;
      const bool ok = jj < nB;
      const double sv = row[min(jj, nB - 1)];
      const bool above = ok && sv > hiT;
      const bool tie = ok && fabs(sv - cut) <= kTieEps;
      const unsigned long long tb = __ballot(tie);
      const int rank = tied_before + __popcll(tb & ((1ull << lane) - 1ull));
      const bool keep = above || (tie && rank < need);
      if (bits == nullptr) {
        if (ok) mask[grow * nB + jj] = keep ? 1 : 0;
      } else {
        const uint64_t kw = __ballot(keep);
        word = lane == u ? kw : word;
      }
      tied_before += __popcll(tb);
    }
    const int nw = (nB + 63) / 64;
    if (bits != nullptr && lane < nw) bits[grow * nw + lane] = word;
  }
}

__global__ void fill_ones_kernel(uint8_t *p, size_t n) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 1;
}

}  // namespace

hipError_t launch_pool(View q, View k, int B, int H, int N, int d, int bs, double *qbar,
                       double *kbar, hipStream_t s) {
  const int nB = (N + bs - 1) / bs;
  dim3 grid(nB, B * H, 2);
  if (d == 128)
    hipLaunchKernelGGL(pool_kernel<128>, grid, dim3(256), 0, s, q, k, H, N, bs, nB, qbar, kbar);
  else
    hipLaunchKernelGGL(pool_kernel<64>, grid, dim3(256), 0, s, q, k, H, N, bs, nB, qbar, kbar);
  return hipGetLastError();
}

template <int D, int R, int W, bool MASS>
static hipError_t launch_select_dr(const double *qbar, const double *kbar, int BH, int nB,
                                   double sigma, double tau, uint8_t *mask, uint64_t *bits,
                                   hipStream_t s) {
  const int G = (nB + R - 1) / R * BH;
  dim3 grid((G + 7) / 8 * 8);
  // the logits, then the pooled rows or phase 2's candidate buffers
  const size_t lds = ((size_t)R * nB + (size_t)max(R * (D + 2), W * 128)) * sizeof(double);
  const int need = (nB + 63) / 64;  // positions per lane
#define CARNATOR_SEL(EE)                                                                          \
  do {                                                                                            \
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(&select_kernel<D, EE, R, W, MASS>), \
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);     \
    if (e != hipSuccess) return e;                                                                \
    hipLaunchKernelGGL((select_kernel<D, EE, R, W, MASS>), grid, dim3(64 * W), lds, s, qbar, kbar, nB, \
                       sigma, tau, mask, bits, BH);                                               \
  } while (0)
  // W = 16 waves (1024 threads, at most 128 VGPRs) only while a lane holds at
  // most 8 positions; the launcher picks R and W accordingly
  if (need <= 1) CARNATOR_SEL(1);
  else if (need <= 2) CARNATOR_SEL(2);
  else if (need <= 3) CARNATOR_SEL(3);
  else if (need <= 4) CARNATOR_SEL(4);
  else if (need <= 6) CARNATOR_SEL(6);
  else if (need <= 8) CARNATOR_SEL(8);
  else if constexpr (W <= 8) {
    if (need <= 10) CARNATOR_SEL(10);
    else if (need <= 12) CARNATOR_SEL(12);
    else if (need <= 16) CARNATOR_SEL(16);
    else if constexpr (R <= 8) {  // R = 16 serves nB <= 1024 only
      if (need <= 24) CARNATOR_SEL(24);
      else if (need <= 32) CARNATOR_SEL(32);
      else return hipErrorInvalidValue;
    } else {
      return hipErrorInvalidValue;
    }
  } else {
    return hipErrorInvalidValue;
  }
#undef CARNATOR_SEL
  return hipGetLastError();
}

// R query blocks per workgroup: their logits and pooled rows (or the
// selection's candidate buffers, 1 KiB per wave) take 8 (R nB + max(R (d + 2),
// 128 W)) bytes of LDS, within 160 KiB for R = 16 up to nB = 1024 and for
// R = 8 up to nB = 2048.  R = 16 fills the 16-row fp64 MFMA tiles
// and halves the kbar re-reads.  W = 16 waves (one row each) while a lane's
// share of a row (E <= 8 positions) fits the 128 registers of a 1024-thread
// workgroup, else W = 8 (two rows each when R = 16).
template <int D>
static hipError_t launch_select_d(const double *qbar, const double *kbar, int BH, int nB,
                                  double sigma, double tau, uint8_t *mask, uint64_t *bits,
                                  hipStream_t s) {
  if (nB <= 512) return launch_select_dr<D, 16, 16, false>(qbar, kbar, BH, nB, sigma, tau, mask, bits, s);
  if (nB <= 1024) return launch_select_dr<D, 16, 8, false>(qbar, kbar, BH, nB, sigma, tau, mask, bits, s);
  return launch_select_dr<D, 8, 8, false>(qbar, kbar, BH, nB, sigma, tau, mask, bits, s);
}

hipError_t launch_select(const double *qbar, const double *kbar, int BH, int nB, int d,
                         double sigma, double tau, uint8_t *mask, uint64_t *bits,
                         hipStream_t s) {
  if (d == 128) return launch_select_d<128>(qbar, kbar, BH, nB, sigma, tau, mask, bits, s);
  return launch_select_d<64>(qbar, kbar, BH, nB, sigma, tau, mask, bits, s);
}

hipError_t launch_select_mass(const double *mass, int BH, int nB, double tau, uint8_t *mask,
                              uint64_t *bits, hipStream_t s) {
  // the pooled-row area of the LDS layout is not used: the smallest D
  if (nB <= 512) return launch_select_dr<64, 16, 16, true>(mass, nullptr, BH, nB, 1.0, tau, mask, bits, s);
  if (nB <= 1024) return launch_select_dr<64, 16, 8, true>(mass, nullptr, BH, nB, 1.0, tau, mask, bits, s);
  return launch_select_dr<64, 8, 8, true>(mass, nullptr, BH, nB, 1.0, tau, mask, bits, s);
}

hipError_t launch_fill_ones(uint8_t *p, size_t n, hipStream_t s) {
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(fill_ones_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, p, n);
  return hipGetLastError();
}

}  // namespace carnator
