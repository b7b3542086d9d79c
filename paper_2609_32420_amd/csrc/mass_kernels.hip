// Exact (token-level) attention mass of every block pair of the historical
// run: Appendix C.3 keeps, per head and query block, the smallest set of key
// blocks covering a fixed fraction of the source attention mass; read
// literally, that mass is the historical softmax attention summed over the
// tokens of each block pair (the pooled builder of mask_kernels.hip
// estimates it from block means).
//
//   M[b,h,i,j] = (1 / n_i) sum_{a in block i} sum_{t in block j}
//                softmax_t(sigma q_a . k_t)        (rows sum to 1)
//
// Pass 1 (mass_pass_kernel): one workgroup of 8 waves per 512 queries (four
// blocks of 128 or eight of 64), 64 queries per wave in two sets of 32 (each
// K operand read from LDS feeds two MFMAs), streams every key block of its
// head through LDS (each load serves 512 queries) and computes
// S^T = K Q^T on bf16 MFMA 32x32x16 (fp32 accumulation), keys as MFMA rows so
// that a query's scores sit in one lane pair.  After key block j each query
// records (m_j, s_j): its running maximum (log2 units) and the block's
// sum of 2^(x - m_j); at the end its log2-sum-exp L.  Pass 2
// (mass_reduce_kernel) forms M_ij = sum_a s_j 2^(m_j - L) / n_i (the powers in
// fp32, the sum in fp64).
// The records are block-major ([bh][j][a]) so a wave's 32 queries write 256
// contiguous bytes.
#include "internal.h"

#include <algorithm>

namespace carnator {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

// 16-byte chunk c of K row r sits in slot c ^ swz(r): the 32 rows an operand
// read touches at one chunk spread over the LDS banks.
template <int CPR>
__device__ inline int mswz(int r) {
  if constexpr (CPR == 16) return r & 15;
  else return (r >> 1) & 7;
}

constexpr int kMassWaves = 8;  // 64 queries per wave, 512 per workgroup
constexpr int kMassQueries = 64 * kMassWaves;

// Softmax statistics of one query (pair-uniform): the running maximum and
// sum over the key blocks done, and the current block's maximum and this
// lane's share of its sum.
struct MassState {
  float m_run, l_run, mb, sl;
};

// Fold one 32-key tile of scores (raw; with MASK, keys at or past lim
// masked: only the last key block can be partial) into st.
template <bool MASK>
__device__ __attribute__((always_inline)) inline void mass_tile(MassState &st, f32x16 acc, int m,
                                                                int hh, int lim, float c2) {
  float tm = -INFINITY;
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    if constexpr (MASK) {
      const int key = m * 32 + 8 * (v >> 2) + 4 * hh + (v & 3);
      acc[v] = key < lim ? acc[v] : -INFINITY;
    }
    tm = fmaxf(tm, acc[v]);
  }
  tm = fmaxf(tm, __shfl_xor(tm, 32)) * c2;
  const float mn = fmaxf(st.mb, tm);
  float ts = 0.f;
#pragma unroll
  for (int v = 0; v < 16; ++v) ts += __builtin_amdgcn_exp2f(fmaf(acc[v], c2, -mn));
  st.sl = st.sl * __builtin_amdgcn_exp2f(st.mb == -INFINITY ? -INFINITY : st.mb - mn) + ts;
  st.mb = mn;
}

// One 32-key tile of S^T = K Q^T for both query sets: each K operand (row r
// of the tile for this lane, chunks 2 t + hh, from LDS) feeds two MFMAs.
template <int D, int CPR>
__device__ __attribute__((always_inline)) inline void qk_tile2(const unsigned char *row, int r,
                                                                int hh, const bf16x8 (&q0)[D / 16],
                                                                const bf16x8 (&q1)[D / 16],
                                                                f32x16 &acc0, f32x16 &acc1) {
  acc0 = f32x16{};
  acc1 = f32x16{};
#pragma unroll
  for (int t = 0; t < D / 16; ++t) {
    const int c = 2 * t + hh;
    const bf16x8 kv = *reinterpret_cast<const bf16x8 *>(row + 16 * (c ^ mswz<CPR>(r)));
    acc0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kv, q0[t], acc0, 0, 0, 0);
    acc1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kv, q1[t], acc1, 0, 0, 0);
  }
}

template <int D, int BS>
struct MassCfg {
  static constexpr int QPW = kMassQueries / BS;  // query blocks per workgroup
  static constexpr int NT = 64 * kMassWaves;
  static constexpr int CPR = D / 8;        // 16-byte chunks per K row
  static constexpr int RB = D * 2;         // bytes per K row
  static constexpr int TILE = BS * RB;     // one key block in LDS
  static constexpr int LDS = 2 * TILE;     // double buffer
  static constexpr int CPT = BS * CPR / NT;  // chunks loaded per thread per block
  static_assert(BS * CPR % NT == 0, "chunk split");
};

template <int D, int BS>
__global__ void __launch_bounds__(64 * kMassWaves)
mass_pass_kernel(View q, View k, int H, int N, int nB, int bh0, float c2,
                 float2 *__restrict__ rec, float *__restrict__ lse2) {
  using C = MassCfg<D, BS>;
  extern __shared__ __attribute__((aligned(1024))) unsigned char lds[];
  const int ng = (nB + C::QPW - 1) / C::QPW;  // query groups per head
  const int qg = (int)(blockIdx.x % ng);
  // heads bh0 .. of the chunk this launch covers; records and log2-sum-exps
  // are indexed inside the chunk
  const int bc = (int)(blockIdx.x / ng);
  const int bh = bh0 + bc;
  const int b = bh / H, h = bh - b * H;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int l32 = lane & 31, hh = lane >> 5;
  // this lane's two queries: l32 of each of the wave's two sets of 32
  const int a0 = qg * kMassQueries + wave * 64 + l32, a1 = a0 + 32;
  const bool qv0 = a0 < N, qv1 = a1 < N;

  // Q as the B operand: query l32 of a set, channels 16 t + 8 hh .. + 8
  bf16x8 q0[D / 16], q1[D / 16];
  {
    const uint16_t *qh = q.data + (int64_t)b * q.sb + (int64_t)h * q.sh;
    const uint16_t *p0 = qh + (int64_t)min(a0, N - 1) * q.sn;
    const uint16_t *p1 = qh + (int64_t)min(a1, N - 1) * q.sn;
#pragma unroll
    for (int t = 0; t < D / 16; ++t) {
      const uint4 v0 = *reinterpret_cast<const uint4 *>(p0 + 16 * t + 8 * hh);
      const uint4 v1 = *reinterpret_cast<const uint4 *>(p1 + 16 * t + 8 * hh);
      q0[t] = qv0 ? __builtin_bit_cast(bf16x8, v0) : bf16x8{};
      q1[t] = qv1 ? __builtin_bit_cast(bf16x8, v1) : bf16x8{};
    }
  }
  const uint16_t *kbase = k.data + (int64_t)b * k.sb + (int64_t)h * k.sh;

  // staged chunks of a key block: chunk x = tid + u NT covers row x / CPR,
  // 16-byte chunk x % CPR (rows past N read row N - 1, blocks past nB - 1
  // block nB - 1; their scores are masked or unused).
  // Two register stages: the load of key block j + 2 is issued right after
  // block j + 1 is stored to LDS, so it has two blocks of compute to land.
  // The loop is unrolled by two so both stage arrays stay in registers, and
  // runs an even number of bodies (an odd nB ends with one masked body over
  // the LDS buffer it finds: nothing is recorded from it).
  // (named registers, not arrays: arrays live across the loop's back edge
  // were kept in scratch memory, each prefetch then waited for at once)
  static_assert(C::CPT <= 4, "stage size");
  uint4 sa0, sa1, sa2, sa3, sb0, sb1, sb2, sb3;
#define CARNATOR_MASS_CHUNK_LOAD(V, U, J)                                                \
  if constexpr ((U) < C::CPT) {                                                          \
    const int x = (int)threadIdx.x + (U) * C::NT;                                        \
    const int r = x / C::CPR, c = x - r * C::CPR;                                        \
    const int tok = min(min(J, nB - 1) * BS + r, N - 1);                                 \
    V = *reinterpret_cast<const uint4 *>(kbase + (int64_t)tok * k.sn + 8 * c);           \
  }
#define CARNATOR_MASS_CHUNK_STORE(V, U, BUF)                                             \
  if constexpr ((U) < C::CPT) {                                                          \
    const int x = (int)threadIdx.x + (U) * C::NT;                                        \
    const int r = x / C::CPR, c = x - r * C::CPR;                                        \
    *reinterpret_cast<uint4 *>(lds + (BUF) * C::TILE + r * C::RB +                       \
                               16 * (c ^ mswz<C::CPR>(r))) = V;                          \
  }
#define CARNATOR_MASS_LOAD(ST, J)                                                        \
  CARNATOR_MASS_CHUNK_LOAD(ST##0, 0, J) CARNATOR_MASS_CHUNK_LOAD(ST##1, 1, J)            \
  CARNATOR_MASS_CHUNK_LOAD(ST##2, 2, J) CARNATOR_MASS_CHUNK_LOAD(ST##3, 3, J)
#define CARNATOR_MASS_STORE(ST, BUF)                                                     \
  CARNATOR_MASS_CHUNK_STORE(ST##0, 0, BUF) CARNATOR_MASS_CHUNK_STORE(ST##1, 1, BUF)      \
  CARNATOR_MASS_CHUNK_STORE(ST##2, 2, BUF) CARNATOR_MASS_CHUNK_STORE(ST##3, 3, BUF)

  CARNATOR_MASS_LOAD(sa, 0)
  CARNATOR_MASS_STORE(sa, 0)
  CARNATOR_MASS_LOAD(sa, 1)
  CARNATOR_MASS_LOAD(sb, 2)
  __syncthreads();

  MassState s0 = {-INFINITY, 0.f, -INFINITY, 0.f}, s1 = s0;
  // one key block: LDS buffer jj & 1 holds block jj, S1 holds block jj + 1
  // and S2 block jj + 2 (both in flight); S1 is stored for the next body and
  // refilled with block jj + 3
#define CARNATOR_MASS_BODY(JJ, S1, MASK)                                                 \
  {                                                                                      \
    const int jj = (JJ);                                                                 \
    const bool live = jj < nB;                                                           \
    const unsigned char *base = lds + (jj & 1) * C::TILE;                                \
    const int lim = N - jj * BS;                                                         \
    s0.mb = s0.m_run, s0.sl = 0.f, s1.mb = s1.m_run, s1.sl = 0.f;                        \
    _Pragma("unroll") for (int m = 0; m < BS / 32; ++m) {                                \
      const int r = m * 32 + l32;                                                        \
      f32x16 acc0, acc1;                                                                 \
      qk_tile2<D, C::CPR>(base + r * C::RB, r, hh, q0, q1, acc0, acc1);                  \
      mass_tile<MASK>(s0, acc0, m, hh, lim, c2);                                         \
      mass_tile<MASK>(s1, acc1, m, hh, lim, c2);                                         \
    }                                                                                    \
    const float t0 = s0.sl + __shfl_xor(s0.sl, 32), t1 = s1.sl + __shfl_xor(s1.sl, 32);  \
    if (live) {                                                                          \
      s0.l_run = s0.l_run * __builtin_amdgcn_exp2f(s0.m_run == -INFINITY ? -INFINITY : s0.m_run - s0.mb) + t0; \
      s0.m_run = s0.mb;                                                                  \
      s1.l_run = s1.l_run * __builtin_amdgcn_exp2f(s1.m_run == -INFINITY ? -INFINITY : s1.m_run - s1.mb) + t1; \
      s1.m_run = s1.mb;                                                                  \
      float2 *rj = rec + ((int64_t)bc * nB + jj) * N;                                    \
      if (hh == 0 && qv0) rj[a0] = make_float2(s0.mb, t0);                               \
      if (hh == 0 && qv1) rj[a1] = make_float2(s1.mb, t1);                               \
    }                                                                                    \
    CARNATOR_MASS_STORE(S1, (jj + 1) & 1)                                                \
    __syncthreads();                                                                     \
    CARNATOR_MASS_LOAD(S1, jj + 3)                                                       \
  }

  // every key block but the last is full: the pairs before the one holding
  // block nB - 1 take no key mask
  const int jl = (nB - 1) & ~1;
  for (int j = 0; j < jl; j += 2) {
    CARNATOR_MASS_BODY(j, sa, false)
    CARNATOR_MASS_BODY(j + 1, sb, false)
  }
  CARNATOR_MASS_BODY(jl, sa, true)
  CARNATOR_MASS_BODY(jl + 1, sb, true)
#undef CARNATOR_MASS_BODY
#undef CARNATOR_MASS_LOAD
#undef CARNATOR_MASS_STORE
#undef CARNATOR_MASS_CHUNK_LOAD
#undef CARNATOR_MASS_CHUNK_STORE
  if (hh == 0 && qv0) lse2[(int64_t)bc * N + a0] = s0.m_run + log2f(s0.l_run);
  if (hh == 0 && qv1) lse2[(int64_t)bc * N + a1] = s1.m_run + log2f(s1.l_run);
}

// One wave per (bh, i): lane l holds queries a0 + l and a0 + 64 + l of block
// i (the valid ones among them) and their L; the wave walks the key blocks
// j, eight at a time with all their record loads in flight, and forms
// M_ij = sum_a s 2^(m - L_a) / n_i with one wave sum per j.  2^(m - L) is
// taken in fp32 (m <= L, both fp32 log2 values; relative error ~1e-6) and
// the terms are summed in fp64.
constexpr int kReduceUnroll = 8;
__global__ void __launch_bounds__(256) mass_reduce_kernel(const float2 *__restrict__ rec,
                                                          const float *__restrict__ lse2, int N,
                                                          int nB, int bs, int rows,
                                                          double *__restrict__ mass) {
  const int w = (int)blockIdx.x * 4 + (int)(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (w >= rows) return;  // the whole wave
  const int i = w % nB, bh = w / nB;
  const int a0 = i * bs, a1 = min(a0 + bs, N);
  const int qa = a0 + lane, qb = a0 + 64 + lane;
  const bool va = qa < a1, vb = qb < a1;
  const int ca = min(qa, N - 1), cb = min(qb, N - 1);  // clamped: loads stay in the head
  const float *lh = lse2 + (int64_t)bh * N;
  const float La = lh[ca], Lb = lh[cb];
  const float2 *rh = rec + (int64_t)bh * nB * N;
  const double inv = 1.0 / (double)(a1 - a0);
  double *out = mass + (int64_t)w * nB;
  for (int j0 = 0; j0 < nB; j0 += kReduceUnroll) {
    float2 ra[kReduceUnroll], rb[kReduceUnroll];
#pragma unroll
    for (int u = 0; u < kReduceUnroll; ++u) {
      const float2 *rj = rh + (int64_t)min(j0 + u, nB - 1) * N;
      ra[u] = rj[ca];
      rb[u] = rj[cb];
    }
#pragma unroll
    for (int u = 0; u < kReduceUnroll; ++u) {
      double t = va ? (double)(ra[u].y * __builtin_amdgcn_exp2f(ra[u].x - La)) : 0.0;
      t += vb ? (double)(rb[u].y * __builtin_amdgcn_exp2f(rb[u].x - Lb)) : 0.0;
      t = wave_sum(t);
      if (lane == 0 && j0 + u < nB) out[j0 + u] = t * inv;
    }
  }
}

}  // namespace

// The records take 8 bytes per (query, key block) of a head: 67 MB at 32K
// tokens, 887 MB at 119K.  Heads are processed in chunks whose records fit
// in kMassScratchCap (at least one head per chunk), so the workspace stays
// bounded whatever the number of heads.
constexpr size_t kMassScratchCap = (size_t)4 << 30;

static size_t mass_head_bytes(int N, int nB) {
  return (size_t)nB * N * sizeof(float2) + (size_t)N * sizeof(float);
}

static int mass_chunk_heads(int BH, int N, int nB) {
  const size_t per = mass_head_bytes(N, nB);
  const size_t fit = kMassScratchCap / per;
  return (int)std::max<size_t>(1, std::min<size_t>(fit, (size_t)BH));
}

size_t mass_scratch_bytes(int BH, int N, int nB) {
  const int ch = mass_chunk_heads(BH, N, nB);
  return align_up((size_t)ch * nB * N * sizeof(float2)) + align_up((size_t)ch * N * sizeof(float));
}

hipError_t launch_mass(View q, View k, int B, int H, int N, int d, int bs, float scale,
                       double *mass, void *scratch, hipStream_t s) {
  const int nB = (N + bs - 1) / bs;
  const int BH = B * H;
  const int ch = mass_chunk_heads(BH, N, nB);
  float2 *rec = static_cast<float2 *>(scratch);
  float *lse2 = reinterpret_cast<float *>(static_cast<char *>(scratch) +
                                          align_up((size_t)ch * nB * N * sizeof(float2)));
  const float c2 = scale * 1.4426950408889634f;
  const int qpw = kMassQueries / bs;
  for (int bh0 = 0; bh0 < BH; bh0 += ch) {
    const int nh = std::min(ch, BH - bh0);
    const dim3 grid((unsigned)(nh * ((nB + qpw - 1) / qpw)));
    hipError_t e = hipSuccess;
#define CARNATOR_MASS(DD, BB)                                                                    \
  do {                                                                                           \
    using C = MassCfg<DD, BB>;                                                                   \
    e = hipFuncSetAttribute(reinterpret_cast<const void *>(&mass_pass_kernel<DD, BB>),           \
                            hipFuncAttributeMaxDynamicSharedMemorySize, C::LDS);                 \
    if (e != hipSuccess) return e;                                                               \
    hipLaunchKernelGGL((mass_pass_kernel<DD, BB>), grid, dim3(C::NT), C::LDS, s, q, k, H, N, nB, \
                       bh0, c2, rec, lse2);                                                      \
  } while (0)
    if (d == 128 && bs == 128) CARNATOR_MASS(128, 128);
    else if (d == 128 && bs == 64) CARNATOR_MASS(128, 64);
    else if (d == 64 && bs == 128) CARNATOR_MASS(64, 128);
    else CARNATOR_MASS(64, 64);
#undef CARNATOR_MASS
    const int rows = nh * nB;
    hipLaunchKernelGGL(mass_reduce_kernel, dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, s, rec,
                       lse2, N, nB, bs, rows, mass + (int64_t)bh0 * nB * nB);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace carnator
