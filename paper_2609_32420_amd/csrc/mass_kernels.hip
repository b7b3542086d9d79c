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
// Pass 1 (mass_pass_kernel): one workgroup per query block, 32 queries per
// wave, streams every key block of its head through LDS and computes
// S^T = K Q^T on bf16 MFMA 32x32x16 (fp32 accumulation), keys as MFMA rows so
// that a query's scores sit in one lane pair.  After key block j each query
// records (m_j, s_j): its running maximum (log2 units) and the block's
// sum of 2^(x - m_j); at the end its log2-sum-exp L.  Pass 2
// (mass_reduce_kernel) forms M_ij = sum_a s_j 2^(m_j - L) / n_i in fp64.
// The records are block-major ([bh][j][a]) so a wave's 32 queries write 256
// contiguous bytes.
#include "internal.h"

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

template <int D, int BS>
struct MassCfg {
  static constexpr int NT = 2 * BS;        // BS / 32 waves of 64 lanes
  static constexpr int CPR = D / 8;        // 16-byte chunks per K row
  static constexpr int RB = D * 2;         // bytes per K row
  static constexpr int TILE = BS * RB;     // one key block in LDS
  static constexpr int LDS = 2 * TILE;     // double buffer
  static constexpr int CPT = BS * CPR / NT;  // chunks loaded per thread per block
  static_assert(BS * CPR % NT == 0, "chunk split");
};

template <int D, int BS>
__global__ void __launch_bounds__(2 * BS, 2)
mass_pass_kernel(View q, View k, int H, int N, int nB, float c2, float2 *__restrict__ rec,
                 float *__restrict__ lse2) {
  using C = MassCfg<D, BS>;
  extern __shared__ __attribute__((aligned(1024))) unsigned char lds[];
  const int qb = (int)(blockIdx.x % nB);
  const int bh = (int)(blockIdx.x / nB);
  const int b = bh / H, h = bh - b * H;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int l32 = lane & 31, hh = lane >> 5;
  const int a = qb * BS + wave * 32 + l32;  // this lane's query
  const bool qvalid = a < N;

  // Q as the B operand: query l32, channels 16 t + 8 hh .. + 8
  bf16x8 qreg[D / 16];
  {
    const uint16_t *qp = q.data + (int64_t)b * q.sb + (int64_t)h * q.sh + (int64_t)min(a, N - 1) * q.sn;
#pragma unroll
    for (int t = 0; t < D / 16; ++t) {
      const uint4 v = *reinterpret_cast<const uint4 *>(qp + 16 * t + 8 * hh);
      qreg[t] = qvalid ? __builtin_bit_cast(bf16x8, v) : bf16x8{};
    }
  }
  const uint16_t *kbase = k.data + (int64_t)b * k.sb + (int64_t)h * k.sh;

  // staged chunks of the next key block: chunk x = tid + u NT covers row
  // x / CPR, 16-byte chunk x % CPR (rows past N read row N - 1; their scores
  // are masked).
  uint4 stage[C::CPT];
#define CARNATOR_MASS_LOAD(J)                                                           \
  _Pragma("unroll") for (int u = 0; u < C::CPT; ++u) {                                  \
    const int x = (int)threadIdx.x + u * C::NT;                                         \
    const int r = x / C::CPR, c = x - r * C::CPR;                                       \
    const int tok = min((J) * BS + r, N - 1);                                           \
    stage[u] = *reinterpret_cast<const uint4 *>(kbase + (int64_t)tok * k.sn + 8 * c);   \
  }
#define CARNATOR_MASS_STORE(BUF)                                                        \
  _Pragma("unroll") for (int u = 0; u < C::CPT; ++u) {                                  \
    const int x = (int)threadIdx.x + u * C::NT;                                         \
    const int r = x / C::CPR, c = x - r * C::CPR;                                       \
    *reinterpret_cast<uint4 *>(lds + (BUF) * C::TILE + r * C::RB +                      \
                               16 * (c ^ mswz<C::CPR>(r))) = stage[u];                  \
  }

  CARNATOR_MASS_LOAD(0)
  CARNATOR_MASS_STORE(0)
  __syncthreads();

  float m_run = -INFINITY, l_run = 0.f;
  for (int j = 0; j < nB; ++j) {
    // unconditional (the last iteration reloads block nB - 1 into the idle
    // buffer, which nothing reads afterwards): a load and a store under
    // branches would keep the staging array in scratch memory
    CARNATOR_MASS_LOAD(min(j + 1, nB - 1))
    const unsigned char *base = lds + (j & 1) * C::TILE;
    float x[BS / 32][16];
#pragma unroll
    for (int m = 0; m < BS / 32; ++m) {
      f32x16 acc = {};
      const int r = m * 32 + l32;
      const unsigned char *row = base + r * C::RB;
#pragma unroll
      for (int t = 0; t < D / 16; ++t) {
        const int c = 2 * t + hh;
        const bf16x8 kv = *reinterpret_cast<const bf16x8 *>(row + 16 * (c ^ mswz<C::CPR>(r)));
        acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kv, qreg[t], acc, 0, 0, 0);
      }
      // acc[v] is key 8 (v / 4) + 4 hh + (v % 4) of the tile for query l32
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int key = j * BS + m * 32 + 8 * (v >> 2) + 4 * hh + (v & 3);
        x[m][v] = key < N ? acc[v] * c2 : -INFINITY;
      }
    }
    float mb = -INFINITY;
#pragma unroll
    for (int m = 0; m < BS / 32; ++m)
#pragma unroll
      for (int v = 0; v < 16; ++v) mb = fmaxf(mb, x[m][v]);
    mb = fmaxf(mb, __shfl_xor(mb, 32));
    const float m_new = fmaxf(m_run, mb);
    float s = 0.f;
#pragma unroll
    for (int m = 0; m < BS / 32; ++m)
#pragma unroll
      for (int v = 0; v < 16; ++v) s += exp2f(x[m][v] - m_new);
    s += __shfl_xor(s, 32);
    l_run = l_run * exp2f(m_run - m_new) + s;
    m_run = m_new;
    if (hh == 0 && qvalid) rec[((int64_t)bh * nB + j) * N + a] = make_float2(m_new, s);
    CARNATOR_MASS_STORE((j + 1) & 1)
    __syncthreads();
  }
#undef CARNATOR_MASS_LOAD
#undef CARNATOR_MASS_STORE
  if (hh == 0 && qvalid) lse2[(int64_t)bh * N + a] = m_run + log2f(l_run);
}

// One wave per (bh, i, j): M_ij = sum over the valid queries a of block i of
// s 2^(m - L_a), divided by their number, in fp64.
__global__ void __launch_bounds__(256) mass_reduce_kernel(const float2 *__restrict__ rec,
                                                          const float *__restrict__ lse2, int N,
                                                          int nB, int bs, int64_t total,
                                                          double *__restrict__ mass) {
  const int64_t w = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (w >= total) return;
  const int j = (int)(w % nB);
  const int64_t bhi = w / nB;
  const int i = (int)(bhi % nB);
  const int64_t bh = bhi / nB;
  const int a0 = i * bs, a1 = min(a0 + bs, N);
  double acc = 0.0;
  for (int a = a0 + lane; a < a1; a += 64) {
    const float2 r = rec[(bh * nB + j) * N + a];
    acc += (double)r.y * exp2((double)r.x - (double)lse2[bh * N + a]);
  }
  acc = wave_sum(acc);
  if (lane == 0) mass[w] = acc / (double)(a1 - a0);
}

}  // namespace

size_t mass_scratch_bytes(int BH, int N, int nB) {
  return align_up((size_t)BH * nB * N * sizeof(float2)) + align_up((size_t)BH * N * sizeof(float));
}

hipError_t launch_mass(View q, View k, int B, int H, int N, int d, int bs, float scale,
                       double *mass, void *scratch, hipStream_t s) {
  const int nB = (N + bs - 1) / bs;
  const int BH = B * H;
  float2 *rec = static_cast<float2 *>(scratch);
  float *lse2 = reinterpret_cast<float *>(static_cast<char *>(scratch) +
                                          align_up((size_t)BH * nB * N * sizeof(float2)));
  const float c2 = scale * 1.4426950408889634f;
  const dim3 grid((unsigned)(BH * nB));
  hipError_t e = hipSuccess;
#define CARNATOR_MASS(DD, BB)                                                                   \
  do {                                                                                          \
    using C = MassCfg<DD, BB>;                                                                  \
    e = hipFuncSetAttribute(reinterpret_cast<const void *>(&mass_pass_kernel<DD, BB>),          \
                            hipFuncAttributeMaxDynamicSharedMemorySize, C::LDS);                \
    if (e != hipSuccess) return e;                                                              \
    hipLaunchKernelGGL((mass_pass_kernel<DD, BB>), grid, dim3(C::NT), C::LDS, s, q, k, H, N, nB, \
                       c2, rec, lse2);                                                          \
  } while (0)
  if (d == 128 && bs == 128) CARNATOR_MASS(128, 128);
  else if (d == 128 && bs == 64) CARNATOR_MASS(128, 64);
  else if (d == 64 && bs == 128) CARNATOR_MASS(64, 128);
  else CARNATOR_MASS(64, 64);
#undef CARNATOR_MASS
  const int64_t total = (int64_t)BH * nB * nB;
  hipLaunchKernelGGL(mass_reduce_kernel, dim3((unsigned)((total + 3) / 4)), dim3(256), 0, s, rec,
                     lse2, N, nB, bs, total, mass);
  return hipGetLastError();
}

}  // namespace carnator
