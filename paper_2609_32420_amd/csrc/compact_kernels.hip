// Target-row widening of the reused mask and its compaction into per-row
// lists of kept key blocks.
//
// Widening (Sec. 3.3, joint reuse in the middle layers): a target-specific
// query block evaluates every key block, and dense text key blocks are kept
// in every row.  Compaction produces the list the sparse executor walks:
// row_ptr / col_idx (ascending key blocks per row) and an order of rows by
// descending list length (lower row first on equal length), so the longest
// rows start first.
#include "internal.h"

namespace carnator {
namespace {

// One thread per mask byte.
__global__ void __launch_bounds__(256) merge_kernel(uint8_t *__restrict__ mask, int H, int nB,
                                                    int64_t total,
                                                    const uint8_t *__restrict__ rows,
                                                    const uint8_t *__restrict__ cols) {
  const int64_t x = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (x >= total) return;
  const int64_t nb2 = (int64_t)nB * nB;
  const int64_t bh = x / nb2;
  const int b = (int)(bh / H);
  const int rem = (int)(x - bh * nb2);
  const int i = rem / nB, j = rem - i * nB;
  const bool keep = mask[x] != 0 || rows[(int64_t)b * nB + i] != 0 ||
                    (cols != nullptr && cols[(int64_t)b * nB + j] != 0);
  mask[x] = keep ? 1 : 0;
}

// One wave per row: number of kept key blocks.
__global__ void __launch_bounds__(256) count_kernel(const uint8_t *__restrict__ mask, int64_t R,
                                                    int nB, int32_t *__restrict__ len) {
  const int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (r >= R) return;
  const uint8_t *row = mask + r * nB;
  int n = 0;
  for (int base = 0; base < nB; base += 64) {
    const int j = base + lane;
    n += __popcll(__ballot(j < nB && row[j] != 0));
  }
  if (lane == 0) len[r] = n;
}

// One wave per row: ascending kept key blocks at col_idx[row_ptr[r] ...].
__global__ void __launch_bounds__(256) fill_kernel(const uint8_t *__restrict__ mask, int64_t R,
                                                   int nB, const int32_t *__restrict__ row_ptr,
                                                   int32_t *__restrict__ col_idx) {
  const int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (r >= R) return;
  const uint8_t *row = mask + r * nB;
  int pos = row_ptr[r];
  for (int base = 0; base < nB; base += 64) {
    const int j = base + lane;
    const bool kept = j < nB && row[j] != 0;
    const unsigned long long bits = __ballot(kept);
    if (kept) col_idx[pos + __popcll(bits & ((1ull << lane) - 1ull))] = j;
    pos += __popcll(bits);
  }
}

constexpr int kScanThreads = 1024;
constexpr int kRadixBits = 3;
constexpr int kBins = 1 << kRadixBits;

// Block-wide exclusive scan of one int per thread (1024 threads); returns the
// exclusive prefix and writes the total to *total.
__device__ int block_excl_scan(int v, int *sh, int *total) {
  const int t = threadIdx.x;
  const int lane = t & 63, w = t >> 6;
  int x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  if (lane == 63) sh[w] = x;
  __syncthreads();
  if (w == 0) {
    int s = lane < kScanThreads / 64 ? sh[lane] : 0;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int y = __shfl_up(s, o);
      if (lane >= o) s += y;
    }
    if (lane < kScanThreads / 64) sh[lane] = s;
  }
  __syncthreads();
  const int before = (w > 0 ? sh[w - 1] : 0) + x - v;
  *total = sh[kScanThreads / 64 - 1];
  __syncthreads();
  return before;
}

// Rows up to which the lengths and both intermediate permutations of the
// sort live in LDS (3 x 32 KiB beside the 32 KiB histogram) instead of HBM:
// the passes are chains of dependent accesses, and in LDS each costs a few
// hundred cycles instead of an L2 round trip.
constexpr int64_t kLdsRows = 8192;

// Single workgroup: row_ptr = exclusive scan of len, and a stable LSD radix
// sort of the rows by key (nB - len), i.e. descending length, ascending row.
// Each thread owns a contiguous range of rows, so every pass is stable.
template <bool IN_LDS>
__global__ void __launch_bounds__(kScanThreads) scan_sort_kernel(const int32_t *__restrict__ len_g,
                                                                 int64_t R, int nB,
                                                                 int32_t *__restrict__ row_ptr,
                                                                 int32_t *__restrict__ order,
                                                                 int32_t *__restrict__ tmp0,
                                                                 int32_t *__restrict__ tmp1) {
  __shared__ int sh[kScanThreads / 64];
  __shared__ int hist[kBins][kScanThreads];
  extern __shared__ int rows_lds[];  // IN_LDS: len [R], then two permutations [R]
  const int t = threadIdx.x;
  // Accessors: with IN_LDS the arrays are indexed through the LDS array itself
  // (plain LDS instructions; through a generic pointer every access would be a
  // flat one, waiting on both the LDS and the memory counters).
  auto lenv = [&](int64_t r) __attribute__((always_inline)) -> int {
    if constexpr (IN_LDS) return rows_lds[r];
    else return len_g[r];
  };
  auto perm_get = [&](int buf, int64_t x) __attribute__((always_inline)) -> int {
    if constexpr (IN_LDS) return rows_lds[R * (1 + buf) + x];
    else return (buf ? tmp1 : tmp0)[x];
  };
  auto perm_put = [&](bool last, int buf, int64_t pos, int r) __attribute__((always_inline)) {
    if (last) order[pos] = r;
    else if constexpr (IN_LDS) rows_lds[R * (1 + buf) + pos] = r;
    else (buf ? tmp1 : tmp0)[pos] = r;
  };
  if constexpr (IN_LDS) {
    // all of a thread's loads in flight at once (R <= kLdsRows), clamped
    // indices instead of branches
    constexpr int kPer = (int)(kLdsRows / kScanThreads);
    int v[kPer];
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      const int64_t r = t + (int64_t)i * kScanThreads;
      v[i] = len_g[r < R ? r : R - 1];
    }
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      const int64_t r = t + (int64_t)i * kScanThreads;
      if (r < R) rows_lds[r] = v[i];
    }
    __syncthreads();
  }
  const int64_t per = (R + kScanThreads - 1) / kScanThreads;
  const int64_t lo = min<int64_t>(R, per * t), hi = min<int64_t>(R, lo + per);

  // ---- row_ptr
  int local = 0;
  for (int64_t r = lo; r < hi; ++r) local += lenv(r);
  int total;
  int run = block_excl_scan(local, sh, &total);
  for (int64_t r = lo; r < hi; ++r) {
    row_ptr[r] = run;
    run += lenv(r);
  }
  if (t == 0) row_ptr[R] = total;

  // ---- order: key = nB - len, passes of 3 bits; pass p reads the
  // permutation of pass p - 1 (buffer (p - 1) & 1; identity for p = 0) and
  // writes buffer p & 1, the last pass `order`
  int passes = 0;
  for (int v = nB; v > 0; v >>= kRadixBits) ++passes;
  for (int p = 0; p < passes; ++p) {
    const int shift = p * kRadixBits;
    const bool last = p == passes - 1;
#pragma unroll
    for (int bin = 0; bin < kBins; ++bin) hist[bin][t] = 0;
    for (int64_t x = lo; x < hi; ++x) {
      const int r = p ? perm_get((p - 1) & 1, x) : (int)x;
      const int dig = ((nB - lenv(r)) >> shift) & (kBins - 1);
      hist[dig][t] += 1;
    }
    __syncthreads();
    // exclusive scan over hist in (bin, thread) order: thread t owns the kBins
    // consecutive entries [kBins*t, kBins*t + kBins) of the flattened array
    int *flat = &hist[0][0];
    int vals[kBins];
    int s = 0;
#pragma unroll
    for (int q = 0; q < kBins; ++q) {
      vals[q] = flat[kBins * t + q];
      s += vals[q];
    }
    int tot;
    int base = block_excl_scan(s, sh, &tot);
#pragma unroll
    for (int q = 0; q < kBins; ++q) {
      flat[kBins * t + q] = base;
      base += vals[q];
    }
    __syncthreads();
    for (int64_t x = lo; x < hi; ++x) {
      const int r = p ? perm_get((p - 1) & 1, x) : (int)x;
      const int dig = ((nB - lenv(r)) >> shift) & (kBins - 1);
      perm_put(last, p & 1, hist[dig][t]++, r);
    }
    if constexpr (!IN_LDS) __threadfence_block();
    __syncthreads();
  }
  if (passes == 0) {
    for (int64_t x = lo; x < hi; ++x) order[x] = (int)x;
  }
}

}  // namespace

hipError_t launch_merge(uint8_t *mask, int B, int H, int nB, const uint8_t *rows,
                        const uint8_t *cols, hipStream_t s) {
  const int64_t total = (int64_t)B * H * nB * nB;
  hipLaunchKernelGGL(merge_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, s, mask, H,
                     nB, total, rows, cols);
  return hipGetLastError();
}

size_t compact_scratch_bytes(int64_t R) { return 3 * align_up((size_t)R * sizeof(int32_t)); }

hipError_t launch_compact(const uint8_t *mask, int64_t R, int nB, int32_t *row_ptr,
                          int32_t *col_idx, int32_t *order, void *scratch, hipStream_t s) {
  char *ws = static_cast<char *>(scratch);
  const size_t part = align_up((size_t)R * sizeof(int32_t));
  int32_t *len = reinterpret_cast<int32_t *>(ws);
  int32_t *tmp0 = reinterpret_cast<int32_t *>(ws + part);
  int32_t *tmp1 = reinterpret_cast<int32_t *>(ws + 2 * part);
  const unsigned g = (unsigned)((R + 3) / 4);
  hipLaunchKernelGGL(count_kernel, dim3(g), dim3(256), 0, s, mask, R, nB, len);
  if (R <= kLdsRows) {
    const size_t lds = (size_t)3 * R * sizeof(int32_t);
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(&scan_sort_kernel<true>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(scan_sort_kernel<true>, dim3(1), dim3(kScanThreads), lds, s, len, R, nB,
                       row_ptr, order, tmp0, tmp1);
  } else {
    hipLaunchKernelGGL(scan_sort_kernel<false>, dim3(1), dim3(kScanThreads), 0, s, len, R, nB,
                       row_ptr, order, tmp0, tmp1);
  }
  hipLaunchKernelGGL(fill_kernel, dim3(g), dim3(256), 0, s, mask, R, nB, row_ptr, col_idx);
  return hipGetLastError();
}

}  // namespace carnator
