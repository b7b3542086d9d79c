// Internal declarations of the HIP library: launchers implemented in the
// kernel files and called by the C-ABI entry points in api.hip.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stddef.h>

namespace carnator {

constexpr size_t kAlign = 256;
inline size_t align_up(size_t x, size_t a = kAlign) { return (x + a - 1) / a * a; }

// Strided bf16 [B, H, N, d] view in element units.
struct View {
  const uint16_t *data;
  int64_t sb, sh, sn;
};

// ---- wave-wide reductions (device code of every kernel file) ----------------
// Cross-lane partner values for wave-wide reductions without LDS round
// trips: quad permutes (lane ^ 1, lane ^ 2), the half-row and row mirrors
// (lane 7 - i and 15 - i within 8 and 16 lanes) and the 16- and 32-lane
// swaps.  After the steps below 2^s every lane of a 2^s-lane group holds the
// group's value, so the mirrors pair each group with its sibling, and every
// lane ends with the same result (each step combines the same two operands
// in every lane; + and max are commutative).
template <int O>
__device__ inline uint32_t partner32(uint32_t x, int lane) {
  if constexpr (O == 1) return __builtin_amdgcn_update_dpp(0u, x, 0xB1, 0xF, 0xF, false);
  else if constexpr (O == 2) return __builtin_amdgcn_update_dpp(0u, x, 0x4E, 0xF, 0xF, false);
  else if constexpr (O == 4) return __builtin_amdgcn_update_dpp(0u, x, 0x141, 0xF, 0xF, false);
  else if constexpr (O == 8) return __builtin_amdgcn_update_dpp(0u, x, 0x140, 0xF, 0xF, false);
  else if constexpr (O == 16) {
    const auto r = __builtin_amdgcn_permlane16_swap(x, x, false, false);
    return (lane & 16) ? r[0] : r[1];
  } else {
    const auto r = __builtin_amdgcn_permlane32_swap(x, x, false, false);
    return (lane & 32) ? r[0] : r[1];
  }
}
template <int O>
__device__ inline uint64_t partner64(uint64_t x, int lane) {
  const uint32_t lo = partner32<O>((uint32_t)x, lane);
  const uint32_t hi = partner32<O>((uint32_t)(x >> 32), lane);
  return ((uint64_t)hi << 32) | lo;
}
template <int O>
__device__ inline double partner_f64(double x, int lane) {
  return __longlong_as_double((long long)partner64<O>((uint64_t)__double_as_longlong(x), lane));
}
template <typename T, typename F>
__device__ inline T dpp_reduce(T x, int lane, F op) {
  if constexpr (sizeof(T) == 8 && !__is_same(T, double)) {
    x = op(x, partner64<1>(x, lane));
    x = op(x, partner64<2>(x, lane));
    x = op(x, partner64<4>(x, lane));
    x = op(x, partner64<8>(x, lane));
    x = op(x, partner64<16>(x, lane));
    x = op(x, partner64<32>(x, lane));
  } else {
    x = op(x, partner_f64<1>(x, lane));
    x = op(x, partner_f64<2>(x, lane));
    x = op(x, partner_f64<4>(x, lane));
    x = op(x, partner_f64<8>(x, lane));
    x = op(x, partner_f64<16>(x, lane));
    x = op(x, partner_f64<32>(x, lane));
  }
  return x;
}
__device__ inline double dpp_sum(double x, int lane) {
  return dpp_reduce(x, lane, [](double a, double b) { return a + b; });
}
__device__ inline double dpp_max(double x, int lane) {
  return dpp_reduce(x, lane, [](double a, double b) { return fmax(a, b); });
}
__device__ inline uint64_t dpp_min_u64(uint64_t x, int lane) {
  return dpp_reduce(x, lane, [](uint64_t a, uint64_t b) { return b < a ? b : a; });
}
__device__ inline uint64_t dpp_max_u64(uint64_t x, int lane) {
  return dpp_reduce(x, lane, [](uint64_t a, uint64_t b) { return b > a ? b : a; });
}


// ---- block mask builder ----------------------------------------------------
// Pools Q_hist and K_hist per block (fp64 means over valid tokens).
//   qbar:  fp64 [BH][nB][d]   (row-major)
//   kbar:  fp64 [BH][nB][d]
hipError_t launch_pool(View q, View k, int B, int H, int N, int d, int bs, double *qbar,
                       double *kbar, hipStream_t s);
// Scores, softmax over key blocks, top-mass selection with the tie rule; writes
// uint8 [BH][nB][nB].
hipError_t launch_select(const double *qbar, const double *kbar, int BH, int nB, int d,
                         double sigma, double tau, uint8_t *mask, hipStream_t s);
hipError_t launch_fill_ones(uint8_t *p, size_t n, hipStream_t s);

// ---- merge -----------------------------------------------------------------
hipError_t launch_merge(uint8_t *mask, int B, int H, int nB, const uint8_t *rows,
                        const uint8_t *cols, hipStream_t s);

// ---- compaction ------------------------------------------------------------
// Scratch needed by launch_compact, in bytes.
size_t compact_scratch_bytes(int64_t R);
hipError_t launch_compact(const uint8_t *mask, int64_t R, int nB, int32_t *row_ptr,
                          int32_t *col_idx, int32_t *order, void *scratch, hipStream_t s);

// ---- attention -------------------------------------------------------------
hipError_t launch_bsattn(View q, View k, View v, uint16_t *out, int64_t osb, int64_t osh,
                         int64_t osn, int B, int H, int N, int d, int bs, const int32_t *row_ptr,
                         const int32_t *col_idx, const int32_t *order, float scale, float *lse,
                         hipStream_t s);

// ---- signature scan ----------------------------------------------------------
hipError_t launch_sig(const float *query, int64_t nq, const float *bank, int64_t m, int64_t dim,
                      int64_t ld, int topk, int32_t *idx, float *sim, float *all_sim,
                      double *sims, hipStream_t s);

}  // namespace carnator
