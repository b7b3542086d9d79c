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
