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
// x of lane l (l the same in every lane), in scalar registers.
__device__ inline uint64_t read_lane(uint64_t x, int l) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)x, l);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(x >> 32), l);
  return ((uint64_t)hi << 32) | lo;
}
// A value that is the same in every lane, moved to scalar registers (the
// compiler cannot prove it uniform by itself).
__device__ inline bool uniform(bool x) { return __builtin_amdgcn_readfirstlane((int)x) != 0; }
__device__ inline uint64_t uniform(uint64_t x) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)x);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(x >> 32));
  return ((uint64_t)hi << 32) | lo;
}
__device__ inline double uniform(double x) {
  return __longlong_as_double((long long)uniform((uint64_t)__double_as_longlong(x)));
}

// 64-bit DPP move: CTRL is the DPP control, ROWS the 16-lane rows written
// (the others are left undefined).
template <int CTRL, int ROWS>
__device__ inline uint64_t dpp64(uint64_t x) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_mov_dpp((int)(uint32_t)x, CTRL, ROWS, 0xF, false);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_mov_dpp((int)(uint32_t)(x >> 32), CTRL, ROWS, 0xF, false);
  return ((uint64_t)hi << 32) | lo;
}
// Wave-wide reduction to a scalar.  Four DPP steps combine each lane with
// lane ^ 1 and lane ^ 2 (quad permutes), then with its half-row and row
// mirrors (7 - i within 8 lanes, 15 - i within 16), after which every lane of
// a 16-lane row holds the row's value; two row broadcasts then add row 0
// into row 1 and row 2 into row 3 (lanes 15 and 47), and row 1 into row 3
// (lane 31), so that lane 63 holds the wave's value.  Lanes outside the rows
// a broadcast writes end with values that are never read.  The order of
// combination is fixed, so the result does not depend on scheduling.
template <typename F>
__device__ inline uint64_t wave_reduce_bits(uint64_t x, F op) {
  x = op(x, dpp64<0xB1, 0xF>(x));   // quad_perm [1, 0, 3, 2]
  x = op(x, dpp64<0x4E, 0xF>(x));   // quad_perm [2, 3, 0, 1]
  x = op(x, dpp64<0x141, 0xF>(x));  // row_half_mirror
  x = op(x, dpp64<0x140, 0xF>(x));  // row_mirror
  x = op(x, dpp64<0x142, 0xA>(x));  // row_bcast:15 into rows 1 and 3
  x = op(x, dpp64<0x143, 0xC>(x));  // row_bcast:31 into rows 2 and 3
  return read_lane(x, 63);
}
__device__ inline double bits_f64(uint64_t x) { return __longlong_as_double((long long)x); }
__device__ inline uint64_t f64_bits(double x) { return (uint64_t)__double_as_longlong(x); }
__device__ inline double wave_sum(double x) {
  return bits_f64(wave_reduce_bits(f64_bits(x), [](uint64_t a, uint64_t b) { return f64_bits(bits_f64(a) + bits_f64(b)); }));
}
__device__ inline double wave_max(double x) {
  return bits_f64(wave_reduce_bits(f64_bits(x), [](uint64_t a, uint64_t b) { return f64_bits(fmax(bits_f64(a), bits_f64(b))); }));
}
__device__ inline double wave_min(double x) {
  return bits_f64(wave_reduce_bits(f64_bits(x), [](uint64_t a, uint64_t b) { return f64_bits(fmin(bits_f64(a), bits_f64(b))); }));
}
__device__ inline uint64_t wave_min_u64(uint64_t x) {
  return wave_reduce_bits(x, [](uint64_t a, uint64_t b) { return b < a ? b : a; });
}
__device__ inline uint64_t wave_max_u64(uint64_t x) {
  return wave_reduce_bits(x, [](uint64_t a, uint64_t b) { return b > a ? b : a; });
}

// ---- block mask builder ----------------------------------------------------
// Pools Q_hist and K_hist per block (fp64 means over valid tokens).
//   qbar:  fp64 [BH][nB][d]   (row-major)
//   kbar:  fp64 [BH][nB][d]
hipError_t launch_pool(View q, View k, int B, int H, int N, int d, int bs, double *qbar,
                       double *kbar, hipStream_t s);
// Scores, softmax over key blocks, top-mass selection with the tie rule; writes
// uint8 [BH][nB][nB] to mask, or, when bits is non-NULL (mask then unused),
// bit-packed uint64 [BH][nB][ceil(nB / 64)].
hipError_t launch_select(const double *qbar, const double *kbar, int BH, int nB, int d,
                         double sigma, double tau, uint8_t *mask, uint64_t *bits, hipStream_t s);
hipError_t launch_fill_ones(uint8_t *p, size_t n, hipStream_t s);
// The same selection on given block masses [BH][nB][nB] (no softmax).
hipError_t launch_select_mass(const double *mass, int BH, int nB, double tau, uint8_t *mask,
                              uint64_t *bits, hipStream_t s);

// ---- exact block mass ----------------------------------------------------------
// M[bh][i][j] = mean over the valid queries of block i of the softmax mass of
// key block j (fp64, rows sum to 1), by a dense bf16 MFMA pass over the
// historical Q and K; scratch of mass_scratch_bytes.
size_t mass_scratch_bytes(int BH, int N, int nB);
hipError_t launch_mass(View q, View k, int B, int H, int N, int d, int bs, float scale,
                       double *mass, void *scratch, hipStream_t s);

// ---- merge -----------------------------------------------------------------
hipError_t launch_merge(uint8_t *mask, int B, int H, int nB, const uint8_t *rows,
                        const uint8_t *cols, hipStream_t s);

// ---- compaction ------------------------------------------------------------
// Scratch needed by launch_compact, in bytes (R rows of nB key blocks).
size_t compact_scratch_bytes(int64_t R, int nB);
// Heads per group of the row order: the most heads whose K and V (bf16,
// N x d each) fit kOrderGroupBytes, at least one and at least heads / 63;
// heads when all of them fit.
constexpr int64_t kOrderGroupBytes = (int64_t)256 << 20;
int order_group_heads(int heads, int64_t N, int d);
// group_rows: rows per head group of the order (>= R: the plain
// longest-first order).
hipError_t launch_compact(const uint8_t *mask, int64_t R, int nB, int64_t group_rows,
                          int32_t *row_ptr, int32_t *col_idx, int32_t *order, void *scratch,
                          hipStream_t s);

// ---- bit-packed masks --------------------------------------------------------
// R rows of nB keep flags as uint64 [R][ceil(nB / 64)], key block j at bit
// j mod 64 of word j / 64, bits past nB zero.
hipError_t launch_pack(const uint8_t *mask, int64_t R, int nB, uint64_t *bits, hipStream_t s);
hipError_t launch_unpack(const uint64_t *bits, int64_t R, int nB, uint8_t *mask, hipStream_t s);
hipError_t launch_fill_ones_bits(uint64_t *bits, int64_t R, int nB, hipStream_t s);
// Compaction of the packed mask [B][H][nB] rows, rows / cols uint8 [B][nB]
// each or NULL; scratch of compact_bits_scratch_bytes.  Widening (narrow
// false): flagged rows become full, flagged columns are added.  Restriction
// (narrow true): only flagged (active) rows and flagged (context) columns
// are kept; order lists the active rows first and *n_active (if not NULL)
// receives their number.
size_t compact_bits_scratch_bytes(int64_t R, int B, int nB);
hipError_t launch_compact_bits(const uint64_t *bits, int B, int H, int nB, int64_t group_rows,
                               const uint8_t *rows, const uint8_t *cols, bool narrow, int32_t *row_ptr,
                               int32_t *col_idx, int32_t *order, int32_t *n_active, void *scratch,
                               hipStream_t s);

// ---- region-restricted reuse -------------------------------------------------
// Region codes (3 evidence, 2 band, 1 context, 0 outside) and the blend
// weight W over [B][T][H][W] tokens from the evidence; scratch of
// region_scratch_bytes; a frame must fit region_frame_lds bytes of LDS (a
// workgroup stages a band of its rows with the rows within reach).
size_t region_frame_lds(int H, int W);
size_t region_scratch_bytes(int B, int T, int H, int W);
hipError_t launch_regions(const uint8_t *evidence, int B, int T, int H, int W, int ra, int rc,
                          uint8_t *region, float *weight, void *scratch, hipStream_t s);
// zo = W zt + (1 - W) zh over fp32 latents [B][C][Tl][Hl][Wl], W on the token
// grid [B][Tl / pt][Hl / ph][Wl / pw].
hipError_t launch_fusion(const float *zt, const float *zh, const float *weight, float *zo, int B,
                         int C, int Tl, int Hl, int Wl, int pt, int ph, int pw, hipStream_t s);
// Active query blocks and context key blocks (uint8 [B][nB]) from the region
// codes of the video tokens [B][N - n_text]; text tokens count as both.
hipError_t launch_block_flags(const uint8_t *region, int B, int n_text, int N, int bs, uint8_t *act,
                              uint8_t *ctx, hipStream_t s);

// ---- compatibility gate (host code) -------------------------------------------
// CIEDE2000 of two CIELAB colours (3 doubles each), kL = kC = kH = 1.
double ciede2000_pair(const double *lab1, const double *lab2);
// log P(X <= u) for X ~ Binomial(n, p), 0 < p < 1.
double log_binom_tail(int64_t u, int64_t n, double p);

// ---- attention -------------------------------------------------------------
// Rows order[0 .. *n_rows) when n_rows is not NULL, else all B H nB rows.
hipError_t launch_bsattn(View q, View k, View v, uint16_t *out, int64_t osb, int64_t osh,
                         int64_t osn, int B, int H, int N, int d, int bs, const int32_t *row_ptr,
                         const int32_t *col_idx, const int32_t *order, const int32_t *n_rows,
                         float scale, float *lse, hipStream_t s);

// ---- signature scan ----------------------------------------------------------
// sims: fp64 [nq][m] scratch.
hipError_t launch_sig(const float *query, int64_t nq, const float *bank, int64_t m, int64_t dim,
                      int64_t ld, int topk, int32_t *idx, float *sim, float *all_sim,
                      double *sims, hipStream_t s);
// The library-owned scratch of the no-allocation signature call (fp64
// cosines): the device address of this GPU's copy (the current device),
// looked up once per device.
constexpr size_t kSigStaticScratchBytes = (size_t)4 << 20;
hipError_t sig_static_scratch(void **ptr);

}  // namespace carnator
