// C ABI of the cache-hit block-sparse attention path (declared in
// include/carnator.h): argument checks, workspace layout and launches.
// Every check runs before the first HIP call, so a rejected call enqueues
// nothing and writes nothing.
#include "carnator.h"
#include "internal.h"

#include <math.h>
#include <stdarg.h>
#include <stdio.h>

using namespace carnator;

namespace {

thread_local char g_err[512] = "";

int fail(int code, const char *fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof g_err, fmt, ap);
  va_end(ap);
  return code;
}

int ok() {
  g_err[0] = '\0';
  return CARNATOR_OK;
}

int hip_fail(hipError_t e, const char *what) {
  return fail(CARNATOR_E_HIP, "%s: %s", what, hipGetErrorString(e));
}

constexpr int kMaxBlocks = 2048;  // nB limit of the selection kernel
// region transform: distances are bytes (radius sum < 255) and a frame's
// evidence and row distances sit in LDS (2 bytes per token)
constexpr int kMaxRegionRadius = 250;
constexpr size_t kMaxRegionFrameLds = 128 * 1024;

int check_shape(const carnator_shape *s) {
  if (!s) return fail(CARNATOR_E_NULL, "shape is NULL");
  if (s->batch < 1 || s->heads < 1 || s->seq_len < 1)
    return fail(CARNATOR_E_SHAPE, "batch, heads and seq_len must be >= 1 (got %d, %d, %d)",
                s->batch, s->heads, s->seq_len);
  if (s->head_dim != 64 && s->head_dim != 128)
    return fail(CARNATOR_E_UNSUPPORTED, "head_dim must be 64 or 128 (got %d)", s->head_dim);
  if (s->block != 64 && s->block != 128)
    return fail(CARNATOR_E_UNSUPPORTED, "block must be 64 or 128 (got %d)", s->block);
  const int64_t nB = ((int64_t)s->seq_len + s->block - 1) / s->block;
  if (nB > kMaxBlocks)
    return fail(CARNATOR_E_UNSUPPORTED, "seq_len/block gives %lld blocks; at most %d supported",
                (long long)nB, kMaxBlocks);
  if ((int64_t)s->batch * s->heads * nB * nB > (int64_t)INT32_MAX)
    return fail(CARNATOR_E_SHAPE, "batch*heads*nB*nB exceeds 2^31-1");
  return CARNATOR_OK;
}

int n_blocks(const carnator_shape *s) { return (s->seq_len + s->block - 1) / s->block; }

// Rows per head group of the row order (a valid shape).
int64_t group_rows(const carnator_shape *s) {
  return (int64_t)order_group_heads(s->batch * s->heads, s->seq_len, s->head_dim) * n_blocks(s);
}

int check_view(const carnator_view *v, const carnator_shape *s, const char *name) {
  if (!v || !v->data) return fail(CARNATOR_E_NULL, "%s is NULL", name);
  if (reinterpret_cast<uintptr_t>(v->data) % 16 != 0)
    return fail(CARNATOR_E_ALIGN, "%s data must be 16-byte aligned", name);
  if (v->stride_b % 8 || v->stride_h % 8 || v->stride_n % 8)
    return fail(CARNATOR_E_ALIGN, "%s strides must be multiples of 8 elements", name);
  if (v->stride_n < s->head_dim || v->stride_b < 0 || v->stride_h < 0)
    return fail(CARNATOR_E_SHAPE, "%s strides out of range (stride_n >= head_dim, others >= 0)", name);
  return CARNATOR_OK;
}

// Q, K and V of the attention: the kernel addresses the rows of a K or V
// tile by 32-bit byte offsets from its first row (64 rows at most).
constexpr int64_t kMaxAttnStrideN = (int64_t)1 << 24;

int check_attn_views(const carnator_view *q, const carnator_view *k, const carnator_view *v,
                     const carnator_shape *s) {
  int rc;
  if ((rc = check_view(q, s, "q")) || (rc = check_view(k, s, "k")) || (rc = check_view(v, s, "v")))
    return rc;
  if (q->stride_n > kMaxAttnStrideN || k->stride_n > kMaxAttnStrideN || v->stride_n > kMaxAttnStrideN)
    return fail(CARNATOR_E_UNSUPPORTED, "q, k and v stride_n must be at most %lld elements",
                (long long)kMaxAttnStrideN);
  return CARNATOR_OK;
}

View to_view(const carnator_view *v) {
  return View{static_cast<const uint16_t *>(v->data), v->stride_b, v->stride_h, v->stride_n};
}

int check_ws(const void *ws, size_t have, size_t need) {
  if (need > 0 && !ws) return fail(CARNATOR_E_WORKSPACE, "workspace is NULL (%zu bytes needed)", need);
  if (have < need) return fail(CARNATOR_E_WORKSPACE, "workspace has %zu bytes, %zu needed", have, need);
  if (need > 0 && reinterpret_cast<uintptr_t>(ws) % kAlign != 0)
    return fail(CARNATOR_E_ALIGN, "workspace must be %zu-byte aligned", kAlign);
  return CARNATOR_OK;
}

// Attention workspace: compacted lists and compaction scratch.
struct AttnWs {
  size_t row_ptr, col_idx, order, scratch, total;
};

AttnWs attn_layout(const carnator_shape *s) {
  const int64_t nB = n_blocks(s);
  const int64_t R = (int64_t)s->batch * s->heads * nB;
  AttnWs w;
  size_t off = 0;
  w.row_ptr = off;
  off += align_up((size_t)(R + 1) * 4);
  w.col_idx = off;
  off += align_up((size_t)(R * nB) * 4);
  w.order = off;
  off += align_up((size_t)R * 4);
  w.scratch = off;
  off += compact_scratch_bytes(R, (int)nB);
  w.total = off;
  return w;
}

}  // namespace

extern "C" {

int carnator_abi_version(void) { return CARNATOR_ABI_VERSION; }

int32_t carnator_order_group_heads(const carnator_shape *s) {
  if (!s || check_shape(s) != CARNATOR_OK) return 0;
  return order_group_heads(s->batch * s->heads, s->seq_len, s->head_dim);
}

const char *carnator_status_str(int status) {
  switch (status) {
    case CARNATOR_OK: return "ok";
    case CARNATOR_E_NULL: return "null pointer";
    case CARNATOR_E_SHAPE: return "bad shape";
    case CARNATOR_E_UNSUPPORTED: return "unsupported configuration";
    case CARNATOR_E_ALIGN: return "misaligned pointer or stride";
    case CARNATOR_E_WORKSPACE: return "workspace missing or too small";
    case CARNATOR_E_HIP: return "HIP runtime error";
    default: return "unknown status";
  }
}

const char *carnator_last_error(void) { return g_err; }

// ---------------------------------------------------------------- mask builder

// Builder workspace: pooled Q and K rows (fp64 [BH][nB][d] each).
size_t carnator_build_block_mask_workspace_size(const carnator_shape *s) {
  if (check_shape(s) != CARNATOR_OK) return 0;
  const size_t per = align_up((size_t)s->batch * s->heads * n_blocks(s) * s->head_dim * sizeof(double));
  return 2 * per;
}

// The builder behind both output forms: exactly one of mask_out and bits_out
// is non-NULL.
static int build_mask(const carnator_view *q_hist, const carnator_view *k_hist,
                      const carnator_shape *s, float scale, double mass_threshold,
                      uint8_t *mask_out, uint64_t *bits_out, void *workspace, size_t ws_bytes,
                      hipStream_t stream) {
  int rc;
  if ((rc = check_shape(s))) return rc;
  if ((rc = check_view(q_hist, s, "q_hist"))) return rc;
  if ((rc = check_view(k_hist, s, "k_hist"))) return rc;
  if (!mask_out && !bits_out) return fail(CARNATOR_E_NULL, "the output is NULL");
  if (bits_out && reinterpret_cast<uintptr_t>(bits_out) % 8 != 0)
    return fail(CARNATOR_E_ALIGN, "bits_out must be 8-byte aligned");
  if (!(mass_threshold > 0.0)) return fail(CARNATOR_E_SHAPE, "mass_threshold must be > 0");
  if (!isfinite(scale)) return fail(CARNATOR_E_SHAPE, "scale must be finite");
  const int nB = n_blocks(s);
  const int BH = s->batch * s->heads;
  if (mass_threshold >= 1.0) {
    // every block pair is kept; no workspace is touched
    hipError_t e = bits_out ? launch_fill_ones_bits(bits_out, (int64_t)BH * nB, nB, stream)
                            : launch_fill_ones(mask_out, (size_t)BH * nB * nB, stream);
    if (e != hipSuccess) return hip_fail(e, "fill");
    return ok();
  }
  const size_t need = carnator_build_block_mask_workspace_size(s);
  if ((rc = check_ws(workspace, ws_bytes, need))) return rc;
  const size_t per = need / 2;
  double *qbar = static_cast<double *>(workspace);
  double *kbar = reinterpret_cast<double *>(static_cast<char *>(workspace) + per);
  const double sigma = scale > 0.f ? (double)scale : 1.0 / sqrt((double)s->head_dim);
  hipError_t e = launch_pool(to_view(q_hist), to_view(k_hist), s->batch, s->heads, s->seq_len,
                             s->head_dim, s->block, qbar, kbar, stream);
  if (e != hipSuccess) return hip_fail(e, "pool");
  e = launch_select(qbar, kbar, BH, nB, s->head_dim, sigma, mass_threshold, mask_out, bits_out,
                    stream);
  if (e != hipSuccess) return hip_fail(e, "select");
  return ok();
}

int carnator_build_block_mask(const carnator_view *q_hist, const carnator_view *k_hist,
                              const carnator_shape *s, float scale, double mass_threshold,
                              uint8_t *mask_out, void *workspace, size_t ws_bytes,
                              hipStream_t stream) {
  if (!mask_out) return fail(CARNATOR_E_NULL, "mask_out is NULL");
  return build_mask(q_hist, k_hist, s, scale, mass_threshold, mask_out, nullptr, workspace,
                    ws_bytes, stream);
}

int carnator_build_block_mask_bits(const carnator_view *q_hist, const carnator_view *k_hist,
                                   const carnator_shape *s, float scale, double mass_threshold,
                                   uint64_t *bits_out, void *workspace, size_t ws_bytes,
                                   hipStream_t stream) {
  if (!bits_out) return fail(CARNATOR_E_NULL, "bits_out is NULL");
  return build_mask(q_hist, k_hist, s, scale, mass_threshold, nullptr, bits_out, workspace,
                    ws_bytes, stream);
}

// ---------------------------------------------------------------- exact block mass

size_t carnator_block_mass_exact_workspace_size(const carnator_shape *s) {
  if (check_shape(s) != CARNATOR_OK) return 0;
  return mass_scratch_bytes(s->batch * s->heads, s->seq_len, n_blocks(s));
}

int carnator_block_mass_exact(const carnator_view *q_hist, const carnator_view *k_hist,
                              const carnator_shape *s, float scale, double *mass, void *workspace,
                              size_t ws_bytes, hipStream_t stream) {
  int rc;
  if ((rc = check_shape(s))) return rc;
  if ((rc = check_view(q_hist, s, "q_hist"))) return rc;
  if ((rc = check_view(k_hist, s, "k_hist"))) return rc;
  if (!mass) return fail(CARNATOR_E_NULL, "mass is NULL");
  if (reinterpret_cast<uintptr_t>(mass) % 8 != 0)
    return fail(CARNATOR_E_ALIGN, "mass must be 8-byte aligned");
  if (!isfinite(scale)) return fail(CARNATOR_E_SHAPE, "scale must be finite");
  if ((rc = check_ws(workspace, ws_bytes, carnator_block_mass_exact_workspace_size(s)))) return rc;
  const float sc = scale > 0.f ? scale : (float)(1.0 / sqrt((double)s->head_dim));
  hipError_t e = launch_mass(to_view(q_hist), to_view(k_hist), s->batch, s->heads, s->seq_len,
                             s->head_dim, s->block, sc, mass, workspace, stream);
  if (e != hipSuccess) return hip_fail(e, "mass");
  return ok();
}

int carnator_select_block_mask(const double *mass, const carnator_shape *s, double mass_threshold,
                               uint8_t *mask_out, uint64_t *bits_out, hipStream_t stream) {
  int rc;
  if ((rc = check_shape(s))) return rc;
  if (!mass) return fail(CARNATOR_E_NULL, "mass is NULL");
  if ((mask_out == nullptr) == (bits_out == nullptr))
    return fail(CARNATOR_E_NULL, "exactly one of mask_out and bits_out must be non-NULL");
  if (reinterpret_cast<uintptr_t>(mass) % 8 != 0 ||
      (bits_out && reinterpret_cast<uintptr_t>(bits_out) % 8 != 0))
    return fail(CARNATOR_E_ALIGN, "mass and bits_out must be 8-byte aligned");
  if (!(mass_threshold > 0.0)) return fail(CARNATOR_E_SHAPE, "mass_threshold must be > 0");
  const int nB = n_blocks(s);
  const int BH = s->batch * s->heads;
  hipError_t e;
  if (mass_threshold >= 1.0)
    e = bits_out ? launch_fill_ones_bits(bits_out, (int64_t)BH * nB, nB, stream)
                 : launch_fill_ones(mask_out, (size_t)BH * nB * nB, stream);
  else
    e = launch_select_mass(mass, BH, nB, mass_threshold, mask_out, bits_out, stream);
  if (e != hipSuccess) return hip_fail(e, "select_mass");
  return ok();
}

// ---------------------------------------------------------------- merge

int carnator_merge_target_rows(uint8_t *mask, const carnator_shape *s, const uint8_t *target_rows,
                               const uint8_t *dense_cols, hipStream_t stream) {
  int rc;
  if ((rc = check_shape(s))) return rc;
  if (!mask) return fail(CARNATOR_E_NULL, "mask is NULL");
  if (!target_rows) return fail(CARNATOR_E_NULL, "target_rows is NULL");
  hipError_t e = launch_merge(mask, s->batch, s->heads, n_blocks(s), target_rows, dense_cols, stream);
  if (e != hipSuccess) return hip_fail(e, "merge");
  return ok();
}

// ---------------------------------------------------------------- compaction

size_t carnator_compact_block_mask_workspace_size(const carnator_shape *s) {
  if (check_shape(s) != CARNATOR_OK) return 0;
  return compact_scratch_bytes((int64_t)s->batch * s->heads * n_blocks(s), n_blocks(s));
}

int carnator_compact_block_mask(const uint8_t *mask, const carnator_shape *s, int32_t *row_ptr,
                                int32_t *col_idx, int32_t *order, void *workspace,
                                size_t ws_bytes, hipStream_t stream) {
  int rc;
  if ((rc = check_shape(s))) return rc;
  if (!mask || !row_ptr || !col_idx || !order)
    return fail(CARNATOR_E_NULL, "mask, row_ptr, col_idx and order must be non-NULL");
  if ((rc = check_ws(workspace, ws_bytes, carnator_compact_block_mask_workspace_size(s)))) return rc;
  const int nB = n_blocks(s);
  hipError_t e = launch_compact(mask, (int64_t)s->batch * s->heads * nB, nB, group_rows(s), row_ptr, col_idx,
                                order, workspace, stream);
  if (e != hipSuccess) return hip_fail(e, "compact");
  return ok();
}

// ---------------------------------------------------------------- bit-packed masks

int carnator_pack_block_mask(const uint8_t *mask, const carnator_shape *s, uint64_t *bits,
                             hipStream_t stream) {
  int rc;
  if ((rc = check_shape(s))) return rc;
  if (!mask || !bits) return fail(CARNATOR_E_NULL, "mask and bits must be non-NULL");
  if (reinterpret_cast<uintptr_t>(bits) % 8 != 0)
    return fail(CARNATOR_E_ALIGN, "bits must be 8-byte aligned");
  const int nB = n_blocks(s);
  hipError_t e = launch_pack(mask, (int64_t)s->batch * s->heads * nB, nB, bits, stream);
  if (e != hipSuccess) return hip_fail(e, "pack");
  return ok();
}

int carnator_unpack_block_mask(const uint64_t *bits, const carnator_shape *s, uint8_t *mask,
                               hipStream_t stream) {
  int rc;
  if ((rc = check_shape(s))) return rc;
  if (!mask || !bits) return fail(CARNATOR_E_NULL, "bits and mask must be non-NULL");
  if (reinterpret_cast<uintptr_t>(bits) % 8 != 0)
    return fail(CARNATOR_E_ALIGN, "bits must be 8-byte aligned");
  const int nB = n_blocks(s);
  hipError_t e = launch_unpack(bits, (int64_t)s->batch * s->heads * nB, nB, mask, stream);
  if (e != hipSuccess) return hip_fail(e, "unpack");
  return ok();
}

size_t carnator_compact_block_mask_bits_workspace_size(const carnator_shape *s) {
  if (check_shape(s) != CARNATOR_OK) return 0;
  return compact_bits_scratch_bytes((int64_t)s->batch * s->heads * n_blocks(s), s->batch,
                                    n_blocks(s));
}

int carnator_compact_block_mask_bits(const uint64_t *bits, const carnator_shape *s,
                                     const uint8_t *target_rows, const uint8_t *dense_cols,
                                     int32_t *row_ptr, int32_t *col_idx, int32_t *order,
                                     void *workspace, size_t ws_bytes, hipStream_t stream) {
  int rc;
  if ((rc = check_shape(s))) return rc;
  if (!bits || !row_ptr || !col_idx || !order)
    return fail(CARNATOR_E_NULL, "bits, row_ptr, col_idx and order must be non-NULL");
  if (reinterpret_cast<uintptr_t>(bits) % 8 != 0)
    return fail(CARNATOR_E_ALIGN, "bits must be 8-byte aligned");
  if ((rc = check_ws(workspace, ws_bytes, carnator_compact_block_mask_bits_workspace_size(s))))
    return rc;
  hipError_t e = launch_compact_bits(bits, s->batch, s->heads, n_blocks(s), group_rows(s), target_rows,
                                     dense_cols, false, row_ptr, col_idx, order, nullptr, workspace,
                                     stream);
  if (e != hipSuccess) return hip_fail(e, "compact_bits");
  return ok();
}

// ---------------------------------------------------------------- region-restricted reuse

size_t carnator_region_weights_workspace_size(int32_t batch, int32_t frames, int32_t height,
                                              int32_t width) {
  if (batch < 1 || frames < 1 || height < 1 || width < 1) return 0;
  return region_scratch_bytes(batch, frames, height, width);
}

int carnator_region_weights(const uint8_t *evidence, int32_t batch, int32_t frames, int32_t height,
                            int32_t width, int32_t r_active, int32_t r_context, uint8_t *region,
                            float *weight, void *workspace, size_t ws_bytes, hipStream_t stream) {
  int rc;
  if (!evidence || !region || !weight)
    return fail(CARNATOR_E_NULL, "evidence, region and weight must be non-NULL");
  if (batch < 1 || frames < 1 || height < 1 || width < 1)
    return fail(CARNATOR_E_SHAPE, "batch, frames, height and width must be >= 1");
  if ((int64_t)batch * frames * height * width > (int64_t)INT32_MAX)
    return fail(CARNATOR_E_SHAPE, "batch*frames*height*width exceeds 2^31-1");
  if (r_active < 0 || r_context < 0 || r_active + r_context > kMaxRegionRadius)
    return fail(CARNATOR_E_SHAPE, "radii must be >= 0 with r_active + r_context <= %d",
                kMaxRegionRadius);
  if (region_frame_lds(height, width) > kMaxRegionFrameLds)
    return fail(CARNATOR_E_UNSUPPORTED, "a frame of %d x %d tokens exceeds %d tokens", height, width,
                (int)(kMaxRegionFrameLds / 2));
  if ((rc = check_ws(workspace, ws_bytes,
                     carnator_region_weights_workspace_size(batch, frames, height, width))))
    return rc;
  if (reinterpret_cast<uintptr_t>(weight) % 4 != 0)
    return fail(CARNATOR_E_ALIGN, "weight must be 4-byte aligned");
  hipError_t e = launch_regions(evidence, batch, frames, height, width, r_active, r_context, region,
                                weight, workspace, stream);
  if (e != hipSuccess) return hip_fail(e, "regions");
  return ok();
}

int carnator_latent_fusion(const float *z_target, const float *z_hist, const float *weight,
                           float *z_out, int32_t batch, int32_t channels, int32_t frames,
                           int32_t height, int32_t width, int32_t patch_t, int32_t patch_h,
                           int32_t patch_w, hipStream_t stream) {
  if (!z_target || !z_hist || !weight || !z_out)
    return fail(CARNATOR_E_NULL, "z_target, z_hist, weight and z_out must be non-NULL");
  if (batch < 1 || channels < 1 || frames < 1 || height < 1 || width < 1)
    return fail(CARNATOR_E_SHAPE, "batch, channels, frames, height and width must be >= 1");
  if (patch_t < 1 || patch_h < 1 || patch_w < 1 || frames % patch_t || height % patch_h ||
      width % patch_w)
    return fail(CARNATOR_E_SHAPE, "patch sizes must be >= 1 and divide frames, height and width");
  if ((reinterpret_cast<uintptr_t>(z_target) | reinterpret_cast<uintptr_t>(z_hist) |
       reinterpret_cast<uintptr_t>(z_out) | reinterpret_cast<uintptr_t>(weight)) % 4)
    return fail(CARNATOR_E_ALIGN, "latents and weight must be 4-byte aligned");
  hipError_t e = launch_fusion(z_target, z_hist, weight, z_out, batch, channels, frames, height,
                               width, patch_t, patch_h, patch_w, stream);
  if (e != hipSuccess) return hip_fail(e, "fusion");
  return ok();
}

int carnator_region_block_flags(const uint8_t *region, int32_t n_text, const carnator_shape *s,
                                uint8_t *active_q, uint8_t *context_k, hipStream_t stream) {
  int rc;
  if ((rc = check_shape(s))) return rc;
  if (!region || !active_q || !context_k)
    return fail(CARNATOR_E_NULL, "region, active_q and context_k must be non-NULL");
  if (n_text < 0 || n_text >= s->seq_len)
    return fail(CARNATOR_E_SHAPE, "n_text must be in [0, seq_len) (got %d)", n_text);
  hipError_t e = launch_block_flags(region, s->batch, n_text, s->seq_len, s->block, active_q,
                                    context_k, stream);
  if (e != hipSuccess) return hip_fail(e, "block_flags");
  return ok();
}

int carnator_compact_block_mask_bits_region(const uint64_t *bits, const carnator_shape *s,
                                            const uint8_t *active_q, const uint8_t *context_k,
                                            int32_t *row_ptr, int32_t *col_idx, int32_t *order,
                                            int32_t *n_active, void *workspace, size_t ws_bytes,
                                            hipStream_t stream) {
  int rc;
  if ((rc = check_shape(s))) return rc;
  if (!bits || !active_q || !context_k || !row_ptr || !col_idx || !order || !n_active)
    return fail(CARNATOR_E_NULL,
                "bits, active_q, context_k, row_ptr, col_idx, order and n_active must be non-NULL");
  if (reinterpret_cast<uintptr_t>(bits) % 8 != 0)
    return fail(CARNATOR_E_ALIGN, "bits must be 8-byte aligned");
  if ((rc = check_ws(workspace, ws_bytes, carnator_compact_block_mask_bits_workspace_size(s))))
    return rc;
  hipError_t e = launch_compact_bits(bits, s->batch, s->heads, n_blocks(s), group_rows(s), active_q, context_k,
                                     true, row_ptr, col_idx, order, n_active, workspace, stream);
  if (e != hipSuccess) return hip_fail(e, "compact_bits_region");
  return ok();
}

// ---------------------------------------------------------------- attention

size_t carnator_block_sparse_attn_workspace_size(const carnator_shape *s) {
  if (check_shape(s) != CARNATOR_OK) return 0;
  return attn_layout(s).total;
}

int carnator_block_sparse_attn(const carnator_view *q, const carnator_view *k,
                               const carnator_view *v, void *out, int64_t osb, int64_t osh,
                               int64_t osn, const carnator_shape *s, const uint8_t *mask,
                               float scale, float *lse, void *workspace, size_t ws_bytes,
                               hipStream_t stream) {
  int rc;
  if ((rc = check_shape(s))) return rc;
  if ((rc = check_attn_views(q, k, v, s))) return rc;
  if (!out) return fail(CARNATOR_E_NULL, "out is NULL");
  if (!mask) return fail(CARNATOR_E_NULL, "mask is NULL");
  if (reinterpret_cast<uintptr_t>(out) % 16 != 0)
    return fail(CARNATOR_E_ALIGN, "out must be 16-byte aligned");
  if (osb % 8 || osh % 8 || osn % 8) return fail(CARNATOR_E_ALIGN, "out strides must be multiples of 8");
  if (osn < s->head_dim || osb < 0 || osh < 0) return fail(CARNATOR_E_SHAPE, "out strides out of range");
  if (!isfinite(scale)) return fail(CARNATOR_E_SHAPE, "scale must be finite");
  const AttnWs L = attn_layout(s);
  if ((rc = check_ws(workspace, ws_bytes, L.total))) return rc;
  char *ws = static_cast<char *>(workspace);
  int32_t *row_ptr = reinterpret_cast<int32_t *>(ws + L.row_ptr);
  int32_t *col_idx = reinterpret_cast<int32_t *>(ws + L.col_idx);
  int32_t *order = reinterpret_cast<int32_t *>(ws + L.order);
  const int nB = n_blocks(s);
  const float sc = scale > 0.f ? scale : (float)(1.0 / sqrt((double)s->head_dim));
  hipError_t e = launch_compact(mask, (int64_t)s->batch * s->heads * nB, nB, group_rows(s), row_ptr, col_idx,
                                order, ws + L.scratch, stream);
  if (e != hipSuccess) return hip_fail(e, "compact");
  e = launch_bsattn(to_view(q), to_view(k), to_view(v), static_cast<uint16_t *>(out), osb, osh, osn,
                    s->batch, s->heads, s->seq_len, s->head_dim, s->block, row_ptr, col_idx, order,
                    nullptr, sc, lse, stream);
  if (e != hipSuccess) return hip_fail(e, "bsattn");
  return ok();
}

// The attention from lists behind both entry points; n_rows NULL walks all rows.
static int attn_lists(const carnator_view *q, const carnator_view *k, const carnator_view *v,
                      void *out, int64_t osb, int64_t osh, int64_t osn, const carnator_shape *s,
                      const int32_t *row_ptr, const int32_t *col_idx, const int32_t *order,
                      const int32_t *n_rows, float scale, float *lse, hipStream_t stream) {
  int rc;
  if ((rc = check_shape(s))) return rc;
  if ((rc = check_attn_views(q, k, v, s))) return rc;
  if (!out) return fail(CARNATOR_E_NULL, "out is NULL");
  if (!row_ptr || !col_idx || !order) return fail(CARNATOR_E_NULL, "row_ptr, col_idx and order must be non-NULL");
  if (reinterpret_cast<uintptr_t>(out) % 16 != 0)
    return fail(CARNATOR_E_ALIGN, "out must be 16-byte aligned");
  if (osb % 8 || osh % 8 || osn % 8) return fail(CARNATOR_E_ALIGN, "out strides must be multiples of 8");
  if (osn < s->head_dim || osb < 0 || osh < 0) return fail(CARNATOR_E_SHAPE, "out strides out of range");
  if (!isfinite(scale)) return fail(CARNATOR_E_SHAPE, "scale must be finite");
  const float sc = scale > 0.f ? scale : (float)(1.0 / sqrt((double)s->head_dim));
  hipError_t e = launch_bsattn(to_view(q), to_view(k), to_view(v), static_cast<uint16_t *>(out), osb, osh,
                               osn, s->batch, s->heads, s->seq_len, s->head_dim, s->block, row_ptr,
                               col_idx, order, n_rows, sc, lse, stream);
  if (e != hipSuccess) return hip_fail(e, "bsattn");
  return ok();
}

int carnator_block_sparse_attn_lists(const carnator_view *q, const carnator_view *k,
                                     const carnator_view *v, void *out, int64_t osb, int64_t osh,
                                     int64_t osn, const carnator_shape *s, const int32_t *row_ptr,
                                     const int32_t *col_idx, const int32_t *order, float scale,
                                     float *lse, hipStream_t stream) {
  return attn_lists(q, k, v, out, osb, osh, osn, s, row_ptr, col_idx, order, nullptr, scale, lse,
                    stream);
}

int carnator_block_sparse_attn_rows(const carnator_view *q, const carnator_view *k,
                                    const carnator_view *v, void *out, int64_t osb, int64_t osh,
                                    int64_t osn, const carnator_shape *s, const int32_t *row_ptr,
                                    const int32_t *col_idx, const int32_t *order,
                                    const int32_t *n_rows, float scale, float *lse,
                                    hipStream_t stream) {
  if (!n_rows) return fail(CARNATOR_E_NULL, "n_rows is NULL");
  return attn_lists(q, k, v, out, osb, osh, osn, s, row_ptr, col_idx, order, n_rows, scale, lse,
                    stream);
}

// ---------------------------------------------------------------- signature scan

// Signature workspace: the fp64 cosines [nq][m].
size_t carnator_signature_sim_workspace_size(int64_t nq, int64_t m, int32_t topk) {
  (void)topk;
  if (nq < 1 || m < 1) return 0;
  return align_up((size_t)nq * m * 8);
}

static int check_signature(const float *query, int64_t nq, const float *bank, int64_t m,
                           int64_t dim, int64_t ld, int32_t topk, const int32_t *idx_out,
                           const float *sim_out) {
  if (!query || !bank || !idx_out || !sim_out)
    return fail(CARNATOR_E_NULL, "query, bank, idx_out and sim_out must be non-NULL");
  if (nq < 1 || m < 1 || dim < 1 || ld < dim)
    return fail(CARNATOR_E_SHAPE, "need nq, m, dim >= 1 and ld >= dim");
  if (m > INT32_MAX) return fail(CARNATOR_E_SHAPE, "m must fit in int32");
  if (topk < 1 || topk > m) return fail(CARNATOR_E_SHAPE, "topk must be in [1, m]");
  if (topk > 64) return fail(CARNATOR_E_UNSUPPORTED, "topk must be <= 64");
  if (dim % 4 || ld % 4 || reinterpret_cast<uintptr_t>(query) % 16 || reinterpret_cast<uintptr_t>(bank) % 16)
    return fail(CARNATOR_E_ALIGN, "dim and ld must be multiples of 4 and query/bank 16-byte aligned");
  return CARNATOR_OK;
}

int carnator_signature_sim(const float *query, int64_t nq, const float *bank, int64_t m,
                           int64_t dim, int64_t ld, int32_t topk, int32_t *idx_out,
                           float *sim_out, float *all_sim_out, void *workspace, size_t ws_bytes,
                           hipStream_t stream) {
  int rc;
  if ((rc = check_signature(query, nq, bank, m, dim, ld, topk, idx_out, sim_out))) return rc;
  const size_t need = carnator_signature_sim_workspace_size(nq, m, topk);
  if ((rc = check_ws(workspace, ws_bytes, need))) return rc;
  double *sims = static_cast<double *>(workspace);
  hipError_t e = launch_sig(query, nq, bank, m, dim, ld, topk, idx_out, sim_out, all_sim_out, sims,
                            stream);
  if (e != hipSuccess) return hip_fail(e, "signature_sim");
  return ok();
}

// The same call on the library's own scratch: no workspace argument and no
// allocation of any kind.
int carnator_signature_sim_noalloc(const float *query, int64_t nq, const float *bank, int64_t m,
                                   int64_t dim, int64_t ld, int32_t topk, int32_t *idx_out,
                                   float *sim_out, float *all_sim_out, hipStream_t stream) {
  int rc;
  if ((rc = check_signature(query, nq, bank, m, dim, ld, topk, idx_out, sim_out))) return rc;
  const size_t need = carnator_signature_sim_workspace_size(nq, m, topk);
  if (need > kSigStaticScratchBytes)
    return fail(CARNATOR_E_WORKSPACE,
                "nq * m = %lld cosines need %zu bytes of scratch; the no-allocation call holds %zu "
                "(nq * m <= %zu)",
                (long long)(nq * m), need, kSigStaticScratchBytes,
                kSigStaticScratchBytes / sizeof(double));
  void *base = nullptr;
  hipError_t e = sig_static_scratch(&base);
  if (e != hipSuccess) return hip_fail(e, "signature_sim_noalloc: scratch address");
  e = launch_sig(query, nq, bank, m, dim, ld, topk, idx_out, sim_out, all_sim_out,
                 static_cast<double *>(base), stream);
  if (e != hipSuccess) return hip_fail(e, "signature_sim_noalloc");
  return ok();
}

}  // extern "C"

// ---------------------------------------------------------------- compatibility gate (host)

int carnator_ciede2000(const double *lab1, const double *lab2, int64_t n, double *out) {
  if (!lab1 || !lab2 || !out) return fail(CARNATOR_E_NULL, "lab1, lab2 and out must be non-NULL");
  if (n < 0) return fail(CARNATOR_E_SHAPE, "n must be >= 0");
  for (int64_t i = 0; i < n; ++i) out[i] = ciede2000_pair(lab1 + 3 * i, lab2 + 3 * i);
  return ok();
}

int carnator_shape_descriptor(const uint8_t *mask, int32_t height, int32_t width, int32_t res,
                              double *area, uint8_t *shape) {
  if (!mask || !area || !shape) return fail(CARNATOR_E_NULL, "mask, area and shape must be non-NULL");
  if (height < 1 || width < 1 || res < 1) return fail(CARNATOR_E_SHAPE, "height, width and res must be >= 1");
  int y0 = height, y1 = -1, x0 = width, x1 = -1;
  int64_t cnt = 0;
  for (int y = 0; y < height; ++y)
    for (int x = 0; x < width; ++x)
      if (mask[(int64_t)y * width + x]) {
        ++cnt;
        y0 = y < y0 ? y : y0, y1 = y > y1 ? y : y1;
        x0 = x < x0 ? x : x0, x1 = x > x1 ? x : x1;
      }
  *area = (double)cnt / ((double)height * width);
  for (int64_t i = 0; i < (int64_t)res * res; ++i) shape[i] = 0;
  if (cnt == 0) return ok();
  const int h = y1 - y0 + 1, w = x1 - x0 + 1;
  for (int y = 0; y < res; ++y) {
    // floor((y + 0.5) h / res) = (2 y + 1) h / (2 res) in integers
    const int sy = (int)(((int64_t)(2 * y + 1) * h) / (2 * (int64_t)res));
    for (int x = 0; x < res; ++x) {
      const int sx = (int)(((int64_t)(2 * x + 1) * w) / (2 * (int64_t)res));
      shape[(int64_t)y * res + x] = mask[(int64_t)(y0 + sy) * width + (x0 + sx)] ? 1 : 0;
    }
  }
  return ok();
}

int carnator_object_discrepancy(double area_q, double area_j, const uint8_t *shape_q,
                                const uint8_t *shape_j, int32_t res, const double *lab_q,
                                const double *lab_j, double *d) {
  if (!shape_q || !shape_j || !lab_q || !lab_j || !d)
    return fail(CARNATOR_E_NULL, "shapes, colours and d must be non-NULL");
  if (res < 1 || !(area_q >= 0.0) || !(area_j >= 0.0))
    return fail(CARNATOR_E_SHAPE, "res must be >= 1 and the areas >= 0");
  if (area_q == 0.0 && area_j == 0.0) d[0] = 0.0;
  else if (area_q == 0.0 || area_j == 0.0) d[0] = INFINITY;
  else d[0] = fabs(log(area_q / area_j));
  int64_t inter = 0, tot = 0;
  for (int64_t i = 0; i < (int64_t)res * res; ++i) {
    const bool a = shape_q[i] != 0, b = shape_j[i] != 0;
    inter += a && b;
    tot += (int)a + (int)b;
  }
  d[1] = tot == 0 ? 0.0 : 1.0 - 2.0 * (double)inter / (double)tot;
  d[2] = ciede2000_pair(lab_q, lab_j);
  return ok();
}

int carnator_compat_gate(const double *d, int64_t n_candidates, int32_t n_terms, const double *tau,
                         int32_t *chosen) {
  if (!d || !tau || !chosen) return fail(CARNATOR_E_NULL, "d, tau and chosen must be non-NULL");
  if (n_candidates < 0 || n_terms < 1) return fail(CARNATOR_E_SHAPE, "bad candidate or term count");
  *chosen = -1;
  for (int64_t c = 0; c < n_candidates; ++c) {
    bool pass = true;
    for (int k = 0; k < n_terms; ++k) pass = pass && d[c * n_terms + k] <= tau[k];
    if (pass) {
      *chosen = (int32_t)c;
      break;
    }
  }
  return ok();
}

int carnator_clopper_pearson_upper(int64_t u, int64_t n, double alpha, double *upper) {
  if (!upper) return fail(CARNATOR_E_NULL, "upper is NULL");
  if (n < 1 || u < 0 || u > n) return fail(CARNATOR_E_SHAPE, "need 0 <= u <= n and n >= 1");
  if (!(alpha > 0.0 && alpha < 1.0)) return fail(CARNATOR_E_SHAPE, "alpha must lie in (0, 1)");
  if (u == n) {
    *upper = 1.0;
    return ok();
  }
  const double la = log(alpha);
  double lo = 0.0, hi = 1.0;
  for (int it = 0; it < 200 && hi - lo > 0.0; ++it) {
    const double mid = 0.5 * (lo + hi);
    if (mid <= lo || mid >= hi) break;
    if (log_binom_tail(u, n, mid) > la) lo = mid;  // tail still above alpha: p larger
    else hi = mid;
  }
  *upper = 0.5 * (lo + hi);
  return ok();
}
