/*
 * carnator.h -- C ABI of the cache-hit block-sparse attention path on MI355X
 * (gfx950).
 *
 * The operations follow the paper "Carnator: Fast Text-to-Video Generation
 * with Generation-Native Compatibility-Guided Cross-Request Reuse":
 *
 *   carnator_build_block_mask   historical block connectivity (Appendix C.3)
 *   carnator_block_mass_exact, carnator_select_block_mask
 *                               the builder on the exact token-level
 *                               attention mass of each block pair
 *                               (Appendix C.3, "source attention mass")
 *   carnator_merge_target_rows  target-specific query blocks widened to full
 *                               rows (Sec. 3.3, joint reuse in the middle
 *                               layers)
 *   carnator_compact_block_mask per-row lists of kept key blocks
 *   carnator_*_bits, carnator_pack_block_mask, carnator_unpack_block_mask
 *                               the same masks bit-packed, the form in which
 *                               the historical connectivity is stored and
 *                               reused (Sec. 3.3, Appendix C.3)
 *   carnator_block_sparse_attn  attention of the recomputed target Q, K, V
 *                               under the reused structure (Sec. 3.3,
 *                               historical sparse-connectivity reuse)
 *   carnator_region_weights, carnator_latent_fusion,
 *   carnator_region_block_flags, carnator_compact_block_mask_bits_region,
 *   carnator_block_sparse_attn_rows
 *                               region-restricted reuse in the middle layers
 *                               (Sec. 3.3, region-guided latent reuse and
 *                               joint reuse in intermediate layers; Appendix
 *                               C.3)
 *   carnator_ciede2000, carnator_shape_descriptor,
 *   carnator_object_discrepancy, carnator_compat_gate,
 *   carnator_clopper_pearson_upper
 *                               the compatibility gate of a recalled cache
 *                               and its certification (Sec. 3.2, Appendix
 *                               F); host code
 *   carnator_signature_sim      cosine scoring of an early-step signature
 *                               against a bank of cached signatures (Sec. 3.1,
 *                               Sec. 4.1 candidate recall)
 *
 * Conventions shared by every call
 * --------------------------------
 * - Pointers named in the argument lists are DEVICE pointers unless a comment
 *   says "host".  Descriptor structs (carnator_shape, carnator_view) are read
 *   on the host during the call and not retained.
 * - Every call that takes a stream only enqueues work on it and returns; the
 *   results are ready when the stream is synchronised.  stream may be NULL
 *   (the default stream).
 * - Ownership: the caller owns every buffer, the workspace and the stream.
 *   The library allocates no device memory, keeps no pointer after it returns
 *   and holds no global mutable state apart from a thread-local error string
 *   and, for carnator_signature_sim_noalloc only, a static device scratch
 *   array and its address on each device.  Calls that run concurrently need
 *   separate workspaces.
 * - Errors: each call returns a carnator_status.  On a non-OK status nothing
 *   has been enqueued and no output has been written.  All argument checks
 *   happen before the first HIP call.  A failed launch returns
 *   CARNATOR_E_HIP; faults inside a kernel surface at the caller's next
 *   synchronisation.  carnator_last_error() gives a text detail for the
 *   calling thread.
 * - Token layout: Q, K, V and O are bf16 [B, H, N, d] with d contiguous and
 *   arbitrary element strides for B, H and N (stride_n a multiple of 8,
 *   data 16-byte aligned).  The attention calls also need stride_n of Q, K
 *   and V at most 2^24 elements (a tile's rows are addressed by 32-bit byte
 *   offsets from the tile's first row); larger gives
 *   CARNATOR_E_UNSUPPORTED.  Blocks are runs of `block` consecutive tokens;
 *   block j covers tokens [j*block, min((j+1)*block, N)), so only the last
 *   block can be partial.  nB = ceil(N / block).  Tokens past N are never
 *   read or written.
 * - Block masks are uint8 [B, H, nB, nB], contiguous; 0 drops a block pair,
 *   any other byte keeps it.  The builder writes exactly 0 or 1.
 * - Bit-packed block masks are uint64 [B, H, nB, W], W = ceil(nB / 64),
 *   contiguous, 8-byte aligned: key block j of row (b, h, i) is bit j mod 64
 *   (least significant first) of word j / 64 of that row.  Bits j >= nB of
 *   a row's last word are written as 0 and ignored when read.  A bank of
 *   masks over S denoising steps, C branches and L layers is one array
 *   [S, C, L, B, H, nB, W]; each slot is a mask of this layout.
 * - Supported: head_dim in {64, 128}, block in {64, 128}.  Anything else
 *   returns CARNATOR_E_UNSUPPORTED.
 */
#ifndef CARNATOR_H
#define CARNATOR_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define CARNATOR_ABI_VERSION 7

typedef enum {
  CARNATOR_OK = 0,
  CARNATOR_E_NULL = -1,        /* a required pointer is NULL */
  CARNATOR_E_SHAPE = -2,       /* a size or stride is out of range */
  CARNATOR_E_UNSUPPORTED = -3, /* head_dim / block / topk not supported */
  CARNATOR_E_ALIGN = -4,       /* pointer or stride misaligned */
  CARNATOR_E_WORKSPACE = -5,   /* workspace NULL or smaller than required */
  CARNATOR_E_HIP = -6          /* a HIP launch or runtime call failed */
} carnator_status;

/* Problem shape.  seq_len is the number of valid tokens N. */
typedef struct {
  int32_t batch;
  int32_t heads;
  int32_t seq_len;
  int32_t head_dim; /* 64 or 128 */
  int32_t block;    /* 64 or 128 */
} carnator_shape;

/* A bf16 [B, H, N, d] tensor: element strides, d contiguous. */
typedef struct {
  const void *data;
  int64_t stride_b;
  int64_t stride_h;
  int64_t stride_n;
} carnator_view;

/* ABI version of the loaded library (CARNATOR_ABI_VERSION). */
int carnator_abi_version(void);

/*
 * Row order of the compaction entry points (the order in which the attention
 * kernel runs the rows; an execution schedule the paper leaves open).  The
 * B*H heads are cut into consecutive groups of G heads, G the most heads
 * whose K and V (2 * seq_len * head_dim bf16 values per head) fit in 256 MiB,
 * the size of MI355X's Infinity Cache (at least 1 head, and at least
 * B*H / 63 heads so that there are at most 63 groups; all heads when they
 * fit).  The order lists group 0's rows by descending list length (lower row
 * first on equal length), then group 1's, and so on; a restricting call then
 * lists the rows it leaves out, in ascending order.  With one group this is
 * the plain longest-first order.  Running one group of heads at a time keeps
 * their K and V in the Infinity Cache while they are streamed.
 * carnator_order_group_heads returns G for a shape (0 if the shape is
 * invalid).
 */
int32_t carnator_order_group_heads(const carnator_shape *shape);

/* Static text of a status code (host). */
const char *carnator_status_str(int status);

/* Detail of the last failure on the calling thread (host); "" if none. */
const char *carnator_last_error(void);

/*
 * Historical block connectivity -- Appendix C.3 ("Reuse-Scope
 * Implementation Details"): for each head and query block, keep the smallest
 * set of key blocks covering a fixed fraction of the attention mass.
 *
 * The mass of key block j for query block i is the softmax over j of the
 * pooled logit s_ij = sigma * <mean_i(Q_hist), mean_j(K_hist)>, means over
 * the valid tokens of each block, sigma = scale, or 1/sqrt(head_dim) when
 * scale <= 0.  Key blocks are taken in descending s (lower j first on
 * equality) until the cumulative mass reaches mass_threshold; k is that
 * count.  Blocks whose score lies within 1e-6 of the k-th score are tied and
 * the lower block indices among them fill the remaining places.
 * mass_threshold >= 1 keeps every block.  Pooling, scores, softmax and
 * selection are computed in fp64.
 *
 *   q_hist, k_hist  bf16 views of the historical copy [B, H, N, d]
 *   mask_out        uint8 [B, H, nB, nB], written with 0/1
 *   workspace       device scratch of at least
 *                   carnator_build_block_mask_workspace_size(shape) bytes,
 *                   256-byte aligned
 * Errors: E_NULL, E_SHAPE (any size < 1, mass_threshold <= 0 or NaN),
 * E_UNSUPPORTED, E_ALIGN, E_WORKSPACE, E_HIP.
 */
size_t carnator_build_block_mask_workspace_size(const carnator_shape *shape);
int carnator_build_block_mask(const carnator_view *q_hist, const carnator_view *k_hist,
                              const carnator_shape *shape, float scale, double mass_threshold,
                              uint8_t *mask_out, void *workspace, size_t workspace_bytes,
                              hipStream_t stream);

/*
 * Target-specific widening -- Sec. 3.3 ("Joint Reuse in Intermediate
 * Layers"): target-specific computation is preserved for the localized
 * region, so its query blocks evaluate every key block.
 *
 *   mask         uint8 [B, H, nB, nB], updated in place:
 *                M[b,h,i,j] = (M != 0) | row_flags[b,i] | col_flags[b,j]
 *   target_rows  uint8 [B, nB]; nonzero widens query block i to a full row
 *   dense_cols   uint8 [B, nB] or NULL; nonzero makes key block j a full
 *                column (dense text tokens)
 * The result is written as 0/1 bytes.  Errors: E_NULL, E_SHAPE, E_HIP.
 */
int carnator_merge_target_rows(uint8_t *mask, const carnator_shape *shape,
                               const uint8_t *target_rows, const uint8_t *dense_cols,
                               hipStream_t stream);

/*
 * Per-row lists of kept key blocks (the compacted list the sparse executor
 * walks; rows are (b, h, i) in row-major order, R = B*H*nB).
 *
 *   mask      uint8 [B, H, nB, nB]
 *   row_ptr   int32 [R + 1]; row r's list is col_idx[row_ptr[r] .. row_ptr[r+1])
 *   col_idx   int32 [B*H*nB*nB] capacity; ascending key blocks per row
 *   order     int32 [R]; the row order above: per group of heads (one group
 *             whenever the shape's K and V fit 256 MiB) the rows by descending
 *             list length, lower row first on equal length
 *   workspace at least carnator_compact_block_mask_workspace_size(shape) bytes
 * Errors: E_NULL, E_SHAPE, E_UNSUPPORTED, E_WORKSPACE, E_HIP.
 */
size_t carnator_compact_block_mask_workspace_size(const carnator_shape *shape);
int carnator_compact_block_mask(const uint8_t *mask, const carnator_shape *shape,
                                int32_t *row_ptr, int32_t *col_idx, int32_t *order,
                                void *workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * Exact block mass -- Appendix C.3 keeps, per head and query block, the
 * smallest set of key blocks covering a fixed fraction of the source
 * attention mass.  carnator_build_block_mask estimates that mass from block
 * means; these calls compute it from the tokens:
 *
 *   M[b,h,i,j] = (1 / n_i) sum_{a in block i, a < N} sum_{t in block j}
 *                softmax_t(sigma q_a . k_t)
 *
 * the softmax over all N keys, sigma = scale or 1/sqrt(head_dim) when
 * scale <= 0; n_i the valid queries of block i; each row sums to 1.  A dense
 * bf16 matrix-core pass (fp32 accumulation and softmax statistics), the
 * masses summed over the queries in fp64 (each query's term in fp32).
 *
 * carnator_block_mass_exact:
 *   q_hist, k_hist  bf16 views [B, H, N, d]
 *   mass            fp64 [B, H, nB, nB] out
 *   workspace       carnator_block_mass_exact_workspace_size(shape) bytes,
 *                   256-byte aligned: 8 B per (query, key block) plus 4 B
 *                   per query for each head of a chunk.  Heads are processed
 *                   in chunks whose records fit in 4 GiB (at least one head
 *                   per chunk), so the workspace is at most
 *                   max(4 GiB, one head's records): 0.81 GB at B=1, H=12,
 *                   N=32,760, block 128 (all heads in one chunk), 3.55 GB
 *                   at H=24, N=119,056 (4 heads per chunk, 6 chunks),
 *                   4.3 GB for one head at the largest N (2048 blocks of
 *                   128).  A smaller workspace gives E_WORKSPACE.
 * Errors: E_NULL, E_SHAPE, E_UNSUPPORTED, E_ALIGN, E_WORKSPACE, E_HIP.
 *
 * carnator_select_block_mask: the selection of carnator_build_block_mask
 * applied to given masses: per row, the smallest prefix of the key blocks
 * by descending mass (lower index first on equal mass) whose mass reaches
 * mass_threshold of the row total; masses within 1e-6 of the cut mass are
 * tied and the lower block indices among them are kept; mass_threshold
 * >= 1 keeps every block.
 *   mass      fp64 [B, H, nB, nB] (non-negative)
 *   mask_out  uint8 [B, H, nB, nB] or NULL; bits_out uint64 [B, H, nB, W]
 *             or NULL: exactly one of them
 * Errors: E_NULL, E_SHAPE, E_UNSUPPORTED, E_ALIGN, E_HIP.
 */
size_t carnator_block_mass_exact_workspace_size(const carnator_shape *shape);
int carnator_block_mass_exact(const carnator_view *q_hist, const carnator_view *k_hist,
                              const carnator_shape *shape, float scale, double *mass,
                              void *workspace, size_t workspace_bytes, hipStream_t stream);
int carnator_select_block_mask(const double *mass, const carnator_shape *shape,
                               double mass_threshold, uint8_t *mask_out, uint64_t *bits_out,
                               hipStream_t stream);

/*
 * Compatibility gate -- Sec. 3.2 ("Reuse Validity with Generation-Native
 * Evidence": compatibility filtering and risk-aware compatibility decisions)
 * and Appendix F.  Per object the Early Signature holds the normalised
 * support size A of its binary tail-frame mask (the mean over the H x W
 * grid), the mask and a CIELAB colour.  Against a candidate:
 *   d_size  = |ln(A_q / A_j)|  (0 if both areas are 0, +inf if one is),
 *   d_shape = 1 - 2 |S_q and S_j| / (|S_q| + |S_j|) over the masks cropped
 *             to their bounding boxes and resampled to res x res (0 if both
 *             are empty),
 *   d_color = CIEDE2000 (kL = kC = kH = 1); d_context is the largest
 *             CIEDE2000 over the objects both requests share.
 * A candidate passes when every discrepancy is within its threshold; the
 * first passing candidate in recall order is reused, else the request runs
 * dense.  A threshold setting is certified by the one-sided Clopper-Pearson
 * upper bound U_alpha(u, n) on the unsafe-reuse rate.
 *
 * All of these run on the host, on HOST pointers, and enqueue nothing.
 *
 * carnator_ciede2000: out[i] = CIEDE2000(lab1[i], lab2[i]); lab1, lab2
 *   double [n][3] (L, a, b); out double [n].
 * carnator_shape_descriptor: area = mean of mask != 0; shape uint8
 *   [res][res] = the bounding-box crop (h x w) sampled at source row
 *   floor((y + 0.5) h / res), column floor((x + 0.5) w / res); all 0 for an
 *   empty mask.  mask uint8 [height][width].
 * carnator_object_discrepancy: d double [3] = (d_size, d_shape, d_color) of
 *   one object; shapes uint8 [res][res], colours double [3].
 * carnator_compat_gate: d double [n_candidates][n_terms] in recall order,
 *   tau double [n_terms]; *chosen = the first candidate with d <= tau in
 *   every term, or -1.
 * carnator_clopper_pearson_upper: *upper = the p at which the probability of
 *   at most u failures in n Bernoulli(p) trials equals alpha (1 when u = n);
 *   0 <= u <= n, n >= 1, 0 < alpha < 1.
 * Errors: E_NULL, E_SHAPE.
 */
int carnator_ciede2000(const double *lab1, const double *lab2, int64_t n, double *out);
int carnator_shape_descriptor(const uint8_t *mask, int32_t height, int32_t width, int32_t res,
                              double *area, uint8_t *shape);
int carnator_object_discrepancy(double area_q, double area_j, const uint8_t *shape_q,
                                const uint8_t *shape_j, int32_t res, const double *lab_q,
                                const double *lab_j, double *d);
int carnator_compat_gate(const double *d, int64_t n_candidates, int32_t n_terms, const double *tau,
                         int32_t *chosen);
int carnator_clopper_pearson_upper(int64_t u, int64_t n, double alpha, double *upper);

/*
 * Bit-packed masks: the historical block connectivity in its stored form.
 * The paper keeps the sparse connectivity of the historical run per
 * denoising step, branch, layer and head and reuses it for later requests
 * (Sec. 3.3, Appendix C.3); one bit per block pair is an eighth of the
 * uint8 mask.  Layout: see "Bit-packed block masks" above.
 *
 * carnator_build_block_mask_bits: carnator_build_block_mask with the mask
 * written bit-packed (same arguments, same workspace size, the same decisions
 * bit for bit).
 *   bits_out  uint64 [B, H, nB, W]
 * Errors: E_NULL, E_SHAPE, E_UNSUPPORTED, E_ALIGN, E_WORKSPACE, E_HIP.
 *
 * carnator_pack_block_mask: bits[b,h,i] bit j = (mask[b,h,i,j] != 0).
 * carnator_unpack_block_mask: mask[b,h,i,j] = bit j of bits[b,h,i] as 0/1
 * bytes.
 *   mask  uint8 [B, H, nB, nB]; bits uint64 [B, H, nB, W]
 * Errors: E_NULL, E_SHAPE, E_UNSUPPORTED, E_ALIGN, E_HIP.
 *
 * carnator_compact_block_mask_bits: the lists carnator_compact_block_mask
 * writes for the mask carnator_merge_target_rows would make of the unpacked
 * bits (same row_ptr, col_idx and order), computed from the words directly;
 * the bits are only read, so one stored mask serves any target.
 *   bits         uint64 [B, H, nB, W]
 *   target_rows  uint8 [B, nB] or NULL; nonzero widens query block i to a
 *                full row
 *   dense_cols   uint8 [B, nB] or NULL; nonzero keeps key block j in every
 *                row
 *   row_ptr, col_idx, order: as carnator_compact_block_mask
 *   workspace    at least carnator_compact_block_mask_bits_workspace_size
 *                (shape) bytes, 256-byte aligned
 * Errors: E_NULL, E_SHAPE, E_UNSUPPORTED, E_ALIGN, E_WORKSPACE, E_HIP.
 */
int carnator_build_block_mask_bits(const carnator_view *q_hist, const carnator_view *k_hist,
                                   const carnator_shape *shape, float scale,
                                   double mass_threshold, uint64_t *bits_out, void *workspace,
                                   size_t workspace_bytes, hipStream_t stream);
int carnator_pack_block_mask(const uint8_t *mask, const carnator_shape *shape, uint64_t *bits,
                             hipStream_t stream);
int carnator_unpack_block_mask(const uint64_t *bits, const carnator_shape *shape, uint8_t *mask,
                               hipStream_t stream);
size_t carnator_compact_block_mask_bits_workspace_size(const carnator_shape *shape);
int carnator_compact_block_mask_bits(const uint64_t *bits, const carnator_shape *shape,
                                     const uint8_t *target_rows, const uint8_t *dense_cols,
                                     int32_t *row_ptr, int32_t *col_idx, int32_t *order,
                                     void *workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * Region-restricted reuse in the middle layers.
 *
 * Sec. 3.3 ("Region-Guided Latent Reuse"): the Evidence Region of the
 * accepted cache is expanded into an Active Region and a larger Context
 * Region (evidence within active within context) on the T x H x W token
 * grid; each later latent is z = W * z_target + (1 - W) * z_hist with
 * W = 1 on the evidence, W = 1 - s(d / d_max) on the transition band (active
 * minus evidence) and W = 0 outside the active region, s the smoothstep
 * 3 t^2 - 2 t^3, d the Chebyshev distance to the evidence within the token's
 * frame and d_max its largest value over the band of the batch entry.
 * Appendix C.3: active = evidence dilated by 2 tokens, context = active
 * dilated by 3 more, per latent frame on the H x W grid (dilation by the
 * (2r+1) x (2r+1) square).  Sec. 3.3 ("Joint Reuse in Intermediate Layers"):
 * in the middle layers only the historical connectivity of active queries to
 * context keys is kept; tokens outside the active region keep their cached
 * computation.
 *
 * carnator_region_weights: region codes and W from the evidence.
 *   evidence   uint8 [B, T, H, W], nonzero = evidence token
 *   r_active, r_context  dilation radii (2 and 3 in the paper);
 *              r_active + r_context <= 250
 *   region     uint8 [B, T, H, W] out: 3 evidence, 2 band, 1 context minus
 *              active, 0 outside the context region
 *   weight     fp32 [B, T, H, W] out: W
 *   workspace  carnator_region_weights_workspace_size(B, T, H, W) bytes,
 *              256-byte aligned
 *   H * W <= 65536 tokens per frame (else E_UNSUPPORTED).
 * Errors: E_NULL, E_SHAPE, E_UNSUPPORTED, E_ALIGN, E_WORKSPACE, E_HIP.
 *
 * carnator_latent_fusion: z_out = W * z_target + (1 - W) * z_hist.
 *   z_target, z_hist, z_out  fp32 [B, C, T, H, W] contiguous (latent grid);
 *              z_out may be z_target or z_hist
 *   weight     fp32 [B, T / patch_t, H / patch_h, W / patch_w] (token grid);
 *              a latent element takes the weight of the token whose patch
 *              holds it (patch sizes >= 1 dividing T, H, W)
 * Errors: E_NULL, E_SHAPE, E_ALIGN (4-byte), E_HIP.
 *
 * carnator_region_block_flags: active query blocks and context key blocks.
 *   region     uint8 [B, N - n_text]: the codes of the video tokens in the
 *              attention's (t, y, x) raster order
 *   n_text     text tokens placed before the video tokens (they carry the
 *              target prompt and count as active and as context)
 *   shape      batch, seq_len = N, block (head fields as for any call)
 *   active_q   uint8 [B, nB] out: 1 if a token of query block i is active
 *              (code >= 2 or text)
 *   context_k  uint8 [B, nB] out: 1 if a token of key block j is context
 *              (code >= 1 or text)
 * Errors: E_NULL, E_SHAPE, E_UNSUPPORTED, E_HIP.
 *
 * carnator_compact_block_mask_bits_region: the lists of the stored mask
 * restricted to active rows and context columns,
 * M'[b,h,i,j] = M[b,h,i,j] and active_q[b,i] and context_k[b,j].
 *   bits, row_ptr, col_idx: as carnator_compact_block_mask_bits
 *   order      int32 [R]: the active rows in the row order above (per
 *              group of heads, by descending list length, lower row first on
 *              equal length), then the inactive rows in ascending order
 *              (their lists are empty)
 *   n_active   int32 [1] out (device): the number of active rows
 *   workspace  carnator_compact_block_mask_bits_workspace_size(shape) bytes
 * Errors: E_NULL, E_SHAPE, E_UNSUPPORTED, E_ALIGN, E_WORKSPACE, E_HIP.
 *
 * carnator_block_sparse_attn_rows: carnator_block_sparse_attn_lists over
 * the rows order[0 .. *n_rows) only (n_rows a device int32, e.g. the
 * n_active written above); the output and LSE of every other row are left
 * untouched.  Errors: as carnator_block_sparse_attn_lists.
 */
size_t carnator_region_weights_workspace_size(int32_t batch, int32_t frames, int32_t height,
                                              int32_t width);
int carnator_region_weights(const uint8_t *evidence, int32_t batch, int32_t frames, int32_t height,
                            int32_t width, int32_t r_active, int32_t r_context, uint8_t *region,
                            float *weight, void *workspace, size_t workspace_bytes,
                            hipStream_t stream);
int carnator_latent_fusion(const float *z_target, const float *z_hist, const float *weight,
                           float *z_out, int32_t batch, int32_t channels, int32_t frames,
                           int32_t height, int32_t width, int32_t patch_t, int32_t patch_h,
                           int32_t patch_w, hipStream_t stream);
int carnator_region_block_flags(const uint8_t *region, int32_t n_text, const carnator_shape *shape,
                                uint8_t *active_q, uint8_t *context_k, hipStream_t stream);
int carnator_compact_block_mask_bits_region(const uint64_t *bits, const carnator_shape *shape,
                                            const uint8_t *active_q, const uint8_t *context_k,
                                            int32_t *row_ptr, int32_t *col_idx, int32_t *order,
                                            int32_t *n_active, void *workspace,
                                            size_t workspace_bytes, hipStream_t stream);
int carnator_block_sparse_attn_rows(const carnator_view *q, const carnator_view *k,
                                    const carnator_view *v, void *out, int64_t out_stride_b,
                                    int64_t out_stride_h, int64_t out_stride_n,
                                    const carnator_shape *shape, const int32_t *row_ptr,
                                    const int32_t *col_idx, const int32_t *order,
                                    const int32_t *n_rows, float scale, float *lse,
                                    hipStream_t stream);

/*
 * Block-sparse attention -- Sec. 3.3 ("Historical Sparse-Connectivity
 * Reuse") and Appendix C.3: the target's Q, K, V are recomputed and only the
 * block pairs kept by the reused mask are evaluated.
 *
 * For a valid query token a in block i, with A(a) the keys t < N whose block
 * is kept in row (b, h, i):
 *   o_a = sum_{t in A(a)} softmax_t(sigma * q_a . k_t) v_t,
 *   lse_a = log sum_{t in A(a)} exp(sigma * q_a . k_t),
 * sigma = scale, or 1/sqrt(head_dim) when scale <= 0.  A row with no kept
 * block gives o = 0 and lse = -inf.  bf16 matrix cores for Q.K^T and P.V,
 * fp32 accumulation and online softmax; O is rounded to bf16.
 *
 *   q, k, v        bf16 views [B, H, N, d]
 *   out            bf16 [B, H, N, d] at element strides out_stride_{b,h,n}
 *                  (d contiguous); may not alias q, k or v
 *   mask           uint8 [B, H, nB, nB]
 *   lse            fp32 [B, H, N] contiguous, or NULL
 *   workspace      at least carnator_block_sparse_attn_workspace_size(shape)
 *                  bytes, 256-byte aligned (holds the compacted lists)
 * Errors: E_NULL, E_SHAPE, E_UNSUPPORTED, E_ALIGN, E_WORKSPACE, E_HIP.
 */
size_t carnator_block_sparse_attn_workspace_size(const carnator_shape *shape);
int carnator_block_sparse_attn(const carnator_view *q, const carnator_view *k,
                               const carnator_view *v, void *out, int64_t out_stride_b,
                               int64_t out_stride_h, int64_t out_stride_n,
                               const carnator_shape *shape, const uint8_t *mask, float scale,
                               float *lse, void *workspace, size_t workspace_bytes,
                               hipStream_t stream);

/*
 * Block-sparse attention from compacted lists -- the same operation as
 * carnator_block_sparse_attn with the kept key blocks given as the lists
 * carnator_compact_block_mask writes for the mask (for callers that reuse one
 * mask for several calls, or time the attention kernel on its own).  One
 * kernel launch, no workspace.
 *
 *   q, k, v, out, out strides, shape, scale, lse: as carnator_block_sparse_attn
 *   row_ptr  int32 [R + 1], col_idx int32 (row lists, ascending), order
 *            int32 [R] (a permutation of the R = B*H*nB rows, the row order
 *            above): as written by carnator_compact_block_mask (any
 *            permutation gives the same output; the order sets the speed)
 * The kernel clamps rows, list bounds and block indices into range, so
 * malformed lists give wrong output but no access outside q, k, v, out,
 * lse and the lists' documented extents.
 * Errors: E_NULL, E_SHAPE, E_UNSUPPORTED, E_ALIGN, E_HIP.
 */
int carnator_block_sparse_attn_lists(const carnator_view *q, const carnator_view *k,
                                     const carnator_view *v, void *out, int64_t out_stride_b,
                                     int64_t out_stride_h, int64_t out_stride_n,
                                     const carnator_shape *shape, const int32_t *row_ptr,
                                     const int32_t *col_idx, const int32_t *order, float scale,
                                     float *lse, hipStream_t stream);

/*
 * Early-signature cosine scoring -- Sec. 3.1 (a target is compared against
 * a bank built from completed requests) and Sec. 4.1 ("Candidate Recall":
 * rank histories by similarity, keep the top K).
 *
 *   cos_m = <q, b_m> / (|q| |b_m|) accumulated in fp64; 0 when a norm is 0.
 *   The top-k are taken in descending cosine (lower m first on equality);
 *   among bank rows within 1e-6 of the k-th value the lower rows are kept.
 *   idx_out lists the chosen rows in descending cosine, sim_out their values.
 *
 *   query        fp32 [nq, dim] contiguous
 *   bank         fp32 [m, ld] row-major, ld >= dim
 *   idx_out      int32 [nq, topk];  sim_out fp32 [nq, topk]
 *   all_sim_out  fp32 [nq, m] or NULL (every cosine)
 *   topk         1 .. min(m, 64)
 *   workspace    at least carnator_signature_sim_workspace_size(nq, m, topk)
 *                bytes, 256-byte aligned (the fp64 cosines [nq, m])
 * Errors: E_NULL, E_SHAPE, E_UNSUPPORTED (topk > 64), E_ALIGN, E_WORKSPACE, E_HIP.
 */
size_t carnator_signature_sim_workspace_size(int64_t nq, int64_t m, int32_t topk);
int carnator_signature_sim(const float *query, int64_t nq, const float *bank, int64_t m,
                           int64_t dim, int64_t ld, int32_t topk, int32_t *idx_out,
                           float *sim_out, float *all_sim_out, void *workspace,
                           size_t workspace_bytes, hipStream_t stream);

/*
 * carnator_signature_sim without a workspace, for callers that cannot
 * allocate device memory: code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc.  Same arguments (minus the workspace),
 * same results and errors as carnator_signature_sim.
 *
 * The scratch (the fp64 cosines [nq, m]) is a library-owned device array of
 * 4 MiB, one copy per GPU the library runs on, held until the process ends;
 * its device address is looked up on the first call on each device.  The
 * call allocates nothing (no hipMalloc, no hipFree, no allocating library
 * routine).  Limit: nq * m <= 524,288 cosines (e.g. 128 queries against
 * 4,096 rows, or one query against 524,288 rows); beyond it the call returns
 * E_WORKSPACE and enqueues nothing.  Every cosine is written before it is
 * read, so nothing needs clearing between calls.  Every call on one GPU
 * shares that GPU's scratch: calls that overlap on one GPU (other streams,
 * other host threads) RACE and must be serialised by the caller.
 * Errors: E_NULL, E_SHAPE, E_UNSUPPORTED (topk > 64), E_ALIGN, E_WORKSPACE
 * (nq * m above the limit), E_HIP.
 */
int carnator_signature_sim_noalloc(const float *query, int64_t nq, const float *bank, int64_t m,
                                   int64_t dim, int64_t ld, int32_t topk, int32_t *idx_out,
                                   float *sim_out, float *all_sim_out, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* CARNATOR_H */
