// Region-restricted reuse in the middle layers.
//
// Sec. 3.3 ("Region-Guided Latent Reuse"): the Evidence Region grows into an
// Active Region and a larger Context Region over the T x H x W token grid;
// every later latent is W * (target-updated latent) + (1 - W) * (historical
// latent), with W = 1 on the evidence, 1 - smoothstep(normalised Chebyshev
// distance to the evidence) on the transition band (active minus evidence)
// and 0 outside the active region.  Appendix C.3: active = evidence dilated
// by 2 tokens, context = active dilated by 3 more, per latent frame on the
// H x W grid, the band distance normalised by its maximum over the band.
// Sec. 3.3 ("Joint Reuse in Intermediate Layers"): only the connectivity of
// active query blocks to context key blocks is kept (the lists come from
// compact_kernels.hip).
//
// Dilating by a square of radius r is thresholding the Chebyshev distance to
// the evidence at r (squares compose: radius 2 then 3 is radius 5), so one
// distance transform per frame gives all three regions and the band
// distance.  The transform is separable: the distance along the row to the
// nearest evidence token, then the minimum over the rows within reach of
// max(|dy|, row distance), capped at r_active + r_context + 1.
#include "internal.h"

namespace carnator {
namespace {

constexpr int kRegionThreads = 256;

// One workgroup of 256 threads per band of BR rows of a (b, t) frame (grid
// x the frame, y the band: at most 512 bands, any number of frames), so a
// frame's rows spread over several CUs (a frame per workgroup left most of
// the chip idle: 21 frames at 32K tokens).  The band's rows and the R =
// r_active + r_context rows on either side that its distances can reach
// (clipped at the frame border) are staged in LDS with their row distances
// (2 bytes per staged token).  Writes the region code (3 evidence, 2 band,
// 1 context, 0 outside) and the capped distance of the band's tokens, and
// the largest band distance of the band to band_max (0 when it has none).
__global__ void __launch_bounds__(kRegionThreads) region_kernel(
    const uint8_t *__restrict__ evidence, int H, int W, int BR, int nbands, int ra, int rc,
    uint8_t *__restrict__ region, uint8_t *__restrict__ dist, int32_t *__restrict__ band_max) {
  extern __shared__ uint8_t fr[];
  __shared__ int wmax[kRegionThreads / 64];
  const int frame = blockIdx.x, band = blockIdx.y;
  const int R = ra + rc, cap = R + 1;
  const int y0 = band * BR, y1 = min(H, y0 + BR);
  const int ya = max(0, y0 - R), yb = min(H, y1 + R);
  const int staged = (yb - ya) * W;
  uint8_t *ev = fr, *rowd = fr + staged;
  const int64_t base = (int64_t)frame * H * W;
  const int t = threadIdx.x;
  {
    // four loads in flight per thread before any is stored
    const uint8_t *src = evidence + base + (int64_t)ya * W;
    for (int p0 = 0; p0 < staged; p0 += 4 * kRegionThreads) {
      uint8_t v[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int p = p0 + u * kRegionThreads + t;
        v[u] = src[min(p, staged - 1)];
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int p = p0 + u * kRegionThreads + t;
        if (p < staged) ev[p] = v[u] != 0;
      }
    }
  }
  __syncthreads();
  for (int p = t; p < staged; p += kRegionThreads) {
    const int ly = p / W, x = p - ly * W;
    const uint8_t *row = ev + ly * W;
    int d = cap;
    for (int k = 0; k <= R; ++k) {
      if ((x - k >= 0 && row[x - k]) || (x + k < W && row[x + k])) {
        d = k;
        break;
      }
    }
    rowd[p] = (uint8_t)d;
  }
  __syncthreads();
  // rows y - k >= 0 and y + k < H within reach lie in [ya, yb)
  int bmax = 0;
  for (int p = t; p < (y1 - y0) * W; p += kRegionThreads) {
    const int y = y0 + p / W, x = p - (p / W) * W;
    const int q = (y - ya) * W + x;
    int d = rowd[q];
    for (int k = 1; k <= R && k < d; ++k) {
      if (y - k >= 0) d = min(d, max(k, (int)rowd[q - k * W]));
      if (y + k < H) d = min(d, max(k, (int)rowd[q + k * W]));
    }
    const uint8_t code = d == 0 ? 3 : d <= ra ? 2 : d <= R ? 1 : 0;
    region[base + (int64_t)y * W + x] = code;
    dist[base + (int64_t)y * W + x] = (uint8_t)d;
    if (code == 2) bmax = max(bmax, d);
  }
  // workgroup maximum
  for (int o = 32; o > 0; o >>= 1) bmax = max(bmax, __shfl_xor(bmax, o));
  if ((t & 63) == 0) wmax[t >> 6] = bmax;
  __syncthreads();
  if (t == 0) {
    int m = 0;
    for (int w = 0; w < kRegionThreads / 64; ++w) m = max(m, wmax[w]);
    band_max[(int64_t)frame * nbands + band] = m;
  }
}

// One thread per token: W from the region code, the distance and the band
// maximum over the bands (of every frame) of the token's batch entry.  The
// workgroup first takes that maximum for each batch entry its tokens belong
// to (usually one), all threads sharing the walk over the nper band maxima.
__global__ void __launch_bounds__(256) weight_kernel(const uint8_t *__restrict__ region,
                                                     const uint8_t *__restrict__ dist,
                                                     const int32_t *__restrict__ band_max,
                                                     int nper, int64_t per_batch, int64_t total,
                                                     float *__restrict__ weight) {
  __shared__ int wm[4];
  const int t = threadIdx.x;
  const int64_t x0 = (int64_t)blockIdx.x * 256;
  const int64_t x = x0 + t;
  const int64_t xl = (x0 + 255 < total ? x0 + 255 : total - 1);
  const int64_t b0 = x0 / per_batch, b1 = xl / per_batch;
  const int64_t myb = (x < total ? x : xl) / per_batch;
  // this thread's token first: its loads are in flight during the walk
  const int64_t xc = x < total ? x : total - 1;
  const uint8_t code = region[xc];
  const uint8_t dd = dist[xc];
  int m = 1;
  for (int64_t bb = b0; bb <= b1; ++bb) {
    int v = 0;
    for (int f = t; f < nper; f += 256) v = max(v, band_max[bb * nper + f]);
    for (int o = 32; o > 0; o >>= 1) v = max(v, __shfl_xor(v, o));
    if ((t & 63) == 0) wm[t >> 6] = v;
    __syncthreads();
    v = max(max(wm[0], wm[1]), max(wm[2], wm[3]));
    __syncthreads();
    if (bb == myb) m = max(m, v);
  }
  if (x >= total) return;
  float w = 0.f;
  if (code == 3) {
    w = 1.f;
  } else if (code == 2) {
    const float s = (float)dd / (float)m;
    w = 1.f - s * s * (3.f - 2.f * s);
  }
  weight[x] = w;
}

// z_out = W z_target + (1 - W) z_hist over latents [B, C, Tl, Hl, Wl], W on
// the token grid [B, Tl / pt, Hl / ph, Wl / pw].  Four consecutive elements
// of a row per thread (Wl % 4 == 0, 16-byte aligned tensors: 16-byte loads
// and stores).  z_out may be z_target or z_hist: each element is read before
// it is written, by the same thread.  I is the index type: 32-bit whenever
// the latent has fewer than 2^32 elements (the row and column of a quad take
// a few divisions, which 64-bit integers make several times dearer).
template <typename I>
__global__ void __launch_bounds__(256) fusion4_kernel(const float4 *zt, const float4 *zh,
                                                      const float *__restrict__ weight,
                                                      float4 *zo, I quads, I C, I Tl, I Hl, I Wl,
                                                      I pt, I ph, I pw) {
  const I qi = (I)blockIdx.x * 256 + threadIdx.x;
  if (qi >= quads) return;
  const I e = qi * 4;
  const I row = e / Wl;  // (b, c, t, y)
  const I x0 = e - row * Wl;
  const I bct = row / Hl;
  const I y = row - bct * Hl;
  const I bc = bct / Tl;
  const I tt = bct - bc * Tl;
  const I b = bc / C;
  const I Tg = Tl / pt, Hg = Hl / ph, Wg = Wl / pw;
  const float *wrow = weight + ((size_t)(b * Tg + tt / pt) * Hg + y / ph) * Wg;
  const float4 a = zt[qi], h = zh[qi];
  float w0, w1, w2, w3;
  if (pw == 1) {
    w0 = wrow[x0], w1 = wrow[x0 + 1], w2 = wrow[x0 + 2], w3 = wrow[x0 + 3];
  } else {
    w0 = wrow[x0 / pw], w1 = wrow[(x0 + 1) / pw], w2 = wrow[(x0 + 2) / pw], w3 = wrow[(x0 + 3) / pw];
  }
  float4 o;
  o.x = w0 * a.x + (1.f - w0) * h.x;
  o.y = w1 * a.y + (1.f - w1) * h.y;
  o.z = w2 * a.z + (1.f - w2) * h.z;
  o.w = w3 * a.w + (1.f - w3) * h.w;
  zo[qi] = o;
}

// The same one element per thread (any Wl, any 4-byte alignment).
__global__ void __launch_bounds__(256) fusion1_kernel(const float *zt, const float *zh,
                                                      const float *__restrict__ weight, float *zo,
                                                      int64_t total, int C, int Tl, int Hl,
                                                      int Wl, int pt, int ph, int pw) {
  const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (e >= total) return;
  const int x = (int)(e % Wl);
  int64_t r = e / Wl;
  const int y = (int)(r % Hl);
  r /= Hl;
  const int tt = (int)(r % Tl);
  const int b = (int)(r / Tl / C);
  const int Tg = Tl / pt, Hg = Hl / ph, Wg = Wl / pw;
  const float w = weight[(((int64_t)b * Tg + tt / pt) * Hg + y / ph) * Wg + x / pw];
  zo[e] = w * zt[e] + (1.f - w) * zh[e];
}

// One wave per (b, block): a query block is active if one of its tokens is
// (code >= 2), a key block is context if one of its tokens is (code >= 1);
// text tokens, before the video tokens, count as both.  Lane l looks at
// tokens l and l + 64 of the block (blocks are at most 128 tokens).
__global__ void __launch_bounds__(256) block_flags_kernel(const uint8_t *__restrict__ region,
                                                          int n_text, int N, int bs, int nB,
                                                          int64_t total, uint8_t *__restrict__ act,
                                                          uint8_t *__restrict__ ctx) {
  const int64_t g = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (g >= total) return;
  const int b = (int)(g / nB), i = (int)(g - (int64_t)b * nB);
  const int nv = N - n_text;
  int best = 0;
  for (int u = 0; u < 2; ++u) {
    const int off = u * 64 + lane;
    const int tok = i * bs + off;
    if (off < bs && tok < N)
      best = max(best, tok < n_text ? 3 : (int)region[(int64_t)b * nv + (tok - n_text)]);
  }
  const bool a = __ballot(best >= 2) != 0, c = __ballot(best >= 1) != 0;
  if (lane == 0) {
    act[g] = a ? 1 : 0;
    ctx[g] = c ? 1 : 0;
  }
}

}  // namespace

size_t region_frame_lds(int H, int W) { return (size_t)2 * H * W; }

size_t region_scratch_bytes(int B, int T, int H, int W) {
  return align_up((size_t)B * T * H * W) + align_up((size_t)B * T * H * sizeof(int32_t));
}

// Bands per frame: enough workgroups for every CU to take about two
// (B T nbands >= 512 when the frames have the rows), at most one band per row.
static int region_bands(int BT, int H) {
  int nb = (512 + BT - 1) / BT;
  nb = nb < 1 ? 1 : (nb > H ? H : nb);
  const int BR = (H + nb - 1) / nb;
  return (H + BR - 1) / BR;
}

hipError_t launch_regions(const uint8_t *evidence, int B, int T, int H, int W, int ra, int rc,
                          uint8_t *region, float *weight, void *scratch, hipStream_t s) {
  const int HW = H * W;
  uint8_t *dist = static_cast<uint8_t *>(scratch);
  int32_t *bmax = reinterpret_cast<int32_t *>(static_cast<char *>(scratch) +
                                              align_up((size_t)B * T * HW));
  const int nbands = region_bands(B * T, H);
  const int BR = (H + nbands - 1) / nbands;
  // staged rows: the band and R rows on either side, within the frame
  const int R = ra + rc;
  const int staged_rows = BR + 2 * R < H ? BR + 2 * R : H;
  const size_t lds = (size_t)2 * staged_rows * W;
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(&region_kernel),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(region_kernel, dim3((unsigned)(B * T), (unsigned)nbands), dim3(kRegionThreads),
                     lds, s, evidence, H, W, BR, nbands, ra, rc, region, dist, bmax);
  const int64_t per = (int64_t)T * HW, total = (int64_t)B * per;
  hipLaunchKernelGGL(weight_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, s, region,
                     dist, bmax, T * nbands, per, total, weight);
  return hipGetLastError();
}

hipError_t launch_fusion(const float *zt, const float *zh, const float *weight, float *zo, int B,
                         int C, int Tl, int Hl, int Wl, int pt, int ph, int pw, hipStream_t s) {
  const int64_t total = (int64_t)B * C * Tl * Hl * Wl;
  if (total == 0) return hipSuccess;
  const bool vec = Wl % 4 == 0 && ((reinterpret_cast<uintptr_t>(zt) | reinterpret_cast<uintptr_t>(zh) |
                                    reinterpret_cast<uintptr_t>(zo)) % 16) == 0;
  if (vec) {
    const int64_t quads = total / 4;
    const dim3 grid((unsigned)((quads + 255) / 256));
    auto f4 = reinterpret_cast<const float4 *>(zt);
    auto h4 = reinterpret_cast<const float4 *>(zh);
    auto o4 = reinterpret_cast<float4 *>(zo);
    if (total < ((int64_t)1 << 32))
      hipLaunchKernelGGL(fusion4_kernel<uint32_t>, grid, dim3(256), 0, s, f4, h4, weight, o4,
                         (uint32_t)quads, (uint32_t)C, (uint32_t)Tl, (uint32_t)Hl, (uint32_t)Wl,
                         (uint32_t)pt, (uint32_t)ph, (uint32_t)pw);
    else
      hipLaunchKernelGGL(fusion4_kernel<uint64_t>, grid, dim3(256), 0, s, f4, h4, weight, o4,
                         (uint64_t)quads, (uint64_t)C, (uint64_t)Tl, (uint64_t)Hl, (uint64_t)Wl,
                         (uint64_t)pt, (uint64_t)ph, (uint64_t)pw);
  } else {
    hipLaunchKernelGGL(fusion1_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, s, zt,
                       zh, weight, zo, total, C, Tl, Hl, Wl, pt, ph, pw);
  }
  return hipGetLastError();
}

hipError_t launch_block_flags(const uint8_t *region, int B, int n_text, int N, int bs, uint8_t *act,
                              uint8_t *ctx, hipStream_t s) {
  const int nB = (N + bs - 1) / bs;
  const int64_t total = (int64_t)B * nB;
  hipLaunchKernelGGL(block_flags_kernel, dim3((unsigned)((total + 3) / 4)), dim3(256), 0, s, region,
                     n_text, N, bs, nB, total, act, ctx);
  return hipGetLastError();
}

}  // namespace carnator
