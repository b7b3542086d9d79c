// Target-row widening of the reused mask and its compaction into per-row
// lists of kept key blocks, from the uint8 mask or from its bit-packed form.
//
// Widening (Sec. 3.3, joint reuse in the middle layers): a target-specific
// query block evaluates every key block, and dense text key blocks are kept
// in every row.  Compaction produces the list the sparse executor walks:
// row_ptr / col_idx (ascending key blocks per row) and an order of rows by
// descending list length (lower row first on equal length), so the longest
// rows start first.
//
// Bit-packed masks (the stored form of the reused connectivity, one bit per
// block pair): uint64 [rows][nw], nw = ceil(nB / 64), key block j of a row
// at bit j mod 64 of word j / 64; bits past nB are written as 0 and ignored
// when read.  Compaction from bits applies the widening while it reads the
// words, so a stored mask is never modified.
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

// A row's mask bytes, lane l holding columns l, l + 64, ... (NC of them, at
// least ceil(nB / 64)).  The column index is clamped to the row rather than
// the load predicated, so all loads are issued before any is used and a row
// costs one memory round trip; columns past nB then read as 0.
template <int NC>
__device__ inline void load_row(const uint8_t *row, int nB, int lane, uint8_t (&v)[NC]) {
#pragma unroll
  for (int c = 0; c < NC; ++c) v[c] = row[min(c * 64 + lane, nB - 1)];
#pragma unroll
  for (int c = 0; c < NC; ++c) v[c] = c * 64 + lane < nB ? v[c] : 0;
}

// One wave per row: number of kept key blocks.
template <int NC>
__global__ void __launch_bounds__(256) count_kernel(const uint8_t *__restrict__ mask, int64_t R,
                                                    int nB, int32_t *__restrict__ len) {
  const int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (r >= R) return;
  uint8_t v[NC];
  load_row(mask + r * nB, nB, lane, v);
  int n = 0;
#pragma unroll
  for (int c = 0; c < NC; ++c) n += __popcll(__ballot(v[c] != 0));
  if (lane == 0) len[r] = n;
}

// One wave per row: ascending kept key blocks at col_idx[row_ptr[r] ...].
template <int NC>
__global__ void __launch_bounds__(256) fill_kernel(const uint8_t *__restrict__ mask, int64_t R,
                                                   int nB, const int32_t *__restrict__ row_ptr,
                                                   int32_t *__restrict__ col_idx) {
  const int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (r >= R) return;
  uint8_t v[NC];
  load_row(mask + r * nB, nB, lane, v);
  int pos = row_ptr[r];
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    const bool kept = v[c] != 0;
    const unsigned long long bits = __ballot(kept);
    if (kept) col_idx[pos + __popcll(bits & ((1ull << lane) - 1ull))] = c * 64 + lane;
    pos += __popcll(bits);
  }
}

// ---- bit-packed masks

// Valid-column bits of word c of a row (the last word may be partial).
__device__ inline uint64_t valid_bits(int c, int nB, int nw) {
  return (c == nw - 1 && (nB & 63)) ? (1ull << (nB & 63)) - 1ull : ~0ull;
}

// One wave per row of nB bytes: lane c < nw writes word c, the ballot of
// chunk c's nonzero bytes.
template <int NC>
__global__ void __launch_bounds__(256) pack_kernel(const uint8_t *__restrict__ mask, int64_t R,
                                                   int nB, uint64_t *__restrict__ bits) {
  const int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (r >= R) return;
  uint8_t v[NC];
  load_row(mask + r * nB, nB, lane, v);
  uint64_t mine = 0;
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    const uint64_t w = __ballot(v[c] != 0);
    mine = lane == c ? w : mine;
  }
  const int nw = (nB + 63) / 64;
  if (lane < nw) bits[r * nw + lane] = mine;
}

// One wave per row: lane c < nw loads word c, then each chunk is broadcast
// and written as 0/1 bytes, 64 columns per store.
__global__ void __launch_bounds__(256) unpack_kernel(const uint64_t *__restrict__ bits, int64_t R,
                                                     int nB, uint8_t *__restrict__ mask) {
  const int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (r >= R) return;
  const int nw = (nB + 63) / 64;
  const uint64_t mine = lane < nw ? bits[r * nw + lane] : 0ull;
  uint8_t *out = mask + r * nB;
  for (int c = 0; c < nw; ++c) {
    const uint64_t w = read_lane(mine, c);
    const int j = c * 64 + lane;
    if (j < nB) out[j] = (uint8_t)((w >> lane) & 1ull);
  }
}

// Every block pair kept: all valid bits set, the rest 0.  One thread per word.
__global__ void __launch_bounds__(256) fill_ones_bits_kernel(uint64_t *__restrict__ bits,
                                                             int64_t words, int nB) {
  const int64_t x = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (x >= words) return;
  const int nw = (nB + 63) / 64;
  bits[x] = valid_bits((int)(x % nw), nB, nw);
}

// Word c of row r as the call reads it (HnB = H nB rows per batch entry;
// rows uint8 [B][nB] and colw, packed column flags [B][nw], may be NULL).
// Widening: all valid bits when the row's query block is flagged, OR the
// column word.  Restriction (narrow): AND the column word (context key
// blocks); whether the row is kept at all is row_kept's.
__device__ inline uint64_t merged_word(const uint64_t *__restrict__ bits, int r, int c, int nB,
                                       int nw, int HnB, const uint8_t *__restrict__ rows,
                                       const uint64_t *__restrict__ colw, bool narrow) {
  uint64_t w = bits[(int64_t)r * nw + c];
  if (rows != nullptr || colw != nullptr) {
    const int b = r / HnB;
    if (narrow) {
      if (colw != nullptr) w &= colw[(int64_t)b * nw + c];
    } else {
      if (rows != nullptr && rows[(int64_t)b * nB + r % nB] != 0) w = ~0ull;
      if (colw != nullptr) w |= colw[(int64_t)b * nw + c];
    }
  }
  return w & valid_bits(c, nB, nw);
}

// Whether row r takes part: always when widening, else when its query block
// is active.
__device__ inline bool row_kept(int r, int nB, int HnB, const uint8_t *__restrict__ rows,
                                bool narrow) {
  return !narrow || rows == nullptr || rows[(int64_t)(r / HnB) * nB + r % nB] != 0;
}

// G lanes per row (G a power of two >= nw), 64 / G rows per wave: list
// lengths as popcounts summed over each row's lanes; -1 for a row a
// restriction leaves out.
template <int G>
__global__ void __launch_bounds__(256) count_bits_kernel(const uint64_t *__restrict__ bits, int R,
                                                         int nB, int HnB,
                                                         const uint8_t *__restrict__ rows,
                                                         const uint64_t *__restrict__ colw,
                                                         bool narrow, int32_t *__restrict__ len) {
  const int lane = threadIdx.x & 63;
  const int64_t r = ((int64_t)blockIdx.x * 4 + (threadIdx.x >> 6)) * (64 / G) + lane / G;
  const int c = lane % G;
  const int nw = (nB + 63) / 64;
  const bool kept = r < R && row_kept((int)r, nB, HnB, rows, narrow);
  int n = 0;
  if (kept && c < nw) n = __popcll(merged_word(bits, (int)r, c, nB, nw, HnB, rows, colw, narrow));
#pragma unroll
  for (int o = 1; o < G; o <<= 1) n += __shfl_xor(n, o);
  if (r < R && c == 0) len[r] = kept ? n : -1;
}

// One wave per row: ascending kept key blocks at col_idx[row_ptr[r] ...].
// Lane c < nw holds word c; chunk c is broadcast and each lane writes its
// column when its bit is set, at the count of set bits below it.
__global__ void __launch_bounds__(256) fill_bits_kernel(const uint64_t *__restrict__ bits, int R,
                                                        int nB, int HnB,
                                                        const uint8_t *__restrict__ rows,
                                                        const uint64_t *__restrict__ colw,
                                                        bool narrow,
                                                        const int32_t *__restrict__ row_ptr,
                                                        int32_t *__restrict__ col_idx) {
  const int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (r >= R || !row_kept((int)r, nB, HnB, rows, narrow)) return;
  const int nw = (nB + 63) / 64;
  const uint64_t mine =
      lane < nw ? merged_word(bits, (int)r, lane, nB, nw, HnB, rows, colw, narrow) : 0ull;
  const uint64_t below = (1ull << lane) - 1ull;
  int pos = row_ptr[r];
  for (int c = 0; c < nw; ++c) {
    const uint64_t w = read_lane(mine, c);
    if ((w >> lane) & 1ull) col_idx[pos + __popcll(w & below)] = c * 64 + lane;
    pos += __popcll(w);
  }
}

constexpr int kScanThreads = 1024;

// Inclusive scan over the 64 lanes of a wave: four DPP row shifts (by 1, 2,
// 4, 8 lanes; lanes shifted in from outside the 16-lane row read 0) scan each
// row, then two row broadcasts add lane 15 into row 1, lane 47 into row 3
// and lane 31 into rows 2 and 3.
__device__ inline int wave_incl_scan(int x) {
  x += __builtin_amdgcn_update_dpp(0, x, 0x111, 0xF, 0xF, true);  // row_shr:1
  x += __builtin_amdgcn_update_dpp(0, x, 0x112, 0xF, 0xF, true);  // row_shr:2
  x += __builtin_amdgcn_update_dpp(0, x, 0x114, 0xF, 0xF, true);  // row_shr:4
  x += __builtin_amdgcn_update_dpp(0, x, 0x118, 0xF, 0xF, true);  // row_shr:8
  x += __builtin_amdgcn_update_dpp(0, x, 0x142, 0xA, 0xF, false);  // row_bcast:15
  x += __builtin_amdgcn_update_dpp(0, x, 0x143, 0xC, 0xF, false);  // row_bcast:31
  return x;
}

// Block-wide exclusive scan of one int per thread (1024 threads); returns the
// exclusive prefix and writes the total to *total.
__device__ int block_excl_scan(int v, int *sh, int *total) {
  const int t = threadIdx.x;
  const int lane = t & 63, w = t >> 6;
  const int x = wave_incl_scan(v);
  if (lane == 63) sh[w] = x;
  __syncthreads();
  if (w == 0) {
    const int s = wave_incl_scan(lane < kScanThreads / 64 ? sh[lane] : 0);
    if (lane < kScanThreads / 64) sh[lane] = s;
  }
  __syncthreads();
  const int before = (w > 0 ? sh[w - 1] : 0) + x - v;
  *total = sh[kScanThreads / 64 - 1];
  __syncthreads();
  return before;
}

// LDS budget of the counting sort: its counters and, when they fit beside
// them, the row lengths.
constexpr size_t kCountSortLds = 152 * 1024;

// Single workgroup: row_ptr = exclusive scan of the list lengths, and the
// order of rows by descending length (lower row first on equal lengths) as a
// counting sort on the length.  Wave w owns the contiguous rows
// [w C, (w + 1) C) and walks them 64 at a time in row order.
//   row_ptr: each wave sums its rows, the 16 wave totals give each wave its
//     first offset, and a second walk writes the offsets with wave scans.
//   order: pass 1 counts rows per (length, wave) with LDS atomics; an
//     exclusive scan in (length descending, wave) order turns the counts into
//     the first slot of each (length, wave) group; pass 2 walks the rows again
//     in order: lanes holding equal lengths find each other with one ballot
//     per key bit, each takes its group's next slot plus its rank among those
//     lanes, and the lowest of them advances the counter.  Lengths descend,
//     waves and rows ascend: the order the oracle defines.
// A length of -1 marks a row left out of a restricted call: its list is
// empty and it sorts after every row of length >= 0 (key nB + 1), in row
// order; *n_active (when not NULL) receives the number of the other rows,
// which the exclusive scan leaves as the first slot of key nB + 1.
// LDS: uint32 counters [nB + 2][16] (index (nB - L) 16 + w), then with
// LEN_LDS the lengths as int16 [R]; otherwise they are read from len_g.
template <bool LEN_LDS>
__global__ void __launch_bounds__(kScanThreads) count_sort_kernel(const int32_t *__restrict__ len_g,
                                                                  int R, int nB,
                                                                  int32_t *__restrict__ row_ptr,
                                                                  int32_t *__restrict__ order,
                                                                  int32_t *__restrict__ n_active) {
  constexpr int kWaves = kScanThreads / 64;
  __shared__ int sh[kWaves];
  extern __shared__ uint32_t cnt[];
  const int K = (nB + 2) * kWaves;
  int16_t *len16 = reinterpret_cast<int16_t *>(cnt + K);
  const int t = threadIdx.x, lane = t & 63;
  const int w = __builtin_amdgcn_readfirstlane(t >> 6);
  for (int i = t; i < K; i += kScanThreads) cnt[i] = 0;
  if constexpr (LEN_LDS) {
    // eight loads in flight per thread, clamped indices
    for (int r0 = 0; r0 < R; r0 += 8 * kScanThreads) {
      int v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int r = r0 + u * kScanThreads + t;
        v[u] = len_g[r < R ? r : R - 1];
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int r = r0 + u * kScanThreads + t;
        if (r < R) len16[r] = (int16_t)v[u];
      }
    }
  }
  __syncthreads();
  auto lenv = [&](int r) __attribute__((always_inline)) -> int {
    if constexpr (LEN_LDS) return len16[r];
    else return len_g[r];
  };
  const int C = (R + kWaves - 1) / kWaves;
  const int rlo = min(R, w * C), rhi = min(R, rlo + C);

  // ---- row_ptr
  {
    int part = 0;
    for (int r0 = rlo; r0 < rhi; r0 += 64) {
      const int r = r0 + lane;
      part += r < rhi ? max(lenv(r), 0) : 0;
    }
    const int wtot = __builtin_amdgcn_readlane(wave_incl_scan(part), 63);
    if (lane == 0) sh[w] = wtot;
    __syncthreads();
    int off = 0, total = 0;
    for (int q = 0; q < kWaves; ++q) {
      const int c = sh[q];
      off += q < w ? c : 0;
      total += c;
    }
    for (int r0 = rlo; r0 < rhi; r0 += 64) {
      const int r = r0 + lane;
      const int v = r < rhi ? max(lenv(r), 0) : 0;
      const int incl = wave_incl_scan(v);
      if (r < rhi) row_ptr[r] = off + incl - v;
      off += __builtin_amdgcn_readlane(incl, 63);
    }
    if (t == 0) row_ptr[R] = total;
  }

  // ---- order
  int kbits = 0;
  while ((1 << kbits) <= nB + 1) ++kbits;
  // the lanes of this walk step holding the same key (nB - length) as this lane
  auto peers_of = [&](bool on, int key) __attribute__((always_inline)) {
    unsigned long long m = __ballot(on);
    for (int b = 0; b < kbits; ++b) {
      const unsigned long long ones = __ballot(on && ((key >> b) & 1));
      m &= ((key >> b) & 1) ? ones : ~ones;
    }
    return m;
  };
  for (int r0 = rlo; r0 < rhi; r0 += 64) {
    const int r = r0 + lane;
    if (r < rhi) atomicAdd(&cnt[(nB - lenv(r)) * kWaves + w], 1u);
  }
  __syncthreads();
  {
    // exclusive scan of the counters in index order, a contiguous segment per
    // thread
    const int per = (K + kScanThreads - 1) / kScanThreads;
    const int lo = min(K, per * t), hi = min(K, lo + per);
    int local = 0;
    for (int i = lo; i < hi; ++i) local += (int)cnt[i];
    int total;
    int run = block_excl_scan(local, sh, &total);
    for (int i = lo; i < hi; ++i) {
      const int c = (int)cnt[i];
      cnt[i] = (uint32_t)run;
      run += c;
    }
  }
  __syncthreads();
  // (wave 0 reads the slot before its own pass-2 updates; other waves never
  // update counter (nB + 1) 16 + 0)
  if (t == 0 && n_active != nullptr) *n_active = (int32_t)cnt[(nB + 1) * kWaves];
  for (int r0 = rlo; r0 < rhi; r0 += 64) {
    const int r = r0 + lane;
    const bool on = r < rhi;
    const int key = on ? nB - lenv(r) : 0;
    const unsigned long long m = peers_of(on, key);
    if (on) {
      uint32_t &c = cnt[key * kWaves + w];
      order[(int)c + __popcll(m & ((1ull << lane) - 1ull))] = r;
      // every lane of the group has read the counter before the lowest lane
      // writes it back (one wave: its LDS accesses complete in program order)
      if (lane == __builtin_ctzll(m)) c += (uint32_t)__popcll(m);
    }
  }
}

// ---- the same row_ptr and order by several workgroups (chunks of kChunk rows)
//
//   sort_hist_kernel, one workgroup per chunk g: the chunk's key histogram
//     (key = nB - length, nB + 1 for a left-out row) to hist[g K + key],
//     K = nB + 2, and its length sum to csum[g];
//   sort_scan_kernel, one workgroup: for each key, the exclusive prefix of
//     its counts over the chunks plus the exclusive prefix of the key totals
//     (key order) -- the first slot of chunk g's rows of each key -- and the
//     exclusive scan of csum;
//   sort_place_kernel, one workgroup per chunk: row_ptr of its rows (chunk
//     offset plus a block scan), and each row's slot in order: its chunk's
//     first slot for its key, plus the rows of that key in earlier waves of
//     the chunk (per-wave counts, scanned per key), plus the lanes below it
//     in its wave holding the same key (one ballot per key bit).
// Within a chunk wave w holds rows 64 w .. 64 w + 63 in row order, so rows
// of equal key keep their row order: the order the oracle defines.
constexpr int kChunk = 1024;

__device__ inline int sort_key(int L, int nB) { return L < 0 ? nB + 1 : nB - L; }

__global__ void __launch_bounds__(kScanThreads) sort_hist_kernel(const int32_t *__restrict__ len,
                                                                 int R, int nB, int G,
                                                                 int32_t *__restrict__ hist,
                                                                 int32_t *__restrict__ csum) {
  extern __shared__ int hk[];  // nB + 2 counters
  __shared__ int sh[kScanThreads / 64];
  const int g = blockIdx.x, t = threadIdx.x;
  for (int k = t; k < nB + 2; k += kScanThreads) hk[k] = 0;
  __syncthreads();
  const int r = g * kChunk + t;
  const int L = r < R ? len[r] : 0;
  if (r < R) atomicAdd(&hk[sort_key(L, nB)], 1);
  int total;
  (void)block_excl_scan(max(L, 0), sh, &total);
  for (int k = t; k < nB + 2; k += kScanThreads) hist[(int64_t)g * (nB + 2) + k] = hk[k];
  if (t == 0) csum[g] = total;
}

// One workgroup, thread t owning keys t, t + 1024, t + 2048: the chunk
// prefix of each of its keys (G coalesced loads and stores per key, eight
// loads in flight), then the key totals scanned in key order one pass of
// 1024 keys at a time and added back; the chunk offsets of row_ptr, row_ptr[R]
// and the number of rows not left out (the first slot of key nB + 1).
__global__ void __launch_bounds__(kScanThreads) sort_scan_kernel(int R, int nB, int G,
                                                                 int32_t *__restrict__ hist,
                                                                 int32_t *__restrict__ csum,
                                                                 int32_t *__restrict__ row_ptr,
                                                                 int32_t *__restrict__ n_active) {
  __shared__ int sh[kScanThreads / 64];
  const int t = threadIdx.x;
  const int K = nB + 2;
  int carry = 0;
  for (int k0 = 0; k0 < K; k0 += kScanThreads) {
    const int k = k0 + t;
    int tot = 0;
    if (k < K) {
      for (int g0 = 0; g0 < G; g0 += 8) {
        int v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] = g0 + u < G ? hist[(int64_t)(g0 + u) * K + k] : 0;
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          if (g0 + u < G) hist[(int64_t)(g0 + u) * K + k] = tot;
          tot += v[u];
        }
      }
    }
    int all;
    const int ex = block_excl_scan(tot, sh, &all) + carry;
    carry += all;
    if (k < K) {
      for (int g = 0; g < G; ++g) hist[(int64_t)g * K + k] += ex;
    }
  }
  // chunk offsets of row_ptr
  int rcarry = 0;
  for (int g0 = 0; g0 < G; g0 += kScanThreads) {
    const int g = g0 + t;
    const int v = g < G ? csum[g] : 0;
    int tot;
    const int ex = block_excl_scan(v, sh, &tot);
    if (g < G) csum[g] = rcarry + ex;
    rcarry += tot;
  }
  if (t == 0) row_ptr[R] = rcarry;
  // the first slot of key nB + 1 (chunk 0): written by the thread owning it
  if (n_active != nullptr && t == (nB + 1) % kScanThreads) {
    __threadfence_block();
    *n_active = hist[nB + 1];
  }
}

__global__ void __launch_bounds__(kScanThreads) sort_place_kernel(const int32_t *__restrict__ len,
                                                                  int R, int nB, int G,
                                                                  const int32_t *__restrict__ base,
                                                                  const int32_t *__restrict__ coff,
                                                                  int32_t *__restrict__ row_ptr,
                                                                  int32_t *__restrict__ order) {
  constexpr int kWaves = kScanThreads / 64;
  extern __shared__ int wc[];  // (nB + 2) * kWaves per-wave counts, then slots
  __shared__ int sh[kWaves];
  const int g = blockIdx.x, t = threadIdx.x, lane = t & 63;
  const int w = __builtin_amdgcn_readfirstlane(t >> 6);
  const int K = nB + 2;
  for (int i = t; i < K * kWaves; i += kScanThreads) wc[i] = 0;
  __syncthreads();
  const int r = g * kChunk + t;
  const bool on = r < R;
  const int L = on ? len[r] : 0;
  const int key = on ? sort_key(L, nB) : 0;
  if (on) atomicAdd(&wc[key * kWaves + w], 1);
  int total;
  const int ex = block_excl_scan(on ? max(L, 0) : 0, sh, &total);  // ends with a barrier
  if (on) row_ptr[r] = coff[g] + ex;
  for (int k = t; k < K; k += kScanThreads) {
    int run = base[(int64_t)g * K + k];
#pragma unroll
    for (int q = 0; q < kWaves; ++q) {
      const int c = wc[k * kWaves + q];
      wc[k * kWaves + q] = run;
      run += c;
    }
  }
  __syncthreads();
  int kbits = 0;
  while ((1 << kbits) <= nB + 1) ++kbits;
  unsigned long long m = __ballot(on);
  for (int b = 0; b < kbits; ++b) {
    const unsigned long long ones = __ballot(on && ((key >> b) & 1));
    m &= ((key >> b) & 1) ? ones : ~ones;
  }
  if (on) order[wc[key * kWaves + w] + __popcll(m & ((1ull << lane) - 1ull))] = r;
}

}  // namespace

hipError_t launch_merge(uint8_t *mask, int B, int H, int nB, const uint8_t *rows,
                        const uint8_t *cols, hipStream_t s) {
  const int64_t total = (int64_t)B * H * nB * nB;
  hipLaunchKernelGGL(merge_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, s, mask, H,
                     nB, total, rows, cols);
  return hipGetLastError();
}

static int sort_chunks(int64_t R) { return (int)((R + kChunk - 1) / kChunk); }

// Lengths, then the chunk histograms and offsets of the multi-workgroup sort.
size_t compact_scratch_bytes(int64_t R, int nB) {
  const int G = sort_chunks(R);
  return align_up((size_t)R * sizeof(int32_t)) + align_up((size_t)(nB + 2) * G * sizeof(int32_t)) +
         align_up((size_t)G * sizeof(int32_t));
}

// Rows up to which the single-workgroup counting sort runs (one launch);
// beyond, the chunked sort (three launches) spreads the walk over the CUs.
constexpr int64_t kSingleSortRows = 4096;

// row_ptr and order from the list lengths; sort_scratch: the histogram and
// chunk offsets of compact_scratch_bytes.
static hipError_t launch_sort(const int32_t *len, int64_t R, int nB, int32_t *row_ptr, int32_t *order,
                              int32_t *n_active, void *sort_scratch, hipStream_t s) {
  if (R > kSingleSortRows) {
    const int G = sort_chunks(R);
    int32_t *hist = static_cast<int32_t *>(sort_scratch);
    int32_t *csum = reinterpret_cast<int32_t *>(static_cast<char *>(sort_scratch) +
                                                align_up((size_t)(nB + 2) * G * sizeof(int32_t)));
    const size_t hl = (size_t)(nB + 2) * sizeof(int32_t);
    const size_t pl = (size_t)(nB + 2) * (kScanThreads / 64) * sizeof(int32_t);
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(&sort_place_kernel),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)pl);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(sort_hist_kernel, dim3((unsigned)G), dim3(kScanThreads), hl, s, len, (int)R, nB,
                       G, hist, csum);
    hipLaunchKernelGGL(sort_scan_kernel, dim3(1), dim3(kScanThreads), 0, s, (int)R, nB, G, hist, csum,
                       row_ptr, n_active);
    hipLaunchKernelGGL(sort_place_kernel, dim3((unsigned)G), dim3(kScanThreads), pl, s, len, (int)R, nB,
                       G, hist, csum, row_ptr, order);
    return hipGetLastError();
  }
  const size_t cnt_lds = (size_t)(nB + 2) * (kScanThreads / 64) * sizeof(uint32_t);
  const size_t len_lds = (size_t)R * sizeof(int16_t);
  hipError_t e;
  if (cnt_lds + len_lds <= kCountSortLds) {
    e = hipFuncSetAttribute(reinterpret_cast<const void *>(&count_sort_kernel<true>),
                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)(cnt_lds + len_lds));
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(count_sort_kernel<true>, dim3(1), dim3(kScanThreads), cnt_lds + len_lds, s,
                       len, (int)R, nB, row_ptr, order, n_active);
  } else {
    e = hipFuncSetAttribute(reinterpret_cast<const void *>(&count_sort_kernel<false>),
                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)cnt_lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(count_sort_kernel<false>, dim3(1), dim3(kScanThreads), cnt_lds, s, len,
                       (int)R, nB, row_ptr, order, n_active);
  }
  return hipGetLastError();
}

hipError_t launch_compact(const uint8_t *mask, int64_t R, int nB, int32_t *row_ptr,
                          int32_t *col_idx, int32_t *order, void *scratch, hipStream_t s) {
  int32_t *len = static_cast<int32_t *>(scratch);
  const unsigned g = (unsigned)((R + 3) / 4);
  const int nc = (nB + 63) / 64;  // nB <= 2048
#define CARNATOR_ROWS(KERNEL, ...)                                                         \
  do {                                                                                   \
    if (nc <= 4) hipLaunchKernelGGL(KERNEL<4>, dim3(g), dim3(256), 0, s, __VA_ARGS__);   \
    else if (nc <= 8) hipLaunchKernelGGL(KERNEL<8>, dim3(g), dim3(256), 0, s, __VA_ARGS__); \
    else if (nc <= 16) hipLaunchKernelGGL(KERNEL<16>, dim3(g), dim3(256), 0, s, __VA_ARGS__); \
    else hipLaunchKernelGGL(KERNEL<32>, dim3(g), dim3(256), 0, s, __VA_ARGS__);          \
  } while (0)
  CARNATOR_ROWS(count_kernel, mask, R, nB, len);
  hipError_t e = launch_sort(len, R, nB, row_ptr, order, nullptr,
                             static_cast<char *>(scratch) + align_up((size_t)R * sizeof(int32_t)), s);
  if (e != hipSuccess) return e;
  CARNATOR_ROWS(fill_kernel, mask, R, nB, row_ptr, col_idx);
  return hipGetLastError();
}

hipError_t launch_pack(const uint8_t *mask, int64_t R, int nB, uint64_t *bits, hipStream_t s) {
  if (R == 0) return hipSuccess;
  const unsigned g = (unsigned)((R + 3) / 4);
  const int nc = (nB + 63) / 64;
  CARNATOR_ROWS(pack_kernel, mask, R, nB, bits);
  return hipGetLastError();
}
#undef CARNATOR_ROWS

hipError_t launch_unpack(const uint64_t *bits, int64_t R, int nB, uint8_t *mask, hipStream_t s) {
  hipLaunchKernelGGL(unpack_kernel, dim3((unsigned)((R + 3) / 4)), dim3(256), 0, s, bits, R, nB,
                     mask);
  return hipGetLastError();
}

hipError_t launch_fill_ones_bits(uint64_t *bits, int64_t R, int nB, hipStream_t s) {
  const int64_t words = R * ((nB + 63) / 64);
  hipLaunchKernelGGL(fill_ones_bits_kernel, dim3((unsigned)((words + 255) / 256)), dim3(256), 0, s,
                     bits, words, nB);
  return hipGetLastError();
}

size_t compact_bits_scratch_bytes(int64_t R, int B, int nB) {
  return compact_scratch_bytes(R, nB) + align_up((size_t)B * ((nB + 63) / 64) * sizeof(uint64_t));
}

hipError_t launch_compact_bits(const uint64_t *bits, int B, int H, int nB, const uint8_t *rows,
                               const uint8_t *cols, bool narrow, int32_t *row_ptr,
                               int32_t *col_idx, int32_t *order, int32_t *n_active, void *scratch,
                               hipStream_t s) {
  const int64_t R = (int64_t)B * H * nB;
  int32_t *len = static_cast<int32_t *>(scratch);
  uint64_t *colw = nullptr;
  hipError_t e;
  if (cols != nullptr) {
    // the column flags of each batch entry, packed once like a mask row
    colw = reinterpret_cast<uint64_t *>(static_cast<char *>(scratch) + compact_scratch_bytes(R, nB));
    if ((e = launch_pack(cols, B, nB, colw, s)) != hipSuccess) return e;
  }
  const int nw = (nB + 63) / 64;  // nB <= 2048
  const int HnB = H * nB;
  int G = 1;
  while (G < nw) G <<= 1;
  const unsigned gc = (unsigned)((R + 4 * (64 / G) - 1) / (4 * (64 / G)));
  switch (G) {
#define CARNATOR_G(GG)                                                                            \
  case GG:                                                                                        \
    hipLaunchKernelGGL(count_bits_kernel<GG>, dim3(gc), dim3(256), 0, s, bits, (int)R, nB, HnB,   \
                       rows, colw, narrow, len);                                                  \
    break;
    CARNATOR_G(1) CARNATOR_G(2) CARNATOR_G(4) CARNATOR_G(8) CARNATOR_G(16) CARNATOR_G(32)
#undef CARNATOR_G
    default: return hipErrorInvalidValue;
  }
  if ((e = launch_sort(len, R, nB, row_ptr, order, n_active,
                       static_cast<char *>(scratch) + align_up((size_t)R * sizeof(int32_t)), s)) !=
      hipSuccess)
    return e;
  hipLaunchKernelGGL(fill_bits_kernel, dim3((unsigned)((R + 3) / 4)), dim3(256), 0, s, bits,
                     (int)R, nB, HnB, rows, colw, narrow, row_ptr, col_idx);
  return hipGetLastError();
}

}  // namespace carnator
