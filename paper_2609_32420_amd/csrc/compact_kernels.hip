// Target-row widening of the reused mask and its compaction into per-row
// lists of kept key blocks, from the uint8 mask or from its bit-packed form.
//
// Widening (Sec. 3.3, joint reuse in the middle layers): a target-specific
// query block evaluates every key block, and dense text key blocks are kept
// in every row.  Compaction produces the list the sparse executor walks:
// row_ptr / col_idx (ascending key blocks per row) and an order of rows:
// the heads in consecutive groups whose K and V fit the Infinity Cache
// (order_group_heads), group after group, and inside a group the rows by
// descending list length (lower row first on equal length), so a group's
// longest rows start first.
//
// Bit-packed masks (the stored form of the reused connectivity, one bit per
// block pair): uint64 [rows][nw], nw = ceil(nB / 64), key block j of a row
// at bit j mod 64 of word j / 64; bits past nB are written as 0 and ignored
// when read.  Compaction from bits applies the widening while it reads the
// words, so a stored mask is never modified.
#include "internal.h"

#include <type_traits>

namespace carnator {
namespace {

// Rows per chunk of the row sort (one thread per row of a chunk).
constexpr int kChunk = 1024;

// Rows in head groups of gr rows (gr a multiple of nB; one group when
// gr >= R), each group cut into chunks of kChunk rows: chunk c is chunk
// c mod cpg of group c / cpg, cpg = ceil(gr / kChunk), so no chunk spans two
// groups (the last chunk of a group, and chunks past R, may be partial or
// empty).
struct Chunks {
  int64_t R, gr;
  int cpg;
  __host__ __device__ int64_t lo(int c) const {
    const int g = c / cpg;
    const int64_t r = (int64_t)g * gr + (int64_t)(c - g * cpg) * kChunk;
    return r < R ? r : R;
  }
  __host__ __device__ int64_t hi(int c) const {
    const int g = c / cpg;
    int64_t r = (int64_t)g * gr + (int64_t)(c - g * cpg + 1) * kChunk;
    const int64_t ge = (int64_t)(g + 1) * gr;
    r = r < ge ? r : ge;
    return r < R ? r : R;
  }
  __host__ __device__ int of(int64_t r) const {
    const int64_t g = r / gr;
    return (int)(g * cpg + (r - g * gr) / kChunk);
  }
};

// Sixteen bytes of the flat mask per thread (one 16-byte load and store when
// the mask is 16-byte aligned); a thread's bytes may run over row ends, so
// it finds (b, h, i, j) of its first byte once and steps from there.
// B*H*nB*nB < 2^31 (the shape check), so 32-bit indices.
__global__ void __launch_bounds__(256) merge_kernel(uint8_t *__restrict__ mask, int H, int nB,
                                                    int total, bool vec,
                                                    const uint8_t *__restrict__ rows,
                                                    const uint8_t *__restrict__ cols) {
  const int64_t x64 = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 16;
  if (x64 >= total) return;
  const int x0 = (int)x64;
  const int n = min(16, total - x0);
  const int gr = x0 / nB;  // row of the flat mask: (b * H + h) * nB + i
  int j = x0 - gr * nB;
  const int bh = gr / nB;
  int i = gr - bh * nB;
  int b = bh / H;
  int h = bh - b * H;
  union {
    uint4 q;
    uint8_t c[16];
  } v;
  if (vec && n == 16) {
    v.q = *reinterpret_cast<const uint4 *>(mask + x0);
  } else {
#pragma unroll
    for (int k = 0; k < 16; ++k) v.c[k] = k < n ? mask[x0 + k] : 0;
  }
  bool rf = rows[b * nB + i] != 0;
#pragma unroll
  for (int k = 0; k < 16; ++k) {
    const bool cf = cols != nullptr && k < n && cols[b * nB + j] != 0;
    v.c[k] = (v.c[k] != 0 || rf || cf) ? 1 : 0;
    if (++j == nB) {  // the next byte starts a row
      j = 0;
      if (++i == nB) {
        i = 0;
        if (++h == H) h = 0, ++b;
      }
      rf = k + 1 < n && rows[b * nB + i] != 0;
    }
  }
  if (vec && n == 16) {
    *reinterpret_cast<uint4 *>(mask + x0) = v.q;
  } else {
#pragma unroll
    for (int k = 0; k < 16; ++k)
      if (k < n) mask[x0 + k] = v.c[k];
  }
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
struct FillBits {
  const uint64_t *bits;
  int R, nB, HnB;
  const uint8_t *rows;
  const uint64_t *colw;
  bool narrow;
  const int32_t *coff, *rloc;
  Chunks ch;
  int32_t *col_idx;
  __device__ void operator()(int64_t r, int lane, int *) const {
    if (r >= R || !row_kept((int)r, nB, HnB, rows, narrow)) return;
    const int nw = (nB + 63) / 64;
    const uint64_t mine =
        lane < nw ? merged_word(bits, (int)r, lane, nB, nw, HnB, rows, colw, narrow) : 0ull;
    const uint64_t below = (1ull << lane) - 1ull;
    int pos = coff[ch.of(r)] + rloc[r];
    for (int c = 0; c < nw; ++c) {
      const uint64_t w = read_lane(mine, c);
      if ((w >> lane) & 1ull) col_idx[pos + __popcll(w & below)] = c * 64 + lane;
      pos += __popcll(w);
    }
  }
};

constexpr int kScanThreads = 1024;
static_assert(kChunk == kScanThreads, "one sort thread per row of a chunk");

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

// ---- compaction of uint8 masks
//
// A row of nB mask bytes as aligned 16-byte chunks: lane l loads chunk
// l + 64 u (u < NU) of the span, so a row costs one 16-byte load per lane
// and round.  keep[u] holds one bit per byte of the chunk, set for a nonzero
// byte inside the row; col0[u] is the column of the chunk's first byte
// (negative when the row starts inside it).  Bytes outside the row are
// read (they lie in the same aligned 16 bytes as row bytes) but not used.
template <int NU>
__device__ inline void load_row16(const uint8_t *row, int nB, int lane, uint32_t (&keep)[NU],
                                  int (&col0)[NU]) {
  const uintptr_t p = reinterpret_cast<uintptr_t>(row);
  const uintptr_t pa = p & ~(uintptr_t)15;
  const int head = (int)(p - pa);  // row bytes start at this byte of chunk 0
  const int nch = (head + nB + 15) >> 4;
  uint4 w[NU];
#pragma unroll
  for (int u = 0; u < NU; ++u) {
    const int c = min(u * 64 + lane, nch - 1);
    w[u] = *reinterpret_cast<const uint4 *>(pa + 16 * (uintptr_t)c);
  }
  // bit 7 of each byte: set when the byte is nonzero; then the four bytes'
  // flags of a word gathered into 4 bits
  auto nz4 = [](uint32_t x) __attribute__((always_inline)) {
    const uint32_t f = (((x & 0x7F7F7F7Fu) + 0x7F7F7F7Fu) | x) & 0x80808080u;
    return ((f >> 7) & 1u) | ((f >> 14) & 2u) | ((f >> 21) & 4u) | ((f >> 28) & 8u);
  };
#pragma unroll
  for (int u = 0; u < NU; ++u) {
    const int c = u * 64 + lane;
    const int off = 16 * c - head;
    const int lo = max(0, -off), hi = min(16, nB - off);
    const uint32_t valid = (c < nch && hi > lo) ? (((1u << hi) - 1u) & ~((1u << lo) - 1u)) : 0u;
    const uint32_t f = nz4(w[u].x) | (nz4(w[u].y) << 4) | (nz4(w[u].z) << 8) | (nz4(w[u].w) << 12);
    keep[u] = f & valid;
    col0[u] = off;
  }
}

// One wave per row: number of kept key blocks.
template <int NU>
__global__ void __launch_bounds__(256) count_kernel(const uint8_t *__restrict__ mask, int64_t R,
                                                    int nB, int32_t *__restrict__ len) {
  const int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (r >= R) return;
  uint32_t keep[NU];
  int col0[NU];
  load_row16<NU>(mask + r * nB, nB, lane, keep, col0);
  int n = 0;
#pragma unroll
  for (int u = 0; u < NU; ++u) n += __popc(keep[u]);
  n = __builtin_amdgcn_readlane(wave_incl_scan(n), 63);
  if (lane == 0) len[r] = n;
}

// One wave per row (row r, lane lane): ascending kept key blocks from
// col_idx[row_ptr[r]] on, row_ptr[r] being the offset of r's chunk of rows
// plus its prefix inside the chunk (both written by the sort).  A lane
// writes its 16 bytes' columns into the wave's LDS staging area (nB + 2
// ints) at the count of kept columns in the lanes below it (a wave scan);
// the wave then copies the list out, 64 consecutive entries per store.
template <int NU>
struct FillBytes {
  const uint8_t *mask;
  int64_t R;
  int nB;
  const int32_t *coff, *rloc;
  Chunks ch;
  int32_t *col_idx;
  __device__ void operator()(int64_t r, int lane, int *stage) const {
    if (r >= R) return;
    uint32_t keep[NU];
    int col0[NU];
    load_row16<NU>(mask + r * nB, nB, lane, keep, col0);
    const int pos = coff[ch.of(r)] + rloc[r];
    int n = 0;
#pragma unroll
    for (int u = 0; u < NU; ++u) {
      const int cnt = __popc(keep[u]);
      const int incl = wave_incl_scan(cnt);
      int q = n + incl - cnt;
      for (uint32_t k = keep[u]; k != 0u; k &= k - 1u) stage[q++] = col0[u] + __builtin_ctz(k);
      n += __builtin_amdgcn_readlane(incl, 63);
    }
    // one wave: its LDS writes complete before its reads
    for (int i = lane; i < n; i += 64) col_idx[pos + i] = stage[i];
  }
};

// ---- row_ptr and the order of rows
//
// Sort key of a row: nB - length, so that longer lists come first, and
// nB + 1 for a row a restriction leaves out (length -1: an empty list,
// placed after every other row).  The order lists the rows group by group
// (the Chunks groups of heads; one group when they all fit), each group's
// rows by key, lower row first on equal key, then the rows left out in row
// order.
//   sort_hist_kernel, one workgroup per chunk c: the chunk's key histogram
//     to hist[c K + key] (K = nB + 2), each row's exclusive prefix of the
//     lengths inside the chunk to rloc, the chunk's length sum to csum[c];
//   sort_scan_kernel, one workgroup, thread t owning keys t, t + 1024, ...:
//     for each active key the exclusive prefix of its counts over the chunks
//     of each group and the group's total of that key (gtot[g (nB + 1) +
//     key]); for the left-out key the prefix over all chunks.  The totals,
//     scanned in (group, key) order, give the first slot of each group's
//     rows of each key and are added to the prefixes: hist[c K + key] is
//     then the first slot in order of chunk c's rows of that key (the
//     left-out rows start after all active ones).  csum in place: the chunk
//     offsets of row_ptr; row_ptr[R]; *n_active, the number of active rows;
//   place_fill_kernel, workgroups 0 .. G - 1, one per chunk: row_ptr of its
//     rows (chunk offset plus rloc), and each row's slot in order: its
//     chunk's first slot for its key, plus the rows of that key in earlier
//     waves of the chunk (per-wave counts, scanned per key), plus the lanes
//     below it in its wave holding the same key (one ballot per key bit).
//     The other workgroups write col_idx, one wave per row, from the same
//     chunk offset and rloc: the two parts share the launch and nothing
//     else.
// Within a chunk wave w holds rows 64 w .. 64 w + 63 in row order, so rows
// of equal key keep their row order: the order the oracle defines.
constexpr int kSortWaves = kScanThreads / 64;

__device__ inline int sort_key(int L, int nB) { return L < 0 ? nB + 1 : nB - L; }

__global__ void __launch_bounds__(kScanThreads) sort_hist_kernel(const int32_t *__restrict__ len,
                                                                 Chunks ch, int nB,
                                                                 int32_t *__restrict__ hist,
                                                                 int32_t *__restrict__ csum,
                                                                 int32_t *__restrict__ rloc) {
  extern __shared__ int hk[];  // nB + 2 counters
  __shared__ int sh[kSortWaves];
  const int c = blockIdx.x, t = threadIdx.x;
  const int K = nB + 2;
  for (int k = t; k < K; k += kScanThreads) hk[k] = 0;
  __syncthreads();
  const int64_t r = ch.lo(c) + t;
  const bool on = r < ch.hi(c);
  const int L = on ? len[r] : 0;
  if (on) atomicAdd(&hk[sort_key(L, nB)], 1);
  int total;
  const int ex = block_excl_scan(max(L, 0), sh, &total);  // ends with a barrier
  if (on) rloc[r] = ex;
  for (int k = t; k < K; k += kScanThreads) hist[(int64_t)c * K + k] = hk[k];
  if (t == 0) csum[c] = total;
}

// Up to REGS chunks a key's counts stay in registers (one round trip; REGS
// >= G, the smallest of 4, 8, 16, 32); beyond, they are read sixteen at a
// time.
template <int REGS>
__global__ void __launch_bounds__(kScanThreads) sort_scan_kernel(int R, int nB, int G, int cpg,
                                                                 int ngroups,
                                                                 int32_t *__restrict__ hist,
                                                                 int32_t *__restrict__ csum,
                                                                 int32_t *__restrict__ gtot,
                                                                 int32_t *__restrict__ row_ptr,
                                                                 int32_t *__restrict__ n_active) {
  __shared__ int sh[kSortWaves];
  const int t = threadIdx.x;
  const int K = nB + 2, KA = nB + 1;
  // in-group prefixes (a key's running count restarts at each group's first
  // chunk; the left-out key's does not) and the group totals
  for (int k = t; k < K; k += kScanThreads) {
    const bool left_out = k == KA;
    int run = 0;
    auto step = [&](int c, int v) __attribute__((always_inline)) {
      if (!left_out && c % cpg == 0 && c > 0) {
        gtot[(int64_t)(c / cpg - 1) * KA + k] = run;
        run = 0;
      }
      hist[(int64_t)c * K + k] = run;
      run += v;
    };
    if (G <= REGS) {
      int v[REGS];
#pragma unroll
      for (int u = 0; u < REGS; ++u) v[u] = u < G ? hist[(int64_t)u * K + k] : 0;
#pragma unroll
      for (int u = 0; u < REGS; ++u)
        if (u < G) step(u, v[u]);
    } else {
      for (int c0 = 0; c0 < G; c0 += 16) {
        int v[16];
#pragma unroll
        for (int u = 0; u < 16; ++u) v[u] = c0 + u < G ? hist[(int64_t)(c0 + u) * K + k] : 0;
#pragma unroll
        for (int u = 0; u < 16; ++u)
          if (c0 + u < G) step(c0 + u, v[u]);
      }
    }
    if (!left_out) gtot[(int64_t)(ngroups - 1) * KA + k] = run;
  }
  __threadfence_block();  // gtot, written and then read by other threads of the workgroup
  __syncthreads();
  // the group totals scanned in (group, key) order, a contiguous run of
  // entries per thread
  int active;
  {
    const int64_t M = (int64_t)ngroups * KA;
    const int64_t per = (M + kScanThreads - 1) / kScanThreads;
    const int64_t lo = min(M, per * t), hi = min(M, lo + per);
    int local = 0;
    for (int64_t i = lo; i < hi; ++i) local += gtot[i];
    int run = block_excl_scan(local, sh, &active);  // ends with a barrier
    for (int64_t i = lo; i < hi; ++i) {
      const int c = gtot[i];
      gtot[i] = run;
      run += c;
    }
  }
  __threadfence_block();
  __syncthreads();
  // first slots: prefix + the group's start for the key (the active rows'
  // count for the left-out key)
  for (int k = t; k < K; k += kScanThreads) {
    const bool left_out = k == KA;
    for (int c0 = 0; c0 < G; c0 += 8) {
      int add[8], v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int c = c0 + u;
        add[u] = c < G ? (left_out ? active : gtot[(int64_t)(c / cpg) * KA + k]) : 0;
        v[u] = c < G ? hist[(int64_t)c * K + k] : 0;
      }
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (c0 + u < G) hist[(int64_t)(c0 + u) * K + k] = v[u] + add[u];
    }
  }
  // chunk offsets of row_ptr (the chunks are in row order)
  int rcarry = 0;
  for (int g0 = 0; g0 < G; g0 += kScanThreads) {
    const int g = g0 + t;
    const int v = g < G ? csum[g] : 0;
    int tot;
    const int ex = block_excl_scan(v, sh, &tot);
    if (g < G) csum[g] = rcarry + ex;
    rcarry += tot;
  }
  if (t == 0) {
    row_ptr[R] = rcarry;
    if (n_active != nullptr) *n_active = active;
  }
}

// The same when every key has a thread (nB + 2 <= 1024), a key's counts fit
// REGS registers (G <= REGS) and the group totals fit the LDS.  The counts
// are read once and each first slot written once.  The group totals sit in
// LDS as [group][active key] followed by [group] of the left-out key, so one
// exclusive scan in that order yields every group's start for every key (the
// left-out key's after all active rows), and a key's running count restarts
// at each group's first chunk for every key alike.
template <int REGS>
__global__ void __launch_bounds__(kScanThreads) sort_scan_fast_kernel(int R, int nB, int G, int cpg,
                                                                      int ngroups,
                                                                      int32_t *__restrict__ hist,
                                                                      int32_t *__restrict__ csum,
                                                                      int32_t *__restrict__ row_ptr,
                                                                      int32_t *__restrict__ n_active) {
  extern __shared__ int gt[];  // [ngroups][nB + 1], then [ngroups]
  __shared__ int sh[kSortWaves];
  const int t = threadIdx.x;
  const int K = nB + 2, KA = nB + 1;
  const int M = ngroups * KA;
  const bool on = t < K;
  // a key's total of group g at gt[slot0 + g * gstride]
  const int slot0 = t == KA ? M : t, gstride = t == KA ? 1 : KA;
  int pre[REGS];
  if (on) {
    int v[REGS];
#pragma unroll
    for (int u = 0; u < REGS; ++u) {  // branch-free: chunk G - 1 again past the last
      const int x = hist[(int64_t)min(u, G - 1) * K + t];
      v[u] = u < G ? x : 0;
    }
    int run = 0, j = 0, g = 0;
#pragma unroll
    for (int u = 0; u < REGS; ++u) {
      if (j == cpg && u < G) {
        gt[slot0 + g * gstride] = run;
        run = 0, j = 0, ++g;
      }
      pre[u] = run;
      run += v[u];
      ++j;
    }
    gt[slot0 + g * gstride] = run;
  }
  __syncthreads();
  {
    const int n = M + ngroups;
    const int per = (n + kScanThreads - 1) / kScanThreads;
    const int lo = min(n, per * t), hi = min(n, lo + per);
    int local = 0;
    for (int i = lo; i < hi; ++i) local += gt[i];
    int total;
    int run = block_excl_scan(local, sh, &total);  // ends with a barrier
    for (int i = lo; i < hi; ++i) {
      const int c = gt[i];
      gt[i] = run;
      run += c;
    }
  }
  __syncthreads();
  if (on) {
    int j = 0, g = 0;
    int off = gt[slot0];  // the key's start in group g
#pragma unroll
    for (int u = 0; u < REGS; ++u) {
      if (u < G) {
        if (j == cpg) {
          j = 0, ++g;
          off = gt[slot0 + g * gstride];
        }
        hist[(int64_t)u * K + t] = pre[u] + off;
        ++j;
      }
    }
  }
  int rcarry = 0;
  for (int g0 = 0; g0 < G; g0 += kScanThreads) {
    const int g = g0 + t;
    const int x = g < G ? csum[g] : 0;
    int tot;
    const int ex = block_excl_scan(x, sh, &tot);
    if (g < G) csum[g] = rcarry + ex;
    rcarry += tot;
  }
  if (t == 0) {
    row_ptr[R] = rcarry;
    if (n_active != nullptr) *n_active = gt[M];  // the left-out rows' start: all active rows
  }
}

template <class Fill>
__global__ void __launch_bounds__(kScanThreads) place_fill_kernel(const int32_t *__restrict__ len,
                                                                  Chunks ch, int nB, int G,
                                                                  const int32_t *__restrict__ base,
                                                                  const int32_t *__restrict__ coff,
                                                                  const int32_t *__restrict__ rloc,
                                                                  int32_t *__restrict__ row_ptr,
                                                                  int32_t *__restrict__ order,
                                                                  Fill fill) {
  extern __shared__ int wc[];  // (nB + 2) * kSortWaves per-wave counts, then slots
  const int t = threadIdx.x, lane = t & 63;
  const int w = __builtin_amdgcn_readfirstlane(t >> 6);
  const int K = nB + 2;
  if ((int)blockIdx.x >= G) {
    // a filling workgroup: nB + 2 ints of staging per wave
    fill(((int64_t)blockIdx.x - G) * kSortWaves + w, lane, wc + w * K);
    return;
  }
  const int c = blockIdx.x;
  for (int i = t; i < K * kSortWaves; i += kScanThreads) wc[i] = 0;
  __syncthreads();
  const int64_t r = ch.lo(c) + t;
  const bool on = r < ch.hi(c);
  const int key = on ? sort_key(len[r], nB) : 0;
  if (on) {
    atomicAdd(&wc[key * kSortWaves + w], 1);
    row_ptr[r] = coff[c] + rloc[r];
  }
  __syncthreads();
  for (int k = t; k < K; k += kScanThreads) {
    int run = base[(int64_t)c * K + k];
#pragma unroll
    for (int q = 0; q < kSortWaves; ++q) {
      const int n = wc[k * kSortWaves + q];
      wc[k * kSortWaves + q] = run;
      run += n;
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
  if (on) order[wc[key * kSortWaves + w] + __popcll(m & ((1ull << lane) - 1ull))] = (int32_t)r;
}

}  // namespace

hipError_t launch_merge(uint8_t *mask, int B, int H, int nB, const uint8_t *rows,
                        const uint8_t *cols, hipStream_t s) {
  const int64_t total = (int64_t)B * H * nB * nB;  // < 2^31 (the shape check)
  const bool vec = reinterpret_cast<uintptr_t>(mask) % 16 == 0;
  const int64_t threads = (total + 15) / 16;
  hipLaunchKernelGGL(merge_kernel, dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, s, mask, H,
                     nB, (int)total, vec, rows, cols);
  return hipGetLastError();
}

int order_group_heads(int heads, int64_t N, int d) {
  const int64_t per = 2 * N * d * (int64_t)sizeof(uint16_t);  // K and V of one head
  int64_t g = per > 0 ? kOrderGroupBytes / per : heads;
  const int64_t least = (heads + 62) / 63;  // at most 63 groups
  g = g < 1 ? 1 : g;
  g = g < least ? least : g;
  return g >= heads ? heads : (int)g;
}

// The chunks of R rows in groups of group_rows (>= R or <= 0: one group).
static Chunks make_chunks(int64_t R, int64_t group_rows) {
  const int64_t gr = (group_rows <= 0 || group_rows >= R) ? (R > 0 ? R : 1) : group_rows;
  return Chunks{R, gr, (int)((gr + kChunk - 1) / kChunk)};
}
static int n_groups(const Chunks &ch) { return (int)((ch.R + ch.gr - 1) / ch.gr); }

// LDS of the single-pass scan's group totals.
constexpr size_t kScanFastLds = 128 * 1024;

// At most 63 groups, each adding at most one partial chunk (the launch counts
// the last group's chunks only as far as its rows reach).
static int64_t max_chunks(int64_t R) { return (R + kChunk - 1) / kChunk + 63; }

// The list lengths, then the chunk histograms (key offsets after the scan),
// the chunk length sums (chunk offsets after the scan), the in-chunk
// prefixes of the lengths and the per-group key totals (sized for any
// grouping of the heads).
size_t compact_scratch_bytes(int64_t R, int nB) {
  if (R <= 0) return 0;
  const int64_t G = max_chunks(R);
  return 2 * align_up((size_t)R * sizeof(int32_t)) + align_up((size_t)(nB + 2) * G * sizeof(int32_t)) +
         align_up((size_t)G * sizeof(int32_t)) + align_up((size_t)63 * (nB + 1) * sizeof(int32_t));
}

// row_ptr and order from the list lengths, then col_idx by `fill` (built by
// make_fill from the chunk offsets, the in-chunk prefixes and the chunks);
// sort_scratch: the part of compact_scratch_bytes after the lengths.
template <class MakeFill>
static hipError_t launch_sort_fill(const int32_t *len, int64_t R, int nB, int32_t *row_ptr,
                                   int32_t *order, int32_t *n_active, void *sort_scratch,
                                   int64_t group_rows, const MakeFill &make_fill, hipStream_t s) {
  if (R < 1) return hipErrorInvalidValue;  // G >= 1 below
  const Chunks ch = make_chunks(R, group_rows);
  const int ngroups = n_groups(ch);
  if (ngroups > 63) return hipErrorInvalidValue;
  // every group's chunks, the last group's only as far as its rows reach
  const int64_t last = R - (int64_t)(ngroups - 1) * ch.gr;
  const int G = (ngroups - 1) * ch.cpg + (int)((last + kChunk - 1) / kChunk);
  const int K = nB + 2;
  const int64_t Gmax = max_chunks(R);
  char *p = static_cast<char *>(sort_scratch);
  int32_t *hist = reinterpret_cast<int32_t *>(p);
  p += align_up((size_t)K * Gmax * sizeof(int32_t));
  int32_t *csum = reinterpret_cast<int32_t *>(p);
  p += align_up((size_t)Gmax * sizeof(int32_t));
  int32_t *rloc = reinterpret_cast<int32_t *>(p);
  p += align_up((size_t)R * sizeof(int32_t));
  int32_t *gtot = reinterpret_cast<int32_t *>(p);
  const auto fill = make_fill(csum, rloc, ch);
  using Fill = std::decay_t<decltype(fill)>;
  const size_t hl = (size_t)K * sizeof(int32_t);
  const size_t pl = (size_t)K * kSortWaves * sizeof(int32_t);
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(&place_fill_kernel<Fill>),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)pl);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(sort_hist_kernel, dim3((unsigned)G), dim3(kScanThreads), hl, s, len, ch, nB, hist,
                     csum, rloc);
  const size_t gl = (size_t)ngroups * (nB + 2) * sizeof(int32_t);
  if (K <= kScanThreads && G <= 32 && gl <= kScanFastLds) {
    auto scan = G <= 4 ? sort_scan_fast_kernel<4> : G <= 8 ? sort_scan_fast_kernel<8>
              : G <= 16 ? sort_scan_fast_kernel<16> : sort_scan_fast_kernel<32>;
    if ((e = hipFuncSetAttribute(reinterpret_cast<const void *>(scan),
                                 hipFuncAttributeMaxDynamicSharedMemorySize, (int)gl)) != hipSuccess)
      return e;
    hipLaunchKernelGGL(scan, dim3(1), dim3(kScanThreads), gl, s, (int)R, nB, G, ch.cpg, ngroups, hist,
                       csum, row_ptr, n_active);
  } else {
    auto scan = G <= 4 ? sort_scan_kernel<4> : G <= 8 ? sort_scan_kernel<8> : G <= 16 ? sort_scan_kernel<16> : sort_scan_kernel<32>;
    hipLaunchKernelGGL(scan, dim3(1), dim3(kScanThreads), 0, s, (int)R, nB, G, ch.cpg, ngroups, hist, csum,
                       gtot, row_ptr, n_active);
  }
  const int64_t fill_groups = (R + kSortWaves - 1) / kSortWaves;
  hipLaunchKernelGGL(place_fill_kernel<Fill>, dim3((unsigned)(G + fill_groups)), dim3(kScanThreads),
                     pl, s, len, ch, nB, G, hist, csum, rloc, row_ptr, order, fill);
  return hipGetLastError();
}

hipError_t launch_compact(const uint8_t *mask, int64_t R, int nB, int64_t group_rows,
                          int32_t *row_ptr, int32_t *col_idx, int32_t *order, void *scratch,
                          hipStream_t s) {
  int32_t *len = static_cast<int32_t *>(scratch);
  void *sort_scratch = static_cast<char *>(scratch) + align_up((size_t)R * sizeof(int32_t));
  const unsigned g = (unsigned)((R + 3) / 4);
  // 16-byte chunks of a row: at most (15 + nB + 15) / 16 (nB <= 2048)
  const int nu = ((15 + nB + 15) / 16 + 63) / 64;
#define CARNATOR_COMPACT(NU)                                                                     \
  do {                                                                                           \
    hipLaunchKernelGGL(count_kernel<NU>, dim3(g), dim3(256), 0, s, mask, R, nB, len);            \
    return launch_sort_fill(len, R, nB, row_ptr, order, nullptr, sort_scratch, group_rows,       \
                            [&](const int32_t *coff, const int32_t *rloc, Chunks ch) {           \
                              return FillBytes<NU>{mask, R, nB, coff, rloc, ch, col_idx};        \
                            },                                                                   \
                            s);                                                                  \
  } while (0)
  if (nu <= 1) CARNATOR_COMPACT(1);
  else if (nu <= 2) CARNATOR_COMPACT(2);
  else CARNATOR_COMPACT(3);
#undef CARNATOR_COMPACT
}

#define CARNATOR_ROWS(KERNEL, ...)                                                         \
  do {                                                                                   \
    if (nc <= 4) hipLaunchKernelGGL(KERNEL<4>, dim3(g), dim3(256), 0, s, __VA_ARGS__);   \
    else if (nc <= 8) hipLaunchKernelGGL(KERNEL<8>, dim3(g), dim3(256), 0, s, __VA_ARGS__); \
    else if (nc <= 16) hipLaunchKernelGGL(KERNEL<16>, dim3(g), dim3(256), 0, s, __VA_ARGS__); \
    else hipLaunchKernelGGL(KERNEL<32>, dim3(g), dim3(256), 0, s, __VA_ARGS__);          \
  } while (0)

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

hipError_t launch_compact_bits(const uint64_t *bits, int B, int H, int nB, int64_t group_rows,
                               const uint8_t *rows, const uint8_t *cols, bool narrow, int32_t *row_ptr,
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
  return launch_sort_fill(len, R, nB, row_ptr, order, n_active,
                          static_cast<char *>(scratch) + align_up((size_t)R * sizeof(int32_t)), group_rows,
                          [&](const int32_t *coff, const int32_t *rloc, Chunks ch) {
                            return FillBits{bits, (int)R, nB, HnB, rows, colw, narrow, coff, rloc, ch, col_idx};
                          },
                          s);
}

}  // namespace carnator
