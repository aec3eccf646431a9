// Device-side preprocessing: degree sort and block-level partition
// (Sec. III-C "Degree Sorting" and "Block-level Partition", Alg. 1 and Alg. 2).
//
// Pipeline (all on one stream; the host reads back the maximum degree and the
// tail size, which decide between the two sorts, and the partition's summary,
// while the GPU keeps running). With W * Z >= 255 and a tail of at most
// kTailCap rows (the short sort):
//   k_degree        deg[i] = rowptr[i+1] - rowptr[i]; validates the row pointer;
//                   per-workgroup maximum degree, tail size, lower nonzeros and
//                   error flags; per-tile histograms of min(deg, 255); clears
//                   the error word and the scans' tickets; further workgroups
//                   check the column indices against n_cols (graphs of at most
//                   kEarlyCheckMaxNnz nonzeros)
//   scan            bin starts of every (digit, tile); its first tile also
//                   reduces k_degree's per-workgroup results (every input error
//                   is then known) and writes the maximum degree, the tail size
//                   and the lower nonzeros to the device and to pinned host
//                   memory (graphs whose scan takes several launches run k_dmax
//                   for that first, and the host reads the tail size before
//                   the scan)
//   k_scatter_low   stable scatter by min(deg, 255): rows of degree < 255 reach
//                   their final sorted place, with their sorted row pointer in
//                   closed form; the tail (degree >= 255) follows in row order
//   k_tail_relayout workgroup 0: the tail sorted by degree in LDS, its row
//                   pointers, the class starts, the segment scan of Alg. 2 and
//                   the summary with the host's done flag; the others: the
//                   sorted CSR of the rows below the tail
//   k_relayout_fill the partition's int4 entries {deg, loc, row, info} in
//                   Alg. 2's order, the first chunk of each hub row and the
//                   launch order (hub chunks, then the other entries heaviest
//                   first), side by side with the sorted CSR of the tail's rows;
//                   it may still run when agcn_plan_create returns
// The last two are queued without waiting for the read-back: they read the
// tail size from the device and return at once if it is over the cap. On a
// graph of more than kEarlyCheckMaxNnz nonzeros the relayout copies check the
// column indices instead of k_degree, and k_publish after k_relayout_fill sets
// the done flag.
// A graph of at most kTinyMaxRows rows and kTinyMaxNnz nonzeros instead runs
//   k_plan_tiny     one workgroup: the input checks, every row sorted by degree
//                   (the tail's code), row pointers, class starts, segment scan
//                   and summary with the done flag
//   k_relayout_fill as above, over the whole sorted CSR
// Otherwise (the multi-pass sort):
//   radix passes    stable LSD radix sort of row ids by degree, 8-bit digits:
//                   k_radix_hist -> exclusive scan -> k_radix_scatter. Buffers
//                   alternate so that the last pass writes the final
//                   (keys, perm) pair. Passes 0 and 1 are queued before the
//                   maximum degree is read back unless it is known already.
//   scan            rowptr_s = exclusive scan of the sorted degrees
//   k_relayout      sorted CSR copy
//   k_class_start   first sorted row of each degree class 0..deg_bound+1
//   k_seg_count     blocks per degree class / chunks per hub row
//   scan            entry offsets of every segment
//   k_partition_fill the entries, hub-row chunk offsets, launch order and summary
// Both: (host wait) entry counts read back; when hub rows are long, hub-chunk
// entries re-sorted into the order of a 16-bit key of their first column (two
// radix passes), then the other entries.
//
// The two read-backs (maximum degree, summary) are written by the kernels
// straight into pinned, host-coherent memory, each followed by a ready flag
// that the host polls, with no copy launched. Polling keeps event markers out
// of the stream (the GPU idles several microseconds around each) and avoids a
// blocking synchronisation's wake-up (about 30 us from the partition's last
// kernel to the next launch).
//
// Stability of the radix sort comes from giving each 64-lane wave a tile of
// consecutive rows that it walks in order, ranking equal digits inside a
// round with ballots; every count is an integer, so the result is exact.
//
// The warp-level plan of the ablation (Table II) has its own short pipeline:
// k_degree and k_dmax as above, k_wl_groups (groups per row), k_wl_copy (the
// CSR copied in input order, columns checked, identity permutation), a scan
// of the group counts, k_wl_fill (one {row, first nnz, count, 0} per group)
// and k_wl_summary.
#include <algorithm>
#include <chrono>
#include <climits>
#include <cstdlib>
#include <atomic>
#include <string>
#include <thread>

#include "agcn_internal.hpp"

namespace agcn {
namespace {

constexpr int kThreads = 256;

// Exclusive scan geometry.
constexpr int kScanItems = 16;
constexpr int kScanBlock = kThreads * kScanItems;  // 4096 elements per workgroup
constexpr int kScanTopThreads = 1024;
constexpr int kScanTopItems = 64;                   // <= 65536 partial sums
constexpr int64_t kScanMaxN = (int64_t)kScanBlock * kScanTopThreads * kScanTopItems;
constexpr int kScanChunkItems = 8;                  // single-workgroup scan: 8192 per chunk
constexpr int kScanChunk = kScanTopThreads * kScanChunkItems;
constexpr int64_t kScanSingleMax = 2 * kScanChunk;  // up to two chunks in one workgroup
constexpr int64_t kScanTwoPassMaxBlocks = 1024;     // reduce + down, partial prefix inline
constexpr int kMaxChainedScans = 16;                 // single-pass scans per plan (ticket counters)
constexpr unsigned kChainedMaxTiles = 64;            // single-pass scans: at most one look-back window

// Radix sort geometry: one wave owns kRadixTile consecutive rows.
constexpr int kRadixBins = 256;
constexpr int kRadixItems = 8;
constexpr int kRadixTile = 64 * kRadixItems;  // 512
constexpr int kRadixWaves = kThreads / 64;    // 4 tiles per workgroup

constexpr int kDegRows = kRadixTile * kRadixWaves;  // rows per k_degree workgroup

// Short sort: one 8-bit pass over min(degree, kTailKey) finishes every row of
// degree < kTailKey; the rows of degree >= kTailKey (the tail, in row order
// after that pass) are sorted by one workgroup holding them in LDS.
constexpr int kTailKey = 255;
constexpr int kTailThreads = 1024;
constexpr int kTailWaves = kTailThreads / 64;
constexpr int kTailItems = 16;
constexpr int32_t kTailCap = kTailThreads * kTailItems;  // 16384 rows

// Relayout tile (sorted nnz positions per workgroup).
constexpr int kRelayItems = 8;
constexpr int kRelayTile = kThreads * kRelayItems;  // 2048

// Launch-order sort of hub chunks: minimum mean chunks per hub row.
constexpr int kOrderMinChunks = 8;
constexpr int32_t kOrderMinTotalChunks = 32768;

__device__ inline bool failed(const uint32_t* err) { return err[0] != 0; }

// Radix passes the maximum degree needs (at least one).
__device__ inline int passes_needed(int32_t dmax) {
  const int bits = dmax > 0 ? 32 - __clz(dmax) : 0;
  return bits > 8 ? (bits + 7) / 8 : 1;
}

// A gated scan belongs to radix pass `pass` and is skipped with it.
__device__ inline bool gate_closed(const int32_t* dmax, int pass) {
  return dmax != nullptr && pass >= passes_needed(dmax[0]);
}

__device__ inline int32_t wave_sum(int32_t v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

__device__ inline int32_t wave_max(int32_t v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = max(v, __shfl_xor(v, o, 64));
  return v;
}

__device__ inline uint32_t wave_or(uint32_t v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v |= (uint32_t)__shfl_xor((int32_t)v, o, 64);
  return v;
}

// Inclusive scan over the 64 lanes of a wave with DPP row operations (no LDS
// round trip per step): prefixes of 4 lanes from three row shifts of the
// input, then of 8 and 16 lanes (row shifts by 4 and 8 on the upper banks of
// each 16-lane row), then across rows by broadcasting lane 15 into rows 1 and
// 3 and lane 31 into rows 2 and 3. Disabled or out-of-row lanes contribute 0,
// the identity of op (sums, and maxima of non-negative values).
template <typename Op>
__device__ inline int32_t wave_scan_dpp(int32_t v, Op op) {
  int32_t x = v;
  x = op(x, __builtin_amdgcn_update_dpp(0, v, 0x111, 0xf, 0xf, true));   // row_shr:1
  x = op(x, __builtin_amdgcn_update_dpp(0, v, 0x112, 0xf, 0xf, true));   // row_shr:2
  x = op(x, __builtin_amdgcn_update_dpp(0, v, 0x113, 0xf, 0xf, true));   // row_shr:3
  x = op(x, __builtin_amdgcn_update_dpp(0, x, 0x114, 0xf, 0xe, false));  // row_shr:4, banks 1-3
  x = op(x, __builtin_amdgcn_update_dpp(0, x, 0x118, 0xf, 0xc, false));  // row_shr:8, banks 2-3
  x = op(x, __builtin_amdgcn_update_dpp(0, x, 0x142, 0xa, 0xf, false));  // row_bcast:15, rows 1, 3
  x = op(x, __builtin_amdgcn_update_dpp(0, x, 0x143, 0xc, 0xf, false));  // row_bcast:31, rows 2, 3
  return x;
}

struct OpAdd {
  __device__ int32_t operator()(int32_t a, int32_t b) const { return a + b; }
};
struct OpMax {
  __device__ int32_t operator()(int32_t a, int32_t b) const { return max(a, b); }
};

// Inclusive scan over the 64 lanes of a wave.
__device__ inline int32_t wave_inclusive_scan(int32_t v, int lane) {
  (void)lane;
  return wave_scan_dpp(v, OpAdd());
}

// Exclusive scan across a workgroup of T threads; *total receives the sum.
// Ends with a barrier, so it may be called again right away.
template <int T>
__device__ inline int32_t block_exclusive_scan(int32_t v, int32_t* total) {
  __shared__ int32_t wsum[T / 64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int32_t inc = wave_inclusive_scan(v, lane);
  if (lane == 63) wsum[w] = inc;
  __syncthreads();
  if (w == 0) {
    const int32_t s = lane < T / 64 ? wsum[lane] : 0;
    const int32_t si = wave_inclusive_scan(s, lane);
    if (lane < T / 64) wsum[lane] = si;
  }
  __syncthreads();
  *total = wsum[T / 64 - 1];
  const int32_t r = (w > 0 ? wsum[w - 1] : 0) + inc - v;
  __syncthreads();
  return r;
}

// Lanes of the wave holding the same 8-bit digit (among valid lanes).
__device__ inline uint64_t match_digit(uint32_t digit, bool valid) {
  uint64_t m = __ballot(valid);
#pragma unroll
  for (int b = 0; b < 8; ++b) {
    const bool bit = (digit >> b) & 1u;
    const uint64_t bal = __ballot(bit);
    m &= bit ? bal : ~bal;
  }
  return m;
}

// As match_digit for a digit of `bits` <= 8 bits.
__device__ inline uint64_t match_bits(uint32_t digit, bool valid, int bits) {
  uint64_t m = __ballot(valid);
#pragma unroll
  for (int b = 0; b < 8; ++b) {
    if (b < bits) {
      const bool bit = (digit >> b) & 1u;
      const uint64_t bal = __ballot(bit);
      m &= bit ? bal : ~bal;
    }
  }
  return m;
}

// Alg. 1 for one degree: the smallest factor f of W with f * Z >= d gives
// block_rows = W / f and warp_nzs = ceil(d / f); returned as
// warp_nzs << 16 | block_rows. Degree 0 gets W rows and warp_nzs 0.
__device__ inline int32_t pattern_of(int32_t d, int32_t W, int32_t Z) {
  if (d == 0) return W;
  for (int32_t f = (d + Z - 1) / Z; f <= W; ++f)  // f * Z >= d from the first f on
    if (W % f == 0) return (((d + f - 1) / f) << 16) | (W / f);
  return 0;  // d > W * Z: not a degree class
}

// ---------------------------------------------------------------------------

__global__ void k_set(int32_t* p, int32_t v) {
  if (threadIdx.x == 0 && blockIdx.x == 0) p[0] = v;
}

// Raises error flags from the host's side (fault injection for tests).
__global__ void k_raise(uint32_t* err, uint32_t bits) {
  if (threadIdx.x == 0 && blockIdx.x == 0) atomicOr(err, bits);
}

// For the short sort of a graph of at most kEarlyCheckMaxNnz nonzeros, the
// column indices are checked against n_cols by workgroups that k_degree
// carries past its own, so that every input error is known when the tail's
// workgroup publishes the summary, before the last relayout: chunk c of the
// input's colidx per workgroup, chunks a multiple of this many entries.
// (Split between k_degree and k_scatter_low, the check cost more in all.)
// Otherwise the relayout copies check them.
constexpr int kColCheckItems = 8;
constexpr int64_t kColCheckChunk = (int64_t)kThreads * kColCheckItems * 8;  // 16384
constexpr int32_t kColCheckMaxBlocks = 2048;
// Largest graph whose columns k_degree checks (about 4 us of the plan at
// 11.4 M nonzeros, and growing with them, against the host latency that the
// early summary hides).
constexpr int64_t kEarlyCheckMaxNnz = int64_t(1) << 24;

struct ColumnCheck {
  const int32_t* colidx;
  int64_t nnz, chunk;
  int32_t n_cols;
  int32_t c0;  // first chunk
};

// Error flag (kErrColumn or 0) of chunk c0 + c, by one workgroup of kThreads
// (the result in thread 0).
__device__ inline uint32_t check_chunk(const ColumnCheck& cc, int32_t c) {
  __shared__ uint32_t s_bad[kThreads / 64];
  const int64_t lo = (int64_t)(cc.c0 + c) * cc.chunk;
  const int64_t hi = lo + cc.chunk < cc.nnz ? lo + cc.chunk : cc.nnz;
  uint32_t bad = 0;
  for (int64_t i = lo + threadIdx.x; i < hi; i += (int64_t)kThreads * kColCheckItems) {
    int32_t col[kColCheckItems];
#pragma unroll
    for (int u = 0; u < kColCheckItems; ++u) {
      const int64_t k = i + (int64_t)u * kThreads;
      col[u] = k < hi ? cc.colidx[k] : 0;
    }
#pragma unroll
    for (int u = 0; u < kColCheckItems; ++u)
      bad |= (uint32_t)col[u] >= (uint32_t)cc.n_cols ? kErrColumn : 0u;
  }
  bad = wave_or(bad);
  if ((threadIdx.x & 63) == 0) s_bad[threadIdx.x >> 6] = bad;
  __syncthreads();
  uint32_t f = 0;
  if (threadIdx.x == 0)
    for (int w = 0; w < kThreads / 64; ++w) f |= s_bad[w];
  return f;
}

// Step (1) of the degree sort, plus the input checks. Workgroups [0, nb)
// cover kDegRows rows each, each wave the kRadixTile consecutive rows of one
// radix tile, and write: the degrees; the workgroup's maximum degree, error
// flags and number of rows of degree >= kTailKey; and, when `counts` is given,
// each tile's histogram of min(degree, kTailKey) in the digit-major layout of
// k_radix_hist (the counts of the first pass of the short sort). Workgroup
// nb + c checks the column indices of chunk c and writes its flag to
// block_err[nb + c], which the reduction of the per-workgroup results reads.
__global__ __launch_bounds__(kThreads) void k_degree(int32_t n, int64_t nnz,
                                                     const int32_t* __restrict__ rowptr,
                                                     int32_t* __restrict__ deg,
                                                     int32_t* __restrict__ block_max,
                                                     uint32_t* __restrict__ block_err,
                                                     int32_t* __restrict__ block_tail,
                                                     int32_t* __restrict__ block_low,
                                                     int32_t* __restrict__ counts, int32_t n_tiles,
                                                     uint32_t* err_init, int32_t* tickets_init,
                                                     int32_t nb, ColumnCheck cc) {
  if ((int32_t)blockIdx.x >= nb) {  // uniform per workgroup
    const uint32_t f = check_chunk(cc, blockIdx.x - nb);
    if (threadIdx.x == 0) block_err[blockIdx.x] = f;
    return;
  }
  __shared__ int32_t s_max[kRadixWaves], s_tail[kRadixWaves], s_low[kRadixWaves];
  // The error word and the scans' ticket counters start at zero for the
  // kernels after this one (when no k_dmax follows to do it).
  if (blockIdx.x == 0 && err_init != nullptr) {
    if (threadIdx.x == 0) err_init[0] = 0;
    if (threadIdx.x < kMaxChainedScans) tickets_init[threadIdx.x] = 0;
  }
  __shared__ uint32_t s_err[kRadixWaves];
  __shared__ int32_t cnt[kRadixWaves][kRadixBins];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t tile = (int64_t)blockIdx.x * kRadixWaves + wave;
  const int64_t base = tile * kRadixTile;
  if (counts)
    for (int d = lane; d < kRadixBins; d += 64) cnt[wave][d] = 0;
  uint32_t e = 0;
  int32_t m = 0, tail = 0, low = 0;
#pragma unroll
  for (int j = 0; j < kRadixItems; ++j) {
    const int64_t i = base + (int64_t)j * 64 + lane;
    const bool valid = i < n;
    int32_t d = 0;
    if (valid) {
      const int32_t a = rowptr[i], b = rowptr[i + 1];
      d = b - a;
      if (a < 0 || b < a || (int64_t)b > nnz) {
        e |= kErrRowptrOrder;
        d = 0;
      }
      if (i == 0 && a != 0) e |= kErrRowptrStart;
      if (i == n - 1 && (int64_t)b != nnz) e |= kErrRowptrEnd;
      deg[i] = d;
    }
    m = max(m, d);
    tail += d >= kTailKey;
    low += d < kTailKey ? d : 0;
    if (counts && valid) atomicAdd(&cnt[wave][min(d, kTailKey)], 1);  // counts only: any order
  }
  if (counts && tile < n_tiles)
    for (int d = lane; d < kRadixBins; d += 64) counts[(int64_t)d * n_tiles + tile] = cnt[wave][d];
  m = wave_max(m);
  tail = wave_sum(tail);
  low = wave_sum(low);
  e = wave_or(e);
  if (lane == 0) {
    s_max[wave] = m;
    s_tail[wave] = tail;
    s_low[wave] = low;
    s_err[wave] = e;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    int32_t t = 0, c = 0, l = 0;
    uint32_t f = 0;
    for (int w = 0; w < kRadixWaves; ++w) {
      t = max(t, s_max[w]);
      c += s_tail[w];
      l += s_low[w];
      f |= s_err[w];
    }
    block_max[blockIdx.x] = t;
    block_err[blockIdx.x] = f;
    block_tail[blockIdx.x] = c;
    block_low[blockIdx.x] = l;
  }
}

// Per-workgroup results of k_degree and where their reduction goes: the
// maximum degree, tail size and lower nonzeros to dmax[0], dmax[1], dmax[2]
// and to pinned host memory.
struct DegreeBlocks {
  const int32_t* block_max;
  const uint32_t* block_err;
  const int32_t* block_tail;
  const int32_t* block_low;
  int32_t nb;      // degree workgroups
  int32_t nb_err;  // error flags: nb, then one per column-check workgroup
  int32_t* dmax;
  uint32_t* err;
  PlanSummary* host_sum;
};

// Maximum of the per-workgroup maxima, sums of their tail-row counts and
// lower nonzeros, and OR of their error flags, by a workgroup of T threads;
// written to the plan (the error word by OR, as other workgroups of the
// calling kernel may raise flags meanwhile) and to pinned host memory,
// followed by the host's ready flag.
template <int T>
__device__ inline void reduce_degree_blocks(const DegreeBlocks& a) {
  __shared__ int32_t s_max[T / 64], s_tail[T / 64], s_low[T / 64];
  __shared__ uint32_t s_err[T / 64];
  int32_t m = 0, c = 0, l = 0;
  uint32_t e = 0;
  for (int32_t i = threadIdx.x; i < a.nb; i += T) {
    m = max(m, a.block_max[i]);
    c += a.block_tail[i];
    l += a.block_low[i];
  }
  for (int32_t i = threadIdx.x; i < a.nb_err; i += T) e |= a.block_err[i];
  m = wave_max(m);
  c = wave_sum(c);
  l = wave_sum(l);
  e = wave_or(e);
  if ((threadIdx.x & 63) == 0) {
    s_max[threadIdx.x >> 6] = m;
    s_tail[threadIdx.x >> 6] = c;
    s_low[threadIdx.x >> 6] = l;
    s_err[threadIdx.x >> 6] = e;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    int32_t t = 0, tc = 0, tl = 0;
    uint32_t f = 0;
    for (int w = 0; w < T / 64; ++w) {
      t = max(t, s_max[w]);
      tc += s_tail[w];
      tl += s_low[w];
      f |= s_err[w];
    }
    a.dmax[0] = t;
    a.dmax[1] = tc;
    a.dmax[2] = tl;
    if (f) atomicOr(a.err, f);
    a.host_sum->max_deg = t;
    a.host_sum->n_tail = tc;
    a.host_sum->nnz_low = tl;
    __threadfence_system();
    a.host_sum->dmax_ready = 1;
    __threadfence_system();
  }
}

// The reduction in a kernel of its own (one workgroup of kScanTopThreads). It
// is the first writer of the plan's error word and maximum degree (nb = 0:
// both become 0) when k_degree did not clear them, and clears the scans'
// ticket counters.
__global__ __launch_bounds__(kScanTopThreads) void k_dmax(DegreeBlocks a, int32_t* tickets) {
  if (tickets && threadIdx.x < kMaxChainedScans) tickets[threadIdx.x] = 0;  // the plan's scans
  if (threadIdx.x == 0) a.err[0] = 0;
  __syncthreads();
  reduce_degree_blocks<kScanTopThreads>(a);
}

// Buffers of the radix passes: pass p (if it runs) writes slot (need - 1 - p) % 2
// of (keys, ids), slot 0 being the final (keys, perm); pass 0 reads the
// degrees in row order.
struct RadixBufs {
  const int32_t* deg;
  int32_t* keys[2];
  int32_t* ids[2];
};

// Digit histogram of each wave tile; counts are stored digit-major so that one
// exclusive scan yields every (digit, tile) start position.
__global__ __launch_bounds__(kThreads) void k_radix_hist(int32_t n, RadixBufs bufs, int pass,
                                                         int32_t* __restrict__ counts,
                                                         int32_t n_tiles, const uint32_t* err,
                                                         const int32_t* dmax) {
  if (failed(err)) return;
  const int need = passes_needed(dmax[0]);
  if (pass >= need) return;
  const int32_t* keys = pass == 0 ? bufs.deg : bufs.keys[(need - pass) & 1];
  const int shift = 8 * pass;
  __shared__ int32_t cnt[kRadixWaves][kRadixBins];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t tile = (int64_t)blockIdx.x * kRadixWaves + wave;
  if (tile >= n_tiles) return;  // uniform per wave; no workgroup barrier below
  for (int d = lane; d < kRadixBins; d += 64) cnt[wave][d] = 0;
  const int64_t base = tile * kRadixTile;
  int32_t k[kRadixItems];
#pragma unroll
  for (int j = 0; j < kRadixItems; ++j) {
    const int64_t i = base + (int64_t)j * 64 + lane;
    k[j] = i < n ? keys[i] : 0;
  }
#pragma unroll
  for (int j = 0; j < kRadixItems; ++j) {
    const bool valid = base + (int64_t)j * 64 + lane < n;
    const uint32_t digit = (((uint32_t)k[j]) >> shift) & 0xFFu;
    if (valid) atomicAdd(&cnt[wave][digit], 1);  // counts only: any order
  }
  for (int d = lane; d < kRadixBins; d += 64) counts[(int64_t)d * n_tiles + tile] = cnt[wave][d];
}

// Stable scatter: a row's new position is its (digit, tile) start plus the
// number of earlier rows of the tile with the same digit.
__global__ __launch_bounds__(kThreads) void k_radix_scatter(int32_t n, RadixBufs bufs, int pass,
                                                            const int32_t* __restrict__ offsets,
                                                            int32_t n_tiles, const uint32_t* err,
                                                            const int32_t* dmax) {
  if (failed(err)) return;
  const int need = passes_needed(dmax[0]);
  if (pass >= need) return;
  const int out = (need - 1 - pass) & 1;
  const int32_t* keys_in = pass == 0 ? bufs.deg : bufs.keys[out ^ 1];
  const int32_t* ids_in = pass == 0 ? nullptr : bufs.ids[out ^ 1];
  int32_t* __restrict__ keys_out = bufs.keys[out];
  int32_t* __restrict__ ids_out = bufs.ids[out];
  const int shift = 8 * pass;
  __shared__ int32_t start[kRadixWaves][kRadixBins];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t tile = (int64_t)blockIdx.x * kRadixWaves + wave;
  if (tile >= n_tiles) return;
  for (int d = lane; d < kRadixBins; d += 64) start[wave][d] = offsets[(int64_t)d * n_tiles + tile];
  const int64_t base = tile * kRadixTile;
  int32_t k[kRadixItems], id[kRadixItems];
#pragma unroll
  for (int j = 0; j < kRadixItems; ++j) {
    const int64_t i = base + (int64_t)j * 64 + lane;
    k[j] = i < n ? keys_in[i] : 0;
    id[j] = i < n ? (ids_in ? ids_in[i] : (int32_t)i) : 0;
  }
#pragma unroll
  for (int j = 0; j < kRadixItems; ++j) {
    const bool valid = base + (int64_t)j * 64 + lane < n;
    const uint32_t digit = (((uint32_t)k[j]) >> shift) & 0xFFu;
    const uint64_t peers = match_digit(digit, valid);
    const int32_t rank = (int32_t)__popcll(peers & __lanemask_lt());
    // All lanes read the digit's start before its single writer advances it
    // (LDS operations of one wave complete in program order).
    const int32_t pos = start[wave][digit] + rank;
    if (valid) {
      keys_out[pos] = k[j];
      ids_out[pos] = id[j];
    }
    if (valid && rank == 0) start[wave][digit] += __popcll(peers);
  }
}

// First pass of the short sort: a stable scatter by min(degree, kTailKey),
// the counts of k_degree scanned in `offsets`. A row of degree d < kTailKey is
// then in its final place, and so is its sorted row pointer: with R[d] the
// rows and NZ[d] the nonzeros of all degrees below d, the rows of degree d
// occupy positions R[d] + k and start at NZ[d] + k * d. The tail rows go to
// positions [n - m, n) of (tail_keys, tail_ids) in row order.
__global__ __launch_bounds__(kThreads) void k_scatter_low(
    int32_t n, const int32_t* __restrict__ deg, const int32_t* __restrict__ offsets, int32_t n_tiles,
    int32_t* __restrict__ keys, int32_t* __restrict__ perm, int32_t* __restrict__ rowptr_s,
    int32_t* __restrict__ tail_keys, int32_t* __restrict__ tail_ids, const uint32_t* err) {
  if (failed(err)) return;
  __shared__ int32_t start[kRadixWaves][kRadixBins];
  __shared__ int32_t s_r[kRadixBins + 1], s_nz[kRadixBins];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  {
    const int d = threadIdx.x;  // kThreads == kRadixBins
    s_r[d] = offsets[(int64_t)d * n_tiles];
    if (d == 0) s_r[kRadixBins] = n;
    __syncthreads();
    // Rows of degree d < kTailKey times d; the tail's term is not needed.
    const int32_t v = d < kTailKey ? (s_r[d + 1] - s_r[d]) * d : 0;
    int32_t total;
    s_nz[d] = block_exclusive_scan<kThreads>(v, &total);
    __syncthreads();
    // The tail's first row pointer closes the rows below it.
    if (blockIdx.x == 0 && d == kTailKey) rowptr_s[s_r[kTailKey]] = s_nz[kTailKey];
  }
  const int64_t tile = (int64_t)blockIdx.x * kRadixWaves + wave;
  if (tile >= n_tiles) return;  // uniform per wave; no workgroup barrier below
  for (int d = lane; d < kRadixBins; d += 64) start[wave][d] = offsets[(int64_t)d * n_tiles + tile];
  const int64_t base = tile * kRadixTile;
  int32_t k[kRadixItems];
#pragma unroll
  for (int j = 0; j < kRadixItems; ++j) {
    const int64_t i = base + (int64_t)j * 64 + lane;
    k[j] = i < n ? deg[i] : 0;
  }
#pragma unroll
  for (int j = 0; j < kRadixItems; ++j) {
    const int64_t i = base + (int64_t)j * 64 + lane;
    const bool valid = i < n;
    const uint32_t key = (uint32_t)min(k[j], kTailKey);
    const uint64_t peers = match_digit(key, valid);
    const int32_t rank = (int32_t)__popcll(peers & __lanemask_lt());
    const int32_t pos = start[wave][key] + rank;
    if (valid) {
      if (key < (uint32_t)kTailKey) {
        keys[pos] = k[j];
        perm[pos] = (int32_t)i;
        rowptr_s[pos] = s_nz[key] + (pos - s_r[key]) * (int32_t)key;
      } else {
        tail_keys[pos] = k[j];
        tail_ids[pos] = (int32_t)i;
      }
    }
    if (valid && rank == 0) start[wave][key] += __popcll(peers);
  }
}

// What the tail's workgroup leaves for k_relayout_fill: the number of
// partition segments (degree classes 0..DB and one per hub row).
struct TailInfo {
  int32_t n_segments;
};

// The short sort's second half as the reduction of k_degree's results
// decides it, read on the device, so that its launches need no read-back.
struct TailShape {
  bool take;         // the tail fits: these launches sort it (else they return at once)
  int32_t m, T0;     // tail rows; its first sorted position
  int32_t passes, width;  // LSD passes over degree - kTailKey
  int64_t nnz_low;   // nonzeros of the rows below the tail
};

__device__ inline TailShape tail_shape(const int32_t* dmax, int32_t n, int32_t cap) {
  TailShape s;
  s.m = dmax[1];
  s.nnz_low = dmax[2];
  s.take = s.m >= 0 && s.m <= cap && s.m <= kTailCap;
  s.T0 = n - s.m;
  int bits = 0;
  while (bits < 31 && (int64_t(1) << bits) <= (int64_t)dmax[0] - kTailKey) ++bits;
  s.passes = (bits + 7) / 8;
  s.width = s.passes > 0 ? (bits + s.passes - 1) / s.passes : 8;
  return s;
}

// --- exclusive scan of int32 -------------------------------------------------

// Phase 1: one total per block of kScanBlock values.
__global__ __launch_bounds__(kThreads) void k_scan_reduce(const int32_t* __restrict__ in, int64_t n,
                                                          int32_t* __restrict__ partials,
                                                          const uint32_t* err, const int32_t* gate,
                                                          int gate_pass) {
  if (failed(err) || gate_closed(gate, gate_pass)) return;
  __shared__ int32_t ws[kThreads / 64];
  const int64_t base = (int64_t)blockIdx.x * kScanBlock;
  int32_t s = 0;
#pragma unroll
  for (int k = 0; k < kScanItems; ++k) {
    const int64_t i = base + (int64_t)k * kThreads + threadIdx.x;
    if (i < n) s += in[i];
  }
  s = wave_sum(s);
  if ((threadIdx.x & 63) == 0) ws[threadIdx.x >> 6] = s;
  __syncthreads();
  if (threadIdx.x == 0) {
    int32_t t = 0;
    for (int w = 0; w < kThreads / 64; ++w) t += ws[w];
    partials[blockIdx.x] = t;
  }
}

// Phase 2 (many blocks only): exclusive scan of the block totals in place.
__global__ __launch_bounds__(kScanTopThreads) void k_scan_top(int32_t* __restrict__ partials,
                                                              int32_t m, int32_t* total_out,
                                                              const uint32_t* err,
                                                              const int32_t* gate, int gate_pass) {
  if (failed(err) || gate_closed(gate, gate_pass)) return;
  const int64_t b0 = (int64_t)threadIdx.x * kScanTopItems;
  int32_t s = 0;
  for (int k = 0; k < kScanTopItems; ++k)
    if (b0 + k < m) s += partials[b0 + k];
  int32_t total;
  int32_t run = block_exclusive_scan<kScanTopThreads>(s, &total);
  for (int k = 0; k < kScanTopItems; ++k) {
    if (b0 + k < m) {
      const int32_t v = partials[b0 + k];
      partials[b0 + k] = run;
      run += v;
    }
  }
  if (threadIdx.x == 0 && total_out) total_out[0] = total;
}

// Last phase. With `inline_prefix` the block adds up the totals of the blocks
// before it itself (partials hold raw totals; few blocks), and the last block
// writes the grand total; otherwise partials already hold exclusive offsets.
__global__ __launch_bounds__(kThreads) void k_scan_down(const int32_t* __restrict__ in, int64_t n,
                                                        const int32_t* __restrict__ partials,
                                                        int32_t* __restrict__ out, int32_t* total_out,
                                                        int inline_prefix, const uint32_t* err,
                                                        const int32_t* gate, int gate_pass) {
  if (failed(err) || gate_closed(gate, gate_pass)) return;
  __shared__ int32_t s_base;
  if (inline_prefix) {
    if (threadIdx.x < 64) {
      int32_t s = 0;
      for (int b = threadIdx.x; b < (int)blockIdx.x; b += 64) s += partials[b];
      s = wave_sum(s);
      if (threadIdx.x == 0) s_base = s;
    }
  } else if (threadIdx.x == 0) {
    s_base = partials[blockIdx.x];
  }
  // Coalesced load into registers, thread-contiguous ownership through LDS.
  __shared__ int32_t tile[kScanBlock + kScanBlock / 32];
  const int64_t base = (int64_t)blockIdx.x * kScanBlock;
#pragma unroll
  for (int k = 0; k < kScanItems; ++k) {
    const int j = k * kThreads + threadIdx.x;
    const int64_t i = base + j;
    tile[j + (j >> 5)] = i < n ? in[i] : 0;
  }
  __syncthreads();
  int32_t v[kScanItems];
  int32_t s = 0;
#pragma unroll
  for (int k = 0; k < kScanItems; ++k) {
    const int j = threadIdx.x * kScanItems + k;
    v[k] = tile[j + (j >> 5)];
    s += v[k];
  }
  int32_t total;
  int32_t run = block_exclusive_scan<kThreads>(s, &total) + s_base;
#pragma unroll
  for (int k = 0; k < kScanItems; ++k) {
    const int j = threadIdx.x * kScanItems + k;
    tile[j + (j >> 5)] = run;
    run += v[k];
  }
  __syncthreads();
#pragma unroll
  for (int k = 0; k < kScanItems; ++k) {
    const int j = k * kThreads + threadIdx.x;
    const int64_t i = base + j;
    if (i < n) out[i] = tile[j + (j >> 5)];
  }
  if (inline_prefix && total_out && blockIdx.x == gridDim.x - 1 && threadIdx.x == 0)
    total_out[0] = s_base + total;
}

// Single-pass scan (decoupled look-back). Workgroups take tiles in the order
// of a ticket counter, so every tile's predecessors started before it. Each
// tile publishes its sum (state 1) as soon as it has it, then its inclusive
// prefix (state 2); a tile's prefix is the sum of the predecessors' words
// back to the nearest state-2 one, read 64 at a time by one wave. A status
// word is state (2 bits) | epoch (30 bits) | value (32 bits); the epoch is
// new for every scan, so words left by earlier scans read as not ready and
// the status array needs no clearing. The wait is bounded; running out of it
// raises the internal-error flag instead of hanging.
// The status word is the only data one workgroup reads from another, and it
// carries its value, so its loads and stores are relaxed device-scope atomics
// (coherent past the per-XCD L2s): acquire and release would add an L2
// invalidate to every poll and an L2 write-back to every publish.
constexpr uint32_t kLookBackSpins = 1u << 22;

__device__ inline void publish(unsigned long long* w, uint32_t state, uint32_t epoch, int32_t v) {
  const unsigned long long x = ((unsigned long long)state << 62) |
                               ((unsigned long long)(epoch & 0x3FFFFFFFu) << 32) | (uint32_t)v;
  __hip_atomic_store(w, x, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__global__ __launch_bounds__(kThreads) void k_scan_chained(
    const int32_t* __restrict__ in, int64_t n, int32_t* __restrict__ out, int32_t* total_out,
    unsigned long long* status, int32_t* ticket, uint32_t epoch, uint32_t* err,
    const int32_t* gate, int gate_pass, DegreeBlocks db) {
  if (failed(err) || gate_closed(gate, gate_pass)) return;
  __shared__ int32_t tile[kScanBlock + kScanBlock / 32];
  __shared__ int32_t s_t, s_base;
  if (threadIdx.x == 0)
    s_t = __hip_atomic_fetch_add(ticket, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __syncthreads();
  const int32_t t = s_t;
  if (t >= (int32_t)gridDim.x) {  // the counter was not zeroed: never read past the status words
    if (threadIdx.x == 0) atomicOr(err, kErrInternal);
    return;
  }
  const int64_t base = (int64_t)t * kScanBlock;
#pragma unroll
  for (int k = 0; k < kScanItems; ++k) {
    const int j = k * kThreads + threadIdx.x;
    const int64_t i = base + j;
    tile[j + (j >> 5)] = i < n ? in[i] : 0;
  }
  __syncthreads();
  int32_t v[kScanItems];
  int32_t s = 0;
#pragma unroll
  for (int k = 0; k < kScanItems; ++k) {
    const int j = threadIdx.x * kScanItems + k;
    v[k] = tile[j + (j >> 5)];
    s += v[k];
  }
  int32_t total;
  int32_t run = block_exclusive_scan<kThreads>(s, &total);
  if (threadIdx.x < 64) {
    const int lane = threadIdx.x;
    if (lane == 0) publish(status + t, t == 0 ? 2u : 1u, epoch, total);
    int32_t prefix = 0;
    if (t > 0) {
      int64_t hi = (int64_t)t - 1;  // nearest predecessor not yet added
      uint32_t spins = 0;
      for (;;) {
        const int64_t j = hi - lane;
        uint32_t state = 0;
        int32_t val = 0;
        if (j >= 0) {
          const unsigned long long w = __hip_atomic_load(status + j, __ATOMIC_RELAXED,
                                                         __HIP_MEMORY_SCOPE_AGENT);
          if ((uint32_t)(w >> 32 & 0x3FFFFFFFu) == (epoch & 0x3FFFFFFFu)) state = (uint32_t)(w >> 62);
          val = (int32_t)(uint32_t)w;
        }
        const uint64_t pref = __ballot(j >= 0 && state == 2u);
        const uint64_t wait = __ballot(j >= 0 && state == 0u);
        // Lanes up to the nearest prefix (all 64 when there is none) are needed.
        const int first = pref ? __ffsll((long long)pref) - 1 : 64;
        const uint64_t need = first >= 63 ? ~0ull : ((2ull << first) - 1);
        if (wait & need) {
          if (++spins > kLookBackSpins) {
            if (lane == 0) atomicOr(err, kErrInternal);
            break;
          }
          __builtin_amdgcn_s_sleep(1);
          continue;
        }
        prefix += wave_sum(lane <= first && j >= 0 ? val : 0);
        if (first < 64) break;
        hi -= 64;
      }
      if (lane == 0) publish(status + t, 2u, epoch, prefix + total);
    }
    if (lane == 0) s_base = prefix;
  }
  __syncthreads();
  // With db given, the first tile (no look-back to wait for) also reduces
  // k_degree's per-workgroup results, in place of a k_dmax launch.
  if (t == 0 && db.dmax != nullptr) reduce_degree_blocks<kThreads>(db);
  run += s_base;
#pragma unroll
  for (int k = 0; k < kScanItems; ++k) {
    const int j = threadIdx.x * kScanItems + k;
    tile[j + (j >> 5)] = run;
    run += v[k];
  }
  __syncthreads();
#pragma unroll
  for (int k = 0; k < kScanItems; ++k) {
    const int j = k * kThreads + threadIdx.x;
    const int64_t i = base + j;
    if (i < n) out[i] = tile[j + (j >> 5)];
  }
  if (total_out && threadIdx.x == 0 && base + kScanBlock >= n) total_out[0] = s_base + total;
}

// One workgroup scans the whole array in chunks (n <= kScanSingleMax).
__global__ __launch_bounds__(kScanTopThreads) void k_scan_single(
    const int32_t* __restrict__ in, int32_t n, int32_t* __restrict__ out, int32_t* total_out,
    const uint32_t* err, const int32_t* gate, int gate_pass) {
  if (failed(err) || gate_closed(gate, gate_pass)) return;
  __shared__ int32_t tile[kScanChunk + kScanChunk / 32];
  int32_t carry = 0;
  for (int32_t c0 = 0; c0 < n; c0 += kScanChunk) {
#pragma unroll
    for (int k = 0; k < kScanChunkItems; ++k) {
      const int j = k * kScanTopThreads + threadIdx.x;
      tile[j + (j >> 5)] = c0 + j < n ? in[c0 + j] : 0;
    }
    __syncthreads();
    int32_t v[kScanChunkItems];
    int32_t s = 0;
#pragma unroll
    for (int k = 0; k < kScanChunkItems; ++k) {
      const int j = threadIdx.x * kScanChunkItems + k;
      v[k] = tile[j + (j >> 5)];
      s += v[k];
    }
    int32_t total;
    int32_t run = block_exclusive_scan<kScanTopThreads>(s, &total) + carry;
#pragma unroll
    for (int k = 0; k < kScanChunkItems; ++k) {
      const int j = threadIdx.x * kScanChunkItems + k;
      tile[j + (j >> 5)] = run;
      run += v[k];
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < kScanChunkItems; ++k) {
      const int j = k * kScanTopThreads + threadIdx.x;
      if (c0 + j < n) out[c0 + j] = tile[j + (j >> 5)];
    }
    carry += total;
    __syncthreads();
  }
  if (threadIdx.x == 0 && total_out) total_out[0] = carry;
}

// --- relayout (step (3) of the degree sort) ----------------------------------

// Largest r in [0, n) with rowptr_s[r] <= e (the row holding sorted nnz e),
// found by one whole wave: each step probes 64 evenly spaced rows and keeps
// the interval between the last probe <= e and the next, so a search over
// n rows takes about log64(n) dependent loads. Call with all 64 lanes.
__device__ inline int32_t wave_row_of(const int32_t* rowptr_s, int32_t n, int64_t e, int lane) {
  int32_t a = 0, b = n - 1;  // invariant: rowptr_s[a] <= e, answer in [a, b]
  while (b > a) {
    const int64_t span = (int64_t)b - a;
    const int32_t probe = a + (int32_t)((span * (lane + 1) + 63) / 64);  // in (a, b]
    const bool le = rowptr_s[probe] <= e;
    const uint64_t mask = __ballot(le);
    // Probes increase with the lane and rowptr_s is non-decreasing, so the
    // lanes with rowptr_s[probe] <= e form a prefix.
    const int k = __popcll(mask);  // number of probes <= e
    const int32_t na = k > 0 ? __shfl(probe, k - 1, 64) : a;
    const int32_t nb = k < 64 ? __shfl(probe, k, 64) - 1 : b;
    a = na;
    b = nb;
  }
  return a;
}

__device__ inline int rpad(int i) { return i + (i >> 5); }

// Each workgroup fills kRelayTile consecutive positions of the sorted CSR.
// Degree-0 rows sort first, so every row owning one of these positions is
// non-empty and at most kRelayTile rows (the "window") are involved. Each
// window row marks its first position; an inclusive max-scan of the marks
// then gives every position its row in O(1). Called by whole workgroups.
// Column indices are checked against check_cols (INT32_MAX when k_degree has
// checked them already).
// LDS of one relayout tile (int32 words), also lent to the tail's workgroup.
constexpr int kRelayLds = (kRelayTile + 1) + kRelayTile + (kRelayTile + kRelayTile / 32) +
                          kThreads / 64 + 2;

__device__ inline void relayout_tile(int64_t tile, bool active, int tid, int32_t n, int64_t nnz,
                                     int32_t check_cols, const int32_t* __restrict__ rowptr,
                                     const int32_t* __restrict__ colidx,
                                     const float* __restrict__ vals,
                                     const int32_t* __restrict__ perm,
                                     const int32_t* __restrict__ rowptr_s,
                                     int32_t* __restrict__ colidx_s, float* __restrict__ vals_s,
                                     uint32_t* err, int32_t* lds) {
  // kThreads threads (tid) work on the tile; several such groups of one
  // workgroup may each run a tile (or none: !active), meeting at the same
  // workgroup barriers.
  int32_t* s_ptr = lds;                        // rowptr_s over the window rows (+1 end)
  int32_t* s_src = s_ptr + kRelayTile + 1;     // first nnz of each window row in the input CSR
  int32_t* s_row = s_src + kRelayTile;         // window row of each position (padded)
  int32_t* s_wmax = s_row + kRelayTile + kRelayTile / 32;
  int32_t& s_lo = s_wmax[kThreads / 64];
  int32_t& s_hi = s_wmax[kThreads / 64 + 1];
  const int64_t e0 = tile * kRelayTile;
  const int64_t e1 = e0 + kRelayTile < nnz ? e0 + kRelayTile : nnz;
  if (active) {
    if (tid < 64) {
      const int32_t r = wave_row_of(rowptr_s, n, e0, tid);
      if (tid == 0) s_lo = r;
    } else if (tid < 128) {
      const int32_t r = wave_row_of(rowptr_s, n, e1 - 1, tid - 64);
      if (tid == 64) s_hi = r;
    }
    for (int k = tid; k < kRelayTile; k += kThreads) s_row[rpad(k)] = 0;
  }
  __syncthreads();
  const int32_t lo = active ? s_lo : 0;
  const int32_t nw = active ? s_hi - lo + 1 : 0;
  if (active && (nw > kRelayTile || nw < 1)) {  // cannot happen for a sorted row order
    if (tid == 0) atomicOr(err, kErrRelayout);
    active = false;
  }
  if (active) {
    for (int k = tid; k <= nw; k += kThreads) s_ptr[k] = rowptr_s[lo + k];
    for (int k = tid; k < nw; k += kThreads) s_src[k] = rowptr[perm[lo + k]];
  }
  __syncthreads();
  // Window rows 1..nw-1 start strictly inside the tile.
  for (int w = 1 + tid; w < nw; w += kThreads) s_row[rpad((int)(s_ptr[w] - e0))] = w;
  __syncthreads();
  // Inclusive max-scan of the marks; thread t owns positions 8t .. 8t+7.
  int32_t v[kRelayItems];
  int32_t m = 0;
#pragma unroll
  for (int k = 0; k < kRelayItems; ++k) {
    m = max(m, s_row[rpad(tid * kRelayItems + k)]);
    v[k] = m;
  }
  const int lane = tid & 63, wv = tid >> 6;
  const int32_t inc = wave_scan_dpp(m, OpMax());  // marks are >= 0
  if (lane == 63) s_wmax[wv] = inc;
  int32_t before = __shfl_up(inc, 1, 64);
  if (lane == 0) before = 0;
  __syncthreads();
  for (int w = 0; w < wv; ++w) before = max(before, s_wmax[w]);
#pragma unroll
  for (int k = 0; k < kRelayItems; ++k)
    s_row[rpad(tid * kRelayItems + k)] = max(before, v[k]);
  __syncthreads();
  if (!active) return;  // no barrier below
  uint32_t bad = 0;
#pragma unroll
  for (int k = 0; k < kRelayItems; ++k) {
    const int j = k * kThreads + tid;
    const int64_t e = e0 + j;
    if (e < e1) {
      const int32_t w = s_row[rpad(j)];
      const int64_t src = (int64_t)s_src[w] + (e - s_ptr[w]);
      const int32_t c = colidx[src];
      if ((uint32_t)c >= (uint32_t)check_cols) bad = kErrColumn;
      colidx_s[e] = c;
      vals_s[e] = vals[src];
    }
  }
  if (bad) atomicOr(err, bad);
}

// A run of the relayout: sorted positions [p0, p1) filled by one workgroup,
// in steps of kRelayTile positions. The rows of one step (its window, at most
// kRelayTile rows, all non-empty) are consecutive: the row of the step's
// first position, found once per run by a wave search and then carried from
// step to step, and the rows after it that start before the step's end. A
// step loads the window's row starts and permutation entries in rounds of
// kThreads rows until a start at or past the step's end shows up (one round
// unless the rows are short), then each window row's first nonzero in the
// input CSR, then copies its positions, each finding its row by binary
// lifting over the window's starts: three dependent global loads per step
// where relayout_tile takes six. n bounds the rows searched (rowptr_s[n] >= p1
// is final). Column indices are checked against check_cols (INT32_MAX when
// they were checked before). Called by whole workgroups of kThreads.
constexpr int kRelaySpanLds = 2 * (kRelayTile + 1) + kThreads / 64;

__device__ __forceinline__ void relay_span(int64_t p0, int64_t p1, int32_t n, int32_t check_cols,
                                           const int32_t* __restrict__ rowptr,
                                           const int32_t* __restrict__ colidx,
                                           const float* __restrict__ vals,
                                           const int32_t* __restrict__ perm,
                                           const int32_t* __restrict__ rowptr_s,
                                           int32_t* __restrict__ colidx_s,
                                           float* __restrict__ vals_s, uint32_t* err,
                                           int32_t* lds) {
  constexpr int G = kThreads, T = kRelayTile;
  int32_t* s_ptr = lds;            // window row starts, [0, T]
  int32_t* s_src = s_ptr + T + 1;  // window rows' permutation entries, then input starts
  int32_t* s_cnt = s_src + T + 1;  // per wave: rows of a round starting before the end
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  if (p0 >= p1) return;  // uniform over the workgroup
  if (tid < 64) {
    const int32_t r = wave_row_of(rowptr_s, n, p0, tid);
    if (tid == 0) s_cnt[0] = r;
  }
  __syncthreads();
  int32_t lo = s_cnt[0];
  uint32_t bad = 0;
  for (int64_t e0 = p0; e0 < p1; e0 += T) {
    // Positions as unsigned 32-bit values (nnz < 2^31; those past the step's
    // end, whose searches go unused, stay below 2^32).
    const uint32_t u0 = (uint32_t)e0, u1 = (uint32_t)(e0 + T < p1 ? e0 + T : p1);
    __syncthreads();  // the previous step's readers of the LDS are done
    // Window rows lo + k for k < K: those starting before the step's end u1.
    // The starts ascend, so the rows below u1 are a prefix; a round that is
    // not all below u1 holds the first start at or past it (s_ptr[K],
    // rowptr_s[n] at the latest). Rows past k = T or past n are never
    // counted, so the loop ends by round kRelayItems.
    int32_t K = 0;
    for (int c = 0;; ++c) {
      const int32_t k = c * G + tid;
      bool below = false;
      if (k <= T && (int64_t)lo + k <= n) {
        const int32_t v = rowptr_s[lo + k];
        const bool row = (int64_t)lo + k < n;  // else the end of the rows
        if (row) s_src[k] = perm[lo + k];
        s_ptr[k] = v;
        below = row && (uint32_t)v < u1;
      }
      const uint64_t m = __ballot(below);
      if (lane == 0) s_cnt[wv] = __popcll(m);
      __syncthreads();
      int32_t cnt = 0;
#pragma unroll
      for (int w = 0; w < G / 64; ++w) cnt += s_cnt[w];
      __syncthreads();
      K += cnt;
      if (cnt < G) break;
    }
    if (K < 1 || K > T) {  // cannot happen for a sorted row order (uniform)
      if (tid == 0) atomicOr(err, kErrRelayout);
      return;
    }
    // Each thread converts the permutation entries it loaded itself, all
    // loads issued before the first store.
    int32_t first[kRelayItems];
#pragma unroll
    for (int c = 0; c < kRelayItems; ++c)
      if (c * G + tid < K) first[c] = rowptr[s_src[c * G + tid]];
#pragma unroll
    for (int c = 0; c < kRelayItems; ++c)
      if (c * G + tid < K) s_src[c * G + tid] = first[c];
    __syncthreads();
    // Each position's row: the last window row starting at or before it; a
    // lifting step past the window probes its last row, which is then the
    // answer or stays unchosen. K is uniform, so every lane takes the same
    // steps, and the kRelayItems searches advance side by side.
    int32_t w[kRelayItems];
#pragma unroll
    for (int i = 0; i < kRelayItems; ++i) w[i] = 0;
    for (int32_t step = K > 1 ? 1 << (31 - __builtin_clz((uint32_t)(K - 1))) : 0; step > 0;
         step >>= 1) {
      int32_t v[kRelayItems], m[kRelayItems];
#pragma unroll
      for (int i = 0; i < kRelayItems; ++i) {
        m[i] = min(w[i] + step, K - 1);
        v[i] = s_ptr[m[i]];
      }
#pragma unroll
      for (int i = 0; i < kRelayItems; ++i)
        if ((uint32_t)v[i] <= u0 + i * G + tid) w[i] = m[i];
    }
    // Input positions (below nnz < 2^31 for the positions copied; unsigned,
    // so the unused ones past the step's end cannot overflow).
    uint32_t src[kRelayItems];
#pragma unroll
    for (int i = 0; i < kRelayItems; ++i)
      src[i] = (uint32_t)s_src[w[i]] + (u0 + i * G + tid - (uint32_t)s_ptr[w[i]]);
    int32_t cv[kRelayItems];
    float vv[kRelayItems];
#pragma unroll
    for (int i = 0; i < kRelayItems; ++i) {
      if (u0 + i * G + tid < u1) {
        cv[i] = colidx[src[i]];
        vv[i] = vals[src[i]];
      }
    }
#pragma unroll
    for (int i = 0; i < kRelayItems; ++i) {
      const uint32_t e = u0 + i * G + tid;
      if (e < u1) {
        if ((uint32_t)cv[i] >= (uint32_t)check_cols) bad = kErrColumn;
        colidx_s[e] = cv[i];
        vals_s[e] = vv[i];
      }
    }
    // The next step's first row: the row starting exactly at u1, if any, else
    // the window's last row.
    lo = (int64_t)lo + K < n && (uint32_t)s_ptr[K] == u1 ? lo + K : lo + K - 1;
  }
  if (bad) atomicOr(err, bad);
}

// The share [t_a, t_b) of part b out of parts of `tiles` relayout tiles
// (kRelayTile positions each), as sorted positions [p0, p1) clipped to end.
__device__ inline void relay_share(int64_t first_tile, int64_t tiles, int64_t b, int64_t parts,
                                   int64_t end, int64_t* p0, int64_t* p1) {
  const int64_t ta = first_tile + tiles * b / parts, tb = first_tile + tiles * (b + 1) / parts;
  *p0 = ta * kRelayTile < end ? ta * kRelayTile : end;
  *p1 = tb * kRelayTile < end ? tb * kRelayTile : end;
}

// The error word as one workgroup sees it, read once (other workgroups may
// raise flags meanwhile, and every thread must take the same branch).
__device__ inline bool block_failed(const uint32_t* err) {
  __shared__ uint32_t s_e;
  if (threadIdx.x == 0) s_e = err[0];
  __syncthreads();
  const bool f = s_e != 0;
  __syncthreads();
  return f;
}

// A tile's copy costs about as much per window row as per kRelayRowCost
// positions (a tile of short rows, 455 rows of 1-8 nonzeros, took twice as
// long as a tile inside one long row).
constexpr int64_t kRelayRowCost = 4;

// Start of part b of `parts` of the sorted positions when the parts share the
// cost of positions plus kRelayRowCost per row: the tile holding the start of
// the last row r with rowptr_s[r] + kRelayRowCost r <= b / parts of the total
// (rows [0, n], rowptr_s[n] = nnz). Non-decreasing in b; part 0 starts at 0,
// part `parts` at nnz. Called by one whole wave.
__device__ inline int64_t relay_cost_bound(const int32_t* rowptr_s, int32_t n, int64_t nnz,
                                           int64_t b, int64_t parts, int lane) {
  if (b <= 0) return 0;
  if (b >= parts) return nnz;
  const int64_t target = (nnz + kRelayRowCost * n) * b / parts;
  int32_t a = 0, c = n;  // invariant: cost(a) <= target, answer in [a, c]
  while (c > a) {
    const int64_t span = (int64_t)c - a;
    const int32_t probe = a + (int32_t)((span * (lane + 1) + 63) / 64);  // in (a, c]
    const bool le = (int64_t)rowptr_s[probe] + kRelayRowCost * probe <= target;
    const int k = __popcll(__ballot(le));  // the costs ascend: a prefix of the probes
    const int32_t na = k > 0 ? __shfl(probe, k - 1, 64) : a;
    const int32_t nc = k < 64 ? __shfl(probe, k, 64) - 1 : c;
    a = na;
    c = nc;
  }
  const int64_t pos = (int64_t)rowptr_s[a] / kRelayTile * kRelayTile;
  return pos < nnz ? pos : nnz;
}

// The multi-pass sort's relayout: workgroup b fills part b of the sorted
// positions, the parts sharing the copy's cost (whole tiles but the last).
__global__ __launch_bounds__(kThreads) void k_relayout(
    int32_t n, int64_t nnz, int32_t n_cols, const int32_t* __restrict__ rowptr,
    const int32_t* __restrict__ colidx, const float* __restrict__ vals,
    const int32_t* __restrict__ perm, const int32_t* __restrict__ rowptr_s,
    int32_t* __restrict__ colidx_s, float* __restrict__ vals_s, uint32_t* err) {
  __shared__ int32_t lds[kRelaySpanLds];
  __shared__ int64_t s_bound[2];
  if (block_failed(err)) return;
  const int w = threadIdx.x >> 6;
  if (w < 2) {
    const int64_t v =
        relay_cost_bound(rowptr_s, n, nnz, (int64_t)blockIdx.x + w, gridDim.x, threadIdx.x & 63);
    if ((threadIdx.x & 63) == 0) s_bound[w] = v;
  }
  __syncthreads();
  relay_span(s_bound[0], s_bound[1], n, n_cols, rowptr, colidx, vals, perm, rowptr_s, colidx_s,
             vals_s, err, lds);
}

// --- partition ---------------------------------------------------------------

// cls[d] = first sorted row whose degree is >= d, for d in [0, DB + 1] (n if none).
__global__ __launch_bounds__(kThreads) void k_class_start(int32_t n, const int32_t* __restrict__ deg_s,
                                                          int32_t DB, int32_t* __restrict__ cls,
                                                          const uint32_t* err) {
  if (failed(err)) return;
  const int64_t r = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (r > n) return;
  const int32_t prev = r == 0 ? -1 : deg_s[r - 1];
  const int32_t cur = r == n ? INT_MAX : deg_s[r];
  const int32_t hi = cur < DB + 1 ? cur : DB + 1;
  for (int32_t d = prev + 1; d <= hi; ++d) cls[d] = (int32_t)r;
}

// Segments: s <= DB is degree class s (ceil(count / block_rows) entries);
// s > DB is hub row s - DB - 1 in sorted order (ceil(deg / H) chunk entries).
__global__ __launch_bounds__(kThreads) void k_seg_count(int32_t n, const int32_t* __restrict__ deg_s,
                                                        const int32_t* __restrict__ cls, int32_t W,
                                                        int32_t Z, int32_t DB, int32_t H, int32_t S,
                                                        int32_t* __restrict__ nb,
                                                        const uint32_t* err) {
  if (failed(err)) return;
  const int64_t s = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (s >= S) return;
  int64_t v = 0;
  if (s <= DB) {
    const int64_t cnt = cls[s + 1] - cls[s];
    if (cnt > 0) {
      const int64_t br = pattern_of((int32_t)s, W, Z) & 0xFFFF;
      v = (cnt + br - 1) / br;
    }
  } else {
    const int64_t r = (int64_t)cls[DB + 1] + (s - DB - 1);
    if (r < n) v = ((int64_t)deg_s[r] + H - 1) / H;
  }
  nb[s] = (int32_t)v;
}

// The partition's outputs from the segment offsets and class starts (S
// segments, seg_off[S] the entry count), for threads t0, t0 + stride, ...:
//   - Alg. 2's entries, each from its segment;
//   - the first chunk of each hub row;
//   - the SpMM launch order: hub chunks, then the other entries heaviest
//     first (rewritten after the host has read the summary when hub chunks are
//     launched in column order; it never changes a result).
__device__ inline void fill_partition(int64_t t0, int64_t stride, int32_t n,
                                      const int32_t* __restrict__ rowptr_s,
                                      const int32_t* __restrict__ deg_s,
                                      const int32_t* __restrict__ cls,
                                      const int32_t* __restrict__ seg_off, int32_t S, int32_t W,
                                      int32_t Z, int32_t DB, int32_t H, int4* __restrict__ meta,
                                      int64_t cap, int32_t hub_ub,
                                      int32_t* __restrict__ hub_chunk_off,
                                      int32_t* __restrict__ order) {
  const int32_t total = seg_off[S];
  const int32_t hub_first_entry = seg_off[DB + 1];
  const int32_t first_hub_row = cls[DB + 1];
  const int32_t n_hub = n - first_hub_row;
  const int32_t n_chunks = n_hub > 0 ? total - hub_first_entry : 0;
  for (int64_t b = t0; b < total && b < cap; b += stride) {
    int32_t a = 0, c = S - 1;  // largest segment starting at or before b
    while (a < c) {
      const int32_t mid = (int32_t)(((int64_t)a + c + 1) >> 1);
      if (seg_off[mid] <= b) a = mid; else c = mid - 1;
    }
    const int32_t j = (int32_t)(b - seg_off[a]);
    int4 m;
    if (a <= DB) {
      const int32_t p = pattern_of(a, W, Z), br = p & 0xFFFF, wn = p >> 16;
      const int32_t r0 = cls[a] + j * br;
      const int32_t left = cls[a + 1] - r0;
      const int32_t rows = left < br ? left : br;
      m = make_int4(a, rowptr_s[r0], r0, (wn << 16) | rows);
    } else {
      const int32_t r = cls[DB + 1] + (a - DB - 1);
      const int32_t d = deg_s[r];
      const int32_t off = j * H;
      const int32_t left = d - off;
      m = make_int4(d, rowptr_s[r] + off, r, left < H ? left : H);
    }
    meta[b] = m;
    order[b] = b < n_chunks ? total - 1 - (int32_t)b : hub_first_entry - 1 - (int32_t)(b - n_chunks);
  }
  for (int64_t h = t0; h <= n_hub && h <= hub_ub; h += stride)
    hub_chunk_off[h] = seg_off[DB + 1 + h] - seg_off[DB + 1];
}

// The partition after the two-pass segment scan (S an upper bound on the
// segments: those past the last hub row are empty), and the summary for the
// host.
__global__ __launch_bounds__(kThreads) void k_partition_fill(
    int32_t n, const int32_t* __restrict__ rowptr_s, const int32_t* __restrict__ deg_s,
    const int32_t* __restrict__ cls, const int32_t* __restrict__ seg_off, int32_t S, int32_t W,
    int32_t Z, int32_t DB, int32_t H, int4* __restrict__ meta, int64_t cap, int32_t hub_ub,
    int32_t* __restrict__ hub_chunk_off, int32_t* __restrict__ order, PlanSummary* sum,
    const uint32_t* err) {
  const int64_t t0 = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  const int64_t stride = (int64_t)gridDim.x * kThreads;
  const uint32_t e = err[0];
  if (t0 == 0) {
    sum->err = e;
    if (e) {
      __threadfence_system();
      sum->done = 1;
      __threadfence_system();
    }
  }
  if (e) return;
  fill_partition(t0, stride, n, rowptr_s, deg_s, cls, seg_off, S, W, Z, DB, H, meta, cap, hub_ub,
                 hub_chunk_off, order);
  if (t0 == 0) {
    const int32_t first_hub_row = cls[DB + 1];
    sum->n_entries = seg_off[S];
    sum->hub_first_entry = seg_off[DB + 1];
    sum->n_hub_rows = n - first_hub_row;
    sum->hub_first_row = first_hub_row;
    sum->max_deg = n > 0 ? deg_s[n - 1] : 0;
    __threadfence_system();
    sum->done = 1;
    __threadfence_system();
  }
}

// The last partition launch of the short-sort plan: workgroups [0, n_fill)
// fill the partition from the tail workgroup's segment scan while the other
// n_copy build the sorted CSR from the tile holding the tail's first nonzero
// on (the tiles before it went with the tail), each a run of whole tiles.
// Returns at once when the tail is over the cap (the multi-pass sort follows).
__global__ __launch_bounds__(kThreads) void k_relayout_fill(
    int32_t n_fill, int32_t n_copy, int32_t n, int64_t nnz, const int32_t* __restrict__ rowptr,
    const int32_t* __restrict__ colidx, const float* __restrict__ vals,
    const int32_t* __restrict__ perm, const int32_t* __restrict__ rowptr_s,
    int32_t* __restrict__ colidx_s, float* __restrict__ vals_s, const int32_t* __restrict__ deg_s,
    const int32_t* __restrict__ cls, const int32_t* __restrict__ seg_off,
    const TailInfo* __restrict__ info, int32_t W, int32_t Z, int32_t DB, int32_t H,
    int4* __restrict__ meta, int64_t cap, int32_t hub_ub, int32_t* __restrict__ hub_chunk_off,
    int32_t* __restrict__ order, const int32_t* __restrict__ dmax, int32_t tail_cap,
    int32_t check_cols, uint32_t* err) {
  __shared__ int32_t lds[kRelaySpanLds];
  const TailShape ts = tail_shape(dmax, n, tail_cap);
  if (!ts.take || block_failed(err)) return;
  if ((int32_t)blockIdx.x < n_fill) {
    fill_partition((int64_t)blockIdx.x * kThreads + threadIdx.x, (int64_t)n_fill * kThreads, n,
                   rowptr_s, deg_s, cls, seg_off, info->n_segments, W, Z, DB, H, meta, cap, hub_ub,
                   hub_chunk_off, order);
    return;
  }
  const int64_t first = ts.nnz_low / kRelayTile;
  int64_t p0, p1;
  relay_share(first, (nnz + kRelayTile - 1) / kRelayTile - first, blockIdx.x - n_fill, n_copy, nnz,
              &p0, &p1);
  relay_span(p0, p1, n, check_cols, rowptr, colidx, vals, perm, rowptr_s, colidx_s, vals_s, err,
             lds);
}

// The rest of the plan up to the partition, in one workgroup of kTailThreads
// (the tail has at most kTailCap rows; T0 = n - m is its first sorted
// position):
//   - the tail sorted stably by degree: LSD passes of `width` <= 8 bits over
//     degree - key_base. Wave w holds the tail's elements [w c, (w + 1) c) (c a
//     multiple of 64, ceil(m / 16) rounded up) in registers, walking them in
//     rounds of 64; ranks come from per-wave digit counts and ballots as in
//     the radix passes, so equal degrees keep row order, and the (degree,
//     row) pairs are exchanged through LDS;
//   - perm and sorted degrees of the tail, and its row pointers (the nonzeros
//     before it are nnz minus the tail's);
//   - cls[d], the first sorted row of degree >= d, for d in [0, DB + 1]:
//     the short pass's bin starts up to key_base when `offsets` is given, a
//     search of the sorted tail above (DB >= kTailKey, so every hub row is a
//     tail row) or, without `offsets`, for every d;
//   - the segment scan of the partition (Alg. 2): ceil(count / block_rows)
//     entries for each degree class, ceil(deg / H) chunks for each hub row;
//   - the partition's summary, in pinned host memory (the segment count in
//     `info`).
struct TailArgs {
  int32_t n, nnz, W, Z, DB, H;
  int32_t cap;               // the short sort's largest tail
  int32_t check_cols;        // the relayout's column bound (INT32_MAX: checked before)
  int32_t publish;           // the tail's workgroup sets the host's done flag
  int32_t key_base;          // the sort's keys are degree - key_base (>= 0)
  const int32_t* tail_keys;  // [T0, n): the tail's degrees and rows in row order
  const int32_t* tail_ids;
  const int32_t* rowptr_in;  // instead of tail_keys / tail_ids (the whole graph,
                             // T0 = 0): degrees from the row pointer, rows in order
  const int32_t* offsets;    // the short pass's (digit, tile) starts, or null
  int32_t n_tiles;
  int32_t* keys;             // outputs: sorted degrees, perm, rowptr_s, cls, seg
  int32_t* perm;
  int32_t* rowptr_s;
  int32_t* cls;
  int32_t* seg;
  TailInfo* info;
  PlanSummary* sum;
  const int32_t* dmax;       // maximum degree, tail size, lower nonzeros
  const uint32_t* err;
};


// LDS of the tail's workgroup (int32 words).
constexpr int kTailLds = 2 * kTailCap + kTailWaves * kRadixBins + kTailWaves + 1;

__device__ inline void tail_block(const TailArgs& a, const TailShape& ts, int32_t* lds) {
  const int32_t n = a.n, nnz = a.nnz, T0 = ts.T0, W = a.W, Z = a.Z, DB = a.DB, H = a.H;
  const int32_t* __restrict__ tail_keys = a.tail_keys;
  const int32_t* __restrict__ tail_ids = a.tail_ids;
  const int32_t* __restrict__ offsets = a.offsets;
  const int32_t n_tiles = a.n_tiles;
  int32_t* __restrict__ keys = a.keys;
  int32_t* __restrict__ perm = a.perm;
  int32_t* __restrict__ rowptr_s = a.rowptr_s;
  int32_t* __restrict__ cls = a.cls;
  int32_t* __restrict__ seg = a.seg;
  int32_t* s_key = lds;                              // kTailCap
  int32_t* s_id = s_key + kTailCap;                  // kTailCap; cls once the tail is written
  int32_t (*s_cnt)[kRadixBins] = reinterpret_cast<int32_t (*)[kRadixBins]>(s_id + kTailCap);
  int32_t* s_wsum = s_id + kTailCap + kTailWaves * kRadixBins;
  int32_t& s_hub_first_entry = s_wsum[kTailWaves];
  const uint32_t dmask = (1u << ts.width) - 1;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int32_t m = n - T0;
  const int32_t c = ((m + kTailWaves * 64 - 1) / (kTailWaves * 64)) * 64;  // per wave
  const int32_t rounds = c / 64;
  const int32_t w0 = wave * c;
  int32_t k[kTailItems], id[kTailItems];
#pragma unroll
  for (int j = 0; j < kTailItems; ++j) {
    if (j < rounds) {
      const int32_t e = w0 + j * 64 + lane;
      if (a.rowptr_in != nullptr) {
        k[j] = e < m ? a.rowptr_in[e + 1] - a.rowptr_in[e] : 0;
        id[j] = e;
      } else {
        k[j] = e < m ? tail_keys[T0 + e] : 0;
        id[j] = e < m ? tail_ids[T0 + e] : 0;
      }
    }
  }
  for (int p = 0; p < ts.passes; ++p) {
    const int shift = ts.width * p;
    for (int q = t; q < kTailWaves * kRadixBins; q += kTailThreads) (&s_cnt[0][0])[q] = 0;
    __syncthreads();
    // Digit, rank among the round's equal digits and their number, packed
    // per item for the scatter walk.
    uint32_t pk[kTailItems];
#pragma unroll
    for (int j = 0; j < kTailItems; ++j) {
      if (j < rounds) {
        const bool valid = w0 + j * 64 + lane < m;
        const uint32_t digit = ((uint32_t)(k[j] - a.key_base) >> shift) & dmask;
        const uint64_t peers = match_bits(digit, valid, ts.width);
        const uint32_t rank = (uint32_t)__popcll(peers & __lanemask_lt());
        const uint32_t size = (uint32_t)__popcll(peers);
        pk[j] = digit | rank << 8 | size << 16;
        if (valid && rank == 0) s_cnt[wave][digit] += (int32_t)size;
      }
    }
    __syncthreads();
    {  // exclusive scan in (digit, wave) order: thread t owns digit t / 4, waves 4 (t % 4) ..
      const int d = t >> 2, v0 = (t & 3) * 4;
      int32_t cv[4], sm = 0;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        cv[r] = s_cnt[v0 + r][d];
        sm += cv[r];
      }
      int32_t total;
      int32_t run = block_exclusive_scan<kTailThreads>(sm, &total);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        s_cnt[v0 + r][d] = run;
        run += cv[r];
      }
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < kTailItems; ++j) {
      if (j < rounds) {
        const bool valid = w0 + j * 64 + lane < m;
        const uint32_t digit = pk[j] & 0xFFu, rank = (pk[j] >> 8) & 0xFFu;
        const int32_t pos = s_cnt[wave][digit] + (int32_t)rank;
        if (valid) {
          s_key[pos] = k[j];
          s_id[pos] = id[j];
        }
        if (valid && rank == 0) s_cnt[wave][digit] += (int32_t)(pk[j] >> 16);
      }
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < kTailItems; ++j) {
      if (j < rounds) {
        const int32_t e = w0 + j * 64 + lane;
        if (e < m) {
          k[j] = s_key[e];
          id[j] = s_id[e];
        }
      }
    }
    __syncthreads();
  }
  // The sorted tail: perm, degrees, s_key (also written when no pass ran)
  // and the wave's running sum of degrees for the row pointers.
  int32_t run = 0;
#pragma unroll
  for (int j = 0; j < kTailItems; ++j) {
    if (j < rounds) {
      const int32_t e = w0 + j * 64 + lane;
      const int32_t v = e < m ? k[j] : 0;
      if (e < m) {
        perm[T0 + e] = id[j];
        keys[T0 + e] = v;
        s_key[e] = v;
      }
      const int32_t inc = wave_inclusive_scan(v, lane);
      k[j] = run + inc - v;  // exclusive within the wave's chunk
      run += __shfl(inc, 63, 64);
    }
  }
  if (lane == 0) s_wsum[wave] = run;
  __syncthreads();
  {
    int32_t before = 0, total = 0;
    for (int w = 0; w < kTailWaves; ++w) {
      before += w < wave ? s_wsum[w] : 0;
      total += s_wsum[w];
    }
    const int32_t base = nnz - total + before;  // the tail's nonzeros end at nnz
#pragma unroll
    for (int j = 0; j < kTailItems; ++j) {
      if (j < rounds) {
        const int32_t e = w0 + j * 64 + lane;
        if (e < m) rowptr_s[T0 + e] = base + k[j];
      }
    }
    if (t == 0) rowptr_s[n] = nnz;
  }
  // Class starts.
  int32_t* s_cls = s_id;
  for (int32_t d = t; d <= DB + 1; d += kTailThreads) {
    int32_t r;
    if (offsets != nullptr && d <= a.key_base) {
      r = offsets[(int64_t)d * n_tiles];
    } else {
      int32_t a = 0, b = m;  // first tail element of degree >= d
      while (a < b) {
        const int32_t mid = (a + b) >> 1;
        if (s_key[mid] < d) a = mid + 1; else b = mid;
      }
      r = T0 + a;
    }
    s_cls[d] = r;
    cls[d] = r;
  }
  __syncthreads();
  const int32_t hub_first_row = s_cls[DB + 1];
  const int32_t S = DB + 1 + (n - hub_first_row);
  int32_t carry = 0;
  for (int32_t c0 = 0; c0 < S; c0 += kTailThreads * 4) {
    int32_t v[4], sm = 0;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int32_t q = c0 + t * 4 + r;
      int32_t x = 0;
      if (q <= DB) {
        const int32_t cnt = s_cls[q + 1] - s_cls[q];
        if (cnt > 0) {
          const int32_t br = pattern_of(q, W, Z) & 0xFFFF;
          x = (cnt + br - 1) / br;
        }
      } else if (q < S) {
        x = (int32_t)(((int64_t)s_key[hub_first_row - T0 + (q - DB - 1)] + H - 1) / H);
      }
      v[r] = x;
      sm += x;
    }
    int32_t total;
    int32_t rs = block_exclusive_scan<kTailThreads>(sm, &total) + carry;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int32_t q = c0 + t * 4 + r;
      if (q < S) seg[q] = rs;
      if (q == DB + 1) s_hub_first_entry = rs;
      rs += v[r];
    }
    carry += total;
  }
  __syncthreads();
  if (t == 0) {
    seg[S] = carry;
    const int32_t hfe = S > DB + 1 ? s_hub_first_entry : carry;
    a.info->n_segments = S;
    a.sum->n_entries = carry;
    a.sum->hub_first_entry = hfe;
    a.sum->n_hub_rows = n - hub_first_row;
    a.sum->hub_first_row = hub_first_row;
    a.sum->max_deg = a.dmax[0];
    if (a.publish) {  // every input error is known: k_degree checked the columns
      a.sum->err = a.err[0];  // final but for kErrRelayout, which k_relayout_fill may raise
      __threadfence_system();
      a.sum->done = 1;
    }
    __threadfence_system();
  }
}


// The short-sort plan's second launch: workgroup 0 finishes the plan up to the
// partition (tail_block) and publishes the summary, while the other n_groups
// copy the sorted CSR of the rows below the tail, which need nothing from it:
// kTailThreads / kThreads tiles per workgroup and round, the tiles of sorted
// nonzeros wholly before the tail's first nonzero. The LDS is one buffer that
// either role carves. Returns at once when the tail is over the cap (the
// multi-pass sort follows); on an input error workgroup 0 publishes it.
constexpr int kTilesPerTailGroup = kTailThreads / kThreads;
// Relayout workgroups of kThreads per CU (k_relayout, k_relayout_fill; their
// registers allow six). Each copies one run of tiles, so the grids stay
// within what the CUs hold at once: a late workgroup would add its whole run.
constexpr int kRelayGroupsPerCu = 6;
constexpr int kXLds = kTailLds > kTilesPerTailGroup * kRelayLds ? kTailLds
                                                                 : kTilesPerTailGroup * kRelayLds;

__global__ __launch_bounds__(kTailThreads) void k_tail_relayout(
    TailArgs ta, int32_t n_groups, const int32_t* __restrict__ rowptr,
    const int32_t* __restrict__ colidx, const float* __restrict__ vals,
    int32_t* __restrict__ colidx_s, float* __restrict__ vals_s, uint32_t* err) {
  __shared__ int32_t lds[kXLds];
  const TailShape ts = tail_shape(ta.dmax, ta.n, ta.cap);
  if (!ts.take) return;
  if (block_failed(err)) {
    if (ta.publish && blockIdx.x == 0 && threadIdx.x == 0) {
      ta.sum->err = err[0];
      __threadfence_system();
      ta.sum->done = 1;
      __threadfence_system();
    }
    return;
  }
  if (blockIdx.x == 0) {
    tail_block(ta, ts, lds);
    return;
  }
  const int q = threadIdx.x / kThreads;
  // Rows [0, T0) with rowptr_s[T0] (the tail's first nonzero) are final.
  const int64_t low_tiles = ts.nnz_low / kRelayTile;
  for (int64_t t0 = (int64_t)(blockIdx.x - 1) * kTilesPerTailGroup; t0 < low_tiles;
       t0 += (int64_t)n_groups * kTilesPerTailGroup) {
    const int64_t tile = t0 + q;
    relayout_tile(tile, tile < low_tiles, threadIdx.x % kThreads, ts.T0, ta.nnz, ta.check_cols, rowptr, colidx,
                  vals, ta.perm, ta.rowptr_s, colidx_s, vals_s, err, lds + q * kRelayLds);
  }
}

// The plan of a small graph (at most kTinyMaxRows rows and kTinyMaxNnz
// nonzeros) up to the partition, in one workgroup of kTailThreads, in place of
// k_degree, the scans and k_scatter_low: the input checked (row pointer and
// column indices), every row sorted by degree by the tail's code (key base 0,
// any W and Z), the class starts, the segment scan and the summary with the
// host's done flag. k_relayout_fill then copies the whole sorted CSR and fills
// the partition, reading the tail size (all rows) and the lower nonzeros (none)
// that this kernel leaves in dmax.
constexpr int32_t kTinyMaxRows = kTailCap;
constexpr int64_t kTinyMaxNnz = int64_t(1) << 17;
constexpr int kTinyCheckItems = 16;

__global__ __launch_bounds__(kTailThreads) void k_plan_tiny(TailArgs ta, int32_t n_cols,
                                                            const int32_t* __restrict__ rowptr,
                                                            const int32_t* __restrict__ colidx,
                                                            uint32_t* err, int32_t* tickets,
                                                            int32_t* dmax) {
  __shared__ int32_t lds[kXLds];
  __shared__ uint32_t s_err;
  __shared__ int32_t s_max;
  const int t = threadIdx.x;
  const int32_t n = ta.n;
  const int64_t nnz = ta.nnz;
  if (t == 0) {
    s_err = 0;
    s_max = 0;
  }
  if (t < kMaxChainedScans) tickets[t] = 0;  // the scans of the hub-chunk order sort
  __syncthreads();
  uint32_t e = 0;
  int32_t mx = 0;
#pragma unroll
  for (int j = 0; j < kTailItems; ++j) {  // n <= kTailThreads * kTailItems
    const int32_t i = j * kTailThreads + t;
    if (i < n) {
      const int32_t a0 = rowptr[i], b0 = rowptr[i + 1];
      if (a0 < 0 || b0 < a0 || (int64_t)b0 > nnz) e |= kErrRowptrOrder;
      else mx = max(mx, b0 - a0);
      if (i == 0 && a0 != 0) e |= kErrRowptrStart;
      if (i == n - 1 && (int64_t)b0 != nnz) e |= kErrRowptrEnd;
    }
  }
  for (int64_t k0 = t; k0 < nnz; k0 += (int64_t)kTailThreads * kTinyCheckItems) {
    int32_t c[kTinyCheckItems];
#pragma unroll
    for (int u = 0; u < kTinyCheckItems; ++u) {
      const int64_t k = k0 + (int64_t)u * kTailThreads;
      c[u] = k < nnz ? colidx[k] : 0;
    }
#pragma unroll
    for (int u = 0; u < kTinyCheckItems; ++u)
      e |= (uint32_t)c[u] >= (uint32_t)n_cols ? kErrColumn : 0u;
  }
  e = wave_or(e);
  mx = wave_max(mx);
  if ((t & 63) == 0) {
    if (e) atomicOr(&s_err, e);
    atomicMax(&s_max, mx);
  }
  __syncthreads();
  if (t == 0) {
    err[0] = s_err;
    dmax[0] = s_max;
    dmax[1] = n;  // for k_relayout_fill: every row sorted here, no lower nonzeros
    dmax[2] = 0;
  }
  if (s_err != 0) {
    if (t == 0) {
      ta.sum->err = s_err;
      __threadfence_system();
      ta.sum->done = 1;
      __threadfence_system();
    }
    return;
  }
  TailShape ts;
  ts.take = true;
  ts.m = n;
  ts.T0 = 0;
  ts.nnz_low = 0;
  int bits = 0;
  while (bits < 31 && (int64_t(1) << bits) <= (int64_t)s_max) ++bits;
  ts.passes = (bits + 7) / 8;
  ts.width = ts.passes > 0 ? (bits + ts.passes - 1) / ts.passes : 8;
  tail_block(ta, ts, lds);
}

// The summary's error word (the relayout's column check included) and done
// flag, after k_relayout_fill, when the tail's workgroup could not publish
// them. One small launch: a completion count kept by the relayout's
// workgroups themselves cost more (one device-scope atomic each on one word,
// serialised). Like the launches before it, it returns at once when the tail
// is over the cap (the multi-pass sort publishes instead).
__global__ void k_publish(const uint32_t* err, PlanSummary* sum, const int32_t* dmax, int32_t n,
                          int32_t tail_cap) {
  if (!tail_shape(dmax, n, tail_cap).take) return;
  if (threadIdx.x == 0 && blockIdx.x == 0) {
    sum->err = err[0];
    __threadfence_system();
    sum->done = 1;
    __threadfence_system();
  }
}

// --- launch order -----------------------------------------------------------

// Key of hub chunk i: its first column scaled to 16 bits. Chunks of a row
// with sorted columns cover narrow column ranges, so ordering chunks by this
// key makes chunks that run side by side gather neighbouring X rows.
__global__ __launch_bounds__(kThreads) void k_hub_keys(const int4* __restrict__ meta,
                                                       const int32_t* __restrict__ colidx_s,
                                                       int32_t hub_first, int32_t n_chunks,
                                                       int32_t n_cols, int32_t* __restrict__ keys,
                                                       int32_t* gate) {
  const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (i == 0) gate[0] = 0xFFFF;  // two 8-bit passes
  if (i >= n_chunks) return;
  const int32_t c = colidx_s[meta[hub_first + i].y];
  keys[i] = (int32_t)(((int64_t)c << 16) / n_cols);
}

// order[i] = entry launched by workgroup i: the n_chunks hub entries first
// (sorted ids, or in reverse entry order without them), then the remaining
// entries from the heaviest down. This sort runs after the host has read the
// plan's summary, so nothing reads the error word again: if a scan of the sort
// gave up its bounded wait (or any earlier step failed), the sorted ids were
// never written, and the plain order -- a permutation of every entry whatever
// happened -- is written instead.
__global__ __launch_bounds__(kThreads) void k_order_fill(int32_t* __restrict__ order,
                                                         int32_t n_entries, int32_t hub_first,
                                                         int32_t n_chunks,
                                                         const int32_t* __restrict__ sorted_ids,
                                                         const uint32_t* err) {
  const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (i >= n_entries) return;
  const bool use_sorted = sorted_ids != nullptr && !failed(err);
  if (i < n_chunks)
    order[i] = use_sorted ? hub_first + sorted_ids[i] : n_entries - 1 - (int32_t)i;
  else
    order[i] = hub_first - 1 - (int32_t)(i - n_chunks);
}

// Hub-row windows: win_tab[k * n_hub + h] = first position of sorted hub row h
// whose column is >= k * kWinCols (k = 0 and k = n_win give the row's ends).
// search_lb: an 8-way search over [lo, hi) -- each round loads the last
// element of the first seven of eight equal parts at once and keeps the part
// after the m whose element is below the key (about 6 rounds for 10^5
// elements where a binary search chains 17 loads); at most 8 elements left are
// counted. Every choice is a count of elements below the key, which does not
// decrease as the key grows, so over a fixed range the result does not
// decrease in the key, whether or not the columns ascend.
__device__ inline int32_t search_lb(const int32_t* __restrict__ a, int32_t lo, int32_t hi,
                                    int64_t key) {
  while (hi - lo > 8) {
    const int64_t n = hi - lo;
    int32_t m = 0;
#pragma unroll
    for (int q = 1; q < 8; ++q) m += a[lo + (int32_t)((n * q) >> 3) - 1] < key ? 1 : 0;
    const int32_t nlo = lo + (int32_t)((n * m) >> 3);
    hi = m < 7 ? lo + (int32_t)((n * (m + 1)) >> 3) - 1 : hi;
    lo = nlo;
  }
  int32_t below = 0;
  for (int32_t j = lo; j < hi; ++j) below += a[j] < key ? 1 : 0;
  return lo + below;
}

// Windows one wave of k_hub_win_table covers: kWinTableLanes per lane.
constexpr int kWinTableLanes = 4;
constexpr int32_t kWinTableSpan = 64 * kWinTableLanes;

// One wave per (hub row, kWinTableSpan consecutive windows from k0): every lane
// first brackets the wave's positions by two searches over the whole row (the
// same addresses in every lane, one request each), [b0, b1] = the positions
// of k0 and k0 + kWinTableSpan; lane t then searches windows k0 + t + 64 q
// within the bracket, the kWinTableLanes searches advancing side by side so
// their loads are in flight together (the kernel waits on load latency, not
// bandwidth). b1 is the next wave's b0, so positions do not decrease across
// waves either, and the windows partition every row.
__global__ __launch_bounds__(kThreads) void k_hub_win_table(const int32_t* __restrict__ rowptr_s,
                                                            const int32_t* __restrict__ colidx_s,
                                                            int32_t hub_first_row, int32_t n_hub,
                                                            int32_t n_win,
                                                            int32_t* __restrict__ win_tab) {
  constexpr int Q = kWinTableLanes;
  const int32_t per_row = n_win / kWinTableSpan + 1;  // waves per row: windows 0 .. n_win
  const int64_t waves = (int64_t)n_hub * per_row;
  const int lane = threadIdx.x & 63;
  const int64_t stride = (int64_t)gridDim.x * (kThreads / 64);
  for (int64_t w = (int64_t)blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6); w < waves;
       w += stride) {
    const int32_t h = (int32_t)(w / per_row);
    const int32_t k0 = (int32_t)(w - (int64_t)h * per_row) * kWinTableSpan;
    const int32_t s = rowptr_s[hub_first_row + h], e = rowptr_s[hub_first_row + h + 1];
    const int32_t b0 = k0 == 0 ? s : search_lb(colidx_s, s, e, (int64_t)k0 * kWinCols);
    const int32_t b1 = k0 + kWinTableSpan >= n_win
                           ? e
                           : search_lb(colidx_s, s, e, (int64_t)(k0 + kWinTableSpan) * kWinCols);
    int64_t key[Q];
    int32_t lo[Q], hi[Q];
#pragma unroll
    for (int q = 0; q < Q; ++q) {
      key[q] = (int64_t)(k0 + q * 64 + lane) * kWinCols;
      lo[q] = b0;
      hi[q] = b1;
    }
    // the 8-way search of search_lb, Q chains in step
    for (bool more = b1 - b0 > 8; more;) {
      more = false;
#pragma unroll
      for (int q = 0; q < Q; ++q) {
        const int64_t n = hi[q] - lo[q];
        if (n > 8) {
          int32_t m = 0;
#pragma unroll
          for (int t = 1; t < 8; ++t)
            m += colidx_s[lo[q] + (int32_t)((n * t) >> 3) - 1] < key[q] ? 1 : 0;
          const int32_t nlo = lo[q] + (int32_t)((n * m) >> 3);
          hi[q] = m < 7 ? lo[q] + (int32_t)((n * (m + 1)) >> 3) - 1 : hi[q];
          lo[q] = nlo;
          more = more || hi[q] - lo[q] > 8;
        }
      }
    }
#pragma unroll
    for (int q = 0; q < Q; ++q) {
      const int32_t k = k0 + q * 64 + lane;
      if (k > n_win) continue;
      int32_t below = 0;
      for (int32_t j = lo[q]; j < hi[q]; ++j) below += colidx_s[j] < key[q] ? 1 : 0;
      win_tab[(int64_t)k * n_hub + h] = k == 0 ? s : (k == n_win ? e : lo[q] + below);
    }
  }
}

// --- warp-level partition (the baseline of the paper's Table II) -----------

// Groups per row: ceil(deg / Z), at least one so an empty row is still written.
__global__ __launch_bounds__(kThreads) void k_wl_groups(int32_t n, const int32_t* __restrict__ deg,
                                                        int32_t Z, int32_t* __restrict__ ng,
                                                        const uint32_t* err) {
  if (failed(err)) return;
  const int64_t r = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (r >= n) return;
  const int32_t d = deg[r];
  ng[r] = d > 0 ? (d + Z - 1) / Z : 1;
}

// Unsorted copy of the CSR (checked columns) and the identity permutation.
__global__ __launch_bounds__(kThreads) void k_wl_copy(int32_t n, int64_t nnz, int32_t n_cols,
                                                      const int32_t* __restrict__ rowptr,
                                                      const int32_t* __restrict__ colidx,
                                                      const float* __restrict__ vals,
                                                      int32_t* __restrict__ perm,
                                                      int32_t* __restrict__ rowptr_s,
                                                      int32_t* __restrict__ colidx_s,
                                                      float* __restrict__ vals_s, uint32_t* err) {
  if (failed(err)) return;
  uint32_t bad = 0;
  for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < nnz || i <= n;
       i += (int64_t)gridDim.x * kThreads) {
    if (i < nnz) {
      const int32_t c = colidx[i];
      if ((uint32_t)c >= (uint32_t)n_cols) bad = kErrColumn;
      colidx_s[i] = c;
      vals_s[i] = vals[i];
    }
    if (i <= n) rowptr_s[i] = rowptr[i];
    if (i < n) perm[i] = (int32_t)i;
  }
  if (bad) atomicOr(err, bad);
}

// Group g: row r = the last row whose first group is <= g; its j-th group
// covers nnz [rowptr[r] + j Z, + min(Z, deg - j Z)).
__global__ __launch_bounds__(kThreads) void k_wl_fill(int32_t n, const int32_t* __restrict__ rowptr,
                                                      const int32_t* __restrict__ goff, int32_t Z,
                                                      int4* __restrict__ meta, int64_t cap,
                                                      const uint32_t* err) {
  if (failed(err)) return;
  const int64_t total = goff[n];
  for (int64_t g = (int64_t)blockIdx.x * kThreads + threadIdx.x; g < total && g < cap;
       g += (int64_t)gridDim.x * kThreads) {
    int32_t a = 0, b = n - 1;
    while (a < b) {
      const int32_t mid = (int32_t)(((int64_t)a + b + 1) >> 1);
      if (goff[mid] <= g) a = mid; else b = mid - 1;
    }
    const int32_t j = (int32_t)(g - goff[a]);
    const int32_t d = rowptr[a + 1] - rowptr[a];
    const int32_t left = d - j * Z;
    meta[g] = make_int4(a, rowptr[a] + j * Z, left < Z ? left : Z, 0);
  }
}

__global__ void k_wl_summary(int32_t n, const int32_t* __restrict__ goff,
                             const int32_t* __restrict__ dmax, PlanSummary* sum,
                             const uint32_t* err) {
  if (threadIdx.x != 0 || blockIdx.x != 0) return;
  const uint32_t e = err[0];
  sum->err = e;
  if (!e) {
    sum->n_entries = goff[n];
    sum->hub_first_entry = goff[n];
    sum->n_hub_rows = 0;
    sum->hub_first_row = n;
    sum->max_deg = dmax[0];
  }
  __threadfence_system();
}

// ---------------------------------------------------------------------------

inline unsigned grid_for(int64_t work, int per_block) {
  return (unsigned)ceil_div64(work, per_block);
}

int check_launch(const char* what) {
  const hipError_t e = hipGetLastError();
  return e == hipSuccess ? AGCN_OK : hip_fail(e, what);
}

// out[i] = sum of in[0..i) for i < n, and *total = sum of all (may alias out + n).
// In place (out == in) is allowed. With `gate`, the scan belongs to radix
// pass `gate_pass` and is skipped on the device when that pass is.
// Single-pass scans of one plan: status words (one per tile of the largest
// scan) and one ticket counter per scan, zeroed by k_dmax.
struct ChainedScans {
  unsigned long long* status = nullptr;
  int64_t capacity = 0;  // status words
  int32_t* tickets = nullptr;
  int next = 0;
};

uint32_t next_scan_epoch() {
  static std::atomic<uint32_t> epoch{0};
  uint32_t e;
  do e = (epoch.fetch_add(1, std::memory_order_relaxed) + 1) & 0x3FFFFFFFu; while (e == 0);
  return e;
}

// With db (dmax non-null), the scan also performs k_degree's reduction: in
// its first tile when the scan runs in one pass, else by a k_dmax launch
// before it.
int scan_exclusive(const int32_t* in, int64_t n, int32_t* out, int32_t* total, int32_t* partials,
                   const uint32_t* err, hipStream_t st, const int32_t* gate = nullptr,
                   int gate_pass = 0, ChainedScans* chain = nullptr, DegreeBlocks db = {}) {
  if (n > kScanMaxN) return fail(AGCN_ERR_UNSUPPORTED, "scan longer than the supported maximum");
  const unsigned nb_tiles = n > 0 ? grid_for(n, kScanBlock) : 0;
  const bool fused = db.dmax != nullptr && chain && chain->next < kMaxChainedScans &&
                     n > kScanSingleMax && (int64_t)nb_tiles <= chain->capacity &&
                     nb_tiles <= kChainedMaxTiles;
  if (db.dmax != nullptr && !fused) {
    k_dmax<<<1, kScanTopThreads, 0, st>>>(db, chain ? chain->tickets : nullptr);
    if (int rc = check_launch("k_dmax")) return rc;
    db = DegreeBlocks{};
  }
  if (n == 0) {
    if (total) k_set<<<1, 64, 0, st>>>(total, 0);
    return check_launch("k_set");
  }
  if (n <= kScanSingleMax) {
    k_scan_single<<<1, kScanTopThreads, 0, st>>>(in, (int32_t)n, out, total, err, gate, gate_pass);
    return check_launch("k_scan_single");
  }
  const unsigned nb = grid_for(n, kScanBlock);
  // Single pass up to kChainedMaxTiles tiles, where one wave's look-back spans
  // every predecessor; longer scans walk back window by window and ran
  // slower than the two passes (measured on 2.4 M rows).
  if (chain && chain->next < kMaxChainedScans && (int64_t)nb <= chain->capacity &&
      nb <= kChainedMaxTiles) {
    k_scan_chained<<<nb, kThreads, 0, st>>>(in, n, out, total, chain->status,
                                            chain->tickets + chain->next, next_scan_epoch(),
                                            const_cast<uint32_t*>(err), gate, gate_pass, db);
    ++chain->next;
    return check_launch("k_scan_chained");
  }
  k_scan_reduce<<<nb, kThreads, 0, st>>>(in, n, partials, err, gate, gate_pass);
  if (nb <= kScanTwoPassMaxBlocks) {
    k_scan_down<<<nb, kThreads, 0, st>>>(in, n, partials, out, total, 1, err, gate, gate_pass);
  } else {
    k_scan_top<<<1, kScanTopThreads, 0, st>>>(partials, (int32_t)nb, total, err, gate, gate_pass);
    k_scan_down<<<nb, kThreads, 0, st>>>(in, n, partials, out, nullptr, 0, err, gate, gate_pass);
  }
  return check_launch("scan");
}

// Hub-chunk launch order by column (AGCN_HUB_ORDER=0 keeps the plain
// heaviest-first order, for measurements).
bool hub_windows_setting() {
  const char* s = std::getenv("AGCN_HUB_WINDOWS");
  return s == nullptr || std::atoi(s) != 0;
}

bool hub_order_setting() {
  static const bool v = [] {
    const char* s = std::getenv("AGCN_HUB_ORDER");
    return s == nullptr || std::atoi(s) != 0;
  }();
  return v;
}

// Largest tail the short sort's single workgroup takes (AGCN_TEST_TAIL_CAP
// lowers it, so that tests reach the multi-pass sort on small graphs; -1
// sends every plan there).
int32_t tail_cap_setting() {
  const int v = test_tail_cap();
  return v < -1 ? kTailCap : std::min<int32_t>(v, kTailCap);
}

// Compute units of a device, queried once per device.
int32_t device_cus(int dev) {
  static std::atomic<int32_t> cached[64];
  if (dev < 0 || dev >= 64) return 256;
  const int32_t v = cached[dev].load(std::memory_order_relaxed);
  if (v > 0) return v;
  int cus = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      cus <= 0) {
    (void)hipGetLastError();
    cus = 256;
  }
  cached[dev].store(cus, std::memory_order_relaxed);
  return cus;
}

// Per-thread pinned, host-coherent buffer for the plan's read-backs (the
// kernels write it directly), allocated on the first plan built by the thread
// and kept for the life of the process. *dev receives its device address.
PlanSummary* pinned_summary(PlanSummary** dev) {
  thread_local PlanSummary* buf = nullptr;
  thread_local PlanSummary* dbuf = nullptr;
  if (buf == nullptr) {
    void* q = nullptr;
    if (test_alloc_fails()) return nullptr;
    // Portable: one buffer serves plans built on any device from this thread.
    if (hipHostMalloc(&q, sizeof(PlanSummary),
                      hipHostMallocMapped | hipHostMallocCoherent | hipHostMallocPortable) !=
        hipSuccess) {
      (void)hipGetLastError();
      return nullptr;
    }
    void* d = nullptr;
    if (hipHostGetDevicePointer(&d, q, 0) != hipSuccess) {
      (void)hipGetLastError();
      (void)hipHostFree(q);
      return nullptr;
    }
    buf = static_cast<PlanSummary*>(q);
    dbuf = static_cast<PlanSummary*>(d);
  }
  *dev = dbuf;
  return buf;
}

// Waits until the device sets *flag, a word of the pinned summary, polling
// it. Once the wait has taken kQueryAfterUs, the stream is queried every 64
// polls, so a failed launch or a stream that finished without setting the
// flag ends the wait with an error. (A query of a busy stream queues a
// marker behind its work, around which the GPU idles several microseconds;
// a plan queued behind a whole step of other work waits milliseconds.)
constexpr int kQueryAfterUs = 2000000;

int wait_flag(const uint32_t* flag, hipStream_t st, const char* what) {
  const auto t0 = std::chrono::steady_clock::now();
  bool query = false;
  for (uint32_t it = 1;; ++it) {
    if (__atomic_load_n(flag, __ATOMIC_ACQUIRE) != 0) return AGCN_OK;
    if (!query && (it & 63) == 0)
      query = std::chrono::steady_clock::now() - t0 > std::chrono::microseconds(kQueryAfterUs);
    if (query && (it & 63) == 0) {
      const hipError_t q = hipStreamQuery(st);
      if (q == hipSuccess) {
        if (__atomic_load_n(flag, __ATOMIC_ACQUIRE) != 0) return AGCN_OK;
        return fail(AGCN_ERR_HIP, std::string(what) + ": the stream finished without the result");
      }
      if (q != hipErrorNotReady) return hip_fail(q, what);
    }
    std::this_thread::yield();
  }
}

struct Layout {
  size_t off = 0;
  size_t take(size_t bytes) {
    const size_t at = off;
    off += (bytes + 255) & ~size_t(255);
    return at;
  }
};

}  // namespace

namespace {

// Warp-level plan: validation, an unsorted CSR copy, one group per <= Z nnz.
int build_plan_warp_level(agcn_plan* p, const int32_t* d_rowptr, const int32_t* d_colidx,
                          const float* d_vals, hipStream_t st) {
  const int64_t n = p->n_rows, nnz = p->nnz;
  const int32_t Z = p->Z;
  const int64_t g_ub = n + nnz / Z + 1;
  const int64_t n_partials = ceil_div64(n + 1, kScanBlock) + 1;
  if (g_ub >= INT32_MAX) return fail(AGCN_ERR_UNSUPPORTED, "too many warp groups for int32 indexing");
  Layout L;
  const size_t o_perm = L.take(4 * n);
  const size_t o_rowptr_s = L.take(4 * (n + 1));
  const size_t o_colidx_s = L.take(4 * nnz);
  const size_t o_vals_s = L.take(4 * nnz);
  const size_t o_meta = L.take(16 * g_ub);
  const size_t o_goff = L.take(4 * (n + 1));
  const size_t o_deg = L.take(4 * n);
  const size_t o_ng = L.take(4 * n);
  const int64_t n_deg_blocks = ceil_div64(n, kDegRows);
  const size_t o_bmax = L.take(4 * 4 * (n_deg_blocks + 1));  // maxima, error flags, tails, lows
  const size_t o_partials = L.take(4 * n_partials);
  const size_t o_err = L.take(64);
  const size_t o_dmax = L.take(64);
  const size_t o_tickets = L.take(4 * kMaxChainedScans);
  const size_t o_status = L.take(8 * n_partials);
  void* base = nullptr;
  size_t got = 0;
  int rc = device_alloc(p->device, L.off, st, &base, &got);
  if (rc) return rc;
  char* b = static_cast<char*>(base);
  p->base = base;
  p->bytes = got;
  p->perm = reinterpret_cast<int32_t*>(b + o_perm);
  p->rowptr_s = reinterpret_cast<int32_t*>(b + o_rowptr_s);
  p->colidx_s = reinterpret_cast<int32_t*>(b + o_colidx_s);
  p->vals_s = reinterpret_cast<float*>(b + o_vals_s);
  p->meta = reinterpret_cast<int4*>(b + o_meta);
  p->group_off = reinterpret_cast<int32_t*>(b + o_goff);
  int32_t* deg = reinterpret_cast<int32_t*>(b + o_deg);
  int32_t* ng = reinterpret_cast<int32_t*>(b + o_ng);
  int32_t* bmax = reinterpret_cast<int32_t*>(b + o_bmax);
  int32_t* partials = reinterpret_cast<int32_t*>(b + o_partials);
  uint32_t* err = reinterpret_cast<uint32_t*>(b + o_err);
  int32_t* dmax = reinterpret_cast<int32_t*>(b + o_dmax);
  PlanSummary* dsum = nullptr;
  PlanSummary* hs = pinned_summary(&dsum);
  if (hs == nullptr) return fail(AGCN_ERR_OUT_OF_MEMORY, "pinned host buffer allocation failed");
  *hs = PlanSummary{};
  const int64_t nb = ceil_div64(n, kThreads);
  uint32_t* berr = reinterpret_cast<uint32_t*>(bmax + n_deg_blocks + 1);
  int32_t* btail = bmax + 2 * (n_deg_blocks + 1);
  int32_t* blow = bmax + 3 * (n_deg_blocks + 1);
  if (n > 0)
    k_degree<<<(unsigned)n_deg_blocks, kThreads, 0, st>>>(
        (int32_t)n, nnz, d_rowptr, deg, bmax, berr, btail, blow, nullptr, 0, nullptr, nullptr,
        (int32_t)n_deg_blocks, ColumnCheck{});  // k_wl_copy checks the columns
  ChainedScans chain;
  chain.status = reinterpret_cast<unsigned long long*>(b + o_status);
  chain.capacity = n_partials;
  chain.tickets = reinterpret_cast<int32_t*>(b + o_tickets);
  k_dmax<<<1, kScanTopThreads, 0, st>>>(
      DegreeBlocks{bmax, berr, btail, blow, (int32_t)n_deg_blocks, (int32_t)n_deg_blocks, dmax, err,
                   dsum},
      chain.tickets);
  if (n > 0) k_wl_groups<<<(unsigned)nb, kThreads, 0, st>>>((int32_t)n, deg, Z, ng, err);
  const unsigned cgrid = (unsigned)std::min<int64_t>(grid_for(std::max(nnz, n + 1), kThreads), 65536);
  k_wl_copy<<<cgrid, kThreads, 0, st>>>((int32_t)n, nnz, p->n_cols, d_rowptr, d_colidx, d_vals,
                                        p->perm, p->rowptr_s, p->colidx_s, p->vals_s, err);
  if ((rc = check_launch("warp-level plan"))) return rc;
  if ((rc = scan_exclusive(ng, n, p->group_off, p->group_off + n, partials, err, st, nullptr, 0,
                           &chain)))
    return rc;
  if (n > 0) {
    const unsigned fgrid = (unsigned)std::min<int64_t>(grid_for(g_ub, kThreads), 16384);
    k_wl_fill<<<fgrid, kThreads, 0, st>>>((int32_t)n, d_rowptr, p->group_off, Z, p->meta, g_ub, err);
  }
  k_wl_summary<<<1, 64, 0, st>>>((int32_t)n, p->group_off, dmax, dsum, err);
  if ((rc = check_launch("warp-level plan"))) return rc;
  hipError_t he = hipStreamSynchronize(st);
  if (he != hipSuccess) return hip_fail(he, "hipStreamSynchronize(plan)");
  if (hs->err) {
    if (hs->err & (kErrInternal | kErrRelayout))
      return fail(AGCN_ERR_HIP, "internal plan consistency check failed");
    return fail(AGCN_ERR_INVALID_INPUT, "invalid CSR (row pointer or column index)");
  }
  p->n_entries = hs->n_entries;
  p->hub_first_entry = hs->hub_first_entry;
  p->n_hub_rows = 0;
  p->hub_first_row = (int32_t)n;
  p->max_deg = hs->max_deg;
  return AGCN_OK;
}

// The hub rows' column windows, for plans whose hub rows are dense enough
// (kWinMinPairs nonzeros per row and window on average, counted from the hub
// chunks: a row of c chunks holds more than (c - 1) * H nonzeros). Queued
// after the summary read-back, last of the plan's kernels; the table lies in
// the plan's working buffers (`space`, `cap` bytes). An execute on another
// stream waits for it as for the plan's other kernels.
int build_hub_windows(agcn_plan* p, int32_t n_chunks, int32_t* space, size_t cap,
                      hipStream_t st) {
  const int64_t n_hub = p->n_hub_rows;
  if (p->flags != 0 || n_hub < kWinMinHubRows || !hub_windows_setting()) return AGCN_OK;
  const int64_t n_win = ceil_div64(p->n_cols, kWinCols);
  const int64_t hub_nnz_lb = ((int64_t)n_chunks - n_hub) * p->H;
  if (hub_nnz_lb < (int64_t)kWinMinPairs * n_hub * n_win) return AGCN_OK;
  if ((size_t)(n_win + 1) * (size_t)n_hub * sizeof(int32_t) > cap)
    return fail(AGCN_ERR_HIP, "internal: hub window table larger than its reserved space");
  p->win_tab = space;
  p->n_win = (int32_t)n_win;
  const int64_t waves = n_hub * ceil_div64(n_win + 1, kWinTableSpan);
  const unsigned grid = (unsigned)std::min<int64_t>(grid_for(waves, kThreads / 64), 65536);
  k_hub_win_table<<<grid, kThreads, 0, st>>>(p->rowptr_s, p->colidx_s, p->hub_first_row,
                                             (int32_t)n_hub, (int32_t)n_win, p->win_tab);
  return check_launch("k_hub_win_table");
}

int build_plan_block(agcn_plan* p, const int32_t* d_rowptr, const int32_t* d_colidx,
                     const float* d_vals, hipStream_t st) {
  const int64_t n = p->n_rows, nnz = p->nnz;
  const int32_t W = p->W, Z = p->Z, DB = p->deg_bound, H = p->H;
  const int64_t ent_ub = n + nnz / H + 1;         // every entry holds a row or a full chunk
  const int64_t hub_ub = std::min<int64_t>(n, nnz / (DB + 1));
  const int64_t S = (int64_t)DB + 1 + hub_ub;     // segments: degree classes + hub rows
  const int64_t chunk_ub = nnz / H + hub_ub + 1;   // hub-chunk entries
  const int64_t n_tiles = ceil_div64(n, kRadixTile);
  const int64_t n_counts = ceil_div64(std::max<int64_t>(n, chunk_ub), kRadixTile) * kRadixBins;
  const int64_t scan_max = std::max<int64_t>({n_counts, n + 1, S + 1});
  const int64_t n_partials = ceil_div64(scan_max, kScanBlock) + 1;
  if (ent_ub >= INT32_MAX || S + 1 >= INT32_MAX || n_counts > kScanMaxN)
    return fail(AGCN_ERR_UNSUPPORTED, "graph too large for the int32 metadata format");

  Layout L;
  const size_t o_perm = L.take(4 * n);
  const size_t o_rowptr_s = L.take(4 * (n + 1));
  const size_t o_colidx_s = L.take(4 * nnz);
  const size_t o_vals_s = L.take(4 * nnz);
  const size_t o_meta = L.take(16 * ent_ub);
  const size_t o_hub = L.take(4 * (hub_ub + 1));
  const size_t o_order = L.take(4 * ent_ub);
  // working buffers
  const size_t o_deg = L.take(4 * n);
  const size_t o_keys = L.take(4 * n);    // sorted degrees end here
  const size_t o_keys2 = L.take(4 * n);
  const size_t o_ids2 = L.take(4 * n);
  const size_t o_counts = L.take(4 * n_counts);
  // The hub rows' window table, when the plan gets one, is written over these
  // five buffers (its kernel is the plan's last; nothing reads them after the
  // plan), padded to its largest size: a table is only built when the hub rows
  // average kWinMinPairs nonzeros per window, so it holds at most
  // nnz / kWinMinPairs + hub rows entries.
  const int64_t n_win_max = ceil_div64(p->n_cols, kWinCols);
  const int64_t win_ub =
      p->flags == 0 && hub_ub >= kWinMinHubRows
          ? std::min<int64_t>(hub_ub * (n_win_max + 1), nnz / kWinMinPairs + hub_ub)
          : 0;
  const size_t win_span = L.off - o_deg;
  if ((size_t)(4 * win_ub) > win_span) L.take((size_t)(4 * win_ub) - win_span);
  const size_t win_cap = std::max<size_t>(win_span, (size_t)(4 * win_ub));
  const size_t o_partials = L.take(4 * n_partials);
  const size_t o_cls = L.take(4 * (DB + 2));
  const size_t o_nb = L.take(4 * S);
  const size_t o_seg = L.take(4 * (S + 1));
  const size_t o_err = L.take(64);
  const size_t o_dmax = L.take(64);
  const int64_t n_deg_blocks = ceil_div64(n, kDegRows);
  // Column-check chunks: at least kColCheckChunk entries, at most
  // kColCheckMaxBlocks of them.
  int64_t col_chunk = kColCheckChunk;
  if (nnz > col_chunk * kColCheckMaxBlocks)
    col_chunk = ceil_div64(ceil_div64(nnz, kColCheckMaxBlocks), kColCheckChunk) * kColCheckChunk;
  // k_degree checks the columns when the short sort's summary is to be read
  // before its last relayout (graphs of at most kEarlyCheckMaxNnz nonzeros);
  // otherwise the relayout copies check them for free.
  const long long early_max = test_early_check_nnz();
  const bool early_check =
      n > 0 && DB >= kTailKey && nnz <= (early_max >= 0 ? early_max : kEarlyCheckMaxNnz);
  const int64_t n_col_chunks = early_check ? ceil_div64(nnz, col_chunk) : 0;
  const size_t o_bmax = L.take(4 * 4 * (n_deg_blocks + 1));  // maxima, (unused), tails, lows
  const size_t o_berr = L.take(4 * (n_deg_blocks + n_col_chunks + 1));  // error flags
  const size_t o_hsort = L.take(4 * 5 * chunk_ub);  // keys in, 2 x keys, 2 x ids
  const size_t o_hgate = L.take(64);
  const size_t o_tickets = L.take(4 * kMaxChainedScans);
  const size_t o_status = L.take(8 * n_partials);
  const size_t o_info = L.take(sizeof(TailInfo));

  void* base = nullptr;
  size_t got = 0;
  int rc = device_alloc(p->device, L.off, st, &base, &got);
  if (rc) return rc;
  char* b = static_cast<char*>(base);
  p->base = base;
  p->bytes = got;
  p->perm = reinterpret_cast<int32_t*>(b + o_perm);
  p->rowptr_s = reinterpret_cast<int32_t*>(b + o_rowptr_s);
  p->colidx_s = reinterpret_cast<int32_t*>(b + o_colidx_s);
  p->vals_s = reinterpret_cast<float*>(b + o_vals_s);
  p->meta = reinterpret_cast<int4*>(b + o_meta);
  p->hub_chunk_off = reinterpret_cast<int32_t*>(b + o_hub);
  p->order = reinterpret_cast<int32_t*>(b + o_order);
  int32_t* const win_space = reinterpret_cast<int32_t*>(b + o_deg);
  int32_t* deg = reinterpret_cast<int32_t*>(b + o_deg);
  int32_t* keys = reinterpret_cast<int32_t*>(b + o_keys);
  int32_t* keys2 = reinterpret_cast<int32_t*>(b + o_keys2);
  int32_t* ids2 = reinterpret_cast<int32_t*>(b + o_ids2);
  int32_t* counts = reinterpret_cast<int32_t*>(b + o_counts);
  int32_t* partials = reinterpret_cast<int32_t*>(b + o_partials);
  int32_t* cls = reinterpret_cast<int32_t*>(b + o_cls);
  int32_t* nb = reinterpret_cast<int32_t*>(b + o_nb);
  int32_t* seg = reinterpret_cast<int32_t*>(b + o_seg);
  uint32_t* err = reinterpret_cast<uint32_t*>(b + o_err);
  p->err_word = err;
  int32_t* dmax = reinterpret_cast<int32_t*>(b + o_dmax);
  int32_t* bmax = reinterpret_cast<int32_t*>(b + o_bmax);
  int32_t* hsort = reinterpret_cast<int32_t*>(b + o_hsort);
  int32_t* hgate = reinterpret_cast<int32_t*>(b + o_hgate);
  TailInfo* info = reinterpret_cast<TailInfo*>(b + o_info);

  PlanSummary* dsum = nullptr;
  PlanSummary* hs = pinned_summary(&dsum);
  if (hs == nullptr) return fail(AGCN_ERR_OUT_OF_MEMORY, "pinned host buffer allocation failed");
  // No kernel of this thread's previous plan writes the summary any more: its
  // last write came before the flag that plan waited for.
  *hs = PlanSummary{};
  uint32_t* berr = reinterpret_cast<uint32_t*>(b + o_berr);
  int32_t* btail = bmax + 2 * (n_deg_blocks + 1);
  int32_t* blow = bmax + 3 * (n_deg_blocks + 1);
  // A small graph's plan: one workgroup up to the partition (k_plan_tiny).
  const bool tiny = n > 0 && n <= kTinyMaxRows && nnz <= kTinyMaxNnz && test_tiny_plan() != 0;
  // The short sort needs every hub row in the tail (DB >= kTailKey).
  const bool short_sort = n > 0 && DB >= kTailKey && !tiny;
  ChainedScans chain;
  chain.status = reinterpret_cast<unsigned long long*>(b + o_status);
  chain.capacity = n_partials;
  chain.tickets = reinterpret_cast<int32_t*>(b + o_tickets);
  const DegreeBlocks dblocks{bmax,  berr, btail, blow, (int32_t)n_deg_blocks,
                            (int32_t)(n_deg_blocks + n_col_chunks), dmax, err, dsum};
  // With the short sort, k_degree clears the error word and the tickets and
  // the scan of its counts does the reduction (or launches k_dmax). Its
  // column checks make every input error known at the reduction, before the
  // short sort's second half (n > 0 whenever nnz > 0).
  if (n > 0 && !tiny)
    k_degree<<<(unsigned)(n_deg_blocks + n_col_chunks), kThreads, 0, st>>>(
        (int32_t)n, nnz, d_rowptr, deg, bmax, berr, btail, blow, short_sort ? counts : nullptr,
        (int32_t)n_tiles, short_sort ? err : nullptr, short_sort ? chain.tickets : nullptr,
        (int32_t)n_deg_blocks, ColumnCheck{d_colidx, nnz, col_chunk, p->n_cols, 0});
  if (!short_sort && !tiny) k_dmax<<<1, kScanTopThreads, 0, st>>>(dblocks, chain.tickets);
  if ((rc = check_launch("k_degree"))) return rc;
  const unsigned rgrid = grid_for(n_tiles, kRadixWaves);
  bool short_done = false, have_max = false;
  int32_t md = 0;
  // When the counts scan takes several launches (graphs of over 512 K rows),
  // the reduction runs first and the host reads the tail size before
  // queueing the short sort's first pass, which a tail over the cap would
  // waste; otherwise the first tile of the scan does the reduction and the
  // read-back arrives while the pass runs.
  const bool reduce_first =
      short_sort && n_tiles * kRadixBins > (int64_t)kChainedMaxTiles * kScanBlock;
  bool take_short = short_sort;
  const int32_t cap = tail_cap_setting();
  if (reduce_first) {
    k_dmax<<<1, kScanTopThreads, 0, st>>>(dblocks, chain.tickets);
    if ((rc = check_launch("k_dmax"))) return rc;
    if ((rc = wait_flag(&hs->dmax_ready, st, "maximum degree read-back"))) return rc;
    md = hs->max_deg;
    have_max = true;
    take_short = hs->n_tail >= 0 && hs->n_tail <= cap;
  }
  if (take_short) {
    // Pass one of the short sort.
    if ((rc = scan_exclusive(counts, n_tiles * kRadixBins, counts, nullptr, partials, err, st,
                             nullptr, 0, &chain, reduce_first ? DegreeBlocks{} : dblocks)))
      return rc;
    k_scatter_low<<<rgrid, kThreads, 0, st>>>((int32_t)n, deg, counts, (int32_t)n_tiles, keys,
                                              p->perm, p->rowptr_s, keys2, ids2, err);
    if ((rc = check_launch("k_scatter_low"))) return rc;
    // The second half is queued at once: its kernels read the tail's size,
    // the maximum degree and the lower nonzeros on the device and return at
    // once when the tail is over the cap, so the GPU need not wait for the
    // host's read-back. Their copies loop over tiles on grids of a size that
    // needs none of it.
    TailArgs ta;
    ta.n = (int32_t)n;
    ta.nnz = (int32_t)nnz;
    ta.W = W;
    ta.Z = Z;
    ta.DB = DB;
    ta.H = H;
    ta.cap = cap;
    ta.check_cols = early_check ? INT32_MAX : p->n_cols;
    ta.publish = early_check;
    ta.key_base = kTailKey;
    ta.tail_keys = keys2;
    ta.tail_ids = ids2;
    ta.rowptr_in = nullptr;
    ta.offsets = counts;
    ta.n_tiles = (int32_t)n_tiles;
    ta.keys = keys;
    ta.perm = p->perm;
    ta.rowptr_s = p->rowptr_s;
    ta.cls = cls;
    ta.seg = seg;
    ta.info = info;
    ta.sum = dsum;
    ta.dmax = dmax;
    ta.err = err;
    const int32_t cus = device_cus(p->device);
    const int64_t max_tiles = ceil_div64(nnz, kRelayTile);
    // One 1024-thread workgroup per CU (the tail's LDS), the tail's on one.
    const int32_t n_groups = (int32_t)std::max<int64_t>(
        1, std::min<int64_t>(ceil_div64(max_tiles, kTilesPerTailGroup), cus - 1));
    k_tail_relayout<<<(unsigned)(1 + n_groups), kTailThreads, 0, st>>>(
        ta, n_groups, d_rowptr, d_colidx, d_vals, p->colidx_s, p->vals_s, err);
    if ((rc = check_launch("k_tail_relayout"))) return rc;
    const int32_t n_fill = (int32_t)std::min<int64_t>(grid_for(ent_ub, kThreads), 64);
    const int32_t n_copy = (int32_t)std::max<int64_t>(
        1, std::min<int64_t>(max_tiles, (int64_t)kRelayGroupsPerCu * cus - n_fill));
    k_relayout_fill<<<(unsigned)(n_fill + n_copy), kThreads, 0, st>>>(
        n_fill, n_copy, (int32_t)n, nnz, d_rowptr, d_colidx, d_vals, p->perm, p->rowptr_s,
        p->colidx_s, p->vals_s, keys, cls, seg, info, W, Z, DB, H, p->meta, ent_ub,
        (int32_t)hub_ub, p->hub_chunk_off, p->order, dmax, cap, ta.check_cols, err);
    if ((rc = check_launch("k_relayout_fill"))) return rc;
    if (!early_check) {
      k_publish<<<1, 64, 0, st>>>(err, dsum, dmax, (int32_t)n, cap);
      if ((rc = check_launch("k_publish"))) return rc;
    }
    if (!have_max) {
      if ((rc = wait_flag(&hs->dmax_ready, st, "maximum degree read-back"))) return rc;
      md = hs->max_deg;
      have_max = true;
    }
    // The same test the two kernels made; otherwise they returned at once.
    short_done = hs->n_tail >= 0 && hs->n_tail <= cap;
  }
  if (tiny) {
    TailArgs ta{};
    ta.n = (int32_t)n;
    ta.nnz = (int32_t)nnz;
    ta.W = W;
    ta.Z = Z;
    ta.DB = DB;
    ta.H = H;
    ta.cap = kTailCap;
    ta.check_cols = INT32_MAX;  // checked by k_plan_tiny
    ta.publish = 1;
    ta.key_base = 0;
    ta.rowptr_in = d_rowptr;
    ta.offsets = nullptr;
    ta.keys = keys;
    ta.perm = p->perm;
    ta.rowptr_s = p->rowptr_s;
    ta.cls = cls;
    ta.seg = seg;
    ta.info = info;
    ta.sum = dsum;
    ta.dmax = dmax;
    ta.err = err;
    k_plan_tiny<<<1, kTailThreads, 0, st>>>(ta, p->n_cols, d_rowptr, d_colidx, err, chain.tickets,
                                            dmax);
    if ((rc = check_launch("k_plan_tiny"))) return rc;
    const int32_t cus = device_cus(p->device);
    const int32_t n_fill = (int32_t)std::min<int64_t>(grid_for(ent_ub, kThreads), 64);
    const int32_t n_copy = (int32_t)std::max<int64_t>(
        1, std::min<int64_t>(ceil_div64(nnz, kRelayTile), (int64_t)kRelayGroupsPerCu * cus - n_fill));
    k_relayout_fill<<<(unsigned)(n_fill + n_copy), kThreads, 0, st>>>(
        n_fill, n_copy, (int32_t)n, nnz, d_rowptr, d_colidx, d_vals, p->perm, p->rowptr_s,
        p->colidx_s, p->vals_s, keys, cls, seg, info, W, Z, DB, H, p->meta, ent_ub,
        (int32_t)hub_ub, p->hub_chunk_off, p->order, dmax, kTailCap, INT32_MAX, err);
    if ((rc = check_launch("k_relayout_fill"))) return rc;
    short_done = true;
  }
  if (n > 0 && !short_done) {
    // Stable LSD radix sort of row ids by degree, 8-bit digits. Unless the
    // maximum degree is already known, passes 0 and 1 are queued before the
    // host reads it (pass 1 returns at once on the device when one pass
    // suffices), so the GPU keeps busy while the read-back reaches the host;
    // passes 2 and 3 follow if needed.
    const RadixBufs bufs{deg, {keys, keys2}, {p->perm, ids2}};
    constexpr int kPassesBeforeReadback = 2;
    int passes = kPassesBeforeReadback;
    for (int pass = 0; pass < passes; ++pass) {
      k_radix_hist<<<rgrid, kThreads, 0, st>>>((int32_t)n, bufs, pass, counts, (int32_t)n_tiles, err,
                                               dmax);
      if ((rc = check_launch("k_radix_hist"))) return rc;
      if ((rc = scan_exclusive(counts, n_counts, counts, nullptr, partials, err, st, dmax, pass,
                               &chain)))
        return rc;
      k_radix_scatter<<<rgrid, kThreads, 0, st>>>((int32_t)n, bufs, pass, counts, (int32_t)n_tiles,
                                                  err, dmax);
      if ((rc = check_launch("k_radix_scatter"))) return rc;
      if (pass == kPassesBeforeReadback - 1) {
        if (!have_max) {
          if ((rc = wait_flag(&hs->dmax_ready, st, "maximum degree read-back"))) return rc;
          md = hs->max_deg;
        }
        int bits = 0;
        while (bits < 31 && (int64_t(1) << bits) <= md) ++bits;
        passes = std::max(kPassesBeforeReadback, (bits + 7) / 8);
      }
    }
  }
  if (!short_done) {
    // rowptr_s = exclusive scan of the sorted degrees; rowptr_s[n] = nnz.
    if ((rc = scan_exclusive(keys, n, p->rowptr_s, p->rowptr_s + n, partials, err, st, nullptr, 0,
                             &chain)))
      return rc;
    if (nnz > 0) {
      const unsigned rgrid = (unsigned)std::min<int64_t>(
          ceil_div64(nnz, kRelayTile), (int64_t)kRelayGroupsPerCu * device_cus(p->device));
      k_relayout<<<rgrid, kThreads, 0, st>>>(
          (int32_t)n, nnz, p->n_cols, d_rowptr, d_colidx, d_vals, p->perm, p->rowptr_s,
          p->colidx_s, p->vals_s, err);
      if ((rc = check_launch("k_relayout"))) return rc;
    }
    k_class_start<<<grid_for(n + 1, kThreads), kThreads, 0, st>>>((int32_t)n, keys, DB, cls, err);
    k_seg_count<<<grid_for(S, kThreads), kThreads, 0, st>>>((int32_t)n, keys, cls, W, Z, DB, H,
                                                           (int32_t)S, nb, err);
    if ((rc = check_launch("partition counts"))) return rc;
    if ((rc = scan_exclusive(nb, S, seg, seg + S, partials, err, st, nullptr, 0, &chain))) return rc;
    const unsigned mgrid = (unsigned)std::min<int64_t>(grid_for(ent_ub, kThreads), 16384);
    k_partition_fill<<<mgrid, kThreads, 0, st>>>((int32_t)n, p->rowptr_s, keys, cls, seg,
                                                 (int32_t)S, W, Z, DB, H, p->meta, ent_ub,
                                                 (int32_t)hub_ub, p->hub_chunk_off, p->order, dsum,
                                                 err);
    if ((rc = check_launch("partition fill"))) return rc;
  }

  if ((rc = wait_flag(&hs->done, st, "plan summary read-back"))) return rc;
  if (hs->err) {
    std::string why;
    if (hs->err & kErrRowptrStart) why += " rowptr[0] != 0;";
    if (hs->err & kErrRowptrOrder) why += " rowptr decreases or leaves [0, nnz];";
    if (hs->err & kErrRowptrEnd) why += " rowptr[n_rows] != nnz;";
    if (hs->err & kErrColumn) why += " column index outside [0, n_cols);";
    if (hs->err & (kErrInternal | kErrRelayout))
      return fail(AGCN_ERR_HIP, "internal plan consistency check failed");
    return fail(AGCN_ERR_INVALID_INPUT, "invalid CSR:" + why);
  }
  p->n_entries = hs->n_entries;
  p->hub_first_entry = hs->hub_first_entry;
  p->n_hub_rows = hs->n_hub_rows;
  p->hub_first_row = hs->hub_first_row;
  p->max_deg = hs->max_deg;

  // Hub chunks in column order: queued after the summary read-back (an
  // execute on another stream waits for the plan's kernels, see
  // plan_ready_event).
  const int32_t n_chunks = p->n_hub_rows > 0 ? p->n_entries - p->hub_first_entry : 0;
  const int32_t* sorted_ids = nullptr;
  // Only long rows have chunks with narrow column ranges: sort when the hub
  // rows average at least kOrderMinChunks chunks, or when there are so many
  // chunks that even a small gain per chunk repays the ~20 us sort (measured:
  // 2.4% off the 2.4 M-row graph's execute; a net loss on a 2.4 M-nnz graph).
  const bool long_hubs = (int64_t)n_chunks >= (int64_t)kOrderMinChunks * p->n_hub_rows;
  if (n_chunks > 0 && hub_order_setting() && (long_hubs || n_chunks >= kOrderMinTotalChunks)) {
    p->hub_wide = long_hubs;
    if (test_order_sort_fails()) k_raise<<<1, 64, 0, st>>>(err, kErrInternal);
    const int64_t ct = ceil_div64(n_chunks, kRadixTile);
    int32_t* hk_in = hsort;
    const RadixBufs hb{hk_in, {hsort + chunk_ub, hsort + 2 * chunk_ub},
                       {hsort + 3 * chunk_ub, hsort + 4 * chunk_ub}};
    k_hub_keys<<<grid_for(n_chunks, kThreads), kThreads, 0, st>>>(
        p->meta, p->colidx_s, p->hub_first_entry, n_chunks, p->n_cols, hk_in, hgate);
    const unsigned hgrid = grid_for(ct, kRadixWaves);
    for (int pass = 0; pass < 2; ++pass) {
      k_radix_hist<<<hgrid, kThreads, 0, st>>>(n_chunks, hb, pass, counts, (int32_t)ct, err, hgate);
      if ((rc = scan_exclusive(counts, ct * kRadixBins, counts, nullptr, partials, err, st, nullptr,
                               0, &chain)))
        return rc;
      k_radix_scatter<<<hgrid, kThreads, 0, st>>>(n_chunks, hb, pass, counts, (int32_t)ct, err,
                                                  hgate);
    }
    sorted_ids = hb.ids[0];
    k_order_fill<<<grid_for(p->n_entries, kThreads), kThreads, 0, st>>>(
        p->order, p->n_entries, p->hub_first_entry, n_chunks, sorted_ids, err);
  }
  if ((rc = check_launch("launch order"))) return rc;
  return build_hub_windows(p, n_chunks, win_space, win_cap, st);
}

}  // namespace

int build_plan(agcn_plan* p, const int32_t* d_rowptr, const int32_t* d_colidx,
               const float* d_vals, hipStream_t st) {
  p->stream = st;
  if (p->flags & AGCN_PLAN_WARP_LEVEL) return build_plan_warp_level(p, d_rowptr, d_colidx, d_vals, st);
  const int rc = build_plan_block(p, d_rowptr, d_colidx, d_vals, st);
  // A plan that failed after launching kernels lets them finish first: they
  // write this thread's pinned summary, which the next plan polls.
  if (rc != AGCN_OK) (void)hipStreamSynchronize(st);
  return rc;
}

}  // namespace agcn
