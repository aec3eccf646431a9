// Execute: Y = A X over the block-level partition (Sec. III-C, III-D).
//
// k_spmm: one workgroup per (metadata entry, column slice). A column slice is
// 32 floats -- one 128-byte line of an X row -- unless F is smaller. The grid
// is (entries, slices) and workgroups are dispatched x-fastest, so the whole
// GPU sweeps the entries for slice 0, then slice 1, ...: at any moment the
// L2 of every XCD holds only 128-byte pieces of X rows, which lets it keep
// 8x more rows than whole 1-KiB rows (F = 256) and raises its hit rate on the
// power-law column reuse. Slices narrower than a line would fetch unused
// halves, so the slice never drops below 128 bytes.
//   1. The entry {deg, loc, row, info} is read once (uniform, scalar load).
//   2. Its column indices and values -- contiguous in the sorted CSR -- are
//      staged into LDS with plain loads (measured: non-temporal ones were
//      2-6% slower), 4 pairs per thread in flight.
//      The LDS index is padded by one word per 32 so the vwarps of a wave,
//      which read slices a fixed stride apart, fall in different banks.
//   3. Virtual warps (the paper's warps): a row of degree d is covered by
//      ceil(d / warp_nzs) consecutive vwarps of warp_nzs nnz. Each vwarp owns
//      L lanes laid across the slice's columns, one float4 per lane (the
//      paper's combined warp, built from 64-lane waves: 64 / L vwarps share a
//      wave). Workgroup threads map to (vwarp, lane) in `rounds` passes when
//      W * L exceeds 1024.
//   4. Each lane gathers X rows with 16-byte loads, 8 in flight, and
//      accumulates with fp32 FMA in nnz order.
//   5. Rows held by one vwarp store straight to Y (non-temporal). Rows split
//      over several vwarps add their partials from LDS in vwarp order; hub
//      chunks (deg > deg_bound) add all W slices in order and write one
//      partial row to the workspace. No atomics: results are bitwise
//      reproducible and independent of a row's position in the sorted order.
// k_hub_reduce: one workgroup per (hub row, column slice); G lane groups each
//   add a contiguous run of the row's chunk partials, then a fixed pairwise
//   tree combines the G sums and the row is written once.
//
// Launch order (built by the plan): hub-chunk entries sorted by the first
// column they gather, so chunks running side by side read neighbouring X rows
// and share them in L2; then the other entries heaviest first (the metadata
// is in ascending degree order).
//
// Plans with hub-row windows (dense hub rows; the plan's window table), at
// F >= 64 on the float4 path with room for the window partials: k_spmm runs
// over the entries after the hub chunks only, and k_hub_win +
// k_hub_win_reduce aggregate the hub rows window by window (described at the
// kernels below).
//
// Every kernel that writes Y takes `act` and applies the layer's activation
// there (ReLU, Sec. II-A), after a split row's final sum.
//
// The two baselines of Table II live here too: k_spmm_wl + k_wl_fixup execute
// the warp-level partition, k_spmm_colloop the block-level partition without
// the combined warp (one float per lane, a loop over F).
#include <algorithm>
#include <climits>
#include <cstdlib>
#include <mutex>

#include <hip/hip_ext.h>

#include "agcn_internal.hpp"

namespace agcn {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));

template <int VW>
struct VecOf;
template <>
struct VecOf<4> {
  using T = f4;
};
template <>
struct VecOf<1> {
  using T = float;
};

constexpr int kDefaultSliceCols = 32;  // one 128-byte line per X row per pass
// Slice width of column-ordered hub chunks of long hub rows (two lines).
constexpr int kHubSliceCols = 64;
constexpr int kStageUnroll = 4;
constexpr int kGatherUnroll = 8;

__device__ inline int pad_idx(int i) { return i + (i >> 5); }

// Partial-sum slots: one padding slot per 8 float4 (per 32 floats) keeps
// rows that are a multiple of 128 bytes apart in different banks.
template <int VW>
__device__ __host__ inline int part_idx(int i) {
  return VW == 4 ? i + (i >> 3) : i + (i >> 5);
}

__device__ inline f4 fma_v(float a, f4 x, f4 acc) {
  f4 r;
  r.x = __builtin_fmaf(a, x.x, acc.x);
  r.y = __builtin_fmaf(a, x.y, acc.y);
  r.z = __builtin_fmaf(a, x.z, acc.z);
  r.w = __builtin_fmaf(a, x.w, acc.w);
  return r;
}
__device__ inline float fma_v(float a, float x, float acc) { return __builtin_fmaf(a, x, acc); }

// Epilogue at the Y write: act = 1 applies ReLU (negative values become 0;
// NaN and -0 pass through, as max(v, 0) defined by v < 0 ? 0 : v).
__device__ inline float act_v(float v, int32_t act) { return (act && v < 0.0f) ? 0.0f : v; }
__device__ inline f4 act_v(f4 v, int32_t act) {
  return act ? f4{act_v(v.x, 1), act_v(v.y, 1), act_v(v.z, 1), act_v(v.w, 1)} : v;
}

// acc = sum over j in [s0, s0 + len) of val[j] * X[col[j], lane], in order.
// Groups of kGatherUnroll loads are issued before the first is consumed; the
// tail of a group is predicated, so short slices still overlap their loads.
template <int VW>
__device__ inline typename VecOf<VW>::T gather_row(const int32_t* s_col, const float* s_val,
                                                   int s0, int len,
                                                   const typename VecOf<VW>::T* __restrict__ Xv,
                                                   int64_t ldv, int32_t lane_col) {
  using V = typename VecOf<VW>::T;
  V acc = V(0.0f);
  for (int j = 0; j < len; j += kGatherUnroll) {
    V x[kGatherUnroll];
    float a[kGatherUnroll];
#pragma unroll
    for (int u = 0; u < kGatherUnroll; ++u) {
      if (j + u < len) {
        const int p = pad_idx(s0 + j + u);
        a[u] = s_val[p];
        x[u] = Xv[(int64_t)s_col[p] * ldv + lane_col];
      }
    }
#pragma unroll
    for (int u = 0; u < kGatherUnroll; ++u)
      if (j + u < len) acc = fma_v(a[u], x[u], acc);
  }
  return acc;
}

// LT > 0: lanes per vwarp fixed at compile time; LT == 0: taken from L.
template <int VW, int LT>
__global__ __launch_bounds__(1024) void k_spmm(
    const int4* __restrict__ meta, const int32_t* __restrict__ order, int32_t entry_base,
    int32_t hub_first_entry,
    int32_t deg_bound, int32_t W, const int32_t* __restrict__ colidx_s,
    const float* __restrict__ vals_s, const int32_t* __restrict__ perm, const float* __restrict__ X,
    int64_t ldx, float* __restrict__ Y, int64_t ldy, float* __restrict__ ws, int32_t F,
    int32_t col_base, int32_t slice_cols, int32_t L_rt, int32_t rounds, int32_t cap_pad,
    int32_t act) {
  using V = typename VecOf<VW>::T;
  const int L = LT > 0 ? LT : L_rt;
  extern __shared__ float smem[];
  int32_t* s_col = reinterpret_cast<int32_t*>(smem);
  float* s_val = smem + cap_pad;
  V* s_part = reinterpret_cast<V*>(smem + 2 * cap_pad);

  const int T = blockDim.x;
  const int32_t b = order[entry_base + (int32_t)blockIdx.x];
  const int32_t col0 = col_base + (int32_t)blockIdx.y * slice_cols;
  const int4 m = meta[b];
  const int32_t deg = m.x, loc = m.y, row = m.z, info = m.w;
  const bool hub = deg > deg_bound;
  const int32_t rows = info & 0xFFFF;
  const int32_t n_e = hub ? info : rows * deg;

  for (int i0 = 0; i0 < n_e; i0 += T * kStageUnroll) {
    int32_t c[kStageUnroll];
    float v[kStageUnroll];
#pragma unroll
    for (int u = 0; u < kStageUnroll; ++u) {
      const int i = i0 + u * T + threadIdx.x;
      if (i < n_e) {
        c[u] = colidx_s[loc + i];
        v[u] = vals_s[loc + i];
      }
    }
#pragma unroll
    for (int u = 0; u < kStageUnroll; ++u) {
      const int i = i0 + u * T + threadIdx.x;
      if (i < n_e) {
        s_col[pad_idx(i)] = c[u];
        s_val[pad_idx(i)] = v[u];
      }
    }
  }
  __syncthreads();

  const V* __restrict__ Xv = reinterpret_cast<const V*>(X + col0);
  const int64_t ldxv = ldx / VW;
  if (!hub) {
    const int32_t wn = (int32_t)((uint32_t)info >> 16);
    const int32_t wpr = deg > 0 ? (deg + wn - 1) / wn : 1;  // vwarps per row
    const int32_t nv = rows * wpr;
    for (int k = 0; k < rounds; ++k) {
      const int vt = threadIdx.x + k * T;
      const int v = vt / L, l = vt - v * L;
      if (v < nv) {
        const int rl = v / wpr, part = v - rl * wpr;
        const int s0 = rl * deg + part * wn;
        const int len = deg > 0 ? min(wn, deg - part * wn) : 0;
        const V acc = gather_row<VW>(s_col, s_val, s0, len, Xv, ldxv, l);
        if (wpr == 1) {
          V* yr = reinterpret_cast<V*>(Y + (int64_t)perm[row + rl] * ldy + col0);
          __builtin_nontemporal_store(act_v(acc, act), yr + l);
        } else {
          s_part[part_idx<VW>(v * L + l)] = acc;
        }
      }
    }
    if (wpr > 1) {  // uniform over the workgroup
      __syncthreads();
      for (int k = 0; k < rounds; ++k) {
        const int vt = threadIdx.x + k * T;
        const int r = vt / L, l = vt - r * L;
        if (r < rows) {
          V sum = s_part[part_idx<VW>((r * wpr) * L + l)];
          for (int q = 1; q < wpr; ++q) sum += s_part[part_idx<VW>((r * wpr + q) * L + l)];
          V* yr = reinterpret_cast<V*>(Y + (int64_t)perm[row + r] * ldy + col0);
          __builtin_nontemporal_store(act_v(sum, act), yr + l);
        }
      }
    }
  } else {
    const int32_t sl = (n_e + W - 1) / W;  // nnz per vwarp inside the chunk
    for (int k = 0; k < rounds; ++k) {
      const int vt = threadIdx.x + k * T;
      const int v = vt / L, l = vt - v * L;
      if (v < W) {
        const int s0 = v * sl;
        const int left = n_e - s0;
        const int len = left < 0 ? 0 : (left < sl ? left : sl);
        s_part[part_idx<VW>(v * L + l)] = gather_row<VW>(s_col, s_val, s0, len, Xv, ldxv, l);
      }
    }
    __syncthreads();
    for (int k = 0; k < rounds; ++k) {
      const int l = threadIdx.x + k * T;
      if (l < L) {
        V sum = s_part[part_idx<VW>(l)];
        for (int v = 1; v < W; ++v) sum += s_part[part_idx<VW>(v * L + l)];
        V* wr = reinterpret_cast<V*>(ws + (int64_t)(b - hub_first_entry) * F + col0);
        wr[l] = sum;
      }
    }
  }
}

template <int VW>
__global__ __launch_bounds__(1024) void k_hub_reduce(const int32_t* __restrict__ hub_chunk_off,
                                                     int32_t hub_first_row,
                                                     const int32_t* __restrict__ perm,
                                                     const float* __restrict__ ws, int32_t F,
                                                     float* __restrict__ Y, int64_t ldy,
                                                     int32_t col_base, int32_t slice_cols,
                                                     int32_t L, int32_t G, int32_t act) {
  using V = typename VecOf<VW>::T;
  extern __shared__ float smem[];
  V* s_acc = reinterpret_cast<V*>(smem);  // [G][L]
  const int32_t h = blockIdx.x;
  const int32_t col0 = col_base + (int32_t)blockIdx.y * slice_cols;
  const int32_t c0 = hub_chunk_off[h], c1 = hub_chunk_off[h + 1];
  const int32_t nc = c1 - c0;
  const int g = threadIdx.x / L, l = threadIdx.x - g * L;
  const int32_t q = (nc + G - 1) / G;
  if (g < G) {
    V acc = V(0.0f);
    const int32_t a = c0 + g * q;
    const int32_t e = a + q < c1 ? a + q : c1;
    for (int32_t c = a; c < e; ++c)
      acc += reinterpret_cast<const V*>(ws + (int64_t)c * F + col0)[l];
    s_acc[g * L + l] = acc;
  }
  __syncthreads();
  for (int stride = G / 2; stride > 0; stride >>= 1) {
    if (g < stride) s_acc[g * L + l] += s_acc[(g + stride) * L + l];
    __syncthreads();
  }
  if (g == 0) {
    V* yr = reinterpret_cast<V*>(Y + (int64_t)perm[hub_first_row + h] * ldy + col0);
    __builtin_nontemporal_store(act_v(s_acc[l], act), yr + l);
  }
}

// Hub rows of at most MC chunks (every hub row of a plan whose maximum degree
// is at most MC * H): one vwarp of L lanes per (hub row, slice), each lane
// loading all of the row's chunk partials at once and adding them in chunk
// order. The tree of k_hub_reduce leaves most of its 16 lane groups idle on
// such rows and pays four barriers; the sum here is just as fixed (a
// different order, so Y may differ from the tree's in the last bits).
constexpr int kFlatThreads = 64;
constexpr int kFlatMaxChunks = 32;

template <int VW, int MC>
__global__ __launch_bounds__(kFlatThreads) void k_hub_reduce_flat(
    const int32_t* __restrict__ hub_chunk_off, int32_t hub_first_row,
    const int32_t* __restrict__ perm, const float* __restrict__ ws, int32_t F,
    float* __restrict__ Y, int64_t ldy, int32_t col_base, int32_t slice_cols, int32_t L,
    int32_t n_hub, int32_t act) {
  using V = typename VecOf<VW>::T;
  const int64_t t = (int64_t)blockIdx.x * kFlatThreads + threadIdx.x;
  const int32_t h = (int32_t)(t / L);
  const int l = (int)(t - (int64_t)h * L);
  if (h >= n_hub) return;
  const int32_t col0 = col_base + (int32_t)blockIdx.y * slice_cols;
  const int32_t c0 = hub_chunk_off[h];
  const int32_t nc = hub_chunk_off[h + 1] - c0;
  V part[MC];
#pragma unroll
  for (int k = 0; k < MC; ++k)
    if (k < nc) part[k] = reinterpret_cast<const V*>(ws + (int64_t)(c0 + k) * F + col0)[l];
  V acc = V(0.0f);
#pragma unroll
  for (int k = 0; k < MC; ++k)
    if (k < nc) acc += part[k];
  V* yr = reinterpret_cast<V*>(Y + (int64_t)perm[hub_first_row + h] * ldy + col0);
  __builtin_nontemporal_store(act_v(acc, act), yr + l);
}

// Hub rows over column windows (plans with a window table, F >= kWinMinF).
// One workgroup of 1024 threads per (row batch, window group, slice of
// kWinSliceCols columns); the row batches of one window group are adjacent
// in the grid, so they run side by side and share that part of X in L2. For
// each of its G windows of kWinCols columns the workgroup stages
// X[window, slice] (128 KiB) and its rows' ranges in the window in LDS. Each
// 16-lane group then takes kWinRowsPerGroup rows (batch row group + 64 r):
// lane l loads one (column, value) pair of a batch of 16 and the group walks
// the batch with row_newbcast DPP broadcasts, each pair one LDS float4 read
// and four FMAs per lane (lane l owns columns 4l..4l+3 of the slice). The
// next batch, of this row or of the next, is loaded before the current one is
// used. A row's sum stays in registers over the G windows (pairs of a window
// range alternate between two accumulators, added at the range's end) and
// one partial row per (hub row, window group) goes to ws; k_hub_win_reduce
// adds them in window order. Against the hub chunks, which gather every X row
// of a hub row through L2 (about 27 GB of 128-byte requests for 1.1e8 hub
// nonzeros at F = 64), X crosses L2 once per row batch and the gathers become
// LDS reads (measured on that graph: 1339 -> 582 us, the VALU then 84% busy).
// A row whose columns do not ascend still has its nonzeros split over the
// windows (the table's positions do not decrease); a pair whose column lies
// outside the current window counts zero here and flags its (row, window
// group), and k_hub_win_reduce adds those pairs from X.
template <int U>
__device__ inline int32_t row_bcast(int32_t v) {
  return __builtin_amdgcn_mov_dpp(v, 0x150 + U, 0xF, 0xF, true);  // row_newbcast:U
}

template <int U>
struct WinSteps {
  // Pairs 0..U-1 of the batch held by the group's lanes (o_l: byte offset of
  // the pair's X row in the staged window; v_l: the value's bits).
  __device__ static inline void run(int32_t o_l, int32_t v_l, const char* __restrict__ sxb,
                                    int32_t l16, f4& a0, f4& a1) {
    WinSteps<U - 1>::run(o_l, v_l, sxb, l16, a0, a1);
    const f4 x = *reinterpret_cast<const f4*>(sxb + row_bcast<U - 1>(o_l) + l16);
    const float v = __int_as_float(row_bcast<U - 1>(v_l));
    f4& a = ((U - 1) & 1) ? a1 : a0;
    a.x = __builtin_fmaf(v, x.x, a.x);
    a.y = __builtin_fmaf(v, x.y, a.y);
    a.z = __builtin_fmaf(v, x.z, a.z);
    a.w = __builtin_fmaf(v, x.w, a.w);
  }
};
template <>
struct WinSteps<0> {
  __device__ static inline void run(int32_t, int32_t, const char*, int32_t, f4&, f4&) {}
};

__global__ __launch_bounds__(1024) void k_hub_win(
    const int32_t* __restrict__ win_tab, int32_t n_hub, int32_t n_win, int32_t G, int32_t n_grp,
    const int32_t* __restrict__ colidx_s, const float* __restrict__ vals_s,
    const float* __restrict__ X, int64_t ldx, int32_t n_cols, float* __restrict__ ws, int32_t F) {
  constexpr int NR = kWinRowsPerGroup;
  __shared__ f4 sx[kWinCols * 16];
  __shared__ int32_t s_lo[kWinRows], s_hi[kWinRows];
  const int32_t hb0 = (int32_t)blockIdx.x * kWinRows;
  const int32_t kg = (int32_t)blockIdx.y;
  const int32_t col0 = (int32_t)blockIdx.z * kWinSliceCols;
  const int32_t cols = min(kWinSliceCols, F - col0);
  const int t = threadIdx.x;
  const int lane = t & 63, l = lane & 15;
  const int32_t grp = (t >> 6) * 4 + (lane >> 4);
  const int32_t l16 = l * 16;
  const bool lane_cols = 4 * l < cols;
  const int32_t k0 = kg * G, k1 = min(n_win, k0 + G);
  const int32_t n_my = min(kWinRows, n_hub - hb0);
  const char* sxb = reinterpret_cast<const char*>(sx);
  f4 acc[NR];
#pragma unroll
  for (int r = 0; r < NR; ++r) acc[r] = f4(0.0f);
  uint32_t stray_rows = 0;  // bit r: a pair of row r fell outside its window
  for (int32_t k = k0; k < k1; ++k) {
    __syncthreads();  // the previous window's reads are done
    for (int i = t; i < kWinCols * 16; i += 1024) {
      const int32_t xr = k * kWinCols + i / 16;
      const int q = i % 16;
      sx[i] = (xr < n_cols && 4 * q < cols)
                  ? reinterpret_cast<const f4*>(X + (int64_t)xr * ldx + col0)[q]
                  : f4(0.0f);
    }
    for (int i = t; i < n_my; i += 1024) {
      s_lo[i] = win_tab[(int64_t)k * n_hub + hb0 + i];
      s_hi[i] = win_tab[(int64_t)(k + 1) * n_hub + hb0 + i];
    }
    __syncthreads();
    if (grp >= n_my) continue;
    const int32_t cbase = k * kWinCols;
    // The lane's pair of the batch at [j, end): loaded unconditionally from a
    // clamped position (no branch around the loads) and used only in the next
    // iteration, so the loads overlap the current batch's steps.
    auto load_pair = [&](int32_t j, int32_t end, int32_t& c, int32_t& v, int32_t& in) {
      in = j + l < end;
      const int32_t at = in ? j + l : 0;
      c = colidx_s[at];
      v = __float_as_int(vals_s[at]);
    };
    int32_t s = s_lo[grp], e = s_hi[grp];
    int32_t c_n, v_n, in_n;
    load_pair(s, e, c_n, v_n, in_n);
#pragma unroll
    for (int r = 0; r < NR; ++r) {
      const int32_t i = grp + r * 64;
      if (i < n_my) {
        const bool more = r + 1 < NR && i + 64 < n_my;
        const int32_t s_nx = more ? s_lo[i + 64] : 0, e_nx = more ? s_hi[i + 64] : 0;
        f4 a1 = f4(0.0f);
        for (int32_t j = s; j < e; j += 16) {
          const int32_t c_c = c_n, v_c = v_n, in_c = in_n;
          const bool same = j + 16 < e;
          load_pair(same ? j + 16 : s_nx, same ? e : e_nx, c_n, v_n, in_n);
          // A column outside the window (a row whose columns do not ascend)
          // counts zero here; the reduction adds it from X.
          const bool inside = (uint32_t)(c_c - cbase) < (uint32_t)kWinCols;
          stray_rows |= (uint32_t)(in_c && !inside) << r;
          const bool use = in_c && inside;
          // (unsigned arithmetic: a masked lane's column may lie far outside)
          const int32_t off = (int32_t)((uint32_t)(c_c - cbase) << 8);
          WinSteps<16>::run(use ? off : 0, use ? v_c : 0, sxb, l16, acc[r], a1);
        }
        acc[r] += a1;
        if (s == e) load_pair(s_nx, e_nx, c_n, v_n, in_n);  // its preloaded batch was empty
        s = s_nx;
        e = e_nx;
      }
    }
  }
  // Stray flags after the partial rows, one word per (hub row, window group),
  // written (0 or 1) by the first slice's workgroups.
  if (blockIdx.z == 0) {
    int32_t* flags = reinterpret_cast<int32_t*>(ws + (int64_t)n_hub * n_grp * F);
#pragma unroll
    for (int r = 0; r < NR; ++r) {
      const uint64_t any = __ballot((stray_rows >> r) & 1u);
      const int32_t i = grp + r * 64;
      if (l == 0 && i < n_my)
        flags[(int64_t)(hb0 + i) * n_grp + kg] = ((any >> (lane & 48)) & 0xFFFFu) ? 1 : 0;
    }
  }
  if (!lane_cols) return;
#pragma unroll
  for (int r = 0; r < NR; ++r) {
    const int32_t i = grp + r * 64;
    if (i < n_my)
      reinterpret_cast<f4*>(ws + ((int64_t)(hb0 + i) * n_grp + kg) * F + col0)[l] = acc[r];
  }
}

// Y row of hub row h = the sum of its n_grp window-group partials, in window
// order, plus the pairs k_hub_win flagged as lying outside their window,
// gathered from X in position order. One workgroup per (hub row, 64
// columns): kWinReduceParts parts of 16 lanes (one float4 column each) take
// contiguous runs of the window groups -- each summing its run in four
// interleaved chains (kg mod 4, added pairwise), then its stray pairs -- and
// the part sums are added in part order. With a thread per column walking
// all the partials, the loads of a row were one dependent chain and the launch
// had a workgroup per 16 rows (153 us on 1000 rows x 489 groups at F = 64).
constexpr int kWinReduceParts = 8;

__global__ __launch_bounds__(kWinReduceParts * 16) void k_hub_win_reduce(
    const float* __restrict__ ws, int32_t n_hub, int32_t n_win, int32_t G, int32_t n_grp,
    int32_t F, const int32_t* __restrict__ win_tab, const int32_t* __restrict__ colidx_s,
    const float* __restrict__ vals_s, const float* __restrict__ X, int64_t ldx,
    const int32_t* __restrict__ perm, int32_t hub_first_row, float* __restrict__ Y, int64_t ldy,
    int32_t act) {
  __shared__ f4 s_part[kWinReduceParts][16];
  const int32_t q = F / 4;
  const int32_t chunks = (q + 15) / 16;
  const int32_t h = (int32_t)(blockIdx.x / chunks);
  const int32_t c4 = (int32_t)(blockIdx.x - (int64_t)h * chunks) * 16 + (threadIdx.x & 15);
  const int part = threadIdx.x >> 4;
  const bool col_ok = c4 < q;
  const int32_t per = (n_grp + kWinReduceParts - 1) / kWinReduceParts;
  const int32_t g0 = min(n_grp, part * per), g1 = min(n_grp, g0 + per);
  f4 sum = f4(0.0f);
  if (col_ok) {
    const f4* src = reinterpret_cast<const f4*>(ws + (int64_t)h * n_grp * F) + c4;
    f4 s0 = f4(0.0f), s1 = f4(0.0f), s2 = f4(0.0f), s3 = f4(0.0f);
    int32_t kg = g0;
    for (; kg + 4 <= g1; kg += 4) {
      s0 += src[(int64_t)kg * q];
      s1 += src[(int64_t)(kg + 1) * q];
      s2 += src[(int64_t)(kg + 2) * q];
      s3 += src[(int64_t)(kg + 3) * q];
    }
    for (; kg < g1; ++kg) s0 += src[(int64_t)kg * q];
    sum = (s0 + s1) + (s2 + s3);
    const int32_t* flags = reinterpret_cast<const int32_t*>(ws + (int64_t)n_hub * n_grp * F) +
                           (int64_t)h * n_grp;
    for (kg = g0; kg < g1; ++kg) {
      if (flags[kg] == 0) continue;
      const int32_t k1 = min(n_win, (kg + 1) * G);
      for (int32_t k = kg * G; k < k1; ++k) {
        const int32_t lo = win_tab[(int64_t)k * n_hub + h];
        const int32_t hi = win_tab[(int64_t)(k + 1) * n_hub + h];
        for (int32_t j = lo; j < hi; ++j) {
          const int32_t c = colidx_s[j];
          if ((uint32_t)(c - k * kWinCols) < (uint32_t)kWinCols) continue;
          const float v = vals_s[j];
          const f4 x = reinterpret_cast<const f4*>(X + (int64_t)c * ldx)[c4];
          sum.x = __builtin_fmaf(v, x.x, sum.x);
          sum.y = __builtin_fmaf(v, x.y, sum.y);
          sum.z = __builtin_fmaf(v, x.z, sum.z);
          sum.w = __builtin_fmaf(v, x.w, sum.w);
        }
      }
    }
  }
  s_part[part][threadIdx.x & 15] = sum;
  __syncthreads();
  if (part != 0 || !col_ok) return;
  f4 total = s_part[0][threadIdx.x];
#pragma unroll
  for (int p = 1; p < kWinReduceParts; ++p) total += s_part[p][threadIdx.x];
  f4* yr = reinterpret_cast<f4*>(Y + (int64_t)perm[hub_first_row + h] * ldy);
  __builtin_nontemporal_store(act_v(total, act), yr + c4);
}

// Small plans (no hub rows, every degree <= min(Z, kSmallMaxDeg), few rows):
// the whole launch is a chain of dependent memory round trips on a mostly idle
// GPU, so this path drops the two that k_spmm adds before its gathers (the
// launch-order / metadata reads and the LDS staging with its barrier). One
// vwarp of L lanes (one float4 or float each, laid across the slice as in
// k_spmm) takes one sorted row, heaviest rows first: it reads the row's
// bounds, loads all of its (column, value) pairs at once, issues every gather
// before the first FMA, and adds in nnz order. With every degree <= Z each
// row is one vwarp of the block-level partition, so Y equals k_spmm's bit for
// bit. The kernel is unrolled for MD pairs, the plan's maximum degree rounded
// up to a multiple of kSmallDegStep: a shorter kernel (fewer registers, less
// code) launches and runs measurably faster (4096-row graph of maximum degree
// 21: 4.8 us for 32-deep loops, 4.3 us for 24-deep ones).
constexpr int kSmallMaxDeg = 32;
constexpr int kSmallDegStep = 8;
constexpr int kSmallThreads = 256;  // measured: 64-thread workgroups (every CU busy) were slower

template <int VW, int LT, int MD>
__global__ __launch_bounds__(kSmallThreads) void k_spmm_rows(
    int32_t n_rows, const int32_t* __restrict__ rowptr_s, const int32_t* __restrict__ colidx_s,
    const float* __restrict__ vals_s, const int32_t* __restrict__ perm, const float* __restrict__ X,
    int64_t ldx, float* __restrict__ Y, int64_t ldy, int32_t col_base, int32_t slice_cols,
    int32_t L_rt, int32_t act) {
  using V = typename VecOf<VW>::T;
  const int L = LT > 0 ? LT : L_rt;
  const int64_t t = (int64_t)blockIdx.x * kSmallThreads + threadIdx.x;
  const int64_t v = t / L;
  const int lane = (int)(t - v * L);
  if (v >= n_rows) return;
  const int32_t r = n_rows - 1 - (int32_t)v;  // heaviest first
  const int32_t a = rowptr_s[r];
  const int32_t d = rowptr_s[r + 1] - a;
  const int32_t col0 = col_base + (int32_t)blockIdx.y * slice_cols;
  const V* __restrict__ Xv = reinterpret_cast<const V*>(X + col0);
  const int64_t ldxv = ldx / VW;
  int32_t c[MD];
  float w[MD];
#pragma unroll
  for (int k = 0; k < MD; ++k) {
    if (k < d) {
      c[k] = colidx_s[a + k];
      w[k] = vals_s[a + k];
    }
  }
  V x[MD];
#pragma unroll
  for (int k = 0; k < MD; ++k)
    if (k < d) x[k] = Xv[(int64_t)c[k] * ldxv + lane];
  V acc = V(0.0f);
#pragma unroll
  for (int k = 0; k < MD; ++k)
    if (k < d) acc = fma_v(w[k], x[k], acc);
  V* yr = reinterpret_cast<V*>(Y + (int64_t)perm[r] * ldy + col0);
  __builtin_nontemporal_store(act_v(acc, act), yr + lane);
}

// --- ablation baselines (the paper's Table II) ------------------------------

// Warp-level partition: workgroup b runs groups [b W, b W + W); vwarp v takes
// group b W + v (one row's slice of <= Z nnz). Consecutive vwarps of the same
// row add their partials in order. A row cut by the workgroup's start or end
// leaves its partial in ws[b][0] (cut at the start) or ws[b][1] (cut only at
// the end); k_wl_fixup finishes those rows in workgroup order.
template <int VW, int LT>
__global__ __launch_bounds__(1024) void k_spmm_wl(
    const int4* __restrict__ meta, int32_t n_groups, int32_t W, int64_t block_base,
    const int32_t* __restrict__ colidx_s, const float* __restrict__ vals_s,
    const float* __restrict__ X, int64_t ldx, float* __restrict__ Y, int64_t ldy,
    float* __restrict__ ws, int32_t F, int32_t col_base, int32_t slice_cols, int32_t L_rt,
    int32_t rounds, int32_t cap_pad, int32_t act) {
  using V = typename VecOf<VW>::T;
  const int L = LT > 0 ? LT : L_rt;
  extern __shared__ float smem[];
  int32_t* s_col = reinterpret_cast<int32_t*>(smem);
  float* s_val = smem + cap_pad;
  V* s_part = reinterpret_cast<V*>(smem + 2 * cap_pad);
  __shared__ int4 s_meta[kMaxBlockWaves];
  __shared__ int32_t s_prev_row, s_next_row;
  const int T = blockDim.x;
  const int64_t blk = block_base + blockIdx.x;
  const int32_t g0 = (int32_t)(blk * W);
  const int32_t nv = min(W, n_groups - g0);
  const int32_t col0 = col_base + (int32_t)blockIdx.y * slice_cols;
  if (threadIdx.x < nv) s_meta[threadIdx.x] = meta[g0 + threadIdx.x];
  if (threadIdx.x == kMaxBlockWaves) s_prev_row = g0 > 0 ? meta[g0 - 1].x : -1;
  if (threadIdx.x == kMaxBlockWaves + 1) s_next_row = g0 + nv < n_groups ? meta[g0 + nv].x : -1;
  __syncthreads();
  const int32_t base = s_meta[0].y;
  const int32_t n_e = s_meta[nv - 1].y + s_meta[nv - 1].z - base;  // groups are contiguous
  for (int i0 = 0; i0 < n_e; i0 += T * kStageUnroll) {
    int32_t c[kStageUnroll];
    float v[kStageUnroll];
#pragma unroll
    for (int u = 0; u < kStageUnroll; ++u) {
      const int i = i0 + u * T + threadIdx.x;
      if (i < n_e) {
        c[u] = colidx_s[base + i];
        v[u] = vals_s[base + i];
      }
    }
#pragma unroll
    for (int u = 0; u < kStageUnroll; ++u) {
      const int i = i0 + u * T + threadIdx.x;
      if (i < n_e) {
        s_col[pad_idx(i)] = c[u];
        s_val[pad_idx(i)] = v[u];
      }
    }
  }
  __syncthreads();
  const V* __restrict__ Xv = reinterpret_cast<const V*>(X + col0);
  const int64_t ldxv = ldx / VW;
  for (int k = 0; k < rounds; ++k) {
    const int vt = threadIdx.x + k * T;
    const int v = vt / L, l = vt - v * L;
    if (v < nv)
      s_part[part_idx<VW>(v * L + l)] =
          gather_row<VW>(s_col, s_val, s_meta[v].y - base, s_meta[v].z, Xv, ldxv, l);
  }
  __syncthreads();
  for (int k = 0; k < rounds; ++k) {
    const int vt = threadIdx.x + k * T;
    const int v = vt / L, l = vt - v * L;
    if (v < nv && (v == 0 || s_meta[v].x != s_meta[v - 1].x)) {
      const int32_t row = s_meta[v].x;
      int e = v;
      V sum = s_part[part_idx<VW>(v * L + l)];
      while (e + 1 < nv && s_meta[e + 1].x == row) {
        ++e;
        sum += s_part[part_idx<VW>(e * L + l)];
      }
      const bool start_cut = v == 0 && s_prev_row == row;
      const bool end_cut = e == nv - 1 && s_next_row == row;
      if (start_cut || end_cut) {
        V* wr = reinterpret_cast<V*>(ws + (blk * 2 + (start_cut ? 0 : 1)) * F + col0);
        wr[l] = sum;
      } else {
        V* yr = reinterpret_cast<V*>(Y + (int64_t)row * ldy + col0);
        __builtin_nontemporal_store(act_v(sum, act), yr + l);
      }
    }
  }
}

// Rows cut by workgroup boundaries: partials ws[b0][1], ws[b0+1][0], ...,
// ws[b1][0] added in order, in runs of 16 (bounded rounding depth).
template <int VW>
__global__ __launch_bounds__(256) void k_wl_fixup(const int32_t* __restrict__ goff, int32_t n_rows,
                                                  int32_t W, const float* __restrict__ ws, int32_t F,
                                                  float* __restrict__ Y, int64_t ldy,
                                                  int32_t col_base, int32_t slice_cols, int32_t L,
                                                  int32_t act) {
  using V = typename VecOf<VW>::T;
  const int32_t col0 = col_base + (int32_t)blockIdx.y * slice_cols;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < (int64_t)n_rows * L;
       t += stride) {
    const int64_t r = t / L;
    const int l = (int)(t - r * L);
    const int32_t b0 = goff[r] / W, b1 = (goff[r + 1] - 1) / W;
    if (b0 == b1) continue;
    auto part = [&](int32_t b) {
      const int slot = b == b0 ? 1 : 0;
      return reinterpret_cast<const V*>(ws + ((int64_t)b * 2 + slot) * F + col0)[l];
    };
    V total = V(0.0f);
    for (int32_t b = b0; b <= b1; b += 16) {
      V run = part(b);
      const int32_t e = b + 16 <= b1 + 1 ? b + 16 : b1 + 1;
      for (int32_t q = b + 1; q < e; ++q) run += part(q);
      total = b == b0 ? run : total + run;
    }
    V* yr = reinterpret_cast<V*>(Y + r * ldy + col0);
    __builtin_nontemporal_store(act_v(total, act), yr + l);
  }
}

// Block-level partition without the combined warp: every vwarp is one
// 64-lane wave, one float per lane, and loops over F in strips of 64 columns.
// Split rows and hub chunks keep one F-wide partial per vwarp in LDS.
__global__ __launch_bounds__(1024) void k_spmm_colloop(
    const int4* __restrict__ meta, const int32_t* __restrict__ order, int32_t entry_base,
    int32_t hub_first_entry, int32_t deg_bound, int32_t W, const int32_t* __restrict__ colidx_s,
    const float* __restrict__ vals_s, const int32_t* __restrict__ perm, const float* __restrict__ X,
    int64_t ldx, float* __restrict__ Y, int64_t ldy, float* __restrict__ ws, int32_t F,
    int32_t rounds, int32_t cap_pad, int32_t act) {
  extern __shared__ float smem[];
  int32_t* s_col = reinterpret_cast<int32_t*>(smem);
  float* s_val = smem + cap_pad;
  float* s_part = smem + 2 * cap_pad;  // [W][F]
  const int T = blockDim.x;
  const int32_t b = order[entry_base + (int32_t)blockIdx.x];
  const int4 m = meta[b];
  const int32_t deg = m.x, loc = m.y, row = m.z, info = m.w;
  const bool hub = deg > deg_bound;
  const int32_t rows = info & 0xFFFF;
  const int32_t n_e = hub ? info : rows * deg;
  for (int i = threadIdx.x; i < n_e; i += T) {
    s_col[pad_idx(i)] = colidx_s[loc + i];
    s_val[pad_idx(i)] = vals_s[loc + i];
  }
  __syncthreads();
  const int32_t wn = (int32_t)((uint32_t)info >> 16);
  const int32_t wpr = hub ? W : (deg > 0 ? (deg + wn - 1) / wn : 1);
  const int32_t nv = hub ? W : rows * wpr;
  const int32_t sl = hub ? (n_e + W - 1) / W : 0;
  for (int k = 0; k < rounds; ++k) {
    const int vt = threadIdx.x + k * T;
    const int v = vt >> 6, lane = vt & 63;
    if (v >= nv) continue;
    int s0, len, rl = 0;
    if (hub) {
      s0 = v * sl;
      const int left = n_e - s0;
      len = left < 0 ? 0 : (left < sl ? left : sl);
    } else {
      rl = v / wpr;
      const int part = v - rl * wpr;
      s0 = rl * deg + part * wn;
      len = deg > 0 ? min(wn, deg - part * wn) : 0;
    }
    for (int c = lane; c < F; c += 64) {  // the single-warp column loop
      const float acc = gather_row<1>(s_col, s_val, s0, len, X, ldx, c);
      if (!hub && wpr == 1)
        __builtin_nontemporal_store(act_v(acc, act), Y + (int64_t)perm[row + rl] * ldy + c);
      else
        s_part[(int64_t)v * F + c] = acc;
    }
  }
  if (hub || wpr > 1) {
    __syncthreads();
    const int n_out = hub ? 1 : rows;
    for (int64_t i = threadIdx.x; i < (int64_t)n_out * F; i += T) {
      const int r = (int)(i / F), c = (int)(i - (int64_t)r * F);
      const int first = hub ? 0 : r * wpr;
      float sum = s_part[(int64_t)first * F + c];
      for (int q = 1; q < wpr; ++q) sum += s_part[(int64_t)(first + q) * F + c];
      if (hub) ws[(int64_t)(b - hub_first_entry) * F + c] = sum;
      else __builtin_nontemporal_store(act_v(sum, act), Y + (int64_t)perm[row + r] * ldy + c);
    }
  }
}

inline int round_up(int a, int b) { return (a + b - 1) / b * b; }

// LDS words for the staged (column, value) pairs of the largest entry.
inline int stage_words(int32_t max_entry_nnz) {
  const int last = max_entry_nnz > 0 ? max_entry_nnz - 1 : 0;
  return round_up(last + (last >> 5) + 1, 4);
}

// Floats of partial-sum storage for W vwarps of L lanes.
inline int part_floats(int VW, int W, int L) {
  const int n = W * L;
  return VW * (VW == 4 ? n + (n >> 3) + 1 : n + (n >> 5) + 1);
}

// Column-slice width: 32 floats (one 128-byte line) by default. The variable
// AGCN_SLICE_COLS (a multiple of 4, 4..256) overrides it for measurements.
int slice_cols_setting() {
  static const int v = [] {
    const char* s = std::getenv("AGCN_SLICE_COLS");
    const int x = s ? std::atoi(s) : kDefaultSliceCols;
    return (x >= 4 && x <= 256 && x % 4 == 0) ? x : kDefaultSliceCols;
  }();
  return v;
}

struct SpmmArgs {
  const agcn_plan* p;
  int32_t F;
  const float* X;
  int64_t ldx;
  float* Y;
  int64_t ldy;
  float* ws;
  hipStream_t st;
  int32_t act;
};

// Timing marks for k_spmm: the first launch records `start` when it begins
// and the last records `stop` when it ends (hipExtLaunchKernel), so no
// separate marker packets sit between the kernels.
struct Marks {
  hipEvent_t start = nullptr;
  hipEvent_t stop = nullptr;
};

// Launch positions [e_begin, e_end) of the plan's launch order, every column
// slice of one width; no entry of the range holds more than max_nnz nonzeros
// (the LDS staged per workgroup is sized for it).
struct EntryRange {
  int32_t begin, end;
  int32_t max_nnz;
};

template <int VW, int LT>
void launch_spmm(const SpmmArgs& a, int L, int n_slices, int col_base, int slice_cols,
                 Marks& mk, bool last_part, EntryRange er) {
  const agcn_plan* p = a.p;
  const int cap_pad = stage_words(er.max_nnz);
  const int want = p->W * L;
  const int T = std::min(1024, round_up(want, 64));
  const int rounds = (want + T - 1) / T;
  const size_t lds = (size_t)2 * cap_pad * 4 + (size_t)part_floats(VW, p->W, L) * 4;
  const int64_t max_grid = (int64_t)(UINT32_MAX / (uint32_t)T);
  for (int64_t e0 = er.begin; e0 < er.end; e0 += max_grid) {
    const int64_t cnt = std::min<int64_t>(max_grid, er.end - e0);
    dim3 grid((unsigned)cnt, (unsigned)n_slices);
    const hipEvent_t stop = (last_part && e0 + cnt >= er.end) ? mk.stop : nullptr;
    if (mk.start || stop) {
      hipExtLaunchKernelGGL(k_spmm<VW, LT>, grid, dim3(T), (uint32_t)lds, a.st, mk.start, stop, 0,
                            p->meta, p->order, (int32_t)e0, p->hub_first_entry, p->deg_bound, p->W,
                            p->colidx_s, p->vals_s, p->perm, a.X, a.ldx, a.Y, a.ldy, a.ws, a.F,
                            col_base, slice_cols, L, rounds, cap_pad, a.act);
      mk.start = nullptr;
    } else {
      k_spmm<VW, LT><<<grid, T, lds, a.st>>>(p->meta, p->order, (int32_t)e0, p->hub_first_entry,
                                             p->deg_bound, p->W, p->colidx_s, p->vals_s, p->perm,
                                             a.X, a.ldx, a.Y, a.ldy, a.ws, a.F, col_base,
                                             slice_cols, L, rounds, cap_pad, a.act);
    }
  }
}

template <int VW>
void dispatch_spmm(const SpmmArgs& a, int L, int n_slices, int col_base, int slice_cols, Marks& mk,
                   bool last_part, EntryRange er) {
  switch (L) {
    case 1: return launch_spmm<VW, 1>(a, L, n_slices, col_base, slice_cols, mk, last_part, er);
    case 2: return launch_spmm<VW, 2>(a, L, n_slices, col_base, slice_cols, mk, last_part, er);
    case 4: return launch_spmm<VW, 4>(a, L, n_slices, col_base, slice_cols, mk, last_part, er);
    case 8: return launch_spmm<VW, 8>(a, L, n_slices, col_base, slice_cols, mk, last_part, er);
    case 16: return launch_spmm<VW, 16>(a, L, n_slices, col_base, slice_cols, mk, last_part, er);
    case 32: return launch_spmm<VW, 32>(a, L, n_slices, col_base, slice_cols, mk, last_part, er);
    case 64: return launch_spmm<VW, 64>(a, L, n_slices, col_base, slice_cols, mk, last_part, er);
    default: return launch_spmm<VW, 0>(a, L, n_slices, col_base, slice_cols, mk, last_part, er);
  }
}

template <int VW, int MC>
void launch_hub_flat(const SpmmArgs& a, int L, int n_slices, int col_base, int slice_cols) {
  const agcn_plan* p = a.p;
  dim3 grid((unsigned)ceil_div64((int64_t)p->n_hub_rows * L, kFlatThreads), (unsigned)n_slices);
  k_hub_reduce_flat<VW, MC><<<grid, kFlatThreads, 0, a.st>>>(
      p->hub_chunk_off, p->hub_first_row, p->perm, a.ws, a.F, a.Y, a.ldy, col_base, slice_cols, L,
      p->n_hub_rows, a.act);
}

template <int VW>
void launch_hub(const SpmmArgs& a, int L, int n_slices, int col_base, int slice_cols) {
  const agcn_plan* p = a.p;
  // The flat kernel when every hub row has few chunks and the launch covers
  // several slices (sweep_powerlaw, 7 chunks at most, per launch: 9.5 against
  // 13.8 us at 8 slices, 6.3 against 7.8 at 4; at 1 and 2 slices the tree's
  // one workgroup per row was faster, 4.6 against 5.1 and 5.2 against 5.4).
  const int64_t max_chunks = ceil_div64(std::max(p->max_deg, 1), p->H);
  if (max_chunks <= kFlatMaxChunks && n_slices > 2) {
    if (max_chunks <= 8) return launch_hub_flat<VW, 8>(a, L, n_slices, col_base, slice_cols);
    if (max_chunks <= 16) return launch_hub_flat<VW, 16>(a, L, n_slices, col_base, slice_cols);
    return launch_hub_flat<VW, 32>(a, L, n_slices, col_base, slice_cols);
  }
  int G = 1;
  while (G < 16 && 2 * G * L <= 1024) G *= 2;
  const int T = round_up(G * L, 64);
  const size_t lds = (size_t)G * L * VW * 4;
  dim3 grid((unsigned)p->n_hub_rows, (unsigned)n_slices);
  k_hub_reduce<VW><<<grid, T, lds, a.st>>>(p->hub_chunk_off, p->hub_first_row, p->perm, a.ws, a.F,
                                           a.Y, a.ldy, col_base, slice_cols, L, G, a.act);
}

// Runs one phase (aggregation or hub reduction) over all column slices of
// width sc_max (at most F): the full slices in one launch, a narrower last
// slice in a second one. The aggregation covers the launch positions `er`.
template <int VW>
int run_phase(const SpmmArgs& a, bool hub_phase, Marks& mk, int sc_max, EntryRange er,
              bool last_range) {
  const int sc = std::min(a.F, sc_max);
  const int n_full = a.F / sc;
  const int tail = a.F - n_full * sc;
  for (int part = 0; part < 2; ++part) {
    const int n_slices = part == 0 ? n_full : (tail > 0 ? 1 : 0);
    if (n_slices == 0) continue;
    const int cols = part == 0 ? sc : tail;
    const int L = cols / VW;
    const int col_base = part == 0 ? 0 : n_full * sc;
    const bool last_part = last_range && (part == 1 || tail == 0);
    if (hub_phase) launch_hub<VW>(a, L, n_slices, col_base, sc);
    else dispatch_spmm<VW>(a, L, n_slices, col_base, sc, mk, last_part, er);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return hip_fail(e, hub_phase ? "k_hub_reduce launch" : "k_spmm launch");
  }
  return AGCN_OK;
}

// Plans small enough that k_spmm_rows runs instead of k_spmm.
constexpr int64_t kSmallMaxNnz = (int64_t)1 << 18;
constexpr int32_t kSmallMaxRows = 1 << 16;

bool small_path(const agcn_plan* p) {
  return p->flags == 0 && p->n_hub_rows == 0 && p->max_deg <= std::min(p->Z, kSmallMaxDeg) &&
         p->nnz <= kSmallMaxNnz && p->n_rows <= kSmallMaxRows;
}

template <int VW, int LT, int MD>
void launch_rows_md(const SpmmArgs& a, int L, int n_slices, int col_base, int slice_cols,
                    Marks& mk, bool last_part) {
  const agcn_plan* p = a.p;
  const int64_t threads = (int64_t)p->n_rows * L;
  dim3 grid((unsigned)ceil_div64(threads, kSmallThreads), (unsigned)n_slices);
  const hipEvent_t stop = last_part ? mk.stop : nullptr;
  hipExtLaunchKernelGGL(k_spmm_rows<VW, LT, MD>, grid, dim3(kSmallThreads), 0, a.st, mk.start,
                        stop, 0, p->n_rows, p->rowptr_s, p->colidx_s, p->vals_s, p->perm, a.X,
                        a.ldx, a.Y, a.ldy, col_base, slice_cols, L, a.act);
  mk.start = nullptr;
}

template <int VW, int LT>
void launch_rows(const SpmmArgs& a, int L, int n_slices, int col_base, int slice_cols, Marks& mk,
                 bool last_part) {
  // The loops' depth: the maximum degree rounded up to a multiple of kSmallDegStep.
  switch ((std::max(a.p->max_deg, 1) + kSmallDegStep - 1) / kSmallDegStep) {
    case 1: launch_rows_md<VW, LT, 8>(a, L, n_slices, col_base, slice_cols, mk, last_part); break;
    case 2: launch_rows_md<VW, LT, 16>(a, L, n_slices, col_base, slice_cols, mk, last_part); break;
    case 3: launch_rows_md<VW, LT, 24>(a, L, n_slices, col_base, slice_cols, mk, last_part); break;
    default: launch_rows_md<VW, LT, 32>(a, L, n_slices, col_base, slice_cols, mk, last_part); break;
  }
}

template <int VW>
int run_small(const SpmmArgs& a, Marks& mk) {
  const int sc = std::min(a.F, VW == 4 ? kDefaultSliceCols : 64);
  const int n_full = a.F / sc;
  const int tail = a.F - n_full * sc;
  for (int part = 0; part < 2; ++part) {
    const int n_slices = part == 0 ? n_full : (tail > 0 ? 1 : 0);
    if (n_slices == 0) continue;
    const int L = (part == 0 ? sc : tail) / VW;
    const int col_base = part == 0 ? 0 : n_full * sc;
    const bool last_part = part == 1 || tail == 0;
    switch (L) {
      case 4: launch_rows<VW, 4>(a, L, n_slices, col_base, sc, mk, last_part); break;
      case 8: launch_rows<VW, 8>(a, L, n_slices, col_base, sc, mk, last_part); break;
      default: launch_rows<VW, 0>(a, L, n_slices, col_base, sc, mk, last_part); break;
    }
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return hip_fail(e, "k_spmm_rows launch");
  }
  return AGCN_OK;
}

template <int VW>
int default_slice_cols() {
  return VW == 4 ? slice_cols_setting() : std::min(64, slice_cols_setting());
}

// The aggregation over every entry. When the hub chunks run in column order
// and hub rows are long (plan flag hub_wide), the chunks in flight gather
// from a narrow column range, so one XCD's L2 holds that range for several
// 128-byte slices at once: the hub chunks then take slices of
// kHubSliceCols columns (staging their CSR pairs once per wide slice instead
// of once per 128-byte slice) and the other entries the default slices.
template <int VW>
int run_aggregation(const SpmmArgs& a, Marks& mk) {
  const agcn_plan* p = a.p;
  const int sc = default_slice_cols<VW>();
  const int32_t n_chunks = p->n_hub_rows > 0 ? p->n_entries - p->hub_first_entry : 0;
  const int wide = VW == 4 ? kHubSliceCols : std::min(64, kHubSliceCols);
  if (p->hub_wide && n_chunks > 0 && std::min(a.F, wide) > std::min(a.F, sc)) {
    // Hub chunks hold at most H nonzeros, the other entries at most W * Z.
    int rc = run_phase<VW>(a, false, mk, wide, EntryRange{0, n_chunks, p->H},
                           n_chunks == p->n_entries);
    if (rc || n_chunks == p->n_entries) return rc;
    return run_phase<VW>(a, false, mk, sc, EntryRange{n_chunks, p->n_entries, p->deg_bound}, true);
  }
  return run_phase<VW>(a, false, mk, sc,
                       EntryRange{0, p->n_entries, std::max(p->deg_bound, p->H)}, true);
}


// The hub-window execute: the aggregation over every entry but the hub
// chunks (first in the launch order), then k_hub_win and k_hub_win_reduce.
int run_windows(const SpmmArgs& a, Marks& mk, hipEvent_t ev_end) {
  const agcn_plan* p = a.p;
  const int32_t n_chunks = p->n_entries - p->hub_first_entry;
  hipError_t e;
  if (n_chunks < p->n_entries) {
    const int rc = run_phase<4>(a, false, mk, default_slice_cols<4>(),
                                EntryRange{n_chunks, p->n_entries, p->deg_bound}, true);
    if (rc) return rc;
  } else {  // hub rows only: the marks frame an empty aggregation
    for (hipEvent_t ev : {mk.start, mk.stop})
      if (ev && (e = hipEventRecord(ev, a.st)) != hipSuccess) return hip_fail(e, "hipEventRecord");
  }
  const WinShape w = win_shape(p, a.F);
  k_hub_win<<<dim3((unsigned)w.n_b, (unsigned)w.n_grp, (unsigned)w.n_slices), 1024, 0, a.st>>>(
      p->win_tab, p->n_hub_rows, p->n_win, w.G, w.n_grp, p->colidx_s, p->vals_s, a.X, a.ldx,
      p->n_cols, a.ws, a.F);
  if ((e = hipGetLastError()) != hipSuccess) return hip_fail(e, "k_hub_win launch");
  const int64_t blocks = (int64_t)p->n_hub_rows * ceil_div64(a.F / 4, 16);
  k_hub_win_reduce<<<(unsigned)blocks, kWinReduceParts * 16, 0, a.st>>>(
      a.ws, p->n_hub_rows, p->n_win, w.G, w.n_grp, a.F, p->win_tab, p->colidx_s, p->vals_s, a.X,
      a.ldx, p->perm, p->hub_first_row, a.Y, a.ldy, a.act);
  if ((e = hipGetLastError()) != hipSuccess) return hip_fail(e, "k_hub_win_reduce launch");
  if (ev_end && (e = hipEventRecord(ev_end, a.st)) != hipSuccess) return hip_fail(e, "hipEventRecord");
  return AGCN_OK;
}

}  // namespace

WinShape win_shape(const agcn_plan* p, int32_t F) {
  WinShape w{};
  w.n_slices = (int32_t)ceil_div64(F, kWinSliceCols);
  w.n_b = (int32_t)ceil_div64(p->n_hub_rows, kWinRows);
  const int64_t per_group = std::max<int64_t>(1, (int64_t)w.n_slices * w.n_b);
  const int64_t want = std::max<int64_t>(1, ceil_div64(kWinTargetGroups, per_group));
  w.G = (int32_t)std::max<int64_t>(1, ceil_div64(p->n_win, want));
  w.n_grp = (int32_t)ceil_div64(p->n_win, w.G);
  return w;
}

size_t win_workspace_bytes(const agcn_plan* p, int32_t F) {
  // (grid limits: slices in grid z, the reduction's (hub row, 64 columns) in grid x)
  if (p->n_win <= 0 || p->n_hub_rows <= 0 || F < kWinMinF || ceil_div64(F, kWinSliceCols) > 65535 ||
      (int64_t)p->n_hub_rows * ceil_div64(F, kWinSliceCols) > INT32_MAX)
    return 0;
  const WinShape w = win_shape(p, F);
  // partial rows, then one stray flag per (hub row, window group)
  return (size_t)p->n_hub_rows * (size_t)w.n_grp * ((size_t)F * sizeof(float) + sizeof(int32_t));
}

size_t chunk_workspace_bytes(const agcn_plan* p, int32_t F) {
  const int64_t chunks =
      p->flags & AGCN_PLAN_WARP_LEVEL
          ? 2 * warp_level_blocks(p)
          : (p->n_hub_rows > 0 ? (int64_t)p->n_entries - p->hub_first_entry : 0);
  return (size_t)chunks * (size_t)F * sizeof(float);
}

size_t spmm_lds_bytes_max(int32_t W, int32_t max_entry_nnz) {
  // Worst case over slice widths: 64 lanes of float4 per vwarp.
  return (size_t)2 * stage_words(max_entry_nnz) * 4 + (size_t)part_floats(4, W, 64) * 4;
}

namespace {

template <int VW, int LT>
void launch_wl(const SpmmArgs& a, int L, int n_slices, int col_base, int slice_cols, Marks& mk,
               bool last_part) {
  const agcn_plan* p = a.p;
  const int cap_pad = stage_words(p->W * p->Z);
  const int want = p->W * L;
  const int T = std::min(1024, std::max(64, round_up(want, 64)));
  const int rounds = (want + T - 1) / T;
  const size_t lds = (size_t)2 * cap_pad * 4 + (size_t)part_floats(VW, p->W, L) * 4;
  const int64_t blocks = warp_level_blocks(p);
  const int64_t max_grid = (int64_t)(UINT32_MAX / (uint32_t)T);
  for (int64_t b0 = 0; b0 < blocks; b0 += max_grid) {
    const int64_t cnt = std::min<int64_t>(max_grid, blocks - b0);
    const hipEvent_t stop = (last_part && b0 + cnt >= blocks) ? mk.stop : nullptr;
    hipExtLaunchKernelGGL(k_spmm_wl<VW, LT>, dim3((unsigned)cnt, (unsigned)n_slices), dim3(T),
                          (uint32_t)lds, a.st, mk.start, stop, 0, p->meta, p->n_entries, p->W, b0,
                          p->colidx_s, p->vals_s, a.X, a.ldx, a.Y, a.ldy, a.ws, a.F, col_base,
                          slice_cols, L, rounds, cap_pad, a.act);
    mk.start = nullptr;
  }
}

template <int VW>
int run_warp_level(const SpmmArgs& a, Marks& mk, hipEvent_t ev_end) {
  const agcn_plan* p = a.p;
  const int sc_max = VW == 4 ? slice_cols_setting() : std::min(64, slice_cols_setting());
  const int sc = std::min(a.F, sc_max);
  const int n_full = a.F / sc;
  const int tail = a.F - n_full * sc;
  for (int part = 0; part < 2; ++part) {
    const int n_slices = part == 0 ? n_full : (tail > 0 ? 1 : 0);
    if (n_slices == 0) continue;
    const int L = (part == 0 ? sc : tail) / VW;
    const int col_base = part == 0 ? 0 : n_full * sc;
    const bool last_part = part == 1 || tail == 0;
    switch (L) {
      case 4: launch_wl<VW, 4>(a, L, n_slices, col_base, sc, mk, last_part); break;
      case 8: launch_wl<VW, 8>(a, L, n_slices, col_base, sc, mk, last_part); break;
      default: launch_wl<VW, 0>(a, L, n_slices, col_base, sc, mk, last_part); break;
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return hip_fail(e, "k_spmm_wl launch");
    const int rows_per_block = std::max(1, 256 / L);
    dim3 fgrid((unsigned)std::min<int64_t>(ceil_div64(p->n_rows, rows_per_block), 1 << 20),
               (unsigned)n_slices);
    k_wl_fixup<VW><<<fgrid, rows_per_block * L, 0, a.st>>>(p->group_off, p->n_rows, p->W, a.ws, a.F,
                                                           a.Y, a.ldy, col_base, sc, L, a.act);
    if ((e = hipGetLastError()) != hipSuccess) return hip_fail(e, "k_wl_fixup launch");
  }
  hipError_t e;
  if (ev_end && (e = hipEventRecord(ev_end, a.st)) != hipSuccess) return hip_fail(e, "hipEventRecord");
  return AGCN_OK;
}

int run_colloop(const SpmmArgs& a, Marks& mk, hipEvent_t ev_end) {
  const agcn_plan* p = a.p;
  const int cap_pad = stage_words(std::max(p->deg_bound, p->H));
  const size_t lds = (size_t)2 * cap_pad * 4 + (size_t)p->W * a.F * 4;
  if (lds > 65536)
    return fail(AGCN_ERR_UNSUPPORTED, "column-loop execution needs W * F * 4 + staging <= 64 KiB of LDS");
  const int want = p->W * 64;
  const int T = std::min(1024, want);
  const int rounds = (want + T - 1) / T;
  hipError_t e;
  const int64_t max_grid = (int64_t)(UINT32_MAX / (uint32_t)T);
  for (int64_t e0 = 0; e0 < p->n_entries; e0 += max_grid) {
    const int64_t cnt = std::min<int64_t>(max_grid, p->n_entries - e0);
    const hipEvent_t stop = e0 + cnt >= p->n_entries ? mk.stop : nullptr;
    hipExtLaunchKernelGGL(k_spmm_colloop, dim3((unsigned)cnt), dim3(T), (uint32_t)lds, a.st,
                          mk.start, stop, 0, p->meta, p->order, (int32_t)e0, p->hub_first_entry,
                          p->deg_bound, p->W, p->colidx_s, p->vals_s, p->perm, a.X, a.ldx, a.Y,
                          a.ldy, a.ws, a.F, rounds, cap_pad, a.act);
    mk.start = nullptr;
  }
  if ((e = hipGetLastError()) != hipSuccess) return hip_fail(e, "k_spmm_colloop launch");
  if (p->n_hub_rows > 0) {
    const int L = std::min(64, a.F);
    int G = 1;
    while (G < 16 && 2 * G * L <= 1024) G *= 2;
    const int n_slices = (int)ceil_div64(a.F, 64);
    // one launch per 64-column strip (the last may be narrower)
    for (int s = 0; s < n_slices; ++s) {
      const int cols = std::min(64, a.F - s * 64);
      k_hub_reduce<1><<<dim3((unsigned)p->n_hub_rows, 1), round_up(G * cols, 64),
                        (size_t)G * cols * 4, a.st>>>(p->hub_chunk_off, p->hub_first_row, p->perm,
                                                      a.ws, a.F, a.Y, a.ldy, s * 64, 64, cols, G,
                                                      a.act);
    }
    if ((e = hipGetLastError()) != hipSuccess) return hip_fail(e, "k_hub_reduce launch");
  }
  if (ev_end && (e = hipEventRecord(ev_end, a.st)) != hipSuccess) return hip_fail(e, "hipEventRecord");
  return AGCN_OK;
}

}  // namespace

// Workspace of agcn_spmm_noalloc: a fixed device array (every GPU the
// library runs on holds its own copy until the process ends). Host code must
// not use the name `scratch` as an address -- in host code it is only a
// stand-in symbol; noalloc_scratch() returns the device's real address, looked
// up once per device. The kernels write every partial they later read within
// one call (hub-chunk partials, rows cut by warp-level workgroups), so the
// array needs no clearing; calls that overlap on one GPU share it and race.
namespace {
__device__ __align__(256) float scratch[kNoallocScratchBytes / sizeof(float)];

std::mutex g_scratch_mu;
float* g_scratch_ptr[kMaxDevices] = {};
}  // namespace

int noalloc_scratch(int device, float** out) {
  if (device < 0 || device >= kMaxDevices)
    return fail(AGCN_ERR_UNSUPPORTED, "device ordinal beyond the library's table");
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (g_scratch_ptr[device] == nullptr) {
    void* ptr = nullptr;
    const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
    if (ptr == nullptr) return fail(AGCN_ERR_HIP, "hipGetSymbolAddress(scratch) returned NULL");
    g_scratch_ptr[device] = static_cast<float*>(ptr);
  }
  *out = g_scratch_ptr[device];
  return AGCN_OK;
}

int run_spmm(const agcn_plan* p, int32_t F, const float* X, int64_t ldx, float* Y, int64_t ldy,
             float* ws, size_t ws_bytes, hipStream_t st, hipEvent_t ev_begin, hipEvent_t ev_mid,
             hipEvent_t ev_end, int32_t act) {
  const bool vec = (F % 4 == 0) && (ldx % 4 == 0) && (ldy % 4 == 0) && aligned16(X) &&
                   aligned16(Y) && (ws == nullptr || aligned16(ws));
  const SpmmArgs a{p, F, X, ldx, Y, ldy, ws, st, act};
  hipError_t e;
  if (p->n_entries == 0) {  // no rows (hub rows need entries): keep the marks meaningful
    for (hipEvent_t ev : {ev_begin, ev_mid, ev_end})
      if (ev && (e = hipEventRecord(ev, st)) != hipSuccess) return hip_fail(e, "hipEventRecord");
    return AGCN_OK;
  }
  Marks mk{ev_begin, ev_mid};
  if (p->flags & AGCN_PLAN_WARP_LEVEL)
    return vec ? run_warp_level<4>(a, mk, ev_end) : run_warp_level<1>(a, mk, ev_end);
  if (p->flags & AGCN_PLAN_COLUMN_LOOP) return run_colloop(a, mk, ev_end);
  if (small_path(p)) {
    const int rc = vec ? run_small<4>(a, mk) : run_small<1>(a, mk);
    if (rc) return rc;
    if (ev_end && (e = hipEventRecord(ev_end, st)) != hipSuccess) return hip_fail(e, "hipEventRecord");
    return AGCN_OK;
  }
  const size_t win_ws = vec ? win_workspace_bytes(p, F) : 0;
  if (win_ws > 0 && ws_bytes >= win_ws) return run_windows(a, mk, ev_end);
  int rc = vec ? run_aggregation<4>(a, mk) : run_aggregation<1>(a, mk);
  if (rc) return rc;
  Marks none{};
  const EntryRange all{0, p->n_entries, std::max(p->deg_bound, p->H)};
  if (p->n_hub_rows > 0)
    rc = vec ? run_phase<4>(a, true, none, default_slice_cols<4>(), all, true)
             : run_phase<1>(a, true, none, default_slice_cols<1>(), all, true);
  if (rc) return rc;
  if (ev_end && (e = hipEventRecord(ev_end, st)) != hipSuccess) return hip_fail(e, "hipEventRecord");
  return AGCN_OK;
}

}  // namespace agcn
