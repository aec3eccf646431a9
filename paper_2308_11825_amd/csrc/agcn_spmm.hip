// Execute: Y = A X over the block-level partition (Sec. III-C, III-D).
//
// k_spmm: one workgroup per metadata entry and per slice of <= 64 lanes of
// the feature dimension (256 columns on the 128-bit path, 64 on the 32-bit
// path; a slice exists only when F exceeds that width).
//   1. The entry {deg, loc, row, info} is read once (uniform, scalar load).
//   2. The entry's column indices and values -- contiguous in the sorted
//      CSR -- are staged into LDS with coalesced non-temporal loads. The LDS
//      index is padded by one word per 32 so the vwarps of a wave, which read
//      slices a fixed stride apart, hit different banks.
//   3. Virtual warps (the paper's warps): a row of degree d is covered by
//      ceil(d / warp_nzs) consecutive vwarps of warp_nzs nnz; each vwarp owns
//      L lanes laid across the columns, one float4 per lane (the combined
//      warp of Sec. III-D, built from 64-lane waves: several vwarps share a
//      wave when F < 256). Workgroup lanes are mapped to (vwarp, lane) in
//      `rounds` passes when W * L exceeds the workgroup size.
//   4. Each lane gathers X rows (16-byte loads, 4 independent loads in
//      flight per lane) and accumulates with fp32 FMA in nnz order.
//   5. Rows held by a single vwarp store straight to Y (non-temporal). Rows
//      split over several vwarps sum their partials from LDS in vwarp order;
//      hub chunks (deg > deg_bound) sum all W slices in order and write one
//      partial row to the workspace. No atomics: the result is bitwise
//      reproducible and does not depend on the row's position in the order.
// k_hub_reduce: one workgroup per hub row; G groups of lanes each add a
//   contiguous run of the row's chunk partials, then a fixed pairwise tree
//   combines the G group sums and the row is written once.
//
// Entries are launched heaviest first (metadata is in ascending degree order).
#include <algorithm>
#include <climits>

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

__device__ inline int pad_idx(int i) { return i + (i >> 5); }

__device__ inline f4 fma_v(float a, f4 x, f4 acc) {
  f4 r;
  r.x = __builtin_fmaf(a, x.x, acc.x);
  r.y = __builtin_fmaf(a, x.y, acc.y);
  r.z = __builtin_fmaf(a, x.z, acc.z);
  r.w = __builtin_fmaf(a, x.w, acc.w);
  return r;
}
__device__ inline float fma_v(float a, float x, float acc) { return __builtin_fmaf(a, x, acc); }

template <typename V>
__device__ inline V zero_v() {
  return V(0.0f);
}

// acc = sum over j in [s0, s0 + len) of val[j] * X[col[j], lane], in order.
template <int VW>
__device__ inline typename VecOf<VW>::T gather_row(const int32_t* s_col, const float* s_val,
                                                   int s0, int len,
                                                   const typename VecOf<VW>::T* __restrict__ Xv,
                                                   int64_t ldv, int32_t lane_col) {
  using V = typename VecOf<VW>::T;
  V acc = zero_v<V>();
  int j = 0;
  for (; j + 4 <= len; j += 4) {
    const int p0 = pad_idx(s0 + j), p1 = pad_idx(s0 + j + 1);
    const int p2 = pad_idx(s0 + j + 2), p3 = pad_idx(s0 + j + 3);
    const int32_t c0 = s_col[p0], c1 = s_col[p1], c2 = s_col[p2], c3 = s_col[p3];
    const float a0 = s_val[p0], a1 = s_val[p1], a2 = s_val[p2], a3 = s_val[p3];
    const V x0 = Xv[(int64_t)c0 * ldv + lane_col];
    const V x1 = Xv[(int64_t)c1 * ldv + lane_col];
    const V x2 = Xv[(int64_t)c2 * ldv + lane_col];
    const V x3 = Xv[(int64_t)c3 * ldv + lane_col];
    acc = fma_v(a0, x0, acc);
    acc = fma_v(a1, x1, acc);
    acc = fma_v(a2, x2, acc);
    acc = fma_v(a3, x3, acc);
  }
  for (; j < len; ++j) {
    const int pj = pad_idx(s0 + j);
    acc = fma_v(s_val[pj], Xv[(int64_t)s_col[pj] * ldv + lane_col], acc);
  }
  return acc;
}

template <int VW>
__global__ __launch_bounds__(1024) void k_spmm(
    const int4* __restrict__ meta, int32_t n_entries, int32_t entry_base, int32_t hub_first_entry,
    int32_t deg_bound, int32_t W, const int32_t* __restrict__ colidx_s,
    const float* __restrict__ vals_s, const int32_t* __restrict__ perm, const float* __restrict__ X,
    int64_t ldx, float* __restrict__ Y, int64_t ldy, float* __restrict__ ws, int32_t F,
    int32_t col_base, int32_t L, int32_t rounds, int32_t cap_pad) {
  using V = typename VecOf<VW>::T;
  extern __shared__ float smem[];
  int32_t* s_col = reinterpret_cast<int32_t*>(smem);
  float* s_val = smem + cap_pad;
  V* s_part = reinterpret_cast<V*>(smem + 2 * cap_pad);

  const int T = blockDim.x;
  const int32_t b = n_entries - 1 - (entry_base + (int32_t)blockIdx.x);
  const int32_t col0 = col_base + (int32_t)blockIdx.y * kSliceLanes * VW;
  const int4 m = meta[b];
  const int32_t deg = m.x, loc = m.y, row = m.z, info = m.w;
  const bool hub = deg > deg_bound;
  const int32_t rows = info & 0xFFFF;
  const int32_t n_e = hub ? info : rows * deg;

  for (int i = threadIdx.x; i < n_e; i += T) {
    s_col[pad_idx(i)] = __builtin_nontemporal_load(colidx_s + loc + i);
    s_val[pad_idx(i)] = __builtin_nontemporal_load(vals_s + loc + i);
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
          __builtin_nontemporal_store(acc, yr + l);
        } else {
          s_part[v * L + l] = acc;
        }
      }
    }
    if (wpr > 1) {  // uniform over the workgroup
      __syncthreads();
      for (int k = 0; k < rounds; ++k) {
        const int vt = threadIdx.x + k * T;
        const int r = vt / L, l = vt - r * L;
        if (r < rows) {
          V sum = s_part[(r * wpr) * L + l];
          for (int q = 1; q < wpr; ++q) sum += s_part[(r * wpr + q) * L + l];
          V* yr = reinterpret_cast<V*>(Y + (int64_t)perm[row + r] * ldy + col0);
          __builtin_nontemporal_store(sum, yr + l);
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
        s_part[v * L + l] = gather_row<VW>(s_col, s_val, s0, len, Xv, ldxv, l);
      }
    }
    __syncthreads();
    for (int k = 0; k < rounds; ++k) {
      const int l = threadIdx.x + k * T;
      if (l < L) {
        V sum = s_part[l];
        for (int v = 1; v < W; ++v) sum += s_part[v * L + l];
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
                                                     int32_t col_base, int32_t L, int32_t G) {
  using V = typename VecOf<VW>::T;
  extern __shared__ float smem[];
  V* s_acc = reinterpret_cast<V*>(smem);  // [G][L]
  const int32_t h = blockIdx.x;
  const int32_t col0 = col_base + (int32_t)blockIdx.y * kSliceLanes * VW;
  const int32_t c0 = hub_chunk_off[h], c1 = hub_chunk_off[h + 1];
  const int32_t nc = c1 - c0;
  const int g = threadIdx.x / L, l = threadIdx.x - g * L;
  const int32_t q = (nc + G - 1) / G;
  if (g < G) {
    V acc = zero_v<V>();
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
    __builtin_nontemporal_store(s_acc[l], yr + l);
  }
}

inline int round_up(int a, int b) { return (a + b - 1) / b * b; }

// LDS words for the staged (column, value) pairs of the largest entry.
inline int stage_words(int32_t max_entry_nnz) {
  const int last = max_entry_nnz > 0 ? max_entry_nnz - 1 : 0;
  return round_up(last + (last >> 5) + 1, 4);
}

template <int VW>
int launch_slices(const agcn_plan* p, int32_t F, const float* X, int64_t ldx, float* Y,
                  int64_t ldy, float* ws, hipStream_t st, bool hub_phase) {
  const int slice_cols = kSliceLanes * VW;
  const int n_full = F / slice_cols;
  const int tail_cols = F - n_full * slice_cols;
  const int cap = std::max(p->deg_bound, p->H);
  const int cap_pad = stage_words(cap);
  for (int part = 0; part < 2; ++part) {
    const int n_slices = part == 0 ? n_full : (tail_cols > 0 ? 1 : 0);
    if (n_slices == 0) continue;
    const int cols = part == 0 ? slice_cols : tail_cols;
    const int L = cols / VW;
    const int col_base = part == 0 ? 0 : n_full * slice_cols;
    if (!hub_phase) {
      const int want = p->W * L;
      const int T = std::min(1024, round_up(want, 64));
      const int rounds = (want + T - 1) / T;
      const size_t lds = (size_t)2 * cap_pad * 4 + (size_t)p->W * L * VW * 4;
      const int64_t max_grid = (int64_t)(UINT32_MAX / (uint32_t)T);
      for (int64_t e0 = 0; e0 < p->n_entries; e0 += max_grid) {
        const int64_t cnt = std::min<int64_t>(max_grid, p->n_entries - e0);
        dim3 grid((unsigned)cnt, (unsigned)n_slices);
        k_spmm<VW><<<grid, T, lds, st>>>(p->meta, p->n_entries, (int32_t)e0, p->hub_first_entry,
                                         p->deg_bound, p->W, p->colidx_s, p->vals_s, p->perm, X,
                                         ldx, Y, ldy, ws, F, col_base, L, rounds, cap_pad);
      }
    } else {
      int G = 1;
      while (G < 16 && 2 * G * L <= 1024) G *= 2;
      const int T = round_up(G * L, 64);
      const size_t lds = (size_t)G * L * VW * 4;
      dim3 grid((unsigned)p->n_hub_rows, (unsigned)n_slices);
      k_hub_reduce<VW><<<grid, T, lds, st>>>(p->hub_chunk_off, p->hub_first_row, p->perm, ws, F,
                                             Y, ldy, col_base, L, G);
    }
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return hip_fail(e, hub_phase ? "k_hub_reduce launch" : "k_spmm launch");
  }
  return AGCN_OK;
}

inline bool aligned16(const void* q) { return (reinterpret_cast<uintptr_t>(q) & 15u) == 0; }

}  // namespace

size_t spmm_lds_bytes_max(int32_t W, int32_t max_entry_nnz) {
  return (size_t)2 * stage_words(max_entry_nnz) * 4 + (size_t)W * kSliceLanes * 4 * 4;
}

int run_spmm(const agcn_plan* p, int32_t F, const float* X, int64_t ldx, float* Y, int64_t ldy,
             float* ws, hipStream_t st, hipEvent_t ev_begin, hipEvent_t ev_mid,
             hipEvent_t ev_end) {
  const bool vec = (F % 4 == 0) && (ldx % 4 == 0) && (ldy % 4 == 0) && aligned16(X) &&
                   aligned16(Y) && (ws == nullptr || aligned16(ws));
  hipError_t e;
  if (ev_begin && (e = hipEventRecord(ev_begin, st)) != hipSuccess)
    return hip_fail(e, "hipEventRecord");
  int rc = AGCN_OK;
  if (p->n_entries > 0)
    rc = vec ? launch_slices<4>(p, F, X, ldx, Y, ldy, ws, st, false)
             : launch_slices<1>(p, F, X, ldx, Y, ldy, ws, st, false);
  if (rc) return rc;
  if (ev_mid && (e = hipEventRecord(ev_mid, st)) != hipSuccess) return hip_fail(e, "hipEventRecord");
  if (p->n_hub_rows > 0)
    rc = vec ? launch_slices<4>(p, F, X, ldx, Y, ldy, ws, st, true)
             : launch_slices<1>(p, F, X, ldx, Y, ldy, ws, st, true);
  if (rc) return rc;
  if (ev_end && (e = hipEventRecord(ev_end, st)) != hipSuccess) return hip_fail(e, "hipEventRecord");
  return AGCN_OK;
}

}  // namespace agcn
