// Linear transformation of a GCNConv layer, H = X W (Sec. II-A), on the
// fp32 matrix cores of gfx950.
//
// k_linear: one workgroup of 4 waves per (128-row tile of X, BN-column tile of
// W). The K dimension (fin) is walked in steps of 32:
//   1. the next X tile (128 x 32) and W tile (32 x BN) are loaded into
//      registers while the current ones are multiplied from LDS;
//   2. wave w owns rows [32 w, 32 w + 32) of the tile and BN / 32 accumulator
//      blocks of 32 x 32 (v_mfma_f32_32x32x2f32: lane l supplies A[l % 32][l / 32]
//      and B[l / 32][l % 32]; accumulator register r of lane l holds
//      C[8 (r / 4) + 4 (l / 32) + r % 4][l % 32]);
//   3. the X tile sits in LDS with a row pitch of 33 floats, so the 32 rows a
//      wave reads for one k fall in 32 different banks; W rows are read
//      contiguously.
// Rows, columns and k beyond the matrices are zero-filled on load and masked
// on store, so any n, fin, fout and leading dimension works; the 128-bit load
// path needs fin, fout, ldx, ldw multiples of 4 and 16-byte aligned X and W.
// Tall-skinny GEMM (n up to millions, fin and fout in the tens to hundreds):
// X is read once per column tile, and the column tiles of one row tile are
// consecutive workgroups, so the second read of X hits L2.
#include <algorithm>
#include <cstdlib>

#include "agcn_internal.hpp"

namespace agcn {
namespace {

typedef float f16v __attribute__((ext_vector_type(16)));
typedef float f4 __attribute__((ext_vector_type(4)));
typedef unsigned v4u __attribute__((ext_vector_type(4)));

constexpr int kBM = 128;
constexpr int kBK = 32;
constexpr int kXP = kBK + 1;
constexpr int kThreads = 256;

template <int BN, bool VEC>
struct Tiles {
  static constexpr int XN = VEC ? 4 : 16;          // X elements (f4 or float) per thread
  static constexpr int WN = VEC ? BN / 32 : BN / 8;  // W elements per thread
  using T = typename std::conditional<VEC, f4, float>::type;
  T x[XN];
  T w[WN];
};

template <int BN, bool VEC>
__device__ inline void load_tiles(Tiles<BN, VEC>& tl, int t, int64_t row0, int col0, int k0,
                                  int64_t n, int32_t fin, int32_t fout,
                                  const float* __restrict__ X, int64_t ldx,
                                  const float* __restrict__ W, int64_t ldw) {
  if constexpr (VEC) {
#pragma unroll
    for (int u = 0; u < Tiles<BN, VEC>::XN; ++u) {
      const int idx = t + u * kThreads;
      const int r = idx >> 3, c = (idx & 7) * 4;
      const int64_t gr = row0 + r;
      f4 v = {0.0f, 0.0f, 0.0f, 0.0f};
      if (gr < n && k0 + c < fin) v = *reinterpret_cast<const f4*>(X + gr * ldx + k0 + c);
      tl.x[u] = v;
    }
    constexpr int per_row = BN / 4;
#pragma unroll
    for (int u = 0; u < Tiles<BN, VEC>::WN; ++u) {
      const int idx = t + u * kThreads;
      const int r = idx / per_row, c = (idx - r * per_row) * 4;
      f4 v = {0.0f, 0.0f, 0.0f, 0.0f};
      if (k0 + r < fin && col0 + c < fout)
        v = *reinterpret_cast<const f4*>(W + (int64_t)(k0 + r) * ldw + col0 + c);
      tl.w[u] = v;
    }
  } else {
#pragma unroll
    for (int u = 0; u < Tiles<BN, VEC>::XN; ++u) {
      const int idx = t + u * kThreads;
      const int r = idx >> 5, c = idx & 31;
      const int64_t gr = row0 + r;
      tl.x[u] = (gr < n && k0 + c < fin) ? X[gr * ldx + k0 + c] : 0.0f;
    }
#pragma unroll
    for (int u = 0; u < Tiles<BN, VEC>::WN; ++u) {
      const int idx = t + u * kThreads;
      const int r = idx / BN, c = idx - r * BN;
      tl.w[u] = (k0 + r < fin && col0 + c < fout) ? W[(int64_t)(k0 + r) * ldw + col0 + c] : 0.0f;
    }
  }
}

template <int BN, bool VEC>
__device__ inline void store_tiles(const Tiles<BN, VEC>& tl, int t, float* sx, float* sw) {
  if constexpr (VEC) {
#pragma unroll
    for (int u = 0; u < Tiles<BN, VEC>::XN; ++u) {
      const int idx = t + u * kThreads;
      const int r = idx >> 3, c = (idx & 7) * 4;
      float* d = sx + r * kXP + c;
      d[0] = tl.x[u].x;
      d[1] = tl.x[u].y;
      d[2] = tl.x[u].z;
      d[3] = tl.x[u].w;
    }
    constexpr int per_row = BN / 4;
#pragma unroll
    for (int u = 0; u < Tiles<BN, VEC>::WN; ++u) {
      const int idx = t + u * kThreads;
      const int r = idx / per_row, c = (idx - r * per_row) * 4;
      *reinterpret_cast<f4*>(sw + r * BN + c) = tl.w[u];
    }
  } else {
#pragma unroll
    for (int u = 0; u < Tiles<BN, VEC>::XN; ++u) {
      const int idx = t + u * kThreads;
      sx[(idx >> 5) * kXP + (idx & 31)] = tl.x[u];
    }
#pragma unroll
    for (int u = 0; u < Tiles<BN, VEC>::WN; ++u) sw[t + u * kThreads] = tl.w[u];
  }
}

template <int BN, bool VEC>
__global__ __launch_bounds__(kThreads) void k_linear(int64_t n, int32_t fin, int32_t fout,
                                                     int32_t n_ct, const float* __restrict__ X,
                                                     int64_t ldx, const float* __restrict__ W,
                                                     int64_t ldw, float* __restrict__ H,
                                                     int64_t ldh) {
  __shared__ float sx[kBM * kXP];
  __shared__ __attribute__((aligned(16))) float sw[kBK * BN];
  const int t = threadIdx.x, wave = t >> 6, lane = t & 63;
  const int64_t rt = (int64_t)blockIdx.x / n_ct;
  const int ct = (int)((int64_t)blockIdx.x - rt * n_ct);
  const int64_t row0 = rt * kBM;
  const int col0 = ct * BN;
  f16v acc[BN / 32];
#pragma unroll
  for (int j = 0; j < BN / 32; ++j)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[j][r] = 0.0f;

  Tiles<BN, VEC> tl;
  load_tiles<BN, VEC>(tl, t, row0, col0, 0, n, fin, fout, X, ldx, W, ldw);
  for (int k0 = 0; k0 < fin; k0 += kBK) {
    store_tiles<BN, VEC>(tl, t, sx, sw);
    __syncthreads();
    if (k0 + kBK < fin)  // uniform
      load_tiles<BN, VEC>(tl, t, row0, col0, k0 + kBK, n, fin, fout, X, ldx, W, ldw);
    const float* xa = sx + (wave * 32 + (lane & 31)) * kXP + (lane >> 5);
    const float* wb = sw + (lane >> 5) * BN + (lane & 31);
#pragma unroll
    for (int kk = 0; kk < kBK; kk += 2) {
      const float a = xa[kk];
#pragma unroll
      for (int j = 0; j < BN / 32; ++j)
        acc[j] = __builtin_amdgcn_mfma_f32_32x32x2f32(a, wb[kk * BN + j * 32], acc[j], 0, 0, 0);
    }
    __syncthreads();
  }
  const int64_t rbase = row0 + wave * 32 + (lane >> 5) * 4;
#pragma unroll
  for (int j = 0; j < BN / 32; ++j) {
    const int col = col0 + j * 32 + (lane & 31);
    if (col >= fout) continue;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int64_t row = rbase + (r >> 2) * 8 + (r & 3);
      if (row < n) H[row * ldh + col] = acc[j][r];
    }
  }
}

// --- W resident in LDS --------------------------------------------------------
//
// k_linear_rw: for fin <= 128 and fout <= 128 (wider outputs: one launch per
// 128 columns; 128-bit path, X and H each under 4 GiB), W^T stays in
// LDS for the whole kernel and every wave works alone on 16-row tiles of X, so
// the main loop has no workgroup barrier:
//   1. each workgroup (4 waves) writes W^T into LDS once: NB * 16 rows (output
//      columns) of KP floats (fin rounded up to KS * 16), zero outside W; the
//      16-byte chunk c of row j sits at chunk c ^ (j & 7), so the 8 rows a
//      group of lanes reads for one chunk fall in 8 different bank groups;
//   2. wave v takes tiles v, v + waves, ... of 16 rows while every wave has a
//      whole round left; the next tile's X is loaded into registers while the
//      current one is multiplied. The tiles of the last, partial round are
//      cut by output columns into as many ranges (1, 2, 4 or 8) as still give
//      each range a wave of its own, so that round takes a fraction of a
//      tile's time instead of a whole one;
//   3. v_mfma_f32_16x16x4f32 with W^T as the left operand, so one instruction
//      computes (X W)^T for 16 rows and 16 output columns (lane l supplies
//      A[l % 16][l / 16] = W^T[col][k] and B[l / 16][l % 16] = X[row][k];
//      accumulator register r of lane l holds C[4 (l / 16) + r][l % 16], that
//      is H[row l % 16][4 (l / 16) + r]: four consecutive columns of one row,
//      written with one 16-byte store). The contraction order is permuted so
//      that one 16-byte load per lane feeds four instructions: in k-step s,
//      lane l loads X[row][16 s + 4 g .. + 3] (g = l / 16) and instruction t
//      takes element t, paired with W^T[col][16 s + 4 g + t] from one 16-byte
//      LDS read; the four instructions together cover k = 16 s .. 16 s + 15.
//      The compiler keeps all of W^T in registers across the tile loop (one
//      wave per SIMD); re-reading it from LDS at two waves per SIMD measured
//      no faster.
constexpr int kRwThreads = 256;
constexpr int kRwWaves = kRwThreads / 64;
constexpr int kRwRows = 16;

// Offset of a masked element. A raw buffer access is out of range when its
// offset is >= the resource's byte count; every resource here covers at most
// kRwOutOfRange - 16 bytes (checked by the host), so this offset is always
// out of range: the load returns 0 and the store is dropped.
constexpr uint32_t kRwOutOfRange = 0xFFFFFFF0u;

__device__ inline __amdgpu_buffer_rsrc_t rw_resource(const void* base, uint32_t bytes) {
  // Raw buffer (stride 0) of `bytes` bytes; dword3 = 32-bit data format (gfx9 family).
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes,
                                           0x00020000);
}

__device__ inline int wt_index(int j, int k, int kc) {  // float index of W^T[j][k]
  return (j * kc + ((k >> 2) ^ (j & 7))) * 4 + (k & 3);
}

template <int NB, int KS>
__global__ __launch_bounds__(kRwThreads) void k_linear_rw(int64_t n, int32_t fin, int32_t fout,
                                                          const float* __restrict__ X, int64_t ldx,
                                                          const float* __restrict__ W, int64_t ldw,
                                                          float* __restrict__ H, int64_t ldh) {
  constexpr int KP = KS * 16, KC = KP / 4, NJ = NB * 16;
  __shared__ __attribute__((aligned(16))) float swt[NJ * KP];
  // 1. W^T into LDS: W row k is read as float4 (4 output columns) and
  //    scattered into 4 rows of W^T. Consecutive lanes take consecutive k, so
  //    their LDS writes land in consecutive words of one W^T row.
  for (int idx = threadIdx.x; idx < KP * (NJ / 4); idx += kRwThreads) {
    const int j0 = (idx / KP) * 4, k = idx - (idx / KP) * KP;
    f4 w = {0.0f, 0.0f, 0.0f, 0.0f};
    if (k < fin && j0 < fout) w = *reinterpret_cast<const f4*>(W + (int64_t)k * ldw + j0);
    swt[wt_index(j0 + 0, k, KC)] = w.x;
    swt[wt_index(j0 + 1, k, KC)] = w.y;
    swt[wt_index(j0 + 2, k, KC)] = w.z;
    swt[wt_index(j0 + 3, k, KC)] = w.w;
  }
  __syncthreads();

  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int i = lane & 15, g = lane >> 4;
  const int64_t n_tiles = (n + kRwRows - 1) / kRwRows;
  const int64_t n_waves = (int64_t)gridDim.x * kRwWaves;
  // X and H through buffer resources: a masked element gets an offset past
  // the 4 GiB range, so its load returns 0 and its store is dropped, with no
  // branch; the compiler then counts the memory operations in flight exactly
  // and waits only for the loads it needs.
  const __amdgpu_buffer_rsrc_t xr = rw_resource(X, (uint32_t)(n * ldx * 4));
  const __amdgpu_buffer_rsrc_t hr = rw_resource(H, (uint32_t)(n * ldh * 4));
  auto load_x = [&](int64_t tile, f4* xv) {
    const int64_t row = tile * kRwRows + i;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const int k = 16 * s + 4 * g;
      const uint32_t off = (row < n && k < fin) ? (uint32_t)((row * ldx + k) * 4) : kRwOutOfRange;
      xv[s] = __builtin_bit_cast(f4, __builtin_amdgcn_raw_buffer_load_b128(xr, (int)off, 0, 0));
    }
  };
  // H stores of one tile: lane (i, g) holds H[row i][16 b + 4 g .. + 3] of
  // every column block b, one 16-byte store each.
  const uint32_t ldh4 = (uint32_t)(ldh * 4);
  auto store_h = [&](int64_t tile, const f4* acc) {
    const int64_t row = tile * kRwRows + i;
    const uint32_t base = (uint32_t)(row * ldh4) + (uint32_t)(16 * g);
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      const bool ok = row < n && 16 * b + 4 * g < fout;
      const uint32_t off = ok ? base + (uint32_t)(64 * b) : kRwOutOfRange;
      __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(v4u, acc[b]), hr, (int)off, 0, 0);
    }
  };
  // Full rounds: every wave takes n_tiles / n_waves tiles.
  const int64_t wid = (int64_t)blockIdx.x * kRwWaves + wave;
  const int64_t n_full = (n_tiles / n_waves) * n_waves;
  f4 xa[KS], xb[KS];
  int64_t tile = wid;
  if (tile < n_full) load_x(tile, xa);
  for (; tile < n_full; tile += n_waves) {
    if (tile + n_waves < n_full) load_x(tile + n_waves, xb);  // uniform
    f4 acc[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b) acc[b] = f4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      f4 wv[NB];
#pragma unroll
      for (int b = 0; b < NB; ++b)
        wv[b] = *reinterpret_cast<const f4*>(swt + wt_index(16 * b + i, 16 * s + 4 * g, KC));
#pragma unroll
      for (int t = 0; t < 4; ++t)
#pragma unroll
        for (int b = 0; b < NB; ++b)
          acc[b] = __builtin_amdgcn_mfma_f32_16x16x4f32(wv[b][t], xa[s][t], acc[b], 0, 0, 0);
    }
    store_h(tile, acc);
#pragma unroll
    for (int s = 0; s < KS; ++s) xa[s] = xb[s];
  }
  // The last, partial round: its tiles are cut into `split` column ranges of
  // NB / split blocks each, as many as keep every unit on its own wave.
  const int64_t rem = n_tiles - n_full;
  if (rem == 0) return;
  int split = 1;
  while (split < NB && rem * split * 2 <= n_waves) split *= 2;
  const int per = NB / split;
  for (int64_t u = wid; u < rem * split; u += n_waves) {
    const int64_t t2 = n_full + u / split;
    const int b0 = (int)(u % split) * per;
    load_x(t2, xa);
    const int64_t row = t2 * kRwRows + i;
    for (int bb = 0; bb < per; ++bb) {
      const int b = b0 + bb;
      f4 acc = f4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        const f4 wv = *reinterpret_cast<const f4*>(swt + wt_index(16 * b + i, 16 * s + 4 * g, KC));
#pragma unroll
        for (int t = 0; t < 4; ++t)
          acc = __builtin_amdgcn_mfma_f32_16x16x4f32(wv[t], xa[s][t], acc, 0, 0, 0);
      }
      const bool ok = row < n && 16 * b + 4 * g < fout;
      const uint32_t off = ok ? (uint32_t)(row * ldh4) + (uint32_t)(16 * g) + (uint32_t)(64 * b)
                              : kRwOutOfRange;
      __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(v4u, acc), hr, (int)off, 0, 0);
    }
  }
}

// AGCN_LINEAR_RW=0 selects the tiled kernel for every shape (for measurements).
bool rw_disabled() {
  static const bool v = [] {
    const char* e = std::getenv("AGCN_LINEAR_RW");
    return e != nullptr && std::atoi(e) == 0;
  }();
  return v;
}

// Workgroups for k_linear_rw: as many as are resident at once on the device
// (each loads W^T once and then loops over tiles), fewer when there are fewer
// tiles.
template <int NB, int KS>
int rw_grid(int64_t n) {
  static const int resident = [] {
    int dev = 0, cus = 0, per_cu = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k_linear_rw<NB, KS>, kRwThreads, 0) !=
            hipSuccess) {
      (void)hipGetLastError();
      cus = 256;
      per_cu = 1;
    }
    return std::max(1, cus) * std::max(1, per_cu);
  }();
  const int64_t tiles = (n + kRwRows - 1) / kRwRows;
  return (int)std::max<int64_t>(1, std::min<int64_t>(resident, (tiles + kRwWaves - 1) / kRwWaves));
}

template <int NB, int KS>
int launch_rw(int64_t n, int32_t fin, int32_t fout, const float* X, int64_t ldx, const float* W,
              int64_t ldw, float* H, int64_t ldh, hipStream_t st) {
  k_linear_rw<NB, KS><<<rw_grid<NB, KS>(n), kRwThreads, 0, st>>>(n, fin, fout, X, ldx, W, ldw, H,
                                                                 ldh);
  const hipError_t e = hipGetLastError();
  return e == hipSuccess ? AGCN_OK : hip_fail(e, "k_linear_rw launch");
}

template <int NB>
int dispatch_rw(int64_t n, int32_t fin, int32_t fout, const float* X, int64_t ldx, const float* W,
                int64_t ldw, float* H, int64_t ldh, hipStream_t st) {
  if (fin <= 32) return launch_rw<NB, 2>(n, fin, fout, X, ldx, W, ldw, H, ldh, st);
  if (fin <= 64) return launch_rw<NB, 4>(n, fin, fout, X, ldx, W, ldw, H, ldh, st);
  return launch_rw<NB, 8>(n, fin, fout, X, ldx, W, ldw, H, ldh, st);
}

template <int BN>
int launch_linear(int64_t n, int32_t fin, int32_t fout, const float* X, int64_t ldx,
                  const float* W, int64_t ldw, float* H, int64_t ldh, hipStream_t st, bool vec) {
  const int64_t n_rt = ceil_div64(n, kBM);
  const int32_t n_ct = (int32_t)ceil_div64(fout, BN);
  const int64_t blocks = n_rt * n_ct;
  if (blocks > (int64_t)UINT32_MAX) return fail(AGCN_ERR_UNSUPPORTED, "matrix too large for one launch");
  if (vec)
    k_linear<BN, true><<<dim3((unsigned)blocks), kThreads, 0, st>>>(n, fin, fout, n_ct, X, ldx, W,
                                                                    ldw, H, ldh);
  else
    k_linear<BN, false><<<dim3((unsigned)blocks), kThreads, 0, st>>>(n, fin, fout, n_ct, X, ldx,
                                                                     W, ldw, H, ldh);
  const hipError_t e = hipGetLastError();
  return e == hipSuccess ? AGCN_OK : hip_fail(e, "k_linear launch");
}

}  // namespace

int run_linear(int64_t n, int32_t fin, int32_t fout, const float* X, int64_t ldx, const float* W,
               int64_t ldw, float* H, int64_t ldh, hipStream_t st) {
  if (n == 0 || fout == 0) return AGCN_OK;
  const bool vec = fin % 4 == 0 && fout % 4 == 0 && ldx % 4 == 0 && ldw % 4 == 0 &&
                   aligned16(X) && aligned16(W);
  // k_linear_rw addresses X and H with 32-bit byte offsets, and its masked
  // offset must lie past both (see kRwOutOfRange); it writes H in 16-byte
  // pieces, so H's rows must be 16-byte aligned too.
  const int64_t lim = (int64_t)kRwOutOfRange - 16;
  const bool rw_fits = n * ldx * 4 <= lim && n * ldh * 4 <= lim && ldh % 4 == 0 && aligned16(H);
  if (vec && rw_fits && fin >= 1 && fin <= 128 && !rw_disabled()) {
    // Wider outputs run as one launch per 128 columns of W and H, each
    // streaming X again (measured at 230,000 x 128 -> 256: two launches take
    // less time than the tiled kernel). Every column's sum is the same as in
    // a single launch.
    for (int32_t c0 = 0; c0 < fout; c0 += 128) {
      const int32_t w = std::min<int32_t>(128, fout - c0);
      const float* Wc = W + c0;
      float* Hc = H + c0;
      int rc;
      if (w <= 32) rc = dispatch_rw<2>(n, fin, w, X, ldx, Wc, ldw, Hc, ldh, st);
      else if (w <= 64) rc = dispatch_rw<4>(n, fin, w, X, ldx, Wc, ldw, Hc, ldh, st);
      else rc = dispatch_rw<8>(n, fin, w, X, ldx, Wc, ldw, Hc, ldh, st);
      if (rc) return rc;
    }
    return AGCN_OK;
  }
  if (fout <= 32) return launch_linear<32>(n, fin, fout, X, ldx, W, ldw, H, ldh, st, vec);
  if (fout <= 64) return launch_linear<64>(n, fin, fout, X, ldx, W, ldw, H, ldh, st, vec);
  return launch_linear<128>(n, fin, fout, X, ldx, W, ldw, H, ldh, st, vec);
}

}  // namespace agcn
