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

#include "agcn_internal.hpp"

namespace agcn {
namespace {

typedef float f16v __attribute__((ext_vector_type(16)));
typedef float f4 __attribute__((ext_vector_type(4)));

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
  if (fout <= 32) return launch_linear<32>(n, fin, fout, X, ldx, W, ldw, H, ldh, st, vec);
  if (fout <= 64) return launch_linear<64>(n, fin, fout, X, ldx, W, ldw, H, ldh, st, vec);
  return launch_linear<128>(n, fin, fout, X, ldx, W, ldw, H, ldh, st, vec);
}

}  // namespace agcn
