// CPU oracle for the Accel-GCN aggregation path (arXiv 2308.11825).
//
// TEST INFRASTRUCTURE ONLY: the plain statement of what the device path must
// compute, used by the tests, the smoke check and the CPU-baseline timing.
// Nothing here is shared with the device library. The readings R1-R9 of the
// paper that this file follows are listed in agcn_oracle.h.
//
// Style: single-threaded, straight loops following the paper's definitions, float64
// accumulation. Built with -O2 -ffp-contract=off.
#include "agcn_oracle.h"

#include <algorithm>
#include <cstdint>
#include <cstring>
#include <vector>

namespace {

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

bool rowptr_ok(int32_t n_rows, const int32_t* rowptr) {
  if (n_rows < 0 || rowptr == nullptr) return false;
  if (rowptr[0] != 0) return false;
  for (int32_t i = 0; i < n_rows; ++i)
    if (rowptr[i + 1] < rowptr[i]) return false;
  return true;
}

// Alg. 1 by its definition (R4): for a degree d in 1..W*Z, f(d) is the
// smallest divisor f of W for which f warps of Z nnz hold d nnz (f * Z >= d).
// A block then holds W / f rows of that degree, and each of a row's f warps
// ceil(d / f) of its nnz. f = W always qualifies, since W * Z = deg_bound >= d.
void patterns(int32_t W, int32_t Z, std::vector<int32_t>& block_rows,
              std::vector<int32_t>& warp_nzs) {
  const int32_t deg_bound = W * Z;
  block_rows.assign(deg_bound + 1, 0);
  warp_nzs.assign(deg_bound + 1, 0);
  for (int32_t d = 1; d <= deg_bound; ++d) {
    int32_t f = 1;
    while (W % f != 0 || (int64_t)f * Z < d) ++f;
    block_rows[d] = W / f;
    warp_nzs[d] = (int32_t)ceil_div(d, f);
  }
}

}  // namespace

extern "C" {

// Sec. III-C, degree sorting: (1) degrees from the row pointer, (2) a stable
// counting sort by degree, ascending (R1).
int oracle_degree_sort(int32_t n_rows, const int32_t* rowptr, int32_t* perm) {
  if (!rowptr_ok(n_rows, rowptr) || (n_rows > 0 && perm == nullptr)) return -1;
  int32_t max_deg = 0;
  for (int32_t i = 0; i < n_rows; ++i) {
    int32_t d = rowptr[i + 1] - rowptr[i];
    if (d > max_deg) max_deg = d;
  }
  // count[d] = number of rows of degree d; start[d] = exclusive prefix sum.
  std::vector<int64_t> start((size_t)max_deg + 2, 0);
  for (int32_t i = 0; i < n_rows; ++i) start[rowptr[i + 1] - rowptr[i] + 1] += 1;
  for (size_t d = 1; d < start.size(); ++d) start[d] += start[d - 1];
  // Visiting rows in original order keeps ties in original order.
  for (int32_t i = 0; i < n_rows; ++i) {
    int32_t d = rowptr[i + 1] - rowptr[i];
    perm[start[d]++] = i;
  }
  return 0;
}

// Sec. III-C, degree sorting step (3) with R2: rows copied in sorted order.
int oracle_relayout(int32_t n_rows, const int32_t* rowptr, const int32_t* colidx,
                    const float* vals, const int32_t* perm, int32_t* rowptr_s,
                    int32_t* colidx_s, float* vals_s) {
  if (!rowptr_ok(n_rows, rowptr) || rowptr_s == nullptr) return -1;
  rowptr_s[0] = 0;
  for (int32_t r = 0; r < n_rows; ++r) {
    int32_t i = perm[r];
    if (i < 0 || i >= n_rows) return -1;
    int32_t d = rowptr[i + 1] - rowptr[i];
    rowptr_s[r + 1] = rowptr_s[r] + d;
    for (int32_t t = 0; t < d; ++t) {
      colidx_s[rowptr_s[r] + t] = colidx[rowptr[i] + t];
      vals_s[rowptr_s[r] + t] = vals[rowptr[i] + t];
    }
  }
  return 0;
}

int oracle_patterns(int32_t max_block_warps, int32_t max_warp_nzs, int32_t* block_rows,
                    int32_t* warp_nzs) {
  if (max_block_warps < 1 || max_warp_nzs < 1 || block_rows == nullptr || warp_nzs == nullptr)
    return -1;
  if ((int64_t)max_block_warps * max_warp_nzs > (1 << 24)) return -1;
  std::vector<int32_t> br, wn;
  patterns(max_block_warps, max_warp_nzs, br, wn);
  std::memcpy(block_rows, br.data(), br.size() * sizeof(int32_t));
  std::memcpy(warp_nzs, wn.data(), wn.size() * sizeof(int32_t));
  return 0;
}

// Alg. 2 by its definition. The degree sort leaves the rows of each degree as
// one run of consecutive sorted rows; runs are taken in ascending degree and
// each is cut on its own (R3, R5-R8):
//   d <= deg_bound: ceil(c / b) entries of b = block_rows(d) consecutive rows
//                   (b = W for d = 0), the last one holding what remains;
//   d >  deg_bound: every row of the run, in sorted order, becomes
//                   ceil(d / H) entries of H consecutive nnz, the last one
//                   holding what remains.
int64_t oracle_partition(int32_t n_rows, const int32_t* rowptr_s, int32_t max_block_warps,
                         int32_t max_warp_nzs, int32_t hub_chunk_nnz, int32_t* meta,
                         int64_t cap) {
  if (!rowptr_ok(n_rows, rowptr_s) || max_block_warps < 1 || max_warp_nzs < 1) return -1;
  const int64_t W = max_block_warps;
  const int64_t deg_bound = W * max_warp_nzs;
  if (deg_bound > (1 << 24) || max_block_warps > 0xFFFF || max_warp_nzs > 0xFFFF) return -1;
  const int64_t H = hub_chunk_nnz > 0 ? hub_chunk_nnz : deg_bound;
  std::vector<int32_t> block_rows, warp_nzs;
  patterns(max_block_warps, max_warp_nzs, block_rows, warp_nzs);

  int64_t count = 0;
  auto emit = [&](int64_t deg, int64_t loc, int64_t row, int64_t info) {
    if (meta != nullptr) {
      if (count >= cap) return false;
      meta[4 * count + 0] = (int32_t)deg;
      meta[4 * count + 1] = (int32_t)loc;
      meta[4 * count + 2] = (int32_t)row;
      meta[4 * count + 3] = (int32_t)info;
    }
    ++count;
    return true;
  };
  auto degree = [&](int64_t r) { return (int64_t)rowptr_s[r + 1] - rowptr_s[r]; };

  for (int64_t r0 = 0; r0 < n_rows;) {
    const int64_t d = degree(r0);
    int64_t r1 = r0 + 1;  // the run of rows of degree d is [r0, r1)
    while (r1 < n_rows && degree(r1) == d) ++r1;
    const int64_t c = r1 - r0;
    if (d <= deg_bound) {
      const int64_t b = d == 0 ? W : block_rows[d];
      const int64_t wn = d == 0 ? 0 : warp_nzs[d];
      for (int64_t k = 0; k < ceil_div(c, b); ++k) {
        const int64_t row = r0 + k * b;
        const int64_t rows = std::min(b, c - k * b);
        if (!emit(d, rowptr_s[row], row, (wn << 16) | rows)) return -2;
      }
    } else {
      for (int64_t row = r0; row < r1; ++row)
        for (int64_t k = 0; k < ceil_div(d, H); ++k)
          if (!emit(d, rowptr_s[row] + k * H, row, std::min(H, d - k * H))) return -2;
    }
    r0 = r1;
  }
  return count;
}

// Sec. III-C, panel (b) of the metadata example: the warp-level partition.
int64_t oracle_warp_partition(int32_t n_rows, const int32_t* rowptr, int32_t max_warp_nzs,
                              int32_t* meta, int64_t cap) {
  if (!rowptr_ok(n_rows, rowptr) || max_warp_nzs < 1) return -1;
  int64_t count = 0;
  for (int32_t row = 0; row < n_rows; ++row) {
    const int64_t deg = rowptr[row + 1] - rowptr[row];
    int64_t start = 0;
    do {  // at least one group per row (R14)
      const int64_t len = std::min<int64_t>(max_warp_nzs, deg - start);
      if (meta != nullptr) {
        if (count >= cap) return -2;
        meta[4 * count + 0] = row;
        meta[4 * count + 1] = (int32_t)(rowptr[row] + start);
        meta[4 * count + 2] = (int32_t)len;
        meta[4 * count + 3] = 0;
      }
      ++count;
      start += max_warp_nzs;
    } while (start < deg);
  }
  return count;
}

// Sec. II-A/II-B: the aggregation A' Y by its definition.
int oracle_spmm(int32_t n_rows, int32_t n_cols, int32_t F, const int32_t* rowptr,
                const int32_t* colidx, const float* vals, const float* X, int64_t ldx,
                float* Y, int64_t ldy, double* Yd, double* S) {
  if (!rowptr_ok(n_rows, rowptr) || F < 0 || ldx < F || ldy < F) return -1;
  std::vector<double> acc((size_t)F), mag((size_t)F);
  for (int32_t i = 0; i < n_rows; ++i) {
    std::fill(acc.begin(), acc.end(), 0.0);
    std::fill(mag.begin(), mag.end(), 0.0);
    for (int32_t e = rowptr[i]; e < rowptr[i + 1]; ++e) {
      const int32_t j = colidx[e];
      if (j < 0 || j >= n_cols) return -1;
      const double a = (double)vals[e];
      const float* xr = X + (int64_t)j * ldx;
      for (int32_t k = 0; k < F; ++k) {
        const double p = a * (double)xr[k];
        acc[k] += p;
        mag[k] += p < 0 ? -p : p;
      }
    }
    for (int32_t k = 0; k < F; ++k) {
      Y[(int64_t)i * ldy + k] = (float)acc[k];
      if (Yd) Yd[(int64_t)i * F + k] = acc[k];
      if (S) S[(int64_t)i * F + k] = mag[k];
    }
  }
  return 0;
}

int oracle_spmm_rows(int32_t n_rows, int32_t n_cols, int32_t F, const int32_t* rowptr,
                     const int32_t* colidx, const float* vals, const float* X, int64_t ldx,
                     const int32_t* rows, int32_t m, float* Y, double* S) {
  if (n_rows < 0 || rowptr == nullptr || F < 0 || ldx < F || m < 0) return -1;
  std::vector<double> acc((size_t)F), mag((size_t)F);
  for (int32_t q = 0; q < m; ++q) {
    const int32_t i = rows[q];
    if (i < 0 || i >= n_rows || rowptr[i + 1] < rowptr[i]) return -1;
    std::fill(acc.begin(), acc.end(), 0.0);
    std::fill(mag.begin(), mag.end(), 0.0);
    for (int32_t e = rowptr[i]; e < rowptr[i + 1]; ++e) {
      const int32_t j = colidx[e];
      if (j < 0 || j >= n_cols) return -1;
      const double a = (double)vals[e];
      const float* xr = X + (int64_t)j * ldx;
      for (int32_t k = 0; k < F; ++k) {
        const double p = a * (double)xr[k];
        acc[k] += p;
        mag[k] += p < 0 ? -p : p;
      }
    }
    for (int32_t k = 0; k < F; ++k) {
      Y[(int64_t)q * F + k] = (float)acc[k];
      if (S) S[(int64_t)q * F + k] = mag[k];
    }
  }
  return 0;
}

// Sec. III-C, last paragraph: a warp's workload follows from its block's entry.
int oracle_replay_meta(int32_t n_rows, int32_t n_cols, int32_t F, const int32_t* rowptr_s,
                       const int32_t* colidx_s, const float* vals_s, const int32_t* perm,
                       const int32_t* meta, int64_t n_entries, int32_t max_block_warps,
                       int32_t max_warp_nzs, const float* X, int64_t ldx, float* Y,
                       int32_t* cover, int32_t* row_hits, int32_t* hub_chunks) {
  if (!rowptr_ok(n_rows, rowptr_s) || max_block_warps < 1 || max_warp_nzs < 1 || F < 0)
    return -1;
  const int64_t W = max_block_warps;
  const int64_t deg_bound = W * max_warp_nzs;
  const int64_t nnz = rowptr_s[n_rows];
  std::vector<double> acc((size_t)n_rows * (size_t)F, 0.0);
  std::memset(cover, 0, (size_t)nnz * sizeof(int32_t));
  std::memset(row_hits, 0, (size_t)n_rows * sizeof(int32_t));
  std::memset(hub_chunks, 0, (size_t)n_rows * sizeof(int32_t));

  auto visit = [&](int64_t r, int64_t begin, int64_t len) {
    if (r < 0 || r >= n_rows || begin < rowptr_s[r] || begin + len > rowptr_s[r + 1]) return false;
    double* a = acc.data() + (size_t)r * F;
    for (int64_t e = begin; e < begin + len; ++e) {
      cover[e] += 1;
      const int32_t j = colidx_s[e];
      if (j < 0 || j >= n_cols) return false;
      const float* xr = X + (int64_t)j * ldx;
      for (int32_t k = 0; k < F; ++k) a[k] += (double)vals_s[e] * (double)xr[k];
    }
    return true;
  };

  for (int64_t b = 0; b < n_entries; ++b) {
    const int64_t deg = meta[4 * b + 0], loc = meta[4 * b + 1];
    const int64_t row = meta[4 * b + 2], info = (uint32_t)meta[4 * b + 3];
    if (deg < 0) return -1;
    if (deg <= deg_bound) {
      const int64_t wn = info >> 16, rows = info & 0xFFFF;
      if (row < 0 || row + rows > n_rows) return -1;
      if (deg == 0) {
        for (int64_t k = 0; k < rows; ++k) row_hits[row + k] += 1;
        continue;
      }
      if (wn <= 0) return -1;
      const int64_t wpr = ceil_div(deg, wn);  // warps per row
      for (int64_t v = 0; v < rows * wpr; ++v) {
        const int64_t rl = v / wpr, part = v % wpr;
        const int64_t begin = loc + rl * deg + part * wn;
        const int64_t len = std::min<int64_t>(wn, deg - part * wn);
        if (part == 0) row_hits[row + rl] += 1;
        if (!visit(row + rl, begin, len)) return -1;
      }
    } else {
      if (row < 0 || row >= n_rows) return -1;
      hub_chunks[row] += 1;
      const int64_t s = ceil_div(info, W);
      for (int64_t v = 0; v < W; ++v) {
        const int64_t begin = loc + v * s;
        const int64_t end = std::min<int64_t>(loc + (v + 1) * s, loc + info);
        if (end > begin && !visit(row, begin, end - begin)) return -1;
      }
    }
  }
  for (int32_t r = 0; r < n_rows; ++r) {
    const int32_t i = perm[r];
    if (i < 0 || i >= n_rows) return -1;
    for (int32_t k = 0; k < F; ++k)
      Y[(int64_t)i * F + k] = (float)acc[(size_t)r * F + k];
  }
  return 0;
}

// Sec. II-A, linear transformation.
int oracle_linear(int64_t n, int32_t fin, int32_t fout, const float* X, int64_t ldx,
                  const float* W, int64_t ldw, float* H, int64_t ldh) {
  if (n < 0 || fin < 0 || fout < 0 || ldx < fin || ldw < fout || ldh < fout) return -1;
  if (n > 0 && fout > 0 && (H == nullptr || (fin > 0 && (X == nullptr || W == nullptr))))
    return -1;
  for (int64_t i = 0; i < n; ++i)
    for (int32_t c = 0; c < fout; ++c) {
      double acc = 0.0;
      for (int32_t k = 0; k < fin; ++k) acc += (double)X[i * ldx + k] * (double)W[(int64_t)k * ldw + c];
      H[i * ldh + c] = (float)acc;
    }
  return 0;
}

// Sec. II-A, GCNConv forward in the paper's two steps: (1) the linear
// transformation H = X W, kept in float64 (with |X| |W| for the scale), for
// every node some selected row references; (2) the aggregation A' H with the
// activation, float64, rounded once.
int oracle_gcn_layer_rows(int32_t n_rows, int32_t n_cols, int32_t fin, int32_t fout,
                          const int32_t* rowptr, const int32_t* colidx, const float* vals,
                          const float* X, int64_t ldx, const float* W, int64_t ldw, int32_t act,
                          const int32_t* rows, int32_t m, float* Y, double* S2) {
  if (n_rows < 0 || n_cols < 0 || fin < 0 || fout < 0 || ldx < fin || ldw < fout ||
      rowptr == nullptr || (act != 0 && act != 1))
    return -1;
  if (rows == nullptr) m = n_rows;
  if (m < 0) return -1;
  // nodes whose row of H is needed
  std::vector<int64_t> slot((size_t)n_cols, -1);
  int64_t n_need = 0;
  for (int32_t q = 0; q < m; ++q) {
    const int32_t i = rows ? rows[q] : q;
    if (i < 0 || i >= n_rows || rowptr[i + 1] < rowptr[i]) return -1;
    for (int32_t e = rowptr[i]; e < rowptr[i + 1]; ++e) {
      const int32_t j = colidx[e];
      if (j < 0 || j >= n_cols) return -1;
      if (slot[j] < 0) slot[j] = n_need++;
    }
  }
  // step (1): H = X W and |X| |W| for those nodes
  std::vector<double> H((size_t)n_need * fout), Hm((size_t)n_need * fout);
  for (int32_t j = 0; j < n_cols; ++j) {
    if (slot[j] < 0) continue;
    double* h = &H[(size_t)slot[j] * fout];
    double* hm = &Hm[(size_t)slot[j] * fout];
    for (int32_t c = 0; c < fout; ++c) {
      double s = 0.0, sm = 0.0;
      for (int32_t k = 0; k < fin; ++k) {
        const double p = (double)X[(int64_t)j * ldx + k] * (double)W[(int64_t)k * ldw + c];
        s += p;
        sm += p < 0 ? -p : p;
      }
      h[c] = s;
      hm[c] = sm;
    }
  }
  // step (2): act(A' H)
  std::vector<double> acc((size_t)fout), mag((size_t)fout);
  for (int32_t q = 0; q < m; ++q) {
    const int32_t i = rows ? rows[q] : q;
    std::fill(acc.begin(), acc.end(), 0.0);
    std::fill(mag.begin(), mag.end(), 0.0);
    for (int32_t e = rowptr[i]; e < rowptr[i + 1]; ++e) {
      const double* h = &H[(size_t)slot[colidx[e]] * fout];
      const double* hm = &Hm[(size_t)slot[colidx[e]] * fout];
      const double a = (double)vals[e];
      const double am = a < 0 ? -a : a;
      for (int32_t c = 0; c < fout; ++c) {
        acc[c] += a * h[c];
        mag[c] += am * hm[c];
      }
    }
    for (int32_t c = 0; c < fout; ++c) {
      const double v = (act == 1 && acc[c] < 0.0) ? 0.0 : acc[c];
      Y[(int64_t)q * fout + c] = (float)v;
      if (S2) S2[(int64_t)q * fout + c] = mag[c];
    }
  }
  return 0;
}

}  // extern "C"
