// Drives every oracle function on small and degenerate inputs so that a
// build with AddressSanitizer and UndefinedBehaviorSanitizer sees all of its
// code paths: empty matrices, all-empty rows, repeated columns, hub rows over
// several chunks, a metadata buffer that is too small, invalid inputs. The
// few values it checks are fixed by the paper or by plain definitions: the
// worked example of Sec. III-C, every sorted nnz covered once by the
// partition, and A = I giving Y = X. Prints "oracle sanitize check ok".
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <vector>

#include "../oracle/agcn_oracle.h"

namespace {

int g_fail = 0;
void expect(bool c, const char* what) {
  if (!c) {
    std::printf("FAILED: %s\n", what);
    g_fail = 1;
  }
}

struct Csr {
  int32_t n, n_cols;
  std::vector<int32_t> rowptr, colidx;
  std::vector<float> vals;
};

uint32_t lcg(uint32_t& s) { return s = s * 1664525u + 1013904223u; }

Csr random_csr(int32_t n, int32_t n_cols, const std::vector<int32_t>& deg, uint32_t seed) {
  Csr a{n, n_cols, {0}, {}, {}};
  for (int32_t i = 0; i < n; ++i) {
    for (int32_t t = 0; t < deg[i]; ++t) {
      a.colidx.push_back(n_cols > 0 ? (int32_t)(lcg(seed) % (uint32_t)n_cols) : 0);
      a.vals.push_back((float)((lcg(seed) >> 8) % 1000) / 999.0f - 0.5f);
    }
    a.rowptr.push_back((int32_t)a.colidx.size());
  }
  return a;
}

void run_all(const Csr& a, int32_t W, int32_t Z, int32_t H, int32_t F) {
  const int32_t n = a.n;
  const int64_t nnz = a.rowptr[n];
  std::vector<int32_t> perm(n + 1), rowptr_s(n + 1), colidx_s(nnz + 1);
  std::vector<float> vals_s(nnz + 1);
  expect(oracle_degree_sort(n, a.rowptr.data(), perm.data()) == 0, "degree_sort");
  expect(oracle_relayout(n, a.rowptr.data(), a.colidx.data(), a.vals.data(), perm.data(),
                         rowptr_s.data(), colidx_s.data(), vals_s.data()) == 0, "relayout");
  std::vector<int32_t> br((size_t)W * Z + 1), wn((size_t)W * Z + 1);
  expect(oracle_patterns(W, Z, br.data(), wn.data()) == 0, "patterns");
  const int64_t cnt = oracle_partition(n, rowptr_s.data(), W, Z, H, nullptr, 0);
  expect(cnt >= 0, "partition count");
  std::vector<int32_t> meta(4 * (size_t)(cnt + 1));
  expect(oracle_partition(n, rowptr_s.data(), W, Z, H, meta.data(), cnt) == cnt, "partition");
  if (cnt > 0)
    expect(oracle_partition(n, rowptr_s.data(), W, Z, H, meta.data(), cnt - 1) == -2,
           "partition with too small a buffer");
  std::vector<float> X((size_t)a.n_cols * F + 1), Y((size_t)n * F + 1), Yr((size_t)n * F + 1);
  uint32_t s = 7;
  for (float& x : X) x = (float)((lcg(s) >> 8) % 2001) / 1000.0f - 1.0f;
  std::vector<double> Yd((size_t)n * F + 1), S((size_t)n * F + 1);
  expect(oracle_spmm(n, a.n_cols, F, a.rowptr.data(), a.colidx.data(), a.vals.data(), X.data(), F,
                     Y.data(), F, Yd.data(), S.data()) == 0, "spmm");
  std::vector<int32_t> rows;
  for (int32_t i = n - 1; i >= 0; i -= 3) rows.push_back(i);
  std::vector<float> Ys(rows.size() * F + 1);
  std::vector<double> Ss(rows.size() * F + 1);
  expect(oracle_spmm_rows(n, a.n_cols, F, a.rowptr.data(), a.colidx.data(), a.vals.data(),
                          X.data(), F, rows.data(), (int32_t)rows.size(), Ys.data(),
                          Ss.data()) == 0, "spmm_rows");
  for (size_t q = 0; q < rows.size(); ++q)
    for (int32_t k = 0; k < F; ++k)
      expect(Ys[q * F + k] == Y[(size_t)rows[q] * F + k], "spmm_rows equals spmm");
  std::vector<int32_t> cover(nnz + 1), row_hits(n + 1), hub_chunks(n + 1);
  expect(oracle_replay_meta(n, a.n_cols, F, rowptr_s.data(), colidx_s.data(), vals_s.data(),
                            perm.data(), meta.data(), cnt, W, Z, X.data(), F, Yr.data(),
                            cover.data(), row_hits.data(), hub_chunks.data()) == 0, "replay");
  for (int64_t e = 0; e < nnz; ++e) expect(cover[e] == 1, "every sorted nnz covered once");
  const int64_t gcnt = oracle_warp_partition(n, a.rowptr.data(), Z, nullptr, 0);
  std::vector<int32_t> gmeta(4 * (size_t)(gcnt + 1));
  expect(oracle_warp_partition(n, a.rowptr.data(), Z, gmeta.data(), gcnt) == gcnt, "warp partition");
  const int32_t fout = 3;
  std::vector<float> Wm((size_t)F * fout + 1, 0.25f), Hm((size_t)a.n_cols * fout + 1);
  expect(oracle_linear(a.n_cols, F, fout, X.data(), F, Wm.data(), fout, Hm.data(), fout) == 0,
         "linear");
  std::vector<float> Yl((size_t)n * fout + 1);
  std::vector<double> S2((size_t)n * fout + 1);
  expect(oracle_gcn_layer_rows(n, a.n_cols, F, fout, a.rowptr.data(), a.colidx.data(),
                               a.vals.data(), X.data(), F, Wm.data(), fout, 1, nullptr, 0,
                               Yl.data(), S2.data()) == 0, "gcn layer");
}

}  // namespace

int main() {
  // Sec. III-C worked example: degrees (2, 4, 2), (W, Z) = (2, 2).
  {
    const int32_t rowptr[] = {0, 2, 6, 8};
    int32_t perm[3], rowptr_s[4], colidx_s[8];
    float vals_s[8];
    const int32_t colidx[] = {0, 1, 0, 1, 2, 2, 1, 2};
    const float vals[] = {1, 2, 3, 4, 5, 6, 7, 8};
    expect(oracle_degree_sort(3, rowptr, perm) == 0 && perm[0] == 0 && perm[1] == 2 &&
               perm[2] == 1, "worked example perm");
    oracle_relayout(3, rowptr, colidx, vals, perm, rowptr_s, colidx_s, vals_s);
    expect(rowptr_s[1] == 2 && rowptr_s[2] == 4 && rowptr_s[3] == 8, "worked example rowptr_s");
    int32_t meta[8];
    expect(oracle_partition(3, rowptr_s, 2, 2, 0, meta, 2) == 2, "worked example entries");
    const int32_t want[8] = {2, 0, 0, (2 << 16) | 2, 4, 4, 2, (2 << 16) | 1};
    for (int k = 0; k < 8; ++k) expect(meta[k] == want[k], "worked example meta");
  }
  // A = I gives Y = X exactly.
  {
    const int32_t n = 5, F = 3;
    std::vector<int32_t> rp(n + 1), ci(n);
    std::vector<float> v(n, 1.0f), X(n * F), Y(n * F);
    for (int32_t i = 0; i <= n; ++i) rp[i] = i;
    for (int32_t i = 0; i < n; ++i) ci[i] = i;
    for (int32_t i = 0; i < n * F; ++i) X[i] = 0.1f * (float)i - 0.7f;
    expect(oracle_spmm(n, n, F, rp.data(), ci.data(), v.data(), X.data(), F, Y.data(), F, nullptr,
                       nullptr) == 0, "identity");
    for (int32_t i = 0; i < n * F; ++i) expect(Y[i] == X[i], "identity exact");
  }
  // Degenerate and mixed inputs under several parameter sets.
  run_all(Csr{0, 0, {0}, {}, {}}, 12, 32, 0, 4);
  run_all(random_csr(9, 9, std::vector<int32_t>(9, 0), 1), 4, 8, 0, 5);
  {
    std::vector<int32_t> deg;
    const int32_t pattern[] = {0, 1, 2, 3, 7, 8, 9, 31, 32, 33, 64, 65, 200, 511, 512, 513, 1500};
    for (int r = 0; r < 6; ++r)
      for (int32_t d : pattern) deg.push_back(d);
    const int32_t n = (int32_t)deg.size();
    const Csr a = random_csr(n, 50, deg, 3);  // few columns: repeated entries in most rows
    run_all(a, 16, 32, 0, 8);
    run_all(a, 12, 32, 100, 3);
    run_all(a, 1, 1, 1, 1);
    run_all(a, 32, 2, 4096, 2);
    run_all(a, 6, 3, 7, 17);
  }
  // Invalid inputs are refused, not read out of bounds.
  {
    const int32_t bad_rowptr[] = {0, 3, 2};
    int32_t perm[2];
    expect(oracle_degree_sort(2, bad_rowptr, perm) == -1, "decreasing row pointer refused");
    int32_t br[4], wn[4];
    expect(oracle_patterns(0, 3, br, wn) == -1, "W = 0 refused");
    const int32_t rp[] = {0, 1};
    const int32_t ci[] = {5};
    const float v[] = {1.0f};
    float X[2] = {1, 2}, Y[1];
    expect(oracle_spmm(1, 2, 1, rp, ci, v, X, 1, Y, 1, nullptr, nullptr) == -1,
           "column outside n_cols refused");
  }
  if (g_fail) return 1;
  std::printf("oracle sanitize check ok\n");
  return 0;
}
