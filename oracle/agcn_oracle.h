/*
 * CPU oracle for the Accel-GCN aggregation path (arXiv 2308.11825).
 *
 * TEST INFRASTRUCTURE ONLY. This library is the plain, slow, single-threaded
 * statement of what the device path must compute. Only the test-suite, the
 * package smoke check and the benchmark's CPU-baseline leg load it; the
 * device library neither links nor calls it, and the two share no code.
 *
 * Every function takes host pointers, never allocates memory the caller must
 * free, and returns a negative value on invalid arguments.
 *
 * Arithmetic: float64 accumulation, one round-to-nearest-even conversion to
 * float32 at the end; no FMA contraction (built with -ffp-contract=off).
 *
 * Readings of the paper taken here (where it is silent or inconsistent):
 *   R1  the degree sort is ascending and stable (ties keep the original row
 *       order) -- fixed by the metadata example of Sec. III-C;
 *   R2  the sort reorders the column-index and value arrays too, not only
 *       the row pointer -- the example's second block starts at nnz 4;
 *   R3  a metadata entry's row field is the sorted position; output rows are
 *       written through the permutation;
 *   R4  Alg. 1 covers degrees 1..deg_bound inclusive (Alg. 2 tests
 *       deg <= deg_bound and the example gives a degree-4 row a pattern at
 *       deg_bound = 4);
 *   R5  entry field order {deg, loc, row, info}; for deg <= deg_bound,
 *       info = warp_nzs << 16 | rows, otherwise info = the chunk's nnz;
 *   R6  Alg. 2 never emits an empty residual entry;
 *   R7  degree-0 rows get entries of up to max_block_warps rows with
 *       warp_nzs = 0, so every output row is written exactly once;
 *   R8  a row of degree > deg_bound is cut into consecutive chunks of
 *       hub_chunk_nnz nnz (the paper uses deg_bound); each chunk's loc is
 *       its own first nnz, and Alg. 2's hub branch runs once per such row;
 *   R9  inside a chunk the block's warps take contiguous slices of
 *       ceil(info / max_block_warps) nnz; inside a non-hub entry a row of
 *       degree d is covered by ceil(d / warp_nzs) consecutive warps.
 */
#ifndef AGCN_ORACLE_H
#define AGCN_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Sec. III-C, degree sorting steps (1)-(2): deg[i] = rowptr[i+1] - rowptr[i],
 * then a stable counting sort, ascending (R1). perm[r] = original row placed
 * at sorted position r. Returns 0, or -1 on a bad argument or a row pointer
 * that decreases. */
int oracle_degree_sort(int32_t n_rows, const int32_t* rowptr, int32_t* perm);

/* Sec. III-C, degree sorting step (3) with R2: the CSR rebuilt with its rows
 * taken in perm order; row-internal order kept. rowptr_s has n_rows + 1
 * entries; colidx_s / vals_s have rowptr[n_rows] entries. */
int oracle_relayout(int32_t n_rows, const int32_t* rowptr, const int32_t* colidx,
                    const float* vals, const int32_t* perm, int32_t* rowptr_s,
                    int32_t* colidx_s, float* vals_s);

/* Alg. 1 (partition patterns) with R4, by its definition: for d = 1..W*Z
 * writes block_rows[d] = W / f and warp_nzs[d] = ceil(d / f), f being the
 * smallest divisor of W with f * Z >= d. Index 0 is set to 0. Both arrays
 * hold W*Z + 1 entries. */
int oracle_patterns(int32_t max_block_warps, int32_t max_warp_nzs,
                    int32_t* block_rows, int32_t* warp_nzs);

/* Alg. 2 (block-level partitioning) with R3-R9 over the sorted row pointer,
 * by its definition: each run of equal-degree sorted rows, in ascending
 * degree, gives ceil(count / block_rows) entries (degree <= deg_bound) or,
 * per row, ceil(degree / hub_chunk_nnz) chunk entries (degree > deg_bound).
 * hub_chunk_nnz <= 0 means deg_bound. meta receives 4 int32 per entry
 * {deg, loc, row, info}; pass meta = NULL to count only. Returns the number
 * of entries, or -1 on a bad argument, or -2 if cap is too small. */
int64_t oracle_partition(int32_t n_rows, const int32_t* rowptr_s,
                         int32_t max_block_warps, int32_t max_warp_nzs,
                         int32_t hub_chunk_nnz, int32_t* meta, int64_t cap);

/* Warp-level partition, the baseline the paper compares block-level
 * partitioning against (Sec. III-C metadata example, panel (b); Table II):
 * no degree sort; each row, in original order, is cut into groups of at most
 * max_warp_nzs consecutive nnz, one group per warp, metadata
 * {row, first nnz, nnz count, 0} (96 bits padded to 128). Reading R14: an
 * empty row gets one group of length 0 so its output row is still written.
 * meta = NULL counts only. Returns the number of groups, -1 on a bad
 * argument, -2 if cap is too small. */
int64_t oracle_warp_partition(int32_t n_rows, const int32_t* rowptr, int32_t max_warp_nzs,
                              int32_t* meta, int64_t cap);

/* Sec. II-A / II-B: Y = A X by its definition. For each row i and column k,
 * Y[i,k] = sum over e in [rowptr[i], rowptr[i+1]) of vals[e] * X[colidx[e], k],
 * summed in float64 in ascending e and rounded once to float32. Optional
 * outputs (NULL to skip): Yd (float64 sums, ld = F) and S (float64 sums of
 * |vals[e]| |X[colidx[e], k]|, ld = F), the scale used by tolerances. */
int oracle_spmm(int32_t n_rows, int32_t n_cols, int32_t F, const int32_t* rowptr,
                const int32_t* colidx, const float* vals, const float* X, int64_t ldx,
                float* Y, int64_t ldy, double* Yd, double* S);

/* The same definition for a list of rows only: out row j holds row rows[j].
 * Y is m x F (ld F); S optional (m x F). */
int oracle_spmm_rows(int32_t n_rows, int32_t n_cols, int32_t F, const int32_t* rowptr,
                     const int32_t* colidx, const float* vals, const float* X,
                     int64_t ldx, const int32_t* rows, int32_t m, float* Y, double* S);

/* Sec. III-C, last paragraph: each warp's workload is deduced from its
 * block's metadata entry (R9). Replays every entry over the sorted CSR:
 * cover[e] counts how often sorted nnz e is visited, row_hits[r] how many
 * entries name sorted row r as one of their rows (0 for rows only reached
 * through hub chunks, which count separately in hub_chunks[r]). Y (n_rows x F,
 * ld F, original row order through perm) is accumulated in float64 in the
 * visiting order and rounded once. Returns 0, or -1 if an entry decodes
 * outside the sorted CSR. */
int oracle_replay_meta(int32_t n_rows, int32_t n_cols, int32_t F, const int32_t* rowptr_s,
                       const int32_t* colidx_s, const float* vals_s, const int32_t* perm,
                       const int32_t* meta, int64_t n_entries, int32_t max_block_warps,
                       int32_t max_warp_nzs, const float* X, int64_t ldx, float* Y,
                       int32_t* cover, int32_t* row_hits, int32_t* hub_chunks);

/* Sec. II-A, the linear transformation of a GCNConv layer: H = X W by its
 * definition. X is n x fin (ld ldx), W is fin x fout (ld ldw), H is n x fout
 * (ld ldh), all row-major. H[i,c] = sum over k ascending of X[i,k] W[k,c],
 * summed in float64 and rounded once to float32. */
int oracle_linear(int64_t n, int32_t fin, int32_t fout, const float* X, int64_t ldx,
                  const float* W, int64_t ldw, float* H, int64_t ldh);

/* Sec. II-A, one GCNConv layer's forward: the linear transformation followed
 * by the aggregation and the element-wise activation,
 *   Y[q,c] = act( sum_e vals[e] * sum_k X[colidx[e],k] W[k,c] ),  i = rows[q],
 * e over row i of the CSR in ascending order, all in float64 (the product
 * X W is not rounded), then rounded once to float32. act: 0 = identity,
 * 1 = ReLU, max(v, 0). Optional S2 (NULL to skip) receives
 * sum_e |vals[e]| sum_k |X[colidx[e],k]| |W[k,c]|, the scale used by
 * tolerances. rows = NULL means every row in order (then m = n_rows). Y and S2
 * are m x fout (ld fout). */
int oracle_gcn_layer_rows(int32_t n_rows, int32_t n_cols, int32_t fin, int32_t fout,
                          const int32_t* rowptr, const int32_t* colidx, const float* vals,
                          const float* X, int64_t ldx, const float* W, int64_t ldw, int32_t act,
                          const int32_t* rows, int32_t m, float* Y, double* S2);

#ifdef __cplusplus
}
#endif
#endif
