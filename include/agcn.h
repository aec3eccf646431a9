/*
 * agcn.h -- C ABI of libagcn, the MI355X (gfx950) implementation of the
 * Accel-GCN neighbour-aggregation SpMM (arXiv 2308.11825).
 *
 * The path computes Y = A X, where A is an n_rows x n_cols sparse matrix in
 * CSR (int32 row pointer and column indices, float32 values) -- in a GCN
 * layer, the normalised adjacency A' of Sec. II-A -- and X is a dense
 * row-major n_cols x F float32 matrix. It has two calls, following the
 * paper's split between preprocessing and kernel (Sec. III-C / III-D):
 *
 *   agcn_plan_create  degree sort (Sec. III-C "Degree Sorting") and
 *                     block-level partitioning (Alg. 1, Alg. 2), all on the
 *                     device; independent of F.
 *   agcn_spmm         the SpMM for one F (Sec. III-D): per-block staging of
 *                     the block's column indices and values, warp workloads
 *                     deduced from the block's metadata entry, lanes laid
 *                     across F ("combined warp"), fixed-order partial sums
 *                     in place of the paper's atomics. agcn_spmm_ex adds the
 *                     layer's activation at the Y writes.
 *
 * and, for a whole GCNConv layer (Sec. II-A), agcn_linear (X W on the matrix
 * cores, no plan needed) and agcn_gcn_layer (linear, then the aggregation
 * with the activation).
 *
 * Conventions for every call:
 *   - Pointers named d_* are device pointers (memory of the current HIP
 *     device); h_* are host pointers. The caller owns every pointer it
 *     passes; the library never frees caller memory.
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *   - Return value: AGCN_OK (0) or one of the AGCN_ERR_* codes. On error,
 *     agcn_last_error() describes it (thread-local). Argument checks run on
 *     the host before any HIP call. No C++ exception crosses this boundary.
 *   - Terminology: a "wave" is one 64-lane CDNA wavefront; a "virtual warp"
 *     (vwarp) is the unit the paper calls a warp: one slice of one row's
 *     nnz, covering all F columns. max_block_waves counts vwarps per block.
 */
#ifndef AGCN_H
#define AGCN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum agcn_status {
  AGCN_OK = 0,
  AGCN_ERR_INVALID_ARGUMENT = 1, /* bad pointer, size, parameter or aliasing */
  AGCN_ERR_INVALID_INPUT = 2,    /* CSR content invalid (see agcn_plan_create) */
  AGCN_ERR_UNSUPPORTED = 3,      /* sizes beyond the int32 metadata format */
  AGCN_ERR_OUT_OF_MEMORY = 4,    /* device allocation failed */
  AGCN_ERR_HIP = 5               /* a HIP runtime call or launch failed */
};

/* Partition parameters (Alg. 1): W = max_block_waves vwarps per block, each
 * vwarp holding at most Z = max_wave_nzs nnz; deg_bound = W * Z. Rows of
 * degree > deg_bound are cut into chunks of hub_chunk_nnz nnz (the paper
 * uses deg_bound; 0 selects deg_bound).
 * Limits: 1 <= W <= 32; 1 <= Z; W * Z <= 4096; 0 <= hub_chunk_nnz <= 4096;
 * and one entry must fit the aggregation kernel's 64 KiB of LDS: the staged
 * (column, value) pairs of the largest entry (max(W * Z, H), one pad word per
 * 32) plus W * 64 float4 partial sums (one pad per 8). W = 32 with
 * W * Z = 4096 exceeds it; agcn_plan_create then returns INVALID_ARGUMENT.
 * flags: 0 for the method itself, or one of the two baselines of the paper's
 * ablation study (Table II):
 *   AGCN_PLAN_WARP_LEVEL   no degree sort; each row in original order is cut
 *                          into groups of at most Z nnz, one group per vwarp,
 *                          W vwarps per workgroup regardless of row
 *                          boundaries (the warp-level partition of Sec.
 *                          III-C, panel (b)). Metadata per group:
 *                          {row, first nnz, nnz count, 0}. Rows cut by a
 *                          workgroup boundary are finished by a fixed-order
 *                          reduction kernel (no atomics).
 *   AGCN_PLAN_COLUMN_LOOP  the block-level partition, executed without the
 *                          combined warp: each vwarp is one 64-lane wave,
 *                          one float per lane, looping over F in strips of
 *                          64 columns (the single-warp column traversal of
 *                          Sec. III-D). */
#define AGCN_PLAN_WARP_LEVEL 0x1u
#define AGCN_PLAN_COLUMN_LOOP 0x2u

typedef struct agcn_plan_params {
  int32_t max_block_waves;
  int32_t max_wave_nzs;
  int32_t hub_chunk_nnz;
  uint32_t flags;
} agcn_plan_params;

/* Plan facts, for reporting and for sizing host export buffers. */
typedef struct agcn_plan_stats {
  int32_t n_rows;
  int32_t n_cols;
  int64_t nnz;
  int64_t n_entries;       /* metadata entries = blocks of the partition */
  int64_t hub_first_entry; /* index of the first hub-chunk entry (= n_entries if none) */
  int64_t n_hub_chunks;    /* entries with deg > deg_bound */
  int32_t n_hub_rows;      /* rows with degree > deg_bound */
  int32_t hub_first_row;   /* sorted position of the first such row */
  int32_t deg_bound;       /* W * Z */
  int32_t hub_chunk_nnz;   /* effective H */
  int32_t max_deg;
  int32_t max_block_waves;
  int32_t max_wave_nzs;
  uint32_t flags;          /* the plan's AGCN_PLAN_* flags */
  size_t device_bytes;     /* device memory the plan holds */
  int32_t hub_windows;     /* column windows of 512 columns over which the hub rows are
                              aggregated at F >= 64 (0: hub chunks at every F) */
} agcn_plan_stats;

typedef struct agcn_plan* agcn_plan_t;

/* Fills *p with the library defaults (tuned for MI355X; the paper's own
 * values are W = 12, Z = 32). */
void agcn_default_params(agcn_plan_params* p);

/* Degree sort + block-level partition on the device (Sec. III-C, Alg. 1-2).
 *
 * Inputs: d_rowptr[n_rows + 1], d_colidx[nnz], d_vals[nnz] on the current
 * device; params NULL = defaults. The plan copies what it needs (sorted
 * permutation, sorted CSR copy, metadata). The call's last kernel may still
 * read the inputs when it returns: keep them unchanged until the work it
 * queued on `stream` has run (free or overwrite them in `stream`'s order, or
 * after synchronising it). Work is
 * ordered on `stream`. The call waits on the host, by polling pinned memory,
 * for results the device writes there: the maximum degree with the number of
 * rows of degree >= 255 (which chooses between the plan's degree sorts; the
 * kernels that depend on it are queued before it arrives) and the summary
 * with the number of metadata entries. The plan's last kernels may still run
 * on `stream` when it returns; later work on that stream comes after them,
 * and agcn_spmm* on another stream waits for them. The warp-level plan (AGCN_PLAN_WARP_LEVEL)
 * synchronises `stream` instead. `stream` must remain valid until the plan is
 * destroyed (agcn_plan_destroy marks the plan's last work on it).
 *
 * The CSR is validated on the device: rowptr[0] == 0, non-decreasing,
 * rowptr[n_rows] == nnz, 0 <= colidx[e] < n_cols. A violation returns
 * AGCN_ERR_INVALID_INPUT and no plan. Column indices need not be sorted and
 * may repeat (repeated entries add up).
 *
 * Errors: INVALID_ARGUMENT (null out, negative sizes, null arrays with
 * n_rows > 0 or nnz > 0, parameters outside the limits), UNSUPPORTED
 * (nnz >= 2^31 or n_rows + nnz / H + 1 >= 2^31), OUT_OF_MEMORY, HIP.
 * On any error *out is set to NULL and the device memory the call allocated
 * is released (it may stay in the library's plan-memory cache, which
 * agcn_release_cached_memory empties).
 *
 * Fault injection for tests (environment variables, read on every call;
 * leave them unset in normal use): AGCN_TEST_FAIL_ALLOC=k makes the k-th
 * memory allocation attempt of each agcn_plan_create call on the calling
 * thread fail with OUT_OF_MEMORY; AGCN_TEST_FAIL_ORDER_SORT=1 raises the
 * internal-error flag before the hub-chunk launch-order sort, which then
 * keeps the plain heaviest-first order (the plan stays valid);
 * AGCN_TEST_TAIL_CAP=c lowers to c the number of rows of degree >= 255 that
 * the short degree sort takes (-1: none, so every plan takes the multi-pass
 * sort; the result is the same stable sort either way);
 * AGCN_TEST_EARLY_CHECK_NNZ=k sets to k the largest graph whose column
 * indices the short sort checks before its last relayout, returning while
 * that relayout runs (larger graphs: checked by the relayout, and the call
 * returns after it; the plan is the same either way); AGCN_TEST_TINY=0 keeps
 * graphs of at most 16384 rows and 2^17 nonzeros off the single-workgroup
 * plan (the same plan again).
 *
 * Hub-row windows: when the rows of degree > deg_bound average at least 16
 * nonzeros per window of 512 columns, over at least 64 such rows, the plan
 * also keeps, for each of those rows and each window, the position of the
 * row's first nonzero in the window (built by the call's last kernel, in the
 * plan's own memory; agcn_plan_stats.hub_windows = the number of windows).
 * agcn_spmm at F >= 64 on the 128-bit path then aggregates those rows window
 * by window from X staged in LDS. The columns of a row may come in any order;
 * ascending is fastest. AGCN_HUB_WINDOWS=0 (read on every call) builds no
 * table, so the hub chunks serve every F. */
int agcn_plan_create(agcn_plan_t* out, int32_t n_rows, int32_t n_cols, int64_t nnz,
                     const int32_t* d_rowptr, const int32_t* d_colidx, const float* d_vals,
                     const agcn_plan_params* params, void* stream);

/* Device workspace agcn_spmm needs for feature width F: n_hub_chunks * F * 4
 * bytes (partial rows of the hub chunks; 0 when the plan has no hub rows),
 * or, for a plan with hub-row windows at F >= 64 when that is larger,
 * n_hub_rows * n_groups * (F + 1) * 4 bytes (one partial row and one flag
 * per hub row and group of windows, n_groups about 512 / (ceil(F / 64) *
 * ceil(n_hub_rows / 1024)); 127 MB for 1000 hub rows at F = 64).
 * For AGCN_PLAN_WARP_LEVEL plans: 2 * workgroups * F * 4 bytes (partial rows
 * of the rows cut by workgroup boundaries). */
int agcn_spmm_workspace_size(agcn_plan_t plan, int32_t F, size_t* bytes);

/* Y = A X for one F (Sec. III-D). Asynchronous on `stream`.
 *
 * d_X: n_cols rows of F floats, row stride ldx >= F (elements); d_Y: n_rows
 * rows, stride ldy >= F. Every Y row is written exactly once (empty rows get
 * zeros), so Y needs no clearing. X and Y must not overlap. d_ws: at least
 * agcn_spmm_workspace_size(plan, F) bytes, may be NULL when that is 0.
 * The 128-bit path runs when F, ldx and ldy are multiples of 4 and X, Y, ws
 * are 16-byte aligned; otherwise a 32-bit path runs (same results up to
 * float rounding order, both deterministic).
 * Result: bitwise reproducible run to run; no atomics. The hub rows of a plan
 * with hub-row windows are summed window by window at F >= 64 on the
 * 128-bit path and by hub chunks otherwise (same sums, another rounding
 * order).
 * The plan is read-only here: concurrent calls on different streams are
 * safe when each has its own Y and ws. Must run on the plan's device.
 * The call launches kernels only (no allocation, no memset, no host wait), so
 * it may be captured into a HIP graph; the plan must then outlive every
 * replay of that graph.
 * Errors: INVALID_ARGUMENT (null plan or pointers, F < 1, ld < F, overlap,
 * missing workspace, wrong device), UNSUPPORTED (AGCN_PLAN_COLUMN_LOOP plans
 * when W * F * 4 bytes of partial rows plus the staged entry exceed 64 KiB
 * of LDS), HIP. */
int agcn_spmm(agcn_plan_t plan, int32_t F, const float* d_X, int64_t ldx, float* d_Y,
              int64_t ldy, void* d_ws, void* stream);

/* agcn_spmm plus timing marks on the caller's hipEvent_t handles (each may be
 * NULL): ev_begin is recorded when the aggregation kernel starts and ev_mid
 * when it ends (attached to the kernel's own launch, so no marker packet sits
 * between kernels), ev_end after the hub-row reduction (or the hub-row
 * windows and their reduction). Same kernels, same
 * launch shapes; used to time the aggregation kernel by itself. */
int agcn_spmm_timed(agcn_plan_t plan, int32_t F, const float* d_X, int64_t ldx, float* d_Y,
                    int64_t ldy, void* d_ws, void* stream, void* ev_begin, void* ev_mid,
                    void* ev_end);

/* Epilogues of the aggregation, applied where Y is written: the layer's
 * element-wise activation of Sec. II-A, X^{l+1} = act(A' Y^l). ReLU maps
 * v < 0 to 0 and keeps every other value (NaN and -0 included). */
#define AGCN_EPILOGUE_NONE 0
#define AGCN_EPILOGUE_RELU 1

/* agcn_spmm followed by the epilogue on every element of Y (Sec. II-A). Same
 * arguments, layouts, errors and launches as agcn_spmm, plus epilogue
 * (AGCN_EPILOGUE_NONE or AGCN_EPILOGUE_RELU, else INVALID_ARGUMENT). Rows
 * split over several vwarps or hub chunks get it after their final sum. */
int agcn_spmm_ex(agcn_plan_t plan, int32_t F, const float* d_X, int64_t ldx, float* d_Y,
                 int64_t ldy, void* d_ws, void* stream, int32_t epilogue);

/* agcn_spmm_ex for callers that cannot allocate memory: code being captured
 * into a HIP graph, tight serving loops, harnesses that forbid hipMalloc.
 * Same arguments, kernels and results (bit for bit) as agcn_spmm_ex, without
 * d_ws, except that a plan whose hub-row window partials at this F exceed the
 * fixed workspace takes the hub chunks (same sums, another rounding order):
 * the hub-row partial sums go to a fixed workspace the library keeps in
 * device memory, AGCN_NOALLOC_MAX_WORKSPACE bytes on every GPU it runs on,
 * held until the process ends. The call allocates nothing (no device or host
 * memory, no HIP event): on a stream other than the plan's own on which the
 * plan has not run agcn_spmm / agcn_spmm_ex before, it marks the plan so that
 * agcn_plan_destroy waits for the device instead of tracking the stream with
 * an event. All calls on one GPU share the workspace, and each call writes
 * every part of it that it reads, so nothing needs clearing between calls;
 * calls that may overlap in time on one GPU (different streams, or graph
 * replays running concurrently) race on it and must be ordered by the caller.
 * Errors: those of agcn_spmm_ex, plus UNSUPPORTED when the hub chunks'
 * workspace at F (agcn_spmm_workspace_size for a plan without hub-row
 * windows) exceeds AGCN_NOALLOC_MAX_WORKSPACE. */
#define AGCN_NOALLOC_MAX_WORKSPACE ((size_t)64 << 20)
int agcn_spmm_noalloc(agcn_plan_t plan, int32_t F, const float* d_X, int64_t ldx, float* d_Y,
                      int64_t ldy, void* stream, int32_t epilogue);

/* H = X W, the linear transformation of a GCNConv layer (Sec. II-A), on the
 * fp32 matrix cores. Asynchronous on `stream`; no plan needed.
 *
 * d_X: n rows of fin floats, row stride ldx >= fin; d_W: fin rows of fout
 * floats, stride ldw >= fout; d_H: n rows of fout floats, stride ldh >= fout.
 * All row-major, device memory owned by the caller; H must not overlap X or
 * W. fin = 0 gives H = 0. fp32 products and sums (matrix-core accumulation,
 * fin terms per element). Kernel choice: with fin at most 128, fin, fout,
 * ldx, ldw and ldh multiples of 4, X, W and H 16-byte aligned and X and H
 * each under 4 GiB, W stays resident on chip while X streams past (once per
 * 128 output columns); otherwise a tiled kernel runs (128-bit loads when fin, fout, ldx and ldw are
 * multiples of 4 and X, W are 16-byte aligned, else 32-bit loads with the
 * same results). The two kernels add the fin products in different orders,
 * so their results may differ in the last bits; each is deterministic.
 * Errors: INVALID_ARGUMENT (negative sizes, ld too small, NULL pointers with
 * non-empty extents, overlap), UNSUPPORTED (more than 2^32 - 1 tiles), HIP. */
int agcn_linear(int64_t n, int32_t fin, int32_t fout, const float* d_X, int64_t ldx,
                const float* d_W, int64_t ldw, float* d_H, int64_t ldh, void* stream);

/* Workspace bytes for agcn_gcn_layer with output width fout: H (n_cols x
 * fout floats, rounded up to 256 bytes) followed by the SpMM workspace of
 * agcn_spmm_workspace_size(plan, fout). */
int agcn_gcn_workspace_size(agcn_plan_t plan, int32_t fout, size_t* bytes);

/* One GCNConv layer forward over the plan's graph (Sec. II-A):
 *   H = X W  (agcn_linear into the workspace),  Y = epilogue(A' H)  (the
 *   plan's SpMM with the epilogue fused into its Y writes).
 * d_X: n_cols rows of fin floats (stride ldx); d_W: fin x fout (stride ldw);
 * d_Y: n_rows rows of fout floats (stride ldy); d_ws: at least
 * agcn_gcn_workspace_size(plan, fout) bytes, 16-byte aligned, not
 * overlapping X, W or Y. Asynchronous on `stream`; two launches (three with
 * hub rows). Errors: those of agcn_linear and agcn_spmm_ex, plus
 * INVALID_ARGUMENT for a missing or misaligned workspace. */
int agcn_gcn_layer(agcn_plan_t plan, int32_t fin, int32_t fout, const float* d_X, int64_t ldx,
                   const float* d_W, int64_t ldw, float* d_Y, int64_t ldy, void* d_ws,
                   void* stream, int32_t epilogue);

/* Fills *out. Host-only, no HIP call. */
int agcn_plan_info(agcn_plan_t plan, agcn_plan_stats* out);

/* Copies the plan to host memory (synchronous: waits for the plan's kernels
 * first).
 * Any pointer may be NULL to skip that array. Sizes: h_perm[n_rows] (sorted
 * position -> original row), h_rowptr_s[n_rows + 1], h_colidx_s[nnz],
 * h_vals_s[nnz] (the CSR with rows in sorted order), h_meta[4 * n_entries]
 * ({deg, loc, row, info} per entry: degree of the entry's rows; first nnz
 * in the sorted CSR; first sorted row; for deg <= deg_bound
 * warp_nzs << 16 | rows, else the chunk's nnz). AGCN_PLAN_WARP_LEVEL plans:
 * perm is the identity, the CSR is the input's, and h_meta holds one
 * {row, first nnz, nnz count, 0} per group. Errors: INVALID_ARGUMENT (NULL
 * plan, another current device), HIP (including an internal consistency
 * check of the plan's last relayout, which runs after agcn_plan_create
 * returns: a row order that is not sorted). */
int agcn_plan_export(agcn_plan_t plan, int32_t* h_perm, int32_t* h_rowptr_s,
                     int32_t* h_colidx_s, float* h_vals_s, int32_t* h_meta);

/* Releases the plan without blocking. Its device block is kept in a
 * per-device cache (one block per device) together with events that mark the
 * plan's last work on every stream that used it: one recorded here on the
 * stream the plan was created on (covering its creation and every call made
 * on that stream), and one per other stream, re-recorded by each agcn_spmm* /
 * agcn_gcn_layer call made on it. The next agcn_plan_create on that device
 * that reuses the block makes its own stream wait on those events, so work
 * still queued with the old plan finishes before the memory is overwritten;
 * see agcn_release_cached_memory. The plan must not be used after this call.
 * NULL is ignored. */
void agcn_plan_destroy(agcn_plan_t plan);

/* Frees the device memory cached by destroyed plans, on every device, after
 * waiting (on the host) for the work those plans still had queued. Plans that
 * are still alive are not affected. */
void agcn_release_cached_memory(void);

/* Static text for a status code. */
const char* agcn_status_string(int status);

/* Description of the last error on this thread ("" if none). Valid until the
 * next failing call on the same thread. */
const char* agcn_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* AGCN_H */
