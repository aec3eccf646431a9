// Internal declarations shared by the libagcn sources (plan, SpMM, C ABI).
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>
#include <mutex>
#include <string>
#include <utility>
#include <vector>

#include "../../include/agcn.h"

namespace agcn {

// Error flags the plan kernels raise on the device (OR-ed into one word).
enum : uint32_t {
  kErrRowptrStart = 1u << 0,   // rowptr[0] != 0
  kErrRowptrOrder = 1u << 1,   // rowptr decreases
  kErrRowptrEnd = 1u << 2,     // rowptr[n_rows] != nnz
  kErrColumn = 1u << 3,        // a column index outside [0, n_cols)
  kErrInternal = 1u << 8,      // a consistency check of the plan's own kernels
  kErrRelayout = 1u << 9,      // the relayout's window check (a row order that is not
                               // sorted); may be raised after the summary was read
};

// Facts the device computes while partitioning, written into pinned host
// memory. dmax_ready and done are set (after a system-scope fence) once
// max_deg, and then everything else, can be read.
struct PlanSummary {
  int32_t n_entries;
  int32_t hub_first_entry;
  int32_t n_hub_rows;
  int32_t hub_first_row;
  int32_t max_deg;
  int32_t n_tail;   // rows of degree >= 255 (the short sort's tail)
  int32_t nnz_low;  // nonzeros of the rows of degree < 255
  uint32_t err;
  uint32_t dmax_ready;
  uint32_t done;
};

// Largest number of (column, value) pairs one metadata entry stages in LDS.
constexpr int kMaxEntryNnz = 4096;
constexpr int kMaxBlockWaves = 32;
// Feature columns one workgroup covers: 64 lanes x (4 or 1) floats.
constexpr int kSliceLanes = 64;

// Column windows of the hub rows. A plan whose hub rows average at least
// kWinMinPairs nonzeros per (hub row, window of kWinCols columns), over at
// least kWinMinHubRows hub rows, gets a table of where each hub row's
// nonzeros of each window start; executes at F >= kWinMinF then aggregate
// the hub rows window by window from X staged in LDS (k_hub_win) instead of
// by hub chunks. A workgroup holds kWinRows hub rows: 64 lane groups of 16
// lanes, kWinRowsPerGroup rows each.
constexpr int32_t kWinCols = 512;
constexpr int32_t kWinMinPairs = 16;
constexpr int32_t kWinMinHubRows = 64;
constexpr int32_t kWinMinF = 64;
constexpr int32_t kWinSliceCols = 64;
constexpr int32_t kWinRowsPerGroup = 16;
constexpr int32_t kWinRows = 64 * kWinRowsPerGroup;
// Workgroups a launch aims for (one fits per CU: about two rounds on 256 CUs).
constexpr int64_t kWinTargetGroups = 512;

// AGCN_HUB_WINDOWS=0 builds no window table (plans then aggregate hub rows by
// chunks at every F); read at each agcn_plan_create.
bool hub_windows_setting();

}  // namespace agcn

struct agcn_plan {
  int device = 0;
  int32_t n_rows = 0, n_cols = 0;
  int64_t nnz = 0;
  int32_t W = 0, Z = 0, deg_bound = 0, H = 0;
  uint32_t flags = 0;  // AGCN_PLAN_* (0: the block-level method)
  int32_t n_entries = 0, hub_first_entry = 0, n_hub_rows = 0, hub_first_row = 0, max_deg = 0;
  void* base = nullptr;  // single device allocation holding everything below
  size_t bytes = 0;
  int32_t* perm = nullptr;          // [n_rows]   sorted position -> original row
  int32_t* rowptr_s = nullptr;      // [n_rows+1] sorted CSR
  int32_t* colidx_s = nullptr;      // [nnz]
  float* vals_s = nullptr;          // [nnz]
  int4* meta = nullptr;             // [entries upper bound] {deg, loc, row, info}
  int32_t* hub_chunk_off = nullptr; // [hub rows upper bound + 1] first chunk of each hub row
  int32_t* order = nullptr;         // [entries] launch order of k_spmm (entry per workgroup)
  bool hub_wide = false;            // hub chunks of long rows launched in column order
  int32_t* group_off = nullptr;     // warp-level plans: [n_rows + 1] first group of each row
  // Hub-row windows (n_win > 0 only when built): win_tab[k * n_hub_rows + h],
  // k in [0, n_win], is the position in colidx_s of the first nonzero of
  // sorted hub row hub_first_row + h whose column is >= k * kWinCols (a lower
  // bound by search; [0] and [n_win] are the row's ends). Positions do not
  // decrease in k even where a row's columns do not ascend, so the windows
  // always partition each row. It lies in the block at `base`, over the
  // working buffers of the plan's construction.
  int32_t n_win = 0;
  int32_t* win_tab = nullptr;
  uint32_t* err_word = nullptr;     // the plan kernels' error flags (device)
  hipEvent_t ready = nullptr;       // the plan's kernels done (created with the plan,
                                    // recorded on first need: plan_ready_event; use_mu)
  bool ready_recorded = false;
  hipStream_t stream = nullptr;     // the stream the plan was built on (valid until destroy)
  // Last work of the plan on each stream other than its own that ran an
  // execute with it (one event per stream, re-recorded by every call; guarded
  // by use_mu). Release adds one event recorded on the plan's own stream. A
  // later plan that reuses this memory makes its stream wait on them.
  std::mutex use_mu;
  std::vector<std::pair<hipStream_t, hipEvent_t>> uses;
  bool sync_on_release = false;     // an event could not be created: release waits on the device
};

namespace agcn {

// Fault injection for the error-path tests, read from the environment on
// every call (unset in normal use):
//   AGCN_TEST_FAIL_ALLOC=k       the k-th memory allocation attempt (device
//                                block, pinned read-back buffer) of each
//                                agcn_plan_create call on the calling thread
//                                fails as if the memory were exhausted;
//   AGCN_TEST_FAIL_ORDER_SORT=1  the launch-order sort of hub chunks starts
//                                with the internal-error flag raised, as when
//                                one of its scans gives up its bounded wait;
//   AGCN_TEST_TAIL_CAP=c         the short sort takes tails of at most c rows;
//   AGCN_TEST_EARLY_CHECK_NNZ=k  the short sort checks the column indices in
//                                k_degree (and publishes its summary before
//                                the last relayout) for graphs of at most k
//                                nonzeros;
//   AGCN_TEST_TINY=0             no small graph takes the single-workgroup
//                                plan (k_plan_tiny).
void test_alloc_reset();    // start of agcn_plan_create
bool test_alloc_fails();    // counts one allocation attempt; true: fail it
bool test_order_sort_fails();
int test_tail_cap();         // AGCN_TEST_TAIL_CAP, or -2 when unset
long long test_early_check_nnz();  // AGCN_TEST_EARLY_CHECK_NNZ, or -1 when unset
int test_tiny_plan();        // AGCN_TEST_TINY (0: no single-workgroup plan), or 1 when unset

// Thread-local error text (set by the failing call).
void set_error(const std::string& msg);
int fail(int status, const std::string& msg);
int hip_fail(hipError_t e, const char* what);

// Plan construction (agcn_plan.hip). build_plan dispatches on p->flags.
int build_plan(agcn_plan* p, const int32_t* d_rowptr, const int32_t* d_colidx,
               const float* d_vals, hipStream_t stream);

// Workgroups of a warp-level plan (W groups each).
inline int64_t warp_level_blocks(const agcn_plan* p) {
  return p->W > 0 ? (p->n_entries + p->W - 1) / p->W : 0;
}

// Execute (agcn_spmm.hip). act: 0 = identity, 1 = ReLU on every Y write.
// ws holds ws_bytes; the hub windows run when the plan has them, F >=
// kWinMinF, the float4 path applies and ws_bytes >= win_workspace_bytes.
int run_spmm(const agcn_plan* p, int32_t F, const float* X, int64_t ldx, float* Y, int64_t ldy,
             float* ws, size_t ws_bytes, hipStream_t stream, hipEvent_t ev_begin,
             hipEvent_t ev_mid, hipEvent_t ev_end, int32_t act);

// Launch shape of the hub windows at F: n_slices slices of kWinSliceCols
// columns, n_b batches of kWinRows hub rows, the plan's n_win windows taken G
// at a time by n_grp window groups (G chosen so that n_b * n_slices * n_grp is
// about kWinTargetGroups).
struct WinShape {
  int32_t n_slices, n_b, G, n_grp;
};
WinShape win_shape(const agcn_plan* p, int32_t F);
// Workspace of the hub windows at F (0 when the plan has none or F < kWinMinF):
// one partial row of F floats per (hub row, window group).
size_t win_workspace_bytes(const agcn_plan* p, int32_t F);
// Workspace of the hub chunks (and warp-level blocks) at F.
size_t chunk_workspace_bytes(const agcn_plan* p, int32_t F);

// H = X W on matrix cores (agcn_linear.hip).
int run_linear(int64_t n, int32_t fin, int32_t fout, const float* X, int64_t ldx, const float* W,
               int64_t ldw, float* H, int64_t ldh, hipStream_t stream);

// agcn_spmm_noalloc's workspace: a fixed device array of this many bytes in
// agcn_spmm.hip; noalloc_scratch returns its address on `device` (the
// current device), looked up on the first call for that device.
constexpr size_t kNoallocScratchBytes = AGCN_NOALLOC_MAX_WORKSPACE;
constexpr int kMaxDevices = 64;
int noalloc_scratch(int device, float** out);

// Dynamic LDS bytes the SpMM kernel needs for a plan (worst case over F).
size_t spmm_lds_bytes_max(int32_t W, int32_t max_entry_nnz);

// An event and the stream it was recorded on. ev == nullptr stands for the
// work a released plan queued on its own stream, marked by no event.
struct StreamEvent {
  hipEvent_t ev;
  hipStream_t stream;
};

// Plan memory. device_alloc may hand back the block a destroyed plan left in
// the per-device cache (*got receives its size, >= bytes); `stream` then
// waits (device-side) on the events that mark the previous owner's last work
// on other streams; on `stream` itself its own order already puts that work
// first. Work marked by no event on another stream makes it synchronise the
// device instead. device_release keeps the block cached (one per device) with
// those entries and takes ownership of the events; it does not block.
int device_alloc(int device, size_t bytes, hipStream_t stream, void** out, size_t* got);
void device_release(int device, void* ptr, size_t bytes, std::vector<StreamEvent> pending);

// Records, on `stream`, the event that marks the plan's last work there.
void note_use(agcn_plan* p, hipStream_t stream);

// The event after the plan's kernels, recorded on the plan's stream on the
// first call (so it also covers work queued there since) and reused after.
// The event object itself is created with the plan, so this allocates nothing.
int plan_ready_event(agcn_plan* p, hipEvent_t* out);

// Like note_use, but creates no event: a stream that has no event yet marks
// the plan to wait for the device when it is released.
void note_use_noalloc(agcn_plan* p, hipStream_t stream);

inline int64_t ceil_div64(int64_t a, int64_t b) { return (a + b - 1) / b; }
inline bool aligned16(const void* q) { return (reinterpret_cast<uintptr_t>(q) & 15u) == 0; }

}  // namespace agcn
