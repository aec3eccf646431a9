// C ABI of libagcn: argument checking, error reporting, plan lifetime.
// Every check that can be made on the host runs before the first HIP call.
#include <algorithm>
#include <climits>
#include <cstdlib>
#include <cstring>
#include <map>
#include <mutex>
#include <new>
#include <string>

#include "agcn_internal.hpp"

namespace agcn {

namespace {
thread_local std::string g_last_error;

bool ranges_overlap(const void* a, size_t a_bytes, const void* b, size_t b_bytes) {
  if (a_bytes == 0 || b_bytes == 0) return false;
  const uintptr_t a0 = reinterpret_cast<uintptr_t>(a), b0 = reinterpret_cast<uintptr_t>(b);
  return a0 < b0 + b_bytes && b0 < a0 + a_bytes;
}

// Bytes spanned by `rows` rows of F floats with stride ld (0 if rows == 0);
// false if it does not fit in size_t.
bool span_bytes(int64_t rows, int64_t ld, int64_t F, size_t* out) {
  if (rows <= 0) {
    *out = 0;
    return true;
  }
  if (ld > (INT64_MAX / 4 - F) / rows) return false;
  *out = (size_t)(((rows - 1) * ld + F) * 4);
  return true;
}
}  // namespace

namespace {
thread_local int g_alloc_attempts = 0;

int env_int(const char* name) {
  const char* v = std::getenv(name);
  return v ? std::atoi(v) : 0;
}
}  // namespace

void test_alloc_reset() { g_alloc_attempts = 0; }

bool test_alloc_fails() {
  const int k = env_int("AGCN_TEST_FAIL_ALLOC");
  return ++g_alloc_attempts == k && k > 0;
}

bool test_order_sort_fails() { return env_int("AGCN_TEST_FAIL_ORDER_SORT") != 0; }

int test_tail_cap() {
  const char* v = std::getenv("AGCN_TEST_TAIL_CAP");
  return v ? std::atoi(v) : -2;
}

int test_tiny_plan() {
  const char* v = std::getenv("AGCN_TEST_TINY");
  return v ? std::atoi(v) : 1;
}

long long test_early_check_nnz() {
  const char* v = std::getenv("AGCN_TEST_EARLY_CHECK_NNZ");
  return v ? std::atoll(v) : -1;
}

void set_error(const std::string& msg) { g_last_error = msg; }

int fail(int status, const std::string& msg) {
  g_last_error = msg;
  return status;
}

int hip_fail(hipError_t e, const char* what) {
  (void)hipGetLastError();
  g_last_error = std::string(what) + ": " + hipGetErrorName(e) + " (" + hipGetErrorString(e) + ")";
  return AGCN_ERR_HIP;
}

// --- plan memory cache ------------------------------------------------------
// Creating and destroying plans of similar size (a new graph per batch, or the
// same graph re-planned) would otherwise pay a hipMalloc and a hipFree --
// which synchronises the device -- each time. A destroyed plan's block stays
// cached, one block per device, and the next plan on that device reuses it
// when it fits without wasting more than half of it. The block travels with
// events marking its previous owner's last work on the streams its executes
// ran on; the reusing plan's stream waits on those of the other streams (on
// its own stream, stream order already does it, and a wait would add a
// barrier packet, around which the GPU idles for microseconds), so nothing
// blocks on the host. The previous owner's own stream has no event (the same
// marker cost at every release): a plan on another stream synchronises the
// device before reusing the block.
namespace {
// Events that only order device work (another stream's wait) or precede a
// hipFree: a device-scope release, without the system-scope cache writeback
// that makes the GPU idle for microseconds around the marker.
constexpr unsigned kOrderEventFlags = hipEventDisableTiming | hipEventReleaseToDevice;

struct CachedBlock {
  void* ptr = nullptr;
  size_t bytes = 0;
  std::vector<StreamEvent> pending;
};
std::mutex g_cache_mu;
std::map<int, CachedBlock> g_cache;

// Frees a block no plan will reuse (the caller has made its device current).
void free_block(CachedBlock& b) {
  bool sync = false;
  for (const StreamEvent& se : b.pending) {
    if (se.ev == nullptr) {
      sync = true;
      continue;
    }
    (void)hipEventSynchronize(se.ev);
    (void)hipEventDestroy(se.ev);
  }
  if (sync) (void)hipDeviceSynchronize();
  b.pending.clear();
  if (b.ptr) (void)hipFree(b.ptr);
  b.ptr = nullptr;
  b.bytes = 0;
}

int with_device(int device, int* prev) {
  hipError_t e = hipGetDevice(prev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (*prev != device && (e = hipSetDevice(device)) != hipSuccess) return hip_fail(e, "hipSetDevice");
  return AGCN_OK;
}
}  // namespace

int device_alloc(int device, size_t bytes, hipStream_t stream, void** out, size_t* got) {
  CachedBlock reuse;
  {
    std::lock_guard<std::mutex> lk(g_cache_mu);
    auto it = g_cache.find(device);
    if (it != g_cache.end() && it->second.ptr != nullptr && it->second.bytes >= bytes &&
        it->second.bytes / 2 <= bytes) {
      reuse = std::move(it->second);
      it->second = CachedBlock{};
    }
  }
  if (reuse.ptr != nullptr) {
    bool sync = false;
    for (const StreamEvent& se : reuse.pending) {
      if (se.ev == nullptr) {  // no event: stream order, or the whole device
        sync = sync || se.stream != stream;
        continue;
      }
      if (se.stream != stream && hipStreamWaitEvent(stream, se.ev, 0) != hipSuccess) {
        (void)hipGetLastError();
        (void)hipEventSynchronize(se.ev);
      }
      (void)hipEventDestroy(se.ev);
    }
    if (sync) (void)hipDeviceSynchronize();
    *out = reuse.ptr;
    *got = reuse.bytes;
    return AGCN_OK;
  }
  void* p = nullptr;
  const bool injected = test_alloc_fails();  // the attempt fails, retry included
  hipError_t e = injected ? hipErrorOutOfMemory : hipMalloc(&p, bytes);
  if (e == hipErrorOutOfMemory && !injected) {
    // Give the cached block back to the device and try once more.
    (void)hipGetLastError();
    CachedBlock old;
    {
      std::lock_guard<std::mutex> lk(g_cache_mu);
      old = std::move(g_cache[device]);
      g_cache[device] = CachedBlock{};
    }
    free_block(old);
    e = hipMalloc(&p, bytes);
  }
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return fail(e == hipErrorOutOfMemory ? AGCN_ERR_OUT_OF_MEMORY : AGCN_ERR_HIP,
                std::string("hipMalloc of ") + std::to_string(bytes) + " bytes failed: " +
                    hipGetErrorString(e));
  }
  *out = p;
  *got = bytes;
  return AGCN_OK;
}

void device_release(int device, void* ptr, size_t bytes, std::vector<StreamEvent> pending) {
  int prev = 0;
  if (with_device(device, &prev) != AGCN_OK) return;
  CachedBlock incoming{ptr, bytes, std::move(pending)};
  CachedBlock evict;
  if (ptr == nullptr) {
    evict = std::move(incoming);
  } else {
    std::lock_guard<std::mutex> lk(g_cache_mu);
    CachedBlock& slot = g_cache[device];
    if (slot.ptr == nullptr || slot.bytes <= bytes) {
      evict = std::move(slot);
      slot = std::move(incoming);
    } else {
      evict = std::move(incoming);
    }
  }
  free_block(evict);
  if (prev != device) (void)hipSetDevice(prev);
}

// Recorded only when needed: an execute on another stream, or a host copy.
// Recording it at the end of every plan cost about 5 us of host time on the
// way to the first execute, which usually runs on the plan's own stream.
int plan_ready_event(agcn_plan* p, hipEvent_t* out) {
  std::lock_guard<std::mutex> lk(p->use_mu);
  if (p->ready == nullptr) return fail(AGCN_ERR_HIP, "the plan has no readiness event");
  if (!p->ready_recorded) {
    const hipError_t e = hipEventRecord(p->ready, p->stream);
    if (e != hipSuccess) return hip_fail(e, "hipEventRecord(plan ready)");
    p->ready_recorded = true;
  }
  *out = p->ready;
  return AGCN_OK;
}

void note_use_noalloc(agcn_plan* p, hipStream_t stream) {
  std::lock_guard<std::mutex> lk(p->use_mu);
  for (auto& u : p->uses) {
    if (u.first == stream) {
      if (hipEventRecord(u.second, stream) != hipSuccess) {
        (void)hipGetLastError();
        p->sync_on_release = true;
      }
      return;
    }
  }
  p->sync_on_release = true;
}

void note_use(agcn_plan* p, hipStream_t stream) {
  std::lock_guard<std::mutex> lk(p->use_mu);
  for (auto& u : p->uses) {
    if (u.first == stream) {
      if (hipEventRecord(u.second, stream) != hipSuccess) {
        (void)hipGetLastError();
        p->sync_on_release = true;
      }
      return;
    }
  }
  hipEvent_t ev = nullptr;
  if (hipEventCreateWithFlags(&ev, kOrderEventFlags) != hipSuccess ||
      hipEventRecord(ev, stream) != hipSuccess) {
    (void)hipGetLastError();
    if (ev) (void)hipEventDestroy(ev);
    p->sync_on_release = true;
    return;
  }
  p->uses.emplace_back(stream, ev);
}

}  // namespace agcn

using agcn::fail;

extern "C" {

void agcn_default_params(agcn_plan_params* p) {
  if (p == nullptr) return;
  p->max_block_waves = 16;
  p->max_wave_nzs = 32;
  p->hub_chunk_nnz = 0;
  p->flags = 0;
}

const char* agcn_status_string(int status) {
  switch (status) {
    case AGCN_OK: return "AGCN_OK";
    case AGCN_ERR_INVALID_ARGUMENT: return "AGCN_ERR_INVALID_ARGUMENT";
    case AGCN_ERR_INVALID_INPUT: return "AGCN_ERR_INVALID_INPUT";
    case AGCN_ERR_UNSUPPORTED: return "AGCN_ERR_UNSUPPORTED";
    case AGCN_ERR_OUT_OF_MEMORY: return "AGCN_ERR_OUT_OF_MEMORY";
    case AGCN_ERR_HIP: return "AGCN_ERR_HIP";
    default: return "AGCN_ERR_UNKNOWN";
  }
}

const char* agcn_last_error(void) { return agcn::g_last_error.c_str(); }

static void plan_free(agcn_plan* p) {
  if (p == nullptr) return;
  std::vector<agcn::StreamEvent> pending;
  if (p->ready != nullptr) {
    if (p->ready_recorded) pending.push_back({p->ready, p->stream});
    else (void)hipEventDestroy(p->ready);
  }
  for (auto& u : p->uses) pending.push_back({u.second, u.first});
  // The plan's own stream gets no event: recording one queues a marker
  // packet, around which the GPU idles for microseconds between this plan's
  // work and the next call's. A later plan on that stream follows in stream
  // order; one on another stream, or a hipFree, synchronises the device.
  if (p->base != nullptr) pending.push_back({nullptr, p->stream});
  if (p->sync_on_release) {
    int prev = 0;
    if (agcn::with_device(p->device, &prev) == AGCN_OK) {
      (void)hipDeviceSynchronize();
      if (prev != p->device) (void)hipSetDevice(prev);
    }
  }
  agcn::device_release(p->device, p->base, p->bytes, std::move(pending));
  delete p;
}

void agcn_release_cached_memory(void) {
  std::map<int, agcn::CachedBlock> blocks;
  {
    std::lock_guard<std::mutex> lk(agcn::g_cache_mu);
    blocks.swap(agcn::g_cache);
  }
  for (auto& kv : blocks) {
    if (kv.second.ptr == nullptr && kv.second.pending.empty()) continue;
    int prev = 0;
    if (agcn::with_device(kv.first, &prev) != AGCN_OK) continue;
    agcn::free_block(kv.second);
    if (prev != kv.first) (void)hipSetDevice(prev);
  }
}

int agcn_plan_create(agcn_plan_t* out, int32_t n_rows, int32_t n_cols, int64_t nnz,
                     const int32_t* d_rowptr, const int32_t* d_colidx, const float* d_vals,
                     const agcn_plan_params* params, void* stream) {
  if (out == nullptr) return fail(AGCN_ERR_INVALID_ARGUMENT, "out is NULL");
  *out = nullptr;
  if (n_rows < 0 || n_cols < 0 || nnz < 0)
    return fail(AGCN_ERR_INVALID_ARGUMENT, "n_rows, n_cols and nnz must be >= 0");
  if (n_rows == 0 && nnz > 0)
    return fail(AGCN_ERR_INVALID_ARGUMENT, "nnz > 0 with no rows");
  if (nnz >= ((int64_t)1 << 31))
    return fail(AGCN_ERR_UNSUPPORTED, "nnz >= 2^31 does not fit the int32 metadata format");
  if (n_rows > 0 && d_rowptr == nullptr) return fail(AGCN_ERR_INVALID_ARGUMENT, "rowptr is NULL");
  if (nnz > 0 && (d_colidx == nullptr || d_vals == nullptr))
    return fail(AGCN_ERR_INVALID_ARGUMENT, "colidx or vals is NULL");
  agcn_plan_params prm;
  if (params == nullptr) agcn_default_params(&prm); else prm = *params;
  if (prm.flags != 0 && prm.flags != AGCN_PLAN_WARP_LEVEL && prm.flags != AGCN_PLAN_COLUMN_LOOP)
    return fail(AGCN_ERR_INVALID_ARGUMENT,
                "flags must be 0, AGCN_PLAN_WARP_LEVEL or AGCN_PLAN_COLUMN_LOOP");
  if (prm.max_block_waves < 1 || prm.max_block_waves > agcn::kMaxBlockWaves)
    return fail(AGCN_ERR_INVALID_ARGUMENT, "max_block_waves must be in [1, 32]");
  if (prm.max_wave_nzs < 1 ||
      (int64_t)prm.max_block_waves * prm.max_wave_nzs > agcn::kMaxEntryNnz)
    return fail(AGCN_ERR_INVALID_ARGUMENT, "need max_wave_nzs >= 1 and W * Z <= 4096");
  if (prm.hub_chunk_nnz < 0 || prm.hub_chunk_nnz > agcn::kMaxEntryNnz)
    return fail(AGCN_ERR_INVALID_ARGUMENT, "hub_chunk_nnz must be in [0, 4096]");
  const int32_t deg_bound = prm.max_block_waves * prm.max_wave_nzs;
  const int32_t H = prm.hub_chunk_nnz > 0 ? prm.hub_chunk_nnz : deg_bound;
  if (agcn::spmm_lds_bytes_max(prm.max_block_waves, std::max(deg_bound, H)) > 65536)
    return fail(AGCN_ERR_INVALID_ARGUMENT,
                "parameters need more than 64 KiB of LDS per workgroup (reduce W, Z or H)");
  if ((int64_t)n_rows + nnz / H + 1 >= INT32_MAX)
    return fail(AGCN_ERR_UNSUPPORTED, "too many metadata entries for int32 indexing");

  int dev = 0;
  hipError_t he = hipGetDevice(&dev);
  if (he != hipSuccess) return agcn::hip_fail(he, "hipGetDevice");

  agcn::test_alloc_reset();
  agcn_plan* p = new (std::nothrow) agcn_plan();
  if (p == nullptr) return fail(AGCN_ERR_OUT_OF_MEMORY, "host allocation failed");
  p->device = dev;
  p->n_rows = n_rows;
  p->n_cols = n_cols;
  p->nnz = nnz;
  p->W = prm.max_block_waves;
  p->Z = prm.max_wave_nzs;
  p->deg_bound = deg_bound;
  p->H = H;
  p->flags = prm.flags;
  int rc;
  try {
    // The readiness event is created now and recorded only when first needed
    // (an execute on another stream, an export), so no execute allocates it.
    he = hipEventCreateWithFlags(&p->ready, hipEventDisableTiming);
    if (he != hipSuccess) {
      p->ready = nullptr;
      rc = agcn::hip_fail(he, "hipEventCreate(plan ready)");
    } else {
      rc = agcn::build_plan(p, d_rowptr, d_colidx, d_vals, static_cast<hipStream_t>(stream));
    }
  } catch (const std::bad_alloc&) {
    rc = fail(AGCN_ERR_OUT_OF_MEMORY, "host allocation failed");
  } catch (...) {
    rc = fail(AGCN_ERR_HIP, "unexpected exception while building the plan");
  }
  if (rc != AGCN_OK) {
    // Let queued plan kernels finish before their memory is released.
    (void)hipStreamSynchronize(static_cast<hipStream_t>(stream));
    plan_free(p);
    return rc;
  }
  *out = p;
  return AGCN_OK;
}

int agcn_spmm_workspace_size(agcn_plan_t plan, int32_t F, size_t* bytes) {
  if (plan == nullptr || bytes == nullptr) return fail(AGCN_ERR_INVALID_ARGUMENT, "NULL argument");
  if (F < 1) return fail(AGCN_ERR_INVALID_ARGUMENT, "F must be >= 1");
  *bytes = std::max(agcn::chunk_workspace_bytes(plan, F), agcn::win_workspace_bytes(plan, F));
  return AGCN_OK;
}

}  // extern "C"

namespace {

int check_device(const agcn_plan* plan) {
  int dev = -1;
  hipError_t he = hipGetDevice(&dev);
  if (he != hipSuccess) return agcn::hip_fail(he, "hipGetDevice");
  if (dev != plan->device)
    return fail(AGCN_ERR_INVALID_ARGUMENT, "current device differs from the plan's device");
  return AGCN_OK;
}

// noalloc: the workspace is the library's fixed device array (d_ws unused),
// and the call creates no event either.
int spmm_checked(agcn_plan_t plan, int32_t F, const float* d_X, int64_t ldx, float* d_Y,
                 int64_t ldy, void* d_ws, void* stream, void* ev_begin, void* ev_mid,
                 void* ev_end, int32_t epilogue, bool noalloc = false) {
  if (plan == nullptr) return fail(AGCN_ERR_INVALID_ARGUMENT, "plan is NULL");
  if (epilogue != AGCN_EPILOGUE_NONE && epilogue != AGCN_EPILOGUE_RELU)
    return fail(AGCN_ERR_INVALID_ARGUMENT, "epilogue must be AGCN_EPILOGUE_NONE or AGCN_EPILOGUE_RELU");
  if (F < 1) return fail(AGCN_ERR_INVALID_ARGUMENT, "F must be >= 1");
  if (ldx < F || ldy < F) return fail(AGCN_ERR_INVALID_ARGUMENT, "ldx and ldy must be >= F");
  if (plan->n_rows > 0 && d_Y == nullptr) return fail(AGCN_ERR_INVALID_ARGUMENT, "Y is NULL");
  if (plan->nnz > 0 && d_X == nullptr) return fail(AGCN_ERR_INVALID_ARGUMENT, "X is NULL");
  size_t ws_need = 0;
  agcn_spmm_workspace_size(plan, F, &ws_need);
  if (noalloc) {
    // The hub windows only when their partials fit the fixed workspace; the
    // hub chunks need less.
    if (ws_need > agcn::kNoallocScratchBytes) ws_need = agcn::chunk_workspace_bytes(plan, F);
    if (ws_need > agcn::kNoallocScratchBytes)
      return fail(AGCN_ERR_UNSUPPORTED,
                  "agcn_spmm_noalloc: this plan needs " + std::to_string(ws_need) +
                      " bytes of workspace at F = " + std::to_string(F) + ", above the " +
                      std::to_string(agcn::kNoallocScratchBytes) +
                      "-byte fixed workspace (use agcn_spmm with a workspace)");
    d_ws = nullptr;
    if (ws_need > 0) {
      int dev = -1;
      hipError_t he = hipGetDevice(&dev);
      if (he != hipSuccess) return agcn::hip_fail(he, "hipGetDevice");
      float* scratch = nullptr;
      if (int rc = agcn::noalloc_scratch(dev, &scratch)) return rc;
      d_ws = scratch;
    }
  }
  if (ws_need > 0 && d_ws == nullptr)
    return fail(AGCN_ERR_INVALID_ARGUMENT, "this plan has hub rows: a workspace is required");
  size_t xb = 0, yb = 0;
  if (!agcn::span_bytes(d_X ? plan->n_cols : 0, ldx, F, &xb) ||
      !agcn::span_bytes(plan->n_rows, ldy, F, &yb))
    return fail(AGCN_ERR_INVALID_ARGUMENT, "matrix extent overflows");
  if (agcn::ranges_overlap(d_X, xb, d_Y, yb))
    return fail(AGCN_ERR_INVALID_ARGUMENT, "X and Y overlap");
  if (ws_need > 0 && (agcn::ranges_overlap(d_ws, ws_need, d_Y, yb) ||
                      agcn::ranges_overlap(d_ws, ws_need, d_X, xb)))
    return fail(AGCN_ERR_INVALID_ARGUMENT, "workspace overlaps X or Y");
  if (int rc = check_device(plan)) return rc;
  // The plan's last kernels may still run on its stream: order another
  // stream after them (on the plan's own stream they already come first).
  if (static_cast<hipStream_t>(stream) != plan->stream) {
    hipEvent_t ready = nullptr;
    if (int rc = agcn::plan_ready_event(plan, &ready)) return rc;
    const hipError_t e = hipStreamWaitEvent(static_cast<hipStream_t>(stream), ready, 0);
    if (e != hipSuccess) return agcn::hip_fail(e, "hipStreamWaitEvent(plan ready)");
  }
  const int rc = agcn::run_spmm(plan, F, d_X, ldx, d_Y, ldy, static_cast<float*>(d_ws), ws_need,
                                static_cast<hipStream_t>(stream), static_cast<hipEvent_t>(ev_begin),
                                static_cast<hipEvent_t>(ev_mid), static_cast<hipEvent_t>(ev_end),
                                epilogue);
  // Last use on a stream other than the plan's own (also after a failed
  // launch); uses on the plan's stream are covered at release.
  if (static_cast<hipStream_t>(stream) != plan->stream) {
    if (noalloc) agcn::note_use_noalloc(plan, static_cast<hipStream_t>(stream));
    else agcn::note_use(plan, static_cast<hipStream_t>(stream));
  }
  return rc;
}

// Bytes of the transformed features H (n_cols x fout floats) at the start of
// a layer workspace, rounded up so the SpMM workspace after it is aligned.
size_t layer_h_bytes(const agcn_plan* plan, int32_t fout) {
  const size_t b = (size_t)plan->n_cols * (size_t)fout * sizeof(float);
  return (b + 255) & ~(size_t)255;
}

int linear_checked(int64_t n, int32_t fin, int32_t fout, const float* d_X, int64_t ldx,
                   const float* d_W, int64_t ldw, float* d_H, int64_t ldh, void* stream) {
  if (n < 0 || fin < 0 || fout < 0)
    return fail(AGCN_ERR_INVALID_ARGUMENT, "n, fin and fout must be >= 0");
  if (ldx < fin || ldw < fout || ldh < fout)
    return fail(AGCN_ERR_INVALID_ARGUMENT, "ldx >= fin, ldw >= fout and ldh >= fout are required");
  if (n > 0 && fout > 0 && d_H == nullptr) return fail(AGCN_ERR_INVALID_ARGUMENT, "H is NULL");
  if (n > 0 && fin > 0 && d_X == nullptr) return fail(AGCN_ERR_INVALID_ARGUMENT, "X is NULL");
  if (fin > 0 && fout > 0 && d_W == nullptr) return fail(AGCN_ERR_INVALID_ARGUMENT, "W is NULL");
  size_t xb = 0, wb = 0, hb = 0;
  if (!agcn::span_bytes(n, ldx, fin, &xb) || !agcn::span_bytes(fin, ldw, fout, &wb) ||
      !agcn::span_bytes(n, ldh, fout, &hb))
    return fail(AGCN_ERR_INVALID_ARGUMENT, "matrix extent overflows");
  if (agcn::ranges_overlap(d_H, hb, d_X, xb) || agcn::ranges_overlap(d_H, hb, d_W, wb))
    return fail(AGCN_ERR_INVALID_ARGUMENT, "H overlaps X or W");
  return agcn::run_linear(n, fin, fout, d_X, ldx, d_W, ldw, d_H, ldh,
                          static_cast<hipStream_t>(stream));
}

}  // namespace

extern "C" {

int agcn_spmm_timed(agcn_plan_t plan, int32_t F, const float* d_X, int64_t ldx, float* d_Y,
                    int64_t ldy, void* d_ws, void* stream, void* ev_begin, void* ev_mid,
                    void* ev_end) {
  return spmm_checked(plan, F, d_X, ldx, d_Y, ldy, d_ws, stream, ev_begin, ev_mid, ev_end,
                      AGCN_EPILOGUE_NONE);
}

int agcn_spmm(agcn_plan_t plan, int32_t F, const float* d_X, int64_t ldx, float* d_Y,
              int64_t ldy, void* d_ws, void* stream) {
  return spmm_checked(plan, F, d_X, ldx, d_Y, ldy, d_ws, stream, nullptr, nullptr, nullptr,
                      AGCN_EPILOGUE_NONE);
}

int agcn_spmm_ex(agcn_plan_t plan, int32_t F, const float* d_X, int64_t ldx, float* d_Y,
                 int64_t ldy, void* d_ws, void* stream, int32_t epilogue) {
  return spmm_checked(plan, F, d_X, ldx, d_Y, ldy, d_ws, stream, nullptr, nullptr, nullptr,
                      epilogue);
}

int agcn_spmm_noalloc(agcn_plan_t plan, int32_t F, const float* d_X, int64_t ldx, float* d_Y,
                      int64_t ldy, void* stream, int32_t epilogue) {
  return spmm_checked(plan, F, d_X, ldx, d_Y, ldy, nullptr, stream, nullptr, nullptr, nullptr,
                      epilogue, /*noalloc=*/true);
}

int agcn_linear(int64_t n, int32_t fin, int32_t fout, const float* d_X, int64_t ldx,
                const float* d_W, int64_t ldw, float* d_H, int64_t ldh, void* stream) {
  return linear_checked(n, fin, fout, d_X, ldx, d_W, ldw, d_H, ldh, stream);
}

int agcn_gcn_workspace_size(agcn_plan_t plan, int32_t fout, size_t* bytes) {
  if (plan == nullptr || bytes == nullptr) return fail(AGCN_ERR_INVALID_ARGUMENT, "NULL argument");
  if (fout < 1) return fail(AGCN_ERR_INVALID_ARGUMENT, "fout must be >= 1");
  size_t spmm_ws = 0;
  if (int rc = agcn_spmm_workspace_size(plan, fout, &spmm_ws)) return rc;
  *bytes = layer_h_bytes(plan, fout) + spmm_ws;
  return AGCN_OK;
}

int agcn_gcn_layer(agcn_plan_t plan, int32_t fin, int32_t fout, const float* d_X, int64_t ldx,
                   const float* d_W, int64_t ldw, float* d_Y, int64_t ldy, void* d_ws,
                   void* stream, int32_t epilogue) {
  if (plan == nullptr) return fail(AGCN_ERR_INVALID_ARGUMENT, "plan is NULL");
  if (fin < 0 || fout < 1) return fail(AGCN_ERR_INVALID_ARGUMENT, "fin >= 0 and fout >= 1 are required");
  if (epilogue != AGCN_EPILOGUE_NONE && epilogue != AGCN_EPILOGUE_RELU)
    return fail(AGCN_ERR_INVALID_ARGUMENT, "epilogue must be AGCN_EPILOGUE_NONE or AGCN_EPILOGUE_RELU");
  size_t need = 0;
  agcn_gcn_workspace_size(plan, fout, &need);
  const size_t hbytes = layer_h_bytes(plan, fout);
  if (plan->n_cols > 0 && d_ws == nullptr)
    return fail(AGCN_ERR_INVALID_ARGUMENT, "a workspace of agcn_gcn_workspace_size bytes is required");
  if (d_ws != nullptr && !agcn::aligned16(d_ws))
    return fail(AGCN_ERR_INVALID_ARGUMENT, "the workspace must be 16-byte aligned");
  size_t xb = 0, yb = 0;
  if (!agcn::span_bytes(plan->n_cols, ldx, fin, &xb) || !agcn::span_bytes(plan->n_rows, ldy, fout, &yb))
    return fail(AGCN_ERR_INVALID_ARGUMENT, "matrix extent overflows");
  size_t wb = 0;
  if (!agcn::span_bytes(fin, ldw, fout, &wb))
    return fail(AGCN_ERR_INVALID_ARGUMENT, "matrix extent overflows");
  if (agcn::ranges_overlap(d_ws, need, d_X, xb) || agcn::ranges_overlap(d_ws, need, d_Y, yb) ||
      agcn::ranges_overlap(d_ws, need, d_W, wb))
    return fail(AGCN_ERR_INVALID_ARGUMENT, "workspace overlaps X, W or Y");
  if (agcn::ranges_overlap(d_Y, yb, d_X, xb) || agcn::ranges_overlap(d_Y, yb, d_W, wb))
    return fail(AGCN_ERR_INVALID_ARGUMENT, "Y overlaps X or W");
  if (int rc = check_device(plan)) return rc;
  float* H = static_cast<float*>(d_ws);
  if (int rc = linear_checked(plan->n_cols, fin, fout, d_X, ldx, d_W, ldw, H, fout, stream))
    return rc;
  void* spmm_ws = need > hbytes ? static_cast<char*>(d_ws) + hbytes : nullptr;
  return spmm_checked(plan, fout, H, fout, d_Y, ldy, spmm_ws, stream, nullptr, nullptr, nullptr,
                      epilogue);
}

int agcn_plan_info(agcn_plan_t plan, agcn_plan_stats* s) {
  if (plan == nullptr || s == nullptr) return fail(AGCN_ERR_INVALID_ARGUMENT, "NULL argument");
  std::memset(s, 0, sizeof(*s));
  s->n_rows = plan->n_rows;
  s->n_cols = plan->n_cols;
  s->nnz = plan->nnz;
  s->n_entries = plan->n_entries;
  s->hub_first_entry = plan->hub_first_entry;
  s->n_hub_chunks = plan->n_hub_rows > 0 ? plan->n_entries - plan->hub_first_entry : 0;
  s->n_hub_rows = plan->n_hub_rows;
  s->hub_first_row = plan->hub_first_row;
  s->deg_bound = plan->deg_bound;
  s->hub_chunk_nnz = plan->H;
  s->max_deg = plan->max_deg;
  s->max_block_waves = plan->W;
  s->max_wave_nzs = plan->Z;
  s->flags = plan->flags;
  s->device_bytes = plan->bytes;
  s->hub_windows = plan->n_win;
  return AGCN_OK;
}

int agcn_plan_export(agcn_plan_t plan, int32_t* h_perm, int32_t* h_rowptr_s, int32_t* h_colidx_s,
                     float* h_vals_s, int32_t* h_meta) {
  if (plan == nullptr) return fail(AGCN_ERR_INVALID_ARGUMENT, "plan is NULL");
  struct Item {
    void* dst;
    const void* src;
    size_t bytes;
  } items[] = {
      {h_perm, plan->perm, (size_t)plan->n_rows * 4},
      {h_rowptr_s, plan->rowptr_s, ((size_t)plan->n_rows + 1) * 4},
      {h_colidx_s, plan->colidx_s, (size_t)plan->nnz * 4},
      {h_vals_s, plan->vals_s, (size_t)plan->nnz * 4},
      {h_meta, plan->meta, (size_t)plan->n_entries * 16},
  };
  int dev = -1;
  hipError_t he = hipGetDevice(&dev);
  if (he != hipSuccess) return agcn::hip_fail(he, "hipGetDevice");
  if (dev != plan->device)
    return fail(AGCN_ERR_INVALID_ARGUMENT, "current device differs from the plan's device");
  // The plan's last kernels may still run on its stream, which the copies
  // below (on the null stream) need not wait for.
  hipEvent_t ready = nullptr;
  if (int rc = agcn::plan_ready_event(plan, &ready)) return rc;
  if ((he = hipEventSynchronize(ready)) != hipSuccess)
    return agcn::hip_fail(he, "hipEventSynchronize(plan ready)");
  // The short sort's last relayout runs after agcn_plan_create returned; its
  // window check (never raised for a sorted row order) is reported here.
  if (plan->err_word != nullptr) {
    uint32_t e = 0;
    if ((he = hipMemcpy(&e, plan->err_word, sizeof(e), hipMemcpyDeviceToHost)) != hipSuccess)
      return agcn::hip_fail(he, "hipMemcpy(export error word)");
    if (e & agcn::kErrRelayout) return fail(AGCN_ERR_HIP, "internal plan consistency check failed");
  }
  for (const Item& it : items) {
    if (it.dst == nullptr || it.bytes == 0) continue;
    he = hipMemcpy(it.dst, it.src, it.bytes, hipMemcpyDeviceToHost);
    if (he != hipSuccess) return agcn::hip_fail(he, "hipMemcpy(export)");
  }
  return AGCN_OK;
}

void agcn_plan_destroy(agcn_plan_t plan) { plan_free(plan); }

}  // extern "C"
