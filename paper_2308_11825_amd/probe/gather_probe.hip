// Memory-ceiling probe for the aggregation's access pattern on one GPU.
//
// The aggregation SpMM gathers one 128-byte piece of an X row per nonzero at
// effectively random row addresses; this probe measures how fast the device
// serves exactly that, with no sparse-matrix work around it:
//   gather<C>  lanes in groups of C / 16, each group loading one C-byte chunk
//              (16 bytes per lane) at a pseudo-random chunk-aligned address in
//              a buffer of the given size, 8 loads in flight per lane;
//   seq        every lane streaming consecutive 16-byte words through the
//              same buffer (the sequential-read reference);
//   lds        groups of 8 lanes reading a random 128-byte row of a 128 KiB
//              LDS table.
// The buffer sizes cover the L2 of one XCD (4 MB), the Infinity Cache
// (256 MB) and HBM. Random addresses come from a counter hash, so no index
// traffic is added. Output: one JSON object per line.
//
// Build: python -m paper_2308_11825_amd.build (writes probe/gather_probe).
#include <hip/hip_runtime.h>

#include <cstdio>
#include <cstdlib>

namespace {

typedef float f4 __attribute__((ext_vector_type(4)));

#define CHECK(x)                                                                         \
  do {                                                                                   \
    hipError_t e_ = (x);                                                                 \
    if (e_ != hipSuccess) {                                                              \
      std::fprintf(stderr, "gather_probe: %s at line %d\n", hipGetErrorString(e_), __LINE__); \
      std::exit(1);                                                                      \
    }                                                                                    \
  } while (0)

__device__ inline uint32_t mix32(uint32_t x) {  // integer finaliser (xorshift-multiply)
  x ^= x >> 16;
  x *= 0x7feb352dU;
  x ^= x >> 15;
  x *= 0x846ca68bU;
  x ^= x >> 16;
  return x;
}

constexpr int kInFlight = 8;
constexpr int kIters = 64;

// chunk_mask + 1 chunks of LPC * 16 bytes; lane group g, iteration i loads
// chunk mix32(g, i) & chunk_mask. Every index is < (chunk_mask + 1) * LPC.
template <int LPC>
__global__ __launch_bounds__(256) void k_gather(const f4* __restrict__ buf, uint32_t chunk_mask,
                                                f4* __restrict__ out) {
  const uint32_t t = blockIdx.x * blockDim.x + threadIdx.x;
  const uint32_t grp = t / LPC, lane = t % LPC;
  f4 acc = f4(0.0f);
  for (int it = 0; it < kIters; it += kInFlight) {
    f4 x[kInFlight];
#pragma unroll
    for (int u = 0; u < kInFlight; ++u) {
      const uint32_t c = mix32(grp * 0x9E3779B9U + (uint32_t)(it + u) * 0x85EBCA6BU) & chunk_mask;
      x[u] = buf[(size_t)c * LPC + lane];
    }
#pragma unroll
    for (int u = 0; u < kInFlight; ++u) acc += x[u];
  }
  out[t] = acc;
}

__global__ __launch_bounds__(256) void k_seq(const f4* __restrict__ buf, uint32_t word_mask,
                                             f4* __restrict__ out) {
  const uint32_t t = blockIdx.x * blockDim.x + threadIdx.x;
  const uint32_t nt = gridDim.x * blockDim.x;
  f4 acc = f4(0.0f);
  for (int it = 0; it < kIters; it += kInFlight) {
    f4 x[kInFlight];
#pragma unroll
    for (int u = 0; u < kInFlight; ++u) x[u] = buf[(t + (uint32_t)(it + u) * nt) & word_mask];
#pragma unroll
    for (int u = 0; u < kInFlight; ++u) acc += x[u];
  }
  out[t] = acc;
}

constexpr int kLdsRows = 1024;  // 1024 rows x 128 bytes = 128 KiB

__global__ __launch_bounds__(1024) void k_lds(const f4* __restrict__ buf, int iters,
                                              f4* __restrict__ out) {
  __shared__ f4 s[kLdsRows * 8];
  for (int i = threadIdx.x; i < kLdsRows * 8; i += blockDim.x) s[i] = buf[i];
  __syncthreads();
  const uint32_t t = blockIdx.x * blockDim.x + threadIdx.x;
  const uint32_t grp = t / 8, lane = t % 8;
  f4 acc = f4(0.0f);
  for (int it = 0; it < iters; it += kInFlight) {
    f4 x[kInFlight];
#pragma unroll
    for (int u = 0; u < kInFlight; ++u) {
      const uint32_t r = mix32(grp * 0x9E3779B9U + (uint32_t)(it + u) * 0x85EBCA6BU) & (kLdsRows - 1);
      x[u] = s[r * 8 + lane];
    }
#pragma unroll
    for (int u = 0; u < kInFlight; ++u) acc += x[u];
  }
  out[t] = acc;
}

}  // namespace

int main() {
  const size_t max_bytes = (size_t)2 << 30;
  const int blocks = 8192, threads = 256;  // 2M lanes, 32 workgroups per CU
  f4 *buf = nullptr, *out = nullptr;
  CHECK(hipMalloc(&buf, max_bytes));
  CHECK(hipMemset(buf, 0, max_bytes));
  CHECK(hipMalloc(&out, (size_t)blocks * threads * sizeof(f4)));
  hipEvent_t e0, e1;
  CHECK(hipEventCreate(&e0));
  CHECK(hipEventCreate(&e1));
  const int reps = 5;
  auto run = [&](const char* kind, int chunk, size_t ws, double bytes, auto launch) {
    launch();
    CHECK(hipGetLastError());
    CHECK(hipDeviceSynchronize());
    CHECK(hipEventRecord(e0));
    for (int r = 0; r < reps; ++r) launch();
    CHECK(hipEventRecord(e1));
    CHECK(hipEventSynchronize(e1));
    float ms = 0;
    CHECK(hipEventElapsedTime(&ms, e0, e1));
    const double t = ms / reps;
    std::printf("{\"kind\": \"%s\", \"chunk_bytes\": %d, \"working_set_MiB\": %zu, \"ms\": %.4f, "
                "\"TBps\": %.3f}\n", kind, chunk, ws >> 20, t, bytes / (t * 1e-3) / 1e12);
    std::fflush(stdout);
  };
  const double lanes_bytes = (double)blocks * threads * kIters * 16;
  for (int sh = 21; sh <= 31; ++sh) {
    const size_t ws = (size_t)1 << sh;
    run("gather", 128, ws, lanes_bytes,
        [&] { k_gather<8><<<blocks, threads>>>(buf, (uint32_t)(ws / 128 - 1), out); });
    run("gather", 64, ws, lanes_bytes,
        [&] { k_gather<4><<<blocks, threads>>>(buf, (uint32_t)(ws / 64 - 1), out); });
    run("gather", 256, ws, lanes_bytes,
        [&] { k_gather<16><<<blocks, threads>>>(buf, (uint32_t)(ws / 256 - 1), out); });
    run("seq", 16, ws, lanes_bytes,
        [&] { k_seq<<<blocks, threads>>>(buf, (uint32_t)(ws / 16 - 1), out); });
  }
  const int lds_iters = 256;
  run("lds", 128, 0, (double)1024 * 1024 * lds_iters * 16,
      [&] { k_lds<<<1024, 1024>>>(buf, lds_iters, out); });
  CHECK(hipFree(buf));
  CHECK(hipFree(out));
  return 0;
}
