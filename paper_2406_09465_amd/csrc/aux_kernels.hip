// Helper kernels of the profiler (a cache-flushing write and a seeded fill),
// and the static device scratch of allocation-free plan execution.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <mutex>

namespace {

// Streams `n` 16-byte words into `p`, evicting L2 and the Infinity Cache
// (and leaving them full of dirty lines of `p`).
__global__ void flush_kernel(uint4* __restrict__ p, size_t n, uint32_t v) {
  size_t stride = (size_t)gridDim.x * blockDim.x;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) p[i] = make_uint4(v, i, v, i);
}

// Reads `n` 16-byte words of `p`, evicting L2 and the Infinity Cache (whose
// dirty lines are written back during this kernel) and leaving them full of
// clean lines.  The loaded words are folded into one value that is stored
// (into p[0]) only when it equals an arbitrary constant, so the loads stay live.
__global__ void read_flush_kernel(uint4* __restrict__ p, size_t n) {
  size_t stride = (size_t)gridDim.x * blockDim.x;
  uint32_t a = 0;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
    const uint4 v = p[i];
    a ^= v.x ^ v.y ^ v.z ^ v.w;
  }
  if (a == 0x9e3779b9u) p[0] = make_uint4(a, a, a, a);
}

__device__ __forceinline__ uint64_t splitmix64(uint64_t x) {
  x += 0x9E3779B97F4A7C15ULL;
  x = (x ^ (x >> 30)) * 0xBF58476D1CE4E5B9ULL;
  x = (x ^ (x >> 27)) * 0x94D049BB133111EBULL;
  return x ^ (x >> 31);
}

// Element i = 0.5 + u_i, u_i uniform in [0, 1) from a counter-based hash of (seed, i).
__global__ void fill_kernel(void* __restrict__ p, size_t n, int dtype, uint64_t seed) {
  size_t stride = (size_t)gridDim.x * blockDim.x;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
    uint64_t h = splitmix64(seed * 0x100000001B3ULL + i);
    float u = 0.5f + (float)(h >> 40) * (1.0f / 16777216.0f);
    if (dtype == 0)
      ((float*)p)[i] = u;
    else if (dtype == 1)
      ((_Float16*)p)[i] = (_Float16)u;
    else
      ((__bf16*)p)[i] = (__bf16)u;
  }
}

// Reads `n` 16-byte words of `p` (bringing them into L2 and the Infinity
// Cache, as a producing kernel leaves its output) without changing them; each
// workgroup stores the XOR of what it read in sink[blockIdx.x], so the loads
// are not dead.
__global__ void touch_kernel(const uint4* __restrict__ p, size_t n, uint4* __restrict__ sink) {
  __shared__ uint32_t red[256];
  size_t stride = (size_t)gridDim.x * blockDim.x;
  uint32_t acc = 0;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
    uint4 v = p[i];
    acc ^= v.x ^ v.y ^ v.z ^ v.w;
  }
  red[threadIdx.x] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t a = 0;
    for (int t = 0; t < (int)blockDim.x; ++t) a ^= red[t];
    sink[blockIdx.x] = make_uint4(a, 0, 0, 0);
  }
}

// Zeroes `n` 16-byte words (clears counters without a memset node, so a
// caller may capture the launch in a graph).
__global__ void zero_kernel(uint4* __restrict__ p, size_t n) {
  size_t stride = (size_t)gridDim.x * blockDim.x;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) p[i] = make_uint4(0, 0, 0, 0);
}

// Device memory of korch_plan_execute_noalloc: hand-off counters in the first
// kStaticCounterBytes, the plan's workspace after them.  One copy per device,
// held until the process ends.  Host code never passes this name to a kernel
// (on the host it is only a stand-in); it uses the per-device address that
// hipGetSymbolAddress returns.
constexpr size_t kStaticScratchBytes = (size_t)32 << 20;
constexpr int kMaxDevices = 64;
static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

std::mutex g_scratch_mu;
void* g_scratch_addr[kMaxDevices];

}  // namespace

namespace korch {

size_t static_scratch_bytes() { return kStaticScratchBytes; }

// Set-up, once per device, with that device current: looks up and keeps this
// device's address of the static scratch.
hipError_t static_scratch_setup(int dev) {
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (g_scratch_addr[dev]) return hipSuccess;
  void* q = nullptr;
  hipError_t e = hipGetSymbolAddress(&q, HIP_SYMBOL(scratch));
  if (e != hipSuccess) return e;
  if (!q) return hipErrorInvalidSymbol;
  g_scratch_addr[dev] = q;
  return hipSuccess;
}

// The address kept by static_scratch_setup for `dev`, or NULL before it.
void* static_scratch_address(int dev) {
  if (dev < 0 || dev >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  return g_scratch_addr[dev];
}

hipError_t launch_zero(void* p, size_t bytes, hipStream_t s) {
  size_t n = bytes / 16;
  if (n == 0) return hipSuccess;
  size_t blocks = (n + 255) / 256;
  if (blocks > 1024) blocks = 1024;
  hipLaunchKernelGGL(zero_kernel, dim3((unsigned)blocks), dim3(256), 0, s, (uint4*)p, n);
  return hipGetLastError();
}

// Evicts L2 and the Infinity Cache through `bytes` of the device buffer `p`:
// a read of it (write = 0), after which the caches hold clean lines, or a write.
hipError_t launch_flush(void* p, size_t bytes, int write, hipStream_t s) {
  size_t n = bytes / 16;
  if (n == 0) return hipSuccess;
  if (write)
    hipLaunchKernelGGL(flush_kernel, dim3(4096), dim3(256), 0, s, (uint4*)p, n, 0x5a5a5a5au);
  else
    hipLaunchKernelGGL(read_flush_kernel, dim3(4096), dim3(256), 0, s, (uint4*)p, n);
  return hipGetLastError();
}

// `sink` holds kTouchBlocks 16-byte words.
constexpr unsigned kTouchBlocks = 1024;
size_t touch_sink_bytes() { return (size_t)kTouchBlocks * 16; }

hipError_t launch_touch(const void* p, size_t bytes, void* sink, hipStream_t s) {
  size_t n = bytes / 16;
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(touch_kernel, dim3(kTouchBlocks), dim3(256), 0, s, (const uint4*)p, n, (uint4*)sink);
  return hipGetLastError();
}

hipError_t launch_fill(void* p, size_t n, int dtype, uint64_t seed, hipStream_t s) {
  if (n == 0) return hipSuccess;
  size_t blocks = (n + 255) / 256;
  if (blocks > 8192) blocks = 8192;
  hipLaunchKernelGGL(fill_kernel, dim3((unsigned)blocks), dim3(256), 0, s, p, n, dtype, seed);
  return hipGetLastError();
}

}  // namespace korch
