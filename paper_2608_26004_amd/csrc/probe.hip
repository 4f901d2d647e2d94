// Read-ceiling probe: a plain read-reduce kernel over one device buffer.
//
// It streams the buffer once with 16-byte non-temporal loads (the load width
// and cache policy of the decision kernel's logit streams), folds every word
// into a per-workgroup XOR so that no load can be dropped, and writes one
// word per workgroup.  The rate it reaches over a buffer far larger than the
// caches is the practical HBM read ceiling of the part, which the decision
// kernel's achieved rate is set against next to the 8 TB/s specification.
//
// Not part of the decision step; built as its own library.

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "asymspec_probe.h"

namespace {

typedef uint32_t v4u __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int kUnroll = 8;   // 16-byte vectors in flight per thread

__global__ __launch_bounds__(kThreads) void read_reduce_kernel(const v4u* src, long long nvec,
                                                               uint32_t* out) {
  const long long step = (long long)gridDim.x * kThreads * kUnroll;
  uint32_t acc = 0u;
  for (long long base = (long long)blockIdx.x * kThreads * kUnroll + threadIdx.x; base < nvec;
       base += step) {
    v4u v[kUnroll];
#pragma unroll
    for (int k = 0; k < kUnroll; ++k) {
      const long long i = base + (long long)k * kThreads;
      v[k] = i < nvec ? __builtin_nontemporal_load(src + i) : v4u{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int k = 0; k < kUnroll; ++k) acc ^= v[k].x ^ v[k].y ^ v[k].z ^ v[k].w;
  }
  // workgroup XOR: within each wave by shuffles, then across the 4 waves
  for (int off = 32; off > 0; off >>= 1) acc ^= (uint32_t)__shfl_xor((int)acc, off, 64);
  __shared__ uint32_t part[kThreads / 64];
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t r = 0u;
#pragma unroll
    for (int w = 0; w < kThreads / 64; ++w) r ^= part[w];
    out[blockIdx.x] = r;
  }
}

// Core-clock probe: the first lane of each workgroup spins on the 100 MHz
// real-time counter for `ticks` ticks and records how far the shader-clock
// counter (s_memtime) advanced meanwhile; the ratio of the two, times
// 100 MHz, is the clock the workgroup's compute unit ran at.  The loop ends
// once the real-time counter has moved `ticks` (bounded on the host).
__global__ __launch_bounds__(64) void clock_kernel(uint32_t ticks, uint32_t* out) {
  if (threadIdx.x != 0) return;
  const uint64_t r0 = __builtin_amdgcn_s_memrealtime();
  const uint64_t c0 = __builtin_amdgcn_s_memtime();
  uint64_t r1 = r0;
  while (r1 - r0 < (uint64_t)ticks) {
    __builtin_amdgcn_s_sleep(1);
    r1 = __builtin_amdgcn_s_memrealtime();
  }
  const uint64_t c1 = __builtin_amdgcn_s_memtime();
  out[2 * blockIdx.x] = (uint32_t)(c1 - c0);
  out[2 * blockIdx.x + 1] = (uint32_t)(r1 - r0);
}

}  // namespace

extern "C" {

int asymspec_probe_clock(uint32_t* out, int nblocks, uint32_t ticks, void* stream) {
  if (out == nullptr || (reinterpret_cast<uintptr_t>(out) & 3u) != 0u) return ASYMSPEC_PROBE_E_ARG;
  if (nblocks < 1 || nblocks > ASYMSPEC_PROBE_MAX_CLOCK_BLOCKS) return ASYMSPEC_PROBE_E_ARG;
  if (ticks < 1u || ticks > ASYMSPEC_PROBE_MAX_CLOCK_TICKS) return ASYMSPEC_PROBE_E_ARG;
  hipLaunchKernelGGL(clock_kernel, dim3((unsigned)nblocks), dim3(64), 0,
                     reinterpret_cast<hipStream_t>(stream), ticks, out);
  return hipGetLastError() == hipSuccess ? 0 : ASYMSPEC_PROBE_E_DEVICE;
}

int asymspec_probe_read(const void* src, size_t nbytes, uint32_t* out, int nblocks, void* stream) {
  if (src == nullptr || out == nullptr) return ASYMSPEC_PROBE_E_ARG;
  if (nbytes == 0 || nbytes % 16 != 0 || nbytes > ((size_t)1 << 40)) return ASYMSPEC_PROBE_E_ARG;
  if (nblocks < 1 || nblocks > ASYMSPEC_PROBE_MAX_BLOCKS) return ASYMSPEC_PROBE_E_ARG;
  if ((reinterpret_cast<uintptr_t>(src) & 15u) != 0u || (reinterpret_cast<uintptr_t>(out) & 3u) != 0u)
    return ASYMSPEC_PROBE_E_ARG;
  hipLaunchKernelGGL(read_reduce_kernel, dim3((unsigned)nblocks), dim3(kThreads), 0,
                     reinterpret_cast<hipStream_t>(stream), reinterpret_cast<const v4u*>(src),
                     (long long)(nbytes / 16), out);
  return hipGetLastError() == hipSuccess ? 0 : ASYMSPEC_PROBE_E_DEVICE;
}

}  // extern "C"
