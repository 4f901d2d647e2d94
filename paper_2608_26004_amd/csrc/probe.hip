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

}  // namespace

extern "C" {

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
