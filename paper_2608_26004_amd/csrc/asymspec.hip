// AsymSpec fused decision step for MI355X (gfx950, CDNA4, wave64).
//
// One persistent launch does the whole step of Alg. 1 for every
// request: the vocabulary-wide statistics of the verifier logits t and the
// drafter logits a (full view) and b (compressed view), the delta-fused logits
// f = t + beta (a - b) (Sec. 3.2, Eq. 1-2), the Jensen-Shannon divergence D and
// the CDA gate gamma * exp(-D) (Sec. 3.3, Eq. 3), the acceptance test (Eq. 4,
// or its speculative-sampling form for temperature > 0), and the emission at
// the first rejection or the bonus token.
//
// The launch is a work queue (schedule.h): workgroups take items in order
// from an atomic counter.  Statistics items (stats.h) stream every logit
// once from HBM and never wait; per request, a decide, S pass-2 and a pick
// item (resolve.h) follow a few requests behind and re-read only the rows
// whose outcome needs a second pass, while those rows are still in the
// memory-side cache.
//
// Cross-workgroup records are arrays of 64-bit slots whose high word is the
// launch epoch and low word a payload, written and read with relaxed
// agent-scope atomics (no cache flushes).  An aligned 64-bit access is
// single-copy atomic, so a reader that sees the epoch in a slot sees its
// payload; writers never wait, readers poll until every slot they need is
// in.  The workspace therefore needs no initialisation.

#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <chrono>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <mutex>
#include <unistd.h>

#include "asymspec.h"
#include "device.h"
#include "resolve.h"
#include "schedule.h"
#include "stats.h"

namespace asym {

// Work queues: kQueues counters, each in its own 128-byte line, and an
// arrival counter.  A workgroup serves queue (arrival order) % nq, whose
// items are the global indices q, q + nq, ... in increasing order.  Every
// queue is thus served by a running workgroup and hands out its items in
// list order, so the lowest unfinished item can always run, whether or not
// the whole grid is resident.  A counter holds (epoch, count); the first
// workgroup of a launch to touch it raises it to (epoch, 0) with one atomic
// max (epochs grow within a process), and values are then taken with
// fetch-add.
constexpr int kQueues = 8;
constexpr int kQueueStride = 16;   // 64-bit words between counters (arrival counter last)

DEV void queue_init(const KArgs& A, uint64_t* ctr) {
  const uint64_t want = (uint64_t)A.epoch << 32;
  const uint64_t old = __hip_atomic_fetch_max(ctr, want, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  if ((uint32_t)(old >> 32) <= A.epoch) return;
  // a counter left by a later epoch (another library instance on this
  // workspace): replace it by compare-and-swap
  uint64_t v = old;
  Poll pl;
  while (!tag_ok(v, A.epoch)) {
    uint64_t expect = v;
    if (__hip_atomic_compare_exchange_strong(ctr, &expect, want, __ATOMIC_RELAXED, __ATOMIC_RELAXED,
                                             __HIP_MEMORY_SCOPE_AGENT))
      break;
    v = expect;
    if (!pl.again(A)) break;
  }
}
DEV uint32_t take(uint64_t* ctr) {
  return (uint32_t)__hip_atomic_fetch_add(ctr, (uint64_t)1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
DEV uint32_t grab(uint64_t* ctr, int nq, int q) { return take(ctr) * (uint32_t)nq + (uint32_t)q; }

template <int DT, bool kB1>
DEV void stats_dispatch(const KArgs& A, int req, int sub, Smem& sm) {
  const int i = sub / A.S, m = sub - (sub / A.S) * A.S;
  const int row = req * (A.K + 1) + i;
  const float tau = sload_f32(A.tau, req);
  if (i == A.K) {
    if (tau > 0.0f) stats_item<DT, kSampleBonus, kB1>(A, row, m, sm);
    else stats_item<DT, kGreedyBonus, kB1>(A, row, m, sm);
  } else if (!(tau > 0.0f)) {
    stats_item<DT, kGreedyDraft, kB1>(A, row, m, sm);
  } else if (tau == 1.0f) {
    stats_item<DT, kSampleDraft1, kB1>(A, row, m, sm);
  } else {
    stats_item<DT, kSampleDraftT, kB1>(A, row, m, sm);
  }
}

#ifndef ASYMSPEC_WAVES
#define ASYMSPEC_WAVES 4
#endif

template <int DT, bool kB1>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(ASYMSPEC_WAVES)))
void fuse_verify_kernel(KArgs A) {
  __shared__ Smem sm;
  const int tid = threadIdx.x;
  const int nq = min((int)gridDim.x, kQueues);
  if (tid == 0) {
    uint64_t* arrive = A.qctr + (size_t)kQueues * kQueueStride;
    queue_init(A, arrive);
    const int q = (int)(take(arrive) % (uint32_t)nq);
    uint64_t* c = A.qctr + (size_t)q * kQueueStride;
    queue_init(A, c);
    sm.next[0] = (int)grab(c, nq, q);
    sm.queue = q;
  }
  __syncthreads();
  const int q = sm.queue;
  uint64_t* ctr = A.qctr + (size_t)q * kQueueStride;
  uint32_t cur = (uint32_t)sm.next[0];
  int par = 1;
  while (cur < (uint32_t)A.sc.total) {
    uint32_t nx = 0;
    if (tid == 0) nx = grab(ctr, nq, q);   // in flight while this item runs
    // The arguments are re-read in every iteration through an opaque copy of
    // the kernarg-segment pointer (scalar loads), so that no item's address
    // arithmetic is hoisted out of the loop and kept live across the others.
    auto kp = (const __attribute__((address_space(4))) KArgs*)__builtin_amdgcn_kernarg_segment_ptr();
    asm volatile("" : "+s"(kp));
    const KArgs& B = *(const KArgs*)kp;
    const Item it = sched_item(B.sc, B.K, B.S, (int)cur);
    switch (it.type) {
      case kItemStats: stats_dispatch<DT, kB1>(B, it.req, it.sub, sm); break;
      case kItemDecide: decide_item<DT>(B, it.req, sm); break;
      case kItemPass2: pass2_item<DT>(B, it.req, it.sub, sm); break;
      case kItemPick: pick_item<DT>(B, it.req, sm); break;
      default: break;
    }
    if (tid == 0) sm.next[par] = (int)nx;
    __syncthreads();
    cur = (uint32_t)sm.next[par];
    par ^= 1;
  }
}

__global__ void fill_zero_kernel(uint32_t* p, size_t n) {
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
    p[i] = 0u;
}

// ---------------------------------------------------------------- host side
struct Layout {
  int S, VE;
  size_t rows;
  size_t off_rec1, off_dec, off_rec2, off_q, off_err, total;
};

static size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

static bool make_layout(int B, int K, int V, int dtype, Layout& L) {
  if (B < 1 || K < 0 || K > kMaxK || V < 1) return false;
  if (dtype != ASYMSPEC_BF16 && dtype != ASYMSPEC_FP32) return false;
  const long double elems = (long double)B * (K + 1) * V;
  if (elems >= (long double)(1ull << 40)) return false;
  L.VE = dtype == ASYMSPEC_BF16 ? 8 : 4;
  // a row spans at most this many 16-byte vectors (it may start mid-vector)
  const long long nvec_max = ((long long)V + 2LL * L.VE - 2) / L.VE;
  const long long S = (nvec_max + kChunkVec - 1) / kChunkVec;
  if (S > (1 << 20)) return false;
  L.S = (int)S;
  L.rows = (size_t)B * (K + 1);
  size_t off = 0;
  L.off_rec1 = off; off = align_up(off + L.rows * L.S * kR1 * 8, 256);
  L.off_dec = off;  off = align_up(off + (size_t)B * (kDecHdr + (size_t)(K + 1) * kDecRow) * 8, 256);
  L.off_rec2 = off; off = align_up(off + L.rows * L.S * kR2 * 8, 256);
  L.off_q = off;    off = align_up(off + (size_t)(kQueues + 1) * kQueueStride * 8, 256);
  L.off_err = off;  off = align_up(off + 8, 256);
  L.total = off;
  return true;
}

struct DevInfo {
  int ok = 0;
  int n_cu = 0;
  int max_blocks[2] = {0, 0};   // co-resident workgroups, per dtype
};

static DevInfo g_dev[64];
static std::mutex g_dev_mu;

static const void* kernel_ptr(int dtype, bool beta1) {
  if (dtype == ASYMSPEC_BF16)
    return beta1 ? (const void*)fuse_verify_kernel<ASYMSPEC_BF16, true>
                 : (const void*)fuse_verify_kernel<ASYMSPEC_BF16, false>;
  return beta1 ? (const void*)fuse_verify_kernel<ASYMSPEC_FP32, true>
               : (const void*)fuse_verify_kernel<ASYMSPEC_FP32, false>;
}

static const DevInfo* device_info() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return nullptr;
  std::lock_guard<std::mutex> lk(g_dev_mu);
  DevInfo& di = g_dev[dev];
  if (di.ok) return &di;
  hipDeviceProp_t pr;
  if (hipGetDeviceProperties(&pr, dev) != hipSuccess) return nullptr;
  if (std::strncmp(pr.gcnArchName, "gfx950", 6) != 0) return nullptr;
  di.n_cu = pr.multiProcessorCount;
  for (int dt = 0; dt < 2; ++dt) {
    int nb = 1 << 30;
    for (int b1 = 0; b1 < 2; ++b1) {
      int x = 0;
      if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&x, kernel_ptr(dt, b1 != 0), kThreads, 0) != hipSuccess)
        return nullptr;
      nb = std::min(nb, x);
    }
    if (nb < 1) return nullptr;
    di.max_blocks[dt] = nb * di.n_cu;
  }
  di.ok = 1;
  return &di;
}

static uint32_t next_epoch() {
  static std::atomic<uint32_t> ctr{0};
  static std::once_flag once;
  std::call_once(once, [] {
    const uint64_t t = (uint64_t)std::chrono::steady_clock::now().time_since_epoch().count();
    // a varying start well below 2^31, so that epochs keep growing (the
    // work-queue counters rely on it) for 2^31 launches
    ctr.store((uint32_t)((t ^ (t >> 32) ^ ((uint64_t)getpid() << 16)) & 0x3FFFFFFFu) | 1u);
  });
  uint32_t e;
  do { e = ctr.fetch_add(1u); } while (e == 0u);
  return e;
}

static bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

}  // namespace asym

using namespace asym;

extern "C" {

size_t asymspec_workspace_size(int B, int K, int V, int dtype) {
  Layout L;
  if (!make_layout(B, K, V, dtype, L)) return 0;
  return L.total;
}

int asymspec_workspace_clear(void* workspace, size_t workspace_bytes, void* stream) {
  if (workspace == nullptr || workspace_bytes % 4 != 0 || !aligned(workspace, 4)) return ASYMSPEC_E_ARG;
  if (workspace_bytes == 0) return ASYMSPEC_OK;
  const size_t n = workspace_bytes / 4;
  const int blocks = (int)std::min<size_t>((n + 255) / 256, 4096);
  hipLaunchKernelGGL(fill_zero_kernel, dim3(blocks), dim3(256), 0, (hipStream_t)stream,
                     (uint32_t*)workspace, n);
  return hipGetLastError() == hipSuccess ? ASYMSPEC_OK : ASYMSPEC_E_DEVICE;
}

int asymspec_fuse_verify(const void* t, const void* a, const void* b, int dtype,
                         const int32_t* draft_tokens, const float* draft_probs,
                         const float* uniforms, const float* temperature,
                         int B, int K, int V, const asymspec_params* params,
                         int32_t* accept_len, int32_t* next_token, float* fused_logprobs,
                         float* gate_out, void* workspace, size_t workspace_bytes,
                         void* stream) {
  Layout L;
  if (params == nullptr) return ASYMSPEC_E_ARG;
  if (!make_layout(B, K, V, dtype, L)) return ASYMSPEC_E_ARG;
  if (t == nullptr || uniforms == nullptr || temperature == nullptr || accept_len == nullptr ||
      next_token == nullptr || fused_logprobs == nullptr || workspace == nullptr)
    return ASYMSPEC_E_ARG;
  if (K > 0 && (a == nullptr || b == nullptr || draft_tokens == nullptr)) return ASYMSPEC_E_ARG;
  if (!std::isfinite(params->beta) || params->beta < 0.0f) return ASYMSPEC_E_ARG;
  if (!(params->gamma > 0.0f && params->gamma <= 1.0f)) return ASYMSPEC_E_ARG;
  if (params->gate_mode != ASYMSPEC_GATE_CDA && params->gate_mode != ASYMSPEC_GATE_FIXED) return ASYMSPEC_E_ARG;
  if (params->flags != 0u) return ASYMSPEC_E_ARG;
  if (!aligned(t, 16) || (K > 0 && (!aligned(a, 16) || !aligned(b, 16)))) return ASYMSPEC_E_ALIGN;
  if (!aligned(uniforms, 4) || !aligned(temperature, 4) || !aligned(accept_len, 4) ||
      !aligned(next_token, 4) || !aligned(fused_logprobs, 4) ||
      (draft_tokens && !aligned(draft_tokens, 4)) || (draft_probs && !aligned(draft_probs, 4)) ||
      (gate_out && !aligned(gate_out, 4)))
    return ASYMSPEC_E_ALIGN;
  if (!aligned(workspace, 256)) return ASYMSPEC_E_ALIGN;
  if (workspace_bytes < L.total) return ASYMSPEC_E_WORKSPACE;
  const DevInfo* di = device_info();
  if (di == nullptr) return ASYMSPEC_E_DEVICE;

  KArgs A;
  std::memset(&A, 0, sizeof(A));
  A.t = t; A.a = (K > 0) ? a : t; A.b = (K > 0) ? b : t;
  A.d = (K > 0) ? draft_tokens : (const int32_t*)uniforms;
  A.dp = draft_probs; A.u = uniforms; A.tau = temperature;
  A.acc_out = accept_len; A.next_out = next_token; A.flp_out = fused_logprobs; A.gate_out = gate_out;
  char* ws = (char*)workspace;
  A.rec1 = (uint64_t*)(ws + L.off_rec1);
  A.dec = (uint64_t*)(ws + L.off_dec);
  A.rec2 = (uint64_t*)(ws + L.off_rec2);
  A.qctr = (uint64_t*)(ws + L.off_q);
  A.err = (uint32_t*)(ws + L.off_err);
  A.stream_bytes = (unsigned long long)B * (K + 1) * (unsigned long long)V * (dtype == ASYMSPEC_BF16 ? 2ull : 4ull);
  A.B = B; A.K = K; A.V = V; A.S = L.S;
  A.beta = params->beta; A.gamma = params->gamma; A.gate_mode = params->gate_mode;
  A.want_gate = gate_out != nullptr;
  A.ln_gamma = std::log((double)params->gamma);
  A.epoch = next_epoch();
  const int gmax = di->max_blocks[dtype];
  if (!sched_build(B, K, L.S, gmax, A.sc)) return ASYMSPEC_E_ARG;
  const int grid = std::min(gmax, A.sc.total);

  // An ordinary launch: the queues need no co-residency (see queue_init).
  void* args[] = {&A};
  const hipError_t e = hipLaunchKernel(kernel_ptr(dtype, params->beta == 1.0f), dim3(grid),
                                       dim3(kThreads), args, 0, (hipStream_t)stream);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return ASYMSPEC_E_DEVICE;
  }
  return ASYMSPEC_OK;
}

const char* asymspec_status_string(int status) {
  switch (status) {
    case ASYMSPEC_OK: return "ok";
    case ASYMSPEC_E_ARG: return "invalid argument";
    case ASYMSPEC_E_ALIGN: return "misaligned pointer";
    case ASYMSPEC_E_WORKSPACE: return "workspace too small";
    case ASYMSPEC_E_DEVICE: return "device error (no gfx950 device current, or launch failed)";
    default: return "unknown status";
  }
}

int asymspec_version(void) { return 200; }

}  // extern "C"
