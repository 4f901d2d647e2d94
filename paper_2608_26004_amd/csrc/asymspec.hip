// AsymSpec fused decision step for MI355X (gfx950, CDNA4, wave64).
//
// One launch does the whole step of Alg. 1 for every request: the
// vocabulary-wide statistics of the verifier logits t and the drafter logits
// a (full view) and b (compressed view), the delta-fused logits
// f = t + beta (a - b) (Sec. 3.2, Eq. 1-2), the Jensen-Shannon divergence D and
// the CDA gate gamma * exp(-D) (Sec. 3.3, Eq. 3), the acceptance test (Eq. 4,
// or its speculative-sampling form for temperature > 0), and the emission at
// the first rejection or the bonus token.
//
// The launch is an ordered list of work items (schedule.h), one workgroup per
// item, so the hardware dispatcher hands them out in list order and balances
// them over the compute units.  Statistics items (stats.h) stream every logit
// once from HBM and never wait; per request, a decide, S pass-2 and a pick
// item (resolve.h) follow a few requests behind and re-read only the rows
// whose outcome needs a second pass.
//
// Cross-workgroup records are arrays of 64-bit slots whose high word is the
// launch epoch and low word a payload, written and read with relaxed
// system-scope atomics (no cache flushes).  An aligned 64-bit access is
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
#include "dump.h"
#include "resolve.h"
#include "schedule.h"
#include "stats.h"

namespace asym {

template <int DT, bool kB1, int DM, bool kKL>
DEV void stats_chunk(const KArgs& A, int req, int i, int m, Smem& sm) {
  const int row = req * (A.K + 1) + i;
  const float tau = sload_f32(A.tau, req);
  if (i == A.K) {
    if (A.fuse_bonus) {
      if (tau > 0.0f) stats_item<DT, kSampleBonusF, kB1, DM>(A, row, m, sm);
      else stats_item<DT, kGreedyBonusF, kB1, DM>(A, row, m, sm);
    } else if (tau > 0.0f) {
      stats_item<DT, kSampleBonus, kB1, DM>(A, row, m, sm);
    } else {
      stats_item<DT, kGreedyBonus, kB1, DM>(A, row, m, sm);
    }
  } else if (!(tau > 0.0f)) {
    stats_item<DT, kGreedyDraft, kB1, DM, kKL>(A, row, m, sm);
  } else if (tau == 1.0f) {
    stats_item<DT, kSampleDraft1, kB1, DM, kKL>(A, row, m, sm);
  } else {
    stats_item<DT, kSampleDraftT, kB1, DM, kKL>(A, row, m, sm);
  }
}

// Workgroups go to the 8 XCDs in turn, so consecutive items of a request
// sit on different XCDs.  Through a vocabulary map every chunk of a row
// gathers from the whole of the row's drafter logits; the items of a request
// are then renumbered so that those sharing an XCD take consecutive chunks
// of the same rows, and each XCD's L2 holds few drafter rows at a time.
template <int DT, bool kB1, int DM, bool kKL>
DEV void stats_dispatch(const KArgs& A, int req, int sub, Smem& sm) {
  int p = sub;
  if (A.vmap != nullptr) {
    // within each group of rows (all rows, or the two groups of early exit)
    const int n1 = A.sc.G * A.S, n = (A.K + 1) * A.S;
    p = sub < n1 ? xcd_grouped(sub, n1) : n1 + xcd_grouped(sub - n1, n - n1);
  }
  const int i = p / A.S, m = p - i * A.S;
  stats_chunk<DT, kB1, DM, kKL>(A, req, i, m, sm);
}


#ifndef ASYMSPEC_WAVES
#define ASYMSPEC_WAVES 4
#endif

// One workgroup per item.  An item waits only for items earlier in the list
// (lower workgroup index), and each XCD starts its share of the workgroups in
// index order, so the lowest waiting workgroup always waits on items that are
// running or queued behind workgroups that never wait: the list drains
// whether or not every workgroup fits on the chip at once.  The waits are
// bounded besides (Poll), and a timeout is counted in the workspace.
// kKL: calls with the KL gate, whose draft rows also sum the divergence
// beside the A slot (a kernel of its own, so that the extra registers of
// those items do not weigh on the other gates' kernels).
template <int DT, bool kB1, int DM, bool kKL>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(ASYMSPEC_WAVES)))
void fuse_verify_kernel(KArgs A) {
  __shared__ Smem sm;
#ifdef ASYMSPEC_TRACE
  const uint64_t t_start = __builtin_amdgcn_s_memrealtime();
  if (threadIdx.x == 0) sm.t_mark[0] = sm.t_mark[1] = t_start;
#endif
  const Item it = sched_item(A.sc, A.K, A.S, (int)blockIdx.x);
  int type = it.type;
  if (type == kItemStats2) {
    // early exit: the rows after the first group are read unless the
    // verdict found a sure rejection among the first rows
    type = load_verdict(A, it.req, sm) == kVerdictSkip ? kItemNone : kItemStats;
  }
  // one call site per item kind keeps a single inlined copy of each
  switch (type) {
    case kItemStats: stats_dispatch<DT, kB1, DM, kKL>(A, it.req, it.sub, sm); break;
    case kItemVerdict:
    case kItemDecide: decide_item<DT>(A, it.req, sm, type == kItemVerdict); break;
    case kItemPass2: pass2_item<DT, DM>(A, it.req, it.sub, sm); break;
    case kItemPick: pick_item<DT, DM>(A, it.req, sm); break;
    default: break;
  }
#ifdef ASYMSPEC_TRACE
  // timeline of the launch (a build option for measurement): per item its
  // start and end on the 100 MHz clock, kind and request, and for statistics
  // items when the first streaming load went out and when the stream ended
  if (threadIdx.x == 0 && A.trace != nullptr && blockIdx.x < A.trace_items) {
    uint64_t* tr = A.trace + (size_t)blockIdx.x * 4;
    tr[0] = t_start;
    tr[1] = __builtin_amdgcn_s_memrealtime();
    tr[2] = (uint64_t)(uint32_t)it.type | ((uint64_t)(uint32_t)it.req << 8) | ((uint64_t)(uint32_t)it.sub << 40);
    tr[3] = (sm.t_mark[0] - t_start) | ((sm.t_mark[1] - t_start) << 32);
  }
#endif
}

// The drafter-to-verifier map of a cross-family call: inv[j] = x for the
// verifier token x with vmap[x] = j, else -1; inv[Vd] is set when two
// verifier tokens name the same drafter id (the map is then not used).
__global__ void inv_clear_kernel(int32_t* inv, int Vd) {
  for (int j = blockIdx.x * blockDim.x + threadIdx.x; j <= Vd; j += gridDim.x * blockDim.x)
    inv[j] = j < Vd ? -1 : 0;
}
__global__ void inv_fill_kernel(const int32_t* vmap, int V, int32_t* inv, int Vd) {
  for (int x = blockIdx.x * blockDim.x + threadIdx.x; x < V; x += gridDim.x * blockDim.x) {
    const int j = vmap[x];
    if (j >= 0 && j < Vd && atomicCAS(&inv[j], -1, x) != -1) inv[Vd] = 1;
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
  size_t off_rec1, off_dec, off_rec2, off_err, off_inv, off_trace, total;
};

static size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Vd > 0: a drafter vocabulary of Vd tokens (cross-family calls); rows then
// have as many chunks as the longer of the two vocabularies needs, and the
// workspace holds the drafter-to-verifier map.
static bool make_layout(int B, int K, int V, int dtype, Layout& L, int Vd = 0) {
  if (B < 1 || K < 0 || K > kMaxK || V < 1 || Vd < 0) return false;
  if (dtype != ASYMSPEC_BF16 && dtype != ASYMSPEC_FP32) return false;
  const long double elems = (long double)B * (K + 1) * V;
  if (elems >= (long double)(1ull << 40)) return false;
  if ((long double)B * (K + 1) * Vd >= (long double)(1ull << 40)) return false;
  L.VE = dtype == ASYMSPEC_BF16 ? 8 : 4;
  // a row spans at most this many 16-byte vectors (it may start mid-vector)
  const long long nvec_max = ((long long)(V > Vd ? V : Vd) + 2LL * L.VE - 2) / L.VE;
  const long long S = (nvec_max + kChunkVec - 1) / kChunkVec;
  // a request's decision combines each row's chunks in one workgroup pass
  if (S > kThreads) return false;
  L.S = (int)S;
  L.rows = (size_t)B * (K + 1);
  size_t off = 0;
  // the timeout counter first, at a place that does not depend on the shape
  L.off_err = off;  off = align_up(off + 8, 256);
  L.off_rec1 = off; off = align_up(off + L.rows * L.S * kR1 * 8, 256);
  L.off_dec = off;  off = align_up(off + (size_t)B * (kDecHdr + (size_t)(K + 1) * kDecRow) * 8, 256);
  L.off_rec2 = off; off = align_up(off + L.rows * L.S * kR2 * 8, 256);
  // cross-family: inverse map [Vd] and its duplicate flag
  L.off_inv = off;  off = align_up(off + (Vd > 0 ? (size_t)Vd * 4 + 4 : 0), 256);
#ifdef ASYMSPEC_TRACE
  // 32 bytes per work item, for at most (K + 1 + kMaxP2) S + 3 items per
  // request (statistics, pass 2, decide, pick, verdict)
  L.off_trace = off;  off = align_up(off + (size_t)B * ((size_t)(K + 1 + kMaxP2) * L.S + 3) * 32, 256);
#endif
  L.total = off;
  return true;
}

// Through a vocabulary map every chunk of a row gathers from the whole of
// the row's drafter logits; launched with this much unused dynamic LDS per
// workgroup, fewer workgroups share a CU, so each XCD works on fewer rows at
// a time and its L2 keeps their drafter rows.
#ifndef ASYMSPEC_XV_LDS
#define ASYMSPEC_XV_LDS 49152
#endif
constexpr size_t kXvLds = ASYMSPEC_XV_LDS;

struct DevInfo {
  int ok = 0;
  int n_cu = 0;
  int max_blocks[2] = {0, 0};   // co-resident workgroups, per dtype
  int max_blocks_xv[2] = {0, 0};   // the same with kXvLds of dynamic LDS
};

static DevInfo g_dev[64];
static std::mutex g_dev_mu;

static_assert(kDeltaAB == ASYMSPEC_DELTA_AB && kDeltaA == ASYMSPEC_DELTA_A && kDeltaTB == ASYMSPEC_DELTA_TB,
              "delta sources");

// One kernel per storage type, beta == 1 or not, and source of delta; the
// KL gate has its own kernels (beta taken at run time: fl(1 * x) = x, so a
// call with beta = 1 computes the same values).
template <int DT>
static const void* kernel_ptr_dt(bool beta1, int dm, bool kl) {
  if (kl) {
    if (dm == kDeltaA) return (const void*)fuse_verify_kernel<DT, false, kDeltaA, true>;
    if (dm == kDeltaTB) return (const void*)fuse_verify_kernel<DT, false, kDeltaTB, true>;
    return (const void*)fuse_verify_kernel<DT, false, kDeltaAB, true>;
  }
  if (beta1) {
    if (dm == kDeltaA) return (const void*)fuse_verify_kernel<DT, true, kDeltaA, false>;
    if (dm == kDeltaTB) return (const void*)fuse_verify_kernel<DT, true, kDeltaTB, false>;
    return (const void*)fuse_verify_kernel<DT, true, kDeltaAB, false>;
  }
  if (dm == kDeltaA) return (const void*)fuse_verify_kernel<DT, false, kDeltaA, false>;
  if (dm == kDeltaTB) return (const void*)fuse_verify_kernel<DT, false, kDeltaTB, false>;
  return (const void*)fuse_verify_kernel<DT, false, kDeltaAB, false>;
}
static const void* kernel_ptr(int dtype, bool beta1, int dm, bool kl) {
  return dtype == ASYMSPEC_BF16 ? kernel_ptr_dt<ASYMSPEC_BF16>(beta1, dm, kl)
                                : kernel_ptr_dt<ASYMSPEC_FP32>(beta1, dm, kl);
}
template <int DT>
static const void* dump_ptr_dt(int dm) {
  if (dm == kDeltaA) return (const void*)dump_kernel<DT, kDeltaA>;
  if (dm == kDeltaTB) return (const void*)dump_kernel<DT, kDeltaTB>;
  return (const void*)dump_kernel<DT, kDeltaAB>;
}
static const void* dump_ptr(int dtype, int dm) {
  return dtype == ASYMSPEC_BF16 ? dump_ptr_dt<ASYMSPEC_BF16>(dm) : dump_ptr_dt<ASYMSPEC_FP32>(dm);
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
    int nb = 1 << 30, nx = 1 << 30;
    for (int v = 0; v < 3; ++v)
      for (int dm = 0; dm < 3; ++dm) {
        int x = 0, y = 0;
        const void* k = kernel_ptr(dt, v == 0, dm, v == 2);
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&x, k, kThreads, 0) != hipSuccess ||
            hipOccupancyMaxActiveBlocksPerMultiprocessor(&y, k, kThreads, kXvLds) != hipSuccess)
          return nullptr;
        nb = std::min(nb, x);
        nx = std::min(nx, y);
      }
    if (nb < 1 || nx < 1) return nullptr;
    di.max_blocks[dt] = nb * di.n_cu;
    di.max_blocks_xv[dt] = nx * di.n_cu;
  }
  di.ok = 1;
  return &di;
}

// Static scratch of the non-allocating entry point: the workspace of calls
// whose callers cannot allocate.  Each device that loads the library holds
// its own copy until the process ends; its address on a device comes from
// hipGetSymbolAddress with that device current (the array's name in host
// code is not a device address).
constexpr size_t kScratchBytes = (size_t)ASYMSPEC_NOALLOC_MAX_WORKSPACE;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];
static void* g_scratch[64];
static std::mutex g_scratch_mu;

// The device address of the current device's scratch, looked up once per
// device; null when the lookup fails.
static void* scratch_ptr() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return nullptr;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (g_scratch[dev] == nullptr) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) {
      (void)hipGetLastError();
      return nullptr;
    }
    g_scratch[dev] = p;
  }
  return g_scratch[dev];
}

static uint32_t next_epoch() {
  static std::atomic<uint32_t> ctr{0};
  static std::once_flag once;
  std::call_once(once, [] {
    const uint64_t t = (uint64_t)std::chrono::steady_clock::now().time_since_epoch().count();
    // a varying start, so that a workspace reused by another process or
    // library instance is unlikely to hold slots tagged with a live epoch
    ctr.store((uint32_t)((t ^ (t >> 32) ^ ((uint64_t)getpid() << 16)) & 0x3FFFFFFFu) | 1u);
  });
  uint32_t e;
  do { e = ctr.fetch_add(1u); } while (e == 0u);
  return e;
}

static bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

// Bound of every wait between workgroups, in ticks of the 100 MHz clock.
static std::atomic<unsigned long long> g_poll_ticks{kPollTicks};

}  // namespace asym

using namespace asym;

extern "C" {

size_t asymspec_workspace_size(int B, int K, int V, int dtype) {
  Layout L;
  if (!make_layout(B, K, V, dtype, L)) return 0;
  return L.total;
}

size_t asymspec_workspace_size_xvocab(int B, int K, int V, int Vd, int dtype) {
  Layout L;
  if (Vd < 1 || !make_layout(B, K, V, dtype, L, Vd)) return 0;
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

// Both entry points: vmap == nullptr for one shared vocabulary, else a and b
// are [B][K+1][Vd] drafter rows reached through vmap.
static int fuse_verify_impl(const void* t, const void* a, const void* b, int dtype, const int32_t* vmap,
                            int Vd, const int32_t* draft_tokens, const float* draft_probs,
                            const float* uniforms, const float* temperature, int B, int K, int V,
                            const asymspec_params* params, int32_t* accept_len, int32_t* next_token,
                            float* fused_logprobs, float* gate_out, float* fused_logprobs_full,
                            void* workspace, size_t workspace_bytes, void* stream) {
  Layout L;
  if (params == nullptr) return ASYMSPEC_E_ARG;
  if (vmap != nullptr && Vd < 1) return ASYMSPEC_E_ARG;
  if (!make_layout(B, K, V, dtype, L, vmap != nullptr ? Vd : 0)) return ASYMSPEC_E_ARG;
  if (t == nullptr || uniforms == nullptr || temperature == nullptr || accept_len == nullptr ||
      next_token == nullptr || fused_logprobs == nullptr || workspace == nullptr)
    return ASYMSPEC_E_ARG;
  const bool fb = (params->flags & ASYMSPEC_FUSE_BONUS) != 0u;
  if (K > 0 && draft_tokens == nullptr) return ASYMSPEC_E_ARG;
  if ((K > 0 || fb) && (a == nullptr || b == nullptr)) return ASYMSPEC_E_ARG;
  if (!std::isfinite(params->beta) || params->beta < 0.0f) return ASYMSPEC_E_ARG;
  if (!(params->gamma > 0.0f && params->gamma <= 1.0f)) return ASYMSPEC_E_ARG;
  if (params->gate_mode < ASYMSPEC_GATE_CDA || params->gate_mode > ASYMSPEC_GATE_LAMBDA) return ASYMSPEC_E_ARG;
  if (params->delta_mode < ASYMSPEC_DELTA_AB || params->delta_mode > ASYMSPEC_DELTA_TB) return ASYMSPEC_E_ARG;
  if (params->gate_mode == ASYMSPEC_GATE_LAMBDA && !std::isfinite(params->lambda)) return ASYMSPEC_E_ARG;
  if ((params->flags & ~(uint32_t)(ASYMSPEC_FUSE_BONUS | ASYMSPEC_EARLY_EXIT)) != 0u) return ASYMSPEC_E_ARG;
  const bool ee = (params->flags & ASYMSPEC_EARLY_EXIT) != 0u;
  if (ee && (params->early_rows < 0 || params->early_rows > 63)) return ASYMSPEC_E_ARG;
  // rows after the first rejection are not read, so they have no full rows
  if (ee && fused_logprobs_full != nullptr) return ASYMSPEC_E_ARG;
  if (vmap != nullptr) {
    // drafter rows are read element by element through the map
    if (Vd < 1 || (unsigned long long)B * (K + 1) * (unsigned long long)Vd >= (1ull << 40)) return ASYMSPEC_E_ARG;
    if (!aligned(vmap, 4) || ((K > 0 || fb) && (!aligned(a, 4) || !aligned(b, 4)))) return ASYMSPEC_E_ALIGN;
    if (!aligned(t, 16)) return ASYMSPEC_E_ALIGN;
  } else if (!aligned(t, 16) || ((K > 0 || fb) && (!aligned(a, 16) || !aligned(b, 16)))) {
    return ASYMSPEC_E_ALIGN;
  }
  if (!aligned(uniforms, 4) || !aligned(temperature, 4) || !aligned(accept_len, 4) ||
      !aligned(next_token, 4) || !aligned(fused_logprobs, 4) ||
      (draft_tokens && !aligned(draft_tokens, 4)) || (draft_probs && !aligned(draft_probs, 4)) ||
      (gate_out && !aligned(gate_out, 4)) || (fused_logprobs_full && !aligned(fused_logprobs_full, 16)))
    return ASYMSPEC_E_ALIGN;
  if (!aligned(workspace, 256)) return ASYMSPEC_E_ALIGN;
  if (workspace_bytes < L.total) return ASYMSPEC_E_WORKSPACE;
  const DevInfo* di = device_info();
  if (di == nullptr) return ASYMSPEC_E_DEVICE;

  KArgs A;
  std::memset(&A, 0, sizeof(A));
  A.t = t; A.a = (K > 0 || fb) ? a : t; A.b = (K > 0 || fb) ? b : t;
  A.d = (K > 0) ? draft_tokens : (const int32_t*)uniforms;
  A.dp = draft_probs; A.u = uniforms; A.tau = temperature;
  A.acc_out = accept_len; A.next_out = next_token; A.flp_out = fused_logprobs; A.gate_out = gate_out;
  char* ws = (char*)workspace;
  A.rec1 = (uint64_t*)(ws + L.off_rec1);
  A.dec = (uint64_t*)(ws + L.off_dec);
  A.rec2 = (uint64_t*)(ws + L.off_rec2);
  A.err = (uint32_t*)(ws + L.off_err);
  A.stream_bytes = (unsigned long long)B * (K + 1) * (unsigned long long)V * (dtype == ASYMSPEC_BF16 ? 2ull : 4ull);
  A.B = B; A.K = K; A.V = V; A.S = L.S;
  A.beta = params->beta; A.gamma = params->gamma; A.gate_mode = params->gate_mode;
  A.want_gate = gate_out != nullptr;
  A.delta_mode = params->delta_mode;
  A.fuse_bonus = fb ? 1 : 0;
  A.vmap = vmap;
  A.Vd = vmap != nullptr ? Vd : V;
  A.inv = vmap != nullptr ? (const int32_t*)(ws + L.off_inv) : nullptr;
#ifdef ASYMSPEC_TRACE
  A.trace = (uint64_t*)(ws + L.off_trace);
  A.trace_items = (unsigned)((size_t)B * ((size_t)(K + 1 + kMaxP2) * L.S + 3));
#endif
  A.lam = params->gate_mode == ASYMSPEC_GATE_LAMBDA ? params->lambda : 0.0f;
  A.ln_gamma = std::log((double)params->gamma);
  A.epoch = next_epoch();
  A.poll_ticks = g_poll_ticks.load();
  // lags scale with the number of workgroups the chip holds at once
  const int ee_rows = ee ? (params->early_rows > 0 ? params->early_rows : 2) : 0;
  const int in_flight = vmap != nullptr ? di->max_blocks_xv[dtype] : di->max_blocks[dtype];
  // pass 2 in 8, 4 or 2 items per chunk while that many still fit on the
  // chip at once: a small batch leaves most of it idle, and pass 2's
  // divergence terms are arithmetic-bound within one workgroup
  const long long p2_items = (long long)B * L.S;
  A.P2 = 1;
  while (A.P2 < kMaxP2 && p2_items * 2 * A.P2 <= in_flight) A.P2 *= 2;
  // with the gate output and a JSD-based gate, pass 2 sums the divergence of
  // every draft row whose views differ, not only of the open ones: at least
  // two parts per chunk then shorten the last requests' pass 2
  if (A.want_gate && params->gate_mode != ASYMSPEC_GATE_KL && params->gate_mode != ASYMSPEC_GATE_LAMBDA &&
      A.P2 < 2)
    A.P2 = 2;
  // a launch whose statistics items fit the chip at most four times over
  // polls every slot it waits for (measured: 0.5-0.8 us less per call
  // there; on larger launches it saves nothing and its polling traffic
  // costs a little)
  A.full_poll = (long long)B * (K + 1) * L.S <= 4LL * in_flight ? 1 : 0;
  if (!sched_build(B, K, L.S, in_flight, A.sc, ee_rows, A.P2)) return ASYMSPEC_E_ARG;
  const int grid = A.sc.total;

  const unsigned long long nblk = (unsigned long long)B * (K + 1) * L.S;
  if (fused_logprobs_full != nullptr && nblk > 0x7FFFFFFFull) return ASYMSPEC_E_ARG;
  hipError_t e = hipSuccess;
  if (vmap != nullptr) {
    // the drafter-to-verifier map, rebuilt for every call (the caller's map
    // may change between calls)
    int32_t* inv = (int32_t*)(ws + L.off_inv);
    const int nb_d = (int)std::min<long long>((Vd + 1 + 255) / 256, 4096);
    const int nb_v = (int)std::min<long long>((V + 255) / 256, 4096);
    hipLaunchKernelGGL(inv_clear_kernel, dim3(nb_d), dim3(256), 0, (hipStream_t)stream, inv, Vd);
    hipLaunchKernelGGL(inv_fill_kernel, dim3(nb_v), dim3(256), 0, (hipStream_t)stream, vmap, V, inv, Vd);
    e = hipGetLastError();
    if (e != hipSuccess) return ASYMSPEC_E_DEVICE;
  }
  void* args[] = {&A};
  e = hipLaunchKernel(kernel_ptr(dtype, params->beta == 1.0f, params->delta_mode,
                                 params->gate_mode == ASYMSPEC_GATE_KL), dim3(grid),
                                 dim3(kThreads), args, vmap != nullptr ? kXvLds : 0, (hipStream_t)stream);
  if (e == hipSuccess && fused_logprobs_full != nullptr) {
    // one workgroup per (row, chunk), after the decision kernel on the stream
    float* full = fused_logprobs_full;
    void* dargs[] = {&A, &full};
    e = hipLaunchKernel(dump_ptr(dtype, params->delta_mode), dim3((unsigned)nblk), dim3(kThreads), dargs,
                        vmap != nullptr ? kXvLds : 0, (hipStream_t)stream);
  }
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return ASYMSPEC_E_DEVICE;
  }
  return ASYMSPEC_OK;
}

int asymspec_fuse_verify(const void* t, const void* a, const void* b, int dtype,
                         const int32_t* draft_tokens, const float* draft_probs,
                         const float* uniforms, const float* temperature,
                         int B, int K, int V, const asymspec_params* params,
                         int32_t* accept_len, int32_t* next_token, float* fused_logprobs,
                         float* gate_out, float* fused_logprobs_full, void* workspace,
                         size_t workspace_bytes, void* stream) {
  return fuse_verify_impl(t, a, b, dtype, nullptr, 0, draft_tokens, draft_probs, uniforms, temperature, B, K, V,
                          params, accept_len, next_token, fused_logprobs, gate_out, fused_logprobs_full,
                          workspace, workspace_bytes, stream);
}

int asymspec_fuse_verify_xvocab(const void* t, const void* a, const void* b, int dtype,
                                const int32_t* vocab_map, int Vd, const int32_t* draft_tokens,
                                const float* draft_probs, const float* uniforms,
                                const float* temperature, int B, int K, int V,
                                const asymspec_params* params, int32_t* accept_len,
                                int32_t* next_token, float* fused_logprobs, float* gate_out,
                                float* fused_logprobs_full, void* workspace,
                                size_t workspace_bytes, void* stream) {
  if (vocab_map == nullptr) return ASYMSPEC_E_ARG;
  return fuse_verify_impl(t, a, b, dtype, vocab_map, Vd, draft_tokens, draft_probs, uniforms, temperature, B, K,
                          V, params, accept_len, next_token, fused_logprobs, gate_out, fused_logprobs_full,
                          workspace, workspace_bytes, stream);
}

int asymspec_fuse_verify_noalloc(const void* t, const void* a, const void* b, int dtype,
                                 const int32_t* draft_tokens, const float* draft_probs,
                                 const float* uniforms, const float* temperature,
                                 int B, int K, int V, const asymspec_params* params,
                                 int32_t* accept_len, int32_t* next_token, float* fused_logprobs,
                                 float* gate_out, float* fused_logprobs_full, void* stream) {
  Layout L;
  if (!make_layout(B, K, V, dtype, L)) return ASYMSPEC_E_ARG;
  if (L.total > kScratchBytes) return ASYMSPEC_E_WORKSPACE;
  void* ws = scratch_ptr();
  if (ws == nullptr) return ASYMSPEC_E_DEVICE;
  return fuse_verify_impl(t, a, b, dtype, nullptr, 0, draft_tokens, draft_probs, uniforms, temperature, B, K, V,
                          params, accept_len, next_token, fused_logprobs, gate_out, fused_logprobs_full, ws,
                          kScratchBytes, stream);
}

int asymspec_noalloc_timeouts(void* stream, uint32_t* count) {
  if (count == nullptr) return ASYMSPEC_E_ARG;
  void* ws = scratch_ptr();
  if (ws == nullptr) return ASYMSPEC_E_DEVICE;
  return asymspec_workspace_timeouts(ws, kScratchBytes, stream, count);
}

int asymspec_workspace_timeouts(const void* workspace, size_t workspace_bytes, void* stream,
                                uint32_t* count) {
  if (workspace == nullptr || count == nullptr || workspace_bytes < 256 || !aligned(workspace, 256))
    return ASYMSPEC_E_ARG;
  uint32_t v = 0;
  if (hipMemcpyAsync(&v, workspace, sizeof(v), hipMemcpyDeviceToHost, (hipStream_t)stream) != hipSuccess ||
      hipStreamSynchronize((hipStream_t)stream) != hipSuccess) {
    (void)hipGetLastError();
    return ASYMSPEC_E_DEVICE;
  }
  *count = v;
  return ASYMSPEC_OK;
}

int asymspec_set_wait_limit(unsigned long long ticks) {
  if (ticks > 100000000ull) return ASYMSPEC_E_ARG;
  g_poll_ticks.store(ticks == 0 ? kPollTicks : ticks);
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

int asymspec_version(void) { return 300; }

}  // extern "C"
