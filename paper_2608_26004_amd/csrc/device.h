// Device-side building blocks of the fused decision step (gfx950, wave64):
// constants, record formats, epoch-tagged slots, buffer loads, logit decode,
// DPP wave reductions, the online log-sum-exp accumulator and the pass-2
// element functions.

#ifndef ASYMSPEC_DEVICE_H_
#define ASYMSPEC_DEVICE_H_

#include <hip/hip_runtime.h>

#include <cfloat>
#include <cstdint>

#include "asymspec.h"

#define DEV __device__ __forceinline__
#define ASYM_HD __host__ __device__
#include "schedule.h"

namespace asym {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
// A chunk is 2048 vectors (32 KiB of bf16).  One sub-tile of 8 vectors per
// thread measured 2% faster than two of 4 on the bench workload.
#ifndef ASYMSPEC_NV
#define ASYMSPEC_NV 8
#endif
#ifndef ASYMSPEC_NSUB
#define ASYMSPEC_NSUB 1
#endif
constexpr int kNV = ASYMSPEC_NV;                // 16-byte vectors per thread per sub-tile
constexpr int kNSub = ASYMSPEC_NSUB;            // sub-tiles per statistics item
constexpr int kTileVec = kThreads * kNV;        // vectors per sub-tile
constexpr int kChunkVec = kTileVec * kNSub;     // vectors per vocabulary chunk
constexpr int kSegVec = kChunkVec / kWaves;     // one wave's contiguous segment (pass 2)
constexpr int kSegPerLane = kSegVec / 64;       // vectors per lane in a segment
// Pass 2 sums the weights of a chunk per sub-block of 64 consecutive vectors
// (one vector per lane of a wave): kSegPerLane sub-blocks per wave segment.
constexpr int kSubPerChunk = kWaves * kSegPerLane;
constexpr int kMaxK = 63;                       // K + 1 rows of a request fit one wave
// pass 2 reads a lane's segment in groups of 4 vectors
static_assert(kSegPerLane % 4 == 0, "the tile size must give whole pass-2 groups");

constexpr float kL2E = 1.44269504088896340736f;
constexpr double kLn2 = 0.693147180559945309417232121458;
constexpr float kFloorM = -1.0e30f;             // start value of running maxima
constexpr uint32_t kBf16NegInf = 0xFF80u;
constexpr uint32_t kF32NegInf = 0xFF800000u;
constexpr uint64_t kPollTicks = 20000000;      // give up a wait after 0.2 s (100 MHz clock): the default

typedef uint32_t u4 __attribute__((ext_vector_type(4)));
typedef const __attribute__((address_space(4))) uint32_t* cptr32;

// Row kinds.  Every row of a request has the request's temperature; row K is
// the bonus position, taken from t (Alg. 1) or, when the bonus row is fused,
// from f = t + beta delta.
enum Kind {
  kGreedyDraft = 0, kSampleDraft1 = 1, kSampleDraftT = 2, kGreedyBonus = 3, kSampleBonus = 4,
  kGreedyBonusF = 5, kSampleBonusF = 6
};
// Statistics slots: t, a and b at temperature 1 (greedy t, and the JSD of
// Eq. 3 at temperature 1), f (fused logits, at the row's temperature), and a
// at the row's temperature when that is not 1 (the proposal q).
enum Slot { sT = 0, sA = 1, sB = 2, sF = 3, sAT = 4, kSlots = 5 };

// Statistics record of one (row, chunk): per slot a reference exponent R
// (fp32, log2 units; at most the chunk maximum of x * c) and the sum of
// exp2(x * c - R) over the chunk (fp32), the maximum of the argmax slot (f
// for greedy drafts, t for the greedy bonus row) and the first index where
// the chunk attains it, and whether a and b differ bitwise anywhere in the
// chunk.
// Calls with the KL gate also carry W, the sum of exp2(a * log2 e - R_A) (a -
// b) relative to the A slot's reference: KL(P || Q) = W / S_A - (LA - LB) in
// nats, with no second pass.
enum { R1_R = 0, R1_S = kSlots, R1_ARG = 2 * kSlots, R1_NEQ = 2 * kSlots + 1, R1_MARG = 2 * kSlots + 2,
       R1_W = 2 * kSlots + 3, R1_USED = 2 * kSlots + 4, kR1 = 16 };

// Decision record of one request: a header and one block per row, published
// by the decide item; pass-2 and pick items load it into LDS (Smem::req,
// Smem::rows).
enum { H_STATE = 0, H_J = 1, H_TASK_LO = 2, H_TASK_HI = 3, H_SAMP = 4, H_USED = 5, H_VERDICT = 5, kDecHdr = 8 };
// Early exit: the verdict on a request's first rows (a sure rejection among
// them makes the other rows unneeded).
enum { kVerdictRead = 1, kVerdictSkip = 2 };
// kStateFailed: a wait of the decide item timed out (or, as seen by a later
// item, its own wait for the decision did); the request's outputs are marked
// invalid (accept_len = -1).
enum { kStateFinal = 1, kStatePending = 2, kStateFailed = 3 };
enum { R_J = 0, R_TASK_LO = 1, R_TASK_HI = 2, R_FIN = 3, R_SAMP = 4, R_FAIL = 5, kReqWords = 6 };
enum {
  D_TASK = 0,   // pass-2 work on the row: kTaskJsd | kTaskRes | kTaskBonus
  D_C,          // exponent scale of the row's emission distribution (log2 e / tau, or log2 e)
  D_RF,         // reference exponent of p~ (drafts) or of the bonus weights
  D_ISF,        // 1 / sum of p~ weights (drafts)
  D_RQ, D_ISQ,  // the same for the proposal q = softmax(a / tau)
  D_RA, D_RB,   // reference exponents of a and b at temperature 1 (JSD)
  D_KAHI, D_KALO, D_KBHI, D_KBLO,  // log2 of the a and b sums, as hi + lo floats
  D_LPD,        // log p~(d): fused log-probability of the draft token
  D_STATUS,     // kStDecided | kStAccept | kStDraft | kStNeq
  D_THR_LO, D_THR_HI,   // open rows: accepted iff D > thr (fp64)
  D_L2E_LO, D_L2E_HI,   // log2 normaliser (fp64) of the emission distribution
  D_ARG,        // greedy: argmax of f (drafts) or t (bonus)
  D_LPEMIT,     // greedy: log-probability of that argmax
  D_GD_LO, D_GD_HI,     // D known at the decide (lambda and KL gates; fp64)
  D_USED,
  kDecRow = 24
};
enum { kTaskJsd = 1, kTaskRes = 2, kTaskBonus = 4 };
// kStSkip: a row after a sure rejection that early exit did not read.
enum { kStDecided = 1, kStAccept = 2, kStDraft = 4, kStNeq = 8, kStSkip = 16 };

// Pass 2 splits each chunk into P2 in {1, 2, 4, 8} contiguous parts, one
// item each.  Pass-2 record of one (request, row, chunk): the JSD partial of each
// part (fp32, in log2 units) and the weight sums of the chunk's sub-blocks
// (fp32, in vocabulary order), one slot each.
constexpr int kMaxP2 = 8;
static_assert(kSegPerLane % kMaxP2 == 0, "a pass-2 part must give each lane whole vectors");
enum { P2_J = 0, P2_SEG = kMaxP2, P2_USED = P2_SEG + kSubPerChunk, kR2 = P2_USED };

struct KArgs {
  const void* t; const void* a; const void* b;
  const int32_t* d; const float* dp; const float* u; const float* tau;
  int32_t* acc_out; int32_t* next_out; float* flp_out; float* gate_out;
  uint64_t* rec1; uint64_t* dec; uint64_t* rec2;
  uint32_t* err;
  unsigned long long stream_bytes;   // bytes of each logit array
  int B, K, V, S;
  int P2;             // pass-2 items per chunk
  int full_poll;      // waits poll every slot they need, not a sentinel
  float beta, gamma; int gate_mode; int want_gate;
  int delta_mode;     // source of delta in f = t + beta * delta
  int fuse_bonus;     // the bonus row emits from f rather than t
  float lam;          // scale of the lambda gate
  // cross-family vocabularies: a and b are [B][K+1][Vd] in the drafter's
  // vocabulary and vmap[x] is the drafter id of verifier token x (or < 0 /
  // >= Vd: not shared); null when both sides share one vocabulary
  const int32_t* vmap;
  int Vd;
  // the drafter-to-verifier map built from vmap for this call ([Vd], then a
  // word that is non-zero when two verifier tokens share a drafter id), or
  // null
  const int32_t* inv;
  double ln_gamma;
  uint32_t epoch;
  uint64_t poll_ticks;   // bound of every wait, in ticks of the 100 MHz clock
  Sched sc;
#ifdef ASYMSPEC_TRACE
  uint64_t* trace;    // per-item timeline (measurement builds only)
  unsigned trace_items;   // items the timeline holds
#endif
};

// Thread coordinates for item code.  They pass through empty asm so that the
// compiler cannot hoist index arithmetic of one item type out of the
// persistent loop and keep it live across all the others; the wave index
// stays a scalar.
DEV int lane_id() {
  int l = (int)threadIdx.x & 63;
  asm volatile("" : "+v"(l));
  return l;
}
DEV int wave_id() {
  int w = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6);
  asm volatile("" : "+s"(w));
  return w;
}

// ------------------------------------------------------------------ memory
// Tagged slots are written and polled at system scope.  Each XCD of the chip
// has its own L2; an agent-scope load may be served from a line that this
// XCD cached before another XCD wrote the slot, and a poller can then read
// the stale value for as long as the line stays resident.  System-scope
// accesses go to the coherent memory side.
DEV void st_tag(uint64_t* p, uint32_t v, uint32_t ep) {
  __hip_atomic_store(p, ((uint64_t)ep << 32) | (uint64_t)v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}
DEV uint64_t ld_tag(const uint64_t* p) {
  return __hip_atomic_load(const_cast<uint64_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}
DEV bool tag_ok(uint64_t v, uint32_t ep) { return (uint32_t)(v >> 32) == ep; }
DEV uint32_t pay(uint64_t v) { return (uint32_t)v; }
DEV float payf(uint64_t v) { return __uint_as_float((uint32_t)v); }
DEV double payd(uint64_t lo, uint64_t hi) {
  return __builtin_bit_cast(double, (uint64_t)(uint32_t)lo | ((uint64_t)(uint32_t)hi << 32));
}
DEV uint32_t dlo(double x) { return (uint32_t)__builtin_bit_cast(uint64_t, x); }
DEV uint32_t dhi(double x) { return (uint32_t)(__builtin_bit_cast(uint64_t, x) >> 32); }
DEV double u2d(uint32_t lo, uint32_t hi) {
  return __builtin_bit_cast(double, (uint64_t)lo | ((uint64_t)hi << 32));
}
DEV void err_count(const uint32_t* e) {
  __hip_atomic_fetch_add(const_cast<uint32_t*>(e), 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// Bounded polling with exponential backoff: the n-th retry sleeps
// 128 * 2^min(n, kPollMaxShift) cycles, so a wave that waits long issues few
// loads and leaves the memory system to the streaming work; a wait gives up
// (and counts an error) after A.poll_ticks of the 100 MHz real-time clock
// (kPollTicks unless the host set another bound).
#ifndef ASYMSPEC_POLL_SHIFT
#define ASYMSPEC_POLL_SHIFT 3
#endif
constexpr int kPollMaxShift = ASYMSPEC_POLL_SHIFT;
struct Poll {
  uint64_t t0;
  int n;
  DEV Poll() : t0(__builtin_amdgcn_s_memrealtime()), n(0) {}
  // Sleeps before the next poll; false once the wait has timed out.
  DEV bool again(const KArgs& A) {
    const int reps = 1 << (n < kPollMaxShift ? n : kPollMaxShift);
    for (int i = 0; i < reps; ++i) __builtin_amdgcn_s_sleep(2);
    ++n;
    if (__builtin_amdgcn_s_memrealtime() - t0 > A.poll_ticks) {
      err_count(A.err);
      return false;
    }
    return true;
  }
};

// Workgroup-wide polling step: done() is true once every thread's ok holds;
// otherwise it sleeps with the same backoff as Poll and returns false, or
// gives up (true, with timed_out set, and counts an error) when thread 0
// finds the wait timed out.  Every thread gets the same answer.
struct BlockPoll {
  uint64_t t0;
  int n;
  bool timed_out;
  DEV BlockPoll() : t0(__builtin_amdgcn_s_memrealtime()), n(0), timed_out(false) {}
  DEV bool done(bool ok, const KArgs& A) {
    if (__syncthreads_and(ok)) return true;
    const int reps = 1 << (n < kPollMaxShift ? n : kPollMaxShift);
    for (int i = 0; i < reps; ++i) __builtin_amdgcn_s_sleep(2);
    ++n;
    const bool late = threadIdx.x == 0 && __builtin_amdgcn_s_memrealtime() - t0 > A.poll_ticks;
    if (__syncthreads_or(late)) {
      if (threadIdx.x == 0) err_count(A.err);
      timed_out = true;
      return true;
    }
    return false;
  }
};

// Whole workgroup: wait (bounded) until slot p carries the launch epoch,
// with one load per poll.  False (in every thread) when the wait timed out.
DEV bool wait_one(const uint64_t* p, const KArgs& A) {
  BlockPoll bp;
  while (!bp.done(threadIdx.x != 0 || tag_ok(ld_tag(p), A.epoch), A)) {
  }
  return !bp.timed_out;
}

// Whole workgroup: load() requests a set of tagged slots and returns whether
// this thread's share all carry the launch epoch.  When the first attempt
// misses, the workgroup polls only the slot `sentinel` (written about last)
// until it is in, so that a waiting workgroup adds little traffic, and then
// loads until every share is in (bounded).  In a launch small enough that
// the traffic does not matter (A.full_poll) every share is polled on each
// round instead, which saves that last round trip.  False (in every thread)
// when a wait timed out: the loaded values are then not this launch's.
template <class F>
DEV bool load_tagged(const KArgs& A, const uint64_t* sentinel, F&& load) {
  if (__syncthreads_and(load())) return true;
  if (!A.full_poll && !wait_one(sentinel, A)) return false;
  BlockPoll bp;
  while (!bp.done(load(), A)) {
  }
  return !bp.timed_out;
}

// The fp64 value in the tagged slot pair at p (low word first); both loads
// go out together, and the pair is polled until both carry the epoch.  ok is
// cleared when the wait timed out.
DEV double wait_pair(const uint64_t* p, const KArgs& A, bool& ok) {
  uint64_t lo = ld_tag(p), hi = ld_tag(p + 1);
  Poll pl;
  while (!(tag_ok(lo, A.epoch) && tag_ok(hi, A.epoch))) {
    if (!pl.again(A)) {
      ok = false;
      break;
    }
    lo = ld_tag(p);
    hi = ld_tag(p + 1);
  }
  return payd(lo, hi);
}

// The fp32 value in the tagged slot at p, polled until it carries the
// epoch; ok is cleared when the wait timed out.
DEV float wait_f32(const uint64_t* p, const KArgs& A, bool& ok) {
  uint64_t v = ld_tag(p);
  Poll pl;
  while (!tag_ok(v, A.epoch)) {
    if (!pl.again(A)) {
      ok = false;
      break;
    }
    v = ld_tag(p);
  }
  return payf(v);
}

// Poll a tagged slot until it carries the launch epoch (bounded).
DEV uint64_t wait_tag(const uint64_t* p, const KArgs& A) {
  uint64_t v = ld_tag(p);
  Poll pl;
  while (!tag_ok(v, A.epoch) && pl.again(A)) v = ld_tag(p);
  return v;
}

DEV __amdgpu_buffer_rsrc_t make_rsrc(const void* base, unsigned long long nbytes) {
  const unsigned long long n = nbytes > 0xFFFFFFFFull ? 0xFFFFFFFFull : nbytes;
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)(uint32_t)n, 0x00020000);
}
// 16-byte load through a buffer resource: bytes at or past the resource's
// size read as zero without touching memory.
DEV u4 buf_load(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, 0);
}
// Streaming read of logits: the non-temporal cache policy (nt), which keeps
// the once-read lines from displacing others and measurably raises the read
// rate of the whole-chip sweep.
#ifndef ASYMSPEC_AUX_NT
#define ASYMSPEC_AUX_NT 2
#endif
constexpr int kAuxNT = ASYMSPEC_AUX_NT;
DEV u4 buf_load_nt(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, kAuxNT);
}

// ------------------------------------------------------------------ decode
template <int DT> struct Elem;
template <> struct Elem<ASYMSPEC_BF16> {
  static constexpr int VE = 8;
  DEV static float get(const u4& v, int e) {
    const uint32_t w = v[e >> 1];
    return __uint_as_float((e & 1) ? (w & 0xFFFF0000u) : (w << 16));
  }
  DEV static float load_one(const void* base, long long idx) {
    const uint32_t h = reinterpret_cast<const uint16_t*>(base)[idx];
    return __uint_as_float(h << 16);
  }
  DEV static void mask_to_neginf(u4& v, int lo, int hi) {
    #pragma unroll
    for (int j = 0; j < 4; ++j) {
      uint32_t w = v[j];
      if (2 * j < lo || 2 * j >= hi) w = (w & 0xFFFF0000u) | kBf16NegInf;
      if (2 * j + 1 < lo || 2 * j + 1 >= hi) w = (w & 0x0000FFFFu) | (kBf16NegInf << 16);
      v[j] = w;
    }
  }
  DEV static void put_one(u4& v, int e, float x) {
    const uint32_t h = __float_as_uint(x) >> 16;
    v[e >> 1] |= (e & 1) ? (h << 16) : h;
  }
};
template <> struct Elem<ASYMSPEC_FP32> {
  static constexpr int VE = 4;
  DEV static float get(const u4& v, int e) { return __uint_as_float(v[e]); }
  DEV static float load_one(const void* base, long long idx) {
    return reinterpret_cast<const float*>(base)[idx];
  }
  DEV static void mask_to_neginf(u4& v, int lo, int hi) {
    #pragma unroll
    for (int j = 0; j < 4; ++j)
      if (j < lo || j >= hi) v[j] = kF32NegInf;
  }
  DEV static void put_one(u4& v, int e, float x) { v[e] = __float_as_uint(x); }
};

// Fused logit of Eq. 2 in fp32: t + beta * (a - b), in that order, no
// contraction.  A NaN (a = b = -inf) stays NaN here; consumers treat it as a
// masked token (maxima ignore it, exponent arguments are clamped).
// Sources of the context-gain signal: delta = a - b (Eq. 1), or the
// mechanism ablation's delta = a (raw-augmented) and delta = t - b
// (SCD-style).  The values match the public ASYMSPEC_DELTA_* constants.
enum { kDeltaAB = 0, kDeltaA = 1, kDeltaTB = 2 };
template <int DM>
DEV float delta_of(float t, float a, float b) {
  if (DM == kDeltaA) return a;
  if (DM == kDeltaTB) return __fsub_rn(t, b);
  return __fsub_rn(a, b);
}
// f = fl(t + fl(beta * delta)), in this order and without contraction.
template <int DM>
DEV float fuse(float t, float a, float b, float beta) {
  return __fadd_rn(t, __fmul_rn(beta, delta_of<DM>(t, a, b)));
}
// beta = 1: fl(1 * x) = x, so this is bit-identical to fuse<DM>(t, a, b, 1).
template <int DM>
DEV float fuse1(float t, float a, float b) { return __fadd_rn(t, delta_of<DM>(t, a, b)); }
// The same with the source chosen at run time (the resolve items): the
// identical operations, so bit-identical to fuse<DM>.
DEV float fuse_rt(float t, float a, float b, float beta, int dm) {
  const float d = dm == kDeltaA ? a : (dm == kDeltaTB ? __fsub_rn(t, b) : __fsub_rn(a, b));
  return __fadd_rn(t, __fmul_rn(beta, d));
}
DEV float fuse_masked(float t, float a, float b, float beta, int dm) {
  const float f = fuse_rt(t, a, b, beta, dm);
  return (f != f) ? -INFINITY : f;
}

// ------------------------------------------------------------- reductions
// Wave64 reductions with gfx9 DPP patterns (xor-1 and xor-2 quad
// permutations, half-row and row mirrors, row_bcast15 and row_bcast31); the
// result lands in lane 63 and is read back as a wave-uniform value.  All 64
// lanes must be active.
template <int CTRL, int ROWMASK = 0xF>
DEV float dppf(float x) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(__builtin_bit_cast(int, x),
                                                              __builtin_bit_cast(int, x),
                                                              CTRL, ROWMASK, 0xF, false));
}
template <int CTRL, int ROWMASK = 0xF>
DEV int dppi(int x) {
  return __builtin_amdgcn_update_dpp(x, x, CTRL, ROWMASK, 0xF, false);
}
DEV float lane63f(float x) {
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, x), 63));
}
DEV float wave_max(float x) {
  x = fmaxf(x, dppf<0xB1>(x));
  x = fmaxf(x, dppf<0x4E>(x));
  x = fmaxf(x, dppf<0x141>(x));
  x = fmaxf(x, dppf<0x140>(x));
  x = fmaxf(x, dppf<0x142, 0xA>(x));
  x = fmaxf(x, dppf<0x143, 0xC>(x));
  return lane63f(x);
}
DEV float wave_sum(float x) {
  x += dppf<0xB1>(x);
  x += dppf<0x4E>(x);
  x += dppf<0x141>(x);
  x += dppf<0x140>(x);
  x += dppf<0x142, 0xA>(x);
  x += dppf<0x143, 0xC>(x);
  return lane63f(x);
}
DEV int wave_min_i(int x) {
  x = min(x, dppi<0xB1>(x));
  x = min(x, dppi<0x4E>(x));
  x = min(x, dppi<0x141>(x));
  x = min(x, dppi<0x140>(x));
  x = min(x, dppi<0x142, 0xA>(x));
  x = min(x, dppi<0x143, 0xC>(x));
  return __builtin_amdgcn_readlane(x, 63);
}
// DPP move of both halves of an fp64 value; lanes whose source is outside
// the pattern (or in a row that ROWMASK leaves out) read 0.
template <int CTRL, int ROWMASK = 0xF>
DEV double dpp_d0(double x) {
  const uint64_t b = __builtin_bit_cast(uint64_t, x);
  const int lo = __builtin_amdgcn_update_dpp(0, (int)(uint32_t)b, CTRL, ROWMASK, 0xF, false);
  const int hi = __builtin_amdgcn_update_dpp(0, (int)(uint32_t)(b >> 32), CTRL, ROWMASK, 0xF, false);
  return __builtin_bit_cast(double, (uint64_t)(uint32_t)lo | ((uint64_t)(uint32_t)hi << 32));
}
// Reductions over the 16 lanes of each DPP row (lanes 16r .. 16r + 15),
// the result in every lane of the row: rotations by 8, 4, 2 and 1 lanes
// within the row.
template <int N>
DEV int ror16_i(int x) { return __builtin_amdgcn_update_dpp(x, x, 0x120 + N, 0xF, 0xF, false); }
template <int N>
DEV double ror16_d(double x) {
  const uint64_t b = __builtin_bit_cast(uint64_t, x);
  const uint32_t lo = (uint32_t)ror16_i<N>((int)(uint32_t)b);
  const uint32_t hi = (uint32_t)ror16_i<N>((int)(uint32_t)(b >> 32));
  return __builtin_bit_cast(double, (uint64_t)lo | ((uint64_t)hi << 32));
}
DEV float row16_max(float x) {
  x = fmaxf(x, __int_as_float(ror16_i<8>(__float_as_int(x))));
  x = fmaxf(x, __int_as_float(ror16_i<4>(__float_as_int(x))));
  x = fmaxf(x, __int_as_float(ror16_i<2>(__float_as_int(x))));
  return fmaxf(x, __int_as_float(ror16_i<1>(__float_as_int(x))));
}
DEV int row16_min(int x) {
  x = min(x, ror16_i<8>(x));
  x = min(x, ror16_i<4>(x));
  x = min(x, ror16_i<2>(x));
  return min(x, ror16_i<1>(x));
}
DEV int row16_or(int x) {
  x |= ror16_i<8>(x);
  x |= ror16_i<4>(x);
  x |= ror16_i<2>(x);
  return x | ror16_i<1>(x);
}
DEV double row16_sum(double x) {
  x += ror16_d<8>(x);
  x += ror16_d<4>(x);
  x += ror16_d<2>(x);
  return x + ror16_d<1>(x);
}

// An fp64 value of one lane, in every lane.
DEV double readlane_d(double x, int lane) {
  const uint64_t b = __builtin_bit_cast(uint64_t, x);
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)b, lane);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(b >> 32), lane);
  return __builtin_bit_cast(double, (uint64_t)lo | ((uint64_t)hi << 32));
}
// Inclusive and exclusive prefix sums of an fp64 value over the lanes of a
// wave, in lane order: row shifts by 1, 2, 4 and 8 within each row of 16
// lanes, then row 0's total into row 1 and row 2's into row 3 (row_bcast15),
// then rows 0-1 into rows 2-3 (row_bcast31); the exclusive sum is the
// inclusive one shifted by a lane (wave_shr1).  All 64 lanes must be active.
DEV void wave_scan_d(double x, double& incl, double& excl) {
  x += dpp_d0<0x111>(x);
  x += dpp_d0<0x112>(x);
  x += dpp_d0<0x114>(x);
  x += dpp_d0<0x118>(x);
  x += dpp_d0<0x142, 0xA>(x);
  x += dpp_d0<0x143, 0xC>(x);
  incl = x;
  excl = dpp_d0<0x138>(x);
}
DEV double wave_sum_d(double x) {    // fp64 sum over lanes, in every lane
  #pragma unroll
  for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o, 64);
  return x;
}

// ---------------------------------------------------- online log-sum-exp
// Running (reference R, sum s of exp2(x * c - R)), one vector of VE elements
// at a time.  acc_vec keeps R = fl(m * c) for the running maximum m; with
// kTrackArg, pos = k of the first vector (in this thread's order) that
// attains it (the element inside it is found afterwards).  acc_vec_lazy
// keeps R where it is while no term exceeds 2^64, which saves the maxima of
// every vector; any R at or below the maximum gives the same normaliser.
struct Acc { float m, R, s; int pos; };
DEV void acc_init(Acc& q, float c) { q.m = kFloorM; q.R = kFloorM * c; q.s = 0.0f; q.pos = 0; }

template <int VE, bool kClampNaN, bool kTrackArg>
DEV void acc_vec(Acc& q, const float (&x)[VE], float c, int k) {
  float vm = x[0];
  #pragma unroll
  for (int e = 1; e < VE; ++e) vm = fmaxf(vm, x[e]);
  if (kTrackArg) q.pos = vm > q.m ? k : q.pos;
  const float mn = fmaxf(q.m, vm);
  const float Rn = mn * c;
  const float scale = __builtin_amdgcn_exp2f(q.R - Rn);
  float ex[VE];
  #pragma unroll
  for (int e = 0; e < VE; ++e) {
    float arg = __builtin_fmaf(x[e], c, -Rn);
    if (kClampNaN) arg = fmaxf(arg, -200.0f);
    ex[e] = __builtin_amdgcn_exp2f(arg);
  }
  #pragma unroll
  for (int st = 1; st < VE; st <<= 1)
    #pragma unroll
    for (int e = 0; e + st < VE; e += 2 * st) ex[e] += ex[e + st];
  q.s = __builtin_fmaf(q.s, scale, ex[0]);
  q.m = mn;
  q.R = Rn;
}

// Lazy step: the terms at the current reference; only when some lane's
// vector sum exceeds 2^64 (or overflows) does the wave raise those lanes'
// references to their vector maxima and redo the vector.  A NaN sum is left
// to the caller (the chunk is then redone on the NaN-safe path).
template <int VE, bool kClampNaN>
DEV void acc_vec_lazy(Acc& q, const float (&x)[VE], float c) {
  float ex[VE];
  #pragma unroll
  for (int e = 0; e < VE; ++e) {
    float arg = __builtin_fmaf(x[e], c, -q.R);
    if (kClampNaN) arg = fmaxf(arg, -200.0f);
    ex[e] = __builtin_amdgcn_exp2f(arg);
  }
  #pragma unroll
  for (int st = 1; st < VE; st <<= 1)
    #pragma unroll
    for (int e = 0; e + st < VE; e += 2 * st) ex[e] += ex[e + st];
  float v = ex[0];
  if (__builtin_expect(__ballot(v > 0x1p64f) != 0, 0)) {
    float vm = x[0];
    #pragma unroll
    for (int e = 1; e < VE; ++e) vm = fmaxf(vm, x[e]);
    const float Rn = fmaxf(q.R, vm * c);
    const float scale = __builtin_amdgcn_exp2f(q.R - Rn);
    #pragma unroll
    for (int e = 0; e < VE; ++e) {
      float arg = __builtin_fmaf(x[e], c, -Rn);
      if (kClampNaN) arg = fmaxf(arg, -200.0f);
      ex[e] = __builtin_amdgcn_exp2f(arg);
    }
    #pragma unroll
    for (int st = 1; st < VE; st <<= 1)
      #pragma unroll
      for (int e = 0; e + st < VE; e += 2 * st) ex[e] += ex[e + st];
    v = ex[0];
    q.s *= scale;
    q.R = Rn;
  }
  q.s += v;
}

// The same two steps for the A slot of calls with the KL gate, which also
// keep W = sum of exp2(x * c - R) d, d = a - b with -inf (a token the full
// view masks, whose term is 0) raised to -FLT_MAX so that 0 * d stays 0.
template <int VE, bool kFirst>
DEV void acc_vec_w(Acc& q, float& W, const float (&x)[VE], const float (&d)[VE], float c) {
  float ex[VE];
  float R = q.R;
  if (kFirst) {
    float vm = x[0];
    #pragma unroll
    for (int e = 1; e < VE; ++e) vm = fmaxf(vm, x[e]);
    q.m = fmaxf(q.m, vm);
    R = q.m * c;
  }
  #pragma unroll
  for (int e = 0; e < VE; ++e) ex[e] = __builtin_amdgcn_exp2f(__builtin_fmaf(x[e], c, -R));
  float v = ex[0], w = ex[0] * fmaxf(d[0], -FLT_MAX);
  #pragma unroll
  for (int e = 1; e < VE; ++e) {
    v += ex[e];
    w = __builtin_fmaf(ex[e], fmaxf(d[e], -FLT_MAX), w);
  }
  if (!kFirst && __builtin_expect(__ballot(v > 0x1p64f) != 0, 0)) {
    float vm = x[0];
    #pragma unroll
    for (int e = 1; e < VE; ++e) vm = fmaxf(vm, x[e]);
    R = fmaxf(q.R, vm * c);
    #pragma unroll
    for (int e = 0; e < VE; ++e) ex[e] = __builtin_amdgcn_exp2f(__builtin_fmaf(x[e], c, -R));
    v = ex[0];
    w = ex[0] * fmaxf(d[0], -FLT_MAX);
    #pragma unroll
    for (int e = 1; e < VE; ++e) {
      v += ex[e];
      w = __builtin_fmaf(ex[e], fmaxf(d[e], -FLT_MAX), w);
    }
  }
  if (R != q.R) {
    const float scale = __builtin_amdgcn_exp2f(q.R - R);
    q.s *= scale;
    W *= scale;
    q.R = R;
  }
  q.s += v;
  W += w;
}

// --------------------------------------------------- pass-2 element terms
// Shared by pass 2 and the emission scan so that both see identical values.
struct ResidConst { float beta, c, Rf, isf, Rq, isq; };
// max(0, p~(x) - q(x)) with p~ = softmax(f / tau), q = softmax(a / tau).  A
// NaN fused logit (a masked token) gives p = NaN and max(NaN, 0) = 0.
template <int DM>
DEV float resid_elem(float t, float a, float b, const ResidConst& k) {
  const float f = fuse<DM>(t, a, b, k.beta);
  const float p = __builtin_amdgcn_exp2f(__builtin_fmaf(f, k.c, -k.Rf)) * k.isf;
  const float q = __builtin_amdgcn_exp2f(__builtin_fmaf(a, k.c, -k.Rq)) * k.isq;
  return fmaxf(p - q, 0.0f);
}
// Unnormalised bonus weight exp2(t * c - R_t) of softmax(t / tau).
DEV float bonus_elem(float t, float c, float Rt) {
  return __builtin_amdgcn_exp2f(__builtin_fmaf(t, c, -Rt));
}
// JSD term P log2(2P/(P+Q)) + Q log2(2Q/(P+Q)) with P = softmax(a), Q =
// softmax(b) (Eq. 3), from log2 P and log2 Q.
struct JsdConst { float Ra, Rb, kahi, kalo, kbhi, kblo; };
DEV float jsd_elem(float a, float b, const JsdConst& k) {
  const float lp = (fmaxf(__builtin_fmaf(a, kL2E, -k.Ra), kFloorM) - k.kahi) - k.kalo;
  const float lq = (fmaxf(__builtin_fmaf(b, kL2E, -k.Rb), kFloorM) - k.kbhi) - k.kblo;
  const float P = __builtin_amdgcn_exp2f(lp);
  const float Q = __builtin_amdgcn_exp2f(lq);
  const float g = 1.0f - __builtin_amdgcn_logf(fmaxf(P + Q, 1e-37f));
  return __builtin_fmaf(P, lp + g, Q * (lq + g));
}
// log2 of a positive double to ~1e-7 absolute: exact exponent split plus the
// hardware log2 of the mantissa.
DEV double log2_dbl(double x) {
  int e;
  const double m = frexp(x, &e);
  return (double)e + (double)__builtin_amdgcn_logf((float)m);
}
DEV double ln_f(float x) { return (double)__builtin_amdgcn_logf(x) * kLn2; }

// ----------------------------------------------------------- row geometry
struct RowGeo {
  int row, req, pos, kind;
  float tau, c;               // c = log2(e) / tau when sampling, log2(e) when greedy
  long long e0;               // flat index of the row's first element
  long long vbeg, vend;       // the row's 16-byte vector range (vend exclusive)
};

DEV float sload_f32(const void* base, long long idx) {
  return __uint_as_float(((cptr32)base)[idx]);
}

// The geometry of a row without its temperature (kind and c unset): for
// the items that only address the row, so that no load of tau stands
// before their first memory access.
template <int DT>
DEV RowGeo row_span(const KArgs& A, int row) {
  constexpr int VE = Elem<DT>::VE;
  RowGeo g;
  g.row = row;
  g.req = row / (A.K + 1);
  g.pos = row - g.req * (A.K + 1);
  g.tau = 0.0f;
  g.kind = -1;
  g.c = 0.0f;
  g.e0 = (long long)row * A.V;
  g.vbeg = g.e0 / VE;
  g.vend = (g.e0 + A.V + VE - 1) / VE;
  return g;
}

template <int DT>
DEV RowGeo row_geo(const KArgs& A, int row) {
  constexpr int VE = Elem<DT>::VE;
  RowGeo g;
  g.row = row;
  g.req = row / (A.K + 1);
  g.pos = row - g.req * (A.K + 1);
  g.tau = sload_f32(A.tau, g.req);
  const bool samp = g.tau > 0.0f;
  const bool bonus = g.pos == A.K;
  if (bonus && A.fuse_bonus) g.kind = samp ? kSampleBonusF : kGreedyBonusF;
  else if (bonus) g.kind = samp ? kSampleBonus : kGreedyBonus;
  else g.kind = samp ? (g.tau == 1.0f ? kSampleDraft1 : kSampleDraftT) : kGreedyDraft;
  g.c = samp ? (kL2E / g.tau) : kL2E;
  g.e0 = (long long)row * A.V;
  g.vbeg = g.e0 / VE;
  g.vend = (g.e0 + A.V + VE - 1) / VE;
  return g;
}
DEV bool kind_draft(int k) { return k == kGreedyDraft || k == kSampleDraft1 || k == kSampleDraftT; }
DEV bool kind_samp(int k) {
  return k == kSampleDraft1 || k == kSampleDraftT || k == kSampleBonus || k == kSampleBonusF;
}
// Rows whose statistics are those of the fused logits f (slot sF).
DEV bool kind_fused(int k) { return kind_draft(k) || k == kGreedyBonusF || k == kSampleBonusF; }

// Buffer resource over one stream's vectors of row g, clamped to the array
// end: vectors past the row (or the array) read as zero.
DEV __amdgpu_buffer_rsrc_t row_rsrc(const KArgs& A, const void* base, const RowGeo& g) {
  const unsigned long long rbase = (unsigned long long)g.vbeg * 16ull;
  unsigned long long span = (unsigned long long)(g.vend - g.vbeg) * 16ull;
  // a row past the array's end (never for a valid row index) reads nothing
  const unsigned long long rem = rbase < A.stream_bytes ? A.stream_bytes - rbase : 0ull;
  if (span > rem) span = rem;
  // drafter rows of another vocabulary are reached through the map only:
  // a resource over them reads zeros and touches no memory
  if (A.vmap != nullptr && base != A.t) span = 0;
  return make_rsrc((const char*)base + rbase, span);
}

// Elements of the vector at index vi that lie outside the row become -inf
// (branch-free: selects only).
template <int DT>
DEV void mask_vec(const KArgs& A, const RowGeo& g, long long vi, u4& v) {
  constexpr int VE = Elem<DT>::VE;
  const long long lo = g.e0 - vi * VE;
  const long long hi = lo + A.V;
  const int ilo = (int)(lo < 0 ? 0 : (lo > VE ? VE : lo));
  const int ihi = (int)(hi < 0 ? 0 : (hi > VE ? VE : hi));
  Elem<DT>::mask_to_neginf(v, ilo, ihi);
}
// True when the vector range [v0, v1) of row g holds the partial 16-byte
// vector at the end of an array whose size is not a multiple of 16 bytes.
DEV bool has_tail(const KArgs& A, long long v0, long long v1) {
  if (A.stream_bytes % 16ull == 0) return false;
  const long long last_full = (long long)(A.stream_bytes / 16ull);
  return v0 <= last_full && last_full < v1;
}

// Repair one loaded vector of stream `src` at vector index vi: the vector
// holding the last bytes of an array whose size is not a multiple of 16 is
// re-read element by element, then elements outside the row become -inf.
template <int DT>
DEV void fix_vec(const KArgs& A, const RowGeo& g, const void* src, long long vi, u4& v) {
  constexpr int VE = Elem<DT>::VE;
  constexpr int ES = 16 / VE;
  if (A.vmap != nullptr && src != A.t) return;   // drafter rows: map_vecs
  const long long last_full = (long long)(A.stream_bytes / 16ull);
  if (vi >= last_full && vi < g.vend) {
    const long long n_el = (long long)(A.stream_bytes / ES);
    u4 r = {0, 0, 0, 0};
    #pragma unroll
    for (int e = 0; e < VE; ++e) {
      const long long idx = vi * VE + e;
      if (idx < n_el) Elem<DT>::put_one(r, e, Elem<DT>::load_one(src, idx));
    }
    v = r;
  }
  const long long first = vi * VE;
  const long long lo = g.e0 - first;
  const long long hi = g.e0 + A.V - first;
  if (lo > 0 || hi < VE) {
    const int ilo = (int)(lo < 0 ? 0 : (lo > VE ? VE : lo));
    const int ihi = (int)(hi < 0 ? 0 : (hi > VE ? VE : hi));
    Elem<DT>::mask_to_neginf(v, ilo, ihi);
  }
}

// Cross-family vocabularies (the alignment of App. "Cross-family
// portability"): the drafter logits of verifier token x are a[vmap[x]] and
// b[vmap[x]]; a verifier token without a shared counterpart cannot be
// committed, so it counts as masked in every view (t = a = b = -inf).
DEV int map_id(const KArgs& A, long long x) {
  if (x < 0 || x >= A.V) return -1;
  const int j = A.vmap[x];
  return (j >= 0 && j < A.Vd) ? j : -1;
}
// The vector vi of row g in the verifier's layout: vt (loaded and repaired)
// gets -inf where the token is not shared, and, when ab, va and vb are
// gathered from the drafter rows through the map (-inf where not shared).
template <int DT>
DEV void map_vecs(const KArgs& A, const RowGeo& g, long long vi, u4& vt, u4& va, u4& vb, bool ab) {
  constexpr int VE = Elem<DT>::VE;
  u4 t2 = {0, 0, 0, 0}, a2 = t2, b2 = t2;
  const long long dbase = (long long)g.row * A.Vd;
  #pragma unroll
  for (int e = 0; e < VE; ++e) {
    const int j = map_id(A, vi * VE + e - g.e0);
    float xt = -INFINITY, xa = -INFINITY, xb = -INFINITY;
    if (j >= 0) {
      xt = Elem<DT>::get(vt, e);
      if (ab) {
        xa = Elem<DT>::load_one(A.a, dbase + j);
        xb = Elem<DT>::load_one(A.b, dbase + j);
      }
    }
    Elem<DT>::put_one(t2, e, xt);
    Elem<DT>::put_one(a2, e, xa);
    Elem<DT>::put_one(b2, e, xb);
  }
  vt = t2;
  if (ab) { va = a2; vb = b2; }
}
// True when the drafter-to-verifier map of this call is usable (every shared
// drafter id belongs to one verifier token).  Wave-uniform.
DEV bool inv_ok(const KArgs& A) {
  return A.inv != nullptr && ((cptr32)(const void*)A.inv)[A.Vd] == 0u;
}

// The three logits of verifier token x (0 <= x < V) of row g, mapped.
template <int DT>
DEV void mapped_tab(const KArgs& A, const RowGeo& g, int x, float& t, float& a, float& b) {
  const int j = A.vmap != nullptr ? map_id(A, x) : ((x >= 0 && x < A.V) ? x : -1);
  if (j < 0) {
    t = a = b = -INFINITY;
    return;
  }
  t = Elem<DT>::load_one(A.t, g.e0 + x);
  const long long d = A.vmap != nullptr ? (long long)g.row * A.Vd + j : g.e0 + x;
  a = Elem<DT>::load_one(A.a, d);
  b = Elem<DT>::load_one(A.b, d);
}

// Draft-token gathers of one row through the scalar cache (wave-uniform
// addresses into inputs the kernel never writes).
struct Gather { float t, a, b, p, u; };

template <int DT>
DEV float sload_elem(const void* base, long long idx) {
  if (DT == ASYMSPEC_BF16) {
    const uint32_t w = ((cptr32)base)[idx >> 1];
    return __uint_as_float((idx & 1) ? (w & 0xFFFF0000u) : (w << 16));
  }
  return __uint_as_float(((cptr32)base)[idx]);
}

// The draft token's logits and the caller's proposal probability and
// uniform for draft row g (g.pos < K); a bonus row gets neutral values.
template <int DT>
DEV Gather sgather(const KArgs& A, const RowGeo& g) {
  Gather q{0.0f, 0.0f, 0.0f, 1.0f, 0.0f};
  if (g.pos < A.K) {
    int dtok = (int)((cptr32)(const void*)A.d)[g.req * A.K + g.pos];
    dtok = dtok < 0 ? 0 : (dtok >= A.V ? A.V - 1 : dtok);
    const long long idx = g.e0 + dtok;
    if (A.vmap != nullptr) {
      // a draft outside the shared set has no mass in any view
      const int j = ((cptr32)(const void*)A.vmap)[dtok];
      if (j >= 0 && j < A.Vd) {
        const long long di = (long long)g.row * A.Vd + j;
        q.t = sload_elem<DT>(A.t, idx);
        q.a = sload_elem<DT>(A.a, di);
        q.b = sload_elem<DT>(A.b, di);
      } else {
        q.t = q.a = q.b = -INFINITY;
      }
    } else {
      q.t = sload_elem<DT>(A.t, idx);
      q.a = sload_elem<DT>(A.a, idx);
      q.b = sload_elem<DT>(A.b, idx);
    }
    if (A.dp != nullptr) q.p = sload_f32(A.dp, (long long)g.req * A.K + g.pos);
    q.u = sload_f32(A.u, (long long)g.req * (A.K + 1) + g.pos);
  }
  return q;
}

// --------------------------------------------------------- shared memory
struct Smem {
  // statistics item: per-wave partials
  float wm[kWaves][kSlots];
  float ws[kWaves][kSlots];
  int warg[kWaves];
  int wneq[kWaves];
  float wmarg[kWaves];
  float wkl[kWaves];
  // decision of a request: per-row blocks, request words, and the
  // per-(row, chunk) values the decide item combines into them
  uint32_t rows[kMaxK + 1][kDecRow];
  uint32_t req[kReqWords];
  float dm[kThreads][kSlots];
  float dmarg[kThreads];
  double dw[kThreads];
  double dt[kThreads][kSlots];
  int darg[kThreads];
  int dneq[kThreads];
  // pass 2 / pick: partials, scans
  float wj[kWaves];
  int flags[8];
  double dd[8];
  double djsd[kMaxK + 1];   // pick: D of the rows with a JSD task
  double scan[kWaves];
  int imin[kWaves];
#ifdef ASYMSPEC_TRACE
  uint64_t t_mark[2];   // measurement builds: first streaming load, end of the stream
#endif
};

// Inclusive and exclusive prefix sums over the workgroup, in thread order.
DEV void block_scan(double x, Smem& sm, double& incl, double& excl) {
  const int lane = lane_id(), w = wave_id();
  double v = x;
  #pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const double y = __shfl_up(v, o, 64);
    if (lane >= o) v += y;
  }
  double prev = __shfl_up(v, 1, 64);
  if (lane == 0) prev = 0.0;
  __syncthreads();
  if (lane == 63) sm.scan[w] = v;
  __syncthreads();
  double off = 0.0;
  for (int i = 0; i < w; ++i) off += sm.scan[i];
  incl = off + v;
  excl = off + prev;
}
DEV int block_min_i(int x, Smem& sm) {
  const int lane = lane_id(), w = wave_id();
  x = wave_min_i(x);
  __syncthreads();
  if (lane == 0) sm.imin[w] = x;
  __syncthreads();
  int r = sm.imin[0];
  #pragma unroll
  for (int i = 1; i < kWaves; ++i) r = min(r, sm.imin[i]);
  return r;
}

}  // namespace asym

#endif  // ASYMSPEC_DEVICE_H_
