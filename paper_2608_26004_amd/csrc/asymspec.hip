// AsymSpec fused decision step for MI355X (gfx950, CDNA4, wave64).
//
// One persistent cooperative launch does the whole step of Alg. 1 for every
// request: the vocabulary-wide statistics of the verifier logits t and the
// drafter logits a (full view) and b (compressed view), the delta-fused logits
// f = t + beta (a - b) (Sec. 3.2, Eq. 1-2), the Jensen-Shannon divergence D and
// the CDA gate gamma * exp(-D) (Sec. 3.3, Eq. 3), the acceptance test (Eq. 4,
// or its speculative-sampling form for temperature > 0), and the emission at
// the first rejection or the bonus token.
//
// Work decomposition.  A logit row [V] is cut into S chunks of
// kThreads * NV 16-byte vectors.  A team of S workgroups owns a sequence of
// rows; member m always takes chunk m.  Each workgroup runs a two-stage row
// pipeline; iteration i
//   * prefetches the tile of row i+1 into registers,
//   * runs pass 1 on the tile of row i: per-chunk max / sum-exp statistics
//     of t, a, b and f, the fused-logit argmax and an a-vs-b bitwise flag,
//     and publishes them as an epoch-tagged record;
//   * combines the S records of row i-1 (published one iteration ago, so the
//     team barrier rarely waits) and classifies that row as surely accepted,
//     surely rejected or open, using D in [0, ln 2];
//   * runs pass 2 of row i-1 on its tile, stashed in LDS, only where needed:
//     the JSD term (open rows, or when the caller asks for D) and per-wave
//     sums of the residual max(0, p~ - q) (sampling rows that may reject) or
//     of the bonus weights;
//   * settles row i-1 (or, when it needed D, row i-2 from its JSD partials);
//   * stashes the tile of row i in LDS.
// After the last row each workgroup runs the request epilogues assigned to
// it: accept_len, the inverse-CDF scan of one wave segment for sampled
// emissions, and the outputs.
//
// Cross-workgroup records are arrays of 64-bit slots whose high word is the
// launch epoch and low word a payload, written and read with relaxed
// agent-scope atomics (sc1, no cache flushes).  An aligned 64-bit atomic is
// single-copy atomic, so a reader that sees the epoch in a slot sees its
// payload; writers never wait, readers poll until every slot they need is in.

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

#define DEV __device__ __forceinline__

namespace asym {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
constexpr float kL2E = 1.44269504088896340736f;
constexpr double kLn2 = 0.693147180559945309417232121458;
constexpr float kFloorM = -1.0e30f;            // start value of running maxima
constexpr uint32_t kBf16NegInf = 0xFF80u;
constexpr uint32_t kF32NegInf = 0xFF800000u;
constexpr long kSpinLimit = 1L << 20;          // bounded polls (tens of ms)

typedef uint32_t u4 __attribute__((ext_vector_type(4)));
typedef const __attribute__((address_space(4))) uint32_t* cptr32;

enum Kind { kGreedyDraft = 0, kSampleDraft = 1, kGreedyBonus = 2, kSampleBonus = 3 };
enum Slot { sT = 0, sA = 1, sB = 2, sF = 3, sAT = 4, kSlots = 5 };
// What a team knows, at a row, about the earlier drafts of the same request
// it processed: all accepted so far, some still open (waiting for D), or one
// surely rejected.
enum { kReqOpen = 0, kReqUnknown = 1, kReqRejected = 2 };


constexpr int kR1 = 16;   // pass-1 chunk record slots (12 used)
constexpr int kR2 = 12;   // pass-2 chunk record slots (10 used)
constexpr int kRW = 16;   // settled-row record slots (14 used)

// pass-1 record payloads: M[5] (fp32 max), S[5] (fp32 sum-exp relative to
// fl(M * c)), argmax, a-vs-b flag
enum { P1_M = 0, P1_S = 5, P1_ARG = 10, P1_NEQ = 11, P1_USED = 12 };

struct KArgs {
  const void* t; const void* a; const void* b;
  const int32_t* d; const float* dp; const float* u; const float* tau;
  int32_t* acc_out; int32_t* next_out; float* flp_out; float* gate_out;
  uint64_t* rec1; uint64_t* rec2; uint64_t* rowres;
  uint32_t* err;
  unsigned long long stream_bytes;   // bytes of each logit array
  int B, K, V, S, n_teams, rows, grid;
  float beta, gamma; int gate_mode; int want_gate;
  double ln_gamma;
  uint32_t epoch;
};

// ------------------------------------------------------------------ memory
DEV void st_tag(uint64_t* p, uint32_t v, uint32_t ep) {
  __hip_atomic_store(p, ((uint64_t)ep << 32) | (uint64_t)v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
DEV uint64_t ld_tag(const uint64_t* p) {
  return __hip_atomic_load(const_cast<uint64_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
DEV bool tag_ok(uint64_t v, uint32_t ep) { return (uint32_t)(v >> 32) == ep; }
DEV uint32_t pay(uint64_t v) { return (uint32_t)v; }
DEV float payf(uint64_t v) { return __uint_as_float((uint32_t)v); }
DEV double payd(uint64_t lo, uint64_t hi) {
  return __builtin_bit_cast(double, (uint64_t)(uint32_t)lo | ((uint64_t)(uint32_t)hi << 32));
}
DEV uint32_t dlo(double x) { return (uint32_t)__builtin_bit_cast(uint64_t, x); }
DEV uint32_t dhi(double x) { return (uint32_t)(__builtin_bit_cast(uint64_t, x) >> 32); }
DEV void err_count(const uint32_t* e) {
  __hip_atomic_fetch_add(const_cast<uint32_t*>(e), 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

DEV __amdgpu_buffer_rsrc_t make_rsrc(const void* base, unsigned long long nbytes) {
  unsigned long long n = nbytes > 0xFFFFFFFFull ? 0xFFFFFFFFull : nbytes;
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)(uint32_t)n, 0x00020000);
}
DEV u4 buf_load(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, 0);
}

// ------------------------------------------------------------------ decode
template <int DT> struct Elem;
template <> struct Elem<ASYMSPEC_BF16> {
  static constexpr int VE = 8;
  DEV static float get(const u4& v, int e) {
    uint32_t w = v[e >> 1];
    return __uint_as_float((e & 1) ? (w & 0xFFFF0000u) : (w << 16));
  }
  DEV static float load_one(const void* base, long long idx) {
    uint32_t h = reinterpret_cast<const uint16_t*>(base)[idx];
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
};

// Fused logit of Eq. 2 in fp32, t + beta * (a - b) in that order, no
// contraction.  A NaN (a = b = -inf) stays NaN here and is treated as masked
// by every consumer (max ignores it, exp arguments are clamped).
DEV float fuse(float t, float a, float b, float beta) {
  float d = __fsub_rn(a, b);
  return __fadd_rn(t, __fmul_rn(beta, d));
}
DEV float fuse_masked(float t, float a, float b, float beta) {
  float f = fuse(t, a, b, beta);
  return (f != f) ? -INFINITY : f;
}

// ------------------------------------------------------------- reductions

// ------------------------------------------------------------- reductions
// Wave64 reductions with gfx9 DPP patterns: xor-1 and xor-2 quad
// permutations, half-row and row mirrors, then row_bcast15 / row_bcast31.
// The complete result lands in lane 63 and is read back as a wave-uniform
// value.  Must be called with all 64 lanes active.
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
// fp64 wave sum over lanes (rare paths only).
DEV double wave_sum_d(double x) {
  #pragma unroll
  for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o, 64);
  return x;
}

// ----------------------------------------------------------- row geometry
struct RowGeo {
  int row, req, pos, kind;
  float tau, c;               // c = log2(e) / tau for sampling, log2(e) for greedy
  long long e0;               // flat index of the row's first element
  long long vbeg, vend;       // row's 16-B vector range (vend exclusive)
};

DEV float sload_f32(const void* base, long long idx) {
  return __uint_as_float(((cptr32)base)[idx]);
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
  g.kind = bonus ? (samp ? kSampleBonus : kGreedyBonus) : (samp ? kSampleDraft : kGreedyDraft);
  g.c = samp ? (kL2E / g.tau) : kL2E;
  g.e0 = (long long)row * A.V;
  g.vbeg = g.e0 / VE;
  g.vend = (g.e0 + A.V + VE - 1) / VE;
  return g;
}
DEV bool is_draft(int kind) { return kind == kGreedyDraft || kind == kSampleDraft; }
DEV int n_streams(int kind) { return is_draft(kind) ? 3 : 1; }

// Issues this thread's vector loads of chunk `mem` of row g into buf: t, a
// and b for draft rows.  Every row issues the same number of loads (bonus
// rows point the a and b loads at the row's first 16 bytes), so the compiler
// can wait for a tile without waiting for the prefetch issued after it.
// Loads are bounds-checked by the buffer resource; the one vector that may
// run past the end of an array is repaired in sanitize().
template <int DT, int NV>
DEV void issue_loads(const KArgs& A, const RowGeo& g, int mem, u4 (&buf)[3][NV]) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const long long cv0 = g.vbeg + (long long)mem * (kThreads * NV) + (long long)w * (64 * NV);
  const unsigned long long rbase = (unsigned long long)g.vbeg * 16ull;
  const unsigned long long rem = A.stream_bytes - rbase;
  const bool draft = is_draft(g.kind);
  const __amdgpu_buffer_rsrc_t r0 = make_rsrc((const char*)A.t + rbase, rem);
  const __amdgpu_buffer_rsrc_t r1 = make_rsrc((const char*)(draft ? A.a : A.t) + rbase, rem);
  const __amdgpu_buffer_rsrc_t r2 = make_rsrc((const char*)(draft ? A.b : A.t) + rbase, rem);
  #pragma unroll
  for (int k = 0; k < NV; ++k) {
    const uint32_t off = (uint32_t)((cv0 + (long long)k * 64 + lane - g.vbeg) * 16);
    const uint32_t offab = draft ? off : 0u;
    buf[0][k] = buf_load(r0, off);
    buf[1][k] = buf_load(r1, offab);
    buf[2][k] = buf_load(r2, offab);
  }
}

// Replace elements outside [row start, row end) by -inf (a masked token).
// The vector holding the last bytes of an array, when the array size is not
// a multiple of 16 bytes, is re-read element by element first.
template <int DT, int NV>
DEV void sanitize(const RowGeo& g, const KArgs& A, int mem, u4 (&buf)[3][NV]) {
  constexpr int VE = Elem<DT>::VE;
  constexpr int ES = 16 / VE;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const long long cv0 = g.vbeg + (long long)mem * (kThreads * NV) + (long long)w * (64 * NV);
  const int ns = n_streams(g.kind);
  const long long last_full = (long long)(A.stream_bytes / 16ull);
  const long long n_el = (long long)(A.stream_bytes / ES);
  #pragma unroll
  for (int k = 0; k < NV; ++k) {
    const long long vi = cv0 + (long long)k * 64 + lane;
    if (vi >= last_full && vi < g.vend) {
      #pragma unroll
      for (int s = 0; s < 3; ++s) {
        if (s < ns) {
          const void* src = s == 0 ? A.t : (s == 1 ? A.a : A.b);
          u4 v = {0, 0, 0, 0};
          #pragma unroll
          for (int e = 0; e < VE; ++e) {
            const long long idx = vi * VE + e;
            if (idx < n_el) {
              const uint32_t bits = __float_as_uint(Elem<DT>::load_one(src, idx));
              if (DT == ASYMSPEC_BF16) {
                const uint32_t h = bits >> 16;
                v[e >> 1] |= (e & 1) ? (h << 16) : h;
              } else {
                v[e] = bits;
              }
            }
          }
          buf[s][k] = v;
        }
      }
    }
    const long long first = vi * VE;
    const long long lo = g.e0 - first;
    const long long hi = g.e0 + A.V - first;
    if (lo > 0 || hi < VE) {
      const int ilo = (int)(lo < 0 ? 0 : (lo > VE ? VE : lo));
      const int ihi = (int)(hi < 0 ? 0 : (hi > VE ? VE : hi));
      #pragma unroll
      for (int s = 0; s < 3; ++s)
        if (s < ns) Elem<DT>::mask_to_neginf(buf[s][k], ilo, ihi);
    }
  }
}

// Running (max, sum of exp2(x*c - R)) with R = fl(max * c), updated one
// vector at a time.  With kTrackArg, pos holds k * VE + e of the first
// element (in this thread's order) that attains the running maximum.
struct Acc { float m, R, s; int pos; };
DEV void acc_init(Acc& q, float c) { q.m = kFloorM; q.R = kFloorM * c; q.s = 0.0f; q.pos = 0; }

template <int VE, bool kClampNaN, bool kTrackArg = false>
DEV void acc_vec(Acc& q, const float (&x)[VE], float c, int k) {
  float vm = x[0];
  #pragma unroll
  for (int e = 1; e < VE; ++e) vm = fmaxf(vm, x[e]);
  if (kTrackArg) {
    int ei = VE - 1;
    #pragma unroll
    for (int e = VE - 2; e >= 0; --e) ei = (x[e] == vm) ? e : ei;
    if (vm > q.m) q.pos = k * VE + ei;
  }
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

// Pass-2 element functions, shared by pass 2 and the epilogue scan so that
// both see bit-identical values.
struct ResidConst { float beta, c, Rf, isf, Rq, isq; };
DEV float resid_elem(float t, float a, float b, const ResidConst& k) {
  const float f = fuse(t, a, b, k.beta);
  const float p = __builtin_amdgcn_exp2f(fmaxf(__builtin_fmaf(f, k.c, -k.Rf), -200.0f)) * k.isf;
  const float q = __builtin_amdgcn_exp2f(__builtin_fmaf(a, k.c, -k.Rq)) * k.isq;
  return fmaxf(p - q, 0.0f);
}
struct BonusConst { float c, Rt; };
DEV float bonus_elem(float t, const BonusConst& k) {
  return __builtin_amdgcn_exp2f(__builtin_fmaf(t, k.c, -k.Rt));
}

// log2 of a positive double to ~1e-7 absolute: exact exponent split plus the
// hardware log2 of the mantissa.
DEV double log2_dbl(double x) {
  int e;
  const double m = frexp(x, &e);            // x = m * 2^e, m in [0.5, 1)
  return (double)e + (double)__builtin_amdgcn_logf((float)m);
}
DEV double ln_f(float x) { return (double)__builtin_amdgcn_logf(x) * kLn2; }

// Draft-token gathers of one row through the scalar cache (uniform
// addresses), so that waiting for them never waits for tile loads.
struct Gather { float t, a, b, p, u; };

template <int DT>
DEV float sload_elem(const void* base, long long idx) {
  if (DT == ASYMSPEC_BF16) {
    const uint32_t w = ((cptr32)base)[idx >> 1];
    return __uint_as_float((idx & 1) ? (w & 0xFFFF0000u) : (w << 16));
  }
  return __uint_as_float(((cptr32)base)[idx]);
}

template <int DT>
DEV Gather sgather(const KArgs& A, const RowGeo& g) {
  Gather q{0.0f, 0.0f, 0.0f, 1.0f, 0.0f};
  if (is_draft(g.kind)) {
    int dtok = (int)((cptr32)(const void*)A.d)[g.req * A.K + g.pos];
    dtok = dtok < 0 ? 0 : (dtok >= A.V ? A.V - 1 : dtok);
    const long long idx = g.e0 + dtok;
    q.t = sload_elem<DT>(A.t, idx);
    q.a = sload_elem<DT>(A.a, idx);
    q.b = sload_elem<DT>(A.b, idx);
    if (A.dp != nullptr) q.p = sload_f32(A.dp, (long long)g.req * A.K + g.pos);
    q.u = sload_f32(A.u, (long long)g.req * (A.K + 1) + g.pos);
  }
  return q;
}

// Per-row scalars, computed once by lane 0 after the team barrier.
struct RowScal {
  float M[kSlots], R[kSlots];
  double S[kSlots], L2[kSlots];   // L2 = R + log2 S: log2-domain LSE at the slot scale
  float khi[2], klo[2];           // log2 S of a and b split in two floats (JSD)
  float isF, isQ, Rq;             // residual constants
  int arg;                        // argmax (greedy draft: f; greedy bonus: t)
  int neq;                        // a and b differ somewhere in the row
  int needD, needRes, needBonus, decided, accept;
  double margin;                  // greedy: log Eq.-4 ratio without D; sampling: x
  double lp_d, lp_emit, lnu;
};

struct Smem {
  float wm[kWaves][kSlots];
  float ws[kWaves][kSlots];
  int   warg[kWaves];
  int   wneq[kWaves];
  float wj[kWaves];
  float wseg[kWaves];
  uint32_t rec[kR1];
  RowScal rs;                     // row in pass 2
  RowScal rsp;                    // row whose settlement waits for its JSD partials
  int   flags[8];
  double dd[8];
  double scan[kWaves];
  uint32_t rw[kWaves * 4];        // epilogue: record of the emitting row
};

// Inclusive and exclusive prefix sums over the workgroup, in thread order.
DEV void block_scan(double x, Smem& sm, double& incl, double& excl) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
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
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  x = wave_min_i(x);
  __syncthreads();
  if (lane == 0) sm.warg[w] = x;
  __syncthreads();
  int r = sm.warg[0];
  #pragma unroll
  for (int i = 1; i < kWaves; ++i) r = min(r, sm.warg[i]);
  return r;
}

// Settled-row record slots.
enum {
  RW_ACCEPT = 0, RW_EMIT = 1, RW_LPD = 2, RW_LPEMIT = 3, RW_D = 4, RW_GEFF = 5,
  RW_C = 6, RW_R1 = 7, RW_IS1 = 8, RW_R2 = 9, RW_IS2 = 10, RW_KIND = 11,
  RW_L2P_LO = 12, RW_L2P_HI = 13, RW_USED = 14
};

// Lane 0: decide the row from its combined statistics and D (Eq. 3-4, or the
// sampling form), and publish the settled-row record.
DEV void write_row_t0(const KArgs& A, const RowGeo& g, const RowScal& rs, double D) {
  bool accept = rs.accept != 0;
  const bool cda = A.gate_mode == ASYMSPEC_GATE_CDA;
  if (!rs.decided) {
    if (g.kind == kGreedyDraft) accept = (rs.margin + (cda ? D : 0.0)) > 0.0;
    else if (g.kind == kSampleDraft) accept = rs.lnu < rs.margin + (cda ? D : 0.0);
  }
  const float geff = cda ? A.gamma * __builtin_amdgcn_exp2f((float)(-D * 1.4426950408889634)) : A.gamma;
  uint64_t* rw = A.rowres + (size_t)g.row * kRW;
  const uint32_t ep = A.epoch;
  uint32_t v[RW_USED];
  v[RW_ACCEPT] = accept ? 1u : 0u;
  v[RW_EMIT] = (uint32_t)rs.arg;
  v[RW_LPD] = __float_as_uint((float)rs.lp_d);
  v[RW_LPEMIT] = __float_as_uint((float)rs.lp_emit);
  v[RW_D] = __float_as_uint((float)D);
  v[RW_GEFF] = __float_as_uint(geff);
  v[RW_KIND] = (uint32_t)g.kind;
  v[RW_C] = __float_as_uint(g.c);
  v[RW_R1] = __float_as_uint(g.kind == kSampleDraft ? rs.R[sF] : rs.R[sT]);
  v[RW_IS1] = __float_as_uint(rs.isF);
  v[RW_R2] = __float_as_uint(rs.Rq);
  v[RW_IS2] = __float_as_uint(rs.isQ);
  const double l2 = g.kind == kSampleDraft ? rs.L2[sF] : rs.L2[sT];
  v[RW_L2P_LO] = dlo(l2);
  v[RW_L2P_HI] = dhi(l2);
  #pragma unroll
  for (int i = 0; i < RW_USED; ++i) st_tag(rw + i, v[i], ep);
}

// Wave 0: wait until all S pass-2 records of `row` are in; returns the fp64
// sum of their JSD partials (every lane gets it).
DEV double collect_jsd(const KArgs& A, int row) {
  const int lane = threadIdx.x & 63;
  const uint64_t* base = A.rec2 + (size_t)row * A.S * kR2;
  long spins = 0;
  double dj = 0.0;
  while (true) {
    bool ok = true;
    dj = 0.0;
    for (int c = lane; c < A.S; c += 64) {
      const uint64_t lo = ld_tag(base + (size_t)c * kR2), hi = ld_tag(base + (size_t)c * kR2 + 1);
      ok = ok && tag_ok(lo, A.epoch) && tag_ok(hi, A.epoch);
      dj += payd(lo, hi);
    }
    if (__all(ok)) break;
    __builtin_amdgcn_s_sleep(2);
    if (++spins > kSpinLimit) { if (lane == 0) err_count(A.err); break; }
  }
  return wave_sum_d(dj);
}

// Inverse-CDF emission: the first element x of row `row` whose cumulative
// weight exceeds u * total; weights are the residual (draft rows) or the
// bonus weights, recomputed with the same element functions as pass 2.
// Returns -1 when no element carries weight.  Whole workgroup.
template <int DT, int NV>
DEV int cdf_pick(const KArgs& A, int row, double u, bool bonus, Smem& sm) {
  constexpr int VE = Elem<DT>::VE;
  constexpr int kSegVec = 64 * NV;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const RowGeo g = row_geo<DT>(A, row);
  const int nseg = A.S * kWaves;
  const uint64_t* base2 = A.rec2 + (size_t)row * A.S * kR2;
  // total weight of the row (wave 0 waits for every segment sum)
  if (w == 0) {
    long spins = 0;
    double tot = 0.0;
    while (true) {
      bool ok = true;
      tot = 0.0;
      for (int sg = lane; sg < nseg; sg += 64) {
        const uint64_t* p = base2 + (size_t)(sg / kWaves) * kR2 + 2 + 2 * (sg % kWaves);
        const uint64_t lo = ld_tag(p), hi = ld_tag(p + 1);
        ok = ok && tag_ok(lo, A.epoch) && tag_ok(hi, A.epoch);
        tot += payd(lo, hi);
      }
      if (__all(ok)) break;
      __builtin_amdgcn_s_sleep(2);
      if (++spins > kSpinLimit) { if (lane == 0) err_count(A.err); break; }
    }
    tot = wave_sum_d(tot);
    if (lane == 0) sm.dd[4] = tot;
  }
  __syncthreads();
  const double total = sm.dd[4];
  if (!(total > 0.0)) return -1;
  const double target = u * total;
  // 1. the segment holding the target: scan of segment sums in index order
  double carry = 0.0;
  int sel = 0x7FFFFFFF, last_nz = -1;
  for (int s0 = 0; s0 < nseg && sel == 0x7FFFFFFF; s0 += kThreads) {
    const int sg = s0 + tid;
    double v = 0.0;
    if (sg < nseg) {
      const uint64_t* p = base2 + (size_t)(sg / kWaves) * kR2 + 2 + 2 * (sg % kWaves);
      v = payd(ld_tag(p), ld_tag(p + 1));
    }
    double incl, excl;
    block_scan(v, sm, incl, excl);
    incl += carry;
    excl += carry;
    const int cand = block_min_i((v > 0.0 && incl > target) ? sg : 0x7FFFFFFF, sm);
    const int lnz = block_min_i(v > 0.0 ? -sg : 0x7FFFFFFF, sm);
    if (lnz != 0x7FFFFFFF) last_nz = -lnz;
    __syncthreads();
    if (sg == cand) sm.dd[6] = excl;
    if (sg == last_nz) sm.dd[7] = excl;
    if (tid == kThreads - 1) sm.dd[5] = incl;
    __syncthreads();
    carry = sm.dd[5];
    sel = cand;
  }
  if (sel == 0x7FFFFFFF) {
    if (last_nz < 0) return -1;
    sel = last_nz;
    if (tid == 0) sm.dd[6] = sm.dd[7];
  }
  __syncthreads();
  const double before = sm.dd[6];
  // 2. scan inside the segment: thread tid < kSegVec takes its vector tid
  static_assert(kSegVec <= kThreads, "at most one segment vector per thread");
  const int c = sel / kWaves, ww = sel % kWaves;
  const uint32_t* rw = sm.rw;
  const ResidConst rk{A.beta, __uint_as_float(rw[RW_C]), __uint_as_float(rw[RW_R1]),
                      __uint_as_float(rw[RW_IS1]), __uint_as_float(rw[RW_R2]),
                      __uint_as_float(rw[RW_IS2])};
  const BonusConst bk{rk.c, rk.Rf};
  const long long vi = g.vbeg + (long long)c * (kThreads * NV) + (long long)ww * kSegVec + tid;
  float w8[VE];
  double tsum = 0.0;
  int last_pos = -1;
  #pragma unroll
  for (int e = 0; e < VE; ++e) {
    const long long idx = vi * VE + e;
    float wv = 0.0f;
    if (tid < kSegVec && idx >= g.e0 && idx < g.e0 + A.V) {
      const float xt = Elem<DT>::load_one(A.t, idx);
      if (bonus) {
        wv = bonus_elem(xt, bk);
      } else {
        const float xa = Elem<DT>::load_one(A.a, idx);
        const float xb = Elem<DT>::load_one(A.b, idx);
        wv = resid_elem(xt, xa, xb, rk);
      }
    }
    w8[e] = wv;
    tsum += (double)wv;
    if (wv > 0.0f) last_pos = (int)(idx - g.e0);
  }
  double incl, excl;
  block_scan(tsum, sm, incl, excl);
  double run = before + excl;
  int first_ok = 0x7FFFFFFF;
  #pragma unroll
  for (int e = 0; e < VE; ++e) {
    run += (double)w8[e];
    if (w8[e] > 0.0f && run > target && first_ok == 0x7FFFFFFF)
      first_ok = (int)(vi * VE + e - g.e0);
  }
  int pick = block_min_i(first_ok, sm);
  if (pick == 0x7FFFFFFF) {
    // rounding left the target past the segment's own sum: its last nonzero
    const int neg = block_min_i(last_pos >= 0 ? -last_pos : 0x7FFFFFFF, sm);
    pick = (neg == 0x7FFFFFFF) ? -1 : -neg;
  }
  return pick;
}

// Argmax of the fused logits of one row by a full scan (whole workgroup);
// only used when a residual is empty (p~ equal to q in fp32).
template <int DT>
DEV int row_argmax_f(const KArgs& A, const RowGeo& g, Smem& sm) {
  float best = kFloorM;
  int bi = 0x7FFFFFFF;
  for (int x = threadIdx.x; x < A.V; x += kThreads) {
    const long long idx = g.e0 + x;
    const float f = fuse(Elem<DT>::load_one(A.t, idx), Elem<DT>::load_one(A.a, idx),
                         Elem<DT>::load_one(A.b, idx), A.beta);
    if (f > best) { best = f; bi = x; }
  }
  const float M = wave_max(best);
  __syncthreads();
  if ((threadIdx.x & 63) == 0) sm.wm[threadIdx.x >> 6][0] = M;
  __syncthreads();
  float Mb = sm.wm[0][0];
  #pragma unroll
  for (int i = 1; i < kWaves; ++i) Mb = fmaxf(Mb, sm.wm[i][0]);
  return block_min_i(best == Mb ? bi : 0x7FFFFFFF, sm);
}

// Request epilogue (whole workgroup): wait for the K+1 settled rows of the
// request, take accept_len = the first rejected draft (Alg. 1), emit the token
// and write the outputs.
template <int DT, int NV>
DEV void request_epilogue(const KArgs& A, int req, Smem& sm) {
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int K = A.K;
  const size_t row0 = (size_t)req * (K + 1);
  if (w == 0) {
    long spins = 0;
    int rej = 0x7FFFFFFF;
    while (true) {
      bool ok = true;
      rej = 0x7FFFFFFF;
      for (int i = lane; i <= K; i += 64) {
        const uint64_t v = ld_tag(A.rowres + (row0 + i) * kRW + RW_ACCEPT);
        ok = ok && tag_ok(v, A.epoch);
        if (i < K && pay(v) == 0u) rej = min(rej, i);
      }
      if (__all(ok)) break;
      __builtin_amdgcn_s_sleep(2);
      if (++spins > kSpinLimit) { if (lane == 0) err_count(A.err); break; }
    }
    rej = wave_min_i(rej);
    const int j = (rej == 0x7FFFFFFF) ? K : rej;
    if (lane < RW_USED) {
      uint64_t v;
      long sp = 0;
      do {
        v = ld_tag(A.rowres + (row0 + j) * kRW + lane);
        if (tag_ok(v, A.epoch)) break;
        __builtin_amdgcn_s_sleep(1);
      } while (++sp < kSpinLimit);
      sm.rw[lane] = pay(v);
    }
    if (lane == 0) sm.flags[6] = j;
  }
  __syncthreads();
  const int j = sm.flags[6];
  const uint32_t kind = sm.rw[RW_KIND];
  int next = 0;
  double lpn = 0.0;
  if (kind == kGreedyDraft || kind == kGreedyBonus) {
    next = (int)sm.rw[RW_EMIT];
    lpn = (double)__uint_as_float(sm.rw[RW_LPEMIT]);
  } else {
    const double u = (double)A.u[req * (K + 1) + K];
    const bool bonus = kind == kSampleBonus;
    int pick = cdf_pick<DT, NV>(A, (int)(row0 + j), u, bonus, sm);
    if (pick < 0) pick = row_argmax_f<DT>(A, row_geo<DT>(A, (int)(row0 + j)), sm);
    next = pick;
    const long long idx = (long long)(row0 + j) * A.V + next;
    const float xt = Elem<DT>::load_one(A.t, idx);
    float x = xt;
    if (!bonus) {
      const float xa = Elem<DT>::load_one(A.a, idx);
      const float xb = Elem<DT>::load_one(A.b, idx);
      x = fuse_masked(xt, xa, xb, A.beta);
    }
    const double c = (double)__uint_as_float(sm.rw[RW_C]);
    const double l2 = __builtin_bit_cast(double, (uint64_t)sm.rw[RW_L2P_LO] | ((uint64_t)sm.rw[RW_L2P_HI] << 32));
    lpn = ((double)x * c - l2) * kLn2;
  }
  for (int i = tid; i < K; i += kThreads) {
    const uint64_t* ri = A.rowres + (row0 + i) * kRW;
    A.flp_out[req * (K + 1) + i] = payf(ld_tag(ri + RW_LPD));
    if (A.gate_out != nullptr) {
      A.gate_out[(req * K + i) * 2 + 0] = payf(ld_tag(ri + RW_D));
      A.gate_out[(req * K + i) * 2 + 1] = payf(ld_tag(ri + RW_GEFF));
    }
  }
  if (tid == 0) {
    A.acc_out[req] = j;
    A.next_out[req] = next;
    A.flp_out[req * (K + 1) + K] = (float)lpn;
  }
  __syncthreads();
}

// Wave 0: wait for the S pass-1 records of the row (the team barrier),
// combine them (lane c owns record c), and let lane 0 classify the row
// (Eq. 3-4; the sampling form for tau > 0) into sm.rs.
template <int DT>
DEV void team_combine(const KArgs& A, const RowGeo& g, const Gather& gq, int status, Smem& sm) {
  const int lane = threadIdx.x & 63;
  const bool draft = is_draft(g.kind);
  const bool samp = g.kind == kSampleDraft || g.kind == kSampleBonus;
  const bool tau1 = g.tau == 1.0f;
  float cs[kSlots];
  cs[sT] = samp ? g.c : kL2E;
  cs[sA] = kL2E;
  cs[sB] = kL2E;
  cs[sF] = samp ? g.c : kL2E;
  cs[sAT] = g.c;
  const uint64_t* base = A.rec1 + (size_t)g.row * A.S * kR1;
  const uint32_t ep = A.epoch;
  // own record (c = lane) kept in registers; records c >= 64 are re-read
  uint64_t r[P1_USED];
  const bool have = lane < A.S;
  long spins = 0;
  while (true) {
    bool ok = true;
    if (have) {
      #pragma unroll
      for (int j = 0; j < P1_USED; ++j) { r[j] = ld_tag(base + (size_t)lane * kR1 + j); ok = ok && tag_ok(r[j], ep); }
    }
    for (int c = lane + 64; c < A.S; c += 64) {
      #pragma unroll
      for (int j = 0; j < P1_USED; ++j) ok = ok && tag_ok(ld_tag(base + (size_t)c * kR1 + j), ep);
    }
    if (__all(ok)) break;
    __builtin_amdgcn_s_sleep(1);
    if (++spins > kSpinLimit) { if (lane == 0) err_count(A.err); break; }
  }
  float M[kSlots];
  #pragma unroll
  for (int s = 0; s < kSlots; ++s) M[s] = have ? payf(r[P1_M + s]) : kFloorM;
  for (int c = lane + 64; c < A.S; c += 64) {
    #pragma unroll
    for (int s = 0; s < kSlots; ++s) M[s] = fmaxf(M[s], payf(ld_tag(base + (size_t)c * kR1 + P1_M + s)));
  }
  #pragma unroll
  for (int s = 0; s < kSlots; ++s) M[s] = wave_max(M[s]);
  const int asl = draft ? sF : sT;
  double Sp[kSlots];
  int arg = 0x7FFFFFFF, nq = 0;
  #pragma unroll
  for (int s = 0; s < kSlots; ++s) {
    Sp[s] = have ? (double)payf(r[P1_S + s]) *
                       (double)__builtin_amdgcn_exp2f(payf(r[P1_M + s]) * cs[s] - M[s] * cs[s])
                 : 0.0;
  }
  const float Masl = draft ? M[sF] : M[sT];
  if (have) {
    const float mine = draft ? payf(r[P1_M + sF]) : payf(r[P1_M + sT]);
    if (mine == Masl) arg = (int)pay(r[P1_ARG]);
    nq = (int)pay(r[P1_NEQ]);
  }
  for (int c = lane + 64; c < A.S; c += 64) {
    const uint64_t* rc = base + (size_t)c * kR1;
    #pragma unroll
    for (int s = 0; s < kSlots; ++s) {
      const float mc = payf(ld_tag(rc + P1_M + s));
      Sp[s] += (double)payf(ld_tag(rc + P1_S + s)) *
               (double)__builtin_amdgcn_exp2f(mc * cs[s] - M[s] * cs[s]);
    }
    if (payf(ld_tag(rc + P1_M + asl)) == Masl) arg = min(arg, (int)pay(ld_tag(rc + P1_ARG)));
    nq |= (int)pay(ld_tag(rc + P1_NEQ));
  }
  #pragma unroll
  for (int s = 0; s < kSlots; ++s) Sp[s] = wave_sum_d(Sp[s]);
  arg = wave_min_i(arg);
  const bool neq_row = __any(nq != 0);
  if (lane != 0) return;

  RowScal& rs = sm.rs;
  #pragma unroll
  for (int s = 0; s < kSlots; ++s) {
    rs.M[s] = M[s];
    rs.R[s] = M[s] * cs[s];
    rs.S[s] = Sp[s];
    rs.L2[s] = (double)rs.R[s] + log2_dbl(Sp[s]);
  }
  rs.arg = arg;
  rs.neq = neq_row ? 1 : 0;
  const bool cda = A.gate_mode == ASYMSPEC_GATE_CDA;
  rs.decided = 1;
  rs.accept = 0;
  rs.needD = rs.needRes = 0;
  rs.needBonus = g.kind == kSampleBonus;
  rs.margin = rs.lp_d = rs.lp_emit = rs.lnu = 0.0;
  rs.isF = rs.isQ = rs.Rq = 0.0f;
  if (draft) {
    const double ka = log2_dbl(rs.S[sA]), kb = log2_dbl(rs.S[sB]);
    rs.khi[0] = (float)ka; rs.klo[0] = (float)(ka - (double)rs.khi[0]);
    rs.khi[1] = (float)kb; rs.klo[1] = (float)(kb - (double)rs.khi[1]);
    const float fd = fuse_masked(gq.t, gq.a, gq.b, A.beta);
    if (g.kind == kGreedyDraft) {
      const double lpt = ((double)gq.t * (double)kL2E - rs.L2[sT]) * kLn2;
      const double lpb = ((double)gq.b * (double)kL2E - rs.L2[sB]) * kLn2;
      double m0 = lpt - lpb - A.ln_gamma;
      if (m0 != m0) m0 = -INFINITY;
      rs.margin = m0;
      rs.lp_d = ((double)fd * (double)kL2E - rs.L2[sF]) * kLn2;
      rs.lp_emit = ((double)rs.M[sF] * (double)kL2E - rs.L2[sF]) * kLn2;
      if (!cda || !rs.neq) rs.accept = m0 > 0.0;
      else if (m0 > 0.0) rs.accept = 1;
      else if (m0 + kLn2 <= 0.0) rs.accept = 0;
      else rs.decided = 0;
      rs.needD = rs.neq && (!rs.decided || A.want_gate);
    } else {
      const int qs = tau1 ? sA : sAT;
      rs.lp_d = ((double)fd * (double)g.c - rs.L2[sF]) * kLn2;
      double lq;
      if (A.dp != nullptr) lq = gq.p > 0.0f ? ln_f(gq.p) : -INFINITY;
      else lq = ((double)gq.a * (double)g.c - rs.L2[qs]) * kLn2;
      double x;
      if (rs.lp_d == -INFINITY) x = -INFINITY;
      else if (lq == -INFINITY) x = INFINITY;
      else x = rs.lp_d - lq - A.ln_gamma;
      rs.margin = x;
      rs.lnu = gq.u > 0.0f ? ln_f(gq.u) : -INFINITY;
      // accept iff ln u < x + D  (u < min(1, exp(x + D)) for u in [0, 1))
      if (!cda || !rs.neq) rs.accept = rs.lnu < x;
      else if (rs.lnu < x) rs.accept = 1;
      else if (rs.lnu >= x + kLn2) rs.accept = 0;
      else rs.decided = 0;
      rs.needD = rs.neq && (!rs.decided || A.want_gate);
      rs.needRes = !(rs.decided && rs.accept);
      rs.isF = (float)(1.0 / rs.S[sF]);
      rs.isQ = (float)(1.0 / rs.S[qs]);
      rs.Rq = rs.R[qs];
    }
  } else if (g.kind == kGreedyBonus) {
    rs.lp_emit = ((double)rs.M[sT] * (double)kL2E - rs.L2[sT]) * kLn2;
  }
  if (status == kReqRejected) {
    // an earlier draft of this request is already rejected: this row cannot
    // emit and its own decision does not matter (Alg. 1 stops at the first
    // rejection); D is still computed when the caller asks for it
    rs.decided = 1;
    rs.accept = 0;
    rs.needRes = 0;
    rs.needBonus = 0;
    rs.needD = draft && rs.neq && A.want_gate;
  }
}

// The member of a team that settles a row: rotated over the members.
DEV int settler(const KArgs& A, int row) { return row % A.S; }

// Fused logit with beta = 1: fl(1 * d) = d, so this is bit-identical to fuse().
DEV float fuse1(float t, float a, float b) { return __fadd_rn(t, __fsub_rn(a, b)); }

typedef uint64_t u2l __attribute__((ext_vector_type(2)));

// Pass 1 on the register tile of row g; publishes the chunk record.
template <int DT, int NV, bool kBeta1>
DEV void pass1(const KArgs& A, const RowGeo& g, int mem, const u4 (&cur)[3][NV], Smem& sm) {
  constexpr int VE = Elem<DT>::VE;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const bool draft = is_draft(g.kind);
  const bool samp = g.kind == kSampleDraft || g.kind == kSampleBonus;
  const bool greedy_draft = g.kind == kGreedyDraft;
  const bool needT = !draft || greedy_draft;
  const bool needAT = g.kind == kSampleDraft && g.tau != 1.0f;
  const float cT = samp ? g.c : kL2E;
  const float cF = samp ? g.c : kL2E;

  Acc qT, qA, qB, qF, qAT;
  acc_init(qT, cT); acc_init(qA, kL2E); acc_init(qB, kL2E); acc_init(qF, cF); acc_init(qAT, g.c);
  bool neqb = false;
  if (draft) {
    #pragma unroll
    for (int k = 0; k < NV; ++k) {
      float xt[VE], xa[VE], xb[VE], xf[VE];
      #pragma unroll
      for (int e = 0; e < VE; ++e) {
        xt[e] = Elem<DT>::get(cur[0][k], e);
        xa[e] = Elem<DT>::get(cur[1][k], e);
        xb[e] = Elem<DT>::get(cur[2][k], e);
        xf[e] = kBeta1 ? fuse1(xt[e], xa[e], xb[e]) : fuse(xt[e], xa[e], xb[e], A.beta);
      }
      const u2l va = __builtin_bit_cast(u2l, cur[1][k]), vb = __builtin_bit_cast(u2l, cur[2][k]);
      neqb = neqb | (va.x != vb.x) | (va.y != vb.y);
      if (greedy_draft) {
        acc_vec<VE, false>(qT, xt, cT, k);
        acc_vec<VE, false, true>(qF, xf, cF, k);
      } else {
        acc_vec<VE, false>(qF, xf, cF, k);
      }
      acc_vec<VE, false>(qA, xa, kL2E, k);
      acc_vec<VE, false>(qB, xb, kL2E, k);
      if (needAT) acc_vec<VE, false>(qAT, xa, g.c, k);
      // one vector's temporaries at a time: keeps the tile buffers in VGPRs
      __builtin_amdgcn_sched_barrier(0);
    }
    // A fused logit that is not a number (a = b = -inf, a masked token) makes
    // the f sum NaN; only then redo it with the NaN-clamping exponent.
    // The tile is passed through an empty asm first: otherwise the compiler
    // reuses the decoded elements of the loop above and keeps all of them
    // live until this test.
    if (qF.s != qF.s) {
      acc_init(qF, cF);
      #pragma unroll
      for (int k = 0; k < NV; ++k) {
        u4 vt = cur[0][k], va = cur[1][k], vb = cur[2][k];
        asm volatile("" : "+v"(vt), "+v"(va), "+v"(vb));
        float xf[VE];
        #pragma unroll
        for (int e = 0; e < VE; ++e)
          xf[e] = fuse(Elem<DT>::get(vt, e), Elem<DT>::get(va, e), Elem<DT>::get(vb, e), A.beta);
        if (greedy_draft) acc_vec<VE, true, true>(qF, xf, cF, k);
        else acc_vec<VE, true>(qF, xf, cF, k);
      }
    }
  } else {
    #pragma unroll
    for (int k = 0; k < NV; ++k) {
      float xt[VE];
      #pragma unroll
      for (int e = 0; e < VE; ++e) xt[e] = Elem<DT>::get(cur[0][k], e);
      if (g.kind == kGreedyBonus) acc_vec<VE, false, true>(qT, xt, cT, k);
      else acc_vec<VE, false>(qT, xt, cT, k);
    }
  }

  // wave level: max, sums rescaled to the wave max, argmax candidate
  #define ASYM_WAVE_SLOT(S_, Q_, C_, USED_)                                      \
    {                                                                           \
      float mw = kFloorM, sw = 0.0f;                                            \
      if (USED_) {                                                              \
        mw = wave_max(Q_.m);                                                    \
        sw = wave_sum(Q_.s * __builtin_amdgcn_exp2f(Q_.R - mw * (C_)));         \
      }                                                                         \
      if (lane == 0) { sm.wm[w][S_] = mw; sm.ws[w][S_] = sw; }                  \
    }
  ASYM_WAVE_SLOT(sT, qT, cT, needT)
  ASYM_WAVE_SLOT(sA, qA, kL2E, draft)
  ASYM_WAVE_SLOT(sB, qB, kL2E, draft)
  ASYM_WAVE_SLOT(sF, qF, cF, draft)
  ASYM_WAVE_SLOT(sAT, qAT, g.c, needAT)
  #undef ASYM_WAVE_SLOT
  {
    const bool need_arg = greedy_draft || g.kind == kGreedyBonus;
    int cand = 0x7FFFFFFF;
    if (need_arg) {
      const float qam = greedy_draft ? qF.m : qT.m;
      const int qpos = greedy_draft ? qF.pos : qT.pos;
      const float mw = wave_max(qam);
      if (qam == mw && mw > kFloorM) {
        // this thread's first maximum: vector k = qpos / VE, element qpos % VE
        const long long vi = g.vbeg + (long long)mem * (kThreads * NV) + (long long)w * (64 * NV) +
                             (long long)(qpos / VE) * 64 + lane;
        cand = (int)(vi * VE + (qpos % VE) - g.e0);
      }
      cand = wave_min_i(cand);
    }
    const int wn = __any(neqb) ? 1 : 0;
    if (lane == 0) { sm.warg[w] = cand; sm.wneq[w] = wn; }
  }
  __syncthreads();
  // thread 0: the chunk record (fp64 across waves, fp32 payloads)
  if (tid == 0) {
    const float cs[kSlots] = {cT, kL2E, kL2E, cF, g.c};
    int arg = 0x7FFFFFFF, nq = 0;
    const int asl = draft ? sF : sT;
    float Mall = kFloorM;
    #pragma unroll
    for (int i = 0; i < kWaves; ++i) Mall = fmaxf(Mall, sm.wm[i][asl]);
    #pragma unroll
    for (int s = 0; s < kSlots; ++s) {
      float M = kFloorM;
      #pragma unroll
      for (int i = 0; i < kWaves; ++i) M = fmaxf(M, sm.wm[i][s]);
      const float R = M * cs[s];
      double S = 0.0;
      #pragma unroll
      for (int i = 0; i < kWaves; ++i)
        S += (double)sm.ws[i][s] * (double)__builtin_amdgcn_exp2f(sm.wm[i][s] * cs[s] - R);
      sm.rec[P1_M + s] = __float_as_uint(M);
      sm.rec[P1_S + s] = __float_as_uint((float)S);
    }
    #pragma unroll
    for (int i = 0; i < kWaves; ++i) {
      if (sm.wm[i][asl] == Mall) arg = min(arg, sm.warg[i]);
      nq |= sm.wneq[i];
    }
    sm.rec[P1_ARG] = (uint32_t)arg;
    sm.rec[P1_NEQ] = (uint32_t)nq;
  }
  __syncthreads();
  if (w == 0 && lane < P1_USED)
    st_tag(A.rec1 + ((size_t)g.row * A.S + mem) * kR1 + lane, sm.rec[lane], A.epoch);
}

// Pass-2 partial sums of one thread over its stashed tile: the JSD term
// (kD) and/or the residual weights (kR).
template <int DT, int NV, bool kD, bool kR>
DEV void pass2_sums(const KArgs& A, const RowGeo& g, const u4* stash, const Smem& sm,
                    float& accj, float& seg) {
  constexpr int VE = Elem<DT>::VE;
  const int tid = threadIdx.x;
  const float kahi = sm.rs.khi[0], kalo = sm.rs.klo[0];
  const float kbhi = sm.rs.khi[1], kblo = sm.rs.klo[1];
  const float Ra = sm.rs.R[sA], Rb = sm.rs.R[sB];
  const ResidConst rk{A.beta, g.c, sm.rs.R[sF], sm.rs.isF, sm.rs.Rq, sm.rs.isQ};
  #pragma unroll
  for (int k = 0; k < NV; ++k) {
    const u4 va = stash[(1 * NV + k) * kThreads + tid];
    const u4 vb = stash[(2 * NV + k) * kThreads + tid];
    u4 vt = va;
    if (kR) vt = stash[(0 * NV + k) * kThreads + tid];
    float vj[VE], vr[VE];
    #pragma unroll
    for (int e = 0; e < VE; ++e) {
      const float xa = Elem<DT>::get(va, e);
      const float xb = Elem<DT>::get(vb, e);
      vj[e] = 0.0f;
      vr[e] = 0.0f;
      if (kD) {
        // P log2(2P/(P+Q)) + Q log2(2Q/(P+Q)) with lp = log2 P, lq = log2 Q
        const float lp = (fmaxf(__builtin_fmaf(xa, kL2E, -Ra), kFloorM) - kahi) - kalo;
        const float lq = (fmaxf(__builtin_fmaf(xb, kL2E, -Rb), kFloorM) - kbhi) - kblo;
        const float P = __builtin_amdgcn_exp2f(lp);
        const float Q = __builtin_amdgcn_exp2f(lq);
        const float gg = 1.0f - __builtin_amdgcn_logf(fmaxf(P + Q, 1e-37f));
        vj[e] = __builtin_fmaf(P, lp + gg, Q * (lq + gg));
      }
      if (kR) vr[e] = resid_elem(Elem<DT>::get(vt, e), xa, xb, rk);
    }
    #pragma unroll
    for (int st = 1; st < VE; st <<= 1)
      #pragma unroll
      for (int e = 0; e + st < VE; e += 2 * st) { vj[e] += vj[e + st]; vr[e] += vr[e + st]; }
    accj += vj[0];
    seg += vr[0];
    __builtin_amdgcn_sched_barrier(0);
  }
}

// Pass 2 of row g on its tile in the LDS stash (thread-private slots), when
// the row needs it; publishes the chunk's pass-2 record.
template <int DT, int NV>
DEV void pass2(const KArgs& A, const RowGeo& g, int mem, const u4* stash, Smem& sm) {
  constexpr int VE = Elem<DT>::VE;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int needD = sm.rs.needD, needRes = sm.rs.needRes, needBonus = sm.rs.needBonus;
  if (!(needD || needRes || needBonus)) return;
  float accj = 0.0f, seg = 0.0f;
  if (needD && needRes) pass2_sums<DT, NV, true, true>(A, g, stash, sm, accj, seg);
  else if (needD) pass2_sums<DT, NV, true, false>(A, g, stash, sm, accj, seg);
  else if (needRes) pass2_sums<DT, NV, false, true>(A, g, stash, sm, accj, seg);
  else {
    const BonusConst bk{g.c, sm.rs.R[sT]};
    #pragma unroll
    for (int k = 0; k < NV; ++k) {
      const u4 vt = stash[(0 * NV + k) * kThreads + tid];
      float vb[VE];
      #pragma unroll
      for (int e = 0; e < VE; ++e) vb[e] = bonus_elem(Elem<DT>::get(vt, e), bk);
      #pragma unroll
      for (int st = 1; st < VE; st <<= 1)
        #pragma unroll
        for (int e = 0; e + st < VE; e += 2 * st) vb[e] += vb[e + st];
      seg += vb[0];
    }
  }
  const float wj = needD ? wave_sum(accj) : 0.0f;
  const float wseg = (needRes || needBonus) ? wave_sum(seg) : 0.0f;
  if (lane == 0) { sm.wj[w] = wj; sm.wseg[w] = wseg; }
  __syncthreads();
  if (w == 0) {
    double v = 0.0;
    if (lane < 2) {
      #pragma unroll
      for (int i = 0; i < kWaves; ++i) v += (double)sm.wj[i];
    } else if (lane < 2 + 2 * kWaves) {
      v = (double)sm.wseg[(lane - 2) >> 1];
    }
    if (lane < 2 + 2 * kWaves)
      st_tag(A.rec2 + ((size_t)g.row * A.S + mem) * kR2 + lane, (lane & 1) ? dhi(v) : dlo(v), A.epoch);
  }
}

// Settlement of a row whose D waited for the JSD partials of all members.
template <int DT>
DEV void settle_pending(const KArgs& A, int row, Smem& sm) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  if (w == 0) {
    const double dj = collect_jsd(A, row);
    if (lane == 0) {
      double D = 0.5 * kLn2 * dj;
      D = D < 0.0 ? 0.0 : (D > kLn2 ? kLn2 : D);
      write_row_t0(A, row_geo<DT>(A, row), sm.rsp, D);
    }
  }
}

#ifndef ASYMSPEC_WAVES
#define ASYMSPEC_WAVES 2
#endif
template <int DT, int NV, bool kBeta1>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(ASYMSPEC_WAVES)))
void fuse_verify_kernel(KArgs A) {
  __shared__ Smem sm;
  __shared__ u4 stash[3 * NV * kThreads];
  const int team = blockIdx.x / A.S;
  const int mem = blockIdx.x - team * A.S;
  const int tid = threadIdx.x;
  // each team owns a contiguous block of rows (request-major order), so the
  // drafts of a request mostly pass through one team in order
  const int lo = team < A.n_teams ? (int)((long long)team * A.rows / A.n_teams) : 0;
  const int hi = team < A.n_teams ? (int)((long long)(team + 1) * A.rows / A.n_teams) : 0;
  const int nrows = hi - lo;
  u4 cur[3][NV], nxt[3][NV];
  if (nrows > 0) issue_loads<DT, NV>(A, row_geo<DT>(A, lo), mem, cur);
  int prev = -1;       // row whose pass 2 is pending (its tile is in the stash)
  int pend = -1;       // row this workgroup settles once its JSD partials are in
  int st_req = -1, status = kReqOpen;
  for (int it = 0; it <= nrows && nrows > 0; ++it) {
    const bool have = it < nrows;
    const int r = lo + it;
    RowGeo gp;
    Gather gq{0.0f, 0.0f, 0.0f, 1.0f, 0.0f};
    if (prev >= 0) {
      gp = row_geo<DT>(A, prev);
      gq = sgather<DT>(A, gp);
    }
    RowGeo g;
    if (have) {
      g = row_geo<DT>(A, r);
      if (it + 1 < nrows) issue_loads<DT, NV>(A, row_geo<DT>(A, r + 1), mem, nxt);
      sanitize<DT, NV>(g, A, mem, cur);
      pass1<DT, NV, kBeta1>(A, g, mem, cur, sm);
    }
    if (pend >= 0) {
      settle_pending<DT>(A, pend, sm);
      pend = -1;
    }
    if (prev >= 0) {
      if (gp.req != st_req) { st_req = gp.req; status = kReqOpen; }
      if ((tid >> 6) == 0) team_combine<DT>(A, gp, gq, status, sm);
      __syncthreads();
      pass2<DT, NV>(A, gp, mem, stash, sm);
      if (is_draft(gp.kind)) {
        if (sm.rs.decided && !sm.rs.accept) status = kReqRejected;
        else if (!sm.rs.decided && status == kReqOpen) status = kReqUnknown;
      }
      if (mem == settler(A, prev)) {
        if (sm.rs.needD) {
          if (tid == 0) sm.rsp = sm.rs;
          pend = prev;
        } else if (tid == 0) {
          write_row_t0(A, gp, sm.rs, 0.0);
        }
      }
    }
    __syncthreads();
    if (have) {
      const int ns = n_streams(g.kind);
      #pragma unroll
      for (int s = 0; s < 3; ++s)
        if (s < ns) {
          #pragma unroll
          for (int k = 0; k < NV; ++k) stash[(s * NV + k) * kThreads + tid] = cur[s][k];
        }
      #pragma unroll
      for (int s = 0; s < 3; ++s)
        #pragma unroll
        for (int k = 0; k < NV; ++k) cur[s][k] = nxt[s][k];
    }
    __syncthreads();
    prev = have ? r : -1;
  }
  if (pend >= 0) {
    settle_pending<DT>(A, pend, sm);
    __syncthreads();
  }
  for (int req = blockIdx.x; req < A.B; req += A.grid) request_epilogue<DT, NV>(A, req, sm);
}

__global__ void fill_zero_kernel(uint32_t* p, size_t n) {
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
    p[i] = 0u;
}

// ---------------------------------------------------------------- host side
// 16-byte vectors per thread per stream: four for bf16 (32 logits), four for
// fp32 (16 logits); a chunk is kThreads * kNVHost vectors.
#ifndef ASYMSPEC_NV
#define ASYMSPEC_NV 4
#endif
constexpr int kNVHost = ASYMSPEC_NV;

struct Layout {
  int S, VE;
  size_t rows;
  size_t off_rec1, off_rec2, off_row, off_err, total;
};

static size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

static bool make_layout(int B, int K, int V, int dtype, Layout& L) {
  if (B < 1 || K < 0 || V < 1) return false;
  if (dtype != ASYMSPEC_BF16 && dtype != ASYMSPEC_FP32) return false;
  const long double elems = (long double)B * (K + 1) * V;
  if (elems >= (long double)(1ull << 40)) return false;
  L.VE = dtype == ASYMSPEC_BF16 ? 8 : 4;
  const long long chunk_vec = (long long)kThreads * kNVHost;
  const long long nvec_max = ((long long)V + 2LL * L.VE - 2) / L.VE;
  L.S = (int)((nvec_max + chunk_vec - 1) / chunk_vec);
  L.rows = (size_t)B * (K + 1);
  size_t off = 0;
  L.off_rec1 = off; off = align_up(off + L.rows * L.S * kR1 * 8, 256);
  L.off_rec2 = off; off = align_up(off + L.rows * L.S * kR2 * 8, 256);
  L.off_row = off;  off = align_up(off + L.rows * kRW * 8, 256);
  L.off_err = off;  off = align_up(off + 256, 256);
  L.total = off;
  return true;
}

struct DevInfo {
  int ok = 0;
  int n_cu = 0;
  int max_blocks[2] = {0, 0};
};

static DevInfo g_dev[64];
static std::mutex g_dev_mu;

static const void* kernel_ptr(int dtype, bool beta1) {
  if (dtype == ASYMSPEC_BF16)
    return beta1 ? (const void*)fuse_verify_kernel<ASYMSPEC_BF16, kNVHost, true>
                 : (const void*)fuse_verify_kernel<ASYMSPEC_BF16, kNVHost, false>;
  return beta1 ? (const void*)fuse_verify_kernel<ASYMSPEC_FP32, kNVHost, true>
               : (const void*)fuse_verify_kernel<ASYMSPEC_FP32, kNVHost, false>;
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
  if (!pr.cooperativeLaunch) return nullptr;
  di.n_cu = pr.multiProcessorCount;
  for (int dt = 0; dt < 2; ++dt) {
    int lo = 1 << 30;
    for (int b1 = 0; b1 < 2; ++b1) {
      int nb = 0;
      if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, kernel_ptr(dt, b1 != 0), kThreads, 0) != hipSuccess)
        return nullptr;
      lo = std::min(lo, nb);
    }
    di.max_blocks[dt] = lo * di.n_cu;
  }
  di.ok = 1;
  return &di;
}

static uint32_t next_epoch() {
  static std::atomic<uint32_t> ctr{0};
  static std::once_flag once;
  std::call_once(once, [] {
    const uint64_t t = (uint64_t)std::chrono::steady_clock::now().time_since_epoch().count();
    ctr.store((uint32_t)(t ^ (t >> 32) ^ ((uint64_t)getpid() << 16)) | 1u);
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
  const int gmax = di->max_blocks[dtype];
  if (L.S > gmax) return ASYMSPEC_E_ARG;

  KArgs A;
  A.t = t; A.a = (K > 0) ? a : t; A.b = (K > 0) ? b : t;
  A.d = (K > 0) ? draft_tokens : (const int32_t*)uniforms;
  A.dp = draft_probs; A.u = uniforms; A.tau = temperature;
  A.acc_out = accept_len; A.next_out = next_token; A.flp_out = fused_logprobs; A.gate_out = gate_out;
  char* ws = (char*)workspace;
  A.rec1 = (uint64_t*)(ws + L.off_rec1);
  A.rec2 = (uint64_t*)(ws + L.off_rec2);
  A.rowres = (uint64_t*)(ws + L.off_row);
  A.err = (uint32_t*)(ws + L.off_err);
  A.stream_bytes = (unsigned long long)B * (K + 1) * (unsigned long long)V * (dtype == ASYMSPEC_BF16 ? 2ull : 4ull);
  A.B = B; A.K = K; A.V = V; A.S = L.S;
  A.rows = (int)L.rows;
  const int teams_fit = gmax / L.S;
  A.n_teams = (int)std::min<long long>((long long)L.rows, teams_fit);
  A.grid = A.n_teams * L.S;
  A.beta = params->beta; A.gamma = params->gamma; A.gate_mode = params->gate_mode;
  A.want_gate = gate_out != nullptr;
  A.ln_gamma = std::log((double)params->gamma);
  A.epoch = next_epoch();

  const dim3 grid(A.grid), block(kThreads);
  void* args[] = {&A};
  const hipError_t e = hipLaunchCooperativeKernel(kernel_ptr(dtype, params->beta == 1.0f), grid, block, args, 0,
                                                  (hipStream_t)stream);
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

int asymspec_version(void) { return 100; }

}  // extern "C"
