// Statistics item: one vocabulary chunk of one row, streamed once from HBM.
//
// Per chunk it produces the maximum and the sum of exp2(x * c - fl(M * c))
// of every logit stream the row's decision needs (the normalisers of the
// log-softmaxes in Eq. 3-4, at the row's temperature where the emission
// distribution needs it), the first index of the chunk's maximum fused logit
// f = t + beta (a - b) (Eq. 2; greedy drafts) or verifier logit (greedy bonus
// row, Alg. 1), and whether a and b differ anywhere in the chunk (a row with
// a == b everywhere has D = 0 exactly).
//
// Layout: chunk m of a row covers its vectors [m * kChunkVec, (m+1) *
// kChunkVec); sub-tile s holds kTileVec of them, wave w a run of 64 * kNV and
// lane l every 64th from there, so each load instruction of a wave reads 1 KiB
// of contiguous memory.  A rolling window keeps the next vectors of every
// stream in flight while the current one is reduced.

#ifndef ASYMSPEC_STATS_H_
#define ASYMSPEC_STATS_H_

#include "device.h"

namespace asym {

typedef uint64_t u2l __attribute__((ext_vector_type(2)));

template <int KIND> struct KindTraits;
template <> struct KindTraits<kGreedyDraft> {
  static constexpr int NS = 3; static constexpr bool kArg = true; static constexpr int argslot = sF;
  static constexpr bool kT = true, kF = true, kA = true, kB = true, kAT = false;
};
template <> struct KindTraits<kSampleDraft1> {
  static constexpr int NS = 3; static constexpr bool kArg = false; static constexpr int argslot = sF;
  static constexpr bool kT = false, kF = true, kA = true, kB = true, kAT = false;
};
template <> struct KindTraits<kSampleDraftT> {
  static constexpr int NS = 3; static constexpr bool kArg = false; static constexpr int argslot = sF;
  static constexpr bool kT = false, kF = true, kA = true, kB = true, kAT = true;
};
template <> struct KindTraits<kGreedyBonus> {
  static constexpr int NS = 1; static constexpr bool kArg = true; static constexpr int argslot = sT;
  static constexpr bool kT = true, kF = false, kA = false, kB = false, kAT = false;
};
template <> struct KindTraits<kSampleBonus> {
  static constexpr int NS = 1; static constexpr bool kArg = false; static constexpr int argslot = sT;
  static constexpr bool kT = true, kF = false, kA = false, kB = false, kAT = false;
};
// fused bonus row: f alone, from all three streams
template <> struct KindTraits<kGreedyBonusF> {
  static constexpr int NS = 3; static constexpr bool kArg = true; static constexpr int argslot = sF;
  static constexpr bool kT = false, kF = true, kA = false, kB = false, kAT = false;
};
template <> struct KindTraits<kSampleBonusF> {
  static constexpr int NS = 3; static constexpr bool kArg = false; static constexpr int argslot = sF;
  static constexpr bool kT = false, kF = true, kA = false, kB = false, kAT = false;
};

// Offset, in vectors from the thread's first vector, of its j-th vector
// (sub-tile j / kNV, step j % kNV).
constexpr int vec_rel(int j) { return (j / kNV) * kTileVec + (j % kNV) * 64; }
#ifndef ASYMSPEC_WIN
#define ASYMSPEC_WIN 4
#endif
constexpr int kWin = ASYMSPEC_WIN;   // vectors per stream in flight per thread

// Per-slot accumulators of one thread.
struct StatsAcc {
  Acc T, A, B, F, AT;
  uint64_t neq;   // lanes that saw a != b (wave-uniform mask)
  // wave-uniform: a and b have been equal bitwise in every lane so far, so B
  // would have received exactly A's updates; B is not updated then and takes
  // A's state when the first difference comes (or at the end)
  bool bsame;
  float W;        // KL gate: the A-weighted sum of a - b (see R1_W)
};

// Wave partials, cross-wave combine and the tagged chunk record.
template <int DT, int KIND, int DM, bool kKL>
DEV void publish_stats(const KArgs& A, const RowGeo& g, int m, long long rel0, const StatsAcc& q0,
                       Smem& sm) {
  using TR = KindTraits<KIND>;
  constexpr int VE = Elem<DT>::VE;
  constexpr bool kDraft = TR::NS == 3;
  const int lane = lane_id(), w = wave_id();
  StatsAcc q = q0;
  if (TR::kB && q.bsame) q.B = q.A;
  // wave partials: the largest reference, the sums rescaled to it
  #define ASYM_WAVE_SLOT(S_, Q_, USED_)                                      \
    {                                                                       \
      float rw = kFloorM, sw = 0.0f;                                        \
      if (USED_) {                                                          \
        rw = wave_max(Q_.R);                                                \
        sw = wave_sum(Q_.s * __builtin_amdgcn_exp2f(Q_.R - rw));            \
      }                                                                     \
      if (lane == 0) { sm.wm[w][S_] = rw; sm.ws[w][S_] = sw; }              \
    }
  ASYM_WAVE_SLOT(sT, q.T, TR::kT)
  ASYM_WAVE_SLOT(sA, q.A, TR::kA)
  ASYM_WAVE_SLOT(sB, q.B, TR::kB)
  ASYM_WAVE_SLOT(sF, q.F, TR::kF)
  ASYM_WAVE_SLOT(sAT, q.AT, TR::kAT)
  #undef ASYM_WAVE_SLOT
  if (kKL && TR::kA) {
    const float rw = wave_max(q.A.R);
    const float ww = wave_sum(q.W * __builtin_amdgcn_exp2f(q.A.R - rw));
    if (lane == 0) sm.wkl[w] = ww;
  }
  {
    int cand = 0x7FFFFFFF;
    float mw = kFloorM;
    if (TR::kArg) {
      // the lanes holding the wave maximum re-read the vector where their
      // running maximum first reached it and take its first such element
      const Acc& qa = TR::argslot == sF ? q.F : q.T;
      mw = wave_max(qa.m);
      if (qa.m == mw && mw > kFloorM) {
        const long long rv = rel0 + vec_rel(qa.pos);
        const long long vi = g.vbeg + rv;
        const uint32_t off = (uint32_t)(rv * 16);
        u4 vt = buf_load(row_rsrc(A, A.t, g), off);
        fix_vec<DT>(A, g, A.t, vi, vt);
        u4 va = vt, vb = vt;
        if (A.vmap != nullptr) {
          map_vecs<DT>(A, g, vi, vt, va, vb, kDraft);
        } else if (kDraft) {
          va = buf_load(row_rsrc(A, A.a, g), off);
          vb = buf_load(row_rsrc(A, A.b, g), off);
          fix_vec<DT>(A, g, A.a, vi, va);
          fix_vec<DT>(A, g, A.b, vi, vb);
        }
        int ei = VE;
        #pragma unroll
        for (int e = VE - 1; e >= 0; --e) {
          const float xt = Elem<DT>::get(vt, e);
          const float x = kDraft ? fuse<DM>(xt, Elem<DT>::get(va, e), Elem<DT>::get(vb, e), A.beta) : xt;
          ei = (x == mw) ? e : ei;
        }
        if (ei < VE) cand = (int)(vi * VE + ei - g.e0);
      }
      cand = wave_min_i(cand);
    }
    const int wn = q.neq != 0 ? 1 : 0;
    if (lane == 0) { sm.warg[w] = cand; sm.wneq[w] = wn; sm.wmarg[w] = mw; }
  }
  __syncthreads();
  // wave 0: lane s < kSlots combines slot s over the waves; lane kSlots the
  // argmax slot's maximum and index and the a-vs-b flag; then the lanes
  // publish the record
  if (w == 0) {
    uint64_t* rec = A.rec1 + ((size_t)g.row * A.S + m) * kR1;
    if (lane < kSlots) {
      float R = kFloorM;
      #pragma unroll
      for (int i = 0; i < kWaves; ++i) R = fmaxf(R, sm.wm[i][lane]);
      float S = 0.0f;
      #pragma unroll
      for (int i = 0; i < kWaves; ++i) S += sm.ws[i][lane] * __builtin_amdgcn_exp2f(sm.wm[i][lane] - R);
      st_tag(rec + R1_R + lane, __float_as_uint(R), A.epoch);
      st_tag(rec + R1_S + lane, __float_as_uint(S), A.epoch);
    } else if (lane == kSlots) {
      float Mall = kFloorM;
      #pragma unroll
      for (int i = 0; i < kWaves; ++i) Mall = fmaxf(Mall, sm.wmarg[i]);
      int arg = 0x7FFFFFFF, nq = 0;
      #pragma unroll
      for (int i = 0; i < kWaves; ++i) {
        if (sm.wmarg[i] == Mall) arg = min(arg, sm.warg[i]);
        nq |= sm.wneq[i];
      }
      st_tag(rec + R1_ARG, (uint32_t)arg, A.epoch);
      st_tag(rec + R1_NEQ, (uint32_t)nq, A.epoch);
      st_tag(rec + R1_MARG, __float_as_uint(Mall), A.epoch);
    } else if (lane == kSlots + 1) {
      // the KL sum, relative to the A slot's chunk reference (0 without it)
      float W = 0.0f;
      if (kKL && TR::kA) {
        float R = kFloorM;
        #pragma unroll
        for (int i = 0; i < kWaves; ++i) R = fmaxf(R, sm.wm[i][sA]);
        #pragma unroll
        for (int i = 0; i < kWaves; ++i) W += sm.wkl[i] * __builtin_amdgcn_exp2f(sm.wm[i][sA] - R);
      }
      st_tag(rec + R1_W, __float_as_uint(W), A.epoch);
    }
  }
}

// Ties the accumulator state to this point of the program: without it the
// compiler sinks the arithmetic of later vectors to the end of the chunk and
// keeps all their loaded data live at once.
DEV void pin(Acc& q) { asm volatile("" : "+v"(q.m), "+v"(q.R), "+v"(q.s)); }
DEV void pin_lazy(Acc& q) { asm volatile("" : "+v"(q.R), "+v"(q.s)); }

// One vector into a slot that needs no maximum: the full step on a thread's
// first vector (kFirst), the lazy step after it.
template <int VE, bool kClamp, bool kFirst>
DEV void acc_sum(Acc& q, const float (&x)[VE], float c) {
  if (kFirst) acc_vec<VE, kClamp, false>(q, x, c, 0);
  else acc_vec_lazy<VE, kClamp>(q, x, c);
}

// One vector of each stream into the accumulators.
template <int DT, int KIND, bool kB1, int DM, bool kKL, bool kClamp, bool kFirst>
DEV void stats_vec(const KArgs& A, float c, const u4& vt, const u4& va, const u4& vb, int kk, StatsAcc& q) {
  using TR = KindTraits<KIND>;
  constexpr int VE = Elem<DT>::VE;
  float xt[VE];
  #pragma unroll
  for (int e = 0; e < VE; ++e) xt[e] = Elem<DT>::get(vt, e);
  if (TR::NS == 3) {
    float xa[VE], xb[VE], xf[VE];
    #pragma unroll
    for (int e = 0; e < VE; ++e) {
      xa[e] = Elem<DT>::get(va, e);
      xb[e] = Elem<DT>::get(vb, e);
      xf[e] = kB1 ? fuse1<DM>(xt[e], xa[e], xb[e]) : fuse<DM>(xt[e], xa[e], xb[e], A.beta);
    }
    // the compare is folded into a wave mask at once and pinned there: left
    // to itself the compiler re-materialises it at its only use, keeping
    // every loaded vector of a and b live to the end of the chunk
    const u2l pa = __builtin_bit_cast(u2l, va), pb = __builtin_bit_cast(u2l, vb);
    uint64_t nm = __ballot((pa.x != pb.x) | (pa.y != pb.y));
    asm volatile("" : "+s"(nm));
    q.neq |= nm;
    // B before A: while the views agree in every lane B is A (bsame)
    if (TR::kB && !(q.bsame && nm == 0)) {
      if (q.bsame) {
        q.B = q.A;
        q.bsame = false;
      }
      acc_sum<VE, false, kFirst>(q.B, xb, kL2E);
    }
    if (TR::kT) acc_sum<VE, false, kFirst>(q.T, xt, kL2E);
    if (TR::kArg) acc_vec<VE, kClamp, true>(q.F, xf, c, kk);
    else acc_sum<VE, kClamp, kFirst>(q.F, xf, c);
    if (kKL && TR::kA) {
      float dab[VE];
      #pragma unroll
      for (int e = 0; e < VE; ++e) dab[e] = __fsub_rn(xa[e], xb[e]);
      acc_vec_w<VE, kFirst>(q.A, q.W, xa, dab, kL2E);
    } else if (TR::kA) {
      acc_sum<VE, false, kFirst>(q.A, xa, kL2E);
    }
    if (TR::kAT) acc_sum<VE, false, kFirst>(q.AT, xa, c);
    if (TR::kT) pin_lazy(q.T);
    if (TR::kArg) pin(q.F);
    else pin_lazy(q.F);
    if (TR::kA) pin_lazy(q.A);
    if (TR::kB) pin_lazy(q.B);
    if (TR::kAT) pin_lazy(q.AT);
  } else {
    if (TR::kArg) {
      acc_vec<VE, false, true>(q.T, xt, c, kk);
      pin(q.T);
    } else {
      acc_sum<VE, false, kFirst>(q.T, xt, c);
      pin_lazy(q.T);
    }
  }
}

DEV void stats_init(StatsAcc& q, float c) {
  acc_init(q.T, c); acc_init(q.A, kL2E); acc_init(q.B, kL2E); acc_init(q.F, c); acc_init(q.AT, c);
  q.neq = 0;
  q.bsame = true;
  q.W = 0.0f;
}

// Generic path: one vector at a time, every vector repaired (row boundary,
// array end), NaN-safe exponent for f.  Used for the chunk that holds a
// ragged array end, to redo a chunk whose f sum came out NaN, and for every
// chunk when the drafter rows are reached through a vocabulary map.
template <int DT, int KIND, bool kB1, int DM, bool kKL>
DEV void stats_slow(const KArgs& A, const RowGeo& g, int m, Smem& sm) {
  using TR = KindTraits<KIND>;
  constexpr bool kDraft = TR::NS == 3;
  const int lane = lane_id(), w = wave_id();
  const __amdgpu_buffer_rsrc_t rt = row_rsrc(A, A.t, g);
  const __amdgpu_buffer_rsrc_t ra = row_rsrc(A, kDraft ? A.a : A.t, g);
  const __amdgpu_buffer_rsrc_t rb = row_rsrc(A, kDraft ? A.b : A.t, g);
  const long long rel0 = (long long)m * kChunkVec + (long long)w * (64 * kNV) + lane;
  StatsAcc q;
  stats_init(q, g.c);
  #pragma unroll 1
  for (int kk = 0; kk < kNSub * kNV; ++kk) {
    const long long rv = rel0 + (long long)(kk / kNV) * kTileVec + (kk % kNV) * 64;
    const uint32_t off = (uint32_t)(rv * 16);
    const long long vi = g.vbeg + rv;
    u4 vt = buf_load(rt, off), va = vt, vb = vt;
    fix_vec<DT>(A, g, A.t, vi, vt);
    if (A.vmap != nullptr) {
      map_vecs<DT>(A, g, vi, vt, va, vb, kDraft);
    } else if (kDraft) {
      va = buf_load(ra, off);
      vb = buf_load(rb, off);
      fix_vec<DT>(A, g, A.a, vi, va);
      fix_vec<DT>(A, g, A.b, vi, vb);
    }
    stats_vec<DT, KIND, kB1, DM, kKL, true, true>(A, g.c, vt, va, vb, kk, q);
  }
  publish_stats<DT, KIND, DM, kKL>(A, g, m, rel0, q, sm);
}

// Fast path; kMask for the first and last chunk of a row (elements outside
// the row are masked, without branches).  Returns false, without publishing,
// when the chunk must be redone on the generic path.
template <int DT, int KIND, bool kB1, int DM, bool kKL, bool kMask>
DEV bool stats_fast(const KArgs& A, const RowGeo& g, int m, Smem& sm) {
  using TR = KindTraits<KIND>;
  constexpr int VE = Elem<DT>::VE;
  constexpr int NS = TR::NS;
  constexpr bool kDraft = NS == 3;
  const int lane = lane_id(), w = wave_id();
  const float c = g.c;
  const __amdgpu_buffer_rsrc_t r[3] = {row_rsrc(A, A.t, g), row_rsrc(A, kDraft ? A.a : A.t, g),
                                       row_rsrc(A, kDraft ? A.b : A.t, g)};
  // this thread's first vector, relative to the row's first vector
  const int rel0 = m * kChunkVec + w * (64 * kNV) + lane;
  const uint32_t off0 = (uint32_t)rel0 * 16u;
  // the row starts lo_e elements into its first vector
  const int lo_e = (int)(g.e0 - g.vbeg * VE);

  StatsAcc q;
  stats_init(q, c);
  // rolling prefetch: slot j % W holds vector j; it is refilled with vector
  // j + W as soon as vector j is reduced (one vector less in flight with the
  // KL sum, which needs the registers)
  constexpr int kVecs = kNSub * kNV;
  constexpr int W = kKL ? kWin - 1 : kWin;
#ifdef ASYMSPEC_TRACE
  if (threadIdx.x == 0) sm.t_mark[0] = __builtin_amdgcn_s_memrealtime();
#endif
  u4 buf[3][W];
  #pragma unroll
  for (int j = 0; j < W; ++j)
    #pragma unroll
    for (int s = 0; s < NS; ++s) buf[s][j] = buf_load_nt(r[s], off0 + (uint32_t)(vec_rel(j) * 16));
  #pragma unroll
  for (int j = 0; j < kVecs; ++j) {
    const int sl = j % W;
    if (kMask) {
      // elements outside the row become -inf (selects, no branches)
      const int e_lo = lo_e - (rel0 + vec_rel(j)) * VE;
      const int ilo = min(max(e_lo, 0), VE), ihi = min(max(e_lo + A.V, 0), VE);
      #pragma unroll
      for (int s = 0; s < NS; ++s) Elem<DT>::mask_to_neginf(buf[s][sl], ilo, ihi);
    }
    // masked elements have a = b = -inf, so f is NaN there: the boundary
    // chunks clamp the exponent of f
    if (j == 0)
      stats_vec<DT, KIND, kB1, DM, kKL, kMask, true>(A, c, buf[0][sl], buf[NS == 3 ? 1 : 0][sl],
                                                     buf[NS == 3 ? 2 : 0][sl], j, q);
    else
      stats_vec<DT, KIND, kB1, DM, kKL, kMask, false>(A, c, buf[0][sl], buf[NS == 3 ? 1 : 0][sl],
                                                      buf[NS == 3 ? 2 : 0][sl], j, q);
    if (j + W < kVecs) {
      #pragma unroll
      for (int s = 0; s < NS; ++s) buf[s][sl] = buf_load_nt(r[s], off0 + (uint32_t)(vec_rel(j + W) * 16));
    }
    // one vector's temporaries at a time
    __builtin_amdgcn_sched_barrier(0);
  }
  // In an interior chunk a fused logit that is not a number (a = b = -inf:
  // a token both views mask) makes some thread's f sum NaN; only then is the
  // chunk redone on the NaN-safe path.  The test is workgroup-wide, so every
  // thread takes the same path.
#ifdef ASYMSPEC_TRACE
  if (threadIdx.x == 0) sm.t_mark[1] = __builtin_amdgcn_s_memrealtime();
#endif
  if (kDraft && !kMask && __syncthreads_or(q.F.s != q.F.s)) return false;
  publish_stats<DT, KIND, DM, kKL>(A, g, m, rel0, q, sm);
  return true;
}

// Cross-family vocabularies, rows with no argmax to find (sampling drafts and
// a sampling fused bonus row): the drafter rows are read in their own order,
// contiguously, and t is gathered through the drafter-to-verifier map, so a
// shared token costs one gather instead of two (a and b through the
// verifier-to-drafter map) and the gathers hit the shorter verifier row.
// The statistics are the same sums over the shared set in another order;
// chunk m covers drafter vectors [m * kChunkVec, (m+1) * kChunkVec).
template <int DT, int KIND, bool kB1, int DM, bool kKL>
DEV void stats_dorder(const KArgs& A, const RowGeo& g, int m, Smem& sm) {
  constexpr int VE = Elem<DT>::VE;
  constexpr int ES = 16 / VE;
  const int lane = lane_id(), w = wave_id();
  const long long e0d = (long long)g.row * A.Vd;
  const long long vbeg = e0d / VE, vend = (e0d + A.Vd + VE - 1) / VE;
  const unsigned long long dbytes = (unsigned long long)A.B * (A.K + 1) * (unsigned long long)A.Vd * ES;
  unsigned long long span = (unsigned long long)(vend - vbeg) * 16ull;
  if (span > dbytes - (unsigned long long)vbeg * 16ull) span = dbytes - (unsigned long long)vbeg * 16ull;
  const __amdgpu_buffer_rsrc_t ra = make_rsrc((const char*)A.a + vbeg * 16, span);
  const __amdgpu_buffer_rsrc_t rb = make_rsrc((const char*)A.b + vbeg * 16, span);
  const long long last_full = (long long)(dbytes / 16ull), n_el = (long long)(dbytes / ES);
  const long long rel0 = (long long)m * kChunkVec + (long long)w * (64 * kNV) + lane;
  StatsAcc q;
  stats_init(q, g.c);
  #pragma unroll 1
  for (int kk = 0; kk < kNSub * kNV; ++kk) {
    const long long rv = rel0 + (long long)(kk / kNV) * kTileVec + (kk % kNV) * 64;
    const long long vi = vbeg + rv;
    const uint32_t off = (uint32_t)(rv * 16);
    u4 va = buf_load_nt(ra, off), vb = buf_load_nt(rb, off);
    u4 t2 = {0, 0, 0, 0}, a2 = t2, b2 = t2;
    #pragma unroll
    for (int e = 0; e < VE; ++e) {
      const long long jg = vi * VE + e;            // flat drafter index
      const long long jr = jg - e0d;               // drafter id in the row
      float xt = -INFINITY, xa = -INFINITY, xb = -INFINITY;
      const int x = (jr >= 0 && jr < A.Vd) ? A.inv[jr] : -1;
      if (x >= 0 && x < A.V) {
        xt = Elem<DT>::load_one(A.t, g.e0 + x);
        if (vi >= last_full && jg < n_el) {       // the partial vector at the array end
          xa = Elem<DT>::load_one(A.a, jg);
          xb = Elem<DT>::load_one(A.b, jg);
        } else {
          xa = Elem<DT>::get(va, e);
          xb = Elem<DT>::get(vb, e);
        }
      }
      Elem<DT>::put_one(t2, e, xt);
      Elem<DT>::put_one(a2, e, xa);
      Elem<DT>::put_one(b2, e, xb);
    }
    stats_vec<DT, KIND, kB1, DM, kKL, true, true>(A, g.c, t2, a2, b2, kk, q);
  }
  publish_stats<DT, KIND, DM, kKL>(A, g, m, rel0, q, sm);
}

template <int DT, int KIND, bool kB1, int DM, bool kKL = false>
DEV void stats_item(const KArgs& A, int row, int m, Smem& sm) {
  constexpr int VE = Elem<DT>::VE;
  const RowGeo g = row_geo<DT>(A, row);
  if (!KindTraits<KIND>::kArg && KindTraits<KIND>::NS == 3 && A.vmap != nullptr && inv_ok(A)) {
    stats_dorder<DT, KIND, kB1, DM, kKL>(A, g, m, sm);
    return;
  }
  const long long c0 = g.vbeg + (long long)m * kChunkVec, c1 = c0 + kChunkVec;
  bool done = false;
  if (A.vmap == nullptr && !has_tail(A, c0, c1)) {
    // a chunk whose vectors lie wholly inside the row needs no masking
    const bool interior = c0 * VE >= g.e0 && c1 * VE <= g.e0 + A.V;
    done = interior ? stats_fast<DT, KIND, kB1, DM, kKL, false>(A, g, m, sm)
                    : stats_fast<DT, KIND, kB1, DM, kKL, true>(A, g, m, sm);
  }
  if (!done) stats_slow<DT, KIND, kB1, DM, kKL>(A, g, m, sm);
}

}  // namespace asym

#endif  // ASYMSPEC_STATS_H_
