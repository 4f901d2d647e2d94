// Resolve items of one request: decide, pass 2 and pick (and, with early
// exit, the verdict on the first rows, which is a decide over those rows).
//
// decide  combines the chunk statistics of the request's K+1 rows into their
//         log-normalisers, gathers the draft tokens' logits, and classifies
//         each draft with Eq. 4 (or its sampling form) using only the bound
//         D in [0, ln 2] (Sec. 3.3): surely accepted, surely rejected, or
//         open (the outcome depends on D).  Alg. 1 stops at the first
//         rejection, so only the open drafts before the first sure rejection
//         and the rows that can emit need a second look at the logits.  A
//         greedy request with nothing open is finished here.
// pass 2  one chunk (or one of P2 parts of it) of every row that needs it:
//         the JSD partial of Eq. 3 and the sums over each 64-vector sub-block
//         of the residual max(0, p~ - q) (sampling drafts that can emit, and
//         a fused bonus row) or of the bonus weights of softmax(t_K / tau).
// pick    D for the open drafts, the final accept length, and the emitted
//         token: the fused argmax (greedy, Eq. 2) or an inverse-CDF draw with
//         the caller's uniform u_K; then every output of the request.

#ifndef ASYMSPEC_RESOLVE_H_
#define ASYMSPEC_RESOLVE_H_

#include "device.h"

namespace asym {

DEV uint64_t* dec_hdr(const KArgs& A, int req) {
  return A.dec + (size_t)req * (kDecHdr + (size_t)(A.K + 1) * kDecRow);
}
DEV uint64_t* dec_row(const KArgs& A, int req, int i) {
  return dec_hdr(A, req) + kDecHdr + (size_t)i * kDecRow;
}
DEV uint64_t* p2_rec(const KArgs& A, int req, int i, int m) {
  return A.rec2 + (((size_t)req * (A.K + 1) + i) * A.S + m) * kR2;
}

// Element-term constants of a row from its decision block.
DEV ResidConst resid_const(const KArgs& A, const uint32_t* cst) {
  return ResidConst{A.beta, __uint_as_float(cst[D_C]), __uint_as_float(cst[D_RF]),
                    __uint_as_float(cst[D_ISF]), __uint_as_float(cst[D_RQ]), __uint_as_float(cst[D_ISQ])};
}
DEV JsdConst jsd_const(const uint32_t* cst) {
  return JsdConst{__uint_as_float(cst[D_RA]), __uint_as_float(cst[D_RB]), __uint_as_float(cst[D_KAHI]),
                  __uint_as_float(cst[D_KALO]), __uint_as_float(cst[D_KBHI]), __uint_as_float(cst[D_KBLO])};
}

// ------------------------------------------------------------------ decide
// Classification of one row from its combined statistics: reference
// exponents R per slot and the sums Sp of exp2(x * c - R) (fp64), the
// maximum Marg of the argmax slot and the first index attaining it, and
// whether a and b differ.  Fills the row's decision block v (kDecRow words).
template <int DT>
DEV void classify_row(const KArgs& A, const RowGeo& g, const Gather& gq, float Marg,
                      const float (&R)[kSlots], const double (&Sp)[kSlots], double Wkl, int arg, bool neq,
                      uint32_t* v) {
  const int kind = g.kind;
  const bool draft = kind_draft(kind);
  const bool samp = kind_samp(kind);
  double L2[kSlots];
  #pragma unroll
  for (int s = 0; s < kSlots; ++s) L2[s] = (double)R[s] + log2_dbl(Sp[s]);
  const int gm = A.gate_mode;
  #pragma unroll
  for (int i = 0; i < kDecRow; ++i) v[i] = 0u;
  int decided = 1, accept = 0;
  double thr = 0.0;
  v[D_C] = __float_as_uint(g.c);
  if (draft) {
    const double ka = log2_dbl(Sp[sA]), kb = log2_dbl(Sp[sB]);
    const float kahi = (float)ka, kbhi = (float)kb;
    v[D_RA] = __float_as_uint(R[sA]);
    v[D_RB] = __float_as_uint(R[sB]);
    v[D_KAHI] = __float_as_uint(kahi);
    v[D_KALO] = __float_as_uint((float)(ka - (double)kahi));
    v[D_KBHI] = __float_as_uint(kbhi);
    v[D_KBLO] = __float_as_uint((float)(kb - (double)kbhi));
    const float fd = fuse_masked(gq.t, gq.a, gq.b, A.beta, A.delta_mode);
    // gates whose D is known here, so that the row is decided at once:
    // lambda (App. B), D = lambda * Delta(d), Delta the drafter views'
    // log-probability difference at the draft token; KL (App. G),
    // D = KL(P || Q) = E_P[a - b] - (LA - LB) from the statistics (a
    // negative rounding residue is 0; an undefined sum, only from an input
    // with b = -inf under a finite a, is +inf)
    double Dl = 0.0;
    const bool dknown = gm == ASYMSPEC_GATE_LAMBDA || gm == ASYMSPEC_GATE_KL;
    if (gm == ASYMSPEC_GATE_LAMBDA) {
      const double lpa = ((double)gq.a * (double)kL2E - L2[sA]) * kLn2;
      const double lpb1 = ((double)gq.b * (double)kL2E - L2[sB]) * kLn2;
      Dl = (double)A.lam * (lpa - lpb1);
    } else if (gm == ASYMSPEC_GATE_KL) {
      Dl = neq ? Wkl / Sp[sA] - (L2[sA] - L2[sB]) * kLn2 : 0.0;
      Dl = Dl != Dl ? INFINITY : (Dl < 0.0 ? 0.0 : Dl);
    }
    if (dknown) {
      v[D_GD_LO] = dlo(Dl);
      v[D_GD_HI] = dhi(Dl);
    }
    if (!samp) {
      // Eq. 4 in log form: ln p_t(d) - ln p_b(d) - ln gamma + D > 0
      const double lpt = ((double)gq.t * (double)kL2E - L2[sT]) * kLn2;
      const double lpb = ((double)gq.b * (double)kL2E - L2[sB]) * kLn2;
      double m0 = lpt - lpb - A.ln_gamma;
      if (m0 != m0) m0 = -INFINITY;
      const double lpd = ((double)fd * (double)kL2E - L2[sF]) * kLn2;
      v[D_LPD] = __float_as_uint((float)lpd);
      v[D_LPEMIT] = __float_as_uint((float)(((double)Marg * (double)kL2E - L2[sF]) * kLn2));
      v[D_ARG] = (uint32_t)arg;
      v[D_L2E_LO] = dlo(L2[sF]);
      v[D_L2E_HI] = dhi(L2[sF]);
      // D >= 0 for the divergence gates (and D = 0 when a == b bitwise),
      // D <= ln 2 for the JSD; outside those bounds the row stays open
      if (dknown) accept = m0 + Dl > 0.0;
      else if (gm == ASYMSPEC_GATE_FIXED || !neq) accept = m0 > 0.0;
      else if (m0 > 0.0) accept = 1;
      else if (gm == ASYMSPEC_GATE_CDA && m0 + kLn2 <= 0.0) accept = 0;
      else { decided = 0; thr = -m0; }
    } else {
      // accept iff u < min(1, p~(d) / (gamma_eff q(d))), i.e. ln u < x + D
      const bool t1 = kind == kSampleDraft1;
      const double L2q = t1 ? L2[sA] : L2[sAT];
      const double Sq = t1 ? Sp[sA] : Sp[sAT];
      const float Rq = t1 ? R[sA] : R[sAT];
      const double lpd = ((double)fd * (double)g.c - L2[sF]) * kLn2;
      v[D_LPD] = __float_as_uint((float)lpd);
      double lq;
      if (A.dp != nullptr) lq = gq.p > 0.0f ? ln_f(gq.p) : -INFINITY;
      else lq = ((double)gq.a * (double)g.c - L2q) * kLn2;
      double x;
      if (lpd == -INFINITY) x = -INFINITY;
      else if (lq == -INFINITY) x = INFINITY;
      else x = lpd - lq - A.ln_gamma;
      const double lnu = gq.u > 0.0f ? ln_f(gq.u) : -INFINITY;
      if (dknown) {
        if (lpd == -INFINITY) accept = 0;          // p~(d) = 0 rejects
        else if (lq == -INFINITY) accept = 1;      // q(d) = 0 accepts
        else accept = lnu < x + Dl;
      } else if (gm == ASYMSPEC_GATE_FIXED || !neq) {
        accept = lnu < x;
      } else if (lnu < x) {
        accept = 1;
      } else if (gm == ASYMSPEC_GATE_CDA && lnu >= x + kLn2) {
        accept = 0;
      } else {
        decided = 0;
        thr = lnu - x;
      }
      v[D_RF] = __float_as_uint(R[sF]);
      v[D_ISF] = __float_as_uint((float)(1.0 / Sp[sF]));
      v[D_RQ] = __float_as_uint(Rq);
      v[D_ISQ] = __float_as_uint((float)(1.0 / Sq));
      v[D_L2E_LO] = dlo(L2[sF]);
      v[D_L2E_HI] = dhi(L2[sF]);
    }
  } else if (kind == kGreedyBonusF || kind == kSampleBonusF) {
    // fused bonus row: greedy argmax of f, or a draw from softmax(f / tau),
    // drawn through the residual weights with q = 0 (q's reference exponent
    // +inf and scale 0 make its term vanish for every finite a)
    v[D_RF] = __float_as_uint(R[sF]);
    v[D_ISF] = __float_as_uint((float)(1.0 / Sp[sF]));
    v[D_RQ] = __float_as_uint(INFINITY);
    v[D_ISQ] = 0u;
    v[D_L2E_LO] = dlo(L2[sF]);
    v[D_L2E_HI] = dhi(L2[sF]);
    v[D_ARG] = (uint32_t)arg;
    v[D_LPEMIT] = __float_as_uint((float)(((double)Marg * (double)g.c - L2[sF]) * kLn2));
  } else {
    // bonus row (Alg. 1): greedy argmax of t, or a draw from softmax(t / tau)
    v[D_RF] = __float_as_uint(R[sT]);
    v[D_L2E_LO] = dlo(L2[sT]);
    v[D_L2E_HI] = dhi(L2[sT]);
    v[D_ARG] = (uint32_t)arg;
    v[D_LPEMIT] = __float_as_uint((float)(((double)Marg * (double)g.c - L2[sT]) * kLn2));
  }
  v[D_THR_LO] = dlo(thr);
  v[D_THR_HI] = dhi(thr);
  v[D_STATUS] = (decided ? kStDecided : 0) | (accept ? kStAccept : 0) | (draft ? kStDraft : 0) |
                (neq ? kStNeq : 0);
}

// The decision of request req (Alg. 1, Eq. 2-4) from the statistics records
// of its first nread rows, into sm.rows (one decision block per row) and
// sm.req (first sure rejection, pass-2 tasks, whether the request is final
// without pass 2).  Rows from nread on (early exit: they follow a sure
// rejection and were not read) get placeholder blocks.  Thread (i, ch) of a
// group of rows takes record ch of row i, so all records arrive in one round
// trip; the row's maxima, sums, argmax and a-vs-b flag are combined (for
// S <= 16 within the 16 lanes of a DPP row given to each row, else through
// LDS in chunk order) and the row's first thread classifies it.  Whole
// workgroup; S must not exceed kThreads.
template <int DT>
DEV void decide_request(const KArgs& A, int req, Smem& sm, int nread) {
  const int lane = lane_id(), w = wave_id(), tid = w * 64 + lane;
  const int K = A.K, S = A.S, nrow = K + 1;
  const bool dpp = S <= 16;                     // a row's chunks in one DPP row
  const int stride = dpp ? 16 : S;              // lanes per row
  const int rpg = kThreads / stride;            // rows per group
  const int li = tid / stride, ch = tid - li * stride;
  // the last statistics item read in list order is about the last to
  // finish: a waiting workgroup polls its record only
  const uint64_t* sentinel = A.rec1 + (((size_t)req * nrow + (nread - 1)) * S + (S - 1)) * kR1 + R1_MARG;
  bool all_in = true;
  for (int r0 = 0; r0 < nread; r0 += rpg) {
    const int nr = min(rpg, nread - r0);
    const bool have = li < nr && ch < S;
    const int i = r0 + (have ? li : 0);
    // first requests: the records, the draft token and its logits (row
    // leaders), then the temperature; none waits for another but the
    // logits for the token
    const uint64_t* base = A.rec1 + ((size_t)(req * nrow + i) * S + ch) * kR1;
    uint64_t r[R1_USED];
    #pragma unroll
    for (int j = 0; j < R1_USED; ++j) r[j] = have ? ld_tag(base + j) : ((uint64_t)A.epoch << 32);
    Gather gq{0.0f, 0.0f, 0.0f, 1.0f, 0.0f};
    if (have && ch == 0) gq = sgather<DT>(A, row_span<DT>(A, req * nrow + i));
    const RowGeo g = row_geo<DT>(A, req * nrow + i);
    bool first = true;
    all_in = load_tagged(A, sentinel, [&]() {
      if (first) {
        first = false;
        bool ok = true;
        #pragma unroll
        for (int j = 0; j < R1_USED; ++j) ok = ok && tag_ok(r[j], A.epoch);
        return ok;
      }
      // a slot that carries the epoch is final: only the others are read
      // again
      bool ok = true;
      #pragma unroll
      for (int j = 0; j < R1_USED; ++j) {
        if (have && !tag_ok(r[j], A.epoch)) r[j] = ld_tag(base + j);
        ok = ok && tag_ok(r[j], A.epoch);
      }
      return ok;
    }) && all_in;
    if (dpp) {
      // the row's lanes: maxima, then the rescaled sums (fp64), the argmax
      // among the chunks holding the maximum, and the a-vs-b flag; lanes
      // without a chunk contribute nothing
      float Rr[kSlots];
      #pragma unroll
      for (int s = 0; s < kSlots; ++s) Rr[s] = row16_max(have ? payf(r[R1_R + s]) : kFloorM);
      const float Marg = row16_max(have ? payf(r[R1_MARG]) : kFloorM);
      double Sp[kSlots];
      #pragma unroll
      for (int s = 0; s < kSlots; ++s)
        Sp[s] = row16_sum(have ? (double)(payf(r[R1_S + s]) * __builtin_amdgcn_exp2f(payf(r[R1_R + s]) - Rr[s]))
                               : 0.0);
      const double Wkl =
          row16_sum(have ? (double)(payf(r[R1_W]) * __builtin_amdgcn_exp2f(payf(r[R1_R + sA]) - Rr[sA])) : 0.0);
      const int arg = row16_min(have && payf(r[R1_MARG]) == Marg ? (int)pay(r[R1_ARG]) : 0x7FFFFFFF);
      const int nq = row16_or(have ? (int)pay(r[R1_NEQ]) : 0);
      if (have && ch == 0) classify_row<DT>(A, g, gq, Marg, Rr, Sp, Wkl, arg, nq != 0, sm.rows[i]);
      __syncthreads();
      continue;
    }
    // row references and the argmax slot's row maximum: every thread of the
    // row reads the row's records from LDS
    if (have) {
      #pragma unroll
      for (int s = 0; s < kSlots; ++s) sm.dm[tid][s] = payf(r[R1_R + s]);
      sm.dmarg[tid] = payf(r[R1_MARG]);
    }
    __syncthreads();
    float Rr[kSlots], Marg = kFloorM;
    #pragma unroll
    for (int s = 0; s < kSlots; ++s) Rr[s] = kFloorM;
    if (have) {
      const int t0 = li * S;
      for (int c = 0; c < S; ++c) {
        #pragma unroll
        for (int s = 0; s < kSlots; ++s) Rr[s] = fmaxf(Rr[s], sm.dm[t0 + c][s]);
        Marg = fmaxf(Marg, sm.dmarg[t0 + c]);
      }
    }
    // this chunk's terms of the row sums, rescaled to the row's reference
    // (the factor 2^(R_chunk - R_row) <= 1 in fp32: its error is far below
    // that of the fp32 chunk sums it scales)
    if (have) {
      #pragma unroll
      for (int s = 0; s < kSlots; ++s)
        sm.dt[tid][s] = (double)(payf(r[R1_S + s]) * __builtin_amdgcn_exp2f(payf(r[R1_R + s]) - Rr[s]));
      sm.dw[tid] = (double)(payf(r[R1_W]) * __builtin_amdgcn_exp2f(payf(r[R1_R + sA]) - Rr[sA]));
      sm.darg[tid] = payf(r[R1_MARG]) == Marg ? (int)pay(r[R1_ARG]) : 0x7FFFFFFF;
      sm.dneq[tid] = (int)pay(r[R1_NEQ]);
    }
    __syncthreads();
    if (have && ch == 0) {
      double Sp[kSlots];
      #pragma unroll
      for (int s = 0; s < kSlots; ++s) Sp[s] = 0.0;
      int arg = 0x7FFFFFFF, nq = 0;
      double Wkl = 0.0;
      for (int c = 0; c < S; ++c) {
        #pragma unroll
        for (int s = 0; s < kSlots; ++s) Sp[s] += sm.dt[tid + c][s];
        Wkl += sm.dw[tid + c];
        arg = min(arg, sm.darg[tid + c]);
        nq |= sm.dneq[tid + c];
      }
      classify_row<DT>(A, g, gq, Marg, Rr, Sp, Wkl, arg, nq != 0, sm.rows[i]);
    }
    __syncthreads();
  }
  if (nread < nrow) {
    // unread rows: decided, not accepted, outputs not a number
    for (int k = tid; k < (nrow - nread) * kDecRow; k += kThreads) {
      const int i = nread + k / kDecRow, j = k - (k / kDecRow) * kDecRow;
      uint32_t v = 0u;
      if (j == D_STATUS) v = kStDecided | kStDraft | kStSkip;
      else if (j == D_LPD || j == D_LPEMIT) v = 0x7FC00000u;
      else if (j == D_GD_HI) v = 0x7FF80000u;
      sm.rows[i][j] = v;
    }
    __syncthreads();
  }
  // request level (wave 0, lane i = row i): the first sure rejection j*, and
  // the rows pass 2 must look at
  if (w == 0) {
    const float tau = sload_f32(A.tau, req);
    const bool samp = tau > 0.0f;
    const bool row_ok = lane <= K;
    const uint32_t st = row_ok ? sm.rows[lane][D_STATUS] : 0u;
    const bool is_draft = lane < K;
    const bool decided = st & kStDecided, accept = st & kStAccept, neq = st & kStNeq;
    const int jr = wave_min_i(is_draft && decided && !accept ? lane : 0x7FFFFFFF);
    const int jstar = jr == 0x7FFFFFFF ? K : jr;
    const bool open = is_draft && lane < jstar && !decided;
    uint32_t task = 0;
    // pass 2 computes D (JSD, or KL for that gate) for the open rows and,
    // when the gate output is wanted, for every row whose views differ; the
    // lambda gate's D is known here
    const bool dknown = A.gate_mode == ASYMSPEC_GATE_LAMBDA || A.gate_mode == ASYMSPEC_GATE_KL;
    if (is_draft && !dknown && (open || (A.want_gate && neq))) task |= kTaskJsd;
    if (samp && is_draft && (open || lane == jstar)) task |= kTaskRes;
    // the bonus draw: softmax(t / tau), or the fused row's p~ as a residual
    if (samp && lane == K && jstar == K) task |= A.fuse_bonus ? kTaskRes : kTaskBonus;
    const unsigned long long tmask = __ballot(task != 0);
    const bool fin = !samp && !__any((task & kTaskJsd) != 0);
    if (row_ok) sm.rows[lane][D_TASK] = task;
    if (lane == 0) {
      sm.req[R_J] = (uint32_t)jstar;
      sm.req[R_TASK_LO] = (uint32_t)tmask;
      sm.req[R_TASK_HI] = (uint32_t)(tmask >> 32);
      sm.req[R_FIN] = fin ? 1u : 0u;
      sm.req[R_SAMP] = samp ? 1u : 0u;
      sm.req[R_FAIL] = all_in ? 0u : 1u;
    }
  }
  __syncthreads();
}

// Every output of request `req`, written by wave 0: lane i < K holds draft
// i's fused log-probability and D_i.
DEV void write_outputs(const KArgs& A, int req, int j, int next, float lp_next, float lpd_lane,
                       double d_lane, bool skip_lane) {
  const int lane = lane_id();
  const int K = A.K;
  if (lane < K) {
    // a row early exit did not read has no outputs
    if (skip_lane) {
      lpd_lane = __builtin_nanf("");
      d_lane = __builtin_nan("");
    }
    A.flp_out[(size_t)req * (K + 1) + lane] = lpd_lane;
    if (A.gate_out != nullptr) {
      // gamma_eff = gamma (fixed gate) or gamma exp(-D) (Eq. 3 and the
      // KL and lambda variants)
      float ge = A.gate_mode == ASYMSPEC_GATE_FIXED ? A.gamma : (float)((double)A.gamma * exp(-d_lane));
      if (skip_lane) ge = __builtin_nanf("");
      A.gate_out[((size_t)req * K + lane) * 2 + 0] = (float)d_lane;
      A.gate_out[((size_t)req * K + lane) * 2 + 1] = ge;
    }
  }
  if (lane == 0) {
    A.acc_out[req] = j;
    A.next_out[req] = next;
    A.flp_out[(size_t)req * (K + 1) + K] = lp_next;
  }
}

// Early exit: the verdict of request req (kVerdictRead or kVerdictSkip),
// the same in every thread.  Whole workgroup.
DEV uint32_t load_verdict(const KArgs& A, int req, Smem& sm) {
  if (wave_id() == 0 && lane_id() == 0) {
    // the verdict is written long before most readers come: a first read
    // that may be served by this XCD's L2 (a stale line carries an older
    // epoch and falls through to the polling read)
    const uint64_t* p = dec_hdr(A, req) + H_VERDICT;
    uint64_t v = __hip_atomic_load(const_cast<uint64_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (!tag_ok(v, A.epoch)) v = wait_tag(p, A);
    // a verdict that never arrived (counted as a timeout) reads every row
    sm.flags[3] = (tag_ok(v, A.epoch) && pay(v) == kVerdictSkip) ? 1 : 0;
  }
  __syncthreads();
  const uint32_t r = sm.flags[3] ? kVerdictSkip : kVerdictRead;
  __syncthreads();
  return r;
}

// The decide item, and (verdict) the early-exit verdict item: it classifies
// the first G rows only, and a sure rejection among them (Alg. 1 stops at
// the first rejection) means the other rows need not be read.  Both share
// one instance of decide_request.
template <int DT>
DEV void decide_item(const KArgs& A, int req, Smem& sm, bool verdict) {
  const int lane = lane_id(), w = wave_id(), tid = w * 64 + lane;
  const int K = A.K, nrow = K + 1;
  int nread = nrow;
  if (verdict || (A.sc.ee && load_verdict(A, req, sm) == kVerdictSkip)) nread = A.sc.G;
  decide_request<DT>(A, req, sm, nread);
  // a timed-out wait for the records: the request fails (an early-exit
  // verdict then reads every row)
  const bool failed = sm.req[R_FAIL] != 0u;
  if (verdict) {
    if (w == 0) {
      const uint32_t st = lane < nread ? sm.rows[lane][D_STATUS] : 0u;
      const bool skip = !failed && __any((st & kStDecided) != 0u && (st & kStAccept) == 0u);
      if (lane == 0) st_tag(dec_hdr(A, req) + H_VERDICT, skip ? kVerdictSkip : kVerdictRead, A.epoch);
    }
    return;
  }
  // publish: every word of every row block, then the header
  for (int k = tid; k < nrow * D_USED; k += kThreads) {
    const int i = k / D_USED, j = k - i * D_USED;
    st_tag(dec_row(A, req, i) + j, sm.rows[i][j], A.epoch);
  }
  const bool fin = sm.req[R_FIN] != 0u;
  __syncthreads();   // the header goes out after every row word
  if (w == 0) {
    uint64_t* hdr = dec_hdr(A, req);
    if (lane == 0) {
      st_tag(hdr + H_J, sm.req[R_J], A.epoch);
      st_tag(hdr + H_TASK_LO, sm.req[R_TASK_LO], A.epoch);
      st_tag(hdr + H_TASK_HI, sm.req[R_TASK_HI], A.epoch);
      st_tag(hdr + H_SAMP, sm.req[R_SAMP], A.epoch);
      st_tag(hdr + H_STATE, failed ? kStateFailed : (fin ? kStateFinal : kStatePending), A.epoch);
      if (failed) A.acc_out[req] = -1;
    }
    if (fin && !failed) {
      // greedy with no open draft: accept_len = j*, emit the fused argmax of
      // row j* (Eq. 2) or the verifier argmax of the bonus row (Alg. 1)
      const int jstar = (int)sm.req[R_J];
      const int next = (int)sm.rows[jstar][D_ARG];
      const float lpn = __uint_as_float(sm.rows[jstar][D_LPEMIT]);
      const float lpd = lane < K ? __uint_as_float(sm.rows[lane][D_LPD]) : 0.0f;
      // D of the rows: 0 (no view difference, or no D wanted) or the
      // lambda gate's, known here
      const double dl = (lane < K && (A.gate_mode == ASYMSPEC_GATE_LAMBDA || A.gate_mode == ASYMSPEC_GATE_KL))
                            ? u2d(sm.rows[lane][D_GD_LO], sm.rows[lane][D_GD_HI])
                            : 0.0;
      const bool skip = lane <= K && (sm.rows[lane][D_STATUS] & kStSkip) != 0u;
      write_outputs(A, req, jstar, next, lpn, lpd, dl, skip);
    }
  }
}

// The published decision of request req into sm.req and sm.rows: the
// header and every row block are requested at once and polled together.
// Returns the request's state (kStateFinal or kStatePending).  Whole
// workgroup.
DEV uint32_t load_decision(const KArgs& A, int req, Smem& sm) {
  const int tid = wave_id() * 64 + lane_id();
  const int nrow = A.K + 1;
  const int nw = H_USED + nrow * D_USED;
  constexpr int kPer = ((kMaxK + 1) * D_USED + H_USED + kThreads - 1) / kThreads;
  uint64_t v[kPer];
  auto load = [&]() {
    bool ok = true;
    #pragma unroll
    for (int q = 0; q < kPer; ++q) {
      const int k = tid + q * kThreads;
      if (k < nw) {
        const uint64_t* p = k < H_USED ? dec_hdr(A, req) + k
                                       : dec_row(A, req, (k - H_USED) / D_USED) + (k - H_USED) % D_USED;
        v[q] = ld_tag(p);
        ok = ok && tag_ok(v[q], A.epoch);
      }
    }
    return ok;
  };
  // the header goes out after the rows: a waiting workgroup polls it only
  const bool in = load_tagged(A, dec_hdr(A, req) + H_STATE, load);
  #pragma unroll
  for (int q = 0; q < kPer; ++q) {
    const int k = tid + q * kThreads;
    if (k < nw) {
      if (k >= H_USED) {
        const int i = (k - H_USED) / D_USED;
        sm.rows[i][(k - H_USED) % D_USED] = pay(v[q]);
      } else if (k == H_STATE) {
        sm.req[R_FIN] = pay(v[q]) == kStateFinal ? 1u : 0u;
        sm.req[R_FAIL] = (!in || pay(v[q]) == kStateFailed) ? 1u : 0u;
      } else if (k == H_J) {
        sm.req[R_J] = pay(v[q]);
      } else if (k == H_TASK_LO) {
        sm.req[R_TASK_LO] = pay(v[q]);
      } else if (k == H_TASK_HI) {
        sm.req[R_TASK_HI] = pay(v[q]);
      } else {
        sm.req[R_SAMP] = pay(v[q]);
      }
    }
  }
  if (!in && tid == 0) sm.req[R_FAIL] = 1u;
  __syncthreads();
  if (sm.req[R_FAIL] != 0u) return kStateFailed;
  return sm.req[R_FIN] != 0u ? (uint32_t)kStateFinal : (uint32_t)kStatePending;
}

// ------------------------------------------------------------------ pass 2
// Pass-2 sums of one thread over its nk vectors (64 apart) of a chunk part;
// the weight sum of vector k goes to seg[k].
// kMode 0: interior part (no masking); 1: masked, branch-free; 2: generic
// (one vector at a time, array-end repair).  kGF vectors per group (4, or
// fewer when a lane has fewer).
// kNb: a and b differ somewhere in the row; otherwise b is a bitwise copy of
// a and a's vectors stand in for it (such a row has no divergence task).
template <int DT, int kMode, int DM, bool kNb, bool kResOnly = false, int kGF = 4>
DEV void pass2_sums(const KArgs& A, const RowGeo& g, long long rel0, int nk, bool dj_in, bool dr_in, bool db_in,
                    const ResidConst& rk, const JsdConst& jk, float& accj, float (&seg)[kSegPerLane]) {
  constexpr int VE = Elem<DT>::VE;
  constexpr int kG = kMode == 2 ? 1 : kGF;    // vectors per group
  // kResOnly: the row's only task is the residual (the usual emitting row),
  // an instance without the other tasks' code
  const bool dj = kResOnly ? false : dj_in, dr = kResOnly ? true : dr_in, db = kResOnly ? false : db_in;
  const bool nt = dr || db, nab = dj || dr;
  const __amdgpu_buffer_rsrc_t rt = row_rsrc(A, A.t, g);
  const __amdgpu_buffer_rsrc_t ra = row_rsrc(A, nab ? A.a : A.t, g);
  const __amdgpu_buffer_rsrc_t rb = row_rsrc(A, nab ? A.b : A.t, g);
  #pragma unroll 1
  for (int k0 = 0; k0 < nk; k0 += kG) {
    u4 vt[kG], va[kG], vb[kG];
    #pragma unroll
    for (int k = 0; k < kG; ++k) {
      const uint32_t off = (uint32_t)((rel0 + (long long)(k0 + k) * 64) * 16);
      vt[k] = nt ? buf_load_nt(rt, off) : u4{0, 0, 0, 0};
      va[k] = nab ? buf_load_nt(ra, off) : u4{0, 0, 0, 0};
      if (kNb) vb[k] = nab ? buf_load_nt(rb, off) : u4{0, 0, 0, 0};
    }
    #pragma unroll
    for (int k = 0; k < kG; ++k) {
      const long long vi = g.vbeg + rel0 + (long long)(k0 + k) * 64;
      if (kMode == 1) {
        mask_vec<DT>(A, g, vi, vt[k]);
        mask_vec<DT>(A, g, vi, va[k]);
        if (kNb) mask_vec<DT>(A, g, vi, vb[k]);
      } else if (kMode == 2) {
        if (nt) fix_vec<DT>(A, g, A.t, vi, vt[k]);
        if (A.vmap != nullptr) {
          map_vecs<DT>(A, g, vi, vt[k], va[k], vb[k], nab);
        } else if (nab) {
          fix_vec<DT>(A, g, A.a, vi, va[k]);
          if (kNb) fix_vec<DT>(A, g, A.b, vi, vb[k]);
        }
      }
      if (!kNb) vb[k] = va[k];
      // each task's element terms under its own (uniform) branch, so that a
      // row without a task never evaluates that task's terms
      if (dj) {
        float vj[VE];
        #pragma unroll
        for (int e = 0; e < VE; ++e) {
          const float xa = Elem<DT>::get(va[k], e), xb = Elem<DT>::get(vb[k], e);
          vj[e] = jsd_elem(xa, xb, jk);
        }
        #pragma unroll
        for (int st = 1; st < VE; st <<= 1)
          #pragma unroll
          for (int e = 0; e + st < VE; e += 2 * st) vj[e] += vj[e + st];
        accj += vj[0];
      }
      if (dr || db) {
        float vr[VE];
        #pragma unroll
        for (int e = 0; e < VE; ++e) {
          const float xa = Elem<DT>::get(va[k], e), xb = Elem<DT>::get(vb[k], e);
          const float xt = Elem<DT>::get(vt[k], e);
          vr[e] = dr ? resid_elem<DM>(xt, xa, xb, rk) : bonus_elem(xt, rk.c, rk.Rf);
        }
        #pragma unroll
        for (int st = 1; st < VE; st <<= 1)
          #pragma unroll
          for (int e = 0; e + st < VE; e += 2 * st) vr[e] += vr[e + st];
        // vector k0 + k: selects on the run-time group start keep every
        // sum in its own register
        #pragma unroll
        for (int q = 0; q < kSegPerLane; q += kG) seg[q + k] += (q == k0) ? vr[0] : 0.0f;
      }
    }
  }
}

template <int DT, int DM, bool kNb, int kGF>
DEV void pass2_sums_any(const KArgs& A, const RowGeo& g, long long rel0, int nk, long long c0, long long c1,
                        bool dj, bool dr, bool db, const ResidConst& rk, const JsdConst& jk, float& accj,
                        float (&seg)[kSegPerLane]) {
  constexpr int VE = Elem<DT>::VE;
  if (A.vmap != nullptr || has_tail(A, c0, c1))
    pass2_sums<DT, 2, DM, kNb>(A, g, rel0, nk, dj, dr, db, rk, jk, accj, seg);
  else if (dr && !dj && !db && c0 * VE >= g.e0 && c1 * VE <= g.e0 + A.V)
    pass2_sums<DT, 0, DM, kNb, true, kGF>(A, g, rel0, nk, dj, dr, db, rk, jk, accj, seg);
  else if (dr && !dj && !db)
    pass2_sums<DT, 1, DM, kNb, true, kGF>(A, g, rel0, nk, dj, dr, db, rk, jk, accj, seg);
  else if (c0 * VE >= g.e0 && c1 * VE <= g.e0 + A.V)
    pass2_sums<DT, 0, DM, kNb, false, kGF>(A, g, rel0, nk, dj, dr, db, rk, jk, accj, seg);
  else
    pass2_sums<DT, 1, DM, kNb, false, kGF>(A, g, rel0, nk, dj, dr, db, rk, jk, accj, seg);
}

template <int DT, int DM>
DEV void pass2_item(const KArgs& A, int req, int sub, Smem& sm) {
  const int lane = lane_id(), w = wave_id();
  // part `part` of chunk m: kChunkVec / P2 vectors, wave w's nk * 64 of
  // them from pbase + w * 64 * nk, lane l every 64th from there
  const int m = sub / A.P2, part = sub - m * A.P2;
  const int nk = kSegPerLane / A.P2;
  const long long pbase = (long long)m * kChunkVec + (long long)part * (kChunkVec / A.P2);
  if (load_decision(A, req, sm) != kStatePending) return;
  unsigned long long tmask = (unsigned long long)sm.req[R_TASK_LO] | ((unsigned long long)sm.req[R_TASK_HI] << 32);
  // only rows 0..K of the request (K + 1 <= 64)
  if (A.K + 1 < 64) tmask &= (1ull << (A.K + 1)) - 1ull;
  while (tmask != 0) {
    const int i = __builtin_ctzll(tmask);
    tmask &= tmask - 1;
    const uint32_t* cst = sm.rows[i];
    const uint32_t task = cst[D_TASK];
    const RowGeo g = row_span<DT>(A, req * (A.K + 1) + i);
    const bool dj = task & kTaskJsd, dr = task & kTaskRes, db = task & kTaskBonus;
    const ResidConst rk = resid_const(A, cst);
    const JsdConst jk = jsd_const(cst);
    const long long rel0 = pbase + (long long)w * 64 * nk + lane;
    const long long c0 = g.vbeg + pbase, c1 = c0 + kChunkVec / A.P2;
    float accj = 0.0f, seg[kSegPerLane];
    #pragma unroll
    for (int k = 0; k < kSegPerLane; ++k) seg[k] = 0.0f;
    if (task != 0) {
      // a row with a == b bitwise has no divergence task and skips b
      const bool nbr = (cst[D_STATUS] & kStNeq) != 0u || A.vmap != nullptr;
      if (nk >= 4) {
        if (nbr) pass2_sums_any<DT, DM, true, 4>(A, g, rel0, nk, c0, c1, dj, dr, db, rk, jk, accj, seg);
        else pass2_sums_any<DT, DM, false, 4>(A, g, rel0, nk, c0, c1, dj, dr, db, rk, jk, accj, seg);
      } else if (nk >= 2) {
        if (nbr) pass2_sums_any<DT, DM, true, 2>(A, g, rel0, nk, c0, c1, dj, dr, db, rk, jk, accj, seg);
        else pass2_sums_any<DT, DM, false, 2>(A, g, rel0, nk, c0, c1, dj, dr, db, rk, jk, accj, seg);
      } else {
        if (nbr) pass2_sums_any<DT, DM, true, 1>(A, g, rel0, nk, c0, c1, dj, dr, db, rk, jk, accj, seg);
        else pass2_sums_any<DT, DM, false, 1>(A, g, rel0, nk, c0, c1, dj, dr, db, rk, jk, accj, seg);
      }
    }
    // this wave's sub-block sums: lane k < nk publishes the wave's k-th
    // sub-block; the part's JSD partial goes through LDS
    float mine = 0.0f;
    #pragma unroll
    for (int k = 0; k < kSegPerLane; ++k) {
      if (k < nk) {
        const float sk = wave_sum(seg[k]);
        mine = lane == k ? sk : mine;
      }
    }
    uint64_t* rec = p2_rec(A, req, i, m);
    if (lane < nk)
      st_tag(rec + P2_SEG + part * (kSubPerChunk / A.P2) + w * nk + lane, __float_as_uint(mine), A.epoch);
    const float wj = wave_sum(accj);
    if (lane == 0) sm.wj[w] = wj;
    __syncthreads();
    if (threadIdx.x == 0) {
      float v = 0.0f;
      #pragma unroll
      for (int q = 0; q < kWaves; ++q) v += sm.wj[q];
      st_tag(rec + P2_J + part, __float_as_uint(v), A.epoch);
    }
    __syncthreads();
  }
}

// -------------------------------------------------------------------- pick
// Sub-block sums a lane of the pick holds at once.
constexpr int kPickRun = 8;

// The tagged slots of sub-blocks [s0, s0 + n) (n <= kPickRun) of pass-2
// record area rec, requested at once and polled until all are in (bounded;
// ok cleared on a timeout); the other entries of v are zero.
DEV void load_sub_run(const KArgs& A, const uint64_t* rec, int s0, int n, float (&v)[kPickRun], bool& ok) {
  auto slot = [&](int sb) { return rec + (size_t)(sb / kSubPerChunk) * kR2 + P2_SEG + sb % kSubPerChunk; };
  const uint64_t zero = (uint64_t)A.epoch << 32;
  uint64_t r[kPickRun];
  #pragma unroll
  for (int j = 0; j < kPickRun; ++j) r[j] = j < n ? ld_tag(slot(s0 + j)) : zero;
  Poll pl;
  for (;;) {
    bool in = true;
    #pragma unroll
    for (int j = 0; j < kPickRun; ++j) in = in && tag_ok(r[j], A.epoch);
    if (in) break;
    if (!pl.again(A)) {
      ok = false;
      break;
    }
    #pragma unroll
    for (int j = 0; j < kPickRun; ++j) r[j] = j < n ? ld_tag(slot(s0 + j)) : zero;
  }
  #pragma unroll
  for (int j = 0; j < kPickRun; ++j) v[j] = payf(r[j]);
}

// Inverse-CDF draw over row i of request req: the first element x whose
// cumulative weight exceeds u * total, with the weights of pass 2 (residual
// for drafts, bonus weights for the bonus row) recomputed by the same element
// functions.  Pass 2's sums locate the 64-vector sub-block that holds it and
// a scan of that sub-block the element; wave 0 does both, without barriers.
// Row constants are in sm.rows[i].  Returns -1 when no element carries
// weight; otherwise the element's index, and, when the scan itself found it,
// sm.flags[2] = 1 and its logit (f for drafts, t for the bonus row) in
// sm.dd[3].  Whole workgroup.
template <int DT, int DM>
DEV int cdf_pick(const KArgs& A, int req, int i, double u, bool bonus, Smem& sm, bool& ok) {
  constexpr int VE = Elem<DT>::VE;
  const int lane = lane_id(), w = wave_id();
  if (w == 0) {
    const RowGeo g = row_span<DT>(A, req * (A.K + 1) + i);
    const int nsub = A.S * kSubPerChunk;
    // lane l holds sub-blocks [l * per, l * per + per) in runs of kPickRun
    const int per = (nsub + 63) / 64;
    const int nrun = (per + kPickRun - 1) / kPickRun;
    const int s0 = min(lane * per, nsub), s1 = min(s0 + per, nsub);
    const uint64_t* rec = p2_rec(A, req, i, 0);
    float v[kPickRun];
    double lsum = 0.0;
    for (int q = 0; q < nrun; ++q) {
      const int a = min(s0 + q * kPickRun, s1);
      load_sub_run(A, rec, a, min(kPickRun, s1 - a), v, ok);
      #pragma unroll
      for (int j = 0; j < kPickRun; ++j) lsum += (double)v[j];
    }
    double incl, excl;
    wave_scan_d(lsum, incl, excl);
    const double total = readlane_d(incl, 63);
    int pick = -1;
    if (total > 0.0) {
      const double target = u * total;
      // the sub-block: the first with weight whose cumulative sum passes the
      // target, else (rounding left the target at the total) the last one
      // with weight; only the lane whose run holds it walks its run again
      int cand = 0x7FFFFFFF, last = -1;
      double cb = 0.0, lb = 0.0;
      const bool mine = incl > target && excl <= target;
      const bool any_w = lsum > 0.0;
      if (mine || any_w) {
        double run = excl;
        for (int q = 0; q < nrun; ++q) {
          const int a = min(s0 + q * kPickRun, s1);
          if (nrun > 1) load_sub_run(A, rec, a, min(kPickRun, s1 - a), v, ok);
          #pragma unroll
          for (int j = 0; j < kPickRun; ++j) {
            const double nx = run + (double)v[j];
            if (v[j] > 0.0f && nx > target && cand == 0x7FFFFFFF) { cand = a + j; cb = run; }
            if (v[j] > 0.0f) { last = a + j; lb = run; }
            run = nx;
          }
        }
      }
      int sel = wave_min_i(cand);
      double before;
      if (sel == 0x7FFFFFFF) {
        const int neg = wave_min_i(last >= 0 ? -last : 0x7FFFFFFF);
        sel = neg == 0x7FFFFFFF ? -1 : -neg;
        const unsigned long long src = __ballot(last == sel);
        before = __shfl(lb, src ? (int)__builtin_ctzll(src) : 0, 64);
      } else {
        const unsigned long long src = __ballot(cand == sel);
        before = __shfl(cb, (int)__builtin_ctzll(src), 64);
      }
      if (sel >= 0) {
        // lane l scans vector l of the sub-block
        const int ch = sel / kSubPerChunk, sub = sel % kSubPerChunk;
        const long long sv0 = g.vbeg + (long long)ch * kChunkVec + (long long)sub * 64;
        const long long vi = sv0 + lane;
        const uint32_t* cst = sm.rows[i];
        const ResidConst rk = resid_const(A, cst);
        const __amdgpu_buffer_rsrc_t rt = row_rsrc(A, A.t, g);
        const __amdgpu_buffer_rsrc_t ra = row_rsrc(A, bonus ? A.t : A.a, g);
        // a row whose a and b are equal bitwise reads a for b (same weights)
        const bool nb = !bonus && (cst[D_STATUS] & kStNeq) != 0u;
        const __amdgpu_buffer_rsrc_t rb = row_rsrc(A, nb ? A.b : A.t, g);
        const uint32_t off = (uint32_t)((vi - g.vbeg) * 16);
        u4 vt = buf_load(rt, off);
        u4 va = bonus ? vt : buf_load(ra, off);
        u4 vb = nb ? buf_load(rb, off) : u4{0, 0, 0, 0};
        if (A.vmap != nullptr) {
          fix_vec<DT>(A, g, A.t, vi, vt);
          map_vecs<DT>(A, g, vi, vt, va, vb, !bonus);
          if (bonus) va = vt;
        } else if (has_tail(A, sv0, sv0 + 64)) {
          fix_vec<DT>(A, g, A.t, vi, vt);
          if (!bonus) fix_vec<DT>(A, g, A.a, vi, va);
          if (nb) fix_vec<DT>(A, g, A.b, vi, vb);
        } else {
          mask_vec<DT>(A, g, vi, vt);
          mask_vec<DT>(A, g, vi, va);
          mask_vec<DT>(A, g, vi, vb);
        }
        if (!nb) vb = va;
        float x[VE];
        double vsum = 0.0;
        #pragma unroll
        for (int e = 0; e < VE; ++e) {
          const float xt = Elem<DT>::get(vt, e);
          x[e] = bonus ? bonus_elem(xt, rk.c, rk.Rf)
                       : resid_elem<DM>(xt, Elem<DT>::get(va, e), Elem<DT>::get(vb, e), rk);
          vsum += (double)x[e];
        }
        double vin, vex;
        wave_scan_d(vsum, vin, vex);
        double run = before + vex;
        int first_ok = 0x7FFFFFFF, last_pos = -1;
        float fx = 0.0f;
        #pragma unroll
        for (int e = 0; e < VE; ++e) {
          run += (double)x[e];
          const int idx = (int)(vi * VE + e - g.e0);
          if (x[e] > 0.0f && run > target && first_ok == 0x7FFFFFFF) {
            first_ok = idx;
            const float xt = Elem<DT>::get(vt, e);
            fx = bonus ? xt
                       : fuse_masked(xt, Elem<DT>::get(va, e), Elem<DT>::get(vb, e), A.beta, A.delta_mode);
          }
          if (x[e] > 0.0f) last_pos = idx;
        }
        pick = wave_min_i(first_ok);
        if (pick == 0x7FFFFFFF) {
          // rounding left the target past the sub-block's own sum: its
          // last element with weight
          const int neg = wave_min_i(last_pos >= 0 ? -last_pos : 0x7FFFFFFF);
          pick = neg == 0x7FFFFFFF ? -1 : -neg;
          if (lane == 0) sm.flags[2] = 0;
        } else {
          if (first_ok == pick) sm.dd[3] = (double)fx;
          if (lane == 0) sm.flags[2] = 1;
        }
      } else if (lane == 0) {
        sm.flags[2] = 0;
      }
    } else if (lane == 0) {
      sm.flags[2] = 0;
    }
    if (lane == 0) sm.flags[3] = pick;
  }
  __syncthreads();
  return sm.flags[3];
}

// Argmax of the fused logits of a row by a full scan (whole workgroup); only
// used when a residual is empty (p~ equal to q in fp32).
template <int DT>
DEV int row_argmax_f(const KArgs& A, const RowGeo& g, Smem& sm) {
  float best = kFloorM;
  int bi = 0x7FFFFFFF;
  for (int x = wave_id() * 64 + lane_id(); x < A.V; x += kThreads) {
    float xt, xa, xb;
    mapped_tab<DT>(A, g, x, xt, xa, xb);
    const float f = fuse_rt(xt, xa, xb, A.beta, A.delta_mode);
    if (f > best) { best = f; bi = x; }
  }
  const float M = wave_max(best);
  __syncthreads();
  if (lane_id() == 0) sm.wj[wave_id()] = M;
  __syncthreads();
  float Mb = sm.wj[0];
  #pragma unroll
  for (int q = 1; q < kWaves; ++q) Mb = fmaxf(Mb, sm.wj[q]);
  const int r = block_min_i(best == Mb ? bi : 0x7FFFFFFF, sm);
  return r == 0x7FFFFFFF ? 0 : r;   // a row with no finite f: token 0, as argmax of all -inf
}

template <int DT, int DM>
DEV void pick_item(const KArgs& A, int req, Smem& sm) {
  const int lane = lane_id(), w = wave_id();
  const int K = A.K;
  const uint32_t state = load_decision(A, req, sm);
  if (state != kStatePending) {
    // final: the decide wrote the outputs; failed: mark them invalid
    if (state == kStateFailed && threadIdx.x == 0) A.acc_out[req] = -1;
    return;
  }
  bool ok = true;   // this thread's waits all ended in time
  const bool samp = sm.req[R_SAMP] != 0u;
  // requested now, used after the sub-block sums arrive
  const float uK = samp ? A.u[(size_t)req * (K + 1) + K] : 0.0f;
  // D of each row with a JSD task, the rows dealt out over the waves (the
  // k-th such row to wave k mod 4, its chunk partials over the lanes)
  {
    const uint32_t tk = lane <= K ? sm.rows[lane][D_TASK] : 0u;
    unsigned long long jm = __ballot((tk & kTaskJsd) != 0u);
    for (int k = 0; jm != 0; jm &= jm - 1, ++k) {
      if (k % kWaves != w) continue;
      const int i = __builtin_ctzll(jm);
      double part = 0.0;
      for (int c = lane; c < A.S * A.P2; c += 64)
        part += (double)wait_f32(p2_rec(A, req, i, c / A.P2) + P2_J + c % A.P2, A, ok);
      part = wave_sum_d(part);
      // the partials are in log2 units; JSD = half their sum, within [0, ln 2]
      const double D = 0.5 * kLn2 * part;
      if (lane == 0) sm.djsd[i] = D < 0.0 ? 0.0 : (D > kLn2 ? kLn2 : D);
    }
  }
  __syncthreads();
  // wave 0: final decisions, the emitting row
  float lpd = 0.0f;
  double Dl = 0.0;
  if (w == 0) {
    const bool is_draft = lane < K;
    uint32_t st = 0, task = 0, arg = 0;
    double thr = 0.0;
    float lpe = 0.0f;
    if (lane <= K) {
      const uint32_t* v = sm.rows[lane];
      st = v[D_STATUS];
      task = v[D_TASK];
      thr = u2d(v[D_THR_LO], v[D_THR_HI]);
      lpd = __uint_as_float(v[D_LPD]);
      arg = v[D_ARG];
      lpe = __uint_as_float(v[D_LPEMIT]);
    }
    if (task & kTaskJsd) Dl = sm.djsd[lane];
    if ((A.gate_mode == ASYMSPEC_GATE_LAMBDA || A.gate_mode == ASYMSPEC_GATE_KL) && lane < K)
      Dl = u2d(sm.rows[lane][D_GD_LO], sm.rows[lane][D_GD_HI]);
    const bool decided = st & kStDecided;
    const bool acc = decided ? (st & kStAccept) != 0 : (Dl > thr);
    const int jr = wave_min_i(is_draft && !acc ? lane : 0x7FFFFFFF);
    const int j = jr == 0x7FFFFFFF ? K : jr;
    const int argj = __builtin_amdgcn_readlane((int)arg, j);
    const float lpej = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, lpe), j));
    if (lane == 0) { sm.flags[0] = j; sm.flags[1] = argj; sm.dd[0] = (double)lpej; }
  }
  __syncthreads();
  const int j = sm.flags[0];
  int next = sm.flags[1];
  float lpn = (float)sm.dd[0];
  if (samp) {
    const bool bonus = j == K && !A.fuse_bonus;   // weights from t alone
    const double u = (double)uK;
    int pick = cdf_pick<DT, DM>(A, req, j, u, bonus, sm, ok);
    const RowGeo g = row_span<DT>(A, req * (K + 1) + j);
    const bool have_x = pick >= 0 && sm.flags[2] != 0;
    if (pick < 0) pick = row_argmax_f<DT>(A, g, sm);
    next = pick;
    float x;
    if (have_x) {
      x = (float)sm.dd[3];
    } else {
      float xa, xb;
      mapped_tab<DT>(A, g, next, x, xa, xb);
      if (!bonus) x = fuse_masked(x, xa, xb, A.beta, A.delta_mode);
    }
    const double c = (double)__uint_as_float(sm.rows[j][D_C]);
    const double l2 = u2d(sm.rows[j][D_L2E_LO], sm.rows[j][D_L2E_HI]);
    lpn = (float)(((double)x * c - l2) * kLn2);
  }
  // a wait that timed out leaves the decision incomplete: invalid outputs
  const bool failed = __syncthreads_or(!ok);
  if (w == 0) {
    const bool skip = lane <= K && (sm.rows[lane][D_STATUS] & kStSkip) != 0u;
    write_outputs(A, req, j, next, lpn, lpd, Dl, skip);
    if (failed && lane == 0) A.acc_out[req] = -1;
  }
}

}  // namespace asym

#endif  // ASYMSPEC_RESOLVE_H_
