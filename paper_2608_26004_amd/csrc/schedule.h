// Work-item schedule of the fused decision step.
//
// Plain C++ (no HIP types) so that the same code runs in the kernel, in the
// host launcher and in a host-only test.
//
// The step is a single ordered list of work items, one workgroup each, which
// the hardware starts in index order.  Items are grouped in steps q = 0, 1,
// 2, ...; step q holds
//   * the statistics items of request q       (G * S items: one per row of
//     the first G rows and vocabulary chunk), when q < B,
//   * the verdict item of request q - Lv      (1 item; early exit only),
//   * the statistics items of the other rows of request q - Ls
//                                             ((K+1-G) * S items; early exit
//                                             only),
//   * the decide item of request q - L1       (1 item),
//   * the pass-2 items of request q - L2      (S2 = P2 * S items: P2 parts
//                                             of each chunk),
//   * the pick item of request q - L3         (1 item),
// each present only when its request index lies in [0, B).  Without early
// exit G = K + 1 and Lv = Ls = 0.  An item only ever waits for items earlier
// in the list, so the lowest unfinished item can always proceed.  The lags
// keep those waits rare: each spans a multiple of the number of items in
// flight at once.
//
// Steps fall into at most 11 runs of equal composition (the boundaries are
// 0, Lv, Ls, L1, L2, L3 and B plus each of them); an item index is decoded by
// finding its run.

#ifndef ASYMSPEC_SCHEDULE_H_
#define ASYMSPEC_SCHEDULE_H_

#ifndef ASYM_HD
#define ASYM_HD
#endif

namespace asym {

enum ItemType {
  kItemNone = -1, kItemStats = 0, kItemDecide = 1, kItemPass2 = 2, kItemPick = 3,
  kItemVerdict = 4, kItemStats2 = 5
};
enum PartBits {
  kPartStats = 1, kPartDecide = 2, kPartPass2 = 4, kPartPick = 8, kPartVerdict = 16, kPartStats2 = 32
};

constexpr int kMaxRuns = 12;

struct Sched {
  int n_runs;
  int total;              // number of items
  int G;                  // rows in the first group (K + 1 without early exit)
  int S2;                 // pass-2 items per request (P2 parts of each of S chunks)
  int ee;                 // early exit: verdict and second-group items present
  int Lv, Ls, L1, L2, L3;
  int q0[kMaxRuns];       // first step of the run
  int i0[kMaxRuns];       // index of the run's first item
  int blk[kMaxRuns];      // items per step in the run (> 0)
  int parts[kMaxRuns];    // PartBits present in every step of the run
};

struct Item {
  int type;   // ItemType
  int req;    // request index
  int sub;    // statistics: row-in-request * S + chunk; pass 2: chunk * P2 + part; else 0
};

ASYM_HD inline bool sched_in(int q, int lag, int B) { return q - lag >= 0 && q - lag < B; }

ASYM_HD inline int sched_parts(const Sched& sc, int q, int B) {
  int p = 0;
  if (sched_in(q, 0, B)) p |= kPartStats;
  if (sc.ee && sched_in(q, sc.Lv, B)) p |= kPartVerdict;
  if (sc.ee && sched_in(q, sc.Ls, B)) p |= kPartStats2;
  if (sched_in(q, sc.L1, B)) p |= kPartDecide;
  if (sched_in(q, sc.L2, B)) p |= kPartPass2;
  if (sched_in(q, sc.L3, B)) p |= kPartPick;
  return p;
}

ASYM_HD inline int sched_block(const Sched& sc, int parts, int K, int S) {
  return ((parts & kPartStats) ? sc.G * S : 0) + ((parts & kPartVerdict) ? 1 : 0) +
         ((parts & kPartStats2) ? (K + 1 - sc.G) * S : 0) + ((parts & kPartDecide) ? 1 : 0) +
         ((parts & kPartPass2) ? sc.S2 : 0) + ((parts & kPartPick) ? 1 : 0);
}

#ifndef ASYMSPEC_LAG_PCT
#define ASYMSPEC_LAG_PCT 400
#endif
#ifndef ASYMSPEC_LAG2_PCT
#define ASYMSPEC_LAG2_PCT ASYMSPEC_LAG_PCT
#endif
#ifndef ASYMSPEC_LAG3_PCT
#define ASYMSPEC_LAG3_PCT ASYMSPEC_LAG2_PCT
#endif
#ifndef ASYMSPEC_LAGV_PCT
#define ASYMSPEC_LAGV_PCT 150
#endif
#ifndef ASYMSPEC_LAGS_PCT
#define ASYMSPEC_LAGS_PCT 100
#endif

// Lags in steps.  items_in_flight is the number of workgroups the chip holds
// at once; the items of one request finish about that many items after the
// first of them starts, and a resolve item that waits holds its workgroup, so
// the decide lag spans lag_pct percent of items_in_flight statistics items,
// and the pass-2 and pick lags add lag2_pct and lag3_pct percent to the lag
// before them.  With early exit (ee_rows in [1, K]) the first ee_rows rows of
// a request are read first, its verdict follows LAGV_PCT later and the other
// rows LAGS_PCT after that; the decide lag then counts from those.  Pass 2
// takes p2 items per chunk.  Returns false when the schedule would not fit in
// 31-bit indices.
inline bool sched_build(int B, int K, int S, int items_in_flight, Sched& sc, int ee_rows = 0, int p2 = 1,
                        int lag_pct = ASYMSPEC_LAG_PCT, int lag2_pct = ASYMSPEC_LAG2_PCT,
                        int lag3_pct = ASYMSPEC_LAG3_PCT) {
  if (B < 1 || K < 0 || S < 1 || items_in_flight < 1 || ee_rows < 0 || p2 < 1) return false;
  if ((long long)S * p2 > (1LL << 24)) return false;
  sc.S2 = S * p2;
  // steps hold at least the (K+1) * S statistics items of their request
  const long long per_step = (long long)(K + 1) * S;
  auto window = [&](int pct) {
    const long long span = (long long)items_in_flight * pct / 100;
    return (int)((span + per_step - 1) / per_step);
  };
  sc.ee = (ee_rows >= 1 && ee_rows <= K) ? 1 : 0;
  sc.G = sc.ee ? ee_rows : K + 1;
  sc.Lv = sc.ee ? window(ASYMSPEC_LAGV_PCT) + 1 : 0;
  sc.Ls = sc.ee ? sc.Lv + window(ASYMSPEC_LAGS_PCT) + 1 : 0;
  sc.L1 = sc.Ls + window(lag_pct) + 1;
  sc.L2 = sc.L1 + window(lag2_pct) + 1;
  sc.L3 = sc.L2 + window(lag3_pct) + 1;
  const int lags[6] = {0, sc.Lv, sc.Ls, sc.L1, sc.L2, sc.L3};
  int bp[12];
  for (int i = 0; i < 6; ++i) {
    bp[i] = lags[i];
    bp[6 + i] = B + lags[i];
  }
  // sort the 12 boundaries (insertion sort); equal ones give empty runs
  for (int i = 1; i < 12; ++i)
    for (int j = i; j > 0 && bp[j - 1] > bp[j]; --j) {
      const int t = bp[j]; bp[j] = bp[j - 1]; bp[j - 1] = t;
    }
  long long idx = 0;
  sc.n_runs = 0;
  for (int i = 0; i + 1 < 12; ++i) {
    const int qa = bp[i], qb = bp[i + 1];
    if (qb <= qa) continue;
    const int parts = sched_parts(sc, qa, B);
    const int blk = sched_block(sc, parts, K, S);
    if (blk == 0) continue;
    if (sc.n_runs >= kMaxRuns) return false;
    sc.q0[sc.n_runs] = qa;
    sc.i0[sc.n_runs] = (int)idx;
    sc.blk[sc.n_runs] = blk;
    sc.parts[sc.n_runs] = parts;
    ++sc.n_runs;
    idx += (long long)(qb - qa) * blk;
    if (idx >= (1LL << 31) - 1) return false;
  }
  sc.total = (int)idx;
  return true;
}

ASYM_HD inline Item sched_item(const Sched& sc, int K, int S, int idx) {
  Item it{kItemNone, 0, 0};
  if (idx < 0 || idx >= sc.total) return it;
  // the run holding idx, found with constant indices and selects only: in a
  // kernel the schedule is part of a by-value argument, which a variable
  // index would force into private memory, and loads under a condition would
  // each wait for the one before
  int i0 = sc.i0[0], blk = sc.blk[0], q0 = sc.q0[0], parts = sc.parts[0];
  #pragma unroll
  for (int k = 1; k < kMaxRuns; ++k) {
    const int ik = sc.i0[k], bk = sc.blk[k], qk = sc.q0[k], pk = sc.parts[k];
    const bool take = k < sc.n_runs && idx >= ik;
    i0 = take ? ik : i0;
    blk = take ? bk : blk;
    q0 = take ? qk : q0;
    parts = take ? pk : parts;
  }
  const int off = idx - i0;
  const int qs = off / blk;
  int o = off - qs * blk;
  const int q = q0 + qs;
  const int n1 = sc.G * S, n2 = (K + 1 - sc.G) * S;
  if (parts & kPartStats) {
    if (o < n1) { it.type = kItemStats; it.req = q; it.sub = o; return it; }
    o -= n1;
  }
  if (parts & kPartVerdict) {
    if (o < 1) { it.type = kItemVerdict; it.req = q - sc.Lv; it.sub = 0; return it; }
    o -= 1;
  }
  if (parts & kPartStats2) {
    if (o < n2) { it.type = kItemStats2; it.req = q - sc.Ls; it.sub = n1 + o; return it; }
    o -= n2;
  }
  if (parts & kPartDecide) {
    if (o < 1) { it.type = kItemDecide; it.req = q - sc.L1; it.sub = 0; return it; }
    o -= 1;
  }
  if (parts & kPartPass2) {
    if (o < sc.S2) { it.type = kItemPass2; it.req = q - sc.L2; it.sub = o; return it; }
    o -= sc.S2;
  }
  it.type = kItemPick;
  it.req = q - sc.L3;
  it.sub = 0;
  return it;
}

// Renumbering of the n consecutive items of one block so that items 8 apart
// (which the hardware sends to the same XCD) take consecutive positions:
// position = (items of the block in lower residue classes mod 8) + sub / 8.
// A bijection on [0, n).
ASYM_HD inline int xcd_grouped(int sub, int n) {
  const int r = sub & 7;
  int before = 0;
  for (int c = 0; c < r; ++c) before += (n - c + 7) >> 3;
  return before + (sub >> 3);
}

}  // namespace asym

#endif  // ASYMSPEC_SCHEDULE_H_
