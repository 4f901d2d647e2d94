// Full-vocabulary fused log-probabilities (optional output).
//
// A second kernel on the same stream, after the decision kernel: every row is
// streamed once more and each element's log-probability is written under the
// distribution its row defines,
//   rows i < K   log softmax(f_i / tau), f_i = t_i + beta delta_i (Eq. 1-2),
//   row K        log softmax(t_K / tau) (Alg. 1 bonus row), or of f_K when the
//                bonus row is fused,
// at tau = 1 for greedy requests.  The row normalisers come from the decision
// blocks the decide items published (the kernel boundary orders them), so no
// statistic is recomputed.  A token whose fused logit is not a number (a = b
// = -inf) gets -inf, as everywhere else.
//
// One workgroup per (row, chunk); thread j takes vectors j, j + 256, ... of
// the chunk, so each load and store instruction of a wave covers contiguous
// memory.  Elements of a row's boundary vectors that belong to the
// neighbouring row are left to that row's workgroup.

#ifndef ASYMSPEC_DUMP_H_
#define ASYMSPEC_DUMP_H_

#include "device.h"
#include "schedule.h"

namespace asym {

typedef float f4v __attribute__((ext_vector_type(4)));

// One output element: (x c - L2) ln 2, in double (c = log2(e) / tau).
DEV float dump_elem(float x, double c, double l2) {
  const float r = (float)(((double)x * c - l2) * kLn2);
  return r != r ? -INFINITY : r;
}

template <int DT, int DM>
__global__ __launch_bounds__(kThreads) void dump_kernel(KArgs A, float* out) {
  constexpr int VE = Elem<DT>::VE;
  constexpr int kPerThread = kChunkVec / kThreads;
  const int S = A.S, nrow = A.K + 1;
  // through a vocabulary map, the workgroups one XCD runs take consecutive
  // chunks of the same rows (each chunk gathers from the whole drafter row)
  const int b = A.vmap != nullptr ? xcd_grouped((int)blockIdx.x, (int)gridDim.x) : (int)blockIdx.x;
  const int row = b / S;
  const int m = b - row * S;
  const int req = row / nrow, i = row - req * nrow;
  const uint64_t* blk = A.dec + (size_t)req * (kDecHdr + (size_t)nrow * kDecRow) + kDecHdr + (size_t)i * kDecRow;
  const double c = (double)payf(blk[D_C]);
  const double l2 = payd(blk[D_L2E_LO], blk[D_L2E_HI]);
  const bool fused = i < A.K || A.fuse_bonus != 0;
  // b is a bitwise copy of a on a row whose views never differ
  const bool nb = (pay(blk[D_STATUS]) & kStNeq) != 0u;
  const RowGeo g = row_span<DT>(A, row);
  const __amdgpu_buffer_rsrc_t rt = row_rsrc(A, A.t, g);
  const __amdgpu_buffer_rsrc_t ra = row_rsrc(A, A.a, g);
  const __amdgpu_buffer_rsrc_t rb = row_rsrc(A, A.b, g);
  const long long v0 = (long long)m * kChunkVec;
  const long long c0 = g.vbeg + v0;
  const bool tail = has_tail(A, c0, c0 + kChunkVec);
  const int tid = (int)threadIdx.x;
  #pragma unroll 2
  for (int k = 0; k < kPerThread; ++k) {
    const long long rel = v0 + tid + (long long)k * kThreads;
    const long long vi = g.vbeg + rel;
    if (vi >= g.vend) break;
    const uint32_t off = (uint32_t)(rel * 16);
    u4 vt = buf_load_nt(rt, off), va = vt, vb = vt;
    if (A.vmap != nullptr) {
      fix_vec<DT>(A, g, A.t, vi, vt);
      map_vecs<DT>(A, g, vi, vt, va, vb, fused);
    } else if (fused) {
      va = buf_load_nt(ra, off);
      vb = nb ? buf_load_nt(rb, off) : va;
    }
    if (tail && A.vmap == nullptr) {
      fix_vec<DT>(A, g, A.t, vi, vt);
      if (fused) {
        fix_vec<DT>(A, g, A.a, vi, va);
        if (nb) fix_vec<DT>(A, g, A.b, vi, vb);
        else vb = va;
      }
    }
    float r[VE];
    #pragma unroll
    for (int e = 0; e < VE; ++e) {
      const float xt = Elem<DT>::get(vt, e);
      const float x = fused ? fuse<DM>(xt, Elem<DT>::get(va, e), Elem<DT>::get(vb, e), A.beta) : xt;
      r[e] = dump_elem(x, c, l2);
    }
    const long long f0 = vi * VE;   // flat index of the vector's first element
    if (f0 >= g.e0 && f0 + VE <= g.e0 + A.V) {
      #pragma unroll
      for (int q = 0; q < VE / 4; ++q) {
        const f4v w = {r[4 * q], r[4 * q + 1], r[4 * q + 2], r[4 * q + 3]};
        __builtin_nontemporal_store(w, reinterpret_cast<f4v*>(out + f0) + q);
      }
    } else {
      #pragma unroll
      for (int e = 0; e < VE; ++e)
        if (f0 + e >= g.e0 && f0 + e < g.e0 + A.V) out[f0 + e] = r[e];
    }
  }
}

}  // namespace asym

#endif  // ASYMSPEC_DUMP_H_
