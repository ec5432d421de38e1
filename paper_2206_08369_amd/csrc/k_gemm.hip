// Generic input-layer GEMMs on the fp32 matrix cores (any batch and F).

#include "device_common.h"

namespace pmlpk {

// ---------------------------------------------------------------------------
// Input-layer GEMMs on the fp32 matrix cores.
//
//   C[p][q] = sum_k P[p][k] * Q[q][k]
//
// P is the big operand (one row per hidden unit: W1 for the forward
// product of Section 3 step 1, dZ^T for dW1), Q the small one (the batch,
// or its transpose).  Both are k-contiguous.  One v_mfma_f32_16x16x4f32
// takes a 16x4 tile of Q (lane l: row l%16, k l/16) and a 4x16 tile of P
// and accumulates the 16x16 block D[q][p]; lane l holds p = l%16 and the
// four consecutive q = 4*(l/16) + r, so each lane stores one float4 along
// q.  Within a 16-wide k chunk every lane loads 4 consecutive k with one
// 16-byte load and feeds them to four MFMAs; the products are summed in a
// permuted k order, which is the same sum.
//
// Each wave owns TQ x TP MFMA tiles; a workgroup of four waves is arranged
// WQ (along q) x 4/WQ (along p).  Operands are read straight from global
// memory (the small operand stays in L2, the big one is streamed once).
// ---------------------------------------------------------------------------

template <int TQ, int TP>
__device__ __forceinline__ void load_chunk(f32x4 (&cq)[TQ], f32x4 (&cp)[TP],
                                           const float* const (&qrow)[TQ],
                                           const float* const (&prow)[TP], int off) {
#pragma unroll
  for (int t = 0; t < TQ; ++t) cq[t] = *(const f32x4*)(qrow[t] + off);
#pragma unroll
  for (int t = 0; t < TP; ++t) cp[t] = *(const f32x4*)(prow[t] + off);
}

template <int TQ, int TP>
__device__ __forceinline__ void mma_chunk(f32x4 (&acc)[TQ][TP], const f32x4 (&cq)[TQ],
                                          const f32x4 (&cp)[TP]) {
#pragma unroll
  for (int s = 0; s < 4; ++s)
#pragma unroll
    for (int i = 0; i < TQ; ++i)
#pragma unroll
      for (int j = 0; j < TP; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(cq[i][s], cp[j][s], acc[i][j], 0, 0, 0);
}

template <int TQ, int TP, int EPI>
__global__ __launch_bounds__(kBlock) void k_gemm_nt(GemmArgs a, int WQ) {
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  const int WP = 4 / WQ;
  const int wq = wave % WQ, wp = wave / WQ;
  const int64_t p0 = ((int64_t)blockIdx.x * WP + wp) * (16 * TP);
  const int q0 = ((int)blockIdx.y * WQ + wq) * (16 * TQ);
  if (p0 >= a.NP || q0 >= a.NQ) return;
  const int li = lane & 15, lk = lane >> 4;

  const float* qrow[TQ];
  const float* prow[TP];
#pragma unroll
  for (int t = 0; t < TQ; ++t) {
    const int q = min(q0 + 16 * t + li, a.NQ - 1);
    qrow[t] = a.Q + (int64_t)q * a.ldq;
  }
#pragma unroll
  for (int t = 0; t < TP; ++t) {
    int64_t p = p0 + 16 * t + li;
    if (p > a.NP - 1) p = a.NP - 1;
    prow[t] = a.P + p * a.ldp;
  }

  f32x4 acc[TQ][TP];
#pragma unroll
  for (int i = 0; i < TQ; ++i)
#pragma unroll
    for (int j = 0; j < TP; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  // Main loop over 16-wide k chunks, two register buffers in ping-pong: the
  // loads of chunk c+1 are issued before the 4 x TQ x TP MFMAs of chunk c,
  // and scheduling barriers keep the compiler from sinking them below.
  const int K = a.K;
  const int nch = K >> 4;
  const int K16 = nch << 4;
  if (nch > 0) {
    f32x4 qa[TQ], pa[TP], qb[TQ], pb[TP];
    load_chunk<TQ, TP>(qa, pa, qrow, prow, 4 * lk);
    int c = 0;
    // Loop body without branches: the wait counts stay exact (each MFMA
    // group waits only for its own buffer, never for the chunk in flight).
    for (; c + 2 < nch; c += 2) {
      load_chunk<TQ, TP>(qb, pb, qrow, prow, (c + 1) * 16 + 4 * lk);
      __builtin_amdgcn_sched_barrier(0);
      mma_chunk<TQ, TP>(acc, qa, pa);
      __builtin_amdgcn_sched_barrier(0);
      load_chunk<TQ, TP>(qa, pa, qrow, prow, (c + 2) * 16 + 4 * lk);
      __builtin_amdgcn_sched_barrier(0);
      mma_chunk<TQ, TP>(acc, qb, pb);
      __builtin_amdgcn_sched_barrier(0);
    }
    if (c + 1 < nch) {
      load_chunk<TQ, TP>(qb, pb, qrow, prow, (c + 1) * 16 + 4 * lk);
      __builtin_amdgcn_sched_barrier(0);
      mma_chunk<TQ, TP>(acc, qa, pa);
      mma_chunk<TQ, TP>(acc, qb, pb);
    } else {
      mma_chunk<TQ, TP>(acc, qa, pa);
    }
  }
  for (int k = K16; k < K; k += 4) {
    float aq[TQ], ap[TP];
#pragma unroll
    for (int t = 0; t < TQ; ++t) aq[t] = qrow[t][k + lk];
#pragma unroll
    for (int t = 0; t < TP; ++t) ap[t] = prow[t][k + lk];
#pragma unroll
    for (int i = 0; i < TQ; ++i)
#pragma unroll
      for (int j = 0; j < TP; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(aq[i], ap[j], acc[i][j], 0, 0, 0);
  }

#pragma unroll
  for (int j = 0; j < TP; ++j) {
    const int64_t p = p0 + 16 * j + li;
    if (p >= a.NP) continue;
    float* orow = a.out + p * a.ldo;
    const float lr = (EPI == EPI_SGD && a.lrm) ? a.lrm[a.mid[p]] : a.lr;
    const int mrow = (EPI != EPI_STORE && a.fmask) ? a.mid[p] : 0;
#pragma unroll
    for (int i = 0; i < TQ; ++i) {
      const int q = q0 + 16 * i + 4 * lk;
      if (q >= a.NQ) continue;
      if (EPI == EPI_STORE) {
        *(f32x4*)(orow + q) = acc[i][j];
        continue;
      }
      // masked features: zero gradient, so their weights stay 0
      const f32x4 g = fmask4(a.fmask, a.fmw, mrow, q, acc[i][j]);
      if (EPI == EPI_SGD) {
        f32x4 w = *(f32x4*)(orow + q);
        w -= lr * g;
        *(f32x4*)(orow + q) = w;
      } else {
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (q + r < a.ncols) orow[q + r] = g[r];
          else if (q + r == a.bcol && a.db1) a.db1[p] = g[r];
      }
    }
  }
}

template <int TQ, int TP>
static void gemm_dispatch(const GemmArgs& a, int epi, int WQ, hipStream_t s) {
  const int WP = 4 / WQ;
  dim3 grid((unsigned)ceil_div_i(a.NP, (int64_t)WP * 16 * TP),
            (unsigned)ceil_div_i(a.NQ, (int64_t)WQ * 16 * TQ));
  switch (epi) {
    case EPI_STORE: k_gemm_nt<TQ, TP, EPI_STORE><<<grid, kBlock, 0, s>>>(a, WQ); break;
    case EPI_SGD: k_gemm_nt<TQ, TP, EPI_SGD><<<grid, kBlock, 0, s>>>(a, WQ); break;
    default: k_gemm_nt<TQ, TP, EPI_GRAD><<<grid, kBlock, 0, s>>>(a, WQ); break;
  }
}

hipError_t launch_gemm(const GemmArgs& a, int epi, hipStream_t s) {
  note_variant("k_gemm_nt", kArithFp32);
  if (a.NP <= 0 || a.NQ <= 0) return hipSuccess;
  if (a.NQ <= 16) gemm_dispatch<1, 8>(a, epi, 1, s);
  else if (a.NQ <= 32) gemm_dispatch<2, 8>(a, epi, 1, s);
  else if (a.NQ <= 64) gemm_dispatch<4, 4>(a, epi, 1, s);
  else if (a.NQ <= 112) gemm_dispatch<7, 2>(a, epi, 1, s);
  else if (a.NQ <= 128) gemm_dispatch<4, 4>(a, epi, 2, s);
  else gemm_dispatch<4, 4>(a, epi, 4, s);
  return hipGetLastError();
}

}  // namespace pmlpk
