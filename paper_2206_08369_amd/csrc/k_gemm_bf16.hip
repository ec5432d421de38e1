// Input-layer GEMMs with bf16 operands and fp32 accumulation on the bf16
// matrix cores (the bf16-in / fp32-accumulate precision mode).
//
//   C[p][q] = sum_k bf16(P[p][k]) * Q[q][k]
//
// P is the big fp32 operand (W1 for the forward product of Section 3 step 1,
// dZ^T for dW1), rounded to bf16 (nearest even, v_cvt_pk_bf16_f32) as it is
// loaded, so the fp32 master weights and activations are never copied.  Q is
// the small operand (the batch or its transpose), already bf16.  Both are
// k-contiguous.
//
// One v_mfma_f32_32x32x16_bf16 takes a 32x16 tile of Q (lane l: row l%32,
// eight k in half l/32) and a 16x32 tile of P^T laid out the same way, and
// accumulates the 32x32 block D[q][p]; lane l holds p = l%32 and, in
// register 4i+r, q = 8i + 4(l/32) + r, so each lane stores float4s along q.
// Within a 32-wide k stage, lane l of half h owns the 16 consecutive k
// 16h..16h+15 and feeds them to two MFMAs (8 each); A and B use the same
// permutation of k, so the sum is unchanged.
//
// A workgroup of WP x WQ waves computes an MP x MQ tile (MP = 32 TP WP,
// MQ = 32 TQ WQ), each wave TP x TQ MFMA blocks.  Per stage, every thread
// loads 16 consecutive k of one or more operand rows (fp32 P converted to
// bf16 in registers), writes them to LDS in MFMA-operand order (fragment
// (g, s) = 64 lanes x 16 bytes, g the 32-row group, s the 8-k step), and
// every wave reads its fragments with conflict-free ds_read_b128.  Two LDS
// stages: the global loads of stage k+1 are in flight during the MFMAs of
// stage k, one barrier per stage.
//
// Tile order is XCD-aware: workgroup b runs on XCD b % 8, and the nqt
// q-tiles of one p-tile are consecutive workgroups of the same XCD, so the
// p-tile (the operand streamed from HBM) is fetched once and served from
// that XCD's L2 to the other q-tiles.

#include "device_common.h"

namespace pmlpk {

namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kKs = 32;  // k per pipeline stage

__device__ __forceinline__ u32x4 pack_bf16x8(const f32x4& a, const f32x4& b) {
  bf16x8 r;
  r[0] = (__bf16)a[0];
  r[1] = (__bf16)a[1];
  r[2] = (__bf16)a[2];
  r[3] = (__bf16)a[3];
  r[4] = (__bf16)b[0];
  r[5] = (__bf16)b[1];
  r[6] = (__bf16)b[2];
  r[7] = (__bf16)b[3];
  return __builtin_bit_cast(u32x4, r);
}

template <int TP, int TQ, int WP, int WQ, int EPI>
__global__ __launch_bounds__(64 * WP * WQ) void k_gemm_bf(GemmBfArgs a, int npt, int nqt) {
  constexpr int NT = 64 * WP * WQ;
  constexpr int MP = 32 * TP * WP, MQ = 32 * TQ * WQ;
  // (row, half) pairs per thread; with fewer pairs than threads the last
  // waves of the workgroup skip the load (a wave-uniform condition)
  constexpr int LP = (2 * MP + NT - 1) / NT, LQ = (2 * MQ + NT - 1) / NT;
  static_assert((2 * MP) % NT == 0 || 2 * MP < NT, "loader shape");
  static_assert((2 * MQ) % NT == 0 || 2 * MQ < NT, "loader shape");
  static_assert((2 * MP) % 64 == 0 && (2 * MQ) % 64 == 0, "loader shape");
  constexpr int PS = MP * 4, QS = MQ * 4;  // 16-byte slots per stage
  __shared__ u32x4 lds[2 * (PS + QS)];

  const int blk = blockIdx.x;
  const int xcd = blk & 7, jb = blk >> 3;
  const int pt = (jb / nqt) * 8 + xcd;
  const int qt = jb - (jb / nqt) * nqt;
  if (pt >= npt) return;
  const int64_t p0 = (int64_t)pt * MP;
  const int q0 = qt * MQ;
  const int t = threadIdx.x, lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int wp = wave / WQ, wq = wave - (wave / WQ) * WQ;

  // Loader: pair e covers row idx/2 of the tile, k half idx%2.
  const float* prow[LP];
  int pslot[LP], ph[LP];
#pragma unroll
  for (int e = 0; e < LP; ++e) {
    const int idx = (t + e * NT) % (2 * MP), row = idx >> 1, h = idx & 1;
    int64_t p = p0 + row;
    if (p > a.NP - 1) p = a.NP - 1;
    prow[e] = a.P + p * a.ldp + 16 * h;
    ph[e] = 16 * h;
    pslot[e] = (row >> 5) * 128 + (row & 31) + 32 * h;
  }
  const unsigned short* qrow[LQ];
  int qslot[LQ];
#pragma unroll
  for (int e = 0; e < LQ; ++e) {
    const int idx = (t + e * NT) % (2 * MQ), row = idx >> 1, h = idx & 1;
    const int q = min(q0 + row, a.NQ - 1);
    qrow[e] = a.Q + (int64_t)q * a.ldq + 16 * h;
    qslot[e] = (row >> 5) * 128 + (row & 31) + 32 * h;
  }

  f32x4 pr[LP][4];
  u32x4 qr[LQ][2];
  auto load = [&](int kt, bool masked) {
    const int k0 = kt * kKs;
#pragma unroll
    for (int e = 0; e < LP; ++e)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        if (2 * MP < NT && t >= 2 * MP) continue;
        if (masked) {
          pr[e][v] = f32x4{0.f, 0.f, 0.f, 0.f};
          if (k0 + ph[e] + 4 * v < a.K) pr[e][v] = *(const f32x4*)(prow[e] + k0 + 4 * v);
        } else {
          pr[e][v] = *(const f32x4*)(prow[e] + k0 + 4 * v);
        }
      }
#pragma unroll
    for (int e = 0; e < LQ; ++e) {
      if (2 * MQ < NT && t >= 2 * MQ) continue;
      qr[e][0] = *(const u32x4*)(qrow[e] + k0);
      qr[e][1] = *(const u32x4*)(qrow[e] + k0 + 8);
    }
  };
  auto store = [&](int sb) {
    u32x4* ps = lds + sb * (PS + QS);
    u32x4* qs = ps + PS;
#pragma unroll
    for (int e = 0; e < LP; ++e) {
      if (2 * MP < NT && t >= 2 * MP) continue;
      ps[pslot[e]] = pack_bf16x8(pr[e][0], pr[e][1]);
      ps[pslot[e] + 64] = pack_bf16x8(pr[e][2], pr[e][3]);
    }
#pragma unroll
    for (int e = 0; e < LQ; ++e) {
      if (2 * MQ < NT && t >= 2 * MQ) continue;
      qs[qslot[e]] = qr[e][0];
      qs[qslot[e] + 64] = qr[e][1];
    }
  };

  f32x16 acc[TQ][TP];
#pragma unroll
  for (int i = 0; i < TQ; ++i)
#pragma unroll
    for (int j = 0; j < TP; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  auto compute = [&](int sb) {
    const u32x4* ps = lds + sb * (PS + QS) + lane;
    const u32x4* qs = ps + PS;
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      bf16x8 pf[TP], qf[TQ];
#pragma unroll
      for (int j = 0; j < TP; ++j)
        pf[j] = __builtin_bit_cast(bf16x8, ps[((wp * TP + j) * 2 + s) * 64]);
#pragma unroll
      for (int i = 0; i < TQ; ++i)
        qf[i] = __builtin_bit_cast(bf16x8, qs[((wq * TQ + i) * 2 + s) * 64]);
#pragma unroll
      for (int i = 0; i < TQ; ++i)
#pragma unroll
        for (int j = 0; j < TP; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qf[i], pf[j], acc[i][j], 0, 0, 0);
    }
  };

  const int K = a.K;
  const int nfull = K / kKs;
  const int nk = (K + kKs - 1) / kKs;
  load(0, nfull == 0);
  store(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int nx = kt + 1;
    if (nx < nfull) load(nx, false);
    else if (nx < nk) load(nx, true);
    __builtin_amdgcn_sched_barrier(0);
    compute(kt & 1);
    __builtin_amdgcn_sched_barrier(0);
    if (nx < nk) store(nx & 1);
    __syncthreads();
  }

#pragma unroll
  for (int j = 0; j < TP; ++j) {
    const int64_t p = p0 + 32 * (wp * TP + j) + (lane & 31);
    if (p >= a.NP) continue;
    float* orow = a.out + p * a.ldo;
#pragma unroll
    for (int i = 0; i < TQ; ++i)
#pragma unroll
      for (int i4 = 0; i4 < 4; ++i4) {
        const int q = q0 + 32 * (wq * TQ + i) + 8 * i4 + 4 * (lane >> 5);
        if (q >= a.NQ) continue;
        const f32x4 v = {acc[i][j][4 * i4], acc[i][j][4 * i4 + 1], acc[i][j][4 * i4 + 2],
                         acc[i][j][4 * i4 + 3]};
        if (EPI == EPI_STORE) {
          *(f32x4*)(orow + q) = v;
        } else if (EPI == EPI_SGD) {
          f32x4 w = *(f32x4*)(orow + q);
          w -= a.lr * v;
          *(f32x4*)(orow + q) = w;
        } else {
#pragma unroll
          for (int r = 0; r < 4; ++r)
            if (q + r < a.ncols) orow[q + r] = v[r];
        }
      }
  }
}

template <int TP, int TQ, int WP, int WQ>
hipError_t gemm_bf_go(const GemmBfArgs& a, int epi, hipStream_t s) {
  constexpr int MP = 32 * TP * WP, MQ = 32 * TQ * WQ;
  const int64_t npt64 = (a.NP + MP - 1) / MP;
  const int nqt = (a.NQ + MQ - 1) / MQ;
  const int64_t nblk = ((npt64 + 7) / 8) * 8 * nqt;
  if (nblk > 0x7fffffff) return hipErrorInvalidValue;
  const int npt = (int)npt64;
  const dim3 grid((unsigned)nblk), block(64 * WP * WQ);
  switch (epi) {
    case EPI_STORE: k_gemm_bf<TP, TQ, WP, WQ, EPI_STORE><<<grid, block, 0, s>>>(a, npt, nqt); break;
    case EPI_SGD: k_gemm_bf<TP, TQ, WP, WQ, EPI_SGD><<<grid, block, 0, s>>>(a, npt, nqt); break;
    default: k_gemm_bf<TP, TQ, WP, WQ, EPI_GRAD><<<grid, block, 0, s>>>(a, npt, nqt); break;
  }
  return hipGetLastError();
}

}  // namespace

bool gemm_bf16_args_ok(const GemmBfArgs& a) {
  return a.NP > 0 && a.NQ > 0 && a.K > 0 && a.K % 4 == 0 && a.NQ % 4 == 0 && a.ldp >= a.K &&
         a.ldq % 64 == 0 && a.ldq >= ((a.K + 63) / 64) * 64;
}

hipError_t launch_gemm_bf16(const GemmBfArgs& a, int epi, hipStream_t s) {
  if (a.NP <= 0 || a.NQ <= 0) return hipSuccess;
  if (!gemm_bf16_args_ok(a)) return hipErrorInvalidValue;
  if (a.NQ <= 64) return gemm_bf_go<4, 1, 2, 2>(a, epi, s);
  return gemm_bf_go<2, 2, 2, 2>(a, epi, s);
}

}  // namespace pmlpk
