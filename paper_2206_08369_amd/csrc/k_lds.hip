// Persistent LDS-resident GEMMs: forward and fused backward.

#include "device_common.h"

namespace pmlpk {

// ---------------------------------------------------------------------------
// Persistent input-layer GEMMs with the batch operand resident in LDS.
//
// The small operand of both input-layer products is the batch itself (Xp
// for Z = X W1^T, Xt for dW1 = dZ^T X): a few hundred KB at most for the
// shapes these kernels accept, so each workgroup of 8 waves copies it into
// LDS once and then streams its share of the hidden units.  Each wave takes
// tiles t, t + stride, ... (stride = all waves of the grid), so every wave
// reaches the end of the tile range and exits.  MFMA operands of the batch
// come from LDS with ds_read_b128 (row stride chosen so 16 consecutive rows
// hit distinct banks); operands of the big matrix come from global memory.
// ---------------------------------------------------------------------------

static constexpr int kLdsBlock = 512;
static constexpr int kLdsWaves = kLdsBlock / 64;
static constexpr int kKCMax = 8;  // forward: up to 8 full 16-wide chunks of F

// Forward: Zt[p][q] = sum_k W1[p][k] Xp[q][k] for one tile of 16 hidden
// units p and all Bp = 16*TQ samples q.  The whole W1 strip of the next
// tile (K/4 floats per lane) is loaded while the current tile computes, so
// the memory latency is hidden behind a full tile of MFMAs.  Chunks past
// the last one repeat its (in-row) address and are skipped at compute
// time; the 4/8/12-wide remainder of K uses one MFMA step per 4 values
// with lane l/16 holding k = K16 + 4s + l/16.
__device__ __forceinline__ void fwd_lds_load(f32x4 (&pc)[kKCMax], float (&pt)[3],
                                             const float* __restrict__ W1, int64_t t, int64_t N,
                                             int K, int nch, int li, int lk) {
  int64_t p = t * 16 + li;
  if (p > N - 1) p = N - 1;
  const float* row = W1 + p * K;
  const int clast = nch > 0 ? nch - 1 : 0;
#pragma unroll
  for (int c = 0; c < kKCMax; ++c) {
    int off = 16 * (c < clast ? c : clast) + 4 * lk;
    if (off > K - 4) off = K - 4;
    pc[c] = *(const f32x4*)(row + off);
  }
#pragma unroll
  for (int s = 0; s < 3; ++s) {
    int off = 16 * nch + 4 * s + lk;
    if (off > K - 1) off = K - 1;
    pt[s] = row[off];
  }
}

template <int TQ>
__global__ __launch_bounds__(kLdsBlock) void k_fwd_lds(FwdLdsArgs a) {
  extern __shared__ float lds[];
  const int K = a.K, SQ = a.SQ, K4 = K >> 2;
  for (int idx = threadIdx.x; idx < 16 * TQ * K4; idx += kLdsBlock) {
    const int row = idx / K4;
    const int c4 = idx - row * K4;
    *(f32x4*)(lds + row * SQ + 4 * c4) = *(const f32x4*)(a.Xp + (int64_t)row * K + 4 * c4);
  }
  __syncthreads();
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  const int li = lane & 15, lk = lane >> 4;
  const int nch = K >> 4, tr = (K & 15) >> 2;
  const int64_t T = (a.N + 15) >> 4;
  const int64_t tstride = (int64_t)gridDim.x * kLdsWaves;
  int64_t t = (int64_t)blockIdx.x * kLdsWaves + wave;
  if (t >= T) return;
  const float* qbase = lds + li * SQ + 4 * lk;        // + 16*i*SQ + 16*c
  const float* qtail = lds + li * SQ + 16 * nch + lk;  // + 16*i*SQ + 4*s
  f32x4 pc[kKCMax];
  float pt[3];
  fwd_lds_load(pc, pt, a.W1, t, a.N, K, nch, li, lk);
  for (; t < T; t += tstride) {
    f32x4 pn[kKCMax];
    float ptn[3];
    const int64_t tn = t + tstride < T ? t + tstride : t;
    fwd_lds_load(pn, ptn, a.W1, tn, a.N, K, nch, li, lk);
    __builtin_amdgcn_sched_barrier(0);
    f32x4 acc[TQ];
#pragma unroll
    for (int i = 0; i < TQ; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int c = 0; c < kKCMax; ++c) {
      if (c < nch) {
        // one LDS operand at a time; the four steps accumulate back to back
#pragma unroll
        for (int i = 0; i < TQ; ++i) {
          const f32x4 q = *(const f32x4*)(qbase + 16 * i * SQ + 16 * c);
#pragma unroll
          for (int s = 0; s < 4; ++s)
            acc[i] = __builtin_amdgcn_mfma_f32_16x16x4f32(q[s], pc[c][s], acc[i], 0, 0, 0);
        }
      }
    }
#pragma unroll
    for (int s = 0; s < 3; ++s) {
      if (s < tr) {
#pragma unroll
        for (int i = 0; i < TQ; ++i)
          acc[i] = __builtin_amdgcn_mfma_f32_16x16x4f32(qtail[16 * i * SQ + 4 * s], pt[s], acc[i],
                                                        0, 0, 0);
      }
    }
    // Zt rows are padded to a multiple of 64, so every store is in bounds.
    float* zrow = a.Zt + (t * 16 + li) * (int64_t)(16 * TQ) + 4 * lk;
#pragma unroll
    for (int i = 0; i < TQ; ++i) *(f32x4*)(zrow + 16 * i) = acc[i];
#pragma unroll
    for (int c = 0; c < kKCMax; ++c) pc[c] = pn[c];
#pragma unroll
    for (int s = 0; s < 3; ++s) pt[s] = ptn[s];
  }
}

// ---------------------------------------------------------------------------
// Fused backward: M3 backward + activation derivative + dW1 GEMM + both SGD
// updates in one pass over Zt (dZ is never stored).
//
// For every hidden unit n (row p of the GEMM), model m = mid[n]:
//   dZ[n][b] = (sum_o G[m][b][o] W2[o][n]) * act'(Z[n][b])   (old W2)
//   dW1[n][f] = sum_b dZ[n][b] X[b][f]                      (MFMA, K = batch)
//   dW2[o][n] = sum_b G[m][b][o] act(Z[n][b])
//   W1 -= lr dW1, W2 -= lr dW2  (or both gradients stored)
// Lane (li, lk) owns rows p0 + 16j + li and, in each 16-wide batch chunk,
// the four samples b = c*16 + 4lk .. +3: every dZ element is formed once,
// in registers, by the lane that feeds it to the MFMA (the backward of the
// scatter-add is this gather of G by model id, Section 3).  dW2 partial
// sums stay in registers and are combined over the four lk lanes of a row
// at the end of the tile; one wave covers all F columns, so each row's dW2
// comes from exactly one wave.  Z and G chunks are double-buffered in
// registers (loop body without branches, so wait counts stay exact).
// ---------------------------------------------------------------------------

template <int TP, int OM>
__device__ __forceinline__ void bwdl_load(f32x4 (&cz)[TP], f32x4 (&cg)[TP][OM],
                                          const float* const (&zrow)[TP],
                                          const float* const (&grow)[TP], int kofs) {
#pragma unroll
  for (int j = 0; j < TP; ++j) {
    cz[j] = *(const f32x4*)(zrow[j] + kofs);
    // G[m][b .. b+3][0 .. OM-1] is 4*OM consecutive floats (OM == O)
#pragma unroll
    for (int v = 0; v < OM; ++v) cg[j][v] = *(const f32x4*)(grow[j] + kofs * OM + 4 * v);
  }
}

template <int TQ, int TP, int OM>
__device__ __forceinline__ void bwdl_chunk(f32x4 (&acc)[TQ][TP], float (&dw)[TP][OM],
                                           const float* qptr, int SQ, const f32x4 (&cz)[TP],
                                           const f32x4 (&cg)[TP][OM],
                                           const float (&w2)[TP][OM], const int (&arow)[TP],
                                           int auni) {
  f32x4 q[TQ];
#pragma unroll
  for (int i = 0; i < TQ; ++i) q[i] = *(const f32x4*)(qptr + 16 * i * SQ);
  float dz[TP][4];
#pragma unroll
  for (int j = 0; j < TP; ++j) {
    const float* g = (const float*)&cg[j][0];  // g[s*OM + o] = G[m][b+s][o]
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      float hp;
      // auni >= 0: every row of the tile has this activation (wave-uniform
      // branch); otherwise each lane dispatches on its own row's id.
      const float h = auni >= 0 ? act_fwd_bwd(auni, cz[j][s], &hp)
                                : act_fwd_bwd(arow[j], cz[j][s], &hp);
      float dh = 0.f;
#pragma unroll
      for (int o = 0; o < OM; ++o) {
        dh = fmaf(g[s * OM + o], w2[j][o], dh);
        dw[j][o] = fmaf(g[s * OM + o], h, dw[j][o]);
      }
      dz[j][s] = dh * hp;
    }
  }
#pragma unroll
  for (int s = 0; s < 4; ++s)
#pragma unroll
    for (int i = 0; i < TQ; ++i)
#pragma unroll
      for (int j = 0; j < TP; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(q[i][s], dz[j][s], acc[i][j], 0, 0, 0);
}

template <int TQ, int TP, int OM, bool GRAD>
__global__ __launch_bounds__(kLdsBlock) void k_bwd_lds(BwdArgs a) {
  extern __shared__ float lds[];
  const int Bp = a.Bp, SQ = a.SQ, B4 = Bp >> 2;
  for (int idx = threadIdx.x; idx < 16 * TQ * B4; idx += kLdsBlock) {
    const int row = idx / B4;
    const int c4 = idx - row * B4;
    const f32x4 v = row < a.F4 ? *(const f32x4*)(a.Xt + (int64_t)row * Bp + 4 * c4)
                               : f32x4{0.f, 0.f, 0.f, 0.f};
    *(f32x4*)(lds + row * SQ + 4 * c4) = v;
  }
  __syncthreads();
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  const int li = lane & 15, lk = lane >> 4;
  const int nch = Bp >> 4;
  const int64_t T = (a.N + 16 * TP - 1) / (16 * TP);
  const int64_t tstride = (int64_t)gridDim.x * kLdsWaves;
  const float* qbase = lds + li * SQ + 4 * lk;  // + 16*i*SQ + 16*c
  for (int64_t t = (int64_t)blockIdx.x * kLdsWaves + wave; t < T; t += tstride) {
    const int64_t p0 = t * 16 * TP;
    const float* zrow[TP];
    const float* grow[TP];
    float w2[TP][OM];
    int arow[TP];
#pragma unroll
    for (int j = 0; j < TP; ++j) {
      int64_t p = p0 + 16 * j + li;
      if (p > a.N - 1) p = a.N - 1;
      const int m = a.mid[p];
      arow[j] = a.act[m];
      zrow[j] = a.Zt + p * Bp;
      grow[j] = a.G + (int64_t)m * Bp * OM;
#pragma unroll
      for (int o = 0; o < OM; ++o) w2[j][o] = a.W2[(int64_t)o * a.ldw + p];
    }
    // one activation for the whole tile (the common case: segments are wide)
    const int a0 = __builtin_amdgcn_readfirstlane(arow[0]);
    bool same = true;
#pragma unroll
    for (int j = 0; j < TP; ++j) same = same && arow[j] == a0;
    const int auni = __all(same) ? a0 : -1;
    f32x4 acc[TQ][TP];
    float dw[TP][OM];
#pragma unroll
    for (int i = 0; i < TQ; ++i)
#pragma unroll
      for (int j = 0; j < TP; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int j = 0; j < TP; ++j)
#pragma unroll
      for (int o = 0; o < OM; ++o) dw[j][o] = 0.f;
    {
      f32x4 za[TP], ga[TP][OM], zb[TP], gb[TP][OM];
      bwdl_load<TP, OM>(za, ga, zrow, grow, 4 * lk);
      int c = 0;
      for (; c + 2 < nch; c += 2) {
        bwdl_load<TP, OM>(zb, gb, zrow, grow, (c + 1) * 16 + 4 * lk);
        __builtin_amdgcn_sched_barrier(0);
        bwdl_chunk<TQ, TP, OM>(acc, dw, qbase + 16 * c, SQ, za, ga, w2, arow, auni);
        __builtin_amdgcn_sched_barrier(0);
        bwdl_load<TP, OM>(za, ga, zrow, grow, (c + 2) * 16 + 4 * lk);
        __builtin_amdgcn_sched_barrier(0);
        bwdl_chunk<TQ, TP, OM>(acc, dw, qbase + 16 * (c + 1), SQ, zb, gb, w2, arow, auni);
        __builtin_amdgcn_sched_barrier(0);
      }
      if (c + 1 < nch) {
        bwdl_load<TP, OM>(zb, gb, zrow, grow, (c + 1) * 16 + 4 * lk);
        __builtin_amdgcn_sched_barrier(0);
        bwdl_chunk<TQ, TP, OM>(acc, dw, qbase + 16 * c, SQ, za, ga, w2, arow, auni);
        bwdl_chunk<TQ, TP, OM>(acc, dw, qbase + 16 * (c + 1), SQ, zb, gb, w2, arow, auni);
      } else {
        bwdl_chunk<TQ, TP, OM>(acc, dw, qbase + 16 * c, SQ, za, ga, w2, arow, auni);
      }
    }
    // dW2: combine the four lk lanes of each row; lanes lk == 0 write.
#pragma unroll
    for (int j = 0; j < TP; ++j)
#pragma unroll
      for (int o = 0; o < OM; ++o) {
        float v = dw[j][o];
        v += __shfl_xor(v, 16);
        v += __shfl_xor(v, 32);
        dw[j][o] = v;
      }
#pragma unroll
    for (int j = 0; j < TP; ++j) {
      const int64_t p = p0 + 16 * j + li;  // < Npad: padded rows absorb the tail
      if (GRAD) {
        if (p >= a.N) continue;
        if (lk == 0)
#pragma unroll
          for (int o = 0; o < OM; ++o) a.dW2[(int64_t)o * a.N + p] = dw[j][o];
        float* orow = a.dW1 + p * a.F;
#pragma unroll
        for (int i = 0; i < TQ; ++i) {
          const int q = 16 * i + 4 * lk;
#pragma unroll
          for (int r = 0; r < 4; ++r)
            if (q + r < a.F) orow[q + r] = acc[i][j][r];
        }
      } else {
        if (lk == 0)
#pragma unroll
          for (int o = 0; o < OM; ++o)
            a.W2[(int64_t)o * a.ldw + p] = w2[j][o] - a.lr * dw[j][o];
        float* orow = a.W1 + p * a.F4;
#pragma unroll
        for (int i = 0; i < TQ; ++i) {
          const int q = 16 * i + 4 * lk;
          if (q < a.F4) {
            f32x4 w = *(f32x4*)(orow + q);
            w -= a.lr * acc[i][j];
            *(f32x4*)(orow + q) = w;
          }
        }
      }
    }
  }
}

// LDS row stride (floats) for rows of K floats: an odd number of float4
// per row keeps ds_read_b128 of 16 consecutive rows free of bank conflicts.
static int lds_stride(int K) { return ((K >> 2) & 1) ? K : K + 4; }

struct DevInfo {
  int cus = 0;
  int lds_max = 0;
};

static DevInfo dev_info() {
  static DevInfo info[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return DevInfo{};
  DevInfo& d = info[dev];
  if (d.cus == 0) {
    (void)hipDeviceGetAttribute(&d.cus, hipDeviceAttributeMultiprocessorCount, dev);
    (void)hipDeviceGetAttribute(&d.lds_max, hipDeviceAttributeMaxSharedMemoryPerBlock, dev);
  }
  return d;
}

template <class Arg>
static hipError_t launch_persistent(void (*kern)(Arg), size_t lds_bytes, int64_t waves_needed,
                                    hipStream_t s, const Arg& arg) {
  const DevInfo d = dev_info();
  if (d.cus <= 0) return hipErrorNoDevice;
  if (lds_bytes > 65536) {
    hipError_t e = hipFuncSetAttribute((const void*)kern,
                                       hipFuncAttributeMaxDynamicSharedMemorySize,
                                       (int)lds_bytes);
    if (e != hipSuccess) return e;
  }
  int per_cu = 0;
  hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, (const void*)kern,
                                                              kLdsBlock, lds_bytes);
  if (e != hipSuccess) return e;
  if (per_cu < 1) return hipErrorInvalidConfiguration;
  int64_t blocks = (int64_t)d.cus * per_cu;
  const int64_t need = (waves_needed + kLdsWaves - 1) / kLdsWaves;
  if (blocks > need) blocks = need;
  if (blocks < 1) blocks = 1;
  kern<<<(unsigned)blocks, kLdsBlock, lds_bytes, s>>>(arg);
  return hipGetLastError();
}

static size_t fwd_lds_bytes(int32_t Bp, int32_t F4) { return (size_t)Bp * lds_stride(F4) * 4; }

bool fwd_lds_supported(int32_t Bp, int32_t F4) {
  const DevInfo d = dev_info();
  const bool tq_ok = Bp == 16 || Bp == 32 || Bp == 64 || Bp == 128 || Bp == 256;
  return tq_ok && F4 <= 16 * kKCMax + 12 && fwd_lds_bytes(Bp, F4) <= (size_t)d.lds_max;
}

hipError_t launch_fwd_lds(const FwdLdsArgs& a0, hipStream_t s) {
  if (a0.N <= 0) return hipSuccess;
  if (!fwd_lds_supported(a0.Bp, a0.K)) return hipErrorInvalidValue;
  FwdLdsArgs a = a0;
  a.SQ = lds_stride(a.K);
  const size_t lds = fwd_lds_bytes(a.Bp, a.K);
  const int64_t T = (a.N + 15) / 16;
  switch (a.Bp) {
    case 16: return launch_persistent(k_fwd_lds<1>, lds, T, s, a);
    case 32: return launch_persistent(k_fwd_lds<2>, lds, T, s, a);
    case 64: return launch_persistent(k_fwd_lds<4>, lds, T, s, a);
    case 128: return launch_persistent(k_fwd_lds<8>, lds, T, s, a);
    default: return launch_persistent(k_fwd_lds<16>, lds, T, s, a);
  }
}

static int bwd_tq(int32_t F4) {
  return F4 <= 16 ? 1 : F4 <= 32 ? 2 : F4 <= 64 ? 4 : F4 <= 112 ? 7 : 8;
}

static size_t bwd_lds_bytes(int32_t Bp, int32_t F4) {
  return (size_t)16 * bwd_tq(F4) * lds_stride(Bp) * 4;
}

bool bwd_lds_supported(int32_t Bp, int32_t F4, int32_t O) {
  const DevInfo d = dev_info();
  return F4 <= 128 && (O == 2 || O == 4 || O == 10) &&
         bwd_lds_bytes(Bp, F4) <= (size_t)d.lds_max;
}

template <int TQ, int TP, int OM>
static hipError_t bwd_lds_go(const BwdArgs& a, size_t lds, hipStream_t s) {
  const int64_t T = (a.N + 16 * TP - 1) / (16 * TP);
  if (a.dW1) return launch_persistent(k_bwd_lds<TQ, TP, OM, true>, lds, T, s, a);
  return launch_persistent(k_bwd_lds<TQ, TP, OM, false>, lds, T, s, a);
}

// Row tiles per wave (TP): two when the per-row G buffers are small (O = 2),
// one otherwise, which keeps the double-buffered operands in registers.
template <int OM>
static hipError_t bwd_lds_by_f(const BwdArgs& a, size_t lds, hipStream_t s) {
  constexpr int tp = OM >= 4 ? 1 : 2;
  switch (bwd_tq(a.F4)) {
    case 1: return bwd_lds_go<1, tp, OM>(a, lds, s);
    case 2: return bwd_lds_go<2, tp, OM>(a, lds, s);
    case 4: return bwd_lds_go<4, tp, OM>(a, lds, s);
    case 7: return bwd_lds_go<7, tp, OM>(a, lds, s);
    default: return bwd_lds_go<8, 1, OM>(a, lds, s);
  }
}

hipError_t launch_bwd_lds(const BwdArgs& a0, hipStream_t s) {
  if (a0.N <= 0) return hipSuccess;
  if (!bwd_lds_supported(a0.Bp, a0.F4, a0.O)) return hipErrorInvalidValue;
  BwdArgs a = a0;
  a.SQ = lds_stride(a.Bp);
  const size_t lds = bwd_lds_bytes(a.Bp, a.F4);
  if (a.O == 2) return bwd_lds_by_f<2>(a, lds, s);
  if (a.O == 4) return bwd_lds_by_f<4>(a, lds, s);
  return bwd_lds_by_f<10>(a, lds, s);
}

}  // namespace pmlpk
