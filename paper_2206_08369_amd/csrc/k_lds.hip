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
// reaches the end of the tile range and exits.  The batch is stored in LDS
// in MFMA-operand order: for each (16-row tile i, 16-wide k chunk c) one
// block of 64 x 16 bytes whose slot l holds the four k values lane l feeds
// to the MFMA, so every ds_read_b128 reads one contiguous 1 KB block (no
// bank conflicts whatever the lane grouping).  Operands of the big matrix
// come from global memory.
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
  const int K = a.K;
  const int nch = K >> 4, tr = (K & 15) >> 2;
  // full chunks: float4 slot ((i*nch + c)*64 + l) = Xp[16i + l%16][16c + 4(l/16) .. +3]
  for (int slot = threadIdx.x; slot < TQ * nch * 64; slot += kLdsBlock) {
    const int l = slot & 63, rest = slot >> 6;
    const int i = rest / nch, c = rest - (rest / nch) * nch;
    *(f32x4*)(lds + 4 * slot) =
        *(const f32x4*)(a.Xp + (int64_t)(16 * i + (l & 15)) * K + 16 * c + 4 * (l >> 4));
  }
  // remainder: float slot T0 + (i*tr + s)*64 + l = Xp[16i + l%16][16nch + 4s + l/16]
  const int T0 = TQ * nch * 256;
  for (int slot = threadIdx.x; slot < TQ * tr * 64; slot += kLdsBlock) {
    const int l = slot & 63, rest = slot >> 6;
    const int i = rest / tr, s = rest - (rest / tr) * tr;
    lds[T0 + slot] = a.Xp[(int64_t)(16 * i + (l & 15)) * K + 16 * nch + 4 * s + (l >> 4)];
  }
  __syncthreads();
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  const int li = lane & 15, lk = lane >> 4;
  const int64_t T = (a.N + 15) >> 4;
  const int64_t tstride = (int64_t)gridDim.x * kLdsWaves;
  int64_t t = (int64_t)blockIdx.x * kLdsWaves + wave;
  if (t >= T) return;
  const f32x4* qbase = (const f32x4*)lds + lane;  // + (i*nch + c)*64
  const float* qtail = lds + T0 + lane;            // + (i*tr + s)*64
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
          const f32x4 q = qbase[(i * nch + c) * 64];
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
          acc[i] = __builtin_amdgcn_mfma_f32_16x16x4f32(qtail[(i * tr + s) * 64], pt[s], acc[i],
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

// Forward for narrow inputs and batches, where a tile is only a few MFMAs
// and the kernel is bound by the W1 stream: the W1 strips of the wave's
// next R-1 tiles are in flight while the current tile computes (a ring of
// R strip buffers).  KC chunk registers cover the 16-wide chunks of K and
// TRM scalar registers the 4/8/12-wide remainder; every tile issues the
// same loads, so the wait counts stay exact.
template <int KC, int TRM>
struct FwdStrip {
  f32x4 c[KC];
  float t[TRM > 0 ? TRM : 1];
};

template <int KC, int TRM>
__device__ __forceinline__ void fwd_ring_load(FwdStrip<KC, TRM>& st, const float* __restrict__ W1,
                                             int64_t t, int64_t N, int K, int nch, int li,
                                             int lk) {
  int64_t p = t * 16 + li;
  if (p > N - 1) p = N - 1;
  const float* row = W1 + p * K;
  const int clast = nch > 0 ? nch - 1 : 0;
#pragma unroll
  for (int c = 0; c < KC; ++c) {
    int off = 16 * (c < clast ? c : clast) + 4 * lk;
    if (off > K - 4) off = K - 4;
    st.c[c] = *(const f32x4*)(row + off);
  }
#pragma unroll
  for (int s = 0; s < TRM; ++s) {
    int off = 16 * nch + 4 * s + lk;
    if (off > K - 1) off = K - 1;
    st.t[s] = row[off];
  }
}

template <int TQ, int KC, int TRM>
__device__ __forceinline__ void fwd_ring_tile(float* __restrict__ Zt, const FwdStrip<KC, TRM>& st,
                                             const f32x4* qbase, const float* qtail, int64_t t,
                                             int nch, int tr, int li, int lk) {
  f32x4 acc[TQ];
#pragma unroll
  for (int i = 0; i < TQ; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int c = 0; c < KC; ++c) {
    if (c < nch) {
      // one LDS operand at a time; the four steps accumulate back to back
#pragma unroll
      for (int i = 0; i < TQ; ++i) {
        const f32x4 q = qbase[(i * nch + c) * 64];
#pragma unroll
        for (int s = 0; s < 4; ++s)
          acc[i] = __builtin_amdgcn_mfma_f32_16x16x4f32(q[s], st.c[c][s], acc[i], 0, 0, 0);
      }
    }
  }
#pragma unroll
  for (int s = 0; s < TRM; ++s) {
    if (s < tr) {
#pragma unroll
      for (int i = 0; i < TQ; ++i)
        acc[i] = __builtin_amdgcn_mfma_f32_16x16x4f32(qtail[(i * tr + s) * 64], st.t[s], acc[i],
                                                      0, 0, 0);
    }
  }
  // Zt rows are padded to a multiple of 64, so every store is in bounds.
  float* zrow = Zt + (t * 16 + li) * (int64_t)(16 * TQ) + 4 * lk;
#pragma unroll
  for (int i = 0; i < TQ; ++i) *(f32x4*)(zrow + 16 * i) = acc[i];
}

template <int TQ, int KC, int TRM, int R>
__global__ __launch_bounds__(kLdsBlock) void k_fwd_lds_ring(FwdLdsArgs a) {
  extern __shared__ float lds[];
  const int K = a.K;
  const int nch = K >> 4, tr = (K & 15) >> 2;
  // full chunks: float4 slot ((i*nch + c)*64 + l) = Xp[16i + l%16][16c + 4(l/16) .. +3]
  for (int slot = threadIdx.x; slot < TQ * nch * 64; slot += kLdsBlock) {
    const int l = slot & 63, rest = slot >> 6;
    const int i = rest / nch, c = rest - (rest / nch) * nch;
    *(f32x4*)(lds + 4 * slot) =
        *(const f32x4*)(a.Xp + (int64_t)(16 * i + (l & 15)) * K + 16 * c + 4 * (l >> 4));
  }
  // remainder: float slot T0 + (i*tr + s)*64 + l = Xp[16i + l%16][16nch + 4s + l/16]
  const int T0 = TQ * nch * 256;
  for (int slot = threadIdx.x; slot < TQ * tr * 64; slot += kLdsBlock) {
    const int l = slot & 63, rest = slot >> 6;
    const int i = rest / tr, s = rest - (rest / tr) * tr;
    lds[T0 + slot] = a.Xp[(int64_t)(16 * i + (l & 15)) * K + 16 * nch + 4 * s + (l >> 4)];
  }
  __syncthreads();
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  const int li = lane & 15, lk = lane >> 4;
  const int64_t T = (a.N + 15) >> 4;
  const int64_t tstride = (int64_t)gridDim.x * kLdsWaves;
  const int64_t t0 = (int64_t)blockIdx.x * kLdsWaves + wave;
  if (t0 >= T) return;
  const f32x4* qbase = (const f32x4*)lds + lane;  // + (i*nch + c)*64
  const float* qtail = lds + T0 + lane;            // + (i*tr + s)*64
  // the wave's tiles are t0 + k*tstride; tiles past the end are clamped to
  // the last one (loaded, never computed)
  FwdStrip<KC, TRM> ring[R];
#pragma unroll
  for (int r = 0; r < R - 1; ++r) {
    int64_t t = t0 + r * tstride;
    if (t > T - 1) t = T - 1;
    fwd_ring_load(ring[r], a.W1, t, a.N, K, nch, li, lk);
  }
  for (int64_t k0 = 0;; k0 += R) {
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const int64_t t = t0 + (k0 + r) * tstride;
      if (t >= T) return;
      int64_t tn = t + (R - 1) * tstride;
      if (tn > T - 1) tn = T - 1;
      fwd_ring_load(ring[(r + R - 1) % R], a.W1, tn, a.N, K, nch, li, lk);
      __builtin_amdgcn_sched_barrier(0);
      fwd_ring_tile<TQ, KC, TRM>(a.Zt, ring[r], qbase, qtail, t, nch, tr, li, lk);
    }
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
// Each wave takes tiles of 16 rows; lane (li, lk) owns row t*16 + li and,
// in each 16-wide batch chunk, the four samples b = c*16 + 4lk .. +3: every
// dZ element is formed once, in registers, by the lane that feeds it to the
// MFMA (the backward of the scatter-add is this gather of G by model id,
// Section 3).  dW2 partial sums stay in registers and are combined over the
// four lk lanes of a row at the end of the tile; one wave covers all F
// columns, so each row's dW2 comes from exactly one wave.  The tile's W1
// strip is loaded before its chunks, so the update at the end of the tile
// does not wait on memory.
// ---------------------------------------------------------------------------

template <int OM>
__device__ __forceinline__ void bwdl_load(f32x4& cz, f32x4 (&cg)[OM], const float* zrow,
                                          const float* grow, int kofs) {
  cz = *(const f32x4*)(zrow + kofs);
  // G[m][b .. b+3][0 .. OM-1] is 4*OM consecutive floats (OM == O)
#pragma unroll
  for (int v = 0; v < OM; ++v) cg[v] = *(const f32x4*)(grow + kofs * OM + 4 * v);
}

// One batch chunk of one tile row: dZ = (sum_o G W2) act'(Z) for the lane's
// four samples, the dW2 partial sums, then the TQ x 4 MFMAs with the batch
// operand from LDS.  A < 0: each lane dispatches on its own row's id.
// TAIL: four more columns (16 TQ .. 16 TQ + 3) by plain FMAs instead of a
// 16-column MFMA block that would be three quarters padding; tptr points
// at the lane's four LDS slots of those columns (rows 16 TQ + q, q < 4).
template <int TQ, int OM, int A, bool TAIL>
__device__ __forceinline__ void bwdl_chunk(f32x4 (&acc)[TQ], float (&dw)[OM], float (&tacc)[4],
                                           const f32x4* qptr, int qstride, const f32x4* tptr,
                                           const f32x4& cz, const f32x4 (&cg)[OM],
                                           const float (&w2)[OM], int arow) {
  const float* g = (const float*)&cg[0];  // g[s*OM + o] = G[m][b+s][o]
  float dz[4];
#pragma unroll
  for (int s = 0; s < 4; ++s) {
    float hp;
    const float h = act_fwd_bwd(A >= 0 ? A : arow, cz[s], &hp);
    float dh = 0.f;
#pragma unroll
    for (int o = 0; o < OM; ++o) {
      dh = fmaf(g[s * OM + o], w2[o], dh);
      dw[o] = fmaf(g[s * OM + o], h, dw[o]);
    }
    dz[s] = dh * hp;
  }
  // one LDS operand at a time; the four steps accumulate back to back
#pragma unroll
  for (int i = 0; i < TQ; ++i) {
    const f32x4 q = qptr[i * qstride];
#pragma unroll
    for (int s = 0; s < 4; ++s)
      acc[i] = __builtin_amdgcn_mfma_f32_16x16x4f32(q[s], dz[s], acc[i], 0, 0, 0);
  }
  if (TAIL) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const f32x4 x = tptr[q];  // X[b .. b+3][16 TQ + q]
#pragma unroll
      for (int s = 0; s < 4; ++s) tacc[q] = fmaf(dz[s], x[s], tacc[q]);
    }
  }
}

// All batch chunks of one tile.  Z and G chunks go through a ring of RING
// register buffers, loaded RING-1 chunks ahead of their use; chunk indices
// past the end are clamped to the last chunk (redundant in-bounds loads) so
// every pass issues the same loads and wait counts stay exact.  The loop is
// instantiated per activation so that no activation switch sits inside it.
template <int TQ, int OM, int RING, int A, bool TAIL>
__device__ __forceinline__ void bwdl_tile(f32x4 (&acc)[TQ], float (&dw)[OM], float (&tacc)[4],
                                          const f32x4* qbase, const f32x4* tbase, int qstride,
                                          int nch, const float* zrow, const float* grow, int lk,
                                          const float (&w2)[OM], int arow) {
  f32x4 zb[RING], gb[RING][OM];
#pragma unroll
  for (int r = 0; r < RING - 1; ++r)
    bwdl_load<OM>(zb[r], gb[r], zrow, grow, 16 * (r < nch ? r : nch - 1) + 4 * lk);
  for (int c0 = 0; c0 < nch; c0 += RING) {
#pragma unroll
    for (int r = 0; r < RING; ++r) {
      const int c = c0 + r;
      const int cl = c + RING - 1 < nch ? c + RING - 1 : nch - 1;
      bwdl_load<OM>(zb[(r + RING - 1) % RING], gb[(r + RING - 1) % RING], zrow, grow,
                    16 * cl + 4 * lk);
      if (c < nch)
        bwdl_chunk<TQ, OM, A, TAIL>(acc, dw, tacc, qbase + 64 * c, qstride, tbase + 64 * c, zb[r],
                                    gb[r], w2, arow);
    }
  }
}

template <int TQ, int OM, int RING, int NT, bool TAIL>
__global__ __launch_bounds__(NT) void k_bwd_lds(BwdArgs a) {
  constexpr int NW = NT / 64;
  constexpr int TB = TQ + (TAIL ? 1 : 0);  // column blocks held in LDS
  extern __shared__ float lds[];
  const int Bp = a.Bp;
  const int nch = Bp >> 4;
  const bool grad = a.dW1 != nullptr;
  // float4 slot ((i*nch + c)*64 + l) = Xt[16i + l%16][16c + 4(l/16) .. +3] (0 past F4)
  for (int slot = threadIdx.x; slot < TB * nch * 64; slot += NT) {
    const int l = slot & 63, rest = slot >> 6;
    const int i = rest / nch, c = rest - (rest / nch) * nch;
    const int row = 16 * i + (l & 15);
    *(f32x4*)(lds + 4 * slot) =
        row < a.F4 ? *(const f32x4*)(a.Xt + (int64_t)row * Bp + 16 * c + 4 * (l >> 4))
                   : f32x4{0.f, 0.f, 0.f, 0.f};
  }
  __syncthreads();
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  const int li = lane & 15, lk = lane >> 4;
  const int64_t T = (a.N + 15) >> 4;
  const int64_t tstride = (int64_t)gridDim.x * NW;
  const f32x4* qbase = (const f32x4*)lds + lane;  // + (i*nch + c)*64
  const int qstride = nch * 64;
  // tail columns: the slots of lanes (q, lk), q < 4, of block TQ
  const f32x4* tbase = (const f32x4*)lds + TQ * qstride + 16 * lk;  // + c*64 + q
  for (int64_t t = (int64_t)blockIdx.x * NW + wave; t < T; t += tstride) {
    const int64_t p = t * 16 + li;          // this lane's row; < Npad
    const int64_t pc = p < a.N ? p : a.N - 1;
    const int m = a.mid[pc];
    const int arow = a.actn[pc];
    const float lr = a.lrm ? a.lrm[m] : a.lr;
    float w2[OM];
#pragma unroll
    for (int o = 0; o < OM; ++o) w2[o] = a.W2[(int64_t)o * a.ldw + pc];
    const float* zrow = a.Zt + pc * Bp;
    const float* grow = a.G + (int64_t)m * Bp * OM;
    // W1 strip for the update at the end of the tile
    f32x4 w1v[TQ];
    float* orow = a.W1 + p * a.F4;
    if (!grad) {
#pragma unroll
      for (int i = 0; i < TQ; ++i) {
        int q = 16 * i + 4 * lk;
        if (q > a.F4 - 4) q = a.F4 - 4;  // columns past F4 are never stored
        w1v[i] = *(const f32x4*)(orow + q);
      }
    }
    f32x4 w1t = f32x4{0.f, 0.f, 0.f, 0.f};
    if (TAIL && !grad) w1t = *(const f32x4*)(orow + 16 * TQ);
    f32x4 acc[TQ];
    float dw[OM];
    float tacc[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int i = 0; i < TQ; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int o = 0; o < OM; ++o) dw[o] = 0.f;
    // One activation for the whole tile in the common case (segments are
    // wide): a single wave-uniform branch selects the instantiated loop.
    const int a0 = __builtin_amdgcn_readfirstlane(arow);
    const int auni = __all(arow == a0) ? a0 : -1;
    switch (auni) {
      case 0: bwdl_tile<TQ, OM, RING, 0, TAIL>(acc, dw, tacc, qbase, tbase, qstride, nch, zrow, grow, lk, w2, arow); break;
      case 1: bwdl_tile<TQ, OM, RING, 1, TAIL>(acc, dw, tacc, qbase, tbase, qstride, nch, zrow, grow, lk, w2, arow); break;
      case 2: bwdl_tile<TQ, OM, RING, 2, TAIL>(acc, dw, tacc, qbase, tbase, qstride, nch, zrow, grow, lk, w2, arow); break;
      case 3: bwdl_tile<TQ, OM, RING, 3, TAIL>(acc, dw, tacc, qbase, tbase, qstride, nch, zrow, grow, lk, w2, arow); break;
      case 4: bwdl_tile<TQ, OM, RING, 4, TAIL>(acc, dw, tacc, qbase, tbase, qstride, nch, zrow, grow, lk, w2, arow); break;
      case 5: bwdl_tile<TQ, OM, RING, 5, TAIL>(acc, dw, tacc, qbase, tbase, qstride, nch, zrow, grow, lk, w2, arow); break;
      case 6: bwdl_tile<TQ, OM, RING, 6, TAIL>(acc, dw, tacc, qbase, tbase, qstride, nch, zrow, grow, lk, w2, arow); break;
      case 7: bwdl_tile<TQ, OM, RING, 7, TAIL>(acc, dw, tacc, qbase, tbase, qstride, nch, zrow, grow, lk, w2, arow); break;
      case 8: bwdl_tile<TQ, OM, RING, 8, TAIL>(acc, dw, tacc, qbase, tbase, qstride, nch, zrow, grow, lk, w2, arow); break;
      case 9: bwdl_tile<TQ, OM, RING, 9, TAIL>(acc, dw, tacc, qbase, tbase, qstride, nch, zrow, grow, lk, w2, arow); break;
      case 10: bwdl_tile<TQ, OM, RING, 10, TAIL>(acc, dw, tacc, qbase, tbase, qstride, nch, zrow, grow, lk, w2, arow); break;
      case 11: bwdl_tile<TQ, OM, RING, 11, TAIL>(acc, dw, tacc, qbase, tbase, qstride, nch, zrow, grow, lk, w2, arow); break;
      case 12: bwdl_tile<TQ, OM, RING, 12, TAIL>(acc, dw, tacc, qbase, tbase, qstride, nch, zrow, grow, lk, w2, arow); break;
      default: bwdl_tile<TQ, OM, RING, -1, TAIL>(acc, dw, tacc, qbase, tbase, qstride, nch, zrow, grow, lk, w2, arow); break;
    }
    // dW2: combine the four lk lanes of the row; lanes lk == 0 write.
#pragma unroll
    for (int o = 0; o < OM; ++o) {
      float v = dw[o];
      v += __shfl_xor(v, 16);
      v += __shfl_xor(v, 32);
      dw[o] = v;
    }
    if (TAIL) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        float v = tacc[q];
        v += __shfl_xor(v, 16);
        v += __shfl_xor(v, 32);
        tacc[q] = v;
      }
    }
    if (grad) {
      if (p < a.N) {
        if (lk == 0)
#pragma unroll
          for (int o = 0; o < OM; ++o) a.dW2[(int64_t)o * a.N + p] = dw[o];
        float* grow1 = a.dW1 + p * a.F;
#pragma unroll
        for (int i = 0; i < TQ; ++i) {
          const int q = 16 * i + 4 * lk;
#pragma unroll
          for (int r = 0; r < 4; ++r)
            if (q + r < a.F) grow1[q + r] = acc[i][r];
            else if (q + r == a.bcol && a.db1) a.db1[p] = acc[i][r];
        }
        if (TAIL && lk == 0) {
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int q = 16 * TQ + r;
            if (q < a.F) grow1[q] = tacc[r];
            else if (q == a.bcol && a.db1) a.db1[p] = tacc[r];
          }
        }
      }
    } else {
      // padded rows (p >= N) absorb the tail of the last tile
      if (lk == 0)
#pragma unroll
        for (int o = 0; o < OM; ++o) a.W2[(int64_t)o * a.ldw + p] = w2[o] - lr * dw[o];
#pragma unroll
      for (int i = 0; i < TQ; ++i) {
        const int q = 16 * i + 4 * lk;
        if (q < a.F4) *(f32x4*)(orow + q) = w1v[i] - lr * acc[i];
      }
      if (TAIL && lk == 0)
        *(f32x4*)(orow + 16 * TQ) = w1t - lr * f32x4{tacc[0], tacc[1], tacc[2], tacc[3]};
    }
  }
}

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
static hipError_t launch_persistent(void (*kern)(Arg), int nthreads, size_t lds_bytes,
                                    int64_t waves_needed, hipStream_t s, const Arg& arg) {
  const int nwaves = nthreads / 64;
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
                                                              nthreads, lds_bytes);
  if (e != hipSuccess) return e;
  if (per_cu < 1) return hipErrorInvalidConfiguration;
  int64_t blocks = (int64_t)d.cus * per_cu;
  const int64_t need = (waves_needed + nwaves - 1) / nwaves;
  if (blocks > need) blocks = need;
  if (blocks < 1) blocks = 1;
  kern<<<(unsigned)blocks, nthreads, lds_bytes, s>>>(arg);
  return hipGetLastError();
}

static size_t fwd_lds_bytes(int32_t Bp, int32_t F4) { return (size_t)Bp * F4 * 4; }

bool fwd_lds_supported(int32_t Bp, int32_t F4) {
  const DevInfo d = dev_info();
  const bool tq_ok = Bp == 16 || Bp == 32 || Bp == 64 || Bp == 128 || Bp == 256;
  return tq_ok && F4 <= 16 * kKCMax + 12 && fwd_lds_bytes(Bp, F4) <= (size_t)d.lds_max;
}

// Narrow inputs and batches (K = 16 or 32, Bp <= 64): two chunk registers,
// no remainder, four strips in flight; otherwise the one-tile-ahead kernel.
template <int TQ>
static hipError_t fwd_lds_go(const FwdLdsArgs& a, size_t lds, int64_t T, hipStream_t s) {
  if constexpr (TQ <= 4)
    if (a.K <= 32 && a.K % 16 == 0)
      return launch_persistent(k_fwd_lds_ring<TQ, 2, 0, 4>, kLdsBlock, lds, T, s, a);
  return launch_persistent(k_fwd_lds<TQ>, kLdsBlock, lds, T, s, a);
}

hipError_t launch_fwd_lds(const FwdLdsArgs& a0, hipStream_t s) {
  if (a0.N <= 0) return hipSuccess;
  if (!fwd_lds_supported(a0.Bp, a0.K)) return hipErrorInvalidValue;
  const FwdLdsArgs& a = a0;
  const size_t lds = fwd_lds_bytes(a.Bp, a.K);
  const int64_t T = (a.N + 15) / 16;
  switch (a.Bp) {
    case 16: return fwd_lds_go<1>(a, lds, T, s);
    case 32: return fwd_lds_go<2>(a, lds, T, s);
    case 64: return fwd_lds_go<4>(a, lds, T, s);
    case 128: return fwd_lds_go<8>(a, lds, T, s);
    default: return fwd_lds_go<16>(a, lds, T, s);
  }
}

// Column blocks of 16 held in LDS (the last one is the four-column tail when
// bwd_tail is set: F4 = 100, six MFMA blocks and four columns of FMAs).
static int bwd_tq(int32_t F4) {
  return F4 <= 16 ? 1 : F4 <= 32 ? 2 : F4 <= 64 ? 4 : F4 <= 112 ? 7 : 8;
}

static bool bwd_tail(int32_t F4) { return F4 == 100; }

static size_t bwd_lds_bytes(int32_t Bp, int32_t F4) { return (size_t)16 * bwd_tq(F4) * Bp * 4; }

bool bwd_lds_supported(int32_t Bp, int32_t F4, int32_t O) {
  const DevInfo d = dev_info();
  return F4 <= 128 && (O == 2 || O == 4 || O == 10) &&
         bwd_lds_bytes(Bp, F4) <= (size_t)d.lds_max;
}

template <int TQ, int OM, bool TAIL = false>
static hipError_t bwd_lds_go(const BwdArgs& a, size_t lds, hipStream_t s) {
  // One 16-row tile per wave; 12 waves per workgroup (3 per SIMD) when the
  // per-chunk G buffers are small, 8 otherwise; prefetch depth set by the
  // size of those buffers.
  constexpr int RING = OM <= 2 && !TAIL ? 4 : (OM <= 4 ? 3 : 2);
  constexpr int NT = OM <= 2 && TQ <= 7 ? 768 : 512;
  const int64_t T = (a.N + 15) / 16;
  return launch_persistent(k_bwd_lds<TQ, OM, RING, NT, TAIL>, NT, lds, T, s, a);
}

template <int OM>
static hipError_t bwd_lds_by_f(const BwdArgs& a, size_t lds, hipStream_t s) {
  switch (bwd_tq(a.F4)) {
    case 1: return bwd_lds_go<1, OM>(a, lds, s);
    case 2: return bwd_lds_go<2, OM>(a, lds, s);
    case 4: return bwd_lds_go<4, OM>(a, lds, s);
    case 7:
      if constexpr (OM == 2)
        if (bwd_tail(a.F4)) return bwd_lds_go<6, OM, true>(a, lds, s);
      return bwd_lds_go<7, OM>(a, lds, s);
    default: return bwd_lds_go<8, OM>(a, lds, s);
  }
}

hipError_t launch_bwd_lds(const BwdArgs& a0, hipStream_t s) {
  if (a0.N <= 0) return hipSuccess;
  if (!bwd_lds_supported(a0.Bp, a0.F4, a0.O)) return hipErrorInvalidValue;
  const BwdArgs& a = a0;
  const size_t lds = bwd_lds_bytes(a.Bp, a.F4);
  if (a.O == 2) return bwd_lds_by_f<2>(a, lds, s);
  if (a.O == 4) return bwd_lds_by_f<4>(a, lds, s);
  return bwd_lds_by_f<10>(a, lds, s);
}

}  // namespace pmlpk
