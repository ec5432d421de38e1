// Persistent LDS-resident GEMMs: forward and fused backward.

#include <type_traits>

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
// Forward for wide batches on the bf16 matrix cores at fp32 accuracy.
//
// Every fp32 operand a is split into three bf16 pieces, each the
// round-to-nearest of what the previous ones leave:
//   a = a0 + a1 + a2 exactly,  |a1| <= 2^-8 |a|,  |a2| <= 2^-16 |a|
// (a has 24 significant bits, each piece takes 8; exact for normal a whose
// last piece is not subnormal).  A product a b is taken as the six piece
// products a0 b0, a0 b1, a1 b0, a0 b2, a1 b1, a2 b0, each exact in the fp32
// accumulator; the three left out (a1 b2, a2 b1, a2 b2) are at most
// 2^-23 |a b| together, two units of fp32 rounding and usually far less, so
// the result carries the error of an fp32 dot product, while six
// v_mfma_f32_16x16x32_bf16 (32 k values each) stand in for the eight
// v_mfma_f32_16x16x4f32 of the same 32 k values at about a third of their
// issue time.  The batch is split once per workgroup into three LDS planes
// in MFMA-operand order (plane slot (i*NC + c)*64 + l holds the eight k
// values 32c + 8(l/16) .. +7 of sample 16i + l%16); the W1 strips are split
// in registers, each piece then serving all TQ sample tiles.  A wave takes
// U tiles of 16 units at a time, so every LDS operand feeds U products.
// The last K mod 32 columns (a multiple of 4) take fp32 MFMA steps as in
// k_fwd_lds.  Operands above about 3.4e38 in magnitude would overflow the
// first piece; weights and inputs of a network in training are far below.
// ---------------------------------------------------------------------------

static constexpr int kX3RemMax = 7;  // fp32 remainder steps: K mod 32 <= 28

// two values at a time: one packed conversion per piece, the pieces read
// back as floats from the low and high halves
__device__ __forceinline__ uint32_t bf16_pair(f32x2 v) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
}
__device__ __forceinline__ f32x2 bf16_pair_value(uint32_t p) {
  return f32x2{__builtin_bit_cast(float, p << 16), __builtin_bit_cast(float, p & 0xffff0000u)};
}

__device__ __forceinline__ void split3(const f32x4& a, const f32x4& b, bf16x8& p0, bf16x8& p1,
                                       bf16x8& p2) {
  uint32_t q0[4], q1[4], q2[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const f32x2 x = j < 2 ? f32x2{a[2 * j], a[2 * j + 1]} : f32x2{b[2 * j - 4], b[2 * j - 3]};
    q0[j] = bf16_pair(x);
    const f32x2 r1 = x - bf16_pair_value(q0[j]);
    q1[j] = bf16_pair(r1);
    q2[j] = bf16_pair(r1 - bf16_pair_value(q1[j]));
  }
  p0 = __builtin_bit_cast(bf16x8, q0);
  p1 = __builtin_bit_cast(bf16x8, q1);
  p2 = __builtin_bit_cast(bf16x8, q2);
}

// acc += a b for one 32-wide k chunk, smallest piece products first
__device__ __forceinline__ f32x4 mfma_x3(const bf16x8& a0, const bf16x8& a1, const bf16x8& a2,
                                         const bf16x8& b0, const bf16x8& b1, const bf16x8& b2,
                                         f32x4 acc) {
  acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a2, b0, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a1, b1, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a0, b2, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a1, b0, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a0, b1, acc, 0, 0, 0);
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a0, b0, acc, 0, 0, 0);
}

// Product k (0..5) of mfma_x3, in the same order.
__device__ __forceinline__ f32x4 mfma_x3_step(int k, const bf16x8& a0, const bf16x8& a1,
                                              const bf16x8& a2, const bf16x8& b0,
                                              const bf16x8& b1, const bf16x8& b2, f32x4 acc) {
  switch (k) {
    case 0: return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a2, b0, acc, 0, 0, 0);
    case 1: return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a1, b1, acc, 0, 0, 0);
    case 2: return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a0, b2, acc, 0, 0, 0);
    case 3: return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a1, b0, acc, 0, 0, 0);
    case 4: return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a0, b1, acc, 0, 0, 0);
    default: return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a0, b0, acc, 0, 0, 0);
  }
}

template <int NC, int U, int RM>
struct X3Strip {
  f32x4 c[U][2 * NC];
  float t[U][RM > 0 ? RM : 1];
};

// W1 rows (t*U + u)*16 + li: k = 32c + 8lk .. +7 per chunk and the
// remainder values k = 32NC + 4s + lk (steps past rem repeat step 0).
template <int NC, int U, int RM>
__device__ __forceinline__ void x3_load(X3Strip<NC, U, RM>& st, const float* __restrict__ W1,
                                        int64_t t, int64_t N, int K, int rem, int li, int lk) {
#pragma unroll
  for (int u = 0; u < U; ++u) {
    int64_t p = (t * U + u) * 16 + li;
    if (p > N - 1) p = N - 1;
    const float* row = W1 + p * K;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      st.c[u][2 * c] = *(const f32x4*)(row + 32 * c + 8 * lk);
      st.c[u][2 * c + 1] = *(const f32x4*)(row + 32 * c + 8 * lk + 4);
    }
#pragma unroll
    for (int s = 0; s < RM; ++s) {
      int off = 32 * NC + 4 * (s < rem ? s : 0) + lk;
      if (off > K - 1) off = K - 1;
      st.t[u][s] = row[off];
    }
  }
}

// RM: the number of fp32 remainder steps when below kX3RemMax, else a
// bound on the run-time number.
template <int TQ, int NC, int U, int RM>
__global__ __launch_bounds__(kLdsBlock) void k_fwd_x3(FwdLdsArgs a) {
  extern __shared__ float lds[];
  const int K = a.K;
  const int rem = RM < kX3RemMax ? RM : (K - 32 * NC) >> 2;
  constexpr int PS = TQ * NC * 64;  // 16-byte slots per plane
  bf16x8* planes = (bf16x8*)lds;
  for (int slot = threadIdx.x; slot < PS; slot += kLdsBlock) {
    const int l = slot & 63, rest = slot >> 6;
    const int i = rest / NC, c = rest - (rest / NC) * NC;
    const float* src = a.Xp + (int64_t)(16 * i + (l & 15)) * K + 32 * c + 8 * (l >> 4);
    bf16x8 p0, p1, p2;
    split3(*(const f32x4*)src, *(const f32x4*)(src + 4), p0, p1, p2);
    planes[slot] = p0;
    planes[PS + slot] = p1;
    planes[2 * PS + slot] = p2;
  }
  // remainder: float slot T0 + (i*rem + s)*64 + l = Xp[16i + l%16][32NC + 4s + l/16]
  constexpr int T0 = 3 * PS * 4;
  const int rdiv = rem > 0 ? rem : 1;
  for (int slot = threadIdx.x; slot < TQ * rem * 64; slot += kLdsBlock) {
    const int l = slot & 63, rest = slot >> 6;
    const int i = rest / rdiv, s = rest - (rest / rdiv) * rdiv;
    lds[T0 + slot] = a.Xp[(int64_t)(16 * i + (l & 15)) * K + 32 * NC + 4 * s + (l >> 4)];
  }
  __syncthreads();
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  const int li = lane & 15, lk = lane >> 4;
  const int64_t T = (a.N + 16 * U - 1) / (16 * U);
  const int64_t tstride = (int64_t)gridDim.x * kLdsWaves;
  int64_t t = (int64_t)blockIdx.x * kLdsWaves + wave;
  if (t >= T) return;
  const bf16x8* xq = planes + lane;  // + plane*PS + (i*NC + c)*64
  const float* qtail = lds + T0 + lane;
  // The strip of the next tile is loaded at the top of each tile and split
  // at its end, so the products only read registers written by VALU
  // instructions and no wait on memory falls inside the tile.
  X3Strip<NC, U, RM> nxt;
  x3_load(nxt, a.W1, t, a.N, K, rem, li, lk);
  bf16x8 w0[U][NC], w1[U][NC], w2[U][NC];
  float wt[U][RM > 0 ? RM : 1];
#pragma unroll
  for (int u = 0; u < U; ++u) {
#pragma unroll
    for (int c = 0; c < NC; ++c)
      split3(nxt.c[u][2 * c], nxt.c[u][2 * c + 1], w0[u][c], w1[u][c], w2[u][c]);
#pragma unroll
    for (int s = 0; s < RM; ++s) wt[u][s] = nxt.t[u][s];
  }
  for (; t < T; t += tstride) {
    const int64_t tn = t + tstride < T ? t + tstride : t;
    x3_load(nxt, a.W1, tn, a.N, K, rem, li, lk);
    __builtin_amdgcn_sched_barrier(0);
    // The six products of one accumulator issue back to back (the chained
    // accumulator is forwarded instead of read back from VGPRs, which
    // roughly halves the issue time of this MFMA); the LDS operands of the
    // next chunk are read one chunk ahead.
    bf16x8 xn0 = xq[0], xn1 = xq[PS], xn2 = xq[2 * PS];
#pragma unroll
    for (int i = 0; i < TQ; ++i) {
      f32x4 acc[U];
#pragma unroll
      for (int u = 0; u < U; ++u) acc[u] = f32x4{0.f, 0.f, 0.f, 0.f};
      // remainder operands of this sample tile, read before the chunks
      float qt[RM > 0 ? RM : 1];
      if (rem > 0) {
#pragma unroll
        for (int s = 0; s < RM; ++s) qt[s] = qtail[(i * rem + (s < rem ? s : rem - 1)) * 64];
      }
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        const bf16x8 x0 = xn0, x1 = xn1, x2 = xn2;
        if (i * NC + c + 1 < TQ * NC) {
          const int o = (i * NC + c + 1) * 64;
          xn0 = xq[o];
          xn1 = xq[PS + o];
          xn2 = xq[2 * PS + o];
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
          __builtin_amdgcn_sched_barrier(0);
          acc[u] = mfma_x3(x0, x1, x2, w0[u][c], w1[u][c], w2[u][c], acc[u]);
        }
        __builtin_amdgcn_sched_barrier(0);
      }
#pragma unroll
      for (int s = 0; s < RM; ++s) {
        if (s < rem) {
#pragma unroll
          for (int u = 0; u < U; ++u)
            acc[u] = __builtin_amdgcn_mfma_f32_16x16x4f32(qt[s], wt[u][s], acc[u], 0, 0, 0);
        }
      }
      // Zt rows are padded to a multiple of 64, so every store is in bounds.
#pragma unroll
      for (int u = 0; u < U; ++u)
        *(f32x4*)(a.Zt + ((t * U + u) * 16 + li) * (int64_t)(16 * TQ) + 16 * i + 4 * lk) = acc[u];
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int u = 0; u < U; ++u) {
#pragma unroll
      for (int c = 0; c < NC; ++c)
        split3(nxt.c[u][2 * c], nxt.c[u][2 * c + 1], w0[u][c], w1[u][c], w2[u][c]);
#pragma unroll
      for (int s = 0; s < RM; ++s) wt[u][s] = nxt.t[u][s];
    }
  }
}

// ---------------------------------------------------------------------------
// The forward product with the activation and the M3 forward in its
// epilogue (Section 3, steps 1-4 in one pass; the closing suggestion of
// Section 5, a kernel specialised for the packed forward).  The products are
// those of k_fwd_x3 with the operand roles swapped, so that lane (li, lk)
// ends a 16-sample block i holding Z of the four consecutive units
// base + 4lk .. +3 for the one sample 16i + li: the sum over a model's units
// is then mostly a sum over the lane's own registers.  Z is still stored
// (the fused backward reads it).
//
// Work units are the runs of the M3 plan (whole segments up to the tile
// cap, or one half of a wider segment), taken widest first.  A wave walks
// each model's piece of its run in 16-unit blocks that start at the
// piece's first unit, so every block holds units of one model only (the
// last block of a piece computes, but neither stores nor sums, the units
// past it; at most 15 wasted rows per piece).  Per lane and 16-sample block
// a running sum per output carries the piece across blocks; at the piece's
// last block it is combined over the four lk lanes and written once: plain
// stores for whole segments, two atomic additions onto zeroed logits for
// the halves of a wider one, so the result does not depend on the
// schedule.
//
// A block runs in parts of two 16-sample blocks, and the epilogue of each
// part (Z store, activation, products with W2) is spread one unit at a time
// between the matrix products of the next part, so the wave's vector work
// issues while its products run.  The activation is resolved once per
// block.  One 16-unit block per step keeps the strip, the running sums and
// the M3 weights within 256 VGPRs (two waves per SIMD).
// ---------------------------------------------------------------------------

struct X3MStrip {
  f32x4 c[2 * kKCMax / 2];
  float t[kX3RemMax];
};

// W1 row base + li, k = 32c + 8lk .. +7 per chunk and the remainder values
// k = 32NC + 4s + lk (rows past N clamp to the last unit; steps past rem
// repeat step 0).
template <int NC, int RM>
__device__ __forceinline__ void x3m_load(X3MStrip& st, const float* __restrict__ W1,
                                         int64_t base, int64_t N, int K, int rem, int li,
                                         int lk) {
  int64_t p = base + li;
  if (p > N - 1) p = N - 1;
  const float* row = W1 + p * K;
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    st.c[2 * c] = *(const f32x4*)(row + 32 * c + 8 * lk);
    st.c[2 * c + 1] = *(const f32x4*)(row + 32 * c + 8 * lk + 4);
  }
#pragma unroll
  for (int s = 0; s < RM; ++s) {
    int off = 32 * NC + 4 * (s < rem ? s : 0) + lk;
    if (off > K - 1) off = K - 1;
    st.t[s] = row[off];
  }
}

// f(integral_constant<int, 0>) ... f(integral_constant<int, N - 1>), in order.
template <int N, class F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (N > 0) {
    static_for<N - 1>(f);
    f(std::integral_constant<int, N - 1>{});
  }
}

template <int TQ, int NC, int RM, int OM>
__global__ __launch_bounds__(kLdsBlock) void k_fwd_x3m(FwdM3Args a) {
  extern __shared__ float lds[];
  const int K = a.K;
  const int rem = RM < kX3RemMax ? RM : (K - 32 * NC) >> 2;
  constexpr int PS = TQ * NC * 64;  // 16-byte slots per plane
  constexpr int BP = 16 * TQ;       // the padded batch (the launcher checks)
  bf16x8* planes = (bf16x8*)lds;
  for (int slot = threadIdx.x; slot < PS; slot += kLdsBlock) {
    const int l = slot & 63, rest = slot >> 6;
    const int i = rest / NC, c = rest - (rest / NC) * NC;
    const float* src = a.Xp + (int64_t)(16 * i + (l & 15)) * K + 32 * c + 8 * (l >> 4);
    bf16x8 p0, p1, p2;
    split3(*(const f32x4*)src, *(const f32x4*)(src + 4), p0, p1, p2);
    planes[slot] = p0;
    planes[PS + slot] = p1;
    planes[2 * PS + slot] = p2;
  }
  constexpr int T0 = 3 * PS * 4;
  const int rdiv = rem > 0 ? rem : 1;
  for (int slot = threadIdx.x; slot < TQ * rem * 64; slot += kLdsBlock) {
    const int l = slot & 63, rest = slot >> 6;
    const int i = rest / rdiv, s = rest - (rest / rdiv) * rdiv;
    lds[T0 + slot] = a.Xp[(int64_t)(16 * i + (l & 15)) * K + 32 * NC + 4 * s + (l >> 4)];
  }
  __syncthreads();
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  const int li = lane & 15, lk = lane >> 4;
  const int rstride = gridDim.x * kLdsWaves;
  int r = blockIdx.x * kLdsWaves + wave;
  if (r >= a.ntiles) return;
  const bf16x8* xq = planes + lane;
  const float* qtail = lds + T0 + lane;

  // run r: units [n0, n0 + len) of tile order[r]
  Tile3 run = a.tiles[__builtin_amdgcn_readfirstlane(a.order[r])];
  int64_t base = run.n0;
  int m = run.m0;  // model of the block's units
  X3MStrip nxt;
  x3m_load<NC, RM>(nxt, a.W1, base, a.N, K, rem, li, lk);
  bf16x8 w0[NC], w1[NC], w2p[NC];
  float wt[RM > 0 ? RM : 1];
#pragma unroll
  for (int c = 0; c < NC; ++c) split3(nxt.c[2 * c], nxt.c[2 * c + 1], w0[c], w1[c], w2p[c]);
#pragma unroll
  for (int s = 0; s < RM; ++s) wt[s] = nxt.t[s];
  float macc[TQ][OM];  // running sums of the open piece, sample 16i + li
#pragma unroll
  for (int i = 0; i < TQ; ++i)
#pragma unroll
    for (int o = 0; o < OM; ++o) macc[i][o] = 0.f;
  while (true) {
    const int64_t rend = run.n0 + run.len;
    int64_t pend = a.seg_off[m + 1];  // end of model m's piece of the run
    if (pend > rend) pend = rend;
    const int64_t bend = base + 16 < pend ? base + 16 : pend;
    const bool last = bend == pend;
    // the next block: in this piece, the next model's piece of this run,
    // or the first block of the wave's next run
    int rn = r, mn = m;
    int64_t bn;
    Tile3 nrun = run;
    if (!last) {
      bn = base + 16;
    } else if (pend < rend) {
      bn = pend;
      mn = m + 1;
    } else {
      rn = r + rstride;
      bn = -1;
      if (rn < a.ntiles) {
        nrun = a.tiles[__builtin_amdgcn_readfirstlane(a.order[rn])];
        bn = nrun.n0;
        mn = nrun.m0;
      }
    }
    x3m_load<NC, RM>(nxt, a.W1, bn >= 0 ? bn : base, a.N, K, rem, li, lk);
    // the lane's four units and their output weights; units past the
    // piece get zero weights and are neither stored nor activated
    const int64_t u0 = base + 4 * lk;
    bool in[4];
    float w2v[OM][4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      in[q] = u0 + q < bend;
      int64_t u = u0 + q;
      if (u > a.N - 1) u = a.N - 1;
#pragma unroll
      for (int o = 0; o < OM; ++o) {
        const float w = o < a.O ? a.W2[(int64_t)o * a.ldw + u] : 0.f;
        w2v[o][q] = in[q] ? w : 0.f;
      }
    }
    __builtin_amdgcn_sched_barrier(0);
    float* zp = a.Zt + u0 * (int64_t)BP + li;
    bf16x8 xn0 = xq[0], xn1 = xq[PS], xn2 = xq[2 * PS];
    // The block in parts of TP sample blocks; the epilogue of part P - 1
    // goes between the products of part P, that of the last part after them.
    auto blk = [&](auto ac) __attribute__((always_inline)) {
      constexpr int A = decltype(ac)::value;
      constexpr int TP = 2;           // sample blocks per part
      constexpr int S = TP * 6 * NC;  // bf16 product slots per part
      constexpr int E = 4 * TP;       // epilogue units per part
      f32x4 acc[2][TP];
      // unit e of the epilogue of part P (sample block P TP + e/4, unit e%4)
      auto epi = [&](auto pc, int e) __attribute__((always_inline)) {
        constexpr int P = decltype(pc)::value;
        const int j = e >> 2, q = e & 3, i = P * TP + j;
        const float z = acc[P & 1][j][q];
        if (in[q]) zp[q * BP + 16 * i] = z;
        const float h = in[q] ? act_fwd(A, z) : 0.f;
#pragma unroll
        for (int o = 0; o < OM; ++o) macc[i][o] = fmaf(h, w2v[o][q], macc[i][o]);
      };
      auto step = [&](auto pc) __attribute__((always_inline)) {
        constexpr int P = decltype(pc)::value;
#pragma unroll
        for (int j = 0; j < TP; ++j) {
          const int i = P * TP + j;
          f32x4 c4 = f32x4{0.f, 0.f, 0.f, 0.f};
          float qt[RM > 0 ? RM : 1];
          if (rem > 0) {
#pragma unroll
            for (int s = 0; s < RM; ++s) qt[s] = qtail[(i * rem + (s < rem ? s : rem - 1)) * 64];
          }
#pragma unroll
          for (int c = 0; c < NC; ++c) {
            const bf16x8 x0 = xn0, x1 = xn1, x2 = xn2;
            if (i * NC + c + 1 < TQ * NC) {
              const int o = (i * NC + c + 1) * 64;
              xn0 = xq[o];
              xn1 = xq[PS + o];
              xn2 = xq[2 * PS + o];
            }
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int k = 0; k < 6; ++k) {
              c4 = mfma_x3_step(k, w0[c], w1[c], w2p[c], x0, x1, x2, c4);
              if constexpr (P > 0) {
                const int slot = (j * NC + c) * 6 + k;
#pragma unroll
                for (int e = 0; e < E; ++e)
                  if (e * S / E == slot) epi(std::integral_constant<int, P - 1>{}, e);
              }
              __builtin_amdgcn_sched_barrier(0);
            }
          }
#pragma unroll
          for (int s = 0; s < RM; ++s)
            if (s < rem) c4 = __builtin_amdgcn_mfma_f32_16x16x4f32(wt[s], qt[s], c4, 0, 0, 0);
          acc[P & 1][j] = c4;
        }
      };
      static_for<TQ / TP>(step);
#pragma unroll
      for (int e = 0; e < E; ++e) epi(std::integral_constant<int, TQ / TP - 1>{}, e);
    };
    switch (a.act[m]) {
      case 0: blk(std::integral_constant<int, 0>{}); break;
      case 1: blk(std::integral_constant<int, 1>{}); break;
      case 2: blk(std::integral_constant<int, 2>{}); break;
      case 3: blk(std::integral_constant<int, 3>{}); break;
      case 4: blk(std::integral_constant<int, 4>{}); break;
      case 5: blk(std::integral_constant<int, 5>{}); break;
      case 6: blk(std::integral_constant<int, 6>{}); break;
      case 7: blk(std::integral_constant<int, 7>{}); break;
      case 8: blk(std::integral_constant<int, 8>{}); break;
      case 9: blk(std::integral_constant<int, 9>{}); break;
      case 10: blk(std::integral_constant<int, 10>{}); break;
      case 11: blk(std::integral_constant<int, 11>{}); break;
      default: blk(std::integral_constant<int, 12>{}); break;
    }
    if (last) {
      // model m's piece ends here: combine the four lk lanes and write each
      // sample's logits once
      const bool with_b2 = a.b2 && a.seg_off[m] >= run.n0;
      // one lane address; the sample blocks step by a wave-uniform stride
      float* const dst0 = a.out + (int64_t)m * a.sm + (int64_t)li * a.sb;
#pragma unroll
      for (int i = 0; i < TQ; ++i) {
        float v[OM];
#pragma unroll
        for (int o = 0; o < OM; ++o) {
          v[o] = macc[i][o];
          v[o] += __shfl_xor(v[o], 16);
          v[o] += __shfl_xor(v[o], 32);
          macc[i][o] = 0.f;
        }
        const int b = 16 * i + li;
        if (lk == 0 && b < a.B) {
          float* dst = dst0 + (int64_t)(16 * i) * a.sb;
#pragma unroll
          for (int o = 0; o < OM; ++o)
            if (o < a.O) {
              const float val = v[o] + (with_b2 ? a.b2[(int64_t)m * a.O + o] : 0.f);
              if (run.atomic) atomicAdd(dst + o, val);
              else dst[o] = val;
            }
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    __builtin_amdgcn_sched_barrier(0);
    if (bn < 0) break;
    if (rn != r) {
      r = rn;
      run = nrun;
    }
    m = mn;
    base = bn;
#pragma unroll
    for (int c = 0; c < NC; ++c) split3(nxt.c[2 * c], nxt.c[2 * c + 1], w0[c], w1[c], w2p[c]);
#pragma unroll
    for (int s = 0; s < RM; ++s) wt[s] = nxt.t[s];
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
    if (a.fmask) {  // masked features: zero gradient, so their weights stay 0
#pragma unroll
      for (int i = 0; i < TQ; ++i) acc[i] = fmask4(a.fmask, a.fmw, m, 16 * i + 4 * lk, acc[i]);
      if (TAIL) {
        const f32x4 t = fmask4(a.fmask, a.fmw, m, 16 * TQ, f32x4{tacc[0], tacc[1], tacc[2], tacc[3]});
#pragma unroll
        for (int q = 0; q < 4; ++q) tacc[q] = t[q];
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

// ---------------------------------------------------------------------------
// Fused backward with the dW1 product on the bf16 matrix cores at fp32
// accuracy (the three-piece split of k_fwd_x3), for batches of 128 and 256
// samples and O <= 4.  The batch goes through 32-sample chunks: lane
// (li, lk) forms dZ of row li for the eight samples 32c + 8lk .. +7, splits
// them into three bf16 pieces, and six v_mfma_f32_16x16x32_bf16 per column
// block replace the eight fp32 steps of the same 32 samples.  The batch Xt
// sits in LDS as three planes of pieces (slot (i*nc + c)*64 + l holds
// Xt[16i + l%16][32c + 8(l/16) .. +7]); with TAIL the four columns past
// 16 TQ have planes of their own (slot (c*4 + lk)*4 + q holds
// Xt[16 TQ + q][32c + 8lk .. +7]) and take one more block of products in
// which lanes li >= 4 read a zero slot, so lane (li, 0) ends with those four
// columns of row li.  The rest (gather of G, dW2, updates) is as in
// k_bwd_lds.
// ---------------------------------------------------------------------------

template <int OM>
__device__ __forceinline__ void bx3_load(f32x4 (&cz)[2], f32x4 (&cg)[2 * OM], const float* zrow,
                                         const float* grow, int kofs) {
  cz[0] = *(const f32x4*)(zrow + kofs);
  cz[1] = *(const f32x4*)(zrow + kofs + 4);
  // G[m][b .. b+7][0 .. OM-1] is 8*OM consecutive floats
#pragma unroll
  for (int v = 0; v < 2 * OM; ++v) cg[v] = *(const f32x4*)(grow + kofs * OM + 4 * v);
}

template <int TQ, int OM, int A, bool TAIL>
__device__ __forceinline__ void bx3_chunk(f32x4 (&acc)[TQ + 1], float (&dw)[OM],
                                          const bf16x8* xq, int QS, int PS, const bf16x8* xt,
                                          int TS,
                                          const f32x4 (&cz)[2],
                                          const f32x4 (&cg)[2 * OM], const float (&w2)[OM],
                                          int arow) {
  const float* g = (const float*)&cg[0];  // g[j*OM + o] = G[m][b+j][o]
  float dz[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    float hp;
    const float h = act_fwd_bwd(A >= 0 ? A : arow, cz[j >> 2][j & 3], &hp);
    float dh = 0.f;
#pragma unroll
    for (int o = 0; o < OM; ++o) {
      dh = fmaf(g[j * OM + o], w2[o], dh);
      dw[o] = fmaf(g[j * OM + o], h, dw[o]);
    }
    dz[j] = dh * hp;
    if (j == 3) __builtin_amdgcn_sched_barrier(0);  // four activations in flight at a time
  }
  bf16x8 d0, d1, d2;
  split3(f32x4{dz[0], dz[1], dz[2], dz[3]}, f32x4{dz[4], dz[5], dz[6], dz[7]}, d0, d1, d2);
  // the LDS operands of block i + 1 are read while block i multiplies
  // (two blocks of pieces live at a time)
  bf16x8 xn0 = xq[0], xn1 = xq[PS], xn2 = xq[2 * PS];
#pragma unroll
  for (int i = 0; i < TQ; ++i) {
    const bf16x8 x0 = xn0, x1 = xn1, x2 = xn2;
    if (i + 1 < TQ) {
      xn0 = xq[(i + 1) * QS];
      xn1 = xq[PS + (i + 1) * QS];
      xn2 = xq[2 * PS + (i + 1) * QS];
    } else if (TAIL) {
      xn0 = xt[0];
      xn1 = xt[TS];
      xn2 = xt[2 * TS];
    }
    __builtin_amdgcn_sched_barrier(0);
    acc[i] = mfma_x3(x0, x1, x2, d0, d1, d2, acc[i]);
    __builtin_amdgcn_sched_barrier(0);
  }
  if (TAIL) acc[TQ] = mfma_x3(xn0, xn1, xn2, d0, d1, d2, acc[TQ]);
}

template <int TQ, int OM, int RING, int A, bool TAIL>
__device__ __forceinline__ void bx3_tile(f32x4 (&acc)[TQ + 1], float (&dw)[OM],
                                         const bf16x8* xq, int PS, const bf16x8* xt, int TS,
                                         int tcs, int nc, const float* zrow, const float* grow,
                                         int lk, const float (&w2)[OM], int arow) {
  f32x4 zb[RING][2], gb[RING][2 * OM];
#pragma unroll
  for (int r = 0; r < RING - 1; ++r)
    bx3_load<OM>(zb[r], gb[r], zrow, grow, 32 * (r < nc ? r : nc - 1) + 8 * lk);
  for (int c0 = 0; c0 < nc; c0 += RING) {
#pragma unroll
    for (int r = 0; r < RING; ++r) {
      const int c = c0 + r;
      const int cl = c + RING - 1 < nc ? c + RING - 1 : nc - 1;
      bx3_load<OM>(zb[(r + RING - 1) % RING], gb[(r + RING - 1) % RING], zrow, grow,
                   32 * cl + 8 * lk);
      if (c < nc)
        bx3_chunk<TQ, OM, A, TAIL>(acc, dw, xq + c * 64, nc * 64, PS, xt + c * tcs, TS, zb[r],
                                   gb[r], w2, arow);
    }
  }
}

template <int TQ, int OM, int RING, int NT, bool TAIL>
__global__ __launch_bounds__(NT) void k_bwd_x3(BwdArgs a) {
  constexpr int NW = NT / 64;
  extern __shared__ float lds[];
  const int Bp = a.Bp;
  const int nc = Bp >> 5;
  const bool grad = a.dW1 != nullptr;
  const int PS = TQ * nc * 64;          // main slots per plane
  const int TS = TAIL ? nc * 16 : 0;    // tail slots per plane
  bf16x8* planes = (bf16x8*)lds;        // plane p: main at p*PS, tail at 3*PS + p*TS
  for (int slot = threadIdx.x; slot < PS + TS; slot += NT) {
    int row, col;
    if (slot < PS) {
      const int l = slot & 63, rest = slot >> 6;
      const int i = rest / nc, c = rest - (rest / nc) * nc;
      row = 16 * i + (l & 15);
      col = 32 * c + 8 * (l >> 4);
    } else {
      const int s = slot - PS, q = s & 3, lk = (s >> 2) & 3, c = s >> 4;
      row = 16 * TQ + q;
      col = 32 * c + 8 * lk;
    }
    const float* src = a.Xt + (int64_t)row * Bp + col;
    bf16x8 p0, p1, p2;
    split3(*(const f32x4*)src, *(const f32x4*)(src + 4), p0, p1, p2);
    const int base = slot < PS ? slot : 3 * PS + (slot - PS);
    const int pstride = slot < PS ? PS : TS;
    planes[base] = p0;
    planes[base + pstride] = p1;
    planes[base + 2 * pstride] = p2;
  }
  if (TAIL && threadIdx.x == 0)
    planes[3 * PS + 3 * TS] = __builtin_bit_cast(bf16x8, f32x4{0.f, 0.f, 0.f, 0.f});
  __syncthreads();
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  const int li = lane & 15, lk = lane >> 4;
  const int64_t T = (a.N + 15) >> 4;
  const int64_t tstride = (int64_t)gridDim.x * NW;
  const bf16x8* xq = planes + lane;                               // + (i*nc + c)*64
  // tail operands: lanes li < 4 read their slots (stride 16 per chunk, TS
  // per plane), the others one zero slot past the tail planes (stride 0)
  const bool tlane = li < 4;
  const bf16x8* xt = planes + (tlane ? 3 * PS + 4 * lk + li : 3 * PS + 3 * TS);
  const int tcs = tlane ? 16 : 0, tps = tlane ? TS : 0;
  for (int64_t t = (int64_t)blockIdx.x * NW + wave; t < T; t += tstride) {
    const int64_t p = t * 16 + li;  // this lane's row; < Npad
    const int64_t pc = p < a.N ? p : a.N - 1;
    const int m = a.mid[pc];
    const int arow = a.actn[pc];
    const float lr = a.lrm ? a.lrm[m] : a.lr;
    float w2[OM];
#pragma unroll
    for (int o = 0; o < OM; ++o) w2[o] = a.W2[(int64_t)o * a.ldw + pc];
    const float* zrow = a.Zt + pc * Bp;
    const float* grow = a.G + (int64_t)m * Bp * OM;
    float* orow = a.W1 + p * a.F4;
    f32x4 acc[TQ + 1];
    float dw[OM];
#pragma unroll
    for (int i = 0; i <= TQ; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int o = 0; o < OM; ++o) dw[o] = 0.f;
    const int a0 = __builtin_amdgcn_readfirstlane(arow);
    const int auni = __all(arow == a0) ? a0 : -1;
#define PMLP_BX3(AA) \
  bx3_tile<TQ, OM, RING, AA, TAIL>(acc, dw, xq, PS, xt, tps, tcs, nc, zrow, grow, lk, w2, arow)
    switch (auni) {
      case 0: PMLP_BX3(0); break;
      case 1: PMLP_BX3(1); break;
      case 2: PMLP_BX3(2); break;
      case 3: PMLP_BX3(3); break;
      case 4: PMLP_BX3(4); break;
      case 5: PMLP_BX3(5); break;
      case 6: PMLP_BX3(6); break;
      case 7: PMLP_BX3(7); break;
      case 8: PMLP_BX3(8); break;
      case 9: PMLP_BX3(9); break;
      case 10: PMLP_BX3(10); break;
      case 11: PMLP_BX3(11); break;
      case 12: PMLP_BX3(12); break;
      default: PMLP_BX3(-1); break;
    }
#undef PMLP_BX3
#pragma unroll
    for (int o = 0; o < OM; ++o) {
      float v = dw[o];
      v += __shfl_xor(v, 16);
      v += __shfl_xor(v, 32);
      dw[o] = v;
    }
    if (a.fmask) {  // masked features: zero gradient, so their weights stay 0
#pragma unroll
      for (int i = 0; i < TQ; ++i) acc[i] = fmask4(a.fmask, a.fmw, m, 16 * i + 4 * lk, acc[i]);
      if (TAIL) acc[TQ] = fmask4(a.fmask, a.fmw, m, 16 * TQ, acc[TQ]);
    }
    if (grad) {
      if (p < a.N) {
        if (lk == 0)
#pragma unroll
          for (int o = 0; o < OM; ++o) a.dW2[(int64_t)o * a.N + p] = dw[o];
        float* grow1 = a.dW1 + p * a.F;
#pragma unroll
        for (int i = 0; i <= TQ; ++i) {
          if (i == TQ && (!TAIL || lk != 0)) continue;
          const int q = 16 * i + 4 * lk;
#pragma unroll
          for (int r = 0; r < 4; ++r)
            if (q + r < a.F) grow1[q + r] = acc[i][r];
            else if (q + r == a.bcol && a.db1) a.db1[p] = acc[i][r];
        }
      }
    } else {
      // padded rows (p >= N) absorb the tail of the last tile; the W1
      // strip is read here (other waves cover the latency) to keep the
      // registers of the chunk loop free
      f32x4 w1v[TQ + 1];
#pragma unroll
      for (int i = 0; i < TQ; ++i) w1v[i] = *(const f32x4*)(orow + 16 * i + 4 * lk);
      if (TAIL) w1v[TQ] = *(const f32x4*)(orow + 16 * TQ);
      if (lk == 0)
#pragma unroll
        for (int o = 0; o < OM; ++o) a.W2[(int64_t)o * a.ldw + p] = w2[o] - lr * dw[o];
#pragma unroll
      for (int i = 0; i < TQ; ++i)
        *(f32x4*)(orow + 16 * i + 4 * lk) = w1v[i] - lr * acc[i];
      if (TAIL && lk == 0) *(f32x4*)(orow + 16 * TQ) = w1v[TQ] - lr * acc[TQ];
    }
  }
}

// ---------------------------------------------------------------------------
// Fused backward for wider output layers (O = 5 .. 16).  The gather of G by
// model id and its products with W2 and with the hidden activations are,
// for the units of one model, two small dense contractions per 16-sample
// batch chunk, taken by v_mfma_f32_16x16x4f32:
//   dH^T[b][n] = sum_o G[m][b][o] W2[o][n]     (K = o, ceil(O/4) steps)
//   dW2[o][n] += sum_b G[m][b][o] act(Z[n][b]) (K = b, four steps)
// Lane (li, lk) supplies G[m][16c + li][4j + lk] and W2[4j + lk][row li]
// for the first and G[m][16c + 4lk + s][li] and act(Z[row li][16c + 4lk + s])
// for the second; the first lands dH exactly where the lane holds its Z
// values (row li, samples 4lk .. +3), the second leaves dW2[4lk + r][row li]
// in the lane that updates it.  A tile whose rows belong to several models
// repeats both products once per model with the other models' rows zeroed
// in the W2 and activation operands; the G operand is shared by all 16
// rows, so in such a tile non-finite G values (a diverged model, whose own
// loss is already non-finite) are taken as zero rather than let them reach
// the other models' rows.  Per chunk a lane holds 4 + 4 values
// of G instead of 4 O, so the kernel keeps more waves in flight; the dW1
// product, the W1 update and the batch in LDS are as in k_bwd_lds.
// ---------------------------------------------------------------------------

// G operands of one model for chunk c: g1[j] = G[mm][16c + li][4j + lk],
// g2[s] = G[mm][16c + 4lk + s][li], read at the wave-uniform chunk base
// gc = G + (mm Bp + 16c) O plus the lane's chunk-invariant offsets (outputs
// past O clamped there, so every chunk issues the same loads, and their
// values zeroed here).
struct BwdmOffsets {
  uint32_t o1[4], o2[4];
  bool v1[4], v2;
};

__device__ __forceinline__ void bwdm_gload(float (&g1)[4], float (&g2)[4],
                                           const float* __restrict__ gc, const BwdmOffsets& of) {
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const float v = gc[of.o1[j]];
    g1[j] = of.v1[j] ? v : 0.f;
  }
#pragma unroll
  for (int s = 0; s < 4; ++s) {
    const float v = gc[of.o2[s]];
    g2[s] = of.v2 ? v : 0.f;
  }
}

// dH^T += G W2 and dW2 += G^T act(Z) for one model's rows of the tile.
__device__ __forceinline__ void bwdm_products(f32x4& dh, f32x4& acc2, const float (&g1)[4],
                                              const float (&g2)[4], const float (&wB)[4],
                                              const float (&h)[4], bool mine, bool multi,
                                              int JO) {
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    if (j < JO) {
      const float g = multi && !isfinite(g1[j]) ? 0.f : g1[j];
      dh = __builtin_amdgcn_mfma_f32_16x16x4f32(g, mine ? wB[j] : 0.f, dh, 0, 0, 0);
    }
  }
#pragma unroll
  for (int s = 0; s < 4; ++s) {
    const float g = multi && !isfinite(g2[s]) ? 0.f : g2[s];
    acc2 = __builtin_amdgcn_mfma_f32_16x16x4f32(g, mine ? h[s] : 0.f, acc2, 0, 0, 0);
  }
}

// All batch chunks of one tile.  Z and the G operands of the tile's first
// model go through a ring of RING register buffers, RING-1 chunks ahead
// (chunk indices past the end clamped to the last chunk); the G operands of
// further models (tiles that span a segment boundary) are loaded in place.
template <int TQ, int RING, int A>
__device__ __forceinline__ void bwdm_tile(f32x4 (&acc)[TQ], f32x4& acc2, const f32x4* qbase,
                                          int qstride, int nch, const float* zrow,
                                          const float* __restrict__ G, int Bp, int O,
                                          int m_first, int m_last, int m_row,
                                          const float (&wB)[4], int arow, int li, int lk) {
  const int JO = (O + 3) >> 2;
  const bool multi = m_first != m_last;
  const float* g0 = G + (int64_t)m_first * Bp * O;
  BwdmOffsets of;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int o = 4 * j + lk;
    of.o1[j] = (uint32_t)(li * O + (o < O ? o : O - 1));
    of.v1[j] = o < O;
    of.o2[j] = (uint32_t)((4 * lk + j) * O + (li < O ? li : O - 1));
  }
  of.v2 = li < O;
  f32x4 zb[RING];
  float g1b[RING][4], g2b[RING][4];
#pragma unroll
  for (int r = 0; r < RING - 1; ++r) {
    const int c = r < nch ? r : nch - 1;
    zb[r] = *(const f32x4*)(zrow + 16 * c + 4 * lk);
    bwdm_gload(g1b[r], g2b[r], g0 + 16 * c * O, of);
  }
  for (int c0 = 0; c0 < nch; c0 += RING) {
#pragma unroll
    for (int r = 0; r < RING; ++r) {
      const int c = c0 + r;
      const int cl = c + RING - 1 < nch ? c + RING - 1 : nch - 1;
      const int rn = (r + RING - 1) % RING;
      zb[rn] = *(const f32x4*)(zrow + 16 * cl + 4 * lk);
      bwdm_gload(g1b[rn], g2b[rn], g0 + 16 * cl * O, of);
      if (c < nch) {
        float h[4], hp[4];
#pragma unroll
        for (int s = 0; s < 4; ++s) h[s] = act_fwd_bwd(A >= 0 ? A : arow, zb[r][s], &hp[s]);
        f32x4 dh = f32x4{0.f, 0.f, 0.f, 0.f};
        bwdm_products(dh, acc2, g1b[r], g2b[r], wB, h, m_row == m_first, multi, JO);
        for (int mm = m_first + 1; mm <= m_last; ++mm) {
          float g1[4], g2[4];
          bwdm_gload(g1, g2, G + ((int64_t)mm * Bp + 16 * c) * O, of);
          bwdm_products(dh, acc2, g1, g2, wB, h, m_row == mm, multi, JO);
        }
        float dz[4];
#pragma unroll
        for (int s = 0; s < 4; ++s) dz[s] = dh[s] * hp[s];
#pragma unroll
        for (int i = 0; i < TQ; ++i) {
          const f32x4 q = qbase[i * qstride + 64 * c];
#pragma unroll
          for (int s = 0; s < 4; ++s)
            acc[i] = __builtin_amdgcn_mfma_f32_16x16x4f32(q[s], dz[s], acc[i], 0, 0, 0);
        }
      }
    }
  }
}

template <int TQ, int RING, int NT>
__global__ __launch_bounds__(NT, TQ <= 2 ? 3 : 2) void k_bwd_mf(BwdArgs a) {
  constexpr int NW = NT / 64;
  extern __shared__ float lds[];
  const int Bp = a.Bp, O = a.O;
  const int nch = Bp >> 4;
  const bool grad = a.dW1 != nullptr;
  // float4 slot ((i*nch + c)*64 + l) = Xt[16i + l%16][16c + 4(l/16) .. +3] (0 past F4)
  for (int slot = threadIdx.x; slot < TQ * nch * 64; slot += NT) {
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
  for (int64_t t = (int64_t)blockIdx.x * NW + wave; t < T; t += tstride) {
    const int64_t p = t * 16 + li;  // this lane's row; < Npad
    const int64_t pc = p < a.N ? p : a.N - 1;
    const int m_row = a.mid[pc];
    const int arow = a.actn[pc];
    const float lr = a.lrm ? a.lrm[m_row] : a.lr;
    // models of the tile's rows: a contiguous range (segments are contiguous)
    const int64_t plast = t * 16 + 15 < a.N ? t * 16 + 15 : a.N - 1;
    const int m_first = __builtin_amdgcn_readfirstlane(a.mid[t * 16]);
    const int m_last = __builtin_amdgcn_readfirstlane(a.mid[plast]);
    // W2 operand of dH (rows 4j + lk) and old W2 of the update (rows 4lk + r)
    float wB[4], w2u[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int o = 4 * j + lk;
      wB[j] = o < O ? a.W2[(int64_t)o * a.ldw + pc] : 0.f;
      const int ou = 4 * lk + j;
      w2u[j] = ou < O ? a.W2[(int64_t)ou * a.ldw + pc] : 0.f;
    }
    const float* zrow = a.Zt + pc * Bp;
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
    f32x4 acc[TQ], acc2 = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int i = 0; i < TQ; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
    const int a0 = __builtin_amdgcn_readfirstlane(arow);
    const int auni = __all(arow == a0) ? a0 : -1;
#define PMLP_BWDM(AA)                                                                      \
  bwdm_tile<TQ, RING, AA>(acc, acc2, qbase, qstride, nch, zrow, a.G, Bp, O, m_first, m_last, \
                          m_row, wB, arow, li, lk)
    switch (auni) {
      case 0: PMLP_BWDM(0); break;
      case 1: PMLP_BWDM(1); break;
      case 2: PMLP_BWDM(2); break;
      case 3: PMLP_BWDM(3); break;
      case 4: PMLP_BWDM(4); break;
      case 5: PMLP_BWDM(5); break;
      case 6: PMLP_BWDM(6); break;
      case 7: PMLP_BWDM(7); break;
      case 8: PMLP_BWDM(8); break;
      case 9: PMLP_BWDM(9); break;
      case 10: PMLP_BWDM(10); break;
      case 11: PMLP_BWDM(11); break;
      case 12: PMLP_BWDM(12); break;
      default: PMLP_BWDM(-1); break;
    }
#undef PMLP_BWDM
    if (a.fmask) {  // masked features: zero gradient, so their weights stay 0
#pragma unroll
      for (int i = 0; i < TQ; ++i)
        acc[i] = fmask4(a.fmask, a.fmw, m_row, 16 * i + 4 * lk, acc[i]);
    }
    // lane (li, lk) holds dW2[4lk + r][row li]
    if (grad) {
      if (p < a.N) {
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (4 * lk + r < O) a.dW2[(int64_t)(4 * lk + r) * a.N + p] = acc2[r];
        float* grow1 = a.dW1 + p * a.F;
#pragma unroll
        for (int i = 0; i < TQ; ++i) {
          const int q = 16 * i + 4 * lk;
#pragma unroll
          for (int r = 0; r < 4; ++r)
            if (q + r < a.F) grow1[q + r] = acc[i][r];
            else if (q + r == a.bcol && a.db1) a.db1[p] = acc[i][r];
        }
      }
    } else {
      // padded rows (p >= N) absorb the tail of the last tile
#pragma unroll
      for (int r = 0; r < 4; ++r)
        if (4 * lk + r < O) a.W2[(int64_t)(4 * lk + r) * a.ldw + p] = w2u[r] - lr * acc2[r];
#pragma unroll
      for (int i = 0; i < TQ; ++i) {
        const int q = 16 * i + 4 * lk;
        if (q < a.F4) *(f32x4*)(orow + q) = w1v[i] - lr * acc[i];
      }
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
// Batches of 128 and 256 samples: the bf16 three-piece kernel when its
// three planes fit in LDS; two unit tiles per wave while the split strips
// of both fit in registers (K < 128), one above.
static size_t fwd_x3_bytes(int32_t Bp, int32_t K) {
  return (size_t)3 * Bp * (K / 32) * 64 + (size_t)Bp * ((K % 32) / 4) * 16;
}

template <int TQ, int NC>
static hipError_t fwd_x3_go(const FwdLdsArgs& a, hipStream_t s) {
  constexpr int U = NC <= 3 ? 2 : 1;
  const int64_t T = (a.N + 16 * U - 1) / (16 * U);
  const size_t lds = fwd_x3_bytes(a.Bp, a.K);
  note_variant("k_fwd_x3", kArithX3);
  switch ((a.K % 32) / 4) {
    case 0: return launch_persistent(k_fwd_x3<TQ, NC, U, 0>, kLdsBlock, lds, T, s, a);
    case 1: return launch_persistent(k_fwd_x3<TQ, NC, U, 1>, kLdsBlock, lds, T, s, a);
    default: return launch_persistent(k_fwd_x3<TQ, NC, U, kX3RemMax>, kLdsBlock, lds, T, s, a);
  }
}

template <int TQ>
static hipError_t fwd_lds_go(const FwdLdsArgs& a, size_t lds, int64_t T, hipStream_t s) {
  if constexpr (TQ <= 4) {
    if (a.K <= 32 && a.K % 16 == 0) {
      note_variant("k_fwd_lds_ring", kArithFp32);
      return launch_persistent(k_fwd_lds_ring<TQ, 2, 0, 4>, kLdsBlock, lds, T, s, a);
    }
  } else {
    if (fwd_x3_bytes(a.Bp, a.K) <= (size_t)dev_info().lds_max) {
      switch (a.K / 32) {
        case 1: return fwd_x3_go<TQ, 1>(a, s);
        case 2: return fwd_x3_go<TQ, 2>(a, s);
        case 3: return fwd_x3_go<TQ, 3>(a, s);
        case 4: if constexpr (TQ == 8) return fwd_x3_go<TQ, 4>(a, s); break;  // K <= 140
        default: break;
      }
    }
  }
  note_variant("k_fwd_lds", kArithFp32);
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

// The forward with the M3 epilogue: batches of 128 and 256 samples, the
// three planes of k_fwd_x3 in LDS, O <= 2.
bool fwd_m3_supported(int32_t Bp, int32_t F4, int32_t O) {
  if ((Bp != 128 && Bp != 256) || O > 2 || F4 < 32) return false;
  const int nc = F4 / 32;
  if (nc < 1 || nc > (Bp == 128 ? 4 : 3)) return false;
  // with more than one fp32 remainder step the wider instances would spill
  // registers (two or more chunks at 256 samples, four at 128); those
  // shapes take the two-kernel forward
  if ((F4 % 32) / 4 > 1 && (Bp == 256 ? nc >= 2 : nc >= 4)) return false;
  return fwd_x3_bytes(Bp, F4) <= (size_t)dev_info().lds_max;
}

template <int TQ, int NC>
static hipError_t fwd_m3_go(const FwdM3Args& a, hipStream_t s) {
  const size_t lds = fwd_x3_bytes(a.Bp, a.K);
  note_variant("k_fwd_x3m", kArithX3);
  switch ((a.K % 32) / 4) {
    case 0: return launch_persistent(k_fwd_x3m<TQ, NC, 0, 2>, kLdsBlock, lds, a.ntiles, s, a);
    case 1: return launch_persistent(k_fwd_x3m<TQ, NC, 1, 2>, kLdsBlock, lds, a.ntiles, s, a);
    default:
      return launch_persistent(k_fwd_x3m<TQ, NC, kX3RemMax, 2>, kLdsBlock, lds, a.ntiles, s, a);
  }
}

hipError_t launch_fwd_m3(const FwdM3Args& a, hipStream_t s) {
  if (a.N <= 0 || a.ntiles <= 0) return hipSuccess;
  if (!fwd_m3_supported(a.Bp, a.K, a.O)) return hipErrorInvalidValue;
  if (a.Bp == 128) {
    switch (a.K / 32) {
      case 1: return fwd_m3_go<8, 1>(a, s);
      case 2: return fwd_m3_go<8, 2>(a, s);
      case 3: return fwd_m3_go<8, 3>(a, s);
      default: return fwd_m3_go<8, 4>(a, s);
    }
  }
  switch (a.K / 32) {
    case 1: return fwd_m3_go<16, 1>(a, s);
    case 2: return fwd_m3_go<16, 2>(a, s);
    default: return fwd_m3_go<16, 3>(a, s);
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
  return F4 <= 128 && (O == 2 || O == 4 || (O >= 5 && O <= 16)) &&
         bwd_lds_bytes(Bp, F4) <= (size_t)d.lds_max;
}

// Narrow inputs (two column blocks or fewer): workgroups of four waves and
// at least three waves per SIMD (the batch copy is at most 32 KB, so several
// workgroups share a CU); eight-wave workgroups otherwise.
template <int TQ>
static hipError_t bwd_mf_go(const BwdArgs& a, size_t lds, hipStream_t s) {
  const int64_t T = (a.N + 15) / 16;
  constexpr int NT = TQ <= 2 ? 256 : 512;
  note_variant("k_bwd_mf", kArithFp32);
  return launch_persistent(k_bwd_mf<TQ, 2, NT>, NT, lds, T, s, a);
}

// Batches of 128 and 256 samples with F4 = 16 TQ or 16 TQ + 4 (TQ column
// blocks and the four-column tail), 32 <= F4 <= 128, and O = 2 or 4: the
// bf16 three-piece kernel.
static size_t bwd_x3_bytes(int32_t Bp, int32_t F4) {
  const int tq = F4 / 16, nc = Bp / 32;
  return (size_t)3 * (tq * nc * 64 + (F4 % 16 ? nc * 16 : 0)) * 16 + (F4 % 16 ? 16 : 0);
}

static bool bwd_x3_shape(const BwdArgs& a) {
  return (a.Bp == 128 || a.Bp == 256) && (a.O == 2 || a.O == 4) && a.F4 >= 32 &&
         a.F4 <= 128 && (a.F4 % 16 == 0 || a.F4 % 16 == 4) &&
         bwd_x3_bytes(a.Bp, a.F4) <= (size_t)dev_info().lds_max;
}

template <int TQ, int OM, bool TAIL>
static hipError_t bwd_x3_go_t(const BwdArgs& a, size_t lds, int64_t T, hipStream_t s) {
  return launch_persistent(k_bwd_x3<TQ, OM, 2, 512, TAIL>, 512, lds, T, s, a);
}

template <int OM>
static hipError_t bwd_x3_go_o(const BwdArgs& a, size_t lds, int64_t T, hipStream_t s) {
  const bool tail = a.F4 % 16 != 0;
  switch (a.F4 / 16) {
    case 2: return tail ? bwd_x3_go_t<2, OM, true>(a, lds, T, s) : bwd_x3_go_t<2, OM, false>(a, lds, T, s);
    case 3: return tail ? bwd_x3_go_t<3, OM, true>(a, lds, T, s) : bwd_x3_go_t<3, OM, false>(a, lds, T, s);
    case 4: return tail ? bwd_x3_go_t<4, OM, true>(a, lds, T, s) : bwd_x3_go_t<4, OM, false>(a, lds, T, s);
    case 5: return tail ? bwd_x3_go_t<5, OM, true>(a, lds, T, s) : bwd_x3_go_t<5, OM, false>(a, lds, T, s);
    case 6: return tail ? bwd_x3_go_t<6, OM, true>(a, lds, T, s) : bwd_x3_go_t<6, OM, false>(a, lds, T, s);
    case 7: return tail ? bwd_x3_go_t<7, OM, true>(a, lds, T, s) : bwd_x3_go_t<7, OM, false>(a, lds, T, s);
    default: return bwd_x3_go_t<8, OM, false>(a, lds, T, s);
  }
}

static hipError_t bwd_x3_go(const BwdArgs& a, hipStream_t s) {
  const int64_t T = (a.N + 15) / 16;
  const size_t lds = bwd_x3_bytes(a.Bp, a.F4);
  note_variant("k_bwd_x3", kArithX3);
  if (a.O == 4) return bwd_x3_go_o<4>(a, lds, T, s);
  return bwd_x3_go_o<2>(a, lds, T, s);
}

template <int TQ, int OM, bool TAIL = false>
static hipError_t bwd_lds_go(const BwdArgs& a, size_t lds, hipStream_t s) {
  // One 16-row tile per wave; 12 waves per workgroup (3 per SIMD) when the
  // per-chunk G buffers are small, 8 otherwise; prefetch depth set by the
  // size of those buffers.
  constexpr int RING = OM <= 2 && !TAIL ? 4 : (OM <= 4 ? 3 : 2);
  constexpr int NT = OM <= 2 && TQ <= 7 ? 768 : 512;
  const int64_t T = (a.N + 15) / 16;
  note_variant("k_bwd_lds", kArithFp32);
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
  if (bwd_x3_shape(a)) return bwd_x3_go(a, s);
  if (a.O == 2) return bwd_lds_by_f<2>(a, lds, s);
  if (a.O == 4) return bwd_lds_by_f<4>(a, lds, s);
  // O = 5 .. 16: the gather of G and the dW2 product on the matrix cores
  switch (bwd_tq(a.F4)) {
    case 1: return bwd_mf_go<1>(a, lds, s);
    case 2: return bwd_mf_go<2>(a, lds, s);
    case 4: return bwd_mf_go<4>(a, lds, s);
    case 7: return bwd_mf_go<7>(a, lds, s);
    default: return bwd_mf_go<8>(a, lds, s);
  }
}

}  // namespace pmlpk
