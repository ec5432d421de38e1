// HIP kernels for packed ParallelMLPs training on gfx950 (MI355X).
//
// Notation: N hidden units in total, M models, F inputs, O outputs, B
// samples in the batch, Bp = B rounded up to a multiple of 16.  Model m
// owns the contiguous hidden units [seg_off[m], seg_off[m+1]) and mid[n]
// is the model of hidden unit n (the Scatter Add index of Section 3,
// collapsed to one row).
//
// Device layouts:
//   W1  [N][F4]   fp32, F4 = F rounded up to 4, pad columns held at 0
//   W2  [O][N]    fp32
//   Xp  [Bp][F4]  batch copy, zero padded          (operand of Z = X W1^T)
//   Xt  [F4][Bp]  transposed batch copy, zero padded (operand of dW1)
//   Zt  [N][Bp]   hidden pre-activations, batch-minor: the Bp values of one
//                 hidden unit are contiguous.  Overwritten in place by dZ.
//   LG  [M][Bp][O] per-model logits, overwritten in place by dLoss/dlogits.
// Zero padding of the batch (rows b >= B of Xp, columns b >= B of Xt, and
// G = 0 for b >= B) makes every padded lane contribute exactly nothing to
// the gradients, so no kernel needs the true B except the loss.

#include "pmlp_internal.h"

#include <math.h>

namespace pmlpk {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

static constexpr int kBlock = 256;  // 4 waves of 64 lanes

static inline int ceil_div_i(int64_t a, int64_t b) { return (int)((a + b - 1) / b); }

static inline unsigned grid_for(int64_t n) {
  int64_t g = (n + kBlock - 1) / kBlock;
  if (g > 1048576) g = 1048576;
  if (g < 1) g = 1;
  return (unsigned)g;
}

// ---------------------------------------------------------------------------
// Activations (Section 3, last paragraph: one activation per contiguous
// portion of the hidden layer).  Ids as in include/pmlp.h.
// ---------------------------------------------------------------------------

__device__ __forceinline__ float logistic(float z) { return 1.0f / (1.0f + expf(-z)); }

__device__ __forceinline__ float act_fwd(int a, float z) {
  switch (a) {
    case 0: return z;
    case 1: return z > 0.f ? z : 0.f;
    case 2: return tanhf(z);
    case 3: return logistic(z);
    case 4: return z > 0.f ? z : expm1f(z);
    case 5: return z > 0.f ? z : 0.01f * z;
    case 6: return z * (0.5f * erfcf(-z * 0.70710678118654752f));
    case 7: return z * logistic(z);
    case 8: return z > 20.f ? z : fmaxf(z, 0.f) + log1pf(expf(-fabsf(z)));
    case 9: return z * logistic(2.f * z);
    default: return 0.f;
  }
}

// Value and derivative together.
__device__ __forceinline__ float act_fwd_bwd(int a, float z, float* d) {
  switch (a) {
    case 0: *d = 1.f; return z;
    case 1: *d = z > 0.f ? 1.f : 0.f; return z > 0.f ? z : 0.f;
    case 2: { float t = tanhf(z); *d = 1.f - t * t; return t; }
    case 3: { float s = logistic(z); *d = s * (1.f - s); return s; }
    case 4: {
      if (z > 0.f) { *d = 1.f; return z; }
      *d = expf(z);
      return expm1f(z);
    }
    case 5: *d = z > 0.f ? 1.f : 0.01f; return z > 0.f ? z : 0.01f * z;
    case 6: {
      float cdf = 0.5f * erfcf(-z * 0.70710678118654752f);
      float pdf = 0.39894228040143268f * expf(-0.5f * z * z);
      *d = cdf + z * pdf;
      return z * cdf;
    }
    case 7: { float s = logistic(z); *d = s + z * s * (1.f - s); return z * s; }
    case 8: {
      if (z > 20.f) { *d = 1.f; return z; }
      *d = logistic(z);
      return fmaxf(z, 0.f) + log1pf(expf(-fabsf(z)));
    }
    case 9: { float s = logistic(2.f * z); *d = s + 2.f * z * s * (1.f - s); return z * s; }
    default: *d = 0.f; return 0.f;
  }
}

// ---------------------------------------------------------------------------
// Initialisation: counter-based splitmix64 draws (Steele, Lea and Flood,
// OOPSLA 2014), U(-bound, bound) with bound = 1/sqrt(fan_in).
// ---------------------------------------------------------------------------

__device__ __forceinline__ uint64_t splitmix64(uint64_t x) {
  uint64_t z = x + 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

__device__ __forceinline__ float uniform_weight(uint64_t key, uint64_t tag, uint64_t idx,
                                                float bound) {
  const uint64_t r = splitmix64(key ^ (tag << 60) ^ idx);
  const int32_t k = (int32_t)(r >> 40);                             // 24 random bits
  const float c = (float)(2 * k - 16777216) * 5.9604644775390625e-08f;  // exact: (2u - 1)
  return c * bound;                                                // one rounding
}

__global__ __launch_bounds__(kBlock) void k_init_w1(float* __restrict__ W1, int64_t N, int F,
                                                    int F4, float bound, uint64_t key) {
  const int64_t total = N * F4;
  for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * kBlock) {
    const int64_t n = i / F4;
    const int f = (int)(i - n * F4);
    W1[i] = f < F ? uniform_weight(key, 1, (uint64_t)(n * F + f), bound) : 0.f;
  }
}

__global__ __launch_bounds__(kBlock) void k_init_w2(float* __restrict__ W2, int64_t N, int O,
                                                    const int32_t* __restrict__ mid,
                                                    const float* __restrict__ bound2,
                                                    uint64_t key) {
  const int64_t total = N * O;
  for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * kBlock) {
    const int64_t n = i % N;
    W2[i] = uniform_weight(key, 2, (uint64_t)i, bound2[mid[n]]);
  }
}

hipError_t launch_init_params(float* W1, int64_t N, int32_t F, int32_t F4, float bound1,
                              float* W2, int32_t O, const int32_t* mid, const float* bound2,
                              uint64_t key, hipStream_t s) {
  k_init_w1<<<grid_for(N * F4), kBlock, 0, s>>>(W1, N, F, F4, bound1, key);
  k_init_w2<<<grid_for(N * O), kBlock, 0, s>>>(W2, N, O, mid, bound2, key);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Batch packing: X [B][F] -> Xp [Bp][F4] and Xt [F4][Bp], zero padded.
// ---------------------------------------------------------------------------

__global__ __launch_bounds__(kBlock) void k_pack_x(const float* __restrict__ X, int B, int F,
                                                   int Bp, int F4, float* __restrict__ Xp,
                                                   float* __restrict__ Xt) {
  const int64_t total = (int64_t)Bp * F4;
  for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * kBlock) {
    const int b = (int)(i / F4);
    const int f = (int)(i - (int64_t)b * F4);
    const float v = (b < B && f < F) ? X[(int64_t)b * F + f] : 0.f;
    Xp[i] = v;
    Xt[(int64_t)f * Bp + b] = v;
  }
}

hipError_t launch_pack_x(const float* X, int32_t B, int32_t F, int32_t Bp, int32_t F4,
                         float* Xp, float* Xt, hipStream_t s) {
  k_pack_x<<<grid_for((int64_t)Bp * F4), kBlock, 0, s>>>(X, B, F, Bp, F4, Xp, Xt);
  return hipGetLastError();
}

__global__ __launch_bounds__(kBlock) void k_fill(float* __restrict__ p, int64_t n, float v) {
  for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * kBlock)
    p[i] = v;
}

hipError_t launch_fill(float* p, int64_t n, float v, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  k_fill<<<grid_for(n), kBlock, 0, s>>>(p, n, v);
  return hipGetLastError();
}

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

  const int K = a.K;
  const int K16 = K & ~15;
  if (K16 > 0) {
    f32x4 cq[TQ], cp[TP];
    load_chunk<TQ, TP>(cq, cp, qrow, prow, 4 * lk);
    for (int k = 16; k < K16; k += 16) {
      f32x4 nq[TQ], np[TP];
      load_chunk<TQ, TP>(nq, np, qrow, prow, k + 4 * lk);
      mma_chunk<TQ, TP>(acc, cq, cp);
#pragma unroll
      for (int t = 0; t < TQ; ++t) cq[t] = nq[t];
#pragma unroll
      for (int t = 0; t < TP; ++t) cp[t] = np[t];
    }
    mma_chunk<TQ, TP>(acc, cq, cp);
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
#pragma unroll
    for (int i = 0; i < TQ; ++i) {
      const int q = q0 + 16 * i + 4 * lk;
      if (q >= a.NQ) continue;
      if (EPI == EPI_STORE) {
        *(f32x4*)(orow + q) = acc[i][j];
      } else if (EPI == EPI_SGD) {
        f32x4 w = *(f32x4*)(orow + q);
        w -= a.lr * acc[i][j];
        *(f32x4*)(orow + q) = w;
      } else {
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (q + r < a.ncols) orow[q + r] = acc[i][j][r];
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
  if (a.NP <= 0 || a.NQ <= 0) return hipSuccess;
  if (a.NQ <= 16) gemm_dispatch<1, 8>(a, epi, 1, s);
  else if (a.NQ <= 32) gemm_dispatch<2, 8>(a, epi, 1, s);
  else if (a.NQ <= 64) gemm_dispatch<4, 4>(a, epi, 1, s);
  else if (a.NQ <= 112) gemm_dispatch<7, 2>(a, epi, 1, s);
  else if (a.NQ <= 128) gemm_dispatch<4, 4>(a, epi, 2, s);
  else gemm_dispatch<4, 4>(a, epi, 4, s);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// M3 forward (Section 3, steps 3-4 of the packed procedure): the product of
// the hidden activations with W2 followed by the scatter-add over each
// model's hidden units, fused so that the [B, O, N] product is never
// stored:
//   out[m, b, o] = sum_{n in tile, n in model m} act_m(Zt[n][b]) * W2[o][n]
//
// One wave per (tile, block of BW samples).  Lane l handles the four
// samples b = 4*(l % LG) .. +3 (LG = BW/4 lanes per hidden unit) and
// hidden units n = first + l/LG, stepping by NG = 64/LG; all groups stay
// inside one segment at a time, so the activation id is wave-uniform and
// the running sums never mix models.  At the end of a segment the NG
// groups' partial sums are combined with lane shuffles and written once
// (plain store); the two halves of a segment wider than the tile limit are
// added with atomics onto zeroed logits instead (two additions onto zero
// are order-independent, so the result is still deterministic).
// ---------------------------------------------------------------------------

template <int OM>
__global__ __launch_bounds__(kBlock) void k_m3_fwd(
    const float* __restrict__ Zt, int Bp, int B, const float* __restrict__ W2, int64_t N, int O,
    const int64_t* __restrict__ seg_off, const int32_t* __restrict__ act,
    const Tile3* __restrict__ tiles, int ntiles, int BW, int LG, int nbblk,
    float* __restrict__ out, int64_t sm, int64_t sb) {
  const int lane = threadIdx.x & 63;
  const int wv = __builtin_amdgcn_readfirstlane((int)(blockIdx.x * 4 + (threadIdx.x >> 6)));
  const int tile = wv / nbblk;
  const int bblk = wv - tile * nbblk;
  if (tile >= ntiles) return;
  const int NG = 64 / LG;
  const int g = lane / LG;
  const int pp = lane - g * LG;
  const int b = bblk * BW + 4 * pp;
  const bool bvalid = b < Bp;
  const Tile3 t = tiles[tile];
  const int64_t nend = t.n0 + t.len;
  int64_t n = t.n0;
  int m = t.m0;
  while (n < nend) {
    int64_t se = seg_off[m + 1];
    if (se > nend) se = nend;
    const int a = act[m];
    float acc[4][OM];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int o = 0; o < OM; ++o) acc[i][o] = 0.f;
#pragma unroll 2
    for (int64_t nn = n + g; nn < se; nn += NG) {
      f32x4 z = {0.f, 0.f, 0.f, 0.f};
      if (bvalid) z = *(const f32x4*)(Zt + nn * Bp + b);
      float w[OM];
#pragma unroll
      for (int o = 0; o < OM; ++o) w[o] = (o < O) ? W2[(int64_t)o * N + nn] : 0.f;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float h = act_fwd(a, z[i]);
#pragma unroll
        for (int o = 0; o < OM; ++o) acc[i][o] = fmaf(h, w[o], acc[i][o]);
      }
    }
    for (int s = LG; s < 64; s <<= 1)
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int o = 0; o < OM; ++o) acc[i][o] += __shfl_xor(acc[i][o], s);
    if (g == 0 && bvalid) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        if (b + i >= B) continue;
        float* dst = out + (int64_t)m * sm + (int64_t)(b + i) * sb;
#pragma unroll
        for (int o = 0; o < OM; ++o) {
          if (o >= O) continue;
          if (t.atomic) unsafeAtomicAdd(dst + o, acc[i][o]);
          else dst[o] = acc[i][o];
        }
      }
    }
    n = se;
    ++m;
  }
}

template <int OM>
static void m3_fwd_dispatch(const float* Zt, int32_t Bp, int32_t B, const float* W2, int64_t N,
                            int32_t O, const int64_t* seg_off, const int32_t* act,
                            const Tile3* tiles, int32_t ntiles, float* out, int64_t sm,
                            int64_t sb, hipStream_t s) {
  int BW = 64;
  if (Bp < 64) BW = Bp <= 16 ? 16 : (Bp <= 32 ? 32 : 64);
  const int LG = BW / 4;
  const int nbblk = ceil_div_i(Bp, BW);
  const int64_t waves = (int64_t)ntiles * nbblk;
  const unsigned blocks = (unsigned)((waves + 3) / 4);
  k_m3_fwd<OM><<<blocks, kBlock, 0, s>>>(Zt, Bp, B, W2, N, O, seg_off, act, tiles, ntiles, BW,
                                         LG, nbblk, out, sm, sb);
}

hipError_t launch_m3_fwd(const float* Zt, int32_t Bp, int32_t B, const float* W2, int64_t N,
                         int32_t O, const int64_t* seg_off, const int32_t* act,
                         const Tile3* tiles, int32_t ntiles, float* out, int64_t sm,
                         int64_t sb, hipStream_t s) {
  if (ntiles <= 0) return hipSuccess;
  if (O <= 2) m3_fwd_dispatch<2>(Zt, Bp, B, W2, N, O, seg_off, act, tiles, ntiles, out, sm, sb, s);
  else if (O <= 4) m3_fwd_dispatch<4>(Zt, Bp, B, W2, N, O, seg_off, act, tiles, ntiles, out, sm, sb, s);
  else if (O <= 8) m3_fwd_dispatch<8>(Zt, Bp, B, W2, N, O, seg_off, act, tiles, ntiles, out, sm, sb, s);
  else m3_fwd_dispatch<16>(Zt, Bp, B, W2, N, O, seg_off, act, tiles, ntiles, out, sm, sb, s);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Per-model softmax cross-entropy, mean over the batch (the loss the
// packed training minimises; its sum over models has per-model gradients
// equal to each model's own).  One wave per model; in place:
//   LG[m][b][:] (logits) -> G = (softmax - onehot(y_b)) / B,  G = 0 for b >= B
//   loss[m] = mean_b (logsumexp - logit_y)
// A label outside [0, O) raises *flag.
// ---------------------------------------------------------------------------

template <int OM>
__global__ __launch_bounds__(kBlock) void k_ce(float* __restrict__ LG,
                                               const int32_t* __restrict__ y, int M, int Bp,
                                               int B, int O, float invB,
                                               float* __restrict__ loss,
                                               int32_t* __restrict__ flag) {
  const int lane = threadIdx.x & 63;
  const int m = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (m >= M) return;
  float part = 0.f;
  for (int b = lane; b < Bp; b += 64) {
    float* row = LG + ((int64_t)m * Bp + b) * O;
    if (b < B) {
      float l[OM];
      float mx = -INFINITY;
#pragma unroll
      for (int o = 0; o < OM; ++o) {
        l[o] = o < O ? row[o] : -INFINITY;
        mx = fmaxf(mx, l[o]);
      }
      float se = 0.f;
#pragma unroll
      for (int o = 0; o < OM; ++o)
        if (o < O) se += expf(l[o] - mx);
      const float lse = mx + logf(se);
      const int yb = y[b];
      if (yb < 0 || yb >= O) flag[0] = 1;
      float ly = 0.f;
#pragma unroll
      for (int o = 0; o < OM; ++o)
        if (o == yb) ly = l[o];
      part += lse - ly;
#pragma unroll
      for (int o = 0; o < OM; ++o)
        if (o < O) row[o] = (expf(l[o] - lse) - (o == yb ? 1.f : 0.f)) * invB;
    } else {
      for (int o = 0; o < O; ++o) row[o] = 0.f;
    }
  }
#pragma unroll
  for (int s = 32; s > 0; s >>= 1) part += __shfl_xor(part, s);
  if (lane == 0) loss[m] = part * invB;
}

hipError_t launch_ce(float* LG, const int32_t* y, int32_t M, int32_t Bp, int32_t B, int32_t O,
                     float* loss, int32_t* flag, hipStream_t s) {
  const unsigned blocks = (unsigned)((M + 3) / 4);
  const float invB = 1.0f / (float)B;
  if (O <= 2) k_ce<2><<<blocks, kBlock, 0, s>>>(LG, y, M, Bp, B, O, invB, loss, flag);
  else if (O <= 4) k_ce<4><<<blocks, kBlock, 0, s>>>(LG, y, M, Bp, B, O, invB, loss, flag);
  else if (O <= 8) k_ce<8><<<blocks, kBlock, 0, s>>>(LG, y, M, Bp, B, O, invB, loss, flag);
  else k_ce<16><<<blocks, kBlock, 0, s>>>(LG, y, M, Bp, B, O, invB, loss, flag);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// M3 backward + activation derivative + W2 update.  The gradient of the
// scatter-add is a gather by model id (each hidden unit only ever sees its
// own model's output gradient, Section 3):
//   dH[b][n] = sum_o G[mid[n]][b][o] * W2[o][n]          (W2 before update)
//   dZ[b][n] = dH[b][n] * act'(Z[b][n])                  (in place over Zt)
//   dW2[o][n] = sum_b G[mid[n]][b][o] * act(Z[b][n])
//   W2[o][n] -= lr * dW2[o][n]        (or dW2 stored, gradient mode)
// One wave per run of T5 consecutive hidden units; lanes as in the forward
// (groups of LG lanes per hidden unit, four samples per lane), with
// `slots` passes when the batch is wider than 256.  Per-unit dW2 partial
// sums are reduced across the group with shuffles and accumulated in LDS.
// ---------------------------------------------------------------------------

static constexpr int kT5 = 256;

template <int OM, bool GRAD>
__global__ __launch_bounds__(kBlock) void k_m3_bwd(
    float* __restrict__ Zt, int Bp, float* __restrict__ W2, int64_t N, int O,
    const int32_t* __restrict__ mid, const int32_t* __restrict__ act,
    const float* __restrict__ G, int LG, int slots, float lr, float* __restrict__ dW2) {
  __shared__ float lds[4 * kT5 * OM];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  float* dwl = lds + wave * kT5 * OM;
  const int64_t r0 = ((int64_t)blockIdx.x * 4 + wave) * kT5;
  int64_t r1 = r0 + kT5;
  if (r1 > N) r1 = N;
  const int NG = 64 / LG;
  const int g = lane / LG;
  const int pp = lane - g * LG;
  for (int slot = 0; slot < slots; ++slot) {
    const int b = slot * 4 * LG + 4 * pp;
    const bool bvalid = b < Bp;
    int cur_m = -1, a = 0;
    float gr[4][OM];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int o = 0; o < OM; ++o) gr[i][o] = 0.f;
    for (int64_t n = r0 + g; n < r1; n += NG) {
      const int m = mid[n];
      if (m != cur_m) {
        cur_m = m;
        a = act[m];
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int o = 0; o < OM; ++o)
            gr[i][o] = (bvalid && o < O) ? G[((int64_t)m * Bp + b + i) * O + o] : 0.f;
      }
      float w[OM];
#pragma unroll
      for (int o = 0; o < OM; ++o) w[o] = (o < O) ? W2[(int64_t)o * N + n] : 0.f;
      f32x4 z = {0.f, 0.f, 0.f, 0.f};
      if (bvalid) z = *(const f32x4*)(Zt + n * Bp + b);
      float dw[OM];
#pragma unroll
      for (int o = 0; o < OM; ++o) dw[o] = 0.f;
      f32x4 dz;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float hp;
        const float h = act_fwd_bwd(a, z[i], &hp);
        float dh = 0.f;
#pragma unroll
        for (int o = 0; o < OM; ++o) dh = fmaf(gr[i][o], w[o], dh);
        dz[i] = dh * hp;
#pragma unroll
        for (int o = 0; o < OM; ++o) dw[o] = fmaf(gr[i][o], h, dw[o]);
      }
      if (bvalid) *(f32x4*)(Zt + n * Bp + b) = dz;
      for (int s = 1; s < LG; s <<= 1)
#pragma unroll
        for (int o = 0; o < OM; ++o) dw[o] += __shfl_xor(dw[o], s);
      if (pp == 0) {
        float* d = dwl + (n - r0) * OM;
#pragma unroll
        for (int o = 0; o < OM; ++o)
          if (o < O) d[o] = slot == 0 ? dw[o] : d[o] + dw[o];
      }
    }
  }
  __syncthreads();
  const int64_t cnt = r1 > r0 ? (r1 - r0) * O : 0;
  for (int64_t idx = lane; idx < cnt; idx += 64) {
    const int64_t nl = idx / O;
    const int o = (int)(idx - nl * O);
    const int64_t n = r0 + nl;
    const float d = dwl[nl * OM + o];
    if (GRAD) dW2[(int64_t)o * N + n] = d;
    else W2[(int64_t)o * N + n] -= lr * d;
  }
}

template <int OM>
static void m3_bwd_dispatch(float* Zt, int32_t Bp, float* W2, int64_t N, int32_t O,
                            const int32_t* mid, const int32_t* act, const float* G, float lr,
                            float* dW2, hipStream_t s) {
  int LG = 64;
  const int q = (Bp + 3) / 4;
  if (q < 64) {
    LG = 1;
    while (LG < q) LG <<= 1;
  }
  const int slots = ceil_div_i(Bp, 4 * LG);
  const int64_t waves = (N + kT5 - 1) / kT5;
  const unsigned blocks = (unsigned)((waves + 3) / 4);
  if (dW2)
    k_m3_bwd<OM, true><<<blocks, kBlock, 0, s>>>(Zt, Bp, W2, N, O, mid, act, G, LG, slots, lr, dW2);
  else
    k_m3_bwd<OM, false><<<blocks, kBlock, 0, s>>>(Zt, Bp, W2, N, O, mid, act, G, LG, slots, lr, dW2);
}

hipError_t launch_m3_bwd(float* Zt, int32_t Bp, float* W2, int64_t N, int32_t O,
                         const int32_t* mid, const int32_t* act, const float* G, float lr,
                         float* dW2, hipStream_t s) {
  if (O <= 2) m3_bwd_dispatch<2>(Zt, Bp, W2, N, O, mid, act, G, lr, dW2, s);
  else if (O <= 4) m3_bwd_dispatch<4>(Zt, Bp, W2, N, O, mid, act, G, lr, dW2, s);
  else if (O <= 8) m3_bwd_dispatch<8>(Zt, Bp, W2, N, O, mid, act, G, lr, dW2, s);
  else m3_bwd_dispatch<16>(Zt, Bp, W2, N, O, mid, act, G, lr, dW2, s);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Hidden layer in the caller's [B][N] layout (inspection path).
// ---------------------------------------------------------------------------

__global__ __launch_bounds__(kBlock) void k_hidden_out(const float* __restrict__ Zt, int Bp,
                                                       int B, int64_t N,
                                                       const int32_t* __restrict__ mid,
                                                       const int32_t* __restrict__ act,
                                                       float* __restrict__ Z,
                                                       float* __restrict__ H) {
  const int64_t total = (int64_t)B * N;
  for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * kBlock) {
    const int64_t b = i / N;
    const int64_t n = i - b * N;
    const float z = Zt[n * Bp + b];
    if (Z) Z[i] = z;
    if (H) H[i] = act_fwd(act[mid[n]], z);
  }
}

hipError_t launch_hidden_out(const float* Zt, int32_t Bp, int32_t B, int64_t N,
                             const int32_t* mid, const int32_t* act, float* Z, float* H,
                             hipStream_t s) {
  k_hidden_out<<<grid_for((int64_t)B * N), kBlock, 0, s>>>(Zt, Bp, B, N, mid, act, Z, H);
  return hipGetLastError();
}

}  // namespace pmlpk
