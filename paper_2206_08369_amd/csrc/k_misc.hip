// Initialisation, batch packing, fills, the loss and the hidden-layer view.

#include "device_common.h"

namespace pmlpk {

// ---------------------------------------------------------------------------
// Initialisation: U(-bound, bound) with bound = 1/sqrt(fan_in), from the
// counter-based draws of device_common.h.
// ---------------------------------------------------------------------------

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

__global__ __launch_bounds__(kBlock) void k_init_w2(float* __restrict__ W2, int64_t N,
                                                    int64_t ldw, int O,
                                                    const int32_t* __restrict__ mid,
                                                    const float* __restrict__ bound2,
                                                    uint64_t key) {
  const int64_t total = N * O;
  for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * kBlock) {
    const int64_t o = i / N;
    const int64_t n = i - o * N;
    W2[o * ldw + n] = uniform_weight(key, 2, (uint64_t)i, bound2[mid[n]]);  // counter o*N + n
  }
}

hipError_t launch_init_params(float* W1, int64_t N, int32_t F, int32_t F4, float bound1,
                              float* W2, int64_t ldw, int32_t O, const int32_t* mid,
                              const float* bound2, uint64_t key, hipStream_t s) {
  k_init_w1<<<grid_for(N * F4), kBlock, 0, s>>>(W1, N, F, F4, bound1, key);
  k_init_w2<<<grid_for(N * O), kBlock, 0, s>>>(W2, N, ldw, O, mid, bound2, key);
  return hipGetLastError();
}

hipError_t launch_init_w2(float* W2, int64_t N, int64_t ldw, int32_t O, const int32_t* mid,
                          const float* bound2, uint64_t key, hipStream_t s) {
  k_init_w2<<<grid_for(N * O), kBlock, 0, s>>>(W2, N, ldw, O, mid, bound2, key);
  return hipGetLastError();
}

__global__ __launch_bounds__(kBlock) void k_init_b(float* __restrict__ W1, int64_t N, int F4,
                                                   int bcol, float bound1,
                                                   float* __restrict__ b2, int M, int O,
                                                   const float* __restrict__ bound2,
                                                   uint64_t key) {
  const int64_t total = N + (int64_t)M * O;
  for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * kBlock) {
    if (i < N) {
      W1[i * F4 + bcol] = uniform_weight(key, 3, (uint64_t)i, bound1);
    } else {
      const int64_t j = i - N;  // counter m*O + o
      b2[j] = uniform_weight(key, 4, (uint64_t)j, bound2[j / O]);
    }
  }
}

hipError_t launch_init_biases(float* W1, int64_t N, int32_t F4, int32_t bcol, float bound1,
                              float* b2, int32_t M, int32_t O, const float* bound2,
                              uint64_t key, hipStream_t s) {
  k_init_b<<<grid_for(N + (int64_t)M * O), kBlock, 0, s>>>(W1, N, F4, bcol, bound1, b2, M, O,
                                                           bound2, key);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Batch packing: X [B][F] -> Xp [Bp][F4] and Xt [F4][Bp], zero padded.
// ---------------------------------------------------------------------------

__global__ __launch_bounds__(kBlock) void k_pack_x(const float* __restrict__ X, int B, int F,
                                                   int Bp, int F4, int bcol,
                                                   float* __restrict__ Xp,
                                                   float* __restrict__ Xt) {
  const int64_t total = (int64_t)Bp * F4;
  for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * kBlock) {
    const int b = (int)(i / F4);
    const int f = (int)(i - (int64_t)b * F4);
    const float v = b < B ? (f < F ? X[(int64_t)b * F + f] : (f == bcol ? 1.f : 0.f)) : 0.f;
    Xp[i] = v;
    Xt[(int64_t)f * Bp + b] = v;
  }
}

hipError_t launch_pack_x(const float* X, int32_t B, int32_t F, int32_t Bp, int32_t F4,
                         int32_t bcol, float* Xp, float* Xt, hipStream_t s) {
  note_variant("k_pack_x", kArithNone);
  k_pack_x<<<grid_for((int64_t)Bp * F4), kBlock, 0, s>>>(X, B, F, Bp, F4, bcol, Xp, Xt);
  return hipGetLastError();
}

// bf16 copies of the batch for the bf16-in GEMMs (nearest-even rounding,
// v_cvt_pk_bf16_f32); padding (b >= B, f >= F, and the row tails up to the
// 64-element stride) is zero.
__global__ __launch_bounds__(kBlock) void k_pack_x_bf16(const float* __restrict__ X, int B,
                                                        int F, int Bp, int F4, int bcol,
                                                        int ldp, int ldt,
                                                        unsigned short* __restrict__ Xp16,
                                                        unsigned short* __restrict__ Xt16) {
  const int64_t np = (int64_t)Bp * ldp, nt = (int64_t)F4 * ldt;
  for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < np + nt;
       i += (int64_t)gridDim.x * kBlock) {
    int b, f;
    if (i < np) {
      b = (int)(i / ldp);
      f = (int)(i - (int64_t)b * ldp);
    } else {
      f = (int)((i - np) / ldt);
      b = (int)(i - np - (int64_t)f * ldt);
    }
    const float v = (b < B && f < F4) ? (f < F ? X[(int64_t)b * F + f] : (f == bcol ? 1.f : 0.f))
                                      : 0.f;
    const unsigned short u = __builtin_bit_cast(unsigned short, (__bf16)v);
    if (i < np) Xp16[i] = u;
    else Xt16[i - np] = u;
  }
}

hipError_t launch_pack_x_bf16(const float* X, int32_t B, int32_t F, int32_t Bp, int32_t F4,
                              int32_t bcol, unsigned short* Xp16, unsigned short* Xt16,
                              hipStream_t s) {
  note_variant("k_pack_x_bf16", kArithNone);
  const int ldp = bf16_ld(F4), ldt = bf16_ld(Bp);
  k_pack_x_bf16<<<grid_for((int64_t)Bp * ldp + (int64_t)F4 * ldt), kBlock, 0, s>>>(
      X, B, F, Bp, F4, bcol, ldp, ldt, Xp16, Xt16);
  return hipGetLastError();
}

__global__ __launch_bounds__(kBlock) void k_w1_to_bf16(const float* __restrict__ W1,
                                                       int64_t total, int F4, int ldb,
                                                       unsigned short* __restrict__ W1b) {
  for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * kBlock) {
    const int64_t n = i / ldb;
    const int c = (int)(i - n * ldb);
    const float v = c < F4 ? W1[n * F4 + c] : 0.f;
    W1b[i] = __builtin_bit_cast(unsigned short, (__bf16)v);
  }
}

hipError_t launch_w1_to_bf16(const float* W1, int64_t Npad, int32_t F4, unsigned short* W1b,
                             int32_t ldb, hipStream_t s) {
  note_variant("k_w1_to_bf16", kArithNone);
  const int64_t total = Npad * ldb;
  k_w1_to_bf16<<<grid_for(total), kBlock, 0, s>>>(W1, total, F4, ldb, W1b);
  return hipGetLastError();
}

__global__ __launch_bounds__(kBlock) void k_fill(float* __restrict__ p, int64_t n, float v) {
  for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * kBlock)
    p[i] = v;
}

hipError_t launch_fill(float* p, int64_t n, float v, hipStream_t s) {
  note_variant("k_fill", kArithNone);
  if (n <= 0) return hipSuccess;
  k_fill<<<grid_for(n), kBlock, 0, s>>>(p, n, v);
  return hipGetLastError();
}

// Zero the weights of the input features a model does not see (run when
// the masks or the weights are set; the SGD steps then keep them at zero).
__global__ __launch_bounds__(kBlock) void k_apply_fmask(float* __restrict__ W1, int64_t total,
                                                        int F4, const int32_t* __restrict__ mid,
                                                        const uint32_t* __restrict__ fm,
                                                        int fmw) {
  for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * kBlock) {
    const int64_t n = i / F4;
    const int q = (int)(i - n * F4);
    if (!((fm[(int64_t)mid[n] * fmw + (q >> 5)] >> (q & 31)) & 1u)) W1[i] = 0.f;
  }
}

hipError_t launch_apply_fmask(float* W1, int64_t Npad, int32_t F4, const int32_t* mid,
                              const uint32_t* fmask, int32_t fmw, hipStream_t s) {
  const int64_t total = Npad * F4;
  if (total <= 0 || !fmask) return hipSuccess;
  k_apply_fmask<<<grid_for(total), kBlock, 0, s>>>(W1, total, F4, mid, fmask, fmw);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Per-model softmax cross-entropy, mean over the batch (the loss the
// packed training minimises; its sum over models has per-model gradients
// equal to each model's own).  One wave per model; in place:
//   LG[m][b][:] (logits) -> G = (softmax - onehot(y_b)) / B,  G = 0 for b >= B
//   loss[m] = mean_b (logsumexp - logit_y)
// A label outside [0, O) raises flag[0]; a non-finite per-model rate (lrm,
// may be null) raises flag[1]; every model whose loss is not finite adds one
// to flag[2].
// ---------------------------------------------------------------------------

template <int OM>
__global__ __launch_bounds__(kBlock) void k_ce(float* __restrict__ LG,
                                               const int32_t* __restrict__ y, int M, int Bp,
                                               int B, int O, float invB,
                                               float* __restrict__ loss,
                                               int32_t* __restrict__ flag,
                                               const float* __restrict__ lrm,
                                               float* __restrict__ b2, float* __restrict__ db2,
                                               float lr) {
  const int lane = threadIdx.x & 63;
  const int m = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (m >= M) return;
  if (lrm && lane == 0 && !isfinite(lrm[m])) flag[1] = 1;
  float part = 0.f;
  float gs[OM];  // this lane's share of db2 = sum_b G
#pragma unroll
  for (int o = 0; o < OM; ++o) gs[o] = 0.f;
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
        if (o < O) {
          const float g = (expf(l[o] - lse) - (o == yb ? 1.f : 0.f)) * invB;
          row[o] = g;
          gs[o] += g;
        }
    } else {
      for (int o = 0; o < O; ++o) row[o] = 0.f;
    }
  }
#pragma unroll
  for (int s = 32; s > 0; s >>= 1) part += __shfl_xor(part, s);
  if (lane == 0) {
    loss[m] = part * invB;
    if (!isfinite(part)) atomicAdd(flag + 2, 1);
  }
  if (b2) {
    const float rate = lrm ? lrm[m] : lr;
#pragma unroll
    for (int o = 0; o < OM; ++o) {
      float v = gs[o];
      for (int s = 32; s > 0; s >>= 1) v += __shfl_xor(v, s);
      if (lane == 0 && o < O) {
        if (db2) db2[(int64_t)m * O + o] = v;
        else b2[(int64_t)m * O + o] -= rate * v;
      }
    }
  }
}

hipError_t launch_ce(float* LG, const int32_t* y, int32_t M, int32_t Bp, int32_t B, int32_t O,
                     float* loss, int32_t* flag, const float* lrm, float* b2, float* db2,
                     float lr, hipStream_t s) {
  note_variant("k_ce", kArithNone);
  const unsigned blocks = (unsigned)((M + 3) / 4);
  const float invB = 1.0f / (float)B;
  if (O <= 2) k_ce<2><<<blocks, kBlock, 0, s>>>(LG, y, M, Bp, B, O, invB, loss, flag, lrm, b2, db2, lr);
  else if (O <= 4) k_ce<4><<<blocks, kBlock, 0, s>>>(LG, y, M, Bp, B, O, invB, loss, flag, lrm, b2, db2, lr);
  else if (O <= 8) k_ce<8><<<blocks, kBlock, 0, s>>>(LG, y, M, Bp, B, O, invB, loss, flag, lrm, b2, db2, lr);
  else k_ce<16><<<blocks, kBlock, 0, s>>>(LG, y, M, Bp, B, O, invB, loss, flag, lrm, b2, db2, lr);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Regression head: per-model mean squared error against real targets and
// its gradient, G = 2 (logit - Y) / (B O), in place over the logits; one
// wave per model, lanes over samples.
// ---------------------------------------------------------------------------

template <int OM>
__global__ __launch_bounds__(kBlock) void k_mse(float* __restrict__ LG,
                                                const float* __restrict__ Y, int M, int Bp,
                                                int B, int O, float inv,
                                                float* __restrict__ loss,
                                                int32_t* __restrict__ flag,
                                                const float* __restrict__ lrm,
                                                float* __restrict__ b2, float* __restrict__ db2,
                                                float lr) {
  const int lane = threadIdx.x & 63;
  const int m = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (m >= M) return;
  if (lrm && lane == 0 && !isfinite(lrm[m])) flag[1] = 1;
  float part = 0.f;
  float gs[OM];  // this lane's share of db2 = sum_b G
#pragma unroll
  for (int o = 0; o < OM; ++o) gs[o] = 0.f;
  for (int b = lane; b < Bp; b += 64) {
    float* row = LG + ((int64_t)m * Bp + b) * O;
    if (b < B) {
      const float* t = Y + (int64_t)b * O;
#pragma unroll
      for (int o = 0; o < OM; ++o)
        if (o < O) {
          const float d = row[o] - t[o];
          part = fmaf(d, d, part);
          const float g = 2.f * d * inv;
          row[o] = g;
          gs[o] += g;
        }
    } else {
      for (int o = 0; o < O; ++o) row[o] = 0.f;
    }
  }
#pragma unroll
  for (int s = 32; s > 0; s >>= 1) part += __shfl_xor(part, s);
  if (lane == 0) {
    loss[m] = part * inv;
    if (!isfinite(part)) atomicAdd(flag + 2, 1);
  }
  if (b2) {
    const float rate = lrm ? lrm[m] : lr;
#pragma unroll
    for (int o = 0; o < OM; ++o) {
      float v = gs[o];
      for (int s = 32; s > 0; s >>= 1) v += __shfl_xor(v, s);
      if (lane == 0 && o < O) {
        if (db2) db2[(int64_t)m * O + o] = v;
        else b2[(int64_t)m * O + o] -= rate * v;
      }
    }
  }
}

hipError_t launch_mse(float* LG, const float* Y, int32_t M, int32_t Bp, int32_t B, int32_t O,
                      float* loss, int32_t* flag, const float* lrm, float* b2, float* db2,
                      float lr, hipStream_t s) {
  note_variant("k_mse", kArithNone);
  const unsigned blocks = (unsigned)((M + 3) / 4);
  const float inv = 1.0f / ((float)B * (float)O);
  if (O <= 2) k_mse<2><<<blocks, kBlock, 0, s>>>(LG, Y, M, Bp, B, O, inv, loss, flag, lrm, b2, db2, lr);
  else if (O <= 4) k_mse<4><<<blocks, kBlock, 0, s>>>(LG, Y, M, Bp, B, O, inv, loss, flag, lrm, b2, db2, lr);
  else if (O <= 8) k_mse<8><<<blocks, kBlock, 0, s>>>(LG, Y, M, Bp, B, O, inv, loss, flag, lrm, b2, db2, lr);
  else k_mse<16><<<blocks, kBlock, 0, s>>>(LG, Y, M, Bp, B, O, inv, loss, flag, lrm, b2, db2, lr);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Hidden layer in the caller's [B][N] layout (inspection path).
// ---------------------------------------------------------------------------

__global__ __launch_bounds__(kBlock) void k_hidden_out(const float* __restrict__ Zt, bool zb, int Bp,
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
    const float z = load_z1(Zt, zb, n * Bp + b);
    if (Z) Z[i] = z;
    if (H) H[i] = act_fwd(act[mid[n]], z);
  }
}

hipError_t launch_hidden_out(const float* Zt, int32_t Bp, int32_t B, int64_t N,
                             const int32_t* mid, const int32_t* act, float* Z, float* H,
                             hipStream_t s, bool zb) {
  note_variant("k_hidden_out", kArithNone);
  k_hidden_out<<<grid_for((int64_t)B * N), kBlock, 0, s>>>(Zt, zb, Bp, B, N, mid, act, Z, H);
  return hipGetLastError();
}

}  // namespace pmlpk
