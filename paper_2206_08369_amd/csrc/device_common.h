// Device-side definitions shared by the HIP kernels of libpmlp (gfx950).
//
// Notation: N hidden units in total, M models, F inputs, O outputs, B
// samples in the batch, Bp = B rounded up to a multiple of 16.  Model m
// owns the contiguous hidden units [seg_off[m], seg_off[m+1]) and mid[n]
// is the model of hidden unit n (the Scatter Add index of Section 3,
// collapsed to one row).
//
// Device layouts (Npad = N rounded up to a multiple of 64; rows n >= N are
// padding that kernels may write but never read back into a result):
//   W1  [Npad][F4] fp32, F4 = F rounded up to 4, pad columns held at 0
//   W2  [O][Npad]  fp32 (row stride ldw = Npad)
//   Xp  [Bp][F4]   batch copy, zero padded          (operand of Z = X W1^T)
//   Xt  [F4][Bp]   transposed batch copy, zero padded (operand of dW1)
//   Zt  [Npad][Bp] hidden pre-activations, batch-minor: the Bp values of one
//                  hidden unit are contiguous.
//   LG  [M][Bp][O] per-model logits, overwritten in place by dLoss/dlogits.
// Zero padding of the batch (rows b >= B of Xp, columns b >= B of Xt, and
// G = 0 for b >= B) makes every padded lane contribute exactly nothing to
// the gradients, so no kernel needs the true B except the loss.

#pragma once

#include "pmlp_internal.h"

#include <math.h>

namespace pmlpk {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

constexpr int kBlock = 256;  // 4 waves of 64 lanes

inline int ceil_div_i(int64_t a, int64_t b) { return (int)((a + b - 1) / b); }

inline unsigned grid_for(int64_t n) {
  int64_t g = (n + kBlock - 1) / kBlock;
  if (g > 1048576) g = 1048576;
  if (g < 1) g = 1;
  return (unsigned)g;
}

// ---------------------------------------------------------------------------
// Counter-based draws for the initial weights: splitmix64 (Steele, Lea and
// Flood, OOPSLA 2014) of key ^ (tag << 60) ^ idx, whose top 24 bits give
// u in [0, 1); the weight is (2u - 1) * bound with one fp32 rounding.
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

// ---------------------------------------------------------------------------
// Per-model input feature masks (feature selection, Section 7): bit q of
// word fm[m * fmw + q / 32] is 1 when model m sees input column q (columns
// from F on, padding and the bias column, always 1).  A masked weight is
// held at zero by zeroing its gradient wherever the dW1 product is stored
// or applied, so Z = X W1^T needs no mask.  fm null: no masks.
// ---------------------------------------------------------------------------

// v with the entries of columns q .. q+3 (q a multiple of 4) that model m
// does not see set to zero.
__device__ __forceinline__ f32x4 fmask4(const uint32_t* __restrict__ fm, int fmw, int m, int q,
                                        f32x4 v) {
  if (!fm) return v;
  const uint32_t bits = fm[(int64_t)m * fmw + (q >> 5)] >> (q & 31);
  return f32x4{(bits & 1u) ? v[0] : 0.f, (bits & 2u) ? v[1] : 0.f, (bits & 4u) ? v[2] : 0.f,
               (bits & 8u) ? v[3] : 0.f};
}

// ---------------------------------------------------------------------------
// Activations (Section 3, last paragraph: one activation per contiguous
// portion of the hidden layer; the list of Section 4.2).  Ids as in
// include/pmlp.h.
// ---------------------------------------------------------------------------

// The transcendental pieces use the hardware approximations (v_exp_f32 on
// x*log2(e), v_log_f32, v_rcp_f32; about 1 ulp each), which keeps the
// per-element cost of the activation far below the memory time of the
// kernels that apply it.  Absolute errors stay near 1e-7 for the values
// these networks see, well inside the per-model normwise tolerance.

__device__ __forceinline__ float fexp(float x) { return __expf(x); }
__device__ __forceinline__ float frcp(float x) { return __builtin_amdgcn_rcpf(x); }
__device__ __forceinline__ float flog(float x) { return __logf(x); }

__device__ __forceinline__ float logistic(float z) { return frcp(1.0f + fexp(-z)); }

// Normal CDF and density for GELU.  Phi(-|z|) = erfc(|z|/sqrt 2)/2 with
// erfc from the rational approximation 7.1.26 of Abramowitz and Stegun
// (Handbook of Mathematical Functions, 1964):
//   erfc(x) = (a1 t + a2 t^2 + a3 t^3 + a4 t^4 + a5 t^5) exp(-x^2),
//   t = 1 / (1 + p x), x >= 0, absolute error at most 1.5e-7,
// whose factor exp(-x^2) = exp(-z^2/2) is also the density's.  About a
// third of the instructions of the library erfc, in a kernel where every
// VALU instruction competes with the matrix instructions for issue.
__device__ __forceinline__ float normal_cdf_pdf(float z, float* pdf) {
  const float x = fabsf(z) * 0.70710678118654752f;
  const float t = frcp(fmaf(0.3275911f, x, 1.0f));
  float q = fmaf(1.061405429f, t, -1.453152027f);
  q = fmaf(q, t, 1.421413741f);
  q = fmaf(q, t, -0.284496736f);
  q = fmaf(q, t, 0.254829592f);
  const float e = fexp(-x * x);
  const float lower = 0.5f * (q * t) * e;  // Phi(-|z|)
  *pdf = 0.39894228040143268f * e;
  return z < 0.f ? lower : 1.0f - lower;
}

// SELU constants (Klambauer et al., 2017)
constexpr float kSeluAlpha = 1.6732632423543772f;
constexpr float kSeluLambda = 1.0507009873554805f;

// Mish: tanh(softplus z) = n / (n + 2) with n = e^z (e^z + 2), free of
// cancellation for z << 0; 1 (to fp32) above 20.
__device__ __forceinline__ float mish_t(float z, float* u_out) {
  if (z > 20.f) { *u_out = 0.f; return 1.f; }
  const float u = fexp(z);
  const float n = u * (u + 2.f);
  *u_out = u;
  return n * frcp(n + 2.f);
}

// Z of the hidden layer as stored: fp32, or (zb, the bf16 storage mode)
// the bfloat16 bit patterns in the first half of the same buffer, widened
// exactly to fp32.  idx is an element index of the [Npad][Bp] layout.
__device__ __forceinline__ float bf16_bits_to_f32(uint32_t b16) {
  return __uint_as_float(b16 << 16);
}
__device__ __forceinline__ f32x4 load_z4(const float* Zt, bool zb, int64_t idx) {
  if (zb) {
    const uint2 v = *(const uint2*)((const unsigned short*)Zt + idx);
    return f32x4{__uint_as_float(v.x << 16), __uint_as_float(v.x & 0xFFFF0000u),
                 __uint_as_float(v.y << 16), __uint_as_float(v.y & 0xFFFF0000u)};
  }
  return *(const f32x4*)(Zt + idx);
}
__device__ __forceinline__ f32x2 load_z2(const float* Zt, bool zb, int64_t idx) {
  if (zb) {
    const uint32_t v = *(const uint32_t*)((const unsigned short*)Zt + idx);
    return f32x2{__uint_as_float(v << 16), __uint_as_float(v & 0xFFFF0000u)};
  }
  return *(const f32x2*)(Zt + idx);
}
__device__ __forceinline__ float load_z1(const float* Zt, bool zb, int64_t idx) {
  return zb ? bf16_bits_to_f32(((const unsigned short*)Zt)[idx]) : Zt[idx];
}

__device__ __forceinline__ float act_fwd(int a, float z) {
  switch (a) {
    case 0: return z;
    case 1: return z > 0.f ? z : 0.f;
    case 2: return 1.f - 2.f * frcp(1.f + fexp(2.f * z));  // tanh
    case 3: return logistic(z);
    case 4: return z > 0.f ? z : fexp(z) - 1.f;
    case 5: return z > 0.f ? z : 0.01f * z;
    case 6: { float pdf; return z * normal_cdf_pdf(z, &pdf); }
    case 7: return z * logistic(z);
    case 8: return z > 20.f ? z : fmaxf(z, 0.f) + flog(1.f + fexp(-fabsf(z)));
    case 9: return z * logistic(2.f * z);
    case 10: return z > 0.f ? kSeluLambda * z : (kSeluLambda * kSeluAlpha) * (fexp(z) - 1.f);
    case 11: return (z > 0.5f || z < -0.5f) ? z : 0.f;
    case 12: { float u; return z * mish_t(z, &u); }
    default: return 0.f;
  }
}

// Value and derivative together.
__device__ __forceinline__ float act_fwd_bwd(int a, float z, float* d) {
  switch (a) {
    case 0: *d = 1.f; return z;
    case 1: *d = z > 0.f ? 1.f : 0.f; return z > 0.f ? z : 0.f;
    case 2: {
      const float t = 1.f - 2.f * frcp(1.f + fexp(2.f * z));
      *d = 1.f - t * t;
      return t;
    }
    case 3: { const float s = logistic(z); *d = s * (1.f - s); return s; }
    case 4: {
      if (z > 0.f) { *d = 1.f; return z; }
      const float e = fexp(z);
      *d = e;
      return e - 1.f;
    }
    case 5: *d = z > 0.f ? 1.f : 0.01f; return z > 0.f ? z : 0.01f * z;
    case 6: {
      float pdf;
      const float cdf = normal_cdf_pdf(z, &pdf);
      *d = cdf + z * pdf;
      return z * cdf;
    }
    case 7: { const float s = logistic(z); *d = s + z * s * (1.f - s); return z * s; }
    case 8: {
      if (z > 20.f) { *d = 1.f; return z; }
      *d = logistic(z);
      return fmaxf(z, 0.f) + flog(1.f + fexp(-fabsf(z)));
    }
    case 9: {
      const float s = logistic(2.f * z);
      *d = s + 2.f * z * s * (1.f - s);
      return z * s;
    }
    case 10: {
      if (z > 0.f) { *d = kSeluLambda; return kSeluLambda * z; }
      const float e = (kSeluLambda * kSeluAlpha) * fexp(z);
      *d = e;
      return e - kSeluLambda * kSeluAlpha;
    }
    case 11: {
      const bool on = z > 0.5f || z < -0.5f;
      *d = on ? 1.f : 0.f;
      return on ? z : 0.f;
    }
    case 12: {
      float u;
      const float t = mish_t(z, &u);
      const float s = z > 20.f ? 1.f : u * frcp(1.f + u);
      *d = t + z * (1.f - t * t) * s;
      return z * t;
    }
    default: *d = 0.f; return 0.f;
  }
}

// ---------------------------------------------------------------------------
// Lane-group sums with DPP (register-only cross-lane moves).  A Hillis-Steele
// scan with row shifts 1, 2, 4, 8 (zero fill outside the 16-lane row) and
// the row broadcasts 15 and 31 leaves in the last lane of every aligned
// group of LG lanes (LG a power of two up to 64) the sum over that group.
// Each step only reads lanes inside the window that ends at a group's last
// lane, so groups that are inactive do not affect active ones.
// ---------------------------------------------------------------------------

template <int CTRL, int ROWMASK>
__device__ __forceinline__ float dpp_add(float v) {
  const int moved = __builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, ROWMASK, 0xf, true);
  return v + __int_as_float(moved);
}

__device__ __forceinline__ float group_sum_to_last(float v, int LG) {
  if (LG > 1) v = dpp_add<0x111, 0xf>(v);   // row_shr:1
  if (LG > 2) v = dpp_add<0x112, 0xf>(v);   // row_shr:2
  if (LG > 4) v = dpp_add<0x114, 0xf>(v);   // row_shr:4
  if (LG > 8) v = dpp_add<0x118, 0xf>(v);   // row_shr:8
  if (LG > 16) v = dpp_add<0x142, 0xa>(v);  // row_bcast:15 into rows 1 and 3
  if (LG > 32) v = dpp_add<0x143, 0xc>(v);  // row_bcast:31 into rows 2 and 3
  return v;
}

}  // namespace pmlpk
