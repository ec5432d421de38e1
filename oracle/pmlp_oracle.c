/*
 * pmlp_oracle.c -- plain, slow, fp64 CPU oracle for ParallelMLPs training.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library calls, links or
 * includes this file; only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg load it.  It shares no code, header, table or
 * constant with the HIP implementation.
 *
 * What it computes (Farias, Ludermir, Bastos-Filho, "Embarrassingly Parallel
 * Independent Training of Multi-Layer Perceptrons with Heterogeneous
 * Architectures", 2022):
 *
 *   The packed method (Section 3, the four-step summary after the Scatter Add
 *   example) is built so that the per-model gradient paths never mix and every
 *   internal MLP trains exactly as it would alone (Section 3, the paragraph on
 *   the Scatter Add keeping gradients separate).  The plain definition of the
 *   result is therefore "train each MLP separately with ordinary matrix
 *   products", and that is what this file does: for every model m it slices
 *   its rows of the packed W1 [N,F] and its columns of the packed W2 [O,N],
 *   runs the three-step forward of Section 3 (input-to-hidden product, hidden
 *   activation, hidden-to-output product; no biases, as Section 3 drops them),
 *   a softmax cross-entropy loss (or, for regression, a mean squared error
 *   against real targets), back-propagation (Section 2.3, Section 3) and a
 *   plain SGD update, batch after batch, in fp64.
 *
 *   Readings of points the paper leaves open (loss, optimizer, activation
 *   kink conventions, initialisation) are listed in the design notes and
 *   restated at each function below.
 *
 * Inputs are fp32 (as the GPU path receives them); all arithmetic and all
 * weight state are fp64.  Models are processed in parallel with OpenMP; each
 * model's arithmetic is sequential and independent of the thread count, so
 * results are bitwise reproducible.
 *
 * Optional operand rounding of the two input-layer products (Z = X W1^T and
 * dW1 = dZ^T X) emulates the bf16-in / fp32-accumulate variant: X, W1 and
 * dZ are first taken to fp32 and then to the nearest bfloat16 (ties to
 * even) before they are multiplied; everything else stays fp64.  A hidden
 * bias is the weight of a constant input 1, so in that variant it is rounded
 * like W1, and db1 sums the rounded dZ.
 *
 * Parity pins (see tests/test_oracle_*.py): the Scatter Add worked example of
 * Section 3, the 4-1-2 + 4-2-2 packing example of Section 3, closed forms for
 * W2 = 0, reductions to textbook matrix products (M = 1 identity; all h = 1),
 * central finite differences of the loss, the independence invariant, the
 * pack-equals-alone invariant, activation values against library special
 * functions, and published splitmix64 output values.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define ORC_OK 0
#define ORC_EINVAL (-1)
#define ORC_ENOMEM (-2)

/* ------------------------------------------------------------------------ */
/* Activations.  Ids: 0 identity, 1 ReLU, 2 tanh, 3 sigmoid, 4 ELU(alpha=1), */
/* 5 LeakyReLU(0.01), 6 GELU (exact: z * normal CDF), 7 SiLU, 8 softplus  */
/* (beta=1, linear above 20), 9 Swish with beta=2, and the remaining       */
/* functions of the paper's list (Section 4.2): 10 SELU (the self-        */
/* normalising constants of Klambauer et al., 2017), 11 Hardshrink with    */
/* threshold 0.5, 12 Mish (z tanh(softplus z), Misra 2019).                */
/* Section 3 (last paragraph) applies a different activation to each       */
/* contiguous portion of the hidden layer; which functions is a workload   */
/* choice.  Kinks follow the usual autograd conventions: ReLU'(0)=0,        */
/* LeakyReLU'(0)=0.01, ELU'(0)=1, SELU'(0)=lambda*alpha (the negative       */
/* branch), Hardshrink'(+-0.5)=0 and Hardshrink(+-0.5)=0.                   */
/* ------------------------------------------------------------------------ */

#define ORC_SELU_ALPHA 1.6732632423543772848170429916717
#define ORC_SELU_LAMBDA 1.0507009873554804934193349852946
#define ORC_NUM_ACTS 13

static double orc_softplus(double z) {
  return (z > 0.0 ? z : 0.0) + log1p(exp(-fabs(z)));
}

static double orc_logistic(double x) {
  /* 1/(1+e^-x) written so that exp never overflows */
  if (x >= 0.0) {
    double e = exp(-x);
    return 1.0 / (1.0 + e);
  } else {
    double e = exp(x);
    return e / (1.0 + e);
  }
}

double orc_act(int id, double z) {
  switch (id) {
    case 0: return z;
    case 1: return z > 0.0 ? z : 0.0;
    case 2: return tanh(z);
    case 3: return orc_logistic(z);
    case 4: return z > 0.0 ? z : expm1(z);
    case 5: return z > 0.0 ? z : 0.01 * z;
    case 6: return z * (0.5 * erfc(-z / sqrt(2.0))); /* z * Phi(z), erfc keeps Phi accurate for z << 0 */
    case 7: return z * orc_logistic(z);
    case 8: return z > 20.0 ? z : (z > 0.0 ? z : 0.0) + log1p(exp(-fabs(z)));
    case 9: return z * orc_logistic(2.0 * z);
    case 10: return ORC_SELU_LAMBDA * (z > 0.0 ? z : ORC_SELU_ALPHA * expm1(z));
    case 11: return (z > 0.5 || z < -0.5) ? z : 0.0;
    case 12: return z * tanh(orc_softplus(z));
    default: return NAN;
  }
}

double orc_act_deriv(int id, double z) {
  switch (id) {
    case 0: return 1.0;
    case 1: return z > 0.0 ? 1.0 : 0.0;
    case 2: { double t = tanh(z); return 1.0 - t * t; }
    case 3: { double s = orc_logistic(z); return s * (1.0 - s); }
    case 4: return z > 0.0 ? 1.0 : exp(z);
    case 5: return z > 0.0 ? 1.0 : 0.01;
    case 6: {
      double cdf = 0.5 * erfc(-z / sqrt(2.0));
      double pdf = exp(-0.5 * z * z) / sqrt(2.0 * 3.14159265358979323846);
      return cdf + z * pdf;
    }
    case 7: { double s = orc_logistic(z); return s + z * s * (1.0 - s); }
    case 8: return z > 20.0 ? 1.0 : orc_logistic(z);
    case 9: { double s = orc_logistic(2.0 * z); return s + 2.0 * z * s * (1.0 - s); }
    case 10: return z > 0.0 ? ORC_SELU_LAMBDA : ORC_SELU_LAMBDA * ORC_SELU_ALPHA * exp(z);
    case 11: return (z > 0.5 || z < -0.5) ? 1.0 : 0.0;
    case 12: {
      double t = tanh(orc_softplus(z));
      return t + z * (1.0 - t * t) * orc_logistic(z);
    }
    default: return NAN;
  }
}

/* Size of the slope jump at the activation's kinks (0 for activations
 * differentiable everywhere): ReLU and LeakyReLU at 0, SELU at 0
 * (lambda*alpha left, lambda right), Hardshrink at +-0.5. */
static double orc_kink_jump(int id) {
  switch (id) {
    case 1: return 1.0;
    case 5: return 0.99;
    case 10: return ORC_SELU_LAMBDA * (ORC_SELU_ALPHA - 1.0);
    case 11: return 1.0;
    default: return 0.0;
  }
}

/* Distance of z from the nearest kink of the activation. */
static double orc_kink_dist(int id, double z) {
  return id == 11 ? fabs(fabs(z) - 0.5) : fabs(z);
}

/* ------------------------------------------------------------------------ */
/* Initialisation: U(-1/sqrt(fan_in), +1/sqrt(fan_in)), fan_in = F for W1   */
/* and h_m for model m's W2.  The paper does not say how weights start; the */
/* draws come from splitmix64 (Steele, Lea, Flood, OOPSLA 2014) used as a   */
/* counter-based generator so the value of each weight depends only on      */
/* (seed, tensor, index):                                                    */
/*   key = sm(seed);  r = sm(key ^ (tag << 60) ^ idx)                        */
/*   tag 1: W1, idx = n*F + f;  tag 2: W2, idx = o*N + n                     */
/*   u = (r >> 40) * 2^-24;  w = (float)(2u - 1) * (float)(1/sqrt(fan_in))  */
/* where sm(x) is the splitmix64 output for generator state x.               */
/* ------------------------------------------------------------------------ */

uint64_t orc_splitmix64(uint64_t state) {
  uint64_t z = state + 0x9E3779B97F4A7C15ULL;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

static float orc_uniform_weight(uint64_t key, uint64_t tag, uint64_t idx, float bound) {
  uint64_t r = orc_splitmix64(key ^ (tag << 60) ^ idx);
  double u = (double)(r >> 40) * (1.0 / 16777216.0);
  float centred = (float)(2.0 * u - 1.0); /* exact: a multiple of 2^-23 in [-1,1) */
  volatile float w = centred * bound;     /* one fp32 rounding */
  return w;
}

int orc_init_params(int32_t F, int32_t O, int32_t M, const int32_t* hidden_sizes,
                    uint64_t seed, float* W1, float* W2) {
  if (F < 1 || O < 1 || M < 1 || !hidden_sizes || !W1 || !W2) return ORC_EINVAL;
  int64_t N = 0;
  for (int m = 0; m < M; ++m) {
    if (hidden_sizes[m] < 1) return ORC_EINVAL;
    N += hidden_sizes[m];
  }
  uint64_t key = orc_splitmix64(seed);
  float b1 = (float)(1.0 / sqrt((double)F));
  for (int64_t n = 0; n < N; ++n)
    for (int64_t f = 0; f < F; ++f)
      W1[n * F + f] = orc_uniform_weight(key, 1, (uint64_t)(n * F + f), b1);
  int64_t n0 = 0;
  for (int m = 0; m < M; ++m) {
    int64_t h = hidden_sizes[m];
    float b2 = (float)(1.0 / sqrt((double)h));
    for (int64_t o = 0; o < O; ++o)
      for (int64_t n = n0; n < n0 + h; ++n)
        W2[o * N + n] = orc_uniform_weight(key, 2, (uint64_t)(o * N + n), b2);
    n0 += h;
  }
  return ORC_OK;
}

/* Biases from the same stream: tag 3 for b1 (idx = n, fan_in = F), tag 4
 * for b2 (idx = m*O + o, fan_in = h_m). */
int orc_init_biases(int32_t F, int32_t O, int32_t M, const int32_t* hidden_sizes,
                    uint64_t seed, float* b1, float* b2) {
  if (F < 1 || O < 1 || M < 1 || !hidden_sizes || !b1 || !b2) return ORC_EINVAL;
  int64_t N = 0;
  for (int m = 0; m < M; ++m) {
    if (hidden_sizes[m] < 1) return ORC_EINVAL;
    N += hidden_sizes[m];
  }
  uint64_t key = orc_splitmix64(seed);
  float bound1 = (float)(1.0 / sqrt((double)F));
  for (int64_t n = 0; n < N; ++n) b1[n] = orc_uniform_weight(key, 3, (uint64_t)n, bound1);
  for (int m = 0; m < M; ++m) {
    float bound2 = (float)(1.0 / sqrt((double)hidden_sizes[m]));
    for (int o = 0; o < O; ++o)
      b2[(int64_t)m * O + o] = orc_uniform_weight(key, 4, (uint64_t)((int64_t)m * O + o), bound2);
  }
  return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* Operand rounding of the input-layer products.                            */
/* ------------------------------------------------------------------------ */

/* 0: exact (fp64 products of the given values); 1: bfloat16 operands;
 * 2: bfloat16 operands and Z kept in bfloat16 (the storage variant: the
 * hidden pre-activation is stored as the bfloat16 nearest to its fp32
 * value, and the activation, its slope and everything after them see that
 * stored value). */
static int orc_rounding = 0;

int orc_set_input_rounding(int mode) {
  if (mode < 0 || mode > 2) return ORC_EINVAL;
  orc_rounding = mode;
  return ORC_OK;
}

/* Nearest bfloat16 of an fp32 value, ties to even.  bfloat16 keeps the
 * sign, the 8 exponent bits and the top 7 fraction bits of fp32, so the
 * rounding works on the bit pattern: adding 0x7FFF plus the lowest kept
 * bit carries into the kept bits exactly when the dropped 16 bits exceed
 * half an ulp, or equal it with an odd kept part; the carry may run into
 * the exponent (the next binade, or infinity past the largest finite
 * bfloat16).  NaNs stay NaN (the quiet bit is set before truncation). */
float orc_bf16(float x) {
  uint32_t u;
  memcpy(&u, &x, sizeof u);
  if ((u & 0x7F800000u) == 0x7F800000u && (u & 0x007FFFFFu)) {
    u |= 0x00400000u;
  } else {
    u += 0x7FFFu + ((u >> 16) & 1u);
  }
  u &= 0xFFFF0000u;
  memcpy(&x, &u, sizeof x);
  return x;
}

void orc_bf16_array(const float* in, float* out, int64_t n) {
  for (int64_t i = 0; i < n; ++i) out[i] = orc_bf16(in[i]);
}

/* An operand of the input-layer products as the selected variant sees it. */
static double orc_in(double v) {
  return orc_rounding ? (double)orc_bf16((float)v) : v;
}

/* ------------------------------------------------------------------------ */
/* One model's forward / backward on one batch, Section 3 and Section 2.3.  */
/* ------------------------------------------------------------------------ */

typedef struct {
  int F, O, h, act;
  double* Z;  /* [B,h]  pre-activation */
  double* H;  /* [B,h]  activation */
  double* L;  /* [B,O]  logits */
  double* G;  /* [B,O]  dLoss/dlogits */
  double* dH; /* [B,h] */
  double* dZ; /* [B,h] */
  /* Branch choices at activation jumps (see orc_set_branch): br points at
   * this model's first unit in the first sample row of the current batch
   * (NULL: no choices given); pass [B,h] records the branch taken. */
  const uint8_t* br;
  uint8_t* pass;
  /* Stored-Z choices of rounding mode 2 (see orc_set_stored_z): zc points
   * at this model's first unit in the first sample row of the current
   * batch (NULL: none given). */
  const float* zc;
} orc_scratch;

/* Every caller declares its scratch zero-initialised, so that a failed
 * allocation before this call leaves only NULL pointers to free. */
static int orc_scratch_alloc(orc_scratch* s, int B, int h, int F, int O, int act) {
  s->F = F; s->O = O; s->h = h; s->act = act;
  s->Z = (double*)malloc(sizeof(double) * (size_t)B * h);
  s->H = (double*)malloc(sizeof(double) * (size_t)B * h);
  s->L = (double*)malloc(sizeof(double) * (size_t)B * O);
  s->G = (double*)malloc(sizeof(double) * (size_t)B * O);
  s->dH = (double*)malloc(sizeof(double) * (size_t)B * h);
  s->dZ = (double*)malloc(sizeof(double) * (size_t)B * h);
  s->br = NULL;
  s->zc = NULL;
  s->pass = (uint8_t*)malloc((size_t)B * h);
  return (s->Z && s->H && s->L && s->G && s->dH && s->dZ && s->pass) ? ORC_OK : ORC_ENOMEM;
}

static void orc_scratch_free(orc_scratch* s) {
  free(s->Z); free(s->H); free(s->L); free(s->G); free(s->dH); free(s->dZ); free(s->pass);
}

/* ------------------------------------------------------------------------ */
/* Branch choices at the jumps of an activation (Hardshrink at |z| = 0.5).  */
/* Where Z lies within band * sum_f |x_f w_f| of the jump, a correct fp32   */
/* evaluation may land on either side, and the hidden value and the slope   */
/* then differ by the jump: several results are correct.  A caller that    */
/* wants to check one particular such result against this oracle gives the  */
/* side it took for every (sample, unit): br[row * ld + n] != 0 means the   */
/* value passes (|z| above the threshold), 0 means it is zeroed.  The       */
/* oracle takes the given side only inside the band; everywhere else it     */
/* keeps its own and counts a disagreement (orc_branch_conflicts), so a    */
/* choice outside the band can never be accepted.  Rows are sample indices */
/* of the X given to the call (train: offsets into the sample arrays).     */
/* ------------------------------------------------------------------------ */

static const uint8_t* orc_branch = NULL;
static int64_t orc_branch_ld = 0;
static double orc_branch_band = 0.0;
static int64_t orc_branch_conflict_count = 0;

int orc_set_branch(const uint8_t* br, int64_t ld, double band) {
  if (br && (ld < 1 || !(band >= 0.0))) return ORC_EINVAL;
  orc_branch = br;
  orc_branch_ld = br ? ld : 0;
  orc_branch_band = br ? band : 0.0;
  orc_branch_conflict_count = 0;
  return ORC_OK;
}

int64_t orc_branch_conflicts(void) { return orc_branch_conflict_count; }

/* The branch of Hardshrink for z given the caller's choice g (mag is
 * sum_f |x_f w_f|): inside the band the caller's, else the oracle's own. */
static int orc_hardshrink_pass(double z, double mag, int g) {
  const int own = (z > 0.5 || z < -0.5);
  if (fabs(fabs(z) - 0.5) <= orc_branch_band * mag) return g;
  if (g != own) {
#pragma omp atomic
    orc_branch_conflict_count += 1;
  }
  return own;
}

/* ------------------------------------------------------------------------ */
/* Stored Z of rounding mode 2.  Z is kept as the bfloat16 nearest to its   */
/* fp32 value.  An fp32 evaluation of Z that is correct to within rounding  */
/* may lie on the other side of a bfloat16 rounding midpoint than the fp32  */
/* value of the exact Z, and is then stored as another bfloat16: several    */
/* stored values are correct there.  A caller that wants to check one       */
/* particular such result gives the stored value it produced for every    */
/* (sample, unit): zc[row * ld + n].  The oracle takes the given value only */
/* where some value within band * sum_f |x_f w_f| of the exact Z rounds to  */
/* it (see orc_store_z); anywhere else it keeps its own and counts a        */
/* disagreement (orc_stored_z_conflicts).                                   */
/* ------------------------------------------------------------------------ */

static const float* orc_zc = NULL;
static int64_t orc_zc_ld = 0;
static double orc_zc_band = 0.0;
static int64_t orc_zc_conflict_count = 0;

int orc_set_stored_z(const float* zc, int64_t ld, double band) {
  if (zc && (ld < 1 || !(band >= 0.0))) return ORC_EINVAL;
  orc_zc = zc;
  orc_zc_ld = zc ? ld : 0;
  orc_zc_band = zc ? band : 0.0;
  orc_zc_conflict_count = 0;
  return ORC_OK;
}

int64_t orc_stored_z_conflicts(void) { return orc_zc_conflict_count; }

static float orc_bf16_bits(uint32_t u) {
  float f;
  memcpy(&f, &u, sizeof f);
  return f;
}

/* The stored value of an exact Z z (mag = sum_f |x_f w_f|) under rounding
 * mode 2, given the caller's stored value g (NULL: none).  g is correct if
 * it is the bfloat16 that some value within band * mag of z rounds to: its
 * rounding interval (half-way to each bfloat16 neighbour) reaches within
 * band * mag of z.  Under heavy cancellation (|z| far below mag) that holds
 * for more than the two neighbours of z. */
static double orc_store_z(double z, double mag, const float* g) {
  const float own = orc_bf16((float)z);
  if (!g || *g == own || (isnan(*g) && isnan(own))) return (double)own;
  uint32_t ug;
  memcpy(&ug, g, sizeof ug);
  if ((ug & 0xFFFFu) == 0 && isfinite(*g)) {
    /* the bfloat16 neighbours of g by value (through zero as well) */
    const uint32_t mag_bits = ug & 0x7FFFFFFFu, sign = ug & 0x80000000u;
    double up, dn;
    if (mag_bits == 0) {
      up = (double)orc_bf16_bits(0x00010000u);
      dn = (double)orc_bf16_bits(0x80010000u);
    } else if (!sign) {
      up = (double)orc_bf16_bits(ug + 0x10000u);
      dn = (double)orc_bf16_bits(ug - 0x10000u);
    } else {
      up = (double)orc_bf16_bits(ug - 0x10000u);
      dn = (double)orc_bf16_bits(ug + 0x10000u);
    }
    const double gv = (double)*g;
    const double lo = 0.5 * (gv + dn), hi = 0.5 * (gv + up);
    const double dist = z < lo ? lo - z : (z > hi ? z - hi : 0.0);
    if (dist <= orc_zc_band * mag) return gv;
  }
#pragma omp atomic
  orc_zc_conflict_count += 1;
  return (double)own;
}

/* The slope used by back-propagation for element i of a model's scratch. */
static double orc_slope(const orc_scratch* s, int64_t i) {
  if (s->br && s->act == 11) return s->pass[i] ? 1.0 : 0.0;
  return orc_act_deriv(s->act, s->Z[i]);
}

/* Forward of one standalone MLP (Section 3, three-step procedure):
 *   Z = X W1^T (+ b1)   [B,h]   (input-to-hidden product)
 *   H = act(Z)                  (hidden activation)
 *   L = H W2^T (+ b2)   [B,O]   (hidden-to-output product)
 * w1 is the model's [h,F] block, w2 its [O,h] block; the biases b1 [h] and
 * b2 [O] (the paper drops them only to keep the explanation short) are
 * optional (NULL: none). */
static void orc_model_forward(const orc_scratch* s, int B, const float* X,
                              const double* w1, const double* w2, const double* b1,
                              const double* b2) {
  const int F = s->F, O = s->O, h = s->h;
  for (int b = 0; b < B; ++b)
    for (int j = 0; j < h; ++j) {
      double acc = 0.0;
      for (int f = 0; f < F; ++f)
        acc += orc_in(X[(int64_t)b * F + f]) * orc_in(w1[(int64_t)j * F + f]);
      if (b1) acc += orc_in(b1[j]);   /* the weight of a constant input 1 */
      if (orc_rounding == 2) {
        double mag = b1 ? fabs(orc_in(b1[j])) : 0.0;
        if (s->zc)
          for (int f = 0; f < F; ++f)
            mag += fabs(orc_in(X[(int64_t)b * F + f]) * orc_in(w1[(int64_t)j * F + f]));
        acc = orc_store_z(acc, mag, s->zc ? s->zc + (int64_t)b * orc_zc_ld + j : NULL);
      }
      s->Z[(int64_t)b * h + j] = acc;
      s->H[(int64_t)b * h + j] = orc_act(s->act, acc);
      if (s->br && s->act == 11 && orc_rounding != 2) {
        double mag = b1 ? fabs(orc_in(b1[j])) : 0.0;
        for (int f = 0; f < F; ++f)
          mag += fabs(orc_in(X[(int64_t)b * F + f]) * orc_in(w1[(int64_t)j * F + f]));
        const int p = orc_hardshrink_pass(acc, mag, s->br[(int64_t)b * orc_branch_ld + j] != 0);
        s->pass[(int64_t)b * h + j] = (uint8_t)p;
        s->H[(int64_t)b * h + j] = p ? acc : 0.0;
      }
    }
  for (int b = 0; b < B; ++b)
    for (int o = 0; o < O; ++o) {
      double acc = 0.0;
      for (int j = 0; j < h; ++j) acc += s->H[(int64_t)b * h + j] * w2[(int64_t)o * h + j];
      if (b2) acc += b2[o];
      s->L[(int64_t)b * O + o] = acc;
    }
}

/* Softmax cross-entropy, mean over the batch.  Returns the loss and fills
 * G = dLoss/dL = (softmax(L) - onehot(y)) / B.  Labels outside [0,O) -> NaN. */
static double orc_model_ce(const orc_scratch* s, int B, const int32_t* y) {
  const int O = s->O;
  double total = 0.0;
  for (int b = 0; b < B; ++b) {
    const double* l = s->L + (int64_t)b * O;
    double* g = s->G + (int64_t)b * O;
    int yb = y[b];
    if (yb < 0 || yb >= O) return NAN;
    double mx = l[0];
    for (int o = 1; o < O; ++o) mx = l[o] > mx ? l[o] : mx;
    double se = 0.0;
    for (int o = 0; o < O; ++o) se += exp(l[o] - mx);
    double lse = mx + log(se);
    total += lse - l[yb];
    for (int o = 0; o < O; ++o) g[o] = (exp(l[o] - lse) - (o == yb ? 1.0 : 0.0)) / (double)B;
  }
  return total / (double)B;
}

/* The loss head (both heads are per model, mean over the batch):
 *   0  softmax cross-entropy with integer labels y [B] (classification);
 *   1  mean squared error against real targets t [B,O] (regression, which
 *      the paper names as the method's other use, Section 5):
 *        L = 1/(B O) sum_b sum_o (L[b,o] - t[b,o])^2,
 *        G = dLoss/dL = 2 (L - t) / (B O).
 * The label argument of the entry points is an int32 [B] array under head
 * 0 and a float32 [B,O] array under head 1. */
static int orc_head = 0;

int orc_set_head(int head) {
  if (head != 0 && head != 1) return ORC_EINVAL;
  orc_head = head;
  return ORC_OK;
}

static double orc_model_mse(const orc_scratch* s, int B, const float* t) {
  const int O = s->O;
  const double inv = 1.0 / ((double)B * O);
  double total = 0.0;
  for (int b = 0; b < B; ++b)
    for (int o = 0; o < O; ++o) {
      const double d = s->L[(int64_t)b * O + o] - (double)t[(int64_t)b * O + o];
      total += d * d;
      s->G[(int64_t)b * O + o] = 2.0 * d * inv;
    }
  return total * inv;
}

/* The labels (or targets) of samples s0 .. of a label array. */
static const void* orc_labels_at(const void* y, int64_t s0, int O) {
  return orc_head == 1 ? (const void*)((const float*)y + s0 * O)
                       : (const void*)((const int32_t*)y + s0);
}

static double orc_model_loss(const orc_scratch* s, int B, const void* y) {
  return orc_head == 1 ? orc_model_mse(s, B, (const float*)y)
                       : orc_model_ce(s, B, (const int32_t*)y);
}

/* Back-propagation of the loss through one model (chain rule of the three
 * forward steps):
 *   dW2 = G^T H        [O,h]
 *   dH  = G W2         [B,h]   (W2 before this step's update)
 *   dZ  = dH * act'(Z)
 *   dW1 = dZ^T X       [h,F]                                              */
static void orc_model_backward(const orc_scratch* s, int B, const float* X,
                               const double* w2, double* dw1, double* dw2, double* db1,
                               double* db2) {
  const int F = s->F, O = s->O, h = s->h;
  for (int o = 0; o < O; ++o)
    for (int j = 0; j < h; ++j) {
      double acc = 0.0;
      for (int b = 0; b < B; ++b) acc += s->G[(int64_t)b * O + o] * s->H[(int64_t)b * h + j];
      dw2[(int64_t)o * h + j] = acc;
    }
  for (int b = 0; b < B; ++b)
    for (int j = 0; j < h; ++j) {
      double acc = 0.0;
      for (int o = 0; o < O; ++o) acc += s->G[(int64_t)b * O + o] * w2[(int64_t)o * h + j];
      s->dH[(int64_t)b * h + j] = acc;
      s->dZ[(int64_t)b * h + j] = acc * orc_slope(s, (int64_t)b * h + j);
    }
  for (int j = 0; j < h; ++j)
    for (int f = 0; f < F; ++f) {
      double acc = 0.0;
      for (int b = 0; b < B; ++b)
        acc += orc_in(s->dZ[(int64_t)b * h + j]) * orc_in(X[(int64_t)b * F + f]);
      dw1[(int64_t)j * F + f] = acc;
    }
  /* biases: db1 = sum_b dZ, db2 = sum_b G */
  if (db1)
    for (int j = 0; j < h; ++j) {
      double acc = 0.0;
      for (int b = 0; b < B; ++b) acc += orc_in(s->dZ[(int64_t)b * h + j]);
      db1[j] = acc;
    }
  if (db2)
    for (int o = 0; o < O; ++o) {
      double acc = 0.0;
      for (int b = 0; b < B; ++b) acc += s->G[(int64_t)b * O + o];
      db2[o] = acc;
    }
}

/* Kink allowance for piecewise-linear activations.  When |Z| lies within
 * rounding distance of the kink at 0 (|Z| <= kink_rel * sum_f |x_f w_f|), a
 * correct fp32 evaluation may take either derivative branch; dW1 can then
 * move by at most
 *   allow[j,f] = sum over such b of |dH[b,j]| * slope_jump * |X[b,f]|.     */
static void orc_model_kink_allow(const orc_scratch* s, int B, const float* X,
                                 const double* w1, const double* b1, double* allow,
                                 double* allow_b, double kink_rel) {
  const int F = s->F, h = s->h;
  double jump = orc_kink_jump(s->act);
  for (int64_t i = 0; i < (int64_t)h * F; ++i) allow[i] = 0.0;
  if (allow_b)
    for (int j = 0; j < h; ++j) allow_b[j] = 0.0;
  if (jump == 0.0) return;
  for (int b = 0; b < B; ++b)
    for (int j = 0; j < h; ++j) {
      double mag = 0.0;
      for (int f = 0; f < F; ++f)
        mag += fabs(orc_in(X[(int64_t)b * F + f]) * orc_in(w1[(int64_t)j * F + f]));
      if (b1) mag += fabs(orc_in(b1[j]));
      double z = s->Z[(int64_t)b * h + j];
      if (orc_kink_dist(s->act, z) <= kink_rel * mag) {
        double d = fabs(s->dH[(int64_t)b * h + j]) * jump;
        for (int f = 0; f < F; ++f)
          allow[(int64_t)j * F + f] += d * fabs(orc_in(X[(int64_t)b * F + f]));
        if (allow_b) allow_b[j] += d;   /* the bias: an input fixed at 1 */
      }
    }
}

/* Number of samples b and units j of one model whose Z lies within
 * rel * sum_f |x_f w_f| of a jump of the activation (Hardshrink at +-0.5). */
static int32_t orc_model_value_ties(const orc_scratch* s, int B, const float* X,
                                    const double* w1, const double* b1, double rel) {
  if (s->act != 11) return 0;
  const int F = s->F, h = s->h;
  int32_t n = 0;
  for (int b = 0; b < B; ++b)
    for (int j = 0; j < h; ++j) {
      double mag = 0.0;
      for (int f = 0; f < F; ++f)
        mag += fabs(orc_in(X[(int64_t)b * F + f]) * orc_in(w1[(int64_t)j * F + f]));
      if (b1) mag += fabs(orc_in(b1[j]));
      if (fabs(fabs(s->Z[(int64_t)b * h + j]) - 0.5) <= rel * mag) ++n;
    }
  return n;
}

/* Cancellation allowance of dH = sum_o G[b,o] W2[o,j].  The rows of G sum
 * to zero, so dH can be much smaller than its terms (O = 2 with nearly equal
 * W2 entries).  An fp32 evaluation of G = (softmax - onehot)/B is off by a
 * few units in the last place of Ghat[b,o] = (p[b,o] + [o == y_b]) / B, so
 * dH is off by up to a few ulp of mag = sum_o Ghat |W2[o,j]|.  The per-model
 * tolerance absorbs that while mag stays within 16 |dH|; beyond it, dW1 can
 * move by
 *   allow[j,f] += cond_rel * (mag - 16 |dH|) * |act'(Z)| * |X[b,f]|
 * summed over b (nothing where dH does not cancel). */
static void orc_model_cond_allow(const orc_scratch* s, int B, const float* X,
                                 const void* yv, const double* w2, double* allow,
                                 double* allow_b, double cond_rel) {
  const int F = s->F, O = s->O, h = s->h;
  const int32_t* y = (const int32_t*)yv;
  const float* t = (const float*)yv;
  for (int b = 0; b < B; ++b)
    for (int j = 0; j < h; ++j) {
      double mag = 0.0;
      for (int o = 0; o < O; ++o) {
        double gh;
        if (orc_head == 1) {
          /* an fp32 G = 2 (L - t) / (B O) is off by a few ulp of
           * 2 (|L| + |t|) / (B O) where L and t nearly cancel */
          gh = 2.0 * (fabs(s->L[(int64_t)b * O + o]) + fabs((double)t[(int64_t)b * O + o])) /
               ((double)B * O);
        } else {
          const double g = s->G[(int64_t)b * O + o];
          gh = o == y[b] ? g + 2.0 / B : g;   /* (p + [o == y]) / B */
        }
        mag += gh * fabs(w2[(int64_t)o * h + j]);
      }
      const double excess = mag - 16.0 * fabs(s->dH[(int64_t)b * h + j]);
      if (!(excess > 0.0)) continue;
      const double d = cond_rel * excess * fabs(orc_slope(s, (int64_t)b * h + j));
      for (int f = 0; f < F; ++f)
        allow[(int64_t)j * F + f] += d * fabs(orc_in(X[(int64_t)b * F + f]));
      if (allow_b) allow_b[j] += d;
    }
}

/* Rounding-tie allowance of the bf16 operand mode.  dZ reaches the dW1
 * product as the bfloat16 nearest to its fp32 value; an fp32 evaluation of
 * dZ that is correct to within rounding may sit on the other side of a
 * bfloat16 rounding midpoint than the fp32 value of the exact dZ, and then
 * rounds to the neighbouring bfloat16.  When the fp32 value of dZ lies
 * within tie_rel * mag of a midpoint, with
 *   mag = sum_o |G[b,o] W2[o,j]| * |act'(Z[b,j])|
 * (a bound on the size of the terms dZ is computed from), dW1 can move by
 * at most
 *   allow[j,f] += (the larger bfloat16 spacing next to dZ) * |X[b,f]|.     */
static void orc_model_tie_allow(const orc_scratch* s, int B, const float* X,
                                const double* w2, double* allow, double* allow_b,
                                double tie_rel) {
  const int F = s->F, O = s->O, h = s->h;
  for (int b = 0; b < B; ++b)
    for (int j = 0; j < h; ++j) {
      const float z32 = (float)s->dZ[(int64_t)b * h + j];
      if (!(fabsf(z32) > 1e-30f) || isinf(z32)) continue;
      double mag = 0.0;
      for (int o = 0; o < O; ++o) mag += fabs(s->G[(int64_t)b * O + o] * w2[(int64_t)o * h + j]);
      mag *= fabs(orc_slope(s, (int64_t)b * h + j));
      /* the bfloat16 r nearest to z32 and its two neighbours (bit patterns
       * one unit of the 16-bit pattern apart, same sign) */
      const float r = orc_bf16(z32);
      uint32_t u;
      memcpy(&u, &r, sizeof u);
      const uint32_t uu = u + 0x10000u, ud = u - 0x10000u;
      float up, dn;
      memcpy(&up, &uu, sizeof up);
      memcpy(&dn, &ud, sizeof dn);
      const double a = fabs((double)z32), ar = fabs((double)r);
      const double mid_up = 0.5 * (ar + fabs((double)up));
      const double mid_dn = 0.5 * (ar + fabs((double)dn));
      const double dist = fmin(fabs(a - mid_up), fabs(a - mid_dn));
      if (dist <= tie_rel * mag) {
        const double gap = fmax(fabs((double)up) - ar, ar - fabs((double)dn));
        for (int f = 0; f < F; ++f)
          allow[(int64_t)j * F + f] += gap * fabs(orc_in(X[(int64_t)b * F + f]));
        if (allow_b) allow_b[j] += gap;
      }
    }
}

/* ------------------------------------------------------------------------ */
/* Packed-layout helpers: model m owns rows [off_m, off_m+h_m) of W1 [N,F]  */
/* and columns [off_m, off_m+h_m) of W2 [O,N] (Section 3, Figure 2 layout). */
/* ------------------------------------------------------------------------ */

static int orc_offsets(int M, const int32_t* hs, int64_t* off) {
  off[0] = 0;
  for (int m = 0; m < M; ++m) {
    if (hs[m] < 1) return ORC_EINVAL;
    off[m + 1] = off[m] + hs[m];
  }
  return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* Per-model input feature masks (feature selection, Section 7): model m    */
/* sees input feature f only where mask[m*F + f] != 0; it is then an MLP   */
/* with those k_m features as its whole input, and its W1 block is [h, k_m] */
/* (in the packed [N,F] layout its other columns are zero).  The oracle     */
/* takes the definition literally: it copies the model's columns of X and  */
/* W1 out, trains on them, and writes the results back with zeros in the   */
/* masked columns.  NULL: every model sees every feature.                  */
/* ------------------------------------------------------------------------ */

static const uint8_t* orc_fmask = NULL;

int orc_set_feature_mask(const uint8_t* mask) {
  orc_fmask = mask;
  return ORC_OK;
}

typedef struct {
  int F;      /* features of the shared input */
  int k;      /* features this model sees */
  int* sel;   /* their columns, ascending */
  float* Xm;  /* [Bmax, k]: the model's columns of a batch (NULL: no mask, X as given) */
} orc_view;

static int orc_view_init(orc_view* v, int m, int F, int Bmax) {
  v->F = F;
  v->k = 0;
  v->Xm = NULL;
  v->sel = (int*)malloc(sizeof(int) * (size_t)F);
  if (!v->sel) return ORC_ENOMEM;
  for (int f = 0; f < F; ++f)
    if (!orc_fmask || orc_fmask[(int64_t)m * F + f]) v->sel[v->k++] = f;
  if (orc_fmask) {
    v->Xm = (float*)malloc(sizeof(float) * (size_t)Bmax * (v->k ? v->k : 1));
    if (!v->Xm) return ORC_ENOMEM;
  }
  return ORC_OK;
}

static void orc_view_free(orc_view* v) {
  free(v->sel);
  free(v->Xm);
}

/* Rows [0, B) of X as the model sees them ([B, k], row stride k). */
static const float* orc_view_rows(const orc_view* v, const float* X, int B) {
  if (!v->Xm) return X;
  for (int b = 0; b < B; ++b)
    for (int t = 0; t < v->k; ++t) v->Xm[(int64_t)b * v->k + t] = X[(int64_t)b * v->F + v->sel[t]];
  return v->Xm;
}

/* The model's blocks of the packed parameters: w1 [h, k] (its columns of
 * rows [off, off+h) of W1 [N,F]) and w2 [O, h] (columns of W2 [O,N]). */
static void orc_take(int64_t N, int O, int64_t off, int h, const orc_view* v, const double* W1,
                     const double* W2, double* w1, double* w2) {
  const int F = v->F, k = v->k;
  for (int j = 0; j < h; ++j)
    for (int t = 0; t < k; ++t) w1[(int64_t)j * k + t] = W1[(off + j) * F + v->sel[t]];
  for (int o = 0; o < O; ++o)
    for (int j = 0; j < h; ++j) w2[(int64_t)o * h + j] = W2[(int64_t)o * N + off + j];
}

static void orc_put(int64_t N, int O, int64_t off, int h, const orc_view* v, const double* w1,
                    const double* w2, double* W1, double* W2) {
  const int F = v->F, k = v->k;
  if (W1)
    for (int j = 0; j < h; ++j) {
      double* row = W1 + (off + j) * F;
      for (int f = 0; f < F; ++f) row[f] = 0.0;
      for (int t = 0; t < k; ++t) row[v->sel[t]] = w1[(int64_t)j * k + t];
    }
  if (W2)
    for (int o = 0; o < O; ++o)
      for (int j = 0; j < h; ++j) W2[(int64_t)o * N + off + j] = w2[(int64_t)o * h + j];
}

static int orc_check(int F, int O, int M, const int32_t* hs, const int32_t* acts) {
  if (F < 1 || O < 2 || M < 1 || !hs || !acts) return ORC_EINVAL;
  for (int m = 0; m < M; ++m)
    if (hs[m] < 1 || acts[m] < 0 || acts[m] >= ORC_NUM_ACTS) return ORC_EINVAL;
  return ORC_OK;
}

static void orc_set_threads(int nthreads) {
#ifdef _OPENMP
  if (nthreads > 0) omp_set_num_threads(nthreads);
#else
  (void)nthreads;
#endif
}

int orc_max_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

/* Forward only: logits [B,M,O] (model-major inside each sample row), the
 * layout of the Scatter Add result Y[batch, model, out] of Section 3. */
int orc_forward(int32_t F, int32_t O, int32_t M, const int32_t* hs, const int32_t* acts,
                const double* W1, const double* W2, const double* b1, const double* b2,
                const float* X, int32_t B, double* logits, int nthreads) {
  if (orc_check(F, O, M, hs, acts) || B < 1 || !W1 || !W2 || !X || !logits) return ORC_EINVAL;
  int64_t* off = (int64_t*)malloc(sizeof(int64_t) * (M + 1));
  if (!off) return ORC_ENOMEM;
  orc_offsets(M, hs, off);
  const int64_t N = off[M];
  int err = ORC_OK;
  orc_set_threads(nthreads);
#pragma omp parallel for schedule(dynamic, 1)
  for (int m = 0; m < M; ++m) {
    const int h = hs[m];
    orc_scratch s = {0};
    orc_view v = {0};
    double* w1 = (double*)malloc(sizeof(double) * (size_t)h * F);
    double* w2 = (double*)malloc(sizeof(double) * (size_t)h * O);
    if (!w1 || !w2 || orc_view_init(&v, m, F, B) || orc_scratch_alloc(&s, B, h, v.k, O, acts[m])) {
      err = ORC_ENOMEM;
    } else {
      orc_take(N, O, off[m], h, &v, W1, W2, w1, w2);
      s.br = orc_branch ? orc_branch + off[m] : NULL;
      s.zc = orc_zc ? orc_zc + off[m] : NULL;
      orc_model_forward(&s, B, orc_view_rows(&v, X, B), w1, w2, b1 ? b1 + off[m] : NULL,
                        b2 ? b2 + (int64_t)m * O : NULL);
      for (int b = 0; b < B; ++b)
        for (int o = 0; o < O; ++o)
          logits[((int64_t)b * M + m) * O + o] = s.L[(int64_t)b * O + o];
    }
    orc_scratch_free(&s);
    orc_view_free(&v);
    free(w1); free(w2);
  }
  free(off);
  return err;
}

/* Gradients of L = sum_m L_m on one batch, without an update.  dW1 [N,F],
 * dW2 [O,N], loss [M] (per-model mean cross-entropy).  allow_dW1 [N,F]
 * (may be NULL) receives the kink allowance described above, with
 * kink_rel the relative distance to the kink treated as undetermined, plus
 * in the bf16 operand mode the rounding-tie allowance with tie_rel, plus the
 * cancellation allowance of dH with cond_rel (0 switches it off). */
int orc_gradients(int32_t F, int32_t O, int32_t M, const int32_t* hs, const int32_t* acts,
                  const double* W1, const double* W2, const double* b1, const double* b2,
                  const float* X, const void* y, int32_t B, double* dW1, double* dW2,
                  double* db1, double* db2, double* loss, double* allow_dW1,
                  double* allow_db1, double kink_rel, double tie_rel, double cond_rel,
                  int nthreads) {
  if (orc_check(F, O, M, hs, acts) || B < 1 || !W1 || !W2 || !X || !y || !dW1 || !dW2 || !loss)
    return ORC_EINVAL;
  int64_t* off = (int64_t*)malloc(sizeof(int64_t) * (M + 1));
  if (!off) return ORC_ENOMEM;
  orc_offsets(M, hs, off);
  const int64_t N = off[M];
  int err = ORC_OK;
  orc_set_threads(nthreads);
#pragma omp parallel for schedule(dynamic, 1)
  for (int m = 0; m < M; ++m) {
    const int h = hs[m];
    orc_scratch s = {0};
    orc_view v = {0};
    double* w1 = (double*)malloc(sizeof(double) * (size_t)h * F);
    double* w2 = (double*)malloc(sizeof(double) * (size_t)h * O);
    double* g1 = (double*)malloc(sizeof(double) * (size_t)h * F);
    double* g2 = (double*)malloc(sizeof(double) * (size_t)h * O);
    double* al = allow_dW1 ? (double*)malloc(sizeof(double) * (size_t)h * F) : NULL;
    if (!w1 || !w2 || !g1 || !g2 || (allow_dW1 && !al) || orc_view_init(&v, m, F, B) ||
        orc_scratch_alloc(&s, B, h, v.k, O, acts[m])) {
      err = ORC_ENOMEM;
    } else {
      orc_take(N, O, off[m], h, &v, W1, W2, w1, w2);
      const float* Xm = orc_view_rows(&v, X, B);
      const double* bm1 = b1 ? b1 + off[m] : NULL;
      s.br = orc_branch ? orc_branch + off[m] : NULL;
      s.zc = orc_zc ? orc_zc + off[m] : NULL;
      orc_model_forward(&s, B, Xm, w1, w2, bm1, b2 ? b2 + (int64_t)m * O : NULL);
      loss[m] = orc_model_loss(&s, B, y);
      orc_model_backward(&s, B, Xm, w2, g1, g2, db1 ? db1 + off[m] : NULL,
                         db2 ? db2 + (int64_t)m * O : NULL);
      orc_put(N, O, off[m], h, &v, g1, g2, dW1, dW2);
      if (al) {
        double* ab = allow_db1 ? allow_db1 + off[m] : NULL;
        orc_model_kink_allow(&s, B, Xm, w1, bm1, al, ab, kink_rel);
        if (orc_rounding) orc_model_tie_allow(&s, B, Xm, w2, al, ab, tie_rel);
        if (cond_rel > 0.0) orc_model_cond_allow(&s, B, Xm, y, w2, al, ab, cond_rel);
        orc_put(N, O, off[m], h, &v, al, NULL, allow_dW1, NULL);
      }
    }
    orc_scratch_free(&s);
    orc_view_free(&v);
    free(w1); free(w2); free(g1); free(g2); free(al);
  }
  free(off);
  return err;
}

/* SGD training.  Batches are given explicitly as (offset, length) pairs into
 * the sample arrays X [S,F], y [S]; each batch performs, for every model
 * independently, forward, loss, backward and the simultaneous update
 *   W1 -= lr dW1;  W2 -= lr dW2
 * with one learning rate for all models, or model m's own lr_model[m] when
 * lr_model is given (per-model hyper-parameters, Section 7)
 * (dH uses W2 before the update).  W1_out/W2_out receive the final fp64
 * weights (only the chosen models' entries are written); loss_last [M]
 * receives each model's loss on the last batch, before that batch's
 * update.  models/nmodels select a subset of the models (NULL: all).      */
int orc_train(int32_t F, int32_t O, int32_t M, const int32_t* hs, const int32_t* acts,
              const double* W1, const double* W2, const double* b1, const double* b2,
              const float* X, const void* y,
              int32_t nbatches, const int64_t* batch_off, const int32_t* batch_len,
              double lr, const double* lr_model, double* W1_out, double* W2_out,
              double* b1_out, double* b2_out, double* loss_last,
              const int32_t* models, int32_t nmodels, int32_t* ties, double tie_rel,
              int nthreads) {
  if (orc_check(F, O, M, hs, acts) || nbatches < 0 || !W1 || !W2 || !X || !y ||
      (nbatches > 0 && (!batch_off || !batch_len)) || !W1_out || !W2_out)
    return ORC_EINVAL;
  int Bmax = 1;
  for (int k = 0; k < nbatches; ++k) {
    if (batch_len[k] < 1 || batch_off[k] < 0) return ORC_EINVAL;
    if (batch_len[k] > Bmax) Bmax = batch_len[k];
  }
  int64_t* off = (int64_t*)malloc(sizeof(int64_t) * (M + 1));
  if (!off) return ORC_ENOMEM;
  orc_offsets(M, hs, off);
  const int64_t N = off[M];
  const int count = models ? nmodels : M;
  if (ties)
    for (int m = 0; m < M; ++m) ties[m] = 0;
  int err = ORC_OK;
  orc_set_threads(nthreads);
#pragma omp parallel for schedule(dynamic, 1)
  for (int i = 0; i < count; ++i) {
    const int m = models ? models[i] : i;
    if (m < 0 || m >= M) { err = ORC_EINVAL; continue; }
    const int h = hs[m];
    orc_scratch s = {0};
    double* w1 = (double*)malloc(sizeof(double) * (size_t)h * F);
    double* w2 = (double*)malloc(sizeof(double) * (size_t)h * O);
    double* g1 = (double*)malloc(sizeof(double) * (size_t)h * F);
    double* g2 = (double*)malloc(sizeof(double) * (size_t)h * O);
    /* the model's biases (updated in place) and their gradients */
    double* c1 = b1 ? (double*)malloc(sizeof(double) * (size_t)h * 2) : NULL;
    double* c2 = b2 ? (double*)malloc(sizeof(double) * (size_t)O * 2) : NULL;
    orc_view v = {0};
    if (!w1 || !w2 || !g1 || !g2 || (b1 && !c1) || (b2 && !c2) ||
        orc_view_init(&v, m, F, Bmax) || orc_scratch_alloc(&s, Bmax, h, v.k, O, acts[m])) {
      err = ORC_ENOMEM;
    } else {
      orc_take(N, O, off[m], h, &v, W1, W2, w1, w2);
      if (c1) memcpy(c1, b1 + off[m], sizeof(double) * (size_t)h);
      if (c2) memcpy(c2, b2 + (int64_t)m * O, sizeof(double) * (size_t)O);
      double last = NAN;
      for (int k = 0; k < nbatches; ++k) {
        const int B = batch_len[k];
        const float* Xb = orc_view_rows(&v, X + batch_off[k] * F, B);
        const void* yb = orc_labels_at(y, batch_off[k], O);
        s.br = orc_branch ? orc_branch + batch_off[k] * orc_branch_ld + off[m] : NULL;
        s.zc = orc_zc ? orc_zc + batch_off[k] * orc_zc_ld + off[m] : NULL;
        orc_model_forward(&s, B, Xb, w1, w2, c1, c2);
        last = orc_model_loss(&s, B, yb);
        if (ties) ties[m] += orc_model_value_ties(&s, B, Xb, w1, c1, tie_rel);
        orc_model_backward(&s, B, Xb, w2, g1, g2, c1 ? c1 + h : NULL, c2 ? c2 + O : NULL);
        const double lm = lr_model ? lr_model[m] : lr;
        for (int64_t t = 0; t < (int64_t)h * v.k; ++t) w1[t] -= lm * g1[t];
        for (int64_t t = 0; t < (int64_t)h * O; ++t) w2[t] -= lm * g2[t];
        if (c1)
          for (int j = 0; j < h; ++j) c1[j] -= lm * c1[h + j];
        if (c2)
          for (int o = 0; o < O; ++o) c2[o] -= lm * c2[O + o];
      }
      if (loss_last) loss_last[m] = last;
      orc_put(N, O, off[m], h, &v, w1, w2, W1_out, W2_out);
      if (c1 && b1_out) memcpy(b1_out + off[m], c1, sizeof(double) * (size_t)h);
      if (c2 && b2_out) memcpy(b2_out + (int64_t)m * O, c2, sizeof(double) * (size_t)O);
    }
    orc_scratch_free(&s);
    orc_view_free(&v);
    free(w1); free(w2); free(g1); free(g2); free(c1); free(c2);
  }
  free(off);
  return err;
}

/* Hidden layer of the packed network (Section 3, steps 1 and 2 of the
 * packed procedure, with each contiguous portion of the hidden layer taking
 * its own model's activation): Z [B,N] = X W1^T and H [B,N] = act(Z),
 * both fp64, sample-major. */
int orc_hidden(int32_t F, int32_t M, const int32_t* hs, const int32_t* acts,
               const double* W1, const double* b1, const float* X, int32_t B, double* Z,
               double* H) {
  if (F < 1 || M < 1 || !hs || !acts || !W1 || !X || B < 1 || !Z || !H) return ORC_EINVAL;
  int64_t N = 0;
  for (int m = 0; m < M; ++m) {
    if (hs[m] < 1 || acts[m] < 0 || acts[m] >= ORC_NUM_ACTS) return ORC_EINVAL;
    N += hs[m];
  }
  int64_t n = 0;
  for (int m = 0; m < M; ++m) {
    for (int j = 0; j < hs[m]; ++j, ++n) {
      for (int b = 0; b < B; ++b) {
        double acc = 0.0;
        for (int f = 0; f < F; ++f)
          if (!orc_fmask || orc_fmask[(int64_t)m * F + f])
            acc += orc_in(X[(int64_t)b * F + f]) * orc_in(W1[n * F + f]);
        if (b1) acc += orc_in(b1[n]);
        if (orc_rounding == 2) {
          double mag = b1 ? fabs(orc_in(b1[n])) : 0.0;
          if (orc_zc)
            for (int f = 0; f < F; ++f)
              if (!orc_fmask || orc_fmask[(int64_t)m * F + f])
                mag += fabs(orc_in(X[(int64_t)b * F + f]) * orc_in(W1[n * F + f]));
          acc = orc_store_z(acc, mag, orc_zc ? orc_zc + (int64_t)b * orc_zc_ld + n : NULL);
        }
        Z[(int64_t)b * N + n] = acc;
        H[(int64_t)b * N + n] = orc_act(acts[m], acc);
        if (orc_branch && acts[m] == 11 && orc_rounding != 2) {
          double mag = b1 ? fabs(orc_in(b1[n])) : 0.0;
          for (int f = 0; f < F; ++f)
            if (!orc_fmask || orc_fmask[(int64_t)m * F + f])
              mag += fabs(orc_in(X[(int64_t)b * F + f]) * orc_in(W1[n * F + f]));
          const int p = orc_hardshrink_pass(acc, mag, orc_branch[(int64_t)b * orc_branch_ld + n] != 0);
          H[(int64_t)b * N + n] = p ? acc : 0.0;
        }
      }
    }
  }
  return ORC_OK;
}

/* Value ties of activations with a jump (Hardshrink at +-0.5): counts[m]
 * receives the number of (sample, hidden unit) pairs of model m whose Z lies
 * within rel * sum_f |x_f w_f| of a jump.  An fp32 evaluation that is correct
 * to within rounding may land on either side there, and the hidden value
 * then differs by the size of the jump; a comparison leaves such models out
 * (several results are correct for them). */
int orc_value_ties(int32_t F, int32_t M, const int32_t* hs, const int32_t* acts,
                   const double* W1, const double* b1, const float* X, int32_t B, double rel,
                   int32_t* counts) {
  if (F < 1 || M < 1 || !hs || !acts || !W1 || !X || B < 1 || !counts) return ORC_EINVAL;
  int64_t n = 0;
  for (int m = 0; m < M; ++m) {
    if (hs[m] < 1 || acts[m] < 0 || acts[m] >= ORC_NUM_ACTS) return ORC_EINVAL;
    counts[m] = 0;
    for (int j = 0; j < hs[m]; ++j, ++n) {
      if (acts[m] != 11) continue;
      for (int b = 0; b < B; ++b) {
        double acc = 0.0, mag = 0.0;
        for (int f = 0; f < F; ++f) {
          if (orc_fmask && !orc_fmask[(int64_t)m * F + f]) continue;
          const double t = orc_in(X[(int64_t)b * F + f]) * orc_in(W1[n * F + f]);
          acc += t;
          mag += fabs(t);
        }
        if (b1) {
          acc += orc_in(b1[n]);
          mag += fabs(orc_in(b1[n]));
        }
        if (fabs(fabs(acc) - 0.5) <= rel * mag) counts[m] += 1;
      }
    }
  }
  return ORC_OK;
}

/* Mean loss (the head's) of every model over a whole sample set (no update),
 * evaluated in chunks of at most chunk samples. */
int orc_dataset_loss(int32_t F, int32_t O, int32_t M, const int32_t* hs, const int32_t* acts,
                     const double* W1, const double* W2, const double* b1, const double* b2,
                     const float* X, const void* y, int64_t S, int32_t chunk, double* loss,
                     int nthreads) {
  if (orc_check(F, O, M, hs, acts) || S < 1 || chunk < 1 || !W1 || !W2 || !X || !y || !loss)
    return ORC_EINVAL;
  int64_t* off = (int64_t*)malloc(sizeof(int64_t) * (M + 1));
  if (!off) return ORC_ENOMEM;
  orc_offsets(M, hs, off);
  const int64_t N = off[M];
  int err = ORC_OK;
  orc_set_threads(nthreads);
#pragma omp parallel for schedule(dynamic, 1)
  for (int m = 0; m < M; ++m) {
    const int h = hs[m];
    orc_scratch s = {0};
    orc_view v = {0};
    double* w1 = (double*)malloc(sizeof(double) * (size_t)h * F);
    double* w2 = (double*)malloc(sizeof(double) * (size_t)h * O);
    if (!w1 || !w2 || orc_view_init(&v, m, F, chunk) ||
        orc_scratch_alloc(&s, chunk, h, v.k, O, acts[m])) {
      err = ORC_ENOMEM;
    } else {
      orc_take(N, O, off[m], h, &v, W1, W2, w1, w2);
      double total = 0.0;
      for (int64_t s0 = 0; s0 < S; s0 += chunk) {
        int B = (int)((S - s0) < chunk ? (S - s0) : chunk);
        orc_model_forward(&s, B, orc_view_rows(&v, X + s0 * F, B), w1, w2,
                          b1 ? b1 + off[m] : NULL, b2 ? b2 + (int64_t)m * O : NULL);
        total += orc_model_loss(&s, B, orc_labels_at(y, s0, O)) * B;
      }
      loss[m] = total / (double)S;
    }
    orc_scratch_free(&s);
    orc_view_free(&v);
    free(w1); free(w2);
  }
  free(off);
  return err;
}

/* ======================================================================== */
/* Two hidden layers per model (Section 7, Figure 3: the packing extended   */
/* to MLPs with a second hidden layer, where the hidden-to-hidden product   */
/* of the packed network only ever combines units of the same model).       */
/*                                                                           */
/* Model m has h1_m units in its first hidden layer and h2_m in its second, */
/* one activation act_m for both, and weights                               */
/*   W1  rows [off1_m, off1_m + h1_m) of the packed [N1, F] matrix,          */
/*   W12 the block [h2_m, h1_m] stored row-major at offset K_m of the packed */
/*       vector of all blocks (K_m = sum over earlier models of h1 h2),      */
/*   W2  columns [off2_m, off2_m + h2_m) of the packed [O, N2] matrix.       */
/* The plain definition is each model trained alone with ordinary matrix    */
/* products:                                                                */
/*   Z1 = X W1^T, H1 = act(Z1), Z2 = H1 W12^T, H2 = act(Z2), L = H2 W2^T     */
/* followed by the loss head, back-propagation through the five steps and  */
/* plain SGD with simultaneous updates.                                     */
/* Initialisation: W1 and W2 as for one hidden layer (tags 1 and 2, W2 over */
/* the N2 second-layer units, fan_in h2_m), W12 with tag 5, idx = K_m +      */
/* i h1_m + j, fan_in h1_m.                                                  */
/* ======================================================================== */

typedef struct {
  int F, O, h1, h2, act;
  double *Z1, *H1, *Z2, *H2, *L, *G, *dH2, *dZ2, *dH1, *dZ1;
} orc_deep;

static int orc_deep_alloc(orc_deep* d, int B, int h1, int h2, int F, int O, int act) {
  d->F = F; d->O = O; d->h1 = h1; d->h2 = h2; d->act = act;
  d->Z1 = (double*)malloc(sizeof(double) * (size_t)B * h1);
  d->H1 = (double*)malloc(sizeof(double) * (size_t)B * h1);
  d->Z2 = (double*)malloc(sizeof(double) * (size_t)B * h2);
  d->H2 = (double*)malloc(sizeof(double) * (size_t)B * h2);
  d->L = (double*)malloc(sizeof(double) * (size_t)B * O);
  d->G = (double*)malloc(sizeof(double) * (size_t)B * O);
  d->dH2 = (double*)malloc(sizeof(double) * (size_t)B * h2);
  d->dZ2 = (double*)malloc(sizeof(double) * (size_t)B * h2);
  d->dH1 = (double*)malloc(sizeof(double) * (size_t)B * h1);
  d->dZ1 = (double*)malloc(sizeof(double) * (size_t)B * h1);
  return (d->Z1 && d->H1 && d->Z2 && d->H2 && d->L && d->G && d->dH2 && d->dZ2 && d->dH1 &&
          d->dZ1) ? ORC_OK : ORC_ENOMEM;
}

static void orc_deep_free(orc_deep* d) {
  free(d->Z1); free(d->H1); free(d->Z2); free(d->H2); free(d->L); free(d->G);
  free(d->dH2); free(d->dZ2); free(d->dH1); free(d->dZ1);
}

/* Z1 = X w1^T, H1 = act(Z1), Z2 = H1 w12^T, H2 = act(Z2), L = H2 w2^T. */
static void orc_deep_forward(const orc_deep* d, int B, const float* X, const double* w1,
                             const double* w12, const double* w2) {
  const int F = d->F, O = d->O, h1 = d->h1, h2 = d->h2;
  for (int b = 0; b < B; ++b)
    for (int j = 0; j < h1; ++j) {
      double acc = 0.0;
      for (int f = 0; f < F; ++f) acc += (double)X[(int64_t)b * F + f] * w1[(int64_t)j * F + f];
      d->Z1[(int64_t)b * h1 + j] = acc;
      d->H1[(int64_t)b * h1 + j] = orc_act(d->act, acc);
    }
  for (int b = 0; b < B; ++b)
    for (int i = 0; i < h2; ++i) {
      double acc = 0.0;
      for (int j = 0; j < h1; ++j) acc += d->H1[(int64_t)b * h1 + j] * w12[(int64_t)i * h1 + j];
      d->Z2[(int64_t)b * h2 + i] = acc;
      d->H2[(int64_t)b * h2 + i] = orc_act(d->act, acc);
    }
  for (int b = 0; b < B; ++b)
    for (int o = 0; o < O; ++o) {
      double acc = 0.0;
      for (int i = 0; i < h2; ++i) acc += d->H2[(int64_t)b * h2 + i] * w2[(int64_t)o * h2 + i];
      d->L[(int64_t)b * O + o] = acc;
    }
}

/* The loss head of the one-layer code, on this model's logits. */
static double orc_deep_loss(const orc_deep* d, int B, const void* y) {
  orc_scratch s = {0};
  s.O = d->O;
  s.L = d->L;
  s.G = d->G;
  return orc_model_loss(&s, B, y);
}

/* Back-propagation through the five forward steps:
 *   dW2 = G^T H2, dH2 = G W2, dZ2 = dH2 act'(Z2), dW12 = dZ2^T H1,
 *   dH1 = dZ2 W12, dZ1 = dH1 act'(Z1), dW1 = dZ1^T X
 * (W12 and W2 before this step's update). */
static void orc_deep_backward(const orc_deep* d, int B, const float* X, const double* w12,
                              const double* w2, double* g1, double* g12, double* g2) {
  const int F = d->F, O = d->O, h1 = d->h1, h2 = d->h2;
  for (int o = 0; o < O; ++o)
    for (int i = 0; i < h2; ++i) {
      double acc = 0.0;
      for (int b = 0; b < B; ++b) acc += d->G[(int64_t)b * O + o] * d->H2[(int64_t)b * h2 + i];
      g2[(int64_t)o * h2 + i] = acc;
    }
  for (int b = 0; b < B; ++b)
    for (int i = 0; i < h2; ++i) {
      double acc = 0.0;
      for (int o = 0; o < O; ++o) acc += d->G[(int64_t)b * O + o] * w2[(int64_t)o * h2 + i];
      d->dH2[(int64_t)b * h2 + i] = acc;
      d->dZ2[(int64_t)b * h2 + i] = acc * orc_act_deriv(d->act, d->Z2[(int64_t)b * h2 + i]);
    }
  for (int i = 0; i < h2; ++i)
    for (int j = 0; j < h1; ++j) {
      double acc = 0.0;
      for (int b = 0; b < B; ++b) acc += d->dZ2[(int64_t)b * h2 + i] * d->H1[(int64_t)b * h1 + j];
      g12[(int64_t)i * h1 + j] = acc;
    }
  for (int b = 0; b < B; ++b)
    for (int j = 0; j < h1; ++j) {
      double acc = 0.0;
      for (int i = 0; i < h2; ++i) acc += d->dZ2[(int64_t)b * h2 + i] * w12[(int64_t)i * h1 + j];
      d->dH1[(int64_t)b * h1 + j] = acc;
      d->dZ1[(int64_t)b * h1 + j] = acc * orc_act_deriv(d->act, d->Z1[(int64_t)b * h1 + j]);
    }
  for (int j = 0; j < h1; ++j)
    for (int f = 0; f < F; ++f) {
      double acc = 0.0;
      for (int b = 0; b < B; ++b) acc += d->dZ1[(int64_t)b * h1 + j] * (double)X[(int64_t)b * F + f];
      g1[(int64_t)j * F + f] = acc;
    }
}

/* Allowances of dW1 [h1,F] and dW12 [h2,h1] for what a correct fp32
 * evaluation may differ by (the readings of the one-layer code carried
 * through the second layer):
 *  - a kink tie at a second-layer unit (|Z2| within kink_rel * sum_j
 *    |H1 w12| of a slope jump) moves dZ2[b,i] by jump |dH2[b,i]|, hence
 *    dW12[i,j] by that times |H1[b,j]| and dW1[j,f] by that times
 *    |w12[i,j]| |act'(Z1[b,j])| |X[b,f]|;
 *  - a kink tie at a first-layer unit moves dZ1[b,j] by jump |dH1[b,j]|,
 *    hence dW1[j,f] by that times |X[b,f]|;
 *  - cancellation in dH2 = G W2 (cond_rel, as in the one-layer code) moves
 *    dZ2 by cond_rel (mag - 16 |dH2|) |act'(Z2)| and is carried the same
 *    way as a second-layer tie.
 * Value jumps (Hardshrink at +-0.5) are not allowed for here: a step that
 * meets one is counted by orc_deep_value_ties instead. */
static void orc_deep_allow(const orc_deep* d, int B, const float* X, const void* yv,
                           const double* w1, const double* w12, const double* w2, double* a1,
                           double* a12, double kink_rel, double cond_rel) {
  const int F = d->F, O = d->O, h1 = d->h1, h2 = d->h2;
  const double jump = orc_kink_jump(d->act);
  const int32_t* y = (const int32_t*)yv;
  const float* t = (const float*)yv;
  for (int64_t k = 0; k < (int64_t)h1 * F; ++k) a1[k] = 0.0;
  for (int64_t k = 0; k < (int64_t)h2 * h1; ++k) a12[k] = 0.0;
  for (int b = 0; b < B; ++b) {
    for (int i = 0; i < h2; ++i) {
      double e = 0.0;  /* bound on the change of dZ2[b,i] */
      const double z2 = d->Z2[(int64_t)b * h2 + i];
      if (jump != 0.0) {
        double mag = 0.0;
        for (int j = 0; j < h1; ++j) mag += fabs(d->H1[(int64_t)b * h1 + j] * w12[(int64_t)i * h1 + j]);
        if (orc_kink_dist(d->act, z2) <= kink_rel * mag) e += jump * fabs(d->dH2[(int64_t)b * h2 + i]);
      }
      if (cond_rel > 0.0) {
        double mag = 0.0;
        for (int o = 0; o < O; ++o) {
          double gh;
          if (orc_head == 1) {
            gh = 2.0 * (fabs(d->L[(int64_t)b * O + o]) + fabs((double)t[(int64_t)b * O + o])) /
                 ((double)B * O);
          } else {
            const double g = d->G[(int64_t)b * O + o];
            gh = o == y[b] ? g + 2.0 / B : g;
          }
          mag += gh * fabs(w2[(int64_t)o * h2 + i]);
        }
        const double excess = mag - 16.0 * fabs(d->dH2[(int64_t)b * h2 + i]);
        if (excess > 0.0) e += cond_rel * excess * fabs(orc_act_deriv(d->act, z2));
      }
      if (e == 0.0) continue;
      for (int j = 0; j < h1; ++j) {
        a12[(int64_t)i * h1 + j] += e * fabs(d->H1[(int64_t)b * h1 + j]);
        const double e1 = e * fabs(w12[(int64_t)i * h1 + j]) *
                          fabs(orc_act_deriv(d->act, d->Z1[(int64_t)b * h1 + j]));
        for (int f = 0; f < F; ++f) a1[(int64_t)j * F + f] += e1 * fabs((double)X[(int64_t)b * F + f]);
      }
    }
    if (jump != 0.0)
      for (int j = 0; j < h1; ++j) {
        double mag = 0.0;
        for (int f = 0; f < F; ++f) mag += fabs((double)X[(int64_t)b * F + f] * w1[(int64_t)j * F + f]);
        if (orc_kink_dist(d->act, d->Z1[(int64_t)b * h1 + j]) <= kink_rel * mag) {
          const double e1 = jump * fabs(d->dH1[(int64_t)b * h1 + j]);
          for (int f = 0; f < F; ++f) a1[(int64_t)j * F + f] += e1 * fabs((double)X[(int64_t)b * F + f]);
        }
      }
  }
}

/* Value ties (Hardshrink at +-0.5) of both hidden layers of one model. */
static int32_t orc_deep_value_ties(const orc_deep* d, int B, const float* X, const double* w1,
                                   const double* w12, double rel) {
  if (d->act != 11) return 0;
  const int F = d->F, h1 = d->h1, h2 = d->h2;
  int32_t n = 0;
  for (int b = 0; b < B; ++b) {
    for (int j = 0; j < h1; ++j) {
      double mag = 0.0;
      for (int f = 0; f < F; ++f) mag += fabs((double)X[(int64_t)b * F + f] * w1[(int64_t)j * F + f]);
      if (fabs(fabs(d->Z1[(int64_t)b * h1 + j]) - 0.5) <= rel * mag) ++n;
    }
    for (int i = 0; i < h2; ++i) {
      double mag = 0.0;
      for (int j = 0; j < h1; ++j) mag += fabs(d->H1[(int64_t)b * h1 + j] * w12[(int64_t)i * h1 + j]);
      if (fabs(fabs(d->Z2[(int64_t)b * h2 + i]) - 0.5) <= rel * mag) ++n;
    }
  }
  return n;
}

static int orc_deep_check(int F, int O, int M, const int32_t* h1, const int32_t* h2,
                          const int32_t* acts) {
  if (F < 1 || O < 2 || M < 1 || !h1 || !h2 || !acts) return ORC_EINVAL;
  for (int m = 0; m < M; ++m)
    if (h1[m] < 1 || h2[m] < 1 || acts[m] < 0 || acts[m] >= ORC_NUM_ACTS) return ORC_EINVAL;
  return ORC_OK;
}

/* Offsets of the packed layout: off1 [M+1] rows of W1, off2 [M+1] columns
 * of W2, koff [M+1] entries of the W12 blocks. */
static int orc_deep_offsets(int M, const int32_t* h1, const int32_t* h2, int64_t* off1,
                            int64_t* off2, int64_t* koff) {
  off1[0] = off2[0] = koff[0] = 0;
  for (int m = 0; m < M; ++m) {
    off1[m + 1] = off1[m] + h1[m];
    off2[m + 1] = off2[m] + h2[m];
    koff[m + 1] = koff[m] + (int64_t)h1[m] * h2[m];
  }
  return ORC_OK;
}

int orc_deep_init(int32_t F, int32_t O, int32_t M, const int32_t* h1, const int32_t* h2,
                  uint64_t seed, float* W1, float* W12, float* W2) {
  if (F < 1 || O < 1 || M < 1 || !h1 || !h2 || !W1 || !W12 || !W2) return ORC_EINVAL;
  int64_t N1 = 0, N2 = 0;
  for (int m = 0; m < M; ++m) {
    if (h1[m] < 1 || h2[m] < 1) return ORC_EINVAL;
    N1 += h1[m];
    N2 += h2[m];
  }
  const uint64_t key = orc_splitmix64(seed);
  const float b1 = (float)(1.0 / sqrt((double)F));
  for (int64_t n = 0; n < N1; ++n)
    for (int64_t f = 0; f < F; ++f)
      W1[n * F + f] = orc_uniform_weight(key, 1, (uint64_t)(n * F + f), b1);
  int64_t k = 0, n2 = 0;
  for (int m = 0; m < M; ++m) {
    const float b12 = (float)(1.0 / sqrt((double)h1[m]));
    for (int64_t t = 0; t < (int64_t)h1[m] * h2[m]; ++t, ++k)
      W12[k] = orc_uniform_weight(key, 5, (uint64_t)k, b12);
    const float b2 = (float)(1.0 / sqrt((double)h2[m]));
    for (int64_t o = 0; o < O; ++o)
      for (int64_t n = n2; n < n2 + h2[m]; ++n)
        W2[o * N2 + n] = orc_uniform_weight(key, 2, (uint64_t)(o * N2 + n), b2);
    n2 += h2[m];
  }
  return ORC_OK;
}

/* One model's weights out of the packed arrays and back. */
static void orc_deep_take(int64_t N2, int F, int O, int h1, int h2, int64_t o1, int64_t o2,
                          int64_t ko, const double* W1, const double* W12, const double* W2,
                          double* w1, double* w12, double* w2) {
  memcpy(w1, W1 + o1 * F, sizeof(double) * (size_t)h1 * F);
  memcpy(w12, W12 + ko, sizeof(double) * (size_t)h1 * h2);
  for (int o = 0; o < O; ++o)
    for (int i = 0; i < h2; ++i) w2[(int64_t)o * h2 + i] = W2[(int64_t)o * N2 + o2 + i];
}

static void orc_deep_put(int64_t N2, int F, int O, int h1, int h2, int64_t o1, int64_t o2,
                         int64_t ko, const double* w1, const double* w12, const double* w2,
                         double* W1, double* W12, double* W2) {
  if (W1) memcpy(W1 + o1 * F, w1, sizeof(double) * (size_t)h1 * F);
  if (W12) memcpy(W12 + ko, w12, sizeof(double) * (size_t)h1 * h2);
  if (W2)
    for (int o = 0; o < O; ++o)
      for (int i = 0; i < h2; ++i) W2[(int64_t)o * N2 + o2 + i] = w2[(int64_t)o * h2 + i];
}

/* Forward only: logits [B, M, O]. */
int orc_deep_forward_all(int32_t F, int32_t O, int32_t M, const int32_t* h1, const int32_t* h2,
                         const int32_t* acts, const double* W1, const double* W12,
                         const double* W2, const float* X, int32_t B, double* logits,
                         int nthreads) {
  if (orc_deep_check(F, O, M, h1, h2, acts) || B < 1 || !W1 || !W12 || !W2 || !X || !logits)
    return ORC_EINVAL;
  int64_t* off = (int64_t*)malloc(sizeof(int64_t) * 3 * (M + 1));
  if (!off) return ORC_ENOMEM;
  int64_t *off1 = off, *off2 = off + M + 1, *koff = off + 2 * (M + 1);
  orc_deep_offsets(M, h1, h2, off1, off2, koff);
  const int64_t N2 = off2[M];
  int err = ORC_OK;
  orc_set_threads(nthreads);
#pragma omp parallel for schedule(dynamic, 1)
  for (int m = 0; m < M; ++m) {
    orc_deep d = {0};
    double* w1 = (double*)malloc(sizeof(double) * (size_t)h1[m] * F);
    double* w12 = (double*)malloc(sizeof(double) * (size_t)h1[m] * h2[m]);
    double* w2 = (double*)malloc(sizeof(double) * (size_t)h2[m] * O);
    if (!w1 || !w12 || !w2 || orc_deep_alloc(&d, B, h1[m], h2[m], F, O, acts[m])) {
      err = ORC_ENOMEM;
    } else {
      orc_deep_take(N2, F, O, h1[m], h2[m], off1[m], off2[m], koff[m], W1, W12, W2, w1, w12, w2);
      orc_deep_forward(&d, B, X, w1, w12, w2);
      for (int b = 0; b < B; ++b)
        for (int o = 0; o < O; ++o) logits[((int64_t)b * M + m) * O + o] = d.L[(int64_t)b * O + o];
    }
    orc_deep_free(&d);
    free(w1); free(w12); free(w2);
  }
  free(off);
  return err;
}

/* Gradients of sum_m L_m on one batch (no update), with the allowances of
 * orc_deep_allow (allow_dW1 / allow_dW12 may be NULL) and the per-model
 * count of value ties (ties may be NULL; rel = tie_rel). */
int orc_deep_gradients(int32_t F, int32_t O, int32_t M, const int32_t* h1, const int32_t* h2,
                       const int32_t* acts, const double* W1, const double* W12,
                       const double* W2, const float* X, const void* y, int32_t B,
                       double* dW1, double* dW12, double* dW2, double* loss, double* allow_dW1,
                       double* allow_dW12, int32_t* ties, double kink_rel, double cond_rel,
                       double tie_rel, int nthreads) {
  if (orc_deep_check(F, O, M, h1, h2, acts) || B < 1 || !W1 || !W12 || !W2 || !X || !y ||
      !dW1 || !dW12 || !dW2 || !loss || (!allow_dW1) != (!allow_dW12))
    return ORC_EINVAL;
  int64_t* off = (int64_t*)malloc(sizeof(int64_t) * 3 * (M + 1));
  if (!off) return ORC_ENOMEM;
  int64_t *off1 = off, *off2 = off + M + 1, *koff = off + 2 * (M + 1);
  orc_deep_offsets(M, h1, h2, off1, off2, koff);
  const int64_t N2 = off2[M];
  int err = ORC_OK;
  orc_set_threads(nthreads);
#pragma omp parallel for schedule(dynamic, 1)
  for (int m = 0; m < M; ++m) {
    const int a = h1[m], c = h2[m];
    orc_deep d = {0};
    double* w1 = (double*)malloc(sizeof(double) * (size_t)a * F);
    double* w12 = (double*)malloc(sizeof(double) * (size_t)a * c);
    double* w2 = (double*)malloc(sizeof(double) * (size_t)c * O);
    double* g1 = (double*)malloc(sizeof(double) * (size_t)a * F);
    double* g12 = (double*)malloc(sizeof(double) * (size_t)a * c);
    double* g2 = (double*)malloc(sizeof(double) * (size_t)c * O);
    double* al1 = allow_dW1 ? (double*)malloc(sizeof(double) * (size_t)a * F) : NULL;
    double* al12 = allow_dW1 ? (double*)malloc(sizeof(double) * (size_t)a * c) : NULL;
    if (!w1 || !w12 || !w2 || !g1 || !g12 || !g2 || (allow_dW1 && (!al1 || !al12)) ||
        orc_deep_alloc(&d, B, a, c, F, O, acts[m])) {
      err = ORC_ENOMEM;
    } else {
      orc_deep_take(N2, F, O, a, c, off1[m], off2[m], koff[m], W1, W12, W2, w1, w12, w2);
      orc_deep_forward(&d, B, X, w1, w12, w2);
      loss[m] = orc_deep_loss(&d, B, y);
      orc_deep_backward(&d, B, X, w12, w2, g1, g12, g2);
      orc_deep_put(N2, F, O, a, c, off1[m], off2[m], koff[m], g1, g12, g2, dW1, dW12, dW2);
      if (al1) {
        orc_deep_allow(&d, B, X, y, w1, w12, w2, al1, al12, kink_rel, cond_rel);
        orc_deep_put(N2, F, O, a, c, off1[m], off2[m], koff[m], al1, al12, NULL, allow_dW1,
                     allow_dW12, NULL);
      }
      if (ties) ties[m] = orc_deep_value_ties(&d, B, X, w1, w12, tie_rel);
    }
    orc_deep_free(&d);
    free(w1); free(w12); free(w2); free(g1); free(g12); free(g2); free(al1); free(al12);
  }
  free(off);
  return err;
}

/* SGD over the given (offset, length) batches, every model independently
 * (one learning rate); final fp64 weights of the chosen models (models /
 * nmodels, NULL: all) into W1_out, W12_out, W2_out; the loss of the last
 * batch into loss_last; value ties met during training into ties. */
int orc_deep_train(int32_t F, int32_t O, int32_t M, const int32_t* h1, const int32_t* h2,
                   const int32_t* acts, const double* W1, const double* W12, const double* W2,
                   const float* X, const void* y, int32_t nbatches, const int64_t* batch_off,
                   const int32_t* batch_len, double lr, double* W1_out, double* W12_out,
                   double* W2_out, double* loss_last, const int32_t* models, int32_t nmodels,
                   int32_t* ties, double tie_rel, int nthreads) {
  if (orc_deep_check(F, O, M, h1, h2, acts) || nbatches < 0 || !W1 || !W12 || !W2 || !X || !y ||
      (nbatches > 0 && (!batch_off || !batch_len)) || !W1_out || !W12_out || !W2_out)
    return ORC_EINVAL;
  int Bmax = 1;
  for (int k = 0; k < nbatches; ++k) {
    if (batch_len[k] < 1 || batch_off[k] < 0) return ORC_EINVAL;
    if (batch_len[k] > Bmax) Bmax = batch_len[k];
  }
  int64_t* off = (int64_t*)malloc(sizeof(int64_t) * 3 * (M + 1));
  if (!off) return ORC_ENOMEM;
  int64_t *off1 = off, *off2 = off + M + 1, *koff = off + 2 * (M + 1);
  orc_deep_offsets(M, h1, h2, off1, off2, koff);
  const int64_t N2 = off2[M];
  const int count = models ? nmodels : M;
  if (ties)
    for (int m = 0; m < M; ++m) ties[m] = 0;
  int err = ORC_OK;
  orc_set_threads(nthreads);
#pragma omp parallel for schedule(dynamic, 1)
  for (int t = 0; t < count; ++t) {
    const int m = models ? models[t] : t;
    if (m < 0 || m >= M) { err = ORC_EINVAL; continue; }
    const int a = h1[m], c = h2[m];
    orc_deep d = {0};
    double* w1 = (double*)malloc(sizeof(double) * (size_t)a * F);
    double* w12 = (double*)malloc(sizeof(double) * (size_t)a * c);
    double* w2 = (double*)malloc(sizeof(double) * (size_t)c * O);
    double* g1 = (double*)malloc(sizeof(double) * (size_t)a * F);
    double* g12 = (double*)malloc(sizeof(double) * (size_t)a * c);
    double* g2 = (double*)malloc(sizeof(double) * (size_t)c * O);
    if (!w1 || !w12 || !w2 || !g1 || !g12 || !g2 ||
        orc_deep_alloc(&d, Bmax, a, c, F, O, acts[m])) {
      err = ORC_ENOMEM;
    } else {
      orc_deep_take(N2, F, O, a, c, off1[m], off2[m], koff[m], W1, W12, W2, w1, w12, w2);
      double last = NAN;
      for (int k = 0; k < nbatches; ++k) {
        const float* Xb = X + batch_off[k] * F;
        const int B = batch_len[k];
        orc_deep_forward(&d, B, Xb, w1, w12, w2);
        last = orc_deep_loss(&d, B, orc_labels_at(y, batch_off[k], O));
        if (ties) ties[m] += orc_deep_value_ties(&d, B, Xb, w1, w12, tie_rel);
        orc_deep_backward(&d, B, Xb, w12, w2, g1, g12, g2);
        for (int64_t q = 0; q < (int64_t)a * F; ++q) w1[q] -= lr * g1[q];
        for (int64_t q = 0; q < (int64_t)a * c; ++q) w12[q] -= lr * g12[q];
        for (int64_t q = 0; q < (int64_t)c * O; ++q) w2[q] -= lr * g2[q];
      }
      if (loss_last) loss_last[m] = last;
      orc_deep_put(N2, F, O, a, c, off1[m], off2[m], koff[m], w1, w12, w2, W1_out, W12_out,
                   W2_out);
    }
    orc_deep_free(&d);
    free(w1); free(w12); free(w2); free(g1); free(g12); free(g2);
  }
  free(off);
  return err;
}
