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

/* 0: exact (fp64 products of the given values); 1: bfloat16 operands. */
static int orc_rounding = 0;

int orc_set_input_rounding(int mode) {
  if (mode != 0 && mode != 1) return ORC_EINVAL;
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
} orc_scratch;

static int orc_scratch_alloc(orc_scratch* s, int B, int h, int F, int O, int act) {
  s->F = F; s->O = O; s->h = h; s->act = act;
  s->Z = (double*)malloc(sizeof(double) * (size_t)B * h);
  s->H = (double*)malloc(sizeof(double) * (size_t)B * h);
  s->L = (double*)malloc(sizeof(double) * (size_t)B * O);
  s->G = (double*)malloc(sizeof(double) * (size_t)B * O);
  s->dH = (double*)malloc(sizeof(double) * (size_t)B * h);
  s->dZ = (double*)malloc(sizeof(double) * (size_t)B * h);
  return (s->Z && s->H && s->L && s->G && s->dH && s->dZ) ? ORC_OK : ORC_ENOMEM;
}

static void orc_scratch_free(orc_scratch* s) {
  free(s->Z); free(s->H); free(s->L); free(s->G); free(s->dH); free(s->dZ);
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
      s->Z[(int64_t)b * h + j] = acc;
      s->H[(int64_t)b * h + j] = orc_act(s->act, acc);
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
      s->dZ[(int64_t)b * h + j] = acc * orc_act_deriv(s->act, s->Z[(int64_t)b * h + j]);
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
      const double d = cond_rel * excess * fabs(orc_act_deriv(s->act, s->Z[(int64_t)b * h + j]));
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
      mag *= fabs(orc_act_deriv(s->act, s->Z[(int64_t)b * h + j]));
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

static void orc_take(int64_t N, int F, int O, int64_t off, int h, const double* W1,
                     const double* W2, double* w1, double* w2) {
  memcpy(w1, W1 + off * F, sizeof(double) * (size_t)h * F);
  for (int o = 0; o < O; ++o)
    for (int j = 0; j < h; ++j) w2[(int64_t)o * h + j] = W2[(int64_t)o * N + off + j];
}

static void orc_put(int64_t N, int F, int O, int64_t off, int h, const double* w1,
                    const double* w2, double* W1, double* W2) {
  if (W1) memcpy(W1 + off * F, w1, sizeof(double) * (size_t)h * F);
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
    orc_scratch s;
    double* w1 = (double*)malloc(sizeof(double) * (size_t)h * F);
    double* w2 = (double*)malloc(sizeof(double) * (size_t)h * O);
    if (!w1 || !w2 || orc_scratch_alloc(&s, B, h, F, O, acts[m])) {
      err = ORC_ENOMEM;
    } else {
      orc_take(N, F, O, off[m], h, W1, W2, w1, w2);
      orc_model_forward(&s, B, X, w1, w2, b1 ? b1 + off[m] : NULL, b2 ? b2 + (int64_t)m * O : NULL);
      for (int b = 0; b < B; ++b)
        for (int o = 0; o < O; ++o)
          logits[((int64_t)b * M + m) * O + o] = s.L[(int64_t)b * O + o];
    }
    orc_scratch_free(&s);
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
    orc_scratch s;
    double* w1 = (double*)malloc(sizeof(double) * (size_t)h * F);
    double* w2 = (double*)malloc(sizeof(double) * (size_t)h * O);
    double* g1 = (double*)malloc(sizeof(double) * (size_t)h * F);
    double* g2 = (double*)malloc(sizeof(double) * (size_t)h * O);
    double* al = allow_dW1 ? (double*)malloc(sizeof(double) * (size_t)h * F) : NULL;
    if (!w1 || !w2 || !g1 || !g2 || (allow_dW1 && !al) ||
        orc_scratch_alloc(&s, B, h, F, O, acts[m])) {
      err = ORC_ENOMEM;
    } else {
      orc_take(N, F, O, off[m], h, W1, W2, w1, w2);
      const double* bm1 = b1 ? b1 + off[m] : NULL;
      orc_model_forward(&s, B, X, w1, w2, bm1, b2 ? b2 + (int64_t)m * O : NULL);
      loss[m] = orc_model_loss(&s, B, y);
      orc_model_backward(&s, B, X, w2, g1, g2, db1 ? db1 + off[m] : NULL,
                         db2 ? db2 + (int64_t)m * O : NULL);
      orc_put(N, F, O, off[m], h, g1, g2, dW1, dW2);
      if (al) {
        double* ab = allow_db1 ? allow_db1 + off[m] : NULL;
        orc_model_kink_allow(&s, B, X, w1, bm1, al, ab, kink_rel);
        if (orc_rounding) orc_model_tie_allow(&s, B, X, w2, al, ab, tie_rel);
        if (cond_rel > 0.0) orc_model_cond_allow(&s, B, X, y, w2, al, ab, cond_rel);
        memcpy(allow_dW1 + off[m] * F, al, sizeof(double) * (size_t)h * F);
      }
    }
    orc_scratch_free(&s);
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
    orc_scratch s;
    double* w1 = (double*)malloc(sizeof(double) * (size_t)h * F);
    double* w2 = (double*)malloc(sizeof(double) * (size_t)h * O);
    double* g1 = (double*)malloc(sizeof(double) * (size_t)h * F);
    double* g2 = (double*)malloc(sizeof(double) * (size_t)h * O);
    /* the model's biases (updated in place) and their gradients */
    double* c1 = b1 ? (double*)malloc(sizeof(double) * (size_t)h * 2) : NULL;
    double* c2 = b2 ? (double*)malloc(sizeof(double) * (size_t)O * 2) : NULL;
    if (!w1 || !w2 || !g1 || !g2 || (b1 && !c1) || (b2 && !c2) ||
        orc_scratch_alloc(&s, Bmax, h, F, O, acts[m])) {
      err = ORC_ENOMEM;
    } else {
      orc_take(N, F, O, off[m], h, W1, W2, w1, w2);
      if (c1) memcpy(c1, b1 + off[m], sizeof(double) * (size_t)h);
      if (c2) memcpy(c2, b2 + (int64_t)m * O, sizeof(double) * (size_t)O);
      double last = NAN;
      for (int k = 0; k < nbatches; ++k) {
        const float* Xb = X + batch_off[k] * F;
        const void* yb = orc_labels_at(y, batch_off[k], O);
        const int B = batch_len[k];
        orc_model_forward(&s, B, Xb, w1, w2, c1, c2);
        last = orc_model_loss(&s, B, yb);
        if (ties) ties[m] += orc_model_value_ties(&s, B, Xb, w1, c1, tie_rel);
        orc_model_backward(&s, B, Xb, w2, g1, g2, c1 ? c1 + h : NULL, c2 ? c2 + O : NULL);
        const double lm = lr_model ? lr_model[m] : lr;
        for (int64_t t = 0; t < (int64_t)h * F; ++t) w1[t] -= lm * g1[t];
        for (int64_t t = 0; t < (int64_t)h * O; ++t) w2[t] -= lm * g2[t];
        if (c1)
          for (int j = 0; j < h; ++j) c1[j] -= lm * c1[h + j];
        if (c2)
          for (int o = 0; o < O; ++o) c2[o] -= lm * c2[O + o];
      }
      if (loss_last) loss_last[m] = last;
      orc_put(N, F, O, off[m], h, w1, w2, W1_out, W2_out);
      if (c1 && b1_out) memcpy(b1_out + off[m], c1, sizeof(double) * (size_t)h);
      if (c2 && b2_out) memcpy(b2_out + (int64_t)m * O, c2, sizeof(double) * (size_t)O);
    }
    orc_scratch_free(&s);
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
        for (int f = 0; f < F; ++f) acc += orc_in(X[(int64_t)b * F + f]) * orc_in(W1[n * F + f]);
        if (b1) acc += orc_in(b1[n]);
        Z[(int64_t)b * N + n] = acc;
        H[(int64_t)b * N + n] = orc_act(acts[m], acc);
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
    orc_scratch s;
    double* w1 = (double*)malloc(sizeof(double) * (size_t)h * F);
    double* w2 = (double*)malloc(sizeof(double) * (size_t)h * O);
    if (!w1 || !w2 || orc_scratch_alloc(&s, chunk, h, F, O, acts[m])) {
      err = ORC_ENOMEM;
    } else {
      orc_take(N, F, O, off[m], h, W1, W2, w1, w2);
      double total = 0.0;
      for (int64_t s0 = 0; s0 < S; s0 += chunk) {
        int B = (int)((S - s0) < chunk ? (S - s0) : chunk);
        orc_model_forward(&s, B, X + s0 * F, w1, w2, b1 ? b1 + off[m] : NULL,
                          b2 ? b2 + (int64_t)m * O : NULL);
        total += orc_model_loss(&s, B, orc_labels_at(y, s0, O)) * B;
      }
      loss[m] = total / (double)S;
    }
    orc_scratch_free(&s);
    free(w1); free(w2);
  }
  free(off);
  return err;
}
