/*
 * pmlp.h -- C ABI of libpmlp: packed training of many independent
 * one-hidden-layer MLPs ("ParallelMLPs", Farias, Ludermir and Bastos-Filho,
 * 2022) on one AMD Instinct MI355X (gfx950).
 *
 * The problem (Section 3): M independent MLPs share the input features and
 * are trained on the same batches.  Model m has h_m hidden units, its own
 * activation function and no biases (Section 3 drops them).  The hidden
 * units of all models are concatenated into one wide layer of
 * N = sum_m h_m units (Section 3, Figure 2); model m owns the contiguous
 * units [off_m, off_m + h_m).  The hidden-to-output product is replaced by
 * the paper's Modified Matrix Multiplication: an elementwise product of the
 * hidden activations with the output weights followed by a scatter-add
 * keyed by model id (Section 3, Scatter Add definition and the four-step
 * procedure after it), so the per-model gradient paths never mix.
 *
 * Parameter layout (what pmlp_get_params / pmlp_set_params exchange):
 *   W1 [N, F] row-major  -- row n holds the input weights of hidden unit n
 *                           (the paper's W_{hid,in}).
 *   W2 [O, N] row-major  -- column n holds the output weights of hidden
 *                           unit n towards its own model's O outputs.
 * Per-model outputs are laid out as [B, M, O] (o fastest), the paper's
 * Y[batch, model, out].
 *
 * Each training step does, for every model independently: forward,
 * softmax cross-entropy averaged over the batch, back-propagation and a
 * plain SGD update with one learning rate (W1 -= lr dW1, W2 -= lr dW2,
 * both gradients taken at the pre-update weights).
 *
 * Activation ids: 0 identity, 1 ReLU, 2 tanh, 3 logistic sigmoid,
 * 4 ELU (alpha 1), 5 LeakyReLU (slope 0.01), 6 GELU (exact, z * normal
 * CDF), 7 SiLU, 8 softplus (beta 1, identity above 20), 9 Swish with
 * beta 2 (z * sigmoid(2z)), and the rest of the activation list of
 * Section 4.2: 10 SELU (alpha 1.6732632423543772, lambda
 * 1.0507009873554805), 11 Hardshrink (threshold 0.5: z if |z| > 0.5,
 * else 0), 12 Mish (z * tanh(softplus z)).  Derivatives at the kinks:
 * ReLU'(0) = 0, LeakyReLU'(0) = 0.01, ELU'(0) = 1, SELU'(0) =
 * lambda * alpha, Hardshrink'(+-0.5) = 0.
 *
 * Conventions for every call:
 *   - Return value: PMLP_OK (0) or a negative PMLP_E* code; a message for
 *     the last failure on the calling thread is in pmlp_last_error().
 *   - "_dev" pointers are device memory on the handle's device; "_host"
 *     pointers are ordinary host memory.  The caller owns every buffer it
 *     passes and must keep it alive until the handle's stream has reached
 *     the call (enqueueing calls return before the GPU work is done).
 *   - Enqueueing calls (pmlp_forward, pmlp_train_step[_lr], pmlp_gradients,
 *     pmlp_hidden) never synchronise.  Device-side problems such as labels
 *     outside [0, O) are recorded on the device and reported by the next
 *     synchronising call (pmlp_losses).
 *   - A handle is not thread-safe; use one handle per thread or serialise.
 *   - Sizes: B >= 1 samples per batch; rows of X_dev are F contiguous
 *     floats (row stride F).  Batches of any size up to 2^20 are accepted;
 *     internal workspaces grow to the largest batch seen.
 */
#ifndef PMLP_H
#define PMLP_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define PMLP_OK 0
#define PMLP_EINVAL (-1)  /* bad argument (null pointer, size, id, lr) */
#define PMLP_ENOMEM (-2)  /* device or host allocation failed; state unchanged */
#define PMLP_EDEVICE (-3) /* HIP runtime error; see pmlp_last_error() */
#define PMLP_ESTATE (-4)  /* call not valid in the current state */

#define PMLP_FP32 0       /* fp32 operands, fp32 accumulation (default) */
#define PMLP_BF16_GEMM 1  /* the two input-layer GEMMs take bf16-rounded
                             operands with fp32 accumulation */
#define PMLP_BF16_STORE 2 /* PMLP_BF16_GEMM with the hidden pre-activation Z
                             also stored in bf16 between the kernels */

#define PMLP_NUM_ACTS 13

#define PMLP_BIAS 1       /* pmlp_create_ex flag: hidden biases b1 [N] and output
                             biases b2 [M, O] (Section 3 drops them only to keep
                             the explanation short) */

#define PMLP_MSE 2        /* pmlp_create_ex flag: regression head, per-model mean
                             squared error against real targets, trained with
                             pmlp_train_step_mse / pmlp_gradients_mse (the
                             paper names regression as the method's other use,
                             Section 5) */

typedef struct pmlp* pmlp_t;

/* Create a packed model of M MLPs with F inputs and O outputs each.
 * hidden_sizes[M] (each >= 1) and act_ids[M] (each in [0, 12]) are copied;
 * models are packed in the given order.  Weights start uniform in
 * (-1/sqrt(fan_in), +1/sqrt(fan_in)) with fan_in = F for W1 and h_m for
 * model m's W2, drawn from a counter-based splitmix64 stream:
 *   key = sm(seed); r = sm(key ^ (tag << 60) ^ idx), tag 1 for W1
 *   (idx = n*F + f), tag 2 for W2 (idx = o*N + n); u = (r >> 40) * 2^-24;
 *   w = (float)(2u - 1) * (float)(1/sqrt(fan_in))
 * where sm(x) is the splitmix64 output for state x (Steele, Lea and
 * Flood, OOPSLA 2014).  Requires F >= 1, O >= 2, M >= 1.  Uses the
 * current HIP device; the stream defaults to the null stream.
 * On success *out receives a handle the caller frees with pmlp_destroy. */
int pmlp_create(pmlp_t* out, int32_t F, int32_t O, int32_t M,
                const int32_t* hidden_sizes, const int32_t* act_ids,
                uint64_t seed);

/* pmlp_create with flags (0, PMLP_BIAS, PMLP_MSE or both).  With PMLP_BIAS every model
 * computes Z = X W1^T + b1 and logits = act(Z) W2^T + b2, trains b1 and b2
 * by the same SGD (db1 = sum_b dZ, db2 = sum_b G), and the biases start
 * uniform in (-1/sqrt(fan_in), +1/sqrt(fan_in)) from the same stream as the
 * weights: tag 3 for b1 (idx = n, fan_in = F), tag 4 for b2 (idx = m*O + o,
 * fan_in = h_m).  b1 is stored as the weight of a constant input 1, so in
 * the PMLP_BF16_GEMM mode it is rounded with W1.  With PMLP_MSE the loss of
 * model m on a batch is L_m = 1/(B O) sum_b sum_o (logit[b,m,o] - Y[b,o])^2
 * and dLoss/dlogit = 2 (logit - Y) / (B O); such a handle trains only
 * through the _mse calls, and the label-taking calls return PMLP_ESTATE
 * (and the _mse calls on a classification handle).  Unknown flags return
 * PMLP_EINVAL. */
int pmlp_create_ex(pmlp_t* out, int32_t F, int32_t O, int32_t M,
                   const int32_t* hidden_sizes, const int32_t* act_ids,
                   uint64_t seed, int32_t flags);

/* A pack of M MLPs with two hidden layers each (Section 7, Figure 3: the
 * packing extended to deeper MLPs, where a second-layer unit sums only the
 * first-layer units of its own model).  Model m maps F inputs through h1[m]
 * units, then h2[m] units, both with activation act_ids[m], to O outputs:
 *   Z1 = X W1^T, H1 = act(Z1), Z2 = H1 W12_m^T, H2 = act(Z2),
 *   logits = M3 of H2 with W2 (Section 3)
 * and trains, like every pack, by independent per-model softmax
 * cross-entropy and plain SGD.  Parameters (pmlp_get_params_deep):
 *   W1  [N1, F]  rows of the N1 = sum h1 first-layer units, model-major;
 *   W12 [K]      model m's block [h2[m], h1[m]] row-major at offset
 *                K_m = sum over earlier models of h1 h2 (K = the total);
 *   W2  [O, N2]  columns of the N2 = sum h2 second-layer units.
 * Initial values: W1 as pmlp_create (tag 1, fan_in F); W12 uniform with
 * bound 1/sqrt(h1[m]) from the same stream with tag 5 and idx = the packed
 * position; W2 with tag 2, idx = o*N2 + n, bound 1/sqrt(h2[m]).
 * Such a handle takes pmlp_forward, pmlp_train_step, pmlp_losses,
 * pmlp_nonfinite, pmlp_info (N = N1), pmlp_set_stream, profiling and the
 * _deep calls below; the other calls, the PMLP_BF16_GEMM mode, biases,
 * masks and the regression head return PMLP_ESTATE.  Arguments as for
 * pmlp_create (h2[m] >= 1). */
int pmlp_create_deep(pmlp_t* out, int32_t F, int32_t O, int32_t M, const int32_t* h1,
                     const int32_t* h2, const int32_t* act_ids, uint64_t seed);

/* Gradients of sum_m L_m of a two-hidden-layer pack on one batch without an
 * update (device, fp32): dW1_dev [N1, F], dW12_dev [K], dW2_dev [O, N2].
 * Records the batch losses.  PMLP_ESTATE for a one-layer handle. */
int pmlp_gradients_deep(pmlp_t h, const float* X_dev, const int32_t* y_dev, int32_t B,
                        float* dW1_dev, float* dW12_dev, float* dW2_dev);

/* Parameters of a two-hidden-layer pack to / from host memory in the
 * layout above (any pointer may be null).  Synchronous. */
int pmlp_get_params_deep(pmlp_t h, float* W1_host, float* W12_host, float* W2_host);
int pmlp_set_params_deep(pmlp_t h, const float* W1_host, const float* W12_host,
                         const float* W2_host);

/* N2 (second-layer units) and K (entries of all W12 blocks) of a
 * two-hidden-layer pack; PMLP_ESTATE for a one-layer handle. */
int pmlp_info_deep(pmlp_t h, int64_t* N2, int64_t* K);

/* Free the handle and every device buffer it owns (synchronises its
 * stream first).  A null handle is accepted. */
int pmlp_destroy(pmlp_t h);

/* Launch all later work on `stream` (a hipStream_t, passed as void*;
 * null selects the null stream).  The stream must belong to the device
 * the handle was created on; a stream of another device returns
 * PMLP_EINVAL and the handle keeps its stream. */
int pmlp_set_stream(pmlp_t h, void* stream);

/* Select the arithmetic of the two input-layer products (Section 3 step 1,
 * Z = X W1^T, and its gradient dW1 = dZ^T X) for all later calls:
 *   PMLP_FP32 (default): fp32 operands, fp32 accumulation.  For batches
 *     of 65 to 256 samples the products may run on the bf16 matrix cores
 *     with every operand split exactly into three bf16 pieces and six piece
 *     products accumulated in fp32; what that leaves out is at most 2^-23
 *     of each product, the error of fp32 arithmetic (no operand is rounded).
 *   PMLP_BF16_GEMM: X, W1 and dZ are rounded to bf16 (nearest even) as
 *     the products read them and the products accumulate in fp32; the
 *     weights, Z, the activations, logits, loss, gradients of W2 and the
 *     SGD updates stay fp32.  Every shape is supported.
 *   PMLP_BF16_STORE: PMLP_BF16_GEMM, and Z is kept between the kernels as
 *     the bf16 nearest (ties to even) to the fp32 accumulator, in half the
 *     bytes (the memory remark of Section 5: Z is the largest tensor a
 *     step moves); the activation, its derivative and everything after
 *     them use the stored value, and pmlp_hidden returns it (as fp32).
 *     bf16 keeps fp32's exponent range, so nothing in this mode needs
 *     loss scaling.
 * Both bf16 modes are for packs with one hidden layer (PMLP_ESTATE for a
 * pmlp_create_deep handle).  Returns PMLP_EINVAL for any other mode; the
 * handle keeps its mode. */
int pmlp_set_precision(pmlp_t h, int32_t mode);

/* Forward pass only (Section 3: input-to-hidden product, per-model
 * activation, Modified Matrix Multiplication):
 *   logits[b, m, o] = sum_{n in model m} act_m(sum_f X[b,f] W1[n,f]) W2[o,n]
 * X_dev [B, F] fp32, logits_dev [B, M, O] fp32 (written).  No state
 * changes. */
int pmlp_forward(pmlp_t h, const float* X_dev, int32_t B, float* logits_dev);

/* One SGD step on the batch (X_dev [B, F], y_dev [B] int32 labels in
 * [0, O)): forward, per-model mean softmax cross-entropy, back-propagation
 * and the update W -= lr * dW for every model at once.  lr must be
 * finite.  The per-model losses of this batch (at the pre-update weights)
 * are kept for pmlp_losses. */
int pmlp_train_step(pmlp_t h, const float* X_dev, const int32_t* y_dev,
                    int32_t B, float lr);

/* pmlp_train_step with a learning rate per model (per-model
 * hyper-parameters, Section 7): model m's parameters take
 * W -= lr_dev[m] * dW.  lr_dev [M] fp32, device memory, read by the step's
 * kernels.  A non-finite rate is not detected before the step (its model's
 * weights become non-finite); the next pmlp_losses then returns
 * PMLP_EINVAL.  Null pointers return PMLP_EINVAL. */
int pmlp_train_step_lr(pmlp_t h, const float* X_dev, const int32_t* y_dev,
                       int32_t B, const float* lr_dev);

/* pmlp_train_step for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): the same kernels and results, but the step's workspaces (the
 * batch copies, the hidden pre-activations Z [Npad, Bp] and the logits
 * [M, Bp, O], Bp the padded batch) live in one static 256 MiB device array
 * per GPU instead of the handle's growable workspace, and the call makes
 * no hipMalloc, hipFree or event.  The first call on a device looks the
 * array's device address up (hipGetSymbolAddress) and keeps it.
 *   - Returns PMLP_EINVAL, before any device work, when those workspaces
 *     exceed 256 MiB (about Npad * Bp * 4 bytes, e.g. 50,560 units at
 *     1,024 samples fit, 5,005,056 units at 256 do not), and for the
 *     arguments pmlp_train_step rejects.
 *   - PMLP_ESTATE in the PMLP_BF16_GEMM mode (whose bf16 copies the handle
 *     allocates) and for a PMLP_MSE handle.
 *   - Every call on one GPU shares that GPU's array, which keeps the last
 *     call's contents; every part a step reads is written earlier in the
 *     same step, so nothing needs clearing between calls.  Calls that
 *     overlap on one GPU (other handles, other streams, other threads)
 *     race on the array: serialise them.
 *   - Per-kernel profiling records nothing for this call. */
int pmlp_train_step_noalloc(pmlp_t h, const float* X_dev, const int32_t* y_dev, int32_t B,
                            float lr);

/* Copy the per-model loss (mean cross-entropy, or mean squared error for a
 * PMLP_MSE handle) of the last training or gradient batch into out_host [M]
 * (fp32).  Synchronises the
 * stream.  PMLP_ESTATE before any step; PMLP_EINVAL if that batch held a
 * label outside [0, O) (the flag is cleared by the call). */
int pmlp_losses(pmlp_t h, float* out_host);

/* Gradients of sum_m L_m on one batch without updating the weights
 * (L_m is model m's mean cross-entropy, so each model's slice is the
 * gradient of its own loss): dW1_dev [N, F], dW2_dev [O, N], fp32,
 * written.  Uses the same kernels as pmlp_train_step with the update
 * replaced by a store.  Also records the batch losses for pmlp_losses. */
int pmlp_gradients(pmlp_t h, const float* X_dev, const int32_t* y_dev,
                   int32_t B, float* dW1_dev, float* dW2_dev);

/* pmlp_gradients of a handle with biases, which also stores db1_dev [N]
 * and db2_dev [M, O] (device, fp32).  PMLP_ESTATE for a handle without
 * biases; null pointers return PMLP_EINVAL. */
int pmlp_gradients_ex(pmlp_t h, const float* X_dev, const int32_t* y_dev,
                      int32_t B, float* dW1_dev, float* dW2_dev,
                      float* db1_dev, float* db2_dev);

/* Regression head (a handle created with PMLP_MSE): one SGD step and the
 * gradients without update, as pmlp_train_step and pmlp_gradients but with
 * real targets Y_dev [B, O] (device, fp32, row-major) in place of labels;
 * pmlp_losses then returns the per-model mean squared errors.  With
 * PMLP_BIAS the output biases are trained too (db2 = sum_b G).  PMLP_ESTATE
 * for a classification handle; null pointers return PMLP_EINVAL. */
int pmlp_train_step_mse(pmlp_t h, const float* X_dev, const float* Y_dev,
                        int32_t B, float lr);
int pmlp_gradients_mse(pmlp_t h, const float* X_dev, const float* Y_dev,
                       int32_t B, float* dW1_dev, float* dW2_dev);

/* Hidden layer of the packed network: Z_dev [B, N] = X W1^T and
 * H_dev [B, N] = act_{model of n}(Z) (either pointer may be null).  A
 * view of the first two forward steps for inspection and testing. */
int pmlp_hidden(pmlp_t h, const float* X_dev, int32_t B, float* Z_dev,
                float* H_dev);

/* Number of (step, model) pairs whose loss was not finite (NaN or
 * infinite: a diverged model) since the last call or since creation, into
 * *count_host; the count is then cleared.  Synchronises the stream.  The
 * models train independently (Section 3), so a diverged model changes
 * nothing for the others and the steps go on; this is how a caller learns
 * that one diverged without reading every loss.  Null count_host returns
 * PMLP_EINVAL. */
int pmlp_nonfinite(pmlp_t h, int32_t* count_host);

/* Copy the parameters to / from host memory in the layout above
 * (W1_host [N, F], W2_host [O, N], fp32).  Synchronous.  Either pointer
 * may be null to skip that tensor. */
int pmlp_get_params(pmlp_t h, float* W1_host, float* W2_host);
int pmlp_set_params(pmlp_t h, const float* W1_host, const float* W2_host);

/* Parameters of some of the models (model selection in the pool of trained
 * MLPs, Section 7; also a cheap hand-off of a sample of models to a
 * checker): models_host [count] model indices (host, each in [0, M), any
 * order, repeats allowed); with R = the sum of their hidden sizes,
 * W1_host [R, F] receives their W1 rows and W2_host [O, R] their W2
 * columns, model after model in the given order (the layout of a pack of
 * just those models).  Either output may be null.  Synchronous.  Bad
 * indices return PMLP_EINVAL before any copy. */
int pmlp_get_models(pmlp_t h, const int32_t* models_host, int32_t count, float* W1_host,
                    float* W2_host);

/* Per-model input feature masks (feature selection, Section 7: each model
 * may see its own subset of the input features).  mask_host [M, F] (host,
 * row-major, one byte per entry): model m sees feature f where
 * mask_host[m*F + f] != 0 and is then trained as the MLP whose whole input
 * is those features.  The weights of the features a model does not see are
 * set to zero now and held there: every later pmlp_set_params zeroes them
 * again, every SGD step leaves them at zero and pmlp_gradients[_ex|_mse]
 * returns zero for them; no step makes an extra pass over W1 for it (the
 * dW1 product's epilogue drops their gradient).  Biases are never masked.
 * Z = X W1^T then sums over the seen features only, as long as the unseen
 * features of X are finite (they meet zero weights).  A null mask_host
 * removes the masks (the zeroed weights stay zero until set or trained).
 * Synchronises the stream.  The initial weights keep fan_in = F. */
int pmlp_set_feature_mask(pmlp_t h, const uint8_t* mask_host);

/* Biases of a handle created with PMLP_BIAS (PMLP_ESTATE otherwise):
 * b1_host [N], b2_host [M, O] (model-major), host memory, either may be
 * null.  Synchronise the handle's stream. */
int pmlp_get_biases(pmlp_t h, float* b1_host, float* b2_host);
int pmlp_set_biases(pmlp_t h, const float* b1_host, const float* b2_host);

/* Sizes of the packed model; any output pointer may be null. */
int pmlp_info(pmlp_t h, int64_t* N, int32_t* M, int32_t* F, int32_t* O);

/* Per-kernel timing with HIP events on the handle's stream.  While
 * enabled, every kernel launch is bracketed by two events.
 * pmlp_kernel_time synchronises and returns, for kernel id k (0 ..
 * PMLP_NUM_KERNELS-1, names from pmlp_kernel_name), the summed duration
 * in milliseconds and the number of launches since the last reset;
 * pmlp_profile_reset clears the totals. */
#define PMLP_NUM_KERNELS 11
int pmlp_set_profiling(pmlp_t h, int32_t enable);
int pmlp_kernel_time(pmlp_t h, int32_t k, double* total_ms, int64_t* launches);
int pmlp_profile_reset(pmlp_t h);
const char* pmlp_kernel_name(int32_t k);

/* The kernel that role k (as in pmlp_kernel_name) ran at its last launch
 * on this handle, and the arithmetic of its matrix products, as chosen by
 * the library for the shapes it was given: *name receives a library-owned
 * string ("" before the first launch), *arith one of
 *   PMLP_ARITH_NONE  no matrix products (memory and vector ALU work),
 *   PMLP_ARITH_FP32  fp32 matrix-core products,
 *   PMLP_ARITH_X3    fp32 products as six bf16 products of three-piece
 *                    operand splits (fp32 accuracy),
 *   PMLP_ARITH_BF16  bf16 operands, fp32 accumulation.
 * Either pointer may be null.  Lets a caller price a kernel against the
 * ceiling of the arithmetic it really ran. */
#define PMLP_ARITH_NONE 0
#define PMLP_ARITH_FP32 1
#define PMLP_ARITH_X3 2
#define PMLP_ARITH_BF16 3
int pmlp_kernel_variant(pmlp_t h, int32_t k, const char** name, int32_t* arith);

/* Message describing the last failure on the calling thread (a
 * library-owned string, valid until the next failing call on it). */
const char* pmlp_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* PMLP_H */
