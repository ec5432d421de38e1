// Internal declarations shared by the host library and the kernel launchers.
// Not part of the public C ABI (include/pmlp.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pmlpk {

// One unit of work of the M3 forward kernel: either a run of whole
// segments (models) whose total width is at most the tile limit, or one
// piece of a segment wider than that limit.  Pieces are summed into the
// logits with atomics; whole segments are written with plain stores.
struct Tile3 {
  int64_t n0;      // first hidden unit
  int32_t len;     // number of hidden units
  int32_t m0;      // model owning hidden unit n0
  int32_t atomic;  // 1: a piece of a split segment
  int32_t reserved;
};
static_assert(sizeof(Tile3) == 24, "Tile3 layout");

enum KernelId {
  KID_PACK_X = 0,
  KID_GEMM_FWD = 1,
  KID_ACT = 2,
  KID_M3_FWD = 3,
  KID_CE = 4,
  KID_M3_BWD = 5,
  KID_GEMM_BWD = 6,
  KID_AUX = 7,
  KID_BWD_FUSED = 8,  // fused backward (M3 backward + dW1 GEMM + updates)
  KID_DEEP = 9,       // the hidden-to-hidden layer of two-layer packs
  KID_FWD_M3 = 10,    // forward product with the activation and M3 in its epilogue
  KID_COUNT = 11
};

// The kernel a launcher chose and the arithmetic of its matrix products
// (PMLP_ARITH_* of include/pmlp.h): every launcher notes it for the host
// library, which keeps the last one per kernel role for pmlp_kernel_variant.
struct KernelVariant {
  const char* name;
  int32_t arith;
};
inline KernelVariant& last_variant() {
  static thread_local KernelVariant v{"", 0};
  return v;
}
inline void note_variant(const char* name, int32_t arith) { last_variant() = KernelVariant{name, arith}; }
constexpr int32_t kArithNone = 0, kArithFp32 = 1, kArithX3 = 2, kArithBf16 = 3;

// GEMM epilogues: C[p][q] = sum_k P[p][k] Q[q][k]
enum GemmEpi {
  EPI_STORE = 0,  // out[p*ldo + q] = C        (float4 over q)
  EPI_SGD = 1,    // out[p*ldo + q] -= lr * C  (float4 over q)
  EPI_GRAD = 2    // out[p*ldo + q] = C for q < ncols (scalar stores)
};

struct GemmArgs {
  const float* P;  // big operand [NP][K], row stride ldp
  int64_t ldp;
  int64_t NP;
  const float* Q;  // small operand [NQ][K], row stride ldq
  int64_t ldq;
  int32_t NQ;      // multiple of 4
  int32_t K;       // multiple of 4
  float* out;
  int64_t ldo;
  int32_t ncols;   // EPI_GRAD: number of valid q columns
  float lr;
  const float* lrm;    // EPI_SGD: per-model rates (null: lr for every row)
  const int32_t* mid;  // model of each row p (with lrm)
  float* db1;          // EPI_GRAD: column bcol (the hidden bias) goes to db1[p]
  int32_t bcol;
  const uint32_t* fmask;  // EPI_SGD / EPI_GRAD: per-model feature masks (null: none)
  int32_t fmw;            // words per model of fmask
};

hipError_t launch_gemm(const GemmArgs& a, int epi, hipStream_t s);

// Input-layer GEMM on the bf16 matrix cores, epilogues as above:
// C[p][q] = sum_k bf16(P[p][k]) Q[q][k] with bf16 Q, or, with fp32 Qf and
// fp32 P, the fp32 product at fp32 accuracy (three-piece splits of both
// operands, six bf16 products per k step).
struct GemmBfArgs {
  const float* P;           // [NP][ldp] fp32 (rounded to bf16 on load, or split), or null and
  const unsigned short* Pb; // [NP][ldp] bf16 bit patterns
  int64_t ldp;              // >= kp
  int32_t kp;               // P columns k < kp are read (finite); later k count as 0
  int64_t NP;
  const unsigned short* Q;  // [NQ][ldq] bf16 bit patterns, zero for K <= k < ldq
  const float* Qf;          // or [NQ][ldq] fp32 (with fp32 P): the three-piece mode
  int64_t ldq;              // bf16 Q: multiple of 64, >= K rounded up to 64;
                            // fp32 Q: multiple of 4, >= K
  int32_t NQ;               // multiple of 4
  int32_t K;                // multiple of 4
  float* out;
  int64_t ldo;
  int32_t ncols;            // EPI_GRAD: number of valid q columns
  float lr;
  const float* lrm;         // EPI_SGD: per-model rates (null: lr for every row)
  const int32_t* mid;       // model of each row p (with lrm)
  float* db1;               // EPI_GRAD: column bcol (the hidden bias) goes to db1[p]
  int32_t bcol;
  unsigned short* outb;     // EPI_SGD: also store bf16 of the updated values (or null);
                            // EPI_STORE: store bf16 of C here instead of fp32 to out
  int64_t ldob;
  const uint32_t* fmask;    // EPI_SGD / EPI_GRAD: per-model feature masks (null: none)
  int32_t fmw;              // words per model of fmask
};
bool gemm_bf16_args_ok(const GemmBfArgs& a);
hipError_t launch_gemm_bf16(const GemmBfArgs& a, int epi, hipStream_t s);

// Row stride (elements) of the bf16 batch copies: n rounded up to 64.
inline int32_t bf16_ld(int32_t n) { return (n + 63) & ~63; }

// Persistent forward GEMM with the batch resident in LDS:
// Zt[p][q] = sum_k W1[p][k] Xp[q][k], p < N, q < Bp (Bp in {16,...,256}).
struct FwdLdsArgs {
  const float* W1;   // [Npad][K]
  const float* Xp;   // [Bp][K]
  float* Zt;         // [Npad][Bp]
  int64_t N;
  int32_t Bp;
  int32_t K;         // F4
};
bool fwd_lds_supported(int32_t Bp, int32_t F4);
hipError_t launch_fwd_lds(const FwdLdsArgs& a, hipStream_t s);

// The forward product with the activation and the M3 forward in its
// epilogue: Zt as launch_fwd_lds, and the logits of every model,
//   out[m*sm + b*sb + o] = sum_{n in model m} act_m(Zt[n][b]) W2[o][n] (+ b2[m][o]),
// written per run of the M3 plan (plain stores; the halves of a split
// segment add atomically onto zeroed logits).  Bp in {128, 256}, O <= 2.
struct FwdM3Args {
  const float* W1;  // [Npad][K]
  const float* Xp;  // [Bp][K]
  float* Zt;        // [Npad][Bp]
  int64_t N;
  int32_t Bp, K, B, O;
  const float* W2;  // [O][ldw]
  int64_t ldw;
  const int64_t* seg_off;
  const int32_t* act;
  const Tile3* tiles;
  const int32_t* order;
  int32_t ntiles;
  const float* b2;  // [M][O] or null
  float* out;
  int64_t sm, sb;
};
bool fwd_m3_supported(int32_t Bp, int32_t F4, int32_t O);
hipError_t launch_fwd_m3(const FwdM3Args& a, hipStream_t s);

// Fused backward (dZ formed in registers, dW1 GEMM, dW2, both updates),
// persistent, with Xt resident in LDS.
struct BwdArgs {
  const float* Zt;   // [Npad][Bp] pre-activations
  const float* G;    // [M][Bp][O] dLoss/dlogits (0 for padded samples)
  const float* Xt;   // [F4][Bp]
  const int32_t* mid;   // [Npad] model of each hidden unit
  const int32_t* actn;  // [Npad] activation id of each hidden unit
  float* W1;         // [Npad][F4], updated unless dW1 is set
  float* W2;         // [O][ldw], updated unless dW2 is set
  float* dW1;        // gradient mode: [N][F]
  float* dW2;        // gradient mode: [O][N]
  int64_t N;
  int64_t ldw;
  int32_t Bp, F, F4, O;
  float lr;
  const float* lrm;  // per-model rates (null: lr for every row)
  float* db1;        // gradient mode: column bcol (the hidden bias) goes to db1[p]
  int32_t bcol;
  const uint32_t* fmask;  // per-model feature masks of the dW1 product (null: none)
  int32_t fmw;            // words per model of fmask
};
bool bwd_lds_supported(int32_t Bp, int32_t F4, int32_t O);
hipError_t launch_bwd_lds(const BwdArgs& a, hipStream_t s);

hipError_t launch_init_params(float* W1, int64_t N, int32_t F, int32_t F4, float bound1,
                              float* W2, int64_t ldw, int32_t O, const int32_t* mid,
                              const float* bound2, uint64_t key, hipStream_t s);

// Hidden biases into W1's column bcol (the weight of a constant input 1) and
// output biases b2 [M][O]; bound2 is per model.
hipError_t launch_init_biases(float* W1, int64_t N, int32_t F4, int32_t bcol, float bound1,
                              float* b2, int32_t M, int32_t O, const float* bound2,
                              uint64_t key, hipStream_t s);

// Column bcol (>= F, or -1 for none) of the copies is 1 for the B real
// samples: the constant input whose weight is the hidden bias.
hipError_t launch_pack_x(const float* X, int32_t B, int32_t F, int32_t Bp, int32_t F4,
                         int32_t bcol, float* Xp, float* Xt, hipStream_t s);

// bf16 copies of the batch (round to nearest even), zero padded:
//   Xp16 [Bp][bf16_ld(F4)]  (operand of Z = X W1^T)
//   Xt16 [F4][bf16_ld(Bp)]  (operand of dW1)
// W1b [Npad][ldb] = bf16(W1 [Npad][F4]), zero for F4 <= k < ldb.
hipError_t launch_w1_to_bf16(const float* W1, int64_t Npad, int32_t F4, unsigned short* W1b,
                             int32_t ldb, hipStream_t s);

hipError_t launch_pack_x_bf16(const float* X, int32_t B, int32_t F, int32_t Bp, int32_t F4,
                              int32_t bcol, unsigned short* Xp16, unsigned short* Xt16,
                              hipStream_t s);

// order: tile indices in launch order (widest first).
hipError_t launch_m3_fwd(const float* Zt, int32_t Bp, int32_t B, const float* W2, int64_t ldw,
                         int32_t O, const int64_t* seg_off, const int32_t* act,
                         const Tile3* tiles, const int32_t* order, int32_t ntiles, const float* b2, float* out,
                         int64_t sm, int64_t sb, hipStream_t s, bool zb = false);

// flag[0] is raised by a label outside [0, O), flag[1] by a non-finite
// per-model rate in lrm (may be null); flag[2] counts models whose loss is
// not finite (the regression head as well).
// With b2 set, db2[m][o] = sum_b G[m][b][o] is stored into db2 (gradient
// mode) or applied as b2 -= lr_m db2 (the rate lrm[m], or lr).
hipError_t launch_ce(float* LG, const int32_t* y, int32_t M, int32_t Bp, int32_t B, int32_t O,
                     float* loss, int32_t* flag, const float* lrm, float* b2, float* db2,
                     float lr, hipStream_t s);

// Regression head: loss[m] = 1/(B O) sum_{b<B,o} (LG[m][b][o] - Y[b][o])^2 and
// LG overwritten by G = 2 (LG - Y) / (B O) (0 for padded samples); flags,
// per-model rates and b2/db2 as launch_ce.
hipError_t launch_mse(float* LG, const float* Y, int32_t M, int32_t Bp, int32_t B, int32_t O,
                      float* loss, int32_t* flag, const float* lrm, float* b2, float* db2,
                      float lr, hipStream_t s);

// M3 backward + activation derivative: dZ over Zt in place (fp32), or, with
// dZ16 set, as bf16 into dZ16 [Npad][Bp] leaving Zt unchanged; then the W2
// update (dW2 null) or the dW2 store.
hipError_t launch_m3_bwd(float* Zt, unsigned short* dZ16, int32_t Bp, float* W2, int64_t N,
                         int64_t ldw, int32_t O, const int32_t* mid, const int64_t* seg_off,
                         const int32_t* act, const float* G, float lr, const float* lrm,
                         float* dW2, hipStream_t s, bool zb = false);

hipError_t launch_hidden_out(const float* Zt, int32_t Bp, int32_t B, int64_t N,
                             const int32_t* mid, const int32_t* act, float* Z, float* H,
                             hipStream_t s, bool zb = false);

hipError_t launch_fill(float* p, int64_t n, float v, hipStream_t s);

// Two hidden layers per model (Section 7, Figure 3).  Model m has h1[m]
// first-layer units (rows off1[m].. of Zt1), h2[m] second-layer units (rows
// off2[m].. of Zt2) and the hidden-to-hidden block W12[koff[m] ..] of
// [h2[m]][h1[m]] (row-major).
struct DeepArgs {
  const int64_t* off1;  // [M+1]
  const int64_t* off2;  // [M+1]
  const int64_t* koff;  // [M+1]
  const int32_t* h1;    // [M]
  const int32_t* h2;    // [M]
  const int32_t* act;   // [M]
  const float* W12;     // [K]
};
struct SegUnit {   // rows r0 .. r0+7 (those that exist) of one layer of model m
  int32_t m, r0;
};
struct SegTile {   // rows i0 .. i0+15, columns j0 .. j0+63 of model m's W12 block
  int32_t m, i0, j0, pad;
};

hipError_t launch_init_w2(float* W2, int64_t N, int64_t ldw, int32_t O, const int32_t* mid,
                          const float* bound2, uint64_t key, hipStream_t s);
hipError_t launch_init_w12(float* W12, int64_t K, const int64_t* koff, int32_t M,
                           const float* bound12, uint64_t key, hipStream_t s);
// Zt2 = W12 act(Zt1) per model; units over second-layer rows.
hipError_t launch_seg_fwd(const float* Zt1, float* Zt2, int32_t Bp, const DeepArgs& a,
                          const SegUnit* units, int32_t nunits, hipStream_t s);
// G12 = dZ2 act(Zt1)^T per model; tiles of the W12 blocks.
hipError_t launch_seg_grad(const float* Zt1, const float* dZ2, int32_t Bp, const DeepArgs& a,
                           const SegTile* tiles, int32_t ntiles, float* G12, hipStream_t s);
// Zt1 <- (W12^T dZ2) * act'(Zt1) per model; units over first-layer rows.
hipError_t launch_seg_back(float* Zt1, const float* dZ2, int32_t Bp, const DeepArgs& a,
                           const SegUnit* units, int32_t nunits, hipStream_t s);
// W -= lr G
hipError_t launch_sgd(float* W, const float* G, int64_t n, float lr, hipStream_t s);

// W1[n][q] = 0 wherever model mid[n] does not see column q (fmask as in
// the argument structs above), for n < Npad and q < F4.
hipError_t launch_apply_fmask(float* W1, int64_t Npad, int32_t F4, const int32_t* mid,
                              const uint32_t* fmask, int32_t fmw, hipStream_t s);

}  // namespace pmlpk
