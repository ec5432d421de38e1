// libpmlp host side: argument checking, the packing plan, parameter and
// workspace ownership, and step sequencing on one HIP stream.  The C ABI is
// declared and documented in include/pmlp.h.

#include "pmlp.h"
#include "pmlp_internal.h"

#include <algorithm>
#include <cmath>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

using namespace pmlpk;

namespace {

thread_local std::string g_err;

int fail(int code, const std::string& msg) {
  g_err = msg;
  return code;
}

#define PMLP_HIP(expr)                                                                    \
  do {                                                                                    \
    hipError_t e_ = (expr);                                                               \
    if (e_ != hipSuccess)                                                                 \
      return fail(PMLP_EDEVICE, std::string(#expr) + " failed: " + hipGetErrorString(e_)); \
  } while (0)

constexpr int64_t kTile3 = 512;      // M3 forward tile width, largest (hidden units)
constexpr int64_t kTile3Min = 32;    // smallest
constexpr int64_t kTile3Count = 2048;  // tiles wanted to fill the chip
constexpr int32_t kMaxBatch = 1 << 20;
constexpr int32_t kMaxO = 16;

static_assert(KID_COUNT == PMLP_NUM_KERNELS, "kernel id table");

const char* const kKernelNames[KID_COUNT] = {
    "pack_x", "gemm_fwd", "act", "m3_fwd", "ce", "m3_bwd", "gemm_bwd", "aux", "bwd_fused",
    "hidden2", "fwd_m3"};

uint64_t splitmix64_host(uint64_t x) {
  uint64_t z = x + 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

// Workspace of pmlp_train_step_noalloc: one static device array per GPU
// (every GPU the library runs on holds it until the process ends).  Host
// code never uses the array's name as an address: the device address comes
// from hipGetSymbolAddress, once per device, with that device current.
constexpr size_t kScratchBytes = (size_t)256 << 20;
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

template <class T>
void dfree(T*& p) {
  if (p) (void)hipFree(p);
  p = nullptr;
}

}  // namespace

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

// The second hidden layer of a pack made by pmlp_create_deep (the first
// layer is the handle's own plan, W1 and workspaces).
struct PmlpDeep {
  int64_t N2 = 0, N2pad = 0, K = 0;
  std::vector<int32_t> h2;
  std::vector<int64_t> off2, koff;
  int64_t* d_off1 = nullptr;
  int64_t* d_off2 = nullptr;
  int64_t* d_koff = nullptr;
  int32_t* d_h1 = nullptr;
  int32_t* d_h2 = nullptr;
  int32_t* d_mid2 = nullptr;  // [N2pad] model of each second-layer unit
  float* W12 = nullptr;       // [K] hidden-to-hidden blocks
  float* G12 = nullptr;       // [K] their gradient in a training step
  Tile3* d_tiles2 = nullptr;  // M3 forward tiles of the second layer
  int32_t* d_order2 = nullptr;
  int32_t ntiles2 = 0;
  bool has_split2 = false;
  SegUnit* d_ufwd = nullptr;  // row blocks of the second layer
  int32_t nufwd = 0;
  SegUnit* d_uback = nullptr; // row blocks of the first layer
  int32_t nuback = 0;
  SegTile* d_tgrad = nullptr; // tiles of the W12 blocks
  int32_t ntgrad = 0;
  int32_t capBp = 0;
  float* Zt2 = nullptr;       // [N2pad][Bp]
};

struct pmlp {
  int dev = 0;
  hipStream_t stream = nullptr;
  int32_t F = 0, F4 = 0, O = 0, M = 0;
  int64_t N = 0;
  int64_t Npad = 0;  // rows of W1/Zt/mid and the row stride of W2
  int32_t precision = PMLP_FP32;
  std::vector<int32_t> hs, acts;
  std::vector<int64_t> seg_off;

  float* W1 = nullptr;  // [Npad][F4] (+ slack); column bcol holds the hidden biases
  float* W2 = nullptr;  // [O][Npad]
  int32_t bcol = -1;    // with biases: the column of the constant input 1 (F rounded to 4)
  float* b2 = nullptr;  // with biases: output biases [M][O]
  int64_t* d_seg_off = nullptr;
  int32_t* d_act = nullptr;
  int32_t* d_mid = nullptr;   // [Npad] model of each hidden unit
  int32_t* d_actn = nullptr;  // [Npad] activation id of each hidden unit
  Tile3* d_tiles = nullptr;
  int32_t* d_order = nullptr;  // tile indices, widest first
  int32_t ntiles = 0;
  bool has_split = false;
  float* loss = nullptr;   // [M]
  int32_t* flag = nullptr; // [4]: bad label, bad rate, count of non-finite losses, spare

  int32_t capBp = 0;
  float* Xp = nullptr;
  float* Xt = nullptr;
  float* Zt = nullptr;
  float* LG = nullptr;
  int32_t capBp16 = 0;            // bf16 batch copies (bf16 GEMM mode only)
  unsigned short* Xp16 = nullptr; // [Bp][bf16_ld(F4)]
  unsigned short* Xt16 = nullptr; // [F4][bf16_ld(Bp)]
  unsigned short* dZ16 = nullptr; // [Npad][Bp] dZ rounded to bf16
  unsigned short* W1b = nullptr;  // [Npad][bf16_ld(F4)] bf16 of W1 (operand of Z = X W1^T)
  bool w1b_valid = false;         // W1b equals bf16(W1)
  PmlpDeep* deep = nullptr;     // second hidden layer (pmlp_create_deep), or null
  uint32_t* d_fmask = nullptr;  // per-model feature masks [M][fmw] (null: none)
  int32_t fmw = 0;
  bool have_loss = false;
  bool mse = false;         // regression head (PMLP_MSE)
  bool lds_kernels = true;  // persistent LDS-resident GEMMs where they apply
  // the forward product with activation and M3 in one kernel (opt-in: on
  // the 10,000-model shapes the two-kernel forward measures faster)
  bool fused_forward = false;

  bool prof = false;
  struct Pending {
    int k;
    hipEvent_t a, b;
  };
  std::vector<hipEvent_t> ev_free;
  std::vector<Pending> pending;
  double tot_ms[KID_COUNT] = {};
  int64_t launches[KID_COUNT] = {};
  KernelVariant variant[KID_COUNT] = {};  // the kernel each role launched last
};

namespace {

void release(pmlp* h) {
  dfree(h->W1);
  dfree(h->W2);
  dfree(h->b2);
  dfree(h->d_seg_off);
  dfree(h->d_act);
  dfree(h->d_mid);
  dfree(h->d_actn);
  dfree(h->d_tiles);
  dfree(h->d_order);
  dfree(h->loss);
  dfree(h->flag);
  dfree(h->Xp);
  dfree(h->Xt);
  dfree(h->Zt);
  dfree(h->LG);
  dfree(h->Xp16);
  dfree(h->Xt16);
  dfree(h->dZ16);
  dfree(h->W1b);
  dfree(h->d_fmask);
  if (PmlpDeep* d = h->deep) {
    dfree(d->d_off1);
    dfree(d->d_off2);
    dfree(d->d_koff);
    dfree(d->d_h1);
    dfree(d->d_h2);
    dfree(d->d_mid2);
    dfree(d->W12);
    dfree(d->G12);
    dfree(d->d_tiles2);
    dfree(d->d_order2);
    dfree(d->d_ufwd);
    dfree(d->d_uback);
    dfree(d->d_tgrad);
    dfree(d->Zt2);
    delete d;
    h->deep = nullptr;
  }
  h->w1b_valid = false;
  h->capBp = 0;
  h->capBp16 = 0;
  for (auto& p : h->pending) {
    (void)hipEventDestroy(p.a);
    (void)hipEventDestroy(p.b);
  }
  h->pending.clear();
  for (auto e : h->ev_free) (void)hipEventDestroy(e);
  h->ev_free.clear();
}

int take_event(pmlp* h, hipEvent_t* e) {
  if (!h->ev_free.empty()) {
    *e = h->ev_free.back();
    h->ev_free.pop_back();
    return PMLP_OK;
  }
  PMLP_HIP(hipEventCreate(e));
  return PMLP_OK;
}

// Launch `fn` (returning hipError_t) as kernel `kid`, bracketed by events
// when profiling is on.
template <class Fn>
int run(pmlp* h, int kid, Fn fn) {
  hipEvent_t a = nullptr, b = nullptr;
  if (h->prof) {
    int rc = take_event(h, &a);
    if (rc) return rc;
    rc = take_event(h, &b);
    if (rc) return rc;
    PMLP_HIP(hipEventRecord(a, h->stream));
  }
  note_variant("", kArithNone);
  hipError_t e = fn();
  if (e != hipSuccess)
    return fail(PMLP_EDEVICE, std::string("launch of ") + kKernelNames[kid] +
                                  " failed: " + hipGetErrorString(e));
  if (last_variant().name[0]) h->variant[kid] = last_variant();
  if (h->prof) {
    PMLP_HIP(hipEventRecord(b, h->stream));
    h->pending.push_back({kid, a, b});
  }
  return PMLP_OK;
}

int use_device(pmlp* h) {
  int cur = -1;
  PMLP_HIP(hipGetDevice(&cur));
  if (cur != h->dev) PMLP_HIP(hipSetDevice(h->dev));
  return PMLP_OK;
}

int ensure_workspace(pmlp* h, int32_t Bp) {
  if (Bp <= h->capBp) return PMLP_OK;
  PMLP_HIP(hipStreamSynchronize(h->stream));
  dfree(h->Xp);
  dfree(h->Xt);
  dfree(h->Zt);
  dfree(h->LG);
  h->capBp = 0;
  const size_t nx = (size_t)Bp * h->F4 * sizeof(float);
  const size_t nz = (size_t)h->Npad * Bp * sizeof(float);
  const size_t nl = (size_t)h->M * Bp * h->O * sizeof(float);
  if (hipMalloc(&h->Xp, nx) != hipSuccess || hipMalloc(&h->Xt, nx) != hipSuccess ||
      hipMalloc(&h->Zt, nz) != hipSuccess || hipMalloc(&h->LG, nl) != hipSuccess) {
    (void)hipGetLastError();
    dfree(h->Xp);
    dfree(h->Xt);
    dfree(h->Zt);
    dfree(h->LG);
    return fail(PMLP_ENOMEM, "workspace allocation failed for batch " + std::to_string(Bp) +
                                 " (" + std::to_string((nz + 2 * nx + nl) >> 20) + " MiB)");
  }
  h->capBp = Bp;
  return PMLP_OK;
}

// The per-batch workspaces of a step: the batch copies, the hidden
// pre-activations and the logits (overwritten by dLoss/dlogits).
struct Work {
  float* Xp;  // [Bp][F4]
  float* Xt;  // [F4][Bp]
  float* Zt;  // [Npad][Bp]
  float* LG;  // [M][Bp][O]
};

Work handle_work(const pmlp* h) { return Work{h->Xp, h->Xt, h->Zt, h->LG}; }

size_t align256(size_t n) { return (n + 255) & ~(size_t)255; }

// Bytes of the four workspaces of a Bp-sample batch, each 256-byte aligned.
size_t work_bytes(const pmlp* h, int32_t Bp) {
  return 2 * align256((size_t)Bp * h->F4 * sizeof(float)) +
         align256((size_t)h->Npad * Bp * sizeof(float)) +
         align256((size_t)h->M * Bp * h->O * sizeof(float));
}

// Device address of the static workspace on the current device `dev`.
int scratch_base(int dev, unsigned char** out) {
  if (dev < 0 || dev >= kMaxDevices) return fail(PMLP_EDEVICE, "device index out of range");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return fail(PMLP_EDEVICE, std::string("hipGetSymbolAddress of the static workspace failed: ") +
                                    hipGetErrorString(e));
    g_scratch_ptr[dev] = p;
  }
  *out = (unsigned char*)g_scratch_ptr[dev];
  return PMLP_OK;
}

// The workspaces of a Bp-sample batch laid out in the static workspace.
Work carve_work(const pmlp* h, int32_t Bp, unsigned char* base) {
  Work w{};
  size_t at = 0;
  auto take = [&](size_t n) {
    float* p = (float*)(base + at);
    at += align256(n);
    return p;
  };
  w.Xp = take((size_t)Bp * h->F4 * sizeof(float));
  w.Xt = take((size_t)Bp * h->F4 * sizeof(float));
  w.Zt = take((size_t)h->Npad * Bp * sizeof(float));
  w.LG = take((size_t)h->M * Bp * h->O * sizeof(float));
  return w;
}

// bf16 copies of the batch, allocated on the first bf16-mode call.
int ensure_workspace_bf16(pmlp* h, int32_t Bp) {
  if (Bp <= h->capBp16) return PMLP_OK;
  PMLP_HIP(hipStreamSynchronize(h->stream));
  dfree(h->Xp16);
  dfree(h->Xt16);
  dfree(h->dZ16);
  h->capBp16 = 0;
  const size_t np = (size_t)Bp * bf16_ld(h->F4) * 2;
  const size_t nt = (size_t)h->F4 * bf16_ld(Bp) * 2;
  const size_t nd = (size_t)h->Npad * Bp * 2;
  if (hipMalloc(&h->Xp16, np) != hipSuccess || hipMalloc(&h->Xt16, nt) != hipSuccess ||
      hipMalloc(&h->dZ16, nd) != hipSuccess) {
    (void)hipGetLastError();
    dfree(h->Xp16);
    dfree(h->Xt16);
    dfree(h->dZ16);
    return fail(PMLP_ENOMEM, "bf16 workspace allocation failed for batch " + std::to_string(Bp));
  }
  h->capBp16 = Bp;
  return PMLP_OK;
}

// Both bf16 modes round the operands of the input-layer products; the
// storage mode also keeps Z as bfloat16 (in the first half of Zt).
bool bf16_mode(const pmlp* h) { return h->precision != PMLP_FP32; }
bool z_bf16(const pmlp* h) { return h->precision == PMLP_BF16_STORE; }

// The bf16 copy of W1 read by the bf16 input-to-hidden product: allocated
// on first use, rebuilt whenever W1 changed outside a bf16-mode SGD step
// (whose update epilogue keeps it current).
int ensure_w1b(pmlp* h) {
  if (!h->W1b) {
    const size_t n = (size_t)h->Npad * bf16_ld(h->F4) * 2;
    if (hipMalloc(&h->W1b, n) != hipSuccess) {
      (void)hipGetLastError();
      h->W1b = nullptr;
      return fail(PMLP_ENOMEM, "bf16 weight copy allocation failed (" +
                                   std::to_string(n >> 20) + " MiB)");
    }
    h->w1b_valid = false;
  }
  if (!h->w1b_valid) {
    if (int rc = run(h, KID_AUX, [&] {
          return launch_w1_to_bf16(h->W1, h->Npad, h->F4, h->W1b, bf16_ld(h->F4), h->stream);
        }))
      return rc;
    h->w1b_valid = true;
  }
  return PMLP_OK;
}

int check_handle(pmlp* h) {
  if (!h) return fail(PMLP_EINVAL, "null handle");
  return PMLP_OK;
}

// Calls that a pack with two hidden layers does not provide.
int one_layer_only(pmlp* h, const char* what) {
  if (h->deep)
    return fail(PMLP_ESTATE, std::string(what) + " is not provided for a pack with two hidden "
                                                 "layers");
  return PMLP_OK;
}

int check_batch(pmlp* h, const void* X, int32_t B) {
  if (int rc = check_handle(h)) return rc;
  if (!X) return fail(PMLP_EINVAL, "null X");
  if (B < 1 || B > kMaxBatch) return fail(PMLP_EINVAL, "batch size out of range [1, 2^20]");
  return PMLP_OK;
}

// Batch padding: a multiple of 16, and a power of two up to 256 so that the
// LDS-resident forward GEMM has an instance for it.
int32_t pad_batch(int32_t B) {
  int32_t Bp = (B + 15) & ~15;
  if (Bp <= 256) {
    int32_t p = 16;
    while (p < Bp) p <<= 1;
    Bp = p;
  }
  return Bp;
}

// Batch copy and the input-to-hidden product (Section 3, step 1).
int forward_hidden(pmlp* h, const float* X, int32_t B, int32_t Bp, const Work& w) {
  if (bf16_mode(h)) {
    if (int rc = ensure_workspace_bf16(h, Bp)) return rc;
    if (int rc = ensure_w1b(h)) return rc;
    if (int rc = run(h, KID_PACK_X, [&] {
          return launch_pack_x_bf16(X, B, h->F, Bp, h->F4, h->bcol, h->Xp16, h->Xt16,
                                    h->stream);
        }))
      return rc;
    GemmBfArgs g{};
    g.Pb = h->W1b;
    g.ldp = bf16_ld(h->F4);
    g.kp = bf16_ld(h->F4);  // zero past F4
    g.NP = h->N;
    g.Q = h->Xp16;
    g.ldq = bf16_ld(h->F4);
    g.NQ = Bp;
    g.K = h->F4;
    g.out = w.Zt;
    g.ldo = Bp;
    g.ncols = Bp;
    if (z_bf16(h)) {
      g.outb = (unsigned short*)w.Zt;
      g.ldob = Bp;
    }
    return run(h, KID_GEMM_FWD, [&] { return launch_gemm_bf16(g, EPI_STORE, h->stream); });
  }
  if (int rc = run(h, KID_PACK_X, [&] {
        return launch_pack_x(X, B, h->F, Bp, h->F4, h->bcol, w.Xp, w.Xt, h->stream);
      }))
    return rc;
  if (h->lds_kernels && fwd_lds_supported(Bp, h->F4)) {
    FwdLdsArgs f{};
    f.W1 = h->W1;
    f.Xp = w.Xp;
    f.Zt = w.Zt;
    f.N = h->N;
    f.Bp = Bp;
    f.K = h->F4;
    return run(h, KID_GEMM_FWD, [&] { return launch_fwd_lds(f, h->stream); });
  }
  if (h->lds_kernels) {  // fp32 accuracy on the bf16 matrix cores
    GemmBfArgs g{};
    g.P = h->W1;
    g.ldp = h->F4;
    g.kp = h->F4;
    g.NP = h->N;
    g.Qf = w.Xp;
    g.ldq = h->F4;
    g.NQ = Bp;
    g.K = h->F4;
    g.out = w.Zt;
    g.ldo = Bp;
    g.ncols = Bp;
    return run(h, KID_GEMM_FWD, [&] { return launch_gemm_bf16(g, EPI_STORE, h->stream); });
  }
  GemmArgs g{};
  g.P = h->W1;
  g.ldp = h->F4;
  g.NP = h->N;
  g.Q = w.Xp;
  g.ldq = h->F4;
  g.NQ = Bp;
  g.K = h->F4;
  g.out = w.Zt;
  g.ldo = Bp;
  g.ncols = Bp;
  g.lr = 0.f;
  return run(h, KID_GEMM_FWD, [&] { return launch_gemm(g, EPI_STORE, h->stream); });
}

// Whether the forward runs as one kernel: the input-to-hidden product with
// the activation and the M3 forward in its epilogue.
bool forward_fused(const pmlp* h, int32_t Bp) {
  return h->lds_kernels && h->fused_forward && !bf16_mode(h) && !h->deep &&
         fwd_m3_supported(Bp, h->F4, h->O);
}

// Batch copy and the whole forward of Section 3 (steps 1-4) in one kernel:
// Zt and the logits out[m*sm + b*sb + o] (cleared first where the halves
// of a wide segment add atomically).
int forward_m3(pmlp* h, const float* X, int32_t B, int32_t Bp, const Work& w, float* out,
               int64_t sm, int64_t sb, int64_t nout) {
  if (int rc = run(h, KID_PACK_X, [&] {
        return launch_pack_x(X, B, h->F, Bp, h->F4, h->bcol, w.Xp, w.Xt, h->stream);
      }))
    return rc;
  if (h->has_split) {
    if (int rc = run(h, KID_AUX, [&] { return launch_fill(out, nout, 0.f, h->stream); })) return rc;
  }
  FwdM3Args f{};
  f.W1 = h->W1;
  f.Xp = w.Xp;
  f.Zt = w.Zt;
  f.N = h->N;
  f.Bp = Bp;
  f.K = h->F4;
  f.B = B;
  f.O = h->O;
  f.W2 = h->W2;
  f.ldw = h->Npad;
  f.seg_off = h->d_seg_off;
  f.act = h->d_act;
  f.tiles = h->d_tiles;
  f.order = h->d_order;
  f.ntiles = h->ntiles;
  f.b2 = h->b2;
  f.out = out;
  f.sm = sm;
  f.sb = sb;
  return run(h, KID_FWD_M3, [&] { return launch_fwd_m3(f, h->stream); });
}

// Full step: forward, loss, backward and either the SGD update (dW1 and
// dW2 null) or gradient stores.
// With `work` set, the step runs in those workspaces (sized for the batch by
// the caller) and allocates nothing; otherwise in the handle's, grown as
// needed.
int step(pmlp* h, const float* X, const void* y, int32_t B, float lr, const float* lrm,
         float* dW1, float* dW2, float* db1 = nullptr, float* db2 = nullptr,
         const Work* work = nullptr) {
  const int32_t Bp = pad_batch(B);
  if (int rc = use_device(h)) return rc;
  if (!work)
    if (int rc = ensure_workspace(h, Bp)) return rc;
  const Work w = work ? *work : handle_work(h);
  if (forward_fused(h, Bp)) {
    if (int rc = forward_m3(h, X, B, Bp, w, w.LG, (int64_t)Bp * h->O, h->O,
                            (int64_t)h->M * Bp * h->O))
      return rc;
  } else {
    if (int rc = forward_hidden(h, X, B, Bp, w)) return rc;
    if (h->has_split) {
      if (int rc = run(h, KID_AUX, [&] {
            return launch_fill(w.LG, (int64_t)h->M * Bp * h->O, 0.f, h->stream);
          }))
        return rc;
    }
    if (int rc = run(h, KID_M3_FWD, [&] {
          return launch_m3_fwd(w.Zt, Bp, B, h->W2, h->Npad, h->O, h->d_seg_off, h->d_act,
                               h->d_tiles, h->d_order, h->ntiles, h->b2, w.LG, (int64_t)Bp * h->O,
                               h->O, h->stream, z_bf16(h));
        }))
      return rc;
  }
  // an fp32-mode update leaves the bf16 copy of W1 behind
  if (!bf16_mode(h) && !dW1) h->w1b_valid = false;
  if (int rc = run(h, KID_CE, [&] {
        // output biases: updated here (db2 = sum_b G), or their gradient stored
        float* b2 = dW1 ? (db2 ? h->b2 : nullptr) : h->b2;
        float* g2 = dW1 ? db2 : nullptr;
        const float* rates = dW1 ? nullptr : lrm;
        if (h->mse)
          return launch_mse(w.LG, (const float*)y, h->M, Bp, B, h->O, h->loss, h->flag, rates,
                            b2, g2, lr, h->stream);
        return launch_ce(w.LG, (const int32_t*)y, h->M, Bp, B, h->O, h->loss, h->flag, rates,
                         b2, g2, lr, h->stream);
      }))
    return rc;
  if (h->lds_kernels && !bf16_mode(h) && bwd_lds_supported(Bp, h->F4, h->O)) {
    BwdArgs b{};
    b.Zt = w.Zt;
    b.G = w.LG;
    b.Xt = w.Xt;
    b.mid = h->d_mid;
    b.actn = h->d_actn;
    b.W1 = h->W1;
    b.W2 = h->W2;
    b.dW1 = dW1;
    b.dW2 = dW2;
    b.N = h->N;
    b.ldw = h->Npad;
    b.Bp = Bp;
    b.F = h->F;
    b.F4 = h->F4;
    b.O = h->O;
    b.lr = lr;
    b.lrm = lrm;
    b.db1 = dW1 ? db1 : nullptr;
    b.bcol = h->bcol;
    b.fmask = h->d_fmask;
    b.fmw = h->fmw;
    if (int rc = run(h, KID_BWD_FUSED, [&] { return launch_bwd_lds(b, h->stream); })) return rc;
    h->have_loss = true;
    return PMLP_OK;
  }
  if (int rc = run(h, KID_M3_BWD, [&] {
        return launch_m3_bwd(w.Zt, bf16_mode(h) ? h->dZ16 : nullptr, Bp, h->W2, h->N, h->Npad,
                             h->O, h->d_mid, h->d_seg_off,
                             h->d_act, w.LG, lr, lrm, dW2, h->stream, z_bf16(h));
      }))
    return rc;
  if (bf16_mode(h)) {
    GemmBfArgs g{};
    g.Pb = h->dZ16;
    g.ldp = Bp;
    g.kp = Bp;
    g.NP = h->N;
    g.Q = h->Xt16;
    g.ldq = bf16_ld(Bp);
    g.NQ = h->F4;
    g.K = Bp;
    g.out = dW1 ? dW1 : h->W1;
    g.ldo = dW1 ? h->F : h->F4;
    g.ncols = h->F;
    g.lr = lr;
    g.lrm = lrm;
    g.mid = h->d_mid;
    g.db1 = dW1 ? db1 : nullptr;
    g.bcol = h->bcol;
    g.outb = dW1 ? nullptr : h->W1b;  // the update keeps the bf16 copy current
    g.ldob = bf16_ld(h->F4);
    g.fmask = h->d_fmask;
    g.fmw = h->fmw;
    if (int rc = run(h, KID_GEMM_BWD, [&] {
          return launch_gemm_bf16(g, dW1 ? EPI_GRAD : EPI_SGD, h->stream);
        }))
      return rc;
    h->have_loss = true;
    return PMLP_OK;
  }
  if (h->lds_kernels) {  // fp32 accuracy on the bf16 matrix cores
    GemmBfArgs g{};
    g.P = w.Zt;
    g.ldp = Bp;
    g.kp = Bp;
    g.NP = h->N;
    g.Qf = w.Xt;
    g.ldq = Bp;
    g.NQ = h->F4;
    g.K = Bp;
    g.out = dW1 ? dW1 : h->W1;
    g.ldo = dW1 ? h->F : h->F4;
    g.ncols = h->F;
    g.lr = lr;
    g.lrm = lrm;
    g.mid = h->d_mid;
    g.db1 = dW1 ? db1 : nullptr;
    g.bcol = h->bcol;
    g.fmask = h->d_fmask;
    g.fmw = h->fmw;
    if (int rc = run(h, KID_GEMM_BWD, [&] {
          return launch_gemm_bf16(g, dW1 ? EPI_GRAD : EPI_SGD, h->stream);
        }))
      return rc;
    h->have_loss = true;
    return PMLP_OK;
  }
  GemmArgs g{};
  g.P = w.Zt;
  g.ldp = Bp;
  g.NP = h->N;
  g.Q = w.Xt;
  g.ldq = Bp;
  g.NQ = h->F4;
  g.K = Bp;
  g.out = dW1 ? dW1 : h->W1;
  g.ldo = dW1 ? h->F : h->F4;
  g.ncols = h->F;
  g.lr = lr;
  g.lrm = lrm;
  g.mid = h->d_mid;
  g.db1 = dW1 ? db1 : nullptr;
  g.bcol = h->bcol;
  g.fmask = h->d_fmask;
  g.fmw = h->fmw;
  if (int rc = run(h, KID_GEMM_BWD, [&] {
        return launch_gemm(g, dW1 ? EPI_GRAD : EPI_SGD, h->stream);
      }))
    return rc;
  h->have_loss = true;
  return PMLP_OK;
}

// Second-layer workspace of a pack with two hidden layers.
int ensure_deep_workspace(pmlp* h, int32_t Bp) {
  PmlpDeep* d = h->deep;
  if (Bp <= d->capBp) return PMLP_OK;
  PMLP_HIP(hipStreamSynchronize(h->stream));
  dfree(d->Zt2);
  d->capBp = 0;
  const size_t n = (size_t)d->N2pad * Bp * sizeof(float);
  if (hipMalloc(&d->Zt2, n) != hipSuccess) {
    (void)hipGetLastError();
    d->Zt2 = nullptr;
    return fail(PMLP_ENOMEM, "second-layer workspace allocation failed for batch " +
                                 std::to_string(Bp) + " (" + std::to_string(n >> 20) + " MiB)");
  }
  d->capBp = Bp;
  return PMLP_OK;
}

DeepArgs deep_args(const pmlp* h) {
  const PmlpDeep* d = h->deep;
  return DeepArgs{d->d_off1, d->d_off2, d->d_koff, d->d_h1, d->d_h2, h->d_act, d->W12};
}

// Forward of a pack with two hidden layers up to the second layer's
// pre-activations: Z1 = X W1^T (the one-layer product), then per model
// Z2 = W12 act(Z1) (Section 7, Figure 3).
int forward_deep(pmlp* h, const float* X, int32_t B, int32_t Bp, const Work& w) {
  PmlpDeep* d = h->deep;
  if (int rc = forward_hidden(h, X, B, Bp, w)) return rc;
  const DeepArgs a = deep_args(h);
  return run(h, KID_DEEP, [&] {
    return launch_seg_fwd(w.Zt, d->Zt2, Bp, a, d->d_ufwd, d->nufwd, h->stream);
  });
}

// One step of a pack with two hidden layers: forward, loss, backward and
// the SGD update (dW1 null) or the gradient stores.
int step_deep(pmlp* h, const float* X, const int32_t* y, int32_t B, float lr, float* dW1,
              float* dW12, float* dW2) {
  PmlpDeep* d = h->deep;
  const int32_t Bp = pad_batch(B);
  if (int rc = use_device(h)) return rc;
  if (int rc = ensure_workspace(h, Bp)) return rc;
  if (int rc = ensure_deep_workspace(h, Bp)) return rc;
  const Work w = handle_work(h);
  if (int rc = forward_deep(h, X, B, Bp, w)) return rc;
  if (d->has_split2) {
    if (int rc = run(h, KID_AUX, [&] {
          return launch_fill(w.LG, (int64_t)h->M * Bp * h->O, 0.f, h->stream);
        }))
      return rc;
  }
  if (int rc = run(h, KID_M3_FWD, [&] {
        return launch_m3_fwd(d->Zt2, Bp, B, h->W2, d->N2pad, h->O, d->d_off2, h->d_act,
                             d->d_tiles2, d->d_order2, d->ntiles2, nullptr, w.LG,
                             (int64_t)Bp * h->O, h->O, h->stream);
      }))
    return rc;
  if (int rc = run(h, KID_CE, [&] {
        return launch_ce(w.LG, y, h->M, Bp, B, h->O, h->loss, h->flag, nullptr, nullptr, nullptr,
                         lr, h->stream);
      }))
    return rc;
  // dZ2 over Z2 in place; W2 updated (or dW2 stored)
  if (int rc = run(h, KID_M3_BWD, [&] {
        return launch_m3_bwd(d->Zt2, nullptr, Bp, h->W2, d->N2, d->N2pad, h->O, d->d_mid2,
                             d->d_off2, h->d_act, w.LG, lr, nullptr, dW2, h->stream);
      }))
    return rc;
  const DeepArgs a = deep_args(h);
  float* g12 = dW1 ? dW12 : d->G12;
  if (int rc = run(h, KID_DEEP, [&] {
        return launch_seg_grad(w.Zt, d->Zt2, Bp, a, d->d_tgrad, d->ntgrad, g12, h->stream);
      }))
    return rc;
  // dZ1 over Z1 in place, from the W12 of before this step
  if (int rc = run(h, KID_DEEP, [&] {
        return launch_seg_back(w.Zt, d->Zt2, Bp, a, d->d_uback, d->nuback, h->stream);
      }))
    return rc;
  if (!dW1) {
    if (int rc = run(h, KID_DEEP, [&] { return launch_sgd(d->W12, d->G12, d->K, lr, h->stream); }))
      return rc;
  }
  if (h->lds_kernels) {  // fp32 accuracy on the bf16 matrix cores
    GemmBfArgs g{};
    g.P = w.Zt;
    g.ldp = Bp;
    g.kp = Bp;
    g.NP = h->N;
    g.Qf = w.Xt;
    g.ldq = Bp;
    g.NQ = h->F4;
    g.K = Bp;
    g.out = dW1 ? dW1 : h->W1;
    g.ldo = dW1 ? h->F : h->F4;
    g.ncols = h->F;
    g.lr = lr;
    g.mid = h->d_mid;
    g.bcol = -1;
    if (int rc = run(h, KID_GEMM_BWD, [&] {
          return launch_gemm_bf16(g, dW1 ? EPI_GRAD : EPI_SGD, h->stream);
        }))
      return rc;
    h->have_loss = true;
    return PMLP_OK;
  }
  GemmArgs g{};
  g.P = w.Zt;
  g.ldp = Bp;
  g.NP = h->N;
  g.Q = w.Xt;
  g.ldq = Bp;
  g.NQ = h->F4;
  g.K = Bp;
  g.out = dW1 ? dW1 : h->W1;
  g.ldo = dW1 ? h->F : h->F4;
  g.ncols = h->F;
  g.lr = lr;
  g.mid = h->d_mid;
  g.bcol = -1;
  if (int rc = run(h, KID_GEMM_BWD, [&] {
        return launch_gemm(g, dW1 ? EPI_GRAD : EPI_SGD, h->stream);
      }))
    return rc;
  h->have_loss = true;
  return PMLP_OK;
}

// Tiles of the M3 forward: runs of whole segments up to `cap` units wide;
// a wider segment becomes two halves added with atomics onto zeroed logits.
// Two additions onto zero give the same sum in either order, so the
// forward is deterministic for every segment width.  The cap is the power
// of two in [kTile3Min, kTile3] nearest below N / kTile3Count, so that a
// small pack still gives the M3 forward a few thousand waves.
int64_t tile_cap(int64_t N) {
  int64_t cap = kTile3;
  while (cap > kTile3Min && cap * kTile3Count > N) cap >>= 1;
  return cap;
}

void build_tiles(const std::vector<int32_t>& hs, int64_t cap, std::vector<Tile3>& tiles,
                 bool& has_split) {
  tiles.clear();
  has_split = false;
  Tile3 cur{0, 0, 0, 0, 0};
  int64_t n = 0;
  for (size_t m = 0; m < hs.size(); ++m) {
    const int64_t w = hs[m];
    if (w > cap) {
      if (cur.len > 0) tiles.push_back(cur);
      cur.len = 0;
      const int64_t half = (w + 1) / 2;
      tiles.push_back(Tile3{n, (int32_t)half, (int32_t)m, 1, 0});
      tiles.push_back(Tile3{n + half, (int32_t)(w - half), (int32_t)m, 1, 0});
      has_split = true;
    } else {
      if (cur.len > 0 && cur.len + w > cap) {
        tiles.push_back(cur);
        cur.len = 0;
      }
      if (cur.len == 0) cur = Tile3{n, 0, (int32_t)m, 0, 0};
      cur.len += (int32_t)w;
    }
    n += w;
  }
  if (cur.len > 0) tiles.push_back(cur);
}

}  // namespace

extern "C" {

int pmlp_create(pmlp_t* out, int32_t F, int32_t O, int32_t M, const int32_t* hidden_sizes,
                const int32_t* act_ids, uint64_t seed) {
  return pmlp_create_ex(out, F, O, M, hidden_sizes, act_ids, seed, 0);
}

int pmlp_create_ex(pmlp_t* out, int32_t F, int32_t O, int32_t M, const int32_t* hidden_sizes,
                   const int32_t* act_ids, uint64_t seed, int32_t flags) {
  if (!out) return fail(PMLP_EINVAL, "null output handle pointer");
  *out = nullptr;
  if (flags & ~(PMLP_BIAS | PMLP_MSE)) return fail(PMLP_EINVAL, "unknown flags");
  const bool biases = (flags & PMLP_BIAS) != 0;
  if (F < 1) return fail(PMLP_EINVAL, "F must be >= 1");
  if (O < 2 || O > kMaxO) return fail(PMLP_EINVAL, "O must be in [2, 16]");
  if (M < 1) return fail(PMLP_EINVAL, "M must be >= 1");
  if (!hidden_sizes || !act_ids) return fail(PMLP_EINVAL, "null hidden_sizes or act_ids");
  int64_t N = 0;
  for (int32_t m = 0; m < M; ++m) {
    if (hidden_sizes[m] < 1) return fail(PMLP_EINVAL, "hidden size < 1 at model " + std::to_string(m));
    if (act_ids[m] < 0 || act_ids[m] >= PMLP_NUM_ACTS)
      return fail(PMLP_EINVAL, "activation id out of range at model " + std::to_string(m));
    N += hidden_sizes[m];
  }
  if (N > ((int64_t)1 << 31) - 1) return fail(PMLP_EINVAL, "total hidden units exceed 2^31-1");
  // With biases the input gets a constant 1 at column bcol = F rounded up
  // to 4, whose weight is the hidden bias; rows are then 4 floats longer.
  const int32_t bcol = biases ? (F + 3) & ~3 : -1;
  const int32_t F4 = ((F + 3) & ~3) + (biases ? 4 : 0);

  pmlp* h = new (std::nothrow) pmlp();
  if (!h) return fail(PMLP_ENOMEM, "host allocation failed");
  h->F = F;
  h->F4 = F4;
  h->mse = (flags & PMLP_MSE) != 0;
  h->bcol = bcol;
  h->O = O;
  h->M = M;
  h->N = N;
  h->Npad = (N + 63) / 64 * 64;
  if (const char* env = getenv("PMLP_GENERIC_KERNELS")) h->lds_kernels = env[0] == '0';
  if (const char* env = getenv("PMLP_FUSED_FORWARD")) h->fused_forward = env[0] == '1';
  h->hs.assign(hidden_sizes, hidden_sizes + M);
  h->acts.assign(act_ids, act_ids + M);
  h->seg_off.resize((size_t)M + 1);
  h->seg_off[0] = 0;
  for (int32_t m = 0; m < M; ++m) h->seg_off[m + 1] = h->seg_off[m] + hidden_sizes[m];
  std::vector<int32_t> mid((size_t)h->Npad, M - 1);  // padding rows map to the last model
  std::vector<int32_t> actn((size_t)h->Npad, act_ids[M - 1]);
  for (int32_t m = 0; m < M; ++m)
    for (int64_t n = h->seg_off[m]; n < h->seg_off[m + 1]; ++n) {
      mid[n] = m;
      actn[n] = act_ids[m];
    }
  std::vector<Tile3> tiles;
  build_tiles(h->hs, tile_cap(N), tiles, h->has_split);
  h->ntiles = (int32_t)tiles.size();
  // the M3 forward launches its waves widest tile first (ties in plan order),
  // so the dispatcher schedules the longest work first
  std::vector<int32_t> order(tiles.size());
  for (size_t i = 0; i < order.size(); ++i) order[i] = (int32_t)i;
  std::stable_sort(order.begin(), order.end(),
                   [&](int32_t x, int32_t y) { return tiles[x].len > tiles[y].len; });
  std::vector<float> bound2((size_t)M);
  for (int32_t m = 0; m < M; ++m) bound2[m] = (float)(1.0 / std::sqrt((double)hidden_sizes[m]));
  const float bound1 = (float)(1.0 / std::sqrt((double)F));

  auto bail = [&](int rc) {
    release(h);
    delete h;
    return rc;
  };
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) {
    (void)hipGetLastError();
    return bail(fail(PMLP_EDEVICE, "no HIP device available"));
  }
  h->dev = dev;
  float* d_bound2 = nullptr;
  const int64_t Npad = h->Npad;
  const size_t w1_bytes = ((size_t)Npad * F4 + 64) * sizeof(float);  // slack for clamped loads
  if (hipMalloc(&h->W1, w1_bytes) != hipSuccess ||
      hipMalloc(&h->W2, (size_t)O * Npad * sizeof(float)) != hipSuccess ||
      hipMalloc(&h->d_seg_off, ((size_t)M + 1) * sizeof(int64_t)) != hipSuccess ||
      hipMalloc(&h->d_act, (size_t)M * sizeof(int32_t)) != hipSuccess ||
      hipMalloc(&h->d_mid, (size_t)Npad * sizeof(int32_t)) != hipSuccess ||
      hipMalloc(&h->d_actn, (size_t)Npad * sizeof(int32_t)) != hipSuccess ||
      hipMalloc(&h->d_tiles, tiles.size() * sizeof(Tile3)) != hipSuccess ||
      hipMalloc(&h->d_order, order.size() * sizeof(int32_t)) != hipSuccess ||
      hipMalloc(&h->loss, (size_t)M * sizeof(float)) != hipSuccess ||
      hipMalloc(&h->flag, 4 * sizeof(int32_t)) != hipSuccess ||
      hipMalloc(&d_bound2, (size_t)M * sizeof(float)) != hipSuccess ||
      (biases && hipMalloc(&h->b2, (size_t)M * O * sizeof(float)) != hipSuccess)) {
    (void)hipGetLastError();
    dfree(d_bound2);
    return bail(fail(PMLP_ENOMEM, "device allocation failed for the packed parameters"));
  }
  auto setup = [&]() -> int {
    PMLP_HIP(hipMemcpy(h->d_seg_off, h->seg_off.data(), ((size_t)M + 1) * sizeof(int64_t),
                       hipMemcpyHostToDevice));
    PMLP_HIP(hipMemcpy(h->d_act, act_ids, (size_t)M * sizeof(int32_t), hipMemcpyHostToDevice));
    PMLP_HIP(hipMemcpy(h->d_mid, mid.data(), (size_t)Npad * sizeof(int32_t),
                       hipMemcpyHostToDevice));
    PMLP_HIP(hipMemcpy(h->d_actn, actn.data(), (size_t)Npad * sizeof(int32_t),
                       hipMemcpyHostToDevice));
    PMLP_HIP(hipMemset(h->W1, 0, w1_bytes));
    PMLP_HIP(hipMemset(h->W2, 0, (size_t)O * Npad * sizeof(float)));
    PMLP_HIP(hipMemcpy(h->d_tiles, tiles.data(), tiles.size() * sizeof(Tile3),
                       hipMemcpyHostToDevice));
    PMLP_HIP(hipMemcpy(h->d_order, order.data(), order.size() * sizeof(int32_t),
                       hipMemcpyHostToDevice));
    PMLP_HIP(hipMemcpy(d_bound2, bound2.data(), (size_t)M * sizeof(float), hipMemcpyHostToDevice));
    PMLP_HIP(hipMemset(h->flag, 0, 4 * sizeof(int32_t)));
    PMLP_HIP(launch_init_params(h->W1, N, F, F4, bound1, h->W2, Npad, O, h->d_mid, d_bound2,
                                splitmix64_host(seed), nullptr));
    if (biases)
      PMLP_HIP(launch_init_biases(h->W1, N, F4, bcol, bound1, h->b2, M, O, d_bound2,
                                  splitmix64_host(seed), nullptr));
    PMLP_HIP(hipStreamSynchronize(nullptr));
    return PMLP_OK;
  };
  int rc = setup();
  dfree(d_bound2);
  if (rc) return bail(rc);
  *out = h;
  return PMLP_OK;
}

int pmlp_destroy(pmlp_t h) {
  if (!h) return PMLP_OK;
  (void)hipSetDevice(h->dev);
  (void)hipStreamSynchronize(h->stream);
  release(h);
  delete h;
  return PMLP_OK;
}

int pmlp_set_stream(pmlp_t h, void* stream) {
  if (int rc = check_handle(h)) return rc;
  if (stream) {
    int sdev = -1;
    PMLP_HIP(hipStreamGetDevice((hipStream_t)stream, &sdev));
    if (sdev != h->dev)
      return fail(PMLP_EINVAL, "the stream belongs to device " + std::to_string(sdev) +
                                   ", the handle to device " + std::to_string(h->dev));
  }
  h->stream = (hipStream_t)stream;
  return PMLP_OK;
}

int pmlp_set_precision(pmlp_t h, int32_t mode) {
  if (int rc = check_handle(h)) return rc;
  if (mode != PMLP_FP32 && mode != PMLP_BF16_GEMM && mode != PMLP_BF16_STORE)
    return fail(PMLP_EINVAL, "unknown precision mode");
  if (mode != PMLP_FP32)
    if (int rc = one_layer_only(h, "the bf16 modes")) return rc;
  h->precision = mode;
  return PMLP_OK;
}

int pmlp_forward(pmlp_t h, const float* X_dev, int32_t B, float* logits_dev) {
  if (int rc = check_batch(h, X_dev, B)) return rc;
  if (!logits_dev) return fail(PMLP_EINVAL, "null logits");
  const int32_t Bp = pad_batch(B);
  if (int rc = use_device(h)) return rc;
  if (int rc = ensure_workspace(h, Bp)) return rc;
  if (PmlpDeep* d = h->deep) {
    if (int rc = ensure_deep_workspace(h, Bp)) return rc;
    if (int rc = forward_deep(h, X_dev, B, Bp, handle_work(h))) return rc;
    if (d->has_split2) {
      if (int rc = run(h, KID_AUX, [&] {
            return launch_fill(logits_dev, (int64_t)B * h->M * h->O, 0.f, h->stream);
          }))
        return rc;
    }
    return run(h, KID_M3_FWD, [&] {
      return launch_m3_fwd(d->Zt2, Bp, B, h->W2, d->N2pad, h->O, d->d_off2, h->d_act, d->d_tiles2,
                           d->d_order2, d->ntiles2, nullptr, logits_dev, h->O,
                           (int64_t)h->M * h->O, h->stream);
    });
  }
  if (forward_fused(h, Bp))
    return forward_m3(h, X_dev, B, Bp, handle_work(h), logits_dev, h->O, (int64_t)h->M * h->O,
                      (int64_t)B * h->M * h->O);
  if (int rc = forward_hidden(h, X_dev, B, Bp, handle_work(h))) return rc;
  if (h->has_split) {
    if (int rc = run(h, KID_AUX, [&] {
          return launch_fill(logits_dev, (int64_t)B * h->M * h->O, 0.f, h->stream);
        }))
      return rc;
  }
  return run(h, KID_M3_FWD, [&] {
    return launch_m3_fwd(h->Zt, Bp, B, h->W2, h->Npad, h->O, h->d_seg_off, h->d_act, h->d_tiles,
                         h->d_order, h->ntiles, h->b2, logits_dev, h->O, (int64_t)h->M * h->O,
                         h->stream, z_bf16(h));
  });
}

int pmlp_train_step(pmlp_t h, const float* X_dev, const int32_t* y_dev, int32_t B, float lr) {
  if (int rc = check_batch(h, X_dev, B)) return rc;
  if (h->mse) return fail(PMLP_ESTATE, "a regression handle trains with pmlp_train_step_mse");
  if (!y_dev) return fail(PMLP_EINVAL, "null labels");
  if (!std::isfinite(lr)) return fail(PMLP_EINVAL, "learning rate is not finite");
  if (h->deep) return step_deep(h, X_dev, y_dev, B, lr, nullptr, nullptr, nullptr);
  return step(h, X_dev, y_dev, B, lr, nullptr, nullptr, nullptr);
}

int pmlp_train_step_noalloc(pmlp_t h, const float* X_dev, const int32_t* y_dev, int32_t B,
                            float lr) {
  if (int rc = check_batch(h, X_dev, B)) return rc;
  if (int rc = one_layer_only(h, "pmlp_train_step_noalloc")) return rc;
  if (h->mse) return fail(PMLP_ESTATE, "a regression handle trains with pmlp_train_step_mse");
  if (!y_dev) return fail(PMLP_EINVAL, "null labels");
  if (!std::isfinite(lr)) return fail(PMLP_EINVAL, "learning rate is not finite");
  if (bf16_mode(h))
    return fail(PMLP_ESTATE, "the allocation-free step runs in the PMLP_FP32 mode only");
  const int32_t Bp = pad_batch(B);
  const size_t need = work_bytes(h, Bp);
  if (need > kScratchBytes)
    return fail(PMLP_EINVAL, "the allocation-free step needs " + std::to_string(need >> 20) +
                                 " MiB of workspace for this pack and batch; its limit is " +
                                 std::to_string(kScratchBytes >> 20) + " MiB");
  if (int rc = use_device(h)) return rc;
  unsigned char* base = nullptr;
  if (int rc = scratch_base(h->dev, &base)) return rc;
  const Work w = carve_work(h, Bp, base);
  // per-kernel timing would create events; this call records none
  const bool prof = h->prof;
  h->prof = false;
  const int rc = step(h, X_dev, y_dev, B, lr, nullptr, nullptr, nullptr, nullptr, nullptr, &w);
  h->prof = prof;
  return rc;
}

int pmlp_train_step_lr(pmlp_t h, const float* X_dev, const int32_t* y_dev, int32_t B,
                       const float* lr_dev) {
  if (int rc = check_batch(h, X_dev, B)) return rc;
  if (int rc = one_layer_only(h, "pmlp_train_step_lr")) return rc;
  if (h->mse) return fail(PMLP_ESTATE, "a regression handle trains with pmlp_train_step_mse");
  if (!y_dev) return fail(PMLP_EINVAL, "null labels");
  if (!lr_dev) return fail(PMLP_EINVAL, "null per-model learning rates");
  return step(h, X_dev, y_dev, B, 0.f, lr_dev, nullptr, nullptr);
}

int pmlp_gradients(pmlp_t h, const float* X_dev, const int32_t* y_dev, int32_t B,
                   float* dW1_dev, float* dW2_dev) {
  if (int rc = check_batch(h, X_dev, B)) return rc;
  if (int rc = one_layer_only(h, "pmlp_gradients (use pmlp_gradients_deep)")) return rc;
  if (h->mse) return fail(PMLP_ESTATE, "a regression handle uses pmlp_gradients_mse");
  if (!y_dev || !dW1_dev || !dW2_dev) return fail(PMLP_EINVAL, "null labels or gradient buffer");
  return step(h, X_dev, y_dev, B, 0.f, nullptr, dW1_dev, dW2_dev);
}

int pmlp_train_step_mse(pmlp_t h, const float* X_dev, const float* Y_dev, int32_t B, float lr) {
  if (int rc = check_batch(h, X_dev, B)) return rc;
  if (int rc = one_layer_only(h, "pmlp_train_step_mse")) return rc;
  if (!h->mse) return fail(PMLP_ESTATE, "the handle was created without PMLP_MSE");
  if (!Y_dev) return fail(PMLP_EINVAL, "null targets");
  if (!std::isfinite(lr)) return fail(PMLP_EINVAL, "learning rate is not finite");
  return step(h, X_dev, Y_dev, B, lr, nullptr, nullptr, nullptr);
}

int pmlp_gradients_mse(pmlp_t h, const float* X_dev, const float* Y_dev, int32_t B,
                       float* dW1_dev, float* dW2_dev) {
  if (int rc = check_batch(h, X_dev, B)) return rc;
  if (int rc = one_layer_only(h, "pmlp_gradients_mse")) return rc;
  if (!h->mse) return fail(PMLP_ESTATE, "the handle was created without PMLP_MSE");
  if (!Y_dev || !dW1_dev || !dW2_dev) return fail(PMLP_EINVAL, "null targets or gradient buffer");
  return step(h, X_dev, Y_dev, B, 0.f, nullptr, dW1_dev, dW2_dev);
}

int pmlp_gradients_ex(pmlp_t h, const float* X_dev, const int32_t* y_dev, int32_t B,
                      float* dW1_dev, float* dW2_dev, float* db1_dev, float* db2_dev) {
  if (int rc = check_batch(h, X_dev, B)) return rc;
  if (int rc = one_layer_only(h, "pmlp_gradients_ex")) return rc;
  if (h->mse) return fail(PMLP_ESTATE, "a regression handle uses pmlp_gradients_mse");
  if (!y_dev || !dW1_dev || !dW2_dev) return fail(PMLP_EINVAL, "null labels or gradient buffer");
  if (h->bcol < 0) return fail(PMLP_ESTATE, "the handle was created without biases");
  if (!db1_dev || !db2_dev) return fail(PMLP_EINVAL, "null bias gradient buffer");
  return step(h, X_dev, y_dev, B, 0.f, nullptr, dW1_dev, dW2_dev, db1_dev, db2_dev);
}

int pmlp_get_biases(pmlp_t h, float* b1_host, float* b2_host) {
  if (int rc = check_handle(h)) return rc;
  if (h->bcol < 0) return fail(PMLP_ESTATE, "the handle was created without biases");
  if (int rc = use_device(h)) return rc;
  PMLP_HIP(hipStreamSynchronize(h->stream));
  if (b1_host)  // column bcol of W1
    PMLP_HIP(hipMemcpy2D(b1_host, sizeof(float), h->W1 + h->bcol, (size_t)h->F4 * sizeof(float),
                         sizeof(float), (size_t)h->N, hipMemcpyDeviceToHost));
  if (b2_host)
    PMLP_HIP(hipMemcpy(b2_host, h->b2, (size_t)h->M * h->O * sizeof(float),
                       hipMemcpyDeviceToHost));
  return PMLP_OK;
}

int pmlp_set_biases(pmlp_t h, const float* b1_host, const float* b2_host) {
  if (int rc = check_handle(h)) return rc;
  if (h->bcol < 0) return fail(PMLP_ESTATE, "the handle was created without biases");
  if (int rc = use_device(h)) return rc;
  PMLP_HIP(hipStreamSynchronize(h->stream));
  if (b1_host) {
    h->w1b_valid = false;
    PMLP_HIP(hipMemcpy2D(h->W1 + h->bcol, (size_t)h->F4 * sizeof(float), b1_host, sizeof(float),
                         sizeof(float), (size_t)h->N, hipMemcpyHostToDevice));
  }
  if (b2_host)
    PMLP_HIP(hipMemcpy(h->b2, b2_host, (size_t)h->M * h->O * sizeof(float),
                       hipMemcpyHostToDevice));
  return PMLP_OK;
}

int pmlp_hidden(pmlp_t h, const float* X_dev, int32_t B, float* Z_dev, float* H_dev) {
  if (int rc = check_batch(h, X_dev, B)) return rc;
  if (int rc = one_layer_only(h, "pmlp_hidden")) return rc;
  const int32_t Bp = pad_batch(B);
  if (int rc = use_device(h)) return rc;
  if (int rc = ensure_workspace(h, Bp)) return rc;
  if (int rc = forward_hidden(h, X_dev, B, Bp, handle_work(h))) return rc;
  if (!Z_dev && !H_dev) return PMLP_OK;
  return run(h, KID_ACT, [&] {
    return launch_hidden_out(h->Zt, Bp, B, h->N, h->d_mid, h->d_act, Z_dev, H_dev, h->stream,
                             z_bf16(h));
  });
}

int pmlp_losses(pmlp_t h, float* out_host) {
  if (int rc = check_handle(h)) return rc;
  if (!out_host) return fail(PMLP_EINVAL, "null output");
  if (!h->have_loss) return fail(PMLP_ESTATE, "no training step has run yet");
  if (int rc = use_device(h)) return rc;
  PMLP_HIP(hipStreamSynchronize(h->stream));
  PMLP_HIP(hipMemcpy(out_host, h->loss, (size_t)h->M * sizeof(float), hipMemcpyDeviceToHost));
  int32_t flag[2] = {0, 0};
  PMLP_HIP(hipMemcpy(flag, h->flag, 2 * sizeof(int32_t), hipMemcpyDeviceToHost));
  if (flag[0] || flag[1]) {
    PMLP_HIP(hipMemset(h->flag, 0, 2 * sizeof(int32_t)));
    return fail(PMLP_EINVAL, flag[0] ? "a label outside [0, O) was seen since the last pmlp_losses call"
                                     : "a non-finite per-model learning rate was seen since the "
                                       "last pmlp_losses call");
  }
  return PMLP_OK;
}

int pmlp_get_params(pmlp_t h, float* W1_host, float* W2_host) {
  if (int rc = check_handle(h)) return rc;
  if (int rc = one_layer_only(h, "pmlp_get_params (use pmlp_get_params_deep)")) return rc;
  if (int rc = use_device(h)) return rc;
  PMLP_HIP(hipStreamSynchronize(h->stream));
  if (W1_host)
    PMLP_HIP(hipMemcpy2D(W1_host, (size_t)h->F * sizeof(float), h->W1,
                         (size_t)h->F4 * sizeof(float), (size_t)h->F * sizeof(float),
                         (size_t)h->N, hipMemcpyDeviceToHost));
  if (W2_host)
    PMLP_HIP(hipMemcpy2D(W2_host, (size_t)h->N * sizeof(float), h->W2,
                         (size_t)h->Npad * sizeof(float), (size_t)h->N * sizeof(float),
                         (size_t)h->O, hipMemcpyDeviceToHost));
  return PMLP_OK;
}

int pmlp_set_params(pmlp_t h, const float* W1_host, const float* W2_host) {
  if (int rc = check_handle(h)) return rc;
  if (int rc = one_layer_only(h, "pmlp_set_params (use pmlp_set_params_deep)")) return rc;
  if (int rc = use_device(h)) return rc;
  PMLP_HIP(hipStreamSynchronize(h->stream));
  if (W1_host) h->w1b_valid = false;
  if (W1_host) {
    PMLP_HIP(hipMemcpy2D(h->W1, (size_t)h->F4 * sizeof(float), W1_host,
                         (size_t)h->F * sizeof(float), (size_t)h->F * sizeof(float),
                         (size_t)h->N, hipMemcpyHostToDevice));
    if (h->d_fmask) {  // weights of features a model does not see are held at zero
      PMLP_HIP(launch_apply_fmask(h->W1, h->Npad, h->F4, h->d_mid, h->d_fmask, h->fmw, h->stream));
      PMLP_HIP(hipStreamSynchronize(h->stream));
    }
  }
  if (W2_host)
    PMLP_HIP(hipMemcpy2D(h->W2, (size_t)h->Npad * sizeof(float), W2_host,
                         (size_t)h->N * sizeof(float), (size_t)h->N * sizeof(float),
                         (size_t)h->O, hipMemcpyHostToDevice));
  return PMLP_OK;
}

int pmlp_get_models(pmlp_t h, const int32_t* models_host, int32_t count, float* W1_host,
                    float* W2_host) {
  if (int rc = check_handle(h)) return rc;
  if (int rc = one_layer_only(h, "pmlp_get_models")) return rc;
  if (count < 0 || (count > 0 && !models_host)) return fail(PMLP_EINVAL, "bad model list");
  int64_t rows = 0;
  for (int32_t i = 0; i < count; ++i) {
    const int32_t m = models_host[i];
    if (m < 0 || m >= h->M) return fail(PMLP_EINVAL, "model index out of range at " + std::to_string(i));
    rows += h->hs[m];
  }
  if (int rc = use_device(h)) return rc;
  PMLP_HIP(hipStreamSynchronize(h->stream));
  int64_t r = 0;
  for (int32_t i = 0; i < count; ++i) {
    const int32_t m = models_host[i];
    const int64_t off = h->seg_off[m], w = h->hs[m];
    if (W1_host)
      PMLP_HIP(hipMemcpy2D(W1_host + r * h->F, (size_t)h->F * sizeof(float), h->W1 + off * h->F4,
                           (size_t)h->F4 * sizeof(float), (size_t)h->F * sizeof(float), (size_t)w,
                           hipMemcpyDeviceToHost));
    if (W2_host)
      PMLP_HIP(hipMemcpy2D(W2_host + r, (size_t)rows * sizeof(float), h->W2 + off,
                           (size_t)h->Npad * sizeof(float), (size_t)w * sizeof(float),
                           (size_t)h->O, hipMemcpyDeviceToHost));
    r += w;
  }
  return PMLP_OK;
}

int pmlp_set_feature_mask(pmlp_t h, const uint8_t* mask_host) {
  if (int rc = check_handle(h)) return rc;
  if (int rc = one_layer_only(h, "pmlp_set_feature_mask")) return rc;
  if (int rc = use_device(h)) return rc;
  PMLP_HIP(hipStreamSynchronize(h->stream));
  if (!mask_host) {
    dfree(h->d_fmask);
    h->fmw = 0;
    return PMLP_OK;
  }
  // words cover every column the dW1 epilogues touch (F4 and the partial
  // 16-column block past it); columns from F on are always seen
  const int32_t fmw = (h->F4 + 16 + 31) / 32;
  std::vector<uint32_t> bits((size_t)h->M * fmw, 0u);
  for (int32_t m = 0; m < h->M; ++m)
    for (int32_t q = 0; q < 32 * fmw; ++q)
      if (q >= h->F || mask_host[(size_t)m * h->F + q])
        bits[(size_t)m * fmw + (q >> 5)] |= 1u << (q & 31);
  uint32_t* d = h->d_fmask;
  if (!d || h->fmw != fmw) {
    dfree(h->d_fmask);
    if (hipMalloc(&d, bits.size() * sizeof(uint32_t)) != hipSuccess) {
      (void)hipGetLastError();
      h->fmw = 0;
      return fail(PMLP_ENOMEM, "feature mask allocation failed");
    }
  }
  h->d_fmask = d;
  h->fmw = fmw;
  PMLP_HIP(hipMemcpy(d, bits.data(), bits.size() * sizeof(uint32_t), hipMemcpyHostToDevice));
  PMLP_HIP(launch_apply_fmask(h->W1, h->Npad, h->F4, h->d_mid, d, fmw, h->stream));
  PMLP_HIP(hipStreamSynchronize(h->stream));
  h->w1b_valid = false;
  return PMLP_OK;
}

int pmlp_info(pmlp_t h, int64_t* N, int32_t* M, int32_t* F, int32_t* O) {
  if (int rc = check_handle(h)) return rc;
  if (N) *N = h->N;
  if (M) *M = h->M;
  if (F) *F = h->F;
  if (O) *O = h->O;
  return PMLP_OK;
}

int pmlp_set_profiling(pmlp_t h, int32_t enable) {
  if (int rc = check_handle(h)) return rc;
  h->prof = enable != 0;
  return PMLP_OK;
}

int pmlp_kernel_time(pmlp_t h, int32_t k, double* total_ms, int64_t* launches) {
  if (int rc = check_handle(h)) return rc;
  if (k < 0 || k >= KID_COUNT) return fail(PMLP_EINVAL, "kernel id out of range");
  if (!h->pending.empty()) {
    if (int rc = use_device(h)) return rc;
    PMLP_HIP(hipStreamSynchronize(h->stream));
    for (auto& p : h->pending) {
      float ms = 0.f;
      PMLP_HIP(hipEventElapsedTime(&ms, p.a, p.b));
      h->tot_ms[p.k] += ms;
      h->launches[p.k] += 1;
      h->ev_free.push_back(p.a);
      h->ev_free.push_back(p.b);
    }
    h->pending.clear();
  }
  if (total_ms) *total_ms = h->tot_ms[k];
  if (launches) *launches = h->launches[k];
  return PMLP_OK;
}

int pmlp_profile_reset(pmlp_t h) {
  if (int rc = check_handle(h)) return rc;
  if (!h->pending.empty()) {
    if (int rc = use_device(h)) return rc;
    PMLP_HIP(hipStreamSynchronize(h->stream));
    for (auto& p : h->pending) {
      h->ev_free.push_back(p.a);
      h->ev_free.push_back(p.b);
    }
    h->pending.clear();
  }
  for (int k = 0; k < KID_COUNT; ++k) {
    h->tot_ms[k] = 0.0;
    h->launches[k] = 0;
  }
  return PMLP_OK;
}

int pmlp_create_deep(pmlp_t* out, int32_t F, int32_t O, int32_t M, const int32_t* h1,
                     const int32_t* h2, const int32_t* act_ids, uint64_t seed) {
  if (!out) return fail(PMLP_EINVAL, "null output handle pointer");
  *out = nullptr;
  if (M < 1) return fail(PMLP_EINVAL, "M must be >= 1");
  if (!h2) return fail(PMLP_EINVAL, "null second-layer sizes");
  int64_t N2 = 0, K = 0;
  for (int32_t m = 0; m < M; ++m) {
    if (h2[m] < 1) return fail(PMLP_EINVAL, "second-layer size < 1 at model " + std::to_string(m));
    N2 += h2[m];
    if (h1 && h1[m] > 0) K += (int64_t)h1[m] * h2[m];
  }
  if (N2 > ((int64_t)1 << 31) - 1) return fail(PMLP_EINVAL, "second-layer units exceed 2^31-1");
  pmlp_t h = nullptr;
  if (int rc = pmlp_create_ex(&h, F, O, M, h1, act_ids, seed, 0)) return rc;  // checks the rest
  PmlpDeep* d = new (std::nothrow) PmlpDeep();
  if (!d) {
    pmlp_destroy(h);
    return fail(PMLP_ENOMEM, "host allocation failed");
  }
  h->deep = d;
  d->N2 = N2;
  d->N2pad = (N2 + 63) / 64 * 64;
  d->K = K;
  d->h2.assign(h2, h2 + M);
  d->off2.assign((size_t)M + 1, 0);
  d->koff.assign((size_t)M + 1, 0);
  for (int32_t m = 0; m < M; ++m) {
    d->off2[m + 1] = d->off2[m] + h2[m];
    d->koff[m + 1] = d->koff[m] + (int64_t)h1[m] * h2[m];
  }
  std::vector<int32_t> mid2((size_t)d->N2pad, M - 1);  // padding rows map to the last model
  for (int32_t m = 0; m < M; ++m)
    for (int64_t n = d->off2[m]; n < d->off2[m + 1]; ++n) mid2[n] = m;
  std::vector<Tile3> tiles;
  build_tiles(d->h2, tile_cap(N2), tiles, d->has_split2);
  d->ntiles2 = (int32_t)tiles.size();
  std::vector<int32_t> order(tiles.size());
  for (size_t i = 0; i < order.size(); ++i) order[i] = (int32_t)i;
  std::stable_sort(order.begin(), order.end(),
                   [&](int32_t x, int32_t y) { return tiles[x].len > tiles[y].len; });
  std::vector<SegUnit> ufwd, uback;
  std::vector<SegTile> tgrad;
  for (int32_t m = 0; m < M; ++m) {
    for (int32_t r = 0; r < h2[m]; r += 8) ufwd.push_back(SegUnit{m, r});
    for (int32_t r = 0; r < h1[m]; r += 8) uback.push_back(SegUnit{m, r});
    for (int32_t i = 0; i < h2[m]; i += 16)
      for (int32_t j = 0; j < h1[m]; j += 64) tgrad.push_back(SegTile{m, i, j, 0});
  }
  if (ufwd.size() > 0x7fffffff || uback.size() > 0x7fffffff || tgrad.size() > 0x7fffffff) {
    pmlp_destroy(h);
    return fail(PMLP_EINVAL, "too many work units for one launch");
  }
  d->nufwd = (int32_t)ufwd.size();
  d->nuback = (int32_t)uback.size();
  d->ntgrad = (int32_t)tgrad.size();
  std::vector<float> bound12((size_t)M), bound2((size_t)M);
  for (int32_t m = 0; m < M; ++m) {
    bound12[m] = (float)(1.0 / std::sqrt((double)h1[m]));
    bound2[m] = (float)(1.0 / std::sqrt((double)h2[m]));
  }
  float* d_b12 = nullptr;
  float* d_b2 = nullptr;
  dfree(h->W2);  // the one-layer W2 [O][Npad] gives way to [O][N2pad]
  const size_t w2_bytes = (size_t)O * d->N2pad * sizeof(float);
  const size_t nk = (size_t)(K > 0 ? K : 1);
  if (hipMalloc(&h->W2, w2_bytes) != hipSuccess ||
      hipMalloc(&d->d_off1, ((size_t)M + 1) * sizeof(int64_t)) != hipSuccess ||
      hipMalloc(&d->d_off2, ((size_t)M + 1) * sizeof(int64_t)) != hipSuccess ||
      hipMalloc(&d->d_koff, ((size_t)M + 1) * sizeof(int64_t)) != hipSuccess ||
      hipMalloc(&d->d_h1, (size_t)M * sizeof(int32_t)) != hipSuccess ||
      hipMalloc(&d->d_h2, (size_t)M * sizeof(int32_t)) != hipSuccess ||
      hipMalloc(&d->d_mid2, (size_t)d->N2pad * sizeof(int32_t)) != hipSuccess ||
      hipMalloc(&d->W12, nk * sizeof(float)) != hipSuccess ||
      hipMalloc(&d->G12, nk * sizeof(float)) != hipSuccess ||
      hipMalloc(&d->d_tiles2, tiles.size() * sizeof(Tile3)) != hipSuccess ||
      hipMalloc(&d->d_order2, order.size() * sizeof(int32_t)) != hipSuccess ||
      hipMalloc(&d->d_ufwd, ufwd.size() * sizeof(SegUnit)) != hipSuccess ||
      hipMalloc(&d->d_uback, uback.size() * sizeof(SegUnit)) != hipSuccess ||
      hipMalloc(&d->d_tgrad, tgrad.size() * sizeof(SegTile)) != hipSuccess ||
      hipMalloc(&d_b12, (size_t)M * sizeof(float)) != hipSuccess ||
      hipMalloc(&d_b2, (size_t)M * sizeof(float)) != hipSuccess) {
    (void)hipGetLastError();
    dfree(d_b12);
    dfree(d_b2);
    pmlp_destroy(h);
    return fail(PMLP_ENOMEM, "device allocation failed for the second hidden layer");
  }
  auto setup = [&]() -> int {
    PMLP_HIP(hipMemcpy(d->d_off1, h->seg_off.data(), ((size_t)M + 1) * sizeof(int64_t),
                       hipMemcpyHostToDevice));
    PMLP_HIP(hipMemcpy(d->d_off2, d->off2.data(), ((size_t)M + 1) * sizeof(int64_t),
                       hipMemcpyHostToDevice));
    PMLP_HIP(hipMemcpy(d->d_koff, d->koff.data(), ((size_t)M + 1) * sizeof(int64_t),
                       hipMemcpyHostToDevice));
    PMLP_HIP(hipMemcpy(d->d_h1, h1, (size_t)M * sizeof(int32_t), hipMemcpyHostToDevice));
    PMLP_HIP(hipMemcpy(d->d_h2, h2, (size_t)M * sizeof(int32_t), hipMemcpyHostToDevice));
    PMLP_HIP(hipMemcpy(d->d_mid2, mid2.data(), (size_t)d->N2pad * sizeof(int32_t),
                       hipMemcpyHostToDevice));
    PMLP_HIP(hipMemcpy(d->d_tiles2, tiles.data(), tiles.size() * sizeof(Tile3),
                       hipMemcpyHostToDevice));
    PMLP_HIP(hipMemcpy(d->d_order2, order.data(), order.size() * sizeof(int32_t),
                       hipMemcpyHostToDevice));
    PMLP_HIP(hipMemcpy(d->d_ufwd, ufwd.data(), ufwd.size() * sizeof(SegUnit),
                       hipMemcpyHostToDevice));
    PMLP_HIP(hipMemcpy(d->d_uback, uback.data(), uback.size() * sizeof(SegUnit),
                       hipMemcpyHostToDevice));
    PMLP_HIP(hipMemcpy(d->d_tgrad, tgrad.data(), tgrad.size() * sizeof(SegTile),
                       hipMemcpyHostToDevice));
    PMLP_HIP(hipMemcpy(d_b12, bound12.data(), (size_t)M * sizeof(float), hipMemcpyHostToDevice));
    PMLP_HIP(hipMemcpy(d_b2, bound2.data(), (size_t)M * sizeof(float), hipMemcpyHostToDevice));
    PMLP_HIP(hipMemset(h->W2, 0, w2_bytes));
    const uint64_t key = splitmix64_host(seed);
    PMLP_HIP(launch_init_w12(d->W12, K, d->d_koff, M, d_b12, key, nullptr));
    PMLP_HIP(launch_init_w2(h->W2, N2, d->N2pad, O, d->d_mid2, d_b2, key, nullptr));
    PMLP_HIP(hipStreamSynchronize(nullptr));
    return PMLP_OK;
  };
  const int rc = setup();
  dfree(d_b12);
  dfree(d_b2);
  if (rc) {
    pmlp_destroy(h);
    return rc;
  }
  *out = h;
  return PMLP_OK;
}

int pmlp_gradients_deep(pmlp_t h, const float* X_dev, const int32_t* y_dev, int32_t B,
                        float* dW1_dev, float* dW12_dev, float* dW2_dev) {
  if (int rc = check_batch(h, X_dev, B)) return rc;
  if (!h->deep) return fail(PMLP_ESTATE, "the handle has one hidden layer (use pmlp_gradients)");
  if (!y_dev || !dW1_dev || !dW12_dev || !dW2_dev)
    return fail(PMLP_EINVAL, "null labels or gradient buffer");
  return step_deep(h, X_dev, y_dev, B, 0.f, dW1_dev, dW12_dev, dW2_dev);
}

int pmlp_get_params_deep(pmlp_t h, float* W1_host, float* W12_host, float* W2_host) {
  if (int rc = check_handle(h)) return rc;
  PmlpDeep* d = h->deep;
  if (!d) return fail(PMLP_ESTATE, "the handle has one hidden layer (use pmlp_get_params)");
  if (int rc = use_device(h)) return rc;
  PMLP_HIP(hipStreamSynchronize(h->stream));
  if (W1_host)
    PMLP_HIP(hipMemcpy2D(W1_host, (size_t)h->F * sizeof(float), h->W1,
                         (size_t)h->F4 * sizeof(float), (size_t)h->F * sizeof(float),
                         (size_t)h->N, hipMemcpyDeviceToHost));
  if (W12_host && d->K > 0)
    PMLP_HIP(hipMemcpy(W12_host, d->W12, (size_t)d->K * sizeof(float), hipMemcpyDeviceToHost));
  if (W2_host)
    PMLP_HIP(hipMemcpy2D(W2_host, (size_t)d->N2 * sizeof(float), h->W2,
                         (size_t)d->N2pad * sizeof(float), (size_t)d->N2 * sizeof(float),
                         (size_t)h->O, hipMemcpyDeviceToHost));
  return PMLP_OK;
}

int pmlp_set_params_deep(pmlp_t h, const float* W1_host, const float* W12_host,
                         const float* W2_host) {
  if (int rc = check_handle(h)) return rc;
  PmlpDeep* d = h->deep;
  if (!d) return fail(PMLP_ESTATE, "the handle has one hidden layer (use pmlp_set_params)");
  if (int rc = use_device(h)) return rc;
  PMLP_HIP(hipStreamSynchronize(h->stream));
  if (W1_host)
    PMLP_HIP(hipMemcpy2D(h->W1, (size_t)h->F4 * sizeof(float), W1_host,
                         (size_t)h->F * sizeof(float), (size_t)h->F * sizeof(float),
                         (size_t)h->N, hipMemcpyHostToDevice));
  if (W12_host && d->K > 0)
    PMLP_HIP(hipMemcpy(d->W12, W12_host, (size_t)d->K * sizeof(float), hipMemcpyHostToDevice));
  if (W2_host)
    PMLP_HIP(hipMemcpy2D(h->W2, (size_t)d->N2pad * sizeof(float), W2_host,
                         (size_t)d->N2 * sizeof(float), (size_t)d->N2 * sizeof(float),
                         (size_t)h->O, hipMemcpyHostToDevice));
  return PMLP_OK;
}

int pmlp_info_deep(pmlp_t h, int64_t* N2, int64_t* K) {
  if (int rc = check_handle(h)) return rc;
  if (!h->deep) return fail(PMLP_ESTATE, "the handle has one hidden layer");
  if (N2) *N2 = h->deep->N2;
  if (K) *K = h->deep->K;
  return PMLP_OK;
}

int pmlp_nonfinite(pmlp_t h, int32_t* count_host) {
  if (int rc = check_handle(h)) return rc;
  if (!count_host) return fail(PMLP_EINVAL, "null output");
  if (int rc = use_device(h)) return rc;
  PMLP_HIP(hipStreamSynchronize(h->stream));
  PMLP_HIP(hipMemcpy(count_host, h->flag + 2, sizeof(int32_t), hipMemcpyDeviceToHost));
  PMLP_HIP(hipMemset(h->flag + 2, 0, sizeof(int32_t)));
  return PMLP_OK;
}

int pmlp_kernel_variant(pmlp_t h, int32_t k, const char** name, int32_t* arith) {
  if (int rc = check_handle(h)) return rc;
  if (k < 0 || k >= KID_COUNT) return fail(PMLP_EINVAL, "kernel id out of range");
  const KernelVariant v = h->variant[k];
  if (name) *name = v.name ? v.name : "";
  if (arith) *arith = v.name ? v.arith : PMLP_ARITH_NONE;
  return PMLP_OK;
}

const char* pmlp_kernel_name(int32_t k) {
  if (k < 0 || k >= KID_COUNT) return "";
  return kKernelNames[k];
}

const char* pmlp_last_error(void) { return g_err.c_str(); }

}  // extern "C"
