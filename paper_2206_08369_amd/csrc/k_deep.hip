// Kernels of packs whose models have two hidden layers (Section 7, Figure 3:
// the packed network extended by a second hidden layer in which a unit only
// ever sums the first-layer units of its own model).
//
// The hidden-to-hidden weights are block diagonal: model m's block W12_m
// [h2_m, h1_m] is stored row-major at offset koff[m] of one packed vector.
// With Zt1 [N1pad][Bp] and Zt2 [N2pad][Bp] batch-minor as everywhere else,
// the products of this layer are, per model,
//   forward   Z2_m  = W12_m act(Z1_m)                 [h2_m, Bp]
//   gradient  dW12_m = dZ2_m act(Z1_m)^T               [h2_m, h1_m]
//   backward  dZ1_m = (W12_m^T dZ2_m) * act'(Z1_m)     [h1_m, Bp]
// The first layer's product, the M3 forward / backward of the output layer,
// the loss and the dW1 product are the one-hidden-layer kernels.

#include "device_common.h"

namespace pmlpk {

// W12[k] = uniform(tag 5, idx k) * bound12[model of k]; the model is found
// by binary search over koff [M+1].
__global__ __launch_bounds__(kBlock) void k_init_w12(float* __restrict__ W12, int64_t K,
                                                     const int64_t* __restrict__ koff, int M,
                                                     const float* __restrict__ bound12,
                                                     uint64_t key) {
  for (int64_t k = (int64_t)blockIdx.x * kBlock + threadIdx.x; k < K;
       k += (int64_t)gridDim.x * kBlock) {
    int lo = 0, hi = M - 1;  // last m with koff[m] <= k
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (koff[mid] <= k) lo = mid;
      else hi = mid - 1;
    }
    W12[k] = uniform_weight(key, 5, (uint64_t)k, bound12[lo]);
  }
}

hipError_t launch_init_w12(float* W12, int64_t K, const int64_t* koff, int32_t M,
                           const float* bound12, uint64_t key, hipStream_t s) {
  if (K <= 0) return hipSuccess;
  k_init_w12<<<grid_for(K), kBlock, 0, s>>>(W12, K, koff, M, bound12, key);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Forward: one wave per (unit: model m, RB consecutive rows r0.. of its
// second layer) and 64-sample chunk; lane = sample.  The wave walks the
// model's h1 first-layer units: one coalesced load of Z1, the activation
// once, and RB multiply-adds with wave-uniform weights.  Rows past the
// model's h2 repeat its last row (never stored), so every load stays inside
// the model's block.
// ---------------------------------------------------------------------------

constexpr int kSegRows = 8;

template <int ACT>
__device__ __forceinline__ void seg_fwd_rows(float (&acc)[kSegRows], const float* __restrict__ z1,
                                             int Bp, const float* __restrict__ w, int a,
                                             int last) {
  for (int j = 0; j < a; ++j) {
    const float hv = act_fwd(ACT, z1[(int64_t)j * Bp]);
#pragma unroll
    for (int r = 0; r < kSegRows; ++r)
      acc[r] = fmaf(w[(int64_t)(r < last ? r : last) * a + j], hv, acc[r]);
  }
}

__global__ __launch_bounds__(64) void k_seg_fwd(const float* __restrict__ Zt1,
                                                float* __restrict__ Zt2, int Bp,
                                                const DeepArgs a, const SegUnit* __restrict__ units) {
  const SegUnit u = units[blockIdx.x];
  const int m = u.m;
  const int h1 = a.h1[m], h2 = a.h2[m];
  const int b = blockIdx.y * 64 + threadIdx.x;
  const int bb = b < Bp ? b : Bp - 1;
  const int last = (h2 - u.r0 < kSegRows ? h2 - u.r0 : kSegRows) - 1;
  const float* w = a.W12 + a.koff[m] + (int64_t)u.r0 * h1;
  const float* z1 = Zt1 + a.off1[m] * Bp + bb;
  float acc[kSegRows];
#pragma unroll
  for (int r = 0; r < kSegRows; ++r) acc[r] = 0.f;
  switch (a.act[m]) {
    case 0: seg_fwd_rows<0>(acc, z1, Bp, w, h1, last); break;
    case 1: seg_fwd_rows<1>(acc, z1, Bp, w, h1, last); break;
    case 2: seg_fwd_rows<2>(acc, z1, Bp, w, h1, last); break;
    case 3: seg_fwd_rows<3>(acc, z1, Bp, w, h1, last); break;
    case 4: seg_fwd_rows<4>(acc, z1, Bp, w, h1, last); break;
    case 5: seg_fwd_rows<5>(acc, z1, Bp, w, h1, last); break;
    case 6: seg_fwd_rows<6>(acc, z1, Bp, w, h1, last); break;
    case 7: seg_fwd_rows<7>(acc, z1, Bp, w, h1, last); break;
    case 8: seg_fwd_rows<8>(acc, z1, Bp, w, h1, last); break;
    case 9: seg_fwd_rows<9>(acc, z1, Bp, w, h1, last); break;
    case 10: seg_fwd_rows<10>(acc, z1, Bp, w, h1, last); break;
    case 11: seg_fwd_rows<11>(acc, z1, Bp, w, h1, last); break;
    default: seg_fwd_rows<12>(acc, z1, Bp, w, h1, last); break;
  }
  if (b >= Bp) return;
  float* z2 = Zt2 + (a.off2[m] + u.r0) * Bp + b;
#pragma unroll
  for (int r = 0; r < kSegRows; ++r)
    if (r <= last) z2[(int64_t)r * Bp] = acc[r];
}

hipError_t launch_seg_fwd(const float* Zt1, float* Zt2, int32_t Bp, const DeepArgs& a,
                          const SegUnit* units, int32_t nunits, hipStream_t s) {
  note_variant("k_seg_fwd", kArithNone);
  if (nunits <= 0) return hipSuccess;
  k_seg_fwd<<<dim3((unsigned)nunits, (unsigned)((Bp + 63) / 64)), 64, 0, s>>>(Zt1, Zt2, Bp, a,
                                                                                units);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Weight gradient: one workgroup (4 waves) per tile of 16 rows x 64 columns
// of a model's block.  Per 64-sample chunk it stages act(Z1) of the tile's
// 64 columns (rows of 65 floats: the column reads below are conflict-free)
// and dZ2 of its 16 rows in LDS; thread (group g, column j) then sums the
// chunk for rows 4g .. 4g+3 (dZ2 reads are broadcasts within a wave).
// Out-of-block rows and columns are staged as zeros and never stored.
// ---------------------------------------------------------------------------

__global__ __launch_bounds__(256) void k_seg_grad(const float* __restrict__ Zt1,
                                                  const float* __restrict__ dZ2, int Bp,
                                                  const DeepArgs a,
                                                  const SegTile* __restrict__ tiles,
                                                  float* __restrict__ G12) {
  __shared__ float hs[64][65];
  __shared__ float ds[16][64];
  const SegTile t = tiles[blockIdx.x];
  const int m = t.m;
  const int h1 = a.h1[m], h2 = a.h2[m];
  const int am = a.act[m];
  const float* z1 = Zt1 + a.off1[m] * Bp;
  const float* d2 = dZ2 + a.off2[m] * Bp;
  const int tid = threadIdx.x, lj = tid & 63, g = tid >> 6;
  float acc[4] = {0.f, 0.f, 0.f, 0.f};
  for (int b0 = 0; b0 < Bp; b0 += 64) {
    for (int e = tid; e < 64 * 64; e += 256) {
      const int r = e >> 6, c = e & 63, j = t.j0 + r, b = b0 + c;
      hs[r][c] = (j < h1 && b < Bp) ? act_fwd(am, z1[(int64_t)j * Bp + b]) : 0.f;
    }
    for (int e = tid; e < 16 * 64; e += 256) {
      const int r = e >> 6, c = e & 63, i = t.i0 + r, b = b0 + c;
      ds[r][c] = (i < h2 && b < Bp) ? d2[(int64_t)i * Bp + b] : 0.f;
    }
    __syncthreads();
#pragma unroll 8
    for (int c = 0; c < 64; ++c) {
      const float hv = hs[lj][c];
#pragma unroll
      for (int r = 0; r < 4; ++r) acc[r] = fmaf(ds[4 * g + r][c], hv, acc[r]);
    }
    __syncthreads();
  }
  const int j = t.j0 + lj;
  if (j >= h1) return;
  float* out = G12 + a.koff[m];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int i = t.i0 + 4 * g + r;
    if (i < h2) out[(int64_t)i * h1 + j] = acc[r];
  }
}

hipError_t launch_seg_grad(const float* Zt1, const float* dZ2, int32_t Bp, const DeepArgs& a,
                           const SegTile* tiles, int32_t ntiles, float* G12, hipStream_t s) {
  note_variant("k_seg_grad", kArithNone);
  if (ntiles <= 0) return hipSuccess;
  k_seg_grad<<<(unsigned)ntiles, 256, 0, s>>>(Zt1, dZ2, Bp, a, tiles, G12);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Backward into the first layer: one wave per (unit: model m, RB rows r0..
// of its first layer) and 64-sample chunk; lane = sample.  The wave walks
// the model's h2 second-layer units (one coalesced load of dZ2 each, RB
// multiply-adds with the wave-uniform column entries of W12_m), then
// multiplies by act'(Z1) and writes dZ1 over Z1 in place (each element is
// read and written by the same lane).  W12 is read before its update.
// ---------------------------------------------------------------------------

__global__ __launch_bounds__(64) void k_seg_back(float* __restrict__ Zt1,
                                                 const float* __restrict__ dZ2, int Bp,
                                                 const DeepArgs a,
                                                 const SegUnit* __restrict__ units) {
  const SegUnit u = units[blockIdx.x];
  const int m = u.m;
  const int h1 = a.h1[m], h2 = a.h2[m];
  const int b = blockIdx.y * 64 + threadIdx.x;
  const int bb = b < Bp ? b : Bp - 1;
  const int last = (h1 - u.r0 < kSegRows ? h1 - u.r0 : kSegRows) - 1;
  const float* w = a.W12 + a.koff[m] + u.r0;  // w[i h1 + r] = W12_m[i][r0 + r]
  const float* d2 = dZ2 + a.off2[m] * Bp + bb;
  float acc[kSegRows];
#pragma unroll
  for (int r = 0; r < kSegRows; ++r) acc[r] = 0.f;
  for (int i = 0; i < h2; ++i) {
    const float d = d2[(int64_t)i * Bp];
#pragma unroll
    for (int r = 0; r < kSegRows; ++r)
      acc[r] = fmaf(w[(int64_t)i * h1 + (r < last ? r : last)], d, acc[r]);
  }
  if (b >= Bp) return;
  const int am = a.act[m];
  float* z1 = Zt1 + (a.off1[m] + u.r0) * Bp + b;
#pragma unroll
  for (int r = 0; r < kSegRows; ++r)
    if (r <= last) {
      float der;
      (void)act_fwd_bwd(am, z1[(int64_t)r * Bp], &der);
      z1[(int64_t)r * Bp] = acc[r] * der;
    }
}

hipError_t launch_seg_back(float* Zt1, const float* dZ2, int32_t Bp, const DeepArgs& a,
                           const SegUnit* units, int32_t nunits, hipStream_t s) {
  note_variant("k_seg_back", kArithNone);
  if (nunits <= 0) return hipSuccess;
  k_seg_back<<<dim3((unsigned)nunits, (unsigned)((Bp + 63) / 64)), 64, 0, s>>>(Zt1, dZ2, Bp, a,
                                                                                 units);
  return hipGetLastError();
}

// W -= lr G over n entries (the hidden-to-hidden SGD update, after the
// backward has read the old weights).
__global__ __launch_bounds__(kBlock) void k_sgd(float* __restrict__ W,
                                                const float* __restrict__ G, int64_t n,
                                                float lr) {
  for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * kBlock)
    W[i] -= lr * G[i];
}

hipError_t launch_sgd(float* W, const float* G, int64_t n, float lr, hipStream_t s) {
  note_variant("k_sgd", kArithNone);
  if (n <= 0) return hipSuccess;
  k_sgd<<<grid_for(n), kBlock, 0, s>>>(W, G, n, lr);
  return hipGetLastError();
}

}  // namespace pmlpk
