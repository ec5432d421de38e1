// Modified Matrix Multiplication kernels: fused forward and backward (generic path).

#include "device_common.h"

namespace pmlpk {

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
// inside one segment at a time, so the activation id is wave-uniform (the
// inner loop is instantiated per activation) and the running sums never
// mix models.  At the end of a segment the NG groups' partial sums are
// combined with lane shuffles and written once (plain store); the two
// halves of a segment wider than the tile limit are added with atomics onto
// zeroed logits instead (two additions onto zero are order-independent, so
// the result is still deterministic).
// ---------------------------------------------------------------------------

static constexpr int kU = 4;  // hidden units per lane group per pass (loads in flight)

template <int OM, int A, bool ZB>
__device__ __forceinline__ void fwd_segment(const float* __restrict__ Zt, int Bp, int bl,
                                            const float* __restrict__ W2, int64_t ldw, int O,
                                            int64_t nbeg, int64_t nend, int g, int NG,
                                            float (&acc)[4][OM]) {
  // Four hidden units per group per pass, all loads first; addresses past
  // the segment end are clamped to its last unit so every load is in bounds
  // and unconditional.
  for (int64_t n0 = nbeg + g; n0 < nend; n0 += kU * NG) {
    f32x4 z[kU];
    float w[kU][OM];
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      int64_t n = n0 + u * NG;
      if (n >= nend) n = nend - 1;
      z[u] = load_z4(Zt, ZB, n * Bp + bl);
#pragma unroll
      for (int o = 0; o < OM; ++o) {
        const float v = W2[(int64_t)(o < O ? o : O - 1) * ldw + n];
        w[u][o] = o < O ? v : 0.f;
      }
    }
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      if (n0 + u * NG >= nend) break;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float h = act_fwd(A, z[u][i]);
#pragma unroll
        for (int o = 0; o < OM; ++o) acc[i][o] = fmaf(h, w[u][o], acc[i][o]);
      }
    }
  }
}

template <int OM, bool ZB>
__global__ __launch_bounds__(kBlock) void k_m3_fwd(
    const float* __restrict__ Zt, int Bp, int B, const float* __restrict__ W2, int64_t ldw,
    int O, const int64_t* __restrict__ seg_off, const int32_t* __restrict__ act,
    const Tile3* __restrict__ tiles, const int32_t* __restrict__ order, int ntiles, int BW,
    int LG, int nbblk,
    const float* __restrict__ b2, float* __restrict__ out, int64_t sm, int64_t sb) {
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
  const int bl = bvalid ? b : Bp - 4;  // lanes past the batch read a valid row, store nothing
  const Tile3 t = tiles[__builtin_amdgcn_readfirstlane(order[tile])];
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
    switch (a) {
      case 0: fwd_segment<OM, 0, ZB>(Zt, Bp, bl, W2, ldw, O, n, se, g, NG, acc); break;
      case 1: fwd_segment<OM, 1, ZB>(Zt, Bp, bl, W2, ldw, O, n, se, g, NG, acc); break;
      case 2: fwd_segment<OM, 2, ZB>(Zt, Bp, bl, W2, ldw, O, n, se, g, NG, acc); break;
      case 3: fwd_segment<OM, 3, ZB>(Zt, Bp, bl, W2, ldw, O, n, se, g, NG, acc); break;
      case 4: fwd_segment<OM, 4, ZB>(Zt, Bp, bl, W2, ldw, O, n, se, g, NG, acc); break;
      case 5: fwd_segment<OM, 5, ZB>(Zt, Bp, bl, W2, ldw, O, n, se, g, NG, acc); break;
      case 6: fwd_segment<OM, 6, ZB>(Zt, Bp, bl, W2, ldw, O, n, se, g, NG, acc); break;
      case 7: fwd_segment<OM, 7, ZB>(Zt, Bp, bl, W2, ldw, O, n, se, g, NG, acc); break;
      case 8: fwd_segment<OM, 8, ZB>(Zt, Bp, bl, W2, ldw, O, n, se, g, NG, acc); break;
      case 9: fwd_segment<OM, 9, ZB>(Zt, Bp, bl, W2, ldw, O, n, se, g, NG, acc); break;
      case 10: fwd_segment<OM, 10, ZB>(Zt, Bp, bl, W2, ldw, O, n, se, g, NG, acc); break;
      case 11: fwd_segment<OM, 11, ZB>(Zt, Bp, bl, W2, ldw, O, n, se, g, NG, acc); break;
      default: fwd_segment<OM, 12, ZB>(Zt, Bp, bl, W2, ldw, O, n, se, g, NG, acc); break;
    }
    for (int s = LG; s < 64; s <<= 1)
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int o = 0; o < OM; ++o) acc[i][o] += __shfl_xor(acc[i][o], s);
    if (g == 0 && bvalid) {
      // the output bias goes with the piece that starts the segment
      const bool with_b2 = b2 && n == seg_off[m];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        if (b + i >= B) continue;
        float* dst = out + (int64_t)m * sm + (int64_t)(b + i) * sb;
#pragma unroll
        for (int o = 0; o < OM; ++o) {
          if (o >= O) continue;
          const float v = with_b2 ? acc[i][o] + b2[(int64_t)m * O + o] : acc[i][o];
          if (t.atomic) unsafeAtomicAdd(dst + o, v);
          else dst[o] = v;
        }
      }
    }
    n = se;
    ++m;
  }
}

// ---------------------------------------------------------------------------
// M3 forward for wider output layers (O > 4).  For one model the product
// with W2 followed by the scatter-add over its hidden units is a dense
// contraction over those units,
//   out[b][o] = sum_n act(Z[n][b]) W2[o][n],
// which v_mfma_f32_16x16x4f32 takes four units at a time: A[b][k] =
// act(Z[n0+k][b]) for 16 samples, B[k][o] = W2[o][n0+k] for 16 outputs (rows
// o >= O are zero).  Lane (li, lk) supplies row li of each 16-sample block
// and output li of unit n0 + lk, and ends with rows 4lk + r of the outputs;
// with NBB blocks, row li of block i is sample NBB li + i of the wave's
// range.  Per four units a lane loads NBB consecutive Z values (one vector
// load) and one weight (against O weights per unit and 4 O running sums
// per lane in the scalar kernel); units past the segment
// end are zero in both operands, so a model's sums never see another
// model's values.  One wave per (tile of whole segments, 16 NBB samples).
// ---------------------------------------------------------------------------

template <int NBB, int A, bool ZB>
__device__ __forceinline__ void fwd_segment_mf(f32x4 (&acc)[NBB], const float* __restrict__ Zt,
                                               int Bp, int b0, const float* __restrict__ wrow,
                                               bool orow_ok, int64_t nbeg, int64_t nend, int li,
                                               int lk) {
  // kUM four-unit MFMA steps per pass, the loads of the next pass in flight
  // while the current one is multiplied (loads in flight per lane: up to
  // 2 kUM (NBB + 1) values).  Row li of block i is sample b0 + NBB li + i,
  // so a lane's NBB values of one unit are one vector load and the 16 lanes
  // of a unit read 64 NBB contiguous bytes of its row (a group past the
  // batch reads the last NBB samples instead; their outputs are not stored).
  constexpr int kUM = NBB <= 2 ? 8 : 4;
  constexpr int STEP = 4 * kUM;
  int bl = b0 + NBB * li;
  if (bl > Bp - NBB) bl = Bp - NBB;
  struct Pass {
    float z[kUM][NBB];
    float w[kUM];
  };
  auto fetch = [&](Pass& P, int64_t n0) {
#pragma unroll
    for (int u = 0; u < kUM; ++u) {
      int64_t n = n0 + 4 * u + lk;
      if (n > nend - 1) n = nend - 1;
      const int64_t zi = n * Bp + bl;
      if constexpr (NBB == 4) {
        const f32x4 v = load_z4(Zt, ZB, zi);
#pragma unroll
        for (int i = 0; i < 4; ++i) P.z[u][i] = v[i];
      } else if constexpr (NBB == 2) {
        const f32x2 v = load_z2(Zt, ZB, zi);
        P.z[u][0] = v[0];
        P.z[u][1] = v[1];
      } else {
        P.z[u][0] = load_z1(Zt, ZB, zi);
      }
      P.w[u] = wrow[n];
    }
  };
  auto use = [&](const Pass& P, int64_t n0) {
#pragma unroll
    for (int u = 0; u < kUM; ++u) {
      if (n0 + 4 * u >= nend) break;  // wave-uniform: the whole step is past the end
      const bool in = n0 + 4 * u + lk < nend;
      const float wv = in && orow_ok ? P.w[u] : 0.f;
#pragma unroll
      for (int i = 0; i < NBB; ++i) {
        const float h = in ? act_fwd(A, P.z[u][i]) : 0.f;
        acc[i] = __builtin_amdgcn_mfma_f32_16x16x4f32(h, wv, acc[i], 0, 0, 0);
      }
    }
  };
  Pass p0, p1;
  if (nbeg < nend) fetch(p0, nbeg);
  for (int64_t n0 = nbeg; n0 < nend; n0 += 2 * STEP) {
    if (n0 + STEP < nend) fetch(p1, n0 + STEP);
    use(p0, n0);
    if (n0 + STEP >= nend) break;
    if (n0 + 2 * STEP < nend) fetch(p0, n0 + 2 * STEP);
    use(p1, n0 + STEP);
  }
}

template <int NBB, bool ZB>
__global__ __launch_bounds__(kBlock) void k_m3_fwd_mf(
    const float* __restrict__ Zt, int Bp, int B, const float* __restrict__ W2, int64_t ldw,
    int O, const int64_t* __restrict__ seg_off, const int32_t* __restrict__ act,
    const Tile3* __restrict__ tiles, const int32_t* __restrict__ order, int ntiles, int nbblk,
    const float* __restrict__ b2,
    float* __restrict__ out, int64_t sm, int64_t sb) {
  const int lane = threadIdx.x & 63;
  const int wv = __builtin_amdgcn_readfirstlane((int)(blockIdx.x * 4 + (threadIdx.x >> 6)));
  const int tile = wv / nbblk;
  const int bblk = wv - tile * nbblk;
  if (tile >= ntiles) return;
  const int li = lane & 15, lk = lane >> 4;
  const int b0 = bblk * 16 * NBB;
  const bool orow_ok = li < O;
  const float* wrow = W2 + (int64_t)(orow_ok ? li : O - 1) * ldw;
  const Tile3 t = tiles[__builtin_amdgcn_readfirstlane(order[tile])];
  const int64_t nend = t.n0 + t.len;
  int64_t n = t.n0;
  int m = t.m0;
  while (n < nend) {
    int64_t se = seg_off[m + 1];
    if (se > nend) se = nend;
    const int a = act[m];
    f32x4 acc[NBB];
#pragma unroll
    for (int i = 0; i < NBB; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
    switch (a) {
      case 0: fwd_segment_mf<NBB, 0, ZB>(acc, Zt, Bp, b0, wrow, orow_ok, n, se, li, lk); break;
      case 1: fwd_segment_mf<NBB, 1, ZB>(acc, Zt, Bp, b0, wrow, orow_ok, n, se, li, lk); break;
      case 2: fwd_segment_mf<NBB, 2, ZB>(acc, Zt, Bp, b0, wrow, orow_ok, n, se, li, lk); break;
      case 3: fwd_segment_mf<NBB, 3, ZB>(acc, Zt, Bp, b0, wrow, orow_ok, n, se, li, lk); break;
      case 4: fwd_segment_mf<NBB, 4, ZB>(acc, Zt, Bp, b0, wrow, orow_ok, n, se, li, lk); break;
      case 5: fwd_segment_mf<NBB, 5, ZB>(acc, Zt, Bp, b0, wrow, orow_ok, n, se, li, lk); break;
      case 6: fwd_segment_mf<NBB, 6, ZB>(acc, Zt, Bp, b0, wrow, orow_ok, n, se, li, lk); break;
      case 7: fwd_segment_mf<NBB, 7, ZB>(acc, Zt, Bp, b0, wrow, orow_ok, n, se, li, lk); break;
      case 8: fwd_segment_mf<NBB, 8, ZB>(acc, Zt, Bp, b0, wrow, orow_ok, n, se, li, lk); break;
      case 9: fwd_segment_mf<NBB, 9, ZB>(acc, Zt, Bp, b0, wrow, orow_ok, n, se, li, lk); break;
      case 10: fwd_segment_mf<NBB, 10, ZB>(acc, Zt, Bp, b0, wrow, orow_ok, n, se, li, lk); break;
      case 11: fwd_segment_mf<NBB, 11, ZB>(acc, Zt, Bp, b0, wrow, orow_ok, n, se, li, lk); break;
      default: fwd_segment_mf<NBB, 12, ZB>(acc, Zt, Bp, b0, wrow, orow_ok, n, se, li, lk); break;
    }
    if (orow_ok) {
      // the output bias goes with the piece that starts the segment
      const float bias = b2 && n == seg_off[m] ? b2[(int64_t)m * O + li] : 0.f;
      float* dst = out + (int64_t)m * sm + li;
#pragma unroll
      for (int i = 0; i < NBB; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int b = b0 + NBB * (4 * lk + r) + i;
          if (b >= B) continue;
          const float v = acc[i][r] + bias;
          if (t.atomic) unsafeAtomicAdd(dst + (int64_t)b * sb, v);
          else dst[(int64_t)b * sb] = v;
        }
    }
    n = se;
    ++m;
  }
}

template <int NBB>
static void m3_fwd_mf_dispatch(const float* Zt, bool zb, int32_t Bp, int32_t B, const float* W2,
                               int64_t ldw, int32_t O, const int64_t* seg_off,
                               const int32_t* act, const Tile3* tiles, const int32_t* order, int32_t ntiles,
                               const float* b2, float* out, int64_t sm, int64_t sb,
                               hipStream_t s) {
  const int nbblk = ceil_div_i(Bp, 16 * NBB);
  const int64_t waves = (int64_t)ntiles * nbblk;
  const unsigned blocks = (unsigned)((waves + 3) / 4);
  if (zb)
    k_m3_fwd_mf<NBB, true><<<blocks, kBlock, 0, s>>>(Zt, Bp, B, W2, ldw, O, seg_off, act, tiles,
                                                     order, ntiles, nbblk, b2, out, sm, sb);
  else
    k_m3_fwd_mf<NBB, false><<<blocks, kBlock, 0, s>>>(Zt, Bp, B, W2, ldw, O, seg_off, act, tiles, order,
                                             ntiles, nbblk, b2, out, sm, sb);
}

template <int OM>
static void m3_fwd_dispatch(const float* Zt, bool zb, int32_t Bp, int32_t B, const float* W2,
                            int64_t ldw, int32_t O, const int64_t* seg_off, const int32_t* act,
                            const Tile3* tiles, const int32_t* order, int32_t ntiles, const float* b2, float* out,
                            int64_t sm, int64_t sb, hipStream_t s) {
  int BW = 64;
  if (Bp < 64) BW = Bp <= 16 ? 16 : (Bp <= 32 ? 32 : 64);
  const int LG = BW / 4;
  const int nbblk = ceil_div_i(Bp, BW);
  const int64_t waves = (int64_t)ntiles * nbblk;
  const unsigned blocks = (unsigned)((waves + 3) / 4);
  if (zb)
    k_m3_fwd<OM, true><<<blocks, kBlock, 0, s>>>(Zt, Bp, B, W2, ldw, O, seg_off, act, tiles,
                                                 order, ntiles, BW, LG, nbblk, b2, out, sm, sb);
  else
    k_m3_fwd<OM, false><<<blocks, kBlock, 0, s>>>(Zt, Bp, B, W2, ldw, O, seg_off, act, tiles, order, ntiles,
                                         BW, LG, nbblk, b2, out, sm, sb);
}

hipError_t launch_m3_fwd(const float* Zt, int32_t Bp, int32_t B, const float* W2, int64_t ldw,
                         int32_t O, const int64_t* seg_off, const int32_t* act,
                         const Tile3* tiles, const int32_t* order, int32_t ntiles, const float* b2, float* out,
                         int64_t sm, int64_t sb, hipStream_t s, bool zb) {
  if (ntiles <= 0) return hipSuccess;
  note_variant(O <= 4 ? "k_m3_fwd" : "k_m3_fwd_mf", O <= 4 ? kArithNone : kArithFp32);
  if (O <= 2) m3_fwd_dispatch<2>(Zt, zb, Bp, B, W2, ldw, O, seg_off, act, tiles, order, ntiles, b2, out, sm, sb, s);
  else if (O <= 4) m3_fwd_dispatch<4>(Zt, zb, Bp, B, W2, ldw, O, seg_off, act, tiles, order, ntiles, b2, out, sm, sb, s);
  // wider output layers: one MFMA per four units and 16 samples
  else if (Bp <= 16) m3_fwd_mf_dispatch<1>(Zt, zb, Bp, B, W2, ldw, O, seg_off, act, tiles, order, ntiles, b2, out, sm, sb, s);
  else if (Bp <= 32) m3_fwd_mf_dispatch<2>(Zt, zb, Bp, B, W2, ldw, O, seg_off, act, tiles, order, ntiles, b2, out, sm, sb, s);
  else m3_fwd_mf_dispatch<4>(Zt, zb, Bp, B, W2, ldw, O, seg_off, act, tiles, order, ntiles, b2, out, sm, sb, s);
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
// One wave per run of kT5 consecutive hidden units and the whole batch.
// Lanes as in the forward (groups of LG lanes per hidden unit, four samples
// per lane), with `slots` passes when the batch is wider than 256.  The
// wave walks the segments of its run, so the model (its G rows, held in
// registers) and the activation are wave-uniform.  Per-unit dW2 partial
// sums are reduced over the group with DPP and accumulated in LDS across
// passes; W2 is updated once at the end.
// ---------------------------------------------------------------------------

static constexpr int kT5 = 256;

template <int OM, int A, bool ZB>
__device__ __forceinline__ void bwd_segment(float* __restrict__ Zt,
                                            unsigned short* __restrict__ dZ16, int Bp, int bl, bool bvalid,
                                            const float* __restrict__ W2, int64_t ldw, int O,
                                            int64_t nbeg, int64_t nend, int g, int NG, int LG,
                                            int pp, const float (&gr)[4][OM],
                                            float* __restrict__ dwl, int64_t r0, bool first) {
  for (int64_t n0 = nbeg + g; n0 < nend; n0 += kU * NG) {
    f32x4 z[kU];
    float w[kU][OM];
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      int64_t n = n0 + u * NG;
      if (n >= nend) n = nend - 1;
      z[u] = load_z4(Zt, ZB, n * Bp + bl);
#pragma unroll
      for (int o = 0; o < OM; ++o) {
        const float v = W2[(int64_t)(o < O ? o : O - 1) * ldw + n];
        w[u][o] = o < O ? v : 0.f;
      }
    }
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      const int64_t n = n0 + u * NG;
      if (n >= nend) break;
      float dw[OM];
#pragma unroll
      for (int o = 0; o < OM; ++o) dw[o] = 0.f;
      f32x4 dz;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float hp;
        const float h = act_fwd_bwd(A, z[u][i], &hp);
        float dh = 0.f;
#pragma unroll
        for (int o = 0; o < OM; ++o) dh = fmaf(gr[i][o], w[u][o], dh);
        dz[i] = dh * hp;
#pragma unroll
        for (int o = 0; o < OM; ++o) dw[o] = fmaf(gr[i][o], h, dw[o]);
      }
      if (bvalid) {
        if (dZ16) {
          typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
          const bf16x4 v = {(__bf16)dz[0], (__bf16)dz[1], (__bf16)dz[2], (__bf16)dz[3]};
          *(bf16x4*)(dZ16 + n * Bp + bl) = v;
        } else {
          *(f32x4*)(Zt + n * Bp + bl) = dz;
        }
      }
#pragma unroll
      for (int o = 0; o < OM; ++o) dw[o] = group_sum_to_last(dw[o], LG);
      if (pp == LG - 1) {
        float* d = dwl + (n - r0) * OM;
#pragma unroll
        for (int o = 0; o < OM; ++o)
          if (o < O) d[o] = first ? dw[o] : d[o] + dw[o];
      }
    }
  }
}

template <int OM, bool GRAD, bool ZB>
__global__ __launch_bounds__(kBlock) void k_m3_bwd(
    float* __restrict__ Zt, unsigned short* __restrict__ dZ16, int Bp,
    float* __restrict__ W2,
    int64_t N, int64_t ldw, int O, const int32_t* __restrict__ mid,
    const int64_t* __restrict__ seg_off, const int32_t* __restrict__ act,
    const float* __restrict__ G, int LG, int slots, float lr, const float* __restrict__ lrm,
    float* __restrict__ dW2) {
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
  if (r0 < N) {
    const int m_first = mid[r0];
    for (int slot = 0; slot < slots; ++slot) {
      const int b = slot * 4 * LG + 4 * pp;
      const bool bvalid = b < Bp;
      const int bl = bvalid ? b : Bp - 4;  // lanes past the batch read a valid row, add nothing
      int64_t n = r0;
      int m = m_first;
      while (n < r1) {
        int64_t se = seg_off[m + 1];
        if (se > r1) se = r1;
        const int a = act[m];
        float gr[4][OM];
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int o = 0; o < OM; ++o) {
            const float v = G[((int64_t)m * Bp + bl + i) * O + (o < O ? o : O - 1)];
            gr[i][o] = (bvalid && o < O) ? v : 0.f;
          }
        const bool first = slot == 0;
        switch (a) {
          case 0: bwd_segment<OM, 0, ZB>(Zt, dZ16, Bp, bl, bvalid, W2, ldw, O, n, se, g, NG, LG, pp, gr, dwl, r0, first); break;
          case 1: bwd_segment<OM, 1, ZB>(Zt, dZ16, Bp, bl, bvalid, W2, ldw, O, n, se, g, NG, LG, pp, gr, dwl, r0, first); break;
          case 2: bwd_segment<OM, 2, ZB>(Zt, dZ16, Bp, bl, bvalid, W2, ldw, O, n, se, g, NG, LG, pp, gr, dwl, r0, first); break;
          case 3: bwd_segment<OM, 3, ZB>(Zt, dZ16, Bp, bl, bvalid, W2, ldw, O, n, se, g, NG, LG, pp, gr, dwl, r0, first); break;
          case 4: bwd_segment<OM, 4, ZB>(Zt, dZ16, Bp, bl, bvalid, W2, ldw, O, n, se, g, NG, LG, pp, gr, dwl, r0, first); break;
          case 5: bwd_segment<OM, 5, ZB>(Zt, dZ16, Bp, bl, bvalid, W2, ldw, O, n, se, g, NG, LG, pp, gr, dwl, r0, first); break;
          case 6: bwd_segment<OM, 6, ZB>(Zt, dZ16, Bp, bl, bvalid, W2, ldw, O, n, se, g, NG, LG, pp, gr, dwl, r0, first); break;
          case 7: bwd_segment<OM, 7, ZB>(Zt, dZ16, Bp, bl, bvalid, W2, ldw, O, n, se, g, NG, LG, pp, gr, dwl, r0, first); break;
          case 8: bwd_segment<OM, 8, ZB>(Zt, dZ16, Bp, bl, bvalid, W2, ldw, O, n, se, g, NG, LG, pp, gr, dwl, r0, first); break;
          case 9: bwd_segment<OM, 9, ZB>(Zt, dZ16, Bp, bl, bvalid, W2, ldw, O, n, se, g, NG, LG, pp, gr, dwl, r0, first); break;
          case 10: bwd_segment<OM, 10, ZB>(Zt, dZ16, Bp, bl, bvalid, W2, ldw, O, n, se, g, NG, LG, pp, gr, dwl, r0, first); break;
          case 11: bwd_segment<OM, 11, ZB>(Zt, dZ16, Bp, bl, bvalid, W2, ldw, O, n, se, g, NG, LG, pp, gr, dwl, r0, first); break;
          default: bwd_segment<OM, 12, ZB>(Zt, dZ16, Bp, bl, bvalid, W2, ldw, O, n, se, g, NG, LG, pp, gr, dwl, r0, first); break;
        }
        n = se;
        ++m;
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
    else W2[(int64_t)o * ldw + n] -= (lrm ? lrm[mid[n]] : lr) * d;
  }
}

template <int OM>
static void m3_bwd_dispatch(float* Zt, bool zb, unsigned short* dZ16, int32_t Bp, float* W2, int64_t N,
                            int64_t ldw, int32_t O, const int32_t* mid, const int64_t* seg_off,
                            const int32_t* act, const float* G, float lr, const float* lrm,
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
  if (dW2 && zb)
    k_m3_bwd<OM, true, true><<<blocks, kBlock, 0, s>>>(Zt, dZ16, Bp, W2, N, ldw, O, mid, seg_off,
                                                       act, G, LG, slots, lr, lrm, dW2);
  else if (dW2)
    k_m3_bwd<OM, true, false><<<blocks, kBlock, 0, s>>>(Zt, dZ16, Bp, W2, N, ldw, O, mid, seg_off,
                                                        act, G, LG, slots, lr, lrm, dW2);
  else if (zb)
    k_m3_bwd<OM, false, true><<<blocks, kBlock, 0, s>>>(Zt, dZ16, Bp, W2, N, ldw, O, mid, seg_off,
                                                        act, G, LG, slots, lr, lrm, dW2);
  else
    k_m3_bwd<OM, false, false><<<blocks, kBlock, 0, s>>>(Zt, dZ16, Bp, W2, N, ldw, O, mid, seg_off,
                                                         act, G, LG, slots, lr, lrm, dW2);
}

hipError_t launch_m3_bwd(float* Zt, unsigned short* dZ16, int32_t Bp, float* W2, int64_t N,
                         int64_t ldw, int32_t O, const int32_t* mid, const int64_t* seg_off,
                         const int32_t* act, const float* G, float lr, const float* lrm,
                         float* dW2, hipStream_t s, bool zb) {
  note_variant("k_m3_bwd", kArithNone);
  if (O <= 2) m3_bwd_dispatch<2>(Zt, zb, dZ16, Bp, W2, N, ldw, O, mid, seg_off, act, G, lr, lrm, dW2, s);
  else if (O <= 4) m3_bwd_dispatch<4>(Zt, zb, dZ16, Bp, W2, N, ldw, O, mid, seg_off, act, G, lr, lrm, dW2, s);
  else if (O <= 8) m3_bwd_dispatch<8>(Zt, zb, dZ16, Bp, W2, N, ldw, O, mid, seg_off, act, G, lr, lrm, dW2, s);
  else if (O <= 10) m3_bwd_dispatch<10>(Zt, zb, dZ16, Bp, W2, N, ldw, O, mid, seg_off, act, G, lr, lrm, dW2, s);
  else m3_bwd_dispatch<16>(Zt, zb, dZ16, Bp, W2, N, ldw, O, mid, seg_off, act, G, lr, lrm, dW2, s);
  return hipGetLastError();
}

}  // namespace pmlpk
