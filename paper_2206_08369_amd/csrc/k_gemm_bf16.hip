// Input-layer GEMMs on the bf16 matrix cores with fp32 accumulation, in
// two arithmetics:
//
// * bf16 operands (the bf16-in / fp32-accumulate precision mode):
//     C[p][q] = sum_k bf16(P[p][k]) * Q[q][k]
// * fp32 accuracy from three-piece splits (the fp32 mode, for the shapes the
//   LDS-resident kernels do not take): both operands fp32, each element split
//   as it is staged into bf16 pieces a = a0 + a1 + a2 (every piece the
//   round-to-nearest of what the previous ones leave, exact for normal a),
//   and every k step taken as the six piece products q0 p0, q1 p0, q0 p1,
//   q1 p1, q2 p0, q0 p2 (in this order) in fp32 accumulation; the three
//   left out are at most 2^-23 of each product, so C carries the error of
//   an fp32 dot product.
//
// P is the big operand (W1 for the forward product of Section 3 step 1,
// dZ^T for dW1): bf16, or fp32 rounded to bf16 (nearest even) or split into
// pieces as it is staged, so the fp32 master weights and activations are
// never copied.  Q is the small operand (the batch or its transpose): bf16,
// or fp32 in the three-piece mode.  Both are k-contiguous.
//
// One v_mfma_f32_32x32x16_bf16 takes a 32x16 tile of Q (lane l: row l%32,
// eight k in half l/32) and a 16x32 tile of P^T laid out the same way, and
// accumulates the 32x32 block D[q][p]; lane l holds p = l%32 and, in
// register 4i+r, q = 8i + 4(l/32) + r, so each lane stores float4s along q.
// Within a 32-wide k stage, lane l of half h owns the 16 consecutive k
// 16h..16h+15 and feeds them to two MFMAs (8 each); A and B use the same
// permutation of k, so the sum is unchanged.
//
// A workgroup of WP x WQ waves computes an MP x MQ tile (MP = 32 TP WP,
// MQ = 32 TQ WQ), each wave TP x TQ MFMA blocks.  Per stage, every thread
// loads 16-byte chunks (eight bf16 or four fp32 k values) of one or more
// operand rows (fp32 converted or split in registers), writes them to LDS
// in MFMA-operand order (fragment (g, s) = 64 lanes x 16 bytes, g the
// 32-row group, s the 8-k step), and every wave reads its fragments with
// conflict-free ds_read_b128.  Two LDS
// stages and two register stages: the global loads of stage k+2 are in
// flight during the MFMAs of stage k, stage k+1 is written to LDS between
// them, and each stage ends with one barrier.
//
// In the three-piece mode each operand has three LDS planes per stage (the
// pieces), the stage is 16 k deep (one MFMA k step), global loads run two
// stages ahead, the next stage is split into LDS between the products of
// the current one, and k past K reads as zero on both operands.
//
// Tile order is XCD-aware: workgroup b runs on XCD b % 8, and the nqt
// q-tiles of one p-tile are consecutive workgroups of the same XCD, so the
// p-tile (the operand streamed from HBM) is fetched once and served from
// that XCD's L2 to the other q-tiles.

#include "device_common.h"

#include <type_traits>

namespace pmlpk {

namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// Three bf16 pieces of four fp32 values: v = p0 + p1 + p2, each piece the
// round-to-nearest-even of the remainder (exact subtractions in fp32).
__device__ __forceinline__ void split3x4(const f32x4& v, bf16x4& p0, bf16x4& p1, bf16x4& p2) {
  p0 = __builtin_convertvector(v, bf16x4);
  const f32x4 r1 = v - __builtin_convertvector(p0, f32x4);
  p1 = __builtin_convertvector(r1, bf16x4);
  p2 = __builtin_convertvector(r1 - __builtin_convertvector(p1, f32x4), bf16x4);
}

template <int TP, int TQ, int WP, int WQ, int KS, bool PB, int EPI, bool X3 = false>
__global__ __launch_bounds__(64 * WP * WQ) __attribute__((amdgpu_waves_per_eu(2)))
void k_gemm_bf(GemmBfArgs a, int npt, int nqt) {
  constexpr int NT = 64 * WP * WQ;
  constexpr int MP = 32 * TP * WP, MQ = 32 * TQ * WQ;
  constexpr int KH = KS / 2;   // k owned by one lane half of an MFMA operand
  constexpr int NS = KS / 16;  // MFMA k-steps per stage
  // Loader: consecutive lanes read consecutive 16-byte chunks of one row, so
  // one wave load covers whole cache lines of a few rows.  fp32 P chunks are
  // four fp32 (half of one lane's 8-k bf16 operand entry); bf16 P (PB) and
  // Q chunks are eight bf16.
  // In the three-piece mode Q is fp32 too (four per chunk).
  static_assert(!X3 || (!PB && KS == 16), "three-piece mode: fp32 P, one k step per stage");
  constexpr int PE = PB ? 8 : 4;            // P elements per chunk
  constexpr int QE = X3 ? 4 : 8;            // Q elements per chunk
  constexpr int CP = KS / PE, CQ = KS / QE;  // chunks per row and stage
  constexpr int LP = (MP * CP + NT - 1) / NT, LQ = (MQ * CQ + NT - 1) / NT;
  static_assert((MP * CP) % NT == 0 || MP * CP < NT, "loader shape");
  static_assert((MQ * CQ) % NT == 0 || MQ * CQ < NT, "loader shape");
  static_assert((MP * CP) % 64 == 0 && (MQ * CQ) % 64 == 0, "loader shape");
  constexpr int PS = MP * 2 * NS, QS = MQ * 2 * NS;  // 16-byte entries per plane and stage
  constexpr int PL = X3 ? 3 : 1;                     // planes (pieces) per operand
  constexpr int SS = PL * (PS + QS);                 // entries per stage
  // epilogue scratch: QB adjacent 32 x 32 blocks per wave, rows padded by 4
  constexpr int QB = TQ % 2 == 0 ? 2 : 1, LDT = 32 * QB + 4;
  constexpr int SCR = NT / 64 * 32 * LDT / 4;  // 16-byte units
  constexpr int LDSN = 2 * SS > SCR ? 2 * SS : SCR;
  __shared__ u32x4 lds[LDSN];

  const int blk = blockIdx.x;
  const int xcd = blk & 7, jb = blk >> 3;
  const int pt = (jb / nqt) * 8 + xcd;
  const int qt = jb - (jb / nqt) * nqt;
  if (pt >= npt) return;
  const int64_t p0 = (int64_t)pt * MP;
  const int q0 = qt * MQ;
  const int t = threadIdx.x, lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int wp = wave / WQ, wq = wave - (wave / WQ) * WQ;

  // LDS position of operand entry (32-row group g, k-step s, MFMA lane l):
  // fragment (g, s) is 64 consecutive 16-byte entries; inside it lane l's
  // entry sits at l ^ 8(l/32) ^ 4(s&1), a permutation that keeps the MFMA
  // reads conflict-free and spreads the loader's scattered writes evenly
  // over the banks.
  auto entry = [](int g, int s, int l) {
    return (g * NS + s) * 64 + (l ^ (8 * (l >> 5)) ^ (4 * (s & 1)));
  };
  typedef typename std::conditional<PB, unsigned short, float>::type PT;
  const PT* pbase = PB ? (const PT*)a.Pb : (const PT*)a.P;
  // A thread's chunks e = 0 .. LP-1 lie RP rows apart at the same k (and its
  // Q chunks RQ rows apart), so their LDS entries are a fixed distance
  // apart; addresses are formed at each load from the first row, which
  // keeps three values per operand in registers instead of a pointer per
  // chunk.
  constexpr int RP = NT / CP, RQ = NT / CQ;
  static_assert(LP == 1 || (NT % CP == 0 && RP % 32 == 0), "loader rows");
  static_assert(LQ == 1 || (NT % CQ == 0 && RQ % 32 == 0), "loader rows");
  int prow, pk, poff;  // first row, k of the chunk within the stage, LDS byte offset
  {
    const int idx = t % (MP * CP), row = idx / CP, c = idx % CP;
    const int k = PE * c, h = k / KH, st = (k % KH) / 8;
    prow = row;
    pk = k;
    poff = entry(row >> 5, st, (row & 31) + 32 * h) * 16 + (PB ? 0 : 8 * (c & 1));
  }
  typedef typename std::conditional<X3, float, unsigned short>::type QT;
  const QT* qbase = X3 ? (const QT*)a.Qf : (const QT*)a.Q;
  int qrow, qk, qoff;
  {
    const int idx = t % (MQ * CQ), row = idx / CQ, c = idx % CQ;
    const int k = QE * c, h = k / KH, st = (k % KH) / 8;
    qrow = row;
    qk = k;
    qoff = entry(row >> 5, st, (row & 31) + 32 * h) * 16 + (X3 ? 8 * (c & 1) : 0);
  }
  constexpr int PSTEP = RP / 32 * NS * 64 * 16, QSTEP = RQ / 32 * NS * 64 * 16;  // bytes

  // Global loads of one stage into registers, without branches so that the
  // compiler's wait counts stay exact: the stage index is clamped to the
  // last stage, and P reads at or past kp (the last stage when kp is not a
  // multiple of KS) are redirected to the start of the row, a finite value
  // that meets the zero padding of Q.  In the three-piece mode Q reads at or
  // past K are redirected the same way, and both operands' chunks past the
  // end are stored as zero.
  struct Regs {
    u32x4 p[LP];
    u32x4 q[LQ];
    int k0;
  };
  const int K = a.K, kp = a.kp;
  const int nk = (K + KS - 1) / KS;
  auto load = [&](Regs& r, int kt) {
    const int k0 = min(kt, nk - 1) * KS;
    r.k0 = k0;
    const int pkk = k0 + pk < kp ? k0 + pk : 0;
#pragma unroll
    for (int e = 0; e < LP; ++e) {
      if (MP * CP < NT && t >= MP * CP) continue;
      const int64_t p = min(p0 + prow + e * RP, a.NP - 1);
      r.p[e] = *(const u32x4*)(pbase + p * a.ldp + pkk);
    }
    const int qkk = !X3 || k0 + qk < K ? k0 + qk : 0;
#pragma unroll
    for (int e = 0; e < LQ; ++e) {
      if (MQ * CQ < NT && t >= MQ * CQ) continue;
      const int q = min(q0 + qrow + e * RQ, a.NQ - 1);
      r.q[e] = *(const u32x4*)(qbase + (int64_t)q * a.ldq + qkk);
    }
  };
  auto store = [&](const Regs& r, int sb) {
    char* ps = (char*)(lds + sb * SS);
    char* qs = ps + PL * PS * 16;
    if constexpr (X3) {
#pragma unroll
      for (int e = 0; e < LP; ++e) {
        if (MP * CP < NT && t >= MP * CP) continue;
        const f32x4 f = r.k0 + pk < kp ? __builtin_bit_cast(f32x4, r.p[e]) : f32x4{0, 0, 0, 0};
        bf16x4 v0, v1, v2;
        split3x4(f, v0, v1, v2);
        char* d = ps + poff + e * PSTEP;
        *(bf16x4*)d = v0;
        *(bf16x4*)(d + PS * 16) = v1;
        *(bf16x4*)(d + 2 * PS * 16) = v2;
      }
#pragma unroll
      for (int e = 0; e < LQ; ++e) {
        if (MQ * CQ < NT && t >= MQ * CQ) continue;
        const f32x4 f = r.k0 + qk < K ? __builtin_bit_cast(f32x4, r.q[e]) : f32x4{0, 0, 0, 0};
        bf16x4 v0, v1, v2;
        split3x4(f, v0, v1, v2);
        char* d = qs + qoff + e * QSTEP;
        *(bf16x4*)d = v0;
        *(bf16x4*)(d + QS * 16) = v1;
        *(bf16x4*)(d + 2 * QS * 16) = v2;
      }
      return;
    }
#pragma unroll
    for (int e = 0; e < LP; ++e) {
      if (MP * CP < NT && t >= MP * CP) continue;
      if (PB) {
        *(u32x4*)(ps + poff + e * PSTEP) = r.p[e];
      } else {
        const f32x4 f = __builtin_bit_cast(f32x4, r.p[e]);
        bf16x4 v;
        v[0] = (__bf16)f[0];
        v[1] = (__bf16)f[1];
        v[2] = (__bf16)f[2];
        v[3] = (__bf16)f[3];
        *(bf16x4*)(ps + poff + e * PSTEP) = v;
      }
    }
#pragma unroll
    for (int e = 0; e < LQ; ++e) {
      if (MQ * CQ < NT && t >= MQ * CQ) continue;
      *(u32x4*)(qs + qoff + e * QSTEP) = r.q[e];
    }
  };

  f32x16 acc[TQ][TP];
#pragma unroll
  for (int i = 0; i < TQ; ++i)
#pragma unroll
    for (int j = 0; j < TP; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  // bf16 operands: NS k steps of TQ x TP products; `mid` runs after the
  // first half of them.
  auto compute = [&](int sb, auto mid) {
    const u32x4* ps = lds + sb * SS;
    const u32x4* qs = ps + PL * PS;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      if (s == NS / 2) {
        __builtin_amdgcn_sched_barrier(0);
        mid();
        __builtin_amdgcn_sched_barrier(0);
      }
      bf16x8 pf[TP], qf[TQ];
#pragma unroll
      for (int j = 0; j < TP; ++j)
        pf[j] = __builtin_bit_cast(bf16x8, ps[entry(wp * TP + j, s, lane)]);
#pragma unroll
      for (int i = 0; i < TQ; ++i)
        qf[i] = __builtin_bit_cast(bf16x8, qs[entry(wq * TQ + i, s, lane)]);
#pragma unroll
      for (int i = 0; i < TQ; ++i)
#pragma unroll
        for (int j = 0; j < TP; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qf[i], pf[j], acc[i][j], 0, 0, 0);
    }
  };

  // Three-piece mode: the fragments of planes 0 and 1, the four piece
  // products they make (q0 p0, q1 p0, q0 p1, q1 p1), then the fragments of
  // plane 2 (in the registers plane 1 held) and `mid`, then q2 p0 and q0 p2.
  // Each pass over the TQ x TP blocks issues independent MFMAs back to back.
  auto compute_x3 = [&](int sb, auto mid) {
    const u32x4* ps = lds + sb * SS;
    const u32x4* qs = ps + PL * PS;
    bf16x8 p0[TP], q0[TQ], p1[TP], q1[TQ];
    auto frags = [&](int c, bf16x8(&pf)[TP], bf16x8(&qf)[TQ]) {
#pragma unroll
      for (int j = 0; j < TP; ++j)
        pf[j] = __builtin_bit_cast(bf16x8, ps[c * PS + entry(wp * TP + j, 0, lane)]);
#pragma unroll
      for (int i = 0; i < TQ; ++i)
        qf[i] = __builtin_bit_cast(bf16x8, qs[c * QS + entry(wq * TQ + i, 0, lane)]);
    };
    auto pass = [&](const bf16x8(&qf)[TQ], const bf16x8(&pf)[TP]) {
#pragma unroll
      for (int i = 0; i < TQ; ++i)
#pragma unroll
        for (int j = 0; j < TP; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qf[i], pf[j], acc[i][j], 0, 0, 0);
    };
    frags(0, p0, q0);
    frags(1, p1, q1);
    pass(q0, p0);
    pass(q1, p0);
    pass(q0, p1);
    pass(q1, p1);
    __builtin_amdgcn_sched_barrier(0);
    frags(2, p1, q1);
    mid();
    __builtin_amdgcn_sched_barrier(0);
    pass(q1, p0);
    pass(q0, p1);
  };

  // Stage kt+2 is loaded while stage kt is multiplied, and stage kt+1
  // (loaded a stage earlier) is written to the other LDS buffer (split into
  // pieces in the three-piece mode) between the products of stage kt: one
  // barrier per stage, and the LDS writes overlap the matrix work.  The
  // other buffer is free then: its last reader, stage kt-1, ended before
  // the previous barrier.
  auto stage = [&](int sb, auto mid) {
    if constexpr (X3)
      compute_x3(sb, mid);
    else
      compute(sb, mid);
  };
  {
    Regs r0, r1;
    load(r0, 0);
    store(r0, 0);
    load(r1, 1);
    __syncthreads();
    for (int kt = 0;; kt += 2) {
      load(r0, kt + 2);
      stage(0, [&] {
        if (kt + 1 < nk) store(r1, 1);
      });
      if (kt + 1 >= nk) break;
      __syncthreads();
      load(r1, kt + 3);
      stage(1, [&] {
        if (kt + 2 < nk) store(r0, 0);
      });
      if (kt + 2 >= nk) break;
      __syncthreads();
    }
  }

  // Epilogue: QB horizontally adjacent 32 x 32 blocks at a time go through a
  // per-wave LDS scratch so that 8*QB consecutive lanes hold one row's 32*QB
  // consecutive q; every store (and the read of the SGD update) then covers
  // whole row segments -- 256 bytes of fp32 and a full 128-byte line of the
  // bf16 copy when QB = 2 -- instead of 16 bytes of 32 rows.  Scratch rows
  // are padded by four floats: the column writes of the MFMA layout and the
  // row reads both stay conflict-free.
  float* scr = (float*)lds + wave * (32 * LDT);
  __syncthreads();  // every wave is done with the operand stages
#pragma unroll
  for (int j = 0; j < TP; ++j)
#pragma unroll
    for (int i0 = 0; i0 < TQ; i0 += QB) {
#pragma unroll
      for (int ib = 0; ib < QB; ++ib)
#pragma unroll
        for (int i4 = 0; i4 < 4; ++i4) {
          const int i = i0 + ib;
          const f32x4 v = {acc[i][j][4 * i4], acc[i][j][4 * i4 + 1], acc[i][j][4 * i4 + 2],
                           acc[i][j][4 * i4 + 3]};
          *(f32x4*)(scr + (lane & 31) * LDT + 32 * ib + 8 * i4 + 4 * (lane >> 5)) = v;
        }
      __syncthreads();
      const int64_t pb = p0 + 32 * (wp * TP + j);
      const int qb = q0 + 32 * (wq * TQ + i0);
      constexpr int LPR = 8 * QB;  // lanes per row
      constexpr int NPASS = 32 * LPR / 64;
      // Every global load of the round (the weights to update, per-model
      // rates, feature-mask words) comes before its first store: a load
      // after a store to `out` may not be moved above it, so each pass would
      // wait a full memory round trip.  Lanes past the edge load from the
      // last row and column and store nothing.
      f32x4 wv[NPASS];
      float lrv[NPASS];
      uint32_t mbits[NPASS];
      if constexpr (EPI != EPI_STORE) {
#pragma unroll
        for (int pass = 0; pass < NPASS; ++pass) {
          const int r = pass * (64 / LPR) + lane / LPR, c4 = 4 * (lane % LPR);
          const int64_t p = min(pb + r, a.NP - 1);
          const int q = min(qb + c4, a.NQ - 4);
          const int m = (a.lrm || a.fmask) ? a.mid[p] : 0;
          // masked features: zero gradient, so their weights stay 0
          mbits[pass] = a.fmask ? a.fmask[(int64_t)m * a.fmw + (q >> 5)] >> (q & 31) : 0xFu;
          if constexpr (EPI == EPI_SGD) {
            lrv[pass] = a.lrm ? a.lrm[m] : a.lr;
            wv[pass] = *(const f32x4*)(a.out + p * a.ldo + q);
          }
        }
      }
#pragma unroll
      for (int pass = 0; pass < NPASS; ++pass) {
        const int r = pass * (64 / LPR) + lane / LPR, c4 = 4 * (lane % LPR);
        const f32x4 v0 = *(const f32x4*)(scr + r * LDT + c4);
        const int64_t p = pb + r;
        const int q = qb + c4;
        if (p >= a.NP || q >= a.NQ) continue;
        float* o = a.out + p * a.ldo + q;
        if constexpr (EPI == EPI_STORE) {
          if (a.outb) {  // the bf16 storage mode keeps Z as bfloat16 (nearest even)
            const bf16x4 zb = {(__bf16)v0[0], (__bf16)v0[1], (__bf16)v0[2], (__bf16)v0[3]};
            *(bf16x4*)(a.outb + p * a.ldob + q) = zb;
          } else {
            *(f32x4*)o = v0;
          }
        } else {
          const uint32_t b = mbits[pass];
          const f32x4 v = {(b & 1u) ? v0[0] : 0.f, (b & 2u) ? v0[1] : 0.f, (b & 4u) ? v0[2] : 0.f,
                           (b & 8u) ? v0[3] : 0.f};
          if constexpr (EPI == EPI_SGD) {
            const f32x4 w = wv[pass] - lrv[pass] * v;
            *(f32x4*)o = w;
            if (a.outb) {
              const bf16x4 wb = {(__bf16)w[0], (__bf16)w[1], (__bf16)w[2], (__bf16)w[3]};
              *(bf16x4*)(a.outb + p * a.ldob + q) = wb;
            }
          } else {
#pragma unroll
            for (int e = 0; e < 4; ++e)
              if (q + e < a.ncols) o[e] = v[e];
              else if (q + e == a.bcol && a.db1) a.db1[p] = v[e];
          }
        }
      }
      __syncthreads();
    }
}

template <int TP, int TQ, int WP, int WQ, int KS, bool PB, bool X3 = false>
hipError_t gemm_bf_go(const GemmBfArgs& a, int epi, hipStream_t s) {
  constexpr int MP = 32 * TP * WP, MQ = 32 * TQ * WQ;
  const int64_t npt64 = (a.NP + MP - 1) / MP;
  const int nqt = (a.NQ + MQ - 1) / MQ;
  const int64_t nblk = ((npt64 + 7) / 8) * 8 * nqt;
  if (nblk > 0x7fffffff) return hipErrorInvalidValue;
  const int npt = (int)npt64;
  const dim3 grid((unsigned)nblk), block(64 * WP * WQ);
  switch (epi) {
    case EPI_STORE:
      k_gemm_bf<TP, TQ, WP, WQ, KS, PB, EPI_STORE, X3><<<grid, block, 0, s>>>(a, npt, nqt);
      break;
    case EPI_SGD:
      k_gemm_bf<TP, TQ, WP, WQ, KS, PB, EPI_SGD, X3><<<grid, block, 0, s>>>(a, npt, nqt);
      break;
    default:
      k_gemm_bf<TP, TQ, WP, WQ, KS, PB, EPI_GRAD, X3><<<grid, block, 0, s>>>(a, npt, nqt);
      break;
  }
  return hipGetLastError();
}

}  // namespace

bool gemm_bf16_args_ok(const GemmBfArgs& a) {
  const int pe = a.Pb ? 8 : 4;
  if (!(a.NP > 0 && a.NQ > 0 && a.K > 0 && a.K % 4 == 0 && a.NQ % 4 == 0 &&
        (a.P != nullptr) != (a.Pb != nullptr) && a.kp > 0 && a.kp % pe == 0 && a.ldp >= a.kp &&
        a.ldp % 4 == 0))
    return false;
  if (a.Qf)  // three-piece mode: fp32 P and Q, rows 16-byte aligned
    return a.P != nullptr && a.Q == nullptr && a.ldq % 4 == 0 && a.ldq >= a.K;
  return a.Q != nullptr && a.ldq % 64 == 0 && a.ldq >= ((a.K + 63) / 64) * 64;
}

template <int TP, int TQ, int WP, int WQ, int KS>
hipError_t gemm_bf_p(const GemmBfArgs& a, int epi, hipStream_t s) {
  if (a.Pb) return gemm_bf_go<TP, TQ, WP, WQ, KS, true>(a, epi, s);
  return gemm_bf_go<TP, TQ, WP, WQ, KS, false>(a, epi, s);
}

hipError_t launch_gemm_bf16(const GemmBfArgs& a, int epi, hipStream_t s) {
  if (a.Qf) {
    note_variant("k_gemm_x3", kArithX3);
    if (a.NP <= 0 || a.NQ <= 0) return hipSuccess;
    if (!gemm_bf16_args_ok(a)) return hipErrorInvalidValue;
    // 16-k stages of three planes per operand; four-wave workgroups of at
    // most 72 KB of LDS, two per CU, so that one's barrier waits and
    // epilogue overlap the other's products
    if (a.NQ <= 64) return gemm_bf_go<4, 1, 2, 2, 16, false, true>(a, epi, s);
    if (a.NQ <= 128) return gemm_bf_go<2, 2, 2, 2, 16, false, true>(a, epi, s);
    return gemm_bf_go<4, 2, 2, 4, 16, false, true>(a, epi, s);
  }
  note_variant("k_gemm_bf", kArithBf16);
  if (a.NP <= 0 || a.NQ <= 0) return hipSuccess;
  if (!gemm_bf16_args_ok(a)) return hipErrorInvalidValue;
  // q tile no wider than needed for small q; 256 x 256 tiles otherwise (the
  // largest that keeps the accumulators in registers, and the least operand
  // traffic per product from L2)
  if (a.NQ <= 64) return gemm_bf_p<4, 1, 2, 2, 32>(a, epi, s);
  if (a.NQ <= 128) return gemm_bf_p<2, 2, 2, 2, 32>(a, epi, s);
  return gemm_bf_p<4, 2, 2, 4, 32>(a, epi, s);
}

}  // namespace pmlpk
