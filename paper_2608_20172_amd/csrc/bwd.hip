// Fused backward pass of the causal Full Relation operator.
//
// Gradient identities used (App. A.1.7, with G = dO and the flow F):
//   H_ij = G_i . v_j,  D_i = sum_k F_ik H_ik = G_i . y_i,  dR_ij = F_ij (H_ij - D_i)
//   Exchange (j < i): F_ij = exp(E_ij - M_i), dU_ij = dR_ij * SiLU'(U_ij),
//                     SiLU'(U) = sigmoid(U) (1 + U (1 - sigmoid(U)))
//   Self (j = i):     F_ii = exp(S_i - M_i + lambda ln i),
//                     dU_ii = dR_ii * S_i (1 - S_i) / tau_S
//   dq = scale * dU k,  dk = scale * dU^T q,  dv = F^T G
//   dlambda = -sum_i ln i sum_{j<i} dR_ij = sum_i ln i * dR_ii
// (softmax-gradient rows sum to zero, so dlambda needs only the diagonal).
// M_i = ln Z_i + lambda ln i is the one statistic saved by the forward pass.
//
// Work split: one workgroup owns 128 keys (32 per wave) and walks over the
// 64-row query tiles at or below its diagonal. Per tile a wave forms the
// evidence block U = Q K^T and dP = dO V^T with keys on lanes and queries in
// accumulator registers, so dV += F^T dO and dK += dU^T Q contract over queries
// straight from registers; Q^T and dO^T come from transpose reads of the
// row-major LDS tiles. dU is written to LDS as [key][query] and read back
// transposed for dQ += dU K over the workgroup's 128 keys, which is added to
// an fp32 accumulator with device atomics.
#include "kernels.h"

#include <algorithm>

namespace rel {

namespace {

constexpr int kBKW = 128;  // keys per workgroup
constexpr int kBQI = 64;   // query rows per iteration
constexpr int kNT = 256;

__global__ void fill_zero_kernel(float* p, int64_t n) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) p[i] = 0.0f;
}

// Per-element backward of one (query row i, key j) entry. Returns F (for dV)
// and dU (for dK, dQ). Mi and the Self exponent are in log2 units.
struct Grad {
  float F, dU;
};

__device__ __forceinline__ Grad exchange_grad(float u, float dp, float Mi2, float Di, float c,
                                              float scale_ln2) {
  (void)scale_ln2;
  const float up = u * c;                              // U log2(e)
  const float sg = fast_rcp(1.0f + fast_exp2(-up));    // sigmoid(U)
  const float wl = up * sg;                            // E log2(e)
  const float F = fast_exp2(wl - Mi2);                 // F_ij = exp(E_ij - M_i)
  const float t1 = __builtin_fmaf(-wl, sg, wl);        // E log2(e) (1 - sigmoid)
  const float dsilu = __builtin_fmaf(t1, kLn2, sg);    // sigmoid + E (1 - sigmoid)
  Grad r;
  r.F = F;
  r.dU = F * (dp - Di) * dsilu;
  return r;
}

template <int D>
__global__ __launch_bounds__(kNT) void bwd_bf16_kernel(BwdArgs a) {
  constexpr int KS = D / 16;
  constexpr int DB = D / 32;
  constexpr int NCH = D / 8;
  constexpr int ROWB = 2 * D;
  constexpr int SWZ = (NCH < 8 ? NCH : 8) - 1;
  constexpr int NLQ = kBQI * NCH / kNT;   // chunks per thread for a query tile
  constexpr int NLK = kBKW * NCH / kNT;   // chunks per thread for the key tile
  constexpr int QROWB = kBQI * 2;         // bytes per row of the dU^T tile
  static_assert(NLQ >= 1, "query tile too small");
  __shared__ __attribute__((aligned(16))) unsigned char Qs[kBQI * ROWB];
  __shared__ __attribute__((aligned(16))) unsigned char dOs[kBQI * ROWB];
  __shared__ __attribute__((aligned(16))) unsigned char Ksh[kBKW * ROWB];
  __shared__ __attribute__((aligned(16))) unsigned char dUt[kBKW * QROWB];
  __shared__ __attribute__((aligned(16))) float Mrow[kBQI];
  __shared__ __attribute__((aligned(16))) float Drow[kBQI];
  __shared__ float red[kNT / 64];

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int n = lane & 31, g = lane >> 5;
  int head, kt;
  if (!map_tile(a.map, blockIdx.x, head, kt, false)) {
    if (tid == 0) a.dlam_part[blockIdx.x] = 0.0f;
    return;
  }
  const int T = a.T;
  const int64_t st = a.st;
  const int64_t hoff = (int64_t)(head / a.H) * a.sb + (int64_t)(head % a.H) * a.sh;
  const bf16* q = (const bf16*)a.q + hoff;
  const bf16* k = (const bf16*)a.k + hoff;
  const bf16* v = (const bf16*)a.v + hoff;
  const bf16* o = (const bf16*)a.o + hoff;
  const bf16* dO = (const bf16*)a.dout + hoff;
  const float* Mst = a.row_stat + (int64_t)head * T;
  float* dq_acc = a.dq_acc + (int64_t)head * T * D;
  const float c = a.scale * kLog2e;
  const float lam = *a.lambda;

  const int j0 = kt * kBKW;
  const int kw0 = j0 + 32 * w;        // first key of this wave
  const int kj = kw0 + n;             // this lane's key
  const bool wave_keys = kw0 < T;

  // B operands of U = Q K^T and dP = dO V^T: lane (n, g) holds K[kj][16 ks + 8 g ..]
  bf16x8 kop[KS], vop[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    if (kj < T) {
      kop[ks] = *(const bf16x8*)(k + kj * st + 16 * ks + 8 * g);
      vop[ks] = *(const bf16x8*)(v + kj * st + 16 * ks + 8 * g);
    } else {
      kop[ks] = bf16x8{};
      vop[ks] = bf16x8{};
    }
  }
  // key tile in LDS, row-major with swizzled 16-byte chunks (B operand of dQ)
#pragma unroll
  for (int jj = 0; jj < NLK; ++jj) {
    const int ci = tid + kNT * jj, row = ci / NCH, ch = ci % NCH, key = j0 + row;
    uintx4 val = uintx4{};
    if (key < T) val = *(const uintx4*)(k + key * st + 8 * ch);
    *(uintx4*)(Ksh + row * ROWB + ((ch ^ (row & SWZ)) << 4)) = val;
  }

  floatx16 dKt[DB], dVt[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) {
    dKt[db] = floatx16{};
    dVt[db] = floatx16{};
  }
  float dlam = 0.0f;

  // transpose-read lane constants
  const int tG = lane >> 4, ti = lane & 15;
  const int t_row = 4 * (tG >> 1) + (ti >> 2);
  const int t_col = 16 * (tG & 1) + 4 * (ti & 3);

  uintx4 qreg[NLQ], dreg[NLQ], oreg[NLQ];
  auto prefetch = [&](int i0) {
#pragma unroll
    for (int jj = 0; jj < NLQ; ++jj) {
      const int ci = tid + kNT * jj, row = ci / NCH, ch = ci % NCH, qi = i0 + row;
      if (qi < T) {
        qreg[jj] = *(const uintx4*)(q + qi * st + 8 * ch);
        dreg[jj] = *(const uintx4*)(dO + qi * st + 8 * ch);
        oreg[jj] = *(const uintx4*)(o + qi * st + 8 * ch);
      } else {
        qreg[jj] = uintx4{};
        dreg[jj] = uintx4{};
        oreg[jj] = uintx4{};
      }
    }
  };

  const int nqt = (T + kBQI - 1) / kBQI;
  const int qt0 = j0 / kBQI;
  prefetch(qt0 * kBQI);
  for (int qt = qt0; qt < nqt; ++qt) {
    const int i0 = qt * kBQI;
    __syncthreads();  // previous tile's Qs, dOs, dUt, Drow, Mrow are no longer read
#pragma unroll
    for (int jj = 0; jj < NLQ; ++jj) {
      const int ci = tid + kNT * jj, row = ci / NCH, ch = ci % NCH;
      const int off = row * ROWB + ((ch ^ (row & SWZ)) << 4);
      *(uintx4*)(Qs + off) = qreg[jj];
      *(uintx4*)(dOs + off) = dreg[jj];
      // D_i = dO_i . O_i, reduced over the NCH lanes holding the row's chunks
      float part = 0.0f;
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        part = __builtin_fmaf(bf16_lo(dreg[jj][t]), bf16_lo(oreg[jj][t]), part);
        part = __builtin_fmaf(bf16_hi(dreg[jj][t]), bf16_hi(oreg[jj][t]), part);
      }
#pragma unroll
      for (int s = 1; s < NCH; s <<= 1) part += __shfl_xor(part, s, 64);
      if (ch == 0) Drow[row] = part;
    }
    if (tid < kBQI) {
      const int qi = i0 + tid;
      Mrow[tid] = qi < T ? Mst[qi] * kLog2e : 0.0f;
    }
    __syncthreads();
    if (qt + 1 < nqt) prefetch(i0 + kBQI);

    // ---- per wave: U and dP blocks for 2 x 32 query rows against 32 keys
    bf16x8 fop[2][2], uop[2][2];  // [query block][half]: packed F and dU operands
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
      const int qb0 = i0 + 32 * qb;
      const bool act = wave_keys && (qb0 + 31 >= kw0) && (qb0 < T);
      if (!act) {
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
          fop[qb][hh] = bf16x8{};
          uop[qb][hh] = bf16x8{};
        }
        continue;
      }
      floatx16 s = floatx16{}, dp = floatx16{};
      const int row = 32 * qb + n;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const int off = row * ROWB + (((2 * ks + g) ^ (row & SWZ)) << 4);
        s = mfma32(*(const bf16x8*)(Qs + off), kop[ks], s);
        dp = mfma32(*(const bf16x8*)(dOs + off), vop[ks], dp);
      }
      const bool full = qb0 > kw0 + 31;  // every row of the block is after every key
      float Fv[16], dUv[16];
#pragma unroll
      for (int rq = 0; rq < 4; ++rq) {
        const int r0 = 32 * qb + 8 * rq + 4 * g;  // tile row of register 4*rq
        const floatx4 M4 = *(const floatx4*)(Mrow + r0);
        const floatx4 D4 = *(const floatx4*)(Drow + r0);
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          const int r = 4 * rq + t;
          const int qi = i0 + r0 + t;
          if (full) {
            const Grad gr = exchange_grad(s[r], dp[r], M4[t], D4[t], c, 0.0f);
            Fv[r] = gr.F;
            dUv[r] = gr.dU;
          } else if (qi > kj && qi < T) {
            const Grad gr = exchange_grad(s[r], dp[r], M4[t], D4[t], c, 0.0f);
            Fv[r] = gr.F;
            dUv[r] = gr.dU;
          } else if (qi == kj && qi < T) {
            // Self entry (diagonal)
            const float S = 1.0f / (1.0f + expf(-s[r] * a.scale * a.inv_tau));
            const float ln_i = logf((float)(qi + 1));
            const float F = exp2f((S + lam * ln_i) * kLog2e - M4[t]);
            const float dR = F * (dp[r] - D4[t]);
            Fv[r] = F;
            dUv[r] = dR * S * (1.0f - S) * a.inv_tau;
            dlam = __builtin_fmaf(ln_i, dR, dlam);
            if (a.dself) a.dself[(int64_t)head * T + qi] = dR;
          } else {
            Fv[r] = 0.0f;
            dUv[r] = 0.0f;
          }
        }
      }
#pragma unroll
      for (int hh = 0; hh < 2; ++hh)
#pragma unroll
        for (int t = 0; t < 8; ++t) {
          fop[qb][hh][t] = f2bf(Fv[8 * hh + t]);
          uop[qb][hh][t] = f2bf(dUv[8 * hh + t]);
        }
    }

    // ---- dV^T += dO^T F and dK^T += Q^T dU  (contraction over the tile's queries)
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
      const int qb0 = i0 + 32 * qb;
      const bool act = wave_keys && (qb0 + 31 >= kw0) && (qb0 < T);
      if (!act) continue;
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        const int ks = 2 * qb + hh;
#pragma unroll
        for (int db = 0; db < DB; ++db) {
          const int col = 32 * db + t_col;
          const int row0 = 16 * ks + t_row, row1 = row0 + 8;
          const int off0 = row0 * ROWB + (((col >> 3) ^ (row0 & SWZ)) << 4) + ((col & 7) << 1);
          const int off1 = row1 * ROWB + (((col >> 3) ^ (row1 & SWZ)) << 4) + ((col & 7) << 1);
          const bf16x8 dOt = tr_operand(dOs + off0, dOs + off1);
          const bf16x8 Qt = tr_operand(Qs + off0, Qs + off1);
          dVt[db] = mfma32(dOt, fop[qb][hh], dVt[db]);
          dKt[db] = mfma32(Qt, uop[qb][hh], dKt[db]);
        }
      }
    }

    // ---- dU^T to LDS: row = key (within the workgroup tile), column = query
    {
      const int krow = 32 * w + n;
#pragma unroll
      for (int qb = 0; qb < 2; ++qb)
#pragma unroll
        for (int rq = 0; rq < 4; ++rq) {
          const int col = 32 * qb + 8 * rq + 4 * g;  // first of 4 consecutive queries
          const int off = krow * QROWB + (((col >> 3) ^ (krow & 7)) << 4) + ((col & 7) << 1);
          *(uintx2*)(dUt + off) = half_of(uop[qb][rq >> 1], rq & 1);
        }
    }
    __syncthreads();

    // ---- dQ (64 x D) += dU (64 x 128) K (128 x D); output blocks split over waves
    constexpr int NOUT = 2 * DB;
#pragma unroll
    for (int ob = w; ob < NOUT; ob += 4) {
      const int qb = ob & 1, db = ob >> 1;
      const int qb0 = i0 + 32 * qb;
      if (qb0 >= T) continue;
      floatx16 acc = floatx16{};
#pragma unroll
      for (int ks = 0; ks < kBKW / 16; ++ks) {
        const int row0 = 16 * ks + t_row, row1 = row0 + 8;  // keys within the workgroup tile
        const int qcol = 32 * qb + t_col;
        const int dcol = 32 * db + t_col;
        const bf16x8 aop =
            tr_operand(dUt + row0 * QROWB + (((qcol >> 3) ^ (row0 & 7)) << 4) + ((qcol & 7) << 1),
                       dUt + row1 * QROWB + (((qcol >> 3) ^ (row1 & 7)) << 4) + ((qcol & 7) << 1));
        const bf16x8 bop =
            tr_operand(Ksh + row0 * ROWB + (((dcol >> 3) ^ (row0 & SWZ)) << 4) + ((dcol & 7) << 1),
                       Ksh + row1 * ROWB + (((dcol >> 3) ^ (row1 & SWZ)) << 4) + ((dcol & 7) << 1));
        acc = mfma32(aop, bop, acc);
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int qi = qb0 + acc_row(r, g);
        if (qi < T) unsafeAtomicAdd(dq_acc + (int64_t)qi * D + 32 * db + n, acc[r]);
      }
    }
  }

  // ---- epilogue: dK = scale * dK^T, dV, and this workgroup's dlambda partial
  if (kj < T) {
    bf16* dk = (bf16*)a.dk + hoff;
    bf16* dv = (bf16*)a.dv + hoff;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int rq = 0; rq < 4; ++rq) {
        const int d0 = 32 * db + 8 * rq + 4 * g;
        bf16x4 kk, vv;
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          kk[t] = f2bf(a.scale * dKt[db][4 * rq + t]);
          vv[t] = f2bf(dVt[db][4 * rq + t]);
        }
        *(bf16x4*)(dk + kj * st + d0) = kk;
        *(bf16x4*)(dv + kj * st + d0) = vv;
      }
  }
#pragma unroll
  for (int s = 32; s >= 1; s >>= 1) dlam += __shfl_xor(dlam, s, 64);
  if (lane == 0) red[w] = dlam;
  __syncthreads();
  if (tid == 0) a.dlam_part[blockIdx.x] = (red[0] + red[1]) + (red[2] + red[3]);
}

// ---------------------------------------------------------------------------
// fp32 kernel (parity path): same decomposition, 32x32x2 f32 MFMAs,
// plain padded LDS tiles.
// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(kNT) void bwd_f32_kernel(BwdArgs a) {
  constexpr int DB = D / 32;
  constexpr int LDR = D + 1;
  constexpr int NCH = D / 4;
  constexpr int NLQ = kBQI * NCH / kNT;
  constexpr int NLK = kBKW * NCH / kNT;
  static_assert(NLQ >= 1, "query tile too small");
  __shared__ float Qs[kBQI * LDR];
  __shared__ float dOs[kBQI * LDR];
  __shared__ float Ksh[kBKW * LDR];
  __shared__ float dUs[kBQI * (kBKW + 1)];  // [query][key]
  __shared__ float Mrow[kBQI];
  __shared__ float Drow[kBQI];
  __shared__ float red[kNT / 64];

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int n = lane & 31, g = lane >> 5;
  int head, kt;
  if (!map_tile(a.map, blockIdx.x, head, kt, false)) {
    if (tid == 0) a.dlam_part[blockIdx.x] = 0.0f;
    return;
  }
  const int T = a.T;
  const int64_t st = a.st;
  const int64_t hoff = (int64_t)(head / a.H) * a.sb + (int64_t)(head % a.H) * a.sh;
  const float* q = (const float*)a.q + hoff;
  const float* k = (const float*)a.k + hoff;
  const float* v = (const float*)a.v + hoff;
  const float* o = (const float*)a.o + hoff;
  const float* dO = (const float*)a.dout + hoff;
  const float* Mst = a.row_stat + (int64_t)head * T;
  float* dq_acc = a.dq_acc + (int64_t)head * T * D;
  const float c = a.scale * kLog2e;
  const float lam = *a.lambda;

  const int j0 = kt * kBKW;
  const int kw0 = j0 + 32 * w;
  const int kj = kw0 + n;
  const bool wave_keys = kw0 < T;

  // B operands: lane (n, g) holds K[kj][2 ks + g]
  float kop[D / 2], vop[D / 2];
#pragma unroll
  for (int ks = 0; ks < D / 2; ++ks) {
    kop[ks] = kj < T ? k[kj * st + 2 * ks + g] : 0.0f;
    vop[ks] = kj < T ? v[kj * st + 2 * ks + g] : 0.0f;
  }
#pragma unroll
  for (int jj = 0; jj < NLK; ++jj) {
    const int ci = tid + kNT * jj, row = ci / NCH, ch = ci % NCH, key = j0 + row;
    floatx4 val = floatx4{};
    if (key < T) val = *(const floatx4*)(k + key * st + 4 * ch);
#pragma unroll
    for (int t = 0; t < 4; ++t) Ksh[row * LDR + 4 * ch + t] = val[t];
  }

  floatx16 dKt[DB], dVt[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) {
    dKt[db] = floatx16{};
    dVt[db] = floatx16{};
  }
  float dlam = 0.0f;

  const int nqt = (T + kBQI - 1) / kBQI;
  const int qt0 = j0 / kBQI;
  for (int qt = qt0; qt < nqt; ++qt) {
    const int i0 = qt * kBQI;
    __syncthreads();
#pragma unroll
    for (int jj = 0; jj < NLQ; ++jj) {
      const int ci = tid + kNT * jj, row = ci / NCH, ch = ci % NCH, qi = i0 + row;
      floatx4 qv = floatx4{}, dv = floatx4{}, ov = floatx4{};
      if (qi < T) {
        qv = *(const floatx4*)(q + qi * st + 4 * ch);
        dv = *(const floatx4*)(dO + qi * st + 4 * ch);
        ov = *(const floatx4*)(o + qi * st + 4 * ch);
      }
      float part = 0.0f;
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        Qs[row * LDR + 4 * ch + t] = qv[t];
        dOs[row * LDR + 4 * ch + t] = dv[t];
        part = __builtin_fmaf(dv[t], ov[t], part);
      }
#pragma unroll
      for (int s = 1; s < NCH; s <<= 1) part += __shfl_xor(part, s, 64);
      if (ch == 0) Drow[row] = part;
    }
    if (tid < kBQI) {
      const int qi = i0 + tid;
      Mrow[tid] = qi < T ? Mst[qi] * kLog2e : 0.0f;
    }
    __syncthreads();

    float Fv[2][16], dUv[2][16];
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
      const int qb0 = i0 + 32 * qb;
      const bool act = wave_keys && (qb0 + 31 >= kw0) && (qb0 < T);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        Fv[qb][r] = 0.0f;
        dUv[qb][r] = 0.0f;
      }
      if (!act) continue;
      floatx16 s = floatx16{}, dp = floatx16{};
      const int row = 32 * qb + n;
#pragma unroll
      for (int ks = 0; ks < D / 2; ++ks) {
        s = mfma32f(Qs[row * LDR + 2 * ks + g], kop[ks], s);
        dp = mfma32f(dOs[row * LDR + 2 * ks + g], vop[ks], dp);
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int tr = 32 * qb + acc_row(r, g);
        const int qi = i0 + tr;
        const float Mi = Mrow[tr], Di = Drow[tr];
        if (qi > kj && qi < T) {
          const Grad gr = exchange_grad(s[r], dp[r], Mi, Di, c, 0.0f);
          Fv[qb][r] = gr.F;
          dUv[qb][r] = gr.dU;
        } else if (qi == kj && qi < T) {
          const float S = 1.0f / (1.0f + expf(-s[r] * a.scale * a.inv_tau));
          const float ln_i = logf((float)(qi + 1));
          const float F = exp2f((S + lam * ln_i) * kLog2e - Mi);
          const float dR = F * (dp[r] - Di);
          Fv[qb][r] = F;
          dUv[qb][r] = dR * S * (1.0f - S) * a.inv_tau;
          dlam = __builtin_fmaf(ln_i, dR, dlam);
          if (a.dself) a.dself[(int64_t)head * T + qi] = dR;
        }
      }
    }
    // dV^T += dO^T F, dK^T += Q^T dU: k-step r covers query acc_row(r, g) of block qb
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
      const int qb0 = i0 + 32 * qb;
      const bool act = wave_keys && (qb0 + 31 >= kw0) && (qb0 < T);
      if (!act) continue;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int tr = 32 * qb + acc_row(r, g);
#pragma unroll
        for (int db = 0; db < DB; ++db) {
          dVt[db] = mfma32f(dOs[tr * LDR + 32 * db + n], Fv[qb][r], dVt[db]);
          dKt[db] = mfma32f(Qs[tr * LDR + 32 * db + n], dUv[qb][r], dKt[db]);
        }
      }
    }
    // dU to LDS as [query][key]
#pragma unroll
    for (int qb = 0; qb < 2; ++qb)
#pragma unroll
      for (int r = 0; r < 16; ++r) dUs[(32 * qb + acc_row(r, g)) * (kBKW + 1) + 32 * w + n] = dUv[qb][r];
    __syncthreads();
    // dQ (64 x D) += dU (64 x 128) K (128 x D)
    constexpr int NOUT = 2 * DB;
    for (int ob = w; ob < NOUT; ob += 4) {
      const int qb = ob & 1, db = ob >> 1;
      const int qb0 = i0 + 32 * qb;
      if (qb0 >= T) continue;
      floatx16 acc = floatx16{};
      for (int ks = 0; ks < kBKW / 2; ++ks)
        acc = mfma32f(dUs[(32 * qb + n) * (kBKW + 1) + 2 * ks + g], Ksh[(2 * ks + g) * LDR + 32 * db + n], acc);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int qi = qb0 + acc_row(r, g);
        if (qi < T) unsafeAtomicAdd(dq_acc + (int64_t)qi * D + 32 * db + n, acc[r]);
      }
    }
  }

  if (kj < T) {
    float* dk = (float*)a.dk + hoff;
    float* dv = (float*)a.dv + hoff;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int d = 32 * db + acc_row(r, g);
        dk[kj * st + d] = a.scale * dKt[db][r];
        dv[kj * st + d] = dVt[db][r];
      }
  }
#pragma unroll
  for (int s = 32; s >= 1; s >>= 1) dlam += __shfl_xor(dlam, s, 64);
  if (lane == 0) red[w] = dlam;
  __syncthreads();
  if (tid == 0) a.dlam_part[blockIdx.x] = (red[0] + red[1]) + (red[2] + red[3]);
}

// dq = scale * dq_acc, written with the problem's strides.
template <typename TO, int D>
__global__ void finalize_dq_kernel(const float* __restrict__ acc, TO* __restrict__ dq, int64_t rows,
                                   int H, int T, int64_t sb, int64_t sh, int64_t st, float scale) {
  constexpr int V4 = D / 4;
  const int64_t total = rows * V4;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < total; idx += stride) {
    const int64_t row = idx / V4;
    const int d0 = (int)(idx % V4) * 4;
    const int64_t head = row / T;
    const int t = (int)(row % T);
    const floatx4 x = *(const floatx4*)(acc + row * D + d0);
    TO* dst = dq + (head / H) * sb + (head % H) * sh + (int64_t)t * st + d0;
#pragma unroll
    for (int e = 0; e < 4; ++e) Elem<TO>::store(dst + e, scale * x[e]);
  }
}

// dlambda = sum of the per-workgroup partials, in a fixed order.
__global__ void finalize_dlam_kernel(const float* __restrict__ part, int np, float* __restrict__ out) {
  __shared__ float s[256];
  float acc = 0.0f;
  for (int i = threadIdx.x; i < np; i += 256) acc += part[i];
  s[threadIdx.x] = acc;
  __syncthreads();
  for (int h = 128; h >= 1; h >>= 1) {
    if ((int)threadIdx.x < h) s[threadIdx.x] += s[threadIdx.x + h];
    __syncthreads();
  }
  if (threadIdx.x == 0) *out = s[0];
}

}  // namespace

int bwd_partials(int N, int T, int D, int dtype) {
  (void)D;
  (void)dtype;
  return (int)grid_size(make_tilemap(N, (T + kBKW - 1) / kBKW));
}

hipError_t launch_bwd(const BwdArgs& a0, int dtype, int D, void* dq_out, hipStream_t stream) {
  BwdArgs a = a0;
  const int N = a.map.N;
  a.map = make_tilemap(N, (a.T + kBKW - 1) / kBKW);
  const int64_t nacc = (int64_t)N * a.T * D;
  {
    const int64_t blocks = std::min<int64_t>((nacc + 1023) / 1024, 4096);
    hipLaunchKernelGGL(fill_zero_kernel, dim3((unsigned)std::max<int64_t>(blocks, 1)), dim3(256), 0,
                       stream, a.dq_acc, nacc);
  }
  const dim3 grid((unsigned)grid_size(a.map)), block(kNT);
  hipEvent_t ev0, ev1;
  const bool prof = profile_slot("bwd", &ev0, &ev1);
  if (prof) (void)hipEventRecord(ev0, stream);
  if (dtype == 1) {
    if (D == 32) hipLaunchKernelGGL(bwd_bf16_kernel<32>, grid, block, 0, stream, a);
    else if (D == 64) hipLaunchKernelGGL(bwd_bf16_kernel<64>, grid, block, 0, stream, a);
    else hipLaunchKernelGGL(bwd_bf16_kernel<128>, grid, block, 0, stream, a);
  } else {
    // fp32 tiles for D = 128 would not fit the 160 KB of LDS; the C-ABI rejects it
    if (D == 32) hipLaunchKernelGGL(bwd_f32_kernel<32>, grid, block, 0, stream, a);
    else if (D == 64) hipLaunchKernelGGL(bwd_f32_kernel<64>, grid, block, 0, stream, a);
    else return hipErrorInvalidValue;
  }
  if (prof) (void)hipEventRecord(ev1, stream);
  const int64_t rows = (int64_t)N * a.T;
  const unsigned fb = (unsigned)std::min<int64_t>((rows * D / 4 + 255) / 256, 8192);
  if (dtype == 1) {
    if (D == 32) hipLaunchKernelGGL((finalize_dq_kernel<bf16, 32>), dim3(fb), dim3(256), 0, stream, a.dq_acc, (bf16*)dq_out, rows, a.H, a.T, a.sb, a.sh, a.st, a.scale);
    else if (D == 64) hipLaunchKernelGGL((finalize_dq_kernel<bf16, 64>), dim3(fb), dim3(256), 0, stream, a.dq_acc, (bf16*)dq_out, rows, a.H, a.T, a.sb, a.sh, a.st, a.scale);
    else hipLaunchKernelGGL((finalize_dq_kernel<bf16, 128>), dim3(fb), dim3(256), 0, stream, a.dq_acc, (bf16*)dq_out, rows, a.H, a.T, a.sb, a.sh, a.st, a.scale);
  } else {
    if (D == 32) hipLaunchKernelGGL((finalize_dq_kernel<float, 32>), dim3(fb), dim3(256), 0, stream, a.dq_acc, (float*)dq_out, rows, a.H, a.T, a.sb, a.sh, a.st, a.scale);
    else if (D == 64) hipLaunchKernelGGL((finalize_dq_kernel<float, 64>), dim3(fb), dim3(256), 0, stream, a.dq_acc, (float*)dq_out, rows, a.H, a.T, a.sb, a.sh, a.st, a.scale);
    else hipLaunchKernelGGL((finalize_dq_kernel<float, 128>), dim3(fb), dim3(256), 0, stream, a.dq_acc, (float*)dq_out, rows, a.H, a.T, a.sb, a.sh, a.st, a.scale);
  }
  return hipGetLastError();
}

hipError_t launch_fill_zero(float* p, int64_t n, hipStream_t stream) {
  const int64_t blocks = std::min<int64_t>((n + 1023) / 1024, 4096);
  hipLaunchKernelGGL(fill_zero_kernel, dim3((unsigned)std::max<int64_t>(blocks, 1)), dim3(256), 0, stream, p, n);
  return hipGetLastError();
}

hipError_t launch_dlambda(const float* part, int np, float* out, hipStream_t stream) {
  hipLaunchKernelGGL(finalize_dlam_kernel, dim3(1), dim3(256), 0, stream, part, np, out);
  return hipGetLastError();
}

}  // namespace rel
