// Fused forward pass of the causal Full Relation operator (FlashRelation).
//
// One workgroup = 4 waves = 128 query rows of one head; each wave owns 32 rows.
// Key/value tiles of 64 rows stream HBM -> registers -> LDS. Per tile a wave
// computes the transposed evidence block U^T = K Q^T with 32x32 MFMAs, so each
// lane holds one query row and 16 keys per block: the row reductions of the
// online scan stay inside the lane, plus one exchange with the partner lane
// 32 away. The Exchange scan keeps (m, l, z) per row exactly as in eqs. (11)-(12)
// of Sec. 5.1 / App. A.3, with Self excluded; Self and the count correction
// join only in the epilogue (eq. 13).
//
// Running reference m. SiLU(U) >= -0.2785, so exp(E - m) with m = 0 can never
// underflow to an all-zero row; the reference is raised only when a tile's
// largest E exceeds it by more than 8 (in log2 units), which keeps every
// exp2 argument <= 8 and the sums far from fp32 overflow. Any reference gives
// the same ratios z/l and L^E = m + ln l, so the result is exact.
#include "kernels.h"

namespace rel {

namespace {

constexpr int kBQ = 128;  // query rows per workgroup
constexpr int kBK = 64;   // keys per tile
constexpr int kNT = 256;  // threads per workgroup
constexpr float kRescale = 8.0f;

// Exchange logits of one 32x32 block, in place: s[r] (raw q.k) becomes
// E*log2(e) - m, or -inf where j >= i. Tracks the diagonal entry (Self).
__device__ __forceinline__ void exchange_logits(floatx16& s, bool diag_block, int n, int g, float c,
                                                float m, float& mx, float& uii, bool& hasd) {
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int kr = acc_row(r, g);
    const float x = s[r];
    if (diag_block && kr == n) {
      uii = x;
      hasd = true;
    }
    const float up = x * c;                                // U * log2(e)
    const float sg = fast_rcp(1.0f + fast_exp2(-up));      // sigmoid(U)
    float e = __builtin_fmaf(up, sg, -m);                  // SiLU(U) * log2(e) - m
    if (diag_block && kr >= n) e = kNegInf;                // strictly historical: j < i
    s[r] = e;
    mx = fmaxf(mx, e);
  }
}

struct RowEpilogue {
  float g, omg, inv_l, LE, lnZ, S;
};

// Completes row i (one-based index i1) from the terminal scan state (eqs. 12-13):
// L^E = m + ln l, A = L^E - lambda ln i, g = sigmoid(A - S), 1-g = sigmoid(S - A).
__device__ __forceinline__ RowEpilogue row_epilogue(float m_log2, float l, float uii, float scale,
                                                    float inv_tau, float lam, float ln_i) {
  RowEpilogue e;
  e.S = 1.0f / (1.0f + expf(-uii * scale * inv_tau));
  if (l > 0.0f) {
    e.LE = (m_log2 + log2f(l)) * kLn2;
    const float A = e.LE - lam * ln_i;
    const float d = A - e.S;
    e.g = 1.0f / (1.0f + expf(-d));
    e.omg = 1.0f / (1.0f + expf(d));
    e.lnZ = fmaxf(e.S, A) + log1pf(expf(-fabsf(d)));
    e.inv_l = e.g / l;
  } else {  // empty history (row 1): g = 0, y = v (App. A.1.8)
    e.LE = kNegInf;
    e.g = 0.0f;
    e.omg = 1.0f;
    e.lnZ = e.S;
    e.inv_l = 0.0f;
  }
  return e;
}

__device__ __forceinline__ void store_row_stats(const FwdArgs& a, int64_t ridx, const RowEpilogue& e,
                                                float lam, float ln_i) {
  if (a.row_stat) a.row_stat[ridx] = e.lnZ + lam * ln_i;
  if (a.self_mass) a.self_mass[ridx] = e.omg;
  if (a.exch_mass) a.exch_mass[ridx] = e.g;
  if (a.exch_lse) a.exch_lse[ridx] = e.LE;
}

// ---------------------------------------------------------------------------
// bf16 kernel
// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(kNT, 2) void fwd_bf16_kernel(FwdArgs a) {
  constexpr int KS = D / 16;                      // MFMA k-steps over d
  constexpr int DB = D / 32;                      // 32-row blocks of O^T
  constexpr int NCH = D / 8;                      // 16-byte chunks per tile row
  constexpr int SB = kBK / 32;                    // 32-key blocks per tile
  constexpr int ROWB = D * 2;                     // bytes per tile row
  constexpr int SWZ = (NCH < 8 ? NCH : 8) - 1;    // chunk swizzle mask
  constexpr int NLD = kBK * NCH / kNT;            // chunks per thread per tensor
  static_assert(NLD >= 1, "tile too small for the workgroup");
  __shared__ __attribute__((aligned(16))) unsigned char lds[2 * kBK * ROWB];
  unsigned char* Ks = lds;
  unsigned char* Vs = lds + kBK * ROWB;

  int head, qt;
  if (!map_tile(a.map, blockIdx.x, head, qt, true)) return;
  const int T = a.T;
  const int64_t st = a.st;
  const int64_t hoff = (int64_t)(head / a.H) * a.sb + (int64_t)(head % a.H) * a.sh;
  const bf16* q = (const bf16*)a.q + hoff;
  const bf16* k = (const bf16*)a.k + hoff;
  const bf16* v = (const bf16*)a.v + hoff;
  bf16* o = (bf16*)a.o + hoff;

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int n = lane & 31, g = lane >> 5;
  const int i0 = qt * kBQ, qr0 = i0 + 32 * w, qi = qr0 + n;
  const bool wave_live = qr0 < T;
  const float c = a.scale * kLog2e;

  // B operand of U^T = K Q^T: lane (n, g) holds Q[qi][16 ks + 8 g .. +7]
  bf16x8 qop[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    if (qi < T) qop[ks] = *(const bf16x8*)(q + qi * st + 16 * ks + 8 * g);
    else qop[ks] = bf16x8{};
  }

  uintx4 kreg[NLD], vreg[NLD];
  auto prefetch = [&](int j0) {
#pragma unroll
    for (int j = 0; j < NLD; ++j) {
      const int ci = tid + kNT * j, row = ci / NCH, ch = ci % NCH, key = j0 + row;
      if (key < T) {
        kreg[j] = *(const uintx4*)(k + key * st + 8 * ch);
        vreg[j] = *(const uintx4*)(v + key * st + 8 * ch);
      } else {
        kreg[j] = uintx4{};
        vreg[j] = uintx4{};
      }
    }
  };
  auto stage = [&]() {
#pragma unroll
    for (int j = 0; j < NLD; ++j) {
      const int ci = tid + kNT * j, row = ci / NCH, ch = ci % NCH;
      const int off = row * ROWB + ((ch ^ (row & SWZ)) << 4);
      *(uintx4*)(Ks + off) = kreg[j];
      *(uintx4*)(Vs + off) = vreg[j];
    }
  };

  float m = 0.0f, l = 0.0f, uii = 0.0f;
  bool hasd = false;
  floatx16 oacc[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) oacc[db] = floatx16{};

  // lane constants of the transpose read of V: 16-lane group G, index i in group
  const int tG = lane >> 4, ti = lane & 15;
  const int t_row = 4 * (tG >> 1) + (ti >> 2);               // + 16 ks + 8 h
  const int t_col = 16 * (tG & 1) + 4 * (ti & 3);            // + 32 db (elements)

  const int kmax = min(i0 + kBQ, T) - 1;  // the diagonal of the last row is included
  const int nkt = kmax / kBK + 1;
  prefetch(0);
  for (int kt = 0; kt < nkt; ++kt) {
    __syncthreads();
    stage();
    __syncthreads();
    if (kt + 1 < nkt) prefetch((kt + 1) * kBK);
    if (!wave_live) continue;
    const int j0 = kt * kBK;

    floatx16 sacc[SB];
    bool act[SB];
#pragma unroll
    for (int sb = 0; sb < SB; ++sb) {
      act[sb] = (j0 + 32 * sb) <= qr0;  // some key of the block is <= some row of the wave
      sacc[sb] = floatx16{};
      if (act[sb]) {
        const int row = 32 * sb + n;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          const bf16x8 kop =
              *(const bf16x8*)(Ks + row * ROWB + (((2 * ks + g) ^ (row & SWZ)) << 4));
          sacc[sb] = mfma32(kop, qop[ks], sacc[sb]);
        }
      }
    }

    float mx = kNegInf;
#pragma unroll
    for (int sb = 0; sb < SB; ++sb)
      if (act[sb]) exchange_logits(sacc[sb], j0 + 32 * sb == qr0, n, g, c, m, mx, uii, hasd);
    mx = fmaxf(mx, xor32(mx));
    if (wave_any(mx > kRescale)) {
      const float d = fmaxf(mx, 0.0f);
      m += d;
      const float al = fast_exp2(-d);
      l *= al;
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int r = 0; r < 16; ++r) oacc[db][r] *= al;
#pragma unroll
      for (int sb = 0; sb < SB; ++sb)
#pragma unroll
        for (int r = 0; r < 16; ++r) sacc[sb][r] -= d;
    }

#pragma unroll
    for (int sb = 0; sb < SB; ++sb) {
      if (!act[sb]) continue;
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        bf16x8 pop;
#pragma unroll
        for (int t = 0; t < 8; ++t) {
          const float p = fast_exp2(sacc[sb][8 * hh + t]);
          l += p;
          pop[t] = f2bf(p);
        }
        const int ks = 2 * sb + hh;
#pragma unroll
        for (int db = 0; db < DB; ++db) {
          const int col = 32 * db + t_col;
          const int row0 = 16 * ks + t_row, row1 = row0 + 8;
          const bf16x8 vop = tr_operand(
              Vs + row0 * ROWB + (((col >> 3) ^ (row0 & SWZ)) << 4) + ((col & 7) << 1),
              Vs + row1 * ROWB + (((col >> 3) ^ (row1 & SWZ)) << 4) + ((col & 7) << 1));
          oacc[db] = mfma32(vop, pop, oacc[db]);
        }
      }
    }
  }
  if (!wave_live) return;

  // ---- epilogue: combine the two lane halves of each row, then eq. (13)
  const float lt = l + xor32(l);
  const float u_other = xor32(hasd ? uii : 0.0f);
  const float un = hasd ? uii : u_other;
  if (qi >= T) return;
  const float lam = *a.lambda;
  const float ln_i = logf((float)(qi + 1));
  const RowEpilogue e = row_epilogue(m, lt, un, a.scale, a.inv_tau, lam, ln_i);
#pragma unroll
  for (int db = 0; db < DB; ++db) {
#pragma unroll
    for (int rq = 0; rq < 4; ++rq) {
      const int d0 = 32 * db + 8 * rq + 4 * g;
      const bf16x4 vi = *(const bf16x4*)(v + qi * st + d0);
      bf16x4 out;
#pragma unroll
      for (int t = 0; t < 4; ++t)
        out[t] = f2bf(__builtin_fmaf(e.omg, bf2f(vi[t]), e.inv_l * oacc[db][4 * rq + t]));
      *(bf16x4*)(o + qi * st + d0) = out;
    }
  }
  if (g == 0) store_row_stats(a, (int64_t)head * T + qi, e, lam, ln_i);
}

// ---------------------------------------------------------------------------
// fp32 kernel (parity path): same scan, 32x32x2 f32 MFMAs, padded LDS rows.
// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(kNT, 1) void fwd_f32_kernel(FwdArgs a) {
  constexpr int DB = D / 32;
  constexpr int KS = D / 2;
  constexpr int NCH = D / 4;          // 16-byte chunks per row
  constexpr int SB = kBK / 32;
  constexpr int LDR = D + 1;          // padded LDS row (floats)
  constexpr int NLD = kBK * NCH / kNT;
  static_assert(NLD >= 1, "tile too small for the workgroup");
  __shared__ float Ks[kBK * LDR];
  __shared__ float Vs[kBK * LDR];

  int head, qt;
  if (!map_tile(a.map, blockIdx.x, head, qt, true)) return;
  const int T = a.T;
  const int64_t st = a.st;
  const int64_t hoff = (int64_t)(head / a.H) * a.sb + (int64_t)(head % a.H) * a.sh;
  const float* q = (const float*)a.q + hoff;
  const float* k = (const float*)a.k + hoff;
  const float* v = (const float*)a.v + hoff;
  float* o = (float*)a.o + hoff;

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int n = lane & 31, g = lane >> 5;
  const int i0 = qt * kBQ, qr0 = i0 + 32 * w, qi = qr0 + n;
  const bool wave_live = qr0 < T;
  const float c = a.scale * kLog2e;

  float qop[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) qop[ks] = (qi < T) ? q[qi * st + 2 * ks + g] : 0.0f;

  floatx4 kreg[NLD], vreg[NLD];
  auto prefetch = [&](int j0) {
#pragma unroll
    for (int j = 0; j < NLD; ++j) {
      const int ci = tid + kNT * j, row = ci / NCH, ch = ci % NCH, key = j0 + row;
      if (key < T) {
        kreg[j] = *(const floatx4*)(k + key * st + 4 * ch);
        vreg[j] = *(const floatx4*)(v + key * st + 4 * ch);
      } else {
        kreg[j] = floatx4{};
        vreg[j] = floatx4{};
      }
    }
  };
  auto stage = [&]() {
#pragma unroll
    for (int j = 0; j < NLD; ++j) {
      const int ci = tid + kNT * j, row = ci / NCH, ch = ci % NCH;
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        Ks[row * LDR + 4 * ch + t] = kreg[j][t];
        Vs[row * LDR + 4 * ch + t] = vreg[j][t];
      }
    }
  };

  float m = 0.0f, l = 0.0f, uii = 0.0f;
  bool hasd = false;
  floatx16 oacc[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) oacc[db] = floatx16{};

  const int kmax = min(i0 + kBQ, T) - 1;
  const int nkt = kmax / kBK + 1;
  prefetch(0);
  for (int kt = 0; kt < nkt; ++kt) {
    __syncthreads();
    stage();
    __syncthreads();
    if (kt + 1 < nkt) prefetch((kt + 1) * kBK);
    if (!wave_live) continue;
    const int j0 = kt * kBK;

    floatx16 sacc[SB];
    bool act[SB];
#pragma unroll
    for (int sb = 0; sb < SB; ++sb) {
      act[sb] = (j0 + 32 * sb) <= qr0;
      sacc[sb] = floatx16{};
      if (act[sb]) {
        const int row = 32 * sb + n;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) sacc[sb] = mfma32f(Ks[row * LDR + 2 * ks + g], qop[ks], sacc[sb]);
      }
    }

    float mx = kNegInf;
#pragma unroll
    for (int sb = 0; sb < SB; ++sb)
      if (act[sb]) exchange_logits(sacc[sb], j0 + 32 * sb == qr0, n, g, c, m, mx, uii, hasd);
    mx = fmaxf(mx, xor32(mx));
    if (wave_any(mx > kRescale)) {
      const float d = fmaxf(mx, 0.0f);
      m += d;
      const float al = fast_exp2(-d);
      l *= al;
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int r = 0; r < 16; ++r) oacc[db][r] *= al;
#pragma unroll
      for (int sb = 0; sb < SB; ++sb)
#pragma unroll
        for (int r = 0; r < 16; ++r) sacc[sb][r] -= d;
    }

#pragma unroll
    for (int sb = 0; sb < SB; ++sb) {
      if (!act[sb]) continue;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float p = fast_exp2(sacc[sb][r]);
        l += p;
        const int key = 32 * sb + acc_row(r, g);  // row of the LDS tile
#pragma unroll
        for (int db = 0; db < DB; ++db) oacc[db] = mfma32f(Vs[key * LDR + 32 * db + n], p, oacc[db]);
      }
    }
  }
  if (!wave_live) return;

  const float lt = l + xor32(l);
  const float u_other = xor32(hasd ? uii : 0.0f);
  const float un = hasd ? uii : u_other;
  if (qi >= T) return;
  const float lam = *a.lambda;
  const float ln_i = logf((float)(qi + 1));
  const RowEpilogue e = row_epilogue(m, lt, un, a.scale, a.inv_tau, lam, ln_i);
#pragma unroll
  for (int db = 0; db < DB; ++db) {
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int d = 32 * db + acc_row(r, g);
      o[qi * st + d] = __builtin_fmaf(e.omg, v[qi * st + d], e.inv_l * oacc[db][r]);
    }
  }
  if (g == 0) store_row_stats(a, (int64_t)head * T + qi, e, lam, ln_i);
}

}  // namespace

hipError_t launch_fwd(const FwdArgs& a0, int dtype, int D, hipStream_t stream) {
  FwdArgs a = a0;
  const int N = a.map.N;
  a.map = make_tilemap(N, (a.T + kBQ - 1) / kBQ);
  const dim3 grid((unsigned)grid_size(a.map)), block(kNT);
  hipEvent_t ev0, ev1;
  const bool prof = profile_slot("fwd", &ev0, &ev1);
  if (prof) (void)hipEventRecord(ev0, stream);
  if (dtype == 1) {
    if (D == 32) hipLaunchKernelGGL(fwd_bf16_kernel<32>, grid, block, 0, stream, a);
    else if (D == 64) hipLaunchKernelGGL(fwd_bf16_kernel<64>, grid, block, 0, stream, a);
    else hipLaunchKernelGGL(fwd_bf16_kernel<128>, grid, block, 0, stream, a);
  } else {
    if (D == 32) hipLaunchKernelGGL(fwd_f32_kernel<32>, grid, block, 0, stream, a);
    else if (D == 64) hipLaunchKernelGGL(fwd_f32_kernel<64>, grid, block, 0, stream, a);
    else hipLaunchKernelGGL(fwd_f32_kernel<128>, grid, block, 0, stream, a);
  }
  hipError_t e = hipGetLastError();
  if (prof) (void)hipEventRecord(ev1, stream);
  return e;
}

}  // namespace rel
