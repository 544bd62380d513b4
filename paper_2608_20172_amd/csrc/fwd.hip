// Fused forward pass of the causal Full Relation operator (FlashRelation).
//
// One workgroup = 4 waves = 128 query rows of one head; each wave owns 32 rows.
// Key/value tiles of 64 rows stream HBM -> registers -> LDS. Per tile a wave
// computes the transposed evidence block U^T = K Q^T with 32x32 MFMAs, so each
// lane holds one query row and 16 keys per block: the row reductions of the
// online scan stay inside the lane, plus one exchange with the partner lane
// 32 away. The Exchange scan keeps (m, l, z) per row exactly as in eqs. (11)-(12)
// of Sec. 5.1 / App. A.3, with Self excluded; Self and the count correction
// join only in the epilogue (eq. 13). The Self logit U_ii is read off the
// diagonal entry of the evidence tile that holds row i.
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
#ifndef REL_FWD_WAVES_PER_SIMD
#define REL_FWD_WAVES_PER_SIMD 2  // occupancy the register allocation is held to
#endif

// Exchange logits of one 32x32 block, in place: s[r] (raw q.k) becomes
// E log2(e) - m; in the diagonal block (DIAG) entries with key >= query get -inf.
template <bool DIAG>
__device__ __forceinline__ void exchange_logits(floatx16& s, const Lane& L, float c, float m, float& mx) {
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const float up = s[r] * c;                             // U log2(e)
    const float sg = fast_rcp(1.0f + fast_exp2(-up));      // sigmoid(U)
    float e = __builtin_fmaf(up, sg, -m);                  // SiLU(U) log2(e) - m
    if (DIAG && acc_row(r, L.g) >= L.n) e = kNegInf;       // strictly historical: j < i
    s[r] = e;
    mx = fmaxf(mx, e);
  }
}

struct RowEpilogue {
  float g, omg, inv_l, LE, lnZ, S;
};

// Completes row i from the terminal scan state (eqs. 12-13):
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

template <class P, int D>
__global__ __launch_bounds__(kNT, REL_FWD_WAVES_PER_SIMD) void fwd_kernel(FwdArgs a) {
  using E = typename P::T;
  using Op = typename P::Op;
  using Chunk = typename P::Chunk;
  constexpr int KS = D / 16;                      // 16-wide slices of d
  constexpr int DB = D / 32;                      // 32-row blocks of O^T
  constexpr int SB = kBK / 32;                    // 32-key blocks per tile
  constexpr int NLD = kBK * P::NCH / kNT;         // chunks per thread per tensor
  static_assert(NLD >= 1, "tile too small for the workgroup");
  constexpr int TB = P::tile_bytes(kBK);
  __shared__ __attribute__((aligned(16))) unsigned char lds[2 * TB];
  unsigned char* Ks = lds;
  unsigned char* Vs = lds + TB;

  int head, qt;
  if (!map_tile(a.map, blockIdx.x, head, qt, true)) return;
  const int T = a.T;
  const int64_t st = a.st;
  const int64_t hoff = (int64_t)(head / a.H) * a.sb + (int64_t)(head % a.H) * a.sh;
  const E* q = (const E*)a.q + hoff;
  const E* k = (const E*)a.k + hoff;
  const E* v = (const E*)a.v + hoff;
  E* o = (E*)a.o + hoff;

  const int tid = threadIdx.x, w = tid >> 6;
  const Lane L(tid & 63);
  const int n = L.n, g = L.g;
  const int i0 = qt * kBQ, qr0 = i0 + 32 * w, qi = qr0 + n;
  const bool wave_live = qr0 < T;
  const float c = a.scale * kLog2e;

  // B operand of U^T = K Q^T: this lane's query row
  Op qop[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) qop[ks] = qi < T ? P::row_op_g(q + qi * st, ks, L) : Op{};

  Chunk kreg[NLD], vreg[NLD];
  auto prefetch = [&](int j0) {
#pragma unroll
    for (int j = 0; j < NLD; ++j) {
      const int ci = tid + kNT * j, row = ci / P::NCH, ch = ci % P::NCH, key = j0 + row;
      if (key < T) {
        kreg[j] = *(const Chunk*)(k + key * st + P::CE * ch);
        vreg[j] = *(const Chunk*)(v + key * st + P::CE * ch);
      } else {
        kreg[j] = Chunk{};
        vreg[j] = Chunk{};
      }
    }
  };
  auto stage = [&]() {
#pragma unroll
    for (int j = 0; j < NLD; ++j) {
      const int ci = tid + kNT * j, row = ci / P::NCH, ch = ci % P::NCH;
      P::stage(Ks, row, ch, kreg[j]);
      P::stage(Vs, row, ch, vreg[j]);
    }
  };

  // l sums the fp32 p (not the bf16-rounded MFMA operand), so that L^E and the
  // saved statistic M carry no operand rounding
  float m = 0.0f, l = 0.0f, uii = 0.0f;
  floatx16 oacc[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) oacc[db] = floatx16{};

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
    float mx = kNegInf;
#pragma unroll
    for (int sb = 0; sb < SB; ++sb) {
      const int kb0 = j0 + 32 * sb;
      if (kb0 > qr0) continue;  // no key of the block precedes or meets a row of the wave
      const int row = 32 * sb + n;
      sacc[sb] = P::mma(P::row_op(Ks, row, 0, L), qop[0], floatx16{});
#pragma unroll
      for (int ks = 1; ks < KS; ++ks) sacc[sb] = P::mma(P::row_op(Ks, row, ks, L), qop[ks], sacc[sb]);
      if (kb0 == qr0) {
        if (holds_row(n, g)) uii = pick(sacc[sb], row_reg(n));  // the Self evidence U_ii
        exchange_logits<true>(sacc[sb], L, c, m, mx);
      } else {
        exchange_logits<false>(sacc[sb], L, c, m, mx);
      }
    }
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
      if (j0 + 32 * sb > qr0) continue;
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        float p[8];
#pragma unroll
        for (int t = 0; t < 8; ++t) {
          p[t] = fast_exp2(sacc[sb][8 * hh + t]);
          l += p[t];
        }
        const Op pop = P::pack(p);
#pragma unroll
        for (int db = 0; db < DB; ++db)
          oacc[db] = P::mma(P::col_op(Vs, 2 * sb + hh, 32 * db, L), pop, oacc[db]);
      }
    }
  }
  if (!wave_live) return;

  // ---- epilogue: combine the two lane halves of each row, then eq. (13)
  const float lt = l + xor32(l);
  const float u_other = xor32(uii);
  const float un = holds_row(n, g) ? uii : u_other;
  if (qi >= T) return;
  const float lam = *a.lambda;
  const float ln_i = logf((float)(qi + 1));
  const RowEpilogue e = row_epilogue(m, lt, un, a.scale, a.inv_tau, lam, ln_i);
#pragma unroll
  for (int db = 0; db < DB; ++db) {
#pragma unroll
    for (int rq = 0; rq < 4; ++rq) {
      const int d0 = 32 * db + 8 * rq + 4 * g;
      const floatx4 vi = P::load4(v + qi * st + d0);
      floatx4 out;
#pragma unroll
      for (int t = 0; t < 4; ++t) out[t] = __builtin_fmaf(e.omg, vi[t], e.inv_l * oacc[db][4 * rq + t]);
      P::store4(o + qi * st + d0, out);
    }
  }
  if (g == 0) {
    const int64_t ridx = (int64_t)head * T + qi;
    if (a.row_stat) a.row_stat[ridx] = e.lnZ + lam * ln_i;
    if (a.self_mass) a.self_mass[ridx] = e.omg;
    if (a.exch_mass) a.exch_mass[ridx] = e.g;
    if (a.exch_lse) a.exch_lse[ridx] = e.LE;
  }
}

template <class P, int D>
void launch_one(const FwdArgs& a, hipStream_t stream) {
  hipLaunchKernelGGL((fwd_kernel<P, D>), dim3((unsigned)grid_size(a.map)), dim3(kNT), 0, stream, a);
}

}  // namespace

hipError_t launch_fwd(const FwdArgs& a0, int dtype, int D, hipStream_t stream) {
  FwdArgs a = a0;
  a.map = make_tilemap(a.map.N, (a.T + kBQ - 1) / kBQ);
  hipEvent_t ev0, ev1;
  const bool prof = profile_slot("fwd", &ev0, &ev1);
  if (prof) (void)hipEventRecord(ev0, stream);
  if (dtype == 1) {
    if (D == 32) launch_one<PolBF16<32>, 32>(a, stream);
    else if (D == 64) launch_one<PolBF16<64>, 64>(a, stream);
    else launch_one<PolBF16<128>, 128>(a, stream);
  } else {
    if (D == 32) launch_one<PolF32<32>, 32>(a, stream);
    else if (D == 64) launch_one<PolF32<64>, 64>(a, stream);
    else launch_one<PolF32<128>, 128>(a, stream);
  }
  hipError_t e = hipGetLastError();
  if (prof) (void)hipEventRecord(ev1, stream);
  return e;
}

}  // namespace rel
