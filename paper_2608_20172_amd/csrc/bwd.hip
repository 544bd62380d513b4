// Fused backward pass of the causal Full Relation operator.
//
// Gradient identities used (App. A.1.7, with G = dO and the flow F):
//   H_ij = G_i . v_j,  D_i = sum_k F_ik H_ik = G_i . y_i,  dR_ij = F_ij (H_ij - D_i)
//   Exchange (j < i): F_ij = exp(E_ij - M_i), dU_ij = dR_ij * SiLU'(U_ij),
//                     SiLU'(U) = sigmoid(U) + E (1 - sigmoid(U))
//   Self (j = i):     F_ii = exp(S_i - M_i + lambda ln i),
//                     dU_ii = dR_ii * S_i (1 - S_i) / tau_S
//   dq = scale * dU k,  dk = scale * dU^T q,  dv = F^T G
//   dlambda = -sum_i ln i sum_{j<i} dR_ij = sum_i ln i * dR_ii
// (softmax-gradient rows sum to zero, so dlambda needs only the diagonal).
// M_i = ln Z_i + lambda ln i is the one statistic saved by the forward pass.
//
// Two kernels, both recomputing the evidence tiles from q, k, v, dO:
//  * dK/dV, key-major: a workgroup owns 128 keys (32 per wave) and walks the
//    64-row query tiles at or below its diagonal. U = Q K^T and dP = dO V^T are
//    formed with keys on lanes, so dV += F^T dO and dK += dU^T Q contract over
//    queries straight from registers; Q^T and dO^T come from the row-major LDS
//    tiles by transpose reads.
//  * dQ, query-major, shaped like the forward pass: lanes hold query rows and
//    dQ^T += K^T dU^T contracts over keys straight from registers. It runs
//    first and also stores D_i for the dK/dV kernel.
// Every gradient is written exactly once: no atomics, run-to-run identical.
// The dP chains start from an accumulator holding -D_i, so the matrix cores
// deliver dP_ij - D_i directly.
#include "kernels.h"

#include <algorithm>

namespace rel {

namespace {

constexpr int kBKW = 128;  // keys per dK/dV workgroup
constexpr int kBQI = 64;   // query rows per dK/dV iteration
constexpr int kBQ = 128;   // query rows per dQ workgroup
constexpr int kBK = 64;    // keys per dQ tile
constexpr int kNT = 256;
#ifndef REL_DQ_WAVES_PER_SIMD
#define REL_DQ_WAVES_PER_SIMD 2   // occupancy the register allocation is held to
#endif
#ifndef REL_DKDV_WAVES_PER_SIMD
#define REL_DKDV_WAVES_PER_SIMD 2
#endif

__global__ void fill_zero_kernel(float* p, int64_t n) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) p[i] = 0.0f;
}

struct Grad {
  float F, dU;
};

// One Exchange entry (j < i). u = q_i . k_j (raw), dpd = dO_i . v_j - D_i,
// Mi2 = M_i log2(e).
__device__ __forceinline__ Grad exchange_grad(float u, float dpd, float Mi2, float c) {
  const float up = u * c;                              // U log2(e)
  const float sg = fast_rcp(1.0f + fast_exp2(-up));    // sigmoid(U)
  const float wl = up * sg;                            // E log2(e)
  const float F = fast_exp2(wl - Mi2);                 // F_ij = exp(E_ij - M_i)
  const float t1 = __builtin_fmaf(-wl, sg, wl);        // E log2(e) (1 - sigmoid)
  const float dsilu = __builtin_fmaf(t1, kLn2, sg);    // sigmoid + E (1 - sigmoid)
  Grad r;
  r.F = F;
  r.dU = F * dpd * dsilu;
  return r;
}

struct SelfGrad {
  float F, dU, dR;
};

// The Self entry (j = i): U_ii = scale u, S_i = sigmoid(U_ii / tau_S). Row 1
// has no history, so F_11 = 1 and dR_11 = 0 exactly (App. A.1.8).
__device__ __forceinline__ SelfGrad self_grad(float u, float dpd, float Mi2, float scale,
                                              float inv_tau, float lam, float ln_i, bool first_row) {
  const float S = fast_rcp(1.0f + fast_exp2(-u * scale * inv_tau * kLog2e));
  SelfGrad r;
  r.F = first_row ? 1.0f : fast_exp2((S + lam * ln_i) * kLog2e - Mi2);
  r.dR = first_row ? 0.0f : r.F * dpd;
  r.dU = r.dR * S * (1.0f - S) * inv_tau;
  return r;
}

// ---------------------------------------------------------------------------
// dK / dV
// ---------------------------------------------------------------------------
template <class P, int D>
__global__ __launch_bounds__(kNT, (D <= 64 ? REL_DKDV_WAVES_PER_SIMD : 1)) void bwd_dkdv_kernel(BwdArgs a) {
  using E = typename P::T;
  using Op = typename P::Op;
  using Chunk = typename P::Chunk;
  constexpr int KS = D / 16;
  constexpr int DB = D / 32;
  constexpr int NCH = P::NCH;
  constexpr int NLQ = kBQI * NCH / kNT;   // chunks per thread for a query tile
  static_assert(NLQ >= 1, "query tile too small");
  constexpr int TB = P::tile_bytes(kBQI);
  __shared__ __attribute__((aligned(16))) unsigned char Qs[TB];
  __shared__ __attribute__((aligned(16))) unsigned char dOs[TB];
  __shared__ __attribute__((aligned(16))) float Mrow[kBQI];
  __shared__ __attribute__((aligned(16))) float Drow[kBQI];

  const int tid = threadIdx.x, w = tid >> 6;
  const Lane L(tid & 63);
  const int n = L.n, g = L.g;
  int head, kt;
  if (!map_tile(a.map, blockIdx.x, head, kt, false)) return;
  const int T = a.T;
  const int64_t st = a.st;
  const int64_t hoff = (int64_t)(head / a.H) * a.sb + (int64_t)(head % a.H) * a.sh;
  const E* q = (const E*)a.q + hoff;
  const E* k = (const E*)a.k + hoff;
  const E* v = (const E*)a.v + hoff;
  const E* dO = (const E*)a.dout + hoff;
  const float* Mst = a.row_stat + (int64_t)head * T;
  const float* Dst = a.dvec + (int64_t)head * T;
  const float c = a.scale * kLog2e;
  const float lam = *a.lambda;

  const int j0 = kt * kBKW;
  const int kw0 = j0 + 32 * w;        // first key of this wave
  const int kj = kw0 + n;             // this lane's key
  const bool wave_keys = kw0 < T;

  // B operands of U = Q K^T and dP = dO V^T: this lane's key row
  Op kop[KS], vop[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    kop[ks] = kj < T ? P::row_op_g(k + kj * st, ks, L) : Op{};
    vop[ks] = kj < T ? P::row_op_g(v + kj * st, ks, L) : Op{};
  }

  floatx16 dKt[DB], dVt[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) {
    dKt[db] = floatx16{};
    dVt[db] = floatx16{};
  }

  Chunk qreg[NLQ], dreg[NLQ];
  auto prefetch = [&](int i0) {
#pragma unroll
    for (int jj = 0; jj < NLQ; ++jj) {
      const int ci = tid + kNT * jj, row = ci / NCH, ch = ci % NCH, qi = i0 + row;
      if (qi < T) {
        qreg[jj] = *(const Chunk*)(q + qi * st + P::CE * ch);
        dreg[jj] = *(const Chunk*)(dO + qi * st + P::CE * ch);
      } else {
        qreg[jj] = Chunk{};
        dreg[jj] = Chunk{};
      }
    }
  };

  const int nqt = (T + kBQI - 1) / kBQI;
  const int qt0 = j0 / kBQI;
  prefetch(qt0 * kBQI);
  for (int qt = qt0; qt < nqt; ++qt) {
    const int i0 = qt * kBQI;
    __syncthreads();  // the previous tile is no longer read
#pragma unroll
    for (int jj = 0; jj < NLQ; ++jj) {
      const int ci = tid + kNT * jj, row = ci / NCH, ch = ci % NCH;
      P::stage(Qs, row, ch, qreg[jj]);
      P::stage(dOs, row, ch, dreg[jj]);
    }
    if (tid < kBQI) {
      const int qi = i0 + tid;
      Mrow[tid] = qi < T ? Mst[qi] * kLog2e : 0.0f;
      Drow[tid] = qi < T ? -Dst[qi] : 0.0f;  // the dP chains start from -D_i
    }
    __syncthreads();
    if (qt + 1 < nqt) prefetch(i0 + kBQI);

#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
      const int qb0 = i0 + 32 * qb;
      if (!wave_keys || qb0 < kw0 || qb0 >= T) continue;  // no row of the block reaches a key
      const int row = 32 * qb + n;
      floatx16 negD, Mb;  // per register: -D and M log2(e) of its query row
#pragma unroll
      for (int rq = 0; rq < 4; ++rq) {
        const int r0 = 32 * qb + 8 * rq + 4 * g;  // tile row of register 4 rq
        const floatx4 D4 = *(const floatx4*)(Drow + r0);
        const floatx4 M4 = *(const floatx4*)(Mrow + r0);
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          negD[4 * rq + t] = D4[t];
          Mb[4 * rq + t] = M4[t];
        }
      }
      floatx16 s = P::mma(P::row_op(Qs, row, 0, L), kop[0], floatx16{});
      floatx16 dp = P::mma(P::row_op(dOs, row, 0, L), vop[0], negD);  // dP - D
#pragma unroll
      for (int ks = 1; ks < KS; ++ks) {
        s = P::mma(P::row_op(Qs, row, ks, L), kop[ks], s);
        dp = P::mma(P::row_op(dOs, row, ks, L), vop[ks], dp);
      }
      float F[16], dU[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const Grad gr = exchange_grad(s[r], dp[r], Mb[r], c);
        F[r] = gr.F;
        dU[r] = gr.dU;
      }
      if (qb0 == kw0) {  // diagonal block: row offset acc_row(r, g) against key offset n
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          if (acc_row(r, g) < n) {
            F[r] = 0.0f;
            dU[r] = 0.0f;
          }
        }
        if (holds_row(n, g)) {
          const int rs = row_reg(n);
          const SelfGrad sg = self_grad(pick(s, rs), pick(dp, rs), Mrow[row], a.scale, a.inv_tau,
                                        lam, logf((float)(kj + 1)), kj == 0);
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            F[r] = r == rs ? sg.F : F[r];
            dU[r] = r == rs ? sg.dU : dU[r];
          }
        }
      }
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        const Op fop = P::pack(F + 8 * hh);
        const Op uop = P::pack(dU + 8 * hh);
        const int ks = 2 * qb + hh;
#pragma unroll
        for (int db = 0; db < DB; ++db) {
          dVt[db] = P::mma(P::col_op(dOs, ks, 32 * db, L), fop, dVt[db]);
          dKt[db] = P::mma(P::col_op(Qs, ks, 32 * db, L), uop, dKt[db]);
        }
      }
    }
  }

  if (kj < T) {
    E* dk = (E*)a.dk + hoff;
    E* dv = (E*)a.dv + hoff;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int rq = 0; rq < 4; ++rq) {
        const int d0 = 32 * db + 8 * rq + 4 * g;
        floatx4 kk, vv;
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          kk[t] = a.scale * dKt[db][4 * rq + t];
          vv[t] = dVt[db][4 * rq + t];
        }
        P::store4(dk + kj * st + d0, kk);
        P::store4(dv + kj * st + d0, vv);
      }
  }
}

// ---------------------------------------------------------------------------
// dQ (plus dself and the per-workgroup dlambda partials)
// ---------------------------------------------------------------------------
template <class P, int D>
__global__ __launch_bounds__(kNT, REL_DQ_WAVES_PER_SIMD) void bwd_dq_kernel(BwdArgs a) {
  using E = typename P::T;
  using Op = typename P::Op;
  using Chunk = typename P::Chunk;
  constexpr int KS = D / 16;
  constexpr int DB = D / 32;
  constexpr int SB = kBK / 32;
  constexpr int NLD = kBK * P::NCH / kNT;
  static_assert(NLD >= 1, "tile too small for the workgroup");
  constexpr int TB = P::tile_bytes(kBK);
  __shared__ __attribute__((aligned(16))) unsigned char lds[2 * TB];
  __shared__ float red[kNT / 64];
  unsigned char* Ks = lds;
  unsigned char* Vs = lds + TB;

  const int tid = threadIdx.x, w = tid >> 6;
  const Lane L(tid & 63);
  const int n = L.n, g = L.g;
  int head, qt;
  if (!map_tile(a.map, blockIdx.x, head, qt, true)) {
    if (tid == 0) a.dlam_part[blockIdx.x] = 0.0f;
    return;
  }
  const int T = a.T;
  const int64_t st = a.st;
  const int64_t hoff = (int64_t)(head / a.H) * a.sb + (int64_t)(head % a.H) * a.sh;
  const E* q = (const E*)a.q + hoff;
  const E* k = (const E*)a.k + hoff;
  const E* v = (const E*)a.v + hoff;
  const E* o = (const E*)a.o + hoff;
  const E* dO = (const E*)a.dout + hoff;
  const float c = a.scale * kLog2e;
  const float lam = *a.lambda;

  const int i0 = qt * kBQ, qr0 = i0 + 32 * w, qi = qr0 + n;
  const bool wave_live = qr0 < T;
  const bool row_ok = qi < T;

  // B operands: this lane's query row of Q and dO; D_i = dO_i . O_i from the
  // same slices, completed across the two lane halves
  Op qop[KS], doop[KS];
  float part = 0.0f;
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    qop[ks] = row_ok ? P::row_op_g(q + qi * st, ks, L) : Op{};
    doop[ks] = row_ok ? P::row_op_g(dO + qi * st, ks, L) : Op{};
    const Op oo = row_ok ? P::row_op_g(o + qi * st, ks, L) : Op{};
    part += P::op_dot(doop[ks], oo);
  }
  const float Di = part + xor32(part);
  const float Mi2 = row_ok ? a.row_stat[(int64_t)head * T + qi] * kLog2e : 0.0f;
  if (row_ok && g == 0) a.dvec[(int64_t)head * T + qi] = Di;
  floatx16 negD;  // the dP chains start from -D_i
#pragma unroll
  for (int r = 0; r < 16; ++r) negD[r] = -Di;

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

  floatx16 dQt[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) dQt[db] = floatx16{};
  float dlam = 0.0f;

  const int kmax = min(i0 + kBQ, T) - 1;
  const int nkt = kmax / kBK + 1;
  prefetch(0);
  for (int kt = 0; kt < nkt; ++kt) {
    __syncthreads();
#pragma unroll
    for (int j = 0; j < NLD; ++j) {
      const int ci = tid + kNT * j, row = ci / P::NCH, ch = ci % P::NCH;
      P::stage(Ks, row, ch, kreg[j]);
      P::stage(Vs, row, ch, vreg[j]);
    }
    __syncthreads();
    if (kt + 1 < nkt) prefetch((kt + 1) * kBK);
    if (!wave_live) continue;
    const int j0 = kt * kBK;
#pragma unroll
    for (int sb = 0; sb < SB; ++sb) {
      const int kb0 = j0 + 32 * sb;
      if (kb0 > qr0) continue;
      const int row = 32 * sb + n;
      floatx16 s = P::mma(P::row_op(Ks, row, 0, L), qop[0], floatx16{});
      floatx16 dp = P::mma(P::row_op(Vs, row, 0, L), doop[0], negD);  // dP - D
#pragma unroll
      for (int ks = 1; ks < KS; ++ks) {
        s = P::mma(P::row_op(Ks, row, ks, L), qop[ks], s);
        dp = P::mma(P::row_op(Vs, row, ks, L), doop[ks], dp);
      }
      float dU[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) dU[r] = exchange_grad(s[r], dp[r], Mi2, c).dU;
      if (kb0 == qr0) {  // diagonal block: key offset acc_row(r, g) against row offset n
#pragma unroll
        for (int r = 0; r < 16; ++r)
          if (acc_row(r, g) >= n) dU[r] = 0.0f;
        if (holds_row(n, g) && row_ok) {
          const int rs = row_reg(n);
          const float ln_i = logf((float)(qi + 1));
          const SelfGrad sg = self_grad(pick(s, rs), pick(dp, rs), Mi2, a.scale, a.inv_tau, lam, ln_i, qi == 0);
#pragma unroll
          for (int r = 0; r < 16; ++r) dU[r] = r == rs ? sg.dU : dU[r];
          dlam = __builtin_fmaf(ln_i, sg.dR, dlam);
          if (a.dself) a.dself[(int64_t)head * T + qi] = sg.dR;
        }
      }
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        const Op uop = P::pack(dU + 8 * hh);
#pragma unroll
        for (int db = 0; db < DB; ++db)
          dQt[db] = P::mma(P::col_op(Ks, 2 * sb + hh, 32 * db, L), uop, dQt[db]);
      }
    }
  }

  if (wave_live && row_ok) {
    E* dq = (E*)a.dq + hoff;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int rq = 0; rq < 4; ++rq) {
        const int d0 = 32 * db + 8 * rq + 4 * g;
        floatx4 out;
#pragma unroll
        for (int t = 0; t < 4; ++t) out[t] = a.scale * dQt[db][4 * rq + t];
        P::store4(dq + qi * st + d0, out);
      }
  }
  // this workgroup's dlambda partial, summed in a fixed order
#pragma unroll
  for (int s = 32; s >= 1; s >>= 1) dlam += __shfl_xor(dlam, s, 64);
  if ((tid & 63) == 0) red[w] = dlam;
  __syncthreads();
  if (tid == 0) a.dlam_part[blockIdx.x] = (red[0] + red[1]) + (red[2] + red[3]);
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

template <class P, int D>
void launch_pair(const BwdArgs& a, const TileMap& mkv, const TileMap& mq, hipStream_t stream,
                 hipEvent_t* prof) {
  // dQ first: it also writes D_i, which the dK/dV kernel reads
  BwdArgs b = a;
  hipEvent_t e0, e1;
  const bool p_all = prof != nullptr;
  if (p_all) (void)hipEventRecord(prof[0], stream);
  b.map = mq;
  const bool p_q = !p_all && profile_slot("bwd_dq", &e0, &e1);
  if (p_q) (void)hipEventRecord(e0, stream);
  hipLaunchKernelGGL((bwd_dq_kernel<P, D>), dim3((unsigned)grid_size(mq)), dim3(kNT), 0, stream, b);
  if (p_q) (void)hipEventRecord(e1, stream);
  b.map = mkv;
  const bool p_kv = !p_all && profile_slot("bwd_dkdv", &e0, &e1);
  if (p_kv) (void)hipEventRecord(e0, stream);
  hipLaunchKernelGGL((bwd_dkdv_kernel<P, D>), dim3((unsigned)grid_size(mkv)), dim3(kNT), 0, stream, b);
  if (p_kv) (void)hipEventRecord(e1, stream);
  if (p_all) (void)hipEventRecord(prof[1], stream);
}

}  // namespace

int bwd_partials(int N, int T, int D, int dtype) {
  (void)D;
  (void)dtype;
  return (int)grid_size(make_tilemap(N, (T + kBQ - 1) / kBQ));
}

hipError_t launch_bwd(const BwdArgs& a, int dtype, int D, hipStream_t stream) {
  const int N = a.map.N;
  const TileMap mkv = make_tilemap(N, (a.T + kBKW - 1) / kBKW);
  const TileMap mq = make_tilemap(N, (a.T + kBQ - 1) / kBQ);
  hipEvent_t ev[2];
  const bool prof = profile_slot("bwd", &ev[0], &ev[1]);
  hipEvent_t* pe = prof ? ev : nullptr;
  if (dtype == 1) {
    if (D == 32) launch_pair<PolBF16<32>, 32>(a, mkv, mq, stream, pe);
    else if (D == 64) launch_pair<PolBF16<64>, 64>(a, mkv, mq, stream, pe);
    else launch_pair<PolBF16<128>, 128>(a, mkv, mq, stream, pe);
  } else {
    if (D == 32) launch_pair<PolF32<32>, 32>(a, mkv, mq, stream, pe);
    else if (D == 64) launch_pair<PolF32<64>, 64>(a, mkv, mq, stream, pe);
    else launch_pair<PolF32<128>, 128>(a, mkv, mq, stream, pe);
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
