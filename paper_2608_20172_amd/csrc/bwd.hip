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
//  * dQ, query-major, shaped like the forward pass: lanes hold query rows and
//    dQ^T += K^T dU^T contracts over keys straight from registers. It runs
//    first and stores -D_i and M_i log2(e) per row for the dK/dV kernel.
//  * dK/dV, key-major: a workgroup owns 128 keys (32 per wave) and walks the
//    64-row query tiles at or below its diagonal. U = Q K^T and dP = dO V^T are
//    formed with keys on lanes, so dV += F^T dO and dK += dU^T Q contract over
//    queries straight from registers; Q^T and dO^T come from the row-major LDS
//    tiles by transpose reads.
// Tiles go HBM -> LDS by buffer loads that write LDS directly (two buffers,
// one barrier per tile; rows past T read as zeros). Every gradient is written
// exactly once: no atomics, run-to-run identical. The matrix cores deliver
// dP_ij - D_i directly: in dK/dV the dP chains start from an accumulator
// holding -D of each query row, in dQ one more product adds -D_i.
#include "kernels.h"
#include "lanes.h"

#include <algorithm>
#include <type_traits>

namespace rel {

namespace {

constexpr int kBKW = 128;  // keys per dK/dV workgroup
constexpr int kBQI = 64;   // query rows per dK/dV tile
constexpr int kBQ = 128;   // query rows per dQ workgroup
constexpr int kBK = 64;    // keys per dQ tile
constexpr int kNT = 256;
constexpr int kFusedWaves = 8;  // fused backward: 8 waves, 256 keys per workgroup
constexpr int kDqIlValu = 28;    // dQ full tiles: vector instructions after each matrix instruction
constexpr int kDkdvIlValu = 12;  // dK/dV full tiles: the same

// Scheduling pattern for one basic block holding NM matrix instructions and
// independent vector work: the LDS reads first, then each matrix instruction
// followed by NV vector instructions.
template <int NM, int NV, int ID>
__device__ __forceinline__ void interleave() {
  __builtin_amdgcn_sched_group_barrier(0x100, 64, ID);  // LDS reads
#pragma unroll
  for (int i = 0; i < NM; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, ID);   // matrix
    __builtin_amdgcn_sched_group_barrier(0x002, NV, ID);  // vector
  }
}

// Waves per SIMD the kernels are compiled for.
template <class P, int D>
constexpr int dq_occupancy() {
  return sizeof(typename P::T) == 2 ? (D <= 64 ? 3 : 2) : (D <= 32 ? 2 : 1);
}
template <class P, int D>
constexpr int dkdv_occupancy() {
  return sizeof(typename P::T) == 2 ? (D <= 64 ? 2 : 1) : 1;
}

__global__ void fill_zero_kernel(float* p, int64_t n) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) p[i] = 0.0f;
}

// Exchange entries (j < i) of one 32x32 block, in place: s holds raw q . k and
// becomes F_ij = exp(E_ij - M_i); dp holds dP_ij - D_i and becomes dU_ij.
// M2(r) = M log2(e) of the query row of register r. Passes over groups of 4
// independent entries keep instructions off transcendental results.
template <class MF>
__device__ __forceinline__ void exchange_grads(floatx16& s, floatx16& dp, MF M2, float c, float dsub = 0.0f) {
#pragma unroll
  for (int r0 = 0; r0 < 16; r0 += 4) {
    float up[4], sg[4], wl[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) up[r] = s[r0 + r] * c;                  // U log2(e)
#pragma unroll
    for (int r = 0; r < 4; ++r) sg[r] = fast_exp2(-up[r]);
#pragma unroll
    for (int r = 0; r < 4; ++r) sg[r] = fast_rcp(1.0f + sg[r]);         // sigmoid(U)
#pragma unroll
    for (int r = 0; r < 4; ++r) wl[r] = up[r] * sg[r];                  // E log2(e)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const float F = fast_exp2(wl[r] - M2(r0 + r));                    // F_ij = exp(E_ij - M_i)
      const float t1 = __builtin_fmaf(-wl[r], sg[r], wl[r]);            // E log2(e) (1 - sigmoid)
      const float dsilu = __builtin_fmaf(t1, kLn2, sg[r]);              // sigmoid + E (1 - sigmoid)
      s[r0 + r] = F;
      dp[r0 + r] = F * (dp[r0 + r] - dsub) * dsilu;
    }
  }
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
// dQ (plus dself, -D, M log2(e) and the per-workgroup dlambda partials)
// ---------------------------------------------------------------------------
template <class P, int D>
__global__ __launch_bounds__(kNT, (dq_occupancy<P, D>())) void bwd_dq_kernel(BwdArgs a) {
  using E = typename P::T;
  using Op = typename P::Op;
  constexpr int KS = D / 16;
  constexpr int DB = D / 32;
  constexpr int TB = kBK * P::ROWB;
  constexpr int NSEG = TB / 1024;
  constexpr int SEGW = 2 * NSEG / 4;
  static_assert(SEGW >= 1 && 2 * NSEG % 4 == 0, "tile does not split over the waves");
  // two tile buffers as distinct objects: the compiler can then see that
  // reads of one do not wait for the loads in flight into the other
  __shared__ __attribute__((aligned(1024))) unsigned char bufA[2 * TB];
  __shared__ __attribute__((aligned(1024))) unsigned char bufB[2 * TB];
  __shared__ float red[kNT / 64];

  const int tid = threadIdx.x, w = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
  const int lane = tid & 63;
  const Lane L(lane);
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

  const int row_bytes = (int)(st * (int64_t)sizeof(E));
  const __amdgpu_buffer_rsrc_t krs = make_rsrc(k, T * row_bytes);
  const __amdgpu_buffer_rsrc_t vrs = make_rsrc(v, T * row_bytes);
  auto load_tile = [&](int j0, unsigned char* buf) {
#pragma unroll
    for (int s = 0; s < SEGW; ++s) {
      const int seg = w * SEGW + s, tens = seg / NSEG;
      dma_segment<P>(tens ? vrs : krs, buf + tens * TB, seg % NSEG, row_bytes, j0, lane);
    }
  };
  load_tile(0, bufA);

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
  if (row_ok && g == 0) {
    a.negd[(int64_t)head * T + qi] = -Di;
    a.m2[(int64_t)head * T + qi] = Mi2;
  }
  // -D_i enters the dP chains as one more product of a 0/1 column against -D_i
  // split into two bf16 terms (bf16: every key row of this lane's query gets
  // -D_hi - D_lo), or by a subtraction per entry (fp32)
  constexpr int NDM = sizeof(E) == 2 ? 2 : 0;
  const float dsub = NDM == 0 ? Di : 0.0f;
  Op dcol{}, dval{};
  if constexpr (NDM == 2) {
    const bf16 hi = f2bf(-Di);
    const bf16 lo = f2bf(-Di - bf2f(hi));
    const unsigned w = (unsigned)__builtin_bit_cast(unsigned short, hi) |
                       ((unsigned)__builtin_bit_cast(unsigned short, lo) << 16);
    const bool g0 = g == 0;  // contraction indices 0 and 1 live in elements 0, 1 of lane group 0
    dcol = __builtin_bit_cast(Op, uintx4{g0 ? 0x3f803f80u : 0u, 0u, 0u, 0u});
    dval = __builtin_bit_cast(Op, uintx4{g0 ? w : 0u, 0u, 0u, 0u});
  }

  floatx16 dQt[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) dQt[db] = floatx16{};
  float dlam = 0.0f;

  // Key block (keys krow0 .. krow0+31 of the tile): the evidence and dP - D
  // chains on the matrix cores ...
  auto evid = [&](const unsigned char* Ks, const unsigned char* Vs, int krow0, floatx16& s, floatx16& dp) {
    const int row = krow0 + n;
    s = floatx16{};
    dp = floatx16{};
#pragma unroll
    for (int k0 = 0; k0 < KS; ++k0) {
      const Op ka = P::row_op(Ks, row, k0, L);
      const Op va = P::row_op(Vs, row, k0, L);
      s = P::mma(ka, qop[k0], s);
      dp = P::mma(va, doop[k0], dp);
    }
    if constexpr (NDM == 2) dp = P::mma(dcol, dval, dp);
  };
  // ... then dU on the vector units, packed as the operands of the two 16-key
  // halves; DIAG: the wave's own diagonal block (key offset acc_row(r, g)
  // against row offset n)
  auto grads = [&](floatx16& s, floatx16& dp, Op (&uop)[2], auto diag_c) {
    constexpr bool DIAG = decltype(diag_c)::value;
    float uself = 0.0f, dself = 0.0f;
    const int rs = row_reg(n);
    if (DIAG) {
      uself = pick(s, rs);
      dself = pick(dp, rs);
    }
    if (NDM == 0 && DIAG) dself -= Di;
    if (DIAG && a.exch_only) dself = -Di;  // exchange-only: dL/dF_ii = 0, so dR_ii = -F_ii D_i
    exchange_grads(s, dp, [&](int) { return Mi2; }, c, dsub);
    if (DIAG) {
#pragma unroll
      for (int r = 0; r < 16; ++r)
        if (acc_row(r, g) >= n) dp[r] = 0.0f;  // strictly historical: j < i
      if (holds_row(n, g) && row_ok) {
        const float ln_i = logf((float)(qi + 1));
        const SelfGrad sg = self_grad(uself, dself, Mi2, a.scale, a.inv_tau, lam, ln_i, qi == 0);
#pragma unroll
        for (int r = 0; r < 16; ++r) dp[r] = r == rs ? sg.dU : dp[r];
        dlam = __builtin_fmaf(ln_i, sg.dR, dlam);
        if (a.dself) a.dself[(int64_t)head * T + qi] = sg.dR;
      }
    }
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
      float u8[8];
#pragma unroll
      for (int t = 0; t < 8; ++t) u8[t] = dp[8 * hh + t];
      uop[hh] = P::pack(u8);
    }
  };
  // dQ^T += K^T dU^T for key block b of the tile
  auto accum = [&](const unsigned char* Ks, int b, const Op (&uop)[2]) {
#pragma unroll
    for (int hh = 0; hh < 2; ++hh)
#pragma unroll
      for (int db = 0; db < DB; ++db) dQt[db] = P::mma(P::col_op(Ks, 2 * b + hh, 32 * db, L), uop[hh], dQt[db]);
  };

  const int kmax = min(i0 + kBQ, T) - 1;
  const int nkt = kmax / kBK + 1;
  const int qlast = wave_live ? qr0 : -1;  // rows of a wave past T meet no key
  // One key tile. A block at or above the wave's rows contributes zero dU, so
  // the dQ products (and the accumulators) run on every path. Order: evidence
  // of block 0, its vector work, evidence of block 1, then the products of
  // block 0 (which run under the vector work of block 1).
  auto step = [&](int kt, const unsigned char* Ks, unsigned char* nxt) __attribute__((always_inline)) {
    wait_loads();
    __syncthreads();
    if (kt + 1 < nkt) load_tile((kt + 1) * kBK, nxt);
    const unsigned char* Vs = Ks + TB;
    const int k0 = kt * kBK;
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      const int kb = k0 + 32 * b;
      Op u[2] = {Op{}, Op{}};
      floatx16 s, dp;
      if (kb < qlast) {
        evid(Ks, Vs, 32 * b, s, dp);
        grads(s, dp, u, std::false_type{});
      } else if (kb == qlast) {
        evid(Ks, Vs, 32 * b, s, dp);
        grads(s, dp, u, std::true_type{});
      }
      accum(Ks, b, u);
    }
  };
  // A full tile (both blocks below every wave's rows) runs without branches.
  auto full = [&](int kt, const unsigned char* Ks, unsigned char* nxt) __attribute__((always_inline)) {
    wait_loads();
    __syncthreads();
    if (kt + 1 < nkt) load_tile((kt + 1) * kBK, nxt);
    const unsigned char* Vs = Ks + TB;
    // the products of block 0 between the vector work of block 1
    Op u0[2], u1[2];
    floatx16 s, dp;
    evid(Ks, Vs, 0, s, dp);
    grads(s, dp, u0, std::false_type{});
    __builtin_amdgcn_sched_barrier(0);
    evid(Ks, Vs, 32, s, dp);
    __builtin_amdgcn_sched_barrier(0);
    accum(Ks, 0, u0);
    grads(s, dp, u1, std::false_type{});
    interleave<2 * DB, kDqIlValu, 0>();
    __builtin_amdgcn_sched_barrier(0);
    accum(Ks, 1, u1);
  };
  // even tiles in bufA, odd ones in bufB
  auto run = [&](int ka, int kb, auto st) __attribute__((always_inline)) {
    int kt = ka;
    if (kt < kb && (kt & 1)) {
      st(kt, bufB, bufA);
      ++kt;
    }
    for (; kt < kb; kt += 2) {
      st(kt, bufA, bufB);
      if (kt + 1 < kb) st(kt + 1, bufB, bufA);
    }
  };
  const int kf = min(i0 / kBK, nkt);  // tiles below the workgroup's diagonal
  run(0, kf, full);
  run(kf, nkt, step);

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
  if (lane == 0) red[w] = dlam;
  __syncthreads();
  if (tid == 0) a.dlam_part[blockIdx.x] = (red[0] + red[1]) + (red[2] + red[3]);
}

// ---------------------------------------------------------------------------
// dK / dV
// ---------------------------------------------------------------------------
// NW waves of 32 keys each. FQ (bf16, fused backward): the workgroup also
// forms dQ. The dU tile of each query tile (keys x queries, bf16) goes to LDS;
// after the next barrier, waves 0 .. 2 D/32 - 1 each take one 32 x 32 block of
// the tile's dQ partial, dU[64 x NW*32] K[NW*32 x D] on the matrix cores (K of
// the workgroup's keys is held in LDS), and add it to the fp32 dQ accumulator
// with global atomics. The diagonal (Self) entry sits in dU, so dQ needs no
// separate Self term; dself and the dlambda partials come from the diagonal
// blocks here.
// CS = 2 (channel split, two-kernel path at D = 128): two waves share each 32
// keys. Each forms U, dP, F and dU of one of the tile's two 32-query blocks,
// the pair swap their packed F and dU through LDS, and each accumulates dK and
// dV for half of the channels over both blocks. So a wave holds half of the
// 128 accumulator registers of its keys, and two waves per SIMD fit where one
// did (at one wave per SIMD a wave issues vector work at half the SIMD's rate).
template <class P, int D, int NW, bool FQ, int CS = 1>
__global__ __launch_bounds__(NW * 64, (CS == 2 ? 2 : dkdv_occupancy<P, D>())) void bwd_dkdv_kernel(BwdArgs a) {
  using E = typename P::T;
  using Op = typename P::Op;
  using PU = PolBF16<64>;                       // layout of the dU tile: 64 query columns
  constexpr int NT = NW * 64;
  constexpr int KW = NW * 32 / CS;              // keys per workgroup
  constexpr int KS = D / 16;
  constexpr int DB = D / 32;
  constexpr int DBH = DB / CS;                  // 32-channel blocks of dK and dV per wave
  static_assert(CS == 1 || (CS == 2 && !FQ && DB % 2 == 0), "channel split: two-kernel path, even channel blocks");
  constexpr int TB = kBQI * P::ROWB;            // one tensor tile (Q or dO)
  constexpr int NSEG = TB / 1024;
  constexpr int SEGW = 2 * NSEG / NW;
  static_assert(SEGW >= 1 && 2 * NSEG % NW == 0, "tile does not split over the waves");
  static_assert(!FQ || (sizeof(E) == 2 && KW % 64 == 0 && 2 * DB <= NW), "fused dQ: bf16, whole 64-key tiles");
  constexpr int BUF = 2 * TB + 2 * kBQI * 4;    // Q, dO, M log2(e), -D
  constexpr int DUT = PU::tile_bytes(kBQI);     // dU of 64 keys x 64 queries
  constexpr int KQB = FQ ? (KW / 64) * TB : 16; // K of the workgroup's keys
  constexpr int DUB = FQ ? (KW / 64) * DUT : 16;
  // tile buffers as distinct objects: the compiler can then see that reads of
  // one do not wait for the loads in flight into another
  __shared__ __attribute__((aligned(1024))) unsigned char bufA[BUF];
  __shared__ __attribute__((aligned(1024))) unsigned char bufB[BUF];
  __shared__ __attribute__((aligned(1024))) unsigned char Kq[KQB];
  __shared__ __attribute__((aligned(1024))) unsigned char dUA[DUB];
  __shared__ __attribute__((aligned(1024))) unsigned char dUB[DUB];
  // CS: per key group and query block, the packed F and dU operands (two
  // 16-row halves each) of the wave that formed them, one 16-byte lane slot each
  constexpr int XCH = CS == 2 ? (KW / 32) * 2 * 4 * 64 * 16 : 16;
  __shared__ __attribute__((aligned(1024))) unsigned char Xch[XCH];
  __shared__ float red[NT];

  const int tid = threadIdx.x, w = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
  const int lane = tid & 63;
  const Lane L(lane);
  const int n = L.n, g = L.g;
  if (!FQ && blockIdx.x == 0 && a.dlambda) {
    // dlambda: the dQ kernel (which ran before this one) left one partial per
    // workgroup; summed here in a fixed order, so the result is run-to-run
    // identical
    float acc = 0.0f;
    for (int i = tid; i < a.nparts; i += NT) acc += a.dlam_part[i];
    red[tid] = acc;
    __syncthreads();
    for (int h = NT / 2; h >= 1; h >>= 1) {
      if (tid < h) red[tid] += red[tid + h];
      __syncthreads();
    }
    if (tid == 0) *a.dlambda = red[0];
    __syncthreads();
  }
  int head, kt;
  if (!map_tile(a.map, blockIdx.x, head, kt, false)) {
    if (FQ && tid == 0) a.dlam_part[blockIdx.x] = 0.0f;
    return;
  }
  const int T = a.T;
  const int64_t st = a.st;
  const int64_t hoff = (int64_t)(head / a.H) * a.sb + (int64_t)(head % a.H) * a.sh;
  const E* q = (const E*)a.q + hoff;
  const E* k = (const E*)a.k + hoff;
  const E* v = (const E*)a.v + hoff;
  const E* dO = (const E*)a.dout + hoff;
  const float c = a.scale * kLog2e;
  const float lam = *a.lambda;

  const int j0 = kt * KW;
  const int kgw = w / CS, chw = w % CS;  // key group; with CS, the query block and channel half of the wave
  const int kw0 = j0 + 32 * kgw;      // first key of this wave
  const int kj = kw0 + n;             // this lane's key
  const bool wave_keys = kw0 < T;

  // query tiles of Q and dO, and the per-row -D and M log2(e); rows past T
  // read as zeros, so they add nothing to dK and dV
  const int row_bytes = (int)(st * (int64_t)sizeof(E));
  const __amdgpu_buffer_rsrc_t qrs = make_rsrc(q, T * row_bytes);
  const __amdgpu_buffer_rsrc_t drs = make_rsrc(dO, T * row_bytes);
  const __amdgpu_buffer_rsrc_t mrs = make_rsrc(a.m2 + (int64_t)head * T, T * 4);
  const __amdgpu_buffer_rsrc_t nrs = make_rsrc(a.negd + (int64_t)head * T, T * 4);
  auto load_tile = [&](int i0, unsigned char* buf) {
#pragma unroll
    for (int s = 0; s < SEGW; ++s) {
      const int seg = w * SEGW + s, tens = seg / NSEG;
      dma_segment<P>(tens ? drs : qrs, buf + tens * TB, seg % NSEG, row_bytes, i0, lane);
    }
    if (w < 2) dma_row64(w ? nrs : mrs, (float*)(buf + 2 * TB) + w * kBQI, i0, lane);
  };

  const int nqt = (T + kBQI - 1) / kBQI;
  const int qt0 = j0 / kBQI;
  load_tile(qt0 * kBQI, bufA);
  if constexpr (FQ) {
    // K of the workgroup's keys, the second operand of dQ = dU K
    const __amdgpu_buffer_rsrc_t krs = make_rsrc(k, T * row_bytes);
#pragma unroll
    for (int s = 0; s < (KW / 64) * NSEG / NW; ++s) {
      const int seg = w * ((KW / 64) * NSEG / NW) + s;
      dma_segment<P>(krs, Kq + (seg / NSEG) * TB, seg % NSEG, row_bytes, j0 + 64 * (seg / NSEG), lane);
    }
  }
  if (FQ) red[tid] = 0.0f;  // fused: per-key dlambda terms, written in the diagonal blocks

  // B operands of U = Q K^T and dP = dO V^T: this lane's key row
  Op kop[KS], vop[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    kop[ks] = kj < T ? P::row_op_g(k + kj * st, ks, L) : Op{};
    vop[ks] = kj < T ? P::row_op_g(v + kj * st, ks, L) : Op{};
  }

  floatx16 dKt[DBH], dVt[DBH];
#pragma unroll
  for (int db = 0; db < DBH; ++db) {
    dKt[db] = floatx16{};
    dVt[db] = floatx16{};
  }

  // Query block qb (rows 32 qb .. 32 qb + 31 of the tile): the evidence and
  // dP - D chains on the matrix cores ...
  auto evid = [&](const unsigned char* buf, int qb, floatx16& s, floatx16& dp) {
    const unsigned char* Qs = buf;
    const unsigned char* dOs = buf + TB;
    const float* Nrow = (const float*)(buf + 2 * TB) + kBQI;
    const int row = 32 * qb + n;
#pragma unroll
    for (int rq = 0; rq < 4; ++rq) {  // -D of the query row of every register
      const floatx4 D4 = *(const floatx4*)(Nrow + 32 * qb + 8 * rq + 4 * g);
#pragma unroll
      for (int t = 0; t < 4; ++t) dp[4 * rq + t] = D4[t];
    }
    s = floatx16{};
#pragma unroll
    for (int k0 = 0; k0 < KS; k0 += 2) {
      Op qa[2], da[2];
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        qa[j] = P::row_op(Qs, row, k0 + j, L);
        da[j] = P::row_op(dOs, row, k0 + j, L);
      }
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        s = P::mma(qa[j], kop[k0 + j], s);
        dp = P::mma(da[j], vop[k0 + j], dp);  // dP - D
      }
    }
  };
  // ... then F and dU on the vector units, packed as the operands of the two
  // 16-row halves; DIAG: the block whose rows start at this wave's first key
  // (row offset acc_row(r, g) against key offset n)
  auto grads = [&](const unsigned char* buf, int qb, floatx16& s, floatx16& dp, Op (&fop)[2], Op (&uop)[2],
                   auto diag_c) {
    constexpr bool DIAG = decltype(diag_c)::value;
    const float* Mrow = (const float*)(buf + 2 * TB);
    floatx16 Mb;  // per register: M log2(e) of its query row
#pragma unroll
    for (int rq = 0; rq < 4; ++rq) {
      const floatx4 M4 = *(const floatx4*)(Mrow + 32 * qb + 8 * rq + 4 * g);
#pragma unroll
      for (int t = 0; t < 4; ++t) Mb[4 * rq + t] = M4[t];
    }
    float uself = 0.0f, dself = 0.0f;
    const int rs = row_reg(n);
    if (DIAG) {
      uself = pick(s, rs);
      dself = pick(dp, rs);
      // exchange-only: dL/dF_ii = 0, so dR_ii = -F_ii D_i with -D_i of the query row equal to the key
      if (a.exch_only) dself = ((const float*)(buf + 2 * TB) + kBQI)[32 * qb + n];
    }
    exchange_grads(s, dp, [&](int r) { return Mb[r]; }, c);
    if (DIAG) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        if (acc_row(r, g) < n) {  // query before the key: no flow
          s[r] = 0.0f;
          dp[r] = 0.0f;
        }
      }
      if (holds_row(n, g)) {
        const float ln_i = logf((float)(kj + 1));
        const SelfGrad sg = self_grad(uself, dself, Mb[rs], a.scale, a.inv_tau, lam, ln_i, kj == 0);
        if (FQ && kj < T) {
          red[32 * w + n] = ln_i * sg.dR;  // this key's dlambda term (each key's diagonal is met once)
          if (a.dself) a.dself[(int64_t)head * T + kj] = sg.dR;
        }
        const float fself = a.exch_only ? 0.0f : sg.F;  // F_ii carries dO_i to v_i unless exchange-only
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          s[r] = r == rs ? fself : s[r];
          dp[r] = r == rs ? sg.dU : dp[r];
        }
      }
    }
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
      float f8[8], u8[8];
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        f8[t] = s[8 * hh + t];
        u8[t] = dp[8 * hh + t];
      }
      fop[hh] = P::pack(f8);
      uop[hh] = P::pack(u8);
    }
  };
  // dV += F^T dO and dK += dU^T Q for 16-row half hh of query block qb (the wave's channels)
  auto accum_half = [&](const unsigned char* buf, int qb, int hh, const Op& fop, const Op& uop) {
    const unsigned char* Qs = buf;
    const unsigned char* dOs = buf + TB;
#pragma unroll
    for (int db = 0; db < DBH; ++db) {
      const int c0 = 32 * (db + chw * DBH);
      dVt[db] = P::mma(P::col_op(dOs, 2 * qb + hh, c0, L), fop, dVt[db]);
      dKt[db] = P::mma(P::col_op(Qs, 2 * qb + hh, c0, L), uop, dKt[db]);
    }
  };
  auto accum = [&](const unsigned char* buf, int qb, const Op (&fop)[2], const Op (&uop)[2]) {
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) accum_half(buf, qb, hh, fop[hh], uop[hh]);
  };
  // CS: slot of operand k (0, 1: F halves; 2, 3: dU halves) of query block qb of the wave's key group
  auto xslot = [&](int qb, int k) { return (uintx4*)(Xch + ((((kgw * 2 + qb) * 4 + k) * 64) + lane) * 16); };

  // fused: dU of one query block (rows 32 qb .. of the tile) into the LDS dU
  // tile, row = key, column = query position. Positions within each block are
  // the queries with bits 2 and 3 of their index swapped, so that the 8 queries
  // of a lane's operand half (16 hh + 4 g + 0..3 and 16 hh + 8 + 4 g + 0..3) are
  // one 16-byte chunk: one write per half, and the 16 lanes of each write phase
  // meet distinct banks.
  auto write_dU = [&](unsigned char* dUw, int qb, const Op (&uop)[2]) __attribute__((always_inline)) {
    if constexpr (FQ) {
      int kr = 32 * w + n;
      asm volatile("" : "+v"(kr));  // formed here, not held in a register across the tile loop
      unsigned char* t = dUw + (kr >> 6) * DUT;
#pragma unroll
      for (int hh = 0; hh < 2; ++hh)
        *(uintx4*)(t + PU::off(kr & 63, 32 * qb + 16 * hh + 8 * g)) = __builtin_bit_cast(uintx4, uop[hh]);
    }
  };
  // fused: the dQ partial of query tile i0 .. i0+63 from its dU tile, one
  // 32 x 32 block per wave (waves 0 .. 2 D/32 - 1), added to the fp32
  // accumulator. (A 16x16x32 split over all eight waves was slower: its
  // atomics touch four 64-byte row pieces per instruction instead of two
  // 128-byte rows.)
  auto dq_tile = [&](const unsigned char* dUr, int i0) __attribute__((always_inline)) {
    if constexpr (FQ) if (w < 2 * DB) {
      const int qb = w / DB, db = w % DB;
      // two independent accumulation chains (even and odd key slices), so that
      // consecutive products do not wait on each other's result
      floatx16 acc = {}, acc2 = {};
#pragma unroll
      for (int kq = 0; kq < KW / 16; kq += 2) {
        const Op ua = PU::col_op(dUr + (kq >> 2) * DUT, kq & 3, 32 * qb, L);
        const Op kb = P::col_op(Kq + (kq >> 2) * TB, kq & 3, 32 * db, L);
        const Op ua2 = PU::col_op(dUr + ((kq + 1) >> 2) * DUT, (kq + 1) & 3, 32 * qb, L);
        const Op kb2 = P::col_op(Kq + ((kq + 1) >> 2) * TB, (kq + 1) & 3, 32 * db, L);
        acc = P::mma(ua, kb, acc);
        acc2 = P::mma(ua2, kb2, acc2);
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[r] += acc2[r];
      // register r holds position acc_row(r, g) = 8 (r / 4) + 4 g + r % 4 of the
      // block, that is query 16 (r / 8) + 8 g + r % 8 (bits 2 and 3 swapped back),
      // column n: a uniform base, one lane offset and a constant per register
      float* base = a.dq_acc + ((int64_t)head * T + i0 + 32 * qb) * D + 32 * db;
      int off = 8 * g * D + n;
      asm volatile("" : "+v"(off));  // formed here, not held in a register across the tile loop
      const int lim = T - i0 - 32 * qb;  // rows of the block inside the sequence
      if (lim >= 32) {
#pragma unroll
        for (int r = 0; r < 16; ++r) unsafeAtomicAdd(base + off + (16 * (r >> 3) + (r & 7)) * D, acc[r]);
      } else {
#pragma unroll
        for (int r = 0; r < 16; ++r)
          if (16 * (r >> 3) + (r & 7) + 8 * g < lim) unsafeAtomicAdd(base + off + (16 * (r >> 3) + (r & 7)) * D, acc[r]);
      }
    }
  };

  const int kfirst = wave_keys ? kw0 : (1 << 30);  // a wave past T meets no query
  // One query tile. A block before the wave's keys or past T contributes zero
  // F and dU, so the dV / dK products (and the accumulators) run on every
  // path. Order: evidence of block 0, its vector work, evidence of block 1,
  // then the products of block 0 (which run under the vector work of block 1).
  auto step = [&](int qt, const unsigned char* buf, unsigned char* nxt, unsigned char* dUw,
                  const unsigned char* dUr) __attribute__((always_inline)) {
    const int i0 = qt * kBQI;
    wait_loads();
    __syncthreads();
    if (qt + 1 < nqt) load_tile(i0 + kBQI, nxt);
    if (FQ && qt > qt0) {
      __builtin_amdgcn_sched_barrier(0);
      dq_tile(dUr, i0 - kBQI);
      __builtin_amdgcn_sched_barrier(0);
    }
    if constexpr (CS == 2) {
      // this wave's query block: its F and dU, swapped with the partner's
      const int qm = i0 + 32 * chw;
      floatx16 sm, dpm;
      Op fm[2] = {Op{}, Op{}}, um[2] = {Op{}, Op{}};
      if (qm >= kfirst && qm < T) {
        evid(buf, chw, sm, dpm);
        if (qm == kfirst) grads(buf, chw, sm, dpm, fm, um, std::true_type{});
        else grads(buf, chw, sm, dpm, fm, um, std::false_type{});
      }
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        *xslot(chw, hh) = __builtin_bit_cast(uintx4, fm[hh]);
        *xslot(chw, 2 + hh) = __builtin_bit_cast(uintx4, um[hh]);
      }
      accum(buf, chw, fm, um);  // its own block first: these products run while the partner catches up
      __syncthreads();
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {  // the partner's block, one 16-row half at a time
        const Op fo = __builtin_bit_cast(Op, *xslot(1 - chw, hh));
        const Op uo = __builtin_bit_cast(Op, *xslot(1 - chw, 2 + hh));
        accum_half(buf, 1 - chw, hh, fo, uo);
      }
      return;
    }
    const int q0 = i0, q1 = i0 + 32;
    const bool live0 = q0 >= kfirst && q0 < T, live1 = q1 >= kfirst && q1 < T;
    floatx16 s0, dp0, s1, dp1;
    Op f0[2] = {Op{}, Op{}}, u0[2] = {Op{}, Op{}}, f1[2] = {Op{}, Op{}}, u1[2] = {Op{}, Op{}};
    if (live0) {
      evid(buf, 0, s0, dp0);
      if (q0 == kfirst) grads(buf, 0, s0, dp0, f0, u0, std::true_type{});
      else grads(buf, 0, s0, dp0, f0, u0, std::false_type{});
    }
    if (live1) evid(buf, 1, s1, dp1);
    __builtin_amdgcn_sched_barrier(0);
    accum(buf, 0, f0, u0);
    write_dU(dUw, 0, u0);
    __builtin_amdgcn_sched_barrier(0);
    if (live1) {
      if (q1 == kfirst) grads(buf, 1, s1, dp1, f1, u1, std::true_type{});
      else grads(buf, 1, s1, dp1, f1, u1, std::false_type{});
    }
    accum(buf, 1, f1, u1);
    write_dU(dUw, 1, u1);
  };
  // A full tile (both blocks live and past every wave's diagonal) is one
  // basic block: the evidence of block 1 and then the products of block 0 are
  // interleaved with the vector work of blocks 0 and 1, so that one wave keeps
  // the matrix and the vector units busy together.
  auto full = [&](int qt, const unsigned char* buf, unsigned char* nxt, unsigned char* dUw,
                  const unsigned char* dUr) __attribute__((always_inline)) {
    const int i0 = qt * kBQI;
    wait_loads();
    __syncthreads();
    if (qt + 1 < nqt) load_tile(i0 + kBQI, nxt);
    if (FQ && qt > qt0) {
      __builtin_amdgcn_sched_barrier(0);
      dq_tile(dUr, i0 - kBQI);
      __builtin_amdgcn_sched_barrier(0);
    }
    floatx16 s0, dp0, s1, dp1;
    Op f0[2], u0[2], f1[2], u1[2];
    evid(buf, 0, s0, dp0);
    __builtin_amdgcn_sched_barrier(0);
    evid(buf, 1, s1, dp1);
    grads(buf, 0, s0, dp0, f0, u0, std::false_type{});
    interleave<2 * KS, kDkdvIlValu, 0>();
    __builtin_amdgcn_sched_barrier(0);
    accum(buf, 0, f0, u0);
    write_dU(dUw, 0, u0);
    grads(buf, 1, s1, dp1, f1, u1, std::false_type{});
    interleave<4 * DB, kDkdvIlValu, 1>();
    __builtin_amdgcn_sched_barrier(0);
    accum(buf, 1, f1, u1);
    write_dU(dUw, 1, u1);
  };
  // tiles alternate between bufA and bufB (and the dU tiles between dUA and
  // dUB), starting with bufA at qt0
  auto run = [&](int qa, int qb, auto st) __attribute__((always_inline)) {
    int qt = qa;
    if (qt < qb && ((qt - qt0) & 1)) {
      st(qt, bufB, bufA, dUB, dUA);
      ++qt;
    }
    for (; qt < qb; qt += 2) {
      st(qt, bufA, bufB, dUA, dUB);
      if (qt + 1 < qb) st(qt + 1, bufB, bufA, dUB, dUA);
    }
  };
  const int qf0 = min(qt0 + KW / kBQI, nqt);  // tiles with the workgroup's diagonals
  const int qf1 = max(qf0, T / kBQI);           // full tiles end here
  if constexpr (CS == 2) {
    run(qt0, nqt, step);
  } else {
    run(qt0, qf0, step);
    run(qf0, qf1, full);
    run(qf1, nqt, step);
  }
  if constexpr (FQ) {
    // the last tile's dQ, and this workgroup's dlambda partial in a fixed order
    __syncthreads();
    dq_tile(((nqt - 1 - qt0) & 1) ? dUB : dUA, (nqt - 1) * kBQI);
    float t = tid < KW ? red[tid] : 0.0f;
#pragma unroll
    for (int s = 32; s >= 1; s >>= 1) t += __shfl_xor(t, s, 64);
    __syncthreads();
    if (lane == 0) red[w] = t;
    __syncthreads();
    if (tid == 0) {
      float sum = 0.0f;
      for (int i = 0; i < NW; ++i) sum += red[i];
      a.dlam_part[blockIdx.x] = sum;
    }
  }

  if (kj < T) {
    E* dk = (E*)a.dk + hoff;
    E* dv = (E*)a.dv + hoff;
#pragma unroll
    for (int db = 0; db < DBH; ++db)
#pragma unroll
      for (int rq = 0; rq < 4; ++rq) {
        const int d0 = 32 * (db + chw * DBH) + 8 * rq + 4 * g;
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
// Fused backward (bf16, D <= 64): the row pass before and the dQ pass after
// the dK/dV/dQ kernel.
// ---------------------------------------------------------------------------
constexpr int kRowNT = 256;

// Row r of the [N, T] row space: its head and the element offset of its row.
__device__ __forceinline__ int64_t row_offset(const BwdArgs& a, int64_t r) {
  const int head = (int)(r / a.T), t = (int)(r % a.T);
  return (int64_t)(head / a.H) * a.sb + (int64_t)(head % a.H) * a.sh + (int64_t)t * a.st;
}

// D_i = dO_i . o_i (stored as -D_i), M_i log2(e), and the row's fp32 dQ
// accumulator cleared. D/8 lanes per row, 16 bytes each.
template <int D>
__global__ __launch_bounds__(kRowNT) void bwd_prep_kernel(BwdArgs a) {
  constexpr int LPR = D / 8, RPB = kRowNT / LPR;
  const int tid = threadIdx.x, c = tid % LPR;
  const int64_t r = (int64_t)blockIdx.x * RPB + tid / LPR;
  const bool ok = r < (int64_t)a.map.N * a.T;
  float part = 0.0f;
  if (ok) {
    const int64_t off = row_offset(a, r) + 8 * c;
    part = PolBF16<D>::chunk_dot(*(const uintx4*)((const bf16*)a.o + off), *(const uintx4*)((const bf16*)a.dout + off));
  }
  const float Di = lane_group_sum<LPR>(part);  // every lane takes part
  if (ok) {
    if (c == 0) {
      a.negd[r] = -Di;
      a.m2[r] = a.row_stat[r] * kLog2e;
    }
    floatx4* acc = (floatx4*)(a.dq_acc + r * D + 8 * c);
    acc[0] = floatx4{};
    acc[1] = floatx4{};
  }
}

// dq = scale * (fp32 accumulator) in bf16; block 0 first sums the dlambda
// partials of the fused kernel (which ran before on the stream) in a fixed
// order.
template <int D>
__global__ __launch_bounds__(kRowNT) void bwd_dq_convert_kernel(BwdArgs a) {
  constexpr int LPR = D / 8, RPB = kRowNT / LPR;
  const int tid = threadIdx.x, c = tid % LPR;
  if (blockIdx.x == 0 && a.dlambda) {
    __shared__ float red[kRowNT];
    float acc = 0.0f;
    for (int i = tid; i < a.nparts; i += kRowNT) acc += a.dlam_part[i];
    red[tid] = acc;
    __syncthreads();
    for (int h = kRowNT / 2; h >= 1; h >>= 1) {
      if (tid < h) red[tid] += red[tid + h];
      __syncthreads();
    }
    if (tid == 0) *a.dlambda = red[0];
  }
  const int64_t r = (int64_t)blockIdx.x * RPB + tid / LPR;
  if (r >= (int64_t)a.map.N * a.T) return;
  const floatx4* acc = (const floatx4*)(a.dq_acc + r * D + 8 * c);
  const floatx4 x0 = acc[0], x1 = acc[1];
  bf16x8 y;
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    y[t] = (bf16)(a.scale * x0[t]);
    y[4 + t] = (bf16)(a.scale * x1[t]);
  }
  *(bf16x8*)((bf16*)a.dq + row_offset(a, r) + 8 * c) = y;
}

// The two-kernel dK/dV kernel runs with its channels split over wave pairs
// (CS = 2, 8 waves for 128 keys) at bf16 D = 128, where one wave's dK and dV
// accumulators would take 128 registers.
template <class P, int D>
constexpr bool kSplitChannels = sizeof(typename P::T) == 2 && D == 128;

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
  if constexpr (kSplitChannels<P, D>) {
    hipLaunchKernelGGL((bwd_dkdv_kernel<P, D, 8, false, 2>), dim3((unsigned)grid_size(mkv)), dim3(512), 0, stream, b);
  } else {
    hipLaunchKernelGGL((bwd_dkdv_kernel<P, D, 4, false>), dim3((unsigned)grid_size(mkv)), dim3(kNT), 0, stream, b);
  }
  if (p_kv) (void)hipEventRecord(e1, stream);
  if (p_all) (void)hipEventRecord(prof[1], stream);
}

// The fused backward: row pass, the dK/dV/dQ kernel (256 keys per workgroup),
// dQ pass.
template <int D>
void launch_fused(const BwdArgs& a, hipStream_t stream, hipEvent_t* prof) {
  constexpr int NW = kFusedWaves;
  BwdArgs b = a;
  const int64_t rows = (int64_t)a.map.N * a.T;
  const unsigned row_blocks = (unsigned)((rows + kRowNT / (D / 8) - 1) / (kRowNT / (D / 8)));
  hipEvent_t e0, e1;
  const bool p_all = prof != nullptr;
  if (p_all) (void)hipEventRecord(prof[0], stream);
  const bool p_r = !p_all && profile_slot("bwd_prep", &e0, &e1);
  if (p_r) (void)hipEventRecord(e0, stream);
  hipLaunchKernelGGL((bwd_prep_kernel<D>), dim3(row_blocks), dim3(kRowNT), 0, stream, b);
  if (p_r) (void)hipEventRecord(e1, stream);
  b.map = make_tilemap(a.map.N, (a.T + 32 * NW - 1) / (32 * NW));
  const bool p_kv = !p_all && profile_slot("bwd_dkdv", &e0, &e1);
  if (p_kv) (void)hipEventRecord(e0, stream);
  hipLaunchKernelGGL((bwd_dkdv_kernel<PolBF16<D>, D, NW, true>), dim3((unsigned)grid_size(b.map)), dim3(64 * NW), 0,
                     stream, b);
  if (p_kv) (void)hipEventRecord(e1, stream);
  b.map = a.map;
  const bool p_c = !p_all && profile_slot("bwd_convert", &e0, &e1);
  if (p_c) (void)hipEventRecord(e0, stream);
  hipLaunchKernelGGL((bwd_dq_convert_kernel<D>), dim3(row_blocks), dim3(kRowNT), 0, stream, b);
  if (p_c) (void)hipEventRecord(e1, stream);
  if (p_all) (void)hipEventRecord(prof[1], stream);
}

}  // namespace

// The one-kernel backward pays a fixed cost per row (the row pass and the dq
// pass move about 5 D bytes per row) that the removed dq recompute, whose cost
// grows with T, outweighs from T of about 1.6K on (measured at T = 1024 and 2048).
bool bwd_fused_supported(int T, int D, int dtype) { return dtype == 1 && (D == 32 || D == 64) && T >= 1536; }

int bwd_partials(int N, int T, int D, int dtype, bool fused) {
  (void)D;
  (void)dtype;
  if (fused) return (int)grid_size(make_tilemap(N, (T + 32 * kFusedWaves - 1) / (32 * kFusedWaves)));
  return (int)grid_size(make_tilemap(N, (T + kBQ - 1) / kBQ));
}

hipError_t launch_bwd(const BwdArgs& a, int dtype, int D, hipStream_t stream) {
  const int N = a.map.N;
  if (a.dq_acc) {
    hipEvent_t ev[2];
    const bool prof = profile_slot("bwd", &ev[0], &ev[1]);
    if (D == 32) launch_fused<32>(a, stream, prof ? ev : nullptr);
    else launch_fused<64>(a, stream, prof ? ev : nullptr);
    return hipGetLastError();
  }
  const TileMap mkv = make_tilemap(N, (a.T + kBKW - 1) / kBKW);
  const TileMap mq = make_tilemap(N, (a.T + kBQ - 1) / kBQ);
  hipEvent_t ev[2];
  const bool prof = profile_slot("bwd", &ev[0], &ev[1]);
  hipEvent_t* pe = prof ? ev : nullptr;
  if (dtype == 1) {
    if (D == 32) launch_pair<PolBF16<32>, 32>(a, mkv, mq, stream, pe);
    else if (D == 64) launch_pair<PolBF16<64>, 64>(a, mkv, mq, stream, pe);
    else if (D == 96) launch_pair<PolBF16<96>, 96>(a, mkv, mq, stream, pe);
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


}  // namespace rel
