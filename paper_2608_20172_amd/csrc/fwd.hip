// Fused forward pass of the causal Full Relation operator (FlashRelation).
//
// A workgroup owns 128 query rows of one head; a wave computes 32 of them. Per
// 32-key block a wave forms the transposed evidence block U^T = K Q^T with 32x32
// MFMAs, so each lane holds one query row and 16 keys of the block: the row
// reductions of the online scan stay inside the lane, plus one exchange with the
// partner lane 32 away at the end. The Exchange scan keeps (m, l, z) per row as
// in eqs. (11)-(12) of Sec. 5.1 / App. A.3, with Self excluded; Self and the
// count correction join only in the epilogue (eq. 13). The Self logit U_ii is
// read off the diagonal entry of the evidence block that holds row i.
//
// Running reference m. SiLU(U) >= -0.2785, so exp(E - m) with m = 0 can never
// underflow to an all-zero row. Any reference gives the same ratios z/l and
// L^E = m + ln l, so the result is exact as long as nothing overflows. The
// scan therefore runs with m fixed at 0 and checks the row total at the end:
// every weight is at most l, so l <= 2^64 bounds every weight and |z|. A wave
// with a row above that rescans with a lazy reference, raised only when a
// block's largest E exceeds it by more than 8 (in log2 units), which keeps
// every exp2 argument <= 8.
//
// K/V tiles of 64 keys go HBM -> LDS by buffer loads that write LDS directly
// (no staging registers), into two buffers with one barrier per tile; four
// waves per workgroup, three per SIMD for bf16 with d <= 64.
#include "kernels.h"

#include <type_traits>

namespace rel {

namespace {

constexpr int kBQ = 128;  // query rows per workgroup
constexpr float kRescale = 8.0f;
constexpr float kSpecMax = 18446744073709551616.0f;  // 2^64

constexpr int kIlValu = 28;  // vector instructions scheduled after each matrix instruction in full tiles

// How the query operand carries c = scale log2(e):
//   0 (bf16): raw q; each evidence entry is multiplied by c in fp32
//   1 (fp32): q c in the operand
template <class P, int D>
constexpr int qmode() {
  return sizeof(typename P::T) == 4 ? 1 : 0;
}

// Exchange logits of one 32x32 block, in place: s[r] (U log2 e, or raw q.k in
// mode 0) becomes E log2(e) - m; in the diagonal block (DIAG) entries with
// key >= query get -inf. mx tracks the lane's largest value.
template <bool DIAG, int QM, bool TRACK = true>
__device__ __forceinline__ void exchange_logits(floatx16& s, const Lane& L, float c, float m, float& mx) {
  // passes over groups of 4 independent entries: consecutive instructions do
  // not wait on a transcendental result, and few temporaries are live
#pragma unroll
  for (int r0 = 0; r0 < 16; r0 += 4) {
    float up[4], t[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) up[r] = QM == 0 ? s[r0 + r] * c : s[r0 + r];   // U log2(e)
#pragma unroll
    for (int r = 0; r < 4; ++r) t[r] = fast_exp2(-up[r]);
#pragma unroll
    for (int r = 0; r < 4; ++r) t[r] = fast_rcp(1.0f + t[r]);                  // sigmoid(U)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      float e = __builtin_fmaf(up[r], t[r], -m);                               // SiLU(U) log2(e) - m
      if (DIAG && acc_row(r0 + r, L.g) >= L.n) e = kNegInf;                    // strictly historical: j < i
      s[r0 + r] = e;
    }
    if (TRACK) mx = fmaxf(mx, fmaxf(fmaxf(s[r0], s[r0 + 1]), fmaxf(s[r0 + 2], s[r0 + 3])));
  }
}

// One 32-key block of the scan for this wave's 32 rows: s holds the block's
// evidence (layout of a 32x32 accumulator, keys on rows, queries on lanes);
// Vs is the V tile and vslice the index of the block's first 16-key slice.
template <class P, int D, int QM, bool DIAG>
__device__ __forceinline__ void scan_block(floatx16 s, floatx16 (&oacc)[D / 32], float& m, float& l,
                                           float& uii, const unsigned char* Vs, int vslice,
                                           const Lane& L, float c) {
  constexpr int DB = D / 32;
  using Op = typename P::Op;
  if (DIAG && holds_row(L.n, L.g)) uii = pick(s, row_reg(L.n));  // the Self evidence
  float mx = kNegInf;
  exchange_logits<DIAG, QM>(s, L, c, m, mx);
  if (wave_any(mx > kRescale)) {
    const float d = fmaxf(fmaxf(mx, xor32(mx)), 0.0f);  // row max over both halves
    m += d;
    const float al = fast_exp2(-d);
    l *= al;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int r = 0; r < 16; ++r) oacc[db][r] *= al;
#pragma unroll
    for (int r = 0; r < 16; ++r) s[r] -= d;
  }
  // l sums the fp32 p (not the bf16-rounded MFMA operand), so that L^E and the
  // saved statistic M carry no operand rounding
#pragma unroll
  for (int hh = 0; hh < 2; ++hh) {
    float p[8];
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      p[t] = fast_exp2(s[8 * hh + t]);
      l += p[t];
    }
    const Op pop = P::pack(p);
#pragma unroll
    for (int db = 0; db < DB; ++db) oacc[db] = P::mma(P::col_op(Vs, vslice + hh, 32 * db, L), pop, oacc[db]);
  }
}

// Evidence block: keys krow0 .. krow0+31 of the K tile against this lane's row.
template <class P, int KS>
__device__ __forceinline__ floatx16 evidence(const unsigned char* Ks, int krow0, const typename P::Op (&qop)[KS],
                                             const Lane& L) {
  floatx16 s = {};
#pragma unroll
  for (int k0 = 0; k0 < KS; k0 += 2) {  // operands two slices at a time
    typename P::Op ka[2];
#pragma unroll
    for (int j = 0; j < 2; ++j) ka[j] = P::row_op(Ks, krow0 + L.n, k0 + j, L);
#pragma unroll
    for (int j = 0; j < 2; ++j) s = P::mma(ka[j], qop[k0 + j], s);
  }
  return s;
}

// A block of the scan with the reference m held fixed: the logits of the block,
// the packed weights P of its two 16-key halves and their sum into l.
template <class P, int D, int QM, bool DIAG>
__device__ __forceinline__ void fast_block(floatx16 s, float m, float& l, float& uii, typename P::Op (&pop)[2],
                                           const Lane& L, float c) {
  if (DIAG && holds_row(L.n, L.g)) uii = pick(s, row_reg(L.n));  // the Self evidence
  float mx = kNegInf;
  exchange_logits<DIAG, QM, false>(s, L, c, m, mx);
  // l sums the fp32 p (not the bf16-rounded MFMA operand), so that L^E and the
  // saved statistic M carry no operand rounding
#pragma unroll
  for (int hh = 0; hh < 2; ++hh) {
    float p[8];
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      p[t] = fast_exp2(s[8 * hh + t]);
      l += p[t];
    }
    pop[hh] = P::pack(p);
  }
}

// The 64 keys krow0 .. krow0+63 of a tile (two 32-key blocks, the first at
// global key kglob) for a wave whose rows start at qr0, with the reference
// held fixed. A block above the wave's rows contributes zero weights, so the
// P V products (and the accumulators) run on every path. FULL: both blocks lie
// below every row of the wave.
template <class P, int D, int QM, bool FULL>
__device__ __forceinline__ void fast_keys64(const unsigned char* Ks, const unsigned char* Vs, int krow0, int kglob,
                                            int qr0, const typename P::Op (&qop)[D / 16], floatx16 (&oacc)[D / 32],
                                            float m, float& l, float& uii, const Lane& L, float c) {
  constexpr int KS = D / 16, DB = D / 32;
  using Op = typename P::Op;
  auto pv = [&](int b, const Op (&pop)[2]) {
#pragma unroll
    for (int hh = 0; hh < 2; ++hh)
#pragma unroll
      for (int db = 0; db < DB; ++db)
        oacc[db] = P::mma(P::col_op(Vs, krow0 / 16 + 2 * b + hh, 32 * db, L), pop[hh], oacc[db]);
  };
  const int k0 = kglob, k1 = kglob + 32;
  Op p0[2] = {Op{}, Op{}}, p1[2] = {Op{}, Op{}};
  floatx16 s1;
  if (FULL) {
    // one basic block: the evidence of block 1 under the vector work of block
    // 0, the P V products of block 0 under that of block 1
    const floatx16 s0 = evidence<P, KS>(Ks, krow0, qop, L);
    __builtin_amdgcn_sched_barrier(0);
    s1 = evidence<P, KS>(Ks, krow0 + 32, qop, L);
    fast_block<P, D, QM, false>(s0, m, l, uii, p0, L, c);
    __builtin_amdgcn_sched_group_barrier(0x100, 64, 0);
#pragma unroll
    for (int i = 0; i < KS; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x002, kIlValu, 0);
    }
    __builtin_amdgcn_sched_barrier(0);
    pv(0, p0);
    fast_block<P, D, QM, false>(s1, m, l, uii, p1, L, c);
    __builtin_amdgcn_sched_group_barrier(0x100, 64, 1);
#pragma unroll
    for (int i = 0; i < 2 * DB; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 1);
      __builtin_amdgcn_sched_group_barrier(0x002, kIlValu, 1);
    }
    __builtin_amdgcn_sched_barrier(0);
    pv(1, p1);
    return;
  }
  // order: evidence of block 0, its vector work, evidence of block 1, then the
  // P V products of block 0 (which run under the vector work of block 1)
  if (k0 <= qr0) {
    const floatx16 s0 = evidence<P, KS>(Ks, krow0, qop, L);
    if (k0 == qr0) fast_block<P, D, QM, true>(s0, m, l, uii, p0, L, c);
    else fast_block<P, D, QM, false>(s0, m, l, uii, p0, L, c);
  }
  if (k1 <= qr0) s1 = evidence<P, KS>(Ks, krow0 + 32, qop, L);
  __builtin_amdgcn_sched_barrier(0);
  pv(0, p0);
  __builtin_amdgcn_sched_barrier(0);
  if (k1 <= qr0) {
    if (k1 == qr0) fast_block<P, D, QM, true>(s1, m, l, uii, p1, L, c);
    else fast_block<P, D, QM, false>(s1, m, l, uii, p1, L, c);
  }
  pv(1, p1);
}

// The same 64 keys, raising the running reference as needed (the rescan of a
// wave whose fixed-reference scan failed its row-total check; rare).
template <class P, int D, int QM>
__device__ __forceinline__ void slow_keys64(const unsigned char* Ks, const unsigned char* Vs, int krow0, int kglob,
                                            int qr0, const typename P::Op (&qop)[D / 16], floatx16 (&oacc)[D / 32],
                                            float& m, float& l, float& uii, const Lane& L, float c) {
  constexpr int KS = D / 16;
  for (int b = 0; b < 2; ++b) {
    const int kb0 = kglob + 32 * b;
    if (kb0 > qr0) break;
    const floatx16 s = evidence<P, KS>(Ks, krow0 + 32 * b, qop, L);
    if (kb0 == qr0) scan_block<P, D, QM, true>(s, oacc, m, l, uii, Vs, krow0 / 16 + 2 * b, L, c);
    else scan_block<P, D, QM, false>(s, oacc, m, l, uii, Vs, krow0 / 16 + 2 * b, L, c);
  }
}

struct RowEpilogue {
  float g, omg, inv_l, LE, lnZ, S;
};

// Completes row i from the terminal scan state (eqs. 12-13):
// L^E = m + ln l, A = L^E - lambda ln i, g = sigmoid(A - S), 1-g = sigmoid(S - A).
// uii2 = U_ii log2(e).
__device__ __forceinline__ RowEpilogue row_epilogue(float m_log2, float l, float uii2, float inv_tau,
                                                    float lam, float ln_i) {
  RowEpilogue e;
  e.S = 1.0f / (1.0f + exp2f(-uii2 * inv_tau));
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

// Row epilogue and stores for this lane's row qi from the terminal state of
// both lanes of the row (l, uii not yet combined across the two halves).
template <class P, int D, int QM>
__device__ __forceinline__ void finish_row(const FwdArgs& a, typename P::T* o, const typename P::T* v, int64_t st,
                                           int head, int qi, float m, float l, float uii,
                                           const floatx16 (&oacc)[D / 32], const Lane& L, float c) {
  constexpr int DB = D / 32;
  const int T = a.T;
  const float lt = l + xor32(l);
  const float u_other = xor32(uii);
  float un = holds_row(L.n, L.g) ? uii : u_other;
  if (QM == 0) un *= c;
  if (qi >= T) return;
  const float lam = *a.lambda;
  const float ln_i = logf((float)(qi + 1));
  const RowEpilogue e = row_epilogue(m, lt, un, a.inv_tau, lam, ln_i);
  const float wself = a.exch_only ? 0.0f : e.omg;  // the exchange-only ablation drops the Self term
#pragma unroll
  for (int db = 0; db < DB; ++db) {
#pragma unroll
    for (int rq = 0; rq < 4; ++rq) {
      const int d0 = 32 * db + 8 * rq + 4 * L.g;
      const floatx4 vi = P::load4(v + qi * st + d0);
      floatx4 out;
#pragma unroll
      for (int t = 0; t < 4; ++t) out[t] = __builtin_fmaf(wself, vi[t], e.inv_l * oacc[db][4 * rq + t]);
      P::store4(o + qi * st + d0, out);
    }
  }
  if (L.g == 0) {
    const int64_t ridx = (int64_t)head * T + qi;
    if (a.row_stat) a.row_stat[ridx] = e.lnZ + lam * ln_i;
    if (a.self_mass) a.self_mass[ridx] = e.omg;
    if (a.exch_mass) a.exch_mass[ridx] = e.g;
    if (a.exch_lse) a.exch_lse[ridx] = e.LE;
  }
}

// The query operand of this lane's row (times c in mode 1).
template <class P, int KS, int QM>
__device__ __forceinline__ void load_query(const typename P::T* q, int64_t st, int qi, int T, const Lane& L, float c,
                                           typename P::Op (&qop)[KS]) {
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    qop[ks] = typename P::Op{};
    if (qi < T) {
      if (QM == 0) {
        qop[ks] = P::row_op_g(q + qi * st, ks, L);
      } else {
        typename P::Op unused;
        P::row_op_scaled(q + qi * st, ks, L, c, qop[ks], unused);
      }
    }
  }
}

constexpr int kBK = 64;   // keys per tile
constexpr int kNT = 256;  // threads per workgroup

template <class P, int D>
constexpr int fwd_occupancy() {
  return sizeof(typename P::T) == 2 ? (D <= 64 ? 3 : 2) : (D <= 64 ? 2 : 1);  // waves per SIMD
}

template <class P, int D>
__global__ __launch_bounds__(kNT, (fwd_occupancy<P, D>())) void fwd_kernel(FwdArgs a) {
  using E = typename P::T;
  using Op = typename P::Op;
  constexpr int QM = qmode<P, D>();
  constexpr int KS = D / 16, DB = D / 32;
  constexpr int TB = kBK * P::ROWB;            // bytes of one tensor tile
  constexpr int NSEG = TB / 1024;              // 1 KB loads per tensor tile
  constexpr int SEGW = NSEG / 4;               // per wave and tensor
  static_assert(SEGW >= 1 && NSEG % 4 == 0, "tile does not split over the waves");
  // K and V tiles, two of each, as distinct objects: the compiler can then see
  // that reads of one do not wait for the loads in flight into another
  __shared__ __attribute__((aligned(1024))) unsigned char KA[TB];
  __shared__ __attribute__((aligned(1024))) unsigned char VA[TB];
  __shared__ __attribute__((aligned(1024))) unsigned char KB[TB];
  __shared__ __attribute__((aligned(1024))) unsigned char VB[TB];

  int head, qt;
  if (!map_tile(a.map, blockIdx.x, head, qt, true)) return;
  const int T = a.T;
  const int64_t st = a.st;
  const int64_t hoff = (int64_t)(head / a.H) * a.sb + (int64_t)(head % a.H) * a.sh;
  const E* q = (const E*)a.q + hoff;
  const E* k = (const E*)a.k + hoff;
  const E* v = (const E*)a.v + hoff;
  E* o = (E*)a.o + hoff;

  const int tid = threadIdx.x, w = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
  const int lane = tid & 63;
  const Lane L(lane);
  const int i0 = qt * kBQ, qr0 = i0 + 32 * w, qi = qr0 + L.n;
  const bool wave_live = qr0 < T;
  const float c = a.scale * kLog2e;

  // the head's K and V rows; keys past T read as zeros (they only meet masked
  // weights). The host keeps one head within 2 GiB.
  const int row_bytes = (int)(st * (int64_t)sizeof(E));
  const __amdgpu_buffer_rsrc_t krs = make_rsrc(k, T * row_bytes);
  const __amdgpu_buffer_rsrc_t vrs = make_rsrc(v, T * row_bytes);
  auto load_tile = [&](int j0, unsigned char* Kd, unsigned char* Vd) {
#pragma unroll
    for (int s = 0; s < SEGW; ++s) {
      dma_segment<P>(krs, Kd, w * SEGW + s, row_bytes, j0, lane);
      dma_segment<P>(vrs, Vd, w * SEGW + s, row_bytes, j0, lane);
    }
  };

  Op qop[KS];
  load_query<P, KS, QM>(q, st, qi, T, L, c, qop);

  float m = 0.0f, l = 0.0f, uii = 0.0f;
  floatx16 oacc[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) oacc[db] = floatx16{};

  const int kmax = min(i0 + kBQ, T) - 1;  // the diagonal of the last row is included
  const int nkt = kmax / kBK + 1;
  // Tiles alternate between the buffers: even ones in KA/VA, odd ones in KB/VB.
  const int qlast = wave_live ? qr0 : -1;  // rows of a wave past T meet no key
  auto fast_step = [&](auto full, int kt, const unsigned char* Ks, const unsigned char* Vs, unsigned char* Kn,
                       unsigned char* Vn) __attribute__((always_inline)) {
    wait_loads();      // this wave's part of tile kt is in LDS
    __syncthreads();   // ... and every wave's; tile kt-1 is no longer read
    if (kt + 1 < nkt) load_tile((kt + 1) * kBK, Kn, Vn);
    fast_keys64<P, D, QM, decltype(full)::value>(Ks, Vs, 0, kt * kBK, qlast, qop, oacc, m, l, uii, L, c);
  };
  auto run_fast = [&](int ka, int kb, auto full) __attribute__((always_inline)) {
    int kt = ka;
    if (kt < kb && (kt & 1)) {
      fast_step(full, kt, KB, VB, KA, VA);
      ++kt;
    }
    for (; kt < kb; kt += 2) {
      fast_step(full, kt, KA, VA, KB, VB);
      if (kt + 1 < kb) fast_step(full, kt + 1, KB, VB, KA, VA);
    }
  };
  load_tile(0, KA, VA);
  // tiles below the workgroup's first row have both blocks below every wave's rows
  const int kf = min(i0 / kBK, nkt);
  run_fast(0, kf, std::true_type{});
  run_fast(kf, nkt, std::false_type{});
  // The scan ran with the reference fixed at 0. Every weight is at most the row
  // total l, so l <= 2^64 bounds every weight and |z| <= l max|v|: then nothing
  // overflowed and the result is exact. Otherwise (or on inf / NaN) the wave's
  // rows are scanned again with the rescaling loop; the whole workgroup passes
  // the tiles again for the barriers.
  const float lt = l + xor32(l);
  const bool bad = wave_live && !(lt <= kSpecMax);
  if (__syncthreads_or(bad ? 1 : 0)) {
    const bool redo = wave_any(bad);
    if (redo) {
      m = 0.0f;
      l = 0.0f;
      uii = 0.0f;
#pragma unroll
      for (int db = 0; db < DB; ++db) oacc[db] = floatx16{};
    }
    load_tile(0, KA, VA);
    for (int kt = 0; kt < nkt; ++kt) {
      const bool odd = kt & 1;
      wait_loads();
      __syncthreads();
      if (kt + 1 < nkt) load_tile((kt + 1) * kBK, odd ? KA : KB, odd ? VA : VB);
      if (redo) slow_keys64<P, D, QM>(odd ? KB : KA, odd ? VB : VA, 0, kt * kBK, qlast, qop, oacc, m, l, uii, L, c);
    }
  }
  if (!wave_live) return;
  finish_row<P, D, QM>(a, o, v, st, head, qi, m, l, uii, oacc, L, c);
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
    else if (D == 96) launch_one<PolBF16<96>, 96>(a, stream);
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
