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
// underflow to an all-zero row; the reference is raised only when a block's
// largest E exceeds it by more than 8 (in log2 units), which keeps every
// exp2 argument <= 8 and the sums far from fp32 overflow. Any reference gives
// the same ratios z/l and L^E = m + ln l, so the result is exact. The test is
// lane-local; only a raise combines the two halves of a row.
//
// Two kernels:
//  * bf16 (fwdb_kernel): K/V tiles go HBM -> LDS directly (buffer loads to
//    LDS, 16 bytes per lane), two buffers, one barrier per tile, so no staging
//    registers are held. With 4 waves a wave scans every 64-key tile for its 32
//    rows; with 8 waves, waves 0-3 scan the first 64 keys of every 128-key tile
//    and waves 4-7 the last 64 for the same rows, and the two partial scan
//    states of a row are merged at the end (the (m, l, z) state is
//    associative: m = max, l and z rescaled and added).
//  * fp32 (fwd_kernel): 4 waves per workgroup, 64-key tiles staged through
//    registers into padded LDS rows.
#include "kernels.h"

#include <type_traits>

namespace rel {

namespace {

constexpr int kBQ = 128;  // query rows per workgroup
constexpr float kRescale = 8.0f;
#ifndef REL_FWD_WAVES_PER_SIMD
#define REL_FWD_WAVES_PER_SIMD 2  // occupancy of the fp32 kernel
#endif

// How the query operand carries c = scale log2(e):
//   0: raw q; each evidence entry is multiplied by c
//   1: q c in the operand (fp32)
//   2: q c as bf16 hi + lo, two MFMAs per slice
#ifndef REL_FWD_BF16_QMODE
#define REL_FWD_BF16_QMODE 0
#endif
template <class P, int D>
constexpr int qmode() {
  return sizeof(typename P::T) == 4 ? 1 : (D <= 64 ? REL_FWD_BF16_QMODE : 0);
}

// Exchange logits of one 32x32 block, in place: s[r] (U log2 e, or raw q.k in
// mode 0) becomes E log2(e) - m; in the diagonal block (DIAG) entries with
// key >= query get -inf. mx tracks the lane's largest value.
template <bool DIAG, int QM>
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
    mx = fmaxf(mx, fmaxf(fmaxf(s[r0], s[r0 + 1]), fmaxf(s[r0 + 2], s[r0 + 3])));
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
template <class P, int KS, int QM>
__device__ __forceinline__ floatx16 evidence(const unsigned char* Ks, int krow0, const typename P::Op (&qhi)[KS],
                                             const typename P::Op (&qlo)[KS], const Lane& L) {
  floatx16 s = {};
#pragma unroll
  for (int k0 = 0; k0 < KS; k0 += 2) {  // operands two slices at a time
    typename P::Op ka[2];
#pragma unroll
    for (int j = 0; j < 2; ++j) ka[j] = P::row_op(Ks, krow0 + L.n, k0 + j, L);
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      s = P::mma(ka[j], qhi[k0 + j], s);
      if (QM == 2) s = P::mma(ka[j], qlo[k0 + j], s);
    }
  }
  return s;
}

// The 64 keys krow0 .. krow0+63 of a tile (two 32-key blocks) for a wave whose
// rows start at qr0 and whose keys start at kglob (global index of krow0).
template <class P, int D, int QM>
__device__ __forceinline__ void scan_keys64(const unsigned char* Ks, const unsigned char* Vs, int krow0, int kglob,
                                            int qr0, const typename P::Op (&qhi)[D / 16],
                                            const typename P::Op (&qlo)[D / 16], floatx16 (&oacc)[D / 32], float& m,
                                            float& l, float& uii, const Lane& L, float c) {
  constexpr int KS = D / 16;
  const int vs0 = krow0 / 16;
  // one block at a time: the evidence of block 1 is formed only after block 0
  // is mapped, which keeps the register footprint small enough for four
  // waves per SIMD (the other waves fill the matrix-core latency)
  if (kglob + 64 <= qr0) {  // both blocks before every row: the common case
    scan_block<P, D, QM, false>(evidence<P, KS, QM>(Ks, krow0, qhi, qlo, L), oacc, m, l, uii, Vs, vs0, L, c);
    scan_block<P, D, QM, false>(evidence<P, KS, QM>(Ks, krow0 + 32, qhi, qlo, L), oacc, m, l, uii, Vs, vs0 + 2, L, c);
  } else if (kglob + 32 == qr0) {  // block 1 is the diagonal block
    scan_block<P, D, QM, false>(evidence<P, KS, QM>(Ks, krow0, qhi, qlo, L), oacc, m, l, uii, Vs, vs0, L, c);
    scan_block<P, D, QM, true>(evidence<P, KS, QM>(Ks, krow0 + 32, qhi, qlo, L), oacc, m, l, uii, Vs, vs0 + 2, L, c);
  } else if (kglob == qr0) {  // block 0 is the diagonal block, block 1 lies above it
    scan_block<P, D, QM, true>(evidence<P, KS, QM>(Ks, krow0, qhi, qlo, L), oacc, m, l, uii, Vs, vs0, L, c);
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
#pragma unroll
  for (int db = 0; db < DB; ++db) {
#pragma unroll
    for (int rq = 0; rq < 4; ++rq) {
      const int d0 = 32 * db + 8 * rq + 4 * L.g;
      const floatx4 vi = P::load4(v + qi * st + d0);
      floatx4 out;
#pragma unroll
      for (int t = 0; t < 4; ++t) out[t] = __builtin_fmaf(e.omg, vi[t], e.inv_l * oacc[db][4 * rq + t]);
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

// The query operand of this lane's row (times c unless mode 0).
template <class P, int KS, int QM>
__device__ __forceinline__ void load_query(const typename P::T* q, int64_t st, int qi, int T, const Lane& L, float c,
                                           typename P::Op (&qhi)[KS], typename P::Op (&qlo)[KS]) {
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    qhi[ks] = typename P::Op{};
    qlo[ks] = typename P::Op{};
    if (qi < T) {
      if (QM == 0) qhi[ks] = P::row_op_g(q + qi * st, ks, L);
      else P::row_op_scaled(q + qi * st, ks, L, c, qhi[ks], qlo[ks]);
    }
  }
}

// ---------------------------------------------------------------------------
// bf16: NW = 4 or 8 waves. With 8, waves 0-3 and 4-7 take the two 64-key
// halves of every 128-key tile for the same 128 rows and merge at the end.
// ---------------------------------------------------------------------------
#ifndef REL_FWD_BF16_WAVES
#define REL_FWD_BF16_WAVES 4
#endif
template <int NW, int D>
constexpr int fwd_bf16_occupancy() {
  return D > 64 ? 2 : (NW == 8 ? 4 : 3);
}

template <int D, int NW>
__global__ __launch_bounds__(NW * 64, (fwd_bf16_occupancy<NW, D>())) void fwdb_kernel(FwdArgs a) {
  using P = PolBF16<D>;
  using E = bf16;
  using Op = typename P::Op;
  constexpr int QM = qmode<P, D>();
  constexpr int KS = D / 16, DB = D / 32;
  constexpr int KH = NW / 4;                   // key halves
  constexpr int BK = 64 * KH;                  // keys per tile
  constexpr int TB = BK * P::ROWB;             // bytes of one tensor tile
  constexpr int SEG_ROWS = 1024 / P::ROWB;     // tile rows filled by one 64-lane load
  constexpr int NSEG = BK / SEG_ROWS;          // such loads per tensor tile
  constexpr int SEGW = 2 * NSEG / NW;          // per wave, K and V together
  static_assert(2 * NSEG % NW == 0 && 64 % P::NCH == 0, "tile does not split over the waves");
  __shared__ __attribute__((aligned(1024))) unsigned char lds[2][2 * TB];

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
  const int rw = w & 3, kh = w >> 2;  // row group, key half
  const int i0 = qt * kBQ, qr0 = i0 + 32 * rw, qi = qr0 + L.n;
  const bool wave_live = qr0 < T;
  const float c = a.scale * kLog2e;

  // One 1 KB segment per load: lane l fills physical chunk l % NCH of tile row
  // r0 + l / NCH, which holds logical chunk (l % NCH) ^ (row & SWZ) (the XOR
  // swizzle of the tile layout). Rows past T repeat row T-1: such keys only
  // meet masked (zero) weights. Buffer loads take a scalar base per tensor and
  // head and a 32-bit byte offset per lane (the host keeps a head within 2 GiB).
  const int row_bytes = (int)(st * 2);
  const __amdgpu_buffer_rsrc_t krs = __builtin_amdgcn_make_buffer_rsrc((void*)k, (short)0, T * row_bytes, 0x00020000);
  const __amdgpu_buffer_rsrc_t vrs = __builtin_amdgcn_make_buffer_rsrc((void*)v, (short)0, T * row_bytes, 0x00020000);
  auto load_tile = [&](int j0, int buf) {
    const int last = T - 1 - j0;  // last valid row of this tile
#pragma unroll
    for (int s = 0; s < SEGW; ++s) {
      const int seg = w * SEGW + s;
      const int tens = seg / NSEG, r0 = (seg % NSEG) * SEG_ROWS;
      const int row = r0 + lane / P::NCH, ch = (lane % P::NCH) ^ (row & P::SWZ);
      const int voff = min(row, last) * row_bytes + 16 * ch;
      unsigned char* dst = lds[buf] + tens * TB + r0 * P::ROWB;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(tens ? vrs : krs, (__attribute__((address_space(3))) void*)dst, 16,
                                               voff, j0 * row_bytes, 0, 0);
    }
  };

  Op qhi[KS], qlo[KS];
  load_query<P, KS, QM>(q, st, qi, T, L, c, qhi, qlo);

  float m = 0.0f, l = 0.0f, uii = 0.0f;
  floatx16 oacc[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) oacc[db] = floatx16{};

  const int kmax = min(i0 + kBQ, T) - 1;  // the diagonal of the last row is included
  const int nkt = kmax / BK + 1;
  load_tile(0, 0);
  for (int kt = 0; kt < nkt; ++kt) {
    __builtin_amdgcn_s_waitcnt(0x0f70);  // vmcnt(0): this wave's part of tile kt is in LDS
    __syncthreads();                     // ... and every wave's; tile kt-1 is no longer read
    if (kt + 1 < nkt) load_tile((kt + 1) * BK, (kt + 1) & 1);
    if (wave_live) {
      const unsigned char* Ks = lds[kt & 1];
      scan_keys64<P, D, QM>(Ks, Ks + TB, 64 * kh, kt * BK + 64 * kh, qr0, qhi, qlo, oacc, m, l, uii, L, c);
    }
  }

  if (KH == 2) {
    // ---- merge the two key halves of every row (waves w and w + 4)
    constexpr int NV = DB * 16 + 3;  // values per lane: z, then m, l, U_ii
    static_assert(KH == 1 || 4 * NV * 64 * 4 <= 2 * 2 * TB, "merge buffer exceeds the tile buffers");
    float* red = (float*)&lds[0][0];
    __syncthreads();
    if (kh == 1 && wave_live) {
      float* r = red + rw * NV * 64 + lane;
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int t = 0; t < 16; ++t) r[(16 * db + t) * 64] = oacc[db][t];
      r[(DB * 16) * 64] = m;
      r[(DB * 16 + 1) * 64] = l;
      r[(DB * 16 + 2) * 64] = uii;
    }
    __syncthreads();
    if (kh == 1 || !wave_live) return;
    const float* r = red + rw * NV * 64 + lane;
    const float m1 = r[(DB * 16) * 64], l1 = r[(DB * 16 + 1) * 64], u1 = r[(DB * 16 + 2) * 64];
    const float mt = fmaxf(m, m1);
    const float a0 = fast_exp2(m - mt), a1 = fast_exp2(m1 - mt);
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int t = 0; t < 16; ++t) oacc[db][t] = __builtin_fmaf(oacc[db][t], a0, r[(16 * db + t) * 64] * a1);
    l = __builtin_fmaf(l, a0, l1 * a1);
    m = mt;
    uii += u1;  // only the half that met the diagonal block set it
  }
  if (!wave_live) return;
  finish_row<P, D, QM>(a, o, v, st, head, qi, m, l, uii, oacc, L, c);
}

// ---------------------------------------------------------------------------
// fp32: 4 waves, 64-key tiles through registers into padded LDS rows
// ---------------------------------------------------------------------------
constexpr int kBK = 64;   // keys per tile
constexpr int kNT = 256;  // threads per workgroup

template <class P, int D>
__global__ __launch_bounds__(kNT, REL_FWD_WAVES_PER_SIMD) void fwd_kernel(FwdArgs a) {
  using E = typename P::T;
  using Op = typename P::Op;
  using Chunk = typename P::Chunk;
  constexpr int QM = qmode<P, D>();
  constexpr int KS = D / 16;                      // 16-wide slices of d
  constexpr int DB = D / 32;                      // 32-row blocks of O^T
  constexpr int NLD = kBK * P::NCH / kNT;         // chunks per thread per tensor
  static_assert(NLD >= 1, "tile too small for the workgroup");
  constexpr int TB = P::tile_bytes(kBK);
  __shared__ __attribute__((aligned(16))) unsigned char lds[2][2 * TB];

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
  const Lane L(tid & 63);
  const int i0 = qt * kBQ, qr0 = i0 + 32 * w, qi = qr0 + L.n;
  const bool wave_live = qr0 < T;
  const float c = a.scale * kLog2e;

  Op qhi[KS], qlo[KS];
  load_query<P, KS, QM>(q, st, qi, T, L, c, qhi, qlo);

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
  auto stage = [&](int buf) {
#pragma unroll
    for (int j = 0; j < NLD; ++j) {
      const int ci = tid + kNT * j, row = ci / P::NCH, ch = ci % P::NCH;
      P::stage(lds[buf], row, ch, kreg[j]);
      P::stage(lds[buf] + TB, row, ch, vreg[j]);
    }
  };

  float m = 0.0f, l = 0.0f, uii = 0.0f;
  floatx16 oacc[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) oacc[db] = floatx16{};

  const int kmax = min(i0 + kBQ, T) - 1;  // the diagonal of the last row is included
  const int nkt = kmax / kBK + 1;
  prefetch(0);
  stage(0);
  if (nkt > 1) prefetch(kBK);
  __syncthreads();
  for (int kt = 0; kt < nkt; ++kt) {
    if (wave_live) {
      const unsigned char* Ks = lds[kt & 1];
      scan_keys64<P, D, QM>(Ks, Ks + TB, 0, kt * kBK, qr0, qhi, qlo, oacc, m, l, uii, L, c);
    }
    if (kt + 1 < nkt) {
      stage((kt + 1) & 1);
      __syncthreads();
      if (kt + 2 < nkt) prefetch((kt + 2) * kBK);
    }
  }
  if (!wave_live) return;
  finish_row<P, D, QM>(a, o, v, st, head, qi, m, l, uii, oacc, L, c);
}

template <int D>
void launch_bf16(const FwdArgs& a, hipStream_t stream) {
  constexpr int NW = REL_FWD_BF16_WAVES;
  hipLaunchKernelGGL((fwdb_kernel<D, NW>), dim3((unsigned)grid_size(a.map)), dim3(NW * 64), 0, stream, a);
}
template <int D>
void launch_f32(const FwdArgs& a, hipStream_t stream) {
  hipLaunchKernelGGL((fwd_kernel<PolF32<D>, D>), dim3((unsigned)grid_size(a.map)), dim3(kNT), 0, stream, a);
}

}  // namespace

hipError_t launch_fwd(const FwdArgs& a0, int dtype, int D, hipStream_t stream) {
  FwdArgs a = a0;
  a.map = make_tilemap(a.map.N, (a.T + kBQ - 1) / kBQ);
  hipEvent_t ev0, ev1;
  const bool prof = profile_slot("fwd", &ev0, &ev1);
  if (prof) (void)hipEventRecord(ev0, stream);
  if (dtype == 1) {
    if (D == 32) launch_bf16<32>(a, stream);
    else if (D == 64) launch_bf16<64>(a, stream);
    else launch_bf16<128>(a, stream);
  } else {
    if (D == 32) launch_f32<32>(a, stream);
    else if (D == 64) launch_f32<64>(a, stream);
    else launch_f32<128>(a, stream);
  }
  hipError_t e = hipGetLastError();
  if (prof) (void)hipEventRecord(ev1, stream);
  return e;
}

}  // namespace rel
