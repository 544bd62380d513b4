// Linear Relation (Sec. 5.2, App. A.4): Self stays explicit, Exchange reads a
// recurrent state C (D x D per head) with channel-wise retention alpha = exp(g).
//   S_t = sigmoid(p1_t . p2_t / (tau_S sqrt(D))),  ^p = p / |p|
//   C_t^- = Diag(alpha_t) C_{t-1};  Y_t = I~_t + S_t (C_t^-)^T ^p1_t;
//   C_t = C_t^- + S_t ^p2_t I~_t^T.
// The sequence is cut into chunks of kL tokens. With b the running sum of g
// inside a chunk (b_t = sum of g_u over the chunk's tokens u <= t), qt = S ^p1,
// kt = S ^p2, and C0 the state entering the chunk:
//   Y_t = I~_t + sum_a qt_{t,a} e^{b_{t,a}} C0[a, :]                     (inter)
//             + sum_{j<t in chunk} [sum_a qt_{t,a} kt_{j,a} e^{b_{t,a} - b_{j,a}}] I~_j   (intra)
//   C_end = Diag(e^{b_last}) C0 + sum_j (kt_j e^{b_last - b_j}) I~_j^T.
// Every exponent is <= 0 (g <= 0), so nothing overflows, whatever the decay.
// Forward launches: per chunk the state contribution (dC, gamma = e^{b_last});
// the scan over chunks in segments (the state entering every chunk); per chunk
// the output. Dense products run on the matrix cores (fp32 MFMA for fp32
// inputs; for bf16 inputs bf16 MFMA with fp32 accumulation, except in the
// backward's products that reach the decay gradient), the decay weights on
// the vector units in fp32, and the diagonal sub-blocks of the intra-chunk
// pairs on the matrix cores where the chunk's decay lets them be factored,
// else term by term on the vector units. With
// the gated entry points the kernels also form g from the KDA gate and rotate
// p1, p2 with RoPE as they load a chunk (and take both back in the gradient).
#include "kernels.h"
#include "lanes.h"

namespace rel {

namespace {

constexpr int kL = 64;      // tokens per chunk
constexpr int kLT = 512;    // threads per workgroup of the state kernels
constexpr int kLT2 = 512;   // threads per workgroup of the output kernel (8 waves)
constexpr int kTPRG = 16;   // threads per token row in the gradient kernel
constexpr int kLTG = kL * kTPRG;
constexpr int kRowsPerWave = 64 / kTPRG;

struct ChunkPos {
  int n, c, t0, len;  // head, chunk, first token, valid tokens
};

__device__ __forceinline__ ChunkPos chunk_pos(const LinearArgs& a) {
  ChunkPos p;
  p.c = blockIdx.x;
  p.n = blockIdx.y;
  p.t0 = p.c * kL;
  p.len = min(kL, a.T - p.t0);
  return p;
}

// Virtual heads: with SPLIT (the D = 128 backward cut into four problems of
// D channels) virtual head nv is sub-problem (A, E) = ((nv >> 1) & 1, nv & 1)
// of head nv >> 2; otherwise it is the head itself.
__host__ __device__ __forceinline__ int virtual_heads(const LinearArgs& a) { return a.B * a.H * (a.split ? 4 : 1); }

struct HeadRef {
  int n;         // head (b * H + h)
  int64_t hoff;  // element offset of its [T, D] slice in p1, p2, v, dY and their gradients
  int pa, pe;    // first relation channel (qt, kt, g) and first information channel (v, dY)
};

template <bool SPLIT, int D>
__device__ __forceinline__ HeadRef head_ref(const LinearArgs& a, int nv) {
  HeadRef r;
  r.n = SPLIT ? nv >> 2 : nv;
  r.pa = SPLIT ? ((nv >> 1) & 1) * D : 0;
  r.pe = SPLIT ? (nv & 1) * D : 0;
  r.hoff = (int64_t)(r.n / a.H) * a.sb + (int64_t)(r.n % a.H) * a.sh;
  return r;
}

// softplus(x) = max(x, 0) + ln(1 + e^-|x|): no overflow for any x; the
// logarithm's argument lies in (1, 2], where the hardware log2 is accurate
// (for x below about -17 the e^-|x| term is lost against 1 and softplus
// comes out 0: g then differs from the exact value by less than 1e-7 e^A_log).
__device__ __forceinline__ float softplus_f(float x) {
  return fmaxf(x, 0.0f) + kLn2 * __builtin_amdgcn_logf(1.0f + fast_exp2(-fabsf(x) * kLog2e));
}

// RoPE angle of position t, channel pair j: the table holds (cos, sin) of the
// angle at every chunk start (rows 0 .. nchunks - 1) and at every offset
// inside a chunk (rows nchunks .. nchunks + kL - 1); the angle at t is their
// sum (a few kB instead of a [T, rope_half] table read by every head).
__device__ __forceinline__ float2 rope_cs(const LinearArgs& a, int64_t t, int j) {
  const int h = a.rope_half;
  const float2 A = a.rope[(t / kL) * h + j];
  const float2 B = a.rope[(int64_t)(a.nchunks + t % kL) * h + j];
  return make_float2(A.x * B.x - A.y * B.y, A.y * B.x + A.x * B.y);
}

// The retention gate of eq. 15: g = -exp(A_log) softplus(r + dt_bias), with
// ea = exp(A_log) of the channel.
__device__ __forceinline__ float kda_gate(float r, float ea, float dtb) { return -ea * softplus_f(r + dtb); }

// K consecutive fp32 values from a 16-byte aligned address.
template <int K>
__device__ __forceinline__ void load_f32(const float* p, float (&x)[K]) {
  static_assert(K % 4 == 0, "whole 16-byte chunks");
#pragma unroll
  for (int i = 0; i < K; i += 4) {
    const float4 u = *reinterpret_cast<const float4*>(p + i);
    x[i] = u.x; x[i + 1] = u.y; x[i + 2] = u.z; x[i + 3] = u.w;
  }
}

// Column of element (r, c) of a row-major [kL][D] array stored with its
// 16-byte chunks XOR-swizzled by row: rows read together at one column (lanes
// over rows) then hit different banks, and four consecutive columns from a
// multiple of 4 stay one aligned 16-byte chunk.
template <int D>
__device__ __forceinline__ int swz(int r, int c) {
  return (((c >> 2) ^ (r & (D / 4 - 1))) << 2) | (c & 3);
}

// 16 bytes of a row (8 bf16 or 4 fp32 elements) as floats.
template <typename TI> struct Vec16;
template <> struct Vec16<bf16> {
  static __device__ __forceinline__ void load(const bf16* p, float (&x)[8]) {
    const uintx4 u = *reinterpret_cast<const uintx4*>(p);
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      x[2 * t] = bf16_lo(u[t]);
      x[2 * t + 1] = bf16_hi(u[t]);
    }
  }
};
template <> struct Vec16<float> {
  static __device__ __forceinline__ void load(const float* p, float (&x)[4]) {
    const float4 u = *reinterpret_cast<const float4*>(p);
    x[0] = u.x; x[1] = u.y; x[2] = u.z; x[3] = u.w;
  }
};

// 4 consecutive elements (8 bytes of bf16, 16 of fp32), for rows that start
// on 16-byte boundaries and offsets that are multiples of 4.
template <typename TI> struct Vec4;
template <> struct Vec4<bf16> {
  static __device__ __forceinline__ void load(const bf16* p, float (&x)[4]) {
    const uint2 u = *reinterpret_cast<const uint2*>(p);
    x[0] = bf16_lo(u.x); x[1] = bf16_hi(u.x); x[2] = bf16_lo(u.y); x[3] = bf16_hi(u.y);
  }
  static __device__ __forceinline__ void store(bf16* p, const float (&x)[4]) {
    typedef bf16 bf16x4 __attribute__((ext_vector_type(4)));
    bf16x4 o;
#pragma unroll
    for (int t = 0; t < 4; ++t) o[t] = (bf16)x[t];
    *reinterpret_cast<bf16x4*>(p) = o;
  }
};
template <> struct Vec4<float> {
  static __device__ __forceinline__ void load(const float* p, float (&x)[4]) {
    const float4 u = *reinterpret_cast<const float4*>(p);
    x[0] = u.x; x[1] = u.y; x[2] = u.z; x[3] = u.w;
  }
  static __device__ __forceinline__ void store(float* p, const float (&x)[4]) {
    *reinterpret_cast<float4*>(p) = make_float4(x[0], x[1], x[2], x[3]);
  }
};

// Loads the chunk into LDS as fp32 and forms qt = S ^p1, kt = S ^p2 (rows past
// the sequence are zero), v, optionally dY, and b = running sum of g (zero g
// past the end, so b stays at its last value). SWZ_VD stores v and dY
// swizzled (swz), SWZ_QKB qt, kt and b; qt may be null (not stored). One wave
// per row for the norms and S. With a.a_log the g read is the gate's
// pre-activation r and g = kda_gate(r); with a.rope qt and kt are rotated
// after S and the norms are formed (neither changes under the rotation).
// SPLIT: qt and kt are read as formed (fp32, from qn and kn, already rotated)
// and the chunk holds the sub-problem's halves of the channels.
template <typename TI, int D, int NT, bool SWZ_VD = false, bool WITH_DY = false, bool SWZ_QKB = false,
          bool SPLIT = false>
__device__ __forceinline__ void load_chunk(const LinearArgs& a, const ChunkPos& p, float (*qt)[D], float (*kt)[D],
                                           float (*vv)[D], float (*bb)[D], float* Srow,
                                           float (*dyl)[D] = nullptr) {
  static_assert(NT % 64 == 0 && kL % (NT / 64) == 0 && NT % D == 0, "rows and channels split evenly");
  constexpr int RPW = kL / (NT / 64);  // rows per wave
  constexpr int U = (D + 63) / 64;     // channels per lane
  constexpr int GW = SPLIT ? 2 * D : D;  // row length of g, qn and kn
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63;
  const HeadRef hr = head_ref<SPLIT, D>(a, p.n);
  const TI* P1 = (const TI*)a.p1 + hr.hoff;
  const TI* P2 = (const TI*)a.p2 + hr.hoff;
  const float* Q1 = SPLIT ? a.qn + (int64_t)hr.n * a.T * GW + hr.pa : nullptr;
  const float* Q2 = SPLIT ? a.kn + (int64_t)hr.n * a.T * GW + hr.pa : nullptr;
  const TI* V = (const TI*)a.v + hr.hoff + hr.pe;
  const TI* DY = WITH_DY ? (const TI*)a.dy + hr.hoff + hr.pe : nullptr;
  const float* G = a.g + (int64_t)hr.n * a.T * GW + hr.pa;
  auto col = [&](bool swzd, int row, int c) { return swzd ? swz<D>(row, c) : c; };
  if (a.vec16) {
    // 16 bytes per lane: LPR lanes hold a row, a wave RPI rows per step. Rows
    // past the sequence read its last row and then count as zero.
    constexpr int EPL = 16 / (int)sizeof(TI), LPR = D / EPL, RPI = 64 / LPR, NW = NT / 64;
    static_assert(LPR >= 2 && LPR <= 64 && EPL % 4 == 0, "a row is whole 16-byte chunks over a lane group");
    constexpr int STEPS = (kL + NW * RPI - 1) / (NW * RPI);
    const int cg = lane % LPR, c0 = cg * EPL;
    // the gate's parameters of this lane's channels: read with the rows (their
    // loads issued before anything waits), A_log turned into exp(A_log) at use
    const float* AL = a.a_log ? a.a_log + (int64_t)(hr.n % a.H) * GW + hr.pa + c0 : nullptr;
    const float* DB = a.a_log ? a.dt_bias + (int64_t)(hr.n % a.H) * GW + hr.pa + c0 : nullptr;
#pragma unroll
    for (int st = 0; st < STEPS; ++st) {
      const int r = st * NW * RPI + w * RPI + lane / LPR;
      if (st * NW * RPI + w * RPI < kL) {  // wave-uniform: the wave's rows are all in the chunk
        const int64_t row = (int64_t)min(p.t0 + r, a.T - 1);
        float x1[EPL], x2[EPL], vx[EPL], gx[EPL], dx[EPL];
        if constexpr (SPLIT) {
          load_f32<EPL>(Q1 + row * GW + c0, x1);
          load_f32<EPL>(Q2 + row * GW + c0, x2);
        } else {
          Vec16<TI>::load(P1 + row * a.st + c0, x1);
          Vec16<TI>::load(P2 + row * a.st + c0, x2);
        }
        Vec16<TI>::load(V + row * a.st + c0, vx);
        if constexpr (WITH_DY) Vec16<TI>::load(DY + row * a.st + c0, dx);
        load_f32<EPL>(G + row * GW + c0, gx);
        if (AL) {
          float al[EPL], dtb[EPL];
          load_f32<EPL>(AL, al);
          load_f32<EPL>(DB, dtb);
#pragma unroll
          for (int e = 0; e < EPL; ++e) gx[e] = kda_gate(gx[e], fast_exp2(al[e] * kLog2e), dtb[e]);
        }
        const bool ok = r < p.len;
        float s11 = 0.0f, s22 = 0.0f, s12 = 0.0f;
#pragma unroll
        for (int e = 0; e < EPL; ++e) {
          if (!ok) x1[e] = x2[e] = vx[e] = gx[e] = dx[e] = 0.0f;
          s11 += x1[e] * x1[e];
          s22 += x2[e] * x2[e];
          s12 += x1[e] * x2[e];
        }
        float S = 1.0f, i1 = 1.0f, i2 = 1.0f;  // SPLIT: qt and kt as read
        if constexpr (!SPLIT) {
          s11 = lane_group_sum<LPR>(s11);
          s22 = lane_group_sum<LPR>(s22);
          s12 = lane_group_sum<LPR>(s12);
          S = ok ? 1.0f / (1.0f + expf(-s12 * a.scale * a.inv_tau)) : 0.0f;
          i1 = ok && s11 > 0.0f ? S * rsqrtf(s11) : 0.0f;
          i2 = ok && s22 > 0.0f ? S * rsqrtf(s22) : 0.0f;
        }
#pragma unroll
        for (int e = 0; e < EPL; e += 4) {
          const int c = c0 + e;
          *reinterpret_cast<float4*>(&vv[r][col(SWZ_VD, r, c)]) = make_float4(vx[e], vx[e + 1], vx[e + 2], vx[e + 3]);
          *reinterpret_cast<float4*>(&bb[r][col(SWZ_QKB, r, c)]) = make_float4(gx[e], gx[e + 1], gx[e + 2], gx[e + 3]);
          if constexpr (WITH_DY)
            *reinterpret_cast<float4*>(&dyl[r][col(SWZ_VD, r, c)]) = make_float4(dx[e], dx[e + 1], dx[e + 2], dx[e + 3]);
          if (qt)
            *reinterpret_cast<float4*>(&qt[r][col(SWZ_QKB, r, c)]) =
                make_float4(x1[e] * i1, x1[e + 1] * i1, x1[e + 2] * i1, x1[e + 3] * i1);
          *reinterpret_cast<float4*>(&kt[r][col(SWZ_QKB, r, c)]) =
              make_float4(x2[e] * i2, x2[e + 1] * i2, x2[e + 2] * i2, x2[e + 3] * i2);
        }
        if (cg == 0 && Srow) Srow[r] = S;
      }
    }
  } else {
  // rows in batches whose loads are issued together: the loads are
  // unconditional (rows past the sequence read its last row, then count as
  // zero) so that the compiler can hoist them over the reductions
  constexpr int BATCH = RPW < 8 / U ? RPW : 8 / U;
  static_assert(RPW % BATCH == 0, "whole batches");
  for (int k0 = 0; k0 < RPW; k0 += BATCH) {
    float x1[BATCH][U], x2[BATCH][U], vx[BATCH][U], gx[BATCH][U], dx[BATCH][U];
#pragma unroll
    for (int kb = 0; kb < BATCH; ++kb) {
      const int r = w + (k0 + kb) * (NT / 64);
      const int64_t row = (int64_t)min(p.t0 + r, a.T - 1);
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int d = min(lane + 64 * u, D - 1);
        x1[kb][u] = SPLIT ? Q1[row * GW + d] : Elem<TI>::load(P1 + row * a.st + d);
        x2[kb][u] = SPLIT ? Q2[row * GW + d] : Elem<TI>::load(P2 + row * a.st + d);
        vx[kb][u] = Elem<TI>::load(V + row * a.st + d);
        gx[kb][u] = G[row * GW + d];
        if (a.a_log) {
          const int64_t pc = (int64_t)(hr.n % a.H) * GW + hr.pa + d;
          gx[kb][u] = kda_gate(gx[kb][u], fast_exp2(a.a_log[pc] * kLog2e), a.dt_bias[pc]);
        }
        dx[kb][u] = WITH_DY ? Elem<TI>::load(DY + row * a.st + d) : 0.0f;
      }
    }
#pragma unroll
    for (int kb = 0; kb < BATCH; ++kb) {
      const int r = w + (k0 + kb) * (NT / 64);
      const bool ok = r < p.len;
      float s11 = 0.0f, s22 = 0.0f, s12 = 0.0f;
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int d = lane + 64 * u;
        if (!ok || d >= D) x1[kb][u] = x2[kb][u] = vx[kb][u] = gx[kb][u] = dx[kb][u] = 0.0f;
        if (d < D) {
          const int ds = SWZ_VD ? swz<D>(r, d) : d;
          vv[r][ds] = vx[kb][u];
          bb[r][SWZ_QKB ? swz<D>(r, d) : d] = gx[kb][u];
          if constexpr (WITH_DY) dyl[r][ds] = dx[kb][u];
        }
        s11 += x1[kb][u] * x1[kb][u];
        s22 += x2[kb][u] * x2[kb][u];
        s12 += x1[kb][u] * x2[kb][u];
      }
      float S = 1.0f, i1 = 1.0f, i2 = 1.0f;  // SPLIT: qt and kt as read
      if constexpr (!SPLIT) {
        s11 = lane_group_sum<64>(s11);
        s22 = lane_group_sum<64>(s22);
        s12 = lane_group_sum<64>(s12);
        S = ok ? 1.0f / (1.0f + expf(-s12 * a.scale * a.inv_tau)) : 0.0f;
        i1 = ok && s11 > 0.0f ? S * rsqrtf(s11) : 0.0f;
        i2 = ok && s22 > 0.0f ? S * rsqrtf(s22) : 0.0f;
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int d = lane + 64 * u;
        if (d < D) {
          const int dq = SWZ_QKB ? swz<D>(r, d) : d;
          if (qt) qt[r][dq] = x1[kb][u] * i1;
          kt[r][dq] = x2[kb][u] * i2;
        }
      }
      if (lane == 0 && Srow) Srow[r] = S;
    }
  }
  }
  __syncthreads();
  if (!SPLIT && a.rope) {
    // RoPE on the chunk's qt and kt (scaled, not yet rotated): pairs (j, j + h)
    // of every row; S and the norms above are the same before and after
    const int h = a.rope_half;
    for (int i = tid; i < kL * h; i += NT) {
      const int r = i / h, j = i % h;
      const float2 cs = rope_cs(a, min(p.t0 + r, a.T - 1), j);
      const int c1 = col(SWZ_QKB, r, j), c2 = col(SWZ_QKB, r, j + h);
      if (qt) {
        const float x = qt[r][c1], y = qt[r][c2];
        qt[r][c1] = x * cs.x - y * cs.y;
        qt[r][c2] = x * cs.y + y * cs.x;
      }
      const float x = kt[r][c1], y = kt[r][c2];
      kt[r][c1] = x * cs.x - y * cs.y;
      kt[r][c2] = x * cs.y + y * cs.x;
    }
  }
  // running sum of g down the chunk: thread (channel, segment of SR rows) sums
  // its segment in place, then adds the totals of the segments above it
  constexpr int NSEG = NT / D, SR = kL / NSEG;
  const int d = tid % D, sg = tid / D;
  auto bcol = [&](int row) { return col(SWZ_QKB, row, d); };
  float x[SR];
  float acc = 0.0f;
#pragma unroll
  for (int i = 0; i < SR; ++i) x[i] = bb[sg * SR + i][bcol(sg * SR + i)];
#pragma unroll
  for (int i = 0; i < SR; ++i) x[i] = acc += x[i];
#pragma unroll
  for (int i = 0; i < SR; ++i) bb[sg * SR + i][bcol(sg * SR + i)] = x[i];
  __syncthreads();
  float off = 0.0f;  // the totals of the segments above, added in order (reads issued together)
#pragma unroll
  for (int u = 0; u < NSEG - 1; ++u) {
    const float t = bb[u * SR + SR - 1][bcol(u * SR + SR - 1)];
    if (u < sg) off += t;
  }
  __syncthreads();  // every segment total read
  if (sg > 0) {
#pragma unroll
    for (int i = 0; i < SR; ++i) bb[sg * SR + i][bcol(sg * SR + i)] = x[i] + off;
  }
  __syncthreads();
}

// Matrix-core operands. With fp32 inputs every product runs on fp32 MFMA
// steps. With bf16 inputs (BF) the operands, formed in fp32, are rounded to
// bf16 and the products run on bf16 MFMA steps with fp32 accumulation, eight
// fp32 steps' worth of contraction per instruction. A lane supplies the values
// of its row of the left operand and of its column of the right operand at the
// same contraction indices; which indices go to which lane and slot does not
// matter to the sum, so each lane keeps the index range it has on the fp32 path.
// The backward keeps fp32 accuracy in every product that reaches the
// gradient of the decay (dq, dk, and the states C0 and G): fp32 steps, or,
// where one operand is a bf16 input, bf16 steps with the other split in three
// bf16 parts (exact products). That gradient is a small difference of large
// terms (the scores depend on b only through b_t - b_j, so the intra-chunk
// parts of qt dq and kt dk cancel over a chunk), and operands rounded to bf16
// leave a residual of their rounding in it that adds up coherently over the
// tokens in dA_log.
template <typename TI> constexpr bool kBF = sizeof(TI) == 2;

template <int N>
__device__ __forceinline__ void pack_bf16(const float* x, __bf16 __attribute__((ext_vector_type(N))) & o) {
#pragma unroll
  for (int t = 0; t < N; ++t) o[t] = (bf16)x[t];
}
__device__ __forceinline__ floatx4 mfma16b(const float (&a)[8], const float (&b)[8], const floatx4& c) {
  bf16x8 x, y;
  pack_bf16<8>(a, x);
  pack_bf16<8>(b, y);
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(x, y, c, 0, 0, 0);
}
__device__ __forceinline__ floatx4 mfma16b4(const float (&a)[4], const float (&b)[4], const floatx4& c) {
  bf16x4 x, y;
  pack_bf16<4>(a, x);
  pack_bf16<4>(b, y);
  return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(shortx4, x), __builtin_bit_cast(shortx4, y), c,
                                                   0, 0, 0);
}
__device__ __forceinline__ floatx16 mfma32b(const float (&a)[8], const float (&b)[8], const floatx16& c) {
  bf16x8 x, y;
  pack_bf16<8>(a, x);
  pack_bf16<8>(b, y);
  return mfma32(x, y, c);
}

// One 32 x 32 block (rows ab.., columns eb..) of X^T Y, the contraction over
// the kL rows of the chunk (X, Y plain [kL][D] arrays), on the matrix cores
// (lane group g takes the rows of parity g: 32x32x2 fp32 steps, or 32x32x16
// bf16 steps of eight such rows with BF).
template <int D, bool BF = false>
__device__ __forceinline__ floatx16 gram_block(const float (*X)[D], const float (*Y)[D], int ab, int eb) {
  const int lane = threadIdx.x & 63, ln = lane & 31, lg = lane >> 5;
  floatx16 acc;
#pragma unroll
  for (int v = 0; v < 16; ++v) acc[v] = 0.0f;
  if constexpr (BF) {
#pragma unroll
    for (int s = 0; s < kL / 16; ++s) {
      float x[8], y[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int r = 16 * s + 2 * u + lg;
        x[u] = X[r][ab + ln];
        y[u] = Y[r][eb + ln];
      }
      acc = mfma32b(x, y, acc);
    }
  } else {
#pragma unroll 8
    for (int s2 = 0; s2 < kL / 2; ++s2) {
      const int r = 2 * s2 + lg;
      acc = mfma32f(X[r][ab + ln], Y[r][eb + ln], acc);
    }
  }
  return acc;
}

// gram_block for a right operand Y whose values are bf16 numbers (the bf16
// inputs, held in fp32): X is split as hi + mid + lo, three bf16 numbers that
// carry its 24 significant bits, so the three 32x32x16 bf16 steps per 16 rows
// give exact products with fp32 accumulation, as the fp32 steps would.
template <int D>
__device__ __forceinline__ floatx16 gram_block_split3(const float (*X)[D], const float (*Y)[D], int ab, int eb) {
  const int lane = threadIdx.x & 63, ln = lane & 31, lg = lane >> 5;
  floatx16 acc;
#pragma unroll
  for (int v = 0; v < 16; ++v) acc[v] = 0.0f;
#pragma unroll 1
  for (int s = 0; s < kL / 16; ++s) {
    bf16x8 hv, mv, lv, yv;
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int r = 16 * s + 2 * u + lg;
      const float x = X[r][ab + ln];
      const bf16 h = (bf16)x;
      const float r1 = x - (float)h;
      const bf16 m = (bf16)r1;
      hv[u] = h;
      mv[u] = m;
      lv[u] = (bf16)(r1 - (float)m);
      yv[u] = (bf16)Y[r][eb + ln];
    }
    acc = mfma32(hv, yv, acc);
    acc = mfma32(mv, yv, acc);
    acc = mfma32(lv, yv, acc);
  }
  return acc;
}

// Stores a 32 x 32 accumulator block at (ab, eb) of a dense D x D matrix.
template <int D>
__device__ __forceinline__ void store_block(float* out, const floatx16& acc, int ab, int eb) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int v = 0; v < 16; ++v) out[(ab + acc_row(v, lane >> 5)) * D + eb + (lane & 31)] = acc[v];
}

// Per chunk: dC[a][e] = sum_j kt_{j,a} e^{b_last,a - b_j,a} v_{j,e}, gamma_a = e^{b_last,a}.
template <typename TI, int D>
__global__ __launch_bounds__(kLT) void linear_state_kernel(LinearArgs a) {
  __shared__ float kt[kL][D], vv[kL][D], bb[kL][D];  // qt is not needed here
  const ChunkPos p = chunk_pos(a);
  load_chunk<TI, D, kLT>(a, p, nullptr, kt, vv, bb, nullptr);
  const int tid = threadIdx.x;
  // kt <- kt e^{b_last - b}
  for (int i = tid; i < kL * D; i += kLT) {
    const int r = i / D, d = i % D;
    kt[r][d] *= fast_exp2((bb[kL - 1][d] - bb[r][d]) * kLog2e);
  }
  __syncthreads();
  const int64_t base = ((int64_t)p.n * a.nchunks + p.c);
  if (tid < D) a.gamma[base * D + tid] = fast_exp2(bb[kL - 1][tid] * kLog2e);
  // dC on the matrix cores, 32 x 32 blocks, wave w takes blocks w, w + 4, ...
  constexpr int NBE = D / 32;
  for (int bk = __builtin_amdgcn_readfirstlane(tid >> 6); bk < NBE * NBE; bk += kLT / 64) {
    const int ab = 32 * (bk / NBE), eb = 32 * (bk % NBE);
    store_block<D>(a.dstate + base * D * D, gram_block<D, kBF<TI>>(kt, vv, ab, eb), ab, eb);
  }
}

// The state scans. Per head and state element, over the chunks c:
//   forward   C_c = gamma_c C_{c-1} + dstate_c   (cprev_c = C_{c-1}, C_{-1} = 0)
//   reverse   G_c = gamma_c G_{c+1} + pstate_c   (gout_c = G_{c+1}, G_{nchunks} = 0)
// with gamma_c per state row. The chunks are cut into segments of kSegChunks so
// that the grid is wide enough to keep HBM busy: linear_seg_kernel reduces each
// segment to its retention product and its result from a zero start;
// linear_seg_apply_kernel folds the summaries of the segments before (forward)
// or after (reverse) its own into the state entering it, then walks its chunks.
constexpr int kSegChunks = 16;

__device__ __forceinline__ int seg_begin(int s) { return s * kSegChunks; }
__device__ __forceinline__ int seg_end(const LinearArgs& a, int s) { return min(a.nchunks, (s + 1) * kSegChunks); }

// The retention row and one state element of every chunk of segment [c0, c1)
// (in reverse order with REV), all loads issued before any is used: the walk
// over the chunks is a dependent chain, and loading inside it left one
// round trip per step. Slots past the segment repeat its last (first) chunk
// and are not used.
template <bool REV>
__device__ __forceinline__ void load_segment(const float* gamma, const float* st, int64_t hb, int c0, int c1, int D,
                                             int ar, int64_t idx, float (&gv)[kSegChunks], float (&sv)[kSegChunks]) {
#pragma unroll
  for (int k = 0; k < kSegChunks; ++k) {
    const int c = REV ? max(c1 - 1 - k, c0) : min(c0 + k, c1 - 1);
    gv[k] = gamma[(hb + c) * D + ar];
    sv[k] = st[(hb + c) * D * D + idx];
  }
}

__global__ __launch_bounds__(256) void linear_seg_kernel(LinearArgs a, int reverse) {
  const int D = a.D;
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (int64_t)D * D) return;
  const int s = blockIdx.y, n = blockIdx.z;
  const int ar = (int)(idx / D);
  const int c0 = seg_begin(s), c1 = seg_end(a, s);
  const int64_t hb = (int64_t)n * a.nchunks;
  float gv[kSegChunks], sv[kSegChunks];
  load_segment<false>(a.gamma, a.dstate, hb, c0, c1, D, ar, idx, gv, sv);
  float C = 0.0f, prod = 1.0f;
#pragma unroll
  for (int k = 0; k < kSegChunks; ++k) {
    if (c0 + k < c1) {
      C = gv[k] * C + sv[k];
      prod *= gv[k];
    }
  }
  const int64_t sb = (int64_t)n * a.nseg + s;
  a.segc[sb * D * D + idx] = C;
  if (idx % D == 0) a.segg[sb * D + ar] = prod;
  if (reverse) {
    load_segment<true>(a.gamma, a.pstate, hb, c0, c1, D, ar, idx, gv, sv);
    float G = 0.0f;
#pragma unroll
    for (int k = 0; k < kSegChunks; ++k)
      if (c1 - 1 - k >= c0) G = gv[k] * G + sv[k];
    a.segp[sb * D * D + idx] = G;
  }
}

__global__ __launch_bounds__(256) void linear_seg_apply_kernel(LinearArgs a, int reverse) {
  const int D = a.D;
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (int64_t)D * D) return;
  const int s = blockIdx.y, n = blockIdx.z;
  const int ar = (int)(idx / D);
  const int c0 = seg_begin(s), c1 = seg_end(a, s);
  const int64_t hb = (int64_t)n * a.nchunks, sh = (int64_t)n * a.nseg;
  float gv[kSegChunks], sv[kSegChunks];
  load_segment<false>(a.gamma, a.dstate, hb, c0, c1, D, ar, idx, gv, sv);
  float C = 0.0f;
#pragma unroll 4
  for (int u = 0; u < s; ++u) C = a.segg[(sh + u) * D + ar] * C + a.segc[(sh + u) * D * D + idx];
#pragma unroll
  for (int k = 0; k < kSegChunks; ++k) {
    if (c0 + k < c1) {
      a.cprev[(hb + c0 + k) * D * D + idx] = C;
      C = gv[k] * C + sv[k];
    }
  }
  if (a.state_out && s == a.nseg - 1) a.state_out[(int64_t)n * D * D + idx] = C;
  if (reverse) {
    load_segment<true>(a.gamma, a.pstate, hb, c0, c1, D, ar, idx, gv, sv);
    float G = 0.0f;
#pragma unroll 4
    for (int u = a.nseg - 1; u > s; --u) G = a.segg[(sh + u) * D + ar] * G + a.segp[(sh + u) * D * D + idx];
#pragma unroll
    for (int k = 0; k < kSegChunks; ++k) {
      if (c1 - 1 - k >= c0) {
        a.gout[(hb + c1 - 1 - k) * D * D + idx] = G;
        G = gv[k] * G + sv[k];
      }
    }
  }
}

hipError_t launch_state_scan(const LinearArgs& a, int reverse, hipStream_t stream) {
  const dim3 grid((unsigned)((a.D * a.D + 255) / 256), (unsigned)a.nseg, (unsigned)virtual_heads(a));
  if (a.nseg > 1) {
    hipLaunchKernelGGL(linear_seg_kernel, grid, dim3(256), 0, stream, a, reverse);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(linear_seg_apply_kernel, grid, dim3(256), 0, stream, a, reverse);
  return hipGetLastError();
}

// acc += one 32 x 32 block (rows rb.., columns cb..) of a product X B whose
// contraction runs over the K columns of X, on the matrix cores (32x32x2 fp32
// steps, or 32x32x16 bf16 steps with BF). X is a swizzled (swz) row-major
// [kL][K] array; B(k, j) gives the column operand. Lane group g takes the
// contraction indices K/2 g .. K/2 g + K/2 - 1 in order, four per 16-byte read
// of its row of X.
template <int K, bool BF = false, typename ColOp>
__device__ __forceinline__ floatx16 block_product(const float (*X)[K], int rb, int cb, floatx16 acc, ColOp B) {
  constexpr int KH = K / 2;
  const int lane = threadIdx.x & 63, ln = lane & 31, lg = lane >> 5;
  const int xr = rb + ln;
  if constexpr (BF) {
    static_assert(KH % 8 == 0, "whole bf16 steps");
#pragma unroll 2
    for (int s0 = 0; s0 < KH; s0 += 8) {
      const int kk = KH * lg + s0;
      const floatx4 x0 = *reinterpret_cast<const floatx4*>(&X[xr][swz<K>(xr, kk)]);
      const floatx4 x1 = *reinterpret_cast<const floatx4*>(&X[xr][swz<K>(xr, kk + 4)]);
      float xa[8], xb[8];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        xa[u] = x0[u];
        xa[4 + u] = x1[u];
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) xb[u] = B(kk + u, cb + ln);
      acc = mfma32b(xa, xb, acc);
    }
  } else {
#pragma unroll 2
    for (int s0 = 0; s0 < KH; s0 += 4) {
      const int kk = KH * lg + s0;
      const floatx4 xa = *reinterpret_cast<const floatx4*>(&X[xr][swz<K>(xr, kk)]);
#pragma unroll
      for (int u = 0; u < 4; ++u) acc = mfma32f(xa[u], B(kk + u, cb + ln), acc);
    }
  }
  return acc;
}

// acc += one 32 x 32 block of X B as block_product, for a row operand X whose
// values are bf16 numbers (the bf16 inputs, held in fp32) and any fp32 column
// operand: B is split as b = hi + mid + lo, three bf16 numbers that carry its
// 24 significant bits, and the block takes three 32x32x16 bf16 steps per 16
// contraction indices, with the products exact and fp32 accumulation, where
// fp32 steps take eight.
template <int K, typename ColOp>
__device__ __forceinline__ floatx16 block_product_split3(const float (*X)[K], int rb, int cb, floatx16 acc, ColOp B) {
  constexpr int KH = K / 2;
  static_assert(KH % 8 == 0, "whole bf16 steps");
  const int lane = threadIdx.x & 63, ln = lane & 31, lg = lane >> 5;
  const int xr = rb + ln;
#pragma unroll 1
  for (int s0 = 0; s0 < KH; s0 += 8) {
    const int kk = KH * lg + s0;
    const floatx4 x0 = *reinterpret_cast<const floatx4*>(&X[xr][swz<K>(xr, kk)]);
    const floatx4 x1 = *reinterpret_cast<const floatx4*>(&X[xr][swz<K>(xr, kk + 4)]);
    bf16x8 xv, hv, mv, lv;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      xv[u] = (bf16)x0[u];
      xv[4 + u] = (bf16)x1[u];
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const float b = B(kk + u, cb + ln);
      const bf16 h = (bf16)b;
      const float r1 = b - (float)h;
      const bf16 m = (bf16)r1;
      hv[u] = h;
      mv[u] = m;
      lv[u] = (bf16)(r1 - (float)m);
    }
    acc = mfma32(xv, hv, acc);
    acc = mfma32(xv, mv, acc);
    acc = mfma32(xv, lv, acc);
  }
  return acc;
}

__device__ __forceinline__ floatx16 zero16() {
  floatx16 z;
#pragma unroll
  for (int v = 0; v < 16; ++v) z[v] = 0.0f;
  return z;
}

__device__ __forceinline__ floatx4 mfma16f(float a, float b, const floatx4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// Chunk c (4 channels) of row r of a swizzled (swz) [kL][D] array.
template <int D>
__device__ __forceinline__ floatx4 ld4(const float (*X)[D], int r, int c) {
  return *reinterpret_cast<const floatx4*>(&X[r][(c ^ (r & (D / 4 - 1))) << 2]);
}

// Largest decay (log2 units) over a 16-row block of the chunk for which the
// diagonal blocks are factored at a reference row like the blocks below: the
// factors then lie in [2^-kFactLim, 2^kFactLim], far inside the fp32 range.
constexpr float kFactLim = 64.0f;

// True when on every channel the decay across each 16-row block, from the
// row before the block (the first row for the first block) to its last row,
// is at most 2^kFactLim (false for any NaN). Every wave checks all of them
// itself (no barrier, no LDS of its own), so the result is the same in every
// wave of the workgroup.
template <int D>
__device__ __forceinline__ bool diag_factorable(const float (*bb)[D]) {
  bool over = false;
  for (int i = threadIdx.x & 63; i < 4 * D; i += 64) {
    const int blk = i / D, c = i % D;
    const int r0 = blk ? 16 * blk - 1 : 0, r1 = 16 * blk + 15;
    over |= !((bb[r0][swz<D>(r0, c)] - bb[r1][swz<D>(r1, c)]) * kLog2e <= kFactLim);
  }
  return !wave_any(over);
}

// Intra-chunk scores A[t][j] = sum_a qt_{t,a} kt_{j,a} e^{b_{t,a} - b_{j,a}}
// (j < t) into the swizzled A, in 16 x 16 sub-blocks. qt, kt and b are
// swizzled. Below the diagonal, block (tb, jb) factors the decay at the last
// row rf of key block jb: e^{b_t - b_j} = e^{b_t - b_rf} e^{b_rf - b_j}, both
// factors <= 1 (b does not increase down the chunk), so the block is a plain
// product of qt e^{b - b_rf} and kt e^{b_rf - b} on the matrix cores
// (16x16x4 fp32 steps, the operands formed in registers). A diagonal block is
// the same product factored at its first row when FACT (diag_factorable: the
// key factor e^{b_rf - b_j} >= 1 stays below 2^kFactLim), with the pairs
// j >= t set to zero; otherwise it is summed term by term on the vector units.
// Waves 0-3 of the workgroup: diagonal block w; waves 4-7: blocks w - 4 and w
// (of the six below the diagonal). With TRANS the scores go to A as A^T (A[j][t]).
template <int D, bool BF = false>
__device__ __forceinline__ floatx4 scaled_block(const float (*qt)[D], const float (*kt)[D], const float (*bb)[D],
                                                int tb, int jb, int rf) {
  constexpr int CH = D / 4;
  const int lane = threadIdx.x & 63, i = lane & 15, g = lane >> 4;
  const int tr = 16 * tb + i, jr = 16 * jb + i;
  floatx4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
  // the scaled operands of channel chunk c (4 channels)
  auto operands = [&](int c, float* qa, float* kb) {
    const floatx4 q4 = ld4<D>(qt, tr, c), bt4 = ld4<D>(bb, tr, c), br4 = ld4<D>(bb, rf, c);
    const floatx4 k4 = ld4<D>(kt, jr, c), bj4 = ld4<D>(bb, jr, c);
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      qa[u] = q4[u] * fast_exp2((bt4[u] - br4[u]) * kLog2e);
      kb[u] = k4[u] * fast_exp2((br4[u] - bj4[u]) * kLog2e);
    }
  };
  // lane group g takes the channel chunks CH/4 g .. CH/4 g + CH/4 - 1
  if constexpr (BF) {
    static_assert(CH % 8 == 0, "two chunks per bf16 step");
#pragma unroll 2
    for (int c0 = 0; c0 < CH / 4; c0 += 2) {
      float qa[8], kb[8];
      operands((CH / 4) * g + c0, qa, kb);
      operands((CH / 4) * g + c0 + 1, qa + 4, kb + 4);
      acc = mfma16b(qa, kb, acc);
    }
  } else {
#pragma unroll 2
    for (int c0 = 0; c0 < CH / 4; ++c0) {
      float qa[4], kb[4];
      operands((CH / 4) * g + c0, qa, kb);
#pragma unroll
      for (int u = 0; u < 4; ++u) acc = mfma16f(qa[u], kb[u], acc);
    }
  }
  return acc;
}

template <int D, bool TRANS = false, bool BF = false>
__device__ __forceinline__ void chunk_scores(const float (*qt)[D], const float (*kt)[D], const float (*bb)[D],
                                             float (*A)[kL], bool fact) {
  constexpr int SB = 16, NSB = kL / SB, CH = D / 4;
  static_assert(NSB == 4, "four diagonal blocks, six below");
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  auto put = [&](int t, int j, float x) {
    if (TRANS) A[j][swz<kL>(j, t)] = x;
    else A[t][swz<kL>(t, j)] = x;
  };
  if (w < NSB && fact) {
    const int i = lane & 15, g = lane >> 4;
    const floatx4 acc = scaled_block<D, BF>(qt, kt, bb, w, w, SB * w);
#pragma unroll
    for (int v = 0; v < 4; ++v) put(SB * w + 4 * g + v, SB * w + i, i < 4 * g + v ? acc[v] : 0.0f);
    for (int jb = w + 1; jb < NSB; ++jb) {  // the blocks above the diagonal in the row band are zero
#pragma unroll
      for (int v = 0; v < 4; ++v) put(SB * w + 4 * g + v, SB * jb + i, 0.0f);
    }
  } else if (w < NSB) {
    // the block's 120 pairs j < t, two per lane (slot s: pair lane + 64 s in
    // row-major order); the rest of the block is zero
    const int base = SB * w, t = base + (lane >> 2), jq = lane & 3;
#pragma unroll
    for (int m = 0; m < 4; ++m) put(t, base + jq + 4 * m, 0.0f);  // same wave: the pairs land after
    int tt[2], jj[2];
    bool live[2];
#pragma unroll
    for (int sl = 0; sl < 2; ++sl) {
      const int idx = lane + 64 * sl;
      live[sl] = idx < SB * (SB - 1) / 2;
      int r = 1, rem = live[sl] ? idx : 0;
      while (rem >= r) {  // row r (of the block) holds r pairs
        rem -= r;
        ++r;
      }
      tt[sl] = base + r;
      jj[sl] = base + rem;
    }
    float acc[2] = {0.0f, 0.0f};
#pragma unroll 2
    for (int c = 0; c < CH; ++c) {
#pragma unroll
      for (int sl = 0; sl < 2; ++sl) {
        const floatx4 q4 = ld4<D>(qt, tt[sl], c), bt4 = ld4<D>(bb, tt[sl], c);
        const floatx4 k4 = ld4<D>(kt, jj[sl], c), bj4 = ld4<D>(bb, jj[sl], c);
#pragma unroll
        for (int u = 0; u < 4; ++u)
          acc[sl] = __builtin_fmaf(q4[u] * k4[u], fast_exp2((bt4[u] - bj4[u]) * kLog2e), acc[sl]);
      }
    }
#pragma unroll
    for (int sl = 0; sl < 2; ++sl)
      if (live[sl]) put(tt[sl], jj[sl], acc[sl]);
    // the blocks above the diagonal block's row band are zero
    for (int jb = w + 1; jb < NSB; ++jb) {
#pragma unroll
      for (int m = 0; m < 4; ++m) {
        put(t, SB * jb + jq + 4 * m, 0.0f);
      }
    }
  } else if (w < 2 * NSB) {
    const int i = lane & 15, g = lane >> 4;
    for (int bi = w - NSB; bi < NSB * (NSB - 1) / 2; bi += NSB) {
      // blocks below the diagonal, bi = 0..5: (1,0) (2,0) (3,0) (2,1) (3,1) (3,2)
      const int jb = bi < 3 ? 0 : bi < 5 ? 1 : 2;
      const int tb = jb + 1 + (bi < 3 ? bi : bi < 5 ? bi - 3 : 0);
      const floatx4 acc = scaled_block<D, BF>(qt, kt, bb, tb, jb, SB * jb + SB - 1);
      // register v of lane (i, g): row 4 g + v, column i of the block
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        put(SB * tb + 4 * g + v, SB * jb + i, acc[v]);
      }
    }
  }
}

// Per chunk: Y_t = v_t + intra + inter (see the top of the file). The scores
// A (j < t) come from chunk_scores; then Y = v + A V + Qe C0 (Qe = qt e^{b})
// is two dense products on the matrix cores, 32 x 32 output blocks per wave.
template <typename TI, int D>
__global__ __launch_bounds__(kLT2) void linear_out_kernel(LinearArgs a) {
  static_assert(2 * kL * D >= D * D, "the state entering the chunk is staged over qt and bb");
  __shared__ float qb[2][kL][D];  // qt, bb (swizzled); then the state entering the chunk
  __shared__ float kt[kL][D];     // kt; then Qe (both swizzled)
  __shared__ float vv[kL][D];
  __shared__ float A[kL][kL];     // scores, swizzled; then a partial output
  float (*qt)[D] = qb[0];
  float (*bb)[D] = qb[1];
  const ChunkPos p = chunk_pos(a);
  const int tid = threadIdx.x;
  const float* C0 = a.cprev + ((int64_t)p.n * a.nchunks + p.c) * D * D;
  constexpr int NC0 = D * D / kLT2;  // elements of C0 per thread
  constexpr bool PREFETCH = NC0 <= 32;  // 32 registers at D = 128 (two waves per SIMD: LDS-bound)
  float c0r[PREFETCH ? NC0 : 1];
  if constexpr (PREFETCH) {
#pragma unroll
    for (int k = 0; k < NC0; ++k) c0r[k] = C0[tid + k * kLT2];
  }
  load_chunk<TI, D, kLT2, false, false, true>(a, p, qt, kt, vv, bb, nullptr);
  chunk_scores<D, false, kBF<TI>>(qt, kt, bb, A, diag_factorable<D>(bb));
  __syncthreads();
  // Qe = qt e^{b} (the inter read's query), over kt; all three swizzled alike
  for (int i = tid; i < kL * D; i += kLT2) {
    const int r = i / D, c = i % D;
    kt[r][c] = qt[r][c] * fast_exp2(bb[r][c] * kLog2e);
  }
  __syncthreads();
  // the state entering the chunk, over qt and bb
  float* C0s = &qb[0][0][0];
  if constexpr (PREFETCH) {
#pragma unroll
    for (int k = 0; k < NC0; ++k) C0s[tid + k * kLT2] = c0r[k];
  } else {
    for (int i = tid; i < D * D; i += kLT2) C0s[i] = C0[i];
  }
  __syncthreads();
  // wave -> output block; with few blocks, waves NB .. 2 NB - 1 take the
  // inter product of block w - NB and hand it over through LDS
  constexpr int NBC = D / 32, NB = (kL / 32) * NBC, NW = kLT2 / 64;
  constexpr bool SPLIT = 2 * NB <= NW;
  static_assert(NB <= NW, "one block per wave");
  const int w = tid >> 6, lane = tid & 63;
  const int blk = w % NB, part = SPLIT ? w / NB : 0;
  const int rb = 32 * (blk / NBC), cb = 32 * (blk % NBC);
  const bool busy = w < (SPLIT ? 2 * NB : NB);
  floatx16 acc = zero16();
  if (busy && part == 0) acc = block_product<kL, kBF<TI>>(A, rb, cb, acc, [&](int k, int j) { return vv[k][j]; });
  if (busy && (!SPLIT || part == 1))
    acc = block_product<D, kBF<TI>>(kt, rb, cb, acc, [&](int k, int j) { return C0s[k * D + j]; });
  float* Ap = &A[0][0];
  if constexpr (SPLIT) {
    __syncthreads();  // every operand of A read
    if (busy && part == 1) {
#pragma unroll
      for (int v = 0; v < 16; ++v) Ap[(rb + acc_row(v, lane >> 5)) * D + cb + (lane & 31)] = acc[v];
    }
    __syncthreads();
  }
  if (busy && part == 0) {
    const int b = p.n / a.H, h = p.n % a.H;
    TI* Y = (TI*)a.out + (int64_t)b * a.sb + (int64_t)h * a.sh;
    const int col = cb + (lane & 31);
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int row = rb + acc_row(v, lane >> 5);
      float y = acc[v] + vv[row][col];
      if constexpr (SPLIT) y += Ap[row * D + col];
      if (row < p.len) Elem<TI>::store(Y + (int64_t)(p.t0 + row) * a.st + col, y);
    }
  }
}

// ---------------------------------------------------------------------------
// Backward. With Qe = qt e^{b}, Kd = kt e^{b_last - b} and the chunk's state
// C0 (entering) and G (gradient of the state leaving the chunk):
//   inter read   E = Qe C0:            dQe = dY C0^T,  P = Qe^T dY (to the scan)
//   state write  C1 = gamma C0 + Kd^T v: dKd = v G^T, dv += Kd G, dgamma_a = sum_e G C0
//   intra        A_tj = sum_a qt_ta kt_ja e^{b_ta - b_ja} (j < t):
//                dA_tj = dY_t . v_j, dv_j += sum_t A_tj dY_t,
//                dqt_t += sum_j dA_tj kt_j e^{..}, dkt_j += sum_t dA_tj qt_t e^{..}
//   b (running sum of g): db_t = qt dqt_intra - kt dkt_intra + dQe Qe - dKd Kd,
//                db_last += sum_j dKd Kd + dgamma gamma; dg = reverse running sum of db
//   then qt = S ^p1, kt = S ^p2 through S and the normalisation.
// The scan runs forward for C0 and backward for G, both per state entry.
// ---------------------------------------------------------------------------

// Per chunk: the state contribution (as in the forward pass) and P = Qe^T dY.
template <typename TI, int D, bool SPLIT = false>
__global__ __launch_bounds__(kLT) void linear_bstate_kernel(LinearArgs a) {
  __shared__ float qt[kL][D], kt[kL][D], vv[kL][D], bb[kL][D], dy[kL][D];
  const ChunkPos p = chunk_pos(a);
  load_chunk<TI, D, kLT, false, true, false, SPLIT>(a, p, qt, kt, vv, bb, nullptr, dy);
  const int tid = threadIdx.x;
  for (int i = tid; i < kL * D; i += kLT) {
    const int r = i / D, d = i % D;
    kt[r][d] *= fast_exp2((bb[kL - 1][d] - bb[r][d]) * kLog2e);
    qt[r][d] *= fast_exp2(bb[r][d] * kLog2e);
  }
  __syncthreads();
  const int64_t base = ((int64_t)p.n * a.nchunks + p.c);
  if (tid < D) a.gamma[base * D + tid] = fast_exp2(bb[kL - 1][tid] * kLog2e);
  // dC = Kd^T v and P = Qe^T dY on the matrix cores, 32 x 32 blocks; wave w
  // takes blocks w, w + 4, ... of the two products
  constexpr int NBE = D / 32, NBB = NBE * NBE;
  for (int bk = __builtin_amdgcn_readfirstlane(tid >> 6); bk < 2 * NBB; bk += kLT / 64) {
    const int ab = 32 * ((bk % NBB) / NBE), eb = 32 * (bk % NBE);
    // C0 and G reach the decay gradient: fp32 steps, or with bf16 inputs
    // (v and dY exact in bf16) bf16 steps on Kd and Qe split in three
    floatx16 acc;
    if constexpr (kBF<TI>) acc = bk < NBB ? gram_block_split3<D>(kt, vv, ab, eb) : gram_block_split3<D>(qt, dy, ab, eb);
    else acc = bk < NBB ? gram_block<D>(kt, vv, ab, eb) : gram_block<D>(qt, dy, ab, eb);
    store_block<D>((bk < NBB ? a.dstate : a.pstate) + base * D * D, acc, ab, eb);
  }
}

// One 16 x 16 tile of a product on the matrix cores (16x16x4 fp32 steps; with
// BF, 16x16x32 bf16 steps and a 16x16x16 one for a remainder of four indices):
// acc[v] of lane (i, g) = sum over k in [k0, k0 + K) of X[r0 + i][k] B(k, c0 + ...)
// for output row r0 + 4 g + v and column c0 + i. X is a swizzled [kL][W]
// array; B(k, j) gives the column operand. K is a multiple of 16 and k0 of 4;
// lane group g takes the indices k0 + K/4 g .. k0 + K/4 g + K/4 - 1.
template <int W, bool BF = false, typename ColOp>
__device__ __forceinline__ floatx4 tile_product(const float (*X)[W], int r0, int c0, int k0, int K, ColOp B) {
  const int lane = threadIdx.x & 63, i = lane & 15, g = lane >> 4;
  const int kq = K >> 2, xr = r0 + i;
  floatx4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
  if constexpr (BF) {
    int s0 = 0;
    for (; s0 + 8 <= kq; s0 += 8) {
      const int k = k0 + kq * g + s0;
      const floatx4 x0 = ld4<W>(X, xr, k >> 2), x1 = ld4<W>(X, xr, (k >> 2) + 1);
      float xa[8], xb[8];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        xa[u] = x0[u];
        xa[4 + u] = x1[u];
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) xb[u] = B(k + u, c0 + i);
      acc = mfma16b(xa, xb, acc);
    }
    if (s0 < kq) {  // four indices left (K / 4 is a multiple of 4)
      const int k = k0 + kq * g + s0;
      const floatx4 x0 = ld4<W>(X, xr, k >> 2);
      float xa[4], xb[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        xa[u] = x0[u];
        xb[u] = B(k + u, c0 + i);
      }
      acc = mfma16b4(xa, xb, acc);
    }
  } else {
    for (int s0 = 0; s0 < kq; s0 += 4) {
      const int k = k0 + kq * g + s0;
      const floatx4 xa = ld4<W>(X, xr, k >> 2);
#pragma unroll
      for (int u = 0; u < 4; ++u) acc = mfma16f(xa[u], B(k + u, c0 + i), acc);
    }
  }
  return acc;
}

// Per chunk: every input gradient. Thread (row r = tid / kTPRG, part Q of the
// channels) keeps its row's gradients for the channels of Q in registers.
// The intra-chunk terms use the 16-row sub-blocks of the forward scores:
//   A (chunk_scores) and dA = dY V^T (j <= t blocks) on the matrix cores;
//   dv_intra = A^T dY; dq_intra, dk_intra below the diagonal as products with
//   the decay factored at a block boundary (q side: the row before the
//   query block; k side: the last row of the key block), both factors <= 1;
//   the diagonal blocks in the same products when the chunk's decay allows
//   (diag_factorable: the factors past the boundary stay below 2^kFactLim),
//   else term by term on the vector units.
// The three inter-chunk products are dense (kL x D by D x D), 32 x 32 blocks.
// SPLIT: a sub-problem of the D = 128 backward; it ends at dqt, dkt, dv and
// dg, its partials of the head's gradients, stored in fp32.
template <typename TI, int D, bool SPLIT = false>
__global__ __launch_bounds__(kLTG) void linear_grad_kernel(LinearArgs a) {
  static_assert(D == 32 || D == 64, "the backward kernel keeps the chunk of D <= 64 channels in LDS");
  constexpr int SB = 16, NSB = kL / SB, NE = D / 16;
  // all swizzled (swz) unless noted
  __shared__ float qt[kL][D], kt[kL][D], vv[kL][D], bb[kL][D], dy[kL][D];
  // M0: A^T; then dv_intra (plain); then Kd; then dKd Kd (plain)
  // M1: dA;  then dq_intra (plain); then G
  // M2: dA^T; then dk_intra (plain); then dVx and db (plain)
  __shared__ float M0[kL][kL], M1[kL][kL], M2[kL][kL];
  __shared__ float C0s[kL][kL + 1];  // plain, padded
  __shared__ float Srow[kL];
  constexpr int QW = D / kTPRG;      // channels per thread
  constexpr int NCG = D * D / kLTG;  // elements of C0 and of G per thread
  static_assert(D * D % kLTG == 0, "C0 and G split evenly over the threads");
  const ChunkPos p = chunk_pos(a);
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  // C0 and G are read from HBM now and reach LDS later
  const int64_t base = (int64_t)p.n * a.nchunks + p.c;
  float c0r[NCG], gr[NCG];
#pragma unroll
  for (int k = 0; k < NCG; ++k) {
    c0r[k] = a.cprev[base * D * D + tid + k * kLTG];
    gr[k] = a.gout[base * D * D + tid + k * kLTG];
  }
  load_chunk<TI, D, kLTG, true, true, true, SPLIT>(a, p, qt, kt, vv, bb, SPLIT ? nullptr : Srow, dy);
#pragma unroll
  for (int k = 0; k < NCG; ++k) {
    const int e = tid + k * kLTG;
    C0s[e / D][e % D] = c0r[k];
  }
  const HeadRef hr = head_ref<SPLIT, D>(a, p.n);
  const int64_t hoff = hr.hoff;
  constexpr int GW = SPLIT ? 2 * D : D;  // row length of g, dg and the partial gradients
  const int64_t plane = (int64_t)a.B * a.H * a.T * GW;
  const int ia = hr.pa ? 1 : 0, ie = hr.pe ? 1 : 0;
  const int r = tid / kTPRG, q0 = (tid % kTPRG) * QW;
  const int qs = swz<D>(r, q0);  // this thread's channels in a swizzled row r (contiguous)
  const int wrow = w * kRowsPerWave;
  // FACT: the diagonal blocks are factored at a reference row and join the
  // matrix-core products (the score blocks, and the dq and dk tiles below take
  // one more 16-row block); otherwise they are summed term by term
  const bool fact = diag_factorable<D>(bb);
  // ---- scores and dA: waves 0-7 the scores (to M0 as A^T), waves 8-15 dA
  if (w < 8) {
    chunk_scores<D, true, kBF<TI>>(qt, kt, bb, M0, fact);
  } else {
    // the ten blocks (tb, jb) with jb <= tb; wave 8 + i takes blocks i and i + 8
    const int i = lane & 15, g = lane >> 4;
    for (int bi = w - 8; bi < NSB * (NSB + 1) / 2; bi += 8) {
      int tb = 0, jb = bi;
      while (jb > tb) {
        jb -= tb + 1;
        ++tb;
      }
      const floatx4 acc = tile_product<D, kBF<TI>>(dy, SB * tb, SB * jb, 0, D, [&](int k, int j) { return vv[j][swz<D>(j, k)]; });
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int t = SB * tb + 4 * g + v, j = SB * jb + i;
        const float x = j < t ? acc[v] : 0.0f;
        M1[t][swz<kL>(t, j)] = x;
        M2[j][swz<kL>(j, t)] = x;
      }
    }
  }
  __syncthreads();
  // ---- intra products as 16 x 16 tiles, wave w takes tiles w, w + 16, w + 32
  //   type 0 (4 NE tiles): dv_intra[j][e] = sum_{t >= 16 jb} A^T[j][t] dY[t][e]
  //   type 1 (3 NE, 4 NE with FACT): dq_intra[t][d] = e^{b_t - b_rf} sum_j dA[t][j] kt[j][d] e^{b_rf - b_j},
  //     rf = 16 tb - 1 (0 for tb = 0), over j < 16 tb (below the diagonal) or j < 16 tb + 16 (FACT)
  //   type 2 (3 NE, 4 NE with FACT): dk_intra[j][d] = e^{b_rf - b_j} sum_t dA^T[j][t] qt[t][d] e^{b_t - b_rf},
  //     rf = 16 jb + 15, over t > rf or t >= 16 jb (FACT)
  // dA is zero for j >= t, so the diagonal blocks' upper triangles add nothing.
  // Types 1 and 2 reach the decay gradient: fp32 steps at any input type.
  constexpr int NT0 = NSB * NE, NTT = NT0 + 2 * NSB * NE;
  constexpr int MAXT = (NTT + 15) / 16;
  const int nt1 = fact ? NSB * NE : (NSB - 1) * NE, tb1 = fact ? 0 : 1;
  const int ntt = NT0 + 2 * nt1;
  floatx4 res[MAXT];
#pragma unroll
  for (int m = 0; m < MAXT; ++m) {
    const int tau = w + 16 * m;
    res[m] = floatx4{0.0f, 0.0f, 0.0f, 0.0f};
    if (tau < NT0) {
      const int jb = tau / NE, eb = tau % NE;
      res[m] = tile_product<kL, kBF<TI>>(M0, SB * jb, SB * eb, SB * jb, kL - SB * jb,
                                [&](int k, int e) { return dy[k][swz<D>(k, e)]; });
    } else if (tau < NT0 + nt1) {
      const int tb = tb1 + (tau - NT0) / NE, db = (tau - NT0) % NE;
      const int rf = tb ? SB * tb - 1 : 0, col = SB * db + (lane & 15);
      const float brf = bb[rf][swz<D>(rf, col)];
      floatx4 acc = tile_product<kL>(M1, SB * tb, SB * db, 0, SB * tb + (fact ? SB : 0), [&](int k, int d) {
        const int c = swz<D>(k, d);
        return kt[k][c] * fast_exp2((brf - bb[k][c]) * kLog2e);
      });
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int t = SB * tb + 4 * (lane >> 4) + v;
        acc[v] *= fast_exp2((bb[t][swz<D>(t, col)] - brf) * kLog2e);
      }
      res[m] = acc;
    } else if (tau < ntt) {
      const int jb = (tau - NT0 - nt1) / NE, db = (tau - NT0 - nt1) % NE;
      const int rf = SB * jb + SB - 1, col = SB * db + (lane & 15);
      const float brf = bb[rf][swz<D>(rf, col)];
      const int k0 = fact ? SB * jb : rf + 1;
      floatx4 acc = tile_product<kL>(M2, SB * jb, SB * db, k0, kL - k0, [&](int k, int d) {
        const int c = swz<D>(k, d);
        return qt[k][c] * fast_exp2((bb[k][c] - brf) * kLog2e);
      });
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int j = SB * jb + 4 * (lane >> 4) + v;
        acc[v] *= fast_exp2((brf - bb[j][swz<D>(j, col)]) * kLog2e);
      }
      res[m] = acc;
    }
  }
  // ---- diagonal blocks on the vector units (unless FACT), in the thread's row and channels
  float dq[QW], dk[QW], dv[QW], db[QW];
  float qself[QW], kself[QW], bself[QW];
#pragma unroll
  for (int i = 0; i < QW; ++i) {
    qself[i] = qt[r][qs + i];
    kself[i] = kt[r][qs + i];
    bself[i] = bb[r][qs + i];
    dq[i] = dk[i] = 0.0f;
    dv[i] = SPLIT && ia ? 0.0f : dy[r][qs + i];  // Y = I~ + E (once over the halves A)
  }
  if (!fact) {
    const int blo = (wrow / SB) * SB;  // the wave's rows share one 16-row block
    // dq: j in [blo, r)
    for (int j = blo; j < wrow + kRowsPerWave - 1; ++j) {
      if (j < r) {
        const float dA = M1[r][swz<kL>(r, j)];
        const int js = swz<D>(j, q0);
#pragma unroll
        for (int i = 0; i < QW; ++i)
          dq[i] = __builtin_fmaf(dA * kt[j][js + i], fast_exp2((bself[i] - bb[j][js + i]) * kLog2e), dq[i]);
      }
    }
    // dk: t in (r, blo + SB)
    for (int t = wrow + 1; t < blo + SB; ++t) {
      if (t > r) {
        const float dA = M2[r][swz<kL>(r, t)];
        const int ts = swz<D>(t, q0);
#pragma unroll
        for (int i = 0; i < QW; ++i)
          dk[i] = __builtin_fmaf(dA * qt[t][ts + i], fast_exp2((bb[t][ts + i] - bself[i]) * kLog2e), dk[i]);
      }
    }
  }
  __syncthreads();  // every read of A^T, dA, dA^T done
  {
    float(*R0)[D] = reinterpret_cast<float(*)[D]>(&M0[0][0]);
    float(*R1)[D] = reinterpret_cast<float(*)[D]>(&M1[0][0]);
    float(*R2)[D] = reinterpret_cast<float(*)[D]>(&M2[0][0]);
#pragma unroll
    for (int m = 0; m < MAXT; ++m) {
      const int tau = w + 16 * m;
      if (tau < ntt) {
        const int ty = tau < NT0 ? 0 : tau < NT0 + nt1 ? 1 : 2;
        const int u = tau - (ty == 0 ? 0 : ty == 1 ? NT0 : NT0 + nt1);
        const int rb = ty == 1 ? SB * (tb1 + u / NE) : SB * (u / NE), cb = SB * (u % NE);
        float(*R)[D] = ty == 0 ? R0 : ty == 1 ? R1 : R2;
#pragma unroll
        for (int v = 0; v < 4; ++v) R[rb + 4 * (lane >> 4) + v][cb + (lane & 15)] = res[m][v];
      }
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < QW; ++i) {
      dv[i] += R0[r][q0 + i];
      if (fact || r >= SB) dq[i] += R1[r][q0 + i];
      if (fact || r < kL - SB) dk[i] += R2[r][q0 + i];
      db[i] = qself[i] * dq[i] - kself[i] * dk[i];
    }
  }
  __syncthreads();  // M0, M1 free
  // Kd = kt e^{b_last - b} (row operand of dV += Kd G) to M0, G to M1, both swizzled [kL][D]
  float(*Kd)[D] = reinterpret_cast<float(*)[D]>(&M0[0][0]);
  float(*Gs)[D] = reinterpret_cast<float(*)[D]>(&M1[0][0]);
  float ek[QW], kd[QW];
#pragma unroll
  for (int i = 0; i < QW; ++i) {
    const int d = q0 + i;
    ek[i] = fast_exp2((bb[kL - 1][swz<D>(kL - 1, d)] - bself[i]) * kLog2e);
    kd[i] = kself[i] * ek[i];
    Kd[r][qs + i] = kd[i];
  }
#pragma unroll
  for (int k = 0; k < NCG; ++k) {
    const int e = tid + k * kLTG, gd = e / D, ge = e % D;
    Gs[gd][swz<D>(gd, ge)] = gr[k];
  }
  // p1 and p2 of this thread's row and channels, for the last step
  const int64_t prow = (int64_t)min(p.t0 + r, a.T - 1);  // rows past the sequence: loaded, then zero
  const TI* P1 = (const TI*)a.p1 + hoff + prow * a.st;
  const TI* P2 = (const TI*)a.p2 + hoff + prow * a.st;
  const bool ok = r < p.len;
  float x1[QW], x2[QW];
  float2 rq[QW];  // RoPE (cos, sin) of this thread's channels, read now for the last step
  if (!SPLIT && a.rope) {
    const int h = a.rope_half;
#pragma unroll
    for (int i = 0; i < QW; ++i) {
      const int c = q0 + i;
      rq[i] = c < 2 * h ? rope_cs(a, min(p.t0 + r, a.T - 1), c < h ? c : c - h) : make_float2(1.0f, 0.0f);
    }
  }
  if constexpr (!SPLIT) {
    if constexpr (QW == 4) {
      if (a.vec16) {
        Vec4<TI>::load(P1 + q0, x1);
        Vec4<TI>::load(P2 + q0, x2);
      }
    }
    if (QW != 4 || !a.vec16) {
#pragma unroll
      for (int i = 0; i < QW; ++i) {
        x1[i] = Elem<TI>::load(P1 + q0 + i);
        x2[i] = Elem<TI>::load(P2 + q0 + i);
      }
    }
#pragma unroll
    for (int i = 0; i < QW; ++i) {
      x1[i] = ok ? x1[i] : 0.0f;
      x2[i] = ok ? x2[i] : 0.0f;
    }
  }
  __syncthreads();
  // ---- inter-chunk terms: wave w < 3 NB takes block w % NB of
  //   product 0: dQe = dY C0^T,  1: dKd = V G^T,  2: dVx = Kd G.
  constexpr int NBC = D / 32, NB = (kL / 32) * NBC;
  static_assert(3 * NB <= kLTG / 64, "one block per wave");
  const int prod = w / NB, blk = w % NB;
  const int rb = 32 * (blk / NBC), cb = 32 * (blk % NBC);
  floatx16 acc;
  // dQe and dKd reach the decay gradient: fp32 steps, or with bf16 inputs
  // (dY and v exact in bf16) bf16 steps on C0 and G split in three, which
  // give the fp32 products
  auto c0t = [&](int k, int j) { return C0s[j][k]; };
  auto gt = [&](int k, int j) { return Gs[j][swz<D>(j, k)]; };
  if (prod == 0) {
    if constexpr (kBF<TI>) acc = block_product_split3<D>(dy, rb, cb, zero16(), c0t);
    else acc = block_product<D>(dy, rb, cb, zero16(), c0t);
  } else if (prod == 1) {
    if constexpr (kBF<TI>) acc = block_product_split3<D>(vv, rb, cb, zero16(), gt);
    else acc = block_product<D>(vv, rb, cb, zero16(), gt);
  } else if (prod == 2) {
    acc = block_product<D, kBF<TI>>(Kd, rb, cb, zero16(), [&](int k, int j) { return Gs[k][swz<D>(k, j)]; });
  }
  __syncthreads();  // every operand read: dy, vv, M2 take the three results (plain)
  float(*Dx)[D] = reinterpret_cast<float(*)[D]>(&M2[0][0]);
  if (prod < 3) {
    float(*O)[D] = prod == 0 ? dy : prod == 1 ? vv : Dx;
#pragma unroll
    for (int v = 0; v < 16; ++v) O[rb + acc_row(v, lane >> 5)][cb + (lane & 31)] = acc[v];
  }
  __syncthreads();
  float(*tmp)[D] = Kd;  // now plain: the column sums of dKd Kd go to the chunk's last row
#pragma unroll
  for (int i = 0; i < QW; ++i) {
    const int d = q0 + i;
    const float dqe = dy[r][d], dkd = vv[r][d];
    const float eb = fast_exp2(bself[i] * kLog2e);
    dq[i] = __builtin_fmaf(dqe, eb, dq[i]);
    dk[i] = __builtin_fmaf(dkd, ek[i], dk[i]);
    dv[i] += Dx[r][d];
    db[i] += dqe * qself[i] * eb - dkd * kd[i];
    tmp[r][d] = dkd * kd[i];
  }
#pragma unroll
  for (int i = 0; i < QW; ++i) Dx[r][q0 + i] = db[i];
  __syncthreads();
  // dg: reverse running sum of db down the chunk, plus the last row's extra
  // terms (column sums of dKd Kd, and dgamma e^{b_last}), which reach every row.
  // Thread (channel d, segment sg of RS rows) sums its rows from the bottom and
  // its shares of the extra terms; the partials meet in LDS (dy and vv are free).
  {
    constexpr int NSG = kLTG / D, RS = kL / NSG, ES = D / NSG;
    static_assert(RS * NSG == kL && ES * NSG == D && 2 * kLTG <= kL * D, "segments split evenly");
    const int d = tid % D, sg = tid / D;
    float* PT = &dy[0][0];         // [NSG][D]: segment totals of db
    float* PE = &dy[0][0] + kLTG;  // [NSG][D]: column sums of dKd Kd over the segment
    float* PG = &vv[0][0];         // [NSG][D]: shares of dgamma = sum_e G C0
    float suf[RS];
    float acc_t = 0.0f, ex = 0.0f, gm = 0.0f;
#pragma unroll
    for (int i = RS - 1; i >= 0; --i) {
      acc_t += Dx[sg * RS + i][d];
      suf[i] = acc_t;
      ex += tmp[sg * RS + i][d];
    }
#pragma unroll
    for (int i = 0; i < ES; ++i) {
      const int e = sg * ES + i;
      gm = __builtin_fmaf(Gs[d][swz<D>(d, e)], C0s[d][e], gm);
    }
    PT[sg * D + d] = acc_t;
    PE[sg * D + d] = ex;
    PG[sg * D + d] = gm;
    __syncthreads();
    float extra = 0.0f, dgam = 0.0f, later = 0.0f;
    for (int u = 0; u < NSG; ++u) {
      extra += PE[u * D + d];
      dgam += PG[u * D + d];
      if (u > sg) later += PT[u * D + d];
    }
    const float base_g = extra + dgam * fast_exp2(bb[kL - 1][swz<D>(kL - 1, d)] * kLog2e) + later;
    float* dG = SPLIT ? a.part + (6 + ie) * plane + (int64_t)hr.n * a.T * GW + hr.pa : a.dg + (int64_t)p.n * a.T * D;
    if (!SPLIT && a.a_log) {
      // the retention gate of eq. 15 (g = -exp(A_log) softplus(r + dt_bias)):
      // dr = dg (-exp(A_log) sigmoid(r + dt_bias)) goes out in place of dg, and
      // the chunk's per-channel sums of dg g and dr (its shares of dA_log and
      // d dt_bias) meet over the segments in LDS, in a fixed order
      const int64_t pc = (int64_t)(p.n % a.H) * D + d;
      const float ea = fast_exp2(a.a_log[pc] * kLog2e), dtb = a.dt_bias[pc];
      const float* Rg = a.g + (int64_t)p.n * a.T * D;
      float sa = 0.0f, sd = 0.0f;
#pragma unroll
      for (int i = 0; i < RS; ++i) {
        const int j = sg * RS + i;
        if (j < p.len) {
          const int64_t at = (int64_t)(p.t0 + j) * D + d;
          const float dgv = base_g + suf[i], x = Rg[at] + dtb;
          const float dr = dgv * (-ea * fast_rcp(1.0f + fast_exp2(-x * kLog2e)));
          sa = __builtin_fmaf(dgv, -ea * softplus_f(x), sa);
          sd += dr;
          dG[at] = dr;
        }
      }
      __syncthreads();  // every read of PT and PE done
      PT[sg * D + d] = sa;
      PE[sg * D + d] = sd;
      __syncthreads();
      if (sg == 0) {
        float ta = 0.0f, td = 0.0f;
        for (int u = 0; u < NSG; ++u) {
          ta += PT[u * D + d];
          td += PE[u * D + d];
        }
        float* P = a.gpart + ((int64_t)p.n * a.nchunks + p.c) * 2 * D;
        P[d] = ta;
        P[D + d] = td;
      }
    } else {
#pragma unroll
      for (int i = 0; i < RS; ++i) {
        const int j = sg * RS + i;
        if (j < p.len) dG[(int64_t)(p.t0 + j) * GW + d] = base_g + suf[i];
      }
    }
  }
  if constexpr (SPLIT) {
    static_assert(QW == 4, "a thread's channels are one 16-byte chunk");
    if (ok) {
      const int64_t row = ((int64_t)hr.n * a.T + p.t0 + r) * GW;
      Vec4<float>::store(a.part + ie * plane + row + hr.pa + q0, dq);
      Vec4<float>::store(a.part + (2 + ie) * plane + row + hr.pa + q0, dk);
      Vec4<float>::store(a.part + (4 + ia) * plane + row + hr.pe + q0, dv);
    }
    return;
  }
  // through qt = S p1 / |p1|, kt = S p2 / |p2|, S = sigmoid(scale p1 . p2 / tau_S)
  float s11 = 0.0f, s22 = 0.0f, s12 = 0.0f;
#pragma unroll
  for (int i = 0; i < QW; ++i) {
    s11 += x1[i] * x1[i];
    s22 += x2[i] * x2[i];
    s12 += x1[i] * x2[i];
  }
  s11 = group_sum<kTPRG>(s11);
  s22 = group_sum<kTPRG>(s22);
  s12 = group_sum<kTPRG>(s12);
  const float S = Srow[r];
  const float in1 = s11 > 0.0f ? rsqrtf(s11) : 0.0f, in2 = s22 > 0.0f ? rsqrtf(s22) : 0.0f;
  // with RoPE the projections below take the rotated p1, p2, and the result
  // goes back through the rotation's transpose. A channel's partner lives in
  // another thread of the row (the row's kTPRG threads are one lane group of
  // a wave): when it is the same element of that thread (h a multiple of
  // QW) it comes by a lane shuffle, else through the free qt and kt arrays
  // (plain layout) between two barriers.
  float(*X1)[D] = qt;
  float(*X2)[D] = kt;
  auto rotate = [&](float(&u1)[QW], float(&u2)[QW], bool transpose) {
    const int h = a.rope_half;
    float y1[QW], y2[QW];  // the partners' values
    if (h % QW == 0) {
      const bool lo = q0 < h;
      const int src = q0 < 2 * h ? lane + (lo ? h / QW : -(h / QW)) : lane;
#pragma unroll
      for (int i = 0; i < QW; ++i) {
        y1[i] = __shfl(u1[i], src, 64);
        y2[i] = __shfl(u2[i], src, 64);
      }
    } else {
#pragma unroll
      for (int i = 0; i < QW; ++i) {
        X1[r][q0 + i] = u1[i];
        X2[r][q0 + i] = u2[i];
      }
      __syncthreads();
#pragma unroll
      for (int i = 0; i < QW; ++i) {
        const int c = q0 + i, pc = c < h ? c + h : c < 2 * h ? c - h : c;
        y1[i] = X1[r][pc];
        y2[i] = X2[r][pc];
      }
      __syncthreads();
    }
#pragma unroll
    for (int i = 0; i < QW; ++i) {
      const int c = q0 + i;
      if (c < 2 * h) {
        const bool lo = c < h;
        const float2 cs = rq[i];
        const float sn = transpose ? -cs.y : cs.y;  // R^T: the angle negated
        u1[i] = lo ? u1[i] * cs.x - y1[i] * sn : y1[i] * sn + u1[i] * cs.x;
        u2[i] = lo ? u2[i] * cs.x - y2[i] * sn : y2[i] * sn + u2[i] * cs.x;
      }
    }
  };
  if (a.rope) rotate(x1, x2, false);
  // dS = dqt . ^p1 + dkt . ^p2; ^p . d^p for the projections
  float ds = 0.0f, h1d = 0.0f, h2d = 0.0f;
#pragma unroll
  for (int i = 0; i < QW; ++i) {
    ds += dq[i] * x1[i] * in1 + dk[i] * x2[i] * in2;
    h1d += x1[i] * in1 * dq[i];
    h2d += x2[i] * in2 * dk[i];
  }
  ds = group_sum<kTPRG>(ds);
  h1d = group_sum<kTPRG>(h1d);
  h2d = group_sum<kTPRG>(h2d);
  const float dU = ds * S * (1.0f - S) * a.scale * a.inv_tau;
  float g1[QW], g2[QW];
#pragma unroll
  for (int i = 0; i < QW; ++i) {
    // d^p1 = S dqt; dp1 = dU p2 + (d^p1 - ^p1 (^p1 . d^p1)) / |p1|
    g1[i] = dU * x2[i] + S * (dq[i] - x1[i] * in1 * h1d) * in1;
    g2[i] = dU * x1[i] + S * (dk[i] - x2[i] * in2 * h2d) * in2;
  }
  if (a.rope) rotate(g1, g2, true);
  if (ok) {
    TI* DP1 = (TI*)a.dp1 + hoff + (int64_t)(p.t0 + r) * a.st;
    TI* DP2 = (TI*)a.dp2 + hoff + (int64_t)(p.t0 + r) * a.st;
    TI* DV = (TI*)a.dv + hoff + (int64_t)(p.t0 + r) * a.st;
    if constexpr (QW == 4) {
      if (a.vec16) {
        Vec4<TI>::store(DP1 + q0, g1);
        Vec4<TI>::store(DP2 + q0, g2);
        Vec4<TI>::store(DV + q0, dv);
      }
    }
    if (QW != 4 || !a.vec16) {
#pragma unroll
      for (int i = 0; i < QW; ++i) {
        Elem<TI>::store(DP1 + q0 + i, g1[i]);
        Elem<TI>::store(DP2 + q0 + i, g2[i]);
        Elem<TI>::store(DV + q0 + i, dv[i]);
      }
    }
  }
}

template <typename TI, int D, bool SPLIT = false>
hipError_t launch_bwd_d(const LinearArgs& a, hipStream_t stream) {
  const dim3 grid((unsigned)a.nchunks, (unsigned)virtual_heads(a));
  hipLaunchKernelGGL((linear_bstate_kernel<TI, D, SPLIT>), grid, dim3(kLT), 0, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  e = launch_state_scan(a, 1, stream);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((linear_grad_kernel<TI, D, SPLIT>), grid, dim3(kLTG), 0, stream, a);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// D = 128 backward. The state's rows evolve with their own retention and its
// columns do not mix, so the state splits into four 64 x 64 blocks (relation
// half A, information half E), each a recurrence of its own driven by
// kt[A], v[E], alpha[A] and read by qt[A]. The scores of the intra-chunk
// pairs and their gradients split the same way: a score is the sum of its
// two relation halves, dA the sum of the information halves of dY . v. So
// every gradient is the sum over the other half of the four problems' terms.
// Only qt = S ^p1 and kt = S ^p2 (S and the norms over all 128 channels) do
// not split: a row pass forms them before, and another takes the summed dqt,
// dkt through S and the normalisation after.
// ---------------------------------------------------------------------------
constexpr int kSW = 128;            // channels
constexpr int kSLanes = kSW / 4;    // lanes per row, 4 channels each
constexpr int kSRows = 256 / kSLanes;

// The row of flat index row (n * T + t) that this lane's group works on, its
// first channel, and whether the row exists (rows past the end are clamped
// to the last one and then not stored, so that every lane takes part in the
// lane sums).
struct SplitRow {
  int64_t nt;
  int c0;
  bool ok;
  int64_t off;  // element offset of the row in p1, p2, v, dY and their gradients
};

__device__ __forceinline__ SplitRow split_row(const LinearArgs& a) {
  SplitRow s;
  const int64_t rows = (int64_t)a.B * a.H * a.T;
  const int64_t nt = (int64_t)blockIdx.x * kSRows + threadIdx.x / kSLanes;
  s.ok = nt < rows;
  s.nt = s.ok ? nt : rows - 1;
  s.c0 = (threadIdx.x % kSLanes) * 4;
  const int64_t n = s.nt / a.T, t = s.nt % a.T;
  s.off = (n / a.H) * a.sb + (n % a.H) * a.sh + t * a.st + s.c0;
  return s;
}

template <typename TI>
__device__ __forceinline__ void load4(const LinearArgs& a, const TI* p, float (&x)[4]) {
  if (a.vec16) {
    Vec4<TI>::load(p, x);
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i) x[i] = Elem<TI>::load(p + i);
  }
}

template <typename TI>
__device__ __forceinline__ void store4(const LinearArgs& a, TI* p, const float (&x)[4]) {
  if (a.vec16) {
    Vec4<TI>::store(p, x);
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i) Elem<TI>::store(p + i, x[i]);
  }
}

// S, 1/|p1| and 1/|p2| of a row held as 4 channels per lane over kSLanes lanes.
__device__ __forceinline__ void row_self(const LinearArgs& a, const float (&x1)[4], const float (&x2)[4], float& S,
                                        float& in1, float& in2) {
  float s11 = 0.0f, s22 = 0.0f, s12 = 0.0f;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    s11 += x1[i] * x1[i];
    s22 += x2[i] * x2[i];
    s12 += x1[i] * x2[i];
  }
  s11 = lane_group_sum<kSLanes>(s11);
  s22 = lane_group_sum<kSLanes>(s22);
  s12 = lane_group_sum<kSLanes>(s12);
  S = 1.0f / (1.0f + expf(-s12 * a.scale * a.inv_tau));
  in1 = s11 > 0.0f ? rsqrtf(s11) : 0.0f;
  in2 = s22 > 0.0f ? rsqrtf(s22) : 0.0f;
}

// RoPE of a row held as 4 channels per lane over kSLanes lanes (pairs (j,
// j + h) with h a multiple of 4, so a lane's partner chunk is one lane):
// transpose = false rotates, true applies the transposed rotation. Every lane
// of the wave takes part (the exchange is a lane shuffle).
__device__ __forceinline__ void rope_row(const LinearArgs& a, int64_t t, int c0, float (&u)[4], bool transpose) {
  const int h = a.rope_half, lane = threadIdx.x & 63;
  const bool lo = c0 < h, on = c0 < 2 * h;
  const int src = on ? (lo ? lane + h / 4 : lane - h / 4) : lane;
  float pv[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) pv[e] = __shfl(u[e], src, 64);
  if (on) {
    const int j0 = lo ? c0 : c0 - h;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float2 cs = rope_cs(a, t, j0 + e);
      const float sn = transpose ? -cs.y : cs.y;
      u[e] = lo ? u[e] * cs.x - pv[e] * sn : pv[e] * sn + u[e] * cs.x;
    }
  }
}

// qn = S ^p1, kn = S ^p2 per row (rotated with RoPE).
template <typename TI>
__global__ __launch_bounds__(256) void linear_split_prep_kernel(LinearArgs a) {
  const SplitRow w = split_row(a);
  float x1[4], x2[4], S, in1, in2;
  load4<TI>(a, (const TI*)a.p1 + w.off, x1);
  load4<TI>(a, (const TI*)a.p2 + w.off, x2);
  row_self(a, x1, x2, S, in1, in2);
  if (a.rope) {
    rope_row(a, w.nt % a.T, w.c0, x1, false);
    rope_row(a, w.nt % a.T, w.c0, x2, false);
  }
  if (w.ok) {
    float q[4], k[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      q[i] = x1[i] * (S * in1);
      k[i] = x2[i] * (S * in2);
    }
    Vec4<float>::store(a.qn + w.nt * kSW + w.c0, q);
    Vec4<float>::store(a.kn + w.nt * kSW + w.c0, k);
  }
}

// Sums the four problems' partials and takes dqt, dkt through
// qt = S p1 / |p1|, kt = S p2 / |p2|, S = sigmoid(scale p1 . p2 / tau_S).
template <typename TI>
__global__ __launch_bounds__(256) void linear_split_combine_kernel(LinearArgs a) {
  const SplitRow w = split_row(a);
  const int64_t plane = (int64_t)a.B * a.H * a.T * kSW, at = w.nt * kSW + w.c0;
  float x1[4], x2[4], S, in1, in2;
  load4<TI>(a, (const TI*)a.p1 + w.off, x1);
  load4<TI>(a, (const TI*)a.p2 + w.off, x2);
  float pr[8][4];
#pragma unroll
  for (int k = 0; k < 8; ++k) Vec4<float>::load(a.part + k * plane + at, pr[k]);
  row_self(a, x1, x2, S, in1, in2);
  if (a.rope) {  // the projections take the rotated coordinates
    rope_row(a, w.nt % a.T, w.c0, x1, false);
    rope_row(a, w.nt % a.T, w.c0, x2, false);
  }
  float dq[4], dk[4], dv[4], dg[4];
  float ds = 0.0f, h1d = 0.0f, h2d = 0.0f;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    dq[i] = pr[0][i] + pr[1][i];
    dk[i] = pr[2][i] + pr[3][i];
    dv[i] = pr[4][i] + pr[5][i];
    dg[i] = pr[6][i] + pr[7][i];
    ds += dq[i] * x1[i] * in1 + dk[i] * x2[i] * in2;
    h1d += x1[i] * in1 * dq[i];
    h2d += x2[i] * in2 * dk[i];
  }
  ds = lane_group_sum<kSLanes>(ds);
  h1d = lane_group_sum<kSLanes>(h1d);
  h2d = lane_group_sum<kSLanes>(h2d);
  const float dU = ds * S * (1.0f - S) * a.scale * a.inv_tau;
  float g1[4], g2[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    g1[i] = dU * x2[i] + S * (dq[i] - x1[i] * in1 * h1d) * in1;
    g2[i] = dU * x1[i] + S * (dk[i] - x2[i] * in2 * h2d) * in2;
  }
  if (a.rope) {  // back through the rotation
    rope_row(a, w.nt % a.T, w.c0, g1, true);
    rope_row(a, w.nt % a.T, w.c0, g2, true);
  }
  if (w.ok) {
    store4<TI>(a, (TI*)a.dp1 + w.off, g1);
    store4<TI>(a, (TI*)a.dp2 + w.off, g2);
    store4<TI>(a, (TI*)a.dv + w.off, dv);
    Vec4<float>::store(a.dg + at, dg);
  }
}

template <typename TI>
hipError_t launch_bwd_split(const LinearArgs& a, hipStream_t stream) {
  const int64_t rows = (int64_t)a.B * a.H * a.T;
  const dim3 rgrid((unsigned)((rows + kSRows - 1) / kSRows));
  hipLaunchKernelGGL((linear_split_prep_kernel<TI>), rgrid, dim3(256), 0, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  LinearArgs s = a;
  s.D = kSW / 2;
  s.split = 1;
  s.rope = nullptr;  // qn and kn are rotated already
  e = launch_bwd_d<TI, kSW / 2, true>(s, stream);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((linear_split_combine_kernel<TI>), rgrid, dim3(256), 0, stream, a);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Backward through the retention gate of eq. 15 at width 128, after the
// combine pass has left dg in a.dg: per element dr = dg (-exp(A_log)
// sigmoid(r + dt_bias)), written over dg; per head, token segment and channel
// the sums of dg g (d A_log, since dg/dA_log = g) and of dr (d dt_bias). Then,
// at every width, per head and channel the sum of those (per segment, or per
// chunk as the gradient kernel leaves them) over batch entries, in a fixed
// order.
// ---------------------------------------------------------------------------
constexpr int kGateSeg = 256;  // tokens per segment

template <int D>
__global__ __launch_bounds__(256) void linear_gate_bwd_kernel(LinearArgs a) {
  constexpr int RG = 256 / D;  // rows in flight per step
  __shared__ float red[2][RG][D];
  const int n = blockIdx.y, seg = blockIdx.x;
  const int c = threadIdx.x % D, rg = threadIdx.x / D;
  const int64_t pc = (int64_t)(n % a.H) * D + c;
  const float ea = fast_exp2(a.a_log[pc] * kLog2e), dtb = a.dt_bias[pc];
  const int t0 = seg * kGateSeg, t1 = min(a.T, t0 + kGateSeg);
  const float* R = a.g + (int64_t)n * a.T * D;
  float* DG = a.dg + (int64_t)n * a.T * D;
  float sa = 0.0f, sd = 0.0f;
  for (int t = t0 + rg; t < t1; t += RG) {
    const int64_t i = (int64_t)t * D + c;
    const float x = R[i] + dtb, dg = DG[i];
    const float dr = dg * (-ea * fast_rcp(1.0f + fast_exp2(-x * kLog2e)));  // softplus' = sigmoid
    sa = __builtin_fmaf(dg, -ea * softplus_f(x), sa);
    sd += dr;
    DG[i] = dr;
  }
  red[0][rg][c] = sa;
  red[1][rg][c] = sd;
  __syncthreads();
  if (rg == 0) {
    for (int k = 1; k < RG; ++k) {
      sa += red[0][k][c];
      sd += red[1][k][c];
    }
    float* P = a.gpart + (((int64_t)n * gridDim.x + seg) * 2) * D;
    P[c] = sa;
    P[D + c] = sd;
  }
}

// One wave per (head, channel): lane l sums the (batch entry, segment) items
// l, l + 64, ... in order, then the 64 lane sums meet in a fixed butterfly, so
// the result does not depend on timing.
__global__ __launch_bounds__(256) void linear_gate_reduce_kernel(LinearArgs a, int nseg) {
  const int idx = blockIdx.x * 4 + (int)(threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (idx >= a.H * a.D) return;  // wave-uniform
  const int h = idx / a.D, c = idx % a.D;
  float sa = 0.0f, sd = 0.0f;
  for (int it = lane; it < a.B * nseg; it += 64) {
    const int b = it / nseg, sg = it % nseg;
    const float* P = a.gpart + (((int64_t)(b * a.H + h) * nseg + sg) * 2) * a.D + c;
    sa += P[0];
    sd += P[a.D];
  }
  for (int o = 32; o >= 1; o >>= 1) {
    sa += __shfl_xor(sa, o, 64);
    sd += __shfl_xor(sd, o, 64);
  }
  if (lane == 0) {
    a.da_log[idx] = sa;
    a.ddt_bias[idx] = sd;
  }
}

// The gradient kernel (D <= 64) forms dr and per-chunk sums itself; the
// width-128 backward (its dg comes from the combine pass) takes the row pass.
hipError_t launch_gate_bwd(const LinearArgs& a, hipStream_t stream) {
  int nseg = a.nchunks;
  if (a.D == 128) {
    nseg = (a.T + kGateSeg - 1) / kGateSeg;
    hipLaunchKernelGGL(linear_gate_bwd_kernel<128>, dim3((unsigned)nseg, (unsigned)(a.B * a.H)), dim3(256), 0,
                       stream, a);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(linear_gate_reduce_kernel, dim3((unsigned)((a.H * a.D + 3) / 4)), dim3(256), 0, stream, a, nseg);
  return hipGetLastError();
}

template <typename TI>
hipError_t launch_bwd_t(const LinearArgs& a, hipStream_t stream) {
  switch (a.D) {
    case 32: return launch_bwd_d<TI, 32>(a, stream);
    case 64: return launch_bwd_d<TI, 64>(a, stream);
    case kSW: return launch_bwd_split<TI>(a, stream);
    default: return hipErrorInvalidValue;
  }
}

template <typename TI, int D>
hipError_t launch_fwd_d(const LinearArgs& a, hipStream_t stream) {
  const dim3 grid((unsigned)a.nchunks, (unsigned)(a.B * a.H));
  hipLaunchKernelGGL((linear_state_kernel<TI, D>), grid, dim3(kLT), 0, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  e = launch_state_scan(a, 0, stream);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((linear_out_kernel<TI, D>), grid, dim3(kLT2), 0, stream, a);
  return hipGetLastError();
}

template <typename TI>
hipError_t launch_fwd_t(const LinearArgs& a, hipStream_t stream) {
  switch (a.D) {
    case 32: return launch_fwd_d<TI, 32>(a, stream);
    case 64: return launch_fwd_d<TI, 64>(a, stream);
    case 128: return launch_fwd_d<TI, 128>(a, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

// The RoPE table of rope_cs: (cos, sin) of t * base^(-2j/rope_dim) for t at
// the chunk starts and the offsets inside a chunk, evaluated in fp64.
__global__ __launch_bounds__(256) void linear_rope_table_kernel(float2* tab, int nch, int rope_dim, double log_base) {
  const int h = rope_dim / 2;
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (int64_t)(nch + kL) * h) return;
  const int row = (int)(idx / h), j = (int)(idx % h);
  const double t = row < nch ? (double)row * kL : (double)(row - nch);
  double sn, cs;
  sincos(t * exp(-2.0 * (double)j / (double)rope_dim * log_base), &sn, &cs);
  tab[idx] = make_float2((float)cs, (float)sn);
}

int linear_chunk() { return kL; }

hipError_t launch_linear_rope_table(float2* tab, int T, int rope_dim, double base, hipStream_t stream) {
  const int nch = (T + kL - 1) / kL;
  const int64_t n = (int64_t)(nch + kL) * (rope_dim / 2);
  hipLaunchKernelGGL(linear_rope_table_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, stream, tab, nch,
                     rope_dim, log(base));
  return hipGetLastError();
}
int linear_scan_segment() { return kSegChunks; }

hipError_t launch_linear_fwd(const LinearArgs& a, int dtype, hipStream_t stream) {
  return dtype == 1 ? launch_fwd_t<bf16>(a, stream) : launch_fwd_t<float>(a, stream);
}

hipError_t launch_linear_bwd(const LinearArgs& a, int dtype, hipStream_t stream) {
  const hipError_t e = dtype == 1 ? launch_bwd_t<bf16>(a, stream) : launch_bwd_t<float>(a, stream);
  if (e != hipSuccess || !a.a_log) return e;
  return launch_gate_bwd(a, stream);
}

int linear_gate_segment() { return kGateSeg; }

}  // namespace rel
