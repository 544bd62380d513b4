// Prologue and epilogue kernels of the layer entry points: RoPE on the two
// relation projections (Sec. 3.1), Givens head-pair mixing of the information
// state (eq. 4, App. A.2.2-A.2.3), zero padding of the head width to the width
// the fused kernels tile, and the backward of all three.
//
// Each of these is a pass over [B, H, T, D] rows whose cost is linear in T,
// against the T^2 work of the fused kernels, so the rotation, the mixing and the
// padding run once per row here instead of once per key tile inside the fused
// kernels. They are bound by HBM: every thread moves VEC contiguous channels
// (16 bytes when the caller's layout allows it), TPR threads (a power of two,
// at most 64) cover one row, and rows are contiguous in the padded layout.
//
// RoPE rotates channel d with channel d + D/2 by t * base^(-2d/D) (t zero-based),
// with cos and sin from a per-call [T, D/2] table evaluated in fp64.
// Givens mixing writes, for head h of pair p with partner head h':
//   I~_h = cos(theta_p) I_h + sigma_h sin(theta_p) I_h'
// where sigma_h = -1 for the pair's first head and +1 for its second.
#include "kernels.h"

namespace rel {

namespace {

constexpr int kLThreads = 256;
constexpr int kSumParts = 64;  // first-stage partial sums per dtheta segment

// VEC contiguous elements of type TI at p + i, as floats (i a multiple of VEC).
template <typename TI, int VEC>
struct Chunk;

template <>
struct Chunk<bf16, 8> {
  static __device__ __forceinline__ void load(const void* p, int64_t i, float (&x)[8]) {
    const uintx4 u = *reinterpret_cast<const uintx4*>((const bf16*)p + i);
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      x[2 * t] = bf16_lo(u[t]);
      x[2 * t + 1] = bf16_hi(u[t]);
    }
  }
  static __device__ __forceinline__ void store(void* p, int64_t i, const float (&x)[8]) {
    bf16x8 o;
#pragma unroll
    for (int t = 0; t < 8; ++t) o[t] = (bf16)x[t];
    *reinterpret_cast<bf16x8*>((bf16*)p + i) = o;
  }
};

template <>
struct Chunk<bf16, 2> {
  static __device__ __forceinline__ void load(const void* p, int64_t i, float (&x)[2]) {
    const unsigned int u = *reinterpret_cast<const unsigned int*>((const bf16*)p + i);
    x[0] = bf16_lo(u);
    x[1] = bf16_hi(u);
  }
  static __device__ __forceinline__ void store(void* p, int64_t i, const float (&x)[2]) {
    typedef bf16 bf16x2 __attribute__((ext_vector_type(2)));
    bf16x2 o;
    o[0] = (bf16)x[0];
    o[1] = (bf16)x[1];
    *reinterpret_cast<bf16x2*>((bf16*)p + i) = o;
  }
};

template <>
struct Chunk<float, 4> {
  static __device__ __forceinline__ void load(const void* p, int64_t i, float (&x)[4]) {
    const float4 u = *reinterpret_cast<const float4*>((const float*)p + i);
    x[0] = u.x; x[1] = u.y; x[2] = u.z; x[3] = u.w;
  }
  static __device__ __forceinline__ void store(void* p, int64_t i, const float (&x)[4]) {
    *reinterpret_cast<float4*>((float*)p + i) = make_float4(x[0], x[1], x[2], x[3]);
  }
};

template <>
struct Chunk<float, 2> {
  static __device__ __forceinline__ void load(const void* p, int64_t i, float (&x)[2]) {
    const float2 u = *reinterpret_cast<const float2*>((const float*)p + i);
    x[0] = u.x; x[1] = u.y;
  }
  static __device__ __forceinline__ void store(void* p, int64_t i, const float (&x)[2]) {
    *reinterpret_cast<float2*>((float*)p + i) = make_float2(x[0], x[1]);
  }
};

template <typename TI>
struct Chunk<TI, 1> {
  static __device__ __forceinline__ void load(const void* p, int64_t i, float (&x)[1]) {
    x[0] = Elem<TI>::load((const TI*)p + i);
  }
  static __device__ __forceinline__ void store(void* p, int64_t i, const float (&x)[1]) {
    Elem<TI>::store((TI*)p + i, x[0]);
  }
};

// Pair index, partner head and sign sigma of head h in pairing 1 (A: (1,2),
// (3,4), ...) or 2 (B: (2,3), ..., (H,1)); heads are zero-based here.
__device__ __forceinline__ void givens_role(int h, int H, int mode, int& pair, int& partner,
                                            float& sigma) {
  if (mode == 1) {
    pair = h >> 1;
    partner = h ^ 1;
    sigma = (h & 1) ? 1.0f : -1.0f;
  } else if (h & 1) {
    pair = (h - 1) >> 1;
    partner = h + 1 == H ? 0 : h + 1;
    sigma = -1.0f;
  } else {
    const int hh = h == 0 ? H : h;
    pair = (hh >> 1) - 1;
    partner = hh - 1;
    sigma = 1.0f;
  }
}

// The row (b, h, t) a thread works on, and its position among the row's threads.
struct RowPos {
  int64_t row;  // (b H + h) T + t
  int t, h, b, lane;
  bool valid;
};

template <int TPR>
__device__ __forceinline__ RowPos row_pos(const LayerArgs& a) {
  RowPos r;
  r.row = (int64_t)blockIdx.x * (kLThreads / TPR) + threadIdx.x / TPR;
  r.lane = threadIdx.x % TPR;
  r.valid = r.row < (int64_t)a.B * a.H * a.T;
  const int64_t row = r.valid ? r.row : 0;
  r.t = (int)(row % a.T);
  const int64_t n = row / a.T;
  r.h = (int)(n % a.H);
  r.b = (int)(n / a.H);
  return r;
}

__global__ __launch_bounds__(256) void rope_table_kernel(float2* tab, int T, int D, double log_base) {
  const int half = D >> 1;
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (int64_t)T * half) return;
  const int t = (int)(idx / half), j = (int)(idx % half);
  const double ang = (double)t * exp(-2.0 * (double)j / (double)D * log_base);
  double s, c;
  sincos(ang, &s, &c);
  tab[idx] = make_float2((float)c, (float)s);
}

template <typename TI, int VEC, int TPR>
__global__ __launch_bounds__(kLThreads) void prologue_kernel(LayerArgs a) {
  const RowPos r = row_pos<TPR>(a);
  if (!r.valid) return;
  const int64_t src = r.b * a.sb + r.h * a.sh + (int64_t)r.t * a.st;
  const int64_t dst = r.row * a.DP;
  const int half = a.D >> 1;
  int pair = 0, partner = r.h;
  float sigma = 0.0f, cth = 1.0f, sth = 0.0f;
  if (a.givens) {
    givens_role(r.h, a.H, a.givens, pair, partner, sigma);
    sincosf(a.theta[pair], &sth, &cth);
  }
  const int64_t srcp = r.b * a.sb + partner * a.sh + (int64_t)r.t * a.st;
  for (int c0 = r.lane * VEC; c0 < a.DP; c0 += TPR * VEC) {
    float yq[VEC], yk[VEC], yv[VEC];
#pragma unroll
    for (int e = 0; e < VEC; ++e) yq[e] = yk[e] = yv[e] = 0.0f;
    if (c0 < a.D) {
      if (a.rope) {
        // a chunk never straddles the two halves: VEC divides D / 2
        const bool lo = c0 < half;
        const int j0 = lo ? c0 : c0 - half;
        float q1[VEC], q2[VEC], k1[VEC], k2[VEC];
        Chunk<TI, VEC>::load(a.q, src + j0, q1);
        Chunk<TI, VEC>::load(a.q, src + j0 + half, q2);
        Chunk<TI, VEC>::load(a.k, src + j0, k1);
        Chunk<TI, VEC>::load(a.k, src + j0 + half, k2);
#pragma unroll
        for (int e = 0; e < VEC; ++e) {
          const float2 cs = a.rope[(int64_t)r.t * half + j0 + e];
          yq[e] = lo ? q1[e] * cs.x - q2[e] * cs.y : q1[e] * cs.y + q2[e] * cs.x;
          yk[e] = lo ? k1[e] * cs.x - k2[e] * cs.y : k1[e] * cs.y + k2[e] * cs.x;
        }
      } else {
        Chunk<TI, VEC>::load(a.q, src + c0, yq);
        Chunk<TI, VEC>::load(a.k, src + c0, yk);
      }
      Chunk<TI, VEC>::load(a.v, src + c0, yv);
      if (a.givens) {
        float vp[VEC];
        Chunk<TI, VEC>::load(a.v, srcp + c0, vp);
#pragma unroll
        for (int e = 0; e < VEC; ++e) yv[e] = cth * yv[e] + sigma * sth * vp[e];
      }
    }
    Chunk<TI, VEC>::store(a.qr, dst + c0, yq);
    Chunk<TI, VEC>::store(a.kr, dst + c0, yk);
    Chunk<TI, VEC>::store(a.vt, dst + c0, yv);
  }
}

// Copies rows between the caller's layout (true width D) and the contiguous
// padded layout (width DP): to_padded = 1 writes zeros in channels D .. DP-1.
template <typename TI, int VEC, int TPR>
__global__ __launch_bounds__(kLThreads) void repad_kernel(const void* src, void* dst, LayerArgs a,
                                                          int to_padded) {
  const RowPos r = row_pos<TPR>(a);
  if (!r.valid) return;
  const int64_t cl = r.b * a.sb + r.h * a.sh + (int64_t)r.t * a.st;
  const int64_t pd = r.row * a.DP;
  for (int c0 = r.lane * VEC; c0 < a.DP; c0 += TPR * VEC) {
    float x[VEC];
    if (to_padded) {
      if (c0 < a.D) {
        Chunk<TI, VEC>::load(src, cl + c0, x);
      } else {
#pragma unroll
        for (int e = 0; e < VEC; ++e) x[e] = 0.0f;
      }
      Chunk<TI, VEC>::store(dst, pd + c0, x);
    } else if (c0 < a.D) {
      Chunk<TI, VEC>::load(src, pd + c0, x);
      Chunk<TI, VEC>::store(dst, cl + c0, x);
    }
  }
}

// Backward: gradients in the padded layout (gq, gk with respect to the rotated
// projections, gv with respect to I~) to the caller's tensors, and each row's
// term of dL/dtheta for the pair whose first head this row belongs to:
//   dL/dtheta_p += dI~_a . (-s I_a - c I_b) + dI~_b . (c I_a - s I_b).
// Threads past the last row still join the row reduction (they add zero).
template <typename TI, int VEC, int TPR>
__global__ __launch_bounds__(kLThreads) void epilogue_kernel(LayerArgs a) {
  const RowPos r = row_pos<TPR>(a);
  const int64_t cl = r.b * a.sb + r.h * a.sh + (int64_t)r.t * a.st;
  const int64_t pd = r.row * a.DP;
  const int half = a.D >> 1;
  int pair = 0, partner = r.h;
  float sigma = 0.0f, cth = 1.0f, sth = 0.0f;
  if (a.givens) {
    givens_role(r.h, a.H, a.givens, pair, partner, sigma);
    sincosf(a.theta[pair], &sth, &cth);
  }
  const int64_t pdp = (((int64_t)r.b * a.H + partner) * a.T + r.t) * a.DP;  // partner row, padded
  const int64_t clp = r.b * a.sb + partner * a.sh + (int64_t)r.t * a.st;    // partner row, caller
  const bool first = a.givens && sigma < 0.0f;
  float dth = 0.0f;
  for (int c0 = r.lane * VEC; r.valid && c0 < a.D; c0 += TPR * VEC) {
    float oq[VEC], ok[VEC];
    if (a.rope) {
      const bool lo = c0 < half;
      const int j0 = lo ? c0 : c0 - half;
      float q1[VEC], q2[VEC], k1[VEC], k2[VEC];
      Chunk<TI, VEC>::load(a.gq, pd + j0, q1);
      Chunk<TI, VEC>::load(a.gq, pd + j0 + half, q2);
      Chunk<TI, VEC>::load(a.gk, pd + j0, k1);
      Chunk<TI, VEC>::load(a.gk, pd + j0 + half, k2);
#pragma unroll
      for (int e = 0; e < VEC; ++e) {
        const float2 cs = a.rope[(int64_t)r.t * half + j0 + e];
        oq[e] = lo ? q1[e] * cs.x + q2[e] * cs.y : -q1[e] * cs.y + q2[e] * cs.x;
        ok[e] = lo ? k1[e] * cs.x + k2[e] * cs.y : -k1[e] * cs.y + k2[e] * cs.x;
      }
    } else {
      Chunk<TI, VEC>::load(a.gq, pd + c0, oq);
      Chunk<TI, VEC>::load(a.gk, pd + c0, ok);
    }
    Chunk<TI, VEC>::store(a.dq, cl + c0, oq);
    Chunk<TI, VEC>::store(a.dk, cl + c0, ok);
    float gh[VEC];
    Chunk<TI, VEC>::load(a.gv, pd + c0, gh);
    if (a.givens) {
      float gp[VEC], ov[VEC];
      Chunk<TI, VEC>::load(a.gv, pdp + c0, gp);
#pragma unroll
      for (int e = 0; e < VEC; ++e) ov[e] = cth * gh[e] - sigma * sth * gp[e];
      if (first) {  // h = a, partner = b
        float va[VEC], vb[VEC];
        Chunk<TI, VEC>::load(a.v, cl + c0, va);
        Chunk<TI, VEC>::load(a.v, clp + c0, vb);
#pragma unroll
        for (int e = 0; e < VEC; ++e)
          dth += gh[e] * (-sth * va[e] - cth * vb[e]) + gp[e] * (cth * va[e] - sth * vb[e]);
      }
      Chunk<TI, VEC>::store(a.dv, cl + c0, ov);
    } else {
      Chunk<TI, VEC>::store(a.dv, cl + c0, gh);
    }
  }
  if (a.givens) {
    for (int o = TPR / 2; o >= 1; o >>= 1) dth += __shfl_xor(dth, o, 64);
    if (r.valid && first && r.lane == 0) a.dth_rows[((int64_t)pair * a.B + r.b) * a.T + r.t] = dth;
  }
}

// Fixed-order sums of nseg segments of seg_len floats: stage 1 (grid
// nseg x kSumParts) sums contiguous parts of each segment, stage 2 (grid nseg)
// sums a segment's kSumParts partials.
__device__ __forceinline__ float block_sum(float acc) {
  __shared__ float sh[256];
  sh[threadIdx.x] = acc;
  __syncthreads();
  for (int hh = 128; hh >= 1; hh >>= 1) {
    if ((int)threadIdx.x < hh) sh[threadIdx.x] += sh[threadIdx.x + hh];
    __syncthreads();
  }
  return sh[0];
}

__global__ __launch_bounds__(256) void segment_parts_kernel(const float* x, int64_t seg_len, float* part) {
  const int seg = blockIdx.y, pi = blockIdx.x;
  const int64_t chunk = (seg_len + kSumParts - 1) / kSumParts;
  const int64_t i0 = pi * chunk, i1 = i0 + chunk < seg_len ? i0 + chunk : seg_len;
  const float* xs = x + (int64_t)seg * seg_len;
  float acc = 0.0f;
  for (int64_t i = i0 + threadIdx.x; i < i1; i += 256) acc += xs[i];
  acc = block_sum(acc);
  if (threadIdx.x == 0) part[seg * kSumParts + pi] = acc;
}

__global__ __launch_bounds__(256) void segment_total_kernel(const float* part, float* out) {
  const float v = (int)threadIdx.x < kSumParts ? part[blockIdx.x * kSumParts + threadIdx.x] : 0.0f;
  const float s = block_sum(v);
  if (threadIdx.x == 0) out[blockIdx.x] = s;
}

dim3 row_grid(const LayerArgs& a, int tpr) {
  const int64_t rows = (int64_t)a.B * a.H * a.T;
  const int64_t per = kLThreads / tpr;
  return dim3((unsigned)((rows + per - 1) / per));
}

// Instantiates kernel K for (TI, VEC) with TPR = the power of two at or above
// DP / VEC, at most 64 (with DP = 96 some threads of a row stay idle, which
// keeps a row's loads in one pass and the row groups aligned within a wave).
#define REL_LAYER_DISPATCH(K, TI, VEC, ...)                                                           \
  do {                                                                                                \
    int tpr_ = 4;                                                                                     \
    while (tpr_ < 64 && tpr_ * (VEC) < a.DP) tpr_ *= 2;                                               \
    if (tpr_ == 64)                                                                                   \
      hipLaunchKernelGGL((K<TI, VEC, 64>), row_grid(a, 64), dim3(kLThreads), 0, stream, __VA_ARGS__); \
    else if (tpr_ == 32)                                                                              \
      hipLaunchKernelGGL((K<TI, VEC, 32>), row_grid(a, 32), dim3(kLThreads), 0, stream, __VA_ARGS__); \
    else if (tpr_ == 16)                                                                              \
      hipLaunchKernelGGL((K<TI, VEC, 16>), row_grid(a, 16), dim3(kLThreads), 0, stream, __VA_ARGS__); \
    else if (tpr_ == 8)                                                                               \
      hipLaunchKernelGGL((K<TI, VEC, 8>), row_grid(a, 8), dim3(kLThreads), 0, stream, __VA_ARGS__);   \
    else                                                                                              \
      hipLaunchKernelGGL((K<TI, VEC, 4>), row_grid(a, 4), dim3(kLThreads), 0, stream, __VA_ARGS__);   \
  } while (0)

#define REL_LAYER_BY_TYPE(K, ...)                                         \
  do {                                                                    \
    if (dtype == 1) {                                                     \
      if (vec == 8) REL_LAYER_DISPATCH(K, bf16, 8, __VA_ARGS__);          \
      else if (vec == 2) REL_LAYER_DISPATCH(K, bf16, 2, __VA_ARGS__);     \
      else REL_LAYER_DISPATCH(K, bf16, 1, __VA_ARGS__);                   \
    } else {                                                              \
      if (vec == 4) REL_LAYER_DISPATCH(K, float, 4, __VA_ARGS__);         \
      else if (vec == 2) REL_LAYER_DISPATCH(K, float, 2, __VA_ARGS__);    \
      else REL_LAYER_DISPATCH(K, float, 1, __VA_ARGS__);                  \
    }                                                                     \
  } while (0)

bool vec_ok(int dtype, int vec) {
  return dtype == 1 ? (vec == 8 || vec == 2 || vec == 1) : (vec == 4 || vec == 2 || vec == 1);
}

}  // namespace

int layer_sum_parts() { return kSumParts; }

hipError_t launch_rope_table(float2* tab, int T, int D, double base, hipStream_t stream) {
  const int64_t n = (int64_t)T * (D / 2);
  hipLaunchKernelGGL(rope_table_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, stream, tab, T, D,
                     log(base));
  return hipGetLastError();
}

hipError_t launch_layer_prologue(const LayerArgs& a, int dtype, int vec, hipStream_t stream) {
  if (!vec_ok(dtype, vec)) return hipErrorInvalidValue;
  REL_LAYER_BY_TYPE(prologue_kernel, a);
  return hipGetLastError();
}

hipError_t launch_layer_repad(const void* src, void* dst, const LayerArgs& a, bool to_padded, int dtype,
                              int vec, hipStream_t stream) {
  if (!vec_ok(dtype, vec)) return hipErrorInvalidValue;
  const int tp = to_padded ? 1 : 0;
  REL_LAYER_BY_TYPE(repad_kernel, src, dst, a, tp);
  return hipGetLastError();
}

hipError_t launch_layer_epilogue(const LayerArgs& a, int dtype, int vec, hipStream_t stream) {
  if (!vec_ok(dtype, vec)) return hipErrorInvalidValue;
  REL_LAYER_BY_TYPE(epilogue_kernel, a);
  return hipGetLastError();
}

hipError_t launch_segment_sum(const float* x, int nseg, int64_t seg_len, float* part, float* out,
                              hipStream_t stream) {
  hipLaunchKernelGGL(segment_parts_kernel, dim3(kSumParts, (unsigned)nseg), dim3(256), 0, stream, x, seg_len,
                     part);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(segment_total_kernel, dim3((unsigned)nseg), dim3(256), 0, stream, (const float*)part, out);
  return hipGetLastError();
}

}  // namespace rel
