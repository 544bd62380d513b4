// Prologue and epilogue kernels of the layer entry points: RoPE on the two
// relation projections (Sec. 3.1), Givens head-pair mixing of the information
// state (eq. 4, App. A.2.2-A.2.3), zero padding of the head width to the width
// the fused kernels tile, and the backward of all three.
//
// Each of these is a pass over [B, H, T, D] rows whose cost is linear in T,
// against the T^2 work of the fused kernels, so the rotation, the mixing and the
// padding run once per row here instead of once per key tile inside the fused
// kernels. One wave handles one row (b, h, t); lanes run over channels.
//
// RoPE rotates channel d with channel d + D/2 by t * base^(-2d/D) (t zero-based),
// with cos and sin from a per-call [T, D/2] table evaluated in fp64.
// Givens mixing writes, for head h of pair p with partner head h':
//   I~_h = cos(theta_p) I_h + sigma_h sin(theta_p) I_h'
// where sigma_h = -1 for the pair's first head and +1 for its second.
#include "kernels.h"

namespace rel {

namespace {

constexpr int kLRows = 4;  // rows (waves) per workgroup

template <typename TI>
__device__ __forceinline__ float ld(const void* p, int64_t i) {
  return Elem<TI>::load((const TI*)p + i);
}

template <typename TI>
__device__ __forceinline__ void st(void* p, int64_t i, float x) {
  Elem<TI>::store((TI*)p + i, x);
}

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

__device__ __forceinline__ float wave_sum(float x) {
  for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o, 64);
  return x;
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

template <typename TI>
__global__ __launch_bounds__(64 * kLRows) void prologue_kernel(LayerArgs a) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * kLRows + (threadIdx.x >> 6);  // (b H + h) T + t
  if (row >= (int64_t)a.B * a.H * a.T) return;
  const int t = (int)(row % a.T);
  const int64_t n = row / a.T;
  const int h = (int)(n % a.H), b = (int)(n / a.H);
  const int64_t src = b * a.sb + h * a.sh + (int64_t)t * a.st;
  const int64_t dst = row * a.DP;
  const int half = a.D >> 1;
  int pair = 0, partner = h;
  float sigma = 0.0f, cth = 1.0f, sth = 0.0f;
  if (a.givens) {
    givens_role(h, a.H, a.givens, pair, partner, sigma);
    sincosf(a.theta[pair], &sth, &cth);
  }
  const int64_t srcp = b * a.sb + partner * a.sh + (int64_t)t * a.st;
  for (int c = lane; c < a.DP; c += 64) {
    float yq = 0.0f, yk = 0.0f, yv = 0.0f;
    if (c < a.D) {
      if (a.rope) {
        const int j = c < half ? c : c - half;
        const float2 cs = a.rope[(int64_t)t * half + j];
        const float q1 = ld<TI>(a.q, src + j), q2 = ld<TI>(a.q, src + j + half);
        const float k1 = ld<TI>(a.k, src + j), k2 = ld<TI>(a.k, src + j + half);
        yq = c < half ? q1 * cs.x - q2 * cs.y : q1 * cs.y + q2 * cs.x;
        yk = c < half ? k1 * cs.x - k2 * cs.y : k1 * cs.y + k2 * cs.x;
      } else {
        yq = ld<TI>(a.q, src + c);
        yk = ld<TI>(a.k, src + c);
      }
      yv = ld<TI>(a.v, src + c);
      if (a.givens) yv = cth * yv + sigma * sth * ld<TI>(a.v, srcp + c);
    }
    if (a.qr) {
      st<TI>(a.qr, dst + c, yq);
      st<TI>(a.kr, dst + c, yk);
    }
    if (a.vt) st<TI>(a.vt, dst + c, yv);
  }
}

// Copies rows between the caller's layout (true width D) and the contiguous
// padded layout (width DP): to_padded = 1 writes zeros in channels D .. DP-1.
template <typename TI>
__global__ __launch_bounds__(64 * kLRows) void repad_kernel(const void* src, void* dst, LayerArgs a,
                                                            int to_padded) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * kLRows + (threadIdx.x >> 6);
  if (row >= (int64_t)a.B * a.H * a.T) return;
  const int t = (int)(row % a.T);
  const int64_t n = row / a.T;
  const int h = (int)(n % a.H), b = (int)(n / a.H);
  const int64_t cl = b * a.sb + h * a.sh + (int64_t)t * a.st;
  const int64_t pd = row * a.DP;
  if (to_padded) {
    for (int c = lane; c < a.DP; c += 64) st<TI>(dst, pd + c, c < a.D ? ld<TI>(src, cl + c) : 0.0f);
  } else {
    for (int c = lane; c < a.D; c += 64) st<TI>(dst, cl + c, ld<TI>(src, pd + c));
  }
}

// Backward: gradients in the padded layout (gq, gk with respect to the rotated
// projections, gv with respect to I~) to the caller's tensors, and each row's
// term of dL/dtheta for the pair whose first head this row belongs to:
//   dL/dtheta_p += dI~_a . (-s I_a - c I_b) + dI~_b . (c I_a - s I_b).
template <typename TI>
__global__ __launch_bounds__(64 * kLRows) void epilogue_kernel(LayerArgs a) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * kLRows + (threadIdx.x >> 6);
  if (row >= (int64_t)a.B * a.H * a.T) return;
  const int t = (int)(row % a.T);
  const int64_t n = row / a.T;
  const int h = (int)(n % a.H), b = (int)(n / a.H);
  const int64_t cl = b * a.sb + h * a.sh + (int64_t)t * a.st;
  const int64_t pd = row * a.DP;
  const int half = a.D >> 1;
  int pair = 0, partner = h;
  float sigma = 0.0f, cth = 1.0f, sth = 0.0f;
  if (a.givens) {
    givens_role(h, a.H, a.givens, pair, partner, sigma);
    sincosf(a.theta[pair], &sth, &cth);
  }
  const int64_t pdp = (((int64_t)b * a.H + partner) * a.T + t) * a.DP;  // partner row, padded
  const int64_t clp = b * a.sb + partner * a.sh + (int64_t)t * a.st;    // partner row, caller
  float dth = 0.0f;
  for (int c = lane; c < a.D; c += 64) {
    if (a.gq) {
      float oq, ok;
      if (a.rope) {
        const int j = c < half ? c : c - half;
        const float2 cs = a.rope[(int64_t)t * half + j];
        const float q1 = ld<TI>(a.gq, pd + j), q2 = ld<TI>(a.gq, pd + j + half);
        const float k1 = ld<TI>(a.gk, pd + j), k2 = ld<TI>(a.gk, pd + j + half);
        oq = c < half ? q1 * cs.x + q2 * cs.y : -q1 * cs.y + q2 * cs.x;
        ok = c < half ? k1 * cs.x + k2 * cs.y : -k1 * cs.y + k2 * cs.x;
      } else {
        oq = ld<TI>(a.gq, pd + c);
        ok = ld<TI>(a.gk, pd + c);
      }
      st<TI>(a.dq, cl + c, oq);
      st<TI>(a.dk, cl + c, ok);
    }
    if (a.gv) {
      const float gh = ld<TI>(a.gv, pd + c);
      float ov = gh;
      if (a.givens) {
        const float gp = ld<TI>(a.gv, pdp + c);
        ov = cth * gh - sigma * sth * gp;
        if (sigma < 0.0f) {  // first head of the pair: h = a, partner = b
          const float va = ld<TI>(a.v, cl + c), vb = ld<TI>(a.v, clp + c);
          dth += gh * (-sth * va - cth * vb) + gp * (cth * va - sth * vb);
        }
      }
      st<TI>(a.dv, cl + c, ov);
    }
  }
  if (a.givens && sigma < 0.0f) {
    dth = wave_sum(dth);
    if (lane == 0) a.dth_rows[((int64_t)pair * a.B + b) * a.T + t] = dth;
  }
}

// out[s] = sum of segment s of x (segments of seg_len floats), one workgroup
// per segment, in a fixed order.
__global__ __launch_bounds__(256) void segment_sum_kernel(const float* x, int64_t seg_len, float* out) {
  __shared__ float sh[256];
  const float* xs = x + (int64_t)blockIdx.x * seg_len;
  float acc = 0.0f;
  for (int64_t i = threadIdx.x; i < seg_len; i += 256) acc += xs[i];
  sh[threadIdx.x] = acc;
  __syncthreads();
  for (int hh = 128; hh >= 1; hh >>= 1) {
    if ((int)threadIdx.x < hh) sh[threadIdx.x] += sh[threadIdx.x + hh];
    __syncthreads();
  }
  if (threadIdx.x == 0) out[blockIdx.x] = sh[0];
}

dim3 row_grid(const LayerArgs& a) {
  const int64_t rows = (int64_t)a.B * a.H * a.T;
  return dim3((unsigned)((rows + kLRows - 1) / kLRows));
}

}  // namespace

hipError_t launch_rope_table(float2* tab, int T, int D, double base, hipStream_t stream) {
  const int64_t n = (int64_t)T * (D / 2);
  hipLaunchKernelGGL(rope_table_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, stream, tab, T, D,
                     log(base));
  return hipGetLastError();
}

hipError_t launch_layer_prologue(const LayerArgs& a, int dtype, hipStream_t stream) {
  if (dtype == 1)
    hipLaunchKernelGGL(prologue_kernel<bf16>, row_grid(a), dim3(64 * kLRows), 0, stream, a);
  else
    hipLaunchKernelGGL(prologue_kernel<float>, row_grid(a), dim3(64 * kLRows), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_layer_repad(const void* src, void* dst, const LayerArgs& a, bool to_padded, int dtype,
                              hipStream_t stream) {
  if (dtype == 1)
    hipLaunchKernelGGL(repad_kernel<bf16>, row_grid(a), dim3(64 * kLRows), 0, stream, src, dst, a,
                       to_padded ? 1 : 0);
  else
    hipLaunchKernelGGL(repad_kernel<float>, row_grid(a), dim3(64 * kLRows), 0, stream, src, dst, a,
                       to_padded ? 1 : 0);
  return hipGetLastError();
}

hipError_t launch_layer_epilogue(const LayerArgs& a, int dtype, hipStream_t stream) {
  if (dtype == 1)
    hipLaunchKernelGGL(epilogue_kernel<bf16>, row_grid(a), dim3(64 * kLRows), 0, stream, a);
  else
    hipLaunchKernelGGL(epilogue_kernel<float>, row_grid(a), dim3(64 * kLRows), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_segment_sum(const float* x, int nseg, int64_t seg_len, float* out, hipStream_t stream) {
  hipLaunchKernelGGL(segment_sum_kernel, dim3((unsigned)nseg), dim3(256), 0, stream, x, seg_len, out);
  return hipGetLastError();
}

}  // namespace rel
