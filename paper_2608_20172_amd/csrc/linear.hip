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
// Three launches: per chunk the state contribution (dC, gamma = e^{b_last});
// per head the scan over chunks (the state entering every chunk); per chunk the
// output. All arithmetic is fp32 on the vector units.
#include "kernels.h"

namespace rel {

namespace {

constexpr int kL = 64;      // tokens per chunk
constexpr int kLT = 256;    // threads per workgroup

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

// Loads the chunk into LDS as fp32 and forms qt = S ^p1, kt = S ^p2 (rows past
// the sequence are zero), v, and b = running sum of g (zero g past the end, so
// b stays at its last value). One wave per row for the norms and S.
template <typename TI, int D>
__device__ __forceinline__ void load_chunk(const LinearArgs& a, const ChunkPos& p, float (*qt)[D], float (*kt)[D],
                                           float (*vv)[D], float (*bb)[D], float* Srow) {
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63;
  const int b = p.n / a.H, h = p.n % a.H;
  const int64_t hoff = (int64_t)b * a.sb + (int64_t)h * a.sh;
  const TI* P1 = (const TI*)a.p1 + hoff;
  const TI* P2 = (const TI*)a.p2 + hoff;
  const TI* V = (const TI*)a.v + hoff;
  const float* G = a.g + (int64_t)p.n * a.T * D;
  for (int r = w; r < kL; r += kLT / 64) {
    const bool ok = r < p.len;
    const int64_t row = (int64_t)(p.t0 + r);
    float x1[2] = {0.0f, 0.0f}, x2[2] = {0.0f, 0.0f};
    float s11 = 0.0f, s22 = 0.0f, s12 = 0.0f;
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int d = lane + 64 * u;
      if (d < D) {
        float vx = 0.0f, gx = 0.0f;
        if (ok) {
          x1[u] = Elem<TI>::load(P1 + row * a.st + d);
          x2[u] = Elem<TI>::load(P2 + row * a.st + d);
          vx = Elem<TI>::load(V + row * a.st + d);
          gx = G[row * D + d];
        }
        vv[r][d] = vx;
        bb[r][d] = gx;
        s11 += x1[u] * x1[u];
        s22 += x2[u] * x2[u];
        s12 += x1[u] * x2[u];
      }
    }
    for (int o = 32; o >= 1; o >>= 1) {
      s11 += __shfl_xor(s11, o, 64);
      s22 += __shfl_xor(s22, o, 64);
      s12 += __shfl_xor(s12, o, 64);
    }
    const float S = ok ? 1.0f / (1.0f + expf(-s12 * a.scale * a.inv_tau)) : 0.0f;
    const float i1 = ok && s11 > 0.0f ? S * rsqrtf(s11) : 0.0f;
    const float i2 = ok && s22 > 0.0f ? S * rsqrtf(s22) : 0.0f;
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int d = lane + 64 * u;
      if (d < D) {
        qt[r][d] = x1[u] * i1;
        kt[r][d] = x2[u] * i2;
      }
    }
    if (lane == 0) Srow[r] = S;
  }
  __syncthreads();
  if (tid < D) {  // running sum of g down the chunk, one channel per thread
    float acc = 0.0f;
    for (int r = 0; r < kL; ++r) {
      acc += bb[r][tid];
      bb[r][tid] = acc;
    }
  }
  __syncthreads();
}

// Per chunk: dC[a][e] = sum_j kt_{j,a} e^{b_last,a - b_j,a} v_{j,e}, gamma_a = e^{b_last,a}.
template <typename TI, int D>
__global__ __launch_bounds__(kLT) void linear_state_kernel(LinearArgs a) {
  __shared__ float qt[kL][D], kt[kL][D], vv[kL][D], bb[kL][D];
  __shared__ float Srow[kL];
  const ChunkPos p = chunk_pos(a);
  load_chunk<TI, D>(a, p, qt, kt, vv, bb, Srow);
  const int tid = threadIdx.x;
  // kt <- kt e^{b_last - b}
  for (int i = tid; i < kL * D; i += kLT) {
    const int r = i / D, d = i % D;
    kt[r][d] *= fast_exp2((bb[kL - 1][d] - bb[r][d]) * kLog2e);
  }
  __syncthreads();
  const int64_t base = ((int64_t)p.n * a.nchunks + p.c);
  if (tid < D) a.gamma[base * D + tid] = fast_exp2(bb[kL - 1][tid] * kLog2e);
  // thread tile: TA rows a x TE columns e of dC
  constexpr int TE = D <= 64 ? 4 : 8;
  constexpr int TA = D * D / (kLT * TE);
  constexpr int NE = D / TE;
  const int a0 = (tid / NE) * TA, e0 = (tid % NE) * TE;
  float acc[TA][TE];
#pragma unroll
  for (int i = 0; i < TA; ++i)
#pragma unroll
    for (int j = 0; j < TE; ++j) acc[i][j] = 0.0f;
  for (int r = 0; r < kL; ++r) {
    float kr[TA], vr[TE];
#pragma unroll
    for (int i = 0; i < TA; ++i) kr[i] = kt[r][a0 + i];
#pragma unroll
    for (int j = 0; j < TE; ++j) vr[j] = vv[r][e0 + j];
#pragma unroll
    for (int i = 0; i < TA; ++i)
#pragma unroll
      for (int j = 0; j < TE; ++j) acc[i][j] = __builtin_fmaf(kr[i], vr[j], acc[i][j]);
  }
  float* dC = a.dstate + base * D * D;
#pragma unroll
  for (int i = 0; i < TA; ++i)
#pragma unroll
    for (int j = 0; j < TE; ++j) dC[(a0 + i) * D + e0 + j] = acc[i][j];
}

// Per head and state entry: C entering chunk c, C_0 = 0, C_{c+1} = gamma_c C_c + dC_c.
__global__ __launch_bounds__(256) void linear_scan_kernel(LinearArgs a) {
  const int D = a.D;
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (int64_t)D * D) return;
  const int n = blockIdx.y;
  const int ar = (int)(idx / D);
  float C = 0.0f;
  for (int c = 0; c < a.nchunks; ++c) {
    const int64_t base = (int64_t)n * a.nchunks + c;
    a.cprev[base * D * D + idx] = C;
    C = a.gamma[base * D + ar] * C + a.dstate[base * D * D + idx];
  }
  if (a.state_out) a.state_out[(int64_t)n * D * D + idx] = C;
}

// Per chunk: Y_t = v_t + intra + inter (see the top of the file).
template <typename TI, int D>
__global__ __launch_bounds__(kLT) void linear_out_kernel(LinearArgs a) {
  __shared__ float qt[kL][D], kt[kL][D], vv[kL][D], bb[kL][D];
  __shared__ float A[kL][kL + 1];
  __shared__ float Srow[kL];
  const ChunkPos p = chunk_pos(a);
  load_chunk<TI, D>(a, p, qt, kt, vv, bb, Srow);
  const int tid = threadIdx.x;
  // intra scores A[t][j], j < t: thread -> row t = tid / 4, columns j = tid % 4 + 4 m
  {
    const int t = tid >> 2, j0 = tid & 3;
    float acc[kL / 4];
#pragma unroll
    for (int m = 0; m < kL / 4; ++m) acc[m] = 0.0f;
    for (int d = 0; d < D; ++d) {
      const float qd = qt[t][d], bd = bb[t][d];
#pragma unroll
      for (int m = 0; m < kL / 4; ++m) {
        const int j = j0 + 4 * m;
        if (j < t) acc[m] = __builtin_fmaf(qd * kt[j][d], fast_exp2((bd - bb[j][d]) * kLog2e), acc[m]);
      }
    }
#pragma unroll
    for (int m = 0; m < kL / 4; ++m) A[t][j0 + 4 * m] = acc[m];
  }
  __syncthreads();
  // qt <- qt e^{b} (the inter read's query)
  for (int i = tid; i < kL * D; i += kLT) {
    const int r = i / D, d = i % D;
    qt[r][d] *= fast_exp2(bb[r][d] * kLog2e);
  }
  __syncthreads();
  // outputs: thread -> row t = tid / 4, channels e0 .. e0 + D/4
  constexpr int TE = D / 4;
  const int t = tid >> 2, e0 = (tid & 3) * TE;
  float acc[TE];
#pragma unroll
  for (int j = 0; j < TE; ++j) acc[j] = vv[t][e0 + j];
  for (int j = 0; j < t; ++j) {
    const float w = A[t][j];
#pragma unroll
    for (int e = 0; e < TE; ++e) acc[e] = __builtin_fmaf(w, vv[j][e0 + e], acc[e]);
  }
  const float* C0 = a.cprev + ((int64_t)p.n * a.nchunks + p.c) * D * D;
  for (int d = 0; d < D; ++d) {
    const float qd = qt[t][d];
    const float* crow = C0 + d * D + e0;
#pragma unroll
    for (int e = 0; e < TE; ++e) acc[e] = __builtin_fmaf(qd, crow[e], acc[e]);
  }
  if (t < p.len) {
    const int b = p.n / a.H, h = p.n % a.H;
    TI* Y = (TI*)a.out + (int64_t)b * a.sb + (int64_t)h * a.sh + (int64_t)(p.t0 + t) * a.st;
#pragma unroll
    for (int e = 0; e < TE; ++e) Elem<TI>::store(Y + e0 + e, acc[e]);
  }
}

template <typename TI, int D>
hipError_t launch_fwd_d(const LinearArgs& a, hipStream_t stream) {
  const dim3 grid((unsigned)a.nchunks, (unsigned)(a.B * a.H));
  hipLaunchKernelGGL((linear_state_kernel<TI, D>), grid, dim3(kLT), 0, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const dim3 sgrid((unsigned)((D * D + 255) / 256), (unsigned)(a.B * a.H));
  hipLaunchKernelGGL(linear_scan_kernel, sgrid, dim3(256), 0, stream, a);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((linear_out_kernel<TI, D>), grid, dim3(kLT), 0, stream, a);
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

int linear_chunk() { return kL; }

hipError_t launch_linear_fwd(const LinearArgs& a, int dtype, hipStream_t stream) {
  return dtype == 1 ? launch_fwd_t<bf16>(a, stream) : launch_fwd_t<float>(a, stream);
}

}  // namespace rel
