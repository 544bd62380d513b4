// Row kernels of the materialised baseline and of the allocation diagnostic.
//
// Materialised baseline: U = scale q k^T sits in HBM (rocBLAS); one wave per
// row i reads U_i, assembles R_i (eq. 2), normalises it
// (F_i = softmax(R_i), eq. 3) and writes F_i in the GEMM's operand type for
// the following o = F v GEMM, plus the optional fp32 R, F, pi (eq. 7) and the
// Self / Exchange masses (eq. 6).
//
// Materialised backward: from U and H = dO v^T in HBM, one wave per row
// forms F_i again, D_i, dR_i and dU_i (App. A.1.7) and writes dU_i and F_i in
// the GEMM operand type for the dq / dk / dv GEMMs, plus the row's dlambda term.
//
// Allocation diagnostic: pi_ij = exp(E_ij - L^E_i) for j < i (eq. 7), from q, k
// and the L^E written by the fused forward pass.
#include "kernels.h"

namespace rel {

namespace {

constexpr int kRT = 256;

__device__ __forceinline__ float silu(float u) { return u / (1.0f + expf(-u)); }

// The materialised row kernels give one wave to one row (four rows per
// workgroup) and keep nothing in LDS: a first pass over U_i (and H_i) gathers
// the row's softmax statistics with per-lane online (max, sum) pairs merged
// across the wave, a second pass reads the row again (from L2) and writes the
// T x T outputs. Rows are read with 16-byte loads when T % 4 == 0 (V = 4).
constexpr int kRowsPerBlock = 4;
constexpr int kNB = 4;  // chunks of a row loaded before any is used (loads in flight per lane)

// Hardware exp2 and reciprocal (about 1 ulp each) on the per-element path of
// the row kernels; the library expf and division cost about ten instructions each.
__device__ __forceinline__ float fexp(float x) { return fast_exp2(x * kLog2e); }
__device__ __forceinline__ float sigmoid(float u) { return fast_rcp(1.0f + fexp(-u)); }

// Merges per-lane (m, l[, d]) running statistics across the wave, where
// l = sum exp(r - m) and d = sum exp(r - m) h; an empty lane holds m = -inf, l = d = 0.
__device__ __forceinline__ void wave_merge(float& m, float& l, float& d) {
  for (int o = 32; o >= 1; o >>= 1) {
    const float mo = __shfl_xor(m, o, 64), lo = __shfl_xor(l, o, 64), dd = __shfl_xor(d, o, 64);
    const float mn = fmaxf(m, mo);
    const float a = m == kNegInf ? 0.0f : fexp(m - mn);
    const float b = mo == kNegInf ? 0.0f : fexp(mo - mn);
    l = l * a + lo * b;
    d = d * a + dd * b;
    m = mn;
  }
}

__device__ __forceinline__ float wave_sum(float x) {
  for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o, 64);
  return x;
}

template <int V>
__device__ __forceinline__ void load_row(const float* p, float (&x)[V]) {
  if constexpr (V == 4) {
    const float4 t = *reinterpret_cast<const float4*>(p);
    x[0] = t.x; x[1] = t.y; x[2] = t.z; x[3] = t.w;
  } else {
    x[0] = *p;
  }
}

template <typename TF, int V>
__device__ __forceinline__ void store_row(TF* p, const float (&x)[V]) {
  if constexpr (V == 4 && sizeof(TF) == 2) {
    typedef TF tf4 __attribute__((ext_vector_type(4)));
    tf4 o;
#pragma unroll
    for (int t = 0; t < 4; ++t) o[t] = (TF)x[t];
    *reinterpret_cast<tf4*>(p) = o;
  } else if constexpr (V == 4) {
    *reinterpret_cast<float4*>(p) = make_float4(x[0], x[1], x[2], x[3]);
  } else {
    Elem<TF>::store(p, x[0]);
  }
}

// Forward row i of one head: R_i (eq. 2) from U_i, F_i = softmax(R_i) (eq. 3)
// written in the GEMM operand type for o = F v, plus the optional fp32 R, F,
// pi (eq. 7) and the Self / Exchange masses (eq. 6).
template <typename TF, int V>
__global__ __launch_bounds__(64 * kRowsPerBlock) void materialized_row_kernel(RowArgs a, int64_t rows) {
  constexpr int kStep = 64 * V;  // elements of the row one wave covers per chunk
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * kRowsPerBlock + (threadIdx.x >> 6);  // n * T + i
  if (row >= rows) return;  // whole wave; the kernel has no barrier
  const int T = a.T;
  const int i = (int)(row % T);
  const float* U = a.U + row * (int64_t)T;
  const float lam_ln = *a.lambda * logf((float)(i + 1));
  const float S = sigmoid(U[i] * a.inv_tau);  // Self logit R_ii

  // Exchange statistics over j < i
  float m = kNegInf, l = 0.0f, unused = 0.0f;
  for (int jb = lane * V; jb < i; jb += kStep * kNB) {
    float ub[kNB][V];
#pragma unroll
    for (int c = 0; c < kNB; ++c)
      if (jb + c * kStep < i) load_row<V>(U + jb + c * kStep, ub[c]);
#pragma unroll
    for (int c = 0; c < kNB; ++c) {
    const int j0 = jb + c * kStep;
    if (j0 >= i) break;
    const float(&u)[V] = ub[c];
    float r[V];
    float mx = kNegInf;
#pragma unroll
    for (int t = 0; t < V; ++t) {
      r[t] = j0 + t < i ? u[t] * sigmoid(u[t]) - lam_ln : kNegInf;
      mx = fmaxf(mx, r[t]);
    }
    const float mn = fmaxf(m, mx);
    float acc = m == kNegInf ? 0.0f : l * fexp(m - mn);
#pragma unroll
    for (int t = 0; t < V; ++t) acc += fexp(r[t] - mn);
    l = acc;
    m = mn;
    }
  }
  wave_merge(m, l, unused);
  const float M = fmaxf(m, S);
  const float le = m == kNegInf ? 0.0f : l * fexp(m - M);  // Exchange part of the denominator
  const float inv = 1.0f / (le + fexp(S - M));
  const float fii = fexp(S - M) * inv;
  const float g = le * inv;
  const float inv_g = g > 0.0f ? 1.0f / g : 0.0f;

  TF* Fw = (TF*)a.Fw + row * (int64_t)T;
  float* Ro = a.R ? a.R + row * (int64_t)T : nullptr;
  float* Fo = a.F ? a.F + row * (int64_t)T : nullptr;
  float* Po = a.pi ? a.pi + row * (int64_t)T : nullptr;
  for (int jb = lane * V; jb < T; jb += kStep * kNB) {
    float ub[kNB][V];
#pragma unroll
    for (int c = 0; c < kNB; ++c)
      if (jb + c * kStep <= i) load_row<V>(U + jb + c * kStep, ub[c]);
#pragma unroll
    for (int c = 0; c < kNB; ++c) {
    const int j0 = jb + c * kStep;
    if (j0 >= T) break;
    const float(&u)[V] = ub[c];
    float f[V], r[V];
#pragma unroll
    for (int t = 0; t < V; ++t) {
      const int j = j0 + t;
      r[t] = kNegInf;
      f[t] = 0.0f;
      if (j < i) {
        r[t] = u[t] * sigmoid(u[t]) - lam_ln;
        f[t] = fexp(r[t] - M) * inv;
      } else if (j == i) {
        r[t] = S;
        f[t] = fii;
      }
    }
    store_row<TF, V>(Fw + j0, f);
    if (Ro || Fo || Po) {
#pragma unroll
      for (int t = 0; t < V; ++t) {
        const int j = j0 + t;
        if (Ro) Ro[j] = r[t];
        if (Fo) Fo[j] = f[t];
        if (Po) Po[j] = j < i ? f[t] * inv_g : 0.0f;
      }
    }
    }
  }
  if (lane == 0) {
    if (a.self_mass) a.self_mass[row] = fii;
    if (a.exch_mass) a.exch_mass[row] = g;
  }
}

// Backward row i of one head (App. A.1.7): F_i = softmax(R_i) again from U_i,
// then with H_i = dO_i v^T (from a GEMM)
//   D_i = sum_j F_ij H_ij,  dR_ij = F_ij (H_ij - D_i)            (j <= i)
//   dU_ij = dR_ij SiLU'(U_ij) for j < i,  SiLU'(u) = s(u) (1 + u (1 - s(u)))
//   dU_ii = dR_ii S_i (1 - S_i) / tau_S
//   dlambda_i = -ln i sum_{j<i} dR_ij                          (dR_ij/dlambda = -ln i)
// dU and F go out in the GEMM operand type for dq = s dU k, dk = s dU^T q, dv = F^T dO.
template <typename TF, int V>
__global__ __launch_bounds__(64 * kRowsPerBlock) void materialized_bwd_row_kernel(RowBwdArgs a, int64_t rows) {
  constexpr int kStep = 64 * V;
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * kRowsPerBlock + (threadIdx.x >> 6);  // n * T + i
  if (row >= rows) return;  // whole wave; the kernel has no barrier
  const int T = a.T;
  const int i = (int)(row % T);
  const float* U = a.U + row * (int64_t)T;
  const float* Hg = a.Hm + row * (int64_t)T;
  const float ln_i = logf((float)(i + 1));
  const float lam_ln = *a.lambda * ln_i;
  const float S = sigmoid(U[i] * a.inv_tau);
  const float Hii = Hg[i];

  // Exchange statistics over j < i: m, l = sum exp(R - m), d = sum exp(R - m) H
  float m = kNegInf, l = 0.0f, d = 0.0f;
  for (int jb = lane * V; jb < i; jb += kStep * kNB) {
    float ub[kNB][V], hb[kNB][V];
#pragma unroll
    for (int c = 0; c < kNB; ++c)
      if (jb + c * kStep < i) {
        load_row<V>(U + jb + c * kStep, ub[c]);
        load_row<V>(Hg + jb + c * kStep, hb[c]);
      }
#pragma unroll
    for (int c = 0; c < kNB; ++c) {
    const int j0 = jb + c * kStep;
    if (j0 >= i) break;
    const float(&u)[V] = ub[c];
    const float(&h)[V] = hb[c];
    float r[V];
    float mx = kNegInf;
#pragma unroll
    for (int t = 0; t < V; ++t) {
      r[t] = j0 + t < i ? u[t] * sigmoid(u[t]) - lam_ln : kNegInf;
      mx = fmaxf(mx, r[t]);
    }
    const float mn = fmaxf(m, mx);
    const float sc = m == kNegInf ? 0.0f : fexp(m - mn);
    float al = l * sc, ad = d * sc;
#pragma unroll
    for (int t = 0; t < V; ++t) {
      const float e = fexp(r[t] - mn);
      al += e;
      ad += j0 + t < i ? e * h[t] : 0.0f;
    }
    l = al;
    d = ad;
    m = mn;
    }
  }
  wave_merge(m, l, d);
  const float M = fmaxf(m, S);
  const float c = m == kNegInf ? 0.0f : fexp(m - M);
  const float es = fexp(S - M);
  const float inv = 1.0f / (l * c + es);
  const float fii = es * inv;
  const float Di = (d * c + es * Hii) * inv;

  TF* dUo = (TF*)a.dUw + row * (int64_t)T;
  TF* Fo = (TF*)a.Fw + row * (int64_t)T;
  float ex = 0.0f;  // sum_{j<i} dR_ij
  for (int jb = lane * V; jb < T; jb += kStep * kNB) {
    float ub[kNB][V], hb[kNB][V];
#pragma unroll
    for (int c = 0; c < kNB; ++c)
      if (jb + c * kStep <= i) {
        load_row<V>(U + jb + c * kStep, ub[c]);
        load_row<V>(Hg + jb + c * kStep, hb[c]);
      }
#pragma unroll
    for (int c = 0; c < kNB; ++c) {
    const int j0 = jb + c * kStep;
    if (j0 >= T) break;
    const float(&u)[V] = ub[c];
    const float(&h)[V] = hb[c];
    float f[V], du[V];
#pragma unroll
    for (int t = 0; t < V; ++t) {
      const int j = j0 + t;
      f[t] = 0.0f;
      du[t] = 0.0f;
      if (j < i) {
        const float s = sigmoid(u[t]);
        f[t] = fexp(u[t] * s - lam_ln - M) * inv;
        const float dr = f[t] * (h[t] - Di);
        du[t] = dr * s * (1.0f + u[t] * (1.0f - s));
        ex += dr;
      } else if (j == i) {
        f[t] = fii;
        du[t] = fii * (Hii - Di) * S * (1.0f - S) * a.inv_tau;
      }
    }
    store_row<TF, V>(Fo + j0, f);
    store_row<TF, V>(dUo + j0, du);
    }
  }
  ex = wave_sum(ex);
  if (lane == 0) a.dlam_row[row] = -ln_i * ex;
}

// Fixed-order sum of n floats in two launches: workgroup b sums the b-th
// contiguous chunk (each thread a strided part, then a tree), one workgroup
// then sums the partials in the same way. Run-to-run identical.
constexpr int kSumParts = 256;

__device__ __forceinline__ float block_tree_sum(float acc) {
  __shared__ float s[kRT];
  s[threadIdx.x] = acc;
  __syncthreads();
  for (int h = kRT / 2; h >= 1; h >>= 1) {
    if ((int)threadIdx.x < h) s[threadIdx.x] += s[threadIdx.x + h];
    __syncthreads();
  }
  return s[0];
}

__global__ __launch_bounds__(kRT) void sum_chunks_kernel(const float* x, int64_t n, int64_t chunk,
                                                         float* partial) {
  const int64_t b0 = (int64_t)blockIdx.x * chunk;
  const int64_t b1 = b0 + chunk < n ? b0 + chunk : n;
  float acc = 0.0f;
  for (int64_t i = b0 + threadIdx.x; i < b1; i += kRT) acc += x[i];
  acc = block_tree_sum(acc);
  if (threadIdx.x == 0) partial[blockIdx.x] = acc;
}

template <typename TI>
__global__ __launch_bounds__(kRT) void allocation_kernel(RowArgs a) {
  extern __shared__ float qrow[];  // D floats
  const int T = a.T, D = a.D;
  const int64_t row = blockIdx.x;
  const int64_t head = row / T;
  const int i = (int)(row % T);
  const int64_t hoff = (head / a.H) * a.sb + (head % a.H) * a.sh;
  const TI* q = (const TI*)a.q + hoff;
  const TI* k = (const TI*)a.k + hoff;
  for (int d = threadIdx.x; d < D; d += kRT) qrow[d] = Elem<TI>::load(q + (int64_t)i * a.st + d);
  __syncthreads();
  const float LE = a.exch_lse[row];
  float* P = a.pi + row * (int64_t)T;
  for (int j = threadIdx.x; j < T; j += kRT) {
    float p = 0.0f;
    if (j < i) {
      float acc = 0.0f;
      for (int d = 0; d < D; ++d) acc = __builtin_fmaf(qrow[d], Elem<TI>::load(k + (int64_t)j * a.st + d), acc);
      p = expf(silu(acc * a.scale) - LE);
    }
    P[j] = p;
  }
}

}  // namespace

hipError_t launch_materialized_rows(const RowArgs& a, int dtype, int N, hipStream_t stream) {
  const int64_t rows = (int64_t)N * a.T;
  const dim3 grid((unsigned)((rows + kRowsPerBlock - 1) / kRowsPerBlock)), block(64 * kRowsPerBlock);
  const bool v4 = a.T % 4 == 0;  // rows of U and F then start on 16- and 8-byte boundaries
  if (dtype == 1) {
    if (v4) hipLaunchKernelGGL((materialized_row_kernel<bf16, 4>), grid, block, 0, stream, a, rows);
    else hipLaunchKernelGGL((materialized_row_kernel<bf16, 1>), grid, block, 0, stream, a, rows);
  } else {
    if (v4) hipLaunchKernelGGL((materialized_row_kernel<float, 4>), grid, block, 0, stream, a, rows);
    else hipLaunchKernelGGL((materialized_row_kernel<float, 1>), grid, block, 0, stream, a, rows);
  }
  return hipGetLastError();
}

hipError_t launch_materialized_bwd_rows(const RowBwdArgs& a, int dtype, int N, hipStream_t stream) {
  const int64_t rows = (int64_t)N * a.T;
  const dim3 grid((unsigned)((rows + kRowsPerBlock - 1) / kRowsPerBlock)), block(64 * kRowsPerBlock);
  const bool v4 = a.T % 4 == 0;
  if (dtype == 1) {
    if (v4) hipLaunchKernelGGL((materialized_bwd_row_kernel<bf16, 4>), grid, block, 0, stream, a, rows);
    else hipLaunchKernelGGL((materialized_bwd_row_kernel<bf16, 1>), grid, block, 0, stream, a, rows);
  } else {
    if (v4) hipLaunchKernelGGL((materialized_bwd_row_kernel<float, 4>), grid, block, 0, stream, a, rows);
    else hipLaunchKernelGGL((materialized_bwd_row_kernel<float, 1>), grid, block, 0, stream, a, rows);
  }
  return hipGetLastError();
}

int sum_fixed_order_parts() { return kSumParts; }

hipError_t launch_sum_fixed_order(const float* x, int64_t n, float* partial, float* out, hipStream_t stream) {
  const int64_t chunk = (n + kSumParts - 1) / kSumParts;
  hipLaunchKernelGGL(sum_chunks_kernel, dim3(kSumParts), dim3(kRT), 0, stream, x, n, chunk > 0 ? chunk : 1,
                     partial);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(sum_chunks_kernel, dim3(1), dim3(kRT), 0, stream, (const float*)partial,
                     (int64_t)kSumParts, (int64_t)kSumParts, out);
  return hipGetLastError();
}

hipError_t launch_allocation(const RowArgs& a, int dtype, int N, hipStream_t stream) {
  const int64_t rows = (int64_t)N * a.T;
  const size_t shm = (size_t)a.D * sizeof(float);
  if (dtype == 1)
    hipLaunchKernelGGL(allocation_kernel<bf16>, dim3((unsigned)rows), dim3(kRT), shm, stream, a);
  else
    hipLaunchKernelGGL(allocation_kernel<float>, dim3((unsigned)rows), dim3(kRT), shm, stream, a);
  return hipGetLastError();
}

}  // namespace rel
