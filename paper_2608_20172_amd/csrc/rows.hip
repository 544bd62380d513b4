// Row kernels of the materialised baseline and of the allocation diagnostic.
//
// Materialised baseline: U = scale q k^T sits in HBM (rocBLAS); one workgroup
// per row i reads U_i into LDS, assembles R_i (eq. 2), normalises it
// (F_i = softmax(R_i), eq. 3) and writes F_i in the GEMM's operand type for
// the following o = F v GEMM, plus the optional fp32 R, F, pi (eq. 7) and the
// Self / Exchange masses (eq. 6).
//
// Materialised backward: from U and H = dO v^T in HBM, one workgroup per row
// forms F_i again, D_i, dR_i and dU_i (App. A.1.7) and writes dU_i and F_i in
// the GEMM operand type for the dq / dk / dv GEMMs, plus the row's dlambda term.
//
// Allocation diagnostic: pi_ij = exp(E_ij - L^E_i) for j < i (eq. 7), from q, k
// and the L^E written by the fused forward pass.
#include "kernels.h"

namespace rel {

namespace {

constexpr int kRT = 256;

__device__ __forceinline__ float block_reduce_max(float x, float* s) {
  for (int o = 32; o >= 1; o >>= 1) x = fmaxf(x, __shfl_xor(x, o, 64));
  const int w = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) s[w] = x;
  __syncthreads();
  float r = s[0];
  for (int i = 1; i < kRT / 64; ++i) r = fmaxf(r, s[i]);
  return r;
}

__device__ __forceinline__ float block_reduce_sum(float x, float* s) {
  for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o, 64);
  const int w = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) s[w] = x;
  __syncthreads();
  float r = 0.0f;
  for (int i = 0; i < kRT / 64; ++i) r += s[i];
  return r;
}

__device__ __forceinline__ float silu(float u) { return u / (1.0f + expf(-u)); }

template <typename TF>
__global__ __launch_bounds__(kRT) void materialized_row_kernel(RowArgs a) {
  extern __shared__ float Rrow[];  // T floats
  __shared__ float red[kRT / 64];
  const int T = a.T;
  const int64_t row = blockIdx.x;  // n * T + i
  const int i = (int)(row % T);
  const float* U = a.U + row * (int64_t)T;
  const float lam = *a.lambda;
  const float ln_i = logf((float)(i + 1));

  // R_i: Self on the diagonal, count-corrected Exchange before it (eq. 2)
  float mx = kNegInf;
  for (int j = threadIdx.x; j <= i; j += kRT) {
    const float u = U[j];
    const float r = (j == i) ? 1.0f / (1.0f + expf(-u * a.inv_tau)) : silu(u) - lam * ln_i;
    Rrow[j] = r;
    mx = fmaxf(mx, r);
  }
  mx = block_reduce_max(mx, red);
  float sum = 0.0f;
  for (int j = threadIdx.x; j <= i; j += kRT) sum += expf(Rrow[j] - mx);
  sum = block_reduce_sum(sum, red);
  const float inv = 1.0f / sum;
  // g_i = sum_{j<i} F_ij, and F_ii
  float ex = 0.0f;
  for (int j = threadIdx.x; j < i; j += kRT) ex += expf(Rrow[j] - mx) * inv;
  ex = block_reduce_sum(ex, red);
  const float fii = expf(Rrow[i] - mx) * inv;
  TF* Fw = (TF*)a.Fw + row * (int64_t)T;
  float* Ro = a.R ? a.R + row * (int64_t)T : nullptr;
  float* Fo = a.F ? a.F + row * (int64_t)T : nullptr;
  float* Po = a.pi ? a.pi + row * (int64_t)T : nullptr;
  const float inv_g = ex > 0.0f ? 1.0f / ex : 0.0f;
  for (int j = threadIdx.x; j < T; j += kRT) {
    const float f = j <= i ? expf(Rrow[j] - mx) * inv : 0.0f;
    Elem<TF>::store(Fw + j, f);
    if (Ro) Ro[j] = j <= i ? Rrow[j] : kNegInf;
    if (Fo) Fo[j] = f;
    if (Po) Po[j] = j < i ? f * inv_g : 0.0f;
  }
  if (threadIdx.x == 0) {
    if (a.self_mass) a.self_mass[row] = fii;
    if (a.exch_mass) a.exch_mass[row] = ex;
  }
}

// Materialised backward, row i of one head (App. A.1.7): R_i and F_i = softmax(R_i)
// again from U_i, then with H_i = dO_i v^T (from a GEMM)
//   D_i = sum_j F_ij H_ij,  dR_ij = F_ij (H_ij - D_i)            (j <= i)
//   dU_ij = dR_ij SiLU'(U_ij) for j < i,  SiLU'(u) = s(u) (1 + u (1 - s(u)))
//   dU_ii = dR_ii S_i (1 - S_i) / tau_S
//   dlambda_i = -ln i sum_{j<i} dR_ij                          (dR_ij/dlambda = -ln i)
// dU and F go out in the GEMM operand type for dq = s dU k, dk = s dU^T q, dv = F^T dO.
template <typename TF>
__global__ __launch_bounds__(kRT) void materialized_bwd_row_kernel(RowBwdArgs a) {
  extern __shared__ float sh[];  // R_i then F_i (T floats), H_i (T floats)
  float* Rrow = sh;
  float* Hrow = sh + a.T;
  __shared__ float red[kRT / 64];
  const int T = a.T;
  const int64_t row = blockIdx.x;  // n * T + i
  const int i = (int)(row % T);
  const float* U = a.U + row * (int64_t)T;
  const float* Hg = a.Hm + row * (int64_t)T;
  const float lam = *a.lambda;
  const float ln_i = logf((float)(i + 1));

  float mx = kNegInf;
  for (int j = threadIdx.x; j <= i; j += kRT) {
    const float u = U[j];
    const float r = (j == i) ? 1.0f / (1.0f + expf(-u * a.inv_tau)) : silu(u) - lam * ln_i;
    Rrow[j] = r;
    Hrow[j] = Hg[j];
    mx = fmaxf(mx, r);
  }
  mx = block_reduce_max(mx, red);
  float sum = 0.0f;
  for (int j = threadIdx.x; j <= i; j += kRT) sum += expf(Rrow[j] - mx);
  sum = block_reduce_sum(sum, red);
  const float inv = 1.0f / sum;
  float dsum = 0.0f;  // D_i
  for (int j = threadIdx.x; j <= i; j += kRT) {
    const float f = expf(Rrow[j] - mx) * inv;
    Rrow[j] = f;
    dsum += f * Hrow[j];
  }
  const float Di = block_reduce_sum(dsum, red);
  TF* dUo = (TF*)a.dUw + row * (int64_t)T;
  TF* Fo = (TF*)a.Fw + row * (int64_t)T;
  float ex = 0.0f;  // sum_{j<i} dR_ij
  for (int j = threadIdx.x; j < T; j += kRT) {
    float f = 0.0f, du = 0.0f;
    if (j <= i) {
      f = Rrow[j];
      const float dr = f * (Hrow[j] - Di);
      const float u = U[j];
      if (j < i) {
        const float s = 1.0f / (1.0f + expf(-u));
        du = dr * s * (1.0f + u * (1.0f - s));
        ex += dr;
      } else {
        const float S = 1.0f / (1.0f + expf(-u * a.inv_tau));
        du = dr * S * (1.0f - S) * a.inv_tau;
      }
    }
    Elem<TF>::store(Fo + j, f);
    Elem<TF>::store(dUo + j, du);
  }
  ex = block_reduce_sum(ex, red);
  if (threadIdx.x == 0) a.dlam_row[row] = -ln_i * ex;
}

// Sum of n floats in one fixed order (one workgroup): run-to-run identical.
__global__ __launch_bounds__(kRT) void sum_fixed_order_kernel(const float* x, int64_t n, float* out) {
  __shared__ float s[kRT];
  float acc = 0.0f;
  for (int64_t i = threadIdx.x; i < n; i += kRT) acc += x[i];
  s[threadIdx.x] = acc;
  __syncthreads();
  for (int h = kRT / 2; h >= 1; h >>= 1) {
    if ((int)threadIdx.x < h) s[threadIdx.x] += s[threadIdx.x + h];
    __syncthreads();
  }
  if (threadIdx.x == 0) *out = s[0];
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
  const size_t shm = (size_t)a.T * sizeof(float);
  if (shm > 159 * 1024) return hipErrorInvalidValue;  // plus the static reduction buffer
  if (dtype == 1) {
    hipError_t e = hipFuncSetAttribute((const void*)materialized_row_kernel<bf16>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)shm);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(materialized_row_kernel<bf16>, dim3((unsigned)rows), dim3(kRT), shm, stream, a);
  } else {
    hipError_t e = hipFuncSetAttribute((const void*)materialized_row_kernel<float>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)shm);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(materialized_row_kernel<float>, dim3((unsigned)rows), dim3(kRT), shm, stream, a);
  }
  return hipGetLastError();
}

hipError_t launch_materialized_bwd_rows(const RowBwdArgs& a, int dtype, int N, hipStream_t stream) {
  const int64_t rows = (int64_t)N * a.T;
  const size_t shm = 2 * (size_t)a.T * sizeof(float);
  if (shm > 159 * 1024) return hipErrorInvalidValue;  // plus the static reduction buffer
  if (dtype == 1) {
    hipError_t e = hipFuncSetAttribute((const void*)materialized_bwd_row_kernel<bf16>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)shm);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(materialized_bwd_row_kernel<bf16>, dim3((unsigned)rows), dim3(kRT), shm, stream, a);
  } else {
    hipError_t e = hipFuncSetAttribute((const void*)materialized_bwd_row_kernel<float>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)shm);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(materialized_bwd_row_kernel<float>, dim3((unsigned)rows), dim3(kRT), shm, stream, a);
  }
  return hipGetLastError();
}

hipError_t launch_sum_fixed_order(const float* x, int64_t n, float* out, hipStream_t stream) {
  hipLaunchKernelGGL(sum_fixed_order_kernel, dim3(1), dim3(kRT), 0, stream, x, n, out);
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
