// Decode step of the causal Full Relation operator: the one new row of every
// (b, h) against a KV cache, with the count correction at the token's absolute
// position i (eq. 2 with i = the cache length).
//
// The row is read-bound: every historical key and value is read once and used
// for one dot product and one weighted add. The history is split into slices
// of kSlice keys, one workgroup each, so that the chip has enough independent
// reads in flight; a workgroup leaves the Exchange scan state (m, l, z) of its
// slice (eq. 11). The merge kernel rescales the states of a row to their common
// maximum, adds them, and applies the epilogue of eqs. 12-13 with the Self
// entry (the token's own key and value, the last valid cache entry). The same
// merge serves a cache split over devices: each holds states of its shard.
//
// In the states kernel LPK lanes share one key: lane c of the group holds VEC
// channels of q (16 bytes of bf16 or fp32) and reads the same channels of the
// key and value rows; the dot product is finished by shuffles inside the group.
// Every lane group keeps its own running (m, l) and VEC channels of z, and the
// groups of a workgroup are merged at the end.
#include "kernels.h"

namespace rel {

namespace {

constexpr int kDT = 256;      // threads of the states kernel
constexpr int kSlice = 256;   // keys per workgroup in relation_decode

template <typename TI, int VEC>
struct Row;

template <>
struct Row<bf16, 8> {
  static __device__ __forceinline__ void load(const bf16* p, float (&x)[8]) {
    const uintx4 u = *reinterpret_cast<const uintx4*>(p);
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      x[2 * t] = bf16_lo(u[t]);
      x[2 * t + 1] = bf16_hi(u[t]);
    }
  }
};

template <>
struct Row<float, 4> {
  static __device__ __forceinline__ void load(const float* p, float (&x)[4]) {
    const float4 u = *reinterpret_cast<const float4*>(p);
    x[0] = u.x; x[1] = u.y; x[2] = u.z; x[3] = u.w;
  }
};

__device__ __forceinline__ float sigm(float x) { return fast_rcp(1.0f + fast_exp2(-x * kLog2e)); }

__device__ __forceinline__ int clamp_len(const int32_t* lengths, int b, int Tmax) {
  const int n = lengths[b];
  return n < 1 ? 1 : (n > Tmax ? Tmax : n);
}

// Merges state (mo, lo, zo) into (m, l, z); an empty state has m = -inf, l = 0.
template <int VEC>
__device__ __forceinline__ void merge_into(float& m, float& l, float (&z)[VEC], float mo, float lo,
                                           const float (&zo)[VEC]) {
  const float mn = fmaxf(m, mo);
  const float a = m == kNegInf ? 0.0f : fast_exp2((m - mn) * kLog2e);
  const float b = mo == kNegInf ? 0.0f : fast_exp2((mo - mn) * kLog2e);
  l = l * a + lo * b;
#pragma unroll
  for (int e = 0; e < VEC; ++e) z[e] = z[e] * a + zo[e] * b;
  m = mn;
}

// Exchange state of keys [j0, j1) of one (b, h) row, split into a.nsplit slices
// (grid: nsplit x B*H); keys at or after the row's own entry are never read.
template <typename TI, int VEC, int LPK>
__global__ __launch_bounds__(kDT) void decode_states_kernel(DecodeArgs a) {
  constexpr int KPW = 64 / LPK;          // keys per wave and step
  constexpr int NW = kDT / 64;
  __shared__ float red[NW][2 + 128];
  const int slice = blockIdx.x;
  const int n = blockIdx.y;              // b * H + h
  const int b = n / a.H, h = n % a.H;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int c = lane % LPK, kg = lane / LPK;
  const int c0 = c * VEC;
  const bool chan = c0 < a.D;
  const int len = clamp_len(a.lengths, b, a.Tmax);
  const int hist_end = min(a.key1, len - 1);      // Exchange keys only: j < i - 1 (zero-based)
  const int span = a.key1 - a.key0;
  const int per = (span + a.nsplit - 1) / a.nsplit;
  const int s0 = a.key0 + slice * per;
  const int s1 = min(s0 + per, hist_end);

  float q[VEC];
  const TI* qrow = (const TI*)a.q + (int64_t)n * a.D;
#pragma unroll
  for (int e = 0; e < VEC; ++e) q[e] = 0.0f;
  if (chan) Row<TI, VEC>::load(qrow + c0, q);
  const int64_t hoff = (int64_t)b * a.sb + (int64_t)h * a.sh;
  const TI* K = (const TI*)a.k + hoff;
  const TI* V = (const TI*)a.v + hoff;

  float m = kNegInf, l = 0.0f, z[VEC];
#pragma unroll
  for (int e = 0; e < VEC; ++e) z[e] = 0.0f;
  // two keys per lane group in flight: j = s0 + (2 it NW + 2 w + u) KPW + kg.
  // The loop runs on a wave-uniform base, so every lane reaches the shuffles.
  for (int base = s0 + 2 * w * KPW; base < s1; base += 2 * NW * KPW) {
    float kx[2][VEC], vx[2][VEC];
    bool ok[2];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int j = base + u * KPW + kg;
      ok[u] = j < s1;
#pragma unroll
      for (int e = 0; e < VEC; ++e) kx[u][e] = vx[u][e] = 0.0f;
      if (ok[u] && chan) {
        Row<TI, VEC>::load(K + (int64_t)j * a.st + c0, kx[u]);
        Row<TI, VEC>::load(V + (int64_t)j * a.st + c0, vx[u]);
      }
    }
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      float d = 0.0f;
#pragma unroll
      for (int e = 0; e < VEC; ++e) d = __builtin_fmaf(q[e], kx[u][e], d);
#pragma unroll
      for (int o = LPK / 2; o >= 1; o >>= 1) d += __shfl_xor(d, o, 64);
      if (ok[u]) {
        const float uu = d * a.scale;
        const float E = uu * sigm(uu);             // Exchange map, eq. (2)
        const float mn = fmaxf(m, E);
        const float cr = m == kNegInf ? 0.0f : fast_exp2((m - mn) * kLog2e);
        const float p = fast_exp2((E - mn) * kLog2e);
        l = l * cr + p;
#pragma unroll
        for (int e = 0; e < VEC; ++e) z[e] = __builtin_fmaf(p, vx[u][e], z[e] * cr);
        m = mn;
      }
    }
  }
  // merge the lane groups of the wave (lanes with equal c hold the same channels)
#pragma unroll
  for (int o = LPK; o < 64; o <<= 1) {
    float zo[VEC];
    const float mo = __shfl_xor(m, o, 64), lo = __shfl_xor(l, o, 64);
#pragma unroll
    for (int e = 0; e < VEC; ++e) zo[e] = __shfl_xor(z[e], o, 64);
    merge_into<VEC>(m, l, z, mo, lo, zo);
  }
  // then the waves, in a fixed order
  if (kg == 0) {
    if (c == 0) {
      red[w][0] = m;
      red[w][1] = l;
    }
    if (chan) {
#pragma unroll
      for (int e = 0; e < VEC; ++e) red[w][2 + c0 + e] = z[e];
    }
  }
  __syncthreads();
  if (w == 0 && kg == 0) {
    for (int ow = 1; ow < NW; ++ow) {
      float zo[VEC];
#pragma unroll
      for (int e = 0; e < VEC; ++e) zo[e] = chan ? red[ow][2 + c0 + e] : 0.0f;
      merge_into<VEC>(m, l, z, red[ow][0], red[ow][1], zo);
    }
    float* st = a.states + ((int64_t)slice * a.B * a.H + n) * (a.D + 2);
    if (c == 0) {
      st[0] = m;
      st[1] = l;
    }
    if (chan) {
#pragma unroll
      for (int e = 0; e < VEC; ++e) st[2 + c0 + e] = z[e];
    }
  }
}

// One wave per (b, h) row: merge the row's a.nstates states, then Self and the
// count correction (eqs. 12-13) at i = the row's cache length.
template <typename TI>
__global__ __launch_bounds__(256) void decode_merge_kernel(DecodeArgs a) {
  const int64_t n = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (n >= (int64_t)a.B * a.H) return;  // whole wave
  const int b = (int)(n / a.H), h = (int)(n % a.H);
  const int len = clamp_len(a.lengths, b, a.Tmax);
  const int64_t NS = (int64_t)a.B * a.H;
  const int64_t selfrow = (int64_t)b * a.sb + (int64_t)h * a.sh + (int64_t)(len - 1) * a.st;
  const TI* q = (const TI*)a.q + n * a.D;
  // merged Exchange state; lanes hold channels lane and lane + 64
  float m = kNegInf;
  for (int s = 0; s < a.nstates; ++s) m = fmaxf(m, a.states[(s * NS + n) * (a.D + 2)]);
  float l = 0.0f, z0 = 0.0f, z1 = 0.0f;
  for (int s = 0; s < a.nstates; ++s) {
    const float* st = a.states + (s * NS + n) * (a.D + 2);
    const float ms = st[0];
    if (ms == kNegInf) continue;
    const float f = fast_exp2((ms - m) * kLog2e);
    l += st[1] * f;
    if (lane < a.D) z0 += st[2 + lane] * f;
    if (lane + 64 < a.D) z1 += st[2 + lane + 64] * f;
  }
  // Self: U_ii = scale q . k_i, S = sigmoid(U_ii / tau_S)
  float d = 0.0f;
  if (lane < a.D) d = Elem<TI>::load(q + lane) * Elem<TI>::load((const TI*)a.k + selfrow + lane);
  if (lane + 64 < a.D) d += Elem<TI>::load(q + lane + 64) * Elem<TI>::load((const TI*)a.k + selfrow + lane + 64);
  for (int o = 32; o >= 1; o >>= 1) d += __shfl_xor(d, o, 64);
  const float S = 1.0f / (1.0f + expf(-d * a.scale * a.inv_tau));
  const float ln_i = logf((float)len);
  const float lam = *a.lambda;
  float g = 0.0f, omg = 1.0f, zr0 = 0.0f, zr1 = 0.0f, lnZ = S;
  if (l > 0.0f) {
    const float A = m + logf(l) - lam * ln_i;       // A_i = L^E_i - lambda ln i (eq. 5)
    g = 1.0f / (1.0f + expf(S - A));                // g = sigmoid(A - S)
    omg = 1.0f / (1.0f + expf(A - S));              // 1 - g = sigmoid(S - A)
    const float il = 1.0f / l;
    zr0 = z0 * il;
    zr1 = z1 * il;
    lnZ = fmaxf(S, A) + log1pf(expf(-fabsf(S - A)));
  }
  TI* o = (TI*)a.out + n * a.D;
  if (lane < a.D) {
    const float vi = Elem<TI>::load((const TI*)a.v + selfrow + lane);
    Elem<TI>::store(o + lane, omg * vi + g * zr0);
  }
  if (lane + 64 < a.D) {
    const float vi = Elem<TI>::load((const TI*)a.v + selfrow + lane + 64);
    Elem<TI>::store(o + lane + 64, omg * vi + g * zr1);
  }
  if (lane == 0 && a.row_stat) a.row_stat[n] = lnZ + lam * ln_i;
}

template <typename TI, int VEC>
hipError_t launch_states_t(const DecodeArgs& a, hipStream_t stream) {
  const dim3 grid((unsigned)a.nsplit, (unsigned)(a.B * a.H));
  const int lanes = (a.D + VEC - 1) / VEC;
  if (lanes <= 4)
    hipLaunchKernelGGL((decode_states_kernel<TI, VEC, 4>), grid, dim3(kDT), 0, stream, a);
  else if (lanes <= 8)
    hipLaunchKernelGGL((decode_states_kernel<TI, VEC, 8>), grid, dim3(kDT), 0, stream, a);
  else if (lanes <= 16)
    hipLaunchKernelGGL((decode_states_kernel<TI, VEC, 16>), grid, dim3(kDT), 0, stream, a);
  else
    hipLaunchKernelGGL((decode_states_kernel<TI, VEC, 32>), grid, dim3(kDT), 0, stream, a);
  return hipGetLastError();
}

}  // namespace

int decode_slice_keys() { return kSlice; }

hipError_t launch_decode_states(const DecodeArgs& a, int dtype, hipStream_t stream) {
  return dtype == 1 ? launch_states_t<bf16, 8>(a, stream) : launch_states_t<float, 4>(a, stream);
}

hipError_t launch_decode_merge(const DecodeArgs& a, int dtype, hipStream_t stream) {
  const dim3 grid((unsigned)((a.B * a.H + 3) / 4));
  if (dtype == 1)
    hipLaunchKernelGGL(decode_merge_kernel<bf16>, grid, dim3(256), 0, stream, a);
  else
    hipLaunchKernelGGL(decode_merge_kernel<float>, grid, dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace rel
