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
#include "lanes.h"

namespace rel {

namespace {

constexpr int kDT = 256;      // threads of the states kernel
constexpr int kSlice = 256;   // keys per workgroup in relation_decode
constexpr int kUnroll = 2;    // keys per lane group whose loads are in flight together

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

// The cache length of batch entry b, clamped to 1 .. Tmax so that every read
// stays inside the cache; the merge writes NaN for an entry outside that range.
__device__ __forceinline__ int clamp_len(const int32_t* lengths, int b, int Tmax) {
  const int n = lengths[b];
  return n < 1 ? 1 : (n > Tmax ? Tmax : n);
}
__device__ __forceinline__ bool len_valid(const int32_t* lengths, int b, int Tmax) {
  const int n = lengths[b];
  return n >= 1 && n <= Tmax;
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
  // kUnroll keys per lane group in flight: j = s0 + (kUnroll (it NW + w) + u) KPW + kg.
  // The loop runs on a wave-uniform base, so every lane reaches the shuffles.
  for (int base = s0 + kUnroll * w * KPW; base < s1; base += kUnroll * NW * KPW) {
    float kx[kUnroll][VEC], vx[kUnroll][VEC];
    bool ok[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
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
    for (int u = 0; u < kUnroll; ++u) {
      float d = 0.0f;
#pragma unroll
      for (int e = 0; e < VEC; ++e) d = __builtin_fmaf(q[e], kx[u][e], d);
      d = lane_group_sum<LPK>(d);
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

// One workgroup per (b, h) row: merge the row's a.nstates states, then Self
// and the count correction (eqs. 12-13) at i = the row's cache length. Lanes
// run over states and wave w over channels 32 w .. 32 w + 31, so the loads of
// all states are in flight at once; the lane sums then meet by shuffles.
template <typename TI>
__global__ __launch_bounds__(256) void decode_merge_kernel(DecodeArgs a) {
  __shared__ float zsh[128];
  __shared__ float lsh;
  const int n = blockIdx.x;  // b * H + h
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63;
  const int b = n / a.H, h = n % a.H;
  const int len = clamp_len(a.lengths, b, a.Tmax);
  const int64_t stride_s = (int64_t)a.B * a.H * (a.D + 2);
  const float* st0 = a.states + (int64_t)n * (a.D + 2);
  // the Self entry's reads first (the first wave), so that they overlap the states' reads
  const int64_t selfrow = (int64_t)b * a.sb + (int64_t)h * a.sh + (int64_t)(len - 1) * a.st;
  const TI* q = (const TI*)a.q + (int64_t)n * a.D;
  float d = 0.0f, vi0 = 0.0f, vi1 = 0.0f;
  if (w == 0) {
    if (lane < a.D) {
      d = Elem<TI>::load(q + lane) * Elem<TI>::load((const TI*)a.k + selfrow + lane);
      vi0 = Elem<TI>::load((const TI*)a.v + selfrow + lane);
    }
    if (lane + 64 < a.D) {
      d += Elem<TI>::load(q + lane + 64) * Elem<TI>::load((const TI*)a.k + selfrow + lane + 64);
      vi1 = Elem<TI>::load((const TI*)a.v + selfrow + lane + 64);
    }
  }
  float m = kNegInf;
  for (int s = lane; s < a.nstates; s += 64) m = fmaxf(m, st0[s * stride_s]);
  for (int o = 32; o >= 1; o >>= 1) m = fmaxf(m, __shfl_xor(m, o, 64));
  const int cb = 32 * w;
  if (cb < a.D) {  // wave-uniform
    float acc[32];
#pragma unroll
    for (int e = 0; e < 32; ++e) acc[e] = 0.0f;
    float l = 0.0f;
    for (int s = lane; s < a.nstates; s += 64) {
      const float* st = st0 + s * stride_s;
      const float ms = st[0];
      const float f = ms == kNegInf ? 0.0f : fast_exp2((ms - m) * kLog2e);
      l = __builtin_fmaf(st[1], f, l);
      const float2* zp = reinterpret_cast<const float2*>(st + 2 + cb);  // 8-byte aligned: D + 2 and cb even
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const float2 zz = zp[e];
        acc[2 * e] = __builtin_fmaf(zz.x, f, acc[2 * e]);
        acc[2 * e + 1] = __builtin_fmaf(zz.y, f, acc[2 * e + 1]);
      }
    }
#pragma unroll
    for (int e = 0; e < 32; ++e)
      for (int o = 32; o >= 1; o >>= 1) acc[e] += __shfl_xor(acc[e], o, 64);
    for (int o = 32; o >= 1; o >>= 1) l += __shfl_xor(l, o, 64);
    if (lane == 0) {
#pragma unroll
      for (int e = 0; e < 32; ++e) zsh[cb + e] = acc[e];
      if (w == 0) lsh = l;
    }
  }
  __syncthreads();
  if (w != 0) return;  // the first wave finishes the row
  const float l = lsh;
  const float z0 = lane < a.D ? zsh[lane] : 0.0f;
  const float z1 = lane + 64 < a.D ? zsh[lane + 64] : 0.0f;
  // Self: U_ii = scale q . k_i, S = sigmoid(U_ii / tau_S)
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
  // an entry whose cache length lies outside 1 .. Tmax gets NaN: the error is
  // visible in the output instead of a result at a clamped position
  const bool valid = len_valid(a.lengths, b, a.Tmax);
  const float nan = __builtin_nanf("");
  TI* o = (TI*)a.out + (int64_t)n * a.D;
  if (lane < a.D) Elem<TI>::store(o + lane, valid ? omg * vi0 + g * zr0 : nan);
  if (lane + 64 < a.D) Elem<TI>::store(o + lane + 64, valid ? omg * vi1 + g * zr1 : nan);
  if (lane == 0 && a.row_stat) a.row_stat[n] = valid ? lnZ + lam * ln_i : nan;
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
  const dim3 grid((unsigned)(a.B * a.H));
  if (dtype == 1)
    hipLaunchKernelGGL(decode_merge_kernel<bf16>, grid, dim3(256), 0, stream, a);
  else
    hipLaunchKernelGGL(decode_merge_kernel<float>, grid, dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace rel
