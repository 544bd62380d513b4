// Device-side helpers shared by the Relation kernels (gfx950 / CDNA4 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace rel {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef short shortx4 __attribute__((ext_vector_type(4)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef float floatx2 __attribute__((ext_vector_type(2)));
typedef unsigned int uintx4 __attribute__((ext_vector_type(4)));
typedef unsigned int uintx2 __attribute__((ext_vector_type(2)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr float kNegInf = -__builtin_inff();

// ---------------------------------------------------------------------------
// Matrix cores.
// 32x32x16 bf16: A lane l holds A[l%32][8*(l/32) .. +7], B lane l holds
// B[8*(l/32) .. +7][l%32]; accumulator register r of lane l is
// C[8*(r/4) + 4*(l/32) + r%4][l%32].
// 32x32x2 f32: A lane l holds A[l%32][l/32], B lane l holds B[l/32][l%32];
// same accumulator layout.
// ---------------------------------------------------------------------------
__device__ __forceinline__ floatx16 mfma32(const bf16x8& a, const bf16x8& b, const floatx16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ floatx16 mfma32f(float a, float b, const floatx16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
}

// Row of accumulator register r for lane group g (= lane / 32) in a 32x32 block.
__device__ __forceinline__ constexpr int acc_row(int r, int g) { return 8 * (r >> 2) + 4 * g + (r & 3); }

// ---------------------------------------------------------------------------
// LDS transpose read (ds_read_b64_tr_b16). Within every 16-lane group, source
// lane a supplies the address of four consecutive 16-bit elements M[a][0..3];
// lane i receives element e = M[4e + i/4][i%4]. If lanes 4e..4e+3 point at row
// e of a row-major tile, at columns c0 + 4*(a%4), lane i receives column c0 + i
// of rows 0..3.
// ---------------------------------------------------------------------------
typedef __attribute__((address_space(3))) shortx4 lds_shortx4;
__device__ __forceinline__ uintx2 lds_read_tr16(const void* lds_ptr) {
  return __builtin_bit_cast(uintx2, __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_shortx4*)(lds_ptr)));
}
// An MFMA operand from two transpose reads (elements 0-3, then 4-7). The
// operand is assembled from whole 32-bit registers: extracting the 16-bit
// elements one by one and reinserting them as bf16 was miscompiled by the
// ROCm 7.2 compiler (element 0 replicated into the other lanes of the vector).
__device__ __forceinline__ bf16x8 tr_operand(const void* lo, const void* hi) {
  const uintx2 a = lds_read_tr16(lo), b = lds_read_tr16(hi);
  const uintx4 u = {a[0], a[1], b[0], b[1]};
  return __builtin_bit_cast(bf16x8, u);
}
// Elements 4h .. 4h+3 of a bf16x8, as one 64-bit value.
__device__ __forceinline__ uintx2 half_of(const bf16x8& x, int h) {
  const uintx4 u = __builtin_bit_cast(uintx4, x);
  return h ? uintx2{u[2], u[3]} : uintx2{u[0], u[1]};
}

// ---------------------------------------------------------------------------
// Fast transcendentals (hardware v_exp_f32 = 2^x, v_rcp_f32 = 1/x).
// ---------------------------------------------------------------------------
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float fast_rcp(float x) { return __builtin_amdgcn_rcpf(x); }

// ---------------------------------------------------------------------------
// bf16 <-> f32
// ---------------------------------------------------------------------------
__device__ __forceinline__ float bf2f(bf16 x) { return (float)x; }
__device__ __forceinline__ bf16 f2bf(float x) { return (bf16)x; }  // round to nearest even

// The two bf16 values packed in a 32-bit word (element 0 in the low half).
__device__ __forceinline__ float bf16_lo(unsigned int u) { return __builtin_bit_cast(float, u << 16); }
__device__ __forceinline__ float bf16_hi(unsigned int u) { return __builtin_bit_cast(float, u & 0xffff0000u); }

template <typename T> struct Elem;
template <> struct Elem<float> {
  static __device__ __forceinline__ float load(const float* p) { return *p; }
  static __device__ __forceinline__ void store(float* p, float v) { *p = v; }
};
template <> struct Elem<bf16> {
  static __device__ __forceinline__ float load(const bf16* p) { return (float)*p; }
  static __device__ __forceinline__ void store(bf16* p, float v) { *p = (bf16)v; }
};

// ---------------------------------------------------------------------------
// Wave-level helpers
// ---------------------------------------------------------------------------
__device__ __forceinline__ float xor32(float x) { return __shfl_xor(x, 32, 64); }
__device__ __forceinline__ bool wave_any(bool p) { return __any((int)p); }

// ---------------------------------------------------------------------------
// Workgroup -> (head, tile) mapping. Workgroups are handed to the 8 XCDs in
// round-robin order of their id, and every XCD has its own L2. All tiles of a
// head are put on one XCD (head h on XCD h % 8) so that the head's K/V stream
// is shared in that XCD's L2; within an XCD the tiles are issued in
// decreasing order of causal work, so the longest rows start first.
// The grid is 8 * ceil(N/8) * ntiles; ids that map past the last head exit.
// ---------------------------------------------------------------------------
struct TileMap {
  int N, ntiles, hpx;  // heads, tiles per head, heads per XCD
};
__host__ __device__ inline TileMap make_tilemap(int N, int ntiles) {
  TileMap m;
  m.N = N;
  m.ntiles = ntiles;
  m.hpx = (N + 7) / 8;
  return m;
}
__host__ __device__ inline long grid_size(const TileMap& m) { return 8L * m.hpx * m.ntiles; }
// Returns false for an idle workgroup.
__device__ __forceinline__ bool map_tile(const TileMap& m, int bid, int& head, int& tile,
                                         bool heavy_high) {
  const int xcd = bid & 7;
  const int k = bid >> 3;
  const int slot = k % m.hpx;
  const int round = k / m.hpx;
  head = xcd + 8 * slot;
  tile = heavy_high ? (m.ntiles - 1 - round) : round;
  return head < m.N && round < m.ntiles;
}

}  // namespace rel
