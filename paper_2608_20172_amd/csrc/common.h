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
// Operand policies. A kernel is written once against a policy that says how
// one 16-wide slice of an MFMA contraction is fetched and multiplied.
// For lane group g (= lane / 32) and element t in 0..7, both policies address
// the same contraction index whenever the operand comes from a tile row
// ("col" operands and register operands): index 16 ks + 8 (t / 4) + 4 g + t % 4,
// which is also the row of accumulator register 8 h + t (h = ks % 2) of a
// 32x32 block. So a 32x32 result block, re-packed from its registers, is
// directly the operand of the next product along its rows.
//   bf16: one 32x32x16 MFMA per slice; tiles are row-major in LDS with
//         16-byte chunks XOR-swizzled by row (swz); "col" operands by
//         transpose reads.
//   f32:  eight 32x32x2 MFMAs per slice; plain row-major tiles.
// ---------------------------------------------------------------------------
typedef float floatx8 __attribute__((ext_vector_type(8)));

struct Lane {
  int n, g;            // lane % 32, lane / 32
  int t_row, t_col;    // transpose-read source row / column offsets (bf16)
  __device__ explicit Lane(int lane) {
    n = lane & 31;
    g = lane >> 5;
    const int G = lane >> 4, i = lane & 15;
    t_row = 4 * (G >> 1) + (i >> 2);
    t_col = 16 * (G & 1) + 4 * (i & 3);
  }
};

template <int D>
struct PolBF16 {
  using T = bf16;
  using Op = bf16x8;
  using Chunk = uintx4;                        // 16 bytes = 8 elements
  static constexpr int CE = 8;                 // elements per chunk
  static constexpr int NCH = D / 8;            // chunks per row
  static constexpr int ROWB = 2 * D;           // bytes of one tile row
  static constexpr int TR = 64;                // rows of every tile
  static constexpr int SUB = TR * 64;          // bytes of a 32-column sub-tile
  static constexpr int tile_bytes(int rows) { return rows * ROWB; }
  // A 64-row tile is stored as D/32 sub-tiles of 32 columns (64-byte rows),
  // so a 32-column block is an immediate offset. Within a sub-tile, 16-byte
  // chunk c of row r sits at chunk c ^ swz(r): swz mixes row bits 1-3 so that
  // both access patterns below are free of bank conflicts with 32 or 64 LDS
  // banks (16-byte reads of consecutive rows, and transpose reads of 4 rows x
  // 32 bytes per 16 lanes).
  static __device__ __forceinline__ constexpr int swz(int r) {
    return ((r >> 2) & 1) | ((((r >> 1) ^ (r >> 3)) & 1) << 1);
  }
  static __device__ __forceinline__ int off(int row, int col) {
    return (col >> 5) * SUB + row * 64 + ((((col >> 3) & 3) ^ swz(row)) << 4) + ((col & 7) << 1);
  }
  // contraction over the row's elements: element t = row[16 ks + 8 g + t]
  static __device__ __forceinline__ Op row_op(const unsigned char* lds, int row, int ks, const Lane& L) {
    const int ch = 2 * ks + L.g;  // 16-byte chunk of the row
    return *(const Op*)(lds + (ch >> 2) * SUB + row * 64 + (((ch & 3) ^ swz(row)) << 4));
  }
  static __device__ __forceinline__ Op row_op_g(const T* rowp, int ks, const Lane& L) {
    return *(const Op*)(rowp + 16 * ks + 8 * L.g);
  }
  // contraction over tile rows: element t = M[16 ks + 8 (t/4) + 4 g + t%4][col0 + n]
  static __device__ __forceinline__ Op col_op(const unsigned char* lds, int ks, int col0, const Lane& L) {
    // rows 16 ks + t_row and 16 ks + t_row + 8; the swizzle sees only t_row
    const int c = L.t_col;  // column within the 32-column block col0
    const int base = (col0 >> 5) * SUB + (16 * ks + L.t_row) * 64 + ((c & 7) << 1);
    return tr_operand(lds + base + (((c >> 3) ^ swz(L.t_row)) << 4),
                      lds + base + 8 * 64 + (((c >> 3) ^ swz(L.t_row + 8)) << 4));
  }
  // Direct-load slot of lane `lane` in 1 KB segment `seg` of a tile: the tile
  // row, the byte offset of its 16 bytes within the tensor row, and the LDS
  // byte offset of the segment (16 rows of one sub-tile).
  static __device__ __forceinline__ void seg_map(int seg, int lane, int& row, int& gbyte, int& lds_off) {
    constexpr int SPS = TR / 16;  // segments per sub-tile
    const int db = seg / SPS, r0 = (seg % SPS) * 16;
    row = r0 + (lane >> 2);
    gbyte = 64 * db + 16 * ((lane & 3) ^ swz(row));
    lds_off = db * SUB + r0 * 64;
  }
  // row_op_g of the row times c, split as hi + lo with hi = bf16(x c) and
  // lo = bf16(x c - hi): a product against hi and then lo carries the factor c
  // to about 2^-16 relative, with no per-entry multiply afterwards.
  static __device__ __forceinline__ void row_op_scaled(const T* rowp, int ks, const Lane& L, float c,
                                                       Op& hi, Op& lo) {
    const uintx4 u = *(const uintx4*)(rowp + 16 * ks + 8 * L.g);
    float x[8], r[8];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      x[2 * t] = bf16_lo(u[t]) * c;
      x[2 * t + 1] = bf16_hi(u[t]) * c;
    }
    hi = pack(x);
    const uintx4 h = __builtin_bit_cast(uintx4, hi);
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      r[2 * t] = x[2 * t] - bf16_lo(h[t]);
      r[2 * t + 1] = x[2 * t + 1] - bf16_hi(h[t]);
    }
    lo = pack(r);
  }
  static __device__ __forceinline__ Op pack(const float* x) {
    Op o;
#pragma unroll
    for (int t = 0; t < 8; ++t) o[t] = (bf16)x[t];
    return o;
  }
  static __device__ __forceinline__ floatx16 mma(const Op& a, const Op& b, const floatx16& c) {
    return mfma32(a, b, c);
  }
  static __device__ __forceinline__ Op ones() {
    const uintx4 u = {0x3f803f80u, 0x3f803f80u, 0x3f803f80u, 0x3f803f80u};  // bf16 1.0 x 8
    return __builtin_bit_cast(Op, u);
  }
  // dot product of two chunks (8 products)
  static __device__ __forceinline__ float chunk_dot(const Chunk& a, const Chunk& b) {
    float s = 0.0f;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      s = __builtin_fmaf(bf16_lo(a[t]), bf16_lo(b[t]), s);
      s = __builtin_fmaf(bf16_hi(a[t]), bf16_hi(b[t]), s);
    }
    return s;
  }
  // dot product of two operands (8 products)
  static __device__ __forceinline__ float op_dot(const Op& a, const Op& b) {
    return chunk_dot(__builtin_bit_cast(uintx4, a), __builtin_bit_cast(uintx4, b));
  }
  // 4 consecutive elements
  static __device__ __forceinline__ floatx4 load4(const T* p) {
    const uintx2 u = *(const uintx2*)p;
    return floatx4{bf16_lo(u[0]), bf16_hi(u[0]), bf16_lo(u[1]), bf16_hi(u[1])};
  }
  static __device__ __forceinline__ void store4(T* p, const floatx4& x) {
    bf16x4 v;
#pragma unroll
    for (int e = 0; e < 4; ++e) v[e] = (bf16)x[e];
    *(bf16x4*)p = v;
  }
};

template <int D>
struct PolF32 {
  using T = float;
  using Op = floatx8;
  using Chunk = floatx4;                       // 16 bytes = 4 elements
  static constexpr int CE = 4;
  static constexpr int NCH = D / 4;
  static constexpr int ROWF = D;               // row, floats (no padding: tiles are filled by DMA)
  static constexpr int ROWB = 4 * D;           // bytes per LDS row
  static constexpr int TR = 64;                // rows of every tile
  // Direct-load slot (see PolBF16::seg_map): plain row-major rows.
  static __device__ __forceinline__ void seg_map(int seg, int lane, int& row, int& gbyte, int& lds_off) {
    constexpr int CH = ROWB / 16, SEG_ROWS = 1024 / ROWB;
    static_assert(SEG_ROWS * ROWB == 1024, "a row must divide 1 KB");
    const int r0 = seg * SEG_ROWS;
    row = r0 + lane / CH;
    gbyte = 16 * (lane % CH);
    lds_off = r0 * ROWB;
  }
  static constexpr int tile_bytes(int rows) { return rows * ROWF * 4; }
  static __device__ __forceinline__ const float* fp(const unsigned char* lds) { return (const float*)lds; }
  // element t = row[16 ks + 2 t + g]  (MFMA step t covers 16 ks + 2 t .. +1)
  static __device__ __forceinline__ Op row_op(const unsigned char* lds, int row, int ks, const Lane& L) {
    const float* f = fp(lds) + row * ROWF + 16 * ks + L.g;
    Op o;
#pragma unroll
    for (int t = 0; t < 8; ++t) o[t] = f[2 * t];
    return o;
  }
  static __device__ __forceinline__ Op row_op_g(const T* rowp, int ks, const Lane& L) {
    Op o;
#pragma unroll
    for (int t = 0; t < 8; ++t) o[t] = rowp[16 * ks + 2 * t + L.g];
    return o;
  }
  // fp32 rows take the factor c in one rounding; lo stays unused
  static __device__ __forceinline__ void row_op_scaled(const T* rowp, int ks, const Lane& L, float c,
                                                       Op& hi, Op& lo) {
#pragma unroll
    for (int t = 0; t < 8; ++t) hi[t] = rowp[16 * ks + 2 * t + L.g] * c;
    lo = Op{};
  }
  static __device__ __forceinline__ Op col_op(const unsigned char* lds, int ks, int col0, const Lane& L) {
    const float* f = fp(lds) + col0 + L.n;
    Op o;
#pragma unroll
    for (int t = 0; t < 8; ++t) o[t] = f[(16 * ks + 8 * (t >> 2) + 4 * L.g + (t & 3)) * ROWF];
    return o;
  }
  static __device__ __forceinline__ Op pack(const float* x) {
    Op o;
#pragma unroll
    for (int t = 0; t < 8; ++t) o[t] = x[t];
    return o;
  }
  static __device__ __forceinline__ floatx16 mma(const Op& a, const Op& b, floatx16 c) {
#pragma unroll
    for (int t = 0; t < 8; ++t) c = mfma32f(a[t], b[t], c);
    return c;
  }
  static __device__ __forceinline__ Op ones() {
    Op o;
#pragma unroll
    for (int t = 0; t < 8; ++t) o[t] = 1.0f;
    return o;
  }
  static __device__ __forceinline__ float chunk_dot(const Chunk& a, const Chunk& b) {
    return __builtin_fmaf(a[0], b[0], __builtin_fmaf(a[1], b[1], __builtin_fmaf(a[2], b[2], a[3] * b[3])));
  }
  static __device__ __forceinline__ float op_dot(const Op& a, const Op& b) {
    float s = 0.0f;
#pragma unroll
    for (int t = 0; t < 8; ++t) s = __builtin_fmaf(a[t], b[t], s);
    return s;
  }
  static __device__ __forceinline__ floatx4 load4(const T* p) { return *(const floatx4*)p; }
  static __device__ __forceinline__ void store4(T* p, const floatx4& x) { *(floatx4*)p = x; }
};

// ---------------------------------------------------------------------------
// Tiles HBM -> LDS without registers: buffer loads that write LDS directly.
// One 64-lane load moves 1 KB: lane l's 16 bytes land at segment + 16 l, so
// each lane fetches whichever 16 bytes of the tensor the policy's layout puts
// in that slot (seg_map). Rows past the end of the buffer resource read as
// zeros (the hardware range check), which is how tiles running past T are
// padded.
// ---------------------------------------------------------------------------
typedef __attribute__((address_space(3))) void lds_void;
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, int bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, bytes, 0x00020000);
}
// 1 KB segment `seg` of a 64-row tile whose row 0 is tensor row j0 (row
// stride row_bytes); `tile` is the LDS tile, wave-uniform.
template <class P>
__device__ __forceinline__ void dma_segment(__amdgpu_buffer_rsrc_t rs, unsigned char* tile, int seg, int row_bytes,
                                            int j0, int lane) {
  int row, gbyte, lds_off;
  P::seg_map(seg, lane, row, gbyte, lds_off);
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_void*)(tile + lds_off), 16, row * row_bytes + gbyte,
                                           j0 * row_bytes, 0, 0);
}
// 64 consecutive fp32 values from element j0 of a row vector into dst[0..63].
__device__ __forceinline__ void dma_row64(__amdgpu_buffer_rsrc_t rs, float* dst, int j0, int lane) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_void*)dst, 4, 4 * lane, 4 * j0, 0, 0);
}
// Waits until this wave's loads have landed (vmcnt 0; other counters untouched).
__device__ __forceinline__ void wait_loads() { __builtin_amdgcn_s_waitcnt(0x0f70); }

// Register r* of a 32x32 block that holds row n for lane group g, if any:
// acc_row(r, g) == n  <=>  g == (n >> 2) & 1  and  r == 4 (n >> 3) + (n & 3).
__device__ __forceinline__ bool holds_row(int n, int g) { return ((n >> 2) & 1) == g; }
__device__ __forceinline__ int row_reg(int n) { return 4 * (n >> 3) + (n & 3); }
__device__ __forceinline__ float pick(const floatx16& x, int r) {
  float v = 0.0f;
#pragma unroll
  for (int i = 0; i < 16; ++i) v = (i == r) ? x[i] : v;
  return v;
}
__device__ __forceinline__ float pick(const float* x, int r) {
  float v = 0.0f;
#pragma unroll
  for (int i = 0; i < 16; ++i) v = (i == r) ? x[i] : v;
  return v;
}

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
