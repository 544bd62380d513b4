// Internal launch interface between the C-ABI layer and the HIP kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "common.h"

namespace rel {

// Arguments of the fused forward pass (FlashRelation, Sec. 5.1).
struct FwdArgs {
  const void* q;
  const void* k;
  const void* v;
  const float* lambda;
  void* o;
  float* row_stat;   // M_i = ln Z_i + lambda ln i, or null
  float* self_mass;  // optional
  float* exch_mass;  // optional
  float* exch_lse;   // optional
  int64_t sb, sh, st;
  int H, T;
  float scale;    // multiplier inside U
  float inv_tau;  // 1 / tau_S
  int exch_only;  // 1: exchange-only transport, y_i = sum_{j<i} F_ij v_j
  TileMap map;
};

// Arguments of the fused backward pass.
struct BwdArgs {
  const void* q;
  const void* k;
  const void* v;
  const void* o;
  const void* dout;
  const float* lambda;
  const float* row_stat;
  void* dq;
  void* dk;
  void* dv;
  float* dlam_part;  // one partial per dQ-kernel workgroup slot
  int nparts;        // number of those partials
  float* dlambda;    // out: their sum in a fixed order
  float* negd;       // -D_i = -dO_i . o_i, [N, T], written by the dQ kernel
  float* m2;         // M_i log2(e), [N, T], written by the dQ kernel
  float* dself;      // optional [N, T]
  float* dq_acc;     // fused backward: fp32 dQ accumulator [N, T, D]; null selects the two-kernel backward
  int64_t sb, sh, st;
  int H, T;
  float scale;
  float inv_tau;
  int exch_only;     // 1: gradients of the exchange-only output
  TileMap map;
};

// Arguments of the allocation (pi) diagnostic and the materialised row kernel.
struct RowArgs {
  const float* U;      // [N, T, T] scale * q k^T (materialised path) or null
  const void* q;       // allocation kernel: recomputes U from q, k
  const void* k;
  const float* exch_lse;
  const float* lambda;
  void* Fw;            // materialised: F in the storage dtype (GEMM operand)
  float* R;
  float* F;
  float* pi;
  float* self_mass;
  float* exch_mass;
  int64_t sb, sh, st;
  int H, T, D;
  float scale;
  float inv_tau;
};

// Arguments of the materialised backward row kernel (one wave per row).
struct RowBwdArgs {
  const float* U;      // [N, T, T] scale * q k^T
  const float* Hm;     // [N, T, T] dO v^T
  const float* lambda;
  void* dUw;           // out: dU in the storage dtype (GEMM operand), zeros above the diagonal
  void* Fw;            // out: F in the storage dtype (GEMM operand), zeros above the diagonal
  float* dlam_row;     // out: [N, T] per-row terms of dlambda
  int T;
  float inv_tau;
};

// Arguments of the layer prologue / epilogue kernels (RoPE, Givens mixing,
// padding). Caller tensors use (sb, sh, st); prepared tensors are contiguous
// [B, H, T, DP].
struct LayerArgs {
  const void* q;        // caller projections / information state (true width D)
  const void* k;
  const void* v;
  int64_t sb, sh, st;
  void* qr;             // out: rotated, padded q and k, or null (not written)
  void* kr;
  void* vt;             // out: mixed, padded v, or null
  const float2* rope;   // [T, D/2] (cos, sin), or null: no RoPE
  const float* theta;   // [H/2] Givens angles (givens != 0)
  int givens;           // 0 none, 1 pairing A, 2 pairing B
  int B, H, T, D, DP;
  const void* gq;       // epilogue in: gradients in the padded layout, or null
  const void* gk;
  const void* gv;
  void* dq;             // epilogue out: caller layout
  void* dk;
  void* dv;
  float* dth_rows;      // epilogue out: [H/2, B, T] per-row terms of dL/dtheta
};

// Arguments of the decode kernels (one new row per (b, h) against a KV cache).
struct DecodeArgs {
  const void* q;            // [B, H, D] dense: the new token's relation query
  const void* k;            // caches [B, H, Tmax, D] with (sb, sh, st)
  const void* v;
  const int32_t* lengths;   // [B] valid entries per batch entry (the new token's own included)
  int64_t sb, sh, st;
  int B, H, Tmax, D;
  float scale, inv_tau;
  const float* lambda;
  int key0, key1;           // states kernel: keys scanned (zero-based, half-open)
  int nsplit;               // states kernel: slices of [key0, key1)
  float* states;            // [nsplit or nstates][B H][D + 2]: m, l, z
  int nstates;              // merge kernel: states per row
  void* out;                // merge kernel: [B, H, D] dense
  float* row_stat;          // merge kernel: [B, H] or null
};

// Arguments of the Linear Relation kernels (chunks of linear_chunk() tokens).
struct LinearArgs {
  const void* p1;        // [B, H, T, D] dtype with (sb, sh, st): relation coordinates after RoPE
  const void* p2;
  const void* v;         // information state I~
  const float* g;        // [B, H, T, D] fp32, dense: log-retention (<= 0)
  int64_t sb, sh, st;
  int B, H, T, D;
  float scale, inv_tau;
  int nchunks;
  float* dstate;         // [N, nchunks, D, D]: each chunk's state contribution
  float* gamma;          // [N, nchunks, D]: each chunk's retention product
  float* cprev;          // [N, nchunks, D, D]: the state entering each chunk
  float* state_out;      // [N, D, D] or null: the state after the last token
  void* out;             // [B, H, T, D] dtype: Y
  // backward
  const void* dy;        // [B, H, T, D] dtype: dL/dY
  float* pstate;         // [N, nchunks, D, D]: Qe^T dY of each chunk
  float* gout;           // [N, nchunks, D, D]: dL/d(state leaving each chunk)
  void* dp1;             // [B, H, T, D] dtype
  void* dp2;
  void* dv;
  float* dg;             // [B, H, T, D] fp32, dense
  // 1: p1, p2, v (and dy, dp1, dp2, dv) rows start on 16-byte boundaries and
  // g is 16-byte aligned, so the chunk loads move 16 bytes per lane
  int vec16;
  // state scans over segments of linear_scan_segment() chunks
  int nseg;
  float* segc;           // [N, nseg, D, D]: each segment's forward result from a zero start
  float* segg;           // [N, nseg, D]: each segment's retention product
  float* segp;           // [N, nseg, D, D]: each segment's reverse (gradient) result from a zero start
  // The D = 128 backward runs as four 64-channel sub-problems: relation half A
  // (state rows: channels 64 A .. of qt, kt and g) times information half E
  // (state columns: channels 64 E .. of v and dY), each a D = 64 problem on
  // virtual head 4 n + 2 A + E with its own chunk states. A row pass forms qt
  // and kt over all 128 channels first; another sums the sub-problems' partial
  // gradients and takes them through S and the normalisation.
  // The retention gate of eq. 15 inside the kernels: with a_log set, g holds
  // the gate's pre-activation r and the chunk loads form
  // g = -exp(A_log) softplus(r + dt_bias); the backward's dg then goes on to
  // dr (in place), dA_log and d dt_bias.
  const float* a_log;    // [H, D] fp32, or null: g is the log-retention itself
  const float* dt_bias;  // [H, D] fp32
  float* gpart;          // [B H, ceil(T / 256), 2, D] fp32: per token segment, the sums of dg g and dr
  float* da_log;         // [H, D] fp32: d A_log
  float* ddt_bias;       // [H, D] fp32: d dt_bias
  // RoPE on p1 and p2 (the rotation of Sec. 3.1, applied before S and the
  // normalised coordinates are formed): channel j with channel j + rope_half
  // (j < rope_half) by the angle of the token's position, from a table of
  // (cos, sin) at the chunk starts and the offsets inside a chunk
  // (launch_linear_rope_table). Null: no rotation. The norms and p1 . p2 do not change.
  const float2* rope;
  int rope_half;
  int split;             // 1: D = 64 sub-problem kernels of a D = 128 backward
  float* qn;             // [N, T, 128] fp32 (split): qt = S ^p1
  float* kn;             // [N, T, 128] fp32 (split): kt = S ^p2
  float* part;           // [8][N, T, 128] fp32 (split): dqt from E = 0, 1; dkt from E = 0, 1;
                         // dv from A = 0, 1 (A = 0 holds the dY of Y = I~ + E); dg from E = 0, 1
};

// Measurement aid: if armed for kernel `name`, returns the event pair to record
// around the next launch of that kernel (see relation_profile_arm).
bool profile_slot(const char* name, hipEvent_t* start, hipEvent_t* stop);

hipError_t launch_fwd(const FwdArgs& a, int dtype, int D, hipStream_t stream);
// Measurement aid: dense bf16 MFMA chains (4 waves per workgroup).
int64_t mfma_peak_flops_per_launch(int workgroups, int iters);
hipError_t launch_mfma_peak(int workgroups, int iters, float* sink, unsigned long long* clocks, hipStream_t stream);
hipError_t launch_bwd(const BwdArgs& a, int dtype, int D, hipStream_t stream);
// The fused backward (one kernel for dK, dV and dQ, dQ summed by atomics) covers
// these problems; the two-kernel backward covers all.
bool bwd_fused_supported(int T, int D, int dtype);
int bwd_partials(int N, int T, int D, int dtype, bool fused);
hipError_t launch_fill_zero(float* p, int64_t n, hipStream_t stream);
hipError_t launch_allocation(const RowArgs& a, int dtype, int N, hipStream_t stream);
// Layer passes. `vec` (8, 2 or 1 for bf16; 4, 2 or 1 for fp32) is the number
// of contiguous channels one thread moves; the caller's tensors must allow it
// (D, D/2 with RoPE, and the strides multiples of vec; pointers aligned to it).
int linear_chunk();
int linear_scan_segment();  // chunks per segment of the state scans
hipError_t launch_linear_fwd(const LinearArgs& a, int dtype, hipStream_t stream);
hipError_t launch_linear_bwd(const LinearArgs& a, int dtype, hipStream_t stream);
int linear_gate_segment();  // tokens per segment of the gate's parameter-gradient sums
// RoPE table of the Linear Relation kernels: (linear_chunk() + chunks) x rope_dim/2 (cos, sin)
hipError_t launch_linear_rope_table(float2* tab, int T, int rope_dim, double base, hipStream_t stream);
int decode_slice_keys();
hipError_t launch_decode_states(const DecodeArgs& a, int dtype, hipStream_t stream);
hipError_t launch_decode_merge(const DecodeArgs& a, int dtype, hipStream_t stream);
hipError_t launch_rope_table(float2* tab, int T, int D, double base, hipStream_t stream);
hipError_t launch_layer_prologue(const LayerArgs& a, int dtype, int vec, hipStream_t stream);
hipError_t launch_layer_repad(const void* src, void* dst, const LayerArgs& a, bool to_padded, int dtype,
                              int vec, hipStream_t stream);
hipError_t launch_layer_epilogue(const LayerArgs& a, int dtype, int vec, hipStream_t stream);
// Fixed-order sums of nseg segments; `part` holds nseg * layer_sum_parts() floats.
int layer_sum_parts();
hipError_t launch_segment_sum(const float* x, int nseg, int64_t seg_len, float* part, float* out,
                              hipStream_t stream);
hipError_t launch_materialized_rows(const RowArgs& a, int dtype, int N, hipStream_t stream);
hipError_t launch_materialized_bwd_rows(const RowBwdArgs& a, int dtype, int N, hipStream_t stream);
// Fixed-order sum of n floats; `partial` holds sum_fixed_order_parts() floats.
int sum_fixed_order_parts();
hipError_t launch_sum_fixed_order(const float* x, int64_t n, float* partial, float* out, hipStream_t stream);

}  // namespace rel
