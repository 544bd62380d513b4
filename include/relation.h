/*
 * relation.h - C ABI of the FlashRelation library: the exact causal Full
 * Relation operator (Self-Exchange Relation, one head per (b, h)) on gfx950.
 *
 * Operator (per head, rows i = 1..T one-based, from the paper's Sec. 3.1,
 * eqs. (1)-(3), restated in App. A.1.1):
 *   U_ij = scale * q_i . k_j                       scale = 1/sqrt(D) by default
 *   S_i  = sigmoid(U_ii / tau_s)                   Self, on the diagonal
 *   E_ij = SiLU(U_ij) = U_ij * sigmoid(U_ij)       Exchange, for j < i
 *   R_ij = S_i (j = i); E_ij - lambda * ln(i) (j < i); -inf (j > i)
 *   F_i  = softmax(R_i),   y_i = sum_{j <= i} F_ij v_j
 * q and k are the two relation projections after RoPE, v is the information
 * state after Givens head mixing; lambda is the layer's count-calibration
 * scalar, shared by all heads (App. A.1.1), tau_s the fixed Self temperature
 * (2 in the paper). The flash entry points never form U, R or F in memory:
 * they run the tiled online Exchange scan of Sec. 5.1 (eqs. 11-13, App. A.3)
 * and apply Self and lambda after the scan.
 *
 * Conventions shared by every entry point
 *  - Tensors q, k, v, o, dout, dq, dk, dv are [B, H, T, D] with element
 *    strides (stride_b, stride_h, stride_t) taken from rel_problem and a
 *    contiguous last dimension. They all have the element type `dtype`.
 *    The rows of one head must span less than 2 GiB (T * stride_t elements).
 *  - Row vectors (row_stat, self_mass, exch_mass, exch_lse, dself) are fp32,
 *    dense [B, H, T]. T x T outputs (R, F, pi) are fp32, dense [B, H, T, T].
 *  - lambda and dlambda point to one fp32 scalar in device memory.
 *  - All pointers are device pointers owned by the caller. The library keeps
 *    no allocation between calls; scratch memory comes from the caller's
 *    workspace, sized by the *_workspace_bytes queries.
 *  - Work is enqueued asynchronously on `stream` (a hipStream_t; NULL means
 *    the default stream). No entry point synchronises the host.
 *  - Outputs are overwritten, never accumulated into.
 *  - Arguments are validated on the host before any HIP call; on failure
 *    nothing is launched and a rel_status < 0 is returned. The message of the
 *    last failure on the calling thread is returned by relation_last_error().
 *  - B * H * T == 0 returns REL_OK without launching anything.
 */
#ifndef RELATION_H
#define RELATION_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define RELATION_ABI_VERSION 1

typedef enum rel_status {
  REL_OK = 0,
  REL_ERR_INVALID_ARG = -1, /* null/overlapping/misaligned pointer, bad size or stride, bad tau_s */
  REL_ERR_UNSUPPORTED = -2, /* dtype, head dimension or causal flag this build has no kernel for,
                               T > 2^24, B*H > 2^30, or T * stride_t * element size >= 2^31 bytes */
  REL_ERR_WORKSPACE = -3,   /* workspace pointer null or smaller than the query result */
  REL_ERR_HIP = -4,         /* a HIP/rocBLAS call failed; see relation_last_error() */
  /* Widens the enumeration to every int32 value, so that any status code a C
   * caller passes (relation_status_string) is a valid value of the type in C++
   * as well; never returned. */
  REL_STATUS_MAX_ENUM = 0x7fffffff
} rel_status;

typedef enum rel_dtype {
  REL_F32 = 0,  /* fp32 storage, fp32 MFMA (parity path) */
  REL_BF16 = 1  /* bf16 storage, bf16 MFMA with fp32 accumulation and statistics */
} rel_dtype;

typedef struct rel_problem {
  int64_t B, H, T, D;   /* batch, heads, sequence length, head width. D in {32, 64, 128},
                           or 96 with bf16 (the layer entry points take any D <= 128) */
  int32_t dtype;        /* rel_dtype of q, k, v, o, dout, dq, dk, dv */
  int32_t causal;       /* must be 1: the paper defines only the causal R (eq. 2) */
  float tau_s;          /* Self temperature, finite and > 0 (paper: 2.0) */
  float scale;          /* multiplier inside U; <= 0 selects 1/sqrt(D) (eq. 1) */
  int64_t stride_b;     /* element strides shared by all [B,H,T,D] tensors; */
  int64_t stride_h;     /* the last dimension is contiguous. stride_t must be a */
  int64_t stride_t;     /* multiple of 16 bytes / element size and >= D (any
                           multiple of the element size for the layer entry points) */
} rel_problem;

/* Forward pass (FlashRelation, Sec. 5.1).
 *   q, k, v   in  [B,H,T,D] dtype
 *   lambda    in  device fp32 scalar
 *   o         out [B,H,T,D] dtype: y_i = (1 - g_i) v_i + g_i * Ibar_i (eq. 13)
 *   row_stat  out [B,H,T] fp32: M_i = ln Z_i + lambda ln i, the one statistic the
 *             backward pass needs (then F_ij = exp(E_ij - M_i) for j < i). May be
 *             NULL when no backward pass follows.
 *   self_mass out [B,H,T] fp32, optional: F_ii = sigmoid(S_i - A_i) (eq. 6)
 *   exch_mass out [B,H,T] fp32, optional: g_i = sigmoid(A_i - S_i) (eq. 6)
 *   exch_lse  out [B,H,T] fp32, optional: L^E_i = LSE_{j<i} E_ij (eq. 5); -inf on
 *             row 1. With it, the within-history allocation is
 *             pi_ij = exp(E_ij - L^E_i) (eq. 7).
 *   All optional outputs may be NULL. Row 1 has no history: g = 0, y = v (App. A.1.8). */
rel_status relation_fwd(const rel_problem* p, const void* q, const void* k, const void* v,
                        const float* lambda, void* o, float* row_stat, float* self_mass,
                        float* exch_mass, float* exch_lse, void* stream);

/* Within-history Exchange allocation pi (eq. 7), written densely:
 *   pi    out [B,H,T,T] fp32: pi_ij = exp(E_ij - L^E_i) for j < i, 0 elsewhere
 *         (all of row 1 is 0). This is O(T^2) output by nature; it is a
 *         diagnostic, not part of the fused path.
 *   exch_lse in [B,H,T] fp32, as written by relation_fwd. */
rel_status relation_exchange_allocation(const rel_problem* p, const void* q, const void* k,
                                        const float* exch_lse, float* pi, void* stream);

/* Backward pass: gradients of sum(dout * o) (App. A.1.7), recomputed tile by
 * tile from q, k, v, o and row_stat.
 * relation_bwd runs one kernel for dk, dv and dq when dtype is bf16, D is 32
 * or 64 and T >= 1536 (a row pass before it and a dq pass after it; at shorter
 * T the two-kernel backward is faster): each workgroup of 256
 * keys adds its dq partials into an fp32 accumulator with atomics, so dq is
 * correct to fp32 rounding but not bitwise run-to-run repeatable; dk, dv,
 * dlambda and dself are. Other problems, and relation_bwd_deterministic
 * always, run the two-kernel backward (a query-major dq kernel, then a
 * key-major dk/dv kernel), where every output is written exactly once and all
 * results are bitwise repeatable.
 *   dq, dk, dv out [B,H,T,D] dtype
 *   dlambda    out device fp32 scalar: sum over b, h, i of ln(i) * dR_ii, which
 *              equals -sum g_i (1-g_i) c_i ln i of App. A.1.7. Reduced in a fixed
 *              order.
 *   dself      out [B,H,T] fp32, optional: dL/dS_i, the gradient reaching the
 *              Self logit R_ii = S_i (-g_i (1 - g_i) c_i in App. A.1.7).
 *   workspace  at least relation_bwd_workspace_bytes(p) bytes of device memory
 *              (enough for either path), 16-byte aligned: two fp32 values per
 *              row (-D_i = -dout_i . o_i and M_i log2(e), read by the dk/dv
 *              kernel), one dlambda partial per workgroup for the fixed-order
 *              reduction, and on the one-kernel path the fp32 dq accumulator
 *              [B,H,T,D]; contents on entry are ignored. */
size_t relation_bwd_workspace_bytes(const rel_problem* p);
rel_status relation_bwd(const rel_problem* p, const void* q, const void* k, const void* v,
                        const void* o, const void* dout, const float* lambda,
                        const float* row_stat, void* dq, void* dk, void* dv, float* dlambda,
                        float* dself, void* workspace, size_t workspace_bytes, void* stream);
rel_status relation_bwd_deterministic(const rel_problem* p, const void* q, const void* k,
                                      const void* v, const void* o, const void* dout,
                                      const float* lambda, const float* row_stat, void* dq, void* dk,
                                      void* dv, float* dlambda, float* dself, void* workspace,
                                      size_t workspace_bytes, void* stream);

/* Backward pass for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * relation_bwd_deterministic (the two-kernel backward, bitwise repeatable) with
 * the same kernels and results, but no workspace argument.
 * Its scratch (the two fp32 values per row and the dlambda partials that
 * relation_bwd takes from its workspace) lives in a device array inside the
 * library, one copy per GPU, allocated when the library's code is loaded on
 * that GPU and held until the process ends. The call itself allocates
 * nothing (no hipMalloc, hipFree or allocating library routine).
 *   Limit: relation_bwd_workspace_bytes(p) must not exceed
 *   relation_bwd_noalloc_max_scratch_bytes() (32 MiB, about 4 million rows
 *   B*H*T); larger problems return REL_ERR_WORKSPACE without launching.
 *   Every call on one GPU shares that GPU's array: calls that overlap in time
 *   on one GPU (two streams, two host threads) race and give wrong results;
 *   serialise them. The array's contents on entry are ignored.
 * Other arguments, errors and outputs as relation_bwd. */
size_t relation_bwd_noalloc_max_scratch_bytes(void);
rel_status relation_bwd_noalloc(const rel_problem* p, const void* q, const void* k, const void* v,
                                const void* o, const void* dout, const float* lambda,
                                const float* row_stat, void* dq, void* dk, void* dv,
                                float* dlambda, float* dself, void* stream);

/* Materialised Full Relation: U = scale q k^T is written to HBM in full
 * (rocBLAS batched GEMM), a row kernel builds R and F = softmax(R) (eqs. 2-3),
 * and a second GEMM forms o = F v. The baseline the fused path is measured
 * against (Table 5(a)).
 *   R, F, pi   out [B,H,T,T] fp32, optional: R with -inf above the diagonal,
 *              F and pi (eq. 7) with 0 there.
 *   self_mass, exch_mass  out [B,H,T] fp32, optional.
 *   workspace  at least relation_fwd_materialized_workspace_bytes(p) bytes:
 *              U in fp32 plus F in dtype, i.e. B*H*T*T*(4 + sizeof(dtype)). */
size_t relation_fwd_materialized_workspace_bytes(const rel_problem* p);
rel_status relation_fwd_materialized(const rel_problem* p, const void* q, const void* k,
                                     const void* v, const float* lambda, void* o, float* R,
                                     float* F, float* pi, float* self_mass, float* exch_mass,
                                     void* workspace, size_t workspace_bytes, void* stream);

/* Materialised backward pass (App. A.1.7 with every T x T tensor in HBM): the
 * baseline of the fused backward. U = scale q k^T and H = dout v^T are
 * written by rocBLAS batched GEMMs; a row kernel forms F_i = softmax(R_i) again
 * from U_i, D_i = sum_j F_ij H_ij, dR_ij = F_ij (H_ij - D_i) and
 * dU_ij = dR_ij SiLU'(U_ij) (j < i), dU_ii = dR_ii S_i (1 - S_i) / tau_S, and
 * the row's term -ln(i) sum_{j<i} dR_ij of dlambda; three GEMMs form
 * dq = scale dU k, dk = scale dU^T q, dv = F^T dout.
 *   q, k, v, dout  in [B,H,T,D] dtype; lambda in device fp32 scalar
 *   dq, dk, dv     out [B,H,T,D] dtype (overwritten)
 *   dlambda        out device fp32 scalar, the row terms summed in a fixed order
 *   workspace      at least relation_bwd_materialized_workspace_bytes(p) bytes,
 *                  16-byte aligned: U and H in fp32, dU and F in dtype, one
 *                  fp32 per row and 256 fp32 partial sums; i.e.
 *                  B*H*T*T*(8 + 2 sizeof(dtype)) + 4 B*H*T + 1024 bytes (with
 *                  256-byte alignment of each part). Contents on entry are
 *                  ignored.
 *   T <= 65536 and T*T <= 2^31, else REL_ERR_UNSUPPORTED. */
size_t relation_bwd_materialized_workspace_bytes(const rel_problem* p);
rel_status relation_bwd_materialized(const rel_problem* p, const void* q, const void* k,
                                     const void* v, const void* dout, const float* lambda, void* dq,
                                     void* dk, void* dv, float* dlambda, void* workspace,
                                     size_t workspace_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * Layer entry points: the operator together with the steps that surround it in
 * a Relation layer (Sec. 3.1 and eq. 4; App. A.2.2-A.2.3; App. B):
 *   q, k  -> RoPE over the full head width, channel d turned with channel
 *            d + D/2 by t * rope_base^(-2d/D), t the zero-based position;
 *   v     -> Givens mixing of head pairs: for pair p = (a, b),
 *            v~_a = cos(theta_p) v_a - sin(theta_p) v_b,
 *            v~_b = sin(theta_p) v_a + cos(theta_p) v_b,
 *            pairing A = (1,2), (3,4), ..., (H-1,H), pairing B = (2,3), (4,5),
 *            ..., (H,1) (one-based heads; the pairing alternates over depth);
 *   y     =  the causal Full Relation of (RoPE(q), RoPE(k), v~).
 * Here p->D is the true head width d_h: any D <= 128 (even when RoPE is on).
 * Widths the fused kernels do not tile (e.g. the paper's 48, 60, 80) are run
 * with zero channels appended up to 32, 64, 96 (bf16) or 128; scale <= 0 still means
 * 1/sqrt(d_h) of the true width. Strides need only be multiples of the
 * element size here.
 *   opts        rope_base > 0 turns RoPE on (the paper uses 1e4), 0 off;
 *               givens = REL_GIVENS_NONE / _A / _B (H even for A and B);
 *               transport = REL_TRANSPORT_FULL, or _EXCHANGE for the
 *               exchange-only ablation (forward and backward). The other
 *               structural ablations need no flag: lambda = 0 is "no count
 *               calibration", givens = NONE is "no Givens mixing".
 *   theta       device fp32 [H/2] angles (read when givens != NONE).
 *   out         [B,H,T,D] dtype: y.   row_stat  [B,H,T] fp32: M_i for the
 *               backward pass (as relation_fwd).
 *   saved       relation_layer_saved_bytes(p, opts) bytes of device memory,
 *               16-byte aligned, owned by the caller from the forward call to
 *               the backward call: the prepared operands (rotated q and k,
 *               mixed v, the forward's output, each [B,H,T,DP] with DP = 32,
 *               64, 96 or 128 the tiled width) and a [T, D/2] cos/sin table. The
 *               forward pass writes it; the backward pass reads it instead of
 *               preparing the operands again. NULL: the forward pass prepares
 *               them in its workspace and the backward pass recomputes them.
 *               A layer with no RoPE, no mixing, a tiled width and contiguous
 *               tensors needs none of this (0 bytes) and runs relation_fwd /
 *               relation_bwd on the caller's tensors, which must then meet
 *               their alignment rules.
 *   workspace   forward: relation_layer_fwd_workspace_bytes(p, opts) bytes
 *               when saved is NULL (none otherwise). Backward:
 *               relation_layer_bwd_workspace_bytes(p, opts) bytes (which
 *               include room to recompute the prepared operands; with saved,
 *               the saved size may be subtracted): padded dout, the gradients
 *               in the padded layout, relation_bwd's own workspace, one fp32
 *               dtheta term per (pair, b, t) and their partial sums.
 *               16-byte aligned, contents ignored on entry.
 *   out (backward) must be the tensor the forward call wrote, at the same
 *               address: from its address and layout the backward pass
 *               decides whether the forward's output sits there or in the
 *               saved buffer (a copy elsewhere, with a different 16-byte
 *               alignment, would make it read a region the forward did not
 *               write).
 * The backward pass returns dq, dk, dv with respect to the unrotated, unmixed
 * inputs, dlambda as relation_bwd, and dtheta [H/2] fp32 (required when
 * givens != NONE, each angle's gradient summed over batch, positions and
 * channels in a fixed order). Results are run-to-run identical. */
typedef enum rel_givens {
  REL_GIVENS_NONE = 0,
  REL_GIVENS_A = 1,
  REL_GIVENS_B = 2
} rel_givens;

typedef enum rel_transport {
  REL_TRANSPORT_FULL = 0,     /* y_i = sum_{j <= i} F_ij v~_j (eq. 3) */
  REL_TRANSPORT_EXCHANGE = 1  /* exchange-only ablation (App. D): y_i = sum_{j < i} F_ij v~_j,
                                 the same F, historical weights not renormalised */
} rel_transport;

typedef struct rel_layer_opts {
  double rope_base;   /* > 0: RoPE with this base; 0: no RoPE */
  int32_t givens;     /* rel_givens */
  int32_t transport;  /* rel_transport */
} rel_layer_opts;

size_t relation_layer_saved_bytes(const rel_problem* p, const rel_layer_opts* opts);
size_t relation_layer_fwd_workspace_bytes(const rel_problem* p, const rel_layer_opts* opts);
rel_status relation_layer_fwd(const rel_problem* p, const rel_layer_opts* opts, const void* q,
                              const void* k, const void* v, const float* lambda, const float* theta,
                              void* out, float* row_stat, void* saved, size_t saved_bytes,
                              void* workspace, size_t workspace_bytes, void* stream);
size_t relation_layer_bwd_workspace_bytes(const rel_problem* p, const rel_layer_opts* opts);
rel_status relation_layer_bwd(const rel_problem* p, const rel_layer_opts* opts, const void* q,
                              const void* k, const void* v, const void* out, const void* dout,
                              const float* lambda, const float* theta, const float* row_stat,
                              const void* saved, size_t saved_bytes, void* dq, void* dk, void* dv,
                              float* dlambda, float* dtheta, void* workspace, size_t workspace_bytes,
                              void* stream);

/* ---------------------------------------------------------------------------
 * Decode step: the one new row of every (b, h) against a KV cache (eq. 2 at
 * the token's absolute position). The new token's own key and value must
 * already be in the cache at entry lengths[b] (one-based), which is its
 * position i, so the count correction is -lambda ln(lengths[b]); entries
 * 1 .. lengths[b] - 1 are its history. The result equals row i of
 * relation_fwd over the sequence (and its row_stat).
 *   p          B, H, D, dtype, tau_s, scale as for relation_fwd; T is the cache
 *              capacity Tmax >= 1, and the strides are those of the caches.
 *   q          [B,H,D] dtype, dense: the new token's relation query.
 *   k_cache, v_cache  [B,H,Tmax,D] dtype with the problem's strides.
 *   lengths    device int32 [B]: entries of the cache in use, new token
 *              included. They are device data, so the host cannot check
 *              them: for an entry outside 1..Tmax the kernels read only
 *              inside the cache and that entry's rows of out and row_stat
 *              are written as NaN.
 *   out        [B,H,D] dtype, dense: y_i.   row_stat  [B,H] fp32, optional:
 *              M_i = ln Z_i + lambda ln i.
 *   workspace  relation_decode_workspace_bytes(p) bytes, 16-byte aligned: the
 *              Exchange scan states of the history's slices of 256 keys.
 * relation_decode_states and relation_decode_merge are its two halves, for a
 * cache split over devices (context parallelism): each device writes the
 * states of its keys [key_begin, key_end) of its own cache (only keys before
 * the row's own entry count) as nstates slices, in
 *   states     fp32 [nstates][B*H][D + 2], 8-byte aligned: per slice and row m = max E_ij,
 *              l = sum exp(E_ij - m), z = sum exp(E_ij - m) v_j (eq. 11;
 *              an empty slice has m = -inf, l = 0, z = 0);
 * the device that holds the new token's entry merges any number of such
 * states (concatenated along the first axis) with the Self entry read at
 * lengths[b] of its k_cache / v_cache. The merge rescales the states to their
 * common maximum and adds them, then applies eqs. 12-13. */
size_t relation_decode_workspace_bytes(const rel_problem* p);
rel_status relation_decode(const rel_problem* p, const void* q, const void* k_cache, const void* v_cache,
                           const int32_t* lengths, const float* lambda, void* out, float* row_stat,
                           void* workspace, size_t workspace_bytes, void* stream);
rel_status relation_decode_states(const rel_problem* p, const void* q, const void* k_cache,
                                  const void* v_cache, const int32_t* lengths, int32_t key_begin,
                                  int32_t key_end, int32_t nstates, float* states, void* stream);
rel_status relation_decode_merge(const rel_problem* p, int32_t nstates, const float* states, const void* q,
                                 const void* k_cache, const void* v_cache, const int32_t* lengths,
                                 const float* lambda, void* out, float* row_stat, void* stream);

/* ---------------------------------------------------------------------------
 * Linear Relation (Sec. 5.2, App. A.4): Self explicit, Exchange read from a
 * recurrent D x D state per head with channel-wise retention alpha = exp(g):
 *   S_t = sigmoid(scale p1_t . p2_t / tau_s), ^p = p / |p|,
 *   C_t^- = Diag(alpha_t) C_{t-1} (C_0 = 0),  y_t = v_t + S_t (C_t^-)^T ^p1_t,
 *   C_t = C_t^- + S_t ^p2_t v_t^T.
 *   p          B, H, T, D (32, 64 or 128), dtype, tau_s, scale, strides of
 *              p1, p2, v, out, as for relation_fwd.
 *   p1, p2     [B,H,T,D] dtype: the two relation coordinates after RoPE.
 *   v          [B,H,T,D] dtype: the information state I~.
 *   g          [B,H,T,D] fp32, dense: log-retention g_t = log alpha_t <= 0 (the
 *              gate of eq. 15 is the caller's elementwise map; positive values
 *              are not checked and grow the state).
 *   out        [B,H,T,D] dtype: y.
 *   state_out  [B,H,D,D] fp32, optional: C_T, the decode state after the last
 *              token (rows: relation channel, columns: information channel).
 *   workspace  relation_linear_fwd_workspace_bytes(p) bytes, 16-byte aligned:
 *              per chunk of 64 tokens its state contribution and retention
 *              product, and the state entering it; per segment of 16 chunks
 *              the scan's summary (fp32).
 * Precision: fp32 inputs run every product in fp32. bf16 inputs take the
 * chunk products on bf16 operands with fp32 accumulation, except that the
 * backward keeps fp32 accuracy in the products that reach dg (and so dr,
 * dA_log, d dt_bias); decay weights, state scans and statistics are fp32. */
size_t relation_linear_fwd_workspace_bytes(const rel_problem* p);
rel_status relation_linear_fwd(const rel_problem* p, const void* p1, const void* p2, const void* v,
                               const float* g, void* out, float* state_out, void* workspace,
                               size_t workspace_bytes, void* stream);

/* Linear Relation backward: gradients of sum(dout * y) with respect to p1,
 * p2, v (dtype, the problem's strides) and g (fp32, dense [B,H,T,D]). The
 * chunk states are recomputed from the inputs. D in {32, 64, 128}. At D = 128
 * the state is taken as four 64 x 64 blocks (halves of the relation and of
 * the information channels), each of which evolves on its own, and the
 * gradient is the sum of the four blocks' terms; the result matches the
 * one-block computation up to fp32 rounding order. Head widths between these
 * (the paper's 48, 60, 80) run zero-padded to the next one, with an explicit
 * scale of 1/sqrt(true width).
 *   workspace  relation_linear_bwd_workspace_bytes(p) bytes, 16-byte aligned:
 *              the forward workspace plus, per chunk, the D x D products that
 *              the reverse scan over chunks reads and the state gradients it
 *              writes, and per segment of 16 chunks the reverse summary. At
 *              D = 128 the chunk states are those of 4 B H heads of width 64,
 *              plus S ^p1 and S ^p2 of every row and eight fp32 [B,H,T,128]
 *              planes of partial gradients (5 KiB per token and head). */
size_t relation_linear_bwd_workspace_bytes(const rel_problem* p);
rel_status relation_linear_bwd(const rel_problem* p, const void* p1, const void* p2, const void* v,
                               const float* g, const void* dout, void* dp1, void* dp2, void* dv, float* dg,
                               void* workspace, size_t workspace_bytes, void* stream);

/* Linear Relation as the paper's layer runs it (Sec. 5.2, App. A.4), with the
 * retention gate of eq. 15 formed inside the kernels,
 *   g_t = -exp(A_log) * softplus(r_t + dt_bias),  alpha_t = exp(g_t) in (0, 1],
 * in place of a caller-made g, and optionally the RoPE of Sec. 3.1 on p1 and p2
 * before S_t and the normalised coordinates are formed.
 *   r          [B,H,T,D] fp32, dense: the gate's pre-activation (the caller's
 *              low-rank projection of the token's input).
 *   a_log,     [H,D] fp32, dense: one value per head and channel, shared by
 *   dt_bias    every batch entry and token.
 *   rope_dim   0: p1, p2 as given. Else the rotated width, even and <= D (a
 *              multiple of 8 at D = 128): channel j < rope_dim/2 turns with
 *              channel j + rope_dim/2 by t * rope_base^(-2j/rope_dim) at the
 *              zero-based position t; channels from rope_dim on are not turned
 *              (a head of width 80 zero-padded to 128 takes rope_dim = 80).
 *   rope_base  the base, finite and > 0 (the paper's 10^4) when rope_dim > 0.
 * Forward: as relation_linear_fwd, with workspace
 * relation_linear_gated_fwd_workspace_bytes(p, rope_dim) (the ungated
 * forward's plus a table of (cos, sin) at the 64-token chunk starts and at
 * the offsets inside a chunk, ((T + 63)/64 + 64) x rope_dim/2). Backward: as
 * relation_linear_bwd, the gradients with respect to the unrotated p1, p2, with
 *   dr         [B,H,T,D] fp32, dense: dL/dr (in place of dg);
 *   da_log,    [H,D] fp32: dL/dA_log and dL/d dt_bias, each summed over batch
 *   ddt_bias   entries and tokens in a fixed order (run-to-run identical);
 *   workspace  relation_linear_gated_bwd_workspace_bytes(p, rope_dim) bytes:
 *              the ungated backward's plus the two sums per head and chunk (or
 *              segment of 256 tokens) and the RoPE table.
 * Missing a_log or dt_bias, a bad rope_dim or rope_base: REL_ERR_INVALID_ARG
 * (REL_ERR_UNSUPPORTED for a rope_dim at D = 128 that is not a multiple of 8). */
size_t relation_linear_gated_fwd_workspace_bytes(const rel_problem* p, int32_t rope_dim);
rel_status relation_linear_gated_fwd(const rel_problem* p, const void* p1, const void* p2, const void* v,
                                     const float* r, const float* a_log, const float* dt_bias, int32_t rope_dim,
                                     float rope_base, void* out, float* state_out, void* workspace,
                                     size_t workspace_bytes, void* stream);
size_t relation_linear_gated_bwd_workspace_bytes(const rel_problem* p, int32_t rope_dim);
rel_status relation_linear_gated_bwd(const rel_problem* p, const void* p1, const void* p2, const void* v,
                                     const float* r, const float* a_log, const float* dt_bias, int32_t rope_dim,
                                     float rope_base, const void* dout, void* dp1, void* dp2, void* dv, float* dr,
                                     float* da_log, float* ddt_bias, void* workspace, size_t workspace_bytes,
                                     void* stream);

/* Measurement aid. While armed, every launch of the named kernel ("fwd": the
 * fused forward kernel; "bwd": all kernels of one relation_bwd call, back to
 * back; "bwd_dkdv": the dk/dv kernel, or the one-kernel backward's main
 * kernel; "bwd_dq": the two-kernel backward's dq kernel; "bwd_prep",
 * "bwd_convert": the one-kernel backward's row pass and dq pass) is bracketed by
 * hipEventRecord on its launch stream, using the caller's events in pairs
 * (events[2i] before launch i, events[2i+1] after it) until n_pairs launches
 * have been recorded. The events are owned by the caller (hipEvent_t, created
 * without the disable-timing flag). Arming replaces any previous arming.
 * relation_profile_disarm() returns the number of pairs recorded. The state
 * is process-wide and guarded by a mutex. */
rel_status relation_profile_arm(const char* kernel, void** events, int n_pairs);
int relation_profile_disarm(void);

/* Measurement aid, not part of the operator: the achievable dense bf16 MFMA
 * rate. Launches `workgroups` workgroups of 4 waves; every wave runs `iters`
 * rounds of 8 independent v_mfma_f32_32x32x16_bf16 chains, in all
 * relation_mfma_peak_flops(workgroups, iters) flop; time it with events on
 * `stream`. sink: device fp32 [workgroups * 256] (results, so nothing is
 * optimised away). clocks: device uint64 [2], wave 0 of workgroup 0's
 * s_memtime and s_memrealtime differences over its loop. */
int64_t relation_mfma_peak_flops(int workgroups, int iters);
rel_status relation_mfma_peak_probe(int workgroups, int iters, float* sink, unsigned long long* clocks,
                                    void* stream);

const char* relation_status_string(rel_status s);
const char* relation_last_error(void);
int relation_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* RELATION_H */
