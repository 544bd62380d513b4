// C-ABI layer: argument validation on the host, workspace sizing, dispatch to
// the HIP kernels, and the rocBLAS handle used by the materialised baseline.
#include "../../include/relation.h"

#include <rocblas/rocblas.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <initializer_list>
#include <mutex>
#include <string>
#include <vector>

#include "kernels.h"

namespace {

thread_local std::string g_last_error;

rel_status fail(rel_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return s;
}

rel_status hip_fail(hipError_t e, const char* where) {
  return fail(REL_ERR_HIP, "%s: %s", where, hipGetErrorString(e));
}

size_t elem_size(int32_t dtype) { return dtype == REL_BF16 ? 2 : 4; }

// A [B, H, T, D] tensor with the problem's strides, as a set of element offsets
// base + b*sb + h*sh + t*st + d.
struct Lattice {
  int64_t stride[4];
  int64_t count[4];
};

Lattice lattice_of(const rel_problem* p) {
  // ordered by decreasing stride so that the nested decomposition below works
  int64_t s[4] = {p->stride_b, p->stride_h, p->stride_t, 1};
  int64_t c[4] = {p->B, p->H, p->T, p->D};
  int idx[4] = {0, 1, 2, 3};
  std::sort(idx, idx + 3, [&](int a, int b) { return s[a] > s[b]; });
  Lattice L;
  for (int i = 0; i < 4; ++i) {
    L.stride[i] = s[idx[i]];
    L.count[i] = c[idx[i]];
  }
  return L;
}

// Strides are nested if each dimension's stride exceeds the span of all
// dimensions with smaller strides; then distinct indices never share memory.
bool nested(const Lattice& L) {
  int64_t span = 0;
  for (int i = 3; i >= 0; --i) {
    if (L.count[i] > 1 && L.stride[i] <= span) return false;
    span += (L.count[i] - 1) * L.stride[i];
  }
  return true;
}

// Is delta = sum_i c_i * stride_i with |c_i| < count_i ? (nested strides)
bool representable(const Lattice& L, int dim, int64_t delta) {
  if (dim == 3) return delta > -L.count[3] && delta < L.count[3];
  const int64_t s = L.stride[dim];
  if (L.count[dim] <= 1 || s == 0) return representable(L, dim + 1, delta);
  int64_t lo = delta / s;  // truncation; try the two neighbours of delta / s
  for (int64_t c : {lo - 1, lo, lo + 1}) {
    if (c <= -L.count[dim] || c >= L.count[dim]) continue;
    if (representable(L, dim + 1, delta - c * s)) return true;
  }
  return false;
}

int64_t extent_elems(const rel_problem* p) {
  return (p->B - 1) * p->stride_b + (p->H - 1) * p->stride_h + (p->T - 1) * p->stride_t + p->D;
}

struct Buf {
  const void* ptr;
  size_t bytes;       // byte range starting at ptr
  bool tensor;        // [B,H,T,D] lattice with the problem's strides
  bool output;
  const char* name;
};

bool ranges_overlap(const Buf& a, const Buf& b) {
  const uintptr_t a0 = (uintptr_t)a.ptr, b0 = (uintptr_t)b.ptr;
  return a0 < b0 + b.bytes && b0 < a0 + a.bytes;
}

bool aliases(const rel_problem* p, const Lattice& L, const Buf& a, const Buf& b) {
  if (!ranges_overlap(a, b)) return false;
  if (a.tensor && b.tensor) {
    const size_t es = elem_size(p->dtype);
    const int64_t delta = (int64_t)((intptr_t)b.ptr - (intptr_t)a.ptr);
    if (delta % (int64_t)es != 0) return true;
    return representable(L, 0, delta / (int64_t)es);
  }
  return true;
}

rel_status check_buffers(const rel_problem* p, const std::vector<Buf>& bufs) {
  const Lattice L = lattice_of(p);
  for (size_t i = 0; i < bufs.size(); ++i) {
    if (!bufs[i].ptr || !bufs[i].output) continue;
    for (size_t j = 0; j < bufs.size(); ++j) {
      if (i == j || !bufs[j].ptr) continue;
      if (bufs[j].output && j < i) continue;  // output pairs once
      if (aliases(p, L, bufs[i], bufs[j]))
        return fail(REL_ERR_INVALID_ARG, "output %s overlaps %s", bufs[i].name, bufs[j].name);
    }
  }
  return REL_OK;
}

// Problem-level validation shared by every entry point. Sets *empty when there
// is nothing to compute.
rel_status check_problem(const rel_problem* p, bool* empty) {
  if (!p) return fail(REL_ERR_INVALID_ARG, "problem is null");
  if (p->B < 0 || p->H < 0 || p->T < 0 || p->D < 0)
    return fail(REL_ERR_INVALID_ARG, "negative size B=%lld H=%lld T=%lld D=%lld", (long long)p->B,
                (long long)p->H, (long long)p->T, (long long)p->D);
  if (p->dtype != REL_F32 && p->dtype != REL_BF16)
    return fail(REL_ERR_UNSUPPORTED, "unknown dtype %d", (int)p->dtype);
  if (p->causal != 1)
    return fail(REL_ERR_UNSUPPORTED, "only the causal operator is defined (causal=%d)", (int)p->causal);
  if (!(std::isfinite(p->tau_s) && p->tau_s > 0.0f))
    return fail(REL_ERR_INVALID_ARG, "tau_s must be finite and > 0 (got %g)", (double)p->tau_s);
  if (!std::isfinite(p->scale)) return fail(REL_ERR_INVALID_ARG, "scale must be finite");
  if (p->D != 32 && p->D != 64 && p->D != 128 && !(p->D == 96 && p->dtype == REL_BF16))
    return fail(REL_ERR_UNSUPPORTED, "head dimension %lld not in {32, 64, 128} (or 96 for bf16)",
                (long long)p->D);
  *empty = (p->B == 0 || p->H == 0 || p->T == 0);
  if (*empty) return REL_OK;
  if (p->T > (1 << 24)) return fail(REL_ERR_UNSUPPORTED, "T = %lld exceeds 2^24", (long long)p->T);
  if (p->B * p->H > (1LL << 30)) return fail(REL_ERR_UNSUPPORTED, "B*H exceeds 2^30");
  const int64_t es = (int64_t)elem_size(p->dtype);
  const int64_t vec = 16 / es;  // elements per 16 bytes
  if (p->stride_t < p->D) return fail(REL_ERR_INVALID_ARG, "stride_t (%lld) < D", (long long)p->stride_t);
  if (p->stride_b < 0 || p->stride_h < 0) return fail(REL_ERR_INVALID_ARG, "negative stride");
  if (p->stride_t % vec || p->stride_h % vec || p->stride_b % vec)
    return fail(REL_ERR_INVALID_ARG, "strides must be multiples of 16 bytes");
  if (!nested(lattice_of(p)))
    return fail(REL_ERR_INVALID_ARG, "strides make distinct (b, h, t) rows overlap");
  // the kernels address the rows of one head with 32-bit byte offsets
  if (p->T * p->stride_t * es >= (1LL << 31))
    return fail(REL_ERR_UNSUPPORTED, "one head spans T * stride_t = %lld elements, over 2 GiB",
                (long long)(p->T * p->stride_t));
  return REL_OK;
}

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// Validation of the layer entry points: as check_problem, but any head width
// up to 128 (even with RoPE), element-aligned strides, and the option checks.
rel_status check_layer_problem(const rel_problem* p, const rel_layer_opts* o, bool* empty) {
  if (!p) return fail(REL_ERR_INVALID_ARG, "problem is null");
  if (!o) return fail(REL_ERR_INVALID_ARG, "layer options are null");
  if (p->B < 0 || p->H < 0 || p->T < 0 || p->D < 0)
    return fail(REL_ERR_INVALID_ARG, "negative size B=%lld H=%lld T=%lld D=%lld", (long long)p->B,
                (long long)p->H, (long long)p->T, (long long)p->D);
  if (p->dtype != REL_F32 && p->dtype != REL_BF16)
    return fail(REL_ERR_UNSUPPORTED, "unknown dtype %d", (int)p->dtype);
  if (p->causal != 1)
    return fail(REL_ERR_UNSUPPORTED, "only the causal operator is defined (causal=%d)", (int)p->causal);
  if (!(std::isfinite(p->tau_s) && p->tau_s > 0.0f))
    return fail(REL_ERR_INVALID_ARG, "tau_s must be finite and > 0 (got %g)", (double)p->tau_s);
  if (!std::isfinite(p->scale)) return fail(REL_ERR_INVALID_ARG, "scale must be finite");
  if (!(std::isfinite(o->rope_base) && o->rope_base >= 0.0))
    return fail(REL_ERR_INVALID_ARG, "rope_base must be finite and >= 0");
  if (o->rope_base > 0.0 && o->rope_base <= 1.0)
    return fail(REL_ERR_INVALID_ARG, "rope_base must exceed 1");
  if (o->givens < REL_GIVENS_NONE || o->givens > REL_GIVENS_B)
    return fail(REL_ERR_INVALID_ARG, "unknown Givens pairing %d", (int)o->givens);
  if (o->transport != REL_TRANSPORT_FULL && o->transport != REL_TRANSPORT_EXCHANGE)
    return fail(REL_ERR_INVALID_ARG, "unknown transport %d", (int)o->transport);
  if (p->D < 1 || p->D > 128)
    return fail(REL_ERR_UNSUPPORTED, "head width %lld not in 1..128", (long long)p->D);
  if (o->rope_base > 0.0 && p->D % 2)
    return fail(REL_ERR_INVALID_ARG, "RoPE needs an even head width (D = %lld)", (long long)p->D);
  if (o->givens != REL_GIVENS_NONE && p->H % 2)
    return fail(REL_ERR_INVALID_ARG, "Givens mixing pairs heads: H = %lld is odd", (long long)p->H);
  *empty = (p->B == 0 || p->H == 0 || p->T == 0);
  if (*empty) return REL_OK;
  if (p->T > (1 << 24)) return fail(REL_ERR_UNSUPPORTED, "T = %lld exceeds 2^24", (long long)p->T);
  if (p->B * p->H > (1LL << 30)) return fail(REL_ERR_UNSUPPORTED, "B*H exceeds 2^30");
  if (p->stride_t < p->D) return fail(REL_ERR_INVALID_ARG, "stride_t (%lld) < D", (long long)p->stride_t);
  if (p->stride_b < 0 || p->stride_h < 0) return fail(REL_ERR_INVALID_ARG, "negative stride");
  if (!nested(lattice_of(p)))
    return fail(REL_ERR_INVALID_ARG, "strides make distinct (b, h, t) rows overlap");
  const int64_t es = (int64_t)elem_size(p->dtype);
  if (p->T * std::max<int64_t>(p->stride_t, 128) * es >= (1LL << 31))
    return fail(REL_ERR_UNSUPPORTED, "one head spans over 2 GiB");
  return REL_OK;
}

// Memory plan of the layer entry points. The prepared operands (rotated q and
// k, mixed v, the forward's output, all contiguous [B, H, T, DP]) and the cos /
// sin table form the "prepared" region: the caller's saved buffer, or the
// start of the workspace. The backward pass's own scratch follows in the
// workspace. A pass-through layer (no RoPE, no mixing, a tiled width,
// contiguous tensors) has no prepared region and calls the operator directly.
constexpr size_t kNone = (size_t)-1;

struct LayerPlan {
  rel_problem pp;       // the problem the fused kernels see
  int64_t DP;
  bool pass;            // pass-through
  bool contiguous_tiled;  // the caller's layout equals the padded layout
  size_t tab, qr, kr, vt, yp, prep;                 // prepared region
  size_t dop, gq, gk, gv, bws, dth, dpart, scratch;  // backward scratch
};

LayerPlan plan_layer(const rel_problem* p, const rel_layer_opts* o) {
  LayerPlan L{};
  L.DP = p->D <= 32 ? 32 : p->D <= 64 ? 64 : (p->D <= 96 && p->dtype == REL_BF16) ? 96 : 128;
  const bool contiguous = p->stride_t == p->D && (p->H == 1 || p->stride_h == p->T * p->D) &&
                          (p->B == 1 || p->stride_b == p->H * p->T * p->D);
  const bool rope = o->rope_base > 0.0, giv = o->givens != REL_GIVENS_NONE;
  L.contiguous_tiled = contiguous && L.DP == p->D;
  L.pass = L.contiguous_tiled && !rope && !giv;
  L.pp = *p;
  L.pp.D = L.DP;
  L.pp.stride_t = L.DP;
  L.pp.stride_h = p->T * L.DP;
  L.pp.stride_b = p->H * p->T * L.DP;
  L.pp.scale = p->scale > 0.0f ? p->scale : 1.0f / std::sqrt((float)p->D);
  const size_t es = elem_size(p->dtype);
  const size_t tensor = align256((size_t)(p->B * p->H * p->T * L.DP) * es);
  size_t off = 0;
  auto take = [&](bool need, size_t bytes) {
    if (!need) return kNone;
    const size_t at = off;
    off += bytes;
    return at;
  };
  const bool prep = !L.pass;
  L.tab = take(prep && rope, align256((size_t)p->T * (size_t)(p->D / 2) * 8));
  L.qr = take(prep, tensor);
  L.kr = take(prep, tensor);
  L.vt = take(prep, tensor);
  L.yp = take(prep, tensor);
  L.prep = off;
  off = 0;
  L.dop = take(prep, tensor);
  L.gq = take(prep, tensor);
  L.gk = take(prep, tensor);
  L.gv = take(prep, tensor);
  L.bws = take(true, align256(relation_bwd_workspace_bytes(&L.pp)));
  L.dth = take(prep && giv, align256((size_t)(p->H / 2) * (size_t)p->B * (size_t)p->T * 4));
  L.dpart = take(prep && giv, align256((size_t)(p->H / 2) * (size_t)rel::layer_sum_parts() * 4));
  L.scratch = off;
  return L;
}

// The widest chunk (channels per thread) the caller's tensors allow: D, D/2
// (with RoPE) and the strides must be multiples of it, the pointers aligned to it.
int layer_vec(const rel_problem* p, const rel_layer_opts* o, std::initializer_list<const void*> ptrs) {
  const size_t es = elem_size(p->dtype);
  const int vmax = (int)(16 / es);
  for (int v : {vmax, 2, 1}) {
    bool ok = p->D % v == 0 && p->stride_t % v == 0 && p->stride_h % v == 0 && p->stride_b % v == 0;
    if (o->rope_base > 0.0) ok = ok && (p->D / 2) % v == 0;
    for (const void* x : ptrs) ok = ok && (uintptr_t)x % (v * es) == 0;
    if (ok) return v;
  }
  return 1;
}

rel_status check_aligned(const void* ptr, size_t align, const char* name, bool required) {
  if (!ptr) {
    if (required) return fail(REL_ERR_INVALID_ARG, "%s is null", name);
    return REL_OK;
  }
  if ((uintptr_t)ptr % align) return fail(REL_ERR_INVALID_ARG, "%s is not %zu-byte aligned", name, align);
  return REL_OK;
}

float eff_scale(const rel_problem* p) {
  return p->scale > 0.0f ? p->scale : 1.0f / std::sqrt((float)p->D);
}

bool test_fail_launch() {
  const char* e = std::getenv("RELATION_TEST_FAIL_LAUNCH");
  return e && e[0] == '1';
}

// rocBLAS handle shared by the materialised path, guarded by a mutex.
std::mutex g_blas_mu;
rocblas_handle g_blas = nullptr;
int g_blas_dev = -1;

// The rocBLAS handle of the current device, bound to `stream`. Call with
// g_blas_mu held.
rel_status blas_on_stream(void* stream) {
  int dev = 0;
  hipError_t he = hipGetDevice(&dev);
  if (he != hipSuccess) return hip_fail(he, "hipGetDevice");
  if (!g_blas || g_blas_dev != dev) {
    if (g_blas) rocblas_destroy_handle(g_blas);
    g_blas = nullptr;
    if (rocblas_create_handle(&g_blas) != rocblas_status_success)
      return fail(REL_ERR_HIP, "rocblas_create_handle failed");
    g_blas_dev = dev;
  }
  if (rocblas_set_stream(g_blas, (hipStream_t)stream) != rocblas_status_success)
    return fail(REL_ERR_HIP, "rocblas_set_stream failed");
  return REL_OK;
}

// Measurement aid state (relation_profile_arm).
std::mutex g_prof_mu;
std::string g_prof_name;
std::vector<hipEvent_t> g_prof_events;
int g_prof_next = 0;

}  // namespace

bool rel::profile_slot(const char* name, hipEvent_t* start, hipEvent_t* stop) {
  std::lock_guard<std::mutex> lock(g_prof_mu);
  if (g_prof_name.empty() || g_prof_name != name) return false;
  if (2 * (size_t)g_prof_next + 1 >= g_prof_events.size()) return false;
  *start = g_prof_events[2 * g_prof_next];
  *stop = g_prof_events[2 * g_prof_next + 1];
  ++g_prof_next;
  return true;
}

#define REL_TRY(x)                  \
  do {                              \
    rel_status _s = (x);            \
    if (_s != REL_OK) return _s;    \
  } while (0)

extern "C" {

int relation_abi_version(void) { return RELATION_ABI_VERSION; }

const char* relation_status_string(rel_status s) {
  switch (s) {
    case REL_OK: return "ok";
    case REL_ERR_INVALID_ARG: return "invalid argument";
    case REL_ERR_UNSUPPORTED: return "unsupported problem";
    case REL_ERR_WORKSPACE: return "workspace too small";
    case REL_ERR_HIP: return "HIP error";
    case REL_STATUS_MAX_ENUM: break;
  }
  return "unknown status";
}

const char* relation_last_error(void) { return g_last_error.c_str(); }

rel_status relation_profile_arm(const char* kernel, void** events, int n_pairs) {
  static const char* kNames[] = {"fwd", "bwd", "bwd_dkdv", "bwd_dq", "bwd_prep", "bwd_convert"};
  bool known = false;
  for (const char* nm : kNames) known = known || (kernel && std::string(kernel) == nm);
  if (!known) return fail(REL_ERR_INVALID_ARG, "unknown kernel name for profiling");
  if (n_pairs < 0 || (n_pairs > 0 && !events)) return fail(REL_ERR_INVALID_ARG, "bad event array");
  std::lock_guard<std::mutex> lock(g_prof_mu);
  g_prof_name = kernel;
  g_prof_events.clear();
  for (int i = 0; i < 2 * n_pairs; ++i) g_prof_events.push_back((hipEvent_t)events[i]);
  g_prof_next = 0;
  return REL_OK;
}

int64_t relation_mfma_peak_flops(int workgroups, int iters) {
  if (workgroups <= 0 || iters <= 0) return 0;
  return rel::mfma_peak_flops_per_launch(workgroups, iters);
}

rel_status relation_mfma_peak_probe(int workgroups, int iters, float* sink, unsigned long long* clocks,
                                    void* stream) {
  if (workgroups <= 0 || iters <= 0) return fail(REL_ERR_INVALID_ARG, "workgroups and iters must be > 0");
  if (!sink || !clocks) return fail(REL_ERR_INVALID_ARG, "sink and clocks are required");
  hipError_t e = rel::launch_mfma_peak(workgroups, iters, sink, clocks, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "relation_mfma_peak_probe launch");
  return REL_OK;
}

int relation_profile_disarm(void) {
  std::lock_guard<std::mutex> lock(g_prof_mu);
  const int n = g_prof_next;
  g_prof_name.clear();
  g_prof_events.clear();
  g_prof_next = 0;
  return n;
}

static rel_status fwd_impl(const rel_problem* p, const void* q, const void* k, const void* v,
                           const float* lambda, void* o, float* row_stat, float* self_mass,
                           float* exch_mass, float* exch_lse, void* stream, int exch_only) {
  bool empty = false;
  REL_TRY(check_problem(p, &empty));
  if (empty) return REL_OK;
  REL_TRY(check_aligned(q, 16, "q", true));
  REL_TRY(check_aligned(k, 16, "k", true));
  REL_TRY(check_aligned(v, 16, "v", true));
  REL_TRY(check_aligned(o, 16, "o", true));
  REL_TRY(check_aligned(lambda, 4, "lambda", true));
  REL_TRY(check_aligned(row_stat, 4, "row_stat", false));
  REL_TRY(check_aligned(self_mass, 4, "self_mass", false));
  REL_TRY(check_aligned(exch_mass, 4, "exch_mass", false));
  REL_TRY(check_aligned(exch_lse, 4, "exch_lse", false));
  const size_t es = elem_size(p->dtype);
  const size_t tb = (size_t)extent_elems(p) * es, rb = (size_t)(p->B * p->H * p->T) * 4;
  REL_TRY(check_buffers(p, {{q, tb, true, false, "q"},
                            {k, tb, true, false, "k"},
                            {v, tb, true, false, "v"},
                            {lambda, 4, false, false, "lambda"},
                            {o, tb, true, true, "o"},
                            {row_stat, rb, false, true, "row_stat"},
                            {self_mass, rb, false, true, "self_mass"},
                            {exch_mass, rb, false, true, "exch_mass"},
                            {exch_lse, rb, false, true, "exch_lse"}}));
  if (test_fail_launch()) return fail(REL_ERR_HIP, "launch failure injected by RELATION_TEST_FAIL_LAUNCH");
  rel::FwdArgs a{};
  a.q = q; a.k = k; a.v = v; a.lambda = lambda; a.o = o;
  a.row_stat = row_stat; a.self_mass = self_mass; a.exch_mass = exch_mass; a.exch_lse = exch_lse;
  a.sb = p->stride_b; a.sh = p->stride_h; a.st = p->stride_t;
  a.H = (int)p->H; a.T = (int)p->T;
  a.scale = eff_scale(p);
  a.exch_only = exch_only;
  a.inv_tau = 1.0f / p->tau_s;
  a.map = rel::make_tilemap((int)(p->B * p->H), 1);
  hipError_t e = rel::launch_fwd(a, p->dtype, (int)p->D, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "relation_fwd launch");
  return REL_OK;
}

rel_status relation_fwd(const rel_problem* p, const void* q, const void* k, const void* v,
                        const float* lambda, void* o, float* row_stat, float* self_mass,
                        float* exch_mass, float* exch_lse, void* stream) {
  return fwd_impl(p, q, k, v, lambda, o, row_stat, self_mass, exch_mass, exch_lse, stream, 0);
}

rel_status relation_exchange_allocation(const rel_problem* p, const void* q, const void* k,
                                        const float* exch_lse, float* pi, void* stream) {
  bool empty = false;
  REL_TRY(check_problem(p, &empty));
  if (empty) return REL_OK;
  REL_TRY(check_aligned(q, 16, "q", true));
  REL_TRY(check_aligned(k, 16, "k", true));
  REL_TRY(check_aligned(exch_lse, 4, "exch_lse", true));
  REL_TRY(check_aligned(pi, 4, "pi", true));
  const size_t es = elem_size(p->dtype);
  const size_t tb = (size_t)extent_elems(p) * es, rb = (size_t)(p->B * p->H * p->T) * 4;
  const size_t mb = (size_t)(p->B * p->H) * (size_t)p->T * (size_t)p->T * 4;
  REL_TRY(check_buffers(p, {{q, tb, true, false, "q"},
                            {k, tb, true, false, "k"},
                            {exch_lse, rb, false, false, "exch_lse"},
                            {pi, mb, false, true, "pi"}}));
  if (test_fail_launch()) return fail(REL_ERR_HIP, "launch failure injected by RELATION_TEST_FAIL_LAUNCH");
  rel::RowArgs a{};
  a.q = q; a.k = k; a.exch_lse = exch_lse; a.pi = pi;
  a.sb = p->stride_b; a.sh = p->stride_h; a.st = p->stride_t;
  a.H = (int)p->H; a.T = (int)p->T; a.D = (int)p->D;
  a.scale = eff_scale(p);
  a.inv_tau = 1.0f / p->tau_s;
  hipError_t e = rel::launch_allocation(a, p->dtype, (int)(p->B * p->H), (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "relation_exchange_allocation launch");
  return REL_OK;
}


}  // extern "C"

namespace {
// Backward workspace of one path (valid, non-empty problem): -D_i and
// M_i log2(e) per row, the dlambda partials, and for the fused path the fp32
// dQ accumulator.
size_t bwd_workspace(const rel_problem* p, bool fused) {
  const size_t N = (size_t)(p->B * p->H), rows = N * (size_t)p->T;
  size_t b = 2 * align256(rows * 4) +
             align256((size_t)rel::bwd_partials((int)N, (int)p->T, (int)p->D, p->dtype, fused) * 4);
  if (fused) b += align256(rows * (size_t)p->D * 4);
  return b;
}
bool bwd_fused(const rel_problem* p) { return rel::bwd_fused_supported((int)p->T, (int)p->D, p->dtype); }
}  // namespace

extern "C" {

size_t relation_bwd_workspace_bytes(const rel_problem* p) {
  bool empty = false;
  if (check_problem(p, &empty) != REL_OK) return 0;
  if (empty) return 0;
  const size_t two = bwd_workspace(p, false);
  return bwd_fused(p) ? std::max(two, bwd_workspace(p, true)) : two;
}

// fused: take the one-kernel backward where it covers the problem (dq summed
// by atomics); otherwise, and with fused = false, the two-kernel backward.
static rel_status bwd_impl(const rel_problem* p, const void* q, const void* k, const void* v,
                           const void* o, const void* dout, const float* lambda,
                           const float* row_stat, void* dq, void* dk, void* dv, float* dlambda,
                           float* dself, void* workspace, size_t workspace_bytes, void* stream,
                           int exch_only, bool fused) {
  bool empty = false;
  REL_TRY(check_problem(p, &empty));
  if (empty) {
    if (dlambda) {
      // nothing to differentiate: dlambda is still an output and must be zero
      if (test_fail_launch()) return fail(REL_ERR_HIP, "launch failure injected");
      hipError_t e = rel::launch_fill_zero(dlambda, 1, (hipStream_t)stream);
      if (e != hipSuccess) return hip_fail(e, "relation_bwd dlambda clear");
    }
    return REL_OK;
  }
  REL_TRY(check_aligned(q, 16, "q", true));
  REL_TRY(check_aligned(k, 16, "k", true));
  REL_TRY(check_aligned(v, 16, "v", true));
  REL_TRY(check_aligned(o, 16, "o", true));
  REL_TRY(check_aligned(dout, 16, "dout", true));
  REL_TRY(check_aligned(dq, 16, "dq", true));
  REL_TRY(check_aligned(dk, 16, "dk", true));
  REL_TRY(check_aligned(dv, 16, "dv", true));
  REL_TRY(check_aligned(lambda, 4, "lambda", true));
  REL_TRY(check_aligned(row_stat, 4, "row_stat", true));
  REL_TRY(check_aligned(dlambda, 4, "dlambda", true));
  REL_TRY(check_aligned(dself, 4, "dself", false));
  fused = fused && bwd_fused(p);
  const size_t need = bwd_workspace(p, fused);
  if (!workspace || workspace_bytes < need)
    return fail(REL_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", need,
                workspace ? workspace_bytes : (size_t)0);
  if ((uintptr_t)workspace % 16) return fail(REL_ERR_INVALID_ARG, "workspace is not 16-byte aligned");
  const size_t es = elem_size(p->dtype);
  const size_t tb = (size_t)extent_elems(p) * es, rb = (size_t)(p->B * p->H * p->T) * 4;
  REL_TRY(check_buffers(p, {{q, tb, true, false, "q"},
                            {k, tb, true, false, "k"},
                            {v, tb, true, false, "v"},
                            {o, tb, true, false, "o"},
                            {dout, tb, true, false, "dout"},
                            {lambda, 4, false, false, "lambda"},
                            {row_stat, rb, false, false, "row_stat"},
                            {dq, tb, true, true, "dq"},
                            {dk, tb, true, true, "dk"},
                            {dv, tb, true, true, "dv"},
                            {dlambda, 4, false, true, "dlambda"},
                            {dself, rb, false, true, "dself"},
                            {workspace, need, false, true, "workspace"}}));
  if (test_fail_launch()) return fail(REL_ERR_HIP, "launch failure injected by RELATION_TEST_FAIL_LAUNCH");
  const size_t N = (size_t)(p->B * p->H);
  rel::BwdArgs a{};
  a.q = q; a.k = k; a.v = v; a.o = o; a.dout = dout; a.lambda = lambda; a.row_stat = row_stat;
  a.dq = dq; a.dk = dk; a.dv = dv; a.dself = dself;
  const size_t rowv = align256(N * (size_t)p->T * 4);
  const int nparts = rel::bwd_partials((int)N, (int)p->T, (int)p->D, p->dtype, fused);
  a.negd = (float*)workspace;
  a.m2 = (float*)((char*)workspace + rowv);
  a.dlam_part = (float*)((char*)workspace + 2 * rowv);
  a.dq_acc = fused ? (float*)((char*)workspace + 2 * rowv + align256((size_t)nparts * 4)) : nullptr;
  a.sb = p->stride_b; a.sh = p->stride_h; a.st = p->stride_t;
  a.H = (int)p->H; a.T = (int)p->T;
  a.scale = eff_scale(p);
  a.exch_only = exch_only;
  a.inv_tau = 1.0f / p->tau_s;
  a.map = rel::make_tilemap((int)N, 1);
  a.nparts = nparts;
  a.dlambda = dlambda;
  hipError_t e = rel::launch_bwd(a, p->dtype, (int)p->D, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "relation_bwd launch");
  return REL_OK;
}

rel_status relation_bwd(const rel_problem* p, const void* q, const void* k, const void* v,
                        const void* o, const void* dout, const float* lambda,
                        const float* row_stat, void* dq, void* dk, void* dv, float* dlambda,
                        float* dself, void* workspace, size_t workspace_bytes, void* stream) {
  return bwd_impl(p, q, k, v, o, dout, lambda, row_stat, dq, dk, dv, dlambda, dself, workspace,
                  workspace_bytes, stream, 0, true);
}

rel_status relation_bwd_deterministic(const rel_problem* p, const void* q, const void* k, const void* v,
                                      const void* o, const void* dout, const float* lambda,
                                      const float* row_stat, void* dq, void* dk, void* dv, float* dlambda,
                                      float* dself, void* workspace, size_t workspace_bytes, void* stream) {
  return bwd_impl(p, q, k, v, o, dout, lambda, row_stat, dq, dk, dv, dlambda, dself, workspace,
                  workspace_bytes, stream, 0, false);
}

}  // extern "C"

// ---------------------------------------------------------------------------
// Scratch of the backward pass without a caller workspace: a file-scope device
// array, one copy per GPU, held until the process ends. Host code never passes
// the array's name to a kernel or a copy: it is a host-side stand-in. The
// device address of each GPU's copy comes from hipGetSymbolAddress, taken once
// per device with that device current, and only that address is used.
// ---------------------------------------------------------------------------
static constexpr size_t kNoAllocScratchBytes = 32u << 20;
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// The device address of the current device's copy of `scratch`.
rel_status scratch_address(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices) return fail(REL_ERR_UNSUPPORTED, "device index %d >= %d", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
    if (!ptr) return fail(REL_ERR_HIP, "hipGetSymbolAddress(scratch) returned null");
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return REL_OK;
}
}  // namespace

extern "C" {

size_t relation_bwd_noalloc_max_scratch_bytes(void) { return kNoAllocScratchBytes; }

rel_status relation_bwd_noalloc(const rel_problem* p, const void* q, const void* k, const void* v,
                                const void* o, const void* dout, const float* lambda,
                                const float* row_stat, void* dq, void* dk, void* dv, float* dlambda,
                                float* dself, void* stream) {
  // the same per-row scratch relation_bwd takes from its workspace; its
  // contents on entry are ignored (every word read is written first)
  // 0 for an empty or invalid problem (bwd_impl then reports it)
  const size_t need = relation_bwd_workspace_bytes(p) ? bwd_workspace(p, false) : 0;
  void* ws = nullptr;
  if (need > 0) {
    if (need > kNoAllocScratchBytes)
      return fail(REL_ERR_WORKSPACE,
                  "relation_bwd_noalloc: the problem needs %zu bytes of scratch, over the %zu bytes "
                  "this entry point holds per device",
                  need, kNoAllocScratchBytes);
    REL_TRY(scratch_address(&ws));
  }
  return bwd_impl(p, q, k, v, o, dout, lambda, row_stat, dq, dk, dv, dlambda, dself, ws,
                  need > 0 ? kNoAllocScratchBytes : 0, stream, 0, false);
}

size_t relation_fwd_materialized_workspace_bytes(const rel_problem* p) {
  bool empty = false;
  if (check_problem(p, &empty) != REL_OK) return 0;
  if (empty) return 0;
  const size_t NTT = (size_t)(p->B * p->H) * (size_t)p->T * (size_t)p->T;
  return align256(NTT * 4) + align256(NTT * elem_size(p->dtype));
}

rel_status relation_fwd_materialized(const rel_problem* p, const void* q, const void* k,
                                     const void* v, const float* lambda, void* o, float* R,
                                     float* F, float* pi, float* self_mass, float* exch_mass,
                                     void* workspace, size_t workspace_bytes, void* stream) {
  bool empty = false;
  REL_TRY(check_problem(p, &empty));
  if (empty) return REL_OK;
  REL_TRY(check_aligned(q, 16, "q", true));
  REL_TRY(check_aligned(k, 16, "k", true));
  REL_TRY(check_aligned(v, 16, "v", true));
  REL_TRY(check_aligned(o, 16, "o", true));
  REL_TRY(check_aligned(lambda, 4, "lambda", true));
  REL_TRY(check_aligned(R, 4, "R", false));
  REL_TRY(check_aligned(F, 4, "F", false));
  REL_TRY(check_aligned(pi, 4, "pi", false));
  REL_TRY(check_aligned(self_mass, 4, "self_mass", false));
  REL_TRY(check_aligned(exch_mass, 4, "exch_mass", false));
  if (p->T > 65536 || (p->T * (int64_t)p->T) > (1LL << 31))
    return fail(REL_ERR_UNSUPPORTED, "materialised path limited to T <= 65536 and T*T <= 2^31 per head");
  const size_t need = relation_fwd_materialized_workspace_bytes(p);
  if (!workspace || workspace_bytes < need)
    return fail(REL_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", need,
                workspace ? workspace_bytes : (size_t)0);
  if ((uintptr_t)workspace % 16) return fail(REL_ERR_INVALID_ARG, "workspace is not 16-byte aligned");
  const size_t es = elem_size(p->dtype);
  const size_t tb = (size_t)extent_elems(p) * es, rb = (size_t)(p->B * p->H * p->T) * 4;
  const size_t N = (size_t)(p->B * p->H);
  const size_t mb = N * (size_t)p->T * (size_t)p->T * 4;
  REL_TRY(check_buffers(p, {{q, tb, true, false, "q"},
                            {k, tb, true, false, "k"},
                            {v, tb, true, false, "v"},
                            {lambda, 4, false, false, "lambda"},
                            {o, tb, true, true, "o"},
                            {R, mb, false, true, "R"},
                            {F, mb, false, true, "F"},
                            {pi, mb, false, true, "pi"},
                            {self_mass, rb, false, true, "self_mass"},
                            {exch_mass, rb, false, true, "exch_mass"},
                            {workspace, need, false, true, "workspace"}}));
  if (test_fail_launch()) return fail(REL_ERR_HIP, "launch failure injected by RELATION_TEST_FAIL_LAUNCH");

  const int T = (int)p->T, D = (int)p->D;
  const float scale = eff_scale(p);
  float* U = (float*)workspace;
  void* Fw = (char*)workspace + align256(N * (size_t)T * (size_t)T * 4);
  const rocblas_datatype io = p->dtype == REL_BF16 ? rocblas_datatype_bf16_r : rocblas_datatype_f32_r;

  std::lock_guard<std::mutex> lock(g_blas_mu);
  REL_TRY(blas_on_stream(stream));
  hipError_t he = hipSuccess;

  const float one = 1.0f, zero = 0.0f;
  // Heads of one batch index are equally spaced by stride_h, so each GEMM call
  // batches over H; the calls loop over B.
  for (int64_t b = 0; b < p->B; ++b) {
    const char* qb = (const char*)q + (size_t)(b * p->stride_b) * es;
    const char* kb = (const char*)k + (size_t)(b * p->stride_b) * es;
    float* Ub = U + (size_t)b * p->H * T * (size_t)T;
    // column-major view: U^T (T x T) = K Q^T  ->  row-major U = scale * Q K^T (eq. 1)
    rocblas_status st = rocblas_gemm_strided_batched_ex(
        g_blas, rocblas_operation_transpose, rocblas_operation_none, T, T, D, &scale, kb, io,
        (rocblas_int)p->stride_t, p->stride_h, qb, io, (rocblas_int)p->stride_t, p->stride_h, &zero,
        Ub, rocblas_datatype_f32_r, T, (rocblas_stride)T * T, Ub, rocblas_datatype_f32_r, T,
        (rocblas_stride)T * T, (rocblas_int)p->H, rocblas_datatype_f32_r, rocblas_gemm_algo_standard,
        0, 0);
    if (st != rocblas_status_success) return fail(REL_ERR_HIP, "rocBLAS U GEMM failed (%d)", (int)st);
  }
  rel::RowArgs a{};
  a.U = U; a.lambda = lambda; a.Fw = Fw; a.R = R; a.F = F; a.pi = pi;
  a.self_mass = self_mass; a.exch_mass = exch_mass;
  a.H = (int)p->H; a.T = T; a.D = D;
  a.scale = scale;
  a.inv_tau = 1.0f / p->tau_s;
  he = rel::launch_materialized_rows(a, p->dtype, (int)N, (hipStream_t)stream);
  if (he != hipSuccess) return hip_fail(he, "materialised row kernel launch");
  for (int64_t b = 0; b < p->B; ++b) {
    const char* vb = (const char*)v + (size_t)(b * p->stride_b) * es;
    char* ob = (char*)o + (size_t)(b * p->stride_b) * es;
    const char* Fb = (const char*)Fw + (size_t)b * p->H * T * (size_t)T * es;
    // column-major view: Y^T (D x T) = V^T F^T  ->  row-major Y = F V (eq. 3)
    rocblas_status st = rocblas_gemm_strided_batched_ex(
        g_blas, rocblas_operation_none, rocblas_operation_none, D, T, T, &one, vb, io,
        (rocblas_int)p->stride_t, p->stride_h, Fb, io, T, (rocblas_stride)T * T, &zero, ob, io,
        (rocblas_int)p->stride_t, p->stride_h, ob, io, (rocblas_int)p->stride_t, p->stride_h,
        (rocblas_int)p->H, rocblas_datatype_f32_r, rocblas_gemm_algo_standard, 0, 0);
    if (st != rocblas_status_success) return fail(REL_ERR_HIP, "rocBLAS F.V GEMM failed (%d)", (int)st);
  }
  return REL_OK;
}

size_t relation_bwd_materialized_workspace_bytes(const rel_problem* p) {
  bool empty = false;
  if (check_problem(p, &empty) != REL_OK) return 0;
  if (empty) return 0;
  const size_t N = (size_t)(p->B * p->H);
  const size_t NTT = N * (size_t)p->T * (size_t)p->T;
  const size_t es = elem_size(p->dtype);
  return 2 * align256(NTT * 4) + 2 * align256(NTT * es) + align256(N * (size_t)p->T * 4) +
         align256((size_t)rel::sum_fixed_order_parts() * 4);
}

rel_status relation_bwd_materialized(const rel_problem* p, const void* q, const void* k,
                                     const void* v, const void* dout, const float* lambda, void* dq,
                                     void* dk, void* dv, float* dlambda, void* workspace,
                                     size_t workspace_bytes, void* stream) {
  bool empty = false;
  REL_TRY(check_problem(p, &empty));
  if (empty) {
    if (dlambda) {
      if (test_fail_launch()) return fail(REL_ERR_HIP, "launch failure injected");
      hipError_t e = rel::launch_fill_zero(dlambda, 1, (hipStream_t)stream);
      if (e != hipSuccess) return hip_fail(e, "relation_bwd_materialized dlambda clear");
    }
    return REL_OK;
  }
  REL_TRY(check_aligned(q, 16, "q", true));
  REL_TRY(check_aligned(k, 16, "k", true));
  REL_TRY(check_aligned(v, 16, "v", true));
  REL_TRY(check_aligned(dout, 16, "dout", true));
  REL_TRY(check_aligned(dq, 16, "dq", true));
  REL_TRY(check_aligned(dk, 16, "dk", true));
  REL_TRY(check_aligned(dv, 16, "dv", true));
  REL_TRY(check_aligned(lambda, 4, "lambda", true));
  REL_TRY(check_aligned(dlambda, 4, "dlambda", true));
  if (p->T > 65536 || (p->T * (int64_t)p->T) > (1LL << 31))
    return fail(REL_ERR_UNSUPPORTED, "materialised path limited to T <= 65536 and T*T <= 2^31 per head");
  const size_t need = relation_bwd_materialized_workspace_bytes(p);
  if (!workspace || workspace_bytes < need)
    return fail(REL_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", need,
                workspace ? workspace_bytes : (size_t)0);
  if ((uintptr_t)workspace % 16) return fail(REL_ERR_INVALID_ARG, "workspace is not 16-byte aligned");
  const size_t es = elem_size(p->dtype);
  const size_t tb = (size_t)extent_elems(p) * es;
  REL_TRY(check_buffers(p, {{q, tb, true, false, "q"},
                            {k, tb, true, false, "k"},
                            {v, tb, true, false, "v"},
                            {dout, tb, true, false, "dout"},
                            {lambda, 4, false, false, "lambda"},
                            {dq, tb, true, true, "dq"},
                            {dk, tb, true, true, "dk"},
                            {dv, tb, true, true, "dv"},
                            {dlambda, 4, false, true, "dlambda"},
                            {workspace, need, false, true, "workspace"}}));
  if (test_fail_launch()) return fail(REL_ERR_HIP, "launch failure injected by RELATION_TEST_FAIL_LAUNCH");

  const int T = (int)p->T, D = (int)p->D;
  const size_t N = (size_t)(p->B * p->H);
  const size_t NTT = N * (size_t)T * (size_t)T;
  const float scale = eff_scale(p);
  char* ws = (char*)workspace;
  float* U = (float*)ws;
  float* Hm = (float*)(ws + align256(NTT * 4));
  void* dUw = ws + 2 * align256(NTT * 4);
  void* Fw = ws + 2 * align256(NTT * 4) + align256(NTT * es);
  float* dlam_row = (float*)(ws + 2 * align256(NTT * 4) + 2 * align256(NTT * es));
  float* dlam_part = (float*)((char*)dlam_row + align256(N * (size_t)T * 4));
  const rocblas_datatype io = p->dtype == REL_BF16 ? rocblas_datatype_bf16_r : rocblas_datatype_f32_r;
  const rocblas_stride sTT = (rocblas_stride)T * T;
  const rocblas_int ld = (rocblas_int)p->stride_t, nh = (rocblas_int)p->H;

  std::lock_guard<std::mutex> lock(g_blas_mu);
  REL_TRY(blas_on_stream(stream));
  const float one = 1.0f, zero = 0.0f;
  // Row-major T x T results are column-major transposes: X^T = B^T A^T.
  for (int64_t b = 0; b < p->B; ++b) {
    const size_t off = (size_t)(b * p->stride_b) * es;
    const char *qb = (const char*)q + off, *kb = (const char*)k + off, *vb = (const char*)v + off;
    const char* gb = (const char*)dout + off;
    float* Ub = U + (size_t)b * p->H * T * (size_t)T;
    float* Hb = Hm + (size_t)b * p->H * T * (size_t)T;
    // U = scale q k^T (eq. 1) and H = dout v^T
    rocblas_status st = rocblas_gemm_strided_batched_ex(
        g_blas, rocblas_operation_transpose, rocblas_operation_none, T, T, D, &scale, kb, io, ld, p->stride_h,
        qb, io, ld, p->stride_h, &zero, Ub, rocblas_datatype_f32_r, T, sTT, Ub, rocblas_datatype_f32_r, T, sTT, nh,
        rocblas_datatype_f32_r, rocblas_gemm_algo_standard, 0, 0);
    if (st != rocblas_status_success) return fail(REL_ERR_HIP, "rocBLAS U GEMM failed (%d)", (int)st);
    st = rocblas_gemm_strided_batched_ex(
        g_blas, rocblas_operation_transpose, rocblas_operation_none, T, T, D, &one, vb, io, ld, p->stride_h, gb,
        io, ld, p->stride_h, &zero, Hb, rocblas_datatype_f32_r, T, sTT, Hb, rocblas_datatype_f32_r, T, sTT, nh,
        rocblas_datatype_f32_r, rocblas_gemm_algo_standard, 0, 0);
    if (st != rocblas_status_success) return fail(REL_ERR_HIP, "rocBLAS H GEMM failed (%d)", (int)st);
  }
  rel::RowBwdArgs a{};
  a.U = U; a.Hm = Hm; a.lambda = lambda; a.dUw = dUw; a.Fw = Fw; a.dlam_row = dlam_row;
  a.T = T;
  a.inv_tau = 1.0f / p->tau_s;
  hipError_t he = rel::launch_materialized_bwd_rows(a, p->dtype, (int)N, (hipStream_t)stream);
  if (he != hipSuccess) return hip_fail(he, "materialised backward row kernel launch");
  for (int64_t b = 0; b < p->B; ++b) {
    const size_t off = (size_t)(b * p->stride_b) * es;
    const char *qb = (const char*)q + off, *kb = (const char*)k + off, *gb = (const char*)dout + off;
    char *dqb = (char*)dq + off, *dkb = (char*)dk + off, *dvb = (char*)dv + off;
    const char* dUb = (const char*)dUw + (size_t)b * p->H * T * (size_t)T * es;
    const char* Fb = (const char*)Fw + (size_t)b * p->H * T * (size_t)T * es;
    // dq^T (D x T) = k^T dU^T: row-major dq = scale dU k
    rocblas_status st = rocblas_gemm_strided_batched_ex(
        g_blas, rocblas_operation_none, rocblas_operation_none, D, T, T, &scale, kb, io, ld, p->stride_h, dUb,
        io, T, sTT, &zero, dqb, io, ld, p->stride_h, dqb, io, ld, p->stride_h, nh, rocblas_datatype_f32_r,
        rocblas_gemm_algo_standard, 0, 0);
    if (st != rocblas_status_success) return fail(REL_ERR_HIP, "rocBLAS dq GEMM failed (%d)", (int)st);
    // dk^T (D x T) = q^T dU: row-major dk = scale dU^T q
    st = rocblas_gemm_strided_batched_ex(
        g_blas, rocblas_operation_none, rocblas_operation_transpose, D, T, T, &scale, qb, io, ld, p->stride_h,
        dUb, io, T, sTT, &zero, dkb, io, ld, p->stride_h, dkb, io, ld, p->stride_h, nh, rocblas_datatype_f32_r,
        rocblas_gemm_algo_standard, 0, 0);
    if (st != rocblas_status_success) return fail(REL_ERR_HIP, "rocBLAS dk GEMM failed (%d)", (int)st);
    // dv^T (D x T) = dout^T F: row-major dv = F^T dout
    st = rocblas_gemm_strided_batched_ex(
        g_blas, rocblas_operation_none, rocblas_operation_transpose, D, T, T, &one, gb, io, ld, p->stride_h, Fb,
        io, T, sTT, &zero, dvb, io, ld, p->stride_h, dvb, io, ld, p->stride_h, nh, rocblas_datatype_f32_r,
        rocblas_gemm_algo_standard, 0, 0);
    if (st != rocblas_status_success) return fail(REL_ERR_HIP, "rocBLAS dv GEMM failed (%d)", (int)st);
  }
  he = rel::launch_sum_fixed_order(dlam_row, (int64_t)N * T, dlam_part, dlambda, (hipStream_t)stream);
  if (he != hipSuccess) return hip_fail(he, "dlambda reduction launch");
  return REL_OK;
}

bool al16(std::initializer_list<const void*> ps) {
  for (const void* x : ps)
    if ((uintptr_t)x % 16) return false;
  return true;
}

rel::LayerArgs layer_args(const rel_problem* p, const rel_layer_opts* o, const LayerPlan& L, char* prep,
                          const void* q, const void* k, const void* v, const float* theta) {
  rel::LayerArgs a{};
  a.q = q; a.k = k; a.v = v;
  a.sb = p->stride_b; a.sh = p->stride_h; a.st = p->stride_t;
  a.qr = prep + L.qr;
  a.kr = prep + L.kr;
  a.vt = prep + L.vt;
  a.rope = L.tab != kNone ? (const float2*)(prep + L.tab) : nullptr;
  a.theta = theta;
  a.givens = o->givens;
  a.B = (int)p->B; a.H = (int)p->H; a.T = (int)p->T; a.D = (int)p->D; a.DP = (int)L.DP;
  return a;
}

size_t relation_layer_saved_bytes(const rel_problem* p, const rel_layer_opts* opts) {
  bool empty = false;
  if (check_layer_problem(p, opts, &empty) != REL_OK || empty) return 0;
  return plan_layer(p, opts).prep;
}

size_t relation_layer_fwd_workspace_bytes(const rel_problem* p, const rel_layer_opts* opts) {
  return relation_layer_saved_bytes(p, opts);
}

size_t relation_layer_bwd_workspace_bytes(const rel_problem* p, const rel_layer_opts* opts) {
  bool empty = false;
  if (check_layer_problem(p, opts, &empty) != REL_OK || empty) return 0;
  const LayerPlan L = plan_layer(p, opts);
  return L.prep + L.scratch;
}

rel_status relation_layer_fwd(const rel_problem* p, const rel_layer_opts* opts, const void* q,
                              const void* k, const void* v, const float* lambda, const float* theta,
                              void* out, float* row_stat, void* saved, size_t saved_bytes,
                              void* workspace, size_t workspace_bytes, void* stream) {
  bool empty = false;
  REL_TRY(check_layer_problem(p, opts, &empty));
  if (empty) return REL_OK;
  const size_t es = elem_size(p->dtype);
  const bool giv = opts->givens != REL_GIVENS_NONE;
  REL_TRY(check_aligned(q, es, "q", true));
  REL_TRY(check_aligned(k, es, "k", true));
  REL_TRY(check_aligned(v, es, "v", true));
  REL_TRY(check_aligned(out, es, "out", true));
  REL_TRY(check_aligned(lambda, 4, "lambda", true));
  REL_TRY(check_aligned(theta, 4, "theta", giv));
  REL_TRY(check_aligned(row_stat, 4, "row_stat", false));
  REL_TRY(check_aligned(saved, 16, "saved", false));
  const LayerPlan L = plan_layer(p, opts);
  if (L.pass)
    return fwd_impl(&L.pp, q, k, v, lambda, out, row_stat, nullptr, nullptr, nullptr, stream, opts->transport);
  if (saved && saved_bytes < L.prep)
    return fail(REL_ERR_WORKSPACE, "saved buffer of %zu bytes needed, %zu given", L.prep, saved_bytes);
  char* prep = (char*)saved;
  if (!prep) {
    if (!workspace || workspace_bytes < L.prep)
      return fail(REL_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", L.prep,
                  workspace ? workspace_bytes : (size_t)0);
    REL_TRY(check_aligned(workspace, 16, "workspace", true));
    prep = (char*)workspace;
  }
  const size_t tb = (size_t)extent_elems(p) * es, rb = (size_t)(p->B * p->H * p->T) * 4;
  REL_TRY(check_buffers(p, {{q, tb, true, false, "q"},
                            {k, tb, true, false, "k"},
                            {v, tb, true, false, "v"},
                            {lambda, 4, false, false, "lambda"},
                            {giv ? theta : nullptr, (size_t)(p->H / 2) * 4, false, false, "theta"},
                            {out, tb, true, true, "out"},
                            {row_stat, rb, false, true, "row_stat"},
                            {prep, L.prep, false, true, "saved / workspace"}}));
  if (test_fail_launch()) return fail(REL_ERR_HIP, "launch failure injected by RELATION_TEST_FAIL_LAUNCH");
  const hipStream_t s = (hipStream_t)stream;
  const rel::LayerArgs a = layer_args(p, opts, L, prep, q, k, v, theta);
  const int vec = layer_vec(p, opts, {q, k, v, out});
  hipError_t he = hipSuccess;
  if (a.rope && (he = rel::launch_rope_table((float2*)a.rope, (int)p->T, (int)p->D, opts->rope_base, s)))
    return hip_fail(he, "RoPE table launch");
  if ((he = rel::launch_layer_prologue(a, p->dtype, vec, s))) return hip_fail(he, "layer prologue launch");
  // the output goes straight to the caller when its layout is the padded one
  const bool y_direct = L.contiguous_tiled && al16({out});
  void* y = y_direct ? out : prep + L.yp;
  REL_TRY(fwd_impl(&L.pp, a.qr, a.kr, a.vt, lambda, y, row_stat, nullptr, nullptr, nullptr, stream,
                   opts->transport));
  if (!y_direct && (he = rel::launch_layer_repad(y, out, a, false, p->dtype, vec, s)))
    return hip_fail(he, "layer output copy launch");
  return REL_OK;
}

rel_status relation_layer_bwd(const rel_problem* p, const rel_layer_opts* opts, const void* q,
                              const void* k, const void* v, const void* out, const void* dout,
                              const float* lambda, const float* theta, const float* row_stat,
                              const void* saved, size_t saved_bytes, void* dq, void* dk, void* dv,
                              float* dlambda, float* dtheta, void* workspace, size_t workspace_bytes,
                              void* stream) {
  bool empty = false;
  REL_TRY(check_layer_problem(p, opts, &empty));
  const bool giv = opts->givens != REL_GIVENS_NONE;
  const hipStream_t s = (hipStream_t)stream;
  if (empty) {
    // nothing to differentiate: dlambda and dtheta are still outputs and must be zero
    if (test_fail_launch() && (dlambda || (giv && dtheta))) return fail(REL_ERR_HIP, "launch failure injected");
    hipError_t e = hipSuccess;
    if (dlambda && (e = rel::launch_fill_zero(dlambda, 1, s))) return hip_fail(e, "dlambda clear");
    if (giv && dtheta && p->H > 0 && (e = rel::launch_fill_zero(dtheta, p->H / 2, s)))
      return hip_fail(e, "dtheta clear");
    return REL_OK;
  }
  const size_t es = elem_size(p->dtype);
  REL_TRY(check_aligned(q, es, "q", true));
  REL_TRY(check_aligned(k, es, "k", true));
  REL_TRY(check_aligned(v, es, "v", true));
  REL_TRY(check_aligned(out, es, "out", true));
  REL_TRY(check_aligned(dout, es, "dout", true));
  REL_TRY(check_aligned(dq, es, "dq", true));
  REL_TRY(check_aligned(dk, es, "dk", true));
  REL_TRY(check_aligned(dv, es, "dv", true));
  REL_TRY(check_aligned(lambda, 4, "lambda", true));
  REL_TRY(check_aligned(row_stat, 4, "row_stat", true));
  REL_TRY(check_aligned(dlambda, 4, "dlambda", true));
  REL_TRY(check_aligned(theta, 4, "theta", giv));
  REL_TRY(check_aligned(dtheta, 4, "dtheta", giv));
  REL_TRY(check_aligned(saved, 16, "saved", false));
  const LayerPlan L = plan_layer(p, opts);
  if (saved && !L.pass && saved_bytes < L.prep)
    return fail(REL_ERR_WORKSPACE, "saved buffer of %zu bytes needed, %zu given", L.prep, saved_bytes);
  const size_t need = (saved || L.pass ? 0 : L.prep) + L.scratch;
  if (!workspace || workspace_bytes < need)
    return fail(REL_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", need,
                workspace ? workspace_bytes : (size_t)0);
  REL_TRY(check_aligned(workspace, 16, "workspace", true));
  char* ws = (char*)workspace;
  if (L.pass)
    return bwd_impl(&L.pp, q, k, v, out, dout, lambda, row_stat, dq, dk, dv, dlambda, nullptr, ws + L.bws,
                    relation_bwd_workspace_bytes(&L.pp), stream, opts->transport, true);
  char* prep = saved ? (char*)saved : ws;
  char* scr = saved ? ws : ws + L.prep;
  const size_t tb = (size_t)extent_elems(p) * es, rb = (size_t)(p->B * p->H * p->T) * 4;
  const size_t thb = (size_t)(p->H / 2) * 4;
  REL_TRY(check_buffers(p, {{q, tb, true, false, "q"},
                            {k, tb, true, false, "k"},
                            {v, tb, true, false, "v"},
                            {out, tb, true, false, "out"},
                            {dout, tb, true, false, "dout"},
                            {lambda, 4, false, false, "lambda"},
                            {giv ? theta : nullptr, thb, false, false, "theta"},
                            {row_stat, rb, false, false, "row_stat"},
                            {saved, L.prep, false, false, "saved"},
                            {dq, tb, true, true, "dq"},
                            {dk, tb, true, true, "dk"},
                            {dv, tb, true, true, "dv"},
                            {dlambda, 4, false, true, "dlambda"},
                            {giv ? dtheta : nullptr, thb, false, true, "dtheta"},
                            {workspace, need, false, true, "workspace"}}));
  if (test_fail_launch()) return fail(REL_ERR_HIP, "launch failure injected by RELATION_TEST_FAIL_LAUNCH");
  rel::LayerArgs a = layer_args(p, opts, L, prep, q, k, v, theta);
  const int vec = layer_vec(p, opts, {q, k, v, out, dout, dq, dk, dv});
  hipError_t he = hipSuccess;
  const bool y_direct = L.contiguous_tiled && al16({out});
  if (!saved) {
    // recompute what the forward pass prepared
    if (a.rope && (he = rel::launch_rope_table((float2*)a.rope, (int)p->T, (int)p->D, opts->rope_base, s)))
      return hip_fail(he, "RoPE table launch");
    if ((he = rel::launch_layer_prologue(a, p->dtype, vec, s))) return hip_fail(he, "layer prologue launch");
    if (!y_direct && (he = rel::launch_layer_repad(out, prep + L.yp, a, true, p->dtype, vec, s)))
      return hip_fail(he, "layer padding launch");
  }
  const bool do_direct = L.contiguous_tiled && al16({dout});
  if (!do_direct && (he = rel::launch_layer_repad(dout, scr + L.dop, a, true, p->dtype, vec, s)))
    return hip_fail(he, "layer padding launch");
  a.gq = scr + L.gq;
  a.gk = scr + L.gk;
  a.gv = scr + L.gv;
  a.dq = dq; a.dk = dk; a.dv = dv;
  a.dth_rows = giv ? (float*)(scr + L.dth) : nullptr;
  REL_TRY(bwd_impl(&L.pp, a.qr, a.kr, a.vt, y_direct ? out : prep + L.yp, do_direct ? dout : scr + L.dop,
                   lambda, row_stat, (void*)a.gq, (void*)a.gk, (void*)a.gv, dlambda, nullptr, scr + L.bws,
                   relation_bwd_workspace_bytes(&L.pp), stream, opts->transport, true));
  if ((he = rel::launch_layer_epilogue(a, p->dtype, vec, s))) return hip_fail(he, "layer epilogue launch");
  if (giv && (he = rel::launch_segment_sum(a.dth_rows, (int)(p->H / 2), p->B * p->T, (float*)(scr + L.dpart),
                                           dtheta, s)))
    return hip_fail(he, "dtheta reduction launch");
  return REL_OK;
}

// ---------------------------------------------------------------------------
// decode step
// ---------------------------------------------------------------------------
static rel_status check_decode(const rel_problem* p, bool* empty) {
  REL_TRY(check_problem(p, empty));
  if (p && p->B * p->H > 0 && p->T < 1)
    return fail(REL_ERR_INVALID_ARG, "the cache holds at least the new token's own entry (T >= 1)");
  if (p && p->T > (1 << 30)) return fail(REL_ERR_UNSUPPORTED, "cache capacity exceeds 2^30");
  return REL_OK;
}

static rel::DecodeArgs decode_args(const rel_problem* p, const void* q, const void* k, const void* v,
                                   const int32_t* lengths, const float* lambda) {
  rel::DecodeArgs a{};
  a.q = q; a.k = k; a.v = v; a.lengths = lengths; a.lambda = lambda;
  a.sb = p->stride_b; a.sh = p->stride_h; a.st = p->stride_t;
  a.B = (int)p->B; a.H = (int)p->H; a.Tmax = (int)p->T; a.D = (int)p->D;
  a.scale = eff_scale(p);
  a.inv_tau = 1.0f / p->tau_s;
  return a;
}

static int decode_slices(const rel_problem* p) {
  const int64_t hist = std::max<int64_t>(p->T - 1, 1);
  return (int)((hist + rel::decode_slice_keys() - 1) / rel::decode_slice_keys());
}

static rel_status check_decode_io(const rel_problem* p, const void* q, const void* k, const void* v,
                                  const int32_t* lengths, const void* out, const float* row_stat,
                                  const float* states, size_t states_bytes, bool states_out) {
  REL_TRY(check_aligned(q, 16, "q", true));
  REL_TRY(check_aligned(k, 16, "k_cache", true));
  REL_TRY(check_aligned(v, 16, "v_cache", true));
  REL_TRY(check_aligned(lengths, 4, "lengths", true));
  REL_TRY(check_aligned(out, 16, "out", !states_out));
  REL_TRY(check_aligned(row_stat, 4, "row_stat", false));
  REL_TRY(check_aligned(states, 8, "states", states_bytes > 0));
  const size_t es = elem_size(p->dtype);
  const size_t cb = (size_t)extent_elems(p) * es, rowb = (size_t)(p->B * p->H * p->D) * es;
  const size_t nb = (size_t)(p->B * p->H) * 4;
  return check_buffers(p, {{q, rowb, false, false, "q"},
                           {k, cb, true, false, "k_cache"},
                           {v, cb, true, false, "v_cache"},
                           {lengths, (size_t)p->B * 4, false, false, "lengths"},
                           {states, states_bytes, false, states_out, "states"},
                           {states_out ? nullptr : out, rowb, false, true, "out"},
                           {states_out ? nullptr : row_stat, nb, false, true, "row_stat"}});
}

size_t relation_decode_workspace_bytes(const rel_problem* p) {
  bool empty = false;
  if (check_decode(p, &empty) != REL_OK || empty) return 0;
  return align256((size_t)decode_slices(p) * (size_t)(p->B * p->H) * (size_t)(p->D + 2) * 4);
}

rel_status relation_decode_states(const rel_problem* p, const void* q, const void* k_cache,
                                  const void* v_cache, const int32_t* lengths, int32_t key_begin,
                                  int32_t key_end, int32_t nstates, float* states, void* stream) {
  bool empty = false;
  REL_TRY(check_decode(p, &empty));
  if (empty) return REL_OK;
  if (key_begin < 0 || key_end < key_begin || key_end > p->T)
    return fail(REL_ERR_INVALID_ARG, "key range [%d, %d) outside the cache of %lld entries", key_begin,
                key_end, (long long)p->T);
  if (nstates < 1 || nstates > 65535) return fail(REL_ERR_INVALID_ARG, "nstates must be in 1..65535");
  const size_t sb = (size_t)nstates * (size_t)(p->B * p->H) * (size_t)(p->D + 2) * 4;
  REL_TRY(check_decode_io(p, q, k_cache, v_cache, lengths, nullptr, nullptr, states, sb, true));
  if (test_fail_launch()) return fail(REL_ERR_HIP, "launch failure injected by RELATION_TEST_FAIL_LAUNCH");
  rel::DecodeArgs a = decode_args(p, q, k_cache, v_cache, lengths, nullptr);
  a.key0 = key_begin; a.key1 = key_end; a.nsplit = nstates; a.states = states;
  const hipError_t e = rel::launch_decode_states(a, p->dtype, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "decode states launch");
  return REL_OK;
}

rel_status relation_decode_merge(const rel_problem* p, int32_t nstates, const float* states, const void* q,
                                 const void* k_cache, const void* v_cache, const int32_t* lengths,
                                 const float* lambda, void* out, float* row_stat, void* stream) {
  bool empty = false;
  REL_TRY(check_decode(p, &empty));
  if (empty) return REL_OK;
  if (nstates < 0 || nstates > 65535) return fail(REL_ERR_INVALID_ARG, "nstates must be in 0..65535");
  REL_TRY(check_aligned(lambda, 4, "lambda", true));
  const size_t sb = (size_t)nstates * (size_t)(p->B * p->H) * (size_t)(p->D + 2) * 4;
  REL_TRY(check_decode_io(p, q, k_cache, v_cache, lengths, out, row_stat, nstates ? states : nullptr, sb, false));
  if (test_fail_launch()) return fail(REL_ERR_HIP, "launch failure injected by RELATION_TEST_FAIL_LAUNCH");
  rel::DecodeArgs a = decode_args(p, q, k_cache, v_cache, lengths, lambda);
  a.nstates = nstates; a.states = (float*)states; a.out = out; a.row_stat = row_stat;
  const hipError_t e = rel::launch_decode_merge(a, p->dtype, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "decode merge launch");
  return REL_OK;
}

rel_status relation_decode(const rel_problem* p, const void* q, const void* k_cache, const void* v_cache,
                           const int32_t* lengths, const float* lambda, void* out, float* row_stat,
                           void* workspace, size_t workspace_bytes, void* stream) {
  bool empty = false;
  REL_TRY(check_decode(p, &empty));
  if (empty) return REL_OK;
  const size_t need = relation_decode_workspace_bytes(p);
  if (!workspace || workspace_bytes < need)
    return fail(REL_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", need,
                workspace ? workspace_bytes : (size_t)0);
  REL_TRY(check_aligned(workspace, 16, "workspace", true));
  REL_TRY(check_aligned(lambda, 4, "lambda", true));
  REL_TRY(check_decode_io(p, q, k_cache, v_cache, lengths, out, row_stat, (const float*)workspace, need, false));
  if (test_fail_launch()) return fail(REL_ERR_HIP, "launch failure injected by RELATION_TEST_FAIL_LAUNCH");
  rel::DecodeArgs a = decode_args(p, q, k_cache, v_cache, lengths, lambda);
  a.key0 = 0; a.key1 = (int)p->T; a.nsplit = decode_slices(p); a.states = (float*)workspace;
  a.nstates = a.nsplit; a.out = out; a.row_stat = row_stat;
  hipError_t e = rel::launch_decode_states(a, p->dtype, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "decode states launch");
  e = rel::launch_decode_merge(a, p->dtype, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "decode merge launch");
  return REL_OK;
}

// ---------------------------------------------------------------------------
// Linear Relation
// ---------------------------------------------------------------------------
static rel_status check_linear(const rel_problem* p, bool* empty) {
  if (!p) return fail(REL_ERR_INVALID_ARG, "problem is null");
  if (p->D != 32 && p->D != 64 && p->D != 128)
    return fail(REL_ERR_UNSUPPORTED, "Linear Relation head width %lld not in {32, 64, 128}", (long long)p->D);
  return check_problem(p, empty);
}

static int linear_chunks(const rel_problem* p) {
  return (int)((p->T + rel::linear_chunk() - 1) / rel::linear_chunk());
}

static int linear_segments(const rel_problem* p) {
  return (linear_chunks(p) + rel::linear_scan_segment() - 1) / rel::linear_scan_segment();
}

// Forward workspace: per chunk its state contribution, retention product and
// entering state; per segment of chunks the scan summaries. The backward adds
// per chunk the gradient contribution and the gradient of the leaving state,
// and per segment the reverse summaries. The D = 128 backward runs as four
// problems of 64 channels per head (split): its chunk states are those of
// 4 B H heads of width 64, and it adds qt and kt of every row and eight
// planes of partial gradients (fp32, [B H, T, 128] each).
struct LinearPlan {
  size_t dstate, gamma, cprev, segc, segg, total;  // forward
  size_t pstate, gout, segp, total_bwd;            // backward
  size_t qn, kn, part;                             // split backward
  size_t gpart, total_gated;                       // gated backward: the gate's segment sums
};

static bool linear_split(const rel_problem* p) { return p->D == 128; }

static LinearPlan plan_linear(const rel_problem* p, bool split) {
  LinearPlan L{};
  const size_t N = (size_t)(p->B * p->H) * (split ? 4 : 1), nc = (size_t)linear_chunks(p);
  const size_t D = split ? (size_t)p->D / 2 : (size_t)p->D;
  const size_t ns = (size_t)linear_segments(p);
  L.dstate = 0;
  L.gamma = align256(N * nc * D * D * 4);
  L.cprev = L.gamma + align256(N * nc * D * 4);
  L.segc = L.cprev + align256(N * nc * D * D * 4);
  L.segg = L.segc + align256(N * ns * D * D * 4);
  L.total = L.segg + align256(N * ns * D * 4);
  L.pstate = L.total;
  L.gout = L.pstate + align256(N * nc * D * D * 4);
  L.segp = L.gout + align256(N * nc * D * D * 4);
  L.total_bwd = L.segp + align256(N * ns * D * D * 4);
  if (split) {
    const size_t plane = (size_t)(p->B * p->H) * (size_t)p->T * (size_t)p->D * 4;
    L.qn = L.total_bwd;
    L.kn = L.qn + align256(plane);
    L.part = L.kn + align256(plane);
    L.total_bwd = L.part + 8 * align256(plane);
  }
  // the gate's sums: per chunk (D <= 64) or per segment of tokens (D = 128), a chunk being the shorter
  const size_t gseg = std::max((size_t)nc, (size_t)((p->T + rel::linear_gate_segment() - 1) / rel::linear_gate_segment()));
  L.gpart = L.total_bwd;
  L.total_gated = L.gpart + align256((size_t)(p->B * p->H) * gseg * 2 * (size_t)p->D * 4);
  return L;
}

// The chunk loads (and the gradient stores) move 16 bytes per lane when every
// row of p1, p2, v (and dY, dp1, dp2, dv) starts on a 16-byte boundary and g
// (with the gate: r, A_log and dt_bias) is 16-byte aligned.
static int linear_vec16(const rel_problem* p, std::initializer_list<const void*> rows, const float* g) {
  const int64_t epl = 16 / (int64_t)elem_size(p->dtype);
  if (p->stride_b % epl || p->stride_h % epl || p->stride_t % epl || ((uintptr_t)g & 15)) return 0;
  for (const void* x : rows)
    if ((uintptr_t)x & 15) return 0;
  return 1;
}

static void set_linear_workspace(rel::LinearArgs& a, const LinearPlan& L, char* ws, bool backward) {
  a.dstate = (float*)(ws + L.dstate);
  a.gamma = (float*)(ws + L.gamma);
  a.cprev = (float*)(ws + L.cprev);
  a.segc = (float*)(ws + L.segc);
  a.segg = (float*)(ws + L.segg);
  if (backward) {
    a.pstate = (float*)(ws + L.pstate);
    a.gout = (float*)(ws + L.gout);
    a.segp = (float*)(ws + L.segp);
  }
  if (L.part) {
    a.qn = (float*)(ws + L.qn);
    a.kn = (float*)(ws + L.kn);
    a.part = (float*)(ws + L.part);
  }
}

size_t relation_linear_fwd_workspace_bytes(const rel_problem* p) {
  bool empty = false;
  if (check_linear(p, &empty) != REL_OK || empty) return 0;
  return plan_linear(p, false).total;
}

// RoPE of the gated entry points: rope_dim 0 (none), or an even width up to D
// whose channels j < rope_dim / 2 turn with j + rope_dim / 2; at D = 128 (the
// four-block backward, whose row passes hold 4 channels per lane) a multiple of 8.
static rel_status check_rope(const rel_problem* p, int32_t rope_dim, float rope_base) {
  if (rope_dim == 0) return REL_OK;
  if (rope_dim < 0 || rope_dim % 2 || rope_dim > p->D)
    return fail(REL_ERR_INVALID_ARG, "rope_dim %d must be 0 or an even width <= D = %lld", (int)rope_dim,
                (long long)p->D);
  if (p->D == 128 && rope_dim % 8)
    return fail(REL_ERR_UNSUPPORTED, "at D = 128 rope_dim must be a multiple of 8 (got %d)", (int)rope_dim);
  if (!(std::isfinite(rope_base) && rope_base > 0.0f))
    return fail(REL_ERR_INVALID_ARG, "rope_base must be finite and > 0");
  return REL_OK;
}

static size_t rope_table_bytes(const rel_problem* p, int32_t rope_dim) {
  const size_t rows = (size_t)linear_chunks(p) + (size_t)rel::linear_chunk();
  return rope_dim > 0 ? align256(rows * (size_t)(rope_dim / 2) * 8) : 0;
}

size_t relation_linear_gated_fwd_workspace_bytes(const rel_problem* p, int32_t rope_dim) {
  bool empty = false;
  if (check_linear(p, &empty) != REL_OK || empty || check_rope(p, rope_dim, 1.0f) != REL_OK) return 0;
  return plan_linear(p, false).total + rope_table_bytes(p, rope_dim);
}

// The RoPE table (cos, sin at the chunk starts and at the offsets inside a
// chunk) at workspace offset off, and the kernels' view of it.
static rel_status set_rope(rel::LinearArgs& a, const rel_problem* p, int32_t rope_dim, float rope_base, char* ws,
                           size_t off, hipStream_t stream) {
  if (rope_dim == 0) return REL_OK;
  float2* tab = (float2*)(ws + off);
  const hipError_t e = rel::launch_linear_rope_table(tab, (int)p->T, (int)rope_dim, (double)rope_base, stream);
  if (e != hipSuccess) return hip_fail(e, "RoPE table launch");
  a.rope = tab;
  a.rope_half = rope_dim / 2;
  return REL_OK;
}

// g: the log-retention, or with a_log set the gate's pre-activation r.
static rel_status linear_fwd_impl(const rel_problem* p, const void* p1, const void* p2, const void* v, const float* g,
                                  const float* a_log, const float* dt_bias, int32_t rope_dim, float rope_base,
                                  void* out, float* state_out, void* workspace, size_t workspace_bytes,
                                  void* stream) {
  bool empty = false;
  REL_TRY(check_linear(p, &empty));
  REL_TRY(check_rope(p, rope_dim, rope_base));
  if (empty) return REL_OK;
  const size_t es = elem_size(p->dtype);
  REL_TRY(check_aligned(p1, es, "p1", true));
  REL_TRY(check_aligned(p2, es, "p2", true));
  REL_TRY(check_aligned(v, es, "v", true));
  REL_TRY(check_aligned(g, 4, a_log ? "r" : "g", true));
  REL_TRY(check_aligned(a_log, 4, "a_log", false));
  REL_TRY(check_aligned(dt_bias, 4, "dt_bias", false));
  REL_TRY(check_aligned(out, es, "out", true));
  REL_TRY(check_aligned(state_out, 4, "state_out", false));
  const LinearPlan L = plan_linear(p, false);
  const size_t need = L.total + rope_table_bytes(p, rope_dim);
  if (!workspace || workspace_bytes < need)
    return fail(REL_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", need,
                workspace ? workspace_bytes : (size_t)0);
  REL_TRY(check_aligned(workspace, 16, "workspace", true));
  const size_t tb = (size_t)extent_elems(p) * es;
  const size_t N = (size_t)(p->B * p->H);
  const size_t gb = N * (size_t)p->T * (size_t)p->D * 4;
  const size_t pb = a_log ? (size_t)p->H * (size_t)p->D * 4 : 0;
  REL_TRY(check_buffers(p, {{p1, tb, true, false, "p1"},
                            {p2, tb, true, false, "p2"},
                            {v, tb, true, false, "v"},
                            {g, gb, false, false, a_log ? "r" : "g"},
                            {a_log, pb, false, false, "a_log"},
                            {dt_bias, pb, false, false, "dt_bias"},
                            {out, tb, true, true, "out"},
                            {state_out, N * (size_t)(p->D * p->D) * 4, false, true, "state_out"},
                            {workspace, need, false, true, "workspace"}}));
  if (test_fail_launch()) return fail(REL_ERR_HIP, "launch failure injected by RELATION_TEST_FAIL_LAUNCH");
  rel::LinearArgs a{};
  a.p1 = p1; a.p2 = p2; a.v = v; a.g = g; a.out = out; a.state_out = state_out;
  a.a_log = a_log; a.dt_bias = dt_bias;
  a.sb = p->stride_b; a.sh = p->stride_h; a.st = p->stride_t;
  a.B = (int)p->B; a.H = (int)p->H; a.T = (int)p->T; a.D = (int)p->D;
  a.scale = eff_scale(p);
  a.inv_tau = 1.0f / p->tau_s;
  a.nchunks = linear_chunks(p);
  a.nseg = linear_segments(p);
  a.vec16 = linear_vec16(p, {p1, p2, v, a_log, dt_bias}, g);
  set_linear_workspace(a, L, (char*)workspace, false);
  REL_TRY(set_rope(a, p, rope_dim, rope_base, (char*)workspace, L.total, (hipStream_t)stream));
  const hipError_t e = rel::launch_linear_fwd(a, p->dtype, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "Linear Relation launch");
  return REL_OK;
}

rel_status relation_linear_fwd(const rel_problem* p, const void* p1, const void* p2, const void* v,
                               const float* g, void* out, float* state_out, void* workspace,
                               size_t workspace_bytes, void* stream) {
  return linear_fwd_impl(p, p1, p2, v, g, nullptr, nullptr, 0, 0.0f, out, state_out, workspace, workspace_bytes,
                         stream);
}

rel_status relation_linear_gated_fwd(const rel_problem* p, const void* p1, const void* p2, const void* v,
                                     const float* r, const float* a_log, const float* dt_bias, int32_t rope_dim,
                                     float rope_base, void* out, float* state_out, void* workspace,
                                     size_t workspace_bytes, void* stream) {
  if (!a_log || !dt_bias) return fail(REL_ERR_INVALID_ARG, "a_log and dt_bias are required");
  return linear_fwd_impl(p, p1, p2, v, r, a_log, dt_bias, rope_dim, rope_base, out, state_out, workspace,
                         workspace_bytes, stream);
}

static size_t linear_bwd_ws(const rel_problem* p, bool gated, int32_t rope_dim) {
  bool empty = false;
  if (check_linear(p, &empty) != REL_OK || empty || check_rope(p, rope_dim, 1.0f) != REL_OK) return 0;
  const LinearPlan L = plan_linear(p, linear_split(p));
  return (gated ? L.total_gated : L.total_bwd) + rope_table_bytes(p, rope_dim);
}

size_t relation_linear_bwd_workspace_bytes(const rel_problem* p) { return linear_bwd_ws(p, false, 0); }
size_t relation_linear_gated_bwd_workspace_bytes(const rel_problem* p, int32_t rope_dim) {
  return linear_bwd_ws(p, true, rope_dim);
}

// g: the log-retention, or with a_log set the gate's pre-activation r; dg is
// then dr, and da_log, ddt_bias receive the parameters' gradients.
static rel_status linear_bwd_impl(const rel_problem* p, const void* p1, const void* p2, const void* v, const float* g,
                                  const float* a_log, const float* dt_bias, int32_t rope_dim, float rope_base,
                                  const void* dout, void* dp1, void* dp2, void* dv, float* dg, float* da_log,
                                  float* ddt_bias, void* workspace, size_t workspace_bytes, void* stream) {
  bool empty = false;
  const bool gated = a_log != nullptr;
  REL_TRY(check_linear(p, &empty));
  REL_TRY(check_rope(p, rope_dim, rope_base));
  if (empty) return REL_OK;
  const size_t es = elem_size(p->dtype);
  REL_TRY(check_aligned(p1, es, "p1", true));
  REL_TRY(check_aligned(p2, es, "p2", true));
  REL_TRY(check_aligned(v, es, "v", true));
  REL_TRY(check_aligned(g, 4, gated ? "r" : "g", true));
  REL_TRY(check_aligned(dout, es, "dout", true));
  REL_TRY(check_aligned(dp1, es, "dp1", true));
  REL_TRY(check_aligned(dp2, es, "dp2", true));
  REL_TRY(check_aligned(dv, es, "dv", true));
  REL_TRY(check_aligned(dg, 4, gated ? "dr" : "dg", true));
  if (gated) {
    REL_TRY(check_aligned(a_log, 4, "a_log", true));
    REL_TRY(check_aligned(dt_bias, 4, "dt_bias", true));
    REL_TRY(check_aligned(da_log, 4, "da_log", true));
    REL_TRY(check_aligned(ddt_bias, 4, "ddt_bias", true));
  }
  const size_t need = linear_bwd_ws(p, gated, rope_dim);
  if (!workspace || workspace_bytes < need)
    return fail(REL_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", need,
                workspace ? workspace_bytes : (size_t)0);
  REL_TRY(check_aligned(workspace, 16, "workspace", true));
  const size_t tb = (size_t)extent_elems(p) * es;
  const size_t N = (size_t)(p->B * p->H);
  const size_t gb = N * (size_t)p->T * (size_t)p->D * 4;
  const size_t pb = gated ? (size_t)p->H * (size_t)p->D * 4 : 0;
  REL_TRY(check_buffers(p, {{p1, tb, true, false, "p1"},
                            {p2, tb, true, false, "p2"},
                            {v, tb, true, false, "v"},
                            {g, gb, false, false, gated ? "r" : "g"},
                            {a_log, pb, false, false, "a_log"},
                            {dt_bias, pb, false, false, "dt_bias"},
                            {dout, tb, true, false, "dout"},
                            {dp1, tb, true, true, "dp1"},
                            {dp2, tb, true, true, "dp2"},
                            {dv, tb, true, true, "dv"},
                            {dg, gb, false, true, gated ? "dr" : "dg"},
                            {da_log, pb, false, true, "da_log"},
                            {ddt_bias, pb, false, true, "ddt_bias"},
                            {workspace, need, false, true, "workspace"}}));
  if (test_fail_launch()) return fail(REL_ERR_HIP, "launch failure injected by RELATION_TEST_FAIL_LAUNCH");
  const LinearPlan L = plan_linear(p, linear_split(p));
  rel::LinearArgs a{};
  a.p1 = p1; a.p2 = p2; a.v = v; a.g = g; a.dy = dout;
  a.dp1 = dp1; a.dp2 = dp2; a.dv = dv; a.dg = dg;
  a.sb = p->stride_b; a.sh = p->stride_h; a.st = p->stride_t;
  a.B = (int)p->B; a.H = (int)p->H; a.T = (int)p->T; a.D = (int)p->D;
  a.scale = eff_scale(p);
  a.inv_tau = 1.0f / p->tau_s;
  a.nchunks = linear_chunks(p);
  a.nseg = linear_segments(p);
  a.vec16 = linear_vec16(p, {p1, p2, v, dout, dp1, dp2, dv, gated ? a_log : nullptr, gated ? dt_bias : nullptr}, g);
  set_linear_workspace(a, L, (char*)workspace, true);
  if (gated) {
    a.a_log = a_log; a.dt_bias = dt_bias;
    a.gpart = (float*)((char*)workspace + L.gpart);
    a.da_log = da_log; a.ddt_bias = ddt_bias;
  }
  REL_TRY(set_rope(a, p, rope_dim, rope_base, (char*)workspace, gated ? L.total_gated : L.total_bwd,
                   (hipStream_t)stream));
  const hipError_t e = rel::launch_linear_bwd(a, p->dtype, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "Linear Relation backward launch");
  return REL_OK;
}

rel_status relation_linear_bwd(const rel_problem* p, const void* p1, const void* p2, const void* v,
                               const float* g, const void* dout, void* dp1, void* dp2, void* dv, float* dg,
                               void* workspace, size_t workspace_bytes, void* stream) {
  return linear_bwd_impl(p, p1, p2, v, g, nullptr, nullptr, 0, 0.0f, dout, dp1, dp2, dv, dg, nullptr, nullptr,
                         workspace, workspace_bytes, stream);
}

rel_status relation_linear_gated_bwd(const rel_problem* p, const void* p1, const void* p2, const void* v,
                                     const float* r, const float* a_log, const float* dt_bias, int32_t rope_dim,
                                     float rope_base, const void* dout, void* dp1, void* dp2, void* dv, float* dr,
                                     float* da_log, float* ddt_bias, void* workspace, size_t workspace_bytes,
                                     void* stream) {
  if (!a_log || !dt_bias) return fail(REL_ERR_INVALID_ARG, "a_log and dt_bias are required");
  return linear_bwd_impl(p, p1, p2, v, r, a_log, dt_bias, rope_dim, rope_base, dout, dp1, dp2, dv, dr, da_log,
                         ddt_bias, workspace, workspace_bytes, stream);
}

}  // extern "C"
