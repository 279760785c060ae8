// Host side of the C interface declared in include/ec_moe.h: argument
// validation, the capacity rule, the layout of the saved activations and of
// the workspace, and the launch sequence of each entry point on the caller's
// stream.  Nothing here allocates device memory or synchronises.
#include "../../include/ec_moe.h"

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <atomic>

#include "ec_kernels.h"


namespace {

// fixed per-thread buffer: recording an error allocates nothing and cannot throw
thread_local char g_last_error[512];
thread_local hipEvent_t* g_events = nullptr;  // stage timing (ec_set_stage_events)
thread_local int g_n_events = 0;

int fail(int status, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
  va_end(ap);
  return status;
}

constexpr size_t kAlign = 256;
size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

struct Plan {
  int N = 0, d = 0, E = 0, h = 0, G = 0, EP = 0;
  int hs = 0;          // hidden width of the shared experts (0: none)
  long K = 0;          // K_tot
  int dtype = 0;
  size_t esz = 0;      // storage bytes per element
};

// ec_buffers: check the sizes of the [E, K_tot, .] expert buffers of expert
// choice (token choice packs its pairs and checks its own bound).
int validate(const ec_problem* p, Plan* out, bool ec_buffers = true) {
  g_last_error[0] = '\0';
  if (!p) return fail(EC_ERR_ARG, "problem is NULL");
  if (p->dtype != EC_F32 && p->dtype != EC_BF16)
    return fail(EC_ERR_DTYPE, "unknown dtype %d", (int)p->dtype);
  if (p->n_groups < 1) return fail(EC_ERR_SHAPE, "n_groups must be >= 1 (got %d)", p->n_groups);
  if (!p->group_offsets || !p->capacity)
    return fail(EC_ERR_ARG, "group_offsets and capacity must be host arrays");
  if (p->n_experts < 1 || p->n_experts > 256)
    return fail(EC_ERR_SHAPE, "n_experts must be in [1, 256] (got %d)", p->n_experts);
  if (p->d_model < 64 || p->d_model > 16384 || p->d_model % 64)
    return fail(EC_ERR_SHAPE, "d_model must be a multiple of 64 in [64, 16384] (got %d)",
                p->d_model);
  if (p->d_ff < 64 || p->d_ff > 16384 || p->d_ff % 64)
    return fail(EC_ERR_SHAPE, "d_ff must be a multiple of 64 in [64, 16384] (got %d)", p->d_ff);
  if (p->d_shared != 0 && (p->d_shared < 64 || p->d_shared > 16384 || p->d_shared % 64))
    return fail(EC_ERR_SHAPE, "d_shared must be 0 or a multiple of 64 in [64, 16384] (got %d)",
                p->d_shared);
  if (!std::isfinite(p->inv_temperature) || !(p->inv_temperature > 0.f))
    return fail(EC_ERR_ARG, "inv_temperature must be finite and > 0");
  if (p->n_tokens < 0 || p->n_tokens >= (int64_t)1 << 31)
    return fail(EC_ERR_SHAPE, "n_tokens out of range");
  const int32_t* off = p->group_offsets;
  if (off[0] != 0) return fail(EC_ERR_SHAPE, "group_offsets[0] must be 0");
  long K = 0;
  for (int g = 0; g < p->n_groups; ++g) {
    if (off[g + 1] < off[g]) return fail(EC_ERR_SHAPE, "group_offsets must be non-decreasing");
    const int L = off[g + 1] - off[g];
    const int k = p->capacity[g];
    if (k < 0 || k > L)
      return fail(EC_ERR_CAPACITY, "capacity[%d] = %d outside [0, %d]", g, k, L);
    K += k;
  }
  if ((int64_t)off[p->n_groups] != p->n_tokens)
    return fail(EC_ERR_SHAPE, "group_offsets[G] = %d != n_tokens = %lld", off[p->n_groups],
                (long long)p->n_tokens);
  const int64_t maxw = p->d_model > p->d_ff ? p->d_model : p->d_ff;
  if ((ec_buffers && (int64_t)p->n_experts * K * 2 * maxw >= ((int64_t)1 << 31)) ||
      (int64_t)p->n_experts * p->n_tokens >= ((int64_t)1 << 31) ||
      p->n_tokens * 2 * (int64_t)(p->d_shared > p->d_model ? p->d_shared : p->d_model) >=
          ((int64_t)1 << 31))
    return fail(EC_ERR_SHAPE, "problem too large for 32-bit element indices");
  Plan& P = *out;
  P.N = (int)p->n_tokens;
  P.d = p->d_model;
  P.E = p->n_experts;
  P.h = p->d_ff;
  P.hs = p->d_shared;
  P.G = p->n_groups;
  P.K = K;
  P.EP = (P.E + 63) / 64 * 64;
  P.dtype = p->dtype;
  P.esz = p->dtype == EC_F32 ? 4 : 2;
  return EC_OK;
}

// Sub-allocator over a caller buffer; with base == nullptr it only measures.
struct Carve {
  char* base;
  size_t used = 0;
  explicit Carve(void* b) : base((char*)b) {}
  void* take(size_t bytes) {
    void* r = base ? base + used : nullptr;
    used += align_up(bytes);
    return r;
  }
};

struct Saved {
  float* S;
  int32_t* sel;
  float* gate;    // [E, K] S at the selection: the row factors of the expert products
  int32_t* slot;
  void* Xe;
  void* H1;
  void* H3;
  void* A;
  void* O;
  void* Hs1;      // shared experts, [N, hs] each (null when there are none)
  void* Hs3;
  void* As;
};

Saved carve_saved(Carve& c, const Plan& P, bool with_h) {
  Saved s;
  s.S = (float*)c.take((size_t)P.N * P.E * 4);
  s.sel = (int32_t*)c.take((size_t)P.E * P.K * 4);
  s.gate = (float*)c.take((size_t)P.E * P.K * 4);
  s.slot = (int32_t*)c.take((size_t)P.E * P.N * 4);
  // bf16 reads the selected rows of X inside the products that use them (the
  // forward's W1/W3, the backward's dW1/dW3) and needs no gathered copy
  s.Xe = (P.dtype != EC_BF16) ? c.take((size_t)P.E * P.K * P.d * P.esz) : nullptr;
  s.H1 = with_h ? c.take((size_t)P.E * P.K * P.h * P.esz) : nullptr;
  s.H3 = with_h ? c.take((size_t)P.E * P.K * P.h * P.esz) : nullptr;
  s.A = c.take((size_t)P.E * P.K * P.h * P.esz);
  s.O = c.take((size_t)P.E * P.K * P.d * P.esz);
  const size_t sh = (size_t)P.N * P.hs * P.esz;
  s.Hs1 = (with_h && sh) ? c.take(sh) : nullptr;
  s.Hs3 = (with_h && sh) ? c.take(sh) : nullptr;
  s.As = sh ? c.take(sh) : nullptr;
  return s;
}

struct BwdWs {
  void* dYe;      // [E, K, d] fp32: selected rows of dY; then dXe (both dtypes)
  float* dsp;     // [E, K, dsp_parts(h)] gate-gradient partials of the dA product
  void* dH;       // [E, K, 2h]
  float* dZ;      // [N, E]
  uint16_t* dZb;  // [N, EP] (bf16 only)
  float* part;    // [splits, E, d]
  int splits;
  void* dHs;      // [N, 2 hs] shared experts' dH1 | dH3
  float* spart;   // split-K partials of the shared weight gradients
  int s_splits2, s_splits13;
};

BwdWs carve_bwd(Carve& c, const Plan& P) {
  BwdWs w;
  w.dYe = c.take((size_t)P.E * P.K * P.d * P.esz);
  w.dsp = (float*)c.take((size_t)P.E * P.K * ec::dsp_parts(P.dtype, P.h) * 4);
  w.dH = c.take((size_t)P.E * P.K * 2 * P.h * P.esz);
  w.dZ = (float*)c.take((size_t)P.N * P.E * 4);
  w.dZb = P.dtype == EC_BF16 ? (uint16_t*)c.take((size_t)P.N * P.EP * 2) : nullptr;
  w.splits = ec::router_dwg_splits(P.N, P.E, P.d);
  w.part = (float*)c.take((size_t)w.splits * P.E * P.d * 4);
  w.dHs = nullptr;
  w.spart = nullptr;
  w.s_splits2 = w.s_splits13 = 0;
  if (P.hs) {
    w.dHs = c.take((size_t)P.N * 2 * P.hs * P.esz);
    w.s_splits2 = ec::wgrad_splits(P.d, P.hs, P.N);
    w.s_splits13 = ec::wgrad_splits(2 * P.hs, P.d, P.N);
    const size_t a = (size_t)w.s_splits2 * P.d * P.hs, b = (size_t)w.s_splits13 * 2 * P.hs * P.d;
    if (P.dtype == EC_BF16) w.spart = (float*)c.take((a > b ? a : b) * 4);
  }
  return w;
}

size_t route_ws(const Plan& P, bool need_slot) {
  Carve c(nullptr);
  c.take((size_t)P.E * P.N * 4);                   // ST
  if (need_slot) c.take((size_t)P.E * P.N * 4);    // slot when the caller passes none
  return c.used;
}

// have_saved: the caller passes a saved buffer, which then holds the
// activations; otherwise the workspace holds them (without H1, H3).
size_t forward_ws(const Plan& P, bool have_saved) {
  Carve c(nullptr);
  c.take((size_t)P.E * P.N * 4);  // ST
  if (!have_saved) carve_saved(c, P, false);
  return c.used;
}

size_t backward_ws(const Plan& P) {
  Carve c(nullptr);
  carve_bwd(c, P);
  return c.used;
}

size_t saved_bytes(const Plan& P) {
  Carve c(nullptr);
  carve_saved(c, P, true);
  return c.used;
}

int check_ptr(const void* ptr, const char* name, bool optional = false) {
  if (!ptr) {
    if (optional) return EC_OK;
    return fail(EC_ERR_ARG, "%s is NULL", name);
  }
  if ((uintptr_t)ptr % 16) return fail(EC_ERR_ALIGN, "%s is not 16-byte aligned", name);
  return EC_OK;
}

#define EC_TRY(expr)                           \
  do {                                         \
    int _s = (expr);                           \
    if (_s != EC_OK) return _s;                \
  } while (0)

#define EC_HIP(expr)                                                                   \
  do {                                                                                 \
    hipError_t _e = (expr);                                                            \
    if (_e != hipSuccess)                                                              \
      return fail(EC_ERR_HIP, "%s failed: %s", #expr, hipGetErrorString(_e));          \
  } while (0)

// Records stage event `i` (0 = before the first stage) if timing is enabled.
hipError_t mark(int i, hipStream_t st) {
  if (g_events && i < g_n_events) return hipEventRecord(g_events[i], st);
  return hipSuccess;
}

int enqueue_route(const ec_problem* p, const Plan& P, const void* X, const void* Wg, float* S,
                  float* ST, int32_t* sel, float* gate, int32_t* slot, hipStream_t st) {
  EC_HIP(mark(0, st));
  EC_HIP(ec::launch_router_softmax(P.dtype, X, Wg, S, ST, P.N, P.d, P.E, p->inv_temperature, st));
  EC_HIP(mark(1, st));
  ec::GroupTable tab;
  int seg = 0;
  for (int g0 = 0; g0 < P.G; g0 += ec::TOPK_MAX_GROUPS) {
    tab.n = 0;
    for (int g = g0; g < P.G && g < g0 + ec::TOPK_MAX_GROUPS; ++g) {
      tab.off[tab.n] = p->group_offsets[g];
      tab.len[tab.n] = p->group_offsets[g + 1] - p->group_offsets[g];
      tab.k[tab.n] = p->capacity[g];
      tab.seg[tab.n] = seg;
      seg += p->capacity[g];
      ++tab.n;
    }
    EC_HIP(ec::launch_topk(ST, P.N, P.E, (int)P.K, tab, sel, gate, slot, st));
  }
  EC_HIP(mark(2, st));
  return EC_OK;
}

// ---- token choice -------------------------------------------------------------

int tc_validate(const ec_problem* p, int top_k, Plan* P, long* rmax, int* rmax_e) {
  EC_TRY(validate(p, P, false));
  if (top_k < 1 || top_k > P->E)
    return fail(EC_ERR_ARG, "top_k must be in [1, n_experts] (got %d)", top_k);
  // kept pairs: at most top_k per token and sum_g cap_g per expert
  long r = (long)top_k * P->N;
  const long per_e = P->K < P->N ? P->K : P->N;
  if ((long)P->E * per_e < r) r = (long)P->E * per_e;
  const long w = P->d > P->h ? P->d : P->h;
  if (r * w >= ((long)1 << 31))
    return fail(EC_ERR_SHAPE, "too many token-expert pairs for 32-bit element indices");
  *rmax = r;
  *rmax_e = (int)per_e;
  return EC_OK;
}

struct TcRouteWs {
  float* ST;
  int32_t* cnt;
  int32_t* seg;
  int32_t* tiles13;
  int32_t* tiles2;
};

TcRouteWs carve_tc_route(Carve& c, const Plan& P) {
  TcRouteWs w;
  w.ST = (float*)c.take((size_t)P.E * P.N * 4);
  w.cnt = (int32_t*)c.take((size_t)P.G * P.E * 4);
  w.seg = (int32_t*)c.take((size_t)P.G * P.E * 4);
  w.tiles13 = (int32_t*)c.take((size_t)(P.E + 1) * 4);
  w.tiles2 = (int32_t*)c.take((size_t)(P.E + 1) * 4);
  return w;
}

struct TcFwdWs {
  float* S;
  float* G;
  int32_t* slot;
  int32_t* rows;
  int32_t* sel;
  void* Xe;
  void* A;
  void* O;
  void* As;
};

TcFwdWs carve_tc_fwd(Carve& c, const Plan& P, long rmax) {
  TcFwdWs w;
  w.S = (float*)c.take((size_t)P.N * P.E * 4);
  w.G = (float*)c.take((size_t)P.N * P.E * 4);
  w.slot = (int32_t*)c.take((size_t)P.E * P.N * 4);
  w.rows = (int32_t*)c.take((size_t)(P.E + 1) * 4);
  w.sel = (int32_t*)c.take((size_t)rmax * 4);
  w.Xe = P.dtype == EC_BF16 ? nullptr : c.take((size_t)rmax * P.d * P.esz);   // fp32 only
  w.A = c.take((size_t)rmax * P.h * P.esz);
  w.O = c.take((size_t)rmax * P.d * P.esz);
  w.As = P.hs ? c.take((size_t)P.N * P.hs * P.esz) : nullptr;
  return w;
}

// Router, row top-k, per-(group, expert) counts, offsets and placement.
int enqueue_tc_route(const ec_problem* p, const Plan& P, int top_k, const void* X, const void* Wg,
                     float* S, float* G, int32_t* slot, int32_t* rows, int32_t* sel,
                     const TcRouteWs& w, hipStream_t st) {
  EC_HIP(mark(0, st));
  EC_HIP(ec::launch_router_softmax(P.dtype, X, Wg, S, w.ST, P.N, P.d, P.E, p->inv_temperature,
                                   st));
  EC_HIP(mark(1, st));
  EC_HIP(ec::launch_tc_topk(S, P.N, P.E, top_k, G, slot, st));
  ec::GroupTable tab;
  for (int pass = 0; pass < 2; ++pass) {
    for (int g0 = 0; g0 < P.G; g0 += ec::TOPK_MAX_GROUPS) {
      tab.n = 0;
      for (int g = g0; g < P.G && g < g0 + ec::TOPK_MAX_GROUPS; ++g) {
        tab.off[tab.n] = p->group_offsets[g];
        tab.len[tab.n] = p->group_offsets[g + 1] - p->group_offsets[g];
        tab.k[tab.n] = p->capacity[g];
        tab.seg[tab.n] = 0;
        ++tab.n;
      }
      if (pass == 0) EC_HIP(ec::launch_tc_count(slot, P.N, P.E, tab, g0, w.cnt, st));
      else EC_HIP(ec::launch_tc_place(slot, G, P.N, P.E, tab, g0, w.seg, sel, st));
    }
    if (pass == 0)
      EC_HIP(ec::launch_tc_offsets(w.cnt, P.G, P.E, ec::TC_BM, ec::tc_col_blocks_w13(P.h),
                                   ec::tc_col_blocks_w2(P.d), rows, w.seg, w.tiles13, w.tiles2,
                                   st));
  }
  EC_HIP(mark(2, st));
  return EC_OK;
}

// ---- routing without allocation ---------------------------------------------
// ec_route_noalloc's workspace: a library-owned device array, one copy per GPU,
// kept until the process ends.  In host code `scratch` names a host-side stand-in;
// the device address comes from hipGetSymbolAddress, taken once per device on the
// entry point's first call there (with that device current) and kept per device.
constexpr size_t kScratchBytes = EC_ROUTE_NOALLOC_MAX_BYTES;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
// hipGetSymbolAddress gives the same address every time on a device, so two
// threads that both fill an empty entry store the same value: no lock needed.
std::atomic<void*> g_scratch_ptr[kMaxDevices] = {};

// Device address of the current device's scratch array.
int scratch_of_current_device(void** out) {
  int dev = -1;
  EC_HIP(hipGetDevice(&dev));
  if (dev < 0 || dev >= kMaxDevices)
    return fail(EC_ERR_HIP, "device index %d outside [0, %d)", dev, kMaxDevices);
  void* ptr = g_scratch_ptr[dev].load(std::memory_order_acquire);
  if (!ptr) {
    EC_HIP(hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)));
    if (!ptr) return fail(EC_ERR_HIP, "hipGetSymbolAddress returned a null address");
    g_scratch_ptr[dev].store(ptr, std::memory_order_release);
  }
  *out = ptr;
  return EC_OK;
}

}  // namespace

extern "C" {

const char* ec_status_string(int status) {
  switch (status) {
    case EC_OK: return "EC_OK";
    case EC_ERR_ARG: return "EC_ERR_ARG: invalid argument";
    case EC_ERR_SHAPE: return "EC_ERR_SHAPE: invalid or inconsistent sizes";
    case EC_ERR_CAPACITY: return "EC_ERR_CAPACITY: capacity outside [0, group length]";
    case EC_ERR_DTYPE: return "EC_ERR_DTYPE: unknown storage dtype";
    case EC_ERR_ALIGN: return "EC_ERR_ALIGN: device pointer not 16-byte aligned";
    case EC_ERR_WORKSPACE: return "EC_ERR_WORKSPACE: buffer too small";
    case EC_ERR_HIP: return "EC_ERR_HIP: HIP runtime error";
    default: return "unknown ec_status";
  }
}

const char* ec_last_error(void) { return g_last_error; }

int ec_set_stage_events(hipEvent_t* events, int n_events) {
  g_last_error[0] = '\0';
  if (n_events < 0 || (n_events > 0 && !events)) return fail(EC_ERR_ARG, "bad event array");
  g_events = n_events > 0 ? events : nullptr;
  g_n_events = n_events;
  return EC_OK;
}

int64_t ec_total_capacity(const ec_problem* p) {
  Plan P;
  if (validate(p, &P) != EC_OK) return -1;
  return P.K;
}

size_t ec_workspace_size(const ec_problem* p, int mode) {
  Plan P;
  if (validate(p, &P) != EC_OK) return 0;
  switch (mode) {
    case 0: return route_ws(P, true);
    case 1: return forward_ws(P, false);
    case 2: return backward_ws(P);
    case 3: return forward_ws(P, true);
    default: fail(EC_ERR_ARG, "unknown workspace mode %d", mode); return 0;
  }
}

size_t ec_saved_size(const ec_problem* p) {
  Plan P;
  if (validate(p, &P) != EC_OK) return 0;
  return saved_bytes(P);
}

int ec_saved_layout_of(const ec_problem* p, ec_saved_layout* out) {
  Plan P;
  EC_TRY(validate(p, &P));
  if (!out) return fail(EC_ERR_ARG, "out is NULL");
  // carve an imaginary buffer at a nominal address and read the offsets back
  char* const base = (char*)(uintptr_t)4096;
  Carve m(base);
  const Saved s = carve_saved(m, P, true);
  auto off = [&](const void* q) -> size_t { return q ? (size_t)((const char*)q - base) : m.used; };
  out->S = off(s.S);
  out->sel_token = off(s.sel);
  out->sel_gate = off(s.gate);
  out->slot = off(s.slot);
  out->Xe = off(s.Xe);
  out->H1 = off(s.H1);
  out->H3 = off(s.H3);
  out->A = off(s.A);
  out->O = off(s.O);
  out->Hs1 = off(s.Hs1);
  out->Hs3 = off(s.Hs3);
  out->As = off(s.As);
  out->total = m.used;
  return EC_OK;
}

int ec_capacity(int32_t n_groups, const int32_t* group_lengths, int32_t n_experts, double c_fixed,
                const double* t, double c_min, double c_max, int scheduler, int32_t* k_out) {
  g_last_error[0] = '\0';
  if (n_groups < 0 || !group_lengths || !k_out) return fail(EC_ERR_ARG, "bad arguments");
  if (n_experts < 1) return fail(EC_ERR_SHAPE, "n_experts must be >= 1");
  if (t && (scheduler < EC_SCHED_LINEAR || scheduler > EC_SCHED_GAUSSIAN_REV))
    return fail(EC_ERR_ARG, "unknown scheduler %d", scheduler);
  if (t && !(c_min <= c_max)) return fail(EC_ERR_ARG, "c_min must be <= c_max");
  const double pi = 3.14159265358979323846;
  const double sigma = 0.22;
  const double g0 = std::exp(-1.0 / (8.0 * sigma * sigma));
  for (int g = 0; g < n_groups; ++g) {
    const int L = group_lengths[g];
    if (L < 0) return fail(EC_ERR_SHAPE, "group length %d < 0", L);
    double c = c_fixed;
    if (t) {
      const double r = t[g];
      double s;
      switch (scheduler) {
        case EC_SCHED_LINEAR: s = r; break;
        case EC_SCHED_LINEAR_REV: s = 1.0 - r; break;
        case EC_SCHED_COSINE: s = 0.5 * (1.0 - std::cos(pi * r)); break;
        case EC_SCHED_COSINE_REV: s = 0.5 * (1.0 + std::cos(pi * r)); break;
        default: {
          const double gg = std::exp(-(r - 0.5) * (r - 0.5) / (2.0 * sigma * sigma));
          const double gt = (gg - g0) / (1.0 - g0);
          s = scheduler == EC_SCHED_GAUSSIAN ? gt : 1.0 - gt;
        }
      }
      c = c_min + (c_max - c_min) * s;
      c = c < c_min ? c_min : (c > c_max ? c_max : c);
    }
    if (!std::isfinite(c) || c < 0) return fail(EC_ERR_ARG, "capacity factor must be >= 0");
    double k = std::nearbyint((double)L * c / (double)n_experts);  // ties to even
    if (k < 0) k = 0;
    if (k > L) k = L;
    k_out[g] = (int32_t)k;
  }
  return EC_OK;
}

int ec_route(const ec_problem* p, const void* X, const void* Wg, float* S, int32_t* sel_token,
             float* sel_gate, int32_t* slot, void* ws, size_t ws_bytes, hipStream_t stream) {
  Plan P;
  EC_TRY(validate(p, &P));
  EC_TRY(check_ptr(X, "X"));
  EC_TRY(check_ptr(Wg, "Wg"));
  EC_TRY(check_ptr(S, "S"));
  EC_TRY(check_ptr(sel_token, "sel_token", P.K == 0));
  EC_TRY(check_ptr(sel_gate, "sel_gate", true));
  EC_TRY(check_ptr(slot, "slot", true));
  const size_t need = route_ws(P, slot == nullptr);
  EC_TRY(check_ptr(ws, "workspace", need == 0));
  if (ws_bytes < need)
    return fail(EC_ERR_WORKSPACE, "workspace %zu bytes < %zu required", ws_bytes, need);
  if (P.N == 0) return EC_OK;
  Carve c(ws);
  float* ST = (float*)c.take((size_t)P.E * P.N * 4);
  int32_t* sl = slot ? slot : (int32_t*)c.take((size_t)P.E * P.N * 4);
  return enqueue_route(p, P, X, Wg, S, ST, sel_token, sel_gate, sl, stream);
}

int ec_route_noalloc(const ec_problem* p, const void* X, const void* Wg, float* S,
                     int32_t* sel_token, float* sel_gate, int32_t* slot, hipStream_t stream) {
  Plan P;
  EC_TRY(validate(p, &P));
  EC_TRY(check_ptr(X, "X"));
  EC_TRY(check_ptr(Wg, "Wg"));
  EC_TRY(check_ptr(S, "S"));
  EC_TRY(check_ptr(sel_token, "sel_token", P.K == 0));
  EC_TRY(check_ptr(sel_gate, "sel_gate", true));
  EC_TRY(check_ptr(slot, "slot", true));
  const size_t need = route_ws(P, slot == nullptr);
  if (need > kScratchBytes)
    return fail(EC_ERR_WORKSPACE,
                "ec_route_noalloc: the problem needs %zu bytes of scratch (E N 4 for the "
                "transposed scores, twice that without a slot buffer); its static array "
                "holds %zu",
                need, kScratchBytes);
  if (P.N == 0) return EC_OK;
  void* ws = nullptr;
  EC_TRY(scratch_of_current_device(&ws));
  // nothing in the scratch must start at zero: the router writes every score of
  // ST and the top-k writes every entry of the slot map (the groups cover all N)
  Carve c(ws);
  float* ST = (float*)c.take((size_t)P.E * P.N * 4);
  int32_t* sl = slot ? slot : (int32_t*)c.take((size_t)P.E * P.N * 4);
  return enqueue_route(p, P, X, Wg, S, ST, sel_token, sel_gate, sl, stream);
}

int ec_token_coverage(const ec_problem* p, const int32_t* slot, int32_t* experts_per_token,
                      int32_t* dropped, hipStream_t stream) {
  Plan P;
  EC_TRY(validate(p, &P));
  EC_TRY(check_ptr(slot, "slot", P.N == 0));
  EC_TRY(check_ptr(experts_per_token, "experts_per_token", P.N == 0));
  EC_TRY(check_ptr(dropped, "dropped"));
  EC_HIP(ec::launch_coverage_count(slot, (int)P.N, P.E, experts_per_token, stream));
  ec::GroupTable tab;
  for (int g0 = 0; g0 < P.G; g0 += ec::TOPK_MAX_GROUPS) {
    tab.n = 0;
    for (int g = g0; g < P.G && g < g0 + ec::TOPK_MAX_GROUPS; ++g) {
      tab.off[tab.n] = p->group_offsets[g];
      tab.len[tab.n] = p->group_offsets[g + 1] - p->group_offsets[g];
      tab.k[tab.n] = p->capacity[g];
      tab.seg[tab.n] = 0;
      ++tab.n;
    }
    EC_HIP(ec::launch_coverage_drop(experts_per_token, tab, dropped + g0, stream));
  }
  return EC_OK;
}

int ec_moe_forward(const ec_problem* p, const void* X, const void* Wg, const void* W1,
                   const void* W3, const void* W2, const void* Ws1, const void* Ws3,
                   const void* Ws2, void* Y, void* saved, size_t saved_bytes_in, void* ws,
                   size_t ws_bytes, hipStream_t stream) {
  Plan P;
  EC_TRY(validate(p, &P));
  EC_TRY(check_ptr(X, "X"));
  EC_TRY(check_ptr(Wg, "Wg"));
  EC_TRY(check_ptr(W1, "W1"));
  EC_TRY(check_ptr(W3, "W3"));
  EC_TRY(check_ptr(W2, "W2"));
  EC_TRY(check_ptr(Ws1, "Ws1", P.hs == 0));
  EC_TRY(check_ptr(Ws3, "Ws3", P.hs == 0));
  EC_TRY(check_ptr(Ws2, "Ws2", P.hs == 0));
  EC_TRY(check_ptr(Y, "Y"));
  EC_TRY(check_ptr(saved, "saved", true));
  if (saved && saved_bytes_in < saved_bytes(P))
    return fail(EC_ERR_WORKSPACE, "saved buffer %zu bytes < %zu required", saved_bytes_in,
                saved_bytes(P));
  const size_t need = forward_ws(P, saved != nullptr);
  EC_TRY(check_ptr(ws, "workspace"));
  if (ws_bytes < need)
    return fail(EC_ERR_WORKSPACE, "workspace %zu bytes < %zu required", ws_bytes, need);
  if (P.N == 0) return EC_OK;

  Carve c(ws);
  float* ST = (float*)c.take((size_t)P.E * P.N * 4);
  Saved s;
  if (saved) {
    Carve cs(saved);
    s = carve_saved(cs, P, true);
  } else {
    s = carve_saved(c, P, false);
  }
  EC_TRY(enqueue_route(p, P, X, Wg, s.S, ST, s.sel, s.gate, s.slot, stream));
  const int M = (int)P.K;
  // The gate multiplies each expert row inside the W1/W3 product's epilogue
  // (A = g SiLU(H1) H3, so O = A W2^T is already gate-weighted and the combine
  // adds rows with weight 1).
  if (P.dtype == EC_BF16) {
    // the W1/W3 product reads the selected rows of X itself (the gather stage is
    // empty)
    EC_HIP(mark(3, stream));
    EC_HIP(ec::launch_gemm_w13(P.dtype, X, W1, W3, s.A, s.H1, s.H3, P.E, M, P.d, P.h, stream,
                               false, s.sel, s.gate));
  } else {
    EC_HIP(ec::launch_gather(P.dtype, X, s.sel, s.Xe, (long)P.E * M, P.d, P.N, stream));
    EC_HIP(mark(3, stream));
    EC_HIP(ec::launch_gemm_w13(P.dtype, s.Xe, W1, W3, s.A, s.H1, s.H3, P.E, M, P.d, P.h, stream,
                               false, nullptr, s.gate));
  }
  EC_HIP(mark(4, stream));
  EC_HIP(ec::launch_gemm_w2(P.dtype, s.A, W2, s.O, P.E, M, P.d, P.h, stream, false));
  EC_HIP(mark(5, stream));
  if (P.hs) {
    // shared experts on every token; their output goes to Y and the combine adds
    // the routed sum to it
    EC_HIP(ec::launch_gemm_w13(P.dtype, X, Ws1, Ws3, s.As, s.Hs1, s.Hs3, 1, P.N, P.d, P.hs,
                               stream, true));
    EC_HIP(mark(6, stream));
    EC_HIP(ec::launch_gemm_w2(P.dtype, s.As, Ws2, Y, 1, P.N, P.d, P.hs, stream, true));
  } else {
    EC_HIP(mark(6, stream));
  }
  EC_HIP(mark(7, stream));
  EC_HIP(ec::launch_combine(P.dtype, s.O, nullptr, s.slot, P.hs ? Y : nullptr, Y, P.N, P.E, M,
                            P.d, stream));
  EC_HIP(mark(8, stream));
  return EC_OK;
}

int ec_moe_backward(const ec_problem* p, const void* X, const void* Wg, const void* W1,
                    const void* W3, const void* W2, const void* Ws1, const void* Ws3,
                    const void* Ws2, const void* dY, const void* saved, size_t saved_bytes_in,
                    void* dX, float* dWg, void* dW1, void* dW3, void* dW2, void* dWs1,
                    void* dWs3, void* dWs2, void* ws, size_t ws_bytes, hipStream_t stream) {
  Plan P;
  EC_TRY(validate(p, &P));
  EC_TRY(check_ptr(X, "X"));
  EC_TRY(check_ptr(Wg, "Wg"));
  EC_TRY(check_ptr(W1, "W1"));
  EC_TRY(check_ptr(W3, "W3"));
  EC_TRY(check_ptr(W2, "W2"));
  EC_TRY(check_ptr(Ws1, "Ws1", P.hs == 0));
  EC_TRY(check_ptr(Ws3, "Ws3", P.hs == 0));
  EC_TRY(check_ptr(Ws2, "Ws2", P.hs == 0));
  EC_TRY(check_ptr(dY, "dY"));
  EC_TRY(check_ptr(saved, "saved"));
  EC_TRY(check_ptr(dX, "dX"));
  EC_TRY(check_ptr(dWg, "dWg"));
  EC_TRY(check_ptr(dW1, "dW1"));
  EC_TRY(check_ptr(dW3, "dW3"));
  EC_TRY(check_ptr(dW2, "dW2"));
  EC_TRY(check_ptr(dWs1, "dWs1", P.hs == 0));
  EC_TRY(check_ptr(dWs3, "dWs3", P.hs == 0));
  EC_TRY(check_ptr(dWs2, "dWs2", P.hs == 0));
  if (saved_bytes_in < saved_bytes(P))
    return fail(EC_ERR_WORKSPACE, "saved buffer %zu bytes < %zu required", saved_bytes_in,
                saved_bytes(P));
  const size_t need = backward_ws(P);
  EC_TRY(check_ptr(ws, "workspace"));
  if (ws_bytes < need)
    return fail(EC_ERR_WORKSPACE, "workspace %zu bytes < %zu required", ws_bytes, need);

  Carve cs((void*)saved);
  const Saved s = carve_saved(cs, P, true);
  Carve c(ws);
  const BwdWs w = carve_bwd(c, P);
  const int M = (int)P.K;
  const int E = P.E, d = P.d, h = P.h, N = P.N, hs = P.hs;
  void* dYe = w.dYe;  // [E, K, d] the selected rows of dY (not gate-scaled), fp32 only
  void* dXe = w.dYe;  // dYe is dead once dW2 is formed
  // The saved A carries the gate (A = g SiLU(H1) H3), so dW2 = dYe^T A; the
  // dA product scales its rows by g (dA = g dYe W2) and its epilogue also sums
  // dA * SiLU(H1) H3 per row: the gate's gradient times the gate.
  // bf16: dA and dXe = dH1 W1 + dH3 W3 read the weights K-major; dA and dW2
  // read the selected rows of dY, dW1/dW3 those of X, inside their operand
  // loads (the gather stage is empty and no gathered copy exists).
  EC_HIP(mark(0, stream));
  const bool bf = P.dtype == EC_BF16;
  if (!bf) EC_HIP(ec::launch_gather(P.dtype, dY, s.sel, dYe, (long)E * M, d, N, stream));
  EC_HIP(mark(1, stream));
  EC_HIP(ec::launch_gemm_dA(P.dtype, bf ? dY : dYe, W2, s.H1, s.H3, w.dH, E, M, d, h, stream,
                            false, w.dsp, bf ? s.sel : nullptr, s.gate));
  EC_HIP(mark(2, stream));
  EC_HIP(ec::launch_gemm_dW2(P.dtype, bf ? dY : dYe, s.A, dW2, E, M, d, h, stream,
                             bf ? s.sel : nullptr));
  EC_HIP(mark(3, stream));
  EC_HIP(ec::launch_gemm_dXe(P.dtype, w.dH, W1, W3, dXe, E, M, d, h, stream, false));
  EC_HIP(mark(4, stream));
  EC_HIP(ec::launch_gemm_dW13(P.dtype, w.dH, bf ? X : s.Xe, dW1, dW3, E, M, d, h, stream,
                              bf ? s.sel : nullptr));
  EC_HIP(mark(5, stream));
  EC_HIP(ec::launch_router_dz(s.S, w.dsp, ec::dsp_parts(P.dtype, h), s.slot, w.dZ, w.dZb, N, E, P.EP, M,
                              p->inv_temperature, stream));
  EC_HIP(mark(6, stream));
  const void* dZop = P.dtype == EC_BF16 ? (const void*)w.dZb : (const void*)w.dZ;
  EC_HIP(ec::launch_router_dx(P.dtype, dZop, Wg, dX, N, E, P.EP, d, stream));
  EC_HIP(mark(7, stream));
  if (hs && N > 0) {
    // shared experts: their output gradient is dY itself (no gate)
    EC_HIP(ec::launch_gemm_dA(P.dtype, dY, Ws2, s.Hs1, s.Hs3, w.dHs, 1, N, d, hs, stream, true));
    EC_HIP(mark(8, stream));
    EC_HIP(ec::launch_shared_dW2(P.dtype, dY, s.As, dWs2, N, d, hs, w.spart, w.s_splits2, stream));
    EC_HIP(mark(9, stream));
    EC_HIP(ec::launch_gemm_dXe(P.dtype, w.dHs, Ws1, Ws3, dX, 1, N, d, hs, stream, true));
    EC_HIP(mark(10, stream));
    EC_HIP(ec::launch_shared_dW13(P.dtype, w.dHs, X, dWs1, dWs3, N, d, hs, w.spart,
                                  w.s_splits13, stream));
  } else {
    if (hs) {   // no tokens: zero shared weight gradients
      EC_HIP(ec::launch_zero(dWs1, (size_t)hs * d * P.esz, stream));
      EC_HIP(ec::launch_zero(dWs3, (size_t)hs * d * P.esz, stream));
      EC_HIP(ec::launch_zero(dWs2, (size_t)hs * d * P.esz, stream));
    }
    EC_HIP(mark(8, stream));
    EC_HIP(mark(9, stream));
    EC_HIP(mark(10, stream));
  }
  EC_HIP(mark(11, stream));
  EC_HIP(ec::launch_bwd_combine(P.dtype, dXe, s.slot, dX, dX, N, E, M, d, stream));
  EC_HIP(mark(12, stream));
  EC_HIP(ec::launch_router_dwg(P.dtype, dZop, X, dWg, w.part, w.splits, N, E, P.EP, d, stream));
  EC_HIP(mark(13, stream));
  return EC_OK;
}

int ec_tc_capacity(int32_t n_groups, const int32_t* group_lengths, int32_t n_experts,
                   int32_t top_k, double cf, int32_t* cap_out) {
  g_last_error[0] = '\0';
  if (n_groups < 0 || !group_lengths || !cap_out) return fail(EC_ERR_ARG, "bad arguments");
  if (n_experts < 1 || top_k < 1 || top_k > n_experts)
    return fail(EC_ERR_ARG, "need 1 <= top_k <= n_experts");
  if (!std::isfinite(cf)) return fail(EC_ERR_ARG, "capacity factor must be finite");
  for (int g = 0; g < n_groups; ++g) {
    const int L = group_lengths[g];
    if (L < 0) return fail(EC_ERR_SHAPE, "group length %d < 0", L);
    double c = cf <= 0 ? (double)L : std::ceil(cf * top_k * (double)L / n_experts - 1e-9);
    if (c > L) c = L;
    if (c < 0) c = 0;
    cap_out[g] = (int32_t)c;
  }
  return EC_OK;
}

size_t ec_tc_workspace_size(const ec_problem* p, int32_t top_k, int mode) {
  Plan P;
  long rmax;
  int rmax_e;
  if (tc_validate(p, top_k, &P, &rmax, &rmax_e) != EC_OK) return 0;
  Carve c(nullptr);
  carve_tc_route(c, P);
  if (mode == 1) carve_tc_fwd(c, P, rmax);
  else if (mode != 0) { fail(EC_ERR_ARG, "unknown workspace mode %d", mode); return 0; }
  return c.used;
}

int ec_tc_route(const ec_problem* p, int32_t top_k, const void* X, const void* Wg, float* S,
                float* G, int32_t* slot, int32_t* expert_rows, int32_t* sel_token, void* ws,
                size_t ws_bytes, hipStream_t stream) {
  Plan P;
  long rmax;
  int rmax_e;
  EC_TRY(tc_validate(p, top_k, &P, &rmax, &rmax_e));
  EC_TRY(check_ptr(X, "X"));
  EC_TRY(check_ptr(Wg, "Wg"));
  EC_TRY(check_ptr(S, "S", P.N == 0));
  EC_TRY(check_ptr(G, "G", P.N == 0));
  EC_TRY(check_ptr(slot, "slot", P.N == 0));
  EC_TRY(check_ptr(expert_rows, "expert_rows"));
  EC_TRY(check_ptr(sel_token, "sel_token", rmax == 0));
  Carve m(nullptr);
  carve_tc_route(m, P);
  EC_TRY(check_ptr(ws, "workspace"));
  if (ws_bytes < m.used)
    return fail(EC_ERR_WORKSPACE, "workspace %zu bytes < %zu required", ws_bytes, m.used);
  Carve c(ws);
  const TcRouteWs w = carve_tc_route(c, P);
  if (P.N == 0) return ec::launch_zero(expert_rows, (size_t)(P.E + 1) * 4, stream) == hipSuccess
                           ? EC_OK : fail(EC_ERR_HIP, "zero fill failed");
  return enqueue_tc_route(p, P, top_k, X, Wg, S, G, slot, expert_rows, sel_token, w, stream);
}

int ec_tc_forward(const ec_problem* p, int32_t top_k, const void* X, const void* Wg,
                  const void* W1, const void* W3, const void* W2, const void* Ws1,
                  const void* Ws3, const void* Ws2, void* Y, int32_t* expert_rows, void* ws,
                  size_t ws_bytes, hipStream_t stream) {
  Plan P;
  long rmax;
  int rmax_e;
  EC_TRY(tc_validate(p, top_k, &P, &rmax, &rmax_e));
  EC_TRY(check_ptr(X, "X"));
  EC_TRY(check_ptr(Wg, "Wg"));
  EC_TRY(check_ptr(W1, "W1"));
  EC_TRY(check_ptr(W3, "W3"));
  EC_TRY(check_ptr(W2, "W2"));
  EC_TRY(check_ptr(Ws1, "Ws1", P.hs == 0));
  EC_TRY(check_ptr(Ws3, "Ws3", P.hs == 0));
  EC_TRY(check_ptr(Ws2, "Ws2", P.hs == 0));
  EC_TRY(check_ptr(Y, "Y"));
  EC_TRY(check_ptr(expert_rows, "expert_rows", true));
  const size_t need = ec_tc_workspace_size(p, top_k, 1);
  EC_TRY(check_ptr(ws, "workspace"));
  if (ws_bytes < need)
    return fail(EC_ERR_WORKSPACE, "workspace %zu bytes < %zu required", ws_bytes, need);
  if (P.N == 0) return EC_OK;
  Carve c(ws);
  const TcRouteWs rw = carve_tc_route(c, P);
  const TcFwdWs w = carve_tc_fwd(c, P, rmax);
  int32_t* rows = expert_rows ? expert_rows : w.rows;
  EC_TRY(enqueue_tc_route(p, P, top_k, X, Wg, w.S, w.G, w.slot, rows, w.sel, rw, stream));
  if (P.dtype == EC_BF16) {
    // the W1/W3 product reads the kept rows of X itself (empty gather stage)
    EC_HIP(mark(3, stream));
    EC_HIP(ec::launch_gemm_w13_var(P.dtype, X, W1, W3, w.A, P.E, rows, rw.tiles13, rmax, rmax_e,
                                   P.d, P.h, stream, w.sel));
  } else {
    EC_HIP(ec::launch_gather(P.dtype, X, w.sel, w.Xe, rmax, P.d, P.N, stream, rows + P.E));
    EC_HIP(mark(3, stream));
    EC_HIP(ec::launch_gemm_w13_var(P.dtype, w.Xe, W1, W3, w.A, P.E, rows, rw.tiles13, rmax,
                                   rmax_e, P.d, P.h, stream));
  }
  EC_HIP(mark(4, stream));
  EC_HIP(ec::launch_gemm_w2_var(P.dtype, w.A, W2, w.O, P.E, rows, rw.tiles2, rmax, rmax_e, P.d,
                                P.h, stream));
  EC_HIP(mark(5, stream));
  if (P.hs) {
    EC_HIP(ec::launch_gemm_w13(P.dtype, X, Ws1, Ws3, w.As, nullptr, nullptr, 1, P.N, P.d, P.hs,
                               stream, true));
    EC_HIP(mark(6, stream));
    EC_HIP(ec::launch_gemm_w2(P.dtype, w.As, Ws2, Y, 1, P.N, P.d, P.hs, stream, true));
  } else {
    EC_HIP(mark(6, stream));
  }
  EC_HIP(mark(7, stream));
  EC_HIP(ec::launch_combine(P.dtype, w.O, w.G, w.slot, P.hs ? Y : nullptr, Y, P.N, P.E,
                            (int)rmax, P.d, stream, 0));
  EC_HIP(mark(8, stream));
  return EC_OK;
}

}  // extern "C"
