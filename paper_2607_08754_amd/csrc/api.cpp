// C ABI of the SLORR library: validation, workspace tables, per-call pointer
// table, hipGraph capture and replay. See include/slorr.h for the contract.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstring>
#include <list>
#include <mutex>
#include <new>
#include <stdexcept>
#include <string>
#include <utility>
#include <set>
#include <vector>

#include "kernels.hpp"
#include "plan.hpp"
#include "slorr.h"

struct slorr_plan_s {
  slorr::Plan p;
};

namespace {

thread_local std::string g_last_error;

slorr_status_t fail(slorr_status_t s, const std::string &msg) {
  g_last_error = msg;
  return s;
}

struct ApiError {
  slorr_status_t status;
  std::string msg;
};

void hip_check(hipError_t e, const char *what) {
  if (e != hipSuccess) throw ApiError{SLORR_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e)};
}

template <typename F>
slorr_status_t guarded(F &&f) {
  try {
    g_last_error.clear();
    return f();
  } catch (const ApiError &e) {
    return fail(e.status, e.msg);
  } catch (const slorr::HipError &e) {
    return fail(SLORR_ERR_HIP, e.what());
  } catch (const std::invalid_argument &e) {
    return fail(SLORR_ERR_INVALID_ARGUMENT, e.what());
  } catch (const std::domain_error &e) {
    return fail(SLORR_ERR_UNSUPPORTED, e.what());
  } catch (const std::bad_alloc &) {
    return fail(SLORR_ERR_INTERNAL, "host allocation failed");
  } catch (const std::exception &e) {
    return fail(SLORR_ERR_INTERNAL, e.what());
  } catch (...) {
    return fail(SLORR_ERR_INTERNAL, "unknown exception");
  }
}

bool aligned(const void *p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

// The integer an enum argument carries. C callers may pass any int, and in C++
// reading an enum object whose value lies outside its enumerators' range is
// undefined behaviour: the bits are copied out instead, then validated.
template <typename E>
int32_t bits(const E &e) {
  static_assert(sizeof(E) == sizeof(int32_t), "enum size");
  int32_t v;
  std::memcpy(&v, &e, sizeof v);
  return v;
}

void release_runtime(slorr::Plan &p) {
  if (p.device >= 0) {
    (void)hipSetDevice(p.device);
    (void)hipDeviceSynchronize();
  }
  if (p.graph_exec) (void)hipGraphExecDestroy(static_cast<hipGraphExec_t>(p.graph_exec));
  if (p.graph) (void)hipGraphDestroy(static_cast<hipGraph_t>(p.graph));
  p.graph_exec = p.graph = nullptr;
  if (p.capture_stream) (void)hipStreamDestroy(static_cast<hipStream_t>(p.capture_stream));
  p.capture_stream = nullptr;
  for (int k = 0; k < 2; ++k) {
    if (p.staging_event[k]) (void)hipEventDestroy(static_cast<hipEvent_t>(p.staging_event[k]));
    if (p.staging[k]) (void)hipHostFree(p.staging[k]);
    p.staging_event[k] = p.staging[k] = nullptr;
  }
  p.dyn_valid = false;
}

// Checks the arguments every entry point shares against the plan.
slorr::Plan &check_call(slorr_plan_t plan, int32_t n, const void *const *weights,
                        const slorr_shape_t *shapes, int32_t kind, int32_t iters) {
  if (!plan) throw std::invalid_argument("plan is NULL");
  slorr::Plan &p = plan->p;
  if (n != p.n) throw ApiError{SLORR_ERR_PLAN_MISMATCH, "n differs from the plan"};
  if (kind != p.kind) throw ApiError{SLORR_ERR_PLAN_MISMATCH, "kind differs from the plan"};
  if (iters != p.iters) throw ApiError{SLORR_ERR_PLAN_MISMATCH, "iters differs from the plan"};
  if (n > 0 && !shapes) throw std::invalid_argument("shapes is NULL");
  for (int i = 0; i < n; ++i)
    if (shapes[i].rows != p.shapes[i].rows || shapes[i].cols != p.shapes[i].cols)
      throw ApiError{SLORR_ERR_PLAN_MISMATCH, "shape of matrix " + std::to_string(i) + " differs from the plan"};
  if (n > 0 && !weights) throw std::invalid_argument("weights is NULL");
  return p;
}

// Pointer checks of weights and (if want_grad) gradient buffers, and that no
// gradient range overlaps a weight range or another gradient range.
void check_buffers(slorr::Plan &p, const void *const *weights, void *const *out_grads,
                   bool want_grad) {
  const int n = p.n;
  if (want_grad && n > 0 && !out_grads) throw std::invalid_argument("out_grads is NULL");
  auto &spans = p.spans;              // begin, (end, is_grad); capacity 2 n from the plan
  spans.clear();
  for (int i = 0; i < n; ++i) {
    const slorr::MatDesc &d = p.mats[i];
    if (d.empty) continue;
    const size_t elems = size_t(d.rows) * d.cols;
    if (!weights[i]) throw std::invalid_argument("weights[" + std::to_string(i) + "] is NULL");
    if (!aligned(weights[i], 16)) throw std::invalid_argument("weights[" + std::to_string(i) + "] must be 16-byte aligned");
    const uintptr_t wb = reinterpret_cast<uintptr_t>(weights[i]);
    spans.push_back({wb, {wb + elems * p.elem_bytes(), 0}});
    if (want_grad) {
      if (!out_grads[i]) throw std::invalid_argument("out_grads[" + std::to_string(i) + "] is NULL");
      if (!aligned(out_grads[i], 16)) throw std::invalid_argument("out_grads[" + std::to_string(i) + "] must be 16-byte aligned");
      const uintptr_t gb = reinterpret_cast<uintptr_t>(out_grads[i]);
      spans.push_back({gb, {gb + elems * p.grad_bytes(), 1}});
    }
  }
  std::sort(spans.begin(), spans.end());
  uintptr_t reach_all = 0, reach_grad = 0;   // furthest end of earlier spans / grad spans
  for (const auto &s : spans) {
    const bool is_grad = s.second.second != 0;
    if (s.first < reach_grad || (is_grad && s.first < reach_all))
      throw std::invalid_argument("out_grads overlap the weights or each other");
    reach_all = std::max(reach_all, s.second.first);
    if (is_grad) reach_grad = std::max(reach_grad, s.second.first);
  }
}

void check_device(const slorr::Plan &p) {
  if (!p.ws) throw ApiError{SLORR_ERR_WORKSPACE, "no workspace attached to the plan"};
  int dev = -1;
  hip_check(hipGetDevice(&dev), "hipGetDevice");
  if (dev != p.device) throw std::invalid_argument("current device differs from the workspace's device");
}

// Uploads the per-call pointer table and call parameters on stream s, only
// when they differ from what the workspace holds. The pinned staging buffer
// is reused only after its previous copy has completed.
void upload_call(slorr::Plan &p, const void *const *weights, void *const *out_grads, bool want_grad,
                 const slorr::CallParams &call, hipStream_t s) {
  const int n = p.n;
  std::vector<slorr::DynDesc> dyn(n);
  for (int i = 0; i < n; ++i) {
    dyn[i].w = p.mats[i].empty ? nullptr : weights[i];
    dyn[i].g = (want_grad && !p.mats[i].empty) ? out_grads[i] : nullptr;
  }
  const bool same = p.dyn_valid && p.call_cache.out_vals == call.out_vals &&
                    p.call_cache.gscale == call.gscale &&
                    std::memcmp(&p.call_cache.grad_scale, &call.grad_scale, sizeof(float)) == 0 &&
                    std::memcmp(p.dyn_cache.data(), dyn.data(), n * sizeof(slorr::DynDesc)) == 0;
  if (same) return;
  const int k = p.staging_next;
  p.staging_next ^= 1;
  hipEvent_t ev = static_cast<hipEvent_t>(p.staging_event[k]);
  hip_check(hipEventSynchronize(ev), "hipEventSynchronize");
  char *st = static_cast<char *>(p.staging[k]);
  std::memset(st, 0, p.dyn_bytes());
  if (n) std::memcpy(st, dyn.data(), n * sizeof(slorr::DynDesc));
  std::memcpy(st + (p.off_call - p.off_dyn), &call, sizeof(call));
  hip_check(hipMemcpyAsync(static_cast<char *>(p.ws) + p.off_dyn, st, p.dyn_bytes(),
                           hipMemcpyHostToDevice, s),
            "hipMemcpyAsync pointer table");
  hip_check(hipEventRecord(ev, s), "hipEventRecord");
  p.dyn_cache = dyn;
  p.call_cache = call;
  p.dyn_valid = true;
}

// Validates a forward call against the plan and uploads its tables. Returns
// the plan; nothing is enqueued on failure except when the upload itself fails.
slorr::Plan &prepare_call(slorr_plan_t plan, int32_t n, const void *const *weights,
                          const slorr_shape_t *shapes, int32_t kind, int32_t iters,
                          float *out_vals, void *const *out_grads, float grad_scale,
                          hipStream_t s) {
  slorr::Plan &p = check_call(plan, n, weights, shapes, kind, iters);
  if (!out_vals) throw std::invalid_argument("out_vals is NULL");
  if (!aligned(out_vals, 4)) throw std::invalid_argument("out_vals must be 4-byte aligned");
  const bool want_grad = !(p.flags & (SLORR_VALUES_ONLY | SLORR_DEFER_GRAD));
  check_buffers(p, weights, out_grads, want_grad);
  check_device(p);
  slorr::CallParams call{};
  call.out_vals = out_vals;
  call.gscale = nullptr;
  call.grad_scale = grad_scale;
  upload_call(p, weights, out_grads, want_grad, call, s);
  return p;
}

// A plan for a set of shapes with the given options (host only).
slorr_plan_s *new_plan(int32_t n, const slorr_shape_t *shapes, int32_t dtype, int32_t kind,
                       const slorr_options_t &o, size_t *workspace_bytes) {
  if (n < 0) throw std::invalid_argument("n must be >= 0");
  if (n > 0 && !shapes) throw std::invalid_argument("shapes is NULL");
  auto *h = new slorr_plan_s();
  try {
    slorr::Plan &p = h->p;
    p.n = n;
    p.dtype = dtype;
    p.kind = kind;
    p.iters = o.iters == 0 ? 6 : o.iters;
    p.degree = o.degree == 0 ? 5 : o.degree;
    p.ell = o.ell == 0.0 ? 1e-3 : o.ell;
    p.safety = o.safety == 0.0 ? 0.01 : (o.safety < 0.0 ? 0.0 : o.safety);
    p.eps = o.eps;
    p.flags = o.flags;
    p.grad_dtype = bits(o.grad_dtype);
    p.shapes.assign(shapes, shapes + n);
    if (o.coeffs) {
      if (p.iters < 1 || p.iters > 1000) throw std::invalid_argument("iters must be in [1, 1000]");
      p.coeffs.assign(o.coeffs, o.coeffs + size_t(p.iters) * 3);
    }
    slorr::build_plan(p);
    *workspace_bytes = p.ws_bytes;
  } catch (...) {
    delete h;
    throw;
  }
  return h;
}

// Binds caller memory as the plan's workspace: static tables (one synchronous
// copy), pinned staging buffers for the per-call table, the current device.
void attach(slorr::Plan &p, void *dev_ptr, size_t bytes) {
  if (!dev_ptr) throw ApiError{SLORR_ERR_WORKSPACE, "workspace pointer is NULL"};
  if (!aligned(dev_ptr, 256)) throw ApiError{SLORR_ERR_WORKSPACE, "workspace must be 256-byte aligned"};
  if (bytes < p.ws_bytes)
    throw ApiError{SLORR_ERR_WORKSPACE, "workspace too small: need " + std::to_string(p.ws_bytes) +
                                            " bytes, got " + std::to_string(bytes)};
  release_runtime(p);
  p.ws = nullptr;
  p.state_ready = false;
  int dev = -1;
  hip_check(hipGetDevice(&dev), "hipGetDevice");
  std::vector<char> host(p.off_static_end, 0);
  auto put = [&](size_t off, const void *src, size_t n) {
    if (n) std::memcpy(host.data() + off, src, n);
  };
  put(p.off_mats, p.mats.data(), p.mats.size() * sizeof(slorr::MatDesc));
  put(p.off_tiles, p.tiles.data(), p.tiles.size() * sizeof(slorr::Tile));
  put(p.off_chunks, p.chunks.data(), p.chunks.size() * sizeof(slorr::Chunk));
  hip_check(hipMemcpy(dev_ptr, host.data(), host.size(), hipMemcpyHostToDevice), "hipMemcpy tables");
  for (int k = 0; k < 2; ++k) {
    hip_check(hipHostMalloc(&p.staging[k], p.dyn_bytes(), hipHostMallocDefault), "hipHostMalloc");
    hipEvent_t ev;
    hip_check(hipEventCreateWithFlags(&ev, hipEventDisableTiming), "hipEventCreate");
    p.staging_event[k] = ev;
  }
  p.device = dev;
  p.ws = dev_ptr;
  p.dyn_valid = false;
}

// The forward + backward call on a plan: validation, table upload, then the
// captured graph (captured on first use) or the eager schedule.
void run_fwd_bwd(slorr_plan_t plan, int32_t n, const void *const *weights, const slorr_shape_t *shapes,
                 int32_t kind, int32_t iters, float *out_vals, void *const *out_grads, float grad_scale,
                 void *stream) {
  hipStream_t s = static_cast<hipStream_t>(stream);
  slorr::Plan &p = prepare_call(plan, n, weights, shapes, kind, iters, out_vals, out_grads, grad_scale, s);
  p.state_ready = false;
  if (p.flags & SLORR_NO_GRAPH) {
    slorr::enqueue(p, s);
    p.state_ready = !(p.flags & SLORR_VALUES_ONLY);
    return;
  }
  if (!p.graph_exec) {
    hipStream_t cs;
    hip_check(hipStreamCreateWithFlags(&cs, hipStreamNonBlocking), "hipStreamCreate");
    p.capture_stream = cs;
    hip_check(hipStreamBeginCapture(cs, hipStreamCaptureModeRelaxed), "hipStreamBeginCapture");
    try {
      slorr::enqueue(p, cs);
    } catch (...) {
      hipGraph_t g = nullptr;
      (void)hipStreamEndCapture(cs, &g);
      if (g) (void)hipGraphDestroy(g);
      throw;
    }
    hipGraph_t g = nullptr;
    hip_check(hipStreamEndCapture(cs, &g), "hipStreamEndCapture");
    p.graph = g;
    hipGraphExec_t ge = nullptr;
    hip_check(hipGraphInstantiate(&ge, g, nullptr, nullptr, 0), "hipGraphInstantiate");
    p.graph_exec = ge;
  }
  hip_check(hipGraphLaunch(static_cast<hipGraphExec_t>(p.graph_exec), s), "hipGraphLaunch");
  p.state_ready = !(p.flags & SLORR_VALUES_ONLY);
}

// ------------------------------------------------- internal plan cache
// Options of NULL-plan calls, per calling thread (slorr_cache_config).
thread_local int32_t g_call_dtype = SLORR_F32;
thread_local slorr_options_t g_call_opts = {6, 5, 1e-3, nullptr, 0.0f, 0u, SLORR_F32, 0.01};
thread_local std::vector<double> g_call_coeffs;

struct CacheEntry {
  int device;
  void *stream;
  int32_t dtype, kind;
  int32_t iters, degree;
  double ell, safety;
  float eps;
  uint32_t flags;
  int32_t grad_dtype;
  std::vector<double> coeffs;
  std::vector<slorr_shape_t> shapes;
  slorr_plan_t plan = nullptr;
  void *ws = nullptr;
};
constexpr size_t kCacheCapacity = 8;
std::mutex g_cache_mu;
std::list<CacheEntry> g_cache;      // most recently used first

void drop_entry(CacheEntry &e) {
  if (e.plan) {
    release_runtime(e.plan->p);       // waits for the plan's work on its device
    delete e.plan;
    e.plan = nullptr;
  }
  if (e.ws) (void)hipFree(e.ws);
  e.ws = nullptr;
}

bool same_key(const CacheEntry &e, const CacheEntry &k) {
  if (e.device != k.device || e.stream != k.stream || e.dtype != k.dtype || e.kind != k.kind ||
      e.iters != k.iters || e.degree != k.degree || e.flags != k.flags || e.grad_dtype != k.grad_dtype ||
      std::memcmp(&e.ell, &k.ell, sizeof(double)) != 0 || std::memcmp(&e.eps, &k.eps, sizeof(float)) != 0 ||
      std::memcmp(&e.safety, &k.safety, sizeof(double)) != 0 ||
      e.coeffs != k.coeffs || e.shapes.size() != k.shapes.size())
    return false;
  for (size_t i = 0; i < e.shapes.size(); ++i)
    if (e.shapes[i].rows != k.shapes[i].rows || e.shapes[i].cols != k.shapes[i].cols) return false;
  return true;
}

// The cached plan for a NULL-plan call (created with a library-owned workspace
// on the current device if absent); the caller holds g_cache_mu.
slorr_plan_t cached_plan(int32_t n, const slorr_shape_t *shapes, int32_t kind, int32_t iters,
                         void *stream) {
  if (n < 0) throw std::invalid_argument("n must be >= 0");
  if (n > 0 && !shapes) throw std::invalid_argument("shapes is NULL");
  if (iters < 1 || iters > 1000) throw std::invalid_argument("iters must be in [1, 1000]");
  CacheEntry k;
  hip_check(hipGetDevice(&k.device), "hipGetDevice");
  k.stream = stream;
  k.dtype = g_call_dtype;
  k.kind = kind;
  k.iters = iters;
  k.degree = g_call_opts.degree;
  k.ell = g_call_opts.ell;
  k.safety = g_call_opts.safety;
  k.eps = g_call_opts.eps;
  k.flags = g_call_opts.flags;
  k.grad_dtype = bits(g_call_opts.grad_dtype);
  k.coeffs = g_call_coeffs;
  if (!k.coeffs.empty() && k.coeffs.size() != size_t(iters) * 3)
    throw std::invalid_argument("the configured coefficient table has a different number of steps");
  k.shapes.assign(shapes, shapes + n);
  for (auto it = g_cache.begin(); it != g_cache.end(); ++it) {
    if (same_key(*it, k)) {
      g_cache.splice(g_cache.begin(), g_cache, it);
      return g_cache.front().plan;
    }
  }
  slorr_options_t o = g_call_opts;
  o.iters = iters;
  o.coeffs = k.coeffs.empty() ? nullptr : k.coeffs.data();
  size_t bytes = 0;
  CacheEntry e = k;
  e.plan = new_plan(n, shapes, k.dtype, kind, o, &bytes);
  try {
    void *ws = nullptr;
    hip_check(hipMalloc(&ws, bytes), "hipMalloc workspace");
    e.ws = ws;
    attach(e.plan->p, ws, bytes);
  } catch (...) {
    drop_entry(e);
    throw;
  }
  if (g_cache.size() >= kCacheCapacity) {
    drop_entry(g_cache.back());
    g_cache.pop_back();
  }
  g_cache.push_front(std::move(e));
  return g_cache.front().plan;
}

}  // namespace

extern "C" {

void slorr_default_options(slorr_options_t *o) {
  if (!o) return;
  o->iters = 6;
  o->degree = 5;
  o->ell = 1e-3;
  o->coeffs = nullptr;
  o->eps = 0.0f;
  o->flags = 0;
  o->grad_dtype = SLORR_F32;
  o->safety = 0.01;
}

slorr_status_t slorr_pe_coefficients(double ell, int32_t degree, int32_t iters, double *out) {
  return guarded([&]() -> slorr_status_t {
    if (!out) throw std::invalid_argument("out is NULL");
    if (iters < 1 || iters > 1000) throw std::invalid_argument("iters must be in [1, 1000]");
    if (degree != 3 && degree != 5) throw std::domain_error("degree must be 3 or 5");
    if (!(ell > 0.0 && ell < 1.0)) throw std::invalid_argument("ell must be in (0, 1)");
    slorr::greedy_schedule(ell, degree, iters, out);
    return SLORR_OK;
  });
}

slorr_status_t slorr_plan(slorr_plan_t *plan, int32_t n, const slorr_shape_t *shapes, slorr_dtype_t dtype,
                          slorr_kind_t kind, const slorr_options_t *opts, size_t *workspace_bytes) {
  if (plan) *plan = nullptr;
  return guarded([&]() -> slorr_status_t {
    if (!plan) throw std::invalid_argument("plan is NULL");
    if (!workspace_bytes) throw std::invalid_argument("workspace_bytes is NULL");
    slorr_options_t o;
    slorr_default_options(&o);
    if (opts) o = *opts;
    *plan = new_plan(n, shapes, bits(dtype), bits(kind), o, workspace_bytes);
    return SLORR_OK;
  });
}

slorr_status_t slorr_plan_get_info(slorr_plan_t plan, slorr_plan_info_t *info) {
  return guarded([&]() -> slorr_status_t {
    if (!plan || !info) throw std::invalid_argument("NULL argument");
    const slorr::Plan &p = plan->p;
    info->n = p.n;
    info->groups = p.groups;
    info->iters = p.iters;
    info->launches = int32_t(p.launches.size());
    int64_t tiles = 0;
    for (const auto &l : p.launches)
      if (l.op == slorr::Op::Gram || l.op == slorr::Op::Poly || l.op == slorr::Op::Update ||
          l.op == slorr::Op::Last)
        tiles += l.grid;
    info->gemm_tiles = tiles;
    info->paper_flops = p.paper_flops;
    info->mfma_flops = p.mfma_flops;
    info->weight_bytes = p.weight_bytes;
    info->workspace_bytes = p.ws_bytes;
    return SLORR_OK;
  });
}

slorr_status_t slorr_plan_get_launches(slorr_plan_t plan, int32_t *ops, double *alg_flops, int32_t *tile_edge) {
  return guarded([&]() -> slorr_status_t {
    if (!plan) throw std::invalid_argument("plan is NULL");
    const slorr::Plan &p = plan->p;
    for (size_t i = 0; i < p.launches.size(); ++i) {
      const slorr::Launch &l = p.launches[i];
      const bool gemm = l.op == slorr::Op::Gram || l.op == slorr::Op::Poly || l.op == slorr::Op::Update ||
                        l.op == slorr::Op::Last;
      if (ops) ops[i] = int32_t(l.op);
      if (tile_edge) tile_edge[i] = gemm ? (l.cfg == slorr::kCfg256 ? 256 : 128) : 0;
      if (!alg_flops) continue;
      double f = 0.0;
      if (gemm) {
        std::set<int32_t> mats;       // matrices of the launch (one product each)
        for (int k = 0; k < l.grid; ++k) {
          const slorr::Tile &t = p.tiles[l.tile_first + k];
          if (t.mat >= 0) mats.insert(t.mat);
        }
        for (int32_t m : mats) {
          const slorr::MatDesc &d = p.mats[m];
          const double P = d.P, Q = d.Q;
          f += l.op == slorr::Op::Poly ? 2.0 * P * P * P : 2.0 * P * P * Q;
        }
      }
      alg_flops[i] = f;
    }
    return SLORR_OK;
  });
}

slorr_status_t slorr_plan_set_workspace(slorr_plan_t plan, void *dev_ptr, size_t bytes) {
  return guarded([&]() -> slorr_status_t {
    if (!plan) throw std::invalid_argument("plan is NULL");
    attach(plan->p, dev_ptr, bytes);
    return SLORR_OK;
  });
}

slorr_status_t slorr_reg_fwd_bwd(slorr_plan_t plan, int32_t n, const void *const *weights,
                                 const slorr_shape_t *shapes, slorr_kind_t kind, int32_t iters,
                                 float *out_vals, void *const *out_grads, float grad_scale,
                                 void *stream) {
  return guarded([&]() -> slorr_status_t {
    const int32_t k = bits(kind);
    if (plan) {
      run_fwd_bwd(plan, n, weights, shapes, k, iters, out_vals, out_grads, grad_scale, stream);
      return SLORR_OK;
    }
    // internal plan cache: one plan and workspace per (device, stream, dtype,
    // options, kind, iters, shapes); calls on one entry are serialised. The
    // argument checks that need no plan run before any device call.
    if (n < 0) throw std::invalid_argument("n must be >= 0");
    if (n > 0 && (!shapes || !weights)) throw std::invalid_argument("shapes or weights is NULL");
    if (iters < 1 || iters > 1000) throw std::invalid_argument("iters must be in [1, 1000]");
    if (!out_vals) throw std::invalid_argument("out_vals is NULL");
    if (!aligned(out_vals, 4)) throw std::invalid_argument("out_vals must be 4-byte aligned");
    if (n > 0 && !out_grads && !(g_call_opts.flags & (SLORR_VALUES_ONLY | SLORR_DEFER_GRAD)))
      throw std::invalid_argument("out_grads is NULL");
    std::lock_guard<std::mutex> lock(g_cache_mu);
    slorr_plan_t c = cached_plan(n, shapes, k, iters, stream);
    run_fwd_bwd(c, n, weights, shapes, k, iters, out_vals, out_grads, grad_scale, stream);
    return SLORR_OK;
  });
}

void slorr_cache_config(slorr_dtype_t dtype, const slorr_options_t *opts) {
  g_call_dtype = bits(dtype);
  slorr_default_options(&g_call_opts);
  g_call_coeffs.clear();
  if (opts) {
    g_call_opts = *opts;
    if (opts->coeffs && opts->iters > 0 && opts->iters <= 1000)
      g_call_coeffs.assign(opts->coeffs, opts->coeffs + size_t(opts->iters) * 3);
  }
  g_call_opts.coeffs = nullptr;
}

slorr_status_t slorr_cache_clear(void) {
  return guarded([&]() -> slorr_status_t {
    std::lock_guard<std::mutex> lock(g_cache_mu);
    while (!g_cache.empty()) {
      drop_entry(g_cache.back());
      g_cache.pop_back();
    }
    return SLORR_OK;
  });
}

slorr_status_t slorr_reg_grad(slorr_plan_t plan, int32_t n, const void *const *weights,
                              const slorr_shape_t *shapes, slorr_kind_t kind, int32_t iters,
                              void *const *out_grads, const float *scales, float grad_scale,
                              void *stream) {
  return guarded([&]() -> slorr_status_t {
    hipStream_t s = static_cast<hipStream_t>(stream);
    slorr::Plan &p = check_call(plan, n, weights, shapes, bits(kind), iters);
    if (p.flags & SLORR_VALUES_ONLY)
      throw std::invalid_argument("the plan computes values only (SLORR_VALUES_ONLY)");
    if (!p.state_ready) throw std::invalid_argument("no forward state: run slorr_reg_fwd_bwd on this plan first");
    if (scales && !aligned(scales, 4)) throw std::invalid_argument("scales must be 4-byte aligned");
    check_buffers(p, weights, out_grads, true);
    check_device(p);
    slorr::CallParams call = p.call_cache;     // keeps out_vals of the forward call
    call.gscale = scales;
    call.grad_scale = grad_scale;
    upload_call(p, weights, out_grads, true, call, s);
    slorr::enqueue_grad(p, s);
    return SLORR_OK;
  });
}

slorr_status_t slorr_decoupled_apply(slorr_plan_t plan, int32_t n, void *const *weights,
                                     const slorr_shape_t *shapes, const void *const *grads,
                                     const float *steps, float step, void *stream) {
  return guarded([&]() -> slorr_status_t {
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (!plan) throw std::invalid_argument("plan is NULL");
    const void *const *w = reinterpret_cast<const void *const *>(weights);
    void *const *g = const_cast<void *const *>(grads);
    slorr::Plan &p = check_call(plan, n, w, shapes, plan->p.kind, plan->p.iters);
    if (steps && !aligned(steps, 4)) throw std::invalid_argument("steps must be 4-byte aligned");
    check_buffers(p, w, g, true);
    check_device(p);
    slorr::CallParams call = p.call_cache;
    call.gscale = steps;
    call.grad_scale = step;
    upload_call(p, w, g, true, call, s);
    slorr::enqueue_apply(p, s);
    return SLORR_OK;
  });
}

slorr_status_t slorr_reg_fwd_bwd_profiled(slorr_plan_t plan, int32_t n,
                                          const void *const *weights, const slorr_shape_t *shapes,
                                          slorr_kind_t kind, int32_t iters, float *out_vals,
                                          void *const *out_grads, float grad_scale, void *stream,
                                          float *launch_ms, int32_t *launch_op) {
  return guarded([&]() -> slorr_status_t {
    if (!launch_ms) throw std::invalid_argument("launch_ms is NULL");
    hipStream_t s = static_cast<hipStream_t>(stream);
    slorr::Plan &p = prepare_call(plan, n, weights, shapes, bits(kind), iters, out_vals, out_grads,
                                  grad_scale, s);
    const size_t nl = p.launches.size();
    std::vector<hipEvent_t> ev(2 * nl, nullptr);
    struct Guard {
      std::vector<hipEvent_t> &e;
      ~Guard() {
        for (auto x : e)
          if (x) (void)hipEventDestroy(x);
      }
    } guard{ev};
    // device-scope release: the events add no system-scope cache write-back
    // to the interval they time (the graph's launches have none either)
    for (auto &e : ev) hip_check(hipEventCreateWithFlags(&e, hipEventReleaseToDevice), "hipEventCreateWithFlags");
    p.state_ready = false;
    slorr::enqueue(p, s, ev.data());
    p.state_ready = !(p.flags & SLORR_VALUES_ONLY);
    hip_check(hipStreamSynchronize(s), "hipStreamSynchronize");
    for (size_t i = 0; i < nl; ++i) {
      float ms = 0.0f;
      hip_check(hipEventElapsedTime(&ms, ev[2 * i], ev[2 * i + 1]), "hipEventElapsedTime");
      launch_ms[i] = ms;
      if (launch_op) launch_op[i] = int32_t(p.launches[i].op);
    }
    return SLORR_OK;
  });
}

slorr_status_t slorr_reg_fwd_bwd_noalloc(slorr_plan_t plan, int32_t n, const void *const *weights,
                                         const slorr_shape_t *shapes, slorr_kind_t kind, int32_t iters,
                                         float *out_vals, void *const *out_grads, float grad_scale,
                                         void *stream) {
  return guarded([&]() -> slorr_status_t {
    hipStream_t s = static_cast<hipStream_t>(stream);
    slorr::Plan &p = check_call(plan, n, weights, shapes, bits(kind), iters);
    if (p.flags & SLORR_DEFER_GRAD)
      throw std::invalid_argument("SLORR_DEFER_GRAD needs the plan's own workspace (slorr_reg_fwd_bwd)");
    if (!out_vals) throw std::invalid_argument("out_vals is NULL");
    if (!aligned(out_vals, 4)) throw std::invalid_argument("out_vals must be 4-byte aligned");
    const bool want_grad = !(p.flags & SLORR_VALUES_ONLY);
    check_buffers(p, weights, out_grads, want_grad);
    if (p.ws_bytes > slorr::kScratchBytes)
      throw ApiError{SLORR_ERR_WORKSPACE, "the plan needs " + std::to_string(p.ws_bytes) +
                                              " bytes of workspace; the static scratch holds " +
                                              std::to_string(slorr::kScratchBytes)};
    void *scr = slorr::scratch_address();
    // the call's pointer table into the host image, then the whole table
    // region to the scratch array, ordered on the caller's stream
    char *img = p.image.data();
    auto *dyn = reinterpret_cast<slorr::DynDesc *>(img + p.off_dyn);
    for (int i = 0; i < n; ++i) {
      dyn[i].w = p.mats[i].empty ? nullptr : weights[i];
      dyn[i].g = (want_grad && !p.mats[i].empty) ? out_grads[i] : nullptr;
    }
    slorr::CallParams call{};
    call.out_vals = out_vals;
    call.gscale = nullptr;
    call.grad_scale = grad_scale;
    std::memcpy(img + p.off_call, &call, sizeof(call));
    hip_check(hipMemcpyAsync(scr, img, p.image.size(), hipMemcpyHostToDevice, s), "hipMemcpyAsync tables");
    // the iterate state of this call lives in the scratch array, not in the
    // plan's workspace: no deferred gradient can follow it
    p.state_ready = false;
    slorr::enqueue(p, s, nullptr, scr);
    return SLORR_OK;
  });
}

slorr_status_t slorr_plan_destroy(slorr_plan_t plan) {
  return guarded([&]() -> slorr_status_t {
    if (!plan) return SLORR_OK;
    release_runtime(plan->p);
    delete plan;
    return SLORR_OK;
  });
}

const char *slorr_status_string(slorr_status_t status) {
  switch (bits(status)) {
    case SLORR_OK: return "SLORR_OK";
    case SLORR_ERR_INVALID_ARGUMENT: return "SLORR_ERR_INVALID_ARGUMENT";
    case SLORR_ERR_UNSUPPORTED: return "SLORR_ERR_UNSUPPORTED";
    case SLORR_ERR_PLAN_MISMATCH: return "SLORR_ERR_PLAN_MISMATCH";
    case SLORR_ERR_WORKSPACE: return "SLORR_ERR_WORKSPACE";
    case SLORR_ERR_HIP: return "SLORR_ERR_HIP";
    case SLORR_ERR_INTERNAL: return "SLORR_ERR_INTERNAL";
  }
  return "SLORR_UNKNOWN_STATUS";
}

const char *slorr_last_error(void) { return g_last_error.c_str(); }

}  // extern "C"
