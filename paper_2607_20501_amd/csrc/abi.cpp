// The C ABI (include/mk.h): module lifetime, introspection, implementation
// swapping, the executor and per-stage verification.
//
// The executor is MKEvolve's top-level module S (Sec. 3; App. H.1): it only
// binds buffers and chains the subkernels in order on one stream, doing no
// arithmetic of its own.  Verification follows the decomposed checking of
// App. D: every materialised intermediate is a stage that can be compared
// against its own reference, besides the end-to-end output.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstring>
#include <map>
#include <string>
#include <vector>

#include "../../include/mk.h"
#include "impls.hpp"
#include "plan.hpp"

namespace mk {
const char* last_error();
}

struct mk_module {
  mk::Plan plan;
  std::vector<hipEvent_t> events;   // per-subkernel timing
  int event_device = -1;
  std::vector<hipEvent_t> prof;     // launch-level profile (2 per launch)
  mk::LaunchTimer timer;
  bool profiling = false;
  ~mk_module() {
    for (hipEvent_t e : events) (void)hipEventDestroy(e);
    for (hipEvent_t e : prof) (void)hipEventDestroy(e);
  }
};

using mk::fail;

static void copy_shape(const mk_shape& s, mk_shape& d) {
  d = s;
  for (int k = s.ndim; k < 4; ++k) d.dims[k] = 0;
}

extern "C" {

const char* mk_status_str(mk_status s) {
  switch (s) {
    case MK_OK: return "MK_OK";
    case MK_E_INVALID_ARG: return "MK_E_INVALID_ARG";
    case MK_E_SHAPE: return "MK_E_SHAPE";
    case MK_E_DTYPE: return "MK_E_DTYPE";
    case MK_E_DECOMP: return "MK_E_DECOMP";
    case MK_E_UNSUPPORTED: return "MK_E_UNSUPPORTED";
    case MK_E_WORKSPACE: return "MK_E_WORKSPACE";
    case MK_E_HIP: return "MK_E_HIP";
    case MK_E_INTERNAL: return "MK_E_INTERNAL";
  }
  return "unknown status";
}

const char* mk_last_error(void) { return mk::last_error(); }

mk_status mk_decomposition_preset(const mk_module_desc* desc, int32_t preset, int32_t* group_of_op) {
  try {
    return mk::preset(desc, preset, group_of_op);
  } catch (...) {
    return fail(MK_E_INTERNAL, "exception in mk_decomposition_preset");
  }
}

mk_status mk_module_create(const mk_module_desc* desc, const int32_t* group_of_op,
                           mk_module** out) {
  if (!out) return fail(MK_E_INVALID_ARG, "out is null");
  *out = nullptr;
  try {
    mk_module* m = new mk_module();
    mk_status s = mk::build_plan(desc, group_of_op, m->plan);
    if (s != MK_OK) {
      delete m;
      return s;
    }
    *out = m;
    return MK_OK;
  } catch (...) {
    return fail(MK_E_INTERNAL, "exception in mk_module_create");
  }
}

void mk_module_destroy(mk_module* m) { delete m; }

static int64_t ws_total(const mk::Plan& p) {
  return p.scratch_bytes ? p.scratch_off + p.scratch_bytes : p.ws_intermediate;
}

mk_status mk_module_info(const mk_module* m, mk_module_info_t* info) {
  if (!m || !info) return fail(MK_E_INVALID_ARG, "null argument");
  const mk::Plan& p = m->plan;
  info->n_subkernels = (int32_t)p.subs.size();
  info->n_ops = (int32_t)p.ops.size();
  copy_shape(p.vshape.back(), info->out_shape);
  info->ws_bytes = ws_total(p);
  info->ws_intermediate_bytes = p.ws_intermediate;
  info->flops = p.flops;
  info->alg_bytes = p.alg_bytes;
  return MK_OK;
}

mk_status mk_subkernel_info(const mk_module* m, int32_t i, mk_subkernel_info_t* info) {
  if (!m || !info) return fail(MK_E_INVALID_ARG, "null argument");
  const mk::Plan& p = m->plan;
  if (i < 0 || i >= (int32_t)p.subs.size()) return fail(MK_E_INVALID_ARG, "subkernel index");
  const mk::Subkernel& s = p.subs[i];
  info->op_begin = s.op_begin;
  info->op_end = s.op_end;
  info->out_value = s.out_value;
  copy_shape(p.vshape[s.out_value], info->out_shape);
  info->out_bytes = s.out_bytes;
  info->ws_offset = s.ws_offset;
  info->flops = s.flops;
  info->alg_bytes = s.alg_bytes;
  info->family = s.family;
  info->impl = s.impl;
  info->n_launches = mk::impl_launches(p, s, s.impl);
  info->scratch_bytes = mk::impl_scratch(p, s, s.impl);
  info->uses_mfma = mk::impl_uses_mfma(p, s, s.impl) ? 1 : 0;
  info->tuned_limit = mk::tuned_limit(p, s);
  return MK_OK;
}

mk_status mk_subkernel_select(mk_module* m, int32_t i, int32_t impl_id) {
  if (!m) return fail(MK_E_INVALID_ARG, "null module");
  mk::Plan& p = m->plan;
  if (i < 0 || i >= (int32_t)p.subs.size()) return fail(MK_E_INVALID_ARG, "subkernel index");
  if (!mk::impl_exists(p, p.subs[i], impl_id))
    return fail(MK_E_UNSUPPORTED, "subkernel " + std::to_string(i) + " has no implementation " +
                                      std::to_string(impl_id));
  p.subs[i].impl = impl_id;
  return MK_OK;
}

mk_status mk_workspace_size(const mk_module* m, int64_t* bytes) {
  if (!m || !bytes) return fail(MK_E_INVALID_ARG, "null argument");
  *bytes = ws_total(m->plan);
  return MK_OK;
}

static mk_status bind_values(const mk_module* m, const void* const* in, void* out, void* ws,
                      int64_t ws_bytes, std::vector<void*>& vals) {
  const mk::Plan& p = m->plan;
  if (p.n_inputs > 0 && !in) return fail(MK_E_INVALID_ARG, "dev_inputs is null");
  for (int i = 0; i < p.n_inputs; ++i)
    if (!in[i]) return fail(MK_E_INVALID_ARG, "dev_inputs[" + std::to_string(i) + "] is null");
  if (!out) return fail(MK_E_INVALID_ARG, "dev_out is null");
  const int64_t need = ws_total(p);
  if (ws_bytes < need)
    return fail(MK_E_WORKSPACE, "workspace of " + std::to_string(ws_bytes) + " bytes; need " +
                                    std::to_string(need));
  if (need > 0 && !ws) return fail(MK_E_INVALID_ARG, "dev_ws is null");
  vals.assign(p.vshape.size(), nullptr);
  for (int i = 0; i < p.n_inputs; ++i) vals[i] = const_cast<void*>(in[i]);
  for (const mk::Subkernel& s : p.subs)
    vals[s.out_value] = s.ws_offset < 0 ? out : (char*)ws + s.ws_offset;
  return MK_OK;
}

static mk_status hip_fail(hipError_t e, const char* what) {
  return fail(MK_E_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

mk_status mk_run(mk_module* m, const void* const* dev_inputs, void* dev_out, void* dev_ws,
                 int64_t ws_bytes, void* stream, float* per_subkernel_ms) {
  if (!m) return fail(MK_E_INVALID_ARG, "null module");
  try {
    std::vector<void*> vals;
    mk_status s = bind_values(m, dev_inputs, dev_out, dev_ws, ws_bytes, vals);
    if (s != MK_OK) return s;
    const mk::Plan& p = m->plan;
    hipStream_t st = (hipStream_t)stream;
    void* scratch = p.scratch_bytes ? (char*)dev_ws + p.scratch_off : nullptr;
    const size_t ns = p.subs.size();
    if (per_subkernel_ms) {
      int dev = 0;
      hipError_t e = hipGetDevice(&dev);
      if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
      if (m->event_device != dev || m->events.size() != 2 * ns) {
        for (hipEvent_t ev : m->events) (void)hipEventDestroy(ev);
        m->events.assign(2 * ns, nullptr);
        for (auto& ev : m->events) {
          e = hipEventCreate(&ev);
          if (e != hipSuccess) return hip_fail(e, "hipEventCreate");
        }
        m->event_device = dev;
      }
    }
    for (size_t i = 0; i < ns; ++i) {
      const mk::Subkernel& sk = p.subs[i];
      if (per_subkernel_ms) {
        hipError_t e = hipEventRecord(m->events[2 * i], st);
        if (e != hipSuccess) return hip_fail(e, "hipEventRecord");
      }
      mk::LaunchTimer* tm = nullptr;
      if (m->profiling) {
        m->timer.stream = st;
        if (i == 0) m->timer.pos = 0;
        tm = &m->timer;
      }
      s = mk::run_subkernel(p, sk, vals, vals[sk.out_value], scratch, st, tm);
      if (s != MK_OK) return s;
      if (per_subkernel_ms) {
        hipError_t e = hipEventRecord(m->events[2 * i + 1], st);
        if (e != hipSuccess) return hip_fail(e, "hipEventRecord");
      }
    }
    if (per_subkernel_ms) {
      hipError_t e = hipEventSynchronize(m->events[2 * ns - 1]);
      if (e != hipSuccess) return hip_fail(e, "hipEventSynchronize");
      for (size_t i = 0; i < ns; ++i) {
        e = hipEventElapsedTime(&per_subkernel_ms[i], m->events[2 * i], m->events[2 * i + 1]);
        if (e != hipSuccess) return hip_fail(e, "hipEventElapsedTime");
      }
    }
    return MK_OK;
  } catch (...) {
    return fail(MK_E_INTERNAL, "exception in mk_run");
  }
}

mk_status mk_swap_decide(int32_t n, const float* ms_selected, const float* ms_reference,
                         float tau, int32_t* swap, int32_t* triggered) {
  if (n < 0 || (n > 0 && (!ms_selected || !ms_reference || !swap)))
    return fail(MK_E_INVALID_ARG, "mk_swap_decide: null array or n < 0");
  bool any_fast = false;
  for (int32_t i = 0; i < n; ++i) {
    swap[i] = 0;
    if (ms_reference[i] >= 0.f && ms_selected[i] > 0.f && ms_reference[i] >= ms_selected[i])
      any_fast = true;
  }
  const bool go = n >= 2 && any_fast;
  if (triggered) *triggered = go ? 1 : 0;
  if (!go) return MK_OK;
  for (int32_t i = 0; i < n; ++i) {
    if (ms_reference[i] < 0.f || ms_selected[i] <= 0.f) continue;
    swap[i] = ms_reference[i] / ms_selected[i] < tau ? 1 : 0;
  }
  return MK_OK;
}

mk_status mk_budget_shares(int32_t n, const float* ms, const int32_t* needs_work,
                           float* shares) {
  if (n < 0 || (n > 0 && (!ms || !shares)))
    return fail(MK_E_INVALID_ARG, "mk_budget_shares: null array or n < 0");
  int32_t n_work = 0;
  double total = 0.0;
  for (int32_t i = 0; i < n; ++i) {
    if (needs_work && needs_work[i]) ++n_work;
    if (ms[i] < 0.f) return fail(MK_E_INVALID_ARG, "mk_budget_shares: negative time");
    total += ms[i];
  }
  for (int32_t i = 0; i < n; ++i) {
    if (n_work)
      shares[i] = needs_work[i] ? 1.0f / (float)n_work : 0.f;
    else
      shares[i] = total > 0.0 ? (float)(ms[i] / total) : 0.f;
  }
  return MK_OK;
}

mk_status mk_swap(mk_module* m, const void* const* dev_inputs, void* dev_out, void* dev_ws,
                  int64_t ws_bytes, void* stream, int32_t reference_impl, float tau,
                  int32_t n_runs, float* ms_selected, float* ms_reference, int32_t* swapped,
                  int32_t* triggered) {
  if (!m || n_runs < 1) return fail(MK_E_INVALID_ARG, "null module or n_runs < 1");
  try {
    mk::Plan& p = m->plan;
    const size_t ns = p.subs.size();
    std::vector<int32_t> sel(ns), has_ref(ns);
    for (size_t i = 0; i < ns; ++i) {
      sel[i] = p.subs[i].impl;
      has_ref[i] = mk::impl_exists(p, p.subs[i], reference_impl) ? 1 : 0;
    }
    // mean per-subkernel time over n_runs runs (after one warm-up)
    auto time_all = [&](std::vector<float>& mean) -> mk_status {
      std::vector<float> t(ns);
      mean.assign(ns, 0.f);
      for (int32_t r = 0; r <= n_runs; ++r) {
        mk_status s = mk_run(m, dev_inputs, dev_out, dev_ws, ws_bytes, stream, t.data());
        if (s != MK_OK) return s;
        if (r > 0)
          for (size_t i = 0; i < ns; ++i) mean[i] += t[i] / (float)n_runs;
      }
      return MK_OK;
    };
    std::vector<float> t_sel, t_ref;
    mk_status s = time_all(t_sel);
    if (s != MK_OK) return s;
    for (size_t i = 0; i < ns; ++i)
      if (has_ref[i]) p.subs[i].impl = reference_impl;
    s = time_all(t_ref);
    for (size_t i = 0; i < ns; ++i) p.subs[i].impl = sel[i];
    if (s != MK_OK) return s;
    for (size_t i = 0; i < ns; ++i)
      if (!has_ref[i]) t_ref[i] = -1.f;
    std::vector<int32_t> sw(ns);
    int32_t trig = 0;
    s = mk_swap_decide((int32_t)ns, t_sel.data(), t_ref.data(), tau, sw.data(), &trig);
    if (s != MK_OK) return s;
    for (size_t i = 0; i < ns; ++i) {
      if (sw[i]) p.subs[i].impl = reference_impl;
      if (ms_selected) ms_selected[i] = t_sel[i];
      if (ms_reference) ms_reference[i] = t_ref[i];
      if (swapped) swapped[i] = sw[i];
    }
    if (triggered) *triggered = trig;
    return MK_OK;
  } catch (...) {
    return fail(MK_E_INTERNAL, "exception in mk_swap");
  }
}

mk_status mk_profile_begin(mk_module* m, int32_t max_launches, int32_t only_launch) {
  if (!m || max_launches < 1) return fail(MK_E_INVALID_ARG, "null module or max_launches < 1");
  if (m->profiling) return fail(MK_E_INVALID_ARG, "a profile is already open");
  int32_t per_run = 0;
  for (const mk::Subkernel& s : m->plan.subs) per_run += mk::impl_launches(m->plan, s, s.impl);
  if (only_launch < -1 || only_launch >= per_run)
    return fail(MK_E_INVALID_ARG, "only_launch out of range");
  for (hipEvent_t e : m->prof) (void)hipEventDestroy(e);
  m->prof.assign(2 * (size_t)max_launches, nullptr);
  for (auto& e : m->prof) {
    // timing only: no system-scope fence (cache write-back) at each record
    hipError_t r = hipEventCreateWithFlags(&e, hipEventDisableSystemFence);
    if (r != hipSuccess) {
      e = nullptr;
      return hip_fail(r, "hipEventCreate");
    }
  }
  m->timer.events = &m->prof;
  m->timer.next = 0;
  m->timer.only = only_launch;
  m->timer.pos = 0;
  m->profiling = true;
  return MK_OK;
}

mk_status mk_profile_end(mk_module* m, float* launch_ms, int32_t capacity, int32_t* n_recorded) {
  if (!m || !n_recorded || (capacity > 0 && !launch_ms))
    return fail(MK_E_INVALID_ARG, "null argument");
  if (!m->profiling) return fail(MK_E_INVALID_ARG, "no profile is open");
  m->profiling = false;
  const int32_t n = (int32_t)(m->timer.next / 2);
  *n_recorded = n;
  if (n == 0) return MK_OK;
  hipError_t e = hipEventSynchronize(m->prof[2 * n - 1]);
  if (e != hipSuccess) return hip_fail(e, "hipEventSynchronize");
  for (int32_t i = 0; i < n && i < capacity; ++i) {
    e = hipEventElapsedTime(&launch_ms[i], m->prof[2 * i], m->prof[2 * i + 1]);
    if (e != hipSuccess) return hip_fail(e, "hipEventElapsedTime");
  }
  return MK_OK;
}

static double decode(int32_t dtype, const uint8_t* base, int64_t i) {
  if (dtype == MK_BF16) {
    uint16_t b;
    std::memcpy(&b, base + 2 * i, 2);
    uint32_t u = (uint32_t)b << 16;
    float f;
    std::memcpy(&f, &u, 4);
    return f;
  }
  float f;
  std::memcpy(&f, base + 4 * i, 4);
  return f;
}

mk_status mk_verify(mk_module* m, const void* const* dev_inputs, void* dev_out, void* dev_ws,
                    int64_t ws_bytes, void* stream, int32_t n_checks, const mk_check* checks,
                    mk_verify_report* rep) {
  if (!m || !rep) return fail(MK_E_INVALID_ARG, "null argument");
  if (n_checks < 0 || n_checks > MK_MAX_CHECKS || (n_checks > 0 && !checks))
    return fail(MK_E_INVALID_ARG, "checks");
  const mk::Plan& p = m->plan;
  for (int c = 0; c < n_checks; ++c) {
    const mk_check& k = checks[c];
    if (k.stage < 0 || k.stage >= (int32_t)p.subs.size() || k.n < 0 || (k.n > 0 && !k.expect))
      return fail(MK_E_INVALID_ARG, "check " + std::to_string(c));
  }
  try {
    std::vector<void*> vals;
    mk_status s = bind_values(m, dev_inputs, dev_out, dev_ws, ws_bytes, vals);
    if (s != MK_OK) return s;
    hipStream_t st = (hipStream_t)stream;
    const int64_t ws = ws_total(p);
    // NaN bytes in every intermediate and scratch byte and in the output: a
    // subkernel that reads something no earlier subkernel wrote produces NaN,
    // and output elements no kernel writes stay NaN (rather than holding an
    // earlier run's values).
    if (ws > 0) {
      hipError_t e = hipMemsetAsync(dev_ws, 0xFF, (size_t)ws, st);
      if (e != hipSuccess) return hip_fail(e, "hipMemsetAsync");
    }
    {
      const int64_t out_bytes = mk::numel(p.vshape.back()) * mk::elem_size(p.dtype);
      hipError_t e = hipMemsetAsync(dev_out, 0xFF, (size_t)out_bytes, st);
      if (e != hipSuccess) return hip_fail(e, "hipMemsetAsync");
    }
    s = mk_run(m, dev_inputs, dev_out, dev_ws, ws_bytes, stream, nullptr);
    if (s != MK_OK) return s;
    hipError_t e = hipStreamSynchronize(st);
    if (e != hipSuccess) return hip_fail(e, "hipStreamSynchronize");
    std::map<int, std::vector<uint8_t>> host;
    std::memset(rep, 0, sizeof(*rep));
    rep->pass = 1;
    rep->first_failing_stage = -1;
    rep->n_results = n_checks;
    const int64_t es = mk::elem_size(p.dtype);
    for (int c = 0; c < n_checks; ++c) {
      const mk_check& k = checks[c];
      const mk::Subkernel& sk = p.subs[k.stage];
      const int64_t n_el = mk::numel(p.vshape[sk.out_value]);
      auto it = host.find(k.stage);
      if (it == host.end()) {
        std::vector<uint8_t> buf((size_t)(n_el * es));
        e = hipMemcpy(buf.data(), vals[sk.out_value], buf.size(), hipMemcpyDeviceToHost);
        if (e != hipSuccess) return hip_fail(e, "hipMemcpy");
        it = host.emplace(k.stage, std::move(buf)).first;
      }
      const uint8_t* base = it->second.data();
      mk_check_result& r = rep->results[c];
      r.stage = k.stage;
      r.n_checked = k.n;
      r.worst_index = -1;
      for (int64_t j = 0; j < k.n; ++j) {
        const int64_t idx = k.index ? k.index[j] : j;
        if (idx < 0 || idx >= n_el) return fail(MK_E_INVALID_ARG, "check index out of range");
        const double g = decode(p.dtype, base, idx), x = k.expect[j];
        double ratio;
        bool bad;
        if (std::isinf(x)) {
          bad = g != x;
          ratio = bad ? INFINITY : 0.0;
        } else if (!std::isfinite(g) || std::isnan(x)) {
          bad = true;
          ratio = INFINITY;
          ++r.n_nonfinite;
        } else {
          const double err = std::fabs(g - x), tol = k.atol + k.rtol * std::fabs(x);
          bad = err > tol;
          ratio = tol > 0 ? err / tol : (err > 0 ? INFINITY : 0.0);
          if (err > r.max_abs_err) r.max_abs_err = err;
          if (x != 0 && err / std::fabs(x) > r.max_rel_err) r.max_rel_err = err / std::fabs(x);
        }
        if (bad) ++r.n_violations;
        if (ratio > r.worst_ratio || r.worst_index < 0) {
          r.worst_ratio = ratio;
          r.worst_index = idx;
          r.got_at_worst = g;
          r.expect_at_worst = x;
        }
      }
      r.pass = r.n_violations == 0;
      if (!r.pass) {
        rep->pass = 0;
        if (rep->first_failing_stage < 0 || k.stage < rep->first_failing_stage)
          rep->first_failing_stage = k.stage;
      }
    }
    return MK_OK;
  } catch (...) {
    return fail(MK_E_INTERNAL, "exception in mk_verify");
  }
}

}  // extern "C"
