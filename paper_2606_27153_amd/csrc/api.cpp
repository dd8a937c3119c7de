// C ABI of the Muon step library: argument checking, plan lifetime, device
// tables, and the per-step launch sequence.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <new>
#include <string>

#include "muon_internal.h"

struct muon_plan_s {
  muon::Plan p;
};

namespace {

thread_local std::string g_last_error;

muon_status fail(muon_status s, const std::string& msg) {
  g_last_error = msg;
  return s;
}

muon_status ok() {
  g_last_error.clear();
  return MUON_OK;
}

muon_status hip_fail(hipError_t e, const char* what) {
  return fail(MUON_ERR_DEVICE, std::string(what) + ": " + hipGetErrorString(e));
}

bool valid_dtype(int32_t d) { return d == MUON_F32 || d == MUON_BF16; }

muon_status check_opts(const muon_plan_opts& o) {
  if (o.precision != MUON_NS_BF16 && o.precision != MUON_NS_FP32 && o.precision != MUON_NS_FP16)
    return fail(MUON_ERR_INVALID_ARG, "opts.precision must be MUON_NS_BF16, MUON_NS_FP32 or MUON_NS_FP16");
  if (o.max_ns_steps < 1 || o.max_ns_steps > 64)
    return fail(MUON_ERR_INVALID_ARG, "opts.max_ns_steps must be in [1, 64]");
  if (!std::isfinite(o.a) || !std::isfinite(o.b) || !std::isfinite(o.c))
    return fail(MUON_ERR_INVALID_ARG, "opts.a, opts.b, opts.c must be finite");
  if (o.c != 0.f && !std::isfinite(o.b / o.c))
    return fail(MUON_ERR_INVALID_ARG, "opts.c must be 0 or large enough that b / c is finite in fp32");
  if (o.abc_per_step && o.max_ns_steps >= 1 && o.max_ns_steps <= 64) {
    for (int32_t i = 0; i < o.max_ns_steps; ++i) {
      const float a = o.abc_per_step[3 * i], b = o.abc_per_step[3 * i + 1], c = o.abc_per_step[3 * i + 2];
      const std::string at = "opts.abc_per_step step " + std::to_string(i);
      if (!std::isfinite(a) || !std::isfinite(b) || !std::isfinite(c))
        return fail(MUON_ERR_INVALID_ARG, at + ": a, b, c must be finite");
      if (c != 0.f && !std::isfinite(b / c))
        return fail(MUON_ERR_INVALID_ARG, at + ": c must be 0 or large enough that b / c is finite in fp32");
    }
  }
  if (!std::isfinite(o.eps) || o.eps < 0.f) return fail(MUON_ERR_INVALID_ARG, "opts.eps must be finite and >= 0");
  if (o.small_m_threshold < 0) return fail(MUON_ERR_INVALID_ARG, "opts.small_m_threshold must be >= 0");
  if (o.flags & ~uint32_t(MUON_PLAN_HOST_ONLY | MUON_PLAN_CHECK_BUFFERS))
    return fail(MUON_ERR_INVALID_ARG, "opts.flags has unknown bits");
  if (o.wave_bytes < 0) return fail(MUON_ERR_INVALID_ARG, "opts.wave_bytes must be >= 0");
  if (!std::isfinite(o.gram_min_aspect) || (o.gram_min_aspect != 0.f && o.gram_min_aspect < 1.f))
    return fail(MUON_ERR_INVALID_ARG, "opts.gram_min_aspect must be 0 or a finite value >= 1");
  if (o.gram_restart < 0) return fail(MUON_ERR_INVALID_ARG, "opts.gram_restart must be >= 0");
  return MUON_OK;
}

muon_status upload_tables(muon::Plan& p) {
  using namespace muon;
  auto al = [](size_t v) { return (v + 255) / 256 * 256; };
  const size_t b_mats = al(p.h_matdev.size() * sizeof(MatDev));
  const size_t b_pref = al(p.h_prefix.size() * sizeof(int32_t));
  const size_t b_tiles = al(p.h_tiles.size() * sizeof(TileEntry));
  const size_t b_ptrs = al(p.mats.size() * sizeof(PtrEntry));
  const size_t total = b_mats + b_pref + b_tiles + b_ptrs;
  hipError_t e = hipMalloc(&p.d_block, total);
  if (e != hipSuccess) {
    p.d_block = nullptr;
    return e == hipErrorOutOfMemory ? fail(MUON_ERR_OUT_OF_MEMORY, "hipMalloc of plan tables failed")
                                    : hip_fail(e, "hipMalloc of plan tables");
  }
  char* base = static_cast<char*>(p.d_block);
  p.d_mats = reinterpret_cast<MatDev*>(base);
  p.d_prefix = reinterpret_cast<int32_t*>(base + b_mats);
  p.d_tiles = reinterpret_cast<TileEntry*>(base + b_mats + b_pref);
  p.d_ptrs = reinterpret_cast<PtrEntry*>(base + b_mats + b_pref + b_tiles);
  e = hipMemcpy(p.d_mats, p.h_matdev.data(), p.h_matdev.size() * sizeof(MatDev), hipMemcpyHostToDevice);
  if (e == hipSuccess)
    e = hipMemcpy(p.d_prefix, p.h_prefix.data(), p.h_prefix.size() * sizeof(int32_t), hipMemcpyHostToDevice);
  if (e == hipSuccess && !p.h_tiles.empty())
    e = hipMemcpy(p.d_tiles, p.h_tiles.data(), p.h_tiles.size() * sizeof(TileEntry), hipMemcpyHostToDevice);
  if (e != hipSuccess) return hip_fail(e, "upload of plan tables");
  // the pinned ring the step refreshes the pointer table from
  e = hipHostMalloc(reinterpret_cast<void**>(&p.h_ring), size_t(Plan::kRing) * p.mats.size() * sizeof(PtrEntry),
                    hipHostMallocDefault);
  if (e != hipSuccess) {
    p.h_ring = nullptr;
    return e == hipErrorOutOfMemory ? fail(MUON_ERR_OUT_OF_MEMORY, "hipHostMalloc of the pointer ring failed")
                                    : hip_fail(e, "hipHostMalloc of the pointer ring");
  }
  for (int k = 0; k < Plan::kRing; ++k) {
    hipEvent_t ev = nullptr;
    e = hipEventCreateWithFlags(&ev, hipEventDisableTiming);
    if (e != hipSuccess) return hip_fail(e, "hipEventCreateWithFlags");
    p.ring_events[k] = ev;
  }
  return MUON_OK;
}

// Frees what upload_tables allocated (each part only if it exists).
hipError_t release_device(muon::Plan& p) {
  hipError_t first = hipSuccess;
  auto keep = [&](hipError_t e) {
    if (first == hipSuccess) first = e;
  };
  for (int k = 0; k < muon::Plan::kRing; ++k) {
    if (p.ring_events[k]) keep(hipEventDestroy(hipEvent_t(p.ring_events[k])));
    p.ring_events[k] = nullptr;
  }
  if (p.h_ring) keep(hipHostFree(p.h_ring));
  p.h_ring = nullptr;
  if (p.d_block) keep(hipFree(p.d_block));
  p.d_block = nullptr;
  return first;
}

bool aligned(const void* ptr, uintptr_t a) { return (reinterpret_cast<uintptr_t>(ptr) & (a - 1)) == 0; }

// [ptr, ptr + bytes) must be device memory of the plan's device (or managed
// memory) inside one allocation -- the latter where HIP can name the
// allocation (memory mapped through the virtual memory API may not be
// reported; it is then taken on trust).  A failed HIP query leaves its error
// behind, so it is cleared before returning.
muon_status check_memory(const void* ptr, size_t bytes, int device, const std::string& what) {
  hipPointerAttribute_t a;
  std::memset(&a, 0, sizeof(a));
  hipError_t e = hipPointerGetAttributes(&a, ptr);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return fail(MUON_ERR_INVALID_ARG, what + " is not memory the HIP runtime knows (a host pointer?)");
  }
  if (a.type != hipMemoryTypeDevice && a.type != hipMemoryTypeManaged)
    return fail(MUON_ERR_INVALID_ARG, what + " is not device memory");
  if (a.type == hipMemoryTypeDevice && a.device != device)
    return fail(MUON_ERR_INVALID_ARG,
                what + " is on device " + std::to_string(a.device) + ", the plan on device " + std::to_string(device));
  hipDeviceptr_t base = nullptr;
  size_t size = 0;
  e = hipMemGetAddressRange(&base, &size, hipDeviceptr_t(const_cast<void*>(ptr)));
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return MUON_OK;
  }
  const uintptr_t end = uintptr_t(ptr) + bytes, aend = uintptr_t(base) + size;
  if (uintptr_t(ptr) < uintptr_t(base) || end > aend)
    return fail(MUON_ERR_INVALID_ARG, what + " needs " + std::to_string(bytes) + " bytes, its allocation ends " +
                                          std::to_string(aend > uintptr_t(ptr) ? aend - uintptr_t(ptr) : 0) +
                                          " bytes after it");
  return MUON_OK;
}

// The buffer checks of a step: non-NULL (a NULL gradient skips its matrix),
// aligned, the workspace large enough, the current device the plan's; with
// `memory`, also where each buffer lives (check_memory) -- muon_check_buffers
// always, muon_step when its buffer addresses change on a plan created with
// MUON_PLAN_CHECK_BUFFERS.
muon_status check_buffers(const muon::Plan& p, void* const* params, const void* const* grads,
                          void* const* momentum, const void* workspace, size_t workspace_bytes,
                          float* const* update_out, bool memory, bool own_ws = false) {
  if (!params || !grads || !momentum) return fail(MUON_ERR_INVALID_ARG, "params, grads and momentum must be non-NULL");
  if (!workspace) return fail(MUON_ERR_INVALID_ARG, "workspace is NULL");
  if (!aligned(workspace, 256)) return fail(MUON_ERR_INVALID_ARG, "workspace must be 256-byte aligned");
  if (workspace_bytes < size_t(p.ws_bytes))
    return fail(MUON_ERR_WORKSPACE_TOO_SMALL,
                "workspace has " + std::to_string(workspace_bytes) + " bytes, plan needs " + std::to_string(p.ws_bytes));
  const size_t n = p.mats.size();
  for (size_t i = 0; i < n; ++i) {
    if (!params[i] || !momentum[i])
      return fail(MUON_ERR_INVALID_ARG, "NULL param or momentum pointer for matrix " + std::to_string(i));
    if (!aligned(params[i], 16) || !aligned(grads[i], 16) || !aligned(momentum[i], 16) ||
        (update_out && update_out[i] && !aligned(update_out[i], 16)))
      return fail(MUON_ERR_INVALID_ARG, "buffers of matrix " + std::to_string(i) + " must be 16-byte aligned");
  }
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev != p.device)
    return fail(MUON_ERR_INVALID_ARG, "current device " + std::to_string(dev) + " is not the plan's device " +
                                          std::to_string(p.device));
  if (!memory) return MUON_OK;
  // (the library's own static workspace needs no vetting)
  muon_status st = own_ws ? MUON_OK : check_memory(workspace, size_t(p.ws_bytes), dev, "the workspace");
  for (size_t i = 0; i < n && st == MUON_OK; ++i) {
    const muon::MatHost& h = p.mats[i];
    const size_t el = size_t(h.rows) * size_t(h.cols);
    const std::string at = "matrix " + std::to_string(i) + " ";
    st = check_memory(params[i], el * (h.param_dtype == MUON_BF16 ? 2 : 4), dev, at + "param");
    if (st == MUON_OK && grads[i])
      st = check_memory(grads[i], el * (h.grad_dtype == MUON_BF16 ? 2 : 4), dev, at + "grad");
    if (st == MUON_OK) st = check_memory(momentum[i], el * 4, dev, at + "momentum");
    if (st == MUON_OK && update_out && update_out[i]) st = check_memory(update_out[i], el * 4, dev, at + "update_out");
  }
  return st;
}

// One step.  `own_ws`: the workspace is the library's static one (it needs
// no vetting, and the step records no timing events, which would allocate).
muon_status step_impl(muon_plan plan, void* const* params, const void* const* grads, void* const* momentum,
                      float lr, float mu, float wd, int32_t ns_steps, int32_t nesterov, void* workspace,
                      size_t workspace_bytes, void* stream, float* const* update_out, bool own_ws = false) {
  using namespace muon;
  if (!plan) return fail(MUON_ERR_INVALID_ARG, "plan is NULL");
  Plan& p = plan->p;
  if (!p.d_block) return fail(MUON_ERR_INVALID_ARG, "plan was created host-only and cannot be stepped");
  if (!std::isfinite(lr) || lr < 0.f) return fail(MUON_ERR_INVALID_ARG, "lr must be finite and >= 0");
  if (!std::isfinite(wd) || wd < 0.f) return fail(MUON_ERR_INVALID_ARG, "weight_decay must be finite and >= 0");
  if (!(mu >= 0.f && mu < 1.f)) return fail(MUON_ERR_INVALID_ARG, "momentum_coef must be in [0, 1)");
  if (ns_steps < 0 || ns_steps > p.opts.max_ns_steps)
    return fail(MUON_ERR_INVALID_ARG, "ns_steps must be in [0, max_ns_steps]");
  if (nesterov != 0 && nesterov != 1) return fail(MUON_ERR_INVALID_ARG, "nesterov must be 0 or 1");
  muon_status st = check_buffers(p, params, grads, momentum, workspace, workspace_bytes, update_out, false);
  if (st != MUON_OK) return st;
  const size_t n = p.mats.size();
  const bool timing = p.timing && !own_ws;

  // Refresh the device pointer table if the caller's buffers moved: the new
  // table goes into the next slot of the plan's pinned ring and is copied on
  // the caller's stream, ahead of the step's kernels.  The host waits only if
  // that slot's previous copy (kRing refreshes ago) has not run yet.  The
  // workspace's memory is vetted when it changes (two HIP queries); the other
  // buffers' only on plans created with MUON_PLAN_CHECK_BUFFERS.
  bool changed = !p.ptrs_valid;
  for (size_t i = 0; i < n && !changed; ++i) {
    const PtrEntry& h = p.h_ptrs[i];
    float* out = update_out ? update_out[i] : nullptr;
    changed = h.param != params[i] || h.grad != grads[i] || h.mom != momentum[i] || h.out != out;
  }
  if (changed && (p.opts.flags & MUON_PLAN_CHECK_BUFFERS)) {
    st = check_buffers(p, params, grads, momentum, workspace, workspace_bytes, update_out, true, own_ws);
    if (st != MUON_OK) return st;
    if (!own_ws) p.ws_checked = workspace;
  }
  if (workspace != p.ws_checked && !own_ws) {
    st = check_memory(workspace, size_t(p.ws_bytes), p.device, "the workspace");
    if (st != MUON_OK) return st;
    p.ws_checked = workspace;
  }
  hipError_t e = hipSuccess;
  hipStream_t hs = hipStream_t(stream);
  if (changed) {
    hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
    if (hipStreamIsCapturing(hs, &cs) != hipSuccess) {
      (void)hipGetLastError();
      cs = hipStreamCaptureStatusNone;
    }
    if (cs != hipStreamCaptureStatusNone)
      return fail(MUON_ERR_INVALID_ARG,
                  "buffer addresses differ from the previous step's while the stream is being captured; "
                  "step once on these buffers before the capture");
    const int k = p.ring_next;
    if (p.ring_busy[k]) {
      e = hipEventSynchronize(hipEvent_t(p.ring_events[k]));
      if (e != hipSuccess) return hip_fail(e, "waiting for a pointer-ring slot");
    }
    PtrEntry* slot = p.h_ring + size_t(k) * n;
    for (size_t i = 0; i < n; ++i) {
      slot[i] = PtrEntry{params[i], grads[i], static_cast<float*>(momentum[i]), update_out ? update_out[i] : nullptr};
      p.h_ptrs[i] = slot[i];
    }
    p.ptrs_valid = false;
    e = hipMemcpyAsync(p.d_ptrs, slot, n * sizeof(PtrEntry), hipMemcpyHostToDevice, hs);
    if (e == hipSuccess) e = hipEventRecord(hipEvent_t(p.ring_events[k]), hs);
    if (e != hipSuccess) return hip_fail(e, "upload of buffer pointers");
    p.ring_busy[k] = true;
    p.ring_next = (k + 1) % Plan::kRing;
    p.ptrs_valid = true;
  }

  StepScalars s{};
  s.lr = lr;
  s.mu = mu;
  s.wd = wd;
  s.decay = float(1.0 - double(lr) * double(wd));
  s.eps = p.opts.eps;
  s.nesterov = nesterov;
  s.ns_steps = ns_steps;
  char* ws = static_cast<char*>(workspace);
  // Runs one launch, bracketed by timing events when timing is enabled.
  auto run = [&](int32_t kind, int32_t kclass, double flops, double bytes, auto&& launch) -> hipError_t {
    size_t ev = 0;
    if (timing) {
      ev = p.records.size() * 2;
      while (p.events.size() < ev + 2) {
        hipEvent_t e;
        hipError_t er = hipEventCreate(&e);
        if (er != hipSuccess) return er;
        p.events.push_back(e);
      }
      hipError_t er = hipEventRecord(hipEvent_t(p.events[ev]), hs);
      if (er != hipSuccess) return er;
    }
    if (launch()) {
      hipError_t er = hipGetLastError();
      return er == hipSuccess ? hipErrorLaunchFailure : er;
    }
    if (timing) {
      hipError_t er = hipEventRecord(hipEvent_t(p.events[ev + 1]), hs);
      if (er != hipSuccess) return er;
      p.records.push_back(TimingRecord{kind, kclass, flops, bytes, ev});
    }
    return hipSuccess;
  };
  for (const WaveHost& w : p.waves) {
    e = run(MUON_KERNEL_MOMENTUM, -1, 0.0, w.bytes_momentum, [&] { return launch_momentum(p, w, ws, s, stream); });
    if (e != hipSuccess) return hip_fail(e, "momentum kernel launch");
    e = run(MUON_KERNEL_FINALIZE, -1, 0.0, 0.0, [&] { return launch_finalize(p, w, ws, s, stream); });
    if (e != hipSuccess) return hip_fail(e, "finalize kernel launch");
    auto gemm = [&](const ClassLaunch& cl, int32_t stage, int32_t kind, const GemmStep& g) {
      const double fl = (kind == MUON_KERNEL_GRAM ? cl.flops_gram : kind == MUON_KERNEL_BX ? cl.flops_bx : cl.flops_poly) *
                        (g.pair ? 2.0 : 1.0);
      return run(kind, cl.kclass, fl, 0.0, [&] { return launch_ns_gemm(p, w, cl, stage, g, ws, s, stream); });
    };
    // Eq. 2: per step A = s^2 X X^T, B = b A + c A A, X' = s (a X + B X),
    // with step it's (a, b, c).  With c = 0 (a cubic step) the Gram stage
    // writes B = b A itself.
    for (int32_t it = 0; it < ns_steps; ++it) {
      const int32_t first = it == 0, pin = it & 1, last = it == ns_steps - 1;
      const float a = p.abc[size_t(3 * it)], b = p.abc[size_t(3 * it + 1)], c = p.abc[size_t(3 * it + 2)];
      const bool cubic = c == 0.f;
      for (const ClassLaunch& cl : w.launches) {
        if (cl.gram) continue;
        e = gemm(cl, ST_GRAM, MUON_KERNEL_GRAM,
                 GemmStep{first, pin, last, SQ_A, SQ_A, cubic ? SQ_B : SQ_A, 0.f, 0.f, cubic ? b : 1.f});
        if (e != hipSuccess) return hip_fail(e, "NS GEMM launch");
      }
      if (!cubic)
        for (const ClassLaunch& cl : w.launches) {
          if (cl.gram) continue;
          e = gemm(cl, ST_POLY, MUON_KERNEL_POLY, GemmStep{first, pin, last, SQ_A, SQ_A, SQ_B, b / c, 0.f, c});
          if (e != hipSuccess) return hip_fail(e, "NS GEMM launch");
        }
      for (const ClassLaunch& cl : w.launches) {
        if (cl.gram) continue;
        e = gemm(cl, ST_BX, MUON_KERNEL_BX, GemmStep{first, pin, last, SQ_B, SQ_B, SQ_B, a, 0.f, 1.f});
        if (e != hipSuccess) return hip_fail(e, "NS GEMM launch");
      }
    }
    // Gram space (Eq. 4), in segments of at most gram_restart steps.  A
    // segment starting from X (X0 = s u in the first) forms G = X X^T; per
    // step P_i = a_i I + b_i G + c_i G^2 (as c_i (G G + b_i/c_i G + a_i/c_i
    // I); the plan takes this form only when no c_i is 0); Q_{i+1} = P_i Q_i
    // (the segment's first P is written straight into Q0); R = G P_i and
    // G <- P_i R except after the segment's last step; then X <- Q X, which
    // after the last segment is O and goes into the update.  P Q and G P
    // only need P_i, so they share one launch.  In segments of at most two
    // steps R lives in B's memory and the second Q in A's (gram_shares_buffers):
    // this order writes each only after the last read of what it replaces.
    for (const ClassLaunch& cl : w.launches) {
      if (!cl.gram) continue;
      int32_t pin = 0;
      for (int32_t s0 = 0; s0 < ns_steps; s0 += p.gram_restart) {
        const int32_t len = std::min(p.gram_restart, ns_steps - s0);
        const int32_t first = s0 == 0, last = s0 + len == ns_steps;
        e = gemm(cl, ST_GRAM, MUON_KERNEL_GRAM, GemmStep{first, pin, 0, SQ_A, SQ_A, SQ_A, 0.f, 0.f, 1.f});
        if (e != hipSuccess) return hip_fail(e, "NS GEMM launch");
        for (int32_t j = 0; j < len; ++j) {
          const int32_t it = s0 + j;
          const int32_t pbuf = j == 0 ? SQ_Q0 : SQ_B;
          const float a = p.abc[size_t(3 * it)], b = p.abc[size_t(3 * it + 1)], c = p.abc[size_t(3 * it + 2)];
          e = gemm(cl, ST_POLY, MUON_KERNEL_POLY, GemmStep{0, 0, 0, SQ_A, SQ_A, pbuf, b / c, a / c, c});
          const GemmStep qu{0, 0, 0, SQ_B, (j - 1) & 1 ? SQ_Q1 : SQ_Q0, j & 1 ? SQ_Q1 : SQ_Q0, 0.f, 0.f, 1.f};
          GemmStep gr{0, 0, 0, SQ_A, pbuf, SQ_R, 0.f, 0.f, 1.f};
          const bool need_qu = j > 0, need_gr = j + 1 < len;
          if (e == hipSuccess && need_qu && need_gr) {
            gr.pair = 1;
            gr.l2 = qu.l;
            gr.r2 = qu.r;
            gr.out2 = qu.out;
            e = gemm(cl, ST_SYM, MUON_KERNEL_SYMM, gr);
          } else if (e == hipSuccess && (need_qu || need_gr)) {
            e = gemm(cl, ST_SYM, MUON_KERNEL_SYMM, need_qu ? qu : gr);
          }
          if (e == hipSuccess && need_gr)
            e = gemm(cl, ST_SYM, MUON_KERNEL_SYMM, GemmStep{0, 0, 0, pbuf, SQ_R, SQ_A, 0.f, 0.f, 1.f});
          if (e != hipSuccess) return hip_fail(e, "NS GEMM launch");
        }
        const int32_t qk = (len - 1) & 1 ? SQ_Q1 : SQ_Q0;
        e = gemm(cl, ST_BX, MUON_KERNEL_BX, GemmStep{first, pin, last, qk, qk, qk, 0.f, 0.f, 1.f});
        if (e != hipSuccess) return hip_fail(e, "NS GEMM launch");
        pin ^= 1;
      }
    }
    // With k >= 1 the last B*X launch applied the update (zero-gradient
    // matrices included); with k = 0 the update is O = s*u.
    if (ns_steps == 0) {
      e = run(MUON_KERNEL_APPLY, -1, 0.0, w.bytes_apply, [&] { return launch_apply(p, w, ws, s, stream); });
      if (e != hipSuccess) return hip_fail(e, "apply kernel launch");
    }
  }
  return ok();
}

void release_events(muon::Plan& p) {
  for (void* e : p.events) (void)hipEventDestroy(hipEvent_t(e));
  p.events.clear();
  p.records.clear();
}

}  // namespace

extern "C" {

int32_t muon_abi_version(void) { return MUON_ABI_VERSION; }

const char* muon_status_string(muon_status s) {
  switch (s) {
    case MUON_OK: return "MUON_OK";
    case MUON_ERR_INVALID_ARG: return "MUON_ERR_INVALID_ARG";
    case MUON_ERR_UNSUPPORTED: return "MUON_ERR_UNSUPPORTED";
    case MUON_ERR_OUT_OF_MEMORY: return "MUON_ERR_OUT_OF_MEMORY";
    case MUON_ERR_WORKSPACE_TOO_SMALL: return "MUON_ERR_WORKSPACE_TOO_SMALL";
    case MUON_ERR_DEVICE: return "MUON_ERR_DEVICE";
  }
  return "MUON_ERR_UNKNOWN";
}

const char* muon_last_error(void) { return g_last_error.c_str(); }

muon_status muon_plan_opts_default(muon_plan_opts* o) {
  if (!o) return fail(MUON_ERR_INVALID_ARG, "opts is NULL");
  std::memset(o, 0, sizeof(*o));
  o->precision = MUON_NS_BF16;
  o->max_ns_steps = 16;
  o->a = 3.4445f;
  o->b = -4.7750f;
  o->c = 2.0315f;
  o->eps = 1e-7f;
  o->small_m_threshold = 64;
  o->flags = 0;
  o->wave_bytes = 0;
  o->gram_min_aspect = 1.4f;
  o->gram_restart = 0;
  o->abc_per_step = nullptr;
  return ok();
}

muon_status muon_plan_create(const muon_matrix_desc* mats, int32_t n, const muon_plan_opts* opts, muon_plan* out) {
  if (!out) return fail(MUON_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  if (!mats) return fail(MUON_ERR_INVALID_ARG, "mats is NULL");
  if (n < 1) return fail(MUON_ERR_INVALID_ARG, "n must be >= 1");
  muon_plan_opts o;
  if (opts) {
    o = *opts;
  } else {
    muon_plan_opts_default(&o);
  }
  if (muon_status st = check_opts(o)) return st;
  for (int32_t i = 0; i < n; ++i) {
    const muon_matrix_desc& d = mats[i];
    const std::string who = "matrix " + std::to_string(i);
    if (d.rows < 1 || d.cols < 1 || d.rows >= (int64_t(1) << 31) || d.cols >= (int64_t(1) << 31))
      return fail(MUON_ERR_INVALID_ARG, who + ": rows and cols must be in [1, 2^31)");
    if (d.tile_hint != 0 && d.tile_hint != 64 && d.tile_hint != 128 && d.tile_hint != 256)
      return fail(MUON_ERR_INVALID_ARG, who + ": tile_hint must be 0, 64, 128 or 256");
    if (!valid_dtype(d.param_dtype) || !valid_dtype(d.grad_dtype))
      return fail(MUON_ERR_UNSUPPORTED, who + ": param and grad dtypes must be MUON_F32 or MUON_BF16");
    if (d.momentum_dtype != MUON_F32) return fail(MUON_ERR_UNSUPPORTED, who + ": momentum must be MUON_F32");
  }
  muon_plan_s* plan = new (std::nothrow) muon_plan_s();
  if (!plan) return fail(MUON_ERR_OUT_OF_MEMORY, "host allocation of the plan failed");
  std::string err;
  muon_status st;
  try {
    st = muon::build_plan(mats, n, o, plan->p, err);
  } catch (const std::bad_alloc&) {
    st = MUON_ERR_OUT_OF_MEMORY;
    err = "host allocation failed while building the plan";
  }
  if (st != MUON_OK) {
    delete plan;
    return fail(st, err);
  }
  if (!(o.flags & MUON_PLAN_HOST_ONLY)) {
    hipError_t e = hipGetDevice(&plan->p.device);
    if (e != hipSuccess) {
      delete plan;
      return hip_fail(e, "hipGetDevice");
    }
    st = upload_tables(plan->p);
    if (st != MUON_OK) {
      const std::string msg = g_last_error;
      (void)release_device(plan->p);
      delete plan;
      return fail(st, msg);
    }
    // the address of this device's static workspace (muon_step_static)
    plan->p.static_ws_status = muon::static_workspace_init(plan->p.device, &plan->p.static_ws);
    if (plan->p.static_ws_status != hipSuccess) {
      (void)hipGetLastError();
      plan->p.static_ws = nullptr;
    }
  }
  *out = plan;
  return ok();
}

muon_status muon_plan_destroy(muon_plan plan) {
  if (!plan) return ok();
  muon_status st = MUON_OK;
  release_events(plan->p);
  const hipError_t e = release_device(plan->p);
  if (e != hipSuccess) st = hip_fail(e, "releasing the plan's device tables");
  delete plan;
  return st == MUON_OK ? ok() : st;
}

muon_status muon_plan_workspace_bytes(muon_plan plan, size_t* bytes) {
  if (!plan || !bytes) return fail(MUON_ERR_INVALID_ARG, "plan and bytes must be non-NULL");
  *bytes = size_t(plan->p.ws_bytes);
  return ok();
}

muon_status muon_plan_get_info(muon_plan plan, muon_plan_info* info) {
  if (!plan || !info) return fail(MUON_ERR_INVALID_ARG, "plan and info must be non-NULL");
  const muon::Plan& p = plan->p;
  std::memset(info, 0, sizeof(*info));
  info->n_matrices = int32_t(p.mats.size());
  info->n_waves = int32_t(p.waves.size());
  info->n_buckets = p.n_buckets;
  info->device = p.d_block ? p.device : -1;
  info->workspace_bytes = p.ws_bytes;
  info->launches_per_step = muon::launches_per_step(p, p.opts.max_ns_steps);
  info->ns_flops_per_ns_step = p.ns_flops;
  info->padded_flops_per_ns_step = p.padded_flops;
  info->n_gram = p.n_gram;
  info->gram_restart = p.gram_restart;
  return ok();
}

muon_status muon_plan_ns_flops(muon_plan plan, int32_t ns_steps, double* flops) {
  if (!plan || !flops) return fail(MUON_ERR_INVALID_ARG, "plan and flops must be non-NULL");
  if (ns_steps < 0 || ns_steps > plan->p.opts.max_ns_steps)
    return fail(MUON_ERR_INVALID_ARG, "ns_steps must be in [0, max_ns_steps]");
  *flops = muon::plan_ns_flops(plan->p, ns_steps);
  return ok();
}

muon_status muon_plan_matrix_info(muon_plan plan, int32_t index, muon_matrix_info* info) {
  if (!plan || !info) return fail(MUON_ERR_INVALID_ARG, "plan and info must be non-NULL");
  const muon::Plan& p = plan->p;
  if (index < 0 || size_t(index) >= p.mats.size()) return fail(MUON_ERR_INVALID_ARG, "index out of range");
  const muon::MatHost& h = p.mats[size_t(index)];
  std::memset(info, 0, sizeof(*info));
  info->m = h.m;
  info->n = h.n;
  info->m_pad = h.m_pad;
  info->n_pad = h.n_pad;
  info->transposed = h.transposed;
  info->kernel_class = h.kclass;
  info->tile = muon::class_info(h.kclass).tile;
  info->fp32_ns = h.fp32_ns;
  info->wave = h.wave;
  info->bucket = h.bucket;
  info->gram_space = h.gram;
  return ok();
}

muon_status muon_plan_set_timing(muon_plan plan, int32_t enable) {
  if (!plan) return fail(MUON_ERR_INVALID_ARG, "plan is NULL");
  if (!plan->p.d_block) return fail(MUON_ERR_INVALID_ARG, "plan was created host-only");
  plan->p.timing = enable != 0;
  return ok();
}

muon_status muon_plan_timing_read(muon_plan plan, muon_kernel_stat* stats, int32_t capacity, int32_t* count,
                                  int32_t reset) {
  if (!plan || !count || (capacity > 0 && !stats) || capacity < 0)
    return fail(MUON_ERR_INVALID_ARG, "plan, count (and stats when capacity > 0) must be non-NULL");
  muon::Plan& p = plan->p;
  std::vector<muon_kernel_stat> agg;
  for (const muon::TimingRecord& r : p.records) {
    hipEvent_t e0 = hipEvent_t(p.events[r.event]), e1 = hipEvent_t(p.events[r.event + 1]);
    hipError_t e = hipEventSynchronize(e1);
    float ms = 0.f;
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, e0, e1);
    if (e != hipSuccess) return hip_fail(e, "reading timing events");
    muon_kernel_stat* st = nullptr;
    for (auto& a : agg)
      if (a.kind == r.kind && a.kernel_class == r.kclass) st = &a;
    if (!st) {
      agg.push_back(muon_kernel_stat{r.kind, r.kclass, 0, 0.0, 0.0, 0.0});
      st = &agg.back();
    }
    st->launches += 1;
    st->total_ms += double(ms);
    st->algo_flops += r.flops;
    st->algo_bytes += r.bytes;
  }
  *count = int32_t(agg.size());
  for (int32_t i = 0; i < capacity && size_t(i) < agg.size(); ++i) stats[i] = agg[size_t(i)];
  if (reset) p.records.clear();
  return ok();
}

muon_status muon_step(muon_plan plan, void* const* params, const void* const* grads, void* const* momentum,
                      float lr, float momentum_coef, float weight_decay, int32_t ns_steps, int32_t nesterov,
                      void* workspace, size_t workspace_bytes, void* hip_stream) {
  return step_impl(plan, params, grads, momentum, lr, momentum_coef, weight_decay, ns_steps, nesterov, workspace,
                   workspace_bytes, hip_stream, nullptr);
}

muon_status muon_check_buffers(muon_plan plan, void* const* params, const void* const* grads, void* const* momentum,
                               void* workspace, size_t workspace_bytes, float* const* update_out) {
  if (!plan) return fail(MUON_ERR_INVALID_ARG, "plan is NULL");
  if (!plan->p.d_block) return fail(MUON_ERR_INVALID_ARG, "plan was created host-only and cannot be stepped");
  const muon_status st = check_buffers(plan->p, params, grads, momentum, workspace, workspace_bytes, update_out, true);
  return st == MUON_OK ? ok() : st;
}

muon_status muon_step_static(muon_plan plan, void* const* params, const void* const* grads, void* const* momentum,
                             float lr, float momentum_coef, float weight_decay, int32_t ns_steps, int32_t nesterov,
                             void* hip_stream) {
  static_assert(muon::kStaticWorkspaceBytes == size_t(MUON_STATIC_WORKSPACE_BYTES), "static workspace size");
  if (!plan) return fail(MUON_ERR_INVALID_ARG, "plan is NULL");
  muon::Plan& p = plan->p;
  if (!p.d_block) return fail(MUON_ERR_INVALID_ARG, "plan was created host-only and cannot be stepped");
  if (size_t(p.ws_bytes) > muon::kStaticWorkspaceBytes)
    return fail(MUON_ERR_WORKSPACE_TOO_SMALL,
                "plan needs " + std::to_string(p.ws_bytes) + " bytes of workspace, the static workspace holds " +
                    std::to_string(muon::kStaticWorkspaceBytes) + " (use muon_step with a caller workspace)");
  if (!p.static_ws)
    return fail(MUON_ERR_DEVICE, std::string("the static workspace of device ") + std::to_string(p.device) +
                                     " could not be located: " + hipGetErrorString(hipError_t(p.static_ws_status)));
  return step_impl(plan, params, grads, momentum, lr, momentum_coef, weight_decay, ns_steps, nesterov, p.static_ws,
                   muon::kStaticWorkspaceBytes, hip_stream, nullptr, true);
}

muon_status muon_step_debug(muon_plan plan, void* const* params, const void* const* grads, void* const* momentum,
                            float lr, float momentum_coef, float weight_decay, int32_t ns_steps, int32_t nesterov,
                            void* workspace, size_t workspace_bytes, void* hip_stream, float* const* update_out) {
  return step_impl(plan, params, grads, momentum, lr, momentum_coef, weight_decay, ns_steps, nesterov, workspace,
                   workspace_bytes, hip_stream, update_out);
}

}  // extern "C"
