// C ABI of the DTST library: plans, validation and the execute calls.
//
// Every execute call validates its arguments on the host first; on any
// error it launches nothing, leaves the outputs untouched and records a
// message retrievable with dtst_last_error() on the calling thread.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <unordered_set>
#include <vector>

#include "dtst_internal.h"

struct dtst_plan_st {
  dtst::Derived dv;
  int device = 0;
  float* blob = nullptr;  // device copy of every basis image
};

namespace {

thread_local std::string g_last_error;

std::mutex g_plans_mu;
std::unordered_set<const dtst_plan_st*>& live_plans() {
  static std::unordered_set<const dtst_plan_st*> s;
  return s;
}

dtst_status fail(dtst_status s, const std::string& msg) {
  g_last_error = msg;
  return s;
}

dtst_status ok() {
  g_last_error.clear();
  return DTST_OK;
}

bool is_live(const dtst_plan_st* p) {
  std::lock_guard<std::mutex> lk(g_plans_mu);
  return p != nullptr && live_plans().count(p) != 0;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Makes the plan's device current for the duration of a call.
struct DeviceGuard {
  int prev = -1;
  bool switched = false;
  hipError_t err = hipSuccess;
  explicit DeviceGuard(int dev) {
    err = hipGetDevice(&prev);
    if (err == hipSuccess && prev != dev) {
      err = hipSetDevice(dev);
      switched = err == hipSuccess;
    }
  }
  ~DeviceGuard() {
    if (switched) (void)hipSetDevice(prev);
  }
};

dtst_status device_status(int e, const char* what) {
  if (e == hipSuccess) return ok();
  return fail(DTST_ERR_DEVICE, std::string(what) + ": " + hipGetErrorString(static_cast<hipError_t>(e)));
}

dtst_status check_plan(const dtst_plan_st* p) {
  if (!is_live(p)) return fail(DTST_ERR_INVALID_ARG, "plan is null or was destroyed");
  return DTST_OK;
}

dtst_status check_ptr(const void* ptr, const char* name) {
  if (ptr == nullptr) return fail(DTST_ERR_INVALID_ARG, std::string(name) + " is null");
  if (!aligned16(ptr)) return fail(DTST_ERR_INVALID_ARG, std::string(name) + " is not 16-byte aligned");
  return DTST_OK;
}

dtst_status check_ws(const dtst_plan_st* p, const void* ws, size_t ws_bytes) {
  if (ws_bytes < p->dv.ws_bytes)
    return fail(DTST_ERR_INVALID_ARG, "workspace too small: need " + std::to_string(p->dv.ws_bytes) +
                                          " bytes, got " + std::to_string(ws_bytes));
  if (p->dv.ws_bytes > 0) return check_ptr(ws, "workspace");
  return DTST_OK;
}

#define DTST_TRY(expr)                 \
  do {                                 \
    dtst_status s_ = (expr);           \
    if (s_ != DTST_OK) return s_;      \
  } while (0)

// ---- per-kernel event timing (dtst_profile_enable / dtst_profile_collect) ----
enum KernelRole { K_FWD_TZ, K_AXIS_FWD_Y, K_AXIS_FWD_X, K_AXIS_INV_X, K_AXIS_INV_Y, K_INV_ZT, K_MIX, K_MIX_H,
                  K_WGRAD, K_BLOCK, K_FWD_TZY, K_INV_YZT, K_POINTWISE, K_INV_ZT_BLOCK, K_COUNT };
const char* const kRoleNames[K_COUNT] = {"stream_fwd_tz", "axis_fwd_y", "axis_fwd_x", "axis_inv_x", "axis_inv_y",
                                         "stream_inv_zt", "mix", "mix_h", "wgrad", "block_epilogue",
                                         "stream_fwd_tzy", "stream_inv_yzt", "pointwise", "stream_inv_zt_block"};

struct Profiler {
  std::mutex mu;
  bool on = false;
  struct Rec {
    int role;
    hipEvent_t a, b;
  };
  std::vector<Rec> pending;
  std::vector<hipEvent_t> pool;
  double total_ms[K_COUNT] = {};
  int64_t launches[K_COUNT] = {};
  hipEvent_t get() {
    if (!pool.empty()) {
      hipEvent_t e = pool.back();
      pool.pop_back();
      return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
  }
};
Profiler& prof() {
  static Profiler p;
  return p;
}

// Runs one launcher; when profiling is on, brackets it with events on `stream`.
template <class F>
int timed(int role, void* stream, F&& launch) {
  Profiler& P = prof();
  bool on;
  {
    std::lock_guard<std::mutex> lk(P.mu);
    on = P.on;
  }
  if (!on) return launch();
  hipEvent_t a, b;
  {
    std::lock_guard<std::mutex> lk(P.mu);
    a = P.get();
    b = P.get();
  }
  if (a == nullptr || b == nullptr) return launch();
  const hipStream_t s = static_cast<hipStream_t>(stream);
  (void)hipEventRecord(a, s);
  const int e = launch();
  (void)hipEventRecord(b, s);
  std::lock_guard<std::mutex> lk(P.mu);
  P.pending.push_back({role, a, b});
  return e;
}

// Forward-direction chain: streaming t+z, then y (one fused launch when the
// plan allows it), then x (with accumulate).
dtst_status run_forward_chain(const dtst_plan_st* p, int64_t channels, const float* x, void* xhat,
                              int accumulate, void* ws, const float* timg, void* stream) {
  const dtst::Derived& dv = p->dv;
  const int64_t B = dv.d.batch;
  if (B == 0) return ok();
  char* w1 = static_cast<char*>(ws);
  char* w2 = w1 + dv.w1_bytes;
  const int64_t planes = B * channels * dv.d.n_local[0];
  const int64_t rows = planes * dv.d.n_local[1];
  int e;
  if (dv.sc.fuse_y) {
    e = timed(K_FWD_TZY, stream, [&] {
      return dtst::launch_fwd_tzy(dv.sc, dv.ay_f, x, w2, planes, static_cast<int>(dv.d.n_local[1]), timg,
                                  p->blob + dv.img.z_fwd, p->blob + dv.img.y_fwd, stream);
    });
    if (e != hipSuccess) return device_status(e, "t+z+y contraction launch");
  } else {
    e = timed(K_FWD_TZ, stream,
              [&] { return dtst::launch_fwd_tz(dv.sc, x, w1, rows, timg, p->blob + dv.img.z_fwd, stream); });
    if (e != hipSuccess) return device_status(e, "t+z contraction launch");
    e = timed(K_AXIS_FWD_Y, stream, [&] {
      return dtst::launch_axis(dv.ay_f, planes, w1, w2, p->blob + dv.img.y_fwd, 0, stream);
    });
    if (e != hipSuccess) return device_status(e, "y contraction launch");
  }
  e = timed(K_AXIS_FWD_X, stream, [&] {
    return dtst::launch_axis(dv.ax_f, B * channels, w2, xhat, p->blob + dv.img.x_fwd, accumulate, stream);
  });
  if (e != hipSuccess) return device_status(e, "x contraction launch");
  return ok();
}

// Inverse-direction chain: x, then y, then streaming z+t with Re (y, z and t
// in one launch when the plan allows it).
dtst_status run_inverse_chain(const dtst_plan_st* p, int64_t channels, const void* yhat, float* y, void* ws,
                              const float* timg, void* stream) {
  const dtst::Derived& dv = p->dv;
  const int64_t B = dv.d.batch;
  if (B == 0) return ok();
  char* v2 = static_cast<char*>(ws);    // (.., Nx, Ny, Kz, Kt)
  char* v1 = v2 + dv.w1_bytes;          // (.., Nx, Ky, Kz, Kt)
  int e = timed(K_AXIS_INV_X, stream, [&] {
    return dtst::launch_axis(dv.ax_i, B * channels, yhat, v1, p->blob + dv.img.x_inv, 0, stream);
  });
  if (e != hipSuccess) return device_status(e, "x expansion launch");
  const int64_t planes = B * channels * dv.d.n_local[0];
  if (dv.sc.fuse_y) {
    e = timed(K_INV_YZT, stream, [&] {
      return dtst::launch_inv_yzt(dv.sc, dv.ay_i, v1, y, planes, static_cast<int>(dv.d.n_local[1]), timg,
                                  p->blob + dv.img.z_inv, p->blob + dv.img.y_inv, stream);
    });
    if (e != hipSuccess) return device_status(e, "y+z+t expansion launch");
    return ok();
  }
  e = timed(K_AXIS_INV_Y, stream, [&] {
    return dtst::launch_axis(dv.ay_i, planes, v1, v2, p->blob + dv.img.y_inv, 0, stream);
  });
  if (e != hipSuccess) return device_status(e, "y expansion launch");
  const int64_t rows = planes * dv.d.n_local[1];
  e = timed(K_INV_ZT, stream,
            [&] { return dtst::launch_inv_zt(dv.sc, v2, y, rows, timg, p->blob + dv.img.z_inv, stream); });
  if (e != hipSuccess) return device_status(e, "z+t expansion launch");
  return ok();
}

// Descriptor and plan-flag checks shared by dtst_desc_validate and dtst_plan_ex.
dtst_status validate_ex(const dtst_desc* d, uint32_t flags) {
  dtst::Derived dv;
  std::string err;
  const dtst_status s = dtst::derive(d, flags, &dv, &err);
  if (s != DTST_OK) return fail(s, err);
  if (dv.d.c_out > dtst::kMixMaxCout)
    return fail(DTST_ERR_UNSUPPORTED, "c_out above " + std::to_string(dtst::kMixMaxCout) + " for the mix kernels");
  if (dtst::mix_lds_bytes(dv.d.batch, dv.d.c_in, dv.d.c_out) > 160 * 1024)
    return fail(DTST_ERR_UNSUPPORTED, "batch * channels too large for one workgroup of the mix kernels");
  return ok();
}

}  // namespace

extern "C" {

const char* dtst_status_string(dtst_status s) {
  switch (s) {
    case DTST_OK: return "DTST_OK";
    case DTST_ERR_INVALID_ARG: return "DTST_ERR_INVALID_ARG";
    case DTST_ERR_UNSUPPORTED: return "DTST_ERR_UNSUPPORTED";
    case DTST_ERR_OUT_OF_MEMORY: return "DTST_ERR_OUT_OF_MEMORY";
    case DTST_ERR_DEVICE: return "DTST_ERR_DEVICE";
  }
  return "DTST_ERR_UNKNOWN";
}

const char* dtst_last_error(void) { return g_last_error.c_str(); }

dtst_status dtst_desc_validate(const dtst_desc* d) { return validate_ex(d, 0); }

dtst_status dtst_desc_workspace_bytes_ex(const dtst_desc* d, uint32_t flags, size_t* bytes) {
  if (!bytes) return fail(DTST_ERR_INVALID_ARG, "bytes is null");
  dtst::Derived dv;
  std::string err;
  const dtst_status s = dtst::derive(d, flags, &dv, &err);
  if (s != DTST_OK) return fail(s, err);
  *bytes = dv.ws_bytes;
  return ok();
}

dtst_status dtst_desc_workspace_bytes(const dtst_desc* d, size_t* bytes) {
  return dtst_desc_workspace_bytes_ex(d, 0, bytes);
}

dtst_status dtst_basis_host(const dtst_desc* d, int dim, int kind, float* out, size_t count) {
  dtst::Derived dv;
  std::string err;
  const dtst_status s = dtst::derive(d, 0, &dv, &err);
  if (s != DTST_OK) return fail(s, err);
  if (dim < 0 || dim > 3 || (kind != 0 && kind != 1) || out == nullptr)
    return fail(DTST_ERR_INVALID_ARG, "dim must be 0..3, kind 0 or 1, out non-null");
  const size_t need = size_t(2) * dv.K[dim] * d->n_local[dim];
  if (count != need) return fail(DTST_ERR_INVALID_ARG, "count must be 2*K*N_loc = " + std::to_string(need));
  dtst::plain_basis(*d, dim, kind, out);
  return ok();
}

dtst_status dtst_plan_ex(const dtst_desc* d, uint32_t flags, dtst_plan_t* out) {
  if (!out) return fail(DTST_ERR_INVALID_ARG, "out is null");
  const dtst_status vs = validate_ex(d, flags);
  if (vs != DTST_OK) return vs;
  dtst_plan_st* p = new (std::nothrow) dtst_plan_st();
  if (!p) return fail(DTST_ERR_OUT_OF_MEMORY, "host allocation failed");
  std::string err;
  dtst::derive(d, flags, &p->dv, &err);
  std::vector<float> host;
  try {
    dtst::build_images(p->dv, &host);
  } catch (...) {
    delete p;
    return fail(DTST_ERR_OUT_OF_MEMORY, "host allocation of the basis tables failed");
  }
  hipError_t e = hipGetDevice(&p->device);
  if (e != hipSuccess) {
    delete p;
    return fail(DTST_ERR_DEVICE, std::string("hipGetDevice: ") + hipGetErrorString(e));
  }
  e = hipMalloc(&p->blob, host.size() * sizeof(float));
  if (e != hipSuccess) {
    delete p;
    (void)hipGetLastError();
    return fail(e == hipErrorOutOfMemory ? DTST_ERR_OUT_OF_MEMORY : DTST_ERR_DEVICE,
                std::string("hipMalloc of the basis tables: ") + hipGetErrorString(e));
  }
  e = hipMemcpy(p->blob, host.data(), host.size() * sizeof(float), hipMemcpyHostToDevice);
  if (e != hipSuccess) {
    (void)hipFree(p->blob);
    delete p;
    return fail(DTST_ERR_DEVICE, std::string("hipMemcpy of the basis tables: ") + hipGetErrorString(e));
  }
  int pe = dtst::prepare_stream(&p->dv.sc);
  if (pe == hipSuccess && p->dv.blk &&
      dtst::prepare_block_zt(p->dv.sb, p->dv.d.c_in, p->dv.d.c_out, &p->dv.grid_blk) != hipSuccess) {
    // the device does not take the fused block kernel at this size: the
    // plan keeps the two launches (dtst_plan_block_info reports it)
    (void)hipGetLastError();
    p->dv.blk = 0;
  }
  if (pe != hipSuccess) {
    (void)hipFree(p->blob);
    delete p;
    return fail(DTST_ERR_DEVICE, std::string("kernel setup: ") + hipGetErrorString(static_cast<hipError_t>(pe)));
  }
  // Device address of this device's scratch array (dtst_forward_noalloc),
  // looked up once per device while the plan's device is current.  A failed
  // lookup does not fail the plan: dtst_forward_noalloc repeats it and
  // reports the error.
  void* scratch = nullptr;
  (void)dtst::scratch_address(p->device, &scratch);
  {
    std::lock_guard<std::mutex> lk(g_plans_mu);
    live_plans().insert(p);
  }
  *out = p;
  return ok();
}

dtst_status dtst_plan(const dtst_desc* d, dtst_plan_t* out) { return dtst_plan_ex(d, 0, out); }

dtst_status dtst_plan_destroy(dtst_plan_t p) {
  {
    std::lock_guard<std::mutex> lk(g_plans_mu);
    if (p == nullptr || live_plans().erase(p) == 0)
      return fail(DTST_ERR_INVALID_ARG, "plan is null or was destroyed");
  }
  DeviceGuard guard(p->device);
  const hipError_t e = hipFree(p->blob);
  delete p;
  if (e != hipSuccess) return fail(DTST_ERR_DEVICE, std::string("hipFree: ") + hipGetErrorString(e));
  return ok();
}

dtst_status dtst_plan_info(dtst_plan_t p, int64_t* n_modes, size_t* workspace_bytes) {
  DTST_TRY(check_plan(p));
  if (n_modes) *n_modes = p->dv.M;
  if (workspace_bytes) *workspace_bytes = p->dv.ws_bytes;
  return ok();
}

dtst_status dtst_forward(dtst_plan_t p, const float* x, void* xhat, int accumulate, void* workspace,
                         size_t workspace_bytes, void* stream) {
  DTST_TRY(check_plan(p));
  if (p->dv.d.batch == 0) return ok();
  DTST_TRY(check_ptr(x, "x"));
  DTST_TRY(check_ptr(xhat, "xhat"));
  DTST_TRY(check_ws(p, workspace, workspace_bytes));
  if (accumulate != 0 && accumulate != 1) return fail(DTST_ERR_INVALID_ARG, "accumulate must be 0 or 1");
  DeviceGuard guard(p->device);
  if (guard.err != hipSuccess) return device_status(guard.err, "hipSetDevice");
  return run_forward_chain(p, p->dv.d.c_in, x, xhat, accumulate, workspace, p->blob + p->dv.img.t_fwd, stream);
}

dtst_status dtst_forward_noalloc(dtst_plan_t p, const float* x, void* xhat, int accumulate, void* stream) {
  DTST_TRY(check_plan(p));
  if (p->dv.d.batch == 0) return ok();
  DTST_TRY(check_ptr(x, "x"));
  DTST_TRY(check_ptr(xhat, "xhat"));
  if (accumulate != 0 && accumulate != 1) return fail(DTST_ERR_INVALID_ARG, "accumulate must be 0 or 1");
  if (p->dv.ws_bytes > dtst::kScratchBytes)
    return fail(DTST_ERR_UNSUPPORTED, "this plan needs a workspace of " + std::to_string(p->dv.ws_bytes) +
                                          " bytes, above the " + std::to_string(dtst::kScratchBytes) +
                                          "-byte scratch array of dtst_forward_noalloc; use dtst_forward");
  DeviceGuard guard(p->device);
  if (guard.err != hipSuccess) return device_status(guard.err, "hipSetDevice");
  void* scratch = nullptr;  // found at plan creation on this device
  const int se = dtst::scratch_address(p->device, &scratch);
  if (se != hipSuccess) return device_status(se, "scratch array lookup");
  return run_forward_chain(p, p->dv.d.c_in, x, xhat, accumulate, scratch, p->blob + p->dv.img.t_fwd, stream);
}

dtst_status dtst_inverse_adj(dtst_plan_t p, const float* g_y, void* g_yhat, int accumulate, void* workspace,
                             size_t workspace_bytes, void* stream) {
  DTST_TRY(check_plan(p));
  if (p->dv.d.batch == 0) return ok();
  DTST_TRY(check_ptr(g_y, "g_y"));
  DTST_TRY(check_ptr(g_yhat, "g_yhat"));
  DTST_TRY(check_ws(p, workspace, workspace_bytes));
  if (accumulate != 0 && accumulate != 1) return fail(DTST_ERR_INVALID_ARG, "accumulate must be 0 or 1");
  DeviceGuard guard(p->device);
  if (guard.err != hipSuccess) return device_status(guard.err, "hipSetDevice");
  return run_forward_chain(p, p->dv.d.c_out, g_y, g_yhat, accumulate, workspace,
                           p->blob + p->dv.img.t_fwd_adjoint_of_inverse, stream);
}

dtst_status dtst_inverse(dtst_plan_t p, const void* yhat, float* y, void* workspace, size_t workspace_bytes,
                         void* stream) {
  DTST_TRY(check_plan(p));
  if (p->dv.d.batch == 0) return ok();
  DTST_TRY(check_ptr(yhat, "yhat"));
  DTST_TRY(check_ptr(y, "y"));
  DTST_TRY(check_ws(p, workspace, workspace_bytes));
  DeviceGuard guard(p->device);
  if (guard.err != hipSuccess) return device_status(guard.err, "hipSetDevice");
  return run_inverse_chain(p, p->dv.d.c_out, yhat, y, workspace, p->blob + p->dv.img.t_inv, stream);
}

dtst_status dtst_forward_adj(dtst_plan_t p, const void* g_xhat, float* g_x, void* workspace,
                             size_t workspace_bytes, void* stream) {
  DTST_TRY(check_plan(p));
  if (p->dv.d.batch == 0) return ok();
  DTST_TRY(check_ptr(g_xhat, "g_xhat"));
  DTST_TRY(check_ptr(g_x, "g_x"));
  DTST_TRY(check_ws(p, workspace, workspace_bytes));
  DeviceGuard guard(p->device);
  if (guard.err != hipSuccess) return device_status(guard.err, "hipSetDevice");
  return run_inverse_chain(p, p->dv.d.c_in, g_xhat, g_x, workspace,
                           p->blob + p->dv.img.t_inv_adjoint_of_forward, stream);
}

dtst_status dtst_mix(dtst_plan_t p, const void* xhat, const void* w_shard, void* yhat, int64_t m0, int64_t m1,
                     int op, void* stream) {
  DTST_TRY(check_plan(p));
  const dtst::Derived& dv = p->dv;
  if (op != 0 && op != 1) return fail(DTST_ERR_INVALID_ARG, "op must be 0 (W) or 1 (W^H)");
  if (m0 < 0 || m1 < m0 || m1 > dv.M)
    return fail(DTST_ERR_INVALID_ARG, "mode range must satisfy 0 <= m0 <= m1 <= M = " + std::to_string(dv.M));
  if (dv.d.batch == 0 || m1 == m0) return ok();
  DTST_TRY(check_ptr(xhat, "xhat"));
  DTST_TRY(check_ptr(w_shard, "w_shard"));
  DTST_TRY(check_ptr(yhat, "yhat"));
  DeviceGuard guard(p->device);
  if (guard.err != hipSuccess) return device_status(guard.err, "hipSetDevice");
  const int e = timed(op == 0 ? K_MIX : K_MIX_H, stream, [&] {
    return op == 0 ? dtst::launch_mix(xhat, w_shard, yhat, dv.d.batch, dv.d.c_in, dv.d.c_out, dv.M, m0, m1, stream)
                   : dtst::launch_mix_h(xhat, w_shard, yhat, dv.d.batch, dv.d.c_in, dv.d.c_out, dv.M, m0, m1,
                                        stream);
  });
  return device_status(e, "mix launch");
}

dtst_status dtst_mix_wgrad(dtst_plan_t p, const void* xhat, const void* g_yhat, void* g_w_shard, int64_t m0,
                           int64_t m1, int accumulate, void* stream) {
  DTST_TRY(check_plan(p));
  const dtst::Derived& dv = p->dv;
  if (m0 < 0 || m1 < m0 || m1 > dv.M)
    return fail(DTST_ERR_INVALID_ARG, "mode range must satisfy 0 <= m0 <= m1 <= M = " + std::to_string(dv.M));
  if (accumulate != 0 && accumulate != 1) return fail(DTST_ERR_INVALID_ARG, "accumulate must be 0 or 1");
  if (dv.d.batch == 0 || m1 == m0) return ok();
  DTST_TRY(check_ptr(xhat, "xhat"));
  DTST_TRY(check_ptr(g_yhat, "g_yhat"));
  DTST_TRY(check_ptr(g_w_shard, "g_w_shard"));
  DeviceGuard guard(p->device);
  if (guard.err != hipSuccess) return device_status(guard.err, "hipSetDevice");
  const int e = timed(K_WGRAD, stream, [&] {
    return dtst::launch_wgrad(xhat, g_yhat, g_w_shard, dv.d.batch, dv.d.c_in, dv.d.c_out, dv.M, m0, m1,
                              accumulate, stream);
  });
  return device_status(e, "wgrad launch");
}

}  // extern "C"

namespace {

// Argument checks shared by the two block calls: pointers, the LDS limit on
// the bypass matrix, and x not overlapping y (y is written while x is read).
dtst_status check_block(const dtst_plan_st* p, const float* x, const float* w_bypass, const float* y) {
  const dtst::Derived& dv = p->dv;
  DTST_TRY(check_ptr(x, "x"));
  DTST_TRY(check_ptr(w_bypass, "w_bypass"));
  DTST_TRY(check_ptr(y, "y"));
  if (dv.d.c_in * dv.d.c_out * int64_t(sizeof(float)) > 160 * 1024)
    return fail(DTST_ERR_UNSUPPORTED, "c_in * c_out above 40960: the bypass matrix must fit in LDS");
  const int64_t V = dv.d.n_local[0] * dv.d.n_local[1] * dv.d.n_local[2] * dv.d.n_local[3];
  const char* xb = reinterpret_cast<const char*>(x);
  const char* yb = reinterpret_cast<const char*>(y);
  const size_t xbytes = size_t(dv.d.batch) * dv.d.c_in * V * sizeof(float);
  const size_t ybytes = size_t(dv.d.batch) * dv.d.c_out * V * sizeof(float);
  if (xb < yb + ybytes && yb < xb + xbytes) return fail(DTST_ERR_INVALID_ARG, "x and y overlap");
  return ok();
}

dtst_status run_block_epilogue(const dtst_plan_st* p, const float* x, const float* w_bypass, float* y,
                               void* stream) {
  const dtst::Derived& dv = p->dv;
  const int64_t V = dv.d.n_local[0] * dv.d.n_local[1] * dv.d.n_local[2] * dv.d.n_local[3];
  const int e = timed(K_BLOCK, stream, [&] {
    return dtst::launch_block_epilogue(x, w_bypass, y, dv.d.batch, dv.d.c_in, dv.d.c_out, V, stream);
  });
  return device_status(e, "block epilogue launch");
}

}  // namespace

extern "C" {

dtst_status dtst_pointwise(const float* x, const float* w, const float* bias, float* y, int64_t batch, int64_t c_in,
                           int64_t c_out, int64_t points, int act, void* stream) {
  if (batch < 0 || points < 0 || c_in < 1 || c_out < 1)
    return fail(DTST_ERR_INVALID_ARG, "need batch >= 0, points >= 0, c_in >= 1, c_out >= 1");
  if (act != 0 && act != 1) return fail(DTST_ERR_INVALID_ARG, "act must be 0 (identity) or 1 (GELU)");
  if ((c_in * c_out + c_out) * int64_t(sizeof(float)) > 160 * 1024)
    return fail(DTST_ERR_UNSUPPORTED, "c_in * c_out + c_out above 40960: the weights must fit in LDS");
  if (batch == 0 || points == 0) return ok();
  DTST_TRY(check_ptr(x, "x"));
  DTST_TRY(check_ptr(w, "w"));
  if (bias != nullptr) DTST_TRY(check_ptr(bias, "bias"));
  DTST_TRY(check_ptr(y, "y"));
  int64_t nx = 0, ny = 0;
  if (__builtin_mul_overflow(batch * c_in, points, &nx) || __builtin_mul_overflow(batch * c_out, points, &ny) ||
      nx > (int64_t(1) << 50) || ny > (int64_t(1) << 50))
    return fail(DTST_ERR_INVALID_ARG, "problem size overflows the supported element counts");
  const char* xb = reinterpret_cast<const char*>(x);
  const char* yb = reinterpret_cast<const char*>(y);
  if (xb < yb + size_t(ny) * sizeof(float) && yb < xb + size_t(nx) * sizeof(float))
    return fail(DTST_ERR_INVALID_ARG, "x and y overlap");
  const int e = timed(K_POINTWISE, stream, [&] {
    return dtst::launch_pointwise(x, w, bias, y, batch, c_in, c_out, points, act, stream);
  });
  return device_status(e, "point-wise launch");
}

dtst_status dtst_block_epilogue(dtst_plan_t p, const float* x, const float* w_bypass, float* y, void* stream) {
  DTST_TRY(check_plan(p));
  if (p->dv.d.batch == 0) return ok();
  DTST_TRY(check_block(p, x, w_bypass, y));
  DeviceGuard guard(p->device);
  if (guard.err != hipSuccess) return device_status(guard.err, "hipSetDevice");
  return run_block_epilogue(p, x, w_bypass, y, stream);
}

dtst_status dtst_inverse_block(dtst_plan_t p, const void* yhat, const float* x, const float* w_bypass, float* y,
                               void* workspace, size_t workspace_bytes, void* stream) {
  DTST_TRY(check_plan(p));
  const dtst::Derived& dv = p->dv;
  if (dv.d.batch == 0) return ok();
  DTST_TRY(check_ptr(yhat, "yhat"));
  DTST_TRY(check_block(p, x, w_bypass, y));
  if (workspace_bytes < dv.blk_ws_bytes)
    return fail(DTST_ERR_INVALID_ARG, "workspace too small: need " + std::to_string(dv.blk_ws_bytes) +
                                          " bytes, got " + std::to_string(workspace_bytes));
  if (dv.blk_ws_bytes > 0) DTST_TRY(check_ptr(workspace, "workspace"));
  DeviceGuard guard(p->device);
  if (guard.err != hipSuccess) return device_status(guard.err, "hipSetDevice");
  if (!dv.blk) {
    DTST_TRY(run_inverse_chain(p, dv.d.c_out, yhat, y, workspace, p->blob + dv.img.t_inv, stream));
    return run_block_epilogue(p, x, w_bypass, y, stream);
  }
  // x expansion into W2, y expansion into W1, then z + t with the epilogue
  const int64_t B = dv.d.batch, co = dv.d.c_out;
  char* w1 = static_cast<char*>(workspace);
  char* w2 = w1 + dv.blk_w1_bytes;
  int e = timed(K_AXIS_INV_X, stream, [&] {
    return dtst::launch_axis(dv.ax_i, B * co, yhat, w2, p->blob + dv.img.x_inv, 0, stream);
  });
  if (e != hipSuccess) return device_status(e, "x expansion launch");
  const int64_t planes = B * co * dv.d.n_local[0];
  e = timed(K_AXIS_INV_Y, stream,
            [&] { return dtst::launch_axis(dv.ay_b, planes, w2, w1, p->blob + dv.img.y_blk, 0, stream); });
  if (e != hipSuccess) return device_status(e, "y expansion launch");
  e = timed(K_INV_ZT_BLOCK, stream, [&] {
    return dtst::launch_inv_zt_block(dv.sb, dv.grid_blk, w1, x, w_bypass, y, B,
                                     dv.d.n_local[0] * dv.d.n_local[1], dv.d.c_in, co, p->blob + dv.img.t_blk,
                                     p->blob + dv.img.z_blk, stream);
  });
  return device_status(e, "z+t expansion and block epilogue launch");
}

dtst_status dtst_plan_block_info(dtst_plan_t p, size_t* workspace_bytes, int* fused) {
  DTST_TRY(check_plan(p));
  if (workspace_bytes) *workspace_bytes = p->dv.blk_ws_bytes;
  if (fused) *fused = p->dv.blk;
  return ok();
}

dtst_status dtst_profile_enable(int on) {
  Profiler& P = prof();
  std::lock_guard<std::mutex> lk(P.mu);
  P.on = on != 0;
  return ok();
}

dtst_status dtst_profile_collect(dtst_kernel_time* out, int capacity, int* count) {
  if (count == nullptr || (capacity > 0 && out == nullptr) || capacity < 0)
    return fail(DTST_ERR_INVALID_ARG, "need count, and out when capacity > 0");
  Profiler& P = prof();
  std::lock_guard<std::mutex> lk(P.mu);
  hipError_t err = hipSuccess;
  for (const Profiler::Rec& r : P.pending) {
    float ms = 0.f;
    hipError_t e = hipEventSynchronize(r.b);
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, r.a, r.b);
    if (e == hipSuccess) {
      P.total_ms[r.role] += ms;
      P.launches[r.role] += 1;
    } else if (err == hipSuccess) {
      err = e;
    }
    P.pool.push_back(r.a);
    P.pool.push_back(r.b);
  }
  P.pending.clear();
  int n = 0;
  for (int k = 0; k < K_COUNT; ++k) {
    if (P.launches[k] == 0) continue;
    if (n < capacity) {
      std::snprintf(out[n].name, sizeof(out[n].name), "%s", kRoleNames[k]);
      out[n].launches = P.launches[k];
      out[n].total_ms = P.total_ms[k];
    }
    ++n;
    P.launches[k] = 0;
    P.total_ms[k] = 0.0;
  }
  *count = n < capacity ? n : capacity;
  if (err != hipSuccess) return fail(DTST_ERR_DEVICE, std::string("event timing: ") + hipGetErrorString(err));
  return ok();
}

}  // extern "C"
