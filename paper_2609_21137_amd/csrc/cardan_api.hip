// C ABI of libcardan.so: argument validation, launch planning, workspace
// layout and the kernel sequence of every entry point.
#include <hip/hip_runtime.h>

#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <mutex>
#include <vector>

#include "../../include/cardan.h"
#include "cardan_plan.h"

namespace cardan {
const void* route_kernel();
const void* expert_kernel(const Plan& P);
hipError_t launch_route(const Plan&, const Args&, const Chain&, int, size_t, hipStream_t, hipEvent_t, hipEvent_t);
hipError_t launch_expert(const Plan&, const Args&, const Chain&, int, size_t, hipStream_t, hipEvent_t, hipEvent_t);
hipError_t launch_route_reset(const Plan&, const Args&, hipStream_t);
hipError_t launch_zero(void* p, size_t bytes, hipStream_t);
hipError_t launch_rmsnorm(hipStream_t, int, int, const float*, float, uint16_t*, hipEvent_t, hipEvent_t);
}  // namespace cardan

using namespace cardan;

namespace {

thread_local char g_err[512] = "";

int fail(int code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof g_err, fmt, ap);
  va_end(ap);
  return code;
}

bool misaligned(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) != 0; }

// Shape and batch validation shared by every entry point.
int check_shape(const cardan_shape* s, int32_t B) {
  if (!s) return fail(CARDAN_ERR_NULL_PTR, "shape is NULL");
  if (s->H <= 0 || s->I <= 0 || s->E <= 0 || s->top_k <= 0 || s->d <= 0 || s->K <= 0 || s->r < 0)
    return fail(CARDAN_ERR_BAD_SHAPE, "shape fields must be positive (r >= 0)");
  if (s->top_k > s->E) return fail(CARDAN_ERR_BAD_SHAPE, "top_k=%d exceeds E=%d", s->top_k, s->E);
  if (s->H % s->d || s->I % s->d)
    return fail(CARDAN_ERR_BAD_SHAPE, "H=%d and I=%d must be multiples of d=%d", s->H, s->I, s->d);
  if (B < 1 || B > kMaxB) return fail(CARDAN_ERR_BAD_SHAPE, "B=%d outside [1, %d]", B, kMaxB);
  if (s->K > 256) return fail(CARDAN_ERR_BAD_SHAPE, "K=%d exceeds 256 (uint8 codes)", s->K);
  if (s->d != 2 && s->d != 4 && s->d != 8) return fail(CARDAN_ERR_UNSUPPORTED, "d=%d not compiled (2, 4, 8)", s->d);
  if (s->H % 64) return fail(CARDAN_ERR_UNSUPPORTED, "H=%d must be a multiple of 64", s->H);
  if (s->I % 32) return fail(CARDAN_ERR_UNSUPPORTED, "I=%d must be a multiple of 32", s->I);
  if (s->E > kMaxE) return fail(CARDAN_ERR_UNSUPPORTED, "E=%d exceeds %d", s->E, kMaxE);
  if (s->top_k > kMaxK) return fail(CARDAN_ERR_UNSUPPORTED, "top_k=%d exceeds %d", s->top_k, kMaxK);
  if (s->r > kMaxR || (s->r % 8))
    return fail(CARDAN_ERR_UNSUPPORTED, "r=%d must be a multiple of 8 and <= %d", s->r, kMaxR);
  return CARDAN_OK;
}

// Co-resident workgroups of a kernel on the current device for a given
// dynamic LDS size. Cached per (device, kernel, LDS size); the cache is the
// library's only shared host state on the layer path, so lookups and inserts
// hold a mutex (the occupancy query itself runs outside it; two threads that
// miss together both query and insert the same value).
int resident_grid(const void* fn, size_t lds, hipError_t* err) {
  struct Entry {
    int dev;
    const void* fn;
    size_t lds;
    int grid;
  };
  static std::mutex mu;
  static Entry cache[64];
  static int n_cache = 0;
  int dev = 0;
  *err = hipGetDevice(&dev);
  if (*err != hipSuccess) return 0;
  {
    std::lock_guard<std::mutex> lock(mu);
    for (int i = 0; i < n_cache; ++i)
      if (cache[i].dev == dev && cache[i].fn == fn && cache[i].lds == lds) return cache[i].grid;
  }
  int cus = 0, per_cu = 0;
  *err = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (*err != hipSuccess) return 0;
  *err = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, kWG, lds);
  if (*err != hipSuccess) return 0;
  const int g = std::max(1, cus * per_cu);
  std::lock_guard<std::mutex> lock(mu);
  bool have = false;
  for (int i = 0; i < n_cache && !have; ++i)
    have = cache[i].dev == dev && cache[i].fn == fn && cache[i].lds == lds;
  if (!have && n_cache < 64) cache[n_cache++] = {dev, fn, lds, g};
  return g;
}

// Gate/up form of a whole-layer call: the environment variable CARDAN_GATEUP
// = "tbook" requests the projection-code-book tiles, "codeword" the
// code-word tiles; otherwise the default below. The planner drops F_TBOOK
// where it does not apply.
int gateup_form(const cardan_shape*, int) {
  const char* v = getenv("CARDAN_GATEUP");
  if (v && strcmp(v, "tbook") == 0) return F_TBOOK;
  return 0;
}

int check_ws(const Plan& P, const void* ws, size_t ws_bytes) {
  if (!ws) return fail(CARDAN_ERR_NULL_PTR, "workspace is NULL");
  if (misaligned(ws)) return fail(CARDAN_ERR_ALIGN, "workspace is not 16-byte aligned");
  if (ws_bytes < P.total)
    return fail(CARDAN_ERR_WORKSPACE, "workspace of %zu bytes < required %zu", ws_bytes, P.total);
  return CARDAN_OK;
}

// Stacked decode step: buffers after the layer's workspace layout: y and the
// partial sums of squares of two layers (ping-pong), and two normalised bf16
// inputs (used when the caller keeps none).
struct StepBufs {
  size_t o_y, o_ssq, o_x, total;
};
size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }

StepBufs step_bufs(const Plan& P) {
  StepBufs b;
  size_t o = P.total;
  b.o_y = o; o = align256(o + (size_t)2 * P.B * P.H * 4);
  b.o_ssq = o; o = align256(o + (size_t)2 * P.B * combine_col_tiles(P) * 4);
  b.o_x = o; o = align256(o + (size_t)2 * P.B * P.H * 2);
  b.total = o;
  return b;
}

#define REQ(p, name)                                                                  \
  do {                                                                                \
    if (!(p)) return fail(CARDAN_ERR_NULL_PTR, "%s is NULL", name);                   \
    if (misaligned(p)) return fail(CARDAN_ERR_ALIGN, "%s is not 16-byte aligned", name); \
  } while (0)

// need_down: the compressed down projection (code book, codes, A, B) is used;
// need_gate: the gate projection is used (not for up-only experts)
int check_layer(const cardan_shape* s, const cardan_layer* L, bool need_router, bool need_down = true,
                bool need_gate = true) {
  if (!L) return fail(CARDAN_ERR_NULL_PTR, "layer is NULL");
  if (need_router) REQ(L->router_w, "router_w");
  if (L->router_bias && (reinterpret_cast<uintptr_t>(L->router_bias) & 3u))
    return fail(CARDAN_ERR_ALIGN, "router_bias is not 4-byte aligned");
  if (need_gate) {
    REQ(L->cb_gate, "cb_gate");
    REQ(L->codes_gate, "codes_gate");
  }
  REQ(L->cb_up, "cb_up");
  REQ(L->codes_up, "codes_up");
  if (need_down) {
    REQ(L->cb_down, "cb_down");
    REQ(L->codes_down, "codes_down");
  }
  if (s->r > 0) {
    if (need_gate) {
      REQ(L->U_gate, "U_gate");
      REQ(L->V_gate, "V_gate");
    }
    REQ(L->U_up, "U_up");
    REQ(L->V_up, "V_up");
    if (need_down) {
      REQ(L->A_down, "A_down");
      REQ(L->B_down, "B_down");
    }
  }
  return CARDAN_OK;
}

// one expert's dense bf16 matrix is addressed with 32-bit byte offsets
int check_dense_size(const cardan_shape* s) {
  if ((size_t)s->H * s->I * 2 >= 0x80000000ull)
    return fail(CARDAN_ERR_UNSUPPORTED, "dense expert matrix of H=%d x I=%d exceeds 2 GiB", s->H, s->I);
  return CARDAN_OK;
}

// ---- kernel timing ---------------------------------------------------------
struct Profiler {
  bool on = false;
  int cap = 0;
  int calls = 0;
  std::vector<hipEvent_t> ev;       // per call: 2 events per kind
  std::vector<unsigned char> used;  // per call and kind
};
Profiler g_prof;

// Event pair of the next launch of `kind` while profiling (else nulls): the
// launch records them as part of the kernel's dispatch, so they bracket the
// kernel itself.
struct Timed {
  hipEvent_t ev0 = nullptr, ev1 = nullptr;
  size_t slot = 0;
  Timed(hipStream_t, int kind) {
    if (g_prof.on && g_prof.calls < g_prof.cap) {
      slot = (size_t)g_prof.calls * CARDAN_PROFILE_KINDS + kind;
      if (!g_prof.used[slot]) {
        ev0 = g_prof.ev[2 * slot];
        ev1 = g_prof.ev[2 * slot + 1];
      }
    }
  }
  void done() {
    if (ev0) g_prof.used[slot] = 1;
  }
};

void prof_next_call() {
  if (g_prof.on && g_prof.calls < g_prof.cap) ++g_prof.calls;
}

int hip_fail(hipError_t e, const char* what) {
  return fail(CARDAN_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

// Sizes the grids and launches k_route (if the call has routing items) and
// k_expert (if it has expert work) for one call.
int run_layer(const Plan& P, const Args& A, hipStream_t stream, const Chain* chain = nullptr) {
  Chain none;
  memset(&none, 0, sizeof none);
  const Chain& C = chain ? *chain : none;
  if (P.total >= 0x80000000ull)  // workspace offsets must stay below the out-of-range marker
    return fail(CARDAN_ERR_UNSUPPORTED, "workspace layout of %zu bytes exceeds 2 GiB", P.total);
  if (P.lds_route > kLdsMax || P.lds_expert > kLdsMax)
    return fail(CARDAN_ERR_UNSUPPORTED, "shape needs %zu/%zu bytes of LDS (> %zu)", P.lds_route,
                P.lds_expert, kLdsMax);
  hipError_t err;
  // k_route also clears k_expert's counters, so it runs (as one workgroup
  // if it has no items) whenever the call has expert work
  if (P.n_pre > 0 || (P.flags & F_EXPERTS)) {
    const int cap = resident_grid(route_kernel(), P.lds_route, &err);
    if (cap <= 0) return hip_fail(err, "occupancy query");
    Timed tm(stream, CARDAN_KERNEL_ROUTE);
    err = launch_route(P, A, C, std::max(1, std::min(cap, P.n_pre)), P.lds_route, stream, tm.ev0, tm.ev1);
    if (err != hipSuccess) return hip_fail(err, "k_route launch");
    tm.done();
    if (!(P.flags & F_EXPERTS)) {  // k_expert would clear these counters
      err = launch_route_reset(P, A, stream);
      if (err != hipSuccess) return hip_fail(err, "k_route_reset launch");
    }
  }
  if (P.flags & F_EXPERTS) {
    const int cap = resident_grid(expert_kernel(P), P.lds_expert, &err);
    if (cap <= 0) return hip_fail(err, "occupancy query");
    Timed tm(stream, CARDAN_KERNEL_EXPERT);
    err = launch_expert(P, A, C, cap, P.lds_expert, stream, tm.ev0, tm.ev1);
    if (err != hipSuccess) return hip_fail(err, "k_expert launch");
    tm.done();
  }
  prof_next_call();
  return CARDAN_OK;
}

// ---- the library's own scratch array (no-allocation entry point) ----------
// A fixed device-resident workspace for callers that cannot allocate. Each
// GPU holds its own copy, zero-filled when the code object loads, until the
// process ends. Host code never uses the array's name as an address: its
// device address is looked up once per device (hipGetSymbolAddress, with
// that device current) and kept in g_scratch.
constexpr size_t kScratchBytes = (size_t)CARDAN_SCRATCH_BYTES;
static __device__ __align__(256) uint8_t scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
struct ScratchState {
  void* ptr = nullptr;  // device address of `scratch` on this device
  int H = 0, I = 0, E = 0;  // shape of the last call enqueued outside graph capture
};
std::mutex g_scratch_mu;
ScratchState g_scratch[kMaxDevices];

// Device address of the scratch array on the current device, and whether
// its counters must be cleared before a call of shape (H, I, E): counter
// offsets depend on (H, I, E), and a call leaves its expert ticks set for the
// next call of the same shape to clear. They are cleared when the shape
// differs from the last call's, on the first call, and for every call
// recorded under graph capture (a replay may follow calls of any shape; the
// next eager call then clears again).
int scratch_for_call(const Plan& P, hipStream_t stream, void** ptr, bool* clear) {
  int dev = 0;
  hipError_t err = hipGetDevice(&dev);
  if (err != hipSuccess) return hip_fail(err, "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices) return fail(CARDAN_ERR_UNSUPPORTED, "device %d >= %d", dev, kMaxDevices);
  hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
  err = hipStreamIsCapturing(stream, &cap);
  if (err != hipSuccess) return hip_fail(err, "hipStreamIsCapturing");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  ScratchState& st = g_scratch[dev];
  if (!st.ptr) {
    void* p = nullptr;
    err = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (err != hipSuccess || !p) return hip_fail(err, "hipGetSymbolAddress(scratch)");
    st.ptr = p;
  }
  const bool same = st.H == P.H && st.I == P.I && st.E == P.E;
  if (cap != hipStreamCaptureStatusNone) {
    *clear = true;
    st.H = st.I = st.E = 0;
  } else {
    *clear = !same;
    st.H = P.H;
    st.I = P.I;
    st.E = P.E;
  }
  *ptr = st.ptr;
  return CARDAN_OK;
}

Args args_for(const cardan_layer* L, uint8_t* ws) {
  Args A;
  memset(&A, 0, sizeof A);
  if (L) A.L = *L;
  A.ws = ws;
  return A;
}

}  // namespace

extern "C" {

int cardan_abi_version(void) { return CARDAN_ABI_VERSION; }

const char* cardan_last_error(void) { return g_err; }

int cardan_workspace_bytes(const cardan_shape* shape, int32_t B, size_t* out) {
  g_err[0] = 0;
  int rc = check_shape(shape, B);
  if (rc) return rc;
  if (!out) return fail(CARDAN_ERR_NULL_PTR, "out is NULL");
  // the largest layout over batches 1..B, so one workspace serves any batch
  // up to B (split counts, hence layouts, depend on the batch)
  // and every expert-weight form (compressed, dense down, all dense) and
  // activation (gated SiLU, up-only squared ReLU) and gate/up form (code
  // words, projection code book)
  size_t need = 0;
  const int all = F_ROUTE | F_Z | F_GROUP | F_EXPERTS;
  for (int b = 1; b <= B; ++b) {
    for (int form : {0, (int)F_DN_DENSE, F_DN_DENSE | F_GU_DENSE})
      for (int act : {0, (int)F_UP_RELU2})
        for (int gu : {0, (int)F_TBOOK})
          need = std::max(need, make_plan(shape, b, 1, all | form | act | gu).total);
    need = std::max(need, step_bufs(make_plan(shape, b, 1, all | F_NORM_IN | F_SSQ_OUT)).total);
  }
  *out = need;
  return CARDAN_OK;
}

int cardan_route_topk(const cardan_shape* shape, int32_t B, const cardan_bf16* x,
                      const cardan_bf16* router_w, const float* router_bias, int32_t* topk_idx,
                      float* topk_w, void* ws, size_t ws_bytes, hipStream_t stream) {
  g_err[0] = 0;
  int rc = check_shape(shape, B);
  if (rc) return rc;
  REQ(x, "x");
  REQ(router_w, "router_w");
  REQ(topk_idx, "topk_idx");
  REQ(topk_w, "topk_w");
  if (router_bias && (reinterpret_cast<uintptr_t>(router_bias) & 3u))
    return fail(CARDAN_ERR_ALIGN, "router_bias is not 4-byte aligned");
  const Plan P = make_plan(shape, B, 1, F_ROUTE);
  if ((rc = check_ws(P, ws, ws_bytes))) return rc;
  cardan_layer L;
  memset(&L, 0, sizeof L);
  L.router_w = router_w;
  L.router_bias = router_bias;
  Args A = args_for(&L, static_cast<uint8_t*>(ws));
  A.x = x;
  A.topk_idx = topk_idx;
  A.topk_w = topk_w;
  return run_layer(P, A, stream);
}

int cardan_shared_proj(const cardan_shape* shape, int32_t B, const cardan_bf16* x,
                       const cardan_bf16* U_gate, const cardan_bf16* U_up, float* z, void* ws,
                       size_t ws_bytes, hipStream_t stream) {
  g_err[0] = 0;
  int rc = check_shape(shape, B);
  if (rc) return rc;
  if (shape->r == 0) return fail(CARDAN_ERR_BAD_SHAPE, "shared projection needs r > 0");
  REQ(x, "x");
  REQ(U_gate, "U_gate");
  REQ(U_up, "U_up");
  REQ(z, "z");
  const Plan P = make_plan(shape, B, U_up != U_gate, F_Z);
  if ((rc = check_ws(P, ws, ws_bytes))) return rc;
  cardan_layer L;
  memset(&L, 0, sizeof L);
  L.U_gate = U_gate;
  L.U_up = U_up;
  Args A = args_for(&L, static_cast<uint8_t*>(ws));
  A.x = x;
  A.z_out = z;
  return run_layer(P, A, stream);
}

int cardan_vq_lr_expert_ffn(const cardan_shape* shape, int32_t B, const cardan_bf16* x,
                            const int32_t* topk_idx, const float* topk_w, const float* z,
                            const cardan_layer* layer, float* y, void* ws, size_t ws_bytes,
                            hipStream_t stream) {
  g_err[0] = 0;
  int rc = check_shape(shape, B);
  if (rc) return rc;
  REQ(x, "x");
  REQ(topk_idx, "topk_idx");
  REQ(topk_w, "topk_w");
  REQ(y, "y");
  if (shape->r > 0) REQ(z, "z");
  if ((rc = check_layer(shape, layer, false))) return rc;
  const Plan P = make_plan(shape, B, 1, F_GROUP | F_EXPERTS);
  if ((rc = check_ws(P, ws, ws_bytes))) return rc;
  Args A = args_for(layer, static_cast<uint8_t*>(ws));
  A.x = x;
  A.idx_in = topk_idx;
  A.w_in = topk_w;
  A.z_in = z;
  A.y = y;
  return run_layer(P, A, stream);
}

int cardan_moe_layer(const cardan_shape* shape, int32_t B, const cardan_bf16* x,
                     const cardan_layer* layer, float* y, int32_t* topk_idx, float* topk_w,
                     void* ws, size_t ws_bytes, hipStream_t stream) {
  g_err[0] = 0;
  int rc = check_shape(shape, B);
  if (rc) return rc;
  REQ(x, "x");
  REQ(y, "y");
  REQ(topk_idx, "topk_idx");
  REQ(topk_w, "topk_w");
  if ((rc = check_layer(shape, layer, true))) return rc;
  const int z_sep = shape->r > 0 && layer->U_up != layer->U_gate;
  const int flags = F_ROUTE | F_GROUP | F_EXPERTS | (shape->r > 0 ? F_Z : 0) | gateup_form(shape, B);
  const Plan P = make_plan(shape, B, z_sep, flags);
  if ((rc = check_ws(P, ws, ws_bytes))) return rc;
  uint8_t* w = static_cast<uint8_t*>(ws);
  Args A = args_for(layer, w);
  A.x = x;
  A.topk_idx = topk_idx;
  A.topk_w = topk_w;
  A.z_out = reinterpret_cast<float*>(w + P.o_z);
  A.y = y;
  return run_layer(P, A, stream);
}

int cardan_moe_layer_relu2(const cardan_shape* shape, int32_t B, const cardan_bf16* x,
                           const cardan_layer* layer, float* y, int32_t* topk_idx, float* topk_w,
                           void* ws, size_t ws_bytes, hipStream_t stream) {
  g_err[0] = 0;
  int rc = check_shape(shape, B);
  if (rc) return rc;
  REQ(x, "x");
  REQ(y, "y");
  REQ(topk_idx, "topk_idx");
  REQ(topk_w, "topk_w");
  if ((rc = check_layer(shape, layer, true, true, false))) return rc;
  const int flags = F_ROUTE | F_GROUP | F_EXPERTS | F_UP_RELU2 | (shape->r > 0 ? F_Z : 0) | gateup_form(shape, B);
  const Plan P = make_plan(shape, B, 0, flags);
  if ((rc = check_ws(P, ws, ws_bytes))) return rc;
  // the kernels read only the up projection; the gate pointers alias it so
  // that the one z basis (U_gate slot) is the up basis
  cardan_layer L = *layer;
  L.cb_gate = L.cb_up;
  L.codes_gate = L.codes_up;
  L.U_gate = L.U_up;
  L.V_gate = L.V_up;
  uint8_t* w = static_cast<uint8_t*>(ws);
  Args A = args_for(&L, w);
  A.x = x;
  A.topk_idx = topk_idx;
  A.topk_w = topk_w;
  A.z_out = reinterpret_cast<float*>(w + P.o_z);
  A.y = y;
  return run_layer(P, A, stream);
}

int cardan_moe_decode_step(const cardan_shape* shape, int32_t B, int32_t n_layers, const cardan_bf16* x0,
                           const cardan_layer* layers, float eps, float* y, cardan_bf16* x_norm,
                           int32_t* topk_idx, float* topk_w, void* ws, size_t ws_bytes, hipStream_t stream) {
  g_err[0] = 0;
  int rc = check_shape(shape, B);
  if (rc) return rc;
  if (n_layers < 1 || n_layers > 4096) return fail(CARDAN_ERR_BAD_SHAPE, "n_layers=%d outside [1, 4096]", n_layers);
  if (!(eps >= 0.0f) || !isfinite(eps)) return fail(CARDAN_ERR_BAD_SHAPE, "eps must be finite and >= 0");
  REQ(x0, "x0");
  REQ(y, "y");
  REQ(topk_idx, "topk_idx");
  REQ(topk_w, "topk_w");
  if (x_norm && misaligned(x_norm)) return fail(CARDAN_ERR_ALIGN, "x_norm is not 16-byte aligned");
  if (!layers) return fail(CARDAN_ERR_NULL_PTR, "layers is NULL");
  for (int l = 0; l < n_layers; ++l)
    if ((rc = check_layer(shape, &layers[l], true))) {
      char msg[512];
      snprintf(msg, sizeof msg, "layer %d: %s", l, g_err);
      return fail(rc, "%s", msg);
    }
  const int base = F_ROUTE | F_GROUP | F_EXPERTS | (shape->r > 0 ? F_Z : 0);
  // every layer's plan has this layout (flags and bases change item counts only)
  const Plan P0 = make_plan(shape, B, 1, base | F_NORM_IN | F_SSQ_OUT);
  const StepBufs sb = step_bufs(P0);
  if ((rc = check_ws(P0, ws, ws_bytes))) return rc;
  if (ws_bytes < sb.total)
    return fail(CARDAN_ERR_WORKSPACE, "workspace of %zu bytes < required %zu", ws_bytes, sb.total);
  uint8_t* w = static_cast<uint8_t*>(ws);
  float* ybuf[2] = {reinterpret_cast<float*>(w + sb.o_y), reinterpret_cast<float*>(w + sb.o_y) + (size_t)B * shape->H};
  float* ssq[2] = {reinterpret_cast<float*>(w + sb.o_ssq),
                   reinterpret_cast<float*>(w + sb.o_ssq) + (size_t)B * combine_col_tiles(P0)};
  uint16_t* xbuf[2] = {reinterpret_cast<uint16_t*>(w + sb.o_x),
                       reinterpret_cast<uint16_t*>(w + sb.o_x) + (size_t)B * shape->H};
  const size_t BH = (size_t)B * shape->H, Bk = (size_t)B * shape->top_k;
  // Reading the next layer's shared tensors ahead (idle expert-kernel
  // workgroups) measured slower than not doing it, so it is off unless the
  // environment variable CARDAN_PREFETCH is "1".
  const char* pf_env = getenv("CARDAN_PREFETCH");
  const bool prefetch = pf_env && strcmp(pf_env, "1") == 0;
  for (int l = 0; l < n_layers; ++l) {
    const cardan_layer& L = layers[l];
    const bool last = l == n_layers - 1;
    const int z_sep = shape->r > 0 && L.U_up != L.U_gate;
    const int flags = base | (l > 0 ? F_NORM_IN : 0) | (last ? 0 : F_SSQ_OUT | (prefetch ? F_PREFETCH : 0));
    const Plan P = make_plan(shape, B, z_sep, flags);
    uint16_t* xin = l == 0 ? nullptr : (x_norm ? x_norm + (size_t)(l - 1) * BH : xbuf[l % 2]);
    Args A = args_for(&L, w);
    A.x = l == 0 ? x0 : xin;
    A.topk_idx = topk_idx + (size_t)l * Bk;
    A.topk_w = topk_w + (size_t)l * Bk;
    A.z_out = reinterpret_cast<float*>(w + P.o_z);
    A.y = last ? y : ybuf[l % 2];
    Chain C;
    memset(&C, 0, sizeof C);
    C.eps = eps;
    C.nssq = combine_col_tiles(P);
    if (l > 0) {
      C.y_in = ybuf[(l - 1) % 2];
      C.ssq_in = ssq[(l - 1) % 2];
      C.x_norm = xin;
    }
    if (!last) {
      C.ssq_out = ssq[l % 2];
      const cardan_layer& N = layers[l + 1];
      const size_t H = shape->H, E = shape->E, r = shape->r, book = (size_t)shape->K * shape->d * 2;
      const void* pf[kPrefetchTensors] = {N.router_w, N.U_gate, N.U_up != N.U_gate ? N.U_up : nullptr,
                                          N.B_down, N.cb_gate, N.cb_up, N.cb_down};
      const size_t nb[kPrefetchTensors] = {H * E * 2, H * r * 2, H * r * 2, r * H * 2, book, book, book};
      for (int j = 0; j < kPrefetchTensors; ++j) {
        C.pf[j] = nb[j] > 0 && nb[j] < 0x80000000ull ? pf[j] : nullptr;
        C.pf_bytes[j] = C.pf[j] ? (uint32_t)nb[j] : 0;
      }
    }
    if ((rc = run_layer(P, A, stream, &C))) return rc;
  }
  return CARDAN_OK;
}

int cardan_moe_layer_noalloc(const cardan_shape* shape, int32_t B, const cardan_bf16* x,
                             const cardan_layer* layer, float* y, int32_t* topk_idx, float* topk_w,
                             hipStream_t stream) {
  g_err[0] = 0;
  int rc = check_shape(shape, B);
  if (rc) return rc;
  REQ(x, "x");
  REQ(y, "y");
  REQ(topk_idx, "topk_idx");
  REQ(topk_w, "topk_w");
  if ((rc = check_layer(shape, layer, true))) return rc;
  const int z_sep = shape->r > 0 && layer->U_up != layer->U_gate;
  const int flags = F_ROUTE | F_GROUP | F_EXPERTS | (shape->r > 0 ? F_Z : 0);
  const Plan P = make_plan(shape, B, z_sep, flags);
  if (P.total > kScratchBytes)
    return fail(CARDAN_ERR_WORKSPACE, "layer needs %zu bytes of workspace, more than the %zu-byte scratch array",
                P.total, kScratchBytes);
  void* ws = nullptr;
  bool clear = false;
  if ((rc = scratch_for_call(P, stream, &ws, &clear))) return rc;
  if (clear) {
    hipError_t err = launch_zero(ws, P.o_rl, stream);
    if (err != hipSuccess) return hip_fail(err, "scratch clear launch");
  }
  uint8_t* w = static_cast<uint8_t*>(ws);
  Args A = args_for(layer, w);
  A.x = x;
  A.topk_idx = topk_idx;
  A.topk_w = topk_w;
  A.z_out = reinterpret_cast<float*>(w + P.o_z);
  A.y = y;
  return run_layer(P, A, stream);
}

int cardan_moe_layer_dense_down(const cardan_shape* shape, int32_t B, const cardan_bf16* x,
                                const cardan_layer* layer, const cardan_bf16* W_down, float* y,
                                int32_t* topk_idx, float* topk_w, void* ws, size_t ws_bytes,
                                hipStream_t stream) {
  g_err[0] = 0;
  int rc = check_shape(shape, B);
  if (rc) return rc;
  if ((rc = check_dense_size(shape))) return rc;
  REQ(x, "x");
  REQ(y, "y");
  REQ(topk_idx, "topk_idx");
  REQ(topk_w, "topk_w");
  REQ(W_down, "W_down");
  if ((rc = check_layer(shape, layer, true, false))) return rc;
  const int z_sep = shape->r > 0 && layer->U_up != layer->U_gate;
  const int flags = F_ROUTE | F_GROUP | F_EXPERTS | F_DN_DENSE | (shape->r > 0 ? F_Z : 0);
  const Plan P = make_plan(shape, B, z_sep, flags);
  if ((rc = check_ws(P, ws, ws_bytes))) return rc;
  uint8_t* w = static_cast<uint8_t*>(ws);
  Args A = args_for(layer, w);
  // the kernels read the dense down matrices through the down code pointer
  A.L.codes_down = reinterpret_cast<const uint8_t*>(W_down);
  A.L.cb_down = nullptr;
  A.L.A_down = nullptr;
  A.L.B_down = nullptr;
  A.x = x;
  A.topk_idx = topk_idx;
  A.topk_w = topk_w;
  A.z_out = reinterpret_cast<float*>(w + P.o_z);
  A.y = y;
  return run_layer(P, A, stream);
}

}  // extern "C"

namespace {
// the uncompressed layer; relu2: up-only experts (W_gate not read)
int dense_moe_layer(const cardan_shape* shape, int32_t B, const cardan_bf16* x, const cardan_dense_layer* layer,
                    float* y, int32_t* topk_idx, float* topk_w, void* ws, size_t ws_bytes, hipStream_t stream,
                    bool relu2) {
  if (!shape) return fail(CARDAN_ERR_NULL_PTR, "shape is NULL");
  cardan_shape s = *shape;  // only H, I, E and top_k describe a dense layer
  s.d = 8;
  s.K = 1;
  s.r = 0;
  int rc = check_shape(&s, B);
  if (rc) return rc;
  if ((rc = check_dense_size(&s))) return rc;
  REQ(x, "x");
  REQ(y, "y");
  REQ(topk_idx, "topk_idx");
  REQ(topk_w, "topk_w");
  if (!layer) return fail(CARDAN_ERR_NULL_PTR, "layer is NULL");
  REQ(layer->router_w, "router_w");
  if (layer->router_bias && (reinterpret_cast<uintptr_t>(layer->router_bias) & 3u))
    return fail(CARDAN_ERR_ALIGN, "router_bias is not 4-byte aligned");
  if (!relu2) REQ(layer->W_gate, "W_gate");
  REQ(layer->W_up, "W_up");
  REQ(layer->W_down, "W_down");
  const Plan P = make_plan(&s, B, 0, F_ROUTE | F_GROUP | F_EXPERTS | F_GU_DENSE | F_DN_DENSE | (relu2 ? F_UP_RELU2 : 0));
  if ((rc = check_ws(P, ws, ws_bytes))) return rc;
  // the kernels read the dense matrices through the code pointers
  cardan_layer L;
  memset(&L, 0, sizeof L);
  L.router_w = layer->router_w;
  L.router_bias = layer->router_bias;
  L.codes_gate = reinterpret_cast<const uint8_t*>(relu2 ? layer->W_up : layer->W_gate);
  L.codes_up = reinterpret_cast<const uint8_t*>(layer->W_up);
  L.codes_down = reinterpret_cast<const uint8_t*>(layer->W_down);
  Args A = args_for(&L, static_cast<uint8_t*>(ws));
  A.x = x;
  A.topk_idx = topk_idx;
  A.topk_w = topk_w;
  A.y = y;
  return run_layer(P, A, stream);
}
}  // namespace

extern "C" {

int cardan_dense_moe_layer(const cardan_shape* shape, int32_t B, const cardan_bf16* x,
                           const cardan_dense_layer* layer, float* y, int32_t* topk_idx, float* topk_w,
                           void* ws, size_t ws_bytes, hipStream_t stream) {
  g_err[0] = 0;
  return dense_moe_layer(shape, B, x, layer, y, topk_idx, topk_w, ws, ws_bytes, stream, false);
}

int cardan_dense_moe_layer_relu2(const cardan_shape* shape, int32_t B, const cardan_bf16* x,
                                 const cardan_dense_layer* layer, float* y, int32_t* topk_idx, float* topk_w,
                                 void* ws, size_t ws_bytes, hipStream_t stream) {
  g_err[0] = 0;
  return dense_moe_layer(shape, B, x, layer, y, topk_idx, topk_w, ws, ws_bytes, stream, true);
}

int cardan_rmsnorm_bf16(int32_t B, int32_t H, const float* y, float eps, cardan_bf16* x_next,
                        hipStream_t stream) {
  g_err[0] = 0;
  if (B < 1 || H < 1) return fail(CARDAN_ERR_BAD_SHAPE, "B=%d, H=%d must be positive", B, H);
  REQ(y, "y");
  REQ(x_next, "x_next");
  Timed tm(stream, CARDAN_KERNEL_RMSNORM);
  hipError_t e = launch_rmsnorm(stream, B, H, y, eps, x_next, tm.ev0, tm.ev1);
  if (e != hipSuccess) return hip_fail(e, "rmsnorm launch");
  tm.done();
  prof_next_call();
  return CARDAN_OK;
}

int cardan_profile_begin(int32_t max_calls) {
  g_err[0] = 0;
  if (max_calls < 1) return fail(CARDAN_ERR_BAD_SHAPE, "max_calls must be positive");
  const size_t need = (size_t)max_calls * CARDAN_PROFILE_KINDS * 2;
  while (g_prof.ev.size() < need) {
    hipEvent_t e;
    hipError_t err = hipEventCreate(&e);
    if (err != hipSuccess) return hip_fail(err, "hipEventCreate");
    g_prof.ev.push_back(e);
  }
  g_prof.used.assign((size_t)max_calls * CARDAN_PROFILE_KINDS, 0);
  g_prof.cap = max_calls;
  g_prof.calls = 0;
  g_prof.on = true;
  return CARDAN_OK;
}

int cardan_profile_end(float* ms_per_kind, int32_t* launches_per_kind) {
  g_err[0] = 0;
  if (!ms_per_kind || !launches_per_kind) return fail(CARDAN_ERR_NULL_PTR, "output is NULL");
  for (int k = 0; k < CARDAN_PROFILE_KINDS; ++k) {
    ms_per_kind[k] = 0.0f;
    launches_per_kind[k] = 0;
  }
  g_prof.on = false;
  for (int c = 0; c < g_prof.calls; ++c) {
    for (int k = 0; k < CARDAN_PROFILE_KINDS; ++k) {
      const size_t i = (size_t)c * CARDAN_PROFILE_KINDS + k;
      if (!g_prof.used[i]) continue;
      hipError_t err = hipEventSynchronize(g_prof.ev[2 * i + 1]);
      if (err != hipSuccess) return hip_fail(err, "hipEventSynchronize");
      float ms = 0.0f;
      err = hipEventElapsedTime(&ms, g_prof.ev[2 * i], g_prof.ev[2 * i + 1]);
      if (err != hipSuccess) return hip_fail(err, "hipEventElapsedTime");
      ms_per_kind[k] += ms;
      launches_per_kind[k] += 1;
    }
  }
  g_prof.calls = 0;
  return CARDAN_OK;
}

}  // extern "C"
