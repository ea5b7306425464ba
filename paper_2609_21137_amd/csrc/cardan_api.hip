// C ABI of libcardan.so: argument validation, launch planning, workspace
// layout and the kernel sequence of every entry point.
#include <hip/hip_runtime.h>

#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <vector>

#include "../../include/cardan.h"
#include "cardan_plan.h"

namespace cardan {
const void* route_kernel();
const void* expert_kernel(int d, int dnw, int mode, bool csk, bool xpre);
hipError_t launch_route(const Plan&, const Args&, int, size_t, hipStream_t, hipEvent_t, hipEvent_t);
hipError_t launch_expert(const Plan&, const Args&, int, size_t, hipStream_t, hipEvent_t, hipEvent_t);
hipError_t launch_route_reset(const Plan&, const Args&, hipStream_t);
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

size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }

int ceil_div(int a, int b) { return (a + b - 1) / b; }

int pow2_floor(double v) {
  int p = 1;
  while (p * 2 <= v) p *= 2;
  return p;
}

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

constexpr size_t kLdsBudget = 60 * 1024;  // operand staging limit when sizing the K splits
constexpr size_t kLdsMax = 96 * 1024;     // dynamic LDS limit of either kernel

int ks_max(int total, int splits) { return ceil_div(total, splits); }

// Largest x/z staging of a gate/up split (uint4 per token row).
int gateup_ld(int KSX, int KSZ, int ns, int ns_v) {
  int best = 0;
  for (int s = 0; s < ns; ++s) {
    int k0, k1;
    joint_split(s, ns, ns_v, KSX, KSZ, k0, k1);
    const int x = std::min(k1, KSX) - std::min(k0, KSX);
    const int z = std::max(k1, KSX) - std::max(k0, KSX);
    best = std::max(best, (x * 4 + 1) + (z * 8 + 1));
  }
  return best;
}

size_t round256(size_t v) { return (v + 255) & ~(size_t)255; }

// Dynamic LDS of k_route for a plan.
size_t lds_route(const Plan& P) {
  const int KSX = P.H / 32;
  size_t need = (size_t)kTokPass * kRowsRouter * (4 + 4 * 8);          // router chunk
  need = std::max(need, (size_t)kMaxE * 8 + kMaxK * (8 + 8 + 4 + 4) + (size_t)kWG * 8);  // select
  need = std::max(need, (size_t)(kMaxB * kMaxK + 2 * kMaxE + 4) * 4);   // grouping
  if (P.flags & F_Z)
    need = std::max(need, (size_t)4 * kTokPass * (ks_max(KSX, P.nch_z) * 4 + 1) * 16);
  return round256(need);
}

// Dynamic LDS of k_expert for a plan.
size_t lds_expert(const Plan& P) {
  const int KSX = P.H / 32, KSZ = ceil_div(P.r, 32), KSD = P.I / 32;
  size_t need = (size_t)P.nt_max * gateup_ld(KSX, KSZ, P.ns, P.ns_v) * 16;
  // down: p operand rows + a reduction area of 2 float4 per thread
  const int ksd = std::max(ks_max(KSD, P.nsd), ks_max(KSD, P.nsdl));
  need = std::max(need, (size_t)P.nt_max * (ksd * 8 + 1) * 16 + kWG * 2 * 16);
  need = std::max(need, combine_lds(P) + ((P.flags & F_CB_SPLITK) ? kSplitKRed : 0));
  return round256(need);
}

// Launch plan, item counts and workspace layout; depends only on
// (shape, B, z_sep, flags). F_GU_DENSE plans take r = 0.
Plan make_plan(const cardan_shape* s, int B, int z_sep, int flags) {
  Plan P;
  memset(&P, 0, sizeof P);
  P.H = s->H; P.I = s->I; P.E = s->E; P.k = s->top_k; P.d = s->d; P.K = s->K; P.r = s->r;
  P.B = B;
  P.flags = flags;
  const int mode = expert_mode(P);
  if (mode == 2) P.r = 0;
  P.S = B * P.k;
  P.max_act = P.E < P.S ? P.E : P.S;
  P.nch_r = P.H / kRowsRouter;
  P.n_eg = ceil_div(P.E, 64);
  P.z_sep = z_sep;
  P.nt_max = std::min(B, kTokPass);
  // combine tiles of up to B/8 tokens: eight per column group at large
  // batches, so the final gather is spread over more workgroups
  P.tpc = std::min(kTokPass, ceil_div(B, 8));
  const int KSX = P.H / 32, KSZ = ceil_div(P.r, 32), KSD = P.I / 32;
  P.nch_z = std::max(1, KSX / 2);                  // two K-steps of U per z unit
  // Tile sizes: the expected active experts' weight bytes spread over a
  // nominal grid of 512 workgroups (2 per CU), kept between 16 and 64 KB per
  // tile, so small batches run every tile in one round and large ones stream
  // long tiles. Bytes per tile: a gate/up (expert, projection, 256 columns)
  // holds 256 (H/d) code bytes and 256 r * 2 coefficient bytes; a VQ down
  // (expert, 256 columns) 256 I/d; a low-rank down (expert, <= 256 ranks)
  // min(r, 256) I * 2. Dense bf16 weights: 256 H * 2 per gate/up and
  // 256 I * 2 per down (expert, 256 columns).
  const double exp_act = fmax(1.0, P.E * (1.0 - pow(1.0 - (double)P.k / P.E, (double)B)));
  const double gu_expert = mode == 2 ? 2.0 * P.H * P.I * 2 : 2.0 * P.H * P.I / P.d + 2.0 * P.I * P.r * 2;
  const double dn_expert = mode >= 1 ? (double)P.I * P.H * 2 : (double)P.H * P.I / P.d + (double)P.I * P.r * 2;
  const double per_expert = gu_expert + dn_expert;
  // A VQ down K-step costs twice a gate/up one (p enters as hi + lo), so its
  // bytes count double. While the expected items exceed the nominal grid
  // the tile grows (small batches then run in one round).
  // Dense-weight forms stream 4-16x the bytes: once the nominal tile passes
  // two 128 KB tiles, their tiles grow to 512 KB (a tile's set-up and pipeline
  // drain then recur less often; measured 154 -> 143 us for the dense layer
  // at batch 16, while small batches keep the one-round 128 KB tiles).
  const double nominal = exp_act * per_expert / 512.0;
  const double tile_max = (mode != 0 && nominal > 2 * 128.0 * 1024 ? 512.0 : 128.0) * 1024;
  double tile = fmin(tile_max, fmax(16.0 * 1024, nominal));
  auto splits = [&](double bytes, int max_splits) {
    return std::max(1, std::min(max_splits, (int)lround(bytes / tile)));
  };
  P.ncg = ceil_div(P.I, kColsPerGroup);
  P.ncgh = ceil_div(P.H, kColsPerGroup);
  P.ncgr = mode == 0 ? ceil_div(P.r, kColsPerGroup) : 0;  // low-rank down column groups
  for (;;) {
    // code (or dense) splits and low-rank splits of a gate/up (expert, 256 columns)
    const double code_bytes = mode == 2 ? 256.0 * P.H * 2 : 256.0 * (KSX * 32 / P.d);
    const double lr_bytes = 256.0 * P.r * 2;
    if (tile >= 0.75 * (code_bytes + lr_bytes)) {
      P.ns_v = P.ns = 1;  // one tile holds the whole joint axis
    } else {
      P.ns_v = splits(code_bytes, KSX);
      P.ns = P.ns_v + (KSZ > 0 ? splits(lr_bytes, KSZ) : 0);
    }
    P.nsd = mode >= 1 ? splits(256.0 * P.I * 2, KSD) : splits(2.0 * 256.0 * P.I / P.d, KSD);
    P.nsdl = P.r > 0 ? splits((double)std::min(P.r, kColsPerGroup) * P.I * 2, KSD) : 1;
    const double items = exp_act * (2.0 * P.ncg * P.ns + P.ncgh * P.nsd + P.ncgr * P.nsdl);
    if (items <= 512.0 || tile >= tile_max) break;
    tile *= 1.05;
  }
  // Latency shape: while the item count fits the nominal grid (with a
  // quarter more for a short second round), code splits of at most L K-steps
  // for the smallest L in {1, 2, 4} x the pipeline depth, with low-rank splits
  // of kPdDense steps where they fit too, else as many as the byte balance
  // gave. At large r the byte balance alone leaves one code split of H/32
  // steps, a chain of H/32/kPdVq dependent pipeline refills (r = 384 at B=1:
  // 35.7 us).
  if (P.ns > 1) {
    const int pd = mode == 2 ? kPdDenseW : kPdVq;
    const int nl_fine = KSZ > 0 ? ceil_div(KSZ, kPdDense) : 0, nl_keep = P.ns - P.ns_v;
    bool done = false;
    for (int mult = 1; mult <= 4 && !done; mult *= 2) {
      const int nv = std::max(P.ns_v, ceil_div(KSX, pd * mult));
      for (const int nl : {nl_fine, nl_keep}) {
        const double items = exp_act * (2.0 * P.ncg * (nv + nl) + P.ncgh * P.nsd + P.ncgr * P.nsdl);
        if (items <= 1.25 * 512.0) {
          P.ns_v = nv;
          P.ns = nv + nl;
          done = true;
          break;
        }
      }
    }
  }
  // token rows staged per pass: halve (down to 4) before splitting K further
  // to fit the operand staging into LDS; experts with more tokens than one
  // pass stream their weights again per pass (rare at these sizes)
  while (P.nt_max > 4 && (size_t)P.nt_max * gateup_ld(KSX, KSZ, P.ns, P.ns_v) * 16 > kLdsBudget)
    P.nt_max = (P.nt_max + 1) / 2;
  while (P.ns_v < KSX && (size_t)P.nt_max * gateup_ld(KSX, KSZ, P.ns, P.ns_v) * 16 > kLdsBudget) {
    if (P.ns == P.ns_v && KSZ > 0) ++P.ns;  // give the low-rank steps their own split first
    else {
      ++P.ns_v;
      ++P.ns;
    }
  }
  auto down_fits = [&](int n) {
    return (size_t)P.nt_max * (ks_max(KSD, n) * 8 + 1) * 16 + kWG * 2 * 16 <= kLdsBudget;
  };
  // low-rank down tiles cover at least kLrDownSteps K-steps (their weights
  // load while they wait): fewer partials of u_e for the combine to sum
  P.nsdl = std::min(P.nsdl, ceil_div(KSD, kLrDownSteps));
  while (P.nsd < KSD && !down_fits(P.nsd)) ++P.nsd;
  while (P.nsdl < KSD && !down_fits(P.nsdl)) ++P.nsdl;
  // Items for more than two rounds of the nominal grid (throughput-bound):
  // VQ down tiles over two column groups, so that each K-step's activation
  // reads serve twice the columns and the down tiles take half the
  // workgroup slots (fewer rounds, longer tiles)
  const double items_all = exp_act * (2.0 * P.ncg * P.ns + P.ncgh * P.nsd + P.ncgr * P.nsdl);
  if (mode == 0 && items_all > 2 * 512.0 && P.ncgh > 1 && P.d == 8) P.flags |= F_DN_WIDE;
  // Small batches at ranks above 128: B^T u streams more of B than a
  // combine tile primes before its wait, so the tiles shrink to 64 columns
  // with the ranks split over their four waves (each wave's share primed).
  if (mode == 0 && P.r > 128 && B <= 4) P.flags |= F_CB_SPLITK;
  P.n_cb = P.ncgh * ceil_div(B, P.tpc) * ((P.flags & F_CB_SPLITK) ? 4 : 1);
  // Batch 1: every gate/up tile's operands are the one token's x and z rows,
  // so each workgroup stages them once while it builds its routing tables
  if (mode == 0 && B == 1 && P.H <= 8 * kXpreXGroups) P.flags |= F_XPRE;

  const int z_units = (z_sep ? 2 : 1) * ceil_div(P.r, 64) * P.nch_z;
  P.n_rc = (flags & F_ROUTE) ? P.nch_r * P.n_eg * ceil_div(B, kRouterTok) : 0;
  P.n_zc = (flags & F_Z) ? ceil_div(z_units, 4) : 0;
  P.n_sel = (flags & F_ROUTE) ? B : 0;
  P.n_zr = (flags & F_Z) ? ceil_div(2 * B * P.r, kWG) : 0;
  P.n_pre = P.n_rc + P.n_zc + P.n_sel + P.n_zr;

  // Counters first, at offsets that depend only on H, I and E (not on B,
  // r or the expert-weight form): a call leaves its expert ticks set until
  // the next call's k_route clears them, so every call on a workspace must
  // find them at the same place.
  P.n_rc_flags = P.nch_r * P.n_eg * ceil_div(kMaxB, kRouterTok);
  P.n_zc_flags = ceil_div(2 * ceil_div(kMaxR, 64) * P.nch_z, 4);
  size_t o = 0;
  P.o_ctr = o; o = align256(o + (size_t)C_NUM * kCtrStride * 4);
  P.o_rc_flag = o; o = align256(o + (size_t)P.n_rc_flags * kTickPad * 4);
  P.o_zc_flag = o; o = align256(o + (size_t)P.n_zc_flags * kTickPad * 4);
  P.o_gu_tick = o; o = align256(o + (size_t)P.E * ceil_div(P.I, kColsPerGroup) * kTickPad * 4);
  P.o_dn_done = o; o = align256(o + (size_t)P.E * (ceil_div(P.H, kColsPerGroup) + 1) * kTickPad * 4);
  P.o_rl = o; o = align256(o + (size_t)P.nch_r * B * P.E * 8);
  P.o_zp = o; o = align256(o + (size_t)2 * P.nch_z * B * P.r * 4);
  P.o_z = o; o = align256(o + (size_t)2 * B * P.r * 4);
  P.o_gu = o; o = align256(o + (size_t)P.S * 2 * P.ns * P.I * 4);
  P.o_dn = o; o = align256(o + (size_t)P.nsd * P.S * P.H * 4);
  P.o_uap = o; o = align256(o + (size_t)P.nsdl * P.S * P.r * 4);
  P.total = o;
  P.lds_route = lds_route(P);
  // routing tables: active-expert records and four per-slot arrays
  P.lds_routing = round256((size_t)P.max_act * 16 + (size_t)4 * P.S * 4);
  // item LDS, also the grouping scratch at the start of the kernel
  const size_t group_scratch = round256((size_t)2 * P.S * 4 + (size_t)4 * P.E * 4 + 32);
  P.lds_expert = P.lds_routing + std::max(lds_expert(P), group_scratch) + ((P.flags & F_XPRE) ? kXpreBytes : 0);
  // the large-batch kernel holds kBookCopies code books in static LDS: only
  // where two workgroups still fit a CU (80 KB each)
  if ((P.flags & F_DN_WIDE) && P.lds_expert + (size_t)256 * kBookCopies * 16 + 512 > 80 * 1024)
    P.flags &= ~F_DN_WIDE;
  return P;
}

// Co-resident workgroups of a kernel on the current device for a given
// dynamic LDS size (cached per device, kernel and LDS size).
int resident_grid(const void* fn, size_t lds, hipError_t* err) {
  struct Entry {
    int dev;
    const void* fn;
    size_t lds;
    int grid;
  };
  static Entry cache[64];
  static int n_cache = 0;
  int dev = 0;
  *err = hipGetDevice(&dev);
  if (*err != hipSuccess) return 0;
  for (int i = 0; i < n_cache; ++i)
    if (cache[i].dev == dev && cache[i].fn == fn && cache[i].lds == lds) return cache[i].grid;
  int cus = 0, per_cu = 0;
  *err = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (*err != hipSuccess) return 0;
  *err = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, kWG, lds);
  if (*err != hipSuccess) return 0;
  const int g = std::max(1, cus * per_cu);
  if (n_cache < 64) cache[n_cache++] = {dev, fn, lds, g};
  return g;
}

int check_ws(const Plan& P, const void* ws, size_t ws_bytes) {
  if (!ws) return fail(CARDAN_ERR_NULL_PTR, "workspace is NULL");
  if (misaligned(ws)) return fail(CARDAN_ERR_ALIGN, "workspace is not 16-byte aligned");
  if (ws_bytes < P.total)
    return fail(CARDAN_ERR_WORKSPACE, "workspace of %zu bytes < required %zu", ws_bytes, P.total);
  return CARDAN_OK;
}

#define REQ(p, name)                                                                  \
  do {                                                                                \
    if (!(p)) return fail(CARDAN_ERR_NULL_PTR, "%s is NULL", name);                   \
    if (misaligned(p)) return fail(CARDAN_ERR_ALIGN, "%s is not 16-byte aligned", name); \
  } while (0)

// need_down: the compressed down projection (code book, codes, A, B) is used
int check_layer(const cardan_shape* s, const cardan_layer* L, bool need_router, bool need_down = true) {
  if (!L) return fail(CARDAN_ERR_NULL_PTR, "layer is NULL");
  if (need_router) REQ(L->router_w, "router_w");
  if (L->router_bias && (reinterpret_cast<uintptr_t>(L->router_bias) & 3u))
    return fail(CARDAN_ERR_ALIGN, "router_bias is not 4-byte aligned");
  REQ(L->cb_gate, "cb_gate");
  REQ(L->cb_up, "cb_up");
  REQ(L->codes_gate, "codes_gate");
  REQ(L->codes_up, "codes_up");
  if (need_down) {
    REQ(L->cb_down, "cb_down");
    REQ(L->codes_down, "codes_down");
  }
  if (s->r > 0) {
    REQ(L->U_gate, "U_gate");
    REQ(L->U_up, "U_up");
    REQ(L->V_gate, "V_gate");
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
int run_layer(const Plan& P, const Args& A, hipStream_t stream) {
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
    err = launch_route(P, A, std::max(1, std::min(cap, P.n_pre)), P.lds_route, stream, tm.ev0, tm.ev1);
    if (err != hipSuccess) return hip_fail(err, "k_route launch");
    tm.done();
    if (!(P.flags & F_EXPERTS)) {  // k_expert would clear these counters
      err = launch_route_reset(P, A, stream);
      if (err != hipSuccess) return hip_fail(err, "k_route_reset launch");
    }
  }
  if (P.flags & F_EXPERTS) {
    const int cap = resident_grid(expert_kernel(P.d, dn_width(P), expert_mode(P), (P.flags & F_CB_SPLITK) != 0,
                                                (P.flags & F_XPRE) != 0),
                                  P.lds_expert, &err);
    if (cap <= 0) return hip_fail(err, "occupancy query");
    Timed tm(stream, CARDAN_KERNEL_EXPERT);
    err = launch_expert(P, A, cap, P.lds_expert, stream, tm.ev0, tm.ev1);
    if (err != hipSuccess) return hip_fail(err, "k_expert launch");
    tm.done();
  }
  prof_next_call();
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
  // and every expert-weight form (compressed, dense down, all dense)
  size_t need = 0;
  const int all = F_ROUTE | F_Z | F_GROUP | F_EXPERTS;
  for (int b = 1; b <= B; ++b)
    for (int form : {0, (int)F_DN_DENSE, F_DN_DENSE | F_GU_DENSE})
      need = std::max(need, make_plan(shape, b, 1, all | form).total);
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
  const int flags = F_ROUTE | F_GROUP | F_EXPERTS | (shape->r > 0 ? F_Z : 0);
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

int cardan_dense_moe_layer(const cardan_shape* shape, int32_t B, const cardan_bf16* x,
                           const cardan_dense_layer* layer, float* y, int32_t* topk_idx, float* topk_w,
                           void* ws, size_t ws_bytes, hipStream_t stream) {
  g_err[0] = 0;
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
  REQ(layer->W_gate, "W_gate");
  REQ(layer->W_up, "W_up");
  REQ(layer->W_down, "W_down");
  const Plan P = make_plan(&s, B, 0, F_ROUTE | F_GROUP | F_EXPERTS | F_GU_DENSE | F_DN_DENSE);
  if ((rc = check_ws(P, ws, ws_bytes))) return rc;
  // the kernels read the dense matrices through the code pointers
  cardan_layer L;
  memset(&L, 0, sizeof L);
  L.router_w = layer->router_w;
  L.router_bias = layer->router_bias;
  L.codes_gate = reinterpret_cast<const uint8_t*>(layer->W_gate);
  L.codes_up = reinterpret_cast<const uint8_t*>(layer->W_up);
  L.codes_down = reinterpret_cast<const uint8_t*>(layer->W_down);
  Args A = args_for(&L, static_cast<uint8_t*>(ws));
  A.x = x;
  A.topk_idx = topk_idx;
  A.topk_w = topk_w;
  A.y = y;
  return run_layer(P, A, stream);
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
