// HIP kernels for gfx950 (MI355X) of the compressed-MoE decode layer.
//
// k_layer is a persistent kernel that runs a whole layer call (paper Sec. 2.1
// and Sec. 4) as an ordered list of work items (see cardan_plan.h):
//   routing-independent work first -- router partial logits in float64 and
//   the shared projections z = U^T x (Sec. 4.2: computed once per token);
//   then per-token top-k and gating, the grouping of (token, expert) slots by
//   expert, and the expert tiles, which stream each active expert's codes
//   and coefficients from HBM exactly once per step.
// Down-projection tiles issue their HBM loads before they wait for the gate/up
// result of their expert, so weight traffic keeps flowing across the
// gate/up -> down dependency (the GPU form of the paper's overlap windows,
// Sec. 4.1).
//
// Every contraction runs on the matrix cores (v_mfma_f32_16x16x32_bf16) with
// the token slots of an expert as the M dimension: for the VQ part each lane
// decodes one uint8 code into its code word (d bf16 values from the LDS copy
// of the code book) and that code word IS the lane's slice of the weight
// operand, so decoded weights never leave registers; the low-rank factors
// enter the same accumulators as dense bf16 operands, which makes the VQ sum
// and V^T z one float32 accumulation before the activation (Sec. 4.2, joint
// accumulation).
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <math.h>
#include <stdint.h>

#include "cardan_plan.h"

namespace cardan {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr unsigned kSpinLimit = 1u << 24;  // polls before a wait gives up (seconds)

__device__ __forceinline__ float bf(uint32_t b) { return __uint_as_float(b << 16); }

__device__ __forceinline__ uint32_t rne_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return 0x7fc0u;
  u += 0x7fffu + ((u >> 16) & 1u);
  return u >> 16;
}

__device__ __forceinline__ f32x4 mfma_bf16(uint4 a, uint4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

// Weight streams read through buffer resources: a load whose offset is past
// the resource's size returns zeros without a memory access, so every
// pipeline slot is always issued (a static number of loads in flight, hence
// exact waits) while steps past the end cost no traffic.
typedef __amdgpu_buffer_rsrc_t rsrc_t;
constexpr uint32_t kOob = 0x80000000u;  // an offset past every resource

__device__ __forceinline__ rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}

__device__ __forceinline__ int* ctr(const Args& A, int i) {
  return reinterpret_cast<int*>(A.ws) + i * kCtrStride;
}

template <typename T>
__device__ __forceinline__ T* wsp(const Args& A, size_t off) {
  return reinterpret_cast<T*>(A.ws + off);
}

// ---- optional item timeline (debug builds with CARDAN_TRACE) --------------
// Records per work item the device real-time clock (100 MHz, shared by all
// CUs) at start, after its dependency wait and at end, into workspace bytes
// past the normal layout. Compiled out of the library by default.
#ifdef CARDAN_TRACE
__shared__ unsigned long long s_trace[5];  // wait end, then up to 4 phase marks
__device__ __forceinline__ unsigned long long rt_clock() { return __builtin_amdgcn_s_memrealtime(); }
__device__ __forceinline__ void trace_wait_done() {
  if (threadIdx.x == 0) s_trace[0] = rt_clock();
}
__device__ __forceinline__ void trace_mark(int i) {
  if (threadIdx.x == 0) s_trace[1 + i] = rt_clock();
}
struct ItemTrace {
  unsigned long long t0, c0;
  __device__ __forceinline__ ItemTrace() : t0(rt_clock()), c0(__builtin_amdgcn_s_memtime()) {
    if (threadIdx.x < 5) s_trace[threadIdx.x] = 0;
  }
  __device__ __forceinline__ void done(const Args& A, const Plan& P, int slot, int kind) {
    if (threadIdx.x != 0) return;
    unsigned long long* rec = reinterpret_cast<unsigned long long*>(A.ws + P.total) + 10 * (size_t)slot;
    rec[0] = ((unsigned long long)kind << 48) | ((unsigned long long)blockIdx.x << 24) | (unsigned)slot;
    rec[1] = t0;
    rec[2] = s_trace[0];
    rec[3] = rt_clock();
    for (int i = 0; i < 4; ++i) rec[4 + i] = s_trace[1 + i];
    rec[8] = __builtin_amdgcn_s_memtime() - c0;  // core clock cycles of the item
    rec[9] = 0;
  }
};
#else
__device__ __forceinline__ void trace_wait_done() {}
__device__ __forceinline__ void trace_mark(int) {}
struct ItemTrace {
  __device__ __forceinline__ void done(const Args&, const Plan&, int, int) {}
};
#endif

// ---- cross-workgroup communication ------------------------------------------
// Data handed from one workgroup to another inside a kernel is written with
// device-scope stores and read with device-scope loads (sc1: coherent across
// the separate L2 caches of the XCDs), so no cache writeback or invalidation
// is ever issued; a producer only drains its own stores before it signals.
// Counters and flags are zeroed by the other kernel of the call (kernel
// boundaries order that), so every signal is a single relaxed atomic.
__device__ __forceinline__ void st_dev(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_dev(double* p, double v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_dev(int* p, int v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float ld_dev(const float* p) {
  return __hip_atomic_load(const_cast<float*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ double ld_dev(const double* p) {
  return __hip_atomic_load(const_cast<double*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ int ld_dev(const int* p) {
  return __hip_atomic_load(const_cast<int*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Orders this wave's LDS writes before its later LDS reads by other lanes
// (a wave executes its LDS operations in order; this keeps the compiler from
// moving them across each other).
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Waits for this wave's outstanding memory operations (s_waitcnt vmcnt(0)).
__device__ __forceinline__ void drain_stores() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// One arrival on counter c once every wave's stores have completed.
__device__ __forceinline__ void publish(int* c) {
  drain_stores();
  __syncthreads();
  if (threadIdx.x == 0) __hip_atomic_fetch_add(c, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Sets flag f once every wave's stores have completed.
__device__ __forceinline__ void set_flag(int* f) {
  drain_stores();
  __syncthreads();
  if (threadIdx.x == 0) st_dev(f, 1);
}

// Waits until cond(i) holds for every i in [0, n) (threads test in parallel).
// Bounded: on timeout the status counter is raised and the caller proceeds,
// so the grid always drains.
template <typename F>
__device__ __forceinline__ void wait_all(const Args& A, int n, F cond) {
  unsigned it = 0;
  for (;;) {
    bool mine = true;
    for (int i = threadIdx.x; i < n; i += kWG) mine = mine && cond(i);
    if (__syncthreads_and(mine)) {
      trace_wait_done();
      break;
    }
    __builtin_amdgcn_s_sleep(4);
    if (++it > kSpinLimit) {
      if (threadIdx.x == 0) atomicAdd(ctr(A, C_ERR), 1);
      break;
    }
  }
}

// Inclusive prefix sum across a wave64 with DPP row shifts and row
// broadcasts (lanes without a source add the 0 `old` operand).
__device__ __forceinline__ int wave_inclusive_scan(int x) {
  x += __builtin_amdgcn_update_dpp(0, x, 0x111, 0xF, 0xF, false);  // row_shr:1
  x += __builtin_amdgcn_update_dpp(0, x, 0x112, 0xF, 0xF, false);  // row_shr:2
  x += __builtin_amdgcn_update_dpp(0, x, 0x114, 0xF, 0xF, false);  // row_shr:4
  x += __builtin_amdgcn_update_dpp(0, x, 0x118, 0xF, 0xF, false);  // row_shr:8
  x += __builtin_amdgcn_update_dpp(0, x, 0x142, 0xA, 0xF, false);  // row_bcast:15 into rows 1, 3
  x += __builtin_amdgcn_update_dpp(0, x, 0x143, 0xC, 0xF, false);  // row_bcast:31 into rows 2, 3
  return x;
}

// The same DPP lane moves on a double (both halves; lanes without a source
// read +0).
template <int CTRL, int ROWS>
__device__ __forceinline__ double dpp_f64(double x) {
  const long long v = __double_as_longlong(x);
  const int lo = __builtin_amdgcn_update_dpp(0, (int)v, CTRL, ROWS, 0xF, false);
  const int hi = __builtin_amdgcn_update_dpp(0, (int)(v >> 32), CTRL, ROWS, 0xF, false);
  return __longlong_as_double(((long long)hi << 32) | (unsigned)lo);
}

// Sum of x over the wave, in every lane (a fixed tree: the same rounding on
// every call).
__device__ __forceinline__ double wave_sum(double x) {
  x += dpp_f64<0x111, 0xF>(x);
  x += dpp_f64<0x112, 0xF>(x);
  x += dpp_f64<0x114, 0xF>(x);
  x += dpp_f64<0x118, 0xF>(x);
  x += dpp_f64<0x142, 0xA>(x);
  x += dpp_f64<0x143, 0xC>(x);
  const long long v = __double_as_longlong(x);
  const int lo = __builtin_amdgcn_readlane((int)v, 63), hi = __builtin_amdgcn_readlane((int)(v >> 32), 63);
  return __longlong_as_double(((long long)hi << 32) | (unsigned)lo);
}

// Sum of a float over the wave, in every lane (the same fixed tree; all
// lanes active).
__device__ __forceinline__ float wave_sum(float x) {
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x111, 0xF, 0xF, false));
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x112, 0xF, 0xF, false));
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x114, 0xF, 0xF, false));
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x118, 0xF, 0xF, false));
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x142, 0xA, 0xF, false));
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x143, 0xC, 0xF, false));
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 63));
}

// x of lane 0 (all lanes active).
__device__ __forceinline__ double lane0(double x) {
  const long long v = __double_as_longlong(x);
  const int lo = __builtin_amdgcn_readfirstlane((int)v), hi = __builtin_amdgcn_readfirstlane((int)(v >> 32));
  return __longlong_as_double(((long long)hi << 32) | (unsigned)lo);
}

// Exclusive prefix sum of arr[0..n) (n <= 4 * kWG) in place; returns the total.
__device__ int block_exclusive_scan(int* arr, int n, int* tmp4) {
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int base = tid * 4;
  int v[4], s = 0;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    v[j] = (base + j < n) ? arr[base + j] : 0;
    s += v[j];
  }
  const int incl = wave_inclusive_scan(s);
  if (lane == 63) tmp4[w] = incl;
  __syncthreads();
  int pre = 0;
  for (int i = 0; i < w; ++i) pre += tmp4[i];
  const int total = tmp4[0] + tmp4[1] + tmp4[2] + tmp4[3];
  int ex = pre + incl - s;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    if (base + j < n) arr[base + j] = ex;
    ex += v[j];
  }
  __syncthreads();
  return total;
}

// 1 / rms of token t of the previous layer's output (stacked decode step):
// its partial sums of squares added in column-tile order, the same value in
// every item that normalises the token.
__device__ __forceinline__ float norm_inv(const Plan& P, const Chain& C, int t) {
  const float* q = C.ssq_in + (size_t)t * C.nssq;
  float s = 0.0f;
  for (int i = 0; i < C.nssq; ++i) s += q[i];
  return 1.0f / sqrtf(s / (float)P.H + C.eps);
}

// Router chunk (c, g, tb): partial logits over hidden rows [R c, R c + R)
// (R = kRowsRouter) for experts [64g, 64g + 64) of tokens [4tb, 4tb + 4).
// Lane l of wave w owns expert 64g + l and rows R c + (R/4) w .. + R/4 (rows
// past H read zeros; all of its weights are loaded up front); float64 FMAs of
// exact bf16 products in row order per token, in groups of 16 rows, then the
// four waves' partials are added in wave order through LDS.
__device__ void item_router_chunk(const Plan& P, const Args& A, const Chain& C, int item, int c, int g, int tb,
                                  uint8_t* smem) {
  constexpr int RW = kRowsRouter / 4;  // rows per wave
  static_assert(RW % 16 == 0, "rows per wave in groups of 16");
  float* xs = reinterpret_cast<float*>(smem);                                     // [4][R]
  double* part = reinterpret_cast<double*>(smem + kRouterTok * kRowsRouter * 4);  // [4][4][64]
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int E = P.E, H = P.H, B = P.B, h0 = c * kRowsRouter;
  const int e = min(g * 64 + lane, E - 1);  // lanes past E compute a copy that is never stored
  const rsrc_t wr = make_rsrc(A.L.router_w, (uint32_t)H * E * 2);
  uint32_t wv[RW];
#pragma unroll
  for (int i = 0; i < RW; ++i) {
    const int h = h0 + RW * w + i;
    wv[i] = __builtin_amdgcn_raw_buffer_load_b16(wr, h < H ? (uint32_t)((h * E + e) * 2) : kOob, 0, 0);
  }
  double* rl = wsp<double>(A, P.o_rl);
  const int tg = tb * kRouterTok, nt = min(kRouterTok, B - tg);
  if (P.flags & F_NORM_IN) {
    // x = bf16(y * inv_rms) of the previous layer's output; items of expert
    // group 0 also write it for the expert kernel. The y values load
    // together with the partial sums behind inv_rms.
    constexpr int NI = (kRouterTok * kRowsRouter + kWG - 1) / kWG;  // inputs per thread
    float* sinv = reinterpret_cast<float*>(part + 4 * kRouterTok * 64);  // [4]
    float yv[NI];
#pragma unroll
    for (int u = 0; u < NI; ++u) {
      const int i = tid + u * kWG, t = i / kRowsRouter, h = i % kRowsRouter;
      yv[u] = t < nt && h0 + h < H ? C.y_in[(size_t)(tg + t) * H + h0 + h] : 0.0f;
    }
    if (tid < nt) sinv[tid] = norm_inv(P, C, tg + tid);
    __syncthreads();
#pragma unroll
    for (int u = 0; u < NI; ++u) {
      const int i = tid + u * kWG, t = i / kRowsRouter, h = i % kRowsRouter;
      if (t < nt) {
        float v = 0.0f;
        if (h0 + h < H) {
          const uint32_t b = rne_bf16(yv[u] * sinv[t]);
          v = bf(b);
          if (g == 0) C.x_norm[(size_t)(tg + t) * H + h0 + h] = (uint16_t)b;
        }
        xs[i] = v;
      }
    }
  } else {
    for (int i = tid; i < nt * kRowsRouter; i += kWG) {
      const int t = i / kRowsRouter, h = i % kRowsRouter;
      xs[i] = h0 + h < H ? bf(A.x[(size_t)(tg + t) * H + h0 + h]) : 0.0f;
    }
  }
  __syncthreads();
  trace_mark(0);
  for (int t = 0; t < nt; ++t) {
    // the wave's inputs of token t: the same LDS words for every lane
    const float4* xr = reinterpret_cast<const float4*>(xs + t * kRowsRouter + RW * w);
    double a0 = 0.0, a1 = 0.0, a2 = 0.0, a3 = 0.0;
#pragma unroll
    for (int q = 0; q < RW / 4; ++q) {
      const float4 xq = xr[q];
      a0 = fma((double)bf(wv[4 * q + 0]), (double)xq.x, a0);
      a1 = fma((double)bf(wv[4 * q + 1]), (double)xq.y, a1);
      a2 = fma((double)bf(wv[4 * q + 2]), (double)xq.z, a2);
      a3 = fma((double)bf(wv[4 * q + 3]), (double)xq.w, a3);
    }
    part[(w * kRouterTok + t) * 64 + lane] = (a0 + a1) + (a2 + a3);
  }
  __syncthreads();
  trace_mark(1);
  for (int i = tid; i < nt * 64; i += kWG) {
    const int t = i >> 6, el = i & 63;
    if (g * 64 + el < E) {
      const double v = (part[(0 * kRouterTok + t) * 64 + el] + part[(1 * kRouterTok + t) * 64 + el]) +
                       (part[(2 * kRouterTok + t) * 64 + el] + part[(3 * kRouterTok + t) * 64 + el]);
      st_dev(rl + ((size_t)c * B + tg + t) * E + g * 64 + el, v);
    }
  }
  trace_mark(2);
  set_flag(wsp<int>(A, P.o_rc_flag) + item * kTickPad);
}

// Routing tables of a call in LDS. Every workgroup of k_expert rebuilds them
// from the B*k selections; the construction is deterministic, so all
// workgroups agree on every slot number.
struct RouteTab {
  const int4* act;       // [nact] (expert, first slot, slot count, 0), experts ascending
  const int* slot_tok;   // [S] token of each slot
  const float* slot_w;   // [S] gating weight of each slot
  const int* slot_e;     // [S] expert of each slot
  const int* tok_slot;   // [S] slot of selection (t, j), -1 if the expert is invalid
  int nact;
};

// Groups the B*k selections by expert into LDS (`tab`, route_lds_bytes):
// per-expert slot ranges in (token, j) order, the ascending list of active
// experts, slot -> token / weight / expert and (token, j) -> slot. `scratch`
// is item LDS, free before the first expert item. Selections come from the
// routing kernel of the same call or from the caller, both complete before
// this kernel starts. `distinct`: no token selects an expert twice (top-k
// output), so a slot's rank among its expert's slots comes from a token mask.
__device__ RouteTab build_routing(const Plan& P, const int32_t* idx, const float* wts, uint8_t* tab,
                                  uint8_t* scratch, bool distinct) {
  const int tid = threadIdx.x, E = P.E, S = P.S, k = P.k;
  int4* act = reinterpret_cast<int4*>(tab);
  int* slot_tok = reinterpret_cast<int*>(act + P.max_act);
  float* slot_w = reinterpret_cast<float*>(slot_tok + S);
  int* slot_e = reinterpret_cast<int*>(slot_w + S);
  int* tok_slot = slot_e + S;
  int* s_idx = reinterpret_cast<int*>(scratch);            // [S]
  float* s_w = reinterpret_cast<float*>(s_idx + S);        // [S]
  int* s_cnt = reinterpret_cast<int*>(s_w + S);            // [E] count | active << 16
  unsigned* s_mask = reinterpret_cast<unsigned*>(s_cnt + E);  // [E][2] tokens of each expert
  int* s_tmp = reinterpret_cast<int*>(s_mask + 2 * E);     // [4]
  __shared__ int s_nact;
  for (int e = tid; e < E; e += kWG) {
    s_cnt[e] = 0;
    s_mask[2 * e] = s_mask[2 * e + 1] = 0u;
  }
  for (int i = tid; i < S; i += kWG) {
    const int e = ld_dev(idx + i);
    s_idx[i] = (e >= 0 && e < E) ? e : -1;
    s_w[i] = ld_dev(wts + i);
  }
  __syncthreads();
  trace_mark(0);
  for (int i = tid; i < S; i += kWG) {
    const int e = s_idx[i];
    if (e < 0) continue;
    atomicAdd(&s_cnt[e], 1);
    if (distinct) {
      const int t = i / k;
      atomicOr(&s_mask[2 * e + (t >> 5)], 1u << (t & 31));
    }
  }
  __syncthreads();
  // one scan gives both the first slot of every expert (low 16 bits) and
  // its index among the active experts (high bits)
  for (int e = tid; e < E; e += kWG) s_cnt[e] += (s_cnt[e] > 0) << 16;
  __syncthreads();
  int* s_cnt0 = s_tmp + 4;  // [E] counts kept for the records
  for (int e = tid; e < E; e += kWG) s_cnt0[e] = s_cnt[e] & 0xFFFF;
  const int total = block_exclusive_scan(s_cnt, E, s_tmp);
  trace_mark(1);
  for (int e = tid; e < E; e += kWG) {
    const int c = s_cnt0[e];
    const int a = s_cnt[e] >> 16;
    if (c > 0 && a < P.max_act) act[a] = make_int4(e, s_cnt[e] & 0xFFFF, c, 0);
  }
  if (tid == 0) s_nact = min(total >> 16, P.max_act);
  trace_mark(2);
  // slot of selection i: the expert's first slot + the number of earlier
  // selections of the same expert (earlier tokens from the token mask when
  // a token's experts are distinct, else counted)
  for (int i = tid; i < S; i += kWG) {
    const int e = s_idx[i];
    if (e < 0) {
      tok_slot[i] = -1;
      continue;
    }
    int rank = 0;
    if (distinct) {
      const int t = i / k;
      const unsigned lo = s_mask[2 * e], hi = s_mask[2 * e + 1];
      rank = t < 32 ? __popc(lo & ((1u << t) - 1u)) : __popc(lo) + __popc(hi & ((1u << (t - 32)) - 1u));
    } else {
      int j = 0;
      for (; j + 4 <= i; j += 4) {
        const int4 v = *reinterpret_cast<const int4*>(s_idx + j);
        rank += (v.x == e) + (v.y == e) + (v.z == e) + (v.w == e);
      }
      for (; j < i; ++j) rank += (s_idx[j] == e);
    }
    const int pos = min((s_cnt[e] & 0xFFFF) + rank, S - 1);
    slot_tok[pos] = i / k;
    slot_w[pos] = s_w[i];
    slot_e[pos] = e;
    tok_slot[i] = pos;
  }
  __syncthreads();
  trace_mark(3);
  return {act, slot_tok, slot_w, slot_e, tok_slot, s_nact};
}

// The same tables from at most 64 selections held one per lane of wave 0
// (lane i: selection i's expert, -1 if none or invalid, and weight). A
// selection's slot is the number of valid selections of smaller experts plus
// the earlier ones of its own expert (a stable sort by expert); the active
// index of an expert is the number of distinct smaller experts.
__device__ RouteTab build_routing_wave(const Plan& P, int e, float wv, uint8_t* tab) {
  const int S = P.S, k = P.k;
  int4* act = reinterpret_cast<int4*>(tab);
  int* slot_tok = reinterpret_cast<int*>(act + P.max_act);
  float* slot_w = reinterpret_cast<float*>(slot_tok + S);
  int* slot_e = reinterpret_cast<int*>(slot_w + S);
  int* tok_slot = slot_e + S;
  __shared__ int s_nact;
  if (threadIdx.x < 64) {
    const int l = threadIdx.x;
    int below = 0, same = 0, before = 0;
    for (int i = 0; i < S; ++i) {
      const int ei = __builtin_amdgcn_readlane(e, i);
      below += (int)(ei >= 0) & (int)(ei < e);
      same += (int)(ei == e);
      before += (int)(ei == e) & (int)(i < l);
    }
    const int valid = (int)(e >= 0);
    const unsigned long long firsts = __ballot(valid & (int)(before == 0));
    int dbelow = 0;
    for (unsigned long long m = firsts; m; m &= m - 1)
      dbelow += (int)(__builtin_amdgcn_readlane(e, (int)__builtin_ctzll(m)) < e);
    if (l < S) {
      const int pos = min(below + before, S - 1);
      if (valid) {
        slot_tok[pos] = l / k;
        slot_w[pos] = wv;
        slot_e[pos] = e;
      }
      tok_slot[l] = valid ? pos : -1;
      if (valid && before == 0 && dbelow < P.max_act) act[dbelow] = make_int4(e, below, same, 0);
    }
    if (l == 0) s_nact = min(__popcll(firsts), P.max_act);
  }
  __syncthreads();
  trace_mark(3);
  return {act, slot_tok, slot_w, slot_e, tok_slot, s_nact};
}

// ---- exact top-k in one wave ----------------------------------------------
// Logits are ordered by a 64-bit key that preserves the order of doubles
// (-0 and +0 share a key); equal keys fall back to the lower expert index.
__device__ __forceinline__ unsigned long long order_key(double v) {
  if (v == 0.0) v = 0.0;
  const unsigned long long u = (unsigned long long)__double_as_longlong(v);
  return (u >> 63) ? ~u : (u | 0x8000000000000000ull);
}

__device__ __forceinline__ int wave_count(int p) { return __popcll(__ballot(p)); }

// Lanes below this lane with their bit set in mask.
__device__ __forceinline__ int lanes_below(unsigned long long mask) {
  return __builtin_amdgcn_mbcnt_hi((unsigned)(mask >> 32), __builtin_amdgcn_mbcnt_lo((unsigned)mask, 0u));
}

// The m-th largest of the wave's values v[i] with in[i] set (m >= 1 of them
// exist): the largest T with at least m values >= T, found one bit at a
// time from the most significant.
template <int NE>
__device__ __forceinline__ unsigned wave_kth_largest(const unsigned (&v)[NE], const int (&in)[NE], int m) {
  unsigned T = 0;
  for (int b = 31; b >= 0; --b) {
    const unsigned c = T | (1u << b);
    int n = 0;
#pragma unroll
    for (int i = 0; i < NE; ++i) n += wave_count(in[i] & (int)(v[i] >= c));
    if (n >= m) T = c;
  }
  return T;
}

// Top-k of lg[0..E) (E <= 64 NE) by one wave: sel[j] = expert of rank j
// under (descending logit, ascending index). ck/ce: LDS scratch of k keys
// and experts. The k-th largest high key half is found first; only when
// several experts share it are the low halves, then the indices, consulted.
template <int NE>
__device__ void wave_topk(const double* lg, int E, int k, int* sel, unsigned long long* ck, int* ce) {
  const int l = threadIdx.x & 63;
  unsigned long long key[NE];
  unsigned hi[NE], lo[NE];
  int valid[NE];
#pragma unroll
  for (int i = 0; i < NE; ++i) {
    const int e = l + 64 * i;
    valid[i] = e < E;
    key[i] = valid[i] ? order_key(lg[e]) : 0ull;
    hi[i] = (unsigned)(key[i] >> 32);
    lo[i] = (unsigned)key[i];
  }
  const unsigned T = wave_kth_largest<NE>(hi, valid, k);
  int above = 0, at = 0, inq[NE];
#pragma unroll
  for (int i = 0; i < NE; ++i) {
    inq[i] = valid[i] & (int)(hi[i] == T);
    above += wave_count(valid[i] & (int)(hi[i] > T));
    at += wave_count(inq[i]);
  }
  // experts with high half T: all of them are selected, or the need best
  // among them (low half, then index)
  unsigned T2 = 0;
  int need_ties = kMaxE + 1;
  if (above + at > k) {
    const int need = k - above;
    T2 = wave_kth_largest<NE>(lo, inq, need);
    int above2 = 0;
#pragma unroll
    for (int i = 0; i < NE; ++i) above2 += wave_count(inq[i] & (int)(lo[i] > T2));
    need_ties = need - above2;
  }
  // compact the k selected experts in index order
  int base = 0, tie_base = 0;
#pragma unroll
  for (int i = 0; i < NE; ++i) {
    const int tie = inq[i] & (int)(lo[i] == T2);
    const unsigned long long tm = __ballot(tie);
    const int trank = tie_base + lanes_below(tm);
    tie_base += __popcll(tm);
    const int s = valid[i] & ((int)(hi[i] > T) | (inq[i] & ((int)(lo[i] > T2) | (tie & (int)(trank < need_ties)))));
    const unsigned long long sm = __ballot(s);
    if (s) {
      const int pos = base + lanes_below(sm);
      ck[pos] = key[i];
      ce[pos] = l + 64 * i;
    }
    base += __popcll(sm);
  }
  wave_lds_sync();
  // rank among the selected: larger keys, and equal keys of lower index
  // (earlier in the compacted order)
  if (l < k) {
    const unsigned long long kj = ck[l];
    int r = 0;
    for (int f = 0; f < k; ++f) {
      const unsigned long long kf = ck[f];
      r += (int)(kf > kj) | ((int)(kf == kj) & (int)(f < l));
    }
    sel[r] = ce[l];
  }
  wave_lds_sync();
}

// Logit of expert e for token t: the router chunks' partials summed in chunk
// order, plus the bias (the same arithmetic wherever the select runs).
__device__ __forceinline__ double router_logit(const Plan& P, const Args& A, int t, int e, float bias) {
  constexpr int RB = 32;  // partials in flight; past the end re-read the last one, masked out
  const double* rl = wsp<const double>(A, P.o_rl);
  double s = 0.0;
  for (int c0 = 0; c0 < P.nch_r; c0 += RB) {
    double v[RB];
#pragma unroll
    for (int i = 0; i < RB; ++i) v[i] = ld_dev(rl + ((size_t)min(c0 + i, P.nch_r - 1) * P.B + t) * P.E + e);
#pragma unroll
    for (int i = 0; i < RB; ++i) s += (c0 + i < P.nch_r) ? v[i] : 0.0;
  }
  return A.L.router_bias ? s + (double)bias : s;
}

// Top-k and gating of one token from its logits lg[0..E) in LDS (smem, lg_cap
// doubles, then the scratch below) and each thread's own logit (expert tid):
// top-k by descending logit with ties to the lower index, softmax over the k
// selected logits; lanes j < k of wave 0 return selection j (expert, weight).
//
// Up to kWG experts, each thread holds its expert's key and counts the
// experts with a larger high key half (comparisons split over the waves):
// experts sharing a high half share a rank, and rank slot r < k receives the
// best of its group by (low half, then lower index). A group of g > 1 at rank
// r < k - 1 leaves slot r + 1 empty; with no empty slot every rank below k is
// held by a single expert, or by the correct best of a group at rank k - 1,
// so the slots are the exact selection. Otherwise (and for more experts) one
// wave selects exactly on the full keys.
__device__ void select_core(const Plan& P, uint8_t* smem, int lg_cap, double own, int& e_out, float& w_out) {
  const int tid = threadIdx.x;
  const int E = P.E, k = P.k;
  double* lg = reinterpret_cast<double*>(smem);                                    // [E]
  unsigned long long* slot = reinterpret_cast<unsigned long long*>(lg + lg_cap);   // [k]
  unsigned long long* ck = slot + kMaxK;                                           // [k]
  unsigned* hk = reinterpret_cast<unsigned*>(ck + kMaxK);                          // [kWG]
  int* rank = reinterpret_cast<int*>(hk + kWG);                                    // [kWG]
  int* sel = rank + kWG;                                                           // [k]
  int* ce = sel + kMaxK;                                                           // [k]
  const bool counted = E <= kWG;
  if (counted) {
    const int Ep = (E + 31) & ~31;
    const unsigned long long key = tid < E ? order_key(own) : 0ull;
    if (tid < Ep) {
      hk[tid] = (unsigned)(key >> 32);  // padding keys are 0, below every logit's
      rank[tid] = 0;
    }
    if (tid < kMaxK) slot[tid] = 0ull;
    __syncthreads();
    const int parts = max(1, kWG / Ep);
    const int per = ((Ep + parts - 1) / parts + 31) & ~31;
    const int e = tid % Ep, pt = tid / Ep;
    const int f0 = pt * per, f1 = min(Ep, f0 + per);
    const unsigned ke = hk[e];
    int rk = 0;
    for (int f = f0; f < f1; f += 32) {
      const uint4* q = reinterpret_cast<const uint4*>(hk + f);
      uint4 u[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) u[j] = q[j];
#pragma unroll
      for (int j = 0; j < 8; ++j) rk += (int)(u[j].x > ke) + (int)(u[j].y > ke) + (int)(u[j].z > ke) + (int)(u[j].w > ke);
    }
    if (e < E && f0 < f1) atomicAdd(&rank[e], rk);
    __syncthreads();
    if (tid < E) {
      const int r = rank[tid];
      if (r < k) atomicMax(&slot[r], ((unsigned long long)(unsigned)key << 32) | (unsigned)(~tid));
    }
  }
  __syncthreads();
  trace_mark(0);
  e_out = -1;
  w_out = 0.0f;
  if (tid < 64) {
    const unsigned long long v = counted && tid < k ? slot[tid] : 1ull;
    int e;
    if (!counted || __ballot(v == 0ull)) {
      const int ne = (E + 63) / 64;
      if (ne <= 1)
        wave_topk<1>(lg, E, k, sel, ck, ce);
      else if (ne <= 2)
        wave_topk<2>(lg, E, k, sel, ck, ce);
      else if (ne <= 4)
        wave_topk<4>(lg, E, k, sel, ck, ce);
      else if (ne <= 8)
        wave_topk<8>(lg, E, k, sel, ck, ce);
      else
        wave_topk<16>(lg, E, k, sel, ck, ce);
      e = tid < k ? sel[tid] : 0;
    } else {
      e = tid < k ? (int)(~(unsigned)v) : 0;
    }
    trace_mark(1);
    // softmax over the k selected logits (a fixed summation tree); exp of a
    // non-positive difference in single precision is far inside the
    // weights' tolerance
    const double x = lg[e];
    const double mx = lane0(x);
    const double ex = tid < k ? (double)expf((float)(x - mx)) : 0.0;
    const double sum = wave_sum(ex);
    if (tid < k) {
      e_out = e;
      w_out = (float)(ex / sum);
    }
    trace_mark(2);
  }
}

// Select item for token t (see select_core): waits for its token block's
// router chunks, sums their partials per expert in chunk order (plus the
// bias) and writes topk_idx / topk_w.
__device__ void item_select(const Plan& P, const Args& A, int t, uint8_t* smem) {
  const int tid = threadIdx.x;
  const int E = P.E, k = P.k;
  double* lg = reinterpret_cast<double*>(smem);  // [E]
  // the bias is read before the wait so its latency is hidden
  const float b0 = (A.L.router_bias && tid < E) ? A.L.router_bias[tid] : 0.0f;
  const int* rcf = wsp<const int>(A, P.o_rc_flag);
  const int nrt = P.nch_r * P.n_eg;  // router chunks of this token's block
  rcf += (t / kRouterTok) * nrt * kTickPad;
  wait_all(A, nrt, [&](int i) { return ld_dev(rcf + i * kTickPad) != 0; });
  double own = 0.0;  // logit of expert tid
  for (int e = tid; e < E; e += kWG) {
    const double s = router_logit(P, A, t, e, e == tid ? b0 : (A.L.router_bias ? A.L.router_bias[e] : 0.0f));
    lg[e] = s;
    if (e == tid) own = s;
  }
  int e_sel;
  float w_sel;
  select_core(P, smem, kMaxE, own, e_sel, w_sel);
  if (tid < k) {
    st_dev(A.topk_idx + t * k + tid, e_sel);
    st_dev(A.topk_w + t * k + tid, w_sel);
  }
}

// z value (basis src, row-major [B][r] index rem): the z items' partials
// summed in item order.
__device__ __forceinline__ float z_sum(const Plan& P, const Args& A, int src, int rem) {
  constexpr int ZB = 8;
  const int B = P.B, r = P.r;
  const float* zp = wsp<const float>(A, P.o_zp) + ((size_t)src * P.nq_z * B) * r + rem;
  float s = 0.0f;
  for (int c0 = 0; c0 < P.nq_z; c0 += ZB) {
    float v[ZB];
#pragma unroll
    for (int j = 0; j < ZB; ++j) v[j] = ld_dev(zp + (size_t)min(c0 + j, P.nq_z - 1) * B * r);
#pragma unroll
    for (int j = 0; j < ZB; ++j) s += (c0 + j < P.nq_z) ? v[j] : 0.0f;
  }
  return s;
}

// Projection-code-book item j (F_TBOOK; Sec. 4.2): token t, input-side
// projection pj, blocks [b0, b0 + nb) of x: thread k holds code word k of the
// projection's book and writes T[t][pj][b][k] = sum_i x[t][b*d + i] cb[k][i]
// (float32, i ascending) for each block, 1 KB per block across the threads,
// four blocks per round (their LDS reads issued together). Read by the next
// kernel of the call (the stream orders it).
template <int D>
__device__ void tbook_rows(const Plan& P, const Args& A, int t, int pj, int b0, int nb, const float* xs) {
  const int K = P.K, nblk = P.H / D, k = threadIdx.x;
  if (k >= K) return;
  const uint16_t* cb = (pj ? A.L.cb_up : A.L.cb_gate) + (size_t)k * D;
  float c[D];
#pragma unroll
  for (int i = 0; i < D; ++i) c[i] = bf(cb[i]);
  // buffer stores: the compiler cannot take them for writes to xs
  const rsrc_t trs = make_rsrc(wsp<float>(A, tbook_offset(P)), (uint32_t)tbook_bytes(P));
  const uint32_t o = (uint32_t)(((((size_t)t * 2 + pj) * nblk + b0) * K + k) * 4);
  for (int bb0 = 0; bb0 < nb; bb0 += 4) {
    float v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const float* xb = xs + min(bb0 + u, nb - 1) * D;
      float acc = 0.0f;
#pragma unroll
      for (int i = 0; i < D; ++i) acc = fmaf(xb[i], c[i], acc);
      v[u] = acc;
    }
#pragma unroll
    for (int u = 0; u < 4; ++u)
      if (bb0 + u < nb)
        __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v[u]), trs, o + (uint32_t)(bb0 + u) * K * 4, 0, 0);
  }
}

__device__ void item_tbook(const Plan& P, const Args& A, int j, uint8_t* smem) {
  const int d = P.d, nblk = P.H / d, ng = tbook_groups(P), np = n_proj(P);
  const int g = j % ng, rest = j / ng;
  const int pj = np == 2 ? rest % 2 : 1, t = rest / np;
  const int b0 = g * kTBookBlocks, nb = min(kTBookBlocks, nblk - b0);
  float* xs = reinterpret_cast<float*>(smem);  // [nb * d]
  for (int i = threadIdx.x; i < nb * d; i += kWG) xs[i] = bf(A.x[(size_t)t * P.H + b0 * d + i]);
  __syncthreads();
  if (d == 8)
    tbook_rows<8>(P, A, t, pj, b0, nb, xs);
  else if (d == 4)
    tbook_rows<4>(P, A, t, pj, b0, nb, xs);
  else
    tbook_rows<2>(P, A, t, pj, b0, nb, xs);
}

__device__ void item_z_reduce(const Plan& P, const Args& A, int i) {
  const int* zcf = wsp<const int>(A, P.o_zc_flag);
  wait_all(A, P.n_zc, [&](int f) { return ld_dev(zcf + f * kTickPad) != 0; });
  const int o = i * kWG + threadIdx.x;
  const int B = P.B, r = P.r;
  if (o < 2 * B * r) {
    const int pj = o / (B * r), rem = o % (B * r);
    const int src = P.z_sep ? pj : 0;
    A.z_out[o] = z_sum(P, A, src, rem);
  }
}

// ===========================================================================
// MFMA streams
// ===========================================================================
// Every product here is D[token][column] += A[token][K] * W[K][column] on
// v_mfma_f32_16x16x32_bf16, one wave per 64 output columns:
//   A (activations): lane l = 16 g + n holds token row n, inputs
//     32 ks + 8 g .. + 8 of K-step ks, read from LDS (`ops`, [token][uint4]
//     with NOPS interleaved sets: 1 for bf16 x, 2 for the bf16 hi/lo parts of
//     a float32 operand, whose two products are summed).
//   W (weights): lane l holds rows 32 ks + 8 g .. + 8 of output column
//     c0 + 4 n + q for MFMA q = 0..3. For VQ weights this slice is one code
//     word (d = 8) or two (d = 4) read from the LDS code book; for dense bf16
//     factors it is gathered from 8 rows of 4 columns with v_perm.
//   D: accumulator q, element i of lane l = token 4 g + i, column c0 + 4 n + q.
// Weight loads run a fixed-depth register pipeline (PD K-steps in flight);
// prime() issues the first PD steps so callers can start the HBM traffic
// before they wait for their activations.

// MFMA rows are independent, so token rows past nt simply repeat row nt - 1
// (never stored) instead of branching around the LDS read.
__device__ __forceinline__ int a_row(int n, int nt) { return min(n, nt - 1); }

// Scheduling of one K-step: all LDS operand reads first, then the MFMAs, so
// the reads' latencies overlap instead of each MFMA waiting for its own.
template <int NREAD, int NMFMA>
__device__ __forceinline__ void sched_step() {
  __builtin_amdgcn_sched_group_barrier(0x100, NREAD, 0);  // DS reads
  __builtin_amdgcn_sched_group_barrier(0x008, NMFMA, 0);  // MFMA
}

constexpr int kSc1 = 16;  // cache policy operand of a device-scope (sc1) buffer access

// Device-scope reads (and 16-byte writes) of workspace data handed between
// workgroups, through one buffer resource over the workspace: the byte
// offset kOob (past the workspace) reads zeros without a memory access, so a
// skipped term needs no branch and every load of a batch issues back to back.
struct WsAccess {
  rsrc_t rs;
  const uint8_t* base;
  __device__ __forceinline__ WsAccess(const Args& A, const Plan& P)
      : rs(make_rsrc(A.ws, (uint32_t)P.total)), base(A.ws) {}
  __device__ __forceinline__ uint32_t off(const void* p) const {
    return (uint32_t)(reinterpret_cast<const uint8_t*>(p) - base);
  }
  __device__ __forceinline__ float4 f4(uint32_t o) const {
    return __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(rs, o, 0, kSc1));
  }
  // one 16-byte device-scope store (the producers' side of the hand-offs)
  __device__ __forceinline__ void st4(uint32_t o, float4 v) const {
    typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), rs, o, 0, kSc1);
  }
  __device__ __forceinline__ void st1(uint32_t o, float v) const {
    __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v), rs, o, 0, kSc1);
  }
};

// NC: copies of the code book in LDS (d = 8): lane l reads copy l % NC, so
// lanes of one LDS pass collide less on the random code-word rows.
template <int D, int NOPS, int PD, int NC = 1>
struct VqPipe {
  static constexpr int W = 8 / D;  // code rows per lane and K-step (d = 8, 4, 2)
  uint32_t buf[PD][W];
  rsrc_t rs;
  uint32_t lane_off, step_bytes, row_len;
  int ks0, nks;

  // steps i >= nks read zeros without touching memory
  __device__ __forceinline__ void load(int i, uint32_t (&b)[W]) {
    const uint32_t o = i < nks ? lane_off + (uint32_t)(ks0 + i) * step_bytes : kOob;
#pragma unroll
    for (int v = 0; v < W; ++v) b[v] = __builtin_amdgcn_raw_buffer_load_b32(rs, o + v * row_len, 0, 0);
  }
  // codes [n_rows][rl] of one expert; columns [c0, c0 + 64) of n_out (lanes
  // past n_out read the last valid columns, whose results are never stored);
  // K-steps [k0, k1).
  __device__ __forceinline__ void prime(const uint8_t* c, int n_rows, int rl, int c0, int n_out, int k0,
                                        int k1) {
    rs = make_rsrc(c, (uint32_t)n_rows * rl);
    row_len = rl;
    const int g = (threadIdx.x & 63) >> 4;
    const int col = min(c0 + 4 * (threadIdx.x & 15), n_out - 4);
    step_bytes = (uint32_t)(32 / D) * rl;
    lane_off = (uint32_t)(g * (8 / D)) * rl + col;
    ks0 = k0;
    nks = k1 - k0;
#pragma unroll
    for (int u = 0; u < PD; ++u) load(u, buf[u]);
  }
  __device__ __forceinline__ void step(int ks, const uint32_t (&b)[W], const uint4* __restrict__ cb_s,
                                       const uint4* __restrict__ ops, int ops_ld, int ops_ks0, int nt,
                                       f32x4 acc[4]) {
    const int l = threadIdx.x & 63, n = l & 15, g = l >> 4;
    const int oi = a_row(n, nt) * ops_ld + ((ks - ops_ks0) * 4 + g) * NOPS;
    const uint4 a0 = ops[oi];
    uint4 a1 = a0;
    if (NOPS == 2) a1 = ops[oi + 1];
    const uint2* cb2 = reinterpret_cast<const uint2*>(cb_s);
    uint4 w[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      if constexpr (D == 8) {
        w[q] = cb_s[((b[0] >> (8 * q)) & 255u) * NC + (l & (NC - 1))];
      } else if constexpr (D == 4) {
        const uint2 lo = cb2[(b[0] >> (8 * q)) & 255u];
        const uint2 hi = cb2[(b[1] >> (8 * q)) & 255u];
        w[q] = make_uint4(lo.x, lo.y, hi.x, hi.y);
      } else {  // d = 2: four 4-byte code words
        const uint32_t* cb1 = reinterpret_cast<const uint32_t*>(cb_s);
        w[q] = make_uint4(cb1[(b[0] >> (8 * q)) & 255u], cb1[(b[1] >> (8 * q)) & 255u],
                          cb1[(b[2] >> (8 * q)) & 255u], cb1[(b[3] >> (8 * q)) & 255u]);
      }
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      acc[q] = mfma_bf16(a0, w[q], acc[q]);
      if (NOPS == 2) acc[q] = mfma_bf16(a1, w[q], acc[q]);
    }
    sched_step<NOPS + 4 * W, 4 * NOPS>();
  }
  __device__ __forceinline__ void run(const uint4* cb_s, const uint4* ops, int ops_ld, int ops_ks0,
                                      int nt, f32x4 acc[4]) {
    run(cb_s, ops, ops_ld, ops_ks0, nt, acc, []() {});
  }
  // late() runs once when at most PD steps remain (loads for what follows
  // the run go out then, not before the run starts)
  template <typename Late>
  __device__ __forceinline__ void run(const uint4* cb_s, const uint4* ops, int ops_ld, int ops_ks0,
                                      int nt, f32x4 acc[4], Late late) {
    if (nks <= PD) {  // every step was primed: no refills
      late();
#pragma unroll
      for (int u = 0; u < PD; ++u) {
        if (u < nks) step(ks0 + u, buf[u], cb_s, ops, ops_ld, ops_ks0, nt, acc);
        __builtin_amdgcn_sched_barrier(0);
      }
      return;
    }
    for (int i0 = 0; i0 < nks; i0 += PD) {
      if (i0 + PD >= nks) late();
#pragma unroll
      for (int u = 0; u < PD; ++u) {
        const int i = i0 + u;
        if (i < nks) step(ks0 + i, buf[u], cb_s, ops, ops_ld, ops_ks0, nt, acc);
        load(i + PD, buf[u]);
        // keep each step's LDS operand reads inside the step: hoisting them
        // across the unrolled pipeline costs registers, not time
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  }
};

// Two 64-column sub-tiles per wave, kColsPerGroup columns apart (a down tile
// of two column groups, float32 activations as bf16 hi + lo): each K-step's
// activation reads serve both sub-tiles. A second sub-tile past n_out reads
// zeros (its results are never stored).
template <int D, int PD, int NC = 1>
struct VqPipe2 {
  static constexpr int W = D == 8 ? 1 : 2;
  uint32_t buf[PD][2 * W];
  rsrc_t rs;
  uint32_t lane_off, lane_off2, step_bytes, row_len;
  int ks0, nks;
  bool has2;

  __device__ __forceinline__ void load(int i, uint32_t (&b)[2 * W]) {
    const uint32_t st = (uint32_t)(ks0 + i) * step_bytes;
    const uint32_t o = i < nks ? lane_off + st : kOob, o2 = i < nks && has2 ? lane_off2 + st : kOob;
    b[0] = __builtin_amdgcn_raw_buffer_load_b32(rs, o, 0, 0);
    if constexpr (D == 4) b[1] = __builtin_amdgcn_raw_buffer_load_b32(rs, o + row_len, 0, 0);
    b[W] = __builtin_amdgcn_raw_buffer_load_b32(rs, o2, 0, 0);
    if constexpr (D == 4) b[W + 1] = __builtin_amdgcn_raw_buffer_load_b32(rs, o2 + row_len, 0, 0);
  }
  __device__ __forceinline__ void prime(const uint8_t* c, int n_rows, int rl, int c0, int n_out, int k0,
                                        int k1) {
    rs = make_rsrc(c, (uint32_t)n_rows * rl);
    row_len = rl;
    const int g = (threadIdx.x & 63) >> 4;
    const int col = min(c0 + 4 * (threadIdx.x & 15), n_out - 4);
    const int col2 = min(c0 + kColsPerGroup + 4 * (threadIdx.x & 15), n_out - 4);
    has2 = c0 + kColsPerGroup < n_out;
    step_bytes = (uint32_t)(32 / D) * rl;
    lane_off = (uint32_t)(g * (8 / D)) * rl + col;
    lane_off2 = (uint32_t)(g * (8 / D)) * rl + col2;
    ks0 = k0;
    nks = k1 - k0;
#pragma unroll
    for (int u = 0; u < PD; ++u) load(u, buf[u]);
  }
  __device__ __forceinline__ uint4 word(const uint4* __restrict__ cb_s, const uint32_t* b, int q) const {
    if constexpr (D == 8) {
      return cb_s[((b[0] >> (8 * q)) & 255u) * NC + ((threadIdx.x & 63) & (NC - 1))];
    } else {
      const uint2* cb2 = reinterpret_cast<const uint2*>(cb_s);
      const uint2 lo = cb2[(b[0] >> (8 * q)) & 255u];
      const uint2 hi = cb2[(b[1] >> (8 * q)) & 255u];
      return make_uint4(lo.x, lo.y, hi.x, hi.y);
    }
  }
  __device__ __forceinline__ void step(int ks, const uint32_t (&b)[2 * W], const uint4* __restrict__ cb_s,
                                       const uint4* __restrict__ ops, int ops_ld, int ops_ks0, int nt,
                                       f32x4 acc[8]) {
    const int l = threadIdx.x & 63, n = l & 15, g = l >> 4;
    const int oi = a_row(n, nt) * ops_ld + ((ks - ops_ks0) * 4 + g) * 2;
    const uint4 a0 = ops[oi], a1 = ops[oi + 1];
    uint4 w[8];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      w[q] = word(cb_s, b, q);
      w[4 + q] = word(cb_s, b + W, q);
    }
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      acc[q] = mfma_bf16(a0, w[q], acc[q]);
      acc[q] = mfma_bf16(a1, w[q], acc[q]);
    }
    sched_step<2 + (D == 8 ? 8 : 16), 16>();
  }
  __device__ __forceinline__ void run(const uint4* cb_s, const uint4* ops, int ops_ld, int ops_ks0, int nt,
                                      f32x4 acc[8]) {
    if (nks <= PD) {  // every step was primed: no refills
#pragma unroll
      for (int u = 0; u < PD; ++u) {
        if (u < nks) step(ks0 + u, buf[u], cb_s, ops, ops_ld, ops_ks0, nt, acc);
        __builtin_amdgcn_sched_barrier(0);
      }
      return;
    }
    for (int i0 = 0; i0 < nks; i0 += PD) {
#pragma unroll
      for (int u = 0; u < PD; ++u) {
        const int i = i0 + u;
        if (i < nks) step(ks0 + i, buf[u], cb_s, ops, ops_ld, ops_ks0, nt, acc);
        load(i + PD, buf[u]);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  }
};

template <int Q>
__device__ __forceinline__ uint4 dense_w(const uint2 (&b)[8]) {
  constexpr uint32_t sel = (Q & 1) ? 0x07060302u : 0x05040100u;
  if (Q < 2)
    return make_uint4(__builtin_amdgcn_perm(b[1].x, b[0].x, sel), __builtin_amdgcn_perm(b[3].x, b[2].x, sel),
                      __builtin_amdgcn_perm(b[5].x, b[4].x, sel), __builtin_amdgcn_perm(b[7].x, b[6].x, sel));
  return make_uint4(__builtin_amdgcn_perm(b[1].y, b[0].y, sel), __builtin_amdgcn_perm(b[3].y, b[2].y, sel),
                    __builtin_amdgcn_perm(b[5].y, b[4].y, sel), __builtin_amdgcn_perm(b[7].y, b[6].y, sel));
}

template <int NOPS, int PD>
struct DensePipe {
  uint2 buf[PD][8];
  rsrc_t rs;
  uint32_t lane_off, step_bytes, row_bytes;
  int ks0, nks;

  // rows past k_rows and steps i >= nks read zeros without touching memory
  __device__ __forceinline__ void load(int i, uint2 (&b)[8]) {
    const uint32_t o = i < nks ? lane_off + (uint32_t)(ks0 + i) * step_bytes : kOob;
#pragma unroll
    for (int e = 0; e < 8; ++e)
      b[e] = __builtin_bit_cast(uint2, __builtin_amdgcn_raw_buffer_load_b64(rs, o + e * row_bytes, 0, 0));
  }
  // W [k_rows][ld] row-major bf16; columns [c0, c0 + 64) of n_out (lanes
  // past n_out read the last valid columns, whose results are never stored);
  // K-steps [k0, k1).
  __device__ __forceinline__ void prime(const uint16_t* w, int ldw, int c0, int n_out, int kr, int k0,
                                        int k1) {
    rs = make_rsrc(w, (uint32_t)kr * ldw * 2);
    const int g = (threadIdx.x & 63) >> 4;
    const int col = min(c0 + 4 * (threadIdx.x & 15), n_out - 4);
    row_bytes = (uint32_t)ldw * 2;
    step_bytes = 32 * row_bytes;
    lane_off = (uint32_t)(8 * g) * row_bytes + (uint32_t)col * 2;
    ks0 = k0;
    nks = k1 - k0;
#pragma unroll
    for (int u = 0; u < PD; ++u) load(u, buf[u]);
  }
  __device__ __forceinline__ void step(int ks, const uint2 (&b)[8], const uint4* __restrict__ ops, int ops_ld,
                                       int ops_ks0, int nt, f32x4 acc[4]) {
    const int l = threadIdx.x & 63, n = l & 15, g = l >> 4;
    const int oi = a_row(n, nt) * ops_ld + ((ks - ops_ks0) * 4 + g) * NOPS;
    const uint4 a0 = ops[oi];
    uint4 a1 = a0;
    if (NOPS == 2) a1 = ops[oi + 1];
    const uint4 w0 = dense_w<0>(b), w1 = dense_w<1>(b), w2 = dense_w<2>(b), w3 = dense_w<3>(b);
    acc[0] = mfma_bf16(a0, w0, acc[0]);
    acc[1] = mfma_bf16(a0, w1, acc[1]);
    acc[2] = mfma_bf16(a0, w2, acc[2]);
    acc[3] = mfma_bf16(a0, w3, acc[3]);
    if (NOPS == 2) {
      acc[0] = mfma_bf16(a1, w0, acc[0]);
      acc[1] = mfma_bf16(a1, w1, acc[1]);
      acc[2] = mfma_bf16(a1, w2, acc[2]);
      acc[3] = mfma_bf16(a1, w3, acc[3]);
    }
    sched_step<NOPS, 4 * NOPS>();
  }
  __device__ __forceinline__ void run(const uint4* ops, int ops_ld, int ops_ks0, int nt, f32x4 acc[4]) {
    if (nks <= PD) {  // every step was primed: no refills
#pragma unroll
      for (int u = 0; u < PD; ++u)
        if (u < nks) step(ks0 + u, buf[u], ops, ops_ld, ops_ks0, nt, acc);
      return;
    }
    for (int i0 = 0; i0 < nks; i0 += PD) {
#pragma unroll
      for (int u = 0; u < PD; ++u) {
        const int i = i0 + u;
        if (i < nks) step(ks0 + i, buf[u], ops, ops_ld, ops_ks0, nt, acc);
        load(i + PD, buf[u]);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  }
};


__device__ __forceinline__ void zero_acc(f32x4 acc[4]) {
#pragma unroll
  for (int q = 0; q < 4; ++q) acc[q] = f32x4{0.f, 0.f, 0.f, 0.f};
}

// Stores token rows 4g + i < nt of the wave's accumulators with device-scope
// stores: row t goes to dst(t) + c0 + 4n (the 4 MFMAs' columns).
template <typename F>
__device__ __forceinline__ void store_acc(const WsAccess& ws, const f32x4 acc[4], int nt, int c0, int n_out, F dst) {
  const int l = threadIdx.x & 63, n = l & 15, g = l >> 4;
  const int col = c0 + 4 * n;
  if (col >= n_out) return;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int t = 4 * g + i;
    if (t < nt) ws.st4(ws.off(dst(t) + col), make_float4(acc[0][i], acc[1][i], acc[2][i], acc[3][i]));
  }
}

// Stages bf16 activation rows (8 inputs per uint4) for token slots [0, nt):
// ops[t * ld + j] = inputs 8 j .. 8 j + 7 of row src(t). Threads first,
// first + stride, ... share the work (the whole workgroup by default).
template <typename F>
__device__ __forceinline__ void stage_bf16(uint4* ops, int ld, int nt, int n8, F src,
                                           int first = threadIdx.x, int stride = kWG) {
  for (int i = first; i < nt * n8; i += stride) {
    const int t = i / n8, j = i % n8;
    ops[t * ld + j] = *reinterpret_cast<const uint4*>(src(t) + 8 * j);
  }
}

// Writes 4 consecutive fp32 values as bf16 hi/lo halves of an LDS operand
// row of float32 activations (value = hi + lo): inputs 8 j .. 8 j + 7 sit in
// the uint4 pair [2 j] (hi) and [2 j + 1] (lo), so quad q is half (q & 1) of
// the pair at [2 (q >> 1)].
__device__ __forceinline__ void put_split_quad(uint4* row, int q, float4 v) {
  const float f[4] = {v.x, v.y, v.z, v.w};
  uint32_t h[4], lw[4];
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    h[u] = rne_bf16(f[u]);
    lw[u] = rne_bf16(f[u] - bf(h[u]));
  }
  uint2* hi = reinterpret_cast<uint2*>(row + 2 * (q >> 1)) + (q & 1);
  uint2* lo = reinterpret_cast<uint2*>(row + 2 * (q >> 1) + 1) + (q & 1);
  *hi = make_uint2(h[0] | (h[1] << 16), h[2] | (h[3] << 16));
  *lo = make_uint2(lw[0] | (lw[1] << 16), lw[2] | (lw[3] << 16));
}

// Down operand rows from the gate/up partial sums: p = silu(g) * u (up-only
// experts: p = max(u, 0)^2) for token rows [0, nt) (slots slot0 + t) on I columns col0 + [0, 4 nquad), each sum
// over the ns splits in split order, staged as bf16 hi/lo quads. U units
// (token, quad) per thread per round and NSC splits per load batch keep 16
// loads in flight.
template <int U, int NSC, bool RELU2>
__device__ __forceinline__ void stage_p(const WsAccess& ws, const Plan& P, uint4* ops, int ld, int nt, int nquad,
                                        int slot0, int col0) {
  const int ns = P.ns, I = P.I, n = nt * nquad;
  for (int i0 = threadIdx.x; i0 < n; i0 += U * kWG) {
    float4 g[U], u[U];
    uint32_t base[U];
#pragma unroll
    for (int uu = 0; uu < U; ++uu) {
      const int i = i0 + uu * kWG, ii = min(i, n - 1);
      base[uu] = i < n ? (uint32_t)(P.o_gu + ((size_t)(slot0 + ii / nquad) * 2 * ns * I + col0 + 4 * (ii % nquad)) * 4)
                       : kOob;
      g[uu] = u[uu] = make_float4(0.f, 0.f, 0.f, 0.f);
    }
    for (int s0 = 0; s0 < ns; s0 += NSC) {
      float4 v[U][2][NSC];
#pragma unroll
      for (int uu = 0; uu < U; ++uu)
#pragma unroll
        for (int pj = 0; pj < 2; ++pj)
#pragma unroll
          for (int sc = 0; sc < NSC; ++sc)
            // up-only experts: no gate partials, whose loads take the
            // out-of-range offset (zeros, no memory access)
            v[uu][pj][sc] = ws.f4(s0 + sc < ns && (pj || !RELU2) ? base[uu] + (uint32_t)((pj * ns + s0 + sc) * I * 4)
                                                                  : kOob);
#pragma unroll
      for (int uu = 0; uu < U; ++uu)
#pragma unroll
        for (int sc = 0; sc < NSC; ++sc) {
          g[uu] = make_float4(g[uu].x + v[uu][0][sc].x, g[uu].y + v[uu][0][sc].y, g[uu].z + v[uu][0][sc].z,
                              g[uu].w + v[uu][0][sc].w);
          u[uu] = make_float4(u[uu].x + v[uu][1][sc].x, u[uu].y + v[uu][1][sc].y, u[uu].z + v[uu][1][sc].z,
                              u[uu].w + v[uu][1][sc].w);
        }
    }
#pragma unroll
    for (int uu = 0; uu < U; ++uu) {
      const int i = i0 + uu * kWG;
      if (i >= n) continue;
      const float4 x = g[uu], y = u[uu];
      float4 p;
      if constexpr (RELU2) {
        const float4 c = make_float4(fmaxf(y.x, 0.f), fmaxf(y.y, 0.f), fmaxf(y.z, 0.f), fmaxf(y.w, 0.f));
        p = make_float4(c.x * c.x, c.y * c.y, c.z * c.z, c.w * c.w);
      } else {
        p = make_float4(x.x / (1.0f + expf(-x.x)) * y.x, x.y / (1.0f + expf(-x.y)) * y.y,
                        x.z / (1.0f + expf(-x.z)) * y.z, x.w / (1.0f + expf(-x.w)) * y.w);
      }
      put_split_quad(ops + (i / nquad) * ld, i % nquad, p);
    }
  }
}


__device__ __forceinline__ float4 fma4(float w, float4 v, float4 a) {
  return make_float4(fmaf(w, v.x, a.x), fmaf(w, v.y, a.y), fmaf(w, v.z, a.z), fmaf(w, v.w, a.w));
}


// ===========================================================================
// shared projections on MFMA
// ===========================================================================
// z item j: basis pj, 64 columns of z, and four consecutive K-splits of H,
// one per wave (split 4q + w); the waves' partial U^T x are added in wave
// order through LDS and item j stores one partial, zp[pj][q][t][col].
__device__ void item_z(const Plan& P, const Args& A, const Chain& C, int j, uint8_t* smem) {
  const int tid = threadIdx.x, l = tid & 63, w = tid >> 6;
  const int ncol = (P.r + 63) / 64;
  const int q = j % P.nq_z, rem = j / P.nq_z;
  const int c64 = rem % ncol, pj = rem / ncol;
  const int s = 4 * q + w;
  const bool active = s < P.nch_z;
  const int KS = P.H / 32;
  const int ks0 = active ? s * KS / P.nch_z : 0, ks1 = active ? (s + 1) * KS / P.nch_z : 0;
  const int c0 = c64 * 64;
  const uint16_t* U = pj ? A.L.U_up : A.L.U_gate;
  // each wave stages its own activations: [16 tokens][(ks1 - ks0) * 4 + 1] uint4
  const int ld = (KS + P.nch_z - 1) / P.nch_z * 4 + 1;
  uint4* ops = reinterpret_cast<uint4*>(smem) + w * kTokPass * ld;
  float* red = reinterpret_cast<float*>(smem + (size_t)4 * kTokPass * ld * 16);  // [4][64][16]
  float* zinv = red + 4 * 64 * 16;                                                // [16] (F_NORM_IN)
  float* zp = wsp<float>(A, P.o_zp);
  const int B = P.B, H = P.H, r = P.r;
  const WsAccess ws(A, P);
  DensePipe<1, kPdDense> pipe;
  for (int tg = 0; tg < B; tg += kTokPass) {
    const int nt = min(kTokPass, B - tg);
    if (active) pipe.prime(U, r, c0, r, H, ks0, ks1);
    if ((P.flags & F_NORM_IN) && tid < nt) zinv[tid] = norm_inv(P, C, tg + tid);
    __syncthreads();
    if (active) {  // this wave's own region: lanes stride by 64
      if (P.flags & F_NORM_IN) {
        // x = bf16(y * inv_rms), as the router chunks form it
        const int n8 = (ks1 - ks0) * 4;
        for (int i = l; i < nt * n8; i += 64) {
          const int t = i / n8, j8 = i % n8;
          const float4* yr = reinterpret_cast<const float4*>(C.y_in + (size_t)(tg + t) * H + ks0 * 32 + 8 * j8);
          const float4 a = yr[0], b = yr[1];
          const float iv = zinv[t];
          ops[t * ld + j8] = make_uint4(rne_bf16(a.x * iv) | (rne_bf16(a.y * iv) << 16),
                                        rne_bf16(a.z * iv) | (rne_bf16(a.w * iv) << 16),
                                        rne_bf16(b.x * iv) | (rne_bf16(b.y * iv) << 16),
                                        rne_bf16(b.z * iv) | (rne_bf16(b.w * iv) << 16));
        }
      } else {
        stage_bf16(ops, ld, nt, (ks1 - ks0) * 4,
                   [&](int t) { return A.x + (size_t)(tg + t) * H + ks0 * 32; }, l, 64);
      }
    }
    __syncthreads();
    f32x4 acc[4];
    zero_acc(acc);
    if (active) pipe.run(ops, ld, ks0, nt, acc);
    // lane (n, g) holds token rows 4 g + i, columns c0 + 4 n + qq of MFMA qq
#pragma unroll
    for (int qq = 0; qq < 4; ++qq)
      *reinterpret_cast<float4*>(red + (w * 64 + l) * 16 + 4 * qq) =
          make_float4(acc[qq][0], acc[qq][1], acc[qq][2], acc[qq][3]);
    __syncthreads();
    // thread (i = w, lane l): token row 4 (l >> 4) + i, columns c0 + 4 (l & 15) .. + 3
    const int n = l & 15, t = 4 * (l >> 4) + w, col = c0 + 4 * n;
    if (t < nt && col < r) {
      float v[4];
#pragma unroll
      for (int qq = 0; qq < 4; ++qq) {
        float sum = red[(0 * 64 + l) * 16 + 4 * qq + w];
#pragma unroll
        for (int ww = 1; ww < 4; ++ww) sum += red[(ww * 64 + l) * 16 + 4 * qq + w];
        v[qq] = sum;
      }
      ws.st4(ws.off(zp + (((size_t)pj * P.nq_z + q) * B + tg + t) * r + col), make_float4(v[0], v[1], v[2], v[3]));
    }
    __syncthreads();
  }
  set_flag(wsp<int>(A, P.o_zc_flag) + j * kTickPad);
}

// ===========================================================================
// expert tiles
// ===========================================================================
struct Routing {
  int e, s0, ne;
};

// (expert, first slot, slot count) of active expert a, clamped to the valid
// ranges so that no table content can address memory outside the layer
__device__ __forceinline__ Routing expert_of(const Plan& P, const RouteTab& RT, int a) {
  const int4 v = RT.act[a];
  const int s0 = min(max(v.y, 0), P.S);
  return {min(max(v.x, 0), P.E - 1), s0, min(max(v.z, 0), P.S - s0)};
}

// One code book (K words of D bf16) as 16-byte groups, one per thread, zero
// past the book; stored for the item as word c at cb[c] (d = 8) or at the
// 8-byte slot c of the uint2 view (d = 4). Items load their book before
// their weight prime and store it with their activation staging.
template <int D>
__device__ __forceinline__ uint4 book_load(const uint16_t* src, int K) {
  const int n16 = K * D * 2, byte0 = threadIdx.x * 16;
  uint4 v = make_uint4(0, 0, 0, 0);
  if (byte0 + 16 <= n16) {
    v = *reinterpret_cast<const uint4*>(reinterpret_cast<const uint8_t*>(src) + byte0);
  } else if (byte0 < n16) {  // ragged end of the book
    uint16_t e[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    for (int u = 0; byte0 + 2 * u < n16; ++u) e[u] = src[byte0 / 2 + u];
    v = make_uint4(e[0] | (e[1] << 16), e[2] | (e[3] << 16), e[4] | (e[5] << 16), e[6] | (e[7] << 16));
  }
  return v;
}
template <int D>
__device__ __forceinline__ void book_store(uint4* cb, uint4 v) {
  if (threadIdx.x < 256 * D / 8) cb[threadIdx.x] = v;
}
// NC interleaved copies (d = 8): word w of copy c at w * NC + c
template <int NC>
__device__ __forceinline__ void book_store_copies(uint4* cb, uint4 v) {
#pragma unroll
  for (int c = 0; c < NC; ++c) cb[threadIdx.x * NC + c] = v;
}

// Gate/up tile (a, pj, cg, s): 256 output columns of projection pj over
// split s of the joint reduction axis [x (H inputs) | z (r ranks)], i.e. the
// VQ gather sum and V^T z accumulate in the same MFMA accumulators. Each
// tile writes its partial sums.
// LATE: a tile that runs more code steps than its pipeline holds, code
// steps first, loads its coefficients during the last of them (fewer bytes
// requested at once when every tile starts; large batches).
// XP (batch 1): the token's x row and z rows were staged into LDS (xpre,
// zpre) by the workgroup at kernel start, so the tile stages nothing.
// Gate/up code tile (a, pj, cg, s < ns_v) on the projection code book
// (F_TBOOK; Sec. 4.2), for an expert of at most kTBookTok tokens: thread j
// owns column cg * 256 + j and sums T[tok][pj][b][J_e[b][col]] over the
// split's blocks b (ascending) from T rows staged in LDS; the sum goes to the
// same partial-sum slot as the code-word tile's. Its codes (one byte per
// block) load before the T rows.
template <int D>
__device__ void item_gateup_t(const Plan& P, const Args& A, const RouteTab& RT, int a, int pj, int cg, int s,
                              uint8_t* smem) {
  const Routing R = expert_of(P, RT, a);
  const int H = P.H, I = P.I, K = P.K, nblk = H / D;
  constexpr int BPS = 32 / D;  // blocks per K-step
  int ks0, ks1;
  joint_split(s, P.ns, P.ns_v, H / 32, (P.r + 31) / 32, ks0, ks1);
  const int b0 = ks0 * BPS, nb = min(ks1 - ks0, kTBookTileBlocks / BPS) * BPS;
  const int col = cg * kColsPerGroup + threadIdx.x;
  const rsrc_t crs = make_rsrc((pj ? A.L.codes_up : A.L.codes_gate) + (size_t)R.e * nblk * I, (uint32_t)nblk * I);
  const rsrc_t trs = make_rsrc(wsp<const float>(A, tbook_offset(P)), (uint32_t)tbook_bytes(P));
  float* Ts = reinterpret_cast<float*>(smem);  // [nb][K]
  float* gu = wsp<float>(A, P.o_gu);
  const WsAccess ws(A, P);
  constexpr int kT4 = kTBookTileBlocks * 256 / 4 / kWG;  // float4 T loads per thread (K <= 256)
  const int n4 = nb * K / 4;
  for (int t = 0; t < R.ne; ++t) {
    // the T rows first, then the codes: loads return in order, so staging
    // the T rows does not wait for the codes' HBM latency
    const int tok = RT.slot_tok[R.s0 + t];
    const uint32_t row = (uint32_t)((((size_t)tok * 2 + pj) * nblk + b0) * K * 4);
    float4 tv[kT4];
#pragma unroll
    for (int u = 0; u < kT4; ++u) {
      const int i = threadIdx.x + u * kWG;
      tv[u] = __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(trs, i < n4 ? row + 16u * i : kOob, 0, 0));
    }
    uint32_t code[kTBookTileBlocks];
#pragma unroll
    for (int bb = 0; bb < kTBookTileBlocks; ++bb)
      code[bb] = __builtin_amdgcn_raw_buffer_load_b8(
          crs, bb < nb && col < I ? (uint32_t)((b0 + bb) * I + col) : kOob, 0, 0);
#pragma unroll
    for (int u = 0; u < kT4; ++u) {
      const int i = threadIdx.x + u * kWG;
      if (i < n4) reinterpret_cast<float4*>(Ts)[i] = tv[u];
    }
    __syncthreads();
    float acc = 0.0f;
#pragma unroll
    for (int bb = 0; bb < kTBookTileBlocks; ++bb)
      if (bb < nb) acc += Ts[bb * K + (int)code[bb]];
    if (col < I)
      ws.st1(ws.off(gu + (((size_t)(R.s0 + t) * 2 + pj) * P.ns + s) * I + col), acc);
    __syncthreads();
  }
  publish(wsp<int>(A, P.o_gu_tick) + (a * P.ncg + cg) * kTickPad);
}

template <int D, bool LATE, int NC, bool XP, int PDC>
__device__ void item_gateup(const Plan& P, const Args& A, const RouteTab& RT, int a, int pj, int cg, int s,
                            bool lr_first, uint4* cbs, uint8_t* smem, const uint4* xpre, const uint4* zpre) {
  const Routing R = expert_of(P, RT, a);
  const int H = P.H, I = P.I, r = P.r, B = P.B;
  const int KSX = H / 32, KSZ = (r + 31) / 32;
  int ks0, ks1;
  joint_split(s, P.ns, P.ns_v, KSX, KSZ, ks0, ks1);
  const int x0 = min(ks0, KSX), x1 = min(ks1, KSX);
  const int z0 = max(ks0, KSX) - KSX, z1 = max(ks1, KSX) - KSX;
  const int w = threadIdx.x >> 6;
  const int c0 = cg * kColsPerGroup + w * 64;
  const uint8_t* codes = (pj ? A.L.codes_up : A.L.codes_gate) + (size_t)R.e * (H / D) * I;
  const uint16_t* V = r > 0 ? (pj ? A.L.V_up : A.L.V_gate) + (size_t)R.e * r * I : nullptr;

  const int ldx = (x1 - x0) * 4 + 1, ldz = (z1 - z0) * 8 + 1;
  uint4* xs = reinterpret_cast<uint4*>(smem);
  uint4* zs = xs + P.nt_max * ldx;
  float* gu = wsp<float>(A, P.o_gu);
  const int* const slot_tok = RT.slot_tok;
  const float* zsrc = (P.flags & F_Z) ? A.z_out : A.z_in;

  VqPipe<D, 1, PDC, NC> vq;
  DensePipe<2, kPdDense> lr;
  const int n8x = (x1 - x0) * 4, n8z = (z1 - z0) * 4;  // 8-element groups per token row
  // Activation loads through buffer resources over x [B][H] and z [2][B][r]
  // (written before this kernel): groups past the tile's rows, and z rows
  // past r (zero-padded on both operands; r % 8 == 0, so a group of 8 ranks
  // is all valid or all padding), read zeros from the out-of-range offset.
  const rsrc_t xrs = make_rsrc(A.x, (uint32_t)B * H * 2);
  const rsrc_t zrs = make_rsrc(zsrc, (uint32_t)(2 * B * r * 4));
  auto x_group = [&](int tg, int i, int n) -> uint4 {  // group i of the n staged from row tg
    const int ii = min(i, n - 1), t = tg + ii / n8x;
    const uint32_t o = (uint32_t)(((size_t)slot_tok[R.s0 + t] * H + x0 * 32 + 8 * (ii % n8x)) * 2);
    return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(xrs, i < n ? o : kOob, 0, 0));
  };
  auto z_group = [&](int tg, int i, int n, float4& v0, float4& v1) {  // group i of the n from row tg
    const int ii = min(i, n - 1), t = tg + ii / n8z, q = z0 * 32 + 8 * (ii % n8z);
    const uint32_t o = (uint32_t)((((size_t)pj * B + slot_tok[R.s0 + t]) * r + q) * 4);
    const uint32_t oo = i < n && q < r ? o : kOob;
    v0 = __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(zrs, oo, 0, 0));
    v1 = __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(zrs, oo + 16, 0, 0));
  };
  auto put_z = [&](int t, int jj, float4 v0, float4 v1) {
    const float f[8] = {v0.x, v0.y, v0.z, v0.w, v1.x, v1.y, v1.z, v1.w};
    uint32_t h[8], lw[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      h[u] = rne_bf16(f[u]);
      lw[u] = rne_bf16(f[u] - bf(h[u]));
    }
    zs[t * ldz + 2 * jj] = make_uint4(h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16),
                                      h[6] | (h[7] << 16));
    zs[t * ldz + 2 * jj + 1] = make_uint4(lw[0] | (lw[1] << 16), lw[2] | (lw[3] << 16),
                                          lw[4] | (lw[5] << 16), lw[6] | (lw[7] << 16));
  };
  constexpr int kRegStage = 2;  // activation groups per thread loaded ahead of the weights
  const bool lr_late = LATE && !lr_first && x1 - x0 > PDC;
  if constexpr (XP) {  // one token, one pass: operands already in LDS
    const uint4 bk = book_load<D>(pj ? A.L.cb_up : A.L.cb_gate, P.K);
    __builtin_amdgcn_sched_barrier(0);
    vq.prime(codes, H / D, I, c0, I, x0, x1);
    lr.prime(V, I, c0, I, r, z0, z1);
    __syncthreads();
    if constexpr (NC > 1)
      book_store_copies<NC>(cbs, bk);
    else
      book_store<D>(cbs, bk);
    __syncthreads();
    trace_mark(0);
    f32x4 acc[4];
    zero_acc(acc);
    const uint4* zs1 = zpre + pj * kXpreZRow;
    if (lr_first) lr.run(zs1, 1, 0, 1, acc);
    vq.run(cbs, xpre, 1, 0, 1, acc);
    trace_mark(1);
    if (!lr_first) lr.run(zs1, 1, 0, 1, acc);
    // every slot of the expert is token 0 (a caller's routing may repeat an expert)
    for (int t = 0; t < R.ne; ++t)
      store_acc(WsAccess(A, P), acc, 1, c0, I, [&](int) { return gu + (((size_t)(R.s0 + t) * 2 + pj) * P.ns + s) * I; });
    trace_mark(2);
    publish(wsp<int>(A, P.o_gu_tick) + (a * P.ncg + cg) * kTickPad);
    return;
  }
  for (int tg = 0; tg < R.ne; tg += P.nt_max) {
    const int nt = min(P.nt_max, R.ne - tg);
    // Activation loads go out before the weight prime: loads complete in
    // issue order, so waiting for them does not wait for the weights.
    uint4 xv[kRegStage];
    float4 zv[kRegStage][2];
#pragma unroll
    for (int u = 0; u < kRegStage; ++u) {
      const int i = threadIdx.x + u * kWG;
      xv[u] = x_group(tg, i, nt * n8x);
      z_group(tg, i, nt * n8z, zv[u][0], zv[u][1]);
    }
    const uint4 bk = book_load<D>(pj ? A.L.cb_up : A.L.cb_gate, P.K);
    __builtin_amdgcn_sched_barrier(0);  // keep the activation and book loads first
    vq.prime(codes, H / D, I, c0, I, x0, x1);
    if (!lr_late) lr.prime(V, I, c0, I, r, z0, z1);
    __syncthreads();
    if constexpr (NC > 1)
      book_store_copies<NC>(cbs, bk);
    else
      book_store<D>(cbs, bk);
#pragma unroll
    for (int u = 0; u < kRegStage; ++u) {
      const int i = threadIdx.x + u * kWG;
      if (i < nt * n8x) xs[(i / n8x) * ldx + i % n8x] = xv[u];
      if (i < nt * n8z) put_z(i / n8z, i % n8z, zv[u][0], zv[u][1]);
    }
    // groups beyond the register stage (many tokens): batches of 4 per
    // thread with their loads in flight together
    for (int i0 = threadIdx.x + kRegStage * kWG; i0 < nt * n8x; i0 += 4 * kWG) {
      uint4 v[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) v[u] = x_group(tg, i0 + u * kWG, nt * n8x);
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int i = i0 + u * kWG;
        if (i < nt * n8x) xs[(i / n8x) * ldx + i % n8x] = v[u];
      }
    }
    for (int i0 = threadIdx.x + kRegStage * kWG; i0 < nt * n8z; i0 += 2 * kWG) {
      float4 v[2][2];
#pragma unroll
      for (int u = 0; u < 2; ++u) z_group(tg, i0 + u * kWG, nt * n8z, v[u][0], v[u][1]);
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int i = i0 + u * kWG;
        if (i < nt * n8z) put_z(i / n8z, i % n8z, v[u][0], v[u][1]);
      }
    }
    __syncthreads();
    trace_mark(0);
    f32x4 acc[4];
    zero_acc(acc);
    if (lr_first) lr.run(zs, ldz, z0, nt, acc);
    if constexpr (LATE)
      vq.run(cbs, xs, ldx, x0, nt, acc, [&]() {
        if (lr_late) lr.prime(V, I, c0, I, r, z0, z1);
      });
    else
      vq.run(cbs, xs, ldx, x0, nt, acc);
    trace_mark(1);
    if (!lr_first) lr.run(zs, ldz, z0, nt, acc);
    store_acc(WsAccess(A, P), acc, nt, c0, I, [&](int t) { return gu + (((size_t)(R.s0 + tg + t) * 2 + pj) * P.ns + s) * I; });
    trace_mark(2);
  }

  // counts the tile done for (a, cg); the down tiles form p from the
  // n_proj ns partial sums of their columns
  publish(wsp<int>(A, P.o_gu_tick) + (a * P.ncg + cg) * kTickPad);
}

// Down tile (a, cgx, s) over split s of I, 256 output columns: for cgx <
// ncgh the VQ columns of H (Q^T p -> dn[s], nsd splits), else the low-rank
// columns of r (A_e^T p -> uap[s], nsdl splits: the coefficient bytes of a
// K-step are 16x the code bytes). Weight loads are issued before waiting
// for the expert's p.
// stage_p with U and NSC for 16 loads in flight at the plan's split count
template <bool RELU2>
__device__ __forceinline__ void stage_p_ns(const WsAccess& ws, const Plan& P, uint4* ps, int ld, int nt, int nquad,
                                           int slot0, int col0) {
  if (P.ns <= 1)
    stage_p<8, 1, RELU2>(ws, P, ps, ld, nt, nquad, slot0, col0);
  else if (P.ns <= 2)
    stage_p<4, 2, RELU2>(ws, P, ps, ld, nt, nquad, slot0, col0);
  else if (P.ns <= 4)
    stage_p<2, 4, RELU2>(ws, P, ps, ld, nt, nquad, slot0, col0);
  else
    stage_p<1, 8, RELU2>(ws, P, ps, ld, nt, nquad, slot0, col0);
}

template <bool RELU2, typename Prime, typename Stage, typename Run, typename Dst>
__device__ __forceinline__ void down_body(const Plan& P, const Args& A, const Routing& R, int a, int ks0, int ks1,
                                          int c0, int n_out, Prime prime, Stage stage, Run run, Dst dst,
                                          uint8_t* smem) {
  prime();
  // every gate/up tile of the column groups holding inputs [32 ks0, 32 ks1)
  const int cg0 = ks0 * 32 / kColsPerGroup, ncgw = (ks1 * 32 - 1) / kColsPerGroup - cg0 + 1;
  const int* tick = wsp<const int>(A, P.o_gu_tick) + (a * P.ncg + cg0) * kTickPad;
  wait_all(A, ncgw, [&](int i) { return ld_dev(tick + i * kTickPad) >= n_proj(P) * P.ns; });
  const int ld = (ks1 - ks0) * 8 + 1;
  uint4* ps = reinterpret_cast<uint4*>(smem);
  const WsAccess ws(A, P);
  for (int tg = 0; tg < R.ne; tg += P.nt_max) {
    const int nt = min(P.nt_max, R.ne - tg);
    if (tg > 0) prime();
    __syncthreads();
    stage();
    const int nquad = (ks1 - ks0) * 8, slot0 = R.s0 + tg, col0 = ks0 * 32;
    stage_p_ns<RELU2>(ws, P, ps, ld, nt, nquad, slot0, col0);
    __syncthreads();
    trace_mark(0);
    f32x4 acc[4];
    zero_acc(acc);
    run(ps, ld, nt, acc);
    store_acc(ws, acc, nt, c0, n_out, [&](int t) { return dst(R.s0 + tg + t); });
  }
}

template <bool RELU2, int NACC, typename Prime, typename Stage, typename Run, typename Finish>
__device__ __forceinline__ void down_body_wide(const Plan& P, const Args& A, const Routing& R, int a, int ks0, int ks1,
                                          Prime prime, Stage stage, Run run, Finish finish, uint8_t* smem) {
  prime();
  // every gate/up tile of the column groups holding inputs [32 ks0, 32 ks1)
  const int cg0 = ks0 * 32 / kColsPerGroup, ncgw = (ks1 * 32 - 1) / kColsPerGroup - cg0 + 1;
  const int* tick = wsp<const int>(A, P.o_gu_tick) + (a * P.ncg + cg0) * kTickPad;
  wait_all(A, ncgw, [&](int i) { return ld_dev(tick + i * kTickPad) >= n_proj(P) * P.ns; });
  const int ld = (ks1 - ks0) * 8 + 1;
  uint4* ps = reinterpret_cast<uint4*>(smem);
  const WsAccess ws(A, P);
  for (int tg = 0; tg < R.ne; tg += P.nt_max) {
    const int nt = min(P.nt_max, R.ne - tg);
    if (tg > 0) prime();
    __syncthreads();
    stage();
    const int nquad = (ks1 - ks0) * 8, slot0 = R.s0 + tg, col0 = ks0 * 32;
    stage_p_ns<RELU2>(ws, P, ps, ld, nt, nquad, slot0, col0);
    __syncthreads();
    trace_mark(0);
    f32x4 acc[NACC];
#pragma unroll
    for (int q = 0; q < NACC; q += 4) zero_acc(acc + q);
    run(ps, ld, nt, acc);
    finish(ws, acc, nt, R.s0 + tg);
  }
}

template <int D, bool RELU2>
__device__ void item_down_vq(const Plan& P, const Args& A, const RouteTab& RT, int a, int cgx, int s,
                             uint4* cbs, uint8_t* smem) {
  const Routing R = expert_of(P, RT, a);
  const int H = P.H, I = P.I, S = P.S, KS = I / 32;
  const int ks0 = s * KS / P.nsd, ks1 = (s + 1) * KS / P.nsd;
  const int c0 = cgx * kColsPerGroup + (threadIdx.x >> 6) * 64;
  const uint8_t* codes = A.L.codes_down + (size_t)R.e * (I / D) * H;
  float* dn = wsp<float>(A, P.o_dn) + (size_t)s * S * H;
  // d = 2 holds four code rows per K-step: half the steps in flight (same registers as d = 4)
  VqPipe<D, 2, D == 2 ? kPdVq / 2 : kPdVq> pipe;
  uint4 bk;
  down_body<RELU2>(P, A, R, a, ks0, ks1, c0, H,
            [&]() {
              bk = book_load<D>(A.L.cb_down, P.K);
              __builtin_amdgcn_sched_barrier(0);
              pipe.prime(codes, I / D, H, c0, H, ks0, ks1);
            },
            [&]() { book_store<D>(cbs, bk); },
            [&](const uint4* ps, int ld, int nt, f32x4* acc) { pipe.run(cbs, ps, ld, ks0, nt, acc); },
            [&](int slot) { return dn + (size_t)slot * H; }, smem);
  publish(wsp<int>(A, P.o_dn_done) + (R.e * (P.ncgh + 1) + cgx) * kTickPad);
}

// VQ down tile over two column groups (cgx, cgx + 1): as item_down_vq, each
// wave on 64 columns of both groups.
template <int D, bool RELU2>
__device__ void item_down_vq2(const Plan& P, const Args& A, const RouteTab& RT, int a, int cgx, int s,
                              uint4* cbs, uint8_t* smem) {
  const Routing R = expert_of(P, RT, a);
  const int H = P.H, I = P.I, S = P.S, KS = I / 32;
  const int ks0 = s * KS / P.nsd, ks1 = (s + 1) * KS / P.nsd;
  const int c0 = cgx * kColsPerGroup + (threadIdx.x >> 6) * 64;
  const uint8_t* codes = A.L.codes_down + (size_t)R.e * (I / D) * H;
  float* dn = wsp<float>(A, P.o_dn) + (size_t)s * S * H;
  VqPipe2<D, kPdVqWide, kBookCopies> pipe;
  uint4 bk;
  down_body_wide<RELU2, 8>(P, A, R, a, ks0, ks1,
               [&]() {
                 bk = book_load<D>(A.L.cb_down, P.K);
                 __builtin_amdgcn_sched_barrier(0);
                 pipe.prime(codes, I / D, H, c0, H, ks0, ks1);
               },
               [&]() { book_store_copies<kBookCopies>(cbs, bk); },
               [&](const uint4* ps, int ld, int nt, f32x4* acc) { pipe.run(cbs, ps, ld, ks0, nt, acc); },
               [&](const WsAccess& ws, const f32x4* acc, int nt, int slot0) {
                 store_acc(ws, acc, nt, c0, H, [&](int t) { return dn + (size_t)(slot0 + t) * H; });
                 store_acc(ws, acc + 4, nt, c0 + kColsPerGroup, H,
                           [&](int t) { return dn + (size_t)(slot0 + t) * H; });
               },
               smem);
  int* done = wsp<int>(A, P.o_dn_done) + (R.e * (P.ncgh + 1) + cgx) * kTickPad;
  drain_stores();
  __syncthreads();
  if (threadIdx.x == 0) {
    __hip_atomic_fetch_add(done, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (cgx + 1 < P.ncgh) __hip_atomic_fetch_add(done + kTickPad, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

// Low-rank down tile (a, cgr, s): partial A_e^T p over split s of I. The
// last of the expert's ncgr * nsdl tiles sums the splits into u_e[slot]
// (r values per slot) and flags the expert's low-rank part done.
template <bool RELU2>
__device__ void item_down_lr(const Plan& P, const Args& A, const RouteTab& RT, int a, int cgr, int s,
                             uint8_t* smem) {
  const Routing R = expert_of(P, RT, a);
  const int I = P.I, r = P.r, S = P.S, KS = I / 32, nsdl = P.nsdl;
  const int ks0 = s * KS / nsdl, ks1 = (s + 1) * KS / nsdl;
  const int c0 = cgr * kColsPerGroup + (threadIdx.x >> 6) * 64;
  const uint16_t* Ae = A.L.A_down + (size_t)R.e * I * r;
  float* uap = wsp<float>(A, P.o_uap);
  DensePipe<2, kPdDense> pipe;
  down_body<RELU2>(P, A, R, a, ks0, ks1, c0, r, [&]() { pipe.prime(Ae, r, c0, r, I, ks0, ks1); }, [&]() {},
            [&](const uint4* ps, int ld, int nt, f32x4* acc) { pipe.run(ps, ld, ks0, nt, acc); },
            [&](int slot) { return uap + ((size_t)s * S + slot) * r; }, smem);
  // the combine sums the nsdl partials of u_e itself
  publish(wsp<int>(A, P.o_dn_done) + (R.e * (P.ncgh + 1) + P.ncgh) * kTickPad);
}

// ---- dense bf16 expert weights (the uncompressed layer, Sec. 2.1, and the
// layer that keeps its down projection in bf16, Sec. 3.1) -------------------

// Dense gate/up tile (a, pj, cg, s): 256 output columns of W_pj[e] [H][I]
// over split s of the H inputs, partial sums into the same slots as the
// compressed tile, so the down tiles form p unchanged.
__device__ void item_gateup_dense(const Plan& P, const Args& A, const RouteTab& RT, int a, int pj, int cg,
                                  int s, uint8_t* smem) {
  const Routing R = expert_of(P, RT, a);
  const int H = P.H, I = P.I, B = P.B, KSX = H / 32;
  const int x0 = s * KSX / P.ns, x1 = (s + 1) * KSX / P.ns;
  const int c0 = cg * kColsPerGroup + (threadIdx.x >> 6) * 64;
  const uint16_t* W = reinterpret_cast<const uint16_t*>(pj ? A.L.codes_up : A.L.codes_gate) + (size_t)R.e * H * I;
  const int n8x = (x1 - x0) * 4, ldx = n8x + 1;
  uint4* xs = reinterpret_cast<uint4*>(smem);
  float* gu = wsp<float>(A, P.o_gu);
  const int* const slot_tok = RT.slot_tok;
  const rsrc_t xrs = make_rsrc(A.x, (uint32_t)B * H * 2);
  DensePipe<1, kPdDenseW> pipe;
  for (int tg = 0; tg < R.ne; tg += P.nt_max) {
    const int nt = min(P.nt_max, R.ne - tg), n = nt * n8x;
    pipe.prime(W, I, c0, I, H, x0, x1);
    __syncthreads();
    // x rows of the tile's tokens, 8-element groups, 4 loads in flight per thread
    for (int i0 = threadIdx.x; i0 < n; i0 += 4 * kWG) {
      uint4 v[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int i = i0 + u * kWG, ii = min(i, n - 1);
        const uint32_t o = (uint32_t)(((size_t)slot_tok[R.s0 + tg + ii / n8x] * H + x0 * 32 + 8 * (ii % n8x)) * 2);
        v[u] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(xrs, i < n ? o : kOob, 0, 0));
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int i = i0 + u * kWG;
        if (i < n) xs[(i / n8x) * ldx + i % n8x] = v[u];
      }
    }
    __syncthreads();
    f32x4 acc[4];
    zero_acc(acc);
    pipe.run(xs, ldx, x0, nt, acc);
    store_acc(WsAccess(A, P), acc, nt, c0, I,
              [&](int t) { return gu + (((size_t)(R.s0 + tg + t) * 2 + pj) * P.ns + s) * I; });
  }
  publish(wsp<int>(A, P.o_gu_tick) + (a * P.ncg + cg) * kTickPad);
}

// Dense down tile (a, cgx, s): 256 output columns of W_down[e] [I][H] over
// split s of I, partial sums into dn[s] as the VQ down tile.
template <bool RELU2>
__device__ void item_down_dense(const Plan& P, const Args& A, const RouteTab& RT, int a, int cgx, int s,
                                uint8_t* smem) {
  const Routing R = expert_of(P, RT, a);
  const int H = P.H, I = P.I, S = P.S, KS = I / 32;
  const int ks0 = s * KS / P.nsd, ks1 = (s + 1) * KS / P.nsd;
  const int c0 = cgx * kColsPerGroup + (threadIdx.x >> 6) * 64;
  const uint16_t* W = reinterpret_cast<const uint16_t*>(A.L.codes_down) + (size_t)R.e * I * H;
  float* dn = wsp<float>(A, P.o_dn) + (size_t)s * S * H;
  DensePipe<2, kPdDenseW> pipe;
  down_body<RELU2>(P, A, R, a, ks0, ks1, c0, H, [&]() { pipe.prime(W, H, c0, H, I, ks0, ks1); }, [&]() {},
            [&](const uint4* ps, int ld, int nt, f32x4* acc) { pipe.run(ps, ld, ks0, nt, acc); },
            [&](int slot) { return dn + (size_t)slot * H; }, smem);
  publish(wsp<int>(A, P.o_dn_done) + (R.e * (P.ncgh + 1) + cgx) * kTickPad);
}

// Combine tile (cgy, tq): output columns [256 cgy, +256) of tokens
// [tpc tq, tpc tq + tpc): y[t] = sum_j a_j sum_s dn[s][slot_j] + B^T u[t]
// with u[t] = sum_j a_j u_e[slot_j]. B rows are loaded before the
// wait; B^T u runs on MFMA with u as bf16 hi/lo. The partial sums are
// gathered in chunks of kCombineChunk loads in flight per thread.
// LRD: the layer has the low-rank down term (else y is the down sums alone).
// SK (large r, small batches): the tile covers 64 columns and its four waves
// split the ranks of B^T u, so each wave's share of B fits its prime before
// the wait; the waves' accumulators are summed through LDS.
template <bool LRD, bool SK>
__device__ void item_combine(const Plan& P, const Args& A, const Chain& C, const RouteTab& RT, int jc,
                             uint8_t* smem) {
  constexpr int NQ4 = SK ? 4 : 1;  // tiles per 256-column group
  constexpr int CW = 64 / NQ4;     // float4 column quads per token row of a tile
  const int cgq = jc % (P.ncgh * NQ4), tq = jc / (P.ncgh * NQ4);
  const int cgy = cgq / NQ4;
  const int H = P.H, r = LRD ? P.r : 0, k = P.k, S = P.S, nsd = P.nsd;
  const int t0 = tq * P.tpc, nt = min(P.tpc, P.B - t0);
  const int tid = threadIdx.x, w = tid >> 6;
  const int cbase = cgy * kColsPerGroup + (cgq % NQ4) * 64;
  const int KSR = (r + 31) / 32;
  // B is primed in full for r <= 128 (later K-steps load during the run);
  // SK: wave w primes K-steps [w KSR / 4, (w + 1) KSR / 4) of the tile's columns
  const int bk0 = SK ? w * KSR / 4 : 0, bk1 = SK ? (w + 1) * KSR / 4 : KSR;
  DensePipe<2, 4> bp;
  if (r > 0) bp.prime(A.L.B_down, H, cbase + (SK ? 0 : w * 64), H, r, bk0, bk1);

  const int* s_slot = RT.tok_slot + t0 * k;  // (t, j) -> slot of the tile's tokens
  const float* s_w_slot = RT.slot_w;
  const int* s_e_slot = RT.slot_e;
  float* ssq = reinterpret_cast<float*>(smem);                        // [16 tokens][64] sums of y^2
  float* dnb = ssq + kWG * 4;                                         // [nt][256] VQ down sums
  uint4* us = reinterpret_cast<uint4*>(dnb + kTokPass * kColsPerGroup);
  const int ntk = nt * k;
  const int nq = LRD ? KSR * 8 : 8, ld = KSR * 8 + 1;  // (no u rows without LRD)
  const int nsdl = P.nsdl, kd = k * nsd, ku = r > 0 ? k * nsdl : 0;
  constexpr int kB = kCombineChunk;
  // Term tables, built before the wait: per (token, selection j, split) the
  // row offset and weight of a low-rank partial of u_e (ku per token) and of
  // a VQ down partial (kd per token); kOob and 0 for an invalid selection.
  uint2* tab_u = reinterpret_cast<uint2*>(us + (size_t)P.tpc * ld);
  uint2* tab_d = tab_u + nt * ku;
  for (int i = tid; i < nt * (ku + kd); i += kWG) {
    const bool isu = i < nt * ku;
    const int ii = isu ? i : i - nt * ku;
    const int per = isu ? ku : kd, nsp = isu ? nsdl : nsd;
    const int t = ii / per, pp = ii % per, j = pp / nsp, ss = pp % nsp;
    const int sl = s_slot[t * k + j];
    const int slc = max(sl, 0);
    const uint32_t o = isu ? (uint32_t)(P.o_uap + ((size_t)ss * S + slc) * r * 4)
                           : (uint32_t)(P.o_dn + ((size_t)ss * S + slc) * H * 4);
    (isu ? tab_u : tab_d)[ii] = make_uint2(sl >= 0 ? o : kOob, __float_as_uint(sl >= 0 ? s_w_slot[slc] : 0.f));
  }
  {
    // every down tile of this column group (and every low-rank down tile) of
    // every expert of these tokens
    const int* dnd = wsp<const int>(A, P.o_dn_done);
    const int ncol = r > 0 ? 2 : 1, per_e = P.ncgh + 1;
    wait_all(A, ntk * ncol, [&](int i) {
      const int c = i % ncol, tj = i / ncol;
      const int sl = s_slot[tj];
      if (sl < 0) return true;
      return ld_dev(dnd + (s_e_slot[sl] * per_e + (c == 0 ? cgy : P.ncgh)) * kTickPad) >= (c == 0 ? nsd : P.ncgr * nsdl);
    });
  }
  trace_mark(2);
  // One pass with the loads in flight together: u[t] = sum_j a_j u_ej[slot_j]
  // (u_e from its nsdl partials) in quads of ranks (zero past r; staged as
  // bf16 hi/lo for B^T u), and the VQ down sums of this column group, one
  // float4 of 4 columns per item. Each item's terms (selection-major) are
  // cut into chunks of kB taken by separate threads, so a thread has at most
  // kB loads in flight; the chunk sums are added in order afterwards.
  const WsAccess ws(A, P);
  const int nu = r > 0 ? nt * nq : 0, nd = nt * CW;
  const int cu = (ku + kB - 1) / kB, cd = (kd + kB - 1) / kB;
  const int n_units = nu * cu + nd * cd;
  float4* part = reinterpret_cast<float4*>(smem + combine_part_offset(P));
  for (int unit = tid; unit < n_units; unit += kWG) {
    const bool isu = LRD && unit < nu * cu;
    const int uu = isu ? unit : unit - nu * cu;
    // chunk-major: neighbouring threads read neighbouring quads of one row
    const int nuu = max(nu, 1);  // (no low-rank terms: isu is never set)
    const int it = isu ? uu % nuu : uu % nd, c = isu ? uu / nuu : uu / nd;
    const int t = isu ? it / nq : it / CW, q = isu ? it % nq : 0;
    const int col = cbase + 4 * (it % CW);
    // the column's (or rank quad's) byte offset within a term's row; a
    // padding quad or column reads out of range
    const uint32_t ocol = isu ? (4 * q < r ? (uint32_t)(16 * q) : kOob) : (col < H ? (uint32_t)(4 * col) : kOob);
    const int nterm = isu ? ku : kd, p0 = c * kB;
    const uint2* tb = (isu ? tab_u + t * ku : tab_d + t * kd) + p0;
    uint2 e[kB];
#pragma unroll
    for (int b = 0; b < kB; ++b) e[b] = tb[min(b, nterm - 1 - p0)];
    float4 v[kB];
#pragma unroll
    for (int b = 0; b < kB; ++b) v[b] = ws.f4(p0 + b < nterm ? e[b].x + ocol : kOob);
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int b = 0; b < kB; ++b) acc = fma4(p0 + b < nterm ? __uint_as_float(e[b].y) : 0.f, v[b], acc);
    part[unit] = acc;
  }
  __syncthreads();
  for (int item = tid; item < nu + nd; item += kWG) {
    const bool isu = item < nu;
    const int nc = isu ? cu : cd, stride = isu ? nu : nd;
    const float4* pp = part + (isu ? item : nu * cu + (item - nu));
    float4 acc = pp[0];
    for (int c = 1; c < nc; ++c) {
      const float4 q = pp[c * stride];
      acc = make_float4(acc.x + q.x, acc.y + q.y, acc.z + q.z, acc.w + q.w);
    }
    if (isu)
      put_split_quad(us + (item / nq) * ld, item % nq, acc);
    else  // token row (item - nu) / CW, quad (item - nu) % CW, rows 256 floats apart
      reinterpret_cast<float4*>(dnb)[(item - nu) / CW * 64 + (item - nu) % CW] = acc;
  }
  trace_mark(3);
  const bool want_ssq = (P.flags & F_SSQ_OUT) != 0;
  if (want_ssq)
    for (int i = tid; i < kTokPass * 64; i += kWG) ssq[i] = 0.0f;
  __syncthreads();
  trace_mark(0);
  if (SK && r > 0) {
    // each wave's partial B^T u over its ranks, summed through LDS; thread
    // (i, l) writes token row 4 (l >> 4) + i, columns 4 (l & 15) .. + 3
    f32x4 acc[4];
    zero_acc(acc);
    bp.run(us, ld, 0, nt, acc);
    float* red4 = reinterpret_cast<float*>(smem + combine_lds(P));  // [4 waves][64 lanes][16]
    const int l = tid & 63;
#pragma unroll
    for (int q = 0; q < 4; ++q)
      *reinterpret_cast<float4*>(red4 + (w * 64 + l) * 16 + 4 * q) = make_float4(acc[q][0], acc[q][1], acc[q][2], acc[q][3]);
    __syncthreads();
    const int i = w, n = l & 15, t = 4 * (l >> 4) + i;
    if (t < nt && cbase + 4 * n < H) {
      float v[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        float sum = dnb[t * kColsPerGroup + 4 * n + q];
#pragma unroll
        for (int ww = 0; ww < 4; ++ww) sum += red4[(ww * 64 + l) * 16 + 4 * q + i];
        v[q] = sum;
      }
      *reinterpret_cast<float4*>(A.y + (size_t)(t0 + t) * H + cbase + 4 * n) = make_float4(v[0], v[1], v[2], v[3]);
      if (want_ssq) ssq[t * 64 + n] = v[0] * v[0] + v[1] * v[1] + v[2] * v[2] + v[3] * v[3];
    }
  } else if (r > 0) {
    // y = VQ sums + B^T u, written from the accumulators: token rows 4g + i,
    // columns 64 w + 4 n + q
    f32x4 acc[4];
    zero_acc(acc);
    bp.run(us, ld, 0, nt, acc);
    trace_mark(1);
    const int l = tid & 63, n = l & 15, g = l >> 4;
    const int c = w * 64 + 4 * n;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int t = 4 * g + i;
      if (t < nt && cbase + c < H) {
        const float4 d = *reinterpret_cast<const float4*>(dnb + t * kColsPerGroup + c);
        const float4 v = make_float4(d.x + acc[0][i], d.y + acc[1][i], d.z + acc[2][i], d.w + acc[3][i]);
        *reinterpret_cast<float4*>(A.y + (size_t)(t0 + t) * H + cbase + c) = v;
        if (want_ssq) ssq[t * 64 + w * 16 + n] = v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
      }
    }
  } else {
    for (int i = tid; i < nt * CW; i += kWG) {
      const int t = i / CW, col = cbase + 4 * (i % CW);
      if (col < H) {
        const float4 v = reinterpret_cast<const float4*>(dnb)[t * 64 + i % CW];
        *reinterpret_cast<float4*>(A.y + (size_t)(t0 + t) * H + col) = v;
        if (want_ssq) ssq[t * 64 + i % CW] = v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
      }
    }
  }
  if (want_ssq) {
    // this column tile's sum of y^2 per token (its 64 thread-slot partials
    // summed by one wave in a fixed tree), for the next layer's RMS
    // normalisation
    __syncthreads();
    const int l = tid & 63;
    for (int t = w; t < nt; t += 4) {
      const float sum = wave_sum(ssq[t * 64 + l]);
      if (l == 0) C.ssq_out[(size_t)(t0 + t) * C.nssq + cgq] = sum;
    }
  }
}

// ===========================================================================
// the two persistent kernels of a layer call
// ===========================================================================
// Brings the 9 64-byte lines of the kernel arguments (Plan, Args, Chain) into
// the scalar cache with loads issued back to back and one wait, so the
// fields read later hit instead of missing one line at a time. One asm
// statement: the loads' destinations are clobbered until the wait.
static_assert(sizeof(Plan) + sizeof(Args) + sizeof(Chain) > 8 * 64 &&
                  sizeof(Plan) + sizeof(Args) + sizeof(Chain) <= 9 * 64,
              "kernel arguments span 9 lines; update warm_kernargs");
__device__ __forceinline__ void warm_kernargs() {
#if __HIP_DEVICE_COMPILE__
  asm volatile(
      "s_load_dword s90, %0, 0x0\n\t"
      "s_load_dword s91, %0, 0x40\n\t"
      "s_load_dword s92, %0, 0x80\n\t"
      "s_load_dword s93, %0, 0xc0\n\t"
      "s_load_dword s94, %0, 0x100\n\t"
      "s_load_dword s95, %0, 0x140\n\t"
      "s_load_dword s96, %0, 0x180\n\t"
      "s_load_dword s97, %0, 0x1c0\n\t"
      "s_load_dword s98, %0, 0x200\n\t"
      "s_waitcnt lgkmcnt(0)" ::"s"(__builtin_amdgcn_kernarg_segment_ptr())
      : "s90", "s91", "s92", "s93", "s94", "s95", "s96", "s97", "s98", "memory");
#endif
}

// Each kernel clears the counters of the other kernel of the call before
// any of them is used again (the stream orders the two kernels): the flags
// this call's routing items set, and every expert tick of the shape (a call
// leaves no flag set, so calls of different batch sizes can share a
// workspace).
__device__ __forceinline__ void clear_ints(int* p, int n, int stride = 1) {
  for (int i = threadIdx.x; i < n; i += kWG) p[i * stride] = 0;
}

// Stacked decode step: a workgroup whose items are done reads its share
// (part of parts) of
// the next layer's routing-independent shared tensors (router weights, bases,
// code books), so the next layer's route kernel finds them in the last-level
// cache. One 4-byte load per 128-byte line; the loaded words only feed a
// barrier vote (which, if it ever held, would count into the sink counter).
__device__ void prefetch_next_layer(const Args& A, const Chain& C, int part, int parts) {
  unsigned acc = 0;
  // each thread's first line of every tensor, all loads issued together
  // (an absent tensor or a thread past its share reads the out-of-range
  // offset: no memory access)
#pragma unroll
  for (int j = 0; j < kPrefetchTensors; ++j) {
    const uint32_t n = C.pf[j] ? C.pf_bytes[j] : 0u;
    const uint32_t lines = (n + 127) / 128;
    const uint32_t l0 = (uint32_t)((uint64_t)lines * part / parts);
    const uint32_t l1 = (uint32_t)((uint64_t)lines * (part + 1) / parts);
    const uint32_t li = l0 + threadIdx.x;
    acc ^= __builtin_amdgcn_raw_buffer_load_b32(make_rsrc(C.pf[j], n), li < l1 ? li * 128 : kOob, 0, 0);
  }
  // shares of more lines than threads (few idle workgroups)
  for (int j = 0; j < kPrefetchTensors; ++j) {
    const uint32_t n = C.pf[j] ? C.pf_bytes[j] : 0u;
    const uint32_t lines = (n + 127) / 128;
    const uint32_t l0 = (uint32_t)((uint64_t)lines * part / parts);
    const uint32_t l1 = (uint32_t)((uint64_t)lines * (part + 1) / parts);
    const rsrc_t rs = make_rsrc(C.pf[j], n);
    for (uint32_t li = l0 + threadIdx.x + kWG; li < l1; li += kWG)
      acc ^= __builtin_amdgcn_raw_buffer_load_b32(rs, li * 128, 0, 0);
  }
  if (__syncthreads_or(acc == 0x5EED5EEDu) && threadIdx.x == 0) atomicAdd(ctr(A, C_SINK), 1);
}

// Routing-independent work and the routing itself: router chunks, z units,
// per-token select (the last one groups the slots), z reduce.
__global__ __launch_bounds__(kWG) void k_route(Plan P, Args A, Chain C) {
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
  warm_kernargs();
  if (blockIdx.x == 0 && (P.flags & F_EXPERTS)) {
    clear_ints(wsp<int>(A, P.o_gu_tick), P.E * P.ncg, kTickPad);
    clear_ints(wsp<int>(A, P.o_dn_done), P.E * (P.ncgh + 1), kTickPad);
  }
  // items in index order, one loop per kind (contiguous ranges)
  const int e_rc = P.n_rc, e_zc = e_rc + P.n_zc, e_sel = e_zc + P.n_sel;
  int j = blockIdx.x;
  for (; j < e_rc; j += gridDim.x) {
    __syncthreads();
    ItemTrace tr;
    const int nrt = P.nch_r * P.n_eg, jr = j % nrt;
    item_router_chunk(P, A, C, j, jr % P.nch_r, jr / P.nch_r, j / nrt, smem);
    tr.done(A, P, j, 0);
  }
  for (; j < e_zc; j += gridDim.x) {
    __syncthreads();
    ItemTrace tr;
    item_z(P, A, C, j - e_rc, smem);
    tr.done(A, P, j, 1);
  }
  for (; j < e_sel; j += gridDim.x) {
    __syncthreads();
    ItemTrace tr;
    item_select(P, A, j - e_zc, smem);
    tr.done(A, P, j, 2);
  }
  const int e_zr = P.n_pre - P.n_tb;
  for (; j < e_zr; j += gridDim.x) {
    __syncthreads();
    ItemTrace tr;
    item_z_reduce(P, A, j - e_sel);
    tr.done(A, P, j, 3);
  }
  for (; j < P.n_pre; j += gridDim.x) {
    __syncthreads();
    item_tbook(P, A, j - e_zr, smem);
  }
}

// Clears the routing kernel's flags (after calls that run k_route alone).
__global__ __launch_bounds__(kWG) void k_route_reset(Plan P, Args A) {
  clear_ints(wsp<int>(A, P.o_rc_flag), P.n_rc, kTickPad);
  clear_ints(wsp<int>(A, P.o_zc_flag), P.n_zc, kTickPad);
}

// Expert work of the active experts (count published by k_route): gate/up
// tiles, down tiles (waiting per expert for p), combine tiles (waiting for
// every down tile). DNW: column groups per VQ down tile; a separate
// instantiation keeps the wide tiles' registers out of the narrow one.
// MODE: expert-weight form (0 compressed, 1 dense down, 2 all dense).
// CSK: combine tiles split over the ranks of B^T u (large r, small batches).
// XPRE (batch 1): the token's x and z rows are loaded at kernel start, while
// the routing tables build, into an LDS area at the end of dynamic LDS.
// VAR: kVarRelu2 (up-only squared-ReLU experts) and kVarTBook (projection-
// code-book gate/up tiles) bits, each a separate instantiation so that the
// gated code-word kernels carry no code of either.
// Compiled for size (minsize): the explicitly unrolled pipelines keep their
// unrolling, the rest of each instantiation (about 100 KB of machine code)
// shrinks by about a tenth, and every layer form and batch measured faster
// than with the default optimisation.
template <int D, int DNW, int MODE, bool CSK, bool XPRE, int VAR>
__global__ __launch_bounds__(kWG) __attribute__((amdgpu_waves_per_eu(2), minsize)) void k_expert(Plan P, Args A,
                                                                                               Chain C) {
  constexpr bool RELU2 = (VAR & kVarRelu2) != 0, TBOOK = (VAR & kVarTBook) != 0;
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
  // the code book of the current item (zero-padded to 256 words), in
  // kBookCopies copies in the large-batch kernel
  constexpr int NC = DNW == 2 ? kBookCopies : 1;
  __shared__ uint4 cbs[MODE == 2 ? 1 : 256 * NC];
  warm_kernargs();
  const int tid = threadIdx.x;
  ItemTrace tr_route;
  // Small batches: the selections, one per lane of wave 0, are built into
  // the routing tables by that wave.
  const bool wave_routing = P.S <= 64;
  const int32_t* r_idx = (P.flags & F_ROUTE) ? A.topk_idx : A.idx_in;
  const float* r_w = (P.flags & F_ROUTE) ? A.topk_w : A.w_in;
  int sel_e = -1;
  float sel_w = 0.0f;
  if (wave_routing && tid < P.S) {
    sel_e = ld_dev(r_idx + tid);
    sel_w = ld_dev(r_w + tid);
  }
  if (blockIdx.x == 0) {
    clear_ints(wsp<int>(A, P.o_rc_flag), P.n_rc, kTickPad);
    clear_ints(wsp<int>(A, P.o_zc_flag), P.n_zc, kTickPad);
  }
  uint4* xpre = reinterpret_cast<uint4*>(smem + P.lds_expert - kXpreBytes);
  uint4* zpre = xpre + kXpreXGroups;
  uint4 xv[2];
  float4 zv[2];
  if constexpr (XPRE) {  // token 0's x groups and z rank groups (zero past r)
    const int nx = P.H / 8, nzq = P.r / 8;
    const float* zsrc = (P.flags & F_Z) ? A.z_out : A.z_in;
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int i = tid + u * kWG;
      xv[u] = i < nx ? reinterpret_cast<const uint4*>(A.x)[i] : make_uint4(0, 0, 0, 0);
    }
    const int pj = tid / kXpreZGroups, q = tid % kXpreZGroups;
    zv[0] = zv[1] = make_float4(0.f, 0.f, 0.f, 0.f);
    if (pj < 2 && q < nzq) {  // z [2][1][r], written by k_route's z reduce or given by the caller
      zv[0] = *reinterpret_cast<const float4*>(zsrc + (size_t)pj * P.r + 8 * q);
      zv[1] = *reinterpret_cast<const float4*>(zsrc + (size_t)pj * P.r + 8 * q + 4);
    }
  }
  // routing tables at the start of dynamic LDS, item LDS after them
  uint8_t* item_smem = smem + P.lds_routing;
  const RouteTab RT = wave_routing
                          ? build_routing_wave(P, (sel_e >= 0 && sel_e < P.E) ? sel_e : -1, sel_w, smem)
                          : build_routing(P, r_idx, r_w, smem, item_smem, (P.flags & F_ROUTE) != 0);
  if constexpr (XPRE) {  // visible to the items after their first barrier
#pragma unroll
    for (int u = 0; u < 2; ++u)
      if (tid + u * kWG < kXpreXGroups) xpre[tid + u * kWG] = xv[u];
    const int pj = tid / kXpreZGroups, q = tid % kXpreZGroups;
    if (pj < 2) {
      const float f[8] = {zv[0].x, zv[0].y, zv[0].z, zv[0].w, zv[1].x, zv[1].y, zv[1].z, zv[1].w};
      uint32_t h[8], lw[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        h[u] = rne_bf16(f[u]);
        lw[u] = rne_bf16(f[u] - bf(h[u]));
      }
      zpre[pj * kXpreZRow + 2 * q] = make_uint4(h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16),
                                                 h[6] | (h[7] << 16));
      zpre[pj * kXpreZRow + 2 * q + 1] = make_uint4(lw[0] | (lw[1] << 16), lw[2] | (lw[3] << 16),
                                                     lw[4] | (lw[5] << 16), lw[6] | (lw[7] << 16));
    }
  }
  tr_route.done(A, P, P.n_pre + P.max_act * (gateup_tiles_per_expert(P) + down_tiles_per_expert(P)) + P.n_cb +
                          blockIdx.x, 8);
  const int nact = RT.nact;
  const int nvq = (P.ncgh + DNW - 1) / DNW * P.nsd;  // VQ down tiles per expert
  const int tgu = gateup_tiles_per_expert(P), tdn = nvq + P.ncgr * P.nsdl;
  const int s_vq = P.ns_v;  // first gate/up split without code steps
  const int n_gu = nact * tgu, n_dn = nact * tdn, n_items = n_gu + n_dn + P.n_cb;
  // Items in index order, one loop per kind (the kinds are contiguous ranges):
  // each loop's invariant set-up is computed only by workgroups that enter it.
  int jp = blockIdx.x;
  for (; jp < n_gu; jp += gridDim.x) {
    __syncthreads();
    ItemTrace tr;
    const GateUpTile t = gateup_at(P, jp, nact, s_vq, gridDim.x);
    // a tile holding both code and low-rank steps runs the low-rank part
    // first in the second half of the grid, so the two workgroups sharing a
    // CU overlap LDS-bound and HBM-bound phases
    const bool lr_first = (int)(jp % gridDim.x) >= (int)(gridDim.x >> 1);
    if constexpr (MODE == 2) {
      item_gateup_dense(P, A, RT, t.a, t.pj, t.cg, t.s, item_smem);
    } else {
      // projection-code-book tiles (their own instantiations: the code-word
      // kernels carry none of their code)
      if constexpr (TBOOK) {
        if ((P.flags & F_TBOOK) && t.s < P.ns_v && expert_of(P, RT, t.a).ne <= kTBookTok) {
          item_gateup_t<D>(P, A, RT, t.a, t.pj, t.cg, t.s, item_smem);
          tr.done(A, P, P.n_pre + jp, 4);
          continue;
        }
      }
      item_gateup<D, DNW == 2, NC, XPRE, DNW == 2 ? kPdGateUpWide : kPdGateUp>(P, A, RT, t.a, t.pj, t.cg, t.s,
                                                                          lr_first, cbs, item_smem, xpre, zpre);
    }
    tr.done(A, P, P.n_pre + jp, 4);
  }
  for (; jp < n_gu + n_dn; jp += gridDim.x) {
    __syncthreads();
    ItemTrace tr;
    const int j = jp - n_gu, a = j / tdn, rem = j % tdn;
    if (rem < nvq) {
      if constexpr (MODE != 0)
        item_down_dense<RELU2>(P, A, RT, a, rem / P.nsd, rem % P.nsd, item_smem);
      else if constexpr (DNW == 2)
        item_down_vq2<D, RELU2>(P, A, RT, a, rem / P.nsd * 2, rem % P.nsd, cbs, item_smem);
      else
        item_down_vq<D, RELU2>(P, A, RT, a, rem / P.nsd, rem % P.nsd, cbs, item_smem);
      tr.done(A, P, P.n_pre + jp, 5);
    } else {
      item_down_lr<RELU2>(P, A, RT, a, (rem - nvq) / P.nsdl, (rem - nvq) % P.nsdl, item_smem);
      tr.done(A, P, P.n_pre + jp, 6);
    }
  }
  for (; jp < n_items; jp += gridDim.x) {
    __syncthreads();
    ItemTrace tr;
    item_combine<MODE == 0, CSK>(P, A, C, RT, jp - n_gu - n_dn, item_smem);
    tr.done(A, P, P.n_pre + jp, 7);
  }
  // the next layer's shared tensors, read by the workgroups that run no
  // combine (they finish while the combine tiles run)
  if (P.flags & F_PREFETCH) {
    const int G = gridDim.x, n_pf = G - min(P.n_cb, G);
    const int rank = ((int)blockIdx.x - (n_gu + n_dn) % G - min(P.n_cb, G) + 2 * G) % G;
    if (n_pf > 0 && rank < n_pf) prefetch_next_layer(A, C, rank, n_pf);
  }
}

// Zeroes n16 16-byte words at p (vector stores; a grid-stride loop).
__global__ __launch_bounds__(kWG) void k_zero16(uint4* p, size_t n16) {
  for (size_t i = (size_t)blockIdx.x * kWG + threadIdx.x; i < n16; i += (size_t)gridDim.x * kWG)
    p[i] = make_uint4(0, 0, 0, 0);
}

// x_next = bf16_rne(y / sqrt(mean(y^2) + eps)) per token. Rows of up to
// 4096 floats with H % 4 == 0 are held in registers: every load of the row is
// in flight at once and y is read once (a strided loop over the row, read
// twice, took 4.9 us at H = 2048); other rows take that loop.
__global__ __launch_bounds__(kWG) void k_rmsnorm(int H, const float* __restrict__ y, float eps,
                                                 uint16_t* __restrict__ xn) {
  __shared__ float part[4];
  const int t = blockIdx.x, tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const float* yr = y + (size_t)t * H;
  uint16_t* xr = xn + (size_t)t * H;
  constexpr int NV = 4;  // float4 per thread
  const bool vec = (H & 3) == 0 && H <= 4 * NV * kWG;
  float4 v[NV];
  float ss = 0.0f;
  if (vec) {
#pragma unroll
    for (int u = 0; u < NV; ++u) {
      const int i = 4 * (tid + u * kWG);
      v[u] = i < H ? *reinterpret_cast<const float4*>(yr + i) : make_float4(0.f, 0.f, 0.f, 0.f);
    }
#pragma unroll
    for (int u = 0; u < NV; ++u)
      ss = fmaf(v[u].w, v[u].w, fmaf(v[u].z, v[u].z, fmaf(v[u].y, v[u].y, fmaf(v[u].x, v[u].x, ss))));
  } else {
    for (int h = tid; h < H; h += kWG) ss = fmaf(yr[h], yr[h], ss);
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) ss += __shfl_xor(ss, o);
  if (lane == 0) part[w] = ss;
  __syncthreads();
  const float tot = part[0] + part[1] + part[2] + part[3];
  const float inv = 1.0f / sqrtf(tot / (float)H + eps);
  if (vec) {
#pragma unroll
    for (int u = 0; u < NV; ++u) {
      const int i = 4 * (tid + u * kWG);
      if (i < H)
        *reinterpret_cast<uint2*>(xr + i) = make_uint2(rne_bf16(v[u].x * inv) | (rne_bf16(v[u].y * inv) << 16),
                                                       rne_bf16(v[u].z * inv) | (rne_bf16(v[u].w * inv) << 16));
    }
  } else {
    for (int h = tid; h < H; h += kWG) xr[h] = (uint16_t)rne_bf16(yr[h] * inv);
  }
}

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------
const void* route_kernel() { return reinterpret_cast<const void*>(&k_route); }

template <int D, int DNW, int MODE, bool CSK, bool XPRE, int VAR>
const void* kx() {
  return reinterpret_cast<const void*>(&k_expert<D, DNW, MODE, CSK, XPRE, VAR>);
}

template <int D, int VAR>
const void* kx_compressed(bool csk, bool xpre) {
  return csk ? (xpre ? kx<D, 1, 0, true, true, VAR>() : kx<D, 1, 0, true, false, VAR>())
             : (xpre ? kx<D, 1, 0, false, true, VAR>() : kx<D, 1, 0, false, false, VAR>());
}

template <int VAR>
const void* kx_by_d(int d, bool csk, bool xpre) {
  return d == 8 ? kx_compressed<8, VAR>(csk, xpre) : d == 4 ? kx_compressed<4, VAR>(csk, xpre)
                                                            : kx_compressed<2, VAR>(csk, xpre);
}

// The instantiation a plan runs: the dense forms and the wide large-batch
// kernel per activation; the narrow compressed kernels per (d, csk, xpre)
// and activation, with projection-code-book tiles (d = 4, 8; never wide)
// where the plan has them.
const void* expert_kernel(const Plan& P) {
  const bool relu2 = (P.flags & F_UP_RELU2) != 0, tb = (P.flags & F_TBOOK) != 0;
  const bool csk = (P.flags & F_CB_SPLITK) != 0, xpre = (P.flags & F_XPRE) != 0;
  const int mode = expert_mode(P), d = P.d;
  if (mode == 2) return relu2 ? kx<8, 1, 2, false, false, kVarRelu2>() : kx<8, 1, 2, false, false, 0>();
  if (mode == 1)
    return d == 8 ? kx<8, 1, 1, false, false, 0>() : d == 4 ? kx<4, 1, 1, false, false, 0>()
                                                             : kx<2, 1, 1, false, false, 0>();
  if (d == 8 && dn_width(P) == 2) return relu2 ? kx<8, 2, 0, false, false, kVarRelu2>() : kx<8, 2, 0, false, false, 0>();
  if (tb && d != 2) {
    constexpr int T = kVarTBook, TR = kVarTBook | kVarRelu2;
    if (d == 8) return relu2 ? kx_compressed<8, TR>(csk, xpre) : kx_compressed<8, T>(csk, xpre);
    return relu2 ? kx_compressed<4, TR>(csk, xpre) : kx_compressed<4, T>(csk, xpre);
  }
  return relu2 ? kx_by_d<kVarRelu2>(d, csk, xpre) : kx_by_d<0>(d, csk, xpre);
}

// With a start/stop event pair the launch records them as part of the
// dispatch itself (the kernel's own begin and end), else a plain launch.
#define CARDAN_LAUNCH(kernel, grid, lds, st, ev0, ev1, ...)                                        \
  do {                                                                                            \
    if (ev0)                                                                                      \
      hipExtLaunchKernelGGL(kernel, dim3(grid), dim3(kWG), (uint32_t)(lds), st, ev0, ev1, 0,     \
                            __VA_ARGS__);                                                         \
    else                                                                                          \
      hipLaunchKernelGGL(kernel, dim3(grid), dim3(kWG), lds, st, __VA_ARGS__);                    \
  } while (0)

hipError_t launch_route(const Plan& P, const Args& A, const Chain& C, int grid, size_t lds, hipStream_t st,
                        hipEvent_t ev0, hipEvent_t ev1) {
  CARDAN_LAUNCH(k_route, grid, lds, st, ev0, ev1, P, A, C);
  return hipGetLastError();
}

hipError_t launch_route_reset(const Plan& P, const Args& A, hipStream_t st) {
  hipLaunchKernelGGL(k_route_reset, dim3(1), dim3(kWG), 0, st, P, A);
  return hipGetLastError();
}

hipError_t launch_expert(const Plan& P, const Args& A, const Chain& C, int grid, size_t lds, hipStream_t st,
                         hipEvent_t ev0, hipEvent_t ev1) {
  // the instantiation expert_kernel() names, launched with its own arguments
  const void* fn = expert_kernel(P);
  Plan p = P;
  Args a = A;
  Chain c = C;
  void* args[] = {&p, &a, &c};
  if (ev0) return hipExtLaunchKernel(fn, dim3(grid), dim3(kWG), args, lds, st, ev0, ev1, 0);
  return hipLaunchKernel(fn, dim3(grid), dim3(kWG), args, lds, st);
}

hipError_t launch_zero(void* p, size_t bytes, hipStream_t st) {
  const size_t n16 = bytes / 16;
  const int grid = (int)(n16 / kWG < 256 ? n16 / kWG + 1 : 256);
  hipLaunchKernelGGL(k_zero16, dim3(grid), dim3(kWG), 0, st, static_cast<uint4*>(p), n16);
  return hipGetLastError();
}

hipError_t launch_rmsnorm(hipStream_t st, int B, int H, const float* y, float eps, uint16_t* xn, hipEvent_t ev0,
                          hipEvent_t ev1) {
  if (ev0)
    hipExtLaunchKernelGGL(k_rmsnorm, dim3(B), dim3(kWG), 0, st, ev0, ev1, 0, H, y, eps, xn);
  else
    hipLaunchKernelGGL(k_rmsnorm, dim3(B), dim3(kWG), 0, st, H, y, eps, xn);
  return hipGetLastError();
}

}  // namespace cardan
