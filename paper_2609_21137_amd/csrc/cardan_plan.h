// Launch plan, work-item space and workspace layout of one layer call.
//
// One call runs up to two persistent kernels, k_route then k_expert, whose
// workgroups walk static, ordered lists of work items: workgroup w takes
// items w, w + G, w + 2G, ... (G = grid size, never more workgroups than fit
// on the device at once). Every item only waits for items with smaller
// indices of the same kernel, so the earliest unfinished item never waits and
// the grid always makes progress; every wait is also bounded, so a broken
// invariant ends in an error count, never a hang.
//
// Item lists (k_route: router chunks, z items, select, z reduce; k_expert:
// gate/up, down, combine):
//   router chunks   (64 hidden rows x 64 experts x 4 tokens), float64
//                   partial logits
//   z items         (basis, 64 ranks, four consecutive splits of H, one per
//                   wave): partial U^T x on MFMA, the waves' sums added
//   select          per token: logits, top-k, gating
//   z reduce        256 outputs of z = U^T x each
//   gate/up tiles   (active expert a, gate|up, 256 columns, split of the
//                   joint axis [H inputs | r ranks]), partial sums; the down
//                   tiles form p = silu(g) * u from them (up-only experts: up
//                   tiles alone, p = relu(u)^2)
//   down tiles      (a, 256 output columns of [H | r], split of I); the last
//                   low-rank tile of an expert sums its splits into u_e
//   combine tiles   (256 output columns, group of tpc tokens)
// Every k_expert workgroup first groups the selections by expert in its own
// LDS (the routing tables), so items look up experts and slots in LDS.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/cardan.h"

namespace cardan {

constexpr int kWG = 256;            // threads per workgroup (4 wave64)
constexpr int kRowsRouter = 64;     // hidden rows per router chunk (16 per wave)
constexpr int kRouterTok = 4;       // tokens per router chunk item
constexpr int kColsPerGroup = 256;  // output columns per expert tile (4 waves x 64)
constexpr int kTokPass = 16;        // token slots per MFMA pass (N of 16x16x32)
constexpr int kMaxE = 1024, kMaxK = 32, kMaxR = 512, kMaxB = 64;
constexpr int kPdVq = 16;     // code K-steps in flight per wave (4 B per lane each)
constexpr int kPdVqWide = 8;  // the same in the down tiles of two column groups (large batches; 8 KB of
                              // codes per wave: measured faster than 12 and 16 steps at batch 16)
constexpr int kPdGateUp = 8;  // the same for gate/up tiles: half the bytes requested at once when
                              // every tile starts together, the rest as the first steps complete
constexpr int kPdGateUpWide = 16;  // gate/up code steps in flight in the large-batch kernel: 4 KB of
                                   // codes per wave, the bytes in flight HBM needs when every tile streams
constexpr int kPdDense = 2;   // dense K-steps in flight per wave (4 KB each)
constexpr int kCombineChunk = 16;  // terms per load batch in the combine
constexpr int kBookCopies = 4;     // code book copies in LDS of the large-batch expert kernel (d = 8)
constexpr int kLrDownSteps = 4;    // K-steps of a low-rank down tile when the plan would cut finer
constexpr int kSplitKRed = 4 * 64 * 16 * 4;  // [4 waves][64 lanes][16] float
// batch-1 operand area at the end of k_expert's dynamic LDS: x (H <= 4096,
// groups of 8 bf16) and z of both projections as bf16 hi/lo pairs per group
// of 8 ranks (r <= 512, zero past r)
constexpr int kXpreXGroups = 512, kXpreZGroups = 64, kXpreZRow = 2 * kXpreZGroups;
constexpr int kXpreBytes = (kXpreXGroups + 2 * kXpreZRow) * 16;
constexpr int kZRed = 4 * 64 * 16 * 4;       // z item: [4 waves][64 lanes][16] float sums
constexpr int kPdDenseW = 2;       // K-steps in flight per wave of a dense bf16 expert-weight tile
                                   // (measured faster than 3 at batch 1 and 16)
constexpr int kVarRelu2 = 1, kVarTBook = 2;  // k_expert variant bits (activation, gate/up form)
constexpr int kTBookBlocks = 64;       // blocks of x per projection-code-book item of k_route
constexpr int kTBookTok = 1;           // tokens of an expert a T-path gate/up tile takes
constexpr int kTBookTileBlocks = 48;   // blocks of a T-path tile (its T rows fill <= 48 KB of LDS at K = 256)
constexpr size_t kTBookMaxBytes = 64ull << 20;  // largest table the planner accepts


// flags of one call
enum { F_ROUTE = 1, F_Z = 2, F_GROUP = 4, F_EXPERTS = 8,
       F_DN_WIDE = 16,    // set by the plan: VQ down tiles over two column groups
       // dense bf16 expert weights in place of the compressed ones, passed in
       // the code pointers of the layer: W_down [E][I][H] as codes_down (no
       // low-rank down term), W_gate / W_up [E][H][I] as codes_gate / codes_up
       // (r = 0)
       F_DN_DENSE = 32, F_GU_DENSE = 64,
       F_CB_SPLITK = 128,  // set by the plan: combine tiles of 64 columns, ranks split over the waves
       F_XPRE = 256,       // set by the plan (batch 1): x and z staged once per workgroup
       // stacked decode step (Chain below): the layer's input is the previous
       // layer's output y, RMS-normalised by the route kernel, which also
       // writes it as bf16 x for the expert kernel
       F_NORM_IN = 1024,
       F_SSQ_OUT = 2048,   // combine tiles write per-token partial sums of y^2 for the next layer
       F_PREFETCH = 4096,  // idle expert-kernel workgroups touch the next layer's shared tensors
       // up-only experts with a squared-ReLU activation, p = max(u, 0)^2: no
       // gate tiles; the layer's gate pointers are not read
       F_UP_RELU2 = 8192,
       // projection code book (Sec. 4.2): k_route builds, per token and
       // input-side projection, T[b][k] = x[b*d .. b*d+d) . cb[k] (float32);
       // a gate/up code tile whose expert has at most kTBookTok tokens sums
       // T[b][J[b][j]] over its blocks instead of decoding code words on MFMA
       F_TBOOK = 16384 };

// counters at the start of the workspace, one per 64-byte slot: the status
// count of timed-out waits
enum { C_ERR = 0, C_SINK = 1, C_NUM };  // C_SINK: where prefetch loads are folded into one store
constexpr int kCtrStride = 16;      // ints between counters
constexpr int kTickPad = 32;        // ints between the tile counters (one 128-byte line each)

struct Plan {
  int H, I, E, k, d, K, r, B;
  int S;          // routing slots = B * k
  int max_act;    // upper bound on active experts = min(E, S)
  int flags;
  int nch_r;      // router chunks of kRowsRouter hidden rows
  int n_eg;       // router expert groups of 64
  int nch_z;      // splits of H for the shared projection (one wave each)
  int nq_z;       // z partials per value (nch_z / 4 rounded up: one per z item)
  int z_sep;      // 1 when U_up is a different array from U_gate
  int ncg;        // gate/up column groups (I / 256, rounded up)
  int ns;         // gate/up splits of the joint K axis (H/32 + ceil(r/32) steps)
  int ns_v;       // of which splits over the code steps (the rest: low-rank steps)
  int ncgh;       // VQ down column groups (H / 256, rounded up)
  int ncgr;       // low-rank down column groups (r / 256, rounded up)
  int nsd;        // VQ down splits of the I K-steps
  int nsdl;       // low-rank down splits of the I K-steps
  int nt_max;     // token slots an expert tile stages per pass (<= 16; more run in passes)
  int tpc;        // tokens per combine tile
  int n_cb;       // combine tiles
  // item counts of this call
  int n_rc, n_zc, n_sel, n_zr, n_pre;
  int n_rc_flags, n_zc_flags;  // flag slots (shape-wide maxima of n_rc, n_zc)
  int n_tb;       // projection-code-book items of k_route (F_TBOOK), the last of its items
  // workspace byte offsets
  size_t o_ctr, o_rc_flag, o_zc_flag, o_gu_tick, o_dn_done;  // counters
  size_t o_rl, o_zp, o_z, o_gu, o_dn, o_uap, total;
  size_t lds_route, lds_expert;  // dynamic LDS of the two kernels
  size_t lds_routing;            // routing tables at the start of k_expert's dynamic LDS
};

// Combine item LDS: reduction area [kWG] float4, VQ down sums [kTokPass][256]
// float, u operand rows [tpc][ld] uint4, term tables [tpc][k (nsdl + nsd)]
// uint2, then the per-chunk partial sums (float4); with F_CB_SPLITK the
// waves' B^T u accumulators follow (kSplitKRed bytes).
inline __host__ __device__ size_t combine_part_offset(const Plan& P) {
  const size_t ld = (size_t)(P.r + 31) / 32 * 8 + 1;
  const size_t o = (size_t)kWG * 16 + (size_t)kTokPass * kColsPerGroup * 4 + (size_t)P.tpc * ld * 16 +
                   (size_t)P.tpc * P.k * (P.nsdl + P.nsd) * 8;
  return (o + 15) & ~(size_t)15;
}
inline __host__ __device__ size_t combine_lds(const Plan& P) {
  const size_t nq = (size_t)(P.r + 31) / 32 * 8;
  const size_t cu = P.r > 0 ? ((size_t)P.k * P.nsdl + kCombineChunk - 1) / kCombineChunk : 0;
  const size_t cd = ((size_t)P.k * P.nsd + kCombineChunk - 1) / kCombineChunk;
  return combine_part_offset(P) + (size_t)P.tpc * (nq * cu + 64 * cd) * 16;
}

// Projection code book T (F_TBOOK): float32 [B][2][H/d][K] (gate, up) after
// the low-rank partial sums, the last region of the workspace.
__host__ __device__ inline size_t tbook_offset(const Plan& P) {
  return (P.o_uap + (size_t)P.nsdl * P.S * P.r * 4 + 255) & ~(size_t)255;
}
__host__ __device__ inline size_t tbook_bytes(const Plan& P) {
  return (size_t)P.B * 2 * (P.H / P.d) * P.K * 4;
}
__host__ __device__ inline int tbook_groups(const Plan& P) {
  return (P.H / P.d + kTBookBlocks - 1) / kTBookBlocks;
}

// expert-weight form of a call: 0 compressed, 1 dense down, 2 all dense
__host__ __device__ inline int expert_mode(const Plan& P) {
  return (P.flags & F_GU_DENSE) ? 2 : (P.flags & F_DN_DENSE) ? 1 : 0;
}
// projections with gate/up tiles: gate and up, or up alone
__host__ __device__ inline int n_proj(const Plan& P) { return (P.flags & F_UP_RELU2) ? 1 : 2; }
__host__ __device__ inline int gateup_tiles_per_expert(const Plan& P) { return n_proj(P) * P.ncg * P.ns; }
__host__ __device__ inline int dn_width(const Plan& P) { return (P.flags & F_DN_WIDE) ? 2 : 1; }
__host__ __device__ inline int down_tiles_per_expert(const Plan& P) {
  return (P.ncgh + dn_width(P) - 1) / dn_width(P) * P.nsd + P.ncgr * P.nsdl;
}

// K-steps [k0, k1) of gate/up split s over the joint axis of KSX code steps
// and KSZ low-rank steps: splits s < ns_v divide the code steps evenly, the
// remaining ns - ns_v splits divide the low-rank steps (with none left, the
// last code split also takes the low-rank steps).
__host__ __device__ inline void joint_split(int s, int ns, int ns_v, int KSX, int KSZ, int& k0, int& k1) {
  if (s < ns_v) {
    k0 = s * KSX / ns_v;
    k1 = (s + 1) * KSX / ns_v;
    if (s == ns_v - 1 && ns == ns_v) k1 = KSX + KSZ;
  } else {
    const int nl = ns - ns_v, sl = s - ns_v;
    k0 = KSX + sl * KSZ / nl;
    k1 = KSX + (sl + 1) * KSZ / nl;
  }
}

// Gate/up tile of position p. The tiles of splits s < s_vq read codes (LDS
// code-book lookups bound the CU), the others only coefficients (HBM bound).
// Workgroups b and b + G/2 share a CU when two are resident per CU, so code
// tiles take the first half of every grid-sized round of positions and
// coefficient tiles the second, each class in its natural (expert, gate|up,
// column group, split) order; once one class runs out the other fills every
// position. Gate/up tiles wait for nothing, so any order is deadlock-free.
// Up-only experts have up tiles alone (pj = 1).
struct GateUpTile {
  int a, pj, cg, s;
};
__host__ __device__ inline GateUpTile gateup_at(const Plan& P, int p, int nact, int s_vq, int G) {
  const int half = G >> 1, np = n_proj(P);
  const int n_v = nact * np * P.ncg * s_vq, n_l = nact * np * P.ncg * (P.ns - s_vq);
  const int r = p / G, w = p - r * G;
  const int v = r * half + (w < half ? w : half);  // code-preferring positions before p
  const int l = p - v;                             // coefficient-preferring positions before p
  // tiles of each class handed out before p (at most one class runs out)
  int cv = v, cl = l;
  if (v > n_v) {
    cv = n_v;
    cl = p - n_v;
  } else if (l > n_l) {
    cl = n_l;
    cv = p - n_l;
  }
  const bool code = w < half ? cv < n_v : !(cl < n_l);
  int i = code ? cv : cl;
  const int nsc = code ? s_vq : P.ns - s_vq;
  const int s = i % nsc + (code ? 0 : s_vq);
  i /= nsc;
  const int cg = i % P.ncg;
  i /= P.ncg;
  return np == 2 ? GateUpTile{i >> 1, i & 1, cg, s} : GateUpTile{i, 1, cg, s};
}

// Dynamic LDS limit of either kernel; a plan needing more is rejected.
constexpr size_t kLdsMax = 96 * 1024;

// Launch plan, item counts and workspace layout of one call (host only,
// cardan_planner.cpp); depends only on (shape, B, z_sep, flags). Flags with
// F_GU_DENSE plan r = 0. The shape must have passed the entry points' shape
// validation.
Plan make_plan(const cardan_shape* s, int B, int z_sep, int flags);

// Device pointers of one call.
struct Args {
  cardan_layer L;
  const uint16_t* x;      // [B][H]
  const int32_t* idx_in;  // routing given by the caller (grouping only), else NULL
  const float* w_in;
  int32_t* topk_idx;      // [B][k] routing outputs
  float* topk_w;
  const float* z_in;      // [2][B][r] caller z (expert path without F_Z)
  float* z_out;           // [2][B][r] z written by the z reduce items
  float* y;               // [B][H]
  uint8_t* ws;
};

// Stacked decode step: how a layer call chains to its neighbours (unused,
// all zero, for a single layer).
constexpr int kPrefetchTensors = 7;
struct Chain {
  const float* y_in;     // F_NORM_IN: previous layer's y [B][H]
  const float* ssq_in;   // F_NORM_IN: its partial sums of squares [B][nssq]
  uint16_t* x_norm;      // F_NORM_IN: the normalised input, written as bf16 [B][H]
  float* ssq_out;        // F_SSQ_OUT: this layer's partial sums of squares [B][nssq]
  float eps;             // RMS normalisation epsilon
  int nssq;              // partial sums per token (the combine's column tiles)
  const void* pf[kPrefetchTensors];        // F_PREFETCH: next layer's shared tensors
  uint32_t pf_bytes[kPrefetchTensors];
};

// Combine column tiles per token row (each writes one partial sum of squares
// under F_SSQ_OUT).
__host__ __device__ inline int combine_col_tiles(const Plan& P) {
  return P.ncgh * ((P.flags & F_CB_SPLITK) ? 4 : 1);
}

}  // namespace cardan
