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
//   router chunks   (64 hidden rows x 64 experts), float64 partial logits
//   z items         four waves, each (basis, 64 ranks, split of H): partial
//                   U^T x on MFMA
//   select          per token: logits, top-k, gating
//   z reduce        256 outputs of z = U^T x each
//   gate/up tiles   (active expert a, gate|up, 256 columns, split of the
//                   joint axis [H inputs | r ranks]), partial sums; the last
//                   tile of (a, columns) forms p = silu(g) * u
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
constexpr int kRowsRouter = 64;     // hidden rows per router / shared-projection chunk
constexpr int kColsPerGroup = 256;  // output columns per expert tile (4 waves x 64)
constexpr int kTokPass = 16;        // token slots per MFMA pass (N of 16x16x32)
constexpr int kMaxE = 1024, kMaxK = 32, kMaxR = 512, kMaxB = 64;

// flags of one call
enum { F_ROUTE = 1, F_Z = 2, F_GROUP = 4, F_EXPERTS = 8 };

// counters at the start of the workspace, one per 64-byte slot: the status
// count of timed-out waits
enum { C_ERR = 0, C_NUM };
constexpr int kCtrStride = 16;      // ints between counters

struct Plan {
  int H, I, E, k, d, K, r, B;
  int S;          // routing slots = B * k
  int max_act;    // upper bound on active experts = min(E, S)
  int flags;
  int nch_r;      // router chunks of kRowsRouter hidden rows
  int n_eg;       // router expert groups of 64
  int nch_z;      // splits of H for the shared projection
  int z_sep;      // 1 when U_up is a different array from U_gate
  int ncg;        // gate/up column groups (I / 256, rounded up)
  int ns;         // gate/up splits of the joint K axis (H/32 + ceil(r/32) steps)
  int ncgh;       // VQ down column groups (H / 256, rounded up)
  int ncgr;       // low-rank down column groups (r / 256, rounded up)
  int nsd;        // VQ down splits of the I K-steps
  int nsdl;       // low-rank down splits of the I K-steps
  int nt_max;     // most token slots one expert tile stages (min(B, 16))
  int tpc;        // tokens per combine tile
  int n_cb;       // combine tiles
  // item counts of this call
  int n_rc, n_zc, n_sel, n_zr, n_pre;
  int n_rc_flags, n_zc_flags;  // flag slots (shape-wide maxima of n_rc, n_zc)
  // workspace byte offsets
  size_t o_ctr, o_rc_flag, o_zc_flag, o_gu_tick, o_gu_done, o_lr_tick, o_dn_done;  // counters
  size_t o_rl, o_zp, o_z, o_gu, o_p, o_dn, o_uap, o_u, total;
  size_t lds_route, lds_expert;  // dynamic LDS of the two kernels
  size_t lds_routing;            // routing tables at the start of k_expert's dynamic LDS
};

__host__ __device__ inline int gateup_tiles_per_expert(const Plan& P) { return 2 * P.ncg * P.ns; }
__host__ __device__ inline int down_tiles_per_expert(const Plan& P) {
  return P.ncgh * P.nsd + P.ncgr * P.nsdl;
}

// Cost of one low-rank K-step of a gate/up tile relative to one VQ K-step:
// a wave reads 64 x 32/d code bytes per VQ step and 32 x 64 bf16 (4 KB) per
// low-rank step.
__host__ __device__ inline int lr_step_cost(int d) { return 2 * d; }

// K-steps [k0, k1) of gate/up split s of n over the joint axis of KSX VQ
// steps and KSZ low-rank steps, balanced by bytes (lr_step_cost).
// (32-bit arithmetic: 64-bit division is a long software sequence on the GPU;
// total * n stays far below 2^31 for the supported shapes.)
__host__ __device__ inline void joint_split(int s, int n, int KSX, int KSZ, int d, int& k0, int& k1) {
  const int wz = lr_step_cost(d);
  const int total = KSX + KSZ * wz;
  auto step_at = [&](int c) -> int { return c <= KSX ? c : KSX + (c - KSX + wz - 1) / wz; };
  k0 = step_at(s * total / n);
  k1 = step_at((s + 1) * total / n);
}

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

}  // namespace cardan
