// Launch planner of one layer call: split counts, tile shapes, item counts,
// workspace layout and LDS sizes, from the layer shape, the batch and the
// call's flags. Host code only (no HIP calls), so it also builds as a plain
// C++ translation unit for host-side checks.
#include <math.h>
#include <string.h>

#include <algorithm>

#include "cardan_plan.h"

namespace cardan {

namespace {

size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }

int ceil_div(int a, int b) { return (a + b - 1) / b; }


constexpr size_t kLdsBudget = 60 * 1024;  // operand staging limit when sizing the K splits

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
  size_t need = (size_t)kRouterTok * kRowsRouter * 4 + (size_t)4 * kRouterTok * 64 * 8 + 16;  // router chunk
  need = std::max(need, (size_t)kMaxE * 8 + kMaxK * (8 + 8 + 4 + 4) + (size_t)kWG * 8);  // select
  need = std::max(need, (size_t)(kMaxB * kMaxK + 2 * kMaxE + 4) * 4);   // grouping
  if (P.flags & F_Z)
    need = std::max(need, (size_t)4 * kTokPass * (ks_max(KSX, P.nch_z) * 4 + 1) * 16 + kZRed + kTokPass * 4);
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
  // T-path gate/up tiles: the T rows of their blocks for one token
  if (P.flags & F_TBOOK) need = std::max(need, (size_t)ks_max(KSX, P.ns_v) * (32 / P.d) * P.K * 4);
  return round256(need);
}

}  // namespace

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
  P.nch_r = ceil_div(P.H, kRowsRouter);
  P.n_eg = ceil_div(P.E, 64);
  P.z_sep = z_sep;
  // token rows a tile stages per pass: 8 above batch 8 (an expert with more
  // tokens streams its weights again per pass, rare at these batches), which
  // keeps the large-batch kernel's operand staging small enough for its
  // code book copies
  P.nt_max = B > 8 ? 8 : B;
  // combine tiles of up to B/16 tokens: sixteen per column group at large
  // batches, so the final gather is spread over more workgroups (one token
  // per tile at batch 16: the Nemotron-shaped layer 119.9 -> 117.9 us, the
  // Qwen3 one unchanged, against B/8)
  P.tpc = std::min(kTokPass, ceil_div(B, 16));
  const int KSX = P.H / 32, KSZ = ceil_div(P.r, 32), KSD = P.I / 32;
  P.nch_z = std::max(1, KSX / 2);                  // two K-steps of U per z unit (one wave)
  P.nq_z = ceil_div(P.nch_z, 4);                   // four units per z item, summed in LDS
  // Tile sizes: the expected active experts' weight bytes spread over a
  // nominal grid of 512 workgroups (2 per CU), kept between 16 and 64 KB per
  // tile, so small batches run every tile in one round and large ones stream
  // long tiles. Bytes per tile: a gate/up (expert, projection, 256 columns)
  // holds 256 (H/d) code bytes and 256 r * 2 coefficient bytes; a VQ down
  // (expert, 256 columns) 256 I/d; a low-rank down (expert, <= 256 ranks)
  // min(r, 256) I * 2. Dense bf16 weights: 256 H * 2 per gate/up and
  // 256 I * 2 per down (expert, 256 columns).
  const double exp_act = fmax(1.0, P.E * (1.0 - pow(1.0 - (double)P.k / P.E, (double)B)));
  const double npj = n_proj(P);  // gate and up, or up alone
  const double gu_expert = mode == 2 ? npj * P.H * P.I * 2 : npj * P.H * P.I / P.d + npj * P.I * P.r * 2;
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
    const double items = exp_act * (npj * P.ncg * P.ns + P.ncgh * P.nsd + P.ncgr * P.nsdl);
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
        const double items = exp_act * (npj * P.ncg * (nv + nl) + P.ncgh * P.nsd + P.ncgr * P.nsdl);
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
  // Projection code book: only for whole-layer calls on compressed weights
  // with d = 4 or 8, K % 4 == 0 (16-byte T rows) and a table of at most
  // kTBookMaxBytes, in the narrow expert kernel (no F_DN_WIDE); its code splits hold at most the
  // K-steps whose T rows fit kTBookTileBlocks blocks of 1 KB (K = 256), and
  // the low-rank steps get splits of their own (a T-path tile has no MFMA
  // accumulators to add them to)
  if ((P.flags & F_TBOOK) &&
      (mode != 0 || !(P.flags & F_ROUTE) || (P.flags & F_NORM_IN) || P.d == 2 || P.K % 4 ||
       tbook_bytes(P) > kTBookMaxBytes))
    P.flags &= ~F_TBOOK;
  if (P.flags & F_TBOOK) {
    const int bps = 32 / P.d;
    const int nbt = std::min(kTBookTileBlocks, (int)(48 * 1024 / ((size_t)P.K * 4)));
    const int ks_t = std::max(1, nbt / bps);
    const int nl = KSZ > 0 ? std::max(1, P.ns - P.ns_v) : 0;
    P.ns_v = std::min(KSX, std::max(P.ns_v, ceil_div(KSX, ks_t)));
    P.ns = P.ns_v + nl;
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
  const double items_all = exp_act * (npj * P.ncg * P.ns + P.ncgh * P.nsd + P.ncgr * P.nsdl);
  if (mode == 0 && items_all > 2 * 512.0 && P.ncgh > 1 && P.d == 8 && !(P.flags & F_TBOOK)) P.flags |= F_DN_WIDE;

  // Small batches at ranks above 128: B^T u streams more of B than a
  // combine tile primes before its wait, so the tiles shrink to 64 columns
  // with the ranks split over their four waves (each wave's share primed).
  if (mode == 0 && P.r > 128 && B <= 4) P.flags |= F_CB_SPLITK;
  P.n_cb = P.ncgh * ceil_div(B, P.tpc) * ((P.flags & F_CB_SPLITK) ? 4 : 1);
  // Batch 1: every gate/up tile's operands are the one token's x and z rows,
  // so each workgroup stages them once while it builds its routing tables
  if (mode == 0 && B == 1 && P.H <= 8 * kXpreXGroups) P.flags |= F_XPRE;

  const int z_items = (z_sep ? 2 : 1) * ceil_div(P.r, 64) * P.nq_z;
  P.n_rc = (flags & F_ROUTE) ? P.nch_r * P.n_eg * ceil_div(B, kRouterTok) : 0;
  P.n_zc = (flags & F_Z) ? z_items : 0;
  P.n_sel = (flags & F_ROUTE) ? B : 0;
  P.n_zr = (flags & F_Z) ? ceil_div(2 * B * P.r, kWG) : 0;
  P.n_tb = (P.flags & F_TBOOK) ? B * n_proj(P) * tbook_groups(P) : 0;
  P.n_pre = P.n_rc + P.n_zc + P.n_sel + P.n_zr + P.n_tb;

  // Counters first, at offsets that depend only on H, I and E (not on B,
  // r or the expert-weight form): a call leaves its expert ticks set until
  // the next call's k_route clears them, so every call on a workspace must
  // find them at the same place.
  P.n_rc_flags = P.nch_r * P.n_eg * ceil_div(kMaxB, kRouterTok);
  P.n_zc_flags = 2 * ceil_div(kMaxR, 64) * P.nq_z;
  size_t o = 0;
  P.o_ctr = o; o = align256(o + (size_t)C_NUM * kCtrStride * 4);
  P.o_rc_flag = o; o = align256(o + (size_t)P.n_rc_flags * kTickPad * 4);
  P.o_zc_flag = o; o = align256(o + (size_t)P.n_zc_flags * kTickPad * 4);
  P.o_gu_tick = o; o = align256(o + (size_t)P.E * ceil_div(P.I, kColsPerGroup) * kTickPad * 4);
  P.o_dn_done = o; o = align256(o + (size_t)P.E * (ceil_div(P.H, kColsPerGroup) + 1) * kTickPad * 4);
  P.o_rl = o; o = align256(o + (size_t)P.nch_r * B * P.E * 8);
  P.o_zp = o; o = align256(o + (size_t)2 * P.nq_z * B * P.r * 4);
  P.o_z = o; o = align256(o + (size_t)2 * B * P.r * 4);
  P.o_gu = o; o = align256(o + (size_t)P.S * 2 * P.ns * P.I * 4);
  P.o_dn = o; o = align256(o + (size_t)P.nsd * P.S * P.H * 4);
  P.o_uap = o; o = align256(o + (size_t)P.nsdl * P.S * P.r * 4);
  if (P.flags & F_TBOOK) o = tbook_offset(P) + tbook_bytes(P);
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

}  // namespace cardan
