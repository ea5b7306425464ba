// Host-side checks of the launch planner over the supported shape domain,
// built with AddressSanitizer and UndefinedBehaviorSanitizer by
// tests/test_host_planner.py. Exits nonzero (and names the shape) on the
// first broken invariant.
//
// Invariants checked for every plan:
//   - workspace regions are 256-byte aligned, ordered and large enough for
//     the call's flags and counters;
//   - counter offsets depend on (H, I, E) only, so calls of any batch, rank,
//     block length or expert-weight form can share a workspace;
//   - the gate/up splits cover the joint axis [H inputs | r ranks] exactly,
//     in order, with no empty split; down splits lie in [1, I/32];
//   - the gate/up item mapping is a bijection from positions onto
//     (active expert, gate|up, column group, split) for several grid sizes,
//     and a position takes a code split exactly when its split index is
//     below ns_v;
//   - sizes that must fit 32-bit offsets do.
#include <stdio.h>
#include <stdlib.h>

#include <random>
#include <vector>

#include "../../paper_2609_21137_amd/csrc/cardan_plan.h"

using namespace cardan;

static int g_fail = 0;
static char g_ctx[256];

#define CHECK(c)                                                               \
  do {                                                                         \
    if (!(c)) {                                                                \
      fprintf(stderr, "FAIL %s: %s (line %d)\n", g_ctx, #c, __LINE__);         \
      if (++g_fail > 20) exit(1);                                              \
    }                                                                          \
  } while (0)

static int cdiv(int a, int b) { return (a + b - 1) / b; }

struct Counters {
  size_t rc, zc, gu, dn, rl;
};

static void check_plan(const cardan_shape& s, int B, int z_sep, int flags, Counters* ref) {
  const Plan P = make_plan(&s, B, z_sep, flags);
  snprintf(g_ctx, sizeof g_ctx, "H=%d I=%d E=%d k=%d d=%d K=%d r=%d B=%d z_sep=%d flags=%d", s.H, s.I, s.E,
           s.top_k, s.d, s.K, s.r, B, z_sep, flags);
  const int mode = expert_mode(P);
  const int KSX = P.H / 32, KSZ = cdiv(P.r, 32), KSD = P.I / 32;
  // layout: aligned, ordered, every region large enough
  const size_t offs[] = {P.o_ctr, P.o_rc_flag, P.o_zc_flag, P.o_gu_tick, P.o_dn_done, P.o_rl,
                         P.o_zp,  P.o_z,       P.o_gu,      P.o_dn,      P.o_uap,     P.total};
  for (size_t i = 0; i < sizeof offs / sizeof offs[0]; ++i) {
    CHECK(offs[i] % 256 == 0);
    if (i) CHECK(offs[i] >= offs[i - 1]);
  }
  CHECK(P.o_rc_flag - P.o_ctr >= (size_t)C_NUM * kCtrStride * 4);
  CHECK(P.n_rc <= P.n_rc_flags && P.n_zc <= P.n_zc_flags);
  CHECK(P.o_zc_flag - P.o_rc_flag >= (size_t)P.n_rc_flags * kTickPad * 4);
  CHECK(P.o_gu_tick - P.o_zc_flag >= (size_t)P.n_zc_flags * kTickPad * 4);
  CHECK(P.o_dn_done - P.o_gu_tick >= (size_t)P.E * P.ncg * kTickPad * 4);
  CHECK(P.o_rl - P.o_dn_done >= (size_t)P.E * (P.ncgh + 1) * kTickPad * 4);
  CHECK(P.o_zp - P.o_rl >= (size_t)P.nch_r * B * P.E * 8);
  CHECK(P.o_z - P.o_zp >= (size_t)2 * P.nq_z * B * P.r * 4);
  CHECK(P.nq_z * 4 >= P.nch_z && (P.nq_z - 1) * 4 < P.nch_z);
  CHECK(P.o_gu - P.o_z >= (size_t)2 * B * P.r * 4);
  CHECK(P.o_dn - P.o_gu >= (size_t)P.S * 2 * P.ns * P.I * 4);
  CHECK(P.o_uap - P.o_dn >= (size_t)P.nsd * P.S * P.H * 4);
  CHECK(P.total - P.o_uap >= (size_t)P.nsdl * P.S * P.r * 4);
  // counter offsets shared by every call on the shape's workspace
  const Counters c = {P.o_rc_flag, P.o_zc_flag, P.o_gu_tick, P.o_dn_done, P.o_rl};
  if (ref->rc == (size_t)-1) *ref = c;
  CHECK(c.rc == ref->rc && c.zc == ref->zc && c.gu == ref->gu && c.dn == ref->dn && c.rl == ref->rl);
  // splits
  CHECK(P.ns_v >= 1 && P.ns_v <= P.ns && P.ns_v <= KSX);
  CHECK(P.ns - P.ns_v <= KSZ);
  int prev = 0;
  for (int sp = 0; sp < P.ns; ++sp) {
    int k0, k1;
    joint_split(sp, P.ns, P.ns_v, KSX, KSZ, k0, k1);
    CHECK(k0 == prev);
    CHECK(k1 > k0);
    if (sp < P.ns_v) CHECK(k0 < KSX);  // a code split starts among the code steps
    prev = k1;
  }
  CHECK(prev == KSX + KSZ);
  CHECK(P.nsd >= 1 && P.nsd <= KSD);
  if (P.r > 0 && mode == 0) CHECK(P.nsdl >= 1 && P.nsdl <= KSD);
  CHECK(P.nt_max >= 1 && P.nt_max <= kTokPass && P.nt_max <= B);
  CHECK(P.tpc >= 1 && P.tpc <= kTokPass);
  CHECK(P.max_act >= 1 && P.max_act <= P.E && P.max_act <= P.S);
  CHECK(P.lds_routing >= (size_t)P.max_act * 16 + (size_t)4 * P.S * 4);
  CHECK(P.lds_expert > P.lds_routing);
  if (P.flags & F_XPRE) CHECK(B == 1 && mode == 0 && P.H <= 8 * kXpreXGroups);
  if (P.flags & F_DN_WIDE) CHECK(mode == 0 && P.d == 8);
  // projection code book: code splits whose T rows fit the tile's LDS area,
  // low-rank steps in splits of their own, the table last in the workspace
  if (P.flags & F_TBOOK) {
    const int bps = 32 / P.d;
    CHECK(mode == 0 && P.K % 4 == 0 && (P.flags & F_ROUTE) && !(P.flags & F_NORM_IN));
    CHECK(P.d != 2 && !(P.flags & F_DN_WIDE));
    CHECK(tbook_offset(P) >= P.o_uap + (size_t)P.nsdl * P.S * P.r * 4);
    CHECK(P.total == tbook_offset(P) + tbook_bytes(P) && tbook_bytes(P) <= kTBookMaxBytes);
    CHECK(P.n_tb == B * n_proj(P) * tbook_groups(P));
    CHECK(P.n_pre == P.n_rc + P.n_zc + P.n_sel + P.n_zr + P.n_tb);
    for (int sp = 0; sp < P.ns_v; ++sp) {
      int k0, k1;
      joint_split(sp, P.ns, P.ns_v, KSX, KSZ, k0, k1);
      CHECK(k1 <= KSX && (k1 - k0) * bps <= kTBookTileBlocks);
      CHECK((size_t)(k1 - k0) * bps * P.K * 4 <=
            P.lds_expert - P.lds_routing - ((P.flags & F_XPRE) ? kXpreBytes : 0));
    }
  } else {
    CHECK(P.n_tb == 0);
  }
  // item counts fit the kernels' int arithmetic
  const double items = (double)P.max_act * (gateup_tiles_per_expert(P) + down_tiles_per_expert(P)) + P.n_cb;
  CHECK(items < 2.0e9);
  // gate/up item mapping: a bijection for several grids and active counts
  const int n_tiles = gateup_tiles_per_expert(P);
  const int nacts[] = {1, P.max_act, (P.max_act + 1) / 2};
  const int grids[] = {1, 2, 7, 256, 512, 1024};
  std::vector<unsigned char> seen;
  for (int nact : nacts) {
    for (int G : grids) {
      const int n = nact * n_tiles;
      if (n > 200000) continue;
      seen.assign(n, 0);
      for (int p = 0; p < n; ++p) {
        const GateUpTile t = gateup_at(P, p, nact, P.ns_v, G);
        const bool ok = t.a >= 0 && t.a < nact && (t.pj == 0 || t.pj == 1) && t.cg >= 0 && t.cg < P.ncg &&
                        t.s >= 0 && t.s < P.ns && (t.pj == 1 || !(P.flags & F_UP_RELU2));
        CHECK(ok);
        if (!ok) continue;
        const int np = n_proj(P), id = ((t.a * np + (np == 2 ? t.pj : 0)) * P.ncg + t.cg) * P.ns + t.s;
        CHECK(!seen[id]);
        seen[id] = 1;
      }
    }
  }
}

int main(int argc, char** argv) {
  const int n_random = argc > 1 ? atoi(argv[1]) : 400;
  std::mt19937 rng(12345);
  auto pick = [&](std::initializer_list<int> v) { return *(v.begin() + rng() % v.size()); };
  long plans = 0;
  // named shapes of the workloads, then random shapes over the domain
  std::vector<cardan_shape> shapes = {
      {256, 128, 8, 2, 4, 16, 8},      {2048, 768, 128, 8, 8, 256, 128}, {4096, 1536, 64, 6, 8, 256, 256},
      {2048, 1408, 64, 6, 8, 256, 384}, {2048, 1024, 64, 8, 4, 256, 256}, {2816, 704, 128, 8, 8, 256, 384},
      {2688, 1856, 128, 6, 8, 256, 128}, {2688, 1856, 128, 6, 8, 256, 512}, {64, 32, 1, 1, 2, 1, 0},        {8192, 4096, 1024, 32, 8, 256, 512}};
  for (int i = 0; i < n_random; ++i) {
    cardan_shape s;
    s.d = pick({2, 4, 8});
    s.H = 64 * (1 + rng() % 96);
    s.I = 32 * (1 + rng() % 96);
    s.E = pick({1, 2, 8, 60, 64, 128, 256, 300, 1024});
    s.top_k = 1 + rng() % (s.E < 32 ? s.E : 32);
    s.K = pick({1, 2, 16, 255, 256});
    s.r = 8 * (rng() % 65);
    shapes.push_back(s);
  }
  for (const cardan_shape& s : shapes) {
    Counters ref = {(size_t)-1, 0, 0, 0, 0};
    const int all = F_ROUTE | F_Z | F_GROUP | F_EXPERTS;
    const int batches[] = {1, 2, 3, 4, 8, 15, 16, 17, 32, 63, 64};
    for (int B : batches) {
      for (int z_sep = 0; z_sep < 2; ++z_sep) {
        check_plan(s, B, z_sep, all | (s.r > 0 ? 0 : 0), &ref);
        ++plans;
      }
      check_plan(s, B, 0, F_ROUTE | F_GROUP | F_EXPERTS | F_DN_DENSE | F_Z, &ref);
      check_plan(s, B, 0, F_ROUTE | F_GROUP | F_EXPERTS | F_DN_DENSE | F_GU_DENSE, &ref);
      check_plan(s, B, 1, F_ROUTE, &ref);
      check_plan(s, B, 1, F_Z, &ref);
      check_plan(s, B, 1, F_GROUP | F_EXPERTS, &ref);
      // up-only squared-ReLU experts, compressed and dense
      check_plan(s, B, 0, all | F_UP_RELU2, &ref);
      check_plan(s, B, 0, F_ROUTE | F_GROUP | F_EXPERTS | F_DN_DENSE | F_GU_DENSE | F_UP_RELU2, &ref);
      // projection-code-book gate/up tiles (gated and up-only)
      check_plan(s, B, 0, all | F_TBOOK, &ref);
      check_plan(s, B, 1, all | F_TBOOK | F_UP_RELU2, &ref);
      plans += 9;
    }
  }
  printf("%ld plans checked, %d failures\n", plans, g_fail);
  return g_fail ? 1 : 0;
}
