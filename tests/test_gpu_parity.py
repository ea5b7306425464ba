"""GPU parity: the HIP path (through the C ABI) against the float64 oracle.

Bars: top-k indices identical as ordered lists (after checking that the
oracle's k-th/(k+1)-th logit margin exceeds 1e-9, so float64 accumulation on
both sides decides the same set); affinities within 1e-5; layer outputs
within max|y - y_ref| <= 2e-2 * max|y_ref|. A tighter headroom bar (1e-4,
from the float32-accumulation design) is checked separately so that a
numerics regression shows before it reaches the acceptance bar.
"""

import dataclasses
import sys
import zlib

import numpy as np
import pytest
import torch

import oracle.cardan_oracle as O
from paper_2609_21137_amd import synth
from paper_2609_21137_amd.configs import OTHER_MODELS_B1, QWEN3_B1, QWEN3_B16, TINY, WIDE_SKEW_B4

pytestmark = pytest.mark.gpu

TOL = 2e-2          # acceptance bar on max|dy| / max|y_ref|
HEADROOM = 1e-4     # float32 accumulation + split-bf16 operands


@pytest.fixture(scope="module")
def C():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_21137_amd import cardan
    return cardan


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _run_layer(C, w, L, x_bits, B=None):
    shape = C.make_shape(w.H, w.I, w.E, w.top_k, w.d, w.K, w.r)
    DL = C.DeviceLayer.from_numpy(L)
    x = C.bf16_tensor(x_bits)
    ws = C.new_workspace(shape, x.shape[0])
    y, idx, wt = C.moe_layer(shape, x, DL, ws=ws)
    torch.cuda.synchronize()
    assert C.workspace_status(ws) == 0, "an in-kernel wait timed out"
    return y.cpu().numpy().astype(np.float64), idx.cpu().numpy(), wt.cpu().numpy()


def _check(y, idx, wt, y_ref, idx_ref, a_ref, margin, tol=TOL):
    assert np.all(margin > 1e-9), margin.min()
    assert np.array_equal(idx, idx_ref), (idx, idx_ref)
    assert np.abs(wt - a_ref).max() <= 1e-5
    err = np.abs(y - y_ref).max() / np.abs(y_ref).max()
    assert err <= tol, err
    return err


LAYER_CASES = {
    "tiny_d4": (TINY, None),
    "qwen3_b1": (QWEN3_B1, None),
    "qwen3_b16": (QWEN3_B16, None),
    "wide_skew_b4": (WIDE_SKEW_B4, None),
    # the other gate+up shapes of the model table (Table 2), batch 1 and 16
    **{w.name: (w, None) for w in OTHER_MODELS_B1},
    **{w.name + "_b16": (dataclasses.replace(w, B=16, name=w.name + "_b16"), None) for w in OTHER_MODELS_B1},
}


@pytest.mark.parametrize("case", list(LAYER_CASES))
def test_moe_layer_parity(C, case):
    w, _ = LAYER_CASES[case]
    _say(f"[parity] {case} H={w.H} I={w.I} E={w.E} k={w.top_k} d={w.d} r={w.r} B={w.B}")
    L = synth.workload_layer(w)
    x = synth.workload_input(w)
    y_ref, idx_ref, a_ref, margin = O.moe_layer_factored(x, L, w.top_k, w.d)
    y, idx, wt = _run_layer(C, w, L, x)
    err = _check(y, idx, wt, y_ref, idx_ref, a_ref, margin)
    _say(f"[parity] {case} normalised max error {err:.3e}")
    assert err <= HEADROOM, err


def test_tiny_against_dense_reconstruction(C):
    """O1 (dense reconstruction) directly, on the tiny layer at B=3."""
    w = TINY
    L = synth.workload_layer(w)
    x = synth.make_input(w.H, 3, w.seed, step=7)
    y_ref, idx_ref, a_ref, margin = O.moe_layer(x, L, w.top_k, w.d)
    y, idx, wt = _run_layer(C, w, L, x)
    _check(y, idx, wt, y_ref, idx_ref, a_ref, margin, tol=HEADROOM)


def test_route_topk_and_shared_proj(C):
    for w in (TINY, QWEN3_B16, WIDE_SKEW_B4):
        _say(f"[route] {w.name}")
        L = synth.workload_layer(w)
        x_bits = synth.workload_input(w)
        shape = C.shape_of(w)
        x = C.bf16_tensor(x_bits)
        idx, wt = C.route_topk(shape, x, C.bf16_tensor(L["router_w"]),
                               torch.from_numpy(L["router_bias"]).cuda())
        z = C.shared_proj(shape, x, C.bf16_tensor(L["U_gate"]))
        torch.cuda.synchronize()
        idx_ref, a_ref, margin, _ = O.route(x_bits, L["router_w"], L["router_bias"], w.top_k)
        assert np.all(margin > 1e-9)
        assert np.array_equal(idx.cpu().numpy(), idx_ref)
        assert np.abs(wt.cpu().numpy() - a_ref).max() <= 1e-5
        z_ref = O.shared_proj(x_bits, L["U_gate"])
        zz = z.cpu().numpy()
        assert np.abs(zz[0] - z_ref).max() <= 1e-5 * np.abs(z_ref).max()
        assert np.array_equal(zz[0], zz[1])


def test_separate_up_basis_and_expert_ffn_entry(C):
    """U_up != U_gate, and the split entry points route_topk -> shared_proj
    -> vq_lr_expert_ffn against the oracle."""
    w = TINY
    L = synth.make_layer(w.H, w.I, w.E, w.d, w.K, w.r, seed=5, separate_up_basis=True)
    x_bits = synth.make_input(w.H, 4, seed=5)
    shape = C.shape_of(w)
    DL = C.DeviceLayer.from_numpy(L)
    x = C.bf16_tensor(x_bits)
    idx, wt = C.route_topk(shape, x, DL.tensors["router_w"], DL.tensors["router_bias"])
    z = C.shared_proj(shape, x, DL.tensors["U_gate"], DL.tensors["U_up"])
    y = C.vq_lr_expert_ffn(shape, x, idx, wt, z, DL)
    y2, idx2, wt2 = C.moe_layer(shape, x, DL)
    torch.cuda.synchronize()
    y_ref, idx_ref, a_ref, margin = O.moe_layer(x_bits, L, w.top_k, w.d)
    _check(y.cpu().numpy(), idx.cpu().numpy(), wt.cpu().numpy(), y_ref, idx_ref, a_ref, margin,
           tol=HEADROOM)
    assert torch.equal(y, y2) and torch.equal(idx, idx2)


def _caller_routing(w, case):
    if case == "one":  # batch 1 (staged token), one expert twice
        return np.array([[4, 4]], dtype=np.int32), np.array([[0.3, 0.7]], dtype=np.float32)
    if case == "few":  # 6 selections: one wave builds the routing tables
        idx = np.array([[3, 5], [7, 7], [-1, w.E + 3]], dtype=np.int32)
        wts = np.array([[0.6, 0.4], [0.25, 0.75], [0.5, 0.5]], dtype=np.float32)
        return idx, wts
    # 80 selections (the block-wide builder): random experts with repeats
    # within a token, negative and too-large indices
    rng = np.random.default_rng(11)
    idx = rng.integers(0, w.E, size=(40, 2)).astype(np.int32)
    idx[rng.random(idx.shape) < 0.1] = -1
    idx[rng.random(idx.shape) < 0.05] = w.E + 1
    idx[::7, 1] = idx[::7, 0]
    wts = rng.random(idx.shape).astype(np.float32)
    return idx, wts


@pytest.mark.parametrize("case", ["one", "few", "many"])
def test_given_routing_with_invalid_and_duplicate_entries(C, case):
    """vq_lr_expert_ffn with caller routing: an out-of-range index contributes
    nothing; a repeated expert counts twice."""
    w = TINY
    L = synth.workload_layer(w)
    shape = C.shape_of(w)
    DL = C.DeviceLayer.from_numpy(L)
    idx, wts = _caller_routing(w, case)
    x_bits = synth.make_input(w.H, idx.shape[0], seed=6)
    x = C.bf16_tensor(x_bits)
    z = C.shared_proj(shape, x, DL.tensors["U_gate"])
    y = C.vq_lr_expert_ffn(shape, x, torch.from_numpy(idx).cuda(),
                           torch.from_numpy(wts).cuda(), z, DL)
    torch.cuda.synchronize()
    ok = (idx >= 0) & (idx < w.E)
    keep = np.where(ok, idx, 0)
    wref = np.where(ok, wts, 0.0).astype(np.float64)
    y_ref = O.expert_ffn(x_bits, keep, wref, L, w.d)
    err = np.abs(y.cpu().numpy() - y_ref).max() / np.abs(y_ref).max()
    assert err <= HEADROOM, err


@pytest.mark.parametrize("B", [40, 64])
def test_given_routing_block_builders(C, B):
    """Caller routing with repeats and invalid indices through the
    block-wide routing-table builder at B * k = 240 and 384 selections (more
    than one per thread)."""
    H, I, E, k, d, K, r = 256, 128, 16, 6, 8, 64, 8
    w = TINY.__class__(f"routing_b{B}", H=H, I=I, E=E, top_k=k, d=d, K=K, r=r, B=B, seed=0)
    L = synth.make_layer(H, I, E, d, K, r, seed=17)
    shape = C.shape_of(w)
    DL = C.DeviceLayer.from_numpy(L)
    rng = np.random.default_rng(B)
    idx = rng.integers(0, E, size=(B, k)).astype(np.int32)
    idx[rng.random(idx.shape) < 0.08] = -1
    idx[rng.random(idx.shape) < 0.04] = E + 2
    idx[::5, 1] = idx[::5, 0]  # an expert twice within a token
    wts = rng.random(idx.shape).astype(np.float32)
    x_bits = synth.make_input(H, B, seed=9)
    x = C.bf16_tensor(x_bits)
    z = C.shared_proj(shape, x, DL.tensors["U_gate"])
    y = C.vq_lr_expert_ffn(shape, x, torch.from_numpy(idx).cuda(), torch.from_numpy(wts).cuda(), z, DL)
    torch.cuda.synchronize()
    ok = (idx >= 0) & (idx < E)
    y_ref = O.expert_ffn(x_bits, np.where(ok, idx, 0), np.where(ok, wts, 0.0).astype(np.float64), L, d)
    err = np.abs(y.cpu().numpy() - y_ref).max() / np.abs(y_ref).max()
    assert err <= HEADROOM, err


def test_component_isolation(C):
    """Zero code books (pure low rank) and r = 0 (pure VQ)."""
    w = TINY
    L = synth.workload_layer(w)
    Lz = dict(L)
    Lz["cb_gate"] = Lz["cb_up"] = Lz["cb_down"] = np.zeros_like(L["cb_gate"])
    for key in ("V_gate", "V_up", "A_down"):
        Lz[key] = synth.to_bf16_bits(O.bf16_to_f64(L[key]) * 50.0)
    x = synth.make_input(w.H, 2, seed=3)
    for lay, name in ((Lz, "low-rank only"), (None, "vq only")):
        if lay is None:
            lay = synth.make_layer(w.H, w.I, w.E, w.d, w.K, 0, seed=3)
            ww = dataclasses.replace(w, r=0, name="r0")
        else:
            ww = w
        _say(f"[isolation] {name}")
        y_ref, idx_ref, a_ref, margin = O.moe_layer(x, lay, ww.top_k, ww.d)
        y, idx, wt = _run_layer(C, ww, lay, x)
        _check(y, idx, wt, y_ref, idx_ref, a_ref, margin, tol=HEADROOM)


EDGE_SHAPES = [
    # name, H, I, E, k, d, K, r, B
    ("ragged_cols_d8", 192, 96, 10, 3, 8, 256, 8, 5),
    ("one_expert_k1", 128, 64, 1, 1, 8, 7, 16, 2),
    ("e100_k1_d4", 256, 160, 100, 1, 4, 33, 24, 7),
    ("max_batch_64", 256, 128, 16, 4, 8, 64, 8, 64),
    ("rank_512", 1024, 256, 8, 2, 8, 256, 512, 3),
    ("k32_wide", 512, 288, 40, 32, 4, 256, 40, 2),
    # more than 256 experts: exact one-wave radix top-k (5 and 16 keys a lane)
    ("e300_k8", 256, 64, 300, 8, 8, 64, 8, 3),
    ("e1024_k32", 128, 32, 1024, 32, 4, 16, 8, 2),
    # deep inputs: 16 code splits (SiLU staged from 34 partials in 3 rounds),
    # 128 router chunks
    ("deep_h8192", 8192, 64, 8, 2, 8, 64, 16, 1),
    # 512 selections: block-wide routing tables, 16-token combine tiles
    ("b64_e128_k8", 256, 128, 128, 8, 8, 64, 16, 64),
    # large-batch kernel (down tiles over two column groups) with an odd
    # number of column groups, the last one ragged (704 = 2 x 256 + 192)
    ("wide_tiles_ragged", 704, 768, 128, 8, 8, 256, 128, 32),
    # combine tiles of 64 columns with the ranks of B^T u split over the
    # waves (r > 128, B <= 4), ragged H: tiles past H, five rank K-steps
    ("splitk_combine_ragged", 320, 288, 10, 3, 8, 64, 160, 4),
    ("splitk_combine_d4_b1", 512, 256, 16, 4, 4, 256, 264, 1),
    # d = 2 (four 4-byte code words per MFMA operand), including the
    # paper's VQ-only comparison point (d, r) = (2, 0) at the Qwen3 shape
    ("d2_small", 256, 160, 8, 2, 2, 16, 8, 3),
    ("qwen3_d2_r0_b1", 2048, 768, 128, 8, 2, 256, 0, 1),
    ("qwen3_d2_r0_b16", 2048, 768, 128, 8, 2, 256, 0, 16),
    ("d2_r160_b2", 512, 288, 16, 4, 2, 64, 160, 2),
    # corners of the (d, r) sweep at the Qwen3 shape
    ("qwen3_d4_r512_b16", 2048, 768, 128, 8, 4, 256, 512, 16),
    ("qwen3_d8_r0_b16", 2048, 768, 128, 8, 8, 256, 0, 16),
]


@pytest.mark.parametrize("case", EDGE_SHAPES, ids=[c[0] for c in EDGE_SHAPES])
def test_edge_shapes(C, case):
    name, H, I, E, k, d, K, r, B = case
    _say(f"[edge] {case}")
    seed = zlib.crc32(name.encode()) % 1000
    L = synth.make_layer(H, I, E, d, K, r, seed=seed)
    for key in ("cb_gate", "cb_up", "cb_down"):
        L[key] = synth.to_bf16_bits(O.bf16_to_f64(L[key]) * 10.0)
    x = synth.make_input(H, B, seed=seed)
    w = TINY.__class__(name, H=H, I=I, E=E, top_k=k, d=d, K=K, r=r, B=B, seed=0)
    y_ref, idx_ref, a_ref, margin = O.moe_layer_factored(x, L, k, d)
    y, idx, wt = _run_layer(C, w, L, x)
    _check(y, idx, wt, y_ref, idx_ref, a_ref, margin, tol=HEADROOM)


def test_duplicate_tokens_fill_token_passes(C):
    """32 identical tokens: every selected expert holds 32 slots (two MFMA
    token passes); all rows must agree with the oracle and with each other."""
    w = TINY
    L = synth.workload_layer(w)
    x = np.repeat(synth.make_input(w.H, 1, seed=4), 32, axis=0)
    y_ref, idx_ref, a_ref, margin = O.moe_layer_factored(x, L, w.top_k, w.d)
    y, idx, wt = _run_layer(C, w, L, x)
    _check(y, idx, wt, y_ref, idx_ref, a_ref, margin, tol=HEADROOM)
    assert np.abs(y - y[0]).max() <= 1e-6 * np.abs(y).max()


def test_batch_rows_independent_and_repeatable(C):
    w = QWEN3_B16
    L = synth.workload_layer(w)
    x = synth.workload_input(w)
    y16, idx16, _ = _run_layer(C, w, L, x)
    y16b, _, _ = _run_layer(C, w, L, x)
    assert np.array_equal(y16, y16b), "repeat runs differ"
    for t in (0, 7, 15):
        y1, idx1, _ = _run_layer(C, w, L, x[t:t + 1])
        assert np.array_equal(idx1[0], idx16[t])
        assert np.abs(y1[0] - y16[t]).max() <= 1e-5 * np.abs(y16[t]).max()


def test_workspace_reused_across_batch_sizes(C):
    """One workspace serves calls of different batch sizes in turn. Every
    call must find the synchronisation counters cleared whatever batch ran
    before it (their offsets depend on the layer shape only), so each result
    equals that of a fresh workspace bit for bit."""
    w = QWEN3_B16
    L = synth.workload_layer(w)
    x = synth.workload_input(w)
    shape = C.make_shape(w.H, w.I, w.E, w.top_k, w.d, w.K, w.r)
    DL = C.DeviceLayer.from_numpy(L)
    ws = C.new_workspace(shape, x.shape[0])
    for B in (16, 1, 16, 3, 1, 8, 16):
        _say(f"workspace reuse: batch {B}")
        y, idx, wt = C.moe_layer(shape, C.bf16_tensor(x[:B]), DL, ws=ws)
        torch.cuda.synchronize()
        assert C.workspace_status(ws) == 0, "an in-kernel wait timed out"
        y_f, idx_f, wt_f = _run_layer(C, w, L, x[:B])
        assert np.array_equal(idx.cpu().numpy(), idx_f)
        assert np.array_equal(wt.cpu().numpy(), wt_f)
        assert np.array_equal(y.cpu().numpy().astype(np.float64), y_f)


@pytest.mark.parametrize("H", [2048, 2052, 4096, 1001, 8192])  # row in registers; strided loop
def test_rmsnorm(C, H):
    rng = np.random.default_rng(H)
    y = rng.standard_normal((16, H)).astype(np.float32) * 0.3
    xn = C.rmsnorm_bf16(torch.from_numpy(y).cuda(), 1e-6)
    torch.cuda.synchronize()
    got = O.bf16_to_f64(C.bf16_bits(xn))
    ref = O.rmsnorm(y, 1e-6)
    # within one bf16 rounding step of the float64 value
    assert np.all(np.abs(got - ref) <= np.abs(ref) * 2.0 ** -8 + 1e-30)


@pytest.mark.parametrize("k", [4, 6])
def test_exact_and_single_precision_ties(C, k):
    """Logits that tie exactly (lower index first) and logits that differ only
    below single precision (the exact comparison decides): the top-k must
    still match the oracle element for element."""
    import dataclasses
    w = dataclasses.replace(TINY, top_k=k)
    L = synth.workload_layer(w)
    H, E = w.H, w.E
    wr = np.zeros((H, E), dtype=np.float64)
    wr[0] = [1.0, 1.0, 1.0, 0.5, 0.25, 0.25, -1.0, 0.0]
    wr[1, 2] = 1.0
    L["router_w"] = synth.to_bf16_bits(wr)
    L["router_bias"] = np.zeros(E, dtype=np.float32)
    xv = np.zeros((2, H), dtype=np.float64)
    xv[:, 0] = 1.0
    xv[:, 1] = 2.0 ** -30   # expert 2's logit is 1 + 2^-30: above 1 in float64, equal in float32
    x_bits = synth.to_bf16_bits(xv)
    y_ref, idx_ref, a_ref, _ = O.moe_layer_factored(x_bits, L, w.top_k, w.d)
    assert list(idx_ref[0][:3]) == [2, 0, 1]
    y, idx, wt = _run_layer(C, w, L, x_bits)
    assert np.array_equal(idx, idx_ref), (idx, idx_ref)
    assert np.abs(wt - a_ref).max() <= 1e-5
    assert np.abs(y - y_ref).max() <= TOL * np.abs(y_ref).max()


def test_ties_beyond_256_experts(C):
    """300 experts (the exact one-wave radix top-k): a group of exact ties
    across the lanes and key rounds, a near tie below single precision, and
    a tie group straddling the k-th place — indices must match the oracle."""
    H, I, E, k, d, K, r, B = 256, 64, 300, 8, 8, 64, 8, 2
    L = synth.make_layer(H, I, E, d, K, r, seed=31)
    wr = np.zeros((H, E), dtype=np.float64)
    for e in (5, 77, 150, 260, 299):      # exact ties at the top
        wr[0, e] = 1.0
    wr[0, 123] = wr[1, 123] = 1.0           # 1 + 2^-30: above them only in float64
    for e in (3, 64, 128, 192, 256, 298):  # six-way tie around the k-th place
        wr[0, e] = 0.5
    L["router_w"] = synth.to_bf16_bits(wr)
    L["router_bias"] = np.zeros(E, dtype=np.float32)
    xv = np.zeros((B, H), dtype=np.float64)
    xv[:, 0] = 1.0
    xv[:, 1] = 2.0 ** -30
    x_bits = synth.to_bf16_bits(xv)
    y_ref, idx_ref, a_ref, _ = O.moe_layer_factored(x_bits, L, k, d)
    assert list(idx_ref[0]) == [123, 5, 77, 150, 260, 299, 3, 64]
    w = TINY.__class__("ties_e300", H=H, I=I, E=E, top_k=k, d=d, K=K, r=r, B=B, seed=0)
    y, idx, wt = _run_layer(C, w, L, x_bits)
    assert np.array_equal(idx, idx_ref), (idx, idx_ref)
    assert np.abs(wt - a_ref).max() <= 1e-5
    assert np.abs(y - y_ref).max() <= TOL * np.abs(y_ref).max()
