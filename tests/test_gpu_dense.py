"""GPU parity of the dense-weight layers against the float64 oracle.

Two layers share the compressed layer's harness (routing, grouping, tiles,
combine) with dense bf16 expert matrices: the uncompressed MoE layer (the
baseline of Sec. 2.1) and the layer that keeps gate/up compressed (Eq. (1))
with a dense bf16 down projection (Sec. 3.1). Bars as for the compressed
layer: top-k identical as ordered lists (oracle margin > 1e-9), affinities
within 1e-5, max|y - y_ref| <= 2e-2 max|y_ref|, and a 1e-4 headroom bar.

Only the selected experts' matrices are drawn; every other expert is filled
with bf16 NaN, so a read of an expert the routing did not select poisons y.
"""

import sys

import numpy as np
import pytest
import torch

import oracle.cardan_oracle as O
from paper_2609_21137_amd import synth
from paper_2609_21137_amd.configs import QWEN3_B1, QWEN3_B16

pytestmark = pytest.mark.gpu

TOL = 2e-2
HEADROOM = 1e-4
NAN_BF16 = 0x7FC0


@pytest.fixture(scope="module")
def C():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_21137_amd import cardan
    return cardan


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _check(y, idx, wt, y_ref, idx_ref, a_ref, margin):
    assert np.all(margin > 1e-9), margin.min()
    assert np.array_equal(idx, idx_ref), (idx, idx_ref)
    assert np.abs(wt - a_ref).max() <= 1e-5
    assert np.all(np.isfinite(y)), "a non-selected expert was read"
    err = np.abs(y - y_ref).max() / np.abs(y_ref).max()
    assert err <= TOL, err
    assert err <= HEADROOM, err
    return err


# (name, H, I, E, k, d, K, r, B, seed); Qwen3 shapes use the workload's layer
SMALL = [
    ("ragged_cols", 320, 288, 10, 3, 8, 64, 16, 5, 3),   # ragged column groups on I and H
    ("passes_b37", 192, 96, 6, 4, 8, 32, 8, 37, 4),      # experts with > 16 tokens
    ("top1", 128, 64, 4, 1, 4, 16, 0, 2, 5),
    ("d4_r24", 256, 160, 12, 2, 4, 16, 24, 9, 6),
    ("max_batch_64", 256, 128, 16, 4, 8, 64, 8, 64, 7),   # 256 selections
    ("one_expert_i32", 128, 32, 1, 1, 8, 16, 0, 3, 10),   # E = 1, the smallest I
    ("d2_r16", 256, 160, 12, 2, 2, 16, 16, 5, 11),        # d = 2 gate/up codes
]


def _layer_and_input(case):
    if case in ("qwen3_b1", "qwen3_b16"):
        w = QWEN3_B1 if case == "qwen3_b1" else QWEN3_B16
        return (w.H, w.I, w.E, w.top_k, w.d, w.K, w.r, w.B, w.seed,
                synth.workload_layer(w), synth.workload_input(w))
    name, H, I, E, k, d, K, r, B, seed = next(c for c in SMALL if c[0] == case)
    return (H, I, E, k, d, K, r, B, seed, synth.make_layer(H, I, E, d, K, r, seed),
            synth.make_input(H, B, seed))


CASES = [c[0] for c in SMALL] + ["qwen3_b1", "qwen3_b16"]


@pytest.mark.parametrize("case", CASES)
def test_dense_layer_parity(C, case):
    H, I, E, k, d, K, r, B, seed, L, x_bits = _layer_and_input(case)
    _say(f"[dense] {case} H={H} I={I} E={E} k={k} B={B}")
    idx_ref, _, _, _ = O.route(x_bits, L["router_w"], L["router_bias"], k)
    W = synth.make_dense_weights(H, I, E, seed, experts=np.unique(idx_ref), fill_bits=NAN_BF16)
    y_ref, idx_ref, a_ref, margin = O.moe_layer_dense(x_bits, L["router_w"], L["router_bias"],
                                                      W["W_gate"], W["W_up"], W["W_down"], k)
    shape = C.make_shape(H, I, E, k, d, K, r)
    DL = C.DenseLayer({"router_w": C.bf16_tensor(L["router_w"]),
                       "router_bias": torch.from_numpy(L["router_bias"]).cuda(),
                       **{n: C.bf16_tensor(v) for n, v in W.items()}})
    ws = C.new_workspace(shape, B)
    y, idx, wt = C.dense_moe_layer(shape, C.bf16_tensor(x_bits), DL, ws=ws)
    torch.cuda.synchronize()
    assert C.workspace_status(ws) == 0, "an in-kernel wait timed out"
    err = _check(y.cpu().numpy().astype(np.float64), idx.cpu().numpy(), wt.cpu().numpy(), y_ref,
                 idx_ref, a_ref, margin)
    _say(f"[dense] {case} normalised max error {err:.3e}")


@pytest.mark.parametrize("case", CASES)
def test_dense_down_layer_parity(C, case):
    H, I, E, k, d, K, r, B, seed, L, x_bits = _layer_and_input(case)
    _say(f"[dense-down] {case} H={H} I={I} E={E} k={k} d={d} r={r} B={B}")
    idx_ref, _, _, _ = O.route(x_bits, L["router_w"], L["router_bias"], k)
    Wd = synth.make_dense_weights(H, I, E, seed, which=("down",), experts=np.unique(idx_ref),
                                  fill_bits=NAN_BF16)["W_down"]
    y_ref, idx_ref, a_ref, margin = O.moe_layer_dense_down(x_bits, L, Wd, k, d)
    shape = C.make_shape(H, I, E, k, d, K, r)
    # the compressed down fields are left out: the entry point must not read them
    Lg = dict(L, cb_down=None, codes_down=None, A_down=None, B_down=None)
    DL = C.DeviceLayer.from_numpy(Lg)
    ws = C.new_workspace(shape, B)
    y, idx, wt = C.moe_layer_dense_down(shape, C.bf16_tensor(x_bits), DL, C.bf16_tensor(Wd), ws=ws)
    torch.cuda.synchronize()
    assert C.workspace_status(ws) == 0, "an in-kernel wait timed out"
    err = _check(y.cpu().numpy().astype(np.float64), idx.cpu().numpy(), wt.cpu().numpy(), y_ref,
                 idx_ref, a_ref, margin)
    _say(f"[dense-down] {case} normalised max error {err:.3e}")


def test_forms_share_one_workspace(C):
    """Compressed, dense-down and uncompressed calls of several batch sizes
    in turn on one workspace give bitwise the results of fresh workspaces."""
    H, I, E, k, d, K, r, seed = 320, 288, 10, 3, 8, 64, 16, 8
    L = synth.make_layer(H, I, E, d, K, r, seed)
    W = synth.make_dense_weights(H, I, E, seed)
    shape = C.make_shape(H, I, E, k, d, K, r)
    DL = C.DeviceLayer.from_numpy(L)
    DD = C.DenseLayer({"router_w": DL.tensors["router_w"], "router_bias": DL.tensors["router_bias"],
                       **{n: C.bf16_tensor(v) for n, v in W.items()}})
    Wd = DD.tensors["W_down"]
    calls = {
        "compressed": lambda x, ws: C.moe_layer(shape, x, DL, ws=ws),
        "dense_down": lambda x, ws: C.moe_layer_dense_down(shape, x, DL, Wd, ws=ws),
        "dense": lambda x, ws: C.dense_moe_layer(shape, x, DD, ws=ws),
    }
    shared = C.new_workspace(shape, 16)
    for i, (B, form) in enumerate([(16, "dense"), (1, "compressed"), (16, "dense_down"), (3, "dense"),
                                   (16, "compressed"), (1, "dense_down"), (16, "dense")]):
        _say(f"[dense] shared workspace call {i}: {form} B={B}")
        x = C.bf16_tensor(synth.make_input(H, B, seed, step=i))
        y1, i1, w1 = calls[form](x, shared)
        y2, i2, w2 = calls[form](x, C.new_workspace(shape, B))
        torch.cuda.synchronize()
        assert C.workspace_status(shared) == 0
        assert torch.equal(i1, i2) and torch.equal(w1, w2)
        assert torch.equal(y1, y2), form


def test_dense_without_router_bias(C):
    H, I, E, k, B, seed = 128, 96, 8, 2, 4, 9
    L = synth.make_layer(H, I, E, 8, 16, 0, seed)
    W = synth.make_dense_weights(H, I, E, seed)
    x_bits = synth.make_input(H, B, seed)
    y_ref, idx_ref, a_ref, margin = O.moe_layer_dense(x_bits, L["router_w"], None, W["W_gate"],
                                                      W["W_up"], W["W_down"], k)
    shape = C.make_shape(H, I, E, k, 8, 16, 0)
    DL = C.DenseLayer({"router_w": C.bf16_tensor(L["router_w"]),
                       **{n: C.bf16_tensor(v) for n, v in W.items()}})
    y, idx, wt = C.dense_moe_layer(shape, C.bf16_tensor(x_bits), DL)
    torch.cuda.synchronize()
    _check(y.cpu().numpy().astype(np.float64), idx.cpu().numpy(), wt.cpu().numpy(), y_ref, idx_ref,
           a_ref, margin)
