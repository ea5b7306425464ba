"""GPU parity of the projection-code-book gate/up path (Sec. 4.2): with
CARDAN_GATEUP=tbook the routing kernel builds T[t][pj][b][k] = x_b . cb_k per
token and projection, and a gate/up code tile of an expert with one token
sums T over its blocks instead of decoding code words on MFMA (experts with
more tokens keep the code-word tile within the same call).

Bars as for every layer: top-k identical (oracle margin > 1e-9), affinities
within 1e-5, max|y - y_ref| <= 2e-2 max|y_ref| and the 1e-4 headroom bar.
"""

import dataclasses
import os
import sys

import numpy as np
import pytest
import torch

import oracle.cardan_oracle as O
from paper_2609_21137_amd import synth
from paper_2609_21137_amd.configs import NEMOTRON3_B1, OLMOE_B1, QWEN3_B1, QWEN3_B16

pytestmark = pytest.mark.gpu

TOL = 2e-2
HEADROOM = 1e-4


@pytest.fixture(scope="module")
def C():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_21137_amd import cardan
    old = os.environ.get("CARDAN_GATEUP")
    os.environ["CARDAN_GATEUP"] = "tbook"
    yield cardan
    if old is None:
        del os.environ["CARDAN_GATEUP"]
    else:
        os.environ["CARDAN_GATEUP"] = old


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


# (name, H, I, E, k, d, K, r, B, seed, up_only)
SMALL = [
    ("ragged_cols", 320, 288, 10, 3, 8, 64, 16, 5, 3, False),
    ("passes_b37", 192, 96, 6, 4, 8, 32, 8, 37, 4, False),   # most experts take the code-word tile
    ("r0_top1", 128, 64, 4, 1, 4, 16, 0, 2, 5, False),
    ("d4_r24", 256, 160, 12, 2, 4, 16, 24, 9, 6, False),
    ("d2_r16", 256, 160, 12, 2, 2, 16, 16, 5, 11, False),   # d = 2: the planner keeps code words
    ("k4_book", 256, 128, 8, 2, 8, 4, 8, 3, 12, False),      # a 4-word code book
    ("up_only", 320, 288, 10, 3, 8, 64, 16, 5, 13, True),
]
FULL = {"qwen3_b1": QWEN3_B1, "qwen3_b16": QWEN3_B16, "olmoe_d4_b1": OLMOE_B1,
        "nemotron3_b1": NEMOTRON3_B1,
        "qwen3_b4": dataclasses.replace(QWEN3_B1, B=4, name="qwen3_b4")}


def _case(case):
    if case in FULL:
        w = FULL[case]
        return (w.H, w.I, w.E, w.top_k, w.d, w.K, w.r, w.B, w.act,
                synth.workload_layer(w), synth.workload_input(w))
    name, H, I, E, k, d, K, r, B, seed, up = next(c for c in SMALL if c[0] == case)
    return (H, I, E, k, d, K, r, B, "relu2_up" if up else "silu_glu",
            synth.make_layer(H, I, E, d, K, r, seed, up_only=up), synth.make_input(H, B, seed))


@pytest.mark.parametrize("case", [c[0] for c in SMALL] + list(FULL))
def test_tbook_layer_parity(C, case):
    H, I, E, k, d, K, r, B, act, L, x_bits = _case(case)
    _say(f"[tbook] {case} H={H} I={I} E={E} k={k} d={d} K={K} r={r} B={B} {act}")
    y_ref, idx_ref, a_ref, margin = O.moe_layer_factored(x_bits, L, k, d, act=act)
    shape = C.make_shape(H, I, E, k, d, K, r)
    ws = C.new_workspace(shape, B)
    run = C.moe_layer_relu2 if act == "relu2_up" else C.moe_layer
    y, idx, wt = run(shape, C.bf16_tensor(x_bits), C.DeviceLayer.from_numpy(L), ws=ws)
    torch.cuda.synchronize()
    assert C.workspace_status(ws) == 0, "an in-kernel wait timed out"
    y = y.cpu().numpy().astype(np.float64)
    assert np.all(margin > 1e-9), margin.min()
    assert np.array_equal(idx.cpu().numpy(), idx_ref)
    assert np.abs(wt.cpu().numpy() - a_ref).max() <= 1e-5
    err = np.abs(y - y_ref).max() / np.abs(y_ref).max()
    _say(f"[tbook] {case} normalised max error {err:.3e}")
    assert err <= TOL and err <= HEADROOM, err


def test_tbook_and_codeword_share_a_workspace(C):
    """Calls alternating between the two gate/up forms on one workspace (its
    size covers both) match fresh-workspace calls bit for bit."""
    w = QWEN3_B1
    shape = C.shape_of(w)
    DL = C.DeviceLayer.from_numpy(synth.workload_layer(w))
    shared = C.new_workspace(shape, 16)
    for i, (B, form) in enumerate([(1, "tbook"), (16, "codeword"), (4, "tbook"), (1, "codeword"),
                                   (16, "tbook"), (1, "tbook")]):
        os.environ["CARDAN_GATEUP"] = form
        x = C.bf16_tensor(synth.make_input(w.H, B, w.seed, step=40 + i))
        y1, i1, w1 = C.moe_layer(shape, x, DL, ws=shared)
        y2, i2, w2 = C.moe_layer(shape, x, DL, ws=C.new_workspace(shape, B))
        torch.cuda.synchronize()
        assert C.workspace_status(shared) == 0
        assert torch.equal(i1, i2) and torch.equal(w1, w2) and torch.equal(y1, y2), (i, form)
    os.environ["CARDAN_GATEUP"] = "tbook"
