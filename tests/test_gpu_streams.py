"""The entry points on streams other than the default one and under HIP graph
capture: every launch goes to the caller's stream and nothing is allocated,
synchronised or cleared with a memset, so a captured layer call replays
bit-identically to the eager call (each replay checked, with eager work on
other buffers between the replays)."""

import sys

import numpy as np
import pytest
import torch

from paper_2609_21137_amd import synth

pytestmark = pytest.mark.gpu

H, I, E, K_TOP, D, K, R, B, SEED = 512, 384, 16, 4, 8, 64, 32, 8, 21


@pytest.fixture(scope="module")
def C():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_21137_amd import cardan
    return cardan


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def layer(C):
    L = synth.make_layer(H, I, E, D, K, R, SEED)
    W = synth.make_dense_weights(H, I, E, SEED)
    DL = C.DeviceLayer.from_numpy(L)
    DD = C.DenseLayer({"router_w": DL.tensors["router_w"], "router_bias": DL.tensors["router_bias"],
                       **{n: C.bf16_tensor(v) for n, v in W.items()}})
    return DL, DD


def _calls(C, shape, DL, DD):
    return {
        "compressed": lambda x, ws, o: C.moe_layer(shape, x, DL, ws=ws, out=o[0], idx=o[1], w=o[2]),
        "dense_down": lambda x, ws, o: C.moe_layer_dense_down(shape, x, DL, DD.tensors["W_down"], ws=ws,
                                                              out=o[0], idx=o[1], w=o[2]),
        "dense": lambda x, ws, o: C.dense_moe_layer(shape, x, DD, ws=ws, out=o[0], idx=o[1], w=o[2]),
    }


def _outs():
    return (torch.empty((B, H), dtype=torch.float32, device="cuda"),
            torch.empty((B, K_TOP), dtype=torch.int32, device="cuda"),
            torch.empty((B, K_TOP), dtype=torch.float32, device="cuda"))


@pytest.mark.parametrize("form", ["compressed", "dense_down", "dense"])
def test_side_stream_matches_default_stream(C, layer, form):
    _say(f"[streams] side stream, {form}")
    shape = C.make_shape(H, I, E, K_TOP, D, K, R)
    call = _calls(C, shape, *layer)[form]
    x = C.bf16_tensor(synth.make_input(H, B, SEED))
    ref = _outs()
    call(x, C.new_workspace(shape, B), ref)
    torch.cuda.synchronize()
    side = torch.cuda.Stream()
    ws = C.new_workspace(shape, B)
    got = _outs()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        call(x, ws, got)
    side.synchronize()
    for a, b in zip(ref, got):
        assert torch.equal(a, b)
    assert C.workspace_status(ws) == 0


@pytest.mark.parametrize("form", ["compressed", "dense_down", "dense"])
def test_graph_replays_match_eager(C, layer, form):
    _say(f"[streams] graph capture, {form}")
    shape = C.make_shape(H, I, E, K_TOP, D, K, R)
    call = _calls(C, shape, *layer)[form]
    x = C.bf16_tensor(synth.make_input(H, B, SEED, step=1))
    ref = _outs()
    call(x, C.new_workspace(shape, B), ref)
    torch.cuda.synchronize()

    ws = C.new_workspace(shape, B)
    out = _outs()
    g = torch.cuda.CUDAGraph()
    cap = torch.cuda.Stream()
    cap.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(cap):
        with torch.cuda.graph(g, stream=cap):
            call(x, ws, out)
    torch.cuda.current_stream().wait_stream(cap)
    torch.cuda.synchronize()

    other_ws = C.new_workspace(shape, B)
    for rep in range(4):
        for t in out:
            t.zero_()
        g.replay()
        torch.cuda.synchronize()
        for a, b in zip(ref, out):
            assert torch.equal(a, b), (form, rep)
        assert C.workspace_status(ws) == 0
        # eager work of the same kind on other buffers between the replays
        xo = C.bf16_tensor(synth.make_input(H, B, SEED, step=10 + rep))
        call(xo, other_ws, _outs())
        torch.cuda.synchronize()
    assert np.isfinite(out[0].cpu().numpy()).all()
