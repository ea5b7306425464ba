"""The no-allocation entry point against the workspace entry point.

cardan_moe_layer_noalloc runs the same kernels as cardan_moe_layer on the
library's own scratch array; called through the C ABI on the same inputs its
outputs must equal the workspace entry point's bit for bit (both are
deterministic). Several calls in a row share the array: a large batch, then a
smaller one, then a different layer shape (whose counters sit elsewhere), then
the first shape again, each against a fresh workspace call; the first is also
checked against the float64 oracle.
"""

import ctypes
import sys

import numpy as np
import pytest
import torch

import oracle.cardan_oracle as O
from paper_2609_21137_amd import synth
from paper_2609_21137_amd.configs import QWEN3_B16, TINY

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def C():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_21137_amd import cardan
    return cardan


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _noalloc(C, shape, x, DL):
    lib = C.lib()
    B = x.shape[0]
    y = torch.full((B, shape.H), float("nan"), dtype=torch.float32, device="cuda")
    idx = torch.full((B, shape.top_k), -7, dtype=torch.int32, device="cuda")
    w = torch.full((B, shape.top_k), float("nan"), dtype=torch.float32, device="cuda")
    st = DL.struct()
    rc = lib.cardan_moe_layer_noalloc(ctypes.byref(shape), B, ctypes.c_void_p(x.data_ptr()), ctypes.byref(st),
                                      ctypes.c_void_p(y.data_ptr()), ctypes.c_void_p(idx.data_ptr()),
                                      ctypes.c_void_p(w.data_ptr()),
                                      ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert rc == 0, lib.cardan_last_error().decode()
    return y, idx, w


def _with_ws(C, shape, x, DL):
    ws = C.new_workspace(shape, x.shape[0])
    y, idx, w = C.moe_layer(shape, x, DL, ws=ws)
    torch.cuda.synchronize()
    assert C.workspace_status(ws) == 0
    return y, idx, w


def test_noalloc_matches_workspace_entry_point(C):
    cases = [(QWEN3_B16, 16, 0), (QWEN3_B16, 3, 1), (TINY, 2, 2), (QWEN3_B16, 16, 3), (QWEN3_B16, 1, 4)]
    layers = {}
    for w, B, step in cases:
        _say(f"[noalloc] {w.name} B={B} step={step}")
        if w.name not in layers:
            L = synth.workload_layer(w)
            layers[w.name] = (L, C.DeviceLayer.from_numpy(L))
        L, DL = layers[w.name]
        shape = C.shape_of(w)
        x_bits = synth.make_input(w.H, B, w.seed, step=50 + step)
        x = C.bf16_tensor(x_bits)
        y0, i0, w0 = _noalloc(C, shape, x, DL)
        torch.cuda.synchronize()
        y1, i1, w1 = _with_ws(C, shape, x, DL)
        assert torch.equal(i0, i1)
        assert torch.equal(w0, w1)
        assert torch.equal(y0, y1), (y0 - y1).abs().max().item()
        if step == 0:
            y_ref, idx_ref, a_ref, margin = O.moe_layer_factored(x_bits, L, w.top_k, w.d)
            assert np.all(margin > 1e-9)
            assert np.array_equal(i0.cpu().numpy(), idx_ref)
            err = np.abs(y0.cpu().numpy() - y_ref).max() / np.abs(y_ref).max()
            assert err <= 2e-2, err
            _say(f"[noalloc] oracle normalised max error {err:.3e}")


def test_noalloc_rejects_oversized_layer(C):
    """A layer whose workspace exceeds the scratch array is refused before
    anything is enqueued."""
    shape = C.make_shape(4096, 1536, 64, 6, 8, 256, 256)
    need = C.workspace_bytes(shape, 64)
    assert need > (16 << 20)
    lib = C.lib()
    dummy = torch.zeros(16, dtype=torch.uint8, device="cuda")
    p = ctypes.c_void_p(dummy.data_ptr())
    st = C.LayerStruct(*([dummy.data_ptr()] * len(C.LAYER_FIELDS)))
    rc = lib.cardan_moe_layer_noalloc(ctypes.byref(shape), 64, p, ctypes.byref(st), p, p, p,
                                      ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert rc == -4, (rc, lib.cardan_last_error().decode())
