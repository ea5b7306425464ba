"""Layers built by the offline fitter (product quantisation plus the whitened
shared-basis correction, Sec. 3.3 and Appendix A.1) go through the GPU layer
with parity against the oracle on the same fitted factors, gated and up-only,
at batch 1 and 16. Bars as for every layer: top-k identical (oracle margin
> 1e-9), affinities within 1e-5, max|y - y_ref| <= 2e-2 max|y_ref| and the
1e-4 headroom bar. The GPU output of the fitted layer is also closer to the
dense teacher than that of its VQ part alone.
"""

import sys

import numpy as np
import pytest
import torch

import oracle.cardan_oracle as O
from paper_2609_21137_amd import fit, synth
from test_fit import _teacher

pytestmark = pytest.mark.gpu

TOL = 2e-2
HEADROOM = 1e-4


@pytest.fixture(scope="module")
def C():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_21137_amd import cardan
    return cardan


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


H, I, E, K_TOP, D, KW, R = 256, 128, 16, 4, 8, 64, 16


@pytest.fixture(scope="module")
def fitted():
    T = _teacher(H, I, E, D, KW, R, 31)
    L = synth.make_layer(H, I, E, D, KW, 0, seed=31)
    X = synth.make_input(H, 1024, seed=31)
    out = {}
    for act in ("silu_glu", "relu2_up"):
        layer, rep = fit.fit_layer(T, L["router_w"], L["router_bias"], X, K_TOP, D, KW, R, act=act, seed=3)
        out[(act, R)] = layer
        # the VQ part alone: the same codes and code books without the low rank terms
        out[(act, 0)] = dict(layer, U_gate=None, U_up=None, V_gate=None, V_up=None, A_down=None, B_down=None)
        _say(f"[fit] {act}: NMSE gate/up {rep.nmse_vq:.3e} -> {rep.nmse_vq_lr:.3e}, "
             f"down {rep.nmse_down_vq:.3e} -> {rep.nmse_down_vq_lr:.3e}")
    Tb = {n: synth.to_bf16_bits(v) for n, v in T.items()}
    return out, Tb, L


@pytest.mark.parametrize("act", ["silu_glu", "relu2_up"])
@pytest.mark.parametrize("B", [1, 16])
def test_fitted_layer_gpu_parity(C, fitted, act, B):
    layers, Tb, L0 = fitted
    x_bits = synth.make_input(H, B, seed=31, step=5)
    shape = C.make_shape(H, I, E, K_TOP, D, KW, R)
    run = C.moe_layer if act == "silu_glu" else C.moe_layer_relu2
    errs = {}
    for r in (R, 0):
        layer = layers[(act, r)]
        sh = shape if r else C.make_shape(H, I, E, K_TOP, D, KW, 0)
        y_ref, idx_ref, a_ref, margin = O.moe_layer_factored(x_bits, layer, K_TOP, D, act=act)
        y, idx, wt = run(sh, C.bf16_tensor(x_bits), C.DeviceLayer.from_numpy(layer))
        torch.cuda.synchronize()
        y = y.cpu().numpy().astype(np.float64)
        assert np.all(margin > 1e-9)
        assert np.array_equal(idx.cpu().numpy(), idx_ref)
        assert np.abs(wt.cpu().numpy() - a_ref).max() <= 1e-5
        err = np.abs(y - y_ref).max() / np.abs(y_ref).max()
        _say(f"[fit] {act} B={B} r={r}: GPU vs oracle {err:.3e}")
        assert err <= TOL and err <= HEADROOM
        y_t, _, _, _ = O.moe_layer_dense(x_bits, L0["router_w"], L0["router_bias"],
                                         Tb["W_gate"] if act == "silu_glu" else None, Tb["W_up"], Tb["W_down"],
                                         K_TOP, act=act)
        errs[r] = np.sum((y - y_t) ** 2) / np.sum(y_t ** 2)
    _say(f"[fit] {act} B={B}: error against the teacher, VQ only {errs[0]:.3e}, VQ + low rank {errs[R]:.3e}")
    assert errs[R] < errs[0]
