"""Input generator: determinism, bf16 rounding and the stated distributions."""

import numpy as np

from paper_2609_21137_amd import synth
from paper_2609_21137_amd.configs import QWEN3_B1, TINY


def _f(bits):
    return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def test_bf16_round_to_nearest_even():
    f = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, 1.0 + 2 ** -8 + 2 ** -20, -2.5, 0.0],
                 dtype=np.float32)
    bits = synth.f32_to_bf16_bits(f)
    # halfway cases go to the even mantissa; just above halfway rounds up
    assert bits.tolist() == [0x3F80, 0x3F80, 0x3F82, 0x3F81, 0xC020, 0x0000]
    assert synth.f32_to_bf16_bits(np.array([np.nan], np.float32))[0] == 0x7FC0


def test_same_seed_same_bytes_and_layers_differ():
    a = synth.workload_layer(TINY, 0)
    b = synth.workload_layer(TINY, 0)
    c = synth.workload_layer(TINY, 1)
    for key, v in a.items():
        assert np.array_equal(v, b[key]), key
    assert not np.array_equal(a["codes_gate"], c["codes_gate"])
    assert np.array_equal(synth.workload_input(TINY, 0, 3), synth.workload_input(TINY, 0, 3))
    assert not np.array_equal(synth.workload_input(TINY, 0, 3), synth.workload_input(TINY, 0, 4))


def test_shapes_dtypes_and_distributions():
    w = QWEN3_B1
    L = synth.workload_layer(w, 0)
    H, I, E, d, K, r = w.H, w.I, w.E, w.d, w.K, w.r
    assert L["codes_gate"].shape == (E, H // d, I) and L["codes_gate"].dtype == np.uint8
    assert L["codes_down"].shape == (E, I // d, H)
    assert L["V_gate"].shape == (E, r, I) and L["A_down"].shape == (E, I, r)
    assert L["U_gate"].shape == (H, r) and L["B_down"].shape == (r, H)
    assert L["U_up"] is L["U_gate"]
    assert L["cb_gate"].shape == (K, d) and L["cb_gate"].dtype == np.uint16
    # codes uniform over 0..K-1
    cnt = np.bincount(L["codes_up"][:4].ravel(), minlength=K)
    assert cnt.min() > 0 and L["codes_up"].max() == K - 1
    # stated standard deviations (relative tolerance well above sampling noise)
    assert abs(_f(L["router_w"]).std() - H ** -0.5) < 0.02 * H ** -0.5
    assert abs(_f(L["U_gate"]).std() - H ** -0.5) < 0.02 * H ** -0.5
    assert abs(_f(L["V_gate"][:8]).std() - 0.01) < 0.0002
    assert abs(_f(L["A_down"][:8]).std() - 0.01) < 0.0002
    assert abs(_f(L["cb_down"]).std() - 0.02) < 0.002
    assert np.allclose(L["router_bias"], 1e-3 * np.arange(E), atol=1e-9)
    x = synth.workload_input(w, 0, 0, B=64)
    assert abs(_f(x).std() - 1.0) < 0.03


def test_hot_expert_bias():
    L = synth.make_layer(64, 16, 16, 8, 4, 2, seed=2, hot_experts=range(8), hot_bias=2.0)
    assert np.allclose(L["router_bias"][:8], 2.0 + 1e-3 * np.arange(8), atol=1e-6)
    assert np.allclose(L["router_bias"][8:], 1e-3 * np.arange(8, 16), atol=1e-6)
