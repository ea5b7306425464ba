"""Pins of the CPU oracle against facts fixed outside the oracle itself.

Each ``pin_*`` function raises ``AssertionError`` when the oracle disagrees
with the paper, a closed form, a textbook special case or a brute-force
evaluation. ``test_planted_mistakes_are_caught`` plants plausible mistakes in
the oracle (on the CPU) and checks that every one of them trips a pin.
"""

import json
import math
import os

import numpy as np
import pytest
import torch

import oracle.cardan_oracle as O
from paper_2609_21137_amd import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _load(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def _bf(a):
    return synth.to_bf16_bits(np.asarray(a, dtype=np.float64))


# --------------------------------------------------------------------------
# independent dense MoE (torch float64) for the special cases
# --------------------------------------------------------------------------
def dense_moe_torch(x, Wr, bias, Wg, Wu, Wd, k):
    """Plain dense MoE: router, top-k, softmax over the top-k, SiLU-gated
    FFN per expert and the affinity-weighted sum. ``Wg/Wu [E, H, I]``,
    ``Wd [E, I, H]`` are float64 arrays."""
    x = torch.as_tensor(x, dtype=torch.float64)
    logits = x @ torch.as_tensor(Wr, dtype=torch.float64) + torch.as_tensor(bias, dtype=torch.float64)
    vals, idx = torch.topk(logits, k, dim=1)
    a = torch.softmax(vals, dim=1)
    Wg = torch.as_tensor(Wg, dtype=torch.float64)
    Wu = torch.as_tensor(Wu, dtype=torch.float64)
    Wd = torch.as_tensor(Wd, dtype=torch.float64)
    y = torch.zeros_like(x)
    for t in range(x.shape[0]):
        for j in range(k):
            e = int(idx[t, j])
            h = x[t]
            p = torch.nn.functional.silu(h @ Wg[e]) * (h @ Wu[e])
            y[t] += a[t, j] * (p @ Wd[e])
    return y.numpy(), idx.numpy(), a.numpy()


def _rand_layer(H, I, E, d, K, r, seed, **kw):
    return synth.make_layer(H, I, E, d, K, r, seed, **kw)


def _scale_codebooks(L, s):
    """Larger code words so that tiny layers have O(1) outputs."""
    for key in ("cb_gate", "cb_up", "cb_down"):
        L[key] = _bf(O.bf16_to_f64(L[key]) * s)
    return L


# --------------------------------------------------------------------------
# pins
# --------------------------------------------------------------------------
def _worked_layer():
    g = _load("worked_example.json")
    L = {
        "router_w": _bf(g["router_w"]),
        "router_bias": np.asarray(g["router_bias"], dtype=np.float32),
        "cb_gate": _bf(g["cb_gate"]), "cb_up": _bf(g["cb_up"]), "cb_down": _bf(g["cb_down"]),
        "codes_gate": np.asarray(g["codes_gate"], dtype=np.uint8),
        "codes_up": np.asarray(g["codes_up"], dtype=np.uint8),
        "codes_down": np.asarray(g["codes_down"], dtype=np.uint8),
        "U_gate": _bf(g["U"]), "U_up": _bf(g["U"]),
        "V_gate": _bf(g["V_gate"]), "V_up": _bf(g["V_up"]),
        "A_down": _bf(g["A_down"]), "B_down": _bf(g["B_down"]),
    }
    return g, L, _bf(g["x"])


def _worked_expected(g):
    ex = g["expected"]
    p = [gg / (1.0 + math.exp(-gg)) * uu for gg, uu in zip(ex["g"], ex["u"])]
    return np.array([[sum(m * pp for m, pp in zip(row, p)) for row in ex["y_from_p"]]])


def pin_worked_example():
    g, L, x = _worked_layer()
    y_exp = _worked_expected(g)
    k, d = g["shape"]["top_k"], g["shape"]["d"]
    for fn in (O.moe_layer, O.moe_layer_factored, O.moe_layer_scalar):
        y, idx, a, _ = fn(x, L, k, d)
        assert np.array_equal(idx, np.array(g["expected"]["topk_idx"])), fn.__name__
        assert np.allclose(a, g["expected"]["topk_w"], rtol=0, atol=1e-15), fn.__name__
        assert np.allclose(y, y_exp, rtol=1e-13, atol=1e-13), (fn.__name__, y, y_exp)
    logits = O.router_logits(x, L["router_w"], L["router_bias"])
    assert np.allclose(logits, g["expected"]["logits"], rtol=0, atol=1e-7)


TINY_SHAPES = [
    # H, I, E, k, d, K, r, B
    (8, 4, 3, 2, 2, 4, 1, 2),
    (8, 8, 4, 2, 4, 3, 2, 1),
    (12, 4, 5, 3, 1, 5, 0, 2),
    (16, 8, 4, 1, 8, 2, 3, 2),
    (16, 4, 6, 3, 4, 8, 0, 1),
    (6, 6, 3, 3, 3, 2, 2, 2),
]


def pin_o1_equals_scalar_bruteforce():
    for n, (H, I, E, k, d, K, r, B) in enumerate(TINY_SHAPES):
        L = _scale_codebooks(_rand_layer(H, I, E, d, K, r, seed=100 + n), 25.0)
        x = synth.make_input(H, B, seed=100 + n)
        y1, i1, a1, m1 = O.moe_layer(x, L, k, d)
        y2, i2, a2, m2 = O.moe_layer_scalar(x, L, k, d)
        assert np.array_equal(i1, i2), (n, i1, i2)
        assert np.allclose(a1, a2, rtol=0, atol=1e-14)
        assert np.allclose(m1, m2, rtol=1e-9, atol=1e-15)
        scale = max(np.abs(y2).max(), 1e-30)
        assert np.abs(y1 - y2).max() <= 1e-12 * scale, (n, np.abs(y1 - y2).max(), scale)


def pin_o1_equals_factored():
    shapes = TINY_SHAPES + [(256, 128, 8, 2, 4, 16, 8, 3)]
    for n, (H, I, E, k, d, K, r, B) in enumerate(shapes):
        L = _scale_codebooks(_rand_layer(H, I, E, d, K, r, seed=200 + n), 4.0)
        x = synth.make_input(H, B, seed=200 + n)
        y1, i1, _, _ = O.moe_layer(x, L, k, d)
        y3, i3, _, _ = O.moe_layer_factored(x, L, k, d)
        assert np.array_equal(i1, i3)
        scale = np.abs(y1).max()
        assert np.abs(y1 - y3).max() <= 1e-12 * scale


def pin_onehot_codebook_is_dense_moe():
    """r = 0 and code book = identity (K = d): W[i, j] = [i % d == J[i // d, j]]."""
    rng = np.random.default_rng(7)
    H, I, E, k, d, B = 16, 8, 5, 2, 4, 3
    L = _rand_layer(H, I, E, d, d, 0, seed=7)
    eye = _bf(np.eye(d))
    L["cb_gate"] = L["cb_up"] = L["cb_down"] = eye
    x = synth.make_input(H, B, seed=7)

    def onehot(J, n_in):
        rows = np.arange(n_in)
        return (rows[:, None] % d == J[rows // d, :]).astype(np.float64)

    Wg = np.stack([onehot(L["codes_gate"][e], H) for e in range(E)])
    Wu = np.stack([onehot(L["codes_up"][e], H) for e in range(E)])
    Wd = np.stack([onehot(L["codes_down"][e], I) for e in range(E)])
    # small inputs keep silu in its curved range
    xs = _bf(O.bf16_to_f64(x) * 0.25)
    y_ref, idx_ref, a_ref = dense_moe_torch(O.bf16_to_f64(xs), O.bf16_to_f64(L["router_w"]),
                                            L["router_bias"].astype(np.float64), Wg, Wu, Wd, k)
    y, idx, a, _ = O.moe_layer(xs, L, k, d)
    assert np.array_equal(idx, idx_ref)
    assert np.allclose(a, a_ref, rtol=0, atol=1e-14)
    assert np.allclose(y, y_ref, rtol=1e-12, atol=1e-12)
    del rng


def pin_value_table_d1_is_dense_moe():
    """r = 0, d = 1: every weight is a table value, W[i, j] = cb[J[i, j], 0]."""
    H, I, E, k, K, B = 12, 6, 4, 2, 7, 2
    L = _rand_layer(H, I, E, 1, K, 0, seed=8)
    L = _scale_codebooks(L, 10.0)
    x = synth.make_input(H, B, seed=8)

    def table(cb, J):
        return np.take(O.bf16_to_f64(cb)[:, 0], J.astype(np.int64))

    Wg = np.stack([table(L["cb_gate"], L["codes_gate"][e]) for e in range(E)])
    Wu = np.stack([table(L["cb_up"], L["codes_up"][e]) for e in range(E)])
    Wd = np.stack([table(L["cb_down"], L["codes_down"][e]) for e in range(E)])
    y_ref, idx_ref, _ = dense_moe_torch(O.bf16_to_f64(x), O.bf16_to_f64(L["router_w"]),
                                        L["router_bias"].astype(np.float64), Wg, Wu, Wd, k)
    y, idx, _, _ = O.moe_layer(x, L, k, 1)
    assert np.array_equal(idx, idx_ref)
    assert np.allclose(y, y_ref, rtol=1e-12, atol=1e-14)


def pin_zero_codebooks_is_lowrank_moe():
    """Zero code books leave W_e = U V_e (gate/up) and A_e B (down)."""
    H, I, E, k, d, K, r, B = 16, 8, 4, 2, 4, 4, 3, 2
    L = _rand_layer(H, I, E, d, K, r, seed=9, separate_up_basis=True)
    zero = np.zeros_like(L["cb_gate"])
    L["cb_gate"] = L["cb_up"] = L["cb_down"] = zero
    for key in ("V_gate", "V_up", "A_down"):
        L[key] = _bf(O.bf16_to_f64(L[key]) * 300.0)
    x = synth.make_input(H, B, seed=9)
    f = O.bf16_to_f64
    Wg = np.stack([f(L["U_gate"]) @ f(L["V_gate"][e]) for e in range(E)])
    Wu = np.stack([f(L["U_up"]) @ f(L["V_up"][e]) for e in range(E)])
    Wd = np.stack([f(L["A_down"][e]) @ f(L["B_down"]) for e in range(E)])
    y_ref, idx_ref, _ = dense_moe_torch(f(x), f(L["router_w"]), L["router_bias"].astype(np.float64),
                                        Wg, Wu, Wd, k)
    y, idx, _, _ = O.moe_layer(x, L, k, d)
    assert np.array_equal(idx, idx_ref)
    assert np.abs(y).max() > 1e-3
    assert np.allclose(y, y_ref, rtol=1e-11, atol=1e-14)


def pin_expert_permutation_invariance():
    H, I, E, k, d, K, r, B = 16, 8, 6, 2, 4, 8, 2, 3
    L = _scale_codebooks(_rand_layer(H, I, E, d, K, r, seed=10), 20.0)
    x = synth.make_input(H, B, seed=10)
    perm = np.array([3, 0, 5, 1, 4, 2])           # new expert n holds old expert perm[n]
    inv = np.argsort(perm)
    P = dict(L)
    P["router_w"] = L["router_w"][:, perm]
    P["router_bias"] = L["router_bias"][perm]
    for key in ("codes_gate", "codes_up", "codes_down", "V_gate", "V_up", "A_down"):
        P[key] = L[key][perm]
    y0, i0, a0, _ = O.moe_layer(x, L, k, d)
    y1, i1, a1, _ = O.moe_layer(x, P, k, d)
    assert np.array_equal(perm[i1], i0) or np.array_equal(i1, inv[i0])
    assert np.allclose(a0, a1, rtol=0, atol=1e-15)
    assert np.allclose(y0, y1, rtol=1e-13, atol=1e-15)


def pin_batch_rows_independent():
    H, I, E, k, d, K, r = 32, 16, 6, 3, 4, 8, 2
    L = _scale_codebooks(_rand_layer(H, I, E, d, K, r, seed=11), 10.0)
    x = synth.make_input(H, 4, seed=11)
    y, idx, a, _ = O.moe_layer(x, L, k, d)
    for t in range(4):
        yt, it, at, _ = O.moe_layer(x[t:t + 1], L, k, d)
        assert np.array_equal(yt[0], y[t]) and np.array_equal(it[0], idx[t])
    # identical tokens route identically and give identical outputs
    xd = np.repeat(x[:1], 5, axis=0)
    yd, idd, _, _ = O.moe_layer(xd, L, k, d)
    assert (idd == idd[0]).all() and np.allclose(yd, yd[0], rtol=0, atol=0)


def pin_topk_rules():
    # exact tie between experts 0 and 3 at the top -> lower index first
    logits = np.array([[2.0, 1.0, -1.0, 2.0, 0.5]])
    idx, margin = O.select_topk(logits, 3)
    assert idx.tolist() == [[0, 3, 1]]
    assert margin[0] == 0.5
    # tie at the selection boundary -> lower index is selected
    idx, margin = O.select_topk(np.array([[0.0, 5.0, 1.0, 1.0]]), 2)
    assert idx.tolist() == [[1, 2]] and margin[0] == 0.0
    # k = 1 -> affinity 1; k = E -> margin inf
    assert O.gating(logits, np.array([[3]]))[0, 0] == 1.0
    _, m = O.select_topk(logits, 5)
    assert math.isinf(m[0])
    # two-way softmax closed form a0 = 1 / (1 + exp(l1 - l0))
    a = O.gating(np.array([[0.3, -1.7, 9.0]]), np.array([[0, 1]]))
    assert abs(a[0, 0] - 1.0 / (1.0 + math.exp(-2.0))) < 1e-15
    assert abs(a.sum() - 1.0) < 1e-15
    # router tie through the full router: equal logits, expert 0 wins
    x = _bf([[1.0, 0.0, 0.0, 1.0]])
    Wr = _bf([[1.0, 0.0], [0.0, 0.0], [0.0, 0.0], [0.0, 1.0]])
    idx, a, _, _ = O.route(x, Wr, np.zeros(2, np.float32), 1)
    assert idx.tolist() == [[0]] and a[0, 0] == 1.0


def pin_decode_layout():
    """Block b of column j is code word J[b, j], element i at input row b*d+i."""
    cb = _bf([[1, 2, 3], [4, 5, 6]])
    J = np.array([[1, 0], [0, 0]], dtype=np.uint8)
    Q = O.decode_vq(J, cb, 3)
    assert Q.tolist() == [[4, 1], [5, 2], [6, 3], [1, 1], [2, 2], [3, 3]]


def pin_silu_and_rmsnorm():
    assert O.silu(np.array([0.0]))[0] == 0.0
    assert abs(O.silu(np.array([1.0]))[0] - 1.0 / (1.0 + math.exp(-1.0))) < 1e-16
    assert abs(O.silu(np.array([-2.0]))[0] + 2.0 / (1.0 + math.exp(2.0))) < 1e-16
    r = O.rmsnorm(np.array([[3.0, 4.0]]), eps=0.0)
    assert np.allclose(r, [[3.0 / math.sqrt(12.5), 4.0 / math.sqrt(12.5)]], rtol=0, atol=1e-15)
    # eps as large as mean(y^2) = 12.5: the root of 12.5 + 12.5 is 5, so the row
    # becomes the unit vector [0.6, 0.8]; eps outside the root would give
    # [3, 4] / (sqrt(12.5) + 12.5) instead
    r = O.rmsnorm(np.array([[3.0, 4.0], [-6.0, 8.0]]), eps=12.5)
    assert np.allclose(r[0], [0.6, 0.8], rtol=0, atol=1e-15)
    # second row: mean 50, root of 62.5
    assert np.allclose(r[1], np.array([-6.0, 8.0]) / math.sqrt(62.5), rtol=0, atol=1e-15)


def pin_bf16_widening():
    bits = np.array([0x3F80, 0xBF80, 0x0000, 0x8000, 0x3F81, 0x7F7F, 0x0001], dtype=np.uint16)
    v = O.bf16_to_f64(bits)
    assert v[0] == 1.0 and v[1] == -1.0 and v[2] == 0.0
    assert v[4] == 1.0 + 2.0 ** -7
    assert v[5] == (2.0 - 2.0 ** -7) * 2.0 ** 127
    assert v[6] == 2.0 ** -133


def pin_storage_rate_tables():
    t = _load("paper_tables.json")
    models = t["table2_models"]
    for name, comp in t["table5_compression"].items():
        if name.startswith("_"):
            continue
        m = models[name]
        bits = O.storage_bits_per_weight(m["d"], m["K"], m["r"], m["H"], m["I"], m["E"])
        assert round(16.0 / bits, 2) == comp, (name, 16.0 / bits, comp)
    q = models["qwen3_30b_a3b"]
    for name, row in t["table6_bits_per_weight"].items():
        if name.startswith("_"):
            continue
        if row["d"] is None:      # low-rank only: no index map, no code book
            bits = O.storage_bits_per_weight(1, 1, row["r"], q["H"], q["I"], q["E"],
                                             b_index=0, b_codebook=0)
        else:
            bits = O.storage_bits_per_weight(row["d"], 256, row["r"], q["H"], q["I"], q["E"])
        assert round(bits, 2) == row["bits"], (name, bits)


def pin_dense_baseline_against_torch():
    """The dense-weight baseline layer against the independent torch float64
    dense MoE on random bf16 matrices."""
    H, I, E, k, B = 24, 16, 6, 2, 3
    L = _rand_layer(H, I, E, 8, 16, 0, seed=11)  # only the router is used
    W = {key: _bf(O.bf16_to_f64(v) * 10.0) for key, v in synth.make_dense_weights(H, I, E, seed=11).items()}
    x = synth.make_input(H, B, seed=11)
    y_ref, idx_ref, a_ref = dense_moe_torch(O.bf16_to_f64(x), O.bf16_to_f64(L["router_w"]),
                                            L["router_bias"].astype(np.float64), O.bf16_to_f64(W["W_gate"]),
                                            O.bf16_to_f64(W["W_up"]), O.bf16_to_f64(W["W_down"]), k)
    y, idx, a, _ = O.moe_layer_dense(x, L["router_w"], L["router_bias"], W["W_gate"], W["W_up"], W["W_down"], k)
    assert np.array_equal(idx, idx_ref)
    assert np.allclose(a, a_ref, rtol=0, atol=1e-14)
    assert np.allclose(y, y_ref, rtol=1e-12, atol=1e-12)


def pin_dense_down_reduces_to_compressed():
    """With r = 0 the decoded matrices are exact bf16 values: setting the
    dense down matrix to the decoded down codes gives O1 bit for bit, and
    setting dense gate/up matrices to the decoded gate/up codes as well gives
    the dense baseline bit for bit."""
    H, I, E, k, d, K, B = 16, 16, 5, 2, 4, 16, 3
    L = _scale_codebooks(_rand_layer(H, I, E, d, K, 0, seed=12), 10.0)
    x = synth.make_input(H, B, seed=12)
    dec = lambda key, cb: np.stack([_bf(O.decode_vq(L[key][e], L[cb], d)) for e in range(E)])
    Wg, Wu, Wd = dec("codes_gate", "cb_gate"), dec("codes_up", "cb_up"), dec("codes_down", "cb_down")
    y1, idx1, a1, _ = O.moe_layer(x, L, k, d)
    y2, idx2, a2, _ = O.moe_layer_dense_down(x, L, Wd, k, d)
    y3, idx3, a3, _ = O.moe_layer_dense(x, L["router_w"], L["router_bias"], Wg, Wu, Wd, k)
    assert np.array_equal(idx1, idx2) and np.array_equal(idx1, idx3)
    assert np.array_equal(a1, a2) and np.array_equal(a1, a3)
    assert np.array_equal(y1, y2) and np.array_equal(y2, y3)
    assert np.abs(y1).max() > 1e-3  # a non-trivial output


# --------------------------------------------------------------------------
# up-only experts with a squared-ReLU activation (Table 2, projection "up")
# --------------------------------------------------------------------------
def dense_relu2_moe_torch(x, Wr, bias, Wu, Wd, k):
    """Plain dense MoE with up-only experts: router, top-k, softmax over the
    top-k, ``relu(h W_up)^2 W_down`` per expert, affinity-weighted sum
    (torch float64)."""
    x = torch.as_tensor(x, dtype=torch.float64)
    logits = x @ torch.as_tensor(Wr, dtype=torch.float64) + torch.as_tensor(bias, dtype=torch.float64)
    vals, idx = torch.topk(logits, k, dim=1)
    a = torch.softmax(vals, dim=1)
    Wu = torch.as_tensor(Wu, dtype=torch.float64)
    Wd = torch.as_tensor(Wd, dtype=torch.float64)
    y = torch.zeros_like(x)
    for t in range(x.shape[0]):
        for j in range(k):
            e = int(idx[t, j])
            p = torch.square(torch.relu(x[t] @ Wu[e]))
            y[t] += a[t, j] * (p @ Wd[e])
    return y.numpy(), idx.numpy(), a.numpy()


def _up_only(L):
    """The layer without its gate tensors (what an up-only model stores)."""
    L = dict(L)
    for key in ("cb_gate", "codes_gate", "U_gate", "V_gate"):
        L[key] = None
    return L


def pin_relu2_closed_form():
    u = np.array([-2.0, -0.5, 0.0, 0.5, 3.0])
    assert O.relu2(u).tolist() == [0.0, 0.0, 0.0, 0.25, 9.0]
    assert O.activation("relu2_up", None, u).tolist() == [0.0, 0.0, 0.0, 0.25, 9.0]
    # the gated form multiplies by u, the up-only form never reads g
    g = np.array([1.0])
    assert abs(O.activation("silu_glu", g, np.array([2.0]))[0] - 2.0 / (1.0 + math.exp(-1.0))) < 1e-15


def pin_relu2_onehot_is_dense_moe():
    """r = 0 and code book = identity (K = d): the up-only layer equals a
    dense up-only MoE on the 0/1 matrices W[i, j] = [i % d == J[i // d, j]]
    (torch's relu and square); x ~ N(0, 1) gives u of both signs."""
    H, I, E, k, d, B = 16, 8, 5, 2, 4, 3
    L = _up_only(_rand_layer(H, I, E, d, d, 0, seed=17))
    eye = _bf(np.eye(d))
    L["cb_up"] = L["cb_down"] = eye
    x = synth.make_input(H, B, seed=17)

    def onehot(J, n_in):
        rows = np.arange(n_in)
        return (rows[:, None] % d == J[rows // d, :]).astype(np.float64)

    Wu = np.stack([onehot(L["codes_up"][e], H) for e in range(E)])
    Wd = np.stack([onehot(L["codes_down"][e], I) for e in range(E)])
    xf = O.bf16_to_f64(x)
    y_ref, idx_ref, a_ref = dense_relu2_moe_torch(xf, O.bf16_to_f64(L["router_w"]),
                                                  L["router_bias"].astype(np.float64), Wu, Wd, k)
    u_all = np.einsum("th,ehi->tei", xf, Wu)
    assert (u_all > 0).any() and (u_all < 0).any()
    for fn in (O.moe_layer, O.moe_layer_factored, O.moe_layer_scalar):
        y, idx, a, _ = fn(x, L, k, d, "relu2_up")
        assert np.array_equal(idx, idx_ref), fn.__name__
        assert np.allclose(a, a_ref, rtol=0, atol=1e-14), fn.__name__
        assert np.allclose(y, y_ref, rtol=1e-12, atol=1e-12), fn.__name__


def pin_relu2_o1_equals_scalar_and_factored():
    """Up-only layers with the low-rank terms: O1 (dense reconstruction), O2
    (scalar loops) and O3 (factored) agree on tiny shapes; a gated layer's
    gate tensors, where present, change nothing."""
    for n, (H, I, E, k, d, K, r, B) in enumerate(TINY_SHAPES):
        full = _scale_codebooks(_rand_layer(H, I, E, d, K, r, seed=300 + n), 25.0)
        L = _up_only(full)
        x = synth.make_input(H, B, seed=300 + n)
        y1, i1, a1, _ = O.moe_layer(x, L, k, d, "relu2_up")
        y2, i2, a2, _ = O.moe_layer_scalar(x, L, k, d, "relu2_up")
        y3, i3, a3, _ = O.moe_layer_factored(x, L, k, d, "relu2_up")
        y4, _, _, _ = O.moe_layer_factored(x, full, k, d, "relu2_up")
        assert np.array_equal(i1, i2) and np.array_equal(i1, i3)
        scale = max(np.abs(y2).max(), 1e-30)
        assert np.abs(y1 - y2).max() <= 1e-12 * scale, (n, np.abs(y1 - y2).max(), scale)
        assert np.abs(y1 - y3).max() <= 1e-12 * scale
        assert np.array_equal(y3, y4)
        assert scale > 1e-6  # a non-trivial output


def pin_relu2_dense_baseline_against_torch():
    H, I, E, k, B = 16, 12, 6, 3, 4
    W = synth.make_dense_weights(H, I, E, seed=19, which=("up", "down"))
    Wr = _bf(np.random.default_rng(19).standard_normal((H, E)) * 0.5)
    bias = np.linspace(0.0, 1e-2, E).astype(np.float32)
    x = synth.make_input(H, B, seed=19)
    Wu, Wd = (O.bf16_to_f64(W[n]) * 20.0 for n in ("W_up", "W_down"))
    Wu_b, Wd_b = _bf(Wu), _bf(Wd)
    y, idx, a, _ = O.moe_layer_dense(x, Wr, bias, None, Wu_b, Wd_b, k, "relu2_up")
    y_ref, idx_ref, a_ref = dense_relu2_moe_torch(O.bf16_to_f64(x), O.bf16_to_f64(Wr), bias.astype(np.float64),
                                                  O.bf16_to_f64(Wu_b), O.bf16_to_f64(Wd_b), k)
    assert np.array_equal(idx, idx_ref)
    assert np.allclose(a, a_ref, rtol=0, atol=1e-14)
    assert np.allclose(y, y_ref, rtol=1e-12, atol=1e-12)
    assert np.abs(y).max() > 1e-3


def pin_relu2_reduces_to_dense_relu2():
    """With r = 0 the decoded up-only layer equals the dense up-only baseline
    on the decoded matrices bit for bit."""
    H, I, E, k, d, K, B = 16, 16, 5, 2, 4, 16, 3
    L = _up_only(_scale_codebooks(_rand_layer(H, I, E, d, K, 0, seed=21), 10.0))
    x = synth.make_input(H, B, seed=21)
    dec = lambda key, cb: np.stack([_bf(O.decode_vq(L[key][e], L[cb], d)) for e in range(E)])
    Wu, Wd = dec("codes_up", "cb_up"), dec("codes_down", "cb_down")
    y1, idx1, a1, _ = O.moe_layer(x, L, k, d, "relu2_up")
    y2, idx2, a2, _ = O.moe_layer_dense(x, L["router_w"], L["router_bias"], None, Wu, Wd, k, "relu2_up")
    assert np.array_equal(idx1, idx2) and np.array_equal(a1, a2)
    assert np.array_equal(y1, y2)
    assert np.abs(y1).max() > 1e-3


PINS = [
    pin_worked_example, pin_o1_equals_scalar_bruteforce, pin_o1_equals_factored,
    pin_onehot_codebook_is_dense_moe, pin_value_table_d1_is_dense_moe,
    pin_zero_codebooks_is_lowrank_moe, pin_expert_permutation_invariance,
    pin_batch_rows_independent, pin_topk_rules, pin_decode_layout, pin_silu_and_rmsnorm,
    pin_bf16_widening, pin_storage_rate_tables, pin_dense_baseline_against_torch,
    pin_dense_down_reduces_to_compressed, pin_relu2_closed_form, pin_relu2_onehot_is_dense_moe,
    pin_relu2_o1_equals_scalar_and_factored, pin_relu2_dense_baseline_against_torch,
    pin_relu2_reduces_to_dense_relu2,
]


@pytest.mark.parametrize("pin", PINS, ids=[p.__name__ for p in PINS])
def test_pin(pin):
    pin()


# --------------------------------------------------------------------------
# planted mistakes: every one must trip at least one pin
# --------------------------------------------------------------------------
def _mut_decode_reversed(codes, codebook, d):
    Q = _ORIG["decode_vq"](codes, codebook, d)
    nb = Q.shape[0] // d
    return Q.reshape(nb, d, -1)[:, ::-1, :].reshape(Q.shape)


def _mut_decode_blocks_across_columns(codes, codebook, d):
    J = np.asarray(codes).astype(np.int64)
    cb = O.bf16_to_f64(codebook)
    blocks = cb[J]                                  # [nb, n_out, d]
    return blocks.reshape(J.shape[0] * d, J.shape[1])   # element order scrambled


def _mut_drop_gate_lr(layer, e, d, act="silu_glu"):
    Wg, Wu, Wd = _ORIG["expert_matrices"](layer, e, d, act)
    if layer.get("U_gate") is not None and O.bf16_to_f64(layer["U_gate"]).shape[1] > 0:
        Wg = Wg - O.bf16_to_f64(layer["U_gate"]) @ O.bf16_to_f64(layer["V_gate"][e])
    return Wg, Wu, Wd


def _mut_drop_down_lr(layer, e, d, act="silu_glu"):
    Wg, Wu, Wd = _ORIG["expert_matrices"](layer, e, d, act)
    if layer.get("U_up") is not None and O.bf16_to_f64(layer["U_up"]).shape[1] > 0:
        Wd = Wd - O.bf16_to_f64(layer["A_down"][e]) @ O.bf16_to_f64(layer["B_down"])
    return Wg, Wu, Wd


def _mut_swap_gate_up(layer, e, d, act="silu_glu"):
    Wg, Wu, Wd = _ORIG["expert_matrices"](layer, e, d, act)
    return (Wu, Wg, Wd) if Wg is not None else (Wg, Wu, Wd)


def _mut_silu_sign(g):
    g = np.asarray(g, dtype=np.float64)
    return g / (1.0 + np.exp(g))


def _mut_softmax_all(logits, idx):
    logits = np.asarray(logits, dtype=np.float64)
    w = np.exp(logits - logits.max(axis=1, keepdims=True))
    w = w / w.sum(axis=1, keepdims=True)
    return np.take_along_axis(w, np.asarray(idx), axis=1)


def _mut_tie_high(logits, k):
    logits = np.asarray(logits, dtype=np.float64)
    B, E = logits.shape
    idx = np.zeros((B, k), dtype=np.int64)
    margin = np.full(B, np.inf)
    for t in range(B):
        order = sorted(range(E), key=lambda e: (-logits[t, e], -e))
        idx[t] = order[:k]
        if k < E:
            margin[t] = logits[t, order[k - 1]] - logits[t, order[k]]
    return idx, margin


def _mut_no_bias(x, router_w, router_bias=None):
    return _ORIG["router_logits"](x, router_w, None)


def _mut_unweighted(x, idx, a, layer, d, act="silu_glu"):
    return _ORIG["expert_ffn"](x, idx, np.ones_like(np.asarray(a, dtype=np.float64)), layer, d, act)


def _mut_storage_no_basis(d, K, r, H, I, E, b_index=None, b_coef=16, b_codebook=16, b_basis=16):
    return _ORIG["storage_bits_per_weight"](d, K, r, H, I, E, b_index, b_coef, b_codebook, 0)


def _mut_dense_no_silu(x, idx, a, W_gate, W_up, W_down, act="silu_glu"):
    if act != "silu_glu":
        return _ORIG["expert_ffn_dense"](x, idx, a, W_gate, W_up, W_down, act)
    xf = O.bf16_to_f64(x)
    y = np.zeros_like(xf)
    for t in range(xf.shape[0]):
        for j in range(np.asarray(idx).shape[1]):
            e = int(idx[t, j])
            p = (O.bf16_to_f64(W_gate[e]).T @ xf[t]) * (O.bf16_to_f64(W_up[e]).T @ xf[t])
            y[t] += a[t, j] * (O.bf16_to_f64(W_down[e]).T @ p)
    return y


def _mut_rmsnorm_eps_outside(y, eps=1e-6):
    y = np.asarray(y, dtype=np.float64)
    return y / (np.sqrt(np.mean(y * y, axis=1, keepdims=True)) + eps)


def _mut_relu2_unsquared(u):
    return np.maximum(np.asarray(u, dtype=np.float64), 0.0)


def _mut_relu2_no_relu(u):
    return np.asarray(u, dtype=np.float64) ** 2


def _mut_relu2_reads_gate(act, g, u):
    # up-only experts given the gated form's SiLU of u times u
    if act == "relu2_up":
        return O.silu(u) * u
    return _ORIG["activation"](act, g, u)


def _mut_dense_relu2_transposed_up(x, idx, a, W_gate, W_up, W_down, act="silu_glu"):
    if act == "relu2_up":  # input rows of W_up taken in reverse order
        W_up = np.ascontiguousarray(np.asarray(W_up)[:, ::-1, :])
    return _ORIG["expert_ffn_dense"](x, idx, a, W_gate, W_up, W_down, act)


def _mut_dense_down_transposed(x, layer, W_down, k, d):
    Wt = np.ascontiguousarray(np.swapaxes(np.asarray(W_down), 1, 2))
    return _ORIG["moe_layer_dense_down"](x, layer, Wt, k, d)


_ORIG = {name: getattr(O, name) for name in
         ("decode_vq", "expert_matrices", "silu", "gating", "select_topk", "router_logits",
          "expert_ffn", "storage_bits_per_weight", "moe_layer_dense_down", "activation",
          "expert_ffn_dense")}

MUTATIONS = {
    "decode_element_order_reversed": ("decode_vq", _mut_decode_reversed),
    "decode_blocks_across_columns": ("decode_vq", _mut_decode_blocks_across_columns),
    "gate_lowrank_dropped": ("expert_matrices", _mut_drop_gate_lr),
    "down_lowrank_dropped": ("expert_matrices", _mut_drop_down_lr),
    "gate_up_swapped": ("expert_matrices", _mut_swap_gate_up),
    "silu_sign_flipped": ("silu", _mut_silu_sign),
    "softmax_over_all_experts": ("gating", _mut_softmax_all),
    "tie_to_higher_index": ("select_topk", _mut_tie_high),
    "router_bias_dropped": ("router_logits", _mut_no_bias),
    "affinity_not_applied": ("expert_ffn", _mut_unweighted),
    "shared_basis_not_amortised": ("storage_bits_per_weight", _mut_storage_no_basis),
    "dense_baseline_silu_dropped": ("expert_ffn_dense", _mut_dense_no_silu),
    "dense_down_transposed": ("moe_layer_dense_down", _mut_dense_down_transposed),
    "rmsnorm_eps_outside_sqrt": ("rmsnorm", _mut_rmsnorm_eps_outside),
    "relu2_not_squared": ("relu2", _mut_relu2_unsquared),
    "relu2_negative_half_kept": ("relu2", _mut_relu2_no_relu),
    "up_only_given_silu_gating": ("activation", _mut_relu2_reads_gate),
    "dense_relu2_up_rows_reversed": ("expert_ffn_dense", _mut_dense_relu2_transposed_up),
}


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_planted_mistakes_are_caught(name, monkeypatch):
    attr, fn = MUTATIONS[name]
    monkeypatch.setattr(O, attr, fn)
    tripped = []
    for pin in PINS:
        try:
            pin()
        except (AssertionError, ValueError, IndexError):
            tripped.append(pin.__name__)
    assert tripped, f"mutation {name} passed every pin"
