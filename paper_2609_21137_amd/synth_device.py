"""Seeded synthetic layers drawn directly on the GPU (for timing runs).

The same laws as ``synth`` (variance 1/H for the router, U and B; std 0.02
for code books and dense expert matrices; std 0.01 for V and A; codes uniform
over 0..K-1; router bias 1e-3 * e plus the hot-expert bias), drawn with
torch's device generators instead of numpy's PCG64, so a 150 MB layer takes
milliseconds instead of seconds. The values differ from ``synth``'s; only the
timing runs use them (the parity tests use ``synth``, which the oracle reads
too). Like ``synth``, this module draws random numbers only and holds none of
the layer's arithmetic.
"""

from __future__ import annotations

import torch

from .configs import Workload

# stream ids of the tensors (distinct from one another per (seed, layer))
_IDS = {"router_w": 2, "cb_gate": 3, "cb_up": 4, "cb_down": 5, "codes_gate": 6, "codes_up": 7,
        "codes_down": 8, "U_gate": 9, "U_up": 10, "V_gate": 11, "V_up": 12, "A_down": 13, "B_down": 14,
        "W_gate": 15, "W_up": 16, "W_down": 17}


def _gen(seed: int, layer: int, tensor: str) -> torch.Generator:
    g = torch.Generator(device="cuda")
    g.manual_seed(((seed * 1_000_003 + layer) * 101 + _IDS[tensor]) & 0x7FFFFFFFFFFFFFFF)
    return g


def _normal_bf16(shape, std: float, g: torch.Generator) -> torch.Tensor:
    # float32 normals rounded to bf16 (nearest, ties to even)
    return (torch.randn(shape, generator=g, device="cuda", dtype=torch.float32) * std).to(torch.bfloat16)


def _codes(shape, K: int, g: torch.Generator) -> torch.Tensor:
    return torch.randint(0, K, shape, generator=g, device="cuda", dtype=torch.uint8)


def layer_tensors(w: Workload, layer: int) -> dict:
    """One compressed layer's device tensors, keyed like ``cardan_layer``
    (``U_up`` is the same tensor as ``U_gate``; ``None`` where r == 0; up-only
    layers have no gate tensors and their own ``U_up``)."""
    H, I, E, d, K, r = w.H, w.I, w.E, w.d, w.K, w.r
    up_only = w.act == "relu2_up"
    T = {"router_w": _normal_bf16((H, E), H ** -0.5, _gen(w.seed, layer, "router_w"))}
    bias = 1e-3 * torch.arange(E, dtype=torch.float64)
    for e in w.hot_experts:
        bias[e] += w.hot_bias
    T["router_bias"] = bias.to(torch.float32).cuda()
    for cb in ("cb_gate", "cb_up", "cb_down"):
        T[cb] = _normal_bf16((K, d), 0.02, _gen(w.seed, layer, cb))
    T["codes_gate"] = None if up_only else _codes((E, H // d, I), K, _gen(w.seed, layer, "codes_gate"))
    T["codes_up"] = _codes((E, H // d, I), K, _gen(w.seed, layer, "codes_up"))
    T["codes_down"] = _codes((E, I // d, H), K, _gen(w.seed, layer, "codes_down"))
    if up_only:
        T["cb_gate"] = None
    if r > 0:
        T["U_gate"] = None if up_only else _normal_bf16((H, r), H ** -0.5, _gen(w.seed, layer, "U_gate"))
        T["U_up"] = _normal_bf16((H, r), H ** -0.5, _gen(w.seed, layer, "U_up")) if up_only else T["U_gate"]
        T["V_gate"] = None if up_only else _normal_bf16((E, r, I), 0.01, _gen(w.seed, layer, "V_gate"))
        T["V_up"] = _normal_bf16((E, r, I), 0.01, _gen(w.seed, layer, "V_up"))
        T["A_down"] = _normal_bf16((E, I, r), 0.01, _gen(w.seed, layer, "A_down"))
        T["B_down"] = _normal_bf16((r, H), H ** -0.5, _gen(w.seed, layer, "B_down"))
    else:
        for key in ("U_gate", "U_up", "V_gate", "V_up", "A_down", "B_down"):
            T[key] = None
    return T


def dense_tensors(w: Workload, layer: int, names=("W_gate", "W_up", "W_down")) -> dict:
    """Dense bf16 expert matrices W_gate, W_up [E, H, I] and W_down [E, I, H]
    (std 0.02), those named in ``names``."""
    out = {}
    for n in names:
        shp = (w.E, w.I, w.H) if n == "W_down" else (w.E, w.H, w.I)
        out[n] = _normal_bf16(shp, 0.02, _gen(w.seed, layer, n))
    return out
