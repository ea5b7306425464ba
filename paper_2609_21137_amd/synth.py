"""Seeded synthetic inputs for the compressed-MoE decode layer.

This module only draws random numbers and packs them into the storage
formats (bf16 bit patterns, uint8 codes, float32 bias). It holds none of the
layer's arithmetic, so the oracle and the GPU path can both consume its
arrays without sharing any computation.

Recipe (one independent PCG64 stream per tensor, keyed by
``SeedSequence([seed, layer, tensor_id])``):

* ``x ~ N(0, 1)``; router ``Wr[H, E] ~ N(0, 1/H)`` (variance), plus a bias
  ``1e-3 * e`` per expert (``+hot_bias`` for the hot experts).
* Code books ``[K, d]`` (one per gate, up, down) ``~ N(0, 0.02)`` (std).
* Codes uniform over ``0..K-1``, one uint8 per block, row-major
  ``[in/d, out]`` per expert.
* Shared basis ``U[H, r] ~ N(0, 1/H)`` (variance), one matrix used for both
  gate and up; private ``V_e[r, I] ~ N(0, 0.01)`` (std). Up-only layers
  (squared-ReLU experts) draw no gate tensors; their up basis has its own
  stream.
* Down: private ``A_e[I, r] ~ N(0, 0.01)`` (std), shared ``B[r, H] ~ N(0, 1/H)``
  (variance).
* Dense bf16 expert matrices (the uncompressed baseline and the dense-down
  variant): ``W_gate, W_up [E, H, I]`` and ``W_down [E, I, H] ~ N(0, 0.02)``
  (std, the scale of a code-book entry), one stream per (tensor, expert).

Normals are drawn in float64, rounded to float32 (round to nearest even) and
then to bf16 (round to nearest even).
"""

from __future__ import annotations

import numpy as np

from .configs import Workload

# fixed stream ids; never renumber (changing one changes every fixture)
_T_X, _T_WR, _T_CBG, _T_CBU, _T_CBD = 1, 2, 3, 4, 5
_T_JG, _T_JU, _T_JD, _T_U, _T_UU = 6, 7, 8, 9, 10
_T_VG, _T_VU, _T_A, _T_B = 11, 12, 13, 14
_T_WG, _T_WU, _T_WD = 15, 16, 17


def _rng(seed: int, layer: int, tensor_id: int, extra: int = 0) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([seed, layer, tensor_id, extra]))


def f32_to_bf16_bits(a) -> np.ndarray:
    """Round float32 values to bf16 (nearest, ties to even); return uint16 bits."""
    f = np.ascontiguousarray(np.asarray(a, dtype=np.float32))
    u = f.view(np.uint32)
    nan = np.isnan(f)
    if nan.any():
        u = np.where(nan, np.uint32(0x7FC00000), u)
    # finite inputs cannot overflow: the largest is 0xFF7FFFFF + 0x8000
    rounded = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return rounded.astype(np.uint16)


def to_bf16_bits(a) -> np.ndarray:
    """float64 -> float32 (nearest even) -> bf16 (nearest even) bit patterns."""
    return f32_to_bf16_bits(np.asarray(a, dtype=np.float64).astype(np.float32))


def _normal_bf16(rng: np.random.Generator, shape, std: float) -> np.ndarray:
    return to_bf16_bits(rng.standard_normal(shape) * std)


def make_layer(H: int, I: int, E: int, d: int, K: int, r: int, seed: int, layer: int = 0,
               hot_experts=(), hot_bias: float = 0.0, separate_up_basis: bool = False,
               up_only: bool = False) -> dict:
    """All weights of one layer as numpy arrays in their storage formats.

    Keys match the C struct ``cardan_layer``. ``U_up`` is the same array as
    ``U_gate`` unless ``separate_up_basis`` is set (then it gets its own
    stream). With ``r == 0`` the low-rank arrays are ``None``. ``up_only``
    (experts without a gate projection): the gate arrays are ``None`` and
    ``U_up`` has its own stream; the other arrays are the same draws.
    """
    if H % d or I % d:
        raise ValueError("H and I must be multiples of d")
    L = {}
    L["router_w"] = _normal_bf16(_rng(seed, layer, _T_WR), (H, E), H ** -0.5)
    bias = 1e-3 * np.arange(E, dtype=np.float64)
    for e in hot_experts:
        bias[e] += hot_bias
    L["router_bias"] = bias.astype(np.float32)
    L["cb_gate"] = None if up_only else _normal_bf16(_rng(seed, layer, _T_CBG), (K, d), 0.02)
    L["cb_up"] = _normal_bf16(_rng(seed, layer, _T_CBU), (K, d), 0.02)
    L["cb_down"] = _normal_bf16(_rng(seed, layer, _T_CBD), (K, d), 0.02)
    L["codes_gate"] = (None if up_only else
                       _rng(seed, layer, _T_JG).integers(0, K, size=(E, H // d, I), dtype=np.uint8))
    L["codes_up"] = _rng(seed, layer, _T_JU).integers(0, K, size=(E, H // d, I), dtype=np.uint8)
    L["codes_down"] = _rng(seed, layer, _T_JD).integers(0, K, size=(E, I // d, H), dtype=np.uint8)
    if r > 0:
        L["U_gate"] = None if up_only else _normal_bf16(_rng(seed, layer, _T_U), (H, r), H ** -0.5)
        L["U_up"] = (_normal_bf16(_rng(seed, layer, _T_UU), (H, r), H ** -0.5)
                     if separate_up_basis or up_only else L["U_gate"])
        L["V_gate"] = None if up_only else _normal_bf16(_rng(seed, layer, _T_VG), (E, r, I), 0.01)
        L["V_up"] = _normal_bf16(_rng(seed, layer, _T_VU), (E, r, I), 0.01)
        L["A_down"] = _normal_bf16(_rng(seed, layer, _T_A), (E, I, r), 0.01)
        L["B_down"] = _normal_bf16(_rng(seed, layer, _T_B), (r, H), H ** -0.5)
    else:
        for key in ("U_gate", "U_up", "V_gate", "V_up", "A_down", "B_down"):
            L[key] = None
    return L


def make_dense_weights(H: int, I: int, E: int, seed: int, layer: int = 0, which=("gate", "up", "down"),
                       experts=None, fill_bits: int = 0) -> dict:
    """Dense bf16 expert matrices ``W_gate``/``W_up`` [E, H, I] and
    ``W_down`` [E, I, H] (those named in ``which``), as bf16 bits.

    Every expert's matrix has its own stream, so ``experts`` (a list of
    expert ids) can restrict the draw to those experts; the others are filled
    with the bf16 pattern ``fill_bits`` (e.g. 0x7FC0, a NaN, to show that
    they are never read).
    """
    ids = {"gate": (_T_WG, (H, I)), "up": (_T_WU, (H, I)), "down": (_T_WD, (I, H))}
    names = {"gate": "W_gate", "up": "W_up", "down": "W_down"}
    todo = range(E) if experts is None else sorted({int(e) for e in experts})
    out = {}
    for key in which:
        tid, shp = ids[key]
        W = np.full((E,) + shp, fill_bits, dtype=np.uint16)
        for e in todo:
            W[e] = _normal_bf16(_rng(seed, layer, tid, e), shp, 0.02)
        out[names[key]] = W
    return out


def make_input(H: int, B: int, seed: int, layer: int = 0, step: int = 0) -> np.ndarray:
    """Decode-step activations ``x[B, H] ~ N(0, 1)`` as bf16 bits."""
    return _normal_bf16(_rng(seed, layer, _T_X, step), (B, H), 1.0)


def workload_layer(w: Workload, layer: int = 0, **kw) -> dict:
    """``make_layer`` for a named workload."""
    return make_layer(w.H, w.I, w.E, w.d, w.K, w.r, w.seed, layer,
                      hot_experts=w.hot_experts, hot_bias=w.hot_bias, up_only=w.act == "relu2_up", **kw)


def workload_input(w: Workload, layer: int = 0, step: int = 0, B: int | None = None) -> np.ndarray:
    """``make_input`` for a named workload (optionally with another batch)."""
    return make_input(w.H, w.B if B is None else B, w.seed, layer, step)
