"""CPU oracle for one compressed-MoE decode layer (test infrastructure only).

This module is TEST INFRASTRUCTURE. Only the test suite, the smoke check in
``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of ``bench.py`` may
import it. The product path (the HIP library and its Python binding) never
imports, calls or links anything here, and this module imports nothing from
the product package.

It is a plain, slow, obviously-correct float64 numpy implementation of what
the hot path computes, written from the paper:

* MoE block semantics (Sec. 2.1): a router picks ``k`` of ``E`` experts for an
  input ``h`` and assigns each an affinity ``a_e``; each selected expert runs
  gate and up projections, combines them with the activation ``phi`` into
  ``p_e``, maps ``p_e`` back to the hidden size with its down projection, and
  the block returns the affinity-weighted sum of the expert outputs.
* Hybrid representation (Sec. 3.1, Eq. (1)): an expert matrix is a blockwise
  VQ part ``Q_B(J_e)`` (Sec. 2.3: each column is cut into length-``d`` blocks
  running along the input dimension, each block replaced by a code word of the
  shared code book ``B``) plus a low-rank part ``D C_e`` on a basis ``D`` shared
  by all experts.
* Storage rate (Sec. 5.5 display and Appendix A.2, Eq. (7)).

Readings where the paper is silent (recorded with the rest in the design doc):

* The down projection is compressed as ``Q_e + A_e B`` with ``B`` [r, H]
  shared on the output side (the workload definition; the paper itself keeps
  down in BF16, Sec. 3.1).
* ``phi`` is SiLU gating: ``p = silu(g) * u`` (``act="silu_glu"``), or, for
  the up-only experts of the paper's Nemotron-3 row (Table 2, projection
  "up"; the squared-ReLU experts of its fidelity test, Sec. 5.7), the squared
  ReLU of the up projection alone, ``p = max(u, 0)^2`` (``act="relu2_up"``;
  the gate tensors are then absent and never read).
* Top-k order is descending logit with exact ties going to the lower expert
  index; the bias is part of the logit; gating is a softmax over the k
  selected logits.
* Inside a code block, code-word element ``i`` maps to input row ``b*d + i``.

Functions:

* ``moe_layer``            -- O1: dense reconstruction of every selected
                              expert's matrices, then plain matmuls.
* ``moe_layer_factored``   -- O3: Eq. (1) evaluated in factored form,
                              ``Q^T x + V^T (U^T x)`` (gate/up) and
                              ``Q^T p + B^T (A^T p)`` (down).
* ``moe_layer_scalar``     -- O2: pure-Python scalar loops for tiny shapes.
* ``moe_layer_dense``      -- the uncompressed baseline: the same MoE block
                              (Sec. 2.1) with dense bf16 expert matrices.
* ``moe_layer_dense_down`` -- compressed gate/up (Eq. (1)) with the down
                              projection kept as a dense bf16 matrix, the
                              paper's own setting (Sec. 3.1).

The first four take ``act`` (``"silu_glu"`` or ``"relu2_up"``), the expert
activation.

All bf16 inputs arrive as raw uint16 bit patterns and are widened exactly.
"""

from __future__ import annotations

import math

import numpy as np

LAYER_KEYS = (
    "router_w", "router_bias",
    "cb_gate", "cb_up", "cb_down",
    "codes_gate", "codes_up", "codes_down",
    "U_gate", "U_up", "V_gate", "V_up",
    "A_down", "B_down",
)


# --------------------------------------------------------------------------
# exact widening of stored inputs
# --------------------------------------------------------------------------
def bf16_to_f64(bits) -> np.ndarray:
    """Widen raw bf16 bit patterns (uint16) to float64 exactly.

    A bf16 value is the upper half of an IEEE binary32 word, so shifting the
    16 stored bits into the high half of a uint32 gives the binary32 value,
    which float64 represents exactly.
    """
    b = np.ascontiguousarray(np.asarray(bits, dtype=np.uint16))
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


def _f(a) -> np.ndarray:
    """Float64 view of an input: bf16 bit patterns are widened, floats cast."""
    a = np.asarray(a)
    if a.dtype == np.uint16:
        return bf16_to_f64(a)
    return a.astype(np.float64)


# --------------------------------------------------------------------------
# router (Sec. 2.1)
# --------------------------------------------------------------------------
def router_logits(x, router_w, router_bias=None) -> np.ndarray:
    """Router scores ``l[t, e] = sum_h x[t, h] * Wr[h, e] + bias[e]`` (Sec. 2.1)."""
    xf = _f(x)
    wr = _f(router_w)
    logits = xf @ wr
    if router_bias is not None:
        logits = logits + _f(router_bias)[None, :]
    return logits


def select_topk(logits, k: int):
    """Pick the ``k`` largest logits per token (Sec. 2.1).

    Experts are ordered by the key ``(-logit, expert)``, i.e. by descending
    logit with exact ties resolved toward the lower expert index, using a plain
    Python sort. Returns ``(idx [B, k] int64, margin [B])`` where ``margin`` is
    the gap between the k-th and (k+1)-th logit (``inf`` when k == E).
    """
    logits = np.asarray(logits, dtype=np.float64)
    B, E = logits.shape
    idx = np.zeros((B, k), dtype=np.int64)
    margin = np.full(B, np.inf)
    for t in range(B):
        order = sorted(range(E), key=lambda e: (-logits[t, e], e))
        idx[t] = order[:k]
        if k < E:
            margin[t] = logits[t, order[k - 1]] - logits[t, order[k]]
    return idx, margin


def gating(logits, idx) -> np.ndarray:
    """Affinities ``a``: a softmax over the k selected logits of each token."""
    logits = np.asarray(logits, dtype=np.float64)
    sel = np.take_along_axis(logits, np.asarray(idx), axis=1)
    w = np.exp(sel - sel.max(axis=1, keepdims=True))
    return w / w.sum(axis=1, keepdims=True)


def route(x, router_w, router_bias, k: int):
    """Router + top-k + gating: returns ``(idx, a, margin, logits)``."""
    logits = router_logits(x, router_w, router_bias)
    idx, margin = select_topk(logits, k)
    return idx, gating(logits, idx), margin, logits


# --------------------------------------------------------------------------
# hybrid representation (Sec. 2.3 and Sec. 3.1, Eq. (1))
# --------------------------------------------------------------------------
def decode_vq(codes, codebook, d: int) -> np.ndarray:
    """Blockwise VQ matrix ``Q_B(J)`` (Sec. 2.3).

    ``codes`` is the index map ``J`` of shape ``[n_in / d, n_out]``; every
    column of the reconstructed ``[n_in, n_out]`` matrix is cut into
    length-``d`` blocks along the input dimension and block ``b`` of column
    ``j`` is the code word ``codebook[J[b, j]]``, so that
    ``Q[b*d + i, j] = codebook[J[b, j], i]``.
    """
    J = np.asarray(codes).astype(np.int64)
    cb = _f(codebook)
    nb, n_out = J.shape
    assert cb.shape[1] == d
    blocks = cb[J]                      # [nb, n_out, d]: code word of block (b, j)
    return blocks.transpose(0, 2, 1).reshape(nb * d, n_out)


def _rank(layer: dict) -> int:
    """Rank r of the layer's shared basis (0 without a low-rank term)."""
    U = layer.get("U_up")
    return 0 if U is None else _f(U).shape[1]


def expert_matrices(layer: dict, e: int, d: int, act: str = "silu_glu"):
    """Dense reconstructions of expert ``e``'s gate, up and down matrices.

    Gate/up follow Eq. (1): ``W = Q_B(J_e) + D C_e`` with ``D = U`` [H, r]
    and ``C_e = V_e`` [r, I], giving [H, I]. Down is ``Q_B(J^d_e) + A_e B``
    with ``A_e`` [I, r] private and ``B`` [r, H] shared, giving [I, H].
    Up-only experts (``act="relu2_up"``) have no gate matrix (``None``).
    """
    gated = act == "silu_glu"
    Wg = decode_vq(layer["codes_gate"][e], layer["cb_gate"], d) if gated else None
    Wu = decode_vq(layer["codes_up"][e], layer["cb_up"], d)
    Wd = decode_vq(layer["codes_down"][e], layer["cb_down"], d)
    if _rank(layer) > 0:
        if gated:
            Wg = Wg + _f(layer["U_gate"]) @ _f(layer["V_gate"][e])
        Wu = Wu + _f(layer["U_up"]) @ _f(layer["V_up"][e])
        Wd = Wd + _f(layer["A_down"][e]) @ _f(layer["B_down"])
    return Wg, Wu, Wd


def silu(g):
    """SiLU ``g * sigmoid(g)``, the gating activation phi of the workload."""
    g = np.asarray(g, dtype=np.float64)
    return g / (1.0 + np.exp(-g))


def relu2(u):
    """Squared ReLU ``max(u, 0)^2``, the activation of up-only experts."""
    u = np.asarray(u, dtype=np.float64)
    return np.maximum(u, 0.0) ** 2


ACTIVATIONS = ("silu_glu", "relu2_up")


def activation(act: str, g, u):
    """The expert activation phi (Sec. 2.1): ``silu(g) * u`` for gated
    experts, ``max(u, 0)^2`` for up-only ones (``g`` unused, may be None)."""
    if act == "silu_glu":
        return silu(g) * u
    if act == "relu2_up":
        return relu2(u)
    raise ValueError(f"unknown activation {act!r}")


def shared_proj(x, U) -> np.ndarray:
    """Shared rank-r projection ``z = D^T h`` for every token (Sec. 4.2)."""
    return _f(x) @ _f(U)


# --------------------------------------------------------------------------
# O1: the layer from dense reconstructions
# --------------------------------------------------------------------------
def expert_ffn(x, idx, a, layer: dict, d: int, act: str = "silu_glu") -> np.ndarray:
    """Expert computation plus the affinity-weighted sum for fixed routing.

    For token ``t`` and its j-th selected expert ``e``: ``g = Wg^T x_t``,
    ``u = Wu^T x_t``, ``p = silu(g) * u`` (up-only: ``max(u, 0)^2``),
    ``y_e = Wd^T p``; the output is ``sum_j a[t, j] * y_e`` summed in
    selection order (Sec. 2.1).
    """
    xf = _f(x)
    idx = np.asarray(idx)
    a = np.asarray(a, dtype=np.float64)
    B = xf.shape[0]
    H = xf.shape[1]
    y = np.zeros((B, H))
    cache = {}
    for t in range(B):
        for j in range(idx.shape[1]):
            e = int(idx[t, j])
            if e not in cache:
                cache[e] = expert_matrices(layer, e, d, act)
            Wg, Wu, Wd = cache[e]
            g = None if Wg is None else Wg.T @ xf[t]
            u = Wu.T @ xf[t]
            p = activation(act, g, u)
            y[t] += a[t, j] * (Wd.T @ p)
    return y


def moe_layer(x, layer: dict, k: int, d: int, act: str = "silu_glu"):
    """O1: route, then run the selected experts from dense reconstructions.

    Returns ``(y [B, H] f64, idx [B, k], a [B, k], margin [B])``.
    """
    idx, a, margin, _ = route(x, layer["router_w"], layer.get("router_bias"), k)
    y = expert_ffn(x, idx, a, layer, d, act)
    return y, idx, a, margin


# --------------------------------------------------------------------------
# O3: Eq. (1) in factored form
# --------------------------------------------------------------------------
def expert_ffn_factored(x, idx, a, layer: dict, d: int, z=None, act: str = "silu_glu") -> np.ndarray:
    """Same result as ``expert_ffn`` evaluated as in Eq. (1).

    Gate/up: ``o = Q_B(J_e)^T x + V_e^T (U^T x)`` with the shared projection
    ``U^T x`` computed once per token (Sec. 4.2); down:
    ``y_e = Q_B(J^d_e)^T p + B^T (A_e^T p)``. ``z`` optionally supplies the
    shared projections as ``[2, B, r]`` (gate, up; up-only experts read the
    up half alone). Each selected expert's
    VQ matrices are rebuilt once and applied to all of its tokens; the
    per-token expert outputs are then summed in selection order.
    """
    xf = _f(x)
    idx = np.asarray(idx)
    a = np.asarray(a, dtype=np.float64)
    B, H = xf.shape
    k = idx.shape[1]
    has_lr = _rank(layer) > 0
    gated = act == "silu_glu"
    if has_lr and z is None:
        zg = shared_proj(xf, layer["U_gate"]) if gated else None
        z = (zg, shared_proj(xf, layer["U_up"]))
    contrib = np.zeros((B, k, H))
    for e in sorted(set(int(v) for v in idx.ravel())):
        Qg = decode_vq(layer["codes_gate"][e], layer["cb_gate"], d) if gated else None
        Qu = decode_vq(layer["codes_up"][e], layer["cb_up"], d)
        Qd = decode_vq(layer["codes_down"][e], layer["cb_down"], d)
        for t, j in zip(*np.nonzero(idx == e)):
            g = Qg.T @ xf[t] if gated else None
            u = Qu.T @ xf[t]
            if has_lr:
                if gated:
                    g = g + _f(layer["V_gate"][e]).T @ np.asarray(z[0][t], dtype=np.float64)
                u = u + _f(layer["V_up"][e]).T @ np.asarray(z[1][t], dtype=np.float64)
            p = activation(act, g, u)
            ye = Qd.T @ p
            if has_lr:
                ye = ye + _f(layer["B_down"]).T @ (_f(layer["A_down"][e]).T @ p)
            contrib[t, j] = a[t, j] * ye
    y = np.zeros((B, H))
    for j in range(k):
        y += contrib[:, j]
    return y


def moe_layer_factored(x, layer: dict, k: int, d: int, act: str = "silu_glu"):
    """O3: route, then Eq. (1) in factored form. Same return as ``moe_layer``."""
    idx, a, margin, _ = route(x, layer["router_w"], layer.get("router_bias"), k)
    return expert_ffn_factored(x, idx, a, layer, d, act=act), idx, a, margin


# --------------------------------------------------------------------------
# dense-weight baselines
# --------------------------------------------------------------------------
def expert_ffn_dense(x, idx, a, W_gate, W_up, W_down, act: str = "silu_glu") -> np.ndarray:
    """Expert computation for fixed routing with dense expert matrices
    ``W_gate[e]``, ``W_up[e]`` [H, I] and ``W_down[e]`` [I, H] (Sec. 2.1):
    ``y_t = sum_j a[t, j] * W_down[e]^T (silu(W_gate[e]^T x_t) * W_up[e]^T x_t)``
    in selection order (up-only experts: ``max(W_up[e]^T x_t, 0)^2``,
    ``W_gate`` unused)."""
    xf = _f(x)
    idx = np.asarray(idx)
    a = np.asarray(a, dtype=np.float64)
    y = np.zeros((xf.shape[0], xf.shape[1]))
    for t in range(xf.shape[0]):
        for j in range(idx.shape[1]):
            e = int(idx[t, j])
            g = _f(W_gate[e]).T @ xf[t] if act == "silu_glu" else None
            u = _f(W_up[e]).T @ xf[t]
            p = activation(act, g, u)
            y[t] += a[t, j] * (_f(W_down[e]).T @ p)
    return y


def moe_layer_dense(x, router_w, router_bias, W_gate, W_up, W_down, k: int, act: str = "silu_glu"):
    """The uncompressed baseline layer: route, then dense experts.
    Returns ``(y [B, H] f64, idx [B, k], a [B, k], margin [B])``."""
    idx, a, margin, _ = route(x, router_w, router_bias, k)
    return expert_ffn_dense(x, idx, a, W_gate, W_up, W_down, act), idx, a, margin


def moe_layer_dense_down(x, layer: dict, W_down, k: int, d: int):
    """Gate and up from Eq. (1) (VQ plus shared-basis low rank), down a dense
    bf16 matrix ``W_down[e]`` [I, H]. Same return as ``moe_layer``."""
    idx, a, margin, _ = route(x, layer["router_w"], layer.get("router_bias"), k)
    xf = _f(x)
    y = np.zeros((xf.shape[0], xf.shape[1]))
    cache = {}
    for t in range(xf.shape[0]):
        for j in range(idx.shape[1]):
            e = int(idx[t, j])
            if e not in cache:
                Wg, Wu, _ = expert_matrices(layer, e, d)
                cache[e] = (Wg, Wu)
            Wg, Wu = cache[e]
            p = silu(Wg.T @ xf[t]) * (Wu.T @ xf[t])
            y[t] += a[t, j] * (_f(W_down[e]).T @ p)
    return y, idx, a, margin


# --------------------------------------------------------------------------
# O2: scalar brute force (tiny shapes only)
# --------------------------------------------------------------------------
def moe_layer_scalar(x, layer: dict, k: int, d: int, act: str = "silu_glu"):
    """O2: the whole layer with Python floats and explicit loops.

    Every weight is formed element by element from its definition,
    ``W[i][j] = cb[J[i // d][j]][i % d] + sum_q U[i][q] * V[q][j]``, and every
    product is an explicit loop; no numpy arithmetic is used. Intended for
    shapes with H, I <= 32.
    """
    X = _f(x).tolist()
    Wr = _f(layer["router_w"]).tolist()
    bias = None if layer.get("router_bias") is None else _f(layer["router_bias"]).tolist()
    gated = act == "silu_glu"
    if act not in ACTIVATIONS:
        raise ValueError(f"unknown activation {act!r}")
    cbg = _f(layer["cb_gate"]).tolist() if gated else None
    cbu = _f(layer["cb_up"]).tolist()
    cbd = _f(layer["cb_down"]).tolist()
    Jg = np.asarray(layer["codes_gate"]).tolist() if gated else None
    Ju = np.asarray(layer["codes_up"]).tolist()
    Jd = np.asarray(layer["codes_down"]).tolist()
    has_lr = _rank(layer) > 0
    Ug = Vg = None
    if has_lr:
        if gated:
            Ug = _f(layer["U_gate"]).tolist()
            Vg = _f(layer["V_gate"]).tolist()
        Uu = _f(layer["U_up"]).tolist()
        Vu = _f(layer["V_up"]).tolist()
        Ad = _f(layer["A_down"]).tolist()
        Bd = _f(layer["B_down"]).tolist()
        r = len(Uu[0])
    else:
        r = 0
    B = len(X)
    H = len(X[0])
    E = len(Wr[0])
    I = len(Ju[0][0])

    def w_in_out(cb, J, U, V, e, i, j):
        val = cb[J[e][i // d][j]][i % d]
        for q in range(r):
            val += U[i][q] * V[e][q][j]
        return val

    def w_down(e, i, h):
        val = cbd[Jd[e][i // d][h]][i % d]
        for q in range(r):
            val += Ad[e][i][q] * Bd[q][h]
        return val

    Y, IDX, A, MARGIN = [], [], [], []
    for t in range(B):
        logit = []
        for e in range(E):
            s = 0.0
            for h in range(H):
                s += X[t][h] * Wr[h][e]
            if bias is not None:
                s += bias[e]
            logit.append(s)
        # selection sort, descending, lower index wins ties
        remaining = list(range(E))
        chosen = []
        for _ in range(k):
            best = remaining[0]
            for e in remaining[1:]:
                if logit[e] > logit[best]:
                    best = e
            chosen.append(best)
            remaining.remove(best)
        MARGIN.append(logit[chosen[-1]] - max(logit[e] for e in remaining) if remaining else math.inf)
        m = max(logit[e] for e in chosen)
        ex = [math.exp(logit[e] - m) for e in chosen]
        tot = sum(ex)
        aff = [v / tot for v in ex]
        yt = [0.0] * H
        for j, e in enumerate(chosen):
            g = [0.0] * I
            u = [0.0] * I
            for c in range(I):
                for i in range(H):
                    if gated:
                        g[c] += X[t][i] * w_in_out(cbg, Jg, Ug, Vg, e, i, c)
                    u[c] += X[t][i] * w_in_out(cbu, Ju, Uu if r else None, Vu if r else None, e, i, c)
            if gated:
                p = [g[c] / (1.0 + math.exp(-g[c])) * u[c] for c in range(I)]
            else:
                p = [(u[c] if u[c] > 0.0 else 0.0) * (u[c] if u[c] > 0.0 else 0.0) for c in range(I)]
            for h in range(H):
                s = 0.0
                for i in range(I):
                    s += p[i] * w_down(e, i, h)
                yt[h] += aff[j] * s
        Y.append(yt)
        IDX.append(chosen)
        A.append(aff)
    return (np.array(Y), np.array(IDX, dtype=np.int64), np.array(A), np.array(MARGIN))


# --------------------------------------------------------------------------
# RMS normalisation between stacked layers (48-layer decode step)
# --------------------------------------------------------------------------
def rmsnorm(y, eps: float = 1e-6) -> np.ndarray:
    """``y / sqrt(mean(y^2) + eps)`` per row, no learned scale (float64)."""
    y = np.asarray(y, dtype=np.float64)
    return y / np.sqrt(np.mean(y * y, axis=1, keepdims=True) + eps)


# --------------------------------------------------------------------------
# storage accounting (Sec. 5.5 display; Appendix A.2, Eq. (7))
# --------------------------------------------------------------------------
def storage_bits_per_weight(d: int, K: int, r: int, H: int, I: int, E: int,
                            b_index: int | None = None, b_coef: int = 16,
                            b_codebook: int = 16, b_basis: int = 16) -> float:
    """Bits per original weight of one compressed projection, Eq. (7).

    ``log2(K)/d`` for the private index map (stored with ``b_index`` bits per
    index, 8 for K <= 256), ``b_C r / H`` for the private coefficients, and the
    shared code book and basis amortised over the ``E`` experts' ``H I``
    weights. With BF16 factors and one-byte indices this is
    ``8/d + 16 r/H + 16 r/(E I) + 16 K d/(E H I)``.
    """
    if b_index is None:
        b_index = max(1, math.ceil(math.log2(K)))
        b_index = 8 if b_index <= 8 else 16
    return (b_index / d + b_coef * r / H
            + (b_codebook * K * d + b_basis * H * r) / (E * H * I))
