"""Offline construction of a compressed MoE layer from dense expert weights.

This is the training-free initialisation of the hybrid representation
(Sec. 3.3): product quantisation of the expert matrices into one shared code
book per projection and private index maps, then the closed-form whitened
shared-basis correction of the post-VQ residuals (Appendix A.1, Eq. (4)-(6)),
optionally with the route-aware expert weights ``w_e``. The paper's
end-to-end distillation (Eq. (3)) needs a trained model and is not here.

Everything runs on the host in float64 (numpy); the result is a layer dict
in the storage formats the kernels read (bf16 bit patterns, uint8 codes,
keys of ``cardan_layer``), so a fitted layer goes through the same library
calls as any other.

Layouts (as the kernels read them):

* gate/up ``W[e]`` is ``[H, I]`` (input rows, output columns), down ``W[e]``
  is ``[I, H]``; a VQ block is ``d`` consecutive input rows of one column, so
  ``Q[b*d + i, j] = codebook[codes[b, j], i]`` (Sec. 2.3);
* gate/up: ``W_e ~ Q_e + D C_e`` with the basis ``D`` = ``U`` ``[H, r]``
  shared by the layer's experts and ``C_e`` = ``V[e]`` ``[r, I]`` (Eq. (1));
* down: ``W_e ~ Q_e + A_e B`` with ``A_e`` = ``A_down[e]`` ``[I, r]`` private
  and ``B`` = ``B_down`` ``[r, H]`` shared on the output side. The paper
  keeps down in bf16; its correction here is the output-side counterpart of
  Eq. (4)-(6): the minimiser of ``sum_e w_e || S_e^{1/2} (Delta_e - A_e B) ||_F^2``
  with ``S_e`` the second moment of expert e's down input ``p``, solved by
  the same Ky Fan argument (``B`` spans the top-r eigenspace of
  ``sum_e w_e Delta_e^T S_e Delta_e``, then ``A_e = Delta_e B^T``).
"""

from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

from .synth import to_bf16_bits

ACTIVATIONS = ("silu_glu", "relu2_up")


def bf16_value(bits) -> np.ndarray:
    """Exact float64 value of bf16 bit patterns."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32).astype(np.float64)


def _f64(a) -> np.ndarray:
    a = np.asarray(a)
    return bf16_value(a) if a.dtype == np.uint16 else a.astype(np.float64)


# --------------------------------------------------------------------------
# product quantisation (Sec. 3.3): one code book of K words of length d per
# projection, shared by every block of every expert
# --------------------------------------------------------------------------
def to_blocks(W: np.ndarray, d: int) -> np.ndarray:
    """Blocks of ``W [E, n_in, n_out]``: ``[E, n_in/d, n_out, d]`` with block
    ``(e, b, j)`` = ``W[e, b*d:(b+1)*d, j]``."""
    E, n_in, n_out = W.shape
    if n_in % d:
        raise ValueError(f"input size {n_in} is not a multiple of d={d}")
    return W.reshape(E, n_in // d, d, n_out).transpose(0, 1, 3, 2)


def decode(codes: np.ndarray, codebook: np.ndarray, d: int) -> np.ndarray:
    """``[E, n_in/d, n_out]`` codes -> ``[E, n_in, n_out]`` matrices."""
    J = np.asarray(codes).astype(np.int64)
    blk = np.asarray(codebook, dtype=np.float64)[J]          # [E, nb, n_out, d]
    E, nb, n_out, _ = blk.shape
    return blk.transpose(0, 1, 3, 2).reshape(E, nb * d, n_out)


def _nearest(X: np.ndarray, C: np.ndarray, chunk: int = 1 << 16):
    """Index of the nearest row of C for every row of X (squared Euclidean;
    exact ties go to the lower index) and the squared distances."""
    idx = np.empty(X.shape[0], dtype=np.int64)
    dist = np.empty(X.shape[0])
    cc = np.einsum("kd,kd->k", C, C)
    for s in range(0, X.shape[0], chunk):
        x = X[s:s + chunk]
        d2 = np.einsum("nd,nd->n", x, x)[:, None] - 2.0 * (x @ C.T) + cc[None, :]
        i = np.argmin(d2, axis=1)
        idx[s:s + chunk] = i
        dist[s:s + chunk] = np.maximum(d2[np.arange(x.shape[0]), i], 0.0)
    return idx, dist


def kmeans(X: np.ndarray, K: int, iters: int = 25, seed: int = 0, n_init: int = 1):
    """Lloyd's k-means with k-means++ seeding (seeded generators), the best
    of ``n_init`` runs by final sum of squares.

    Returns ``(codebook [K, d], assignment [N], sse per iteration of the
    kept run)``. A cluster that empties is re-seeded with the point farthest
    from its code word. With N <= K every point is its own code word (the
    rest repeat the last point)."""
    X = np.asarray(X, dtype=np.float64)
    N, d = X.shape
    if N <= K:
        C = np.concatenate([X, np.repeat(X[-1:], K - N, axis=0)]) if N < K else X.copy()
        return C, np.arange(N), [0.0]
    runs = [_lloyd(X, K, iters, seed + 7919 * i) for i in range(max(1, n_init))]
    return min(runs, key=lambda run: run[2][-1])


def _lloyd(X: np.ndarray, K: int, iters: int, seed: int):
    N, d = X.shape
    rng = np.random.default_rng(seed)
    C = np.empty((K, d))
    C[0] = X[rng.integers(N)]
    _, best = _nearest(X, C[:1])
    for j in range(1, K):
        tot = best.sum()
        i = rng.choice(N, p=best / tot) if tot > 0 else rng.integers(N)
        C[j] = X[i]
        best = np.minimum(best, np.einsum("nd,nd->n", X - C[j], X - C[j]))
    history = []
    assign, dist = _nearest(X, C)
    for _ in range(iters):
        history.append(float(dist.sum()))
        counts = np.bincount(assign, minlength=K)
        sums = np.stack([np.bincount(assign, weights=X[:, c], minlength=K) for c in range(d)], axis=1)
        empty = counts == 0
        C[~empty] = sums[~empty] / counts[~empty, None]
        for j in np.nonzero(empty)[0]:
            far = int(np.argmax(dist))
            C[j] = X[far]
            dist[far] = 0.0
        new_assign, dist = _nearest(X, C)
        if np.array_equal(new_assign, assign) and not empty.any():
            assign = new_assign
            break
        assign = new_assign
    history.append(float(dist.sum()))
    return C, assign, history


def pq_init(W: np.ndarray, d: int, K: int, iters: int = 25, seed: int = 0, n_init: int = 4):
    """Code book ``[K, d]`` and codes ``[E, n_in/d, n_out]`` (uint8) of the
    projection ``W [E, n_in, n_out]``: k-means over all of its blocks."""
    if not 1 <= K <= 256:
        raise ValueError("K must be in [1, 256] (one byte per code)")
    blk = to_blocks(np.asarray(W, dtype=np.float64), d)
    C, assign, hist = kmeans(blk.reshape(-1, d), K, iters, seed, n_init)
    return C, assign.reshape(blk.shape[:3]).astype(np.uint8), hist


# --------------------------------------------------------------------------
# calibration statistics
# --------------------------------------------------------------------------
def route(X: np.ndarray, router_w, router_bias, k: int):
    """Top-k experts (descending logit, exact ties to the lower index) and
    their softmax affinities, per row of ``X [N, H]``."""
    logits = X @ _f64(router_w)
    if router_bias is not None:
        logits = logits + np.asarray(router_bias, dtype=np.float64)[None, :]
    order = np.argsort(-logits, axis=1, kind="stable")[:, :k]
    sel = np.take_along_axis(logits, order, axis=1)
    ex = np.exp(sel - sel[:, :1])
    return order, ex / ex.sum(axis=1, keepdims=True)


def _weights_of(idx, a, E: int) -> np.ndarray:
    w = np.zeros(E)
    np.add.at(w, idx.ravel(), (a * a).ravel())
    return w / idx.shape[0]


def route_weights(X, router_w, router_bias, k: int, E: int) -> np.ndarray:
    """Route-aware expert weights ``w_e = E[1(e in S(h)) a_e^2]`` over the
    calibration rows (Appendix A.1)."""
    idx, a = route(_f64(X), router_w, router_bias, k)
    return _weights_of(idx, a, E)


def activation(act: str, g, u):
    if act == "silu_glu":
        return g / (1.0 + np.exp(-g)) * u
    if act == "relu2_up":
        return np.maximum(u, 0.0) ** 2
    raise ValueError(f"unknown activation {act!r}")


# --------------------------------------------------------------------------
# the whitened shared-basis correction (Appendix A.1)
# --------------------------------------------------------------------------
def input_basis_fit(residuals, weights, Sigma, r: int):
    """Eq. (4)-(6) for input-side residuals ``Delta_m [H, n]`` sharing one
    basis: ``min sum_m w_m || Sigma^{1/2} (Delta_m - D C_m) ||_F^2``.

    ``R = chol(Sigma)`` (``Sigma = R R^T``), ``U_r`` = the top-r eigenvectors
    of ``R^T (sum_m w_m Delta_m Delta_m^T) R`` (Eq. (5)), ``D = R^{-T} U_r``
    and ``C_m = (D^T Sigma D)^{-1} D^T Sigma Delta_m`` (Eq. (6)). Returns
    ``(D [H, r], [C_m [r, n]], eigenvalues in descending order)``."""
    Sigma = np.asarray(Sigma, dtype=np.float64)
    H = Sigma.shape[0]
    R = np.linalg.cholesky(Sigma)
    G = np.zeros((H, H))
    for Dm, wm in zip(residuals, weights):
        G += wm * (Dm @ Dm.T)
    G = R.T @ G @ R
    lam, vec = np.linalg.eigh((G + G.T) / 2)
    order = np.argsort(lam)[::-1]
    lam, vec = lam[order], vec[:, order]
    U_r = vec[:, :r]
    D = np.linalg.solve(R.T, U_r)
    M = D.T @ Sigma @ D
    C = [np.linalg.solve(M, D.T @ Sigma @ Dm) for Dm in residuals]
    return D, C, lam


def output_basis_fit(residuals, weights, S, r: int):
    """Output-side counterpart for residuals ``Delta_e [n_in, H]`` sharing a
    row basis ``B [r, H]``: ``min sum_e w_e || S_e^{1/2} (Delta_e - A_e B) ||_F^2``
    with ``S_e`` the second moment of expert e's input (``None``: identity).
    ``B`` = the top-r eigenvectors of ``sum_e w_e Delta_e^T S_e Delta_e`` (as
    rows), ``A_e = Delta_e B^T``. Returns ``(B, [A_e], eigenvalues)``."""
    H = residuals[0].shape[1]
    G = np.zeros((H, H))
    for e, (De, we) in enumerate(zip(residuals, weights)):
        SD = De if S is None or S[e] is None else S[e] @ De
        G += we * (De.T @ SD)
    lam, vec = np.linalg.eigh((G + G.T) / 2)
    order = np.argsort(lam)[::-1]
    lam, vec = lam[order], vec[:, order]
    B = vec[:, :r].T
    return B, [De @ B.T for De in residuals], lam


# --------------------------------------------------------------------------
# the whole layer
# --------------------------------------------------------------------------
@dataclass
class FitReport:
    """Quality of a fitted layer on its calibration rows: NMSE of the
    input-side projections (Eq. (2)) for VQ alone and VQ + low rank, the
    whitened objectives, and the expert weights used."""
    nmse_vq: float = 0.0
    nmse_vq_lr: float = 0.0
    nmse_down_vq: float = 0.0
    nmse_down_vq_lr: float = 0.0
    weights: np.ndarray = field(default_factory=lambda: np.zeros(0))
    kmeans_sse: dict = field(default_factory=dict)   # k-means sum of squares per iteration
    factors: dict = field(default_factory=dict)      # float64 D, C, B, A and the eigenvalues
    Q: dict = field(default_factory=dict)            # decoded VQ matrices per projection


def nmse(W_hat, W, X) -> float:
    """Eq. (2): sum ||W_hat^T h - W^T h||^2 / sum ||W^T h||^2 over the rows h
    of X and the matrices given (each ``[n_in, n_out]``)."""
    num = den = 0.0
    for Wh, Wt in zip(W_hat, W):
        ref = X @ Wt
        num += float(np.sum((X @ Wh - ref) ** 2))
        den += float(np.sum(ref ** 2))
    return num / den


def fit_layer(dense: dict, router_w, router_bias, X_calib, k: int, d: int, K: int, r: int,
              act: str = "silu_glu", route_aware: bool = True, kmeans_iters: int = 25,
              kmeans_init: int = 4, seed: int = 0):
    """Compressed layer from dense expert weights.

    ``dense`` holds ``W_up`` (and ``W_gate`` unless ``act == "relu2_up"``)
    ``[E, H, I]`` and ``W_down`` ``[E, I, H]`` as float64 or bf16 bits;
    ``X_calib [N, H]`` are calibration activations (N >= H for a full-rank
    second moment). The gate and up residuals share one basis ``U`` (one
    ``D`` per layer); ``route_aware`` selects ``w_e = E[1(e in S(h)) a_e^2]``
    (else ``w_e = 1``); the down correction weights expert e's input second
    moment by its routing (``1(e in S(h)) a_e^2``) in the route-aware case.

    Returns ``(layer dict in storage formats, FitReport)``; the float64
    factors are in ``report.factors``."""
    if act not in ACTIVATIONS:
        raise ValueError(f"unknown activation {act!r}")
    X = _f64(X_calib)
    N, H = X.shape
    gated = act == "silu_glu"
    projs = (["gate"] if gated else []) + ["up"]
    W = {p: _f64(dense["W_" + p]) for p in projs}
    Wd = _f64(dense["W_down"])
    E, _, I = W["up"].shape
    rep = FitReport()
    layer = {"router_w": np.asarray(router_w, dtype=np.uint16),
             "router_bias": None if router_bias is None else np.asarray(router_bias, dtype=np.float32)}

    # product quantisation, one code book per projection (Sec. 3.3)
    Q, cb_bits = {}, {}
    for i, p in enumerate(projs + ["down"]):
        Wp = Wd if p == "down" else W[p]
        C, codes, hist = pq_init(Wp, d, K, kmeans_iters, seed + i, kmeans_init)
        cb_bits[p] = to_bf16_bits(C)
        layer["cb_" + p] = cb_bits[p]
        layer["codes_" + p] = codes
        # the residual is taken against the code book as stored (bf16)
        Q[p] = decode(codes, bf16_value(cb_bits[p]), d)
        rep.kmeans_sse[p] = hist
    if not gated:
        layer["cb_gate"] = layer["codes_gate"] = None

    # calibration statistics
    Sigma = X.T @ X / N
    idx, a = route(X, router_w, router_bias, k)
    w = _weights_of(idx, a, E) if route_aware else np.ones(E)
    rep.weights = w

    rep.nmse_vq = nmse([Q[p][e] for p in projs for e in range(E)],
                       [W[p][e] for p in projs for e in range(E)], X)
    factors = {}
    if r > 0:
        # Eq. (4)-(6): one basis for the gate and up residuals of every expert
        res = [W[p][e] - Q[p][e] for p in projs for e in range(E)]
        wts = [w[e] for p in projs for e in range(E)]
        D, Cm, lam = input_basis_fit(res, wts, Sigma, r)
        Ce = {p: np.stack(Cm[j * E:(j + 1) * E]) for j, p in enumerate(projs)}
        factors.update(D=D, C=Ce, eig_in=lam)
        U_bits = to_bf16_bits(D)
        layer["U_up"] = U_bits
        layer["U_gate"] = U_bits if gated else None
        layer["V_up"] = to_bf16_bits(Ce["up"])
        layer["V_gate"] = to_bf16_bits(Ce["gate"]) if gated else None
        rep.nmse_vq_lr = nmse([Q[p][e] + D @ Ce[p][e] for p in projs for e in range(E)],
                              [W[p][e] for p in projs for e in range(E)], X)

        # the down input of every expert on the calibration rows (teacher)
        S = []
        for e in range(E):
            u = X @ W["up"][e]
            g = X @ W["gate"][e] if gated else None
            P = activation(act, g, u)                       # [N, I]
            if route_aware:
                sel = (idx == e)
                coef = (a * a * sel).sum(axis=1)              # 1(e in S) a_e^2 per row
                S.append((P * coef[:, None]).T @ P / N)
            else:
                S.append(P.T @ P / N)
        res_d = [Wd[e] - Q["down"][e] for e in range(E)]
        Bm, Ae, lam_d = output_basis_fit(res_d, np.ones(E), S, r)
        factors.update(B=Bm, A=np.stack(Ae), eig_out=lam_d, S_down=S)
        layer["A_down"] = to_bf16_bits(np.stack(Ae))
        layer["B_down"] = to_bf16_bits(Bm)
        Pall = np.concatenate([activation(act, X @ W["gate"][e] if gated else None, X @ W["up"][e])
                               for e in range(E)])
        rep.nmse_down_vq = nmse([Q["down"][e] for e in range(E)], [Wd[e] for e in range(E)], Pall)
        rep.nmse_down_vq_lr = nmse([Q["down"][e] + Ae[e] @ Bm for e in range(E)],
                                   [Wd[e] for e in range(E)], Pall)
    else:
        for key in ("U_gate", "U_up", "V_gate", "V_up", "A_down", "B_down"):
            layer[key] = None
        rep.nmse_vq_lr = rep.nmse_vq
    rep.factors = factors
    rep.Q = Q
    return layer, rep
