"""Offline factor fitting (``paper_2609_21137_amd.fit``) against what the
mathematics fixes, on the CPU.

* k-means / product quantisation (Sec. 3.3): a planted code book is found
  exactly; a run ends at a Lloyd fixed point (every code word the mean of its
  blocks, every block at its nearest word) with a non-increasing sum of
  squares; the block layout is the one the oracle decodes.
* Whitened shared basis (Appendix A.1, Eq. (4)-(6)): the fitted (D, C_e)
  reaches the Ky Fan / Eckart-Young optimum, computed here another way (a
  symmetric square root of the covariance and the singular values of the
  stacked whitened residuals, with the objective evaluated from its
  definition on the calibration rows); one matrix with an identity
  covariance reduces to the truncated SVD; a shared rank-r residual is
  recovered exactly; a perturbed basis, even with its coefficients
  re-fitted, does worse; the coefficients are the weighted least-squares
  solution for their basis.
* The down side's output-basis counterpart obeys the same optimum.
* Route-aware weights equal those computed from the oracle's routing.
* A fitted layer is never worse than its VQ part on the calibration rows,
  and the low-rank term recovers a planted shared subspace.
"""

import numpy as np
import pytest
import scipy.linalg

import oracle.cardan_oracle as O
from paper_2609_21137_amd import fit, synth


def _spd(H, N, seed):
    """Calibration rows with a non-trivial covariance, and that covariance."""
    rng = np.random.default_rng(seed)
    mix = rng.standard_normal((H, H)) / np.sqrt(H) + np.diag(np.linspace(0.5, 2.0, H))
    X = rng.standard_normal((N, H)) @ mix
    return X, X.T @ X / N


def _objective(residuals, weights, D, C, X):
    """Eq. (4) from its definition: sum_m w_m mean_t ||(Delta_m - D C_m)^T h_t||^2."""
    return sum(w * np.mean(np.sum((X @ (R - D @ c)) ** 2, axis=1))
               for R, w, c in zip(residuals, weights, C))


def _ky_fan_optimum(residuals, weights, Sigma, r):
    """Trailing energy of the stacked whitened residuals, via a symmetric
    square root and the singular values (not Cholesky, not eigh)."""
    S_half = np.real(scipy.linalg.sqrtm(Sigma))
    M = np.hstack([np.sqrt(w) * (S_half @ R) for R, w in zip(residuals, weights)])
    s = np.linalg.svd(M, compute_uv=False)
    return float(np.sum(s[r:] ** 2)), S_half


# --------------------------------------------------------------------------
# k-means / product quantisation
# --------------------------------------------------------------------------
def test_kmeans_recovers_planted_codebook():
    rng = np.random.default_rng(1)
    K, d = 12, 4
    words = rng.standard_normal((K, d)) * 3.0
    labels = np.concatenate([np.arange(K), rng.integers(0, K, 500)])
    X = words[labels]
    C, assign, hist = fit.kmeans(X, K, iters=50, seed=3)
    # zero up to the rounding of the expanded distance |x|^2 - 2 x.c + |c|^2
    assert hist[-1] <= 1e-12 * np.sum(X ** 2)
    # the same set of words, and every block labelled with its own word
    match = [int(np.argmin(np.sum((C - w) ** 2, axis=1))) for w in words]
    assert sorted(match) == list(range(K))
    assert np.allclose(C[match], words, atol=1e-12)
    assert np.array_equal(np.asarray(match)[labels], assign)


def test_kmeans_ends_at_a_lloyd_fixed_point():
    rng = np.random.default_rng(2)
    X = rng.standard_normal((600, 3))
    K = 9
    C, assign, hist = fit.kmeans(X, K, iters=200, seed=5)
    assert all(b <= a * (1 + 1e-12) for a, b in zip(hist, hist[1:]))
    for j in range(K):
        members = X[assign == j]
        assert len(members) > 0
        assert np.allclose(C[j], members.mean(axis=0), atol=1e-12)
    for n in range(0, 600, 7):  # brute-force nearest word
        dist = [float(np.sum((X[n] - C[j]) ** 2)) for j in range(K)]
        assert dist[assign[n]] <= min(dist) + 1e-12


def test_pq_layout_is_the_decoded_layout():
    """pq_init on matrices built from bf16 code words: the codes decode (by the
    oracle's Q_B(J)) back to the matrices exactly."""
    rng = np.random.default_rng(3)
    E, n_in, n_out, d, K = 3, 16, 10, 4, 8
    cb_bits = synth.to_bf16_bits(rng.standard_normal((K, d)))
    J = rng.integers(0, K, size=(E, n_in // d, n_out))
    J[0, 0, :K] = np.arange(K)  # every word used
    W = np.stack([O.decode_vq(J[e], cb_bits, d) for e in range(E)])
    C, codes, _ = fit.pq_init(W, d, K, iters=50, seed=1)
    for e in range(E):
        assert np.array_equal(O.decode_vq(codes[e], synth.to_bf16_bits(C), d), W[e])
    assert np.array_equal(fit.decode(codes, C, d), W)


# --------------------------------------------------------------------------
# the whitened shared basis, Eq. (4)-(6)
# --------------------------------------------------------------------------
def _residuals(E, H, n, seed):
    rng = np.random.default_rng(seed)
    return [rng.standard_normal((H, n)) for _ in range(E)], rng.uniform(0.2, 2.0, E)


def test_shared_rank_r_residual_is_recovered_exactly():
    rng = np.random.default_rng(4)
    H, n, E, r = 24, 10, 5, 3
    D0 = rng.standard_normal((H, r))
    res = [D0 @ rng.standard_normal((r, n)) for _ in range(E)]
    X, Sigma = _spd(H, 400, 4)
    D, C, lam = fit.input_basis_fit(res, np.ones(E), Sigma, r)
    assert _objective(res, np.ones(E), D, C, X) <= 1e-20 * sum(np.sum(R ** 2) for R in res)
    assert lam[r] <= 1e-10 * lam[0]


def test_one_matrix_with_identity_covariance_is_the_truncated_svd():
    rng = np.random.default_rng(5)
    H, n, r = 20, 14, 4
    R = rng.standard_normal((H, n))
    D, C, _ = fit.input_basis_fit([R], [1.0], np.eye(H), r)
    s = np.linalg.svd(R, compute_uv=False)
    err = np.sum((R - D @ C[0]) ** 2)
    assert abs(err - np.sum(s[r:] ** 2)) <= 1e-10 * np.sum(s ** 2)


@pytest.mark.parametrize("r", [1, 4, 9])
def test_fitted_basis_attains_the_ky_fan_optimum(r):
    H, n, E = 18, 7, 6
    res, w = _residuals(E, H, n, 6 + r)
    X, Sigma = _spd(H, 500, 6)
    D, C, _ = fit.input_basis_fit(res, w, Sigma, r)
    best, _ = _ky_fan_optimum(res, w, Sigma, r)
    got = _objective(res, w, D, C, X)
    assert abs(got - best) <= 1e-9 * best, (got, best)


def test_perturbed_basis_does_worse():
    H, n, E, r = 18, 7, 6, 4
    res, w = _residuals(E, H, n, 7)
    X, Sigma = _spd(H, 500, 7)
    D, C, _ = fit.input_basis_fit(res, w, Sigma, r)
    best, S_half = _ky_fan_optimum(res, w, Sigma, r)
    rng = np.random.default_rng(8)
    for eps in (1e-3, 1e-1, 1.0):
        Dp = D + eps * rng.standard_normal(D.shape) * np.abs(D).mean()
        # coefficients re-fitted by least squares in whitened coordinates
        Cp = [np.linalg.lstsq(S_half @ Dp, S_half @ R, rcond=None)[0] for R in res]
        assert _objective(res, w, Dp, Cp, X) > best * (1 + 1e-9), eps
    # the fitted coefficients with a perturbed basis, also worse
    Dp = D + 1e-2 * rng.standard_normal(D.shape)
    assert _objective(res, w, Dp, C, X) > best * (1 + 1e-9)


def test_coefficients_are_the_weighted_least_squares_solution():
    H, n, E, r = 16, 9, 4, 5
    res, w = _residuals(E, H, n, 9)
    _, Sigma = _spd(H, 300, 9)
    D, C, _ = fit.input_basis_fit(res, w, Sigma, r)
    S_half = np.real(scipy.linalg.sqrtm(Sigma))
    for R, c in zip(res, C):
        ref = np.linalg.lstsq(S_half @ D, S_half @ R, rcond=None)[0]
        assert np.allclose(c, ref, rtol=1e-9, atol=1e-9 * np.abs(ref).max())


def test_output_basis_attains_its_optimum():
    """Down side: min sum_e w_e ||S_e^{1/2} (Delta_e - A_e B)||^2 over a shared
    row basis; optimum = trailing energy of the stacked [sqrt(w_e) S_e^{1/2}
    Delta_e] rows (singular values), and a perturbed B does worse."""
    rng = np.random.default_rng(10)
    n_in, H, E, r = 9, 15, 5, 4
    res = [rng.standard_normal((n_in, H)) for _ in range(E)]
    w = rng.uniform(0.5, 1.5, E)
    S = [_spd(n_in, 200, 20 + e)[1] for e in range(E)]
    B, A, _ = fit.output_basis_fit(res, w, S, r)
    halves = [np.real(scipy.linalg.sqrtm(Se)) for Se in S]
    M = np.vstack([np.sqrt(we) * (Sh @ R) for R, we, Sh in zip(res, w, halves)])
    s = np.linalg.svd(M, compute_uv=False)
    best = float(np.sum(s[r:] ** 2))

    def obj(Bm, Am):
        return sum(we * np.sum((Sh @ (R - a @ Bm)) ** 2) for R, we, Sh, a in zip(res, w, halves, Am))

    assert abs(obj(B, A) - best) <= 1e-9 * best
    Bp = B + 0.05 * rng.standard_normal(B.shape)
    Ap = [np.linalg.lstsq(Bp.T, R.T, rcond=None)[0].T for R in res]
    assert obj(Bp, Ap) > best * (1 + 1e-9)


def test_route_weights_match_the_oracle_routing():
    H, E, k, N = 32, 10, 3, 200
    L = synth.make_layer(H, 16, E, 4, 8, 0, seed=11, hot_experts=(2,), hot_bias=3.0)
    x = synth.make_input(H, N, seed=11)
    idx, a, _, _ = O.route(x, L["router_w"], L["router_bias"], k)
    ref = np.zeros(E)
    for t in range(N):
        for j in range(k):
            ref[idx[t, j]] += a[t, j] ** 2
    ref /= N
    got = fit.route_weights(x, L["router_w"], L["router_bias"], k, E)
    assert np.allclose(got, ref, rtol=1e-12, atol=1e-15)
    assert got[2] == got.max()  # the hot expert


# --------------------------------------------------------------------------
# the whole layer
# --------------------------------------------------------------------------
def _teacher(H, I, E, d, K, r_true, seed, noise=0.002):
    """Dense expert weights = a VQ part on a shared code book + a low-rank
    part on a shared subspace (one for gate and up, one output-side for
    down) + noise."""
    rng = np.random.default_rng(seed)
    out = {}
    Ds = rng.standard_normal((H, r_true)) / np.sqrt(H)  # one input-side subspace for gate and up
    for name, (n_in, n_out) in (("W_gate", (H, I)), ("W_up", (H, I)), ("W_down", (I, H))):
        cb = rng.standard_normal((K, d)) * 0.3  # well-separated words: the VQ part is found
        J = rng.integers(0, K, size=(E, n_in // d, n_out))
        Q = fit.decode(J, cb, d)
        if name == "W_down":
            Bs = rng.standard_normal((r_true, n_out)) / np.sqrt(n_out)
            low = np.stack([rng.standard_normal((n_in, r_true)) * 0.05 @ Bs for _ in range(E)])
        else:
            low = np.stack([Ds @ rng.standard_normal((r_true, n_out)) * 0.05 for _ in range(E)])
        out[name] = Q + low + noise * rng.standard_normal(Q.shape)
    return out


@pytest.mark.parametrize("act", ["silu_glu", "relu2_up"])
def test_fitted_layer_is_never_worse_than_its_vq_part(act):
    H, I, E, k, d, K, r = 64, 32, 6, 2, 4, 16, 8
    T = _teacher(H, I, E, d, K, r, 12)
    L = synth.make_layer(H, I, E, d, K, 0, seed=12)
    X = synth.make_input(H, 400, seed=12)
    for route_aware in (False, True):
        layer, rep = fit.fit_layer(T, L["router_w"], L["router_bias"], X, k, d, K, r, act=act,
                                   route_aware=route_aware, seed=1)
        assert rep.nmse_vq_lr <= rep.nmse_vq
        assert rep.nmse_down_vq_lr <= rep.nmse_down_vq
        # the planted shared subspace: the low rank term removes most of the
        # post-VQ error of the input-side projections
        assert rep.nmse_vq_lr < 0.5 * rep.nmse_vq, (rep.nmse_vq, rep.nmse_vq_lr)
        if act == "relu2_up":
            assert layer["codes_gate"] is None and layer["U_gate"] is None


def test_fitted_layer_through_the_oracle_tracks_the_teacher():
    """The fitted layer in storage formats (bf16 factors, uint8 codes), run by
    the oracle, is closer to the dense teacher on held-out tokens than the
    VQ-only layer."""
    H, I, E, k, d, K, r = 64, 32, 6, 2, 4, 16, 8
    T = _teacher(H, I, E, d, K, r, 13)
    L = synth.make_layer(H, I, E, d, K, 0, seed=13)
    X = synth.make_input(H, 400, seed=13)
    x_test = synth.make_input(H, 16, seed=13, step=1)
    Tb = {n: synth.to_bf16_bits(v) for n, v in T.items()}
    y_t, idx_t, _, _ = O.moe_layer_dense(x_test, L["router_w"], L["router_bias"], Tb["W_gate"], Tb["W_up"],
                                         Tb["W_down"], k)
    lr_layer, _ = fit.fit_layer(T, L["router_w"], L["router_bias"], X, k, d, K, r, seed=2)
    vq_layer, _ = fit.fit_layer(T, L["router_w"], L["router_bias"], X, k, d, K, 0, seed=2)
    y_lr, idx_lr, _, _ = O.moe_layer_factored(x_test, lr_layer, k, d)
    y_vq, _, _, _ = O.moe_layer_factored(x_test, vq_layer, k, d)
    assert np.array_equal(idx_lr, idx_t)  # the router is the teacher's
    e_lr = np.sum((y_lr - y_t) ** 2) / np.sum(y_t ** 2)
    e_vq = np.sum((y_vq - y_t) ** 2) / np.sum(y_t ** 2)
    assert e_lr < 0.5 * e_vq, (e_lr, e_vq)
