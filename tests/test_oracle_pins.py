"""Pins for the fp64 oracle, each against something other than the oracle itself.

Citations are to the CacheBridge paper.  What pins what:

* bf16 rounding      -- torch's float32->bfloat16 conversion (round to nearest even),
                        hand-built ties, and doubles that sit just off a tie.
* moments G, C        -- Sec. 3.4 Eq. fusedstats in augmented form: numpy matrix
                        products for w == 1 and for general w, exact integer
                        brute force, closed-form last row/column (sum w, sum w x,
                        sum w y), symmetry, PSD, scaling, additivity over
                        sequence splits, token-permutation invariance, and the
                        head-local gather of Sec. 3.2 Eq. localfeature.
* ridge solve         -- Sec. 3.1 Eq. closedform (centered weighted ridge,
                        computed here from X, Y, w by numpy), brute-force
                        minimality of the penalized objective, weighted least
                        squares as lambda -> 0, lambda -> infinity asymptotics,
                        exact planted-map recovery, d_eff <= P (Sec. 2.2 Eq.
                        ridge-effective-dimension), scipy's dense solve, and the
                        non-positive-definite report.
* application         -- identity map copies bits, a pure bias gives RNE(b),
                        a cyclic head assignment permutes outputs (Sec. 4.3),
                        numpy fp64 products.
* coefficient counts  -- numbers printed in the paper (tests/golden/paper_values.json).
"""
import json
import os

import numpy as np
import pytest
import scipy.linalg
import torch

import oracle
import synth

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "paper_values.json")


# ----------------------------------------------------------------------------- helpers

def to_bf16_bits(a) -> np.ndarray:
    t = torch.as_tensor(np.asarray(a, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


def bf16_val(bits) -> np.ndarray:
    return oracle.bf16_to_double(bits)


class Problem:
    """Small explicit problem in the canonical [layer][kv][seq][head][tok][dim] layout."""

    def __init__(self, rng, L_s=2, H_s=3, d_s=8, L_t=2, H_t=2, d_t=5, B=3, T=17,
                 hm=None, values="gauss", wkind="lognormal"):
        self.L_s, self.H_s, self.d_s, self.L_t, self.H_t, self.d_t, self.B, self.T = \
            L_s, H_s, d_s, L_t, H_t, d_t, B, T
        if values == "gauss":
            xs = rng.standard_normal((L_s, 2, B, H_s, T, d_s)) * (1 + np.arange(H_s))[None, None, None, :, None, None]
            ys = rng.standard_normal((L_t, 2, B, H_t, T, d_t)) + 3.0
        else:  # small integers, exact in bf16 and in every fp64 sum
            xs = rng.integers(-4, 5, size=(L_s, 2, B, H_s, T, d_s))
            ys = rng.integers(-4, 5, size=(L_t, 2, B, H_t, T, d_t))
        self.src = to_bf16_bits(xs)
        self.tgt = to_bf16_bits(ys)
        self.X = bf16_val(self.src)
        self.Y = bf16_val(self.tgt)
        if hm is None:
            hm = {"tgt_layer": [], "tgt_head": [], "kv": [], "src_layer": [], "src_head": [], "weight_row": []}
            for l in range(L_t):
                for z in range(2):
                    for h in range(H_t):
                        hm["tgt_layer"].append(l)
                        hm["tgt_head"].append(h)
                        hm["kv"].append(z)
                        hm["src_layer"].append((l + 1) % L_s)
                        hm["src_head"].append((2 * h + 1) % H_s)
                        hm["weight_row"].append(l * H_t + h)
            hm = {k: np.asarray(v, np.int32) for k, v in hm.items()}
        self.hm = hm
        R = int(hm["weight_row"].max()) + 1
        if wkind == "lognormal":
            w = np.exp(rng.standard_normal((R, B * T)))
        elif wkind == "ones":
            w = np.ones((R, B * T))
        else:
            w = rng.choice([0.0, 0.5, 1.0, 2.0, 0.25], size=(R, B * T))
        self.w = w.astype(np.float32)
        self.src_strides = synth.cache_strides(L_s, H_s, B, T, d_s)
        self.tgt_strides = synth.cache_strides(L_t, H_t, B, T, d_t)

    @property
    def n_maps(self):
        return self.hm["kv"].shape[0]

    def stats(self, w=None, src=None):
        return oracle.stats(self.hm, self.src if src is None else src, self.src_strides, self.d_s,
                            self.tgt, self.tgt_strides, self.d_t, self.w if w is None else w,
                            self.B * self.T, self.B, self.T)

    def design(self, m):
        """X~ (n x P), Y (n x d_t), w (n) of map m, gathered with numpy indexing."""
        hm = self.hm
        x = self.X[hm["src_layer"][m], hm["kv"][m], :, hm["src_head"][m]].reshape(-1, self.d_s)
        y = self.Y[hm["tgt_layer"][m], hm["kv"][m], :, hm["tgt_head"][m]].reshape(-1, self.d_t)
        w = self.w[hm["weight_row"][m]].astype(np.float64)
        xt = np.concatenate([x, np.ones((x.shape[0], 1))], axis=1)
        return xt, y, w


def relF(a, b):
    return np.linalg.norm(np.asarray(a) - np.asarray(b)) / max(np.linalg.norm(np.asarray(b)), 1e-300)


# ----------------------------------------------------------------------------- bf16 rounding

def test_bf16_rne_matches_torch_on_float32_values():
    rng = np.random.default_rng(1)
    mags = np.concatenate([rng.standard_normal(20000) * 10.0 ** rng.integers(-40, 38, 20000),
                           rng.standard_normal(2000) * 1e-39,          # bf16 subnormal range
                           np.array([0.0, -0.0, 3.3895314e38, -3.3895314e38, 1.0, -2.0])])
    f32 = mags.astype(np.float32)
    f32 = f32[np.isfinite(f32)]
    ours = oracle.double_to_bf16(f32.astype(np.float64))
    ref = to_bf16_bits(f32)
    assert np.array_equal(ours, ref)


def test_bf16_rne_ties_and_double_rounding():
    # 1 + 2^-8 is exactly halfway between 1 and 1 + 2^-7: ties go to the even (1.0).
    assert oracle.double_to_bf16(1.0 + 2.0 ** -8)[()] == 0x3F80
    # 1 + 3*2^-8 is halfway between 1+2^-7 (odd) and 1+2^-6 (even): rounds up.
    assert oracle.double_to_bf16(1.0 + 3 * 2.0 ** -8)[()] == 0x3F82
    # Just above the tie (not representable in float32): must round up, which a
    # detour through float32 (that would land on the tie) gets wrong.
    assert oracle.double_to_bf16(1.0 + 2.0 ** -8 + 2.0 ** -40)[()] == 0x3F81
    assert oracle.double_to_bf16(-(1.0 + 2.0 ** -8 + 2.0 ** -40))[()] == 0xBF81
    # Overflow past the largest finite bf16 -> inf; NaN stays NaN.
    assert oracle.double_to_bf16(3.4e38)[()] == 0x7F80
    assert (oracle.double_to_bf16(float("nan"))[()] & 0x7FC0) == 0x7FC0


# ----------------------------------------------------------------------------- moments

def test_stats_unit_weights_equal_plain_gram():
    p = Problem(np.random.default_rng(2), wkind="ones")
    G, C = p.stats()
    for m in range(p.n_maps):
        xt, y, _ = p.design(m)
        np.testing.assert_allclose(G[m], xt.T @ xt, rtol=1e-12, atol=1e-9)
        np.testing.assert_allclose(C[m], xt.T @ y, rtol=1e-12, atol=1e-9)


def test_stats_weighted_equal_matrix_form_and_closed_form_entries():
    p = Problem(np.random.default_rng(3))
    G, C = p.stats()
    P = p.d_s + 1
    for m in range(p.n_maps):
        xt, y, w = p.design(m)
        np.testing.assert_allclose(G[m], (xt * w[:, None]).T @ xt, rtol=1e-12, atol=1e-9)
        np.testing.assert_allclose(C[m], (xt * w[:, None]).T @ y, rtol=1e-12, atol=1e-9)
        # last row / column: sum w, sum w x, sum w y
        np.testing.assert_allclose(G[m][P - 1, P - 1], w.sum(), rtol=1e-13)
        np.testing.assert_allclose(G[m][: P - 1, P - 1], (w[:, None] * xt[:, :-1]).sum(0), rtol=1e-12, atol=1e-10)
        np.testing.assert_allclose(G[m][P - 1, : P - 1], (w[:, None] * xt[:, :-1]).sum(0), rtol=1e-12, atol=1e-10)
        np.testing.assert_allclose(C[m][P - 1], (w[:, None] * y).sum(0), rtol=1e-12, atol=1e-10)


def test_stats_exact_integer_brute_force():
    rng = np.random.default_rng(4)
    p = Problem(rng, d_s=4, d_t=3, B=2, T=5, values="int", wkind="dyadic")
    G, C = p.stats()
    for m in range(p.n_maps):
        xt, y, w = p.design(m)
        n = xt.shape[0]
        # exact rational arithmetic: every value is a small integer or dyadic
        for i in range(p.d_s + 1):
            for j in range(p.d_s + 1):
                exact = sum(float(w[t]) * int(xt[t, i]) * int(xt[t, j]) for t in range(n))
                assert G[m][i, j] == exact
            for j in range(p.d_t):
                exact = sum(float(w[t]) * int(xt[t, i]) * int(y[t, j]) for t in range(n))
                assert C[m][i, j] == exact


def test_stats_symmetric_psd_and_scaling():
    p = Problem(np.random.default_rng(5))
    G, C = p.stats()
    for m in range(p.n_maps):
        np.testing.assert_allclose(G[m], G[m].T, rtol=1e-14, atol=1e-12)
        ev = np.linalg.eigvalsh(0.5 * (G[m] + G[m].T))
        assert ev.min() >= -1e-12 * np.trace(G[m])
    G4, C4 = p.stats(w=p.w * 4.0)           # power of two: exact
    assert np.array_equal(G4, 4.0 * G) and np.array_equal(C4, 4.0 * C)
    G3, C3 = p.stats(w=(p.w.astype(np.float64) * 3.0).astype(np.float32))
    assert relF(G3, 3.0 * G) < 1e-6 and relF(C3, 3.0 * C) < 1e-6


def test_stats_additive_over_sequence_splits_and_accumulates():
    p = Problem(np.random.default_rng(6), B=4)
    G, C = p.stats()
    half = 2
    s = np.asarray(p.src_strides)
    t = np.asarray(p.tgt_strides)
    # The same buffers viewed from sequence 2 on: offset pointers, same strides.
    src_b = p.src.reshape(-1)[half * s[2]:]
    tgt_b = p.tgt.reshape(-1)[half * t[2]:]
    w_a = np.ascontiguousarray(p.w[:, : half * p.T])
    w_b = np.ascontiguousarray(p.w[:, half * p.T:])
    Ga, Ca = oracle.stats(p.hm, p.src, p.src_strides, p.d_s, p.tgt, p.tgt_strides, p.d_t,
                          w_a, half * p.T, half, p.T)
    Gab, Cab = oracle.stats(p.hm, src_b, p.src_strides, p.d_s, tgt_b, p.tgt_strides, p.d_t,
                            w_b, (p.B - half) * p.T, p.B - half, p.T, G=Ga.copy(), C=Ca.copy())
    np.testing.assert_allclose(Gab, G, rtol=1e-12, atol=1e-9)
    np.testing.assert_allclose(Cab, C, rtol=1e-12, atol=1e-9)


def test_stats_token_permutation_invariance():
    rng = np.random.default_rng(7)
    p = Problem(rng, B=1, T=40)
    G, C = p.stats()
    perm = rng.permutation(p.T)
    src = p.src.copy()
    tgt = p.tgt.copy()
    src[:, :, :, :, :, :] = p.src[:, :, :, :, perm, :]
    tgt[:, :, :, :, :, :] = p.tgt[:, :, :, :, perm, :]
    w = p.w[:, perm]
    Gp, Cp = oracle.stats(p.hm, src, p.src_strides, p.d_s, tgt, p.tgt_strides, p.d_t, w, p.T, 1, p.T)
    np.testing.assert_allclose(Gp, G, rtol=1e-12, atol=1e-9)
    np.testing.assert_allclose(Cp, C, rtol=1e-12, atol=1e-9)


def test_stats_head_local_gather_selects_the_mapped_source_head():
    # Each source head has a very different scale, so reading a wrong head or
    # layer changes G by orders of magnitude (Sec. 3.2 Eq. localfeature).
    p = Problem(np.random.default_rng(8), L_s=3, H_s=4, L_t=3, H_t=2)
    G, _ = p.stats()
    for m in range(p.n_maps):
        xt, _, w = p.design(m)
        ref = (xt * w[:, None]).T @ xt
        np.testing.assert_allclose(G[m], ref, rtol=1e-12, atol=1e-9)
        for other in range(p.H_s):
            if other != p.hm["src_head"][m]:
                xo = p.X[p.hm["src_layer"][m], p.hm["kv"][m], :, other].reshape(-1, p.d_s)
                assert abs(np.trace(G[m][:-1, :-1]) - (w[:, None] * xo * xo).sum()) > 1e-3 * np.trace(G[m])


# ----------------------------------------------------------------------------- ridge solve

def centered_closed_form(xt, y, w, lam):
    """Sec. 3.1 Eq. closedform written from X, Y, w (weights rescaled to mean one)."""
    n = xt.shape[0]
    w = w * (n / w.sum())
    x = xt[:, :-1]
    xbar = (w[:, None] * x).sum(0) / n
    ybar = (w[:, None] * y).sum(0) / n
    xc, yc = x - xbar, y - ybar
    Wh = np.linalg.solve((xc * w[:, None]).T @ xc + lam * np.eye(x.shape[1]), (xc * w[:, None]).T @ yc)
    bh = ybar - xbar @ Wh
    return Wh, bh


def test_solve_bias_unpenalized_equals_paper_centered_ridge():
    rng = np.random.default_rng(9)
    p = Problem(rng, B=4, T=50)
    # rescale weights to mean one per map row, as the paper assumes
    p.w = (p.w / p.w.mean(axis=1, keepdims=True)).astype(np.float32)
    G, C = p.stats()
    lam = 0.37
    W, info = oracle.ridge_solve(G, C, lam, relative=False, bias_unpenalized=True)
    assert (info == 0).all()
    for m in range(p.n_maps):
        xt, y, w = p.design(m)
        Wh, bh = centered_closed_form(xt, y, w, lam)
        # the paper's centering uses n^-1 sum w x, equal to the true weighted
        # mean only up to the float32 mean-one rescaling; compare at 1e-6
        np.testing.assert_allclose(W[m][:-1], Wh, rtol=1e-6, atol=1e-8)
        np.testing.assert_allclose(W[m][-1], bh, rtol=1e-6, atol=1e-8)


# ----------------------------------------------------------------------------- two-pass centered path

def _centered(p, w=None):
    return oracle.stats_centered(p.hm, p.src, p.src_strides, p.d_s, p.tgt, p.tgt_strides, p.d_t,
                                 p.w if w is None else w, p.B * p.T, p.B, p.T)


def test_centered_moments_equal_numpy_weighted_covariances():
    rng = np.random.default_rng(21)
    p = Problem(rng, B=3, T=40)
    sums, A, B = _centered(p)
    for m in range(p.n_maps):
        xt, y, w = p.design(m)
        x = xt[:, :-1]
        assert sums[m, 0] == pytest.approx(w.sum(), rel=1e-14)
        np.testing.assert_allclose(sums[m, 1:1 + p.d_s], w @ x, rtol=1e-12, atol=1e-12)
        np.testing.assert_allclose(sums[m, 1 + p.d_s:], w @ y, rtol=1e-12, atol=1e-12)
        # numpy's weighted covariance (a library routine), rescaled from mean to sum
        cov = np.cov(np.concatenate([x, y], axis=1).T, aweights=w, bias=True) * w.sum()
        np.testing.assert_allclose(A[m], cov[:p.d_s, :p.d_s], rtol=1e-10, atol=1e-10)
        np.testing.assert_allclose(B[m], cov[:p.d_s, p.d_s:], rtol=1e-10, atol=1e-10)


def test_centered_moments_shift_invariant_exactly():
    # integer data: every sum is exact, so shifting every source row by a
    # constant vector (and the target rows by another) leaves A and B unchanged
    rng = np.random.default_rng(22)
    p = Problem(rng, values="int", wkind="choice", B=2, T=20)
    sums0, A0, B0 = _centered(p)
    shift_x = rng.integers(-8, 9, size=p.d_s)
    shift_y = rng.integers(-8, 9, size=p.d_t)
    p2 = Problem(np.random.default_rng(22), values="int", wkind="choice", B=2, T=20)
    p2.src = to_bf16_bits(bf16_val(p.src) + shift_x)
    p2.tgt = to_bf16_bits(bf16_val(p.tgt) + shift_y)
    sums1, A1, B1 = _centered(p2)
    # the means move by the shifts (where weights are nonzero), the moments not at all
    ok = sums0[:, 0] != 0
    np.testing.assert_allclose(A1[ok], A0[ok], rtol=1e-12, atol=1e-9)
    np.testing.assert_allclose(B1[ok], B0[ok], rtol=1e-12, atol=1e-9)


def test_centered_ridge_equals_unpenalized_augmented_ridge():
    # Schur complement on the bias row: the paper's centered ridge with the
    # trace-of-augmented-moments lambda is the unpenalized augmented solution
    rng = np.random.default_rng(23)
    p = Problem(rng, B=3, T=45)
    G, C = p.stats()
    sums, A, B = _centered(p)
    for relative, lam in ((True, 1e-2), (False, 0.3)):
        Wa, ia = oracle.ridge_solve(G, C, lam, relative=relative, bias_unpenalized=True)
        Wc, ic = oracle.ridge_solve_centered(sums, A, B, lam, relative=relative)
        assert (ia == 0).all() and (ic == 0).all()
        assert relF(Wc, Wa) < 1e-10


def test_centered_ridge_matches_closed_form_and_handles_zero_weights():
    rng = np.random.default_rng(24)
    p = Problem(rng, B=2, T=60)
    sums, A, B = _centered(p)
    lam = 0.21
    W, info = oracle.ridge_solve_centered(sums, A, B, lam, relative=False)
    for m in range(p.n_maps):
        xt, y, w = p.design(m)
        # Eq. closedform with the raw weights (absolute lambda, no mean-one rescaling)
        x = xt[:, :-1]
        xbar, ybar = (w @ x) / w.sum(), (w @ y) / w.sum()
        xc, yc = x - xbar, y - ybar
        Wh = np.linalg.solve((xc * w[:, None]).T @ xc + lam * np.eye(p.d_s), (xc * w[:, None]).T @ yc)
        bh = ybar - xbar @ Wh
        np.testing.assert_allclose(W[m][:-1], Wh, rtol=1e-8, atol=1e-10)
        np.testing.assert_allclose(W[m][-1], bh, rtol=1e-8, atol=1e-10)
    # all-zero weights: zero means and moments; relative lambda is zero too,
    # so the first pivot fails and the maps are zero
    z = np.zeros_like(p.w)
    sz, Az, Bz = _centered(p, w=z)
    assert not sz.any() and not Az.any() and not Bz.any()
    Wz, iz = oracle.ridge_solve_centered(sz, Az, Bz, 1e-2, relative=True)
    assert (iz == 1).all() and not Wz.any()


def objective(Wt, xt, y, w, lam, bias_penalized):
    r = y - xt @ Wt
    pen = (Wt ** 2).sum() if bias_penalized else (Wt[:-1] ** 2).sum()
    return float((w[:, None] * r * r).sum() + lam * pen)


@pytest.mark.parametrize("unpen", [False, True])
def test_solve_is_brute_force_minimizer(unpen):
    rng = np.random.default_rng(10)
    p = Problem(rng, d_s=5, d_t=3, B=2, T=30)
    G, C = p.stats()
    lam = 2.5
    W, info = oracle.ridge_solve(G, C, lam, relative=False, bias_unpenalized=unpen)
    assert (info == 0).all()
    for m in range(p.n_maps):
        xt, y, w = p.design(m)
        j0 = objective(W[m], xt, y, w, lam, not unpen)
        for _ in range(50):
            d = rng.standard_normal(W[m].shape)
            for eps in (1e-2, 1e-4):
                assert objective(W[m] + eps * d, xt, y, w, lam, not unpen) > j0
        # first-order optimality along coordinate directions (central differences)
        h = 1e-5
        for (i, j) in [(0, 0), (p.d_s, 1), (2, 2)]:
            e = np.zeros_like(W[m])
            e[i, j] = h
            g = (objective(W[m] + e, xt, y, w, lam, not unpen) - objective(W[m] - e, xt, y, w, lam, not unpen)) / (2 * h)
            assert abs(g) <= 1e-6 * max(1.0, j0)


def test_solve_small_lambda_is_weighted_least_squares():
    rng = np.random.default_rng(11)
    p = Problem(rng, B=3, T=60)
    G, C = p.stats()
    W, info = oracle.ridge_solve(G, C, 1e-10, relative=False, bias_unpenalized=False)
    for m in range(p.n_maps):
        xt, y, w = p.design(m)
        sw = np.sqrt(w)[:, None]
        ref = np.linalg.lstsq(sw * xt, sw * y, rcond=None)[0]
        np.testing.assert_allclose(W[m], ref, rtol=1e-7, atol=1e-8)


def test_solve_matches_dense_library_solve_and_relative_lambda():
    rng = np.random.default_rng(12)
    p = Problem(rng)
    G, C = p.stats()
    P = p.d_s + 1
    for unpen in (False, True):
        W, info = oracle.ridge_solve(G, C, 1e-2, relative=True, bias_unpenalized=unpen)
        for m in range(p.n_maps):
            lam = 1e-2 * np.trace(G[m]) / P
            D = np.eye(P)
            if unpen:
                D[-1, -1] = 0.0
            ref = scipy.linalg.solve(G[m] + lam * D, C[m], assume_a="pos")
            np.testing.assert_allclose(W[m], ref, rtol=1e-10, atol=1e-12)
    # relative lambda makes the maps invariant to a rescaling of the weights
    G7, C7 = p.stats(w=(p.w.astype(np.float64) * 7.0).astype(np.float32))
    W1, _ = oracle.ridge_solve(G, C, 1e-2, relative=True)
    W7, _ = oracle.ridge_solve(G7, C7, 1e-2, relative=True)
    np.testing.assert_allclose(W7, W1, rtol=1e-5, atol=1e-7)


def test_solve_recovers_planted_map_exactly():
    rng = np.random.default_rng(13)
    d_s, d_t, n = 6, 4, 400
    Wstar = rng.choice([-1.0, -0.5, 0.0, 0.5, 1.0, 2.0], size=(d_s + 1, d_t))
    x = rng.integers(-6, 7, size=(n, d_s)).astype(np.float64)
    y = np.concatenate([x, np.ones((n, 1))], 1) @ Wstar          # small dyadics: exact in bf16
    assert np.array_equal(bf16_val(to_bf16_bits(y)), y)
    hm = {k: np.zeros(1, np.int32) for k in oracle.HEAD_MAP_FIELDS}
    src = to_bf16_bits(x.reshape(1, 1, 1, 1, n, d_s))
    tgt = to_bf16_bits(y.reshape(1, 1, 1, 1, n, d_t))
    w = np.exp(rng.standard_normal((1, n))).astype(np.float32)
    G, C = oracle.stats(hm, src, synth.cache_strides(1, 1, 1, n, d_s), d_s, tgt,
                        synth.cache_strides(1, 1, 1, n, d_t), d_t, w, n, 1, n)
    for unpen in (False, True):
        W, info = oracle.ridge_solve(G, C, 1e-13, relative=True, bias_unpenalized=unpen)
        assert info[0] == 0
        np.testing.assert_allclose(W[0], Wstar, rtol=0, atol=1e-8)


def test_solve_large_lambda_and_effective_dof():
    rng = np.random.default_rng(14)
    p = Problem(rng)
    G, C = p.stats()
    P = p.d_s + 1
    lam = 1e9 * np.abs(G).max()
    W, _ = oracle.ridge_solve(G, C, lam, relative=False, bias_unpenalized=False)
    for m in range(p.n_maps):
        assert relF(lam * W[m], C[m]) < 1e-6
    # d_eff = tr[G (G + lam I)^-1] <= P  (solve with right-hand side G)
    for lr in (1e-4, 1e-2, 1.0):
        R, info = oracle.ridge_solve(G, G, lr, relative=True)
        for m in range(p.n_maps):
            d_eff = np.trace(R[m])
            assert 0 < d_eff <= P + 1e-9
            ev = np.linalg.eigvalsh(G[m])
            lam_m = lr * np.trace(G[m]) / P
            np.testing.assert_allclose(d_eff, (ev / (ev + lam_m)).sum(), rtol=1e-9)


def test_solve_reports_non_positive_definite():
    P, d_t = 5, 3
    G = np.zeros((2, P, P))
    C = np.zeros((2, P, d_t))
    G[1] = np.eye(P)
    G[1][2, 2] = -5.0                     # indefinite even after the ridge term
    C[1] = 1.0
    W, info = oracle.ridge_solve(G, C, 1e-2, relative=True)
    assert info[0] == 1                    # all-zero weights: G = 0 and lambda = 0
    assert info[1] == 3
    assert not W.any()


# ----------------------------------------------------------------------------- application

def apply_problem(rng, d_s=8, d_t=8, hm_kind="identity"):
    wl = synth.Workload("pin", 2, 4, d_s, 3, 4, d_t, 2, 11, hm_kind, "gauss", 0.1, "lognormal")
    hm = synth.head_map(wl)
    xs = rng.standard_normal((wl.L_s, 2, wl.n_seqs, wl.H_s, wl.seq_len, d_s)) * 3
    src = to_bf16_bits(xs)
    out = np.zeros((wl.L_t, 2, wl.n_seqs, wl.H_t, wl.seq_len, d_t), dtype=np.uint16)
    return wl, hm, src, out


def test_apply_identity_map_copies_bits():
    rng = np.random.default_rng(15)
    wl, hm, src, out = apply_problem(rng)
    n = hm["kv"].shape[0]
    W = np.zeros((n, wl.P, wl.d_t))
    W[:, : wl.d_s, :] = np.eye(wl.d_s)
    wl = wl.with_(head_map_kind="qwen")
    hm = synth.head_map(wl)
    oracle.apply(hm, W, src, synth.cache_strides(wl.L_s, wl.H_s, wl.n_seqs, wl.seq_len, wl.d_s), wl.d_s,
                 out, synth.cache_strides(wl.L_t, wl.H_t, wl.n_seqs, wl.seq_len, wl.d_t), wl.d_t,
                 wl.n_seqs, wl.seq_len)
    for m in range(n):
        a = out[hm["tgt_layer"][m], hm["kv"][m], :, hm["tgt_head"][m]]
        b = src[hm["src_layer"][m], hm["kv"][m], :, hm["src_head"][m]]
        assert np.array_equal(a, b)


def test_apply_pure_bias_is_rounded_bias_and_matches_fp64_products():
    rng = np.random.default_rng(16)
    wl, hm, src, out = apply_problem(rng, d_s=6, d_t=5, hm_kind="qwen")
    n = hm["kv"].shape[0]
    ss = synth.cache_strides(wl.L_s, wl.H_s, wl.n_seqs, wl.seq_len, wl.d_s)
    os_ = synth.cache_strides(wl.L_t, wl.H_t, wl.n_seqs, wl.seq_len, wl.d_t)
    W = np.zeros((n, wl.P, wl.d_t))
    bias = rng.standard_normal((n, wl.d_t)).astype(np.float32)
    W[:, -1, :] = bias
    oracle.apply(hm, W, src, ss, wl.d_s, out, os_, wl.d_t, wl.n_seqs, wl.seq_len)
    for m in range(n):
        a = out[hm["tgt_layer"][m], hm["kv"][m], :, hm["tgt_head"][m]]
        assert (a == to_bf16_bits(bias[m])[None, None, :]).all()
    # general maps against numpy fp64 products rounded by the pinned rounding
    W = rng.standard_normal((n, wl.P, wl.d_t))
    oracle.apply(hm, W, src, ss, wl.d_s, out, os_, wl.d_t, wl.n_seqs, wl.seq_len)
    X = bf16_val(src)
    for m in range(n):
        x = X[hm["src_layer"][m], hm["kv"][m], :, hm["src_head"][m]]
        xt = np.concatenate([x, np.ones(x.shape[:-1] + (1,))], -1)
        ref = oracle.double_to_bf16(xt @ W[m])
        assert np.array_equal(out[hm["tgt_layer"][m], hm["kv"][m], :, hm["tgt_head"][m]], ref)


def test_apply_cyclic_head_assignment_permutes_outputs():
    rng = np.random.default_rng(17)
    wl, _, src, out0 = apply_problem(rng, hm_kind="qwen")
    ss = synth.cache_strides(wl.L_s, wl.H_s, wl.n_seqs, wl.seq_len, wl.d_s)
    os_ = synth.cache_strides(wl.L_t, wl.H_t, wl.n_seqs, wl.seq_len, wl.d_t)
    hm0 = synth.head_map(wl)
    hm1 = synth.head_map(wl.with_(head_map_kind="cyclic1"))
    n = hm0["kv"].shape[0]
    W = rng.standard_normal((n, wl.P, wl.d_t))
    out1 = np.zeros_like(out0)
    oracle.apply(hm0, W, src, ss, wl.d_s, out0, os_, wl.d_t, wl.n_seqs, wl.seq_len)
    # shifting the source head by one with the maps moved along gives the
    # outputs of the shifted heads
    W1 = W.reshape(wl.L_t, 2, wl.H_t, wl.P, wl.d_t)
    W1 = np.roll(W1, -1, axis=2).reshape(n, wl.P, wl.d_t)
    oracle.apply(hm1, W1, src, ss, wl.d_s, out1, os_, wl.d_t, wl.n_seqs, wl.seq_len)
    assert np.array_equal(np.roll(out1, 1, axis=3)[:, :, :, :], out0)


# ----------------------------------------------------------------------------- paper values

def test_coefficient_counts_reproduce_printed_sizes():
    g = json.load(open(GOLDEN))
    q = g["qwen3_14b_to_32b"]
    local = oracle.coefficient_count(q["L_t"], q["H_t"], q["k"], 1, q["d_s"], q["d_t"])
    full = oracle.coefficient_count(q["L_t"], q["H_t"], q["k"], q["H_s"], q["d_s"], q["d_t"])
    assert local == 134_217_728
    assert full // local == q["H_s"]                      # C_full / C_local = H_s (Sec. 3.2)
    # fp32 coefficients: the printed sizes (3 decimals) are the coefficient bytes
    # plus about 1 MB of per-map vectors (2 x 128 fp32 per map)
    extra = 2 * q["L_t"] * q["H_t"] * 2 * q["d_t"] * 4
    assert round((4 * local + extra) / 1e9, 3) == q["head_local_GB"]
    assert round((4 * full + extra) / 1e9, 3) == q["full_head_GB"]
    wd = g["input_widths"]
    for k, f_w, l_w in zip(wd["k"], wd["full"], wd["local"]):
        assert oracle.coefficient_count(1, 1, k, wd["H_s"], wd["d_s"], 1) // 2 == f_w
        assert oracle.coefficient_count(1, 1, k, 1, wd["d_s"], 1) // 2 == l_w


# ----------------------------------------------------------------------------- workload generators

def test_generators_mean_one_weights_and_head_maps():
    wl = synth.WORKLOADS["qwen50"]
    hm = synth.head_map(wl)
    assert hm["kv"].shape[0] == 1024
    assert hm["src_layer"].max() == 39 and len(set(hm["src_layer"].tolist())) == 40
    wm = synth.WORKLOADS["mismatch"]
    hmm = synth.head_map(wm)
    assert hmm["kv"].shape[0] == 320 and set(hmm["src_head"].tolist()) == {0, 2, 4, 6}
    small = wl.with_(L_t=2, H_t=2, n_seqs=2, seq_len=128)
    w = synth.gen_weights(small).numpy()
    assert w.shape == (4, 256) and (w >= 0).all()
    np.testing.assert_allclose(w.reshape(4, 2, 128).mean(-1), 1.0, rtol=1e-5)
    # the sink makes position 0 the heaviest column
    assert (w.reshape(4, 2, 128)[:, :, 0] > 10).all()


# ----------------------------------------------------------------------------- layer-selection probes

def _probe_fit(p, lam=0.0):
    """Centered fit of every map of ``p`` (absolute lambda) and its oracle R^2."""
    sums, A, B = _centered(p)
    W, info = oracle.ridge_solve_centered(sums, A, B, lam, relative=False)
    assert (info == 0).all()
    r2 = oracle.probe_r2(p.hm, W, p.src, p.src_strides, p.d_s, p.tgt, p.tgt_strides, p.d_t, p.w,
                         p.B * p.T, p.B, p.T)
    return sums, A, B, W, r2


def test_weighted_squares_match_centered_moments_and_numpy_variance():
    rng = np.random.default_rng(31)
    p = Problem(rng, B=2, T=30)
    sums, A, B = _centered(p)
    sq = oracle.weighted_squares(p.hm, p.src, p.src_strides, p.d_s, p.tgt, p.tgt_strides, p.d_t, p.w,
                                 p.B * p.T, p.B, p.T)
    for m in range(p.n_maps):
        xt, y, w = p.design(m)
        S = sums[m, 0]
        mu_x = sums[m, 1:1 + p.d_s] / S
        # sum w x^2 = diag(A) + S mu^2 (A from the two-pass centered statistics)
        np.testing.assert_allclose(sq[m, :p.d_s], np.diag(A[m]) + S * mu_x ** 2, rtol=1e-11)
        # numpy's weighted variance of y (a library routine), rescaled from mean to sum
        var_y = np.cov(y.T, aweights=w, bias=True).diagonal() * w.sum()
        mu_y = sums[m, 1 + p.d_s:] / S
        np.testing.assert_allclose(sq[m, p.d_s:] - S * mu_y ** 2, var_y, rtol=1e-9)


def test_probe_r2_matches_sklearn_weighted_variance_weighted_score():
    from sklearn.metrics import r2_score
    rng = np.random.default_rng(32)
    p = Problem(rng, B=2, T=40, d_s=6, d_t=4)
    _, _, _, W, r2 = _probe_fit(p, lam=0.3)
    for m in range(p.n_maps):
        xt, y, w = p.design(m)
        pred = xt @ W[m]
        ref = r2_score(y, pred, sample_weight=w, multioutput="variance_weighted")
        assert r2[m] == pytest.approx(ref, abs=1e-12)


def test_probe_r2_scalar_ols_is_squared_weighted_correlation():
    # one source and one target channel, lambda = 0: R^2 = corr_w(x, y)^2
    rng = np.random.default_rng(33)
    p = Problem(rng, B=2, T=50, d_s=1, d_t=1)
    _, _, _, _, r2 = _probe_fit(p, lam=0.0)
    for m in range(p.n_maps):
        xt, y, w = p.design(m)
        c = np.cov(np.stack([xt[:, 0], y[:, 0]]), aweights=w)
        assert r2[m] == pytest.approx(c[0, 1] ** 2 / (c[0, 0] * c[1, 1]), rel=1e-10)


def test_probe_r2_is_one_for_an_exact_planted_map_and_zero_for_constant_targets():
    rng = np.random.default_rng(34)
    p = Problem(rng, values="int", B=2, T=60, d_s=4, d_t=3)
    # y = x M + c exactly (small integers: exact in bf16 and in every sum)
    for m in range(p.n_maps):
        hm = p.hm
        x = p.X[hm["src_layer"][m], hm["kv"][m], :, hm["src_head"][m]]
        M = rng.integers(-2, 3, size=(p.d_s, p.d_t))
        c = rng.integers(-3, 4, size=p.d_t)
        p.Y[hm["tgt_layer"][m], hm["kv"][m], :, hm["tgt_head"][m]] = x @ M + c
    p.tgt = to_bf16_bits(p.Y)
    _, _, _, _, r2 = _probe_fit(p, lam=0.0)
    np.testing.assert_allclose(r2, 1.0, atol=1e-10)
    p.Y[...] = 3.0
    p.tgt = to_bf16_bits(p.Y)
    _, _, _, _, r2 = _probe_fit(p, lam=0.1)
    assert (r2 == 0.0).all()


def test_probe_r2_equals_the_moment_identity():
    # RSS = TSS - 2 tr(W^T B) + tr(W^T A W) with the centered moments: the route
    # that needs no second pass over the tokens
    rng = np.random.default_rng(35)
    p = Problem(rng, B=3, T=35)
    sums, A, B, W, r2 = _probe_fit(p, lam=0.7)
    sq = oracle.weighted_squares(p.hm, p.src, p.src_strides, p.d_s, p.tgt, p.tgt_strides, p.d_t, p.w,
                                 p.B * p.T, p.B, p.T)
    for m in range(p.n_maps):
        S = sums[m, 0]
        tss = (sq[m, p.d_s:] - sums[m, 1 + p.d_s:] ** 2 / S).sum()
        Wm = W[m, :p.d_s]
        rss = tss - 2 * np.sum(Wm * B[m]) + np.trace(Wm.T @ A[m] @ Wm)
        assert r2[m] == pytest.approx(1 - rss / tss, abs=1e-11)


def test_select_layers_ranks_mean_r2_with_ties_to_the_smaller_layer():
    hm = {"tgt_layer": np.array([0, 0, 0, 0, 0, 0, 1, 1], np.int32),
          "src_layer": np.array([0, 0, 1, 1, 2, 2, 2, 0], np.int32)}
    r2 = np.array([0.2, 0.4, 0.9, 0.1, 0.5, 0.1, 0.7, 0.7])
    sel, score = oracle.select_layers(hm, r2, n_tgt_layers=2, n_src_layers=3, k=2)
    np.testing.assert_allclose(score[0], [0.3, 0.5, 0.3])
    assert sel[0].tolist() == [1, 0]                       # 0.5, then the 0.3 tie goes to layer 0
    assert sel[1].tolist() == [0, 2]                       # equal scores: smaller layer first
    assert np.isneginf(score[1, 1])
    sel3, _ = oracle.select_layers(hm, r2, n_tgt_layers=2, n_src_layers=3, k=3)
    assert sel3[1].tolist() == [0, 2, -1]                  # a pair without probes is never chosen


def test_select_layers_recovers_the_planted_source_layer():
    # every target layer is generated from one source layer; probes over all
    # (target, source) pairs must rank that layer first
    rng = np.random.default_rng(36)
    L_s, L_t, H, d, B, T = 4, 3, 2, 6, 2, 80
    planted = [2, 0, 3]
    hm = {k: [] for k in ("tgt_layer", "tgt_head", "kv", "src_layer", "src_head", "weight_row")}
    for l in range(L_t):
        for j in range(L_s):
            for z in range(2):
                for h in range(H):
                    for k, v in zip(hm, (l, h, z, j, h, l * H + h)):
                        hm[k].append(v)
    hm = {k: np.asarray(v, np.int32) for k, v in hm.items()}
    p = Problem(rng, L_s=L_s, H_s=H, d_s=d, L_t=L_t, H_t=H, d_t=d, B=B, T=T, hm=hm)
    for l in range(L_t):
        for z in range(2):
            for h in range(H):
                x = p.X[planted[l], z, :, h]
                p.Y[l, z, :, h] = x @ rng.standard_normal((d, d)) + 0.3 * rng.standard_normal(x.shape[:-1] + (d,))
    p.tgt = to_bf16_bits(p.Y)
    _, _, _, _, r2 = _probe_fit(p, lam=1e-3)
    sel, score = oracle.select_layers(hm, r2, L_t, L_s, k=2)
    assert sel[:, 0].tolist() == planted
    for l in range(L_t):
        assert score[l, planted[l]] > 0.8 and np.sort(score[l])[-2] < 0.3


# ----------------------------------------------------------------------------- attention-aligned weights

def _attn_problem(rng, L=1, H=2, Hq=4, d=8, B=2, T=14, equal_keys=False):
    kv = rng.standard_normal((L, 2, B, H, T, d))
    if equal_keys:
        kv[:, 0] = kv[:, 0, :, :, :1]
    q = rng.standard_normal((L, B, 3, Hq, d)) * 1.5
    kvb, qb = to_bf16_bits(kv), to_bf16_bits(q)
    return kvb, synth.cache_strides(L, H, B, T, d), qb, (B * 3 * Hq * d, 3 * Hq * d, Hq * d, d)


def test_attn_sensitivity_equals_autograd_jacobian_norms():
    # Sec. 3.3: r^V_i and r^K_i are the squared Frobenius norms of the Jacobians
    # of the attention output with respect to v_i (up to the factor d) and k_i
    rng = np.random.default_rng(41)
    L, H, Hq, d, B, T = 1, 2, 4, 8, 2, 14
    bounds, stride = [3, 8, 13], 2
    kvb, ks, qb, qs = _attn_problem(rng, L, H, Hq, d, B, T)
    r = oracle.attn_sensitivity(kvb, ks, L, H, d, B, T, qb, qs, Hq, bounds, stride)
    kv = torch.as_tensor(bf16_val(kvb).reshape(L, 2, B, H, T, d))
    qv = torch.as_tensor(bf16_val(qb).reshape(L, B, 3, Hq, d))
    G = Hq // H
    ref = np.zeros_like(r)
    for b in range(B):
        for h in range(H):
            for k, c in enumerate(bounds):
                pV, pK = np.zeros(T), np.zeros(T)
                for u in range(h * G, (h + 1) * G):
                    qu = qv[0, b, k, u]

                    def out(K, V):
                        a = torch.softmax(K[:c + 1] @ qu / np.sqrt(d), dim=0)
                        return a @ V[:c + 1]
                    JK, JV = torch.autograd.functional.jacobian(out, (kv[0, 0, b, h], kv[0, 1, b, h]))
                    # JK, JV: [d_out][T][d]
                    pK += (JK ** 2).sum(dim=(0, 2)).numpy()
                    pV += (JV ** 2).sum(dim=(0, 2)).numpy() / d
                elig = [i for i in range(c) if i % stride == 0]
                for z, pz in ((0, pK), (1, pV)):
                    ref[0, z, h, b * T + np.array(elig)] += pz[elig] / pz[elig].sum()
    np.testing.assert_allclose(r, ref, rtol=1e-10, atol=1e-13)
    # positions outside every prefix, and non-sampled positions, get nothing
    assert not r[..., 13::T].any() and not r[..., 1::2].any()


def test_attn_sensitivity_equal_keys_is_uniform_over_each_prefix():
    rng = np.random.default_rng(42)
    L, H, Hq, d, B, T = 1, 2, 4, 8, 2, 14
    bounds, stride = [2, 5, 13], 3
    kvb, ks, qb, qs = _attn_problem(rng, L, H, Hq, d, B, T, equal_keys=True)
    r = oracle.attn_sensitivity(kvb, ks, L, H, d, B, T, qb, qs, Hq, bounds, stride)
    ref = np.zeros(T)
    for c in bounds:
        elig = [i for i in range(c) if i % stride == 0]
        ref[elig] += 1.0 / len(elig)
    np.testing.assert_allclose(r[0, 1, :, :T], np.broadcast_to(ref, (H, T)), rtol=1e-12)   # r^V
    # each boundary contributes unit mass
    np.testing.assert_allclose(r.reshape(L, 2, H, B, T).sum(axis=-1), len(bounds), rtol=1e-12)


def test_attn_weights_reach_the_printed_ess_floors():
    # Sec. 4.1: n = 128,000 calibration rows (500 x 1,024 tokens, every fourth),
    # tau = min(n, 2 p_l) gives floors 5,120 / 3,072 / 2,048 for p_l = 2,560 / 1,536 / 1,024
    g = json.load(open(GOLDEN))
    ar, widths = g["attn_repair"], g["input_widths"]["local"]
    B, T, s = ar["n_seqs"], ar["seq_len"], ar["sample_stride"]
    rng = np.random.default_rng(43)
    r = np.exp(2.5 * rng.standard_normal((len(widths), B * T)))         # concentrated raw weights
    for row, (p, floor) in enumerate(zip(widths, ar["floors"])):
        w, alpha = oracle.attn_weights(r[row:row + 1], B, T, s, p)
        cal = w[0].reshape(B, T)[:, ::s].ravel()
        assert cal.size == ar["n"]
        assert 0.0 < alpha[0] < 1.0
        n_eff = cal.sum() ** 2 / (cal ** 2).sum()
        assert n_eff == pytest.approx(floor, rel=1e-9)
        assert cal.mean() == pytest.approx(1.0, rel=1e-12)
        assert not w[0].reshape(B, T)[:, 1::s].any()                    # not calibration rows


def test_attn_weights_kish_closed_form_and_degenerate_rows():
    rng = np.random.default_rng(44)
    B, T, s, p = 3, 40, 1, 8                                            # n = 120, tau = 16
    r = np.stack([np.exp(0.3 * rng.standard_normal(B * T)),           # mild: alpha = 1
                  np.exp(3.0 * rng.standard_normal(B * T)),           # concentrated: alpha < 1
                  np.full(B * T, 2.5),                                # constant: CV^2 = 0
                  np.zeros(B * T)])                                   # no mass: uniform
    w, alpha = oracle.attn_weights(r, B, T, s, p)
    n = B * T
    for row in range(2):
        x = r[row] / r[row].mean()
        cv2 = ((x - 1) ** 2).mean()
        n_eff = w[row].sum() ** 2 / (w[row] ** 2).sum()
        assert n_eff == pytest.approx(n / (1 + alpha[row] ** 2 * cv2), rel=1e-12)
    assert alpha[0] == 1.0 and n / (1 + ((r[0] / r[0].mean() - 1) ** 2).mean()) >= 16
    assert alpha[1] < 1.0 and (w[1].sum() ** 2 / (w[1] ** 2).sum()) == pytest.approx(16, rel=1e-12)
    assert alpha[2] == 1.0 and np.allclose(w[2], 1.0)
    assert alpha[3] == 1.0 and np.allclose(w[3], 1.0)


# ----------------------------------------------------------------------------- rotary positions

def _rope_f64(x, pos, theta, style):
    """Exact rotation of fp64 rows x [..., d] at positions pos (for the pins only)."""
    d = x.shape[-1]
    h = d // 2
    f = theta ** (-2.0 * np.arange(h) / d)
    ang = np.asarray(pos, dtype=np.float64)[..., None] * f
    c, s = np.cos(ang), np.sin(ang)
    ia = np.arange(h) if style == 0 else 2 * np.arange(h)
    ib = ia + h if style == 0 else ia + 1
    y = x.copy()
    y[..., ia] = x[..., ia] * c - x[..., ib] * s
    y[..., ib] = x[..., ib] * c + x[..., ia] * s
    return y


@pytest.mark.parametrize("style", [0, 1])
def test_rope_relative_position_property_and_identity_at_zero(style):
    # RoFormer's defining property: <R_p q, R_r k> = <q, R_(r-p) k>, for any
    # positions; it fixes the frequencies, the pairing and the signs
    rng = np.random.default_rng(51)
    d, theta = 16, 10000.0
    L, H, B, T = 1, 1, 1, 40
    x = rng.integers(-8, 9, size=(L, 2, B, H, T, d)).astype(np.float64)
    bits = to_bf16_bits(x)
    st = synth.cache_strides(L, H, B, T, d)
    rot = bf16_val(oracle.rope(bits, st, L, H, d, B, T, theta, style))
    # the oracle's rotated rows are the exact rotation rounded once to bf16
    exact = _rope_f64(x[0, 0, 0, 0], np.arange(T), theta, style)
    np.testing.assert_array_equal(rot[0, 0, 0, 0], bf16_val(oracle.double_to_bf16(exact)))
    np.testing.assert_array_equal(rot[0, 1], x[0, 1])                   # V rows untouched
    np.testing.assert_array_equal(rot[0, 0, 0, 0, 0], x[0, 0, 0, 0, 0])  # position 0: identity
    q, k = rng.standard_normal(d), rng.standard_normal(d)
    for p, r in ((3, 17), (29, 5), (0, 39)):
        lhs = _rope_f64(q, p, theta, style) @ _rope_f64(k, r, theta, style)
        assert lhs == pytest.approx(q @ _rope_f64(k, r - p, theta, style), abs=1e-12)
    # and pair 0 turns by exactly one radian per position (f_0 = 1)
    e = np.zeros(d)
    e[0] = 1.0
    y = _rope_f64(e, 1, theta, style)
    assert y[0] == pytest.approx(np.cos(1.0)) and y[d // 2 if style == 0 else 1] == pytest.approx(np.sin(1.0))


def test_rope_inverse_undoes_forward_up_to_bf16_rounding():
    rng = np.random.default_rng(52)
    L, H, B, T, d = 2, 2, 2, 33, 64
    x = rng.standard_normal((L, 2, B, H, T, d))
    bits = to_bf16_bits(x)
    st = synth.cache_strides(L, H, B, T, d)
    fwd = oracle.rope(bits, st, L, H, d, B, T, 1e6, 0, pos_offset=100)
    back = oracle.rope(fwd, st, L, H, d, B, T, 1e6, 0, inverse=True, pos_offset=100)
    a, b = bf16_val(bits), bf16_val(back)
    assert relF(b, a) < 2 ** -8                                        # two roundings
    # norms of every pair are preserved up to the same rounding
    na = np.hypot(a[:, 0, ..., :d // 2], a[:, 0, ..., d // 2:])
    nb = np.hypot(bf16_val(fwd)[:, 0, ..., :d // 2], bf16_val(fwd)[:, 0, ..., d // 2:])
    assert np.abs(nb - na).max() <= 2 ** -7 * na.max()


@pytest.mark.parametrize("style", [0, 1])
def test_apply_rope_is_rotation_of_the_unrounded_map_output(style):
    # K outputs: the rotation (pinned above by RoFormer's relative-position
    # property) of the exact x~ W~, rounded once; V outputs: plain cb_apply
    rng = np.random.default_rng(53)
    wl, hm, src, out = apply_problem(rng, d_s=8, d_t=16, hm_kind="qwen")
    n = hm["kv"].shape[0]
    ss = synth.cache_strides(wl.L_s, wl.H_s, wl.n_seqs, wl.seq_len, wl.d_s)
    os_ = synth.cache_strides(wl.L_t, wl.H_t, wl.n_seqs, wl.seq_len, wl.d_t)
    # dyadic coefficients with few bits: x~ W~ is exact in fp64 in any order
    W = rng.integers(-64, 65, size=(n, wl.P, wl.d_t)) / 64.0
    theta, off = 1e4, 7
    oracle.apply_rope(hm, W, src, ss, wl.d_s, out, os_, wl.d_t, wl.n_seqs, wl.seq_len, theta, style, off)
    plain = np.zeros_like(out)
    oracle.apply(hm, W, src, ss, wl.d_s, plain, os_, wl.d_t, wl.n_seqs, wl.seq_len)
    X = bf16_val(src)
    pos = off + np.arange(wl.seq_len)
    for m in range(n):
        got = out[hm["tgt_layer"][m], hm["kv"][m], :, hm["tgt_head"][m]]
        if hm["kv"][m] == 1:
            assert np.array_equal(got, plain[hm["tgt_layer"][m], 1, :, hm["tgt_head"][m]])
            continue
        x = X[hm["src_layer"][m], 0, :, hm["src_head"][m]]
        s = np.concatenate([x, np.ones(x.shape[:-1] + (1,))], -1) @ W[m]
        assert np.array_equal(got, oracle.double_to_bf16(_rope_f64(s, pos[None, :], theta, style)))
    # position 0 is the identity: a one-token call at offset 0 equals cb_apply
    one_src = np.ascontiguousarray(src[..., :1, :])
    o1, p1 = (np.zeros(out.shape[:-2] + (1, wl.d_t), dtype=np.uint16) for _ in range(2))
    ss1 = synth.cache_strides(wl.L_s, wl.H_s, wl.n_seqs, 1, wl.d_s)
    os1 = synth.cache_strides(wl.L_t, wl.H_t, wl.n_seqs, 1, wl.d_t)
    oracle.apply_rope(hm, W, one_src, ss1, wl.d_s, o1, os1, wl.d_t, wl.n_seqs, 1, theta, style, 0)
    oracle.apply(hm, W, one_src, ss1, wl.d_s, p1, os1, wl.d_t, wl.n_seqs, 1)
    assert np.array_equal(o1, p1)


def test_apply_rope_inverse_rotation_recovers_cb_apply():
    # de-rotating the fused output with the pinned inverse transform gives
    # the plain mapped cache back up to the two extra roundings
    rng = np.random.default_rng(54)
    wl, hm, src, out = apply_problem(rng, d_s=8, d_t=32, hm_kind="qwen")
    n = hm["kv"].shape[0]
    ss = synth.cache_strides(wl.L_s, wl.H_s, wl.n_seqs, wl.seq_len, wl.d_s)
    os_ = synth.cache_strides(wl.L_t, wl.H_t, wl.n_seqs, wl.seq_len, wl.d_t)
    W = rng.standard_normal((n, wl.P, wl.d_t)) * 0.3
    oracle.apply_rope(hm, W, src, ss, wl.d_s, out, os_, wl.d_t, wl.n_seqs, wl.seq_len, 1e6, 0, 300)
    plain = np.zeros_like(out)
    oracle.apply(hm, W, src, ss, wl.d_s, plain, os_, wl.d_t, wl.n_seqs, wl.seq_len)
    back = oracle.rope(out, os_, wl.L_t, wl.H_t, wl.d_t, wl.n_seqs, wl.seq_len, 1e6, 0, inverse=True,
                       pos_offset=300)
    a, b = bf16_val(plain), bf16_val(back)
    assert np.array_equal(back[:, 1], out[:, 1]) and np.array_equal(out[:, 1], plain[:, 1])
    assert relF(b, a) < 2 ** -7
    assert not np.array_equal(out[:, 0], plain[:, 0])                 # the keys did turn
