"""Pins for the multi-layer oracle functions (Sec. 3.2, Eq. localfeature with k
selected source layers; calibration rows every ``sample_stride``-th token, Sec. 4.1).

What pins what:

* stats_multi  -- the explicit feature matrix X~ = [x_0 .. x_{k-1} 1] gathered by
                  numpy slicing (``[::stride]``) and multiplied by numpy; exact
                  small-integer brute force in Python integers; the diagonal
                  blocks equal the (separately pinned) single-layer moments;
                  reordering S_l permutes the blocks; sampling equals zero
                  weights off the sampling grid.
* solve at P = k d_s + 1 -- exact recovery of a planted integer multi-layer map.
* apply_multi  -- a map that selects one layer copies its rows bit for bit; a
                  pure bias gives RNE(b); numpy fp64 products rounded once.
"""
import numpy as np
import pytest
import torch

import oracle
import synth


def to_bf16_bits(a) -> np.ndarray:
    t = torch.as_tensor(np.asarray(a, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


def relF(a, b):
    return np.linalg.norm(np.asarray(a) - np.asarray(b)) / max(np.linalg.norm(np.asarray(b)), 1e-300)


class MultiProblem:
    """Small explicit multi-layer problem in the canonical cache layout."""

    def __init__(self, rng, k=3, L_s=5, H_s=2, d_s=8, L_t=2, H_t=2, d_t=5, B=3, T=19, values="gauss"):
        self.k, self.L_s, self.H_s, self.d_s, self.L_t, self.H_t, self.d_t, self.B, self.T = \
            k, L_s, H_s, d_s, L_t, H_t, d_t, B, T
        if values == "gauss":
            xs = rng.standard_normal((L_s, 2, B, H_s, T, d_s)) * (1 + np.arange(L_s))[:, None, None, None, None, None]
            ys = rng.standard_normal((L_t, 2, B, H_t, T, d_t)) + 2.0
            w = np.exp(rng.standard_normal((L_t * H_t, B * T)))
        else:
            xs = rng.integers(-4, 5, size=(L_s, 2, B, H_s, T, d_s))
            ys = rng.integers(-4, 5, size=(L_t, 2, B, H_t, T, d_t))
            w = rng.integers(0, 4, size=(L_t * H_t, B * T))
        self.src, self.tgt = to_bf16_bits(xs), to_bf16_bits(ys)
        self.X, self.Y = oracle.bf16_to_double(self.src), oracle.bf16_to_double(self.tgt)
        self.w = w.astype(np.float32)
        hm = {f: [] for f in oracle.MULTI_MAP_FIELDS}
        for l in range(L_t):
            S = list(rng.permutation(L_s)[:k])             # distinct layers in an arbitrary order
            for z in range(2):
                for h in range(H_t):
                    for f, v in zip(oracle.MULTI_MAP_FIELDS, (l, h, z, S, (h + 1) % H_s, l * H_t + h)):
                        hm[f].append(v)
        self.hm = {f: np.asarray(v, np.int32) for f, v in hm.items()}
        self.ss = synth.cache_strides(L_s, H_s, B, T, d_s)
        self.ts = synth.cache_strides(L_t, H_t, B, T, d_t)

    @property
    def n_maps(self):
        return self.hm["kv"].shape[0]

    def stats(self, stride, w=None, hm=None):
        return oracle.stats_multi(self.hm if hm is None else hm, self.src, self.ss, self.d_s, self.tgt, self.ts,
                                  self.d_t, self.w if w is None else w, self.B * self.T, self.B, self.T, stride)

    def design(self, m, stride):
        """X~ (n x P), Y (n x d_t), w (n) of map m on the sampled tokens, by numpy slicing."""
        hm = self.hm
        z, a = hm["kv"][m], hm["src_head"][m]
        xs = [self.X[j, z, :, a, ::stride].reshape(-1, self.d_s) for j in hm["src_layers"][m]]
        x = np.concatenate(xs + [np.ones((xs[0].shape[0], 1))], axis=1)
        y = self.Y[hm["tgt_layer"][m], z, :, hm["tgt_head"][m], ::stride].reshape(-1, self.d_t)
        w = self.w[hm["weight_row"][m]].reshape(self.B, self.T)[:, ::stride].reshape(-1).astype(np.float64)
        return x, y, w


@pytest.mark.parametrize("stride", [1, 3, 4])
def test_multi_stats_equal_explicit_feature_matrix(stride):
    p = MultiProblem(np.random.default_rng(101 + stride))
    G, C = p.stats(stride)
    P = p.k * p.d_s + 1
    assert G.shape == (p.n_maps, P, P) and C.shape == (p.n_maps, P, p.d_t)
    for m in range(p.n_maps):
        x, y, w = p.design(m, stride)
        assert relF(G[m], x.T @ (w[:, None] * x)) < 1e-13
        assert relF(C[m], x.T @ (w[:, None] * y)) < 1e-13
        assert G[m, P - 1, P - 1] == pytest.approx(w.sum(), rel=1e-14)


def test_multi_stats_exact_integer_brute_force():
    p = MultiProblem(np.random.default_rng(7), k=3, L_s=4, d_s=4, d_t=3, B=2, T=7, values="int")
    stride = 2
    G, C = p.stats(stride)
    hm = p.hm
    Xi = p.X.astype(np.int64)
    Yi = p.Y.astype(np.int64)
    wi = p.w.astype(np.int64)
    for m in range(p.n_maps):
        P = p.k * p.d_s + 1
        Gb = [[0] * P for _ in range(P)]
        Cb = [[0] * p.d_t for _ in range(P)]
        z, a = int(hm["kv"][m]), int(hm["src_head"][m])
        for b in range(p.B):
            for t in range(0, p.T, stride):
                xt = []
                for j in hm["src_layers"][m]:
                    xt += [int(v) for v in Xi[j, z, b, a, t]]
                xt.append(1)
                yv = [int(v) for v in Yi[hm["tgt_layer"][m], z, b, hm["tgt_head"][m], t]]
                wv = int(wi[hm["weight_row"][m], b * p.T + t])
                for r in range(P):
                    for c in range(P):
                        Gb[r][c] += wv * xt[r] * xt[c]
                    for c in range(p.d_t):
                        Cb[r][c] += wv * xt[r] * yv[c]
        assert np.array_equal(G[m], np.asarray(Gb, np.float64))
        assert np.array_equal(C[m], np.asarray(Cb, np.float64))


def test_multi_stats_sampling_equals_zero_weights_off_the_grid():
    p = MultiProblem(np.random.default_rng(3), T=21)
    stride = 4
    w0 = p.w.copy().reshape(-1, p.B, p.T)
    w0[:, :, np.arange(p.T) % stride != 0] = 0.0
    G1, C1 = p.stats(stride)
    G2, C2 = p.stats(1, w=w0.reshape(p.w.shape))
    assert np.array_equal(G1, G2) and np.array_equal(C1, C2)


def test_multi_stats_diagonal_blocks_are_single_layer_moments():
    p = MultiProblem(np.random.default_rng(5))
    stride = 3
    G, C = p.stats(stride)
    ds, P = p.d_s, p.k * p.d_s + 1
    w0 = p.w.copy().reshape(-1, p.B, p.T)
    w0[:, :, np.arange(p.T) % stride != 0] = 0.0
    for i in range(p.k):
        hm1 = {f: p.hm[f] for f in ("tgt_layer", "tgt_head", "kv", "src_head", "weight_row")}
        hm1["src_layer"] = p.hm["src_layers"][:, i]
        G1, C1 = oracle.stats(hm1, p.src, p.ss, ds, p.tgt, p.ts, p.d_t, w0.reshape(p.w.shape), p.B * p.T, p.B, p.T)
        blk = slice(i * ds, (i + 1) * ds)
        np.testing.assert_allclose(G[:, blk, blk], G1[:, :ds, :ds], rtol=1e-13, atol=1e-12)
        np.testing.assert_allclose(G[:, blk, P - 1], G1[:, :ds, ds], rtol=1e-13, atol=1e-12)
        np.testing.assert_allclose(C[:, blk, :], C1[:, :ds, :], rtol=1e-13, atol=1e-12)
        np.testing.assert_allclose(C[:, P - 1, :], C1[:, ds, :], rtol=1e-13, atol=1e-12)


def test_multi_stats_layer_order_permutes_blocks():
    p = MultiProblem(np.random.default_rng(9))
    G, C = p.stats(2)
    perm = [2, 0, 1]
    hm2 = dict(p.hm)
    hm2["src_layers"] = p.hm["src_layers"][:, perm]
    G2, C2 = p.stats(2, hm=hm2)
    ds = p.d_s
    idx = np.concatenate([np.arange(i * ds, (i + 1) * ds) for i in perm] + [np.asarray([p.k * ds])])
    assert np.array_equal(G2, G[:, idx][:, :, idx])
    assert np.array_equal(C2, C[:, idx])


def test_multi_solve_recovers_planted_integer_map():
    rng = np.random.default_rng(17)
    k, d_s, d_t, L_s, B, T, stride = 3, 4, 3, 4, 4, 64, 2
    x = rng.integers(-4, 5, size=(L_s, 2, B, 1, T, d_s)).astype(np.float64)
    S = [3, 0, 2]
    Wstar = rng.integers(-2, 3, size=(k * d_s + 1, d_t)).astype(np.float64)
    feat = np.concatenate([x[j, 0, :, 0].reshape(-1, d_s) for j in S] + [np.ones((B * T, 1))], axis=1)
    y = (feat @ Wstar).reshape(1, 1, B, 1, T, d_t)                # integers below 256: exact in bf16
    y = np.concatenate([y, y], axis=1)
    hm = {"tgt_layer": [0], "tgt_head": [0], "kv": [0], "src_layers": [S], "src_head": [0], "weight_row": [0]}
    w = np.exp(rng.standard_normal((1, B * T))).astype(np.float32)
    G, C = oracle.stats_multi(hm, to_bf16_bits(x), synth.cache_strides(L_s, 1, B, T, d_s), d_s, to_bf16_bits(y),
                              synth.cache_strides(1, 1, B, T, d_t), d_t, w, B * T, B, T, stride)
    for unpen in (False, True):
        W, info = oracle.ridge_solve(G, C, 1e-13, relative=True, bias_unpenalized=unpen)
        assert info[0] == 0
        np.testing.assert_allclose(W[0], Wstar, rtol=0, atol=1e-8)


def _apply_setup(rng, k=3, L_s=4, d_s=8, d_t=8, B=2, T=9):
    x = rng.standard_normal((L_s, 2, B, 1, T, d_s)) * 3.0
    src = to_bf16_bits(x)
    hm = {"tgt_layer": [0, 0], "tgt_head": [0, 0], "kv": [0, 1], "src_layers": [[1, 3, 0], [2, 0, 1]],
          "src_head": [0, 0], "weight_row": [0, 0]}
    hm = {f: np.asarray(v, np.int32) for f, v in hm.items()}
    return src, hm, synth.cache_strides(L_s, 1, B, T, d_s), synth.cache_strides(1, 1, B, T, d_t)


def test_multi_apply_layer_selector_copies_bits_and_bias_rounds():
    rng = np.random.default_rng(21)
    k, d = 3, 8
    src, hm, ss, os_ = _apply_setup(rng)
    P = k * d + 1
    for sel in range(k):
        W = np.zeros((2, P, d))
        W[:, sel * d:(sel + 1) * d] = np.eye(d)
        out = np.zeros((1, 2, 2, 1, 9, d), np.uint16)
        oracle.apply_multi(hm, W, src, ss, d, out, os_, d, 2, 9)
        for m in range(2):
            j = hm["src_layers"][m][sel]
            assert np.array_equal(out[0, hm["kv"][m], :, 0], src[j, hm["kv"][m], :, 0])
    W = np.zeros((2, P, d))
    b = rng.standard_normal((2, d)) * 10
    W[:, P - 1] = b
    out = np.zeros((1, 2, 2, 1, 9, d), np.uint16)
    oracle.apply_multi(hm, W, src, ss, d, out, os_, d, 2, 9)
    for m in range(2):
        assert np.array_equal(out[0, m], np.broadcast_to(oracle.double_to_bf16(b[m]), (2, 1, 9, d)))


def test_multi_apply_matches_fp64_products():
    rng = np.random.default_rng(23)
    k, d = 3, 8
    src, hm, ss, os_ = _apply_setup(rng)
    X = oracle.bf16_to_double(src)
    W = rng.standard_normal((2, k * d + 1, d))
    out = np.zeros((1, 2, 2, 1, 9, d), np.uint16)
    oracle.apply_multi(hm, W, src, ss, d, out, os_, d, 2, 9)
    for m in range(2):
        z = hm["kv"][m]
        feat = np.concatenate([X[j, z, :, 0].reshape(-1, d) for j in hm["src_layers"][m]] +
                              [np.ones((18, 1))], axis=1)
        ref = oracle.double_to_bf16(feat @ W[m]).reshape(2, 1, 9, d)
        got = out[0, z]
        same = np.mean(got == ref)
        assert same >= 0.995
        ulp = np.abs(oracle.bf16_to_double(got) - oracle.bf16_to_double(ref))
        assert np.all(ulp <= np.abs(oracle.bf16_to_double(ref)) * 2.0 ** -7 + 1e-30)


def test_qwen_k8_workload_shape_and_windows():
    wl = synth.WORKLOADS["qwen_k8"]
    hm = synth.head_map_multi(wl)
    assert wl.P == 1025 and hm["src_layers"].shape == (1024, 8)
    assert wl.n_seqs * (wl.seq_len // wl.sample_stride) == 128_000       # Sec. 4.1: 500 x 1,024 / 4
    for S in hm["src_layers"]:
        assert len(set(S.tolist())) == 8 and S.min() >= 0 and S.max() < wl.L_s
    # the window is centred on round(l * 39 / 63)
    for l in range(wl.L_t):
        S = synth.layer_window(wl, l)
        assert S[0] <= (2 * l * 39 + 63) // 126 <= S[-1]


# ----------------------------------------------------------------------------- two-pass centered form
#
# stats_multi_centered (Sec. 3.4 two-pass form over the Sec. 3.2 multi-layer
# feature) is pinned by: numpy's weighted covariance of the explicit feature
# matrix (a library routine); exact invariance of A, B when integer data are
# shifted by a constant vector; the Schur-complement identity between the
# centered ridge and the unpenalized augmented ridge of stats_multi; k = 1
# against the single-layer centered oracle; zero-weight maps; sampling equals
# zero weights off the grid.

def centered(p, stride, w=None):
    return oracle.stats_multi_centered(p.hm, p.src, p.ss, p.d_s, p.tgt, p.ts, p.d_t, p.w if w is None else w,
                                       p.B * p.T, p.B, p.T, stride)


@pytest.mark.parametrize("stride", [1, 4])
def test_multi_centered_equals_numpy_weighted_covariance(stride):
    p = MultiProblem(np.random.default_rng(211 + stride))
    sums, A, B = centered(p, stride)
    Dx = p.k * p.d_s
    assert sums.shape == (p.n_maps, 1 + Dx + p.d_t) and A.shape == (p.n_maps, Dx, Dx)
    for m in range(p.n_maps):
        x, y, w = p.design(m, stride)
        x = x[:, :Dx]
        S = w.sum()
        assert sums[m, 0] == pytest.approx(S, rel=1e-14)
        assert relF(sums[m, 1:1 + Dx], w @ x) < 1e-13 and relF(sums[m, 1 + Dx:], w @ y) < 1e-13
        cov = np.cov(np.concatenate([x, y], axis=1).T, aweights=w, bias=True) * S
        assert relF(A[m], cov[:Dx, :Dx]) < 1e-11
        assert relF(B[m], cov[:Dx, Dx:]) < 1e-11


def test_multi_centered_shift_invariance_on_integers():
    rng = np.random.default_rng(17)
    p = MultiProblem(rng, k=2, L_s=3, d_s=4, d_t=3, B=2, T=9, values="int")
    q = MultiProblem(np.random.default_rng(17), k=2, L_s=3, d_s=4, d_t=3, B=2, T=9, values="int")
    # shift every source channel and target channel by an integer constant (exact in bf16)
    sx = rng.integers(-6, 7, size=p.d_s)
    sy = rng.integers(-6, 7, size=p.d_t)
    q.src = to_bf16_bits(p.X + sx)
    q.tgt = to_bf16_bits(p.Y + sy)
    q.w = np.ones_like(p.w)                       # means are then dyadic-free integers / n: keep weights exact
    p.w = np.ones_like(p.w)
    _, A1, B1 = centered(p, 1)
    _, A2, B2 = centered(q, 1)
    assert np.allclose(A1, A2, rtol=0, atol=1e-9 * np.abs(A1).max())
    assert np.allclose(B1, B2, rtol=0, atol=1e-9 * max(np.abs(B1).max(), 1.0))


@pytest.mark.parametrize("relative,lam", [(True, 1e-2), (False, 0.5)])
def test_multi_centered_ridge_equals_unpenalized_augmented_ridge(relative, lam):
    p = MultiProblem(np.random.default_rng(23), T=29)
    stride = 2
    sums, A, B = centered(p, stride)
    G, C = p.stats(stride)
    Wc, ic = oracle.ridge_solve_centered(sums, A, B, lam, relative=relative)
    Wa, ia = oracle.ridge_solve(G, C, lam, relative=relative, bias_unpenalized=True)
    assert (ic == 0).all() and (ia == 0).all()
    for m in range(p.n_maps):
        assert relF(Wc[m], Wa[m]) < 1e-9


def test_multi_centered_k1_equals_single_layer_centered():
    p = MultiProblem(np.random.default_rng(29), k=1)
    sums, A, B = centered(p, 1)
    hm1 = {"tgt_layer": p.hm["tgt_layer"], "tgt_head": p.hm["tgt_head"], "kv": p.hm["kv"],
           "src_layer": p.hm["src_layers"][:, 0].copy(), "src_head": p.hm["src_head"],
           "weight_row": p.hm["weight_row"]}
    s1, A1, B1 = oracle.stats_centered(hm1, p.src, p.ss, p.d_s, p.tgt, p.ts, p.d_t, p.w, p.B * p.T, p.B, p.T)
    assert np.array_equal(sums, s1) and np.array_equal(A, A1) and np.array_equal(B, B1)


def test_multi_centered_zero_weights_and_sampling():
    p = MultiProblem(np.random.default_rng(31), T=22)
    w = p.w.copy()
    w[0] = 0.0                                    # maps of weight row 0 see no weight
    sums, A, B = centered(p, 3, w=w)
    zero = np.where(p.hm["weight_row"] == 0)[0]
    assert len(zero) > 0
    for m in zero:
        assert not sums[m].any() and not A[m].any() and not B[m].any()
    w0 = p.w.copy().reshape(-1, p.B, p.T)
    w0[:, :, np.arange(p.T) % 3 != 0] = 0.0
    s1, A1, B1 = centered(p, 3)
    s2, A2, B2 = centered(p, 1, w=w0.reshape(p.w.shape))
    assert np.array_equal(s1, s2) and np.array_equal(A1, A2) and np.array_equal(B1, B2)


# ----------------------------------------------------------------------------- target rotation, k > 1

def _rope_f64(x, pos, theta, style):
    """Exact rotation of fp64 rows x [..., d] at positions pos: the transform that
    RoFormer's relative-position property pins in test_oracle_pins."""
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
def test_multi_apply_rope_is_rotation_of_the_unrounded_output(style):
    # K maps: the rotation of the exact x~ W~ (dyadic coefficients with few
    # bits: exact in fp64 in any order), rounded once; V maps: oracle_apply_multi
    rng = np.random.default_rng(61)
    k, d = 3, 8
    src, hm, ss, os_ = _apply_setup(rng)
    X = oracle.bf16_to_double(src)
    W = rng.integers(-64, 65, size=(2, k * d + 1, d)) / 64.0
    theta, off = 1e4, 11
    out = np.zeros((1, 2, 2, 1, 9, d), np.uint16)
    oracle.apply_multi_rope(hm, W, src, ss, d, out, os_, d, 2, 9, theta, style, off)
    plain = np.zeros_like(out)
    oracle.apply_multi(hm, W, src, ss, d, plain, os_, d, 2, 9)
    pos = off + np.arange(9)
    for m in range(2):
        z = hm["kv"][m]
        if z == 1:
            assert np.array_equal(out[0, 1], plain[0, 1])
            continue
        feat = np.concatenate([X[j, z, :, 0] for j in hm["src_layers"][m]] + [np.ones((2, 9, 1))], axis=-1)
        s = feat @ W[m]
        assert np.array_equal(out[0, z, :, 0], oracle.double_to_bf16(_rope_f64(s, pos[None, :], theta, style)))
    # position 0 turns nothing: a one-token call at offset 0 equals oracle_apply_multi
    o1, p1 = (np.zeros((1, 2, 2, 1, 1, d), np.uint16) for _ in range(2))
    s1 = np.ascontiguousarray(src[..., :1, :])
    ss1, os1 = synth.cache_strides(4, 1, 2, 1, d), synth.cache_strides(1, 1, 2, 1, d)
    oracle.apply_multi_rope(hm, W, s1, ss1, d, o1, os1, d, 2, 1, theta, style, 0)
    oracle.apply_multi(hm, W, s1, ss1, d, p1, os1, d, 2, 1)
    assert np.array_equal(o1, p1)


def test_multi_apply_rope_k1_equals_single_layer_apply_rope():
    rng = np.random.default_rng(62)
    L_s, H_s, L_t, H_t, B, T, d = 3, 2, 2, 2, 2, 13, 16
    src = to_bf16_bits(rng.standard_normal((L_s, 2, B, H_s, T, d)) * 2)
    hm1 = {f: [] for f in oracle.HEAD_MAP_FIELDS}
    for l in range(L_t):
        for z in range(2):
            for h in range(H_t):
                for f, v in zip(oracle.HEAD_MAP_FIELDS, (l, h, z, (l + h) % L_s, (h + 1) % H_s, l * H_t + h)):
                    hm1[f].append(v)
    hm1 = {f: np.asarray(v, np.int32) for f, v in hm1.items()}
    hmk = {f: hm1[f] for f in ("tgt_layer", "tgt_head", "kv", "src_head", "weight_row")}
    hmk["src_layers"] = hm1["src_layer"].reshape(-1, 1)
    n = hm1["kv"].shape[0]
    W = rng.standard_normal((n, d + 1, d))
    ss, os_ = synth.cache_strides(L_s, H_s, B, T, d), synth.cache_strides(L_t, H_t, B, T, d)
    for style in (0, 1):
        a = np.zeros((L_t, 2, B, H_t, T, d), np.uint16)
        b = np.zeros_like(a)
        oracle.apply_rope(hm1, W, src, ss, d, a, os_, d, B, T, 5e5, style, 40)
        oracle.apply_multi_rope(hmk, W, src, ss, d, b, os_, d, B, T, 5e5, style, 40)
        assert np.array_equal(a, b)


def test_multi_apply_rope_inverse_rotation_recovers_apply_multi():
    # de-rotating with the pinned inverse transform gives the unrotated mapped
    # cache back up to the two extra roundings
    rng = np.random.default_rng(63)
    k, d = 3, 32
    src, hm, ss, os_ = _apply_setup(rng, d_s=d, d_t=d)
    W = rng.standard_normal((2, k * d + 1, d)) * 0.2
    out = np.zeros((1, 2, 2, 1, 9, d), np.uint16)
    oracle.apply_multi_rope(hm, W, src, ss, d, out, os_, d, 2, 9, 1e6, 0, 2000)
    plain = np.zeros_like(out)
    oracle.apply_multi(hm, W, src, ss, d, plain, os_, d, 2, 9)
    back = oracle.rope(out, os_, 1, 1, d, 2, 9, 1e6, 0, inverse=True, pos_offset=2000)
    a, b = oracle.bf16_to_double(plain), oracle.bf16_to_double(back)
    assert np.array_equal(out[:, 1], plain[:, 1])
    assert relF(b, a) < 2 ** -7
    assert not np.array_equal(out[:, 0], plain[:, 0])
