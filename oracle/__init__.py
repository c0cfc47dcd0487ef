"""fp64 CPU oracle for the CacheBridge mapper path -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The product library
(``paper_2609_00891_amd``) never imports it, and it imports nothing from the
product.  The arithmetic lives in ``cb_oracle.c`` (plain loops, fp64); this
module only marshals numpy arrays through ctypes.

Functions follow the paper (CacheBridge, "Efficient Cross-Model KV Cache
Transfer"):

* :func:`stats` -- augmented weighted moments G, C (Sec. 3.4, Eq. fusedstats,
  over the head-local feature of Sec. 3.2, Eq. localfeature, with k = 1).
* :func:`ridge_solve` -- (G + lambda D)^-1 C (Sec. 3.1, Eq. closedform; Sec. 3.4).
* :func:`stats_centered` -- two-pass weighted means and centered moments A, B
  (Sec. 3.4, Eq. fusedstats as stated: means first, then centered panels).
* :func:`ridge_solve_centered` -- W = (A + lambda I)^-1 B, b = mu_y - W^T mu_x
  (Sec. 3.1, Eq. closedform).
* :func:`apply` -- RNE_bf16([x;1] W~) per token (Sec. 1; Sec. 2.3, Eq. support-cost).
* :func:`weighted_squares` -- sum w x_i^2, sum w y_j^2 per channel.
* :func:`probe_r2` -- held-in R^2 = 1 - RSS/TSS of fitted probes, from explicit
  residuals (Sec. 3.1, layer selection).
* :func:`select_layers` -- mean probe R^2 per (target, source) layer pair over
  KV heads and K/V, ranked; the first k source layers form S_l (Sec. 3.1).
* :func:`attn_sensitivity` -- raw attention-aligned sensitivities r^K, r^V at
  causal prefix boundaries (Sec. 3.3, Eq. attentionlinearization, Eq. sensitivity).
* :func:`attn_weights` -- mean-one normalization and the ESS-floor shrinkage
  w = 1 + alpha* (r - 1) (Sec. 3.3).
* :func:`rope` -- rotary position transform of the K rows of a cache, forward or
  inverse (Sec. 2.1, Sec. 3.1: RoPE removed before fitting, restored after mapping).
* :func:`stats_multi` -- G, C over the multi-layer head-local feature
  x~ = [x_0; ...; x_{k-1}; 1] (Sec. 3.2, Eq. localfeature with k selected
  source layers), on every ``sample_stride``-th token (Sec. 4.1).
* :func:`apply_multi` -- RNE_bf16(x~ W~) for multi-layer maps.
* :func:`coefficient_count` -- C(f) = 2 L_t H_t (k f d_s) d_t (Sec. 2.3, Eq. support-cost).

Parity status: pinned by ``tests/test_oracle_pins.py``.
"""
from __future__ import annotations

import ctypes
import os
from typing import Mapping, Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None

_i32p = ctypes.POINTER(ctypes.c_int32)
_i64p = ctypes.POINTER(ctypes.c_int64)
_u16p = ctypes.POINTER(ctypes.c_uint16)
_f32p = ctypes.POINTER(ctypes.c_float)
_f64p = ctypes.POINTER(ctypes.c_double)

HEAD_MAP_FIELDS = ("tgt_layer", "tgt_head", "kv", "src_layer", "src_head", "weight_row")


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        from . import build as _b  # noqa: PLC0415
        _b.build()
    lib = ctypes.CDLL(_LIB_PATH)
    lib.oracle_stats.restype = ctypes.c_int
    lib.oracle_stats.argtypes = [ctypes.c_int] + [_i32p] * 6 + [
        _u16p, _i64p, ctypes.c_int, _u16p, _i64p, ctypes.c_int,
        _f32p, ctypes.c_int64, ctypes.c_int, ctypes.c_int, _f64p, _f64p, ctypes.c_int]
    lib.oracle_ridge_solve.restype = ctypes.c_int
    lib.oracle_ridge_solve.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, _f64p, _f64p,
                                       ctypes.c_double, ctypes.c_int, ctypes.c_int, _f64p, _i32p,
                                       ctypes.c_int]
    lib.oracle_apply_rope.restype = ctypes.c_int
    lib.oracle_apply_rope.argtypes = [ctypes.c_int] + [_i32p] * 5 + [
        _f64p, _u16p, _i64p, ctypes.c_int, _u16p, _i64p, ctypes.c_int, ctypes.c_int, ctypes.c_int,
        ctypes.c_double, ctypes.c_int, ctypes.c_int, ctypes.c_int]
    lib.oracle_apply.restype = ctypes.c_int
    lib.oracle_apply.argtypes = [ctypes.c_int] + [_i32p] * 5 + [
        _f64p, _u16p, _i64p, ctypes.c_int, _u16p, _i64p, ctypes.c_int,
        ctypes.c_int, ctypes.c_int, ctypes.c_int]
    lib.oracle_stats_centered.restype = ctypes.c_int
    lib.oracle_stats_centered.argtypes = [ctypes.c_int] + [_i32p] * 6 + [
        _u16p, _i64p, ctypes.c_int, _u16p, _i64p, ctypes.c_int,
        _f32p, ctypes.c_int64, ctypes.c_int, ctypes.c_int, _f64p, _f64p, _f64p, ctypes.c_int]
    lib.oracle_ridge_solve_centered.restype = ctypes.c_int
    lib.oracle_ridge_solve_centered.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, _f64p, _f64p, _f64p,
                                                ctypes.c_double, ctypes.c_int, _f64p, _i32p, ctypes.c_int]
    lib.oracle_weighted_squares.restype = ctypes.c_int
    lib.oracle_weighted_squares.argtypes = [ctypes.c_int] + [_i32p] * 6 + [
        _u16p, _i64p, ctypes.c_int, _u16p, _i64p, ctypes.c_int,
        _f32p, ctypes.c_int64, ctypes.c_int, ctypes.c_int, _f64p, ctypes.c_int]
    lib.oracle_probe_r2.restype = ctypes.c_int
    lib.oracle_probe_r2.argtypes = [ctypes.c_int] + [_i32p] * 6 + [
        _f64p, _u16p, _i64p, ctypes.c_int, _u16p, _i64p, ctypes.c_int,
        _f32p, ctypes.c_int64, ctypes.c_int, ctypes.c_int, _f64p, ctypes.c_int]
    lib.oracle_attn_sensitivity.restype = ctypes.c_int
    lib.oracle_attn_sensitivity.argtypes = [ctypes.c_int] * 6 + [_u16p, _i64p, _u16p, _i64p, _i32p, ctypes.c_int,
                                                                 ctypes.c_int, _f64p, ctypes.c_int]
    lib.oracle_attn_weights.restype = ctypes.c_int
    lib.oracle_attn_weights.argtypes = [ctypes.c_int] * 4 + [_f64p, ctypes.c_int, _f64p, _f64p]
    lib.oracle_rope.restype = ctypes.c_int
    lib.oracle_rope.argtypes = [ctypes.c_int] * 5 + [_u16p, _i64p, _u16p, _i64p, ctypes.c_double, ctypes.c_int,
                                                     ctypes.c_int, ctypes.c_int]
    lib.oracle_stats_multi.restype = ctypes.c_int
    lib.oracle_stats_multi.argtypes = [ctypes.c_int, ctypes.c_int] + [_i32p] * 6 + [
        _u16p, _i64p, ctypes.c_int, _u16p, _i64p, ctypes.c_int,
        _f32p, ctypes.c_int64, ctypes.c_int, ctypes.c_int, ctypes.c_int, _f64p, _f64p, ctypes.c_int]
    lib.oracle_stats_multi_centered.restype = ctypes.c_int
    lib.oracle_stats_multi_centered.argtypes = [ctypes.c_int, ctypes.c_int] + [_i32p] * 6 + [
        _u16p, _i64p, ctypes.c_int, _u16p, _i64p, ctypes.c_int,
        _f32p, ctypes.c_int64, ctypes.c_int, ctypes.c_int, ctypes.c_int, _f64p, _f64p, _f64p, ctypes.c_int]
    lib.oracle_apply_multi.restype = ctypes.c_int
    lib.oracle_apply_multi.argtypes = [ctypes.c_int, ctypes.c_int] + [_i32p] * 5 + [
        _f64p, _u16p, _i64p, ctypes.c_int, _u16p, _i64p, ctypes.c_int,
        ctypes.c_int, ctypes.c_int, ctypes.c_int]
    lib.oracle_apply_multi_rope.restype = ctypes.c_int
    lib.oracle_apply_multi_rope.argtypes = [ctypes.c_int, ctypes.c_int] + [_i32p] * 5 + [
        _f64p, _u16p, _i64p, ctypes.c_int, _u16p, _i64p, ctypes.c_int,
        ctypes.c_int, ctypes.c_int, ctypes.c_double, ctypes.c_int, ctypes.c_int, ctypes.c_int]
    lib.oracle_double_to_bf16_array.restype = ctypes.c_int
    lib.oracle_double_to_bf16_array.argtypes = [ctypes.c_int64, _f64p, _u16p]
    _lib = lib
    return lib


def _ptr(a: np.ndarray, ctype):
    return a.ctypes.data_as(ctype)


def _hm_arrays(head_map: Mapping[str, np.ndarray], fields=HEAD_MAP_FIELDS):
    out = []
    n = None
    for f in fields:
        a = np.ascontiguousarray(np.asarray(head_map[f], dtype=np.int32))
        if n is None:
            n = a.shape[0]
        if a.shape != (n,):
            raise ValueError(f"head_map field {f} has shape {a.shape}, expected ({n},)")
        out.append(a)
    return n, out


def _strides5(strides) -> np.ndarray:
    s = np.ascontiguousarray(np.asarray(strides, dtype=np.int64))
    if s.shape != (5,):
        raise ValueError("strides must be (layer, kv, seq, head, tok) element strides")
    return s


def _u16(a: np.ndarray) -> np.ndarray:
    if a.dtype != np.uint16:
        raise TypeError("caches are passed as uint16 arrays holding bfloat16 bits")
    return a


def stats(head_map, src, src_strides, d_s, tgt, tgt_strides, d_t, weights, w_row_stride,
          n_seqs, seq_len, G: Optional[np.ndarray] = None, C: Optional[np.ndarray] = None,
          n_threads: int = 0):
    """Accumulate G += sum w x~ x~^T and C += sum w x~ y^T in fp64 for every map.

    ``src``/``tgt`` are flat (or any-shaped, C-contiguous) uint16 arrays of
    bfloat16 bits addressed with the given element strides
    (layer, kv, seq, head, tok); channel stride is 1.  ``weights`` is fp32,
    indexed ``row * w_row_stride + seq * seq_len + tok``.  Returns (G, C).
    """
    lib = _load()
    n, hm = _hm_arrays(head_map)
    P = d_s + 1
    if G is None:
        G = np.zeros((n, P, P), dtype=np.float64)
    if C is None:
        C = np.zeros((n, P, d_t), dtype=np.float64)
    assert G.dtype == np.float64 and G.flags.c_contiguous and G.shape == (n, P, P)
    assert C.dtype == np.float64 and C.flags.c_contiguous and C.shape == (n, P, d_t)
    src = np.ascontiguousarray(_u16(src))
    tgt = np.ascontiguousarray(_u16(tgt))
    w = np.ascontiguousarray(np.asarray(weights, dtype=np.float32))
    ss, ts = _strides5(src_strides), _strides5(tgt_strides)
    lib.oracle_stats(n, *[_ptr(a, _i32p) for a in hm], _ptr(src, _u16p), _ptr(ss, _i64p), d_s,
                     _ptr(tgt, _u16p), _ptr(ts, _i64p), d_t, _ptr(w, _f32p), int(w_row_stride),
                     int(n_seqs), int(seq_len), _ptr(G, _f64p), _ptr(C, _f64p), int(n_threads))
    return G, C


def ridge_solve(G, C, lam, relative=True, bias_unpenalized=False, n_threads: int = 0):
    """Solve (G + lambda_m D) W~ = C per map in fp64; returns (W~, info)."""
    lib = _load()
    G = np.ascontiguousarray(np.asarray(G, dtype=np.float64))
    C = np.ascontiguousarray(np.asarray(C, dtype=np.float64))
    n, P, P2 = G.shape
    assert P == P2 and C.shape[:2] == (n, P)
    d_t = C.shape[2]
    W = np.zeros((n, P, d_t), dtype=np.float64)
    info = np.zeros((n,), dtype=np.int32)
    lib.oracle_ridge_solve(n, P, d_t, _ptr(G, _f64p), _ptr(C, _f64p), float(lam), int(bool(relative)),
                           int(bool(bias_unpenalized)), _ptr(W, _f64p), _ptr(info, _i32p),
                           int(n_threads))
    return W, info


def stats_centered(head_map, src, src_strides, d_s, tgt, tgt_strides, d_t, weights, w_row_stride,
                   n_seqs, seq_len, n_threads: int = 0):
    """Two-pass centered statistics in fp64: returns (sums, A, B) with
    sums[m] = (sum w, sum w x, sum w y), A[m] = sum w (x-mu_x)(x-mu_x)^T and
    B[m] = sum w (x-mu_x)(y-mu_y)^T.  Same input conventions as :func:`stats`."""
    lib = _load()
    n, hm = _hm_arrays(head_map)
    sums = np.zeros((n, 1 + d_s + d_t), dtype=np.float64)
    A = np.zeros((n, d_s, d_s), dtype=np.float64)
    B = np.zeros((n, d_s, d_t), dtype=np.float64)
    src = np.ascontiguousarray(_u16(src))
    tgt = np.ascontiguousarray(_u16(tgt))
    w = np.ascontiguousarray(np.asarray(weights, dtype=np.float32))
    ss, ts = _strides5(src_strides), _strides5(tgt_strides)
    lib.oracle_stats_centered(n, *[_ptr(a, _i32p) for a in hm], _ptr(src, _u16p), _ptr(ss, _i64p), d_s,
                              _ptr(tgt, _u16p), _ptr(ts, _i64p), d_t, _ptr(w, _f32p), int(w_row_stride),
                              int(n_seqs), int(seq_len), _ptr(sums, _f64p), _ptr(A, _f64p), _ptr(B, _f64p),
                              int(n_threads))
    return sums, A, B


def ridge_solve_centered(sums, A, B, lam, relative=True, n_threads: int = 0):
    """Centered ridge: W = (A + lambda_m I)^-1 B, b = mu_y - W^T mu_x; returns
    (W~ [n][d_s+1][d_t] with the bias as the last row, info)."""
    lib = _load()
    sums = np.ascontiguousarray(np.asarray(sums, dtype=np.float64))
    A = np.ascontiguousarray(np.asarray(A, dtype=np.float64))
    B = np.ascontiguousarray(np.asarray(B, dtype=np.float64))
    n, d_s, d_s2 = A.shape
    assert d_s == d_s2 and B.shape[:2] == (n, d_s)
    d_t = B.shape[2]
    assert sums.shape == (n, 1 + d_s + d_t)
    W = np.zeros((n, d_s + 1, d_t), dtype=np.float64)
    info = np.zeros((n,), dtype=np.int32)
    lib.oracle_ridge_solve_centered(n, d_s, d_t, _ptr(sums, _f64p), _ptr(A, _f64p), _ptr(B, _f64p),
                                    float(lam), int(bool(relative)), _ptr(W, _f64p), _ptr(info, _i32p),
                                    int(n_threads))
    return W, info


def apply(head_map, W, src, src_strides, d_s, out, out_strides, d_t, n_seqs, seq_len,
          n_threads: int = 0):
    """Write RNE_bf16([x;1] W~) for every map and token into ``out`` (uint16 bits)."""
    lib = _load()
    n, hm = _hm_arrays(head_map, HEAD_MAP_FIELDS[:5])
    W = np.ascontiguousarray(np.asarray(W, dtype=np.float64))
    assert W.shape == (n, d_s + 1, d_t)
    src = np.ascontiguousarray(_u16(src))
    if not (out.dtype == np.uint16 and out.flags.c_contiguous):
        raise TypeError("out must be a C-contiguous uint16 array")
    ss, os_ = _strides5(src_strides), _strides5(out_strides)
    lib.oracle_apply(n, *[_ptr(a, _i32p) for a in hm], _ptr(W, _f64p), _ptr(src, _u16p),
                     _ptr(ss, _i64p), d_s, _ptr(out, _u16p), _ptr(os_, _i64p), d_t,
                     int(n_seqs), int(seq_len), int(n_threads))
    return out


def apply_rope(head_map, W, src, src_strides, d_s, out, out_strides, d_t, n_seqs, seq_len, theta: float,
               style: int = 0, pos_offset: int = 0, n_threads: int = 0):
    """Like :func:`apply`, with the K outputs turned by the target RoPE (fp64) before the one rounding."""
    lib = _load()
    n, hm = _hm_arrays(head_map, HEAD_MAP_FIELDS[:5])
    W = np.ascontiguousarray(np.asarray(W, dtype=np.float64))
    assert W.shape == (n, d_s + 1, d_t)
    src = np.ascontiguousarray(_u16(src))
    if not (out.dtype == np.uint16 and out.flags.c_contiguous):
        raise TypeError("out must be a C-contiguous uint16 array")
    ss, os_ = _strides5(src_strides), _strides5(out_strides)
    lib.oracle_apply_rope(n, *[_ptr(a, _i32p) for a in hm], _ptr(W, _f64p), _ptr(src, _u16p),
                          _ptr(ss, _i64p), d_s, _ptr(out, _u16p), _ptr(os_, _i64p), d_t,
                          int(n_seqs), int(seq_len), float(theta), int(style), int(pos_offset), int(n_threads))
    return out


def weighted_squares(head_map, src, src_strides, d_s, tgt, tgt_strides, d_t, weights, w_row_stride,
                     n_seqs, seq_len, n_threads: int = 0):
    """sq[m] = (sum w x_i^2 (d_s), sum w y_j^2 (d_t)) in fp64; conventions of :func:`stats`."""
    lib = _load()
    n, hm = _hm_arrays(head_map)
    sq = np.zeros((n, d_s + d_t), dtype=np.float64)
    src = np.ascontiguousarray(_u16(src))
    tgt = np.ascontiguousarray(_u16(tgt))
    w = np.ascontiguousarray(np.asarray(weights, dtype=np.float32))
    ss, ts = _strides5(src_strides), _strides5(tgt_strides)
    lib.oracle_weighted_squares(n, *[_ptr(a, _i32p) for a in hm], _ptr(src, _u16p), _ptr(ss, _i64p), d_s,
                                _ptr(tgt, _u16p), _ptr(ts, _i64p), d_t, _ptr(w, _f32p), int(w_row_stride),
                                int(n_seqs), int(seq_len), _ptr(sq, _f64p), int(n_threads))
    return sq


def probe_r2(head_map, W, src, src_strides, d_s, tgt, tgt_strides, d_t, weights, w_row_stride,
             n_seqs, seq_len, n_threads: int = 0):
    """r2[m] = 1 - RSS/TSS of the fitted map W~[m] ([n][d_s+1][d_t], bias last) on the
    same weighted tokens, pooled over output channels (0 when TSS = 0)."""
    lib = _load()
    n, hm = _hm_arrays(head_map)
    W = np.ascontiguousarray(np.asarray(W, dtype=np.float64))
    assert W.shape == (n, d_s + 1, d_t)
    r2 = np.zeros((n,), dtype=np.float64)
    src = np.ascontiguousarray(_u16(src))
    tgt = np.ascontiguousarray(_u16(tgt))
    w = np.ascontiguousarray(np.asarray(weights, dtype=np.float32))
    ss, ts = _strides5(src_strides), _strides5(tgt_strides)
    lib.oracle_probe_r2(n, *[_ptr(a, _i32p) for a in hm], _ptr(W, _f64p), _ptr(src, _u16p), _ptr(ss, _i64p),
                        d_s, _ptr(tgt, _u16p), _ptr(ts, _i64p), d_t, _ptr(w, _f32p), int(w_row_stride),
                        int(n_seqs), int(seq_len), _ptr(r2, _f64p), int(n_threads))
    return r2


def select_layers(head_map, r2, n_tgt_layers: int, n_src_layers: int, k: int):
    """Sec. 3.1 layer selection: score[l][j] = mean r2 over the maps with target
    layer l and source layer j (every KV head, K and V); for each l the source
    layers in decreasing score (equal scores: smaller j first), first k of them.
    Pairs without maps get score -inf and are never chosen (-1 pads the list).
    Returns (selected [L_t][k] int32, score [L_t][L_s])."""
    tl = np.asarray(head_map["tgt_layer"])
    sl = np.asarray(head_map["src_layer"])
    r2 = np.asarray(r2, dtype=np.float64)
    score = np.full((n_tgt_layers, n_src_layers), -np.inf)
    for l in range(n_tgt_layers):
        for j in range(n_src_layers):
            sel = (tl == l) & (sl == j)
            if sel.any():
                score[l, j] = r2[sel].mean()
    selected = np.full((n_tgt_layers, k), -1, dtype=np.int32)
    for l in range(n_tgt_layers):
        order = sorted(range(n_src_layers), key=lambda j: (-score[l, j], j))
        chosen = [j for j in order if np.isfinite(score[l, j])][:k]
        selected[l, :len(chosen)] = chosen
    return selected, score


def attn_sensitivity(kv_cache, kv_strides, n_layers: int, n_heads: int, d: int, n_seqs: int, seq_len: int,
                     q, q_strides, n_qheads: int, boundaries, sample_stride: int = 1, n_threads: int = 0):
    """Raw sensitivities r [n_layers][2][n_heads][n_seqs*seq_len] (component 0 = K, 1 = V).

    ``kv_cache``: uint16 bf16 bits of a target cache addressed with ``kv_strides``
    (layer, kv, seq, head, tok); ``q``: uint16 bf16 bits of the boundary queries,
    element (layer, seq, boundary, query head, j) at the dot product with
    ``q_strides`` (4 strides).  ``boundaries``: increasing query positions."""
    lib = _load()
    kvc = np.ascontiguousarray(_u16(kv_cache))
    qa = np.ascontiguousarray(_u16(q))
    ks = _strides5(kv_strides)
    qs = np.ascontiguousarray(np.asarray(q_strides, dtype=np.int64))
    assert qs.shape == (4,)
    bd = np.ascontiguousarray(np.asarray(boundaries, dtype=np.int32))
    assert n_qheads % n_heads == 0 and (np.diff(bd) > 0).all() and bd[0] >= 0 and bd[-1] < seq_len
    r = np.zeros((n_layers, 2, n_heads, n_seqs * seq_len), dtype=np.float64)
    lib.oracle_attn_sensitivity(n_layers, n_heads, n_qheads, d, n_seqs, seq_len, _ptr(kvc, _u16p), _ptr(ks, _i64p),
                                _ptr(qa, _u16p), _ptr(qs, _i64p), _ptr(bd, _i32p), int(bd.shape[0]),
                                int(sample_stride), _ptr(r, _f64p), int(n_threads))
    return r


def attn_weights(r, n_seqs: int, seq_len: int, sample_stride: int, p: int):
    """ESS-floor shrinkage per row of r [..., n_seqs*seq_len]: returns (w, alpha) with
    w = 1 + alpha (r/mean - 1) on calibration rows (t mod sample_stride = 0), 0 elsewhere."""
    lib = _load()
    r = np.ascontiguousarray(np.asarray(r, dtype=np.float64))
    shape = r.shape
    rows = int(np.prod(shape[:-1]))
    assert shape[-1] == n_seqs * seq_len
    w = np.zeros(shape, dtype=np.float64)
    alpha = np.zeros(shape[:-1], dtype=np.float64)
    lib.oracle_attn_weights(rows, n_seqs, seq_len, sample_stride, _ptr(r, _f64p), int(p), _ptr(w, _f64p),
                            _ptr(alpha, _f64p))
    return w, alpha


def rope(cache, strides, n_layers: int, n_heads: int, d: int, n_seqs: int, seq_len: int, theta: float,
         style: int = 0, inverse: bool = False, pos_offset: int = 0):
    """Rotate (or, with inverse, de-rotate) the K rows of a bf16 cache (uint16 bits, canonical
    contiguous layout for the output); V rows are copied.  style 0: pairs (i, i + d/2);
    style 1: pairs (2i, 2i + 1).  Returns the output bits."""
    lib = _load()
    src = np.ascontiguousarray(_u16(cache))
    ss = _strides5(strides)
    out = np.zeros((n_layers, 2, n_seqs, n_heads, seq_len, d), dtype=np.uint16)
    os_ = np.asarray([2 * n_seqs * n_heads * seq_len * d, n_seqs * n_heads * seq_len * d, n_heads * seq_len * d,
                      seq_len * d, d], dtype=np.int64)
    lib.oracle_rope(n_layers, n_heads, d, n_seqs, seq_len, _ptr(src, _u16p), _ptr(ss, _i64p), _ptr(out, _u16p),
                    _ptr(os_, _i64p), float(theta), int(style), int(bool(inverse)), int(pos_offset))
    return out


def double_to_bf16(v) -> np.ndarray:
    """Round fp64 values once to bfloat16 (nearest, ties to even); returns uint16 bits."""
    lib = _load()
    v = np.ascontiguousarray(np.asarray(v, dtype=np.float64))
    out = np.empty(v.shape, dtype=np.uint16)
    lib.oracle_double_to_bf16_array(v.size, _ptr(v, _f64p), _ptr(out, _u16p))
    return out


def bf16_to_double(bits) -> np.ndarray:
    """bfloat16 bits -> fp64 (exact)."""
    b = np.asarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def coefficient_count(L_t: int, H_t: int, k: int, f: int, d_s: int, d_t: int) -> int:
    """Non-bias coefficient count over K and V, C(f) = 2 L_t H_t (k f d_s) d_t (Eq. support-cost)."""
    return 2 * L_t * H_t * (k * f * d_s) * d_t


MULTI_MAP_FIELDS = ("tgt_layer", "tgt_head", "kv", "src_layers", "src_head", "weight_row")


def _multi_arrays(head_map, fields=MULTI_MAP_FIELDS):
    n, k, out = None, None, []
    for f in fields:
        a = np.ascontiguousarray(np.asarray(head_map[f], dtype=np.int32))
        if f == "src_layers":
            if a.ndim != 2:
                raise ValueError("src_layers must be [n_maps][k]")
            k = a.shape[1]
        if n is None:
            n = a.shape[0]
        if a.shape[0] != n:
            raise ValueError(f"head_map field {f} has {a.shape[0]} entries, expected {n}")
        out.append(a)
    return n, k, out


def stats_multi(head_map, src, src_strides, d_s, tgt, tgt_strides, d_t, weights, w_row_stride,
                n_seqs, seq_len, sample_stride=1, G: Optional[np.ndarray] = None,
                C: Optional[np.ndarray] = None, n_threads: int = 0):
    """Accumulate G += sum w x~ x~^T, C += sum w x~ y^T in fp64 over the
    multi-layer feature x~ = [x_0; ...; x_{k-1}; 1] (P = k d_s + 1), visiting
    the tokens t with t mod sample_stride == 0.  ``head_map["src_layers"]`` is
    [n_maps][k]; other conventions as in :func:`stats`.  Returns (G, C)."""
    lib = _load()
    n, k, hm = _multi_arrays(head_map)
    P = k * d_s + 1
    if G is None:
        G = np.zeros((n, P, P), dtype=np.float64)
    if C is None:
        C = np.zeros((n, P, d_t), dtype=np.float64)
    assert G.dtype == np.float64 and G.flags.c_contiguous and G.shape == (n, P, P)
    assert C.dtype == np.float64 and C.flags.c_contiguous and C.shape == (n, P, d_t)
    assert int(sample_stride) >= 1
    src = np.ascontiguousarray(_u16(src))
    tgt = np.ascontiguousarray(_u16(tgt))
    w = np.ascontiguousarray(np.asarray(weights, dtype=np.float32))
    ss, ts = _strides5(src_strides), _strides5(tgt_strides)
    lib.oracle_stats_multi(n, k, *[_ptr(a, _i32p) for a in hm], _ptr(src, _u16p), _ptr(ss, _i64p), d_s,
                           _ptr(tgt, _u16p), _ptr(ts, _i64p), d_t, _ptr(w, _f32p), int(w_row_stride),
                           int(n_seqs), int(seq_len), int(sample_stride), _ptr(G, _f64p), _ptr(C, _f64p),
                           int(n_threads))
    return G, C


def stats_multi_centered(head_map, src, src_strides, d_s, tgt, tgt_strides, d_t, weights, w_row_stride,
                         n_seqs, seq_len, sample_stride=1, n_threads: int = 0):
    """Two-pass centered moments over the multi-layer feature x = [x_0; ...; x_{k-1}]
    (width Dx = k d_s), tokens t with t mod sample_stride == 0: returns
    (sums [n][1 + Dx + d_t], A [n][Dx][Dx], B [n][Dx][d_t]) in fp64; solve them
    with :func:`ridge_solve_centered` (feature width Dx)."""
    lib = _load()
    n, k, hm = _multi_arrays(head_map)
    Dx = k * d_s
    sums = np.zeros((n, 1 + Dx + d_t), dtype=np.float64)
    A = np.zeros((n, Dx, Dx), dtype=np.float64)
    B = np.zeros((n, Dx, d_t), dtype=np.float64)
    assert int(sample_stride) >= 1
    src = np.ascontiguousarray(_u16(src))
    tgt = np.ascontiguousarray(_u16(tgt))
    w = np.ascontiguousarray(np.asarray(weights, dtype=np.float32))
    ss, ts = _strides5(src_strides), _strides5(tgt_strides)
    lib.oracle_stats_multi_centered(n, k, *[_ptr(a, _i32p) for a in hm], _ptr(src, _u16p), _ptr(ss, _i64p), d_s,
                                    _ptr(tgt, _u16p), _ptr(ts, _i64p), d_t, _ptr(w, _f32p), int(w_row_stride),
                                    int(n_seqs), int(seq_len), int(sample_stride), _ptr(sums, _f64p),
                                    _ptr(A, _f64p), _ptr(B, _f64p), int(n_threads))
    return sums, A, B


def apply_multi(head_map, W, src, src_strides, d_s, out, out_strides, d_t, n_seqs, seq_len,
                n_threads: int = 0):
    """Write RNE_bf16(x~ W~) for every multi-layer map and every token into ``out``."""
    lib = _load()
    n, k, hm = _multi_arrays(head_map, MULTI_MAP_FIELDS[:5])
    W = np.ascontiguousarray(np.asarray(W, dtype=np.float64))
    assert W.shape == (n, k * d_s + 1, d_t)
    src = np.ascontiguousarray(_u16(src))
    if not (out.dtype == np.uint16 and out.flags.c_contiguous):
        raise TypeError("out must be a C-contiguous uint16 array")
    ss, os_ = _strides5(src_strides), _strides5(out_strides)
    lib.oracle_apply_multi(n, k, *[_ptr(a, _i32p) for a in hm], _ptr(W, _f64p), _ptr(src, _u16p),
                           _ptr(ss, _i64p), d_s, _ptr(out, _u16p), _ptr(os_, _i64p), d_t,
                           int(n_seqs), int(seq_len), int(n_threads))
    return out


def apply_multi_rope(head_map, W, src, src_strides, d_s, out, out_strides, d_t, n_seqs, seq_len, theta: float,
                     style: int = 0, pos_offset: int = 0, n_threads: int = 0):
    """Like :func:`apply_multi`, with the K outputs turned by the target RoPE (fp64) before the one rounding."""
    lib = _load()
    n, k, hm = _multi_arrays(head_map, MULTI_MAP_FIELDS[:5])
    W = np.ascontiguousarray(np.asarray(W, dtype=np.float64))
    assert W.shape == (n, k * d_s + 1, d_t)
    src = np.ascontiguousarray(_u16(src))
    if not (out.dtype == np.uint16 and out.flags.c_contiguous):
        raise TypeError("out must be a C-contiguous uint16 array")
    ss, os_ = _strides5(src_strides), _strides5(out_strides)
    lib.oracle_apply_multi_rope(n, k, *[_ptr(a, _i32p) for a in hm], _ptr(W, _f64p), _ptr(src, _u16p),
                                _ptr(ss, _i64p), d_s, _ptr(out, _u16p), _ptr(os_, _i64p), d_t,
                                int(n_seqs), int(seq_len), float(theta), int(style), int(pos_offset),
                                int(n_threads))
    return out
