"""Python binding of libcachebridge (CacheBridge mapper path on MI355X / gfx950).

Argument marshalling only: every step of the path runs in the HIP kernels of
``libcachebridge.so`` behind the C ABI of ``include/cachebridge.h``.  torch
tensors are used only as device memory (``data_ptr``/``stride``) and for the
current HIP stream.  The functions keep the C names:

* :func:`cb_plan_create` / :func:`cb_plan_destroy`
* :func:`cb_stats_zero`, :func:`cb_stats_accumulate` -- augmented weighted moments
  G, C (CacheBridge Sec. 3.4, Eq. fusedstats)
* :func:`cb_ridge_solve` -- (G + lambda D)^-1 C (Sec. 3.1, Eq. closedform)
* :func:`cb_apply` -- online application of the maps (Sec. 1; Sec. 2.3)
* :func:`cb_stats_zero_centered`, :func:`cb_stats_means`,
  :func:`cb_stats_accumulate_centered`, :func:`cb_ridge_solve_centered` -- the
  two-pass centered form: weighted sums, centered moments A, B (Sec. 3.4) and
  W = (A + lambda I)^-1 B, b = mu_y - W^T mu_x (Sec. 3.1);
  :func:`cb_stats_accumulate_shifted`, :func:`cb_stats_shift_finish` -- the same
  moments in one pass over the data, formed about a pilot's means and moved to
  the data's own means at the end
* :func:`cb_probe_r2`, :func:`cb_select_layers` -- layer-selection probes: held-in
  R^2 per probe map and the top-k source layers per target layer (Sec. 3.1)
* :func:`cb_attn_sensitivity`, :func:`cb_attn_weights` -- attention-aligned
  calibration weights: raw sensitivities at causal prefix boundaries and the
  ESS-floor shrinkage (Sec. 3.3)
* :func:`cb_rope_table`, :func:`cb_rope` -- rotary position transform of cached
  keys (RoPE removed before fitting, restored after mapping; Sec. 2.1, 3.1);
  :func:`rope_spec` describes a table; :func:`cb_stats_accumulate_rope` folds
  the de-rotation into the statistics gather and :func:`cb_apply_rope` the
  de-rotation of the sender and the target's rotation into the mapping
* :func:`cb_plan_create_multi`, :func:`cb_ridge_solve_ws` -- maps over the
  multi-layer feature of k selected source layers (Sec. 3.2, Eq. localfeature)
  and the blocked solve of their P = k d_s + 1 systems

Caches are bfloat16 tensors indexed ``[layer][kv][seq][head][tok][dim]`` (any
strides with a unit channel stride).  Importing this package fails if the
library has not been built: there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
from typing import Mapping, Optional

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libcachebridge.so")

CB_LAMBDA_RELATIVE = 1
CB_RIDGE_BIAS_UNPENALIZED = 2
CB_ROPE_HALF_SPLIT = 0
CB_ROPE_INTERLEAVED = 1

STATUS_NAMES = {0: "CB_OK", 1: "CB_ERR_INVALID_ARGUMENT", 2: "CB_ERR_SHAPE", 3: "CB_ERR_MISALIGNED",
                4: "CB_ERR_OUT_OF_MEMORY", 5: "CB_ERR_DEVICE", 6: "CB_ERR_UNSUPPORTED"}

HEAD_MAP_FIELDS = ("tgt_layer", "tgt_head", "kv", "src_layer", "src_head", "weight_row")


class CbCache(ctypes.Structure):
    _fields_ = [("data", ctypes.c_void_p), ("n_layers", ctypes.c_int32), ("n_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("n_seqs", ctypes.c_int32), ("seq_len", ctypes.c_int32),
                ("s_layer", ctypes.c_int64), ("s_kv", ctypes.c_int64), ("s_seq", ctypes.c_int64),
                ("s_head", ctypes.c_int64), ("s_tok", ctypes.c_int64)]


_i32p = ctypes.POINTER(ctypes.c_int32)


class CbQueries(ctypes.Structure):
    _fields_ = [("data", ctypes.c_void_p), ("n_layers", ctypes.c_int32), ("n_qheads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("n_seqs", ctypes.c_int32), ("n_bounds", ctypes.c_int32),
                ("s_layer", ctypes.c_int64), ("s_seq", ctypes.c_int64), ("s_bnd", ctypes.c_int64),
                ("s_head", ctypes.c_int64)]


class CbHeadMap(ctypes.Structure):
    _fields_ = [("n_maps", ctypes.c_int32)] + [(f, _i32p) for f in HEAD_MAP_FIELDS]


MULTI_MAP_FIELDS = ("tgt_layer", "tgt_head", "kv", "src_layers", "src_head", "weight_row")


class CbHeadMapMulti(ctypes.Structure):
    _fields_ = [("n_maps", ctypes.c_int32), ("k", ctypes.c_int32)] + [(f, _i32p) for f in MULTI_MAP_FIELDS]


class CacheBridgeError(RuntimeError):
    def __init__(self, status: int, message: str):
        self.status = status
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {message}")


if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is missing: build it with `python -c 'import __graft_entry__ as g; g.build()'`")

_lib = ctypes.CDLL(LIB_PATH)
_vp = ctypes.c_void_p
_lib.cb_plan_create.restype = ctypes.c_int
_lib.cb_plan_create.argtypes = [ctypes.POINTER(CbHeadMap), ctypes.POINTER(CbCache), ctypes.POINTER(CbCache),
                                ctypes.c_int64, ctypes.POINTER(_vp)]
_lib.cb_plan_destroy.restype = ctypes.c_int
_lib.cb_plan_destroy.argtypes = [_vp]
_lib.cb_plan_create_multi.restype = ctypes.c_int
_lib.cb_plan_create_multi.argtypes = [ctypes.POINTER(CbHeadMapMulti), ctypes.POINTER(CbCache),
                                      ctypes.POINTER(CbCache), ctypes.c_int32, ctypes.POINTER(_vp)]
_lib.cb_plan_feature_width.restype = ctypes.c_int
_lib.cb_plan_feature_width.argtypes = [_vp, _i32p, _i32p]
_lib.cb_plan_shape.restype = ctypes.c_int
_lib.cb_plan_shape.argtypes = [_vp, _i32p, _i32p, _i32p]
_lib.cb_stats_zero.restype = ctypes.c_int
_lib.cb_stats_zero.argtypes = [_vp, _vp, _vp, _vp]
_lib.cb_stats_accumulate.restype = ctypes.c_int
_lib.cb_stats_accumulate.argtypes = [_vp, ctypes.POINTER(CbCache), ctypes.POINTER(CbCache), _vp, ctypes.c_int64,
                                     _vp, _vp, _vp]
_lib.cb_ridge_solve.restype = ctypes.c_int
_lib.cb_ridge_solve.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, _vp, _vp, ctypes.c_float,
                                ctypes.c_uint32, _vp, _vp, _vp]
_lib.cb_ridge_solve_ws.restype = ctypes.c_int
_lib.cb_ridge_solve_ws.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, _vp, _vp, ctypes.c_float,
                                   ctypes.c_uint32, _vp, ctypes.c_int64, _vp, _vp, _vp]
_lib.cb_ridge_solve_centered_ws.restype = ctypes.c_int
_lib.cb_ridge_solve_centered_ws.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, _vp, _vp, _vp,
                                            ctypes.c_float, ctypes.c_uint32, _vp, ctypes.c_int64, _vp, _vp, _vp]
_lib.cb_ridge_solve_noalloc.restype = ctypes.c_int
_lib.cb_ridge_solve_noalloc.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, _vp, _vp, ctypes.c_float,
                                        ctypes.c_uint32, _vp, _vp, _vp]
_lib.cb_ridge_solve_noalloc_max_bytes.restype = ctypes.c_int64
_lib.cb_ridge_solve_noalloc_max_bytes.argtypes = []
_lib.cb_ridge_solve_workspace_bytes.restype = ctypes.c_int64
_lib.cb_ridge_solve_workspace_bytes.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_int32]
_lib.cb_stats_zero_centered.restype = ctypes.c_int
_lib.cb_stats_zero_centered.argtypes = [_vp, _vp, _vp, _vp, _vp, _vp]
_lib.cb_stats_means.restype = ctypes.c_int
_lib.cb_stats_means.argtypes = [_vp, ctypes.POINTER(CbCache), ctypes.POINTER(CbCache), _vp, ctypes.c_int64, _vp, _vp,
                                _vp]
_lib.cb_probe_r2.restype = ctypes.c_int
_lib.cb_probe_r2.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, _vp, _vp, _vp, _vp, _vp, _vp, _vp]
_lib.cb_select_layers.restype = ctypes.c_int
_lib.cb_select_layers.argtypes = [ctypes.POINTER(CbHeadMap), _vp, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                  _vp, _vp]
_lib.cb_stats_accumulate_centered.restype = ctypes.c_int
_lib.cb_stats_accumulate_centered.argtypes = [_vp, ctypes.POINTER(CbCache), ctypes.POINTER(CbCache), _vp,
                                              ctypes.c_int64, _vp, _vp, _vp, _vp]
_lib.cb_stats_accumulate_shifted.restype = ctypes.c_int
_lib.cb_stats_accumulate_shifted.argtypes = [_vp, ctypes.POINTER(CbCache), ctypes.POINTER(CbCache), _vp,
                                             ctypes.c_int64, _vp, _vp, _vp, _vp, _vp]
_lib.cb_stats_shift_finish.restype = ctypes.c_int
_lib.cb_stats_shift_finish.argtypes = [_vp, _vp, _vp, _vp, _vp, _vp]
_lib.cb_ridge_solve_centered.restype = ctypes.c_int
_lib.cb_ridge_solve_centered.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, _vp, _vp, _vp,
                                         ctypes.c_float, ctypes.c_uint32, _vp, _vp, _vp]
_lib.cb_attn_sensitivity.restype = ctypes.c_int
_lib.cb_attn_sensitivity.argtypes = [ctypes.POINTER(CbCache), ctypes.POINTER(CbQueries), _vp, ctypes.c_int32, _vp,
                                     ctypes.c_int64, _vp]
_lib.cb_attn_weights.restype = ctypes.c_int
_lib.cb_attn_weights.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, _vp, ctypes.c_int64,
                                 ctypes.c_int32, _vp, ctypes.c_int64, _vp, _vp]
_lib.cb_rope_table.restype = ctypes.c_int
_lib.cb_rope_table.argtypes = [ctypes.c_double, ctypes.c_int32, ctypes.c_int32, _vp, _vp]


class CbRopeSpec(ctypes.Structure):
    _fields_ = [("table", _vp), ("head_dim", ctypes.c_int32), ("n_pos", ctypes.c_int32),
                ("style", ctypes.c_int32), ("pos_offset", ctypes.c_int32)]


_rsp = ctypes.POINTER(CbRopeSpec)
_lib.cb_rope.restype = ctypes.c_int
_lib.cb_rope.argtypes = [ctypes.POINTER(CbCache), ctypes.POINTER(CbCache), _rsp, ctypes.c_int32, _vp]
_lib.cb_apply.restype = ctypes.c_int
_lib.cb_apply.argtypes = [_vp, _vp, ctypes.POINTER(CbCache), ctypes.POINTER(CbCache), _vp]
_lib.cb_apply_rope.restype = ctypes.c_int
_lib.cb_apply_rope.argtypes = [_vp, _vp, ctypes.POINTER(CbCache), ctypes.POINTER(CbCache), _rsp, _rsp, _vp]
_lib.cb_stats_accumulate_rope.restype = ctypes.c_int
_lib.cb_stats_accumulate_rope.argtypes = [_vp, ctypes.POINTER(CbCache), ctypes.POINTER(CbCache), _vp, ctypes.c_int64,
                                          _vp, _vp, _rsp, _rsp, _vp]
_lib.cb_status_string.restype = ctypes.c_char_p
_lib.cb_status_string.argtypes = [ctypes.c_int]
_lib.cb_last_error.restype = ctypes.c_char_p
_lib.cb_last_error.argtypes = []


def library() -> ctypes.CDLL:
    """The loaded libcachebridge handle."""
    return _lib


def cb_status_string(status: int) -> str:
    return _lib.cb_status_string(int(status)).decode()


def cb_last_error() -> str:
    return _lib.cb_last_error().decode()


def _check(status: int):
    if status != 0:
        raise CacheBridgeError(status, cb_last_error())


def _stream(stream) -> Optional[int]:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream if torch.cuda.is_available() else None
    if isinstance(stream, torch.cuda.Stream):
        return stream.cuda_stream
    return int(stream)


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else t.data_ptr()


def _need(t: Optional[torch.Tensor], shape, dtype, name: str):
    """The library writes (or reads) exactly prod(shape) dense elements at t's
    address: check that t holds them."""
    if t is None:
        raise ValueError(f"{name} is required")
    if t.dtype != dtype or tuple(t.shape) != tuple(shape) or not t.is_contiguous():
        raise ValueError(f"{name} must be a contiguous {dtype} tensor of shape {tuple(shape)}, "
                         f"got {t.dtype} {tuple(t.shape)}")


def _check_weights(plan: "Plan", weights: torch.Tensor, row_stride: int, src: torch.Tensor):
    """Every weight the kernels read, w[row * row_stride + seq * T + tok], lies inside
    ``weights``' storage (a row stride shorter than a row is the library's own
    CB_ERR_SHAPE)."""
    if weights.dtype != torch.float32:
        raise ValueError("weights are float32")
    n_tok = src.shape[2] * src.shape[4]
    if plan.n_weight_rows == 0 or n_tok == 0 or row_stride < n_tok:
        return
    if weights.numel() > 1 and weights.stride(-1) != 1:
        raise ValueError("weights rows must be dense")
    if weights.dim() == 2 and weights.shape[0] < plan.n_weight_rows:
        raise ValueError(f"weights must have at least {plan.n_weight_rows} rows")
    need = (plan.n_weight_rows - 1) * row_stride + n_tok
    have = weights.untyped_storage().nbytes() // 4 - weights.storage_offset()
    if have < need:
        raise ValueError(f"weights must hold {need} float32 values from their first element")


def cache_view(t: Optional[torch.Tensor], n_layers=None, n_heads=None, head_dim=None) -> CbCache:
    """Describe a [layer][kv][seq][head][tok][dim] bfloat16 tensor (any strides, unit channel stride)."""
    c = CbCache()
    if t is None:
        c.n_layers, c.n_heads, c.head_dim = n_layers, n_heads, head_dim
        return c
    if t.dtype != torch.bfloat16 or t.dim() != 6 or t.shape[1] != 2:
        raise ValueError("cache tensors are bfloat16 [layer][2][seq][head][tok][dim]")
    if t.shape[5] > 1 and t.stride(5) != 1:
        raise ValueError("cache channel stride must be 1")
    L, _, B, H, T, d = t.shape
    c.data = t.data_ptr()
    c.n_layers, c.n_heads, c.head_dim, c.n_seqs, c.seq_len = L, H, d, B, T
    c.s_layer, c.s_kv, c.s_seq, c.s_head, c.s_tok = t.stride(0), t.stride(1), t.stride(2), t.stride(3), t.stride(4)
    return c


class Plan:
    """Owning handle of a cb_plan (validated head map, gather schedule, workspace)."""

    def __init__(self, handle: int, n_maps: int, d_s: int, d_t: int, keep, P: Optional[int] = None, k: int = 1):
        self.handle = handle
        self.n_maps, self.d_s, self.d_t = n_maps, d_s, d_t
        self.P = d_s + 1 if P is None else P
        self.k = k
        self._keep = keep
        wr = keep[-1]                                  # weight_row is the last head-map field
        self.n_weight_rows = int(wr.max()) + 1 if wr.size else 0

    def close(self):
        if self.handle:
            _check(_lib.cb_plan_destroy(self.handle))
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def cb_plan_create(head_map: Mapping[str, object], src_geom, tgt_geom, max_tokens_per_call: int) -> Plan:
    """Compile ``head_map`` (six int arrays) for source/target geometries given as
    ``(n_layers, n_heads, head_dim)`` tuples or cache tensors."""
    import numpy as np  # noqa: PLC0415

    arrays = [np.ascontiguousarray(np.asarray(head_map[f], dtype=np.int32)) for f in HEAD_MAP_FIELDS]
    n = arrays[0].shape[0]
    hm = CbHeadMap()
    hm.n_maps = n
    for f, a in zip(HEAD_MAP_FIELDS, arrays):
        setattr(hm, f, a.ctypes.data_as(_i32p))

    def geom(g):
        if isinstance(g, torch.Tensor):
            return cache_view(g)
        return cache_view(None, *g)

    sg, tg = geom(src_geom), geom(tgt_geom)
    out = _vp()
    _check(_lib.cb_plan_create(ctypes.byref(hm), ctypes.byref(sg), ctypes.byref(tg), int(max_tokens_per_call),
                               ctypes.byref(out)))
    nm, ds, dt = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int32()
    _check(_lib.cb_plan_shape(out.value, ctypes.byref(nm), ctypes.byref(ds), ctypes.byref(dt)))
    return Plan(out.value, nm.value, ds.value, dt.value, arrays)


def cb_plan_create_multi(head_map: Mapping[str, object], src_geom, tgt_geom, sample_stride: int = 1) -> Plan:
    """Compile a multi-layer head map (``src_layers`` is [n_maps][k]; the other
    five fields as in :func:`cb_plan_create`).  Calibration rows are the tokens
    ``tok % sample_stride == 0``."""
    import numpy as np  # noqa: PLC0415

    arrays = [np.ascontiguousarray(np.asarray(head_map[f], dtype=np.int32)) for f in MULTI_MAP_FIELDS]
    n = arrays[0].shape[0]
    S = arrays[MULTI_MAP_FIELDS.index("src_layers")]
    if S.ndim != 2 or S.shape[0] != n:
        raise ValueError("src_layers must be [n_maps][k]")
    hm = CbHeadMapMulti()
    hm.n_maps, hm.k = n, S.shape[1]
    for f, a in zip(MULTI_MAP_FIELDS, arrays):
        setattr(hm, f, a.ctypes.data_as(_i32p))

    def geom(g):
        if isinstance(g, torch.Tensor):
            return cache_view(g)
        return cache_view(None, *g)

    sg, tg = geom(src_geom), geom(tgt_geom)
    out = _vp()
    _check(_lib.cb_plan_create_multi(ctypes.byref(hm), ctypes.byref(sg), ctypes.byref(tg), int(sample_stride),
                                     ctypes.byref(out)))
    nm, ds, dt = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int32()
    _check(_lib.cb_plan_shape(out.value, ctypes.byref(nm), ctypes.byref(ds), ctypes.byref(dt)))
    P, k = ctypes.c_int32(), ctypes.c_int32()
    _check(_lib.cb_plan_feature_width(out.value, ctypes.byref(P), ctypes.byref(k)))
    return Plan(out.value, nm.value, ds.value, dt.value, arrays, P=P.value, k=k.value)


def cb_plan_destroy(plan: Plan):
    plan.close()


def cb_stats_zero(plan: Plan, G: torch.Tensor, C: torch.Tensor, stream=None):
    _need(G, (plan.n_maps, plan.P, plan.P), torch.float32, "G")
    _need(C, (plan.n_maps, plan.P, plan.d_t), torch.float32, "C")
    _check(_lib.cb_stats_zero(plan.handle, _ptr(G), _ptr(C), _stream(stream)))


def cb_stats_accumulate(plan: Plan, src: torch.Tensor, tgt: torch.Tensor, weights: torch.Tensor,
                        G: torch.Tensor, C: torch.Tensor, w_row_stride: Optional[int] = None, stream=None):
    """G[m] += sum_t w x~ x~^T, C[m] += sum_t w x~ y^T over the batch (fp32 outputs)."""
    _need(G, (plan.n_maps, plan.P, plan.P), torch.float32, "G")
    _need(C, (plan.n_maps, plan.P, plan.d_t), torch.float32, "C")
    if w_row_stride is None:
        w_row_stride = weights.stride(0) if weights.dim() == 2 else weights.numel()
    _check_weights(plan, weights, int(w_row_stride), src)
    sv, tv = cache_view(src), cache_view(tgt)
    _check(_lib.cb_stats_accumulate(plan.handle, ctypes.byref(sv), ctypes.byref(tv), _ptr(weights),
                                    int(w_row_stride), _ptr(G), _ptr(C), _stream(stream)))


def cb_ridge_solve(G: torch.Tensor, C: torch.Tensor, lam: float, flags: int, maps: torch.Tensor,
                   info: torch.Tensor, stream=None):
    """maps[m] = (G[m] + lambda_m D)^-1 C[m]; info[m] = 0 or the first failing pivot (1-based)."""
    n, P, P2 = G.shape
    if P != P2 or C.shape[:2] != (n, P) or maps.shape != C.shape or info.shape != (n,):
        raise ValueError("G [n][P][P], C/maps [n][P][d_t], info [n]")
    if info.dtype != torch.int32:
        raise ValueError("info is int32")
    _check(_lib.cb_ridge_solve(n, P, C.shape[2], _ptr(G), _ptr(C), float(lam), int(flags), _ptr(maps), _ptr(info),
                               _stream(stream)))


def cb_ridge_solve_workspace_bytes(P: int, d_t: int, n_systems: int) -> int:
    """Workspace bytes :func:`cb_ridge_solve_ws` needs for n_systems systems at once (0 if P <= 129)."""
    return int(_lib.cb_ridge_solve_workspace_bytes(int(P), int(d_t), int(n_systems)))


def cb_ridge_solve_ws(G: torch.Tensor, C: torch.Tensor, lam: float, flags: int, maps: torch.Tensor,
                      info: torch.Tensor, workspace: Optional[torch.Tensor], stream=None):
    """maps[m] = (G[m] + lambda_m D)^-1 C[m] for any P; the blocked fp64 solve (P > 129)
    factors in ``workspace`` (a device tensor of at least cb_ridge_solve_workspace_bytes(P, d_t, 1) bytes)."""
    n, P, P2 = G.shape
    if P != P2 or C.shape[:2] != (n, P) or maps.shape != C.shape or info.shape != (n,):
        raise ValueError("G [n][P][P], C/maps [n][P][d_t], info [n]")
    if info.dtype != torch.int32:
        raise ValueError("info is int32")
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(_lib.cb_ridge_solve_ws(n, P, C.shape[2], _ptr(G), _ptr(C), float(lam), int(flags), _ptr(workspace),
                                  int(ws_bytes), _ptr(maps), _ptr(info), _stream(stream)))


def cb_ridge_solve_noalloc(G: torch.Tensor, C: torch.Tensor, lam: float, flags: int, maps: torch.Tensor,
                           info: torch.Tensor, stream=None):
    """cb_ridge_solve_ws without a workspace: the library's fixed device scratch array
    (cb_ridge_solve_noalloc_max_bytes()) holds the factors; nothing is allocated."""
    n, P, P2 = G.shape
    if P != P2 or C.shape[:2] != (n, P) or maps.shape != C.shape or info.shape != (n,):
        raise ValueError("G [n][P][P], C/maps [n][P][d_t], info [n]")
    if info.dtype != torch.int32:
        raise ValueError("info is int32")
    _check(_lib.cb_ridge_solve_noalloc(n, P, C.shape[2], _ptr(G), _ptr(C), float(lam), int(flags), _ptr(maps),
                                       _ptr(info), _stream(stream)))


def cb_ridge_solve_noalloc_max_bytes() -> int:
    return int(_lib.cb_ridge_solve_noalloc_max_bytes())


def _row_stride(weights: torch.Tensor, w_row_stride: Optional[int]) -> int:
    if w_row_stride is not None:
        return int(w_row_stride)
    return weights.stride(0) if weights.dim() == 2 else weights.numel()


def _need_centered(plan: Plan, sums, A, B, sq):
    n, Dx, dt = plan.n_maps, plan.P - 1, plan.d_t
    _need(sums, (n, 1 + Dx + dt), torch.float64, "sums")
    if A is not None:
        _need(A, (n, Dx, Dx), torch.float32, "A")
    if B is not None:
        _need(B, (n, Dx, dt), torch.float32, "B")
    if sq is not None:
        _need(sq, (n, Dx + dt), torch.float64, "sq")


def cb_stats_zero_centered(plan: Plan, sums: torch.Tensor, A: torch.Tensor, B: torch.Tensor,
                           sq: Optional[torch.Tensor] = None, stream=None):
    """Zero sums [n][1 + d_x + d_t] (float64), A [n][d_x][d_x], B [n][d_x][d_t] (float32)
    and, if given (single-layer plans), sq [n][d_s + d_t] (float64); d_x = d_s, or k d_s
    for a multi-layer plan."""
    _need_centered(plan, sums, A, B, sq)
    _check(_lib.cb_stats_zero_centered(plan.handle, _ptr(sums), _ptr(sq), _ptr(A), _ptr(B), _stream(stream)))


def cb_stats_means(plan: Plan, src: torch.Tensor, tgt: torch.Tensor, weights: torch.Tensor, sums: torch.Tensor,
                   sq: Optional[torch.Tensor] = None, w_row_stride: Optional[int] = None, stream=None):
    """Pass 1: sums[m] += (sum w, sum w x, sum w y) and, if given, sq[m] += (sum w x^2, sum w y^2)
    over the batch (float64)."""
    _need_centered(plan, sums, None, None, sq)
    rs = _row_stride(weights, w_row_stride)
    _check_weights(plan, weights, rs, src)
    sv, tv = cache_view(src), cache_view(tgt)
    _check(_lib.cb_stats_means(plan.handle, ctypes.byref(sv), ctypes.byref(tv), _ptr(weights), rs, _ptr(sums), _ptr(sq), _stream(stream)))


def cb_stats_accumulate_centered(plan: Plan, src: torch.Tensor, tgt: torch.Tensor, weights: torch.Tensor,
                                 sums: torch.Tensor, A: torch.Tensor, B: torch.Tensor,
                                 w_row_stride: Optional[int] = None, stream=None):
    """Pass 2: A[m] += sum w (x - mu_x)(x - mu_x)^T, B[m] += sum w (x - mu_x)(y - mu_y)^T."""
    _need_centered(plan, sums, A, B, None)
    rs = _row_stride(weights, w_row_stride)
    _check_weights(plan, weights, rs, src)
    sv, tv = cache_view(src), cache_view(tgt)
    _check(_lib.cb_stats_accumulate_centered(plan.handle, ctypes.byref(sv), ctypes.byref(tv), _ptr(weights), rs, _ptr(sums), _ptr(A), _ptr(B),
                                             _stream(stream)))


def cb_stats_accumulate_shifted(plan: Plan, src: torch.Tensor, tgt: torch.Tensor, weights: torch.Tensor,
                                shift: torch.Tensor, sums: torch.Tensor, A: torch.Tensor, B: torch.Tensor,
                                w_row_stride: Optional[int] = None, stream=None):
    """One-pass centered moments: A[m] += sum w (x - mu'_x)(x - mu'_x)^T, B[m] += sum w (x - mu'_x)(y - mu'_y)^T
    about the means mu' of ``shift`` (a pilot's sums from :func:`cb_stats_means`), and sums[m] +=
    (sum w, sum w (x - mu'_x), sum w y); :func:`cb_stats_shift_finish` completes them."""
    _need_centered(plan, shift, None, None, None)
    _need_centered(plan, sums, A, B, None)
    rs = _row_stride(weights, w_row_stride)
    _check_weights(plan, weights, rs, src)
    sv, tv = cache_view(src), cache_view(tgt)
    _check(_lib.cb_stats_accumulate_shifted(plan.handle, ctypes.byref(sv), ctypes.byref(tv), _ptr(weights), rs,
                                            _ptr(shift), _ptr(sums), _ptr(A), _ptr(B), _stream(stream)))


def cb_stats_shift_finish(plan: Plan, shift: torch.Tensor, sums: torch.Tensor, A: torch.Tensor, B: torch.Tensor,
                          stream=None):
    """Moves A, B from the pilot's means to the data's (A -= S d d^T, B -= S d (mu_y - mu'_y)^T, d = mu - mu')
    and turns sums into (sum w, sum w x, sum w y): then they are those of the two-pass form."""
    _need_centered(plan, shift, None, None, None)
    _need_centered(plan, sums, A, B, None)
    _check(_lib.cb_stats_shift_finish(plan.handle, _ptr(shift), _ptr(sums), _ptr(A), _ptr(B), _stream(stream)))


def cb_ridge_solve_centered(sums: torch.Tensor, A: torch.Tensor, B: torch.Tensor, lam: float, flags: int,
                            maps: torch.Tensor, info: torch.Tensor, stream=None):
    """maps[m] = [W; b^T] with W = (A[m] + lambda_m I)^-1 B[m] and b = mu_y - W^T mu_x."""
    n, d_s, d_s2 = A.shape
    d_t = B.shape[2] if B.dim() == 3 else -1
    if d_s != d_s2 or B.shape[:2] != (n, d_s) or sums.shape != (n, 1 + d_s + d_t) \
            or maps.shape != (n, d_s + 1, d_t) or info.shape != (n,):
        raise ValueError("sums [n][1+d_s+d_t], A [n][d_s][d_s], B [n][d_s][d_t], maps [n][d_s+1][d_t], info [n]")
    if sums.dtype != torch.float64 or info.dtype != torch.int32:
        raise ValueError("sums is float64, info int32")
    _check(_lib.cb_ridge_solve_centered(n, d_s, d_t, _ptr(sums), _ptr(A), _ptr(B), float(lam), int(flags),
                                        _ptr(maps), _ptr(info), _stream(stream)))


def cb_ridge_solve_centered_ws(sums: torch.Tensor, A: torch.Tensor, B: torch.Tensor, lam: float, flags: int,
                               maps: torch.Tensor, info: torch.Tensor, workspace: Optional[torch.Tensor],
                               stream=None):
    """The centered solve for any feature width d_x (the multi-layer feature: d_x = k d_s):
    maps[m] = [W; b^T]; d_x > 128 factors in ``workspace`` (at least
    cb_ridge_solve_workspace_bytes(d_x, d_t, 1) bytes)."""
    n, d_x, d_x2 = A.shape
    d_t = B.shape[2] if B.dim() == 3 else -1
    if d_x != d_x2 or B.shape[:2] != (n, d_x) or sums.shape != (n, 1 + d_x + d_t) \
            or maps.shape != (n, d_x + 1, d_t) or info.shape != (n,):
        raise ValueError("sums [n][1+d_x+d_t], A [n][d_x][d_x], B [n][d_x][d_t], maps [n][d_x+1][d_t], info [n]")
    if sums.dtype != torch.float64 or info.dtype != torch.int32:
        raise ValueError("sums is float64, info int32")
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(_lib.cb_ridge_solve_centered_ws(n, d_x, d_t, _ptr(sums), _ptr(A), _ptr(B), float(lam), int(flags),
                                           _ptr(workspace), int(ws_bytes), _ptr(maps), _ptr(info), _stream(stream)))


def cb_probe_r2(sums: torch.Tensor, sq: torch.Tensor, A: torch.Tensor, B: torch.Tensor, maps: torch.Tensor,
                r2: torch.Tensor, stream=None):
    """r2[m] = 1 - RSS/TSS of the fitted probe maps[m] on its calibration data (float64)."""
    n, d_s, _ = A.shape
    d_t = B.shape[2]
    if sums.shape != (n, 1 + d_s + d_t) or sq.shape != (n, d_s + d_t) or B.shape != (n, d_s, d_t) \
            or maps.shape != (n, d_s + 1, d_t) or r2.shape != (n,):
        raise ValueError("sums [n][1+d_s+d_t], sq [n][d_s+d_t], A [n][d_s][d_s], B [n][d_s][d_t], "
                         "maps [n][d_s+1][d_t], r2 [n]")
    if sums.dtype != torch.float64 or sq.dtype != torch.float64 or r2.dtype != torch.float64:
        raise ValueError("sums, sq and r2 are float64")
    _check(_lib.cb_probe_r2(n, d_s, d_t, _ptr(sums), _ptr(sq), _ptr(A), _ptr(B), _ptr(maps), _ptr(r2),
                            _stream(stream)))


def cb_select_layers(head_map: Mapping[str, object], r2, n_tgt_layers: int, n_src_layers: int, k: int):
    """Host layer selection: returns (selected [L_t][k] int32, score [L_t][L_s] float64) as numpy arrays."""
    import numpy as np  # noqa: PLC0415

    tl = np.ascontiguousarray(np.asarray(head_map["tgt_layer"], dtype=np.int32))
    sl = np.ascontiguousarray(np.asarray(head_map["src_layer"], dtype=np.int32))
    r = np.ascontiguousarray(np.asarray(r2.cpu() if isinstance(r2, torch.Tensor) else r2, dtype=np.float64))
    hm = CbHeadMap()
    hm.n_maps = tl.shape[0]
    hm.tgt_layer = tl.ctypes.data_as(_i32p)
    hm.src_layer = sl.ctypes.data_as(_i32p)
    selected = np.zeros((n_tgt_layers, k), dtype=np.int32)
    score = np.zeros((n_tgt_layers, n_src_layers), dtype=np.float64)
    _check(_lib.cb_select_layers(ctypes.byref(hm), r.ctypes.data, n_tgt_layers, n_src_layers, k,
                                 selected.ctypes.data, score.ctypes.data))
    return selected, score


def queries_view(q: torch.Tensor) -> CbQueries:
    """Describe a [layer][seq][boundary][query head][dim] bfloat16 tensor (unit dim stride)."""
    if q.dtype != torch.bfloat16 or q.dim() != 5 or (q.shape[4] > 1 and q.stride(4) != 1):
        raise ValueError("queries are bfloat16 [layer][seq][boundary][query head][dim] with unit dim stride")
    v = CbQueries()
    v.data = q.data_ptr()
    v.n_layers, v.n_seqs, v.n_bounds, v.n_qheads, v.head_dim = q.shape
    v.s_layer, v.s_seq, v.s_bnd, v.s_head = q.stride(0), q.stride(1), q.stride(2), q.stride(3)
    return v


def cb_attn_sensitivity(tgt: torch.Tensor, q: torch.Tensor, boundaries, sample_stride: int, r: torch.Tensor,
                        r_row_stride: Optional[int] = None, stream=None):
    """Raw sensitivities into r [(l*2 + z)*H + h][seq*seq_len + tok] (float32; z = 0 K, 1 V)."""
    import numpy as np  # noqa: PLC0415

    if r.dtype != torch.float32:
        raise ValueError("r is float32")
    b = np.ascontiguousarray(np.asarray(boundaries, dtype=np.int32))
    tv, qv = cache_view(tgt), queries_view(q)
    rs = r.stride(0) if r_row_stride is None else int(r_row_stride)
    _check(_lib.cb_attn_sensitivity(ctypes.byref(tv), ctypes.byref(qv), b.ctypes.data, int(sample_stride), _ptr(r),
                                    rs, _stream(stream)))


def cb_attn_weights(r: torch.Tensor, n_seqs: int, seq_len: int, sample_stride: int, p: int, w: torch.Tensor,
                    alpha: torch.Tensor, stream=None):
    """w = 1 + alpha (r/mean - 1) on calibration rows, 0 elsewhere; alpha per row (float32)."""
    if r.dtype != torch.float32 or w.dtype != torch.float32 or alpha.dtype != torch.float32:
        raise ValueError("r, w and alpha are float32")
    n_rows = r.shape[0]
    if w.shape[0] != n_rows or alpha.shape != (n_rows,):
        raise ValueError("r, w [rows][...], alpha [rows]")
    _check(_lib.cb_attn_weights(n_rows, int(n_seqs), int(seq_len), int(sample_stride), _ptr(r), r.stride(0), int(p),
                                _ptr(w), w.stride(0), _ptr(alpha), _stream(stream)))


def cb_rope_table(theta: float, head_dim: int, n_pos: int, table: torch.Tensor, stream=None):
    """table [n_pos][head_dim/2][2] float32 = (cos, sin)(pos * theta^(-2i/d))."""
    if table.dtype != torch.float32 or table.numel() < n_pos * head_dim:
        raise ValueError("table is float32 with n_pos * head_dim elements")
    _check(_lib.cb_rope_table(float(theta), int(head_dim), int(n_pos), _ptr(table), _stream(stream)))


def rope_spec(table: torch.Tensor, style: int = CB_ROPE_HALF_SPLIT, pos_offset: int = 0) -> CbRopeSpec:
    """Describe a cb_rope_table output: ``table`` is float32 [n_pos][head_dim/2][2] (its
    shape gives head_dim and n_pos, which the library checks against each call)."""
    if table.dtype != torch.float32 or table.dim() != 3 or table.shape[2] != 2 or not table.is_contiguous():
        raise ValueError("a rope table is a contiguous float32 [n_pos][head_dim/2][2] tensor")
    sp = CbRopeSpec()
    sp.table, sp.head_dim, sp.n_pos = table.data_ptr(), 2 * table.shape[1], table.shape[0]
    sp.style, sp.pos_offset = int(style), int(pos_offset)
    sp._keep = table
    return sp


def _spec(r) -> Optional[CbRopeSpec]:
    if r is None or isinstance(r, CbRopeSpec):
        return r
    return rope_spec(r)


def cb_rope(cache_in: torch.Tensor, cache_out: torch.Tensor, table: torch.Tensor, style: int = CB_ROPE_HALF_SPLIT,
            inverse: bool = False, pos_offset: int = 0, stream=None):
    """Rotate (inverse: de-rotate) the K rows of a cache into cache_out (may be cache_in); V rows copied."""
    sp = rope_spec(table, style, pos_offset)
    iv, ov = cache_view(cache_in), cache_view(cache_out)
    _check(_lib.cb_rope(ctypes.byref(iv), ctypes.byref(ov), ctypes.byref(sp), int(bool(inverse)), _stream(stream)))


def cb_apply(plan: Plan, maps: torch.Tensor, src: torch.Tensor, tgt_out: torch.Tensor, stream=None):
    """tgt_out[l, z, b, h, t, :] = RNE_bf16([x, 1] maps[m]) for every map and token."""
    _need(maps, (plan.n_maps, plan.P, plan.d_t), torch.float32, "maps")
    sv, ov = cache_view(src), cache_view(tgt_out)
    _check(_lib.cb_apply(plan.handle, _ptr(maps), ctypes.byref(sv), ctypes.byref(ov), _stream(stream)))


def cb_apply_rope(plan: Plan, maps: torch.Tensor, src: torch.Tensor, tgt_out: torch.Tensor, tgt_rope=None,
                  src_rope=None, stream=None):
    """cb_apply with the rotary transforms fused: ``src_rope`` turns the sender's K rows back as they are read,
    ``tgt_rope`` turns the K outputs in fp32 before their single rounding.  Each is a :func:`rope_spec`
    (or a table, for style 0 at offset 0) or None."""
    _need(maps, (plan.n_maps, plan.P, plan.d_t), torch.float32, "maps")
    tr, sr = _spec(tgt_rope), _spec(src_rope)
    sv, ov = cache_view(src), cache_view(tgt_out)
    _check(_lib.cb_apply_rope(plan.handle, _ptr(maps), ctypes.byref(sv), ctypes.byref(ov),
                              None if sr is None else ctypes.byref(sr), None if tr is None else ctypes.byref(tr),
                              _stream(stream)))


def cb_stats_accumulate_rope(plan: Plan, src: torch.Tensor, tgt: torch.Tensor, weights: torch.Tensor,
                             G: torch.Tensor, C: torch.Tensor, src_rope=None, tgt_rope=None,
                             w_row_stride: Optional[int] = None, stream=None):
    """cb_stats_accumulate on keys that carry RoPE: the K rows of the source (src_rope) and of the target
    (tgt_rope) are turned back as they are gathered, exactly as cb_rope(inverse) would write them."""
    _need(G, (plan.n_maps, plan.P, plan.P), torch.float32, "G")
    _need(C, (plan.n_maps, plan.P, plan.d_t), torch.float32, "C")
    if w_row_stride is None:
        w_row_stride = weights.stride(0) if weights.dim() == 2 else weights.numel()
    _check_weights(plan, weights, int(w_row_stride), src)
    sr, tr = _spec(src_rope), _spec(tgt_rope)
    sv, tv = cache_view(src), cache_view(tgt)
    _check(_lib.cb_stats_accumulate_rope(plan.handle, ctypes.byref(sv), ctypes.byref(tv), _ptr(weights),
                                         int(w_row_stride), _ptr(G), _ptr(C),
                                         None if sr is None else ctypes.byref(sr),
                                         None if tr is None else ctypes.byref(tr), _stream(stream)))
