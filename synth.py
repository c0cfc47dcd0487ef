"""Seeded synthetic workloads for the CacheBridge mapper path.

This module only *generates inputs*: KV-cache-shaped tensors, calibration
weights, head maps and planted affine maps.  It holds none of the method's
arithmetic (no moments, no solve, no application) and is shared by the tests,
the benchmark and the oracle checks, which is its only role.

The real inputs of the paper (Qwen3 14B/32B traces over FineWeb-Edu, Sec. 4.1)
are not available; these stand-ins take the paper's shapes (8 KV heads x 128
dims, a 64-layer target, fp32 maps) and the structure each workload below names.

Workloads (``WORKLOADS``):

* ``tiny``  -- src 1x2x64, tgt 1x2x64, identity head map, 4 seqs x 256 tokens,
  x ~ N(0,1), y = xA + b + 0.05 N(0,1), w ~ lognormal(0,1) mean-one.
* ``qwen50`` -- Qwen3-14B->32B-shaped: src 40x8x128, tgt 64x8x128, 1024 maps,
  src_layer = round(l*39/63), same head; 50 seqs x 2048 tokens; per-channel
  lognormal(0,1) scales with 4 outlier channels x20; y = xA + b + 0.1 N(0,1);
  weights = causal-attention column mass of Gaussian q, k with a position-0
  sink (logit bonus 4 on key 0), mean-one.
* ``qwen500`` -- as ``qwen50`` with 500 seqs, streamed as 5 batches of 100.
* ``mismatch`` -- src 26x8x96, tgt 40x4x128, src_head = 2h,
  src_layer = round(l*25/39); 200 seqs x 4096 tokens; w = exp(2z)/sqrt(t+1)
  mean-one.
* ``tiny_k3`` -- multi-layer feature, k = 3: src 4x2x128, tgt 3x2x128,
  S_l = 3 consecutive source layers (``window``), 4 seqs x 520 tokens, every
  fourth token a calibration row (520 rows > P = 385; ragged tiles).
* ``qwen_k8`` -- the paper's Qwen3-14B->32B construction shape: k = 8
  (P = 1025), 500 seqs x 1024 tokens, every fourth token (128,000 rows),
  streamed as 5 batches of 100; sources and weights as ``qwen50``.
* ``apply`` -- maps [1024][129][128] fp32 (planted, ``qwen`` statistics) applied
  to a sender cache of 8 x 32768 tokens x 40 layers x 8 heads x 128.

Source kinds: ``gauss`` x ~ N(0,1); ``scaled`` x = s_c z (per-channel lognormal
scales s_c with outliers); ``offset`` x = mu_c + s_c z with per-channel means
mu_c = 30 s_c u_c, u_c ~ N(0,1) (channels whose mean dwarfs their spread, as
in the large-magnitude key channels of real caches).

Cache layout everywhere: ``[layer][kv][seq][head][tok][dim]`` bfloat16.
Weights: fp32 ``[row][seq * seq_len + tok]``; row = tgt_layer * H_t + tgt_head
(one row per target head, shared by K and V).  Map order:
``m = (tgt_layer * 2 + kv) * H_t + tgt_head``.

Seeding: master seed 0; every draw has its own generator keyed by
(workload, tensor, indices), so results do not depend on chunking.
"""
from __future__ import annotations

import dataclasses
import hashlib
import math
from typing import Dict, Optional

import numpy as np
import torch

MASTER_SEED = 0


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    L_s: int
    H_s: int
    d_s: int
    L_t: int
    H_t: int
    d_t: int
    n_seqs: int
    seq_len: int
    head_map_kind: str          # "identity" | "qwen" | "mismatch"
    source_kind: str            # "gauss" | "scaled" | "offset"
    noise: float
    weight_kind: str            # "lognormal" | "colmass" | "decay"
    lam_rel: float = 1e-2
    batch_seqs: Optional[int] = None   # streamed batch size (None = all at once)
    k: int = 1                         # selected source layers per map (multi-layer feature)
    sample_stride: int = 1             # calibration rows: tokens t with t % sample_stride == 0

    @property
    def P(self) -> int:
        return self.k * self.d_s + 1

    @property
    def n_maps(self) -> int:
        return 2 * self.L_t * self.H_t

    @property
    def n_weight_rows(self) -> int:
        return self.L_t * self.H_t

    def with_(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


WORKLOADS: Dict[str, Workload] = {
    "tiny": Workload("tiny", 1, 2, 64, 1, 2, 64, 4, 256, "identity", "gauss", 0.05, "lognormal"),
    "qwen50": Workload("qwen50", 40, 8, 128, 64, 8, 128, 50, 2048, "qwen", "scaled", 0.1, "colmass"),
    "qwen500": Workload("qwen500", 40, 8, 128, 64, 8, 128, 500, 2048, "qwen", "scaled", 0.1, "colmass",
                        batch_seqs=100),
    "mismatch": Workload("mismatch", 26, 8, 96, 40, 4, 128, 200, 4096, "mismatch", "scaled", 0.1, "decay"),
}

# Multi-layer feature (k selected source layers per target layer; the paper's
# Qwen3 direction uses k = 8 over 500 sequences of 1,024 tokens sampled every
# fourth token, 128,000 calibration rows).
WORKLOADS["tiny_k3"] = Workload("tiny_k3", 4, 2, 128, 3, 2, 128, 4, 520, "window", "gauss", 0.05, "lognormal",
                                k=3, sample_stride=4)
WORKLOADS["qwen_k8"] = Workload("qwen_k8", 40, 8, 128, 64, 8, 128, 500, 1024, "window", "scaled", 0.1, "colmass",
                                batch_seqs=100, k=8, sample_stride=4)

# Online application workload: maps from the qwen shapes, sender 8 x 32768.
APPLY = Workload("apply", 40, 8, 128, 64, 8, 128, 8, 32768, "qwen", "scaled", 0.1, "colmass")

SINK_LOGIT = 4.0          # position-0 sink strength for the column-mass weights
N_OUTLIERS = 4            # outlier channels per (source layer, kv, head)
OUTLIER_SCALE = 20.0
OFFSET_RATIO = 30.0       # channel mean / channel scale of the ``offset`` source kind


def _seed(*key) -> int:
    h = hashlib.sha256(("|".join(str(k) for k in (MASTER_SEED,) + key)).encode()).digest()
    return int.from_bytes(h[:8], "little") & ((1 << 63) - 1)


def _gen(device, *key) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(_seed(*key))
    return g


def _round_ratio(l: int, num: int, den: int) -> int:
    """round(l * num / den) in exact integer arithmetic (no ties occur for the
    ratios used here: a tie would need an even number to equal an odd one)."""
    return (2 * l * num + den) // (2 * den)


def head_map(wl: Workload) -> Dict[str, np.ndarray]:
    """Per-map (tgt_layer, tgt_head, kv, src_layer, src_head, weight_row), int32."""
    rows = {k: [] for k in ("tgt_layer", "tgt_head", "kv", "src_layer", "src_head", "weight_row")}
    for l in range(wl.L_t):
        for z in range(2):
            for h in range(wl.H_t):
                if wl.head_map_kind == "identity":
                    sl, sh = l, h
                elif wl.head_map_kind == "qwen":
                    sl, sh = _round_ratio(l, wl.L_s - 1, wl.L_t - 1) if wl.L_t > 1 else 0, h
                elif wl.head_map_kind == "mismatch":
                    sl, sh = _round_ratio(l, wl.L_s - 1, wl.L_t - 1) if wl.L_t > 1 else 0, 2 * h
                elif wl.head_map_kind.startswith("cyclic"):
                    shift = int(wl.head_map_kind[len("cyclic"):])
                    sl, sh = (_round_ratio(l, wl.L_s - 1, wl.L_t - 1) if wl.L_t > 1 else 0,
                              (h + shift) % wl.H_s)
                else:
                    raise ValueError(wl.head_map_kind)
                rows["tgt_layer"].append(l)
                rows["tgt_head"].append(h)
                rows["kv"].append(z)
                rows["src_layer"].append(sl)
                rows["src_head"].append(sh)
                rows["weight_row"].append(l * wl.H_t + h)
    return {k: np.asarray(v, dtype=np.int32) for k, v in rows.items()}


def layer_window(wl: Workload, l: int):
    """S_l of the ``window`` head maps: the k consecutive source layers centred on
    round(l (L_s - 1) / (L_t - 1)), clipped to the source model, ascending."""
    c = _round_ratio(l, wl.L_s - 1, wl.L_t - 1) if wl.L_t > 1 else 0
    start = min(max(c - wl.k // 2, 0), wl.L_s - wl.k)
    return list(range(start, start + wl.k))


def head_map_multi(wl: Workload) -> Dict[str, np.ndarray]:
    """Multi-layer head map: per map (tgt_layer, tgt_head, kv, src_layers [k],
    src_head, weight_row), int32; S_l from :func:`layer_window`, same head index."""
    if wl.head_map_kind != "window":
        raise ValueError(wl.head_map_kind)
    rows = {k: [] for k in ("tgt_layer", "tgt_head", "kv", "src_layers", "src_head", "weight_row")}
    for l in range(wl.L_t):
        S = layer_window(wl, l)
        for z in range(2):
            for h in range(wl.H_t):
                rows["tgt_layer"].append(l)
                rows["tgt_head"].append(h)
                rows["kv"].append(z)
                rows["src_layers"].append(S)
                rows["src_head"].append(h)
                rows["weight_row"].append(l * wl.H_t + h)
    return {k: np.asarray(v, dtype=np.int32) for k, v in rows.items()}


def cache_strides(L: int, H: int, n_seqs: int, seq_len: int, d: int):
    """Element strides (layer, kv, seq, head, tok) of the canonical layout."""
    s_tok = d
    s_head = seq_len * d
    s_seq = H * s_head
    s_kv = n_seqs * s_seq
    s_layer = 2 * s_kv
    return (s_layer, s_kv, s_seq, s_head, s_tok)


def _channel_scales(wl: Workload, device) -> torch.Tensor:
    """[L_s][2][H_s][d_s] fp32 per-channel scales: lognormal(0,1), 4 outliers x20."""
    out = torch.empty((wl.L_s, 2, wl.H_s, wl.d_s), dtype=torch.float32, device=device)
    for l in range(wl.L_s):
        for z in range(2):
            for g in range(wl.H_s):
                gen = _gen(device, wl.name, "scale", l, z, g)
                s = torch.exp(torch.randn(wl.d_s, generator=gen, device=device))
                idx = torch.randperm(wl.d_s, generator=gen, device=device)[:N_OUTLIERS]
                s[idx] *= OUTLIER_SCALE
                out[l, z, g] = s
    return out


def _channel_offsets(wl: Workload, scales: torch.Tensor, device) -> torch.Tensor:
    """[L_s][2][H_s][d_s] fp32 per-channel means OFFSET_RATIO * s_c * N(0,1)."""
    out = torch.empty_like(scales)
    for l in range(wl.L_s):
        for z in range(2):
            for g in range(wl.H_s):
                gen = _gen(device, wl.name, "offset", l, z, g)
                out[l, z, g] = OFFSET_RATIO * scales[l, z, g] * torch.randn(wl.d_s, generator=gen, device=device)
    return out


def gen_source(wl: Workload, seq0: int = 0, n_seqs: Optional[int] = None, seq_len: Optional[int] = None,
               device="cpu", out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Source cache [L_s][2][B][H_s][T][d_s] bf16 for sequences seq0 .. seq0+B-1
    (one generator per (layer, kv, head, batch))."""
    B = wl.n_seqs if n_seqs is None else n_seqs
    T = wl.seq_len if seq_len is None else seq_len
    if out is None:
        out = torch.empty((wl.L_s, 2, B, wl.H_s, T, wl.d_s), dtype=torch.bfloat16, device=device)
    if wl.source_kind not in ("gauss", "scaled", "offset"):
        raise ValueError(wl.source_kind)
    scales = _channel_scales(wl, device) if wl.source_kind in ("scaled", "offset") else None
    offsets = _channel_offsets(wl, scales, device) if wl.source_kind == "offset" else None
    for l in range(wl.L_s):
        for z in range(2):
            for g in range(wl.H_s):
                gen = _gen(device, wl.name, "x", l, z, g, seq0, B, T)
                x = torch.randn((B, T, wl.d_s), generator=gen, device=device, dtype=torch.float32)
                if scales is not None:
                    x *= scales[l, z, g]
                if offsets is not None:
                    x += offsets[l, z, g]
                out[l, z, :, g] = x.to(torch.bfloat16)
    return out


def planted_maps(wl: Workload, device="cpu") -> torch.Tensor:
    """Planted affine maps [n_maps][P][d_t] fp32: rows 0..P-2 ~ N(0, 1/(P-1)), row P-1 ~ N(0,1)."""
    hm = head_map(wl) if wl.head_map_kind != "window" else head_map_multi(wl)
    n = hm["kv"].shape[0]
    p = wl.P - 1
    W = torch.empty((n, wl.P, wl.d_t), dtype=torch.float32, device=device)
    for m in range(n):
        gen = _gen(device, wl.name, "map", int(hm["tgt_layer"][m]), int(hm["kv"][m]), int(hm["tgt_head"][m]))
        W[m, :p] = torch.randn((p, wl.d_t), generator=gen, device=device) / math.sqrt(p)
        W[m, p] = torch.randn((wl.d_t,), generator=gen, device=device)
    return W


def gen_target(wl: Workload, src: torch.Tensor, seq0: int = 0, device="cpu",
               out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Target cache [L_t][2][B][H_t][T][d_t] bf16: y = x A + b + noise * N(0,1) per map,
    with x the mapped source row (bf16 values), computed in fp32 and rounded to bf16."""
    B, T = src.shape[2], src.shape[4]
    if out is None:
        out = torch.empty((wl.L_t, 2, B, wl.H_t, T, wl.d_t), dtype=torch.bfloat16, device=device)
    multi = wl.head_map_kind == "window"
    hm = head_map_multi(wl) if multi else head_map(wl)
    W = planted_maps(wl, device=device)
    p = wl.P - 1
    for m in range(hm["kv"].shape[0]):
        l, z, h = int(hm["tgt_layer"][m]), int(hm["kv"][m]), int(hm["tgt_head"][m])
        sh = int(hm["src_head"][m])
        layers = [int(j) for j in hm["src_layers"][m]] if multi else [int(hm["src_layer"][m])]
        x = torch.cat([src[j, z, :, sh].reshape(B * T, wl.d_s) for j in layers], dim=1).to(torch.float32)
        gen = _gen(device, wl.name, "noise", l, z, h, seq0, B, T)
        e = torch.randn((B * T, wl.d_t), generator=gen, device=device, dtype=torch.float32)
        y = torch.addmm(W[m, p].unsqueeze(0), x, W[m, :p]).add_(e, alpha=wl.noise)
        out[l, z, :, h] = y.reshape(B, T, wl.d_t).to(torch.bfloat16)
    return out


def _column_mass(gen: torch.Generator, n: int, T: int, d: int, device) -> torch.Tensor:
    """Causal softmax column mass of Gaussian q, k (n independent draws), with a
    logit bonus on key 0.  Every query row sums to one, so the mean is one."""
    q = torch.randn((n, T, d), generator=gen, device=device, dtype=torch.float32)
    k = torch.randn((n, T, d), generator=gen, device=device, dtype=torch.float32)
    s = torch.bmm(q, k.transpose(1, 2).contiguous()) * (1.0 / math.sqrt(d))
    s[:, :, 0] += SINK_LOGIT
    causal = torch.ones((T, T), dtype=torch.bool, device=device).triu(1)
    s.masked_fill_(causal, float("-inf"))
    a = torch.softmax(s, dim=-1)
    return a.sum(dim=1)                                                  # [n, T]


def gen_weights(wl: Workload, seq0: int = 0, n_seqs: Optional[int] = None, seq_len: Optional[int] = None,
                device="cpu", out: Optional[torch.Tensor] = None, chunk: int = 16) -> torch.Tensor:
    """Weights [R][B*T] fp32, non-negative, mean one per (row, sequence)."""
    B = wl.n_seqs if n_seqs is None else n_seqs
    T = wl.seq_len if seq_len is None else seq_len
    R = wl.n_weight_rows
    if out is None:
        out = torch.empty((R, B * T), dtype=torch.float32, device=device)
    for r in range(R):
        if wl.weight_kind == "colmass":
            for b0 in range(0, B, chunk):
                nb = min(chunk, B - b0)
                gen = _gen(device, wl.name, "colmass", r, seq0 + b0, nb, T)
                m = _column_mass(gen, nb, T, wl.d_t, device)
                m = m / m.mean(dim=1, keepdim=True)
                out[r, b0 * T:(b0 + nb) * T] = m.reshape(-1)
            continue
        gen = _gen(device, wl.name, "w", r, seq0, B, T)
        z = torch.randn((B, T), generator=gen, device=device, dtype=torch.float32)
        if wl.weight_kind == "lognormal":
            w = torch.exp(z)
        elif wl.weight_kind == "decay":
            t = torch.arange(T, device=device, dtype=torch.float32)
            w = torch.exp(2.0 * z) / torch.sqrt(t + 1.0)
        else:
            raise ValueError(wl.weight_kind)
        out[r] = (w / w.mean(dim=1, keepdim=True)).reshape(-1)
    return out


def attn_boundaries(seq_len: int, n: int = 32, first: int = 12):
    """Logarithmically spaced query positions from ``first`` through seq_len - 1
    (rounded to the nearest integer, repeats dropped): the calibration boundaries
    of Sec. 4.1 (32 from token 12 through 1,023 for 1,024-token sequences)."""
    b = np.unique(np.rint(np.geomspace(first, seq_len - 1, n)).astype(np.int64))
    return b.astype(np.int32)


QUERY_SCORE_STD = 2.0     # target standard deviation of q . k / sqrt(d) for the generated queries


def gen_queries(wl: Workload, tgt: torch.Tensor, n_qheads: int, n_bounds: int, seq0: int = 0,
                device="cpu") -> torch.Tensor:
    """Queries [L_t][B][n_bounds][n_qheads][d_t] bf16 for the attention-aligned weights:
    N(0,1) scaled per (layer, KV head) so that q . k / sqrt(d) has standard
    deviation QUERY_SCORE_STD against that head's keys (one generator per layer
    and batch)."""
    L, B, H, d = wl.L_t, tgt.shape[2], wl.H_t, wl.d_t
    G = n_qheads // H
    out = torch.empty((L, B, n_bounds, n_qheads, d), dtype=torch.bfloat16, device=device)
    for l in range(L):
        gen = _gen(device, wl.name, "q", l, seq0, B, n_bounds)
        q = torch.randn((B, n_bounds, n_qheads, d), generator=gen, device=device, dtype=torch.float32)
        k2 = tgt[l, 0].to(torch.float32).pow(2).mean(dim=(0, 2, 3))                       # [H]
        scale = (QUERY_SCORE_STD / torch.sqrt(k2.clamp_min(1e-12))).repeat_interleave(G)   # [n_qheads]
        out[l] = (q * scale[None, None, :, None]).to(torch.bfloat16)
    return out


def gen_apply_source(wl: Workload = APPLY, n_seqs: Optional[int] = None, seq_len: Optional[int] = None,
                     device="cpu", out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Sender cache for the online application workload (same recipe as the source cache)."""
    return gen_source(wl, 0, n_seqs, seq_len, device=device, out=out)


def bf16_bits(t: torch.Tensor) -> np.ndarray:
    """Host uint16 copy of a bfloat16 tensor's bits."""
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
