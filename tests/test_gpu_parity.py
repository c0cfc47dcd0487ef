"""GPU parity of libcachebridge against the fp64 oracle (MI355X / gfx950).

Every call goes through the C ABI (via the thin binding).  Inputs are seeded
synthetic workloads; the oracle always consumes the exact bits the GPU consumed,
copied back from the device.  Tolerances (relative Frobenius error):
G and C 1e-4, solved maps 1e-3, applied bf16 caches 1e-3 -- checked per map.
"""
import os
import sys

import numpy as np
import pytest
import torch

import oracle
import synth

pytestmark = pytest.mark.gpu

TOL_STATS = 1e-4
TOL_MAPS = 1e-3
TOL_APPLY = 1e-3
NTHREADS = min(16, os.cpu_count() or 1)


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def cb():
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    import paper_2609_00891_amd as cbmod
    return cbmod


@pytest.fixture(autouse=True)
def _free_memory():
    yield
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def relF(a, b):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


def bits(t: torch.Tensor) -> np.ndarray:
    return synth.bf16_bits(t)


def make_inputs(wl, device="cuda", seq0=0):
    src = synth.gen_source(wl, seq0, device=device)
    tgt = synth.gen_target(wl, src, seq0, device=device)
    w = synth.gen_weights(wl, seq0, device=device)
    return src, tgt, w


def gpu_stats(cb, plan, src, tgt, w, G=None, C=None):
    n, P, dt = plan.n_maps, plan.P, plan.d_t
    if G is None:
        G = torch.empty((n, P, P), dtype=torch.float32, device="cuda")
        C = torch.empty((n, P, dt), dtype=torch.float32, device="cuda")
        cb.cb_stats_zero(plan, G, C)
    cb.cb_stats_accumulate(plan, src, tgt, w, G, C)
    torch.cuda.synchronize()
    return G, C


def compact(hm, sel, src, tgt, w):
    """Host copies of the rows the sampled maps read, with a head map onto them."""
    B, T = src.shape[2], src.shape[4]
    xs = torch.stack([src[hm["src_layer"][m], hm["kv"][m], :, hm["src_head"][m]] for m in sel])
    ys = torch.stack([tgt[hm["tgt_layer"][m], hm["kv"][m], :, hm["tgt_head"][m]] for m in sel])
    ws = torch.stack([w[hm["weight_row"][m]] for m in sel]).cpu().numpy()
    n = len(sel)
    d_s, d_t = xs.shape[-1], ys.shape[-1]
    xb = bits(xs).reshape(n, 1, B, 1, T, d_s)
    yb = bits(ys).reshape(n, 1, B, 1, T, d_t)
    chm = {"tgt_layer": np.arange(n, dtype=np.int32), "tgt_head": np.zeros(n, np.int32),
           "kv": np.zeros(n, np.int32), "src_layer": np.arange(n, dtype=np.int32),
           "src_head": np.zeros(n, np.int32), "weight_row": np.arange(n, dtype=np.int32)}
    ss = (B * T * d_s, 0, T * d_s, 0, d_s)
    ts = (B * T * d_t, 0, T * d_t, 0, d_t)
    return chm, xb, ss, yb, ts, np.ascontiguousarray(ws), B, T


def oracle_stats_sel(hm, sel, src, tgt, w):
    chm, xb, ss, yb, ts, ws, B, T = compact(hm, sel, src, tgt, w)
    return oracle.stats(chm, xb, ss, xb.shape[-1], yb, ts, yb.shape[-1], ws, B * T, B, T, n_threads=NTHREADS)


def check_stats(G, C, Go, Co, sel, tol=TOL_STATS):
    Gg = G[torch.as_tensor(sel, device=G.device)].double().cpu().numpy()
    Cg = C[torch.as_tensor(sel, device=C.device)].double().cpu().numpy()
    eg = max(relF(Gg[i], Go[i]) for i in range(len(sel)))
    ec = max(relF(Cg[i], Co[i]) for i in range(len(sel)))
    say(f"  stats parity: max relF G {eg:.3e}, C {ec:.3e}")
    assert eg <= tol and ec <= tol
    assert np.array_equal(Gg, np.transpose(Gg, (0, 2, 1))), "G must be exactly symmetric"
    return eg, ec


def ulp_distance(a_bits, b_bits) -> np.ndarray:
    """Distance in bf16 units in the last place between two bit arrays."""
    def ordered(x):
        x = x.astype(np.int32)
        return np.where(x < 0x8000, x, 0x8000 - x)
    return np.abs(ordered(a_bits) - ordered(b_bits))


def check_apply(ob, ref, label=""):
    """relF within the bar, and every element within one bf16 ulp of the oracle's
    value plus 1e-4 of its map's RMS output (near-zero outputs see the ~2^-17
    relative error of the split coefficients as several ulps).  Caches are
    [layer][kv][seq][head][tok][dim]; a map is one (layer, kv, head) slice."""
    g = oracle.bf16_to_double(ob)
    r = oracle.bf16_to_double(ref)
    e = relF(g, r)
    rms = np.sqrt((r * r).mean(axis=(2, 4, 5), keepdims=True))
    ulp = np.spacing(np.abs(r).astype(np.float32)).astype(np.float64) * 65536.0
    bound = ulp + 1e-4 * rms
    worst = float((np.abs(g - r) / bound).max())
    same = float((ob == ref).mean())
    say(f"  apply parity{label}: relF {e:.3e}, bitwise-equal {same:.6f}, worst err/bound {worst:.3f}")
    assert e <= TOL_APPLY and worst <= 1.0
    return e


def gpu_solve(cb, G, C, lam=1e-2, flags=None):
    if flags is None:
        flags = cb.CB_LAMBDA_RELATIVE
    maps = torch.empty_like(C)
    info = torch.empty((G.shape[0],), dtype=torch.int32, device="cuda")
    cb.cb_ridge_solve(G, C, lam, flags, maps, info)
    torch.cuda.synchronize()
    return maps, info


# ----------------------------------------------------------------------------- small, all maps

def test_tiny_end_to_end(cb):
    wl = synth.WORKLOADS["tiny"]
    say("tiny: generating")
    src, tgt, w = make_inputs(wl)
    hm = synth.head_map(wl)
    plan = cb.cb_plan_create(hm, src, tgt, wl.n_seqs * wl.seq_len)
    G, C = gpu_stats(cb, plan, src, tgt, w)
    sel = list(range(wl.n_maps))
    Go, Co = oracle_stats_sel(hm, sel, src, tgt, w)
    check_stats(G, C, Go, Co, sel)
    for flags, unpen in ((cb.CB_LAMBDA_RELATIVE, False),
                         (cb.CB_LAMBDA_RELATIVE | cb.CB_RIDGE_BIAS_UNPENALIZED, True)):
        maps, info = gpu_solve(cb, G, C, wl.lam_rel, flags)
        assert (info.cpu().numpy() == 0).all()
        Wo, io = oracle.ridge_solve(Go, Co, wl.lam_rel, relative=True, bias_unpenalized=unpen)
        Wg = maps.double().cpu().numpy()
        e = max(relF(Wg[i], Wo[i]) for i in sel)
        # the solver alone: both sides solve the oracle's moments rounded to fp32
        (Gt, G64), (Ct, C64) = shared_f32(Go), shared_f32(Co)
        ms, _ = gpu_solve(cb, Gt, Ct, wl.lam_rel, flags)
        Ws, _ = oracle.ridge_solve(G64, C64, wl.lam_rel, relative=True, bias_unpenalized=unpen)
        es = max(relF(ms[i].double().cpu().numpy(), Ws[i]) for i in sel)
        say(f"  maps parity (unpen={unpen}): end-to-end {e:.3e}, solver alone {es:.3e}")
        assert e <= TOL_MAPS and es <= 1e-6
    # apply the fitted maps back to the source cache
    out = torch.zeros_like(tgt)
    Wt, W64 = shared_f32(Wo)                       # the oracle's maps on both sides
    cb.cb_apply(plan, Wt, src, out)
    torch.cuda.synchronize()
    ref = np.zeros(tuple(out.shape), dtype=np.uint16)
    oracle.apply(hm, W64, bits(src), src.stride()[:5], wl.d_s, ref, out.stride()[:5],
                 wl.d_t, wl.n_seqs, wl.seq_len)
    check_apply(bits(out).reshape(ref.shape), ref)
    plan.close()


def shared_f32(a):
    """An array the oracle made, rounded once to fp32: the device tensor the GPU
    call takes and the exact fp64 copy of the same values the oracle takes."""
    a32 = np.ascontiguousarray(np.asarray(a, dtype=np.float32))
    return torch.from_numpy(a32).to("cuda"), a32.astype(np.float64)


WIDTHS = [(ds, dt) for ds in (64, 96, 128) for dt in (64, 96, 128)]


@pytest.mark.parametrize("d_s,d_t", WIDTHS)
def test_widths_ragged_tokens_and_shared_sources(cb, d_s, d_t):
    # 3 target layers over 2 source layers: some source blocks feed two maps
    # (shared items), others one (paired singles); 3 x 45 tokens leave a
    # ragged last tile and sequences that start inside a tile.
    wl = synth.Workload("ragged", 2, 3, d_s, 3, 2, d_t, 3, 45, "cyclic1", "scaled", 0.1, "lognormal")
    src, tgt, w = make_inputs(wl)
    hm = synth.head_map(wl)
    plan = cb.cb_plan_create(hm, src, tgt, 4096)
    G, C = gpu_stats(cb, plan, src, tgt, w)
    sel = list(range(wl.n_maps))
    Go, Co = oracle_stats_sel(hm, sel, src, tgt, w)
    check_stats(G, C, Go, Co, sel)
    maps, info = gpu_solve(cb, G, C)
    assert (info.cpu().numpy() == 0).all()
    Wo, _ = oracle.ridge_solve(Go, Co, 1e-2, relative=True)
    assert max(relF(maps[i].double().cpu().numpy(), Wo[i]) for i in sel) <= TOL_MAPS
    out = torch.zeros_like(tgt)
    Wt, W64 = shared_f32(Wo)                       # the oracle's maps on both sides
    cb.cb_apply(plan, Wt, src, out)
    torch.cuda.synchronize()
    ref = np.zeros(tuple(out.shape), dtype=np.uint16)
    oracle.apply(hm, W64, bits(src), src.stride()[:5], d_s, ref, out.stride()[:5],
                 d_t, wl.n_seqs, wl.seq_len)
    check_apply(bits(out).reshape(ref.shape), ref)
    plan.close()


@pytest.mark.parametrize("d_s,d_t,T", [(64, 64, 45), (96, 128, 64), (128, 128, 96)])
def test_single_map_items(cb, d_s, d_t, T):
    # Three maps on three different source blocks: the plan pairs two of them
    # and leaves an item with a single map, whose other waves only copy.
    wl = synth.Workload("single", 1, 2, d_s, 1, 2, d_t, 3, T, "identity", "scaled", 0.1, "lognormal")
    src, tgt, w = make_inputs(wl)
    full = synth.head_map(wl)
    keep = [0, 1, 3]
    hm = {k: np.ascontiguousarray(np.asarray(v)[keep]) for k, v in full.items()}
    plan = cb.cb_plan_create(hm, src, tgt, 4096)
    G, C = gpu_stats(cb, plan, src, tgt, w)
    sel = list(range(len(keep)))
    Go, Co = oracle_stats_sel(hm, sel, src, tgt, w)
    check_stats(G, C, Go, Co, sel)
    maps, info = gpu_solve(cb, G, C)
    assert (info.cpu().numpy() == 0).all()
    Wo, _ = oracle.ridge_solve(Go, Co, 1e-2, relative=True)
    assert max(relF(maps[i].double().cpu().numpy(), Wo[i]) for i in sel) <= TOL_MAPS
    out = torch.zeros_like(tgt)
    Wt, W64 = shared_f32(Wo)                       # the oracle's maps on both sides
    cb.cb_apply(plan, Wt, src, out)
    torch.cuda.synchronize()
    ref = np.zeros(tuple(out.shape), dtype=np.uint16)
    oracle.apply(hm, W64, bits(src), src.stride()[:5], d_s, ref, out.stride()[:5],
                 d_t, wl.n_seqs, wl.seq_len)
    check_apply(bits(out).reshape(ref.shape), ref)
    plan.close()


def test_strided_views_match_canonical_layout(cb):
    wl = synth.Workload("strided", 2, 2, 128, 2, 2, 128, 2, 130, "qwen", "scaled", 0.1, "lognormal")
    src, tgt, w = make_inputs(wl)
    hm = synth.head_map(wl)
    # the same values stored [L][2][H][B][T][d] and viewed as [L][2][B][H][T][d]
    src_p = src.permute(0, 1, 3, 2, 4, 5).contiguous().permute(0, 1, 3, 2, 4, 5)
    tgt_p = tgt.permute(0, 1, 3, 2, 4, 5).contiguous().permute(0, 1, 3, 2, 4, 5)
    assert src_p.stride() != src.stride()
    plan = cb.cb_plan_create(hm, src, tgt, 4096)
    G1, C1 = gpu_stats(cb, plan, src, tgt, w)
    G2, C2 = gpu_stats(cb, plan, src_p, tgt_p, w)
    assert torch.equal(G1, G2) and torch.equal(C1, C2)
    maps, _ = gpu_solve(cb, G1, C1)
    o1 = torch.zeros_like(tgt)
    o2 = torch.zeros_like(tgt_p)
    cb.cb_apply(plan, maps, src, o1)
    cb.cb_apply(plan, maps, src_p, o2)
    torch.cuda.synchronize()
    assert torch.equal(o1, o2)
    plan.close()


def test_invariants_determinism_scaling_additivity(cb):
    wl = synth.Workload("inv", 3, 2, 128, 4, 2, 128, 4, 300, "qwen", "scaled", 0.1, "lognormal")
    src, tgt, w = make_inputs(wl)
    hm = synth.head_map(wl)
    plan = cb.cb_plan_create(hm, src, tgt, 4096)
    G1, C1 = gpu_stats(cb, plan, src, tgt, w)
    G2, C2 = gpu_stats(cb, plan, src, tgt, w)
    assert torch.equal(G1, G2) and torch.equal(C1, C2), "bitwise run-to-run determinism"
    G4, C4 = gpu_stats(cb, plan, src, tgt, w * 4.0)
    assert torch.equal(G4, 4.0 * G1) and torch.equal(C4, 4.0 * C1), "power-of-two weight scaling is exact"
    # additivity over sequence splits: two calls (seqs 0-1, 2-3) vs one
    Ga, Ca = gpu_stats(cb, plan, src[:, :, :2], tgt[:, :, :2], w.view(-1, 4, 300)[:, :2].reshape(w.shape[0], -1))
    Ga, Ca = gpu_stats(cb, plan, src[:, :, 2:], tgt[:, :, 2:], w.view(-1, 4, 300)[:, 2:].reshape(w.shape[0], -1),
                       Ga, Ca)
    assert relF(Ga.double().cpu(), G1.double().cpu()) < 1e-6
    assert relF(Ca.double().cpu(), C1.double().cpu()) < 1e-6
    # empty call is a no-op
    Gb = G1.clone()
    Cb = C1.clone()
    cb.cb_stats_accumulate(plan, src[:, :, :0], tgt[:, :, :0], w[:, :0].contiguous(), Gb, Cb, w_row_stride=1)
    torch.cuda.synchronize()
    assert torch.equal(Gb, G1) and torch.equal(Cb, C1)
    # all-zero weights: zero moments, relative lambda 0 -> first pivot fails
    Gz, Cz = gpu_stats(cb, plan, src, tgt, torch.zeros_like(w))
    assert not Gz.any() and not Cz.any()
    maps, info = gpu_solve(cb, Gz, Cz)
    assert (info.cpu().numpy() == 1).all() and not maps.any()
    plan.close()


def test_apply_identity_map_copies_and_bias_only(cb):
    wl = synth.Workload("ident", 3, 2, 128, 5, 2, 128, 2, 77, "qwen", "scaled", 0.1, "lognormal")
    src = synth.gen_source(wl, device="cuda")
    hm = synth.head_map(wl)
    plan = cb.cb_plan_create(hm, (wl.L_s, wl.H_s, wl.d_s), (wl.L_t, wl.H_t, wl.d_t), 1024)
    n = wl.n_maps
    maps = torch.zeros((n, wl.P, wl.d_t), dtype=torch.float32, device="cuda")
    maps[:, :wl.d_s, :] = torch.eye(wl.d_s, device="cuda")
    out = torch.zeros((wl.L_t, 2, wl.n_seqs, wl.H_t, wl.seq_len, wl.d_t), dtype=torch.bfloat16, device="cuda")
    cb.cb_apply(plan, maps, src, out)
    torch.cuda.synchronize()
    for m in range(n):
        a = out[hm["tgt_layer"][m], hm["kv"][m], :, hm["tgt_head"][m]]
        b = src[hm["src_layer"][m], hm["kv"][m], :, hm["src_head"][m]]
        assert torch.equal(a.view(torch.int16), b.view(torch.int16))
    bias = torch.randn((n, wl.d_t), device="cuda")
    maps.zero_()
    maps[:, wl.d_s, :] = bias
    cb.cb_apply(plan, maps, src, out)
    torch.cuda.synchronize()
    for m in range(n):
        a = out[hm["tgt_layer"][m], hm["kv"][m], :, hm["tgt_head"][m]]
        assert torch.equal(a.view(torch.int16), bias[m].to(torch.bfloat16).expand_as(a).view(torch.int16))
    plan.close()


def test_device_side_argument_errors(cb):
    wl = synth.Workload("err", 1, 2, 64, 1, 2, 64, 2, 64, "identity", "gauss", 0.1, "lognormal")
    src, tgt, w = make_inputs(wl)
    hm = synth.head_map(wl)
    plan = cb.cb_plan_create(hm, src, tgt, 100)
    G = torch.zeros((4, 65, 65), device="cuda")
    C = torch.zeros((4, 65, 64), device="cuda")
    with pytest.raises(cb.CacheBridgeError, match="CB_ERR_UNSUPPORTED"):
        cb.cb_stats_accumulate(plan, src, tgt, w, G, C)                  # 128 tokens > 100
    flat = torch.zeros(src.numel() + 8, dtype=torch.bfloat16, device="cuda")
    mis = flat[1:1 + src.numel()].view(src.shape)
    plan2 = cb.cb_plan_create(hm, src, tgt, 4096)
    with pytest.raises(cb.CacheBridgeError, match="CB_ERR_MISALIGNED"):
        cb.cb_stats_accumulate(plan2, mis, tgt, w, G, C)
    with pytest.raises(cb.CacheBridgeError, match="CB_ERR_SHAPE"):
        cb.cb_stats_accumulate(plan2, src[:, :, :1], tgt, w, G, C)
    with pytest.raises(cb.CacheBridgeError, match="CB_ERR_SHAPE"):
        cb.cb_stats_accumulate(plan2, src, tgt, w, G, C, w_row_stride=10)
    plan.close()
    plan2.close()


# ----------------------------------------------------------------------------- full-size workloads

def sample_maps(n, k, seed=0):
    return sorted(np.random.default_rng(seed).choice(n, size=k, replace=False).tolist())


def _full_size_stats(cb, wl, n_sample, seq0=0):
    say(f"{wl.name}: generating {wl.n_seqs} x {wl.seq_len} tokens")
    src, tgt, w = make_inputs(wl, seq0=seq0)
    hm = synth.head_map(wl)
    plan = cb.cb_plan_create(hm, src, tgt, wl.n_seqs * wl.seq_len)
    say(f"{wl.name}: GPU statistics")
    G, C = gpu_stats(cb, plan, src, tgt, w)
    sel = sample_maps(wl.n_maps, n_sample)
    say(f"{wl.name}: oracle on maps {sel}")
    Go, Co = oracle_stats_sel(hm, sel, src, tgt, w)
    check_stats(G, C, Go, Co, sel)
    maps, info = gpu_solve(cb, G, C, wl.lam_rel, cb.CB_LAMBDA_RELATIVE | cb.CB_RIDGE_BIAS_UNPENALIZED)
    assert (info.cpu().numpy() == 0).all()
    Wo, _ = oracle.ridge_solve(Go, Co, wl.lam_rel, relative=True, bias_unpenalized=True, n_threads=NTHREADS)
    e = max(relF(maps[m].double().cpu().numpy(), Wo[i]) for i, m in enumerate(sel))
    say(f"  maps parity: {e:.3e}")
    assert e <= TOL_MAPS
    del src, tgt, w
    plan.close()


def test_qwen50_full_size_sampled_maps(cb):
    _full_size_stats(cb, synth.WORKLOADS["qwen50"], 16)


def test_qwen500_batch_full_size_sampled_maps(cb):
    wl = synth.WORKLOADS["qwen500"]
    _full_size_stats(cb, wl.with_(n_seqs=wl.batch_seqs), 8, seq0=0)


def test_mismatch_full_size_sampled_maps(cb):
    _full_size_stats(cb, synth.WORKLOADS["mismatch"], 4)


def test_apply_full_size_sampled_tokens(cb):
    wl = synth.APPLY
    say("apply: generating sender cache 8 x 32768")
    src = synth.gen_apply_source(wl, device="cuda")
    hm = synth.head_map(wl)
    maps = synth.planted_maps(wl, device="cuda")
    plan = cb.cb_plan_create(hm, (wl.L_s, wl.H_s, wl.d_s), (wl.L_t, wl.H_t, wl.d_t), 1024)
    out = torch.empty((wl.L_t, 2, wl.n_seqs, wl.H_t, wl.seq_len, wl.d_t), dtype=torch.bfloat16, device="cuda")
    say("apply: GPU")
    cb.cb_apply(plan, maps, src, out)
    torch.cuda.synchronize()
    Wd = maps.double().cpu().numpy()
    for (b, t0, t1) in ((0, 0, 1536), (wl.n_seqs - 1, wl.seq_len - 1024, wl.seq_len)):
        say(f"apply: oracle on batch row {b}, tokens {t0}..{t1}")
        s_sub = src[:, :, b:b + 1, :, t0:t1].contiguous()
        ref = np.zeros((wl.L_t, 2, 1, wl.H_t, t1 - t0, wl.d_t), dtype=np.uint16)
        oracle.apply(hm, Wd, bits(s_sub), s_sub.stride()[:5], wl.d_s, ref,
                     synth.cache_strides(wl.L_t, wl.H_t, 1, t1 - t0, wl.d_t), wl.d_t, 1, t1 - t0,
                     n_threads=NTHREADS)
        ob = bits(out[:, :, b:b + 1, :, t0:t1].contiguous()).reshape(ref.shape)
        worst = 0.0
        for m in range(wl.n_maps):
            l, z, h = hm["tgt_layer"][m], hm["kv"][m], hm["tgt_head"][m]
            worst = max(worst, relF(oracle.bf16_to_double(ob[l, z, 0, h]), oracle.bf16_to_double(ref[l, z, 0, h])))
        say(f"  worst per-map relF {worst:.3e}")
        assert worst <= TOL_APPLY
        check_apply(ob, ref, f" (row {b}, tokens {t0}..{t1})")
    plan.close()


# ----------------------------------------------------------------------------- two-pass centered form

TOL_SUMS = 1e-9        # fp64 sums of exact fp64 products: only the summation order differs


def gpu_centered(cb, plan, batches):
    """Pass 1 (means) over every batch, then pass 2 (centered moments) over every
    batch; ``batches`` holds (src, tgt, weights) views of one workload."""
    n, ds, dt = plan.n_maps, plan.d_s, plan.d_t
    sums = torch.empty((n, 1 + ds + dt), dtype=torch.float64, device="cuda")
    A = torch.empty((n, ds, ds), dtype=torch.float32, device="cuda")
    B = torch.empty((n, ds, dt), dtype=torch.float32, device="cuda")
    cb.cb_stats_zero_centered(plan, sums, A, B)
    for s, t, w in batches:
        cb.cb_stats_means(plan, s, t, w, sums)
    for s, t, w in batches:
        cb.cb_stats_accumulate_centered(plan, s, t, w, sums, A, B)
    torch.cuda.synchronize()
    return sums, A, B


def seq_batches(src, tgt, w, bounds):
    """Views of sequences [b0, b1) for each (b0, b1): the weights keep their row stride."""
    T = src.shape[4]
    return [(src[:, :, b0:b1], tgt[:, :, b0:b1], w[:, b0 * T:b1 * T]) for b0, b1 in bounds]


def gpu_solve_centered(cb, sums, A, B, lam, flags):
    maps = torch.empty((A.shape[0], A.shape[1] + 1, B.shape[2]), dtype=torch.float32, device="cuda")
    info = torch.empty((A.shape[0],), dtype=torch.int32, device="cuda")
    cb.cb_ridge_solve_centered(sums, A, B, lam, flags, maps, info)
    torch.cuda.synchronize()
    return maps, info


def oracle_centered_sel(hm, sel, src, tgt, w):
    chm, xb, ss, yb, ts, ws, B, T = compact(hm, sel, src, tgt, w)
    return oracle.stats_centered(chm, xb, ss, xb.shape[-1], yb, ts, yb.shape[-1], ws, B * T, B, T,
                                 n_threads=NTHREADS)


def check_centered(sums, A, B, so, Ao, Bo, sel, tol=TOL_STATS, tol_sums=TOL_SUMS):
    idx = torch.as_tensor(sel, device=A.device)
    sg = sums[idx].cpu().numpy()
    Ag = A[idx].double().cpu().numpy()
    Bg = B[idx].double().cpu().numpy()
    es = max(relF(sg[i], so[i]) for i in range(len(sel)))
    ea = max(relF(Ag[i], Ao[i]) for i in range(len(sel)))
    eb = max(relF(Bg[i], Bo[i]) for i in range(len(sel)))
    say(f"  centered parity: max relF sums {es:.3e}, A {ea:.3e}, B {eb:.3e}")
    assert es <= tol_sums and ea <= tol and eb <= tol
    assert np.array_equal(Ag, np.transpose(Ag, (0, 2, 1))), "A must be exactly symmetric"
    return es, ea, eb


def check_centered_maps(cb, sums, A, B, so, Ao, Bo, sel, lam):
    maps, info = gpu_solve_centered(cb, sums, A, B, lam, cb.CB_LAMBDA_RELATIVE)
    assert (info[torch.as_tensor(sel, device=info.device)].cpu().numpy() == 0).all()
    Wo, io = oracle.ridge_solve_centered(so, Ao, Bo, lam, relative=True, n_threads=NTHREADS)
    assert (io == 0).all()
    Wg = maps.double().cpu().numpy()
    e = max(relF(Wg[m], Wo[i]) for i, m in enumerate(sel))
    # the solver alone: both sides solve the oracle's sums (fp64) and moments rounded to fp32
    (At, A64), (Bt, B64) = shared_f32(Ao), shared_f32(Bo)
    ms, _ = gpu_solve_centered(cb, torch.from_numpy(np.ascontiguousarray(so)).to("cuda"), At, Bt, lam,
                               cb.CB_LAMBDA_RELATIVE)
    Ws, _ = oracle.ridge_solve_centered(so, A64, B64, lam, relative=True, n_threads=NTHREADS)
    es = max(relF(ms[i].double().cpu().numpy(), Ws[i]) for i in range(len(sel)))
    say(f"  centered maps parity: end-to-end {e:.3e}, solver alone {es:.3e}")
    assert e <= TOL_MAPS and es <= 1e-6
    return maps, Wo


def test_centered_tiny_end_to_end(cb):
    wl = synth.WORKLOADS["tiny"]
    src, tgt, w = make_inputs(wl)
    hm = synth.head_map(wl)
    plan = cb.cb_plan_create(hm, src, tgt, wl.n_seqs * wl.seq_len)
    sums, A, B = gpu_centered(cb, plan, seq_batches(src, tgt, w, [(0, 1), (1, 4)]))
    sel = list(range(wl.n_maps))
    so, Ao, Bo = oracle_centered_sel(hm, sel, src, tgt, w)
    check_centered(sums, A, B, so, Ao, Bo, sel)
    maps, Wo = check_centered_maps(cb, sums, A, B, so, Ao, Bo, sel, wl.lam_rel)
    # the uncentered augmented form with an unpenalized bias solves the same problem
    G, C = gpu_stats(cb, plan, src, tgt, w)
    mu, _ = gpu_solve(cb, G, C, wl.lam_rel, cb.CB_LAMBDA_RELATIVE | cb.CB_RIDGE_BIAS_UNPENALIZED)
    ex = max(relF(maps[m].double().cpu().numpy(), mu[m].double().cpu().numpy()) for m in sel)
    say(f"  centered vs uncentered-augmented maps: {ex:.3e}")
    assert ex <= 2 * TOL_MAPS
    out = torch.zeros_like(tgt)
    Wt, W64 = shared_f32(Wo)                       # the oracle's maps on both sides
    cb.cb_apply(plan, Wt, src, out)
    torch.cuda.synchronize()
    ref = np.zeros(tuple(out.shape), dtype=np.uint16)
    oracle.apply(hm, W64, bits(src), src.stride()[:5], wl.d_s, ref, out.stride()[:5],
                 wl.d_t, wl.n_seqs, wl.seq_len)
    check_apply(bits(out).reshape(ref.shape), ref)
    plan.close()


@pytest.mark.parametrize("d_s,d_t", WIDTHS)
def test_centered_widths_ragged_batches_and_shared_sources(cb, d_s, d_t):
    # shared-source items and paired singles, a ragged last tile, and three
    # streamed batches that split the sequences unevenly
    wl = synth.Workload("cragged", 2, 3, d_s, 3, 2, d_t, 4, 45, "cyclic1", "offset", 0.1, "lognormal")
    src, tgt, w = make_inputs(wl)
    hm = synth.head_map(wl)
    plan = cb.cb_plan_create(hm, src, tgt, 4096)
    sums, A, B = gpu_centered(cb, plan, seq_batches(src, tgt, w, [(0, 1), (1, 3), (3, 4)]))
    sel = list(range(wl.n_maps))
    so, Ao, Bo = oracle_centered_sel(hm, sel, src, tgt, w)
    check_centered(sums, A, B, so, Ao, Bo, sel)
    check_centered_maps(cb, sums, A, B, so, Ao, Bo, sel, 1e-2)
    plan.close()


@pytest.mark.parametrize("d_s,d_t,T", [(64, 64, 45), (96, 128, 64), (128, 128, 96)])
def test_centered_single_map_items(cb, d_s, d_t, T):
    wl = synth.Workload("csingle", 1, 2, d_s, 1, 2, d_t, 3, T, "identity", "offset", 0.1, "lognormal")
    src, tgt, w = make_inputs(wl)
    full = synth.head_map(wl)
    keep = [0, 1, 3]
    hm = {k: np.ascontiguousarray(np.asarray(v)[keep]) for k, v in full.items()}
    plan = cb.cb_plan_create(hm, src, tgt, 4096)
    sums, A, B = gpu_centered(cb, plan, [(src, tgt, w)])
    sel = list(range(len(keep)))
    so, Ao, Bo = oracle_centered_sel(hm, sel, src, tgt, w)
    check_centered(sums, A, B, so, Ao, Bo, sel)
    check_centered_maps(cb, sums, A, B, so, Ao, Bo, sel, 1e-2)
    plan.close()


def test_centered_large_channel_means(cb):
    # channel means 30 x their spread (median |mu|/sigma ~ 18): the centered
    # moments stay at the stats bar, where the uncentered moments of the same
    # data lose digits to cancellation when A is recovered from G
    wl = synth.Workload("coffset", 2, 2, 128, 3, 2, 128, 8, 2048, "qwen", "offset", 0.1, "colmass")
    src, tgt, w = make_inputs(wl)
    hm = synth.head_map(wl)
    plan = cb.cb_plan_create(hm, src, tgt, wl.n_seqs * wl.seq_len)
    sums, A, B = gpu_centered(cb, plan, seq_batches(src, tgt, w, [(0, 4), (4, 8)]))
    sel = list(range(wl.n_maps))
    so, Ao, Bo = oracle_centered_sel(hm, sel, src, tgt, w)
    es, ea, eb = check_centered(sums, A, B, so, Ao, Bo, sel)
    check_centered_maps(cb, sums, A, B, so, Ao, Bo, sel, wl.lam_rel)
    # the same A from the uncentered moments, for comparison (reported only)
    G, _ = gpu_stats(cb, plan, src, tgt, w)
    Gd = G.double().cpu().numpy()
    d = wl.d_s
    eu = max(relF(Gd[m, :d, :d] - np.outer(Gd[m, d, :d], Gd[m, d, :d]) / Gd[m, d, d], Ao[m]) for m in sel)
    say(f"  A from uncentered G: relF {eu:.3e} (centered {ea:.3e})")
    assert ea * 10 < eu
    plan.close()


def test_centered_zero_weights_empty_calls_and_determinism(cb):
    wl = synth.Workload("czero", 2, 2, 128, 2, 2, 96, 3, 70, "qwen", "offset", 0.1, "lognormal")
    src, tgt, w = make_inputs(wl)
    w[1].zero_()                                    # weight row 1: target head 1 of layer 0, K and V
    hm = synth.head_map(wl)
    zero_maps = [m for m in range(wl.n_maps) if hm["weight_row"][m] == 1]
    plan = cb.cb_plan_create(hm, src, tgt, 4096)
    s1, A1, B1 = gpu_centered(cb, plan, [(src, tgt, w)])
    s2, A2, B2 = gpu_centered(cb, plan, [(src, tgt, w)])
    assert torch.equal(s1, s2) and torch.equal(A1, A2) and torch.equal(B1, B2), "bitwise determinism"
    # empty calls change nothing
    cb.cb_stats_means(plan, src[:, :, :0], tgt[:, :, :0], w[:, :0], s2, w_row_stride=1)
    cb.cb_stats_accumulate_centered(plan, src[:, :, :0], tgt[:, :, :0], w[:, :0], s2, A2, B2, w_row_stride=1)
    torch.cuda.synchronize()
    assert torch.equal(s1, s2) and torch.equal(A1, A2) and torch.equal(B1, B2)
    for m in zero_maps:
        assert not s1[m].any() and not A1[m].any() and not B1[m].any()
    sel = list(range(wl.n_maps))
    so, Ao, Bo = oracle_centered_sel(hm, sel, src, tgt, w)
    check_centered(s1, A1, B1, so, Ao, Bo, sel)
    # absolute lambda (the largest mean diagonal of A: a strong ridge keeps
    # every system well conditioned, so the moments' error is not amplified):
    # zero-weight maps solve to W = 0 and b = 0
    lam = float(max(np.trace(Ao[m]) for m in sel) / wl.d_s)
    maps, info = gpu_solve_centered(cb, s1, A1, B1, lam, 0)
    assert (info.cpu().numpy() == 0).all()
    Wo, _ = oracle.ridge_solve_centered(so, Ao, Bo, lam, relative=False)
    # the solver alone: both sides solve the oracle's sums and moments (rounded to fp32)
    (At, A64), (Bt, B64) = shared_f32(Ao), shared_f32(Bo)
    ms, _ = gpu_solve_centered(cb, torch.from_numpy(np.ascontiguousarray(so)).to("cuda"), At, Bt, lam, 0)
    Ws, _ = oracle.ridge_solve_centered(so, A64, B64, lam, relative=False)
    live = [m for m in sel if m not in zero_maps]
    e = max(relF(maps[m].double().cpu().numpy(), Wo[m]) for m in live)
    es = max(relF(ms[m].double().cpu().numpy(), Ws[m]) for m in live)
    say(f"  centered maps parity (absolute lambda): end-to-end {e:.3e}, solver alone {es:.3e}")
    assert e <= TOL_MAPS and es <= 1e-6
    for m in zero_maps:
        assert not maps[m].any()
    # relative lambda is zero for them: the first pivot fails, maps are zero-filled
    maps, info = gpu_solve_centered(cb, s1, A1, B1, 1e-2, cb.CB_LAMBDA_RELATIVE)
    inf = info.cpu().numpy()
    assert all(inf[m] == 1 for m in zero_maps) and all(inf[m] == 0 for m in sel if m not in zero_maps)
    for m in zero_maps:
        assert not maps[m].any()
    plan.close()


# one-pass (shifted) form of the centered moments: the sums come from fp32
# partial sums within a work unit, added in fp64 across units (pass 1 is exact)
TOL_SUMS_SHIFTED = 1e-6


def gpu_shifted(cb, plan, pilot, batches, zero_shift=False):
    """Pilot means (cb_stats_means over ``pilot``, or no shift), the moments about
    them in one pass over ``batches``, then cb_stats_shift_finish."""
    n, dx, dt = plan.n_maps, plan.P - 1, plan.d_t
    shift = torch.zeros((n, 1 + dx + dt), dtype=torch.float64, device="cuda")
    sums = torch.empty_like(shift)
    A = torch.empty((n, dx, dx), dtype=torch.float32, device="cuda")
    B = torch.empty((n, dx, dt), dtype=torch.float32, device="cuda")
    cb.cb_stats_zero_centered(plan, sums, A, B)
    if not zero_shift:
        for s, t, w in pilot:
            cb.cb_stats_means(plan, s, t, w, shift)
    for s, t, w in batches:
        cb.cb_stats_accumulate_shifted(plan, s, t, w, shift, sums, A, B)
    cb.cb_stats_shift_finish(plan, shift, sums, A, B)
    torch.cuda.synchronize()
    return sums, A, B


@pytest.mark.parametrize("d_s,d_t", WIDTHS)
def test_shifted_one_pass_matches_oracle_and_two_pass(cb, d_s, d_t):
    # the workload of the two-pass ragged test; the pilot is the first sequence
    wl = synth.Workload("cragged", 2, 3, d_s, 3, 2, d_t, 4, 45, "cyclic1", "offset", 0.1, "lognormal")
    src, tgt, w = make_inputs(wl)
    hm = synth.head_map(wl)
    plan = cb.cb_plan_create(hm, src, tgt, 4096)
    batches = seq_batches(src, tgt, w, [(0, 1), (1, 3), (3, 4)])
    sums, A, B = gpu_shifted(cb, plan, batches[:1], batches)
    sel = list(range(wl.n_maps))
    so, Ao, Bo = oracle_centered_sel(hm, sel, src, tgt, w)
    check_centered(sums, A, B, so, Ao, Bo, sel, tol_sums=TOL_SUMS_SHIFTED)
    check_centered_maps(cb, sums, A, B, so, Ao, Bo, sel, 1e-2)
    s2, A2, B2 = gpu_centered(cb, plan, batches)
    ea = max(relF(A[m].double().cpu().numpy(), A2[m].double().cpu().numpy()) for m in sel)
    eb = max(relF(B[m].double().cpu().numpy(), B2[m].double().cpu().numpy()) for m in sel)
    say(f"  shifted vs two-pass: A {ea:.3e}, B {eb:.3e}")
    assert ea <= TOL_STATS and eb <= TOL_STATS
    plan.close()


def test_shifted_large_channel_means_and_no_shift(cb):
    # channel means 30 x their spread: a pilot of one sequence in eight removes
    # the offsets, so the one-pass moments hold the stats bar like the two-pass
    # ones; with no shift (zero pilot sums) the same call is the uncentered form
    # with its cancellation, which the finishing step cannot undo
    wl = synth.Workload("coffset", 2, 2, 128, 3, 2, 128, 8, 2048, "qwen", "offset", 0.1, "colmass")
    src, tgt, w = make_inputs(wl)
    hm = synth.head_map(wl)
    plan = cb.cb_plan_create(hm, src, tgt, wl.n_seqs * wl.seq_len)
    batches = seq_batches(src, tgt, w, [(0, 4), (4, 8)])
    pilot = seq_batches(src, tgt, w, [(0, 1)])
    sums, A, B = gpu_shifted(cb, plan, pilot, batches)
    sel = list(range(wl.n_maps))
    so, Ao, Bo = oracle_centered_sel(hm, sel, src, tgt, w)
    es, ea, eb = check_centered(sums, A, B, so, Ao, Bo, sel, tol_sums=TOL_SUMS_SHIFTED)
    check_centered_maps(cb, sums, A, B, so, Ao, Bo, sel, wl.lam_rel)
    s0, A0, B0 = gpu_shifted(cb, plan, pilot, batches, zero_shift=True)
    e0 = max(relF(A0[m].double().cpu().numpy(), Ao[m]) for m in sel)
    say(f"  no shift: A relF {e0:.3e} (pilot shift {ea:.3e})")
    assert ea * 10 < e0
    plan.close()


def test_shifted_zero_weights_empty_calls_and_determinism(cb):
    wl = synth.Workload("czero", 2, 2, 128, 2, 2, 96, 3, 70, "qwen", "offset", 0.1, "lognormal")
    src, tgt, w = make_inputs(wl)
    w[1].zero_()
    hm = synth.head_map(wl)
    zero_maps = [m for m in range(wl.n_maps) if hm["weight_row"][m] == 1]
    plan = cb.cb_plan_create(hm, src, tgt, 4096)
    pilot = seq_batches(src, tgt, w, [(0, 1)])
    s1, A1, B1 = gpu_shifted(cb, plan, pilot, [(src, tgt, w)])
    s2, A2, B2 = gpu_shifted(cb, plan, pilot, [(src, tgt, w)])
    assert torch.equal(s1, s2) and torch.equal(A1, A2) and torch.equal(B1, B2), "bitwise determinism"
    shift = torch.zeros_like(s1)
    cb.cb_stats_accumulate_shifted(plan, src[:, :, :0], tgt[:, :, :0], w[:, :0], shift, s2, A2, B2, w_row_stride=1)
    torch.cuda.synchronize()
    assert torch.equal(s1, s2) and torch.equal(A1, A2) and torch.equal(B1, B2), "an empty call changes nothing"
    for m in zero_maps:
        assert not s1[m].any() and not A1[m].any() and not B1[m].any()
    sel = list(range(wl.n_maps))
    so, Ao, Bo = oracle_centered_sel(hm, sel, src, tgt, w)
    check_centered(s1, A1, B1, so, Ao, Bo, sel, tol_sums=TOL_SUMS_SHIFTED)
    n, dx, dt = plan.n_maps, plan.P - 1, plan.d_t
    with pytest.raises(cb.CacheBridgeError, match="CB_ERR_INVALID_ARGUMENT"):
        cb.cb_stats_accumulate_shifted(plan, src, tgt, w, s1, s1, A1, B1)
    with pytest.raises(cb.CacheBridgeError, match="CB_ERR_INVALID_ARGUMENT"):
        cb.cb_stats_shift_finish(plan, s1, s1, A1, B1)
    plan.close()


def test_centered_qwen50_full_size_sampled_maps(cb):
    wl = synth.WORKLOADS["qwen50"]
    say(f"{wl.name}: generating {wl.n_seqs} x {wl.seq_len} tokens")
    src, tgt, w = make_inputs(wl)
    hm = synth.head_map(wl)
    plan = cb.cb_plan_create(hm, src, tgt, wl.n_seqs * wl.seq_len)
    say(f"{wl.name}: GPU centered statistics")
    sums, A, B = gpu_centered(cb, plan, [(src, tgt, w)])
    sel = sample_maps(wl.n_maps, 8, seed=1)
    say(f"{wl.name}: centered oracle on maps {sel}")
    so, Ao, Bo = oracle_centered_sel(hm, sel, src, tgt, w)
    check_centered(sums, A, B, so, Ao, Bo, sel)
    check_centered_maps(cb, sums, A, B, so, Ao, Bo, sel, wl.lam_rel)
    del src, tgt, w
    plan.close()


# ----------------------------------------------------------------------------- layer-selection probes

TOL_R2 = 1e-5          # absolute, R^2 in [0, 1]


def probe_head_map(L_t, L_s, H):
    """Every target (layer, head, K/V) paired with every source layer, same head."""
    hm = {k: [] for k in ("tgt_layer", "tgt_head", "kv", "src_layer", "src_head", "weight_row")}
    for l in range(L_t):
        for j in range(L_s):
            for z in range(2):
                for h in range(H):
                    for k, v in zip(hm, (l, h, z, j, h, l * H + h)):
                        hm[k].append(v)
    return {k: np.asarray(v, np.int32) for k, v in hm.items()}


def gpu_probe(cb, plan, src, tgt, w, lam=0.0, flags=0):
    n, ds, dt = plan.n_maps, plan.d_s, plan.d_t
    sums = torch.empty((n, 1 + ds + dt), dtype=torch.float64, device="cuda")
    sq = torch.empty((n, ds + dt), dtype=torch.float64, device="cuda")
    A = torch.empty((n, ds, ds), dtype=torch.float32, device="cuda")
    B = torch.empty((n, ds, dt), dtype=torch.float32, device="cuda")
    cb.cb_stats_zero_centered(plan, sums, A, B, sq=sq)
    cb.cb_stats_means(plan, src, tgt, w, sums, sq=sq)
    cb.cb_stats_accumulate_centered(plan, src, tgt, w, sums, A, B)
    maps, info = gpu_solve_centered(cb, sums, A, B, lam, flags)
    r2 = torch.empty((n,), dtype=torch.float64, device="cuda")
    cb.cb_probe_r2(sums, sq, A, B, maps, r2)
    torch.cuda.synchronize()
    return sums, sq, A, B, maps, info, r2


@pytest.mark.parametrize("d_s,d_t", [(64, 64), (128, 96)])
def test_probe_r2_and_layer_selection(cb, d_s, d_t):
    # targets are generated from source layers round(l * 3 / 2) = [0, 2, 3];
    # the probes fit every (target layer, source layer) pair by OLS
    L_s, L_t, H = 4, 3, 2
    wl = synth.Workload("probe", L_s, H, d_s, L_t, H, d_t, 4, 300, "qwen", "offset", 0.3, "lognormal")
    src, tgt, w = make_inputs(wl)
    hm = probe_head_map(L_t, L_s, H)
    plan = cb.cb_plan_create(hm, src, tgt, wl.n_seqs * wl.seq_len)
    sums, sq, A, B, maps, info, r2 = gpu_probe(cb, plan, src, tgt, w)
    assert (info.cpu().numpy() == 0).all()
    n = len(hm["kv"])
    sel = list(range(n))
    chm, xb, ss, yb, ts, ws, Bn, T = compact(hm, sel, src, tgt, w)
    sqo = oracle.weighted_squares(chm, xb, ss, d_s, yb, ts, d_t, ws, Bn * T, Bn, T, n_threads=NTHREADS)
    esq = max(relF(sq[m].cpu().numpy(), sqo[m]) for m in sel)
    so, Ao, Bo = oracle.stats_centered(chm, xb, ss, d_s, yb, ts, d_t, ws, Bn * T, Bn, T, n_threads=NTHREADS)
    # every map's (sum w, sum w x, sum w y), including the maps whose target sums another map carries
    esum = max(relF(sums[m].cpu().numpy(), so[m]) for m in sel)
    Wo, io = oracle.ridge_solve_centered(so, Ao, Bo, 0.0, relative=False, n_threads=NTHREADS)
    assert (io == 0).all()
    r2o = oracle.probe_r2(chm, Wo, xb, ss, d_s, yb, ts, d_t, ws, Bn * T, Bn, T, n_threads=NTHREADS)
    # the R^2 kernel alone: the GPU's R^2 from the oracle's sums, squares, moments (fp32) and maps
    # (fp32) against the oracle's residual pass over the data with the same maps
    (At, _), (Bt, _), (Wt, W64) = shared_f32(Ao), shared_f32(Bo), shared_f32(Wo)
    r2k = torch.empty((n,), dtype=torch.float64, device="cuda")
    cb.cb_probe_r2(torch.from_numpy(np.ascontiguousarray(so)).to("cuda"),
                   torch.from_numpy(np.ascontiguousarray(sqo)).to("cuda"), At, Bt, Wt, r2k)
    torch.cuda.synchronize()
    r2s = oracle.probe_r2(chm, W64, xb, ss, d_s, yb, ts, d_t, ws, Bn * T, Bn, T, n_threads=NTHREADS)
    g = r2.cpu().numpy()
    e_end, e_alone = float(np.abs(g - r2o).max()), float(np.abs(r2k.cpu().numpy() - r2s).max())
    say(f"  probes: sums relF {esum:.3e}, sq relF {esq:.3e}; R^2 max |diff| end-to-end {e_end:.3e}, "
        f"kernel alone {e_alone:.3e}")
    assert esum <= TOL_SUMS and esq <= TOL_SUMS and e_end <= TOL_R2 and e_alone <= TOL_R2
    # selection: the planted layer first on both sides; the full order agrees
    # wherever the oracle's scores are separated by more than the R^2 bar
    selg, scg = cb.cb_select_layers(hm, g, L_t, L_s, L_s)
    selo, sco = oracle.select_layers(hm, r2o, L_t, L_s, L_s)
    planted = [synth._round_ratio(l, L_s - 1, L_t - 1) for l in range(L_t)]
    assert selg[:, 0].tolist() == planted and selo[:, 0].tolist() == planted
    for l in range(L_t):
        for a in range(L_s - 1):
            if sco[l, selo[l, a]] - sco[l, selo[l, a + 1]] > 4 * TOL_R2:
                assert selg[l, a] == selo[l, a]
    assert np.abs(scg - sco).max() <= TOL_R2
    # a plan with repeated targets fits probes but cannot apply them
    with pytest.raises(cb.CacheBridgeError, match="CB_ERR_INVALID_ARGUMENT"):
        cb.cb_apply(plan, maps, src, torch.zeros_like(tgt))
    plan.close()


def test_means_shared_and_distinct_target_sums(cb):
    """Maps that read one target block under one weight row share a single set of
    target sums (and sum w) in the means pass; maps that read it under different
    weight rows do not.  Every map's sums and sums of squares against the oracle."""
    L_s, L_t, H = 3, 2, 2
    wl = synth.Workload("probe", L_s, H, 64, L_t, H, 96, 3, 200, "qwen", "offset", 0.3, "lognormal")
    src, tgt, _ = make_inputs(wl)
    hm = probe_head_map(L_t, L_s, H)
    n = len(hm["kv"])
    base = L_t * H
    wr = hm["weight_row"].copy()
    for m in range(n):                      # odd source layers: a weight row of their own per target
        if hm["src_layer"][m] % 2 == 1:
            wr[m] = base + hm["tgt_layer"][m] * H + hm["tgt_head"][m]
    hm["weight_row"] = wr
    N = wl.n_seqs * wl.seq_len
    g = torch.Generator(device="cuda")
    g.manual_seed(5)
    w = torch.exp(torch.randn((2 * base, N), generator=g, device="cuda"))
    plan = cb.cb_plan_create(hm, src, tgt, N)
    sums = torch.empty((n, 1 + 64 + 96), dtype=torch.float64, device="cuda")
    sq = torch.empty((n, 64 + 96), dtype=torch.float64, device="cuda")
    A = torch.empty((n, 64, 64), dtype=torch.float32, device="cuda")
    B = torch.empty((n, 64, 96), dtype=torch.float32, device="cuda")
    cb.cb_stats_zero_centered(plan, sums, A, B, sq=sq)
    cb.cb_stats_means(plan, src, tgt, w, sums, sq=sq)
    torch.cuda.synchronize()
    sel = list(range(n))
    chm, xb, ss, yb, ts, ws, Bn, T = compact(hm, sel, src, tgt, w)
    so, _, _ = oracle.stats_centered(chm, xb, ss, 64, yb, ts, 96, ws, Bn * T, Bn, T, n_threads=NTHREADS)
    sqo = oracle.weighted_squares(chm, xb, ss, 64, yb, ts, 96, ws, Bn * T, Bn, T, n_threads=NTHREADS)
    esum = max(relF(sums[m].cpu().numpy(), so[m]) for m in sel)
    esq = max(relF(sq[m].cpu().numpy(), sqo[m]) for m in sel)
    say(f"  shared / distinct target sums: sums relF {esum:.3e}, sq relF {esq:.3e}")
    assert esum <= TOL_SUMS and esq <= TOL_SUMS
    plan.close()


def test_probe_qwen_shape_all_layer_pairs_sampled_maps(cb):
    # the selector's real size: 64 target layers x 40 source layers x 8 heads x
    # K/V = 40,960 probes over a 2 x 1024-token calibration slice
    wl = synth.WORKLOADS["qwen50"].with_(n_seqs=2, seq_len=1024)
    say(f"probe: generating {wl.n_seqs} x {wl.seq_len} tokens")
    src, tgt, w = make_inputs(wl)
    hm = probe_head_map(wl.L_t, wl.L_s, wl.H_t)
    n = len(hm["kv"])
    plan = cb.cb_plan_create(hm, src, tgt, wl.n_seqs * wl.seq_len)
    say(f"probe: GPU fit of {n} probes")
    sums, sq, A, B, maps, info, r2 = gpu_probe(cb, plan, src, tgt, w, lam=1e-2, flags=cb.CB_LAMBDA_RELATIVE)
    assert (info.cpu().numpy() == 0).all()
    sel = sample_maps(n, 8, seed=2)
    say(f"probe: oracle on probes {sel}")
    chm, xb, ss, yb, ts, ws, Bn, T = compact(hm, sel, src, tgt, w)
    so, Ao, Bo = oracle.stats_centered(chm, xb, ss, wl.d_s, yb, ts, wl.d_t, ws, Bn * T, Bn, T, n_threads=NTHREADS)
    Wo, _ = oracle.ridge_solve_centered(so, Ao, Bo, 1e-2, relative=True, n_threads=NTHREADS)
    r2o = oracle.probe_r2(chm, Wo, xb, ss, wl.d_s, yb, ts, wl.d_t, ws, Bn * T, Bn, T, n_threads=NTHREADS)
    g = r2.cpu().numpy()[sel]
    e = float(np.abs(g - r2o).max())
    say(f"  probe R^2 max |diff| {e:.3e} (values {np.round(g, 4).tolist()})")
    assert e <= TOL_R2
    # the planted source layer of every target layer ranks first
    selg, _ = cb.cb_select_layers(hm, r2.cpu().numpy(), wl.L_t, wl.L_s, 8)
    planted = [synth._round_ratio(l, wl.L_s - 1, wl.L_t - 1) for l in range(wl.L_t)]
    assert selg[:, 0].tolist() == planted
    del src, tgt, w
    plan.close()


# ----------------------------------------------------------------------------- attention-aligned weights

TOL_ATTN = 1e-4        # raw sensitivities and weights: relative Frobenius error per row


def gpu_attn(cb, tgt, q, bounds, stride, p):
    L, _, B, H, T, _ = tgt.shape
    r = torch.empty((2 * L * H, B * T), dtype=torch.float32, device="cuda")
    cb.cb_attn_sensitivity(tgt, q, bounds, stride, r)
    w = torch.empty_like(r)
    alpha = torch.empty((2 * L * H,), dtype=torch.float32, device="cuda")
    cb.cb_attn_weights(r, B, T, stride, p, w, alpha)
    torch.cuda.synchronize()
    return r.double().cpu().numpy(), w.double().cpu().numpy(), alpha.double().cpu().numpy()


def oracle_attn(tgt, q, bounds, stride, p):
    L, _, B, H, T, d = tgt.shape
    tc, qc = tgt.contiguous(), q.contiguous()
    r = oracle.attn_sensitivity(bits(tc), tc.stride()[:5], L, H, d, B, T, bits(qc), qc.stride()[:4], q.shape[3],
                                bounds, stride, n_threads=NTHREADS).reshape(2 * L * H, B * T)
    w, alpha = oracle.attn_weights(r, B, T, stride, p)
    return r, w, alpha


def check_attn(rg, wg, ag, ro, wo, ao, label=""):
    er = max(relF(rg[i], ro[i]) for i in range(ro.shape[0]))
    ew = max(relF(wg[i], wo[i]) for i in range(wo.shape[0]))
    ea = float(np.abs(ag - ao).max())
    say(f"  attention weights{label}: max relF r {er:.3e}, w {ew:.3e}; max |alpha diff| {ea:.2e} "
        f"(alpha {ao.min():.3f}..{ao.max():.3f})")
    assert er <= TOL_ATTN and ew <= TOL_ATTN and ea <= 1e-5


@pytest.mark.parametrize("d,G,stride", [(64, 2, 1), (64, 8, 4), (128, 2, 4), (128, 8, 1)])
def test_attn_weights_small(cb, d, G, stride):
    # 100-token sequences (a ragged last key tile), 8 boundaries from 3 to 99
    wl = synth.Workload("attn", 2, 2, d, 2, 2, d, 2, 100, "qwen", "scaled", 0.1, "lognormal")
    src, tgt, _ = make_inputs(wl)
    bounds = synth.attn_boundaries(wl.seq_len, 8, 3)
    q = synth.gen_queries(wl, tgt, G * wl.H_t, len(bounds), device="cuda")
    rg, wg, ag = gpu_attn(cb, tgt, q, bounds, stride, p=d)
    ro, wo, ao = oracle_attn(tgt, q, bounds, stride, p=d)
    check_attn(rg, wg, ag, ro, wo, ao)
    assert not rg[:, (wl.seq_len - 1)::wl.seq_len].any()      # the last token is in no prefix


@pytest.mark.parametrize("d,G,bounds,T,stride", [
    (128, 4, [0, 5, 31, 32, 33, 100, 640, 1999, 2999], 3000, 3),     # a partial row tile; boundary 0
    (64, 32, [7, 40, 90, 150, 260, 400, 555, 699], 700, 1),          # eight tiles of one boundary each
    (128, 1, "geom", 4096, 4),                                       # two tiles, 64 boundaries, long keys
    (128, 16, [511, 512, 513, 1023], 1024, 2),                        # two equal-length tiles
])
def test_attn_weights_work_splits(cb, d, G, bounds, T, stride):
    # boundary sets that drive the key split differently (short-tile pass,
    # tiles split over several waves, merges of partial sums)
    wl = synth.Workload("attns", 2, 1, d, 2, 1, d, 2, T, "qwen", "scaled", 0.1, "lognormal")
    src, tgt, _ = make_inputs(wl)
    del src
    if bounds == "geom":
        bounds = np.unique(np.rint(np.geomspace(1, T - 1, 64)).astype(np.int32))
        bounds = np.concatenate([bounds, np.arange(T - 1 - (64 - len(bounds)), T - 1)])
        bounds = np.unique(bounds)[:64]
    bounds = np.asarray(bounds, dtype=np.int32)
    q = synth.gen_queries(wl, tgt, G * wl.H_t, len(bounds), device="cuda")
    say(f"attn split: d={d} G={G} {len(bounds)} boundaries up to {int(bounds[-1])}, T={T}, stride {stride}")
    rg, wg, ag = gpu_attn(cb, tgt, q, bounds, stride, p=d)
    ro, wo, ao = oracle_attn(tgt, q, bounds, stride, p=d)
    check_attn(rg, wg, ag, ro, wo, ao)


def test_attn_weights_paper_configuration(cb):
    # Sec. 4.1: 1,024-token sequences, 32 boundaries from 12 to 1,023, every
    # fourth token; eight query heads per KV head (64 / 8), d = 128
    wl = synth.Workload("attnp", 2, 2, 128, 2, 2, 128, 2, 1024, "qwen", "scaled", 0.1, "lognormal")
    src, tgt, _ = make_inputs(wl)
    bounds = synth.attn_boundaries(1024)
    assert len(bounds) == 32 and bounds[0] == 12 and bounds[-1] == 1023
    q = synth.gen_queries(wl, tgt, 8 * wl.H_t, len(bounds), device="cuda")
    rg, wg, ag = gpu_attn(cb, tgt, q, bounds, 4, p=128)
    ro, wo, ao = oracle_attn(tgt, q, bounds, 4, p=128)
    check_attn(rg, wg, ag, ro, wo, ao)
    # the weights feed the statistics unchanged: G, C with them match the oracle
    hm = synth.head_map(wl)
    hm["weight_row"] = np.arange(wl.n_maps, dtype=np.int32)   # map m = (l*2 + z)*H + h uses row m
    plan = cb.cb_plan_create(hm, src, tgt, wl.n_seqs * wl.seq_len)
    wt = torch.as_tensor(wg, dtype=torch.float32, device="cuda")
    G_, C_ = gpu_stats(cb, plan, src, tgt, wt)
    sel = list(range(wl.n_maps))
    Go, Co = oracle_stats_sel(hm, sel, src, tgt, wt)
    check_stats(G_, C_, Go, Co, sel)
    plan.close()


def test_attn_weights_qwen_shape_sampled_heads(cb):
    # the 64-layer x 8-KV-head target of the qwen workloads at 2,048 tokens,
    # 32 boundaries from 12 to 2,047, every token; oracle on sampled (layer, head)
    wl = synth.WORKLOADS["qwen50"].with_(n_seqs=2)
    say(f"attn: generating {wl.n_seqs} x {wl.seq_len} tokens")
    src, tgt, _ = make_inputs(wl)
    del src
    bounds = synth.attn_boundaries(wl.seq_len)
    q = synth.gen_queries(wl, tgt, 8 * wl.H_t, len(bounds), device="cuda")
    say("attn: GPU")
    rg, wg, ag = gpu_attn(cb, tgt, q, bounds, 1, p=wl.d_s)
    for (l, h) in ((0, 0), (37, 5), (63, 7)):
        say(f"attn: oracle on layer {l}, head {h}")
        ro, wo, ao = oracle_attn(tgt[l:l + 1, :, :, h:h + 1], q[l:l + 1, :, :, 8 * h:8 * h + 8], bounds, 1, p=wl.d_s)
        rows = [(l * 2 + z) * wl.H_t + h for z in (0, 1)]
        check_attn(rg[rows], wg[rows], ag[rows], ro, wo, ao, f" (layer {l}, head {h})")


# ----------------------------------------------------------------------------- rotary positions

def gpu_rope_table(cb, theta, d, n_pos):
    t = torch.empty((n_pos, d // 2, 2), dtype=torch.float32, device="cuda")
    cb.cb_rope_table(theta, d, n_pos, t)
    return t


def check_bits_close(g, o, label, min_equal=0.999):
    dist = ulp_distance(g, o)
    same = float((dist == 0).mean())
    say(f"  rope{label}: bitwise-equal {same:.6f}, max ulp distance {int(dist.max())}")
    assert dist.max() <= 1 and same >= min_equal


@pytest.mark.parametrize("d,style,inverse", [(64, 0, False), (128, 0, True), (128, 1, False), (64, 1, True)])
def test_rope_matches_oracle(cb, d, style, inverse):
    wl = synth.Workload("rope", 2, 3, d, 1, 1, 64, 2, 77, "qwen", "scaled", 0.1, "lognormal")
    x = synth.gen_source(wl, device="cuda")
    theta, off = (1e6 if style == 0 else 1e4), 7
    table = gpu_rope_table(cb, theta, d, off + wl.seq_len)
    ref = oracle.rope(bits(x), x.stride()[:5], wl.L_s, wl.H_s, d, wl.n_seqs, wl.seq_len, theta, style,
                      inverse=inverse, pos_offset=off)
    out = torch.empty_like(x)
    cb.cb_rope(x, out, table, style, inverse, off)
    torch.cuda.synchronize()
    check_bits_close(bits(out).reshape(ref.shape), ref, f" d={d} style={style} inverse={inverse}")
    # permuted-layout views give the same bits, and so does the in-place form
    xp = x.permute(0, 1, 3, 2, 4, 5).contiguous().permute(0, 1, 3, 2, 4, 5)
    op = torch.empty_like(xp)
    cb.cb_rope(xp, op, table, style, inverse, off)
    cb.cb_rope(xp, xp, table, style, inverse, off)
    torch.cuda.synchronize()
    assert torch.equal(op, out) and torch.equal(xp, out)


def rotated_caches(cb, wl, ts, tt, style, off, hm_override=None):
    """Caches as a model holds them: content rows generated for wl, then their K
    rows turned by the oracle's RoPE (source base ts, target base tt) at
    positions off + tok; returned as device tensors with their host bits."""
    src_c, tgt_c, w = make_inputs(wl)
    as_bf16 = lambda b: torch.from_numpy(b.view(np.int16)).to("cuda").view(torch.bfloat16)  # noqa: E731
    sb = oracle.rope(bits(src_c), src_c.stride()[:5], wl.L_s, wl.H_s, wl.d_s, wl.n_seqs, wl.seq_len, ts, style,
                     pos_offset=off)
    tb = oracle.rope(bits(tgt_c), tgt_c.stride()[:5], wl.L_t, wl.H_t, wl.d_t, wl.n_seqs, wl.seq_len, tt, style,
                     pos_offset=off)
    return as_bf16(sb), as_bf16(tb), w, sb, tb


@pytest.mark.parametrize("d,style,T,off,sides,kind", [
    (128, 0, 256, 0, "both", "qwen"),          # whole tiles, shared-source items
    (128, 1, 300, 37, "both", "qwen"),         # ragged last tile, interleaved pairs
    (128, 0, 200, 900, "both", "odd"),         # an odd map count: a single-map item with copy-only waves
    (64, 0, 200, 1000, "src", "identity"),     # only the source turns
    (64, 1, 96, 5, "tgt", "qwen"),             # only the target turns
])
def test_stats_rope_fused_equals_separate_passes_and_oracle(cb, d, style, T, off, sides, kind):
    # the de-rotation folded into the gather gives bit for bit the moments of
    # cb_rope(inverse) copies, and matches the oracle's composition (rope
    # inverse in fp64, one rounding, then the moments)
    wl = synth.Workload("strope", 4 if kind == "identity" else 3, 2, d, 4, 2, d, 3, T,
                        "qwen" if kind == "odd" else kind, "scaled", 0.1, "lognormal")
    ts, tt = 1e4, 1e6
    src, tgt, w, sb, tb = rotated_caches(cb, wl, ts, tt, style, off)
    hm = synth.head_map(wl)
    if kind == "odd":
        hm = {f: v[[0, 3, 6, 9, 12]] for f, v in hm.items()}          # five maps
    plan = cb.cb_plan_create(hm, src, tgt, wl.n_seqs * T)
    tab_s = gpu_rope_table(cb, ts, d, off + T)
    tab_t = gpu_rope_table(cb, tt, d, off + T)
    sr = cb.rope_spec(tab_s, style, off) if sides in ("both", "src") else None
    tr = cb.rope_spec(tab_t, style, off) if sides in ("both", "tgt") else None
    say(f"stats rope d={d} style={style} T={T} off={off} sides={sides} maps={plan.n_maps}")
    n, P = plan.n_maps, plan.P
    G = torch.empty((n, P, P), dtype=torch.float32, device="cuda")
    C = torch.empty((n, P, d), dtype=torch.float32, device="cuda")
    cb.cb_stats_zero(plan, G, C)
    cb.cb_stats_accumulate_rope(plan, src, tgt, w, G, C, sr, tr)
    # separate passes: de-rotated copies, then the plain kernel
    src_d = src.clone()
    tgt_d = tgt.clone()
    if sr is not None:
        cb.cb_rope(src, src_d, tab_s, style, True, off)
    if tr is not None:
        cb.cb_rope(tgt, tgt_d, tab_t, style, True, off)
    G2, C2 = gpu_stats(cb, plan, src_d, tgt_d, w)
    torch.cuda.synchronize()
    # oracle: the composition in fp64
    so = sb if sr is None else oracle.rope(sb, src.stride()[:5], wl.L_s, wl.H_s, d, wl.n_seqs, T, ts, style,
                                           inverse=True, pos_offset=off)
    to = tb if tr is None else oracle.rope(tb, tgt.stride()[:5], wl.L_t, wl.H_t, d, wl.n_seqs, T, tt, style,
                                           inverse=True, pos_offset=off)
    Go, Co = oracle.stats(hm, so, src.stride()[:5], d, to, tgt.stride()[:5], d, w.cpu().numpy(),
                          wl.n_seqs * T, wl.n_seqs, T, n_threads=NTHREADS)
    # The products (G and C without their bias row and column) are bit for bit
    # those of the separate passes; the fp32 bias sums (sum w, sum w x, sum w y)
    # may round differently between the two compiled kernels, by a few fp32
    # ulps of each sum (2^-24 ~ 6e-8 relative), which bounds the whole matrix.
    eb = max(max(relF(G[m].double().cpu().numpy(), G2[m].double().cpu().numpy()),
                 relF(C[m].double().cpu().numpy(), C2[m].double().cpu().numpy())) for m in range(n))
    same = torch.equal(G[:, :P - 1, :P - 1], G2[:, :P - 1, :P - 1]) and torch.equal(C[:, :P - 1], C2[:, :P - 1])
    say(f"  fused vs separate: products bitwise {same}, G and C relF {eb:.2e}")
    assert same and eb <= 1e-7
    check_stats(G, C, Go, Co, list(range(n)))
    # the keys did turn: the moments of the rotated caches as they are differ
    G3, _ = gpu_stats(cb, plan, src, tgt, w)
    kmaps = [m for m in range(n) if hm["kv"][m] == 0]
    vmaps = [m for m in range(n) if hm["kv"][m] == 1]
    assert not torch.equal(G[kmaps], G3[kmaps])
    assert torch.equal(G[vmaps][:, :P - 1, :P - 1], G3[vmaps][:, :P - 1, :P - 1])
    plan.close()


def test_stats_rope_qwen50_full_size_sampled_maps(cb):
    """The fused de-rotation at the 14B->32B shape (50 x 2048 tokens, 1024 maps, one
    call): the synthetic caches are taken as caches whose keys carry RoPE (source
    base 1e4, target base 1e6); eight sampled maps against the oracle's composition
    (its fp64 inverse turn of those rows, then its moments)."""
    wl = synth.WORKLOADS["qwen50"]
    say(f"{wl.name}: generating {wl.n_seqs} x {wl.seq_len} tokens")
    src, tgt, w = make_inputs(wl)
    hm = synth.head_map(wl)
    plan = cb.cb_plan_create(hm, src, tgt, wl.n_seqs * wl.seq_len)
    ts_, tt_ = 1e4, 1e6
    tab_s, tab_t = gpu_rope_table(cb, ts_, wl.d_s, wl.seq_len), gpu_rope_table(cb, tt_, wl.d_t, wl.seq_len)
    n, P = plan.n_maps, plan.P
    G = torch.empty((n, P, P), dtype=torch.float32, device="cuda")
    C = torch.empty((n, P, wl.d_t), dtype=torch.float32, device="cuda")
    cb.cb_stats_zero(plan, G, C)
    say(f"{wl.name}: GPU statistics with the de-rotation fused")
    cb.cb_stats_accumulate_rope(plan, src, tgt, w, G, C, cb.rope_spec(tab_s), cb.rope_spec(tab_t))
    torch.cuda.synchronize()
    sel = sample_maps(wl.n_maps, 8, seed=5)
    say(f"{wl.name}: oracle on maps {sel}")
    chm, xb, ss, yb, ts, ws, B, T = compact(hm, sel, src, tgt, w)
    m = len(sel)
    xd = oracle.rope(xb, ss, m, 1, wl.d_s, B, T, ts_, 0, inverse=True)[:, 0:1]
    yd = oracle.rope(yb, ts, m, 1, wl.d_t, B, T, tt_, 0, inverse=True)[:, 0:1]
    for i, mm in enumerate(sel):                   # V maps carry no positions
        if hm["kv"][mm] == 1:
            xd[i], yd[i] = xb[i], yb[i]
    Go, Co = oracle.stats(chm, np.ascontiguousarray(xd), ss, wl.d_s, np.ascontiguousarray(yd), ts, wl.d_t, ws,
                          B * T, B, T, n_threads=NTHREADS)
    check_stats(G, C, Go, Co, sel)
    del src, tgt, w
    plan.close()


def test_stats_rope_rejects_what_it_cannot_fuse(cb):
    wl = synth.Workload("strope96", 2, 2, 96, 2, 2, 128, 2, 64, "qwen", "scaled", 0.1, "lognormal")
    src, tgt, w = make_inputs(wl)
    plan = cb.cb_plan_create(synth.head_map(wl), src, tgt, 1024)
    G = torch.zeros((plan.n_maps, plan.P, plan.P), dtype=torch.float32, device="cuda")
    C = torch.zeros((plan.n_maps, plan.P, plan.d_t), dtype=torch.float32, device="cuda")
    tab96, tab128 = gpu_rope_table(cb, 1e4, 96, 64), gpu_rope_table(cb, 1e4, 128, 64)
    with pytest.raises(cb.CacheBridgeError, match="CB_ERR_UNSUPPORTED"):
        cb.cb_stats_accumulate_rope(plan, src, tgt, w, G, C, cb.rope_spec(tab96), None)
    with pytest.raises(cb.CacheBridgeError, match="CB_ERR_SHAPE"):
        cb.cb_stats_accumulate_rope(plan, src, tgt, w, G, C, cb.rope_spec(tab128), None)   # d_s is 96
    with pytest.raises(cb.CacheBridgeError, match="CB_ERR_SHAPE"):
        cb.cb_stats_accumulate_rope(plan, src, tgt, w, G, C, None, cb.rope_spec(tab128[:63]))
    torch.cuda.synchronize()
    assert not G.any() and not C.any()
    plan.close()


def check_apply_rotated(ob, ref, label=""):
    """check_apply for caches whose K rows (kv 0) were rotated after rounding:
    a difference of one bf16 ulp in a pair before the rotation moves both rotated
    elements by up to one ulp of the pair's norm, which can be many ulps of a
    small element, so K rows get ulp(element) + ulp(pair norm) + 1e-4 of the
    map's RMS; V rows keep the bound of check_apply."""
    g = oracle.bf16_to_double(ob)
    r = oracle.bf16_to_double(ref)
    e = relF(g, r)
    h = r.shape[-1] // 2
    pn = np.hypot(r[..., :h], r[..., h:])
    pn = np.concatenate([pn, pn], axis=-1)
    ulp = lambda x: np.spacing(np.abs(x).astype(np.float32)).astype(np.float64) * 65536.0  # noqa: E731
    rms = np.sqrt((r * r).mean(axis=(2, 4, 5), keepdims=True))
    bound = ulp(r) + 1e-4 * rms
    bound[:, 0] += ulp(pn[:, 0])
    worst = float((np.abs(g - r) / bound).max())
    same = float((ob == ref).mean())
    say(f"  apply parity{label}: relF {e:.3e}, bitwise-equal {same:.6f}, worst err/bound {worst:.3f}")
    assert e <= TOL_APPLY and worst <= 1.0


@pytest.mark.parametrize("d_s,d_t,style,off", [(128, 128, 0, 0), (128, 128, 1, 11), (64, 96, 0, 5),
                                                (96, 64, 1, 0), (128, 64, 0, 3000)])
def test_apply_rope_matches_oracle(cb, d_s, d_t, style, off):
    # three token tiles of 256 with a ragged 88-token tail; K outputs turned
    # by the target RoPE before the single rounding, V outputs as cb_apply
    wl = synth.Workload("aprope", 3, 2, d_s, 4, 2, d_t, 2, 300, "qwen", "scaled", 0.1, "lognormal")
    src = synth.gen_source(wl, device="cuda")
    hm = synth.head_map(wl)
    theta = 1e6 if style == 0 else 1e4
    table = gpu_rope_table(cb, theta, d_t, off + wl.seq_len)
    plan = cb.cb_plan_create(hm, (wl.L_s, wl.H_s, wl.d_s), (wl.L_t, wl.H_t, wl.d_t), 1024)
    maps = synth.planted_maps(wl, device="cuda")
    out = torch.zeros((wl.L_t, 2, wl.n_seqs, wl.H_t, wl.seq_len, d_t), dtype=torch.bfloat16, device="cuda")
    plain = torch.zeros_like(out)
    say(f"apply_rope d_s={d_s} d_t={d_t} style={style} offset={off}")
    cb.cb_apply_rope(plan, maps, src, out, cb.rope_spec(table, style, off))
    cb.cb_apply(plan, maps, src, plain)
    torch.cuda.synchronize()
    ref = np.zeros(tuple(out.shape), dtype=np.uint16)
    oracle.apply_rope(hm, maps.double().cpu().numpy(), bits(src), src.stride()[:5], d_s, ref,
                      tuple(out.stride()[:5]), d_t, wl.n_seqs, wl.seq_len, theta, style, off, n_threads=NTHREADS)
    ob = bits(out).reshape(ref.shape)
    check_apply(ob, ref, f" (fused rope, style {style})")
    assert np.array_equal(ob[:, 1], bits(plain).reshape(ref.shape)[:, 1])     # V: bitwise cb_apply
    assert not np.array_equal(ob[:, 0], bits(plain).reshape(ref.shape)[:, 0])
    with pytest.raises(cb.CacheBridgeError, match="CB_ERR_SHAPE"):
        cb.cb_apply_rope(plan, maps, src, out, cb.rope_spec(table[: off + wl.seq_len - 1], style, off))
    plan.close()


@pytest.mark.parametrize("d_s,d_t,style,off,tgt_too", [(128, 128, 0, 0, False), (128, 128, 1, 11, True),
                                                        (64, 96, 0, 5, False), (64, 64, 0, 3000, True),
                                                        (128, 64, 1, 700, False)])
def test_apply_rope_source_derotation(cb, d_s, d_t, style, off, tgt_too):
    # a sender whose keys carry RoPE: turning its K rows back as they land gives
    # the mapping of cb_rope(inverse) copies, and matches the oracle's composition
    # (rope inverse in fp64, one rounding, then the mapping, with the target
    # rotation when asked)
    wl = synth.Workload("srope", 3, 2, d_s, 4, 2, d_t, 2, 300, "qwen", "scaled", 0.1, "lognormal")
    src_c = synth.gen_source(wl, device="cuda")
    ts, tt = 1e4, 1e6
    sb = oracle.rope(bits(src_c), src_c.stride()[:5], wl.L_s, wl.H_s, d_s, wl.n_seqs, wl.seq_len, ts, style,
                     pos_offset=off)
    src = torch.from_numpy(sb.view(np.int16)).to("cuda").view(torch.bfloat16)
    hm = synth.head_map(wl)
    plan = cb.cb_plan_create(hm, (wl.L_s, wl.H_s, d_s), (wl.L_t, wl.H_t, d_t), 1024)
    maps = synth.planted_maps(wl, device="cuda")
    tab_s = gpu_rope_table(cb, ts, d_s, off + wl.seq_len)
    tab_t = gpu_rope_table(cb, tt, d_t, off + wl.seq_len)
    sr = cb.rope_spec(tab_s, style, off)
    tr = cb.rope_spec(tab_t, style, off) if tgt_too else None
    say(f"apply source de-rotation d_s={d_s} d_t={d_t} style={style} off={off} target rotation={tgt_too}")
    out = torch.zeros((wl.L_t, 2, wl.n_seqs, wl.H_t, wl.seq_len, d_t), dtype=torch.bfloat16, device="cuda")
    cb.cb_apply_rope(plan, maps, src, out, tr, sr)
    src_d = torch.empty_like(src)
    cb.cb_rope(src, src_d, tab_s, style, True, off)
    sep = torch.zeros_like(out)
    cb.cb_apply_rope(plan, maps, src_d, sep, tr)
    torch.cuda.synchronize()
    # the fused turn forms its angles by angle addition (about 1.5 fp32 ulp from
    # the table's), so a share p ~ 3 * 2^-16 of the de-rotated inputs lies one
    # bf16 ulp (2^-8) from cb_rope's: outputs then differ by about
    # sqrt(p) * 2^-8 ~ 3e-5 relative; the bar is 1e-4
    same = float((bits(out) == bits(sep)).mean())
    es = relF(oracle.bf16_to_double(bits(out)), oracle.bf16_to_double(bits(sep)))
    say(f"  fused vs separate passes: bitwise-equal {same:.6f}, relF {es:.2e}")
    assert same >= 0.999 and es <= 1e-4
    so = oracle.rope(sb, src.stride()[:5], wl.L_s, wl.H_s, d_s, wl.n_seqs, wl.seq_len, ts, style, inverse=True,
                     pos_offset=off)
    ref = np.zeros(tuple(out.shape), dtype=np.uint16)
    W = maps.double().cpu().numpy()
    if tgt_too:
        oracle.apply_rope(hm, W, so, src.stride()[:5], d_s, ref, tuple(out.stride()[:5]), d_t, wl.n_seqs,
                          wl.seq_len, tt, style, off, n_threads=NTHREADS)
    else:
        oracle.apply(hm, W, so, src.stride()[:5], d_s, ref, tuple(out.stride()[:5]), d_t, wl.n_seqs, wl.seq_len,
                     n_threads=NTHREADS)
    # The oracle turns the sender back in fp64, the kernel in fp32: a few inputs
    # differ by one bf16 ulp (test_rope_matches_oracle), so the element-wise
    # bound of check_apply (which assumes equal inputs) does not apply here.
    # The element-wise bars are carried by that test and by
    # test_apply_rope_matches_oracle on equal inputs; the composition is held
    # to the relative bar and to a bitwise-equal share.
    ob = bits(out).reshape(ref.shape)
    e = relF(oracle.bf16_to_double(ob), oracle.bf16_to_double(ref))
    eq = float((ob == ref).mean())
    say(f"  against the oracle's composition: relF {e:.3e}, bitwise-equal {eq:.6f}")
    assert e <= TOL_APPLY and eq >= 0.99
    plan.close()


def test_apply_rope_source_derotation_rejects_d96(cb):
    wl = synth.Workload("srope96", 2, 2, 96, 2, 2, 128, 2, 64, "qwen", "scaled", 0.1, "lognormal")
    src = synth.gen_source(wl, device="cuda")
    plan = cb.cb_plan_create(synth.head_map(wl), (wl.L_s, wl.H_s, 96), (wl.L_t, wl.H_t, 128), 1024)
    maps = synth.planted_maps(wl, device="cuda")
    out = torch.zeros((wl.L_t, 2, wl.n_seqs, wl.H_t, wl.seq_len, 128), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(cb.CacheBridgeError, match="CB_ERR_UNSUPPORTED"):
        cb.cb_apply_rope(plan, maps, src, out, None, cb.rope_spec(gpu_rope_table(cb, 1e4, 96, 64)))
    with pytest.raises(cb.CacheBridgeError, match="CB_ERR_SHAPE"):
        cb.cb_apply_rope(plan, maps, src, out, None, cb.rope_spec(gpu_rope_table(cb, 1e4, 128, 64)))
    torch.cuda.synchronize()
    assert not out.view(torch.int16).any()
    plan.close()


def test_apply_rope_edge_cases(cb):
    # an empty sender changes nothing; one token at position 0 equals cb_apply;
    # an unknown style is rejected before anything is enqueued
    wl = synth.Workload("aprope1", 2, 2, 64, 2, 2, 64, 3, 1, "qwen", "scaled", 0.1, "lognormal")
    src = synth.gen_source(wl, device="cuda")
    hm = synth.head_map(wl)
    plan = cb.cb_plan_create(hm, (wl.L_s, wl.H_s, wl.d_s), (wl.L_t, wl.H_t, wl.d_t), 1024)
    maps = synth.planted_maps(wl, device="cuda")
    table = gpu_rope_table(cb, 1e4, wl.d_t, 4)
    out = torch.full((wl.L_t, 2, wl.n_seqs, wl.H_t, 1, wl.d_t), 7.0, dtype=torch.bfloat16, device="cuda")
    keep = out.clone()
    cb.cb_apply_rope(plan, maps, src[:, :, :0], out[:, :, :0], table)
    torch.cuda.synchronize()
    assert torch.equal(out, keep)
    plain = torch.zeros_like(out)
    for style in (0, 1):
        cb.cb_apply_rope(plan, maps, src, out, cb.rope_spec(table, style, 0))
        cb.cb_apply(plan, maps, src, plain)
        torch.cuda.synchronize()
        assert torch.equal(out, plain)
    with pytest.raises(cb.CacheBridgeError, match="CB_ERR_INVALID_ARGUMENT"):
        cb.cb_apply_rope(plan, maps, src, out, cb.rope_spec(table, 2, 0))
    with pytest.raises(cb.CacheBridgeError, match="CB_ERR_SHAPE"):
        cb.cb_apply_rope(plan, maps, src, out, cb.rope_spec(table, 0, 4))             # position 4 needs 5 rows
    plan.close()


def test_rope_fit_and_apply_end_to_end(cb):
    # caches as a model holds them: keys carry RoPE (source base 1e4, target base
    # 1e6).  Fit on de-rotated keys, apply on the de-rotated sender, then
    # restore the target's rotation on the mapped keys.
    wl = synth.Workload("ropee", 2, 2, 128, 2, 2, 128, 8, 96, "qwen", "gauss", 0.05, "lognormal")
    src_c, tgt_c, w = make_inputs(wl)
    ts, tt = 1e4, 1e6
    src_rot_b = oracle.rope(bits(src_c), src_c.stride()[:5], wl.L_s, wl.H_s, wl.d_s, wl.n_seqs, wl.seq_len, ts)
    tgt_rot_b = oracle.rope(bits(tgt_c), tgt_c.stride()[:5], wl.L_t, wl.H_t, wl.d_t, wl.n_seqs, wl.seq_len, tt)
    as_bf16 = lambda b: torch.from_numpy(b.view(np.int16)).to("cuda").view(torch.bfloat16)  # noqa: E731
    src_rot, tgt_rot = as_bf16(src_rot_b), as_bf16(tgt_rot_b)
    tab_s = gpu_rope_table(cb, ts, wl.d_s, wl.seq_len)
    tab_t = gpu_rope_table(cb, tt, wl.d_t, wl.seq_len)
    src_g, tgt_g = torch.empty_like(src_rot), torch.empty_like(tgt_rot)
    cb.cb_rope(src_rot, src_g, tab_s, inverse=True)
    cb.cb_rope(tgt_rot, tgt_g, tab_t, inverse=True)
    hm = synth.head_map(wl)
    plan = cb.cb_plan_create(hm, src_g, tgt_g, wl.n_seqs * wl.seq_len)
    G, C = gpu_stats(cb, plan, src_g, tgt_g, w)
    maps, info = gpu_solve(cb, G, C, wl.lam_rel, cb.CB_LAMBDA_RELATIVE | cb.CB_RIDGE_BIAS_UNPENALIZED)
    assert (info.cpu().numpy() == 0).all()
    # oracle: de-rotation, statistics, solve, apply, rotation -- the same steps in fp64
    src_o = oracle.rope(src_rot_b, src_c.stride()[:5], wl.L_s, wl.H_s, wl.d_s, wl.n_seqs, wl.seq_len, ts, inverse=True)
    tgt_o = oracle.rope(tgt_rot_b, tgt_c.stride()[:5], wl.L_t, wl.H_t, wl.d_t, wl.n_seqs, wl.seq_len, tt, inverse=True)
    check_bits_close(bits(src_g).reshape(src_o.shape), src_o, " (source de-rotation)")
    sel = list(range(wl.n_maps))
    Go, Co = oracle.stats(hm, src_o, src_c.stride()[:5], wl.d_s, tgt_o, tgt_c.stride()[:5], wl.d_t,
                          w.cpu().numpy(), wl.n_seqs * wl.seq_len, wl.n_seqs, wl.seq_len, n_threads=NTHREADS)
    check_stats(G, C, Go, Co, sel)
    Wo, _ = oracle.ridge_solve(Go, Co, wl.lam_rel, relative=True, bias_unpenalized=True)
    e = max(relF(maps[i].double().cpu().numpy(), Wo[i]) for i in sel)
    say(f"  maps parity on de-rotated keys: {e:.3e}")
    assert e <= TOL_MAPS
    # mapping with the target rotation restored, on the oracle's maps and de-rotated sender (both sides)
    Wt, W64 = shared_f32(Wo)
    src_ob = as_bf16(src_o)
    out = torch.zeros_like(tgt_rot)
    cb.cb_apply(plan, Wt, src_ob, out)
    cb.cb_rope(out, out, tab_t)
    torch.cuda.synchronize()
    mapped = np.zeros(tuple(out.shape), dtype=np.uint16)
    oracle.apply(hm, W64, src_o, src_c.stride()[:5], wl.d_s, mapped,
                 tuple(out.stride()[:5]), wl.d_t, wl.n_seqs, wl.seq_len)
    ref = oracle.rope(mapped, tuple(out.stride()[:5]), wl.L_t, wl.H_t, wl.d_t, wl.n_seqs, wl.seq_len, tt)
    check_apply_rotated(bits(out).reshape(ref.shape), ref, " (rotated keys)")
    # the fused form rounds once: within check_apply's bound of the oracle's fused result
    fused = torch.zeros_like(tgt_rot)
    cb.cb_apply_rope(plan, Wt, src_ob, fused, tab_t)
    torch.cuda.synchronize()
    ref1 = np.zeros(tuple(out.shape), dtype=np.uint16)
    oracle.apply_rope(hm, W64, src_o, src_c.stride()[:5], wl.d_s, ref1,
                      tuple(out.stride()[:5]), wl.d_t, wl.n_seqs, wl.seq_len, tt)
    check_apply(bits(fused).reshape(ref1.shape), ref1, " (fused target rotation)")
    # the K maps recover the planted content map: fitted without de-rotation they do not
    Gr, Cr = gpu_stats(cb, plan, src_rot, tgt_rot, w)
    mr, _ = gpu_solve(cb, Gr, Cr, wl.lam_rel, cb.CB_LAMBDA_RELATIVE | cb.CB_RIDGE_BIAS_UNPENALIZED)
    planted = synth.planted_maps(wl, device="cuda").cpu()    # the generator make_inputs used
    kmaps = [m for m in sel if hm["kv"][m] == 0]
    e_c = max(relF(maps[m].cpu().numpy(), planted[m].numpy()) for m in kmaps)
    e_r = min(relF(mr[m].cpu().numpy(), planted[m].numpy()) for m in kmaps)
    say(f"  K maps vs the planted content map: de-rotated fit (worst) {e_c:.3e}, rotated fit (best) {e_r:.3e}")
    assert e_c < 0.1 and e_r > 5 * e_c
    plan.close()
