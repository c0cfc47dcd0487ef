"""GPU parity of the multi-layer path (Sec. 3.2, Eq. localfeature with k selected
source layers; P = k d_s + 1) against the fp64 oracle, through the C ABI.

Statistics from cb_stats_accumulate on a cb_plan_create_multi plan, solved by
cb_ridge_solve_ws (blocked fp64 Cholesky), compared with oracle.stats_multi and
oracle.ridge_solve on the exact bits the GPU consumed; cb_apply of the maps
compared with oracle.apply_multi on the same fp32 maps.  Bars (relative
Frobenius error per map): G and C 1e-4, maps 1e-3, applied caches 1e-3 with
every element within one bf16 ulp plus 1e-4 of its map's RMS output; the solver
alone (same fp32 moments on both sides, maps rounded to fp32) 1e-6; G exactly
symmetric.
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
TOL_SOLVER = 1e-6
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


def bits(t):
    return synth.bf16_bits(t)


def random_multi_map(rng, k, L_s, H_s, L_t, H_t):
    hm = {f: [] for f in oracle.MULTI_MAP_FIELDS}
    for l in range(L_t):
        S = [int(v) for v in rng.permutation(L_s)[:k]]
        for z in range(2):
            for h in range(H_t):
                for f, v in zip(oracle.MULTI_MAP_FIELDS, (l, h, z, S, int(rng.integers(H_s)), l * H_t + h)):
                    hm[f].append(v)
    return {f: np.asarray(v, np.int32) for f, v in hm.items()}


def small_inputs(rng, L_s, H_s, L_t, H_t, B, T, d=128, device="cuda"):
    g = torch.Generator(device="cpu")
    g.manual_seed(int(rng.integers(1 << 31)))
    scale = torch.exp(torch.randn((L_s, 2, 1, H_s, 1, d), generator=g))
    src = (torch.randn((L_s, 2, B, H_s, T, d), generator=g) * scale).to(torch.bfloat16)
    tgt = (torch.randn((L_t, 2, B, H_t, T, d), generator=g) * 2.0 + 1.0).to(torch.bfloat16)
    w = torch.exp(torch.randn((L_t * H_t, B * T), generator=g))
    return src.to(device), tgt.to(device), w.to(device)


def gpu_stats(cb, plan, batches, G=None, C=None):
    n, P, dt = plan.n_maps, plan.P, plan.d_t
    if G is None:
        G = torch.empty((n, P, P), dtype=torch.float32, device="cuda")
        C = torch.empty((n, P, dt), dtype=torch.float32, device="cuda")
        cb.cb_stats_zero(plan, G, C)
    for src, tgt, w in batches:
        cb.cb_stats_accumulate(plan, src, tgt, w, G, C)
    torch.cuda.synchronize()
    return G, C


def oracle_stats_full(hm, src, tgt, w, stride, sel=None):
    """Oracle moments of the maps `sel` (all by default) on host copies of the caches."""
    if sel is not None:
        hm = {f: v[sel] for f, v in hm.items()}
    sb, tb = bits(src), bits(tgt)
    L_s, _, B, H_s, T, d_s = src.shape
    L_t, _, _, H_t, _, d_t = tgt.shape
    return oracle.stats_multi(hm, sb, synth.cache_strides(L_s, H_s, B, T, d_s), d_s, tb,
                              synth.cache_strides(L_t, H_t, B, T, d_t), d_t, w.cpu().numpy(), B * T, B, T, stride,
                              n_threads=NTHREADS)


def compact_multi(hm, sel, src, tgt, w, stride):
    """Host copies of only the sampled rows that the maps `sel` read (sliced on the
    device), with a head map onto them; the oracle then runs with stride 1."""
    k = hm["src_layers"].shape[1]
    B, T = src.shape[2], src.shape[4]
    xs, ys, ws = [], [], []
    for m in sel:
        z, a = int(hm["kv"][m]), int(hm["src_head"][m])
        for j in hm["src_layers"][m]:
            xs.append(src[int(j), z, :, a, ::stride])
        ys.append(tgt[int(hm["tgt_layer"][m]), z, :, int(hm["tgt_head"][m]), ::stride])
        ws.append(w[int(hm["weight_row"][m])].reshape(B, T)[:, ::stride].reshape(-1))
    n, Ts = len(sel), xs[0].shape[1]
    d_s, d_t = xs[0].shape[-1], ys[0].shape[-1]
    xb = bits(torch.stack(xs)).reshape(n * k, 1, B, 1, Ts, d_s)
    yb = bits(torch.stack(ys)).reshape(n, 1, B, 1, Ts, d_t)
    wb = torch.stack(ws).cpu().numpy()
    chm = {"tgt_layer": np.arange(n, dtype=np.int32), "tgt_head": np.zeros(n, np.int32),
           "kv": np.zeros(n, np.int32), "src_layers": np.arange(n * k, dtype=np.int32).reshape(n, k),
           "src_head": np.zeros(n, np.int32), "weight_row": np.arange(n, dtype=np.int32)}
    ss = (B * Ts * d_s, 0, Ts * d_s, 0, d_s)          # [layer][1][seq][1][tok][dim]: one component
    ts = (B * Ts * d_t, 0, Ts * d_t, 0, d_t)
    return oracle.stats_multi(chm, xb, ss, d_s, yb, ts, d_t, np.ascontiguousarray(wb), B * Ts, B, Ts, 1,
                              n_threads=NTHREADS)


def check_stats(G, C, Go, Co, sel, tol=TOL_STATS):
    idx = torch.as_tensor(np.asarray(sel), device=G.device)
    Gg = G[idx].double().cpu().numpy()
    Cg = C[idx].double().cpu().numpy()
    eg = max(relF(Gg[i], Go[i]) for i in range(len(sel)))
    ec = max(relF(Cg[i], Co[i]) for i in range(len(sel)))
    say(f"  stats parity: max relF G {eg:.3e}, C {ec:.3e}")
    assert eg <= tol and ec <= tol
    assert np.array_equal(Gg, np.transpose(Gg, (0, 2, 1))), "G must be exactly symmetric"
    return eg, ec


def gpu_solve_ws(cb, G, C, lam=1e-2, flags=None):
    if flags is None:
        flags = cb.CB_LAMBDA_RELATIVE
    n, P, _ = G.shape
    d_t = C.shape[2]
    maps = torch.empty_like(C)
    info = torch.empty((n,), dtype=torch.int32, device="cuda")
    per = cb.cb_ridge_solve_workspace_bytes(P, d_t, 1)
    nsys = max(1, min(n, (8 << 30) // max(per, 1)))
    ws = torch.empty((max(per * nsys, 8),), dtype=torch.uint8, device="cuda")
    cb.cb_ridge_solve_ws(G, C, lam, flags, maps, info, ws)
    torch.cuda.synchronize()
    return maps, info


def shared_f32(a):
    """An array the oracle made, rounded once to fp32: the device tensor the GPU
    call takes and the exact fp64 copy of the same values the oracle takes."""
    a32 = np.ascontiguousarray(np.asarray(a, dtype=np.float32))
    return torch.from_numpy(a32).to("cuda"), a32.astype(np.float64)


def check_solve(cb, G, C, maps, info, Go, Co, sel, unpen, label=""):
    """End to end (the GPU's maps from its own moments against the oracle's solve
    of the oracle's moments) and the solver alone (both sides solve the oracle's
    moments rounded to fp32)."""
    idx = torch.as_tensor(np.asarray(sel), device=G.device)
    Wo, io = oracle.ridge_solve(Go, Co, 1e-2, relative=True, bias_unpenalized=unpen, n_threads=NTHREADS)
    Wg = maps[idx].double().cpu().numpy()
    (Gt, G64), (Ct, C64) = shared_f32(Go), shared_f32(Co)
    flags = cb.CB_LAMBDA_RELATIVE | (cb.CB_RIDGE_BIAS_UNPENALIZED if unpen else 0)
    ms, _ = gpu_solve_ws(cb, Gt, Ct, 1e-2, flags)
    del Gt, Ct
    Ws, _ = oracle.ridge_solve(G64, C64, 1e-2, relative=True, bias_unpenalized=unpen, n_threads=NTHREADS)
    e2e = max(relF(Wg[i], Wo[i]) for i in range(len(sel)))
    alone = max(relF(ms[i].double().cpu().numpy(), Ws[i]) for i in range(len(sel)))
    say(f"  solve{label}: maps relF end-to-end {e2e:.3e}, solver alone {alone:.3e}")
    assert (info[idx].cpu().numpy() == 0).all() and (io == 0).all()
    assert e2e <= TOL_MAPS and alone <= TOL_SOLVER
    return e2e, alone


# ----------------------------------------------------------------------------- small, all maps

def test_multi_tiny_k3_end_to_end(cb):
    wl = synth.WORKLOADS["tiny_k3"]
    say(f"multi tiny_k3: P={wl.P}, {wl.n_seqs} x {wl.seq_len} tokens, stride {wl.sample_stride}")
    src = synth.gen_source(wl, device="cuda")
    tgt = synth.gen_target(wl, src, device="cuda")
    w = synth.gen_weights(wl, device="cuda")
    hm = synth.head_map_multi(wl)
    plan = cb.cb_plan_create_multi(hm, src, tgt, wl.sample_stride)
    assert plan.P == wl.P and plan.k == wl.k
    G, C = gpu_stats(cb, plan, [(src, tgt, w)])
    Go, Co = oracle_stats_full(hm, src, tgt, w, wl.sample_stride)
    sel = list(range(plan.n_maps))
    check_stats(G, C, Go, Co, sel)
    for unpen in (False, True):
        flags = cb.CB_LAMBDA_RELATIVE | (cb.CB_RIDGE_BIAS_UNPENALIZED if unpen else 0)
        maps, info = gpu_solve_ws(cb, G, C, 1e-2, flags)
        check_solve(cb, G, C, maps, info, Go, Co, sel, unpen, " (bias unpenalized)" if unpen else "")
    plan.close()


# T gives at least 2P calibration rows over the 3 sequences (a well-posed fit,
# so the maps bar measures the arithmetic, not the conditioning of a rank-
# deficient problem), with a partial last tile in every sequence.
@pytest.mark.parametrize("k,stride,T", [(1, 1, 100), (2, 3, 520), (3, 4, 1030), (5, 2, 858)])
def test_multi_widths_strides_ragged_tiles_and_batches(cb, k, stride, T):
    rng = np.random.default_rng(1000 + 10 * k + stride)
    L_s, H_s, L_t, H_t, B = 6, 2, 2, 2, 3
    say(f"multi k={k} stride={stride} T={T}")
    src, tgt, w = small_inputs(rng, L_s, H_s, L_t, H_t, B, T)
    hm = random_multi_map(rng, k, L_s, H_s, L_t, H_t)
    plan = cb.cb_plan_create_multi(hm, src, tgt, stride)
    # three uneven batches of sequences, accumulated across calls
    cuts = [(0, 1), (1, 1), (1, 3)]
    batches = [(src[:, :, a:b], tgt[:, :, a:b], w.reshape(-1, B, T)[:, a:b].reshape(w.shape[0], -1))
               for a, b in cuts]
    G, C = gpu_stats(cb, plan, batches)
    Go, Co = oracle_stats_full(hm, src, tgt, w, stride)
    sel = list(range(plan.n_maps))
    check_stats(G, C, Go, Co, sel)
    maps, info = gpu_solve_ws(cb, G, C)
    check_solve(cb, G, C, maps, info, Go, Co, sel, False)
    plan.close()


def test_multi_max_width_k32_stats_and_apply(cb):
    # the widest feature a plan takes: k = 32 source layers, P = 4,097 (two maps,
    # 640 rows in two sequences with ragged tiles): moments and application
    rng = np.random.default_rng(32)
    k, L_s, H_s, L_t, H_t, B, T = 32, 33, 1, 1, 1, 2, 320
    src, tgt, w = small_inputs(rng, L_s, H_s, L_t, H_t, B, T)
    hm = random_multi_map(rng, k, L_s, H_s, L_t, H_t)
    plan = cb.cb_plan_create_multi(hm, src, tgt, 1)
    assert plan.P == 4097 and plan.n_maps == 2
    say(f"multi k=32: P={plan.P}, {B} x {T} tokens")
    G, C = gpu_stats(cb, plan, [(src, tgt, w)])
    Go, Co = oracle_stats_full(hm, src, tgt, w, 1)
    check_stats(G, C, Go, Co, [0, 1])
    maps = random_maps(rng, plan.n_maps, plan.P, plan.d_t)
    out = gpu_apply(cb, plan, maps, src, L_t, H_t)
    ref = oracle_apply_multi(hm, maps, src, L_t, H_t, 128)
    check_apply_multi(bits(out), ref, hm, range(2), " (k=32)")
    plan.close()


def test_multi_wide_solve_p2049_solver_alone(cb):
    # the blocked fp64 solve at P = 2,049 (k = 16) on the oracle's moments of
    # 1,200 rows rounded to fp32 (fewer rows than P: only the relative ridge
    # makes it definite), against the oracle's solve of the same values; both
    # ridge modes
    rng = np.random.default_rng(16)
    k, L_s, H_s, L_t, H_t, B, T = 16, 17, 1, 1, 1, 3, 400
    src, tgt, w = small_inputs(rng, L_s, H_s, L_t, H_t, B, T)
    hm = random_multi_map(rng, k, L_s, H_s, L_t, H_t)
    plan = cb.cb_plan_create_multi(hm, src, tgt, 1)
    Go, Co = oracle_stats_full(hm, src, tgt, w, 1)
    (Gt, G64), (Ct, C64) = shared_f32(Go), shared_f32(Co)        # the oracle's moments on both sides
    for unpen in (False, True):
        flags = cb.CB_LAMBDA_RELATIVE | (cb.CB_RIDGE_BIAS_UNPENALIZED if unpen else 0)
        maps, info = gpu_solve_ws(cb, Gt, Ct, 1e-2, flags)
        assert (info.cpu().numpy() == 0).all()
        Ws, io = oracle.ridge_solve(G64, C64, 1e-2, relative=True, bias_unpenalized=unpen, n_threads=NTHREADS)
        assert (io == 0).all()
        e = max(relF(maps[i].double().cpu().numpy(), Ws[i]) for i in range(plan.n_maps))
        say(f"  P=2049 solver alone (bias unpenalized={unpen}): {e:.3e}")
        assert e <= TOL_SOLVER
    plan.close()


def test_multi_wide_solve_pivot_failures_inside_and_in_the_last_panel(cb):
    # the blocked solve's first non-positive pivot, in the middle of a 32-column
    # panel (column 101, panel 3) and in the last one-column panel (column 385),
    # reported like the oracle's and with zero maps; the other systems of the
    # same call solve as in the oracle (absolute lambda 0, SPD Gram matrices)
    rng = np.random.default_rng(385)
    n, P, d_t = 5, 385, 128
    X = rng.standard_normal((n, 2 * P, P))
    G = np.einsum("nrp,nrq->npq", X, X) / (2 * P) + 0.1 * np.eye(P)
    C = rng.standard_normal((n, P, d_t))
    G[1, 100, 100] = -1.0                       # fails at column 101
    G[3, 384, 384] = -1.0                       # fails in the last panel
    G[4, 200, :] = G[4, :, 200] = 0.0           # a zero row and column: pivot 201 is 0
    (Gt, G64), (Ct, C64) = shared_f32(G), shared_f32(C)
    maps, info = gpu_solve_ws(cb, Gt, Ct, 0.0, 0)
    Wo, io = oracle.ridge_solve(G64, C64, 0.0, relative=False, n_threads=NTHREADS)
    inf = info.cpu().numpy()
    say(f"  pivots: gpu {inf.tolist()}, oracle {io.tolist()}")
    assert inf.tolist() == [0, 101, 0, 385, 201] and io.tolist() == inf.tolist()
    for m in (1, 3, 4):
        assert not maps[m].any()
    e = max(relF(maps[m].double().cpu().numpy(), Wo[m]) for m in (0, 2))
    say(f"  healthy systems: maps relF {e:.3e}")
    assert e <= TOL_SOLVER


def test_multi_determinism_scaling_and_zero_weights(cb):
    rng = np.random.default_rng(77)
    L_s, H_s, L_t, H_t, B, T, k, stride = 5, 2, 2, 2, 2, 150, 3, 4
    src, tgt, w = small_inputs(rng, L_s, H_s, L_t, H_t, B, T)
    hm = random_multi_map(rng, k, L_s, H_s, L_t, H_t)
    plan = cb.cb_plan_create_multi(hm, src, tgt, stride)
    G1, C1 = gpu_stats(cb, plan, [(src, tgt, w)])
    G2, C2 = gpu_stats(cb, plan, [(src, tgt, w)])
    assert torch.equal(G1, G2) and torch.equal(C1, C2), "results must be bitwise reproducible"
    G4, C4 = gpu_stats(cb, plan, [(src, tgt, 4.0 * w)])
    assert torch.equal(G4, 4.0 * G1) and torch.equal(C4, 4.0 * C1), "power-of-two weight scaling must be exact"
    # an empty call adds nothing
    cb.cb_stats_accumulate(plan, src[:, :, :0], tgt[:, :, :0], w, G1, C1)
    torch.cuda.synchronize()
    assert torch.equal(G1, G2)
    # weight rows of zero: zero moments, relative lambda 0, first pivot fails
    wz = w.clone()
    wz[0] = 0.0
    Gz, Cz = gpu_stats(cb, plan, [(src, tgt, wz)])
    zero_maps = [m for m in range(plan.n_maps) if hm["weight_row"][m] == 0]
    assert zero_maps and all(float(Gz[m].abs().max()) == 0.0 and float(Cz[m].abs().max()) == 0.0
                             for m in zero_maps)
    maps, info = gpu_solve_ws(cb, Gz, Cz)
    inf = info.cpu().numpy()
    for m in range(plan.n_maps):
        if m in zero_maps:
            assert inf[m] == 1 and float(maps[m].abs().max()) == 0.0
        else:
            assert inf[m] == 0
    plan.close()


def test_multi_device_side_argument_errors(cb):
    rng = np.random.default_rng(5)
    src, tgt, w = small_inputs(rng, 4, 2, 2, 2, 1, 32)
    hm = random_multi_map(rng, 2, 4, 2, 2, 2)
    plan = cb.cb_plan_create_multi(hm, src, tgt, 2)
    n, P = plan.n_maps, plan.P
    G = torch.zeros((n, P, P), dtype=torch.float32, device="cuda")
    C = torch.zeros((n, P, 128), dtype=torch.float32, device="cuda")
    with pytest.raises(cb.CacheBridgeError, match="CB_ERR_SHAPE"):
        cb.cb_stats_accumulate(plan, src[:2], tgt, w, G, C)              # wrong source layer count
    with pytest.raises(cb.CacheBridgeError, match="CB_ERR_SHAPE"):
        cb.cb_apply(plan, C, src, tgt[:1])                               # wrong target layer count
    with pytest.raises(cb.CacheBridgeError, match="CB_ERR_SHAPE"):
        cb.cb_apply(plan, C, src[:, :, :, :, :16], tgt)                  # token counts disagree
    # outputs the plan does not fit are refused before any launch: the centered
    # sums of a k = 2 plan are [n][1 + 256 + 128], not the single-layer [n][257]
    sums = torch.zeros((n, 257), dtype=torch.float64, device="cuda")
    with pytest.raises(ValueError, match="sums"):
        cb.cb_stats_means(plan, src, tgt, w, sums)
    with pytest.raises(ValueError, match="G"):
        cb.cb_stats_accumulate(plan, src, tgt, w, G[:, :-1], C)
    with pytest.raises(ValueError, match="maps"):
        cb.cb_apply(plan, C[:1], src, tgt)
    with pytest.raises(ValueError, match="weights"):
        cb.cb_stats_accumulate(plan, src, tgt, w[:1], G, C)
    maps = torch.empty_like(C)
    info = torch.empty((n,), dtype=torch.int32, device="cuda")
    small = torch.empty((1024,), dtype=torch.uint8, device="cuda")
    with pytest.raises(cb.CacheBridgeError, match="CB_ERR_SHAPE"):
        cb.cb_ridge_solve_ws(G, C, 1e-2, cb.CB_LAMBDA_RELATIVE, maps, info, small)
    with pytest.raises(cb.CacheBridgeError, match="CB_ERR_UNSUPPORTED"):
        cb.cb_ridge_solve(G, C, 1e-2, cb.CB_LAMBDA_RELATIVE, maps, info)
    plan.close()


# ----------------------------------------------------------------------------- full size

def test_multi_qwen_k8_batch_full_size_sampled_maps(cb):
    """The resident 100-sequence batch of the k = 8 construction (40 -> 64 layers x
    8 heads x 128, 1,024 tokens per sequence, every fourth token: 25,600 rows per
    call), launched as the benchmark launches it; eight sampled maps against the
    oracle, all 1,024 systems solved."""
    wl = synth.WORKLOADS["qwen_k8"]
    bw = wl.with_(n_seqs=wl.batch_seqs)
    say(f"multi qwen_k8 batch: {bw.n_seqs} x {bw.seq_len} tokens, stride {bw.sample_stride}, P={bw.P}")
    src = synth.gen_source(bw, device="cuda")
    tgt = synth.gen_target(bw, src, device="cuda")
    w = synth.gen_weights(bw, device="cuda", chunk=50)
    hm = synth.head_map_multi(wl)
    plan = cb.cb_plan_create_multi(hm, src, tgt, wl.sample_stride)
    G, C = gpu_stats(cb, plan, [(src, tgt, w)])
    sel = [0, 1, 135, 511, 512, 777, 1022, 1023]
    say("  oracle on the sampled maps ...")
    Go, Co = compact_multi(hm, sel, src, tgt, w, wl.sample_stride)
    check_stats(G, C, Go, Co, sel)
    del src, tgt
    torch.cuda.empty_cache()
    maps, info = gpu_solve_ws(cb, G, C, 1e-2, cb.CB_LAMBDA_RELATIVE | cb.CB_RIDGE_BIAS_UNPENALIZED)
    assert int((info != 0).sum()) == 0
    check_solve(cb, G, C, maps, info, Go, Co, sel, True)
    plan.close()


# ----------------------------------------------------------------------------- application

TOL_APPLY = 1e-3


def gpu_apply(cb, plan, maps, src, L_t, H_t, out=None):
    if out is None:
        B, T = src.shape[2], src.shape[4]
        out = torch.zeros((L_t, 2, B, H_t, T, plan.d_t), dtype=torch.bfloat16, device="cuda")
    cb.cb_apply(plan, maps, src, out)
    torch.cuda.synchronize()
    return out


def oracle_apply_multi(hm, maps, src, L_t, H_t, d_t, sel=None):
    """Oracle application of the maps `sel` (all by default) on a host copy of the
    sender cache; `maps` is the device tensor the GPU used or an fp64 array."""
    if isinstance(maps, torch.Tensor):
        maps = maps.double().cpu().numpy()
    if sel is not None:
        hm = {f: v[sel] for f, v in hm.items()}
        maps = maps[np.asarray(sel)]
    L_s, _, B, H_s, T, d_s = src.shape
    ref = np.zeros((L_t, 2, B, H_t, T, d_t), dtype=np.uint16)
    oracle.apply_multi(hm, np.ascontiguousarray(maps, dtype=np.float64), bits(src), synth.cache_strides(L_s, H_s, B, T, d_s), d_s,
                       ref, synth.cache_strides(L_t, H_t, B, T, d_t), d_t, B, T, n_threads=NTHREADS)
    return ref


def check_apply_multi(ob, ref, hm, sel, label=""):
    """Per map in `sel`: relF within the bar and every element within one bf16 ulp
    of the oracle's value plus 1e-4 of the map's RMS output (near-zero outputs see
    the ~2^-17 relative error of the split coefficients as several ulps)."""
    worst_e, worst_b, same, cnt = 0.0, 0.0, 0, 0
    for m in sel:
        l, z, h = int(hm["tgt_layer"][m]), int(hm["kv"][m]), int(hm["tgt_head"][m])
        og, orf = ob[l, z, :, h], ref[l, z, :, h]
        g = oracle.bf16_to_double(og)
        r = oracle.bf16_to_double(orf)
        worst_e = max(worst_e, relF(g, r))
        rms = np.sqrt((r * r).mean())
        ulp = np.spacing(np.abs(r).astype(np.float32)).astype(np.float64) * 65536.0
        worst_b = max(worst_b, float((np.abs(g - r) / (ulp + 1e-4 * rms)).max()))
        same += int((og == orf).sum())
        cnt += og.size
    say(f"  multi apply parity{label}: worst per-map relF {worst_e:.3e}, bitwise-equal {same / cnt:.6f}, "
        f"worst err/bound {worst_b:.3f}")
    assert worst_e <= TOL_APPLY and worst_b <= 1.0


def random_maps(rng, n, P, d_t):
    g = torch.Generator(device="cpu")
    g.manual_seed(int(rng.integers(1 << 31)))
    W = torch.randn((n, P, d_t), generator=g) / np.sqrt(P - 1)
    W[:, P - 1] = torch.randn((n, d_t), generator=g)
    return W.to("cuda")


def test_multi_apply_tiny_k3_fitted_maps(cb):
    # Maps fitted on tiny_k3 applied to the same sender: 4 x 520 tokens (eight
    # full 256-token tiles and a 32-token tail).  Two checks:
    #  * the apply alone: the oracle's fitted maps, rounded once to fp32, on both
    #    sides (per-element bar);
    #  * the whole chain: the GPU's statistics -> solve -> apply against the
    #    oracle's statistics -> solve -> apply (relative Frobenius bar).
    wl = synth.WORKLOADS["tiny_k3"]
    src = synth.gen_source(wl, device="cuda")
    tgt = synth.gen_target(wl, src, device="cuda")
    w = synth.gen_weights(wl, device="cuda")
    hm = synth.head_map_multi(wl)
    plan = cb.cb_plan_create_multi(hm, src, tgt, wl.sample_stride)
    flags = cb.CB_LAMBDA_RELATIVE | cb.CB_RIDGE_BIAS_UNPENALIZED
    G, C = gpu_stats(cb, plan, [(src, tgt, w)])
    maps_gpu, info = gpu_solve_ws(cb, G, C, 1e-2, flags)
    assert int((info != 0).sum()) == 0
    Go, Co = oracle_stats_full(hm, src, tgt, w, wl.sample_stride)
    Wo, io = oracle.ridge_solve(Go, Co, 1e-2, relative=True, bias_unpenalized=True, n_threads=NTHREADS)
    assert (io == 0).all()
    maps_t, maps64 = shared_f32(Wo)
    out = gpu_apply(cb, plan, maps_t, src, wl.L_t, wl.H_t)
    ref = oracle_apply_multi(hm, maps64, src, wl.L_t, wl.H_t, wl.d_t)
    check_apply_multi(bits(out), ref, hm, range(plan.n_maps), " (tiny_k3, oracle's fitted maps)")
    # chained: the GPU's own fitted maps against the oracle's unrounded fp64 maps
    out2 = gpu_apply(cb, plan, maps_gpu, src, wl.L_t, wl.H_t)
    ref2 = oracle_apply_multi(hm, Wo, src, wl.L_t, wl.H_t, wl.d_t)
    ob2 = bits(out2)
    worst = 0.0
    for m in range(plan.n_maps):
        l, z, h = int(hm["tgt_layer"][m]), int(hm["kv"][m]), int(hm["tgt_head"][m])
        worst = max(worst, relF(oracle.bf16_to_double(ob2[l, z, :, h]), oracle.bf16_to_double(ref2[l, z, :, h])))
    say(f"  chained statistics -> solve -> apply (tiny_k3): worst per-map relF {worst:.3e}")
    assert worst <= TOL_APPLY
    plan.close()


@pytest.mark.parametrize("k,B,T", [(1, 1, 37), (2, 3, 100), (4, 2, 300), (5, 1, 256), (8, 2, 129)])
def test_multi_apply_random_maps_ragged_tokens(cb, k, B, T):
    rng = np.random.default_rng(100 + k)
    L_s, H_s, L_t, H_t = max(k, 3) + 1, 2, 3, 2
    src, tgt, _ = small_inputs(rng, L_s, H_s, L_t, H_t, B, T)
    hm = random_multi_map(rng, k, L_s, H_s, L_t, H_t)
    plan = cb.cb_plan_create_multi(hm, src, tgt, 1)
    maps = random_maps(rng, plan.n_maps, plan.P, plan.d_t)
    say(f"multi apply k={k}: {B} x {T} tokens, {plan.n_maps} maps")
    out = gpu_apply(cb, plan, maps, src, L_t, H_t)
    ref = oracle_apply_multi(hm, maps, src, L_t, H_t, 128)
    check_apply_multi(bits(out), ref, hm, range(plan.n_maps), f" (k={k}, N={B * T})")
    plan.close()


@pytest.mark.parametrize("style,both", [(None, False), (1, False), (0, True)])
def test_multi_apply_paired_maps_permuted_and_lone(cb, style, both):
    # maps of one (kv, source head) whose source-layer sets are equal share
    # their staged blocks: equal sets listed in different orders (each map's
    # block order differs from the staging order), and maps with no partner
    # (which take the single-map path), against the oracle: plain, with the
    # target rotation, and with the sender's keys turned back as well (the K
    # pairs then read the de-rotated copy)
    rng = np.random.default_rng(31)
    k, L_s, H_s, L_t, H_t, B, T = 3, 6, 2, 6, 2, 2, 600
    src, tgt, _ = small_inputs(rng, L_s, H_s, L_t, H_t, B, T)
    sets = [[0, 1, 2], [2, 0, 1], [3, 4, 1], [1, 3, 4], [4, 5, 0], [1, 2, 5]]
    hm = {f: [] for f in oracle.MULTI_MAP_FIELDS}
    for l in range(L_t):
        for z in range(2):
            for h in range(H_t):
                for f, v in zip(oracle.MULTI_MAP_FIELDS, (l, h, z, sets[l], h, l * H_t + h)):
                    hm[f].append(v)
    hm = {f: np.asarray(v, np.int32) for f, v in hm.items()}
    plan = cb.cb_plan_create_multi(hm, src, tgt, 1)
    maps = random_maps(rng, plan.n_maps, plan.P, plan.d_t)
    say(f"multi apply paired maps (permuted, lone), rotation style {style}")
    out = torch.zeros((L_t, 2, B, H_t, T, 128), dtype=torch.bfloat16, device="cuda")
    ref = np.zeros(tuple(out.shape), dtype=np.uint16)
    ss, os_ = synth.cache_strides(L_s, H_s, B, T, 128), synth.cache_strides(L_t, H_t, B, T, 128)
    W = maps.double().cpu().numpy()
    if style is None:
        cb.cb_apply(plan, maps, src, out)
        oracle.apply_multi(hm, W, bits(src), ss, 128, ref, os_, 128, B, T, n_threads=NTHREADS)
    elif not both:
        table = gpu_rope_table(cb, 1e6, 128, T)
        cb.cb_apply_rope(plan, maps, src, out, cb.rope_spec(table, style, 0))
        oracle.apply_multi_rope(hm, W, bits(src), ss, 128, ref, os_, 128, B, T, 1e6, style, 0, n_threads=NTHREADS)
    else:
        src_r, sb = rotated(src, 1e4, style, 0)
        tab_s, tab_t = gpu_rope_table(cb, 1e4, 128, T), gpu_rope_table(cb, 1e6, 128, T)
        cb.cb_apply_rope(plan, maps, src_r, out, cb.rope_spec(tab_t, style, 0), cb.rope_spec(tab_s, style, 0))
        oracle.apply_multi_rope(hm, W, unrotated(sb, 1e4, style, 0), ss, 128, ref, os_, 128, B, T, 1e6, style, 0,
                                n_threads=NTHREADS)
    torch.cuda.synchronize()
    if not both:
        check_apply_multi(bits(out), ref, hm, range(plan.n_maps), " (paired maps)")
    else:
        # the oracle turns back in fp64, the kernel in fp32: a few inputs differ by one ulp
        ob = bits(out)
        e = relF(oracle.bf16_to_double(ob), oracle.bf16_to_double(ref))
        eq = float((ob == ref).mean())
        say(f"  paired maps, both rotations: relF {e:.3e}, bitwise-equal {eq:.6f}")
        assert e <= TOL_APPLY and eq >= 0.99
    plan.close()


def test_multi_apply_selector_maps_copy_bits_strided_output(cb):
    # map m copies source layer j_m of its window (identity block, zero bias): the
    # output bits equal the sender's bits.  The target is a view with room for
    # more tokens (sequence stride larger than the written rows), and the rows
    # past the written ones must stay untouched.
    rng = np.random.default_rng(9)
    k, L_s, H_s, L_t, H_t, B, T = 3, 5, 2, 4, 2, 3, 300
    src, tgt, _ = small_inputs(rng, L_s, H_s, L_t, H_t, B, T)
    hm = random_multi_map(rng, k, L_s, H_s, L_t, H_t)
    plan = cb.cb_plan_create_multi(hm, src, tgt, 1)
    n, P = plan.n_maps, plan.P
    maps = torch.zeros((n, P, 128), dtype=torch.float32)
    pick = rng.integers(k, size=n)
    for m in range(n):
        maps[m, 128 * pick[m]:128 * pick[m] + 128] = torch.eye(128)
    maps = maps.to("cuda")
    big = torch.full((L_t, 2, B, H_t, T + 64, 128), 7.0, dtype=torch.bfloat16, device="cuda")
    out = gpu_apply(cb, plan, maps, src, L_t, H_t, out=big[:, :, :, :, :T])
    ob, sb = bits(big), bits(src)
    for m in range(n):
        l, z, h = int(hm["tgt_layer"][m]), int(hm["kv"][m]), int(hm["tgt_head"][m])
        j, a = int(hm["src_layers"][m][pick[m]]), int(hm["src_head"][m])
        assert np.array_equal(ob[l, z, :, h, :T], sb[j, z, :, a]), f"map {m} must copy source layer {j}"
    assert (big[:, :, :, :, T:] == 7.0).all(), "rows past the written tokens must stay untouched"
    # an empty call writes nothing
    before = big.clone()
    cb.cb_apply(plan, maps * 2.0, src[:, :, :0], big[:, :, :0, :, :T])
    torch.cuda.synchronize()
    assert torch.equal(big, before)
    plan.close()


def test_multi_apply_qwen_k8_batch_sampled(cb):
    """The k = 8 construction's maps (40 -> 64 layers x 8 heads, 1,024 maps, P =
    1,025) applied to a 100-sequence x 1,024-token sender batch, as the benchmark
    launches it; eight sampled maps on the first and last 512 tokens of two
    sequences against the oracle."""
    wl = synth.WORKLOADS["qwen_k8"]
    bw = wl.with_(n_seqs=wl.batch_seqs)
    rng = np.random.default_rng(8)
    src = synth.gen_source(bw, device="cuda")
    hm = synth.head_map_multi(wl)
    plan = cb.cb_plan_create_multi(hm, src, (wl.L_t, wl.H_t, wl.d_t), wl.sample_stride)
    maps = random_maps(rng, plan.n_maps, plan.P, plan.d_t)
    say(f"multi apply qwen_k8: {bw.n_seqs} x {bw.seq_len} tokens, {plan.n_maps} maps")
    out = gpu_apply(cb, plan, maps, src, wl.L_t, wl.H_t)
    sel = [0, 1, 135, 511, 512, 777, 1022, 1023]
    hs = {f: v[sel] for f, v in hm.items()}
    ms = maps[torch.as_tensor(sel, device=maps.device)]
    for b, t0, t1 in ((0, 0, 512), (bw.n_seqs - 1, bw.seq_len - 512, bw.seq_len)):
        s_sub = src[:, :, b:b + 1, :, t0:t1].contiguous()
        ref = oracle_apply_multi(hs, ms, s_sub, wl.L_t, wl.H_t, wl.d_t)
        ob = bits(out[:, :, b:b + 1, :, t0:t1].contiguous())
        check_apply_multi(ob, ref, hs, range(len(sel)), f" (seq {b}, tokens {t0}..{t1})")
    plan.close()


# ----------------------------------------------------------------------------- rotary keys, k > 1

def gpu_rope_table(cb, theta, d, n_pos):
    t = torch.empty((n_pos, d // 2, 2), dtype=torch.float32, device="cuda")
    cb.cb_rope_table(theta, d, n_pos, t)
    return t


def rotated(x, theta, style, off):
    """A cache as a model holds it: the K rows of content cache x turned by the
    oracle's RoPE at positions off + tok; device tensor and host bits."""
    L, _, B, H, T, d = x.shape
    b = oracle.rope(bits(x), synth.cache_strides(L, H, B, T, d), L, H, d, B, T, theta, style, pos_offset=off)
    return torch.from_numpy(b.view(np.int16)).to("cuda").view(torch.bfloat16), b


def unrotated(b, theta, style, off):
    """The oracle's inverse turn of cache bits b (fp64, one rounding)."""
    L, _, B, H, T, d = b.shape
    return oracle.rope(b, synth.cache_strides(L, H, B, T, d), L, H, d, B, T, theta, style, inverse=True,
                       pos_offset=off)


@pytest.mark.parametrize("style,off", [(0, 0), (1, 300)])
def test_multi_apply_rope_target_rotation(cb, style, off):
    # the K outputs turned in fp32 before the one rounding (the half split on
    # permuted fragments); V outputs bit for bit those of cb_apply
    rng = np.random.default_rng(70 + style)
    k, L_s, H_s, L_t, H_t, B, T = 3, 5, 2, 2, 2, 2, 300
    src, tgt, _ = small_inputs(rng, L_s, H_s, L_t, H_t, B, T)
    hm = random_multi_map(rng, k, L_s, H_s, L_t, H_t)
    plan = cb.cb_plan_create_multi(hm, src, tgt, 1)
    maps = random_maps(rng, plan.n_maps, plan.P, plan.d_t)
    table = gpu_rope_table(cb, 1e6, 128, off + T)
    say(f"multi apply target rotation style={style} off={off}")
    out = torch.zeros((L_t, 2, B, H_t, T, 128), dtype=torch.bfloat16, device="cuda")
    cb.cb_apply_rope(plan, maps, src, out, cb.rope_spec(table, style, off))
    plain = gpu_apply(cb, plan, maps, src, L_t, H_t)
    ref = np.zeros(tuple(out.shape), dtype=np.uint16)
    oracle.apply_multi_rope(hm, maps.double().cpu().numpy(), bits(src), synth.cache_strides(L_s, H_s, B, T, 128),
                            128, ref, synth.cache_strides(L_t, H_t, B, T, 128), 128, B, T, 1e6, style, off,
                            n_threads=NTHREADS)
    ob = bits(out)
    check_apply_multi(ob, ref, hm, range(plan.n_maps), " (target rotation)")
    assert np.array_equal(ob[:, 1], bits(plain)[:, 1]) and not np.array_equal(ob[:, 0], bits(plain)[:, 0])
    plan.close()


@pytest.mark.parametrize("style,off,tgt_too", [(0, 0, False), (1, 77, True)])
def test_multi_apply_rope_source_derotation(cb, style, off, tgt_too):
    # the sender's keys carry RoPE: one rotation pass into the plan's workspace
    # gives bit for bit cb_rope(inverse) + the mapping, and matches the
    # oracle's composition (the oracle turns back in fp64, the kernel in fp32,
    # so a few inputs differ by one ulp: relative bar and bitwise share)
    rng = np.random.default_rng(80 + style)
    k, L_s, H_s, L_t, H_t, B, T = 3, 5, 2, 2, 2, 2, 300
    src_c, tgt, _ = small_inputs(rng, L_s, H_s, L_t, H_t, B, T)
    src, sb = rotated(src_c, 1e4, style, off)
    hm = random_multi_map(rng, k, L_s, H_s, L_t, H_t)
    plan = cb.cb_plan_create_multi(hm, src, tgt, 1)
    maps = random_maps(rng, plan.n_maps, plan.P, plan.d_t)
    tab_s, tab_t = gpu_rope_table(cb, 1e4, 128, off + T), gpu_rope_table(cb, 1e6, 128, off + T)
    sr = cb.rope_spec(tab_s, style, off)
    tr = cb.rope_spec(tab_t, style, off) if tgt_too else None
    say(f"multi apply source de-rotation style={style} off={off} target rotation={tgt_too}")
    out = torch.zeros((L_t, 2, B, H_t, T, 128), dtype=torch.bfloat16, device="cuda")
    cb.cb_apply_rope(plan, maps, src, out, tr, sr)
    src_d = torch.empty_like(src)
    cb.cb_rope(src, src_d, tab_s, style, True, off)
    sep = torch.zeros_like(out)
    cb.cb_apply_rope(plan, maps, src_d, sep, tr)
    torch.cuda.synchronize()
    assert torch.equal(out, sep)
    so = unrotated(sb, 1e4, style, off)
    ref = np.zeros(tuple(out.shape), dtype=np.uint16)
    W = maps.double().cpu().numpy()
    ss, os_ = synth.cache_strides(L_s, H_s, B, T, 128), synth.cache_strides(L_t, H_t, B, T, 128)
    if tgt_too:
        oracle.apply_multi_rope(hm, W, so, ss, 128, ref, os_, 128, B, T, 1e6, style, off, n_threads=NTHREADS)
    else:
        oracle.apply_multi(hm, W, so, ss, 128, ref, os_, 128, B, T, n_threads=NTHREADS)
    ob = bits(out)
    e = relF(oracle.bf16_to_double(ob), oracle.bf16_to_double(ref))
    eq = float((ob == ref).mean())
    say(f"  fused == separate passes; against the oracle's composition: relF {e:.3e}, bitwise-equal {eq:.6f}")
    assert e <= TOL_APPLY and eq >= 0.99
    plan.close()


@pytest.mark.parametrize("stride,sides,style", [(4, "both", 0), (3, "src", 1), (1, "tgt", 0)])
def test_multi_stats_rope_compact_derotation(cb, stride, sides, style):
    # the K calibration rows turned back once into a compact workspace: moments
    # bit for bit those of cb_rope(inverse) copies (same kernel, same rows),
    # streamed over two uneven batches (the workspace is reused), and the
    # oracle's composition within the statistics bar
    rng = np.random.default_rng(90 + stride)
    k, L_s, H_s, L_t, H_t, B, T, off = 3, 5, 2, 2, 2, 3, 520, 41
    src_c, tgt_c, w = small_inputs(rng, L_s, H_s, L_t, H_t, B, T)
    src, sb = rotated(src_c, 1e4, style, off)
    tgt, tb = rotated(tgt_c, 1e6, style, off)
    hm = random_multi_map(rng, k, L_s, H_s, L_t, H_t)
    plan = cb.cb_plan_create_multi(hm, src, tgt, stride)
    tab_s, tab_t = gpu_rope_table(cb, 1e4, 128, off + T), gpu_rope_table(cb, 1e6, 128, off + T)
    sr = cb.rope_spec(tab_s, style, off) if sides in ("both", "src") else None
    tr = cb.rope_spec(tab_t, style, off) if sides in ("both", "tgt") else None
    say(f"multi stats rope stride={stride} sides={sides} style={style}")
    n, P = plan.n_maps, plan.P
    G = torch.empty((n, P, P), dtype=torch.float32, device="cuda")
    C = torch.empty((n, P, 128), dtype=torch.float32, device="cuda")
    cb.cb_stats_zero(plan, G, C)
    for a, b in ((0, 1), (1, B)):
        wb = w.reshape(-1, B, T)[:, a:b].reshape(w.shape[0], -1)
        cb.cb_stats_accumulate_rope(plan, src[:, :, a:b], tgt[:, :, a:b], wb, G, C, sr, tr)
    src_d, tgt_d = src.clone(), tgt.clone()
    if sr is not None:
        cb.cb_rope(src, src_d, tab_s, style, True, off)
    if tr is not None:
        cb.cb_rope(tgt, tgt_d, tab_t, style, True, off)
    batches = [(src_d[:, :, a:b], tgt_d[:, :, a:b], w.reshape(-1, B, T)[:, a:b].reshape(w.shape[0], -1))
               for a, b in ((0, 1), (1, B))]
    G2, C2 = gpu_stats(cb, plan, batches)
    assert torch.equal(G, G2) and torch.equal(C, C2)
    so = unrotated(sb, 1e4, style, off) if sr is not None else sb
    to = unrotated(tb, 1e6, style, off) if tr is not None else tb
    ss, ts = synth.cache_strides(L_s, H_s, B, T, 128), synth.cache_strides(L_t, H_t, B, T, 128)
    Go, Co = oracle.stats_multi(hm, so, ss, 128, to, ts, 128, w.cpu().numpy(), B * T, B, T, stride,
                                n_threads=NTHREADS)
    check_stats(G, C, Go, Co, list(range(n)))
    G3, _ = gpu_stats(cb, plan, [(src, tgt, w)])
    kmaps = [m for m in range(n) if hm["kv"][m] == 0]
    vmaps = [m for m in range(n) if hm["kv"][m] == 1]
    assert not torch.equal(G[kmaps], G3[kmaps])
    assert relF(G[vmaps].double().cpu().numpy(), G3[vmaps].double().cpu().numpy()) <= 1e-6
    plan.close()


def test_multi_stats_rope_qwen_k8_batch_full_size_sampled_maps(cb):
    """The compact de-rotated gather at the k = 8 construction's resident batch
    (100 x 1,024 tokens, every fourth): the synthetic caches taken as caches whose
    keys carry RoPE; four sampled maps against the oracle's composition (its inverse
    turn of all their rows, then its moments on every fourth token)."""
    wl = synth.WORKLOADS["qwen_k8"]
    bw = wl.with_(n_seqs=wl.batch_seqs)
    say(f"multi rope qwen_k8 batch: {bw.n_seqs} x {bw.seq_len} tokens, stride {bw.sample_stride}")
    src = synth.gen_source(bw, device="cuda")
    tgt = synth.gen_target(bw, src, device="cuda")
    w = synth.gen_weights(bw, device="cuda", chunk=50)
    hm = synth.head_map_multi(wl)
    plan = cb.cb_plan_create_multi(hm, src, tgt, wl.sample_stride)
    T = bw.seq_len
    tab = gpu_rope_table(cb, 1e6, 128, T)
    n, P = plan.n_maps, plan.P
    G = torch.empty((n, P, P), dtype=torch.float32, device="cuda")
    C = torch.empty((n, P, 128), dtype=torch.float32, device="cuda")
    cb.cb_stats_zero(plan, G, C)
    cb.cb_stats_accumulate_rope(plan, src, tgt, w, G, C, cb.rope_spec(tab), cb.rope_spec(tab))
    torch.cuda.synchronize()
    sel = [3, 400, 641, 1020]
    say(f"  oracle on maps {sel}")
    k, B_ = wl.k, bw.n_seqs
    xs, ys, ws = [], [], []
    for m in sel:
        z, a = int(hm["kv"][m]), int(hm["src_head"][m])
        for j in hm["src_layers"][m]:
            xs.append(src[int(j), z, :, a])
        ys.append(tgt[int(hm["tgt_layer"][m]), z, :, int(hm["tgt_head"][m])])
        ws.append(w[int(hm["weight_row"][m])])
    ns = len(sel)
    xb = bits(torch.stack(xs)).reshape(ns * k, 1, B_, 1, T, 128)
    yb = bits(torch.stack(ys)).reshape(ns, 1, B_, 1, T, 128)
    del src, tgt
    torch.cuda.empty_cache()
    ss = (B_ * T * 128, 0, T * 128, 0, 128)
    xd = oracle.rope(xb, ss, ns * k, 1, 128, B_, T, 1e6, 0, inverse=True)[:, 0:1]
    yd = oracle.rope(yb, ss, ns, 1, 128, B_, T, 1e6, 0, inverse=True)[:, 0:1]
    for i, m in enumerate(sel):                    # V maps carry no positions
        if hm["kv"][m] == 1:
            xd[i * k:(i + 1) * k], yd[i] = xb[i * k:(i + 1) * k], yb[i]
    chm = {"tgt_layer": np.arange(ns, dtype=np.int32), "tgt_head": np.zeros(ns, np.int32),
           "kv": np.zeros(ns, np.int32), "src_layers": np.arange(ns * k, dtype=np.int32).reshape(ns, k),
           "src_head": np.zeros(ns, np.int32), "weight_row": np.arange(ns, dtype=np.int32)}
    Go, Co = oracle.stats_multi(chm, np.ascontiguousarray(xd), ss, 128, np.ascontiguousarray(yd), ss, 128,
                                np.ascontiguousarray(torch.stack(ws).cpu().numpy()), B_ * T, B_, T,
                                wl.sample_stride, n_threads=NTHREADS)
    check_stats(G, C, Go, Co, sel)
    plan.close()


# ----------------------------------------------------------------------------- two-pass centered form, k > 1

TOL_SUMS = 1e-9        # fp64 sums of exact fp64 products: only the summation order differs


def gpu_centered_multi(cb, plan, batches):
    """Pass 1 (means) over every batch, then pass 2 (centered moments) over every batch."""
    n, Dx, dt = plan.n_maps, plan.P - 1, plan.d_t
    sums = torch.empty((n, 1 + Dx + dt), dtype=torch.float64, device="cuda")
    A = torch.empty((n, Dx, Dx), dtype=torch.float32, device="cuda")
    B = torch.empty((n, Dx, dt), dtype=torch.float32, device="cuda")
    cb.cb_stats_zero_centered(plan, sums, A, B)
    for s, t, w in batches:
        cb.cb_stats_means(plan, s, t, w, sums)
    for s, t, w in batches:
        cb.cb_stats_accumulate_centered(plan, s, t, w, sums, A, B)
    torch.cuda.synchronize()
    return sums, A, B


def gpu_solve_centered_ws(cb, sums, A, B, lam=1e-2, flags=None):
    if flags is None:
        flags = cb.CB_LAMBDA_RELATIVE
    n, Dx, _ = A.shape
    dt = B.shape[2]
    maps = torch.empty((n, Dx + 1, dt), dtype=torch.float32, device="cuda")
    info = torch.empty((n,), dtype=torch.int32, device="cuda")
    per = cb.cb_ridge_solve_workspace_bytes(Dx, dt, 1)
    nsys = max(1, min(n, (8 << 30) // max(per, 1)))
    ws = torch.empty((max(per * nsys, 8),), dtype=torch.uint8, device="cuda")
    cb.cb_ridge_solve_centered_ws(sums, A, B, lam, flags, maps, info, ws)
    torch.cuda.synchronize()
    return maps, info


def oracle_centered_full(hm, src, tgt, w, stride):
    sb, tb = bits(src), bits(tgt)
    L_s, _, Bn, H_s, T, d_s = src.shape
    L_t, _, _, H_t, _, d_t = tgt.shape
    return oracle.stats_multi_centered(hm, sb, synth.cache_strides(L_s, H_s, Bn, T, d_s), d_s, tb,
                                       synth.cache_strides(L_t, H_t, Bn, T, d_t), d_t, w.cpu().numpy(), Bn * T, Bn,
                                       T, stride, n_threads=NTHREADS)


def check_centered_multi(cb, sums, A, B, so, Ao, Bo, sel, label=""):
    """Sums to 1e-9, A and B to the stats bar, A exactly symmetric; then the solve
    end to end and alone (both sides on the oracle's moments rounded to fp32)."""
    idx = torch.as_tensor(np.asarray(sel), device=A.device)
    sg = sums[idx].cpu().numpy()
    Ag = A[idx].double().cpu().numpy()
    Bg = B[idx].double().cpu().numpy()
    es = max(relF(sg[i], so[i]) for i in range(len(sel)))
    ea = max(relF(Ag[i], Ao[i]) for i in range(len(sel)))
    eb = max(relF(Bg[i], Bo[i]) for i in range(len(sel)))
    say(f"  centered{label}: sums {es:.3e}, A {ea:.3e}, B {eb:.3e}")
    assert es <= TOL_SUMS and ea <= TOL_STATS and eb <= TOL_STATS
    assert np.array_equal(Ag, np.transpose(Ag, (0, 2, 1))), "A must be exactly symmetric"
    Wo, io = oracle.ridge_solve_centered(so, Ao, Bo, 1e-2, relative=True, n_threads=NTHREADS)
    assert (io == 0).all()
    return Wo


@pytest.mark.parametrize("offset", [False, True])
def test_multi_centered_tiny_k3_end_to_end(cb, offset):
    # tiny_k3 (k = 3, P = 385, every fourth token), streamed in two batches; with
    # `offset` the source channels carry means far above their spread
    wl = synth.WORKLOADS["tiny_k3"]
    if offset:
        wl = wl.with_(source_kind="offset")
    src = synth.gen_source(wl, device="cuda")
    tgt = synth.gen_target(wl, src, device="cuda")
    w = synth.gen_weights(wl, device="cuda")
    hm = synth.head_map_multi(wl)
    plan = cb.cb_plan_create_multi(hm, src, tgt, wl.sample_stride)
    B_ = wl.n_seqs
    T = wl.seq_len
    batches = [(src[:, :, a:b], tgt[:, :, a:b], w.reshape(-1, B_, T)[:, a:b].reshape(w.shape[0], -1))
               for a, b in ((0, 1), (1, B_))]
    sums, A, B = gpu_centered_multi(cb, plan, batches)
    so, Ao, Bo = oracle_centered_full(hm, src, tgt, w, wl.sample_stride)
    sel = list(range(plan.n_maps))
    Wo = check_centered_multi(cb, sums, A, B, so, Ao, Bo, sel, " (tiny_k3, offset)" if offset else " (tiny_k3)")
    maps, info = gpu_solve_centered_ws(cb, sums, A, B)
    assert int((info != 0).sum()) == 0
    e2e = max(relF(maps[m].double().cpu().numpy(), Wo[m]) for m in sel)
    # the solver alone: the oracle's sums, A, B (A, B rounded once to fp32) on both sides
    (At, A64), (Bt, B64) = shared_f32(Ao), shared_f32(Bo)
    st = torch.from_numpy(np.ascontiguousarray(so)).to("cuda")
    ms, inf2 = gpu_solve_centered_ws(cb, st, At, Bt)
    Ws, _ = oracle.ridge_solve_centered(so, A64, B64, 1e-2, relative=True, n_threads=NTHREADS)
    alone = max(relF(ms[m].double().cpu().numpy(), Ws[m]) for m in sel)
    say(f"  centered solve: maps end-to-end {e2e:.3e}, solver alone {alone:.3e}")
    assert e2e <= TOL_MAPS and alone <= TOL_SOLVER and int((inf2 != 0).sum()) == 0
    if not offset:
        # the same problem as the unpenalized augmented ridge of the one-pass moments (Schur complement)
        G, C = gpu_stats(cb, plan, [(src, tgt, w)])
        mu, _ = gpu_solve_ws(cb, G, C, 1e-2, cb.CB_LAMBDA_RELATIVE | cb.CB_RIDGE_BIAS_UNPENALIZED)
        d = max(relF(maps[m].double().cpu().numpy(), mu[m].double().cpu().numpy()) for m in sel)
        say(f"  centered maps vs unpenalized augmented maps: {d:.3e}")
        assert d <= TOL_MAPS
    plan.close()


@pytest.mark.parametrize("k,stride,T", [(2, 3, 520), (5, 2, 858)])
def test_multi_centered_widths_ragged_offset_and_uncentered_gap(cb, k, stride, T):
    # large channel means (the purpose of the centered form): the centered A is
    # within the bar, while A recovered from the one-pass uncentered moments of
    # the same data is far worse
    rng = np.random.default_rng(3000 + 10 * k + stride)
    L_s, H_s, L_t, H_t, B_ = 6, 2, 2, 2, 3
    src, tgt, w = small_inputs(rng, L_s, H_s, L_t, H_t, B_, T)
    g = torch.Generator(device="cpu")
    g.manual_seed(77 + k)
    mu = (40.0 * torch.randn((L_s, 2, 1, H_s, 1, 128), generator=g)).to("cuda")
    src = (src.float() + mu).to(torch.bfloat16)
    hm = random_multi_map(rng, k, L_s, H_s, L_t, H_t)
    plan = cb.cb_plan_create_multi(hm, src, tgt, stride)
    cuts = [(0, 1), (1, 1), (1, 3)]
    batches = [(src[:, :, a:b], tgt[:, :, a:b], w.reshape(-1, B_, T)[:, a:b].reshape(w.shape[0], -1))
               for a, b in cuts]
    sums, A, B = gpu_centered_multi(cb, plan, batches)
    so, Ao, Bo = oracle_centered_full(hm, src, tgt, w, stride)
    sel = list(range(plan.n_maps))
    check_centered_multi(cb, sums, A, B, so, Ao, Bo, sel, f" (k={k}, stride {stride}, offset means)")
    # A from the uncentered G: G_xx - s s^T / S
    G, C = gpu_stats(cb, plan, [(src, tgt, w)])
    Gd = G.double().cpu().numpy()
    P = plan.P
    gap = []
    for m in sel:
        s_ = Gd[m, :P - 1, P - 1]
        Au = Gd[m, :P - 1, :P - 1] - np.outer(s_, s_) / Gd[m, P - 1, P - 1]
        gap.append(relF(Au, Ao[m]))
    ea = max(relF(A[m].double().cpu().numpy(), Ao[m]) for m in sel)
    say(f"  A from the uncentered moments: {max(gap):.3e} (centered {ea:.3e})")
    assert max(gap) >= 10 * ea
    maps, info = gpu_solve_centered_ws(cb, sums, A, B)
    assert int((info != 0).sum()) == 0
    plan.close()


TOL_SUMS_SHIFTED = 1e-6   # one-pass form: sums of fp32 partials, added in fp64 at every flush


@pytest.mark.parametrize("k,stride,T", [(2, 3, 520), (5, 2, 858)])
def test_multi_shifted_one_pass_offset_means(cb, k, stride, T):
    # the offset-means inputs of the two-pass test, in one pass about the means
    # of a one-sequence pilot, then moved to the data's means: the oracle's
    # centered sums, A and B, and the two-pass GPU moments
    rng = np.random.default_rng(3000 + 10 * k + stride)
    L_s, H_s, L_t, H_t, B_ = 6, 2, 2, 2, 3
    src, tgt, w = small_inputs(rng, L_s, H_s, L_t, H_t, B_, T)
    g = torch.Generator(device="cpu")
    g.manual_seed(77 + k)
    mu = (40.0 * torch.randn((L_s, 2, 1, H_s, 1, 128), generator=g)).to("cuda")
    src = (src.float() + mu).to(torch.bfloat16)
    hm = random_multi_map(rng, k, L_s, H_s, L_t, H_t)
    plan = cb.cb_plan_create_multi(hm, src, tgt, stride)
    cut = lambda a, b: (src[:, :, a:b], tgt[:, :, a:b], w.reshape(-1, B_, T)[:, a:b].reshape(w.shape[0], -1))  # noqa: E731
    batches = [cut(0, 1), cut(1, 3)]
    n, Dx, dt = plan.n_maps, plan.P - 1, plan.d_t
    shift = torch.zeros((n, 1 + Dx + dt), dtype=torch.float64, device="cuda")
    sums = torch.empty_like(shift)
    A = torch.empty((n, Dx, Dx), dtype=torch.float32, device="cuda")
    B = torch.empty((n, Dx, dt), dtype=torch.float32, device="cuda")
    cb.cb_stats_zero_centered(plan, sums, A, B)
    cb.cb_stats_means(plan, *cut(0, 1), shift)
    for s_, t_, w_ in batches:
        cb.cb_stats_accumulate_shifted(plan, s_, t_, w_, shift, sums, A, B)
    cb.cb_stats_shift_finish(plan, shift, sums, A, B)
    torch.cuda.synchronize()
    so, Ao, Bo = oracle_centered_full(hm, src, tgt, w, stride)
    sel = list(range(n))
    Ag, Bg, sg = A.double().cpu().numpy(), B.double().cpu().numpy(), sums.cpu().numpy()
    es = max(relF(sg[m], so[m]) for m in sel)
    ea = max(relF(Ag[m], Ao[m]) for m in sel)
    eb = max(relF(Bg[m], Bo[m]) for m in sel)
    say(f"  shifted (k={k}, stride {stride}): sums {es:.3e}, A {ea:.3e}, B {eb:.3e}")
    assert es <= TOL_SUMS_SHIFTED and ea <= TOL_STATS and eb <= TOL_STATS
    assert np.array_equal(Ag, np.transpose(Ag, (0, 2, 1))), "A must be exactly symmetric"
    s2, A2, B2 = gpu_centered_multi(cb, plan, batches)
    d = max(relF(Ag[m], A2[m].double().cpu().numpy()) for m in sel)
    say(f"  shifted vs two-pass A: {d:.3e}")
    assert d <= TOL_STATS
    Wo, io = oracle.ridge_solve_centered(so, Ao, Bo, 1e-2, relative=True, n_threads=NTHREADS)
    maps, info = gpu_solve_centered_ws(cb, sums, A, B)
    assert int((info != 0).sum()) == 0 and (io == 0).all()
    e2e = max(relF(maps[m].double().cpu().numpy(), Wo[m]) for m in sel)
    say(f"  shifted maps end to end: {e2e:.3e}")
    assert e2e <= TOL_MAPS
    plan.close()


def test_multi_centered_zero_weights_and_determinism(cb):
    rng = np.random.default_rng(41)
    k, stride, L_s, H_s, L_t, H_t, B_, T = 3, 4, 5, 2, 2, 2, 2, 600
    src, tgt, w = small_inputs(rng, L_s, H_s, L_t, H_t, B_, T)
    w[1] = 0.0                                           # maps of weight row 1 see no weight
    hm = random_multi_map(rng, k, L_s, H_s, L_t, H_t)
    plan = cb.cb_plan_create_multi(hm, src, tgt, stride)
    s1, A1, B1 = gpu_centered_multi(cb, plan, [(src, tgt, w)])
    s2, A2, B2 = gpu_centered_multi(cb, plan, [(src, tgt, w)])
    assert torch.equal(s1, s2) and torch.equal(A1, A2) and torch.equal(B1, B2)
    zero = [m for m in range(plan.n_maps) if int(hm["weight_row"][m]) == 1]
    assert zero
    for m in zero:
        assert not s1[m].any() and not A1[m].any() and not B1[m].any()
    # empty call: nothing changes
    cb.cb_stats_means(plan, src[:, :, :0], tgt[:, :, :0], w[:, :0], s1)
    cb.cb_stats_accumulate_centered(plan, src[:, :, :0], tgt[:, :, :0], w[:, :0], s1, A1, B1)
    torch.cuda.synchronize()
    assert torch.equal(s1, s2) and torch.equal(A1, A2)
    maps, info = gpu_solve_centered_ws(cb, s1, A1, B1, 0.5, 0)          # absolute lambda: W = 0, b = 0
    for m in zero:
        assert int(info[m]) == 0 and not maps[m].any()
    plan.close()


def compact_multi_centered(hm, sel, src, tgt, w, stride):
    """Oracle centered moments of the maps `sel` on host copies of only their sampled rows."""
    k = hm["src_layers"].shape[1]
    B_, T = src.shape[2], src.shape[4]
    xs, ys, ws = [], [], []
    for m in sel:
        z, a = int(hm["kv"][m]), int(hm["src_head"][m])
        for j in hm["src_layers"][m]:
            xs.append(src[int(j), z, :, a, ::stride])
        ys.append(tgt[int(hm["tgt_layer"][m]), z, :, int(hm["tgt_head"][m]), ::stride])
        ws.append(w[int(hm["weight_row"][m])].reshape(B_, T)[:, ::stride].reshape(-1))
    n, Ts = len(sel), xs[0].shape[1]
    d_s, d_t = xs[0].shape[-1], ys[0].shape[-1]
    xb = bits(torch.stack(xs)).reshape(n * k, 1, B_, 1, Ts, d_s)
    yb = bits(torch.stack(ys)).reshape(n, 1, B_, 1, Ts, d_t)
    wb = torch.stack(ws).cpu().numpy()
    chm = {"tgt_layer": np.arange(n, dtype=np.int32), "tgt_head": np.zeros(n, np.int32),
           "kv": np.zeros(n, np.int32), "src_layers": np.arange(n * k, dtype=np.int32).reshape(n, k),
           "src_head": np.zeros(n, np.int32), "weight_row": np.arange(n, dtype=np.int32)}
    ss = (B_ * Ts * d_s, 0, Ts * d_s, 0, d_s)
    ts = (B_ * Ts * d_t, 0, Ts * d_t, 0, d_t)
    return oracle.stats_multi_centered(chm, xb, ss, d_s, yb, ts, d_t, np.ascontiguousarray(wb), B_ * Ts, B_, Ts, 1,
                                       n_threads=NTHREADS)


def test_multi_centered_qwen_k8_batch_full_size_sampled_maps(cb):
    """The k = 8 construction's resident batch (100 x 1,024 tokens, every fourth),
    both centered passes as the benchmark launches them; four sampled maps against
    the oracle, all 1,024 centered systems solved."""
    wl = synth.WORKLOADS["qwen_k8"]
    bw = wl.with_(n_seqs=wl.batch_seqs)
    say(f"multi centered qwen_k8 batch: {bw.n_seqs} x {bw.seq_len} tokens, stride {bw.sample_stride}")
    src = synth.gen_source(bw, device="cuda")
    tgt = synth.gen_target(bw, src, device="cuda")
    w = synth.gen_weights(bw, device="cuda", chunk=50)
    hm = synth.head_map_multi(wl)
    plan = cb.cb_plan_create_multi(hm, src, tgt, wl.sample_stride)
    sums, A, B = gpu_centered_multi(cb, plan, [(src, tgt, w)])
    sel = [0, 300, 777, 1023]
    say("  oracle on the sampled maps ...")
    so, Ao, Bo = compact_multi_centered(hm, sel, src, tgt, w, wl.sample_stride)
    del src, tgt
    torch.cuda.empty_cache()
    Wo = check_centered_multi(cb, sums, A, B, so, Ao, Bo, sel, " (qwen_k8 batch)")
    maps, info = gpu_solve_centered_ws(cb, sums, A, B)
    assert int((info != 0).sum()) == 0
    e2e = max(relF(maps[m].double().cpu().numpy(), Wo[i]) for i, m in enumerate(sel))
    say(f"  centered maps end-to-end {e2e:.3e}")
    assert e2e <= TOL_MAPS
    plan.close()
