"""Host-side checks of the C ABI (no GPU needed): the library loads, exports every
function declared in include/cachebridge.h, and rejects bad arguments on the host
before touching a device."""
import ctypes
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "cachebridge.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(cb_[a-z_]+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for required in ("cb_plan_create", "cb_plan_destroy", "cb_stats_zero", "cb_stats_accumulate",
                     "cb_ridge_solve", "cb_apply", "cb_status_string", "cb_last_error"):
        assert required in names


def test_library_exports_every_declared_symbol():
    import paper_2609_00891_amd as cb
    lib = cb.library()
    for name in declared_functions():
        assert hasattr(lib, name), name
    # and nothing torch-typed: the library links only the HIP runtime
    import subprocess
    out = subprocess.run(["ldd", cb.LIB_PATH], capture_output=True, text=True).stdout
    assert "libtorch" not in out and "libc10" not in out


def test_status_strings():
    import paper_2609_00891_amd as cb
    for code, name in cb.STATUS_NAMES.items():
        assert cb.cb_status_string(code) == name


def _hm(n=2):
    return {"tgt_layer": np.zeros(n, np.int32), "tgt_head": np.arange(n, dtype=np.int32),
            "kv": np.zeros(n, np.int32), "src_layer": np.zeros(n, np.int32),
            "src_head": np.arange(n, dtype=np.int32), "weight_row": np.arange(n, dtype=np.int32)}


@pytest.mark.parametrize("mutate,status", [
    (lambda h: h.update(kv=np.array([0, 2], np.int32)), "CB_ERR_INVALID_ARGUMENT"),
    (lambda h: h.update(src_head=np.array([0, 9], np.int32)), "CB_ERR_INVALID_ARGUMENT"),
    (lambda h: h.update(tgt_layer=np.array([0, -1], np.int32)), "CB_ERR_INVALID_ARGUMENT"),
    (lambda h: h.update(weight_row=np.array([0, -3], np.int32)), "CB_ERR_INVALID_ARGUMENT"),
])
def test_plan_create_rejects_bad_head_maps(mutate, status):
    import paper_2609_00891_amd as cb
    h = _hm()
    mutate(h)
    with pytest.raises(cb.CacheBridgeError) as e:
        cb.cb_plan_create(h, (1, 2, 64), (1, 2, 64), 1024)
    assert status in str(e.value)


def test_plan_create_rejects_unsupported_widths_and_token_limits():
    import paper_2609_00891_amd as cb
    with pytest.raises(cb.CacheBridgeError, match="CB_ERR_UNSUPPORTED"):
        cb.cb_plan_create(_hm(), (1, 2, 80), (1, 2, 64), 1024)
    with pytest.raises(cb.CacheBridgeError, match="CB_ERR_UNSUPPORTED"):
        cb.cb_plan_create(_hm(), (1, 2, 64), (1, 2, 256), 1024)
    with pytest.raises(cb.CacheBridgeError, match="CB_ERR_UNSUPPORTED"):
        cb.cb_plan_create(_hm(), (1, 2, 64), (1, 2, 64), 2 ** 31)
    with pytest.raises(cb.CacheBridgeError, match="CB_ERR_INVALID_ARGUMENT"):
        cb.cb_plan_create({k: v[:0] for k, v in _hm().items()}, (1, 2, 64), (1, 2, 64), 16)


def test_null_arguments_are_rejected_before_any_launch():
    import paper_2609_00891_amd as cb
    lib = cb.library()
    assert lib.cb_plan_create(None, None, None, 0, None) == 1
    assert lib.cb_stats_accumulate(None, None, None, None, 0, None, None, None) == 1
    assert lib.cb_apply(None, None, None, None, None) == 1
    assert lib.cb_stats_zero(None, None, None, None) == 1
    assert lib.cb_plan_destroy(None) == 0
    # solve: unsupported sizes, bad flags, bad lambda -- all host-side
    assert lib.cb_ridge_solve(4, 100, 128, None, None, ctypes.c_float(0.1), 0, None, None, None) == 6
    assert lib.cb_ridge_solve(4, 129, 128, None, None, ctypes.c_float(0.1), 8, None, None, None) == 1
    assert lib.cb_ridge_solve(4, 129, 128, None, None, ctypes.c_float(-1.0), 0, None, None, None) == 1
    assert lib.cb_ridge_solve(4, 129, 128, None, None, ctypes.c_float(float("nan")), 1, None, None, None) == 1
    assert lib.cb_ridge_solve(4, 129, 128, None, None, ctypes.c_float(0.1), 1, None, None, None) == 1
    assert lib.cb_ridge_solve(0, 129, 128, None, None, ctypes.c_float(0.1), 1, None, None, None) == 0
    assert "NULL" in cb.cb_last_error() or cb.cb_last_error() == ""


def test_centered_entry_points_reject_bad_arguments_on_the_host():
    import paper_2609_00891_amd as cb
    lib = cb.library()
    assert lib.cb_stats_zero_centered(None, None, None, None, None, None) == 1
    assert lib.cb_stats_means(None, None, None, None, 0, None, None, None) == 1
    assert lib.cb_stats_accumulate_centered(None, None, None, None, 0, None, None, None, None) == 1
    assert lib.cb_stats_accumulate_shifted(None, None, None, None, 0, None, None, None, None, None) == 1
    assert lib.cb_stats_shift_finish(None, None, None, None, None, None) == 1
    f = ctypes.c_float
    solve = lib.cb_ridge_solve_centered
    assert solve(4, 80, 128, None, None, None, f(0.1), 0, None, None, None) == 6      # d_s not supported
    assert solve(4, 128, 256, None, None, None, f(0.1), 0, None, None, None) == 6     # d_t not supported
    assert solve(4, 128, 128, None, None, None, f(0.1), 4, None, None, None) == 1     # unknown flag
    assert solve(4, 128, 128, None, None, None, f(-1.0), 1, None, None, None) == 1
    assert solve(4, 128, 128, None, None, None, f(float("inf")), 1, None, None, None) == 1
    assert solve(4, 128, 128, None, None, None, f(0.1), 1, None, None, None) == 1     # NULL pointers
    assert solve(-1, 128, 128, None, None, None, f(0.1), 1, None, None, None) == 1
    assert solve(0, 128, 128, None, None, None, f(0.1), 3, None, None, None) == 0     # nothing to do
    assert "NULL" in cb.cb_last_error() or cb.cb_last_error() == ""


def test_probe_entry_points_reject_bad_arguments_and_rank_on_the_host():
    import paper_2609_00891_amd as cb
    lib = cb.library()
    assert lib.cb_probe_r2(4, 80, 128, None, None, None, None, None, None, None) == 6
    assert lib.cb_probe_r2(4, 128, 128, None, None, None, None, None, None, None) == 1
    assert lib.cb_probe_r2(0, 128, 128, None, None, None, None, None, None, None) == 0
    assert lib.cb_select_layers(None, None, 1, 1, 1, None, None) == 1
    # the host ranking: mean R^2 per (target, source) layer pair, ties to the smaller layer
    hm = {"tgt_layer": [0, 0, 0, 0, 0, 0, 1, 1], "src_layer": [0, 0, 1, 1, 2, 2, 2, 0]}
    r2 = np.array([0.2, 0.4, 0.9, 0.1, 0.5, 0.1, 0.7, 0.7])
    sel, score = cb.cb_select_layers(hm, r2, 2, 3, 3)
    np.testing.assert_allclose(score[0], [0.3, 0.5, 0.3])
    assert sel.tolist() == [[1, 0, 2], [0, 2, -1]]
    assert score[1, 1] == -np.inf
    with pytest.raises(cb.CacheBridgeError, match="CB_ERR_INVALID_ARGUMENT"):
        cb.cb_select_layers({"tgt_layer": [0], "src_layer": [5]}, np.zeros(1), 1, 3, 1)


def test_attn_entry_points_reject_bad_arguments_on_the_host():
    import paper_2609_00891_amd as cb
    lib = cb.library()
    assert lib.cb_attn_sensitivity(None, None, None, 1, None, 0, None) == 1
    bounds = (ctypes.c_int32 * 3)(4, 9, 20)
    tgt = cb.CbCache()
    tgt.n_layers, tgt.n_heads, tgt.head_dim, tgt.n_seqs, tgt.seq_len = 2, 2, 96, 1, 32
    q = cb.CbQueries()
    q.n_layers, q.n_qheads, q.head_dim, q.n_seqs, q.n_bounds = 2, 4, 96, 1, 3
    fake = ctypes.c_void_p(256)
    call = lambda: lib.cb_attn_sensitivity(ctypes.byref(tgt), ctypes.byref(q), bounds, 1, fake, 64, None)  # noqa: E731
    assert call() == 6                                            # head_dim 96
    tgt.head_dim = q.head_dim = 64
    tgt.data = 256                                                # never dereferenced: every case fails first
    q.n_qheads = 5
    assert call() == 2                                            # 5 query heads over 2 KV heads
    q.n_qheads = 6
    assert call() == 6                                            # 3 per KV head: not a power of two
    q.n_qheads = 4
    bounds[2] = 40                                                # past the sequence
    assert call() == 1
    bounds[2] = 9                                                 # not increasing
    assert call() == 1
    bounds[2] = 20
    assert lib.cb_attn_sensitivity(ctypes.byref(tgt), ctypes.byref(q), bounds, 0, fake, 64, None) == 1   # stride 0
    assert lib.cb_attn_sensitivity(ctypes.byref(tgt), ctypes.byref(q), bounds, 1, fake, 16, None) == 2   # row stride
    q.n_seqs = 2
    assert call() == 2                                            # q and tgt disagree
    assert lib.cb_attn_weights(4, 1, 32, 1, None, 32, 8, None, 32, None, None) == 1
    assert lib.cb_attn_weights(4, 1, 32, 0, fake, 32, 8, fake, 32, fake, None) == 1
    assert lib.cb_attn_weights(4, 1, 32, 1, fake, 16, 8, fake, 32, fake, None) == 2
    assert lib.cb_attn_weights(0, 1, 32, 1, None, 32, 8, None, 32, None, None) == 0


def test_rope_entry_points_reject_bad_arguments_on_the_host():
    import paper_2609_00891_amd as cb
    lib = cb.library()
    assert lib.cb_rope_table(ctypes.c_double(0.0), 128, 16, None, None) == 1
    assert lib.cb_rope_table(ctypes.c_double(1e4), 127, 16, None, None) == 6
    assert lib.cb_rope_table(ctypes.c_double(1e4), 128, 16, None, None) == 1
    assert lib.cb_rope_table(ctypes.c_double(1e4), 128, 0, None, None) == 0
    c = cb.CbCache()
    c.data, c.n_layers, c.n_heads, c.head_dim, c.n_seqs, c.seq_len = 256, 1, 1, 40, 1, 8
    c.s_layer, c.s_kv, c.s_seq, c.s_head, c.s_tok = 640, 320, 320, 320, 40

    def spec(head_dim=64, n_pos=64, style=0, off=0, table=256):
        sp = cb.CbRopeSpec()
        sp.table, sp.head_dim, sp.n_pos, sp.style, sp.pos_offset = table, head_dim, n_pos, style, off
        return sp

    def call(**kw):
        sp = spec(**kw)
        return lib.cb_rope(ctypes.byref(c), ctypes.byref(c), ctypes.byref(sp), 0, None)
    assert call(head_dim=40) == 6                        # head_dim 40 is not a multiple of 16
    c.head_dim, c.s_tok, c.s_head, c.s_seq, c.s_kv, c.s_layer = 64, 64, 512, 512, 512, 1024
    assert lib.cb_rope(ctypes.byref(c), ctypes.byref(c), None, 0, None) == 1
    assert call(style=2) == 1
    assert call(n_pos=6) == 2                            # positions 0..7 need 8 table rows
    assert call(off=60) == 2
    assert call(head_dim=128) == 2                       # a table built for another head width
    assert call(head_dim=32) == 2
    assert call(table=0) == 1
    assert call(table=264) == 3                          # tables are 16-byte aligned
    # the fused mapping and statistics: a NULL plan is refused before anything else
    sp = spec()
    assert lib.cb_apply_rope(None, ctypes.c_void_p(256), ctypes.byref(c), ctypes.byref(c), None,
                             ctypes.byref(sp), None) == 1
    assert lib.cb_stats_accumulate_rope(None, ctypes.byref(c), ctypes.byref(c), ctypes.c_void_p(256), 8,
                                        ctypes.c_void_p(256), ctypes.c_void_p(256), ctypes.byref(sp), None,
                                        None) == 1
    # the Python descriptor takes head_dim and n_pos from the table's shape
    import torch
    t = torch.zeros((40, 64, 2), dtype=torch.float32)
    d = cb.rope_spec(t, 1, 7)
    assert (d.head_dim, d.n_pos, d.style, d.pos_offset) == (128, 40, 1, 7)
    with pytest.raises(ValueError):
        cb.rope_spec(t.reshape(40, 128))


def test_multi_layer_entry_points_reject_bad_arguments_on_the_host():
    import paper_2609_00891_amd as cb
    lib = cb.library()
    hm = {"tgt_layer": [0, 1], "tgt_head": [0, 0], "kv": [0, 1], "src_layers": [[0, 1], [1, 2]],
          "src_head": [0, 0], "weight_row": [0, 1]}

    def create(h=hm, src=(3, 1, 128), tgt=(2, 1, 128), stride=1):
        return cb.cb_plan_create_multi(h, src, tgt, stride)
    with pytest.raises(cb.CacheBridgeError, match="CB_ERR_UNSUPPORTED"):
        create(src=(3, 1, 64))                                       # multi-layer maps need d = 128
    with pytest.raises(cb.CacheBridgeError, match="CB_ERR_INVALID_ARGUMENT"):
        create(stride=0)
    with pytest.raises(cb.CacheBridgeError, match="CB_ERR_INVALID_ARGUMENT"):
        create(dict(hm, src_layers=[[0, 0], [1, 2]]))                # a layer selected twice
    with pytest.raises(cb.CacheBridgeError, match="CB_ERR_INVALID_ARGUMENT"):
        create(dict(hm, src_layers=[[0, 1], [1, 3]]))                # layer outside the source model
    with pytest.raises(cb.CacheBridgeError, match="CB_ERR_UNSUPPORTED"):
        create(dict(hm, src_layers=[list(range(33))] * 2), src=(40, 1, 128))   # k > 32
    assert lib.cb_plan_create_multi(None, None, None, 1, None) == 1
    f = ctypes.c_float
    ws = lib.cb_ridge_solve_ws
    assert ws(4, 1025, 128, None, None, f(0.1), 0, None, 0, None, None, None) == 1       # NULL pointers
    assert ws(4, 1025, 100, None, None, f(0.1), 0, None, 0, None, None, None) == 6       # d_t
    assert ws(4, 5000, 128, None, None, f(0.1), 0, None, 0, None, None, None) == 6       # P too wide
    assert ws(4, 1025, 128, None, None, f(0.1), 8, None, 0, None, None, None) == 1       # unknown flag
    assert ws(0, 1025, 128, None, None, f(0.1), 1, None, 0, None, None, None) == 0
    fake = ctypes.c_void_p(256)
    assert ws(4, 1025, 128, fake, fake, f(0.1), 1, fake, 1024, fake, fake, None) == 2    # workspace too small
    assert lib.cb_ridge_solve(4, 1025, 128, fake, fake, f(0.1), 1, fake, fake, None) == 6
    per = cb.cb_ridge_solve_workspace_bytes(1025, 128, 1)
    assert per == (1025 * 1025 + 1025 * 128) * 8
    assert cb.cb_ridge_solve_workspace_bytes(1025, 128, 3) == 3 * per
    assert cb.cb_ridge_solve_workspace_bytes(129, 128, 3) == 0


def test_noalloc_solve_rejects_systems_beyond_its_scratch_before_any_launch():
    # The allocation-free solve factors in a fixed device array; a system whose
    # factor would not fit is refused on the host (no device is touched here).
    import paper_2609_00891_amd as cb
    lib = cb.library()
    cap = int(lib.cb_ridge_solve_noalloc_max_bytes())
    assert cap == 128 << 20
    fake = ctypes.c_void_p(0x1000)
    for P, d_t, ok in ((4032, 128, True), (4033, 128, False), (4097, 64, False)):
        need = int(lib.cb_ridge_solve_workspace_bytes(P, d_t, 1))
        assert (need <= cap) == ok
    rc = lib.cb_ridge_solve_noalloc(1, 4033, 128, fake, fake, ctypes.c_float(1e-2), 1, fake, fake, None)
    assert cb.cb_status_string(rc) == "CB_ERR_UNSUPPORTED"
    assert b"scratch" in lib.cb_last_error()
    rc = lib.cb_ridge_solve_noalloc(1, 4098, 128, fake, fake, ctypes.c_float(1e-2), 1, fake, fake, None)
    assert cb.cb_status_string(rc) == "CB_ERR_UNSUPPORTED"
    rc = lib.cb_ridge_solve_noalloc(1, 1025, 128, None, fake, ctypes.c_float(1e-2), 1, fake, fake, None)
    assert cb.cb_status_string(rc) == "CB_ERR_INVALID_ARGUMENT"


def test_centered_wide_solve_rejects_bad_arguments_on_the_host():
    import paper_2609_00891_amd as cb
    lib = cb.library()
    f = ctypes.c_float
    sv = lib.cb_ridge_solve_centered_ws
    fake = ctypes.c_void_p(256)
    assert sv(4, 1024, 128, None, None, None, f(0.1), 1, None, 0, None, None, None) == 1      # NULL pointers
    assert sv(4, 5000, 128, fake, fake, fake, f(0.1), 1, fake, 1 << 40, fake, fake, None) == 6   # d_x too wide
    assert sv(4, 1024, 100, fake, fake, fake, f(0.1), 1, fake, 1 << 40, fake, fake, None) == 6   # d_t
    assert sv(4, 1024, 128, fake, fake, fake, f(-1.0), 1, fake, 1 << 40, fake, fake, None) == 1  # lambda < 0
    assert sv(4, 1024, 128, fake, fake, fake, f(0.1), 4, fake, 1 << 40, fake, fake, None) == 1   # unknown flag
    assert sv(4, 1024, 128, fake, fake, fake, f(0.1), 1, fake, 1024, fake, fake, None) == 2      # workspace too small
    assert sv(0, 1024, 128, None, None, None, f(0.1), 1, None, 0, None, None, None) == 0


def test_bindings_check_output_sizes_against_the_plan():
    # the C ABI takes bare pointers; the binding refuses tensors that do not hold
    # what the plan's kernels write or read, before any call into the library
    import torch
    import paper_2609_00891_amd as cb
    keep = [np.zeros(4, np.int32)] * 5 + [np.arange(4, dtype=np.int32)]
    plan = cb.Plan(None, 4, 128, 128, keep, P=385, k=3)
    z32 = lambda *s: torch.zeros(s, dtype=torch.float32)           # noqa: E731
    z64 = lambda *s: torch.zeros(s, dtype=torch.float64)           # noqa: E731
    src = torch.zeros((4, 2, 2, 1, 8, 128), dtype=torch.bfloat16)
    with pytest.raises(ValueError, match="sums"):
        cb.cb_stats_zero_centered(plan, z64(4, 257), z32(4, 384, 384), z32(4, 384, 128))
    with pytest.raises(ValueError, match="A"):
        cb.cb_stats_zero_centered(plan, z64(4, 513), z32(4, 128, 128), z32(4, 384, 128))
    with pytest.raises(ValueError, match="sums"):                 # the pilot sums are sized like sums
        cb.cb_stats_shift_finish(plan, z64(4, 257), z64(4, 513), z32(4, 384, 384), z32(4, 384, 128))
    with pytest.raises(ValueError, match="B"):
        cb.cb_stats_shift_finish(plan, z64(4, 513), z64(4, 513), z32(4, 384, 384), z32(4, 128, 128))
    with pytest.raises(ValueError, match="G"):
        cb.cb_stats_zero(plan, z32(4, 129, 129), z32(4, 385, 128))
    with pytest.raises(ValueError, match="maps"):
        cb.cb_apply(plan, z32(4, 129, 128), src, src)
    with pytest.raises(ValueError, match="weights"):
        cb.cb_stats_means(plan, src, src, z32(3, 16), z64(4, 513))                  # 3 rows, the map reads 4
    with pytest.raises(ValueError, match="weights"):
        cb.cb_stats_means(plan, src, src, z32(4, 16)[:, 1:], z64(4, 513), w_row_stride=16)    # 63 < 64 values
    with pytest.raises(ValueError, match="weights"):
        cb.cb_stats_means(plan, src, src, z32(16, 4).t(), z64(4, 513), w_row_stride=16)   # strided rows
