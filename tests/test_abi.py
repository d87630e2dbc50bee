"""Host-side checks of libviscache: it loads, exports every entry point the
header declares, its budget rule agrees with the oracle's on a sweep, and bad
arguments are rejected on the host before anything is enqueued (no GPU
needed: the checks run before any device call)."""
import ctypes
import math
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="session")
def vc():
    import paper_2608_24063_amd as vc
    if not os.path.exists(vc.LIB_PATH):
        from paper_2608_24063_amd import build
        build.build()
    vc.lib()
    return vc


def test_exports_every_declared_symbol(vc):
    hdr = open(os.path.join(ROOT, "include", "viscache.h")).read()
    declared = set(re.findall(r"\b(viscache_\w+)\s*\(", hdr))
    assert len(declared) >= 9
    lib = ctypes.CDLL(vc.LIB_PATH)
    for name in declared:
        assert hasattr(lib, name), name
    assert declared == set(vc.EXPORTED)


def test_defaults_match_paper(vc):
    p = vc.make_params(0.28)
    assert (p.h, p.m, p.tau, p.mu, p.rank_mode, p.v_out_fp32) == (0, 0.75, pytest.approx(1.0),
                                                                    pytest.approx(0.7), 0, 0)
    assert (p.schedule, p.drop_all) == (vc.VC_SCHED_PARABOLIC, 0)


def test_schedule_and_drop_all_are_checked(vc):
    shape = vc.make_shape(1, 4, 8, 2, 64, 4, [64])
    for bad in (dict(schedule=4), dict(schedule=-1), dict(drop_all=2)):
        p = vc.make_params(0.25)
        for k, v in bad.items():
            setattr(p, k, v)
        with pytest.raises(vc.VisCacheError) as ei:
            vc.viscache_budget(shape, p)
        assert ei.value.status == vc.VC_ERR_ARG


@pytest.mark.parametrize("schedule,drop_all", [(0, False), (1, False), (2, False), (3, False), (0, True)])
@pytest.mark.parametrize("L", [2, 3, 4, 8, 28, 36, 64, 80])
def test_budget_matches_oracle(vc, orc, L, schedule, drop_all):
    for n in [0, 1, 7, 64, 511, 512, 3136, 12544, 23040]:
        for rr in [0.05, 0.19, 0.22, 0.25, 0.28, 0.40, 0.5625]:
            for m in [0.75, 0.9]:
                shape = vc.make_shape(1, L, 8, 2, 64, 4, [n])
                params = vc.make_params(rr, m=m, schedule=schedule, drop_all=drop_all)
                try:
                    ref = orc.budget(L=L, n=n, rr=rr, m=m, schedule=schedule, drop_all=drop_all)
                except ValueError:
                    with pytest.raises(vc.VisCacheError) as ei:
                        vc.viscache_budget(shape, params)
                    assert ei.value.status == vc.VC_ERR_BUDGET
                    continue
                k, ns, h = vc.viscache_budget(shape, params)
                assert k == list(ref["k"]) and h == ref["h"]
                assert all(x == ref["n_surv"] for x in ns)


def test_budget_ragged_batch_and_out_rows(vc, orc, sg):
    w = sg.BATCHED
    n = [int(x) for x in w.n_vis()] + [0, 5]
    shape = vc.make_shape(len(n), w.L, w.Hq, w.Hkv, w.d, w.W, n)
    params = vc.make_params(w.retention)
    k, ns, h = vc.viscache_budget(shape, params)
    rows = vc.viscache_out_rows(shape, params)
    B = len(n)
    for b, nb in enumerate(n):
        ref = orc.budget(L=w.L, n=nb, rr=w.retention)
        assert k[b * w.L:(b + 1) * w.L] == list(ref["k"])
    for l in range(w.L):
        acc = 0
        for b in range(B):
            assert rows[l * (B + 1) + b] == acc
            acc += w.Hkv * k[b * w.L + l]
        assert rows[l * (B + 1) + B] == acc
    assert sum(k[:w.L]) == math.floor(w.retention * w.L * n[0] + 0.5)


def test_workspace_sizes(vc, sg):
    for w in sg.WORKLOADS.values():
        shape = vc.make_shape(w.B, w.L, w.Hq, w.Hkv, w.d, w.W, w.n_vis())
        for mode in (0, 1):
            assert vc.viscache_prune_workspace_bytes(shape, vc.make_params(w.retention, rank_mode=mode)) > 0
    ds = vc.vc_decode_shape(1, 28, 28, 4, 128)
    assert vc.viscache_decode_workspace_bytes(ds, 4000) >= 28 * 4 * 16 * 128 * 4


@pytest.mark.parametrize("bad,status", [
    (dict(d=96), "VC_ERR_UNSUPPORTED"), (dict(Hq=7, Hkv=2), "VC_ERR_SHAPE"),
    (dict(n=[40000]), "VC_ERR_UNSUPPORTED"), (dict(n=[-1]), "VC_ERR_SHAPE"),
    (dict(L=1), "VC_ERR_SHAPE"), (dict(W=0), "VC_ERR_SHAPE"), (dict(W=300, Hq=8, Hkv=2), "VC_ERR_UNSUPPORTED"),
    (dict(rr=0.9), "VC_ERR_BUDGET"), (dict(rr=0.0), "VC_ERR_BUDGET"), (dict(h=1), "VC_ERR_BUDGET"),
    (dict(h=99), "VC_ERR_BUDGET"), (dict(m=1.5), "VC_ERR_BUDGET"), (dict(tau=0.0), "VC_ERR_ARG"),
    (dict(mu=1.5), "VC_ERR_ARG"), (dict(rank_mode=7), "VC_ERR_ARG"),
])
def test_bad_arguments_rejected(vc, bad, status):
    a = dict(B=1, L=4, Hq=8, Hkv=2, d=64, W=32, n=[512], rr=0.25, h=0, m=0.75, tau=1.0, mu=0.7, rank_mode=0)
    a.update(bad)
    shape = vc.make_shape(len(a["n"]), a["L"], a["Hq"], a["Hkv"], a["d"], a["W"], a["n"])
    params = vc.make_params(a["rr"], h=a["h"], m=a["m"], tau=a["tau"], mu=a["mu"], rank_mode=a["rank_mode"])
    with pytest.raises(vc.VisCacheError) as ei:
        vc.viscache_budget(shape, params)
    assert ei.value.status == getattr(vc, status)
    assert vc.viscache_prune_workspace_bytes(shape, params) == 0
    # The device entry point fails the same way before touching any pointer.
    L = a["L"]
    with pytest.raises(vc.VisCacheError) as ei:
        vc.viscache_prune(shape, params, [1] * L, [1] * L, [1] * L, [1] * L, [1] * L, [1] * L,
                          256, 1 << 30, 0)
    assert ei.value.status == getattr(vc, status)


def test_prune_rejects_missing_buffers_and_small_workspace(vc):
    shape = vc.make_shape(1, 4, 8, 2, 64, 32, [512])
    params = vc.make_params(0.25)
    need = vc.viscache_prune_workspace_bytes(shape, params)
    with pytest.raises(vc.VisCacheError) as ei:
        vc.viscache_prune(shape, params, [1] * 4, [1] * 4, [1] * 4, [1] * 4, [1] * 4, [1] * 4,
                          256, need - 1, 0)
    assert ei.value.status == vc.VC_ERR_WORKSPACE
    with pytest.raises(vc.VisCacheError) as ei:
        vc.viscache_prune(shape, params, [1] * 4, [1] * 4, [1] * 4, [1] * 4, [1] * 4, [1] * 4,
                          257, need + 512, 0)
    assert ei.value.status == vc.VC_ERR_WORKSPACE
    with pytest.raises(vc.VisCacheError) as ei:
        vc.viscache_prune(shape, params, [0] * 4, [1] * 4, [1] * 4, [1] * 4, [1] * 4, [1] * 4,
                          256, need, 0)
    assert ei.value.status == vc.VC_ERR_ARG


def test_decode_rejects_bad_arguments(vc):
    ds = vc.vc_decode_shape(1, 2, 40, 2, 128)  # 20 query heads per kv head
    c = vc.vc_cache(256, 256, 256, 256, 256)
    with pytest.raises(vc.VisCacheError) as ei:
        vc.viscache_decode_attn(ds, c, 256, 256, 0.1, 100, 256, 1 << 20, 0)
    assert ei.value.status == vc.VC_ERR_UNSUPPORTED
    ds = vc.vc_decode_shape(1, 2, 8, 2, 128)
    need = vc.viscache_decode_workspace_bytes(ds, 100)
    with pytest.raises(vc.VisCacheError) as ei:
        vc.viscache_decode_attn(ds, c, 256, 256, 0.1, 100, 256, need - 1, 0)
    assert ei.value.status == vc.VC_ERR_WORKSPACE
    with pytest.raises(vc.VisCacheError) as ei:
        vc.viscache_decode_attn(ds, c, 256, 256, -1.0, 100, 256, need, 0)
    assert ei.value.status == vc.VC_ERR_ARG
    with pytest.raises(vc.VisCacheError) as ei:
        vc.viscache_append_kv(ds, vc.vc_cache(0, 256, 256, 256, 256), 256, 256, 0)
    assert ei.value.status == vc.VC_ERR_ARG


def test_decode_row_limit(vc):
    """Long caches are accepted: the workspace holds one partial per
    workgroup, and the grid stops growing once it fills the resident slots,
    so it does not grow with the rows; a row bound whose tile count overflows
    31 bits is refused on the host."""
    ds = vc.vc_decode_shape(1, 2, 8, 2, 128)
    big = vc.viscache_decode_workspace_bytes(ds, 1 << 28)
    assert big == vc.viscache_decode_workspace_bytes(ds, 32768) > vc.viscache_decode_workspace_bytes(ds, 64) > 0
    assert vc.viscache_decode_step_workspace_bytes(ds, 1 << 28) > big
    assert vc.viscache_decode_workspace_bytes(ds, 1 << 35) == 0
    assert vc.viscache_decode_step_workspace_bytes(ds, 1 << 35) == 0
    c = vc.vc_cache(256, 256, 256, 256, 256)
    with pytest.raises(vc.VisCacheError) as ei:
        vc.viscache_decode_attn(ds, c, 256, 256, 0.1, 1 << 35, 256, big, 0)
    assert ei.value.status == vc.VC_ERR_UNSUPPORTED


def test_prefill_scoring_arguments(vc):
    """score_queries is validated; prefill scoring lifts the window limit on
    (Hq/Hkv)*W (its rows are G*(n+W) per unit, up to 2^26), needs no bf16
    window-query buffer, and needs the text keys of every scored layer."""
    p = vc.make_params(0.25)
    assert p.score_queries == vc.VC_SCORE_WINDOW
    shape = vc.make_shape(1, 4, 8, 2, 64, 32, [512])
    for bad in (2, -1):
        q = vc.make_params(0.25, score_queries=bad)
        with pytest.raises(vc.VisCacheError) as ei:
            vc.viscache_budget(shape, q)
        assert ei.value.status == vc.VC_ERR_ARG
    wide = vc.make_shape(1, 4, 8, 2, 64, 300, [512])
    assert vc.viscache_prune_workspace_bytes(wide, vc.make_params(0.25)) == 0
    pre = vc.make_params(0.25, score_queries=vc.VC_SCORE_PREFILL)
    assert vc.viscache_prune_workspace_bytes(wide, pre) > 0
    # Window and prefill workspaces differ only in their scratch: the prefill
    # row statistics (G*(n+W) per unit) replace the window's bf16 queries and
    # split statistics.
    assert vc.viscache_prune_workspace_bytes(shape, pre) != vc.viscache_prune_workspace_bytes(shape, p)
    # Rows beyond 2^26 per unit are refused.
    huge = vc.make_shape(1, 4, 4096, 1, 64, 16384, [32768])
    assert vc.viscache_prune_workspace_bytes(huge, pre) == 0
    need = vc.viscache_prune_workspace_bytes(shape, pre)
    with pytest.raises(vc.VisCacheError) as ei:  # no text keys
        vc.viscache_prune(shape, pre, [1] * 4, [1] * 4, [1] * 4, [1] * 4, [1] * 4, [1] * 4, 256, need, 0)
    assert ei.value.status == vc.VC_ERR_ARG
    with pytest.raises(vc.VisCacheError) as ei:  # a scored layer without them
        vc.viscache_prune(shape, pre, [1] * 4, [1] * 4, [1] * 4, [1] * 4, [1] * 4, [1] * 4, 256, need, 0,
                          k_text=[1, 1, 0, 1])
    assert ei.value.status == vc.VC_ERR_ARG


def test_layout_reuse_follows_contents(vc, orc):
    """The library reuses its last plan while shape, lengths and parameters
    are unchanged: results must follow the contents, not the pointers."""
    import ctypes
    arr = (ctypes.c_int32 * 2)(3136, 700)
    shape = vc.vc_shape(2, 28, 28, 4, 128, 64, ctypes.cast(arr, ctypes.POINTER(ctypes.c_int32)))
    p = vc.make_params(0.28)
    k1, _, _ = vc.viscache_budget(shape, p)
    assert k1[:28] == list(orc.budget(L=28, n=3136, rr=0.28)["k"])
    arr[1] = 1500  # same array, new length
    k2, _, _ = vc.viscache_budget(shape, p)
    assert k2[28:] == list(orc.budget(L=28, n=1500, rr=0.28)["k"])
    assert vc.viscache_out_rows(shape, p)[-1] == 4 * (k2[27] + k2[55])
    p.retention = 0.19  # same struct, new retention
    k3, _, _ = vc.viscache_budget(shape, p)
    assert k3[:28] == list(orc.budget(L=28, n=3136, rr=0.19)["k"])
    p.tau = 0.0  # an invalid parameter is still refused after a valid call
    with pytest.raises(vc.VisCacheError) as ei:
        vc.viscache_budget(shape, p)
    assert ei.value.status == vc.VC_ERR_ARG
    p.tau = 1.0
    assert vc.viscache_budget(shape, p)[0] == k3
    one = vc.make_shape(1, 28, 28, 4, 128, 64, [3136])  # fewer sequences than the cached plan
    assert vc.viscache_budget(one, p)[0] == k3[:28]


def test_q4_arguments(vc):
    """4-bit entry points: shape, null and alignment checks run on the host."""
    with pytest.raises(vc.VisCacheError) as ei:
        vc.viscache_quantize_rows(96, 4, 256, 256, 256, 0)
    assert ei.value.status == vc.VC_ERR_UNSUPPORTED
    with pytest.raises(vc.VisCacheError) as ei:
        vc.viscache_quantize_rows(128, -1, 256, 256, 256, 0)
    assert ei.value.status == vc.VC_ERR_ARG
    vc.viscache_quantize_rows(128, 0, 0, 0, 0, 0)  # nothing to do, nothing enqueued
    for src, codes, meta in ((0, 256, 256), (264, 256, 256), (256, 260, 256), (256, 256, 260)):
        with pytest.raises(vc.VisCacheError) as ei:
            vc.viscache_quantize_rows(64, 4, src, codes, meta, 0)
        assert ei.value.status == vc.VC_ERR_ARG
    ds = vc.vc_decode_shape(1, 2, 8, 2, 128)
    c = vc.vc_cache(256, 256, 256, 256, 256)
    need = vc.viscache_decode_step_workspace_bytes(ds, 100)
    good = (256, 256, 256, 256, 256, 256)
    for i in range(6):
        f = list(good)
        f[i] = 0
        with pytest.raises(vc.VisCacheError) as ei:
            vc.viscache_decode_step_q4(ds, c, vc.vc_qcache(*f), 256, 256, 256, 256, 0.1, 100, 256, need, 0)
        assert ei.value.status == vc.VC_ERR_ARG
    for i, bad in ((0, 258), (1, 260), (2, 258), (3, 260)):
        f = list(good)
        f[i] = bad
        with pytest.raises(vc.VisCacheError) as ei:
            vc.viscache_decode_step_q4(ds, c, vc.vc_qcache(*f), 256, 256, 256, 256, 0.1, 100, 256, need, 0)
        assert ei.value.status == vc.VC_ERR_ARG
    with pytest.raises(vc.VisCacheError) as ei:
        vc.viscache_decode_step_q4(ds, c, vc.vc_qcache(*good), 256, 256, 256, 256, 0.1, 100, 256, need - 1, 0)
    assert ei.value.status == vc.VC_ERR_WORKSPACE


def test_fusion_unit_rank_limit(vc):
    """A fusion job packs a unit's rank into 23 bits: 2^23 units with kept
    tokens are refused on the host, one fewer is accepted."""
    def status(Hkv):
        # L = h = 2, RR = 1, m = 1: both layers keep all 4 tokens of every head
        shape = vc.make_shape(1, 2, Hkv, Hkv, 64, 1, [4])
        try:
            vc.viscache_budget(shape, vc.make_params(1.0, h=2, m=1.0))
        except vc.VisCacheError as e:
            return e.status
        return vc.VC_OK

    assert status(1 << 22) == vc.VC_ERR_UNSUPPORTED       # 2 * 2^22 = 2^23 units
    assert status((1 << 22) - 1) == vc.VC_OK              # 2^23 - 2 units
