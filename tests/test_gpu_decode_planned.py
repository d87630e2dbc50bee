"""GPU parity of the planned decode step (viscache_decode_plan on the host,
viscache_decode_step_planned on the device) against the oracle's decode
attention (Sec. 2, decoding), through the C ABI.

The planned kernel reads each wave's first tile before it knows the unit's
length, up to the piece's planned end, and patches rows that are not this
step's.  The pools are therefore filled with NaN past every unit's length
(and at the row each step appends) before the first step: any such row that
reached a product would turn the output into NaN."""
import numpy as np
import pytest

from tests.parity import fused_error

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
TOL = 1e-4
NAN_BF16 = 0x7FC0


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2608_24063_amd as vc
    vc.lib()
    return torch.device("cuda:0")


def _check_out(orc, q, K, V, out, scale, what):
    ref = orc.attend(q, K, V, scale)
    err = fused_error(ref[None, :], out[None, :])
    assert err <= TOL, f"{what}: decode error {err}"


def _fill(c, Kp, Vp, lens, dev):
    """Pool rows [0, len) of each unit from Kp / Vp, NaN everywhere else."""
    from synthgen.device import bf16_tensor
    K = np.full_like(Kp, NAN_BF16)
    V = np.full_like(Vp, NAN_BF16)
    for u, n in enumerate(lens):
        r0 = c.offs_host[u]
        K[r0:r0 + n] = Kp[r0:r0 + n]
        V[r0:r0 + n] = Vp[r0:r0 + n]
    c.k_pool.copy_(bf16_tensor(K, dev))
    c.v_pool.copy_(bf16_tensor(V, dev))
    c.len.copy_(torch.tensor(lens, dtype=torch.int32))


def _bits_equal(a, b):
    return torch.equal(a.view(torch.int16), b.view(torch.int16))


def _counters_zero(c, units):
    import paper_2608_24063_amd as vc
    base = vc.viscache_decode_workspace_bytes(c.shape, c.max_cap)
    assert int(c.step_ws[base:base + 4 * units].view(torch.int32).abs().sum()) == 0


def _step_unplanned(c, kt, vt, qt, out, scale, max_rows):
    import paper_2608_24063_amd as vc
    vc.viscache_decode_step(c.shape, c.c, kt.data_ptr(), vt.data_ptr(), qt.data_ptr(), out.data_ptr(), scale,
                            max_rows, c.step_ws.data_ptr(), c.step_ws_bytes, torch.cuda.current_stream().cuda_stream)


@pytest.mark.parametrize("d,Hq,Hkv,max_rows,hint", [(128, 8, 2, None, "now"), (64, 28, 4, None, "none"),
                                                    (128, 64, 8, None, "now"), (128, 28, 4, 2000, "now"),
                                                    (128, 8, 2, None, "stale"), (64, 28, 4, None, "stale")])
def test_planned_step_random_caches(dev, orc, sg, d, Hq, Hkv, max_rows, hint):
    """Lengths on and around tile edges, empty units, units cut into many
    pieces, capacities with no room, little room and much room (a long NaN
    tail that the first tiles read before the length is known), five steps:
    the same lengths and pools as viscache_decode_step, and every head of
    every unit against the oracle at every step.  The table's length hint is
    the lengths now, none (early reads up to the capacity), or stale (500
    rows short: the early reads fall short and are read again)."""
    from paper_2608_24063_amd.tensors import DecodeCache
    from synthgen.device import bf16_tensor, to_host_bf16
    L, B = 2, 2
    units = L * B * Hkv
    lens = [0, 1, 31, 32, 33, 3100, 511, 1023, 1024, 1100, 5, 64, 2049, 2, 1025, 47, 4097, 63, 65, 95, 96,
            97, 160, 300, 0, 1, 2500, 31, 700, 12, 5000, 128][:units]
    slack = [3, 0, 1, 2, 40, 300, 6, 1, 0, 90, 3, 33, 5, 700, 2, 9, 4, 1, 31, 32, 33, 2, 5, 64, 0, 3, 100, 1,
             2, 3, 4, 5][:units]
    caps = [n + s for n, s in zip(lens, slack)]
    if max_rows is not None:
        # The bound holds every length the steps reach; some capacities
        # reach past it (their tables stop at the bound).
        lens = [min(n, max_rows - 8) for n in lens]
        caps = [n + s + (1500 if i % 3 == 0 else 0) for i, (n, s) in enumerate(zip(lens, slack))]
    rows = max(caps) if max_rows is None else max_rows
    c = DecodeCache(L, B, Hq, Hkv, d, caps, dev)
    a = DecodeCache(L, B, Hq, Hkv, d, caps, dev)
    Kp = sg.normal_bf16(81, 1, (c.total_rows, d))
    Vp = sg.normal_bf16(81, 2, (c.total_rows, d))
    for cc in (c, a):
        _fill(cc, Kp, Vp, lens, dev)
    c.plan(rows, hint={"now": True, "none": False, "stale": [max(0, n - 500) for n in lens]}[hint])
    scale = d ** -0.5
    G = Hq // Hkv
    cur = list(lens)
    for t in range(5):
        kn = sg.normal_bf16(82 + t, 1, (L, B, Hkv, d))
        vn = sg.normal_bf16(82 + t, 2, (L, B, Hkv, d))
        q = sg.normal_bf16(82 + t, 3, (L, B, Hq, d))
        kt, vt, qt = bf16_tensor(kn, dev), bf16_tensor(vn, dev), bf16_tensor(q, dev)
        out_c = torch.full((L, B, Hq, d), float("nan"), dtype=torch.float32, device=dev)
        out_a = torch.full((L, B, Hq, d), float("nan"), dtype=torch.float32, device=dev)
        c.step_planned(kt, vt, qt, out_c, scale)
        _step_unplanned(a, kt, vt, qt, out_a, scale, rows)
        torch.cuda.synchronize()
        cur = [min(x + 1, cap) for x, cap in zip(cur, caps)]
        assert c.len.cpu().tolist() == cur == a.len.cpu().tolist(), f"step {t}: lengths"
        assert _bits_equal(c.k_pool, a.k_pool) and _bits_equal(c.v_pool, a.v_pool), f"step {t}: pools differ"
        K, V, o = to_host_bf16(c.k_pool), to_host_bf16(c.v_pool), out_c.cpu().numpy()
        assert not np.isnan(o).any(), f"step {t}: NaN in the output"
        for l in range(L):
            for b in range(B):
                for g in range(Hkv):
                    u = (l * B + b) * Hkv + g
                    r0, n = c.offs_host[u], min(cur[u], rows)
                    for hh in range(G):
                        h = g * G + hh
                        if n == 0:
                            assert np.all(o[l, b, h] == 0)
                            continue
                        _check_out(orc, q[l, b, h], K[r0:r0 + n], V[r0:r0 + n], o[l, b, h], scale,
                                   f"step {t} u={u} h={h} n={n}")
    _counters_zero(c, units)


def test_planned_step_over_pruned_cache(dev, orc, sg):
    """prune -> cache of (kept visual | text window | 6 generated rows of
    room, NaN) -> planned steps, each checked against the oracle."""
    import paper_2608_24063_amd as vc
    from paper_2608_24063_amd.tensors import DecodeCache, PruneCall
    from synthgen.device import bf16_tensor, to_host_bf16, upload_layers
    w = sg.TINY
    n = [int(x) for x in w.n_vis()]
    params = vc.make_params(w.retention)
    dv, host = upload_layers(w, range(w.L), dev, keep_host=True)
    pc = PruneCall(w.B, w.L, w.Hq, w.Hkv, w.d, w.W, n, params, [dv["K"][l] for l in range(w.L)],
                   [dv["V"][l] for l in range(w.L)], [dv["Q"][l] for l in range(w.L)])
    pc.run()
    steps = 6
    caps, kept = [], []
    for l in range(w.L):
        for b in range(w.B):
            for g in range(w.Hkv):
                k = pc.k[b * w.L + l]
                kept.append(k)
                caps.append(k + w.W + steps)
    c = DecodeCache(w.L, w.B, w.Hq, w.Hkv, w.d, caps, dev)
    c.k_pool.fill_(float("nan"))
    c.v_pool.fill_(float("nan"))
    text_k = sg.normal_bf16(w.seed, 11, (len(caps), w.W, w.d))
    text_v = sg.normal_bf16(w.seed, 12, (len(caps), w.W, w.d))
    lens = []
    for l in range(w.L):
        for b in range(w.B):
            for g in range(w.Hkv):
                u = (l * w.B + b) * w.Hkv + g
                r0, k = c.offs_host[u], kept[u]
                if k:
                    a0, a1 = pc.unit_rows(l, b, g)
                    c.k_pool[r0:r0 + k] = pc.k_out[l][a0:a1]
                    c.v_pool[r0:r0 + k] = pc.v_out[l][a0:a1]
                c.k_pool[r0 + k:r0 + k + w.W] = bf16_tensor(text_k[u], dev)
                c.v_pool[r0 + k:r0 + k + w.W] = bf16_tensor(text_v[u], dev)
                lens.append(k + w.W)
    c.len.copy_(torch.tensor(lens, dtype=torch.int32))
    c.plan()
    scale = w.d ** -0.5
    out = torch.empty((w.L, w.B, w.Hq, w.d), dtype=torch.float32, device=dev)
    for t in range(steps):
        kn = sg.normal_bf16(w.seed, 100 + 3 * t, (w.L, w.B, w.Hkv, w.d))
        vn = sg.normal_bf16(w.seed, 101 + 3 * t, (w.L, w.B, w.Hkv, w.d))
        q = sg.normal_bf16(w.seed, 102 + 3 * t, (w.L, w.B, w.Hq, w.d))
        c.step_planned(bf16_tensor(kn, dev), bf16_tensor(vn, dev), bf16_tensor(q, dev), out, scale)
        torch.cuda.synchronize()
        K, V, o = to_host_bf16(c.k_pool), to_host_bf16(c.v_pool), out.cpu().numpy()
        ln = c.len.cpu().numpy()
        for l in range(w.L):
            for b in range(w.B):
                for g in range(w.Hkv):
                    u = (l * w.B + b) * w.Hkv + g
                    assert ln[u] == lens[u] + t + 1
                    r0 = c.offs_host[u]
                    for hh in range(w.G):
                        h = g * w.G + hh
                        _check_out(orc, q[l, b, h], K[r0:r0 + ln[u]], V[r0:r0 + ln[u]], o[l, b, h], scale,
                                   f"step {t} l={l} b={b} h={h}")


def test_planned_many_units_and_long_unit(dev, orc, sg):
    """1280 units, most short or empty, one of 40000 rows, one with no room:
    more pieces than resident workgroups, merges of many partials."""
    from paper_2608_24063_amd.tensors import DecodeCache
    from synthgen.device import bf16_tensor, to_host_bf16
    L, B, Hq, Hkv, d = 2, 80, 16, 8, 64
    units = L * B * Hkv
    rng = np.random.default_rng(5)
    lens = [int(x) for x in rng.integers(0, 70, size=units)]
    lens[3], lens[700], lens[1279] = 40000, 5000, 0
    caps = [x + 2 for x in lens]
    caps[1279] = 0
    c = DecodeCache(L, B, Hq, Hkv, d, caps, dev)
    Kp = sg.normal_bf16(31, 1, (c.total_rows, d))
    Vp = sg.normal_bf16(31, 2, (c.total_rows, d))
    _fill(c, Kp, Vp, lens, dev)
    c.plan()
    scale = d ** -0.5
    kn = sg.normal_bf16(32, 1, (L, B, Hkv, d))
    vn = sg.normal_bf16(32, 2, (L, B, Hkv, d))
    q = sg.normal_bf16(32, 3, (L, B, Hq, d))
    out = torch.full((L, B, Hq, d), float("nan"), dtype=torch.float32, device=dev)
    c.step_planned(bf16_tensor(kn, dev), bf16_tensor(vn, dev), bf16_tensor(q, dev), out, scale)
    torch.cuda.synchronize()
    cur = [min(x + 1, cap) for x, cap in zip(lens, caps)]
    assert c.len.cpu().tolist() == cur
    _counters_zero(c, units)
    K, V, o = to_host_bf16(c.k_pool), to_host_bf16(c.v_pool), out.cpu().numpy()
    G = Hq // Hkv
    for l in range(L):
        for b in range(B):
            for g in range(Hkv):
                u = (l * B + b) * Hkv + g
                r0, n = c.offs_host[u], cur[u]
                if n == 0:
                    assert np.all(o[l, b, g * G:(g + 1) * G] == 0)
                    continue
                h = g * G + (u % G)
                _check_out(orc, q[l, b, h], K[r0:r0 + n], V[r0:r0 + n], o[l, b, h], scale, f"u={u} n={n}")


def test_planned_table_mismatch(dev, sg):
    """A table built for another row bound fills the output with NaN and
    leaves lengths and pools alone; a table too short for the launch is
    refused on the host."""
    import paper_2608_24063_amd as vc
    from paper_2608_24063_amd.tensors import DecodeCache
    from synthgen.device import bf16_tensor
    L, B, Hq, Hkv, d = 2, 1, 8, 2, 128
    lens = [100, 0, 3000, 64]
    caps = [x + 5 for x in lens]
    c = DecodeCache(L, B, Hq, Hkv, d, caps, dev)
    _fill(c, sg.normal_bf16(91, 1, (c.total_rows, d)), sg.normal_bf16(91, 2, (c.total_rows, d)), lens, dev)
    c.plan(max(caps) - 1)
    k0, v0 = c.k_pool.clone(), c.v_pool.clone()
    kt = bf16_tensor(sg.normal_bf16(92, 1, (L, B, Hkv, d)), dev)
    vt = bf16_tensor(sg.normal_bf16(92, 2, (L, B, Hkv, d)), dev)
    qt = bf16_tensor(sg.normal_bf16(92, 3, (L, B, Hq, d)), dev)
    out = torch.zeros((L, B, Hq, d), dtype=torch.float32, device=dev)
    c.step_planned(kt, vt, qt, out, d ** -0.5, max_rows=max(caps))
    torch.cuda.synchronize()
    assert torch.isnan(out).all()
    assert c.len.cpu().tolist() == lens
    assert _bits_equal(c.k_pool, k0) and _bits_equal(c.v_pool, v0)
    with pytest.raises(vc.VisCacheError) as e:
        vc.viscache_decode_step_planned(c.shape, c.c, None, c.plan_dev.data_ptr(), c.plan_bytes - 32,
                                        kt.data_ptr(), vt.data_ptr(), qt.data_ptr(), out.data_ptr(), d ** -0.5,
                                        c.plan_rows, c.step_ws.data_ptr(), c.step_ws_bytes,
                                        torch.cuda.current_stream().cuda_stream)
    assert e.value.status == vc.VC_ERR_ARG
