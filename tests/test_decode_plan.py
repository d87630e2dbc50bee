"""The host-built piece table of the planned decode step
(viscache_decode_plan), checked on the CPU: every unit's rows are covered once
in whole tiles, slots and piece counts agree, the per-wave share is the
smallest one that fits the launch, pieces are dealt longest first, and bad
caches are refused."""
import numpy as np
import pytest

import paper_2608_24063_amd as vc

TILE = 32


def _table(shape, cap, off, max_rows, hint=None):
    """Header and records, the records unpacked to (u, j, np, p0, r0, r1, rs,
    first pool row)."""
    blob = vc.viscache_decode_plan(shape, cap, off, max_rows, hint)
    a = np.frombuffer(blob, dtype=np.int32)
    r = a[8:].reshape(-1, 8).astype(np.int64)
    rec = np.stack([r[:, 0], r[:, 1] & 0xFFFF, r[:, 1] >> 16, r[:, 2], r[:, 3], r[:, 4], r[:, 5],
                    (r[:, 7] << 32) | (r[:, 6] & 0xFFFFFFFF)], axis=1)
    return a[:8], rec


def _check(shape, cap, off, max_rows, hint=None):
    hdr, rec = _table(shape, cap, off, max_rows, hint)
    units = shape.L * shape.B * shape.Hkv
    nwg, P = int(hdr[2]), int(hdr[5])
    assert hdr[0] == 0x50444356 and hdr[1] == units and hdr[3] == shape.d and hdr[4] == min(max_rows, 2**31 - 1)
    assert len(rec) == nwg and units <= P <= nwg
    assert np.all(rec[P:, 0] == -1)
    live = rec[:P]
    capb = np.minimum(np.asarray(cap, dtype=np.int64), max_rows)
    tiles = -(-capb // TILE)
    # Per unit: pieces j = 0 .. np-1 in row order tile the unit's rows.
    slots = []
    for u in range(units):
        mine = live[live[:, 0] == u]
        assert len(mine) >= 1, f"unit {u} has no piece"
        mine = mine[np.argsort(mine[:, 1])]
        npc = int(mine[0, 2])
        assert list(mine[:, 1]) == list(range(npc)) and np.all(mine[:, 2] == npc)
        assert np.all(mine[:, 3] == mine[0, 3])
        slots.extend(int(mine[0, 3]) + j for j in range(npc))
        assert mine[0, 4] == 0 and mine[-1, 5] == capb[u]
        assert np.all(mine[1:, 4] == mine[:-1, 5]), f"unit {u}: pieces not contiguous"
        assert np.all(mine[:, 4] % TILE == 0)
        assert np.all(mine[:, 7] == off[u])
        # The early-read bound: within the piece, and at the hint plus 64
        # rows (or the piece's end without a hint).
        want = mine[:, 5] if hint is None else np.clip(hint[u] + 64, mine[:, 4], mine[:, 5])
        assert np.all(mine[:, 6] == want), f"unit {u}: early bound {mine[:, 6]} != {want}"
    assert sorted(slots) == list(range(P)), "partial slots are not 0 .. P-1 once each"
    # Longest first.
    ptiles = -(-(live[:, 5] - live[:, 4]) // TILE)
    assert np.all(np.diff(ptiles) <= 0)
    # The per-wave share: a piece of n tiles gives its waves ceil(n / 4); the
    # largest over pieces is the smallest (at least 2) for which splitting
    # every unit into ceil(tiles / 4m) pieces fits the grid, unless no unit
    # is to be cut (below).
    share = int(max(1, (-(-ptiles // 4)).max()))

    def pieces(m):
        return int(np.maximum(1, -(-tiles // (4 * m))).sum())

    m = 2
    while pieces(m) > nwg:
        m += 1
    # More units than the 512 resident slots, and the units past the first
    # round at most a quarter of the longest: no unit is cut.
    ts = np.sort(tiles)[::-1]
    if units > 512 and 4 * ts[512] <= ts[0]:
        assert P == units, f"{P} pieces for {units} units where none should be cut"
    else:
        assert share <= max(m, 1), f"share {share} above the smallest fitting bound {m}"
    return hdr, rec


def _caps_offs(caps):
    off = np.concatenate([[0], np.cumsum(caps)[:-1]]).astype(np.int64)
    return [int(c) for c in caps], [int(o) for o in off]


@pytest.mark.parametrize("case", ["tiny", "vllm7b", "longvideo", "vllm72b", "batched"])
def test_plan_on_pruned_workload_caches(sg, case):
    """Caches shaped like the pruned ones the decode bench builds: per
    (layer, sequence) the retained visual rows, the window and 128 generated
    rows."""
    w = sg.WORKLOADS[case]
    n = [int(x) for x in w.n_vis()]
    shape = vc.vc_decode_shape(w.B, w.L, w.Hq, w.Hkv, w.d)
    k = vc.viscache_budget(vc.make_shape(w.B, w.L, w.Hq, w.Hkv, w.d, w.W, n), vc.make_params(w.retention))[0]
    caps = []
    for l in range(w.L):
        for b in range(w.B):
            for g in range(w.Hkv):
                caps.append(int(k[b * w.L + l]) + w.W + 128)
    cap, off = _caps_offs(caps)
    _check(shape, cap, off, max(cap))
    _check(shape, cap, off, max(cap), [c - 128 for c in cap])


def test_plan_edges():
    shape = vc.vc_decode_shape(2, 2, 8, 4, 128)
    rng = np.random.default_rng(3)
    for trial in range(40):
        caps = rng.integers(0, 3000, size=16)
        caps[rng.integers(0, 16, size=4)] = 0
        if trial % 3 == 0:
            caps[5] = 100000
        cap, off = _caps_offs(caps)
        hint = [int(x) for x in rng.integers(0, 3100, size=16)]
        for max_rows in (max(cap), 0, 1, 33, 4096):
            _check(shape, cap, off, max_rows)
            _check(shape, cap, off, max_rows, hint)
    # A single huge unit (many pieces), and all units empty.
    _check(vc.vc_decode_shape(1, 1, 8, 1, 64), [200000], [0], 200000)
    _check(shape, [0] * 16, [0] * 16, 0)
    # Offsets need not follow unit order; zero-capacity units may share one.
    cap = [64, 0, 32, 0] * 4
    off = [1000 - 64 * i for i in range(16)]
    off = [int(x) for x in np.argsort(off) * 100]
    _check(shape, cap, off, 64)


def test_plan_more_units_than_slots():
    """Past 512 units (the resident slots) no unit is cut when the units past
    the first round are at most a quarter of the longest; else the usual cut."""
    shape = vc.vc_decode_shape(1, 75, 8, 8, 128)  # 600 units
    caps = [2048] * 500 + [128] * 100
    cap, off = _caps_offs(caps)
    hdr, rec = _check(shape, cap, off, max(cap))
    assert int(hdr[5]) == 600
    caps = [2048] * 600
    cap, off = _caps_offs(caps)
    hdr, rec = _check(shape, cap, off, max(cap))
    assert int(hdr[5]) > 600


def test_plan_refusals():
    shape = vc.vc_decode_shape(1, 2, 8, 2, 64)
    cap, off = [10, 10, 10, 10], [0, 10, 20, 30]
    with pytest.raises(vc.VisCacheError) as e:
        vc.viscache_decode_plan(shape, cap, [0, 9, 20, 30], 10)  # overlapping blocks
    assert e.value.status == vc.VC_ERR_ARG
    with pytest.raises(vc.VisCacheError) as e:
        vc.viscache_decode_plan(shape, [10, -1, 10, 10], off, 10)
    assert e.value.status == vc.VC_ERR_ARG
    with pytest.raises(vc.VisCacheError) as e:
        vc.viscache_decode_plan(shape, cap, [0, 10, -20, 30], 10)
    assert e.value.status == vc.VC_ERR_ARG
    with pytest.raises(vc.VisCacheError) as e:
        vc.viscache_decode_plan(shape, cap, off, 10, [3, -1, 0, 0])  # negative length
    assert e.value.status == vc.VC_ERR_ARG
    with pytest.raises(vc.VisCacheError) as e:
        vc.viscache_decode_plan(shape, [2**31 - 64, 1, 1, 1], [0, 2**31, 2**31 + 1, 2**31 + 2], 2**31 - 64)
    assert e.value.status == vc.VC_ERR_UNSUPPORTED
    with pytest.raises(vc.VisCacheError) as e:
        vc.viscache_decode_plan(vc.vc_decode_shape(1, 2, 40, 2, 64), cap, off, 10)  # group of 20 heads
    assert e.value.status == vc.VC_ERR_UNSUPPORTED
    assert vc.viscache_decode_plan_bytes(shape, -1) == 0
    # Too small a buffer, through the C ABI directly.
    import ctypes
    n = vc.viscache_decode_plan_bytes(shape, 10)
    buf = (ctypes.c_int32 * (n // 4))()
    ca = (ctypes.c_int32 * 4)(*cap)
    oa = (ctypes.c_int64 * 4)(*off)
    L = vc.lib()
    assert (L.viscache_decode_plan(ctypes.byref(shape), ca, oa, None, 10, ctypes.addressof(buf), n - 4)
            == vc.VC_ERR_WORKSPACE)
    assert L.viscache_decode_plan(ctypes.byref(shape), ca, oa, None, 10, None, n) == vc.VC_ERR_ARG
    assert L.viscache_decode_plan(ctypes.byref(shape), ca, oa, None, 10, ctypes.addressof(buf), n) == vc.VC_OK
