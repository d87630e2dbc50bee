"""GPU parity of viscache_prune against the oracle, through the C ABI.

Small workloads and the 7B shape are compared unit by unit in full; the
long-video, 72B and batched workloads at full size are in
test_gpu_fullsize.py."""
import json
import os

import numpy as np
import pytest

from tests.parity import SCORE_TOL, SHARED_TOL, TOL_BF16, TOL_FP32, check_sets, fused_error, rel_err, score_err

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2608_24063_amd as vc
    vc.lib()
    return torch.device("cuda:0")


def _diag(rec):
    d = os.environ.get("VC_DIAG_DIR")
    if d:
        os.makedirs(d, exist_ok=True)
        with open(os.path.join(d, "parity_diag.jsonl"), "a") as f:
            f.write(json.dumps(rec) + "\n")


class Run:
    """One viscache_prune call on a seeded workload, with host copies."""

    def __init__(self, w, dev, mode=0, vfp32=False, rr=None, h=0, m=0.75, tau=1.0, mu=0.7, schedule=0,
                 drop_all=False, prefill=False):
        import paper_2608_24063_amd as vc
        from paper_2608_24063_amd.tensors import PruneCall
        from synthgen.device import to_host_bf16, upload_layers
        self.w, self.mode, self.vfp32, self.tau, self.mu = w, mode, vfp32, tau, mu
        self.prefill = prefill
        self.params = vc.make_params(rr if rr is not None else w.retention, h=h, m=m, tau=tau, mu=mu,
                                     rank_mode=mode, v_out_fp32=vfp32, schedule=schedule, drop_all=drop_all,
                                     score_queries=vc.VC_SCORE_PREFILL if prefill else vc.VC_SCORE_WINDOW)
        self.n = [int(x) for x in w.n_vis()]
        self.toff = np.concatenate([[0], np.cumsum(self.n)]).astype(np.int64)
        shape = vc.make_shape(w.B, w.L, w.Hq, w.Hkv, w.d, w.W, self.n)
        _, _, self.h = vc.viscache_budget(shape, self.params)
        self.Ls = w.L if mode == vc.VC_RANK_GLOBAL else self.h
        dev_t, self.host = upload_layers(w, range(self.Ls), dev, keep_host=True, prefill=prefill)
        pc = PruneCall(w.B, w.L, w.Hq, w.Hkv, w.d, w.W, self.n, self.params,
                       [dev_t["K"].get(l) for l in range(w.L)], [dev_t["V"].get(l) for l in range(w.L)],
                       [dev_t["Q"].get(l) for l in range(w.L)], with_drop=True,
                       k_text=[dev_t["KT"].get(l) for l in range(w.L)] if prefill else None)
        pc.run()
        torch.cuda.synchronize()
        self.pc = pc
        self.k, self.ns = pc.k, pc.n_surv
        self.idx = [t.cpu().numpy() for t in pc.idx_out]
        self.drop = [t.cpu().numpy() for t in pc.drop_out]
        self.kout = [to_host_bf16(t) for t in pc.k_out]
        self.vout = [t.float().cpu().numpy() for t in pc.v_out]
        s_off, g_off = vc.viscache_prune_score_offsets(shape, self.params)
        ntot = int(self.toff[-1])
        nS = self.Ls * ntot * w.Hkv
        self.S = pc.ws[s_off:s_off + 4 * nS].view(torch.float32).cpu().numpy().reshape(self.Ls, -1)
        self.gs = pc.ws[g_off:g_off + 4 * ntot].view(torch.float32).cpu().numpy() if g_off is not None else None
        del dev_t

    # host views of one unit
    def unit_kv(self, role, l, b, g):
        n = self.n[b]
        r0 = int(self.toff[b]) * self.w.Hkv + g * n
        return self.host[role][l][r0:r0 + n]

    def unit_q(self, l, b, g):
        """Window: the G*W window queries [G*W, d]; prefill: every token's
        query of the group's heads [G, n_b + W, d]."""
        G, W, d = self.w.G, self.w.W, self.w.d
        if not self.prefill:
            return self.host["Q"][l][b, g * G:(g + 1) * G].reshape(-1, d)
        N = self.n[b] + W
        r0 = (int(self.toff[b]) + b * W) * self.w.Hq + g * G * N
        return self.host["Q"][l][r0:r0 + G * N].reshape(G, N, d)

    def ref_scores(self, orc, l, b, g):
        """The oracle's scores of one unit (fp64)."""
        K = self.unit_kv("K", l, b, g)
        if not self.prefill:
            return orc.scores_unit(K, self.unit_q(l, b, g))
        return orc.scores_unit_prefill(K, self.host["KT"][l][b, g], self.unit_q(l, b, g))

    def gpu_scores(self, l, b, g):
        n = self.n[b]
        r0 = int(self.toff[b]) * self.w.Hkv + g * n
        return self.S[l][r0:r0 + n]

    def gpu_unit(self, l, b, g):
        r0, r1 = self.pc.unit_rows(l, b, g)
        d0, d1 = self.pc.unit_drop_rows(l, b, g)
        return self.idx[l][r0:r1], self.drop[l][d0:d1], self.kout[l][r0:r1], self.vout[l][r0:r1]

    def check_unit(self, orc, l, b, g, S32=None):
        """Full comparison of one unit; S32 = the oracle's ranking scores
        (computed here for the layer/head ranking)."""
        K, V = self.unit_kv("K", l, b, g), self.unit_kv("V", l, b, g)
        k, ns = self.k[b * self.w.L + l], self.ns[b * self.w.L + l]
        if S32 is None:
            S32 = self.ref_scores(orc, l, b, g).astype(np.float32)
        kept, drop, krows, vrows = self.gpu_unit(l, b, g)
        swaps = check_sets(S32, k, ns, kept, drop, what=f"{self.w.name} l={l} b={b} g={g}")
        np.testing.assert_array_equal(krows, K[kept])  # kept keys are bit copies
        ref = orc.fuse(V, kept.astype(np.int32), drop.astype(np.int32), self.tau, self.mu)
        ferr = fused_error(ref, vrows)
        tol = TOL_FP32 if self.vfp32 else TOL_BF16
        assert ferr <= tol, f"fused V error {ferr} > {tol} at l={l} b={b} g={g}"
        return swaps, ferr

    def check_all_layer_head(self, orc, units):
        def one(u):
            return self.ref_scores(orc, *u).astype(np.float32)
        refs = orc.run_units(one, units)
        swaps, ferr, serr = 0, 0.0, 0.0
        for (l, b, g), S32 in zip(units, refs):
            s, f = self.check_unit(orc, l, b, g, S32)
            swaps += s
            ferr = max(ferr, f)
            got = self.gpu_scores(l, b, g)
            # prefill scores sum G (n + W) rows per key: checked at 1e-4
            serr = max(serr, rel_err(S32, got, floor=1e-30) if self.prefill else score_err(S32, got))
        _diag(dict(workload=self.w.name, mode=self.mode, vfp32=self.vfp32, prefill=self.prefill, units=len(units),
                   swaps=swaps, fused_err=ferr, score_rel_err=serr))
        return swaps, ferr, serr


def _all_units(r):
    return [(l, b, g) for l in range(r.h) for b in range(r.w.B) for g in range(r.w.Hkv)]


# ---------------------------------------------------------------- tiny, full
@pytest.mark.parametrize("vfp32", [False, True])
def test_tiny_layer_head_full(dev, orc, sg, vfp32):
    r = Run(sg.TINY, dev, vfp32=vfp32)
    swaps, ferr, serr = r.check_all_layer_head(orc, _all_units(r))
    assert serr < SCORE_TOL


@pytest.mark.parametrize("vfp32", [False, True])
def test_tiny_global_full(dev, orc, sg, vfp32):
    r = Run(sg.TINY, dev, mode=1, vfp32=vfp32)
    w = r.w
    for b in range(w.B):
        units = [(l, b, g) for l in range(w.L) for g in range(w.Hkv)]
        S = orc.run_units(lambda u: orc.scores_unit(r.unit_kv("K", *u), r.unit_q(*u)), units)
        s32 = orc.global_scores(S)
        n = r.n[b]
        gs = r.gs[r.toff[b]:r.toff[b] + n]
        assert score_err(s32, gs) < SHARED_TOL
        for l in range(r.h):
            for g in range(w.Hkv):
                r.check_unit(orc, l, b, g, S32=s32)
        # one shared ranking: deeper layers keep subsets of shallower ones
        for l in range(1, r.h):
            k0, _, _, _ = r.gpu_unit(l - 1, b, 0)
            k1, _, _, _ = r.gpu_unit(l, b, 0)
            assert set(k1.tolist()) <= set(k0.tolist())


# ------------------------------------------------------------ edge cases
def _custom(sg, **kw):
    base = dict(name="edge", seed=0x5EED00E1, B=1, L=4, Hq=8, Hkv=2, d=64, W=32, tokens_per_frame=64,
                frames=8, retention=0.25)
    base.update(kw)
    return sg.Workload(**base)


@pytest.mark.parametrize("d", [64, 128])
def test_ragged_small_batch(dev, orc, sg, d):
    # jittered frame counts with tiny frames give ragged sequences, one of
    # them below a tile; G = 3 and W = 5 make ragged query rows.
    w = _custom(sg, B=5, Hq=6, Hkv=2, d=d, W=5, tokens_per_frame=7, frames=12, frame_jitter=11)
    for vfp32 in (False, True):
        r = Run(w, dev, vfp32=vfp32)
        r.check_all_layer_head(orc, _all_units(r))


def test_empty_sequence_in_batch(dev, orc, sg):
    import paper_2608_24063_amd as vc
    from paper_2608_24063_amd.tensors import PruneCall
    from synthgen.device import bf16_tensor
    w = _custom(sg, B=1)
    n = [0, 130, 0, 64]
    rng = np.random.default_rng(0)
    rows = sum(n) * w.Hkv
    K = [rng.integers(0, 2 ** 15, (rows, w.d), dtype=np.uint16) & 0x3FFF for _ in range(w.L)]
    V = [rng.integers(0, 2 ** 15, (rows, w.d), dtype=np.uint16) & 0x3FFF for _ in range(w.L)]
    Q = [rng.standard_normal((4, w.Hq, w.W, w.d)).astype(np.float32) for _ in range(w.L)]
    params = vc.make_params(0.25)
    pc = PruneCall(4, w.L, w.Hq, w.Hkv, w.d, w.W, n, params, [bf16_tensor(x, dev) for x in K],
                   [bf16_tensor(x, dev) for x in V], [torch.from_numpy(q).to(dev) for q in Q], with_drop=True)
    pc.run()
    torch.cuda.synchronize()
    toff = np.concatenate([[0], np.cumsum(n)])
    for l in range(pc.h):
        for b in range(4):
            for g in range(w.Hkv):
                nb = n[b]
                r0 = toff[b] * w.Hkv + g * nb
                Ku, Vu = K[l][r0:r0 + nb], V[l][r0:r0 + nb]
                Qu = Q[l][b, g * w.G:(g + 1) * w.G].reshape(-1, w.d)
                k, ns = pc.k[b * w.L + l], pc.n_surv[b * w.L + l]
                a0, a1 = pc.unit_rows(l, b, g)
                d0, d1 = pc.unit_drop_rows(l, b, g)
                kept = pc.idx_out[l][a0:a1].cpu().numpy()
                drop = pc.drop_out[l][d0:d1].cpu().numpy()
                if nb == 0:
                    assert k == 0 and len(kept) == 0
                    continue
                S32 = orc.scores_unit(Ku, Qu).astype(np.float32)
                check_sets(S32, k, ns, kept, drop)
                ref = orc.fuse(Vu, kept.astype(np.int32), drop.astype(np.int32))
                got = pc.v_out[l][a0:a1].float().cpu().numpy()
                assert fused_error(ref, got) <= TOL_BF16


def test_keep_all_returns_cache_unchanged(dev, orc, sg):
    # RR = 1, h = L, m = 1: every layer keeps every token, nothing is fused.
    w = _custom(sg, L=3)
    for vfp32 in (False, True):
        r = Run(w, dev, rr=1.0, h=3, m=1.0, vfp32=vfp32)
        for l in range(w.L):
            for g in range(w.Hkv):
                kept, drop, krows, vrows = r.gpu_unit(l, 0, g)
                n = r.n[0]
                np.testing.assert_array_equal(kept, np.arange(n))
                assert len(drop) == 0
                np.testing.assert_array_equal(krows, r.unit_kv("K", l, 0, g))
                V = r.unit_kv("V", l, 0, g)
                np.testing.assert_array_equal(vrows, sg.bf16_bits_to_f32(V))


def test_mu_one_is_plain_pruning(dev, orc, sg):
    w = _custom(sg)
    r = Run(w, dev, mu=1.0, vfp32=True)
    for (l, b, g) in _all_units(r):
        kept, drop, krows, vrows = r.gpu_unit(l, b, g)
        np.testing.assert_array_equal(vrows, sg.bf16_bits_to_f32(r.unit_kv("V", l, b, g)[kept]))


@pytest.mark.parametrize("tau", [0.05, 50.0])
def test_temperature(dev, orc, sg, tau):
    w = _custom(sg, seed=0x5EED00E2)
    r = Run(w, dev, tau=tau, vfp32=True)
    r.check_all_layer_head(orc, _all_units(r))


def test_identical_keys_tie_to_lowest_index(dev, orc, sg):
    import paper_2608_24063_amd as vc
    from paper_2608_24063_amd.tensors import PruneCall
    from synthgen.device import bf16_tensor
    L, Hq, Hkv, d, W, n = 4, 8, 2, 64, 8, 300
    rng = np.random.default_rng(1)
    row = rng.integers(0, 2 ** 14, (1, d), dtype=np.uint16)
    K = [np.repeat(row, Hkv * n, 0) for _ in range(L)]
    V = [rng.integers(0, 2 ** 14, (Hkv * n, d), dtype=np.uint16) for _ in range(L)]
    Q = [rng.standard_normal((1, Hq, W, d)).astype(np.float32) for _ in range(L)]
    params = vc.make_params(0.25)
    pc = PruneCall(1, L, Hq, Hkv, d, W, [n], params, [bf16_tensor(x, dev) for x in K],
                   [bf16_tensor(x, dev) for x in V], [torch.from_numpy(q).to(dev) for q in Q], with_drop=True)
    pc.run()
    torch.cuda.synchronize()
    for l in range(pc.h):
        for g in range(Hkv):
            a0, a1 = pc.unit_rows(l, 0, g)
            d0, d1 = pc.unit_drop_rows(l, 0, g)
            k, ns = pc.k[l], pc.n_surv[l]
            np.testing.assert_array_equal(pc.idx_out[l][a0:a1].cpu().numpy(), np.arange(k))
            np.testing.assert_array_equal(pc.drop_out[l][d0:d1].cpu().numpy(), np.arange(k, ns))


def test_repeat_is_bitwise_deterministic(dev, sg):
    w = _custom(sg)
    a = Run(w, dev)
    b = Run(w, dev)
    for l in range(a.h):
        np.testing.assert_array_equal(a.idx[l], b.idx[l])
        np.testing.assert_array_equal(a.vout[l], b.vout[l])
    np.testing.assert_array_equal(a.S, b.S)


# ----------------------------------------------------------- 7B-shaped, full
@pytest.fixture(scope="module")
def run7b(dev, sg):
    return Run(sg.VLLM7B, dev)


# ------------------------------------- budget ablation schedules, fuse-all
def _budgets_match_oracle(r, orc, schedule=0, drop_all=False):
    for b, nb in enumerate(r.n):
        ref = orc.budget(L=r.w.L, n=nb, rr=r.w.retention, schedule=schedule, drop_all=drop_all)
        assert list(r.k[b * r.w.L:(b + 1) * r.w.L]) == list(ref["k"])
        assert r.ns[b * r.w.L] == ref["n_surv"]


@pytest.mark.parametrize("schedule", [1, 2, 3])
def test_tiny_alternative_schedules_full(dev, orc, sg, schedule):
    """Fixed, arithmetic and geometric budgets (the budget ablation) through
    the whole path, every unit against the oracle."""
    r = Run(sg.TINY, dev, schedule=schedule, vfp32=True)
    _budgets_match_oracle(r, orc, schedule=schedule)
    swaps, ferr, serr = r.check_all_layer_head(orc, _all_units(r))
    assert serr < SCORE_TOL


@pytest.mark.parametrize("vfp32", [False, True])
def test_tiny_fuse_all_full(dev, orc, sg, vfp32):
    """Every non-kept token fused (n_surv = n), every unit."""
    r = Run(sg.TINY, dev, drop_all=True, vfp32=vfp32)
    _budgets_match_oracle(r, orc, drop_all=True)
    assert all(x == n for b, n in enumerate(r.n) for x in r.ns[b * r.w.L:(b + 1) * r.w.L])
    r.check_all_layer_head(orc, _all_units(r))


def test_vllm7b_fuse_all_sampled(dev, orc, sg):
    """7B shape with every non-kept token fused: dropped lists of up to
    n - k_h = 2430 rows per unit (38 tiles)."""
    r = Run(sg.VLLM7B, dev, drop_all=True, vfp32=True)
    _budgets_match_oracle(r, orc, drop_all=True)
    r.check_all_layer_head(orc, [(0, 0, 0), (10, 0, 1), (r.h - 1, 0, 3)])


def test_vllm7b_layer_head_full(run7b, orc):
    swaps, ferr, serr = run7b.check_all_layer_head(orc, _all_units(run7b))
    assert serr < SCORE_TOL


def test_vllm7b_fp32_out(dev, orc, sg):
    r = Run(sg.VLLM7B, dev, vfp32=True)
    units = [(0, 0, 0), (10, 0, 1), (r.h - 1, 0, 3)]
    r.check_all_layer_head(orc, units)


def test_vllm7b_global_full(dev, orc, sg):
    r = Run(sg.VLLM7B, dev, mode=1)
    w = r.w
    units = [(l, 0, g) for l in range(w.L) for g in range(w.Hkv)]
    S = orc.run_units(lambda u: orc.scores_unit(r.unit_kv("K", *u), r.unit_q(*u)), units)
    s32 = orc.global_scores(S)
    assert score_err(s32, r.gs) < SHARED_TOL
    swaps = 0
    for l in range(r.h):
        for g in range(w.Hkv):
            s, _ = r.check_unit(orc, l, 0, g, S32=s32)
            swaps += s
    _diag(dict(workload=w.name, mode=1, swaps=swaps))


# ----------------------- prefill scores: every prefill token queries, causally
@pytest.mark.parametrize("vfp32", [False, True])
def test_tiny_prefill_layer_head_full(dev, orc, sg, vfp32):
    """n = 512, W = 32, G = 4: 2176 query rows per unit (nine row groups, the
    first two inside one head), two 256-key column chunks."""
    r = Run(sg.TINY, dev, vfp32=vfp32, prefill=True)
    swaps, ferr, serr = r.check_all_layer_head(orc, _all_units(r))
    assert serr < 1e-4


def test_tiny_prefill_global_full(dev, orc, sg):
    r = Run(sg.TINY, dev, mode=1, prefill=True)
    w = r.w
    units = [(l, 0, g) for l in range(w.L) for g in range(w.Hkv)]
    s32 = orc.global_scores(orc.run_units(lambda u: r.ref_scores(orc, *u), units))
    assert rel_err(s32, r.gs, floor=1e-30) < 1e-4
    for l in range(r.h):
        for g in range(w.Hkv):
            r.check_unit(orc, l, 0, g, S32=s32)


@pytest.mark.parametrize("d", [64, 128])
def test_prefill_ragged_small_batch(dev, orc, sg, d):
    # Ragged sequences (one below a tile), G = 3 and W = 5: row groups that
    # straddle heads and end mid-tile, key tiles that end inside the text.
    w = _custom(sg, B=5, Hq=6, Hkv=2, d=d, W=5, tokens_per_frame=7, frames=12, frame_jitter=11)
    r = Run(w, dev, vfp32=True, prefill=True)
    r.check_all_layer_head(orc, _all_units(r))


def test_prefill_multi_chunk_ragged(dev, orc, sg):
    # n = 700 (three column chunks, the last 188 keys), G = 2, W = 3.
    w = _custom(sg, B=2, Hq=4, Hkv=2, d=128, W=3, tokens_per_frame=70, frames=10)
    r = Run(w, dev, prefill=True)
    swaps, ferr, serr = r.check_all_layer_head(orc, _all_units(r))
    assert serr < 1e-4


def _prefill_direct(dev, n, L, Hq, Hkv, d, W, K, V, Kt, Q, rr=0.25):
    import paper_2608_24063_amd as vc
    from paper_2608_24063_amd.tensors import PruneCall
    from synthgen.device import bf16_tensor
    params = vc.make_params(rr, score_queries=vc.VC_SCORE_PREFILL)
    pc = PruneCall(len(n), L, Hq, Hkv, d, W, n, params, [bf16_tensor(x, dev) for x in K],
                   [bf16_tensor(x, dev) for x in V], [torch.from_numpy(q).to(dev) for q in Q], with_drop=True,
                   k_text=[bf16_tensor(x, dev) for x in Kt])
    pc.run()
    torch.cuda.synchronize()
    shape = vc.make_shape(len(n), L, Hq, Hkv, d, W, n)
    s_off, _ = vc.viscache_prune_score_offsets(shape, params)
    ntot = sum(n)
    S = pc.ws[s_off:s_off + 4 * pc.h * ntot * Hkv].view(torch.float32).cpu().numpy().reshape(pc.h, -1)
    return pc, S


def test_prefill_empty_sequences_in_batch(dev, orc):
    """Sequences with no visual token: their text rows are still queries but
    there is nothing to score or keep."""
    L, Hq, Hkv, d, W = 4, 8, 2, 64, 6
    G = Hq // Hkv
    n = [0, 300, 0, 65]
    rng = np.random.default_rng(4)
    rows = sum(n) * Hkv
    K = [rng.integers(0, 2 ** 15, (rows, d), dtype=np.uint16) & 0x3FFF for _ in range(L)]
    V = [rng.integers(0, 2 ** 15, (rows, d), dtype=np.uint16) & 0x3FFF for _ in range(L)]
    Kt = [rng.integers(0, 2 ** 15, (len(n), Hkv, W, d), dtype=np.uint16) & 0x3FFF for _ in range(L)]
    Q = [rng.standard_normal((sum(n) * Hq + len(n) * W * Hq, d)).astype(np.float32) for _ in range(L)]
    pc, S = _prefill_direct(dev, n, L, Hq, Hkv, d, W, K, V, Kt, Q)
    toff = np.concatenate([[0], np.cumsum(n)])
    for l in range(pc.h):
        for b in range(len(n)):
            for g in range(Hkv):
                nb, N = n[b], n[b] + W
                a0, a1 = pc.unit_rows(l, b, g)
                d0, d1 = pc.unit_drop_rows(l, b, g)
                kept = pc.idx_out[l][a0:a1].cpu().numpy()
                drop = pc.drop_out[l][d0:d1].cpu().numpy()
                if nb == 0:
                    assert pc.k[b * L + l] == 0 and len(kept) == 0
                    continue
                r0 = toff[b] * Hkv + g * nb
                q0 = (toff[b] + b * W) * Hq + g * G * N
                ref = orc.scores_unit_prefill(K[l][r0:r0 + nb], Kt[l][b, g], Q[l][q0:q0 + G * N].reshape(G, N, d))
                assert rel_err(ref, S[l][r0:r0 + nb], floor=1e-30) < 1e-4
                check_sets(ref.astype(np.float32), pc.k[b * L + l], pc.n_surv[b * L + l], kept, drop)
                fref = orc.fuse(V[l][r0:r0 + nb], kept.astype(np.int32), drop.astype(np.int32))
                assert fused_error(fref, pc.v_out[l][a0:a1].float().cpu().numpy()) <= TOL_BF16


def test_prefill_identical_keys_harmonic(dev):
    """All keys of a unit equal (text keys too): query i spreads 1/(i+1) over
    its prefix, so visual key v scores G (H_N - H_v), strictly decreasing in v,
    and the kept set is the first k tokens, the dropped set the next ones."""
    L, Hq, Hkv, d, W, n = 4, 8, 2, 128, 40, 777
    G, N = Hq // Hkv, n + W
    rng = np.random.default_rng(6)
    row = rng.integers(0, 2 ** 14, (1, d), dtype=np.uint16)
    K = [np.repeat(row, Hkv * n, 0) for _ in range(L)]
    Kt = [np.repeat(row, Hkv * W, 0).reshape(1, Hkv, W, d) for _ in range(L)]
    V = [rng.integers(0, 2 ** 14, (Hkv * n, d), dtype=np.uint16) for _ in range(L)]
    Q = [rng.standard_normal((Hq * N, d)).astype(np.float32) for _ in range(L)]
    pc, S = _prefill_direct(dev, [n], L, Hq, Hkv, d, W, K, V, Kt, Q)
    H = np.concatenate([[0.0], np.cumsum(1.0 / np.arange(1, N + 1))])
    ref = G * (H[N] - H[:n])
    for l in range(pc.h):
        for g in range(Hkv):
            assert rel_err(ref, S[l][g * n:(g + 1) * n]) < 1e-5
            a0, a1 = pc.unit_rows(l, 0, g)
            d0, d1 = pc.unit_drop_rows(l, 0, g)
            k, ns = pc.k[l], pc.n_surv[l]
            np.testing.assert_array_equal(pc.idx_out[l][a0:a1].cpu().numpy(), np.arange(k))
            np.testing.assert_array_equal(pc.drop_out[l][d0:d1].cpu().numpy(), np.arange(k, ns))


def test_vllm7b_prefill_sampled(dev, orc, sg):
    """7B shape, every prefill token queries (22400 rows per unit): sampled
    units against the oracle, and every unit's kept set the exact top-k of the
    GPU's own scores."""
    r = Run(sg.VLLM7B, dev, prefill=True)
    swaps, ferr, serr = r.check_all_layer_head(orc, [(0, 0, 0), (r.h // 2, 0, 1), (r.h - 1, 0, 3)])
    assert serr < 1e-4
    w = r.w
    for l in range(r.h):
        for g in range(w.Hkv):
            kept, drop, _, _ = r.gpu_unit(l, 0, g)
            assert check_sets(r.gpu_scores(l, 0, g), r.k[l], r.ns[l], kept, drop) == 0
            # causal rows are distributions: the visual mass is at most G(n+W) rows' worth
            assert 0 < r.gpu_scores(l, 0, g).sum() <= w.G * (r.n[0] + w.W) * (1 + 1e-5)


# ---------------------------------------------------------------- limits
def test_max_sizes_window(dev, orc, sg):
    """The largest unit the window path takes: n = 32768 visual tokens (the
    selection's register capacity) and G*W = 1024 window rows (the statistics
    pass's row limit), d = 128; both layers in full against the oracle."""
    import paper_2608_24063_amd as vc
    from paper_2608_24063_amd.tensors import PruneCall
    from synthgen.device import bf16_tensor
    L, Hq, Hkv, d, W, n = 2, 16, 1, 128, 64, 32768
    rng = np.random.default_rng(32768)
    K = [sg.normal_bf16(0x5EED0100, l, (n, d)) for l in range(L)]
    V = [sg.normal_bf16(0x5EED0101, l, (n, d)) for l in range(L)]
    Q = [rng.standard_normal((1, Hq, W, d)).astype(np.float32) for _ in range(L)]
    params = vc.make_params(0.25)
    pc = PruneCall(1, L, Hq, Hkv, d, W, [n], params, [bf16_tensor(x, dev) for x in K],
                   [bf16_tensor(x, dev) for x in V], [torch.from_numpy(q).to(dev) for q in Q], with_drop=True)
    pc.run()
    torch.cuda.synchronize()
    assert pc.h == 2 and pc.n_surv[1] > pc.k[1] > 0
    refs = orc.run_units(lambda l: orc.scores_unit(K[l], Q[l][0].reshape(-1, d)).astype(np.float32), range(L))
    for l in range(L):
        a0, a1 = pc.unit_rows(l, 0, 0)
        d0, d1 = pc.unit_drop_rows(l, 0, 0)
        kept = pc.idx_out[l][a0:a1].cpu().numpy()
        drop = pc.drop_out[l][d0:d1].cpu().numpy()
        check_sets(refs[l], pc.k[l], pc.n_surv[l], kept, drop, what=f"max l={l}")
        fref = orc.fuse(V[l], kept.astype(np.int32), drop.astype(np.int32))
        assert fused_error(fref, pc.v_out[l][a0:a1].float().cpu().numpy()) <= TOL_BF16


def test_max_sizes_prefill_identical_keys(dev):
    """Prefill scores at n = 32768 visual tokens (65 664 query rows per unit,
    257 row groups): with all keys equal the scores have the closed form
    G (H_N - H_v) at any size, and the kept and dropped sets are prefixes."""
    L, Hq, Hkv, d, W, n = 2, 2, 1, 64, 64, 32768
    G, N = Hq // Hkv, n + W
    rng = np.random.default_rng(7)
    row = rng.integers(0, 2 ** 14, (1, d), dtype=np.uint16)
    K = [np.repeat(row, n, 0) for _ in range(L)]
    Kt = [np.repeat(row, W, 0).reshape(1, 1, W, d) for _ in range(L)]
    V = [rng.integers(0, 2 ** 14, (n, d), dtype=np.uint16) for _ in range(L)]
    Q = [rng.standard_normal((Hq * N, d)).astype(np.float32) for _ in range(L)]
    pc, S = _prefill_direct(dev, [n], L, Hq, Hkv, d, W, K, V, Kt, Q)
    H = np.concatenate([[0.0], np.cumsum(1.0 / np.arange(1, N + 1))])
    ref = G * (H[N] - H[:n])
    for l in range(pc.h):
        assert rel_err(ref, S[l][:n]) < 1e-4
        a0, a1 = pc.unit_rows(l, 0, 0)
        d0, d1 = pc.unit_drop_rows(l, 0, 0)
        np.testing.assert_array_equal(pc.idx_out[l][a0:a1].cpu().numpy(), np.arange(pc.k[l]))
        np.testing.assert_array_equal(pc.drop_out[l][d0:d1].cpu().numpy(), np.arange(pc.k[l], pc.n_surv[l]))


# ---------------------------------------------------------- graph capture
def test_graph_capture_replays(dev, orc, sg):
    """A captured viscache_prune replays to the eager result every time, with
    eager work and overwritten outputs between the replays."""
    w = _custom(sg, L=8, frame_jitter=0)
    r = Run(w, dev)
    pc = r.pc
    ref = [t.clone() for t in pc.v_out] + [t.clone() for t in pc.idx_out]
    outs = pc.v_out + pc.idx_out
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            pc.run()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    for rep in range(4):
        for t in outs:
            t.fill_(7)
        x = torch.randn(1 << 20, device=dev).sum()  # eager work between replays
        g.replay()
        torch.cuda.synchronize()
        for a, b in zip(ref, outs):
            assert torch.equal(a, b), f"replay {rep}"
        del x
