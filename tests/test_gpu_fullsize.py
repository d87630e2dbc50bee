"""Full-size parity: every (layer, sequence, kv head) unit of the long-video,
72B-shaped and batched workloads against the oracle, in both rankings, in the
launch configuration the benchmark times.

The oracle scores every unit of all L layers once per workload (fp64, one unit
per thread); both rankings are checked against them:
  - per-unit window scores (layer/head ranking) and the shared score (global
    ranking) against the oracle's, element by element;
  - kept and dropped sets of every unit against the oracle's ranking (the
    1e-5 boundary band of the contract);
  - every kept key row bit for bit;
  - fused values of every unit on sampled kept rows (each kept row's fused
    value depends only on that row and the unit's dropped set, so the oracle
    re-fuses exactly those rows on the GPU's sets); on long video, every row
    in fp32 output mode.
"""
import json
import os

import numpy as np
import pytest

from tests.parity import SCORE_TOL, SCORE_TOL_CUT, SHARED_TOL, TOL_BF16, TOL_FP32, check_sets, fused_error, score_err

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

FUSE_SAMPLE_ROWS = 16


def _diag(rec):
    d = os.environ.get("VC_DIAG_DIR")
    if d:
        os.makedirs(d, exist_ok=True)
        with open(os.path.join(d, "parity_diag.jsonl"), "a") as f:
            f.write(json.dumps(rec) + "\n")


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2608_24063_amd as vc
    vc.lib()
    return torch.device("cuda:0")


class FullSize:
    """One workload at full size: host and device copies of every layer and
    the oracle's fp64 scores of every unit of every layer."""

    def __init__(self, w, dev, orc):
        from synthgen.device import upload_layers
        self.w, self.dev = w, dev
        self.n = [int(x) for x in w.n_vis()]
        self.toff = np.concatenate([[0], np.cumsum(self.n)]).astype(np.int64)
        print(f"[fullsize] {w.name}: generating {w.L} layers, n = {self.n}", flush=True)
        self.dv, self.host = upload_layers(w, range(w.L), dev, keep_host=True)
        units = [(l, b, g) for l in range(w.L) for b in range(w.B) for g in range(w.Hkv)]
        print(f"[fullsize] {w.name}: oracle scores of {len(units)} units", flush=True)
        S = orc.run_units(lambda u: orc.scores_unit(self.unit_kv("K", *u), self.unit_q(*u)), units)
        self.S = dict(zip(units, S))
        # The shared ranking: per sequence, the fp64 sum over every layer and
        # kv head in (layer, head) order, rounded to fp32.
        self.gs = [orc.global_scores([self.S[(l, b, g)] for l in range(w.L) for g in range(w.Hkv)])
                   for b in range(w.B)]

    def unit_kv(self, role, l, b, g):
        n = self.n[b]
        r0 = int(self.toff[b]) * self.w.Hkv + g * n
        return self.host[role][l][r0:r0 + n]

    def unit_q(self, l, b, g):
        G, d = self.w.G, self.w.d
        return self.host["Q"][l][b, g * G:(g + 1) * G].reshape(-1, d)

    def run(self, mode, vfp32=False, drop_all=False):
        import paper_2608_24063_amd as vc
        from paper_2608_24063_amd.tensors import PruneCall
        w = self.w
        params = vc.make_params(w.retention, rank_mode=mode, v_out_fp32=vfp32, drop_all=drop_all)
        pc = PruneCall(w.B, w.L, w.Hq, w.Hkv, w.d, w.W, self.n, params, [self.dv["K"][l] for l in range(w.L)],
                       [self.dv["V"][l] for l in range(w.L)], [self.dv["Q"][l] for l in range(w.L)],
                       with_drop=True)
        print(f"[fullsize] {w.name}: prune mode={mode} vfp32={vfp32} drop_all={drop_all}", flush=True)
        pc.run()
        torch.cuda.synchronize()
        return Outputs(self, pc, mode)


class Outputs:
    """Host copies of one call's outputs and scores."""

    def __init__(self, fs, pc, mode):
        import paper_2608_24063_amd as vc
        from synthgen.device import to_host_bf16
        self.fs, self.pc, self.mode = fs, pc, mode
        w = fs.w
        self.k, self.ns, self.h = pc.k, pc.n_surv, pc.h
        self.idx = [t.cpu().numpy() for t in pc.idx_out]
        self.drop = [t.cpu().numpy() for t in pc.drop_out]
        self.kout = [to_host_bf16(t) for t in pc.k_out]
        self.vout = [t.float().cpu().numpy() for t in pc.v_out]
        s_off, g_off = vc.viscache_prune_score_offsets(pc.shape, pc.params)
        ntot = int(fs.toff[-1])
        Ls = w.L if mode == vc.VC_RANK_GLOBAL else pc.h
        self.S = pc.ws[s_off:s_off + 4 * Ls * ntot * w.Hkv].view(torch.float32).cpu().numpy().reshape(Ls, -1)
        self.gs = pc.ws[g_off:g_off + 4 * ntot].view(torch.float32).cpu().numpy() if g_off is not None else None
        del pc.ws, pc.k_out, pc.v_out, pc.idx_out, pc.drop_out

    def unit(self, l, b, g):
        r0, r1 = self.pc.unit_rows(l, b, g)
        d0, d1 = self.pc.unit_drop_rows(l, b, g)
        return self.idx[l][r0:r1], self.drop[l][d0:d1], self.kout[l][r0:r1], self.vout[l][r0:r1]

    def unit_scores(self, l, b, g):
        n = self.fs.n[b]
        r0 = int(self.fs.toff[b]) * self.fs.w.Hkv + g * n
        return self.S[l][r0:r0 + n]


def _sample_rows(k, m=FUSE_SAMPLE_ROWS):
    if k <= m:
        return np.arange(k)
    return np.unique(np.linspace(0, k - 1, m).round().astype(np.int64))


def check_unit(orc, fs, out, l, b, g, rank_scores, tol, all_rows=False, tau=1.0, mu=0.7):
    """Sets, kept keys and fused values of one unit against the oracle;
    returns (boundary swaps, fused-value error)."""
    w = fs.w
    k, ns = out.k[b * w.L + l], out.ns[b * w.L + l]
    kept, drop, krows, vrows = out.unit(l, b, g)
    swaps = check_sets(rank_scores, k, ns, kept, drop, what=f"{w.name} mode={out.mode} l={l} b={b} g={g}")
    K, V = fs.unit_kv("K", l, b, g), fs.unit_kv("V", l, b, g)
    np.testing.assert_array_equal(krows, K[kept], err_msg=f"kept keys l={l} b={b} g={g}")
    rows = np.arange(len(kept)) if all_rows else _sample_rows(len(kept))
    ref = orc.fuse(V, kept[rows].astype(np.int32), drop.astype(np.int32), tau, mu)
    ferr = fused_error(ref, vrows[rows])
    assert ferr <= tol, f"{w.name} mode={out.mode} fused V error {ferr} > {tol} at l={l} b={b} g={g}"
    return swaps, ferr


@pytest.fixture(scope="module")
def cache():
    """One FullSize at a time (the batched inputs alone take 8.5 GB of host
    and device memory), released when the module ends."""
    c = {}
    yield c
    c.clear()
    torch.cuda.empty_cache()


def _fullsize(c, name, dev, orc, sg):
    if name not in c:
        c.clear()
        torch.cuda.empty_cache()
        c[name] = FullSize(sg.WORKLOADS[name], dev, orc)
    return c[name]


def _layer_head(fs, orc, all_rows=False, vfp32=False, drop_all=False):
    w = fs.w
    out = fs.run(0, vfp32=vfp32, drop_all=drop_all)
    units = [(l, b, g) for l in range(out.h) for b in range(w.B) for g in range(w.Hkv)]
    tol = TOL_FP32 if vfp32 else TOL_BF16

    def one(u):
        ref = fs.S[u]
        l, b, g = u
        serr, scut = score_err(ref, out.unit_scores(*u), cut=out.ns[b * w.L + l])
        s, f = check_unit(orc, fs, out, *u, ref.astype(np.float32), tol, all_rows=all_rows)
        return serr, scut, s, f

    res = orc.run_units(one, units)
    serr = max(r[0] for r in res)
    scut = max(r[1] for r in res)
    rec = dict(workload=w.name, mode="layer_head", vfp32=vfp32, drop_all=drop_all, units=len(units),
               swaps=sum(r[2] for r in res), fused_err=max(r[3] for r in res), score_rel_err=serr,
               score_rel_err_cut=scut, all_rows=all_rows)
    print(f"[fullsize] {rec}", flush=True)
    _diag(rec)
    assert serr < SCORE_TOL, f"{w.name}: window score error {serr}"
    assert scut < SCORE_TOL_CUT, f"{w.name}: window score error near the cuts {scut}"
    return out


def _global(fs, orc):
    w = fs.w
    out = fs.run(1)
    gerr, gcut = 0.0, 0.0
    for b in range(w.B):
        e, c = score_err(fs.gs[b], out.gs[fs.toff[b]:fs.toff[b + 1]], cut=out.ns[b * w.L])
        gerr, gcut = max(gerr, e), max(gcut, c)
    # every layer's per-unit scores feed the shared one
    units_all = [(l, b, g) for l in range(w.L) for b in range(w.B) for g in range(w.Hkv)]
    serr = max(orc.run_units(lambda u: score_err(fs.S[u], out.unit_scores(*u)), units_all))
    units = [(l, b, g) for l in range(out.h) for b in range(w.B) for g in range(w.Hkv)]
    res = orc.run_units(lambda u: check_unit(orc, fs, out, *u, fs.gs[u[1]], TOL_BF16), units)
    # one shared ranking: every layer keeps a subset of the layer above
    for b in range(w.B):
        for g in range(w.Hkv):
            for l in range(1, out.h):
                k0 = out.unit(l - 1, b, g)[0]
                k1 = out.unit(l, b, g)[0]
                assert np.isin(k1, k0).all()
    rec = dict(workload=w.name, mode="global", units=len(units), swaps=sum(r[0] for r in res),
               fused_err=max(r[1] for r in res), shared_rel_err=gerr, shared_rel_err_cut=gcut, score_rel_err=serr)
    print(f"[fullsize] {rec}", flush=True)
    _diag(rec)
    assert serr < SCORE_TOL, f"{w.name}: window score error {serr}"
    assert gerr < SHARED_TOL, f"{w.name}: shared score error {gerr}"
    assert gcut < SCORE_TOL_CUT, f"{w.name}: shared score error near the cuts {gcut}"


# Cases in workload order, so each workload is generated and scored by the
# oracle once.  Long video adds fp32 fused values checked on every kept row
# and fuse-all (every non-kept token fused: dropped lists up to 10 000 rows).
CASES = [("longvideo", "layer_head"), ("longvideo", "global"), ("longvideo", "fp32_every_row"),
         ("longvideo", "fuse_all"), ("vllm72b", "layer_head"), ("vllm72b", "global"),
         ("batched", "layer_head"), ("batched", "global")]


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name,case", CASES, ids=[f"{a}-{b}" for a, b in CASES])
def test_full_size_every_unit(dev, orc, sg, cache, name, case):
    fs = _fullsize(cache, name, dev, orc, sg)
    if case == "global":
        _global(fs, orc)
    elif case == "fp32_every_row":
        _layer_head(fs, orc, all_rows=True, vfp32=True)
    elif case == "fuse_all":
        _layer_head(fs, orc, drop_all=True)
    else:
        _layer_head(fs, orc)
