#!/usr/bin/env python3
"""PruneKV benchmark on one MI355X.

One step = one viscache_prune call over the whole visual KV cache of a
workload: window scores, budgets, keep/drop selection, key gather and value
fusion, all layers and sequences.  The default workload is the batched ragged
one (8 sequences of 13.8k-23k visual tokens, 28 layers, 28 query / 4 kv heads,
head dim 128, 64-token windows, overall retention 19%), the largest that the
method's single-GPU configurations take.  Inputs are resident in HBM before
timing starts; L2 and the 256 MB Infinity Cache are flushed before every step
by reading a 1 GiB buffer (outside the timed region).

Prints one JSON line: compression throughput (GB of input visual K+V per
second) with the algorithmic HBM fraction, the binding-roofline fraction and
the roofline of the dominant kernel; the same workload under the shared
(global) ranking; decode-attention latency per step on the full, pruned,
pruned-with-4-bit-kept-rows and empty (no visual rows) caches, in one launch
per step and in one launch per layer; and the CPU oracle timed on a bounded
sample of the same workload, with single-threaded times of the tiny and
7B-shaped workloads.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, GB/s
MFMA_BF16_PEAK_TFLOPS = 2500.0  # dense bf16 matrix peak
# v_exp_f32: 256 CUs x 4 SIMDs x 16 lanes x 2.4 GHz at a quarter of the
# full vector rate.
EXP_PEAK_PER_S = 256 * 4 * 16 * 2.4e9 / 4
STAGES = ["upload", "score_stats", "score_colsum", "score_shared", "select", "gather_fuse"]


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="batched")
    ap.add_argument("--rank-mode", default="layer_head", choices=["layer_head", "global"])
    ap.add_argument("--schedule", default="parabolic", choices=["parabolic", "fixed", "arithmetic", "geometric"],
                    help="layer budget schedule (the budget ablation's alternatives to the parabola)")
    ap.add_argument("--drop-all", action="store_true", help="fuse every non-kept token (n_surv = n)")
    ap.add_argument("--score-queries", default="window", choices=["window", "prefill"],
                    help="window: the W trailing text queries score the visual keys; prefill: every "
                         "prefill token does, causally")
    ap.add_argument("--decode-steps", type=int, default=None)
    ap.add_argument("--no-flush", action="store_true", help="keep caches warm between steps")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-decode", action="store_true")
    ap.add_argument("--no-global", action="store_true", help="skip the shared-ranking line")
    ap.add_argument("--no-single-thread", action="store_true",
                    help="skip the single-threaded oracle times of the tiny and 7B workloads")
    ap.add_argument("--cpu-units", type=int, default=32,
                    help="oracle units in the CPU sample (0: every unit of the workload)")
    ap.add_argument("--copy-probe", action="store_true",
                    help="also run a plain device copy of known size (HBM counter calibration)")
    ap.add_argument("--reduce-pmc", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="reduce two rocprofv3 --pmc runs (FETCH_SIZE, WRITE_SIZE) of this script "
                         "into the traffic summary under profiles/, then exit")
    ap.add_argument("--pmc-command", default="", help="command line recorded in the traffic summary")
    return ap.parse_args()


def algorithmic(w, pc, n_list, prefill=False):
    """Per-launch algorithmic work of each stage (bytes, MFMA flops, exps) and
    of the whole path.

    Whole path (window scores): B_alg counts once each the keys of the scored
    layers, the window queries, the values of the survivors, and the kept
    keys, fused values and indices written; re-reads (the second score pass,
    the kept-key rows the gather reads again) are the implementation's, not
    the method's.  MFMA flops count the score contraction once and both
    fusion products; exps one per (window row, key) and per (kept, dropped)
    pair."""
    L, Hq, Hkv, d, W, G = w.L, w.Hq, w.Hkv, w.d, w.W, w.G
    R = G * W
    Ls = pc.h if pc.params.rank_mode == 0 else L
    out = {}
    k_bytes = sum(Hkv * n * d * 2 for n in n_list) * Ls
    if not prefill:
        q_bytes = w.B * Hq * W * d * 4 * Ls
        flops = sum(Hkv * 2 * R * n * d for n in n_list) * Ls
        exps = sum(Hkv * R * n for n in n_list) * Ls
        out["score_stats"] = dict(bytes=k_bytes + q_bytes, flops=flops, exps=exps)
        out["score_colsum"] = dict(bytes=k_bytes + q_bytes // 2, flops=flops, exps=exps)
        score_flops, score_exps = flops, exps
    else:
        # Every token queries its causal prefix: N(N+1)/2 (query, key) pairs
        # per head for the row statistics, and n(n+1)/2 + W n pairs that reach
        # a visual key for the column sums.  Queries are fp32, read once per pass.
        q_bytes = sum(Hq * (n + W) * d * 4 for n in n_list) * Ls
        t_bytes = w.B * Hkv * W * d * 2 * Ls
        p_all = sum(Hkv * G * (n + W) * (n + W + 1) // 2 for n in n_list) * Ls
        p_vis = sum(Hkv * G * (n * (n + 1) // 2 + W * n) for n in n_list) * Ls
        # One kernel runs both passes (row log-sum-exp, then column sums);
        # the reduction adds its per-workgroup column partials.
        out["score_stats"] = dict(bytes=k_bytes + t_bytes + q_bytes, flops=2 * d * (p_all + p_vis),
                                  exps=p_all + p_vis)
        units = Ls * w.B * Hkv
        groups = max(-(-G * (n + W) // 256) for n in n_list)
        per_wg = max(1, (groups * units + 4 * 512) // (8 * 512))  # the library's rule (about eight rounds)
        pwg = min(groups, -(-groups // per_wg))
        out["score_colsum"] = dict(bytes=units * pwg * max(n_list) * 4 + sum(n_list) * Hkv * Ls * 4, flops=0,
                                   exps=0)
        k_bytes += t_bytes
        score_flops, score_exps = 2 * d * p_all, p_all
    fb, fb_alg, ff, fe = 0, 0, 0, 0
    for b, n in enumerate(n_list):
        for l in range(pc.h):
            k, ns = pc.k[b * L + l], pc.n_surv[b * L + l]
            r = ns - k
            fb_alg += Hkv * (ns * d * 2 + k * (2 * d * 2 + 4))
            fb += Hkv * (ns * d * 2 + k * d * 2 + k * (2 * d * 2 + 4))
            ff += Hkv * 4 * k * r * d
            fe += Hkv * k * r
    out["gather_fuse"] = dict(bytes=fb, flops=ff, exps=fe)
    out["select"] = dict(bytes=sum(Hkv * n * 4 for n in n_list) * pc.h, flops=0, exps=0)
    out["path_bytes"] = k_bytes + q_bytes + fb_alg          # B_alg
    out["path_bytes_kept_reread"] = k_bytes + q_bytes + fb  # plus the kept-key rows read again
    out["path_flops"] = score_flops + ff
    out["path_exps"] = score_exps + fe
    return out


# Kernel of each timed stage, and the sources its code comes from (the hash of
# these files decides whether stored HBM counters still describe the kernel).
STAGE_KERNEL = {
    "score_stats": ("k_score_stats", ["k_score.hip"]),
    "score_colsum": ("k_score_colsum", ["k_score.hip"]),
    "select": ("k_select", ["k_select.hip"]),
    "gather_fuse": ("k_fuse", ["k_fuse.hip"]),
}
PREFILL_STAGE_KERNEL = dict(STAGE_KERNEL, score_stats=("k_pscore", ["k_pscore.hip"]),
                            score_colsum=("k_pscore_reduce", ["k_pscore.hip"]))
COPY_PROBE_BYTES = 1 << 30
TRAFFIC_DEFAULT = "batched"


def traffic_file(workload):
    return os.path.join(ROOT, "profiles", f"traffic_{workload}_hbm_counters.md")


def kernel_hash(files):
    import hashlib
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2608_24063_amd", "csrc")
    for f in sorted(set(files + ["vc_device.h", "vc_internal.h"])):
        with open(os.path.join(csrc, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def copy_probe(torch, dev):
    """A plain device-to-device copy of COPY_PROBE_BYTES: it reads and writes
    exactly that many bytes of HBM, which calibrates FETCH_SIZE / WRITE_SIZE."""
    src = torch.ones(COPY_PROBE_BYTES // 4, dtype=torch.int32, device=dev)
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    del src, dst


# Source file of each library kernel (for the hash that dates stored counters).
KERNEL_SOURCES = {k: files for k, files in list(STAGE_KERNEL.values()) + list(PREFILL_STAGE_KERNEL.values())}
KERNEL_SOURCES.update({"k_score_global": ["k_score.hip"], "k_upload": ["k_setup.hip"]})


def reduce_pmc(fetch_dir, write_dir, command, workload):
    """Per-dispatch HBM bytes of each library kernel from two counter runs,
    scaled by what the same counters read for the copy probe of that run.
    Records are kept per kernel name and merged into the stored summary, so
    runs of different configurations (window and prefill scores) add up."""
    import csv
    import glob
    import re

    def load(d, counter):
        per = {}
        for f in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
            for row in csv.DictReader(open(f)):
                if row["Counter_Name"] != counter:
                    continue
                name = row["Kernel_Name"]
                m = re.search(r"(k_\w+)<", name) or re.search(r"(k_\w+)\(", name)
                # the copy probe is the runtime's device-to-device blit
                key = m.group(1) if (m and "vc::" in name) else ("copy" if "copyBuffer" in name else None)
                if key is None:
                    continue
                per.setdefault(key, []).append((float(row["Counter_Value"]), int(row["Grid_Size"])))
        return per

    fetch, write = load(fetch_dir, "FETCH_SIZE"), load(write_dir, "WRITE_SIZE")
    # The copy probe: the copy dispatch with the largest counter value.
    fc = max(v for v, _ in fetch.get("copy", [(0.0, 0)]))
    wc = max(v for v, _ in write.get("copy", [(0.0, 0)]))
    if fc <= 0 or wc <= 0:
        raise SystemExit("no copy-probe dispatch found in the counter runs (run bench.py --copy-probe)")
    sf, sw = COPY_PROBE_BYTES / (fc * 1024.0), COPY_PROBE_BYTES / (wc * 1024.0)
    old = {}
    try:
        text = open(traffic_file(workload)).read()
        old = json.loads(text.split("```json", 1)[1].split("```", 1)[0])
    except (OSError, IndexError, ValueError):
        pass
    rec = {"copy_probe_bytes": COPY_PROBE_BYTES, "kernels": dict(old.get("kernels", {}))}
    for kname, files in KERNEL_SOURCES.items():
        if kname not in fetch or kname not in write:
            continue
        fk = sum(v for v, _ in fetch[kname]) / len(fetch[kname])
        wk = sum(v for v, _ in write[kname]) / len(write[kname])
        rec["kernels"][kname] = {"fetch_kib": fk, "write_kib": wk, "fetch_scale": sf, "write_scale": sw,
                                 "hbm_bytes": fk * 1024.0 * sf + wk * 1024.0 * sw,
                                 "source_hash": kernel_hash(files), "command": command or "(not recorded)"}
    lines = [f"# HBM traffic per dispatch, {workload} workload (rocprofv3 FETCH_SIZE / WRITE_SIZE)", "",
             "Each counter is taken in its own run of the command recorded with the kernel; the copy probe",
             f"of each run ({COPY_PROBE_BYTES} bytes read and written) calibrates both counters of that run.", "",
             "| kernel | FETCH_SIZE KiB | WRITE_SIZE KiB | fetch scale | write scale | scaled HBM MB | source hash |",
             "|---|---|---|---|---|---|---|"]
    for kname, k in sorted(rec["kernels"].items()):
        lines.append(f"| {kname} | {k['fetch_kib']:.0f} | {k['write_kib']:.0f} | {k['fetch_scale']:.4f} | "
                     f"{k['write_scale']:.4f} | {k['hbm_bytes'] / 1e6:.1f} | {k['source_hash']} |")
    lines += ["", "Commands:", ""]
    for cmd in sorted({k["command"] for k in rec["kernels"].values()}):
        names = ", ".join(sorted(n for n, k in rec["kernels"].items() if k["command"] == cmd))
        lines += [f"- {names}:", "", "  ```", "  " + cmd, "  ```", ""]
    lines += ["Machine-readable (read by bench.py):", "", "```json", json.dumps(rec), "```", ""]
    os.makedirs(os.path.dirname(traffic_file(workload)), exist_ok=True)
    with open(traffic_file(workload), "w") as f:
        f.write("\n".join(lines))
    print("\n".join(lines))


def stored_traffic(stage, workload, kernels=STAGE_KERNEL):
    """Scaled HBM bytes per dispatch of a stage's kernel on a workload, if the
    stored counters were taken on that kernel's current source; else None."""
    try:
        text = open(traffic_file(workload)).read()
        blob = text.split("```json", 1)[1].split("```", 1)[0]
        kname, files = kernels[stage]
        rec = json.loads(blob)["kernels"].get(kname)
    except (OSError, IndexError, ValueError, KeyError):
        return None
    if not rec or rec.get("source_hash") != kernel_hash(files):
        return None
    return rec["hbm_bytes"]


class HipEvents:
    """Timing events without the system-scope release fence (HIP's
    hipEventDisableSystemFence), so bracketing each stage costs little."""
    FLAGS = 0x20000000  # hipEventDisableSystemFence

    def __init__(self, count):
        import ctypes
        self.ct = ctypes
        self.hip = ctypes.CDLL("libamdhip64.so")
        self.hip.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint]
        self.hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
        self.hip.hipEventDestroy.argtypes = [ctypes.c_void_p]
        self.ev = []
        for _ in range(count):
            h = ctypes.c_void_p()
            if self.hip.hipEventCreateWithFlags(ctypes.byref(h), self.FLAGS) != 0:
                raise RuntimeError("hipEventCreateWithFlags failed")
            self.ev.append(h.value)

    def ms(self, a, b):
        out = self.ct.c_float()
        if self.hip.hipEventElapsedTime(self.ct.byref(out), self.ev[a], self.ev[b]) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return out.value

    def close(self):
        for h in self.ev:
            self.hip.hipEventDestroy(h)


def time_prune(pc, steps, warmup, flush_buf, torch):
    """Whole-path time per step (two events per step, nothing between the
    kernels), then per-stage times from separate steps bracketed stage by
    stage.  Caches are flushed before every step, outside the timed region."""
    for _ in range(warmup):
        if flush_buf is not None:
            flush_buf.sum()
        pc.run()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(steps):
        if flush_buf is not None:
            flush_buf.sum()  # reading 1 GiB evicts L2 and the Infinity Cache; not timed
        ev[s][0].record()
        pc.run()
        ev[s][1].record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    tot = [a.elapsed_time(b) for a, b in ev]
    hev = HipEvents(7 * steps)
    for s in range(steps):
        if flush_buf is not None:
            flush_buf.sum()
        pc.run(events=hev.ev[7 * s:7 * s + 7])
    torch.cuda.synchronize()
    stage = [[hev.ms(7 * s + i, 7 * s + i + 1) for i in range(6)] for s in range(steps)]
    hev.close()
    return tot, stage, wall


def median(xs):
    ys = sorted(xs)
    m = len(ys) // 2
    return ys[m] if len(ys) % 2 else 0.5 * (ys[m - 1] + ys[m])


def prune_report(w, pc, n, tot, stage, prefill, workload):
    """Throughput, algorithmic fractions and the dominant kernel's roofline of
    one timed prune configuration."""
    ms = median(tot)
    t = ms * 1e-3
    in_bytes = sum(w.Hkv * x * w.d * 2 * 2 for x in n) * w.L
    alg = algorithmic(w, pc, n, prefill)
    stage_us = {STAGES[i]: 1e3 * median([s[i] for s in stage]) for i in range(6)}
    t_hbm = alg["path_bytes"] / (HBM_PEAK_GBS * 1e9)
    t_mfma = alg["path_flops"] / (MFMA_BF16_PEAK_TFLOPS * 1e12)
    t_exp = alg["path_exps"] / EXP_PEAK_PER_S
    bind = max(("hbm", t_hbm), ("mfma", t_mfma), ("exp", t_exp), key=lambda x: x[1])
    dom = max(("score_stats", "score_colsum", "select", "gather_fuse"), key=lambda s: stage_us[s])
    a = alg[dom]
    td = stage_us[dom] * 1e-6
    fr_hbm = a["bytes"] / td / 1e9 / HBM_PEAK_GBS
    fr_mfma = a["flops"] / td / 1e12 / MFMA_BF16_PEAK_TFLOPS
    if fr_mfma >= fr_hbm:
        roof = dict(bound="mfma", achieved=a["flops"] / td / 1e12, peak=MFMA_BF16_PEAK_TFLOPS, unit="TFLOP/s")
    else:
        roof = dict(bound="hbm", achieved=a["bytes"] / td / 1e9, peak=HBM_PEAK_GBS, unit="GB/s")
    roof["frac"] = roof["achieved"] / roof["peak"]
    kernels = PREFILL_STAGE_KERNEL if prefill else STAGE_KERNEL
    roof["traffic"] = stored_traffic(dom, workload, kernels)
    roof.update(kernel=kernels[dom][0], stage=dom, kernel_us=stage_us[dom], alg_flops=a["flops"],
                alg_bytes=a["bytes"], hbm_frac=fr_hbm, mfma_frac=fr_mfma, exp_per_s=a["exps"] / td)
    return dict(ms=ms, ms_mean=sum(tot) / len(tot), gbs_in=in_bytes / t / 1e9, in_bytes=in_bytes,
                b_alg=alg["path_bytes"], hbm_gbs=alg["path_bytes"] / t / 1e9,
                hbm_frac=alg["path_bytes"] / t / 1e9 / HBM_PEAK_GBS,
                hbm_frac_with_kept_reread=alg["path_bytes_kept_reread"] / t / 1e9 / HBM_PEAK_GBS,
                bind_frac=bind[1] / t, bind_unit=bind[0],
                floors_us=dict(hbm=t_hbm * 1e6, mfma=t_mfma * 1e6, exp=t_exp * 1e6),
                stage_us=stage_us, roofline=roof)


def decode_latency(w, pc, dev, steps, flush_buf, torch, sg):
    """Per-step latency of append + attention over all layers, on the full,
    pruned and empty-visual caches and on the pruned cache with its kept rows
    in 4 bits (whole 32-row tiles; text and generated rows in bf16), in one
    launch per step over a piece table built once per cache
    (viscache_decode_step_planned); the same four with the cut made on the
    device in every step (viscache_decode_step / _q4); and the full, pruned
    and empty caches with one launch per layer (a model's layer loop)."""
    from paper_2608_24063_amd.tensors import DecodeCache
    from synthgen.device import bf16_tensor
    L, B, Hkv, d = w.L, w.B, w.Hkv, w.d
    n = [int(x) for x in w.n_vis()]
    results = {}
    text_k = bf16_tensor(sg.normal_bf16(w.seed, 901, (L * B * Hkv, w.W, d)), dev)
    text_v = bf16_tensor(sg.normal_bf16(w.seed, 902, (L * B * Hkv, w.W, d)), dev)
    kn = bf16_tensor(sg.normal_bf16(w.seed, 903, (steps, L, B, Hkv, d)), dev)
    vn = bf16_tensor(sg.normal_bf16(w.seed, 904, (steps, L, B, Hkv, d)), dev)
    q = bf16_tensor(sg.normal_bf16(w.seed, 905, (steps, L, B, w.Hq, d)), dev)
    out = torch.empty((L, B, w.Hq, d), dtype=torch.float32, device=dev)
    toff = [0]
    for x in n:
        toff.append(toff[-1] + x)
    for variant in ("full", "pruned", "empty", "pruned_q4", "full_cut", "pruned_cut", "empty_cut", "pruned_q4_cut",
                    "full_layers", "pruned_layers", "empty_layers"):
        base = variant.replace("_layers", "").replace("_cut", "")
        vis = []
        for l in range(L):
            for b in range(B):
                for g in range(Hkv):
                    if base == "full":
                        vis.append(n[b])
                    elif base in ("pruned", "pruned_q4"):
                        vis.append(pc.k[b * L + l])
                    else:
                        vis.append(0)
        caps = [v + w.W + steps for v in vis]
        c = DecodeCache(L, B, w.Hq, Hkv, d, caps, dev)
        lens = []
        for l in range(L):
            for b in range(B):
                for g in range(Hkv):
                    u = (l * B + b) * Hkv + g
                    r0, v = c.offs_host[u], vis[u]
                    if base == "full" and v:
                        s0 = toff[b] * Hkv + g * n[b]
                        c.k_pool[r0:r0 + v] = pc.k_in[l][s0:s0 + v]
                        c.v_pool[r0:r0 + v] = pc.v_in[l][s0:s0 + v]
                    elif base in ("pruned", "pruned_q4") and v:
                        a0, a1 = pc.unit_rows(l, b, g)
                        c.k_pool[r0:r0 + v] = pc.k_out[l][a0:a1]
                        c.v_pool[r0:r0 + v] = pc.v_out[l][a0:a1]
                    c.k_pool[r0 + v:r0 + v + w.W] = text_k[u]
                    c.v_pool[r0 + v:r0 + v + w.W] = text_v[u]
                    lens.append(v + w.W)
        c.len.copy_(torch.tensor(lens, dtype=torch.int32))
        rows0 = sum(lens)
        nq = [v // 32 * 32 for v in vis] if base == "pruned_q4" else [0] * len(vis)
        if base == "pruned_q4":
            c.quantize(nq)
        if variant.endswith("_layers"):
            step = c.step_layers
        elif variant.endswith("_cut"):
            step = c.step_q4 if base == "pruned_q4" else c.step
        else:
            c.plan()  # once per cache, outside the timed steps

            def step(k, v, qq, o, sc, _c=c, _q4=(base == "pruned_q4")):
                _c.step_planned(k, v, qq, o, sc, q4=_q4)
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(steps)]
        torch.cuda.synchronize()
        for t in range(steps):
            if flush_buf is not None:
                flush_buf.sum()
            ev[t][0].record()
            step(kn[t], vn[t], q[t], out, d ** -0.5)  # append + attend
            ev[t][1].record()
        torch.cuda.synchronize()
        ts = [a.elapsed_time(b) * 1e3 for a, b in ev]
        # K and V: bf16 rows 2d bytes, 4-bit rows d/2 code bytes + d/32 (scale, lo) pairs
        q4_rows = sum(nq)
        bytes_step0 = ((rows0 + len(lens) - q4_rows) * d * 2 + q4_rows * (d // 2 + d // 32 * 8)) * 2
        results[variant] = dict(mean_us=sum(ts) / len(ts), median_us=median(ts),
                                rows=rows0, bytes_per_step=bytes_step0)
        del c

    def target(full, pr, em):
        rho = pr["bytes_per_step"] / full["bytes_per_step"]
        bound = rho * full["median_us"] + em["median_us"]
        return rho, bound

    full, pr, em, pq = results["full"], results["pruned"], results["empty"], results["pruned_q4"]
    rho, bound = target(full, pr, em)
    fl, pl, el = results["full_layers"], results["pruned_layers"], results["empty_layers"]
    _, bound_l = target(fl, pl, el)
    fc, pcut, ec, pqc = results["full_cut"], results["pruned_cut"], results["empty_cut"], results["pruned_q4_cut"]
    _, bound_c = target(fc, pcut, ec)
    return dict(steps=steps, full_us=full["median_us"], pruned_us=pr["median_us"], empty_us=em["median_us"],
                full_mean_us=full["mean_us"], pruned_mean_us=pr["mean_us"],
                speedup=full["median_us"] / pr["median_us"], rho=rho,
                target_speedup=full["median_us"] / bound, meets_target=pr["median_us"] <= bound,
                full_hbm_gbs=full["bytes_per_step"] / (full["median_us"] * 1e3),
                pruned_hbm_gbs=pr["bytes_per_step"] / (pr["median_us"] * 1e3),
                pruned_q4_us=pq["median_us"], pruned_q4_mean_us=pq["mean_us"],
                speedup_q4=full["median_us"] / pq["median_us"],
                q4_bytes_ratio=pq["bytes_per_step"] / pr["bytes_per_step"],
                pruned_q4_hbm_gbs=pq["bytes_per_step"] / (pq["median_us"] * 1e3),
                device_cut=dict(full_us=fc["median_us"], pruned_us=pcut["median_us"], empty_us=ec["median_us"],
                                pruned_q4_us=pqc["median_us"], speedup=fc["median_us"] / pcut["median_us"],
                                target_speedup=fc["median_us"] / bound_c, meets_target=pcut["median_us"] <= bound_c),
                per_layer_launch=dict(launches_per_step=L, full_us=fl["median_us"], pruned_us=pl["median_us"],
                                      empty_us=el["median_us"], speedup=fl["median_us"] / pl["median_us"],
                                      target_speedup=fl["median_us"] / bound_l,
                                      meets_target=pl["median_us"] <= bound_l),
                cold=flush_buf is not None)


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def oracle_units(orc, sg, w, host, pc_k, pc_ns, h, units, threads, prefill=False):
    """The oracle's whole path (score, select, gather, fuse) on `units`, one
    unit per thread.  Returns (wall s, summed per-unit thread CPU s)."""
    import numpy as np
    L, Hkv = w.L, w.Hkv
    n = [int(x) for x in w.n_vis()]
    toff = [0]
    for x in n:
        toff.append(toff[-1] + x)
    cpu = []

    def one(u):
        c0 = time.thread_time()
        l, b, g = u
        s0 = toff[b] * Hkv + g * n[b]
        K = host["K"][l][s0:s0 + n[b]]
        V = host["V"][l][s0:s0 + n[b]]
        k, ns = pc_k[b * L + l], pc_ns[b * L + l]
        if not prefill:
            Q = host["Q"][l][b, g * w.G:(g + 1) * w.G].reshape(-1, w.d)
            orc.prune_unit(K, V, Q, k, ns)
        else:
            N = n[b] + w.W
            r0 = (toff[b] + b * w.W) * w.Hq + g * w.G * N
            Q = host["Q"][l][r0:r0 + w.G * N].reshape(w.G, N, w.d)
            S32 = orc.scores_unit_prefill(K, host["KT"][l][b, g], Q).astype(np.float32)
            kept, drop = orc.select(S32, k, ns)
            orc.gather(K, kept)
            orc.fuse(V, kept, drop)
        cpu.append(time.thread_time() - c0)
        return 1

    t0 = time.perf_counter()
    orc.run_units(one, units, threads=threads)
    return time.perf_counter() - t0, sum(cpu)


def cpu_baseline(w, pc, host, units_wanted, sg, single_thread=True, prefill=False):
    """The oracle on a bounded sample of the same workload (whole units of the
    layer/head ranking: score, select, gather, fuse), fanned over the host's
    threads (at most 16, the machine's CPU share of one GPU); plus the whole tiny
    and 7B-shaped workloads on one thread."""
    import oracle as orc
    from synthgen.device import upload_layers
    ncpu = os.cpu_count() or 1
    threads = min(16, ncpu)
    L, Hkv = w.L, w.Hkv
    n = [int(x) for x in w.n_vis()]
    allu = [(l, b, g) for l in range(pc.h) for b in range(w.B) for g in range(Hkv)]
    units_wanted = len(allu) if units_wanted <= 0 else min(units_wanted, len(allu))
    step = max(1, len(allu) // units_wanted)
    units = allu[::step][:units_wanted]
    wall, cpu_s = oracle_units(orc, sg, w, host, pc.k, pc.n_surv, pc.h, units, threads, prefill)
    t_full = wall * len(allu) / len(units)
    in_bytes = sum(Hkv * x * w.d * 2 * 2 for x in n) * L
    rec = dict(value=in_bytes / t_full / 1e9, unit="GB/s", cores=threads, kind="oracle",
               sample=f"{len(units)} of {len(allu)} (layer, kv head) units of the {w.name} workload, whole "
                      f"path per unit (score, select, gather, fuse), {wall:.1f} s wall on {threads} threads "
                      f"({cpu_s:.1f} s summed per-unit CPU time); scaled to all units",
               host_cpus=ncpu, cpu_model=cpu_model(), threads=threads, sample_wall_s=wall,
               sample_cpu_s=cpu_s, full_workload_s=t_full)
    if single_thread and not prefill:
        st = {}
        for wl in (sg.TINY, sg.VLLM7B):
            import paper_2608_24063_amd as vc
            nn = [int(x) for x in wl.n_vis()]
            shape = vc.make_shape(wl.B, wl.L, wl.Hq, wl.Hkv, wl.d, wl.W, nn)
            k, ns, h = vc.viscache_budget(shape, vc.make_params(wl.retention))
            _, hh = upload_layers(wl, range(h), None, keep_host=True, host_only=True)
            uu = [(l, b, g) for l in range(h) for b in range(wl.B) for g in range(wl.Hkv)]
            wall1, cpu1 = oracle_units(orc, sg, wl, hh, k, ns, h, uu, 1)
            st[wl.name] = dict(wall_s=wall1, cpu_s=cpu1, units=len(uu))
        rec["single_thread"] = st
    return rec


def main():
    args = parse()
    if args.reduce_pmc:
        reduce_pmc(args.reduce_pmc[0], args.reduce_pmc[1], args.pmc_command, args.workload)
        return
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
              f"(asked for --gpus {args.gpus}, WORLD_SIZE={world}).", file=sys.stderr)
        sys.exit(2)
    import torch

    import paper_2608_24063_amd as vc
    import synthgen as sg
    from paper_2608_24063_amd.tensors import PruneCall
    from synthgen.device import upload_layers

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    vc.lib()
    w = sg.WORKLOADS[args.workload]
    mode = vc.VC_RANK_GLOBAL if args.rank_mode == "global" else vc.VC_RANK_LAYER_HEAD
    n = [int(x) for x in w.n_vis()]
    print(f"[bench] generating {w.name}: B={w.B} L={w.L} Hq={w.Hq} Hkv={w.Hkv} d={w.d} W={w.W} n={n}",
          file=sys.stderr, flush=True)
    keep_host = not args.no_cpu_baseline
    prefill = args.score_queries == "prefill"
    dv, host = upload_layers(w, range(w.L), dev, keep_host=keep_host, prefill=prefill)
    sched = {"parabolic": vc.VC_SCHED_PARABOLIC, "fixed": vc.VC_SCHED_FIXED,
             "arithmetic": vc.VC_SCHED_ARITHMETIC, "geometric": vc.VC_SCHED_GEOMETRIC}[args.schedule]

    def call(rank_mode):
        params = vc.make_params(w.retention, rank_mode=rank_mode, schedule=sched, drop_all=args.drop_all,
                                score_queries=vc.VC_SCORE_PREFILL if prefill else vc.VC_SCORE_WINDOW)
        return PruneCall(w.B, w.L, w.Hq, w.Hkv, w.d, w.W, n, params, [dv["K"][l] for l in range(w.L)],
                         [dv["V"][l] for l in range(w.L)], [dv["Q"][l] for l in range(w.L)],
                         k_text=[dv["KT"][l] for l in range(w.L)] if prefill else None)

    pc = call(mode)
    # Flush by reading (not writing) 1 GiB, so the caches hold clean lines and
    # the measured kernels pay no write-back of the flush data.
    # (float32: a sum of int32 would be widened to int64 first, writing 2 GiB.)
    flush = None if args.no_flush else torch.ones(1 << 28, dtype=torch.float32, device=dev)
    print(f"[bench] timing {args.steps} prune steps after {args.warmup} warm-up ({args.rank_mode})",
          file=sys.stderr, flush=True)
    t_region0 = time.perf_counter()
    tot, stage, wall = time_prune(pc, args.steps, args.warmup, flush, torch)
    rep = prune_report(w, pc, n, tot, stage, prefill, args.workload)
    other = None
    if not args.no_global and not prefill:
        omode = vc.VC_RANK_LAYER_HEAD if mode == vc.VC_RANK_GLOBAL else vc.VC_RANK_GLOBAL
        oname = "layer_head" if omode == vc.VC_RANK_LAYER_HEAD else "global"
        print(f"[bench] timing {args.steps} prune steps ({oname})", file=sys.stderr, flush=True)
        pco = call(omode)
        tot_o, stage_o, _ = time_prune(pco, args.steps, args.warmup, flush, torch)
        rep_o = prune_report(w, pco, n, tot_o, stage_o, prefill, args.workload)
        other = dict(rank_mode=oname, ms_per_step=rep_o["ms"], ms_per_step_mean=rep_o["ms_mean"],
                     value=rep_o["gbs_in"], hbm_frac=rep_o["hbm_frac"], b_alg=rep_o["b_alg"],
                     bind_frac=rep_o["bind_frac"], bind_unit=rep_o["bind_unit"], stage_us=rep_o["stage_us"],
                     dominant=rep_o["roofline"]["kernel"], dominant_frac=rep_o["roofline"]["frac"])
        del pco
    t_region = time.perf_counter() - t_region0

    if args.copy_probe:
        copy_probe(torch, dev)
    dec = None
    if not args.no_decode:
        dsteps = args.decode_steps or w.decode_steps
        print(f"[bench] decode: {dsteps} steps x 7 caches", file=sys.stderr, flush=True)
        dec = decode_latency(w, pc, dev, dsteps, flush, torch, sg)
    cpu = None
    if not args.no_cpu_baseline:
        print(f"[bench] CPU oracle ({args.cpu_units or 'all'} units)", file=sys.stderr, flush=True)
        cpu = cpu_baseline(w, pc, host, args.cpu_units, sg, single_thread=not args.no_single_thread,
                           prefill=prefill)

    rec = {
        "metric": "PruneKV compress GB/s (% of HBM peak) + decode-attn speedup vs full KV",
        "value": rep["gbs_in"],
        "unit": "GB/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": rep["ms"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"{w.name}: B={w.B} L={w.L} Hq={w.Hq} Hkv={w.Hkv} d={w.d} "
                               f"{w.frames}{'+-' + str(w.frame_jitter) if w.frame_jitter else ''}x"
                               f"{w.tokens_per_frame} visual tokens per sequence, W={w.W}, RR={w.retention}",
                   "n_vis": n, "rank_mode": args.rank_mode, "schedule": args.schedule, "drop_all": args.drop_all,
                   "score_queries": args.score_queries, "cold_caches": flush is not None,
                   "input_visual_kv_bytes": rep["in_bytes"]},
        "ms_per_step_mean": rep["ms_mean"],
        "hbm_frac": rep["hbm_frac"],
        "hbm_gbs": rep["hbm_gbs"],
        "b_alg_bytes": rep["b_alg"],
        "hbm_frac_with_kept_reread": rep["hbm_frac_with_kept_reread"],
        "bind_frac": rep["bind_frac"],
        "bind_unit": rep["bind_unit"],
        "floors_us": rep["floors_us"],
        "stage_us": rep["stage_us"],
        "wall_s_timed_region": t_region,
        "roofline": rep["roofline"],
        "other_rank_mode": other,
        "decode": dec,
        "cpu_baseline": cpu,
    }
    print(json.dumps(rec))


if __name__ == "__main__":
    main()
