#!/usr/bin/env python3
"""PruneKV benchmark on one MI355X.

One step = one viscache_prune call over the whole visual KV cache of the
7B-shaped workload (28 layers, 28 query / 4 kv heads, head dim 128, 16 frames x
196 tokens, 64-token window, overall retention 28%): window scores, budgets,
keep/drop selection, key gather and value fusion.  Inputs are resident in HBM
before timing starts; L2 and the 256 MB Infinity Cache are flushed before every
step by reading a 1 GiB buffer (outside the timed region), because the 180 MB
input would otherwise be served from the Infinity Cache.

Prints one JSON line: compression throughput (GB of input visual K+V per second)
with the roofline of the dominant kernel, decode-attention latency per step on
the full, pruned, pruned-with-4-bit-kept-rows and empty (no visual rows)
caches, and the CPU oracle timed
on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, GB/s
MFMA_BF16_PEAK_TFLOPS = 2500.0  # dense bf16 matrix peak
STAGES = ["upload", "score_stats", "score_colsum", "score_shared", "select", "gather_fuse"]


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="vllm7b")
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
    ap.add_argument("--cpu-units", type=int, default=0,
                    help="oracle units in the CPU sample (0: every unit of the workload)")
    ap.add_argument("--copy-probe", action="store_true",
                    help="also run a plain device copy of known size (HBM counter calibration)")
    ap.add_argument("--reduce-pmc", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="reduce two rocprofv3 --pmc runs (FETCH_SIZE, WRITE_SIZE) of this script "
                         "into the traffic summary under profiles/, then exit")
    ap.add_argument("--pmc-command", default="", help="command line recorded in the traffic summary")
    return ap.parse_args()


def algorithmic(w, pc, n_list, prefill=False):
    """Per-launch algorithmic work of each stage (bytes, MFMA flops, exps)."""
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
    fb, ff, fe = 0, 0, 0
    for b, n in enumerate(n_list):
        for l in range(pc.h):
            k, ns = pc.k[b * L + l], pc.n_surv[b * L + l]
            r = ns - k
            fb += Hkv * (ns * d * 2 + k * d * 2 + k * (2 * d * 2 + 4))
            ff += Hkv * 4 * k * r * d
            fe += Hkv * k * r
    out["gather_fuse"] = dict(bytes=fb, flops=ff, exps=fe)
    out["select"] = dict(bytes=sum(Hkv * n * 4 for n in n_list) * pc.h, flops=0, exps=0)
    # whole-path algorithmic bytes: K of scored layers, Q, V of survivors, outputs
    out["path_bytes"] = k_bytes + q_bytes + fb
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
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_vllm7b_hbm_counters.md")


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


def reduce_pmc(fetch_dir, write_dir, command):
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
        text = open(TRAFFIC_FILE).read()
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
    lines = ["# HBM traffic per dispatch, 7B-shaped workload (rocprofv3 FETCH_SIZE / WRITE_SIZE)", "",
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
    os.makedirs(os.path.dirname(TRAFFIC_FILE), exist_ok=True)
    with open(TRAFFIC_FILE, "w") as f:
        f.write("\n".join(lines))
    print("\n".join(lines))


def stored_traffic(stage, kernels=STAGE_KERNEL):
    """Scaled HBM bytes per dispatch of a stage's kernel, if the stored counters
    were taken on that kernel's current source; else None."""
    try:
        text = open(TRAFFIC_FILE).read()
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


def decode_latency(w, pc, dev, steps, flush_buf, torch, sg):
    """Per-step latency of append + attention over all layers, on the full,
    pruned and empty-visual caches, and on the pruned cache with its kept rows
    in 4 bits (whole 32-row tiles; text and generated rows in bf16)."""
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
    for variant in ("full", "pruned", "empty", "pruned_q4"):
        vis = []
        for l in range(L):
            for b in range(B):
                for g in range(Hkv):
                    if variant == "full":
                        vis.append(n[b])
                    elif variant in ("pruned", "pruned_q4"):
                        vis.append(pc.k[b * L + l])
                    else:
                        vis.append(0)
        caps = [v + w.W + steps for v in vis]
        c = DecodeCache(L, B, w.Hq, Hkv, d, caps, dev)
        lens = []
        toff = [0]
        for x in n:
            toff.append(toff[-1] + x)
        for l in range(L):
            for b in range(B):
                for g in range(Hkv):
                    u = (l * B + b) * Hkv + g
                    r0, v = c.offs_host[u], vis[u]
                    if variant == "full" and v:
                        s0 = toff[b] * Hkv + g * n[b]
                        c.k_pool[r0:r0 + v] = pc.k_in[l][s0:s0 + v]
                        c.v_pool[r0:r0 + v] = pc.v_in[l][s0:s0 + v]
                    elif variant in ("pruned", "pruned_q4") and v:
                        a0, a1 = pc.unit_rows(l, b, g)
                        c.k_pool[r0:r0 + v] = pc.k_out[l][a0:a1]
                        c.v_pool[r0:r0 + v] = pc.v_out[l][a0:a1]
                    c.k_pool[r0 + v:r0 + v + w.W] = text_k[u]
                    c.v_pool[r0 + v:r0 + v + w.W] = text_v[u]
                    lens.append(v + w.W)
        c.len.copy_(torch.tensor(lens, dtype=torch.int32))
        rows0 = sum(lens)
        nq = [v // 32 * 32 for v in vis] if variant == "pruned_q4" else [0] * len(vis)
        step = c.step
        if variant == "pruned_q4":
            c.quantize(nq)
            step = c.step_q4
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(steps)]
        # one warm-up step on a copy of the lengths, then restore
        torch.cuda.synchronize()
        for t in range(steps):
            if flush_buf is not None:
                flush_buf.sum()
            ev[t][0].record()
            step(kn[t], vn[t], q[t], out, d ** -0.5)  # append + attend, one launch
            ev[t][1].record()
        torch.cuda.synchronize()
        ts = sorted(a.elapsed_time(b) * 1e3 for a, b in ev)
        # K and V: bf16 rows 2d bytes, 4-bit rows d/2 code bytes + d/32 (scale, lo) pairs
        q4_rows = sum(nq)
        bytes_step0 = ((rows0 + len(lens) - q4_rows) * d * 2 + q4_rows * (d // 2 + d // 32 * 8)) * 2
        results[variant] = dict(mean_us=sum(ts) / len(ts), median_us=ts[len(ts) // 2],
                                rows=rows0, bytes_per_step=bytes_step0)
        del c
    full, pr, em, pq = results["full"], results["pruned"], results["empty"], results["pruned_q4"]
    rho = pr["bytes_per_step"] / full["bytes_per_step"]
    bound = rho * full["median_us"] + em["median_us"]
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
                cold=flush_buf is not None)


def cpu_baseline(w, pc, host, units_wanted, prefill=False):
    """The oracle on a bounded sample of the same workload: whole units
    (score, select, gather, fuse) of layer/head ranking, one unit per thread."""
    import numpy as np

    import oracle as orc
    threads = min(16, os.cpu_count() or 1)
    L, Hkv = w.L, w.Hkv
    n = [int(x) for x in w.n_vis()]
    toff = [0]
    for x in n:
        toff.append(toff[-1] + x)
    allu = [(l, b, g) for l in range(pc.h) for b in range(w.B) for g in range(Hkv)]
    units_wanted = len(allu) if units_wanted <= 0 else min(units_wanted, len(allu))
    step = max(1, len(allu) // units_wanted)
    units = allu[::step][:units_wanted]

    def one(u):
        l, b, g = u
        s0 = toff[b] * Hkv + g * n[b]
        K = host["K"][l][s0:s0 + n[b]]
        V = host["V"][l][s0:s0 + n[b]]
        k, ns = pc.k[b * L + l], pc.n_surv[b * L + l]
        if not prefill:
            Q = host["Q"][l][b, g * w.G:(g + 1) * w.G].reshape(-1, w.d)
            orc.prune_unit(K, V, Q, k, ns)
            return 1
        N = n[b] + w.W
        r0 = (toff[b] + b * w.W) * w.Hq + g * w.G * N
        Q = host["Q"][l][r0:r0 + w.G * N].reshape(w.G, N, w.d)
        S32 = orc.scores_unit_prefill(K, host["KT"][l][b, g], Q).astype(np.float32)
        kept, drop = orc.select(S32, k, ns)
        orc.gather(K, kept)
        orc.fuse(V, kept, drop)
        return 1

    t0 = time.perf_counter()
    orc.run_units(one, units, threads=threads)
    wall = time.perf_counter() - t0
    # whole-workload time at the same per-unit rate and thread count
    t_full = wall * len(allu) / len(units)
    in_bytes = sum(Hkv * x * w.d * 2 * 2 for x in n) * L
    return dict(value=in_bytes / t_full / 1e9, unit="GB/s", cores=threads, kind="oracle",
                sample=f"{len(units)} of {len(allu)} (layer, kv head) units, whole path per unit, "
                       f"{wall:.1f} s wall on {threads} threads; scaled to the full workload",
                full_workload_s=t_full)


def main():
    args = parse()
    if args.reduce_pmc:
        reduce_pmc(args.reduce_pmc[0], args.reduce_pmc[1], args.pmc_command)
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
    print(f"[bench] generating {w.name}: B={w.B} L={w.L} Hq={w.Hq} Hkv={w.Hkv} d={w.d} W={w.W} n={n[:4]}",
          file=sys.stderr, flush=True)
    keep_host = not args.no_cpu_baseline
    prefill = args.score_queries == "prefill"
    dv, host = upload_layers(w, range(w.L), dev, keep_host=keep_host, prefill=prefill)
    sched = {"parabolic": vc.VC_SCHED_PARABOLIC, "fixed": vc.VC_SCHED_FIXED,
             "arithmetic": vc.VC_SCHED_ARITHMETIC, "geometric": vc.VC_SCHED_GEOMETRIC}[args.schedule]
    params = vc.make_params(w.retention, rank_mode=mode, schedule=sched, drop_all=args.drop_all,
                            score_queries=vc.VC_SCORE_PREFILL if prefill else vc.VC_SCORE_WINDOW)
    pc = PruneCall(w.B, w.L, w.Hq, w.Hkv, w.d, w.W, n, params, [dv["K"][l] for l in range(w.L)],
                   [dv["V"][l] for l in range(w.L)], [dv["Q"][l] for l in range(w.L)],
                   k_text=[dv["KT"][l] for l in range(w.L)] if prefill else None)
    # Flush by reading (not writing) 1 GiB, so the caches hold clean lines and
    # the measured kernels pay no write-back of the flush data.
    # (float32: a sum of int32 would be widened to int64 first, writing 2 GiB.)
    flush = None if args.no_flush else torch.ones(1 << 28, dtype=torch.float32, device=dev)
    print(f"[bench] timing {args.steps} prune steps after {args.warmup} warm-up", file=sys.stderr, flush=True)
    tot, stage, wall = time_prune(pc, args.steps, args.warmup, flush, torch)
    ms = sum(tot) / len(tot)
    in_bytes = sum(w.Hkv * x * w.d * 2 * 2 for x in n) * w.L
    alg = algorithmic(w, pc, n, prefill)
    stage_us = {STAGES[i]: 1e3 * sum(s[i] for s in stage) / len(stage) for i in range(6)}
    dom = max(("score_stats", "score_colsum", "select", "gather_fuse"), key=lambda s: stage_us[s])
    a = alg[dom]
    t = stage_us[dom] * 1e-6
    fr_hbm = a["bytes"] / t / 1e9 / HBM_PEAK_GBS
    fr_mfma = a["flops"] / t / 1e12 / MFMA_BF16_PEAK_TFLOPS
    if fr_mfma >= fr_hbm:
        roof = dict(bound="mfma", achieved=a["flops"] / t / 1e12, peak=MFMA_BF16_PEAK_TFLOPS, unit="TFLOP/s")
    else:
        roof = dict(bound="hbm", achieved=a["bytes"] / t / 1e9, peak=HBM_PEAK_GBS, unit="GB/s")
    roof["frac"] = roof["achieved"] / roof["peak"]
    kernels = PREFILL_STAGE_KERNEL if prefill else STAGE_KERNEL
    roof["traffic"] = stored_traffic(dom, kernels)
    roof["kernel"] = kernels[dom][0]
    roof["stage"] = dom
    roof["kernel_us"] = stage_us[dom]
    roof["hbm_frac"] = fr_hbm
    roof["mfma_frac"] = fr_mfma
    roof["exp_per_s"] = a["exps"] / t

    if args.copy_probe:
        copy_probe(torch, dev)
    dec = None
    if not args.no_decode:
        dsteps = args.decode_steps or w.decode_steps
        print(f"[bench] decode: {dsteps} steps x 4 caches", file=sys.stderr, flush=True)
        dec = decode_latency(w, pc, dev, dsteps, flush, torch, sg)
    cpu = None
    if not args.no_cpu_baseline:
        print(f"[bench] CPU oracle ({args.cpu_units or 'all'} units)", file=sys.stderr, flush=True)
        cpu = cpu_baseline(w, pc, host, args.cpu_units, prefill)

    rec = {
        "metric": "PruneKV compress GB/s (% of HBM peak) + decode-attn speedup vs full KV",
        "value": in_bytes / (ms * 1e-3) / 1e9,
        "unit": "GB/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"{w.name}: B={w.B} L={w.L} Hq={w.Hq} Hkv={w.Hkv} d={w.d} "
                               f"{w.frames}x{w.tokens_per_frame} visual tokens, W={w.W}, RR={w.retention}",
                   "rank_mode": args.rank_mode, "schedule": args.schedule, "drop_all": args.drop_all,
                   "score_queries": args.score_queries,
                   "cold_caches": flush is not None,
                   "input_visual_kv_bytes": in_bytes},
        "hbm_frac_path": alg["path_bytes"] / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
        "path_alg_bytes": alg["path_bytes"],
        "stage_us": stage_us,
        "ms_per_step_median": sorted(tot)[len(tot) // 2],
        "wall_s_timed_region": wall,
        "roofline": roof,
        "decode": dec,
        "cpu_baseline": cpu,
    }
    print(json.dumps(rec))


if __name__ == "__main__":
    main()
