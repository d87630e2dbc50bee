"""The host code of libviscache (argument checks, budgets, plan layout and
packing, decode planning) and the oracle, built with the address and
undefined-behaviour sanitizers and run on the CPU over the five workload
shapes, ragged batches and edge shapes (tests/sanitize/host_driver.cpp).  The
kernel launchers are host stubs, so nothing here needs a GPU; every status
the sanitized build returns must equal the regular library's."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2608_24063_amd", "csrc")
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer", "-g", "-O1"]


def _cases(sg):
    """(B, L, Hq, Hkv, d, W, rr, h, m, rank_mode, v_out_fp32, schedule, drop_all, score_queries, n_vis)."""
    out = []
    for w in sg.WORKLOADS.values():
        n = [int(x) for x in w.n_vis()]
        for mode in (0, 1):
            for sq in (0, 1):
                out.append((w.B, w.L, w.Hq, w.Hkv, w.d, w.W, w.retention, 0, 0.75, mode, mode, 0, 0, sq, n))
        out.append((w.B, w.L, w.Hq, w.Hkv, w.d, w.W, w.retention, 0, 0.75, 0, 0, 3, 1, 0, n))
    edge = [
        (5, 4, 6, 2, 64, 5, 0.25, 0, 0.75, 0, 1, 0, 0, 0, [0, 130, 7, 0, 64]),   # empty and ragged sequences
        (3, 2, 16, 1, 128, 64, 0.25, 0, 0.75, 1, 0, 1, 0, 0, [32768, 1, 0]),    # the longest sequence
        (1, 2, 16, 1, 128, 64, 0.25, 0, 0.75, 0, 0, 0, 0, 0, [32769]),         # one token too many
        (1, 3, 8, 2, 64, 4, 1.0, 3, 1.0, 0, 0, 0, 0, 0, [64]),                 # keep-all
        (1, 4, 8, 2, 64, 4, 0.9, 0, 0.75, 0, 0, 0, 0, 0, [64]),                # q > 1
        (1, 4, 8, 2, 96, 4, 0.25, 0, 0.75, 0, 0, 0, 0, 0, [64]),               # unsupported head dim
        (1, 4, 64, 2, 64, 40, 0.25, 0, 0.75, 0, 0, 0, 0, 0, [64]),             # G*W = 1280 window rows
        (2, 80, 64, 8, 128, 128, 0.22, 0, 0.75, 1, 0, 2, 0, 0, [8192, 4000]),  # 72B-shaped, ragged
        (1, 2, 4096, 4096, 64, 1, 1.0, 2, 1.0, 0, 0, 0, 0, 0, [4]),            # 8192 fusion units
        (2000, 2, 8, 2, 64, 4, 0.25, 0, 0.75, 0, 0, 0, 0, 0, [3] * 2000),      # plan beyond the first chunk
        (2600, 2, 8, 2, 64, 4, 0.25, 0, 0.75, 0, 0, 0, 0, 0, [3] * 2600),      # tables too long (refused)
    ]
    return out + edge


def _expected(vc, case):
    B, L, Hq, Hkv, d, W, rr, h, m, mode, vf, sched, da, sq, n = case
    p = vc.make_params(rr, h=h, m=m, rank_mode=mode, v_out_fp32=vf, schedule=sched, drop_all=da, score_queries=sq)
    try:
        vc.viscache_budget(vc.make_shape(B, L, Hq, Hkv, d, W, n), p)
    except vc.VisCacheError as e:
        return e.status
    return vc.VC_OK


@pytest.mark.timeout(900)
def test_host_code_under_sanitizers(tmp_path, sg):
    gxx, gcc = shutil.which("g++"), shutil.which("gcc")
    if not gxx or not gcc:
        pytest.skip("no host compiler")
    import paper_2608_24063_amd as vc
    if not os.path.exists(vc.LIB_PATH):
        from paper_2608_24063_amd import build
        build.build()
    vc.lib()
    inc = ["-I", os.path.join(ROOT, "include"), "-I", "/opt/rocm/include", "-D__HIP_PLATFORM_AMD__"]
    objs = []
    for src in (os.path.join(CSRC, "vc_api.cpp"), os.path.join(CSRC, "vc_budget.cpp"),
                os.path.join(CSRC, "vc_decode_plan.cpp"),
                os.path.join(ROOT, "tests", "sanitize", "launch_stubs.cpp"),
                os.path.join(ROOT, "tests", "sanitize", "host_driver.cpp")):
        obj = str(tmp_path / (os.path.basename(src) + ".o"))
        # the budget rule's double expressions round as written (as in the library build)
        subprocess.check_call([gxx, "-std=c++17", "-ffp-contract=off"] + SAN + inc + ["-c", src, "-o", obj])
        objs.append(obj)
    obj = str(tmp_path / "oracle.o")
    subprocess.check_call([gcc, "-std=c11", "-ffp-contract=off", "-fno-fast-math"] + SAN +
                          ["-c", os.path.join(ROOT, "oracle", "oracle.c"), "-o", obj])
    objs.append(obj)
    exe = str(tmp_path / "host_driver")
    subprocess.check_call([gxx] + SAN + objs + ["-o", exe, "-L/opt/rocm/lib", "-lamdhip64", "-lm",
                                                "-Wl,-rpath,/opt/rocm/lib"])
    cases = _cases(sg)
    cf = tmp_path / "cases.txt"
    cf.write_text("\n".join(" ".join(str(x) for x in c[:14]) + " " + " ".join(str(x) for x in c[14])
                            for c in cases) + "\n")
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0:halt_on_error=1:exitcode=99",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1",
               LSAN_OPTIONS=f"suppressions={os.path.join(ROOT, 'tests', 'sanitize', 'lsan.supp')}")
    r = subprocess.run([exe, str(cf)], capture_output=True, text=True, env=env, timeout=800)
    assert r.returncode == 0, f"rc {r.returncode}\n{r.stdout[-2000:]}\n{r.stderr[-4000:]}"
    assert "runtime error" not in r.stderr and "Sanitizer" not in r.stderr, r.stderr[-4000:]
    got = {}
    for line in r.stdout.splitlines():
        if line.startswith("case "):
            _, i, st = line.split()
            got[int(i)] = int(st)
    assert len(got) == len(cases) and "oracle ok" in r.stdout
    for i, c in enumerate(cases):
        assert got[i] == _expected(vc, c), f"case {i}: {got[i]} vs {_expected(vc, c)}"
