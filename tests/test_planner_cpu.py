"""The dispatch planners' choices and invariants, on the CPU.

tests/planner_probe.hip includes the library's dispatch source and prints
the split plan of the large-M kernel (plan_splits) and the few-row
streaming kernel's plan (stream_plan) for calls given as text.  Checked here:

* invariants every plan must keep for the kernels to be correct: parts of
  whole scale groups (4 steps of 64 k, or 8-block groups for the streaming
  kernel), no empty part, every step covered, at most 4 parts summed in the
  kernel and 16 by the separate launch, no split of a layer with a tile for
  every CU;
* the plans the design documents for its workloads: the q4 step block
  unsplit; single 128-tile layers at 2048 tokens in 2 parts (summed by the
  separate launch with an epilogue, in the kernel without); a d = 1024
  block at 768 tokens summed in the kernel with FFN-down in 4 parts; the
  paper widths at 214 tokens summed by the separate launch.

The probe is built with hipcc against the library's objects (built by
`python -m paper_2607_08526_amd.build`); without a GPU the planners assume
the 256 compute units of the target part.
"""
import os
import shutil
import subprocess

import numpy as np
import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
BUILD = os.path.join(ROOT, "paper_2607_08526_amd", "_build")
CUS = 256
INT8, Q4 = 8, 4


@pytest.fixture(scope="module")
def probe(tmp_path_factory):
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    if not os.path.exists(hipcc):
        pytest.skip("hipcc is not available")
    objs = [os.path.join(BUILD, f) for f in sorted(os.listdir(BUILD))
            if f.endswith(".o") and f != "qlinear.o"] if os.path.isdir(BUILD) else []
    if not objs:
        pytest.fail("library objects missing: run `python -m paper_2607_08526_amd.build`")
    out = tmp_path_factory.mktemp("probe")
    obj, exe = str(out / "probe.o"), str(out / "probe")
    flags = ["--offload-arch=gfx950", "-O1", "-std=c++17", f"-I{os.path.join(ROOT, 'include')}",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
    for cmd in ([hipcc, *flags, "-c", os.path.join(HERE, "planner_probe.hip"), "-o", obj],
                [hipcc, "--offload-arch=gfx950", "-o", exe, obj, *objs]):
        r = subprocess.run(cmd, capture_output=True, text=True)
        assert r.returncode == 0, r.stderr[-2000:]

    def run(lines):
        r = subprocess.run([exe], input="\n".join(lines) + "\n", capture_output=True, text=True,
                           timeout=120)
        assert r.returncode == 0, r.stderr[-2000:]
        return [l.split() for l in r.stdout.strip().splitlines()]
    return run


def wide_plans(probe, calls):
    """calls: (fmt, epi, M, [(N, K), ...]) -> [(ext, [(K, tiles, S, psteps), ...])]"""
    out = probe([f"wide {f} {int(e)} {M} " + " ".join(f"{N} {K}" for N, K in ls)
                 for f, e, M, ls in calls])
    res = []
    for t in out:
        assert t[0] == "wide"
        v = list(map(int, t[2:]))
        res.append((int(t[1]), [tuple(v[i:i + 4]) for i in range(0, len(v), 4)]))
    return res


def block(d):
    return [(3 * d, d), (d, d), (4 * d, d), (d, 4 * d)]


def test_wide_plans_keep_the_kernel_invariants(probe):
    rng = np.random.default_rng(0)
    calls = []
    for _ in range(300):
        M = int(rng.integers(65, 4097))
        fmt, epi = int(rng.choice([INT8, Q4])), bool(rng.integers(0, 2))
        if rng.random() < 0.5:
            d = 256 * int(rng.integers(1, 13))
            calls.append((fmt, epi, M, block(d)))
        else:
            n = int(rng.integers(1, 5))
            calls.append((fmt, epi, M, [(int(rng.integers(1, 65)) * 64,
                                         256 * int(rng.integers(1, 33))) for _ in range(n)]))
    for (fmt, epi, M, ls), (ext, layers) in zip(calls, wide_plans(probe, calls)):
        for K, tiles, S, ps in layers:
            ns = K // 64
            what = (fmt, epi, M, ls, ext, K, S, ps)
            assert S >= 1 and ps >= 1, what
            assert (S - 1) * ps < ns <= S * ps, what        # every step, no empty part
            if S > 1:
                assert ps % 4 == 0, what                     # whole scale groups
                assert S <= (16 if ext else 4), what         # sum launch / in-kernel bound
                assert tiles < CUS, what                     # a tile per CU: never split
        assert ext in (0, 1)


def test_wide_plans_of_the_documented_workloads(probe):
    step, single_epi, single_plain, qkv, mid, widths = wide_plans(probe, [
        (Q4, False, 2048, block(2048)),
        (Q4, True, 2048, [(2048, 8192)]),
        (Q4, False, 2048, [(2048, 2048)]),
        (Q4, True, 2048, [(6144, 2048)]),
        (Q4, True, 768, block(1024)),
        (Q4, False, 214, block(1024)),
    ])
    assert all(S == 1 for _, _, S, _ in step[1])           # the step block: unsplit
    assert single_epi == (1, [(8192, 128, 2, 64)])        # FFN-down alone, epilogue
    assert single_plain == (0, [(2048, 128, 2, 16)])      # out-projection alone, plain
    assert qkv[1][0][2] == 1                              # 384 tiles: whole
    assert mid[0] == 0 and [S for _, _, S, _ in mid[1]] == [4, 2, 2, 2]
    assert widths[0] == 1 and widths[1][0][:3] == (4096, 8, 8)


def test_stream_plans_keep_the_kernel_invariants(probe):
    rng = np.random.default_rng(1)
    calls = []
    for _ in range(200):
        M = int(rng.integers(1, 33))
        fmt = int(rng.choice([INT8, Q4]))
        n = int(rng.integers(1, 5))
        ls = [(int(rng.integers(1, 257)) * 32, 256 * int(rng.integers(1, 49))) for _ in range(n)]
        calls.append((fmt, M, ls))
    out = probe([f"stream {f} {M} " + " ".join(f"{N} {K}" for N, K in ls) for f, M, ls in calls])
    for (fmt, M, ls), t in zip(calls, out):
        assert t[0] == "stream"
        rw, kw, mx = map(int, t[1:4])
        assert rw in (8, 16, 32, 64) and kw in (2, 4, 8) and M <= mx <= 32, (t, M)
        v = list(map(int, t[4:]))
        for K, S, pb in (v[i:i + 3] for i in range(0, len(v), 3)):
            nb = K // 32
            what = (fmt, M, ls, t)
            assert 1 <= S <= 16, what
            assert pb % 8 == 0 and pb >= 8 * kw or S == 1, what
            assert (S - 1) * pb < nb <= S * pb or (S == 1 and pb >= nb), what


def test_stream_plans_of_the_documented_workloads(probe):
    # the grouped d = 2048 block (QKV, out, FFN-up, FFN-down) at few rows:
    # int8 at M = 8 must not take 8-row workgroups, which tie with wider
    # ones in round trips but re-read the activations twice as often (the
    # plan's byte floor separates them); q4 at M = 8 keeps its 32-row plan
    lay = [(6144, 2048), (2048, 2048), (8192, 2048), (2048, 8192)]
    out = probe([f"stream {f} {M} " + " ".join(f"{N} {K}" for N, K in lay)
                 for f, M in ((INT8, 8), (Q4, 8), (INT8, 32))])
    i8, q4, i8_32 = ([int(x) for x in t[1:4]] for t in out)
    assert i8[0] >= 16 and i8[2] == 8, out[0]
    assert q4[0] == 32 and q4[2] == 8, out[1]
    assert i8_32[0] == 32 and i8_32[2] == 32, out[2]
