"""The host part of the library -- planner and band executor -- built with
AddressSanitizer and UndefinedBehaviorSanitizer (g++, host code only) and
driven through its C ABI in dry-run mode: every schedule (forward, backward
with and without dx, layer-wise) of the five benchmark workloads, random
small networks and partitions, every policy, backward refinement, hybrid
depth, the budget search and planner error paths. A dry run walks the whole
band schedule with all host-side checks but launches nothing (the GPU
launchers are replaced by stubs that abort if reached), so the run needs no
GPU; the sanitizers report any out-of-bounds access, use after free, leak
or undefined behaviour in the host code."""
import os
import shutil
import subprocess
from pathlib import Path

import numpy as np
import pytest

from paper_2401_11471_amd import lrcnn as L
from workloads import CONFIGS, NetBuilder, net_nodes

ROOT = Path(__file__).resolve().parent.parent
CSRC = ROOT / "paper_2401_11471_amd" / "csrc"
HERE = Path(__file__).resolve().parent / "asan"


def _line(nodes, batch, h, w, dtype, mode, nb, policy=L.EVEN, refine=1, hybrid=0, first=0,
          bounds=(), expect=0, c=3):
    vals = [len(nodes)]
    for nd in nodes:
        vals += list(nd)
    vals += [batch, c, h, w, dtype, mode, nb, policy, refine, hybrid, first, len(bounds),
             *bounds, expect]
    return " ".join(str(int(v)) for v in vals)


def _random_chain(rng):
    nb = NetBuilder()
    v = 0
    for _ in range(int(rng.integers(2, 6))):
        if rng.random() < 0.25:
            k = int(rng.integers(2, 4))
            v = nb.pool(v, k, int(rng.integers(1, 3)), int(rng.integers(0, k)) // 2)
        else:
            k = int(rng.integers(1, 6))
            v = nb.conv(v, int(rng.integers(1, 9)), k, int(rng.integers(1, 3)),
                        int(rng.integers(0, k)), affine=int(rng.integers(0, 2)),
                        relu=int(rng.integers(0, 2)))
    return nb.nodes


def cases():
    out = []
    for cid in (1, 2, 3, 4, 5):
        c = CONFIGS[cid]
        nodes = net_nodes(c["net"])
        args = (nodes, c["batch"], c["h"], c["w"], c["dtype"])
        out.append(_line(*args, L.CARRY, c["bands"]))
        out.append(_line(*args, L.CARRY, c["bands"], refine=2))
        out.append(_line(*args, L.CARRY, c["bands"], L.PAPER_2PS))
        out.append(_line(*args, L.RECOMPUTE, c["bands"]))
        if cid in (1, 2, 3):
            out.append(_line(*args, L.CARRY, c["bands"], L.BALANCED))
            out.append(_line(*args, L.CARRY, c["bands"], hybrid=L.HYBRID_AUTO))
    rng = np.random.default_rng(1)
    made = 0
    while made < 40:
        nodes = _random_chain(rng)
        h = int(rng.integers(20, 60))
        try:
            L.lrcnn_plan(nodes, 1, 3, h, 9)
        except L.LrcnnError:
            continue  # a layer with no output at this size
        made += 1
        nb = int(rng.integers(1, 6))
        cuts = sorted(rng.integers(0, h + 1, nb - 1).tolist())
        dt = int(rng.integers(0, 2))
        mode = int(rng.integers(0, 2))
        if mode == L.RECOMPUTE:
            # RECOMPUTE bands partition the last node's rows
            ho = L.lrcnn_plan(nodes, 1, 3, h, 9).node_shape(len(nodes) - 1)[0]
            cuts = sorted(rng.integers(0, ho + 1, nb - 1).tolist())
            out.append(_line(nodes, 2, h, 9, dt, mode, nb, L.EXPLICIT, bounds=[0, *cuts, ho]))
        else:
            out.append(_line(nodes, 2, h, 9, dt, mode, nb, L.EXPLICIT, bounds=[0, *cuts, h]))
        out.append(_line(nodes, 1, h, 9, dt, L.CARRY, nb, L.PAPER_2PS,
                         first=int(rng.integers(0, 4)), refine=int(rng.integers(1, 3))))
    tiny = net_nodes("tiny")
    out.append(_line(tiny, 1, 32, 32, L.F32, L.CARRY, 2, L.EXPLICIT, bounds=[0, 20, 10],
                     expect=-3))
    out.append(_line(tiny, 1, 32, 32, L.F32, L.RECOMPUTE, 2, L.PAPER_2PS, expect=-1))
    out.append(_line(tiny, 1, 32, 32, L.F32, L.CARRY, 0, expect=-3))
    out.append(_line(tiny, 1, 32, 32, 9, L.CARRY, 2, expect=-6))
    return out


@pytest.mark.skipif(shutil.which("g++") is None, reason="g++ not available")
def test_sanitized_planner_and_executor_dry_run(tmp_path):
    exe = tmp_path / "asan_dry"
    srcs = [CSRC / "plan.cpp", CSRC / "exec.cpp", HERE / "launch_stubs.cpp",
            HERE / "dry_run_main.cpp"]
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined",
           "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer",
           "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include", f"-I{ROOT / 'include'}",
           f"-I{CSRC}", *map(str, srcs), "-L/opt/rocm/lib", "-lamdhip64",
           "-Wl,-rpath,/opt/rocm/lib", "-o", str(exe)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    env.pop("LD_PRELOAD", None)
    data = "\n".join(cases()) + "\n"
    r = subprocess.run([str(exe)], input=data, capture_output=True, text=True, env=env,
                       timeout=900)
    assert r.returncode == 0, (r.stdout[-3000:], r.stderr[-6000:])
    assert "failures 0" in r.stdout
