"""The executor's stream / event schedule checked on the CPU as a HIP graph
capture of one training step would record it (forward then backward on one
origin stream). The planner and executor are built with g++ (sanitizers
on) against stand-ins for the GPU launchers and the HIP stream calls that
record every launch, event record and stream wait (tests/streams); the
recorded trace must satisfy the capture rules: a second stream joins only
by waiting for an event recorded in the capture and issues nothing before
that, every awaited event was recorded earlier in the same capture, and all
of a forked stream's work is joined back into the origin stream by the end.
The forward launches also carry their footprints (the rows of every buffer
they read or write): no two of them on different streams that the events
leave unordered may touch the same bytes with one of them writing, and none
may reach past its buffer.
Covered: the weight-gradient side stream of the backward, and the opt-in
forward pass pipelined over bands on two streams, at the five workloads
(with the step presets of the 224-pixel ones) and on small nets."""
import os
import re
import shutil
import subprocess
from pathlib import Path

import pytest

from paper_2401_11471_amd import lrcnn as L
from workloads import CONFIGS, net_nodes

ROOT = Path(__file__).resolve().parent.parent
CSRC = ROOT / "paper_2401_11471_amd" / "csrc"
HERE = Path(__file__).resolve().parent / "streams"


def _line(nodes, batch, h, w, dtype, mode, nb, policy=L.EVEN, refine=1, hybrid=0, pipe=0, c=3):
    vals = [len(nodes)]
    for nd in nodes:
        vals += list(nd)
    vals += [batch, c, h, w, dtype, mode, nb, policy, refine, hybrid, 0, 0, pipe]
    return " ".join(str(int(v)) for v in vals)


def cases():
    out = []
    for cid in (1, 2, 3, 4, 5):
        c = CONFIGS[cid]
        nodes = net_nodes(c["net"])
        args = (nodes, c["batch"], c["h"], c["w"], c["dtype"])
        for pipe in (0, 1, 3):
            out.append(_line(*args, L.CARRY, c["bands"], pipe=pipe))
            if "step" in c:
                s = c["step"]
                out.append(_line(*args, L.CARRY, c["bands"], s["policy"], s["bp_refine"],
                                 L.HYBRID_AUTO if s["hybrid_from"] < 0 else s["hybrid_from"],
                                 pipe=pipe))
        out.append(_line(*args, L.RECOMPUTE, c["bands"]))
    return out


@pytest.fixture(scope="module")
def checker(tmp_path_factory):
    if shutil.which("g++") is None:
        pytest.skip("g++ not available")
    exe = tmp_path_factory.mktemp("streams") / "trace_check"
    srcs = [CSRC / "plan.cpp", CSRC / "exec.cpp", HERE / "trace_stubs.cpp",
            HERE / "trace_main.cpp"]
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined",
           "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer",
           "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include", f"-I{ROOT / 'include'}",
           f"-I{CSRC}", f"-I{HERE}", *map(str, srcs), "-o", str(exe)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    return exe


def _run(exe, lines):
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    env.pop("LD_PRELOAD", None)
    return subprocess.run([str(exe)], input="\n".join(lines) + "\n", capture_output=True,
                          text=True, env=env, timeout=900)


def test_captured_step_schedule_is_joined_and_ordered(checker):
    r = _run(checker, cases())
    assert r.returncode == 0, (r.stdout[-4000:], r.stderr[-4000:])
    assert "failures 0" in r.stdout
    # the pipelined forward does put bands on a second stream
    piped = [l for l in r.stdout.splitlines() if "side" in l]
    assert piped, r.stdout[-2000:]


def test_block_outputs_need_no_separate_window_initialisation(checker):
    # ResNet-50 bf16 at 2400x3600, 32 CARRY bands: each residual block's
    # output window (the add's rows plus the row carried in from the band
    # above) is stored by the add's backward, so the separate zeroing and
    # carry copy-in launches are not one per block and band (16 blocks x 32
    # bands alone would be 512; the step makes 186)
    c = CONFIGS[5]
    line = _line(net_nodes(c["net"]), c["batch"], c["h"], c["w"], c["dtype"], L.CARRY,
                 c["bands"])
    r = _run(checker, [line])
    assert r.returncode == 0, (r.stdout[-4000:], r.stderr[-4000:])
    assert "failures 0" in r.stdout
    inits = [int(m) for m in re.findall(r"inits (\d+)", r.stdout)]
    assert inits and max(inits) < 16 * c["bands"], r.stdout[-2000:]


def _planted(tmp_path, old, new, name):
    # the executor with a mistake planted on the CPU, built against the stubs
    src = (CSRC / "exec.cpp").read_text()
    assert old in src
    bad = tmp_path / f"exec_{name}.cpp"
    bad.write_text(src.replace(old, new))
    exe = tmp_path / f"trace_{name}"
    srcs = [CSRC / "plan.cpp", bad, HERE / "trace_stubs.cpp", HERE / "trace_main.cpp"]
    cmd = ["g++", "-std=c++17", "-O1", "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include",
           f"-I{ROOT / 'include'}", f"-I{CSRC}", f"-I{HERE}", *map(str, srcs), "-o", str(exe)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    c = CONFIGS[3]
    # the pipelined forward alone (flag 3) of the ResNet-50 workload at 224 px
    return _run(exe, [_line(net_nodes("resnet50"), c["batch"], c["h"], c["w"], c["dtype"],
                            L.CARRY, c["bands"], pipe=3)])


def test_checker_finds_an_unjoined_fork(checker, tmp_path):
    # without the forward's final join the side stream's last band is left
    # outside the origin stream's order
    r = _planted(tmp_path,
                 'LAUNCH(hipStreamWaitEvent(sides[0], (hipEvent_t)evs[(rs & 1) * P.n + P.n - 1], 0),',
                 'LAUNCH(0 * (int)(uintptr_t)(evs[(rs & 1) * P.n + P.n - 1]),', "unjoined")
    assert r.returncode != 0
    assert "work after its last join" in r.stdout


def test_checker_finds_a_missing_band_wait(checker, tmp_path):
    # without the waits for the previous band, band r overwrites windows
    # band r - 1 still reads on the other stream
    r = _planted(tmp_path, "if (!pipe || !ev_prev) return LRCNN_OK;", "return LRCNN_OK;",
                 "nowait")
    assert r.returncode != 0
    assert "race:" in r.stdout
