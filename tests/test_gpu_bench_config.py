"""GPU parity in the launch configuration bench.py times.

The benchmark's step is the save-for-backward pair on the lm-bf16 workload,
pipelined over eight input sets (step i: forward of set i mod 8, backward of
set (i - 2) mod 8, one saved-state buffer per set), captured in a HIP graph
and replayed.  Here the same runner (bench.ScanRunner) runs eagerly and under
graph capture, and:

* after eager steps, the forward's Y of the newest set and the backward's
  outputs of the set two steps older are checked against the float64 oracle
  on sampled heads (all batch rows), which also checks that the rotating
  saved-state buffers pair every backward with its own forward;
* a graph of the same steps is replayed three times, with eager work and
  synchronisations between the replays, and every replay's outputs must
  equal the eager run of the same steps bitwise (the kernels reduce in a
  fixed order).
"""

import os
import sys

import pytest

from oracle import gradlev_oracle as orc
from paper_2609_34174_amd import workloads as W
from parity_util import check, log, to_host

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

import paper_2609_34174_amd as gl  # noqa: E402

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)
import bench  # noqa: E402


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.fail("no ROCm GPU visible")
    gl.lib()
    yield
    torch.cuda.synchronize()


@pytest.fixture(scope="module")
def runner():
    wl = W.SCAN_WORKLOADS["lm-bf16"]
    log("building the benchmark's pipelined runner (8 input sets, saved pair)")
    run = bench.ScanRunner(gl, torch, W, wl, 8, torch.device("cuda:0"), saved=True, pipelined=True)
    yield wl, run
    del run
    torch.cuda.empty_cache()


def _snapshot(run):
    torch.cuda.synchronize()
    out = {k: v.clone() for k, v in run.outs.items()}
    out["y"] = run.Y.clone()
    return out


@pytest.mark.timeout(300)
def test_pipelined_steps_match_oracle(runner):
    wl, run = runner
    n = len(run.sets)
    last = 11  # past one full rotation of the saved-state buffers
    log(f"eager pipelined steps 0..{last}")
    for i in range(last + 1):
        run.step(i)
    got = _snapshot(run)
    fset, bset = run.sets[last % n], run.sets[(last - run.LAG) % n]

    def eta_of(s, h):
        e = s["eta"]
        return to_host(e[:, h:h + 1]) if isinstance(e, torch.Tensor) else e

    for h in (3, 12):
        log(f"  oracle: forward of set {last % n}, backward of set {(last - run.LAG) % n}, head {h}")
        fs = {k: to_host(fset[k][:, h:h + 1]) for k in ("X", "G")}
        y_ref = orc.scan_fwd(to_host(fset["W0"][h:h + 1]), fs["X"], fs["G"], eta_of(fset, h))
        check("y", to_host(got["y"][:, h:h + 1]), y_ref, "bf16")
        bs = {k: to_host(bset[k][:, h:h + 1]) for k in ("X", "G", "dY")}
        ref = orc.scan_bwd(to_host(bset["W0"][h:h + 1]), bs["X"], bs["G"], eta_of(bset, h), bs["dY"])
        for k in ("gtilde", "dx", "dg", "deta"):
            check(k, to_host(got[k][:, h:h + 1]), ref[k], "bf16")
        check("dw0", to_host(got["dw0"][h:h + 1]), ref["dw0"], "bf16")


@pytest.mark.timeout(300)
def test_graph_replays_match_eager(runner):
    wl, run = runner
    steps = list(range(20, 26))
    log("eager reference of steps 20..25")
    for i in steps:
        run.step(i)
    ref = _snapshot(run)
    log("capturing the same steps in a HIP graph")
    stream = torch.cuda.Stream()
    stream.wait_stream(torch.cuda.current_stream())
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.stream(stream):
        with torch.cuda.graph(graph, stream=stream):
            for i in steps:
                run.step(i)
    torch.cuda.current_stream().wait_stream(stream)
    for rep in range(3):
        # Eager work in between: other steps overwrite the shared outputs.
        for i in range(30, 33):
            run.step(i)
        torch.cuda.synchronize()
        graph.replay()
        got = _snapshot(run)
        log(f"  replay {rep}: comparing with the eager run")
        for k in ref:
            assert torch.equal(got[k], ref[k]), f"replay {rep}: {k} differs from the eager run"
    del graph
