"""Host checks of bench.py: the byte model behind the roofline figure and the
one-GPU contract.

The algorithmic bytes of a launch are re-derived here from the sizes of the
arrays the workload actually holds (numpy nbytes), not from the bench's own
formula, so that a dropped or doubled tensor in the bench shows up."""
import os
import subprocess
import sys

import numpy as np
import pytest

from paper_2607_06763_amd import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def _path_nodes(w):
    """Nodes on the accepted root-to-node paths (the commit's inputs)."""
    n = 0
    for b in range(w.B):
        a = int(w.accepted[b])
        while a >= 0:
            n += 1
            a = int(w.parent[b, a])
    return n


@pytest.mark.parametrize("cfg", [0, 3, 4])
def test_algorithmic_bytes_from_array_sizes(cfg):
    w = W.make_config(cfg)
    nodes = w.B * w.T
    out = 4 * nodes * w.Hv * w.dv                      # fp32 outputs, one row per node and head
    meta = 4 * 4 * nodes + 2 * 4 * w.B                 # order, depth, parent, position; status, count
    verify = (w.S0.nbytes + w.q.nbytes + w.k.nbytes + w.v.nbytes + w.alpha.nbytes + w.beta.nbytes
              + w.conv_state.nbytes + w.conv_w.nbytes + meta + out)
    # commit: state and conv state read and written; raw q / k / v and the two
    # gates of every node on the accepted paths; conv weights; the metadata
    # it reads (ancestor words of the accepted nodes are within 8 B per slot)
    L = _path_nodes(w)
    row = (w.q.nbytes + w.k.nbytes + w.v.nbytes) // nodes
    gates = (w.alpha.nbytes + w.beta.nbytes) // nodes
    commit = (2 * w.S0.nbytes + 2 * w.conv_state.nbytes + L * (row + gates) + w.conv_w.nbytes
              + 8 * nodes + 8 * w.B)
    # the fused step reads S, the conv state and the conv weights once
    step = verify + commit - w.S0.nbytes - w.conv_state.nbytes - w.conv_w.nbytes
    got = bench.algorithmic_bytes(w)
    assert got["verify"] == verify
    assert got["commit"] == commit
    assert got["step"] == step
    if cfg == 4:  # the headline figures quoted with the roofline
        assert got["step"] == 401_673_152
        assert got["verify"] == 290_160_896


def test_bench_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120, cwd=ROOT)
    assert r.returncode == 2
    assert "exactly one GPU" in r.stderr
    assert r.stdout.strip() == ""


def test_traffic_is_gated_on_the_kernel_source():
    """The HBM bytes quoted with the roofline come from the committed counter
    summary only while it was taken on the current verify / step source."""
    h = bench.verify_source_hash()
    got = bench.measured_traffic(h, "step", "large")
    with open(os.path.join(ROOT, "profiles", "step_large_hbm_traffic.md")) as f:
        text = f.read()
    if f"`{h}`" in text:
        assert got is not None and 4.0e8 < got < 4.6e8   # 1.0-1.15 x the 401.7 MB of the step
    else:
        assert got is None
    assert bench.measured_traffic("0" * 16, "step", "large") is None
    gv = bench.measured_traffic(h, "verify", "large")
    assert gv is None or 2.9e8 < gv < 3.35e8             # 1.0-1.15 x the 290.2 MB of the verify
