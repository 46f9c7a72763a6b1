"""bench.py's contract on the host (no GPU): the one-GPU refusal, the algorithmic bytes the
roofline divides by, and the counter-derived traffic that follows the kernels' sources."""
import os
import shutil
import subprocess
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from workloads import HEADLINE, gen  # noqa: E402


def test_more_than_one_gpu_is_refused():
    out = subprocess.run([sys.executable, "bench.py", "--gpus", "2"], cwd=ROOT, capture_output=True,
                         text=True, timeout=300)
    assert out.returncode != 0
    assert "one GPU" in out.stderr
    assert out.stdout.strip() == ""


def test_encode_bytes_are_the_transmitted_rows():
    """At the headline the encode's compulsory bytes are the transmitting rows of T (4 L
    bytes each) plus inputs read once, which add well under 1%."""
    wl, ell = HEADLINE, 1
    psi = gen.psi(wl)
    sent = int((psi > 0).sum())
    ab = bench.algorithmic_bytes(wl, ell, wl.P, sent)
    t_bytes = 4 * sent * wl.d
    assert t_bytes <= ab["gc_encode"] < 1.01 * t_bytes
    assert t_bytes <= ab["gc_reconstruct"] < 1.05 * t_bytes  # + the estimate, 4 d per pattern
    assert 0 < sent < wl.P * wl.m  # the stragglers' rows are not counted


def test_traffic_follows_the_kernel_sources(tmp_path, monkeypatch):
    """roofline.traffic comes from the counter summary (profiles/hbm_traffic_<workload>.txt)
    only while the counted kernel's sources hash to what they were when the counters were
    taken; here a summary written for the current sources, then one source edited."""
    import hashlib
    import json
    csrc = tmp_path / "paper_2405_19509_amd" / "csrc"
    shutil.copytree(os.path.join(ROOT, "paper_2405_19509_amd", "csrc"), csrc)
    (tmp_path / "profiles").mkdir()

    def sha(files):
        h = hashlib.sha256()
        for f in files:
            h.update(open(tmp_path / f, "rb").read())
        return h.hexdigest()[:16]

    kernels = {}
    for name, srcs, nbytes in (("encode_kernel<float, 4>", ["encode.hip", "common.h"], 2.2e10),
                               ("reconstruct_kernel<1, 4, 8>", ["reconstruct.hip", "common.h"], 2.3e10)):
        files = [f"paper_2405_19509_amd/csrc/{f}" for f in srcs]
        kernels[name] = {"hbm_bytes": nbytes, "sources": files, "sources_sha256_16": sha(files)}
    (tmp_path / "profiles" / f"hbm_traffic_{HEADLINE.name}.txt").write_text(
        "summary\nJSON " + json.dumps({"workload": HEADLINE.name, "kernels": kernels}) + "\n")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    assert bench.measured_traffic(HEADLINE, "gc_encode") == 2.2e10
    assert bench.measured_traffic(HEADLINE, "gc_reconstruct") == 2.3e10
    with open(csrc / "encode.hip", "a") as f:
        f.write("\n// edited\n")
    assert bench.measured_traffic(HEADLINE, "gc_encode") is None
    assert bench.measured_traffic(HEADLINE, "gc_reconstruct") == 2.3e10
    with open(csrc / "common.h", "a") as f:
        f.write("\n// edited\n")
    assert bench.measured_traffic(HEADLINE, "gc_reconstruct") is None


def test_cpu_baseline_pool_runs_the_oracle():
    """The oracle baseline's process pool: every pattern of the tiny workload on two worker
    processes and a one-core sample; per-step CPU seconds, rates, the d-slice scaling."""
    from workloads import BANDWIDTH, TINY
    r = bench.cpu_oracle_config(TINY, 1, 2, one_core_count=10)
    assert r["patterns"] == TINY.P and r["procs"] == 2
    assert r["patterns_per_s"] > 0 and r["one_core"]["patterns"] == 10
    assert set(r["cpu_seconds"]) == {"chunk_grads", "decode_coeffs", "encode", "reconstruct"}
    s = bench.cpu_oracle_config(BANDWIDTH, 1, 2, count=2, cols=slice(0, 64))
    assert s["d_slice"].startswith("64 of 1048576") and s["patterns_per_s"] > 0


def test_pattern_windows_cover_every_pattern_once():
    for P, parts in ((10000, 64), (100000, 160), (7, 3), (1, 5)):
        w = bench._windows(P, parts)
        assert w[0][0] == 0 and w[-1][1] == P
        assert all(a[1] == b[0] for a, b in zip(w, w[1:])) and all(lo < hi for lo, hi in w)
