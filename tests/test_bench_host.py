"""Host-side pieces of bench.py (no GPU): the multi-GPU refusal, the popcount
used by the regime check, the traffic digest and the CPU baseline leg."""
import os
import random
import subprocess
import sys

import pytest
import torch

from conftest import ROOT

sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_popcount64_matches_python():
    rnd = random.Random(5)
    vals = [0, 1, -1, 2**63 - 1, -2**63] + [rnd.getrandbits(64) - 2**63 for _ in range(500)]
    got = bench._popcount64(torch.tensor(vals, dtype=torch.int64)).tolist()
    assert got == [bin(v & (2**64 - 1)).count("1") for v in vals]


@pytest.mark.parametrize("kernel,main", [("fanout_gather", "dg_pack.hip"),
                                         ("assemble", "dg_assemble.hip")])
def test_traffic_digest_covers_the_kernel_translation_unit(tmp_path, monkeypatch, kernel, main):
    d = bench.kernel_source_digest(kernel)
    assert len(d) == 16
    # the digest changes with any file of the translation unit
    src = os.path.join(ROOT, "paper_2405_05231_amd", "csrc")
    fake = tmp_path / "paper_2405_05231_amd" / "csrc"
    fake.mkdir(parents=True)
    for n in bench.KERNEL_TU[kernel]:
        (fake / n).write_bytes(open(os.path.join(src, n), "rb").read())
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    assert bench.kernel_source_digest(kernel) == d
    (fake / main).write_bytes(b"// changed\n" + (fake / main).read_bytes())
    assert bench.kernel_source_digest(kernel) != d


def test_cpu_baseline_runs_two_groups_on_the_host():
    """The CPU baseline leg (the oracle on the host) on the tiny workload: two
    consecutive groups, the first of which is the benchmark's own."""
    import synth
    w = synth.make_workload("T")
    cfg = w.cfg
    r = bench.cpu_baseline(w, cfg, cfg.B, groups=2)
    assert r["kind"] == "oracle" and r["cores"] == 1 and r["unit"] == "GB/s"
    assert r["value"] > 0 and r["sampled_edges_per_s"] > 0
    assert "2 consecutive groups" in r["sample"]
    assert set(r["seconds"]) == {"sample", "pack", "assemble"}
