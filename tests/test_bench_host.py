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


@pytest.mark.parametrize("kernel,main", [("fanout_gather", "dg_gather.hip"),
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
    consecutive groups (the first is the benchmark's own) on the host's cores,
    and the first group on one core."""
    import oracle
    import synth
    w = synth.make_workload("T")
    cfg = w.cfg
    r = bench.cpu_baseline(w, cfg, cfg.B, groups=2, small=False)
    assert r["kind"] == "oracle" and r["unit"] == "GB/s"
    assert r["cores"] == oracle.host_threads() and r["one_core"]["cores"] == 1
    assert r["value"] > 0 and r["sampled_edges_per_s"] > 0 and r["one_core"]["value"] > 0
    assert "2 consecutive groups" in r["sample"]
    assert set(r["seconds"]) == {"sample", "pack", "assemble"}
    assert r["cpu_model"]


def test_oracle_on_runs_of_batches_gives_the_group_result():
    """Splitting a group into runs of mini-batches over host threads (as the
    CPU baseline does) gives every mini-batch the outputs of one pass over the
    whole group: sampled lists, packed chunk, packed order, address table."""
    import numpy as np

    import oracle
    import synth
    w = synth.make_workload("T")
    cfg = w.cfg
    args = (w.offsets.numpy(), w.indices.numpy(), w.feats.numpy(), w.cache_slot.numpy(),
            w.cache.numpy(), w.seeds.numpy(), list(cfg.fanouts), w.rng_seed, 0, cfg.row_bytes)
    _, rs1, p1, _ = bench._oracle_pass(oracle, *args, 1)
    _, rs3, p3, runs = bench._oracle_pass(oracle, *args, 3)
    assert len(runs) == 3
    for k in ("nodes", "edge_src", "edge_dst", "hop_ptr", "edge_ptr"):
        assert all(np.array_equal(a, b) for a, b in zip(rs1[k], rs3[k])), k
    whole = p1[0]
    for (lo, hi), part in zip(runs, p3):
        for b in range(lo, hi):
            assert np.array_equal(whole["loc"][b], part["loc"][b - lo])
            w0, w1 = whole["packed_ptr"][b], whole["packed_ptr"][b + 1]
            q0, q1 = part["packed_ptr"][b - lo], part["packed_ptr"][b - lo + 1]
            assert np.array_equal(whole["packed_ids"][w0:w1], part["packed_ids"][q0:q1])
            assert np.array_equal(whole["packed"][w0:w1], part["packed"][q0:q1])
