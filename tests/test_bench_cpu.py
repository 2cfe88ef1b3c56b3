"""Host logic of bench.py, on the CPU: the algorithmic byte model that the
roofline divides by, the one-GPU guard, and the gate that reports counter
traffic only for the kernel source it was measured on.

The byte model is pinned to totals worked out by hand from the workload
definitions (x read once, y read and written once, each referenced adapter
once at its own rank, 16 B of plan record per token), not to the function's own
formula."""
import os
import shutil
import subprocess
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_2608_03579_amd import synth  # noqa: E402


def _step_bytes(w):
    return sum(bench.apply_bytes(w, (w.tok_c, w.tok_u), t) for t in range(len(w.tables)))


def test_headline_bytes_per_apply():
    # Llama-3.2-3B q_proj decode: 64 tokens, 3072 -> 3072, bf16; 4 centroids of
    # rank 32 and 64 rank-2 residuals, all referenced
    x = 64 * 3072 * 2                     # 393,216
    y = 2 * 64 * 3072 * 2                 # 786,432 (read + write)
    cent = 4 * 32 * (3072 + 3072) * 2     # 1,572,864
    res = 64 * 2 * (3072 + 3072) * 2      # 1,572,864
    plan = 64 * 16
    assert _step_bytes(synth.make(2, 0)) == x + y + cent + res + plan == 4_326_400


def test_llama31_8b_decode_layer_bytes():
    # 256 distinct users (rank 2) over 16 centroids of rank 32, one layer:
    # sum(in) = 38912, sum(out) = 43008
    w = synth.make(4, 0)
    assert len(np.unique(w.tok_u)) == 256 and len(np.unique(w.tok_c)) == 16
    s_in, s_out = 38912, 43008
    want = (256 * s_in * 2 + 2 * 256 * s_out * 2 + 16 * 32 * (s_in + s_out) * 2 + 256 * 2 * (s_in + s_out) * 2
            + 7 * 256 * 16)
    assert _step_bytes(w) == want
    assert abs(want / 1e6 - 231.7) < 0.1


def test_zipf_batch_bytes_count_each_referenced_adapter_once():
    # a user with many tokens in the batch moves its residual once
    w = synth.make(5, 0)
    s_in, s_out = 26624, 27648
    users = np.unique(w.tok_u[w.tok_u >= 0])
    cents = np.unique(w.tok_c[w.tok_c >= 0])
    ranks = int(sum(int(w.slot_rank[u]) for u in users))
    want = (512 * s_in * 2 + 2 * 512 * s_out * 2 + len(cents) * 64 * (s_in + s_out) * 2
            + ranks * (s_in + s_out) * 2 + 7 * 512 * 16)
    assert _step_bytes(w) == want
    assert len(users) < 512                # Zipf: repeated users
    base = synth.make(5, 0, baseline=True)
    assert _step_bytes(base) > 2 * _step_bytes(w)   # rank-16 residuals, no centroids


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_kernel_bytes_split_the_apply_bytes():
    # shrink (x + A factors) and expand (y read + write + B factors) together are
    # the apply's bytes, with the 16 B token records read by both
    for cfg in (2, 4, 5):
        w = synth.make(cfg, 0)
        maps = (w.tok_c, w.tok_u)
        for t in range(len(w.tables)):
            sh, ex = bench.kernel_bytes(w, maps, t)
            assert sh + ex == bench.apply_bytes(w, maps, t) + 16 * w.T
    w = synth.make(2, 0)
    sh, ex = bench.kernel_bytes(w, (w.tok_c, w.tok_u), 0)
    assert sh == 64 * 3072 * 2 + (4 * 32 + 64 * 2) * 3072 * 2 + 64 * 16
    assert ex == 2 * 64 * 3072 * 2 + (4 * 32 + 64 * 2) * 3072 * 2 + 64 * 16


def test_layer_groups():
    assert [len(g) for g in bench.layer_groups(synth.make(3, 0))] == [7] * 28
    assert bench.layer_groups(synth.make(4, 0)) == [list(range(7))]
    assert bench.layer_groups(synth.make(2, 0)) == [[0]]


def test_traffic_is_reported_only_for_the_profiled_kernel_source(tmp_path, monkeypatch):
    for workload, rel in bench.TRAFFIC_PROFILES.items():
        path = os.path.join(ROOT, rel)
        if not os.path.exists(path):
            assert bench.measured_traffic(workload, "k_expand") is None
            continue
        fields = bench.read_fields(path)
        for kernel in ("k_shrink", "k_expand"):
            got = bench.measured_traffic(workload, kernel)
            key = f"traffic_bytes_per_launch_{kernel}"
            if fields.get("kernel_source_sha256_16") == bench.kernel_source_hash() and key in fields:
                assert got == int(fields[key])
            else:
                assert got is None
    # a copy of the tree whose kernel sources differ by one byte: no traffic
    fake = tmp_path / "root"
    csrc = fake / "paper_2608_03579_amd" / "csrc"
    csrc.mkdir(parents=True)
    for n in bench.KERNEL_SOURCES:
        shutil.copy(os.path.join(ROOT, "paper_2608_03579_amd", "csrc", n), csrc / n)
    for rel in bench.TRAFFIC_PROFILES.values():
        if os.path.exists(os.path.join(ROOT, rel)):
            (fake / os.path.dirname(rel)).mkdir(parents=True, exist_ok=True)
            shutil.copy(os.path.join(ROOT, rel), fake / rel)
    with open(csrc / "salt_apply.hip", "ab") as f:
        f.write(b"\n")
    monkeypatch.setattr(bench, "ROOT", str(fake))
    for workload in bench.TRAFFIC_PROFILES:
        assert bench.measured_traffic(workload, "k_expand") is None
    assert bench.measured_traffic("no-such-workload", "k_expand") is None
