"""The benchmark's contract on the CPU: its algorithmic byte counts (the
numerator of `value` and of the roofline) against hand-computed sums, the
workload figure quoted in its output, and the command-line refusals."""

import os
import subprocess
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
import synth  # noqa: E402


def test_decode_bytes_by_hand():
    # two rows of 1 and 17 tokens, 4 query / 1 KV heads, d = 64, bf16
    kv, qo, pt = bench.decode_bytes([1, 17], 4, 1, 64, 2)
    assert kv == (1 + 17) * 1 * 64 * 2 * 2          # K and V of each valid token
    assert qo == 2 * 4 * 64 * 2 * 2                 # Q in and out, per row and query head
    assert pt == 4 * (1 + 2) + 4 * 2                # page-table entries of used pages + lengths
    # the split kernel reads K/V, Q, the page table and the lengths, and writes no output
    assert bench.split_kernel_bytes([1, 17], 4, 1, 64, 2) == kv + qo // 2 + pt


def test_layer_workload_bytes():
    """The layer workload (B = 32, seed 0): 676,602 tokens and the split
    kernel's 1,386,112,380 algorithmic bytes per launch quoted in the profiles."""
    w = synth.config_layer(0, batch=32)
    assert int(w.seq_lens.sum()) == 676602
    assert bench.split_kernel_bytes(w.seq_lens, 32, 4, 128, 2) == 1386112380
    kv, qo, pt = bench.decode_bytes(w.seq_lens, 32, 4, 128, 2)
    assert kv == 676602 * 4 * 128 * 2 * 2
    assert kv + qo + pt == 1386374524                # the bench line's decode_bytes


def _run(*args):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args], capture_output=True,
                          text=True, timeout=120, cwd=ROOT)


def test_more_than_one_gpu_is_refused():
    r = _run("--gpus", "2")
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_unknown_section_is_refused():
    r = _run("--sections", "resume48,nonsense")
    assert r.returncode == 2
    assert "nonsense" in r.stderr
