"""The benchmark's contract on the CPU: its algorithmic byte counts (the
numerator of `value` and of the roofline) against hand-computed sums, the
workload figure quoted in its output, and the command-line refusals."""

import json
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


def _fake_result():
    """A result dict shaped like a full run's (every section, every sweep row)."""
    row = {"a": 1.0, "b": 2.0, "c": "x" * 40}
    rep = {"decode_ms": {"mean": 1, "p50": 1, "p99": 2}, "step_ms": {"mean": 1, "p50": 1, "p99": 2},
           "replay": {"resume_hit_rate": 0.5, "plateau_counts": {k: 1 for k in "abcdefghij"}},
           "kv_read_per_step_gib": 24.0, "decode_GBps": 5600.0, "config": "y" * 300,
           "kernels_first_300_steps": {k: {"launches": 1, "ms_per_step": 1.0} for k in "abcd"}}
    return {
        "metric": "m", "value": 6000.0, "unit": "GB/s", "decode_call_us": 220.0, "check": {"max_abs_err": 0.001},
        "resume": {"ms_per_session": 0.014}, "roofline": {"frac": 0.84, "measured_read_ceiling": row},
        "cpu_baseline": {"value": 0.6, "sample": "z" * 200}, "split_on_vector_alu": {"same_grid": row},
        "resume48": {"ms_per_session": 2.5, "copy_GBps": 6400.0, "tbt_impact": 3.0, "decode48_ms": 10.7,
                     "single_session": [{"bytes": 1, "ms": 2.0}] * 3, "partial_residency": [row] * 3,
                     "copy_budget": [row] * 3, "lazy_resume": {"budgets": [row] * 3, "x": row},
                     "cu_split_streams": [{"copy_cus": 64, "tbt_impact": 1.6, **row}] * 3},
        "evict48": {"dirty_ms_per_session": 0.66, "copy_GBps": 6400.0, "frac_of_copy_roofline": 0.8,
                    "clean_evict_ms": 0.06, "cold_writes_total": 43152},
        "resume_host_tier": {"layer_8_sessions": row, "step48_1_session": {"pcie_GBps": 57.0, **row},
                             "beside_decode": {"decode48_ms_alone": 4.8, "dma": {"decode48_ms_beside": 5.0},
                                               "kernel": row}},
        "agentic_replay": dict(rep), "agentic_replay_paper_node": dict(rep),
        "spill_decode": {"config": "s" * 100, "rows": [{"cold_tier": "host", "spilled_frac": f, "mode": m,
                                                        "step_ms": 1.0, "GBps": 2.0}
                                                       for f in (0.0025, 0.005, 0.01, 0.02, 0.04, 0.25, 0.5, 1.0)
                                                       for m in ("direct", "prefetch", "prefetch_cu8")] * 2},
        "configs": {n: {"us_per_call": {"median": 1.0, "p10": 1.0, "p90": 1.0}, "GBps": 1.0, "pct_of_peak": 1.0,
                        "workload": "w" * 40} for n in ("tiny", "step48", "skewed")}
        | {"graph_step48": [row] * 6,
           "append": {"sessions": 32, "batched_append": {"ms_per_step": 0.7, **row}, "per_session_write": row,
                      "prompt_write": {"ms": 0.37, "GBps_read_write": 4300.0, **row},
                      "prompt_write_one_call": {"ms": 0.28, "GBps_read_write": 5700.0, **row},
                      "graph_step": {"step_ms": {"a": 1.0, "b": 0.9}, "append_ms_per_step_in_graph": 0.05,
                                     "config": "c" * 100}},
           "context": row},
    }


def test_stdout_line_stays_short_and_keeps_the_headline_fields():
    full = _fake_result()
    line = json.dumps(bench.compact(full))
    assert len(line) < 12000
    out = json.loads(line)
    for k in ("value", "decode_call_us", "check", "resume", "roofline", "cpu_baseline"):
        assert out[k] == full[k]
    assert out["resume48"]["ms_per_session"] == 2.5
    assert out["configs"]["step48"]["GBps"] == 1.0
    assert len(out["spill_decode_step_ms"]) == 24
    assert out["configs"]["append"]["graph_append_ms_per_step"] == 0.05
