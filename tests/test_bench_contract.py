"""Host-side checks of bench.py: the one-GPU guard and the byte accounting
behind its roofline and path fractions (no GPU needed)."""
import os
import subprocess
import sys

import bench
import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _run_bench(args, env_extra=None):
    env = dict(os.environ)
    env.update(env_extra or {})
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args],
                          cwd=ROOT, env=env, capture_output=True, text=True,
                          timeout=120)


def test_more_than_one_gpu_is_refused():
    r = _run_bench(["--gpus", "2"])
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_distributed_launch_is_refused():
    r = _run_bench([], {"WORLD_SIZE": "8"})
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_headline_bytes_per_unit():
    # 32K workload: L = 32768, d = 128, bf16, J = 5, S = 128, k = 2048, B = 64
    w = synth.WORKLOADS["headline32k"]
    a = bench.algorithmic_bytes(w, 2048)
    assert a["keys"] == 32768 * 128 * 2          # every key once
    assert a["pool"] == (128 << 5) * 128 * 2     # S runs of 2^J keys
    assert a["values"] == 2048 * 128 * 2         # the selected values
    assert a["q_and_o"] == 2 * 64 * 128 * 2      # query block in, output out
    assert a["kept"] == 0
    assert a["total"] == 9_994_240
    assert a["kernel"]["token_skim"] * w.units == 1_075_838_976
    assert a["kernel"]["sparse_attn"] == 2 * 2048 * 128 * 2 + 64 * 128 * 2


def test_tail_rows_are_counted_once_for_keys_and_values():
    w = synth.WORKLOADS["tail32k"]
    a = bench.algorithmic_bytes(w, 2048)
    rem = w.ctx_len - ((w.ctx_len >> w.levels) << w.levels)
    assert a["kept"] == 2 * (rem + w.gen_len) * w.head_dim * 2


def test_cached_step_reads_the_approximation_not_the_keys():
    w = synth.WORKLOADS["cached32k"]
    a = bench.algorithmic_bytes(w, 2048)
    assert a["keys"] == (w.ctx_len >> w.levels) * w.head_dim * 4


def test_counter_summary_is_ignored_for_another_kernel_or_workload():
    assert bench.measured_traffic("skim_tile", "headline32k") is None
    assert bench.measured_traffic("token_skim", "long16k") is None


def test_needle_recall_counts_kept_needle_tokens():
    """needle_recall: the share of planted needle tokens in the selection."""
    import numpy as np
    import torch
    w = synth.small_variant(synth.WORKLOADS["tiny"], name="nr", needles=2,
                            batch=2, heads=3)
    spans = [np.concatenate([np.arange(s, s + synth.NEEDLE_LEN)
                             for s in synth.needle_starts(w, 0, b)])
             for b in range(w.batch)]
    tok = torch.zeros((w.batch, w.heads, 2 * synth.NEEDLE_LEN), dtype=torch.int32)
    for b in range(w.batch):
        tok[b] = torch.from_numpy(np.sort(spans[b]).astype(np.int32))
    tok[1, 2, :8] = -1                       # one unit misses 8 needle tokens
    r = bench.needle_recall(w, tok)
    assert r["units"] == 6 and r["min"] == 0.75
    assert abs(r["mean"] - (5 + 0.75) / 6) < 1e-12


def test_cpu_model_is_a_string():
    assert isinstance(bench.cpu_model(), str)


def test_single_thread_oracle_baseline_runs_one_unit_per_call():
    r = bench.cpu_single_thread("tiny", min_seconds=0.0)
    assert r["cores"] == 1 and r["workload"] == "tiny"
    assert r["value"] > 0 and r["unit"] == "tokens/s"


def test_shared_workload_recall_takes_one_list_per_sequence():
    import torch
    w = synth.small_variant(synth.WORKLOADS["tiny"], batch=2, heads=3,
                            shared=True)
    keff = min(w.budget, w.segments << w.levels)
    tok = torch.arange(keff, dtype=torch.int32).repeat(w.batch, 1)
    r = bench.needle_recall(w, tok)
    assert r["units"] == w.batch * w.heads
