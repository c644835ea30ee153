"""bench.py's contract checks that need no GPU: more than one GPU is refused with a message,
and the algorithmic byte and flop counts behind the roofline match their closed forms."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_2607_14568_amd import inputs  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True, text=True,
                       timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_algorithmic_counts_of_the_timed_workload():
    w = inputs.WORKLOADS["prefill_10k_bf16"]
    byts, flops = bench.algorithmic(w, [w.T], w.dk, w.dv, w.H, w.io, True)
    # q, k, v read and o written in bf16, g and beta in fp32; S0 read and S_T written in fp32
    assert byts == 10240 * 16 * ((2 * 128 + 2 * 128) * 2 + 8) + 2 * 16 * 4 * 128 * 128 == 171180032
    # per full chunk of 64: n(n-1)dk + n(n+1)dk + n(n-1)(dk+dv) + n(n+1)dv + 6 n dk dv, 160 chunks, 16 heads
    n, d = 64, 128
    per_chunk = n * (n - 1) * d + n * (n + 1) * d + n * (n - 1) * 2 * d + n * (n + 1) * d + 6 * n * d * d
    assert flops == 160 * 16 * per_chunk == 22796042240


def test_ragged_tail_chunks_are_counted_at_their_length():
    w = inputs.WORKLOADS["ragged_8seq_bf16"]
    _, f_tail = bench.algorithmic(w, [65], 128, 128, 1, "bf16", False)
    _, f_full = bench.algorithmic(w, [64], 128, 128, 1, "bf16", False)
    n, d = 1, 128   # the one-token tail chunk
    assert f_tail - f_full == n * (n - 1) * d + n * (n + 1) * d + n * (n - 1) * 2 * d + n * (n + 1) * d + 6 * n * d * d


def test_attention_workloads_are_declared():
    for name, (B, T, H, Hkv, d) in bench.ATTN.items():
        assert H % Hkv == 0 and d in (64, 128) and T > 0 and B >= 1, name
