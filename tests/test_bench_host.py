"""Host-side checks of the benchmark harness (no GPU): the one-GPU guard, the
byte counts behind `value` and `roofline`, and the traffic-record gate."""
import os
import subprocess
import sys

import paper_2601_07892_amd as sh
import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_decode_step_algorithmic_bytes():
    # LLaMA-3.2-1B: 16 layers x (q, k, v, o, gate, up, down); the fused step
    # moves the packed weights, fp32 x, one fp32 scale and fp32 y per product
    lins = synth.model_linears(synth.LLAMA_1B)
    assert len(lins) == 112
    weights = sum(sh.sherry_packed_bytes(l.n, l.k) for _, l in lins)
    assert weights == 152_043_520
    # 5 bits per 4 weights: 5/32 byte per weight (every shape is whole units)
    assert weights * 32 == 5 * sum(l.n * l.k for _, l in lins)
    fused = sum(sh.sherry_packed_bytes(l.n, l.k) + 4 * l.k + 4 + 4 * l.n for _, l in lins)
    assert fused == 154_862_016
    int8 = sum(sh.sherry_packed_bytes(l.n, l.k) + l.k + 4 + 4 * l.n for _, l in lins)
    assert int8 == 153_878_976


def test_traffic_record_is_gated_by_the_kernel_source():
    h = bench.kernel_source_hash(["gemv.hip", "sherry_internal.h"])
    assert len(h) == 16 and h == bench.kernel_source_hash(["gemv.hip", "sherry_internal.h"])
    assert h != bench.kernel_source_hash(["gemv.hip"])
    assert bench.load_traffic("0" * 16, bench.DECODE_KERNEL) is None
    assert bench.load_traffic(h, "gemv_f32_batched_kernel<false>") is None
    got = bench.load_traffic(h, bench.DECODE_KERNEL)
    assert got is None or got > 154_862_016  # counters see at least the algorithmic bytes
