"""bench.py without a GPU: the algorithmic byte counts behind its rooflines,
and the refusal of more than one GPU.

The byte counts are pinned to an independent sum over the tensors each call
reads and writes once (inputs, outputs, states, cu_seqlens), written out
tensor by tensor here."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def _tensor_bytes_prefill(T, N, hqk, hv, d, e, has_s0):
    q = k = T * hqk * d * e
    v = o = T * hv * d * e
    g = beta = T * hv * 4
    final_state = N * hv * d * d * 4
    initial_state = final_state if has_s0 else 0
    cu = (N + 1) * 4
    return q + k + v + o + g + beta + final_state + initial_state + cu


@pytest.mark.parametrize("T,N,hqk,hv,d,e,s0", [
    (4096, 1, 16, 32, 128, 2, False),     # the benchmark workload
    (62222, 16, 16, 32, 128, 2, True),    # varlen, nonzero initial states
    (64, 1, 1, 1, 32, 4, False),          # fp32 tiny case
])
def test_prefill_bytes(T, N, hqk, hv, d, e, s0):
    assert bench.prefill_bytes(T, N, hqk, hv, d, e, s0) == _tensor_bytes_prefill(T, N, hqk, hv, d, e, s0)


def test_prefill_bytes_and_flops_of_the_benchmark_workload():
    assert bench.prefill_bytes(4096, 1, 16, 32, 128, 2, False) == 103_809_032
    # 21.654 GFLOP: 165,205 flop per token per value head at d = 128, C = 64
    per = bench.prefill_flops(1, 16, 32, 128, 64) / 32
    assert abs(per - (6 * 128 * 128 + 8 * 64 * 128 + 64 * 64 / 3)) < 1e-6
    assert round(bench.prefill_flops(4096, 16, 32, 128, 64) / 1e9, 3) == 21.654


def test_decode_bytes():
    B, hqk, hv, d = 64, 16, 32, 128
    state_rw = 2 * B * hv * d * d * 4
    qk = 2 * B * hqk * d * 2
    vo = 2 * B * hv * d * 2
    gb = 2 * B * hv * 4
    assert bench.decode_bytes(B, hqk, hv, d) == state_rw + qk + vo + gb == 270_024_704


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""
