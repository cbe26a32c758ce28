"""The benchmark's algorithmic counts against values derived by hand from the
workload definitions (the 8B replay, its full reset, the chunked 32k-prefix
replay), so that the reported TFLOP/s and GB/s rest on the right numerators."""
import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
import workloads as W  # noqa: E402


def test_attention_flops_of_the_8b_replay():
    # 4 d FLOPs per (query-head row, visible key) pair: query i of the suffix
    # sees P + i + 1 keys; Hq = 32, d = 128, P = 8189, S = 2048
    pairs = sum(8189 + i + 1 for i in range(2048))
    assert bench.attention_flops(8189, 2048, 32, 128) == pytest.approx(4 * 128 * 32 * pairs, rel=1e-12)
    assert bench.attention_flops(8189, 2048, 32, 128) == pytest.approx(3.0915e11, rel=1e-4)
    # the full reset of the 10237-token trajectory
    assert bench.attention_flops(0, 10237, 32, 128) == pytest.approx(8.5857e11, rel=1e-4)


def test_attention_bytes_of_the_8b_replay():
    # Q and O of the suffix (32 heads), K and V of every position (8 heads), bf16
    want = 2 * (2 * 2048 * 32 * 128 + 2 * (8189 + 2048) * 8 * 128)
    assert bench.attention_bytes(8189, 2048, 32, 8, 128, 2) == want


class _Setup:
    def __init__(self, name, P, S, chunk):
        self.w, self.P, self.S, self.chunk = W.workload(name), P, S, chunk


def test_prefix_bytes():
    # K/V of the cropped prefix: 8189 keys x 8 heads x 128 x 2 bytes x 2
    st = _Setup("llama8b_p8189_s2048_bf16", [8189], [2048], None)
    assert bench.Setup.prefix_bytes(st) == 8189 * 8 * 128 * 2 * 2
    # chunked: chunk c reads the prefix grown by the chunks before it
    st = _Setup("long32k_chunk512_llama8b_bf16", [32768], [4096], 512)
    keys = sum(32768 + 512 * c for c in range(8))
    assert bench.Setup.prefix_bytes(st) == keys * 8 * 128 * 2 * 2
    assert bench.Setup.prefix_bytes(st) == pytest.approx(1.1325e9, rel=1e-4)
