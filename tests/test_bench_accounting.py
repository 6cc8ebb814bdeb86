"""Byte accounting behind the benchmark's roofline figures (CPU only).

The algorithmic bytes of one verify step are every layer weight once, the LM
head twice (the early-exit pass of Sec. 3.1 and the final head), the cached
K/V read once, the block's K/V written and the logits out; written out here
from the model dimensions (Qwen-14B-shaped target of Sec. 4) rather than from
the tensor list the benchmark walks.
"""
import os
import sys

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))

import bench  # noqa: E402
from paper_2510_13161_amd import synth  # noqa: E402


def test_step_bytes_14b_chain_closed_form():
    d, hq, hk, hd, f, v, n = 5120, 40, 8, 128, 13824, 152064, 48
    M, ctx = 9, 1024
    per_layer = 2 * (d * hq * hd + 2 * hk * hd * d + hq * hd * d + 3 * f * d + 2 * d)
    heads = 2 * (2 * v * d)
    kv = n * 2 * hk * hd * 2 * (ctx + M) + n * 2 * hk * hd * 2 * M
    logits = M * v * 4
    sb = bench.step_bytes(synth.QWEN14B, synth.WORKLOADS["14b_chain"], ctx)
    assert sb["weights"] == n * per_layer
    assert sb["heads"] == heads
    assert sb["kv"] == kv
    assert sb["logits"] == logits
    assert sb["total"] == n * per_layer + heads + kv + logits
    assert abs(sb["total"] / 1e9 - 29.75) < 0.01


def test_ffn_up_bytes_14b():
    assert bench.ffn_up_bytes(synth.QWEN14B, 9) == 2 * 13824 * 5120 * 2 + 9 * 5120 * 2 + 9 * 13824 * 2


def test_step_gemm_flops_closed_forms():
    """2·M flops per projection weight, the LM head twice: 14B batch 16
    (M = 144) and the 66B tree (M = 33, ReLU FFN, no gate)."""
    d, hq, hk, hd, f, v, n = 5120, 40, 8, 128, 13824, 152064, 48
    mats = n * (d * hq * hd + 2 * hk * hd * d + hq * hd * d + 3 * f * d) + 2 * v * d
    assert bench.step_gemm_flops(synth.QWEN14B, synth.WORKLOADS["14b_batch16"]) == 2.0 * 144 * mats
    d, h, f, v, n = 9216, 72, 36864, 50272, 64
    mats = n * (4 * d * h * 128 + 2 * f * d) + 2 * v * d
    assert bench.step_gemm_flops(synth.OPT66B, synth.WORKLOADS["66b_tree"]) == 2.0 * 33 * mats
