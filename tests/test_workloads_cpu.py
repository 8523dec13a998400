"""Host checks of the seeded input generator: the grouped-head draw equals
the multi-head draw when every query head has its own key/value head, the
named grouped workloads have key-side tensors with Hkv heads, and the CPU
baseline maps each query head to its key/value head."""
import torch

import bench
from workloads import NAMES, WORKLOADS, Workload, make_gqa_inputs, make_inputs, workload_inputs


def test_grouped_draw_with_one_head_per_group_is_the_multi_head_draw():
    a = make_inputs(2, 3, 17, 8, "bf16", seed=5, qk_scale=0.5)
    b = make_gqa_inputs(2, 3, 3, 17, 8, "bf16", seed=5, qk_scale=0.5)
    for n in NAMES:
        assert torch.equal(a[n], b[n]), n


def test_grouped_workloads_have_shared_key_value_heads():
    for name in ("gqa_bf16_b1h16kv4_n16384_d128", "mqa_bf16_b1h16kv1_n16384_d128",
                 "causal_mqa_bf16_b1h16kv1_n16384_d128"):
        w = WORKLOADS[name]
        assert w.H % w.kv_heads == 0 and w.kv_heads < w.H
    w = Workload("tiny_gqa", 1, 4, 9, 4, "f32", 3, 0.5, Hkv=2)
    x = workload_inputs(w)
    for n in NAMES:
        heads = 2 if n in ("K", "V", "UK", "UV") else 4
        assert tuple(x[n].shape) == (1, heads, 9, 4), n
    ref = make_gqa_inputs(1, 4, 2, 9, 4, "f32", 3, qk_scale=0.5)
    for n in NAMES:
        assert torch.equal(x[n], ref[n]), n
    assert WORKLOADS["bf16_b2h8_n4096_d64"].kv_heads == 8


def test_cpu_baseline_runs_on_a_grouped_workload():
    w = Workload("tiny_gqa", 1, 4, 40, 8, "f32", 3, Hkv=2)
    out = bench.cpu_baseline(workload_inputs(w), w, slab=16, budget_s=0.05)
    assert out["kind"] == "oracle" and out["value"] > 0
