"""Seeded synthetic inputs for attention BoB (shared by tests, bench and smoke).

This module holds no arithmetic of the method: it only draws the seven
input tensors (Q, K, V, dO and the cotangents U_Q, U_K, U_V on the
first-backward outputs), all [B, H, N, d] or, for workloads with shared
key/value heads, K, V, U_K, U_V with Hkv heads, and names the workload
shapes.  Both the HIP path and the float64 oracle consume the exact values
it returns.

Recipe (the same for every workload): a CPU ``torch.Generator`` seeded with
``seed`` draws float32 standard normals of shape [B, H, N, d] in the order
Q, K, V, dO, U_Q, U_K, U_V; Q and K are then multiplied by ``qk_scale`` in
float32; finally every tensor is cast to the workload dtype with
round-to-nearest-even.  The softmax scale is 1/sqrt(d).
"""
from dataclasses import dataclass
import math

import torch

NAMES = ("Q", "K", "V", "dO", "UQ", "UK", "UV")


@dataclass(frozen=True)
class Workload:
    name: str
    B: int
    H: int
    N: int
    d: int
    dtype: str          # "f32" or "bf16"
    seed: int
    qk_scale: float = 1.0
    causal: bool = False  # the problem flag passed with these inputs (not part of the draw)
    Hkv: int = 0          # key/value heads shared by the H query heads; 0 means H (multi-head)

    @property
    def kv_heads(self) -> int:
        return self.Hkv or self.H

    @property
    def scale(self) -> float:
        return 1.0 / math.sqrt(self.d)

    @property
    def torch_dtype(self):
        return torch.float32 if self.dtype == "f32" else torch.bfloat16


# The five dense workloads: a tiny fp32 case, a small bf16 case, the N=16K
# d=128 case, a long-context N=64K case and the N=256K maximum-length case.
# Causal workloads follow at the shape of the paper's own kernel timings
# (causal, B=4, H=12; Table 1 at d=64, the head-dim sweep of Table 11 at
# N=4096), for comparison with those figures.
WORKLOADS = {
    "tiny_f32_n256_d64": Workload("tiny_f32_n256_d64", 1, 1, 256, 64, "f32", 0),
    "bf16_b2h8_n4096_d64": Workload("bf16_b2h8_n4096_d64", 2, 8, 4096, 64, "bf16", 1),
    "bf16_b1h16_n16384_d128": Workload("bf16_b1h16_n16384_d128", 1, 16, 16384, 128, "bf16", 2, 0.5),
    "bf16_b1h8_n65536_d64": Workload("bf16_b1h8_n65536_d64", 1, 8, 65536, 64, "bf16", 3),
    "bf16_b1h4_n262144_d64": Workload("bf16_b1h4_n262144_d64", 1, 4, 262144, 64, "bf16", 4),
    "causal_bf16_b4h12_n16384_d64": Workload("causal_bf16_b4h12_n16384_d64", 4, 12, 16384, 64, "bf16", 5,
                                             causal=True),
    "causal_bf16_b4h12_n65536_d64": Workload("causal_bf16_b4h12_n65536_d64", 4, 12, 65536, 64, "bf16", 6,
                                             causal=True),
}
for _d, _seed in ((32, 8), (64, 9), (128, 10), (256, 11)):
    _n = f"causal_bf16_b4h12_n4096_d{_d}"
    WORKLOADS[_n] = Workload(_n, 4, 12, 4096, _d, "bf16", _seed, causal=True)
# Dense d=256 at N=8K (head-dim extension; 16 heads fill the device).
WORKLOADS["bf16_b1h16_n8192_d256"] = Workload("bf16_b1h16_n8192_d256", 1, 16, 8192, 256, "bf16", 15)
# Grouped key/value heads at the N=16K d=128 shape: 4 and 1 (multi-query) key/value heads for 16 query heads.
for _n, _hkv, _seed, _causal in (("gqa_bf16_b1h16kv4_n16384_d128", 4, 12, False),
                                 ("mqa_bf16_b1h16kv1_n16384_d128", 1, 13, False),
                                 ("causal_mqa_bf16_b1h16kv1_n16384_d128", 1, 14, True)):
    WORKLOADS[_n] = Workload(_n, 1, 16, 16384, 128, "bf16", _seed, 0.5, causal=_causal, Hkv=_hkv)


def make_inputs(B, H, N, d, dtype="bf16", seed=0, qk_scale=1.0, device="cpu"):
    """Return a dict name -> tensor [B, H, N, d] following the module recipe."""
    gen = torch.Generator(device="cpu")
    gen.manual_seed(int(seed))
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    out = {}
    for name in NAMES:
        x = torch.randn((B, H, N, d), generator=gen, dtype=torch.float32)
        if name in ("Q", "K") and qk_scale != 1.0:
            x = x * qk_scale
        out[name] = x.to(tdt).to(device)
    return out


def make_gqa_inputs(B, H, Hkv, N, d, dtype="bf16", seed=0, device="cpu", qk_scale=1.0):
    """Grouped-query inputs: Q, dO, UQ with H heads and K, V, UK, UV with Hkv
    heads, drawn in the order of NAMES from one seeded generator as in
    make_inputs (N(0,1) float32, Q and K times qk_scale, then cast)."""
    gen = torch.Generator(device="cpu")
    gen.manual_seed(int(seed))
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    out = {}
    for name in NAMES:
        heads = Hkv if name in ("K", "V", "UK", "UV") else H
        x = torch.randn((B, heads, N, d), generator=gen, dtype=torch.float32)
        if name in ("Q", "K") and qk_scale != 1.0:
            x = x * qk_scale
        out[name] = x.to(tdt).to(device)
    return out


def workload_inputs(w: Workload, device="cpu"):
    if w.kv_heads != w.H:
        return make_gqa_inputs(w.B, w.H, w.kv_heads, w.N, w.d, w.dtype, w.seed, device, w.qk_scale)
    return make_inputs(w.B, w.H, w.N, w.d, w.dtype, w.seed, w.qk_scale, device)


def as_f64(t):
    """Exact float64 NumPy copy of a CPU or device tensor (bf16/f32 upcast is exact)."""
    return t.detach().to("cpu", torch.float64).numpy()
