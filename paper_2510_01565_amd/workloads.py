"""Model shapes and request batches of the measured workloads.

Image tokens per request follow section 2.2, Table 1 of the paper
(256 / 1024 / 4096 / 16384 tokens at 256 / 512 / 1024 / 2048 px, i.e.
(resolution/16)^2, section 6.1).  The 57-block, 3072-wide, 24x128-head shape
with 512 text tokens is the FLUX.1-dev class model the paper serves
(section 6.1, "Models").  The paper's second model, SD3 (section 6.1 and the
4xA40 experiment of section 6.4), is served at the SD3-Medium shape: 24 joint
blocks with separate weights for the text and image streams, 1536 wide,
24x64 heads, 16 latent channels patchified 2x2 (64 input channels), 4096-wide
text embeddings with 77 + 256 = 333 text tokens, 4096 image tokens at
1024 px.  Only the shape is SD3's: the block is this library's adaLN joint
block with 2-D RoPE (no learned position table, no pooled-text conditioning),
and the weights are seeded random values.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional


@dataclass(frozen=True)
class ModelShape:
    hidden: int
    heads: int
    head_dim: int
    mlp_ratio: int
    n_double: int
    n_single: int
    in_channels: int
    text_dim: int
    time_freq_dim: int = 256
    tie_streams: bool = False
    rope_theta: float = 10000.0
    ln_eps: float = 1e-6
    dtype: str = "bf16"          # "bf16" or "f32"


@dataclass
class Workload:
    name: str
    model: ModelShape
    resolutions: List[int]       # one per request
    n_txt: List[int]
    t: Optional[List[float]] = None   # None: drawn from the seed, U[0, 1)
    dt: float = 1.0 / 28.0
    kind: str = "step"           # "step", "double_block", "attention_share"
    note: str = ""
    extra: dict = field(default_factory=dict)

    def grids(self) -> List[int]:
        return [r // 16 for r in self.resolutions]

    def n_img(self) -> List[int]:
        return [(r // 16) ** 2 for r in self.resolutions]


SMALL_BLOCK = ModelShape(hidden=384, heads=6, head_dim=64, mlp_ratio=4, n_double=1, n_single=0,
                         in_channels=16, text_dim=384, tie_streams=True, dtype="f32")
FLUX_DOUBLE = ModelShape(hidden=3072, heads=24, head_dim=128, mlp_ratio=4, n_double=1, n_single=0,
                         in_channels=64, text_dim=4096)
FLUX_FULL = ModelShape(hidden=3072, heads=24, head_dim=128, mlp_ratio=4, n_double=19, n_single=38,
                       in_channels=64, text_dim=4096)
SD3_MEDIUM = ModelShape(hidden=1536, heads=24, head_dim=64, mlp_ratio=4, n_double=24, n_single=0,
                        in_channels=64, text_dim=4096)
SD3_DOUBLE = ModelShape(hidden=1536, heads=24, head_dim=64, mlp_ratio=4, n_double=1, n_single=0,
                        in_channels=64, text_dim=4096)

WORKLOADS = {
    "small_block_256px_f32": Workload(
        "small_block_256px_f32", SMALL_BLOCK, [256], [32], t=[0.5],
        note="one tied adaLN block, 384 wide, 6x64 heads, 256 image + 32 text tokens, fp32"),
    "mmdit_double_512px_bf16": Workload(
        "mmdit_double_512px_bf16", FLUX_DOUBLE, [512], [512], t=[0.5], kind="double_block",
        note="one double-stream block, 3072 wide, 512 text + 1024 image tokens, bf16"),
    "dit57_1024px_bf16": Workload(
        "dit57_1024px_bf16", FLUX_FULL, [1024], [512], t=[0.5],
        note="19 double + 38 single blocks, 512 text + 4096 image tokens, bf16"),
    "dit57_2048px_bf16": Workload(
        "dit57_2048px_bf16", FLUX_FULL, [2048], [512], t=[0.5],
        note="19 double + 38 single blocks, 512 text + 16384 image tokens, bf16"),
    "dit57_2048px_sp4_share_bf16": Workload(
        "dit57_2048px_sp4_share_bf16", FLUX_FULL, [2048], [512], t=[0.5], kind="attention_share",
        note="one GPU's share of a 4-way sequence-parallel split: 6 of 24 heads over 16896 tokens",
        extra={"sp": 4}),
    "dit57_256px_bf16": Workload(
        "dit57_256px_bf16", FLUX_FULL, [256], [512], t=[0.5],
        note="19 double + 38 single blocks, 512 text + 256 image tokens, bf16 (cost-model row)"),
    "dit57_512px_bf16": Workload(
        "dit57_512px_bf16", FLUX_FULL, [512], [512], t=[0.5],
        note="19 double + 38 single blocks, 512 text + 1024 image tokens, bf16 (cost-model row)"),
    # selective continuous batching (section 3, section 5): B identical small-resolution
    # requests stepped together, each at its own timestep
    "dit57_256px_x4_bf16": Workload(
        "dit57_256px_x4_bf16", FLUX_FULL, [256] * 4, [512] * 4, t=None,
        note="4 identical 256 px requests batched in one step"),
    "dit57_256px_x8_bf16": Workload(
        "dit57_256px_x8_bf16", FLUX_FULL, [256] * 8, [512] * 8, t=None,
        note="8 identical 256 px requests batched in one step"),
    "dit57_512px_x2_bf16": Workload(
        "dit57_512px_x2_bf16", FLUX_FULL, [512] * 2, [512] * 2, t=None,
        note="2 identical 512 px requests batched in one step"),
    "dit57_512px_x4_bf16": Workload(
        "dit57_512px_x4_bf16", FLUX_FULL, [512] * 4, [512] * 4, t=None,
        note="4 identical 512 px requests batched in one step"),
    "sd3m_1024px_bf16": Workload(
        "sd3m_1024px_bf16", SD3_MEDIUM, [1024], [333], t=[0.5],
        note="SD3-Medium shape: 24 joint blocks, 1536 wide, 24x64 heads, 333 text + 4096 image tokens, bf16"),
    "sd3m_512px_bf16": Workload(
        "sd3m_512px_bf16", SD3_MEDIUM, [512], [333], t=[0.5],
        note="SD3-Medium shape: 24 joint blocks, 333 text + 1024 image tokens, bf16"),
    "sd3m_packed_mixed_bf16": Workload(
        "sd3m_packed_mixed_bf16", SD3_MEDIUM, [256, 512, 1024], [333, 333, 333], t=None,
        note="SD3-Medium shape, 3 requests 256/512/1024 px packed, per-request timesteps U[0,1)"),
    "dit57_packed_mixed_bf16": Workload(
        "dit57_packed_mixed_bf16", FLUX_FULL, [256, 512, 1024, 2048], [512, 512, 512, 512], t=None,
        note="4 requests 256/512/1024/2048 px packed, per-request timesteps U[0,1)"),
}

# One GPU's share of a k-way sequence-parallel step at every resolution of the
# paper's workload mix (256 .. 2048 px, section 6.1): the per-GPU compute of
# the cost model's T(k) rows.
for _res in (256, 512, 1024, 2048):
    for _k in (2, 4, 8):
        _name = f"dit57_{_res}px_sp{_k}_share_bf16"
        if _name not in WORKLOADS:
            WORKLOADS[_name] = Workload(
                _name, FLUX_FULL, [_res], [512], t=[0.5], kind="attention_share",
                note=f"one GPU's share of a {_k}-way sequence-parallel split at {_res} px",
                extra={"sp": _k})


def flops_per_step(m: ModelShape, n_txt: List[int], n_img: List[int]) -> dict:
    """Algorithmic FLOPs of one step: 2*M*N*K per GEMM (embedders, modulation
    GEMVs, QKV, output projection, MLP, single-block linears, final layer) and
    4*Lq*Lk*d per head for attention inside each request.  Softmax, norms and
    elementwise work are not counted."""
    H, F, d, nh = m.hidden, m.mlp_ratio * m.hidden, m.head_dim, m.heads
    n_req = len(n_img)
    Tt, Ti = sum(n_txt), sum(n_img)
    T = Tt + Ti
    streams = 1 if m.tie_streams else 2
    mod_rows = (m.n_double * streams * 6 + m.n_single * 3 + 2) * H
    g = 2.0 * n_req * (H * m.time_freq_dim + H * H) + 2.0 * n_req * mod_rows * H
    g += 2.0 * Ti * H * m.in_channels + 2.0 * Tt * H * m.text_dim
    g += m.n_double * 2.0 * T * H * (3 * H + H + F + F)
    g += m.n_single * 2.0 * T * H * ((3 * H + F) + (H + F))
    g += 2.0 * Ti * H * m.in_channels
    a = (m.n_double + m.n_single) * sum(4.0 * (lt + li) ** 2 * d * nh for lt, li in zip(n_txt, n_img))
    return {"gemm": g, "attention": a, "total": g + a}
