"""Offline cost model of the step scheduler on MI355X (section 4.2.1, "Offline
Profiling for Cost Model"): per-step time T(res, k) of a 57-block,
3072-wide model (512 text tokens) at each resolution of the paper's workload
mix and each sequence-parallel degree k, in integer microseconds, as the rows
``ts_allocate`` / ``ts_round_schedule`` take.

How each entry is obtained:
* k = 1: a full ``dit_step`` + ``euler_update`` timed with HIP events on one
  MI355X (``bench.py --extra dit57_<res>px_bf16``);
* k > 1: one GPU's share of a k-way Ulysses split measured the same way (every
  non-attention kernel on the L/k-token shard plus, per block, attention of
  24/k heads over all L tokens; ``bench.py --extra
  dit57_<res>px_sp<k>_share_bf16``), plus the two all-to-alls per block the
  one-GPU measurement leaves out, priced by a link model: each GPU sends 1/k of
  its shard's Q, K, V (3 L H / k bf16 values) and of the attention output
  (L H / k) to each of the k - 1 peers over its own xGMI link, so per block
  (4 L H 2 bytes) / k^2 cross one link of XGMI_LINK_BYTES_PER_S.  This is a
  model, not a measurement: nothing here has run on more than one GPU.
* B identical requests batched in one step (selective continuous batching,
  section 3 / section 5): ``bench.py --extra dit57_<res>px_x<B>_bf16``.

The measured values below come from one bench run on one MI355X (box-to-box
spread about +-5%); regenerate them with the bench commands above.
"""
from __future__ import annotations

from typing import Dict, List

HIDDEN = 3072
BLOCKS = 57
TEXT_TOKENS = 512
XGMI_LINK_BYTES_PER_S = 153e9

# full step on one GPU, ms
STEP_MS_K1: Dict[int, float] = {256: 15.98, 512: 25.41, 1024: 69.49, 2048: 391.76}
# one GPU's share of a k-way split (compute only), ms
SHARE_MS: Dict[int, Dict[int, float]] = {
    256: {2: 13.3, 4: 12.44, 8: 11.93},
    512: {2: 17.69, 4: 14.42, 8: 13.67},
    1024: {2: 39.04, 4: 28.28, 8: 21.03},
    2048: {2: 208.07, 4: 105.13, 8: 56.85},
}
# B identical requests in one step, ms per step (all B advance one step)
BATCH_MS: Dict[int, Dict[int, float]] = {
    256: {1: 15.98, 4: 44.75, 8: 87.25},
    512: {1: 25.41, 2: 46.55, 4: 89.19},
}


def tokens(res: int) -> int:
    """Joint sequence length: (res / 16)^2 image tokens (Table 1) + 512 text tokens."""
    return (res // 16) ** 2 + TEXT_TOKENS


def all_to_all_ms(res: int, k: int) -> float:
    """Modelled cost of the two all-to-alls per block of a k-way Ulysses step."""
    if k == 1:
        return 0.0
    bytes_per_link = 4.0 * tokens(res) * HIDDEN * 2 / (k * k)
    return BLOCKS * bytes_per_link / XGMI_LINK_BYTES_PER_S * 1e3


def step_us(res: int, k: int) -> int:
    """T(res, k) in microseconds (0 when not available)."""
    if k == 1:
        return int(round(STEP_MS_K1[res] * 1e3))
    share = SHARE_MS.get(res, {}).get(k)
    if share is None:
        return 0
    return int(round((share + all_to_all_ms(res, k)) * 1e3))


def row(res: int, max_k: int = 8) -> List[int]:
    """Cost-model row [T(1), T(2), T(4), ...] up to max_k, for the scheduler."""
    out, k = [], 1
    while k <= max_k:
        out.append(step_us(res, k))
        k *= 2
    return out


def batch_step_us(res: int, b: int) -> int:
    """Step time of b identical requests batched together (0 when not measured)."""
    ms = BATCH_MS.get(res, {}).get(b)
    return int(round(ms * 1e3)) if ms is not None else 0
