"""Byte accounting and bandwidth utilisation for one decode step (host-side arithmetic).

``step_bytes`` is Eq. 2 of arXiv 2609.12379 (Sec. 2.2): the weights every projection and the
LM head read, the KV cache attention reads, and the b gathered embedding rows. The full
embedding table is not counted, since decode gathers only b rows. Norm gains, the rotary
table, KV writes, logit writes and activations are excluded, as in the paper.
``mbu`` is Eq. 3: bytes / (time * peak bandwidth).
"""
from __future__ import annotations

MI355X_HBM_PEAK = 8.0e12   # bytes/s, the published MI355X HBM3E peak
H100_HBM_PEAK = 3.35e12    # bytes/s, the paper's H100 80GB HBM3 figure (Sec. 2.2)


def weight_bytes(cfg: dict, w: int = 2) -> int:
    L, h, nh, nkv, d = cfg["n_layers"], cfg["hidden"], cfg["n_heads"], cfg["n_kv_heads"], cfg["head_dim"]
    i, V = cfg["intermediate"], cfg["vocab"]
    return (L * (h * nh * d + 2 * h * nkv * d + nh * d * h + 3 * h * i) + V * h) * w


def kv_bytes(cfg: dict, attended_slots_total: int, w: int = 2) -> int:
    """KV bytes read: 2 L n_kv d_h w per attended slot, summed over lanes."""
    return 2 * cfg["n_layers"] * cfg["n_kv_heads"] * cfg["head_dim"] * attended_slots_total * w


def step_bytes(cfg: dict, S, b: int | None = None, w: int = 2) -> int:
    """Eq. 2. ``S`` is either one context length shared by all b lanes or a per-lane list."""
    if isinstance(S, (list, tuple)):
        b = len(S)
        total = int(sum(S))
    else:
        b = cfg["batch"] if b is None else b
        total = int(S) * b
    return weight_bytes(cfg, w) + kv_bytes(cfg, total, w) + b * cfg["hidden"] * w


def mbu(bytes_per_step: float, seconds_per_step: float, peak: float = MI355X_HBM_PEAK) -> float:
    """Eq. 3, as a fraction (multiply by 100 for %)."""
    return bytes_per_step / (seconds_per_step * peak)


def step_flops(cfg: dict, S) -> float:
    """2 flops per weight element per lane plus attention's 4 d_h flops per (query head, slot)."""
    if not isinstance(S, (list, tuple)):
        S = [S] * cfg["batch"]
    b = len(S)
    params = weight_bytes(cfg, 1)
    return 2.0 * params * b + 4.0 * cfg["n_layers"] * cfg["n_heads"] * cfg["head_dim"] * sum(S)
