"""Seeded random weights, KV prefill and start tokens, stored as bf16.

Weights: N(0, 0.02) drawn in fp32 by a per-tensor ``torch.Generator`` and rounded to bf16
(round to nearest even); RMSNorm gains are 1 (or U[0.5, 1.5] when ``gains="uniform"``).
KV prefill: N(0, 1) bf16 in slots [0, S_i) of lane i; slots from S_i on hold zeros, or
N(0, 100^2) noise when ``poison=True``. Start ids are uniform over the vocabulary; ragged
contexts S_i are uniform integers over the workload's inclusive range.

``device="cuda"`` draws weights and KV with torch's device generator instead (same
distributions and per-tensor seeds, different streams of numbers): the full-size models
take minutes to draw on the host and well under a second on the device. Either way both
sides of a comparison get the very same tensors.
"""
from __future__ import annotations

from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass

import numpy as np
import torch

LAYER_MATS = ("wq", "wk", "wv", "wo", "wg", "wu", "wd")
LAYER_GAINS = ("attn_norm", "mlp_norm", "q_norm", "k_norm")


def as_u16(t: torch.Tensor) -> np.ndarray:
    """Zero-copy uint16 view (bf16 bit patterns) of a CPU bf16 tensor."""
    assert t.dtype == torch.bfloat16 and t.device.type == "cpu"
    return t.contiguous().view(torch.int16).numpy().view(np.uint16)


def _shapes(cfg: dict) -> list:
    """(key, layer, shape, kind) for every tensor, in a fixed order (the order sets seeds)."""
    h, d = cfg["hidden"], cfg["head_dim"]
    nh, nkv, i, V = cfg["n_heads"], cfg["n_kv_heads"], cfg["intermediate"], cfg["vocab"]
    out = [("embed", -1, (V, h), "mat"), ("final_norm", -1, (h,), "gain")]
    if not cfg["tied_embedding"]:
        out.append(("lm_head", -1, (V, h), "mat"))
    for l in range(cfg["n_layers"]):
        out += [("attn_norm", l, (h,), "gain"), ("wq", l, (nh * d, h), "mat"),
                ("wk", l, (nkv * d, h), "mat"), ("wv", l, (nkv * d, h), "mat"),
                ("wo", l, (h, nh * d), "mat"), ("mlp_norm", l, (h,), "gain"),
                ("wg", l, (i, h), "mat"), ("wu", l, (i, h), "mat"), ("wd", l, (h, i), "mat")]
        if cfg["qk_norm"]:
            out += [("q_norm", l, (d,), "gain"), ("k_norm", l, (d,), "gain")]
    return out


def _draw_dev(seed: int, shape, kind: str, gains: str, device: str) -> torch.Tensor:
    g = torch.Generator(device=device).manual_seed(seed)
    if kind == "gain":
        if gains == "ones":
            return torch.ones(shape, dtype=torch.bfloat16, device=device)
        return (torch.rand(shape, generator=g, device=device) + 0.5).to(torch.bfloat16)
    return (torch.randn(shape, generator=g, device=device) * 0.02).to(torch.bfloat16)


def _draw(seed: int, shape, kind: str, gains: str) -> torch.Tensor:
    g = torch.Generator().manual_seed(seed)
    if kind == "gain":
        if gains == "ones":
            return torch.ones(shape, dtype=torch.bfloat16)
        return (torch.rand(shape, generator=g) + 0.5).to(torch.bfloat16)
    n = int(np.prod(shape))
    out = torch.empty(n, dtype=torch.bfloat16)
    chunk = 1 << 24
    for s in range(0, n, chunk):
        e = min(n, s + chunk)
        out[s:e] = (torch.randn(e - s, generator=g) * 0.02).to(torch.bfloat16)
    return out.view(shape)


def make_weights(cfg: dict, seed: int | None = None, gains: str = "ones", threads: int = 8,
                 device: str = "cpu") -> dict:
    """All weights of one model as bf16 tensors on ``device``:
    {embed, final_norm, lm_head?, layers[l]{...}}."""
    if seed is None:
        seed = 1000 + cfg["k"]
    specs = _shapes(cfg)
    seeds = [(seed * 1_000_003 + idx * 7919) % (2**62) for idx in range(len(specs))]
    if device != "cpu":
        tensors = [_draw_dev(sd, sp[2], sp[3], gains, device) for sp, sd in zip(specs, seeds)]
    else:
        with ThreadPoolExecutor(max_workers=threads) as ex:
            tensors = list(ex.map(lambda a: _draw(a[1], a[0][2], a[0][3], gains), zip(specs, seeds)))
    w = {"layers": [dict() for _ in range(cfg["n_layers"])]}
    for (key, l, _, _), t in zip(specs, tensors):
        if l < 0:
            w[key] = t
        else:
            w["layers"][l][key] = t
    return w


def contexts(cfg: dict, seed: int | None = None) -> list:
    lo, hi = cfg["ctx"]
    if lo == hi:
        return [lo] * cfg["batch"]
    if seed is None:
        seed = 4000 + cfg["k"]
    g = torch.Generator().manual_seed(seed)
    return [int(v) for v in torch.randint(lo, hi + 1, (cfg["batch"],), generator=g)]


def make_kv(cfg: dict, S: list, max_ctx: int, seed: int | None = None, poison: bool = False,
            threads: int = 8, device: str = "cpu") -> tuple:
    """Per-layer K and V arenas [b][n_kv][max_ctx][d_h] bf16 with N(0,1) prefill in [0, S_i)."""
    if seed is None:
        seed = 2000 + cfg["k"]
    b, nkv, d, L = cfg["batch"], cfg["n_kv_heads"], cfg["head_dim"], cfg["n_layers"]

    def one(idx):
        g = torch.Generator(device=device).manual_seed((seed * 1_000_003 + idx * 104729) % (2**62))
        t = torch.zeros((b, nkv, max_ctx, d), dtype=torch.bfloat16, device=device)
        for i in range(b):
            t[i, :, : S[i], :] = torch.randn((nkv, S[i], d), generator=g, device=device).to(torch.bfloat16)
        if poison:
            # a separate stream, so the prefill is identical with and without poison
            gp = torch.Generator(device=device).manual_seed((seed * 1_000_003 + idx * 104729 + 1) % (2**62))
            for i in range(b):
                if S[i] < max_ctx:
                    t[i, :, S[i]:, :] = (torch.randn((nkv, max_ctx - S[i], d), generator=gp, device=device)
                                         * 100.0).to(torch.bfloat16)
        return t

    if device != "cpu":
        arenas = [one(idx) for idx in range(2 * L)]
    else:
        with ThreadPoolExecutor(max_workers=threads) as ex:
            arenas = list(ex.map(one, range(2 * L)))
    return arenas[0::2], arenas[1::2]


def make_start(cfg: dict, seed: int | None = None) -> list:
    if seed is None:
        seed = 3000 + cfg["k"]
    g = torch.Generator().manual_seed(seed)
    return [int(v) for v in torch.randint(0, cfg["vocab"], (cfg["batch"],), generator=g)]


@dataclass
class Workload:
    cfg: dict            # shape + b + max_ctx
    weights: dict        # bf16 tensors (on the device they were drawn on)
    kcache: list         # per layer bf16 [b][n_kv][max_ctx][d_h]
    vcache: list
    S: list              # prefilled context per lane
    start: list          # start token per lane
    steps: int


def make_workload(name_or_cfg, gains: str = "ones", poison: bool = False, steps: int | None = None,
                  threads: int = 8, device: str = "cpu") -> Workload:
    from .configs import get_config
    cfg = get_config(name_or_cfg) if isinstance(name_or_cfg, str) else dict(name_or_cfg)
    steps = cfg["steps"] if steps is None else steps
    S = contexts(cfg)
    cfg["max_ctx"] = max(S) + steps
    w = make_weights(cfg, gains=gains, threads=threads, device=device)
    kc, vc = make_kv(cfg, S, cfg["max_ctx"], poison=poison, threads=threads, device=device)
    return Workload(cfg=cfg, weights=w, kcache=kc, vcache=vc, S=S, start=make_start(cfg), steps=steps)
