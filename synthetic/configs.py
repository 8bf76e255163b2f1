"""Model shapes and decode workloads.

The five full-size workloads are decoders shaped like public model families with random
weights: Qwen3-0.6B (b1, context 512, 16 tokens), Llama-3.2-1B (b1, 2048, 64 tokens),
Llama-2-7B (b1, 1024, 128 tokens), Qwen3-8B (b4, ragged U[256,4096], 128 tokens) and
Llama-2-13B (b8, ragged U[512,4096], 128 tokens), plus two batch-1 cells of the 8B and 13B
shapes at context 2048. Small shapes ("toy", "mini-*") keep the same structure at sizes the
CPU oracle finishes in seconds while still spanning several GPU tiles and ragged tails.

RMSNorm epsilon follows the public configs of each family (1e-6 Qwen3, 1e-5 Llama); the
paper does not state it.
"""
from __future__ import annotations

_BASE = dict(qk_norm=0, tied_embedding=0, rope_theta=1e4, rms_eps=1e-5)


def _c(**kw):
    d = dict(_BASE)
    d.update(kw)
    return d


CONFIGS = {
    # index k drives the seeds: weights 1000+k, KV 2000+k, start ids 3000+k, contexts 4000+k
    "qwen3-0.6b": _c(k=1, n_layers=28, hidden=1024, n_heads=16, n_kv_heads=8, head_dim=128,
                     intermediate=3072, vocab=151936, qk_norm=1, tied_embedding=1, rope_theta=1e6,
                     rms_eps=1e-6, batch=1, ctx=(512, 512), steps=16),
    "llama3.2-1b": _c(k=2, n_layers=16, hidden=2048, n_heads=32, n_kv_heads=8, head_dim=64,
                      intermediate=8192, vocab=128256, tied_embedding=1, rope_theta=5e5,
                      batch=1, ctx=(2048, 2048), steps=64),
    "llama2-7b": _c(k=3, n_layers=32, hidden=4096, n_heads=32, n_kv_heads=32, head_dim=128,
                    intermediate=11008, vocab=32000, batch=1, ctx=(1024, 1024), steps=128),
    "qwen3-8b": _c(k=4, n_layers=36, hidden=4096, n_heads=32, n_kv_heads=8, head_dim=128,
                   intermediate=12288, vocab=151936, qk_norm=1, rope_theta=1e6, rms_eps=1e-6,
                   batch=4, ctx=(256, 4096), steps=128),
    "llama2-13b": _c(k=5, n_layers=40, hidden=5120, n_heads=40, n_kv_heads=40, head_dim=128,
                     intermediate=13824, vocab=32000, batch=8, ctx=(512, 4096), steps=128),
    # batch-1 cells of the 8B / 13B shapes
    "qwen3-8b-b1": _c(k=6, n_layers=36, hidden=4096, n_heads=32, n_kv_heads=8, head_dim=128,
                      intermediate=12288, vocab=151936, qk_norm=1, rope_theta=1e6, rms_eps=1e-6,
                      batch=1, ctx=(2048, 2048), steps=128),
    "llama2-13b-b1": _c(k=7, n_layers=40, hidden=5120, n_heads=40, n_kv_heads=40, head_dim=128,
                        intermediate=13824, vocab=32000, batch=1, ctx=(2048, 2048), steps=128),
    # small shapes for CPU-time parity
    "toy": _c(k=10, n_layers=2, hidden=64, n_heads=4, n_kv_heads=2, head_dim=16, intermediate=96,
              vocab=200, qk_norm=1, rope_theta=1e4, rms_eps=1e-6, batch=2, ctx=(5, 12), steps=4),
    "toy-gpu": _c(k=16, n_layers=2, hidden=256, n_heads=4, n_kv_heads=2, head_dim=64, intermediate=392,
                  vocab=1000, qk_norm=1, rope_theta=1e4, rms_eps=1e-6, batch=2, ctx=(5, 40), steps=4),
    "mini-qwen3": _c(k=11, n_layers=3, hidden=1024, n_heads=16, n_kv_heads=8, head_dim=128,
                     intermediate=1376, vocab=5003, qk_norm=1, tied_embedding=1, rope_theta=1e6,
                     rms_eps=1e-6, batch=1, ctx=(300, 300), steps=3),
    "mini-llama3": _c(k=12, n_layers=2, hidden=2048, n_heads=32, n_kv_heads=8, head_dim=64,
                      intermediate=2200, vocab=7001, tied_embedding=1, rope_theta=5e5,
                      batch=1, ctx=(700, 700), steps=3),
    "mini-llama2": _c(k=13, n_layers=2, hidden=1536, n_heads=12, n_kv_heads=12, head_dim=128,
                      intermediate=4104, vocab=3000, batch=1, ctx=(129, 129), steps=3),
    "mini-qwen3-b4": _c(k=14, n_layers=2, hidden=1024, n_heads=8, n_kv_heads=2, head_dim=128,
                        intermediate=2816, vocab=4099, qk_norm=1, rope_theta=1e6, rms_eps=1e-6,
                        batch=4, ctx=(1, 900), steps=3),
    "mini-llama2-b8": _c(k=15, n_layers=2, hidden=1280, n_heads=10, n_kv_heads=10, head_dim=128,
                         intermediate=3456, vocab=3001, batch=8, ctx=(3, 700), steps=3),
    # head_dim 64 with three query heads per KV head (a padded head group on the matrix-core
    # attention path) and four ragged lanes (matrix-core GEMV tiles)
    "mini-gqa3-b4": _c(k=17, n_layers=2, hidden=768, n_heads=12, n_kv_heads=4, head_dim=64,
                       intermediate=2048, vocab=3011, rope_theta=5e5, batch=4, ctx=(1, 600), steps=3),
}


def get_config(name: str) -> dict:
    if name not in CONFIGS:
        raise KeyError(f"unknown workload {name!r}; known: {sorted(CONFIGS)}")
    return dict(CONFIGS[name], name=name)
