"""ctypes binding of the CPU reference decoder (fm_oracle.cpp): TEST INFRASTRUCTURE ONLY.

Only the tests, ``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py`` may import
this module. The GPU library never imports it and shares no code with it.

Everything here is argument marshalling; the arithmetic lives in ``fm_oracle.cpp``, which
follows arXiv 2609.12379 Sec. 2.1 (the decode step) and Eq. 1 (attention).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "fm_oracle.cpp")
_LIB = os.path.join(_HERE, "libfm_oracle.so")

TAP_NAMES = ("a", "qkv", "qrot", "krot", "o", "x1", "a2", "mlp", "x2")


def build(force: bool = True) -> str:
    """Compile the oracle with g++ (IEEE semantics: no fast-math, no FP contraction)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        cmd = ["g++", "-O2", "-std=c++17", "-fPIC", "-shared", "-fopenmp", "-fno-fast-math",
               "-ffp-contract=off", _SRC, "-o", tmp]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB)
    return _LIB


class _Cfg(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "n_layers", "hidden", "n_heads", "n_kv_heads", "head_dim", "intermediate", "vocab",
        "qk_norm", "tied_embedding", "batch", "max_ctx", "reserved")] + [
        ("rope_theta", ctypes.c_double), ("rms_eps", ctypes.c_double)]


class _Layer(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in (
        "attn_norm", "wq", "wk", "wv", "q_norm", "k_norm", "wo", "mlp_norm", "wg", "wu", "wd")]


class _Weights(ctypes.Structure):
    _fields_ = [("embed", ctypes.c_void_p), ("final_norm", ctypes.c_void_p),
                ("lm_head", ctypes.c_void_p), ("layers", ctypes.POINTER(_Layer))]


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=True)
        L = ctypes.CDLL(_LIB)
        P = ctypes.c_void_p
        L.fmo_tap_count.restype = ctypes.c_size_t
        L.fmo_tap_count.argtypes = [ctypes.POINTER(_Cfg)]
        L.fmo_tap_offsets.argtypes = [ctypes.POINTER(_Cfg), P]
        for suf in ("f32", "f64"):
            getattr(L, f"fmo_decode_step_{suf}").argtypes = [
                ctypes.POINTER(_Cfg), ctypes.POINTER(_Weights), P, P, P, P, P, P, P, P]
            getattr(L, f"fmo_decode_step_{suf}").restype = ctypes.c_int
            getattr(L, f"fmo_rmsnorm_{suf}").argtypes = [P, P, ctypes.c_int, ctypes.c_double, P]
            getattr(L, f"fmo_gemv_{suf}").argtypes = [P, ctypes.c_int, ctypes.c_int, P, P]
            getattr(L, f"fmo_rope_{suf}").argtypes = [P, ctypes.c_int, ctypes.c_int, ctypes.c_double]
            getattr(L, f"fmo_attend_{suf}").argtypes = [P, P, P, ctypes.c_int, ctypes.c_int, P]
            getattr(L, f"fmo_silu_mul_{suf}").argtypes = [P, P, ctypes.c_int, P]
            getattr(L, f"fmo_argmax_{suf}").argtypes = [P, ctypes.c_int]
            getattr(L, f"fmo_argmax_{suf}").restype = ctypes.c_int32
            getattr(L, f"fmo_to_bf16_{suf}").argtypes = [P, ctypes.c_int64, P]
        _lib = L
    return _lib


def _ptr(a: np.ndarray) -> int:
    assert a.flags["C_CONTIGUOUS"], "arrays passed to the oracle must be C-contiguous"
    return a.ctypes.data


def _dt(precision: str):
    if precision not in ("f32", "f64"):
        raise ValueError("precision must be 'f32' or 'f64'")
    return np.float32 if precision == "f32" else np.float64


# ---- single operators ----------------------------------------------------------------

def rmsnorm(x, g_bf16, eps, precision="f64"):
    dt = _dt(precision)
    x = np.ascontiguousarray(x, dtype=dt)
    g = np.ascontiguousarray(g_bf16, dtype=np.uint16)
    out = np.empty_like(x)
    getattr(lib(), f"fmo_rmsnorm_{precision}")(_ptr(x), _ptr(g), x.size, float(eps), _ptr(out))
    return out


def gemv(W_bf16, x, precision="f64"):
    dt = _dt(precision)
    W = np.ascontiguousarray(W_bf16, dtype=np.uint16)
    x = np.ascontiguousarray(x, dtype=dt)
    N, K = W.shape
    assert x.size == K
    y = np.empty(N, dtype=dt)
    getattr(lib(), f"fmo_gemv_{precision}")(_ptr(W), N, K, _ptr(x), _ptr(y))
    return y


def rope(v, pos, theta, precision="f64"):
    dt = _dt(precision)
    v = np.array(v, dtype=dt, copy=True)
    getattr(lib(), f"fmo_rope_{precision}")(_ptr(v), v.size, int(pos), float(theta))
    return v


def attend(q, K_bf16, V_bf16, precision="f64"):
    dt = _dt(precision)
    q = np.ascontiguousarray(q, dtype=dt)
    K = np.ascontiguousarray(K_bf16, dtype=np.uint16)
    V = np.ascontiguousarray(V_bf16, dtype=np.uint16)
    n, d = K.shape
    assert V.shape == (n, d) and q.size == d
    o = np.empty(d, dtype=dt)
    getattr(lib(), f"fmo_attend_{precision}")(_ptr(q), _ptr(K), _ptr(V), n, d, _ptr(o))
    return o


def silu_mul(g, u, precision="f64"):
    dt = _dt(precision)
    g = np.ascontiguousarray(g, dtype=dt)
    u = np.ascontiguousarray(u, dtype=dt)
    out = np.empty_like(g)
    getattr(lib(), f"fmo_silu_mul_{precision}")(_ptr(g), _ptr(u), g.size, _ptr(out))
    return out


def argmax(v, precision="f32"):
    dt = _dt(precision)
    v = np.ascontiguousarray(v, dtype=dt)
    return int(getattr(lib(), f"fmo_argmax_{precision}")(_ptr(v), v.size))


def to_bf16(v, precision="f32"):
    dt = _dt(precision)
    v = np.ascontiguousarray(v, dtype=dt)
    out = np.empty(v.shape, dtype=np.uint16)
    getattr(lib(), f"fmo_to_bf16_{precision}")(_ptr(v), v.size, _ptr(out))
    return out


# ---- the whole decode step -----------------------------------------------------------

@dataclass
class StepResult:
    logits: np.ndarray        # [b][V]
    next_ids: np.ndarray      # int32 [b]
    taps: dict | None         # name -> array [L][b][n]; plus "final" [b][h]


def _cfg_struct(cfg: dict) -> _Cfg:
    c = _Cfg()
    for n in ("n_layers", "hidden", "n_heads", "n_kv_heads", "head_dim", "intermediate", "vocab",
              "qk_norm", "tied_embedding", "batch", "max_ctx"):
        setattr(c, n, int(cfg[n]))
    c.reserved = 0
    c.rope_theta = float(cfg["rope_theta"])
    c.rms_eps = float(cfg["rms_eps"])
    return c


def tap_offsets(cfg: dict) -> dict:
    c = _cfg_struct(cfg)
    out = np.zeros(10, dtype=np.int64)
    lib().fmo_tap_offsets(ctypes.byref(c), _ptr(out))
    names = TAP_NAMES + ("block",)
    return {n: int(v) for n, v in zip(names, out)}


class Oracle:
    """Holds one model's bf16 weights (numpy uint16 views) and runs decode steps on the CPU.

    ``weights`` is a dict of uint16 numpy arrays holding bf16 bit patterns, keyed like
    ``synthetic.inputs.make_weights``: embed, final_norm, lm_head (absent when tied) and
    per layer ``layers[l][name]``. The KV cache is owned by the caller: ``kcache[l]`` /
    ``vcache[l]`` uint16 arrays of shape [b][n_kv][max_ctx][d_h], appended to in place.
    """

    def __init__(self, cfg: dict, weights: dict):
        self.cfg = dict(cfg)
        self._c = _cfg_struct(cfg)
        self._keep = []
        L = cfg["n_layers"]
        layers = (_Layer * L)()
        for l in range(L):
            lw = weights["layers"][l]
            for n in _Layer._fields_:
                name = n[0]
                arr = lw.get(name)
                if arr is None:
                    setattr(layers[l], name, None)
                    continue
                arr = np.ascontiguousarray(arr, dtype=np.uint16)
                self._keep.append(arr)
                setattr(layers[l], name, _ptr(arr))
        self._layers = layers
        w = _Weights()
        for name in ("embed", "final_norm", "lm_head"):
            arr = weights.get(name)
            if arr is None:
                setattr(w, name, None)
                continue
            arr = np.ascontiguousarray(arr, dtype=np.uint16)
            self._keep.append(arr)
            setattr(w, name, _ptr(arr))
        w.layers = ctypes.cast(layers, ctypes.POINTER(_Layer))
        self._w = w

    def tap_count(self) -> int:
        return int(lib().fmo_tap_count(ctypes.byref(self._c)))

    def step(self, kcache, vcache, tok, pos, kv_lens, precision="f32", taps=False) -> StepResult:
        cfg = self.cfg
        dt = _dt(precision)
        b, V, L = cfg["batch"], cfg["vocab"], cfg["n_layers"]
        tok = np.ascontiguousarray(tok, dtype=np.int32)
        pos = np.ascontiguousarray(pos, dtype=np.int32)
        kvl = np.ascontiguousarray(kv_lens, dtype=np.int32)
        assert tok.size == b and pos.size == b and kvl.size == b
        for arr in list(kcache) + list(vcache):
            assert arr.dtype == np.uint16 and arr.flags["C_CONTIGUOUS"]
        kp = (ctypes.c_void_p * L)(*[_ptr(a) for a in kcache])
        vp = (ctypes.c_void_p * L)(*[_ptr(a) for a in vcache])
        logits = np.empty((b, V), dtype=dt)
        nxt = np.empty(b, dtype=np.int32)
        tbuf = np.zeros(self.tap_count(), dtype=dt) if taps else None
        rc = getattr(lib(), f"fmo_decode_step_{precision}")(
            ctypes.byref(self._c), ctypes.byref(self._w), kp, vp, _ptr(tok), _ptr(pos), _ptr(kvl),
            _ptr(logits), _ptr(nxt), _ptr(tbuf) if taps else None)
        if rc != 0:
            raise ValueError(f"oracle rejected the step inputs (code {rc})")
        tap_dict = None
        if taps:
            off = tap_offsets(cfg)
            blk = off["block"]
            body = tbuf[: L * b * blk].reshape(L, b, blk)
            sizes = {}
            names = TAP_NAMES
            for k, n in enumerate(names):
                end = off[names[k + 1]] if k + 1 < len(names) else blk
                sizes[n] = (off[n], end)
            tap_dict = {n: body[:, :, s:e].copy() for n, (s, e) in sizes.items()}
            tap_dict["final"] = tbuf[L * b * blk:].reshape(b, cfg["hidden"]).copy()
        return StepResult(logits=logits, next_ids=nxt, taps=tap_dict)
