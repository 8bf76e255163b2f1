"""ctypes binding of the C ABI in include/fm.h (argument marshalling only).

Every step of the decode runs in the HIP library ``libfm.so``; this module only fills the C
structs and forwards device pointers. Importing it does not need a GPU. Loading the library
raises if it has not been built: there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libfm.so")

FM_OK, FM_ERR_INVALID_ARG, FM_ERR_UNSUPPORTED, FM_ERR_CAPACITY, FM_ERR_HIP, FM_ERR_DEVICE = range(6)
FM_DEV_OK, FM_DEV_BAD_TOKEN, FM_DEV_BAD_POSITION, FM_DEV_BAD_KV_LEN, FM_DEV_WATCHDOG = range(5)
FM_OP_QKV, FM_OP_ATTN, FM_OP_OPROJ, FM_OP_GU, FM_OP_DOWN, FM_OP_LM = range(1, 7)


class fm_model_cfg(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "n_layers", "hidden", "n_heads", "n_kv_heads", "head_dim", "intermediate", "vocab",
        "qk_norm", "tied_embedding", "batch", "max_ctx", "n_workgroups", "attn_items", "dyn_chunk_kb")] + [
        ("rope_theta", ctypes.c_double), ("rms_eps", ctypes.c_double)]


class fm_layer_weights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in (
        "attn_norm", "w_q", "w_k", "w_v", "q_norm", "k_norm", "w_o", "mlp_norm", "w_gate", "w_up", "w_down")]


class fm_weight_ptrs(ctypes.Structure):
    _fields_ = [("embed", ctypes.c_void_p), ("final_norm", ctypes.c_void_p), ("lm_head", ctypes.c_void_p),
                ("layers", ctypes.POINTER(fm_layer_weights))]


class fm_kv_ptrs(ctypes.Structure):
    _fields_ = [("k", ctypes.POINTER(ctypes.c_void_p)), ("v", ctypes.POINTER(ctypes.c_void_p))]


class fm_plan_stats(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "n_cu", "n_instr", "n_types", "min_instr_per_layer", "n_counters", "attn_items",
        "attn_max_chunks", "n_stages", "n_dyn_stages")] + [
        ("max_bytes_per_cu", ctypes.c_double), ("mean_bytes_per_cu", ctypes.c_double),
        ("imbalance", ctypes.c_double)]


EXPORTS = ("fm_create", "fm_decode_step", "fm_decode_step_multilaunch", "fm_decode_step_noalloc", "fm_extend",
           "fm_destroy", "fm_last_error", "fm_set_taps", "fm_tap_count", "fm_set_timeline", "fm_instruction_count",
           "fm_noalloc_scratch_bytes", "fm_plan_query", "fm_plan_export", "fm_status_string")

_lib = None


def load():
    """Load libfm.so (raises if it is missing: build it with paper_2609_12379_amd.build)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing; build it with `python -m paper_2609_12379_amd.build`")
    L = ctypes.CDLL(LIB_PATH)
    P, I32 = ctypes.c_void_p, ctypes.c_int32
    L.fm_create.argtypes = [ctypes.POINTER(fm_model_cfg), ctypes.POINTER(fm_weight_ptrs),
                            ctypes.POINTER(fm_kv_ptrs), ctypes.POINTER(P)]
    for n in ("fm_decode_step", "fm_decode_step_multilaunch", "fm_decode_step_noalloc"):
        getattr(L, n).argtypes = [P, P, P, P, P, P, P]
    L.fm_noalloc_scratch_bytes.argtypes = [P]
    L.fm_noalloc_scratch_bytes.restype = ctypes.c_size_t
    L.fm_extend.argtypes = [P, P, P, P, I32, P, P, P]
    L.fm_destroy.argtypes = [P]
    L.fm_last_error.argtypes = [P, ctypes.POINTER(I32)]
    L.fm_set_taps.argtypes = [P, P]
    L.fm_set_timeline.argtypes = [P, P]
    L.fm_instruction_count.argtypes = [P]
    L.fm_tap_count.argtypes = [ctypes.POINTER(fm_model_cfg)]
    L.fm_tap_count.restype = ctypes.c_size_t
    L.fm_plan_query.argtypes = [ctypes.POINTER(fm_model_cfg), I32, ctypes.POINTER(fm_plan_stats)]
    L.fm_plan_export.argtypes = [ctypes.POINTER(fm_model_cfg), I32, P, I32, P, I32]
    L.fm_status_string.argtypes = [I32]
    L.fm_status_string.restype = ctypes.c_char_p
    for n in EXPORTS:
        if n not in ("fm_tap_count", "fm_status_string", "fm_noalloc_scratch_bytes"):
            getattr(L, n).restype = I32
    _lib = L
    return L


class FmError(RuntimeError):
    def __init__(self, status: int, what: str = ""):
        self.status = status
        msg = load().fm_status_string(status).decode()
        super().__init__(f"{what}: {msg} (status {status})" if what else msg)


def check(status: int, what: str = ""):
    if status != FM_OK:
        raise FmError(status, what)


def make_cfg(cfg: dict, n_workgroups: int = 0, attn_items: int = 0, dyn_chunk_kb: int = 0) -> fm_model_cfg:
    c = fm_model_cfg()
    for n in ("n_layers", "hidden", "n_heads", "n_kv_heads", "head_dim", "intermediate", "vocab",
              "qk_norm", "tied_embedding", "batch", "max_ctx"):
        setattr(c, n, int(cfg[n]))
    c.n_workgroups = int(n_workgroups)
    c.attn_items = int(attn_items)
    c.dyn_chunk_kb = int(dyn_chunk_kb)
    c.rope_theta = float(cfg["rope_theta"])
    c.rms_eps = float(cfg["rms_eps"])
    return c


def plan_query(cfg: dict, n_cu: int, attn_items: int = 0, dyn_chunk_kb: int = 0) -> fm_plan_stats:
    s = fm_plan_stats()
    check(load().fm_plan_query(ctypes.byref(make_cfg(cfg, attn_items=attn_items, dyn_chunk_kb=dyn_chunk_kb)),
                               int(n_cu), ctypes.byref(s)),
          "fm_plan_query")
    return s


def plan_export(cfg: dict, n_cu: int, attn_items: int = 0, dyn_chunk_kb: int = 0):
    """Returns (qoff int32[n_cu+1], instrs int32[n][4]) as numpy arrays."""
    import numpy as np
    s = plan_query(cfg, n_cu, attn_items, dyn_chunk_kb)
    qoff = np.zeros(n_cu + 1, dtype=np.int32)
    ins = np.zeros((s.n_instr, 4), dtype=np.int32)
    check(load().fm_plan_export(ctypes.byref(make_cfg(cfg, attn_items=attn_items, dyn_chunk_kb=dyn_chunk_kb)), int(n_cu),
                                qoff.ctypes.data, qoff.size, ins.ctypes.data, ins.size), "fm_plan_export")
    return qoff, ins


def tap_count(cfg: dict) -> int:
    return int(load().fm_tap_count(ctypes.byref(make_cfg(cfg))))


class Decoder:
    """A handle over device-resident bf16 weights and a caller-owned KV arena (torch tensors).

    ``weights``: dict like ``synthetic.inputs.make_weights`` but with CUDA bf16 tensors.
    ``kcache``/``vcache``: per-layer CUDA bf16 tensors [b][n_kv][max_ctx][d_h].
    The tensors must stay alive (this object keeps references).
    """

    def __init__(self, cfg: dict, weights: dict, kcache, vcache, n_workgroups: int = 0, attn_items: int = 0,
                 dyn_chunk_kb: int = 0):
        import torch
        self.cfg = dict(cfg)
        self._keep = [weights, kcache, vcache]
        L = cfg["n_layers"]
        layers = (fm_layer_weights * L)()
        names = {"attn_norm": "attn_norm", "w_q": "wq", "w_k": "wk", "w_v": "wv", "q_norm": "q_norm",
                 "k_norm": "k_norm", "w_o": "wo", "mlp_norm": "mlp_norm", "w_gate": "wg", "w_up": "wu",
                 "w_down": "wd"}
        for l in range(L):
            for cname, key in names.items():
                t = weights["layers"][l].get(key)
                if t is not None:
                    assert t.is_cuda and t.dtype == torch.bfloat16 and t.is_contiguous()
                setattr(layers[l], cname, t.data_ptr() if t is not None else None)
        w = fm_weight_ptrs()
        w.embed = weights["embed"].data_ptr()
        w.final_norm = weights["final_norm"].data_ptr()
        w.lm_head = weights["lm_head"].data_ptr() if weights.get("lm_head") is not None else None
        w.layers = ctypes.cast(layers, ctypes.POINTER(fm_layer_weights))
        kp = (ctypes.c_void_p * L)(*[t.data_ptr() for t in kcache])
        vp = (ctypes.c_void_p * L)(*[t.data_ptr() for t in vcache])
        kv = fm_kv_ptrs(ctypes.cast(kp, ctypes.POINTER(ctypes.c_void_p)), ctypes.cast(vp, ctypes.POINTER(ctypes.c_void_p)))
        self._c = make_cfg(cfg, n_workgroups, attn_items, dyn_chunk_kb)
        self._layers, self._w, self._kp, self._vp, self._kv = layers, w, kp, vp, kv
        h = ctypes.c_void_p()
        check(load().fm_create(ctypes.byref(self._c), ctypes.byref(w), ctypes.byref(kv), ctypes.byref(h)), "fm_create")
        self.h = h
        self._taps = None

    def step(self, token_ids, positions, kv_lens, logits_out, next_ids, stream=None, multilaunch=False,
             noalloc=False):
        """All arguments are CUDA tensors (int32 / float32); stream defaults to torch's current stream.
        ``multilaunch``: the per-stage ablation; ``noalloc``: fm_decode_step_noalloc."""
        import torch
        if stream is None:
            stream = torch.cuda.current_stream().cuda_stream
        assert not (multilaunch and noalloc)
        fn = (load().fm_decode_step_multilaunch if multilaunch else
              load().fm_decode_step_noalloc if noalloc else load().fm_decode_step)
        st = fn(self.h, token_ids.data_ptr(), positions.data_ptr(), kv_lens.data_ptr(),
                logits_out.data_ptr() if logits_out is not None else None, next_ids.data_ptr(), stream)
        check(st, "fm_decode_step")

    def extend(self, token_ids, positions, kv_lens, logits_out, next_ids, stream=None):
        """Prompt extension as single-token steps: token_ids, positions and kv_lens are CUDA
        int32 tensors [n_tokens][b] (row t feeds step t); logits_out ([b][vocab] or None) and
        next_ids ([b]) receive the last step's results."""
        import torch
        if stream is None:
            stream = torch.cuda.current_stream().cuda_stream
        b = self.cfg["batch"]
        for t in (token_ids, positions, kv_lens):
            assert t.is_cuda and t.dtype == torch.int32 and t.is_contiguous() and t.dim() == 2 and t.shape[1] == b
        assert token_ids.shape == positions.shape == kv_lens.shape
        st = load().fm_extend(self.h, token_ids.data_ptr(), positions.data_ptr(), kv_lens.data_ptr(),
                              int(token_ids.shape[0]), logits_out.data_ptr() if logits_out is not None else None,
                              next_ids.data_ptr(), stream)
        check(st, "fm_extend")

    def noalloc_scratch_bytes(self) -> int:
        return int(load().fm_noalloc_scratch_bytes(self.h))

    def set_taps(self, tap_buf):
        self._taps = tap_buf
        check(load().fm_set_taps(self.h, tap_buf.data_ptr() if tap_buf is not None else None), "fm_set_taps")

    def set_timeline(self, buf):
        """buf: CUDA int64 tensor of 8 * instruction_count() words, or None."""
        self._tl = buf
        check(load().fm_set_timeline(self.h, buf.data_ptr() if buf is not None else None), "fm_set_timeline")

    def instruction_count(self) -> int:
        return int(load().fm_instruction_count(self.h))

    def last_error(self) -> int:
        code = ctypes.c_int32(0)
        load().fm_last_error(self.h, ctypes.byref(code))
        return int(code.value)

    def close(self):
        if getattr(self, "h", None):
            load().fm_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
