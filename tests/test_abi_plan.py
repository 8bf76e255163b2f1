"""Host-side checks of the C-ABI library (no GPU needed).

* the library loads and exports every function that include/fm.h declares;
* argument validation of the host-checkable errors (Sec. 4.1's compiler rejects what the
  kernel cannot run);
* the schedule compiler's queues: every output row and attention item appears exactly once
  per layer, each queue is in one global topological order, and the structural
  gates of Sec. 4.3 (instruction types, instructions per layer, queue imbalance, counters)
  hold on every full-size shape;
* deadlock freedom: a simulation of all queues that lets a workgroup run its next
  instruction only once every producer of that instruction's inputs has finished.
"""
from __future__ import annotations

import ctypes
import os
import re

import numpy as np
import pytest

from synthetic import get_config, CONFIGS

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "fm.h")

FULL = ["qwen3-0.6b", "llama3.2-1b", "llama2-7b", "qwen3-8b", "llama2-13b", "qwen3-8b-b1", "llama2-13b-b1"]
OP_QKV, OP_ATTN, OP_OPROJ, OP_GU, OP_DOWN, OP_LM = 1, 2, 3, 4, 5, 6
STAGE = {OP_QKV: 0, OP_ATTN: 1, OP_OPROJ: 2, OP_GU: 3, OP_DOWN: 4}


@pytest.fixture(scope="module")
def fm():
    from paper_2609_12379_amd import fm as fm_mod
    try:
        fm_mod.load()
    except (OSError, RuntimeError) as e:  # pragma: no cover - library not built
        pytest.fail(f"libfm.so is not built: {e}")
    return fm_mod


def _with_ctx(cfg: dict) -> dict:
    cfg = dict(cfg)
    cfg["max_ctx"] = cfg["ctx"][1] + cfg["steps"]
    return cfg


def declared_functions() -> list:
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[A-Za-z_][\w]*\s*\**\s*(fm_[a-z_]+)\s*\(", text, flags=re.M)))


def test_header_symbols_exported(fm):
    names = declared_functions()
    assert "fm_create" in names and "fm_decode_step" in names and "fm_destroy" in names
    lib = ctypes.CDLL(fm.LIB_PATH)
    missing = [n for n in names if not hasattr(lib, n)]
    assert not missing, f"declared but not exported: {missing}"
    assert sorted(fm.EXPORTS) == names, "the Python binding's export list differs from the header"


def test_null_arguments_rejected(fm):
    L = fm.load()
    INVALID = 1
    assert L.fm_destroy(None) == INVALID
    assert L.fm_decode_step(None, None, None, None, None, None, None) == INVALID
    assert L.fm_decode_step_multilaunch(None, None, None, None, None, None, None) == INVALID
    assert L.fm_decode_step_noalloc(None, None, None, None, None, None, None) == INVALID
    assert L.fm_noalloc_scratch_bytes(None) == 0
    assert L.fm_extend(None, None, None, None, 1, None, None, None) == INVALID
    code = ctypes.c_int32(0)
    assert L.fm_last_error(None, ctypes.byref(code)) == INVALID
    assert L.fm_set_taps(None, None) == INVALID
    assert L.fm_set_timeline(None, None) == INVALID
    c = fm.make_cfg(_with_ctx(get_config("toy-gpu")))
    out = ctypes.c_void_p(1)
    assert L.fm_create(ctypes.byref(c), None, None, ctypes.byref(out)) == INVALID
    assert out.value is None, "fm_create must clear the handle on failure"
    assert L.fm_tap_count(None) == 0
    for s in range(6):
        assert L.fm_status_string(s).decode() not in ("", "unknown status")


@pytest.mark.parametrize("field,value,status", [
    ("head_dim", 96, 2), ("head_dim", 0, 1), ("batch", 9, 2), ("batch", 0, 1),
    ("n_kv_heads", 3, 1),            # 4 query heads are not a multiple of 3 KV heads
    ("hidden", 260, 2),              # not a multiple of 8
    ("intermediate", 390, 2), ("n_layers", 0, 1), ("vocab", 0, 1), ("max_ctx", 0, 1),
])
def test_cfg_validation(fm, field, value, status):
    cfg = _with_ctx(get_config("toy-gpu"))
    cfg[field] = value
    s = fm.fm_plan_stats()
    got = fm.load().fm_plan_query(ctypes.byref(fm.make_cfg(cfg)), 64, ctypes.byref(s))
    assert got == status, f"{field}={value}: status {got}, expected {status}"


def test_cfg_validation_group_and_tuning(fm):
    L = fm.load()
    s = fm.fm_plan_stats()
    cfg = _with_ctx(get_config("toy-gpu"))
    cfg.update(n_heads=36, n_kv_heads=4)                      # G = 9 > 8
    assert L.fm_plan_query(ctypes.byref(fm.make_cfg(cfg)), 64, ctypes.byref(s)) == 2
    c = fm.make_cfg(_with_ctx(get_config("toy-gpu")))
    c.dyn_chunk_kb = -2
    assert L.fm_plan_query(ctypes.byref(c), 64, ctypes.byref(s)) == 1
    c = fm.make_cfg(_with_ctx(get_config("toy-gpu")))
    c.rope_theta = 0.0
    assert L.fm_plan_query(ctypes.byref(c), 64, ctypes.byref(s)) == 1
    # attention items must exceed n_kv * b (one item per (lane, KV head) plus chunking room)
    cfg = _with_ctx(get_config("toy-gpu"))
    c = fm.make_cfg(cfg, attn_items=cfg["n_kv_heads"] * cfg["batch"])
    assert L.fm_plan_query(ctypes.byref(c), 64, ctypes.byref(s)) == 1
    assert L.fm_plan_query(ctypes.byref(fm.make_cfg(cfg)), 0, ctypes.byref(s)) == 1


def test_export_capacity(fm):
    L = fm.load()
    cfg = _with_ctx(get_config("toy-gpu"))
    s = fm.plan_query(cfg, 16)
    qoff = np.zeros(17, np.int32)
    ins = np.zeros((s.n_instr, 4), np.int32)
    c = fm.make_cfg(cfg)
    assert L.fm_plan_export(ctypes.byref(c), 16, qoff.ctypes.data, 16, ins.ctypes.data, ins.size) == 3
    assert L.fm_plan_export(ctypes.byref(c), 16, qoff.ctypes.data, 17, ins.ctypes.data, ins.size - 1) == 3
    assert L.fm_plan_export(ctypes.byref(c), 16, qoff.ctypes.data, 17, ins.ctypes.data, ins.size) == 0


def test_tap_count_matches_oracle(fm):
    from oracle.oracle import tap_offsets
    for name in ("toy", "toy-gpu", "mini-qwen3", "qwen3-8b"):
        cfg = _with_ctx(get_config(name))
        per, final = tap_offsets(cfg)["block"], cfg["batch"] * cfg["hidden"]
        assert fm.tap_count(cfg) == cfg["n_layers"] * cfg["batch"] * per + final


# --------------------------------------------------------------------------------------
# schedule compiler


def _gemv_rows(cfg):
    d = cfg["head_dim"]
    return {OP_QKV: (cfg["n_heads"] + 2 * cfg["n_kv_heads"]) * d, OP_OPROJ: cfg["hidden"],
            OP_GU: cfg["intermediate"], OP_DOWN: cfg["hidden"], OP_LM: cfg["vocab"]}


def _gemv_cols(cfg):
    return {OP_QKV: cfg["hidden"], OP_OPROJ: cfg["n_heads"] * cfg["head_dim"], OP_GU: 2 * cfg["hidden"],
            OP_DOWN: cfg["intermediate"], OP_LM: cfg["hidden"]}


def _order_key(op, layer, L):
    return (L, 0) if op == OP_LM else (layer, STAGE[op])


POOLS = 8


def dyn_chunk_rows(n_rows, rc, kp, slots, nwg):
    """Row ranges of a stage in dynamic chunks, rebuilt from its record as the header
    describes it, after checking what the kernel relies on: every pool holds at least one
    chunk per workgroup (each takes its own one) and at most `slots` per workgroup (so the
    pool is always drained, whoever takes its chunks)."""
    assert rc >= 1 and kp in (1, 2, 4, 8) and slots >= 2
    nch = -(-n_rows // rc)
    np_ = min(POOLS, nwg)
    out = []
    start = 0
    for x in range(np_):
        nwx = len(range(x, nwg, np_))
        c0 = nch * start // nwg
        c1 = nch * (start + nwx) // nwg
        assert nwx <= c1 - c0 <= nwx * slots, (x, nwx, c0, c1, slots)
        for c in range(c0, c1):
            out.append((c * rc, min(n_rows, (c + 1) * rc)))
        start += nwx
    return out


def check_plan(cfg, nwg, fm):
    s = fm.plan_query(cfg, nwg)
    qoff, ins = fm.plan_export(cfg, nwg)
    L, b, nkv = cfg["n_layers"], cfg["batch"], cfg["n_kv_heads"]
    assert qoff[0] == 0 and qoff[-1] == len(ins) == s.n_instr and np.all(np.diff(qoff) >= 0)
    P = s.attn_items
    assert P > nkv * b and s.attn_max_chunks == (P - nkv * b) // nkv + 1
    rows = _gemv_rows(cfg)
    cover = {}
    dyn = {}
    for op, layer, a, bb in ins:
        op, layer = int(op), int(layer)
        if op in rows and a < 0:
            dyn.setdefault((op, layer), []).append((int(-a), int(bb)))
        elif op in rows:
            assert 0 <= a < bb <= rows[op], (op, layer, a, bb)
            cover.setdefault((op, layer), []).append((int(a), int(bb)))
        elif op == OP_ATTN:
            assert 0 <= a < P and 0 <= layer < L
            cover.setdefault((op, layer), []).append((int(a), int(a) + 1))
        else:
            raise AssertionError(f"unknown op {op}")
    # stages in dynamic chunks: every workgroup holds the same record, and the pools' chunk
    # ranges cover the rows exactly once
    for (op, l), recs in dyn.items():
        assert len(recs) == nwg and len(set(recs)) == 1, (op, l)
        rc, packed = recs[0]
        cover.setdefault((op, l), []).extend(dyn_chunk_rows(rows[op], rc, packed & 255, packed >> 8, nwg))
    assert s.n_dyn_stages == len(dyn)
    # every row / item / group exactly once
    for l in range(L):
        for op, n in ((OP_QKV, rows[OP_QKV]), (OP_OPROJ, rows[OP_OPROJ]), (OP_GU, rows[OP_GU]),
                      (OP_DOWN, rows[OP_DOWN]), (OP_ATTN, P)):
            iv = sorted(cover[(op, l)])
            assert iv[0][0] == 0 and iv[-1][1] == n and all(x[1] == y[0] for x, y in zip(iv, iv[1:])), (op, l)
    iv = sorted(cover[(OP_LM, L)])
    assert iv[0][0] == 0 and iv[-1][1] == rows[OP_LM] and all(x[1] == y[0] for x, y in zip(iv, iv[1:]))
    # each queue follows the one global (layer, stage) order
    for w in range(nwg):
        keys = [_order_key(int(o), int(l), L) for o, l, _, _ in ins[qoff[w]:qoff[w + 1]]]
        assert keys == sorted(keys), f"queue {w} is out of topological order"
    # structural gates
    assert s.n_types >= 5
    assert s.min_instr_per_layer >= 6
    assert s.n_counters >= 4 * L
    assert s.n_stages == 5 * L + 1
    # imbalance in weight bytes per queue, recomputed from the exported queues
    cols = _gemv_cols(cfg)
    per = np.zeros(nwg)
    for w in range(nwg):
        for o, l, a, bb in ins[qoff[w]:qoff[w + 1]]:
            if int(o) in cols:
                # a dynamic stage counts its mean share
                per[w] += (rows[int(o)] / nwg if a < 0 else bb - a) * cols[int(o)] * 2
    assert abs(per.max() - s.max_bytes_per_cu) <= 1e-6 * per.max()
    assert abs(per.mean() - s.mean_bytes_per_cu) <= 1e-6 * per.mean()
    return s, qoff, ins


@pytest.mark.parametrize("name", FULL)
def test_plan_full_shapes(fm, name):
    cfg = _with_ctx(get_config(name))
    s, _, _ = check_plan(cfg, 256, fm)
    assert s.imbalance <= 1.35, f"queue imbalance {s.imbalance:.3f}"


@pytest.mark.parametrize("name", ["toy-gpu", "mini-qwen3", "mini-llama3", "mini-llama2", "mini-qwen3-b4",
                                  "mini-llama2-b8"])
@pytest.mark.parametrize("nwg", [1, 7, 256])
def test_plan_small_shapes(fm, name, nwg):
    check_plan(_with_ctx(get_config(name)), nwg, fm)


def simulate(cfg, qoff, ins, P):
    """Run all queues with coarse dependencies (a superset of what the kernel waits on):
    QKV(l) needs all of DOWN(l-1); ATTN(l) all of QKV(l); OPROJ(l) all of ATTN(l) (the merge
    runs inside the group's last item); GU(l) all of OPROJ(l); DOWN(l) all of GU(l); LM all of
    DOWN(L-1).
    Returns True when every queue drains."""
    L = cfg["n_layers"]
    total, done = {}, {}
    for o, l, _, _ in ins:
        total[(int(o), int(l))] = total.get((int(o), int(l)), 0) + 1
    prev = {OP_ATTN: OP_QKV, OP_OPROJ: OP_ATTN, OP_GU: OP_OPROJ, OP_DOWN: OP_GU}

    def ready(o, l):
        if o == OP_QKV:
            return l == 0 or done.get((OP_DOWN, l - 1), 0) == total[(OP_DOWN, l - 1)]
        if o == OP_LM:
            return done.get((OP_DOWN, L - 1), 0) == total[(OP_DOWN, L - 1)]
        p = prev[o]
        return done.get((p, l), 0) == total[(p, l)]

    nwg = len(qoff) - 1
    head = [int(qoff[w]) for w in range(nwg)]
    progress = True
    while progress:
        progress = False
        for w in range(nwg):
            while head[w] < qoff[w + 1]:
                o, l = int(ins[head[w]][0]), int(ins[head[w]][1])
                if not ready(o, l):
                    break
                done[(o, l)] = done.get((o, l), 0) + 1
                head[w] += 1
                progress = True
    return all(head[w] == qoff[w + 1] for w in range(nwg))


@pytest.mark.parametrize("name,nwg", [("llama3.2-1b", 256), ("qwen3-8b", 256), ("llama2-13b", 256),
                                      ("mini-qwen3-b4", 5), ("toy-gpu", 1), ("mini-llama2-b8", 33)])
def test_schedule_drains(fm, name, nwg):
    cfg = _with_ctx(get_config(name))
    s = fm.plan_query(cfg, nwg)
    qoff, ins = fm.plan_export(cfg, nwg)
    assert simulate(cfg, qoff, ins, s.attn_items)


def test_simulator_detects_a_cycle(fm):
    """The simulator itself: swapping two instructions of different stages inside a single
    queue (so that a workgroup waits on work queued behind it) must be reported as stuck."""
    cfg = _with_ctx(get_config("toy-gpu"))
    qoff, ins = fm.plan_export(cfg, 1)
    bad = ins.copy()
    i_qkv = int(np.where(bad[:, 0] == OP_QKV)[0][0])
    i_down = int(np.where(bad[:, 0] == OP_DOWN)[0][0])
    bad[[i_qkv, i_down]] = bad[[i_down, i_qkv]]
    assert simulate(cfg, qoff, ins, 0)
    assert not simulate(cfg, qoff, bad, 0)
