"""Run the HIP decode step and the CPU oracle side by side on the same seeded workload.

Both sides start from the same bf16 weights, KV prefill and start tokens (from ``synthetic``).
The reference is the oracle's fp64 instantiation, the float64 golden against which the paper
measures error (Sec. 4.2).

Both sides are teacher-forced at every step:
  * both consume the oracle's greedy token, so a single near-tie cannot make them answer
    different prompts (the paper's reason for teacher forcing);
  * after the step's checks, the GPU's appended KV row is replaced by the oracle's rounding of
    it, so both attend over the same cache at the next step.

The second kind of forcing is needed because each side rounds its own K/V to bf16. The
caches then differ by one-ulp flips in about 1-2% of the appended elements. Attention over
those slots moves the next step's values by far more than either side's arithmetic error.
On the Llama-2-13B b8 shape, the fp32 and fp64 oracle instantiations, each keeping its own
cache, already differ by 0.16 max-abs in the last layer's residual at the second step. That
is above the 3e-2 bar, even though both are correct decoders.
(``force_kv=False`` keeps separate caches.)

Acceptance bars per step:
  * logits and every per-layer tap: max-abs <= 3e-2 and relative L2 <= 1e-2;
  * KV arena: every byte except slot kv_len[i] of each lane is unchanged (bit-exact). The
    slot's bf16 value must round from a value within tau * rms(row) of the reference's
    pre-rounding value (one head row of d_h elements), with tau = 1e-3. The GPU's appended rows
    sit within 3.3e-4 rms of the fp64 values on the full shapes, so tau keeps a 3x margin. Two
    correct decoders that sum in different orders may land on either side of a bf16 rounding
    boundary; such one-step flips are counted, and at most MAX_FLIP_FRAC of a step's appended
    elements may differ from the reference's own rounding;
  * greedy ids: each lane's id is the lowest-index maximum of the GPU's own logits row
    (checked exactly), and it equals the reference's id unless the reference's logit at the
    GPU's id is within 1e-2 of the reference's maximum (a near-tie; any other token fails).
"""
from __future__ import annotations

import math
import time

import numpy as np
import torch

from synthetic import make_workload, as_u16

MAX_ABS = 3e-2
REL_L2 = 1e-2
TAU = 1e-3
TOP2_GAP = 1e-2
# Fraction of a step's appended K/V elements whose bf16 value may differ from the reference's
# own rounding of its fp64 value. The fp32 and fp64 oracle instantiations disagree on 0.2-0.5%
# of them at the full shapes; the GPU, closer to fp64 than the fp32 oracle, stays below that.
MAX_FLIP_FRAC = 2e-2


def check_greedy(gpu_logits_row, gpu_id, ref_logits_row, ref_id, what=""):
    """The greedy-id rule. Returns the reference's gap at the GPU's id when the ids differ
    (a near-tie), else None. Raises AssertionError on a violation."""
    g = np.asarray(gpu_logits_row)
    own = int(np.argmax(g))            # numpy returns the first (lowest-index) maximum
    assert int(gpu_id) == own, f"{what}: next_id {int(gpu_id)} is not the first argmax {own} of the GPU's logits"
    if int(gpu_id) == int(ref_id):
        return None
    ref = np.asarray(ref_logits_row, np.float64)
    gap = float(ref.max() - ref[int(gpu_id)])
    assert gap < TOP2_GAP, f"{what}: token {int(gpu_id)} vs {int(ref_id)}: reference logit {gap:.3g} below its maximum"
    return gap


def to_dev(w: dict) -> dict:
    out = {k: v.cuda() for k, v in w.items() if k != "layers" and v is not None}
    out["layers"] = [{k: v.cuda() for k, v in lw.items()} for lw in w["layers"]]
    return out


def to_u16(w: dict) -> dict:
    out = {k: as_u16(v.cpu()) for k, v in w.items() if k != "layers" and v is not None}
    out["layers"] = [{k: as_u16(v.cpu()) for k, v in lw.items()} for lw in w["layers"]]
    return out


def rel_l2(a, b):
    a = np.asarray(a, np.float64); b = np.asarray(b, np.float64)
    den = np.linalg.norm(b)
    return float(np.linalg.norm(a - b) / den) if den > 0 else float(np.linalg.norm(a - b))


def bf16_bits_to_f32(u):
    return (np.asarray(u, np.uint16).astype(np.uint32) << 16).view(np.float32)


def f32_to_bf16_rne(x):
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(torch.bfloat16)
    return as_u16(t)


def kv_slot_ok(got_u16, y_f32):
    """got: bf16 bits [n_kv][d]; y: oracle fp32 pre-rounding values [n_kv][d]."""
    y = np.asarray(y_f32, np.float32)
    rms = np.sqrt(np.mean(y.astype(np.float64) ** 2, axis=-1, keepdims=True)).astype(np.float32)
    lo = bf16_bits_to_f32(f32_to_bf16_rne(y - TAU * rms))
    hi = bf16_bits_to_f32(f32_to_bf16_rne(y + TAU * rms))
    g = bf16_bits_to_f32(got_u16)
    ok = (g >= lo) & (g <= hi)
    exact = got_u16 == f32_to_bf16_rne(y)
    return bool(ok.all()), int((~exact).sum())


class Pair:
    """A workload loaded on both sides."""

    def __init__(self, name, steps=None, gains="ones", poison=False, n_workgroups=0, attn_items=0, taps=True,
                 cfg_override=None, device="cpu", dyn_chunk_kb=0):
        """``device``: where the seeded inputs are drawn ("cuda" for the full-size shapes)."""
        from oracle.oracle import Oracle
        from paper_2609_12379_amd.fm import Decoder, tap_count
        cfg_in = name
        if cfg_override is not None:
            from synthetic import get_config
            cfg_in = dict(get_config(name), **cfg_override)
        self.wl = make_workload(cfg_in, gains=gains, steps=steps, poison=poison, device=device)
        cfg = self.wl.cfg
        self.cfg = cfg
        self.orc = Oracle(cfg, to_u16(self.wl.weights))
        self.kc_o = [as_u16(t.cpu()).copy() for t in self.wl.kcache]
        self.vc_o = [as_u16(t.cpu()).copy() for t in self.wl.vcache]
        self.wdev = to_dev(self.wl.weights)
        self.kc_d = [t.cuda() for t in self.wl.kcache]
        self.vc_d = [t.cuda() for t in self.wl.vcache]
        self.dec = Decoder(cfg, self.wdev, self.kc_d, self.vc_d, n_workgroups=n_workgroups, attn_items=attn_items,
                           dyn_chunk_kb=dyn_chunk_kb)
        self.taps = None
        if taps:
            self.taps = torch.zeros(tap_count(cfg), dtype=torch.float32, device="cuda")
            self.dec.set_taps(self.taps)
        b, V = cfg["batch"], cfg["vocab"]
        self.logits = torch.zeros((b, V), dtype=torch.float32, device="cuda")
        self.next = torch.zeros(b, dtype=torch.int32, device="cuda")

    def gpu_step(self, tok, pos, kvl, multilaunch=False):
        t = torch.tensor(tok, dtype=torch.int32, device="cuda")
        p = torch.tensor(pos, dtype=torch.int32, device="cuda")
        k = torch.tensor(kvl, dtype=torch.int32, device="cuda")
        self.dec.step(t, p, k, self.logits, self.next, multilaunch=multilaunch)
        torch.cuda.synchronize()
        return self.logits.cpu().numpy().copy(), self.next.cpu().numpy().copy()

    def gpu_taps(self):
        from oracle.oracle import tap_offsets, TAP_NAMES
        cfg = self.cfg
        L, b = cfg["n_layers"], cfg["batch"]
        off = tap_offsets(cfg)
        blk = off["block"]
        buf = self.taps.cpu().numpy()
        body = buf[: L * b * blk].reshape(L, b, blk)
        out = {}
        for k, n in enumerate(TAP_NAMES):
            end = off[TAP_NAMES[k + 1]] if k + 1 < len(TAP_NAMES) else blk
            out[n] = body[:, :, off[n]:end]
        out["final"] = buf[L * b * blk:].reshape(b, cfg["hidden"])
        return out

    def run(self, steps=None, multilaunch=False, check_kv=True, log=None, precision="f64", force_kv=True):
        """Teacher-forced decode; returns a list of per-step report dicts. Raises on failure."""
        cfg = self.cfg
        steps = self.wl.steps if steps is None else steps
        S = self.wl.S
        tok = list(self.wl.start)
        reports = []
        for t in range(steps):
            pos = [s + t for s in S]
            kvl = list(pos)
            if check_kv:
                before = [a.clone() for a in self.kc_d], [a.clone() for a in self.vc_d]
            t0 = time.time()
            r = self.orc.step(self.kc_o, self.vc_o, tok, pos, kvl, precision=precision, taps=True)
            t1 = time.time()
            lg, nx = self.gpu_step(tok, pos, kvl, multilaunch=multilaunch)
            rep = {"step": t, "oracle_s": t1 - t0}
            assert np.isfinite(lg).all(), f"step {t}: non-finite logits"
            rep["logits_max_abs"] = float(np.abs(lg - r.logits).max())
            rep["logits_rel_l2"] = rel_l2(lg, r.logits)
            assert rep["logits_max_abs"] <= MAX_ABS and rep["logits_rel_l2"] <= REL_L2, rep
            if self.taps is not None:
                gt = self.gpu_taps()
                worst = (0.0, 0.0, "")
                for n, ref in r.taps.items():
                    got = gt[n]
                    if n == "final":
                        pairs = [(got, ref)]
                    else:
                        pairs = [(got[l], ref[l]) for l in range(cfg["n_layers"])]
                    for li, (g_, r_) in enumerate(pairs):
                        ma = float(np.abs(g_ - r_).max())
                        rl = rel_l2(g_, r_)
                        assert ma <= MAX_ABS and rl <= REL_L2, f"step {t} tap {n} layer {li}: max-abs {ma} rel-l2 {rl}"
                        if ma > worst[0]:
                            worst = (ma, rl, f"{n}[{li}]")
                rep["worst_tap"] = worst
            # greedy ids
            for i in range(cfg["batch"]):
                gap = check_greedy(lg[i], nx[i], r.logits[i], r.next_ids[i], f"step {t} lane {i}")
                if gap is not None:
                    rep.setdefault("near_ties", []).append((i, gap))
            # KV: strict slot rule and value window
            if check_kv:
                flips, drift = 0, 0.0
                d, nkv = cfg["head_dim"], cfg["n_kv_heads"]
                for l in range(cfg["n_layers"]):
                    for kind, arr_before, arr_dev in (("k", before[0][l], self.kc_d[l]), ("v", before[1][l], self.vc_d[l])):
                        # bit patterns, compared on the device (the full-size arenas are tens of GB)
                        after = arr_dev.view(torch.int16)
                        prev = arr_before.view(torch.int16)
                        for i in range(cfg["batch"]):
                            s_ = kvl[i]
                            assert torch.equal(after[i, :, :s_], prev[i, :, :s_]) and \
                                torch.equal(after[i, :, s_ + 1:], prev[i, :, s_ + 1:]), \
                                f"step {t} layer {l} {kind}: slot outside kv_len written"
                            if kind == "k":
                                y = r.taps["krot"][l, i].reshape(nkv, d)
                            else:
                                y = r.taps["qkv"][l, i][(cfg["n_heads"] + nkv) * d:].reshape(nkv, d)
                            got = after[i, :, s_].cpu().numpy().view(np.uint16)
                            ok, nflip = kv_slot_ok(got, y)
                            if self.taps is not None:
                                gy = gt["krot"][l, i].reshape(nkv, d) if kind == "k" else \
                                    gt["qkv"][l, i][(cfg["n_heads"] + nkv) * d:].reshape(nkv, d)
                                rms = np.sqrt(np.mean(np.asarray(y, np.float64) ** 2, axis=-1, keepdims=True))
                                drift = max(drift, float((np.abs(gy - y) / rms).max()))
                            assert ok, f"step {t} layer {l} lane {i} {kind}: appended values outside the rounding window"
                            flips += nflip
                n_app = 2 * cfg["n_layers"] * cfg["batch"] * nkv * d
                assert flips <= MAX_FLIP_FRAC * n_app, f"step {t}: {flips} of {n_app} appended K/V elements flipped"
                rep["kv_flips"] = flips
                rep["kv_flip_frac"] = flips / n_app
                rep["kv_drift_rms"] = drift
                del before
            if force_kv:
                for l in range(cfg["n_layers"]):
                    for host, dev in ((self.kc_o[l], self.kc_d[l]), (self.vc_o[l], self.vc_d[l])):
                        for i in range(cfg["batch"]):
                            row = np.ascontiguousarray(host[i, :, kvl[i]]).view(np.int16)
                            dev[i, :, kvl[i]].copy_(torch.from_numpy(row).view(torch.bfloat16))
                torch.cuda.synchronize()
            reports.append(rep)
            if log:
                log(rep)
            tok = [int(v) for v in r.next_ids]
        return reports

    def close(self):
        self.dec.close()
