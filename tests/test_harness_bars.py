"""The GPU harness's acceptance checks are not vacuous (CPU only): the KV rounding window accepts
both roundings of a value within the window and rejects a value moved by a plausible bug."""
import numpy as np

from tests.gpu_harness import kv_slot_ok, f32_to_bf16_rne, TAU


def test_kv_window_accepts_rounding_and_rejects_moves():
    rng = np.random.default_rng(5)
    y = rng.standard_normal((4, 128)).astype(np.float32)
    rms = np.sqrt(np.mean(y.astype(np.float64) ** 2, axis=-1, keepdims=True)).astype(np.float32)
    ok, flips = kv_slot_ok(f32_to_bf16_rne(y), y)
    assert ok and flips == 0
    ok, flips = kv_slot_ok(f32_to_bf16_rne(y + 0.5 * TAU * rms), y)
    assert ok
    # one element off by 1% of the row's rms (a wrong term, a stale value) is caught
    z = y.copy()
    z[2, 17] += 0.01 * rms[2, 0]
    assert not kv_slot_ok(f32_to_bf16_rne(z), y)[0]
    # a swapped pair of elements (a wrong index) is caught
    z = y.copy()
    z[1, [3, 4]] = z[1, [4, 3]]
    assert not kv_slot_ok(f32_to_bf16_rne(z), y)[0]
