"""Pins for per-token decay-gate quantisation (Sec. 3, Decay-gate
quantization: levels uniform in log s per channel; a rate error ds changes
the signal kept at the time constant 1/s by exp(-ds/s))."""
import numpy as np
import pytest

from oracle import stats


def _gates(rng, n=50, dk=128):
    # log-uniform rates over [1e-4, 2] with 10 % slow channels, as the prefill workload
    s = np.exp(rng.uniform(np.log(1e-3), np.log(2.0), (n, dk)))
    slow = rng.random((n, dk)) < 0.1
    s[slow] = np.exp(rng.uniform(np.log(1e-4), np.log(1e-3), slow.sum()))
    return s.astype(np.float32)


@pytest.mark.parametrize("bits", [2, 3, 4])
def test_log_codec_error_is_half_a_step_in_log_space(bits):
    s = _gates(np.random.default_rng(bits))
    q = stats.gate_quantize(s, bits, "log")
    ls = np.log(s.astype(np.float64))
    step = (ls.max(1, keepdims=True) - ls.min(1, keepdims=True)) / (2 ** bits - 1)
    err = np.abs(np.log(q.astype(np.float64)) - ls)
    assert np.all(err <= step / 2 + 1e-6)
    # the extreme channels are levels themselves
    i = np.argmin(s, axis=1)
    assert np.allclose(q[np.arange(len(s)), i], s[np.arange(len(s)), i], rtol=1e-6)
    # 2^bits levels at most per token
    assert max(len(np.unique(r)) for r in q) <= 2 ** bits


@pytest.mark.parametrize("bits", [2, 4])
def test_linear_codec_error_is_half_a_step(bits):
    s = _gates(np.random.default_rng(10 + bits))
    q = stats.gate_quantize(s, bits, "linear")
    step = (s.max(1, keepdims=True).astype(np.float64) - s.min(1, keepdims=True)) / (2 ** bits - 1)
    assert np.all(np.abs(q.astype(np.float64) - s) <= step / 2 * (1 + 1e-6) + 1e-7)


def test_log_levels_keep_slow_channels_relative_error_bounded():
    """The retained-signal factor exp(-ds/s) depends on the relative rate error.
    With log levels it is bounded by e^(step/2) - 1 for every channel and falls
    with the width; with levels uniform in g = -s the slow channels collapse
    onto the lowest level, so their relative error does not fall with more bits
    (the paper: uniform-in-g levels fail even at four bits)."""
    s = _gates(np.random.default_rng(7), n=20)
    slow = s < 1e-3
    ls = np.log(s.astype(np.float64))
    med_log, med_lin = [], []
    for bits in (2, 3, 4):
        ql = stats.gate_quantize(s, bits, "log").astype(np.float64)
        qg = stats.gate_quantize(s, bits, "linear").astype(np.float64)
        rl = np.abs(ql - s) / s
        step = (ls.max(1, keepdims=True) - ls.min(1, keepdims=True)) / (2 ** bits - 1)
        assert np.all(rl <= np.expm1(step / 2) + 1e-6)
        med_log.append(np.median(rl[slow]))
        med_lin.append(np.median((np.abs(qg - s) / s)[slow]))
    assert med_log[0] > med_log[1] > med_log[2] and med_log[2] < 0.2
    assert min(med_lin) > 0.5


def test_constant_gates_and_zero_range():
    s = np.full((3, 64), 0.25, np.float32)
    assert np.array_equal(stats.gate_quantize(s, 2, "log"), s)
    assert np.array_equal(stats.gate_quantize(s, 2, "linear"), s)
