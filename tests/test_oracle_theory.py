"""Pins from the paper's analysis (Sec. 4): the counterexample of Sec. 4.1
(a worked example with printed values, stored in tests/golden/), Alg. 3's
weight-difference update, and the delta-approximate compressor inequality.
"""
import json
import os

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "counterexample_sec4_1.json")


def ternary(w):
    """The nearest ternary quantizer of Sec. 4.1 = symmetric quantizer with k = 2 bits."""
    w = np.asarray(w, np.float32)
    q, s, _ = oracle.quant_sym(w, w.size, 2)
    return oracle.dequant_sym(q, s, w.size)


def test_golden_one_step_values():
    gold = json.load(open(GOLDEN))
    w0 = np.array(gold["w_init"], np.float32)
    for eta in (0.01, 0.05, 0.1, 0.12):
        assert eta < gold["eta_bound"]
        pre_a = np.array([1 - 4 * eta, -1], np.float32)    # after g = (4 w1, 0)
        pre_b = np.array([1, -1 + 4 * eta], np.float32)    # after g = (0, 4 w2)
        for pre in (pre_a, pre_b):
            assert np.array_equal(ternary(pre), np.array(gold["quantized_after_one_step"], np.float32))
        # the quantizer itself: s = max|w|, q = round(w / s) * s
        assert np.array_equal(ternary(w0), w0)


def _grad(w, coin):
    return np.array([4 * w[0], 0], np.float32) if coin else np.array([0, 4 * w[1]], np.float32)


def test_direct_weight_quantization_is_stuck():
    gold = json.load(open(GOLDEN))
    coins = np.random.default_rng(0).integers(0, 2, 300)
    eta = np.float32(0.1)
    w = np.array(gold["w_init"], np.float32)
    for c in coins:
        w = ternary(w - eta * _grad(w, c))
        assert np.array_equal(w, np.array(gold["w_init"], np.float32))


def test_weight_difference_quantization_converges():
    """Alg. 3: w_t = w_{t-1} - eta g(w~_{t-1}); w~_t = w~_{t-1} + C(w_t - w~_{t-1})."""
    gold = json.load(open(GOLDEN))
    coins = np.random.default_rng(0).integers(0, 2, 300)
    eta = np.float32(0.1)
    w = np.array(gold["w_init"], np.float32)
    wt = w.copy()
    for c in coins:
        w = (w - eta * _grad(wt, c)).astype(np.float32)
        wt = (wt + ternary(w - wt)).astype(np.float32)
    assert np.linalg.norm(wt) < 1e-6


def test_alg3_error_feedback_with_qwd_codec():
    """qWD encode/decode as C_w in Alg. 3 on least squares: the model weights
    track the main weights within half a quantization step and converge."""
    r = np.random.default_rng(1)
    n, group = 512, 128
    A = r.standard_normal((64, n)).astype(np.float32) / 8
    wstar = r.standard_normal(n).astype(np.float32)
    b = A @ wstar
    w = np.zeros(n, np.float32)          # main weights (fp32)
    wt = np.zeros(n, np.float32)         # model weights = previously communicated
    eta = np.float32(0.05)
    loss0 = np.linalg.norm(A @ wt - b)
    for _ in range(400):
        g = (A.T @ (A @ wt - b)).astype(np.float32)
        w = (w - eta * g).astype(np.float32)
        codes, s, m, _ = oracle.qwd_encode(w, wt, group)
        wt = oracle.qwd_decode(codes, s, m, wt, group)
        step = np.repeat(s, group)
        assert np.all(np.abs(w - wt) <= step / 2 * (1 + 2 ** -10) + 4 * np.spacing(np.abs(w)))
    assert np.linalg.norm(A @ wt - b) < 1e-3 * loss0


@pytest.mark.parametrize("group", [64, 128, 2048])
def test_asym4_is_a_delta_approximate_compressor(group):
    """Definition (delta-approximate): ||C(v) - v||^2 <= (1 - delta) ||v||^2, delta in (0, 1]."""
    import synth
    w = synth.WORKLOADS["c2"]
    v = synth.weight_diff(w, 0, 1 << 16)
    q, s, m, _ = oracle.quant_asym4(v, group)
    err = np.sum((oracle.dequant_asym4(q, s, m, group).astype(np.float64) - v) ** 2)
    ratio = err / np.sum(v.astype(np.float64) ** 2)
    assert 0 < ratio < 0.2
