"""The parity checker used by the GPU tests (tests/_gpu.py) applies the bar
as stated: bit-exact codes except elements within one ulp of a rounding
boundary, at most 1e-6 of the elements, never more than one level off;
headers within 1e-6 relative; float results within 1e-5 relative L2."""
import numpy as np
import pytest

import oracle
from tests._gpu import check_codes, check_f32, check_headers


def _case(n=1 << 21):
    r = np.random.default_rng(0)
    x = r.standard_normal(n).astype(np.float32)
    q, s, pre = oracle.quant_sym(x, 128, 8)
    return x, q, s, pre


def test_identical_codes_pass():
    _, q, _, pre = _case()
    assert check_codes(q.view(np.uint8), q.view(np.uint8), pre, q.size, 8) == 0


def test_mismatch_at_a_tie_is_allowed_once_per_million():
    _, q, _, pre = _case()
    pre = pre.copy()
    i = 1234
    pre[i] = np.float32(np.floor(pre[i]) + 0.5)            # make element i a tie
    got = q.copy()
    got[i] = q[i] + (1 if q[i] < 127 else -1)
    assert check_codes(got.view(np.uint8), q.view(np.uint8), pre, q.size, 8) == 1


def test_mismatch_away_from_a_tie_fails():
    _, q, _, pre = _case()
    got = q.copy()
    i = int(np.argmin(np.abs(np.abs(pre - np.round(pre)) - 0.25)))   # a value far from any .5
    got[i] = q[i] + (1 if q[i] < 127 else -1)
    with pytest.raises(AssertionError):
        check_codes(got.view(np.uint8), q.view(np.uint8), pre, q.size, 8)


def test_too_many_tie_mismatches_fail():
    _, q, _, pre = _case(1 << 20)                          # 1e-6 of 2^20 allows one
    pre = pre.copy()
    got = q.copy()
    for i in (10, 20):
        pre[i] = np.float32(np.floor(pre[i]) + 0.5)
        got[i] = q[i] + (1 if q[i] < 127 else -1)
    with pytest.raises(AssertionError):
        check_codes(got.view(np.uint8), q.view(np.uint8), pre, q.size, 8)


def test_two_level_jump_fails_even_at_a_tie():
    _, q, _, pre = _case()
    pre = pre.copy()
    pre[5] = np.float32(np.floor(pre[5]) + 0.5)
    got = q.copy()
    got[5] = q[5] + (2 if q[5] < 120 else -2)
    with pytest.raises(AssertionError):
        check_codes(got.view(np.uint8), q.view(np.uint8), pre, q.size, 8)


def test_header_and_float_tolerances():
    s = np.array([1.0, 2.0, 0.0], np.float32)
    check_headers(s, s)
    check_headers(s * np.float32(1 + 2e-7), s, exact=False)
    with pytest.raises(AssertionError):
        check_headers(s * np.float32(1 + 2e-6), s, exact=False)
    with pytest.raises(AssertionError):
        check_headers(s * np.float32(1 + 2e-7), s)            # bit-exact mode
    f = np.random.default_rng(1).standard_normal(1000).astype(np.float32)
    check_f32(f * np.float32(1 + 5e-7), f, exact=False)
    with pytest.raises(AssertionError):
        check_f32(f * np.float32(1 + 1e-4), f, exact=False)
    with pytest.raises(AssertionError):
        check_f32(np.where(np.arange(1000) == 3, np.inf, f).astype(np.float32), f, exact=False)
