"""Alg. 3 with the oracle: on a noisy least-squares problem with 8 simulated
workers, SGD whose gradients go through the two-level path (TLq-HS) and
whose model weights are communicated as 4-bit weight differences (qWD)
reaches the same loss as full precision, while direct 4-bit weight
quantization (qW) stalls far above it -- the qualitative result of the
paper's Table 1 and Sec. 4.1, reproduced on the compression path."""
import pytest

from tests._alg3 import OracleBackend, Problem, train


@pytest.fixture(scope="module")
def runs():
    pb = Problem()
    be = OracleBackend(pb)
    out = {m: train(pb, be, m, 40, 0.7) for m in ("full", "qwd", "qw")}
    out["exact"] = train(pb, be, "full", 40, 0.7, compress_grads=False)
    return out


def test_sdp4bit_matches_full_precision(runs):
    floor = runs["exact"][-1]
    assert runs["exact"][0] > 1e4 * floor                   # the problem is far from solved at start
    assert runs["full"][-1] <= floor * 1.01                 # TLq-HS gradients alone
    assert runs["qwd"][-1] <= floor * 1.01                  # qWD + TLq-HS (SDP4Bit)


def test_direct_weight_quantization_stalls(runs):
    floor = runs["exact"][-1]
    assert runs["qw"][-1] > 100 * floor
    assert min(runs["qw"][10:]) > 100 * floor
