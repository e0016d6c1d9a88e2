"""The seeded generators: reproducible, range-independent, and shaped like
the stated recipes (these are inputs, not results of the method)."""
import numpy as np

import synth


def test_range_independence_and_determinism():
    w = synth.WORKLOADS["c3"]
    full = synth.gradient(w, 0, 3 * synth.CHUNK)
    part = synth.gradient(w, synth.CHUNK - 100, 300)
    assert np.array_equal(part, full[synth.CHUNK - 100:synth.CHUNK + 200])
    assert np.array_equal(full, synth.gradient(w, 0, 3 * synth.CHUNK))
    assert not np.array_equal(synth.gradient(w, 0, 1000, peer=0), synth.gradient(w, 0, 1000, peer=1))


def test_uniform_outlier_recipe():
    w = synth.WORKLOADS["c1"]
    g = synth.gradient(w, 0, w.n)
    assert g.dtype == np.float32 and g.size == w.n
    # 0.1% of positions carry x100 outliers: the 1049 largest are them
    big = np.sort(np.abs(g))[::-1]
    assert big[0] > 20 * 1e-4 * 3
    core = np.abs(g) < 6e-4
    assert abs(np.std(g[core]) - 1e-4) < 1e-5


def test_layered_recipe_has_channel_outliers():
    w = synth.WORKLOADS["c3"]
    sig, chans = synth._layer_layout(w, 0)
    assert len(sig) == 4 and all(len(c) == 10 for c in chans)
    assert np.all((sig >= 1e-6) & (sig <= 1e-3))
    g = synth.gradient(w, 0, 1 << 20)
    col = np.arange(g.size) % w.hidden
    m = np.isin(col, chans[0])
    ratio = np.std(g[m]) / np.std(g[~m])
    assert 40 < ratio < 60


def test_weights_recipes():
    w2 = synth.WORKLOADS["c2"]
    d = synth.weight_diff(w2, 0, 1 << 20)
    assert abs(np.std(d.astype(np.float64)) - 5e-4) < 5e-5
    k = np.mean((d.astype(np.float64) / 5e-4) ** 4)     # heavy tails (t3: infinite kurtosis)
    assert k > 5
    w4 = synth.WORKLOADS["c4"]
    p = synth.prev_weights(w4, 0, 4096)
    assert p.dtype == np.uint16
    f = synth.bf16_bits_to_f32(p)
    assert abs(np.std(f) - 0.02) < 2e-3
    nw = synth.new_weights(w4, 0, 4096, prev=p)
    assert nw.dtype == np.float32 and np.std(nw - f) < 1e-3
