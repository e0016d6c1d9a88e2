"""Chunk routing of the two-level gradient path, and lattice-exact inputs.

Routing (Alg. 4 with the all-to-alls replaced by pointer slicing on one
GPU): GPU (node a, local rank 0) receives chunk 0 of every local peer's
8-bit message; after the 8-bit dequantize-reduce and 4-bit re-quantization,
it receives chunk 0 of the 4-bit message of each of the Q nodes.  Here
``grads[a][b]`` is already chunk 0 (length M) of peer b of node a.
"""
import numpy as np


def oracle_chain(grads, P, Q, group, block, out_scale=1.0):
    import oracle
    M = grads[0][0].size
    level2 = []
    for a in range(Q):
        k1 = [oracle.grad_quant(grads[a][b], 8, block, group) for b in range(P)]
        r = oracle.dequant_reduce([c for c, _, _ in k1], [s for _, s, _ in k1], M, 8, group, 4)
        level2.append((r["codes"], r["scales"]))
    m = M // Q
    codes = [c[:m // 2] for c, _ in level2]
    scales = [s[:m // group] for _, s in level2]
    return oracle.dequant_reduce(codes, scales, m, 4, group, 0, block, out_scale)["f32"]


def _sylvester(n):
    i = np.arange(n)
    pc = np.array([[bin(int(v)).count("1") for v in row] for row in (i[:, None] & i[None, :])])
    return np.where(pc % 2 == 0, 1, -1).astype(np.int64)


def _split(total, m, rng, lim=126):
    """m integers in [-lim, lim] summing to ``total`` (|total| <= 56)."""
    if m == 0:
        assert total == 0
        return []
    if m == 1:
        return [int(total)]
    r = (lim - 56) // (m - 1)
    while True:
        head = rng.integers(-r, r + 1, m - 1)
        last = total - int(head.sum())
        if abs(last) <= lim:
            return [int(v) for v in head] + [last]


def build_lattice_exact_peers(P, Q, group, block, m_out, seed):
    """Peer gradients for which the whole two-level path is lossless and exact.

    In the transformed domain peer (a, b) holds integer codes q times 2^e
    (e fixed per segment of max(group, block) elements), every group of
    every peer reaches |q| = 127 (so the 8-bit scale is exactly 2^e), and
    for every node the peer sum is 8 t with t in [-7, 7] reaching |t| = 7 in
    every group (so the 4-bit scale is exactly 2^(e+3)).  The gradients are
    the inverse transform of that, which is exact for blocks that are powers
    of four.  Returns (grads[a][b] float32 of length m_out*Q, expected
    float64 output of length m_out = the plain sum of all peers).
    """
    assert P % 2 == 0 and block in (0, 1, 4, 16, 64, 256, 1024)
    rng = np.random.default_rng(seed)
    M = m_out * Q
    seg = max(group, block)
    assert M % seg == 0 and m_out % seg == 0
    n_seg = M // seg
    e = rng.integers(-22, -6, n_seg)
    anchors = np.stack([rng.choice(group, P // 2, replace=False) for _ in range(M // group)])
    q = np.zeros((Q, P, M), np.int64)
    for a in range(Q):
        t = rng.integers(-7, 8, M)
        for gi in range(M // group):
            base = gi * group
            t[base + anchors[gi]] = 0
            free = np.setdiff1d(np.arange(group), anchors[gi])
            t[base + rng.choice(free)] = 7 * rng.choice([-1, 1])
        for i in range(M):
            gi, off = divmod(i, group)
            hit = np.nonzero(anchors[gi] == off)[0]
            if hit.size:
                k = int(hit[0])
                others = [b for b in range(P) if b not in (2 * k, 2 * k + 1)]
                q[a, 2 * k, i], q[a, 2 * k + 1, i] = 127, -127
                for b, v in zip(others, _split(8 * t[i], len(others), rng)):
                    q[a, b, i] = v
            else:
                q[a, :, i] = _split(8 * t[i], P, rng)
    assert np.abs(q).max() <= 127
    scale = np.repeat(np.ldexp(1.0, e), seg)                      # 2^e per element
    ghat = q.astype(np.float64) * scale                            # transformed-domain values
    if block:
        H = _sylvester(block)
        s = int(round(np.sqrt(block)))
        g = (q.reshape(Q, P, -1, block) @ H.T).reshape(Q, P, M).astype(np.float64) * scale / s
    else:
        g = ghat
    g32 = g.astype(np.float32)
    assert np.array_equal(g32.astype(np.float64), g)               # exactly representable
    grads = [[g32[a, b].copy() for b in range(P)] for a in range(Q)]
    want = g[:, :, :m_out].sum(axis=(0, 1))
    return grads, want
