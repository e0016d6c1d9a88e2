"""The lane scheme of the fused Hadamard kernels, simulated on the CPU.

The kernels hold 16..64 consecutive elements per lane and relabel lanes
inside each row of 16 (physical lane p holds element lane p ^ (3 * bit2(p))),
so that every cross-lane butterfly partner is a DPP pattern: quad_perm
(p ^ 1, p ^ 2), row_half_mirror (p ^ 7) and row_ror:8 (p ^ 8).  Each
cross-lane stage computes v + sg * partner in every lane (sg = -1 in the upper
lane of a pair), so lanes carry their value up to a known sign, removed by the
final scaling fma(v, +-c_n, +0).  This test runs that scheme in numpy float32
(every operation a single IEEE rounding, as on the device) and checks it
against the oracle's transform bit for bit, zeros included."""
import numpy as np
import pytest

import oracle

f32 = np.float32


def element_lane(p):
    b = (p >> 2) & 1
    return p ^ (b * 3)


# physical partner of element-lane distance D
PHYS_XOR = {1: 1, 2: 2, 4: 7, 8: 8, 16: 16, 32: 32}
DPP_PARTNER = {  # what the DPP controls deliver, lane by lane
    1: lambda p: (p & ~3) | [1, 0, 3, 2][p & 3],          # quad_perm [1,0,3,2]
    2: lambda p: (p & ~3) | [2, 3, 0, 1][p & 3],          # quad_perm [2,3,0,1]
    4: lambda p: (p & ~7) | (7 - (p & 7)),                # row_half_mirror
    8: lambda p: (p & ~15) | ((p + 8) & 15),              # row_ror:8
}


def relabeled_transform(x, E, NB, cn):
    el = np.array([element_lane(p) for p in range(64)])
    v = np.stack([x[E * e:E * e + E] for e in el]).astype(np.float32)
    h = 1
    while h < E:
        for i in range(E):
            if i & h:
                continue
            a, b = v[:, i].copy(), v[:, i + h].copy()
            v[:, i] = a + b
            v[:, i + h] = a - b
        h <<= 1
    D = 1
    while D < NB // E:
        part = np.array([PHYS_XOR[D] ^ p for p in range(64)])
        if D in DPP_PARTNER:
            assert all(DPP_PARTNER[D](p) == part[p] for p in range(64))
        assert all(el[part[p]] == el[p] ^ D for p in range(64))
        sg = np.where(el & D, f32(-1), f32(1)).astype(np.float32)
        v = (v + sg[:, None] * v[part]).astype(np.float32)   # one fma with a +-1 factor: exact product
        D <<= 1
    sign = np.array([-1.0 if bin(e & (NB // E - 1)).count("1") & 1 else 1.0 for e in el], np.float32)
    v = ((v * (sign * cn)[:, None]).astype(np.float32) + f32(0)).astype(np.float32)
    out = np.empty(64 * E, np.float32)
    for p in range(64):
        out[E * el[p]:E * el[p] + E] = v[p]
    return out


def test_element_lane_is_an_involution_mapping_aligned_blocks_to_aligned_blocks():
    """Group reductions run over aligned blocks of physical lanes: the element
    lanes of a group (an aligned block) must sit on one aligned block."""
    assert all(element_lane(element_lane(p)) == p for p in range(64))
    for k in (2, 4, 8, 16, 32, 64):
        for blk in range(64 // k):
            phys = {element_lane(e) for e in range(blk * k, (blk + 1) * k)}
            assert len({p // k for p in phys}) == 1           # one aligned physical block
            if k >= 8:
                assert {p // k for p in phys} == {blk}        # the same block from 8 lanes up


@pytest.mark.parametrize("E,NB", [(E, NB) for E in (16, 32, 64) for NB in (32, 64, 128, 256, 512, 1024) if NB > E])
def test_relabeled_signed_butterfly_equals_oracle(E, NB):
    r = np.random.default_rng(E * 7 + NB)
    cn = oracle.hadamard_scale(NB)
    for trial in range(4):
        x = (r.standard_normal(64 * E) * 10.0 ** r.integers(-30, 30)).astype(np.float32)
        x[r.integers(0, x.size, 40)] = 0.0
        if trial == 3:                           # equal pairs: exact zeros in every other output
            x[1::2] = x[0::2]
        got = relabeled_transform(x, E, NB, cn)
        want = oracle.fwht(x.copy(), NB)
        assert np.array_equal(got.view(np.uint32), want.view(np.uint32))
