"""Pins of the CPU oracle against what the paper and the mathematics fix.

None of these tests re-types the oracle's formulas: each checks the oracle
against a library routine, a brute force over tiny inputs, a closed form, an
invariant or a value the paper prints (tests/golden/).
"""
import os
from fractions import Fraction

import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_2208_01944_amd import inputs as I

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden_rows(name):
    rows = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                rows.append(line.split())
    return rows


# ---------------------------------------------------------------------------
# Quantiser (Section 3.2, Eq. 2-3)
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("bits", [2, 3, 4, 8])
def test_quantize_endpoints_and_lattice(bits):
    s = (1 << bits) - 1
    # Eq. 2 clip: everything at or below l maps to 0, at or above u to 2^b-1
    x = np.array([-1e30, -5.0, -1.0, 0.0, float(s), s + 1.0, 1e30], np.float32)
    q = O.quantize(x, 0.0, float(s), bits)
    assert q.tolist() == [0, 0, 0, 0, s, s, s]
    # with l=0, u=2^b-1 every integer level is its own code
    lv = np.arange(s + 1, dtype=np.float32)
    assert O.quantize(lv, 0.0, float(s), bits).tolist() == list(range(s + 1))
    # signed codes are the unsigned ones shifted by 2^(b-1)
    assert O.quantize(lv, 0.0, float(s), bits, signed=True).tolist() == \
        [v - (1 << (bits - 1)) for v in range(s + 1)]


def test_quantize_ties_round_half_even():
    # l=0, u=3, b=2: y = x exactly for these x; halves go to the even code
    x = np.array([0.5, 1.5, 2.5], np.float32)
    assert O.quantize(x, 0.0, 3.0, 2).tolist() == [0, 2, 2]


def test_quantize_special_values():
    x = np.array([np.nan, np.inf, -np.inf, -0.0, 0.0], np.float32)
    assert O.quantize(x, 0.0, 1.0, 2).tolist() == [0, 3, 0, 0, 0]


@pytest.mark.parametrize("bits", [2, 3, 4, 8])
def test_quantize_matches_exact_rational_away_from_ties(bits):
    """Against the exact rational value of Eq. 2: the fp32 pipeline may only
    differ from round-to-nearest of the exact quotient where that quotient
    lies within a few fp32 ulps of a half-integer."""
    g = np.random.default_rng(7 + bits)
    x = g.normal(0.0, 2.0, 4000).astype(np.float32)
    l, u = np.float32(-2.5), np.float32(3.25)
    q = O.quantize(x, l, u, bits)
    s = (1 << bits) - 1
    for xi, qi in zip(x.tolist(), q.tolist()):
        t = (Fraction(xi) - Fraction(float(l))) / (Fraction(float(u)) - Fraction(float(l)))
        t = min(max(t, Fraction(0)), Fraction(1))
        y = t * s
        fl = y.numerator // y.denominator
        frac = y - fl
        if abs(frac - Fraction(1, 2)) < Fraction(1, 1 << 18):
            assert qi in (fl, fl + 1)
        else:
            assert qi == (fl + 1 if frac > Fraction(1, 2) else fl)


@pytest.mark.parametrize("bits", [2, 3, 4])
def test_quantize_round_trip_bound_and_monotone(bits):
    """Eq. 3 inverts Eq. 2 to within half a step; Eq. 2 is monotone."""
    g = np.random.default_rng(3)
    x = np.sort(g.uniform(-1, 2, 5000).astype(np.float32))
    l, u = 0.0, 1.0
    q = O.quantize(x, l, u, bits)
    assert np.all(np.diff(q) >= 0)
    xn = np.clip((x.astype(np.float64) - l) / (u - l), 0, 1)
    deq = O.dequantize(q, bits, "activation")
    assert np.max(np.abs(deq - xn)) <= 0.5 / ((1 << bits) - 1) + 1e-6
    # weight de-quantiser lands in [-1, 1] with both ends reached
    wq = O.dequantize(np.arange((1 << bits)), bits, "weight")
    assert wq.min() == -1.0 and wq.max() == 1.0


def test_calibrate_range_ignores_nan():
    x = np.array([np.nan, -3.0, 2.0, np.nan, 0.5], np.float32)
    assert O.calibrate_range(x) == (np.float32(-3.0), np.float32(2.0))


# ---------------------------------------------------------------------------
# Grouped convolution (Eq. 1 per group, Section 4.1)
# ---------------------------------------------------------------------------
def _torch_group_conv(x, w, stride, pad):
    """torch conv2d in float64 on integer data: exact because every partial
    sum is an integer below 2^53."""
    g, co, kh, kw, ci = w.shape
    xt = torch.from_numpy(np.asarray(x, np.float64)).permute(0, 3, 1, 2)
    wt = torch.from_numpy(np.asarray(w, np.float64)).reshape(g * co, kh, kw, ci).permute(0, 3, 1, 2)
    y = torch.nn.functional.conv2d(xt, wt.contiguous(), stride=stride, padding=pad, groups=g)
    return y.permute(0, 2, 3, 1).numpy().astype(np.int64)


@pytest.mark.parametrize("case", [
    dict(n=2, h=9, w=7, g=3, ci=5, co=4, k=3, s=1, p=1, b=2),
    dict(n=1, h=13, w=13, g=2, ci=16, co=8, k=3, s=2, p=1, b=2),
    dict(n=2, h=8, w=6, g=4, ci=3, co=5, k=1, s=2, p=0, b=4),
    dict(n=1, h=11, w=10, g=1, ci=3, co=6, k=7, s=2, p=3, b=8),
    dict(n=3, h=5, w=5, g=2, ci=7, co=3, k=3, s=1, p=0, b=3),
])
def test_group_conv_matches_torch_float64(case):
    g = np.random.default_rng(11)
    b = case["b"]
    sgn = b == 8
    x = I.codes(g, (case["n"], case["h"], case["w"], case["g"] * case["ci"]), b, sgn)
    w = I.codes(g, (case["g"], case["co"], case["k"], case["k"], case["ci"]), b, True)
    acc = O.group_conv(x, w, case["s"], case["p"])
    np.testing.assert_array_equal(acc, _torch_group_conv(x, w, case["s"], case["p"]))


def test_group_conv_brute_force_tiny():
    """Every output of a tiny conv by Python-int summation over the window."""
    g = np.random.default_rng(5)
    x = g.integers(-8, 8, (1, 4, 3, 4))
    w = g.integers(-8, 8, (2, 3, 3, 2, 2))
    acc = O.group_conv(x, w, 1, 1)
    n, h, wd, _ = x.shape
    G, co, kh, kw, ci = w.shape
    for oy in range(acc.shape[1]):
        for ox in range(acc.shape[2]):
            for gg in range(G):
                for k in range(co):
                    s = 0
                    for ky in range(kh):
                        for kx in range(kw):
                            iy, ix = oy - 1 + ky, ox - 1 + kx
                            if 0 <= iy < h and 0 <= ix < wd:
                                for c in range(ci):
                                    s += int(x[0, iy, ix, gg * ci + c]) * int(w[gg, k, ky, kx, c])
                    assert acc[0, oy, ox, gg * co + k] == s


def test_group_conv_exhaustive_small_k():
    """1x1 conv on one pixel with K=3 channels: every pair of 2-bit code
    vectors gives the textbook dot product."""
    import itertools
    vals_a, vals_w = range(4), range(-2, 2)
    xs = np.array(list(itertools.product(vals_a, repeat=3)))         # 64 inputs
    ws = np.array(list(itertools.product(vals_w, repeat=3)))         # 64 filters
    x = xs.reshape(64, 1, 1, 3)
    w = ws.reshape(1, 64, 1, 1, 3)
    acc = O.group_conv(x, w, 1, 0).reshape(64, 64)
    np.testing.assert_array_equal(acc, xs @ ws.T)


def test_group_conv_equals_block_diagonal_dense_and_g1():
    """A G-group conv equals a G=1 conv whose weight is block diagonal, and
    each group equals an ordinary conv on its channel slice."""
    g = np.random.default_rng(2)
    G, ci, co = 3, 4, 5
    x = g.integers(0, 4, (2, 6, 6, G * ci))
    w = g.integers(-2, 2, (G, co, 3, 3, ci))
    dense = np.zeros((1, G * co, 3, 3, G * ci), np.int64)
    for gg in range(G):
        dense[0, gg * co:(gg + 1) * co, :, :, gg * ci:(gg + 1) * ci] = w[gg]
    a = O.group_conv(x, w, 1, 1)
    np.testing.assert_array_equal(a, O.group_conv(x, dense, 1, 1))
    for gg in range(G):
        one = O.group_conv(x[..., gg * ci:(gg + 1) * ci], w[gg:gg + 1], 1, 1)
        np.testing.assert_array_equal(a[..., gg * co:(gg + 1) * co], one)


def test_group_conv_impulse_returns_weights():
    g = np.random.default_rng(4)
    w = g.integers(-2, 2, (2, 3, 3, 3, 4))
    x = np.zeros((1, 7, 7, 8), np.int64)
    y0, x0, c0 = 3, 4, 5  # group 1, channel 1
    x[0, y0, x0, c0] = 1
    acc = O.group_conv(x, w, 1, 1)
    for oy in range(7):
        for ox in range(7):
            ky, kx = y0 - oy + 1, x0 - ox + 1
            want = np.zeros(6, np.int64)
            if 0 <= ky < 3 and 0 <= kx < 3:
                want[3:6] = w[1, :, ky, kx, 1]
            np.testing.assert_array_equal(acc[0, oy, ox], want)


def test_bit_decomposition_identity_eq4():
    """Eq. 4: an M-bit product equals the shifted sum of all G^2 B-bit chunk
    products (exact integer identity, M=4 and M=6 with B=2)."""
    g = np.random.default_rng(9)
    for m_bits, b in ((4, 2), (6, 2), (6, 3)):
        G = -(-m_bits // b)
        x = g.integers(0, 1 << m_bits, (1, 5, 5, 3))
        w = g.integers(0, 1 << m_bits, (1, 2, 3, 3, 3))
        full = O.group_conv(x, w, 1, 1)
        acc = np.zeros_like(full)
        for i in range(G):
            xi = (x >> (i * b)) & ((1 << b) - 1)
            for j in range(G):
                wj = (w >> (j * b)) & ((1 << b) - 1)
                acc += O.group_conv(xi, wj, 1, 1) << ((i + j) * b)
        np.testing.assert_array_equal(acc, full)


def test_bit_chunk_footnote():
    for v, bits, lo, hi in _golden_rows("bit_chunk_footnote.txt"):
        v = int(v)
        assert format(v, "04b") == bits
        assert v & 3 == int(lo) and v >> 2 == int(hi)


# ---------------------------------------------------------------------------
# Requantisation
# ---------------------------------------------------------------------------
def test_requant_closed_forms():
    m = np.array([3, 16384, 32767], np.int64)
    for sh in (1, 5, 20, 30):
        for k in range(0, 4):
            # t*M = k * 2^sh exactly -> code k (clamped to 2 bits)
            for mi in m:
                if (k << sh) % mi == 0:
                    t = (k << sh) // mi
                    assert O.requant(np.array([t]), mi, sh, 2)[0] == min(k, 3)
    # half-way values round up (floor(x + 1/2))
    assert O.requant(np.array([1]), 1, 1, 4)[0] == 1       # 0.5 -> 1
    assert O.requant(np.array([3]), 1, 1, 4)[0] == 2       # 1.5 -> 2
    assert O.requant(np.array([-1]), 1, 1, 4)[0] == 0      # -0.5 -> 0 (ReLU)
    assert O.requant(np.array([5]), 1, 0 + 2, 4)[0] == 1   # 1.25 -> 1
    # out_bits 32 is the identity on t
    t = np.array([-5, 0, 7 << 20])
    np.testing.assert_array_equal(O.requant(t, 1, 1, 32), t)


def test_requant_matches_rational_rounding_and_saturates():
    g = np.random.default_rng(1)
    t = g.integers(-(1 << 20), 1 << 20, 3000)
    m = g.integers(1 << 14, 1 << 15, 3000)
    for sh, bits in ((20, 2), (21, 3), (23, 4), (30, 2)):
        q = O.requant(t, m, sh, bits)
        for ti, mi, qi in zip(t.tolist(), m.tolist(), q.tolist()):
            v = Fraction(ti * mi, 1 << sh) + Fraction(1, 2)
            want = v.numerator // v.denominator
            assert qi == min(max(want, 0), (1 << bits) - 1)
        srt = np.sort(t)
        assert np.all(np.diff(O.requant(srt, 20000, sh, bits)) >= 0)


# ---------------------------------------------------------------------------
# Cyclic permutation (Eq. 6-8) and Proposition 1
# ---------------------------------------------------------------------------
def test_cyclic_two_line_notation_golden():
    for row in _golden_rows("cyclic_two_line.txt"):
        G = int(row[0])
        image = [int(v) for v in row[1:]]
        # channel c of group i must land in group image[i]
        x = np.repeat(np.arange(G), 3)[None, :]         # group id as the value
        y = O.cyclic_permute(x, G, 1).reshape(G, 3)
        for i in range(G):
            assert np.all(y[image[i]] == i)


@pytest.mark.parametrize("G", [1, 2, 3, 4, 5])
def test_cyclic_invariants(G):
    c = 3
    x = np.arange(2 * G * c).reshape(2, G * c)
    # bijection: a permutation of the channels, nothing lost or duplicated
    for s in range(-G - 1, 2 * G + 2):
        y = O.cyclic_permute(x, G, s)
        assert sorted(y[0].tolist()) == sorted(x[0].tolist())
    # pi^G = id, composition adds steps, G=1 identity
    np.testing.assert_array_equal(O.cyclic_permute(x, G, G), x)
    for a in range(G + 2):
        for b in range(G + 2):
            np.testing.assert_array_equal(
                O.cyclic_permute(O.cyclic_permute(x, G, a), G, b), O.cyclic_permute(x, G, a + b))
    # no group stays in place for 0 < s < G
    for s in range(1, G):
        y = O.cyclic_permute(x, G, s).reshape(2, G, c)
        for i in range(G):
            assert not np.array_equal(y[:, i], x.reshape(2, G, c)[:, i])


@pytest.mark.parametrize("G", [2, 3, 4, 6])
def test_proposition1_reachability(G):
    """Z = X + Conv1x1(pi(X)) (Eq. 9-10) with strictly positive 1x1 group
    weights: an impulse in group i reaches groups {i, ..., i+k} after k
    modules and every group after G-1 modules (Proposition 1)."""
    c = 2
    w = np.ones((G, c, 1, 1, c), np.int64)
    for i in range(G):
        x = np.zeros((1, 1, 1, G * c), np.int64)
        x[0, 0, 0, i * c] = 1
        for k in range(1, G):
            x = x + O.group_conv(O.cyclic_permute(x, G, 1), w, 1, 0)
            nz = {gg for gg in range(G) if np.any(x[0, 0, 0, gg * c:(gg + 1) * c] != 0)}
            assert nz == {(i + j) % G for j in range(k + 1)}
        assert len(nz) == G


@pytest.mark.parametrize("G", [2, 3, 4])
def test_shuffle_module_proposition1(G):
    """The integer module (Eq. 9-10) with positive 1x1 weights and an
    identity-like requant (M = 2^14, shift 14, 8-bit output): an impulse in
    group i reaches exactly groups i..i+k after k modules, all groups after
    G-1 (Proposition 1)."""
    c = 3
    w = np.ones((G, c, 1, 1, c), np.int64)
    mult = np.full(G * c, 1 << 14)
    shift = np.full(G * c, 14)
    rm = np.ones(G * c, np.int64)
    for i in range(G):
        x = np.zeros((1, 2, 2, G * c), np.int64)
        x[0, 1, 0, i * c + 1] = 1
        for k in range(1, G):
            x, _ = O.shuffle_module(x, w, mult, shift, None, rm, 8)
            nz = {gg for gg in range(G) if np.any(x[..., gg * c:(gg + 1) * c])}
            assert nz == {(i + j) % G for j in range(k + 1)}
        assert len(nz) == G


def test_shuffle_module_special_cases():
    g = np.random.default_rng(5)
    G, c = 3, 4
    x = g.integers(0, 4, (2, 3, 5, G * c))
    w = g.integers(-2, 2, (G, c, 1, 1, c))
    mult = g.integers(1 << 14, 1 << 15, G * c)
    shift = np.full(G * c, 12)
    bias = g.integers(-50, 50, G * c)
    rm = g.integers(1, 8, G * c)
    # zero weights: only the (scaled) shortcut and the bias remain
    q0, acc0 = O.shuffle_module(x, np.zeros_like(w), mult, shift, bias, rm, 2)
    assert not acc0.any()
    np.testing.assert_array_equal(q0, O.requant(bias + rm * x, mult, shift, 2))
    # zero shortcut scale: the 1x1 conv of the input one group back
    q1, acc1 = O.shuffle_module(x, w, mult, shift, bias, np.zeros(G * c, np.int64), 2)
    xv = x.reshape(2, 3, 5, G, c)
    for j in range(G):
        ref = np.einsum("nhwc,kc->nhwk", xv[..., (j - 1) % G, :], w[j, :, 0, 0, :])
        np.testing.assert_array_equal(acc1[..., j * c:(j + 1) * c], ref)
    # G = 1: the permutation is the identity, so the module is a 1x1 layer
    # with an identity shortcut taken from its own input
    w1 = w[:1]
    q2, acc2 = O.shuffle_module(x[..., :c], w1, mult[:c], shift[:c], bias[:c], rm[:c], 2)
    q3, acc3 = O.conv_layer(x[..., :c], w1, 1, 0, mult[:c], shift[:c], bias[:c], 2, shuffle=0,
                            res=x[..., :c], res_mult=rm[:c])
    np.testing.assert_array_equal(q2, q3)
    np.testing.assert_array_equal(acc2, acc3)


@pytest.mark.parametrize("G", [1, 2, 3, 4])
def test_shuffle_module_is_a_rotated_layer(G):
    """The reading the GPU path uses: the module equals a 1x1 layer that
    writes its branch one group on (Eq. 8 as the store address) with the
    identity shortcut from its own input, when its per-group parameters are
    rotated by one group (layer group g takes module group g + 1)."""
    g = np.random.default_rng(G)
    c = 5
    x = g.integers(0, 4, (2, 4, 3, G * c))
    w = g.integers(-2, 2, (G, c, 1, 1, c))
    mult = g.integers(1 << 14, 1 << 15, G * c)
    shift = np.full(G * c, 12)
    bias = g.integers(-40, 40, G * c)
    rm = g.integers(1, 16, G * c)
    q, acc = O.shuffle_module(x, w, mult, shift, bias, rm, 2)
    rot = lambda a: np.roll(np.asarray(a).reshape(G, -1), -1, axis=0).reshape(np.asarray(a).shape)
    wr = np.roll(w, -1, axis=0)
    q2, acc2 = O.conv_layer(x, wr, 1, 0, rot(mult), rot(shift), rot(bias), 2, shuffle=1, res=x,
                            res_mult=rot(rm))
    np.testing.assert_array_equal(q, q2)
    np.testing.assert_array_equal(acc, acc2)


def test_channel_shuffle_definition_and_inverse():
    # two groups of three: a0 a1 a2 | b0 b1 b2 -> a0 b0 a1 b1 a2 b2
    x = np.arange(6)[None, :]
    np.testing.assert_array_equal(O.channel_shuffle(x, 2), [[0, 3, 1, 4, 2, 5]])
    g = np.random.default_rng(9)
    for G, C in ((1, 5), (2, 4), (3, 7), (4, 64), (6, 2)):
        x = g.integers(0, 16, (2, 3, G * C))
        y = O.channel_shuffle(x, G)
        # a permutation of each pixel's channels ...
        np.testing.assert_array_equal(np.sort(y, axis=-1), np.sort(x, axis=-1))
        # ... undone by the shuffle with the roles of G and C^ exchanged
        np.testing.assert_array_equal(O.channel_shuffle(y, C), x)
        if G == 1:
            np.testing.assert_array_equal(y, x)
        # output group 0 holds the first C^/G channels of every group, in turn
        if C % G == 0:
            v = x.reshape(2, 3, G, C)
            np.testing.assert_array_equal(y[..., :G], v[..., :, 0])


def test_conv_layer_shuffle_writes_branch_one_group_on():
    """With an identity residual and zero weights in all groups but one, only
    the destination group (g+s) mod G changes."""
    g = np.random.default_rng(0)
    G, ci, co = 4, 3, 3
    x = g.integers(0, 4, (1, 4, 4, G * ci))
    w = np.zeros((G, co, 3, 3, ci), np.int64)
    w[1] = g.integers(1, 2, (co, 3, 3, ci))   # only source group 1 is non-zero
    res = np.zeros((1, 4, 4, G * co), np.int64)
    mult = np.full(G * co, 1 << 14)
    shift = np.full(G * co, 14)
    q, acc = O.conv_layer(x, w, 1, 1, mult, shift, None, 8, shuffle=1, res=res,
                          res_mult=np.ones(G * co, np.int64))
    nz = {gg for gg in range(G) if np.any(q[..., gg * co:(gg + 1) * co])}
    assert nz == {2}
    # and the accumulator there is the plain conv of source group 1
    plain = O.group_conv(x, w, 1, 1)
    np.testing.assert_array_equal(acc[..., 2 * co:3 * co], plain[..., co:2 * co])


@pytest.mark.parametrize("G,shuffle", [(4, 1), (4, 3), (4, -1), (3, 2), (2, 1)])
def test_conv_layer_projection_shortcut_independent(G, shuffle):
    """The projection shortcut (reading A10): destination group j receives the
    main branch of source group (j - s) mod G with that source channel's
    bias, M and shift (Eq. 8 moves the branch), plus the raw accumulator of
    the 1x1, stride-s, pad-0 conv of the block input's OWN group j with the
    projection filter of group j, not permuted.  Rebuilt here from torch
    float64 convolutions (one per destination group for the projection) and
    Python-int requantisation, and compared with conv_layer's acc and codes.
    An odd input size with stride 2 makes a wrong projection stride, pad or
    pixel index visible; distinct groups make a source/destination mix-up
    visible."""
    g = np.random.default_rng(40 + G * 10 + shuffle)
    ci, co, cp, h, stride = 5, 3, 6, 9, 2
    x = I.codes(g, (2, h, h, G * ci), 2, False)
    w = I.codes(g, (G, co, 3, 3, ci), 2, True)
    px = I.codes(g, (2, h, h, G * cp), 2, False)
    pw = I.codes(g, (G, co, 1, 1, cp), 2, True)
    mult = g.integers(1 << 14, 1 << 15, G * co)
    shift = np.full(G * co, 13)
    bias = g.integers(20, 90, G * co)
    q, acc = O.conv_layer(x, w, stride, 1, mult, shift, bias, 8, shuffle=shuffle,
                          proj_x=px, proj_w=pw, proj_stride=stride)
    main = _torch_group_conv(x, w, stride, 1)                     # source channel order
    ho = main.shape[1]
    assert acc.shape == (2, ho, ho, G * co)
    want_acc = np.zeros_like(main)
    want_q = np.zeros_like(main)
    for j in range(G):
        src = (j - shuffle) % G
        pj = _torch_group_conv(px[..., j * cp:(j + 1) * cp], pw[j:j + 1], stride, 0)
        assert pj.shape == (2, ho, ho, co)
        for k in range(co):
            cs, cd = src * co + k, j * co + k
            want_acc[..., cd] = main[..., cs] + pj[..., k]
            for idx in np.ndindex(2, ho, ho):
                t = int(main[idx + (cs,)]) + int(bias[cs]) + int(pj[idx + (k,)])
                m, sh = int(mult[cs]), int(shift[cs])
                want_q[idx + (cd,)] = min(max((t * m + (1 << (sh - 1))) >> sh, 0), 255)
    np.testing.assert_array_equal(acc, want_acc)
    np.testing.assert_array_equal(q, want_q)
    assert len(np.unique(want_q)) > 10  # the codes are not degenerate


def test_layer_epilogue_and_centring_single_pass():
    """conv_layer is group_conv followed by layer_epilogue, and the
    one-pass calibrate_centring returns the logits run_net gives on the
    centred network (identity and projection shortcuts, shuffles)."""
    spec = I.resnet18(n=2, groups=2, bits=2, hw=32, classes=10, seed=3, stages=(1, 1, 1, 1))
    cen, logits = O.calibrate_centring(spec, spec["x"], return_logits=True)
    np.testing.assert_array_equal(logits, O.run_net(cen, spec["x"]))
    assert O.calibrate_centring(spec, spec["x"])["layers"][2]["bias"].tolist() == \
        cen["layers"][2]["bias"].tolist()
    _, tensors, _ = O.run_net(cen, spec["x"], keep=True)
    for L in cen["layers"]:
        if L["op"] == "conv" and L["src"] > 0:
            codes = tensors[L["dst"]]
            assert len(np.unique(codes)) >= 3, L["dst"]   # not degenerate (1x1 maps at stage 4)
    case = I.single_layer(9, n=1, h=6, w=6, groups=3, cin=4, cout=5, residual="identity", shuffle=2)
    L = case["layer"]
    a = O.conv_layer(case["x"], L["w"], 1, 1, L["mult"], L["shift"], L["bias"], 2, 2,
                     res=case["extra"][1], res_mult=L["res_mult"])
    b = O.layer_epilogue(O.group_conv(case["x"], L["w"], 1, 1), 3, L["mult"], L["shift"], L["bias"],
                         2, 2, res=case["extra"][1], res_mult=L["res_mult"])
    np.testing.assert_array_equal(a[0], b[0])
    np.testing.assert_array_equal(a[1], b[1])


# ---------------------------------------------------------------------------
# Glue: pooling, sum, FC
# ---------------------------------------------------------------------------
def test_maxpool_commutes_with_monotone_requant():
    g = np.random.default_rng(8)
    t = g.integers(-3000, 3000, (2, 9, 9, 4))
    m = np.full(4, 20000)
    sh = np.full(4, 20)
    a = O.maxpool(O.requant(t, m, sh, 2), 3, 2, 1)
    b = O.requant(O.maxpool(t, 3, 2, 1), m, sh, 2)
    np.testing.assert_array_equal(a, b)


def test_maxpool_brute_force():
    g = np.random.default_rng(6)
    x = g.integers(0, 4, (1, 5, 6, 2))
    y = O.maxpool(x, 3, 2, 1)
    assert y.shape == (1, 3, 3, 2)
    for oy in range(3):
        for ox in range(3):
            for c in range(2):
                vals = [x[0, iy, ix, c] for iy in range(2 * oy - 1, 2 * oy + 2)
                        for ix in range(2 * ox - 1, 2 * ox + 2) if 0 <= iy < 5 and 0 <= ix < 6]
                assert y[0, oy, ox, c] == max(vals)


def test_avgsum_and_fc_closed_forms():
    x = np.full((2, 7, 7, 5), 3)
    s = O.avgsum(x)
    assert np.all(s == 147)
    w = np.ones((4, 5), np.int64)
    np.testing.assert_array_equal(O.fc(s, w), np.full((2, 4), 147 * 5))
    g = np.random.default_rng(3)
    a = g.integers(0, 148, (3, 6))
    b = g.integers(-128, 128, (2, 6))
    want = [[sum(int(a[i, c]) * int(b[o, c]) for c in range(6)) for o in range(2)] for i in range(3)]
    assert O.fc(a, b).tolist() == want


# ---------------------------------------------------------------------------
# BitOps (Appendix B) against the values the paper prints
# ---------------------------------------------------------------------------
def _net_macs(stages, groups, modules: bool):
    """MAC count of the ResNet layer list the input generator builds (stem,
    grouped 3x3 convs, grouped 1x1 projections, FC and, with modules, the
    cyclic-shuffle modules it places at the start of stages 2-4)."""
    G = max(groups, 1)
    net = I.resnet18(n=1, groups=G, bits=2, stages=stages, modules=modules)
    h = 224
    shapes = {0: (224, 224, 3)}
    macs = 0
    for L in net["layers"]:
        sh = shapes[L["src"]]
        if L["op"] == "conv":
            gg, co, k, _, ci = L["w"].shape
            ho = O.out_size(sh[0], k, L["stride"], L["pad"])
            macs += O.layer_macs(gg * ci, gg * co, gg, k, ho, ho)
            if L.get("proj_w") is not None:
                pg, pco, _, _, pci = L["proj_w"].shape
                macs += O.layer_macs(pg * pci, pg * pco, pg, 1, ho, ho)
            shapes[L["dst"]] = (ho, ho, gg * co)
        elif L["op"] == "shuffle_module":
            gg, co, _, _, ci = L["w"].shape
            macs += O.layer_macs(gg * ci, gg * co, gg, 1, sh[0], sh[1])
            shapes[L["dst"]] = sh
        elif L["op"] == "maxpool":
            ho = O.out_size(sh[0], L["k"], L["stride"], L["pad"])
            shapes[L["dst"]] = (ho, ho, sh[2])
        elif L["op"] == "avgsum":
            shapes[L["dst"]] = (1, 1, sh[2])
        elif L["op"] == "fc":
            macs += O.layer_macs(L["w"].shape[1], L["w"].shape[0], 1, 1, 1, 1)
    del h
    return macs


def test_bitops_match_paper_tables():
    stages = {"resnet18": (2, 2, 2, 2), "resnet34": (3, 4, 6, 3)}
    cache = {}
    for net, B, G, dense, printed, *src in _golden_rows("bitops.txt"):
        B, G, dense, printed = int(B), int(G), int(dense), float(printed)
        key = (net, G)
        if key not in cache:
            cache[key] = _net_macs(stages[net], G, modules=G > 0)
        macs = cache[key]
        got = O.bitops(macs, dense or B, dense or B) / 1e9
        assert abs(got - printed) / printed < 0.005, (net, B, G, dense, got, printed, " ".join(src))


# ---------------------------------------------------------------------------
# Stored inputs: the benchmark networks' centred biases
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("name", ["resnet18_g4_b2", "resnet18_g4_b2_shuffles", "resnet50_g2_b2"])
def test_stored_centred_biases_match_oracle_calibration(name):
    """tests/golden/centred_bias_<name>.npz holds what the oracle's centring
    calibration gives today on the workload's calibration images (so the
    benchmark times, and the full-size tests check, the centred network the
    oracle defines)."""
    import importlib.util
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "make_centred_bias.py")
    spec_m = importlib.util.spec_from_file_location("make_centred_bias", path)
    mk = importlib.util.module_from_spec(spec_m)
    spec_m.loader.exec_module(mk)
    cen, calib = mk.calibrate(name)
    stored = I.with_stored_biases(I.workload(name)[0], name)
    with np.load(I.centred_path(name), allow_pickle=False) as z:
        assert z["calib_images"].tolist() == list(calib)
    n_conv = 0
    for L, S in zip(cen["layers"], stored["layers"]):
        if L["op"] == "conv":
            np.testing.assert_array_equal(S["bias"], L["bias"])
            n_conv += 1
    assert n_conv >= 17  # ResNet-18: stem + 16 (projections are fused)
