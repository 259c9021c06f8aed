"""The FP4 kernel's fp32 requant, checked on the CPU.  With u = t + bias
(+ the identity shortcut) the kernel's accumulator holds u / 4 and one fp32
fma computes y = RN(u/4 * M 2^(2 - sh) + 1/2), a single rounding of
x = (u M + 2^(sh-1)) 2^-sh; it stores min(trunc(y), 3).  For the bounds the
device checks before taking this path (1 <= sh <= 22, |M| < 2^24,
|u| < 2^24) that equals the requant's definition clamp(floor(x), 0, 3)
(the reading of the fixed-point requant with 2-bit outputs).  x is exact in
float64 here (|u M| < 2^48) and numpy's float64 -> float32 conversion
rounds it once to nearest even, as the fma does."""
import numpy as np


def _definition(u, m, sh):
    num = u * m + (1 << (sh - 1))
    return np.clip(np.floor_divide(num, 1 << sh), 0, 3)


def _fp32_path(u, m, sh):
    x = (u.astype(np.float64) * float(m) + 2.0 ** (sh - 1)) / 2.0 ** sh  # exact
    y = x.astype(np.float32).astype(np.float64)                          # one rounding
    return np.minimum(np.where(y > 0, np.trunc(y), 0.0), 3.0).astype(np.int64)


def _cases(m, sh, rng):
    """u near every step of the 2-bit staircase (both sides of each
    threshold), at the ends of the range and at random."""
    us = [np.arange(-3000, 3001)]
    if m != 0:
        for k in range(1, 4):
            th = -(-((2 * k - 1) << (sh - 1)) // m)  # ceil, the step to code k for m > 0
            us.append(np.arange(th - 3000, th + 3001))
    us.append(np.array([-(1 << 24) + 1, (1 << 24) - 1]))
    us.append(rng.integers(-(1 << 24) + 1, 1 << 24, 20000))
    u = np.concatenate(us).astype(np.int64)
    return u[np.abs(u) < (1 << 24)]


MULTS = [1, 2, 3, 5, 7, 255, 1 << 14, (1 << 14) + 1, (1 << 15) - 1, 46341, (1 << 20) - 3, (1 << 23) + 1,
         (1 << 24) - 1, 0, -1, -((1 << 15) - 1)]


def test_fp32_requant_equals_definition_within_bounds():
    rng = np.random.default_rng(2208)
    for sh in range(1, 23):
        for m in MULTS + [int(v) for v in rng.integers(1, 1 << 24, 4)]:
            u = _cases(m, sh, rng)
            want = _definition(u, m, sh)
            got = _fp32_path(u, m, sh)
            bad = np.nonzero(got != want)[0]
            assert bad.size == 0, (sh, m, u[bad[:5]], got[bad[:5]], want[bad[:5]])


def test_fp32_requant_shift_bound_is_needed():
    """Past the bound a single fp32 rounding can cross a step: for large
    shifts some u rounds up onto the next code, which is why the device
    keeps such layers on the fp64 epilogue."""
    rng = np.random.default_rng(7)
    found = False
    for sh in (26, 27, 28):
        for m in [(1 << 24) - 1, (1 << 23) + 1] + [int(v) for v in rng.integers(1 << 20, 1 << 24, 6)]:
            u = _cases(m, sh, rng)
            if np.any(_fp32_path(u, m, sh) != _definition(u, m, sh)):
                found = True
    assert found
