"""Exact-arithmetic proof of the shortcuts the GPU row quantizer takes.

(Q = 1 in the reciprocal sequence is the quantizer variants' binary16
metadata: r = RN32(1/s) for a stored binary16 scale s.)

The quantizer of the "standard symmetric" scheme (Sec. 8) needs, per row with
absmax a (a positive finite binary16 value) and Q in {7, 127}:
    scale = RN32(a / Q),  r = RN32(Q / a),  code = clamp(rne(RN32(x r)), -Q, Q).
The GPU kernels compute the two quotients without a full division:
    scale:  s0 = RN(a c), e = RN(a - s0 Q), scale = RN(s0 + e c),  c = RN32(1/Q)
    r:      r0 = hardware reciprocal of a (within 1 ulp), q0 = RN(Q r0),
            e = RN(Q - q0 a), r = RN(q0 + e r0)
(one Newton-Raphson correction of the quotient, Markstein's scheme; each RN of
an expression with one product is a fused multiply-add), and they skip the
clamp.  This test checks, in exact rational arithmetic, for every positive
finite binary16 a and both Q, that both sequences give the correctly rounded
quotient for any r0 within 2 ulp of 1/a, and that |RN32(x r)| < Q + 1/2 for
|x| <= a, so the clamp never changes a code.  The GPU parity tests then check
the kernels bit for bit against the oracle, which divides and clamps.
"""
from fractions import Fraction

import pytest


def _rn32(x: Fraction) -> Fraction:
    """x rounded to the nearest binary32 value, ties to even (normal range)."""
    if x == 0:
        return Fraction(0)
    neg = x < 0
    p, q = abs(x.numerator), x.denominator
    e = p.bit_length() - q.bit_length()
    if (p << max(0, -e)) < (q << max(0, e)):
        e -= 1
    assert -126 <= e <= 127
    shift = 23 - e  # significand n = round(x * 2^shift), 2^23 <= n < 2^24
    num, den = (p << shift, q) if shift >= 0 else (p, q << -shift)
    n, rem = divmod(num, den)
    if 2 * rem > den or (2 * rem == den and n & 1):
        n += 1
    out = Fraction(n) / Fraction(2) ** shift if shift >= 0 else Fraction(n * 2 ** -shift)
    return -out if neg else out


def _ulp32(x: Fraction) -> Fraction:
    p, q = x.numerator, x.denominator
    e = p.bit_length() - q.bit_length()
    if (p << max(0, -e)) < (q << max(0, e)):
        e -= 1
    return Fraction(2) ** (e - 23)


def _half(h: int) -> Fraction:
    e, f = h >> 10, h & 0x3FF
    if e == 0:
        return Fraction(f, 1 << 24)
    return Fraction(1024 + f) * Fraction(2) ** (e - 25)


def _positive_halves():
    return range(1, 0x7C00)  # every positive subnormal and normal binary16 value


def test_rn32_helper_matches_numpy():
    np = pytest.importorskip("numpy")
    rng = np.random.default_rng(0)
    for v in rng.standard_normal(2000) * 10.0 ** rng.integers(-20, 20, 2000):
        assert float(_rn32(Fraction(float(v)))) == float(np.float32(v))


@pytest.mark.parametrize("Q", [7, 127])
def test_scale_sequence_is_correctly_rounded(Q):
    c = _rn32(Fraction(1, Q))
    for h in _positive_halves():
        a = _half(h)
        s0 = _rn32(a * c)
        e = _rn32(a - s0 * Q)
        assert _rn32(s0 + e * c) == _rn32(a / Q), hex(h)


@pytest.mark.parametrize("Q", [1, 7, 127])
def test_reciprocal_sequence_is_correctly_rounded(Q):
    for h in _positive_halves():
        a = _half(h)
        want = _rn32(Fraction(Q) / a)
        ra = _rn32(1 / a)
        u = _ulp32(ra)
        for k in (-2, -1, 0, 1, 2):
            r0 = ra + k * u
            if k < 0 and _ulp32(r0) < u:  # below a power of two the spacing halves
                r0 = ra + k * u / 2
            q0 = _rn32(Q * r0)
            e = _rn32(Q - q0 * a)
            assert _rn32(q0 + e * r0) == want, (hex(h), k)


@pytest.mark.parametrize("Q", [7, 127])
def test_clamp_never_binds(Q):
    for h in _positive_halves():
        a = _half(h)
        r = _rn32(Fraction(Q) / a)
        assert _rn32(a * r) < Q + Fraction(1, 2), hex(h)  # |x| <= a and RN is monotone


def test_binary32_quotient_sequences_exhaustive(tmp_path):
    """The asymmetric quantizer variants divide a binary32 group range by M
    and M by the range (M in {15, 255}), the cold-tier upgrade's INT8 residual
    a binary32 maximum by 127 and 127 by it.  The GPU computes RN32(a/M) with
    the scale sequence above and RN32(M/a) with the reciprocal sequence after
    one refinement of the reciprocal, y = RN(r0 + RN(1 - a r0) r0), and skips
    the code clamp because RN32(a RN32(M/a)) < M + 1/2.
    tests/native/quotient_sweep.c checks both against IEEE division for every
    binary32 significand in [1, 2) and any r0 within 2 ulp of RN(1/range)
    (plus three other binades: both sequences commute with scaling by powers
    of two while every intermediate stays normal, which holds for ranges in
    [2^-24, 2^17]).  Built with gcc, correctly rounded fmaf, no contraction."""
    import os
    import subprocess
    src = os.path.join(os.path.dirname(__file__), "native", "quotient_sweep.c")
    exe = str(tmp_path / "quotient_sweep")
    subprocess.run(["gcc", "-O2", "-ffp-contract=off", "-fno-fast-math", "-o", exe, src, "-lm"], check=True)
    for lo, hi in ((0, 1), (-24, -23), (-10, -9), (16, 17)):
        res = subprocess.run([exe, str(lo), str(hi)], capture_output=True, text=True)
        assert res.returncode == 0, res.stdout + res.stderr
        assert res.stdout.strip().endswith(" 0 failures"), res.stdout
