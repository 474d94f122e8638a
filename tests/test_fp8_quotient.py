"""Host model of the fp8 quotient the assembly kernel forms: x / scale as
q0 = RN(x * inv), r = RN(x - q0 * scale) (one fused multiply-add), q = RN(q0 +
r * inv) (another), with inv = RN(1 / scale), keeping q0 where it is zero or
not finite (Markstein's correction step).  The E4M3 codes of q must equal the
codes of the IEEE fp32 quotient — the oracle's quantiser of x with this scale —
for every finite bf16 x.

Each fused operation is modelled exactly: x * inv and q0 * scale are exact in
fp64 (24-bit by 24-bit products), x - q0 * scale is exact in fp64 where the
remainder matters, and q0 + r * inv is rounded to fp32 through long double,
with results that land exactly on an fp32 midpoint redone in rationals.
"""
from fractions import Fraction

import numpy as np

import oracle


def _rn32_exact(vals_ld, q1, exact_of):
    """Redo double-rounding cases: where the long double sum sits exactly on an
    fp32 midpoint, round the exact value instead (ties to even)."""
    lo = q1.astype(np.longdouble)
    up = np.nextafter(q1, np.float32(np.inf)).astype(np.longdouble)
    dn = np.nextafter(q1, np.float32(-np.inf)).astype(np.longdouble)
    onmid = (vals_ld == (lo + up) / 2) | (vals_ld == (lo + dn) / 2)
    for i in np.nonzero(onmid)[0]:
        ex = exact_of(i)
        cands = [q1[i], np.nextafter(q1[i], np.float32(-np.inf)), np.nextafter(q1[i], np.float32(np.inf))]
        dist = [abs(Fraction(float(c)) - ex) for c in cands]
        best = [c for c, d in zip(cands, dist) if d == min(dist)]
        q1[i] = best[0] if len(best) == 1 else [c for c in best if (int(c.view(np.uint32)) & 1) == 0][0]
    return q1


def _corrected_quotient(xb, b):
    inv = np.float32(1) / b
    xs = xb.astype(np.float64)
    with np.errstate(over="ignore", invalid="ignore"):
        q0 = (xs * np.float64(inv)).astype(np.float32)
        r = (xs - q0.astype(np.float64) * np.float64(b)).astype(np.float32)
        s = q0.astype(np.longdouble) + r.astype(np.longdouble) * np.longdouble(inv)
        q1 = s.astype(np.float32)
    q1 = _rn32_exact(s, q1, lambda i: Fraction(float(q0[i])) + Fraction(float(r[i])) * Fraction(float(inv)))
    keep = ~np.isfinite(q0) | (q0 == 0)
    return np.where(keep, q0, q1).astype(np.float32)


def test_corrected_quotient_gives_the_division_codes():
    # every finite bf16 value of both signs, zeros included
    bits = np.arange(0, 0x7f80, dtype=np.uint32)
    pos = (bits << 16).view(np.float32)
    xb = np.concatenate([pos, -pos])
    rng = np.random.default_rng(11)
    # scales: amax / 448 for random bf16 maxima (the data-driven scales),
    # random magnitudes, and powers of two with their neighbours
    amax = (rng.integers(0x3400, 0x4c00, 256, dtype=np.uint32) << 16).view(np.float32)
    scales = list((amax / np.float32(448)).astype(np.float32))
    scales += list((2.0 ** rng.uniform(-16, 16, 64)).astype(np.float32))
    for e in range(-20, 21, 4):
        p = np.float32(2.0 ** e)
        scales += [p, np.nextafter(p, np.float32(0)), np.nextafter(p, np.float32(np.inf))]
    assert len(scales) == 353
    for b in scales:
        q = _corrected_quotient(xb, np.float32(b))
        got = oracle.quantize(q.astype(np.float64), 1.0)  # codes of the fp32 value q itself
        want = oracle.quantize(xb.astype(np.float64), float(b))
        assert np.array_equal(got, want), (float(b), int(np.sum(got != want)))
