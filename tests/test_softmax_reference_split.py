"""The arithmetic the bf16 attention kernels rely on to subtract a row
statistic inside the score MFMA (Eq. 3's max subtraction; the log-sum-exp of
the backward), checked on the host with a bit-exact emulation of
round-to-nearest-even fp32 -> bf16.

* Forward: the running reference maximum m is applied as two bf16 terms
  hi = rne(m), lo = rne(m - hi).  hi + lo is exact in fp32 (8 + 8 significant
  bits) and within 2^-17 |m| of m, so scores relative to it stay below
  2^(8 + 2^-17 |m|).  A single bf16 reference is off by up to half an ulp,
  128 .. 256 for |m| in [2^15, 2^17): exp2 of a score then overflows fp32.
* Backward: -lse * log2(e) and -Delta are applied as three bf16 terms whose
  sum is the fp32 value exactly (each rounding leaves an exact residue of at
  most 16, then 8, significant bits).
"""
import numpy as np

import synth


def _bf16(x):
    return synth.bf16_round(np.asarray(x, np.float32))


def _samples(n=400_000, seed=0):
    rng = np.random.default_rng(seed)
    mag = np.exp2(rng.uniform(-30.0, 60.0, n))
    return (rng.choice([-1.0, 1.0], n) * rng.uniform(1.0, 2.0, n) * mag).astype(np.float32)


def test_pair_is_exact_in_fp32_and_close():
    x = _samples()
    hi = _bf16(x)
    lo = _bf16((x - hi).astype(np.float32))
    s32 = (hi + lo).astype(np.float32)
    assert np.array_equal(s32.astype(np.float64), hi.astype(np.float64) + lo.astype(np.float64))
    rel = np.abs(x.astype(np.float64) - s32) / np.abs(x.astype(np.float64))
    assert rel.max() <= 2.0 ** -17


def test_three_terms_are_exact():
    x = _samples(seed=1)
    hi = _bf16(x)
    r1 = (x - hi).astype(np.float32)
    assert np.array_equal(r1.astype(np.float64), x.astype(np.float64) - hi.astype(np.float64))
    mid = _bf16(r1)
    r2 = (r1 - mid).astype(np.float32)
    assert np.array_equal(_bf16(r2), r2)                     # the last residue is a bf16 value
    assert np.array_equal(hi.astype(np.float64) + mid + r2, x.astype(np.float64))


def test_single_bf16_reference_overflows_and_pair_does_not():
    rng = np.random.default_rng(2)
    m = (rng.uniform(2.0 ** 15, 2.0 ** 17, 100_000) * rng.choice([-1.0, 1.0], 100_000)).astype(np.float32)
    lazy = 8.0                                             # headroom before the reference moves
    one = _bf16(m).astype(np.float64)
    worst_one = np.max(m.astype(np.float64) - one) + lazy
    assert worst_one > 128.0                               # exp2 beyond the fp32 range
    hi = _bf16(m)
    pair = hi.astype(np.float64) + _bf16((m - hi).astype(np.float32))
    worst_pair = np.max(m.astype(np.float64) - pair) + lazy
    assert worst_pair < 9.0
