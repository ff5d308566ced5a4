"""Pins of the oracle's SAS (Sec. 4; Appendix B, Algorithm 3) against closed forms.

The paper prints no worked example and no error bound for SAS.  What it fixes:
the decomposition e^{-y} = LUT(int part) * POLY(fraction), the cubic's
coefficients, the [0, 1] fit range and the threshold n_r = -6 (scores more
than 6 below the maximum give 0).  The checks below compare against the
exact exponential (numpy) with bounds that the printed coefficients imply,
so a wrong coefficient, sign, LUT entry, index or threshold fails one of them.
"""
import numpy as np
import pytest


def test_lut_is_rounded_exp(orc):
    for k in range(7):
        assert orc.lut(k) == np.float32(np.exp(-k)), k


def test_poly_close_to_exp_on_unit_interval(orc):
    f = np.linspace(0.0, 1.0, 200001, dtype=np.float32)
    p = orc.poly(f).astype(np.float64)
    e = np.exp(-f.astype(np.float64))
    # A least-squares cubic of e^{-x} on [0, 1] with 4-digit coefficients:
    # absolute error below 5e-4 everywhere, relative below 1.1e-3.
    assert np.max(np.abs(p - e)) < 5e-4
    assert np.max(np.abs(p - e) / e) < 1.1e-3
    # The largest deviations sit at the interval ends (0.9996 at 0).
    assert orc.poly(np.float32([0.0]))[0] == np.float32(0.9996)


@pytest.mark.parametrize("seed", [0, 1])
def test_sas_relative_error_on_kept_range(orc, seed):
    rng = np.random.default_rng(seed)
    y = np.concatenate([rng.uniform(0, 6, 100000), np.arange(0, 7, dtype=np.float64),
                        np.linspace(0, 6, 6001)]).astype(np.float32)
    y = y[y <= 6]
    s = orc.sas_y(y).astype(np.float64)
    e = np.exp(-y.astype(np.float64))
    # LUT is e^{-k} rounded to binary32 (rel 6e-8) times POLY (rel < 1.1e-3),
    # plus one binary32 rounding of the product.
    assert np.max(np.abs(s - e) / e) < 1.1e-3


def test_sas_threshold(orc):
    # x < n_r = -6 gives exactly 0; x = -6 is kept.
    ys = np.float32([6.0, np.nextafter(np.float32(6), np.float32(7)), 6.5, 6.9999, 7.0, 50.0, 1e30])
    out = orc.sas_y(ys)
    assert out[0] > 0 and out[0] == np.float32(np.float32(np.exp(-6)) * np.float32(0.9996))
    assert np.all(out[1:] == 0)


def test_sas_at_zero_and_sign_convention(orc):
    assert orc.sas_y(np.float32([0.0]))[0] == np.float32(0.9996)
    x = np.float32([-0.25, -1.5, -5.75])
    assert np.array_equal(orc.sas(x), orc.sas_y(-x))


def test_sas_integer_steps_and_non_monotone_jump(orc):
    """At integer y the table steps: SAS(k) = LUT[k] * POLY(0) exactly, and it
    sits slightly above the limit from below LUT[k-1] * POLY(1^-), because
    POLY(1) ~ 0.3675 < e^{-1} * POLY(0).  SAS is therefore not monotone;
    nothing downstream may rely on monotonicity."""
    for k in range(1, 7):
        at = orc.sas_y(np.float32([k]))[0]
        below = orc.sas_y(np.float32([np.nextafter(np.float32(k), np.float32(0))]))[0]
        assert at == np.float32(np.float32(np.exp(-k)) * np.float32(0.9996))
        assert at > below


def test_sas_fraction_split(orc):
    """SAS(y) for y = k + f equals LUT[k] * POLY(f) (product in binary32)."""
    rng = np.random.default_rng(3)
    k = rng.integers(0, 6, 1000)
    f = rng.uniform(0, 1, 1000).astype(np.float32)
    y = (k.astype(np.float32) + f).astype(np.float32)
    f_exact = (y - np.floor(y)).astype(np.float32)
    lut = np.float32(np.exp(-np.floor(y).astype(np.float64))).astype(np.float32)
    expect = (lut * orc.poly(f_exact)).astype(np.float32)
    assert np.array_equal(orc.sas_y(y), expect)


def test_algorithm3_row_softmax(orc):
    rng = np.random.default_rng(5)
    x = (rng.standard_normal((64, 96)) * np.where(np.arange(64) < 32, 0.7, 3.0)[:, None]).astype(np.float32)
    p = orc.sas_softmax_rows(x)
    assert np.allclose(p.sum(axis=1), 1.0, atol=1e-12)
    d = x - x.max(axis=1, keepdims=True)
    assert np.all(p[d < -6] == 0)
    assert np.all(p[d >= -6] > 0)
    # rows with nothing dropped match the exact softmax within the SAS bound
    keep = (d >= -6).all(axis=1)
    ex = np.exp(d.astype(np.float64))
    ex /= ex.sum(axis=1, keepdims=True)
    assert keep.sum() > 3
    assert np.max(np.abs(p[keep] - ex[keep]) / ex[keep]) < 2.3e-3
