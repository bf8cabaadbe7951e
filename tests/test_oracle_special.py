"""Pins of the oracle's special functions and of the Beta KL divergence.

Reference values come from textbook identities (tests/golden/special_values.json),
from mpmath / scipy (independent library routines), and from numerical
quadrature of the Beta density of the paper's Eq. 3.
"""

import json
import math
import os

import mpmath
import numpy as np
import pytest
import scipy.special as sp

from oracle import oracle as O

GOLDEN = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "special_values.json")))


@pytest.mark.parametrize("row", GOLDEN["digamma"], ids=lambda r: f"psi({r['x']})")
def test_oracle_digamma_textbook(row):
    assert O.digamma(row["x"]) == pytest.approx(row["value"], abs=1e-14)


def test_oracle_digamma_recurrence_and_mpmath():
    rng = np.random.default_rng(11)
    xs = np.concatenate([rng.uniform(0.05, 2.0, 200), rng.uniform(2.0, 50.0, 200),
                         np.exp(rng.uniform(np.log(50), np.log(1e3), 50)), [0.05, 9.999999, 10.0]])
    for x in xs:
        # psi(x + 1) = psi(x) + 1/x (A&S 6.3.5)
        assert O.digamma(x + 1.0) - O.digamma(x) == pytest.approx(1.0 / x, rel=1e-12, abs=1e-13)
        ref = float(mpmath.digamma(mpmath.mpf(float(x))))
        assert abs(O.digamma(x) - ref) <= 2e-14 * max(1.0, abs(ref))
    # psi(0.05) = -20.4978449913 (mpmath)
    assert O.digamma(0.05) == pytest.approx(-20.497844991299, abs=1e-11)


def test_oracle_lgamma_matches_scipy():
    xs = np.concatenate([np.linspace(0.05, 5, 97), np.linspace(5, 2000, 53)])
    for x in xs:
        assert O.lgamma(x) == pytest.approx(float(sp.gammaln(x)), rel=1e-14, abs=1e-14)
    # ln B(a, b) = ln Gamma(a) + ln Gamma(b) - ln Gamma(a + b); B(2,3) = 1/12
    assert O.lnbeta(2.0, 3.0) == pytest.approx(-math.log(12.0), abs=1e-15)
    assert O.lnbeta(1.0, 1.0) == pytest.approx(0.0, abs=1e-15)


@pytest.mark.parametrize("row", GOLDEN["kl_beta"], ids=lambda r: f"{r['p']}||{r['q']}")
def test_oracle_kl_closed_forms(row):
    (a1, b1), (a2, b2) = row["p"], row["q"]
    assert O.kl_beta(a1, b1, a2, b2) == pytest.approx(row["value"], abs=1e-14)


def test_oracle_kl_uniform_closed_form():
    # KL(Beta(1,1) || Beta(a,b)) = ln B(a,b) + a + b - 2, because E_U[ln x] = -1.
    rng = np.random.default_rng(5)
    for a, b in rng.uniform(0.05, 8.0, size=(50, 2)):
        expect = float(mpmath.log(mpmath.beta(a, b))) + a + b - 2.0
        assert O.kl_beta(1.0, 1.0, a, b) == pytest.approx(expect, abs=1e-12)


def test_oracle_kl_self_and_direction():
    rng = np.random.default_rng(6)
    for a, b in rng.uniform(0.05, 20.0, size=(50, 2)):
        assert abs(O.kl_beta(a, b, a, b)) < 1e-12
    # the divergence is asymmetric: the argument order matters
    assert O.kl_beta(1, 1, 2, 3) != pytest.approx(O.kl_beta(2, 3, 1, 1), abs=0.1)


def _kl_quadrature(a1, b1, a2, b2):
    """KL by integrating p ln(p/q) with the Beta densities of Eq. 3."""
    mpmath.mp.dps = 30
    B1 = mpmath.beta(a1, b1)
    B2 = mpmath.beta(a2, b2)

    def integrand(x):
        lp = (a1 - 1) * mpmath.log(x) + (b1 - 1) * mpmath.log(1 - x) - mpmath.log(B1)
        lq = (a2 - 1) * mpmath.log(x) + (b2 - 1) * mpmath.log(1 - x) - mpmath.log(B2)
        return mpmath.exp(lp) * (lp - lq)

    val = mpmath.quad(integrand, [0, 0.5, 1])
    mpmath.mp.dps = 15
    return float(val)


def test_oracle_kl_matches_quadrature():
    rng = np.random.default_rng(7)
    pairs = rng.uniform(0.6, 6.0, size=(12, 4))
    for a1, b1, a2, b2 in pairs:
        q = _kl_quadrature(a1, b1, a2, b2)
        assert O.kl_beta(a1, b1, a2, b2) == pytest.approx(q, rel=1e-9, abs=1e-10)
        assert O.kl_beta(a1, b1, a2, b2) >= 0.0


def test_oracle_softplus():
    for x in [-1000.0, -50.0, -3.0, -1e-3, 0.0, 1e-3, 0.5, 3.0, 50.0, 1000.0]:
        assert O.softplus(x) == pytest.approx(float(np.logaddexp(0.0, x)), rel=1e-15, abs=1e-300)
    # the inverse used by the input generator: softplus(log(expm1(u))) = u
    for u in [6e-4, 0.01, 0.06, 1.0]:
        assert O.softplus(math.log(math.expm1(u))) == pytest.approx(u, rel=1e-13)
