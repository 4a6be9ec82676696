"""Design-based pins for the oracle's estimator and certificate (Theorem 2, App. A.1, eq. (4)).

An independent enumerator (numpy, below) lists all 2^|T| retained subsets of a
tiny cache with their Poisson-design probabilities.  It fixes:

  * the closed form Var(e_lin) = sum_T (1 - pi)/pi |x_i|^2 of App. A.1 (checked
    against the enumerated second moment of e_lin itself), and the exact
    unbiasedness of the Horvitz-Thompson sum with the true x_i;
  * Theorem 2: E[Vhat] = Var(e_lin) + O(B^2/m^2).  The tail's attention mass is
    shrunk by a factor t through an extra key coordinate; the remainder is then
    O(t) relative, so E[Vhat]/Var(e_lin) -> 1 sharply, and the gap shrinks as
    t does (the linearisation remainder);
  * Monte Carlo over Philox draws: mean Hajek output and mean Vhat agree with
    their enumerated expectations within 5 standard errors;
  * eq. (4): in a one-dimensional Gaussian regime the radius covers the
    realised error at least as often as its variance term alone would under
    normal errors, P(|Z| <= sqrt(2 ln(1/delta))).
"""
import itertools

import numpy as np
import pytest
from scipy.stats import norm

import oracle
from helpers import bf16_to_f64, to_bf16_bits


def tiny_cache(seed, nP=4, nT=12, d=4, shift=-18.375, loc=2.0):
    """Certainty rows 0..nP-1, tail rows after.  The last key coordinate of tail
    rows is `shift` and q's last coordinate is 1, so tail weights carry a factor
    exp(shift / sqrt(d)) (= t)."""
    rng = np.random.default_rng(seed)
    n = nP + nT
    q = rng.standard_normal(d)
    q[-1] = 1.0
    K = rng.standard_normal((n, d))
    K[:, -1] = 0.0
    K[nP:, -1] = shift
    V = loc + rng.standard_normal((n, d))
    pi = np.ones(n, np.float32)
    pi[nP:] = rng.uniform(0.1, 0.9, nT)
    return to_bf16_bits(q)[None], to_bf16_bits(K), to_bf16_bits(V), pi


def enumerate_design(q, K, V, pi, nP):
    """All retained subsets of the tail with their probabilities (Poisson design)."""
    d = K.shape[1]
    n = K.shape[0]
    qf = bf16_to_f64(q)[0]
    Kf = bf16_to_f64(K)
    Vf = bf16_to_f64(V)
    p = pi.astype(np.float64)
    s = Kf @ qf / np.sqrt(d)
    a = np.exp(s - s.max())
    N = a.sum()
    y = (a[:, None] * Vf).sum(0) / N  # eq. (1)
    x = a[:, None] * (Vf - y) / N  # App. A.1: x_i = a_i (v_i - y) / N
    T = np.arange(nP, n)
    var_lin = ((1 - p[T]) / p[T] * (x[T] ** 2).sum(1)).sum()
    cells = []
    for bits in itertools.product([0, 1], repeat=len(T)):
        I = np.array(bits)
        prob = float(np.prod(np.where(I == 1, p[T], 1 - p[T])))
        keep = np.concatenate([np.arange(nP), T[I == 1]])
        e_lin = ((I / p[T] - 1)[:, None] * x[T]).sum(0)
        ht = (((1 - p[T]) / p[T] ** 2 * (x[T] ** 2).sum(1)) * I).sum()
        xb = np.max(np.sqrt(1 - p[T]) / p[T] * np.linalg.norm(x[T], axis=1) * I) if I.any() else 0.0
        cells.append(dict(prob=prob, keep=keep, e_lin=e_lin, ht=ht, xb=xb, ntail=int(I.sum())))
    return dict(y=y, x=x, var_lin=var_lin, cells=cells)


def test_closed_form_linearised_variance_and_ht_unbiasedness():
    q, K, V, pi = tiny_cache(0, shift=0.0)
    E = enumerate_design(q, K, V, pi, 4)
    tot = sum(c["prob"] for c in E["cells"])
    assert abs(tot - 1.0) < 1e-12
    e2 = sum(c["prob"] * (c["e_lin"] ** 2).sum() for c in E["cells"])
    mean_e = sum(c["prob"] * c["e_lin"] for c in E["cells"])
    assert np.linalg.norm(mean_e) < 1e-12 * np.sqrt(E["var_lin"])
    assert abs(e2 - E["var_lin"]) < 1e-12 * E["var_lin"]
    eht = sum(c["prob"] * c["ht"] for c in E["cells"])
    assert abs(eht - E["var_lin"]) < 1e-12 * E["var_lin"]


def _oracle_moments(q, K, V, pi, E):
    Ev = 0.0
    Ev2 = 0.0
    Ey = 0.0
    Ey2 = 0.0
    mse = 0.0
    per = []
    for c in E["cells"]:
        k = c["keep"]
        o = oracle.attend_certify(q, K[k], V[k], pi[k])
        v = o["vhat"][0]
        yh = o["y"][0]
        Ev += c["prob"] * v
        Ev2 += c["prob"] * v * v
        Ey = Ey + c["prob"] * yh
        Ey2 = Ey2 + c["prob"] * yh * yh
        mse += c["prob"] * ((yh - E["y"]) ** 2).sum()
        per.append((c, v, o["b"][0], yh))
    return dict(Ev=Ev, Ev2=Ev2, Ey=Ey, Ey2=Ey2, mse=mse, per=per)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_vhat_unbiased_in_linear_limit(seed):
    q, K, V, pi = tiny_cache(seed, shift=-18.375)  # t ~ 1e-4
    E = enumerate_design(q, K, V, pi, 4)
    M = _oracle_moments(q, K, V, pi, E)
    vl = E["var_lin"]
    assert abs(M["Ev"] / vl - 1) < 3e-3
    assert abs(M["mse"] / vl - 1) < 3e-3
    # Hajek bias is second order: far below the error's standard deviation
    assert np.linalg.norm(M["Ey"] - E["y"]) < 3e-3 * np.sqrt(vl)
    for c, v, b, yh in M["per"]:
        if c["ntail"] == 0:
            assert v == 0 and b == 0
            continue
        # per draw, Vhat is the HT sum with x_i estimated; b is the max term
        assert abs(v / c["ht"] - 1) < 1e-2
        assert abs(b / c["xb"] - 1) < 1e-2


def test_linearisation_gap_shrinks_with_tail_mass():
    gaps = []
    for shift in (0.0, -6.0, -12.0, -18.375):
        q, K, V, pi = tiny_cache(5, shift=shift)
        E = enumerate_design(q, K, V, pi, 4)
        M = _oracle_moments(q, K, V, pi, E)
        gaps.append(abs(M["Ev"] / E["var_lin"] - 1))
    assert all(g1 > g2 for g1, g2 in zip(gaps, gaps[1:])), gaps
    assert gaps[-1] < 3e-3


def _replicate(q, K, V, pi, R, seed, delta=0.1):
    """R independent Poisson draws of one cache, through the batched oracle."""
    n, d = K.shape
    off = np.arange(R + 1, dtype=np.int64) * n
    ev = oracle.evict_batch(off, off, np.zeros(n * R, np.float32), np.tile(K, (R, 1)),
                            np.tile(V, (R, 1)), 0, 0, pi_given=np.tile(pi, R), seed=seed)
    at = oracle.attend_batch(off, ev["count"], np.tile(q, (R, 1)).reshape(R, 1, d), ev["Kc"],
                             ev["Vc"], ev["pic"], delta=delta)
    return ev, at


@pytest.mark.parametrize("R", [20000, pytest.param(100000, marks=pytest.mark.slow)])
def test_monte_carlo_matches_enumeration(R):
    q, K, V, pi = tiny_cache(3, shift=-2.0)
    E = enumerate_design(q, K, V, pi, 4)
    M = _oracle_moments(q, K, V, pi, E)
    ev, at = _replicate(q, K, V, pi, R, seed=4242 + R)
    # the draws are the Poisson design: mean retained tail size
    np.testing.assert_allclose(ev["count"].mean() - 4, pi[4:].astype(np.float64).sum(),
                               atol=5 * np.sqrt((pi[4:] * (1 - pi[4:].astype(np.float64))).sum() / R))
    sd_y = np.sqrt(np.maximum(M["Ey2"] - M["Ey"] ** 2, 1e-300) / R)
    z_y = (at["y"][:, 0, :].mean(0) - M["Ey"]) / sd_y
    assert np.max(np.abs(z_y)) < 5, z_y
    sd_v = np.sqrt((M["Ev2"] - M["Ev"] ** 2) / R)
    z_v = (at["vhat"][:, 0].mean() - M["Ev"]) / sd_v
    assert abs(z_v) < 5, z_v


def _gauss_cache(seed, nP=8, nT=4000, p=0.5):
    """One effective value dimension, many comparable tail terms (CLT regime)."""
    rng = np.random.default_rng(seed)
    n = nP + nT
    q = np.array([0.25, 1.0])
    K = np.zeros((n, 2))
    K[:, 0] = rng.standard_normal(n)
    K[nP:, 1] = -2.0
    V = np.zeros((n, 2))
    V[:, 0] = 1.0 + rng.standard_normal(n)
    pi = np.ones(n, np.float32)
    pi[nP:] = p
    return to_bf16_bits(q)[None], to_bf16_bits(K), to_bf16_bits(V), pi


@pytest.mark.parametrize("delta", [0.1, 0.3])
def test_radius_coverage_gaussian_regime(delta):
    q, K, V, pi = _gauss_cache(0)
    R = 4000
    ev, at = _replicate(q, K, V, pi, R, seed=99, delta=delta)
    y = oracle.full_attention(q, K, V)[0]
    err = np.linalg.norm(at["y"][:, 0, :] - y, axis=1)
    r_abs = at["r"][:, 0] * (np.linalg.norm(at["y"][:, 0, :], axis=1) + 1e-9)
    cov = (err <= r_abs).mean()
    floor = 2 * norm.cdf(np.sqrt(2 * np.log(1 / delta))) - 1
    se = np.sqrt(floor * (1 - floor) / R)
    assert cov >= floor - 4 * se, (cov, floor)
    assert cov >= 1 - delta
    # Vhat tracks the realised mean squared error in this regime
    assert abs(at["vhat"].mean() / (err ** 2).mean() - 1) < 0.05
