"""Pins for the oracle's sampler (Sec. 3.3, eq. (2), certainty set, Poisson tail).

Every check here is fixed by something other than the oracle itself: published
Philox known-answer vectors, the budget identity that defines m, an exact
breakpoint solve written independently below, closed forms of eq. (2) in the
cases where nothing clips, and binomial statistics of the Bernoulli draws.
"""
import os

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _kat_rows():
    rows = []
    with open(os.path.join(GOLDEN, "philox4x32_10_kat.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            w = line.split()
            assert w[0] == "10"
            vals = [int(x, 16) for x in w[1:]]
            rows.append((vals[0:4], vals[4:6], vals[6:10]))
    return rows


@pytest.mark.parametrize("ctr,key,expect", _kat_rows())
def test_philox_known_answers(ctr, key, expect):
    got = oracle.philox4x32_10(ctr, key)
    assert [int(x) for x in got] == expect


def test_token_word_layout():
    # token i uses word (i mod 4) of the block at counter (i / 4, unit, epoch, tag)
    seed = 0x0123456789ABCDEF
    for i in [0, 1, 2, 3, 4, 7, 1023, 123457]:
        blk = oracle.philox4x32_10([i >> 2, 5, 9, 0x45424431], [seed & 0xFFFFFFFF, seed >> 32])
        assert oracle.token_word(seed, 5, 9, i) == int(blk[i & 3])


# ----------------------------------------------------------------------------
# lambda solve
# ----------------------------------------------------------------------------
def exact_lambda(s_tail, m, eps):
    """Independent breakpoint solve of sum clip(lam s, eps, 1) = m.

    g is piecewise linear in lam: a token moves from the floor to the linear
    part at lam = eps / s and from the linear part to 1 at lam = 1 / s.
    """
    s = s_tail[s_tail > 0].astype(np.float64)
    lam_e = np.concatenate([eps / s, 1.0 / s])
    dslope = np.concatenate([s, -s])
    dconst = np.concatenate([-eps * np.ones_like(s), np.ones_like(s)])
    order = np.argsort(lam_e, kind="stable")
    lam_e, dslope, dconst = lam_e[order], dslope[order], dconst[order]
    const0 = eps * len(s_tail)
    const_after = const0 + np.cumsum(dconst)
    slope_after = np.cumsum(dslope)
    const_before = np.concatenate([[const0], const_after[:-1]])
    slope_before = np.concatenate([[0.0], slope_after[:-1]])
    g_at = const_before + lam_e * slope_before
    k = int(np.argmax(g_at >= m))
    assert g_at[k] >= m and k > 0
    return (m - const_before[k]) / slope_before[k]


def _heavy_scores(n, seed):
    rng = np.random.default_rng(seed)
    s = rng.exponential(1.0, n)
    hh = rng.random(n) < 0.02
    s[hh] *= 60.0
    return s.astype(np.float32)


@pytest.mark.parametrize("n,f,eps,seed", [(4096, 0.10, 0.01, 0), (6144, 0.25, 0.01, 1),
                                          (2048, 0.05, 1e-6, 2), (1000, 0.5, 0.01, 3),
                                          (16384, 0.25, 0.01, 4)])
def test_budget_identity_and_exact_solve(n, f, eps, seed):
    s = _heavy_scores(n, seed)
    n_sink, n_recent = 4, 64
    pi, lam, st = oracle.inclusion_probs(s, n_sink, n_recent, f, eps)
    assert st == 0
    tail = np.ones(n, bool)
    tail[:n_sink] = False
    tail[n - n_recent:] = False
    m = f * n - (n - tail.sum())
    # expected tail size hits the budget (definition of m)
    assert abs(pi[tail].sum() - m) <= 1e-9 * m
    assert np.all(pi[~tail] == 1.0)
    # the clip at 1 actually binds on these scores (certainty layer is non-empty)
    assert (pi[tail] == 1.0).sum() > 0
    lam_x = exact_lambda(s[tail], m, eps)
    assert abs(lam - lam_x) <= 1e-12 * lam_x
    pi_x = np.clip(lam_x * s[tail].astype(np.float64), eps, 1.0)
    assert np.max(np.abs(pi[tail] - pi_x)) <= 1e-12


def test_no_clip_reduces_to_eq2_verbatim():
    # scores spread narrowly: m s / sum s stays inside (eps, 1), so lambda = m / sum_T s
    rng = np.random.default_rng(7)
    n = 3000
    s = (1.0 + 0.5 * rng.random(n)).astype(np.float32)
    pi, lam, st = oracle.inclusion_probs(s, 4, 32, 0.2, 1e-6)
    tail = slice(4, n - 32)
    m = 0.2 * n - 36
    ssum = s[tail].astype(np.float64).sum()
    assert abs(lam - m / ssum) <= 1e-13 * lam
    np.testing.assert_allclose(pi[tail], m * s[tail].astype(np.float64) / ssum, rtol=1e-13)
    pi1, lam1, _ = oracle.inclusion_probs(s, 4, 32, 0.2, 1e-6, pi_mode=1)
    assert abs(lam1 - m / ssum) <= 1e-15 * lam1


def test_uniform_scores():
    n = 512
    s = np.full(n, 3.25, np.float32)
    pi, lam, st = oracle.inclusion_probs(s, 1, 1, 0.25, 0.01)
    m = 0.25 * n - 2
    np.testing.assert_allclose(pi[1:-1], m / (n - 2), rtol=1e-13)


def test_literal_mode_spends_less_than_budget_when_clipping():
    s = _heavy_scores(4096, 11)
    pi0, _, _ = oracle.inclusion_probs(s, 4, 64, 0.1, 0.01, pi_mode=0)
    pi1, lam1, _ = oracle.inclusion_probs(s, 4, 64, 0.1, 0.01, pi_mode=1)
    m = 0.1 * 4096 - 68
    tail = slice(4, 4096 - 64)
    assert abs(lam1 - m / s[tail].astype(np.float64).sum()) <= 1e-13 * lam1
    np.testing.assert_allclose(pi1[tail], np.clip(lam1 * s[tail].astype(np.float64), 0.01, 1.0),
                               rtol=0, atol=1e-15)
    assert pi1[tail].sum() < m - 1.0
    assert abs(pi0[tail].sum() - m) < 1e-9 * m


def test_degenerate_budgets():
    n = 300
    s = _heavy_scores(n, 5)
    # floor binds: m <= eps |T|
    pi, lam, st = oracle.inclusion_probs(s, 4, 4, 0.03, 0.2)
    assert st & oracle.ST_BUDGET_FLOOR
    assert np.all(pi[4:-4] == 0.2) and np.all(pi[:4] == 1) and np.all(pi[-4:] == 1)
    # budget covers everything
    pi, lam, st = oracle.inclusion_probs(s, 4, 4, 1.0, 0.01)
    assert st & oracle.ST_NO_EVICTION
    assert np.all(pi == 1.0)
    # zero scores stay at the floor when the rest saturates
    s2 = s.copy()
    s2[10:20] = 0.0
    pi, lam, st = oracle.inclusion_probs(s2, 4, 4, 0.99, 0.01)
    assert st & oracle.ST_NO_EVICTION
    assert np.all(pi[10:20] == 0.01)
    assert np.all(pi[20:-4] == 1.0)
    # no tail at all
    pi, lam, st = oracle.inclusion_probs(s[:50], 30, 30, 0.1, 0.01)
    assert np.all(pi == 1.0)
    # empty unit
    pi, lam, st = oracle.inclusion_probs(np.zeros(0, np.float32), 4, 4, 0.1, 0.01)
    assert pi.shape == (0,)


def test_bad_scores_flagged_and_floored():
    s = _heavy_scores(1000, 6)
    s[100] = np.nan
    s[200] = np.inf
    s[300] = -5.0
    pi, lam, st = oracle.inclusion_probs(s, 4, 64, 0.2, 0.01)
    assert st & oracle.ST_BAD_SCORE
    assert pi[100] == pi[200] == pi[300] == 0.01
    tail = slice(4, 1000 - 64)
    assert abs(pi[tail].sum() - (0.2 * 1000 - 68)) < 1e-9 * 200


# ----------------------------------------------------------------------------
# Poisson mask: exact threshold, inclusion frequencies, budget in expectation
# ----------------------------------------------------------------------------
def test_mask_threshold_is_exact():
    seed, unit, epoch = 99, 3, 0
    n = 4096
    x = np.array([oracle.token_word(seed, unit, epoch, i) for i in range(n)], np.float64)
    pi_lo = (x.astype(np.float32).astype(np.float64) / 4294967296.0).astype(np.float32)
    m = oracle.mask(pi_lo, seed, unit, epoch)
    thr = pi_lo.astype(np.float64) * 4294967296.0
    np.testing.assert_array_equal(m.astype(bool), x < thr)
    ones = oracle.mask(np.ones(n, np.float32), seed, unit, epoch)
    assert ones.all()
    zeros = oracle.mask(np.zeros(n, np.float32), seed, unit, epoch)
    assert not zeros.any()


def test_inclusion_frequencies_match_pi():
    rng = np.random.default_rng(21)
    n = 256
    pi32 = rng.uniform(0.01, 0.99, n).astype(np.float32)
    R = 4000
    hits = np.zeros(n)
    for e in range(R):
        hits += oracle.mask(pi32, 1234, 7, e)
    p = pi32.astype(np.float64)
    z = (hits - R * p) / np.sqrt(R * p * (1 - p))
    assert np.max(np.abs(z)) < 5.0
    chi2 = float((z ** 2).sum())
    # chi-square with n dof: mean n, sd sqrt(2n)
    assert abs(chi2 - n) < 6 * np.sqrt(2 * n)


def test_budget_hit_in_expectation():
    s = _heavy_scores(4096, 31)
    f = 0.1
    pi, _, _ = oracle.inclusion_probs(s, 4, 64, f, 0.01)
    p32 = pi.astype(np.float32)
    R = 400
    sizes = np.array([oracle.mask(p32, 5, u, 0).sum() for u in range(R)], np.float64)
    var = (p32 * (1 - p32.astype(np.float64))).sum()
    assert abs(sizes.mean() - f * 4096) < 5 * np.sqrt(var / R)


# ----------------------------------------------------------------------------
# Compaction
# ----------------------------------------------------------------------------
def test_compaction_definition():
    rng = np.random.default_rng(3)
    n, d = 777, 16
    K = rng.integers(0, 1 << 16, (n, d), dtype=np.uint16)
    V = rng.integers(0, 1 << 16, (n, d), dtype=np.uint16)
    pi32 = rng.uniform(0.05, 1.0, n).astype(np.float32)
    msk = oracle.mask(pi32, 8, 1, 0)
    Kc, Vc, pic, idx, cnt = oracle.compact(msk, pi32, K, V)
    keep = np.nonzero(msk)[0]
    assert cnt == msk.sum() == len(keep)
    np.testing.assert_array_equal(idx, keep)
    assert np.all(np.diff(idx) > 0)
    np.testing.assert_array_equal(Kc, K[keep])
    np.testing.assert_array_equal(Vc, V[keep])
    np.testing.assert_array_equal(pic, pi32[keep])
    # capacity overflow: true count returned, only the first cap rows written
    cap = cnt // 2
    Kc2, Vc2, pic2, idx2, cnt2 = oracle.compact(msk, pi32, K, V, cap=cap)
    assert cnt2 == cnt and len(idx2) == cap
    np.testing.assert_array_equal(idx2, keep[:cap])


def test_evict_batch_ragged_units():
    rng = np.random.default_rng(4)
    lens = [0, 1, 70, 300, 1000, 2049]
    d = 8
    off = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    rows = int(off[-1])
    K = rng.integers(0, 1 << 16, (rows, d), dtype=np.uint16)
    V = rng.integers(0, 1 << 16, (rows, d), dtype=np.uint16)
    s = _heavy_scores(rows, 9)
    caps = [n for n in lens]
    coff = np.concatenate([[0], np.cumsum(caps)]).astype(np.int64)
    out = oracle.evict_batch(off, coff, s, K, V, 4, 16, budget_frac=0.2, pi_min=0.01, seed=77)
    for u, n in enumerate(lens):
        pi, lam, st = oracle.inclusion_probs(s[off[u]:off[u + 1]], 4, 16, 0.2, 0.01)
        p32 = pi.astype(np.float32)
        np.testing.assert_array_equal(out["pi_full"][off[u]:off[u + 1]], p32)
        msk = oracle.mask(p32, 77, u, 0)
        assert out["count"][u] == msk.sum()
        keep = np.nonzero(msk)[0]
        c0 = coff[u]
        np.testing.assert_array_equal(out["idx"][c0:c0 + len(keep)], keep)
        np.testing.assert_array_equal(out["Kc"][c0:c0 + len(keep)], K[off[u] + keep])


def test_evict_batch_unit_ids_select_the_stream():
    """A sample of units evicted on its own, with the units' ids in the larger batch as the Philox
    unit word, retains exactly what the whole batch retains for those units."""
    rng = np.random.default_rng(5)
    lens = [500] * 9
    d = 8
    off = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    K = rng.integers(0, 1 << 16, (int(off[-1]), d), dtype=np.uint16)
    V = rng.integers(0, 1 << 16, (int(off[-1]), d), dtype=np.uint16)
    s = _heavy_scores(int(off[-1]), 3)
    full = oracle.evict_batch(off, off, s, K, V, 4, 16, budget_frac=0.3, seed=5)
    pick = np.array([7, 2, 5], np.int64)
    rows = np.concatenate([np.arange(off[u], off[u + 1]) for u in pick])
    soff = np.arange(len(pick) + 1, dtype=np.int64) * 500
    sub = oracle.evict_batch(soff, soff, s[rows], K[rows], V[rows], 4, 16, budget_frac=0.3, seed=5,
                             unit_ids=pick.astype(np.uint32))
    plain = oracle.evict_batch(soff, soff, s[rows], K[rows], V[rows], 4, 16, budget_frac=0.3, seed=5)
    for i, u in enumerate(pick):
        c = full["count"][u]
        assert sub["count"][i] == c
        np.testing.assert_array_equal(sub["idx"][soff[i]:soff[i] + c], full["idx"][off[u]:off[u] + c])
    assert not np.array_equal(plain["count"], sub["count"]) or not np.array_equal(
        plain["idx"], sub["idx"])  # local ids draw other streams
