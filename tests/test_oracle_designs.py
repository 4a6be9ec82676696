"""Pins for the oracle's other sampling designs (App. "Experimental details": fixed-size
systematic sampling at the same inclusion probabilities; the deterministic top-k and uniform
comparison arms).

Systematic design (Hajek 1964): integer weights a_i = ceil(pi_i 2^32), cumulative C_i, one start
u per unit; position i is kept iff a point u + k 2^32 lies in [C_{i-1}, C_i).
  * exact inclusion probabilities: over a grid of starts, each position is kept for exactly
    a_i / (grid spacing) of them;
  * the size is fixed: floor or ceil of sum a / 2^32, never random beyond that;
  * two adjacent positions with pi_i + pi_j <= 1 are never kept together;
  * the start is Philox4x32-10 word 0 at counter (0, unit, epoch, "EBDS").
Top-k: exactly the k = floor(m + 1/2) largest scores of the tail (ties to the lower position),
plus the protected positions, all with pi = 1.
Uniform: every tail position gets the same pi = clip(m / |T|, eps, 1).
"""
import numpy as np

import oracle


def _sys_mask_for_start(pi32, u):
    """Restatement of the systematic rule for a given start u (brute force over points)."""
    a = np.ceil(pi32.astype(np.float64) * 2.0 ** 32).astype(np.uint64)
    C = np.concatenate([[0], np.cumsum(a, dtype=np.uint64)])
    keep = np.zeros(len(pi32), np.uint8)
    total = int(C[-1])
    p = u
    while p < total:  # every point u + k 2^32 below the total lands in exactly one interval
        i = int(np.searchsorted(C, p, side="right")) - 1
        keep[i] += 1
        p += 1 << 32
    return keep


def test_systematic_start_is_philox_word():
    for seed, unit, epoch in ((0, 0, 0), (12345678901, 17, 3), (2 ** 64 - 1, 2 ** 32 - 1, 9)):
        w = oracle.philox4x32_10([0, unit, epoch, 0x45424453], [seed & 0xFFFFFFFF, seed >> 32])
        assert oracle.systematic_start(seed, unit, epoch) == int(w[0])


def test_systematic_matches_brute_force_points():
    rng = np.random.default_rng(1)
    for trial in range(20):
        n = int(rng.integers(1, 60))
        pi = rng.uniform(0.0, 1.0, n).astype(np.float32)
        pi[rng.random(n) < 0.2] = 1.0
        seed, unit = int(rng.integers(0, 2 ** 63)), trial
        u = oracle.systematic_start(seed, unit, 0)
        np.testing.assert_array_equal(oracle.mask_systematic(pi, seed, unit), _sys_mask_for_start(pi, u))


def test_systematic_exact_inclusion_probabilities_over_starts():
    """pi_i = j_i / 2^16: over the 2^16 starts u = k 2^16 each position is kept exactly j_i
    times (its inclusion probability, exactly)."""
    rng = np.random.default_rng(2)
    n = 12
    j = rng.integers(0, 1 << 16, n)
    j[3] = 1 << 16  # pi = 1
    pi = (j / 65536.0).astype(np.float32)
    counts = np.zeros(n, np.int64)
    for k in range(1 << 16):
        counts += _sys_mask_for_start(pi, k << 16)
    np.testing.assert_array_equal(counts, j)


def test_systematic_fixed_size_and_no_adjacent_pairs():
    rng = np.random.default_rng(3)
    n = 5000
    pi = np.clip(rng.pareto(1.5, n) * 0.05, 0.01, 1.0).astype(np.float32)
    a = np.ceil(pi.astype(np.float64) * 2.0 ** 32)
    expected = a.sum() / 2.0 ** 32
    sizes = set()
    for epoch in range(50):
        m = oracle.mask_systematic(pi, 7, 1, epoch)
        sizes.add(int(m.sum()))
        small = (pi[:-1].astype(np.float64) + pi[1:]) <= 1.0
        assert not np.any(small & (m[:-1] == 1) & (m[1:] == 1))
        assert np.all(m[pi == 1.0] == 1)
    assert sizes <= {int(np.floor(expected)), int(np.ceil(expected))}


def test_systematic_inclusion_frequency_matches_pi():
    """Over independent starts, the empirical inclusion frequency of each position matches its
    pi (z-scores within 5)."""
    rng = np.random.default_rng(4)
    n, R = 40, 4000
    pi = rng.uniform(0.02, 1.0, n).astype(np.float32)
    hits = np.zeros(n)
    for epoch in range(R):
        hits += oracle.mask_systematic(pi, 11, 0, epoch)
    p = pi.astype(np.float64)
    z = (hits - R * p) / np.sqrt(R * p * (1 - p) + 1e-12)
    assert np.all(np.abs(z[p < 1]) < 5)


def test_topk_is_the_k_largest_with_index_ties():
    rng = np.random.default_rng(5)
    n = 300
    s = rng.integers(0, 40, n).astype(np.float32)  # many ties
    s[10] = np.nan
    for f in (0.1, 0.33, 0.5, 0.99):
        pi, st = oracle.topk_probs(s, 4, 16, f)
        tail = np.arange(4, n - 16)
        m = f * n - 20
        k = min(max(int(np.floor(m + 0.5)), 0), len(tail))
        clean = np.where(np.isfinite(s) & (s >= 0), s, 0.0)[tail]
        order = tail[np.lexsort((tail, -clean))]
        want = np.zeros(n)
        want[:4] = want[n - 16:] = 1.0
        want[order[:k]] = 1.0
        np.testing.assert_array_equal(pi, want)
        assert st & oracle.ST_BAD_SCORE


def test_topk_and_uniform_through_the_batch_driver():
    rng = np.random.default_rng(6)
    lengths = [500, 64, 1000]
    off = np.concatenate([[0], np.cumsum(lengths)]).astype(np.int64)
    coff = off.copy()
    s = rng.pareto(1.5, off[-1]).astype(np.float32)
    K = rng.integers(0, 1 << 16, (off[-1], 8), dtype=np.uint16)
    V = rng.integers(0, 1 << 16, (off[-1], 8), dtype=np.uint16)
    top = oracle.evict_batch(off, coff, s, K, V, 4, 16, budget_frac=0.2, design=oracle.DESIGN_TOPK)
    for u, n in enumerate(lengths):
        pi, _ = oracle.topk_probs(s[off[u]:off[u + 1]], 4, 16, 0.2)
        assert top["count"][u] == int(pi.sum())
        np.testing.assert_array_equal(top["idx"][coff[u]:coff[u] + top["count"][u]], np.flatnonzero(pi))
    uni = oracle.evict_batch(off, coff, s, K, V, 4, 16, budget_frac=0.2, pi_min=0.01,
                             design=oracle.DESIGN_UNIFORM)
    for u, n in enumerate(lengths):
        p = uni["pi_full"][off[u]:off[u + 1]]
        tail = p[4:n - 16]
        m = 0.2 * n - 20
        want = np.float32(min(max(m / (n - 20), 0.01), 1.0))
        assert np.all(p[:4] == 1) and np.all(p[n - 16:] == 1)
        assert np.all(np.abs(tail - want) <= 1e-6)
    sy = oracle.evict_batch(off, coff, s, K, V, 4, 16, budget_frac=0.2, pi_min=0.01,
                            design=oracle.DESIGN_SYSTEMATIC, seed=3)
    po = oracle.evict_batch(off, coff, s, K, V, 4, 16, budget_frac=0.2, pi_min=0.01, seed=3)
    np.testing.assert_array_equal(sy["pi_full"], po["pi_full"])  # same pi, other design
    for u, n in enumerate(lengths):
        m = oracle.mask_systematic(po["pi_full"][off[u]:off[u + 1]], 3, u)
        assert sy["count"][u] == int(m.sum())
