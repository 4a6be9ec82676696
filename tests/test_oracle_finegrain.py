"""Pins for the oracle's fine-grained attribution and deployed certificate (Sec. 6 "Finer
grains"; App. "Experimental details": per-retained-token variance contributions pooled into
64-token blocks of original positions, and the certificate averaged over every fourth head and
maximized over the first decode steps).

  * the block contributions of a unit sum to the sum over its heads of Vhat (Theorem 2), since
    each token's contribution is one summand of Vhat;
  * certainty tokens (pi = 1) contribute nothing; a block without retained tail tokens is 0;
  * with one retained tail token per block, each block holds that token's own Vhat (a
    one-token tail makes Vhat equal to its single summand);
  * the certificate step is a mean over the sampled pairs per sequence and a running maximum.
"""
import numpy as np

import oracle
from helpers import rand_bf16


def _unit(seed, n=400, G=3, d=128):
    rng = np.random.default_rng(seed)
    q = rand_bf16(rng, (G, d))
    K = rand_bf16(rng, (n, d), scale=1.5)
    V = rand_bf16(rng, (n, d))
    pi = rng.uniform(0.02, 1.0, n).astype(np.float32)
    pi[rng.random(n) < 0.2] = 1.0
    idx = np.sort(rng.choice(4 * n, n, replace=False)).astype(np.int32)
    return q, K, V, pi, idx


def test_blocks_sum_to_vhat():
    q, K, V, pi, idx = _unit(1)
    out = oracle.attend_certify(q, K, V, pi)
    nb = int(idx.max()) // 64 + 1
    blocks = oracle.block_contributions(q, K, V, pi, idx, out["y"], out["lse"], nb)
    assert blocks.shape == (nb,)
    np.testing.assert_allclose(blocks.sum(), out["vhat"].sum(), rtol=1e-10)
    assert np.all(blocks >= 0)


def test_certainty_tokens_and_empty_blocks_contribute_nothing():
    q, K, V, pi, idx = _unit(2)
    out = oracle.attend_certify(q, K, V, np.ones_like(pi))
    nb = int(idx.max()) // 64 + 1
    assert np.all(oracle.block_contributions(q, K, V, np.ones_like(pi), idx, out["y"], out["lse"], nb) == 0)
    out = oracle.attend_certify(q, K, V, pi)
    blocks = oracle.block_contributions(q, K, V, pi, idx, out["y"], out["lse"], nb)
    occupied = np.zeros(nb, bool)
    occupied[idx[pi < 1] // 64] = True
    assert np.all(blocks[~occupied] == 0) and np.all(blocks[occupied] > 0)
    # positions past the last block and appended rows (idx -1) are ignored
    idx2 = idx.copy()
    idx2[:5] = -1
    short = oracle.block_contributions(q, K, V, pi, idx2, out["y"], out["lse"], 3)
    full = oracle.block_contributions(q, K, V, pi, idx2, out["y"], out["lse"], nb)
    np.testing.assert_array_equal(short, full[:3])


def test_one_tail_token_per_block_is_its_own_vhat():
    rng = np.random.default_rng(3)
    G, d, n = 2, 128, 12
    q = rand_bf16(rng, (G, d))
    K = rand_bf16(rng, (n, d))
    V = rand_bf16(rng, (n, d))
    pi = np.ones(n, np.float32)
    idx = (np.arange(n) * 64 + 5).astype(np.int32)  # token j alone in block j
    tail = [2, 7, 9]
    pi[tail] = [0.3, 0.05, 0.6]
    out = oracle.attend_certify(q, K, V, pi)
    blocks = oracle.block_contributions(q, K, V, pi, idx, out["y"], out["lse"], n)
    # Vhat of the whole set restricted to token j: the same summand (yhat, Nhat fixed)
    for j in range(n):
        if j not in tail:
            assert blocks[j] == 0.0
    np.testing.assert_allclose(blocks[tail].sum(), out["vhat"].sum(), rtol=1e-10)
    # a set whose only tail token is j: Vhat there is exactly that token's summand
    for j in tail:
        keep = [i for i in range(n) if pi[i] == 1.0] + [j]
        keep.sort()
        sub = oracle.attend_certify(q, K[keep], V[keep], pi[keep])
        b1 = oracle.block_contributions(q, K[keep], V[keep], pi[keep], idx[keep], sub["y"], sub["lse"], n)
        np.testing.assert_allclose(b1[j], sub["vhat"].sum(), rtol=1e-10)


def test_certificate_step_mean_and_running_max():
    r = np.array([[0.1, 0.2, 0.3, 0.4],
                  [1.0, 2.0, 3.0, 4.0],
                  [5.0, 6.0, 7.0, 8.0]], np.float32)
    unit_seq = np.array([0, 0, 1], np.int32)
    head0 = np.array([0, 4, 2], np.int32)  # query head index of each unit's first head
    # stride 2: unit 0 heads 0, 2; unit 1 heads 4, 6; unit 2 heads 2 + {0, 2} = 2, 4
    cert, mean = oracle.certificate_step(r, unit_seq, 3, head_stride=2, unit_head0=head0)
    np.testing.assert_allclose(mean, [(0.1 + 0.3 + 1.0 + 3.0) / 4, (5.0 + 7.0) / 2, 0.0], rtol=1e-7)
    np.testing.assert_allclose(cert, [mean[0], mean[1], 0.0])
    cert2, _ = oracle.certificate_step(r * 0.5, unit_seq, 3, head_stride=2, unit_head0=head0, cert=cert)
    np.testing.assert_array_equal(cert2, cert)  # a smaller step leaves the maximum
    cert3, _ = oracle.certificate_step(r * 2, unit_seq, 3, head_stride=2, unit_head0=head0, cert=cert)
    np.testing.assert_allclose(cert3[:2], 2 * np.asarray(mean[:2]), rtol=1e-7)
    _, m4 = oracle.certificate_step(r, unit_seq, 3, head_stride=4)  # heads 0 only (head0 = 0)
    np.testing.assert_allclose(m4[:2], [(0.1 + 1.0) / 2, 5.0], rtol=1e-7)
