"""Pins for the oracle's importance scores (App. "Experimental details", Harness: the attention
mass each key receives from a set of prefill or observation-window queries).

  * every query that sees at least one key spreads exactly mass 1 (softmax rows sum to 1);
  * constant keys: each query spreads its mass uniformly over the keys it sees (closed form);
  * one query over all keys equals torch.softmax in fp64 (a library routine);
  * a causal query at position p gives nothing to keys after p; at position 0 all to key 0;
  * queries enter as an unordered set; q scaled by c with the logit scale divided by c is the
    same score; the batched driver equals the per-unit one.
"""
import numpy as np
import pytest
import torch

import oracle
from helpers import bf16_to_f64, rand_bf16, to_bf16_bits


@pytest.mark.parametrize("n,W,causal", [(1, 1, False), (300, 32, False), (513, 64, True), (97, 5, True)])
def test_mass_per_query_is_one(n, W, causal):
    rng = np.random.default_rng(n + W)
    K = rand_bf16(rng, (n, 128), scale=2.0)
    Q = rand_bf16(rng, (W, 128))
    qpos = rng.integers(-2, n + 3, size=W).astype(np.int32) if causal else None
    s = oracle.window_scores(K, Q, qpos)
    seeing = W if qpos is None else int(np.sum(qpos >= 0))
    assert abs(s.sum() - seeing) <= 1e-12 * max(1, seeing)
    assert np.all(s >= 0.0)


def test_constant_keys_closed_form():
    n, W = 40, 6
    rng = np.random.default_rng(3)
    K = to_bf16_bits(np.full((n, 128), 0.25))
    Q = rand_bf16(rng, (W, 128))
    qpos = np.array([0, 3, 3, 17, 39, 100], np.int32)
    s = oracle.window_scores(K, Q, qpos)
    ref = np.zeros(n)
    for p in qpos:
        seen = min(int(p) + 1, n)
        ref[:seen] += 1.0 / seen
    np.testing.assert_allclose(s, ref, rtol=1e-13, atol=1e-15)
    s_all = oracle.window_scores(K, Q)
    np.testing.assert_allclose(s_all, np.full(n, W / n), rtol=1e-13)


@pytest.mark.parametrize("n", [1, 64, 1000])
def test_single_query_is_torch_softmax(n):
    rng = np.random.default_rng(n)
    K = rand_bf16(rng, (n, 128), scale=3.0)
    q = rand_bf16(rng, (1, 128))
    logits = torch.tensor(bf16_to_f64(K)) @ torch.tensor(bf16_to_f64(q[0])) / np.sqrt(128.0)
    ref = torch.softmax(logits, dim=0).numpy()
    np.testing.assert_allclose(oracle.window_scores(K, q), ref, rtol=1e-12, atol=1e-300)


def test_causal_masks_later_keys():
    n = 50
    rng = np.random.default_rng(5)
    K = rand_bf16(rng, (n, 128))
    Q = rand_bf16(rng, (3, 128))
    s = oracle.window_scores(K, Q, np.array([0, 10, 20], np.int32))
    assert np.all(s[21:] == 0.0)
    only0 = oracle.window_scores(K, Q[:1], np.array([0], np.int32))
    assert only0[0] == 1.0 and np.all(only0[1:] == 0.0)
    none = oracle.window_scores(K, Q, np.array([-1, -5, -1], np.int32))
    assert np.all(none == 0.0)


def test_query_order_and_scale_invariance():
    n, W = 200, 8
    rng = np.random.default_rng(9)
    K = rand_bf16(rng, (n, 128))
    Q = rand_bf16(rng, (W, 128))
    qpos = rng.integers(0, n, size=W).astype(np.int32)
    s = oracle.window_scores(K, Q, qpos)
    perm = rng.permutation(W)
    np.testing.assert_allclose(oracle.window_scores(K, Q[perm], qpos[perm]), s, rtol=1e-12)
    Q2 = to_bf16_bits(bf16_to_f64(Q) * 2.0)  # exact in bf16
    np.testing.assert_allclose(oracle.window_scores(K, Q2, qpos, scale=0.5 / np.sqrt(128)), s,
                               rtol=1e-12)


def test_batch_equals_per_unit():
    rng = np.random.default_rng(11)
    lengths = [0, 1, 70, 300]
    off = np.concatenate([[0], np.cumsum(lengths)]).astype(np.int64)
    K = rand_bf16(rng, (int(off[-1]), 128))
    W = 4
    Q = rand_bf16(rng, (len(lengths), W, 128))
    qpos = rng.integers(-1, 310, size=(len(lengths), W)).astype(np.int32)
    out = oracle.window_scores_batch(off, K, Q, qpos)
    for u in range(len(lengths)):
        ref = oracle.window_scores(K[off[u]:off[u + 1]], Q[u], qpos[u])
        np.testing.assert_array_equal(out[off[u]:off[u + 1]], ref)
