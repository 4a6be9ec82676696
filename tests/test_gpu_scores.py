"""GPU parity of the importance scores (ebd_scores, through the C ABI) against the fp64 oracle.

Bar: every score within 2e-4 relative of the oracle's (plus 1e-9 absolute for scores that
underflow); the scores of a unit sum to its number of seeing queries within 1e-4 relative.
"""
import sys

import numpy as np
import pytest
import torch

import oracle
import synth

pytestmark = pytest.mark.gpu

RTOL, ATOL = 2e-4, 1e-9


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    import paper_2607_21475_amd  # noqa: F401  (fails loudly if libebd.so is missing)
    yield


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _np(t):
    return t.detach().cpu().numpy()


def _run(lengths, W, seed, qpos=None, split_rows=0, accumulate_onto=None):
    from paper_2607_21475_amd import cache

    K, _, seq_off = synth.make_cache(lengths, seed=seed, device="cuda")
    q = synth.make_queries(len(lengths), W, seed=seed + 1, device="cuda")
    qp = None if qpos is None else torch.as_tensor(qpos, dtype=torch.int32, device="cuda")
    out = None
    if accumulate_onto is not None:
        out = torch.as_tensor(accumulate_onto, dtype=torch.float32, device="cuda").clone()
    s, _ = cache.importance_scores(K, seq_off, q, max(lengths), qpos=qp, scores=out,
                                   accumulate=accumulate_onto is not None, split_rows=split_rows)
    torch.cuda.synchronize()
    return K, q, seq_off, s


def _check(K, q, seq_off, s, qpos=None, base=None):
    off = _np(seq_off)
    ref = oracle.window_scores_batch(off, synth.bf16_bits(K), synth.bf16_bits(q),
                                     None if qpos is None else np.asarray(qpos, np.int32))
    if base is not None:
        ref = ref + base
    got = _np(s)[: off[-1]].astype(np.float64)
    bad = np.abs(got - ref) > RTOL * np.abs(ref) + ATOL
    assert not bad.any(), (np.argwhere(bad)[:5].ravel(), got[bad][:5], ref[bad][:5])
    return ref


@pytest.mark.parametrize("lengths,W,split", [
    ([4096] * 8, 32, 0),                       # observation window of 32 queries
    ([0, 1, 5, 70, 777, 2048, 6144, 16384], 7, 0),   # ragged units, one query block
    ([3000, 1000], 64, 0),                     # four query blocks
    ([5000, 333], 33, 48),                     # partial block; many splits per unit
    ([20000], 16, 0),                          # one long unit
])
def test_scores_window(lengths, W, split):
    _say("scores window lengths=%s W=%d split=%d" % (lengths[:6], W, split))
    K, q, seq_off, s = _run(lengths, W, seed=3, split_rows=split)
    ref = _check(K, q, seq_off, s)
    off = _np(seq_off)
    for u, n in enumerate(lengths):  # each query spreads mass 1 over the rows it sees
        tot = float(_np(s)[off[u]:off[u + 1]].sum())
        assert abs(tot - (W if n > 0 else 0)) <= 1e-4 * W, (u, tot)
    assert np.all(ref >= 0)


def test_scores_causal_prefill_queries():
    """Prefill queries see the rows up to their position (negative: none; past the end: all)."""
    lengths = [2048, 600, 1]
    W = 20
    rng = np.random.default_rng(4)
    qpos = np.stack([rng.integers(-3, n + 5, size=W) for n in lengths]).astype(np.int32)
    qpos[0, :4] = [0, 2047, 5000, -1]
    _say("scores causal")
    K, q, seq_off, s = _run(lengths, W, seed=5, qpos=qpos, split_rows=256)
    _check(K, q, seq_off, s, qpos=qpos)


@pytest.mark.parametrize("extra", [32, 16, 40, 64])
def test_scores_accumulate_over_calls(extra):
    """More than 64 queries: a second call (1 to 4 blocks of 16 queries) adds its queries' mass to
    the first call's scores."""
    from paper_2607_21475_amd import cache

    lengths = [4096, 1500]
    _say("scores accumulate, 64 + %d queries" % extra)
    K, _, seq_off = synth.make_cache(lengths, seed=6, device="cuda")
    q = synth.make_queries(len(lengths), 64 + extra, seed=7, device="cuda")
    s, ws = cache.importance_scores(K, seq_off, q[:, :64].contiguous(), max(lengths))
    s, _ = cache.importance_scores(K, seq_off, q[:, 64:].contiguous(), max(lengths), scores=s,
                                   accumulate=True, ws=ws)
    torch.cuda.synchronize()
    _check(K, q, seq_off, s)


def test_scores_full_size_qwen_and_long_context():
    """The benchmark's shapes: 1792 units x 6144 rows with 32 window queries (one split per
    unit), and 131072-row units (16 splits each); sampled units against the oracle."""
    from paper_2607_21475_amd import cache

    for name, W in (("qwen7b_6k", 32), ("long_128k", 64)):
        wl = synth.WORKLOADS[name]
        U = wl.units if name == "qwen7b_6k" else 64
        n = wl.context
        _say("scores full-size %s U=%d n=%d W=%d" % (name, U, n, W))
        K, _, seq_off = synth.make_cache([n] * U, seed=8, device="cuda")
        q = synth.make_queries(U, W, seed=9, device="cuda")
        s, _ = cache.importance_scores(K, seq_off, q, n)
        torch.cuda.synchronize()
        sample = np.sort(np.random.default_rng(2).choice(U, 4, replace=False))
        for u in sample:
            ref = oracle.window_scores(synth.bf16_bits(K[u * n:(u + 1) * n]), synth.bf16_bits(q[u]))
            got = _np(s[u * n:(u + 1) * n]).astype(np.float64)
            assert np.all(np.abs(got - ref) <= RTOL * np.abs(ref) + ATOL), (name, u)
        del K, q, s
        torch.cuda.empty_cache()


def test_scores_feed_the_sampler():
    """End to end: GPU scores -> ebd_evict; the retained set equals the oracle's sampler run on
    the same scores (the scores themselves are checked above)."""
    from paper_2607_21475_amd import cache

    lengths = [4096] * 4
    _say("scores -> evict")
    K, V, seq_off = synth.make_cache(lengths, seed=10, device="cuda")
    q = synth.make_queries(len(lengths), 32, seed=11, device="cuda")
    s, _ = cache.importance_scores(K, seq_off, q, 4096)
    out = cache.evict(K, V, s, seq_off, lengths, budget_frac=0.1, seed=5, want_pi=True)
    torch.cuda.synchronize()
    off = _np(seq_off)
    same = oracle.evict_batch(off, _np(out.cap_off), _np(s)[: off[-1]], synth.bf16_bits(K),
                              synth.bf16_bits(V), 4, 64, pi_given=_np(out.pi_full)[: off[-1]],
                              seed=5)
    np.testing.assert_array_equal(_np(out.count), same["count"])
    ref = oracle.evict_batch(off, _np(out.cap_off), _np(s)[: off[-1]], synth.bf16_bits(K),
                             synth.bf16_bits(V), 4, 64, budget_frac=0.1, pi_min=0.01, seed=5)
    assert np.max(np.abs(_np(out.pi_full)[: off[-1]] - ref["pi_full"])) <= 1e-5
