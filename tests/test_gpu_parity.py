"""GPU parity: the HIP path (through the C ABI) against the fp64 oracle on the same inputs.

Bars (stated in the design notes): pi within 1e-5 absolute; masks, compaction, counts and
status bit-exact given the same fp32 pi (the GPU's pi is fed to the oracle's mask and
compaction); yhat within 2e-3 relative (vector norm per query head); Vhat, b, r within 1e-2
relative to max(|ref|, floor) with floors 1e-12 |yhat|^2, 1e-12 |yhat| and 1e-12 (so that a
certificate that is zero up to fp32 underflow of tiny weights is not failed on round-off);
ln Nhat within 1e-4 absolute.
"""
import sys

import numpy as np
import pytest
import torch

import oracle
import synth

pytestmark = pytest.mark.gpu


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


def _bits(t):
    return synth.bf16_bits(t)


def _cert_floor(key, ynorm):
    """Absolute floor of the certificate tolerance: 1e-12 in the units of the quantity."""
    return 1e-12 * (ynorm ** 2 if key == "vhat" else ynorm if key == "b" else np.ones_like(ynorm)) + 1e-300


def _inputs(lengths, seed=0, group=1, scores="window", bad=None):
    K, V, seq_off = synth.make_cache(lengths, seed=seed, device="cuda")
    if scores == "pareto":
        sc = synth.pareto_scores(K.shape[0], seed=seed + 2, device="cuda")
    else:
        sc = synth.window_scores(K, seq_off, seed=seed + 2)
    if bad is not None:
        sc = sc.clone()
        for i, v in bad:
            sc[i] = v
    q = synth.make_queries(len(lengths), group, seed=seed + 1, device="cuda")
    return K, V, seq_off, sc, q


def _evict(K, V, seq_off, sc, lengths, **kw):
    from paper_2607_21475_amd import cache

    out = cache.evict(K, V, sc, seq_off, lengths, want_pi=True, **kw)
    torch.cuda.synchronize()
    return out


def _check_evict(lengths, K, V, seq_off, sc, out, n_sink=4, n_recent=64, budget=0.1, pi_min=0.01,
                 seed=0, pi_mode=0, epoch=0, design=0):
    Kb, Vb = _bits(K), _bits(V)
    off = _np(seq_off)
    coff = _np(out.cap_off)
    s = _np(sc)
    pi_gpu = _np(out.pi_full)[: off[-1]]
    # (1) pi against the oracle's fp64 solve
    ref = oracle.evict_batch(off, coff, s, Kb, Vb, n_sink, n_recent, budget_frac=budget,
                             pi_min=pi_min, seed=seed, epoch=epoch, pi_mode=pi_mode, design=design)
    assert np.max(np.abs(pi_gpu - ref["pi_full"]), initial=0.0) <= 1e-5
    st_gpu = _np(out.status).astype(np.uint32) & ~np.uint32(oracle.ST_CAP_OVERFLOW)
    st_ref = ref["status"] & ~np.uint32(oracle.ST_CAP_OVERFLOW)
    np.testing.assert_array_equal(st_gpu, st_ref)
    # (2) mask and compaction bit-exact given the GPU's pi
    same = oracle.evict_batch(off, coff, s, Kb, Vb, n_sink, n_recent, pi_given=pi_gpu, seed=seed,
                              epoch=epoch, design=design)
    cnt = _np(out.count)
    np.testing.assert_array_equal(cnt, same["count"])
    np.testing.assert_array_equal(_np(out.status).astype(np.uint32) & oracle.ST_CAP_OVERFLOW,
                                  same["status"] & oracle.ST_CAP_OVERFLOW)
    Kc, Vc, pic, idx = _bits(out.Kc), _bits(out.Vc), _np(out.pic), _np(out.idxc)
    for u in range(len(lengths)):
        a = coff[u]
        k = min(int(cnt[u]), int(coff[u + 1] - coff[u]))
        np.testing.assert_array_equal(idx[a:a + k], same["idx"][a:a + k])
        np.testing.assert_array_equal(pic[a:a + k].view(np.uint32), same["pic"][a:a + k].view(np.uint32))
        np.testing.assert_array_equal(Kc[a:a + k], same["Kc"][a:a + k])
        np.testing.assert_array_equal(Vc[a:a + k], same["Vc"][a:a + k])
    # end-to-end masks from independently solved pi differ only on knife-edge tokens
    diff = np.abs(cnt.astype(np.int64) - ref["count"].astype(np.int64)).sum()
    assert diff <= max(2, int(2e-4 * off[-1]))
    return cnt


# ------------------------------------------------------------------------------------------
# Sampler
# ------------------------------------------------------------------------------------------
@pytest.mark.parametrize("lengths,budget", [
    ([4096] * 8, 0.10),                       # single layer, 8 KV heads, context 4096
    ([6144] * 6, 0.25),                       # 3 chunks per unit
    ([0, 1, 5, 70, 100, 777, 2047, 2048, 2049, 4096, 5000, 6144, 9000, 16384], 0.2),  # ragged
    ([20000, 40001, 3], 0.1),                 # longer than 16384: streamed scores
    # units of at most 6144 tokens: scores held in registers, 2 to 12 groups per thread
    ([0, 1, 5, 70, 100, 777, 2047, 2048, 2049, 4096, 5000, 6144], 0.2),
    ([1, 3, 511, 512, 513, 1024], 0.3),
    ([2000, 17, 1500], 0.15),
    ([3000, 4096, 2500, 100, 2049], 0.3),     # 8 groups per thread
])
def test_evict_parity(lengths, budget):
    _say("evict parity lengths=%s budget=%s" % (lengths[:6], budget))
    K, V, seq_off, sc, _ = _inputs(lengths, seed=3)
    out = _evict(K, V, seq_off, sc, lengths, budget_frac=budget, seed=11)
    _check_evict(lengths, K, V, seq_off, sc, out, budget=budget, seed=11)


def test_evict_pareto_scores_and_floor_0005():
    lengths = [8192] * 4
    _say("evict pareto")
    K, V, seq_off, sc, _ = _inputs(lengths, seed=5, scores="pareto")
    out = _evict(K, V, seq_off, sc, lengths, budget_frac=0.1, pi_min=0.005, seed=2, epoch=3)
    _check_evict(lengths, K, V, seq_off, sc, out, budget=0.1, pi_min=0.005, seed=2, epoch=3)


def test_evict_streamed_pareto_lambda():
    """Units longer than the LDS stage with heavy-tailed scores and the 0.005 floor (many scores
    clip at 1 and at the floor): the streamed sampler's lambda against the oracle's fp64 solve,
    and the full parity check."""
    lengths = [40000, 70001, 131072]
    _say("evict streamed pareto lambda")
    K, V, seq_off, sc, _ = _inputs(lengths, seed=8, scores="pareto")
    out = _evict(K, V, seq_off, sc, lengths, budget_frac=0.1, pi_min=0.005, seed=4)
    _check_evict(lengths, K, V, seq_off, sc, out, budget=0.1, pi_min=0.005, seed=4)
    off = _np(seq_off)
    s = _np(sc)
    lam_gpu = _np(out.lam)
    for u in range(len(lengths)):
        _, lam, _ = oracle.inclusion_probs(s[off[u]:off[u + 1]], 4, 64, 0.1, 0.005)
        assert abs(float(lam_gpu[u]) - lam) <= 1e-6 * lam, (u, float(lam_gpu[u]), lam)


def test_evict_literal_mode_and_protection():
    lengths = [3000, 500, 64]
    _say("evict literal mode")
    K, V, seq_off, sc, _ = _inputs(lengths, seed=6)
    out = _evict(K, V, seq_off, sc, lengths, budget_frac=0.3, n_sink=1, n_recent=7, pi_mode=1,
                 seed=9)
    _check_evict(lengths, K, V, seq_off, sc, out, n_sink=1, n_recent=7, budget=0.3, pi_mode=1,
                 seed=9)


def test_evict_degenerate_budgets_and_bad_scores():
    lengths = [1000, 1000, 1000, 1000]
    _say("evict degenerate")
    K, V, seq_off, sc, _ = _inputs(lengths, seed=7, bad=[(10, float("nan")), (20, float("inf")),
                                                          (30, -3.0)])
    sc = sc.clone()
    sc[2000:3000] = 0.0  # unit 2: all scores zero
    # per-unit budgets: floor binds (unit 0), normal, all-zero scores, nothing evicted (unit 3)
    bpu = torch.tensor([0.07, 0.2, 0.3, 1.0], dtype=torch.float32, device="cuda")
    out = _evict(K, V, seq_off, sc, lengths, budget_frac=0.0, budget_per_unit=bpu, pi_min=0.1,
                 seed=4)
    st = _np(out.status)
    assert st[0] & oracle.ST_BUDGET_FLOOR and st[0] & oracle.ST_BAD_SCORE
    assert st[3] & oracle.ST_NO_EVICTION
    Kb, Vb = _bits(K), _bits(V)
    off, coff = _np(seq_off), _np(out.cap_off)
    ref = oracle.evict_batch(off, coff, _np(sc), Kb, Vb, 4, 64, budget_per_unit=_np(bpu),
                             pi_min=0.1, seed=4)
    np.testing.assert_array_equal(st.astype(np.uint32), ref["status"])
    assert np.max(np.abs(_np(out.pi_full) - ref["pi_full"])) <= 1e-5


def test_evict_capacity_overflow_is_flagged():
    lengths = [4096, 4096]
    _say("evict overflow")
    from paper_2607_21475_amd import cache

    K, V, seq_off, sc, _ = _inputs(lengths, seed=8)
    cap_host = [0, 128, 128 + 4096]  # unit 0 far too small, unit 1 roomy
    out = cache.evict(K, V, sc, seq_off, lengths, budget_frac=0.25, seed=1, cap_off_host=cap_host,
                      want_pi=True)
    torch.cuda.synchronize()
    st = _np(out.status)
    cnt = _np(out.count)
    assert st[0] & oracle.ST_CAP_OVERFLOW and not st[1] & oracle.ST_CAP_OVERFLOW
    assert cnt[0] > 128
    same = oracle.evict_batch(_np(seq_off), np.array(cap_host, np.int64), _np(sc), _bits(K), _bits(V),
                              4, 64, pi_given=_np(out.pi_full), seed=1)
    np.testing.assert_array_equal(cnt, same["count"])
    np.testing.assert_array_equal(_bits(out.Kc)[:128], same["Kc"][:128])
    np.testing.assert_array_equal(_np(out.idxc)[:128], same["idx"][:128])


def test_evict_deterministic():
    lengths = [6144] * 4
    K, V, seq_off, sc, _ = _inputs(lengths, seed=9)
    a = _evict(K, V, seq_off, sc, lengths, budget_frac=0.25, seed=5)
    b = _evict(K, V, seq_off, sc, lengths, budget_frac=0.25, seed=5)
    assert torch.equal(a.count, b.count) and torch.equal(a.pi_full, b.pi_full)
    coff = _np(a.cap_off)
    cnt = _np(a.count)
    for u in range(len(lengths)):  # rows past count are unwritten capacity
        r = slice(int(coff[u]), int(coff[u] + cnt[u]))
        assert torch.equal(a.Kc[r].view(torch.int16), b.Kc[r].view(torch.int16))
        assert torch.equal(a.Vc[r].view(torch.int16), b.Vc[r].view(torch.int16))
        assert torch.equal(a.idxc[r], b.idxc[r]) and torch.equal(a.pic[r], b.pic[r])
    c = _evict(K, V, seq_off, sc, lengths, budget_frac=0.25, seed=5, epoch=1)
    k = int(min(a.count[0], c.count[0]))
    assert not torch.equal(a.idxc[:k], c.idxc[:k])


# ------------------------------------------------------------------------------------------
# Other designs: fixed-size systematic, top-k and uniform comparison arms
# ------------------------------------------------------------------------------------------
@pytest.mark.parametrize("lengths,budget", [
    ([4096] * 8, 0.10),
    ([0, 1, 5, 70, 100, 777, 2047, 2048, 2049, 5000, 16384], 0.25),
    ([20000, 40001, 3], 0.1),                 # streamed scores
    ([0, 1, 5, 70, 777, 2049, 5000, 6144], 0.25),   # scores in registers
    ([1024, 9], 0.2),
])
def test_evict_systematic_design(lengths, budget):
    _say("evict systematic lengths=%s budget=%s" % (lengths[:6], budget))
    K, V, seq_off, sc, _ = _inputs(lengths, seed=21)
    out = _evict(K, V, seq_off, sc, lengths, budget_frac=budget, seed=12,
                 design=oracle.DESIGN_SYSTEMATIC)
    cnt = _check_evict(lengths, K, V, seq_off, sc, out, budget=budget, seed=12,
                       design=oracle.DESIGN_SYSTEMATIC)
    # the size is fixed: floor or ceil of the unit's total integer weight / 2^32
    off = _np(seq_off)
    pi = _np(out.pi_full)
    for u in range(len(lengths)):
        a = np.ceil(pi[off[u]:off[u + 1]].astype(np.float64) * 2.0 ** 32).sum() / 2.0 ** 32
        assert int(np.floor(a)) <= cnt[u] <= int(np.ceil(a))


@pytest.mark.parametrize("lengths,budget,ties", [
    ([4096] * 8, 0.10, False),
    ([0, 1, 5, 70, 777, 2048, 5000, 16384], 0.3, True),   # integer scores: many ties
    ([20000, 40001, 3], 0.1, True),                       # streamed scores
    ([3000, 3000], 1.0, False),                           # k = |T|: keep everything
    ([0, 1, 5, 70, 777, 2048, 5000, 6144], 0.3, True),    # scores in registers
    ([900, 1024], 0.05, False),
])
def test_evict_topk_design(lengths, budget, ties):
    _say("evict top-k lengths=%s budget=%s ties=%s" % (lengths[:6], budget, ties))
    K, V, seq_off, sc, _ = _inputs(lengths, seed=22)
    if ties:
        sc = torch.floor(sc * 2000.0)
        rows = sc.shape[0]
        if rows > 40:
            sc[7] = float("nan")
            sc[30] = -0.0
            sc[31] = -3.0
    out = _evict(K, V, seq_off, sc, lengths, budget_frac=budget, seed=1, design=oracle.DESIGN_TOPK)
    off, coff = _np(seq_off), _np(out.cap_off)
    ref = oracle.evict_batch(off, coff, _np(sc), _bits(K), _bits(V), 4, 64, budget_frac=budget,
                             design=oracle.DESIGN_TOPK)
    np.testing.assert_array_equal(_np(out.pi_full)[: off[-1]], ref["pi_full"])
    np.testing.assert_array_equal(_np(out.count), ref["count"])
    np.testing.assert_array_equal(_np(out.status).astype(np.uint32), ref["status"])
    for u in range(len(lengths)):
        a, k = coff[u], int(ref["count"][u])
        np.testing.assert_array_equal(_np(out.idxc)[a:a + k], ref["idx"][a:a + k])
        np.testing.assert_array_equal(_bits(out.Kc)[a:a + k], ref["Kc"][a:a + k])
        np.testing.assert_array_equal(_bits(out.Vc)[a:a + k], ref["Vc"][a:a + k])


@pytest.mark.parametrize("lengths", [
    [4096, 333, 6144, 20000],   # streamed scores
    [4096, 333, 6144],          # scores in registers
])
def test_evict_uniform_design(lengths):
    _say("evict uniform lengths=%s" % lengths)
    K, V, seq_off, sc, _ = _inputs(lengths, seed=23)
    sc = sc.clone()
    sc[5] = float("nan")  # not read by the uniform design: no flag
    out = _evict(K, V, seq_off, sc, lengths, budget_frac=0.2, seed=4, design=oracle.DESIGN_UNIFORM)
    _check_evict(lengths, K, V, seq_off, sc, out, budget=0.2, seed=4, design=oracle.DESIGN_UNIFORM)
    assert not (_np(out.status) & oracle.ST_BAD_SCORE).any()


# ------------------------------------------------------------------------------------------
# Certified attention
# ------------------------------------------------------------------------------------------
def _check_attend(out, res, q, G, tol_y=2e-3, tol_c=1e-2):
    coff = _np(out.cap_off)
    cnt = _np(out.count)
    ref = oracle.attend_batch(coff, cnt, _bits(q), _bits(out.Kc), _bits(out.Vc), _np(out.pic))
    y, yr = _np(res["y"]).astype(np.float64), ref["y"]
    nrm = np.linalg.norm(yr, axis=2)
    err = np.linalg.norm(y - yr, axis=2)
    empty = cnt == 0
    assert np.all(err[~empty] <= tol_y * nrm[~empty]), np.max(err[~empty] / nrm[~empty])
    assert np.all(y[empty] == 0)
    for key in ("vhat", "b", "r"):
        g, r = _np(res[key]).astype(np.float64), ref[key]
        bad = np.abs(g - r) > tol_c * np.maximum(np.abs(r), _cert_floor(key, nrm))
        assert not bad.any(), (key, np.argwhere(bad)[:5], g[bad][:5], r[bad][:5])
    lse, lr = _np(res["lse"]).astype(np.float64), ref["lse"]
    assert np.all(np.isneginf(lse[empty]))
    assert np.all(np.abs(lse[~empty] - lr[~empty]) <= 1e-4 * np.maximum(1.0, np.abs(lr[~empty])))
    return ref


@pytest.mark.parametrize("lengths,G,budget,split", [
    ([4096] * 8, 1, 0.10, 0),                  # single layer, G = 1
    ([6144] * 8, 7, 0.25, 0),                  # GQA 7
    ([6144] * 8, 7, 0.25, 64),                 # many splits per unit
    ([16384] * 4, 4, 0.25, 0),                 # GQA 4, long cache
    ([2048, 777, 100, 5, 9000, 3000], 8, 0.3, 128),  # ragged tails, G = 8
    ([3000, 1500], 12, 0.2, 0),                # two head blocks (8 + 4)
    ([4096, 1000], 32, 0.25, 0),               # four head blocks of 8
    ([30000], 2, 0.245, 8192),                 # one split of the largest length (capacity 8064),
                                               # finalized in place
    ([4096, 300], 9, 0.5, 256),                # 8 + 1
    ([6144] * 6, 7, 0.5, 512),                 # a candidate chunk ends on the loop's last tiles
    ([8192] * 3, 4, 0.5, 2048),                # four chunks per split, the last one likewise
    ([6144] * 2, 2, 0.7, 64),                  # > 64 splits: split scalars combined in batches
    ([16384] * 2, 4, 0.5, 64),                 # 128 splits: candidate blocks read from the records
    # 2..4 splits and <= 4 heads: a unit's splits are the waves of one work-group, the last to
    # arrive finalizes (ragged units whose later splits are empty, an empty unit)
    ([2048, 777, 100, 5, 0, 3000], 4, 0.5, 512),
    ([20000, 9000, 4100, 513, 0], 4, 0.6, 3072),  # four splits of six chunks, ragged units
    ([9000, 7000, 300], 8, 0.5, 1536),         # three splits, G = 8
    ([16384] * 3, 4, 0.25, 2048),              # three splits
    ([6144] * 4, 1, 0.5, 1024),                # four splits, G = 1
    ([3000, 1500, 2900], 3, 0.6, 1024),        # two splits, G = 3
    ([6144] * 4, 7, 0.25, 1024),               # two splits, G = 7
    ([3000, 1500, 2900, 0], 8, 0.5, 512),      # four splits, G = 8, an empty unit
    ([3000, 1500], 12, 0.4, 768),              # two head blocks (8 + 4), two splits each
    ([2048, 777, 100, 5, 3000], 5, 0.3, 0),    # G = 5, one split per unit
    ([6144] * 3, 6, 0.25, 1024),               # G = 6, two splits in one work-group
    ([4096] * 2, 5, 0.5, 256),                 # G = 5, split records and the finalize launch
    ([3000, 2000], 10, 0.4, 0),                # head blocks of 8 + 2
    ([2500] * 2, 16, 0.3, 512),                # two full head blocks, two splits each
    ([2048, 3000, 700], 6, 0.3, 0),            # G = 6, one split per unit
    ([6144] * 2, 3, 0.5, 256),                 # G = 3 and G = 6, split records and the finalize
    ([4096] * 2, 6, 0.4, 256),                 # launch
])
def test_attend_parity(lengths, G, budget, split):
    _say("attend parity lengths=%s G=%d budget=%s split=%d" % (lengths[:4], G, budget, split))
    from paper_2607_21475_amd import cache

    K, V, seq_off, sc, q = _inputs(lengths, seed=13, group=G)
    out = _evict(K, V, seq_off, sc, lengths, budget_frac=budget, seed=21)
    res = cache.attend_certify(out, q, split_rows=split)
    torch.cuda.synchronize()
    _check_attend(out, res, q, G)


@pytest.mark.parametrize("lengths,G,split", [
    ([6144] * 6, 7, 0),                       # fused finalize
    ([4096, 300, 0, 9000], 4, 256),           # several splits, an empty unit
    ([4096, 300, 0, 9000], 4, 1024),          # the same in one work-group per unit (three splits)
])
def test_attend_without_offset(lengths, G, split):
    """EBD_F_NO_OFFSET: the uncorrected retained softmax as output, the Hajek certificate."""
    _say("attend no-offset lengths=%s G=%d split=%d" % (lengths, G, split))
    from paper_2607_21475_amd import cache

    K, V, seq_off, sc, q = _inputs(lengths, seed=31, group=G)
    out = _evict(K, V, seq_off, sc, lengths, budget_frac=0.25, seed=3)
    res = cache.attend_certify(out, q, split_rows=split, offset=False)
    ref_h = cache.attend_certify(out, q, split_rows=split)
    torch.cuda.synchronize()
    coff, cnt = _np(out.cap_off), _np(out.count)
    ref = oracle.attend_batch(coff, cnt, _bits(q), _bits(out.Kc), _bits(out.Vc), _np(out.pic),
                              use_offset=False)
    y = _np(res["y"]).astype(np.float64)
    nrm = np.linalg.norm(ref["y"], axis=2)
    live = cnt > 0
    assert np.all(np.linalg.norm(y - ref["y"], axis=2)[live] <= 2e-3 * nrm[live])
    lse = _np(res["lse"]).astype(np.float64)
    assert np.all(np.abs(lse[live] - ref["lse"][live]) <= 1e-4 * np.maximum(1.0, np.abs(ref["lse"][live])))
    for key in ("vhat", "b", "r"):  # the certificate does not depend on the flag
        np.testing.assert_array_equal(_np(res[key]), _np(ref_h[key]))
        g = _np(res[key]).astype(np.float64)
        assert np.all(np.abs(g - ref[key]) <= 1e-2 * np.maximum(np.abs(ref[key]), _cert_floor(key, nrm))), key


def test_attend_empty_and_tiny_units():
    _say("attend empty units")
    from paper_2607_21475_amd import cache

    lengths = [0, 1, 2, 17, 64, 65]
    K, V, seq_off, sc, q = _inputs(lengths, seed=14, group=3)
    out = _evict(K, V, seq_off, sc, lengths, budget_frac=0.3, n_sink=0, n_recent=1, seed=2)
    res = cache.attend_certify(out, q)
    torch.cuda.synchronize()
    assert _np(out.count)[0] == 0
    _check_attend(out, res, q, 3)


def test_attend_range_term_rescan_path():
    """Values with equal norms and equal weights: candidate bounds cannot decide, so splits are
    rescanned; b must still equal the oracle's exact maximum."""
    _say("attend rescan path")
    from paper_2607_21475_amd import cache

    U, n, G = 4, 2048, 2
    lengths = [n] * U
    K = torch.zeros((U * n, 128), dtype=torch.bfloat16, device="cuda")
    g = torch.Generator(device="cuda")
    g.manual_seed(3)
    sign = torch.randint(0, 2, (U * n, 128), generator=g, device="cuda").float() * 2 - 1
    V = sign.to(torch.bfloat16)  # every |v| = sqrt(128)
    seq_off = synth.seq_offsets(lengths, "cuda")
    sc = torch.ones(U * n, dtype=torch.float32, device="cuda")
    q = synth.make_queries(U, G, seed=4, device="cuda")
    out = _evict(K, V, seq_off, sc, lengths, budget_frac=0.2, seed=8)
    res = cache.attend_certify(out, q, split_rows=128)
    torch.cuda.synchronize()
    assert cache.rescans(res["ws"], U, G) > 0
    _check_attend(out, res, q, G)


def test_attend_range_term_long_candidate_list():
    """Equal norms and weights in one long split: every candidate's bound beats the best value, so
    the finalize lists far more candidates than one evaluation batch holds (several batches)."""
    _say("attend long candidate list")
    from paper_2607_21475_amd import cache

    U, n, G = 2, 16384, 2
    lengths = [n] * U
    K = torch.zeros((U * n, 128), dtype=torch.bfloat16, device="cuda")
    g = torch.Generator(device="cuda")
    g.manual_seed(5)
    sign = torch.randint(0, 2, (U * n, 128), generator=g, device="cuda").float() * 2 - 1
    V = sign.to(torch.bfloat16)
    seq_off = synth.seq_offsets(lengths, "cuda")
    sc = torch.ones(U * n, dtype=torch.float32, device="cuda")
    q = synth.make_queries(U, G, seed=6, device="cuda")
    out = _evict(K, V, seq_off, sc, lengths, budget_frac=0.45, seed=9)
    assert 4096 < int(_np(out.count).min()) and int(_np(out.count).max()) <= 8192
    res = cache.attend_certify(out, q, split_rows=8192)  # one split per unit: the fused finalize
    torch.cuda.synchronize()
    _check_attend(out, res, q, G)


def test_attend_pi_one_is_full_attention():
    """Budget 1: nothing evicted, pi = 1 everywhere, so yhat is full attention and Vhat = b = r = 0."""
    _say("attend pi=1")
    from paper_2607_21475_amd import cache

    lengths = [3000, 1000]
    K, V, seq_off, sc, q = _inputs(lengths, seed=15, group=4)
    out = _evict(K, V, seq_off, sc, lengths, budget_frac=1.0, seed=1)
    res = cache.attend_certify(out, q)
    torch.cuda.synchronize()
    yfull = oracle.full_batch(_np(seq_off), _bits(q), _bits(K), _bits(V))
    err = np.linalg.norm(_np(res["y"]) - yfull, axis=2) / np.linalg.norm(yfull, axis=2)
    assert np.max(err) <= 2e-3
    assert np.all(_np(res["vhat"]) == 0) and np.all(_np(res["b"]) == 0) and np.all(_np(res["r"]) == 0)


@pytest.mark.parametrize("scores,G,split", [("window", 4, 0), ("pareto", 4, 0), ("window", 7, 256)])
def test_attend_paper_floor_1e6(scores, G, split):
    """The paper's floor pi_min = 1e-6 (Sec. 3.3 eq. (2)), so 1/pi reaches 1e6.  Neither score
    recipe gets near it by itself (window scores vary by a few-fold, Pareto scores are >= 1), so
    a random 30% of the tokens have their score scaled down log-uniformly by up to 1e7 (tokens
    the window barely attends to): their pi then spans 1e-6 .. 0.1, and some are retained."""
    _say("attend floor 1e-6 scores=%s G=%d split=%d" % (scores, G, split))
    from paper_2607_21475_amd import cache

    lengths = [6144] * 48
    K, V, seq_off, sc, q = _inputs(lengths, seed=41, group=G, scores=scores)
    g = torch.Generator(device="cuda")
    g.manual_seed(43)
    low = torch.rand(sc.shape, generator=g, device="cuda") < 0.3
    f = torch.pow(10.0, -7.0 * torch.rand(sc.shape, generator=g, device="cuda"))
    sc = torch.where(low, sc * f, sc)
    out = _evict(K, V, seq_off, sc, lengths, budget_frac=0.1, pi_min=1e-6, seed=17)
    _check_evict(lengths, K, V, seq_off, sc, out, budget=0.1, pi_min=1e-6, seed=17)
    assert (_np(out.pi_full)[: 6144 * 48] == np.float32(1e-6)).sum() > 1000  # the floor binds
    res = cache.attend_certify(out, q, split_rows=split)
    torch.cuda.synchronize()
    _check_attend(out, res, q, G)
    assert not _np(res["status"]).any()
    coff, cnt = _np(out.cap_off), _np(out.count)
    pic = _np(out.pic)
    kept = np.concatenate([pic[coff[u]:coff[u] + cnt[u]] for u in range(len(lengths))])
    assert kept.min() < 1e-3  # rows drawn close to the floor are retained


def _retained_cache(units, extra_cap=0):
    """A compacted cache laid out as ebd_evict writes it, from per-unit host arrays (Kc, Vc bf16
    bits [c, 128], pi fp32 [c]): capacity = c + extra_cap rows, count = c."""
    from paper_2607_21475_amd import cache

    caps = [len(p) + extra_cap for _, _, p in units]
    off = np.concatenate([[0], np.cumsum(caps)]).astype(np.int64)
    rows = int(off[-1])
    Kc = np.zeros((rows, 128), np.uint16)
    Vc = np.zeros((rows, 128), np.uint16)
    pic = np.ones(rows, np.float32)
    for u, (k, v, p) in enumerate(units):
        a = off[u]
        Kc[a:a + len(p)], Vc[a:a + len(p)], pic[a:a + len(p)] = k, v, p
    dev = "cuda"
    as_bf16 = lambda x: torch.from_numpy(x.view(np.int16)).to(dev).view(torch.bfloat16)  # noqa: E731
    return cache.RetainedCache(
        Kc=as_bf16(Kc), Vc=as_bf16(Vc), pic=torch.from_numpy(pic).to(dev),
        idxc=torch.zeros(rows, dtype=torch.int32, device=dev),
        count=torch.tensor([len(p) for _, _, p in units], dtype=torch.int32, device=dev),
        status=torch.zeros(len(units), dtype=torch.int32, device=dev),
        cap_off=torch.from_numpy(off).to(dev), max_cap=max(caps))


def _dominated_unit(rng, n, G, q, boost, pi_floor=1e-6, tail_pi=(0.05, 1.0)):
    """n retained rows: 68 certain, the rest a tail with pi in tail_pi, and one row j drawn at the
    floor whose key is pushed along q's first head so that its Hajek weight a_j / pi_j exceeds the
    rest of Nhat by a large factor (the cancellation case of the one-pass variance)."""
    from helpers import bf16_to_f64, rand_bf16, to_bf16_bits

    K = rand_bf16(rng, (n, 128))
    V = rand_bf16(rng, (n, 128))
    pi = rng.uniform(*tail_pi, n).astype(np.float32)
    pi[:68] = 1.0
    j = n // 2
    qf = bf16_to_f64(q[0])
    K[j] = to_bf16_bits(bf16_to_f64(K[j]) + boost * qf / np.linalg.norm(qf))
    pi[j] = pi_floor
    return K, V, pi


@pytest.mark.parametrize("G,n,boost,split,dup", [
    (1, 600, 0.0, 0, False),     # 1/pi = 1e6 alone: the floor row outweighs the rest ~3e2-fold
    (4, 1500, 4.0, 0, False),    # its key also aligned with head 0's query: ~7e3-fold there
    (7, 3000, 3.0, 0, False),
    (4, 5000, 4.5, 512, False),  # several splits: pivots from every split meet in attend_finalize
    (8, 900, 2.0, 128, False),
    (4, 1500, 9.0, 0, False),    # 1e5 to 1e7-fold: the floor row alone makes yhat to fp32 precision
    (4, 1500, 4.0, 0, True),     # two identical dominating rows: the direct re-summation
    (7, 3000, 3.0, 512, True),
    (4, 1500, 4.0, 512, False),  # three splits in one work-group: pivots meet in its finalize
    (2, 1500, 9.0, 768, True),   # two splits in one work-group, direct re-summation
])
def test_attend_vhat_dominant_tail_row(G, n, boost, split, dup):
    """A floor row (pi = 1e-6) retained and dominating Nhat: yhat ~ v_j, so the one-pass
    C2 - 2 yhat.Cv + |yhat|^2 C0 would cancel by many orders of magnitude.  The split kernel
    keeps the largest-weight row of each head out of its sums and the finalize adds it back in
    closed form, so Vhat, b and r match the oracle's two-pass definition without a second pass.
    With the dominating row duplicated (two identical rows), the rest sums themselves cancel and
    the finalize sums those heads again directly."""
    _say("attend dominant tail row G=%d n=%d boost=%s split=%d dup=%s" % (G, n, boost, split, dup))
    from paper_2607_21475_amd import cache
    from helpers import bf16_to_f64, rand_bf16

    rng = np.random.default_rng(100 + G)
    U = 6
    q = rand_bf16(rng, (U, G, 128))
    units = [_dominated_unit(rng, n, G, q[u], boost) for u in range(U - 1)]
    if dup:  # a copy of the dominating row right after it
        for K_, V_, p_ in units:
            j = n // 2
            K_[j + 1], V_[j + 1], p_[j + 1] = K_[j], V_[j], p_[j]
    units.append((rand_bf16(rng, (n, 128)), rand_bf16(rng, (n, 128)),
                  rng.uniform(0.05, 1.0, n).astype(np.float32)))  # an ordinary unit beside them
    rc = _retained_cache(units)
    qt = torch.from_numpy(q.view(np.int16)).cuda().view(torch.bfloat16)
    res = cache.attend_certify(rc, qt, split_rows=split)
    torch.cuda.synchronize()
    ref = _check_attend(rc, res, qt, G)
    direct = cache.direct_variances(res["ws"], U, G)
    if dup:
        assert direct >= U - 1
    else:
        assert direct == 0
    # the dominated units really are in the cancelling regime: head 0's Vhat is far below the
    # scale |v_j|^2 of the dominating row's own C2 term (more than 6 bits would cancel)
    vj2 = np.array([np.sum(bf16_to_f64(Vu[n // 2]) ** 2) for _, Vu, _ in units[:U - 1]])
    assert np.all(ref["vhat"][: U - 1, 0] < vj2 / 64)


def test_attend_status_reports_unseen_rows():
    """Rows the step cannot see are reported, never silently dropped: a count above the unit's
    capacity (EBD_ST_CAP_OVERFLOW) and units longer than the planned max_rows (EBD_ST_BAD_LAYOUT).
    The outputs cover the rows seen, as the oracle computes them over those rows."""
    _say("attend status")
    import dataclasses

    from paper_2607_21475_amd import cache
    from helpers import rand_bf16

    rng = np.random.default_rng(7)
    G, sizes = 2, [300, 40, 700, 96]
    units = [(rand_bf16(rng, (c, 128)), rand_bf16(rng, (c, 128)),
              rng.uniform(0.05, 1.0, c).astype(np.float32)) for c in sizes]
    rc = _retained_cache(units)
    q = rand_bf16(rng, (len(sizes), G, 128))
    qt = torch.from_numpy(q.view(np.int16)).cuda().view(torch.bfloat16)
    res = cache.attend_certify(rc, qt)
    torch.cuda.synchronize()
    assert not _np(res["status"]).any()
    # unit 1 claims 5 rows beyond its capacity
    rc.count[1] += 5
    res = cache.attend_certify(rc, qt)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(_np(res["status"]), [0, 1, 0, 0])
    rc.count[1] -= 5
    # a plan for at most 128 rows: units 0 and 2 are longer
    short = dataclasses.replace(rc, max_cap=128)
    res = cache.attend_certify(short, qt)
    torch.cuda.synchronize()
    st = _np(res["status"])
    np.testing.assert_array_equal(st & 16, [16, 0, 16, 0])
    seen = [min(c, 128) for c in sizes]  # the planner's single 128-row split per unit
    for u, (k, v, p) in enumerate(units):
        ref = oracle.attend_certify(q[u], k[:seen[u]], v[:seen[u]], p[:seen[u]])
        y = _np(res["y"][u]).astype(np.float64)
        assert np.all(np.linalg.norm(y - ref["y"], axis=1) <= 2e-3 * np.linalg.norm(ref["y"], axis=1))


def test_append_certain():
    _say("append")
    from paper_2607_21475_amd import cache, ebd_append_certain

    lengths = [1000, 1000, 1000]
    K, V, seq_off, sc, q = _inputs(lengths, seed=16, group=2)
    cap_host = cache.plan_capacity(lengths, 0.1, 4, 64, extra=2)
    out = cache.evict(K, V, sc, seq_off, lengths, budget_frac=0.1, seed=3, cap_off_host=cap_host)
    torch.cuda.synchronize()
    c0 = _np(out.count).copy()
    kn = synth.make_queries(3, 1, seed=30, device="cuda")[:, 0].contiguous()
    vn = synth.make_queries(3, 1, seed=31, device="cuda")[:, 0].contiguous()
    pos = torch.tensor([1000, 1000, 1000], dtype=torch.int32, device="cuda")
    ebd_append_certain(3, out.cap_off, out.count, kn, vn, out.Kc, out.Vc, out.pic, out.idxc, pos,
                       out.status)
    torch.cuda.synchronize()
    c1 = _np(out.count)
    np.testing.assert_array_equal(c1, c0 + 1)
    coff = _np(out.cap_off)
    for u in range(3):
        r = coff[u] + c0[u]
        np.testing.assert_array_equal(_bits(out.Kc)[r], _bits(kn)[u])
        np.testing.assert_array_equal(_bits(out.Vc)[r], _bits(vn)[u])
        assert _np(out.pic)[r] == 1.0 and _np(out.idxc)[r] == 1000
    res = cache.attend_certify(out, q)
    torch.cuda.synchronize()
    _check_attend(out, res, q, 2)
    # fill unit 0 to capacity: the next append is refused and flagged
    room = int(coff[1] - coff[0] - c1[0])
    for _ in range(room):
        ebd_append_certain(3, out.cap_off, out.count, kn, vn, out.Kc, out.Vc, out.pic, out.idxc, pos,
                           out.status)
    ebd_append_certain(3, out.cap_off, out.count, kn, vn, out.Kc, out.Vc, out.pic, out.idxc, pos,
                       out.status)
    torch.cuda.synchronize()
    assert _np(out.count)[0] == coff[1] - coff[0]
    assert _np(out.status)[0] & oracle.ST_CAP_OVERFLOW


@pytest.mark.parametrize("lengths,G,split", [
    ([3000, 2500, 4100, 700], 4, 0),     # one split per unit, finalized in place
    ([3000, 2500, 4100, 700], 4, 1024),  # a unit's splits as the waves of one work-group
    ([6144, 6144], 2, 256),              # split records, then the finalize launch
])
def test_decode_step_graph_replay(lengths, G, split):
    """A decode step (append a pi = 1 row, then certified attention) captured in a HIP graph: the
    library launches kernels only (no allocation, copy or memset), so the graph holds the whole
    step.  Each replay, with eager work and a synchronization between replays, matches an eager
    step on a twin cache bit for bit, and the last replay's outputs match the oracle."""
    _say("graph replay of a decode step %s G=%d split=%d" % (lengths, G, split))
    import paper_2607_21475_amd as ebd
    from paper_2607_21475_amd import cache

    U, steps = len(lengths), 4
    K, V, seq_off, sc, _ = _inputs(lengths, seed=23, group=G)
    cap_host = cache.plan_capacity(lengths, 0.25, 4, 64, extra=steps + 1)
    A = cache.evict(K, V, sc, seq_off, lengths, budget_frac=0.25, seed=7, cap_off_host=cap_host)
    B = cache.evict(K, V, sc, seq_off, lengths, budget_frac=0.25, seed=7, cap_off_host=cap_host)
    p = ebd.attend_params(U, G, A.max_cap, A.cap_off, split)
    need = ebd.ebd_workspace_size(ebd.EBD_WS_ATTEND, p)
    wsA, wsB = ebd.workspace(need), ebd.workspace(need)
    keys = ("y", "vhat", "lse", "b", "r", "st")

    def outputs():
        o = {k: torch.empty((U, G), dtype=torch.float32, device="cuda") for k in keys[1:5]}
        o["y"] = torch.empty((U, G, 128), dtype=torch.float32, device="cuda")
        o["st"] = torch.empty((U,), dtype=torch.int32, device="cuda")
        return o

    oA, oB = outputs(), outputs()
    qs = [synth.make_queries(U, G, seed=40 + t, device="cuda") for t in range(steps + 1)]
    kn = [synth.make_queries(U, 1, seed=50 + t, device="cuda")[:, 0].contiguous() for t in range(steps + 1)]
    vn = [synth.make_queries(U, 1, seed=60 + t, device="cuda")[:, 0].contiguous() for t in range(steps + 1)]
    pos = [torch.tensor([n + t for n in lengths], dtype=torch.int32, device="cuda")
           for t in range(steps + 1)]
    q_s, k_s, v_s, p_s = qs[0].clone(), kn[0].clone(), vn[0].clone(), pos[0].clone()

    def step(rc, o, ws, q, k, v, ps):
        ebd.ebd_append_certain(U, rc.cap_off, rc.count, k, v, rc.Kc, rc.Vc, rc.pic, rc.idxc, ps,
                               rc.status)
        ebd.ebd_attend_certify(p, q, rc.Kc, rc.Vc, rc.pic, rc.count, o["y"], o["vhat"], o["lse"], ws,
                               brange=o["b"], radius=o["r"], status=o["st"])

    # step 0 eagerly on both caches (the twin's on a side stream, as before a capture), then capture
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step(B, oB, wsB, q_s, k_s, v_s, p_s)
    torch.cuda.current_stream().wait_stream(side)
    step(A, oA, wsA, qs[0], kn[0], vn[0], pos[0])
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step(B, oB, wsB, q_s, k_s, v_s, p_s)
    torch.cuda.synchronize()
    for t in range(1, steps + 1):
        q_s.copy_(qs[t])
        k_s.copy_(kn[t])
        v_s.copy_(vn[t])
        p_s.copy_(pos[t])
        g.replay()
        step(A, oA, wsA, qs[t], kn[t], vn[t], pos[t])
        torch.cuda.synchronize()
        for k in keys:
            assert torch.equal(oA[k], oB[k]), (t, k)
        assert torch.equal(A.count, B.count), t
        coff, cnt = _np(A.cap_off), _np(A.count)
        for k in ("Kc", "Vc", "pic", "idxc"):  # the retained rows (capacity past them is unwritten)
            a, b = getattr(A, k), getattr(B, k)
            for u in range(U):
                lo, hi = int(coff[u]), int(coff[u] + cnt[u])
                assert torch.equal(a[lo:hi], b[lo:hi]), (t, k, u)
    assert not _np(oB["st"]).any()
    np.testing.assert_array_equal(_np(B.count), _np(A.count))
    _check_attend(B, oB, q_s, G)


# ------------------------------------------------------------------------------------------
# Full-size workload (the benchmark's launch configuration), sampled units
# ------------------------------------------------------------------------------------------
def test_qwen7b_full_size_sampled_units():
    wl = synth.WORKLOADS["qwen7b_6k"]
    _say("full-size %s U=%d" % (wl.name, wl.units))
    from paper_2607_21475_amd import cache

    inp = synth.make_workload_inputs(wl, seed=0, device="cuda")
    lengths = [wl.context] * wl.units
    rng = np.random.default_rng(0)
    sample = np.sort(rng.choice(wl.units, 12, replace=False))
    for budget in wl.budgets:
        out = cache.evict(inp["K"], inp["V"], inp["scores"], inp["seq_off"], lengths,
                          budget_frac=budget, n_sink=wl.n_sink, n_recent=wl.n_recent,
                          pi_min=wl.pi_min, seed=0, want_pi=True)
        res = cache.attend_certify(out, inp["q"])
        torch.cuda.synchronize()
        assert not (_np(out.status) & oracle.ST_CAP_OVERFLOW).any()
        n = wl.context
        cnt = _np(out.count)
        coff = _np(out.cap_off)
        pi_all = _np(out.pi_full)
        for u in sample:
            sl = slice(u * n, (u + 1) * n)
            s = _np(inp["scores"][sl])
            Kb, Vb = _bits(inp["K"][sl]), _bits(inp["V"][sl])
            pi_ref, lam, st = oracle.inclusion_probs(s, wl.n_sink, wl.n_recent, budget, wl.pi_min)
            assert np.max(np.abs(pi_all[sl] - pi_ref)) <= 1e-5
            m = oracle.mask(pi_all[sl], 0, int(u), 0)
            Kc_r, Vc_r, pic_r, idx_r, c_r = oracle.compact(m, pi_all[sl], Kb, Vb)
            assert c_r == cnt[u]
            a = coff[u]
            np.testing.assert_array_equal(_np(out.idxc)[a:a + c_r], idx_r)
            np.testing.assert_array_equal(_bits(out.Kc[a:a + c_r]), Kc_r)
            np.testing.assert_array_equal(_bits(out.Vc[a:a + c_r]), Vc_r)
            ref = oracle.attend_certify(_bits(inp["q"][u]), Kc_r, Vc_r, pic_r)
            y = _np(res["y"][u]).astype(np.float64)
            assert np.all(np.linalg.norm(y - ref["y"], axis=1) <= 2e-3 * np.linalg.norm(ref["y"], axis=1))
            for key in ("vhat", "b", "r"):
                g = _np(res[key][u]).astype(np.float64)
                assert np.all(np.abs(g - ref[key]) <= 1e-2 * np.abs(ref[key])), (key, u, g, ref[key])
        if budget == 0.25:  # the benchmark's block-contribution launch, sampled units
            import paper_2607_21475_amd as ebd

            nb = (n + 63) // 64
            blocks = torch.empty((wl.units, nb), dtype=torch.float32, device="cuda")
            ebd.ebd_block_contributions(wl.units, wl.group, nb, out.max_cap, out.cap_off, inp["q"],
                                        out.Kc, out.Vc, out.pic, out.idxc, out.count, res["y"],
                                        res["lse"], blocks)
            torch.cuda.synchronize()
            got = _np(blocks).astype(np.float64)
            for u in sample[:4]:
                a, c = coff[u], int(cnt[u])
                bref = oracle.block_contributions(
                    _bits(inp["q"][u]), _bits(out.Kc[a:a + c]), _bits(out.Vc[a:a + c]),
                    _np(out.pic[a:a + c]), _np(out.idxc[a:a + c]),
                    _np(res["y"][u]).astype(np.float64), _np(res["lse"][u]).astype(np.float64),
                    nb, 64)
                tol = 1e-3 * np.abs(bref) + 1e-7 * max(bref.max(initial=0.0), 1e-30)
                assert np.all(np.abs(got[u] - bref) <= tol), u
        del out, res
    del inp
    torch.cuda.empty_cache()


def _check_unit_end_to_end(u, sl, scores, K, V, pi_all, out, budget, n_sink, n_recent, pi_min,
                           seed=0, appended=()):
    """One sampled unit: pi against the oracle's solve, then the oracle's mask, compaction and
    appended certain rows give the retained set the GPU holds (bit-exact)."""
    s = _np(scores[sl])
    pi_ref, _, _ = oracle.inclusion_probs(s, n_sink, n_recent, budget, pi_min)
    assert np.max(np.abs(pi_all[sl] - pi_ref)) <= 1e-5
    Kb, Vb = _bits(K[sl]), _bits(V[sl])
    m = oracle.mask(pi_all[sl], seed, int(u), 0)
    Kc_r, Vc_r, pic_r, idx_r, c_r = oracle.compact(m, pi_all[sl], Kb, Vb)
    a = int(_np(out.cap_off[u:u + 1])[0])
    c = c_r + len(appended)
    assert int(_np(out.count[u:u + 1])[0]) == c
    if appended:
        Kc_r = np.concatenate([Kc_r] + [k[None] for k, _, _ in appended])
        Vc_r = np.concatenate([Vc_r] + [v[None] for _, v, _ in appended])
        pic_r = np.concatenate([pic_r, np.ones(len(appended), np.float32)])
        idx_r = np.concatenate([idx_r, np.array([p for _, _, p in appended], np.int32)])
    np.testing.assert_array_equal(_np(out.idxc[a:a + c]), idx_r)
    np.testing.assert_array_equal(_np(out.pic[a:a + c]).view(np.uint32), pic_r.view(np.uint32))
    np.testing.assert_array_equal(_bits(out.Kc[a:a + c]), Kc_r)
    np.testing.assert_array_equal(_bits(out.Vc[a:a + c]), Vc_r)
    return Kc_r, Vc_r, pic_r


def _check_unit_attend(u, q, res, Kc_r, Vc_r, pic_r):
    ref = oracle.attend_certify(_bits(q[u]), Kc_r, Vc_r, pic_r)
    y = _np(res["y"][u]).astype(np.float64)
    err = np.linalg.norm(y - ref["y"], axis=1) / np.linalg.norm(ref["y"], axis=1)
    assert np.all(err <= 2e-3), (u, err)
    for key in ("vhat", "b", "r"):
        g = _np(res[key][u]).astype(np.float64)
        floor = _cert_floor(key, np.linalg.norm(ref["y"], axis=1))
        assert np.all(np.abs(g - ref[key]) <= 1e-2 * np.maximum(np.abs(ref[key]), floor)), (key, u, g, ref[key])
    lse = _np(res["lse"][u]).astype(np.float64)
    assert np.all(np.abs(lse - ref["lse"]) <= 1e-4 * np.maximum(1.0, np.abs(ref["lse"])))
    return ref


def _decode_run(wl, check_steps, n_sample=8):
    """Full-size workload: evict once, then decode steps that each append one certain token per
    unit (pi = 1) and run the certified attention; sampled units are checked end to end against
    the oracle at `check_steps`."""
    from paper_2607_21475_amd import cache, ebd_append_certain

    U, n, G = wl.units, wl.context, wl.group
    budget = wl.budgets[0]
    _say("full-size %s U=%d n=%d G=%d budget=%s steps=%d" % (wl.name, U, n, G, budget, wl.decode_steps))
    inp = synth.make_workload_inputs(wl, seed=0, device="cuda")
    lengths = [n] * U
    out = cache.evict(inp["K"], inp["V"], inp["scores"], inp["seq_off"], lengths, budget_frac=budget,
                      n_sink=wl.n_sink, n_recent=wl.n_recent, pi_min=wl.pi_min, seed=0,
                      extra_rows=wl.decode_steps, want_pi=True)
    torch.cuda.synchronize()
    assert not (_np(out.status) & oracle.ST_CAP_OVERFLOW).any()
    pi_all = _np(out.pi_full)
    sample = np.sort(np.random.default_rng(1).choice(U, n_sample, replace=False))
    appended = {int(u): [] for u in sample}
    ws = None
    checked = 0
    for t in range(wl.decode_steps):
        kn = synth.make_queries(U, 1, seed=10000 + t, device="cuda")[:, 0].contiguous()
        vn = synth.make_queries(U, 1, seed=20000 + t, device="cuda")[:, 0].contiguous()
        pos = torch.full((U,), n + t, dtype=torch.int32, device="cuda")
        ebd_append_certain(U, out.cap_off, out.count, kn, vn, out.Kc, out.Vc, out.pic, out.idxc, pos,
                           out.status)
        q = synth.make_queries(U, G, seed=30000 + t, device="cuda")
        res = cache.attend_certify(out, q, ws=ws)
        ws = res["ws"]
        kb, vb = _bits(kn[torch.as_tensor(sample, device="cuda")]), _bits(vn[torch.as_tensor(sample, device="cuda")])
        for i, u in enumerate(sample):
            appended[int(u)].append((kb[i], vb[i], n + t))
        if t in check_steps:
            torch.cuda.synchronize()
            assert not (_np(out.status) & oracle.ST_CAP_OVERFLOW).any()
            for u in sample:
                sl = slice(int(u) * n, (int(u) + 1) * n)
                Kc_r, Vc_r, pic_r = _check_unit_end_to_end(
                    int(u), sl, inp["scores"], inp["K"], inp["V"], pi_all, out, budget, wl.n_sink,
                    wl.n_recent, wl.pi_min, appended=appended[int(u)])
                _check_unit_attend(int(u), q, res, Kc_r, Vc_r, pic_r)
            checked += 1
            _say("  step %d: %d sampled units match" % (t, len(sample)))
    assert checked == len(check_steps)
    del inp, out, res
    torch.cuda.empty_cache()


def test_llama8b_full_size_decode_with_appends():
    wl = synth.WORKLOADS["llama8b_16k"]
    _decode_run(wl, check_steps=(0, wl.decode_steps - 1))


def test_long_128k_full_size_decode_streamed_scores():
    """131072-token units: the sampler streams scores (they do not fit the work-group's LDS)."""
    wl = synth.WORKLOADS["long_128k"]
    _decode_run(wl, check_steps=(0, wl.decode_steps - 1))


def test_replay_grid_chunk_per_unit_budgets():
    """One chunk of the replay grid: cells cycle through 5 budgets and 3 context lengths, 8 KV
    heads per cell, G = 1, per-unit budgets; one sampled unit per (budget, context) pair is
    checked end to end, and the coverage of the radius is reported (not gated)."""
    from paper_2607_21475_amd import cache

    c0, ncell = 3015, 1512
    cells = [synth.replay_cell(c) for c in range(c0, c0 + ncell)]
    H = synth.REPLAY_KV_HEADS
    lengths = [ctx for (_, ctx, _, _) in cells for _ in range(H)]
    budgets = [b for (b, _, _, _) in cells for _ in range(H)]
    U = len(lengths)
    _say("replay chunk cells %d..%d U=%d rows=%d" % (c0, c0 + ncell, U, sum(lengths)))
    K, V, seq_off = synth.make_cache(lengths, seed=5, device="cuda")
    sc = synth.window_scores(K, seq_off, seed=6)
    q = synth.make_queries(U, 1, seed=7, device="cuda")
    bpu = torch.tensor(budgets, dtype=torch.float32, device="cuda")
    out = cache.evict(K, V, sc, seq_off, lengths, budget_per_unit=bpu, seed=9, want_pi=True)
    res = cache.attend_certify(out, q)
    torch.cuda.synchronize()
    assert not (_np(out.status) & oracle.ST_CAP_OVERFLOW).any()
    pi_all = _np(out.pi_full)
    off = _np(seq_off)
    covered = 0
    for j in range(15):  # cells c0 + j cover every (budget, context) pair once
        u = j * H + (j % H)
        sl = slice(int(off[u]), int(off[u + 1]))
        Kc_r, Vc_r, pic_r = _check_unit_end_to_end(u, sl, sc, K, V, pi_all, out, budgets[u], 4, 64,
                                                   0.01, seed=9)
        ref = _check_unit_attend(u, q, res, Kc_r, Vc_r, pic_r)
        yfull = oracle.full_attention(_bits(q[u]), _bits(K[sl]), _bits(V[sl]))
        err = np.linalg.norm(ref["y"] - yfull) / np.linalg.norm(yfull)
        covered += int(err <= ref["r"][0])
    _say("  radius covered the full-cache output for %d of 15 sampled units" % covered)
