"""Pins for the oracle's attention output and certificate arithmetic.

  * pi = 1 everywhere: the Hajek output (eq. (3)) is full softmax attention
    (eq. (1)), checked against torch's scaled_dot_product_attention in fp64
    on the CPU, and the certificate vanishes.
  * uniform pi: the offset cancels (plain softmax over the retained rows).
  * the logit-offset form softmax(s - ln pi) V equals the oracle's explicit
    ratio form (Sec. 3.3: "add log(1/pi) to the retained logit").
  * invariances the definitions imply (value translation and scaling,
    permutation of the retained rows) and the identity Vhat = b^2 when exactly
    one tail token is retained (Theorem 2 and eq. (4) share that one term).
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
from helpers import bf16_to_f64, rand_bf16, to_bf16_bits


def _sdpa(qb, Kb, Vb, bias=None):
    q = torch.tensor(bf16_to_f64(qb))[None, :, None, :]  # [1, G, 1, d]
    k = torch.tensor(bf16_to_f64(Kb))[None, None].expand(1, q.shape[1], -1, -1)
    v = torch.tensor(bf16_to_f64(Vb))[None, None].expand(1, q.shape[1], -1, -1)
    mask = None
    if bias is not None:
        mask = torch.tensor(bias)[None, None, None, :].expand(1, q.shape[1], 1, -1)
    return F.scaled_dot_product_attention(q, k, v, attn_mask=mask)[0, :, 0, :].numpy()


@pytest.mark.parametrize("G,n,d", [(1, 1, 128), (1, 300, 128), (7, 500, 128), (4, 64, 16)])
def test_pi_one_is_full_attention(G, n, d):
    rng = np.random.default_rng(n + G)
    q = rand_bf16(rng, (G, d))
    K = rand_bf16(rng, (n, d), scale=2.0)
    V = rand_bf16(rng, (n, d))
    out = oracle.attend_certify(q, K, V, np.ones(n, np.float32))
    ref = _sdpa(q, K, V)
    np.testing.assert_allclose(out["y"], ref, rtol=1e-12, atol=1e-13)
    # full-cache eq. (1) routine agrees too
    np.testing.assert_allclose(oracle.full_attention(q, K, V), ref, rtol=1e-12, atol=1e-13)
    # ln Nhat = logsumexp of the scores
    s = bf16_to_f64(q) @ bf16_to_f64(K).T / np.sqrt(d)
    lse = torch.logsumexp(torch.tensor(s), dim=1).numpy()
    np.testing.assert_allclose(out["lse"], lse, rtol=1e-13, atol=1e-13)
    assert np.all(out["vhat"] == 0) and np.all(out["b"] == 0) and np.all(out["r"] == 0)


def test_uniform_pi_offset_cancels():
    rng = np.random.default_rng(1)
    G, n, d = 3, 400, 128
    q = rand_bf16(rng, (G, d))
    K = rand_bf16(rng, (n, d))
    V = rand_bf16(rng, (n, d))
    out = oracle.attend_certify(q, K, V, np.full(n, 0.3, np.float32))
    np.testing.assert_allclose(out["y"], _sdpa(q, K, V), rtol=1e-12, atol=1e-13)
    assert np.all(out["vhat"] > 0)


def test_logit_offset_equals_ratio_form():
    rng = np.random.default_rng(2)
    G, n, d = 5, 333, 128
    q = rand_bf16(rng, (G, d))
    K = rand_bf16(rng, (n, d), scale=1.5)
    V = rand_bf16(rng, (n, d))
    pi = rng.uniform(0.01, 1.0, n).astype(np.float32)
    pi[:20] = 1.0
    out = oracle.attend_certify(q, K, V, pi)
    bias = -np.log(pi.astype(np.float64))
    np.testing.assert_allclose(out["y"], _sdpa(q, K, V, bias=bias), rtol=1e-12, atol=1e-13)
    s = bf16_to_f64(q) @ bf16_to_f64(K).T / np.sqrt(d) + bias[None, :]
    np.testing.assert_allclose(out["lse"], torch.logsumexp(torch.tensor(s), 1).numpy(), rtol=1e-13)
    # use_offset = False: the uncorrected retained softmax as output, the Hajek certificate
    out0 = oracle.attend_certify(q, K, V, pi, use_offset=False)
    np.testing.assert_allclose(out0["y"], _sdpa(q, K, V), rtol=1e-12, atol=1e-13)
    s0 = bf16_to_f64(q) @ bf16_to_f64(K).T / np.sqrt(d)
    np.testing.assert_allclose(out0["lse"], torch.logsumexp(torch.tensor(s0), 1).numpy(), rtol=1e-13)
    for key in ("vhat", "b", "r"):
        np.testing.assert_array_equal(out0[key], out[key])


def _case(seed, G=2, n=200, d=128, loc=0.0):
    rng = np.random.default_rng(seed)
    q = rand_bf16(rng, (G, d))
    K = rand_bf16(rng, (n, d))
    V = rand_bf16(rng, (n, d), loc=loc)
    pi = rng.uniform(0.05, 1.0, n).astype(np.float32)
    pi[:8] = 1.0
    return q, K, V, pi


def test_value_translation_invariance():
    q, K, V, pi = _case(3)
    # adding 1.0 in bf16 is exact for values whose magnitude is < 2^6 with <= 7 mantissa bits
    # -- use a power-of-two-aligned shift on values rounded to a coarse grid instead
    Vf = np.round(bf16_to_f64(V) * 4) / 4
    Vb = to_bf16_bits(Vf)
    Vs = to_bf16_bits(Vf + 3.0)
    assert np.array_equal(bf16_to_f64(Vs), Vf + 3.0)
    a = oracle.attend_certify(q, K, Vb, pi)
    b = oracle.attend_certify(q, K, Vs, pi)
    np.testing.assert_allclose(b["y"], a["y"] + 3.0, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(b["vhat"], a["vhat"], rtol=1e-10)
    np.testing.assert_allclose(b["b"], a["b"], rtol=1e-10)
    np.testing.assert_allclose(b["lse"], a["lse"], rtol=1e-14)


def test_value_scaling():
    q, K, V, pi = _case(4, loc=0.5)
    V2 = to_bf16_bits(bf16_to_f64(V) * 2.0)  # exact in bf16
    a = oracle.attend_certify(q, K, V, pi)
    b = oracle.attend_certify(q, K, V2, pi)
    np.testing.assert_allclose(b["y"], 2 * a["y"], rtol=1e-13)
    np.testing.assert_allclose(b["vhat"], 4 * a["vhat"], rtol=1e-12)
    np.testing.assert_allclose(b["b"], 2 * a["b"], rtol=1e-12)
    np.testing.assert_allclose(b["r"], a["r"], rtol=1e-8)


def test_permutation_invariance():
    q, K, V, pi = _case(5)
    perm = np.random.default_rng(0).permutation(len(pi))
    a = oracle.attend_certify(q, K, V, pi)
    b = oracle.attend_certify(q, K[perm], V[perm], pi[perm])
    for key in ("y", "vhat", "b", "r", "lse"):
        np.testing.assert_allclose(b[key], a[key], rtol=1e-11, atol=1e-14)


def test_single_tail_token_vhat_equals_b_squared():
    q, K, V, pi = _case(6, n=50)
    pi[:] = 1.0
    pi[17] = 0.23
    out = oracle.attend_certify(q, K, V, pi)
    assert np.all(out["vhat"] > 0)
    np.testing.assert_allclose(out["vhat"], out["b"] ** 2, rtol=1e-12)
    # with several tail tokens b^2 <= Vhat <= |S cap T| b^2
    pi[30:40] = 0.5
    out = oracle.attend_certify(q, K, V, pi)
    assert np.all(out["b"] ** 2 <= out["vhat"] * (1 + 1e-12))
    assert np.all(out["vhat"] <= 11 * out["b"] ** 2 * (1 + 1e-12))


def test_radius_combines_variance_and_range_terms():
    q, K, V, pi = _case(7, loc=0.3)
    for delta in (0.1, 0.01):
        out = oracle.attend_certify(q, K, V, pi, delta=delta)
        L = np.log(1 / delta)
        ynorm = np.linalg.norm(out["y"], axis=1)
        num = out["r"] * (ynorm + 1e-9)
        # r is increasing in Vhat and b with the empirical-Bernstein weights sqrt(2 L), L
        assert np.all(num >= np.sqrt(2 * out["vhat"] * L) * (1 - 1e-12))
        assert np.all(num >= out["b"] * L * (1 - 1e-12))
    # a smaller delta widens the radius
    r1 = oracle.attend_certify(q, K, V, pi, delta=0.1)["r"]
    r2 = oracle.attend_certify(q, K, V, pi, delta=0.01)["r"]
    assert np.all(r2 > r1)


def test_empty_retained_set():
    rng = np.random.default_rng(8)
    q = rand_bf16(rng, (2, 128))
    out = oracle.attend_certify(q, np.zeros((0, 128), np.uint16), np.zeros((0, 128), np.uint16),
                                np.zeros(0, np.float32))
    assert np.all(out["y"] == 0) and np.all(out["vhat"] == 0) and np.all(out["r"] == 0)
    assert np.all(np.isneginf(out["lse"]))


def _axis_cache(rows, pis, d=128):
    """q = 0 (every a_j = 1) and value rows given by a few leading coordinates (exact in bf16)."""
    n = len(rows)
    q = np.zeros((1, d), np.uint16)
    K = np.zeros((n, d), np.uint16)
    V = np.zeros((n, d))
    for j, r in enumerate(rows):
        V[j, : len(r)] = r
    return q, K, to_bf16_bits(V), np.asarray(pis, np.float32)


@pytest.mark.parametrize("delta", [0.1, 0.01])
def test_radius_hand_worked_one_tail_row(delta):
    # Rows v0 = 4 e0 and v1 = 4 e1 kept with pi = 1, v2 = 0 kept with pi = 1/2; with q = 0 every
    # a_j = 1, so the Hajek weights a/pi are 1, 1, 2 and Nhat = 4 (eq. (3)):
    #   yhat = (v0 + v1 + 2 v2) / 4 = (1, 1),  |yhat| = sqrt(2)
    #   Theorem 2: Vhat = (1 - 1/2) / (1/2)^2 * 1 * |v2 - yhat|^2 / 4^2 = 2 * 2 / 16 = 1/4
    #   eq. (4):   b = sqrt(1 - 1/2) / (1/2) * 1 * |v2 - yhat| / 4 = 1/2
    #              r = (sqrt(2 Vhat L) + b L) / (|yhat| + eps0),  L = ln(1/delta)
    q, K, V, pi = _axis_cache([(4.0, 0.0), (0.0, 4.0), (0.0, 0.0)], [1.0, 1.0, 0.5])
    out = oracle.attend_certify(q, K, V, pi, delta=delta)
    L = np.log(1.0 / delta)
    np.testing.assert_allclose(out["y"][0, :2], [1.0, 1.0], rtol=1e-15)
    np.testing.assert_allclose(out["vhat"][0], 0.25, rtol=1e-14)
    np.testing.assert_allclose(out["b"][0], 0.5, rtol=1e-14)
    r = (np.sqrt(2 * 0.25 * L) + 0.5 * L) / (np.sqrt(2.0) + 1e-9)
    np.testing.assert_allclose(out["r"][0], r, rtol=1e-13)


@pytest.mark.parametrize("delta", [0.1, 0.3])
def test_radius_hand_worked_two_tail_rows(delta):
    # v0 = 4 e0 (pi = 1), v1 = 0 and v2 = 4 e1 (pi = 1/2 each); q = 0, so a/pi = 1, 2, 2 and
    # Nhat = 5: yhat = (4, 8) / 5 = (0.8, 1.6), |yhat|^2 = 3.2;  |v1 - yhat|^2 = 3.2 and
    # |v2 - yhat|^2 = 0.64 + 5.76 = 6.4.  Each tail term carries (1 - pi)/pi^2 / Nhat^2 = 2/25:
    #   Vhat = 2/25 (3.2 + 6.4) = 0.768,  b = sqrt(2/25 * 6.4) = sqrt(0.512)  (the larger term)
    q, K, V, pi = _axis_cache([(4.0, 0.0), (0.0, 0.0), (0.0, 4.0)], [1.0, 0.5, 0.5])
    out = oracle.attend_certify(q, K, V, pi, delta=delta)
    L = np.log(1.0 / delta)
    np.testing.assert_allclose(out["y"][0, :2], [0.8, 1.6], rtol=1e-15)
    np.testing.assert_allclose(out["vhat"][0], 0.768, rtol=1e-14)
    np.testing.assert_allclose(out["b"][0], np.sqrt(0.512), rtol=1e-14)
    r = (np.sqrt(2 * 0.768 * L) + np.sqrt(0.512) * L) / (np.sqrt(3.2) + 1e-9)
    np.testing.assert_allclose(out["r"][0], r, rtol=1e-13)


@pytest.mark.parametrize("delta", [0.1, 0.05])
def test_radius_single_tail_row_closed_form(delta):
    # One retained tail row j: its Hajek weight w_j = (a_j / pi_j) / Nhat is the softmax of the
    # offset logits s - ln pi (torch, fp64), Theorem 2 has the single term (1 - pi_j) w_j^2
    # |v_j - yhat|^2 and the range term is its square root, so eq. (4) reduces to
    #   r = b (sqrt(2 L) + L) / (|yhat| + eps0),  b = sqrt(1 - pi_j) w_j |v_j - yhat|.
    q, K, V, pi = _case(11, G=3, n=64)
    pi[:] = 1.0
    j = 41
    pi[j] = 0.07
    out = oracle.attend_certify(q, K, V, pi, delta=delta)
    s = bf16_to_f64(q) @ bf16_to_f64(K).T / np.sqrt(128) - np.log(pi.astype(np.float64))
    w = torch.softmax(torch.tensor(s), dim=1).numpy()
    y = w @ bf16_to_f64(V)
    b = np.sqrt(1 - np.float64(pi[j])) * w[:, j] * np.linalg.norm(bf16_to_f64(V)[j] - y, axis=1)
    L = np.log(1.0 / delta)
    np.testing.assert_allclose(out["b"], b, rtol=1e-12)
    np.testing.assert_allclose(out["vhat"], b ** 2, rtol=1e-12)
    r = b * (np.sqrt(2 * L) + L) / (np.linalg.norm(y, axis=1) + 1e-9)
    np.testing.assert_allclose(out["r"], r, rtol=1e-12)
