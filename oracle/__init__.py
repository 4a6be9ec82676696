"""fp64 CPU oracle for the eviction-by-design hot path -- TEST INFRASTRUCTURE ONLY.

Only the test suite, ``__graft_entry__.smoke()`` and the benchmark's CPU-baseline
leg may import this package.  The product path (the HIP library and its Python
binding) never imports it and shares no code with it.

The arithmetic lives in ``ebd_oracle.c`` (plain C, fp64), written from the paper:
  Sec. 3.1 eq. (1) full attention; Sec. 3.3 eq. (2) inclusion probabilities,
  certainty set and Poisson tail; eq. (3) Hajek estimator; Theorem 2 variance
  estimator; Sec. 3.4 eq. (4) radius; App. "Experimental details" importance
  scores from accumulated attention.  This module only marshals numpy arrays.

bf16 tensors are passed as their raw uint16 bit patterns.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "ebd_oracle.c")
_LIB_PATH = os.path.join(_HERE, "libebd_oracle.so")
_lib = None

ST_CAP_OVERFLOW = 1
ST_BUDGET_FLOOR = 2
ST_NO_EVICTION = 4
ST_BAD_SCORE = 8

DESIGN_POISSON = 0
DESIGN_SYSTEMATIC = 1
DESIGN_TOPK = 2
DESIGN_UNIFORM = 3


def build(force: bool = True) -> str:
    """Compile ebd_oracle.c with gcc into libebd_oracle.so (no fast-math)."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-std=c11", "-O2", "-fPIC", "-shared", "-fopenmp", "-ffp-contract=off",
               "-Wall", "-Wextra", "-o", tmp, _SRC, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC):
        build(force=True)
    lib = ctypes.CDLL(_LIB_PATH)
    P = ctypes.c_void_p
    i32, i64, u32, u64, f64 = (ctypes.c_int32, ctypes.c_int64, ctypes.c_uint32,
                               ctypes.c_uint64, ctypes.c_double)
    lib.ebd_ref_philox4x32_10.argtypes = [P, P, P]
    lib.ebd_ref_philox4x32_10.restype = None
    lib.ebd_ref_token_word.argtypes = [u64, u32, u32, i64]
    lib.ebd_ref_token_word.restype = u32
    lib.ebd_ref_inclusion_probs.argtypes = [i64, P, i32, i32, f64, f64, ctypes.c_int, P, P]
    lib.ebd_ref_inclusion_probs.restype = u32
    lib.ebd_ref_mask.argtypes = [i64, P, u64, u32, u32, P]
    lib.ebd_ref_mask.restype = i64
    lib.ebd_ref_compact.argtypes = [i64, i32, P, P, P, P, i64, P, P, P, P]
    lib.ebd_ref_compact.restype = i64
    lib.ebd_ref_attend_certify.argtypes = [i32, i32, i64, P, P, P, P, f64, f64, f64, ctypes.c_int,
                                           P, P, P, P, P]
    lib.ebd_ref_attend_certify.restype = None
    lib.ebd_ref_full_attention.argtypes = [i32, i32, i64, P, P, P, f64, P]
    lib.ebd_ref_full_attention.restype = None
    lib.ebd_ref_evict_batch.argtypes = [i32, i32, P, P, P, P, P, i32, i32, f64, P, f64, u64, P, u32,
                                        i32, i32, P, P, P, P, P, P, P, P, P, P, i32]
    lib.ebd_ref_systematic_start.argtypes = [u64, u32, u32]
    lib.ebd_ref_systematic_start.restype = u32
    lib.ebd_ref_mask_systematic.argtypes = [i64, P, u64, u32, u32, P]
    lib.ebd_ref_mask_systematic.restype = i64
    lib.ebd_ref_topk_probs.argtypes = [i64, P, i32, i32, f64, P]
    lib.ebd_ref_topk_probs.restype = u32
    lib.ebd_ref_evict_batch.restype = None
    lib.ebd_ref_attend_batch.argtypes = [i32, i32, i32, P, P, P, P, P, P, f64, f64, f64, i32,
                                         P, P, P, P, P, i32]
    lib.ebd_ref_attend_batch.restype = None
    lib.ebd_ref_full_batch.argtypes = [i32, i32, i32, P, P, P, P, f64, P, i32]
    lib.ebd_ref_full_batch.restype = None
    lib.ebd_ref_window_scores.argtypes = [i64, i32, i32, P, P, P, f64, P]
    lib.ebd_ref_window_scores.restype = None
    lib.ebd_ref_window_scores_batch.argtypes = [i32, i32, i32, P, P, P, P, f64, P, i32]
    lib.ebd_ref_window_scores_batch.restype = None
    lib.ebd_ref_block_contributions.argtypes = [i32, i32, i64, P, P, P, P, P, P, P, f64, i32, i64, P]
    lib.ebd_ref_block_contributions.restype = None
    lib.ebd_ref_certificate_step.argtypes = [i32, i32, i32, i32, P, P, P, P, P]
    lib.ebd_ref_certificate_step.restype = None
    lib.ebd_ref_max_threads.argtypes = []
    lib.ebd_ref_max_threads.restype = i32
    _lib = lib
    return lib


def _p(a):
    return None if a is None else ctypes.c_void_p(a.ctypes.data)


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


def max_threads() -> int:
    return int(_load().ebd_ref_max_threads())


# --------------------------------------------------------------------------
# Philox4x32-10 (Salmon et al., SC 2011)
# --------------------------------------------------------------------------
def philox4x32_10(ctr, key):
    c = _c(ctr, np.uint32)
    k = _c(key, np.uint32)
    out = np.zeros(4, np.uint32)
    _load().ebd_ref_philox4x32_10(_p(c), _p(k), _p(out))
    return out


def token_word(seed: int, unit: int, epoch: int, i: int) -> int:
    return int(_load().ebd_ref_token_word(seed, unit, epoch, i))


# --------------------------------------------------------------------------
# Sampler pieces for one unit (Sec. 3.3)
# --------------------------------------------------------------------------
def inclusion_probs(scores, n_sink, n_recent, budget_frac, pi_min, pi_mode=0):
    """Returns (pi fp64 [n], lambda, status)."""
    s = _c(scores, np.float32)
    n = s.shape[0]
    pi = np.zeros(max(n, 1), np.float64)
    lam = ctypes.c_double(0.0)
    st = _load().ebd_ref_inclusion_probs(n, _p(s), n_sink, n_recent, float(budget_frac),
                                         float(pi_min), int(pi_mode), ctypes.byref(lam), _p(pi))
    return pi[:n], lam.value, int(st)


def mask(pi32, seed, unit, epoch=0):
    p = _c(pi32, np.float32)
    m = np.zeros(max(p.shape[0], 1), np.uint8)
    _load().ebd_ref_mask(p.shape[0], _p(p), int(seed), int(unit), int(epoch), _p(m))
    return m[: p.shape[0]]


def systematic_start(seed: int, unit: int, epoch: int = 0) -> int:
    return int(_load().ebd_ref_systematic_start(seed, unit, epoch))


def mask_systematic(pi32, seed, unit, epoch=0):
    """Fixed-size systematic design at the stored pi (one start per unit)."""
    p = _c(pi32, np.float32)
    m = np.zeros(max(p.shape[0], 1), np.uint8)
    _load().ebd_ref_mask_systematic(p.shape[0], _p(p), seed, unit, epoch, _p(m))
    return m[: p.shape[0]]


def topk_probs(scores, n_sink, n_recent, budget_frac):
    """Deterministic top-k comparison design: pi in {0, 1}; returns (pi, status)."""
    s = _c(scores, np.float32)
    n = s.shape[0]
    pi = np.zeros(max(n, 1), np.float64)
    st = _load().ebd_ref_topk_probs(n, _p(s), n_sink, n_recent, float(budget_frac), _p(pi))
    return pi[:n], int(st)


def compact(msk, pi32, K, V, cap=None):
    """Stable compaction. K, V uint16 [n, d]. Returns (Kc, Vc, pic, idx, count)."""
    msk = _c(msk, np.uint8)
    p = _c(pi32, np.float32)
    K = _c(K, np.uint16)
    V = _c(V, np.uint16)
    n, d = K.shape
    if cap is None:
        cap = n
    Kc = np.zeros((max(cap, 1), d), np.uint16)
    Vc = np.zeros((max(cap, 1), d), np.uint16)
    pic = np.zeros(max(cap, 1), np.float32)
    idx = np.zeros(max(cap, 1), np.int32)
    cnt = _load().ebd_ref_compact(n, d, _p(msk), _p(p), _p(K), _p(V), cap, _p(Kc), _p(Vc),
                                  _p(pic), _p(idx))
    k = min(cnt, cap)
    return Kc[:k], Vc[:k], pic[:k], idx[:k], int(cnt)


def attend_certify(q, Kc, Vc, pic, scale=None, delta=0.1, eps0=1e-9, use_offset=True):
    """Hajek output + certificate for one unit. q uint16 [G, d]. Returns dict of fp64 arrays."""
    q = _c(q, np.uint16)
    if q.ndim == 1:
        q = q[None, :]
    G, d = q.shape
    Kc = _c(Kc, np.uint16).reshape(-1, d)
    Vc = _c(Vc, np.uint16).reshape(-1, d)
    pic = _c(pic, np.float32)
    count = Kc.shape[0]
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    y = np.zeros((G, d), np.float64)
    vhat = np.zeros(G, np.float64)
    lse = np.zeros(G, np.float64)
    b = np.zeros(G, np.float64)
    r = np.zeros(G, np.float64)
    _load().ebd_ref_attend_certify(G, d, count, _p(q), _p(Kc), _p(Vc), _p(pic), float(scale),
                                   float(delta), float(eps0), int(bool(use_offset)), _p(y),
                                   _p(vhat), _p(lse), _p(b), _p(r))
    return {"y": y, "vhat": vhat, "lse": lse, "b": b, "r": r}


def full_attention(q, K, V, scale=None):
    q = _c(q, np.uint16)
    if q.ndim == 1:
        q = q[None, :]
    G, d = q.shape
    K = _c(K, np.uint16).reshape(-1, d)
    V = _c(V, np.uint16).reshape(-1, d)
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    y = np.zeros((G, d), np.float64)
    _load().ebd_ref_full_attention(G, d, K.shape[0], _p(q), _p(K), _p(V), float(scale), _p(y))
    return y


# --------------------------------------------------------------------------
# Batched drivers (units split across host threads)
# --------------------------------------------------------------------------
def evict_batch(seq_off, cap_off, scores, K, V, n_sink, n_recent, budget_frac=0.1,
                budget_per_unit=None, pi_min=0.01, seed=0, seed_per_unit=None, epoch=0,
                pi_mode=0, pi_given=None, design=0, nthreads=0, unit_ids=None):
    seq_off = _c(seq_off, np.int64)
    cap_off = _c(cap_off, np.int64)
    U = seq_off.shape[0] - 1
    scores = _c(scores, np.float32)
    K = _c(K, np.uint16)
    V = _c(V, np.uint16)
    d = K.shape[-1]
    rows = int(seq_off[-1])
    crow = int(cap_off[-1])
    bpu = None if budget_per_unit is None else _c(budget_per_unit, np.float32)
    spu = None if seed_per_unit is None else _c(seed_per_unit, np.uint64)
    pg = None if pi_given is None else _c(pi_given, np.float32)
    uid = None if unit_ids is None else _c(unit_ids, np.uint32)
    out = {
        "Kc": np.zeros((max(crow, 1), d), np.uint16),
        "Vc": np.zeros((max(crow, 1), d), np.uint16),
        "pic": np.zeros(max(crow, 1), np.float32),
        "idx": np.full(max(crow, 1), -1, np.int32),
        "count": np.zeros(U, np.int32),
        "lambda": np.zeros(U, np.float64),
        "pi_full": np.zeros(max(rows, 1), np.float32),
        "status": np.zeros(U, np.uint32),
    }
    _load().ebd_ref_evict_batch(U, d, _p(seq_off), _p(cap_off), _p(scores), _p(K), _p(V), n_sink,
                                n_recent, float(budget_frac), _p(bpu), float(pi_min), int(seed),
                                _p(spu), int(epoch), int(pi_mode), int(design), _p(pg), _p(uid),
                                _p(out["Kc"]),
                                _p(out["Vc"]), _p(out["pic"]), _p(out["idx"]), _p(out["count"]),
                                _p(out["lambda"]), _p(out["pi_full"]), _p(out["status"]),
                                int(nthreads))
    out["Kc"] = out["Kc"][:crow]
    out["Vc"] = out["Vc"][:crow]
    out["pic"] = out["pic"][:crow]
    out["idx"] = out["idx"][:crow]
    out["pi_full"] = out["pi_full"][:rows]
    return out


def attend_batch(cap_off, count, q, Kc, Vc, pic, scale=None, delta=0.1, eps0=1e-9,
                 use_offset=True, nthreads=0):
    cap_off = _c(cap_off, np.int64)
    count = _c(count, np.int32)
    q = _c(q, np.uint16)
    U, G, d = q.shape
    Kc = _c(Kc, np.uint16)
    Vc = _c(Vc, np.uint16)
    pic = _c(pic, np.float32)
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    out = {
        "y": np.zeros((U, G, d), np.float64),
        "vhat": np.zeros((U, G), np.float64),
        "lse": np.zeros((U, G), np.float64),
        "b": np.zeros((U, G), np.float64),
        "r": np.zeros((U, G), np.float64),
    }
    _load().ebd_ref_attend_batch(U, G, d, _p(cap_off), _p(count), _p(q), _p(Kc), _p(Vc), _p(pic),
                                 float(scale), float(delta), float(eps0), int(bool(use_offset)),
                                 _p(out["y"]), _p(out["vhat"]), _p(out["lse"]), _p(out["b"]),
                                 _p(out["r"]), int(nthreads))
    return out


def full_batch(seq_off, q, K, V, scale=None, nthreads=0):
    seq_off = _c(seq_off, np.int64)
    q = _c(q, np.uint16)
    U, G, d = q.shape
    K = _c(K, np.uint16)
    V = _c(V, np.uint16)
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    y = np.zeros((U, G, d), np.float64)
    _load().ebd_ref_full_batch(U, G, d, _p(seq_off), _p(q), _p(K), _p(V), float(scale), _p(y),
                               int(nthreads))
    return y


# --------------------------------------------------------------------------
# Importance scores (App. "Experimental details", Harness)
# --------------------------------------------------------------------------
def window_scores(K, Q, qpos=None, scale=None):
    """score_i = sum_w softmax_w(scale q_w . k)_i over the keys query w sees (0..qpos[w], or all
    when qpos is None).  K [n, d], Q [W, d] bf16 bits; returns float64 [n]."""
    Q = _c(Q, np.uint16)
    if Q.ndim == 1:
        Q = Q[None, :]
    W, d = Q.shape
    K = _c(K, np.uint16).reshape(-1, d)
    n = K.shape[0]
    qp = None if qpos is None else _c(qpos, np.int32)
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    out = np.zeros(n, np.float64)
    _load().ebd_ref_window_scores(n, d, W, _p(K), _p(Q), _p(qp), float(scale), _p(out))
    return out


def window_scores_batch(seq_off, K, Q, qpos=None, scale=None, nthreads=0):
    """Scores of U units: seq_off [U+1], K [rows, d], Q [U, W, d], qpos [U, W] or None."""
    off = _c(seq_off, np.int64)
    U = off.shape[0] - 1
    Q = _c(Q, np.uint16)
    W, d = Q.shape[1], Q.shape[2]
    K = _c(K, np.uint16).reshape(-1, d)
    qp = None if qpos is None else _c(qpos, np.int32)
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    out = np.zeros(int(off[-1]), np.float64)
    _load().ebd_ref_window_scores_batch(U, d, W, _p(off), _p(K), _p(Q), _p(qp), float(scale),
                                        _p(out), int(nthreads))
    return out


# --------------------------------------------------------------------------
# Fine-grained attribution and the deployed certificate (Sec. 6; App. details)
# --------------------------------------------------------------------------
def block_contributions(q, Kc, Vc, pic, idx, yhat, lse, nblocks, block_rows=64, scale=None):
    """Sum over heads and over retained tokens in each block of original positions of the
    Theorem 2 summand (1-pi)/pi^2 a^2 |v - yhat|^2 / Nhat^2.  q [G, d]; yhat [G, d]; lse [G]."""
    q = _c(q, np.uint16)
    if q.ndim == 1:
        q = q[None, :]
    G, d = q.shape
    Kc = _c(Kc, np.uint16).reshape(-1, d)
    Vc = _c(Vc, np.uint16).reshape(-1, d)
    count = Kc.shape[0]
    pic = _c(pic, np.float32)
    idx = _c(idx, np.int32)
    yh = _c(yhat, np.float64).reshape(G, d)
    ls = _c(lse, np.float64).reshape(G)
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    out = np.zeros(max(int(nblocks), 1), np.float64)
    _load().ebd_ref_block_contributions(G, d, count, _p(q), _p(Kc), _p(Vc), _p(pic), _p(idx),
                                        _p(yh), _p(ls), float(scale), int(block_rows),
                                        int(nblocks), _p(out))
    return out[: int(nblocks)]


def certificate_step(radius, unit_seq, num_seqs, head_stride=4, unit_head0=None, cert=None):
    """Mean radius over the sampled (unit, head) pairs per sequence, folded into the running
    maximum `cert` (returned with the means)."""
    r = _c(radius, np.float32)
    U, G = r.shape
    us = _c(unit_seq, np.int32)
    h0 = None if unit_head0 is None else _c(unit_head0, np.int32)
    c = np.zeros(num_seqs, np.float64) if cert is None else _c(cert, np.float64).copy()
    mean = np.zeros(num_seqs, np.float64)
    _load().ebd_ref_certificate_step(U, G, num_seqs, head_stride, _p(us), _p(h0), _p(r), _p(c),
                                     _p(mean))
    return c, mean
