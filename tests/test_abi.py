"""CPU checks of the C ABI: the library loads, exports every declared symbol, and rejects bad
arguments synchronously (before any device work)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ebd.h")


def _declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    names = re.findall(r"^\s*(?:const\s+)?[A-Za-z_][A-Za-z0-9_]*\s*\*?\s*(ebd_[a-z_]+)\s*\(", src,
                       flags=re.M)
    return sorted(set(names))


def test_header_declares_the_boundary():
    names = _declared_functions()
    for fn in ("ebd_evict", "ebd_attend_certify", "ebd_append_certain", "ebd_scores",
               "ebd_block_contributions", "ebd_certificate_step", "ebd_workspace_size",
               "ebd_status_string", "ebd_version", "ebd_timing_enable", "ebd_timing_read"):
        assert fn in names, fn


def test_library_exports_every_declared_symbol():
    import paper_2607_21475_amd as ebd

    lib = ctypes.CDLL(ebd.LIB_PATH)
    for fn in _declared_functions():
        assert hasattr(lib, fn), fn


def test_version_and_status_strings():
    import paper_2607_21475_amd as ebd

    assert ebd.ebd_version().startswith("ebd-gfx950")
    for code in range(5):
        assert isinstance(ebd.ebd_status_string(code), str)
    assert ebd.ebd_status_string(99) == "unknown status"


def _lib():
    import paper_2607_21475_amd as ebd

    return ebd, ebd._lib


FAKE = 0x100000  # aligned, never dereferenced: validation fails before any device access


def _evict_params(ebd, **kw):
    p = ebd.ebd_evict_params()
    p.num_units = kw.get("U", 4)
    p.head_dim = kw.get("d", 128)
    p.max_rows = kw.get("max_rows", 4096)
    p.max_capacity = kw.get("max_capacity", 1024)
    p.seq_off = FAKE
    p.cap_off = FAKE
    p.n_sink, p.n_recent = 4, 64
    p.budget_frac = 0.1
    p.pi_min = kw.get("pi_min", 0.01)
    p.pi_mode = kw.get("pi_mode", 0)
    return p


def _call_evict(lib, p, ws_bytes=1 << 20, ws=FAKE, nulls=()):
    ptrs = [FAKE] * 11
    for i in nulls:
        ptrs[i] = None
    return lib.ebd_evict(ctypes.byref(p), *ptrs[:8], None, None, ptrs[10], ws, ws_bytes, None)


def test_evict_argument_validation():
    ebd, lib = _lib()
    assert lib.ebd_evict(None, *([None] * 11), None, 0, None) == ebd.EBD_ERR_INVALID_ARG
    assert _call_evict(lib, _evict_params(ebd, d=64)) == ebd.EBD_ERR_UNSUPPORTED
    assert _call_evict(lib, _evict_params(ebd, pi_min=0.0)) == ebd.EBD_ERR_INVALID_ARG
    assert _call_evict(lib, _evict_params(ebd, pi_min=1.5)) == ebd.EBD_ERR_INVALID_ARG
    assert _call_evict(lib, _evict_params(ebd, pi_mode=2)) == ebd.EBD_ERR_INVALID_ARG
    assert _call_evict(lib, _evict_params(ebd, U=-1)) == ebd.EBD_ERR_INVALID_ARG
    assert _call_evict(lib, _evict_params(ebd), nulls=(0,)) == ebd.EBD_ERR_INVALID_ARG
    assert _call_evict(lib, _evict_params(ebd), ws_bytes=16) == ebd.EBD_ERR_WORKSPACE
    assert _call_evict(lib, _evict_params(ebd, max_capacity=-1)) == ebd.EBD_ERR_INVALID_ARG
    assert _call_evict(lib, _evict_params(ebd), ws=FAKE + 8) == ebd.EBD_ERR_WORKSPACE
    assert _call_evict(lib, _evict_params(ebd), ws=None) == ebd.EBD_ERR_WORKSPACE
    # misaligned K
    p = _evict_params(ebd)
    assert lib.ebd_evict(ctypes.byref(p), FAKE, FAKE + 2, *([FAKE] * 6), None, None, FAKE, FAKE,
                         1 << 20, None) == ebd.EBD_ERR_INVALID_ARG
    # zero units is a no-op
    assert _call_evict(lib, _evict_params(ebd, U=0)) == ebd.EBD_OK


def test_attend_argument_validation():
    ebd, lib = _lib()

    def params(**kw):
        p = ebd.ebd_attend_params()
        p.num_units = kw.get("U", 4)
        p.group = kw.get("G", 7)
        p.head_dim = kw.get("d", 128)
        p.split_rows = kw.get("split", 0)
        p.max_rows = kw.get("max_rows", 2000)
        p.cap_off = FAKE
        p.delta = kw.get("delta", 0.1)
        p.flags = kw.get("flags", 0)
        return p

    def call(p, ws=FAKE, ws_bytes=1 << 30):
        return lib.ebd_attend_certify(ctypes.byref(p), *([FAKE] * 11), ws, ws_bytes, None)

    assert call(params(d=96)) == ebd.EBD_ERR_UNSUPPORTED
    assert call(params(G=0)) == ebd.EBD_ERR_INVALID_ARG
    assert call(params(split=100)) == ebd.EBD_ERR_INVALID_ARG
    assert call(params(flags=2)) == ebd.EBD_ERR_INVALID_ARG  # only EBD_F_NO_OFFSET is defined
    assert call(params(delta=1.0)) == ebd.EBD_ERR_INVALID_ARG
    assert call(params(), ws_bytes=100) == ebd.EBD_ERR_WORKSPACE
    assert call(params(U=0)) == ebd.EBD_OK
    # at most 4096 splits per unit
    assert call(params(split=16, max_rows=16 * 4097)) == ebd.EBD_ERR_UNSUPPORTED
    assert call(params(split=16, max_rows=16 * 4096), ws_bytes=100) == ebd.EBD_ERR_WORKSPACE


def test_workspace_sizes():
    ebd, lib = _lib()
    p = _evict_params(ebd, U=1792, max_rows=6144)
    n = ebd.ebd_workspace_size(ebd.EBD_WS_EVICT, p)
    assert n == 256  # reserved: the sampler's launches share only the index list they write
    a = ebd.ebd_attend_params()
    a.num_units, a.group, a.head_dim, a.max_rows, a.cap_off = 1792, 7, 128, 1856, FAKE
    a.delta = 0.1
    m = ebd.ebd_workspace_size(ebd.EBD_WS_ATTEND, a)

    def rec(split_rows):  # floats per record: sums, o, Cv, pivot list, one block per 512-row chunk
        return 264 + 28 + 56 * ((split_rows + 511) // 512)

    def counts(U, G):  # two counts per (unit, block of 8 query heads), 256-byte padded
        return (8 * U * ((G + 7) // 8) + 255) // 256 * 256

    # 1792 units fill the chip: one split each, finalized in the split kernel (no records)
    assert m == counts(1792, 7)
    a.num_units, a.max_rows = 8, 1024
    assert ebd.ebd_workspace_size(ebd.EBD_WS_ATTEND, a) == counts(8, 7) + 8 * 4 * 7 * rec(256) * 4
    a.num_units, a.max_rows = 1024, 13760
    assert ebd.ebd_workspace_size(ebd.EBD_WS_ATTEND, a) == counts(1024, 7) + 1024 * 4 * 7 * rec(3440) * 4
    a.split_rows = 48
    assert ebd.ebd_workspace_size(ebd.EBD_WS_ATTEND, a) == counts(1024, 7) + 1024 * 287 * 7 * rec(48) * 4
    a.group = 12  # two head blocks
    assert ebd.ebd_workspace_size(ebd.EBD_WS_ATTEND, a) == counts(1024, 12) + 1024 * 287 * 12 * rec(48) * 4
    # 1024 units: two splits of up to 8192 rows make one generation of 2048 resident waves when
    # their LDS allows (G = 4); with G = 7 three would be needed, so 4096-row splits stay
    a.split_rows, a.group, a.max_rows = 0, 4, 14048
    assert ebd.ebd_workspace_size(ebd.EBD_WS_ATTEND, a) == counts(1024, 4) + 1024 * 2 * 4 * rec(7024) * 4
    a.num_units = 1025  # 2050 waves: more than one generation either way
    assert ebd.ebd_workspace_size(ebd.EBD_WS_ATTEND, a) == counts(1025, 4) + 1025 * 4 * 4 * rec(3512) * 4
    a.num_units = 1024
    # many units of up to 8192 rows stay one split while its LDS allows two waves per SIMD
    a.split_rows, a.group, a.num_units, a.max_rows = 0, 4, 8192, 4720
    assert ebd.ebd_workspace_size(ebd.EBD_WS_ATTEND, a) == counts(8192, 4)
    a.group = 8  # 8 heads: chunk blocks and finalize LDS exceed 20 KB, cut into 4096-row splits
    assert ebd.ebd_workspace_size(ebd.EBD_WS_ATTEND, a) == counts(8192, 8) + 8192 * 2 * 8 * rec(2368) * 4
    for bad in (40, 8208):  # not a multiple of 16; longer than a wave's candidate store
        a.split_rows = bad
        assert lib.ebd_workspace_size(ebd.EBD_WS_ATTEND, ctypes.byref(a)) == 0
    assert lib.ebd_workspace_size(7, ctypes.byref(a)) == 0


def test_scores_argument_validation_and_workspace():
    ebd, lib = _lib()

    def params(**kw):
        p = ebd.ebd_scores_params()
        p.num_units = kw.get("U", 4)
        p.head_dim = kw.get("d", 128)
        p.num_queries = kw.get("W", 32)
        p.split_rows = kw.get("split", 0)
        p.max_rows = kw.get("max_rows", 6144)
        p.seq_off = FAKE
        p.flags = kw.get("flags", 0)
        return p

    def call(p, ws=FAKE, ws_bytes=1 << 30):
        return lib.ebd_scores(ctypes.byref(p), FAKE, FAKE, FAKE, ws, ws_bytes, None)

    assert call(params(d=64)) == ebd.EBD_ERR_UNSUPPORTED
    for bad in (dict(W=0), dict(W=65), dict(split=40), dict(split=65552), dict(flags=2),
                dict(U=-1), dict(max_rows=-1)):
        assert call(params(**bad)) == ebd.EBD_ERR_INVALID_ARG, bad
    assert call(params(), ws_bytes=64) == ebd.EBD_ERR_WORKSPACE
    assert call(params(), ws=FAKE + 16) == ebd.EBD_ERR_WORKSPACE
    assert call(params(U=0)) == ebd.EBD_OK
    assert lib.ebd_scores(None, FAKE, FAKE, FAKE, FAKE, 1 << 20, None) == ebd.EBD_ERR_INVALID_ARG

    def ws(U, nsplit, W):  # (max, exp-sum) per (unit, split, query), 256-byte padded
        return (8 * U * nsplit * W + 255) // 256 * 256

    p = params(U=1792, W=32, max_rows=6144)  # enough units: one split each
    assert lib.ebd_workspace_size(ebd.EBD_WS_SCORES, ctypes.byref(p)) == ws(1792, 1, 32)
    p = params(U=1024, W=64, max_rows=131072)  # long units: splits of at most 8192 rows
    assert lib.ebd_workspace_size(ebd.EBD_WS_SCORES, ctypes.byref(p)) == ws(1024, 16, 64)
    p = params(U=8, W=7, max_rows=4096)  # few units: 256-row splits
    assert lib.ebd_workspace_size(ebd.EBD_WS_SCORES, ctypes.byref(p)) == ws(8, 16, 7)
    p = params(U=8, W=7, max_rows=4096, split=48)
    assert lib.ebd_workspace_size(ebd.EBD_WS_SCORES, ctypes.byref(p)) == ws(8, 86, 7)


def test_finegrain_argument_validation():
    ebd, lib = _lib()

    def bp(**kw):
        p = ebd.ebd_blocks_params()
        p.num_units, p.group, p.head_dim = kw.get("U", 4), kw.get("G", 7), kw.get("d", 128)
        p.block_rows, p.nblocks = kw.get("rows", 64), kw.get("nb", 96)
        p.max_rows = kw.get("max_rows", 4096)
        p.cap_off = FAKE
        return p

    def call(p):
        return lib.ebd_block_contributions(ctypes.byref(p), *([FAKE] * 9), FAKE, None)

    assert call(bp(d=64)) == ebd.EBD_ERR_UNSUPPORTED
    for bad in (dict(G=0), dict(rows=0), dict(nb=0), dict(nb=8193), dict(U=-1)):
        assert call(bp(**bad)) == ebd.EBD_ERR_INVALID_ARG, bad
    # a unit's rows are addressed as 256-byte rows through 32-bit buffer ranges: 2^24 rows would
    # wrap the range to 0, so the largest accepted unit is 2^24 - 1 rows
    assert call(bp(max_rows=(1 << 24) + 1)) == ebd.EBD_ERR_UNSUPPORTED
    assert call(bp(max_rows=1 << 24)) == ebd.EBD_ERR_UNSUPPORTED
    assert call(bp(max_rows=(1 << 24) - 1, nb=0)) == ebd.EBD_ERR_INVALID_ARG  # size itself accepted
    assert call(bp(U=0)) == ebd.EBD_OK
    c = ebd.ebd_cert_params()
    c.num_units, c.group, c.num_seqs, c.head_stride, c.unit_seq = 4, 7, 2, 0, FAKE
    assert lib.ebd_certificate_step(ctypes.byref(c), FAKE, FAKE, None, None) == ebd.EBD_ERR_INVALID_ARG
    c.head_stride = 4
    assert lib.ebd_certificate_step(ctypes.byref(c), FAKE, None, None, None) == ebd.EBD_ERR_INVALID_ARG
    c.num_units, c.group = 1 << 28, 8  # U G >= 2^31
    assert lib.ebd_certificate_step(ctypes.byref(c), FAKE, FAKE, None, None) == ebd.EBD_ERR_INVALID_ARG
    c.num_units, c.group = 4, 7
    c.num_seqs = 0
    assert lib.ebd_certificate_step(ctypes.byref(c), FAKE, FAKE, None, None) == ebd.EBD_OK


def test_binding_requires_gpu_tensors():
    torch = pytest.importorskip("torch")
    ebd, lib = _lib()
    with pytest.raises(ValueError):
        ebd._ptr(torch.zeros(4), torch.float32, "x")


def test_no_oracle_in_product_path():
    """The package never imports or loads the oracle (test infrastructure only)."""
    pkg = os.path.join(ROOT, "paper_2607_21475_amd")
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".hip", ".cpp", ".hpp", ".h")):
                src = open(os.path.join(dirpath, f)).read()
                assert "oracle" not in src.lower(), f


def test_capacity_plan_covers_floor_and_protected():
    """The planned capacity covers the protected positions plus the expected tail (the budget
    m, or pi_min |T| when the floor exceeds it) with room for its spread."""
    from paper_2607_21475_amd import cache

    # budget below the protected count: the floor alone keeps pi_min of the tail
    c = cache.unit_capacity(300, 0.1, 68, pi_min=0.01)
    assert c >= 68 + 0.01 * 232 + 8 and c % 16 == 0
    c = cache.unit_capacity(300, 0.1, 68, pi_min=0.2)
    assert c >= 68 + 0.2 * 232 + 8 * (0.2 * 232) ** 0.5
    # the usual case: f n + 8 sqrt(m) + 16, rounded up to 16, never above n (+ extra rows)
    c = cache.unit_capacity(6144, 0.25, 68)
    m = 0.25 * 6144 - 68
    assert c == int(-(-(0.25 * 6144 + 8 * (m + 1) ** 0.5 + 16) // 16) * 16)
    assert cache.unit_capacity(100, 1.0, 68, extra=5) == 112  # min(n, ...) + 5, aligned
    assert cache.unit_capacity(0, 0.5, 0, extra=3) == 16
    off = cache.plan_capacity([300, 0, 6144], [0.1, 0.5, 0.25], 4, 64)
    assert off[0] == 0 and off[1] >= 80 and off[2] == off[1] and off[3] > off[2]


def test_noalloc_argument_validation():
    """The entry point without allocation validates like ebd_attend_certify and rejects launches
    whose workspace would exceed its fixed scratch array, before touching the device."""
    ebd, lib = _lib()
    p = ebd.ebd_attend_params()
    p.num_units, p.group, p.head_dim, p.max_rows, p.cap_off, p.delta = 4, 4, 128, 2000, FAKE, 0.1

    def call(p):
        return lib.ebd_attend_certify_noalloc(ctypes.byref(p), *([FAKE] * 11), None)

    assert lib.ebd_attend_certify_noalloc(None, *([FAKE] * 11), None) == ebd.EBD_ERR_INVALID_ARG
    p.head_dim = 64
    assert call(p) == ebd.EBD_ERR_UNSUPPORTED
    p.head_dim, p.group = 128, 0
    assert call(p) == ebd.EBD_ERR_INVALID_ARG
    p.group, p.num_units = 4, 0
    assert call(p) == ebd.EBD_OK
    p.num_units, p.group, p.max_rows, p.split_rows = 200000, 8, 4096, 16
    assert ebd.ebd_workspace_size(ebd.EBD_WS_ATTEND, p) > ebd.EBD_NOALLOC_SCRATCH_BYTES
    assert call(p) == ebd.EBD_ERR_UNSUPPORTED
