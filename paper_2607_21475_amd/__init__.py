"""Python binding of libebd (gfx950): argument marshalling only.

Every step of the eviction-by-design path runs in the library's HIP kernels.  This module
converts torch tensors to device pointers, passes torch's current HIP stream, and raises on
error statuses.  The functions carry the C names:

    ebd_evict            Poisson tail sampler (Sec. 3.3, eq. (2); Sec. 3.1)
    ebd_attend_certify   Hajek decode attention + Theorem 2 variance + eq. (4) radius
    ebd_append_certain   append a decode token with pi = 1
    ebd_workspace_size, ebd_status_string, ebd_version, ebd_timing_enable, ebd_timing_read

The library must be built (``python paper_2607_21475_amd/build.py``); importing this package
without it raises, and there is no other implementation to fall back to.
"""
from __future__ import annotations

import ctypes
import os

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libebd.so")

if not os.path.exists(LIB_PATH):
    raise ImportError("libebd.so is not built (run python paper_2607_21475_amd/build.py); "
                      "the EBD path has no fallback")
_lib = ctypes.CDLL(LIB_PATH)

EBD_OK = 0
EBD_ERR_INVALID_ARG = 1
EBD_ERR_UNSUPPORTED = 2
EBD_ERR_WORKSPACE = 3
EBD_ERR_HIP = 4

EBD_ST_CAP_OVERFLOW = 1
EBD_ST_BUDGET_FLOOR = 2
EBD_ST_NO_EVICTION = 4
EBD_ST_BAD_SCORE = 8
EBD_ST_BAD_LAYOUT = 16

EBD_DESIGN_POISSON = 0
EBD_DESIGN_SYSTEMATIC = 1
EBD_DESIGN_TOPK = 2
EBD_DESIGN_UNIFORM = 3

EBD_F_NO_OFFSET = 1

EBD_WS_EVICT = 0
EBD_WS_ATTEND = 1
EBD_WS_SCORES = 2
EBD_SCORES_ACCUMULATE = 1
EBD_NOALLOC_SCRATCH_BYTES = 64 << 20

HEAD_DIM = 128


class ebd_evict_params(ctypes.Structure):
    _fields_ = [
        ("num_units", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("max_rows", ctypes.c_int64),
        ("max_capacity", ctypes.c_int64),
        ("seq_off", ctypes.c_void_p),
        ("cap_off", ctypes.c_void_p),
        ("n_sink", ctypes.c_int32),
        ("n_recent", ctypes.c_int32),
        ("budget_frac", ctypes.c_float),
        ("budget_per_unit", ctypes.c_void_p),
        ("pi_min", ctypes.c_float),
        ("pi_mode", ctypes.c_int32),
        ("seed", ctypes.c_uint64),
        ("seed_per_unit", ctypes.c_void_p),
        ("epoch", ctypes.c_uint32),
        ("design", ctypes.c_int32),
    ]


class ebd_attend_params(ctypes.Structure):
    _fields_ = [
        ("num_units", ctypes.c_int32),
        ("group", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("split_rows", ctypes.c_int32),
        ("max_rows", ctypes.c_int64),
        ("cap_off", ctypes.c_void_p),
        ("scale", ctypes.c_float),
        ("delta", ctypes.c_float),
        ("eps0", ctypes.c_float),
        ("flags", ctypes.c_uint32),
    ]


class ebd_scores_params(ctypes.Structure):
    _fields_ = [
        ("num_units", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("num_queries", ctypes.c_int32),
        ("split_rows", ctypes.c_int32),
        ("max_rows", ctypes.c_int64),
        ("seq_off", ctypes.c_void_p),
        ("qpos", ctypes.c_void_p),
        ("scale", ctypes.c_float),
        ("flags", ctypes.c_uint32),
    ]


class ebd_blocks_params(ctypes.Structure):
    _fields_ = [
        ("num_units", ctypes.c_int32),
        ("group", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("block_rows", ctypes.c_int32),
        ("nblocks", ctypes.c_int64),
        ("max_rows", ctypes.c_int64),
        ("cap_off", ctypes.c_void_p),
        ("scale", ctypes.c_float),
    ]


class ebd_cert_params(ctypes.Structure):
    _fields_ = [
        ("num_units", ctypes.c_int32),
        ("group", ctypes.c_int32),
        ("num_seqs", ctypes.c_int32),
        ("head_stride", ctypes.c_int32),
        ("unit_seq", ctypes.c_void_p),
        ("unit_head0", ctypes.c_void_p),
    ]


_P = ctypes.c_void_p
_lib.ebd_evict.argtypes = [ctypes.POINTER(ebd_evict_params)] + [_P] * 12 + [ctypes.c_size_t, _P]
_lib.ebd_evict.restype = ctypes.c_int
_lib.ebd_attend_certify.argtypes = [ctypes.POINTER(ebd_attend_params)] + [_P] * 12 + \
    [ctypes.c_size_t, _P]
_lib.ebd_attend_certify.restype = ctypes.c_int
_lib.ebd_attend_certify_noalloc.argtypes = [ctypes.POINTER(ebd_attend_params)] + [_P] * 12
_lib.ebd_attend_certify_noalloc.restype = ctypes.c_int
_lib.ebd_scores.argtypes = [ctypes.POINTER(ebd_scores_params)] + [_P] * 4 + [ctypes.c_size_t, _P]
_lib.ebd_scores.restype = ctypes.c_int
_lib.ebd_block_contributions.argtypes = [ctypes.POINTER(ebd_blocks_params)] + [_P] * 10
_lib.ebd_block_contributions.restype = ctypes.c_int
_lib.ebd_certificate_step.argtypes = [ctypes.POINTER(ebd_cert_params)] + [_P] * 4
_lib.ebd_certificate_step.restype = ctypes.c_int
_lib.ebd_append_certain.argtypes = [ctypes.c_int32, ctypes.c_int32] + [_P] * 11
_lib.ebd_append_certain.restype = ctypes.c_int
_lib.ebd_workspace_size.argtypes = [ctypes.c_int32, _P]
_lib.ebd_workspace_size.restype = ctypes.c_size_t
_lib.ebd_status_string.argtypes = [ctypes.c_int]
_lib.ebd_status_string.restype = ctypes.c_char_p
_lib.ebd_version.argtypes = []
_lib.ebd_version.restype = ctypes.c_char_p
_lib.ebd_timing_enable.argtypes = [ctypes.c_int32]
_lib.ebd_timing_enable.restype = ctypes.c_int
_lib.ebd_timing_read.argtypes = [ctypes.c_char_p, ctypes.POINTER(ctypes.c_double),
                                 ctypes.POINTER(ctypes.c_int64)]
_lib.ebd_timing_read.restype = ctypes.c_int


class EbdError(RuntimeError):
    def __init__(self, fn: str, code: int):
        super().__init__("%s failed: %s (%d)" % (fn, ebd_status_string(code), code))
        self.code = code


def _check(fn: str, code: int) -> None:
    if code != EBD_OK:
        raise EbdError(fn, code)


def _ptr(t, dtype=None, name="tensor"):
    """Device pointer of a contiguous CUDA/HIP tensor (None -> NULL)."""
    if t is None:
        return None
    if not isinstance(t, torch.Tensor):
        raise TypeError("%s must be a torch.Tensor" % name)
    if not t.is_cuda:
        raise ValueError("%s must be on the GPU" % name)
    if dtype is not None and t.dtype != dtype:
        raise TypeError("%s must be %s, got %s" % (name, dtype, t.dtype))
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream=None):
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def ebd_status_string(code: int) -> str:
    return _lib.ebd_status_string(int(code)).decode()


def ebd_version() -> str:
    return _lib.ebd_version().decode()


def evict_params(num_units, max_rows, max_capacity, seq_off, cap_off, n_sink=4, n_recent=64,
                 budget_frac=0.1, budget_per_unit=None, pi_min=0.01, pi_mode=0, seed=0,
                 seed_per_unit=None, epoch=0, design=0) -> ebd_evict_params:
    p = ebd_evict_params()
    p.num_units = int(num_units)
    p.head_dim = HEAD_DIM
    p.max_rows = int(max_rows)
    p.max_capacity = int(max_capacity)
    p.seq_off = _ptr(seq_off, torch.int64, "seq_off")
    p.cap_off = _ptr(cap_off, torch.int64, "cap_off")
    p.n_sink = int(n_sink)
    p.n_recent = int(n_recent)
    p.budget_frac = float(budget_frac)
    p.budget_per_unit = _ptr(budget_per_unit, torch.float32, "budget_per_unit")
    p.pi_min = float(pi_min)
    p.pi_mode = int(pi_mode)
    p.seed = int(seed) & 0xFFFFFFFFFFFFFFFF
    p.seed_per_unit = _ptr(seed_per_unit, torch.int64, "seed_per_unit")
    p.epoch = int(epoch) & 0xFFFFFFFF
    p.design = int(design)
    return p


def attend_params(num_units, group, max_rows, cap_off, split_rows=0, scale=0.0, delta=0.1,
                  eps0=1e-9, flags=0) -> ebd_attend_params:
    p = ebd_attend_params()
    p.num_units = int(num_units)
    p.group = int(group)
    p.head_dim = HEAD_DIM
    p.split_rows = int(split_rows)
    p.max_rows = int(max_rows)
    p.cap_off = _ptr(cap_off, torch.int64, "cap_off")
    p.scale = float(scale)
    p.delta = float(delta)
    p.eps0 = float(eps0)
    p.flags = int(flags)
    return p


def scores_params(num_units, num_queries, max_rows, seq_off, qpos=None, split_rows=0, scale=0.0,
                  accumulate=False) -> ebd_scores_params:
    p = ebd_scores_params()
    p.num_units = int(num_units)
    p.head_dim = HEAD_DIM
    p.num_queries = int(num_queries)
    p.split_rows = int(split_rows)
    p.max_rows = int(max_rows)
    p.seq_off = _ptr(seq_off, torch.int64, "seq_off")
    p.qpos = _ptr(qpos, torch.int32, "qpos")
    p.scale = float(scale)
    p.flags = EBD_SCORES_ACCUMULATE if accumulate else 0
    return p


def ebd_workspace_size(which: int, params) -> int:
    n = _lib.ebd_workspace_size(int(which), ctypes.byref(params))
    if n == 0 and params.num_units > 0:
        raise EbdError("ebd_workspace_size", EBD_ERR_INVALID_ARG)
    return int(n)


def ebd_evict(params: ebd_evict_params, scores, K, V, Kc, Vc, pic, idxc, count, status,
              workspace, lambda_out=None, pi_full=None, stream=None) -> None:
    """Launch the sampler (asynchronous on the current stream)."""
    bf = torch.bfloat16
    code = _lib.ebd_evict(ctypes.byref(params), _ptr(scores, torch.float32, "scores"),
                          _ptr(K, bf, "K"), _ptr(V, bf, "V"), _ptr(Kc, bf, "Kc"),
                          _ptr(Vc, bf, "Vc"), _ptr(pic, torch.float32, "pic"),
                          _ptr(idxc, torch.int32, "idxc"), _ptr(count, torch.int32, "count"),
                          _ptr(lambda_out, torch.float32, "lambda_out"),
                          _ptr(pi_full, torch.float32, "pi_full"),
                          _ptr(status, torch.int32, "status"), _ptr(workspace, None, "workspace"),
                          workspace.numel() * workspace.element_size(), _stream(stream))
    _check("ebd_evict", code)


def ebd_attend_certify(params: ebd_attend_params, q, Kc, Vc, pic, count, y, vhat, lse, workspace,
                       brange=None, radius=None, status=None, stream=None) -> None:
    """Launch certified decode attention (asynchronous on the current stream)."""
    bf = torch.bfloat16
    f32 = torch.float32
    code = _lib.ebd_attend_certify(ctypes.byref(params), _ptr(q, bf, "q"), _ptr(Kc, bf, "Kc"),
                                   _ptr(Vc, bf, "Vc"), _ptr(pic, f32, "pic"),
                                   _ptr(count, torch.int32, "count"), _ptr(y, f32, "y"),
                                   _ptr(vhat, f32, "vhat"), _ptr(lse, f32, "lse"),
                                   _ptr(brange, f32, "brange"), _ptr(radius, f32, "radius"),
                                   _ptr(status, torch.int32, "status"),
                                   _ptr(workspace, None, "workspace"),
                                   workspace.numel() * workspace.element_size(), _stream(stream))
    _check("ebd_attend_certify", code)


def ebd_attend_certify_noalloc(params: ebd_attend_params, q, Kc, Vc, pic, count, y, vhat, lse,
                               brange=None, radius=None, status=None, stream=None) -> None:
    """The same step without a workspace argument (the library's fixed per-GPU scratch array)."""
    bf = torch.bfloat16
    f32 = torch.float32
    code = _lib.ebd_attend_certify_noalloc(ctypes.byref(params), _ptr(q, bf, "q"),
                                           _ptr(Kc, bf, "Kc"), _ptr(Vc, bf, "Vc"),
                                           _ptr(pic, f32, "pic"), _ptr(count, torch.int32, "count"),
                                           _ptr(y, f32, "y"), _ptr(vhat, f32, "vhat"),
                                           _ptr(lse, f32, "lse"), _ptr(brange, f32, "brange"),
                                           _ptr(radius, f32, "radius"),
                                           _ptr(status, torch.int32, "status"), _stream(stream))
    _check("ebd_attend_certify_noalloc", code)


def ebd_scores(params: ebd_scores_params, q, K, scores, workspace, stream=None) -> None:
    """Launch the importance-score passes (asynchronous on the current stream)."""
    bf = torch.bfloat16
    code = _lib.ebd_scores(ctypes.byref(params), _ptr(q, bf, "q"), _ptr(K, bf, "K"),
                           _ptr(scores, torch.float32, "scores"), _ptr(workspace, None, "workspace"),
                           workspace.numel() * workspace.element_size(), _stream(stream))
    _check("ebd_scores", code)


def ebd_block_contributions(num_units, group, nblocks, max_rows, cap_off, q, Kc, Vc, pic, idxc,
                            count, y, lse, blocks, block_rows=64, scale=0.0, stream=None) -> None:
    """Per-block variance contributions of the retained rows (asynchronous)."""
    p = ebd_blocks_params()
    p.num_units, p.group, p.head_dim = int(num_units), int(group), HEAD_DIM
    p.block_rows, p.nblocks, p.max_rows = int(block_rows), int(nblocks), int(max_rows)
    p.cap_off = _ptr(cap_off, torch.int64, "cap_off")
    p.scale = float(scale)
    bf, f32 = torch.bfloat16, torch.float32
    code = _lib.ebd_block_contributions(ctypes.byref(p), _ptr(q, bf, "q"), _ptr(Kc, bf, "Kc"),
                                        _ptr(Vc, bf, "Vc"), _ptr(pic, f32, "pic"),
                                        _ptr(idxc, torch.int32, "idxc"),
                                        _ptr(count, torch.int32, "count"), _ptr(y, f32, "y"),
                                        _ptr(lse, f32, "lse"), _ptr(blocks, f32, "blocks"),
                                        _stream(stream))
    _check("ebd_block_contributions", code)


def ebd_certificate_step(num_units, group, num_seqs, unit_seq, radius, cert, mean_out=None,
                         head_stride=4, unit_head0=None, stream=None) -> None:
    """Fold one decode step's mean sampled radius into the running certificate."""
    p = ebd_cert_params()
    p.num_units, p.group, p.num_seqs, p.head_stride = int(num_units), int(group), int(num_seqs), int(head_stride)
    p.unit_seq = _ptr(unit_seq, torch.int32, "unit_seq")
    p.unit_head0 = _ptr(unit_head0, torch.int32, "unit_head0")
    f32 = torch.float32
    code = _lib.ebd_certificate_step(ctypes.byref(p), _ptr(radius, f32, "radius"),
                                     _ptr(cert, f32, "cert"), _ptr(mean_out, f32, "mean_out"),
                                     _stream(stream))
    _check("ebd_certificate_step", code)


def ebd_append_certain(num_units, cap_off, count, k_new, v_new, Kc, Vc, pic, idxc=None,
                       pos_new=None, status=None, stream=None) -> None:
    bf = torch.bfloat16
    code = _lib.ebd_append_certain(int(num_units), HEAD_DIM, _ptr(cap_off, torch.int64, "cap_off"),
                                   _ptr(count, torch.int32, "count"), _ptr(k_new, bf, "k_new"),
                                   _ptr(v_new, bf, "v_new"), _ptr(pos_new, torch.int32, "pos_new"),
                                   _ptr(Kc, bf, "Kc"), _ptr(Vc, bf, "Vc"),
                                   _ptr(pic, torch.float32, "pic"), _ptr(idxc, torch.int32, "idxc"),
                                   _ptr(status, torch.int32, "status"), _stream(stream))
    _check("ebd_append_certain", code)


def ebd_timing_enable(enable: bool) -> None:
    _check("ebd_timing_enable", _lib.ebd_timing_enable(1 if enable else 0))


def ebd_timing_read(name: str):
    """(total milliseconds, launches) of kernel `name` since the last read."""
    ms = ctypes.c_double(0.0)
    n = ctypes.c_int64(0)
    _check("ebd_timing_read", _lib.ebd_timing_read(name.encode(), ctypes.byref(ms), ctypes.byref(n)))
    return ms.value, n.value


def workspace(nbytes: int, device="cuda") -> torch.Tensor:
    """A caller-owned workspace buffer (256-byte aligned by the caching allocator)."""
    return torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=device)
