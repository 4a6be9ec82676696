"""Host-side planning and allocation around the C ABI (no method arithmetic).

`plan_capacity` sizes each unit's compacted region; `evict` and `attend_certify` allocate the
output tensors and the workspace with torch on the current device and launch the library.
"""
from __future__ import annotations

import math
from dataclasses import dataclass
from typing import Optional, Sequence, Union

import torch

from . import (EBD_F_NO_OFFSET, EBD_WS_ATTEND, EBD_WS_EVICT, EBD_WS_SCORES, HEAD_DIM, attend_params,
               ebd_attend_certify, ebd_evict, ebd_scores, ebd_workspace_size, evict_params,
               scores_params, workspace)


def unit_capacity(n: int, budget_frac: float, n_prot: int, extra: int = 0, align: int = 16,
                  pi_min: float = 0.01) -> int:
    """Rows reserved for one unit's retained set.

    The retained count is |P| plus a sum of independent Bernoullis whose mean is the tail
    budget m = f n - |P|, or pi_min |T| when the floor alone exceeds it, and whose variance is
    at most that mean; mean + 8 sqrt(mean) + 16 rows make an overflow negligible (it is still
    detected and flagged by the kernels).  `extra` reserves rows for appended decode tokens.
    """
    if n <= 0:
        return ((extra + align - 1) // align) * align
    n_tail = max(n - n_prot, 0)
    tail = max(budget_frac * n - n_prot, pi_min * n_tail, 0.0)
    c = n_prot + tail + 8.0 * math.sqrt(tail + 1.0) + 16
    c = min(int(math.ceil(c)), n) + extra
    return ((c + align - 1) // align) * align


def plan_capacity(lengths: Sequence[int], budgets: Union[float, Sequence[float]], n_sink: int,
                  n_recent: int, extra: int = 0, pi_min: float = 0.01):
    """Host list of cap_off [U+1] for the given unit lengths and budget fractions."""
    U = len(lengths)
    if isinstance(budgets, (int, float)):
        budgets = [float(budgets)] * U
    off = [0]
    for n, f in zip(lengths, budgets):
        n_prot = min(int(n), n_sink + n_recent)
        off.append(off[-1] + unit_capacity(int(n), float(f), n_prot, extra, pi_min=pi_min))
    return off


@dataclass
class RetainedCache:
    """Device tensors written by ebd_evict (one compacted region per unit)."""

    Kc: torch.Tensor
    Vc: torch.Tensor
    pic: torch.Tensor
    idxc: torch.Tensor
    count: torch.Tensor
    status: torch.Tensor
    cap_off: torch.Tensor
    max_cap: int
    lam: Optional[torch.Tensor] = None
    pi_full: Optional[torch.Tensor] = None

    @property
    def num_units(self) -> int:
        return self.count.shape[0]


def evict(K: torch.Tensor, V: torch.Tensor, scores: torch.Tensor, seq_off: torch.Tensor,
          lengths: Sequence[int], budget_frac: float = 0.1, budget_per_unit=None,
          n_sink: int = 4, n_recent: int = 64, pi_min: float = 0.01, pi_mode: int = 0,
          seed: int = 0, seed_per_unit=None, epoch: int = 0, extra_rows: int = 0,
          want_pi: bool = False, cap_off_host=None, design: int = 0) -> RetainedCache:
    dev = K.device
    U = len(lengths)
    if cap_off_host is None:
        budgets = budget_frac if budget_per_unit is None else budget_per_unit.tolist()
        cap_off_host = plan_capacity(lengths, budgets, n_sink, n_recent, extra_rows, pi_min)
    caps = [b - a for a, b in zip(cap_off_host[:-1], cap_off_host[1:])]
    rows = cap_off_host[-1]
    cap_off = torch.tensor(cap_off_host, dtype=torch.int64, device=dev)
    out = RetainedCache(
        Kc=torch.empty((max(rows, 1), HEAD_DIM), dtype=torch.bfloat16, device=dev),
        Vc=torch.empty((max(rows, 1), HEAD_DIM), dtype=torch.bfloat16, device=dev),
        pic=torch.empty((max(rows, 1),), dtype=torch.float32, device=dev),
        idxc=torch.empty((max(rows, 1),), dtype=torch.int32, device=dev),
        count=torch.empty((U,), dtype=torch.int32, device=dev),
        status=torch.empty((U,), dtype=torch.int32, device=dev),
        cap_off=cap_off,
        max_cap=max(caps) if caps else 0,
        lam=torch.empty((U,), dtype=torch.float32, device=dev),
        pi_full=torch.empty((max(K.shape[0], 1),), dtype=torch.float32, device=dev) if want_pi else None,
    )
    p = evict_params(U, max(lengths) if lengths else 0, out.max_cap, seq_off, cap_off, n_sink,
                     n_recent, budget_frac, budget_per_unit, pi_min, pi_mode, seed, seed_per_unit,
                     epoch, design)
    ws = workspace(ebd_workspace_size(EBD_WS_EVICT, p), dev)
    ebd_evict(p, scores, K, V, out.Kc, out.Vc, out.pic, out.idxc, out.count, out.status, ws,
              lambda_out=out.lam, pi_full=out.pi_full)
    out._ws = ws  # keep the workspace alive until the launch has run
    return out


def attend_certify(cache: RetainedCache, q: torch.Tensor, split_rows: int = 0, delta: float = 0.1,
                   eps0: float = 1e-9, scale: float = 0.0, ws: Optional[torch.Tensor] = None,
                   offset: bool = True):
    """Outputs y [U, G, 128], vhat, lse, b, r [U, G] (fp32) and the workspace used."""
    U, G, _ = q.shape
    dev = q.device
    p = attend_params(U, G, cache.max_cap, cache.cap_off, split_rows, scale, delta, eps0,
                      0 if offset else EBD_F_NO_OFFSET)
    need = ebd_workspace_size(EBD_WS_ATTEND, p)
    if ws is None or ws.numel() < need:
        ws = workspace(need, dev)
    y = torch.empty((U, G, HEAD_DIM), dtype=torch.float32, device=dev)
    vhat = torch.empty((U, G), dtype=torch.float32, device=dev)
    lse = torch.empty((U, G), dtype=torch.float32, device=dev)
    b = torch.empty((U, G), dtype=torch.float32, device=dev)
    r = torch.empty((U, G), dtype=torch.float32, device=dev)
    st = torch.empty((U,), dtype=torch.int32, device=dev)
    ebd_attend_certify(p, q, cache.Kc, cache.Vc, cache.pic, cache.count, y, vhat, lse, ws,
                       brange=b, radius=r, status=st)
    return {"y": y, "vhat": vhat, "lse": lse, "b": b, "r": r, "status": st, "ws": ws}


def importance_scores(K: torch.Tensor, seq_off: torch.Tensor, q: torch.Tensor, max_rows: int,
                      qpos: Optional[torch.Tensor] = None, scores: Optional[torch.Tensor] = None,
                      accumulate: bool = False, split_rows: int = 0, scale: float = 0.0,
                      ws: Optional[torch.Tensor] = None):
    """Attention mass each cached key receives from the queries q [U, W, 128] (W <= 64 per
    call; more queries: further calls with accumulate=True).  Returns (scores fp32, workspace)."""
    U, W, _ = q.shape
    dev = K.device
    p = scores_params(U, W, max_rows, seq_off, qpos, split_rows, scale, accumulate)
    need = ebd_workspace_size(EBD_WS_SCORES, p)
    if ws is None or ws.numel() < need:
        ws = workspace(need, dev)
    if scores is None:
        scores = torch.empty((max(K.shape[0], 1),), dtype=torch.float32, device=dev)
    ebd_scores(p, q, K, scores, ws)
    return scores, ws


def _diag(ws: torch.Tensor, num_units: int, group: int) -> torch.Tensor:
    nhb = (int(group) + 7) // 8
    return ws[: 8 * num_units * nhb].view(torch.int32).view(num_units * nhb, 2)


def rescans(ws: torch.Tensor, num_units: int, group: int) -> int:
    """512-row chunks the last ebd_attend_certify on `ws` rescanned for the exact range term
    (the workspace starts with two counts per unit and block of 8 query heads)."""
    return int(_diag(ws, num_units, group)[:, 0].sum().item())


def direct_variances(ws: torch.Tensor, num_units: int, group: int) -> int:
    """Query heads whose Vhat the last ebd_attend_certify on `ws` summed directly because the
    one-pass expansion cancelled."""
    return int(_diag(ws, num_units, group)[:, 1].sum().item())


def uses_split_records(ws_bytes: int, num_units: int, group: int) -> bool:
    """Whether an attention launch planned with this workspace size cuts units into several
    splits whose partial records go through the workspace (otherwise it holds only the
    diagnostic counts)."""
    nhb = (int(group) + 7) // 8
    return ws_bytes > (8 * num_units * nhb + 255) // 256 * 256
