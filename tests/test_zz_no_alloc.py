"""The attention entry point without allocation (ebd_attend_certify_noalloc), through the C ABI,
against the workspace entry point ebd_attend_certify on the same inputs: two calls in a row, the
second on a smaller input, both with units cut into several splits so that the split records
live in the library's scratch array; then a third whose units' two splits run as the waves of one
work-group (combined in LDS: of the scratch array only the per-unit diagnostic words are used)."""
import numpy as np
import pytest
import torch

import synth

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)


def _both(lengths, G, budget, split, seed):
    import paper_2607_21475_amd as ebd
    from paper_2607_21475_amd import cache

    U = len(lengths)
    K, V, seq_off = synth.make_cache(lengths, seed=seed, device="cuda")
    sc = synth.window_scores(K, seq_off, seed=seed + 1)
    q = synth.make_queries(U, G, seed=seed + 2, device="cuda")
    out = cache.evict(K, V, sc, seq_off, lengths, budget_frac=budget, seed=seed)
    ref = cache.attend_certify(out, q, split_rows=split)
    p = ebd.attend_params(U, G, out.max_cap, out.cap_off, split)
    need = ebd.ebd_workspace_size(ebd.EBD_WS_ATTEND, p)
    assert cache.uses_split_records(need, U, G)
    assert need <= ebd.EBD_NOALLOC_SCRATCH_BYTES
    got = {k: torch.full(ref[k].shape, float("nan"), dtype=torch.float32, device="cuda")
           for k in ("y", "vhat", "lse", "b", "r")}
    st = torch.full((U,), -1, dtype=torch.int32, device="cuda")
    ebd.ebd_attend_certify_noalloc(p, q, out.Kc, out.Vc, out.pic, out.count, got["y"], got["vhat"],
                                   got["lse"], brange=got["b"], radius=got["r"], status=st)
    torch.cuda.synchronize()
    return ref, got, st


def _check(ref, got, st):
    y, yr = got["y"].double(), ref["y"].double()
    nrm = torch.linalg.norm(yr, dim=2)
    assert torch.all(torch.linalg.norm(y - yr, dim=2) <= 2e-3 * nrm)
    floors = {"vhat": 1e-12 * nrm ** 2, "b": 1e-12 * nrm, "r": torch.full_like(nrm, 1e-12)}
    for k in ("vhat", "b", "r"):
        g, r = got[k].double(), ref[k].double()
        assert torch.all((g - r).abs() <= 1e-2 * torch.maximum(r.abs(), floors[k])), k
    assert torch.all((got["lse"].double() - ref["lse"].double()).abs()
                     <= 1e-4 * torch.clamp(ref["lse"].double().abs(), min=1.0))
    assert torch.equal(st, ref["status"])
    # the same kernels on the same inputs: the outputs are identical
    for k in ("y", "vhat", "lse", "b", "r"):
        assert torch.equal(got[k], ref[k]), k


def test_noalloc_matches_workspace_entry_point_twice():
    _say("no-alloc call 1: 40 units x 6144, G = 4, 25%, 512-row splits")
    _check(*_both([6144] * 40, 4, 0.25, 512, seed=61))
    _say("no-alloc call 2 (smaller): 9 units x 3000, G = 7, 10%, 256-row splits")
    _check(*_both([3000] * 9, 7, 0.10, 256, seed=62))
    _say("no-alloc call 3: 12 units x 4000, G = 4, 30%, two splits as the waves of one work-group")
    _check(*_both([4000] * 12, 4, 0.30, 1024, seed=63))


def test_noalloc_rejects_launches_beyond_its_scratch():
    import paper_2607_21475_amd as ebd

    cap_off = torch.zeros(2, dtype=torch.int64, device="cuda")
    p = ebd.attend_params(200000, 8, 4096, cap_off, 16)  # 256 splits of 16 rows per unit
    assert ebd.ebd_workspace_size(ebd.EBD_WS_ATTEND, p) > ebd.EBD_NOALLOC_SCRATCH_BYTES
    t = torch.zeros(16, dtype=torch.bfloat16, device="cuda")
    f = torch.zeros(16, dtype=torch.float32, device="cuda")
    c = torch.zeros(16, dtype=torch.int32, device="cuda")
    with pytest.raises(ebd.EbdError) as e:
        ebd.ebd_attend_certify_noalloc(p, t, t, t, f, c, f, f, f)
    assert e.value.code == ebd.EBD_ERR_UNSUPPORTED
