"""aj_merge_timelines_noalloc (the merge on the library's built-in per-GPU
workspace, for callers that cannot allocate) against aj_merge_timelines with
a caller-allocated workspace: every output array bit for bit, on two calls in
a row -- the 1.5B-class workload (1.19M unmerged tokens), then the smaller
agent-shaped tiny one -- so the second call runs on what the first left in
the shared array.  Inputs beyond the built-in size are refused on the host."""
import ctypes as C

import numpy as np
import pytest
import torch

from workloads import get_config, make_timelines

pytestmark = pytest.mark.gpu

OUT_KEYS = ("absorber", "cu_seqlens", "seg_src", "cu_targets", "counts", "tok", "pos", "mask",
            "old_logprob", "adv", "targets")


def _outputs(n_tl, n_tok):
    i32 = dict(dtype=torch.int32, device="cuda")
    cap = max(n_tok, 1)
    return {
        "absorber": torch.full((max(n_tl, 1),), -7, **i32),
        "cu_seqlens": torch.full((n_tl + 1,), -7, **i32),
        "seg_src": torch.full((max(n_tl, 1),), -7, **i32),
        "cu_targets": torch.full((n_tl + 1,), -7, **i32),
        "counts": torch.full((4,), -7, dtype=torch.int64, device="cuda"),
        "tok": torch.full((cap,), -7, **i32),
        "pos": torch.full((cap,), -7, **i32),
        "mask": torch.full((cap,), 7, dtype=torch.uint8, device="cuda"),
        "old_logprob": torch.full((cap,), -7.0, device="cuda"),
        "adv": torch.full((cap,), -7.0, device="cuda"),
        "targets": torch.full((cap,), -7, **i32),
    }


def _merge_both(capi, actor, tl):
    dev = actor.upload_timelines(tl, tl.lp_noise)
    n_traj, n_tl, n_tok = tl.n_traj, tl.n_tl, tl.n_tok
    ref, got = _outputs(n_tl, n_tok), _outputs(n_tl, n_tok)
    err_r = torch.zeros(1, dtype=torch.int32, device="cuda")
    err_g = torch.zeros(1, dtype=torch.int32, device="cuda")
    ws = torch.empty(capi.aj_merge_workspace_bytes(n_traj, n_tl, n_tok), dtype=torch.uint8,
                     device="cuda")
    capi.aj_merge_timelines(dev, ref, err_r, ws)
    capi.aj_merge_timelines_noalloc(dev, got, err_g)
    torch.cuda.synchronize()
    assert int(err_r.cpu()[0]) == 0 and int(err_g.cpu()[0]) == 0
    for k in OUT_KEYS:
        assert torch.equal(ref[k], got[k]), k
    return got["counts"].cpu().tolist()


def test_noalloc_merge_matches_workspace_merge_twice():
    from paper_2606_04484_amd import actor, capi
    big = make_timelines(get_config(1))
    small = make_timelines(get_config(0))
    assert capi.aj_merge_workspace_bytes(big.n_traj, big.n_tl, big.n_tok) <= \
        capi.aj_merge_noalloc_max_workspace_bytes()
    print(f"noalloc merge: {big.n_tok} then {small.n_tok} unmerged tokens", flush=True)
    c1 = _merge_both(capi, actor, big)
    c2 = _merge_both(capi, actor, small)
    assert c1[1] > c2[1] > 0 and c1[0] > 0 and c2[0] > 0


def test_noalloc_merge_refuses_inputs_beyond_its_workspace():
    from paper_2606_04484_amd import capi
    cap = capi.aj_merge_noalloc_max_workspace_bytes()
    n_tok = 2 ** 31 - 1              # the largest input: its per-token tables alone do not fit
    assert capi.aj_merge_workspace_bytes(1, 1, n_tok) > cap
    tl = capi.Timelines(1, 1, n_tok, None, None, None, None, None, None)
    out = capi.Packed(*([None] * 11))
    rc = capi.lib().aj_merge_timelines_noalloc(C.byref(tl), C.byref(out), None, None)
    assert rc == 4                   # AJ_ERR_WORKSPACE, before anything is enqueued
    assert b"built-in" in capi.lib().aj_last_error()
