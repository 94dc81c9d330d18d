"""GPU merge / flatten against the oracle: bit-exact on every output array.

Covers the hand-worked golden cases, all five seeded workloads at full size
(merged and unmerged layouts), 16 side-by-side copies of the 1.5B-class
workload, thousands of episodes whose segments are a few tokens long (many
segments per output range, several rounds of the survivor scan), an empty
batch, and offsets that do not tile the token range (reported through the
device error word, every count 0).
"""
import numpy as np
import pytest
import torch

from oracle import merge as om
from workloads import get_config, make_timelines
from tests.cases import golden_merge_cases, case_to_flat

pytestmark = pytest.mark.gpu


def _run(tl, old, merged=True):
    from paper_2606_04484_amd import actor
    dev = actor.upload_timelines(tl, old)
    m = actor.Merger(dev)
    m.launch(merged)
    L = m.layout(pack_tokens=1 << 30)
    torch.cuda.synchronize()
    return m, L


def _check(tl, old, merged):
    eps = om.episodes_from_flat(tl.traj_tl_off, tl.tl_tok_off, tl.tok, tl.flags, old, tl.adv)
    if merged:
        ref, absorbers = om.merge_batch(eps)
    else:
        ref, absorbers = om.unmerged_batch(eps), [[-1] * len(e) for e in eps]
    m, L = _run(tl, old, merged)
    o = {k: v.cpu().numpy() for k, v in m.out.items()}
    n_tl = tl.n_tl
    glob = []
    for e, ab in enumerate(absorbers):
        base = int(tl.traj_tl_off[e])
        glob.extend(a + base if a >= 0 else -1 for a in ab)
    np.testing.assert_array_equal(o["absorber"][:n_tl], glob)
    assert L.n_seg == ref.n_seg and L.n_tok == ref.n_tok
    np.testing.assert_array_equal(o["cu_seqlens"][:L.n_seg + 1], ref.cu_seqlens)
    surv = [i for i, a in enumerate(glob) if a == -1]
    np.testing.assert_array_equal(o["seg_src"][:L.n_seg], surv)
    n = ref.n_tok
    np.testing.assert_array_equal(o["tok"][:n], ref.tok)
    np.testing.assert_array_equal(o["pos"][:n], ref.pos)
    np.testing.assert_array_equal(o["mask"][:n], ref.mask)
    np.testing.assert_array_equal(o["old_logprob"][:n].astype(np.float64), ref.old_logprob)
    np.testing.assert_array_equal(o["adv"][:n].astype(np.float64), ref.adv)
    tgt = np.flatnonzero((ref.mask == 1) & (ref.pos != 0))
    assert L.n_mask == len(tgt)
    np.testing.assert_array_equal(o["targets"][:len(tgt)], tgt)
    np.testing.assert_array_equal(o["cu_targets"][:L.n_seg + 1],
                                  np.searchsorted(tgt, ref.cu_seqlens, side="left"))
    lens = np.diff(ref.cu_seqlens)
    assert L.max_seqlen == (int(lens.max()) if len(lens) else 0)
    assert m.device_error() == 0


@pytest.mark.parametrize("case", golden_merge_cases(), ids=lambda c: c["name"])
def test_golden(case):
    tl, lp = case_to_flat(case)
    _check(tl, lp, merged=True)
    _check(tl, lp, merged=False)


@pytest.mark.parametrize("cfg_id", [0, 1, 2, 3, 4])
@pytest.mark.parametrize("merged", [True, False])
def test_full_workloads(cfg_id, merged):
    tl = make_timelines(get_config(cfg_id))
    print(f"merge parity cfg={cfg_id} merged={merged} n_tok={tl.n_tok}", flush=True)
    _check(tl, tl.lp_noise, merged)


def test_deterministic():
    tl = make_timelines(get_config(3))
    a, La = _run(tl, tl.lp_noise)
    b, Lb = _run(tl, tl.lp_noise)
    valid = {"absorber": tl.n_tl, "cu_seqlens": La.n_seg + 1, "seg_src": La.n_seg,
             "cu_targets": La.n_seg + 1, "counts": 4, "targets": La.n_mask}
    for k in a.out:
        n = valid.get(k, La.n_tok)      # per-token outputs: the merged length
        assert torch.equal(a.out[k][:n], b.out[k][:n]), k


def test_empty_batch():
    from workloads.gen import Timelines
    tl = Timelines(np.zeros(1, np.int32), np.zeros(1, np.int64), np.zeros(0, np.int32),
                   np.zeros(0, np.uint8), np.zeros(0, np.float32), np.zeros(0, np.float32))
    m, L = _run(tl, np.zeros(0, np.float32))
    assert (L.n_seg, L.n_tok, L.n_mask) == (0, 0, 0) and L.packs == []


def test_offsets_not_tiling_are_reported():
    tl = make_timelines(get_config(0))
    tl.tl_tok_off = tl.tl_tok_off.copy()
    tl.tl_tok_off[5], tl.tl_tok_off[6] = tl.tl_tok_off[6], tl.tl_tok_off[5]   # not monotone
    m, L = _run(tl, tl.lp_noise)
    from paper_2606_04484_amd.capi import lib  # noqa: F401
    assert m.device_error() & 8
    assert (L.n_seg, L.n_tok, L.n_mask) == (0, 0, 0)


def _replicate(tl, R):
    """R copies of the timelines side by side (host arrays)."""
    from workloads.gen import Timelines
    k = np.arange(R, dtype=np.int64)[:, None]
    traj = np.concatenate([[0], (tl.traj_tl_off[1:][None, :] + k * tl.n_tl).ravel()]).astype(np.int32)
    tok_off = np.concatenate([[0], (tl.tl_tok_off[1:][None, :] + k * tl.n_tok).ravel()]).astype(np.int64)
    return Timelines(traj, tok_off, np.tile(tl.tok, R), np.tile(tl.flags, R), np.tile(tl.adv, R),
                     np.tile(tl.lp_noise, R))


def test_replicated_workload():
    """16 copies of block1.5b-64x8 (19M unmerged tokens): the episodes are
    independent, so every output is the oracle's merge of one copy, repeated
    with its offsets shifted; bit-exact."""
    R = 16
    base = make_timelines(get_config(1))
    eps = om.episodes_from_flat(base.traj_tl_off, base.tl_tok_off, base.tok, base.flags,
                                base.lp_noise, base.adv)
    ref, absorbers = om.merge_batch(eps)
    glob = []
    for e, ab in enumerate(absorbers):
        b0 = int(base.traj_tl_off[e])
        glob.extend(a + b0 if a >= 0 else -1 for a in ab)
    glob = np.asarray(glob, np.int64)
    tl = _replicate(base, R)
    print(f"replicated merge: {R} copies, {tl.n_tok} unmerged tokens", flush=True)
    m, L = _run(tl, tl.lp_noise)
    o = {k: v.cpu().numpy() for k, v in m.out.items()}
    k = np.arange(R, dtype=np.int64)[:, None]
    n_tl, T = base.n_tl, ref.n_tok
    assert (L.n_seg, L.n_tok) == (R * ref.n_seg, R * T)
    exp_abs = np.where(glob[None, :] >= 0, glob[None, :] + k * n_tl, -1).ravel()
    np.testing.assert_array_equal(o["absorber"][:R * n_tl], exp_abs)
    cu = np.concatenate([(ref.cu_seqlens[:-1][None, :] + k * T).ravel(), [R * T]])
    np.testing.assert_array_equal(o["cu_seqlens"][:L.n_seg + 1], cu)
    surv = np.flatnonzero(glob == -1)
    np.testing.assert_array_equal(o["seg_src"][:L.n_seg], (surv[None, :] + k * n_tl).ravel())
    n = R * T
    np.testing.assert_array_equal(o["tok"][:n], np.tile(ref.tok, R))
    np.testing.assert_array_equal(o["pos"][:n], np.tile(ref.pos, R))
    np.testing.assert_array_equal(o["mask"][:n], np.tile(ref.mask, R))
    np.testing.assert_array_equal(o["old_logprob"][:n].astype(np.float64), np.tile(ref.old_logprob, R))
    np.testing.assert_array_equal(o["adv"][:n].astype(np.float64), np.tile(ref.adv, R))
    tgt = np.flatnonzero((ref.mask == 1) & (ref.pos != 0))
    all_t = (tgt[None, :] + k * T).ravel()
    assert L.n_mask == len(all_t)
    np.testing.assert_array_equal(o["targets"][:len(all_t)], all_t)
    np.testing.assert_array_equal(o["cu_targets"][:L.n_seg + 1],
                                  np.searchsorted(all_t, cu, side="left"))
    assert L.max_seqlen == int(np.diff(ref.cu_seqlens).max())
    assert m.device_error() == 0


def _tiny_timelines(n_ep, seed):
    """Many episodes of short timelines (1-6 token blocks): merged segments
    of a few tokens, so one emit range spans far more than 64 segments and
    the survivor scan runs several rounds; 1 call in 5 rewrites its
    context."""
    from workloads.gen import Timelines, FLAG_BLOCK_START
    rng = np.random.default_rng(seed)
    traj, tl_off, tok, flags, adv, lp = [0], [0], [], [], [], []

    def block(author):
        m = int(rng.integers(1, 7))
        f = np.full(m, author, np.uint8)
        f[0] |= FLAG_BLOCK_START
        return list(rng.integers(0, 50, m)), list(f)

    for _ in range(n_ep):
        n_calls = int(rng.integers(1, 5))
        ctx_t, ctx_f = block(0)
        for _c in range(n_calls):
            if rng.random() < 0.2:
                ctx_t, ctx_f = block(0)
            rt, rf = block(2)
            a = float(rng.normal())
            tok += ctx_t + rt
            flags += ctx_f + rf
            adv += [0.0] * len(ctx_t) + [a] * len(rt)
            lp += [0.0] * len(ctx_t) + list(rng.normal(-2.0, 0.5, len(rt)))
            tl_off.append(tl_off[-1] + len(ctx_t) + len(rt))
            # the next call's context: this one's, its response as context
            # (author kept), then an observation block
            ot, of = block(1)
            ctx_t, ctx_f = ctx_t + rt + ot, ctx_f + rf + of
        traj.append(traj[-1] + n_calls)
    tl = Timelines(np.asarray(traj, np.int32), np.asarray(tl_off, np.int64),
                   np.asarray(tok, np.int32), np.asarray(flags, np.uint8),
                   np.asarray(adv, np.float32), np.zeros(len(tok), np.float32))
    return tl, np.asarray(lp, np.float32)


@pytest.mark.parametrize("merged", [True, False])
def test_many_tiny_segments(merged):
    """~6000 episodes of a few short calls each (segments of ~4-40 tokens,
    >12000 timelines): bit-exact against the oracle."""
    tl, lp = _tiny_timelines(6000, seed=7)
    print(f"tiny segments: {tl.n_traj} episodes, {tl.n_tl} timelines, {tl.n_tok} tokens",
          flush=True)
    _check(tl, lp, merged)
