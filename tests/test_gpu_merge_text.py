"""GPU merge under text-level Match against the oracle: bit-exact on every
output array and on the TI-consistency report.

Covers the hand-worked text golden cases, the token golden cases with text
keys that follow the token ids, the seeded workloads at full size with every
(think_p=1) or half (0.5) of the responses re-rendered without their thinking
section, no re-rendering (text- and token-level GPU merges then agree), an
empty batch, and block keys that do not fit the block-start bits (reported
through the device error word, every count 0).
"""
import numpy as np
import pytest
import torch

from oracle import merge as om
from workloads import get_config, make_timelines
from tests.cases import golden_merge_cases, golden_text_cases, case_to_flat

pytestmark = pytest.mark.gpu


def _run(tl, old, text=True):
    from paper_2606_04484_amd import actor
    dev = actor.upload_timelines(tl, old)
    m = actor.Merger(dev, text=text)
    m.launch(True)
    L = m.layout(pack_tokens=1 << 30)
    torch.cuda.synchronize()
    return m, L


def _check(tl, old):
    eps = om.episodes_from_flat(tl.traj_tl_off, tl.tl_tok_off, tl.tok, tl.flags, old, tl.adv,
                                tl.blk_text)
    ref, absorbers = om.merge_batch(eps, om.match_text)
    m, L = _run(tl, old)
    o = {k: v.cpu().numpy() for k, v in m.out.items()}
    glob = []
    for e, ab in enumerate(absorbers):
        base = int(tl.traj_tl_off[e])
        glob.extend(a + base if a >= 0 else -1 for a in ab)
    np.testing.assert_array_equal(o["absorber"][:tl.n_tl], glob)
    assert L.n_seg == ref.n_seg and L.n_tok == ref.n_tok
    np.testing.assert_array_equal(o["cu_seqlens"][:L.n_seg + 1], ref.cu_seqlens)
    np.testing.assert_array_equal(o["seg_src"][:L.n_seg], [i for i, a in enumerate(glob) if a < 0])
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
    ti = tuple(int(v) for v in m.ti.cpu())
    assert ti == om.ti_report(eps, om.match_text)
    return m, L, ti


@pytest.mark.parametrize("case", golden_text_cases(), ids=lambda c: c["name"])
def test_golden_text(case):
    tl, lp = case_to_flat(case)
    _, _, ti = _check(tl, lp)
    assert list(ti) == case["expect"]["ti"]


@pytest.mark.parametrize("case", golden_merge_cases(), ids=lambda c: c["name"])
def test_token_golden_with_token_keys(case):
    tl, lp = case_to_flat(case)
    starts = np.flatnonzero(tl.flags & 4).tolist() + [tl.n_tok]
    interned = {}
    tl.blk_text = np.array([interned.setdefault(tuple(tl.tok[a:b].tolist()), len(interned) + 1)
                            for a, b in zip(starts[:-1], starts[1:])], np.uint64)
    _, _, ti = _check(tl, lp)
    assert ti == (0, 0)


@pytest.mark.parametrize("cfg_id,think_p", [(0, 1.0), (1, 1.0), (1, 0.5), (2, 1.0), (3, 1.0),
                                            (4, 1.0)])
def test_full_workloads_stripped_thinking(cfg_id, think_p):
    tl = make_timelines(get_config(cfg_id), think_p=think_p)
    print(f"text merge parity cfg={cfg_id} think_p={think_p} n_tok={tl.n_tok} n_blk={tl.n_blk}",
          flush=True)
    _, L, ti = _check(tl, tl.lp_noise)
    assert ti[0] > 0


def test_no_stripping_equals_token_merge():
    tl = make_timelines(get_config(1), think_p=0.0)
    a, La, ti = _check(tl, tl.lp_noise)
    b, Lb = _run(tl, tl.lp_noise, text=False)
    assert ti == (0, 0) and (La.n_seg, La.n_tok, La.n_mask) == (Lb.n_seg, Lb.n_tok, Lb.n_mask)
    for k in ("tok", "pos", "mask", "old_logprob", "adv", "targets"):
        n = La.n_mask if k == "targets" else La.n_tok
        assert torch.equal(a.out[k][:n], b.out[k][:n]), k
    assert torch.equal(a.out["cu_seqlens"][:La.n_seg + 1], b.out["cu_seqlens"][:La.n_seg + 1])


def test_deterministic():
    tl = make_timelines(get_config(3), think_p=0.5)
    a, La = _run(tl, tl.lp_noise)
    b, Lb = _run(tl, tl.lp_noise)
    valid = {"absorber": tl.n_tl, "cu_seqlens": La.n_seg + 1, "seg_src": La.n_seg,
             "cu_targets": La.n_seg + 1, "counts": 4, "targets": La.n_mask}
    for k in a.out:
        n = valid.get(k, La.n_tok)
        assert torch.equal(a.out[k][:n], b.out[k][:n]), k
    assert torch.equal(a.ti, b.ti)


def test_empty_batch():
    from workloads.gen import Timelines
    tl = Timelines(np.zeros(1, np.int32), np.zeros(1, np.int64), np.zeros(0, np.int32),
                   np.zeros(0, np.uint8), np.zeros(0, np.float32), np.zeros(0, np.float32),
                   np.zeros(0, np.uint64))
    m, L = _run(tl, np.zeros(0, np.float32))
    assert (L.n_seg, L.n_tok, L.n_mask) == (0, 0, 0) and L.packs == []
    assert m.device_error() == 0 and m.ti.cpu().tolist() == [0, 0]


def test_block_count_mismatch_is_reported():
    tl = make_timelines(get_config(0), think_p=1.0)
    tl.blk_text = tl.blk_text[:-1]                  # one key short
    m, L = _run(tl, tl.lp_noise)
    assert m.device_error() & 16
    assert (L.n_seg, L.n_tok, L.n_mask) == (0, 0, 0)


def test_timeline_not_starting_a_block_is_reported():
    tl = make_timelines(get_config(0), think_p=1.0)
    tl.flags = tl.flags.copy()
    first = int(tl.tl_tok_off[3])
    k = int(np.count_nonzero(tl.flags[:first] & 4))
    tl.flags[first] &= ~np.uint8(4)                 # timeline 3 no longer starts a block
    tl.blk_text = np.delete(tl.blk_text, k)         # the keys still match the bits
    m, L = _run(tl, tl.lp_noise)
    assert m.device_error() & 16 and m.device_error() & 2
    assert (L.n_seg, L.n_tok, L.n_mask) == (0, 0, 0)
