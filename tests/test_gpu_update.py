"""GRPO advantages, episode selection and AdamW on the GPU against the oracle.

* advantages: float32 arithmetic against float64, 1e-5 absolute; the keep
  decision (an exact comparison of rewards) bit-exact;
* selection: every output array bit-exact, and the merge of the selected
  episodes bit-exact against the oracle's merge of its own selection;
* AdamW: the parameter update against float64 within float32 rounding
  (relative 1e-5 of the step, plus 1e-6 of the parameter), moments likewise,
  the bfloat16 copy exactly the rounding of the float32 result; at the full
  parameter count of the 1.5B-class workload (block + embedding + LM head,
  ~513M values) on sampled elements.
"""
import numpy as np
import pytest
import torch

from oracle import merge as om
from oracle import update as U
from workloads import get_config, make_timelines, make_rewards, bf16_round
from workloads.gen import weight_shapes

pytestmark = pytest.mark.gpu


def grpo_gpu(off, r, eps=1e-6):
    from paper_2606_04484_amd import capi
    n = len(r)
    adv = torch.empty(max(n, 1), dtype=torch.float32, device="cuda")
    keep = torch.empty(max(n, 1), dtype=torch.uint8, device="cuda")
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    capi.aj_grpo_advantages(torch.from_numpy(np.asarray(off, np.int32)).cuda(),
                            torch.from_numpy(np.asarray(r, np.float32)).cuda(), eps, adv, keep,
                            err)
    torch.cuda.synchronize()
    return adv[:n].cpu().numpy(), keep[:n].cpu().numpy(), int(err.cpu()[0])


def test_grpo_advantages():
    rng = np.random.default_rng(4)
    sizes = np.concatenate([rng.integers(1, 40, 60), [300, 1, 2, 700]])
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
    r = rng.integers(0, 3, off[-1]).astype(np.float32) * 0.5
    r[off[3]:off[4]] = 1.0                                    # a flat group
    adv, keep, err = grpo_gpu(off, r)
    ref_adv, ref_keep = U.grpo_advantages(off, r.astype(np.float64))
    assert err == 0
    np.testing.assert_array_equal(keep, ref_keep)
    np.testing.assert_allclose(adv, ref_adv, atol=1e-5, rtol=0)


def test_grpo_bad_offsets_reported():
    _, _, err = grpo_gpu(np.array([0, 3, 2], np.int32), np.zeros(3, np.float32))
    assert err & 8


def select_gpu(tl, old, keep, ep_adv):
    from paper_2606_04484_amd import capi, actor
    dev = actor.upload_timelines(tl, old)
    n_traj, n_tl, n_tok = tl.n_traj, tl.n_tl, tl.n_tok
    out = {"traj_tl_off": torch.empty(n_traj + 1, dtype=torch.int32, device="cuda"),
           "tl_tok_off": torch.empty(n_tl + 1, dtype=torch.int64, device="cuda"),
           "tok": torch.empty(n_tok, dtype=torch.int32, device="cuda"),
           "flags": torch.empty(n_tok, dtype=torch.uint8, device="cuda"),
           "old_logprob": torch.empty(n_tok, dtype=torch.float32, device="cuda"),
           "adv": torch.empty(n_tok, dtype=torch.float32, device="cuda"),
           "counts": torch.zeros(3, dtype=torch.int64, device="cuda")}
    ws = torch.empty(capi.aj_select_workspace_bytes(n_traj, n_tl), dtype=torch.uint8, device="cuda")
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    capi.aj_select_episodes(dev, torch.from_numpy(keep).cuda(),
                            torch.from_numpy(ep_adv.astype(np.float32)).cuda(), out, ws, err)
    torch.cuda.synchronize()
    c = out["counts"].cpu().numpy()
    res = {"traj_tl_off": out["traj_tl_off"][:c[0] + 1], "tl_tok_off": out["tl_tok_off"][:c[1] + 1],
           "tok": out["tok"][:c[2]], "flags": out["flags"][:c[2]],
           "old_logprob": out["old_logprob"][:c[2]], "adv": out["adv"][:c[2]]}
    return res, c, int(err.cpu()[0])


@pytest.mark.parametrize("cfg_i", [0, 1])
def test_select_then_merge(cfg_i):
    """Rewards -> GRPO advantages -> the non-dummy selection -> merge: every
    array bit-exact against the oracle's own pipeline."""
    from paper_2606_04484_amd import actor
    cfg = get_config(cfg_i)
    tl = make_timelines(cfg)
    off, r = make_rewards(tl.n_traj, 8 if tl.n_traj > 8 else 2, seed=cfg_i + 5)
    old = np.where((tl.flags & 3) == 2, -5.0 + tl.lp_noise, 0.0).astype(np.float32)
    adv, keep, err = grpo_gpu(off, r)
    ref_adv, ref_keep = U.grpo_advantages(off, r.astype(np.float64))
    np.testing.assert_array_equal(keep, ref_keep)
    assert 0 < keep.sum() < len(keep)
    # the selection is driven by the GPU's own advantages; both sides use them
    sel, c, err = select_gpu(tl, old, keep, adv)
    ref = U.select_episodes(tl.traj_tl_off, tl.tl_tok_off, tl.tok, tl.flags, old, keep,
                            adv.astype(np.float64))
    assert err == 0 and c[0] == len(ref[0]) - 1 and c[1] == len(ref[1]) - 1 and c[2] == len(ref[2])
    for k, v in zip(("traj_tl_off", "tl_tok_off", "tok", "flags"), ref[:4]):
        np.testing.assert_array_equal(sel[k].cpu().numpy(), v)
    np.testing.assert_array_equal(sel["old_logprob"].cpu().numpy(), ref[4].astype(np.float32))
    np.testing.assert_array_equal(sel["adv"].cpu().numpy(), ref[5].astype(np.float32))
    # merge of the selected episodes
    m = actor.Merger(sel)
    m.launch(True)
    L = m.layout(pack_tokens=1 << 30)
    eps = om.episodes_from_flat(*ref[:4], ref[4], ref[5])
    packed, _ = om.merge_batch(eps)
    n = packed.n_tok
    assert L.n_tok == n and L.n_seg == packed.n_seg
    o = {k: v.cpu().numpy() for k, v in m.out.items()}
    np.testing.assert_array_equal(o["tok"][:n], packed.tok)
    np.testing.assert_array_equal(o["cu_seqlens"][:packed.n_seg + 1], packed.cu_seqlens)
    np.testing.assert_array_equal(o["mask"][:n], packed.mask)
    np.testing.assert_array_equal(o["adv"][:n].astype(np.float64), packed.adv)


def test_select_bad_offsets_give_nothing():
    tl = make_timelines(get_config(0))
    tl.traj_tl_off = tl.traj_tl_off.copy()
    tl.traj_tl_off[3] = tl.traj_tl_off[2] - 1          # not monotone
    keep = np.ones(tl.n_traj, np.uint8)
    _, c, err = select_gpu(tl, np.zeros(tl.n_tok, np.float32), keep, np.zeros(tl.n_traj))
    assert err & 8 and list(c) == [0, 0, 0]


def adamw_gpu(p, g, m, v, copy_dtype=None, offset=0, **hp):
    from paper_2606_04484_amd import capi
    # an element offset makes the streams unaligned (the scalar path)
    mk = lambda a: torch.from_numpy(np.concatenate([np.zeros(offset, np.float32),
                                                    a.astype(np.float32)])).cuda()[offset:]
    P, G, Mm, V = mk(p), mk(g), mk(m), mk(v)
    cp = None if copy_dtype is None else torch.empty(len(p), dtype=copy_dtype, device="cuda")
    capi.aj_adamw_step(P, G, Mm, V, param_copy=cp, **hp)
    torch.cuda.synchronize()
    return (P.cpu().numpy().astype(np.float64), Mm.cpu().numpy().astype(np.float64),
            V.cpu().numpy().astype(np.float64), None if cp is None else cp.float().cpu().numpy())


def check_adamw(p0, p, m, v, rp, rm, rv, m0, gs):
    """float32 rounding bounds: the parameter within 1e-5 of its step (plus
    1e-6 of itself); the first moment within 1e-6 of its two summands' sizes
    (it can cancel); the second moment (no cancellation) relative 1e-5."""
    step = np.abs(rp - p0)
    assert np.all(np.abs(p - rp) <= 1e-5 * step + 1e-6 * np.abs(rp) + 1e-12)
    assert np.all(np.abs(m - rm) <= 1e-6 * (np.abs(m0) + np.abs(gs)) + 1e-15)
    np.testing.assert_allclose(v, rv, rtol=1e-5, atol=1e-18)


@pytest.mark.parametrize("n,offset,copy", [(1, 0, None), (1003, 0, torch.bfloat16),
                                           (4096, 1, torch.float32), (100000, 0, torch.bfloat16)])
def test_adamw(n, offset, copy):
    rng = np.random.default_rng(n)
    # hyperparameters as the float32 values the kernel receives
    hp = {k: float(np.float32(v)) for k, v in
          dict(lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.01, grad_scale=0.5).items()}
    p = rng.normal(0, 0.02, n).astype(np.float32)
    m = rng.normal(0, 1e-3, n).astype(np.float32)
    v = np.abs(rng.normal(0, 1e-5, n)).astype(np.float32)
    g = rng.normal(0, 1e-2, n).astype(np.float32)
    for step in (1, 7):
        gp, gm, gv, cp = adamw_gpu(p, g, m, v, copy, offset, step=step, **hp)
        rp, rm, rv = U.adamw_step(p, g, m, v, hp["lr"], hp["beta1"], hp["beta2"], hp["eps"],
                                  hp["weight_decay"], step, hp["grad_scale"])
        check_adamw(p.astype(np.float64), gp, gm, gv, rp, rm, rv, m, g * hp["grad_scale"])
        if copy is torch.bfloat16:
            np.testing.assert_array_equal(cp, bf16_round(gp.astype(np.float32)))
        elif copy is torch.float32:
            np.testing.assert_array_equal(cp, gp.astype(np.float32))


def test_adamw_full_parameter_count():
    """Every trainable value of the 1.5B-class workload in one call; sampled
    elements against the oracle."""
    m_cfg = get_config(1).model
    n = sum(int(np.prod(s)) for s in weight_shapes(m_cfg).values())
    assert n > 5e8
    gen = torch.Generator(device="cuda").manual_seed(9)
    f32 = dict(generator=gen, device="cuda", dtype=torch.float32)
    P = torch.randn(n, **f32) * 0.02
    G = torch.randn(n, **f32) * 1e-3
    Mm = torch.randn(n, **f32) * 1e-4
    V = torch.rand(n, **f32) * 1e-6
    idx = torch.from_numpy(np.random.default_rng(0).integers(0, n, 4096)).cuda()
    idx = torch.cat([idx, torch.tensor([0, n - 1], device="cuda")])
    p0, g0, m0, v0 = (t[idx].cpu().numpy() for t in (P, G, Mm, V))
    cp = torch.empty(n, dtype=torch.bfloat16, device="cuda")
    from paper_2606_04484_amd import capi
    hp = [float(np.float32(x)) for x in (2e-4, 0.9, 0.95, 1e-8, 0.1)]
    capi.aj_adamw_step(P, G, Mm, V, *hp, 3, param_copy=cp)
    torch.cuda.synchronize()
    rp, rm, rv = U.adamw_step(p0, g0, m0, v0, *hp, 3)
    check_adamw(p0.astype(np.float64), P[idx].cpu().numpy().astype(np.float64),
                Mm[idx].cpu().numpy().astype(np.float64), V[idx].cpu().numpy().astype(np.float64),
                rp, rm, rv, m0, g0)
    np.testing.assert_array_equal(cp[idx].float().cpu().numpy(),
                                  bf16_round(P[idx].cpu().numpy()))
