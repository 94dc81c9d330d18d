"""Pins for the oracle of the steps around the actor update (CPU, float64):
GRPO advantages against scipy's z-score and hand-worked groups, the C3
non-dummy filter on flat groups, episode selection invariants, and AdamW
against torch.optim.AdamW."""
import numpy as np
import pytest
import torch
from scipy import stats

from oracle import update as U
from workloads import get_config, make_timelines, make_rewards


def test_grpo_hand_worked_groups():
    off = np.array([0, 2, 5, 6, 10])
    r = np.array([0, 1, 1, 1, 1, 3, 0, 0, 1, 1], np.float64)
    adv, keep = U.grpo_advantages(off, r, eps=0.0)
    np.testing.assert_allclose(adv[:2], [-np.sqrt(0.5), np.sqrt(0.5)], rtol=1e-14)
    assert np.all(adv[2:6] == 0) and np.all(keep[2:6] == 0)      # flat group, group of one
    np.testing.assert_allclose(adv[6:], [-0.75 ** 0.5] * 2 + [0.75 ** 0.5] * 2, rtol=1e-14)
    assert list(keep) == [1, 1, 0, 0, 0, 0, 1, 1, 1, 1]


def test_grpo_matches_scipy_zscore():
    rng = np.random.default_rng(0)
    sizes = rng.integers(2, 20, 30)
    off = np.concatenate([[0], np.cumsum(sizes)])
    r = rng.normal(0, 2, off[-1])
    adv, keep = U.grpo_advantages(off, r, eps=0.0)
    assert np.all(keep == 1)
    for a, b in zip(off[:-1], off[1:]):
        np.testing.assert_allclose(adv[a:b], stats.zscore(r[a:b], ddof=1), rtol=1e-12)
    # eps only shrinks the scale
    adv_e, _ = U.grpo_advantages(off, r, eps=0.5)
    for a, b in zip(off[:-1], off[1:]):
        sd = np.std(r[a:b], ddof=1)
        np.testing.assert_allclose(adv_e[a:b], adv[a:b] * sd / (sd + 0.5), rtol=1e-12)


def test_rewards_generator_groups():
    off, r = make_rewards(64, 8, seed=3)
    assert off[0] == 0 and off[-1] == 64 and np.all(np.diff(off) == 8)
    adv, keep = U.grpo_advantages(off, r)
    flat = [np.all(r[a:b] == r[a]) for a, b in zip(off[:-1], off[1:])]
    assert any(flat) and not all(flat)
    for f, a, b in zip(flat, off[:-1], off[1:]):
        assert np.all(keep[a:b] == (0 if f else 1))


def test_select_episodes_keeps_slices_in_order():
    tl = make_timelines(get_config(0))
    keep = np.array([1, 0, 1, 1, 0, 0, 1, 0], np.uint8)
    ep_adv = np.arange(8, dtype=np.float64) - 3.5
    old = np.linspace(-3, -1, tl.n_tok)
    t_off, k_off, tok, fl, olp, adv = U.select_episodes(tl.traj_tl_off, tl.tl_tok_off, tl.tok,
                                                         tl.flags, old, keep, ep_adv)
    kept = np.flatnonzero(keep)
    assert len(t_off) == len(kept) + 1
    j = 0
    for n_new, e in enumerate(kept):
        tls = range(tl.traj_tl_off[e], tl.traj_tl_off[e + 1])
        assert t_off[n_new + 1] - t_off[n_new] == len(tls)
        for i in tls:
            a, b = tl.tl_tok_off[i], tl.tl_tok_off[i + 1]
            c, d = k_off[j], k_off[j + 1]
            assert np.array_equal(tok[c:d], tl.tok[a:b]) and np.array_equal(fl[c:d], tl.flags[a:b])
            assert np.array_equal(olp[c:d], old[a:b])
            assert np.array_equal(adv[c:d], np.where((tl.flags[a:b] & 3) == 2, ep_adv[e], 0.0))
            j += 1
    assert k_off[-1] == len(tok)


@pytest.mark.parametrize("wd", [0.0, 0.1])
def test_adamw_matches_torch(wd):
    rng = np.random.default_rng(1)
    p0 = rng.normal(0, 1, 257)
    grads = [rng.normal(0, 1, 257) for _ in range(4)]
    pt = torch.tensor(p0, dtype=torch.float64, requires_grad=True)
    opt = torch.optim.AdamW([pt], lr=3e-3, betas=(0.9, 0.95), eps=1e-8, weight_decay=wd)
    p, m, v = p0.copy(), np.zeros(257), np.zeros(257)
    for t, g in enumerate(grads, start=1):
        pt.grad = torch.tensor(g)
        opt.step()
        p, m, v = U.adamw_step(p, g, m, v, 3e-3, 0.9, 0.95, 1e-8, wd, t)
        np.testing.assert_allclose(p, pt.detach().numpy(), rtol=1e-13, atol=1e-15)
