"""Pins for the model/loss oracle, CPU only, float64.

Each pin checks the oracle against something other than itself: library
routines (torch's rms_norm, scaled_dot_product_attention, log_softmax, silu)
on the special cases that reduce to them, closed forms of the clipped
surrogate, the complex-number form of RoPE, exact special cases (zero
weights), central finite differences for every gradient, and the
merged == unmerged invariant the paper's timeline merging relies on.
"""
import dataclasses

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import merge as om
from oracle import model as M
from workloads import get_config, make_timelines, make_weights_numpy, make_lora_numpy
from workloads.configs import ModelConfig



@pytest.fixture(autouse=True, scope="module")
def _float64_torch():
    """torch references in float64 for this module only (the session default
    is restored afterwards, so other modules' tensors keep float32)."""
    old = torch.get_default_dtype()
    torch.set_default_dtype(torch.float64)
    yield
    torch.set_default_dtype(old)

SMALL = ModelConfig(d_model=16, n_q_heads=4, n_kv_heads=2, head_dim=8, d_ff=24, vocab=37,
                    dtype="f32", init_std=0.3)


def _packed(lens, vocab, rng, mask_p=0.6):
    cu = np.concatenate([[0], np.cumsum(lens)])
    n = int(cu[-1])
    tok = rng.integers(0, vocab, n)
    mask = (rng.random(n) < mask_p).astype(np.uint8)
    pos = np.concatenate([np.arange(L) for L in lens])
    return om.Packed(cu, tok, mask, -np.log(vocab) + rng.normal(0, 0.5, n),
                     rng.normal(0, 1, n), pos)


# ------------------------------------------------------------------ pieces vs library routines

def test_rmsnorm_matches_torch():
    rng = np.random.default_rng(0)
    x, g = rng.normal(size=(7, 16)), rng.normal(size=16)
    y, r = M.rmsnorm(x, g, 1e-6)
    ref = F.rms_norm(torch.tensor(x), (16,), torch.tensor(g), eps=1e-6).numpy()
    np.testing.assert_allclose(y, ref, rtol=1e-13, atol=1e-13)


def test_rope_is_complex_rotation():
    rng = np.random.default_rng(1)
    hd, n = 8, 11
    x = rng.normal(size=(n, 2, hd))
    pos = rng.integers(0, 70000, n)
    cos, sin = M.rope_angles(pos, hd, 1e6)
    y = M.rope(x, cos, sin)
    # pair i = (x_i, x_{i+hd/2}) as a complex number times exp(1j * pos * theta^(-2i/hd))
    z = x[..., :hd // 2] + 1j * x[..., hd // 2:]
    w = np.exp(1j * pos[:, None] * (1e6 ** (-np.arange(0, hd, 2) / hd)))[:, None, :]
    zr = z * w
    np.testing.assert_allclose(y[..., :hd // 2], zr.real, atol=1e-12)
    np.testing.assert_allclose(y[..., hd // 2:], zr.imag, atol=1e-12)
    c0, s0 = M.rope_angles(np.zeros(3), hd, 1e6)
    np.testing.assert_array_equal(M.rope(x[:3], c0, s0), x[:3])


def test_rope_bwd_is_transpose():
    rng = np.random.default_rng(2)
    x, dy = rng.normal(size=(5, 3, 8)), rng.normal(size=(5, 3, 8))
    cos, sin = M.rope_angles(rng.integers(0, 1000, 5), 8, 1e6)
    lhs = np.sum(M.rope(x, cos, sin) * dy)
    rhs = np.sum(x * M.rope_bwd(dy, cos, sin))
    assert abs(lhs - rhs) < 1e-12


def test_attention_single_segment_matches_sdpa():
    rng = np.random.default_rng(3)
    L, Hq, Hkv, hd = 9, 4, 2, 8
    q, k, v = rng.normal(size=(L, Hq, hd)), rng.normal(size=(L, Hkv, hd)), rng.normal(size=(L, Hkv, hd))
    o, lse = M.attention_segment(q, k, v, 1 / np.sqrt(hd))
    tq = torch.tensor(q).permute(1, 0, 2)
    tk = torch.tensor(k).permute(1, 0, 2).repeat_interleave(Hq // Hkv, dim=0)
    tv = torch.tensor(v).permute(1, 0, 2).repeat_interleave(Hq // Hkv, dim=0)
    ref = F.scaled_dot_product_attention(tq, tk, tv, is_causal=True).permute(1, 0, 2).numpy()
    np.testing.assert_allclose(o, ref, atol=1e-12)
    s = torch.einsum("hqd,hkd->hqk", tq, tk) / np.sqrt(hd)
    s = s.masked_fill(~torch.tril(torch.ones(L, L, dtype=torch.bool)), float("-inf"))
    np.testing.assert_allclose(lse, torch.logsumexp(s, dim=-1).numpy(), atol=1e-12)


def test_kv_head_mapping():
    assert [M.kv_head(h, 28, 4) for h in range(28)] == [h // 7 for h in range(28)]
    assert [M.kv_head(h, 12, 2) for h in range(12)] == [h // 6 for h in range(12)]


def test_zero_weights_block_is_identity():
    m = SMALL
    rng = np.random.default_rng(4)
    W = M.f64_weights(make_weights_numpy(m, seed=5))
    W["w_o"][:] = 0
    W["w_down"][:] = 0
    p = _packed([5, 3], m.vocab, rng)
    x = W["emb"][p.tok]
    y, _ = M.block_forward(x, W, p.cu_seqlens, p.pos, m)
    np.testing.assert_array_equal(y, x)


def test_zero_vocab_head_gives_uniform_logprob():
    m = SMALL
    rng = np.random.default_rng(5)
    W = M.f64_weights(make_weights_numpy(m, seed=6))
    W["w_vocab"][:] = 0
    p = _packed([6, 4], m.vocab, rng)
    lp = M.current_logprob(p, W, m)
    tgt = M.target_positions(p.cu_seqlens, p.n_tok)
    np.testing.assert_array_equal(lp[tgt], np.full(len(tgt), -np.log(m.vocab)))
    assert np.isnan(lp[p.cu_seqlens[:-1]]).all()


def test_lm_head_matches_log_softmax():
    m = SMALL
    rng = np.random.default_rng(6)
    W = M.f64_weights(make_weights_numpy(m, seed=7, gain_std=0.3))
    y = rng.normal(size=(10, m.d_model))
    tok = rng.integers(0, m.vocab, 10)
    tgt = np.arange(1, 10)
    hn, _, lp, lse = M.lm_head_forward(y, W, tok, tgt, m, row_chunk=4)
    hn_ref = F.rms_norm(torch.tensor(y), (m.d_model,), torch.tensor(W["final_norm"]), eps=m.rms_eps)
    ls = torch.log_softmax(hn_ref @ torch.tensor(W["w_vocab"]).T, dim=-1).numpy()
    np.testing.assert_allclose(lp, ls[tgt - 1, tok[tgt]], atol=1e-12)


def test_segments_are_independent():
    m = SMALL
    rng = np.random.default_rng(7)
    W = M.f64_weights(make_weights_numpy(m, seed=8))
    p = _packed([4, 7, 3], m.vocab, rng)
    segs = [np.arange(p.cu_seqlens[s], p.cu_seqlens[s + 1]) for s in range(3)]
    perm = [2, 0, 1]
    idx = np.concatenate([segs[s] for s in perm])
    q = om.Packed(np.concatenate([[0], np.cumsum([len(segs[s]) for s in perm])]), p.tok[idx],
                  p.mask[idx], p.old_logprob[idx], p.adv[idx], p.pos[idx])
    a = M.actor_update(p, W, m)
    b = M.actor_update(q, W, m)
    np.testing.assert_allclose(b["logprob"], a["logprob"][idx], atol=1e-13, equal_nan=True)
    assert abs(a["loss"] - b["loss"]) < 1e-13
    for k in a["grads"]:
        np.testing.assert_allclose(a["grads"][k], b["grads"][k], atol=1e-13)


# ------------------------------------------------------------------ clipped surrogate closed forms

def test_pg_on_policy_closed_form():
    """old == current: r = 1 -> loss = -mean_mask(A), dloss/dlogprob = -A / N."""
    m = SMALL
    rng = np.random.default_rng(8)
    W = M.f64_weights(make_weights_numpy(m, seed=9))
    p = _packed([8, 6], m.vocab, rng)
    p.old_logprob = M.current_logprob(p, W, m)
    out = M.actor_update(p, W, m)
    tgt = out["tgt"]
    sel = p.mask[tgt] == 1
    assert abs(out["loss"] + np.mean(p.adv[tgt][sel])) < 1e-13
    np.testing.assert_allclose(out["ratio"], 1.0, atol=1e-14)


def test_pg_terms_branches():
    lp = np.log(np.array([0.5, 0.9, 1.0, 1.1, 1.5, 0.5, 0.9, 1.5, 1.0]))
    old = np.zeros_like(lp)
    A = np.array([1, 1, 1, 1, 1, -1, -1, -1, 0.0])
    term, dterm, r = M.pg_terms(lp, old, A, 0.2)
    # A > 0: -A*min(r, 1.2); A < 0: -A*max(r, 0.8); A == 0: 0
    np.testing.assert_allclose(term, [-0.5, -0.9, -1.0, -1.1, -1.2, 0.8, 0.9, 1.5, 0.0], atol=1e-15)
    # gradient -A*r where the unclipped branch is active
    np.testing.assert_allclose(dterm, [-0.5, -0.9, -1.0, -1.1, 0.0, 0.0, 0.9, 1.5, 0.0], atol=1e-15)
    # ties count as unclipped
    t2, d2, _ = M.pg_terms(np.log([1.2, 0.8]), np.zeros(2), np.array([1.0, -1.0]), 0.2)
    assert d2[0] != 0 and d2[1] != 0


def test_pg_large_eps_and_zero_adv():
    m = dataclasses.replace(SMALL, clip_eps=1e9)
    rng = np.random.default_rng(9)
    W = M.f64_weights(make_weights_numpy(m, seed=10))
    p = _packed([7, 5], m.vocab, rng)
    out = M.actor_update(p, W, m)
    sel = p.mask[out["tgt"]] == 1
    r = np.exp(out["logprob"][out["tgt"]][sel] - p.old_logprob[out["tgt"]][sel])
    assert abs(out["loss"] + np.mean(r * p.adv[out["tgt"]][sel])) < 1e-12
    p.adv[:] = 0
    out = M.actor_update(p, W, SMALL)
    assert out["loss"] == 0.0
    for g in out["grads"].values():
        assert not np.any(g)


# ------------------------------------------------------------------ gradients

def _loss_with(p, W, m, name, idx, h):
    W2 = {k: v.copy() for k, v in W.items()}
    W2[name][idx] += h
    return M.actor_update(p, W2, m, n_mask=7)["loss"]


@pytest.mark.parametrize("name", ["emb", "attn_norm", "w_qkv", "w_o", "mlp_norm", "w_gate_up",
                                  "w_down", "final_norm", "w_vocab"])
def test_gradients_match_finite_differences(name):
    m = SMALL
    rng = np.random.default_rng(11)
    W = M.f64_weights(make_weights_numpy(m, seed=12, gain_std=0.3))
    p = _packed([6, 5, 4], m.vocab, rng, mask_p=0.7)
    out = M.actor_update(p, W, m, n_mask=7)
    # keep every ratio away from the clip kinks so the loss is smooth around W
    tgt = out["tgt"]
    sel = p.mask[tgt] == 1
    assert np.all(np.abs(np.abs(out["ratio"] - 1) - m.clip_eps) > 1e-3)
    g = out["grads"][name]
    flat = list(np.ndindex(g.shape))
    pick = [flat[i] for i in rng.choice(len(flat), size=min(40, len(flat)), replace=False)]
    if name == "emb":
        pick = [(int(p.tok[i]), j) for i, j in zip(rng.integers(0, p.n_tok, 20), rng.integers(0, m.d_model, 20))]
    for idx in pick:
        h = 1e-6 * max(1.0, abs(W[name][idx]))
        fd = (_loss_with(p, W, m, name, idx, h) - _loss_with(p, W, m, name, idx, -h)) / (2 * h)
        assert abs(fd - g[idx]) <= 1e-6 * max(1e-3, abs(fd)) + 1e-9, (name, idx, fd, g[idx])


def _torch_loss(W, p, m, tgt, L=None, scale=0.0):
    """A torch float64 forward built from library ops: log-probs at tgt and the
    clipped loss.  W (and the LoRA matrices L, if any) are torch tensors; a
    projection with adapters is v W^T + scale (v A^T) B^T, written out."""
    Hq, Hkv, hd, Fd = m.n_q_heads, m.n_kv_heads, m.head_dim, m.d_ff
    n = p.n_tok
    ang = torch.tensor(p.pos, dtype=torch.float64)[:, None] * (m.rope_theta ** (-torch.arange(0, hd, 2) / hd))

    def rot(t):
        z = torch.view_as_complex(torch.stack([t[..., :hd // 2], t[..., hd // 2:]], -1).contiguous())
        zr = torch.view_as_real(z * torch.polar(torch.ones_like(ang), ang)[:, None, :])
        return torch.cat([zr[..., 0], zr[..., 1]], -1)

    def proj(v, name, sfx):
        out = v @ W[name + sfx].T
        if L is not None:
            out = out + scale * (v @ L["lora_a." + name + sfx].T) @ L["lora_b." + name + sfx].T
        return out

    def block(x, sfx):
        a = F.rms_norm(x, (m.d_model,), W["attn_norm" + sfx], eps=m.rms_eps)
        qkv = proj(a, "w_qkv", sfx)
        q = qkv[:, :Hq * hd].reshape(n, Hq, hd)
        k = qkv[:, Hq * hd:(Hq + Hkv) * hd].reshape(n, Hkv, hd)
        v = qkv[:, (Hq + Hkv) * hd:].reshape(n, Hkv, hd)
        q, k = rot(q), rot(k)
        outs = []
        for s in range(p.n_seg):
            lo, hi = p.cu_seqlens[s], p.cu_seqlens[s + 1]
            tq = q[lo:hi].permute(1, 0, 2)
            tk = k[lo:hi].permute(1, 0, 2).repeat_interleave(Hq // Hkv, 0)
            tv = v[lo:hi].permute(1, 0, 2).repeat_interleave(Hq // Hkv, 0)
            outs.append(F.scaled_dot_product_attention(tq, tk, tv, is_causal=True).permute(1, 0, 2))
        o = torch.cat(outs).reshape(n, Hq * hd)
        x1 = x + proj(o, "w_o", sfx)
        b = F.rms_norm(x1, (m.d_model,), W["mlp_norm" + sfx], eps=m.rms_eps)
        gu = proj(b, "w_gate_up", sfx)
        return x1 + proj(F.silu(gu[:, :Fd]) * gu[:, Fd:], "w_down", sfx)

    y = W["emb"][torch.tensor(p.tok)]
    for layer in range(m.n_layers):
        y = block(y, "" if layer == 0 else f".{layer}")
    hn = F.rms_norm(y, (m.d_model,), W["final_norm"], eps=m.rms_eps)
    tg = torch.tensor(tgt)
    lp = torch.log_softmax(hn[tg - 1] @ W["w_vocab"].T, -1).gather(1, torch.tensor(p.tok)[tg][:, None])[:, 0]
    sel = torch.tensor(p.mask[tgt] == 1)
    r = torch.exp(lp[sel] - torch.tensor(p.old_logprob[tgt])[sel])
    A = torch.tensor(p.adv[tgt])[sel]
    loss = -torch.minimum(r * A, torch.clamp(r, 1 - m.clip_eps, 1 + m.clip_eps) * A).sum() / sel.sum()
    return lp, loss


@pytest.mark.parametrize("n_layers", [1, 3])
def test_gradients_match_torch_autograd(n_layers):
    """A torch float64 forward built from library ops, differentiated by autograd."""
    m = dataclasses.replace(SMALL, n_layers=n_layers)
    rng = np.random.default_rng(13)
    Wn = M.f64_weights(make_weights_numpy(m, seed=14, gain_std=0.3))
    p = _packed([7, 9], m.vocab, rng, mask_p=0.7)
    out = M.actor_update(p, Wn, m)
    W = {k: torch.tensor(v, requires_grad=True) for k, v in Wn.items()}
    lp, loss = _torch_loss(W, p, m, out["tgt"])
    loss.backward()
    np.testing.assert_allclose(lp.detach().numpy(), out["logprob"][out["tgt"]], atol=1e-12)
    assert abs(loss.item() - out["loss"]) < 1e-12
    for kname, t in W.items():
        np.testing.assert_allclose(out["grads"][kname], t.grad.numpy(), atol=1e-12, rtol=1e-9,
                                   err_msg=kname)


# ------------------------------------------------------------------ LoRA

@pytest.mark.parametrize("n_layers", [1, 2])
def test_lora_gradients_match_torch_autograd(n_layers):
    """Adapters written out as v W^T + scale (v A^T) B^T in torch and
    differentiated by autograd: the oracle's merged-weight form and chain
    rule give the same log-probs, loss and A/B gradients."""
    m = dataclasses.replace(SMALL, n_layers=n_layers)
    rng = np.random.default_rng(31)
    Wn = M.f64_weights(make_weights_numpy(m, seed=32, gain_std=0.3))
    Ln = {k: v.astype(np.float64) for k, v in make_lora_numpy(m, 8, seed=33, b_std=0.2).items()}
    scale = 2.0
    p = _packed([7, 9], m.vocab, rng, mask_p=0.7)
    out = M.lora_actor_update(p, Wn, Ln, scale, m)
    W = {k: torch.tensor(v) for k, v in Wn.items()}
    L = {k: torch.tensor(v, requires_grad=True) for k, v in Ln.items()}
    lp, loss = _torch_loss(W, p, m, out["tgt"], L, scale)
    loss.backward()
    np.testing.assert_allclose(lp.detach().numpy(), out["logprob"][out["tgt"]], atol=1e-12)
    assert abs(loss.item() - out["loss"]) < 1e-12
    assert set(out["grads"]) == set(L)
    for kname, t in L.items():
        np.testing.assert_allclose(out["grads"][kname], t.grad.numpy(), atol=1e-12, rtol=1e-9,
                                   err_msg=kname)


def test_lora_zero_b_is_the_base_model():
    """B = 0 (the usual start): the base model's log-probs and loss exactly, no
    gradient into A (it only reaches the loss through B)."""
    m = dataclasses.replace(SMALL, n_layers=2)
    rng = np.random.default_rng(34)
    W = M.f64_weights(make_weights_numpy(m, seed=35, gain_std=0.3))
    Ln = make_lora_numpy(m, 8, seed=36)
    p = _packed([5, 8], m.vocab, rng, mask_p=0.7)
    a = M.actor_update(p, W, m)
    b = M.lora_actor_update(p, W, Ln, 4.0, m)
    np.testing.assert_array_equal(a["logprob"], b["logprob"])
    assert a["loss"] == b["loss"]
    for k, g in b["grads"].items():
        if k.startswith("lora_a"):
            assert not np.any(g), k
        else:
            assert np.any(g), k


@pytest.mark.parametrize("name", ["lora_a.w_qkv", "lora_b.w_down.1", "lora_a.w_gate_up.1",
                                  "lora_b.w_o"])
def test_lora_gradients_match_finite_differences(name):
    m = dataclasses.replace(SMALL, n_layers=2)
    rng = np.random.default_rng(37)
    W = M.f64_weights(make_weights_numpy(m, seed=38, gain_std=0.3))
    Ln = {k: v.astype(np.float64) for k, v in make_lora_numpy(m, 8, seed=39, b_std=0.2).items()}
    p = _packed([6, 5], m.vocab, rng, mask_p=0.7)
    scale = 0.5
    out = M.lora_actor_update(p, W, Ln, scale, m, n_mask=7)
    assert np.all(np.abs(np.abs(out["ratio"] - 1) - m.clip_eps) > 1e-3)
    g = out["grads"][name]

    def loss_at(idx, h):
        L2 = {k: v.copy() for k, v in Ln.items()}
        L2[name][idx] += h
        return M.lora_actor_update(p, W, L2, scale, m, n_mask=7)["loss"]

    flat = list(np.ndindex(g.shape))
    for idx in [flat[i] for i in rng.choice(len(flat), size=min(20, len(flat)), replace=False)]:
        h = 1e-6 * max(1.0, abs(Ln[name][idx]))
        fd = (loss_at(idx, h) - loss_at(idx, -h)) / (2 * h)
        assert abs(fd - g[idx]) <= 1e-6 * max(1e-3, abs(fd)) + 1e-9, (name, idx, fd, g[idx])


@pytest.mark.parametrize("name", ["w_qkv.1", "w_down.1", "attn_norm.1", "w_o", "mlp_norm"])
def test_two_layer_gradients_match_finite_differences(name):
    m = dataclasses.replace(SMALL, n_layers=2)
    rng = np.random.default_rng(21)
    W = M.f64_weights(make_weights_numpy(m, seed=22, gain_std=0.3))
    p = _packed([6, 5], m.vocab, rng, mask_p=0.7)
    out = M.actor_update(p, W, m, n_mask=7)
    assert np.all(np.abs(np.abs(out["ratio"] - 1) - m.clip_eps) > 1e-3)
    g = out["grads"][name]
    flat = list(np.ndindex(g.shape))
    for idx in [flat[i] for i in rng.choice(len(flat), size=min(25, len(flat)), replace=False)]:
        h = 1e-6 * max(1.0, abs(W[name][idx]))
        fd = (_loss_with(p, W, m, name, idx, h) - _loss_with(p, W, m, name, idx, -h)) / (2 * h)
        assert abs(fd - g[idx]) <= 1e-6 * max(1e-3, abs(fd)) + 1e-9, (name, idx, fd, g[idx])


def test_identity_layers_leave_the_model_unchanged():
    """Layers whose output and down projections are zero pass x through: a
    3-layer stack with two such layers is the 1-layer model exactly."""
    m1 = SMALL
    m3 = dataclasses.replace(SMALL, n_layers=3)
    rng = np.random.default_rng(23)
    W3 = M.f64_weights(make_weights_numpy(m3, seed=24, gain_std=0.3))
    for layer in (1, 2):
        W3[f"w_o.{layer}"][:] = 0.0
        W3[f"w_down.{layer}"][:] = 0.0
    W1 = {k: v for k, v in W3.items() if "." not in k}
    p = _packed([8, 3, 6], m1.vocab, rng, mask_p=0.7)
    a, b = M.actor_update(p, W1, m1), M.actor_update(p, W3, m3)
    np.testing.assert_array_equal(a["logprob"], b["logprob"])
    assert a["loss"] == b["loss"]
    for k in W1:
        np.testing.assert_array_equal(a["grads"][k], b["grads"][k], err_msg=k)
    # nothing flows into the zeroed branches' inputs
    for layer in (1, 2):
        assert not np.any(b["grads"][f"w_qkv.{layer}"]) and not np.any(b["grads"][f"w_gate_up.{layer}"])


# ------------------------------------------------------------------ merged == unmerged

def _tiny_pair():
    cfg = get_config(0)
    m = cfg.model
    tl = make_timelines(cfg)
    W = make_weights_numpy(m)
    zero = np.zeros(tl.n_tok, np.float32)
    un = om.unmerged_batch(om.episodes_from_flat(tl.traj_tl_off, tl.tl_tok_off, tl.tok, tl.flags,
                                                 zero, tl.adv))
    cur = M.current_logprob(un, W, m)
    old = np.where((tl.flags & 3) == 2, cur + tl.lp_noise, 0.0)
    eps = om.episodes_from_flat(tl.traj_tl_off, tl.tl_tok_off, tl.tok, tl.flags, old, tl.adv)
    return m, W, om.merge_batch(eps)[0], om.unmerged_batch(eps), tl


def test_merged_equals_unmerged_on_tiny():
    m, W, mg, un, tl = _tiny_pair()
    assert mg.n_tok < un.n_tok
    a = M.actor_update(mg, W, m)
    b = M.actor_update(un, W, m)
    assert a["n_mask"] == b["n_mask"] == int(((tl.flags & 3) == 2).sum())
    assert abs(a["loss"] - b["loss"]) <= 1e-10 * max(1.0, abs(b["loss"]))
    # per response token: the old log-prob identifies it in both layouts
    ka = np.argsort(mg.old_logprob[mg.mask == 1])
    kb = np.argsort(un.old_logprob[un.mask == 1])
    np.testing.assert_allclose(a["logprob"][mg.mask == 1][ka], b["logprob"][un.mask == 1][kb], atol=1e-10)
    for k in a["grads"]:
        ga, gb = a["grads"][k], b["grads"][k]
        assert np.linalg.norm(ga - gb) <= 1e-9 * np.linalg.norm(gb), k


def test_unmasked_inputs_do_not_matter():
    """Changing old log-probs / advantages on unmasked tokens changes nothing, bit for bit."""
    m, W, mg, un, tl = _tiny_pair()
    a = M.actor_update(mg, W, m)
    rng = np.random.default_rng(15)
    off = mg.mask == 0
    mg.old_logprob = np.where(off, rng.normal(size=mg.n_tok), mg.old_logprob)
    mg.adv = np.where(off, rng.normal(size=mg.n_tok), mg.adv)
    b = M.actor_update(mg, W, m)
    assert a["loss"] == b["loss"]
    for k in a["grads"]:
        np.testing.assert_array_equal(a["grads"][k], b["grads"][k])


def test_rows_after_last_masked_target_get_zero_gradient():
    m, W, mg, un, tl = _tiny_pair()
    out = M.actor_update(mg, W, m)
    for s in range(mg.n_seg):
        lo, hi = mg.cu_seqlens[s], mg.cu_seqlens[s + 1]
        mk = np.flatnonzero(mg.mask[lo + 1:hi]) + lo + 1
        last = mk.max() if len(mk) else lo
        # hidden rows at or after the last masked target only feed later targets
        assert not np.any(out["dx"][last:hi])


def test_block_forward_rows_matches_full():
    m = SMALL
    rng = np.random.default_rng(16)
    W = M.f64_weights(make_weights_numpy(m, seed=17))
    p = _packed([13], m.vocab, rng)
    x = W["emb"][p.tok]
    y, _ = M.block_forward(x, W, p.cu_seqlens, p.pos, m)
    rows = np.array([0, 4, 12])
    np.testing.assert_allclose(M.block_forward_rows(x, p.pos, rows, W, m), y[rows], atol=1e-13)


# ------------------------------------------------------------------ KL penalty

def test_kl_estimate_is_unbiased_for_the_divergence():
    """Averaged over tokens drawn from the policy, exp(d) - d - 1 with
    d = log pi_ref - log pi is exactly KL(pi || pi_ref) (scipy's rel_entr);
    a flipped sign or a missing term breaks the identity."""
    from scipy.special import rel_entr, log_softmax
    rng = np.random.default_rng(3)
    for _ in range(5):
        z = rng.normal(0, 1.5, 50)
        lp = log_softmax(z)
        ref = log_softmax(z + rng.normal(0, 0.5, 50))
        kl, _ = M.kl_terms(lp, ref)
        assert np.all(kl < 10)
        np.testing.assert_allclose(np.sum(np.exp(lp) * kl), np.sum(rel_entr(np.exp(lp), np.exp(ref))),
                                   rtol=1e-12, atol=1e-14)


def test_kl_closed_forms():
    d = np.array([0.0, 1e-4, -1e-4, 40.0])
    lp = np.full(4, -2.0)
    kl, dkl = M.kl_terms(lp, lp + d)
    assert kl[0] == 0.0 and dkl[0] == 0.0
    np.testing.assert_allclose(kl[1:3], d[1:3] ** 2 / 2, rtol=1e-3)   # second order at 0
    np.testing.assert_allclose(dkl[1:3], -d[1:3], rtol=1e-3)
    assert kl[3] == 10.0 and dkl[3] == 0.0                              # the clamp binds


@pytest.mark.parametrize("name", ["w_o", "final_norm", "w_vocab"])
def test_kl_gradients_match_finite_differences(name):
    m = SMALL
    rng = np.random.default_rng(21)
    W = M.f64_weights(make_weights_numpy(m, seed=12, gain_std=0.3))
    p = _packed([6, 5, 4], m.vocab, rng, mask_p=0.7)
    ref = rng.normal(-3.0, 0.7, p.n_tok)
    out = M.actor_update(p, W, m, n_mask=7, ref_logprob=ref, kl_coef=0.37)
    assert np.all(np.abs(np.abs(out["ratio"] - 1) - m.clip_eps) > 1e-3)
    assert np.any(out["kl"] > 0)
    g = out["grads"][name]
    flat = list(np.ndindex(g.shape))

    def loss(h, idx):
        W2 = {k: v.copy() for k, v in W.items()}
        W2[name][idx] += h
        return M.actor_update(p, W2, m, n_mask=7, ref_logprob=ref, kl_coef=0.37)["loss"]

    for idx in [flat[i] for i in rng.choice(len(flat), size=min(25, len(flat)), replace=False)]:
        h = 1e-6 * max(1.0, abs(W[name][idx]))
        fd = (loss(h, idx) - loss(-h, idx)) / (2 * h)
        assert abs(fd - g[idx]) <= 1e-6 * max(1e-3, abs(fd)) + 1e-9, (name, idx, fd, g[idx])


def test_kl_coef_zero_is_the_plain_loss():
    m = SMALL
    rng = np.random.default_rng(5)
    W = M.f64_weights(make_weights_numpy(m, seed=12, gain_std=0.3))
    p = _packed([7, 5], m.vocab, rng)
    a = M.actor_update(p, W, m)
    b = M.actor_update(p, W, m, ref_logprob=rng.normal(-3, 1, p.n_tok), kl_coef=0.0)
    assert a["loss"] == b["loss"]
    for k in a["grads"]:
        assert np.array_equal(a["grads"][k], b["grads"][k])
