"""Decoder block(s) + LM head + clipped policy-gradient loss, float64, forward
and backward -- test infrastructure only.

What is computed (the policy is a one-block Qwen2-style decoder; the paper
trains Qwen2/Qwen2.5/Qwen3 models and defines no architecture, so these are
readings):
  x   = E[tok]
  a   = RMSNorm(x) * g1                     RMSNorm(v) = v / sqrt(mean(v^2) + eps)
  q,k,v = a W_qkv^T, split by heads; rotate-half RoPE on q and k at the token's
        position inside its segment, inverse frequencies theta^(-2i/hd)
  o   = causal softmax(q k^T / sqrt(hd)) v inside each segment; query head h
        reads key/value head floor(h * Hkv / Hq)
  x1  = x + o W_o^T
  b   = RMSNorm(x1) * g2
  y   = x1 + (silu(b W_gate^T) * (b W_up^T)) W_down^T
        (with n_layers > 1 the block repeats, each layer with its own weights,
        the output of one the input of the next: step (4) of Section 4.2
        updates the whole model; the repetition is the standard decoder stack)
  hn  = RMSNorm(y) * gf
  logprob[p] = log softmax(hn[p-1] W_vocab^T)[tok[p]]  for p after its segment's start
The loss is GRPO's clipped surrogate (Section 3 cites GRPO-style updates; the
clip ratio 0.2 is the one the AIME case study in Section 6 uses), averaged over
the loss-masked tokens of the whole batch:
  r = exp(logprob - old_logprob)
  L = sum_mask -min(r A, clip(r, 1-eps, 1+eps) A) / N_mask
Its gradient with respect to logprob is -A r / N_mask where the unclipped
branch is the active one -- (A > 0 and r <= 1+eps) or (A < 0 and r >= 1-eps),
ties counting as unclipped -- and 0 elsewhere.

Optional KL penalty against a frozen reference policy (Section 6's GRPO
recipe names a KL loss with coefficient 2e-3 and the "low_var_kl"
estimator; the paper gives no formula, so this is a reading: the k3
estimator of KL(pi || pi_ref) at the sampled token, clamped to [-10, 10]):
  delta = ref_logprob - logprob,   kl = exp(delta) - delta - 1
  L += kl_coef * sum_mask kl / N_mask,   d kl / d logprob = 1 - exp(delta)
(zero where the clamp binds).

LoRA (Section 4.2, step (4): the update trains "either the full model weights
or the LoRA matrix weights", citing Hu et al.): every block projection
W in {W_qkv, W_o, W_gate_up, W_down} of every layer is used as
  W_eff = W + scale * B A,   A [rank, in], B [out, rank],
with only A and B trained (norm gains, embedding and LM head frozen).  The
oracle runs the model with W_eff and takes A's and B's gradients from
W_eff's by the chain rule: dA = scale B^T dW_eff, dB = scale dW_eff A^T.

The backward pass is written out by hand from these formulas.
"""
import numpy as np

from workloads import BLOCK_WEIGHTS, LORA_PROJ, layer_key, lora_key


# ---------------------------------------------------------------- pieces

def rmsnorm(x, g, eps):
    r = 1.0 / np.sqrt(np.mean(x * x, axis=-1) + eps)
    return x * r[:, None] * g[None, :], r


def rmsnorm_bwd(dy, x, r, g):
    gdy = dy * g[None, :]
    dx = r[:, None] * (gdy - x * (r * r)[:, None] * np.mean(gdy * x, axis=-1)[:, None])
    dg = np.sum(dy * x * r[:, None], axis=0)
    return dx, dg


def rope_angles(pos, head_dim, theta):
    half = head_dim // 2
    inv_freq = theta ** (-(2.0 * np.arange(half, dtype=np.float64)) / head_dim)
    ang = np.asarray(pos, np.float64)[:, None] * inv_freq[None, :]
    return np.cos(ang), np.sin(ang)


def rope(x, cos, sin):
    """x [n, H, hd]: rotate (x_i, x_{i+hd/2}) by the angle of pair i."""
    half = x.shape[-1] // 2
    x1, x2 = x[..., :half], x[..., half:]
    c, s = cos[:, None, :], sin[:, None, :]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def rope_bwd(dy, cos, sin):
    half = dy.shape[-1] // 2
    d1, d2 = dy[..., :half], dy[..., half:]
    c, s = cos[:, None, :], sin[:, None, :]
    return np.concatenate([d1 * c + d2 * s, -d1 * s + d2 * c], axis=-1)


def silu(v):
    return v / (1.0 + np.exp(-v))


def kv_head(h, n_q, n_kv):
    return (h * n_kv) // n_q


def attention_segment(q, k, v, scale):
    """Causal attention of one segment. q [L,Hq,hd], k/v [L,Hkv,hd] -> o [L,Hq,hd], lse [Hq,L]."""
    L, Hq, hd = q.shape
    Hkv = k.shape[1]
    o = np.zeros_like(q)
    lse = np.zeros((Hq, L))
    causal = np.tril(np.ones((L, L), dtype=bool))
    for h in range(Hq):
        g = kv_head(h, Hq, Hkv)
        s = (q[:, h, :] @ k[:, g, :].T) * scale
        s = np.where(causal, s, -np.inf)
        m = s.max(axis=1)
        p = np.exp(s - m[:, None])
        l = p.sum(axis=1)
        o[:, h, :] = (p / l[:, None]) @ v[:, g, :]
        lse[h] = m + np.log(l)
    return o, lse


def attention_segment_bwd(q, k, v, o, lse, do, scale):
    L, Hq, hd = q.shape
    Hkv = k.shape[1]
    dq = np.zeros_like(q)
    dk = np.zeros_like(k)
    dv = np.zeros_like(v)
    causal = np.tril(np.ones((L, L), dtype=bool))
    for h in range(Hq):
        g = kv_head(h, Hq, Hkv)
        s = (q[:, h, :] @ k[:, g, :].T) * scale
        p = np.where(causal, np.exp(s - lse[h][:, None]), 0.0)
        dp = do[:, h, :] @ v[:, g, :].T
        D = np.sum(do[:, h, :] * o[:, h, :], axis=1)
        ds = p * (dp - D[:, None])
        dq[:, h, :] = (ds @ k[:, g, :]) * scale
        dk[:, g, :] += (ds.T @ q[:, h, :]) * scale
        dv[:, g, :] += p.T @ do[:, h, :]
    return dq, dk, dv


def log_softmax_rows(z):
    m = z.max(axis=1)
    return z - (m + np.log(np.sum(np.exp(z - m[:, None]), axis=1)))[:, None]


def pg_terms(logprob, old, adv, eps):
    """Per-token clipped surrogate term and d term / d logprob (unnormalised)."""
    r = np.exp(logprob - old)
    term = -np.minimum(r * adv, np.clip(r, 1.0 - eps, 1.0 + eps) * adv)
    active = ((adv > 0) & (r <= 1.0 + eps)) | ((adv < 0) & (r >= 1.0 - eps))
    dterm = np.where(active, -adv * r, 0.0)
    return term, dterm, r


def kl_terms(logprob, ref_logprob):
    """Per-token low-variance KL estimate and its derivative with respect to logprob."""
    delta = ref_logprob - logprob
    e = np.exp(delta)
    kl = e - delta - 1.0
    inside = (kl >= -10.0) & (kl <= 10.0)
    return np.clip(kl, -10.0, 10.0), np.where(inside, 1.0 - e, 0.0)


def target_positions(cu_seqlens, n_tok):
    """Positions p that have a predecessor in their own segment."""
    starts = np.zeros(n_tok, dtype=bool)
    starts[np.asarray(cu_seqlens[:-1], np.int64)[np.asarray(cu_seqlens[:-1]) < n_tok]] = True
    return np.flatnonzero(~starts)


# ---------------------------------------------------------------- full pass

def f64_weights(W):
    return {k: np.asarray(v, np.float64) for k, v in W.items()}


def block_forward(x, W, cu_seqlens, pos, m):
    n = x.shape[0]
    Hq, Hkv, hd, F = m.n_q_heads, m.n_kv_heads, m.head_dim, m.d_ff
    c = {"x": x}
    a, r1 = rmsnorm(x, W["attn_norm"], m.rms_eps)
    qkv = a @ W["w_qkv"].T
    q = qkv[:, :Hq * hd].reshape(n, Hq, hd)
    k = qkv[:, Hq * hd:(Hq + Hkv) * hd].reshape(n, Hkv, hd)
    v = qkv[:, (Hq + Hkv) * hd:].reshape(n, Hkv, hd)
    cos, sin = rope_angles(pos, hd, m.rope_theta)
    qr, kr = rope(q, cos, sin), rope(k, cos, sin)
    o = np.zeros((n, Hq, hd))
    lse = np.zeros((Hq, n))
    scale = 1.0 / np.sqrt(hd)
    for s in range(len(cu_seqlens) - 1):
        lo, hi = int(cu_seqlens[s]), int(cu_seqlens[s + 1])
        if hi > lo:
            o[lo:hi], lse[:, lo:hi] = attention_segment(qr[lo:hi], kr[lo:hi], v[lo:hi], scale)
    of = o.reshape(n, Hq * hd)
    x1 = x + of @ W["w_o"].T
    b, r2 = rmsnorm(x1, W["mlp_norm"], m.rms_eps)
    gu = b @ W["w_gate_up"].T
    gate, up = gu[:, :F], gu[:, F:]
    sact = silu(gate) * up
    y = x1 + sact @ W["w_down"].T
    c.update(a=a, r1=r1, qr=qr, kr=kr, v=v, cos=cos, sin=sin, o=o, lse=lse, x1=x1,
             b=b, r2=r2, gate=gate, up=up, s=sact, scale=scale)
    return y, c


def block_backward(dy, c, W, cu_seqlens, m):
    n = dy.shape[0]
    Hq, Hkv, hd = m.n_q_heads, m.n_kv_heads, m.head_dim
    g = {}
    dx1 = dy.copy()
    g["w_down"] = dy.T @ c["s"]
    ds = dy @ W["w_down"]
    sg = 1.0 / (1.0 + np.exp(-c["gate"]))
    dup = ds * c["gate"] * sg
    dgate = ds * c["up"] * sg * (1.0 + c["gate"] * (1.0 - sg))
    dgu = np.concatenate([dgate, dup], axis=1)
    g["w_gate_up"] = dgu.T @ c["b"]
    db = dgu @ W["w_gate_up"]
    dx1_n, g["mlp_norm"] = rmsnorm_bwd(db, c["x1"], c["r2"], W["mlp_norm"])
    dx1 += dx1_n
    of = c["o"].reshape(n, Hq * hd)
    g["w_o"] = dx1.T @ of
    do = (dx1 @ W["w_o"]).reshape(n, Hq, hd)
    dqr = np.zeros((n, Hq, hd))
    dkr = np.zeros((n, Hkv, hd))
    dv = np.zeros((n, Hkv, hd))
    for s in range(len(cu_seqlens) - 1):
        lo, hi = int(cu_seqlens[s]), int(cu_seqlens[s + 1])
        if hi > lo:
            dqr[lo:hi], dkr[lo:hi], dv[lo:hi] = attention_segment_bwd(
                c["qr"][lo:hi], c["kr"][lo:hi], c["v"][lo:hi], c["o"][lo:hi],
                c["lse"][:, lo:hi], do[lo:hi], c["scale"])
    dq = rope_bwd(dqr, c["cos"], c["sin"])
    dk = rope_bwd(dkr, c["cos"], c["sin"])
    dqkv = np.concatenate([dq.reshape(n, -1), dk.reshape(n, -1), dv.reshape(n, -1)], axis=1)
    g["w_qkv"] = dqkv.T @ c["a"]
    da = dqkv @ W["w_qkv"]
    dx_n, g["attn_norm"] = rmsnorm_bwd(da, c["x"], c["r1"], W["attn_norm"])
    dx = dx1 + dx_n
    return dx, g


def layer_weights(W, layer):
    return {name: W[layer_key(name, layer)] for name in BLOCK_WEIGHTS}


def stack_forward(x, W, cu_seqlens, pos, m):
    """The m.n_layers blocks in order; returns the last output and every layer's cache."""
    caches = []
    for layer in range(m.n_layers):
        x, c = block_forward(x, layer_weights(W, layer), cu_seqlens, pos, m)
        caches.append(c)
    return x, caches


def stack_backward(dy, caches, W, cu_seqlens, m):
    """The blocks in reverse; gradients keyed like the weights."""
    g = {}
    for layer in reversed(range(m.n_layers)):
        dy, gl = block_backward(dy, caches[layer], layer_weights(W, layer), cu_seqlens, m)
        for name, v in gl.items():
            g[layer_key(name, layer)] = v
    return dy, g


def lm_head_forward(y, W, tok, tgt, m, row_chunk=2048):
    """Final norm, then log-prob of tok[p] from row p-1, for the target positions `tgt`.

    Returns (hn, rf, logprob_tgt, lse_tgt).
    """
    hn, rf = rmsnorm(y, W["final_norm"], m.rms_eps)
    lp = np.zeros(len(tgt))
    lse = np.zeros(len(tgt))
    for s in range(0, len(tgt), row_chunk):
        t = tgt[s:s + row_chunk]
        z = hn[t - 1] @ W["w_vocab"].T
        zm = z.max(axis=1)
        lse[s:s + len(t)] = zm + np.log(np.sum(np.exp(z - zm[:, None]), axis=1))
        lp[s:s + len(t)] = z[np.arange(len(t)), tok[t]] - lse[s:s + len(t)]
    return hn, rf, lp, lse


def lm_head_backward(dlp, hn, rf, y, W, tok, tgt, lse, m, row_chunk=2048):
    """d/d(y, final_norm, w_vocab) given d loss / d logprob at the targets."""
    dhn = np.zeros_like(hn)
    dWv = np.zeros_like(W["w_vocab"])
    for s in range(0, len(tgt), row_chunk):
        t = tgt[s:s + row_chunk]
        h = hn[t - 1]
        z = h @ W["w_vocab"].T
        p = np.exp(z - lse[s:s + len(t)][:, None])
        dz = -dlp[s:s + len(t)][:, None] * p
        dz[np.arange(len(t)), tok[t]] += dlp[s:s + len(t)]
        np.add.at(dhn, t - 1, dz @ W["w_vocab"])
        dWv += dz.T @ h
    dy, dgf = rmsnorm_bwd(dhn, y, rf, W["final_norm"])
    return dy, dgf, dWv


def actor_update(packed, W, m, n_mask=None, ref_logprob=None, kl_coef=0.0):
    """Forward + backward of the whole actor update over one packed batch.

    packed: oracle.merge.Packed (tok, pos, mask, old_logprob, adv, cu_seqlens).
    W: weights (any float dtype; used as float64).  n_mask: the loss
    normaliser, default the batch's own count of masked targets.
    ref_logprob: optional [n_tok] reference-policy log-probs (read at the
    masked targets) for the KL penalty with weight kl_coef.
    Returns dict: logprob [n_tok] (NaN at segment starts), loss, n_mask,
    grads {name: array} including 'emb', plus 'dx' (grad wrt the embeddings
    gathered per token) and per-target 'lse'.
    """
    W = f64_weights(W)
    tok = packed.tok
    n = packed.n_tok
    tgt = target_positions(packed.cu_seqlens, n)
    masked = tgt[packed.mask[tgt] == 1]
    if n_mask is None:
        n_mask = len(masked)
    x = W["emb"][tok]
    y, c = stack_forward(x, W, packed.cu_seqlens, packed.pos, m)
    hn, rf, lp_t, lse_t = lm_head_forward(y, W, tok, tgt, m)
    logprob = np.full(n, np.nan)
    logprob[tgt] = lp_t
    sel = packed.mask[tgt] == 1
    term, dterm, r = pg_terms(lp_t[sel], packed.old_logprob[tgt][sel], packed.adv[tgt][sel],
                              m.clip_eps)
    kl = np.zeros(len(term))
    if ref_logprob is not None and kl_coef != 0.0:
        kl, dkl = kl_terms(lp_t[sel], np.asarray(ref_logprob, np.float64)[tgt][sel])
        term = term + kl_coef * kl
        dterm = dterm + kl_coef * dkl
    loss = float(np.sum(term) / n_mask) if n_mask else 0.0
    dlp = np.zeros(len(tgt))
    if n_mask:
        dlp[sel] = dterm / n_mask
    dy, dgf, dWv = lm_head_backward(dlp, hn, rf, y, W, tok, tgt, lse_t, m)
    dx, g = stack_backward(dy, c, W, packed.cu_seqlens, m)
    g["final_norm"] = dgf
    g["w_vocab"] = dWv
    dE = np.zeros_like(W["emb"])
    np.add.at(dE, tok, dx)
    g["emb"] = dE
    return {"logprob": logprob, "loss": loss, "n_mask": n_mask, "grads": g, "dx": dx,
            "dy": dy, "y": y, "tgt": tgt, "lse": lse_t, "ratio": r, "term": term,
            "kl": kl}


def lora_effective(W, lora, scale, m):
    """The weights with every adapted projection replaced by W + scale B A."""
    W = f64_weights(W)
    for layer in range(m.n_layers):
        for proj in LORA_PROJ:
            A = np.asarray(lora[lora_key("a", proj, layer)], np.float64)
            B = np.asarray(lora[lora_key("b", proj, layer)], np.float64)
            W[layer_key(proj, layer)] = W[layer_key(proj, layer)] + scale * (B @ A)
    return W


def lora_actor_update(packed, W, lora, scale, m, n_mask=None):
    """actor_update with LoRA adapters; grads holds the adapters' gradients only."""
    out = actor_update(packed, lora_effective(W, lora, scale, m), m, n_mask=n_mask)
    g = {}
    for layer in range(m.n_layers):
        for proj in LORA_PROJ:
            dW = out["grads"][layer_key(proj, layer)]
            A = np.asarray(lora[lora_key("a", proj, layer)], np.float64)
            B = np.asarray(lora[lora_key("b", proj, layer)], np.float64)
            g[lora_key("a", proj, layer)] = scale * (B.T @ dW)
            g[lora_key("b", proj, layer)] = scale * (dW @ A.T)
    out["grads"] = g
    return out


def current_logprob(packed, W, m):
    """Log-probs of every target under W (forward only); NaN at segment starts."""
    W = f64_weights(W)
    x = W["emb"][packed.tok]
    y, _ = stack_forward(x, W, packed.cu_seqlens, packed.pos, m)
    tgt = target_positions(packed.cu_seqlens, packed.n_tok)
    _, _, lp, _ = lm_head_forward(y, W, packed.tok, tgt, m)
    out = np.full(packed.n_tok, np.nan)
    out[tgt] = lp
    return out


def block_forward_rows(x_seg, pos_seg, rows, W, m):
    """Block output y at `rows` of one segment (only the prefix up to max(rows) is read).

    Same arithmetic as block_forward restricted to the rows asked for: keys and
    values of every earlier position of the segment, everything else only at
    `rows`.  Used to check outputs of very long segments one row at a time.
    """
    if m.n_layers != 1:
        raise ValueError("block_forward_rows follows one block")
    W = f64_weights(W)
    rows = np.asarray(rows, np.int64)
    Hq, Hkv, hd, F = m.n_q_heads, m.n_kv_heads, m.head_dim, m.d_ff
    L = int(rows.max()) + 1
    x = np.asarray(x_seg[:L], np.float64)
    a, _ = rmsnorm(x, W["attn_norm"], m.rms_eps)
    wq = W["w_qkv"][:Hq * hd]
    wk = W["w_qkv"][Hq * hd:(Hq + Hkv) * hd]
    wv = W["w_qkv"][(Hq + Hkv) * hd:]
    cos, sin = rope_angles(pos_seg[:L], hd, m.rope_theta)
    k = rope((a @ wk.T).reshape(L, Hkv, hd), cos, sin)
    v = (a @ wv.T).reshape(L, Hkv, hd)
    q = rope((a[rows] @ wq.T).reshape(len(rows), Hq, hd), cos[rows], sin[rows])
    scale = 1.0 / np.sqrt(hd)
    o = np.zeros((len(rows), Hq, hd))
    for h in range(Hq):
        g = kv_head(h, Hq, Hkv)
        s = (q[:, h, :] @ k[:, g, :].T) * scale
        s = np.where(np.arange(L)[None, :] <= rows[:, None], s, -np.inf)
        p = np.exp(s - s.max(axis=1)[:, None])
        o[:, h, :] = (p / p.sum(axis=1)[:, None]) @ v[:, g, :]
    x1 = x[rows] + o.reshape(len(rows), -1) @ W["w_o"].T
    b, _ = rmsnorm(x1, W["mlp_norm"], m.rms_eps)
    gu = b @ W["w_gate_up"].T
    y = x1 + (silu(gu[:, :F]) * gu[:, F:]) @ W["w_down"].T
    return y
