"""Tolerance model for the bfloat16 path at large shapes (test infrastructure).

The actor update in bfloat16 stores every activation that feeds a matrix
core, or that is kept between kernels, as bfloat16 with float32 accumulation
(round to nearest even).  Those roundings alone move a token log-prob by an
amount that grows with the model width and the context length.  This module
re-runs the oracle's float64 arithmetic for one segment, at given rows only
(as oracle.model.block_forward_rows does), with a bfloat16 rounding at each
such storage point:

    a = rmsnorm(x) g1,  q/k/v = a W_qkv^T,  q/k after RoPE,  the softmax
    weights that multiply V,  o,  x1 = x + o W_o^T,  b = rmsnorm(x1) g2,
    [gate | up],  s = silu(gate) up,  y = x1 + s W_down^T,  hn = rmsnorm(y) gf

The spread of (this model - the float64 oracle) over sampled targets is
the yardstick the GPU's own error is held to.  It models magnitudes, not the
GPU's exact bits: the GPU rounds the softmax weights against a running
maximum, tile by tile, so individual errors differ.
"""
import numpy as np

from oracle import model as M


def bf16(x):
    """Round to bfloat16 (nearest even) and return as float64."""
    u = np.asarray(x, np.float32).view(np.uint32).astype(np.uint64)
    u = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16) << 16
    return u.astype(np.uint32).view(np.float32).astype(np.float64)


def block_logprob_rows_rounded(x_seg, pos_seg, rows, tok_next, W, m):
    """Log-prob of tok_next[i] from row rows[i] of one segment, with the
    bfloat16 storage roundings listed above (W: float64 copies of bfloat16
    weights)."""
    rows = np.asarray(rows, np.int64)
    Hq, Hkv, hd, F = m.n_q_heads, m.n_kv_heads, m.head_dim, m.d_ff
    L = int(rows.max()) + 1
    x = np.asarray(x_seg[:L], np.float64)
    a, _ = M.rmsnorm(x, W["attn_norm"], m.rms_eps)
    a = bf16(a)
    kv = bf16(a @ W["w_qkv"][Hq * hd:].T)
    k_raw, v = kv[:, :Hkv * hd], kv[:, Hkv * hd:].reshape(L, Hkv, hd)
    q_raw = bf16(a[rows] @ W["w_qkv"][:Hq * hd].T)
    cos, sin = M.rope_angles(pos_seg[:L], hd, m.rope_theta)
    k = bf16(M.rope(k_raw.reshape(L, Hkv, hd), cos, sin))
    q = bf16(M.rope(q_raw.reshape(len(rows), Hq, hd), cos[rows], sin[rows]))
    scale = 1.0 / np.sqrt(hd)
    o = np.zeros((len(rows), Hq, hd))
    for h in range(Hq):
        g = M.kv_head(h, Hq, Hkv)
        s = (q[:, h, :] @ k[:, g, :].T) * scale
        s = np.where(np.arange(L)[None, :] <= rows[:, None], s, -np.inf)
        p = np.exp(s - s.max(axis=1)[:, None])
        o[:, h, :] = (bf16(p) @ v[:, g, :]) / p.sum(axis=1)[:, None]
    o = bf16(o.reshape(len(rows), -1))
    x1 = bf16(x[rows] + o @ W["w_o"].T)
    b, _ = M.rmsnorm(x1, W["mlp_norm"], m.rms_eps)
    gu = bf16(bf16(b) @ W["w_gate_up"].T)
    s_ = bf16(M.silu(gu[:, :F]) * gu[:, F:])
    y = bf16(x1 + s_ @ W["w_down"].T)
    hn, _ = M.rmsnorm(y, W["final_norm"], m.rms_eps)
    z = bf16(hn) @ W["w_vocab"].T
    zm = z.max(axis=1)
    lse = zm + np.log(np.sum(np.exp(z - zm[:, None]), axis=1))
    return z[np.arange(len(rows)), tok_next] - lse
