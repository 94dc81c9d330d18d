"""ctypes binding of libaj (include/aj.h): same names, argument marshalling only.

Every function takes torch tensors (device memory owned by torch), passes
their data pointers and the current HIP stream to the library, and raises
AjError on a non-OK status.  No arithmetic happens here.
"""
import ctypes as C
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libaj.so")

AJ_F32, AJ_BF16 = 0, 1
AUTHOR_LLM = 2
FLAG_BLOCK_START = 4


class AjError(RuntimeError):
    pass


def _load():
    if not os.path.exists(LIB_PATH):
        raise AjError(f"{LIB_PATH} is missing: build it with `python -m paper_2606_04484_amd.build`")
    return C.CDLL(LIB_PATH)


_lib = None


def lib():
    global _lib
    if _lib is None:
        _lib = _load()
        _declare(_lib)
    return _lib


vp = C.c_void_p
i32, i64, f32, sz = C.c_int32, C.c_int64, C.c_float, C.c_size_t


class Timelines(C.Structure):
    _fields_ = [("n_traj", i32), ("n_tl", i32), ("n_tok", i64), ("traj_tl_off", vp),
                ("tl_tok_off", vp), ("tok", vp), ("flags", vp), ("old_logprob", vp), ("adv", vp)]


class Packed(C.Structure):
    _fields_ = [("absorber", vp), ("cu_seqlens", vp), ("seg_src", vp), ("cu_targets", vp),
                ("counts", vp), ("tok", vp), ("pos", vp), ("mask", vp), ("old_logprob", vp),
                ("adv", vp), ("targets", vp)]


class BlockTexts(C.Structure):
    _fields_ = [("n_blk", i32), ("key", vp)]


class TimelinesOut(C.Structure):
    _fields_ = [("traj_tl_off", vp), ("tl_tok_off", vp), ("tok", vp), ("flags", vp),
                ("old_logprob", vp), ("adv", vp), ("counts", vp)]


class BlockCfg(C.Structure):
    _fields_ = [("d_model", i32), ("n_q_heads", i32), ("n_kv_heads", i32), ("head_dim", i32),
                ("d_ff", i32), ("rms_eps", f32), ("rope_theta", f32), ("dtype", i32)]


BLOCK_TRANSPOSED = ("w_qkv_t", "w_o_t", "w_gate_up_t", "w_down_t")


class BlockWeights(C.Structure):
    _fields_ = [(n, vp) for n in ("attn_norm", "w_qkv", "w_o", "mlp_norm", "w_gate_up", "w_down")
                + BLOCK_TRANSPOSED]


class BlockGrads(C.Structure):
    _fields_ = [(n, vp) for n in ("attn_norm", "w_qkv", "w_o", "mlp_norm", "w_gate_up", "w_down")]


LORA_FIELDS = ("a_qkv", "b_qkv", "a_o", "b_o", "a_gate_up", "b_gate_up", "a_down", "b_down")


class Lora(C.Structure):
    _fields_ = [("rank", i32), ("scale", f32)] + [(n, vp) for n in LORA_FIELDS]


class LoraGrads(C.Structure):
    _fields_ = [(n, vp) for n in LORA_FIELDS]


class Varlen(C.Structure):
    _fields_ = [("n_tok", i32), ("n_seg", i32), ("max_seqlen", i32), ("base", i32),
                ("cu_seqlens", vp), ("pos", vp)]


class LossCfg(C.Structure):
    _fields_ = [("d_model", i32), ("vocab", i32), ("vocab_chunk", i32), ("clip_eps", f32),
                ("rms_eps", f32), ("dtype", i32), ("keep_logits", i32)]


class LossIn(C.Structure):
    _fields_ = [("n_tok", i32), ("n_tgt", i32), ("row_base", i32), ("targets", vp), ("tok", vp),
                ("old_logprob", vp), ("adv", vp), ("inv_n_mask", f32), ("ref_logprob", vp),
                ("kl_coef", f32), ("w_vocab_t", vp)]


EXPORTS = {
    "aj_status_str": (C.c_char_p, [C.c_int]),
    "aj_last_error": (C.c_char_p, []),
    "aj_read_device_error": (C.c_int, [vp, vp, C.POINTER(i32)]),
    "aj_merge_workspace_bytes": (sz, [i32, i32, i64]),
    "aj_merge_timelines": (C.c_int, [C.POINTER(Timelines), C.POINTER(Packed), vp, vp, sz, vp]),
    "aj_flatten_timelines": (C.c_int, [C.POINTER(Timelines), C.POINTER(Packed), vp, vp, sz, vp]),
    "aj_merge_noalloc_max_workspace_bytes": (sz, []),
    "aj_merge_timelines_noalloc": (C.c_int, [C.POINTER(Timelines), C.POINTER(Packed), vp, vp]),
    "aj_merge_text_workspace_bytes": (sz, [i32, i32, i64, i32]),
    "aj_merge_timelines_text": (C.c_int, [C.POINTER(Timelines), C.POINTER(BlockTexts),
                                          C.POINTER(Packed), vp, vp, vp, sz, vp]),
    "aj_plan_packs": (C.c_int, [vp, i32, i32, vp, C.POINTER(i32)]),
    "aj_embed_fwd": (C.c_int, [vp, i32, vp, i32, i32, C.c_int, vp, vp, vp]),
    "aj_embed_bwd_workspace_bytes": (sz, [i32, i32]),
    "aj_embed_bwd": (C.c_int, [vp, i32, vp, i32, i32, vp, vp, sz, vp]),
    "aj_block_saved_bytes": (sz, [C.POINTER(BlockCfg), i32]),
    "aj_block_workspace_bytes": (sz, [C.POINTER(BlockCfg), i32, i32]),
    "aj_varlen_block_fwd": (C.c_int, [C.POINTER(BlockCfg), C.POINTER(BlockWeights),
                                      C.POINTER(Varlen), vp, vp, vp, vp, sz, vp]),
    "aj_varlen_block_bwd": (C.c_int, [C.POINTER(BlockCfg), C.POINTER(BlockWeights),
                                      C.POINTER(Varlen), vp, vp, vp, vp,
                                      C.POINTER(BlockGrads), vp, sz, vp]),
    "aj_stack_ckpt_bytes": (sz, [C.POINTER(BlockCfg), i32, i32]),
    "aj_stack_fwd": (C.c_int, [C.POINTER(BlockCfg), i32, C.POINTER(BlockWeights),
                               C.POINTER(Varlen), vp, vp, vp, vp, vp]),
    "aj_stack_bwd": (C.c_int, [C.POINTER(BlockCfg), i32, C.POINTER(BlockWeights),
                               C.POINTER(Varlen), vp, vp, vp, vp, vp, C.POINTER(BlockGrads), vp,
                               sz, vp]),
    "aj_lora_saved_bytes": (sz, [C.POINTER(BlockCfg), i32, i32]),
    "aj_lora_workspace_bytes": (sz, [C.POINTER(BlockCfg), i32, i32]),
    "aj_stack_lora_fwd": (C.c_int, [C.POINTER(BlockCfg), i32, C.POINTER(BlockWeights),
                                    C.POINTER(Lora), C.POINTER(Varlen), vp, vp, vp, vp, vp]),
    "aj_stack_lora_bwd": (C.c_int, [C.POINTER(BlockCfg), i32, C.POINTER(BlockWeights),
                                    C.POINTER(Lora), C.POINTER(Varlen), vp, vp, vp, vp, vp,
                                    C.POINTER(LoraGrads), vp, sz, vp]),
    "aj_loss_saved_bytes": (sz, [C.POINTER(LossCfg), i32]),
    "aj_loss_workspace_bytes": (sz, [C.POINTER(LossCfg), i32]),
    "aj_logprob_pg_loss_fwd": (C.c_int, [C.POINTER(LossCfg), C.POINTER(LossIn), vp, vp, vp, vp,
                                         vp, vp, vp, vp, vp, sz, vp]),
    "aj_logprob_pg_loss_bwd": (C.c_int, [C.POINTER(LossCfg), C.POINTER(LossIn), vp, vp, vp, vp,
                                         vp, vp, vp, vp, vp, vp, sz, vp]),
    "aj_grpo_advantages": (C.c_int, [i32, vp, vp, f32, vp, vp, vp, vp]),
    "aj_select_workspace_bytes": (sz, [i32, i32]),
    "aj_select_episodes": (C.c_int, [C.POINTER(Timelines), vp, vp, C.POINTER(TimelinesOut), vp,
                                     vp, sz, vp]),
    "aj_adamw_step": (C.c_int, [i64, vp, vp, vp, vp, f32, f32, f32, f32, f32, i32, f32, vp,
                                C.c_int, vp]),
    "aj_timing_enable": (C.c_int, [C.c_int]),
    "aj_timing_read": (C.c_int, [C.POINTER(C.c_double), C.POINTER(i64), C.POINTER(C.c_double)]),
    "aj_transpose_bf16": (C.c_int, [vp, i32, i32, vp, vp]),
    "aj_ceiling_mfma_bf16": (C.c_int, [C.c_int, vp, sz, vp, C.POINTER(C.c_double)]),
    "aj_ceiling_copy": (C.c_int, [vp, sz, vp, C.POINTER(C.c_double), C.POINTER(C.c_double)]),
}

KCLASSES = ("merge", "gemm_nt", "gemm_nn", "gemm_tn", "attn_fwd", "attn_bwd", "lm_fwd", "lm_dz",
            "gemm4_nt", "gemm4_nn", "gemm4_tn", "adamw", "select", "stage_block", "stage_loss")


def _declare(L):
    for name, (res, args) in EXPORTS.items():
        fn = getattr(L, name)
        fn.restype = res
        fn.argtypes = args


def _check(status, name):
    if status != 0:
        L = lib()
        raise AjError(f"{name}: {L.aj_status_str(status).decode()}: {L.aj_last_error().decode()}")


def ptr(t):
    """Device (or host) address of a tensor, None for None."""
    return None if t is None else C.c_void_p(t.data_ptr())


def stream_handle(stream=None):
    s = stream if stream is not None else torch.cuda.current_stream()
    return C.c_void_p(s.cuda_stream)


def dtype_code(t):
    if t.dtype == torch.bfloat16:
        return AJ_BF16
    if t.dtype == torch.float32:
        return AJ_F32
    raise AjError(f"unsupported dtype {t.dtype}")


# ------------------------------------------------------------------ merge

def aj_merge_workspace_bytes(n_traj, n_tl, n_tok):
    return int(lib().aj_merge_workspace_bytes(n_traj, n_tl, n_tok))


def _timelines(t):
    return Timelines(int(t["traj_tl_off"].numel() - 1), int(t["tl_tok_off"].numel() - 1),
                     int(t["tok"].numel()), ptr(t["traj_tl_off"]), ptr(t["tl_tok_off"]),
                     ptr(t["tok"]), ptr(t["flags"]), ptr(t["old_logprob"]), ptr(t.get("adv")))


def _packed(o):
    return Packed(*[ptr(o[k]) for k in ("absorber", "cu_seqlens", "seg_src", "cu_targets",
                                        "counts", "tok", "pos", "mask", "old_logprob", "adv",
                                        "targets")])


def aj_merge_timelines(tl, out, err, ws, stream=None):
    """tl: dict of device tensors (traj_tl_off int32, tl_tok_off int64, tok int32, flags uint8,
    old_logprob, adv float32); out: dict of output tensors (see aj_packed)."""
    _check(lib().aj_merge_timelines(C.byref(_timelines(tl)), C.byref(_packed(out)), ptr(err),
                                    ptr(ws), ws.numel() * ws.element_size(),
                                    stream_handle(stream)), "aj_merge_timelines")


def aj_flatten_timelines(tl, out, err, ws, stream=None):
    _check(lib().aj_flatten_timelines(C.byref(_timelines(tl)), C.byref(_packed(out)), ptr(err),
                                      ptr(ws), ws.numel() * ws.element_size(),
                                      stream_handle(stream)), "aj_flatten_timelines")


def aj_merge_noalloc_max_workspace_bytes():
    return int(lib().aj_merge_noalloc_max_workspace_bytes())


def aj_merge_timelines_noalloc(tl, out, err, stream=None):
    """aj_merge_timelines on the library's built-in per-GPU workspace (no ws argument)."""
    _check(lib().aj_merge_timelines_noalloc(C.byref(_timelines(tl)), C.byref(_packed(out)),
                                            ptr(err), stream_handle(stream)),
           "aj_merge_timelines_noalloc")


def aj_merge_text_workspace_bytes(n_traj, n_tl, n_tok, n_blk):
    return int(lib().aj_merge_text_workspace_bytes(n_traj, n_tl, n_tok, n_blk))


def aj_merge_timelines_text(tl, blk_text, out, err, ws, ti=None, stream=None):
    """As aj_merge_timelines with text-level Match; blk_text: device uint64 (or int64) text key
    per block, blocks in token order; ti: optional device int64 [2] for the TI report."""
    if blk_text.dtype not in (torch.int64, torch.uint64):
        raise AjError(f"aj_merge_timelines_text: blk_text must be 64-bit, got {blk_text.dtype}")
    if ti is not None and (ti.dtype != torch.int64 or ti.numel() < 2):
        raise AjError("aj_merge_timelines_text: ti must be int64 [2]")
    texts = BlockTexts(int(blk_text.numel()), ptr(blk_text))
    _check(lib().aj_merge_timelines_text(C.byref(_timelines(tl)), C.byref(texts),
                                         C.byref(_packed(out)), ptr(ti), ptr(err), ptr(ws),
                                         ws.numel() * ws.element_size(), stream_handle(stream)),
           "aj_merge_timelines_text")


def aj_plan_packs(cu_seqlens_host, max_tokens):
    """cu_seqlens_host: int32 CPU tensor [n_seg+1] -> list of pack segment offsets."""
    n_seg = cu_seqlens_host.numel() - 1
    off = torch.zeros(n_seg + 1, dtype=torch.int32)
    n = i32(0)
    cu = cu_seqlens_host.contiguous()
    _check(lib().aj_plan_packs(ptr(cu), n_seg, max_tokens, ptr(off), C.byref(n)), "aj_plan_packs")
    return off[:n.value + 1].tolist()


def aj_read_device_error(err, stream=None):
    v = i32(0)
    _check(lib().aj_read_device_error(ptr(err), stream_handle(stream), C.byref(v)),
           "aj_read_device_error")
    return v.value


# ------------------------------------------------------------------ embedding

def aj_embed_fwd(tok, emb, x, err=None, stream=None):
    _check(lib().aj_embed_fwd(ptr(tok), tok.numel(), ptr(emb), emb.shape[1], emb.shape[0],
                              dtype_code(emb), ptr(x), ptr(err), stream_handle(stream)),
           "aj_embed_fwd")


def aj_embed_bwd_workspace_bytes(n_tok, d):
    return int(lib().aj_embed_bwd_workspace_bytes(int(n_tok), int(d)))


def aj_embed_bwd(tok, dx, d_emb, ws, stream=None):
    """d_emb[tok[p]] += dx[p] (float32), deterministic; ws: a byte tensor of at least
    aj_embed_bwd_workspace_bytes(tok.numel(), d) bytes."""
    _check(lib().aj_embed_bwd(ptr(tok), tok.numel(), ptr(dx), d_emb.shape[1], d_emb.shape[0],
                              ptr(d_emb), ptr(ws), ws.numel() * ws.element_size(),
                              stream_handle(stream)), "aj_embed_bwd")


# ------------------------------------------------------------------ block

def block_cfg(m):
    return BlockCfg(m.d_model, m.n_q_heads, m.n_kv_heads, m.head_dim, m.d_ff, m.rms_eps,
                    m.rope_theta, AJ_BF16 if m.dtype == "bf16" else AJ_F32)


def aj_block_saved_bytes(cfg, n_tok):
    return int(lib().aj_block_saved_bytes(C.byref(cfg), n_tok))


def aj_block_workspace_bytes(cfg, n_tok, n_seg):
    return int(lib().aj_block_workspace_bytes(C.byref(cfg), n_tok, n_seg))


def _varlen(n_tok, n_seg, max_seqlen, base, cu_seqlens, pos):
    return Varlen(n_tok, n_seg, max_seqlen, base, ptr(cu_seqlens), ptr(pos))


def _bw(w):
    return _layers([w], BlockWeights)[0]


def aj_varlen_block_fwd(cfg, w, cu_seqlens, pos, max_seqlen, x, y, saved, ws=None, stream=None,
                        base=0):
    n_tok, n_seg = x.shape[0], cu_seqlens.numel() - 1
    vl = _varlen(n_tok, n_seg, max_seqlen, base, cu_seqlens, pos)
    _check(lib().aj_varlen_block_fwd(C.byref(cfg), C.byref(_bw(w)), C.byref(vl), ptr(x), ptr(y),
                                     ptr(saved), ptr(ws),
                                     0 if ws is None else ws.numel() * ws.element_size(),
                                     stream_handle(stream)), "aj_varlen_block_fwd")


def aj_varlen_block_bwd(cfg, w, cu_seqlens, pos, max_seqlen, x, saved, dy, dx, grads, ws,
                        stream=None, base=0):
    n_tok, n_seg = x.shape[0], cu_seqlens.numel() - 1
    vl = _varlen(n_tok, n_seg, max_seqlen, base, cu_seqlens, pos)
    g = BlockGrads(*[ptr(grads[k]) for k in ("attn_norm", "w_qkv", "w_o", "mlp_norm",
                                             "w_gate_up", "w_down")])
    _check(lib().aj_varlen_block_bwd(C.byref(cfg), C.byref(_bw(w)), C.byref(vl), ptr(x),
                                     ptr(saved), ptr(dy), ptr(dx), C.byref(g), ptr(ws),
                                     ws.numel() * ws.element_size(), stream_handle(stream)),
           "aj_varlen_block_bwd")


def aj_stack_ckpt_bytes(cfg, n_layers, n_tok):
    return int(lib().aj_stack_ckpt_bytes(C.byref(cfg), n_layers, n_tok))


def _layers(ws, kind, names=("attn_norm", "w_qkv", "w_o", "mlp_norm", "w_gate_up", "w_down")):
    """Per-layer structs; weight dicts may also hold the optional transposed
    projection weights (BLOCK_TRANSPOSED keys, all four or none)."""
    arr = (kind * len(ws))()
    for i, w in enumerate(ws):
        extra = BLOCK_TRANSPOSED if kind is BlockWeights else ()
        arr[i] = kind(*[ptr(w[k]) for k in names], *[ptr(w.get(k)) for k in extra])
    return arr


def aj_stack_fwd(cfg, layers, cu_seqlens, pos, max_seqlen, x, y, ckpt, saved, stream=None, base=0):
    """layers: list of per-layer weight dicts (the keys of aj_block_weights)."""
    n_tok, n_seg = x.shape[0], cu_seqlens.numel() - 1
    vl = _varlen(n_tok, n_seg, max_seqlen, base, cu_seqlens, pos)
    _check(lib().aj_stack_fwd(C.byref(cfg), len(layers), _layers(layers, BlockWeights),
                              C.byref(vl), ptr(x), ptr(y), ptr(ckpt), ptr(saved),
                              stream_handle(stream)), "aj_stack_fwd")


def aj_stack_bwd(cfg, layers, cu_seqlens, pos, max_seqlen, x, ckpt, saved, dy, dx, grads, ws,
                 stream=None, base=0):
    """grads: list of per-layer float32 gradient dicts, accumulated into."""
    n_tok, n_seg = x.shape[0], cu_seqlens.numel() - 1
    vl = _varlen(n_tok, n_seg, max_seqlen, base, cu_seqlens, pos)
    _check(lib().aj_stack_bwd(C.byref(cfg), len(layers), _layers(layers, BlockWeights),
                              C.byref(vl), ptr(x), ptr(ckpt), ptr(saved), ptr(dy), ptr(dx),
                              _layers(grads, BlockGrads), ptr(ws), ws.numel() * ws.element_size(),
                              stream_handle(stream)), "aj_stack_bwd")


def aj_lora_saved_bytes(cfg, rank, n_tok):
    return int(lib().aj_lora_saved_bytes(C.byref(cfg), rank, n_tok))


def aj_lora_workspace_bytes(cfg, rank, n_tok):
    return int(lib().aj_lora_workspace_bytes(C.byref(cfg), rank, n_tok))


def _lora_array(adapters, rank, scale):
    """adapters: list (one per layer) of dicts keyed by LORA_FIELDS."""
    arr = (Lora * len(adapters))()
    for i, a in enumerate(adapters):
        arr[i] = Lora(rank, scale, *[ptr(a[k]) for k in LORA_FIELDS])
    return arr


def aj_stack_lora_fwd(cfg, layers, adapters, rank, scale, cu_seqlens, pos, max_seqlen, x, y, ckpt,
                      saved, stream=None, base=0):
    n_tok, n_seg = x.shape[0], cu_seqlens.numel() - 1
    vl = _varlen(n_tok, n_seg, max_seqlen, base, cu_seqlens, pos)
    _check(lib().aj_stack_lora_fwd(C.byref(cfg), len(layers), _layers(layers, BlockWeights),
                                   _lora_array(adapters, rank, scale), C.byref(vl), ptr(x),
                                   ptr(y), ptr(ckpt), ptr(saved), stream_handle(stream)),
           "aj_stack_lora_fwd")


def aj_stack_lora_bwd(cfg, layers, adapters, rank, scale, cu_seqlens, pos, max_seqlen, x, ckpt,
                      saved, dy, dx, grads, ws, stream=None, base=0):
    """grads: list of per-layer float32 dicts keyed by LORA_FIELDS, accumulated into."""
    n_tok, n_seg = x.shape[0], cu_seqlens.numel() - 1
    vl = _varlen(n_tok, n_seg, max_seqlen, base, cu_seqlens, pos)
    _check(lib().aj_stack_lora_bwd(C.byref(cfg), len(layers), _layers(layers, BlockWeights),
                                   _lora_array(adapters, rank, scale), C.byref(vl), ptr(x),
                                   ptr(ckpt), ptr(saved), ptr(dy), ptr(dx),
                                   _layers(grads, LoraGrads, LORA_FIELDS), ptr(ws),
                                   ws.numel() * ws.element_size(), stream_handle(stream)),
           "aj_stack_lora_bwd")


# ------------------------------------------------------------------ loss

def loss_cfg(m, keep_logits=False):
    return LossCfg(m.d_model, m.vocab, m.vocab_chunk, m.clip_eps, m.rms_eps,
                   AJ_BF16 if m.dtype == "bf16" else AJ_F32, 1 if keep_logits else 0)


def aj_loss_saved_bytes(cfg, n_tgt):
    return int(lib().aj_loss_saved_bytes(C.byref(cfg), n_tgt))


def aj_loss_workspace_bytes(cfg, n_tgt):
    return int(lib().aj_loss_workspace_bytes(C.byref(cfg), n_tgt))


def _loss_in(n_tok, row_base, targets, tok, old_logprob, adv, inv_n_mask, ref_logprob, kl_coef,
             w_vocab_t=None):
    return LossIn(n_tok, targets.numel(), row_base, ptr(targets), ptr(tok), ptr(old_logprob),
                  ptr(adv), float(inv_n_mask), ptr(ref_logprob), float(kl_coef), ptr(w_vocab_t))


def aj_logprob_pg_loss_fwd(cfg, targets, tok, old_logprob, adv, inv_n_mask, h, final_norm,
                           w_vocab, saved, logprob, lse, stats, ws, err=None, stream=None,
                           row_base=0, ref_logprob=None, kl_coef=0.0, w_vocab_t=None):
    li = _loss_in(h.shape[0], row_base, targets, tok, old_logprob, adv, inv_n_mask, ref_logprob,
                  kl_coef, w_vocab_t)
    _check(lib().aj_logprob_pg_loss_fwd(C.byref(cfg), C.byref(li), ptr(h), ptr(final_norm),
                                        ptr(w_vocab), ptr(saved), ptr(logprob), ptr(lse),
                                        ptr(stats), ptr(err), ptr(ws),
                                        ws.numel() * ws.element_size(), stream_handle(stream)),
           "aj_logprob_pg_loss_fwd")


def aj_logprob_pg_loss_bwd(cfg, targets, tok, old_logprob, adv, inv_n_mask, h, final_norm,
                           w_vocab, saved, logprob, lse, dh, d_final_norm, d_w_vocab, ws,
                           stream=None, row_base=0, ref_logprob=None, kl_coef=0.0,
                           w_vocab_t=None):
    li = _loss_in(h.shape[0], row_base, targets, tok, old_logprob, adv, inv_n_mask, ref_logprob,
                  kl_coef, w_vocab_t)
    _check(lib().aj_logprob_pg_loss_bwd(C.byref(cfg), C.byref(li), ptr(h), ptr(final_norm),
                                        ptr(w_vocab), ptr(saved), ptr(logprob), ptr(lse),
                                        ptr(dh), ptr(d_final_norm), ptr(d_w_vocab), ptr(ws),
                                        ws.numel() * ws.element_size(), stream_handle(stream)),
           "aj_logprob_pg_loss_bwd")


# ------------------------------------------------------------------ around the update

def aj_grpo_advantages(group_off, reward, eps, ep_adv, ep_keep, err=None, stream=None):
    _check(lib().aj_grpo_advantages(int(group_off.numel() - 1), ptr(group_off), ptr(reward),
                                    float(eps), ptr(ep_adv), ptr(ep_keep), ptr(err),
                                    stream_handle(stream)), "aj_grpo_advantages")


def aj_select_workspace_bytes(n_traj, n_tl):
    return int(lib().aj_select_workspace_bytes(n_traj, n_tl))


def aj_select_episodes(tl, keep, ep_adv, out, ws, err=None, stream=None):
    """tl: dict as for aj_merge_timelines (adv not read); out: dict of capacity-sized tensors
    traj_tl_off, tl_tok_off, tok, flags, old_logprob, adv, counts (int64 [3])."""
    o = TimelinesOut(*[ptr(out[k]) for k in ("traj_tl_off", "tl_tok_off", "tok", "flags",
                                             "old_logprob", "adv", "counts")])
    _check(lib().aj_select_episodes(C.byref(_timelines(tl)), ptr(keep), ptr(ep_adv), C.byref(o),
                                    ptr(err), ptr(ws), ws.numel() * ws.element_size(),
                                    stream_handle(stream)), "aj_select_episodes")


def aj_adamw_step(param, grad, m, v, lr, beta1, beta2, eps, weight_decay, step, grad_scale=1.0,
                  param_copy=None, stream=None):
    """param, grad, m, v: float32 tensors of equal size; param_copy: optional float32 or
    bfloat16 tensor receiving the updated parameters."""
    for t in (param, grad, m, v):
        if t.dtype != torch.float32 or t.numel() != param.numel():
            raise AjError("aj_adamw_step: param, grad, m, v must be float32 of one size")
    dt = 0
    if param_copy is not None:
        if param_copy.dtype not in (torch.float32, torch.bfloat16) or param_copy.numel() != param.numel():
            raise AjError("aj_adamw_step: param_copy must be float32 or bfloat16 of the same size")
        dt = 1 if param_copy.dtype == torch.bfloat16 else 0
    _check(lib().aj_adamw_step(param.numel(), ptr(param), ptr(grad), ptr(m), ptr(v), float(lr),
                               float(beta1), float(beta2), float(eps), float(weight_decay),
                               int(step), float(grad_scale), ptr(param_copy), dt,
                               stream_handle(stream)), "aj_adamw_step")


# ------------------------------------------------------------------ timing

def aj_timing_enable(on=True):
    _check(lib().aj_timing_enable(1 if on else 0), "aj_timing_enable")


def aj_timing_read():
    """{class: (ms, launches, flops)} summed over the launches recorded since enabling."""
    n = len(KCLASSES)
    ms, cnt, fl = (C.c_double * n)(), (i64 * n)(), (C.c_double * n)()
    _check(lib().aj_timing_read(ms, cnt, fl), "aj_timing_read")
    return {k: (ms[i], int(cnt[i]), fl[i]) for i, k in enumerate(KCLASSES)}


# ------------------------------------------------------------------ ceilings

def aj_ceiling_mfma_bf16(random_operands, out, stream=None):
    """TFLOP/s of the register-only bf16 MFMA loop; out: float32 device scratch."""
    r = C.c_double()
    _check(lib().aj_ceiling_mfma_bf16(1 if random_operands else 0, ptr(out),
                                      out.numel() * out.element_size(), stream_handle(stream),
                                      C.byref(r)), "aj_ceiling_mfma_bf16")
    return r.value


def aj_ceiling_copy(buf, stream=None):
    """(copy GB/s counting read + write, read-only GB/s) of streams over buf."""
    r, rd = C.c_double(), C.c_double()
    _check(lib().aj_ceiling_copy(ptr(buf), buf.numel() * buf.element_size(),
                                 stream_handle(stream), C.byref(r), C.byref(rd)),
           "aj_ceiling_copy")
    return r.value, rd.value


def aj_transpose_bf16(src, dst, stream=None):
    """dst (cols x rows) = src (rows x cols)^T, both bfloat16 device tensors."""
    rows, cols = src.shape
    if dst.shape != (cols, rows) or src.dtype != torch.bfloat16 or dst.dtype != torch.bfloat16:
        raise ValueError("aj_transpose_bf16: dst must be the bfloat16 [cols, rows] of src")
    _check(lib().aj_transpose_bf16(ptr(src), rows, cols, ptr(dst), stream_handle(stream)),
           "aj_transpose_bf16")
