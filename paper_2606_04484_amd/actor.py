"""One actor-update step on the GPU, driven from the host through the C ABI.

    merge (or flatten) the timelines -> read back the counts once -> plan packs
    for each pack: embed -> block fwd -> loss fwd -> loss bwd -> block bwd -> embed bwd

Gradients accumulate in float32 across packs; the loss is normalised by the
masked-token count of the whole batch, so the per-pack calls compose into the
batch's token mean.  torch only allocates device memory and provides the
stream; every step of the path is a libaj call.
"""
from dataclasses import dataclass, field

import numpy as np
import torch

from . import capi as C

BLOCK_NAMES = ("attn_norm", "w_qkv", "w_o", "mlp_norm", "w_gate_up", "w_down")


def layer_key(name, layer):
    """Weight-dict key of a block weight: layer 0 under its plain name, layer l >= 1
    under "name.l"."""
    return name if layer == 0 else f"{name}.{layer}"


LORA_PROJ = {"qkv": "w_qkv", "o": "w_o", "gate_up": "w_gate_up", "down": "w_down"}


def lora_key(kind, proj, layer):
    """Key of a LoRA matrix ("a" [rank, in] or "b" [out, rank]) of projection `proj`
    (a block weight name) in `layer`: "lora_a.w_qkv", "lora_b.w_o.2", ..."""
    return layer_key(f"lora_{kind}.{proj}", layer)


def upload_timelines(tl, old_logprob, device="cuda"):
    """Host Timelines (+ rollout log-probs, float32 [n_tok]) -> device tensors; the block
    text keys too when the timelines carry them (bit patterns in an int64 tensor)."""
    def t(a, dt):
        return torch.from_numpy(np.ascontiguousarray(a)).to(device=device, dtype=dt)
    d = {
        "traj_tl_off": t(tl.traj_tl_off, torch.int32),
        "tl_tok_off": t(tl.tl_tok_off, torch.int64),
        "tok": t(tl.tok, torch.int32),
        "flags": t(tl.flags, torch.uint8),
        "old_logprob": t(old_logprob.astype(np.float32), torch.float32),
        "adv": t(tl.adv, torch.float32),
    }
    if getattr(tl, "blk_text", None) is not None:
        d["blk_text"] = t(np.asarray(tl.blk_text, np.uint64).view(np.int64), torch.int64)
    return d


@dataclass
class Layout:
    """Packed segments on the device plus the host-side counts and packs."""
    dev: dict
    n_seg: int
    n_tok: int
    n_mask: int
    max_seqlen: int
    cu_host: np.ndarray
    cut_host: np.ndarray
    packs: list = field(default_factory=list)

    def __getattr__(self, k):
        d = self.__dict__.get("dev")
        if d is not None and k in d:
            return d[k]
        raise AttributeError(k)


class Merger:
    """Owns the output and workspace buffers of aj_merge_timelines (text=False) or
    aj_merge_timelines_text (text=True: Match on tl_dev["blk_text"]) for one input size."""

    def __init__(self, tl_dev, text=False):
        dev = tl_dev["tok"].device
        n_traj = tl_dev["traj_tl_off"].numel() - 1
        n_tl = tl_dev["tl_tok_off"].numel() - 1
        n_tok = tl_dev["tok"].numel()
        cap = max(n_tok, 1)
        i32 = dict(dtype=torch.int32, device=dev)
        self.tl = tl_dev
        self.out = {
            "absorber": torch.empty(max(n_tl, 1), **i32),
            "cu_seqlens": torch.empty(n_tl + 1, **i32),
            "seg_src": torch.empty(max(n_tl, 1), **i32),
            "cu_targets": torch.empty(n_tl + 1, **i32),
            "counts": torch.zeros(4, dtype=torch.int64, device=dev),
            "tok": torch.empty(cap, **i32),
            "pos": torch.empty(cap, **i32),
            "mask": torch.empty(cap, dtype=torch.uint8, device=dev),
            "old_logprob": torch.empty(cap, dtype=torch.float32, device=dev),
            "adv": torch.empty(cap, dtype=torch.float32, device=dev),
            "targets": torch.empty(cap, **i32),
        }
        self.err = torch.zeros(1, **i32)
        self.text = text
        if text:
            n_blk = tl_dev["blk_text"].numel()
            nbytes = C.aj_merge_text_workspace_bytes(n_traj, n_tl, n_tok, n_blk)
            self.ti = torch.zeros(2, dtype=torch.int64, device=dev)
        else:
            nbytes = C.aj_merge_workspace_bytes(n_traj, n_tl, n_tok)
        self.ws = torch.empty(nbytes, dtype=torch.uint8, device=dev)

    def launch(self, merged=True):
        if self.text:
            if not merged:
                raise ValueError("text-level Match is a merge; flatten with text=False")
            C.aj_merge_timelines_text(self.tl, self.tl["blk_text"], self.out, self.err, self.ws,
                                      self.ti)
            return
        fn = C.aj_merge_timelines if merged else C.aj_flatten_timelines
        fn(self.tl, self.out, self.err, self.ws)

    def layout(self, pack_tokens):
        """Reads the counts back (one synchronisation) and plans the packs."""
        counts = self.out["counts"].cpu().tolist()
        n_seg, n_tok, n_mask, max_seqlen = (int(v) for v in counts)
        cu = self.out["cu_seqlens"][:n_seg + 1].cpu()
        cut = self.out["cu_targets"][:n_seg + 1].cpu().numpy()
        L = Layout(self.out, n_seg, n_tok, n_mask, max_seqlen, cu.numpy(), cut)
        if n_seg:
            offs = C.aj_plan_packs(cu, pack_tokens)
            cuh = cu.numpy()
            for a, b in zip(offs[:-1], offs[1:]):
                lens = np.diff(cuh[a:b + 1])
                L.packs.append(dict(s0=a, s1=b, t0=int(cuh[a]), t1=int(cuh[b]), r0=int(cut[a]),
                                    r1=int(cut[b]), max_len=int(lens.max())))
        return L

    def device_error(self):
        return C.aj_read_device_error(self.err)


def merge(tl_dev, merged=True, pack_tokens=131072, text=False):
    m = Merger(tl_dev, text=text)
    m.launch(merged)
    return m.layout(pack_tokens)


class ActorUpdate:
    """Weights, gradient accumulators and step buffers of the policy: embedding,
    m.n_layers decoder blocks (checkpointed: aj_stack_fwd / aj_stack_bwd), LM head."""

    # the share of the free device memory the kept logits of one pack may take
    KEEP_LOGITS_SHARE = 0.5

    def __init__(self, m, weights, device="cuda", lora=None, lora_rank=0, lora_scale=1.0,
                 keep_logits=False, transposed_weights=True):
        """lora: optional dict of LoRA matrices keyed by lora_key (storage dtype of the
        weights); then only they train (self.G holds their gradients) and every
        weight, gain, the embedding and the LM head stay frozen.
        keep_logits: False (the default) streams the vocab projection and the
        LM-head backward recomputes it, so the logits are never materialised;
        True makes the backward read the forward's float32 logits instead
        (bfloat16; bitwise the same result, ~4 bytes per logit of a pack in
        HBM); None = True whenever one pack's logits fit in KEEP_LOGITS_SHARE of
        the free memory.
        transposed_weights: bfloat16 full training keeps [in][out] copies of the
        four projection weights of every block and of the LM head, refreshed at
        the start of every step (so they follow any weight update), which the
        forward's projections read faster than the [out][in] weights."""
        self.m = m
        self.W = weights
        self.n_layers = getattr(m, "n_layers", 1)
        self.dev = torch.device(device)
        self.dt = torch.bfloat16 if m.dtype == "bf16" else torch.float32
        self.bcfg = C.block_cfg(m)
        self.keep_logits = keep_logits
        self.lcfg = C.loss_cfg(m)          # the step's (keep_logits decided per capacity)
        self.lcfg_fwd = C.loss_cfg(m)      # forward-only scoring keeps nothing
        self.lora, self.rank, self.scale = lora, lora_rank, lora_scale
        trained = lora if lora is not None else weights
        self.G = {k: torch.zeros(v.shape, dtype=torch.float32, device=self.dev)
                  for k, v in trained.items()}
        # [0] loss, [1] clipped count, [2] sum of r, [3] targets, [4] sum of KL
        self.stats = torch.zeros(5, dtype=torch.float32, device=self.dev)
        self.err = torch.zeros(1, dtype=torch.int32, device=self.dev)
        self._cap = (0, 0)
        self.layers = [{k: weights[layer_key(k, l)] for k in BLOCK_NAMES}
                       for l in range(self.n_layers)]
        self.WT = None
        if transposed_weights and self.dt == torch.bfloat16 and lora is None:
            self.WT = {}
            for l, lw in enumerate(self.layers):
                for k in ("w_qkv", "w_o", "w_gate_up", "w_down"):
                    t = torch.empty(lw[k].shape[1], lw[k].shape[0], dtype=self.dt, device=self.dev)
                    self.WT[layer_key(k, l)] = t
                    lw[k + "_t"] = t
            if m.vocab % 8 == 0:
                self.WT["w_vocab"] = torch.empty(m.d_model, m.vocab, dtype=self.dt,
                                                 device=self.dev)
        if lora is None:
            self.layer_grads = [{k: self.G[layer_key(k, l)] for k in BLOCK_NAMES}
                                for l in range(self.n_layers)]
        else:
            def fields(src):
                return [{f"{kind}_{short}": src[lora_key(kind, proj, l)]
                         for short, proj in LORA_PROJ.items() for kind in ("a", "b")}
                        for l in range(self.n_layers)]
            self.adapters = fields(lora)
            self.layer_grads = fields(self.G)

    def set_keep_logits(self, keep):
        """Switches the LM-head backward between recomputing and kept logits
        (the step buffers are sized again by the next prepare)."""
        self.keep_logits = keep
        self._cap = (0, 0)
        if hasattr(self, "logprob"):
            del self.logprob

    def refresh_transposed(self):
        """The [in][out] weight copies from the current weights (part of each step)."""
        if self.WT is None:
            return
        for k, t in self.WT.items():
            C.aj_transpose_bf16(self.W[k], t)

    def _w_vocab_t(self):
        return None if self.WT is None else self.WT.get("w_vocab")

    def zero_grads(self):
        for g in self.G.values():
            g.zero_()
        self.stats.zero_()

    def _buffers(self, n_tok, n_tgt):
        if n_tok <= self._cap[0] and n_tgt <= self._cap[1]:
            return
        n_tok, n_tgt = max(n_tok, self._cap[0]), max(n_tgt, self._cap[1])
        d, dev = self.m.d_model, self.dev
        u8 = lambda nb: torch.empty(max(int(nb), 1), dtype=torch.uint8, device=dev)
        self.x = torch.empty(n_tok, d, dtype=self.dt, device=dev)
        self.y = torch.empty(n_tok, d, dtype=self.dt, device=dev)
        self.dh = torch.empty(n_tok, d, dtype=torch.float32, device=dev)
        if self.lora is None:
            self.saved = u8(C.aj_block_saved_bytes(self.bcfg, n_tok))
            self.bws = u8(C.aj_block_workspace_bytes(self.bcfg, n_tok, n_tok))
        else:
            self.saved = u8(C.aj_lora_saved_bytes(self.bcfg, self.rank, n_tok))
            self.bws = u8(C.aj_lora_workspace_bytes(self.bcfg, self.rank, n_tok))
        self.ckpt = u8(C.aj_stack_ckpt_bytes(self.bcfg, self.n_layers, n_tok))
        self.ews = u8(C.aj_embed_bwd_workspace_bytes(n_tok, d))
        self.lsaved = None
        keep = self.keep_logits
        if keep is None:
            logit_bytes = n_tgt * self.m.vocab * 4
            keep = self.m.dtype == "bf16" and \
                logit_bytes <= self.KEEP_LOGITS_SHARE * torch.cuda.mem_get_info(dev)[0]
        self.lcfg = C.loss_cfg(self.m, keep_logits=bool(keep))
        self.lsaved = u8(C.aj_loss_saved_bytes(self.lcfg, n_tgt))
        self.lws = u8(C.aj_loss_workspace_bytes(self.lcfg, n_tgt))
        self._cap = (n_tok, n_tgt)

    def prepare(self, L):
        """Allocates everything a step over layout L needs (outside any timed region)."""
        mt = max((p["t1"] - p["t0"] for p in L.packs), default=0)
        mr = max((p["r1"] - p["r0"] for p in L.packs), default=0)
        self._buffers(mt, mr)
        self.logprob = torch.empty(max(L.n_mask, 1), dtype=torch.float32, device=self.dev)
        self.lse = torch.empty(max(L.n_mask, 1), dtype=torch.float32, device=self.dev)

    def step(self, L, ref_logprob=None, kl_coef=0.0):
        """Forward + backward over every pack of L; gradients accumulate into self.G.

        ref_logprob: optional [n_mask] float32 log-probs of L's targets under a
        reference policy (e.g. forward_logprob of a frozen copy), for the KL
        penalty with weight kl_coef."""
        if not hasattr(self, "logprob") or self.logprob.numel() < max(L.n_mask, 1):
            self.prepare(L)
        W, G = self.W, self.G
        inv = 1.0 / L.n_mask if L.n_mask else 0.0
        self.refresh_transposed()
        wvt = self._w_vocab_t()
        for p in L.packs:
            t0, t1, s0, s1, r0, r1 = p["t0"], p["t1"], p["s0"], p["s1"], p["r0"], p["r1"]
            n = t1 - t0
            x, y, dh = self.x[:n], self.y[:n], self.dh[:n]
            tok = L.tok[t0:t1]
            cu = L.cu_seqlens[s0:s1 + 1]
            pos = L.pos[t0:t1]
            tg = L.targets[r0:r1]
            C.aj_embed_fwd(tok, W["emb"], x, self.err)
            self._stack_fwd(cu, pos, p["max_len"], x, y, t0)
            ref = ref_logprob[r0:r1] if ref_logprob is not None else None
            C.aj_logprob_pg_loss_fwd(self.lcfg, tg, L.tok, L.old_logprob, L.adv, inv, y,
                                     W["final_norm"], W["w_vocab"], self.lsaved,
                                     self.logprob[r0:r1], self.lse[r0:r1], self.stats, self.lws,
                                     self.err, row_base=t0, ref_logprob=ref, kl_coef=kl_coef,
                                     w_vocab_t=wvt)
            C.aj_logprob_pg_loss_bwd(self.lcfg, tg, L.tok, L.old_logprob, L.adv, inv, y,
                                     W["final_norm"], W["w_vocab"], self.lsaved,
                                     self.logprob[r0:r1], self.lse[r0:r1], dh,
                                     G.get("final_norm"), G.get("w_vocab"), self.lws,
                                     row_base=t0, ref_logprob=ref, kl_coef=kl_coef,
                                     w_vocab_t=wvt)
            if self.lora is None:
                C.aj_stack_bwd(self.bcfg, self.layers, cu, pos, p["max_len"], x, self.ckpt,
                               self.saved, dh, dh, self.layer_grads, self.bws, base=t0)
                C.aj_embed_bwd(tok, dh, G["emb"], self.ews)
            else:
                C.aj_stack_lora_bwd(self.bcfg, self.layers, self.adapters, self.rank, self.scale,
                                    cu, pos, p["max_len"], x, self.ckpt, self.saved, dh, dh,
                                    self.layer_grads, self.bws, base=t0)
        return self.stats

    def _stack_fwd(self, cu, pos, max_len, x, y, t0):
        if self.lora is None:
            C.aj_stack_fwd(self.bcfg, self.layers, cu, pos, max_len, x, y, self.ckpt, self.saved,
                           base=t0)
        else:
            C.aj_stack_lora_fwd(self.bcfg, self.layers, self.adapters, self.rank, self.scale, cu,
                                pos, max_len, x, y, self.ckpt, self.saved, base=t0)

    def forward_logprob(self, L):
        """Log-probs of every target under the current weights (forward only)."""
        self.prepare(L)
        inv = 1.0 / L.n_mask if L.n_mask else 0.0
        self.refresh_transposed()
        for p in L.packs:
            t0, t1, s0, s1, r0, r1 = p["t0"], p["t1"], p["s0"], p["s1"], p["r0"], p["r1"]
            n = t1 - t0
            C.aj_embed_fwd(L.tok[t0:t1], self.W["emb"], self.x[:n], self.err)
            self._stack_fwd(L.cu_seqlens[s0:s1 + 1], L.pos[t0:t1], p["max_len"], self.x[:n],
                            self.y[:n], t0)
            C.aj_logprob_pg_loss_fwd(self.lcfg_fwd, L.targets[r0:r1], L.tok, L.old_logprob,
                                     L.adv, inv, self.y[:n], self.W["final_norm"],
                                     self.W["w_vocab"], self.lsaved, self.logprob[r0:r1],
                                     self.lse[r0:r1], self.stats, self.lws, self.err,
                                     row_base=t0, w_vocab_t=self._w_vocab_t())
        return self.logprob[:L.n_mask]
