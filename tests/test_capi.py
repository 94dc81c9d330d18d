"""The C-ABI library: loads, exports every symbol include/aj.h declares, and its
host-side logic (argument validation, pack planning) works without a GPU."""
import ctypes as C
import os
import re

import numpy as np
import pytest
import torch

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _lib():
    from paper_2606_04484_amd import capi
    if not os.path.exists(capi.LIB_PATH):
        from paper_2606_04484_amd.build import build
        build()
    return capi


def _declared():
    src = open(os.path.join(ROOT, "include", "aj.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(aj_[a-z0-9_]+)\s*\(", src)))


def test_every_declared_symbol_is_exported():
    capi = _lib()
    names = _declared()
    assert len(names) >= 17
    raw = C.CDLL(capi.LIB_PATH)
    for n in names:
        assert hasattr(raw, n), n
        assert n in capi.EXPORTS, f"{n} missing from the Python binding"


def test_status_strings():
    capi = _lib()
    L = capi.lib()
    assert L.aj_status_str(0) == b"ok"
    assert L.aj_status_str(4) == b"workspace too small"


def test_plan_packs_greedy_in_order():
    capi = _lib()
    lens = np.array([5, 7, 3, 10, 1, 1, 12, 4])
    cu = torch.tensor(np.concatenate([[0], np.cumsum(lens)]), dtype=torch.int32)
    offs = capi.aj_plan_packs(cu, 12)
    # greedy: [5,7] [3] [10,1,1] [12] [4] -- a segment never splits; packs <= 12 tokens
    assert offs == [0, 2, 3, 6, 7, 8]
    offs = capi.aj_plan_packs(cu, 8)   # 10 and 12 exceed the limit: alone in their packs
    assert offs == [0, 1, 2, 3, 4, 6, 7, 8]


def test_plan_packs_rejects_bad_offsets():
    capi = _lib()
    cu = torch.tensor([0, 5, 3], dtype=torch.int32)
    with pytest.raises(capi.AjError, match="monotone"):
        capi.aj_plan_packs(cu, 16)


def test_host_validation_needs_no_gpu():
    """Argument errors return before any HIP call."""
    capi = _lib()
    L = capi.lib()
    assert L.aj_merge_timelines(None, None, None, None, 0, None) == 1   # AJ_ERR_NULL
    tl = capi.Timelines(1, 1, -5, None, None, None, None, None, None)
    out = capi.Packed()
    assert L.aj_merge_timelines(C.byref(tl), C.byref(out), None, None, 0, None) == 2
    cfg = capi.BlockCfg(128, 4, 3, 32, 512, 1e-6, 1e6, 0)      # 4 % 3 != 0
    w = capi.BlockWeights(*[C.c_void_p(16)] * 6)
    vl = capi.Varlen(0, 0, 0, 0, None, None)
    assert L.aj_varlen_block_fwd(C.byref(cfg), C.byref(w), C.byref(vl), None, None, None, None,
                                 0, None) == 2
    cfg = capi.BlockCfg(128, 4, 4, 256, 512, 1e-6, 1e6, 0)     # head_dim 256 unsupported
    assert L.aj_varlen_block_fwd(C.byref(cfg), C.byref(w), C.byref(vl), None, None, None, None,
                                 0, None) == 3
    assert b"head_dim" in L.aj_last_error()
    lc = capi.LossCfg(128, 1024, 1024, 0.2, 1e-6, 0)
    li = capi.LossIn(10, 11, 0, None, None, None, None, 1.0)      # n_tgt > n_tok
    assert L.aj_logprob_pg_loss_fwd(C.byref(lc), C.byref(li), *([None] * 9), 0, None) == 2
    # transposed weights: all four projections or none; a vocab the transposed
    # LM-head copy cannot hold in 16-byte rows
    cfg = capi.BlockCfg(128, 4, 4, 32, 512, 1e-6, 1e6, 1)
    w = capi.BlockWeights(*[C.c_void_p(16)] * 6, C.c_void_p(16), C.c_void_p(16))
    assert L.aj_varlen_block_fwd(C.byref(cfg), C.byref(w), C.byref(vl), None, None, None, None,
                                 0, None) == 1
    assert b"transposed" in L.aj_last_error()
    w = capi.BlockWeights(*[C.c_void_p(16)] * 10)
    assert L.aj_varlen_block_fwd(C.byref(cfg), C.byref(w), C.byref(vl), None, None, None, None,
                                 0, None) == 0                     # empty pack: nothing to do
    lc = capi.LossCfg(128, 1001, 1024, 0.2, 1e-6, 1)
    li = capi.LossIn(10, 5, 0, None, None, None, None, 1.0, None, 0.0, C.c_void_p(16))
    assert L.aj_logprob_pg_loss_fwd(C.byref(lc), C.byref(li), *([None] * 9), 0, None) == 2
    assert b"vocab" in L.aj_last_error()


def test_ceiling_and_transpose_host_validation():
    """The measurement and transpose entry points check their arguments before
    any device call."""
    capi = _lib()
    L = capi.lib()
    d, d2 = C.c_double(), C.c_double()
    assert L.aj_ceiling_copy(None, 64, None, C.byref(d), C.byref(d2)) == 1
    assert L.aj_ceiling_copy(C.c_void_p(4096), 64, None, None, C.byref(d2)) == 1
    assert L.aj_ceiling_copy(C.c_void_p(4096), 16, None, C.byref(d), C.byref(d2)) == 2
    assert L.aj_ceiling_copy(C.c_void_p(4104), 64, None, C.byref(d), C.byref(d2)) == 2
    assert b"16-byte aligned" in L.aj_last_error()
    assert L.aj_ceiling_mfma_bf16(1, None, 1 << 20, None, C.byref(d)) == 1
    assert L.aj_ceiling_mfma_bf16(1, C.c_void_p(4096), 1 << 20, None, None) == 1
    assert L.aj_transpose_bf16(None, 4, 4, C.c_void_p(16), None) == 1
    assert L.aj_transpose_bf16(C.c_void_p(16), 0, 4, C.c_void_p(16), None) == 2
    assert L.aj_transpose_bf16(C.c_void_p(16), 4, -1, C.c_void_p(16), None) == 2


def test_loss_saved_bytes_with_kept_logits():
    """keep_logits adds the float32 logits of every scored row to the loss's
    saved buffer, in bfloat16 only (the float32 path ignores it)."""
    capi = _lib()
    for dtype, grows in ((capi.AJ_BF16, True), (capi.AJ_F32, False)):
        base = capi.aj_loss_saved_bytes(capi.LossCfg(256, 5000, 1024, 0.2, 1e-6, dtype, 0), 300)
        kept = capi.aj_loss_saved_bytes(capi.LossCfg(256, 5000, 1024, 0.2, 1e-6, dtype, 1), 300)
        if grows:
            assert 300 * 5000 * 4 <= kept - base <= 300 * 5000 * 4 + 256, (base, kept)
        else:
            assert kept == base


def test_text_merge_host_validation():
    """aj_merge_timelines_text: argument errors return before any HIP call."""
    capi = _lib()
    L = capi.lib()
    d = C.c_void_p(256)                       # never dereferenced on the host
    tl = capi.Timelines(1, 2, 10, d, d, d, d, d, d)
    out = capi.Packed(*[d] * 11)
    assert L.aj_merge_timelines_text(C.byref(tl), None, C.byref(out), None, None, d, 1 << 20,
                                     None) == 1
    txt = capi.BlockTexts(11, d)              # more blocks than tokens
    assert L.aj_merge_timelines_text(C.byref(tl), C.byref(txt), C.byref(out), None, None, d,
                                     1 << 20, None) == 2
    assert b"n_blk" in L.aj_last_error()
    txt = capi.BlockTexts(4, None)
    assert L.aj_merge_timelines_text(C.byref(tl), C.byref(txt), C.byref(out), None, None, d,
                                     1 << 20, None) == 1
    txt = capi.BlockTexts(4, d)
    need = capi.aj_merge_text_workspace_bytes(1, 2, 10, 4)
    assert L.aj_merge_timelines_text(C.byref(tl), C.byref(txt), C.byref(out), None, None, d,
                                     need - 1, None) == 4
    assert capi.aj_merge_text_workspace_bytes(4, 32, 5000, 200) > \
        capi.aj_merge_text_workspace_bytes(4, 32, 5000, 100)


def test_stack_host_validation():
    capi = _lib()
    L = capi.lib()
    cfg = capi.BlockCfg(128, 4, 4, 32, 512, 1e-6, 1e6, 1)
    vl = capi.Varlen(0, 0, 0, 0, None, None)
    ws = (capi.BlockWeights * 2)(*[capi.BlockWeights(*[C.c_void_p(16)] * 6)] * 2)
    assert L.aj_stack_fwd(C.byref(cfg), 0, ws, C.byref(vl), None, None, None, None, None) == 2
    assert L.aj_stack_fwd(C.byref(cfg), 2, None, C.byref(vl), None, None, None, None, None) == 1
    ws[1].w_o = None
    assert L.aj_stack_fwd(C.byref(cfg), 2, ws, C.byref(vl), None, None, None, None, None) == 1
    ws[1].w_o = C.c_void_p(16)
    gs = (capi.BlockGrads * 2)(*[capi.BlockGrads(*[C.c_void_p(16)] * 6)] * 2)
    vl = capi.Varlen(10, 1, 10, 0, C.c_void_p(16), C.c_void_p(16))
    # two layers need the checkpoint buffer
    assert L.aj_stack_bwd(C.byref(cfg), 2, ws, C.byref(vl), C.c_void_p(16), None, C.c_void_p(16),
                          C.c_void_p(16), C.c_void_p(16), gs, C.c_void_p(16), 1 << 30, None) == 1
    assert capi.aj_stack_ckpt_bytes(cfg, 1, 1000) == 0
    assert capi.aj_stack_ckpt_bytes(cfg, 4, 1000) == 3 * 1000 * 128 * 2


def test_workspace_queries_grow_with_size():
    capi = _lib()
    L = capi.lib()
    cfg = capi.BlockCfg(3584, 28, 4, 128, 18944, 1e-6, 1e6, 1)
    a = L.aj_block_saved_bytes(C.byref(cfg), 1000)
    b = L.aj_block_saved_bytes(C.byref(cfg), 2000)
    assert 0 < a < b
    # ~150 KB of saved activations per token at the 7B block shape
    assert 140e3 < b / 2000 < 160e3
    # per-token (target bits, range counts), per-item and per-timeline tables
    w = capi.aj_merge_workspace_bytes(4, 32, 5000)
    assert capi.aj_merge_workspace_bytes(4, 32, 500000) > w > 0
    assert capi.aj_merge_workspace_bytes(4, 3200, 5000) > w
