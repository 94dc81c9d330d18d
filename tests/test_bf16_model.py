"""Pins for the bfloat16 storage tolerance model (CPU only): its rounding is
torch's round-to-nearest-even conversion, and with the roundings it stays
close to, but not equal to, the float64 oracle on the tiny workload."""
import numpy as np
import torch

from oracle import model as M
from workloads import get_config, make_weights_numpy
from tests.bf16_model import bf16, block_logprob_rows_rounded


def test_rounding_is_torch_bf16():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.normal(0, 3, 10000), [1 + 2.0 ** -8, 1 + 2.0 ** -8 + 2.0 ** -20,
                                                    -(1 + 3 * 2.0 ** -8), 0.0, 65504.0]])
    ref = torch.from_numpy(x.astype(np.float32)).to(torch.bfloat16).double().numpy()
    np.testing.assert_array_equal(bf16(x), ref)
    assert bf16(1 + 2.0 ** -8) == 1.0                       # tie to even
    assert bf16(1 + 2.0 ** -8 + 2.0 ** -20) == 1 + 2.0 ** -7


def test_model_close_to_oracle():
    m = get_config(0).model
    W = {k: bf16(v) for k, v in make_weights_numpy(m, gain_std=0.1).items()}
    rng = np.random.default_rng(1)
    L = 96
    tok = rng.integers(0, m.vocab, L + 1)
    rows = np.arange(40, L)
    x = W["emb"][tok[:L]]
    y = M.block_forward_rows(x, np.arange(L), rows, W, m)
    _, _, lp, _ = M.lm_head_forward(y, W, np.concatenate([[0], tok[rows + 1]]),
                                    np.arange(1, len(rows) + 1), m)
    lp_r = block_logprob_rows_rounded(x, np.arange(L), rows, tok[rows + 1], W, m)
    e = lp_r - lp
    assert 0 < np.abs(e).max() < 5e-2
    assert abs(e.mean()) < 1e-2
