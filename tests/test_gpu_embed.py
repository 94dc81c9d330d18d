"""The embedding gather and its deterministic scatter-add backward against the
plain definitions: x[p] = E[tok[p]], and dE[v] = sum of dx[p] over tok[p] == v
(numpy's unbuffered np.add.at in float64).  The backward must also be bit-
identical from call to call, including on heavily repeated tokens (Zipf
ids, whose most frequent token spans many 256-row tiles of the sorted rows)
and on a single repeated token."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu


def _ids(rng, n, vocab, kind):
    if kind == "zipf":
        k = np.arange(1, vocab + 1, dtype=np.float64)
        p = k ** -1.1
        return rng.choice(vocab, n, p=p / p.sum()).astype(np.int32)
    if kind == "one":
        return np.full(n, 7, np.int32)
    return rng.integers(0, vocab, n).astype(np.int32)


def _bwd(capi, tok, dx, d_emb):
    ws = torch.empty(capi.aj_embed_bwd_workspace_bytes(tok.numel(), dx.shape[1]),
                     dtype=torch.uint8, device="cuda")
    capi.aj_embed_bwd(tok, dx, d_emb, ws)
    torch.cuda.synchronize()


@pytest.mark.parametrize("n,d,vocab,kind", [
    (1, 8, 16, "uniform"),
    (300, 136, 50, "uniform"),          # two tiles, a partial column block
    (4097, 512, 1000, "zipf"),          # one key past the first sort chunk
    (70001, 1536, 152064, "zipf"),      # several global sort passes, long runs
    (20000, 256, 5000, "one"),          # one run across every tile
    (131072, 1536, 151936, "uniform"),  # a full pack
])
def test_embed_bwd_matches_scatter_add_and_repeats(n, d, vocab, kind):
    from paper_2606_04484_amd import capi
    rng = np.random.default_rng(n + d)
    tok = _ids(rng, n, vocab, kind)
    dx = rng.standard_normal((n, d)).astype(np.float32)
    base = rng.standard_normal((vocab, d)).astype(np.float32)
    print(f"embed_bwd n={n} d={d} vocab={vocab} {kind}", flush=True)
    tok_d, dx_d = torch.from_numpy(tok).cuda(), torch.from_numpy(dx).cuda()
    outs = []
    for _ in range(2):
        g = torch.from_numpy(base).cuda()
        _bwd(capi, tok_d, dx_d, g)
        outs.append(g.cpu().numpy())
    assert np.array_equal(outs[0], outs[1])
    ref = base.astype(np.float64)
    np.add.at(ref, tok, dx.astype(np.float64))
    scale = np.abs(base).astype(np.float64)
    np.add.at(scale, tok, np.abs(dx).astype(np.float64))
    err = np.abs(outs[0] - ref) / (scale + 1e-30)
    assert err.max() <= 1e-5, err.max()


def test_embed_bwd_skips_out_of_range_tokens():
    from paper_2606_04484_amd import capi
    rng = np.random.default_rng(3)
    tok = np.array([0, -1, 5, 99, 5, 100, 2], np.int32)
    dx = rng.standard_normal((len(tok), 8)).astype(np.float32)
    g = torch.zeros(100, 8, device="cuda")
    _bwd(capi, torch.from_numpy(tok).cuda(), torch.from_numpy(dx).cuda(), g)
    ref = np.zeros((100, 8))
    ok = (tok >= 0) & (tok < 100)
    np.add.at(ref, tok[ok], dx[ok].astype(np.float64))
    np.testing.assert_allclose(g.cpu().numpy(), ref, rtol=1e-6, atol=1e-6)


def test_embed_bwd_argument_errors():
    from paper_2606_04484_amd import capi
    tok = torch.zeros(10, dtype=torch.int32, device="cuda")
    dx = torch.zeros(10, 8, device="cuda")
    g = torch.zeros(4, 8, device="cuda")
    small = torch.empty(16, dtype=torch.uint8, device="cuda")
    with pytest.raises(capi.AjError, match="workspace"):
        capi.aj_embed_bwd(tok, dx, g, small)
    g6 = torch.zeros(4, 6, device="cuda")
    with pytest.raises(capi.AjError, match="multiple of 4"):
        capi.aj_embed_bwd(tok, torch.zeros(10, 6, device="cuda"), g6, small)
    # no rows: nothing to do, any workspace
    capi.aj_embed_bwd(tok[:0], dx[:0], g, small)


def test_embed_fwd_gathers_rows():
    from paper_2606_04484_amd import capi
    rng = np.random.default_rng(4)
    emb = rng.standard_normal((300, 24)).astype(np.float32)
    tok = np.array([3, 299, 0, 3, 300], np.int32)
    x = torch.full((5, 24), 9.0, device="cuda")
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    capi.aj_embed_fwd(torch.from_numpy(tok).cuda(), torch.from_numpy(emb).cuda(), x, err)
    got = x.cpu().numpy()
    np.testing.assert_array_equal(got[:4], emb[tok[:4]])
    assert not np.any(got[4])
    assert int(err.cpu()[0]) == 1        # AJ_DEVERR_TOKEN_RANGE: token 300 is out of range
