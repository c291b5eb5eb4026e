"""The allocation-free entry point (mnmt_logits_argmax_noalloc) against the
entry point it varies, mnmt_qlinear with MNMT_EPI_ARGMAX_PARTIAL_PACKED
(partial keys in a caller buffer, reduced here on the host), and against the
oracle's logits: keys and indices bit-exact, on two calls in a row, the second
with a smaller input, so that the second cannot pass on the first's leftovers
in the shared static scratch."""
import numpy as np
import pytest

import oracle
from synth import generate as G

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_dev():
    import torch

    assert torch.cuda.is_available(), "GPU tests need a visible GPU"
    return torch, torch.device("cuda:0")


def _case(torch, dev, M, K, N, seed):
    from paper_2306_04235_amd import mnmt

    X, W, mult, _ = G.sweep_case(M, K, N, seed=seed)
    scale = (mult * 1e-3).astype(np.float32)
    tX = torch.from_numpy(X).to(dev)
    tW = mnmt.mnmt_pack_weights(torch.from_numpy(W).to(dev))
    ts = torch.from_numpy(scale).to(dev)
    return X, W, scale, tX, tW, ts


def _keys_from_partials(part):
    p = part.view(np.uint64)
    best = p.max(axis=1)
    return best, (np.uint64(0xFFFFFFFF) - (best & np.uint64(0xFFFFFFFF))).astype(np.int64)


def test_noalloc_matches_partial_entry_point(torch_dev):
    torch, dev = torch_dev
    from paper_2306_04235_amd import mnmt

    # two calls in a row, the second smaller (fewer rows, narrower K, fewer outputs)
    for M, K, N, seed in ((2, 256, 32000, 11), (1, 128, 1000, 12), (2, 512, 4097, 13), (1, 64, 33, 14)):
        print(f"noalloc M={M} K={K} N={N}", flush=True)
        X, W, scale, tX, tW, ts = _case(torch, dev, M, K, N, seed)
        key, tok = mnmt.mnmt_logits_argmax_noalloc(tX, tW, ts, N)
        part = mnmt.mnmt_qlinear(tX, tW, ts, None, mnmt.EPI_ARGMAX_PARTIAL_PACKED, n_out=N)
        torch.cuda.synchronize()
        ref_key, ref_tok = _keys_from_partials(part.cpu().numpy())
        assert np.array_equal(key.cpu().numpy().view(np.uint64), ref_key)
        assert np.array_equal(tok.cpu().numpy(), ref_tok)
        z = oracle.qlinear(X, W, scale, None, oracle.EPI_LOGITS)
        assert np.array_equal(tok.cpu().numpy(), z.argmax(axis=1))


def test_noalloc_rejects_sizes_beyond_its_scratch(torch_dev):
    torch, dev = torch_dev
    from paper_2306_04235_amd import mnmt

    X, W, scale, tX, tW, ts = _case(torch, dev, 2, 256, 1000, 15)
    key = torch.empty(4, dtype=torch.int64, device=dev)
    # every shape is refused on the host, before any launch
    for M, K, N in ((3, 256, 1000), (2, 576, 1000), (2, 256, 262145), (0, 256, 1000), (2, 96, 1000)):
        rc = mnmt.lib().mnmt_logits_argmax_noalloc(mnmt._ptr(tX), mnmt._ptr(tW), mnmt._ptr(ts), M, K, N,
                                                   mnmt._ptr(key), None, None)
        assert rc == mnmt.E_INVALID_ARG, (M, K, N)
