"""GPU parity of the kernels against the oracle on identical inputs: the
canonical fp32 primitives bit for bit, and the quantized linear layers
(int32 accumulators and int8 outputs bit-exact, fp32 epilogues bit-exact with
the 1e-3 relative bar checked as well) over the sweep shapes and ragged ones."""
import numpy as np
import pytest

import oracle
from synth import generate as G

pytestmark = pytest.mark.gpu

RTOL = 1e-3  # floating-point bar for fp32 outputs


@pytest.fixture(scope="module")
def torch_dev():
    import torch

    assert torch.cuda.is_available(), "GPU tests need a visible GPU"
    from paper_2306_04235_amd import mnmt

    mnmt.lib()
    return torch, torch.device("cuda:0")


def _gpu(torch, dev, a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(dev)


def test_canon_exp_log_sum_bitwise(torch_dev):
    torch, dev = torch_dev
    from paper_2306_04235_amd import mnmt

    lo = np.float32(-87.0).view(np.uint32)
    x = (np.arange(0, lo + 1, 97, dtype=np.uint32) | np.uint32(0x80000000)).view(np.float32)
    x = np.concatenate([x[x >= -87.0], np.float32([0.0, -0.0, -87.0, -86.99999, -1e-30, -87.5])])
    y = mnmt.mnmt_debug_canon(0, _gpu(torch, dev, x)).cpu().numpy()
    assert np.array_equal(y.view(np.uint32), oracle.exp_array(x).view(np.uint32))
    one = np.float32(1.0).view(np.uint32)
    xl = np.arange(np.float32(1e-30).view(np.uint32), np.float32(1e6).view(np.uint32), 131, dtype=np.uint32)
    xl = xl.view(np.float32)
    yl = mnmt.mnmt_debug_canon(1, _gpu(torch, dev, xl)).cpu().numpy()
    assert np.array_equal(yl.view(np.uint32), oracle.log_array(xl).view(np.uint32))
    assert one  # silence linters
    rng = np.random.default_rng(0)
    for n in (1, 3, 63, 64, 65, 130, 256, 1000, 32000):
        v = (rng.standard_normal(n) * rng.uniform(0.1, 1e4)).astype(np.float32)
        s = mnmt.mnmt_debug_canon(2, _gpu(torch, dev, v)).cpu().numpy()[0]
        assert np.float32(s).view(np.uint32) == oracle.canon_sum(v).view(np.uint32), n
    v = np.ones(130, np.float32)
    v[0] = 2 ** 24
    assert mnmt.mnmt_debug_canon(2, _gpu(torch, dev, v)).cpu().numpy()[0] == 16777344.0


SWEEP = [(M, K, N) for M in G.SWEEP_M for (K, N) in G.SWEEP_KN]
RAGGED = [(1, 64, 1), (3, 64, 5), (2, 128, 130), (5, 192, 37), (8, 2048, 77), (9, 128, 130), (31, 256, 100),
          (33, 192, 257), (65, 64, 33), (100, 512, 129), (130, 320, 1000), (257, 1024, 255)]


def _rows_to_check(M, rng):
    if M <= 300:
        return np.arange(M)
    return np.unique(np.concatenate([[0, M - 1], rng.choice(M, 30, replace=False)]))


def _run(torch, dev, X, W, scale, bias, epi, gamma=1.0, resid=None):
    from paper_2306_04235_amd import mnmt

    tX, tW = _gpu(torch, dev, X), _gpu(torch, dev, W)
    ts = _gpu(torch, dev, scale)
    tb = _gpu(torch, dev, bias) if bias is not None else None
    out = None
    if epi == mnmt.EPI_F32_RESID:
        out = _gpu(torch, dev, resid.copy())
    y = mnmt.mnmt_qlinear(tX, tW, ts, tb, epi, gamma=gamma, out=out)
    torch.cuda.synchronize()
    return y.cpu().numpy()


@pytest.mark.parametrize("M,K,N", SWEEP + RAGGED, ids=lambda v: str(v))
def test_qlinear_requant_parity(torch_dev, M, K, N):
    torch, dev = torch_dev
    from paper_2306_04235_amd import mnmt

    print(f"qlinear I8 M={M} K={K} N={N}", flush=True)
    X, W, mult, bias = G.sweep_case(M, K, N)
    got = _run(torch, dev, X, W, mult, bias, mnmt.EPI_I8)
    rows = _rows_to_check(M, np.random.default_rng(M + N))
    ref = oracle.qlinear(X[rows], W, mult, bias, oracle.EPI_I8)
    assert np.array_equal(got[rows], ref)


@pytest.mark.parametrize("M,K,N", [(1, 256, 1024), (4, 1024, 256), (7, 64, 33), (64, 512, 2048), (130, 320, 1000),
                                   (256, 256, 32000)], ids=lambda v: str(v))
def test_qlinear_all_epilogues(torch_dev, M, K, N):
    torch, dev = torch_dev
    from paper_2306_04235_amd import mnmt

    X, W, mult, bias = G.sweep_case(M, K, N, seed=99)
    rows = _rows_to_check(M, np.random.default_rng(1))
    got = _run(torch, dev, X, W, mult, bias, mnmt.EPI_I32)
    assert np.array_equal(got[rows], oracle.qgemm_i32(X[rows], W))
    got = _run(torch, dev, X, W, mult, bias, mnmt.EPI_I8_RELU)
    assert np.array_equal(got[rows], oracle.qlinear(X[rows], W, mult, bias, oracle.EPI_I8_RELU))
    dq = (mult * 1e-3).astype(np.float32)
    for epi in (mnmt.EPI_F32, mnmt.EPI_LOGITS):
        got = _run(torch, dev, X, W, dq, bias, epi)
        ref = oracle.qlinear(X[rows], W, dq, bias, epi)
        assert np.allclose(got[rows], ref, rtol=RTOL, atol=0)
        assert np.array_equal(got[rows].view(np.uint32), ref.view(np.uint32))
    resid = np.random.default_rng(2).normal(0, 1, (M, N)).astype(np.float32)
    got = _run(torch, dev, X, W, dq, bias, mnmt.EPI_F32_RESID, gamma=0.75, resid=resid)
    ref = oracle.qlinear(X[rows], W, dq, bias, oracle.EPI_F32_RESID, gamma=0.75, resid=resid[rows])
    assert np.array_equal(got[rows].view(np.uint32), ref.view(np.uint32))


W4_SHAPES = [(1, 256, 1024), (2, 2048, 77), (4, 1024, 256), (7, 64, 33), (33, 192, 257), (64, 512, 2048),
             (130, 320, 1000), (256, 256, 768), (512, 512, 512), (1000, 256, 1500), (3840, 256, 768),
             (2048, 1024, 300), (2048, 256, 8192), (8192, 512, 2048)]


@pytest.mark.parametrize("M,K,N", W4_SHAPES, ids=lambda v: str(v))
def test_qlinear_4bit_weights(torch_dev, M, K, N):
    """4-bit weights (W-E-A 4-8-8) read packed by every quantized-linear path:
    the wavefront-reduction GEMV (M <= 8), the one-round-trip matrix-core
    kernel (its 32x32 and one-wave 16x16 blocks), the slab-pipelined GEMM and
    the persistent GEMM (the last two shapes).  The codes in [-7, 7] are packed
    as the model file stores them; the int32 sums and every epilogue equal the
    oracle's on the codes."""
    torch, dev = torch_dev
    from paper_2306_04235_amd import mnmt
    from synth.modelfile import pack_int4

    print(f"qlinear 4-bit M={M} K={K} N={N}", flush=True)
    X, _, mult, bias = G.sweep_case(M, K, N, seed=41)
    codes = np.random.Generator(np.random.PCG64(M * 7 + K * 3 + N)).integers(-7, 8, size=(N, K)).astype(np.int8)
    W4 = np.frombuffer(pack_int4(codes), np.uint8).reshape(N, K // 2).copy()
    tX, tW4 = _gpu(torch, dev, X), _gpu(torch, dev, W4)
    rows = _rows_to_check(M, np.random.default_rng(M + 5))
    mult4 = (mult * 127.0 / 7.0).astype(np.float32)  # outputs span about the same codes as int8 weights
    tm, tb = _gpu(torch, dev, mult4), _gpu(torch, dev, bias)

    def run(epi, scale=tm, gamma=1.0, out=None):
        y = mnmt.mnmt_qlinear_w4(tX, tW4, scale, tb, epi, gamma=gamma, out=out)
        torch.cuda.synchronize()
        return y.cpu().numpy()[rows]

    assert np.array_equal(run(mnmt.EPI_I32), oracle.qgemm_i32(X[rows], codes))
    for epi, oepi in ((mnmt.EPI_I8, oracle.EPI_I8), (mnmt.EPI_I8_RELU, oracle.EPI_I8_RELU)):
        assert np.array_equal(run(epi), oracle.qlinear(X[rows], codes, mult4, bias, oepi))
    dq = (mult4 * 1e-3).astype(np.float32)
    for epi in (mnmt.EPI_F32, mnmt.EPI_LOGITS):
        ref = oracle.qlinear(X[rows], codes, dq, bias, epi)
        assert np.array_equal(run(epi, _gpu(torch, dev, dq)).view(np.uint32), ref.view(np.uint32))
    resid = np.random.default_rng(6).normal(0, 1, (M, N)).astype(np.float32)
    got = run(mnmt.EPI_F32_RESID, _gpu(torch, dev, dq), 0.75, _gpu(torch, dev, resid))
    ref = oracle.qlinear(X[rows], codes, dq, bias, oracle.EPI_F32_RESID, gamma=0.75, resid=resid[rows])
    assert np.array_equal(got.view(np.uint32), ref.view(np.uint32))


def test_qlinear_4bit_rejects_argmax(torch_dev):
    torch, dev = torch_dev
    from paper_2306_04235_amd import mnmt

    X = torch.zeros((1, 64), dtype=torch.int8, device=dev)
    W4 = torch.zeros((16, 32), dtype=torch.uint8, device=dev)
    sc = torch.ones(16, dtype=torch.float32, device=dev)
    for epi in (mnmt.EPI_ARGMAX, mnmt.EPI_ARGMAX_PARTIAL, mnmt.EPI_ARGMAX_PARTIAL_PACKED):
        with pytest.raises(mnmt.MnmtError) as e:
            mnmt.mnmt_qlinear_w4(X, W4, sc, None, epi, out=torch.zeros(16, dtype=torch.int64, device=dev))
        assert e.value.status == mnmt.E_UNSUPPORTED


@pytest.mark.parametrize("M,K,N", [(2048, 256, 8192), (1024, 1024, 16384), (768, 2048, 22016), (4096, 512, 4096)],
                         ids=lambda v: str(v))
def test_qlinear_persistent_gemm_epilogues(torch_dev, M, K, N):
    """Whole 256 x 128 tiles and at least 512 of them: the persistent GEMM
    (2, 8, 16 and 4 chunks of 128 bytes of K), every epilogue, sampled rows."""
    torch, dev = torch_dev
    from paper_2306_04235_amd import mnmt

    print(f"persistent GEMM M={M} K={K} N={N}", flush=True)
    X, W, mult, bias = G.sweep_case(M, K, N, seed=7)
    rows = np.unique(np.concatenate([[0, 127, 128, M - 1], np.random.default_rng(3).choice(M, 28, replace=False)]))
    acc = oracle.qgemm_i32(X[rows], W)
    got = _run(torch, dev, X, W, mult, bias, mnmt.EPI_I32)
    assert np.array_equal(got[rows], acc)
    for epi, oepi in ((mnmt.EPI_I8, oracle.EPI_I8), (mnmt.EPI_I8_RELU, oracle.EPI_I8_RELU)):
        got = _run(torch, dev, X, W, mult, bias, epi)
        assert np.array_equal(got[rows], oracle.qlinear(X[rows], W, mult, bias, oepi))
    dq = (mult * 1e-3).astype(np.float32)
    for epi in (mnmt.EPI_F32, mnmt.EPI_LOGITS):
        got = _run(torch, dev, X, W, dq, bias, epi)
        ref = oracle.qlinear(X[rows], W, dq, bias, epi)
        assert np.array_equal(got[rows].view(np.uint32), ref.view(np.uint32))
    resid = np.random.default_rng(4).normal(0, 1, (M, N)).astype(np.float32)
    got = _run(torch, dev, X, W, dq, bias, mnmt.EPI_F32_RESID, gamma=0.75, resid=resid)
    ref = oracle.qlinear(X[rows], W, dq, bias, oracle.EPI_F32_RESID, gamma=0.75, resid=resid[rows])
    assert np.array_equal(got[rows].view(np.uint32), ref.view(np.uint32))


@pytest.mark.parametrize("M,K,N", [(4096, 256, 32000), (4096, 256, 16384), (8192, 256, 8192)], ids=lambda v: str(v))
def test_qlinear_weight_stationary_gemm(torch_dev, M, K, N):
    """K = 256 with at least 16 row steps of 64 per block: the weight-stationary
    kernel (weights in registers, the epilogue of one step interleaved with the
    next step's MFMAs).  Sampled rows include the first two rows of every
    block's first step, which that kernel first fills with a placeholder and
    then rewrites, and each block's last step; every epilogue it takes."""
    torch, dev = torch_dev
    from paper_2306_04235_amd import mnmt

    print(f"weight-stationary GEMM M={M} K={K} N={N}", flush=True)
    X, W, mult, bias = G.sweep_case(M, K, N, seed=11)
    ncol, steps = N // 256, M // 64
    spb = -(-steps // max(1, min(steps, 256 // ncol)))
    starts = np.arange(0, steps, spb) * 64
    rows = np.unique(np.concatenate([starts, starts + 33, np.minimum(starts + spb * 64, M) - 1,
                                     np.random.default_rng(5).choice(M, 12, replace=False)]))
    got = _run(torch, dev, X, W, mult, bias, mnmt.EPI_I32)
    assert np.array_equal(got[rows], oracle.qgemm_i32(X[rows], W))
    for epi, oepi in ((mnmt.EPI_I8, oracle.EPI_I8), (mnmt.EPI_I8_RELU, oracle.EPI_I8_RELU)):
        got = _run(torch, dev, X, W, mult, bias, epi)
        assert np.array_equal(got[rows], oracle.qlinear(X[rows], W, mult, bias, oepi))
    dq = (mult * 1e-3).astype(np.float32)
    for epi in (mnmt.EPI_F32, mnmt.EPI_LOGITS):
        got = _run(torch, dev, X, W, dq, bias, epi)
        ref = oracle.qlinear(X[rows], W, dq, bias, epi)
        assert np.array_equal(got[rows].view(np.uint32), ref.view(np.uint32))


@pytest.mark.parametrize("M,K,N", [(1, 256, 32000), (2, 512, 32000), (1, 64, 1000), (2, 128, 33), (1, 384, 129),
                                   (3, 256, 1000), (8, 1024, 4097), (2, 1024, 500)], ids=lambda v: str(v))
def test_qlinear_fused_argmax(torch_dev, M, K, N):
    # M <= 2 with K <= 512 runs the decoder's logits kernel (matrix cores, one
    # slot per row); other shapes run the GEMV.  Rows of W are duplicated so
    # that the maximum is tied and the smallest index must win.
    torch, dev = torch_dev
    from paper_2306_04235_amd import mnmt

    print(f"qlinear ARGMAX M={M} K={K} N={N}", flush=True)
    X, W, mult, _ = G.sweep_case(M, K, N, seed=7)
    rng = np.random.default_rng(N)
    dq = (mult * 1e-3).astype(np.float32)
    ref_z = oracle.qlinear(X, W, dq, None, oracle.EPI_LOGITS)
    for m in range(M):  # copy each row's winner to a later and an earlier index
        best = int(np.argmax(ref_z[m]))
        for dst in {int(rng.integers(0, N)), N - 1}:
            W[dst] = W[best]
            dq[dst] = dq[best]
    ref_z = oracle.qlinear(X, W, dq, None, oracle.EPI_LOGITS)
    got = _run(torch, dev, X, W, dq, None, mnmt.EPI_ARGMAX)
    idx = mnmt.argmax_index(got)
    assert np.array_equal(idx, np.argmax(ref_z, axis=1))  # numpy: the first maximum
    # the key holds the maximum logit itself
    keys = (got.astype(np.int64) >> 32) & 0xFFFFFFFF
    bits = np.where(keys & 0x80000000, keys & 0x7FFFFFFF, ~keys & 0xFFFFFFFF).astype(np.uint32)
    assert np.array_equal(bits.view(np.float32), ref_z.max(axis=1))
    if M <= 2 and K <= 512:
        # one key per block of 128 outputs: each is its block's arg-max key,
        # and their maximum is the row's
        part = _run(torch, dev, X, W, dq, None, mnmt.EPI_ARGMAX_PARTIAL)
        P = mnmt.argmax_partials(N)
        assert part.shape == (M, P)
        assert np.array_equal(part.view(np.uint64).max(axis=1), got.view(np.uint64))
        for p in sorted({0, P // 2, P - 1}):
            blk = ref_z[:, 128 * p:128 * (p + 1)]
            assert np.array_equal(mnmt.argmax_index(part[:, p]), 128 * p + np.argmax(blk, axis=1))
        # the same kernel on the fragment-order copy of W gives the same keys
        tW = _gpu(torch, dev, W)
        packed = mnmt.mnmt_pack_weights(tW)
        got_p = mnmt.mnmt_qlinear(_gpu(torch, dev, X), packed, _gpu(torch, dev, dq), None,
                                  mnmt.EPI_ARGMAX_PARTIAL_PACKED, n_out=N)
        torch.cuda.synchronize()
        assert np.array_equal(got_p.cpu().numpy().view(np.uint64), part.view(np.uint64))


@pytest.mark.parametrize("N,K", [(33, 64), (1000, 256), (32000, 256), (129, 512), (16, 1024)], ids=lambda v: str(v))
def test_pack_weights_layout(torch_dev, N, K):
    # chunk l of kilobyte (t, j) holds W[16t + l % 16, 64j + 16(l // 16) .. +15], zero rows past N
    torch, dev = torch_dev
    from paper_2306_04235_amd import mnmt

    print(f"pack_weights N={N} K={K}", flush=True)
    W = np.random.default_rng(N + K).integers(-127, 128, (N, K)).astype(np.int8)
    got = mnmt.mnmt_pack_weights(_gpu(torch, dev, W))
    torch.cuda.synchronize()
    tiles = (N + 15) // 16
    assert mnmt.lib().mnmt_packed_bytes(N, K) == tiles * 16 * K == got.numel()
    Wp = np.zeros((tiles * 16, K), np.int8)
    Wp[:N] = W
    # [t, r, j, q, b] -> [t, j, q, r, b]: lane l = 16 q + r
    ref = Wp.reshape(tiles, 16, K // 64, 4, 16).transpose(0, 2, 3, 1, 4).reshape(-1)
    assert np.array_equal(got.cpu().numpy().reshape(-1), ref)


def test_qlinear_timed_matches_and_times_the_kernel(torch_dev):
    torch, dev = torch_dev
    from paper_2306_04235_amd import mnmt

    for M, K, N, epi in ((1, 256, 32000, mnmt.EPI_ARGMAX), (4, 256, 1024, mnmt.EPI_ARGMAX),
                         (1, 256, 32000, mnmt.EPI_ARGMAX_PARTIAL_PACKED)):
        X, W, mult, _ = G.sweep_case(M, K, N, seed=5)
        tX, tW, ts = _gpu(torch, dev, X), _gpu(torch, dev, W), _gpu(torch, dev, (mult * 1e-3).astype(np.float32))
        if epi == mnmt.EPI_ARGMAX_PARTIAL_PACKED:
            tW = mnmt.mnmt_pack_weights(tW)
        ref = mnmt.mnmt_qlinear(tX, tW, ts, None, epi, n_out=N)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        e1.record()
        got = mnmt.mnmt_qlinear_timed(tX, tW, ts, None, epi, e0, e1, n_out=N)
        e1.synchronize()
        assert torch.equal(got, ref)
        assert 0.0 < e0.elapsed_time(e1) < 100.0


def test_qlinear_worst_case_accumulator(torch_dev):
    torch, dev = torch_dev
    from paper_2306_04235_amd import mnmt

    for M in (1, 40):
        X = np.full((M, 4096), 127, np.int8)
        X[0] = -127
        W = np.full((70, 4096), -127, np.int8)
        W[5] = 127
        got = _run(torch, dev, X, W, np.ones(70, np.float32), None, mnmt.EPI_I32)
        assert np.array_equal(got, oracle.qgemm_i32(X, W))
        assert got[0, 0] == 66064384 and got[-1, 0] == (-66064384 if M > 1 else 66064384)


def test_qlinear_rejects_bad_shapes(torch_dev):
    torch, dev = torch_dev
    from paper_2306_04235_amd import mnmt

    X = torch.zeros((4, 100), dtype=torch.int8, device=dev)
    W = torch.zeros((8, 100), dtype=torch.int8, device=dev)
    s = torch.ones(8, dtype=torch.float32, device=dev)
    with pytest.raises(mnmt.MnmtError) as e:
        mnmt.mnmt_qlinear(X, W, s, s, mnmt.EPI_I8)
    assert e.value.status == mnmt.E_INVALID_ARG
    X = torch.zeros((0, 64), dtype=torch.int8, device=dev)
    W = torch.zeros((8, 64), dtype=torch.int8, device=dev)
    out = mnmt.mnmt_qlinear(X, W, s, s, mnmt.EPI_I8)  # empty batch is a no-op
    assert out.shape == (0, 8)
