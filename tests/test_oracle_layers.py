"""Pins for the oracle's integer GEMM, linear-layer epilogues, LayerNorm and
attention against float64 brute force, closed forms and invariants."""
import numpy as np
import pytest

import oracle

F32, F64 = np.float32, np.float64


def _rand_i8(rng, shape, lo=-127, hi=127):
    return rng.integers(lo, hi + 1, size=shape).astype(np.int8)


@pytest.mark.parametrize("M,K,N", [(1, 16, 1), (3, 64, 5), (17, 256, 33), (30, 128, 77), (1, 1024, 9)])
def test_qgemm_exact_vs_float64(M, K, N):
    rng = np.random.default_rng(M * 1000 + K + N)
    X, W = _rand_i8(rng, (M, K)), _rand_i8(rng, (N, K))
    ref = X.astype(F64) @ W.astype(F64).T  # exact: integers far below 2^53
    assert np.array_equal(oracle.qgemm_i32(X, W), ref.astype(np.int64))


def test_qgemm_worst_case_no_overflow():
    K = 4096
    X = np.full((2, K), 127, np.int8)
    X[1] = -127
    W = np.full((3, K), -127, np.int8)
    W[2] = 127
    Y = oracle.qgemm_i32(X, W)
    assert Y[0, 0] == -66064384 and Y[1, 0] == 66064384 and Y[0, 2] == 66064384
    assert 127 * 127 * 4096 == 66064384 < 2 ** 31 - 1


def _acc(X, W):
    return (X.astype(F64) @ W.astype(F64).T)


def test_epilogue_i8_vs_float64():
    rng = np.random.default_rng(7)
    M, K, N = 9, 512, 300
    X, W = _rand_i8(rng, (M, K)), _rand_i8(rng, (N, K))
    scale = (127.0 / (4 * 5418.67 * np.sqrt(K)) * rng.uniform(0.5, 1.5, N)).astype(F32)
    bias = rng.normal(0, 8, N).astype(F32)
    for epi, relu in ((oracle.EPI_I8, False), (oracle.EPI_I8_RELU, True)):
        q = oracle.qlinear(X, W, scale, bias, epi).astype(np.int64)
        y = _acc(X, W).astype(F32).astype(F64) * scale.astype(F64) + bias.astype(F64)
        if relu:
            y = np.maximum(y, 0.0)
        ref = np.clip(np.round(y), -127, 127)
        diff = q - ref
        frac = np.abs(y - np.floor(y) - 0.5)
        assert np.all(np.abs(diff) <= 1)
        assert np.all(frac[diff != 0] < 1e-5)  # differences only at .5 boundaries
        assert (diff != 0).mean() < 1e-3
        if relu:
            assert q.min() >= 0
        assert np.abs(q).max() <= 127


def test_epilogue_f32_resid_logits_vs_float64():
    rng = np.random.default_rng(8)
    M, K, N = 5, 256, 200
    X, W = _rand_i8(rng, (M, K)), _rand_i8(rng, (N, K))
    scale = rng.uniform(1e-5, 1e-4, N).astype(F32)
    bias = rng.normal(0, 0.02, N).astype(F32)
    acc32 = _acc(X, W).astype(F32).astype(F64)
    y = oracle.qlinear(X, W, scale, bias, oracle.EPI_F32).astype(F64)
    exact = acc32 * scale + bias
    assert np.all(np.abs(y - exact) <= np.spacing(np.abs(exact).astype(F32)) * 0.5 + 1e-30)
    x0 = rng.normal(0, 1, (M, N)).astype(F32)
    g = 0.75
    r = oracle.qlinear(X, W, scale, bias, oracle.EPI_F32_RESID, gamma=g, resid=x0).astype(F64)
    exact_r = g * x0.astype(F64) + exact
    assert np.allclose(r, exact_r, rtol=2e-7, atol=2e-7)
    r1 = oracle.qlinear(X, W, scale, bias, oracle.EPI_F32_RESID, gamma=1.0, resid=x0)
    f = oracle.qlinear(X, W, scale, bias, oracle.EPI_F32)
    assert np.array_equal(r1, (x0 + f).astype(F32))  # gamma = 1: fma(1, x, o) = x + o exactly
    z = oracle.qlinear(X, W, scale, None, oracle.EPI_LOGITS).astype(F64)
    assert np.array_equal(z, (acc32 * scale.astype(F64)).astype(F32).astype(F64))
    i32 = oracle.qlinear(X, W, scale, bias, oracle.EPI_I32)
    assert np.array_equal(i32, oracle.qgemm_i32(X, W))


def test_folded_requant_matches_unfolded_chain():
    # (s_in X . s_w W + b) / s_out  ==  acc * scale + bias  with scale, bias folded
    rng = np.random.default_rng(9)
    N, K = 400, 256
    s_in, s_out = 0.031, 0.047
    s_w = rng.uniform(1e-4, 5e-4, N).astype(F32)
    b = rng.normal(0, 0.02, N).astype(F32)
    sc, bi = oracle.fold_requant(s_in, s_w, b, s_out)
    X, W = _rand_i8(rng, (3, K)), _rand_i8(rng, (N, K))
    q = oracle.qlinear(X, W, sc, bi, oracle.EPI_I8).astype(np.int64)
    real = (F64(F32(s_in)) * X.astype(F64)) @ (W.astype(F64) * s_w.astype(F64)[:, None]).T + b.astype(F64)
    y = real / F64(F32(s_out))
    ref = np.clip(np.round(y), -127, 127)
    assert np.all(np.abs(q - ref) <= 1)
    assert (q != ref).mean() < 2e-3


def _ln64(x, g, b, eps):
    x = x.astype(F64)
    mu = x.mean(axis=1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=1, keepdims=True)
    return (x - mu) / np.sqrt(var + eps) * g.astype(F64) + b.astype(F64)


@pytest.mark.parametrize("d", [64, 256, 384, 512])
def test_layernorm_vs_float64(d):
    rng = np.random.default_rng(d)
    x = (rng.normal(0.3, 2.0, (7, d))).astype(F32)
    g = rng.normal(1, 0.02, d).astype(F32)
    b = rng.normal(0, 0.02, d).astype(F32)
    inv_s = F32(127 / 4.0)
    q, y = oracle.layernorm_quant(x, g, b, 1e-5, inv_s, want_y=True)
    ref = _ln64(x, g, b, 1e-5)
    assert np.abs(y - ref).max() <= 1e-5 * np.abs(ref).max()
    refq = np.clip(np.round(y.astype(F32) * inv_s), -127, 127)
    assert np.array_equal(q, refq.astype(np.int8))


def test_layernorm_invariants():
    rng = np.random.default_rng(11)
    d = 256
    x = (rng.normal(5.0, 3.0, (4, d))).astype(F32)
    one, zero = np.ones(d, F32), np.zeros(d, F32)
    _, y = oracle.layernorm_quant(x, one, zero, 1e-5, 1.0, want_y=True)
    assert np.abs(y.astype(F64).mean(axis=1)).max() < 1e-6
    assert np.abs(y.astype(F64).var(axis=1) - 1.0).max() < 1e-5
    # shift invariance of the normalized row (exact shift by a power of two)
    _, y2 = oracle.layernorm_quant(x + F32(64.0), one, zero, 1e-5, 1.0, want_y=True)
    assert np.abs(y2 - y).max() < 1e-4


def _attend64(q, K, V, c_qk, c_pv):
    s = (K.astype(F64) @ q.astype(F64)) * F64(c_qk)
    p = np.exp(s - s.max())
    p /= p.sum()
    return p @ V.astype(F64) * F64(c_pv)


@pytest.mark.parametrize("n,dh", [(1, 64), (5, 16), (30, 64), (64, 64), (80, 64), (130, 32)])
def test_attend_vs_float64(n, dh):
    rng = np.random.default_rng(n * 100 + dh)
    fails = 0
    for trial in range(10):
        q, K, V = _rand_i8(rng, dh), _rand_i8(rng, (n, dh)), _rand_i8(rng, (n, dh))
        c_qk = F32(rng.uniform(1e-4, 2e-3))
        c_pv = F32(rng.uniform(0.3, 1.5))
        out = oracle.attend(q, K, V, c_qk, c_pv).astype(np.int64)
        y = _attend64(q, K, V, c_qk, c_pv)
        ref = np.clip(np.round(y), -127, 127)
        assert np.all(np.abs(out - ref) <= 1)
        frac = np.abs(y - np.floor(y) - 0.5)
        assert np.all(frac[out != ref] < 1e-4)
        fails += int((out != ref).sum())
    assert fails <= 3


def test_attend_special_cases():
    rng = np.random.default_rng(5)
    dh = 64
    q, k, v = _rand_i8(rng, dh), _rand_i8(rng, (1, dh)), _rand_i8(rng, (1, dh))
    # one key: softmax is exactly 1, the context is the value row
    assert np.array_equal(oracle.attend(q, k, v, 1e-3, 1.0), v[0])
    # identical keys and values: uniform weights, context equals the value row
    K = np.repeat(k, 7, axis=0)
    V = np.repeat(v, 7, axis=0)
    assert np.array_equal(oracle.attend(q, K, V, 1e-3, 1.0), v[0])
    # one dominant key: weight 1 on it, exactly
    q = np.full(dh, 127, np.int8)
    K = np.zeros((9, dh), np.int8)
    K[4] = 127
    V = _rand_i8(rng, (9, dh))
    assert np.array_equal(oracle.attend(q, K, V, 1.0, 1.0), V[4])
    # the scores' shift does not matter: adding the same offset to every score
    # (here by an extra key dimension contributing equally) changes nothing
    q2 = np.concatenate([q, [100]]).astype(np.int8)
    K2 = np.concatenate([K, np.full((9, 1), 50, np.int8)], axis=1)
    V2 = np.concatenate([V, np.zeros((9, 1), np.int8)], axis=1)
    assert np.array_equal(oracle.attend(q2, K2, V2, 1.0, 1.0)[:dh], V[4])


def test_softmax_weights_sum_to_one_via_values():
    # with V = c (constant code) the context is c for any scores
    rng = np.random.default_rng(12)
    for n in (3, 50, 100):
        q, K = _rand_i8(rng, 32), _rand_i8(rng, (n, 32))
        V = np.full((n, 32), 100, np.int8)
        assert np.all(oracle.attend(q, K, V, 1e-3, 1.0) == 100)


def test_log_softmax_stats_vs_float64():
    rng = np.random.default_rng(13)
    for n in (6, 1000, 32000):
        z = rng.normal(0, 0.5, n).astype(F32)
        mx, lse = oracle.log_softmax_stats(z)
        assert mx == z.max()
        ref = np.log(np.exp(z.astype(F64) - F64(mx)).sum()) + F64(mx)
        assert abs(F64(lse) - ref) <= 4e-7 * max(1.0, abs(ref))


def _round_f32_exact(fr):
    """The fp32 value nearest to the exact rational fr (ties to even)."""
    import fractions

    f = float(fr)  # nearest double
    lo = np.float32(f)
    # step to the neighbour whose exact distance to fr is smallest
    cands = [np.nextafter(lo, np.float32(-np.inf)), lo, np.nextafter(lo, np.float32(np.inf))]
    best = min(cands, key=lambda c: (abs(fractions.Fraction(float(c)) - fr), int(np.float32(c).view(np.uint32)) & 1))
    return np.float32(best)


def test_folded_constants_are_once_rounded():
    """Folded requant and dequant constants (Section 3.2 quantizers folded into
    one multiplier and one bias per channel) are the fp32 values nearest to the
    exact s_in s_w / s_out, b / s_out and s_in s_w: compared with exact rational
    arithmetic; a double intermediate may rarely differ by one fp32 ulp."""
    import fractions

    rng = np.random.default_rng(17)
    N = 2000
    s_in, s_out = F32(0.0313), F32(0.0471)
    s_w = rng.uniform(1e-4, 5e-4, N).astype(F32)
    b = rng.normal(0, 0.02, N).astype(F32)
    sc, bi = oracle.fold_requant(s_in, s_w, b, s_out)
    dq = oracle.fold_dequant(s_in, s_w)
    Fr = fractions.Fraction
    off = 0
    for n in range(N):
        e_sc = _round_f32_exact(Fr(float(s_in)) * Fr(float(s_w[n])) / Fr(float(s_out)))
        e_bi = _round_f32_exact(Fr(float(b[n])) / Fr(float(s_out)))
        for got, exp in ((sc[n], e_sc), (bi[n], e_bi)):
            d = abs(int(np.float32(got).view(np.int32)) - int(np.float32(exp).view(np.int32)))
            assert d <= 1
            off += d
        # the product of two fp32 values is exact in double: one rounding, so
        # it equals the correctly rounded fp32 product
        assert dq[n] == np.float32(s_in) * np.float32(s_w[n])
        assert dq[n] == _round_f32_exact(Fr(float(s_in)) * Fr(float(s_w[n])))
    assert off <= 4
