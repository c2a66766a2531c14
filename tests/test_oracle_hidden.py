"""Pins for the oracle's hidden-state form of the proxies (CPU only):
Sec. 3.2.1 Eq. 4 (statistics of the prefill hidden states), Eq. 5 (variance-
expanded samples) and Eq. 6 (projection by each head's query weights), as
Algorithm 1 runs them.  Each test names the mistake it would catch.
"""
import math

import numpy as np
import pytest
import torch
from scipy import stats as sps

import brute


def bf16_bits(x):
    """fp32 -> bf16 bits with torch's round-to-nearest-even (a library routine)."""
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(torch.bfloat16) \
        .view(torch.uint16).numpy()


def hidden_states(B, T, D, seed, scale=1.0):
    rng = np.random.default_rng(seed)
    mean = rng.standard_normal((B, 1, D)) * 0.5
    spread = np.exp(rng.standard_normal((B, 1, D)) * 0.3)
    return (mean + spread * rng.standard_normal((B, T, D)) * scale).astype(np.float32)


# ---------------------------------------------------------------- Eq. 4
@pytest.mark.parametrize("T", [1, 2, 5, 40, 300, 512, 777])
def test_hidden_stats_match_numpy(oracle_lib, T):
    """Mean and std per (batch row, feature) over all prompt tokens, against
    numpy's mean / std (ddof 0 and 1); a wrong axis, a dropped token or a
    wrong divisor moves these far off."""
    h = hidden_states(2, T, 24, T)
    st = oracle_lib.hidden_stats(h, ddof=0)
    h64 = h.astype(np.float64)
    np.testing.assert_allclose(st[:, 0], h64.mean(axis=1), rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(st[:, 1], h64.std(axis=1, ddof=0), rtol=1e-10, atol=1e-13)
    if T > 1:
        st1 = oracle_lib.hidden_stats(h, ddof=1)
        np.testing.assert_allclose(st1[:, 1], h64.std(axis=1, ddof=1), rtol=1e-10, atol=1e-13)


def test_hidden_stats_exact_small_case(oracle_lib):
    """Tokens 1..5: mean 3, squared deviations 4, 1, 0, 1, 4 (sum 10), so the
    population std is sqrt(2) and the sample std sqrt(2.5), exactly; a
    dropped token, a missing square or a wrong divisor fails."""
    h = np.array([1, 2, 3, 4, 5], dtype=np.float32).reshape(1, 5, 1)
    st = oracle_lib.hidden_stats(h, ddof=0)
    assert st[0, 0, 0] == 3.0
    assert st[0, 1, 0] == math.sqrt(2.0)
    st1 = oracle_lib.hidden_stats(h, ddof=1)
    assert st1[0, 1, 0] == math.sqrt(2.5)


def test_hidden_stats_large_offset_is_stable(oracle_lib):
    """Features with a mean far above their spread (6e7 + a spread of a few
    units, exact in fp32): the squared deviations about the mean keep the
    std exact to rounding, where E[h^2] - E[h]^2 in fp64 loses every digit
    (the sum of squares ~3.6e18 has an ulp of 512)."""
    rng = np.random.default_rng(5)
    T = 1000
    spread = rng.integers(-8, 9, size=(1, T, 3)).astype(np.float64) * 4.0
    h = (6.0e7 + spread).astype(np.float32)
    assert np.array_equal(h.astype(np.float64), 6.0e7 + spread)
    st = oracle_lib.hidden_stats(h)
    np.testing.assert_allclose(st[0, 1], spread[0].std(axis=0), rtol=1e-12)
    np.testing.assert_allclose(st[0, 0], 6.0e7 + spread[0].mean(axis=0), rtol=1e-15)


def test_hidden_stats_constant_and_bf16_input(oracle_lib):
    """A constant feature has std 0 and its exact value as mean; bf16 inputs
    are read as their exact values."""
    h = hidden_states(1, 300, 8, 7)
    h[0, :, 3] = 1.25
    hb = bf16_bits(h)
    st = oracle_lib.hidden_stats(hb)
    assert st[0, 0, 3] == 1.25 and st[0, 1, 3] == 0.0
    ref = brute.bits_to_f64(hb)
    np.testing.assert_allclose(st[:, 0], ref.mean(axis=1), rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(st[:, 1], ref.std(axis=1), rtol=1e-10, atol=1e-13)


# ---------------------------------------------------------------- Eq. 5
def test_hidden_proxy_law(oracle_lib):
    """Samples ~ N(mu, diag((gamma sigma)^2)): standardised draws have mean 0,
    std 1 and pass a KS test; centring on 0 or scaling the variance by gamma
    fails."""
    h = hidden_states(1, 200, 32, 3, scale=2.0)
    st = oracle_lib.hidden_stats(h)
    P, gamma = 2048, 3.0
    hp = oracle_lib.hidden_proxies(st, P, gamma, seed=9, layer=2)
    x = brute.bits_to_f64(hp)[0]                           # [P, D]
    z = (x - st[0, 0]) / (gamma * st[0, 1])
    assert abs(z.mean()) < 0.01
    assert abs(z.std() - 1.0) < 0.01
    assert sps.kstest(z.ravel(), "norm").pvalue > 1e-3


def test_hidden_proxies_gamma_zero_and_seed_streams(oracle_lib):
    """gamma = 0 gives bf16(mu) in every sample; the hidden-space noise
    stream differs from every query head's stream and from other layers."""
    h = hidden_states(2, 64, 16, 4)
    st = oracle_lib.hidden_stats(h)
    hp0 = oracle_lib.hidden_proxies(st, 8, 0.0, seed=1)
    mu_bits = bf16_bits(st[:, 0].astype(np.float32))
    assert np.array_equal(hp0, np.broadcast_to(mu_bits[:, None, :], hp0.shape))
    a = oracle_lib.hidden_proxies(st, 8, 1.0, seed=1, layer=0)
    b = oracle_lib.hidden_proxies(st, 8, 1.0, seed=1, layer=1)
    assert not np.array_equal(a, b)
    z_hidden = oracle_lib.normal4(1, 0, 0, -1, 0, 0)
    z_head0 = oracle_lib.normal4(1, 0, 0, 0, 0, 0)
    assert not np.array_equal(z_hidden, z_head0)


# ---------------------------------------------------------------- Eq. 6
def test_projection_matches_float64_matmul(oracle_lib):
    """q[b, h, i] = W_Q^(h) H~[b, i] over the bf16 values: a transposed
    weight or a wrong head slice fails against a library matmul."""
    rng = np.random.default_rng(5)
    B, P, D, Hq, d = 2, 6, 40, 3, 8
    hp = bf16_bits(rng.standard_normal((B, P, D)))
    wq = bf16_bits(rng.standard_normal((Hq * d, D)) / math.sqrt(D))
    out, pre = oracle_lib.project_proxies(hp, wq, Hq, with_pre=True)
    x = brute.bits_to_f64(hp)
    w = brute.bits_to_f64(wq).reshape(Hq, d, D)
    ref = np.einsum("bpk,hek->bhpe", x, w) * brute.qscale(d)
    np.testing.assert_allclose(pre, ref, rtol=1e-12, atol=1e-14)
    assert np.array_equal(out, bf16_bits(pre.astype(np.float32)))


def test_projection_selection_matrix_and_rope(oracle_lib):
    """A one-hot W_Q copies hidden features into the heads (times the query
    scale log2(e)/sqrt(d)); identity rotary tables change nothing and
    general tables rotate (e, e + d/2) as the complex product
    (x_e + i x_{e+d/2}) (cos + i sin)."""
    rng = np.random.default_rng(6)
    B, P, D, Hq, d = 1, 4, 16, 2, 8
    hp = bf16_bits(rng.standard_normal((B, P, D)))
    sel = rng.permutation(D)[:Hq * d]
    w = np.zeros((Hq * d, D), dtype=np.float32)
    w[np.arange(Hq * d), sel] = 1.0
    wq = bf16_bits(w)
    out = oracle_lib.project_proxies(hp, wq, Hq)
    copied = brute.bits_to_f64(hp[:, None, :, sel].reshape(B, P, Hq, d).transpose(0, 2, 1, 3))
    assert np.array_equal(out, bf16_bits((copied * brute.qscale(d)).astype(np.float32)))
    ident = (np.ones(d // 2, np.float32), np.zeros(d // 2, np.float32))
    assert np.array_equal(oracle_lib.project_proxies(hp, wq, Hq, rope=ident), out)
    ang = rng.uniform(-3, 3, d // 2).astype(np.float32)
    rope = (np.cos(ang).astype(np.float32), np.sin(ang).astype(np.float32))
    _, pre = oracle_lib.project_proxies(hp, wq, Hq, rope=rope, with_pre=True)
    x = copied * brute.qscale(d)
    zc = (x[..., : d // 2] + 1j * x[..., d // 2:]) * (rope[0].astype(np.float64) + 1j * rope[1].astype(np.float64))
    np.testing.assert_allclose(pre[..., : d // 2], zc.real, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(pre[..., d // 2:], zc.imag, rtol=1e-12, atol=1e-14)


def test_hidden_gamma_zero_path_is_single_query_attention(oracle_lib):
    """gamma = 0: every proxy of head h is W_Q^(h) bf16(mu) (scaled by
    log2(e)/sqrt(d)); the group mass of every group is then
    g * sum_h softmax(ln(2) q~_h k) (Eq. 7-8 closed form), checked against
    scipy's softmax."""
    from scipy.special import softmax
    rng = np.random.default_rng(8)
    B, T, D, Hq, Hkv, d, P, G = 1, 50, 32, 2, 1, 8, 16, 1
    h = hidden_states(B, 20, D, 8)
    wq = bf16_bits(rng.standard_normal((Hq * d, D)) / math.sqrt(D))
    st = oracle_lib.hidden_stats(h)
    hp = oracle_lib.hidden_proxies(st, P, 0.0, seed=2)
    prox = oracle_lib.project_proxies(hp, wq, Hq)
    k = bf16_bits(rng.standard_normal((B, Hkv, T, d)))
    q_last = prox[:, :, 0, :].copy()
    gm, mass, an = oracle_lib.score(prox, q_last, k, Hkv, G)
    kq = brute.bits_to_f64(k)[0, 0]
    expect = np.zeros(T)
    for hh in range(Hq):
        qv = brute.bits_to_f64(prox[0, hh, 0])
        expect += softmax(kq @ qv * math.log(2.0))
    np.testing.assert_allclose(gm[0, 0, 0], P * expect, rtol=1e-12)
