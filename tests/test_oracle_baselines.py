"""Pins of the oracle's baseline selectors (test infrastructure, CPU only).

The paper compares against SnapKV, StreamingLLM and ExpectedAttn with the
settings of its appendix on the baselines (SnapKV: window 32, pooling
kernel 5, average pooling; StreamingLLM: 4 sinks and a recent window of the
remaining budget; ExpectedAttn: 512 samples without variance expansion and
4 sinks).  Each is a per-key score fed to the MASS-mode top-C; the pins
check the scores and selections against numpy and closed forms.
"""
import math

import numpy as np
import pytest
import torch
from scipy.special import softmax

import oracle
import brute


def bits(x):
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(torch.bfloat16).view(torch.uint16).numpy()


def topc(score, C):
    """indices of the C best by (score desc, index asc), ascending"""
    order = np.lexsort((np.arange(score.size), -score))
    return np.sort(order[:C])


@pytest.mark.parametrize("f32", [False, True])
def test_window_rows(f32):
    rng = np.random.default_rng(0)
    q = rng.normal(0, 2, (2, 3, 40, 64)).astype(np.float32)
    qin = q if f32 else bits(q)
    rows = oracle.window_rows(qin, 32)
    ref = brute.scale_to_bf16(brute.bits_to_f64(bits(q)[:, :, 8:]), 64)
    assert np.array_equal(brute.bits_to_f64(rows), ref)


def test_snapkv_scores_pooling():
    rng = np.random.default_rng(1)
    mass = rng.random((2, 3, 50))
    sc = oracle.shape_scores(mass, oracle.SHAPE_SNAPKV, window=7, pool=5)
    for b in range(2):
        for c in range(3):
            pre = np.convolve(mass[b, c, :43], np.ones(5), mode="same") / 5
            np.testing.assert_allclose(sc[b, c, :43], pre, rtol=1e-14)
            assert np.all(sc[b, c, 43:] == oracle.KEEP_SCORE)


def test_streaming_and_sinks_scores():
    mass = np.random.default_rng(2).random((1, 2, 30))
    st = oracle.shape_scores(mass, oracle.SHAPE_STREAMING, sinks=4)
    assert np.all(st[:, :, :4] == oracle.KEEP_SCORE)
    assert np.array_equal(st[0, 0, 4:], np.arange(4, 30, dtype=np.float64))
    sk = oracle.shape_scores(mass, oracle.SHAPE_SINKS, sinks=4)
    assert np.all(sk[:, :, :4] == oracle.KEEP_SCORE) and np.array_equal(sk[:, :, 4:], mass[:, :, 4:])


def small_layer(seed=3, T=90, W=40, d=64, Hq=4, Hkv=2):
    rng = np.random.default_rng(seed)
    q = bits(rng.normal(0, 1.5, (1, Hq, W, d)))
    k = bits(rng.normal(0, 1, (1, Hkv, T, d)))
    v = bits(rng.normal(0, 1, (1, Hkv, T, d)))
    return q, k, v


def test_streaming_selection_closed_form():
    q, k, v = small_layer()
    sel, _, _ = oracle.baseline_select("streaming", q, k, v, Hkv=2, budget=20, sinks=4)
    want = np.concatenate([np.arange(4), np.arange(90 - 16, 90)])
    for c in range(2):
        assert np.array_equal(sel.idx[0, c], want) and sel.counts[0, c] == 20


def test_snapkv_selection_matches_numpy():
    q, k, v = small_layer()
    T, d, win, C = 90, 64, 32, 45
    sel, sc, mass = oracle.baseline_select("snapkv", q, k, v, Hkv=2, budget=C, window=win, pool=5)
    rows = brute.scale_to_bf16(brute.bits_to_f64(q[:, :, -win:]), d)          # [1, Hq, win, d]
    kk = brute.bits_to_f64(k)
    for c in range(2):
        p = softmax(np.matmul(rows[0, 2 * c:2 * c + 2], kk[0, c].T) * math.log(2.0), axis=-1)   # [2, win, T]
        m = p.sum(axis=(0, 1))
        np.testing.assert_allclose(mass[0, c], m, rtol=1e-10)
        pooled = np.convolve(m[:T - win], np.ones(5), mode="same") / 5
        want = np.sort(np.concatenate([topc(pooled, C - win), np.arange(T - win, T)]))
        assert np.array_equal(sel.idx[0, c], want)


def test_expected_attention_selection():
    q, k, v = small_layer(seed=4)
    C = 30
    sel, sc, mass = oracle.baseline_select("expected", q, k, v, Hkv=2, budget=C, sinks=4, P=64, seed=9)
    # the proxies of ExpectedAttn are the gamma = 1 draws of the same generator
    prox, ql, _ = oracle.build_proxies(q, 64, 1.0, 9, 0)
    _, m2, _ = oracle.score(prox, ql, k, 2, 32)
    np.testing.assert_array_equal(mass, m2)
    for c in range(2):
        want = np.sort(np.concatenate([np.arange(4), 4 + topc(mass[0, c, 4:], C - 4)]))
        assert np.array_equal(sel.idx[0, c], want)

