"""Pins of the oracle's decode-time check (test infrastructure, CPU only).

The check measures the attention-mass coverage of Fig. 1b (the share of a
decoding query's softmax mass, over all prompt keys, that falls on the keys
kept after prefilling) and decode attention over the fixed compacted cache
(Sec. 3.1 prefill-only protocol).  The oracle is pinned against an
independent numpy/scipy computation, closed forms and invariants.
"""
import math

import numpy as np
import pytest
import torch
from scipy.special import softmax

import oracle
import brute

pytestmark = pytest.mark.filterwarnings("ignore::DeprecationWarning")


def to_bits(x):
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(torch.bfloat16).view(torch.uint16).numpy()


def make(B=1, Hq=4, Hkv=2, T=50, d=64, n_dec=3, seed=0, kbits=True):
    rng = np.random.default_rng(seed)
    q = to_bits(rng.normal(0, 2.0, (B, Hq, n_dec, d)))
    k = rng.normal(0, 1.0, (B, Hkv, T, d)).astype(np.float32)
    v = rng.normal(0, 1.0, (B, Hkv, T, d)).astype(np.float32)
    if kbits:
        k, v = to_bits(k), to_bits(v)
    return q, k, v


def f64(a):
    a = np.asarray(a)
    return brute.bits_to_f64(a) if a.dtype == np.uint16 else a.astype(np.float32).astype(np.float64)


def kbf16(a):
    """keys as the scoring sees them: fp32 keys rounded to bf16 (nearest even)"""
    a = np.asarray(a)
    return brute.bits_to_f64(a if a.dtype == np.uint16 else to_bits(a))


def compact(x, idx, counts):
    B, H, T, d = x.shape
    c_max = idx.shape[2]
    out = np.zeros((B, H, c_max, d), dtype=x.dtype)
    for b in range(B):
        for c in range(H):
            n = counts[b, c]
            out[b, c, :n] = x[b, c, idx[b, c, :n]]
    return out


def reference(q, k, v, idx, counts):
    """numpy/scipy: softmax(ln 2 * q~ . k) over all keys, coverage = its sum
    over the kept keys; attention of q~ over the kept rows only."""
    B, Hq, n_dec, d = q.shape
    Hkv = k.shape[1]
    Gh = Hq // Hkv
    qs = brute.scale_to_bf16(brute.bits_to_f64(q), d)
    kk, vv = kbf16(k), f64(v)
    cov = np.zeros((B, Hq, n_dec))
    out = np.zeros((B, Hq, n_dec, d))
    for b in range(B):
        for h in range(Hq):
            c = h // Gh
            kept = idx[b, c, :counts[b, c]]
            p = softmax(qs[b, h] @ kk[b, c].T * math.log(2.0), axis=-1)
            cov[b, h] = p[:, kept].sum(-1)
            pk = softmax(qs[b, h] @ kk[b, c, kept].T * math.log(2.0), axis=-1)
            out[b, h] = pk @ vv[b, c, kept]
    return cov, out


@pytest.mark.parametrize("kbits", [True, False])
def test_keep_all_is_full_attention(kbits):
    q, k, v = make(kbits=kbits)
    B, Hkv, T = k.shape[:3]
    idx = np.broadcast_to(np.arange(T, dtype=np.int32), (B, Hkv, T)).copy()
    counts = np.full((B, Hkv), T, dtype=np.int32)
    cov, out = oracle.decode_check(q, k, idx, counts, k, v)
    np.testing.assert_allclose(cov, 1.0, rtol=0, atol=1e-12)
    rc, ro = reference(q, k, v, idx, counts)
    np.testing.assert_allclose(out, ro, rtol=1e-10, atol=1e-13)


@pytest.mark.parametrize("kbits", [True, False])
def test_random_subset_matches_numpy(kbits):
    q, k, v = make(B=2, Hq=6, Hkv=3, T=70, n_dec=4, seed=3, kbits=kbits)
    B, Hkv, T = k.shape[:3]
    rng = np.random.default_rng(7)
    c_max = 20
    idx = np.full((B, Hkv, c_max), -1, dtype=np.int32)
    counts = np.zeros((B, Hkv), dtype=np.int32)
    for b in range(B):
        for c in range(Hkv):
            n = int(rng.integers(1, c_max + 1))
            idx[b, c, :n] = np.sort(rng.choice(T, n, replace=False))
            counts[b, c] = n
    ko, vo = compact(k, idx, counts), compact(v, idx, counts)
    cov, out = oracle.decode_check(q, k, idx, counts, ko, vo)
    rc, ro = reference(q, k, v, idx, counts)
    np.testing.assert_allclose(cov, rc, rtol=1e-11)
    np.testing.assert_allclose(out, ro, rtol=1e-10, atol=1e-13)
    assert np.all((cov > 0) & (cov < 1))


def test_identical_keys_closed_form():
    """Identical keys: every softmax is uniform, so coverage = n / T exactly and
    the compacted attention output is the mean of the kept value rows."""
    q, k, v = make(T=40, seed=5)
    k[:] = k[:, :, :1]
    B, Hkv, T = k.shape[:3]
    idx = np.full((B, Hkv, 12), -1, dtype=np.int32)
    counts = np.array([[12, 5]], dtype=np.int32)
    idx[0, 0, :12] = np.arange(0, 36, 3)
    idx[0, 1, :5] = [1, 2, 20, 30, 39]
    ko, vo = compact(k, idx, counts), compact(v, idx, counts)
    cov, out = oracle.decode_check(q, k, idx, counts, ko, vo)
    Gh = 2
    for h in range(4):
        c = h // Gh
        n = counts[0, c]
        np.testing.assert_allclose(cov[0, h], n / T, rtol=1e-13)
        np.testing.assert_allclose(out[0, h], np.broadcast_to(f64(v)[0, c, idx[0, c, :n]].mean(0), out[0, h].shape),
                                   rtol=1e-12, atol=1e-14)


def test_dominant_key():
    """A key far along the query's direction takes almost all the mass: the
    coverage is ~1 when it is kept and ~0 when it is not."""
    q, k, v = make(Hq=2, Hkv=1, T=64, n_dec=1, seed=9, kbits=False)
    qv = brute.bits_to_f64(q)[0, 0, 0]
    k[0, 0, 17] = (40.0 * qv / np.linalg.norm(qv)).astype(np.float32)
    idx_in = np.array([[[3, 17, 40]]], dtype=np.int32)
    idx_out = np.array([[[3, 18, 40]]], dtype=np.int32)
    counts = np.array([[3]], dtype=np.int32)
    c_in, _ = oracle.decode_check(q[:, :1], k, idx_in, counts, compact(k, idx_in, counts), compact(v, idx_in, counts))
    c_out, _ = oracle.decode_check(q[:, :1], k, idx_out, counts, compact(k, idx_out, counts), compact(v, idx_out, counts))
    assert c_in[0, 0, 0] > 1 - 1e-9 and c_out[0, 0, 0] < 1e-9


def test_permutation_invariance():
    q, k, v = make(B=1, Hq=2, Hkv=1, T=33, n_dec=2, seed=11)
    T = k.shape[2]
    idx = np.array([[[0, 4, 5, 19, 31]]], dtype=np.int32)
    counts = np.array([[5]], dtype=np.int32)
    cov, out = oracle.decode_check(q, k, idx, counts, compact(k, idx, counts), compact(v, idx, counts))
    perm = np.random.default_rng(2).permutation(T)
    inv = np.argsort(perm)
    kp, vp = k[:, :, perm], v[:, :, perm]
    idxp = np.sort(inv[idx[0, 0]])[None, None].astype(np.int32)
    cov2, out2 = oracle.decode_check(q, kp, idxp, counts, compact(kp, idxp, counts), compact(vp, idxp, counts))
    np.testing.assert_allclose(cov2, cov, rtol=1e-12)
    np.testing.assert_allclose(out2, out, rtol=1e-12, atol=1e-14)


def test_rejects_bad_indices():
    q, k, v = make()
    idx = np.zeros((1, 2, 3), dtype=np.int32)
    idx[0, 1, 2] = 50
    counts = np.full((1, 2), 3, dtype=np.int32)
    with pytest.raises(ValueError):
        oracle.decode_check(q, k, idx, counts, compact(k, np.zeros_like(idx), counts), compact(v, np.zeros_like(idx), counts))
