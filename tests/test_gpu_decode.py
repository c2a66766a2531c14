"""Decode-time check on the GPU vs the CPU oracle (GPU).

The check measures the attention-mass coverage of Fig. 1b (the share of a
decoding query's softmax mass over all prompt keys that falls on the keys
kept after prefilling) and decode attention over the fixed compacted cache.
The selection, gather and check run through the C ABI; the oracle gets the
same decode queries, the same keys and the GPU's own selection and
compacted cache (gather is byte-exact, checked elsewhere).  Bars: coverage
within 1e-3 relative (fp32 exps and sums against fp64), attention outputs
within 1e-3 of the largest |v'| of their head (fp32 accumulation).
"""
import numpy as np
import pytest
import torch

import oracle
import parity
from paper_2607_22586_amd import binding as bd
from paper_2607_22586_amd import workloads as wl

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    bd.load_library()
    oracle.build()


def vals(a):
    """fp64 values of a bf16-bits (uint16) or fp32 array"""
    a = np.asarray(a)
    if a.dtype == np.uint16:
        return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return a.astype(np.float64)


def gpu_check(x, cfg, budget, c_max=None):
    q = x["q_win"].to(DEV)
    k, v = x["k"].to(DEV), x["v"].to(DEV)
    out = bd.select_layer(q, k, v, budget, cfg, c_max=c_max)
    cov, o = bd.decode_check(x["q_dec"].to(DEV), k, out.sel, out.k_out, out.v_out)
    torch.cuda.synchronize()
    tn = parity.to_np
    return tn(cov), tn(o), tn(out.sel.idx), tn(out.sel.counts), tn(out.k_out), tn(out.v_out)


def compare(x, g):
    cov, o, idx, counts, ko, vo = g
    rc, ro = oracle.decode_check(wl.to_numpy_bits(x["q_dec"]), wl.to_numpy_bits(x["k"]), idx, counts, ko, vo)
    err = parity.assert_close("coverage", cov, rc)
    B, Hq = cov.shape[:2]
    Hkv = counts.shape[1]
    vmax = np.abs(vals(vo)).max(axis=(2, 3))
    tol = 1e-3 * np.repeat(vmax, Hq // Hkv, axis=1)[:, :, None, None]
    bad = np.abs(o - ro) > tol
    assert not bad.any(), "decode attention outputs outside the bound: %d" % bad.sum()
    return err, rc


@pytest.mark.parametrize("name,n_dec,budget", [("tiny", 8, 64), ("tiny", 5, 300), ("qwen7b_4k", 16, 409),
                                               ("qwen7b_4k", 3, 100)])
def test_decode_check_parity(name, n_dec, budget):
    w = wl.WORKLOADS[name]
    x = wl.make_layer(w, 0, n_dec=n_dec)
    cfg = bd.SelectionConfig(seed=77, layer=0)
    g = gpu_check(x, cfg, budget)
    err, rc = compare(x, g)
    print("coverage rel err %.2e, mean coverage %.4f" % (err, float(rc.mean())), flush=True)


def test_decode_check_keep_all_ragged():
    """Budget above T keeps every key: coverage 1 and attention over the
    whole cache; T = 700 (a ragged key block), d = 64, 7 decode queries."""
    x = wl.custom_layer(1, 4, 2, 700, 4, 64, seed=5)
    x["q_dec"] = (2.0 * torch.randn((1, 4, 7, 64), generator=torch.Generator().manual_seed(9))).to(torch.bfloat16)
    cfg = bd.SelectionConfig(P=64, G=4, seed=3)
    g = gpu_check(x, cfg, budget=700, c_max=704)
    assert np.all(g[3] == 700)
    np.testing.assert_allclose(g[0], 1.0, rtol=0, atol=2e-6)
    compare(x, g)


def test_decode_check_fp32_cache():
    """fp32 K/V (the compacted cache keeps fp32, so decode attention takes the
    fp32 VALU kernel; coverage scores bf16-rounded keys as the prefill does):
    T = 700, d = 64, budget 300 (two chunks of cached keys), 6 decode queries."""
    x = wl.custom_layer(1, 4, 2, 700, 4, 64, dtype="fp32", seed=11)
    x["q_dec"] = (2.0 * torch.randn((1, 4, 6, 64), generator=torch.Generator().manual_seed(13))).to(torch.bfloat16)
    cfg = bd.SelectionConfig(P=64, G=4, seed=5)
    g = gpu_check(x, cfg, budget=300)
    assert g[4].dtype == np.float32
    compare(x, g)


def test_decode_check_full_size_sampled():
    """The benchmark's shape (B=4, T=16384, 28q/4kv, d=128, C=256) with 16
    decode queries per head: every row's coverage and output, checked against
    the oracle on two (batch row, KV head) pairs."""
    w = wl.WORKLOADS["qwen7b_16k_b4"]
    x = wl.make_layer(w, 1, n_dec=16)
    cfg = bd.SelectionConfig(seed=w.wid, layer=1)
    g = gpu_check(x, cfg, w.budget)
    cov, o, idx, counts, ko, vo = g
    Gh = w.Gh
    for b, c in [(0, 0), (3, 2)]:
        sl = slice(c * Gh, (c + 1) * Gh)
        rc, ro = oracle.decode_check(wl.to_numpy_bits(x["q_dec"])[b:b + 1, sl], wl.to_numpy_bits(x["k"])[b:b + 1, c:c + 1],
                                     idx[b:b + 1, c:c + 1], counts[b:b + 1, c:c + 1], ko[b:b + 1, c:c + 1],
                                     vo[b:b + 1, c:c + 1])
        parity.assert_close("coverage", cov[b:b + 1, sl], rc)
        vmax = np.abs(vals(vo[b, c])).max()
        assert np.all(np.abs(o[b:b + 1, sl] - ro) <= 1e-3 * vmax)
    assert np.all((cov > 0) & (cov <= 1 + 1e-6))
    print("mean coverage %.4f" % float(cov.mean()), flush=True)
