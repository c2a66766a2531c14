"""Baseline selectors on the library's kernels vs the CPU oracle (GPU).

SnapKV (window rows scored by the mass pass, average-pooled), StreamingLLM
(sinks and recency) and ExpectedAttn (gamma = 1 proxies, sinks) run through
the C ABI on the same scoring, top-k and gather kernels as the method.
Bars: window rows bit-exact; pooled / sink scores within 1e-6 relative of
the oracle's on the GPU's own masses; masses within 1e-3 relative of the
oracle's; the selection exactly the top-C of the GPU's own scores and
consistent with the oracle's scores widened by 1e-3; StreamingLLM exact.
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


@pytest.mark.parametrize("name", ["tiny", "qwen7b_4k"])
def test_window_rows_bit_exact(name):
    w = wl.WORKLOADS[name]
    x = wl.make_layer(w, 0)
    n = 16 if w.W < 32 else 32
    rows, ql = bd.window_rows(x["q_win"].to(DEV), n, w.T, w.Hkv)
    torch.cuda.synchronize()
    q = wl.to_numpy_bits(x["q_win"])
    assert np.array_equal(parity.to_np(rows), oracle.window_rows(q, n))
    _, rql, _ = oracle.build_proxies(q, 32, 0.0, 0, 0)
    assert np.array_equal(parity.to_np(ql), rql)


def test_shape_scores_match_oracle():
    rng = np.random.default_rng(0)
    mass = torch.from_numpy(rng.random((2, 3, 1000)).astype(np.float32))
    m64 = mass.double().numpy()
    for kind, kw in [(bd.MMSKV_SHAPE_SNAPKV, dict(window=32, pool=5)), (bd.MMSKV_SHAPE_STREAMING, dict(sinks=4)),
                     (bd.MMSKV_SHAPE_SINKS, dict(sinks=4)), (bd.MMSKV_SHAPE_SNAPKV, dict(window=0, pool=1))]:
        g = bd.shape_scores(mass.to(DEV), kind, 2, 3, 1000, **kw)
        torch.cuda.synchronize()
        ref = oracle.shape_scores(m64, kind, **kw)
        np.testing.assert_allclose(g.double().cpu().numpy(), ref, rtol=1e-6, atol=0)


def own_topc(score, C):
    return np.sort(np.lexsort((np.arange(score.size), -score))[:C])


@pytest.mark.parametrize("name,baseline,budget", [
    ("qwen7b_4k", "snapkv", 409), ("qwen7b_4k", "expected", 409), ("qwen7b_4k", "streaming", 409),
    ("tiny", "expected", 64), ("tiny", "streaming", 64), ("qwen7b_4k", "snapkv", 100)])
def test_baseline_parity(name, baseline, budget):
    w = wl.WORKLOADS[name]
    x = wl.make_layer(w, 0)
    seed = 31
    sel, sc, mass, ko, vo = bd.baseline_select(baseline, x["q_win"].to(DEV), x["k"].to(DEV), x["v"].to(DEV),
                                               budget, seed=seed, P=512)
    torch.cuda.synchronize()
    q, k, v = (wl.to_numpy_bits(x[n]) for n in ("q_win", "k", "v"))
    rsel, rsc, rmass = oracle.baseline_select(baseline, q, k, v, Hkv=w.Hkv, budget=budget, seed=seed, P=512)
    idx, counts = parity.to_np(sel.idx), parity.to_np(sel.counts)
    gsc = sc.double().cpu().numpy()
    if baseline == "streaming":
        assert np.array_equal(idx, rsel.idx) and np.array_equal(counts, rsel.counts)
    else:
        parity.assert_close("mass", mass.cpu().numpy(), rmass)
        for b in range(w.B):
            for c in range(w.Hkv):
                got = idx[b, c, :counts[b, c]]
                assert np.array_equal(got, own_topc(gsc[b, c], budget))
                parity.check_selection_interval(got, rsc[b, c], 1e-3 * np.abs(rsc[b, c]), w.T, budget, keep_last=False)
    # the gather of the baseline's selection is byte-exact
    assert np.array_equal(parity.to_np(ko), oracle.gather(k, idx, counts))
    assert np.array_equal(parity.to_np(vo), oracle.gather(v, idx, counts))
