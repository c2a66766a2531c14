"""HIP path vs the CPU oracle, element by element, on seeded inputs (GPU).

Every call goes through the C ABI (ctypes binding); the oracle runs on the
same inputs on the host.  Bars: proxies bit-exact; group mass / mass /
anchor within 1e-3 relative; votes and selections identical outside the
oracle's ambiguity band and exactly consistent with the GPU's own scores;
gather byte-exact.  See tests/parity.py for the comparators.
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


def run_gpu(x, cfg, budget, c_max=None, budgets=None, rope_f=None, rope_l=None, k=None, v=None):
    q = x["q_win"].to(DEV)
    k = (x["k"] if k is None else k).to(DEV)
    v = (x["v"] if v is None else v).to(DEV)
    bt = None if budgets is None else torch.as_tensor(budgets, dtype=torch.int32, device=DEV)
    out = bd.select_layer(q, k, v, budget, cfg, c_max=c_max, budgets=bt, rope_f=rope_f, rope_l=rope_l,
                          want_votes=cfg.mode == bd.MMSKV_VOTE)
    torch.cuda.synchronize()
    tn = parity.to_np
    return dict(proxies=tn(out.proxies), q_last=tn(out.q_last),
                group_mass=None if out.scores.group_mass is None else tn(out.scores.group_mass),
                mass=tn(out.scores.mass), anchor=tn(out.scores.anchor),
                votes=None if out.sel.votes is None else tn(out.sel.votes),
                idx=tn(out.sel.idx), counts=tn(out.sel.counts), k_out=tn(out.k_out), v_out=tn(out.v_out))


def run_oracle(x, cfg, budget, c_max=None, rope_f=None, rope_l=None, Hkv=None):
    q, k, v = (wl.to_numpy_bits(x[n]) for n in ("q_win", "k", "v"))
    Hkv = k.shape[1] if Hkv is None else Hkv
    np_rope = lambda r: None if r is None else (r[0].numpy(), r[1].numpy())  # noqa: E731
    return oracle.select_layer(q, k, v, Hkv=Hkv, budget=budget, P=cfg.P, G=cfg.G, gamma=cfg.gamma,
                               tau=cfg.tau, lam=cfg.lam, seed=cfg.seed, layer=cfg.layer,
                               ddof=cfg.std_ddof, mode=cfg.mode, keep_last=cfg.keep_last, c_max=c_max,
                               rope_f=np_rope(rope_f), rope_l=np_rope(rope_l)), k, v


def parity_case(x, cfg, budget, **kw):
    g = run_gpu(x, cfg, budget)
    ref, k, v = run_oracle(x, cfg, budget)
    rep = parity.check_layer(g, ref, cfg, budget, k, v, keep_last=cfg.keep_last, **kw)
    print("report", rep, flush=True)
    return g, ref, rep


# ---------------------------------------------------------------- proxies
@pytest.mark.parametrize("name,ddof,rope,gamma", [
    ("tiny", 0, False, 10.0), ("qwen7b_4k", 0, False, 10.0), ("qwen7b_4k", 1, False, 3.0),
    ("tiny", 0, True, 10.0), ("qwen7b_4k", 0, True, 0.0)])
def test_proxies_bit_exact(name, ddof, rope, gamma):
    w = wl.WORKLOADS[name]
    x = wl.make_layer(w, 0)
    cfg = bd.SelectionConfig(seed=1234 + ddof, layer=5, std_ddof=ddof, gamma=gamma)
    rf = wl.rope_tables(w.d, w.T + 17) if rope else None
    rl = wl.rope_tables(w.d, w.T - 1) if rope else None
    prox, ql, st = bd.build_proxies(x["q_win"].to(DEV), cfg, w.T, w.Hkv, rf, rl, with_stats=True)
    torch.cuda.synchronize()
    rp, rq, rs = oracle.build_proxies(wl.to_numpy_bits(x["q_win"]), cfg.P, cfg.gamma, cfg.seed, cfg.layer,
                                      ddof, None if rf is None else (rf[0].numpy(), rf[1].numpy()),
                                      None if rl is None else (rl[0].numpy(), rl[1].numpy()))
    assert np.array_equal(st.cpu().numpy(), rs), "window statistics differ (fp64 bits)"
    assert np.array_equal(parity.to_np(ql), rq)
    assert np.array_equal(parity.to_np(prox), rp)


# ---------------------------------------------------------------- full pipeline
CASES = {
    # name: (inputs, cfg kwargs, budget)
    "tiny_vote": (lambda: wl.make_layer("tiny", 0), dict(seed=0), 64),
    "tiny_mass": (lambda: wl.make_layer("tiny", 0), dict(seed=0, mode=bd.MMSKV_MASS), 64),
    "qwen7b_4k_vote": (lambda: wl.make_layer("qwen7b_4k", 0), dict(seed=1), 409),
    "ragged_gqa4": (lambda: wl.custom_layer(2, 8, 2, 1000, 7, 128, seed=3), dict(P=64, G=4, seed=3), 100),
    "short_T37": (lambda: wl.custom_layer(1, 4, 2, 37, 5, 64, seed=4), dict(P=32, G=2, seed=4), 10),
    "T1": (lambda: wl.custom_layer(1, 2, 1, 1, 3, 64, seed=5), dict(P=32, G=2, seed=5), 4),
    "T2_budget1": (lambda: wl.custom_layer(1, 2, 1, 2, 3, 64, seed=6), dict(P=32, G=2, seed=6), 1),
    "budget_ge_T": (lambda: wl.custom_layer(1, 4, 1, 300, 8, 64, seed=7), dict(P=32, G=2, seed=7), 300),
    "mha_d64": (lambda: wl.custom_layer(1, 3, 3, 600, 9, 64, seed=8), dict(P=64, G=4, seed=8), 50),
    "mqa_gh20": (lambda: wl.custom_layer(1, 20, 1, 700, 6, 64, seed=9), dict(P=32, G=2, seed=9), 70),
    "no_keep_last": (lambda: wl.custom_layer(1, 4, 1, 500, 8, 128, seed=10),
                     dict(P=64, G=4, seed=10, keep_last=False), 40),
    "tau_one": (lambda: wl.custom_layer(1, 4, 1, 400, 8, 64, seed=11), dict(P=64, G=4, seed=11, tau=1.0), 30),
    "lambda_zero": (lambda: wl.custom_layer(1, 4, 1, 400, 8, 64, seed=12), dict(P=64, G=4, seed=12, lam=0.0), 30),
    "lambda_50": (lambda: wl.custom_layer(1, 4, 1, 400, 8, 64, seed=13), dict(P=64, G=4, seed=13, lam=50.0), 30),
    "gamma_zero": (lambda: wl.custom_layer(1, 4, 2, 513, 8, 128, seed=14), dict(P=32, G=2, seed=14, gamma=0.0), 33),
    "fp32_d128_mass": (lambda: wl.custom_layer(2, 4, 2, 777, 8, 128, dtype="f32", seed=15),
                       dict(P=64, G=4, seed=15, mode=bd.MMSKV_MASS), 60),
    "window_150": (lambda: wl.custom_layer(1, 4, 1, 520, 150, 128, seed=16), dict(P=64, G=4, seed=16), 50),
    "identical_keys": (lambda: _identical_keys(), dict(P=64, G=4, seed=17), 64),
}


def _identical_keys():
    """Every key equal: equal masses everywhere, so tau-sets and the top-k are
    decided by index order alone (the equal-mass paths of the selection)."""
    x = wl.custom_layer(1, 4, 1, 1024, 16, 64, seed=17)
    x["k"] = x["k"][:, :, :1].expand(-1, -1, 1024, -1).contiguous()
    return x


@pytest.mark.parametrize("case", sorted(CASES))
def test_pipeline_parity(case):
    make, kw, budget = CASES[case]
    x = make()
    parity_case(x, bd.SelectionConfig(**kw), budget)


def test_tiny_keeps_planted_keys():
    x = wl.make_layer("tiny", 0)
    g = run_gpu(x, bd.SelectionConfig(seed=0), 64)
    assert set(x["planted"][0, 0].tolist()) <= set(g["idx"][0, 0].tolist())


def test_rope_pipeline():
    w = wl.WORKLOADS["tiny"]
    x = wl.make_layer(w, 0)
    cfg = bd.SelectionConfig(seed=3)
    rf, rl = wl.rope_tables(w.d, w.T + 64), wl.rope_tables(w.d, w.T - 1)
    g = run_gpu(x, cfg, 64, rope_f=rf, rope_l=rl)
    ref, k, v = run_oracle(x, cfg, 64, rope_f=rf, rope_l=rl)
    parity.check_layer(g, ref, cfg, 64, k, v)


def test_strided_keys_and_values():
    """K/V passed as strided views (every other head of a larger cache)."""
    x = wl.custom_layer(2, 8, 4, 640, 8, 128, seed=21)
    big_k = torch.zeros((2, 8, 640, 128), dtype=torch.bfloat16)
    big_v = torch.zeros_like(big_k)
    big_k[:, ::2] = x["k"]
    big_v[:, ::2] = x["v"]
    cfg = bd.SelectionConfig(P=64, G=4, seed=21)
    kd, vd = big_k.to(DEV)[:, ::2], big_v.to(DEV)[:, ::2]
    assert not kd.is_contiguous()
    g = run_gpu(x, cfg, 77, k=kd, v=vd)
    ref, k, v = run_oracle(x, cfg, 77)
    parity.check_layer(g, ref, cfg, 77, k, v)


def test_per_head_budgets():
    x = wl.custom_layer(2, 8, 2, 900, 8, 128, seed=22)
    budgets = np.array([[5, 100], [1, 900]], dtype=np.int32)
    cfg = bd.SelectionConfig(P=64, G=4, seed=22)
    g = run_gpu(x, cfg, 1, c_max=900, budgets=budgets)
    ref, k, v = run_oracle(x, cfg, 900, c_max=900)
    for b in range(2):
        for c in range(2):
            bud = int(budgets[b, c])
            s = oracle.select(ref.group_mass[b:b + 1, c:c + 1], ref.mass[b:b + 1, c:c + 1],
                              ref.anchor[b:b + 1, c:c + 1], bud, cfg.tau, cfg.lam, c_max=900)
            ref.sel.idx[b, c] = s.idx[0, 0]
            ref.sel.counts[b, c] = s.counts[0, 0]
    parity.check_layer(g, ref, cfg, None, k, v, budgets=budgets)


def test_split_passes_equal_fused_and_deterministic():
    """score = score_lse then score_mass = score_lse_blocks, score_lse_merge,
    score_mass, bit for bit (and the same twice)."""
    x = wl.make_layer("qwen7b_4k", 0)
    cfg = bd.SelectionConfig(seed=2)
    q, k = x["q_win"].to(DEV), x["k"].to(DEV)
    prox, ql = bd.build_proxies(q, cfg, k.shape[2], k.shape[1])
    a = bd.score(prox, ql, k, cfg, q.shape[2])
    ws = torch.empty(bd.score_workspace(1, 28, 4, 4096, 32, 128, cfg), dtype=torch.uint8, device=DEV)
    bd.score_lse(prox, ql, k, cfg, ws, q.shape[2])
    b = bd.score_mass(prox, ql, k, cfg, ws, q.shape[2])
    c = bd.score(prox, ql, k, cfg, q.shape[2])
    # the log-sum-exp pass as its two stage calls (blocks, then merge)
    ws2 = torch.full_like(ws, 0x7F)
    bd.score_lse(prox, ql, k, cfg, ws2, q.shape[2], stage="blocks")
    bd.score_lse(prox, ql, k, cfg, ws2, q.shape[2], stage="merge")
    e = bd.score_mass(prox, ql, k, cfg, ws2, q.shape[2])
    sa = bd.select_topk(a, cfg, 409, Hq=28, want_votes=True)
    sc = bd.select_topk(c, cfg, 409, Hq=28, want_votes=True)
    torch.cuda.synchronize()
    for u, w_ in ((a.group_mass, b.group_mass), (a.mass, b.mass), (a.anchor, b.anchor),
                  (a.group_mass, c.group_mass), (a.anchor, c.anchor),
                  (a.group_mass, e.group_mass), (a.mass, e.mass), (a.anchor, e.anchor)):
        assert torch.equal(u, w_)
    assert torch.equal(sa.idx, sc.idx) and torch.equal(sa.votes, sc.votes)


# ---------------------------------------------------------------- full sizes, sampled heads
@pytest.mark.parametrize("name,heads", [("qwen7b_8k", [(0, 1)]), ("qwen7b_16k_b4", [(1, 2), (3, 0)]),
                                        ("large_32k", [(0, 5)])])
def test_full_size_sampled_heads(name, heads):
    """One layer at full size, in the launch configuration the benchmark
    times; the oracle recomputes sampled (batch row, KV head) pairs on their
    own (their proxies use the global generator counters)."""
    w = wl.WORKLOADS[name]
    layer = 3
    x = wl.make_layer(w, layer)
    cfg = bd.SelectionConfig(seed=w.wid, layer=layer)
    g = run_gpu(x, cfg, w.budget)
    # properties that hold for every head
    Gh = w.Gh
    np.testing.assert_allclose(g["mass"].astype(np.float64).sum(-1), cfg.P * Gh, rtol=1e-3)
    np.testing.assert_allclose(g["anchor"].astype(np.float64).sum(-1), 1.0, rtol=1e-3)
    np.testing.assert_allclose(g["group_mass"].astype(np.float64).sum(-1), 16 * Gh, rtol=1e-3)
    assert np.all(g["counts"] == w.budget)
    assert np.all(g["idx"][:, :, -1] == w.T - 1)
    assert np.all(np.diff(g["idx"], axis=-1) > 0)
    qn, kn, vn = (wl.to_numpy_bits(x[n]) for n in ("q_win", "k", "v"))
    for (b, c) in heads:
        sub = {n: x[n][b:b + 1] for n in ("q_win", "k", "v")}
        sub["q_win"] = sub["q_win"][:, c * Gh:(c + 1) * Gh]
        sub["k"] = sub["k"][:, c:c + 1]
        sub["v"] = sub["v"][:, c:c + 1]
        q1, k1, v1 = (wl.to_numpy_bits(sub[n].contiguous()) for n in ("q_win", "k", "v"))
        prox, ql, _ = oracle.build_proxies(q1, cfg.P, cfg.gamma, cfg.seed, layer, b0=b, h0=c * Gh)
        gm, mass, an = oracle.score(prox, ql, k1, 1, cfg.G)
        sel = oracle.select(gm, mass, an, w.budget, cfg.tau, cfg.lam)
        ref = oracle.LayerResult(prox, ql, None, gm, mass, an, sel, None, None)
        gh = {key: (None if val is None else val[b:b + 1, c:c + 1] if key not in ("proxies", "q_last")
                    else val[b:b + 1, c * Gh:(c + 1) * Gh]) for key, val in g.items()}
        rep = parity.check_layer(gh, ref, cfg, w.budget, k1, v1)
        print(name, (b, c), rep, flush=True)
    del qn, kn, vn
