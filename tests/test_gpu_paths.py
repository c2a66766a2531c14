"""HIP paths that the workloads of the other parity tests do not reach (GPU),
each against the CPU oracle through the C ABI with the bars of
tests/parity.py:
  * the sweep form of the tau cut (more than 16384 keys per group) at a
    ragged key count, and the global-memory top-k (more than 32768 keys);
  * MASS mode on sampled heads of a full-size layer, in the benchmark's
    launch configuration;
  * rows whose base-2 logits are all large (every key identical, logits
    ~100-140): the per-row sums must stay finite and exact, so each proxy's
    softmax is uniform and the masses sum to P * Gh (Sec. 3.2.2 Eq. 7);
  * the hidden-state path with a dense W_Q (Sec. 3.2.1 Eq. 6): the GPU's own
    projected proxies fed to the oracle's scoring and selection, element by
    element on sampled heads.
"""
import numpy as np
import pytest
import torch

import brute
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


def gpu_layer(x, cfg, budget, prox=None, ql=None):
    q, k, v = (x[n].to(DEV) for n in ("q_win", "k", "v"))
    if prox is None:
        out = bd.select_layer(q, k, v, budget, cfg, want_votes=cfg.mode == bd.MMSKV_VOTE)
        prox, ql, sc, sel, ko, vo = out.proxies, out.q_last, out.scores, out.sel, out.k_out, out.v_out
    else:
        sc = bd.score(prox, ql, k, cfg, q.shape[2])
        sel = bd.select_topk(sc, cfg, budget, None, None, q.shape[1], q.shape[2],
                             want_votes=cfg.mode == bd.MMSKV_VOTE)
        ko, vo = bd.gather_kv(k, v, sel)
    torch.cuda.synchronize()
    tn = parity.to_np
    return dict(proxies=tn(prox), q_last=tn(ql),
                group_mass=None if sc.group_mass is None else tn(sc.group_mass),
                mass=tn(sc.mass), anchor=tn(sc.anchor), votes=None if sel.votes is None else tn(sel.votes),
                idx=tn(sel.idx), counts=tn(sel.counts), k_out=tn(ko), v_out=tn(vo))


def oracle_layer(x, cfg, budget):
    q, k, v = (wl.to_numpy_bits(x[n]) for n in ("q_win", "k", "v"))
    ref = oracle.select_layer(q, k, v, Hkv=k.shape[1], budget=budget, P=cfg.P, G=cfg.G, gamma=cfg.gamma,
                              tau=cfg.tau, lam=cfg.lam, seed=cfg.seed, layer=cfg.layer, mode=cfg.mode,
                              keep_last=cfg.keep_last)
    return ref, k, v


@pytest.mark.parametrize("T,Hq,budget,mode", [(20001, 4, 300, bd.MMSKV_VOTE), (32768, 2, 700, bd.MMSKV_VOTE),
                                              (40000, 2, 500, bd.MMSKV_VOTE), (40000, 2, 123, bd.MMSKV_MASS)])
def test_long_rows_sweep_paths(T, Hq, budget, mode):
    """16384 < T <= 32768 takes the 1024-thread register tau cut (ragged at
    T = 20001, full at 32768), T > 32768 the sweep tau cut and the global
    top-k."""
    print("case long rows", T, Hq, budget, mode, flush=True)
    x = wl.custom_layer(1, Hq, 1, T, 8, 64, seed=T + budget)
    cfg = bd.SelectionConfig(P=64, G=4, seed=T, mode=mode)
    g = gpu_layer(x, cfg, budget)
    ref, k, v = oracle_layer(x, cfg, budget)
    rep = parity.check_layer(g, ref, cfg, budget, k, v)
    print("long rows", (T, Hq, budget, mode), rep, flush=True)


def test_full_size_mass_mode_sampled_heads():
    """MASS mode (rank by total proxy mass) on one full layer of the 28-layer
    batch-4 T = 16384 workload; sampled heads recomputed by the oracle."""
    print("case full-size MASS", flush=True)
    w = wl.WORKLOADS["qwen7b_16k_b4"]
    layer = 7
    x = wl.make_layer(w, layer)
    cfg = bd.SelectionConfig(seed=w.wid, layer=layer, mode=bd.MMSKV_MASS)
    g = gpu_layer(x, cfg, w.budget)
    np.testing.assert_allclose(g["mass"].astype(np.float64).sum(-1), cfg.P * w.Gh, rtol=1e-3)
    Gh = w.Gh
    for (b, c) in ((0, 3), (2, 1)):
        q1 = wl.to_numpy_bits(x["q_win"][b:b + 1, c * Gh:(c + 1) * Gh].contiguous())
        k1 = wl.to_numpy_bits(x["k"][b:b + 1, c:c + 1].contiguous())
        v1 = wl.to_numpy_bits(x["v"][b:b + 1, c:c + 1].contiguous())
        prox, ql, _ = oracle.build_proxies(q1, cfg.P, cfg.gamma, cfg.seed, layer, b0=b, h0=c * Gh)
        gm, mass, an = oracle.score(prox, ql, k1, 1, cfg.G)
        sel = oracle.select(gm, mass, an, w.budget, cfg.tau, cfg.lam, mode=bd.MMSKV_MASS)
        ref = oracle.LayerResult(prox, ql, None, gm, mass, an, sel, None, None)
        gh = {key: (None if val is None else val[b:b + 1, c:c + 1] if key not in ("proxies", "q_last")
                    else val[b:b + 1, c * Gh:(c + 1) * Gh]) for key, val in g.items()}
        rep = parity.check_layer(gh, ref, cfg, w.budget, k1, v1)
        print("mass mode", (b, c), rep, flush=True)


def large_logit_layer(T, d, seed):
    """Every key the same vector beta*u and window queries alpha*u plus a
    spread, so each proxy row's logits are all equal and large (base 2,
    ~95-133 across rows with gamma = 4)."""
    g = torch.Generator()
    g.manual_seed(seed)
    u = torch.randn(d, generator=g)
    u = u / u.norm()
    alpha, beta = 80.0, 8.0
    k = (beta * u).expand(1, 1, T, d).contiguous()
    q = alpha * u + 1.4 * torch.randn((1, 4, 2, d), generator=g)
    v = torch.randn((1, 1, T, d), generator=g)
    return dict(q_win=q.to(torch.bfloat16).contiguous(), k=k.to(torch.bfloat16).contiguous(),
                v=v.to(torch.bfloat16).contiguous())


def test_large_logits_stay_exact():
    print("case large logits", flush=True)
    T, d = 16384, 64
    x = large_logit_layer(T, d, 7)
    cfg = bd.SelectionConfig(P=64, G=4, seed=5, gamma=4.0)
    g = gpu_layer(x, cfg, 256)
    # the rows' logits span the fast range's upper end and beyond
    s = brute.bits_to_f64(g["proxies"][0]) @ brute.bits_to_f64(wl.to_numpy_bits(x["k"][0, 0, 0]))
    assert s.min() < 110 and s.max() > 128, (s.min(), s.max())
    Gh = 4
    np.testing.assert_allclose(g["mass"], cfg.P * Gh / T, rtol=1e-4)
    np.testing.assert_allclose(g["group_mass"], (cfg.P // cfg.G) * Gh / T, rtol=1e-4)
    np.testing.assert_allclose(g["anchor"], 1.0 / T, rtol=1e-4)
    ref, k, v = oracle_layer(x, cfg, 256)
    parity.check_layer(g, ref, cfg, 256, k, v)
    # the decode-time coverage of the same keys is the kept share, exactly
    qd = (x["q_win"][:, :, -1:].float().expand(-1, -1, 3, -1)).to(torch.bfloat16).contiguous().to(DEV)
    sel = bd.Selected(torch.from_numpy(g["idx"]).to(DEV), torch.from_numpy(g["counts"]).to(DEV), None)
    cov, _ = bd.decode_check(qd, x["k"].to(DEV), sel, torch.from_numpy(g["k_out"]).view(torch.bfloat16).to(DEV),
                             torch.from_numpy(g["v_out"]).view(torch.bfloat16).to(DEV))
    torch.cuda.synchronize()
    np.testing.assert_allclose(cov.cpu().numpy(), 256.0 / T, rtol=1e-4)


def test_dense_wq_hidden_path_scores_and_selection():
    """Hidden-state proxies through a dense W_Q (every product rounded), at
    full size (B=4, T=16384, D=3584, 28 query / 4 KV heads): the GPU's
    projected proxies and anchor queries go to the oracle's scoring and
    selection (Sec. 3.2.2-3.2.3) on sampled heads, compared element by
    element; the projection itself is checked against its own bound in
    tests/test_gpu_hidden.py."""
    print("case dense W_Q hidden path", flush=True)
    w = wl.WORKLOADS["qwen7b_16k_b4"]
    layer = 2
    hx = wl.make_hidden(w, layer, device=DEV)
    x = wl.make_layer(w, layer, device=DEV)
    cfg = bd.SelectionConfig(seed=w.wid, layer=layer)
    st = bd.hidden_stats(hx["hidden"])
    hp = bd.hidden_proxies(st, cfg)
    prox = bd.project_proxies(hp, hx["wq"], w.Hq)
    ql = hx["q_last"]
    g = gpu_layer(x, cfg, w.budget, prox=prox, ql=ql)
    Gh = w.Gh
    for (b, c) in ((1, 2), (3, 0)):
        k1 = wl.to_numpy_bits(x["k"][b:b + 1, c:c + 1].contiguous())
        v1 = wl.to_numpy_bits(x["v"][b:b + 1, c:c + 1].contiguous())
        p1 = g["proxies"][b:b + 1, c * Gh:(c + 1) * Gh]
        q1 = g["q_last"][b:b + 1, c * Gh:(c + 1) * Gh]
        gm, mass, an = oracle.score(p1, q1, k1, 1, cfg.G)
        sel = oracle.select(gm, mass, an, w.budget, cfg.tau, cfg.lam)
        ref = oracle.LayerResult(p1, q1, None, gm, mass, an, sel, None, None)
        gh = {key: (None if val is None else val[b:b + 1, c:c + 1] if key not in ("proxies", "q_last")
                    else val[b:b + 1, c * Gh:(c + 1) * Gh]) for key, val in g.items()}
        rep = parity.check_layer(gh, ref, cfg, w.budget, k1, v1)
        print("dense W_Q", (b, c), rep, flush=True)


@pytest.mark.parametrize("mode", ["vote", "mass"])
@pytest.mark.parametrize("T", [16384, 3001, 40000])
def test_select_stage_calls_equal_whole_call(T, mode):
    """mmshiftkv_select_tau, _vote and _pick in order give exactly what
    mmshiftkv_select_topk gives (register and sweep paths, both modes)."""
    print("case select stages", T, mode, flush=True)
    dev = torch.device(DEV)
    m = bd.MMSKV_MASS if mode == "mass" else bd.MMSKV_VOTE
    cfg = bd.SelectionConfig(P=64, G=4, seed=T + m, mode=m)
    B, Hkv, Gh, d, W = 2, 2, 2, 64, 16
    torch.manual_seed(T)
    q = torch.randn(B, Hkv * Gh, W, d, device=dev).to(torch.bfloat16)
    k = torch.randn(B, Hkv, T, d, device=dev).to(torch.bfloat16)
    prox, ql = bd.build_proxies(q, cfg, T, Hkv)
    sc = bd.score(prox, ql, k, cfg, W)
    whole = bd.select_topk(sc, cfg, 200, Hq=Hkv * Gh, W=W, want_votes=(m == bd.MMSKV_VOTE))
    ws = torch.empty(bd.select_workspace(B, Hkv * Gh, Hkv, T, W, d, cfg), dtype=torch.uint8, device=dev)
    out = bd.Selected(torch.full_like(whole.idx, -7), torch.full_like(whole.counts, -7),
                      None if whole.votes is None else torch.full_like(whole.votes, 99))
    for stg in ("tau", "vote", "pick"):
        bd.select_topk(sc, cfg, 200, Hq=Hkv * Gh, W=W, out=out, workspace=ws, stage=stg)
    torch.cuda.synchronize()
    assert torch.equal(out.idx, whole.idx)
    assert torch.equal(out.counts, whole.counts)
    if whole.votes is not None:
        assert torch.equal(out.votes, whole.votes)


@pytest.mark.parametrize("Gh,T,P", [(5, 16384, 512), (6, 16384, 512), (7, 16384, 512), (8, 16384, 512),
                                    (7, 16000, 512), (7, 16384, 32)])
def test_early_phases_equal_the_plain_pipeline(Gh, T, P):
    """The early phases of both score passes (the first 8 proxy tiles taken
    sub-tile by sub-tile while the keys arrive; bf16 keys, full key blocks)
    sum in the pipeline's order, so they must give the same bits as the
    plain pipeline.  fp32 keys that hold bf16 values are scored exactly like
    the bf16 keys but always take the plain pipeline, so the two calls are
    compared bit for bit, at a shape where both passes use their early
    phase (batch 4, 4 KV heads, T = 16384: 1024-key pass-1 blocks and
    8-wave pass-2 blocks); at T = 16000 the last key block of each head is
    ragged and takes the plain pipeline within the same launch; with P = 32
    (one 32-row tile per head) neither pass has tiles enough for its early
    phase and both take the plain pipeline."""
    B, Hkv, d, W = 4, 4, 128, 16
    Hq = Gh * Hkv
    g = torch.Generator(device="cpu").manual_seed(100 + Gh + T + P)
    q = torch.randn((B, Hq, W, d), generator=g).to(torch.bfloat16).to(DEV)
    k = torch.randn((B, Hkv, T, d), generator=g).to(torch.bfloat16).to(DEV)
    cfg = bd.SelectionConfig(seed=7, layer=Gh, P=P, G=P // 16)
    prox, ql = bd.build_proxies(q, cfg, T, Hkv)
    a = bd.score(prox, ql, k, cfg, W)
    b = bd.score(prox, ql, k.float(), cfg, W)
    torch.cuda.synchronize()
    for u, v in ((a.group_mass, b.group_mass), (a.mass, b.mass), (a.anchor, b.anchor)):
        assert torch.equal(u, v)
    # and the masses are a softmax's: P * Gh in total per (b, c)
    tot = a.mass.double().sum(dim=2)
    assert torch.allclose(tot, torch.full_like(tot, cfg.P * Gh), rtol=1e-4)
