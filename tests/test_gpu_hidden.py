"""Hidden-state form of the proxies (Sec. 3.2.1 Eqs. 4-6; Algorithm 1): HIP
path vs the CPU oracle through the C ABI (GPU).

Bars: statistics within the fp64 rounding bound of the GPU's summation
against the oracle's two-pass definition (parity.check_hidden_stats);
hidden-space samples bit-exact given the same statistics (same counter-based
generator); projected proxies within
half a bf16 ulp plus an fp32 accumulation bound of the oracle's fp64 values
(the GPU sums bf16 products in fp32 on the matrix cores), and identical to
bf16(fp32(oracle)) for at least 99% of the entries.  With a W_Q whose
products are exact (one +-1 / +-2 entry per row) the whole layer -- proxies,
masses, votes, selection, gather -- meets the same bars as the query-space
path.
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


def bits(t):
    return wl.to_numpy_bits(t)


def values(a):
    """fp64 values of an oracle input array (fp32, or bf16 bits as uint16)."""
    return a.astype(np.float64) if a.dtype == np.float32 else brute.bits_to_f64(a)


def bf16_ulp(x):
    """Spacing of bf16 numbers at |x| (normal range)."""
    _, e = np.frexp(np.maximum(np.abs(x), 2.0 ** -120))
    return np.ldexp(1.0, e - 8)


def check_projection(gpu_bits, hp_bits, wq_bits, Hq, rope=None, min_exact=0.99):
    """GPU proxies vs the oracle's fp64 projection (times the query scale
    c = log2(e)/sqrt(d)): |gpu - pre| <= ulp/2 + acc, acc = c (D + 16)
    2^-24 sum_k |x_k w_k| (fp32 accumulation), widened through the rotation
    when there is one, plus 2^-23 |pre| for the fp32 rounding of the scaled
    value."""
    out, pre = oracle.project_proxies(hp_bits, wq_bits, Hq, rope=rope, with_pre=True)
    B, P, D = hp_bits.shape
    d = wq_bits.shape[0] // Hq
    x = brute.bits_to_f64(hp_bits)
    w = brute.bits_to_f64(wq_bits).reshape(Hq, d, D)
    absdot = np.matmul(np.abs(x)[:, None], np.abs(w).transpose(0, 2, 1)[None])   # [B, Hq, P, d]
    acc = (D + 16) * 2.0 ** -24 * absdot
    if rope is not None:
        _, raw = oracle.project_proxies(hp_bits, wq_bits, Hq, with_pre=True)
        raw = raw / brute.qscale(d)              # the unscaled projection the rotation acts on
        h = d // 2
        c = np.abs(rope[0].astype(np.float64))
        s = np.abs(rope[1].astype(np.float64))
        lo = acc[..., :h] * c + acc[..., h:] * s + 2.0 ** -22 * (np.abs(raw[..., :h]) * c + np.abs(raw[..., h:]) * s)
        hi = acc[..., h:] * c + acc[..., :h] * s + 2.0 ** -22 * (np.abs(raw[..., h:]) * c + np.abs(raw[..., :h]) * s)
        acc = np.concatenate([lo, hi], axis=-1)
    acc = acc * brute.qscale(d) + 2.0 ** -23 * np.abs(pre)
    g = brute.bits_to_f64(gpu_bits)
    err = np.abs(g - pre)
    bound = 0.5 * bf16_ulp(np.abs(pre) + acc) + acc
    bad = err > bound
    assert not bad.any(), "projection: %d entries outside the bound (first %s: gpu %r oracle %r bound %r)" % (
        bad.sum(), tuple(np.argwhere(bad)[0]), g[bad][0], pre[bad][0], bound[bad][0])
    same = float(np.mean(gpu_bits == out))
    assert same >= min_exact, "only %.4f of the proxies equal bf16(fp32(oracle))" % same
    return same


# ---------------------------------------------------------------- Eq. 4
@pytest.mark.parametrize("B,T,D,dtype,ddof,pad", [
    (1, 1, 64, "bf16", 0, 0), (2, 300, 200, "f32", 1, 0), (1, 777, 3584, "bf16", 0, 0),
    (3, 513, 136, "bf16", 1, 16), (2, 256, 8, "f32", 0, 4)])
def test_hidden_stats_within_fp64_bound(B, T, D, dtype, ddof, pad):
    x = wl.custom_hidden(B, T, D + pad, 1, 8, dtype=dtype, seed=T + D)["hidden"]
    h = x.to(DEV)[:, :, :D]                       # strided view when pad > 0
    st = bd.hidden_stats(h, std_ddof=ddof)
    torch.cuda.synchronize()
    hb = bits(x[:, :, :D].contiguous())
    ref = oracle.hidden_stats(hb, ddof=ddof)
    rel = parity.check_hidden_stats(st.cpu().numpy(), values(hb), ref, ddof)
    print("hidden stats", (B, T, D, dtype, ddof), "max relative std difference", rel, flush=True)


def test_hidden_stats_constant_feature_has_zero_std():
    x = wl.custom_hidden(1, 600, 64, 1, 8, seed=3)["hidden"]
    x[:, :, 5] = 0.375
    st = bd.hidden_stats(x.to(DEV)).cpu().numpy()
    assert st[0, 0, 5] == 0.375 and st[0, 1, 5] == 0.0


# ---------------------------------------------------------------- Eq. 5
@pytest.mark.parametrize("B,P,D,gamma,layer", [(1, 512, 3584, 10.0, 3), (2, 37, 64, 2.5, 0),
                                               (3, 16, 200, 0.0, 65535)])
def test_hidden_proxies_bit_exact(B, P, D, gamma, layer):
    x = wl.custom_hidden(B, 100, D, 1, 8, seed=P)["hidden"]
    st = oracle.hidden_stats(bits(x))
    cfg = bd.SelectionConfig(P=P, gamma=gamma, seed=0xDEADBEEF12345, layer=layer)
    hp = bd.hidden_proxies(torch.from_numpy(st).to(DEV), cfg)
    torch.cuda.synchronize()
    ref = oracle.hidden_proxies(st, P, gamma, cfg.seed, layer)
    assert np.array_equal(bits(hp), ref)


# ---------------------------------------------------------------- Eq. 6
@pytest.mark.parametrize("B,P,D,Hq,d,rope", [
    (2, 64, 3584, 28, 128, False), (3, 40, 200, 3, 64, False), (1, 50, 136, 2, 128, True),
    (2, 33, 3584, 4, 64, True), (1, 1, 8, 1, 64, False),
    # full 128 x 224 tiles without rotation, 2, 3 and 5 k steps of 64
    (2, 128, 128, 7, 64, False), (1, 128, 192, 14, 64, False), (1, 256, 320, 7, 64, False)])
def test_projection_within_bound(B, P, D, Hq, d, rope):
    rng_in = wl.custom_hidden(B, P, D, Hq, d, seed=B * 1000 + P)
    hp = rng_in["hidden"]                        # any bf16 [B, P, D] serves as samples
    wq = rng_in["wq"]
    rp = wl.rope_tables(d, 20000 + P) if rope else None
    out = bd.project_proxies(hp.to(DEV), wq.to(DEV), Hq, rope=rp)
    torch.cuda.synchronize()
    same = check_projection(bits(out), bits(hp), bits(wq), Hq,
                            rope=None if rp is None else (rp[0].numpy(), rp[1].numpy()))
    print("projection", (B, P, D, Hq, d, rope), "identical fraction", same, flush=True)


# ---------------------------------------------------------------- whole layer
def test_hidden_path_layer_parity():
    """stats -> samples -> projection -> scores -> selection -> gather, GPU
    vs oracle, on a W_Q whose products are exact (proxies then bit-exact)."""
    B, T, Hq, Hkv, d, D, W = 2, 700, 8, 2, 64, 256, 1
    hx = wl.custom_hidden(B, T, D, Hq, d, seed=21, wq_kind="select")
    kv = wl.custom_layer(B, Hq, Hkv, T, 4, d, seed=22)
    cfg = bd.SelectionConfig(P=64, G=4, seed=23, layer=2)
    budget = 70
    h, wq, ql = (hx[n].to(DEV) for n in ("hidden", "wq", "q_last"))
    k, v = kv["k"].to(DEV), kv["v"].to(DEV)
    st = bd.hidden_stats(h)
    hp = bd.hidden_proxies(st, cfg)
    prox = bd.project_proxies(hp, wq, Hq)
    sc = bd.score(prox, ql, k, cfg, W)
    sel = bd.select_topk(sc, cfg, budget, None, None, Hq, W, want_votes=True)
    ko, vo = bd.gather_kv(k, v, sel)
    torch.cuda.synchronize()
    tn = parity.to_np
    g = dict(proxies=tn(prox), q_last=tn(ql), group_mass=tn(sc.group_mass), mass=tn(sc.mass),
             anchor=tn(sc.anchor), votes=tn(sel.votes), idx=tn(sel.idx), counts=tn(sel.counts),
             k_out=tn(ko), v_out=tn(vo))

    hb = bits(hx["hidden"])
    rst = oracle.hidden_stats(hb)
    st_np = st.cpu().numpy()
    parity.check_hidden_stats(st_np, values(hb), rst)
    # the samples from the GPU's statistics (the generator is checked on equal inputs)
    rhp = oracle.hidden_proxies(st_np, cfg.P, cfg.gamma, cfg.seed, cfg.layer)
    assert np.array_equal(bits(hp), rhp)
    rprox = oracle.project_proxies(rhp, bits(hx["wq"]), Hq)
    rql = bits(hx["q_last"])
    kn, vn = bits(kv["k"]), bits(kv["v"])
    gm, mass, an = oracle.score(rprox, rql, kn, Hkv, cfg.G)
    rsel = oracle.select(gm, mass, an, budget, cfg.tau, cfg.lam)
    ref = oracle.LayerResult(rprox, rql, rst, gm, mass, an, rsel, None, None)
    rep = parity.check_layer(g, ref, cfg, budget, kn, vn)
    print("hidden layer", rep, flush=True)


@pytest.mark.parametrize("name", ["qwen7b_16k_b4"])
def test_full_size_hidden_sampled(name):
    """Full-size hidden states (B=4, T=16384, D=3584, 28 heads of 128) in the
    launch configuration the benchmark times: statistics bit-exact on
    sampled features of every batch row, samples bit-exact for two batch
    rows, projections within the bound on sampled (row, head) blocks, and
    the score invariants (each proxy's softmax sums to 1) on the result."""
    w = wl.WORKLOADS[name]
    layer = 5
    hx = wl.make_hidden(w, layer, device=DEV)
    cfg = bd.SelectionConfig(seed=w.wid, layer=layer)
    st = bd.hidden_stats(hx["hidden"])
    hp = bd.hidden_proxies(st, cfg)
    prox = bd.project_proxies(hp, hx["wq"], w.Hq)
    torch.cuda.synchronize()
    D = w.Hq * w.d
    cols = np.sort(np.random.default_rng(0).choice(D, 48, replace=False))
    sub = bits(hx["hidden"][:, :, torch.as_tensor(cols, device=DEV)].contiguous())
    rst = oracle.hidden_stats(sub)
    st_np = st.cpu().numpy()
    parity.check_hidden_stats(st_np[:, :, cols], values(sub), rst)
    for b in (0, 3):
        rhp = oracle.hidden_proxies(st_np[b:b + 1], cfg.P, cfg.gamma, cfg.seed, layer, b0=b)
        assert np.array_equal(bits(hp[b:b + 1]), rhp), "samples of batch row %d differ" % b
    wq_np = bits(hx["wq"])
    for (b, h, i0) in ((1, 0, 0), (2, 27, 448)):
        rows = bits(hp[b:b + 1, i0:i0 + 64])
        wh = wq_np[h * w.d:(h + 1) * w.d]
        got = bits(prox[b:b + 1, h:h + 1, i0:i0 + 64])
        check_projection(got, rows, wh, 1)
    x = wl.make_layer(w, layer, device=DEV)
    ql = hx["q_last"]
    sc = bd.score(prox, ql, x["k"], cfg, w.W)
    torch.cuda.synchronize()
    mass = sc.mass.double().sum(-1).cpu().numpy()
    np.testing.assert_allclose(mass, cfg.P * w.Gh, rtol=1e-3)
    np.testing.assert_allclose(sc.anchor.double().sum(-1).cpu().numpy(), 1.0, rtol=1e-3)
