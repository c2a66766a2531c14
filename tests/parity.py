"""Comparators between the HIP path and the CPU oracle (test infrastructure).

Floating-point outputs (group mass, mass, anchor) must lie within 1e-3
relative of the oracle (fp32 accumulation from bf16 operands against fp64).
Discrete outputs are derived from those floats, so they are compared as
follows:
  * votes: equal to the oracle's except for keys inside the oracle's
    ambiguity band of some group -- keys whose group mass is within 1e-3
    relative of that group's cut mass, or whose running sum in the sorted
    order is within 1e-3 of the group total from tau * total -- and, exactly,
    to the tau-sets recomputed in numpy from the GPU's own group masses;
  * selection: every kept key must be able to outrank every dropped key once
    each oracle score is widened by its own uncertainty (band votes plus
    1e-3 of the anchor term), and the selection must be exactly the top-k of
    the GPU's own fp64 scores;
  * gather: byte-exact given the GPU's own indices.
"""
from __future__ import annotations

import numpy as np
import torch

REL = 1e-3
ATOL = 1e-30


def to_np(t):
    t = t.detach().cpu().contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.uint16).numpy()
    return t.numpy()


def rel_err(gpu, ref, atol=ATOL):
    gpu = np.asarray(gpu, np.float64)
    ref = np.asarray(ref, np.float64)
    return np.abs(gpu - ref) / (np.abs(ref) + atol)


def assert_close(name, gpu, ref, rel=REL, atol=ATOL):
    gpu = np.asarray(gpu, np.float64)
    ref = np.asarray(ref, np.float64)
    bad = np.abs(gpu - ref) > rel * np.abs(ref) + atol
    if bad.any():
        i = np.argwhere(bad)[0]
        raise AssertionError("%s: %d/%d outside %.0e (first at %s: gpu=%r ref=%r)"
                             % (name, bad.sum(), bad.size, rel, tuple(i), gpu[tuple(i)], ref[tuple(i)]))
    return float(rel_err(gpu, ref, atol).max()) if gpu.size else 0.0


def _order(m):
    """(mass desc, index asc) order of a 1-D mass vector."""
    return np.lexsort((np.arange(m.size), -m))


def vote_band(ref_gm, tau, rel=REL):
    """Number of groups in whose ambiguity band each key lies: [B, Hkv, T]."""
    B, H, G, T = ref_gm.shape
    band = np.zeros((B, H, T), dtype=np.int32)
    for b in range(B):
        for c in range(H):
            for g in range(G):
                m = ref_gm[b, c, g]
                o = _order(m)
                run = np.cumsum(m[o])
                tot = run[-1]
                n = int(np.searchsorted(run >= tau * tot, True))
                theta = m[o[min(n, T - 1)]]
                near_mass = np.abs(m - theta) <= rel * theta
                near_run = np.zeros(T, bool)
                near_run[o] = np.abs(run - tau * tot) <= rel * tot
                band[b, c] += (near_mass | near_run).astype(np.int32)
    return band


def tau_votes_np(gm, tau):
    """tau-sets recomputed from (GPU) group masses in fp64, by the definition.
    Returns (votes, doubtful): doubtful marks keys of groups whose cut sum is
    within 1e-9 of tau*total (where fixed-point and fp64 sums may disagree)."""
    B, H, G, T = gm.shape
    votes = np.zeros((B, H, T), dtype=np.int64)
    doubt = np.zeros((B, H, T), dtype=bool)
    for b in range(B):
        for c in range(H):
            for g in range(G):
                m = gm[b, c, g].astype(np.float64)
                o = _order(m)
                run = np.cumsum(m[o])
                tot = run[-1]
                n = int(np.searchsorted(run >= tau * tot, True)) + 1
                votes[b, c, o[:n]] += 1
                if abs(run[n - 1] - tau * tot) <= 1e-9 * tot or (n >= 2 and abs(run[n - 2] - tau * tot) <= 1e-9 * tot):
                    doubt[b, c, o[max(n - 2, 0):n + 1]] = True
    return votes, doubt


def topk_np(score, T, budget, keep_last=True):
    """Top-k by (score desc, index asc), ascending output (the selection rule)."""
    if T <= budget:
        return np.arange(T)
    pool = T - 1 if keep_last else T
    want = budget - 1 if keep_last else budget
    o = np.lexsort((np.arange(pool), -score[:pool]))
    sel = list(o[:want]) + ([T - 1] if keep_last else [])
    return np.sort(np.asarray(sel, dtype=np.int64))


def check_selection_interval(sel, score_ref, unc, T, budget, keep_last=True):
    """Every kept pool key must be able to outrank every dropped pool key once
    scores are widened by their uncertainty."""
    sel = np.asarray(sel)
    if T <= budget:
        assert np.array_equal(sel, np.arange(T))
        return 0
    pool = T - 1 if keep_last else T
    kept = np.zeros(T, bool)
    kept[sel] = True
    if keep_last:
        assert kept[T - 1]
    kp = kept[:pool]
    hi_kept = (score_ref[:pool] + unc[:pool])[kp]
    lo_drop = (score_ref[:pool] - unc[:pool])[~kp]
    if hi_kept.size and lo_drop.size:
        assert hi_kept.min() >= lo_drop.max() - 1e-12, (hi_kept.min(), lo_drop.max())
    return int(len(set(sel.tolist()) ^ set(topk_np(score_ref, T, budget, keep_last).tolist())))


def check_layer(gpu: dict, ref, cfg, budget, k_np, v_np, keep_last=True, budgets=None,
                check_proxies=True):
    """All parity checks for one layer.  gpu: numpy arrays from the HIP path;
    ref: oracle.LayerResult on the same inputs.  Returns a report dict."""
    rep = {}
    B, H, T = gpu["mass"].shape
    if check_proxies:
        assert np.array_equal(gpu["proxies"], ref.proxies), "proxies differ"
        assert np.array_equal(gpu["q_last"], ref.q_last), "q_last differs"
    rep["mass_rel"] = assert_close("mass", gpu["mass"], ref.mass)
    rep["anchor_rel"] = assert_close("anchor", gpu["anchor"], ref.anchor)
    vote_mode = cfg.mode == 0
    if vote_mode:
        rep["group_mass_rel"] = assert_close("group_mass", gpu["group_mass"], ref.group_mass)
        band = vote_band(ref.group_mass, cfg.tau)
        dv = np.abs(gpu["votes"].astype(np.int64) - ref.sel.votes)
        assert np.all(dv <= band), "votes differ outside the band"
        rep["vote_mismatch"] = int((dv > 0).sum())
        own, doubt = tau_votes_np(gpu["group_mass"], cfg.tau)
        mism = (own != gpu["votes"]) & ~doubt
        assert not mism.any(), "GPU votes are not the tau-sets of its own masses"
        unc = band + cfg.lam * (REL * ref.anchor + 1e-9)
    else:
        band = np.zeros((B, H, T), np.int32)
        unc = REL * ref.mass + ATOL
    exact = 0
    sym = 0
    for b in range(B):
        for c in range(H):
            bud = budget if budgets is None else int(budgets[b, c])
            n = int(gpu["counts"][b, c])
            assert n == min(bud, T), (n, bud, T)
            sel = gpu["idx"][b, c, :n]
            assert np.all(gpu["idx"][b, c, n:] == -1)
            assert np.all(np.diff(sel) > 0), "indices not ascending"
            # exact top-k of the GPU's own fp64 scores
            if vote_mode:
                own_score = gpu["votes"][b, c].astype(np.float64) + cfg.lam * gpu["anchor"][b, c].astype(np.float64)
            else:
                own_score = gpu["mass"][b, c].astype(np.float64)
            assert np.array_equal(sel, topk_np(own_score, T, bud, keep_last)), "not the top-k of own scores"
            ref_score = ref.sel.score[b, c]
            d = check_selection_interval(sel, ref_score, unc[b, c], T, bud, keep_last)
            sym += d
            exact += int(np.array_equal(sel, ref.sel.idx[b, c, :n]))
            # gather: byte-exact given the GPU indices
            assert gpu["k_out"][b, c, :n].tobytes() == k_np[b, c, sel].tobytes()
            assert gpu["v_out"][b, c, :n].tobytes() == v_np[b, c, sel].tobytes()
            assert not gpu["k_out"][b, c, n:].any() and not gpu["v_out"][b, c, n:].any()
    rep["heads_exact"] = exact
    rep["heads"] = B * H
    rep["sel_symdiff"] = sym
    return rep


U64 = 2.0 ** -53     # unit roundoff of fp64


def check_hidden_stats(gpu, h64, ref, ddof=0):
    """GPU hidden-state statistics [B, 2, D] against the oracle's two-pass
    definition (Sec. 3.2.1 Eq. 4), within the fp64 rounding bound of ANY
    summation of the tokens by sums of values and of squares (the GPU's
    chunked one-pass form).  With n = T tokens, u = 2^-53 and every input
    and square exact in fp64:
      |S~ - S| <= (n-1) u sum|h|,  |SS~ - SS| <= (n-1) u SS,
      mean:  |mean~ - mean| <= ((n+1) u sum|h|) / n + u |mean|,
      var:   the numerator SS - S*mean loses at most ~3 n u SS (S^2/n <= SS
             and (sum|h|)^2 <= n SS by Cauchy-Schwarz), so
             |var~ - var| <= tol = (4n + 8) u SS / (n - ddof),
      std:   |sqrt(a) - sqrt(b)| <= min(sqrt|a-b|, |a-b| / (sqrt a + sqrt b)).
    h64: the hidden states [B, T, D] as fp64 values."""
    gpu = np.asarray(gpu, np.float64)
    ref = np.asarray(ref, np.float64)
    n = h64.shape[1]
    sabs = np.abs(h64).sum(axis=1)
    ss = (h64 * h64).sum(axis=1)
    tol_mean = (2 * n + 4) * U64 * sabs / n + 4 * U64 * np.abs(ref[:, 0])
    dm = np.abs(gpu[:, 0] - ref[:, 0])
    assert np.all(dm <= tol_mean), "mean outside the fp64 bound (max excess %r)" % float((dm - tol_mean).max())
    tol_var = (4 * n + 8) * U64 * ss / (n - ddof)
    sg, sr = gpu[:, 1], ref[:, 1]
    tol_std = np.minimum(np.sqrt(tol_var), tol_var / np.maximum(sg + sr, 1e-300)) + 4 * U64 * sr
    ds = np.abs(sg - sr)
    assert np.all(ds <= tol_std), "std outside the fp64 bound (max excess %r)" % float((ds - tol_std).max())
    return float((ds / np.maximum(sr, 1e-300)).max())
