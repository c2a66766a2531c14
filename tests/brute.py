"""Brute-force fp64 reference for tiny shapes, written from the paper's
equations with numpy/scipy library routines (matmul, softmax, exhaustive
subset search).  It shares no code with the C oracle and serves only to pin
it (test infrastructure).

* Sec. 3.2.2 Eq. 7: a_t(q) = softmax_t(q.k_t / sqrt(d)); the queries carry the
  scale c = log2(e)/sqrt(d) (rounded to bf16 after scaling), so the products
  q~.k_t are base-2 logits and a_t = softmax_t(ln(2) * q~.k_t)
* Sec. 3.2.2 Eq. 8: group mass = sum over the group's proxies (and, for GQA,
  the query heads that share the KV head, Appendix B)
* Sec. 3.2.2 Eq. 9: smallest key set whose mass reaches tau * total
* Sec. 3.2.3: keep the most recent key and the C-1 best remaining keys
"""
import math
from itertools import combinations

import numpy as np
import torch
from scipy.special import softmax


def bits_to_f64(h):
    return (np.asarray(h, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def qscale(d):
    """log2(e)/sqrt(d), the softmax scale the queries carry."""
    return math.log2(math.e) / math.sqrt(d)


def scale_to_bf16(x, d):
    """fp64 values times log2(e)/sqrt(d), rounded fp64 -> fp32 (numpy) ->
    bf16 (torch, round to nearest even); returned as fp64."""
    y = (np.asarray(x, dtype=np.float64) * qscale(d)).astype(np.float32)
    b = torch.from_numpy(np.ascontiguousarray(y)).to(torch.bfloat16).view(torch.uint16).numpy()
    return bits_to_f64(b)


def masses(proxies, q_last, k, Hkv, G):
    """proxies [B,Hq,P,d] (scaled, fp64 of the bf16 values), q_last [B,Hq,d]
    (raw anchor queries), k [B,Hkv,T,d] (all fp64)."""
    B, Hq, P, d = proxies.shape
    T = k.shape[2]
    Gh = Hq // Hkv
    k_rep = np.repeat(k, Gh, axis=1)                           # [B, Hq, T, d]
    logits = np.matmul(proxies, np.swapaxes(k_rep, -1, -2)) * math.log(2.0)
    p = softmax(logits, axis=-1)                               # [B, Hq, P, T]
    p = p.reshape(B, Hkv, Gh, G, P // G, T)
    gm = p.sum(axis=(2, 4))                                    # [B, Hkv, G, T]
    qa = scale_to_bf16(q_last, d)
    la = np.einsum("bhd,bhtd->bht", qa, k_rep) * math.log(2.0)
    an = softmax(la, axis=-1).reshape(B, Hkv, Gh, T).mean(axis=2)
    return gm, gm.sum(axis=2), an


def minimal_cover_size(m, tau):
    """Size of the smallest subset of keys whose mass reaches tau * total,
    by exhaustive search over subsets in increasing size."""
    T = len(m)
    target = tau * m.sum()
    for n in range(1, T + 1):
        best = max(sum(m[list(c)]) for c in combinations(range(T), n))
        if best >= target * (1 - 1e-12):
            return n
    return T


def best_subset(score, n):
    """Subset of size n with the largest total score (exhaustive)."""
    best, arg = -np.inf, None
    for c in combinations(range(len(score)), n):
        s = score[list(c)].sum()
        if s > best:
            best, arg = s, c
    return set(arg)
