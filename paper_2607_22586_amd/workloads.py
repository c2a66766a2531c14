"""Seeded synthetic inputs shaped like the paper's multimodal prefill workloads.

This module only draws inputs; it holds none of the selection method's
arithmetic, and it serves both the HIP library's tests/benchmark and the CPU
oracle's tests.  The paper's benchmarks (OCRBench, DocVQA, TextVQA, ChartQA,
TextCaps, MMMU on Qwen2.5-VL-7B / LLaVA-v1.6-7B, Sec. 4.1 and Table 4) are
stood in for by these tensors: no dataset item or model weight is used.

Five named workloads (sizes per layer):

* ``tiny``      1 KV head, 4 query heads, d=64, T=1024, W=16, fp32, C=64.
                K,V ~ N(0,1); 16 planted keys get +3*sqrt(d)*u along a random
                unit direction u that the window queries share (+sqrt(d)*u).
* ``qwen7b_4k`` one 28q/4kv, d=128 layer, T=4096 = 3584 visual + 512 text,
                W=32, bf16, C = floor(0.1*T) = 409.  Visual rows are
                sqrt(1-eps^2)*(A M_c)/sqrt(r) + eps*E (rank r=64 redundancy,
                eps=0.1, unit variance); text rows N(0, 1.5) (variance 1.5).
                Window queries N(0, 1.5) + 0.5*(a_h M_c)/sqrt(r).
* ``qwen7b_8k`` 28 layers, same heads, T=8192 = 7936 + 256, W=32, C=512.
* ``qwen7b_16k_b4`` 28 layers, batch 4, T=16384 = 16128 + 256, W=64, C=256.
* ``large_32k`` 80 layers, 64q/8kv, T=32768 = 8 image blocks of 4032 visual
                rows (block mean shift s ~ N(0, 0.5 I) per block) + 512 text,
                W=64, C=1024.  Each query head's window is N(0,1.5) plus the
                mean shift of one randomly chosen block of its KV head.

Hidden-state inputs (``make_hidden``, for the hidden-state form of the
proxies): per layer, prefill hidden states [B, T, D] with D = Hq*d (3584 for
the 7B shapes, as in a Qwen2-style 7B backbone whose query projection is
square) and a query weight W_Q [Hq*d, D] ~ N(0, 1/D).  Hidden rows are the
normalised inputs of the query projection: per-feature scale s_j =
exp(0.5 n_j), visual rows s * (sqrt(1-eps^2) (A M)/sqrt(r) + eps E) (rank 64,
eps 0.1), text rows s * N(0, 1.5), and 4 outlier features whose values are
scaled by 10 (the few large-magnitude channels of LLM hidden states).

Decode queries (``make_layer(..., n_dec=n)``, for the decode-time coverage
check): n per query head, drawn after all other tensors of the layer from the
same law as that head's window queries but with the noise variance scaled by
DECODE_VAR_SCALE = 16 -- the paper reports hidden-state variance growing by
13x to 22x from prefill to decoding (Appendix, global vs. layer-wise
expansion), so decode queries spread wider than the window the proxies are
built from.

Tensors are drawn in fp32 with a seeded ``torch.Generator`` on the requested
device and rounded to bf16 (round to nearest even) where the workload is bf16.
The CPU stream is reproducible bit for bit; a device stream follows the same
recipe with the device's own generator.
"""
from __future__ import annotations

import math
from dataclasses import dataclass

import torch


@dataclass(frozen=True)
class Workload:
    name: str
    wid: int
    B: int
    L: int
    Hq: int
    Hkv: int
    d: int
    T: int
    W: int
    budget: int
    dtype: str            # "f32" or "bf16"
    kind: str             # "planted", "lowrank", "blocks"
    n_text: int = 0
    n_blocks: int = 0

    @property
    def Gh(self) -> int:
        return self.Hq // self.Hkv


WORKLOADS = {
    "tiny": Workload("tiny", 0, 1, 1, 4, 1, 64, 1024, 16, 64, "f32", "planted"),
    "qwen7b_4k": Workload("qwen7b_4k", 1, 1, 1, 28, 4, 128, 4096, 32, 409, "bf16", "lowrank", 512),
    "qwen7b_8k": Workload("qwen7b_8k", 2, 1, 28, 28, 4, 128, 8192, 32, 512, "bf16", "lowrank", 256),
    "qwen7b_16k_b4": Workload("qwen7b_16k_b4", 3, 4, 28, 28, 4, 128, 16384, 64, 256, "bf16",
                              "lowrank", 256),
    "large_32k": Workload("large_32k", 4, 1, 80, 64, 8, 128, 32768, 64, 1024, "bf16", "blocks",
                          512, 8),
}

# The paper's default method settings (Sec. 4.1 "Implementation and
# Hyperparameters"; Appendix B): N=512 proxies in G=32 groups of 16,
# gamma=10, tau=0.95, lambda=1.
PAPER_DEFAULTS = dict(P=512, G=32, gamma=10.0, tau=0.95, lam=1.0)

N_PLANTED = 16
LOWRANK_R = 64
LOWRANK_EPS = 0.1
TEXT_VAR = 1.5
BLOCK_SHIFT_VAR = 0.5
DECODE_VAR_SCALE = 16.0


def _seed(wid: int, layer: int, stream: int) -> int:
    return (wid * 1_000_003 + layer * 7919 + stream * 104_729 + 12345) & 0x7FFFFFFF


def _gen(device, wid, layer, stream) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(_seed(wid, layer, stream))
    return g


def _randn(shape, gen, device):
    return torch.randn(shape, generator=gen, device=device, dtype=torch.float32)


def _planted(w: Workload, layer: int, device, n_dec: int = 0):
    g = _gen(device, w.wid, layer, 0)
    d, T = w.d, w.T
    u = _randn((w.B, w.Hkv, 1, d), g, device)
    u = u / torch.linalg.vector_norm(u, dim=-1, keepdim=True)
    k = _randn((w.B, w.Hkv, T, d), g, device)
    v = _randn((w.B, w.Hkv, T, d), g, device)
    planted = torch.empty((w.B, w.Hkv, N_PLANTED), dtype=torch.int64, device=device)
    for b in range(w.B):
        for c in range(w.Hkv):
            planted[b, c] = torch.randperm(T - 1, generator=g, device=device)[:N_PLANTED]
    bump = torch.zeros((w.B, w.Hkv, T, 1), device=device)
    bump.scatter_(2, planted.unsqueeze(-1), 1.0)
    k = k + bump * (3.0 * math.sqrt(d)) * u
    u_q = u.repeat_interleave(w.Gh, dim=1)
    q = _randn((w.B, w.Hq, w.W, d), g, device) + math.sqrt(d) * u_q
    q_dec = None
    if n_dec > 0:
        q_dec = math.sqrt(DECODE_VAR_SCALE) * _randn((w.B, w.Hq, n_dec, d), g, device) + math.sqrt(d) * u_q
    return q, k, v, planted, q_dec


def _lowrank_rows(shape_bc, n, r, eps, m, g, device):
    a = _randn(shape_bc + (n, r), g, device)
    e = _randn(shape_bc + (n, m.shape[-1]), g, device)
    return math.sqrt(1.0 - eps * eps) * torch.matmul(a, m) / math.sqrt(r) + eps * e


def _lowrank(w: Workload, layer: int, device, n_dec: int = 0):
    g = _gen(device, w.wid, layer, 1)
    d, T, r = w.d, w.T, LOWRANK_R
    n_vis = T - w.n_text
    bc = (w.B, w.Hkv)
    m_k = _randn(bc + (r, d), g, device)
    m_v = _randn(bc + (r, d), g, device)
    k = torch.cat([_lowrank_rows(bc, n_vis, r, LOWRANK_EPS, m_k, g, device),
                   math.sqrt(TEXT_VAR) * _randn(bc + (w.n_text, d), g, device)], dim=2)
    v = torch.cat([_lowrank_rows(bc, n_vis, r, LOWRANK_EPS, m_v, g, device),
                   math.sqrt(TEXT_VAR) * _randn(bc + (w.n_text, d), g, device)], dim=2)
    a_h = _randn((w.B, w.Hq, 1, r), g, device)
    m_h = 0.5 * torch.matmul(a_h, m_k.repeat_interleave(w.Gh, dim=1)) / math.sqrt(r)
    q = math.sqrt(TEXT_VAR) * _randn((w.B, w.Hq, w.W, d), g, device) + m_h
    q_dec = None
    if n_dec > 0:
        q_dec = math.sqrt(DECODE_VAR_SCALE * TEXT_VAR) * _randn((w.B, w.Hq, n_dec, d), g, device) + m_h
    return q, k.contiguous(), v.contiguous(), None, q_dec


def _blocks(w: Workload, layer: int, device, n_dec: int = 0):
    g = _gen(device, w.wid, layer, 2)
    d, T, nb = w.d, w.T, w.n_blocks
    n_blk = (T - w.n_text) // nb
    bc = (w.B, w.Hkv)

    def one(shift):
        vis = _randn(bc + (nb, n_blk, d), g, device) + shift.unsqueeze(3)
        vis = vis.reshape(bc + (nb * n_blk, d))
        txt = math.sqrt(TEXT_VAR) * _randn(bc + (w.n_text, d), g, device)
        return torch.cat([vis, txt], dim=2).contiguous()

    s_k = math.sqrt(BLOCK_SHIFT_VAR) * _randn(bc + (nb, d), g, device)
    s_v = math.sqrt(BLOCK_SHIFT_VAR) * _randn(bc + (nb, d), g, device)
    k = one(s_k)
    v = one(s_v)
    pick = torch.randint(0, nb, (w.B, w.Hq), generator=g, device=device)
    s_q = s_k.repeat_interleave(w.Gh, dim=1)                    # [B, Hq, nb, d]
    shift_q = torch.gather(s_q, 2, pick[:, :, None, None].expand(w.B, w.Hq, 1, d))
    q = math.sqrt(TEXT_VAR) * _randn((w.B, w.Hq, w.W, d), g, device) + shift_q
    q_dec = None
    if n_dec > 0:
        q_dec = math.sqrt(DECODE_VAR_SCALE * TEXT_VAR) * _randn((w.B, w.Hq, n_dec, d), g, device) + shift_q
    return q, k, v, None, q_dec


def make_layer(w: Workload | str, layer: int = 0, device="cpu", n_dec: int = 0):
    """Inputs of one layer: dict(q_win [B,Hq,W,d], k, v [B,Hkv,T,d], planted,
    q_dec).

    ``planted`` holds the planted key indices for the ``tiny`` workload
    (None otherwise).  ``q_dec`` [B,Hq,n_dec,d] bf16 holds n_dec decode
    queries per head (None when n_dec = 0); drawing them does not change the
    other tensors.  Tensors are fp32 for ``tiny`` and bf16 otherwise (decode
    queries are bf16 always).
    """
    if isinstance(w, str):
        w = WORKLOADS[w]
    fn = {"planted": _planted, "lowrank": _lowrank, "blocks": _blocks}[w.kind]
    with torch.no_grad():
        q, k, v, planted, q_dec = fn(w, layer, torch.device(device), n_dec)
        if w.dtype == "bf16":
            q, k, v = (x.to(torch.bfloat16) for x in (q, k, v))
        if q_dec is not None:
            q_dec = q_dec.to(torch.bfloat16).contiguous()
    return dict(q_win=q.contiguous(), k=k.contiguous(), v=v.contiguous(), planted=planted, q_dec=q_dec)


HIDDEN_OUTLIERS = 4
HIDDEN_OUTLIER_SCALE = 10.0


def make_hidden(w: Workload | str, layer: int = 0, device="cpu", T: int | None = None):
    """Hidden-state inputs of one layer: dict(hidden [B, T, D] bf16 (fp32 for
    ``tiny``), wq [Hq*d, D] bf16, q_last [B, Hq, d] bf16) with D = Hq*d;
    q_last is the model's last query (W_Q times the last hidden row, fp32,
    rounded to bf16).  ``T`` overrides the token count (the visual/text
    split keeps the workload's text share)."""
    if isinstance(w, str):
        w = WORKLOADS[w]
    dev = torch.device(device)
    T = w.T if T is None else int(T)
    D = w.Hq * w.d
    n_text = min(T, w.n_text * T // w.T) if w.n_text else 0
    n_vis = T - n_text
    g = _gen(dev, w.wid, layer, 7)
    with torch.no_grad():
        scale = torch.exp(0.5 * _randn((w.B, 1, D), g, dev))
        m = _randn((w.B, LOWRANK_R, D), g, dev)
        parts = []
        if n_vis:
            parts.append(_lowrank_rows((w.B,), n_vis, LOWRANK_R, LOWRANK_EPS, m, g, dev))
        if n_text:
            parts.append(math.sqrt(TEXT_VAR) * _randn((w.B, n_text, D), g, dev))
        out = torch.cat(parts, dim=1) * scale
        cols = torch.randperm(D, generator=g, device=dev)[:HIDDEN_OUTLIERS]
        out[:, :, cols] *= HIDDEN_OUTLIER_SCALE
        wq = _randn((w.Hq * w.d, D), g, dev) / math.sqrt(D)
        dt = torch.float32 if w.dtype == "f32" else torch.bfloat16
        hidden = out.to(dt).contiguous()
        wq = wq.to(torch.bfloat16).contiguous()
        # the model's own last query (the anchor's input), W_Q h_{T-1} in fp32
        q_last = (hidden[:, -1].float() @ wq.float().t()).reshape(w.B, w.Hq, w.d)
        return dict(hidden=hidden, wq=wq, q_last=q_last.to(torch.bfloat16).contiguous())


def custom_hidden(B, T, D, Hq, d, dtype="bf16", seed=0, device="cpu", wq_kind="dense"):
    """Free-shape hidden-state inputs: hidden [B, T, D] ~ per-feature scaled
    N(0, 1) plus a per-feature mean, W_Q [Hq*d, D] bf16 and the last query
    q_last [B, Hq, d] bf16.  wq_kind "dense": N(0, 1/D); "select": one
    nonzero per row, +-1 or +-2 at a random feature (its products are exact
    in every precision)."""
    g = torch.Generator(device=device)
    g.manual_seed(int(seed) & 0x7FFFFFFF)
    dev = torch.device(device)
    with torch.no_grad():
        scale = torch.exp(0.5 * _randn((B, 1, D), g, dev))
        hidden = (_randn((B, T, D), g, dev) + _randn((B, 1, D), g, dev)) * scale
        if wq_kind == "dense":
            wq = _randn((Hq * d, D), g, dev) / math.sqrt(D)
        else:
            wq = torch.zeros((Hq * d, D), device=dev)
            cols = torch.randint(0, D, (Hq * d,), generator=g, device=dev)
            vals = torch.tensor([-2.0, -1.0, 1.0, 2.0], device=dev)[
                torch.randint(0, 4, (Hq * d,), generator=g, device=dev)]
            wq[torch.arange(Hq * d, device=dev), cols] = vals
        dt = torch.float32 if dtype == "f32" else torch.bfloat16
        hidden = hidden.to(dt).contiguous()
        wq = wq.to(torch.bfloat16).contiguous()
        q_last = (hidden[:, -1].float() @ wq.float().t()).reshape(B, Hq, d)
        return dict(hidden=hidden, wq=wq, q_last=q_last.to(torch.bfloat16).contiguous())


def custom_layer(B, Hq, Hkv, T, W, d, dtype="bf16", seed=0, device="cpu", key_scale=1.0,
                 q_mean_scale=1.0):
    """Free-shape inputs for ragged and edge-case tests: Gaussian K/V, window
    queries with a per-head mean offset.  Same tensor conventions as make_layer."""
    g = torch.Generator(device=device)
    g.manual_seed(int(seed) & 0x7FFFFFFF)
    dev = torch.device(device)
    k = key_scale * _randn((B, Hkv, T, d), g, dev)
    v = _randn((B, Hkv, T, d), g, dev)
    q = _randn((B, Hq, W, d), g, dev) + q_mean_scale * _randn((B, Hq, 1, d), g, dev)
    if dtype == "bf16":
        q, k, v = (x.to(torch.bfloat16) for x in (q, k, v))
    return dict(q_win=q.contiguous(), k=k.contiguous(), v=v.contiguous(), planted=None)


def rope_tables(d: int, position: int, base: float = 10000.0):
    """cos/sin (float32, length d/2) of the rotary embedding at one position,
    rotate-half pairing (j, j + d/2) with frequency base^(-2j/d)."""
    j = torch.arange(d // 2, dtype=torch.float64)
    ang = position * torch.pow(torch.tensor(base, dtype=torch.float64), -2.0 * j / d)
    return torch.cos(ang).to(torch.float32), torch.sin(ang).to(torch.float32)


def to_numpy_bits(x: torch.Tensor):
    """CPU numpy view for the oracle: float32 stays float32; bf16 becomes its
    uint16 bit pattern."""
    x = x.detach().cpu().contiguous()
    if x.dtype == torch.bfloat16:
        return x.view(torch.uint16).numpy()
    return x.numpy()
