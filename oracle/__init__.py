"""Plain fp64 CPU oracle for MM-ShiftKV prefill-stage KV selection.

TEST INFRASTRUCTURE ONLY: the tests, the smoke check and the CPU-baseline leg
of the benchmark may import this package; the product library never does.
The arithmetic lives in ``mmskv_oracle.c`` (plain C loops, double precision);
this module only marshals numpy arrays into it.  bf16 tensors are carried as
``numpy.uint16`` bit patterns.

Paper steps and where they are computed:
  * Sec. 3.2.1 Eqs. 4-5 (statistics, variance-expanded sampling) and the
    optional rotary placement of the proxies       -> ``build_proxies``
  * Sec. 3.2.1 Eqs. 4-6 in hidden-state form (statistics of the prefill
    hidden states, samples, projection by W_Q)     -> ``hidden_stats``,
                                                      ``hidden_proxies``,
                                                      ``project_proxies``
  * Sec. 3.2.2 Eqs. 7-8 (proxy softmax, group mass), Sec. 3.2.3 Eq. 11 (anchor)
                                                   -> ``score``
  * Sec. 3.2.2 Eqs. 9-10 (tau-sets, votes), Sec. 3.2.3 (keep-last + top C-1),
    Appendix B / Algorithm 1 (temporal order)      -> ``select``
  * Appendix B (insertion of the retained K/V)     -> ``gather``
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "mmskv_oracle.c")
_LIB = os.path.join(_HERE, "libmmskv_oracle.so")
_lib = None

MODE_VOTE = 0
MODE_MASS = 1


def build(force: bool = False) -> str:
    """Compile the C oracle (gcc, -O2, no FMA contraction, OpenMP)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-O2", "-ffp-contract=off", "-fno-fast-math", "-fopenmp", "-shared",
               "-fPIC", "-std=c11", "-Wall", "-Wextra", "-o", tmp, _SRC, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is not None:
        return _lib
    build()
    lib = ctypes.CDLL(_LIB)
    P = ctypes.c_void_p
    i32, u64, f64, i64 = ctypes.c_int, ctypes.c_uint64, ctypes.c_double, ctypes.c_int64
    lib.oracle_philox4x32_10.argtypes = [P, P, P]
    lib.oracle_uniform.argtypes = [ctypes.c_uint32]
    lib.oracle_uniform.restype = ctypes.c_float
    lib.oracle_ln.argtypes = [ctypes.c_float]
    lib.oracle_ln.restype = ctypes.c_float
    lib.oracle_sincos_2pi.argtypes = [ctypes.c_uint32, P, P]
    lib.oracle_normal4.argtypes = [u64, i32, i32, i32, i32, i32, P]
    lib.oracle_f32_to_bf16.argtypes = [ctypes.c_float]
    lib.oracle_f32_to_bf16.restype = ctypes.c_uint16
    lib.oracle_build_proxies.argtypes = [i32, i32, i32, i32, i32, f64, i32, u64, i32, P, i32,
                                         P, P, P, P, P, P, P]
    lib.oracle_build_proxies.restype = i32
    lib.oracle_build_proxies_at.argtypes = [i32, i32, i32, i32, i32, f64, i32, u64, i32, i32, i32, P,
                                            i32, P, P, P, P, P, P, P]
    lib.oracle_build_proxies_at.restype = i32
    lib.oracle_score.argtypes = [i32, i32, i32, i32, i32, i32, i32, P, P, P, i32, P, P, P]
    lib.oracle_score.restype = i32
    lib.oracle_select.argtypes = [i32, i32, i32, i32, i32, f64, f64, i32, i32, i32, P, P, P,
                                  P, P, P, P, P, P]
    lib.oracle_select.restype = i32
    lib.oracle_gather.argtypes = [i32, i32, i32, i64, i32, P, P, P, P]
    lib.oracle_gather.restype = i32
    lib.oracle_num_threads.restype = i32
    lib.oracle_hidden_stats.argtypes = [i32, i32, i32, i32, P, i32, P]
    lib.oracle_hidden_stats.restype = i32
    lib.oracle_hidden_proxies.argtypes = [i32, i32, i32, f64, u64, i32, i32, P, P]
    lib.oracle_hidden_proxies.restype = i32
    lib.oracle_project_proxies.argtypes = [i32, i32, i32, i32, i32, P, P, P, P, P, P]
    lib.oracle_query_scale.argtypes = [i32]
    lib.oracle_query_scale.restype = f64
    lib.oracle_project_proxies.restype = i32
    lib.oracle_window_rows.argtypes = [i32, i32, i32, i32, i32, P, i32, P]
    lib.oracle_window_rows.restype = i32
    lib.oracle_shape_scores.argtypes = [i32, i32, i32, i32, i32, i32, i32, P, P]
    lib.oracle_shape_scores.restype = i32
    lib.oracle_decode_check.argtypes = [i32, i32, i32, i32, i32, i32, P, P, i32, P, P, i32, P, P, i32, P, P]
    lib.oracle_decode_check.restype = i32
    _lib = lib
    return lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def num_threads() -> int:
    return int(_load().oracle_num_threads())


# ----------------------------------------------------------------------------
# generator pieces (exposed for pinning)
# ----------------------------------------------------------------------------
def philox4x32_10(ctr, key) -> np.ndarray:
    c = np.ascontiguousarray(np.asarray(ctr, dtype=np.uint32))
    k = np.ascontiguousarray(np.asarray(key, dtype=np.uint32))
    out = np.zeros(4, dtype=np.uint32)
    _load().oracle_philox4x32_10(_ptr(c), _ptr(k), _ptr(out))
    return out


def uniform(x: int) -> float:
    """32-bit word -> (2*(x>>9)+1) * 2^-24 (an fp32 value)."""
    return float(_load().oracle_uniform(int(x)))


def ln(u: float) -> float:
    """The generator's fp32 series natural log (u in (0, 1), an fp32 value)."""
    return float(_load().oracle_ln(float(u)))


def sincos_2pi(x: int):
    """(sin 2 pi u, cos 2 pi u) in fp32 by the generator's series, u = uniform(x)."""
    s, c = ctypes.c_float(), ctypes.c_float()
    _load().oracle_sincos_2pi(int(x), ctypes.byref(s), ctypes.byref(c))
    return float(s.value), float(c.value)


def normal4(seed: int, b: int, layer: int, h: int, i: int, jq: int) -> np.ndarray:
    z = np.zeros(4, dtype=np.float64)
    _load().oracle_normal4(int(seed), b, layer, h, i, jq, _ptr(z))
    return z


def query_scale(d: int) -> float:
    """log2(e)/sqrt(d): the softmax scale the proxies and anchor queries carry."""
    return float(_load().oracle_query_scale(int(d)))


def f32_to_bf16(x: np.ndarray) -> np.ndarray:
    """Round-to-nearest-even fp32 -> bf16 (element-wise call into the oracle)."""
    lib = _load()
    flat = np.asarray(x, dtype=np.float32).ravel()
    out = np.array([lib.oracle_f32_to_bf16(float(v)) for v in flat], dtype=np.uint16)
    return out.reshape(np.shape(x))


def bf16_to_f64(h: np.ndarray) -> np.ndarray:
    return (np.asarray(h, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


# ----------------------------------------------------------------------------
# pipeline steps
# ----------------------------------------------------------------------------
def _dtype_code(a: np.ndarray) -> int:
    if a.dtype == np.float32:
        return 0
    if a.dtype == np.uint16:
        return 1
    raise TypeError("oracle inputs are float32 or bf16 bit patterns (uint16), got %s" % a.dtype)


def build_proxies(q_win: np.ndarray, P: int, gamma: float, seed: int, layer: int = 0, ddof: int = 0,
                  rope_f=None, rope_l=None, b0: int = 0, h0: int = 0):
    """Sec. 3.2.1: window statistics (Eq. 4), variance-expanded samples (Eq. 5).

    q_win: [B, Hq, W, d] float32 or bf16 bits.  rope_f / rope_l: optional
    (cos, sin) float32 tables of length d/2 for the proxies' future position
    and for the last query's own position.  b0 / h0: global batch row and
    query head of q_win[0, 0] when q_win is a slice of a larger problem.
    Returns (proxies [B,Hq,P,d] u16, q_last [B,Hq,d] u16, stats [B,Hq,2,d] f64).
    """
    q = np.ascontiguousarray(q_win)
    B, Hq, W, d = q.shape
    prox = np.zeros((B, Hq, P, d), dtype=np.uint16)
    qlast = np.zeros((B, Hq, d), dtype=np.uint16)
    stats = np.zeros((B, Hq, 2, d), dtype=np.float64)
    tabs = []
    for rp in (rope_f, rope_l):
        if rp is None:
            tabs += [None, None]
        else:
            tabs += [np.ascontiguousarray(rp[0], dtype=np.float32),
                     np.ascontiguousarray(rp[1], dtype=np.float32)]
    rc = _load().oracle_build_proxies_at(B, Hq, W, d, P, float(gamma), int(ddof), int(seed), int(layer),
                                         int(b0), int(h0), _ptr(q), _dtype_code(q),
                                         *[_ptr(t) for t in tabs],
                                         _ptr(prox), _ptr(qlast), _ptr(stats))
    if rc != 0:
        raise ValueError("oracle_build_proxies rejected its arguments")
    return prox, qlast, stats


def score(proxies: np.ndarray, q_last: np.ndarray, k: np.ndarray, Hkv: int, G: int):
    """Sec. 3.2.2 Eqs. 7-8 and Sec. 3.2.3 Eq. 11 (anchor): fp64 masses.

    Returns (group_mass [B,Hkv,G,T], mass [B,Hkv,T], anchor [B,Hkv,T]).
    """
    proxies = np.ascontiguousarray(proxies, dtype=np.uint16)
    q_last = np.ascontiguousarray(q_last, dtype=np.uint16)
    k = np.ascontiguousarray(k)
    B, Hq, P, d = proxies.shape
    T = k.shape[2]
    assert k.shape == (B, Hkv, T, d)
    gm = np.zeros((B, Hkv, G, T), dtype=np.float64)
    mass = np.zeros((B, Hkv, T), dtype=np.float64)
    anchor = np.zeros((B, Hkv, T), dtype=np.float64)
    rc = _load().oracle_score(B, Hq, Hkv, T, d, P, G, _ptr(proxies), _ptr(q_last), _ptr(k),
                              _dtype_code(k), _ptr(gm), _ptr(mass), _ptr(anchor))
    if rc != 0:
        raise ValueError("oracle_score rejected its arguments")
    return gm, mass, anchor


@dataclass
class Selection:
    idx: np.ndarray        # [B, Hkv, c_max] int32, ascending, -1 padded
    counts: np.ndarray     # [B, Hkv] int32
    votes: np.ndarray      # [B, Hkv, T] int32
    score: np.ndarray      # [B, Hkv, T] fp64
    cut_mass: np.ndarray   # [B, Hkv, G] fp64 (mass of the last key entering each tau-set)
    cut_size: np.ndarray   # [B, Hkv, G] int32


def select(group_mass, mass, anchor, budget: int, tau: float, lam: float, mode: int = MODE_VOTE,
           keep_last: bool = True, c_max: int | None = None) -> Selection:
    """Sec. 3.2.2 Eqs. 9-10, Sec. 3.2.3 Eq. 11 and Algorithm 1's selection/order."""
    mass = np.ascontiguousarray(mass, dtype=np.float64)
    anchor = np.ascontiguousarray(anchor, dtype=np.float64)
    B, Hkv, T = mass.shape
    if group_mass is None:
        G = 1
        gm = np.zeros((B, Hkv, 1, T))
    else:
        gm = np.ascontiguousarray(group_mass, dtype=np.float64)
        G = gm.shape[2]
    c_max = budget if c_max is None else c_max
    idx = np.zeros((B, Hkv, c_max), dtype=np.int32)
    counts = np.zeros((B, Hkv), dtype=np.int32)
    votes = np.zeros((B, Hkv, T), dtype=np.int32)
    sc = np.zeros((B, Hkv, T), dtype=np.float64)
    cm = np.zeros((B, Hkv, G), dtype=np.float64)
    cs = np.zeros((B, Hkv, G), dtype=np.int32)
    rc = _load().oracle_select(B, Hkv, T, G, int(mode), float(tau), float(lam), int(bool(keep_last)),
                               int(budget), int(c_max), _ptr(gm), _ptr(mass), _ptr(anchor),
                               _ptr(idx), _ptr(counts), _ptr(votes), _ptr(sc), _ptr(cm), _ptr(cs))
    if rc != 0:
        raise ValueError("oracle_select rejected its arguments")
    return Selection(idx, counts, votes, sc, cm, cs)


def gather(src: np.ndarray, idx: np.ndarray, counts: np.ndarray) -> np.ndarray:
    """Appendix B: copy the retained rows (temporal order) into the compacted cache."""
    src = np.ascontiguousarray(src)
    B, H, T = src.shape[:3]
    c_max = idx.shape[2]
    row_bytes = src[0, 0, 0].nbytes
    dst = np.zeros((B, H, c_max) + src.shape[3:], dtype=src.dtype)
    rc = _load().oracle_gather(B, H, T, row_bytes, c_max, _ptr(src),
                               _ptr(np.ascontiguousarray(idx, dtype=np.int32)),
                               _ptr(np.ascontiguousarray(counts, dtype=np.int32)), _ptr(dst))
    if rc != 0:
        raise ValueError("oracle_gather rejected its arguments")
    return dst


@dataclass
class LayerResult:
    proxies: np.ndarray
    q_last: np.ndarray
    stats: np.ndarray
    group_mass: np.ndarray
    mass: np.ndarray
    anchor: np.ndarray
    sel: Selection
    k_out: np.ndarray
    v_out: np.ndarray


def select_layer(q_win, k, v, Hkv: int, budget: int, P: int = 512, G: int = 32, gamma: float = 10.0,
                 tau: float = 0.95, lam: float = 1.0, seed: int = 0, layer: int = 0, ddof: int = 0,
                 mode: int = MODE_VOTE, keep_last: bool = True, c_max=None, rope_f=None,
                 rope_l=None) -> LayerResult:
    """Algorithm 1 end to end for one layer (every KV head, every batch row)."""
    prox, ql, st = build_proxies(q_win, P, gamma, seed, layer, ddof, rope_f, rope_l)
    gm, mass, anchor = score(prox, ql, k, Hkv, G)
    sel = select(gm, mass, anchor, budget, tau, lam, mode, keep_last, c_max)
    return LayerResult(prox, ql, st, gm, mass, anchor, sel, gather(k, sel.idx, sel.counts),
                       gather(v, sel.idx, sel.counts))


def hidden_stats(hidden: np.ndarray, ddof: int = 0) -> np.ndarray:
    """Sec. 3.2.1 Eq. 4 over the prefill hidden states [B, T, D] (fp32, or
    bf16 bits as uint16): per (batch row, dim) mean, then the standard
    deviation from the squared deviations about it (two passes over the
    tokens, sums in token order).  Returns [B, 2, D] fp64."""
    lib = _load()
    h = np.ascontiguousarray(hidden)
    B, T, D = h.shape
    st = np.zeros((B, 2, D), dtype=np.float64)
    rc = lib.oracle_hidden_stats(B, T, D, ddof, _ptr(h), _dtype_code(h), _ptr(st))
    if rc != 0:
        raise ValueError("oracle_hidden_stats: invalid arguments")
    return st


def hidden_proxies(stats: np.ndarray, P: int, gamma: float, seed: int, layer: int = 0, b0: int = 0) -> np.ndarray:
    """Sec. 3.2.1 Eq. 5 in hidden space: [B, P, D] bf16 bits."""
    lib = _load()
    st = np.ascontiguousarray(stats, dtype=np.float64)
    B, _, D = st.shape
    hp = np.zeros((B, P, D), dtype=np.uint16)
    rc = lib.oracle_hidden_proxies(B, D, P, gamma, seed, layer, b0, _ptr(st), _ptr(hp))
    if rc != 0:
        raise ValueError("oracle_hidden_proxies: invalid arguments")
    return hp


def project_proxies(hp: np.ndarray, wq: np.ndarray, Hq: int, rope=None, with_pre: bool = False):
    """Sec. 3.2.1 Eq. 6: query proxies [B, Hq, P, d] bf16 bits from hidden
    proxies hp [B, P, D] (bf16 bits) and W_Q [Hq*d, D] (bf16 bits); rope =
    (cos, sin) [d/2] fp32 tables or None.  with_pre also returns the fp64
    values before rounding."""
    lib = _load()
    hp = np.ascontiguousarray(hp, dtype=np.uint16)
    wq = np.ascontiguousarray(wq, dtype=np.uint16)
    B, P, D = hp.shape
    d = wq.shape[0] // Hq
    out = np.zeros((B, Hq, P, d), dtype=np.uint16)
    pre = np.zeros((B, Hq, P, d), dtype=np.float64) if with_pre else None
    c = s = None
    if rope is not None:
        c = np.ascontiguousarray(rope[0], dtype=np.float32)
        s = np.ascontiguousarray(rope[1], dtype=np.float32)
    rc = lib.oracle_project_proxies(B, P, D, Hq, d, _ptr(hp), _ptr(wq), _ptr(c) if c is not None else None,
                                    _ptr(s) if s is not None else None, _ptr(out),
                                    _ptr(pre) if pre is not None else None)
    if rc != 0:
        raise ValueError("oracle_project_proxies: invalid arguments")
    return (out, pre) if with_pre else out


def decode_check(q_dec: np.ndarray, k: np.ndarray, idx: np.ndarray, counts: np.ndarray,
                 k_out: np.ndarray, v_out: np.ndarray):
    """Decode-time check (Fig. 1b's attention-mass coverage; decode attention
    over the fixed compacted cache, Sec. 3.1 / Sec. 3.2.3).

    q_dec [B, Hq, n_dec, d] bf16 bits (unscaled); k [B, Hkv, T, d];
    idx [B, Hkv, c_max], counts [B, Hkv]; k_out, v_out [B, Hkv, c_max, d].
    Returns (coverage [B, Hq, n_dec], out [B, Hq, n_dec, d]), fp64.
    """
    q_dec = np.ascontiguousarray(q_dec, dtype=np.uint16)
    k = np.ascontiguousarray(k)
    k_out = np.ascontiguousarray(k_out)
    v_out = np.ascontiguousarray(v_out)
    idx = np.ascontiguousarray(idx, dtype=np.int32)
    counts = np.ascontiguousarray(counts, dtype=np.int32)
    B, Hq, n_dec, d = q_dec.shape
    Hkv, T = k.shape[1], k.shape[2]
    c_max = idx.shape[2]
    assert k.shape == (B, Hkv, T, d) and k_out.shape == (B, Hkv, c_max, d) and v_out.shape == k_out.shape
    assert k_out.dtype == v_out.dtype
    cov = np.zeros((B, Hq, n_dec), dtype=np.float64)
    out = np.zeros((B, Hq, n_dec, d), dtype=np.float64)
    rc = _load().oracle_decode_check(B, Hq, Hkv, T, d, n_dec, _ptr(q_dec), _ptr(k), _dtype_code(k),
                                     _ptr(idx), _ptr(counts), c_max, _ptr(k_out), _ptr(v_out),
                                     _dtype_code(k_out), _ptr(cov), _ptr(out))
    if rc != 0:
        raise ValueError("oracle_decode_check rejected its arguments")
    return cov, out


SHAPE_SNAPKV, SHAPE_STREAMING, SHAPE_SINKS = 0, 1, 2
KEEP_SCORE = 2.0 ** 100


def window_rows(q_win: np.ndarray, n: int) -> np.ndarray:
    """The last n window queries of each head, scaled like the proxies (bf16 bits)."""
    q_win = np.ascontiguousarray(q_win)
    B, Hq, W, d = q_win.shape
    rows = np.zeros((B, Hq, n, d), dtype=np.uint16)
    if _load().oracle_window_rows(B, Hq, W, d, n, _ptr(q_win), _dtype_code(q_win), _ptr(rows)) != 0:
        raise ValueError("oracle_window_rows rejected its arguments")
    return rows


def shape_scores(mass: np.ndarray, kind: int, window: int = 0, pool: int = 1, sinks: int = 0) -> np.ndarray:
    """Per-key scores of the baseline selectors from a mass [B, Hkv, T] (fp64)."""
    mass = np.ascontiguousarray(mass, dtype=np.float64)
    B, Hkv, T = mass.shape
    out = np.zeros_like(mass)
    if _load().oracle_shape_scores(B, Hkv, T, int(kind), int(window), int(pool), int(sinks), _ptr(mass), _ptr(out)) != 0:
        raise ValueError("oracle_shape_scores rejected its arguments")
    return out


def baseline_select(name: str, q_win, k, v, Hkv: int, budget: int, seed: int = 0, layer: int = 0,
                    window: int = 32, pool: int = 5, sinks: int = 4, P: int = 512, c_max=None):
    """The baseline selectors end to end (Sec. 4.1 baselines as configured in the
    paper's appendix on them; LastAttn is the tau = 1 setting of select_layer).
    Returns (selection, score [B, Hkv, T], mass [B, Hkv, T])."""
    q_win = np.ascontiguousarray(q_win)
    k = np.ascontiguousarray(k)
    B, Hq, W, d = q_win.shape
    T = k.shape[2]
    if name == "snapkv":
        rows = window_rows(q_win, window)
        prox, ql, _ = build_proxies(q_win, 32, 0.0, seed, layer)   # q_last only (the anchor query)
        _, mass, anchor = score(rows, ql, k, Hkv, 1)
        sc = shape_scores(mass, SHAPE_SNAPKV, window=window, pool=pool)
    elif name == "streaming":
        mass = np.zeros((B, Hkv, T))
        anchor = np.zeros((B, Hkv, T))
        sc = shape_scores(mass, SHAPE_STREAMING, sinks=sinks)
    elif name == "expected":
        prox, ql, _ = build_proxies(q_win, P, 1.0, seed, layer)
        _, mass, anchor = score(prox, ql, k, Hkv, 32)
        sc = shape_scores(mass, SHAPE_SINKS, sinks=sinks)
    else:
        raise ValueError(name)
    sel = select(None, sc, anchor, budget, 1.0, 0.0, MODE_MASS, keep_last=False, c_max=c_max)
    return sel, sc, mass
