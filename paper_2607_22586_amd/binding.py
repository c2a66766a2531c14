"""ctypes binding of libmmshiftkv (C ABI in include/mmshiftkv.h).

Argument marshalling only: every step runs in the library's HIP kernels on
the GPU.  Tensors are torch tensors on a ROCm device; the library enqueues on
the current torch stream of that device.  If the shared library is missing
or cannot be loaded, every call raises -- there is no CPU fallback.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libmmshiftkv.so")

MMSKV_OK, MMSKV_EINVAL, MMSKV_EUNSUPPORTED, MMSKV_EWORKSPACE, MMSKV_EHIP, MMSKV_ESCRATCH = 0, -1, -2, -3, -4, -5
NOALLOC_SCRATCH_BYTES = 32 << 20
MMSKV_F32, MMSKV_BF16 = 0, 1
MMSKV_VOTE, MMSKV_MASS = 0, 1

EXPORTED = ("mmshiftkv_build_proxies", "mmshiftkv_score_workspace", "mmshiftkv_score",
            "mmshiftkv_score_lse", "mmshiftkv_score_lse_blocks", "mmshiftkv_score_lse_merge",
            "mmshiftkv_score_mass", "mmshiftkv_select_workspace",
            "mmshiftkv_select_topk", "mmshiftkv_select_tau", "mmshiftkv_select_vote", "mmshiftkv_select_pick",
            "mmshiftkv_gather_kv", "mmshiftkv_status_string",
            "mmshiftkv_version", "mmshiftkv_hidden_stats_workspace", "mmshiftkv_hidden_stats",
            "mmshiftkv_hidden_proxies", "mmshiftkv_project_proxies", "mmshiftkv_decode_workspace",
            "mmshiftkv_decode_check", "mmshiftkv_window_rows", "mmshiftkv_shape_scores",
            "mmshiftkv_score_noalloc")


class Shape(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int32), ("Hq", ctypes.c_int32), ("Hkv", ctypes.c_int32),
                ("T", ctypes.c_int32), ("W", ctypes.c_int32), ("d", ctypes.c_int32)]


class HShape(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int32), ("T", ctypes.c_int32), ("D", ctypes.c_int32)]


class Strides(ctypes.Structure):
    _fields_ = [("sb", ctypes.c_int64), ("sh", ctypes.c_int64), ("st", ctypes.c_int64)]


class Params(ctypes.Structure):
    _fields_ = [("P", ctypes.c_int32), ("G", ctypes.c_int32), ("gamma", ctypes.c_double),
                ("tau", ctypes.c_double), ("lambda_", ctypes.c_double),
                ("std_ddof", ctypes.c_int32), ("layer", ctypes.c_int32),
                ("seed", ctypes.c_uint64), ("mode", ctypes.c_int32), ("keep_last", ctypes.c_int32)]


class MMShiftKVError(RuntimeError):
    def __init__(self, fn: str, status: int):
        super().__init__("%s failed: %s (%d)" % (fn, status_string(status), status))
        self.status = status


_lib = None


def load_library(path: str | None = None):
    """Load libmmshiftkv.so (raises if it is missing: there is no fallback)."""
    global _lib
    if _lib is not None and path is None:
        return _lib
    p = path or LIB_PATH
    if not os.path.exists(p):
        raise RuntimeError("libmmshiftkv.so is not built (%s); run __graft_entry__.build() or "
                           "python -m paper_2607_22586_amd.build" % p)
    lib = ctypes.CDLL(p)
    V, I32, I64, SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    PS, PP, PT = ctypes.POINTER(Shape), ctypes.POINTER(Params), ctypes.POINTER(Strides)
    lib.mmshiftkv_build_proxies.argtypes = [PS, PP, V, I32, PT, V, V, V, V, V, V, V, V]
    lib.mmshiftkv_score_workspace.argtypes = [PS, PP]
    lib.mmshiftkv_score_workspace.restype = SZ
    lib.mmshiftkv_score.argtypes = [PS, PP, V, V, V, I32, PT, V, V, V, V, SZ, V]
    lib.mmshiftkv_score_lse.argtypes = [PS, PP, V, V, V, I32, PT, V, SZ, V]
    lib.mmshiftkv_score_lse_blocks.argtypes = [PS, PP, V, V, V, I32, PT, V, SZ, V]
    lib.mmshiftkv_score_lse_merge.argtypes = [PS, PP, V, V, V, I32, PT, V, SZ, V]
    lib.mmshiftkv_score_mass.argtypes = [PS, PP, V, V, V, I32, PT, V, V, V, V, SZ, V]
    lib.mmshiftkv_score_noalloc.argtypes = [PS, PP, V, V, V, I32, PT, V, V, V, V]
    lib.mmshiftkv_select_workspace.argtypes = [PS, PP]
    lib.mmshiftkv_select_workspace.restype = SZ
    lib.mmshiftkv_select_topk.argtypes = [PS, PP, V, V, V, V, I32, I32, V, V, V, V, SZ, V]
    lib.mmshiftkv_select_tau.argtypes = [PS, PP, V, V, SZ, V]
    lib.mmshiftkv_select_vote.argtypes = [PS, PP, V, V, V, V, SZ, V]
    lib.mmshiftkv_select_pick.argtypes = [PS, PP, V, I32, I32, V, V, V, SZ, V]
    lib.mmshiftkv_gather_kv.argtypes = [PS, V, V, I32, PT, PT, V, V, I32, V, V, V]
    PH = ctypes.POINTER(HShape)
    lib.mmshiftkv_hidden_stats_workspace.argtypes = [PH]
    lib.mmshiftkv_hidden_stats_workspace.restype = SZ
    lib.mmshiftkv_hidden_stats.argtypes = [PH, I32, V, I32, I64, I64, V, V, SZ, V]
    lib.mmshiftkv_hidden_proxies.argtypes = [PH, PP, V, V, V]
    lib.mmshiftkv_project_proxies.argtypes = [PH, I32, I32, I32, V, V, V, V, V, V]
    lib.mmshiftkv_decode_workspace.argtypes = [PS, I32]
    lib.mmshiftkv_decode_workspace.restype = SZ
    lib.mmshiftkv_decode_check.argtypes = [PS, I32, V, V, I32, PT, V, V, I32, V, V, V, V, V, SZ, V]
    lib.mmshiftkv_window_rows.argtypes = [PS, I32, V, I32, PT, V, V, V]
    lib.mmshiftkv_shape_scores.argtypes = [PS, I32, I32, I32, I32, V, V, V]
    lib.mmshiftkv_status_string.argtypes = [ctypes.c_int]
    lib.mmshiftkv_status_string.restype = ctypes.c_char_p
    lib.mmshiftkv_version.restype = ctypes.c_int
    for name in ("mmshiftkv_build_proxies", "mmshiftkv_score", "mmshiftkv_score_lse",
                 "mmshiftkv_score_lse_blocks", "mmshiftkv_score_lse_merge",
                 "mmshiftkv_score_mass", "mmshiftkv_select_topk", "mmshiftkv_select_tau",
                 "mmshiftkv_select_vote", "mmshiftkv_select_pick", "mmshiftkv_gather_kv",
                 "mmshiftkv_hidden_stats", "mmshiftkv_hidden_proxies", "mmshiftkv_project_proxies",
                 "mmshiftkv_decode_check", "mmshiftkv_window_rows", "mmshiftkv_shape_scores",
            "mmshiftkv_score_noalloc"):
        getattr(lib, name).restype = ctypes.c_int
    if path is None:
        _lib = lib
    return lib


def status_string(status: int) -> str:
    return load_library().mmshiftkv_status_string(int(status)).decode()


def _check(fn: str, rc: int):
    if rc != MMSKV_OK:
        raise MMShiftKVError(fn, rc)


@dataclass
class SelectionConfig:
    """Method parameters; defaults are the paper's (Sec. 4.1, Appendix B)."""
    P: int = 512
    G: int = 32
    gamma: float = 10.0
    tau: float = 0.95
    lam: float = 1.0
    std_ddof: int = 0
    layer: int = 0
    seed: int = 0
    mode: int = MMSKV_VOTE
    keep_last: bool = True

    def c_params(self) -> Params:
        return Params(int(self.P), int(self.G), float(self.gamma), float(self.tau), float(self.lam),
                      int(self.std_ddof), int(self.layer), int(self.seed) & 0xFFFFFFFFFFFFFFFF,
                      int(self.mode), int(bool(self.keep_last)))


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return MMSKV_F32
    if t.dtype == torch.bfloat16:
        return MMSKV_BF16
    raise TypeError("expected float32 or bfloat16, got %s" % t.dtype)


def _dev(t: torch.Tensor) -> torch.device:
    if not t.is_cuda:
        raise ValueError("libmmshiftkv takes device tensors (got a %s tensor)" % t.device)
    return t.device


def _strides4(t: torch.Tensor) -> Strides:
    if t.dim() != 4 or t.stride(3) != 1:
        raise ValueError("expected a [batch, head, token, d] tensor with contiguous d")
    return Strides(t.stride(0), t.stride(1), t.stride(2))


def _stream(device) -> ctypes.c_void_p:
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _p(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _shape(B, Hq, Hkv, T, W, d) -> Shape:
    return Shape(int(B), int(Hq), int(Hkv), int(T), int(W), int(d))


# ----------------------------------------------------------------------------
# the four calls (plus the split score passes and workspace queries)
# ----------------------------------------------------------------------------
def build_proxies(q_win: torch.Tensor, cfg: SelectionConfig, T: int, Hkv: int, rope_f=None,
                  rope_l=None, with_stats: bool = False, out=None):
    """mmshiftkv_build_proxies: returns (proxies [B,Hq,P,d] bf16, q_last [B,Hq,d] bf16[, stats]).
    `out` may hold preallocated (proxies, q_last) tensors."""
    dev = _dev(q_win)
    B, Hq, W, d = q_win.shape
    shape = _shape(B, Hq, Hkv, T, W, d)
    prm = cfg.c_params()
    if out is None:
        proxies = torch.empty((B, Hq, cfg.P, d), dtype=torch.bfloat16, device=dev)
        q_last = torch.empty((B, Hq, d), dtype=torch.bfloat16, device=dev)
    else:
        proxies, q_last = out
        if (proxies.dtype != torch.bfloat16 or q_last.dtype != torch.bfloat16 or not proxies.is_contiguous()
                or not q_last.is_contiguous() or tuple(proxies.shape) != (B, Hq, cfg.P, d)
                or tuple(q_last.shape) != (B, Hq, d)):
            raise ValueError("preallocated proxies/q_last do not match")
    stats = torch.empty((B, Hq, 2, d), dtype=torch.float64, device=dev) if with_stats else None
    tabs = []
    for rp in (rope_f, rope_l):
        if rp is None:
            tabs += [None, None]
        else:
            tabs += [rp[0].to(device=dev, dtype=torch.float32).contiguous(),
                     rp[1].to(device=dev, dtype=torch.float32).contiguous()]
    with torch.cuda.device(dev):
        rc = load_library().mmshiftkv_build_proxies(
            ctypes.byref(shape), ctypes.byref(prm), _p(q_win), _dtype_code(q_win),
            ctypes.byref(_strides4(q_win)), *[_p(t) for t in tabs], _p(proxies), _p(q_last),
            _p(stats), _stream(dev))
    _check("mmshiftkv_build_proxies", rc)
    return (proxies, q_last, stats) if with_stats else (proxies, q_last)


# hidden-state form of the proxies (statistics of the prefill hidden states,
# samples in hidden space, projection by each head's W_Q)
def hidden_stats_workspace(B: int, T: int, D: int) -> int:
    return int(load_library().mmshiftkv_hidden_stats_workspace(ctypes.byref(HShape(int(B), int(T), int(D)))))


def hidden_stats(hidden: torch.Tensor, std_ddof: int = 0, out=None, workspace=None) -> torch.Tensor:
    """mmshiftkv_hidden_stats: hidden [B, T, D] (features contiguous) -> [B, 2, D] fp64."""
    dev = _dev(hidden)
    if hidden.dim() != 3 or hidden.stride(2) != 1:
        raise ValueError("expected a [batch, token, feature] tensor with contiguous features")
    B, T, D = hidden.shape
    hs = HShape(B, T, D)
    st = out if out is not None else torch.empty((B, 2, D), dtype=torch.float64, device=dev)
    if st.dtype != torch.float64 or not st.is_contiguous() or tuple(st.shape) != (B, 2, D):
        raise ValueError("preallocated stats do not match")
    ws = workspace if workspace is not None else _ws(hidden_stats_workspace(B, T, D), dev)
    with torch.cuda.device(dev):
        rc = load_library().mmshiftkv_hidden_stats(
            ctypes.byref(hs), int(std_ddof), _p(hidden), _dtype_code(hidden), hidden.stride(0),
            hidden.stride(1), _p(st), _p(ws), ws.numel() * ws.element_size(), _stream(dev))
    _check("mmshiftkv_hidden_stats", rc)
    return st


def hidden_proxies(stats: torch.Tensor, cfg: SelectionConfig, T: int = 1, out=None) -> torch.Tensor:
    """mmshiftkv_hidden_proxies: stats [B, 2, D] fp64 -> samples [B, P, D] bf16."""
    dev = _dev(stats)
    B, two, D = stats.shape
    if two != 2 or stats.dtype != torch.float64 or not stats.is_contiguous():
        raise ValueError("expected contiguous fp64 stats [B, 2, D]")
    hp = out if out is not None else torch.empty((B, cfg.P, D), dtype=torch.bfloat16, device=dev)
    if hp.dtype != torch.bfloat16 or not hp.is_contiguous() or tuple(hp.shape) != (B, cfg.P, D):
        raise ValueError("preallocated samples do not match")
    with torch.cuda.device(dev):
        rc = load_library().mmshiftkv_hidden_proxies(ctypes.byref(HShape(B, int(T), D)),
                                                     ctypes.byref(cfg.c_params()), _p(stats), _p(hp),
                                                     _stream(dev))
    _check("mmshiftkv_hidden_proxies", rc)
    return hp


def project_proxies(hp: torch.Tensor, wq: torch.Tensor, Hq: int, rope=None, out=None) -> torch.Tensor:
    """mmshiftkv_project_proxies: samples [B, P, D] bf16 and W_Q [Hq*d, D] bf16
    -> proxies [B, Hq, P, d] bf16; rope = (cos, sin) [d/2] fp32 or None."""
    dev = _dev(hp)
    B, P, D = hp.shape
    N, D2 = wq.shape
    if D2 != D or N % Hq != 0:
        raise ValueError("W_Q must be [Hq*d, D]")
    d = N // Hq
    if hp.dtype != torch.bfloat16 or wq.dtype != torch.bfloat16 or not hp.is_contiguous() \
            or not wq.is_contiguous():
        raise ValueError("samples and W_Q must be contiguous bf16")
    pr = out if out is not None else torch.empty((B, Hq, P, d), dtype=torch.bfloat16, device=dev)
    if pr.dtype != torch.bfloat16 or not pr.is_contiguous() or tuple(pr.shape) != (B, Hq, P, d):
        raise ValueError("preallocated proxies do not match")
    tabs = [None, None]
    if rope is not None:
        tabs = [rope[0].to(device=dev, dtype=torch.float32).contiguous(),
                rope[1].to(device=dev, dtype=torch.float32).contiguous()]
    with torch.cuda.device(dev):
        rc = load_library().mmshiftkv_project_proxies(ctypes.byref(HShape(B, 1, D)), P, int(Hq), d, _p(hp),
                                                      _p(wq), _p(tabs[0]), _p(tabs[1]), _p(pr), _stream(dev))
    _check("mmshiftkv_project_proxies", rc)
    return pr


def score_workspace(B, Hq, Hkv, T, W, d, cfg: SelectionConfig) -> int:
    return int(load_library().mmshiftkv_score_workspace(ctypes.byref(_shape(B, Hq, Hkv, T, W, d)),
                                                         ctypes.byref(cfg.c_params())))


def select_workspace(B, Hq, Hkv, T, W, d, cfg: SelectionConfig) -> int:
    return int(load_library().mmshiftkv_select_workspace(ctypes.byref(_shape(B, Hq, Hkv, T, W, d)),
                                                          ctypes.byref(cfg.c_params())))


def _ws(nbytes: int, dev) -> torch.Tensor:
    return torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=dev)


@dataclass
class ScoreOut:
    group_mass: torch.Tensor | None    # [B, Hkv, G, T] fp32
    mass: torch.Tensor                 # [B, Hkv, T] fp32
    anchor: torch.Tensor               # [B, Hkv, T] fp32


def _score_call(which: str, proxies, q_last, k, cfg, W, out: ScoreOut | None, workspace):
    dev = _dev(k)
    B, Hkv, T, d = k.shape
    Hq = proxies.shape[1]
    if proxies.dtype != torch.bfloat16 or q_last.dtype != torch.bfloat16:
        raise TypeError("proxies and q_last are bf16")
    if not (proxies.is_contiguous() and q_last.is_contiguous()):
        raise ValueError("proxies and q_last must be contiguous")
    if tuple(proxies.shape) != (B, Hq, cfg.P, d) or tuple(q_last.shape) != (B, Hq, d):
        raise ValueError("proxies/q_last shapes do not match k")
    shape = _shape(B, Hq, Hkv, T, W, d)
    prm = cfg.c_params()
    lib = load_library()
    need = int(lib.mmshiftkv_score_workspace(ctypes.byref(shape), ctypes.byref(prm)))
    ws = workspace if workspace is not None else _ws(need, dev)
    strides = _strides4(k)
    with torch.cuda.device(dev):
        if which in ("lse", "lse_blocks", "lse_merge"):
            name = "mmshiftkv_score_" + which
            rc = getattr(lib, name)(ctypes.byref(shape), ctypes.byref(prm), _p(proxies), _p(q_last),
                                    _p(k), _dtype_code(k), ctypes.byref(strides), _p(ws),
                                    ws.numel() * ws.element_size(), _stream(dev))
            _check(name, rc)
            return ws
        if out is None:
            gm = (torch.empty((B, Hkv, cfg.G, T), dtype=torch.float32, device=dev)
                  if cfg.mode == MMSKV_VOTE else None)
            out = ScoreOut(gm, torch.empty((B, Hkv, T), dtype=torch.float32, device=dev),
                           torch.empty((B, Hkv, T), dtype=torch.float32, device=dev))
        fn = lib.mmshiftkv_score if which == "full" else lib.mmshiftkv_score_mass
        rc = fn(ctypes.byref(shape), ctypes.byref(prm), _p(proxies), _p(q_last), _p(k), _dtype_code(k),
                ctypes.byref(strides), _p(out.group_mass), _p(out.mass), _p(out.anchor), _p(ws),
                ws.numel() * ws.element_size(), _stream(dev))
    _check("mmshiftkv_score" if which == "full" else "mmshiftkv_score_mass", rc)
    return out


def score(proxies, q_last, k, cfg: SelectionConfig, W: int = 1, out: ScoreOut | None = None,
          workspace: torch.Tensor | None = None) -> ScoreOut:
    """mmshiftkv_score: group masses, total mass and anchor for every (b, KV head)."""
    return _score_call("full", proxies, q_last, k, cfg, W, out, workspace)


def score_noalloc(proxies, q_last, k, cfg: SelectionConfig, out: ScoreOut, W: int = 1) -> ScoreOut:
    """mmshiftkv_score_noalloc: mmshiftkv_score with the library's per-GPU
    scratch instead of a workspace (the outputs `out` are the caller's)."""
    dev = _dev(k)
    B, Hkv, T, d = k.shape
    Hq = proxies.shape[1]
    if proxies.dtype != torch.bfloat16 or q_last.dtype != torch.bfloat16:
        raise TypeError("proxies and q_last are bf16")
    if not (proxies.is_contiguous() and q_last.is_contiguous()):
        raise ValueError("proxies and q_last must be contiguous")
    shape = _shape(B, Hq, Hkv, T, W, d)
    prm = cfg.c_params()
    with torch.cuda.device(dev):
        rc = load_library().mmshiftkv_score_noalloc(
            ctypes.byref(shape), ctypes.byref(prm), _p(proxies), _p(q_last), _p(k), _dtype_code(k),
            ctypes.byref(_strides4(k)), _p(out.group_mass), _p(out.mass), _p(out.anchor), _stream(dev))
    _check("mmshiftkv_score_noalloc", rc)
    return out


def score_lse(proxies, q_last, k, cfg: SelectionConfig, workspace: torch.Tensor, W: int = 1,
              stage: str | None = None):
    """mmshiftkv_score_lse: the row log-sum-exp pass (result kept in `workspace`);
    with stage "blocks" or "merge" only that half (mmshiftkv_score_lse_blocks /
    _merge), which must run in that order on one workspace."""
    if stage not in (None, "blocks", "merge"):
        raise ValueError("stage is None, 'blocks' or 'merge'")
    return _score_call("lse" if stage is None else "lse_" + stage, proxies, q_last, k, cfg, W, None, workspace)


def score_mass(proxies, q_last, k, cfg: SelectionConfig, workspace: torch.Tensor, W: int = 1,
               out: ScoreOut | None = None) -> ScoreOut:
    """mmshiftkv_score_mass: the mass pass, after score_lse on the same workspace."""
    return _score_call("mass", proxies, q_last, k, cfg, W, out, workspace)


@dataclass
class Selected:
    idx: torch.Tensor        # [B, Hkv, c_max] int32 ascending, -1 padded
    counts: torch.Tensor     # [B, Hkv] int32
    votes: torch.Tensor | None


def select_topk(s: ScoreOut, cfg: SelectionConfig, budget: int, c_max: int | None = None,
                budgets: torch.Tensor | None = None, Hq: int | None = None, W: int = 1,
                want_votes: bool = False, out: Selected | None = None,
                workspace: torch.Tensor | None = None, stage: str | None = None) -> Selected:
    """mmshiftkv_select_topk: tau-sets, votes, score and budgeted top-k; with
    stage "tau", "vote" or "pick" only that stage's call (mmshiftkv_select_tau /
    _vote / _pick), which must run in that order on one workspace."""
    dev = _dev(s.mass)
    B, Hkv, T = s.mass.shape
    Hq = Hkv if Hq is None else Hq
    c_max = int(budget if c_max is None else c_max)
    shape = _shape(B, Hq, Hkv, T, 0, 0)           # W and d are not read by the selection
    prm = cfg.c_params()
    lib = load_library()
    need = int(lib.mmshiftkv_select_workspace(ctypes.byref(shape), ctypes.byref(prm)))
    ws = workspace if workspace is not None else _ws(need, dev)
    if out is None:
        out = Selected(torch.empty((B, Hkv, c_max), dtype=torch.int32, device=dev),
                       torch.empty((B, Hkv), dtype=torch.int32, device=dev),
                       torch.empty((B, Hkv, T), dtype=torch.uint8, device=dev) if want_votes else None)
    if budgets is not None:
        budgets = budgets.to(device=dev, dtype=torch.int32).contiguous()
    nbytes = ws.numel() * ws.element_size()
    S, Pm = ctypes.byref(shape), ctypes.byref(prm)
    with torch.cuda.device(dev):
        if stage is None:
            name = "mmshiftkv_select_topk"
            rc = lib.mmshiftkv_select_topk(S, Pm, _p(s.group_mass), _p(s.mass), _p(s.anchor), _p(budgets),
                                           int(budget), c_max, _p(out.idx), _p(out.counts), _p(out.votes),
                                           _p(ws), nbytes, _stream(dev))
        elif stage == "tau":
            name = "mmshiftkv_select_tau"
            rc = lib.mmshiftkv_select_tau(S, Pm, _p(s.group_mass), _p(ws), nbytes, _stream(dev))
        elif stage == "vote":
            name = "mmshiftkv_select_vote"
            rc = lib.mmshiftkv_select_vote(S, Pm, _p(s.mass), _p(s.anchor), _p(out.votes), _p(ws), nbytes,
                                           _stream(dev))
        elif stage == "pick":
            name = "mmshiftkv_select_pick"
            rc = lib.mmshiftkv_select_pick(S, Pm, _p(budgets), int(budget), c_max, _p(out.idx), _p(out.counts),
                                           _p(ws), nbytes, _stream(dev))
        else:
            raise ValueError("stage must be None, 'tau', 'vote' or 'pick'")
    _check(name, rc)
    return out


def decode_workspace(B, Hq, Hkv, T, d, n_dec) -> int:
    return int(load_library().mmshiftkv_decode_workspace(ctypes.byref(_shape(B, Hq, Hkv, T, 1, d)), int(n_dec)))


def decode_check(q_dec: torch.Tensor, k: torch.Tensor, sel: Selected, k_out: torch.Tensor, v_out: torch.Tensor,
                 workspace: torch.Tensor | None = None, out=None):
    """mmshiftkv_decode_check: (coverage [B, Hq, n_dec] fp32, out [B, Hq, n_dec, d] fp32) of the
    decode queries q_dec [B, Hq, n_dec, d] bf16 against the full cache k and the compacted
    cache (k_out, v_out) of the selection `sel`."""
    dev = _dev(k)
    B, Hq, n_dec, d = q_dec.shape
    Hkv, T = k.shape[1], k.shape[2]
    if q_dec.dtype != torch.bfloat16 or not q_dec.is_contiguous():
        raise ValueError("q_dec must be a contiguous bf16 tensor")
    if k_out.dtype != k.dtype or v_out.dtype != k.dtype or not k_out.is_contiguous() or not v_out.is_contiguous():
        raise ValueError("k_out and v_out must be contiguous and of k's dtype")
    c_max = sel.idx.shape[2]
    shape = _shape(B, Hq, Hkv, T, 1, d)
    lib = load_library()
    need = int(lib.mmshiftkv_decode_workspace(ctypes.byref(shape), int(n_dec)))
    ws = workspace if workspace is not None else _ws(need, dev)
    if out is None:
        out = (torch.empty((B, Hq, n_dec), dtype=torch.float32, device=dev),
               torch.empty((B, Hq, n_dec, d), dtype=torch.float32, device=dev))
    with torch.cuda.device(dev):
        rc = lib.mmshiftkv_decode_check(ctypes.byref(shape), int(n_dec), _p(q_dec), _p(k), _dtype_code(k),
                                        ctypes.byref(_strides4(k)), _p(sel.idx), _p(sel.counts), c_max,
                                        _p(k_out), _p(v_out), _p(out[0]), _p(out[1]), _p(ws),
                                        ws.numel() * ws.element_size(), _stream(dev))
    _check("mmshiftkv_decode_check", rc)
    return out


MMSKV_SHAPE_SNAPKV, MMSKV_SHAPE_STREAMING, MMSKV_SHAPE_SINKS = 0, 1, 2


def window_rows(q_win: torch.Tensor, n: int, T: int, Hkv: int):
    """mmshiftkv_window_rows: (rows [B, Hq, n, d] bf16 scaled like proxies, q_last [B, Hq, d] bf16)."""
    dev = _dev(q_win)
    B, Hq, W, d = q_win.shape
    rows = torch.empty((B, Hq, n, d), dtype=torch.bfloat16, device=dev)
    ql = torch.empty((B, Hq, d), dtype=torch.bfloat16, device=dev)
    shape = _shape(B, Hq, Hkv, T, W, d)
    with torch.cuda.device(dev):
        rc = load_library().mmshiftkv_window_rows(ctypes.byref(shape), int(n), _p(q_win), _dtype_code(q_win),
                                                  ctypes.byref(_strides4(q_win)), _p(rows), _p(ql), _stream(dev))
    _check("mmshiftkv_window_rows", rc)
    return rows, ql


def shape_scores(mass: torch.Tensor | None, kind: int, B: int, Hkv: int, T: int, window: int = 0, pool: int = 1,
                 sinks: int = 0, out: torch.Tensor | None = None, device=None) -> torch.Tensor:
    """mmshiftkv_shape_scores: per-key baseline scores [B, Hkv, T] fp32."""
    dev = _dev(mass) if mass is not None else torch.device(device if device is not None else "cuda:0")
    score = out if out is not None else torch.empty((B, Hkv, T), dtype=torch.float32, device=dev)
    shape = _shape(B, 0, Hkv, T, 0, 0)            # only B, Hkv and T are read
    with torch.cuda.device(dev):
        rc = load_library().mmshiftkv_shape_scores(ctypes.byref(shape), int(kind), int(window), int(pool), int(sinks),
                                                   _p(mass), _p(score), _stream(dev))
    _check("mmshiftkv_shape_scores", rc)
    return score


BASELINES = ("snapkv", "streaming", "expected")


def baseline_select(name: str, q_win, k, v, budget: int, seed: int = 0, layer: int = 0, window: int = 32,
                    pool: int = 5, sinks: int = 4, P: int = 512, c_max=None):
    """A baseline selector end to end on the library's kernels: (Selected, score, mass, k_out, v_out).
    snapkv: window rows -> mass pass -> pooled scores; streaming: sinks + recency;
    expected: gamma = 1 proxies -> mass pass -> sinks; then the MASS-mode top-C and the gather."""
    B, Hkv, T, d = k.shape
    Hq, W = q_win.shape[1], q_win.shape[2]
    dev = _dev(k)
    sel_cfg = SelectionConfig(mode=MMSKV_MASS, keep_last=False, seed=seed, layer=layer)
    mass = None
    anchor = torch.zeros((B, Hkv, T), dtype=torch.float32, device=dev)
    if name == "snapkv":
        rows, ql = window_rows(q_win, window, T, Hkv)
        cfg = SelectionConfig(P=window, G=1, mode=MMSKV_MASS, seed=seed, layer=layer)
        sc = score(rows, ql, k, cfg, W)
        mass, anchor = sc.mass, sc.anchor
        scores = shape_scores(mass, MMSKV_SHAPE_SNAPKV, B, Hkv, T, window=window, pool=pool)
    elif name == "streaming":
        scores = shape_scores(None, MMSKV_SHAPE_STREAMING, B, Hkv, T, sinks=sinks, device=dev)
    elif name == "expected":
        cfg = SelectionConfig(P=P, gamma=1.0, mode=MMSKV_MASS, seed=seed, layer=layer)
        prox, ql = build_proxies(q_win, cfg, T, Hkv)
        sc = score(prox, ql, k, cfg, W)
        mass, anchor = sc.mass, sc.anchor
        scores = shape_scores(mass, MMSKV_SHAPE_SINKS, B, Hkv, T, sinks=sinks)
    else:
        raise ValueError("unknown baseline %r" % name)
    sel = select_topk(ScoreOut(None, scores, anchor), sel_cfg, budget, c_max, None, Hq, W)
    ko, vo = gather_kv(k, v, sel)
    return sel, scores, mass, ko, vo


def gather_kv(k: torch.Tensor, v: torch.Tensor, sel: Selected, out=None):
    """mmshiftkv_gather_kv: compacted K'/V' [B, Hkv, c_max, d] in temporal order."""
    dev = _dev(k)
    B, Hkv, T, d = k.shape
    if v.shape != k.shape or v.dtype != k.dtype:
        raise ValueError("k and v must have the same shape and dtype")
    c_max = sel.idx.shape[2]
    shape = _shape(B, 0, Hkv, T, 0, d)            # Hq and W are not read by the gather
    if out is None:
        out = (torch.empty((B, Hkv, c_max, d), dtype=k.dtype, device=dev),
               torch.empty((B, Hkv, c_max, d), dtype=k.dtype, device=dev))
    with torch.cuda.device(dev):
        rc = load_library().mmshiftkv_gather_kv(
            ctypes.byref(shape), _p(k), _p(v), _dtype_code(k), ctypes.byref(_strides4(k)),
            ctypes.byref(_strides4(v)), _p(sel.idx), _p(sel.counts), c_max, _p(out[0]), _p(out[1]),
            _stream(dev))
    _check("mmshiftkv_gather_kv", rc)
    return out


@dataclass
class LayerOut:
    proxies: torch.Tensor
    q_last: torch.Tensor
    scores: ScoreOut
    sel: Selected
    k_out: torch.Tensor
    v_out: torch.Tensor


def select_layer(q_win, k, v, budget: int, cfg: SelectionConfig | None = None, c_max=None,
                 budgets=None, rope_f=None, rope_l=None, want_votes=False) -> LayerOut:
    """All four calls for one layer (Algorithm 1), on the current stream."""
    cfg = cfg or SelectionConfig()
    B, Hkv, T, d = k.shape
    Hq, W = q_win.shape[1], q_win.shape[2]
    prox, ql = build_proxies(q_win, cfg, T, Hkv, rope_f, rope_l)
    sc = score(prox, ql, k, cfg, W)
    sel = select_topk(sc, cfg, budget, c_max, budgets, Hq, W, want_votes)
    ko, vo = gather_kv(k, v, sel)
    return LayerOut(prox, ql, sc, sel, ko, vo)
