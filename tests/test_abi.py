"""The C-ABI library loads, exports every symbol include/mmshiftkv.h declares,
and validates its arguments on the host (CPU only: no call here reaches a
kernel launch; every call below is rejected before anything is enqueued)."""
import ctypes
import os
import re
import shutil
import subprocess

import pytest

from paper_2607_22586_amd import binding as bd

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "mmshiftkv.h")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(bd.LIB_PATH):
        from paper_2607_22586_amd import build
        build.build()
    return bd.load_library()


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"\b(mmshiftkv_[a-z_]+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for n in ("mmshiftkv_build_proxies", "mmshiftkv_score", "mmshiftkv_select_topk", "mmshiftkv_gather_kv"):
        assert n in names
    assert set(names) == set(bd.EXPORTED)


def test_every_declared_symbol_is_exported(lib):
    for n in declared_functions():
        assert hasattr(lib, n), n
    if shutil.which("nm"):
        out = subprocess.run(["nm", "-D", "--defined-only", bd.LIB_PATH], capture_output=True,
                             text=True).stdout
        exported = set(re.findall(r" T (mmshiftkv_\w+)", out))
        assert set(declared_functions()) <= exported


def test_header_compiles_as_c99(tmp_path):
    if shutil.which("gcc") is None:
        pytest.skip("no gcc")
    src = tmp_path / "t.c"
    src.write_text('#include "mmshiftkv.h"\nint main(void){ mmskv_params p; mmskv_shape s; '
                   '(void)p; (void)s; return (int)sizeof(mmskv_params); }\n')
    subprocess.run(["gcc", "-std=c99", "-Wall", "-Werror", "-I", os.path.dirname(HEADER), "-c",
                    str(src), "-o", str(tmp_path / "t.o")], check=True)


def test_struct_layout_matches_header(tmp_path):
    if shutil.which("gcc") is None:
        pytest.skip("no gcc")
    src = tmp_path / "layout.c"
    src.write_text('#include <stdio.h>\n#include <stddef.h>\n#include "mmshiftkv.h"\nint main(void){'
                   'printf("%zu %zu %zu %zu %zu %zu\\n", sizeof(mmskv_params), offsetof(mmskv_params, gamma),'
                   ' offsetof(mmskv_params, seed), offsetof(mmskv_params, keep_last), sizeof(mmskv_shape),'
                   ' sizeof(mmskv_strides)); return 0; }\n')
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-std=c99", "-I", os.path.dirname(HEADER), str(src), "-o", str(exe)], check=True)
    got = [int(x) for x in subprocess.run([str(exe)], capture_output=True, text=True).stdout.split()]
    want = [ctypes.sizeof(bd.Params), bd.Params.gamma.offset, bd.Params.seed.offset,
            bd.Params.keep_last.offset, ctypes.sizeof(bd.Shape), ctypes.sizeof(bd.Strides)]
    assert got == want


def test_status_strings(lib):
    assert bd.status_string(0) == "ok"
    assert "workspace" in bd.status_string(-3)
    assert lib.mmshiftkv_version() >= 100


# ---------------------------------------------------------------- host validation
FAKE = ctypes.c_void_p(0x10000)        # aligned, never dereferenced: calls fail validation first


def _shape(B=1, Hq=4, Hkv=1, T=1024, W=16, d=64):
    return bd.Shape(B, Hq, Hkv, T, W, d)


def _params(**kw):
    c = bd.SelectionConfig(**kw)
    return c.c_params()


def _build(lib, shape, prm, q=FAKE, prox=FAKE, ql=FAKE, strides=None, dtype=1, rope=(None, None)):
    st = strides or bd.Strides(shape.Hq * shape.W * shape.d, shape.W * shape.d, shape.d)
    return lib.mmshiftkv_build_proxies(ctypes.byref(shape), ctypes.byref(prm), q, dtype, ctypes.byref(st),
                                       rope[0], rope[1], None, None, prox, ql, None, None)


@pytest.mark.parametrize("shape,params,code", [
    (dict(d=96), {}, bd.MMSKV_EUNSUPPORTED),
    (dict(d=0), {}, bd.MMSKV_EINVAL),
    (dict(Hq=6, Hkv=4), {}, bd.MMSKV_EINVAL),
    (dict(B=0), {}, bd.MMSKV_EINVAL),
    (dict(B=70000), {}, bd.MMSKV_EINVAL),
    (dict(T=0), {}, bd.MMSKV_EINVAL),
    (dict(W=0), {}, bd.MMSKV_EINVAL),
    (dict(W=1), dict(std_ddof=1), bd.MMSKV_EINVAL),
    ({}, dict(P=500, G=32), bd.MMSKV_EINVAL),
    ({}, dict(P=256, G=32), bd.MMSKV_EUNSUPPORTED),      # groups of 8 rows
    ({}, dict(P=512 * 16, G=512), bd.MMSKV_EUNSUPPORTED),
    ({}, dict(tau=0.0), bd.MMSKV_EINVAL),
    ({}, dict(tau=1.5), bd.MMSKV_EINVAL),
    ({}, dict(lam=-1.0), bd.MMSKV_EINVAL),
    ({}, dict(gamma=-1.0), bd.MMSKV_EINVAL),
    ({}, dict(gamma=float("inf")), bd.MMSKV_EINVAL),
    ({}, dict(layer=70000), bd.MMSKV_EINVAL),
    ({}, dict(mode=7), bd.MMSKV_EINVAL),
])
def test_build_proxies_rejects(lib, shape, params, code):
    assert _build(lib, _shape(**shape), _params(**params)) == code


def test_build_proxies_rejects_pointers(lib):
    s, p = _shape(), _params()
    assert _build(lib, s, p, q=None) == bd.MMSKV_EINVAL
    assert _build(lib, s, p, prox=None) == bd.MMSKV_EINVAL
    assert _build(lib, s, p, dtype=5) == bd.MMSKV_EINVAL
    assert _build(lib, s, p, rope=(FAKE, None)) == bd.MMSKV_EINVAL
    assert _build(lib, s, p, strides=bd.Strides(-1, 0, 0)) == bd.MMSKV_EINVAL


def test_workspace_queries(lib):
    s, p = _shape(B=4, Hq=28, Hkv=4, T=16384, W=64, d=128), _params()
    ws = lib.mmshiftkv_score_workspace(ctypes.byref(s), ctypes.byref(p))
    # partial (max, sum) per (head, key block of at most 1024 keys, row) +
    # one lse per row; rows = Gh*P proxies + the anchor rows padded to 32
    # (the scaled anchor rows themselves are formed as the kernels stage them)
    rows_pad = 7 * 512 + 32
    assert ws >= 16 * (16384 // 1024) * rows_pad * 8 + 16 * rows_pad * 4
    assert ws % 256 == 0
    wsel = lib.mmshiftkv_select_workspace(ctypes.byref(s), ctypes.byref(p))
    assert wsel >= 16 * 16384 * 8
    bad = _shape(d=96)
    assert lib.mmshiftkv_score_workspace(ctypes.byref(bad), ctypes.byref(p)) == 0


def test_score_rejects(lib):
    s, p = _shape(), _params()
    st = bd.Strides(1024 * 64, 1024 * 64, 64)
    need = lib.mmshiftkv_score_workspace(ctypes.byref(s), ctypes.byref(p))
    call = lambda ws, nbytes, gm=FAKE, k=FAKE, strides=st, dtype=1: lib.mmshiftkv_score(  # noqa: E731
        ctypes.byref(s), ctypes.byref(p), FAKE, FAKE, k, dtype, ctypes.byref(strides), gm, FAKE, FAKE,
        ws, nbytes, None)
    assert call(FAKE, need - 1) == bd.MMSKV_EWORKSPACE
    assert call(None, need) == bd.MMSKV_EWORKSPACE
    assert call(ctypes.c_void_p(0x10010), need) == bd.MMSKV_EWORKSPACE      # not 256-byte aligned
    assert call(FAKE, need, gm=None) == bd.MMSKV_EINVAL                    # VOTE needs group masses
    assert call(FAKE, need, k=ctypes.c_void_p(0x10002)) == bd.MMSKV_EINVAL  # K rows not 16-byte aligned
    assert call(FAKE, need, strides=bd.Strides(0, 0, 3)) == bd.MMSKV_EINVAL
    assert call(FAKE, need, dtype=9) == bd.MMSKV_EINVAL


def test_select_rejects(lib):
    s, p = _shape(), _params()
    need = lib.mmshiftkv_select_workspace(ctypes.byref(s), ctypes.byref(p))
    call = lambda budget, c_max, ws=FAKE, nbytes=need, gm=FAKE, votes=None, prm=p: lib.mmshiftkv_select_topk(  # noqa: E731
        ctypes.byref(s), ctypes.byref(prm), gm, FAKE, FAKE, None, budget, c_max, FAKE, FAKE, votes, ws,
        nbytes, None)
    assert call(0, 64) == bd.MMSKV_EINVAL
    assert call(64, 63) == bd.MMSKV_EINVAL          # c_max below the budget
    assert call(64, 64, nbytes=need - 8) == bd.MMSKV_EWORKSPACE
    assert call(64, 64, gm=None) == bd.MMSKV_EINVAL
    assert call(64, 64, votes=FAKE, prm=_params(mode=bd.MMSKV_MASS)) == bd.MMSKV_EINVAL


def test_select_stages_reject(lib):
    """Each stage call checks the arguments it reads (and only those): the
    calls below stop at argument or workspace checks, before any launch."""
    s, p = _shape(), _params()
    pm = _params(mode=bd.MMSKV_MASS)
    need = lib.mmshiftkv_select_workspace(ctypes.byref(s), ctypes.byref(p))
    S, P, PM = ctypes.byref(s), ctypes.byref(p), ctypes.byref(pm)
    assert lib.mmshiftkv_select_tau(S, P, None, FAKE, need, None) == bd.MMSKV_EINVAL          # VOTE needs masses
    assert lib.mmshiftkv_select_tau(S, P, FAKE, FAKE, need - 8, None) == bd.MMSKV_EWORKSPACE
    assert lib.mmshiftkv_select_tau(S, PM, None, None, need, None) == bd.MMSKV_EWORKSPACE     # MASS: none read
    assert lib.mmshiftkv_select_vote(S, P, FAKE, None, None, FAKE, need, None) == bd.MMSKV_EINVAL   # no anchor
    assert lib.mmshiftkv_select_vote(S, PM, None, FAKE, None, FAKE, need, None) == bd.MMSKV_EINVAL  # no mass
    assert lib.mmshiftkv_select_vote(S, PM, FAKE, None, FAKE, FAKE, need, None) == bd.MMSKV_EINVAL  # votes
    assert lib.mmshiftkv_select_vote(S, P, None, FAKE, FAKE, FAKE, need - 8, None) == bd.MMSKV_EWORKSPACE
    assert lib.mmshiftkv_select_pick(S, P, None, 0, 64, FAKE, FAKE, FAKE, need, None) == bd.MMSKV_EINVAL
    assert lib.mmshiftkv_select_pick(S, P, None, 64, 63, FAKE, FAKE, FAKE, need, None) == bd.MMSKV_EINVAL
    assert lib.mmshiftkv_select_pick(S, P, None, 64, 64, None, FAKE, FAKE, need, None) == bd.MMSKV_EINVAL
    assert lib.mmshiftkv_select_pick(S, P, None, 64, 64, FAKE, FAKE, FAKE, need - 8, None) == bd.MMSKV_EWORKSPACE


def test_select_ignores_window_and_head_dim(lib):
    """The selection reads B, Hq, Hkv, T and the method parameters only: W = 0,
    d = 0 and a gamma / ddof the proxy call would refuse still pass its
    validation (the call below stops at the workspace check)."""
    s = _shape(W=0, d=0)
    p = _params()
    p.gamma = -1.0
    p.std_ddof = 7
    need = lib.mmshiftkv_select_workspace(ctypes.byref(s), ctypes.byref(p))
    assert need == lib.mmshiftkv_select_workspace(ctypes.byref(_shape()), ctypes.byref(_params())) > 0
    rc = lib.mmshiftkv_select_topk(ctypes.byref(s), ctypes.byref(p), FAKE, FAKE, FAKE, None, 64, 64, FAKE, FAKE,
                                   None, FAKE, need - 8, None)
    assert rc == bd.MMSKV_EWORKSPACE
    assert lib.mmshiftkv_select_workspace(ctypes.byref(_shape(Hkv=3)), ctypes.byref(p)) == 0   # Hq % Hkv


def test_gather_rejects(lib):
    s = _shape()
    st = bd.Strides(1024 * 64, 1024 * 64, 64)
    call = lambda k=FAKE, out=FAKE, dtype=1, c_max=64: lib.mmshiftkv_gather_kv(  # noqa: E731
        ctypes.byref(s), k, FAKE, dtype, ctypes.byref(st), ctypes.byref(st), FAKE, FAKE, c_max, out, FAKE, None)
    assert call(k=None) == bd.MMSKV_EINVAL
    assert call(out=ctypes.c_void_p(0x10004)) == bd.MMSKV_EINVAL
    assert call(dtype=3) == bd.MMSKV_EINVAL
    assert call(c_max=0) == bd.MMSKV_EINVAL
    # rows must be whole 16-byte vectors: d = 100 bf16 (200 bytes) is refused
    odd = _shape(d=100)
    assert lib.mmshiftkv_gather_kv(ctypes.byref(odd), FAKE, FAKE, 1, ctypes.byref(st), ctypes.byref(st), FAKE,
                                   FAKE, 64, FAKE, FAKE, None) == bd.MMSKV_EINVAL


def test_binding_refuses_host_tensors():
    import torch
    q = torch.zeros((1, 4, 16, 64))
    with pytest.raises(ValueError):
        bd.build_proxies(q, bd.SelectionConfig(), T=1024, Hkv=1)


def test_hidden_form_rejects(lib):
    """Host validation of the hidden-state proxy calls (Sec. 3.2.1 Eqs. 4-6)."""
    hs = bd.HShape(2, 300, 64)
    need = lib.mmshiftkv_hidden_stats_workspace(ctypes.byref(hs))
    assert need >= 2 * 2 * 64 * 16                  # two chunks of 256 tokens, (sum, sum sq) fp64
    assert lib.mmshiftkv_hidden_stats_workspace(ctypes.byref(bd.HShape(1, 10, 12))) == 0   # D % 8
    stats = lambda shape=hs, ddof=0, h=FAKE, dtype=1, sb=300 * 64, st=64, ws=FAKE, nbytes=need: \
        lib.mmshiftkv_hidden_stats(ctypes.byref(shape), ddof, h, dtype, sb, st, FAKE, ws, nbytes, None)  # noqa: E731
    assert stats(shape=bd.HShape(0, 300, 64)) == bd.MMSKV_EINVAL
    assert stats(shape=bd.HShape(1, 1, 64), ddof=1) == bd.MMSKV_EINVAL     # T - ddof < 1
    assert stats(ddof=2) == bd.MMSKV_EINVAL
    assert stats(h=None) == bd.MMSKV_EINVAL
    assert stats(dtype=5) == bd.MMSKV_EINVAL
    assert stats(st=63) == bd.MMSKV_EINVAL                                 # rows not 16-byte aligned
    assert stats(nbytes=need - 1) == bd.MMSKV_EWORKSPACE
    assert stats(ws=ctypes.c_void_p(0x10010)) == bd.MMSKV_EWORKSPACE
    prox = lambda prm, hp=FAKE: lib.mmshiftkv_hidden_proxies(ctypes.byref(hs), ctypes.byref(prm), FAKE, hp, None)  # noqa: E731
    assert prox(_params(gamma=-1.0)) == bd.MMSKV_EINVAL
    assert prox(_params(layer=-1)) == bd.MMSKV_EINVAL
    assert prox(_params(), hp=None) == bd.MMSKV_EINVAL
    proj = lambda P=512, Hq=4, d=64, out=FAKE, rope=(None, None): lib.mmshiftkv_project_proxies(  # noqa: E731
        ctypes.byref(hs), P, Hq, d, FAKE, FAKE, rope[0], rope[1], out, None)
    assert proj(d=96) == bd.MMSKV_EUNSUPPORTED
    assert proj(P=0) == bd.MMSKV_EINVAL
    assert proj(out=ctypes.c_void_p(0x10008)) == bd.MMSKV_EINVAL
    assert proj(rope=(FAKE, None)) == bd.MMSKV_EINVAL


def test_decode_check_rejects(lib):
    """Host validation of the decode-time check."""
    s = _shape(B=1, Hq=4, Hkv=1, T=1024, W=16, d=64)
    st = bd.Strides(1024 * 64, 1024 * 64, 64)
    need = lib.mmshiftkv_decode_workspace(ctypes.byref(s), 8)
    # (max, all, kept, pad) fp32 per (head, block of 512 keys, row padded to 32)
    assert need >= 1 * 1 * 32 * 16 and need % 256 == 0
    s2 = _shape(B=2, Hq=4, Hkv=2, T=3000, W=16, d=128)
    assert lib.mmshiftkv_decode_workspace(ctypes.byref(s2), 20) >= 2 * 2 * 6 * 64 * 16
    assert lib.mmshiftkv_decode_workspace(ctypes.byref(s), 0) == 0
    assert lib.mmshiftkv_decode_workspace(ctypes.byref(s), 65) == 0            # Gh * n_dec > 256
    call = lambda n_dec=8, q=FAKE, k=FAKE, dtype=1, c_max=64, ws=FAKE, nbytes=need, cov=FAKE, strides=st: \
        lib.mmshiftkv_decode_check(ctypes.byref(s), n_dec, q, k, dtype, ctypes.byref(strides), FAKE, FAKE, c_max,  # noqa: E731
                                   FAKE, FAKE, cov, FAKE, ws, nbytes, None)
    assert call(n_dec=0) == bd.MMSKV_EINVAL
    assert call(n_dec=65) == bd.MMSKV_EUNSUPPORTED
    assert call(c_max=0) == bd.MMSKV_EINVAL
    assert call(c_max=4096) == bd.MMSKV_EUNSUPPORTED
    assert call(q=None) == bd.MMSKV_EINVAL
    assert call(cov=None) == bd.MMSKV_EINVAL
    assert call(q=ctypes.c_void_p(0x10008)) == bd.MMSKV_EINVAL              # q rows not 16-byte aligned
    assert call(k=ctypes.c_void_p(0x10002)) == bd.MMSKV_EINVAL
    assert call(strides=bd.Strides(0, 0, 3)) == bd.MMSKV_EINVAL
    assert call(dtype=5) == bd.MMSKV_EINVAL
    assert call(nbytes=need - 1) == bd.MMSKV_EWORKSPACE
    assert call(ws=None) == bd.MMSKV_EWORKSPACE


def test_baseline_calls_reject(lib):
    """Host validation of the baseline-selector calls."""
    s = _shape(B=1, Hq=4, Hkv=1, T=1024, W=16, d=64)
    st = bd.Strides(16 * 64, 16 * 64, 64)
    rows = lambda n=8, q=FAKE, dtype=1, out=FAKE: lib.mmshiftkv_window_rows(  # noqa: E731
        ctypes.byref(s), n, q, dtype, ctypes.byref(st), out, FAKE, None)
    assert rows(n=0) == bd.MMSKV_EINVAL
    assert rows(n=17) == bd.MMSKV_EINVAL              # more rows than window queries
    assert rows(q=None) == bd.MMSKV_EINVAL
    assert rows(dtype=4) == bd.MMSKV_EINVAL
    assert rows(out=None) == bd.MMSKV_EINVAL
    shp = lambda kind=0, window=32, pool=5, sinks=4, mass=FAKE, score=FAKE: lib.mmshiftkv_shape_scores(  # noqa: E731
        ctypes.byref(s), kind, window, pool, sinks, mass, score, None)
    assert shp(kind=3) == bd.MMSKV_EINVAL
    assert shp(pool=4) == bd.MMSKV_EINVAL             # even pooling kernel
    assert shp(window=2000) == bd.MMSKV_EINVAL        # window longer than the prompt
    assert shp(mass=None) == bd.MMSKV_EINVAL          # SnapKV needs the masses
    assert shp(score=None) == bd.MMSKV_EINVAL
    assert shp(sinks=-1) == bd.MMSKV_EINVAL


def test_score_noalloc_refuses_problems_beyond_its_array(lib):
    """The allocation-free score call refuses, before touching the GPU, a
    problem whose workspace exceeds its fixed per-GPU scratch array."""
    shape = _shape(B=64, Hq=28, Hkv=4, T=16384, W=64, d=128)
    p = _params()
    assert lib.mmshiftkv_score_workspace(ctypes.byref(shape), ctypes.byref(p)) > bd.NOALLOC_SCRATCH_BYTES
    st = bd.Strides(4 * 16384 * 128, 16384 * 128, 128)
    rc = lib.mmshiftkv_score_noalloc(ctypes.byref(shape), ctypes.byref(p), FAKE, FAKE, FAKE, 1, ctypes.byref(st),
                                     FAKE, FAKE, FAKE, None)
    assert rc == bd.MMSKV_ESCRATCH
    assert lib.mmshiftkv_score_noalloc(ctypes.byref(_shape(d=96)), ctypes.byref(p), FAKE, FAKE, FAKE, 1,
                                       ctypes.byref(st), FAKE, FAKE, FAKE, None) == bd.MMSKV_EUNSUPPORTED
    text = open(HEADER).read()
    assert "MMSKV_NOALLOC_SCRATCH_BYTES ((size_t)32 << 20)" in text and bd.NOALLOC_SCRATCH_BYTES == 32 << 20
