"""mmshiftkv_score_noalloc against mmshiftkv_score (GPU): the allocation-free
entry point runs the same kernels on the library's per-GPU scratch array, so
its group masses, masses and anchors must equal the workspace call's bit for
bit -- on two calls in a row, the second on a smaller problem (the array then
holds the first call's contents), and on a problem beyond the array, which is
refused before anything is enqueued."""
import numpy as np
import pytest
import torch

from paper_2607_22586_amd import binding as bd
from paper_2607_22586_amd import workloads as wl

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    bd.load_library()


def _outs(B, Hkv, G, T):
    return bd.ScoreOut(torch.full((B, Hkv, G, T), -1.0, device=DEV), torch.full((B, Hkv, T), -1.0, device=DEV),
                       torch.full((B, Hkv, T), -1.0, device=DEV))


@pytest.mark.parametrize("first,second", [
    (("qwen7b_16k_b4", None), ("qwen7b_4k", None)),
    (("custom", (2, 8, 2, 5000, 8, 128)), ("custom", (1, 4, 1, 777, 5, 64)))])
def test_noalloc_equals_workspace_call(first, second):
    for name, dims in (first, second):
        print("case noalloc", name, dims, flush=True)
        if name == "custom":
            x = wl.custom_layer(*dims, seed=sum(dims))
            cfg = bd.SelectionConfig(P=64, G=4, seed=3)
        else:
            x = wl.make_layer(name, 1)
            cfg = bd.SelectionConfig(seed=wl.WORKLOADS[name].wid, layer=1)
        q, k = x["q_win"].to(DEV), x["k"].to(DEV)
        B, Hkv, T, d = k.shape
        W = q.shape[2]
        prox, ql = bd.build_proxies(q, cfg, T, Hkv)
        need = bd.score_workspace(B, q.shape[1], Hkv, T, W, d, cfg)
        assert need <= bd.NOALLOC_SCRATCH_BYTES
        ref = bd.score(prox, ql, k, cfg, W)
        got = bd.score_noalloc(prox, ql, k, cfg, _outs(B, Hkv, cfg.G, T), W)
        torch.cuda.synchronize()
        for a, b in ((ref.group_mass, got.group_mass), (ref.mass, got.mass), (ref.anchor, got.anchor)):
            assert torch.equal(a, b)
        np.testing.assert_allclose(got.mass.double().sum(-1).cpu().numpy(), cfg.P * q.shape[1] // Hkv, rtol=1e-3)


def test_noalloc_refuses_problems_beyond_its_array():
    # B = 64 rows of the T = 16384 shape need ~240 MiB of score workspace
    shape = bd.Shape(64, 28, 4, 16384, 64, 128)
    cfg = bd.SelectionConfig()
    prm = cfg.c_params()
    lib = bd.load_library()
    import ctypes
    assert lib.mmshiftkv_score_workspace(ctypes.byref(shape), ctypes.byref(prm)) > bd.NOALLOC_SCRATCH_BYTES
    fake = ctypes.c_void_p(0x10000)
    st = bd.Strides(4 * 16384 * 128, 16384 * 128, 128)
    rc = lib.mmshiftkv_score_noalloc(ctypes.byref(shape), ctypes.byref(prm), fake, fake, fake, 1, ctypes.byref(st),
                                     fake, fake, fake, None)
    assert rc == bd.MMSKV_ESCRATCH
