"""MM-ShiftKV prefill-stage KV scoring and selection on MI355X (gfx950).

The product is libmmshiftkv.so (C ABI: include/mmshiftkv.h), built from the
HIP sources in ``csrc/``; ``binding`` is its thin ctypes binding and
``workloads`` draws seeded synthetic inputs.  Importing this package does not
load the library; the first call does, and raises if it is not built.
"""
from .binding import (MMSKV_BF16, MMSKV_F32, MMSKV_MASS, MMSKV_VOTE, LayerOut, MMShiftKVError,  # noqa: F401
                      ScoreOut, Selected, SelectionConfig, build_proxies, decode_check, decode_workspace,
                      gather_kv, load_library,
                      score, score_lse, score_mass, score_workspace, select_layer, select_topk,
                      select_workspace, status_string)
