"""SAKI (score-aware low-rank key indexing) retrieval-index path for MI355X.

The compute lives in libsaki.so (host float64 calibration + gfx950 HIP
kernels, C ABI in include/saki.h); ``paper_2608_03228_amd.saki`` is its thin
ctypes binding.  Build with ``python -m paper_2608_03228_amd.build``.
"""
from . import saki  # noqa: F401
from .saki import (  # noqa: F401
    saki_build_index, saki_calibrate, saki_index_bytes, saki_index_export, saki_recall,
    saki_recall_workspace_bytes, saki_score_topk, saki_score_topk_workspace_bytes,
    saki_status_string, saki_sym_eig, saki_version, saki_weight_svd_factors,
)
