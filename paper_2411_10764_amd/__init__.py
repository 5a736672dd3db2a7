"""MI355X (gfx950) candidate-scoring library for ML2Tuner's configuration
explorer: validity filter, masked performance prediction, top-k selection
over a pool of candidate configurations and the second-level re-rank of the
selected ones, behind the C ABI of
include/ml2.h (libml2.so) and the thin ctypes binding in ``ml2``."""
from .ml2 import (  # noqa: F401
    Ensemble, Explorer, Ml2Error, Pipeline, ml2_filter_topk, ml2_free_ensemble, ml2_load_ensemble,
    ml2_rerank, ml2_rerank_workspace_bytes, ml2_score_perf, ml2_score_validity, ml2_topk_workspace_bytes,
)
