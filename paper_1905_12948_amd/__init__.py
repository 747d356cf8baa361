"""MI355X (gfx950) implementation of the data-parallel hot path of Global
Momentum Compression: the K workers' compressed updates (global momentum,
error feedback, top-s or RBGS, residual), the server's aggregation and the
apply step, as HIP kernels behind the C ABI in include/gmc.h."""
from .gmc import (Gmc, GmcError, load, count, COMPRESSORS, EXPORTS, STAGES, MAX_WORKERS,
                  GMC_OPT_FORCE_FULL_SELECT, GMC_OPT_CAND_MARGIN, GMC_OPT_CAND_CAP_MULT,
                  GMC_OPT_PROFILE, GMC_OPT_SAMPLE_STRATUM,
                  GMC_OPT_SPARSE_MOMENTUM, GMC_OPT_CHANGE_LIST)

__all__ = ["Gmc", "GmcError", "load", "count", "COMPRESSORS", "EXPORTS", "STAGES", "MAX_WORKERS",
           "GMC_OPT_FORCE_FULL_SELECT", "GMC_OPT_CAND_MARGIN", "GMC_OPT_CAND_CAP_MULT",
           "GMC_OPT_PROFILE", "GMC_OPT_SAMPLE_STRATUM", "GMC_OPT_SPARSE_MOMENTUM",
           "GMC_OPT_CHANGE_LIST"]
