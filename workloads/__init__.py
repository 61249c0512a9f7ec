"""Workload shapes and seeded synthetic inputs, shared by the HIP path and the oracle."""
from .configs import PAGE_TOKENS, LayerCfg, Workload, ALL, BY_NAME, TINY, DENSE_8B_B64, \
    DENSE_8B_B256, HYBRID_4L, MOE_B512, DENSE_8B_B256_TP8, SHARES, shrink
from . import gen
