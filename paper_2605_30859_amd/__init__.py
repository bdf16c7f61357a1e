"""MI355X (gfx950) rollout hot path of DARTS: paged-KV batched decode of m
redundant trajectories per prompt, fused Gumbel-max sampling with token
log-prob and entropy, and distribution-aware selection with early stopping
and KV page reclaim -- all in hand-written HIP kernels behind a C ABI
(include/darts.h).  This package is a thin ctypes binding over that library.
"""
from .binding import (DARTS_OK, DARTS_EINVAL, DARTS_ENOMEM, DARTS_ESTATE, DARTS_EHIP,
                      DARTS_F32, DARTS_BF16, FLAG_NO_ABORT, FLAG_PERMUTE_PAGES, FLAG_TIMING,
                      FLAG_SHARED_PREFIX,
                      DartsError, load_library, lib_path, Rollout)

__all__ = ["DARTS_OK", "DARTS_EINVAL", "DARTS_ENOMEM", "DARTS_ESTATE", "DARTS_EHIP",
           "DARTS_F32", "DARTS_BF16", "FLAG_NO_ABORT", "FLAG_PERMUTE_PAGES", "FLAG_TIMING",
           "FLAG_SHARED_PREFIX",
           "DartsError", "load_library", "lib_path", "Rollout"]
