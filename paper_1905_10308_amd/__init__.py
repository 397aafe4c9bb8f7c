"""SCRAM hot path on MI355X: PatchMatch argmax + sparse window attention.

The computation lives in the HIP library ``_lib/libscram.so`` (C ABI:
``include/scram.h``); this package only marshals torch tensors into it.
Importing the package does not load the library; the first call does, and
raises if it is missing.
"""
from .binding import (  # noqa: F401
    CAUSAL,
    MAX_KAPPA,
    MAX_PREV,
    NOALLOC_MAX_QUERIES,
    NO_PROPAGATION,
    NO_RANDOM_SEARCH,
    ScramError,
    forward,
    lib,
    patchmatch,
    patchmatch_kappa,
    patchmatch_noalloc,
    patchmatch_workspace_bytes,
    snis_attend,
    sparse_attend,
    sparse_attend_backward,
    sparse_attend_backward_workspace_bytes,
    status_string,
)
