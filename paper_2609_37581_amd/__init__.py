"""TReVS two-stage visual-token pruning on MI355X (gfx950).

The HIP library libtrevs.so (C ABI in include/trevs.h) does all the work;
`trevs` is its ctypes binding."""

from .trevs import (Inllm, Prellm, TrevsError, inllm_prune, keep_count,  # noqa: F401
                    prellm_prune, topk_select)
