"""MI355X (gfx950) output layer of a beam-search decode step.

Projection onto the vocabulary, softmax fused with k-best extraction, beam
merge with the previous hypothesis scores, and batch compaction, after Hoang
et al., "Fast Neural Machine Translation Implementation" (WNMT 2018).  The
work runs in the HIP kernels of ``libkbest.so`` (C ABI in include/kbest.h);
this package only marshals arguments to it.
"""
from .binding import (KB_BF16, KB_F32, KB_MAX_K, KBestError, abi_version, argmax_step,  # noqa: F401
                      argmax_workspace_bytes, compact_batch, compact_beams, compact_workspace_bytes, gather_rows, kbest_step, kbest_step_unfused,
                      kbest_plan, kbest_step_noalloc, kbest_workspace_bytes, lib, merge_partials, shard_partials, shard_splits,
                      unfused_workspace_bytes, workspace)
