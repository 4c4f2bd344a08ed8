"""MI355X-native Gated DeltaNet tail replay (Tail-Replay, arXiv 2608.30310).

On a prefix-cache hit of a hybrid model, every GDN recurrent state is rebuilt
by replaying only the last r tokens of the matched prefix from a zero state
(paper Section 3, Eq. 2); the same chunked kernels then continue over the new
suffix and emit its outputs, and a decode-step kernel advances the state by
one generated token.  A whole linear-attention layer (projections,
convolution, norms and gates around the recurrence) can be replayed from the
cached hiddens as well.  The work runs in hand-written HIP kernels for gfx950
(the projections through hipBLASLt) behind the C ABI declared in
``include/gdn_tail_replay.h`` and ``include/gdn_la_block.h``; this package is
a thin binding of that library.
"""
from .binding import (GDNError, LIB_PATH, chunk_forward, decode_step, la_block_replay,
                      la_block_stage_names, la_block_workspace_size, load_library, noalloc_scratch_bytes,
                      replay_forward, replay_forward_stage_names, replay_forward_workspace_size,
                      replay_len, stage_names, tail_replay, tail_replay_noalloc, workspace_size)

__all__ = ["GDNError", "LIB_PATH", "chunk_forward", "decode_step", "la_block_replay",
           "la_block_stage_names", "la_block_workspace_size", "load_library", "noalloc_scratch_bytes",
           "replay_forward", "replay_forward_stage_names", "replay_forward_workspace_size", "replay_len",
           "stage_names", "tail_replay", "tail_replay_noalloc", "workspace_size"]
