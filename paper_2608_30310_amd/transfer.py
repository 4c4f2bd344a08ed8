"""Host-to-device transfer beside the tail replay (paper Section 3, "Replay
efficiency"; Table 2, H2D-SER against H2D-OVL).

On a cache hit the full-attention KV of the matched prefix moves from host
memory to the device while the linear-attention layers replay their tails;
the transfer only has to be complete before the query forward over the new
suffix.  This module orders that work on torch streams: the copy on a second
stream, the replay and the suffix forward on the compute stream, and one
stream wait between the copy and the suffix forward.  It only enqueues: the
copy is a device DMA from pinned host memory (``copy_src`` must be pinned for
the copy to be asynchronous), the replay and the forward are the caller's
calls into the library, and nothing here synchronises the host.
"""
from __future__ import annotations

from typing import Callable, Optional

import torch

__all__ = ["rebuild_serial", "rebuild_overlapped"]


def rebuild_serial(copy_src: torch.Tensor, copy_dst: torch.Tensor, replay: Callable[[], None],
                   forward: Callable[[], None], stream: Optional[torch.cuda.Stream] = None) -> None:
    """H2D-SER: the copy, then the replay, then the suffix forward, all on
    ``stream`` (default: the current stream)."""
    main = stream or torch.cuda.current_stream()
    with torch.cuda.stream(main):
        copy_dst.copy_(copy_src, non_blocking=True)
        replay()
        forward()


def rebuild_overlapped(copy_src: torch.Tensor, copy_dst: torch.Tensor, replay: Callable[[], None],
                       forward: Callable[[], None], copy_stream: torch.cuda.Stream,
                       stream: Optional[torch.cuda.Stream] = None) -> None:
    """H2D-OVL: the copy on ``copy_stream`` beside the replay on ``stream``
    (default: the current stream); the suffix forward waits for the copy.

    The copy starts only after the work already queued on ``stream`` (it may
    overwrite a buffer that earlier work reads), and work queued on ``stream``
    after this call is ordered after the copy as well.  ``copy_dst`` must not be
    read by ``replay``; both streams must keep the default priority."""
    main = stream or torch.cuda.current_stream()
    copy_stream.wait_stream(main)
    with torch.cuda.stream(copy_stream):
        copy_dst.copy_(copy_src, non_blocking=True)
    with torch.cuda.stream(main):
        replay()
        main.wait_stream(copy_stream)
        forward()
    # the copy stream used copy_dst; keep the allocator from reusing it early
    copy_dst.record_stream(copy_stream)
