"""Host pacing for the chunk walks.

The walks enqueue every kernel and copy asynchronously, so without a bound
the host runs a whole step (or several) ahead of the device.  A copy
enqueued that early waits on a compute event hundreds of milliseconds away.
With the next step's offload copies queued behind such waits during the
current step's backward, the 128K-token layer walk on one MI355X ran 4-6%
slower: the attention and GEMM kernels and the host-to-device copies all
took longer, with no idle time on the compute stream.  With the host held
to a few chunk boundaries ahead, every step ran as fast as a step started
from an idle device.

HostPacer records an event on the compute stream at every chunk boundary
and, once more than ``ahead`` of them are outstanding, waits on the host for
the oldest.  One pacer lives as long as its walk, so the bound also holds
across step boundaries.
"""
from __future__ import annotations

from collections import deque

import torch


class HostPacer:
    def __init__(self, ahead: int = 2):
        if ahead < 0:
            raise ValueError("ahead must be >= 0 (0 disables pacing)")
        self.ahead = ahead
        self._pending = deque()

    def boundary(self, stream) -> None:
        if self.ahead == 0:
            return
        ev = torch.cuda.Event()
        ev.record(stream)
        self._pending.append(ev)
        while len(self._pending) > self.ahead:
            self._pending.popleft().synchronize()

    def drain(self) -> None:
        while self._pending:
            self._pending.popleft().synchronize()
