"""Multi-step, multi-layer decode loop over one batch of stacked prompts.

At every decode step each still-active question feeds one token, and every
layer runs one decode step over it (Sec. 4.2: one forward emits the next token
of every answer; stopped questions take no token).  DecodeLoop queues, for
steps 0..S-1 and layers 0..L-1, one fused decode-step call of the library
(rotation + append + attention + merge) on the current stream, with each
step's inputs and active mask already resident on the device (or, for the
dense-mask baseline, an append call and a dense decode call).  The queued
sequence can be captured once into a HIP graph and replayed: the kernels and
their arguments are those of the eager sequence, so a replay computes exactly
what the eager run computes, without the host-side cost of the launches.

Every computation runs in the library's kernels; this module only arranges
calls.  Segment lengths advance with each step's appends; reset() restores
the state before step 0 (a device copy, outside any graph).
"""
from __future__ import annotations

from typing import List, Optional, Sequence

import torch

from .session import DecodeBatch


class DecodeLoop:
    """S steps x L layers of fused decode-step calls on one DecodeBatch.

    q/k/v: per step, device tensors [Nt][Hq][D], [Nt][Hkv][D], [Nt][Hkv][D] of
    the batch dtype (every layer of a step is fed the same projections here);
    active: per step, device uint8 [Nt].  standard runs the per-question
    baseline, dense the dense-mask baseline (which has no fused step).
    """

    def __init__(self, batch: DecodeBatch, q: Sequence[torch.Tensor], k: Sequence[torch.Tensor],
                 v: Sequence[torch.Tensor], active: Sequence[torch.Tensor], layers: Optional[int] = None,
                 standard: bool = False, dense: bool = False):
        if not (len(q) == len(k) == len(v) == len(active)) or len(q) == 0:
            raise ValueError("one q, k, v and active tensor per step")
        self.db = batch
        self.q, self.k, self.v, self.active = list(q), list(k), list(v), list(active)
        self.steps = len(q)
        self.layers = batch.layers if layers is None else layers
        if not 1 <= self.layers <= batch.layers:
            raise ValueError("layers must be within the batch's emulated layers")
        if standard and dense:
            raise ValueError("standard and dense are two different baselines")
        self.standard = standard
        self.dense = dense
        self.seg0: List[torch.Tensor] = [batch.seg_len[l].clone() for l in range(self.layers)]
        self.graph: Optional[torch.cuda.CUDAGraph] = None

    def reset(self) -> None:
        """Segment lengths back to their values before step 0."""
        for l in range(self.layers):
            self.db.seg_len[l].copy_(self.seg0[l])

    def _set_active(self, t: int) -> None:
        ptr = self.active[t].data_ptr()
        for bt in self.db.batches:
            bt.active = ptr

    def enqueue(self, steps: Optional[int] = None) -> None:
        """Queue the calls of steps 0..steps-1 on the current stream."""
        for t in range(self.steps if steps is None else steps):
            self._set_active(t)
            for l in range(self.layers):
                if self.dense:
                    self.db.append(l, self.q[t], self.k[t], self.v[t])
                    self.db.decode(l, dense=True)
                else:
                    self.db.decode_step(l, self.q[t], self.k[t], self.v[t], standard=self.standard,
                                        write_q_rot=False)

    def capture(self) -> None:
        """Record the whole loop into a HIP graph (the state is reset first and
        after: capture itself runs nothing)."""
        self.reset()
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            self.enqueue()
        torch.cuda.synchronize()
        self.graph = g
        self.reset()

    def replay(self) -> None:
        if self.graph is None:
            raise RuntimeError("capture() first")
        self.graph.replay()
