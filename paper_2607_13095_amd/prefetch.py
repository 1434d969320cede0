"""Layerwise host-to-device KV prefetch ("Layerwise KVCache Prefetch").

A request whose cached prefix lives in pinned host memory (a lower cache tier)
needs, before each layer's attention, that layer's KV pages in HBM. SWA layers
need only their ring (O(W) pages) and FULL layers the whole prefix, so with a
copy stream running ahead of the compute stream the transfers of layer l+1..
overlap the attention of layer l, and the cost of reading the cache is hidden
as long as each copy is shorter than the compute it overlaps.

The schedule: device pool buffers are a ring of `depth` slots per layer kind
(FULL and SWA pools differ in size), so HBM holds at most `depth` layers of
each kind of loaded prefix at once. The i-th layer of a kind uses slot
i mod depth; its copy waits (an event) until the compute stream has finished
the layer of that kind `depth` places earlier, and the compute of a layer
waits for its copy (an event). Copies are plain asynchronous host-to-device
memcpys on streams of default priority; the attention is the library's
kernels.
"""

from __future__ import annotations

from dataclasses import dataclass
from typing import Callable, List, Sequence


@dataclass
class LayerPlan:
    """One layer: its kind ("full" / "swa"), the pinned host source tensors
    and, per slot, nothing more: the device slot tensors belong to the pool
    ring of the layer's kind."""
    kind: str
    host: Sequence  # pinned host tensors, copied element for element into the slot tensors


def slot_schedule(kinds: Sequence[str], depth: int):
    """For each layer l: (slot index within its kind's ring, index of the
    previous layer that used the same slot or -1). Pure host logic."""
    if depth < 1:
        raise ValueError("depth >= 1")
    seen = {}
    out = []
    for l, k in enumerate(kinds):
        n = seen.get(k, 0)
        seen[k] = n + 1
        slot = n % depth
        prev = -1
        # the previous layer of the same kind that used this slot
        cnt = 0
        for j in range(l - 1, -1, -1):
            if kinds[j] == k:
                cnt += 1
                if cnt == depth:
                    prev = j
                    break
        out.append((slot, prev))
    return out


class LayerwisePrefetch:
    """Runs compute(l, slot_tensors) for every layer with its host KV copied in
    ahead, one copy stream per layer kind (or, with overlap=False, copied then
    computed in order on the compute stream, for comparison).

    A copy is issued as soon as the layer that last used its slot has been
    enqueued on the compute stream, so the large FULL copies start while the
    SWA layers before them compute; per-kind streams keep a FULL copy that
    waits for its slot from holding up the small SWA copies behind it."""

    def __init__(self, rings: dict, depth: int):
        import torch

        self.rings = rings  # kind -> list of `depth` tuples of device tensors
        self.depth = int(depth)
        for k, ring in rings.items():
            if len(ring) != self.depth:
                raise ValueError(f"ring of kind {k} must have {depth} slots")
        self.streams = {k: torch.cuda.Stream() for k in rings}

    def run(self, plans: List[LayerPlan], compute: Callable, overlap: bool = True):
        import torch

        comp = torch.cuda.current_stream()
        kinds = [p.kind for p in plans]
        sched = slot_schedule(kinds, self.depth)
        n = len(plans)
        copied = [torch.cuda.Event() for _ in range(n)]
        done = [torch.cuda.Event() for _ in range(n)]
        # work enqueued on the compute stream before this run (e.g. a previous
        # run's attention, still reading the slots) finishes before any slot is
        # overwritten
        start = torch.cuda.Event()
        start.record(comp)

        def issue_copy(l, stream):
            slot, prev = sched[l]
            dst = self.rings[kinds[l]][slot]
            with torch.cuda.stream(stream):
                if stream is not comp:
                    # the slot's previous user in this run, or anything before it
                    stream.wait_event(done[prev] if prev >= 0 else start)
                for d, h in zip(dst, plans[l].host):
                    d.copy_(h, non_blocking=True)
                copied[l].record(stream)

        if not overlap:
            for l in range(n):
                issue_copy(l, comp)
                compute(l, self.rings[kinds[l]][sched[l][0]])
            return
        todo = {k: [l for l in range(n) if kinds[l] == k] for k in self.rings}
        ptr = {k: 0 for k in self.rings}

        def pump(enqueued):  # copies whose slot's previous user is on the compute stream
            for k, lst in todo.items():
                while ptr[k] < len(lst) and sched[lst[ptr[k]]][1] <= enqueued:
                    issue_copy(lst[ptr[k]], self.streams[k])
                    ptr[k] += 1

        pump(-1)
        for l in range(n):
            comp.wait_event(copied[l])
            compute(l, self.rings[kinds[l]][sched[l][0]])
            done[l].record(comp)
            pump(l)
