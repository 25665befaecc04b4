"""Selective recomputation and activation offloading for stacked parallel blocks.

The paper trades the activation memory of long video sequences against time with a
combination of recomputation and offloading to host memory (Sec. V-B): a tuned share of
the layers' saved activations, the "selective ratio", is recomputed before the backward or
swapped to host memory on a side stream and back; with both combined, the offloaded share
is fixed at 0.2, the most the host link overlaps with computation, and the rest of the
ratio is recomputed (Sec. VI-D, Tab. offload). For the attention of a parallel block the
saved activations are what each branch's backward needs besides q, k, v: its O and LSE
(the joint, spatial and temporal branches; the branch sum needs nothing).

`plan` assigns every layer keep / recompute / offload; `BlockStack` runs the block's
forward through all layers and the backward in reverse under such a plan, with the
library's kernels and its offload engine (vc_offload_*). It only schedules calls: every
step of the computation runs in the library.

Device memory for saved outputs: one set per kept layer, one scratch set shared by the
recomputed layers, and one set (two when some offloaded layers are adjacent) that the
offloaded ones use in turn. An offloaded layer's set is stored to pinned host memory right
after its forward (on the engine's copy stream, overlapping the next layers' forwards) and
loaded back before its backward (overlapping the backward of a later layer).
"""
from __future__ import annotations

MODES = ("keep", "recompute", "offload", "combination")
OFFLOAD_SHARE = 0.2  # offloaded share in the combination (Sec. VI-D)


def _count(share: float, layers: int) -> int:
    return min(layers, max(0, int(share * layers + 0.5)))


def plan(layers: int, ratio: float, mode: str, offload_share: float = OFFLOAD_SHARE) -> list:
    """Strategy per layer ("keep", "recompute" or "offload"), in forward order.

    recompute / offload: round(ratio * layers) layers take that strategy;
    combination: round(offload_share * layers) of them (at most the selected count) are
    offloaded and the rest of the selected ones recomputed; keep: none (ratio ignored).
    Offloaded layers come first: every other layer from layer 0 when they are at most half
    of the layers (then one device set holds them in turn: each store overlaps the next
    layer's forward and each load the backward of the layer after it), else the leading
    ones (two sets in turn). Recomputed layers fill the earliest remaining positions."""
    if mode not in MODES:
        raise ValueError("mode must be one of %s" % (MODES,))
    if layers < 1 or not 0.0 <= ratio <= 1.0:
        raise ValueError("need layers >= 1 and 0 <= ratio <= 1")
    selected = 0 if mode == "keep" else _count(ratio, layers)
    if mode == "recompute":
        n_off, n_rec = 0, selected
    elif mode == "offload":
        n_off, n_rec = selected, 0
    elif mode == "combination":
        n_off = min(selected, _count(offload_share, layers))
        n_rec = selected - n_off
    else:
        n_off = n_rec = 0
    st = ["keep"] * layers
    for i in (range(0, 2 * n_off, 2) if 2 * n_off <= layers else range(n_off)):
        st[i] = "offload"
    rest = [i for i in range(layers) if st[i] == "keep"]
    for i in rest[:n_rec]:
        st[i] = "recompute"
    return st


def ring_size(strategies: list) -> int:
    """Device sets the offloaded layers take in turn: one if no two of them are adjacent
    (a store then has a whole other layer's forward to finish before the set is reused),
    else two."""
    off = [i for i, s in enumerate(strategies) if s == "offload"]
    if not off:
        return 0
    return 2 if any(b == a + 1 for a, b in zip(off, off[1:])) else 1


def device_sets(strategies: list) -> int:
    """Saved-output sets held on the device under a plan."""
    keep = strategies.count("keep")
    rec = 1 if "recompute" in strategies else 0
    return keep + rec + ring_size(strategies)


def ring_slots(strategies: list) -> dict:
    """Device set (ring slot) of each offloaded layer: the ring_size slots in turn."""
    off = [i for i, s in enumerate(strategies) if s == "offload"]
    ring = ring_size(strategies)
    return {i: j % ring for j, i in enumerate(off)}


def forward_ops(strategies: list) -> list:
    """Forward schedule: ("fwd", i) for every layer, ("store", i) after an offloaded
    layer's forward, and ("wait",) (the stream waits for every copy issued so far) where an
    offloaded forward is about to reuse a set whose store may still run: with one set,
    right before that forward (the store overlapped the layers in between); with two,
    right after the previous offloaded forward (its predecessor's store overlapped it)."""
    ring = ring_size(strategies)
    ops, first = [], True
    for i, s in enumerate(strategies):
        if s == "offload" and ring == 1 and not first:
            ops.append(("wait",))
        ops.append(("fwd", i))
        if s == "offload":
            if ring == 2 and not first:
                ops.append(("wait",))
            ops.append(("store", i))
            first = False
    return ops


def backward_ops(strategies: list) -> list:
    """Backward schedule, layers in reverse: ("load", j) prefetches the next offloaded layer
    in backward order into its ring slot as soon as that slot holds no layer whose backward
    is not queued yet (the load is ordered after the work queued before it, and issued
    before the current layer's backward so that the two overlap); ("wait",) after that
    backward makes the stream wait for the load; ("recompute", i) re-runs a recomputed
    layer's forwards before ("bwd", i)."""
    slot = ring_slots(strategies)
    pending = sorted(slot, reverse=True)
    loaded, ops = set(), []
    if pending and pending[0] == len(strategies) - 1:  # the first layer back is offloaded
        j = pending.pop(0)
        loaded.add(j)
        ops += [("load", j), ("wait",)]
    for i in reversed(range(len(strategies))):
        prefetch = None
        if pending and pending[0] < i and all(slot[x] != slot[pending[0]] for x in loaded):
            prefetch = pending.pop(0)
            loaded.add(prefetch)
            ops.append(("load", prefetch))
        if strategies[i] == "recompute":
            ops.append(("recompute", i))
        ops.append(("bwd", i))
        loaded.discard(i)
        if prefetch is not None:
            ops.append(("wait",))
    return ops


class BlockStack:
    """Layers of the parallel block's attention (joint, spatial and temporal branches, the
    sum fused into the temporal forward) over per-layer inputs, run under a plan.

    inputs: per layer (q, k, v) bf16 [B, N, H, D] tensors (layers may share them).
    outs: per layer block-output buffer (may be shared); grads: per layer three
    (dq, dk, dv) triples, one per branch (may be shared)."""

    def __init__(self, desc, inputs, strategies, outs, grads, text_len=None, key_mask=None, offload=None):
        import torch
        import paper_2501_08453_amd as vc
        if len(inputs) != len(strategies) or len(outs) != len(strategies) or len(grads) != len(strategies):
            raise ValueError("one input, output, gradient set and strategy per layer")
        self.vc, self.desc = vc, desc
        self.inputs, self.strategies, self.outs, self.grads = inputs, list(strategies), outs, grads
        self.tl, self.km = text_len, key_mask
        q = inputs[0][0]
        B, N, H, D = q.shape
        dev = q.device
        self.fws = vc.fwd_workspace(desc, dev)
        self.ws_j = vc.workspace(desc, dev)
        self.ws_s = vc.spatial_workspace(desc, dev)

        def new_set():  # O, LSE of the joint, spatial and temporal branches
            s = []
            for _ in range(3):
                s += [torch.empty_like(q), torch.empty((B, H, N), dtype=torch.float32, device=dev)]
            return s

        slots = ring_slots(self.strategies)
        self.off_layers = sorted(slots)
        ring = ring_size(self.strategies)
        self.ring = [new_set() for _ in range(ring)]
        self.scratch = new_set() if "recompute" in self.strategies else None
        self.sets = []
        for i, s in enumerate(self.strategies):
            if s == "keep":
                self.sets.append(new_set())
            elif s == "recompute":
                self.sets.append(self.scratch)
            else:
                self.sets.append(self.ring[slots[i]])
        self.host = {i: [torch.empty(t.shape, dtype=t.dtype, pin_memory=True) for t in self.ring[0]]
                     for i in self.off_layers}
        self.set_bytes = sum(t.numel() * t.element_size() for t in (self.ring[0] if ring else self.sets[0]))
        self.own_offload = offload is None and bool(self.off_layers)
        self.off = vc.Offload() if self.own_offload else offload

    # -- one layer ------------------------------------------------------------------
    def _forward(self, i, stream):
        vc, d = self.vc, self.desc
        q, k, v = self.inputs[i]
        o_j, l_j, o_s, l_s, o_t, l_t = self.sets[i]
        sh = stream.cuda_stream
        vc.vc_jointattn_fwd(d, q, k, v, self.tl, self.km, o_j, l_j, self.fws, self.fws.numel(), sh)
        vc.vc_spatialattn_fwd(d, q, k, v, self.tl, self.km, o_s, l_s, self.fws, self.fws.numel(), sh)
        vc.vc_temporalattn_fwd_sum(d, q, k, v, self.km, o_j, o_s, o_t, l_t, self.outs[i], sh)

    def _backward(self, i, dout, stream):
        vc, d = self.vc, self.desc
        q, k, v = self.inputs[i]
        o_j, l_j, o_s, l_s, o_t, l_t = self.sets[i]
        g = self.grads[i]
        sh = stream.cuda_stream
        vc.vc_jointattn_bwd(d, q, k, v, o_j, l_j, dout, self.tl, self.km, *g[0], self.ws_j, self.ws_j.numel(), sh)
        vc.vc_spatialattn_bwd(d, q, k, v, o_s, l_s, dout, self.tl, self.km, *g[1], self.ws_s, self.ws_s.numel(), sh)
        vc.vc_temporalattn_bwd(d, q, k, v, o_t, l_t, dout, self.km, *g[2], None, 0, sh)

    def _store(self, i, stream):
        for h, t in zip(self.host[i], self.sets[i]):
            self.off.store(h, t, stream)

    def _load(self, i, stream):
        for h, t in zip(self.host[i], self.sets[i]):
            self.off.load(t, h, stream)

    # -- whole stack ----------------------------------------------------------------
    def _run(self, ops, douts, stream):
        for op in ops:
            kind = op[0]
            if kind == "fwd" or kind == "recompute":
                self._forward(op[1], stream)
            elif kind == "bwd":
                self._backward(op[1], douts[op[1]], stream)
            elif kind == "store":
                self._store(op[1], stream)
            elif kind == "load":
                self._load(op[1], stream)
            else:
                self.off.wait(stream)

    def forward(self, stream=None):
        """Forward through every layer (forward_ops); offloaded layers' sets leave for host
        memory."""
        import torch
        self._run(forward_ops(self.strategies), None, torch.cuda.current_stream() if stream is None else stream)

    def backward(self, douts, stream=None):
        """Backward in reverse layer order (backward_ops; douts: per layer upstream gradient).
        Recomputed layers run their forwards again first; offloaded layers are loaded back
        while an earlier layer of the backward runs."""
        import torch
        self._run(backward_ops(self.strategies), douts, torch.cuda.current_stream() if stream is None else stream)

    def close(self):
        if self.own_offload and self.off is not None:
            self.off.close()
        self.off = None
