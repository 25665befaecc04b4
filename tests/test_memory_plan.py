"""Host logic of the block memory strategies (paper_2501_08453_amd.memory.plan): which
layers are kept, recomputed or offloaded for a selective ratio (Sec. V-B; Sec. VI-D,
Tab. offload: ratios 0.2, 0.5, 1 and 0.8; the combination offloads a fixed share of 0.2 and
recomputes the rest)."""
import pytest

from paper_2501_08453_amd import memory as mem


@pytest.mark.parametrize("ratio,selected", [(0.2, 2), (0.5, 5), (0.8, 8), (1.0, 10), (0.0, 0)])
def test_selected_layers_at_the_papers_ratios(ratio, selected):
    for mode in ("recompute", "offload"):
        p = mem.plan(10, ratio, mode)
        assert len(p) == 10 and p.count(mode) == selected and p.count("keep") == 10 - selected
    c = mem.plan(10, ratio, "combination")
    assert c.count("offload") == min(2, selected)  # offloaded share fixed at 0.2
    assert c.count("recompute") == selected - min(2, selected)
    assert c.count("keep") == 10 - selected
    assert mem.plan(10, ratio, "keep") == ["keep"] * 10


def test_combination_at_ratio_02_is_pure_offload():
    """At ratio 0.2 the combination offloads everything it selects (the table's Offload and
    Combination columns agree there)."""
    assert mem.plan(10, 0.2, "combination") == mem.plan(10, 0.2, "offload")
    assert mem.plan(5, 0.2, "combination") == mem.plan(5, 0.2, "offload")


def test_placement_offloaded_spaced_then_recomputed():
    """Offloaded layers every other layer from layer 0 while they are at most half (one
    device set serves them in turn), the leading ones otherwise (two sets); recomputed
    layers take the earliest remaining positions."""
    assert mem.plan(10, 0.8, "combination") == ["offload", "recompute", "offload"] + ["recompute"] * 5 + \
        ["keep"] * 2
    assert mem.plan(4, 0.5, "offload") == ["offload", "keep", "offload", "keep"]
    assert mem.plan(10, 0.8, "offload") == ["offload"] * 8 + ["keep"] * 2
    assert mem.ring_size(mem.plan(10, 0.5, "offload")) == 1
    assert mem.ring_size(mem.plan(10, 0.8, "offload")) == 2
    assert mem.ring_size(mem.plan(10, 0.8, "recompute")) == 0


def test_device_sets():
    assert mem.device_sets(mem.plan(10, 0.0, "keep")) == 10
    assert mem.device_sets(mem.plan(10, 1.0, "recompute")) == 1
    assert mem.device_sets(mem.plan(10, 1.0, "offload")) == 2  # adjacent offloaded layers: two sets
    assert mem.device_sets(mem.plan(10, 0.2, "offload")) == 8 + 1  # spaced: one set for both
    assert mem.device_sets(mem.plan(10, 0.5, "offload")) == 5 + 1
    assert mem.device_sets(mem.plan(10, 0.8, "combination")) == 2 + 1 + 1


def test_bad_arguments():
    with pytest.raises(ValueError):
        mem.plan(4, 0.5, "swap")
    with pytest.raises(ValueError):
        mem.plan(0, 0.5, "offload")
    with pytest.raises(ValueError):
        mem.plan(4, 1.5, "offload")


def _check_schedule(strategies):
    """Replays forward_ops + backward_ops against a model of the device: one compute stream,
    one in-order copy stream; ("wait",) makes the compute stream wait for every copy issued
    so far. A load or a store reads or writes a ring slot when the copy stream reaches it,
    which is after all compute work queued before it. Checks that every offloaded layer's
    slot holds its own data from its forward until its store has run, that every loaded
    layer's data stays in its slot until its backward, and that nothing is read before the
    copy that brings it has completed."""
    slot = mem.ring_slots(strategies)
    owner = {}          # slot -> (layer, "fwd" | "load")
    unwaited = set()    # copies issued since the last wait: ("store"|"load", layer)
    stored, loaded = set(), set()
    backward_queued = set()
    for op in mem.forward_ops(strategies) + mem.backward_ops(strategies):
        kind = op[0]
        if kind == "wait":
            unwaited.clear()
            continue
        i = op[1]
        if kind in ("fwd", "recompute") and strategies[i] == "offload" and kind == "fwd":
            s = slot[i]
            if s in owner:  # overwriting the slot: its previous layer's store must be done
                prev = owner[s][0]
                assert prev in stored and ("store", prev) not in unwaited, (strategies, op)
            owner[s] = (i, "fwd")
        elif kind == "store":
            assert owner[slot[i]] == (i, "fwd"), (strategies, op)
            stored.add(i)
            unwaited.add(("store", i))
        elif kind == "load":
            assert i in stored, (strategies, op)  # the copy stream runs the store first
            s = slot[i]
            if s in owner and owner[s][0] != i:  # the slot's layer must have been backwarded
                assert owner[s][0] in backward_queued or owner[s][1] == "fwd" and \
                    owner[s][0] not in loaded and owner[s][0] in stored and \
                    ("store", owner[s][0]) not in unwaited, (strategies, op)
                if owner[s][1] == "load":
                    assert owner[s][0] in backward_queued, (strategies, op)
            owner[s] = (i, "load")
            loaded.add(i)
            unwaited.add(("load", i))
        elif kind == "bwd":
            if strategies[i] == "offload":
                assert owner[slot[i]] == (i, "load") and ("load", i) not in unwaited, (strategies, op)
            backward_queued.add(i)
    offloaded = {i for i, s in enumerate(strategies) if s == "offload"}
    assert loaded == offloaded and stored == offloaded
    assert backward_queued == set(range(len(strategies)))


def test_schedules_never_reuse_a_slot_too_early():
    import itertools
    for K in range(1, 8):
        for st in itertools.product(["keep", "recompute", "offload"], repeat=K):
            _check_schedule(list(st))
    for K in (10, 24):
        for mode in ("offload", "combination", "recompute", "keep"):
            for r in (0.2, 0.5, 0.8, 1.0):
                _check_schedule(mem.plan(K, r, mode))


def test_schedule_overlaps_loads_with_backwards():
    """Each offloaded layer's load is issued before another layer's backward and waited for
    only after it; each forward wait follows another forward queued after the store it
    covers, or precedes the forward that needs it."""
    for st in (mem.plan(10, 0.5, "offload"), mem.plan(10, 0.8, "offload"), mem.plan(10, 0.8, "combination")):
        ops = mem.backward_ops(st)
        for j in (i for i, s in enumerate(st) if s == "offload"):
            k = ops.index(("load", j))
            assert ops[k + 1][0] in ("bwd", "recompute") and ops[k + 1][1] > j
        fops = mem.forward_ops(st)
        for k, op in enumerate(fops):
            if op == ("wait",):
                last_store = max(m for m in range(k) if fops[m][0] == "store")
                assert any(fops[m][0] == "fwd" for m in range(last_store + 1, k)), (st, k)
