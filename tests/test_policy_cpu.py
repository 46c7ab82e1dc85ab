"""The library's host-tier slot policy against the oracle's, on the CPU.

Bit-exact comparison of every copy list and every slot list on seeded random
traces shaped like a decode loop: per token, each layer's set is staged one
token ahead (the prediction) or on demand (own router), then used in order.
Error behaviour is compared too: a set that cannot fit fails in both.
"""

import numpy as np
import pytest

from oracle import slots as o_slots
from paper_2609_18063_amd import binding as B


def _decode_trace(rng, n_layers, n_ids, k, tokens, overlap):
    """Yields ("stage" | "use", layer, set) and ("release", layer, None) in the
    order a decode loop issues them: layer 0 and token 0 stage on demand,
    after the host has waited for the router (so every earlier set in use is
    released); the prediction for layer n + 1 at token t + 1 is staged one
    layer later, after the host has waited for head n (which releases the sets
    in use up to layer n of token t).  A new set keeps about `overlap` of the
    previous token's set at that layer."""
    prev = {}

    def draw(layer):
        old = prev.get(layer)
        if old is not None and rng.random() < 0.9:
            keep = [e for e in old if rng.random() < overlap]
            rest = [e for e in rng.permutation(n_ids).tolist() if e not in keep]
            s = (keep + rest)[:k]
            rng.shuffle(s)
        else:
            s = rng.choice(n_ids, size=k, replace=False).tolist()
        prev[layer] = s
        return [int(e) for e in s]

    in_use = []          # layers of used sets, in use order

    def release_through(count):
        for _ in range(count):
            yield ("release", in_use.pop(0), None)

    staged = {}
    queued = None        # (t + 1, n + 1, set) predicted by head n, staged one layer later
    for t in range(tokens):
        for n in range(n_layers):
            if t == 0 or n == 0:
                s = draw(n)
                yield from release_through(len(in_use))
                yield ("stage", n, s)
            else:
                s = staged.pop((t, n))
            yield ("use", n, s)
            in_use.append(n)
            if queued is not None:       # head n - 1 finished: sets up to layer n - 1 are done
                yield from release_through(len(in_use) - 1)
                tq, nq, sq = queued
                staged[(tq, nq)] = sq
                yield ("stage", nq, sq)
                queued = None
            if n + 1 < n_layers:
                queued = (t + 1, n + 1, draw(n + 1))
        if queued is not None:
            yield from release_through(len(in_use) - 1)
            tq, nq, sq = queued
            staged[(tq, nq)] = sq
            yield ("stage", nq, sq)
            queued = None


@pytest.mark.parametrize("seed,n_layers,n_ids,k,n_slots,overlap", [
    (0, 24, 64, 4, 12, 0.25),
    (1, 6, 64, 4, 12, 0.0),
    (2, 5, 16, 4, 8, 0.5),
    (3, 3, 9, 3, 6, 0.9),
    (4, 4, 256, 8, 24, 0.25),
])
def test_policy_matches_oracle(seed, n_layers, n_ids, k, n_slots, overlap):
    rng = np.random.default_rng(seed)
    ref = o_slots.SlotPolicy(n_layers, n_ids, n_slots)
    lib = B.SlotPolicy(n_layers, n_ids, n_slots)
    n_copies = 0
    steps = 0
    for op, layer, s in _decode_trace(rng, n_layers, n_ids, k, 40, overlap):
        if op == "stage":
            want = ref.stage(layer, s)
            got = lib.stage(layer, s)
            assert got == [tuple(c) for c in want], (steps, layer, s)
            n_copies += len(got)
        elif op == "release":
            ref.release(layer)
            lib.release(layer)
        else:
            assert lib.use(layer, s) == ref.use(layer, s), (steps, layer, s)
        steps += 1
        if steps % 97 == 0:
            for e in range(n_ids):
                assert lib.lookup(layer, e) == ref.table.lookup(layer, e)
    assert n_copies > 0
    lib.close()


def test_policy_rejects_like_oracle():
    ref = o_slots.SlotPolicy(1, 10, 4)
    lib = B.SlotPolicy(1, 10, 4)
    for p in (ref, lib):
        p.stage(0, [0, 1, 2])
    # the pending set pins three slots: a second set of three new experts cannot fit
    with pytest.raises(RuntimeError):
        ref.stage(0, [3, 4, 5])
    with pytest.raises(B.MoeError) as err:
        lib.stage(0, [3, 4, 5])
    assert err.value.code == B.MOE_ENOMEM
    # both left their state unchanged: the first set is still usable
    assert lib.use(0, [0, 1, 2]) == ref.use(0, [0, 1, 2]) == [0, 1, 2]
    # in use, it stays pinned until released
    with pytest.raises(B.MoeError):
        lib.stage(0, [3, 4, 5])
    lib.release(0)
    ref.release(0)
    assert lib.stage(0, [3, 4, 5]) == ref.stage(0, [3, 4, 5])
    lib.use(0, [3, 4, 5])
    # using a set that is not the oldest staged one is an error
    with pytest.raises(B.MoeError):
        lib.use(0, [0, 1, 2])
    with pytest.raises(B.MoeError):
        lib.release(1)
    lib.release(0)
    lib.stage(0, [7, 8])
    with pytest.raises(B.MoeError):
        lib.use(0, [8, 7])
    # invalid sets: duplicates, out-of-range ids
    with pytest.raises(B.MoeError):
        lib.stage(0, [1, 1])
    with pytest.raises(B.MoeError):
        lib.stage(0, [10])
    lib.close()


def test_policy_reuse_costs_nothing():
    lib = B.SlotPolicy(2, 32, 8)
    assert len(lib.stage(1, [3, 4, 5, 6])) == 4
    lib.use(1, [3, 4, 5, 6])
    assert lib.stage(1, [6, 5, 4, 3]) == []
    assert lib.use(1, [6, 5, 4, 3]) == [3, 2, 1, 0]
    lib.release(1)
    lib.release(1)
    lib.close()
