"""Oracle: slot table and the host-tier slot policy (TEST INFRASTRUCTURE ONLY).

§3.1 (Executor paths, *staged*): routing indices are mapped through a slot
table and never leave the device; the staged path keeps a fixed set of slots
per layer and rewrites only the slots whose expert changed.  §3.2
(Motivation) stages layer N+1's experts from head N's prediction one token
ahead, so the copy for token t+1 overlaps the compute of token t.

Readings (the paper is silent on the policy):

* A layer has ``n_slots`` slots, a queue of staged-but-unused sets and a
  queue of sets in use.  A layer whose routing is not predicted (its own
  router) stages its set and uses it at once (a synchronous fetch).  Staging
  a set walks it in routing order; an expert already resident costs
  nothing, a missing one takes the lowest free slot, else the slot with the
  oldest last use among the slots that are not pinned, ties to the lowest
  slot id.  Pinned: the slots holding any set still queued for the layer
  (staged earlier, not yet consumed), any set in use (consumed, and the
  layer has not finished with it), and the members of the set being staged.
* Using a set moves it from the staged queue to the in-use queue; releasing
  the layer's oldest set in use (its layer finished) unpins it.
* "Last use" is a counter that advances on every stage-copy and every use.
* Copies are issued in routing order; each is ``(expert, slot)``.
"""


class SlotTable:
    """Plain map (layer, expert) -> slot with the inverse map per layer."""

    def __init__(self, n_layers, n_experts, n_slots):
        self.n_layers, self.n_experts, self.n_slots = n_layers, n_experts, n_slots
        self.slot_of = [[-1] * n_experts for _ in range(n_layers)]
        self.expert_in = [[-1] * n_slots for _ in range(n_layers)]

    def bind(self, layer, expert, slot):
        old = self.expert_in[layer][slot]
        if old >= 0:
            self.slot_of[layer][old] = -1
        prev = self.slot_of[layer][expert]
        if prev >= 0:
            self.expert_in[layer][prev] = -1
        self.slot_of[layer][expert] = slot
        self.expert_in[layer][slot] = expert

    def unbind(self, layer, expert):
        s = self.slot_of[layer][expert]
        if s >= 0:
            self.expert_in[layer][s] = -1
        self.slot_of[layer][expert] = -1

    def lookup(self, layer, expert):
        return self.slot_of[layer][expert]


class SlotPolicy:
    """The host-tier policy above, on top of a :class:`SlotTable`."""

    def __init__(self, n_layers, n_experts, n_slots):
        self.table = SlotTable(n_layers, n_experts, n_slots)
        self.last_use = [[-1] * n_slots for _ in range(n_layers)]
        self.pending = [[] for _ in range(n_layers)]   # FIFO of staged sets
        self.in_use = [[] for _ in range(n_layers)]    # FIFO of sets in use
        self.clock = 0

    def _tick(self):
        self.clock += 1
        return self.clock

    def stage(self, layer, experts):
        """Make ``experts`` resident in ``layer`` for a later use; return the
        copy list ``[(expert, slot), ...]``."""
        t = self.table
        keep = set(int(e) for e in experts)
        for pend in self.pending[layer] + self.in_use[layer]:
            keep |= set(pend)
        pinned = {t.lookup(layer, e) for e in keep if t.lookup(layer, e) >= 0}
        misses = [e for e in experts if t.lookup(layer, int(e)) < 0]
        usable = [s for s in range(t.n_slots) if s not in pinned]
        if len(misses) > len(usable):      # refuse before changing anything
            raise RuntimeError("no evictable slot: too few slots")
        copies = []
        for e in experts:
            e = int(e)
            if t.lookup(layer, e) >= 0:
                continue
            free = [s for s in range(t.n_slots) if t.expert_in[layer][s] < 0]
            if free:
                slot = free[0]
            else:
                cand = [s for s in range(t.n_slots) if s not in pinned]
                if not cand:
                    raise RuntimeError("no evictable slot: too few slots")
                slot = min(cand, key=lambda s: (self.last_use[layer][s], s))
            t.bind(layer, e, slot)
            pinned.add(slot)
            self.last_use[layer][slot] = self._tick()
            copies.append((e, slot))
        self.pending[layer].append([int(e) for e in experts])
        return copies

    def use(self, layer, experts):
        """Consume the oldest staged set of ``layer``, which must equal
        ``experts``; every member must be resident.  Returns the slots."""
        t = self.table
        if not self.pending[layer] or self.pending[layer][0] != [int(e) for e in experts]:
            raise RuntimeError("layer %d uses a set that was not staged" % layer)
        self.in_use[layer].append(self.pending[layer].pop(0))
        slots = []
        for e in experts:
            s = t.lookup(layer, int(e))
            if s < 0:
                raise RuntimeError("expert %d not resident in layer %d" % (e, layer))
            self.last_use[layer][s] = self._tick()
            slots.append(s)
        return slots

    def release(self, layer):
        """The layer finished with its oldest set in use: unpin it."""
        if not self.in_use[layer]:
            raise RuntimeError("layer %d has no set in use" % layer)
        self.in_use[layer].pop(0)
