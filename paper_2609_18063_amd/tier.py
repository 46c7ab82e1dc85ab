"""Decode chain with host-tier expert staging (the 8B tier on one GPU).

The experts of every layer live in pinned host memory; each layer has a
small pool of device slots (3 x top-K).  Per token t and layer N (§3.2,
Motivation and Prediction-as-routing; §3.1, staged executor):

* layer 0, and every layer of token 0, route with their own router: the host
  reads the routing back and stages the set on demand (the kernels wait);
* head N's prediction for layer N+1 at token t+1 is read back one layer
  later and staged at once, so its copies overlap the rest of token t and
  the first layers of token t+1;
* the compute stream waits for exactly the copies of the set it uses, and a
  set stays pinned until the host knows its kernels finished.

Everything on the device is the library's: the per-call kernels for the
layer, and the library's stager (policy, slot-table rows, hipMemcpyAsync).
This module only orders the calls and moves the K routing ids to the host.

With a :class:`FilePool` the bundles live in a file instead (the SSD tier of
§3.1, SSD streaming): the library maps it and reads each missing record
through a pinned bounce buffer, so the page cache (warm) or the disk (cold)
sits in front of the PCIe copy.
"""

import os

import time

import torch

from . import binding as B
from . import weights as W


def bundle_layout(bundle):
    """Pack one bundle alone: (packed bytes, MoeBundleLayout)."""
    buf, boffs, _ = W.pack_host([bundle])
    d = boffs[0]
    lay = B.MoeBundleLayout()
    for p in ("gate", "up", "down"):
        arr = getattr(lay, p)
        for i, kind in enumerate(("q", "sz", "a", "b")):
            arr[i] = d.get((p, kind), -1)
    return buf, lay


class HostPool:
    """Pinned host memory holding the packed bundles of every layer:
    ``[n_layers][n_ids]`` bundles of ``stride`` bytes."""

    def __init__(self, n_layers, n_ids, bundle_fn, replicate=False):
        """``bundle_fn(layer, expert)`` gives a bundle; with ``replicate`` only
        layer 0's bundles are built and every layer holds a copy of them (at
        its own addresses)."""
        first, self.layout = bundle_layout(bundle_fn(0, 0))
        self.bundle_bytes = first.nbytes
        self.stride = (first.nbytes + 255) // 256 * 256
        self.n_layers, self.n_ids = n_layers, n_ids
        self.buf = torch.empty(n_layers * n_ids * self.stride, dtype=torch.uint8, pin_memory=True)
        host = self.buf.numpy()
        per_layer = n_ids * self.stride
        for n in range(n_layers):
            if replicate and n > 0:
                host[n * per_layer:(n + 1) * per_layer] = host[:per_layer]
                continue
            for e in range(n_ids):
                b = first if (n, e) == (0, 0) else bundle_layout(bundle_fn(n, e))[0]
                o = (n * n_ids + e) * self.stride
                host[o:o + b.nbytes] = b

    def ptrs(self):
        base = self.buf.data_ptr()
        return [base + i * self.stride for i in range(self.n_layers * self.n_ids)]

    def bytes_of(self, layer, expert):
        o = (layer * self.n_ids + expert) * self.stride
        return self.buf[o:o + self.bundle_bytes]


class FilePool:
    """The bundles of every layer in one file, ``[n_layers][n_ids]`` records
    of ``stride`` bytes (the layout of :class:`HostPool`), read by the
    library's file-tier stager through ``n_bounce`` pinned bounce buffers
    and ``n_io`` host threads."""

    def __init__(self, path, n_layers, n_ids, bundle_fn, replicate=False, n_bounce=4, n_io=4):
        first, self.layout = bundle_layout(bundle_fn(0, 0))
        self.bundle_bytes = first.nbytes
        self.stride = (first.nbytes + 255) // 256 * 256
        self.n_layers, self.n_ids = n_layers, n_ids
        self.path, self.n_bounce, self.n_io = str(path), n_bounce, n_io
        pad = bytes(self.stride - first.nbytes)
        with open(self.path, "wb") as f:
            block = None
            for n in range(n_layers):
                if replicate and block is not None:
                    f.write(block)
                    continue
                parts = []
                for e in range(n_ids):
                    b = first if (n, e) == (0, 0) else bundle_layout(bundle_fn(n, e))[0]
                    parts.append(b.tobytes() + pad)
                blk = b"".join(parts)
                if replicate:
                    block = blk
                f.write(blk)

    def stager_file(self):
        return (self.path, self.stride, self.n_bounce, self.n_io)

    def bytes_of(self, layer, expert):
        o = (layer * self.n_ids + expert) * self.stride
        with open(self.path, "rb") as f:
            f.seek(o)
            data = f.read(self.bundle_bytes)
        return torch.frombuffer(bytearray(data), dtype=torch.uint8)

    def drop_page_cache(self):
        """Ask the kernel to drop the file's clean pages (a cold read next)."""
        fd = os.open(self.path, os.O_RDONLY)
        try:
            os.fsync(fd)
            os.posix_fadvise(fd, 0, 0, os.POSIX_FADV_DONTNEED)
        finally:
            os.close(fd)

    def remove(self):
        try:
            os.remove(self.path)
        except FileNotFoundError:
            pass


class TieredChain:
    """Decode chain of ``len(layers)`` layers whose experts are staged from
    ``pool`` into ``n_slots`` device slots per layer.

    ``layers``: dicts with device tensors ``router``, ``head`` (None on the
    last layer), ``mix_d`` and ``mix_perm``, as for the resident chain.
    """

    def __init__(self, spec, layers, pool, n_slots):
        self.spec, self.layers, self.host = spec, layers, pool
        self.L = len(layers)
        d, K = spec.d_model, spec.top_k
        self.K = K
        n_ids = spec.n_experts + spec.n_shared
        dev = "cuda"
        self.table = B.SlotTable(self.L, n_ids, n_slots)
        self.table.sync()
        self.slots = torch.empty(self.L * n_slots * pool.stride, dtype=torch.uint8, device=dev)
        if isinstance(pool, FilePool):
            self.stager = B.Stager(self.table, pool.layout, pool.bundle_bytes, None, self.slots,
                                   pool.stride, file=pool.stager_file())
        else:
            self.stager = B.Stager(self.table, pool.layout, pool.bundle_bytes, pool.ptrs(), self.slots,
                                   pool.stride)
        # the layers run on `compute`, the staging copies on `copy`: two streams
        # made back to back, so that they never share a hardware queue
        self.streams = B.StreamPair()
        self.copy_stream = self.streams.copy
        self.ws = torch.zeros(B.workspace_bytes(spec, 1), dtype=torch.uint8, device=dev)
        self.r = torch.zeros(1, d, dtype=torch.float32, device=dev)
        self.x = torch.empty(1, d, dtype=torch.float16, device=dev)
        self.xi = torch.zeros(1, d, dtype=torch.float32, device=dev)
        self.own_idx = torch.empty(1, K, dtype=torch.int32, device=dev)
        self.own_w = torch.empty(1, K, dtype=torch.float32, device=dev)
        self.pred_idx = torch.zeros(2, self.L, 1, K, dtype=torch.int32, device=dev)
        self.pred_w = torch.zeros(2, self.L, 1, K, dtype=torch.float32, device=dev)
        self.own_host = torch.empty(K, dtype=torch.int32, pin_memory=True)
        self.pred_host = torch.empty(2, self.L, K, dtype=torch.int32, pin_memory=True)
        self.ye = torch.empty(1, K + spec.n_shared, d, dtype=torch.float32, device=dev)
        self.status = torch.zeros(1, dtype=torch.int32, device=dev)
        self.shared = list(range(spec.n_experts, n_ids))
        self.staged = {}        # (t, n) -> staged host set
        self.queued = None      # (t + 1, n + 1, event) prediction read back, not yet staged
        self.used_layers = []   # layers of the sets used and not yet released, in use order
        self.copy_ms = 0.0
        self.stage_host_s = []  # (copies, host seconds) of every stage call
        self.copy_events = []
        self.stall_s = 0.0
        self.log = []           # (t, n, "demand" | "predicted", set, copies)
        self.ops = []           # every policy call in order: ("stage", n, set, copies) | ("use", n, set) | ("release", n)

    def _release(self, keep):
        while len(self.used_layers) > keep:
            n = self.used_layers.pop(0)
            self.stager.release(n)
            self.ops.append(("release", n))

    def _stage(self, t, n, experts, kind):
        s = [int(e) for e in experts] + self.shared
        start = torch.cuda.Event(enable_timing=True)
        stop = torch.cuda.Event(enable_timing=True)
        start.record(self.copy_stream)
        h0 = time.perf_counter()
        copies = self.stager.stage(n, s, self.copy_stream)
        self.stage_host_s.append((len(copies), time.perf_counter() - h0))
        stop.record(self.copy_stream)
        if copies:
            self.copy_events.append((start, stop))
        self.log.append((t, n, kind, s, copies))
        self.ops.append(("stage", n, s, copies))
        return s

    def _process_queued(self):
        """Head n finished (the event also covers its layer's experts): every
        set in use but the last one is done; stage the prediction."""
        if self.queued is None:
            return
        tq, nq, ev = self.queued
        self.queued = None
        t0 = time.perf_counter()
        ev.synchronize()
        self.stall_s += time.perf_counter() - t0
        self._release(keep=1)
        self.staged[(tq, nq)] = self._stage(tq, nq, self.pred_host[tq % 2, nq].tolist(), "predicted")

    def run_token(self, t, xi_row, record=None):
        """One token through all layers; ``xi_row`` is a device fp32 [1, d]."""
        s = self.spec
        cur = torch.cuda.current_stream()
        self.xi.copy_(xi_row)
        B.chain_token_start(self.xi, self.r)
        for n, lay in enumerate(self.layers):
            B.chain_mix_rmsnorm(lay["mix_d"], lay["mix_perm"], self.r, self.x)
            if record is not None:
                record["r"][t, n].copy_(self.r[0])
            if t > 0 and n > 0:
                idx, w = self.pred_idx[t % 2, n], self.pred_w[t % 2, n]
                st = self.staged.pop((t, n))
            else:
                B.route(s, self.x, lay["router"], self.own_idx, self.own_w, self.ws)
                self.own_host.copy_(self.own_idx[0], non_blocking=True)
                ev = torch.cuda.Event()
                ev.record(cur)
                t0 = time.perf_counter()
                ev.synchronize()                     # demand: the host needs the routing now
                self.stall_s += time.perf_counter() - t0
                self._release(keep=0)
                st = self._stage(t, n, self.own_host.tolist(), "demand")
                idx, w = self.own_idx, self.own_w
            self.stager.use(n, st, cur)
            self.ops.append(("use", n, st))
            self.used_layers.append(n)
            has_head = n + 1 < self.L and lay.get("head") is not None
            if has_head:
                nxt = (t + 1) % 2
                B.preroute(s, self.x, lay["head"], self.pred_idx[nxt, n + 1],
                           self.pred_w[nxt, n + 1], self.ws)
            ye = self.ye if record is None else record["ye"][t, n]
            B.expert_ffn(s, self.table, n, self.x, idx, ye, self.status, self.ws)
            B.combine_add(s, ye, w, self.r)
            if record is not None:
                record["r_post"][t, n].copy_(self.r[0])
                record["x"][t, n].copy_(self.x[0])
                record["idx"][t, n].copy_(idx[0])
                record["w"][t, n].copy_(w[0])
                if has_head:
                    record["pidx"][t, n].copy_(self.pred_idx[(t + 1) % 2, n + 1, 0])
                    record["pw"][t, n].copy_(self.pred_w[(t + 1) % 2, n + 1, 0])
            # the previous layer's prediction: its kernels are done or nearly so
            self._process_queued()
            if has_head:
                self.pred_host[(t + 1) % 2, n + 1].copy_(self.pred_idx[(t + 1) % 2, n + 1, 0],
                                                         non_blocking=True)
                ev = torch.cuda.Event()
                ev.record(cur)                       # after the layer's experts and combine
                self.queued = (t + 1, n + 1, ev)
        self._process_queued()

    def finish(self):
        """Wait for all work; release every set in use."""
        torch.cuda.synchronize()
        self._release(keep=0)
        self.copy_ms += sum(a.elapsed_time(b) for a, b in self.copy_events)
        self.copy_events = []

    def new_record(self, T):
        s = self.spec
        n = s.top_k + s.n_shared
        L, d, K = self.L, s.d_model, s.top_k
        dev = "cuda"
        return {
            "x": torch.zeros(T, L, d, dtype=torch.float16, device=dev),
            "r": torch.zeros(T, L, d, dtype=torch.float32, device=dev),
            "r_post": torch.zeros(T, L, d, dtype=torch.float32, device=dev),
            "idx": torch.zeros(T, L, K, dtype=torch.int32, device=dev),
            "w": torch.zeros(T, L, K, dtype=torch.float32, device=dev),
            "pidx": torch.full((T, L, K), -1, dtype=torch.int32, device=dev),
            "pw": torch.zeros(T, L, K, dtype=torch.float32, device=dev),
            "ye": torch.zeros(T, L, 1, n, d, dtype=torch.float32, device=dev),
        }

    def run(self, xi_tokens, record=False):
        """Eager run over device fp32 draws ``[T, d]``; returns the record or None."""
        T = xi_tokens.shape[0]
        rec = self.new_record(T) if record else None
        self.r.zero_()
        self.streams.compute.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(self.streams.compute):
            for t in range(T):
                self.run_token(t, xi_tokens[t:t + 1], record=rec)
        self.finish()
        return rec

    def slot_bytes(self, layer, slot):
        o = (layer * self.table.n_slots + slot) * self.host.stride
        return self.slots[o:o + self.host.bundle_bytes]

    def close(self):
        self.stager.close()
        self.table.close()
        self.streams.close()


def set_overlap(log, L):
    """Mean fraction of a layer's set kept from the previous token."""
    last, kept, n = {}, 0, 0
    for t, layer, _, s, _ in log:
        if layer in last:
            kept += len(set(s) & set(last[layer]))
            n += len(s)
        last[layer] = s
    return kept / n if n else 0.0


def resident_table(spec, pool, layers):
    """Every bundle of ``pool`` copied to the device and bound (no staging):
    the all-resident reference for the same weights.  Returns (table, keep)."""
    L, n_ids = pool.n_layers, pool.n_ids
    dev = pool.buf.to("cuda")
    table = B.SlotTable(L, n_ids, n_ids)
    base = dev.data_ptr()
    lay = pool.layout
    for n in range(L):
        for e in range(n_ids):
            o = base + (n * n_ids + e) * pool.stride
            projs = []
            for p in ("gate", "up", "down"):
                f = list(getattr(lay, p))
                projs.append(B.MoeProj(o + f[0], o + f[1], None if f[2] < 0 else o + f[2],
                                       None if f[3] < 0 else o + f[3]))
            table.bind(n, e, e, B.MoeBundle(*projs), keep=dev)
    table.sync()
    return table, dev


__all__ = ["HostPool", "TieredChain", "bundle_layout", "set_overlap", "resident_table"]


class WholeLayerPrefill:
    """Prefill of T tokens through the layers of ``pool`` on the whole-layer
    path (§3.1, Executor paths; §3.2, Two consumption profiles): every
    expert of a layer is loaded in one shot, into one of two device layer
    buffers, while the previous layer computes on the other.

    Per layer N (a prefill routes every layer by its own router; the
    residual stream of the T tokens stands in for attention):
    ``x = fp16(rmsnorm(r))``, ``moe_route``, the grouped experts on table
    layer N mod 2, ``r += combine`` (``moe_combine_add``); ``r`` starts at
    the token draws. The loads are single host -> device copies of the
    layer's packed bundles ([n_ids] records of ``stride`` bytes) from the
    pinned pool, or, for a :class:`FilePool`, the layer's records read from
    the file into a pinned staging buffer first (the page cache or the disk
    in front of the copy); the copy of layer N+1 waits for the compute of
    layer N-1, which last used its buffer.

    ``resident=True`` binds every layer at once to a device copy of the
    whole pool instead (the comparison the path must match bit for bit).
    ``routers``: device fp16 [E, d] per layer."""

    def __init__(self, spec, routers, pool, resident=False):
        self.spec, self.routers, self.pool = spec, routers, pool
        self.L, self.n_ids = pool.n_layers, pool.n_ids
        self.resident = resident
        self.per_layer = self.n_ids * pool.stride
        nb = self.L if resident else 2
        self.table = B.SlotTable(nb, self.n_ids, self.n_ids)
        self.buf = torch.empty(nb * self.per_layer, dtype=torch.uint8, device="cuda")
        base = self.buf.data_ptr()
        lay = pool.layout

        def proj(addr, offs):
            return B.MoeProj(addr + offs[0], addr + offs[1],
                             (addr + offs[2]) if offs[2] >= 0 else None,
                             (addr + offs[3]) if offs[3] >= 0 else None)

        for b in range(nb):
            for e in range(self.n_ids):
                a = base + b * self.per_layer + e * pool.stride
                self.table.bind(b, e, e, B.MoeBundle(proj(a, lay.gate), proj(a, lay.up), proj(a, lay.down)))
        self.table.sync()
        # the layers run on `compute`, the loads on `copy`: two streams made
        # back to back, so that they never share a hardware queue
        self.streams = B.StreamPair()
        self.copy_stream = self.streams.copy
        self.stage = None
        if isinstance(pool, FilePool):   # two pinned staging buffers, alternating by layer
            self.stage = [torch.empty(self.per_layer, dtype=torch.uint8, pin_memory=True) for _ in range(2)]
            self.stage_free = [torch.cuda.Event(), torch.cuda.Event()]
        if resident:
            for n in range(self.L):
                self._load(n, n, torch.cuda.current_stream())
            torch.cuda.synchronize()
        self.load_ms = []

    def _load(self, n, b, stream):
        dst = self.buf[b * self.per_layer:(b + 1) * self.per_layer]
        if self.stage is None:
            src = self.pool.buf[n * self.per_layer:(n + 1) * self.per_layer]
        else:
            sb = n % 2
            self.stage_free[sb].synchronize()      # the copy out of this staging buffer is done
            with open(self.pool.path, "rb", buffering=0) as f:
                f.seek(n * self.per_layer)
                mv = memoryview(self.stage[sb].numpy())
                got = 0
                while got < self.per_layer:
                    k = f.readinto(mv[got:])
                    if not k:
                        raise IOError("short read of layer %d" % n)
                    got += k
            src = self.stage[sb]
        with torch.cuda.stream(stream):
            dst.copy_(src, non_blocking=True)
            if self.stage is not None:
                self.stage_free[n % 2].record(stream)

    def run(self, xi, record=False):
        """``xi`` device fp32 [T, d] -> final residual [T, d] (and, with
        ``record``, the per-layer x, idx, w and residual before each layer)."""
        spec = self.spec
        T, d = xi.shape
        K, n = spec.top_k, spec.top_k + spec.n_shared
        caller = torch.cuda.current_stream()
        cur = self.streams.compute
        cur.wait_stream(caller)
        with torch.cuda.stream(cur):
            out = self._run(xi, record, spec, T, d, K, n, cur)
        caller.wait_stream(cur)
        return out

    def _run(self, xi, record, spec, T, d, K, n, cur):
        r = xi.clone()
        x = torch.empty(T, d, dtype=torch.float16, device="cuda")
        idx = torch.empty(T, K, dtype=torch.int32, device="cuda")
        w = torch.empty(T, K, dtype=torch.float32, device="cuda")
        ye = torch.empty(T, n, d, dtype=torch.float32, device="cuda")
        ws = torch.zeros(B.workspace_bytes(spec, T), dtype=torch.uint8, device="cuda")
        self.status = torch.zeros(1, dtype=torch.int32, device="cuda")
        rec = {"x": [], "idx": [], "w": [], "r": []} if record else None
        loaded = [torch.cuda.Event(), torch.cuda.Event()]
        freed = [torch.cuda.Event(), torch.cuda.Event()]
        if not self.resident:
            self.copy_stream.wait_stream(cur)
            self._load(0, 0, self.copy_stream)
            loaded[0].record(self.copy_stream)
        for N in range(self.L):
            b = N if self.resident else N % 2
            if not self.resident:
                cur.wait_event(loaded[b])
            if record:
                rec["r"].append(r.clone())
            B.rmsnorm_f16(r, x)
            B.route(spec, x, self.routers[N], idx, w, ws)
            B.expert_ffn_grouped(spec, self.table, b, x, idx, ye, self.status, ws)
            B.combine_add(spec, ye, w, r)
            if record:
                rec["x"].append(x.clone())
                rec["idx"].append(idx.clone())
                rec["w"].append(w.clone())
            if not self.resident:
                freed[b].record(cur)
                if N + 1 < self.L:   # the next layer's load (host read included) while this one computes
                    if N >= 1:       # its buffer was last read by layer N - 1
                        self.copy_stream.wait_event(freed[(N + 1) % 2])
                    self._load(N + 1, (N + 1) % 2, self.copy_stream)
                    loaded[(N + 1) % 2].record(self.copy_stream)
        return r, rec

    def close(self):
        torch.cuda.synchronize()
        self.table.close()
        self.streams.close()
