"""Shared set-up for the GPU parity tests: one layer of a workload on the
device, driven through the C ABI, plus oracle helpers for comparing it."""

import numpy as np

import synth
from oracle import expert as o_expert, routing as o_routing

NEAR_TIE = 1e-5          # oracle logit gap below which a top-k swap is allowed
TOL_REL_INF = 2e-3       # max |y - y_ref| / max |y_ref| per layer output


def rel_inf(got, ref):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    den = np.max(np.abs(ref))
    return float(np.max(np.abs(got - ref)) / (den if den > 0 else 1.0))


class DeviceLayer:
    """All experts (routed + shared) of one layer of workload ``wl`` resident
    on the device, bound at a seeded permutation of slots."""

    def __init__(self, wl, layer=0, lora=True, seed=0):
        import torch
        from paper_2609_18063_amd import binding as B, weights as W
        self.wl, self.layer = wl, layer
        self.n_ids = wl.E + wl.S
        self.bundles_np = None
        self.lora = lora
        bundles = [synth.bundle(wl, layer, e, lora=lora) for e in range(self.n_ids)]
        self.router = synth.router_weights(wl, layer, 0)
        self.head = synth.router_weights(wl, layer, 1)
        buf, boffs, eoffs = W.pack_host(bundles, extra=[self.router, self.head])
        self.dev = W.upload(buf)
        self.router_t = W.extra_tensor(self.dev, eoffs[0], self.router.shape, torch.float16)
        self.head_t = W.extra_tensor(self.dev, eoffs[1], self.head.shape, torch.float16)
        self.perm = np.random.default_rng(1000 + seed).permutation(self.n_ids)
        self.table = B.SlotTable(1, self.n_ids, self.n_ids)
        self.mbundles = W.bind_layer(self.table, 0, self.dev, boffs, self.perm)
        self.table.sync()
        self.spec = B.spec_from_workload(wl)
        self._cache = {}
        torch.cuda.synchronize()

    def bundle_np(self, e):
        """The oracle's copy of expert ``e`` (regenerated from its seed)."""
        if e not in self._cache:
            self._cache[e] = synth.bundle(self.wl, self.layer, e, lora=self.lora)
        return self._cache[e]

    def alloc(self, T):
        import torch
        from paper_2609_18063_amd import binding as B
        wl = self.wl
        n = wl.K + wl.S
        ws = torch.zeros(B.workspace_bytes(self.spec, T), dtype=torch.uint8, device="cuda")
        return {
            "ws": ws,
            "x": torch.empty(T, wl.d, dtype=torch.float16, device="cuda"),
            "logits": torch.empty(T, wl.E, dtype=torch.float32, device="cuda"),
            "idx": torch.empty(T, wl.K, dtype=torch.int32, device="cuda"),
            "w": torch.empty(T, wl.K, dtype=torch.float32, device="cuda"),
            "plogits": torch.empty(T, wl.E, dtype=torch.float32, device="cuda"),
            "pidx": torch.empty(T, wl.K, dtype=torch.int32, device="cuda"),
            "pw": torch.empty(T, wl.K, dtype=torch.float32, device="cuda"),
            "ye": torch.empty(T, n, wl.d, dtype=torch.float32, device="cuda"),
            "y": torch.empty(T, wl.d, dtype=torch.float32, device="cuda"),
            "status": torch.zeros(1, dtype=torch.int32, device="cuda"),
        }

    def run(self, xi, bufs=None, idx_override=None):
        """Whole layer on fp32 draws ``xi [T, d]``: input norm, route,
        preroute, experts, combine.  Returns host copies."""
        import torch
        from paper_2609_18063_amd import binding as B
        T = xi.shape[0]
        b = bufs or self.alloc(T)
        xi_t = torch.from_numpy(np.ascontiguousarray(xi, dtype=np.float32)).cuda()
        B.rmsnorm_f16(xi_t, b["x"])
        B.route(self.spec, b["x"], self.router_t, b["idx"], b["w"], b["ws"], logits=b["logits"])
        B.preroute(self.spec, b["x"], self.head_t, b["pidx"], b["pw"], b["ws"], logits=b["plogits"])
        idx = b["idx"]
        if idx_override is not None:
            idx = torch.from_numpy(np.ascontiguousarray(idx_override, dtype=np.int32)).cuda()
        B.expert_ffn(self.spec, self.table, 0, b["x"], idx, b["ye"], b["status"], b["ws"])
        w = b["w"]
        B.combine(self.spec, b["ye"], w, b["y"])
        torch.cuda.synchronize()
        out = {k: v.cpu().numpy() for k, v in b.items() if k != "ws"}
        out["idx_used"] = idx.cpu().numpy()
        return out


def oracle_token(dl, xi_row, routing=None):
    """Oracle layer for one token of fp32 draws ``xi_row``."""
    wl = dl.wl
    x16 = o_routing.rms_norm_f16(xi_row)
    shared = [dl.bundle_np(wl.E + s) for s in range(wl.S)]
    out = o_expert.moe_layer(x16, wl.K, dl.bundle_np, shared, wl.lora_scale,
                             w_router16=dl.router, w_head16=dl.head, routing=routing)
    out["x16"] = x16
    return out


def check_routing(got_idx, got_w, ref_logits, k, what, stats):
    """Routing parity: bit-exact set and order, except where the oracle's
    K-th and (K+1)-th logits are within NEAR_TIE (counted); order swaps
    inside the top-K are allowed only between logits within NEAR_TIE."""
    ref_idx, ref_w = o_routing.softmax_topk(ref_logits, k)
    got_idx = np.asarray(got_idx)
    if got_idx.tolist() == ref_idx.tolist():
        assert np.allclose(got_w, ref_w, rtol=2e-6, atol=1e-7), (what, got_w, ref_w)
        return True
    l = np.asarray(ref_logits, dtype=np.float64)
    # every mismatch must be explained by near-equal logits in the oracle
    order = np.argsort(-l, kind="stable")
    for pos in range(k):
        if got_idx[pos] != ref_idx[pos]:
            assert abs(l[got_idx[pos]] - l[ref_idx[pos]]) <= NEAR_TIE, (what, pos, got_idx, ref_idx)
    assert len(set(got_idx.tolist())) == k
    gap = o_routing.near_tie_gap(l, k)
    if set(got_idx.tolist()) != set(ref_idx.tolist()):
        assert gap <= NEAR_TIE, (what, gap)
        stats["near_tie_set"] = stats.get("near_tie_set", 0) + 1
    else:
        stats["near_tie_order"] = stats.get("near_tie_order", 0) + 1
    del order
    return False
