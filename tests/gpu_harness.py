"""Shared set-up for the GPU parity tests: one layer of a workload on the
device, driven through the C ABI, plus oracle helpers for comparing it."""

import numpy as np

import synth
from oracle import expert as o_expert, routing as o_routing

NEAR_TIE = 1e-5          # oracle logit gap below which a top-k swap is allowed
CHAIN_TIE = 5e-4         # chains: logit gap below which a divergence is accepted
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


def build_chain(wl, L, torch):
    from paper_2609_18063_amd import binding as B, weights as W, chain as C
    n_ids = wl.E + wl.S
    table = B.SlotTable(L, n_ids, n_ids)
    dev_layers, np_layers, keep = [], [], []
    for n in range(L):
        bundles = [synth.bundle(wl, n, e) for e in range(n_ids)]
        router = synth.router_weights(wl, n, 0)
        head = synth.router_weights(wl, n, 1)
        mix_d, perm = synth.mixing(wl, n)
        buf, boffs, eoffs = W.pack_host(bundles, extra=[router, head, mix_d, perm])
        del bundles
        dev = W.upload(buf)
        keep.append(dev)
        W.bind_layer(table, n, dev, boffs, np.random.default_rng(2000 + n).permutation(n_ids))
        last = n + 1 == L
        dev_layers.append({
            "router": W.extra_tensor(dev, eoffs[0], router.shape, torch.float16),
            "head": None if last else W.extra_tensor(dev, eoffs[1], head.shape, torch.float16),
            "mix_d": W.extra_tensor(dev, eoffs[2], mix_d.shape, torch.float16),
            "mix_perm": W.extra_tensor(dev, eoffs[3], perm.shape, torch.int32),
        })
        cache = {}

        def routed(e, n=n, cache=cache):
            if e not in cache:
                cache[e] = synth.bundle(wl, n, e)
            return cache[e]

        np_layers.append({"router": router, "head": None if last else head, "mix_d": mix_d,
                          "mix_perm": perm, "routed": routed,
                          "shared": [synth.bundle(wl, n, wl.E + s) for s in range(wl.S)]})
    table.sync()
    spec = B.spec_from_workload(wl)
    chain = C.DeviceChain(spec, table, dev_layers)
    chain.keep = keep
    torch.cuda.synchronize()
    return chain, np_layers


def _gap_between(logits, a, b):
    l = np.asarray(logits, dtype=np.float64)
    return abs(l[a] - l[b])


def compare_chain(rec, ref, np_layers, wl, L):
    """Layer-by-layer comparison until the first routing divergence."""
    T = len(ref)
    x = rec["x"].cpu().numpy()
    idx = rec["idx"].cpu().numpy()
    w = rec["w"].cpu().numpy()
    pidx = rec["pidx"].cpu().numpy()
    pw = rec["pw"].cpu().numpy()
    ye = rec["ye"].cpu().numpy() if "ye" in rec else None
    y = rec["y"].cpu().numpy() if "y" in rec else None
    stats = {"layers": 0, "x_ulp_flips": 0, "max_err": 0.0, "diverged_at": None}
    for t in range(T):
        for n in range(L):
            r = ref[t][n]
                        # x is an intermediate output of the chain: held to the layer bar
            gxf = x[t, n].astype(np.float64)
            rxf = r["x16"].astype(np.float64)
            xerr = rel_inf(gxf, rxf)
            assert xerr <= TOL_REL_INF, ("x", t, n, xerr)
            stats["max_x_err"] = max(stats.get("max_x_err", 0.0), xerr)
            stats["x_ulp_flips"] += int((gxf != rxf).sum())
            got = idx[t, n].tolist()
            want = r["idx"].tolist()
            if got != want:
                # the decision that produced this routing: own router at (t, n), or
                # the head of layer n-1 at token t-1
                if r["src"] == "router":
                    logits = o_routing.logits_fp32(np_layers[n]["router"], r["x16"])
                else:
                    logits = ref[t - 1][n - 1]["pred_logits"]
                pos = next(i for i in range(wl.K) if got[i] != want[i])
                gap = _gap_between(logits, got[pos], want[pos]) if got[pos] >= 0 else np.inf
                assert gap <= CHAIN_TIE, ("routing diverged away from a near-tie", t, n, gap)
                stats["diverged_at"] = (t, n, gap)
                return stats
            # weights follow the drifting logits: held to the layer-output bar
            assert rel_inf(w[t, n], r["w"]) <= TOL_REL_INF, (t, n, w[t, n], r["w"])
            if ye is not None:
                for k in range(wl.K + wl.S):
                    err = rel_inf(ye[t, n, 0, k], r["y_experts"][k])
                    assert err <= TOL_REL_INF, ("expert", t, n, k, err)
                    stats["max_err"] = max(stats["max_err"], err)
            if y is not None:
                err = rel_inf(y[t, n], r["y"])
                assert err <= TOL_REL_INF, ("layer output", t, n, err)
                stats["max_err"] = max(stats["max_err"], err)
            if "pred_idx" in r:
                gp = pidx[t, n].tolist()
                if gp != r["pred_idx"].tolist():
                    pos = next(i for i in range(wl.K) if gp[i] != r["pred_idx"][i])
                    gap = _gap_between(r["pred_logits"], gp[pos], r["pred_idx"][pos])
                    assert gap <= CHAIN_TIE, ("prediction differs away from a near-tie", t, n, gap)
                else:
                    assert rel_inf(pw[t, n], r["pred_w"]) <= TOL_REL_INF, (t, n)
            stats["layers"] += 1
    return stats
