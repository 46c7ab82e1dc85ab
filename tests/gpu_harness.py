"""Shared set-up for the GPU parity tests: one layer of a workload on the
device, driven through the C ABI, plus oracle helpers for comparing it."""

import numpy as np

import synth
from oracle import expert as o_expert, routing as o_routing, stack as o_stack

NEAR_TIE = 1e-5          # oracle logit gap below which a top-k swap is allowed
TOL_REL_INF = 2e-3       # max |y - y_ref| / max |y_ref| per layer output
TOL_RESID = 1e-6         # chains: max |r - r_ref| / max |r_ref| of one stand-in step


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


def check_routing(got_idx, got_w, ref_logits, k, what, stats, tie=NEAR_TIE, w_rtol=2e-6):
    """Routing parity: bit-exact set and order, except where the oracle's
    K-th and (K+1)-th logits are within ``tie`` (NEAR_TIE unless the logits
    carry a stated precision of their own; counted); order swaps inside the
    top-K are allowed only between logits within ``tie``."""
    ref_idx, ref_w = o_routing.softmax_topk(ref_logits, k)
    got_idx = np.asarray(got_idx)
    if got_idx.tolist() == ref_idx.tolist():
        assert np.allclose(got_w, ref_w, rtol=w_rtol, atol=1e-7), (what, got_w, ref_w)
        return True
    l = np.asarray(ref_logits, dtype=np.float64)
    # every mismatch must be explained by near-equal logits in the oracle
    order = np.argsort(-l, kind="stable")
    for pos in range(k):
        if got_idx[pos] != ref_idx[pos]:
            assert abs(l[got_idx[pos]] - l[ref_idx[pos]]) <= tie, (what, pos, got_idx, ref_idx)
    assert len(set(got_idx.tolist())) == k
    gap = o_routing.near_tie_gap(l, k)
    if set(got_idx.tolist()) != set(ref_idx.tolist()):
        assert gap <= tie, (what, gap)
        stats["near_tie_set"] = stats.get("near_tie_set", 0) + 1
    else:
        stats["near_tie_order"] = stats.get("near_tie_order", 0) + 1
    del order
    return False


SG_TIE = 1e-6           # sigmoid-group: oracle score gap below which a selection may differ


def sigmoid_group_decisions(l, n, bias):
    """The oracle's selection scores (sigmoid + bias, float64) and its sorted
    group scores (sum of each group's two largest), for explaining a
    difference as a near-tie."""
    sig = 1.0 / (1.0 + np.exp(-np.asarray(l, dtype=np.float64)))
    sel = sig + (0.0 if bias is None else np.asarray(bias, dtype=np.float64))
    per = sel.size // n
    gs = np.sort(np.array([np.sum(np.sort(r)[::-1][:2]) for r in sel.reshape(n, per)]))[::-1]
    return sel, gs


def check_sigmoid_routing(got_idx, got_w, l, k, n, g, s, bias, stats, what):
    """Sigmoid-group routing parity (App. A): the device takes the sigmoid in
    fp32 where the oracle uses float64, so the set and order must be the
    oracle's except where a decision is within SG_TIE in the oracle (the G-th
    and (G+1)-th group scores, or two members whose order differs), counted
    in ``stats['near_tie']``; exact matches must carry the oracle's weights."""
    ref_idx, ref_w = o_routing.sigmoid_group_topk(l, k, n, g, s, bias)
    if np.asarray(got_idx).tolist() == ref_idx.tolist():
        assert np.allclose(got_w, ref_w, rtol=2e-6, atol=1e-7), (what, got_w, ref_w)
        stats["exact"] = stats.get("exact", 0) + 1
        return True
    sel, gs = sigmoid_group_decisions(l, n, bias)
    group_tie = g < n and gs[g - 1] - gs[g] <= SG_TIE
    got = np.asarray(got_idx)
    assert len(set(got.tolist())) == k, (what, got)
    member_ok = all(abs(sel[a] - sel[b]) <= SG_TIE for a, b in zip(got.tolist(), ref_idx.tolist()) if a != b)
    assert group_tie or member_ok, (what, got, ref_idx)
    stats["near_tie"] = stats.get("near_tie", 0) + 1
    return False


def build_chain(wl, L, torch, spec=None):
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
    if spec is None:
        spec = B.spec_from_workload(wl)
    chain = C.DeviceChain(spec, table, dev_layers)
    chain.keep = keep
    torch.cuda.synchronize()
    return chain, np_layers


def _x_flip_is_tie(r32, j, got16, want16):
    """True if element j of fp16(rmsnorm(r32)) sits on a rounding tie: the
    float64 value is within 1e-12 (relative) of the midpoint of the two fp16
    candidates the device and the oracle chose."""
    r64 = np.asarray(r32, dtype=np.float64)
    v = r64[j] / np.sqrt(np.mean(r64 * r64) + o_routing.RMS_EPS)
    a, b = float(got16), float(want16)
    if np.nextafter(np.float16(a), np.float16(b)) != np.float16(b):
        return False                                    # not neighbours
    return abs(v - 0.5 * (a + b)) <= 1e-12 * abs(v)


def teacher_forced_chain(rec, xi, np_layers, wl, L, y_at=None, what="chain", pred_oracle=None,
                         route_check=None):
    """Teacher-forced per-layer parity of a recorded decode chain.

    ``rec`` holds host arrays [T, L, ...] of what the device did at every
    (token t, layer n): ``r`` the residual after the mixing (fp32), ``x`` the
    layer input (fp16), ``idx``/``w`` the routing used, ``pidx``/``pw`` the
    head's prediction, and the layer output as ``y`` (fp32 [d]) or per expert
    as ``ye`` with the residual after the add as ``r_post``.  Each step is
    checked against the oracle run on the device's own inputs of that step:

    * stand-in: ``r`` equals the oracle's mixing of the device's previous
      residual (the token start from the previous token's last one), within
      TOL_RESID;
    * layer input: ``x`` equals ``fp16(rmsnorm(r))`` bit for bit, except on
      rounding ties (counted);
    * routing: own router (token 0, layer 0) bit-exact against the oracle's
      routing of ``x``, except at near-ties of its logits (within NEAR_TIE;
      counted); every other layer uses exactly the prediction the device made
      for it one token earlier;
    * prediction: bit-exact against the oracle's prerouting of ``x``, except
      at near-ties (counted); ``pred_oracle(t, n, x)``, when given, returns
      the oracle's prediction logits and the tie and weight tolerances of a
      head whose logits carry their own stated precision (the full head);
      ``route_check(idx, w, logits, what, stats)``, when given, replaces the
      softmax-top-k check of both (sigmoid-group routing);
    * output (at the (t, n) where ``y_at(t, n)`` holds, default all): within
      TOL_REL_INF of the oracle layer on ``x`` with the device's routing.
    """
    T = xi.shape[0]
    K = wl.K
    if route_check is None:
        def route_check(idx, w, logits, tag, st):
            return check_routing(idx, w, logits, K, tag, st)
    stats = {"steps": 0, "own_routing": 0, "pred_routing": 0, "predictions": 0,
             "routing_near_ties": {}, "prediction_near_ties": {}, "x_tie_flips": 0,
             "y_checked": 0, "max_y_err": 0.0, "max_r_err": 0.0}
    have_y = "y" in rec

    def post(t, n):
        if have_y:   # the device adds its fp32 layer output to its fp32 residual
            return (rec["r"][t, n].astype(np.float32) + rec["y"][t, n].astype(np.float32))
        return rec["r_post"][t, n]

    for t in range(T):
        for n in range(L):
            lay = np_layers[n]
            tag = (what, t, n)
            start = o_stack.token_start(xi[t], None if t == 0 else post(t - 1, L - 1)) \
                if n == 0 else post(t, n - 1)
            r_ref = o_stack.mix(start, lay["mix_d"], lay["mix_perm"])
            r_got = rec["r"][t, n]
            rerr = rel_inf(r_got, r_ref)
            assert rerr <= TOL_RESID, ("stand-in residual", tag, rerr)
            stats["max_r_err"] = max(stats["max_r_err"], rerr)
            x_got = rec["x"][t, n]
            x_ref = o_routing.rms_norm_f16(r_got)
            bad = np.nonzero(x_got.view(np.uint16) != x_ref.view(np.uint16))[0]
            for j in bad:
                assert _x_flip_is_tie(r_got, j, x_got[j], x_ref[j]), ("layer input", tag, int(j))
            stats["x_tie_flips"] += int(bad.size)
            if t == 0 or n == 0:
                logits = o_routing.logits_fp32(lay["router"], x_got)
                route_check(rec["idx"][t, n], rec["w"][t, n], logits, tag, stats["routing_near_ties"])
                stats["own_routing"] += 1
            else:
                assert rec["idx"][t, n].tolist() == rec["pidx"][t - 1, n - 1].tolist(), \
                    ("prediction not used as routing", tag)
                assert np.array_equal(rec["w"][t, n], rec["pw"][t - 1, n - 1]), ("weights", tag)
                stats["pred_routing"] += 1
            if n + 1 < L and pred_oracle is not None:
                pl, tie, w_rtol = pred_oracle(t, n, x_got)
                check_routing(rec["pidx"][t, n], rec["pw"][t, n], pl, K, tag + ("pred",),
                              stats["prediction_near_ties"], tie=tie, w_rtol=w_rtol)
                stats["predictions"] += 1
            elif n + 1 < L and lay.get("head") is not None:
                pl = o_routing.logits_fp32(lay["head"], x_got)
                route_check(rec["pidx"][t, n], rec["pw"][t, n], pl, tag + ("pred",), stats["prediction_near_ties"])
                stats["predictions"] += 1
            if y_at is None or y_at(t, n):
                idx = np.asarray(rec["idx"][t, n], dtype=np.int64)
                ys = [o_expert.expert_forward(lay["routed"](int(e)), x_got, wl.lora_scale)[0]
                      for e in idx]
                ysh = [o_expert.expert_forward(b, x_got, wl.lora_scale)[0] for b in lay["shared"]]
                if have_y:
                    y_ref = o_expert.combine(rec["w"][t, n], ys, ysh)
                    err = rel_inf(rec["y"][t, n], y_ref)
                    assert err <= TOL_REL_INF, ("layer output", tag, err)
                else:
                    err = 0.0
                    for k, yr in enumerate(ys + ysh):
                        err = max(err, rel_inf(rec["ye"][t, n, 0, k], yr))
                    assert err <= TOL_REL_INF, ("expert outputs", tag, err)
                    # the residual add used these outputs and the routing weights
                    r_add = o_stack.add_output(r_got, o_expert.combine(
                        rec["w"][t, n], [rec["ye"][t, n, 0, k] for k in range(K)],
                        [rec["ye"][t, n, 0, K + s_] for s_ in range(wl.S)]))
                    aerr = rel_inf(rec["r_post"][t, n], r_add)
                    assert aerr <= TOL_RESID, ("residual add", tag, aerr)
                stats["max_y_err"] = max(stats["max_y_err"], err)
                stats["y_checked"] += 1
            stats["steps"] += 1
    return stats


def free_running_divergence(rec, xi, np_layers, wl, L):
    """Report (not a check): the first (t, n) at which the device's free-running
    routing leaves the oracle's free-running chain on the same draws, with the
    oracle's logit gap there; None if they agree over all of ``xi``."""
    ref = o_stack.decode_chain(xi, np_layers, wl.K, wl.lora_scale)
    for t in range(len(ref)):
        for n in range(L):
            r = ref[t][n]
            got = rec["idx"][t, n].tolist()
            if got != r["idx"].tolist():
                if r["src"] == "router":
                    logits = o_routing.logits_fp32(np_layers[n]["router"], r["x16"])
                else:
                    logits = ref[t - 1][n - 1]["pred_logits"]
                return {"token": t, "layer": n, "oracle_gap": o_routing.near_tie_gap(logits, wl.K)}
    return None


def sample_layers(T, L, full_tokens=2, per_token=3, seed=0):
    """(t, n) -> bool: every layer of the first ``full_tokens`` tokens, then
    ``per_token`` seeded layers of each later token."""
    rs = np.random.default_rng(seed)
    pick = {(t, n) for t in range(min(T, full_tokens)) for n in range(L)}
    for t in range(full_tokens, T):
        for n in rs.choice(L, size=min(per_token, L), replace=False):
            pick.add((t, int(n)))
    return lambda t, n: (t, n) in pick


