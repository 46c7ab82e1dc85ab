"""Pins for the oracle's slot table, slot policy, decode chain and batched layer (CPU only).

Slot policy: invariants checked by brute force over random traces and a
hand-traced case.  Decode chain: prediction-as-routing (§3.2) checked on the
trace itself, the boundary cases (first token, first layer) and determinism.
Batched layer: equal to the one-token layer on every token (§3.1, Math
contract).
"""

import numpy as np
import pytest

from oracle import slots, stack, batched, expert, routing
import synth


def test_slot_table_bind_lookup_unbind():
    t = slots.SlotTable(2, 8, 4)
    t.bind(1, 5, 2)
    assert t.lookup(1, 5) == 2 and t.lookup(0, 5) == -1
    t.bind(1, 6, 2)                  # rebinding the slot evicts expert 5
    assert t.lookup(1, 5) == -1 and t.lookup(1, 6) == 2
    t.bind(1, 6, 3)                  # moving an expert frees its old slot
    assert t.expert_in[1][2] == -1 and t.lookup(1, 6) == 3
    t.unbind(1, 6)
    assert t.lookup(1, 6) == -1 and t.expert_in[1][3] == -1


def test_slot_policy_hand_trace():
    p = slots.SlotPolicy(1, 8, 4)
    assert p.stage(0, [1, 2]) == [(1, 0), (2, 1)]
    assert p.stage(0, [2, 3]) == [(3, 2)]
    assert p.use(0, [1, 2]) == [0, 1]
    # {1, 2} is in use: slots 0, 1 and 2 are pinned; the free slot 3 only fits one
    with pytest.raises(RuntimeError):
        p.stage(0, [4, 5])
    p.release(0)
    # pinned: {2, 3} (queued) and {4, 5}; free slot 3 first, then the LRU
    # unpinned slot, slot 0 (expert 1)
    assert p.stage(0, [4, 5]) == [(4, 3), (5, 0)]
    assert p.use(0, [2, 3]) == [1, 2]
    assert p.use(0, [4, 5]) == [3, 0]
    with pytest.raises(RuntimeError):
        p.use(0, [4, 5])
    p.release(0)
    p.release(0)
    with pytest.raises(RuntimeError):
        p.release(0)


@pytest.mark.parametrize("seed", range(6))
def test_slot_policy_invariants_random(seed):
    rs = np.random.default_rng(seed)
    n_layers, n_exp, k = 3, 16, 4
    n_slots = 3 * k
    p = slots.SlotPolicy(n_layers, n_exp, n_slots)
    queued = [[] for _ in range(n_layers)]
    using = [[] for _ in range(n_layers)]
    for step in range(300):
        layer = int(rs.integers(n_layers))
        total = len(queued[layer]) + len(using[layer])   # at most 2 sets pinned + the new one
        if using[layer] and (rs.random() < 0.3 or (total >= 2 and not queued[layer])):
            using[layer].pop(0)
            p.release(layer)
            continue
        if queued[layer] and (total >= 2 or rs.random() < 0.5):
            want = queued[layer].pop(0)
            got = p.use(layer, want)
            assert [p.table.expert_in[layer][s] for s in got] == want
            using[layer].append(want)
            continue
        experts = [int(e) for e in rs.choice(n_exp, size=k, replace=False)]
        before = {s: p.table.expert_in[layer][s] for s in range(n_slots)}
        pinned_experts = set(e for q in queued[layer] + using[layer] for e in q)
        misses = [e for e in experts if p.table.lookup(layer, e) < 0]
        copies = p.stage(layer, experts)
        # copies = misses, in routing order
        assert [e for e, _ in copies] == misses
        # nothing queued or in use was evicted; every member of those sets is resident
        for e in pinned_experts | set(experts):
            assert p.table.lookup(layer, e) >= 0
        # only copied slots changed
        changed = {s for s in range(n_slots) if p.table.expert_in[layer][s] != before[s]}
        assert changed == {s for _, s in copies}
        queued[layer].append(experts)


def _stack_layers(wl, n_layers, with_heads=True):
    layers = []
    for n in range(n_layers):
        d, perm = synth.mixing(wl, n)
        layers.append({
            "router": synth.router_weights(wl, n, 0),
            "head": synth.router_weights(wl, n, 1) if with_heads else None,
            "mix_d": d, "mix_perm": perm,
            "routed": (lambda e, n=n: synth.bundle(wl, n, e)),
            "shared": [synth.bundle(wl, n, wl.E + s) for s in range(wl.S)],
        })
    return layers


def test_chain_prediction_is_routing():
    wl = synth.WORKLOADS["tiny"]
    layers = _stack_layers(wl, 4)
    xi = synth.token_draws(wl, 0, 3)
    out = stack.decode_chain(xi, layers, wl.K, wl.lora_scale)
    for t, recs in enumerate(out):
        for n, rec in enumerate(recs):
            if t == 0 or n == 0:
                assert rec["src"] == "router"
                _, idx, w = routing.route(layers[n]["router"], rec["x16"], wl.K)
                assert rec["idx"].tolist() == idx.tolist()
            else:
                assert rec["src"] == "pred"
                prev = out[t - 1][n - 1]
                assert rec["idx"].tolist() == prev["pred_idx"].tolist()
                assert np.array_equal(rec["w"], prev["pred_w"])
            if n + 1 < len(layers):
                _, pi, _ = routing.route(layers[n]["head"], rec["x16"], wl.K)
                assert rec["pred_idx"].tolist() == pi.tolist()
            else:
                assert "pred_idx" not in rec
    again = stack.decode_chain(xi, layers, wl.K, wl.lora_scale)
    for a, b in zip(out, again):
        for ra, rb in zip(a, b):
            assert np.array_equal(ra["y"], rb["y"]) and np.array_equal(ra["x16"], rb["x16"])


def test_chain_layer_output_matches_single_layer():
    wl = synth.WORKLOADS["tiny"]
    layers = _stack_layers(wl, 2)
    out = stack.decode_chain(synth.token_draws(wl, 0, 2), layers, wl.K, wl.lora_scale)
    rec = out[1][1]
    single = expert.moe_layer(rec["x16"], wl.K, layers[1]["routed"], layers[1]["shared"],
                              wl.lora_scale, routing=(rec["idx"], rec["w"]))
    assert np.array_equal(single["y"], rec["y"])


def test_chain_without_consumers_uses_own_router():
    wl = synth.WORKLOADS["tiny"]
    layers = _stack_layers(wl, 3)
    out = stack.decode_chain(synth.token_draws(wl, 0, 2), layers, wl.K, wl.lora_scale, consumers=set())
    assert all(rec["src"] == "router" for recs in out for rec in recs)


def test_batched_equals_single_token_layer():
    wl = synth.WORKLOADS["tiny"]
    t = 5
    x = routing.rms_norm_f16(synth.token_draws(wl, 0, t))
    logits = synth.zipf_logits(wl, t, seed=1)
    routed = lambda e: synth.bundle(wl, 0, e)
    out = batched.batched_layer(x, logits, wl.K, routed, [], wl.lora_scale)
    for i in range(t):
        inds, w = routing.softmax_topk(logits[i], wl.K)
        one = expert.moe_layer(x[i], wl.K, routed, [], wl.lora_scale, routing=(inds, w))
        assert out["idx"][i].tolist() == inds.tolist()
        assert np.array_equal(out["y"][i], one["y"])
    sub = batched.batched_layer(x, logits, wl.K, routed, [], wl.lora_scale, tokens=[2])
    assert np.array_equal(sub["y"][2], out["y"][2]) and np.isnan(sub["y"][0]).all()


def test_zipf_logits_popularity_is_skewed():
    wl = synth.WORKLOADS["moe35b"]
    logits = synth.zipf_logits(wl, 512, seed=0)
    idx = np.argsort(-logits, axis=1, kind="stable")[:, :wl.K]
    counts = np.bincount(idx.ravel(), minlength=wl.E)
    assert counts.max() > 300 and (counts > 0).sum() > 150


# ---- the attention stand-in of the chain, pinned by hand-derived values ----

def _golden_standin():
    import json
    import os
    return json.load(open(os.path.join(os.path.dirname(__file__), "golden", "chain_standin.json")))


def test_standin_mix_hand_case():
    g = _golden_standin()["mix"]
    got = stack.mix(np.array(g["r"], np.float32), np.array(g["mix_d"], np.float16),
                    np.array(g["mix_perm"], np.int32))
    assert got.dtype == np.float32
    assert got.tolist() == g["value"]


def test_standin_layer_input_hand_case():
    g = _golden_standin()["layer_input"]
    got = routing.rms_norm_f16(np.array(g["r"], np.float32))
    assert got.dtype == np.float16
    assert got.astype(np.float64).tolist() == g["value"]


def test_standin_token_start_hand_case():
    g = _golden_standin()["token_start"]
    xi = np.array(g["xi"], np.float32)
    got = stack.token_start(xi, np.array(g["r_prev"], np.float32))
    assert got.dtype == np.float32
    assert got.astype(np.float64).tolist() == g["value"]
    assert np.array_equal(stack.token_start(xi, None), xi)


def test_standin_residual_add():
    r = np.array([1.0, 2.0 ** 24, -3.0, 0.5], np.float32)
    y = np.array([0.25, 1.0, 3.0, -0.5], np.float64)
    # fp32 sums: 1.25 exact; 2^24 + 1 rounds to even (2^24); -3 + 3 = 0; 0
    assert stack.add_output(r, y).tolist() == [1.25, 2.0 ** 24, 0.0, 0.0]


def test_chain_records_follow_the_standin():
    """Every record of the chain is tied to its neighbours by the pinned
    stand-in steps: x_N is the layer input of the mixed residual, the next
    layer's mixed residual is mix(r + y_N), and a token starts from the
    previous token's last residual."""
    wl = synth.WORKLOADS["tiny"]
    nl = 3
    layers = _stack_layers(wl, nl)
    xi = synth.token_draws(wl, 0, 3)
    out = stack.decode_chain(xi, layers, wl.K, wl.lora_scale)
    r_prev = None
    for t, recs in enumerate(out):
        r = stack.token_start(xi[t], r_prev)
        for n, rec in enumerate(recs):
            r = stack.mix(r, layers[n]["mix_d"], layers[n]["mix_perm"])
            assert rec["r_mixed"].dtype == np.float32
            assert np.array_equal(rec["r_mixed"], r), (t, n)
            assert np.array_equal(rec["x16"], routing.rms_norm_f16(r)), (t, n)
            r = stack.add_output(r, rec["y"])
        r_prev = r


def test_standin_pins_catch_planted_mistakes():
    """Plausible mistakes in the stand-in, planted in copies of its steps,
    each miss a hand-derived value."""
    g = _golden_standin()
    m = g["mix"]
    r, d, p = (np.array(m["r"], np.float32), np.array(m["mix_d"], np.float16),
               np.array(m["mix_perm"], np.int64))
    r64, d64 = r.astype(np.float64), d.astype(np.float64)
    inv = np.argsort(p)
    swapped = (r64 + d64 * r64[inv]).astype(np.float32)          # permutation the other way
    wrong_side = (r64[p] + d64 * r64).astype(np.float32)         # scale on the wrong operand
    no_skip = (d64 * r64[p]).astype(np.float32)                  # residual term dropped
    for bad in (swapped, wrong_side, no_skip):
        assert bad.tolist() != m["value"]
    ts = g["token_start"]
    xi, rp = np.array(ts["xi"], np.float64), np.array(ts["r_prev"], np.float64)
    dropped = xi.astype(np.float32)                              # previous token ignored
    unnormed = (xi + rp).astype(np.float32)                      # normalization dropped
    meannorm = (xi + rp / np.sqrt(np.mean(rp) + 1e-6)).astype(np.float32)  # mean instead of mean square
    for bad in (dropped, unnormed, meannorm):
        assert bad.astype(np.float64).tolist() != ts["value"]
