"""GPU tests of the host-tier decode chain (the 8B tier on one GPU).

The staged chain is held to the same bars as the resident chain:
* teacher-forced per-layer parity with the oracle (each layer on the
  device's own inputs: stand-in residual, layer input, routing bit-exact up
  to counted near-ties, prediction consumed as routing, expert outputs and
  the residual add within the layer bar);
* bit-identical records to the all-resident chain on the same weights and
  tokens (staging moves bytes, it must not change a single result);
* every resident slot holds exactly the host bytes of its expert;
* the copies the library issued equal the oracle policy's replay of the
  same stage / use / release calls.
Sizes: 8B-tier layers (d 4096, 64 experts top-4, I 1024, r 16) at full size,
4 layers x 4 tokens, with 8 slots per layer so that slots get evicted.
"""

import numpy as np
import pytest

import synth
from oracle import slots as o_slots
from tests.gpu_harness import free_running_divergence, teacher_forced_chain

pytestmark = pytest.mark.gpu

L_TEST, T_TEST, SLOTS_TEST = 4, 4, 8


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a visible GPU")
    from paper_2609_18063_amd import binding
    binding.lib()
    return torch


def _layers(wl, L, torch):
    dev, np_layers = [], []
    for n in range(L):
        router = synth.router_weights(wl, n, 0)
        head = synth.router_weights(wl, n, 1)
        mix_d, perm = synth.mixing(wl, n)
        last = n + 1 == L
        dev.append({"router": torch.from_numpy(router).cuda(),
                    "head": None if last else torch.from_numpy(head).cuda(),
                    "mix_d": torch.from_numpy(mix_d).cuda(),
                    "mix_perm": torch.from_numpy(perm).cuda()})
        cache = {}

        def routed(e, n=n, cache=cache):
            if e not in cache:
                cache[e] = synth.bundle(wl, n, e)
            return cache[e]

        np_layers.append({"router": router, "head": None if last else head, "mix_d": mix_d,
                          "mix_perm": perm, "routed": routed,
                          "shared": [synth.bundle(wl, n, wl.E + s) for s in range(wl.S)]})
    return dev, np_layers


@pytest.fixture(scope="module")
def tiered(torch_cuda):
    torch = torch_cuda
    from paper_2609_18063_amd import binding as B, tier
    wl = synth.WORKLOADS["tier8b"]
    spec = B.spec_from_workload(wl)
    layers, np_layers = _layers(wl, L_TEST, torch)
    pool = tier.HostPool(L_TEST, wl.E + wl.S, lambda n, e: synth.bundle(wl, n, e))
    xi = synth.token_draws(wl, 0, T_TEST)
    xi_t = torch.from_numpy(xi).cuda()
    chain = tier.TieredChain(spec, layers, pool, SLOTS_TEST)
    rec = chain.run(xi_t, record=True)
    return {"wl": wl, "spec": spec, "layers": layers, "np_layers": np_layers, "pool": pool,
            "xi": xi, "xi_t": xi_t, "chain": chain, "rec": rec}


def test_tier_status_and_copies(tiered):
    ch = tiered["chain"]
    assert int(ch.status.item()) == 0
    st = ch.stager.stats()
    n_copies = sum(len(c) for *_, c in ch.log)
    assert st["copies"] == n_copies > 0
    assert st["bytes"] == n_copies * tiered["pool"].bundle_bytes
    # every layer of token 0 and layer 0 of every token staged on demand
    kinds = {(t, n): k for t, n, k, _, _ in ch.log}
    for t in range(T_TEST):
        assert kinds[(t, 0)] == "demand"
    for n in range(L_TEST):
        assert kinds[(0, n)] == "demand"
    for t in range(1, T_TEST):
        for n in range(1, L_TEST):
            assert kinds[(t, n)] == "predicted"


def test_tier_copies_equal_oracle_policy(tiered):
    ch = tiered["chain"]
    ref = o_slots.SlotPolicy(L_TEST, tiered["wl"].E + tiered["wl"].S, SLOTS_TEST)
    evictions = 0
    for op in ch.ops:
        if op[0] == "stage":
            _, n, s, copies = op
            occupied = sum(1 for x in ref.table.expert_in[n] if x >= 0)
            want = ref.stage(n, s)
            assert list(copies) == [tuple(c) for c in want], op
            evictions += max(0, occupied + len(want) - SLOTS_TEST)
        elif op[0] == "use":
            ref.use(op[1], op[2])
        else:
            ref.release(op[1])
    assert evictions > 0, "the test should exercise eviction"


def test_tier_slot_bytes_match_host(tiered, torch_cuda):
    ch, pool = tiered["chain"], tiered["pool"]
    torch = torch_cuda
    from paper_2609_18063_amd import binding as B
    checked = 0
    for n in range(L_TEST):
        for e in range(pool.n_ids):
            s = ch.table.lookup(n, e)
            if s < 0:
                continue
            assert torch.equal(ch.slot_bytes(n, s).cpu(), pool.bytes_of(n, e)), (n, e, s)
            checked += 1
    assert checked >= L_TEST * tiered["wl"].K
    del B


def test_tier_matches_resident_chain_bit_exact(tiered, torch_cuda):
    torch = torch_cuda
    from paper_2609_18063_amd import chain as C, tier
    table, keep = tier.resident_table(tiered["spec"], tiered["pool"], tiered["layers"])
    dc = C.DeviceChain(tiered["spec"], table, tiered["layers"])
    ref = dc.run_recorded(tiered["xi_t"])
    rec = tiered["rec"]
    for k in ("x", "r", "r_post", "idx", "w", "pidx", "pw", "ye"):
        assert torch.equal(rec[k], ref[k]), k
    table.close()
    del keep


def test_tier_matches_oracle_chain(tiered):
    """Teacher-forced per-layer parity of the staged chain (every token and
    layer), plus the free-running divergence point as a report."""
    wl = tiered["wl"]
    rec = {k: v.cpu().numpy() for k, v in tiered["rec"].items()}
    stats = teacher_forced_chain(rec, tiered["xi"], tiered["np_layers"], wl, L_TEST, what="tier8b")
    stats["free_running_divergence"] = free_running_divergence(rec, tiered["xi"],
                                                               tiered["np_layers"], wl, L_TEST)
    print("tier8b staged chain:", stats)
    assert stats["steps"] == L_TEST * T_TEST and stats["y_checked"] == L_TEST * T_TEST


def test_tier_close_leaves_no_hip_error(tiered, torch_cuda):
    """Destroying the stager (with sets that needed no copy still queued or
    retired) leaves no error behind for the next HIP call."""
    torch = torch_cuda
    ch = tiered["chain"]
    ch.close()
    x = torch.ones(1024, device="cuda")
    assert float((x * 2).sum().item()) == 2048.0
    torch.cuda.synchronize()
