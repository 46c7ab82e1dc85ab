"""GPU tests of the whole-layer prefill path (every expert of a layer loaded
in one shot into one of two device layer buffers, the next layer's load
overlapping this layer's compute).

* Bit-identical to the same computation with every layer resident (loading
  moves bytes; it must not change a result), from the pinned pool and from
  the file.
* Teacher-forced parity with the oracle on every layer: on the device's own
  layer input x (checked bit for bit against fp16(rmsnorm(r))), the routing
  is bit-exact except at counted near-ties (oracle K-th / (K+1)-th logit gap
  within 1e-5), and the layer output r_{N+1} - r_N is within 2e-3 of the
  oracle's batched layer.
Sizes: the tiny layer (d 512, 16 experts top-2), 4 layers, 37 tokens; and
the 8B-tier layer (d 4096, 64 experts top-4, I 1024) over 2 layers and 64
tokens, whose layer loads are 485 MB each.
"""

import os

import numpy as np
import pytest

import synth
from oracle import batched as o_batched, routing as o_routing
from tests.gpu_harness import TOL_REL_INF, _x_flip_is_tie, check_routing, rel_inf

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a visible GPU")
    from paper_2609_18063_amd import binding
    binding.lib()
    return torch


def _setup(wl, L, T, torch, tmp_path=None):
    from paper_2609_18063_amd import binding as B, tier
    spec = B.spec_from_workload(wl)
    n_ids = wl.E + wl.S
    routers_np = [synth.router_weights(wl, n, 0) for n in range(L)]
    routers = [torch.from_numpy(r).cuda() for r in routers_np]
    pool = tier.HostPool(L, n_ids, lambda n, e: synth.bundle(wl, n, e))
    fpool = None
    if tmp_path is not None:
        fpool = tier.FilePool(os.path.join(str(tmp_path), "layers.bin"), L, n_ids,
                              lambda n, e: synth.bundle(wl, n, e))
    xi = torch.from_numpy(synth.token_draws(wl, 700, T)).cuda()
    return spec, routers_np, routers, pool, fpool, xi


def _run(tier, spec, routers, pool, xi, torch, resident=False, record=False):
    ex = tier.WholeLayerPrefill(spec, routers, pool, resident=resident)
    try:
        r, rec = ex.run(xi, record=record)
        torch.cuda.synchronize()
        assert int(ex.status.item()) == 0, int(ex.status.item())
        out = r.cpu().numpy()
        if rec is not None:
            rec = {k: [v.cpu().numpy() for v in vs] for k, vs in rec.items()}
    finally:
        ex.close()
    return out, rec


def test_whole_layer_tiny_bit_identical_and_oracle(torch_cuda, tmp_path):
    from paper_2609_18063_amd import tier
    torch = torch_cuda
    wl, L, T = synth.WORKLOADS["tiny"], 4, 37
    spec, routers_np, routers, pool, fpool, xi = _setup(wl, L, T, torch, tmp_path)
    print("whole-layer prefill tiny: L=%d T=%d" % (L, T), flush=True)
    r_whole, rec = _run(tier, spec, routers, pool, xi, torch, record=True)
    r_res, _ = _run(tier, spec, routers, pool, xi, torch, resident=True)
    r_file, _ = _run(tier, spec, routers, fpool, xi, torch)
    fpool.remove()
    assert np.array_equal(r_whole.view(np.uint32), r_res.view(np.uint32))
    assert np.array_equal(r_file.view(np.uint32), r_res.view(np.uint32))
    stats = {"routing_near_ties": {}}
    worst = 0.0
    for n in range(L):
        r_in = rec["r"][n]
        x = rec["x"][n]
        for t in range(T):   # the layer input: fp16(rmsnorm(r)) bit for bit, rounding ties aside
            x_ref = o_routing.rms_norm_f16(r_in[t])
            for j in np.nonzero(x[t].view(np.uint16) != x_ref.view(np.uint16))[0]:
                assert _x_flip_is_tie(r_in[t], j, x[t][j], x_ref[j]), (n, t, int(j))
        logits = np.stack([o_routing.logits_fp32(routers_np[n], x[t]) for t in range(T)])
        for t in range(T):
            check_routing(rec["idx"][n][t], rec["w"][n][t], logits[t], wl.K, ("whole", n, t), stats)
        ref = o_batched.batched_layer(x, logits, wl.K, lambda e, n=n: synth.bundle(wl, n, e),
                                      [synth.bundle(wl, n, wl.E + s) for s in range(wl.S)], wl.lora_scale)
        r_out = rec["r"][n + 1] if n + 1 < L else r_whole
        y = r_out.astype(np.float64) - r_in.astype(np.float64)
        err = rel_inf(y, ref["y"])
        worst = max(worst, err)
        assert err <= TOL_REL_INF, (n, err)
    print("whole-layer prefill tiny: max layer error %.2e, near-ties %s" % (worst, stats["routing_near_ties"]),
          flush=True)


def test_whole_layer_8b_tier_bit_identical(torch_cuda):
    from paper_2609_18063_amd import tier
    torch = torch_cuda
    wl, L, T = synth.WORKLOADS["tier8b"], 2, 64
    spec, routers_np, routers, pool, _, xi = _setup(wl, L, T, torch)
    print("whole-layer prefill 8B tier: L=%d T=%d" % (L, T), flush=True)
    r_whole, rec = _run(tier, spec, routers, pool, xi, torch, record=True)
    r_res, _ = _run(tier, spec, routers, pool, xi, torch, resident=True)
    assert np.array_equal(r_whole.view(np.uint32), r_res.view(np.uint32))
    # the last layer against the oracle on two of its tokens
    n = L - 1
    x = rec["x"][n]
    toks = [0, T - 1]
    logits = np.stack([o_routing.logits_fp32(routers_np[n], x[t]) for t in range(T)])
    stats = {"routing_near_ties": {}}
    for t in toks:
        check_routing(rec["idx"][n][t], rec["w"][n][t], logits[t], wl.K, ("whole8b", n, t), stats)
    ref = o_batched.batched_layer(x, logits, wl.K, lambda e: synth.bundle(wl, n, e), [], wl.lora_scale,
                                  tokens=toks)
    y = r_whole.astype(np.float64) - rec["r"][n].astype(np.float64)
    err = rel_inf(y[toks], ref["y"][toks])
    print("whole-layer prefill 8B tier: last-layer error %.2e on tokens %s" % (err, toks), flush=True)
    assert err <= TOL_REL_INF, err
