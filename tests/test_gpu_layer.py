"""GPU parity of one MoE layer through the C ABI against the CPU oracle.

Bars: int routing outputs bit-exact (near-ties within 1e-5 counted), layer and
expert outputs within 2e-3 max-relative error, the fp16 layer input
bit-exact.  Sizes: the tiny layer on 64 tokens, the 35B-class layer at full
size on sampled tokens, launched exactly as the benchmark launches it.
"""

import numpy as np
import pytest

import synth
from oracle import expert as o_expert, routing as o_routing
from tests.gpu_harness import (DeviceLayer, TOL_REL_INF, check_routing, oracle_token, rel_inf)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a visible GPU")
    from paper_2609_18063_amd import binding
    binding.lib()
    return torch


@pytest.fixture(scope="module")
def tiny(torch_cuda):
    return DeviceLayer(synth.WORKLOADS["tiny"])


@pytest.fixture(scope="module")
def big(torch_cuda):
    return DeviceLayer(synth.WORKLOADS["moe35b"])


def _alt_routing(logits, k):
    """The oracle's routing with its K-th and (K+1)-th experts swapped."""
    g = o_routing.softmax(logits)
    order = o_routing.topk_desc(g, k + 1)
    inds = np.concatenate([order[:k - 1], order[k:k + 1]])
    return inds, g[inds] / np.sum(g[inds])


def _check_token(dl, out, t, xi_row, stats, what):
    wl = dl.wl
    ref = oracle_token(dl, xi_row)
    assert np.array_equal(out["x"][t].view(np.uint16), ref["x16"].view(np.uint16)), what
    assert np.allclose(out["logits"][t], ref["logits"], rtol=0, atol=2e-6), what
    assert np.allclose(out["plogits"][t], ref["pred_logits"], rtol=0, atol=2e-6), what
    exact = check_routing(out["idx"][t], out["w"][t], ref["logits"], wl.K, what + " route", stats)
    check_routing(out["pidx"][t], out["pw"][t], ref["pred_logits"], wl.K, what + " preroute", stats)
    if not exact:
        ref = oracle_token(dl, xi_row, routing=_alt_routing(ref["logits"], wl.K))
    got_idx = out["idx"][t].tolist()
    for pos, e in enumerate(ref["idx"].tolist()):
        err = rel_inf(out["ye"][t][got_idx.index(e)], ref["y_experts"][pos])
        assert err <= TOL_REL_INF, (what, "expert", e, err)
    for s in range(wl.S):
        err = rel_inf(out["ye"][t][wl.K + s], ref["y_experts"][wl.K + s])
        assert err <= TOL_REL_INF, (what, "shared", s, err)
    err = rel_inf(out["y"][t], ref["y"])
    assert err <= TOL_REL_INF, (what, "y", err)
    stats["max_err"] = max(stats.get("max_err", 0.0), err)
    return err


def test_rmsnorm_bit_exact(torch_cuda):
    torch = torch_cuda
    from paper_2609_18063_amd import binding as B
    rs = np.random.default_rng(7)
    for T, d, scale in ((1, 512, 1.0), (37, 2048, 3.0), (5, 4096, 0.01), (3, 100, 1.0)):
        xi = rs.normal(0, scale, size=(T, d)).astype(np.float32)
        x = torch.empty(T, d, dtype=torch.float16, device="cuda")
        B.rmsnorm_f16(torch.from_numpy(xi).cuda(), x)
        got = x.cpu().numpy()
        ref = o_routing.rms_norm_f16(xi)
        assert np.array_equal(got.view(np.uint16), ref.view(np.uint16)), (T, d)


def test_tiny_layer_64_tokens(tiny):
    wl = tiny.wl
    xi = synth.token_draws(wl, 0, 64)
    out = tiny.run(xi)
    stats = {}
    for t in range(64):
        _check_token(tiny, out, t, xi[t], stats, "tiny t=%d" % t)
    assert out["status"][0] == 0
    print("tiny layer: max rel err %.3g, near ties %s" % (stats["max_err"], stats))


def test_tiny_layer_single_token_seed0(tiny):
    """The tiny workload's decode token (seed 0) as a T = 1 call."""
    xi = synth.token_draws(tiny.wl, 0, 1)
    out = tiny.run(xi)
    _check_token(tiny, out, 0, xi[0], {}, "tiny seed0")


def test_big_layer_sampled_tokens(big):
    """35B-class layer at full size (256 experts + 1 shared), one T = 1 call
    per token as the benchmark does."""
    wl = big.wl
    bufs = big.alloc(1)
    stats = {}
    for t in (0, 1, 2, 997):
        xi = synth.token_draws(wl, t, 1)
        out = big.run(xi, bufs=bufs)
        _check_token(big, out, 0, xi[0], stats, "moe35b t=%d" % t)
        assert out["status"][0] == 0
    print("moe35b layer: max rel err %.3g, near ties %s" % (stats["max_err"], stats))


def test_big_layer_batch_of_tokens(big):
    """T = 3 tokens in one call (one grid row per token)."""
    xi = synth.token_draws(big.wl, 100, 3)
    out = big.run(xi)
    stats = {}
    for t in range(3):
        _check_token(big, out, t, xi[t], stats, "moe35b batch t=%d" % t)


def test_ffn_given_routing_with_repeats(tiny):
    """Expert list given directly (including a repeated expert)."""
    wl = tiny.wl
    xi = synth.token_draws(wl, 5, 2)
    idx = np.array([[3, 3], [15, 0]], dtype=np.int32)
    out = tiny.run(xi, idx_override=idx)
    for t in range(2):
        x16 = o_routing.rms_norm_f16(xi[t])
        for pos, e in enumerate(idx[t]):
            ref, _ = o_expert.expert_forward(tiny.bundle_np(int(e)), x16, wl.lora_scale)
            assert rel_inf(out["ye"][t][pos], ref) <= TOL_REL_INF


def test_status_bad_index_and_slot_miss(tiny, torch_cuda):
    torch = torch_cuda
    from paper_2609_18063_amd import binding as B, weights as W
    wl = tiny.wl
    # a table where expert 4 is not resident
    table = B.SlotTable(1, tiny.n_ids, tiny.n_ids)
    for e in range(tiny.n_ids):
        table.bind(0, e, int(tiny.perm[e]), tiny.mbundles[e], keep=tiny.dev)
    table.unbind(0, 4)
    table.sync()
    bufs = tiny.alloc(3)
    xi = torch.from_numpy(synth.token_draws(wl, 9, 3)).cuda()
    B.rmsnorm_f16(xi, bufs["x"])
    idx = torch.tensor([[4, 1], [16, 2], [-1, 3]], dtype=torch.int32, device="cuda")
    B.expert_ffn(tiny.spec, table, 0, bufs["x"], idx, bufs["ye"], bufs["status"], bufs["ws"])
    torch.cuda.synchronize()
    status = int(bufs["status"].item())
    assert status == (B.MOE_STATUS_SLOT_MISS | B.MOE_STATUS_BAD_INDEX)
    ye = bufs["ye"].cpu().numpy()
    for t in range(3):
        assert np.all(ye[t][0] == 0)
    x16 = bufs["x"].cpu().numpy()
    for t, e in ((0, 1), (1, 2), (2, 3)):
        ref, _ = o_expert.expert_forward(tiny.bundle_np(e), x16[t], wl.lora_scale)
        assert rel_inf(ye[t][1], ref) <= TOL_REL_INF
    assert table.lookup(0, 4) == -1
    table.close()


def test_zero_adapter_bit_exact_on_gpu(torch_cuda):
    """B = 0 in every adapter reproduces the no-adapter output bit for bit."""
    torch = torch_cuda
    from paper_2609_18063_amd import binding as B, weights as W
    wl = synth.WORKLOADS["tiny"]
    ids = wl.E + wl.S
    plain = [synth.bundle(wl, 0, e, lora=False) for e in range(ids)]
    zero_b = []
    for e in range(ids):
        b = synth.bundle(wl, 0, e)
        b["lora"] = {p: (a, np.zeros_like(bb)) for p, (a, bb) in b["lora"].items()}
        zero_b.append(b)
    outs = []
    xi = torch.from_numpy(synth.token_draws(wl, 0, 4)).cuda()
    for bundles in (plain, zero_b):
        buf, boffs, _ = W.pack_host(bundles)
        dev = W.upload(buf)
        table = B.SlotTable(1, ids, ids)
        W.bind_layer(table, 0, dev, boffs)
        table.sync()
        spec = B.spec_from_workload(wl)
        ws = torch.zeros(B.workspace_bytes(spec, 4), dtype=torch.uint8, device="cuda")
        x = torch.empty(4, wl.d, dtype=torch.float16, device="cuda")
        B.rmsnorm_f16(xi, x)
        idx = torch.tensor([[0, 5], [7, 2], [15, 9], [1, 14]], dtype=torch.int32, device="cuda")
        ye = torch.empty(4, wl.K + wl.S, wl.d, dtype=torch.float32, device="cuda")
        st = torch.zeros(1, dtype=torch.int32, device="cuda")
        B.expert_ffn(spec, table, 0, x, idx, ye, st, ws)
        torch.cuda.synchronize()
        outs.append(ye.cpu().numpy())
        table.close()
        del dev
    assert np.array_equal(outs[0], outs[1])


def test_k_equals_e_full_softmax(torch_cuda):
    torch = torch_cuda
    from paper_2609_18063_amd import binding as B
    wl = synth.Workload(0, "tiny_k16", 512, 16, 16, 0, 256, 8)
    spec = B.spec_from_workload(wl)
    router = synth.router_weights(wl, 0, 0)
    xi = synth.token_draws(wl, 0, 8)
    x16 = o_routing.rms_norm_f16(xi)
    x = torch.from_numpy(x16).cuda()
    w_r = torch.from_numpy(router).cuda()
    ws = torch.zeros(B.workspace_bytes(spec, 8), dtype=torch.uint8, device="cuda")
    idx = torch.empty(8, 16, dtype=torch.int32, device="cuda")
    w = torch.empty(8, 16, dtype=torch.float32, device="cuda")
    B.route(spec, x, w_r, idx, w, ws)
    torch.cuda.synchronize()
    stats = {}
    for t in range(8):
        l = o_routing.logits_fp32(router, x16[t])
        check_routing(idx[t].cpu().numpy(), w[t].cpu().numpy(), l, 16, "k=e", stats)
        assert abs(float(w[t].sum()) - 1.0) < 1e-5


def test_topk_given_logits_ties_and_order(torch_cuda):
    torch = torch_cuda
    from paper_2609_18063_amd import binding as B
    spec = B.make_spec(512, 8, 4, 0, 256, 8, 2.0)
    logits = np.array([[1.0, 3.0, 3.0, 2.0, 3.0, -1.0, 0.0, 2.0],
                       [0.0] * 8,
                       [-np.inf, 5.0, -np.inf, 4.0, 4.0, 4.0, -np.inf, -np.inf]], dtype=np.float32)
    lt = torch.from_numpy(logits).cuda()
    idx = torch.empty(3, 4, dtype=torch.int32, device="cuda")
    w = torch.empty(3, 4, dtype=torch.float32, device="cuda")
    B.topk(spec, lt, idx, w)
    torch.cuda.synchronize()
    for t in range(3):
        ri, rw = o_routing.softmax_topk(logits[t], 4)
        assert idx[t].cpu().tolist() == ri.tolist()
        assert np.allclose(w[t].cpu().numpy(), rw, rtol=2e-6)


def test_zero_tokens_is_noop(tiny, torch_cuda):
    torch = torch_cuda
    from paper_2609_18063_amd import binding as B
    bufs = tiny.alloc(1)
    e = torch.empty(0, tiny.wl.d, dtype=torch.float16, device="cuda")
    e32 = torch.empty(0, tiny.wl.d, dtype=torch.float32, device="cuda")
    i0 = torch.empty(0, tiny.wl.K, dtype=torch.int32, device="cuda")
    B.rmsnorm_f16(e32, e)
    B.expert_ffn(tiny.spec, tiny.table, 0, e, i0, bufs["ye"], bufs["status"], bufs["ws"])
    torch.cuda.synchronize()


def test_deterministic(tiny):
    xi = synth.token_draws(tiny.wl, 20, 4)
    a = tiny.run(xi)
    b = tiny.run(xi)
    for k in ("y", "ye", "idx", "w", "pidx", "pw", "logits"):
        assert np.array_equal(a[k], b[k]), k
