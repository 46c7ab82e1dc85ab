"""GPU parity of the batched / prefill expert path (tokens grouped by expert,
MFMA contractions) against the CPU oracle.

The routing comes from Zipf-popularity logits through the device softmax-top-k
(bit-exact against the oracle, near-ties counted); the layer input is the
device RMSNorm of seeded draws.  Every computed token's layer output is held
to the 2e-3 max-relative bar against the oracle's per-token layer (the oracle
loops over tokens; grouping is the kernels' business).  Sizes: the tiny layer
on ragged batches checked in full; the 35B-class layer at T = 64 and T = 512,
launched as the benchmark launches it, on sampled tokens that cover the
largest groups, their ragged last tiles and the shared expert's tiles.
"""

import numpy as np
import pytest

import synth
from oracle import expert as o_expert, routing as o_routing
from tests.gpu_harness import DeviceLayer, TOL_REL_INF, check_routing, rel_inf

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


def _run(dl, torch, xi, logits=None, idx=None, table=None, status=None):
    """Device: rmsnorm -> top-k on the given logits (or the given idx) ->
    grouped experts -> combine.  Returns host copies."""
    from paper_2609_18063_amd import binding as B
    wl = dl.wl
    T = xi.shape[0]
    n = wl.K + wl.S
    ws = torch.zeros(B.workspace_bytes(dl.spec, T), dtype=torch.uint8, device="cuda")
    x = torch.empty(T, wl.d, dtype=torch.float16, device="cuda")
    B.rmsnorm_f16(torch.from_numpy(np.ascontiguousarray(xi)).cuda(), x)
    w = torch.zeros(T, wl.K, dtype=torch.float32, device="cuda")
    if idx is None:
        idx_t = torch.empty(T, wl.K, dtype=torch.int32, device="cuda")
        B.topk(dl.spec, torch.from_numpy(np.ascontiguousarray(logits)).cuda(), idx_t, w)
    else:
        idx_t = torch.from_numpy(np.ascontiguousarray(idx, dtype=np.int32)).cuda()
        w.fill_(1.0 / wl.K)
    ye = torch.full((T, n, wl.d), float("nan"), dtype=torch.float32, device="cuda")
    y = torch.empty(T, wl.d, dtype=torch.float32, device="cuda")
    st = status if status is not None else torch.zeros(1, dtype=torch.int32, device="cuda")
    B.expert_ffn_grouped(dl.spec, table or dl.table, 0, x, idx_t, ye, st, ws)
    B.combine(dl.spec, ye, w, y)
    torch.cuda.synchronize()
    return {"x": x.cpu().numpy(), "idx": idx_t.cpu().numpy(), "w": w.cpu().numpy(),
            "ye": ye.cpu().numpy(), "y": y.cpu().numpy(), "status": int(st.item())}


def _check_tokens(dl, out, logits, tokens, what, stats):
    """Oracle layer per token, on the device's x (checked bit-exact against
    the oracle's RMSNorm of the same draws separately) and on the oracle's
    own routing of the same logits."""
    wl = dl.wl
    shared = [dl.bundle_np(wl.E + s) for s in range(wl.S)]
    for t in tokens:
        ref_idx, ref_w = o_routing.softmax_topk(logits[t], wl.K)
        exact = check_routing(out["idx"][t], out["w"][t], logits[t], wl.K, what, stats)
        routing = (ref_idx, ref_w) if exact else (out["idx"][t], out["w"][t])
        ref = o_expert.moe_layer(out["x"][t], wl.K, dl.bundle_np, shared, wl.lora_scale,
                                 routing=routing)
        got_idx = out["idx"][t].tolist()
        for pos, e in enumerate(np.asarray(routing[0]).tolist()):
            err = rel_inf(out["ye"][t][got_idx.index(e)], ref["y_experts"][pos])
            assert err <= TOL_REL_INF, (what, t, "expert", e, err)
        for s in range(wl.S):
            err = rel_inf(out["ye"][t][wl.K + s], ref["y_experts"][wl.K + s])
            assert err <= TOL_REL_INF, (what, t, "shared", s, err)
        err = rel_inf(out["y"][t], ref["y"])
        assert err <= TOL_REL_INF, (what, t, "y", err)
        stats["max_err"] = max(stats.get("max_err", 0.0), err)
        stats["tokens"] = stats.get("tokens", 0) + 1


def _x_bit_exact(out, xi):
    for t in range(xi.shape[0]):
        ref = o_routing.rms_norm_f16(xi[t])
        assert np.array_equal(out["x"][t].view(np.uint16), ref.view(np.uint16)), t


def _sample_tokens(idx, E, rows_per_tile=64, extra=()):
    """Tokens that land in the largest groups (first and last tile rows) plus
    a few spread ones."""
    T, K = idx.shape
    counts = np.bincount(idx[idx >= 0].ravel(), minlength=E)
    big = np.argsort(-counts, kind="stable")[:2]
    picks = set(extra)
    for e in big:
        rows = [t for t in range(T) if e in idx[t]]
        picks.update([rows[0], rows[-1]])
        if len(rows) > rows_per_tile:
            picks.add(rows[rows_per_tile])   # first row of the second tile (row order is free;
            # any row of a multi-tile group lands in some tile)
    picks.update([0, T // 2, T - 1])
    return sorted(picks)


@pytest.mark.parametrize("T", [1, 37, 200])
def test_tiny_batched_all_tokens(tiny, torch_cuda, T):
    wl = tiny.wl
    xi = synth.token_draws(wl, 50 + T, T)
    logits = synth.zipf_logits(wl, T, seed=T)
    out = _run(tiny, torch_cuda, xi, logits=logits)
    assert out["status"] == 0
    _x_bit_exact(out, xi)
    stats = {}
    _check_tokens(tiny, out, logits, range(T), f"tiny T={T}", stats)
    print(f"tiny batched T={T}:", stats)


def test_tiny_tile_boundaries(tiny, torch_cuda):
    """Groups of exactly 64 rows, 65 rows (a one-row second tile), 129 rows
    (tiles of 64, 64 and 1) and single rows; other experts empty."""
    wl = tiny.wl
    T = 130
    idx = np.zeros((T, wl.K), dtype=np.int32)
    idx[:, 0] = 3
    idx[:64, 1] = 5
    idx[64:129, 1] = 9
    idx[129, 1] = 12
    idx[0, 0] = 7      # 3 then has 129 rows (three tiles: 64, 64, 1); 7 has one
    xi = synth.token_draws(wl, 77, T)
    out = _run(tiny, torch_cuda, xi, idx=idx)
    assert out["status"] == 0
    for t in range(T):
        for k in range(wl.K):
            ref, _ = o_expert.expert_forward(tiny.bundle_np(int(idx[t, k])), out["x"][t], wl.lora_scale)
            err = rel_inf(out["ye"][t][k], ref)
            assert err <= TOL_REL_INF, (t, k, err)


def test_batched_matches_decode_path(tiny, torch_cuda):
    """The grouped path and the one-token path agree within the layer bar on
    the same inputs (both are also held to the oracle)."""
    from paper_2609_18063_amd import binding as B
    torch = torch_cuda
    wl = tiny.wl
    T = 24
    xi = synth.token_draws(wl, 91, T)
    logits = synth.zipf_logits(wl, T, seed=5)
    out = _run(tiny, torch, xi, logits=logits)
    bufs = tiny.alloc(T)
    x = torch.from_numpy(out["x"]).cuda()
    idx = torch.from_numpy(out["idx"]).cuda()
    B.expert_ffn(tiny.spec, tiny.table, 0, x, idx, bufs["ye"], bufs["status"], bufs["ws"])
    torch.cuda.synchronize()
    ye = bufs["ye"].cpu().numpy()
    for t in range(T):
        for k in range(wl.K + wl.S):
            assert rel_inf(out["ye"][t][k], ye[t][k]) <= TOL_REL_INF


def test_batched_status_bad_index_and_slot_miss(tiny, torch_cuda):
    torch = torch_cuda
    from paper_2609_18063_amd import binding as B
    wl = tiny.wl
    table = B.SlotTable(1, tiny.n_ids, tiny.n_ids)
    for e in range(tiny.n_ids):
        table.bind(0, e, int(tiny.perm[e]), tiny.mbundles[e], keep=tiny.dev)
    table.unbind(0, 4)
    table.sync()
    idx = np.array([[4, 1], [16, 2], [-1, 3], [4, 4]], dtype=np.int32)
    xi = synth.token_draws(wl, 9, 4)
    out = _run(tiny, torch, xi, idx=idx, table=table)
    assert out["status"] == (B.MOE_STATUS_SLOT_MISS | B.MOE_STATUS_BAD_INDEX)
    for t, k in ((0, 0), (1, 0), (2, 0), (3, 0), (3, 1)):
        assert np.all(out["ye"][t][k] == 0), (t, k)
    for t, e in ((0, 1), (1, 2), (2, 3)):
        ref, _ = o_expert.expert_forward(tiny.bundle_np(e), out["x"][t], wl.lora_scale)
        assert rel_inf(out["ye"][t][1], ref) <= TOL_REL_INF
    table.close()


def test_batched_zero_adapter_bit_exact(torch_cuda):
    """B = 0 in every adapter reproduces the no-adapter output bit for bit."""
    torch = torch_cuda
    from paper_2609_18063_amd import binding as B, weights as W
    wl = synth.WORKLOADS["tiny"]
    ids = wl.E + wl.S
    T = 40
    logits = torch.from_numpy(synth.zipf_logits(wl, T, seed=3)).cuda()
    xi = torch.from_numpy(synth.token_draws(wl, 0, T)).cuda()
    outs = []
    for zero in (False, True):
        bundles = []
        for e in range(ids):
            b = synth.bundle(wl, 0, e, lora=zero)
            if zero:
                b["lora"] = {p: (a, np.zeros_like(bb)) for p, (a, bb) in b["lora"].items()}
            bundles.append(b)
        buf, boffs, _ = W.pack_host(bundles)
        dev = W.upload(buf)
        table = B.SlotTable(1, ids, ids)
        W.bind_layer(table, 0, dev, boffs)
        table.sync()
        spec = B.spec_from_workload(wl)
        ws = torch.zeros(B.workspace_bytes(spec, T), dtype=torch.uint8, device="cuda")
        x = torch.empty(T, wl.d, dtype=torch.float16, device="cuda")
        B.rmsnorm_f16(xi, x)
        idx = torch.empty(T, wl.K, dtype=torch.int32, device="cuda")
        w = torch.empty(T, wl.K, dtype=torch.float32, device="cuda")
        B.topk(spec, logits, idx, w)
        ye = torch.empty(T, wl.K + wl.S, wl.d, dtype=torch.float32, device="cuda")
        st = torch.zeros(1, dtype=torch.int32, device="cuda")
        B.expert_ffn_grouped(spec, table, 0, x, idx, ye, st, ws)
        torch.cuda.synchronize()
        outs.append(ye.cpu().numpy())
        table.close()
        del dev
    assert np.array_equal(outs[0], outs[1])


def test_batched_deterministic(tiny, torch_cuda):
    wl = tiny.wl
    T = 150
    xi = synth.token_draws(wl, 3, T)
    logits = synth.zipf_logits(wl, T, seed=11)
    a = _run(tiny, torch_cuda, xi, logits=logits)
    b = _run(tiny, torch_cuda, xi, logits=logits)
    assert np.array_equal(a["ye"].view(np.uint32), b["ye"].view(np.uint32))


@pytest.mark.parametrize("T", [64, 512])
def test_big_batched_sampled_tokens(big, torch_cuda, T):
    wl = big.wl
    xi = synth.token_draws(wl, 300 + T, T)
    logits = synth.zipf_logits(wl, T, seed=T)
    out = _run(big, torch_cuda, xi, logits=logits)
    assert out["status"] == 0
    _x_bit_exact(out, xi[:8])
    assert np.isfinite(out["ye"]).all()
    stats = {}
    # routing of every token against the oracle
    for t in range(T):
        check_routing(out["idx"][t], out["w"][t], logits[t], wl.K, f"big T={T} route", stats)
    tokens = _sample_tokens(out["idx"], wl.E)
    _check_tokens(big, out, logits, tokens, f"big T={T}", stats)
    print(f"big batched T={T}:", stats, "tokens", tokens)


def test_grouped_rejects_unsupported(torch_cuda):
    from paper_2609_18063_amd import binding as B
    torch = torch_cuda
    spec = B.make_spec(512, 16, 2, 0, 256, 32, 2.0)   # rank 32 > 16
    table = B.SlotTable(1, 16, 16)
    table.sync()
    x = torch.zeros(2, 512, dtype=torch.float16, device="cuda")
    idx = torch.zeros(2, 2, dtype=torch.int32, device="cuda")
    ye = torch.zeros(2, 2, 512, dtype=torch.float32, device="cuda")
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    ws = torch.zeros(B.workspace_bytes(spec, 2), dtype=torch.uint8, device="cuda")
    with pytest.raises(B.MoeError) as err:
        B.expert_ffn_grouped(spec, table, 0, x, idx, ye, st, ws)
    assert err.value.code == B.MOE_EINVAL
    table.close()
