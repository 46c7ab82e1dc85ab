"""GPU parity of the two-half decode chain with the full prerouter head
(fc1 -> erf-GELU -> fp16 -> fc2 + linear path; §3.2 Head) as every layer's
head, consumed as routing (§3.2 Prediction-as-routing), through
moe_engine_chain_mlp.

Head N at token t sees layer N's x and the routing layer N used at tokens t
and t-1; from layer 1 on those are the chain's own earlier predictions (the
paper's feature drift). Teacher-forced per (token, layer) like the engine
chain tests: on the device's own x and recorded routing, each prediction
must equal the oracle head's except where the oracle's logits are within
1e-4 of their largest magnitude (the kernel rounds its hidden activation to
fp16 after an fp32 pre-activation, the oracle after an exact one; counted);
the layer that routes by a prediction uses exactly the prediction made for
it a token earlier; the stand-in residual, the layer input and the layer
output are held to the chain's usual bars.
"""

import numpy as np
import pytest

import synth
from oracle import routing as o_routing
from tests.gpu_harness import build_chain, sample_layers, teacher_forced_chain

pytestmark = pytest.mark.gpu

LOGIT_TOL = 1e-4


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a visible GPU")
    from paper_2609_18063_amd import binding
    binding.lib()
    return torch


def _heads(wl, L, hidden, torch):
    """Seeded full heads of layers 0 .. L-2 on the device (fp16), their
    moe_head_mlp device array, and the host copies for the oracle."""
    from paper_2609_18063_amd import binding as B
    heads_np, structs, keep = [], [], []
    for n in range(L):
        if n + 1 == L:
            heads_np.append(None)
            structs.append(None)
            continue
        h = synth.prerouter_mlp(wl, n, hidden)
        d = wl.d

        def t(a):
            return torch.from_numpy(np.ascontiguousarray(a)).cuda()

        dev = {"w1_x": t(h["w1"][:, :d]), "w1_r": t(h["w1"][:, d:].T), "w2": t(h["w2"]),
               "b1": t(h["b1"]), "b2": t(h["b2"]), "w_l": t(h["wl"])}
        keep.append(dev)
        heads_np.append(h)
        structs.append(B.head_mlp(hidden, dev["w1_x"], dev["w1_r"], dev["w2"], dev["b1"], dev["b2"],
                                  dev["w_l"]))
    return heads_np, B.head_mlp_array(structs), keep


def _launch(chain, head_arr, hidden, xi, L, torch, first_token=0, ws=None, r_state=None):
    from paper_2609_18063_amd import binding as B
    spec = chain.spec
    d, K = spec.d_model, spec.top_k
    T = xi.shape[0]
    arr = getattr(chain, "engine_arr", None)
    if arr is None:
        arr = B.engine_layer_array(chain.layers)
        chain.engine_arr = arr
    if ws is None:
        ws = torch.zeros(B.engine_workspace_bytes(spec, L), dtype=torch.uint8, device="cuda")
    if r_state is None:
        r_state = torch.zeros(d, dtype=torch.float32, device="cuda")
    n = T * L
    rec = {
        "x": torch.zeros(n, d, dtype=torch.float16, device="cuda"),
        "r": torch.zeros(n, d, dtype=torch.float32, device="cuda"),
        "idx": torch.full((n, K), -7, dtype=torch.int32, device="cuda"),
        "w": torch.zeros(n, K, dtype=torch.float32, device="cuda"),
        "pidx": torch.full((n, K), -1, dtype=torch.int32, device="cuda"),
        "pw": torch.zeros(n, K, dtype=torch.float32, device="cuda"),
        "y": torch.zeros(n, d, dtype=torch.float32, device="cuda"),
    }
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    xi_t = torch.from_numpy(np.ascontiguousarray(xi)).cuda()
    print("engine chain, full head: L=%d T=%d H=%d first_token=%d" % (L, T, hidden, first_token), flush=True)
    B.engine_chain_mlp(spec, chain.table, arr, head_arr, hidden, L, first_token, xi_t, r_state, ws,
                       x_rec=rec["x"], r_rec=rec["r"], idx=rec["idx"], w=rec["w"], pidx=rec["pidx"],
                       pw=rec["pw"], y_rec=rec["y"], status=status)
    torch.cuda.synchronize()
    assert int(status.item()) == 0, int(status.item())
    rec = {k: v.view(T, L, *v.shape[1:]) for k, v in rec.items()}
    return rec, ws, r_state


def _check(wl, L, T, hidden, torch, y_at):
    from paper_2609_18063_amd import binding as B
    chain, np_layers = build_chain(wl, L, torch)
    assert B.engine_chain_mlp_supported(chain.spec, hidden)
    heads_np, head_arr, keep = _heads(wl, L, hidden, torch)
    xi = synth.token_draws(wl, 0, T)
    rec, _, _ = _launch(chain, head_arr, hidden, xi, L, torch)
    rec = {k: v.cpu().numpy() for k, v in rec.items()}

    def pred_oracle(t, n, x):
        prev = rec["idx"][t - 1, n] if t > 0 else None
        l = o_routing.prerouter_mlp_logits(heads_np[n], x, rec["idx"][t, n], prev)
        return l, LOGIT_TOL * float(np.max(np.abs(l))), LOGIT_TOL

    stats = teacher_forced_chain(rec, xi, np_layers, wl, L, y_at=y_at, what="engine full head " + wl.name,
                                 pred_oracle=pred_oracle)
    print("engine full-head chain %s:" % wl.name, stats)
    assert stats["steps"] == L * T
    assert stats["pred_routing"] == (T - 1) * (L - 1) and stats["predictions"] == T * (L - 1)
    del keep
    chain.table.close()
    return stats


def test_engine_chain_full_head_tiny(torch_cuda):
    _check(synth.WORKLOADS["tiny"], 8, 24, 64, torch_cuda, sample_layers(24, 8, full_tokens=4, per_token=3))


def test_engine_chain_full_head_moe35b(torch_cuda):
    _check(synth.WORKLOADS["moe35b"], 4, 6, 512, torch_cuda, sample_layers(6, 4, full_tokens=1, per_token=1))


def test_engine_chain_full_head_split_launches_match(torch_cuda):
    """Two launches (tokens 0-2, then 3-7 from first_token 3 on the same
    workspace and residual) reproduce one launch of all 8 tokens bit for bit:
    the predictions and the last token's routing words carry over."""
    torch = torch_cuda
    wl = synth.WORKLOADS["tiny"]
    L, T, H = 6, 8, 128
    chain, _ = build_chain(wl, L, torch)
    _, head_arr, keep = _heads(wl, L, H, torch)
    xi = synth.token_draws(wl, 0, T)
    one, _, _ = _launch(chain, head_arr, H, xi, L, torch)
    a, ws, r_state = _launch(chain, head_arr, H, xi[:3], L, torch)
    b, _, _ = _launch(chain, head_arr, H, xi[3:], L, torch, first_token=3, ws=ws, r_state=r_state)
    for k in one:  # bit for bit
        both = torch.cat([a[k], b[k]], dim=0).contiguous().view(torch.uint8)
        assert torch.equal(both, one[k].contiguous().view(torch.uint8)), k
    del keep
    chain.table.close()


def test_engine_chain_full_head_refuses(torch_cuda):
    from paper_2609_18063_amd import binding as B
    moe35b = B.spec_from_workload(synth.WORKLOADS["moe35b"])
    assert B.engine_chain_mlp_supported(moe35b, 512)
    assert not B.engine_chain_mlp_supported(moe35b, 96)       # not a multiple of 64
    assert not B.engine_chain_mlp_supported(moe35b, 1024)     # larger than the rows LDS holds
    assert not B.engine_chain_mlp_supported(B.spec_from_workload(synth.WORKLOADS["tier8b"]), 512)  # d 4096
    sg = B.make_spec(2048, 256, 8, 1, 512, 16, 2.0, sigmoid_group=(8, 4, 2.5))
    assert not B.engine_chain_mlp_supported(sg, 512)
