"""GPU parity of moe_merge_requantize and the merge-vs-unmerged retention
measured through the C ABI (§3.3, Recovery LoRA: the merged alternative).

Bit-exact: the merged codes, scales and zeros against the oracle.  The
device computes every value that decides a code exactly as the oracle does:
the delta's products of fp16 factors and their sums are exact in float64
(all bits lie within 2^1 .. 2^-48), so is ``w + delta``; the one fp32
rounding, the min / max, the fp16 conversions, the fp32 division and the
round-half-to-even are the same IEEE operations on both sides.  The per-group
sums of the weight measure are compared at rtol 1e-12 (summation order).

Retention: the unmerged (U), merged (M) and base (B) experts run through
moe_expert_ffn_int4_lora; each output is held to the layer bar against the
oracle, and the output-level retention computed from the device outputs must
lie within the bound that the measured output errors put on it.
"""

import numpy as np
import pytest

import synth
from oracle import retention as RT, routing as o_routing
from tests.gpu_harness import rel_inf, TOL_REL_INF

pytestmark = pytest.mark.gpu


def _merge_on_device(qsz, lora, out_dim, in_dim, rank, scale):
    import torch
    from paper_2609_18063_amd import binding as B
    proj, keep = B.upload_projection(qsz, lora, "cuda")
    q_out = torch.empty(out_dim, in_dim // 2, dtype=torch.uint8, device="cuda")
    sz_out = torch.empty(out_dim, in_dim // 64, 2, dtype=torch.float16, device="cuda")
    stats = torch.empty(out_dim, in_dim // 64, 2, dtype=torch.float64, device="cuda")
    B.merge_requantize(proj, out_dim, in_dim, rank, scale, q_out, sz_out, stats)
    torch.cuda.synchronize()
    return q_out, sz_out, stats, keep


def _check_merge(qsz, lora, scale, what):
    out_dim, in_dim = qsz[0].shape[0], qsz[0].shape[1] * 2
    rank = 0 if lora is None else lora[0].shape[0]
    q_out, sz_out, stats, _ = _merge_on_device(qsz, lora, out_dim, in_dim, rank, scale)
    if lora is None:
        (qp, s, z), actual = RT.requantize_with(qsz, np.zeros((out_dim, in_dim)))
        delta = np.zeros((out_dim, in_dim))
    else:
        (qp, s, z), delta, actual = RT.merge_requantize(qsz, lora, scale)
    got_q = q_out.cpu().numpy()
    got_sz = sz_out.cpu().numpy()
    assert np.array_equal(got_q, qp), (what, int(np.sum(got_q != qp)))
    assert np.array_equal(got_sz[..., 0].view(np.uint16), s.view(np.uint16)), what
    assert np.array_equal(got_sz[..., 1].view(np.uint16), z.view(np.uint16)), what
    st = stats.cpu().numpy()
    sa, sd = float(st[..., 0].sum()), float(st[..., 1].sum())
    ra, rd = float(np.sum(actual * delta)), float(np.sum(delta * delta))
    assert abs(sa - ra) <= 1e-12 * max(abs(ra), 1e-300) + 1e-300, (what, sa, ra)
    assert abs(sd - rd) <= 1e-12 * max(rd, 1e-300) + 1e-300, (what, sd, rd)
    return (qp, s, z), delta, actual


@pytest.mark.parametrize("wname,b_std", [("tiny", None), ("moe35b", None), ("moe35b", "paper")])
def test_merge_bit_exact(wname, b_std):
    wl = synth.WORKLOADS[wname]
    if b_std == "paper":   # delta entries of std 1e-3
        b_std = 1e-3 / (wl.lora_scale * np.sqrt(wl.r) * wl.a_std)
    b = synth.bundle(wl, 0, 5, b_std=b_std)
    for p in ("gate", "up", "down"):
        _check_merge(b[p], b["lora"][p], wl.lora_scale, (wname, p))


def test_merge_ragged_no_adapter_and_large_delta():
    # 33 rows x 3 groups: 99 groups, a partial last workgroup
    qsz = synth.int4_projection((9, 0, 1, 1), (9, 0, 1, 2), 33, 192)
    _check_merge(qsz, None, 2.0, "plain requantization")
    a, bb = synth.lora_pair((9, 0, 1, 3), (9, 0, 1, 4), 33, 192, 5, 0.3, 0.5)
    _, delta, actual = _check_merge(qsz, (a, bb), 1.5, "large delta")
    assert RT.weight_retention(actual, delta) > 0.9
    # one row, one group
    qsz1 = synth.int4_projection((9, 0, 2, 1), (9, 0, 2, 2), 1, 64)
    a1, b1 = synth.lora_pair((9, 0, 2, 3), (9, 0, 2, 4), 1, 64, 1, 0.25, 0.01)
    _check_merge(qsz1, (a1, b1), 2.0, "1x64")


def _bundle_from(projs):
    from paper_2609_18063_amd import binding as B
    return B.MoeBundle(projs["gate"], projs["up"], projs["down"])


@pytest.mark.parametrize("wname", ["tiny", "moe35b"])
def test_output_retention_through_the_c_abi(wname):
    import torch
    from paper_2609_18063_amd import binding as B
    wl = synth.WORKLOADS[wname]
    b_std = 1e-3 / (wl.lora_scale * np.sqrt(wl.r) * wl.a_std)
    bundle = synth.bundle(wl, 0, 7, b_std=b_std)
    keep, U, M, Bs = [], {}, {}, {}
    dims = {"gate": (wl.I, wl.d), "up": (wl.I, wl.d), "down": (wl.d, wl.I)}
    for p, (o, i) in dims.items():
        U[p], k1 = B.upload_projection(bundle[p], bundle["lora"][p], "cuda")
        Bs[p], k2 = B.upload_projection(bundle[p], None, "cuda")
        q_out, sz_out, _, k3 = _merge_on_device(bundle[p], bundle["lora"][p], o, i, wl.r,
                                                wl.lora_scale)
        M[p] = B.MoeProj(q_out.data_ptr(), sz_out.data_ptr(), None, None)
        keep += [k1, k2, k3, q_out, sz_out]
    spec = B.make_spec(wl.d, 8, 3, 0, wl.I, wl.r, wl.lora_scale)
    table = B.SlotTable(1, 8, 8)
    for e, pj in enumerate((U, M, Bs)):
        table.bind(0, e, e, _bundle_from(pj), keep=keep)
    table.sync()
    T = 8
    x16 = np.stack([o_routing.rms_norm_f16(r) for r in synth.token_draws(wl, 0, T)])
    x = torch.from_numpy(x16).cuda()
    idx = torch.tensor([[0, 1, 2]] * T, dtype=torch.int32, device="cuda")
    ye = torch.empty(T, 3, wl.d, dtype=torch.float32, device="cuda")
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    ws = torch.zeros(B.workspace_bytes(spec, T), dtype=torch.uint8, device="cuda")
    B.expert_ffn(spec, table, 0, x, idx, ye, status, ws)
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    got = ye.cpu().numpy().astype(np.float64)
    ref = RT.expert_retention(bundle, x16, wl.lora_scale)
    for j, key in enumerate(("U", "M", "B")):
        assert rel_inf(got[:, j], ref[key]) <= TOL_REL_INF, (wname, key, rel_inf(got[:, j], ref[key]))
    gu, gm, gb = got[:, 0], got[:, 1], got[:, 2]
    r_dev = RT.output_retention(gu, gm, gb)
    eu, em, eb = gu - ref["U"], gm - ref["M"], gb - ref["B"]
    n1 = np.linalg.norm(ref["U"] - ref["M"])
    n2 = np.linalg.norm(ref["U"] - ref["B"])
    e1, e2 = np.linalg.norm(eu - em), np.linalg.norm(eu - eb)
    bound = (e1 * n2 + n1 * e2) / ((n2 - e2) * n2)
    assert bound < 0.05, (wname, bound)
    assert abs(r_dev - ref["output"]) <= bound + 1e-12, (wname, r_dev, ref["output"], bound)
    print("%s: weight retention %s, output retention oracle %.4f device %.4f" % (
        wname, {k: round(v, 4) for k, v in ref["weight"].items()}, ref["output"], r_dev))
    table.close()
