"""GPU test of moe_expert_ffn_int4_lora_noalloc (the expert FFN entry point
that allocates nothing and keeps its intermediate values in the library's
static per-device scratch): through the C ABI, its expert outputs equal those
of moe_expert_ffn_int4_lora with a caller workspace bit for bit, on two calls
in a row (the second with fewer tokens), and a token count beyond the
scratch is refused."""

import numpy as np
import pytest

import synth
from tests.gpu_harness import DeviceLayer

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a visible GPU")
    from paper_2609_18063_amd import binding
    binding.lib()
    return torch


def _routed_inputs(dl, T, t0, torch):
    from paper_2609_18063_amd import binding as B
    wl = dl.wl
    b = dl.alloc(T)
    xi = torch.from_numpy(synth.token_draws(wl, t0, T)).cuda()
    B.rmsnorm_f16(xi, b["x"])
    B.route(dl.spec, b["x"], dl.router_t, b["idx"], b["w"], b["ws"])
    return b


@pytest.mark.parametrize("name", ["tiny", "moe35b"])
def test_noalloc_equals_workspace_entry_point(torch_cuda, name):
    torch = torch_cuda
    from paper_2609_18063_amd import binding as B
    dl = DeviceLayer(synth.WORKLOADS[name])
    n = dl.wl.K + dl.wl.S
    for T, t0 in ((12, 0), (3, 100)):               # the second call has fewer tokens
        b = _routed_inputs(dl, T, t0, torch)
        print("%s: expert_ffn with a workspace and without, T=%d" % (name, T), flush=True)
        B.expert_ffn(dl.spec, dl.table, 0, b["x"], b["idx"], b["ye"], b["status"], b["ws"])
        ye_na = torch.full((T, n, dl.wl.d), float("nan"), dtype=torch.float32, device="cuda")
        st_na = torch.zeros(1, dtype=torch.int32, device="cuda")
        B.expert_ffn_noalloc(dl.spec, dl.table, 0, b["x"], b["idx"], ye_na, st_na)
        torch.cuda.synchronize()
        assert int(b["status"].item()) == 0 and int(st_na.item()) == 0
        assert torch.equal(ye_na, b["ye"]), (name, T)
        assert np.isfinite(ye_na.cpu().numpy()).all()
    dl.table.close()


def test_noalloc_refuses_beyond_scratch(torch_cuda):
    torch = torch_cuda
    from paper_2609_18063_amd import binding as B
    dl = DeviceLayer(synth.WORKLOADS["tiny"])
    T = 1
    while B.workspace_bytes(dl.spec, T) <= B.MOE_NOALLOC_SCRATCH_BYTES:
        T *= 2
    x = torch.zeros(T, dl.wl.d, dtype=torch.float16, device="cuda")
    idx = torch.zeros(T, dl.wl.K, dtype=torch.int32, device="cuda")
    ye = torch.empty(T, dl.wl.K + dl.wl.S, dl.wl.d, dtype=torch.float32, device="cuda")
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    with pytest.raises(B.MoeError):
        B.expert_ffn_noalloc(dl.spec, dl.table, 0, x, idx, ye, st)
    dl.table.close()
