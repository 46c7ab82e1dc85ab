"""GPU tests of the file tier (§3.1, SSD streaming): the 8B-tier decode
chain with its experts read from a file through the page cache.

The file tier only changes where a copy's bytes come from, so it is held to
the pinned-memory tier bit for bit: the same records, the same copies, every
resident slot equal to its record in the file, and the bytes read equal to the
copies made. A second run after the file's pages are dropped from the page
cache (a cold read) must give the same records again.
Sizes: 8B-tier layers (d 4096, 64 experts top-4, I 1024, r 16) at full size,
3 layers x 3 tokens, 8 slots per layer.
"""

import os
import tempfile

import pytest

import synth
from tests.test_gpu_tier import _layers

pytestmark = pytest.mark.gpu

L_FILE, T_FILE, SLOTS_FILE = 3, 3, 8


@pytest.fixture(scope="module")
def runs():
    import torch
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a visible GPU")
    from paper_2609_18063_amd import binding as B, tier
    wl = synth.WORKLOADS["tier8b"]
    spec = B.spec_from_workload(wl)
    layers, _ = _layers(wl, L_FILE, torch)
    cache = {}

    def bundle(n, e):
        if (n, e) not in cache:
            cache[(n, e)] = synth.bundle(wl, n, e)
        return cache[(n, e)]

    host = tier.HostPool(L_FILE, wl.E + wl.S, bundle)
    fd, path = tempfile.mkstemp(prefix="moe_tier_", suffix=".bin")
    os.close(fd)
    fpool = tier.FilePool(path, L_FILE, wl.E + wl.S, bundle, n_bounce=3, n_io=4)
    cache.clear()
    xi_t = torch.from_numpy(synth.token_draws(wl, 0, T_FILE)).cuda()
    ch_host = tier.TieredChain(spec, layers, host, SLOTS_FILE)
    rec_host = ch_host.run(xi_t, record=True)
    ch_file = tier.TieredChain(spec, layers, fpool, SLOTS_FILE)
    rec_file = ch_file.run(xi_t, record=True)
    out = {"wl": wl, "spec": spec, "layers": layers, "host": host, "file": fpool, "xi_t": xi_t,
           "ch_host": ch_host, "rec_host": rec_host, "ch_file": ch_file, "rec_file": rec_file}
    yield out
    for k in ("ch_host", "ch_file", "ch_cold"):
        if k in out:
            out[k].close()
    fpool.remove()


def test_file_tier_matches_pinned_tier_bit_exact(runs):
    import torch
    assert int(runs["ch_file"].status.item()) == 0
    for k in ("x", "idx", "w", "pidx", "pw", "ye"):
        assert torch.equal(runs["rec_file"][k], runs["rec_host"][k]), k
    assert runs["ch_file"].ops == runs["ch_host"].ops


def test_file_tier_slots_hold_the_file_records(runs):
    import torch
    ch, fpool = runs["ch_file"], runs["file"]
    checked = 0
    for n in range(L_FILE):
        for e in range(fpool.n_ids):
            s = ch.table.lookup(n, e)
            if s < 0:
                continue
            assert torch.equal(ch.slot_bytes(n, s).cpu(), fpool.bytes_of(n, e)), (n, e, s)
            assert torch.equal(fpool.bytes_of(n, e), runs["host"].bytes_of(n, e)), (n, e)
            checked += 1
    assert checked >= L_FILE * runs["wl"].K


def test_file_tier_reads_equal_copies(runs):
    st = runs["ch_file"].stager.stats()
    io = runs["ch_file"].stager.io_stats()
    assert st["copies"] > 0
    assert io["read_bytes"] == st["copies"] * runs["file"].bundle_bytes == st["bytes"]
    assert io["read_ns"] > 0
    assert runs["ch_host"].stager.io_stats() == {"read_ns": 0, "read_bytes": 0}


def test_file_tier_cold_read_same_records(runs):
    import torch
    from paper_2609_18063_amd import tier
    runs["file"].drop_page_cache()
    ch = tier.TieredChain(runs["spec"], runs["layers"], runs["file"], SLOTS_FILE)
    runs["ch_cold"] = ch
    rec = ch.run(runs["xi_t"], record=True)
    for k in ("x", "idx", "w", "pidx", "pw", "ye"):
        assert torch.equal(rec[k], runs["rec_host"][k]), k
