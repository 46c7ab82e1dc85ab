"""C ABI checks that need no GPU: the library loads, every function declared
in include/moe_api.h is exported, specs and arguments are validated, and the
slot table's host logic matches the oracle's slot table."""

import ctypes
import os
import re

import numpy as np
import pytest

import synth
from oracle import slots as o_slots

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "moe_api.h")


@pytest.fixture(scope="module")
def B():
    from paper_2609_18063_amd import binding
    binding.lib()
    return binding


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(moe_[a-z0-9_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported(B):
    names = _declared()
    assert len(names) >= 15
    handle = ctypes.CDLL(B.LIB_PATH)
    for n in names:
        assert hasattr(handle, n), n
        assert n in B.SIGNATURES, n
    assert set(B.SIGNATURES) == set(names)


def test_strerror(B):
    for code in (0, -1, -2, -3, -4, -5):
        assert B.strerror(code)
    assert B.strerror(-99) == "unknown error"


@pytest.mark.parametrize("name", ["tiny", "moe35b", "tier8b"])
def test_spec_check_accepts_workloads(B, name):
    spec = B.spec_from_workload(synth.WORKLOADS[name])
    assert B.spec_check(spec) == 0
    assert B.workspace_bytes(spec, 1) > 0
    assert B.workspace_bytes(spec, 512) > B.workspace_bytes(spec, 1)


@pytest.mark.parametrize("field,value", [
    ("d_model", 384), ("d_model", 256), ("d_expert", 100), ("n_experts", 0), ("n_experts", 2048),
    ("top_k", 0), ("top_k", 33), ("n_shared", 5), ("group_size", 32), ("lora_rank", 65),
    ("routing", 3)])
def test_spec_check_rejects(B, field, value):
    spec = B.spec_from_workload(synth.WORKLOADS["moe35b"])
    setattr(spec, field, value)
    assert B.spec_check(spec) == B.MOE_EINVAL
    assert B.workspace_bytes(spec, 1) == 0


def test_spec_check_rejects_k_above_e_and_reserved(B):
    spec = B.make_spec(512, 4, 5, 0, 256, 8, 2.0)
    assert B.spec_check(spec) == B.MOE_EINVAL
    spec = B.make_spec(512, 16, 2, 0, 256, 8, 2.0)
    spec.reserved[3] = 1
    assert B.spec_check(spec) == B.MOE_EINVAL
    spec = B.make_spec(512, 16, 2, 0, 256, 8, float("nan"))
    assert B.spec_check(spec) == B.MOE_EINVAL


def test_spec_check_sigmoid_group(B):
    """Sigmoid-group routing (App. A): n groups dividing E (E <= 256), 1 <= G <= n,
    K <= G E / n, scale > 0; the group fields must be zero under softmax-topk."""
    ok = B.make_spec(4096, 128, 8, 0, 1024, 16, 2.0, sigmoid_group=(8, 4, 2.5))
    assert B.spec_check(ok) == 0
    for groups in [(7, 4, 2.5), (8, 0, 2.5), (8, 9, 2.5), (8, 4, 0.0), (8, 4, -1.0), (8, 4, float("nan"))]:
        assert B.spec_check(B.make_spec(4096, 128, 8, 0, 1024, 16, 2.0, sigmoid_group=groups)) == B.MOE_EINVAL
    # K above the survivors' experts: 1 group of 16 ids survives, K = 17 > 16
    assert B.spec_check(B.make_spec(4096, 128, 17, 0, 1024, 16, 2.0, sigmoid_group=(8, 1, 1.0))) == B.MOE_EINVAL
    assert B.spec_check(B.make_spec(4096, 512, 8, 0, 1024, 16, 2.0, sigmoid_group=(8, 4, 1.0))) == B.MOE_EINVAL
    soft = B.make_spec(4096, 128, 8, 0, 1024, 16, 2.0)
    soft.n_groups = 8
    assert B.spec_check(soft) == B.MOE_EINVAL
    # the biased top-k exists only for sigmoid-group specs
    L = B.lib()
    ws = ctypes.c_void_p(0x100000)
    sp = B.spec_from_workload(synth.WORKLOADS["tiny"])
    assert L.moe_topk_biased(ctypes.byref(sp), ws, ws, 1, ws, ws, None) == B.MOE_EINVAL
    assert L.moe_topk_biased(ctypes.byref(ok), None, None, 0, None, None, None) == B.MOE_OK


def _fake_bundle(B, base):
    p = B.MoeProj(base, base + 0x1000, base + 0x2000, base + 0x3000)
    return B.MoeBundle(p, p, p)


def test_slot_table_errors(B):
    h = ctypes.c_void_p()
    L = B.lib()
    assert L.moe_slot_table_create(0, 4, 4, ctypes.byref(h)) == B.MOE_EINVAL
    t = B.SlotTable(2, 8, 4)
    mb = _fake_bundle(B, 0x10000)
    assert L.moe_slot_bind(t.handle, 2, 0, 0, ctypes.byref(mb)) == B.MOE_EINVAL
    assert L.moe_slot_bind(t.handle, 0, 8, 0, ctypes.byref(mb)) == B.MOE_EINVAL
    assert L.moe_slot_bind(t.handle, 0, 0, 4, ctypes.byref(mb)) == B.MOE_EINVAL
    bad = _fake_bundle(B, 0x10004)
    assert L.moe_slot_bind(t.handle, 0, 0, 0, ctypes.byref(bad)) == B.MOE_EALIGN
    nul = B.MoeBundle(B.MoeProj(None, None, None, None), mb.up, mb.down)
    assert L.moe_slot_bind(t.handle, 0, 0, 0, ctypes.byref(nul)) == B.MOE_EINVAL
    assert L.moe_slot_lookup(t.handle, 0, 3) == B.MOE_ENOTRESIDENT
    assert L.moe_slot_lookup(t.handle, 5, 3) == B.MOE_EINVAL
    t.close()


@pytest.mark.parametrize("seed", range(4))
def test_slot_table_matches_oracle_table(B, seed):
    rs = np.random.default_rng(seed)
    n_layers, n_ids, n_slots = 3, 20, 7
    t = B.SlotTable(n_layers, n_ids, n_slots)
    ref = o_slots.SlotTable(n_layers, n_ids, n_slots)
    for _ in range(400):
        layer = int(rs.integers(n_layers))
        e = int(rs.integers(n_ids))
        if rs.random() < 0.7:
            s = int(rs.integers(n_slots))
            t.bind(layer, e, s, _fake_bundle(B, 0x100000 * (1 + s)))
            ref.bind(layer, e, s)
        else:
            t.unbind(layer, e)
            ref.unbind(layer, e)
        for ll in range(n_layers):
            for ee in range(n_ids):
                assert t.lookup(ll, ee) == ref.lookup(ll, ee)
    t.close()


def test_hot_path_argument_checks_need_no_gpu(B):
    """These calls fail (or are no-ops) before any device work is enqueued."""
    L = B.lib()
    spec = B.spec_from_workload(synth.WORKLOADS["tiny"])
    sp = ctypes.byref(spec)
    ws = ctypes.c_void_p(0x100000)
    assert L.moe_route(sp, None, None, 0, None, None, None, None, 0, None) == B.MOE_OK
    assert L.moe_route(sp, None, ws, 1, None, ws, ws, ws, 1 << 20, None) == B.MOE_EINVAL
    mis = ctypes.c_void_p(0x100008)
    assert L.moe_route(sp, mis, ws, 1, None, ws, ws, ws, 1 << 20, None) == B.MOE_EALIGN
    assert L.moe_route(sp, ws, ws, 1, None, ws, ws, ws, 16, None) == B.MOE_ENOMEM
    assert L.moe_route(sp, ws, ws, -1, None, ws, ws, ws, 1 << 20, None) == B.MOE_EINVAL
    assert L.moe_combine(sp, None, None, 0, None, None) == B.MOE_OK
    assert L.moe_combine(sp, mis, ws, 2, ws, None) == B.MOE_EALIGN
    odd = ctypes.c_void_p(0x100002)
    assert L.moe_combine(sp, ws, odd, 2, ws, None) == B.MOE_EALIGN
    assert L.moe_route(sp, ws, ws, 1, None, odd, ws, ws, 1 << 20, None) == B.MOE_EALIGN
    assert L.moe_topk(sp, None, 1, ws, ws, None) == B.MOE_EINVAL
    assert L.moe_rmsnorm_f16(None, 0, 512, None, None) == B.MOE_OK
    assert L.moe_rmsnorm_f16(mis, 1, 512, ws, None) == B.MOE_EALIGN
    t = B.SlotTable(1, 16, 16)
    # a table never synced to the device is rejected
    assert L.moe_expert_ffn_int4_lora(sp, t.handle, 0, ws, 1, ws, ws, None, ws, 1 << 20,
                                      None) == B.MOE_EINVAL
    # too few ids for E + S
    spec35 = B.spec_from_workload(synth.WORKLOADS["moe35b"])
    assert L.moe_expert_ffn_int4_lora(ctypes.byref(spec35), t.handle, 0, ws, 1, ws, ws, None, ws,
                                      1 << 20, None) == B.MOE_EINVAL
    t.close()
    bad = B.spec_from_workload(synth.WORKLOADS["tiny"])
    bad.group_size = 32
    assert L.moe_route(ctypes.byref(bad), ws, ws, 1, None, ws, ws, ws, 1 << 20, None) == B.MOE_EINVAL


def test_library_fails_loudly_when_missing(tmp_path, monkeypatch):
    from paper_2609_18063_amd import binding
    monkeypatch.setattr(binding, "LIB_PATH", str(tmp_path / "absent.so"))
    monkeypatch.setattr(binding, "_lib", None)
    with pytest.raises(ImportError):
        binding.lib()


def test_merge_requantize_argument_checks(B):
    """moe_merge_requantize rejects bad shapes and alignments before any
    device work (the pointers below are never dereferenced)."""
    lib = B.lib()
    ok = B.MoeProj(0x10000, 0x20000, None, None)
    ad = B.MoeProj(0x10000, 0x20000, 0x30000, 0x40000)

    def call(p, out_dim, in_dim, rank=0, q_out=0x50000, sz_out=0x60000, stats=None):
        return lib.moe_merge_requantize(None if p is None else ctypes.byref(p), out_dim, in_dim, rank,
                                        2.0, q_out, sz_out, stats, None)

    assert call(None, 4, 64) == B.MOE_EINVAL
    assert call(ok, 0, 64) == B.MOE_EINVAL
    assert call(ok, 4, 32) == B.MOE_EINVAL
    assert call(ok, 4, 96) == B.MOE_EINVAL
    assert call(ok, 4, 64, q_out=None) == B.MOE_EINVAL
    assert call(ad, 4, 64, rank=0) == B.MOE_EINVAL
    assert call(ad, 4, 64, rank=65) == B.MOE_EINVAL
    assert call(B.MoeProj(0x10000, 0x20001, None, None), 4, 64) == B.MOE_EALIGN
    assert call(ok, 4, 64, sz_out=0x60001) == B.MOE_EALIGN
    assert call(ok, 4, 64, stats=0x70004) == B.MOE_EALIGN


def test_stager_file_argument_checks(B):
    """moe_stager_create_file rejects bad arguments before touching the file
    or the device."""
    lib = B.lib()
    h = ctypes.c_void_p()
    lay = B.MoeBundleLayout()
    for args in ((None, 4096, b"/nonexistent", 4096, 2, 2),      # no table
                 (0x1000, 4096, None, 4096, 2, 2),              # no path
                 (0x1000, 4096, b"/nonexistent", 1024, 2, 2),   # stride < bundle
                 (0x1000, 4096, b"/nonexistent", 4096, 0, 2),   # no bounce buffer
                 (0x1000, 4096, b"/nonexistent", 4096, 2, 17)):  # too many threads
        table, nbytes, path, stride, nb, nio = args
        assert lib.moe_stager_create_file(table, ctypes.byref(lay), nbytes, path, stride, nb, nio,
                                          0x100000, 4096, ctypes.byref(h)) == B.MOE_EINVAL
    assert lib.moe_stager_io_stats(None, None, None) == B.MOE_EINVAL


def test_file_pool_records(tmp_path):
    """The file tier's records are the packed bundles, at stride offsets."""
    from paper_2609_18063_amd import tier
    wl = synth.WORKLOADS["tiny"]
    fp = tier.FilePool(tmp_path / "pool.bin", 2, 3, lambda n, e: synth.bundle(wl, n, e), n_bounce=2)
    assert os.path.getsize(fp.path) == 2 * 3 * fp.stride and fp.stride % 256 == 0
    for n in range(2):
        for e in range(3):
            ref = tier.bundle_layout(synth.bundle(wl, n, e))[0]
            assert np.array_equal(fp.bytes_of(n, e).numpy(), ref)
    rp = tier.FilePool(tmp_path / "rep.bin", 3, 2, lambda n, e: synth.bundle(wl, n, e), replicate=True)
    assert np.array_equal(rp.bytes_of(2, 1).numpy(), rp.bytes_of(0, 1).numpy())
    fp.drop_page_cache()
    fp.remove()
    assert not os.path.exists(fp.path)


def test_noalloc_ffn_rejects_sizes_beyond_its_scratch(B):
    """The no-allocation expert entry point refuses, before any runtime call,
    a token count whose workspace layout exceeds its static scratch."""
    spec = B.spec_from_workload(synth.WORKLOADS["moe35b"])
    big = 1
    while B.workspace_bytes(spec, big) <= B.MOE_NOALLOC_SCRATCH_BYTES:
        big *= 2
    assert big > 16              # the scratch holds at least 16 tokens of the 35B-class layer
    rc = B.lib().moe_expert_ffn_int4_lora_noalloc(ctypes.byref(spec), None, 0, None, big, None,
                                                  None, None, None)
    assert rc == B.MOE_ENOMEM
