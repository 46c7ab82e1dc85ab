"""Host logic of the benchmark, on the CPU: the algorithmic byte counts behind
its `value` against the format's stored sizes (int4 codes plus one fp16 scale
and one fp16 zero per group of 64, §2 Quantization; LoRA A and B in fp16 on
the three projections, §3.3), the traffic lookup of the committed counter
summary, and the one-GPU refusal."""

import os
import subprocess
import sys

import pytest

import bench
import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _stored_projection(out_dim, in_dim):
    # written out per element: half a byte per code, 2 + 2 bytes per group of 64
    codes = out_dim * in_dim * 0.5
    groups = out_dim * in_dim / 64
    return int(codes + 4 * groups)


@pytest.mark.parametrize("name,expert,bundle", [
    ("tiny", 221_184, 258_048),
    ("moe35b", 1_769_472, 2_015_232),    # the 35B-class expert of Tab. 1: about 1.77 MB
    ("tier8b", 7_077_888, 7_569_408),
])
def test_expert_and_bundle_bytes(name, expert, bundle):
    wl = synth.WORKLOADS[name]
    assert bench.proj_bytes(wl.I, wl.d) == _stored_projection(wl.I, wl.d)
    assert bench.proj_bytes(wl.d, wl.I) == _stored_projection(wl.d, wl.I)
    e = 2 * bench.proj_bytes(wl.I, wl.d) + bench.proj_bytes(wl.d, wl.I)
    assert e == expert
    lora = 2 * 3 * wl.r * (wl.d + wl.I)    # A [r x in] and B [out x r] of each projection, fp16
    assert e + lora == bundle
    assert bench.layer_bytes(wl)["ffn"] == (wl.K + wl.S) * bundle


def test_chain_bytes_of_the_timed_launch():
    """256 tokens through 40 layers from token 0: per layer step the nine
    bundles and the residual read and written; a head at every layer but the
    last; the router at layer 0, and at every layer of token 0."""
    wl = synth.WORKLOADS["moe35b"]
    mat = 256 * 2048 * 2                    # router or head, fp16 [E x d]
    per_step = 9 * 2_015_232 + 2 * 2048 * 4
    steps = 256 * 40
    routers = 40 + 255                      # token 0: every layer; later tokens: layer 0
    heads = 256 * 39
    want = steps * per_step + (routers + heads) * mat
    assert want == 196_669_865_984
    assert bench.chain_bytes(wl, 40, 256) == want
    # a launch that starts later has no all-router token
    assert bench.chain_bytes(wl, 40, 16, first_token=5) == 16 * 40 * per_step + 16 * 40 * mat


def test_measured_traffic_follows_the_source_hash(monkeypatch):
    per_step = None
    for line in open(os.path.join(ROOT, bench.TRAFFIC_PROFILE)).read().splitlines():
        if line.startswith("traffic_bytes_per_step: "):
            per_step = int(line.split(": ", 1)[1])
    assert per_step is not None
    got = bench.measured_traffic(256)
    if got is not None:  # the committed summary matches the current engine sources
        assert got == per_step * 256
        # about the algorithmic bytes of the launch (the counters read 1.03x)
        assert 1.0 <= got / bench.chain_bytes(synth.WORKLOADS["moe35b"], 40, 256) < 1.1
    monkeypatch.setattr(bench, "sources_sha256", lambda: "0" * 64)
    assert bench.measured_traffic(256) is None


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
