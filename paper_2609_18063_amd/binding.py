"""ctypes binding of libmoe.so (argument marshalling only).

Every function here converts torch tensors to device pointers, passes the
current HIP stream and turns negative return codes into :class:`MoeError`.
All computation happens in the library's HIP kernels.  If the library is
missing, loading fails with ``ImportError``: there is no fallback path.
"""

import ctypes
import sys
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libmoe.so")

c_int, c_int32, c_float, c_void_p, c_size_t = (ctypes.c_int, ctypes.c_int32, ctypes.c_float,
                                               ctypes.c_void_p, ctypes.c_size_t)

MOE_OK, MOE_EINVAL, MOE_EALIGN, MOE_ENOTRESIDENT, MOE_EHIP, MOE_ENOMEM = 0, -1, -2, -3, -4, -5
MOE_STATUS_SLOT_MISS, MOE_STATUS_BAD_INDEX = 1, 2
MOE_ROUTING_SOFTMAX_TOPK, MOE_ROUTING_SIGMOID_GROUP = 0, 1


class MoeLayerSpec(ctypes.Structure):
    _fields_ = [("d_model", c_int32), ("n_experts", c_int32), ("top_k", c_int32),
                ("n_shared", c_int32), ("d_expert", c_int32), ("group_size", c_int32),
                ("lora_rank", c_int32), ("lora_scale", c_float), ("routing", c_int32),
                ("n_groups", c_int32), ("top_groups", c_int32), ("route_scale", c_float),
                ("reserved", c_int32 * 4)]


class MoeProj(ctypes.Structure):
    _fields_ = [("q", c_void_p), ("sz", c_void_p), ("lora_a", c_void_p), ("lora_b", c_void_p)]


class MoeBundle(ctypes.Structure):
    _fields_ = [("gate", MoeProj), ("up", MoeProj), ("down", MoeProj)]


class MoeEngineLayer(ctypes.Structure):
    _fields_ = [("router", c_void_p), ("head", c_void_p), ("mix_d", c_void_p),
                ("mix_perm", c_void_p)]


class MoeHeadMlp(ctypes.Structure):
    _fields_ = [("hidden", c_int32), ("w1_x", c_void_p), ("w1_r", c_void_p), ("b1", c_void_p),
                ("w2", c_void_p), ("b2", c_void_p), ("w_l", c_void_p)]


class MoeBundleLayout(ctypes.Structure):
    _fields_ = [("gate", ctypes.c_int64 * 4), ("up", ctypes.c_int64 * 4),
                ("down", ctypes.c_int64 * 4)]


class MoeStagerStats(ctypes.Structure):
    _fields_ = [("stages", ctypes.c_int64), ("uses", ctypes.c_int64), ("copies", ctypes.c_int64),
                ("bytes", ctypes.c_int64)]


class MoeError(RuntimeError):
    def __init__(self, code, what):
        self.code = code
        super().__init__("%s failed: %s (%d)" % (what, strerror(code), code))


_lib = None

# name -> (restype, argtypes) for every symbol declared in include/moe_api.h
SIGNATURES = {
    "moe_spec_check": (c_int, [ctypes.POINTER(MoeLayerSpec)]),
    "moe_strerror": (ctypes.c_char_p, [c_int]),
    "moe_slot_table_create": (c_int, [c_int, c_int, c_int, ctypes.POINTER(c_void_p)]),
    "moe_slot_table_destroy": (c_int, [c_void_p]),
    "moe_slot_bind": (c_int, [c_void_p, c_int, c_int, c_int, ctypes.POINTER(MoeBundle)]),
    "moe_slot_unbind": (c_int, [c_void_p, c_int, c_int]),
    "moe_slot_lookup": (c_int, [c_void_p, c_int, c_int]),
    "moe_slot_table_sync": (c_int, [c_void_p, c_void_p]),
    "moe_rmsnorm_f16": (c_int, [c_void_p, c_int, c_int, c_void_p, c_void_p]),
    "moe_workspace_bytes": (c_size_t, [ctypes.POINTER(MoeLayerSpec), c_int]),
    "moe_route": (c_int, [ctypes.POINTER(MoeLayerSpec), c_void_p, c_void_p, c_int, c_void_p,
                          c_void_p, c_void_p, c_void_p, c_size_t, c_void_p]),
    "moe_preroute": (c_int, [ctypes.POINTER(MoeLayerSpec), c_void_p, c_void_p, c_int, c_void_p,
                             c_void_p, c_void_p, c_void_p, c_size_t, c_void_p]),
    "moe_preroute_mlp_workspace_bytes": (c_size_t, [ctypes.POINTER(MoeLayerSpec), c_int, c_int]),
    "moe_preroute_mlp": (c_int, [ctypes.POINTER(MoeLayerSpec), ctypes.POINTER(MoeHeadMlp), c_void_p,
                                 c_int, c_void_p, c_void_p, c_void_p, c_void_p, c_void_p, c_void_p,
                                 c_size_t, c_void_p]),
    "moe_expert_ffn_int4_lora": (c_int, [ctypes.POINTER(MoeLayerSpec), c_void_p, c_int, c_void_p,
                                         c_int, c_void_p, c_void_p, c_void_p, c_void_p, c_size_t,
                                         c_void_p]),
    "moe_expert_ffn_int4_lora_noalloc": (c_int, [ctypes.POINTER(MoeLayerSpec), c_void_p, c_int,
                                                 c_void_p, c_int, c_void_p, c_void_p, c_void_p,
                                                 c_void_p]),
    "moe_expert_ffn_grouped_int4_lora": (c_int, [ctypes.POINTER(MoeLayerSpec), c_void_p, c_int,
                                                 c_void_p, c_int, c_void_p, c_void_p, c_void_p,
                                                 c_void_p, c_size_t, c_void_p]),
    "moe_combine": (c_int, [ctypes.POINTER(MoeLayerSpec), c_void_p, c_void_p, c_int, c_void_p,
                            c_void_p]),
    "moe_topk": (c_int, [ctypes.POINTER(MoeLayerSpec), c_void_p, c_int, c_void_p, c_void_p,
                         c_void_p]),
    "moe_topk_biased": (c_int, [ctypes.POINTER(MoeLayerSpec), c_void_p, c_void_p, c_int, c_void_p,
                                c_void_p, c_void_p]),
    "moe_profile_arm": (c_int, [c_int, c_void_p, c_void_p]),
    "moe_merge_requantize": (c_int, [ctypes.POINTER(MoeProj), c_int, c_int, c_int, ctypes.c_float,
                                     c_void_p, c_void_p, c_void_p, c_void_p]),
    "moe_slot_policy_create": (c_int, [c_int, c_int, c_int, ctypes.POINTER(c_void_p)]),
    "moe_slot_policy_destroy": (c_int, [c_void_p]),
    "moe_slot_policy_stage": (c_int, [c_void_p, c_int, c_void_p, c_int, c_void_p]),
    "moe_slot_policy_use": (c_int, [c_void_p, c_int, c_void_p, c_int, c_void_p]),
    "moe_slot_policy_release": (c_int, [c_void_p, c_int]),
    "moe_slot_policy_lookup": (c_int, [c_void_p, c_int, c_int]),
    "moe_stager_create": (c_int, [c_void_p, ctypes.POINTER(MoeBundleLayout), c_size_t, c_void_p,
                                  c_void_p, c_size_t, ctypes.POINTER(c_void_p)]),
    "moe_stager_destroy": (c_int, [c_void_p]),
    "moe_stager_create_file": (c_int, [c_void_p, ctypes.POINTER(MoeBundleLayout), c_size_t,
                                       ctypes.c_char_p, c_size_t, c_int, c_int, c_void_p, c_size_t,
                                       ctypes.POINTER(c_void_p)]),
    "moe_stager_io_stats": (c_int, [c_void_p, ctypes.POINTER(ctypes.c_int64),
                                    ctypes.POINTER(ctypes.c_int64)]),
    "moe_stager_stage": (c_int, [c_void_p, c_int, c_void_p, c_int, c_void_p, c_void_p]),
    "moe_stager_use": (c_int, [c_void_p, c_int, c_void_p, c_int, c_void_p, c_void_p]),
    "moe_stager_release": (c_int, [c_void_p, c_int]),
    "moe_stager_stats_get": (c_int, [c_void_p, ctypes.POINTER(MoeStagerStats)]),
    "moe_combine_add": (c_int, [ctypes.POINTER(MoeLayerSpec), c_void_p, c_void_p, c_int, c_void_p,
                                c_void_p]),
    "moe_chain_token_start": (c_int, [c_void_p, c_int, c_void_p, c_void_p]),
    "moe_chain_mix_rmsnorm": (c_int, [c_void_p, c_void_p, c_int, c_void_p, c_void_p, c_void_p]),
    "moe_engine_supported": (c_int, [ctypes.POINTER(MoeLayerSpec)]),
    "moe_engine_workspace_bytes": (c_size_t, [ctypes.POINTER(MoeLayerSpec), c_int]),
    "moe_engine_layers": (c_int, [ctypes.POINTER(MoeLayerSpec), c_void_p, c_void_p, c_void_p, c_int,
                                  c_void_p, c_void_p, c_void_p, c_void_p, c_void_p, c_void_p,
                                  c_void_p, c_void_p, c_size_t, c_void_p]),
    "moe_engine_tokens_supported": (c_int, [ctypes.POINTER(MoeLayerSpec)]),
    "moe_engine_tokens": (c_int, [ctypes.POINTER(MoeLayerSpec), c_void_p, c_void_p, c_void_p, c_int,
                                  c_void_p, c_void_p, c_void_p, c_void_p, c_void_p, c_void_p,
                                  c_void_p, c_void_p, c_size_t, c_void_p]),
    "moe_engine_chain_supported": (c_int, [ctypes.POINTER(MoeLayerSpec)]),
    "moe_engine_chain_mlp_supported": (c_int, [ctypes.POINTER(MoeLayerSpec), c_int]),
    "moe_engine_chain_mlp": (c_int, [ctypes.POINTER(MoeLayerSpec), c_void_p, c_void_p, c_void_p, c_int, c_int,
                                     c_int, c_int, c_void_p, c_void_p, c_void_p, c_void_p, c_void_p,
                                     c_void_p, c_void_p, c_void_p, c_void_p, c_void_p, c_void_p, ctypes.c_size_t,
                                     c_void_p]),
    "moe_engine_chain": (c_int, [ctypes.POINTER(MoeLayerSpec), c_void_p, c_void_p, c_int, c_int,
                                 c_int, c_void_p, c_void_p, c_void_p, c_void_p, c_void_p, c_void_p,
                                 c_void_p, c_void_p, c_void_p, c_void_p, c_void_p, c_size_t,
                                 c_void_p]),
}

MOE_PROF_FFN_MAIN = 0
MOE_PROF_ENGINE_PHASES = 1


def lib():
    """Load libmoe.so once and declare its signatures."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError("libmoe.so is not built (%s); run __graft_entry__.build()" % LIB_PATH)
        handle = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(handle, name)
            fn.restype, fn.argtypes = res, args
        _lib = handle
    return _lib


def strerror(code):
    return lib().moe_strerror(int(code)).decode()


def _check(rc, what):
    if rc < 0:
        raise MoeError(rc, what)
    return rc


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream=None):
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


class StreamPair:
    """Two streams for work that must overlap (copies beside kernels), taken
    one right after the other from torch's stream pool (default priority).
    The pool creates its streams together, and HIP maps streams onto a few
    hardware queues (GPU_MAX_HW_QUEUES) in creation order, so consecutive pool
    streams sit on different queues; a pool stream paired with the null
    stream can share its queue and serialize against it. Pool streams live as
    long as the process, so ``close`` has nothing to free."""

    def __init__(self):
        import torch
        self.compute = torch.cuda.Stream()
        self.copy = torch.cuda.Stream()

    def close(self):
        pass


def make_spec(d, n_experts, top_k, n_shared, d_expert, lora_rank, lora_scale, group_size=64,
              sigmoid_group=None):
    """``sigmoid_group``: None (softmax-topk) or (n_groups, top_groups, scale)."""
    s = MoeLayerSpec()
    s.d_model, s.n_experts, s.top_k, s.n_shared = d, n_experts, top_k, n_shared
    s.d_expert, s.group_size, s.lora_rank, s.lora_scale = d_expert, group_size, lora_rank, lora_scale
    s.routing = MOE_ROUTING_SOFTMAX_TOPK
    if sigmoid_group is not None:
        s.routing = MOE_ROUTING_SIGMOID_GROUP
        s.n_groups, s.top_groups, s.route_scale = sigmoid_group
    return s


def spec_from_workload(wl):
    return make_spec(wl.d, wl.E, wl.K, wl.S, wl.I, wl.r, wl.lora_scale)


def spec_check(spec):
    return lib().moe_spec_check(ctypes.byref(spec))


def workspace_bytes(spec, T):
    return int(lib().moe_workspace_bytes(ctypes.byref(spec), int(T)))


class SlotTable:
    """Owner of a library slot table (host mirror + device copy)."""

    def __init__(self, n_layers, n_ids, n_slots):
        h = c_void_p()
        _check(lib().moe_slot_table_create(n_layers, n_ids, n_slots, ctypes.byref(h)),
               "moe_slot_table_create")
        self.handle = h
        self.n_layers, self.n_ids, self.n_slots = n_layers, n_ids, n_slots
        self._keep = {}

    def bind(self, layer, expert, slot, bundle, keep=None):
        _check(lib().moe_slot_bind(self.handle, layer, expert, slot, ctypes.byref(bundle)),
               "moe_slot_bind")
        self._keep[(layer, slot)] = keep

    def unbind(self, layer, expert):
        _check(lib().moe_slot_unbind(self.handle, layer, expert), "moe_slot_unbind")

    def lookup(self, layer, expert):
        rc = lib().moe_slot_lookup(self.handle, layer, expert)
        if rc == MOE_ENOTRESIDENT:
            return -1
        return _check(rc, "moe_slot_lookup")

    def sync(self, stream=None):
        _check(lib().moe_slot_table_sync(self.handle, _stream(stream)), "moe_slot_table_sync")

    def close(self):
        if self.handle:
            _check(lib().moe_slot_table_destroy(self.handle), "moe_slot_table_destroy")
            self.handle = None

    def __del__(self, _finalizing=sys.is_finalizing):
        # no runtime calls while the interpreter shuts down: close() explicitly
        if _finalizing():
            return
        try:
            self.close()
        except Exception:
            pass


def _i32(a):
    return np.ascontiguousarray(np.asarray(a, dtype=np.int32))


class SlotPolicy:
    """The library's host-tier slot policy (host logic only)."""

    def __init__(self, n_layers, n_ids, n_slots):
        h = c_void_p()
        _check(lib().moe_slot_policy_create(n_layers, n_ids, n_slots, ctypes.byref(h)),
               "moe_slot_policy_create")
        self.handle = h

    def stage(self, layer, experts):
        e = _i32(experts)
        out = np.zeros((max(len(e), 1), 2), dtype=np.int32)
        n = _check(lib().moe_slot_policy_stage(self.handle, layer, e.ctypes.data, len(e),
                                               out.ctypes.data), "moe_slot_policy_stage")
        return [tuple(int(v) for v in out[i]) for i in range(n)]

    def use(self, layer, experts):
        e = _i32(experts)
        out = np.zeros(max(len(e), 1), dtype=np.int32)
        _check(lib().moe_slot_policy_use(self.handle, layer, e.ctypes.data, len(e), out.ctypes.data),
               "moe_slot_policy_use")
        return out[:len(e)].tolist()

    def release(self, layer):
        _check(lib().moe_slot_policy_release(self.handle, layer), "moe_slot_policy_release")

    def lookup(self, layer, expert):
        rc = lib().moe_slot_policy_lookup(self.handle, layer, expert)
        return -1 if rc == MOE_ENOTRESIDENT else _check(rc, "moe_slot_policy_lookup")

    def close(self):
        if self.handle:
            lib().moe_slot_policy_destroy(self.handle)
            self.handle = None

    def __del__(self, _finalizing=sys.is_finalizing):
        # no runtime calls while the interpreter shuts down: close() explicitly
        if _finalizing():
            return
        try:
            self.close()
        except Exception:
            pass


class Stager:
    """The slot policy driving a slot table: pinned host bundles -> device slots."""

    def __init__(self, table, layout, bundle_bytes, host_ptrs, slot_pool, slot_stride, file=None):
        """``file``: None (bundles at ``host_ptrs`` in pinned memory) or
        ``(path, file_stride, n_bounce, n_io)`` for the file tier."""
        h = c_void_p()
        if file is None:
            ptrs = (c_void_p * len(host_ptrs))(*host_ptrs)
            _check(lib().moe_stager_create(table.handle, ctypes.byref(layout), bundle_bytes, ptrs,
                                           _ptr(slot_pool), slot_stride, ctypes.byref(h)),
                   "moe_stager_create")
        else:
            path, file_stride, n_bounce, n_io = file
            _check(lib().moe_stager_create_file(table.handle, ctypes.byref(layout), bundle_bytes,
                                                str(path).encode(), file_stride, n_bounce, n_io,
                                                _ptr(slot_pool), slot_stride, ctypes.byref(h)),
                   "moe_stager_create_file")
        self.handle = h
        self.table, self.pool = table, slot_pool

    def io_stats(self):
        ns, nb = ctypes.c_int64(), ctypes.c_int64()
        _check(lib().moe_stager_io_stats(self.handle, ctypes.byref(ns), ctypes.byref(nb)),
               "moe_stager_io_stats")
        return {"read_ns": ns.value, "read_bytes": nb.value}

    def stage(self, layer, experts, copy_stream):
        e = _i32(experts)
        out = np.zeros((max(len(e), 1), 2), dtype=np.int32)
        n = _check(lib().moe_stager_stage(self.handle, layer, e.ctypes.data, len(e),
                                          ctypes.c_void_p(copy_stream.cuda_stream),
                                          out.ctypes.data), "moe_stager_stage")
        return [tuple(int(v) for v in out[i]) for i in range(n)]

    def use(self, layer, experts, compute_stream=None):
        e = _i32(experts)
        out = np.zeros(max(len(e), 1), dtype=np.int32)
        _check(lib().moe_stager_use(self.handle, layer, e.ctypes.data, len(e),
                                    _stream(compute_stream), out.ctypes.data), "moe_stager_use")
        return out[:len(e)].tolist()

    def release(self, layer):
        _check(lib().moe_stager_release(self.handle, layer), "moe_stager_release")

    def stats(self):
        st = MoeStagerStats()
        _check(lib().moe_stager_stats_get(self.handle, ctypes.byref(st)), "moe_stager_stats_get")
        return {"stages": st.stages, "uses": st.uses, "copies": st.copies, "bytes": st.bytes}

    def close(self):
        if self.handle:
            lib().moe_stager_destroy(self.handle)
            self.handle = None

    def __del__(self, _finalizing=sys.is_finalizing):
        # no runtime calls while the interpreter shuts down: close() explicitly
        if _finalizing():
            return
        try:
            self.close()
        except Exception:
            pass


# ---- weights: host arrays in the stored format -> device buffers --------------

def upload_projection(qsz, lora, device):
    """(packed q [out, in/2] uint8, s fp16 [out, in/64], z fp16) + (A, B) | None
    -> (MoeProj, tensors to keep alive).  s and z are interleaved into the
    (scale, zero) pairs of the device layout."""
    import torch
    q, s, z = qsz
    qt = torch.from_numpy(np.ascontiguousarray(q)).to(device)
    sz = np.ascontiguousarray(np.stack([np.asarray(s, np.float16), np.asarray(z, np.float16)], -1))
    szt = torch.from_numpy(sz).to(device)
    keep = [qt, szt]
    p = MoeProj(qt.data_ptr(), szt.data_ptr(), None, None)
    if lora is not None:
        at = torch.from_numpy(np.ascontiguousarray(lora[0], dtype=np.float16)).to(device)
        bt = torch.from_numpy(np.ascontiguousarray(lora[1], dtype=np.float16)).to(device)
        keep += [at, bt]
        p.lora_a, p.lora_b = at.data_ptr(), bt.data_ptr()
    return p, keep


def upload_bundle(b, device="cuda"):
    lo = b.get("lora") or {}
    g, kg = upload_projection(b["gate"], lo.get("gate"), device)
    u, ku = upload_projection(b["up"], lo.get("up"), device)
    d, kd = upload_projection(b["down"], lo.get("down"), device)
    return MoeBundle(g, u, d), kg + ku + kd


# ---- hot path -----------------------------------------------------------------

def rmsnorm_f16(xi, x, stream=None):
    T, d = xi.shape
    _check(lib().moe_rmsnorm_f16(_ptr(xi), T, d, _ptr(x), _stream(stream)), "moe_rmsnorm_f16")


def route(spec, x, w_router, idx, w, workspace, logits=None, stream=None):
    T = x.shape[0]
    _check(lib().moe_route(ctypes.byref(spec), _ptr(x), _ptr(w_router), T, _ptr(logits), _ptr(idx),
                           _ptr(w), _ptr(workspace), workspace.numel() * workspace.element_size(),
                           _stream(stream)), "moe_route")


def preroute(spec_next, x, w_head, pred_idx, pred_w, workspace, logits=None, stream=None):
    T = x.shape[0]
    _check(lib().moe_preroute(ctypes.byref(spec_next), _ptr(x), _ptr(w_head), T, _ptr(logits),
                              _ptr(pred_idx), _ptr(pred_w), _ptr(workspace),
                              workspace.numel() * workspace.element_size(), _stream(stream)),
           "moe_preroute")


def head_mlp(hidden, w1_x, w1_r, w2, b1=None, b2=None, w_l=None):
    """moe_head_mlp of device fp16 tensors (layouts as in include/moe_api.h)."""
    def p(t):
        return None if t is None else t.data_ptr()
    return MoeHeadMlp(hidden, p(w1_x), p(w1_r), p(b1), p(w2), p(b2), p(w_l))


def preroute_mlp_workspace_bytes(spec_next, hidden, T):
    return lib().moe_preroute_mlp_workspace_bytes(ctypes.byref(spec_next), hidden, T)


def preroute_mlp(spec_next, head, x, routed_t, routed_tm1, pred_idx, pred_w, workspace, logits=None,
                 stream=None):
    """Full prerouter head (moe_preroute_mlp); ``head`` from ``head_mlp``."""
    T = x.shape[0]
    _check(lib().moe_preroute_mlp(ctypes.byref(spec_next), ctypes.byref(head), _ptr(x), T, _ptr(routed_t),
                                  _ptr(routed_tm1), _ptr(logits), _ptr(pred_idx), _ptr(pred_w),
                                  _ptr(workspace), workspace.numel() * workspace.element_size(),
                                  _stream(stream)), "moe_preroute_mlp")


def expert_ffn(spec, table, layer, x, idx, y_experts, status, workspace, stream=None):
    T = x.shape[0]
    _check(lib().moe_expert_ffn_int4_lora(ctypes.byref(spec), table.handle, layer, _ptr(x), T,
                                          _ptr(idx), _ptr(y_experts), _ptr(status), _ptr(workspace),
                                          workspace.numel() * workspace.element_size(),
                                          _stream(stream)), "moe_expert_ffn_int4_lora")


MOE_NOALLOC_SCRATCH_BYTES = 4 << 20


def expert_ffn_noalloc(spec, table, layer, x, idx, y_experts, status, stream=None):
    """``expert_ffn`` without a workspace: the library's static per-device scratch."""
    T = x.shape[0]
    _check(lib().moe_expert_ffn_int4_lora_noalloc(ctypes.byref(spec), table.handle, layer, _ptr(x),
                                                  T, _ptr(idx), _ptr(y_experts), _ptr(status),
                                                  _stream(stream)),
           "moe_expert_ffn_int4_lora_noalloc")


def expert_ffn_grouped(spec, table, layer, x, idx, y_experts, status, workspace, stream=None):
    """Batched / prefill experts: same contract as ``expert_ffn``, grouped by expert."""
    T = x.shape[0]
    _check(lib().moe_expert_ffn_grouped_int4_lora(ctypes.byref(spec), table.handle, layer, _ptr(x),
                                                  T, _ptr(idx), _ptr(y_experts), _ptr(status),
                                                  _ptr(workspace),
                                                  workspace.numel() * workspace.element_size(),
                                                  _stream(stream)),
           "moe_expert_ffn_grouped_int4_lora")


def combine(spec, y_experts, w, y, stream=None):
    T = y.shape[0]
    _check(lib().moe_combine(ctypes.byref(spec), _ptr(y_experts), _ptr(w), T, _ptr(y),
                             _stream(stream)), "moe_combine")


def topk(spec, logits, idx, w, stream=None):
    T = logits.shape[0]
    _check(lib().moe_topk(ctypes.byref(spec), _ptr(logits), T, _ptr(idx), _ptr(w), _stream(stream)),
           "moe_topk")


def topk_biased(spec, logits, bias, idx, w, stream=None):
    """Sigmoid-group top-k with a selection bias (fp32 [E] device tensor or None)."""
    T = logits.shape[0]
    _check(lib().moe_topk_biased(ctypes.byref(spec), _ptr(logits), _ptr(bias), T, _ptr(idx), _ptr(w),
                                 _stream(stream)), "moe_topk_biased")


def merge_requantize(proj, out_dim, in_dim, rank, lora_scale, q_out, sz_out, stats=None,
                     stream=None):
    """moe_merge_requantize: ``proj`` a MoeProj of device pointers; ``q_out``
    uint8 ``[out, in/2]``, ``sz_out`` fp16 ``[out, in/64, 2]``, ``stats``
    float64 ``[out, in/64, 2]`` or None (device tensors)."""
    _check(lib().moe_merge_requantize(ctypes.byref(proj), out_dim, in_dim, rank, lora_scale,
                                      _ptr(q_out), _ptr(sz_out), _ptr(stats), _stream(stream)),
           "moe_merge_requantize")


def profile_arm(which, start_event, stop_event):
    """Time the next launch of kernel ``which`` with two hipEvent_t handles (ints)."""
    _check(lib().moe_profile_arm(which, ctypes.c_void_p(start_event), ctypes.c_void_p(stop_event)),
           "moe_profile_arm")


def combine_add(spec, y_experts, w, y_inout, stream=None):
    T = y_inout.shape[0]
    _check(lib().moe_combine_add(ctypes.byref(spec), _ptr(y_experts), _ptr(w), T, _ptr(y_inout),
                                 _stream(stream)), "moe_combine_add")


def chain_token_start(xi, r, stream=None):
    _check(lib().moe_chain_token_start(_ptr(xi), r.numel(), _ptr(r), _stream(stream)),
           "moe_chain_token_start")


def chain_mix_rmsnorm(mix_d, perm, r, x, stream=None):
    _check(lib().moe_chain_mix_rmsnorm(_ptr(mix_d), _ptr(perm), r.numel(), _ptr(r), _ptr(x),
                                       _stream(stream)), "moe_chain_mix_rmsnorm")


MOE_STATUS_ENGINE_ABORT = 4


def engine_supported(spec):
    return lib().moe_engine_supported(ctypes.byref(spec)) == MOE_OK


def engine_chain_supported(spec):
    return lib().moe_engine_chain_supported(ctypes.byref(spec)) == MOE_OK


def engine_workspace_bytes(spec, n_layers):
    return int(lib().moe_engine_workspace_bytes(ctypes.byref(spec), int(n_layers)))


def engine_chain_mlp_supported(spec, hidden):
    return lib().moe_engine_chain_mlp_supported(ctypes.byref(spec), int(hidden)) == MOE_OK


def head_mlp_array(heads, device="cuda"):
    """Device array of moe_head_mlp (one per layer; None entries -> all NULL)."""
    import torch
    arr = (MoeHeadMlp * len(heads))()
    for i, h in enumerate(heads):
        if h is not None:
            arr[i] = h
    raw = np.frombuffer(bytes(arr), dtype=np.uint8).copy()
    return torch.from_numpy(raw).to(device)


def engine_layer_array(layers, device="cuda"):
    """Device array of moe_engine_layer from dicts of device tensors
    (router, head, mix_d, mix_perm; missing or None -> NULL)."""
    import torch
    arr = (MoeEngineLayer * len(layers))()
    for i, lay in enumerate(layers):
        def p(k):
            t = lay.get(k)
            return None if t is None else t.data_ptr()
        arr[i] = MoeEngineLayer(p("router"), p("head"), p("mix_d"), p("mix_perm"))
    raw = np.frombuffer(bytes(arr), dtype=np.uint8).copy()
    return torch.from_numpy(raw).to(device)


def engine_layers(spec, table, layer_arr, step_layer, xi, y, workspace, idx=None, w=None,
                  pidx=None, pw=None, status=None, stream=None):
    n = step_layer.numel()
    _check(lib().moe_engine_layers(ctypes.byref(spec), table.handle, _ptr(layer_arr),
                                   _ptr(step_layer), n, _ptr(xi), _ptr(y), _ptr(idx), _ptr(w),
                                   _ptr(pidx), _ptr(pw), _ptr(status), _ptr(workspace),
                                   workspace.numel() * workspace.element_size(), _stream(stream)),
           "moe_engine_layers")


def engine_tokens_supported(spec):
    return lib().moe_engine_tokens_supported(ctypes.byref(spec)) == MOE_OK


def engine_tokens(spec, table, layer_arr, step_layer, xi, y, workspace, idx=None, w=None,
                  pidx=None, pw=None, status=None, stream=None):
    """moe_engine_tokens: the steps of engine_layers, one per team of 16 workgroups in flight."""
    n = step_layer.numel()
    _check(lib().moe_engine_tokens(ctypes.byref(spec), table.handle, _ptr(layer_arr),
                                   _ptr(step_layer), n, _ptr(xi), _ptr(y), _ptr(idx), _ptr(w),
                                   _ptr(pidx), _ptr(pw), _ptr(status), _ptr(workspace),
                                   workspace.numel() * workspace.element_size(), _stream(stream)),
           "moe_engine_tokens")


def engine_chain(spec, table, layer_arr, n_layers, first_token, xi, r_state, workspace,
                 x_rec=None, idx=None, w=None, pidx=None, pw=None, y_rec=None, status=None,
                 stream=None, r_rec=None):
    n_tokens = xi.shape[0]
    _check(lib().moe_engine_chain(ctypes.byref(spec), table.handle, _ptr(layer_arr), n_layers,
                                  first_token, n_tokens, _ptr(xi), _ptr(r_state), _ptr(x_rec),
                                  _ptr(r_rec), _ptr(idx), _ptr(w), _ptr(pidx), _ptr(pw),
                                  _ptr(y_rec),
                                  _ptr(status), _ptr(workspace),
                                  workspace.numel() * workspace.element_size(), _stream(stream)),
           "moe_engine_chain")


def engine_chain_mlp(spec, table, layer_arr, head_arr, hidden, n_layers, first_token, xi, r_state, workspace,
                     x_rec=None, idx=None, w=None, pidx=None, pw=None, y_rec=None, status=None,
                     stream=None, r_rec=None):
    """moe_engine_chain_mlp: the chain with the full prerouter head of every
    layer (head_arr from head_mlp_array)."""
    n_tokens = xi.shape[0]
    _check(lib().moe_engine_chain_mlp(ctypes.byref(spec), table.handle, _ptr(layer_arr), _ptr(head_arr),
                                      int(hidden), n_layers, first_token, n_tokens, _ptr(xi), _ptr(r_state),
                                      _ptr(x_rec), _ptr(r_rec), _ptr(idx), _ptr(w), _ptr(pidx), _ptr(pw),
                                      _ptr(y_rec), _ptr(status), _ptr(workspace),
                                      workspace.numel() * workspace.element_size(), _stream(stream)),
           "moe_engine_chain_mlp")
