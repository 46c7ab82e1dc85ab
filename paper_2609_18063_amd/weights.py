"""Place expert bundles, routers and heads in device memory (plumbing).

Weights arrive as host arrays in the stored format of ``include/moe_api.h``
(packed int4 codes, fp16 scales and zeros, fp16 LoRA factors).  They are
packed into one host byte buffer per layer, with every tensor 256-byte
aligned and each (scale, zero) pair interleaved. The buffer is copied to the
device in one transfer, and the pointers into it are returned as
``MoeBundle`` structs for the slot table.
"""

import numpy as np

from .binding import MoeBundle, MoeProj

_ALIGN = 256
_PROJ = ("gate", "up", "down")


def _arrays(bundle):
    lo = bundle.get("lora") or {}
    out = []
    for p in _PROJ:
        q, s, z = bundle[p]
        sz = np.stack([np.asarray(s, np.float16), np.asarray(z, np.float16)], -1)
        out.append((p, "q", np.ascontiguousarray(q, dtype=np.uint8)))
        out.append((p, "sz", np.ascontiguousarray(sz)))
        if lo.get(p) is not None:
            out.append((p, "a", np.ascontiguousarray(lo[p][0], dtype=np.float16)))
            out.append((p, "b", np.ascontiguousarray(lo[p][1], dtype=np.float16)))
    return out


def pack_host(bundles, extra=()):
    """Pack ``bundles`` (list of dicts) and ``extra`` arrays (e.g. router,
    head) into one uint8 host buffer.  Returns (buffer, bundle offsets,
    extra offsets)."""
    items, off = [], 0
    boffs = []
    for b in bundles:
        d = {}
        for p, kind, arr in _arrays(b):
            d[(p, kind)] = off
            items.append((off, arr))
            off = (off + arr.nbytes + _ALIGN - 1) // _ALIGN * _ALIGN
        boffs.append(d)
    eoffs = []
    for arr in extra:
        arr = np.ascontiguousarray(arr)
        eoffs.append(off)
        items.append((off, arr))
        off = (off + arr.nbytes + _ALIGN - 1) // _ALIGN * _ALIGN
    buf = np.zeros(max(off, _ALIGN), dtype=np.uint8)
    for o, arr in items:
        buf[o:o + arr.nbytes] = arr.reshape(-1).view(np.uint8)
    return buf, boffs, eoffs


def device_bundles(base_ptr, boffs):
    """MoeBundle structs pointing into a device copy of a packed buffer."""
    out = []
    for d in boffs:
        projs = []
        for p in _PROJ:
            a = d.get((p, "a"))
            b = d.get((p, "b"))
            projs.append(MoeProj(base_ptr + d[(p, "q")], base_ptr + d[(p, "sz")],
                                 None if a is None else base_ptr + a,
                                 None if b is None else base_ptr + b))
        out.append(MoeBundle(*projs))
    return out


def upload(buf, device="cuda"):
    """Copy a packed host buffer to a new device tensor (one transfer)."""
    import torch
    return torch.from_numpy(buf).to(device)


def bind_layer(table, layer, dev_buf, boffs, slot_of_id=None):
    """Bind every bundle of a packed layer: id ``i`` goes to slot
    ``slot_of_id[i]`` (identity if None).  Returns the MoeBundle list."""
    bundles = device_bundles(dev_buf.data_ptr(), boffs)
    for i, mb in enumerate(bundles):
        s = i if slot_of_id is None else int(slot_of_id[i])
        table.bind(layer, i, s, mb, keep=dev_buf)
    return bundles


def extra_tensor(dev_buf, off, shape, dtype):
    """View of an ``extra`` array (router, head) inside a device buffer."""
    import torch
    n = int(np.prod(shape)) * torch.empty(0, dtype=dtype).element_size()
    return dev_buf[off:off + n].view(dtype).view(*shape)
