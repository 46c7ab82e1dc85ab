"""Seeded generators for the five workloads.

Every array is a pure function of a key ``(workload, layer, expert, tensor)``
through ``numpy.random.SeedSequence``, so any expert can be regenerated on its
own (the CPU oracle builds only the experts a token touches).

Shapes (hidden ``d``, experts ``E``, top ``K``, shared ``S``, expert
intermediate ``I``, LoRA rank ``r``):

* ``tiny``   d 512,  E 16,  K 2, S 0, I 256,  r 8   (one layer)
* ``moe35b`` d 2048, E 256, K 8, S 1, I 512,  r 16  (35B-class layer; also the
  40-layer stack and the batched / prefill workload)
* ``tier8b`` d 4096, E 64,  K 4, S 0, I 1024, r 16  (24 layers, host staging)

Value distributions:

* Expert weights are drawn directly in the stored int4 group-64 format:
  uniform codes in 0..15, and per group an fp16 scale ``s`` uniform in
  ``[0.9, 1.1] * 0.02 / sqrt(255 / 12)`` and an fp16 zero
  ``z = -7.5 s + 0.005 * u``, ``u`` uniform in ``[-1, 1]``.  The
  reconstructed weights then have mean ~0 and standard deviation ~0.02,
  the scale of N(0, 0.02) weights after int4 quantization.
* LoRA ``A [r, in]`` ~ N(0, 1/r) and ``B [out, r]`` ~ N(0, 0.01) (second
  argument = standard deviation), stored fp16.
* Router and prerouter head weights ``[E, d]`` ~ N(0, 0.02), fp16.
* Token draws ``xi [d]`` ~ N(0, 1), fp32 (the layer input is their RMS
  normalization, computed by the code under test).
* fp32 master weights N(0, 0.02) for the quantizer test.
* Optionally (``bundle(..., quantized=True)``), expert weights made as the
  configurations describe them: fp32 N(0, 0.02) masters quantized int4
  asymmetric per group of 64 inputs (group minimum and maximum in fp32,
  fp16 ``s = (hi - lo) / 15`` and ``z = lo``, codes ``rint((w - z) / s)``
  taken in fp32 and clamped to 0..15, code 0 where ``s`` is 0).  This is
  the recipe of the input data; the arithmetic under test only reads the
  codes and (s, z) it produces.
"""

import numpy as np

__all__ = [
    "WORKLOADS", "Workload", "rng", "int4_projection", "fp32_weights",
    "lora_pair", "bundle", "router_weights", "token_draws", "zipf_logits",
    "mixing", "ar1_token_draws", "prerouter_mlp", "quantized_projection",
]


class Workload:
    def __init__(self, wid, name, d, e, k, s, inter, r, layers=1):
        self.wid, self.name = wid, name
        self.d, self.E, self.K, self.S, self.I, self.r = d, e, k, s, inter, r
        self.layers = layers
        self.a_std = 1.0 / r
        self.b_std = 0.01
        self.w_std = 0.02
        self.lora_alpha = 2 * r           # alpha / r = 32 / 16 = 2

    @property
    def lora_scale(self):
        return self.lora_alpha / self.r

    def __repr__(self):
        return "Workload(%s)" % self.name


WORKLOADS = {
    "tiny": Workload(0, "tiny", 512, 16, 2, 0, 256, 8),
    "moe35b": Workload(1, "moe35b", 2048, 256, 8, 1, 512, 16, layers=40),
    "tier8b": Workload(4, "tier8b", 4096, 64, 4, 0, 1024, 16, layers=24),
}

# tensor ids inside a key
_T_Q = {"gate": 0, "up": 1, "down": 2}
_T_SZ = {"gate": 3, "up": 4, "down": 5}
_T_A = {"gate": 6, "up": 7, "down": 8}
_T_B = {"gate": 9, "up": 10, "down": 11}
_ROUTER_ID = 1 << 20
_TOKEN_BASE = 10 ** 6


def rng(*key):
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([int(k) for k in key])))


def int4_projection(key_q, key_sz, out_dim, in_dim, w_std=0.02):
    """Packed codes ``[out, in/2]`` (even input in the low nibble), fp16 s, z."""
    q = np.frombuffer(rng(*key_q).bytes(out_dim * in_dim // 2), dtype=np.uint8)
    q = q.reshape(out_dim, in_dim // 2).copy()
    g = rng(*key_sz)
    groups = (out_dim, in_dim // 64)
    base = w_std / np.sqrt(255.0 / 12.0)
    s = (base * g.uniform(0.9, 1.1, size=groups)).astype(np.float16)
    z = (-7.5 * s.astype(np.float64) + 0.005 * g.uniform(-1.0, 1.0, size=groups)).astype(np.float16)
    return q, s, z


def quantized_projection(key, out_dim, in_dim, std=0.02):
    """fp32 N(0, std) masters of ``key`` quantized int4 per group of 64 inputs
    (the input recipe above): packed codes ``[out, in/2]``, fp16 s, z."""
    w = fp32_weights(key, out_dim, in_dim, std).reshape(out_dim, in_dim // 64, 64)
    lo = w.min(axis=2)
    hi = w.max(axis=2)
    s = ((hi - lo) / np.float32(15.0)).astype(np.float16)
    z = lo.astype(np.float16)
    s32 = s.astype(np.float32)[:, :, None]
    z32 = z.astype(np.float32)[:, :, None]
    with np.errstate(divide="ignore", invalid="ignore"):
        c = np.rint((w - z32) / s32)
    c = np.where(s32 == 0, 0.0, c)
    q = np.clip(c, 0, 15).astype(np.uint8).reshape(out_dim, in_dim)
    packed = (q[:, 0::2] | (q[:, 1::2] << 4)).astype(np.uint8)
    return np.ascontiguousarray(packed), s, z


def fp32_weights(key, out_dim, in_dim, std=0.02):
    return rng(*key).normal(0.0, std, size=(out_dim, in_dim)).astype(np.float32)


def lora_pair(key_a, key_b, out_dim, in_dim, r, a_std, b_std):
    a = rng(*key_a).normal(0.0, a_std, size=(r, in_dim)).astype(np.float16)
    b = rng(*key_b).normal(0.0, b_std, size=(out_dim, r)).astype(np.float16)
    return a, b


def bundle(wl, layer, expert, lora=True, lora_on=("gate", "up", "down"), b_std=None, quantized=False):
    """Expert ``expert`` of ``layer`` (ids ``E .. E+S-1`` are the shared experts).
    ``b_std`` overrides the workload's std of the LoRA ``B`` entries: the
    delta ``scale * B A`` then has entries of std ``scale * b_std * sqrt(r) * a_std``.
    ``quantized``: weights quantized from fp32 N(0, w_std) masters instead of
    drawn directly as codes."""
    dims = {"gate": (wl.I, wl.d), "up": (wl.I, wl.d), "down": (wl.d, wl.I)}
    out = {"lora": {}}
    for p, (o, i) in dims.items():
        if quantized:
            out[p] = quantized_projection((wl.wid, layer, expert, _T_Q[p], 1), o, i, wl.w_std)
        else:
            out[p] = int4_projection((wl.wid, layer, expert, _T_Q[p]),
                                     (wl.wid, layer, expert, _T_SZ[p]), o, i, wl.w_std)
        if lora and p in lora_on:
            out["lora"][p] = lora_pair((wl.wid, layer, expert, _T_A[p]),
                                       (wl.wid, layer, expert, _T_B[p]),
                                       o, i, wl.r, wl.a_std, wl.b_std if b_std is None else b_std)
        else:
            out["lora"][p] = None
    return out


def router_weights(wl, layer, kind):
    """fp16 ``[E, d]``; ``kind`` 0 = the layer's router, 1 = its prerouter head."""
    return rng(wl.wid, layer, _ROUTER_ID, kind).normal(0.0, 0.02, size=(wl.E, wl.d)).astype(np.float16)


def prerouter_mlp(wl, layer, hidden=512):
    """Full prerouter head of ``layer`` (fp16, N(0, 0.02) entries): ``w1``
    ``[hidden, d + 2E]``, ``b1 [hidden]``, ``w2 [E, hidden]``, ``b2 [E]``, and
    the residual path ``wl`` drawn as the next layer's router."""
    g = rng(wl.wid, layer, _ROUTER_ID, 2)
    w1 = g.normal(0.0, 0.02, size=(hidden, wl.d + 2 * wl.E)).astype(np.float16)
    b1 = g.normal(0.0, 0.02, size=hidden).astype(np.float16)
    w2 = g.normal(0.0, 0.02, size=(wl.E, hidden)).astype(np.float16)
    b2 = g.normal(0.0, 0.02, size=wl.E).astype(np.float16)
    return {"w1": w1, "b1": b1, "w2": w2, "b2": b2, "wl": router_weights(wl, layer + 1, 0)}


def token_draws(wl, t0, count, stream=0):
    """fp32 ``[count, d]`` N(0, 1) draws for tokens ``t0 .. t0+count-1``."""
    return np.stack([rng(wl.wid, _TOKEN_BASE + t, stream).standard_normal(wl.d).astype(np.float32)
                     for t in range(t0, t0 + count)])


def zipf_logits(wl, tokens, seed=0, exponent=1.1):
    """Synthetic router logits ``[T, E]`` fp32 with Zipf popularity.

    ``p_e`` proportional to ``rank_e ** -exponent`` over a seeded permutation of
    ranks; ``l[t, e] = log p_e + Gumbel(0, 1)``, so the top-K of a row is a
    sample of K experts without replacement from ``p``.
    """
    g = rng(wl.wid, 2 << 20, seed)
    ranks = g.permutation(wl.E) + 1
    logp = -exponent * np.log(ranks.astype(np.float64))
    logp -= np.log(np.sum(np.exp(logp)))
    gumbel = g.gumbel(0.0, 1.0, size=(tokens, wl.E))
    return (logp[None, :] + gumbel).astype(np.float32)


def mixing(wl, layer):
    """Residual-mixing stand-in for attention: fp16 ``D [d]`` ~ N(0, 0.5) and a permutation."""
    g = rng(wl.wid, layer, 3 << 20)
    d = g.normal(0.0, 0.5, size=wl.d).astype(np.float16)
    perm = g.permutation(wl.d).astype(np.int32)
    return d, perm


def ar1_token_draws(wl, count, rho, stream=0):
    """AR(1) token draws ``xi_{t+1} = rho xi_t + sqrt(1 - rho^2) eps``, fp32 ``[count, d]``."""
    eps = token_draws(wl, 0, count, stream=stream).astype(np.float64)
    out = np.empty_like(eps)
    out[0] = eps[0]
    c = np.sqrt(1.0 - rho * rho)
    for t in range(1, count):
        out[t] = rho * out[t - 1] + c * eps[t]
    return out.astype(np.float32)
