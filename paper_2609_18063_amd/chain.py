"""Multi-layer decode chain with prediction-as-routing, driven through the C ABI.

Per token t and layer N (§3.2, Motivation and Prediction-as-routing): the
head of layer N runs on layer N's input and writes layer N+1's routing for
token t+1; layer N+1 at token t+1 routes by that prediction.  Layer 0 and
every layer of the first token use their own router.  The predictions live
in two device buffers indexed by the parity of the token they are for, so
the head of layer N at token t+1 never overwrites the routing that layer N+1
is about to use at token t+1.

The attention that precedes every MoE layer in the paper's decoder is
replaced by the O(d) residual mixing of ``moe_chain_mix_rmsnorm``.

With ``heads_mlp`` the prediction comes from the full prerouter head
(``moe_preroute_mlp``, §3.2 Head): its input is layer N's x, the experts layer N
routed to at this token and those at the previous token. At decode those sets
are themselves the predictions of the head before (prediction-as-routing), so
the head sees its own chain's predictions rather than the true routing (the
paper's feature drift).
"""

import torch

from . import binding as B


class DeviceChain:
    """Device state of one decode chain.

    ``layers`` is a list of dicts with device tensors ``router`` and
    ``head`` (fp16 [E, d]; the last layer's head may be None), ``mix_d``
    (fp16 [d]) and ``mix_perm`` (int32 [d]).  Layer ``N``'s experts are
    bound in ``table`` at table layer ``N``.
    """

    def __init__(self, spec, table, layers, consumers=None, heads_mlp=None):
        self.spec, self.table, self.layers = spec, table, layers
        self.L = len(layers)
        self.consumers = set(range(1, self.L)) if consumers is None else set(consumers)
        d, K, E = spec.d_model, spec.top_k, spec.n_experts
        n = K + spec.n_shared
        dev = "cuda"
        self.ws = torch.zeros(B.workspace_bytes(spec, 1), dtype=torch.uint8, device=dev)
        self.r = torch.zeros(1, d, dtype=torch.float32, device=dev)
        self.x = torch.empty(1, d, dtype=torch.float16, device=dev)
        self.xi = torch.zeros(1, d, dtype=torch.float32, device=dev)
        self.own_idx = torch.empty(1, K, dtype=torch.int32, device=dev)
        self.own_w = torch.empty(1, K, dtype=torch.float32, device=dev)
        self.pred_idx = torch.zeros(2, self.L, 1, K, dtype=torch.int32, device=dev)
        self.pred_w = torch.zeros(2, self.L, 1, K, dtype=torch.float32, device=dev)
        self.ye = torch.empty(1, n, d, dtype=torch.float32, device=dev)
        self.status = torch.zeros(1, dtype=torch.int32, device=dev)
        self.graphs = {}
        # full prerouter heads: per layer a moe_head_mlp struct (binding.head_mlp)
        # or None (the linear head, moe_preroute); the routing each layer used
        # at the last two tokens, by token parity, is their one-hot input
        self.heads_mlp = heads_mlp
        if heads_mlp is not None:
            hidden = max(h.hidden for h in heads_mlp if h is not None)
            self.ws_mlp = torch.zeros(B.preroute_mlp_workspace_bytes(spec, hidden, 1), dtype=torch.uint8,
                                      device=dev)
            self.used_idx = torch.full((2, self.L, 1, K), -1, dtype=torch.int32, device=dev)

    def uses_prediction(self, t, n):
        return t > 0 and n > 0 and n in self.consumers

    def enqueue_token(self, t, record=None):
        """Enqueue token ``t`` (its draw already in ``self.xi``) on the current stream."""
        s = self.spec
        B.chain_token_start(self.xi, self.r)
        for n, lay in enumerate(self.layers):
            B.chain_mix_rmsnorm(lay["mix_d"], lay["mix_perm"], self.r, self.x)
            if record is not None:
                record["r"][t, n].copy_(self.r[0])
            if self.uses_prediction(t, n):
                idx, w = self.pred_idx[t % 2, n], self.pred_w[t % 2, n]
            else:
                B.route(s, self.x, lay["router"], self.own_idx, self.own_w, self.ws)
                idx, w = self.own_idx, self.own_w
            mlp = self.heads_mlp[n] if self.heads_mlp is not None else None
            if n + 1 < self.L and mlp is not None:
                nxt = (t + 1) % 2
                prev = self.used_idx[(t - 1) % 2, n] if t > 0 else None
                B.preroute_mlp(s, mlp, self.x, idx, prev, self.pred_idx[nxt, n + 1], self.pred_w[nxt, n + 1],
                               self.ws_mlp)
                self.used_idx[t % 2, n].copy_(idx)
            elif n + 1 < self.L and lay.get("head") is not None:
                nxt = (t + 1) % 2
                B.preroute(s, self.x, lay["head"], self.pred_idx[nxt, n + 1], self.pred_w[nxt, n + 1],
                           self.ws)
            ye = self.ye if record is None else record["ye"][t, n]
            B.expert_ffn(s, self.table, n, self.x, idx, ye, self.status, self.ws)
            B.combine_add(s, ye, w, self.r)
            if record is not None:
                record["r_post"][t, n].copy_(self.r[0])
                record["x"][t, n].copy_(self.x[0])
                record["idx"][t, n].copy_(idx[0])
                record["w"][t, n].copy_(w[0])
                if n + 1 < self.L and (lay.get("head") is not None or mlp is not None):
                    nxt = (t + 1) % 2
                    record["pidx"][t, n].copy_(self.pred_idx[nxt, n + 1, 0])
                    record["pw"][t, n].copy_(self.pred_w[nxt, n + 1, 0])

    def reset(self):
        self.r.zero_()

    def new_record(self, T):
        s = self.spec
        n = s.top_k + s.n_shared
        L, d, K = self.L, s.d_model, s.top_k
        dev = "cuda"
        return {
            "x": torch.zeros(T, L, d, dtype=torch.float16, device=dev),
            "r": torch.zeros(T, L, d, dtype=torch.float32, device=dev),
            "r_post": torch.zeros(T, L, d, dtype=torch.float32, device=dev),
            "idx": torch.zeros(T, L, K, dtype=torch.int32, device=dev),
            "w": torch.zeros(T, L, K, dtype=torch.float32, device=dev),
            "pidx": torch.full((T, L, K), -1, dtype=torch.int32, device=dev),
            "pw": torch.zeros(T, L, K, dtype=torch.float32, device=dev),
            "ye": torch.zeros(T, L, 1, n, d, dtype=torch.float32, device=dev),
        }

    def run_recorded(self, xi_tokens):
        """Eager run over fp32 draws ``xi_tokens [T, d]`` (device), recording every layer."""
        T = xi_tokens.shape[0]
        rec = self.new_record(T)
        self.reset()
        for t in range(T):
            self.xi.copy_(xi_tokens[t:t + 1])
            self.enqueue_token(t, record=rec)
        torch.cuda.synchronize()
        return rec

    def capture(self, stream=None):
        """Capture the three token graphs: first token, even and odd later tokens."""
        stream = stream or torch.cuda.Stream()
        for key, t in (("first", 0), ("odd", 1), ("even", 2)):
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g, stream=stream):
                self.enqueue_token(t)
            self.graphs[key] = g

    def replay_token(self, t):
        key = "first" if t == 0 else ("odd" if t % 2 else "even")
        self.graphs[key].replay()
