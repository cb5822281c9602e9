"""The decode step (and ragged prefill pass) of a Llama-style decoder, float64.

Test infrastructure only (see the package docstring).

What is computed (paper, "Design and Implementation": a row is one token's
hidden state, dense mode runs every layer; "Invariants": every layer writes
its own KV; Algorithm 1 names the SwiGLU product; greedy decoding as in the
paper's evaluation).  For the rows of one pass, each at position ``pos`` of
its sequence and writing cache slot ``slot``:

  x  = E[token]                                    (float residual stream)
  for each layer l:
     h  = R(rmsnorm(x) * g_attn)
     q, k, v = h Wq^T, h Wk^T, h Wv^T
     q, k = rope(q, pos), rope(k, pos);  q, k, v = R(q), R(k), R(v)
     cache[l][slot] = (k, v)                       (all rows, before attention)
     o_h = softmax(q_h . K^T / sqrt(d)) V over the sequence's keys 0..pos,
           K, V read through the block table, KV head floor(h*n_kv/n_q)
     x += R(o) Wo^T
     h2 = R(rmsnorm(x) * g_mlp)
     x += R(silu(h2 Wg^T) * (h2 Wu^T)) Wd^T
  z  = R(rmsnorm(x) * g_final) Wlm^T  for the rows that return logits
  logits = R(z);  token = lowest index of max z

R is round-to-nearest-even to bf16 (the tensors stored between kernels);
everything else is float64.  Paging and split-K only change summation
order, so this plain form is the result the device path must reach.
"""
from __future__ import annotations

import numpy as np

from . import numerics as nm
from .kvcache import PagedKV

MATS = ("wq", "wk", "wv", "wo", "w_gate", "w_up", "w_down")
NORMS = ("attn_norm", "mlp_norm")


class GeneratedWeights:
    """Float64 weights drawn from the seeded input generator, layer by layer.

    Norm gains default to 1 (the random-init reading: N(0, 0.02) applies to
    matrices and embeddings only).  ``overrides`` maps (name, layer) to an
    explicit array for planted special cases; layer is -1 for the
    embedding, lm_head and final norm.
    """

    def __init__(self, model, seed, overrides=None, dist=None, cache=False):
        self.m = model
        self.seed = seed
        self.over = dict(overrides or {})
        self.dist = dist or ("normal", model.weight_sigma)
        self.cache = {} if cache else None

    def shape(self, name):
        m = self.m
        H, F = m.hidden, m.ffn
        return {
            "wq": (m.n_q_heads * m.head_dim, H), "wk": (m.n_kv_heads * m.head_dim, H),
            "wv": (m.n_kv_heads * m.head_dim, H), "wo": (H, m.n_q_heads * m.head_dim),
            "w_gate": (F, H), "w_up": (F, H), "w_down": (H, F),
            "embed": (m.vocab, H), "lm_head": (m.vocab, H),
            "attn_norm": (H,), "mlp_norm": (H,), "final_norm": (H,),
        }[name]

    def key(self, name, layer):
        from workloads.configs import weight_key
        return weight_key(self.seed, self.m, name, layer)

    def get(self, name, layer=-1):
        k = (name, layer)
        if k in self.over:
            return np.asarray(self.over[k], np.float64)
        if self.cache is not None and k in self.cache:
            return self.cache[k]
        shp = self.shape(name)
        if name in NORMS or name == "final_norm":
            w = np.ones(shp)
        else:
            from workloads import gen
            n = int(np.prod(shp))
            w = nm.from_bf16_bits(gen.bf16_bits_np(self.key(name, layer), n, self.dist)).reshape(shp)
        if self.cache is not None:
            self.cache[k] = w
        return w

    def rows(self, name, ids):
        """Rows of the embedding (or lm_head) matrix without drawing the rest."""
        k = (name, -1)
        if k in self.over:
            return np.asarray(self.over[k], np.float64)[np.asarray(ids)]
        from workloads import gen
        H = self.m.hidden
        key = self.key(name, -1)
        out = np.empty((len(ids), H))
        for i, t in enumerate(np.asarray(ids)):
            out[i] = nm.from_bf16_bits(gen.bf16_bits_np(key, H, self.dist, start=int(t) * H))
        return out


def _matmul(x, w):
    return x @ w.T


def forward(model, W, kv: PagedKV, batch, tokens, logit_rows, *, want_hidden=False,
            lm_chunk=16384, x0=None, layers=None):
    """One pass over the rows described by ``batch`` (see kvcache.build_batch).

    tokens     : int [R] token id of each row
    logit_rows : int [n_out] rows whose logits are returned (None: no head)
    x0         : optional residual stream [R][hidden] to start from instead of
                 the embedding rows (the pass then covers only ``layers``)
    layers     : the layer indices to run, in order (default: all)
    Writes every row's K, V into ``kv`` at every layer it runs.
    Returns dict(z [n_out][V] float64, logits (bf16 values, float64), ids int32,
    and optionally the final residual stream x).
    """
    m = model
    Hq, Hk, d = m.n_q_heads, m.n_kv_heads, m.head_dim
    grp = Hq // Hk
    tokens = np.asarray(tokens)
    R = len(tokens)
    pos = batch["pos"]
    slot = batch["slot"]
    cu = batch["cu_q"]
    kv_len = batch["kv_len"]
    table = batch["block_table"]
    bs = kv.block
    x = W.rows("embed", tokens) if x0 is None else np.array(x0, dtype=np.float64)
    for layer in (range(m.n_layers) if layers is None else layers):
        # ---- attention block
        h = nm.bf16_round(nm.rmsnorm(x, W.get("attn_norm", layer), m.rms_eps))
        q = _matmul(h, W.get("wq", layer)).reshape(R, Hq, d)
        k = _matmul(h, W.get("wk", layer)).reshape(R, Hk, d)
        v = _matmul(h, W.get("wv", layer)).reshape(R, Hk, d)
        q = nm.bf16_round(nm.rope(q, pos, m.rope_theta))
        k = nm.bf16_round(nm.rope(k, pos, m.rope_theta))
        v = nm.bf16_round(v)
        kv.write(layer, slot, k, v)
        o = np.empty((R, Hq, d))
        for i in range(len(kv_len)):
            r0, r1 = int(cu[i]), int(cu[i + 1])
            if r1 == r0:
                continue
            n = int(kv_len[i])
            jj = np.arange(n)
            sl = table[i, jj // bs].astype(np.int64) * bs + jj % bs
            K, V = kv.read(layer, sl)                      # [n][Hk][d]
            for r in range(r0, r1):
                p = int(pos[r])
                for hh in range(Hq):
                    g = hh // grp
                    o[r, hh] = nm.attend(q[r, hh], K[:p + 1, g], V[:p + 1, g])
        o = nm.bf16_round(o.reshape(R, Hq * d))
        x = x + _matmul(o, W.get("wo", layer))
        # ---- MLP block
        h2 = nm.bf16_round(nm.rmsnorm(x, W.get("mlp_norm", layer), m.rms_eps))
        a = nm.bf16_round(nm.silu(_matmul(h2, W.get("w_gate", layer))) * _matmul(h2, W.get("w_up", layer)))
        x = x + _matmul(a, W.get("w_down", layer))
    if logit_rows is None:
        return {"x": x}
    lr = np.asarray(logit_rows, np.int64)
    hf = nm.bf16_round(nm.rmsnorm(x[lr], W.get("final_norm", -1), m.rms_eps))
    z = np.empty((len(lr), m.vocab))
    if ("lm_head", -1) in W.over:
        z[:] = _matmul(hf, W.get("lm_head", -1))
    else:
        from workloads import gen
        key = W.key("lm_head", -1)
        H = m.hidden
        for v0 in range(0, m.vocab, lm_chunk):
            v1 = min(m.vocab, v0 + lm_chunk)
            wl = nm.from_bf16_bits(gen.bf16_bits_np(key, (v1 - v0) * H, W.dist, start=v0 * H)).reshape(v1 - v0, H)
            z[:, v0:v1] = _matmul(hf, wl)
    out = {"z": z, "logits": nm.bf16_round(z), "ids": nm.argmax_lowest(z)}
    if want_hidden:
        out["x"] = x
    return out
