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

Routed mode (``route=``; paper Section 3.1, Algorithm 1 and the appendix
"Route-Guided Cohort Execution at the Kernel Level"): in each routed layer
(the last n_routed layers) the route tape gives every row RUN or
Project-Only and a weight w.  Maps: run[] / proj[] list the rows of each
cohort (n_r + n_p = rows).  Every row still writes the layer's own K, V
(Invariant 1); a Project-Only row reads no KV and its attention output is
zero.  Then, with X = R(rmsnorm(x) * g_mlp) for every row:

     x[run]  += w[run]     * (R(silu(X[run] Wg^T) * (X[run] Wu^T)) Wd^T)
     x[proj] += (1-w[proj]) * (R(silu(X[proj] Pg^T) * (X[proj] Pu^T)) Pd^T)

with the layer's projector weights Pg, Pu [proj_ffn][hidden], Pd.  A RUN row
with w = 1 computes exactly what dense mode computes.

R is round-to-nearest-even to bf16 (the tensors stored between kernels);
everything else is float64.  Paging and split-K only change summation
order, so this plain form is the result the device path must reach.

``forward(..., dtype="f32")`` is the contract-mode variant: the same steps and
rounding points with every product, sum, norm and softmax in float32 (the
residual stream too), as an fp32-accumulating implementation computes them.
It does not define the result; it measures how far a correct float32
implementation may drift from the float64 one on a given input.
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
            "p_gate": (m.proj_dim, H), "p_up": (m.proj_dim, H), "p_down": (H, m.proj_dim),
        }[name]

    def key(self, name, layer):
        from workloads.configs import weight_key
        return weight_key(self.seed, self.m, name, layer)

    def get(self, name, layer=-1, dtype=np.float64):
        k = (name, layer)
        if k in self.over:
            return np.asarray(self.over[k], dtype)
        if self.cache is not None and k in self.cache:
            return self.cache[k].astype(dtype, copy=False)
        shp = self.shape(name)
        if name in NORMS or name == "final_norm":
            w = np.ones(shp, dtype)
        else:
            from workloads import gen
            n = int(np.prod(shp))
            w = gen.bf16_values_np(self.key(name, layer), n, self.dist, dtype=dtype).reshape(shp)
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


DTYPES = {"f64": np.float64, "f32": np.float32}


def route_maps(run_row):
    """Algorithm 1's maps of one routed layer: the rows of the RUN cohort, of
    the Project-Only cohort, and their counts."""
    run_row = np.asarray(run_row, bool)
    run = np.nonzero(run_row)[0]
    proj = np.nonzero(~run_row)[0]
    return run, proj, len(run), len(proj)


def _swiglu_down(X, g, u, d, F, R):
    """R(silu(X g^T) * (X u^T)) d^T (the MLP, or a projector of the same form)."""
    return _matmul(R(nm.silu(_matmul(X, g), F) * _matmul(X, u)), d)


def forward(model, W, kv: PagedKV, batch, tokens, logit_rows, *, want_hidden=False,
            lm_chunk=16384, x0=None, layers=None, dtype="f64", route=None):
    """One pass over the rows described by ``batch`` (see kvcache.build_batch).

    tokens     : int [R] token id of each row
    logit_rows : int [n_out] rows whose logits are returned (None: no head)
    x0         : optional residual stream [R][hidden] to start from instead of
                 the embedding rows (the pass then covers only ``layers``)
    layers     : the layer indices to run, in order (default: all)
    Writes every row's K, V into ``kv`` at every layer it runs.
    dtype      : "f64" (the definition) or "f32" (contract-mode variant)
    route      : None (dense mode) or (run [n_routed][rows] bool, w [n_routed][rows])
                 for the model's routed layers (the last n_routed)
    Returns dict(z [n_out][V] float64, logits (bf16 values, float64), ids int32,
    and optionally the final residual stream x).
    """
    F = DTYPES[dtype]

    def R(a):  # a contract rounding point
        return nm.bf16_round(a).astype(F)

    def mat(name, layer=-1):
        return W.get(name, layer, F)

    m = model
    Hq, Hk, d = m.n_q_heads, m.n_kv_heads, m.head_dim
    grp = Hq // Hk
    tokens = np.asarray(tokens)
    n_rows = len(tokens)
    pos = batch["pos"]
    slot = batch["slot"]
    cu = batch["cu_q"]
    kv_len = batch["kv_len"]
    table = batch["block_table"]
    bs = kv.block
    x = (W.rows("embed", tokens) if x0 is None else np.array(x0, dtype=np.float64)).astype(F)
    for layer in (range(m.n_layers) if layers is None else layers):
        routed = route is not None and layer >= m.first_routed
        if routed:
            lr_i = layer - m.first_routed
            run, proj, n_r, n_p = route_maps(route[0][lr_i])
            wl = np.asarray(route[1][lr_i], F)
            project_only = np.zeros(n_rows, bool)
            project_only[proj] = True
        # ---- attention block (every row writes its K, V)
        h = R(nm.rmsnorm(x, W.get("attn_norm", layer), m.rms_eps, F))
        q = _matmul(h, mat("wq", layer)).reshape(n_rows, Hq, d)
        k = _matmul(h, mat("wk", layer)).reshape(n_rows, Hk, d)
        v = _matmul(h, mat("wv", layer)).reshape(n_rows, Hk, d)
        q = R(nm.rope(q, pos, m.rope_theta, F))
        k = R(nm.rope(k, pos, m.rope_theta, F))
        v = R(v)
        kv.write(layer, slot, k, v)
        o = np.empty((n_rows, Hq, d), F)
        for i in range(len(kv_len)):
            r0, r1 = int(cu[i]), int(cu[i + 1])
            if r1 == r0:
                continue
            n = int(kv_len[i])
            jj = np.arange(n)
            sl = table[i, jj // bs].astype(np.int64) * bs + jj % bs
            K, V = kv.read(layer, sl)                      # [n][Hk][d]
            K, V = K.astype(F), V.astype(F)
            for r in range(r0, r1):
                if routed and project_only[r]:
                    o[r] = 0  # a Project-Only row reads no KV and emits zero
                    continue
                p = int(pos[r])
                for hh in range(Hq):
                    g = hh // grp
                    o[r, hh] = nm.attend(q[r, hh], K[:p + 1, g], V[:p + 1, g], F)
        o = R(o.reshape(n_rows, Hq * d))
        x = x + _matmul(o, mat("wo", layer))
        # ---- MLP block
        h2 = R(nm.rmsnorm(x, W.get("mlp_norm", layer), m.rms_eps, F))
        if not routed:
            x = x + _swiglu_down(h2, mat("w_gate", layer), mat("w_up", layer), mat("w_down", layer), F, R)
        else:
            # RUN cohort: the MLP, weight w; Project-Only cohort: the projector, weight 1 - w
            x = x.copy()
            if n_r:
                y = _swiglu_down(h2[run], mat("w_gate", layer), mat("w_up", layer), mat("w_down", layer), F, R)
                x[run] = x[run] + wl[run, None] * y
            if n_p:
                y = _swiglu_down(h2[proj], mat("p_gate", layer), mat("p_up", layer), mat("p_down", layer), F, R)
                x[proj] = x[proj] + (F(1) - wl[proj, None]) * y
    if logit_rows is None:
        return {"x": x.astype(np.float64)}
    lr = np.asarray(logit_rows, np.int64)
    hf = R(nm.rmsnorm(x[lr], W.get("final_norm", -1), m.rms_eps, F))
    z = np.empty((len(lr), m.vocab), F)
    if ("lm_head", -1) in W.over:
        z[:] = _matmul(hf, mat("lm_head", -1))
    else:
        from workloads import gen
        key = W.key("lm_head", -1)
        H = m.hidden
        for v0 in range(0, m.vocab, lm_chunk):
            v1 = min(m.vocab, v0 + lm_chunk)
            wl = gen.bf16_values_np(key, (v1 - v0) * H, W.dist, start=v0 * H, dtype=F).reshape(v1 - v0, H)
            z[:, v0:v1] = _matmul(hf, wl)
    z = z.astype(np.float64)
    out = {"z": z, "logits": nm.bf16_round(z), "ids": nm.argmax_lowest(z)}
    if want_hidden:
        out["x"] = x.astype(np.float64)
    return out
