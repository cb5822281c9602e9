"""The five synthetic decode workloads and their seeded batch recipes.

Model shapes follow the Llama-3 family the paper serves (decoder-only, GQA,
RMSNorm, rotary positions, SwiGLU MLP).  Batch shapes stand in for the
paper's serving workloads: small-batch weight-streaming decode, a shared
few-shot prefix held once in the paged cache (the BBH-like case), a long
prompt prefilled in chunks beside running decodes (the GSM8K-like case), and
a heavy-tailed context-length mix (the CoQA-like case).  No benchmark item
is used or reproduced; every value is drawn from the seeded generators.

Nothing here computes any part of the decode step.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

from . import gen

BLOCK = 16  # tokens per KV block


@dataclass(frozen=True)
class ModelCfg:
    name: str
    n_layers: int
    hidden: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    ffn: int
    vocab: int
    rope_theta: float = 500000.0
    rms_eps: float = 1e-5
    max_pos: int = 8192
    weight_sigma: float = 0.02
    kv_sigma: float = 1.0
    # routed mode: the last `routed_layers` layers are routed (0: the last
    # half, as the paper's skipper routes the last 16 of 32), each with a
    # SwiGLU projector of width proj_ffn (0: ffn / 16 rounded up to 64)
    routed_layers: int = 0
    proj_ffn: int = 0

    @property
    def n_routed(self):
        return self.routed_layers or self.n_layers // 2

    @property
    def first_routed(self):
        return self.n_layers - self.n_routed

    @property
    def proj_dim(self):
        if self.proj_ffn:
            return self.proj_ffn
        return max(64, (self.ffn // 16 + 63) // 64 * 64)

    @property
    def q_dim(self):
        return self.n_q_heads * self.head_dim

    @property
    def kv_dim(self):
        return self.n_kv_heads * self.head_dim

    @property
    def kv_bytes_per_token_layer(self):
        """K and V of one token at one layer, 16-bit elements."""
        return 2 * self.kv_dim * 2

    def matrix_shapes(self):
        """Logical [out][in] shapes of the per-layer matrices."""
        H, F = self.hidden, self.ffn
        return {
            "wq": (self.q_dim, H), "wk": (self.kv_dim, H), "wv": (self.kv_dim, H),
            "wo": (H, self.q_dim), "w_gate": (F, H), "w_up": (F, H), "w_down": (H, F),
        }

    def layer_weight_bytes(self):
        return sum(o * i for o, i in self.matrix_shapes().values()) * 2

    def weight_bytes_streamed(self):
        """Bytes of every matrix read once by one step (embedding rows excluded)."""
        return self.n_layers * self.layer_weight_bytes() + self.vocab * self.hidden * 2


TINY = ModelCfg("tiny-1L", 1, 256, 4, 4, 64, 1024, 1024)
M3B = ModelCfg("3B-class-GQA", 28, 3072, 24, 8, 128, 8192, 128256)
M8B = ModelCfg("8B-class-GQA", 32, 4096, 32, 8, 128, 14336, 128256)


@dataclass
class SeqSpec:
    """One sequence of a pass.

    ctx      : tokens already cached before the pass
    q_len    : new rows of this sequence in the pass (1 for decode)
    blocks   : physical block ids given up front (may be shorter than needed;
               missing blocks are taken from the pool's free list)
    content  : list of (first_pos, n_pos, content_id): which generator stream
               fills the cached positions (shared prefixes reuse one id)
    shared_prefix_of : index of the sequence whose first blocks this one
               shares, with the number of shared tokens (block aligned)
    """
    ctx: int
    q_len: int
    blocks: list
    content: list
    logits: bool = True
    shared_prefix: tuple | None = None


@dataclass
class Workload:
    cfg_id: int
    name: str
    model: ModelCfg
    seqs: list
    n_pool_blocks: int
    tokens: np.ndarray            # int32 [rows]
    seed: int
    description: str = ""
    extra: dict = field(default_factory=dict)

    @property
    def n_rows(self):
        return sum(s.q_len for s in self.seqs)

    @property
    def n_seqs(self):
        return len(self.seqs)

    def logit_rows(self):
        """Row indices whose logits the pass returns (last row of each marked seq)."""
        out, r = [], 0
        for s in self.seqs:
            r += s.q_len
            if s.logits:
                out.append(r - 1)
        return np.asarray(out, np.int32)

    def resident_tokens(self):
        """Logical resident tokens after the pass (sum of per-sequence kv lengths)."""
        return sum(s.ctx + s.q_len for s in self.seqs)

    def unique_resident_tokens(self):
        """Resident tokens counting a shared prefix once."""
        tot = 0
        for s in self.seqs:
            tot += s.ctx + s.q_len
            if s.shared_prefix is not None:
                tot -= s.shared_prefix[1]
        return tot


def _rng(seed, cfg_id, stream):
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, cfg_id, stream])))


def _nblk(n_tokens):
    return (n_tokens + BLOCK - 1) // BLOCK


def kv_content_key(seed, model: ModelCfg, content_id, layer, kind):
    """Generator key of the cached K (kind 0) or V (kind 1) values of one content stream.

    Element index inside the stream: (pos * n_kv_heads + head) * head_dim + dim.
    """
    return gen.key_of(seed, "kv", model.name, content_id, layer, kind)


def weight_key(seed, model: ModelCfg, name, layer=-1):
    return gen.key_of(seed, "w", model.name, name, layer)


def _decode_workload(cfg_id, name, model, ctx, seed, desc, shared=None, pool_factor=1.25):
    """Decode batch with randomly permuted block tables (one new row per sequence)."""
    B = len(ctx)
    need = []
    for c in ctx:
        need.append(_nblk(c + 1))
    shared_blocks = 0
    if shared is not None:
        shared_blocks = shared // BLOCK
        need = [n - shared_blocks for n in need]
    total = shared_blocks + sum(need)
    n_pool = int(math.ceil(1.25 * total)) if pool_factor else total
    perm = _rng(seed, cfg_id, 1).permutation(n_pool).astype(np.int32)
    pos = 0
    prefix_ids = list(perm[:shared_blocks])
    pos = shared_blocks
    seqs = []
    for i, c in enumerate(ctx):
        own = list(perm[pos:pos + need[i]])
        pos += need[i]
        if shared is not None:
            content = [(0, shared, -1), (shared, c - shared, i)]
            seqs.append(SeqSpec(int(c), 1, [int(b) for b in prefix_ids + own], content,
                                shared_prefix=(0, shared) if i > 0 else None))
        else:
            seqs.append(SeqSpec(int(c), 1, [int(b) for b in own], [(0, int(c), i)]))
    tokens = _rng(seed, cfg_id, 2).integers(0, model.vocab, size=B).astype(np.int32)
    return Workload(cfg_id, name, model, seqs, n_pool, tokens, seed, desc)


def workload(cfg_id: int, seed: int = 0, model: ModelCfg | None = None, batch: int | None = None) -> Workload:
    """Build workload 1..5.  ``model``/``batch`` override shapes for scaled-down test runs."""
    if cfg_id == 1:
        m = model or TINY
        B = batch or 4
        ctx = _rng(seed, 1, 0).integers(32, 128, endpoint=True, size=B)
        return _decode_workload(1, "tiny-decode-b4", m, ctx, seed,
                                "1 layer H256 4x64 heads, batch 4, ctx U[32,128]")
    if cfg_id == 2:
        m = model or M3B
        B = batch or 16
        ctx = _rng(seed, 2, 0).integers(512, 1024, endpoint=True, size=B)
        return _decode_workload(2, "3B-decode-b16", m, ctx, seed,
                                "3B-class GQA, batch 16, ctx U[512,1024]")
    if cfg_id == 3:
        m = model or M3B
        B = batch or 64
        prefix = 1536
        suf = _rng(seed, 3, 0).integers(50, 150, endpoint=True, size=B)
        ctx = prefix + suf
        return _decode_workload(3, "3B-shared-prefix-b64", m, ctx, seed,
                                "3B-class GQA, batch 64, 1536-token shared prefix + U[50,150]",
                                shared=prefix)
    if cfg_id == 4:
        m = model or M3B
        n_dec = batch or 32
        ctx = _rng(seed, 4, 0).integers(256, 2048, endpoint=True, size=n_dec)
        return mixed_workload(m, 4, 512, ctx, seed, cfg_id=4, name="3B-mixed-prefill4x512-decode32",
                              desc="3B-class GQA, chunked prefill 4x512 + 32 decodes ctx U[256,2048]")
    if cfg_id == 5:
        m = model or M8B
        B = batch or 128
        z = _rng(seed, 5, 0).standard_normal(B)
        ctx = np.clip(np.rint(np.exp(math.log(600.0) + 0.8 * z)), 16, 4096).astype(np.int64)
        return _decode_workload(5, "8B-decode-b128", m, ctx, seed,
                                "8B-class GQA, batch 128, ctx lognormal(600, 0.8) in [16,4096]")
    raise ValueError(cfg_id)


def decode_workload(model: ModelCfg, ctx, seed=0, cfg_id=0, shared=None, name="decode", desc=""):
    """A decode batch (one new row per sequence) with the given cached lengths."""
    return _decode_workload(cfg_id, name, model, np.asarray(ctx, np.int64), seed, desc, shared=shared)


def prefix_groups_workload(model: ModelCfg, groups, suffixes, seed=0, cfg_id=0, name="prefix-groups", desc=""):
    """A decode batch of several shared-prefix groups.

    groups   : list of (prefix_tokens, n_members); prefix_tokens a multiple of 16
    suffixes : private cached tokens of every sequence, group members first
               (group by group), then sequences of no group
    Block tables are a seeded permutation of the pool; each group's prefix
    blocks are held once and listed first in every member's table.
    """
    suffixes = np.asarray(suffixes, np.int64)
    members = sum(n for _, n in groups)
    assert len(suffixes) >= members and all(p % BLOCK == 0 for p, _ in groups)
    prefix_of = []
    for gi, (p, n) in enumerate(groups):
        prefix_of += [(gi, p)] * n
    prefix_of += [(None, 0)] * (len(suffixes) - members)
    need_shared = sum(p // BLOCK for p, _ in groups)
    need = [_nblk(pr + c + 1) - pr // BLOCK for (_, pr), c in zip(prefix_of, suffixes)]
    n_pool = int(math.ceil(1.25 * (need_shared + sum(need))))
    perm = [int(b) for b in _rng(seed, cfg_id, 1).permutation(n_pool)]
    pos = 0
    shared_ids = []
    for p, _ in groups:
        shared_ids.append(perm[pos:pos + p // BLOCK])
        pos += p // BLOCK
    seqs = []
    first_of_group = {}
    for i, ((gi, pr), c) in enumerate(zip(prefix_of, suffixes)):
        own = perm[pos:pos + need[i]]
        pos += need[i]
        ctx = int(pr + c)
        if gi is None:
            seqs.append(SeqSpec(ctx, 1, own, [(0, ctx, i)]))
            continue
        content = [(0, pr, -1 - gi), (pr, int(c), i)]
        shared = (first_of_group[gi], pr) if gi in first_of_group else None
        first_of_group.setdefault(gi, i)
        seqs.append(SeqSpec(ctx, 1, shared_ids[gi] + own, content, shared_prefix=shared))
    tokens = _rng(seed, cfg_id, 2).integers(0, model.vocab, size=len(seqs)).astype(np.int32)
    return Workload(cfg_id, name, model, seqs, n_pool, tokens, seed, desc)


def mixed_workload(model: ModelCfg, n_pre, plen, ctx, seed=0, cfg_id=0, name="mixed", desc=""):
    """Fresh requests prefilled in one chunk (plen rows each, blocks from the free
    list, lowest id first) beside decoding sequences holding permuted blocks."""
    ctx = np.asarray(ctx, np.int64)
    n_dec = len(ctx)
    need_dec = [_nblk(c + 1) for c in ctx]
    total = sum(need_dec) + n_pre * _nblk(plen)
    n_pool = int(math.ceil(1.25 * total))
    perm = _rng(seed, cfg_id, 1).permutation(n_pool).astype(np.int32)
    pos = 0
    dec = []
    for i, c in enumerate(ctx):
        own = [int(b) for b in perm[pos:pos + need_dec[i]]]
        pos += need_dec[i]
        dec.append(SeqSpec(int(c), 1, own, [(0, int(c), i)]))
    pre = [SeqSpec(0, plen, [], [], logits=True) for _ in range(n_pre)]
    tokens = _rng(seed, cfg_id, 2).integers(0, model.vocab, size=n_pre * plen + n_dec).astype(np.int32)
    return Workload(cfg_id, name, model, pre + dec, n_pool, tokens, seed, desc)
