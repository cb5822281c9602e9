"""Set up and run a synthetic workload on the device through the C ABI.

Weights and cached KV are drawn on the device from the seeded generators in
``workloads`` (the same values the CPU side can redraw), packed and written
through the library, then passes run on one stream.  torch is used for
device memory and streams only.
"""
from __future__ import annotations

import numpy as np
import torch

from workloads import gen
from workloads.configs import Workload, weight_key
from workloads.setup import apply_recipe, kv_fill_ranges, kv_values_torch

from . import vsk

LAYER_MATS = ("wq", "wk", "wv", "wo", "w_gate", "w_up", "w_down")


def _align(n, a=256):
    return (n + a - 1) // a * a


def _dev_buffer(nbytes, device):
    """Byte buffer whose data pointer is 256-byte aligned."""
    t = torch.empty(nbytes + 256, dtype=torch.uint8, device=device)
    off = (-t.data_ptr()) % 256
    return t, t.data_ptr() + off


class DeviceRun:
    """One workload resident on the device: engine, packed weights, KV pool, batch, workspace."""

    def __init__(self, w: Workload, device="cuda", overrides=None, weight_dist=None, max_rows=None,
                 max_kv_len=None, pool_blocks=None, poison_pool=False, routed=False, fill_kv=True):
        assert torch.cuda.is_available(), "a GPU is required"
        self.w = w
        self.m = w.model
        self.device = torch.device(device)
        self.stream = torch.cuda.current_stream(self.device)
        self.sp = self.stream.cuda_stream
        self.eng = vsk.Engine(self.m)
        self.overrides = dict(overrides or {})
        self.dist = weight_dist or ("normal", self.m.weight_sigma)
        self._load_weights()
        self.routed = routed
        if routed:
            self._load_projectors()
        self.n_blocks = pool_blocks or w.n_pool_blocks
        self.pool = torch.empty(self.eng.kv_pool_bytes(self.n_blocks) // 2, dtype=torch.int16, device=self.device)
        if poison_pool:
            self.pool.fill_(-1)  # every unwritten slot holds a bf16 NaN pattern
        elif not fill_kv:
            self.pool.zero_()  # timing runs that skip drawing the cached KV
        self.eng.kv_init(self.pool.data_ptr(), self.n_blocks)
        self.slots = apply_recipe(self.eng, w)
        if fill_kv:
            self._fill_kv()
        seqs = list(range(w.n_seqs))
        self.q_lens = [s.q_len for s in w.seqs]
        self.eng.batch_build(seqs, self.q_lens)
        self.meta_bytes = self.eng.batch_device_bytes()
        self._meta_t, self.meta = _dev_buffer(self.meta_bytes, self.device)
        self.eng.batch_upload(self.meta, self.meta_bytes, self.sp)
        R = w.n_rows
        kvmax = max(s.ctx + s.q_len for s in w.seqs)
        self.cap = (max_rows or R, w.n_seqs, max_kv_len or kvmax)
        self.ws_bytes = self.eng.workspace_bytes(*self.cap)
        self._ws_t, self.ws = _dev_buffer(self.ws_bytes, self.device)
        self.eng.workspace_init(self.ws, self.ws_bytes, *self.cap, self.sp)
        self.ids = torch.from_numpy(np.ascontiguousarray(w.tokens, np.int32)).to(self.device)
        self._ids_all = self.ids
        lr = w.logit_rows()
        self.logit_rows = torch.from_numpy(lr).to(self.device)
        self.n_out = len(lr) if any(s.q_len > 1 for s in w.seqs) else R
        self.logits = torch.empty((self.n_out, self.m.vocab), dtype=torch.int16, device=self.device)
        self.next_ids = torch.empty(self.n_out, dtype=torch.int32, device=self.device)
        torch.cuda.synchronize(self.device)

    # ---------------------------------------------------------- setup
    def _tensor(self, name, layer, shape):
        k = (name, layer)
        if k in self.overrides:
            v = np.asarray(self.overrides[k], np.float32)
            return torch.from_numpy(v).to(torch.bfloat16).to(self.device).view(torch.int16)
        if name in ("attn_norm", "mlp_norm", "final_norm"):
            return torch.ones(shape, dtype=torch.bfloat16, device=self.device).view(torch.int16)
        key = weight_key(self.w.seed, self.m, name, layer)
        return gen.bf16_tensor(key, shape, self.dist, device=self.device).view(torch.int16)

    def _load_weights(self):
        m = self.m
        shapes = m.matrix_shapes()
        self.packed_bytes = self.eng.packed_weight_bytes()
        self._packed_t, self.packed = _dev_buffer(self.packed_bytes, self.device)
        self.eng.weights_bind(self.packed, self.packed_bytes)
        for l in range(m.n_layers):
            t = {n: self._tensor(n, l, shapes[n]) for n in LAYER_MATS}
            t["attn_norm"] = self._tensor("attn_norm", l, (m.hidden,))
            t["mlp_norm"] = self._tensor("mlp_norm", l, (m.hidden,))
            self.eng.weights_pack_layer(l, {k: v.data_ptr() for k, v in t.items()}, self.sp)
            torch.cuda.synchronize(self.device)
            del t
        E = self._tensor("embed", -1, (m.vocab, m.hidden))
        Wl = self._tensor("lm_head", -1, (m.vocab, m.hidden))
        g = self._tensor("final_norm", -1, (m.hidden,))
        self.eng.weights_pack_head(E.data_ptr(), Wl.data_ptr(), g.data_ptr(), self.sp)
        torch.cuda.synchronize(self.device)

    def _load_projectors(self):
        """Routed mode: pack every routed layer's projector (p_gate, p_up, p_down)."""
        m = self.m
        Fp, H = m.proj_dim, m.hidden
        nbytes = self.eng.routed_weight_bytes(m.first_routed, Fp)
        self._proj_t, self.proj = _dev_buffer(nbytes, self.device)
        self.eng.routed_bind(m.first_routed, Fp, self.proj, nbytes)
        for l in range(m.first_routed, m.n_layers):
            t = {n: self._tensor(n, l, shp) for n, shp in (("p_gate", (Fp, H)), ("p_up", (Fp, H)),
                                                             ("p_down", (H, Fp)))}
            self.eng.routed_pack_layer(l, t["p_gate"].data_ptr(), t["p_up"].data_ptr(), t["p_down"].data_ptr(),
                                       self.sp)
            torch.cuda.synchronize(self.device)
            del t

    def set_route(self, run, w):
        """Device copy of a route tape: run bool [n_routed][rows], w float [n_routed][rows]."""
        self.tape_run = torch.from_numpy(np.ascontiguousarray(run, np.uint8)).to(self.device)
        self.tape_w = torch.from_numpy(np.ascontiguousarray(w, np.float32)).to(self.device)

    def step_routed(self, stream=None):
        """One routed pass with the tape set by set_route."""
        sp = self.sp if stream is None else stream
        if all(q == 1 for q in self.q_lens):
            self.eng.decode_step_routed(self.ids.data_ptr(), self.tape_run.data_ptr(), self.tape_w.data_ptr(),
                                        self.logits.data_ptr(), self.next_ids.data_ptr(), self.ws, self.ws_bytes, sp)
        else:
            self.eng.prefill_chunk_routed(self.ids.data_ptr(), self.tape_run.data_ptr(), self.tape_w.data_ptr(),
                                          self.logit_rows.data_ptr(), len(self.logit_rows), self.logits.data_ptr(),
                                          self.next_ids.data_ptr(), self.ws, self.ws_bytes, sp)

    def route_maps(self):
        """(run, proj, inv [n_routed][rows], cnt [n_routed][2]) of the last routed pass."""
        L, R = self.m.n_routed, self.w.n_rows
        bufs = [torch.empty((L, R), dtype=torch.int32, device=self.device) for _ in range(3)]
        cnt = torch.empty((L, 2), dtype=torch.int32, device=self.device)
        self.eng.route_maps_read(*(b.data_ptr() for b in bufs), cnt.data_ptr(), self.sp)
        torch.cuda.synchronize(self.device)
        return tuple(b.cpu().numpy() for b in bufs) + (cnt.cpu().numpy(),)

    def seq_slots(self, i, p0, n):
        ln, table = self.eng.seq_info(i)
        p = np.arange(p0, p0 + n)
        t = np.asarray(table, np.int64)
        return (t[p // 16] * 16 + p % 16).astype(np.int32)

    def _fill_kv(self):
        ranges = kv_fill_ranges(self.w)
        if not ranges:
            return
        slots = np.concatenate([self.seq_slots(i, p0, n) for (i, p0, n, cid) in ranges])
        slots_d = torch.from_numpy(slots).to(self.device)
        n_tot = len(slots)
        for l in range(self.m.n_layers):
            K = torch.cat([kv_values_torch(self.w, l, 0, p0, n, cid, self.device) for (i, p0, n, cid) in ranges])
            V = torch.cat([kv_values_torch(self.w, l, 1, p0, n, cid, self.device) for (i, p0, n, cid) in ranges])
            self.eng.kv_write(l, slots_d.data_ptr(), n_tot, K.data_ptr(), V.data_ptr(), self.sp)
        torch.cuda.synchronize(self.device)

    def rebatch(self, seqs):
        """Make the first decode rows a new batch of the listed sequences (one row
        each; rows, ids and logits buffers keep their capacity)."""
        self.q_lens = [1] * len(seqs)
        self.eng.batch_build(list(seqs), self.q_lens)
        need = self.eng.batch_device_bytes()
        if need > self.meta_bytes:
            self._meta_t, self.meta = _dev_buffer(need, self.device)
            self.meta_bytes = need
        self.eng.batch_upload(self.meta, self.meta_bytes, self.sp)
        self.ids = self._ids_all[:len(seqs)]

    # ---------------------------------------------------------- passes
    def step(self, stream=None):
        """Enqueue one pass (decode_step when every q_len is 1, else prefill_chunk).

        ``stream``: hipStream_t handle to launch on (default: the setup stream)."""
        sp = self.sp if stream is None else stream
        if all(q == 1 for q in self.q_lens):
            self.eng.decode_step(self.ids.data_ptr(), self.logits.data_ptr(), self.next_ids.data_ptr(), self.ws,
                                 self.ws_bytes, sp)
        else:
            self.eng.prefill_chunk(self.ids.data_ptr(), self.logit_rows.data_ptr(), len(self.logit_rows),
                                   self.logits.data_ptr(), self.next_ids.data_ptr(), self.ws, self.ws_bytes, sp)

    def set_layers(self, n):
        """Inspection: run only the first n layers in the following passes (0 = all)."""
        self.eng.set_tuning(1, n)

    def residual(self):
        """The fp32 residual stream x [rows][hidden] after the last pass (float64 copy)."""
        x = torch.empty((self.w.n_rows, self.m.hidden), dtype=torch.float32, device=self.device)
        self.eng.residual_copy(x.data_ptr(), self.w.n_rows, self.sp)
        torch.cuda.synchronize(self.device)
        return x.cpu().numpy().astype(np.float64)

    def results(self):
        torch.cuda.synchronize(self.device)
        lg = self.logits.view(torch.bfloat16).float().cpu().numpy().astype(np.float64)
        return lg, self.next_ids.cpu().numpy()

    def read_kv(self, layer, slots):
        s = torch.from_numpy(np.ascontiguousarray(slots, np.int32)).to(self.device)
        n = len(slots)
        K = torch.empty((n, self.m.n_kv_heads, self.m.head_dim), dtype=torch.int16, device=self.device)
        V = torch.empty_like(K)
        self.eng.kv_read(layer, s.data_ptr(), n, K.data_ptr(), V.data_ptr(), self.sp)
        torch.cuda.synchronize(self.device)
        f = lambda t: t.view(torch.bfloat16).float().cpu().numpy().astype(np.float64)
        return f(K), f(V)

    def release(self):
        self.eng.close()
