"""Thin ctypes binding of libvsk.so (include/vsk.h).

Argument marshalling only: every step of a pass runs in the library's HIP
kernels.  Device buffers are passed as raw pointers (e.g. a torch tensor's
``data_ptr()``); streams as ``hipStream_t`` handles (``torch.cuda.current_stream().cuda_stream``).
The library must be built (``python -m paper_2609_37062_amd.build``); a
missing library is an error, never a silent fallback.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libvsk.so")

VSK_OK = 0
SCRATCH_BYTES = 64 * 1024 * 1024  # VSK_SCRATCH_BYTES in vsk.h
STATUS = {0: "OK", -1: "ARG", -2: "NOMEM", -3: "RANGE", -4: "SHARED_WRITE", -5: "STATE", -6: "HIP",
          -7: "UNSUPPORTED"}


class VskError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"{STATUS.get(code, code)}: {msg}")
        self.code = STATUS.get(code, str(code))
        self.status = code


class ModelCfg(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("hidden", C.c_int32), ("n_q_heads", C.c_int32),
                ("n_kv_heads", C.c_int32), ("head_dim", C.c_int32), ("ffn", C.c_int32),
                ("vocab", C.c_int32), ("block_size", C.c_int32), ("max_pos", C.c_int32),
                ("rope_theta", C.c_float), ("rms_eps", C.c_float)]


class SwitchParams(C.Structure):
    _fields_ = [("tau_s", C.c_double), ("tau_layers", C.c_int32), ("bw_bytes_per_s", C.c_double),
                ("skip", C.c_double), ("routed_layers", C.c_int32), ("kv_bytes_per_token_layer", C.c_double),
                ("enter_factor", C.c_double), ("round_tokens", C.c_double)]


class SwitchThresholds(C.Structure):
    _fields_ = [("v_star", C.c_double), ("exit_tokens", C.c_int64), ("enter_tokens", C.c_int64)]


class LayerWeights(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in ("attn_norm", "wq", "wk", "wv", "wo", "mlp_norm",
                                          "w_gate", "w_up", "w_down")]


# (name, restype, argtypes) of every exported entry point, in header order
_VP, _I32, _I64, _SZ = C.c_void_p, C.c_int32, C.c_int64, C.c_size_t
_PI32, _PI64 = C.POINTER(C.c_int32), C.POINTER(C.c_int64)
SIGNATURES = [
    ("vsk_status_str", C.c_char_p, [C.c_int]),
    ("vsk_last_error", C.c_char_p, [_VP]),
    ("vsk_create", C.c_int, [C.POINTER(ModelCfg), C.POINTER(_VP)]),
    ("vsk_destroy", C.c_int, [_VP]),
    ("vsk_packed_weight_bytes", _SZ, [C.POINTER(ModelCfg)]),
    ("vsk_weights_bind", C.c_int, [_VP, _VP, _SZ]),
    ("vsk_weights_pack_layer", C.c_int, [_VP, _I32, C.POINTER(LayerWeights), _VP]),
    ("vsk_weights_pack_head", C.c_int, [_VP, _VP, _VP, _VP, _VP]),
    ("vsk_kv_pool_bytes", _SZ, [C.POINTER(ModelCfg), _I32]),
    ("vsk_kv_init", C.c_int, [_VP, _VP, _I32]),
    ("vsk_seq_create", C.c_int, [_VP, _I64]),
    ("vsk_seq_release", C.c_int, [_VP, _I64]),
    ("vsk_seq_set_blocks", C.c_int, [_VP, _I64, _PI32, _I32, _I32]),
    ("vsk_seq_share_prefix", C.c_int, [_VP, _I64, _I64, _I32]),
    ("vsk_kv_reserve", C.c_int, [_VP, _I64, _I32, _PI32]),
    ("vsk_seq_info", C.c_int, [_VP, _I64, _PI32, _PI32, _PI32, _I32]),
    ("vsk_kv_free_blocks", C.c_int, [_VP, _PI32]),
    ("vsk_kv_write", C.c_int, [_VP, _I32, _VP, _I32, _VP, _VP, _VP]),
    ("vsk_kv_read", C.c_int, [_VP, _I32, _VP, _I32, _VP, _VP, _VP]),
    ("vsk_batch_build", C.c_int, [_VP, _PI64, _PI32, _I32]),
    ("vsk_batch_shape", C.c_int, [_VP, _PI32, _PI32, _PI32]),
    ("vsk_batch_host_copy", C.c_int, [_VP, _PI32, _PI32, _PI32, _PI32, _PI32, _PI32]),
    ("vsk_batch_prefix_info", C.c_int, [_VP, _PI32, _PI32]),
    ("vsk_batch_device_bytes", _SZ, [_VP]),
    ("vsk_batch_upload", C.c_int, [_VP, _VP, _SZ, _VP]),
    ("vsk_workspace_bytes", _SZ, [_VP, _I32, _I32, _I32]),
    ("vsk_workspace_init", C.c_int, [_VP, _VP, _SZ, _I32, _I32, _I32, _VP]),
    ("vsk_decode_step", C.c_int, [_VP, _VP, _VP, _VP, _VP, _SZ, _VP]),
    ("vsk_decode_step_scratch", C.c_int, [_VP, _VP, _VP, _VP, _VP]),
    ("vsk_prefill_chunk", C.c_int, [_VP, _VP, _VP, _I32, _VP, _VP, _VP, _SZ, _VP]),
    ("vsk_argmax_sample", C.c_int, [_VP, _I32, _I32, _I32, _VP, _VP, _VP]),
    ("vsk_set_tuning", C.c_int, [_VP, _I32, _I32]),
    ("vsk_residual_copy", C.c_int, [_VP, _VP, _I32, _VP]),
    ("vsk_routed_weight_bytes", _SZ, [C.POINTER(ModelCfg), _I32, _I32]),
    ("vsk_routed_bind", C.c_int, [_VP, _I32, _I32, _VP, _SZ]),
    ("vsk_routed_pack_layer", C.c_int, [_VP, _I32, _VP, _VP, _VP, _VP]),
    ("vsk_decode_step_routed", C.c_int, [_VP, _VP, _VP, _VP, _VP, _VP, _VP, _SZ, _VP]),
    ("vsk_prefill_chunk_routed", C.c_int, [_VP, _VP, _VP, _VP, _VP, _I32, _VP, _VP, _VP, _SZ, _VP]),
    ("vsk_route_maps_read", C.c_int, [_VP, _VP, _VP, _VP, _VP, _VP]),
    ("vsk_switch_thresholds", C.c_int, [C.POINTER(SwitchParams), C.POINTER(SwitchThresholds)]),
    ("vsk_switch_step", C.c_int, [C.POINTER(SwitchThresholds), _I32, _I64, _PI32, _PI32]),
    ("vsk_switch_decode_mode", C.c_int, [_I32, _I32, _I32, _PI32]),
    ("vsk_switch_prefill", C.c_int, [_I64, C.c_double, _I64, C.c_double, _PI32]),
    ("vsk_stream_read", C.c_int, [_VP, _SZ, _VP, _I32, _VP]),
    ("vsk_set_probe", C.c_int, [_VP, _I32, C.POINTER(_VP), C.POINTER(_VP), _I32]),
    ("vsk_exec_counters", C.c_int, [_VP, _PI64, _I32]),
    ("vsk_set_step_trace", C.c_int, [_VP, _VP, _SZ, _PI32, _PI32]),
    ("vsk_device_status", C.c_int, [_VP, _VP]),
]

_lib = None


def lib():
    """Load libvsk.so once; raises if it is missing (no fallback path exists)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is not built; run python -m paper_2609_37062_amd.build")
        L = C.CDLL(LIB_PATH)
        for name, res, args in SIGNATURES:
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def _p32(a):
    return a.ctypes.data_as(_PI32) if a is not None else None


def _p64(a):
    return a.ctypes.data_as(_PI64) if a is not None else None


def model_cfg(m) -> ModelCfg:
    """ModelCfg from any object with the model-shape attributes."""
    return ModelCfg(m.n_layers, m.hidden, m.n_q_heads, m.n_kv_heads, m.head_dim, m.ffn, m.vocab, 16,
                    m.max_pos, m.rope_theta, m.rms_eps)


def packed_weight_bytes(m) -> int:
    c = model_cfg(m)
    return lib().vsk_packed_weight_bytes(C.byref(c))


def kv_pool_bytes(m, n_blocks) -> int:
    c = model_cfg(m)
    return lib().vsk_kv_pool_bytes(C.byref(c), n_blocks)


def argmax_sample(logits_ptr, dtype, rows, vocab, ids_ptr, stream=None, no_value_ptr=None):
    st = lib().vsk_argmax_sample(logits_ptr, dtype, rows, vocab, ids_ptr, no_value_ptr, stream)
    if st != VSK_OK:
        raise VskError(st, "argmax_sample")


def stream_read(src_ptr, nbytes, out_ptr, workgroups, stream=None):
    st = lib().vsk_stream_read(src_ptr, nbytes, out_ptr, workgroups, stream)
    if st != VSK_OK:
        raise VskError(st, "stream_read")


# ------------------------------------------------------------------ mode switch
def switch_thresholds(tau_s, bw_bytes_per_s, skip, routed_layers, kv_bytes_per_token_layer, tau_layers=16,
                      enter_factor=1.25, round_tokens=10000.0):
    """(V*, exit tokens, enter tokens) of the decode rule (vsk_switch_thresholds)."""
    p = SwitchParams(tau_s, tau_layers, bw_bytes_per_s, skip, routed_layers, kv_bytes_per_token_layer,
                     enter_factor, round_tokens)
    t = SwitchThresholds()
    st = lib().vsk_switch_thresholds(C.byref(p), C.byref(t))
    if st != VSK_OK:
        raise VskError(st, "switch_thresholds")
    return t.v_star, t.exit_tokens, t.enter_tokens


def switch_step(exit_tokens, enter_tokens, routing, resident_tokens):
    """One hysteresis observation: returns (routing state, promote)."""
    t = SwitchThresholds(0.0, exit_tokens, enter_tokens)
    r, pr = C.c_int32(), C.c_int32()
    st = lib().vsk_switch_step(C.byref(t), routing, resident_tokens, C.byref(r), C.byref(pr))
    if st != VSK_OK:
        raise VskError(st, "switch_step")
    return r.value, pr.value


def switch_decode_mode(mode_in, routing, promote):
    out = C.c_int32()
    st = lib().vsk_switch_decode_mode(mode_in, routing, promote, C.byref(out))
    if st != VSK_OK:
        raise VskError(st, "switch_decode_mode")
    return out.value


def switch_prefill(prompt_tokens, po_share, floor_tokens=1536, share_min=0.35):
    out = C.c_int32()
    st = lib().vsk_switch_prefill(prompt_tokens, po_share, floor_tokens, share_min, C.byref(out))
    if st != VSK_OK:
        raise VskError(st, "switch_prefill")
    return out.value


class Engine:
    """One handle: model shape, packed weights, KV pool + allocator, batch, workspace."""

    def __init__(self, m):
        self.m = m
        self.cfg = model_cfg(m)
        h = C.c_void_p()
        st = lib().vsk_create(C.byref(self.cfg), C.byref(h))
        if st != VSK_OK:
            raise VskError(st, "vsk_create rejected the model shape")
        self.h = h

    def close(self):
        if self.h:
            lib().vsk_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def _ck(self, st, what=""):
        if st != VSK_OK:
            msg = lib().vsk_last_error(self.h)
            raise VskError(st, f"{what}: {msg.decode() if msg else ''}")

    # -- weights
    def packed_weight_bytes(self):
        return lib().vsk_packed_weight_bytes(C.byref(self.cfg))

    def weights_bind(self, ptr, nbytes):
        self._ck(lib().vsk_weights_bind(self.h, ptr, nbytes), "weights_bind")

    def weights_pack_layer(self, layer, ptrs: dict, stream=None):
        w = LayerWeights(**{k: ptrs[k] for k in ("attn_norm", "wq", "wk", "wv", "wo", "mlp_norm",
                                                  "w_gate", "w_up", "w_down")})
        self._ck(lib().vsk_weights_pack_layer(self.h, layer, C.byref(w), stream), "pack_layer")

    def weights_pack_head(self, embed, lm_head, final_norm, stream=None):
        self._ck(lib().vsk_weights_pack_head(self.h, embed, lm_head, final_norm, stream), "pack_head")

    # -- kv
    def kv_pool_bytes(self, n_blocks):
        return lib().vsk_kv_pool_bytes(C.byref(self.cfg), n_blocks)

    def kv_init(self, pool_ptr, n_blocks):
        self._ck(lib().vsk_kv_init(self.h, pool_ptr, n_blocks), "kv_init")

    def seq_create(self, seq):
        self._ck(lib().vsk_seq_create(self.h, seq), "seq_create")

    def seq_release(self, seq):
        self._ck(lib().vsk_seq_release(self.h, seq), "seq_release")

    def seq_set_blocks(self, seq, blocks, ctx_len):
        b = np.ascontiguousarray(blocks, np.int32)
        self._ck(lib().vsk_seq_set_blocks(self.h, seq, _p32(b), len(b), ctx_len), "seq_set_blocks")

    def seq_share_prefix(self, dst, src, n_tokens):
        self._ck(lib().vsk_seq_share_prefix(self.h, dst, src, n_tokens), "seq_share_prefix")

    def reserve(self, seq, n_new):
        out = np.zeros(max(n_new, 1), np.int32)
        self._ck(lib().vsk_kv_reserve(self.h, seq, n_new, _p32(out)), "kv_reserve")
        return out[:n_new].astype(np.int64)

    def seq_info(self, seq):
        ln, nb = C.c_int32(), C.c_int32()
        self._ck(lib().vsk_seq_info(self.h, seq, C.byref(ln), C.byref(nb), None, 0), "seq_info")
        blocks = np.zeros(max(nb.value, 1), np.int32)
        self._ck(lib().vsk_seq_info(self.h, seq, C.byref(ln), C.byref(nb), _p32(blocks), nb.value), "seq_info")
        return ln.value, blocks[:nb.value].tolist()

    def free_blocks(self):
        n = C.c_int32()
        self._ck(lib().vsk_kv_free_blocks(self.h, C.byref(n)), "free_blocks")
        return n.value

    def kv_write(self, layer, slots_ptr, n, k_ptr, v_ptr, stream=None):
        self._ck(lib().vsk_kv_write(self.h, layer, slots_ptr, n, k_ptr, v_ptr, stream), "kv_write")

    def kv_read(self, layer, slots_ptr, n, k_ptr, v_ptr, stream=None):
        self._ck(lib().vsk_kv_read(self.h, layer, slots_ptr, n, k_ptr, v_ptr, stream), "kv_read")

    # -- batch
    def batch_build(self, seqs, q_lens):
        s = np.ascontiguousarray(seqs, np.int64)
        q = np.ascontiguousarray(q_lens, np.int32)
        self._ck(lib().vsk_batch_build(self.h, _p64(s), _p32(q), len(s)), "batch_build")

    def batch_host(self):
        n, r, mb = C.c_int32(), C.c_int32(), C.c_int32()
        self._ck(lib().vsk_batch_shape(self.h, C.byref(n), C.byref(r), C.byref(mb)), "batch_shape")
        n, r, mb = n.value, r.value, mb.value
        out = {"block_table": np.zeros((n, mb), np.int32), "kv_len": np.zeros(n, np.int32),
               "cu_q": np.zeros(n + 1, np.int32), "row_seq": np.zeros(r, np.int32),
               "pos": np.zeros(r, np.int32), "slot": np.zeros(r, np.int32)}
        self._ck(lib().vsk_batch_host_copy(self.h, *[_p32(out[k]) for k in
                                                     ("block_table", "kv_len", "cu_q", "row_seq", "pos", "slot")]),
                 "batch_host_copy")
        return out

    def batch_prefix_info(self):
        """Per row the shared-prefix blocks of its group (0: none), and the group count."""
        n, r, mb = C.c_int32(), C.c_int32(), C.c_int32()
        self._ck(lib().vsk_batch_shape(self.h, C.byref(n), C.byref(r), C.byref(mb)), "batch_shape")
        out = np.zeros(r.value, np.int32)
        ng = C.c_int32()
        self._ck(lib().vsk_batch_prefix_info(self.h, _p32(out), C.byref(ng)), "batch_prefix_info")
        return out, ng.value

    def batch_device_bytes(self):
        return lib().vsk_batch_device_bytes(self.h)

    def batch_upload(self, ptr, nbytes, stream=None):
        self._ck(lib().vsk_batch_upload(self.h, ptr, nbytes, stream), "batch_upload")

    # -- passes
    def workspace_bytes(self, max_rows, max_seqs, max_kv_len):
        return lib().vsk_workspace_bytes(self.h, max_rows, max_seqs, max_kv_len)

    def workspace_init(self, ptr, nbytes, max_rows, max_seqs, max_kv_len, stream=None):
        self._ck(lib().vsk_workspace_init(self.h, ptr, nbytes, max_rows, max_seqs, max_kv_len, stream),
                 "workspace_init")

    def decode_step(self, ids_ptr, logits_ptr, next_ids_ptr, ws_ptr, ws_bytes, stream=None):
        self._ck(lib().vsk_decode_step(self.h, ids_ptr, logits_ptr, next_ids_ptr, ws_ptr, ws_bytes, stream),
                 "decode_step")

    def decode_step_scratch(self, ids_ptr, logits_ptr, next_ids_ptr, stream=None):
        self._ck(lib().vsk_decode_step_scratch(self.h, ids_ptr, logits_ptr, next_ids_ptr, stream),
                 "decode_step_scratch")

    def prefill_chunk(self, ids_ptr, logit_rows_ptr, n_logit_rows, logits_ptr, next_ids_ptr, ws_ptr, ws_bytes,
                      stream=None):
        self._ck(lib().vsk_prefill_chunk(self.h, ids_ptr, logit_rows_ptr, n_logit_rows, logits_ptr, next_ids_ptr,
                                         ws_ptr, ws_bytes, stream), "prefill_chunk")

    # -- routed mode
    def routed_weight_bytes(self, first_routed, proj_ffn):
        return lib().vsk_routed_weight_bytes(C.byref(self.cfg), first_routed, proj_ffn)

    def routed_bind(self, first_routed, proj_ffn, ptr, nbytes):
        self._ck(lib().vsk_routed_bind(self.h, first_routed, proj_ffn, ptr, nbytes), "routed_bind")

    def routed_pack_layer(self, layer, p_gate, p_up, p_down, stream=None):
        self._ck(lib().vsk_routed_pack_layer(self.h, layer, p_gate, p_up, p_down, stream), "routed_pack_layer")

    def decode_step_routed(self, ids_ptr, run_ptr, w_ptr, logits_ptr, next_ids_ptr, ws_ptr, ws_bytes, stream=None):
        self._ck(lib().vsk_decode_step_routed(self.h, ids_ptr, run_ptr, w_ptr, logits_ptr, next_ids_ptr, ws_ptr,
                                              ws_bytes, stream), "decode_step_routed")

    def prefill_chunk_routed(self, ids_ptr, run_ptr, w_ptr, logit_rows_ptr, n_logit_rows, logits_ptr, next_ids_ptr,
                             ws_ptr, ws_bytes, stream=None):
        self._ck(lib().vsk_prefill_chunk_routed(self.h, ids_ptr, run_ptr, w_ptr, logit_rows_ptr, n_logit_rows,
                                                logits_ptr, next_ids_ptr, ws_ptr, ws_bytes, stream),
                 "prefill_chunk_routed")

    def route_maps_read(self, run_ptr, proj_ptr, inv_ptr, cnt_ptr, stream=None):
        self._ck(lib().vsk_route_maps_read(self.h, run_ptr, proj_ptr, inv_ptr, cnt_ptr, stream), "route_maps_read")

    def set_tuning(self, key, value):
        self._ck(lib().vsk_set_tuning(self.h, key, value), "set_tuning")

    def residual_copy(self, dst_ptr, n_rows, stream=None):
        self._ck(lib().vsk_residual_copy(self.h, dst_ptr, n_rows, stream), "residual_copy")

    def set_probe(self, which, begin_events, end_events):
        n = len(begin_events)
        B = (C.c_void_p * max(n, 1))(*begin_events)
        E = (C.c_void_p * max(n, 1))(*end_events)
        self._ck(lib().vsk_set_probe(self.h, which, B, E, n), "set_probe")

    def set_step_trace(self, ptr, nbytes):
        """Point the persistent kernel's timestamp trace at a device buffer (0 clears it).
        Returns (workgroups per launch, synchronisation points per pass)."""
        n, p = C.c_int32(), C.c_int32()
        self._ck(lib().vsk_set_step_trace(self.h, ptr or None, nbytes, C.byref(n), C.byref(p)), "set_step_trace")
        return n.value, p.value

    def device_status(self, stream=None):
        """Synchronise the stream and raise if a persistent pass timed out at a grid sync."""
        self._ck(lib().vsk_device_status(self.h, stream), "device_status")

    def exec_counters(self):
        out = np.zeros(8, np.int64)
        self._ck(lib().vsk_exec_counters(self.h, _p64(out), 8), "exec_counters")
        return out
