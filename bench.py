"""Benchmark of the batched decode step on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W]
    python bench.py --sweep          (row sweep of dense and routed steps; no JSON contract line)

Workload: the 3B-class GQA decoder (28 layers, hidden 3072, 24/8 heads x 128,
SwiGLU 8192, vocab 128256), batch 16, cached contexts U[512,1024], KV blocks of
16 with randomly permuted tables; one decode step + greedy argmax per step.
Random-init bf16 weights and N(0,1) KV from the seeded generators; inputs are
resident in HBM before timing starts and the step is replayed idempotently.

Prints ONE JSON line.  ``value`` is decode tokens/s (rows per step / step
time over exactly K timed steps, the faster of eager launches and a captured
HIP graph of the step).  Beside it: per-replay statistics (median and IQR of
at least 100 event-timed replays, and a t-based 95% interval over 5 repeats
of the K-step loop); a 16-step decode loop that rebuilds and uploads the
batch metadata on the host every step (allocator reserve, batch build,
upload, step); the same workload in routed mode (half the routed decisions
Project-Only); the batch-64 shared-prefix workload; the device's measured
stream-read ceiling; ``roofline`` for the gate/up projection (the largest
kernel of a layer), timed live with HIP events bound to each of its launches
(hipExtLaunchKernel: the kernel's own start and end on the pass stream); and
``cpu_baseline``, the float64 CPU oracle timed on a bounded sample of the
same workload (median of 3 after a warm-up).

``--workload 4`` times the 2,080-row mixed pass (four 512-row prompts
prefilled beside 32 decoding sequences, logits for 36 rows) instead: the
value is rows/s, and ``roofline`` is the gate/up projection's flops over its
launch time against the dense bf16 matrix-core peak (the pass is bound by the
matrix cores, not HBM); ``step_TFLOPs`` is the whole pass's algorithmic flops
over the step time.
"""
from __future__ import annotations

import argparse
import ctypes as C
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

PEAK_HBM = 8.0e12  # MI355X HBM3E, bytes/s
PEAK_MFMA_BF16 = 2.5e15  # MI355X dense bf16 matrix-core rate, flop/s
CALIB_BYTES = 512 << 20  # plain device-to-device copy used to calibrate byte counters


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=40)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", type=int, default=2,
                    help="workload of the value line: 2, 3 or 5 (decode tokens/s), 4 (mixed prefill + decode "
                         "pass, rows/s, matrix-core roofline)")
    ap.add_argument("--no-batch64", action="store_true", help="skip the batch-64 shared-prefix line")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--cpu-layers", type=int, default=1, help="layers in the CPU oracle sample")
    ap.add_argument("--no-graph", action="store_true")
    ap.add_argument("--mode", type=int, default=0,
                    help="execution path: 0 automatic, 1 one kernel per operation, 2 persistent step kernel")
    ap.add_argument("--tune", action="append", default=[], metavar="KEY=VALUE",
                    help="launch-shape tuning passed to vsk_set_tuning before timing (repeatable)")
    ap.add_argument("--trace", action="store_true",
                    help="print the persistent kernel's per-phase timeline (stderr) after the timed steps")
    ap.add_argument("--no-routed", action="store_true", help="skip the routed-mode line")
    ap.add_argument("--no-loop", action="store_true", help="skip the host-rebuild decode loop")
    ap.add_argument("--replays", type=int, default=100, help="event-timed replays for the per-replay statistics")
    ap.add_argument("--sweep", action="store_true",
                    help="row sweep (8B-class, 1k context) of dense and routed steps, eager and graph")
    ap.add_argument("--sweep-rows", default="16,32,64,128,256,384,512,768,1024")
    ap.add_argument("--profile-pass", action="store_true",
                    help="for rocprofv3 runs: set up the workload, run one plain copy and one plain read of "
                         f"{CALIB_BYTES >> 20} MiB (counter calibration), then --steps passes; no JSON")
    return ap.parse_args()


# ------------------------------------------------------------------ HIP events (same runtime as torch)
class HipEvents:
    def __init__(self):
        self.L = C.CDLL("libamdhip64.so.7")
        self.L.hipEventCreate.argtypes = [C.POINTER(C.c_void_p)]
        self.L.hipEventElapsedTime.argtypes = [C.POINTER(C.c_float), C.c_void_p, C.c_void_p]
        self.L.hipEventSynchronize.argtypes = [C.c_void_p]
        self.L.hipEventDestroy.argtypes = [C.c_void_p]
        self.L.hipEventRecord.argtypes = [C.c_void_p, C.c_void_p]

    def create(self, n):
        out = []
        for _ in range(n):
            e = C.c_void_p()
            assert self.L.hipEventCreate(C.byref(e)) == 0
            out.append(e.value)
        return out

    def elapsed_ms(self, a, b):
        ms = C.c_float()
        assert self.L.hipEventSynchronize(C.c_void_p(b)) == 0
        assert self.L.hipEventElapsedTime(C.byref(ms), C.c_void_p(a), C.c_void_p(b)) == 0
        return ms.value

    def destroy(self, evs):
        for e in evs:
            self.L.hipEventDestroy(C.c_void_p(e))


# ------------------------------------------------------------------ accounting
def step_bytes(w):
    """Algorithmic HBM bytes of one decode step: every matrix once, each unique
    resident (layer, token) KV entry once, new KV and logits written, embedding rows."""
    m = w.model
    B = w.n_rows
    wbytes = m.weight_bytes_streamed()
    kv_read = w.unique_resident_tokens() * m.n_layers * m.kv_bytes_per_token_layer
    kv_write = B * m.n_layers * m.kv_bytes_per_token_layer
    logits = len(w.logit_rows()) * m.vocab * 2
    emb = B * m.hidden * 2
    return wbytes + kv_read + kv_write + logits + emb


def gateup_bytes(m, R):
    """Algorithmic bytes of one gate/up launch: its weights, its input rows, its output."""
    return 2 * m.ffn * m.hidden * 2 + R * m.hidden * 2 + R * m.ffn * 2


def gateup_flops(m, R):
    """Algorithmic flops of one gate/up launch over R rows (padding rows excluded)."""
    return 2 * R * m.hidden * 2 * m.ffn


def step_flops(w):
    """Algorithmic flops of one pass: every projection over every row, the
    lm_head over the logit rows, and attention (QK and PV) over every
    attended key (a prefill row attends its own position and those before)."""
    m = w.model
    Nq, Nkv = m.n_q_heads * m.head_dim, m.n_kv_heads * m.head_dim
    per_row = 2 * m.hidden * (Nq + 2 * Nkv) + 2 * Nq * m.hidden + 2 * m.hidden * 2 * m.ffn + 2 * m.ffn * m.hidden
    keys = sum(sum(s.ctx + j + 1 for j in range(s.q_len)) for s in w.seqs)
    attn = 4 * Nq * keys
    return m.n_layers * (w.n_rows * per_row + attn) + 2 * len(w.logit_rows()) * m.hidden * m.vocab


def gemm_kernel_hash():
    """First 16 hex digits of the SHA-256 of the projection kernel's own source:
    the kernel template of k_gemm.hip (up to its launchers) and the headers it
    uses.  Plan and launcher edits leave it unchanged."""
    import hashlib
    csrc = os.path.join(ROOT, "paper_2609_37062_amd", "csrc")
    k = open(os.path.join(csrc, "k_gemm.hip"), "rb").read()
    i = k.index(b"template <int MG, int NT, int WN, int WK, int PF, int EPI, bool XL>\n__global__")
    j = k.index(b"// ---------------------------------------------------------------- launcher")
    h = hashlib.sha256(k[i:j])
    for f in ("dev.hpp", "gemm.hpp"):
        h.update(open(os.path.join(csrc, f), "rb").read())
    return h.hexdigest()[:16]


def gateup_traffic():
    """Counter-measured HBM bytes per gate/up launch from profiles/, or None when
    the projection kernel's source has changed since the counters were taken."""
    try:
        prof = json.load(open(os.path.join(ROOT, "profiles", "gateup_3b_b16_traffic.json")))
        kh = gemm_kernel_hash()
    except (OSError, ValueError):
        return None
    if kh != prof.get("k_gemm_kernel_sha256_16"):
        return None
    return prof["traffic_bytes_per_launch"]


def time_steps(torch, fn, steps, warmup, stream):
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record(stream)
    for _ in range(steps):
        fn()
    e1.record(stream)
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) * 1e3 / steps
    return e0.elapsed_time(e1) / steps, wall


T975_4 = 2.776  # two-sided 95% quantile of Student's t with 4 degrees of freedom


def replay_stats(torch, fn, stream, n):
    """A HIP event pair around each of n replays of fn on `stream`: median,
    interquartile range and mean of the per-replay times (ms)."""
    ev = HipEvents()
    b, e = ev.create(n), ev.create(n)
    sp = stream.cuda_stream
    for i in range(n):
        ev.L.hipEventRecord(b[i], sp)
        fn()
        ev.L.hipEventRecord(e[i], sp)
    torch.cuda.synchronize()
    d = np.array([ev.elapsed_ms(b[i], e[i]) for i in range(n)])
    ev.destroy(b + e)
    q1, med, q3 = np.percentile(d, [25, 50, 75])
    return {"replays": n, "median_ms": round(float(med), 4), "iqr_ms": [round(float(q1), 4), round(float(q3), 4)],
            "mean_ms": round(float(d.mean()), 4)}


def repeat_ci(torch, fn, steps, stream, reps=5):
    """reps repeats of the timed steps loop: mean and a t-based 95% interval."""
    means = np.array([time_steps(torch, fn, steps, 0, stream)[0] for _ in range(reps)])
    m, sd = float(means.mean()), float(means.std(ddof=1))
    half = T975_4 * sd / np.sqrt(reps)
    return {"repeats": reps, "steps_each": steps, "mean_ms": round(m, 4),
            "ci95_ms": [round(m - half, 4), round(m + half, 4)]}


PHASES = ("norm_attn", "qkv", "attention", "o_proj", "norm_mlp", "gate_up", "down")


def step_timeline(torch, d, reps=3):
    """Per-phase times of the persistent kernel from its timestamp trace:
    for each phase kind, the mean over layers of the span from the first
    workgroup's release at the previous point to the last workgroup's arrival
    (span), the median workgroup's busy time (busy) and the release latency
    after the last arrival (sync).  Microseconds, median of `reps` passes."""
    n_wgs, n_pts = d.eng.set_step_trace(0, 0)
    if n_wgs == 0:
        return None
    buf = torch.zeros(n_pts * n_wgs * 2, dtype=torch.int64, device=d.device)
    d.eng.set_step_trace(buf.data_ptr(), buf.numel() * 8)
    runs = []
    for _ in range(reps):
        d.step()
        torch.cuda.synchronize()
        t = buf.cpu().numpy().reshape(n_pts, n_wgs, 2).astype(np.float64) * 0.01  # 100 MHz -> us
        runs.append(t)
    d.eng.set_step_trace(0, 0)
    P = len(PHASES)
    L = (n_pts - 3) // P
    out = {}
    for name, pts in [("embed", [0])] + [(PHASES[k], [1 + P * l + k for l in range(L)]) for k in range(P)] + \
            [("norm_final", [P * L + 1]), ("lm_head", [P * L + 2])]:
        span, busy, sync = [], [], []
        for t in runs:
            for p in pts:
                if p == 0:
                    continue
                arr, rel = t[p, :, 0], t[p, :, 1]
                prev = t[p - 1, :, 1]
                span.append(arr.max() - prev.min())
                busy.append(np.median(arr - prev))
                sync.append(rel.min() - arr.max())
        if span:
            out[name] = {"span_us": round(float(np.median(span)), 2), "busy_us": round(float(np.median(busy)), 2),
                         "sync_us": round(float(np.median(sync)), 2), "count": len(pts)}
    tot = [t[-1, :, 1].max() - t[0, :, 0].min() for t in runs]
    out["total_us_from_first_point"] = round(float(np.median(tot)), 1)
    return out


def apply_tuning(d, mode, tune):
    d.eng.set_tuning(2, mode)
    for kv in tune:
        k, v = kv.split("=")
        d.eng.set_tuning(int(k), int(v))


def capture(torch, step):
    """A HIP graph of one pass (captured on a side stream after a warm-up there)."""
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        step(stream=s.cuda_stream)  # warm the capture stream
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        step(stream=torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    return g


def settle(torch, fn, seconds=0.4):
    """Run fn (a graph replay) untimed for `seconds` after a capture.  For about
    0.2 s after a HIP graph capture every pass on the device runs ~5% slower,
    eager launches as well as replays (measured at batch 16: 2.26 against
    2.145 ms per pass for ~90 passes, then back; an idle gap or a plain
    allocation of the same duration does not do it), so a replay timed right
    after its capture would carry that transient and not the replay's cost."""
    import time
    t0 = time.time()
    while time.time() - t0 < seconds:
        for _ in range(10):
            fn()
        torch.cuda.synchronize()


def measure(torch, w, steps, warmup, use_graph, probe=True, mode=0, trace=False, tune=(), route=None, stats=0):
    """Time one workload: exactly `steps` steps eager and as graph replays;
    with stats > 0 also per-replay statistics and 5 repeats of the faster."""
    from paper_2609_37062_amd.runner import DeviceRun
    print(f"[bench] setting up {w.name}{' (routed)' if route is not None else ''}", file=sys.stderr, flush=True)
    d = DeviceRun(w, routed=route is not None)
    apply_tuning(d, mode, tune)
    if route is not None:
        d.set_route(*route)
    step = d.step_routed if route is not None else d.step
    stream = torch.cuda.current_stream()
    res = {}
    ms_eager, wall_eager = time_steps(torch, step, steps, warmup, stream)
    res["ms_eager"] = ms_eager
    res["ms_eager_wall"] = wall_eager
    print(f"[bench] {w.name}: eager {ms_eager:.3f} ms/step", file=sys.stderr, flush=True)
    best = step
    g = None
    if use_graph:
        g = capture(torch, step)
        settle(torch, g.replay)
        ms_graph, wall_graph = time_steps(torch, g.replay, steps, warmup, stream)
        res["ms_graph"] = ms_graph
        print(f"[bench] {w.name}: graph {ms_graph:.3f} ms/step", file=sys.stderr, flush=True)
        # graph replays must reproduce the eager result
        lg_g, ids_g = d.results()
        step()
        lg_e, ids_e = d.results()
        res["graph_matches_eager"] = bool(np.array_equal(lg_g, lg_e) and np.array_equal(ids_g, ids_e))
        if ms_graph < ms_eager:
            best = g.replay
    if stats > 0:
        res["per_replay"] = replay_stats(torch, best, stream, stats)
        res["repeats"] = repeat_ci(torch, best, steps, stream)
        res["stats_of"] = "graph" if best is not step else "eager"
    del g
    res["persistent"] = bool(d.eng.exec_counters()[5])
    if probe and res["persistent"]:
        # the whole step is one kernel: HIP events around each launch on its stream
        ev = HipEvents()
        b, e = ev.create(steps), ev.create(steps)
        sp = stream.cuda_stream
        for i in range(steps):
            ev.L.hipEventRecord(b[i], sp)
            step(stream=sp)
            ev.L.hipEventRecord(e[i], sp)
        torch.cuda.synchronize()
        durs = [ev.elapsed_ms(b[i], e[i]) for i in range(steps)]
        ev.destroy(b + e)
        res["kernel_ms"] = float(np.mean(durs))
        res["kernel_ms_median"] = float(np.median(durs))
    elif probe:
        ev = HipEvents()
        n = steps * w.model.n_layers
        b, e = ev.create(n), ev.create(n)
        d.eng.set_probe(0, b, e)
        for _ in range(steps):
            step()
        torch.cuda.synchronize()
        durs = [ev.elapsed_ms(b[i], e[i]) for i in range(n)]
        d.eng.set_probe(0, [], [])
        ev.destroy(b + e)
        res["kernel_ms"] = float(np.mean(durs))
        res["kernel_ms_median"] = float(np.median(durs))
    if trace and res["persistent"]:
        res["timeline"] = step_timeline(torch, d)
        print(f"[bench] {w.name} timeline: {json.dumps(res['timeline'])}", file=sys.stderr, flush=True)
    d.eng.device_status(stream.cuda_stream)
    res["counters"] = d.eng.exec_counters().tolist()[:6]
    d.release()
    del d
    torch.cuda.empty_cache()
    return res


def decode_loop(torch, w, n_steps=16, warm=2):
    """A real decode loop: every step reserves one more position per sequence
    in the host allocator, rebuilds and uploads the batch metadata, and runs
    the step on the previous step's greedy ids (device to device, no host
    sync).  Wall-clock per step in steady state, with the host work
    overlapping the device's previous steps."""
    from paper_2609_37062_amd.runner import DeviceRun
    print(f"[bench] decode loop on {w.name}", file=sys.stderr, flush=True)
    kvmax = max(s.ctx + s.q_len for s in w.seqs)
    d = DeviceRun(w, max_kv_len=kvmax + n_steps + warm + 1)
    seqs = list(range(w.n_seqs))
    ones = [1] * w.n_seqs
    meta_t = torch.empty(4 * d.meta_bytes + 4096, dtype=torch.uint8, device=d.device)
    meta = meta_t.data_ptr() + ((-meta_t.data_ptr()) % 256)
    ids = [d.ids.clone(), torch.empty_like(d.ids)]
    sp = d.sp

    def one(i):
        for q in seqs:
            d.eng.reserve(q, 1)
        d.eng.batch_build(seqs, ones)
        d.eng.batch_upload(meta, meta_t.numel() - 256, sp)
        d.eng.decode_step(ids[i % 2].data_ptr(), d.logits.data_ptr(), ids[(i + 1) % 2].data_ptr(), d.ws,
                          d.ws_bytes, sp)

    for i in range(warm):
        one(i)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(warm, warm + n_steps):
        one(i)
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) * 1e3 / n_steps
    d.release()
    del d
    torch.cuda.empty_cache()
    return {"steps": n_steps, "ms_per_step_wall": round(wall, 4),
            "note": "host allocator reserve + batch build + asynchronous upload + decode step per step"}


def stream_ceiling(torch, gib=4):
    """Best stream-read rate of a plain read kernel over `gib` GiB (GB/s)."""
    from paper_2609_37062_amd import vsk
    n = gib << 30
    src = torch.empty(n, dtype=torch.uint8, device="cuda")
    src.fill_(3)
    out = torch.empty(16384, dtype=torch.int32, device="cuda")
    stream = torch.cuda.current_stream()
    best = None
    for wgs in (256, 512, 1024, 2048, 4096):
        fn = lambda: vsk.stream_read(src.data_ptr(), n, out.data_ptr(), wgs, stream.cuda_stream)
        fn()
        r = replay_stats(torch, fn, stream, 10)
        rate = n / (r["median_ms"] / 1e3) / 1e9
        if best is None or rate > best[0]:
            best = (rate, wgs, r["median_ms"])
    del src, out
    torch.cuda.empty_cache()
    return {"GBps": round(best[0], 1), "workgroups": best[1], "bytes": n, "median_ms": best[2],
            "frac_of_peak": round(best[0] * 1e9 / PEAK_HBM, 4)}


def cpu_info():
    model = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return model


def cpu_baseline(w, n_layers_sample, reps=3):
    """Time the float64 oracle on a sample: all rows of the workload through
    1 and 1 + n_layers_sample layers plus the lm_head, each the median of
    `reps` runs after a warm-up, extrapolated per layer to the full step
    (rows per second of the whole step)."""
    import copy
    from dataclasses import replace

    from threadpoolctl import threadpool_info

    sys.path.insert(0, os.path.join(ROOT, "tests"))
    from oracle.model import GeneratedWeights, forward
    from helpers import oracle_state

    times = {}
    for nl in (1, 1 + n_layers_sample):
        ws = copy.copy(w)
        ws.model = replace(w.model, n_layers=nl)
        a, batch, sub, rows, kv, idx = oracle_state(ws)
        W = GeneratedWeights(ws.model, w.seed, cache=True)
        for l in range(nl):  # weights drawn before timing
            for n in ("wq", "wk", "wv", "wo", "w_gate", "w_up", "w_down", "attn_norm", "mlp_norm"):
                W.get(n, l)
        W.over[("lm_head", -1)] = GeneratedWeights(ws.model, w.seed).get("lm_head", -1)
        W.get("final_norm", -1)
        lr = np.arange(w.n_rows)
        runs = []
        for i in range(reps + 1):  # the first is the warm-up
            t0 = time.perf_counter()
            forward(ws.model, W, kv, sub, w.tokens[rows], lr)
            if i:
                runs.append(time.perf_counter() - t0)
        times[nl] = float(np.median(runs))
        del W, kv
    t_layer = (times[1 + n_layers_sample] - times[1]) / n_layers_sample
    t_step = times[1] + (w.model.n_layers - 1) * t_layer
    info = threadpool_info()
    threads = max([i.get("num_threads", 1) for i in info] + [1])
    blas = ", ".join(sorted({f"{i.get('internal_api')} {i.get('version')}" for i in info if i.get("user_api") == "blas"}))
    return {"value": w.n_rows / t_step, "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
            "sample": (f"{w.name}: all {w.n_rows} rows through 1 and {1 + n_layers_sample} of "
                       f"{w.model.n_layers} layers + lm_head (float64 NumPy, weights and KV drawn "
                       f"before timing), each the median of {reps} run(s) after a warm-up; per-layer time "
                       f"extrapolated to the full step"),
            "cpu_model": cpu_info(), "blas": blas or "unknown", "s_per_step": t_step}


def routed_tape(w, s=0.5, seed=7):
    """Random skip over the routed layers: every request skips, each routed
    decision projects with probability s."""
    from workloads import routes
    req = np.arange(w.n_seqs)
    pos = np.array([q.ctx for q in w.seqs])
    return routes.random_skip(seed, w.model.n_routed, req, pos, 1.0, s)


def fit_line(x, y):
    """Least-squares intercept and slope."""
    A = np.stack([np.ones(len(x)), np.asarray(x, np.float64)], axis=1)
    (a, b), *_ = np.linalg.lstsq(A, np.asarray(y, np.float64), rcond=None)
    return float(a), float(b)


def sweep(torch, rows_list, steps=10, warmup=3, ctx=1024, s_skip=0.5):
    """Per-step latency lines of the two modes over the row count at a fixed
    context (8B-class model, 16 of 32 layers routed, half the routed
    decisions Project-Only), eager and captured as a graph at each row count
    (capacity C = rows); the gate/up projection's own time per row count
    locates the ridge.  One JSON line per row count, then the fitted lines,
    tau (routed intercept minus dense intercept), the graph-vs-eager
    overhead, the measured ridge and the decode rule's thresholds on this
    device."""
    from paper_2609_37062_amd import vsk
    from paper_2609_37062_amd.runner import DeviceRun
    from workloads.configs import M8B, decode_workload
    rmax = max(rows_list)
    w = decode_workload(M8B, np.full(rmax, ctx), seed=0, name=f"8B-sweep-ctx{ctx}")
    print(f"[sweep] setting up {rmax} rows x {ctx} context (KV left at zero)", file=sys.stderr, flush=True)
    d = DeviceRun(w, routed=True, fill_kv=False)
    stream = torch.cuda.current_stream()
    ev = HipEvents()
    pts = []
    for R in rows_list:
        d.rebatch(range(R))
        wr = decode_workload(M8B, np.full(R, ctx), seed=0)
        d.set_route(*routed_tape(wr, s_skip))
        rec = {"rows": R}
        for mode, fn in (("dense", d.step), ("routed", d.step_routed)):
            ms_e, _ = time_steps(torch, fn, steps, warmup, stream)
            g = capture(torch, fn)
            settle(torch, g.replay)
            ms_g, _ = time_steps(torch, g.replay, steps, warmup, stream)
            del g
            rec[f"{mode}_eager_ms"] = round(ms_e, 4)
            rec[f"{mode}_graph_ms"] = round(ms_g, 4)
        # gate/up launches of a dense step (the weight-stationary GEMM of the rule)
        n = M8B.n_layers * 3
        b, e = ev.create(n), ev.create(n)
        d.eng.set_probe(0, b, e)
        for _ in range(3):
            d.step()
        torch.cuda.synchronize()
        gu = float(np.median([ev.elapsed_ms(b[i], e[i]) for i in range(n)]))
        d.eng.set_probe(0, [], [])
        ev.destroy(b + e)
        rec["gateup_us"] = round(gu * 1e3, 2)
        pts.append(rec)
        print(json.dumps({"sweep_point": rec}), flush=True)
    d.release()
    rows = [p["rows"] for p in pts]
    best = lambda p, m: min(p[f"{m}_eager_ms"], p[f"{m}_graph_ms"])
    ad, bd = fit_line(rows, [best(p, "dense") for p in pts])
    ar, br = fit_line(rows, [best(p, "routed") for p in pts])
    tau = (ar - ad) * 1e-3
    # ridge: the gate/up time is flat while weight-bound, then grows with rows;
    # M* = rows where the flat level meets the line through the largest counts
    gu = np.array([p["gateup_us"] for p in pts])
    flat = float(np.median(gu[: max(2, len(gu) // 3)]))
    hi = [(r, g) for r, g in zip(rows, gu) if g > 1.5 * flat]
    m_star = None
    if len(hi) >= 2:
        a, bslope = fit_line([r for r, _ in hi], [g for _, g in hi])
        if bslope > 0:
            m_star = round((flat - a) / bslope, 1)
    bw = stream_ceiling(torch)["GBps"] * 1e9
    L_r, kvb = M8B.n_routed, M8B.kv_bytes_per_token_layer
    vstar, ex, en = vsk.switch_thresholds(max(tau, 1e-9), bw, s_skip, L_r, kvb, tau_layers=L_r)
    graph_over = [p["dense_graph_ms"] - p["dense_eager_ms"] for p in pts]
    summary = {"sweep": "8B-class, 1k context, random skip s=0.5 over 16 routed layers",
               "dense_line_ms": {"intercept": round(ad, 4), "slope_per_row": round(bd, 6)},
               "routed_line_ms": {"intercept": round(ar, 4), "slope_per_row": round(br, 6)},
               "tau_ms": round(tau * 1e3, 4), "graph_minus_eager_ms": [round(x, 4) for x in graph_over],
               "gateup_flat_us": round(flat, 2), "ridge_rows_measured": m_star,
               "stream_read_GBps": round(bw / 1e9, 1),
               "rule_on_this_device": {"v_star_tokens": round(vstar), "exit_tokens": ex, "enter_tokens": en,
                                       "tau_layers": L_r, "skip": s_skip, "kv_bytes": kvb}}
    print(json.dumps(summary), flush=True)


def main():
    a = parse()
    if a.gpus != 1:
        print(json.dumps({"error": "the library runs on one GPU; --gpus must be 1", "n_gpus": a.gpus}))
        sys.exit(2)
    import torch

    from workloads.configs import workload

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    if a.sweep:
        sweep(torch, [int(x) for x in a.sweep_rows.split(",")])
        return
    w = workload(a.workload)
    if a.profile_pass:
        from paper_2609_37062_amd.runner import DeviceRun
        d = DeviceRun(w)
        apply_tuning(d, a.mode, a.tune)
        src = torch.empty(CALIB_BYTES, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        src.fill_(1)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        # a plain read of known size (k_stream_read) for the byte counters
        from paper_2609_37062_amd import vsk
        out = torch.empty(4096, dtype=torch.int32, device="cuda")
        vsk.stream_read(src.data_ptr(), CALIB_BYTES, out.data_ptr(), 512, torch.cuda.current_stream().cuda_stream)
        torch.cuda.synchronize()
        for _ in range(a.steps):
            d.step()
        torch.cuda.synchronize()
        print(f"[bench] profile pass: {w.name}, {a.steps} steps, calibration copy and read of {CALIB_BYTES} bytes",
              file=sys.stderr)
        return
    r = measure(torch, w, a.steps, a.warmup, not a.no_graph, mode=a.mode, trace=a.trace, tune=a.tune,
                stats=max(a.replays, a.steps))
    ms = min(r["ms_eager"], r.get("ms_graph", float("inf")))
    tokps = w.n_rows / (ms / 1e3)
    sb = step_bytes(w)
    mixed = a.workload == 4
    if r["persistent"]:
        kname = "persistent decode step (k_step: every layer's projections, attention, lm_head, argmax)"
        kb = sb
    else:
        kname = "gate/up projection + SwiGLU (k_gemm, EPI_SWIGLU)"
        kb = gateup_bytes(w.model, w.n_rows)
    achieved = kb / (r["kernel_ms"] / 1e3)
    traffic = (None if r["persistent"] else gateup_traffic()) if a.workload == 2 else None
    roofline = {"bound": "hbm", "kernel": kname,
                "achieved": round(achieved / 1e9, 1), "peak": PEAK_HBM / 1e9, "unit": "GB/s",
                "frac": round(achieved / PEAK_HBM, 4),
                "traffic": traffic,
                "traffic_source": ("stored rocprofv3 counters of this kernel source "
                                   "(profiles/gateup_3b_b16_traffic.json)") if traffic is not None else None,
                "bytes_per_launch": kb, "avg_launch_ms": round(r["kernel_ms"], 5)}
    if mixed:
        # the 2,080-row pass is bound by the matrix cores: gate/up's flops over its launch time
        fl = gateup_flops(w.model, w.n_rows)
        tf = fl / (r["kernel_ms"] / 1e3) / 1e12
        roofline = {"bound": "mfma", "kernel": kname, "achieved": round(tf, 1), "peak": PEAK_MFMA_BF16 / 1e12,
                    "unit": "TFLOP/s", "frac": round(tf * 1e12 / PEAK_MFMA_BF16, 4), "traffic": None,
                    "flops_per_launch": fl, "avg_launch_ms": round(r["kernel_ms"], 5)}
    out = {
        "metric": ("mixed prefill + decode pass: rows/s; achieved matrix-core TFLOP/s vs peak" if mixed else
                   "decode-step latency (ms) & tokens/s at batch 16/64; achieved HBM TB/s vs peak"),
        "value": round(tokps, 1),
        "unit": "rows/s" if mixed else "tokens/s",
        "n_gpus": 1,
        "steps": a.steps,
        "warmup": a.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": w.name, "batch": w.n_rows, "layers": w.model.n_layers,
                   "hidden": w.model.hidden, "heads": f"{w.model.n_q_heads}/{w.model.n_kv_heads}x{w.model.head_dim}",
                   "ffn": w.model.ffn, "vocab": w.model.vocab,
                   "resident_tokens": w.resident_tokens(), "kv_block": 16},
        "ms_eager": round(r["ms_eager"], 4),
        "ms_graph": round(r["ms_graph"], 4) if "ms_graph" in r else None,
        "graph_matches_eager": r.get("graph_matches_eager"),
        "per_replay": r.get("per_replay"),
        "repeats": r.get("repeats"),
        "stats_of": r.get("stats_of"),
        "step_bytes": sb,
        "step_hbm_TBps": round(sb / (ms / 1e3) / 1e12, 3),
        "step_hbm_frac": round(sb / (ms / 1e3) / PEAK_HBM, 4),
        "roofline": roofline,
        "exec_counters": r["counters"],
    }
    if mixed:
        sf = step_flops(w)
        out["step_flops"] = sf
        out["step_TFLOPs"] = round(sf / (ms / 1e3) / 1e12, 1)
        out["step_mfma_frac"] = round(sf / (ms / 1e3) / PEAK_MFMA_BF16, 4)
    if "timeline" in r:
        out["timeline"] = r["timeline"]
    sc = stream_ceiling(torch)
    out["stream_read_ceiling"] = sc
    out["step_frac_of_stream_ceiling"] = round(sb / (ms / 1e3) / (sc["GBps"] * 1e9), 4)
    if not a.no_loop and a.mode != 2 and not mixed:
        out["decode_loop"] = decode_loop(torch, w)
    if not a.no_routed and a.mode != 2 and not mixed:
        rr = measure(torch, w, a.steps, a.warmup, not a.no_graph, probe=False, tune=a.tune, route=routed_tape(w))
        msr = min(rr["ms_eager"], rr.get("ms_graph", float("inf")))
        out["routed"] = {"workload": w.name, "policy": "random skip, half of the routed decisions Project-Only",
                         "routed_layers": w.model.n_routed, "proj_ffn": w.model.proj_dim,
                         "ms_per_step": round(msr, 4), "ms_eager": round(rr["ms_eager"], 4),
                         "ms_graph": round(rr["ms_graph"], 4) if "ms_graph" in rr else None,
                         "graph_matches_eager": rr.get("graph_matches_eager"),
                         "tokens_per_s": round(w.n_rows / (msr / 1e3), 1)}
    if not a.no_batch64 and a.workload == 2:
        w3 = workload(3)
        r3 = measure(torch, w3, a.steps, a.warmup, not a.no_graph, probe=False, mode=a.mode if a.mode != 2 else 0,
                     tune=a.tune)
        ms3 = min(r3["ms_eager"], r3.get("ms_graph", float("inf")))
        sb3 = step_bytes(w3)
        out["batch64_shared_prefix"] = {
            "workload": w3.name, "ms_per_step": round(ms3, 4), "tokens_per_s": round(w3.n_rows / (ms3 / 1e3), 1),
            "ms_eager": round(r3["ms_eager"], 4), "ms_graph": round(r3["ms_graph"], 4) if "ms_graph" in r3 else None,
            "step_bytes": sb3, "step_hbm_TBps": round(sb3 / (ms3 / 1e3) / 1e12, 3),
            "step_hbm_frac": round(sb3 / (ms3 / 1e3) / PEAK_HBM, 4)}
    if not a.no_cpu:
        print("[bench] timing the CPU oracle sample", file=sys.stderr, flush=True)
        # the 2,080-row pass costs the oracle minutes per layer: one timed run each
        cb = cpu_baseline(w, a.cpu_layers, reps=1 if mixed else 3)
        if mixed:
            cb["unit"] = "rows/s"
        cb.pop("s_per_step")
        cb["value"] = round(cb["value"], 4)
        out["cpu_baseline"] = cb
    print(json.dumps(out))


if __name__ == "__main__":
    main()
