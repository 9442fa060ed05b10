#!/usr/bin/env python3
"""Throughput of the Grouped Cross Attention hot path on one MI355X.

One step = the whole path over one batch of the 64K-context training workload
(B=2, H=16, d=64, L=65,536, S=64, 1,024 chunks, top-8, bf16): landmark scores,
top-k, grouped cross attention forward, and its backward into q, k, v, the
retrieval scores and both landmark tensors.  Inputs are seeded synthetic
N(0,1) tensors already resident in HBM when the timed region starts.

Prints ONE JSON line.  Besides the headline tokens/s it carries:
  roofline     - the dominant kernel's achieved rate against its roofline peak.
                 The timed region (K steps between two events, nothing else on
                 the stream) gives ms_per_step; the same K steps are then run
                 again with every kernel dispatched with its own start and stop
                 events (the kernel alone, on its stream), which give each
                 kernel's average duration; traffic and matrix-core busy
                 fraction come from the committed rocprofv3 counter summaries
                 when they were taken from the current kernel sources;
  cpu_baseline - the CPU oracle timed on a bounded sample of the same workload;
  forward_16k  - the forward of the 16K training workload (B=8, H=12), tokens/s;
  planted_1m   - the forward of the 1M-token planted workload, tokens/s, with the
                 selection's matrix-core rate;
  decode_scan  - the 16M-context decode retrieval (one 64-token chunk scored
                 against 262,144 past landmark keys, top-8, attention over the
                 8 gathered chunks) in GB/s against HBM peak;
  peaks_measured - on-device streaming-read and matrix-core loop rates (the
                 spec peaks stay the roofline reference).
Every leg with an oracle baseline reports it in the leg's own unit.
"""

import argparse
import ctypes
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
BF16_PEAK_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
S, DH = 64, 64


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


# ------------------------------------------------------------ HIP events ----

class Events:
    """Raw hipEvent_t handles (the library records them on the kernels' stream)."""

    def __init__(self, n):
        self.hip = ctypes.CDLL("libamdhip64.so")
        self.n = n
        self.arr = (ctypes.c_void_p * n)()
        for i in range(n):
            assert self.hip.hipEventCreate(ctypes.byref(self.arr, i * ctypes.sizeof(ctypes.c_void_p))) == 0
        self.hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                                 ctypes.c_void_p]
        self.hip.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]

    def record(self, i, stream):
        assert self.hip.hipEventRecord(self.arr[i], ctypes.c_void_p(stream.cuda_stream)) == 0

    def ms(self, a, b):
        out = ctypes.c_float()
        assert self.hip.hipEventElapsedTime(ctypes.byref(out), self.arr[a], self.arr[b]) == 0
        return out.value

    def close(self):
        for i in range(self.n):
            self.hip.hipEventDestroy(self.arr[i])


def timed(run_step, steps, stream):
    """ms between events recorded on `stream` before the first and after the last
    of `steps` steps, with synchronisation on both sides (the timed region)."""
    import torch
    ev = Events(2)
    torch.cuda.synchronize()
    ev.record(0, stream)
    for _ in range(steps):
        run_step()
    ev.record(1, stream)
    torch.cuda.synchronize()
    total = ev.ms(0, 1)
    ev.close()
    return total


def step_latency(run_step, steps, stream, isolated=False):
    """Distribution of one step's duration: an event pair around every step.
    Back to back (isolated=False) each duration is the step's share of the
    stream, queue gaps included; isolated=True waits for the device after every
    step, so a duration also holds the launch of an idle stream.  Returns
    {"median", "p10", "p90", "min", "max"} in ms."""
    import torch
    evs = Events(2 * steps)
    torch.cuda.synchronize()
    for i in range(steps):
        evs.record(2 * i, stream)
        run_step()
        evs.record(2 * i + 1, stream)
        if isolated:
            torch.cuda.synchronize()
    torch.cuda.synchronize()
    d = sorted(evs.ms(2 * i, 2 * i + 1) for i in range(steps))
    evs.close()

    def q(f):
        x = f * (len(d) - 1)
        lo = int(x)
        hi = min(lo + 1, len(d) - 1)
        return d[lo] + (d[hi] - d[lo]) * (x - lo)
    return {"median": q(0.5), "p10": q(0.1), "p90": q(0.9), "min": d[0], "max": d[-1], "n": len(d)}


def kernel_times(run_step, steps, stream, gca, per_step_capacity=32):
    """Run `steps` steps with the per-kernel hook armed: every kernel's dispatch
    carries a start and a stop event, so the hook adds nothing to the stream.
    Returns (ms between events recorded before the first and after the last step,
    {kernel: [durations ms]})."""
    import torch
    outer = Events(2)
    evs = Events(min(4096, 2 * steps * per_step_capacity))
    torch.cuda.synchronize()
    gca.profile_arm(evs.arr, evs.n)
    outer.record(0, stream)
    for _ in range(steps):
        run_step()
    outer.record(1, stream)
    torch.cuda.synchronize()
    names = gca.profile_record()
    gca.profile_arm(None, 0)
    per = {}
    for i, name in enumerate(names):
        per.setdefault(name, []).append(evs.ms(2 * i, 2 * i + 1))
    total = outer.ms(0, 1)
    outer.close()
    evs.close()
    return total, per


def kernel_table(per, steps):
    return {k: {"avg_ms": sum(v) / len(v), "launches_per_step": len(v) / steps, "ms_per_step": sum(v) / steps}
            for k, v in per.items()}


# ------------------------------------------------------------ workloads ----

def upload(w, a, dev):
    import numpy as np
    import torch
    a = np.ascontiguousarray(a)
    if w.dtype == "bf16":
        return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(dev)
    return torch.from_numpy(a).to(dev)


def landmarks(w):
    """Seeded landmark inputs from the shared generator (throughput does not need the
    parity tests' top-k margin check)."""
    from gen import inputs as gi
    return gi.draw_landmarks(w)


def valid_units(idx_host, w):
    """Valid (batch, head, query chunk, slot) tuples the attention kernels process."""
    valid = (idx_host >= 0)
    if w.mode == "causal":
        per_row = valid[:, :, :-1, :].sum()      # row t feeds chunk t+1
    else:
        per_row = valid.sum()
    return int(per_row) * (w.H // w.Hr)


def _profile_entry(path, kernel):
    """Entry `kernel` of a committed rocprofv3 summary, or None when there is none or
    the kernel sources changed since it was taken."""
    try:
        from profiling import source_hash
        data = json.load(open(os.path.join(ROOT, "profiles", path)))
        if data.get("source_sha256") != source_hash():
            return None
        return data["kernels"][kernel]
    except (OSError, KeyError, ValueError):
        return None


def measured_traffic(kernel):
    """HBM bytes per launch (fetch + write) from the committed counter summary."""
    k = _profile_entry("hbm_traffic.json", kernel)
    return None if k is None else k["fetch_bytes_per_launch"] + k["write_bytes_per_launch"]


def measured_mfma(kernel):
    """Matrix-core busy fraction and bf16 matrix-core ops per launch from the
    committed counter summary."""
    k = _profile_entry("mfma_counters.json", kernel)
    if k is None:
        return None
    return {key: k.get(key) for key in ("mfma_busy_frac", "mfma_bf16_flops_per_launch", "l2_hit_frac",
                                        "l2_miss_read_latency_cycles")}


def flops_per_unit():
    # per valid (query token, slot, head): one S x d product is 2*S*d flops
    return {"xattn_fwd_kernel": 2 * (2 * S * DH),     # S = QK^T and PV
            "bwd_dq_kernel": 3 * (2 * S * DH),        # S recompute, dP = dO V^T, dQ = dS K
            "bwd_dkdv_kernel": 2 * (2 * S * DH)}      # dV = P^T dO, dK = dS^T Q (its own S/dP recompute not counted)


def profile_key(kernel, tag=None):
    """Name of a kernel's entry in the committed counter summaries: the 64K train
    step's kernels untagged, other workloads' as kernel@tag."""
    return kernel if tag is None else f"{kernel}@{tag}"


def mfma_roofline(kern, units, dom, tag=None):
    fpu = flops_per_unit()
    fl = units * S * fpu[dom]
    ach = fl / (kern[dom]["avg_ms"] * 1e-3) / 1e12
    key = profile_key(dom, tag)
    traffic = measured_traffic(key)
    return {"kernel": dom, "bound": "mfma", "achieved": ach, "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
            "frac": ach / BF16_PEAK_TFLOPS, "traffic": traffic, "counters": measured_mfma(key),
            # the rate the traffic beyond the L2 moves at in this launch
            "traffic_GBps": None if traffic is None else traffic / (kern[dom]["avg_ms"] * 1e-3) / 1e9,
            "algorithmic_flops_per_launch": fl, "avg_launch_ms": kern[dom]["avg_ms"]}


def forward_outputs(p, gca, dev):
    import torch
    sh = gca.shapes(p)
    dt = torch.bfloat16 if p.dtype == gca.GCA_BF16 else torch.float32
    return {"out": torch.empty(sh.q, dtype=dt, device=dev),
            "idx": torch.empty(sh.rows, dtype=torch.int32, device=dev),
            "sel": torch.empty(sh.rows, dtype=torch.float32, device=dev),
            "lse": torch.empty(sh.lse, dtype=torch.float32, device=dev),
            "w": torch.empty(sh.rows, dtype=torch.float32, device=dev)}


# ------------------------------------------------------ 64K fwd + bwd ----

def bench_train(args, dev, gca):
    import torch
    from gen import get_workload, inputs as gi

    w = get_workload("fwdbwd_64k_bf16")
    lq, lk = landmarks(w)
    t = {"lmk_q": upload(w, lq, dev), "lmk_k": upload(w, lk, dev)}
    t.update(gi.device_tensors(w, ("q", "k", "v", "dout"), dev))
    p = gca.problem(w.B, w.H, w.n_chunks, w.topk, D=w.Dl, Hr=w.Hr, dtype=w.dtype, mode=w.mode)
    sh = gca.shapes(p)
    fo = forward_outputs(p, gca, dev)
    grads = {"dq": torch.empty(sh.q, dtype=torch.bfloat16, device=dev),
             "dk": torch.empty(sh.kv, dtype=torch.bfloat16, device=dev),
             "dv": torch.empty(sh.kv, dtype=torch.bfloat16, device=dev),
             "dsel": torch.empty(sh.rows, dtype=torch.float32, device=dev),
             "dlmk_q": torch.empty(sh.lmk_q, dtype=torch.float32, device=dev),
             "dlmk_k": torch.empty(sh.lmk_k, dtype=torch.float32, device=dev)}
    wsf, _ = gca.workspace(p, gca.OP_FORWARD, dev)
    wsb, _ = gca.workspace(p, gca.OP_BACKWARD, dev)

    def step(pp=p):
        gca.forward(pp, t["lmk_q"], t["lmk_k"], t["q"], t["k"], t["v"], ws=wsf, **fo)
        gca.grouped_xattn_bwd(pp, t["q"], t["k"], t["v"], fo["idx"], fo["sel"], fo["lse"], t["dout"],
                              t["lmk_q"], t["lmk_k"], ws=wsb, grads=grads)

    stream = torch.cuda.current_stream()
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    log(f"warmup done ({args.warmup} steps)")

    # timed region: K steps bracketed by synchronisation, nothing else on the stream
    t0 = time.perf_counter()
    ms_step = timed(step, args.steps, stream) / args.steps
    wall = time.perf_counter() - t0
    log(f"timed {args.steps} steps: {ms_step:.3f} ms/step (wall {wall:.2f}s)")
    # the same K steps again with every kernel's dispatch carrying start/stop events
    prof_ms, per = kernel_times(step, args.steps, stream, gca)
    log(f"profiled {args.steps} steps: {prof_ms / args.steps:.3f} ms/step")
    lat = step_latency(step, max(args.steps, 50), stream)
    log(f"per-step latency: median {lat['median']:.3f} p10 {lat['p10']:.3f} p90 {lat['p90']:.3f} ms")
    idx_host = fo["idx"].cpu().numpy()
    gumbel = lmk_row = None
    if not args.no_variants:
        # the Gumbel top-k variant of the same step (noise in the selection only)
        pg = gca.problem(w.B, w.H, w.n_chunks, w.topk, D=w.Dl, Hr=w.Hr, dtype=w.dtype, mode=w.mode, gumbel_seed=1)
        step(pg)
        g_ms = timed(lambda: step(pg), args.steps, stream) / args.steps
        _, g_per = kernel_times(lambda: step(pg), args.steps, stream, gca)
        gumbel = {"value": w.B * w.Lq / (g_ms * 1e-3), "unit": "tokens/s", "ms_per_step": g_ms,
                  "kernels": {k: {"avg_ms": sum(v) / len(v)} for k, v in g_per.items()
                              if k in ("chunk_scores_kernel", "topk_kernel")}}
        log(f"gumbel top-k {args.steps} steps: {g_ms:.3f} ms/step")
        # the same step with S+1 query rows per chunk (each chunk's LMK token as its
        # last query row); k/v and the landmarks are shared with the step above
        wx = get_workload("fwdbwd_64k_bf16", lmk_row=True)
        tx = dict(t, **gi.device_tensors(wx, ("q", "dout"), dev))
        px = gca.problem(w.B, w.H, w.n_chunks, w.topk, D=w.Dl, Hr=w.Hr, dtype=w.dtype, mode=w.mode, lmk_row=True)
        fox = forward_outputs(px, gca, dev)
        gx = dict(grads, dq=torch.empty(gca.shapes(px).q, dtype=torch.bfloat16, device=dev))
        wsbx, _ = gca.workspace(px, gca.OP_BACKWARD, dev)

        def step_x():
            gca.forward(px, tx["lmk_q"], tx["lmk_k"], tx["q"], tx["k"], tx["v"], ws=wsf, **fox)
            gca.grouped_xattn_bwd(px, tx["q"], tx["k"], tx["v"], fox["idx"], fox["sel"], fox["lse"], tx["dout"],
                                  tx["lmk_q"], tx["lmk_k"], ws=wsbx, grads=gx)

        step_x()
        x_ms = timed(step_x, args.steps, stream) / args.steps
        _, x_per = kernel_times(step_x, args.steps, stream, gca)
        lmk_row = {"value": wx.B * wx.Lq / (x_ms * 1e-3), "unit": "tokens/s", "ms_per_step": x_ms,
                   "query_rows_per_chunk": wx.Sq,
                   "kernels": {k: {"avg_ms": sum(v) / len(v)} for k, v in x_per.items()
                               if k in ("xattn_fwd_kernel", "bwd_dq_kernel", "bwd_dkdv_kernel")}}
        log(f"S+1 query rows {args.steps} steps: {x_ms:.3f} ms/step")
        del tx, fox, gx, wsbx

    units = valid_units(idx_host, w)
    kern = kernel_table(per, args.steps)
    for name in flops_per_unit():
        if name in kern:
            kern[name]["tflops"] = mfma_roofline(kern, units, name)["achieved"]
    dom = max(kern, key=lambda k: kern[k]["ms_per_step"])
    roof = mfma_roofline(kern, units, dom) if dom in flops_per_unit() else \
        {"kernel": dom, "bound": None, "achieved": None, "peak": None, "unit": None, "frac": None, "traffic": None}
    algo_fl = units * S * (flops_per_unit()["xattn_fwd_kernel"] + 5 * 2 * S * DH)
    return {
        "w": w, "t": t, "tokens": w.B * w.Lq, "ms_step": ms_step, "profiled_ms_step": prof_ms / args.steps,
        "gumbel": gumbel, "lmk_row": lmk_row, "kernels": kern, "roofline": roof, "units": units, "latency": lat,
        "path_tflops": algo_fl / (ms_step * 1e-3) / 1e12,
    }


# ---------------------------------------------- forward-only workloads ----

def bench_forward(args, dev, gca, name):
    """Forward tokens/s of a causal workload (train_16k_bf16 or planted_1m_bf16)."""
    import torch
    from gen import get_workload, inputs as gi

    w = get_workload(name)
    lq, lk = landmarks(w)
    t = {"lmk_q": upload(w, lq, dev), "lmk_k": upload(w, lk, dev)}
    t.update(gi.device_tensors(w, ("q", "k", "v"), dev))
    p = gca.problem(w.B, w.H, w.n_chunks, w.topk, D=w.Dl, Hr=w.Hr, dtype=w.dtype, mode=w.mode)
    fo = forward_outputs(p, gca, dev)
    ws, _ = gca.workspace(p, gca.OP_FORWARD, dev)

    def call():
        gca.forward(p, t["lmk_q"], t["lmk_k"], t["q"], t["k"], t["v"], ws=ws, **fo)

    stream = torch.cuda.current_stream()
    for _ in range(args.warmup):
        call()
    steps = args.fwd_steps
    ms = timed(call, steps, stream) / steps
    _, per = kernel_times(call, steps, stream, gca)
    lat = step_latency(call, max(steps, 50), stream)
    kern = kernel_table(per, steps)
    idx_host = fo["idx"].cpu().numpy()
    units = valid_units(idx_host, w)
    tag = {"train_16k_bf16": "forward_16k", "planted_1m_bf16": "planted_1m"}[name]
    roof = mfma_roofline(kern, units, "xattn_fwd_kernel", tag)
    kern["xattn_fwd_kernel"]["tflops"] = roof["achieved"]
    leg = {"metric": "GCA forward tokens/s", "value": w.B * w.Lq / (ms * 1e-3), "unit": "tokens/s",
           "ms_per_call": ms, "calls": steps, "call_ms_distribution": lat, "kernels": kern, "roofline": roof}
    # the selection's matrix-core rate: 2 D flops per causal (row, earlier chunk) pair
    pairs = w.B * w.Hr * w.n_chunks * (w.n_chunks - 1) // 2
    sel_kernel = "select_part_kernel" if "select_part_kernel" in kern else \
        "fused_select_kernel" if "fused_select_kernel" in kern else "chunk_scores_kernel"
    sfl = 2 * w.Dl * pairs
    sach = sfl / (kern[sel_kernel]["avg_ms"] * 1e-3) / 1e12
    leg["selection"] = {"kernel": sel_kernel, "bound": "mfma", "achieved": sach, "peak": BF16_PEAK_TFLOPS,
                        "unit": "TFLOP/s", "frac": sach / BF16_PEAK_TFLOPS, "algorithmic_flops_per_launch": sfl,
                        "avg_launch_ms": kern[sel_kernel]["avg_ms"],
                        "traffic": measured_traffic(profile_key(sel_kernel, tag)),
                        "counters": measured_mfma(profile_key(sel_kernel, tag))}
    if w.planted:
        pos = gi.plant_positions(w)
        leg["planted_retrieved"] = sorted(idx_host[0, 0, -1].tolist()) == sorted(pos.tolist())
    log(f"{name} forward: {ms:.3f} ms/call")
    host = None
    if not args.no_cpu_baseline:
        host = {"lq": lq, "lk": lk, "q": t["q"][:1, :1].cpu(), "k": t["k"][:1, :1].cpu(),
                "v": t["v"][:1, :1].cpu()}
    del t, fo, ws
    torch.cuda.empty_cache()
    return w, leg, host


def cpu_forward_baseline(w, host, rows=None, chunks=None):
    """The oracle's forward on a bounded sample: scores and top-k for `rows` landmark
    rows of batch 0 and attention of head 0 over `chunks` query chunks, each
    extrapolated to the whole workload (selection by causal candidate pairs,
    attention by (batch, head, chunk))."""
    import numpy as np
    from gen import inputs as gi
    from oracle import gca as og
    nQ = w.n_chunks
    rows = np.arange(nQ) if rows is None else np.asarray(rows)
    chunks = range(nQ) if chunks is None else chunks
    lq = gi.decode(w, host["lq"][:1, :1])
    lk = gi.decode(w, host["lk"][:1, :1])
    t0 = time.perf_counter()
    r = og.scores(lq, lk, w.score_scale, w.mode, rows=rows)
    idx_s, sel_s = og.topk(r, w.topk, rows=rows)
    t_sel = time.perf_counter() - t0
    # the attention sample needs the full row set of its chunks' retrieval rows
    need = sorted({c - 1 for c in chunks if c >= 1})
    r2 = og.scores(lq, lk, w.score_scale, w.mode, rows=need)
    i2, s2 = og.topk(r2, w.topk, rows=need)
    idx = np.full((1, 1, nQ, w.topk), -1, np.int32)
    sel = np.full((1, 1, nQ, w.topk), -np.inf)
    idx[0, 0, need], sel[0, 0, need] = i2[0, 0], s2[0, 0]
    wt = og.fusion_weights(sel)
    host64 = lambda x: x.float().double().numpy()
    q, k, v = host64(host["q"]), host64(host["k"]), host64(host["v"])
    t1 = time.perf_counter()
    og.xattn_fwd(q, k, v, idx, wt, w.S, w.attn_scale, w.mode, chunks=chunks)
    t_att = time.perf_counter() - t1
    pairs_sample = int(sum(min(int(t), nQ) for t in rows))
    pairs_all = w.B * w.Hr * nQ * (nQ - 1) // 2
    full = t_sel * pairs_all / max(pairs_sample, 1) + t_att * (w.B * w.H * nQ) / len(list(chunks))
    return {"value": w.B * w.Lq / full, "unit": "tokens/s", "kind": "oracle",
            "sample": f"batch 0, retrieval head 0: scores + top-k for {len(rows)} landmark rows ({t_sel:.2f}s), "
                      f"attention of head 0 over {len(list(chunks))} query chunks ({t_att:.2f}s); extrapolated "
                      f"by candidate pairs and by (batch, head, chunk) to B={w.B}, H={w.H}, {nQ} chunks",
            "sample_seconds": t_sel + t_att, **host_info()}


# -------------------------------------------------------- 16M decode ----

def bench_decode(args, dev, gca):
    """16M-context decode retrieval: GB/s of algorithmic bytes against HBM peak."""
    import torch
    from gen import get_workload, inputs as gi

    w = get_workload("decode_16m_bf16")
    lq, lk = landmarks(w)
    lmk_q = upload(w, lq, dev)
    keys = [upload(w, lk, dev)]
    keys.append(keys[0].clone())                   # 2 x 268 MB: rotation defeats the 256 MB MALL
    kv = gi.device_kv(w, dev)
    q = gi.device_tensors(w, ("q",), dev)["q"]
    p = gca.problem(w.B, w.H, w.n_chunks, w.topk, D=w.Dl, Hr=w.Hr, dtype=w.dtype, mode=w.mode)
    fo = forward_outputs(p, gca, dev)
    ws, _ = gca.workspace(p, gca.OP_FORWARD, dev)
    it = [0]

    def call(pp=p):
        gca.forward(pp, lmk_q, keys[it[0] % 2], q, kv["k"], kv["v"], ws=ws, **fo)
        it[0] += 1

    for _ in range(5):
        call()
    torch.cuda.synchronize()
    steps = args.decode_steps
    stream = torch.cuda.current_stream()
    ms_call = timed(call, steps, stream) / steps
    prof_ms, per = kernel_times(call, steps, stream, gca)
    # per call: back to back (the steady state) and with the device idle before
    # every call (the latency a lone decode step sees)
    lat = {"steady_state": step_latency(call, max(steps, 50), stream),
           "isolated": step_latency(call, max(steps, 50), stream, isolated=True)}
    planted = int(gi.plant_positions(w)[0])
    idx_host = fo["idx"].cpu().numpy()
    found = planted in idx_host.ravel().tolist()
    # the Gumbel top-k variant of the same call
    gumbel = None
    if not args.no_variants:
        pg = gca.problem(w.B, w.H, w.n_chunks, w.topk, D=w.Dl, Hr=w.Hr, dtype=w.dtype, mode=w.mode, gumbel_seed=1)
        call(pg)
        g_ms = timed(lambda: call(pg), steps, stream) / steps
        _, g_per = kernel_times(lambda: call(pg), steps, stream, gca)
        gumbel = {"value": None, "unit": "GB/s", "ms_per_call": g_ms,
                  "kernels": {k: {"avg_ms": sum(v) / len(v)} for k, v in g_per.items()}}
    key_bytes = w.n_chunks * w.Dl * 2
    kv_bytes = 2 * w.topk * w.H * S * DH * 2
    io_bytes = 2 * w.H * S * DH * 2 + w.Dl * 2
    total_bytes = key_bytes + kv_bytes + io_bytes
    scan_ms = sum(per["decode_scan_kernel"]) / len(per["decode_scan_kernel"])
    scan_gbs = key_bytes / (scan_ms * 1e-3) / 1e9
    host = None
    if not args.no_cpu_baseline:
        # what the oracle needs for the same call: the landmarks and the K/V of
        # the chunks it retrieves (the rest of the cache is never read)
        sel_chunks = sorted(set(int(j) for j in idx_host.ravel() if j >= 0))
        host = {"lq": lq, "lk": lk, "q": q.cpu(), "chunks": sel_chunks,
                "k": {j: kv["k"][:, :, j * S:(j + 1) * S].cpu() for j in sel_chunks},
                "v": {j: kv["v"][:, :, j * S:(j + 1) * S].cpu() for j in sel_chunks}}
    del kv, keys
    torch.cuda.empty_cache()
    leg = {
        "metric": "retrieval-scan GB/s at 16M-ctx decode", "unit": "GB/s",
        "value": total_bytes / (ms_call * 1e-3) / 1e9, "ms_per_call": ms_call, "calls": steps,
        "profiled_ms_per_call": prof_ms / steps, "call_ms_distribution": lat,
        "bytes_per_call": total_bytes, "frac_of_hbm_peak": total_bytes / (ms_call * 1e-3) / 1e9 / HBM_PEAK_GBS,
        "planted_retrieved": found,
        "config": {"workload": "decode_16m_bf16: B=1 H=8 d=64, 16,777,216 past tokens (262,144 chunks), "
                               "S=64, top-8, D=512, bf16"},
        "roofline": {"kernel": "decode_scan_kernel", "bound": "hbm", "achieved": scan_gbs, "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": scan_gbs / HBM_PEAK_GBS,
                     "traffic": measured_traffic("decode_scan_kernel@decode_16m"),
                     "algorithmic_bytes_per_launch": key_bytes, "avg_launch_ms": scan_ms},
        "kernels": kernel_table(per, steps),
        "gumbel_topk": gumbel,
    }
    if gumbel is not None:
        gumbel["value"] = total_bytes / (gumbel["ms_per_call"] * 1e-3) / 1e9
    return w, leg, host, total_bytes


def cpu_decode_baseline(w, host, total_bytes):
    """The oracle's whole decode call: scores of the one landmark query against all
    262,144 past keys, top-k, weights, and the attention of all 8 heads over the
    retrieved chunks (the oracle reads only those chunks' K/V)."""
    import numpy as np
    from gen import inputs as gi
    from oracle import gca as og
    t0 = time.perf_counter()
    lq = gi.decode(w, host["lq"])
    lk = gi.decode(w, host["lk"])
    r = og.scores(lq, lk, w.score_scale, w.mode)
    idx, sel = og.topk(r, w.topk)
    wt = og.fusion_weights(sel)
    js = [int(j) for j in idx[0, 0, 0] if j >= 0]
    host64 = lambda x: x.float().double().numpy()
    k = np.concatenate([host64(host["k"][j]) for j in js], axis=2)
    v = np.concatenate([host64(host["v"][j]) for j in js], axis=2)
    loc = np.full_like(idx, -1)
    loc[0, 0, 0, :len(js)] = np.arange(len(js))      # the gathered chunks, in retrieval order
    og.xattn_fwd(host64(host["q"]), k, v, loc, wt, w.S, w.attn_scale, mode="decode")
    sec = time.perf_counter() - t0
    return {"value": total_bytes / sec / 1e9, "unit": "GB/s", "kind": "oracle",
            "sample": "the whole decode call (bf16 landmark keys widened to fp64 included)",
            "sample_seconds": sec, "retrieved_same_set": sorted(js) == host["chunks"], **host_info()}


def bench_decode_host_kv(args, dev, gca):
    """Decode with the past chunks' K/V offloaded to pinned host memory (landmarks,
    q and outputs in HBM): the decode attention gathers the k retrieved chunks over
    the host link.  1M past tokens (16,384 chunks, 2 x 1.07 GB of host K/V)."""
    import torch
    from gen import get_workload, inputs as gi

    w = get_workload("decode_16m_bf16", n_chunks=16384)
    lq, lk = landmarks(w)
    lmk_q, lmk_k = upload(w, lq, dev), upload(w, lk, dev)
    kv = gi.device_kv(w, dev)
    host = {n: torch.empty(kv[n].shape, dtype=kv[n].dtype, pin_memory=True) for n in ("k", "v")}
    for n in ("k", "v"):
        host[n].copy_(kv[n])
    q = gi.device_tensors(w, ("q",), dev)["q"]
    stream = torch.cuda.current_stream()
    res = {}
    for where, flags, k, v in (("device", 0, kv["k"], kv["v"]), ("host", gca.FLAG_HOST_KV, host["k"], host["v"])):
        p = gca.problem(w.B, w.H, w.n_chunks, w.topk, D=w.Dl, Hr=w.Hr, dtype=w.dtype, mode=w.mode, flags=flags)
        fo = forward_outputs(p, gca, dev)
        ws, _ = gca.workspace(p, gca.OP_FORWARD, dev)

        def call():
            gca.forward(p, lmk_q, lmk_k, q, k, v, ws=ws, **fo)

        for _ in range(5):
            call()
        ms = timed(call, args.decode_steps, stream) / args.decode_steps
        _, per = kernel_times(call, args.decode_steps, stream, gca)
        res[where] = {"ms_per_call": ms, "kernels": {n: {"avg_ms": sum(d) / len(d)} for n, d in per.items()}}
    gathered = 2 * w.topk * w.H * S * DH * 2      # K and V tiles of the retrieved chunks, every head
    att_host = res["host"]["kernels"]["xattn_decode_kernel"]["avg_ms"]
    att_dev = res["device"]["kernels"]["xattn_decode_kernel"]["avg_ms"]
    del kv, host
    torch.cuda.empty_cache()
    return {"config": {"workload": "decode with host-resident K/V: B=1 H=8 d=64, 1,048,576 past tokens "
                                   "(16,384 chunks), S=64, top-8, D=512, bf16; K/V in pinned host memory"},
            "ms_per_call": res["host"]["ms_per_call"], "ms_per_call_device_kv": res["device"]["ms_per_call"],
            "host_link_bytes_per_call": gathered,
            "host_link_GBps": gathered / ((att_host - att_dev) * 1e-3) / 1e9 if att_host > att_dev else None,
            "kernels": res["host"]["kernels"], "kernels_device_kv": res["device"]["kernels"]}


# ------------------------------------------------------- CPU baselines ----

def host_info():
    """Threads the oracle's numpy backend uses, the CPU model and the BLAS library."""
    info = {"cores": 1, "cpu_model": None, "blas": None}
    try:
        from threadpoolctl import threadpool_info
        pools = threadpool_info()
        info["cores"] = max([i.get("num_threads", 1) for i in pools] or [1])
        blas = [i for i in pools if i.get("user_api") == "blas"]
        if blas:
            info["blas"] = f"{blas[0].get('internal_api')} {blas[0].get('version')}"
    except Exception:
        pass
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    info["cpu_model"] = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return info


def cpu_baseline(w, t, heads=16):
    """The oracle (as it stands) on a bounded sample: batch 0's scores and top-k over
    all 1,024 landmark rows, then attention forward and backward for `heads` heads of
    batch 0 over every chunk.  Extrapolated to the whole batch in tokens/s."""
    from oracle import gca as og

    def host(x):
        return x.float().cpu().double().numpy()

    lq = host(t["lmk_q"][:1])
    lk = host(t["lmk_k"][:1])
    t0 = time.perf_counter()
    r = og.scores(lq, lk, w.score_scale, w.mode)
    idx, sel = og.topk(r, w.topk)
    wt = og.fusion_weights(sel)
    t_sel = time.perf_counter() - t0
    q = host(t["q"][:1, :heads])
    k = host(t["k"][:1, :heads])
    v = host(t["v"][:1, :heads])
    do = host(t["dout"][:1, :heads])
    t1 = time.perf_counter()
    og.xattn_fwd(q, k, v, idx, wt, w.S, w.attn_scale, w.mode)
    og.xattn_bwd(q, k, v, idx, wt, do, w.S, w.attn_scale, w.mode)
    t_attn = time.perf_counter() - t1
    full = w.B * t_sel + (w.B * w.H / heads) * t_attn
    return {"value": w.B * w.Lq / full, "unit": "tokens/s", "kind": "oracle",
            "sample": f"batch 0: scores+top-k over all {w.n_chunks} landmark rows ({t_sel:.2f}s), then "
                      f"attention fwd+bwd for {heads} of {w.H} heads over all chunks ({t_attn:.2f}s); "
                      f"extrapolated to B={w.B}, H={w.H}",
            "sample_seconds": t_sel + t_attn, **host_info()}


# --------------------------------------------------------------- peaks ----

def measured_peaks(dev):
    """On-device reference rates, each the best over a sweep of launch shapes: a
    streaming read of 4 GiB (the HBM rate a plain coalesced read reaches), gathers
    of random 16 KiB tiles (the rate the attention kernels' L2 misses can reach in
    their access pattern) and a register-resident bf16 32x32x16 product loop (the
    matrix-core rate at the running clock).  The gather is also reported at the
    attention kernels' own concurrency (four workgroups per CU, one 16 KiB tile in
    flight each)."""
    import torch
    path = os.path.join(ROOT, "peaks", "libpeaks.so")
    if not os.path.exists(path):
        return None
    L = ctypes.CDLL(path)
    L.peaks_stream_read.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p]
    L.peaks_mfma_loop.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p]
    L.peaks_tile_gather.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                    ctypes.c_void_p, ctypes.c_void_p]
    cus = torch.cuda.get_device_properties(dev).multi_processor_count
    stream = torch.cuda.current_stream()
    sp = ctypes.c_void_p(stream.cuda_stream)
    nbytes = 4 << 30
    buf = torch.empty(nbytes, dtype=torch.uint8, device=dev)
    buf.fill_(1)
    sink = torch.zeros(16, dtype=torch.float32, device=dev)
    per_cu = (1, 2, 4, 8)                              # 256-thread workgroups per CU

    def rate(run, nread):
        def go():
            assert run() == 0
        for _ in range(3):
            go()
        return nread / (timed(go, 10, stream) / 10 * 1e-3) / 1e9

    read = {}
    for wpc in per_cu:
        read[wpc] = rate(lambda b=cus * wpc: L.peaks_stream_read(
            ctypes.c_void_p(buf.data_ptr()), nbytes // 16, b, ctypes.c_void_p(sink.data_ptr()), sp), nbytes)
    best_read = max(read, key=read.get)
    # random 16 KiB tiles, 4 GiB of reads per call, from a 128 MiB working set (the
    # K/V of the eight (batch, head) slices the XCDs work on at a time at 64K: past
    # the 4 MiB L2s, inside the 256 MiB last-level cache) and from all 4 GiB
    gen = torch.Generator().manual_seed(7)
    gather, gather_shape, gather_at_kernel = {}, {}, {}
    n_reads = nbytes // 16384
    for name, set_bytes in (("128MiB", 128 << 20), ("4GiB", nbytes)):
        idx = torch.randint(0, set_bytes // 16384, (n_reads,), generator=gen, dtype=torch.int32).to(dev)
        got = {}
        for wpc in per_cu:
            for inflight in (1, 2):
                got[(wpc, inflight)] = rate(lambda b=cus * wpc, t=inflight, i=idx: L.peaks_tile_gather(
                    ctypes.c_void_p(buf.data_ptr()), ctypes.c_void_p(i.data_ptr()), n_reads, b, t,
                    ctypes.c_void_p(sink.data_ptr()), sp), n_reads * 16384)
        best = max(got, key=got.get)
        gather[name] = got[best]
        gather_shape[name] = {"workgroups_per_cu": best[0], "tiles_in_flight_per_workgroup": best[1]}
        gather_at_kernel[name] = got[(4, 1)]
        del idx
    del buf
    iters = 20000
    mblocks = cus * 2                                  # 8 waves per CU, two per SIMD

    def mfma():
        assert L.peaks_mfma_loop(mblocks, iters, ctypes.c_void_p(sink.data_ptr()), sp) == 0

    mfma()
    mms = timed(mfma, 5, stream) / 5
    flops = mblocks * 4 * iters * 8 * 32768
    torch.cuda.empty_cache()
    return {"stream_read_GBps": read[best_read], "stream_read_frac_of_spec": read[best_read] / HBM_PEAK_GBS,
            "stream_read_workgroups_per_cu": best_read,
            "tile_gather_GBps": {"working_set_" + k: v for k, v in gather.items()},
            "tile_gather_best_shape": {"working_set_" + k: v for k, v in gather_shape.items()},
            "tile_gather_GBps_at_kernel_concurrency": {"working_set_" + k: v for k, v in gather_at_kernel.items()},
            "mfma_bf16_TFLOPs": flops / (mms * 1e-3) / 1e12,
            "mfma_bf16_frac_of_spec": flops / (mms * 1e-3) / 1e12 / BF16_PEAK_TFLOPS,
            "compute_units": cus, "read_bytes": nbytes}


# ---------------------------------------------------------------- main ----

def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--fwd-steps", type=int, default=50)
    ap.add_argument("--decode-steps", type=int, default=50)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-decode", action="store_true")
    ap.add_argument("--no-host-kv", action="store_true", help="skip the decode leg with host-resident K/V")
    ap.add_argument("--no-forward-legs", action="store_true", help="skip the 16K and 1M forward legs")
    ap.add_argument("--no-peaks", action="store_true")
    ap.add_argument("--no-variants", action="store_true",
                    help="skip the Gumbel and S+1-row variants of the train step (counter runs: only the "
                         "plain step's dispatches)")
    ap.add_argument("--copy-calibration-mb", type=int, default=0,
                    help="first run one plain device copy of this many MiB (a known-size reference for "
                         "rocprofv3 FETCH_SIZE / WRITE_SIZE)")
    ap.add_argument("--only", choices=["train", "decode", "forward_16k", "planted_1m"], default=None,
                    help="run one leg only (for profiling); the JSON line then carries that leg")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: the GCA path here runs on a single MI355X with no "
              "collectives, so --gpus must be 1", file=sys.stderr)
        sys.exit(2)

    import torch
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    from paper_2410_01651_amd import build as _b
    if not os.path.exists(_b.OUT):
        _b.build()
    from paper_2410_01651_amd import gca
    dev = torch.device("cuda:0")
    if args.copy_calibration_mb:
        n = args.copy_calibration_mb << 20
        src = torch.ones(n, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    if args.only:
        args.no_cpu_baseline = True
        if args.only == "decode":
            _, leg, _, _ = bench_decode(args, dev, gca)
            line = {"decode_scan": leg}
        elif args.only == "train":
            tr = bench_train(args, dev, gca)
            line = {"ms_per_step": tr["ms_step"], "step_ms_distribution": tr["latency"],
                    "kernels": tr["kernels"], "roofline": tr["roofline"],
                    "lmk_row": tr["lmk_row"]}
        else:
            name = {"forward_16k": "train_16k_bf16", "planted_1m": "planted_1m_bf16"}[args.only]
            _, leg, _ = bench_forward(args, dev, gca, name)
            line = {args.only: leg}
        print(json.dumps(line), flush=True)
        return

    tr = bench_train(args, dev, gca)
    w = tr["w"]
    line = {
        "metric": "GCA fwd+bwd tokens/s at 64K ctx; retrieval-scan GB/s at 16M-ctx decode",
        "value": tr["tokens"] / (tr["ms_step"] * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": tr["ms_step"], "profiled_ms_per_step": tr["profiled_ms_step"],
        "step_ms_distribution": tr["latency"],
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic",
        "config": {"workload": "fwdbwd_64k_bf16: B=2 H=16 d=64 L=65,536 S=64 (1,024 chunks) top-8 D=1,024, "
                               "bf16 in / fp32 accumulate; forward (scores, top-k, grouped cross attention) + "
                               "backward (dq, dk, dv, dsel, dlmk_q, dlmk_k)",
                   "global_batch": w.B, "seq_len": w.Lq, "parallelism": "none (1 GPU)"},
        "roofline": tr["roofline"],
        "path_algorithmic_tflops": tr["path_tflops"],
        "gumbel_topk": tr["gumbel"],
        "lmk_row": tr["lmk_row"],
        "kernels": tr["kernels"],
    }
    # the GPU legs first, the host oracle last: a host-K/V decode leg measured
    # after the oracle's host-memory churn and the 16M decode leg ran 20x slower
    # per call with unchanged kernel times (a host-side stall, not the library's)
    baselines = []
    if not args.no_cpu_baseline:
        t_host = {n: tr["t"][n][:1, :16].cpu() if n in ("q", "k", "v", "dout") else tr["t"][n][:1].cpu()
                  for n in ("lmk_q", "lmk_k", "q", "k", "v", "dout")}
        baselines.append(("cpu_baseline", lambda: cpu_baseline(w, t_host)))
    del tr
    torch.cuda.empty_cache()
    if not args.no_forward_legs:
        for key, name, sample in (("forward_16k", "train_16k_bf16", dict(rows=None, chunks=None)),
                                  ("planted_1m", "planted_1m_bf16",
                                   dict(rows=list(range(16384 - 512, 16384)), chunks=list(range(2, 16384, 16))))):
            log(f"{key} forward")
            wf, leg, host = bench_forward(args, dev, gca, name)
            line[key] = leg
            if host is not None:
                baselines.append((key, lambda wf=wf, host=host, sample=sample: cpu_forward_baseline(wf, host,
                                                                                                  **sample)))
    if not args.no_decode:
        log("decode scan at 16M context")
        wd, leg, host, nbytes = bench_decode(args, dev, gca)
        line["decode_scan"] = leg
        if host is not None:
            baselines.append(("decode_scan", lambda: cpu_decode_baseline(wd, host, nbytes)))
        if not args.no_host_kv:
            log("decode with host-resident K/V at 1M context")
            line["decode_host_kv"] = bench_decode_host_kv(args, dev, gca)
    if not args.no_peaks:
        log("on-device reference rates")
        line["peaks_measured"] = pk = measured_peaks(dev)
        if pk is not None:
            # the attention kernels' traffic rate against the measured tile-gather rate
            gat = pk["tile_gather_GBps"]["working_set_128MiB"]
            gat_k = pk["tile_gather_GBps_at_kernel_concurrency"]["working_set_128MiB"]
            for roof in [line["roofline"]] + [line[k]["roofline"] for k in ("forward_16k", "planted_1m")
                                              if k in line]:
                if roof.get("traffic_GBps") is not None:
                    roof["traffic_frac_of_measured_gather"] = roof["traffic_GBps"] / gat
                    roof["traffic_frac_of_gather_at_kernel_concurrency"] = roof["traffic_GBps"] / gat_k
    for key, fn in baselines:
        log(f"cpu baseline ({key})")
        if key == "cpu_baseline":
            line["cpu_baseline"] = fn()
        else:
            line[key]["cpu_baseline"] = fn()
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
