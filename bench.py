#!/usr/bin/env python3
"""Benchmark of the pair-biased gated attention layer on one MI355X.

One step = one full layer call (q/k/v/g projection, the fused LayerNorm-bias
attention over all key blocks, the block merge) for every query stripe of the
workload, with all inputs already resident in HBM. Default workload: the
whole-assembly case, N = 24000 tokens (60 x 400), bf16 z[N, N, 128] = 147 GB,
16 heads of width 24, 6 key blocks, last 480 tokens masked.

With an atom workload (--workload atoms96k_bf16) it measures the sparse kNN
pair-biased atom attention instead: one step = one layer call (atom
projections, then the sparse attention over all key blocks) for the query
stripe.

Prints ONE JSON line on stdout; progress goes to stderr.
"""
import argparse
import ctypes
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "ms/layer + achieved HBM GB/s (% peak) for pair-biased attention at N tokens"
PEAK_HBM_GBPS = 8000.0  # MI355X HBM3E, published
KERNEL_SOURCES = ("paper_2607_05439_amd/csrc/fast.hip", "paper_2607_05439_amd/csrc/cdna4.h")
SPARSE_SOURCES = ("paper_2607_05439_amd/csrc/sparse.hip", "paper_2607_05439_amd/csrc/cdna4.h")
SPARSE_METRIC = "ms/layer + gathered GB/s for sparse kNN pair-biased atom attention"
KNN_SOURCES = ("paper_2607_05439_amd/csrc/knn.hip",)
KNN_METRIC = "ms per kNN search + candidate pairs/s for the chunked k-nearest-neighbour top-k"
PEAK_FP32_TFLOPS = 157.3  # MI355X fp32 vector, published
PEAK_BF16_TFLOPS = 2500.0  # MI355X dense bf16 matrix cores, published
TRANS_SOURCES = ("paper_2607_05439_amd/csrc/transition.hip", "paper_2607_05439_amd/csrc/cdna4.h")
TRANS_METRIC = "ms per pair transition (LayerNorm + SwiGLU + residual) + matrix-core TFLOP/s"
SCATTER_SOURCES = ("paper_2607_05439_amd/csrc/scatter.hip",)
SCATTER_METRIC = "us per deterministic atom-to-token mean + achieved HBM GB/s"


def progress(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


class Hip:
    """hipEvent helpers (timing on the library's launch stream)."""

    def __init__(self):
        self.lib = ctypes.CDLL("libamdhip64.so")
        self.lib.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self.lib.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
        self.lib.hipEventSynchronize.argtypes = [ctypes.c_void_p]
        self.lib.hipEventDestroy.argtypes = [ctypes.c_void_p]

    def event(self):
        ev = ctypes.c_void_p()
        assert self.lib.hipEventCreate(ctypes.byref(ev)) == 0
        return ev.value

    def elapsed_ms(self, a, b):
        assert self.lib.hipEventSynchronize(b) == 0
        ms = ctypes.c_float()
        assert self.lib.hipEventElapsedTime(ctypes.byref(ms), a, b) == 0
        return ms.value

    def record(self, ev, stream):
        assert self.lib.hipEventRecord(ctypes.c_void_p(ev), ctypes.c_void_p(stream)) == 0

    def destroy(self, ev):
        self.lib.hipEventDestroy(ev)


def kernel_source_sha(sources=KERNEL_SOURCES):
    """Hash of the kernel's sources and of the compiler flags each .hip among
    them is built with (a flag changes the code as much as an edit does)."""
    from paper_2607_05439_amd import build as dcp_build
    h = hashlib.sha256()
    for p in sources:
        with open(os.path.join(ROOT, p), "rb") as f:
            h.update(f.read())
        if p.endswith(".hip"):
            name = os.path.basename(p)
            h.update(" ".join([*dcp_build.FLAGS, *dcp_build.EXTRA.get(name, [])]).replace(ROOT, "").encode())
    return h.hexdigest()[:16]


def stored_traffic(workload, sources=KERNEL_SOURCES):
    """HBM bytes per launch from committed rocprofv3 counters, if they were
    taken on the current kernel source; else None."""
    path = os.path.join(ROOT, "profiles", f"traffic_attn_{workload}.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        t = json.load(f)
    if t.get("kernel_source_sha") != kernel_source_sha(sources):
        return None
    return t.get("hbm_bytes_per_launch")


def cpu_baseline(wl, s_host, w_host, mask, seconds):
    """The fp64 oracle, as it stands, on a bounded sample of query rows;
    extrapolated to the whole layer (fixed projection cost + N x per-row)."""
    import numpy as np
    import oracle
    import synth
    threads = ctypes.CDLL("libgomp.so.1").omp_get_max_threads()
    s64 = oracle.decode(s_host)
    t0 = time.perf_counter()
    oracle.linear(s64, w_host["w_k"])
    oracle.linear(s64, w_host["w_v"])
    t_fixed = time.perf_counter() - t0
    # first a small batch to size the sample, then the sample itself
    rows = list(range(0, wl.n_tok, max(1, wl.n_tok // threads)))[:threads]
    z = synth.z_host(wl, rows)
    t0 = time.perf_counter()
    oracle.attention(s_host, z, rows, mask, w_host, wl.n_heads, wl.head_dim)
    t_small = time.perf_counter() - t0
    per_row = max((t_small - t_fixed) / len(rows), 1e-9)
    n_rows = int(min(wl.n_tok, max(len(rows), (seconds - t_small) / per_row)))
    n_rows = max(threads, n_rows // threads * threads)
    rng = np.random.default_rng(1)
    rows = sorted(int(x) for x in rng.choice(wl.n_tok, size=min(n_rows, wl.n_tok), replace=False))
    z = synth.z_host(wl, rows)
    t0 = time.perf_counter()
    ref = oracle.attention(s_host, z, rows, mask, w_host, wl.n_heads, wl.head_dim)
    t_run = time.perf_counter() - t0
    per_row = (t_run - t_fixed) / len(rows)
    n_q_total = sum(nq for _, nq in wl.stripes)
    t_layer = t_fixed * len(wl.stripes) + per_row * n_q_total
    # the same oracle on one host thread, over a few of the sampled rows
    gomp = ctypes.CDLL("libgomp.so.1")
    gomp.omp_set_num_threads(1)
    try:
        t0 = time.perf_counter()
        oracle.linear(s64, w_host["w_k"])
        oracle.linear(s64, w_host["w_v"])
        t_fixed1 = time.perf_counter() - t0
        rows1 = rows[:: max(1, len(rows) // 8)][:8]
        z1 = synth.z_host(wl, rows1)
        t0 = time.perf_counter()
        oracle.attention(s_host, z1, rows1, mask, w_host, wl.n_heads, wl.head_dim)
        t_run1 = time.perf_counter() - t0
    finally:
        gomp.omp_set_num_threads(threads)
    per_row1 = max(t_run1 - t_fixed1, 1e-9) / len(rows1)
    t_layer1 = t_fixed1 * len(wl.stripes) + per_row1 * n_q_total
    return {"t_layer_s": t_layer, "rows": len(rows), "t_run_s": t_run, "threads": threads, "t_fixed_s": t_fixed,
            "t_layer_1thread_s": t_layer1, "rows_1thread": len(rows1), "row_ids": rows, "ref": ref}


def host_cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def sparse_cpu_baseline(wl, a_host, w_host, nbr_host, seconds):
    """The fp64 oracle on a bounded sample of query atoms, extrapolated to the
    stripe (fixed K/V projection of all atoms + n_q x per-row)."""
    import numpy as np
    import oracle
    import synth
    threads = ctypes.CDLL("libgomp.so.1").omp_get_max_threads()
    a64 = oracle.decode(a_host) if a_host.dtype == np.uint16 else a_host.astype(np.float64)
    t0 = time.perf_counter()
    oracle.linear(a64, w_host["w_k"])
    oracle.linear(a64, w_host["w_v"])
    t_fixed = time.perf_counter() - t0
    n = min(wl.n_q, 64 * threads)
    rows = np.arange(n) * (wl.n_q // n)
    p = synth.p_gathered_host(wl, wl.q_row0 + rows, nbr_host[rows])
    t0 = time.perf_counter()
    oracle.sparse_attention(a_host, p, nbr_host[rows], wl.q_row0 + rows, w_host, wl.n_heads, wl.head_dim,
                            n_blocks=wl.n_key_blocks)
    t_small = time.perf_counter() - t0
    per_row = max((t_small - t_fixed) / n, 1e-9)
    n_rows = int(min(wl.n_q, max(n, (seconds - t_small) / per_row)))
    rng = np.random.default_rng(1)
    rows = np.sort(rng.choice(wl.n_q, size=n_rows, replace=False))
    p = synth.p_gathered_host(wl, wl.q_row0 + rows, nbr_host[rows])
    t0 = time.perf_counter()
    ref = oracle.sparse_attention(a_host, p, nbr_host[rows], wl.q_row0 + rows, w_host, wl.n_heads, wl.head_dim,
                                  n_blocks=wl.n_key_blocks)
    t_run = time.perf_counter() - t0
    per_row = max((t_run - t_fixed) / n_rows, 1e-12)
    # the same oracle on one host thread, over a few hundred of the sampled rows
    gomp = ctypes.CDLL("libgomp.so.1")
    gomp.omp_set_num_threads(1)
    try:
        rows1 = rows[:: max(1, len(rows) // 256)][:256]
        p1 = synth.p_gathered_host(wl, wl.q_row0 + rows1, nbr_host[rows1])
        t0 = time.perf_counter()
        oracle.linear(a64, w_host["w_k"])
        oracle.linear(a64, w_host["w_v"])
        t_fixed1 = time.perf_counter() - t0
        t0 = time.perf_counter()
        oracle.sparse_attention(a_host, p1, nbr_host[rows1], wl.q_row0 + rows1, w_host, wl.n_heads, wl.head_dim,
                                n_blocks=wl.n_key_blocks)
        t_run1 = time.perf_counter() - t0
    finally:
        gomp.omp_set_num_threads(threads)
    per_row1 = max(t_run1 - t_fixed1, 1e-9) / len(rows1)
    return {"t_layer_s": t_fixed + per_row * wl.n_q, "rows": n_rows, "t_run_s": t_run, "threads": threads,
            "t_fixed_s": t_fixed, "t_layer_1thread_s": t_fixed1 + per_row1 * wl.n_q, "rows_1thread": len(rows1),
            "row_ids": rows, "ref": ref}


def sparse_main(args, wl):
    import numpy as np
    import torch
    import paper_2607_05439_amd as dcp
    import synth

    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()
    sp = stream.cuda_stream
    L, eb, hd = wl.n_atoms, wl.elem_bytes, wl.n_heads * wl.head_dim
    progress(f"workload {wl.name}: L={L} atoms, query rows {wl.q_row0}..{wl.q_row0 + wl.n_q - 1}, k={wl.k}, "
             f"n_kb={wl.n_key_blocks}, P rows {wl.n_q * L * wl.c_ap * eb / 1e9:.1f} GB")

    def to_dev(x):
        if x.dtype == np.uint16:
            return torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).view(torch.bfloat16).to(dev)
        return torch.from_numpy(np.ascontiguousarray(x)).to(dev)

    a_host = synth.a_host(wl)
    w_host = synth.atom_weights(wl)
    nbr_host = synth.neighbours(wl, wl.q_row0, wl.n_q)
    a = to_dev(a_host)
    w = {k: (None if v is None else torch.from_numpy(v).to(dev)) for k, v in w_host.items()}
    nbr = torch.from_numpy(nbr_host).to(dev)
    p = torch.empty((wl.n_q, L, wl.c_ap), dtype=torch.bfloat16 if wl.bf16 else torch.float32, device=dev)
    synth.p_fill_device(wl, p.data_ptr(), wl.q_row0, wl.n_q, sp)
    gathered_form = args.p_form == "gathered"
    if gathered_form:
        # the paper's low-memory form: P_sparse[r, t, :] = P[q_row0 + r, nbr[r, t], :], gathered once by the
        # caller (a torch index copy, outside the timed region); the dense rows are then freed
        idx = nbr.clamp(0, L - 1).long()[:, :, None].expand(-1, -1, wl.c_ap)
        p = torch.gather(p, 1, idx).contiguous()
        del idx
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
    out_dtype = dcp.DCP_BF16 if wl.bf16 else dcp.DCP_F32
    shape = dcp.make_sparse_shape(L, wl.c_atom, wl.c_ap, wl.n_heads, wl.head_dim, wl.k,
                                  dcp.DCP_BF16 if wl.bf16 else dcp.DCP_F32, out_dtype, 1 if gathered_form else 0,
                                  1e-5)
    weights = dcp.make_weights(w["w_q"], w["w_k"], w["w_v"], w["w_g"], w["w_b"])
    ws_bytes = dcp.dcp_sparse_workspace_size(shape, wl.n_q)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    out = torch.empty((wl.n_q, hd), dtype=torch.bfloat16 if wl.bf16 else torch.float32, device=dev)
    valid = (nbr_host >= 0) & (nbr_host < L)
    n_slots = int(valid.sum())
    n_ref = int(np.unique(nbr_host[valid]).size)
    # bytes the kernel moves per valid slot: the pair slice, the K row and the V row
    gathered = n_slots * (wl.c_ap * eb + 2 * hd * eb)
    # bytes that must come from HBM at least once: pair slices, neighbour lists,
    # K/V rows of the referenced atoms, q and g, the output
    compulsory = (n_slots * wl.c_ap * eb + nbr_host.size * 4 + n_ref * 2 * hd * eb + wl.n_q * hd * 4 * 2
                  + wl.n_q * hd * (2 if wl.bf16 else 4))
    torch.cuda.synchronize()
    hip = Hip()

    def step(evs=None):
        if evs is not None:
            dcp.dcp_set_timing_events(*evs)
        dcp.dcp_sparse_pair_bias_attention(shape, weights, a, p, nbr, wl.q_row0, wl.n_q, wl.n_key_blocks, out, ws,
                                           ws_bytes, sp)
        if evs is not None:
            dcp.dcp_set_timing_events(None, None)

    # calibration (outside the timed region): a plain copy of known size for
    # counter scaling
    cal = min(args.calibrate_bytes, p.numel() * p.element_size() // 2 // 16 * 16)
    scratch = torch.empty(cal, dtype=torch.uint8, device=dev)
    synth.device_copy(p.data_ptr(), scratch.data_ptr(), cal, sp)
    torch.cuda.synchronize()
    del scratch
    # ceiling of the K/V gather pattern (same neighbour lists, no arithmetic)
    kbuf = torch.zeros((L, hd), dtype=torch.bfloat16 if wl.bf16 else torch.float32, device=dev)
    vbuf = torch.zeros_like(kbuf)
    sink = torch.zeros(4, dtype=torch.int32, device=dev)
    e0, e1 = hip.event(), hip.event()
    synth.device_gather_pattern(kbuf.data_ptr(), vbuf.data_ptr(), L, nbr.data_ptr(), wl.n_q, wl.k, sink.data_ptr(), sp)
    hip.record(e0, sp)
    synth.device_gather_pattern(kbuf.data_ptr(), vbuf.data_ptr(), L, nbr.data_ptr(), wl.n_q, wl.k, sink.data_ptr(), sp)
    hip.record(e1, sp)
    pattern_ms = hip.elapsed_ms(e0, e1)
    pattern_gbps = n_slots * 2 * hd * eb / (pattern_ms * 1e-3) / 1e9
    del kbuf, vbuf
    progress(f"K/V gather pattern, no arithmetic: {pattern_ms * 1e3:.1f} us, {pattern_gbps:.0f} GB/s")

    progress(f"warmup {args.warmup} steps")
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    kernel_evs = [(hip.event(), hip.event()) for _ in range(args.steps)]
    progress(f"timing {args.steps} steps")
    t_start, t_stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t_start.record(stream)
    for k in range(args.steps):
        step(kernel_evs[k])
    t_stop.record(stream)
    torch.cuda.synchronize()
    ms_per_step = t_start.elapsed_time(t_stop) / args.steps
    k_ms = [hip.elapsed_ms(x, y) for (x, y) in kernel_evs]
    avg_kernel_ms = sum(k_ms) / len(k_ms)
    achieved = compulsory / (avg_kernel_ms * 1e-3) / 1e9
    gathered_gbps = gathered / (avg_kernel_ms * 1e-3) / 1e9
    kv_gbps = n_slots * 2 * hd * eb / (avg_kernel_ms * 1e-3) / 1e9
    value = gathered / (ms_per_step * 1e-3) / 1e9
    progress(f"{ms_per_step * 1e3:.1f} us/layer, sparse attention kernel {avg_kernel_ms * 1e3:.1f} us/launch: "
             f"{gathered_gbps:.0f} GB/s gathered, K/V {kv_gbps:.0f} GB/s ({kv_gbps / pattern_gbps:.1%} of the "
             f"pattern ceiling), compulsory HBM {achieved:.0f} GB/s")

    cpu = None
    err = None
    if not args.no_cpu_baseline:
        progress(f"cpu baseline: oracle on sampled query atoms (~{args.cpu_seconds:.0f} s)")
        cb = sparse_cpu_baseline(wl, a_host, w_host, nbr_host, args.cpu_seconds)
        cpu = {"value": round(gathered / cb["t_layer_s"] / 1e9, 6), "unit": "GB/s", "cores": cb["threads"],
               "kind": "oracle",
               "sample": f"{cb['rows']} of {wl.n_q} query atoms in {cb['t_run_s']:.1f} s (fp64, includes the k/v "
                         f"projection of all {L} atoms, {cb['t_fixed_s']:.1f} s); extrapolated layer time "
                         f"{cb['t_layer_s']:.2f} s",
               "ms_per_layer_extrapolated": round(cb["t_layer_s"] * 1e3, 1),
               "host": {"cpu_model": host_cpu_model(), "logical_cpus": os.cpu_count(),
                        "omp_max_threads": cb["threads"]},
               "one_thread": {"value": round(gathered / cb["t_layer_1thread_s"] / 1e9, 6), "unit": "GB/s",
                              "sample": f"{cb['rows_1thread']} of the sampled rows on one host thread",
                              "ms_per_layer_extrapolated": round(cb["t_layer_1thread_s"] * 1e3, 1)}}
        got = out.float().cpu().numpy()[cb["row_ids"]].astype(np.float64)
        den = float(np.max(np.abs(cb["ref"])))
        e = float(np.max(np.abs(got - cb["ref"]))) / (den if den > 0 else 1.0)
        err = {"max_rel_err": float(f"{e:.4g}"), "rows": cb["rows"], "tolerance": 1e-2 if wl.bf16 else 1e-5,
               "definition": "max|out_gpu - out_oracle| / max|out_oracle| over the sampled query atoms, "
                             "output of the last timed step"}
        progress(f"max rel err on {cb['rows']} sampled query atoms: {e:.3e}")

    line = {
        "metric": SPARSE_METRIC,
        "value": round(value, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if wl.bf16 else "f32",
        "data": "synthetic (seeded; kNN-budget neighbour lists stand in for RFD3 atom neighbourhoods)",
        "config": {"workload": wl.name, "p_form": args.p_form, "n_atoms": L, "q_row0": wl.q_row0, "n_q": wl.n_q,
                   "k": wl.k,
                   "valid_slots": n_slots, "c_atom": wl.c_atom, "c_ap": wl.c_ap, "n_heads": wl.n_heads,
                   "head_dim": wl.head_dim, "n_key_blocks": wl.n_key_blocks,
                   "gathered_bytes_per_step": gathered, "compulsory_bytes_per_step": compulsory},
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBPS, "unit": "GB/s",
                     "frac": round(achieved / PEAK_HBM_GBPS, 4),
                     "traffic": stored_traffic(wl.name + ("_gathered" if gathered_form else ""), SPARSE_SOURCES),
                     "kernel": "sparse_attn_kernel", "kernel_ms": round(avg_kernel_ms, 5),
                     "algorithmic_bytes_per_launch": compulsory},
        "gather": {"gathered_GBps": round(gathered_gbps, 1), "kv_GBps": round(kv_gbps, 1),
                   "kv_pattern_ceiling_GBps": round(pattern_gbps, 1),
                   "frac_of_pattern": round(kv_gbps / pattern_gbps, 4)},
        "max_rel_err": err,
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)


def knn_main(args, wl):
    import numpy as np
    import torch
    import paper_2607_05439_amd as dcp
    import oracle
    import synth

    dev = torch.device("cuda:0")
    sp = torch.cuda.current_stream().cuda_stream
    L, k, n_q = wl.n_atoms, wl.k, wl.n_q
    progress(f"workload {wl.name}: L={L} atoms, query atoms {wl.q_row0}..{wl.q_row0 + n_q - 1}, k={k}")
    x_host = synth.coords(wl)
    x = torch.from_numpy(x_host).to(dev)
    xq = x[wl.q_row0:wl.q_row0 + n_q]
    idx = torch.empty((n_q, k), dtype=torch.int32, device=dev)
    d2 = torch.empty((n_q, k), dtype=torch.float32, device=dev)
    pairs = n_q * L
    ws_bytes = dcp.dcp_knn_workspace_size(L)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    hip = Hip()

    def step(evs=None):
        if evs is not None:
            dcp.dcp_set_timing_events(*evs)
        dcp.dcp_knn_topk(xq, n_q, x, L, 0, wl.q_row0, None, None, 0, k, idx, d2, ws, ws_bytes, sp)
        if evs is not None:
            dcp.dcp_set_timing_events(None, None)

    # calibration for counter scaling: a plain copy of known size
    cal = 1 << 28
    src = torch.empty(cal, dtype=torch.uint8, device=dev)
    dst = torch.empty(cal, dtype=torch.uint8, device=dev)
    synth.device_copy(src.data_ptr(), dst.data_ptr(), cal, sp)
    torch.cuda.synchronize()
    del src, dst
    progress(f"warmup {args.warmup} steps")
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    evs = [(hip.event(), hip.event()) for _ in range(args.steps)]
    t_start, t_stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    progress(f"timing {args.steps} steps")
    t_start.record()
    for i in range(args.steps):
        step(evs[i])
    t_stop.record()
    torch.cuda.synchronize()
    ms_per_step = t_start.elapsed_time(t_stop) / args.steps
    kms = sum(hip.elapsed_ms(a, b) for a, b in evs) / len(evs)
    flops = 8.0 * pairs  # 3 subtractions, 3 products, 2 sums per candidate pair
    achieved = flops / (kms * 1e-3) / 1e12
    value = pairs / (ms_per_step * 1e-3) / 1e9
    progress(f"{ms_per_step:.3f} ms per search, kernel {kms:.3f} ms: {pairs / (kms * 1e-3) / 1e9:.1f} Gpair/s, "
             f"{achieved:.1f} TFLOP/s of distance arithmetic")

    cpu = None
    if not args.no_cpu_baseline:
        progress(f"cpu baseline: oracle on sampled query atoms (~{args.cpu_seconds:.0f} s)")
        threads = ctypes.CDLL("libgomp.so.1").omp_get_max_threads()
        rows = np.arange(0, n_q, max(1, n_q // (4 * threads)))
        t0 = time.perf_counter()
        oracle.knn(x_host[wl.q_row0 + rows], x_host, k)
        per_row = (time.perf_counter() - t0) / len(rows)
        n_rows = int(min(n_q, max(len(rows), args.cpu_seconds / per_row)))
        rows = np.sort(np.random.default_rng(1).choice(n_q, n_rows, replace=False))
        t0 = time.perf_counter()
        oracle.knn(x_host[wl.q_row0 + rows], x_host, k)
        t_run = time.perf_counter() - t0
        t_full = t_run / n_rows * n_q
        cpu = {"value": round(pairs / t_full / 1e9, 6), "unit": "Gpair/s", "cores": threads, "kind": "oracle",
               "sample": f"{n_rows} of {n_q} query atoms in {t_run:.1f} s (brute force + sort per row); "
                         f"extrapolated search time {t_full:.1f} s",
               "ms_per_search_extrapolated": round(t_full * 1e3, 1)}
    line = {
        "metric": KNN_METRIC,
        "value": round(value, 2),
        "unit": "Gpair/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic (seeded chains of residues placed on a sphere; stands in for RFD3 assembly coordinates)",
        "config": {"workload": wl.name, "n_atoms": L, "q_row0": wl.q_row0, "n_q": n_q, "k": k,
                   "candidate_pairs": pairs, "calibration_bytes": cal},
        "roofline": {"bound": "alu", "achieved": round(achieved, 2), "peak": PEAK_FP32_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(achieved / PEAK_FP32_TFLOPS, 4),
                     "traffic": stored_traffic(wl.name, KNN_SOURCES), "kernel": "knn_kernel",
                     "kernel_ms": round(kms, 4), "algorithmic_flops_per_launch": flops},
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)


def transition_main(args, name):
    import numpy as np
    import torch
    import paper_2607_05439_amd as dcp
    import oracle
    import synth

    wl, hidden = synth.transition_workload(name)
    dev = torch.device("cuda:0")
    sp = torch.cuda.current_stream().cuda_stream
    n, c_z = wl.n_tok, wl.c_z
    n_pairs = n * n
    progress(f"workload {name}: z[{n}, {n}, {c_z}] {wl.dtype} in place ({n_pairs * c_z * wl.elem_bytes / 1e9:.1f} GB), "
             f"hidden {hidden}")
    dtype = dcp.DCP_BF16 if wl.bf16 else dcp.DCP_F32
    z = torch.empty((n, n, c_z), dtype=torch.bfloat16 if wl.bf16 else torch.float32, device=dev)
    synth.z_fill_device(wl, z.data_ptr(), 0, n, sp)
    w_host = synth.transition_weights(wl, hidden)
    w = {k: (None if v is None else torch.from_numpy(v).to(dev)) for k, v in w_host.items()}
    ws_bytes = dcp.dcp_transition_workspace_size(c_z, hidden, dtype)
    ws = torch.empty(max(ws_bytes, 256), dtype=torch.uint8, device=dev)
    hip = Hip()

    def step(evs=None):
        if evs is not None:
            dcp.dcp_set_timing_events(*evs)
        dcp.dcp_pair_transition(n_pairs, c_z, hidden, dtype, 1e-5, w["w1"], w["w2"], w["w3"], w["gamma"], w["beta"],
                                z, z, ws, ws.numel(), sp)
        if evs is not None:
            dcp.dcp_set_timing_events(None, None)

    cal = min(args.calibrate_bytes, z.numel() * z.element_size() // 2 // 16 * 16)
    scratch = torch.empty(cal, dtype=torch.uint8, device=dev)
    synth.device_copy(z.data_ptr(), scratch.data_ptr(), cal, sp)
    torch.cuda.synchronize()
    del scratch
    progress(f"warmup {args.warmup} steps")
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    evs = [(hip.event(), hip.event()) for _ in range(args.steps)]
    t_start, t_stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    progress(f"timing {args.steps} steps")
    t_start.record()
    for i in range(args.steps):
        step(evs[i])
    t_stop.record()
    torch.cuda.synchronize()
    ms_per_step = t_start.elapsed_time(t_stop) / args.steps
    kms = sum(hip.elapsed_ms(a, b) for a, b in evs) / len(evs)
    flops = 6.0 * c_z * hidden * n_pairs  # W1, W2 (2 c_z hidden each) and W3 (2 hidden c_z) per pair
    hbm = 2.0 * n_pairs * c_z * wl.elem_bytes  # z read once, written once
    achieved = flops / (kms * 1e-3) / 1e12
    progress(f"{ms_per_step:.2f} ms per transition (weights + kernel {kms:.2f} ms): {achieved:.0f} TFLOP/s "
             f"({achieved / PEAK_BF16_TFLOPS:.1%} of dense bf16), z stream {hbm / (kms * 1e-3) / 1e9:.0f} GB/s")

    cpu = None
    if not args.no_cpu_baseline:
        progress(f"cpu baseline: oracle on sampled pairs (~{args.cpu_seconds:.0f} s)")
        threads = ctypes.CDLL("libgomp.so.1").omp_get_max_threads()
        zs = synth.z_host(wl, [0, n // 2])[:, :, :].reshape(-1, c_z)
        m = min(len(zs), 64 * threads)
        t0 = time.perf_counter()
        oracle.transition(zs[:m], w_host["w1"], w_host["w2"], w_host["w3"])
        per_pair = (time.perf_counter() - t0) / m
        m = int(min(len(zs), max(m, args.cpu_seconds / per_pair)))
        t0 = time.perf_counter()
        oracle.transition(zs[:m], w_host["w1"], w_host["w2"], w_host["w3"])
        t_run = time.perf_counter() - t0
        t_full = t_run / m * n_pairs
        cpu = {"value": round(flops / t_full / 1e12, 6), "unit": "TFLOP/s", "cores": threads, "kind": "oracle",
               "sample": f"{m} of {n_pairs} pairs in {t_run:.1f} s (fp64); extrapolated transition time "
                         f"{t_full:.0f} s",
               "ms_per_transition_extrapolated": round(t_full * 1e3, 1)}
    line = {
        "metric": TRANS_METRIC,
        "value": round(achieved, 1),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if wl.bf16 else "f32",
        "data": "synthetic (seeded; the same pair tensor as the attention workload)",
        "config": {"workload": name, "n_tokens": n, "c_z": c_z, "hidden": hidden, "pairs": n_pairs,
                   "z_bytes": n_pairs * c_z * wl.elem_bytes, "calibration_bytes": cal},
        "roofline": {"bound": "mfma", "achieved": round(achieved, 1), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                     "traffic": stored_traffic(name, TRANS_SOURCES), "kernel": "trans_kernel",
                     "kernel_ms": round(kms, 4), "algorithmic_flops_per_launch": flops,
                     "hbm_GBps": round(hbm / (kms * 1e-3) / 1e9, 1)},
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)


def scatter_main(args, name):
    import numpy as np
    import torch
    import paper_2607_05439_amd as dcp
    import oracle
    import synth

    n_tok, c, dt = synth.SCATTER_WORKLOADS[name]
    dev = torch.device("cuda:0")
    sp = torch.cuda.current_stream().cuda_stream
    idx_host = synth.token_index(n_tok)
    n_atoms = len(idx_host)
    bf16 = dt == "bf16"
    a_host = synth.atom_features(n_atoms, c, bf16)
    progress(f"workload {name}: {n_atoms} atoms -> {n_tok} tokens, {c} channels, {dt} features")
    a = (torch.from_numpy(a_host.view(np.int16)).view(torch.bfloat16) if bf16 else torch.from_numpy(a_host)).to(dev)
    idx = torch.from_numpy(idx_host).to(dev)
    out = torch.empty((n_tok, c), dtype=torch.float32, device=dev)
    ws_bytes = dcp.dcp_scatter_mean_workspace_size(n_tok, c)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    in_dtype = dcp.DCP_BF16 if bf16 else dcp.DCP_F32
    hip = Hip()

    def step(evs=None):
        if evs is not None:
            dcp.dcp_set_timing_events(*evs)
        dcp.dcp_scatter_mean(n_atoms, n_tok, c, in_dtype, dcp.DCP_F32, a, idx, out, ws, ws_bytes, sp)
        if evs is not None:
            dcp.dcp_set_timing_events(None, None)

    cal = 1 << 28
    src = torch.empty(cal, dtype=torch.uint8, device=dev)
    dst = torch.empty(cal, dtype=torch.uint8, device=dev)
    synth.device_copy(src.data_ptr(), dst.data_ptr(), cal, sp)
    torch.cuda.synchronize()
    del src, dst
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    evs = [(hip.event(), hip.event()) for _ in range(args.steps)]
    t_start, t_stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    progress(f"timing {args.steps} steps")
    t_start.record()
    for i in range(args.steps):
        step(evs[i])
    t_stop.record()
    torch.cuda.synchronize()
    ms_per_step = t_start.elapsed_time(t_stop) / args.steps
    kms = sum(hip.elapsed_ms(x, y) for x, y in evs) / len(evs)
    alg = n_atoms * c * a.element_size() + n_atoms * 4 + n_tok * c * 4  # features and indices in, means out
    achieved = alg / (kms * 1e-3) / 1e9
    progress(f"{ms_per_step * 1e3:.1f} us per pooling (kernels {kms * 1e3:.1f} us): {achieved:.0f} GB/s")
    cpu = None
    if not args.no_cpu_baseline:
        t0 = time.perf_counter()
        reps = 0
        while time.perf_counter() - t0 < min(args.cpu_seconds, 10.0):
            oracle.scatter_mean(a_host, idx_host, n_tok)
            reps += 1
        t_one = (time.perf_counter() - t0) / reps
        cpu = {"value": round(alg / t_one / 1e9, 4), "unit": "GB/s", "cores": 1, "kind": "oracle",
               "sample": f"the whole pooling, {reps} repetitions (single-threaded fp64), {t_one * 1e3:.1f} ms each",
               "ms_per_pooling": round(t_one * 1e3, 2)}
    line = {
        "metric": SCATTER_METRIC,
        "value": round(achieved, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": dt,
        "data": "synthetic (seeded; 4-14 atoms per token, ordered by token)",
        "config": {"workload": name, "n_atoms": n_atoms, "n_tokens": n_tok, "c": c, "calibration_bytes": cal,
                   "algorithmic_bytes": alg},
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBPS, "unit": "GB/s",
                     "frac": round(achieved / PEAK_HBM_GBPS, 4), "traffic": stored_traffic(name, SCATTER_SOURCES),
                     "kernel": "pooling (plan + sum; the any-order accumulation and division exit on ordered atoms)", "kernel_ms": round(kms, 5),
                     "algorithmic_bytes_per_launch": alg},
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)


def flops_per_pair(wl):
    """Algorithmic flops per valid (query, key) pair: LayerNorm statistics and
    normalisation (3 c_z), bias projection (2 c_z H), QK^T and PV (4 H d), the
    bias add and the softmax (2 H + 6 H)."""
    return 3 * wl.c_z + 2 * wl.n_heads + 2 * wl.c_z * wl.n_heads + 4 * wl.n_heads * wl.head_dim + 6 * wl.n_heads


class AttentionLayer:
    """Device inputs and buffers of one token-attention workload, and its step."""

    def __init__(self, wl, dev, sp):
        import numpy as np
        import torch
        import paper_2607_05439_amd as dcp
        import synth
        self.wl, self.sp = wl, sp
        n, cz = wl.n_tok, wl.c_z
        zdt = torch.bfloat16 if wl.bf16 else torch.float32
        self.z = torch.empty((n, n, cz), dtype=zdt, device=dev)
        synth.z_fill_device(wl, self.z.data_ptr(), 0, n, sp)
        self.s_host = synth.s_host(wl)
        self.w_host = synth.weights(wl)
        self.mask_host = synth.mask_host(wl)
        if wl.bf16:
            self.s = torch.from_numpy(self.s_host.view(np.int16)).view(torch.bfloat16).to(dev)
        else:
            self.s = torch.from_numpy(self.s_host).to(dev)
        self.w = {k: (None if v is None else torch.from_numpy(v).to(dev)) for k, v in self.w_host.items()}
        self.mask = None if self.mask_host is None else torch.from_numpy(self.mask_host).to(dev)
        out_dtype = dcp.DCP_BF16 if wl.bf16 else dcp.DCP_F32
        act = dcp.DCP_BF16 if wl.bf16 else dcp.DCP_F32
        self.shape = dcp.make_shape(n, wl.c_s, cz, wl.n_heads, wl.head_dim, act, out_dtype, 1e-5)
        w = self.w
        self.weights = dcp.make_weights(w["w_q"], w["w_k"], w["w_v"], w["w_g"], w["w_b"], w["b_b"], w["ln_gamma"],
                                        w["ln_beta"])
        hd = wl.n_heads * wl.head_dim
        self.ws_bytes = max(dcp.dcp_workspace_size(self.shape, nq, wl.n_key_blocks) for _, nq in wl.stripes)
        self.ws = torch.empty(self.ws_bytes, dtype=torch.uint8, device=dev)
        self.outs = [torch.empty((nq, hd), dtype=zdt, device=dev) for _, nq in wl.stripes]
        self.n_valid = n if self.mask_host is None else int(self.mask_host.sum())
        self.bytes_per_launch = [nq * self.n_valid * cz * wl.elem_bytes for _, nq in wl.stripes]
        self.bytes_per_step = sum(self.bytes_per_launch)
        # algorithmic flops: the pairs of every stripe, plus q, g of the query rows and k, v of the keys once
        self.pair_flops_per_launch = [nq * self.n_valid * flops_per_pair(wl) for _, nq in wl.stripes]
        n_q_total = sum(nq for _, nq in wl.stripes)
        self.flops_per_step = (sum(self.pair_flops_per_launch) + 2 * wl.c_s * hd * 2 * (n_q_total + n))

    def step(self, evs=None):
        import paper_2607_05439_amd as dcp
        wl = self.wl
        n, cz = wl.n_tok, wl.c_z
        for i, (q0, nq) in enumerate(wl.stripes):
            if evs is not None:
                dcp.dcp_set_timing_events(*evs[i])
            dcp.dcp_pair_bias_attention(self.shape, self.weights, self.s,
                                        self.z.data_ptr() + q0 * n * cz * wl.elem_bytes, self.mask, q0, nq,
                                        wl.n_key_blocks, self.outs[i], self.ws, self.ws_bytes, self.sp)
        if evs is not None:
            dcp.dcp_set_timing_events(None, None)

    def time(self, hip, stream, steps, warmup):
        """ms per step (torch events around the steps) and the attention
        kernel's time of every launch (HIP events on the library's stream)."""
        import torch
        for _ in range(warmup):
            self.step()
        torch.cuda.synchronize()
        kernel_evs = [[(hip.event(), hip.event()) for _ in self.wl.stripes] for _ in range(steps)]
        t_start, t_stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        t_start.record(stream)
        for k in range(steps):
            self.step(kernel_evs[k])
        t_stop.record(stream)
        torch.cuda.synchronize()
        ms_per_step = t_start.elapsed_time(t_stop) / steps
        k_ms = [hip.elapsed_ms(a, b) for evs in kernel_evs for (a, b) in evs]
        for evs in kernel_evs:
            for a, b in evs:
                hip.destroy(a)
                hip.destroy(b)
        return ms_per_step, k_ms


def launch_stats(k_ms):
    k_sorted = sorted(k_ms)
    return {"median": round(k_sorted[len(k_sorted) // 2], 4), "min": round(k_sorted[0], 4),
            "max": round(k_sorted[-1], 4), "launches": len(k_ms)}


def attention_main(args, wl):
    import numpy as np
    import torch
    import paper_2607_05439_amd as dcp
    import synth

    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()
    sp = stream.cuda_stream
    n, cz = wl.n_tok, wl.c_z
    progress(f"workload {wl.name}: N={n} c_z={cz} H={wl.n_heads} d={wl.head_dim} n_kb={wl.n_key_blocks} "
             f"z={n * n * cz * wl.elem_bytes / 1e9:.1f} GB")
    layer = AttentionLayer(wl, dev, sp)
    z = layer.z
    weights = layer.weights
    torch.cuda.synchronize()
    hip = Hip()

    # calibration kernels (outside the timed region): a plain copy of known size
    # for counter scaling, and a plain streaming read of z for achievable bandwidth
    cal = min(args.calibrate_bytes, z.numel() * z.element_size() // 2 // 16 * 16)
    sink = torch.zeros(4, dtype=torch.int32, device=dev)
    e0, e1 = hip.event(), hip.event()
    scratch = torch.empty(cal, dtype=torch.uint8, device=dev)
    synth.device_copy(z.data_ptr(), scratch.data_ptr(), cal, sp)
    torch.cuda.synchronize()
    del scratch
    read_bytes = z.numel() * z.element_size() // 16 * 16
    synth.device_read(z.data_ptr(), read_bytes, sink.data_ptr(), sp)  # warm
    torch.cuda.synchronize()
    hip.record(e0, sp)
    synth.device_read(z.data_ptr(), read_bytes, sink.data_ptr(), sp)
    hip.record(e1, sp)
    read_gbps = read_bytes / (hip.elapsed_ms(e0, e1) * 1e-3) / 1e9
    # the attention kernel's own z stream over the first stripe (same grid, loads
    # and ring), no arithmetic
    pattern_gbps = pattern_ms = None
    if wl.bf16 and cz == 128:
        q0, nq = wl.stripes[0]
        zp = z.data_ptr() + q0 * n * cz * wl.elem_bytes
        synth.device_read_pattern(zp, n, nq, wl.n_key_blocks, sink.data_ptr(), sp)
        hip.record(e0, sp)
        synth.device_read_pattern(zp, n, nq, wl.n_key_blocks, sink.data_ptr(), sp)
        hip.record(e1, sp)
        pattern_ms = hip.elapsed_ms(e0, e1)
        pattern_gbps = nq * n * cz * wl.elem_bytes / (pattern_ms * 1e-3) / 1e9
    progress(f"streaming read of z: {read_gbps:.0f} GB/s; the attention's z stream, no arithmetic: "
             f"{pattern_gbps or 0:.0f} GB/s")

    progress(f"warmup {args.warmup} steps, timing {args.steps} steps")
    ms_per_step, k_ms = layer.time(hip, stream, args.steps, args.warmup)
    avg_kernel_ms = sum(k_ms) / len(k_ms)
    bytes_per_step = layer.bytes_per_step
    n_valid, bytes_launch0, flops_step = layer.n_valid, layer.bytes_per_launch[0], layer.flops_per_step
    achieved = (bytes_per_step / len(wl.stripes)) / (avg_kernel_ms * 1e-3) / 1e9
    value = bytes_per_step / (ms_per_step * 1e-3) / 1e9
    kernel_tflops = (sum(layer.pair_flops_per_launch) / len(wl.stripes)) / (avg_kernel_ms * 1e-3) / 1e12
    layer_tflops = flops_step / (ms_per_step * 1e-3) / 1e12
    progress(f"{ms_per_step:.3f} ms/layer, attention kernel {avg_kernel_ms:.3f} ms/launch, "
             f"{achieved:.0f} GB/s in the kernel ({achieved / PEAK_HBM_GBPS:.1%} of peak), "
             f"{kernel_tflops:.1f} TFLOP/s in the kernel ({kernel_tflops / PEAK_BF16_TFLOPS:.1%} of bf16 peak)")

    # the materialised bias alone (dcp_bias_project) on a stripe of rows: the z
    # stream with LayerNorm and the c_z -> H projection but no attention, as a
    # pure-stream reference beside the fused kernel (outside the timed region)
    bias_ref = None
    if wl.bf16 and cz == 128:
        nr = min(256, n)
        bout = torch.empty((nr, n, wl.n_heads), dtype=torch.float32, device=dev)
        bsh = dcp.make_shape(n, wl.c_s, cz, wl.n_heads, wl.head_dim, dcp.DCP_BF16, dcp.DCP_F32, 1e-5)
        run_bias = lambda: dcp.dcp_bias_project(bsh, weights, z.data_ptr(), nr, n, n * cz, bout, sp)
        run_bias()
        b_ms = []
        for _ in range(5):
            hip.record(e0, sp)
            run_bias()
            hip.record(e1, sp)
            b_ms.append(hip.elapsed_ms(e0, e1))
        b_med = sorted(b_ms)[len(b_ms) // 2]
        zb = nr * n * cz * wl.elem_bytes
        bias_ref = {"rows": nr, "ms_median": round(b_med, 4), "z_read_GBps": round(zb / (b_med * 1e-3) / 1e9, 1),
                    "read_plus_write_GBps": round((zb + bout.numel() * 4) / (b_med * 1e-3) / 1e9, 1)}
        del bout
        progress(f"dcp_bias_project on {nr} rows: {b_med:.3f} ms, z read at {bias_ref['z_read_GBps']:.0f} GB/s")

    cpu = None
    err = None
    if not args.no_cpu_baseline:
        progress(f"cpu baseline: oracle on sampled rows (~{args.cpu_seconds:.0f} s)")
        cb = cpu_baseline(wl, layer.s_host, layer.w_host, layer.mask_host, args.cpu_seconds)
        cpu = {"value": round(bytes_per_step / cb["t_layer_s"] / 1e9, 6), "unit": "GB/s", "cores": cb["threads"],
               "kind": "oracle",
               "sample": f"{cb['rows']} of {sum(nq for _, nq in wl.stripes)} query rows in {cb['t_run_s']:.1f} s "
                         f"(fp64, includes the k/v projection of all {n} keys, {cb['t_fixed_s']:.1f} s); "
                         f"extrapolated layer time {cb['t_layer_s']:.1f} s",
               "ms_per_layer_extrapolated": round(cb["t_layer_s"] * 1e3, 1),
               "host": {"cpu_model": host_cpu_model(), "logical_cpus": os.cpu_count(),
                        "omp_max_threads": cb["threads"]},
               "one_thread": {"value": round(bytes_per_step / cb["t_layer_1thread_s"] / 1e9, 6), "unit": "GB/s",
                              "sample": f"{cb['rows_1thread']} of the sampled rows on one host thread",
                              "ms_per_layer_extrapolated": round(cb["t_layer_1thread_s"] * 1e3, 1)}}
        # the error of the timed layer's output on the same sampled rows
        got = np.empty_like(cb["ref"])
        for r_i, r in enumerate(cb["row_ids"]):
            for s_i, (q0, nq) in enumerate(wl.stripes):
                if q0 <= r < q0 + nq:
                    got[r_i] = layer.outs[s_i][r - q0].float().cpu().numpy()
                    break
        den = float(np.max(np.abs(cb["ref"])))
        e = float(np.max(np.abs(got - cb["ref"]))) / (den if den > 0 else 1.0)
        err = {"max_rel_err": float(f"{e:.4g}"), "rows": cb["rows"],
               "tolerance": 1e-2 if wl.bf16 else 1e-5,
               "definition": "max|out_gpu - out_oracle| / max|out_oracle| over the sampled query rows, "
                             "output of the last timed step"}
        progress(f"max rel err on {cb['rows']} sampled rows: {e:.3e}")

    # the other attention workloads, each timed after the previous one's tensors are freed
    extras = None
    if not args.no_extra_configs and wl.name == "asm24000_bf16":
        extras = {}
        del z, layer
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
        for name in ("grid12000_bf16", "ico4800_bf16", "pad1024_bf16"):
            xw = synth.WORKLOADS[name]
            progress(f"extra workload {name}")
            xl = AttentionLayer(xw, dev, sp)
            x_ms, x_k = xl.time(hip, stream, args.extra_steps, 3)
            x_avg = sum(x_k) / len(x_k)
            x_gbps = (xl.bytes_per_step / len(xw.stripes)) / (x_avg * 1e-3) / 1e9
            x_tf = (sum(xl.pair_flops_per_launch) / len(xw.stripes)) / (x_avg * 1e-3) / 1e12
            extras[name] = {
                "ms_per_layer": round(x_ms, 4), "layer_GBps": round(xl.bytes_per_step / (x_ms * 1e-3) / 1e9, 1),
                "kernel_ms": round(x_avg, 4), "kernel_launch_ms": launch_stats(x_k),
                "kernel_GBps": round(x_gbps, 1), "frac": round(x_gbps / PEAK_HBM_GBPS, 4),
                "kernel_TFLOPs": round(x_tf, 1), "layer_TFLOPs": round(xl.flops_per_step / (x_ms * 1e-3) / 1e12, 1),
                "per_tile_ms": round(x_avg / xw.n_key_blocks, 4), "n_key_blocks": xw.n_key_blocks,
                "stripes": [list(x) for x in xw.stripes], "algorithmic_bytes_per_step": xl.bytes_per_step,
                "steps": args.extra_steps}
            progress(f"  {x_ms:.3f} ms/layer, kernel {x_avg:.3f} ms/launch, {x_gbps:.0f} GB/s "
                     f"({x_gbps / PEAK_HBM_GBPS:.1%}), {x_tf:.1f} TFLOP/s")
            del xl
            torch.cuda.synchronize()
            torch.cuda.empty_cache()

    traffic = stored_traffic(wl.name)
    line = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if wl.bf16 else "f32",
        "data": "synthetic (seeded; stands in for RFD3 icosahedral-assembly pair tensors)",
        "config": {"workload": wl.name, "n_tokens": n, "valid_keys": n_valid, "c_s": wl.c_s, "c_z": cz,
                   "n_heads": wl.n_heads, "head_dim": wl.head_dim, "n_key_blocks": wl.n_key_blocks,
                   "stripes": [list(x) for x in wl.stripes], "z_bytes": n * n * cz * wl.elem_bytes,
                   "algorithmic_bytes_per_step": bytes_per_step},
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBPS, "unit": "GB/s",
                     "frac": round(achieved / PEAK_HBM_GBPS, 4), "traffic": traffic,
                     "kernel": "attn_kernel", "kernel_ms": round(avg_kernel_ms, 4),
                     "algorithmic_bytes_per_launch": bytes_launch0},
        "tflops": {"kernel": round(kernel_tflops, 1), "layer": round(layer_tflops, 1), "peak": PEAK_BF16_TFLOPS,
                   "kernel_frac_of_bf16_peak": round(kernel_tflops / PEAK_BF16_TFLOPS, 4),
                   "flops_per_valid_pair": flops_per_pair(wl), "flops_per_step": flops_step,
                   "note": "algorithmic flops (pairs x per-pair flops; projections once per token) over HIP-event "
                           "kernel time and the layer's step time; the path is HBM-bound"},
        "max_rel_err": err,
        "attn_launch_ms": launch_stats(k_ms),
        # one launch covers a stripe of query rows against n_key_blocks key blocks:
        # the time of one (stripe, key block) tile of a grid schedule
        "per_tile_ms": round(avg_kernel_ms / wl.n_key_blocks, 4),
        "bias_project_stripe": bias_ref,
        "streaming_read_GBps": round(read_gbps, 1),
        # the kernel's own z stream over the first stripe (same grid, loads and
        # ring, all keys) with no arithmetic, and its time over the kernel's
        "pattern_read_GBps": None if pattern_gbps is None else round(pattern_gbps, 1),
        "pattern_ms": None if pattern_ms is None else round(pattern_ms, 4),
        "pattern_ms_over_kernel_ms": None if pattern_ms is None else round(pattern_ms / avg_kernel_ms, 4),
        "other_configs": extras,
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)

def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="asm24000_bf16")
    ap.add_argument("--cpu-seconds", type=float, default=20.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extra-configs", action="store_true",
                    help="skip timing the smaller attention workloads after the default one")
    ap.add_argument("--extra-steps", type=int, default=20)
    ap.add_argument("--p-form", choices=("dense", "gathered"), default="gathered",
                    help="sparse atom workloads: P as the gathered slices P_sparse[n_q, k, c_ap] (default; the "
                         "paper's sparse form) or as the query stripe's dense rows")
    ap.add_argument("--calibrate-bytes", type=int, default=1 << 31,
                    help="bytes for the plain-copy calibration kernel (counter scaling)")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures a single GPU: the library has no multi-GPU path (no collectives or "
              "sharding across GPUs); run with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    import paper_2607_05439_amd as dcp
    import synth

    if args.workload in synth.ATOM_WORKLOADS:
        return sparse_main(args, synth.ATOM_WORKLOADS[args.workload])
    if args.workload in synth.KNN_WORKLOADS:
        return knn_main(args, synth.KNN_WORKLOADS[args.workload])
    if args.workload in synth.TRANSITION_WORKLOADS:
        return transition_main(args, args.workload)
    if args.workload in synth.SCATTER_WORKLOADS:
        return scatter_main(args, args.workload)
    return attention_main(args, synth.WORKLOADS[args.workload])


if __name__ == "__main__":
    main()
