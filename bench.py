"""Benchmark of KV-PRM verify-token scoring on one MI355X.

One step = one kvprm_score call over the whole hot path (all layers, projections, paged
attention, merge, FFN, reward head) for the ragged long-context batch: the 7B-class shape in
bf16 (28 layers, H=3584, 28/4 heads, d_h=128, FFN 18944), B=8 candidates with cached lengths
L_b ~ U[16384, 32768] on 16-token pages scattered over a pool. Inputs are synthetic (seeded
generator) and resident in HBM before the timed region.

Prints one JSON line: scores/s (value), the end-to-end KV-read rate, the roofline of the
dominant kernel (the split-L attention chunk kernel, timed live with HIP events on its stream;
the whole attention step with its merge is reported beside it), the parity of the timed call's
scores against stored fp64 oracle values (`parity`), the other benchmark workloads measured the
same way (`workloads`: the 7B batch of 16 at L = 4096, the fixed L = 32768 batch of 8, the
64-candidate beam batch with a shared 16k prefix, the large fp8-cache model), the same ragged
workload scored with the base weights and an unmerged rank-256 adapter on every projection
(kvprm_score_lora, `lora_readout`) and with two verify tokens per candidate (the depth-k
readout, kvprm_score_ex, `depth_readout`), KV steering steps on its cache (kvprm_steer,
`kv_steering`), and the fp64 CPU oracle timed on one full call of the same workload.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0  # MI355X HBM3E, published


def _log(msg):
    print(msg, file=sys.stderr, flush=True)


def algorithmic_bytes(w, dw):
    s = w.shape
    kv_bytes = s.num_layers * w.unique_tokens() * 2 * s.num_kv_heads * s.head_dim * s.kv_elem_bytes
    if s.kv_dtype == "fp8":
        kv_bytes += s.num_layers * len(w.used_pages()) * s.num_kv_heads * 2 * 4
    return kv_bytes, dw.weight_bytes()


def time_attention(kv, dw, h, batch, ws, n, reps):
    """Average durations (ms) of one layer's split-L chunk kernel alone (kvprm_attention_partials)
    and of the whole attention step (chunk kernel + merge, kvprm_attention): `reps` back-to-back
    calls each between two HIP events recorded on the stream the kernels are launched on."""
    import torch
    w = dw.w
    s = w.shape
    q = torch.randn(w.batch, s.num_q_heads, s.head_dim, device="cuda")
    ks = torch.randn(w.batch, s.num_kv_heads, s.head_dim, device="cuda")
    vs = torch.randn(w.batch, s.num_kv_heads, s.head_dim, device="cuda")
    o = torch.empty_like(q)
    stream = torch.cuda.current_stream()
    cache = dw.cache(kv)

    def step(layer):
        kv.kvprm_attention(h, cache, batch, layer, q.data_ptr(), ks.data_ptr(), vs.data_ptr(),
                           ws.data_ptr(), n, o.data_ptr(), stream.cuda_stream)

    def partials(layer):
        kv.kvprm_attention_partials(h, cache, batch, layer, q.data_ptr(), ws.data_ptr(), n,
                                    stream.cuda_stream)

    def timed(call):
        for l in range(s.num_layers):
            call(l)
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        for i in range(reps):  # back to back, cycling through the layers' pools
            call(i % s.num_layers)
        b.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(b) / reps

    return timed(partials), timed(step)


def time_graph(kv, h, cache, batch, readout, ws, n, scores, steps):
    """One kvprm_score call captured in a HIP graph (the library enqueues kernels only: no
    allocation, synchronisation or memset), replayed `steps` times between two synchronisations:
    the per-call time a caller that replays captured calls sees."""
    import torch
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())

    def call():
        kv.kvprm_score(h, cache, batch, readout, ws.data_ptr(), n, scores.data_ptr(), 0,
                       torch.cuda.current_stream().cuda_stream)

    with torch.cuda.stream(side):
        call()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        call()
    g.replay()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        g.replay()
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / steps
    del g
    return {"ms_per_call": ms, "scores_per_s": scores.numel() / (ms * 1e-3)}


def time_lora(kv, dw, h, batch, rank, steps, warmup):
    """Whole scoring calls with the base weights and an unmerged adapter of this rank on every
    projection (kvprm_score_lora): the same workload, K calls between two synchronisations."""
    import torch
    import synth
    w = dw.w
    dw.add_lora(rank)
    n = kv.kvprm_workspace_size_lora(h, batch, rank)
    ws = torch.empty(n, dtype=torch.uint8, device="cuda")
    scores = torch.empty(w.batch, dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream()
    cache, base, lora = dw.cache(kv), dw.readout(kv), dw.lora(kv)

    def call():
        kv.kvprm_score_lora(h, cache, batch, base, lora, ws.data_ptr(), n, scores.data_ptr(), 0,
                            stream.cuda_stream)

    for _ in range(warmup):
        call()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        call()
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / steps
    return {"rank": rank, "scale": synth.lora_scale(rank),
            "targets": list(synth.LORA_PROJECTIONS), "ms_per_call": ms,
            "scores_per_s": w.batch / (ms * 1e-3), "adapter_bytes_per_call": dw.lora_bytes()}


def time_depth(kv, dw, h, batch, depth, steps, warmup):
    """Whole scoring calls of the depth-k readout (kvprm_score_ex, `depth` verify tokens per
    candidate, merged weights) on the same workload, K calls between two synchronisations."""
    import torch
    w = dw.w
    opt = kv.make_options(None, depth)
    n = kv.kvprm_workspace_size_ex(h, batch, opt)
    ws = torch.empty(n, dtype=torch.uint8, device="cuda")
    scores = torch.empty(w.batch, dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream()
    cache, ro = dw.cache(kv), dw.readout(kv)

    def call():
        kv.kvprm_score_ex(h, cache, batch, ro, opt, ws.data_ptr(), n, scores.data_ptr(), 0,
                          stream.cuda_stream)

    for _ in range(warmup):
        call()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        call()
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / steps
    return {"depth": depth, "ms_per_call": ms, "scores_per_s": w.batch / (ms * 1e-3),
            "verify_tokens_per_s": w.batch * depth / (ms * 1e-3)}


STEER_ETA = 20.0


def time_steer(kv, dw, h, batch, steps):
    """KV Steering on the workload's cache (kvprm_steer): one call of one step and one call of
    1 + steps steps, each between two synchronisations; a step (forward with the activations
    kept, backward through every layer, in-place update of every cached key and value) costs the
    difference divided by steps. The cache is rewritten. eta = 20: with these random weights the
    gradient is ~1e-6 per cached value, and a step moves a stored bf16 value only where eta |g|
    exceeds half its spacing; much smaller steps change P(+) by less than the scoring pass
    resolves (activations enter the matrix cores with 16 significant bits)."""
    import torch
    w = dw.w
    n = kv.kvprm_workspace_size_grad(h, batch)
    ws = torch.empty(n, dtype=torch.uint8, device="cuda")
    before = torch.empty(w.batch, dtype=torch.float32, device="cuda")
    after = torch.empty(w.batch, dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream()
    cache, ro = dw.cache(kv), dw.readout(kv)

    def call(k):
        kv.kvprm_steer(h, cache, batch, ro, STEER_ETA, k, ws.data_ptr(), n, before.data_ptr(),
                       after.data_ptr(), stream.cuda_stream)

    call(1)  # warm-up
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    call(1)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    call(1 + steps)
    torch.cuda.synchronize()
    t2 = time.perf_counter()
    one, many = (t1 - t0) * 1e3, (t2 - t1) * 1e3
    return {"eta": STEER_ETA, "ms_one_step_call": one, "ms_per_step": (many - one) / steps,
            "p_before": before.cpu().tolist(), "p_after": after.cpu().tolist(),
            "workspace_bytes": n}


def read_bandwidth(kv, nbytes=4 << 30, reps=10):
    """Streaming-read ceiling on this GPU: the library's plain read kernel (kvprm_stream_read:
    the 16-byte non-temporal loads of the cache and weight streams, no arithmetic) over nbytes,
    timed with events on the stream it runs on; the measured ceiling the kernels' HBM fractions
    are set against, beside the 8 TB/s nominal figure."""
    import torch
    a = torch.empty(nbytes // 4, dtype=torch.int32, device="cuda")
    a.fill_(1)
    sink = torch.zeros(1, dtype=torch.int32, device="cuda")
    st = torch.cuda.current_stream()
    kv.kvprm_stream_read(a.data_ptr(), nbytes, sink.data_ptr(), st.cuda_stream)
    torch.cuda.synchronize()
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    s.record(st)
    for _ in range(reps):
        kv.kvprm_stream_read(a.data_ptr(), nbytes, sink.data_ptr(), st.cuda_stream)
    e.record(st)
    torch.cuda.synchronize()
    ms = s.elapsed_time(e) / reps
    del a
    return nbytes / (ms * 1e-3) / 1e9


def copy_bandwidth(nbytes=4 << 30, reps=10):
    """Streaming reference on this GPU: a device-to-device copy of nbytes (read + write bytes
    counted), timed with events; context for the HBM fraction, not a kernel of the path."""
    import torch
    a = torch.empty(nbytes // 4, dtype=torch.float32, device="cuda")
    b = torch.empty_like(a)
    a.fill_(1.0)
    b.copy_(a)
    torch.cuda.synchronize()
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    s.record()
    for _ in range(reps):
        b.copy_(a)
    e.record()
    torch.cuda.synchronize()
    ms = s.elapsed_time(e) / reps
    del a, b
    return 2 * nbytes / (ms * 1e-3) / 1e9


def cpu_baseline(w):
    """The fp64 oracle as it stands (kvprm_oracle.verify_pass, untuned) on one whole call of the
    workload: every candidate through every layer. Its inputs are generated lazily inside the
    call (one layer of weights and the pages it reads at a time, so that host memory stays
    bounded); the time spent in the generator is measured around each generator call and
    subtracted, so the figure is the oracle's own arithmetic. numpy's BLAS runs the projections
    on its threads; the per-candidate, per-head attention loop runs on one thread. Returns the
    baseline record and the oracle's (z, P(+)) of every candidate."""
    from threadpoolctl import threadpool_info

    from oracle import inputs as oin
    from oracle import kvprm_oracle as ko

    s = w.shape
    ro = oin.readout_from_synth(s, w.seed, layer_cache=1)
    npages = sum(-(-L // s.page_size) for L in w.lengths)
    cache = oin.cache_from_synth(w, page_cache=2 * npages + 16)
    gen = [0.0]

    def timed_layer(l):
        t = time.perf_counter()
        r = ro.layer(l)
        gen[0] += time.perf_counter() - t
        return r

    def timed_tiles(l, which, page):
        t = time.perf_counter()
        r = cache.tiles(l, which, page)
        gen[0] += time.perf_counter() - t
        return r

    ro_t = ko.Readout(timed_layer, ro.verify_embed, ro.final_norm, ro.reward_w, ro.reward_b)
    t0 = time.perf_counter()
    z, p = ko.verify_pass(s, ro_t, ko.PagedCache(timed_tiles), w.lengths, w.page_table)
    wall = time.perf_counter() - t0
    oracle_s = wall - gen[0]
    threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    rec = {"value": w.batch / oracle_s, "unit": "scores/s", "cores": threads, "kind": "oracle",
           "sample": (f"{w.name}: one whole call, all {w.batch} candidates through all "
                      f"{s.num_layers} layers (fp64 numpy verify_pass): {wall:.1f} s of wall "
                      f"time, of which {gen[0]:.1f} s in the input generator (subtracted)"),
           "threads": {"blas_projections": threads, "attention_loop": 1},
           "seconds_per_call": oracle_s,
           "host": {"logical_cpus": os.cpu_count(), "cpu_model": _cpu_model()}}
    return rec, z, p


def _cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "attention_ragged_32k_traffic.txt")
ATTN_SOURCES = [os.path.join(ROOT, "paper_2607_09153_amd", "csrc", f)
                for f in ("kvprm_attn.hip", "kvprm_mx_common.h")]


def attention_source_hash():
    import hashlib
    h = hashlib.sha256()
    for f in ATTN_SOURCES:
        h.update(open(f, "rb").read())
    return h.hexdigest()


def measured_traffic(workload):
    """HBM bytes per launch of the attention chunk kernel from the committed FETCH_SIZE /
    WRITE_SIZE summary, scaled by the copy-kernel calibration recorded there; None when the
    summary is for another workload or the attention kernel's sources (kvprm_attn.hip and the
    device helpers it includes) have changed since the counters were taken."""
    if not os.path.exists(TRAFFIC_FILE):
        return None
    kv = {}
    for line in open(TRAFFIC_FILE):
        if ":" in line and not line.startswith("#"):
            k, v = line.split(":", 1)
            kv[k.strip()] = v.strip()
    if kv.get("workload") != workload or kv.get("source_sha256") != attention_source_hash():
        return None
    return float(kv["traffic_bytes_per_launch"])


GOLDEN_DIR = os.path.join(ROOT, "tests", "golden")


def golden_parity(name, p, z):
    """max |dP(+)| and |dz| of a call's scores against the fp64 oracle values stored for this
    workload in tests/golden/ (written by tests/golden/make_golden.py, which calls only the
    oracle), on the candidates stored there; None when there are none."""
    import numpy as np
    path = os.path.join(GOLDEN_DIR, f"{name}.json")
    if not os.path.exists(path):
        return None
    ref = json.load(open(path))
    cand = ref["candidates"]
    dp = float(np.max(np.abs(np.asarray(p, dtype=np.float64)[cand] - np.array(ref["p"]))))
    dz = float(np.max(np.abs(np.asarray(z, dtype=np.float64)[cand] - np.array(ref["z"]))))
    return {"reference": os.path.relpath(path, ROOT), "candidates": cand, "max_abs_dp": dp,
            "max_abs_dz": dz, "tolerance": {"dp": 2e-3, "dz": 2e-2},
            "ok": dp <= 2e-3 and dz <= 2e-2}


def measure_workload(kv, name, steps, warmup, attn_reps):
    """One benchmark workload measured like the headline: whole kvprm_score calls (inputs
    resident in HBM, K calls between two synchronisations, per-call HIP events), the attention
    chunk kernel(s) alone (kvprm_attention_partials: the dominant HBM stream), end-to-end and
    dominant-kernel fractions of the 8 TB/s HBM peak, and parity against the stored oracle
    values. Frees its device memory before returning."""
    import torch
    import synth
    from synth.device import DeviceWorkload

    w = synth.make_workload(name)
    _log(f"workload {name}: B={w.batch} layers={w.shape.num_layers} kv={w.shape.kv_dtype}")
    dw = DeviceWorkload(w)
    torch.cuda.synchronize()
    kv_bytes, w_bytes = algorithmic_bytes(w, dw)
    h = kv.kvprm_create(dw.desc(kv))
    try:
        batch = dw.batch(kv)
        n = kv.kvprm_workspace_size(h, batch)
        ws = torch.empty(n, dtype=torch.uint8, device="cuda")
        scores = torch.empty(w.batch, dtype=torch.float32, device="cuda")
        logits = torch.empty(w.batch, dtype=torch.float32, device="cuda")
        stream = torch.cuda.current_stream()
        cache, readout = dw.cache(kv), dw.readout(kv)

        def step():
            kv.kvprm_score(h, cache, batch, readout, ws.data_ptr(), n, scores.data_ptr(),
                           logits.data_ptr(), stream.cuda_stream)

        for _ in range(warmup):
            step()
        torch.cuda.synchronize()
        evs = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
        t0 = time.perf_counter()
        evs[0].record(stream)
        for i in range(steps):
            step()
            evs[i + 1].record(stream)
        torch.cuda.synchronize()
        ms = (time.perf_counter() - t0) * 1e3 / steps
        per_call = sorted(evs[i].elapsed_time(evs[i + 1]) for i in range(steps))
        kernel_ms, step_ms = time_attention(kv, dw, h, batch, ws, n, attn_reps)
        p, z = scores.cpu().numpy(), logits.cpu().numpy()
    finally:
        kv.kvprm_destroy(h)
    kv_layer = kv_bytes / w.shape.num_layers
    e2e = (kv_bytes + w_bytes) / (ms * 1e-3) / 1e9
    attn = kv_layer / (kernel_ms * 1e-3) / 1e9
    out = {"batch": w.batch, "layers": w.shape.num_layers, "hidden": w.shape.hidden,
           "kv_dtype": w.shape.kv_dtype, "cached_tokens": sum(w.lengths),
           "unique_cached_tokens": w.unique_tokens(),
           "ms_per_call": ms, "scores_per_s": w.batch / (ms * 1e-3),
           "per_call_ms": {"median": per_call[len(per_call) // 2], "min": per_call[0],
                           "max": per_call[-1]},
           "bytes_per_call": {"kv": kv_bytes, "weights": w_bytes},
           "end_to_end_gbps": e2e, "end_to_end_frac": e2e / HBM_PEAK_GBPS,
           "dominant_kernel": {"kernel": ("attention chunk kernels, one layer (shared-prefix + "
                                          "private)" if w.group_start else
                                          "k_attn_mx: attention chunk kernel, one layer"),
                               "avg_us": kernel_ms * 1e3, "bytes_per_launch": kv_layer,
                               "achieved_gbps": attn, "frac": attn / HBM_PEAK_GBPS,
                               "with_merge_us": step_ms * 1e3},
           "parity": golden_parity(name, p, z)}
    if w.shape.kv_dtype == "fp8":
        out["fp8_scale"] = w.fp8_scale
    del dw, ws
    torch.cuda.empty_cache()
    _log(f"  {ms:.3f} ms/call, end to end {e2e:.0f} GB/s, attention {kernel_ms * 1e3:.1f} us "
         f"({attn:.0f} GB/s), parity {out['parity']}")
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="ragged_32k")
    ap.add_argument("--no-cpu", action="store_true",
                    help="skip the CPU oracle baseline (one whole oracle call)")
    ap.add_argument("--other-workloads", default="b7_bf16,fixed_32k,beam_prefix,large_fp8",
                    help="comma-separated workloads measured after the headline ('' = none)")
    ap.add_argument("--attn-reps", type=int, default=56)
    ap.add_argument("--lora-rank", type=int, default=256,
                    help="rank of the unmerged adapter of the second timed line (0 = skip)")
    ap.add_argument("--depth", type=int, default=2,
                    help="verify tokens per candidate of the depth-k timed line (1 = skip)")
    ap.add_argument("--steer-steps", type=int, default=2,
                    help="KV steering steps of the last timed line (0 = skip; it rewrites the "
                         "cache, so it runs after every other measurement)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only: the library has no multi-GPU path "
              f"(--gpus {args.gpus} requested)", file=sys.stderr)
        sys.exit(2)

    import torch

    import synth
    from synth.device import DeviceWorkload
    import paper_2607_09153_amd as kv

    torch.cuda.set_device(0)
    w = synth.make_workload(args.workload)
    _log(f"workload {w.name}: B={w.batch} lengths={w.lengths} pages={w.num_pages}")
    t0 = time.time()
    dw = DeviceWorkload(w)
    torch.cuda.synchronize()
    _log(f"inputs generated in HBM in {time.time() - t0:.1f} s")
    kv_bytes, w_bytes = algorithmic_bytes(w, dw)

    h = kv.kvprm_create(dw.desc(kv))
    batch = dw.batch(kv)
    n = kv.kvprm_workspace_size(h, batch)
    ws = torch.empty(n, dtype=torch.uint8, device="cuda")
    scores = torch.empty(w.batch, dtype=torch.float32, device="cuda")
    logits = torch.empty(w.batch, dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream()
    cache, readout = dw.cache(kv), dw.readout(kv)

    def step():
        kv.kvprm_score(h, cache, batch, readout, ws.data_ptr(), n, scores.data_ptr(),
                       logits.data_ptr(), stream.cuda_stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    _log(f"warmup done ({args.warmup} steps)")
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    t0 = time.perf_counter()
    evs[0].record(stream)
    for i in range(args.steps):
        step()
        evs[i + 1].record(stream)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    per_call = sorted(evs[i].elapsed_time(evs[i + 1]) for i in range(args.steps))
    ms = dt * 1e3 / args.steps
    _log(f"timed {args.steps} steps: {ms:.3f} ms/step")
    timed_p, timed_z = scores.cpu().numpy(), logits.cpu().numpy()
    parity = golden_parity(w.name, timed_p, timed_z)
    _log(f"parity of the timed call: {parity}")

    graph = time_graph(kv, h, cache, batch, readout, ws, n, scores, args.steps)
    _log(f"graph replay: {graph['ms_per_call']:.3f} ms/call")
    lora = None
    if args.lora_rank > 0:
        lora = time_lora(kv, dw, h, batch, args.lora_rank, args.steps, args.warmup)
        _log(f"unmerged rank-{args.lora_rank} adapter: {lora['ms_per_call']:.3f} ms/call")
        lora["end_to_end_gbps"] = (kv_bytes + w_bytes + lora["adapter_bytes_per_call"]) / (
            lora["ms_per_call"] * 1e-3) / 1e9
    depth = None
    if args.depth > 1 and w.batch * args.depth > 64:  # a pass holds at most 64 rows
        _log(f"depth-{args.depth} readout skipped: {w.batch} x {args.depth} rows exceed 64")
    elif args.depth > 1:
        depth = time_depth(kv, dw, h, batch, args.depth, args.steps, args.warmup)
        _log(f"depth-{args.depth} readout: {depth['ms_per_call']:.3f} ms/call")
        depth["end_to_end_gbps"] = (kv_bytes + w_bytes) / (depth["ms_per_call"] * 1e-3) / 1e9
    kernel_ms, step_ms = time_attention(kv, dw, h, batch, ws, n, max(args.attn_reps, 1))
    kv_per_layer = kv_bytes / w.shape.num_layers
    achieved = kv_per_layer / (kernel_ms * 1e-3) / 1e9
    _log(f"attention chunk kernel: {kernel_ms * 1e3:.1f} us/layer, {achieved:.0f} GB/s; "
         f"attention step with merge: {step_ms * 1e3:.1f} us/layer")
    steer = None
    if args.steer_steps > 0:
        steer = time_steer(kv, dw, h, batch, args.steer_steps)
        _log(f"KV steering: {steer['ms_per_step']:.3f} ms per step")
    kv.kvprm_destroy(h)
    del dw, ws
    torch.cuda.empty_cache()
    others = {}
    for name in [x for x in args.other_workloads.split(",") if x]:
        others[name] = measure_workload(kv, name, args.steps, args.warmup, max(args.attn_reps, 1))
    copy_gbps = copy_bandwidth()
    _log(f"device copy reference: {copy_gbps:.0f} GB/s")
    read_gbps = read_bandwidth(kv)
    _log(f"streaming read reference: {read_gbps:.0f} GB/s")

    out = {
        "metric": "verify-token scores/sec + achieved KV-read HBM GB/s at L=32k, B=8",
        "value": w.batch / (ms * 1e-3),
        "unit": "scores/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": w.name, "batch": w.batch, "layers": w.shape.num_layers,
                   "hidden": w.shape.hidden, "heads": [w.shape.num_q_heads, w.shape.num_kv_heads],
                   "head_dim": w.shape.head_dim, "ffn": w.shape.ffn_dim,
                   "kv_dtype": w.shape.kv_dtype, "cached_tokens": sum(w.lengths),
                   "mean_length": sum(w.lengths) / w.batch},
        "kv_read_gbps": kv_bytes / (ms * 1e-3) / 1e9,
        "end_to_end_gbps": (kv_bytes + w_bytes) / (ms * 1e-3) / 1e9,
        "bytes_per_call": {"kv": kv_bytes, "weights": w_bytes},
        "roofline": {"kernel": ("k_attn_mx: split-L paged attention chunk kernel, one layer"
                                + (" (with the shared-prefix kernel)" if w.group_start else "")),
                     "bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s", "frac": achieved / HBM_PEAK_GBPS,
                     "traffic": measured_traffic(w.name),
                     "avg_us": kernel_ms * 1e3, "bytes_per_launch": kv_per_layer},
        "attention_step": {"kernels": "chunk kernel + merge (kvprm_attention), one layer",
                           "avg_us": step_ms * 1e3,
                           "kv_gbps": kv_per_layer / (step_ms * 1e-3) / 1e9},
        "per_call_ms": {"median": per_call[len(per_call) // 2], "min": per_call[0],
                        "max": per_call[-1]},
        "end_to_end_frac": (kv_bytes + w_bytes) / (ms * 1e-3) / 1e9 / HBM_PEAK_GBPS,
        "parity": parity,
        "copy_reference_gbps": copy_gbps,
        "read_reference_gbps": read_gbps,
    }
    out["graph_replay"] = graph
    if lora is not None:
        out["lora_readout"] = lora
    if depth is not None:
        out["depth_readout"] = depth
    if steer is not None:
        out["kv_steering"] = steer
    if others:
        out["workloads"] = others
    if not args.no_cpu:
        import numpy as np
        _log("timing one whole oracle call on the CPU ...")
        base, oz, op = cpu_baseline(w)
        out["cpu_baseline"] = base
        # the timed GPU call against that oracle call, every candidate
        if out["parity"] is None:
            out["parity"] = {}
        out["parity"]["vs_oracle_call"] = {
            "candidates": list(range(w.batch)),
            "max_abs_dp": float(np.max(np.abs(timed_p.astype(np.float64) - op))),
            "max_abs_dz": float(np.max(np.abs(timed_z.astype(np.float64) - oz)))}
        _log(f"oracle: {base['seconds_per_call']:.1f} s per call; "
             f"vs GPU {out['parity']['vs_oracle_call']}")
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
