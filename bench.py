"""Benchmark of KV-PRM verify-token scoring on one MI355X.

One step = one kvprm_score call over the whole hot path (all layers, projections, paged
attention, merge, FFN, reward head) for the ragged long-context batch: the 7B-class shape in
bf16 (28 layers, H=3584, 28/4 heads, d_h=128, FFN 18944), B=8 candidates with cached lengths
L_b ~ U[16384, 32768] on 16-token pages scattered over a pool. Inputs are synthetic (seeded
generator) and resident in HBM before the timed region.

Prints one JSON line: scores/s (value), the end-to-end KV-read rate, the roofline of the
dominant kernel (the split-L attention chunk kernel, timed live with HIP events on its stream;
the whole attention step with its merge is reported beside it), the same workload scored with
the base weights and an unmerged rank-256 adapter on every projection (kvprm_score_lora,
`lora_readout`) and with two verify tokens per candidate (the depth-k readout, kvprm_score_ex,
`depth_readout`), KV steering steps on its cache (kvprm_steer, `kv_steering`), and the fp64
CPU oracle timed on a bounded sample of the same workload.
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


def cpu_baseline(w, layers_sample, min_seconds=10.0):
    """The fp64 oracle, untuned, on all candidates of the workload through its first
    `layers_sample` layers, repeated until at least `min_seconds` of CPU work; input generation
    is done before the clock starts. Scaled to scores/s of the full-depth model."""
    import dataclasses

    from threadpoolctl import threadpool_info

    from oracle import inputs as oin
    from oracle import kvprm_oracle as ko

    s = w.shape
    sub = dataclasses.replace(s, num_layers=layers_sample)
    ro = oin.readout_from_synth(sub, w.seed, layer_cache=layers_sample)
    npages = sum(-(-L // s.page_size) for L in w.lengths)
    cache = oin.cache_from_synth(w, page_cache=2 * layers_sample * npages + 16)
    for l in range(layers_sample):  # materialise inputs outside the timed region
        ro.layer(l)
        for b in range(w.batch):
            for i in range(-(-w.lengths[b] // s.page_size)):
                cache.tiles(l, "k", w.page_table[b][i])
                cache.tiles(l, "v", w.page_table[b][i])
    reps, t0 = 0, time.perf_counter()
    while True:
        ko.verify_pass(sub, ro, cache, w.lengths, w.page_table)
        reps += 1
        dt = time.perf_counter() - t0
        if dt >= min_seconds:
            break
    per_call = dt / reps * s.num_layers / layers_sample
    threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    return {"value": w.batch / per_call, "unit": "scores/s", "cores": threads, "kind": "oracle",
            "sample": (f"{w.name}: all {w.batch} candidates through the first {layers_sample} of "
                       f"{s.num_layers} layers, {reps} passes in {dt:.1f} s (fp64 numpy, inputs "
                       f"pre-generated), scaled by {s.num_layers}/{layers_sample} to one full "
                       f"call"),
            "host": {"logical_cpus": os.cpu_count(), "cpu_model": _cpu_model()}}


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
                for f in ("kvprm_mfma.hip", "kvprm_internal.h")]


def attention_source_hash():
    import hashlib
    h = hashlib.sha256()
    for f in ATTN_SOURCES:
        h.update(open(f, "rb").read())
    return h.hexdigest()


def measured_traffic(workload):
    """HBM bytes per launch of the attention chunk kernel from the committed FETCH_SIZE /
    WRITE_SIZE summary, scaled by the copy-kernel calibration recorded there; None when the
    summary is for another workload or the attention sources have changed since the counters
    were taken."""
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


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="ragged_32k")
    ap.add_argument("--cpu-layers", type=int, default=2,
                    help="layers of the oracle sample for the CPU baseline (0 = skip)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="minimum CPU work of the oracle sample (repeated passes)")
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
    stream = torch.cuda.current_stream()
    cache, readout = dw.cache(kv), dw.readout(kv)

    def step():
        kv.kvprm_score(h, cache, batch, readout, ws.data_ptr(), n, scores.data_ptr(), 0,
                       stream.cuda_stream)

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

    graph = time_graph(kv, h, cache, batch, readout, ws, n, scores, args.steps)
    _log(f"graph replay: {graph['ms_per_call']:.3f} ms/call")
    lora = None
    if args.lora_rank > 0:
        lora = time_lora(kv, dw, h, batch, args.lora_rank, args.steps, args.warmup)
        _log(f"unmerged rank-{args.lora_rank} adapter: {lora['ms_per_call']:.3f} ms/call")
        lora["end_to_end_gbps"] = (kv_bytes + w_bytes + lora["adapter_bytes_per_call"]) / (
            lora["ms_per_call"] * 1e-3) / 1e9
    depth = None
    if args.depth > 1:
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
    if args.cpu_layers > 0:
        _log("timing the oracle on the CPU sample ...")
        out["cpu_baseline"] = cpu_baseline(w, args.cpu_layers, args.cpu_seconds)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
