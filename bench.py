"""Benchmark of the QSVD latent-QKV hot path on one MI355X.

Headline (``value``): decode tokens/s of one LLaVA-1.5-7B-shaped attention
layer (d=4096, 32 heads x 128, joint rank r=1536, W8A8, fp16 latent cache) at
batch 16 over a 4096-token context.  One step is the whole decode hot path
for one layer: per-token quantization of the new activations, the quantized
down-projection to the latent C, the latent cache append, the Q
up-projection, and attention over the cached latent (absorbed form).  Steps
cycle through 32 distinct layers (weights and caches, 6.9 GB of cache) so the
cache is read from HBM and not from the 256 MB last-level cache; each layer's
context grows by one token per visit, 4096 -> 4352 over 256 visits.

Also reported: the quantized low-rank QKV prefill of the same layer (batch
4 x 640 tokens) in TOPS against the int8 matrix-core peak, the kernel-level
roofline of the latent attention kernel, timed with HIP events on its launch
stream during the timed region, and the CPU oracle timed on a bounded sample.

    python bench.py [--gpus 1] [--steps K] [--warmup W]
"""
import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "latent-decode tokens/s + HBM GB/s frac; low-rank QKV prefill TOPS (MFMA frac)"
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, GB/s
INT8_PEAK_TOPS = 5033.0        # MI355X dense int8 matrix peak, TOP/s
N_LAYERS = 32                  # LLaVA-1.5-7B language-model layers
DECODE_BATCH, CTX0, DECODE_VISITS = 16, 4096, 256
GQA_VISITS = 8                 # visits per layer in the GQA decode leg
# hardware-counter summary of the latent attention kernel on this workload
ATTN_TRAFFIC_SUMMARY = "latent_attn_llava7b_decode_traffic.txt"
GEMM_TRAFFIC_SUMMARY = "gemm_i8_llava7b_prefill_traffic.txt"
GQA_TRAFFIC_SUMMARY = "latent_attn_qwen2vl_gqa_decode_traffic.txt"
STACK_TRAFFIC_SUMMARY = "latent_attn_h16_13b_stack_decode_traffic.txt"
STACK_GEMM_TRAFFIC_SUMMARY = "gemm_q4_13b_stack_prefill_traffic.txt"
FLASH_TRAFFIC_SUMMARY = "prefill_flash_llava7b_traffic.txt"
PREFILL_SETS = 8               # distinct weight / activation sets the prefill legs rotate through
CPU_SAMPLE_S = 8.0           # seconds of oracle work per headline CPU baseline sample


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=N_LAYERS * DECODE_VISITS)
    ap.add_argument("--warmup", type=int, default=64)
    ap.add_argument("--prefill-steps", type=int, default=20)
    ap.add_argument("--stack-passes", type=int, default=3, help="passes of the 40-layer prefill stack")
    ap.add_argument("--stack-steps", type=int, default=64, help="decode steps through the 40-layer stack")
    ap.add_argument("--mode", choices=["auto", "absorbed", "reconstruct"], default="auto")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-profile", action="store_true", help="time without the kernel events")
    ap.add_argument("--no-graph", action="store_true", help="skip the graph-replay timings (for profiler runs)")
    ap.add_argument("--legs", default="decode,prefill,gqa,stack",
                    help="comma list of legs to run: decode, prefill, gqa (Qwen2-VL-shaped decode), "
                         "stack (13B-shaped 40-layer prefill and decode)")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="MB",
                    help="also run a plain device copy of MB megabytes (calibrates memory counters)")
    return ap.parse_args()


def file_sha256(rel):
    import hashlib
    with open(os.path.join(ROOT, rel), "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def counted_traffic(summary):
    """HBM bytes per launch of a kernel from its committed hardware-counter
    summary under profiles/ (FETCH_SIZE and WRITE_SIZE per dispatch, each
    scaled by what the counter reads for a plain copy of known size), or None
    when the summary is missing or was taken on another version of the
    kernel's source file."""
    path = os.path.join(ROOT, "profiles", summary)
    if not os.path.exists(path):
        return None
    kv = {}
    with open(path) as f:
        for line in f:
            if ":" in line and not line.lstrip().startswith("#"):
                k, v = line.split(":", 1)
                kv[k.strip()] = v.strip()
    try:
        if file_sha256(kv["source"]) != kv["source_sha256"]:
            return None
        return float(kv["hbm_bytes_per_launch"])
    except (KeyError, ValueError, OSError):
        return None


def copy_probe(mb):
    """A plain copy of mb * 2^20 bytes, 4 times, for scaling hardware byte counters."""
    import torch
    n = mb * (1 << 20) // 2
    src = torch.ones(n, dtype=torch.float16, device="cuda")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(4):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(f"[bench] copy probe: 4 copies of {mb} MiB", file=sys.stderr, flush=True)


def cpu_threads():
    try:
        from threadpoolctl import threadpool_info
        n = max((i.get("num_threads", 1) for i in threadpool_info() if i.get("user_api") == "blas"), default=1)
    except Exception:
        n = 1
    return int(n)


def cpu_host():
    """What the oracle's host offers: logical CPUs, the CPUs this process may
    run on, and the BLAS threading (library, threads, environment)."""
    try:
        from threadpoolctl import threadpool_info
        blas = [f"{i.get('internal_api')} {i.get('num_threads')} threads" for i in threadpool_info()
                if i.get("user_api") == "blas"]
    except Exception:
        blas = []
    env = {k: os.environ[k] for k in ("OMP_NUM_THREADS", "OPENBLAS_NUM_THREADS", "MKL_NUM_THREADS")
           if k in os.environ}
    return {"os_cpu_count": os.cpu_count(), "affinity": len(os.sched_getaffinity(0)), "blas": blas, "blas_env": env}


def timed_sample(fn, budget_s, max_iters):
    """Run fn(i) for i = 0, 1, ... until about budget_s seconds (at least once)."""
    n = 0
    t0 = time.perf_counter()
    while n < max_iters and (n == 0 or time.perf_counter() - t0 < budget_s):
        fn(n)
        n += 1
    return n, time.perf_counter() - t0


def replay_seconds(fn, per_graph, replays=5):
    """Mean seconds per call of fn(stream_handle) when per_graph calls run back
    to back: the calls are captured once into a graph, which is replayed
    `replays` times between two events on the replay stream.  Short launches
    timed one by one with their own events read several microseconds long, and
    a host loop of short calls can be bound by the host; the replayed graph is
    neither."""
    import torch

    from paper_2510_16292_amd import binding as B
    fn(B.stream_handle())
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for _ in range(per_graph):
            fn(B.stream_handle())
    g.replay()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(replays):
        g.replay()
    e1.record()
    e1.synchronize()
    del g
    return e0.elapsed_time(e1) * 1e-3 / (replays * per_graph)


def layer_weights(wl, w_bits=8, w_group=0):
    from paper_2510_16292_amd import prep
    from workloads import gen
    U, s, V = gen.weight_factors(wl)
    L = wl.layer
    return (U, s, V), prep.prepare_from_svd(U, s, V, L.n_q_heads, L.n_kv_heads, L.head_dim, wl.beta,
                                            w_bits, w_group)


def graph_line(res):
    if res.get("graph_tokens_per_s") is None:
        return None
    return {"value": round(res["graph_tokens_per_s"], 1), "unit": "tokens/s",
            "ms_per_step": round(res["graph_ms_per_step"], 5)}


def graph_replay(caches, hold, final, rounds, n_layers, batch, step):
    """The decode steps of a full rotation through the layers captured once as
    a graph and replayed per visit (launch grids follow each cache's host
    max_len, held at the final length; chunks past a sequence's length return
    at once)."""
    import torch

    from paper_2510_16292_amd import binding as B
    hold(final - 1)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        gs = B.stream_handle()
        for i in range(n_layers):
            step(i, gs)
    hold(final)
    g.replay()
    hold(final)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(rounds):
        g.replay()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    del g
    for c in caches:
        c.c.max_len = int(c.seq_len.max().item())        # where the replays left the sequences
    return {"graph_ms_per_step": (t1 - t0) * 1e3 / (rounds * n_layers),
            "graph_tokens_per_s": batch * rounds * n_layers / (t1 - t0)}


def run_decode(wl, host_layer, fmt, n_layers, batch, ctx0, steps, warmup, mode_name, profile, traffic_summary,
               compare_forms, graph=True):
    """Decode steps of one attention layer: quantize the new tokens, project
    them (C, Q(C), Q), append, attend over the latent cache.  Steps cycle
    through n_layers distinct layers (weights and caches) so the working set
    exceeds the last-level cache; each layer's context grows by one per visit."""
    import ctypes

    import torch

    from paper_2510_16292_amd import binding as B
    from workloads import gen

    L = wl.layer
    r, d, nq = L.r, L.d, L.n_q
    # every layer is visited at most this often by one pass (the unfused
    # comparison below makes five visits per layer)
    visits = max(-(-steps // n_layers), -(-warmup // n_layers), 5)
    cap = ctx0 + visits + 1
    mode = {"auto": B.QSVD_ATTN_AUTO, "absorbed": B.QSVD_ATTN_ABSORBED,
            "reconstruct": B.QSVD_ATTN_RECONSTRUCT}[mode_name]
    layers = [B.DeviceLayer(host_layer) for _ in range(n_layers)]
    caches = []
    for li in range(n_layers):
        c = B.DeviceCache(fmt, batch, cap, r, [ctx0] * batch)
        if fmt == B.QSVD_CACHE_F16:
            gen.latent_rows_device(wl, batch, ctx0, seed=1000 + li, out=c.data)
        else:
            gen.latent_codes_device(wl, batch, ctx0, seed=1000 + li, codes=c.data, scales=c.scale)
        caches.append(c)
    xs = [torch.from_numpy(gen.decode_activations(wl, t, batch=batch)).cuda() for t in range(8)]
    xq = torch.empty((batch, d), dtype=torch.int8, device="cuda")
    sx = torch.empty((batch,), dtype=torch.float32, device="cuda")
    c_h = torch.empty((batch, r), dtype=torch.float16, device="cuda")
    cq = torch.empty((batch, r), dtype=torch.int8, device="cuda")
    sc = torch.empty((batch,), dtype=torch.float32, device="cuda")
    q = torch.empty((batch, nq), dtype=torch.float16, device="cuda")
    out = torch.empty_like(q)
    pws_b = B.qsvd_prefill_workspace_size(layers[0].c, batch, B.QSVD_OUT_Q)
    pws = torch.empty((max(pws_b, 1),), dtype=torch.uint8, device="cuda")
    dws_b = max(B.qsvd_decode_workspace_size(layers[0].c, c.c, 1, mode) for c in caches)
    dws = torch.empty((dws_b,), dtype=torch.uint8, device="cuda")
    torch.cuda.synchronize()

    lib = B.lib()
    s = B.stream_handle()
    P = B.ptr
    xq_p, sx_p, ch_p, cq_p, sc_p, q_p, out_p = P(xq), P(sx), P(c_h), P(cq), P(sc), P(q), P(out)
    pws_p, dws_p = P(pws), P(dws)
    xs_p = [P(x) for x in xs]
    lrefs = [ctypes.byref(l.c) for l in layers]
    crefs = [ctypes.byref(c.c) for c in caches]
    f16 = fmt == B.QSVD_CACHE_F16

    def step_unfused(i, s=s):
        li = i % n_layers
        st = lib.qsvd_quantize_act(xs_p[i % 8], batch, d, d, 8, 1.0, xq_p, sx_p, s)
        st |= lib.qsvd_lowrank_qkv_prefill(lrefs[li], xq_p, sx_p, batch, 8, B.QSVD_OUT_Q, ch_p, cq_p, sc_p,
                                           q_p, 0, 0, 0, 0, pws_p, pws_b, s)
        st |= lib.qsvd_latent_cache_append(crefs[li], ch_p if f16 else 0, 0 if f16 else cq_p, 0 if f16 else sc_p,
                                           1, s)
        st |= lib.qsvd_latent_decode_attention(lrefs[li], crefs[li], q_p, 1, mode, 0.0, out_p, dws_p, dws_b, s)
        if st:
            raise B.QsvdError(st, B.last_error())

    # one step: the fused projection with its cache append, then the attention
    def step(i, s=s):
        li = i % n_layers
        st = lib.qsvd_decode_project_append(lrefs[li], crefs[li], xs_p[i % 8], d, 8, 1.0, xq_p, sx_p, ch_p, cq_p,
                                            sc_p, q_p, s)
        st |= lib.qsvd_latent_decode_attention(lrefs[li], crefs[li], q_p, 1, mode, 0.0, out_p, dws_p, dws_b, s)
        if st:
            raise B.QsvdError(st, B.last_error())

    def reset():
        torch.cuda.synchronize()
        for c in caches:
            c.seq_len.fill_(ctx0)
            c.c.max_len = ctx0
        torch.cuda.synchronize()

    for i in range(warmup):
        step(i)
    reset()
    # cached tokens each attention launch reads (context after the append)
    ctx_read = sum(batch * (ctx0 + 1 + i // n_layers) for i in range(steps))
    attn_name = "latent_attn" if mode != B.QSVD_ATTN_RECONSTRUCT else "recon"
    # the attention kernel's launches are timed with their own events on the
    # launch stream in every 16th step of the timed region (an event pair per
    # launch adds a few microseconds to its step)
    sample = 16
    B.profile_reset()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(steps):
        if profile and i % sample == 0:
            B.profile_enable(True, attn_name)
            step(i)
            B.profile_enable(False)
        else:
            step(i)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    B.profile_enable(False)
    ms_step = (t1 - t0) * 1e3 / max(steps, 1)
    # contexts the timed attention launches read: one more per visit of a layer
    res = dict(ms_per_step=ms_step, tokens_per_s=batch * steps / (t1 - t0),
               mean_context=ctx_read / max(steps, 1) / batch,
               ctx_range=(ctx0 + 1, ctx0 + -(-steps // n_layers)))
    if profile:
        kms, n = B.profile_read(attn_name)
        B.profile_reset()
        if n:
            avg_s = kms / n * 1e-3
            row_bytes = r * 2 if f16 else r + 4            # cached latent row (+ fp32 scale)
            # cached tokens the sampled launches read
            ctx_sampled = sum(batch * (ctx0 + 1 + i // n_layers) for i in range(0, steps, sample))
            bytes_per_launch = ctx_sampled / len(range(0, steps, sample)) * row_bytes
            achieved = bytes_per_launch / avg_s / 1e9
            traffic = counted_traffic(traffic_summary) if traffic_summary and mode != B.QSVD_ATTN_RECONSTRUCT \
                else None
            res["attn_kernel_us"] = avg_s * 1e6
            res["roofline"] = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                               "frac": round(achieved / HBM_PEAK_GBS, 4),
                               "traffic": None if traffic is None else int(traffic),
                               "kernel": "latent_attn_kernel", "launches": n,
                               "bytes_per_launch": int(bytes_per_launch)}
    # the same step as four separate calls (quantize, projection, append,
    # attention), four visits of every layer after one, for comparison
    for key, fn in (("unfused_ms_per_step", step_unfused),):
        reset()
        for i in range(n_layers):
            fn(i)
        torch.cuda.synchronize()
        u0 = time.perf_counter()
        for i in range(n_layers, 5 * n_layers):
            fn(i)
        torch.cuda.synchronize()
        res[key] = (time.perf_counter() - u0) * 1e3 / (4 * n_layers)

    # The same steps replayed from one captured graph of a full rotation
    # through the layers (launch grids follow each cache's host max_len, held
    # at the final length; chunks past a sequence's length return at once).
    def hold(max_len):
        torch.cuda.synchronize()
        for c in caches:
            c.seq_len.fill_(ctx0)
            c.c.max_len = max_len
        torch.cuda.synchronize()

    final = ctx0 + visits
    rounds = max(steps // n_layers, 1)
    if not graph:
        res["graph_ms_per_step"] = res["graph_tokens_per_s"] = None
    else:
        res.update(graph_replay(caches, hold, final, rounds, n_layers, batch, step))
    if compare_forms:
        # absorbed vs reconstruct on this layer, attention call alone (a few
        # calls each); with rotary embeddings (base 1e4): the form with the
        # value side in latent space (ABSORBED) and the full rebuild
        forms = {}
        for name, m, theta in (("absorbed", B.QSVD_ATTN_ABSORBED, 0.0),
                               ("reconstruct", B.QSVD_ATTN_RECONSTRUCT, 0.0),
                               ("rope_latent_v", B.QSVD_ATTN_ABSORBED, 1.0e4),
                               ("rope_reconstruct", B.QSVD_ATTN_RECONSTRUCT, 1.0e4)):
            wsb = B.qsvd_decode_workspace_size(layers[0].c, caches[0].c, 1,
                                               B.QSVD_ATTN_RECONSTRUCT if theta else m)
            ws = torch.empty((wsb,), dtype=torch.uint8, device="cuda")
            reps = 3 if (m == B.QSVD_ATTN_RECONSTRUCT or theta) else 20

            def call():
                if theta:
                    return lib.qsvd_latent_decode_attention_rope(lrefs[0], crefs[0], q_p, 1, m, 0.0, theta, out_p,
                                                                 P(ws), wsb, s)
                return lib.qsvd_latent_decode_attention(lrefs[0], crefs[0], q_p, 1, m, 0.0, out_p, P(ws), wsb, s)
            for _ in range(2):
                B.check(call())
            torch.cuda.synchronize()
            a = time.perf_counter()
            for _ in range(reps):
                B.check(call())
            torch.cuda.synchronize()
            forms[name] = round((time.perf_counter() - a) * 1e6 / reps, 1)
            del ws
        res["attention_form_us"] = forms
    del caches, layers
    torch.cuda.empty_cache()
    return res


def bench_decode(args, wl, host_layer):
    from paper_2510_16292_amd import binding as B
    return run_decode(wl, host_layer, B.QSVD_CACHE_F16, N_LAYERS, DECODE_BATCH, CTX0, args.steps, args.warmup,
                      args.mode, not args.no_profile, ATTN_TRAFFIC_SUMMARY, True, not args.no_graph)


def bench_decode_gqa(args):
    """The Qwen2-VL-7B-shaped GQA layer (28/4 heads, r=1024, W4A8 with int4
    per-group-128 weights, int8 latent cache with per-token scales) at batch 32
    over 8192 cached tokens, 28 distinct layers."""
    from paper_2510_16292_amd import binding as B
    from workloads import configs
    wl4 = configs.get(4)
    _, host = layer_weights(wl4, wl4.w_bits, wl4.w_group)
    steps = wl4.n_layers * GQA_VISITS
    res = run_decode(wl4, host, B.QSVD_CACHE_I8, wl4.n_layers, wl4.decode_batch, wl4.decode_ctx, steps,
                     wl4.n_layers, "auto", not args.no_profile, GQA_TRAFFIC_SUMMARY, True, not args.no_graph)
    out = {"value": round(res["tokens_per_s"], 1), "unit": "tokens/s", "ms_per_step": round(res["ms_per_step"], 5),
           "steps": steps,
           "workload": f"qwen2-vl-7b-shaped GQA layer decode: batch {wl4.decode_batch}, int8 latent cache r=1024 "
                       f"with per-token scales, context {res['ctx_range'][0]}..{res['ctx_range'][1]} after the append, "
                       f"W4A8 (int4 per-group-128 weights), {wl4.n_layers} rotated layers; tokens/s per layer step",
           "mean_context": round(res["mean_context"], 1),
           "graph_replay": graph_line(res),
           "unfused_ms_per_step": round(res["unfused_ms_per_step"], 5),
           "attention_form_us": res["attention_form_us"]}
    if "roofline" in res:
        out["roofline"] = res["roofline"]
        out["attn_kernel_us"] = round(res["attn_kernel_us"], 2)
    return out


def bench_prefill(args, wl2, host_layer):
    import torch

    from paper_2510_16292_amd import binding as B
    from workloads import gen

    L = wl2.layer
    M, d, r, nq, nkv = wl2.prefill_M, L.d, L.r, L.n_q, L.n_kv
    # PREFILL_SETS distinct layers (device weights) and activation buffers in
    # rotation, so that the 256 MB last-level cache holds no call's operands
    # from the previous visit: 8 x (25 MB of weights + 21 MB of X + 10.5 MB of
    # codes) = 452 MB
    dls = [B.DeviceLayer(host_layer) for _ in range(PREFILL_SETS)]
    dl = dls[0]
    X0 = torch.from_numpy(gen.prefill_activations(wl2)).cuda()
    Xs = [X0] + [X0.clone() for _ in range(PREFILL_SETS - 1)]
    xqs = [torch.empty((M, d), dtype=torch.int8, device="cuda") for _ in range(PREFILL_SETS)]
    sxs = [torch.empty((M,), dtype=torch.float32, device="cuda") for _ in range(PREFILL_SETS)]
    c_h = torch.empty((M, r), dtype=torch.float16, device="cuda")
    cq = torch.empty((M, r), dtype=torch.int8, device="cuda")
    sc = torch.empty((M,), dtype=torch.float32, device="cuda")
    q = torch.empty((M, nq), dtype=torch.float16, device="cuda")
    k = torch.empty((M, nkv), dtype=torch.float16, device="cuda")
    v = torch.empty((M, nkv), dtype=torch.float16, device="cuda")
    wsb = B.qsvd_prefill_workspace_size(dl.c, M, 7)
    ws = torch.empty((max(wsb, 1),), dtype=torch.uint8, device="cuda")
    s = B.stream_handle()
    P = B.ptr
    nxt = [0]          # the set the next captured call uses

    # one prefill call: the activation quantizer, then the projection (X W^d,
    # the latent quantization Q(C), Q(C) W^u)
    def quantize(st, i):
        B.check(B.qsvd_quantize_act(P(Xs[i]), M, d, d, 8, 1.0, P(xqs[i]), P(sxs[i]), st))

    def project(st, i):
        B.check(B.qsvd_lowrank_qkv_prefill(dls[i].c, P(xqs[i]), P(sxs[i]), M, 8, 7, P(c_h), P(cq), P(sc), P(q),
                                           P(k), P(v), 0, 0, P(ws), wsb, st))

    def rotating(fn):
        def f(st):
            fn(st, nxt[0] % PREFILL_SETS)
            nxt[0] += 1
        return f

    def call(st, i):
        quantize(st, i)
        project(st, i)

    for i in range(PREFILL_SETS):
        quantize(s, i)
    ops = 2.0 * M * (d * r + r * L.N)            # X W^d then Q(C) W^u, multiply-adds counted twice
    replays = max(args.prefill_steps // PREFILL_SETS, 2)
    # the projection proper: both products and the latent quantization between them
    proj_s = replay_seconds(rotating(project), PREFILL_SETS, replays)
    call_s = replay_seconds(rotating(call), PREFILL_SETS, replays)
    # Q(C) alone: the same kernel and grid as inside the projection call
    lq_s = replay_seconds(lambda st: B.check(B.qsvd_quantize_act(P(c_h), M, r, r, 8, 1.0, P(cq), P(sc), st)), 20)
    gemm_s = proj_s - lq_s
    # the activation quantizer alone, plain and with the online H1 rotation
    # (block Walsh-Hadamard of order 4096 with seeded signs): fp16 in, int8 + scale out
    signs = torch.from_numpy(np.where(np.arange(d) % 3 == 0, -1, 1).astype(np.int8)).cuda()
    quant = {}
    for name, fn in (("plain", quantize),
                     ("rotated", lambda st, i: B.check(B.qsvd_quantize_act_rotated(
                         P(Xs[i]), M, d, d, 8, 1.0, P(signs), d, P(xqs[i]), P(sxs[i]), st)))):
        us = replay_seconds(rotating(fn), 2 * PREFILL_SETS) * 1e6
        qbytes = M * (2 * d + d + 4)
        quant[name] = {"us": round(us, 2), "GB/s": round(qbytes / (us * 1e-6) / 1e9, 1),
                       "frac": round(qbytes / (us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4)}
    project(s, 0)          # Q, K, V of set 0 for the attention below
    tops = ops / proj_s / 1e12
    # causal attention of the 4 x 640 prompt over the projection's own Q, K, V
    # (fp16 matrix cores), and the latent (absorbed) form of the same
    # attention over an fp16 latent cache of the prompt, for comparison
    lengths = [M // wl2.prefill_batch] * wl2.prefill_batch
    att_s = time_prefill_attention(q, k, v, lengths, L.n_q_heads, L.n_kv_heads, L.head_dim, 20)
    att_flops = causal_flops(lengths, L.n_q_heads, L.head_dim)
    rope_s = time_prefill_attention(q, k, v, lengths, L.n_q_heads, L.n_kv_heads, L.head_dim, 20, rope_theta=10000.0)
    dc = B.DeviceCache(B.QSVD_CACHE_F16, len(lengths), lengths[0], r, [0] * len(lengths))
    B.check(B.qsvd_latent_cache_append(dc.c, P(c_h), 0, 0, lengths[0], s))
    wsa = B.qsvd_decode_workspace_size(dl.c, dc.c, lengths[0], B.QSVD_ATTN_ABSORBED)
    wsa_t = torch.empty((wsa,), dtype=torch.uint8, device="cuda")
    oa = torch.empty_like(q)
    absorbed = lambda: B.check(B.qsvd_latent_decode_attention(dl.c, dc.c, P(q), lengths[0], B.QSVD_ATTN_ABSORBED,
                                                                0.0, P(oa), P(wsa_t), wsa, s))
    absorbed()
    torch.cuda.synchronize()
    a0 = time.perf_counter()
    for _ in range(3):
        absorbed()
    torch.cuda.synchronize()
    abs_s = (time.perf_counter() - a0) / 3
    del dc, wsa_t, oa
    # HBM bytes of one launch on the 4 x 640 prompt, from the committed counter summary
    flash_traffic = counted_traffic(FLASH_TRAFFIC_SUMMARY) if lengths == [640] * 4 else None
    attention = {"value": round(att_flops / att_s / 1e12, 1), "unit": "TFLOP/s", "us": round(att_s * 1e6, 2),
                 "gflop": round(att_flops / 1e9, 2), "lengths": lengths,
                 "absorbed_form_us": round(abs_s * 1e6, 1),
                 "rotary": {"us": round(rope_s * 1e6, 2), "TFLOP/s": round(att_flops / rope_s / 1e12, 1),
                            "rope_theta": 10000.0, "kernel": "prefill_flash_kernel, q and k turned in the kernel"},
                 "roofline": {"bound": "mfma", "achieved": round(att_flops / att_s / 1e12, 1),
                              "peak": F16_PEAK_TFLOPS, "unit": "TFLOP/s",
                              "frac": round(att_flops / att_s / 1e12 / F16_PEAK_TFLOPS, 4),
                              "traffic": None if flash_traffic is None else int(flash_traffic),
                              "kernel": "prefill_flash_kernel (fp16, 4 dh flop per causal pair and head)"}}
    # HBM bytes of one call's two products (both launches), from the committed counter summary
    traffic = counted_traffic(GEMM_TRAFFIC_SUMMARY) if (M, d, r, L.N) == (2560, 4096, 1536, 12288) else None
    return {"value": round(tops, 1), "unit": "TOPS", "timing": "graph replay of back-to-back calls",
            "ms_per_call": round(call_s * 1e3, 4),
            "projection_ms_per_call": round(proj_s * 1e3, 4), "gemm_ms_per_call": round(gemm_s * 1e3, 4),
            "latent_quant_ms_per_call": round(lq_s * 1e3, 4),
            "gemm_only_tops": round(ops / gemm_s / 1e12, 1), "call_tops": round(ops / call_s / 1e12, 1),
            "tokens": M, "gop_per_call": round(ops / 1e9, 2), "quantizer": quant, "attention": attention,
            "roofline": {"bound": "mfma", "achieved": round(tops, 1), "peak": INT8_PEAK_TOPS, "unit": "TOP/s",
                         "frac": round(tops / INT8_PEAK_TOPS, 4), "traffic": None if traffic is None else int(traffic),
                         "kernel": "gemm_i8 (X W^d, Q(C) W^u) + latent quantization Q(C)",
                         "launches": 3 * PREFILL_SETS * replays}}


F16_PEAK_TFLOPS = 2500.0       # MI355X dense fp16 matrix peak, TFLOP/s


def causal_flops(lengths, n_q_heads, head_dim):
    """Algorithmic flops of causal attention: 4 head_dim per (query, visible key) pair and head."""
    return float(sum(n * (n + 1) // 2 for n in lengths)) * n_q_heads * 4.0 * head_dim


def time_prefill_attention(q, k, v, lengths, n_q_heads, n_kv_heads, head_dim, reps, rope_theta=None):
    """Mean time (s) per causal prefill attention launch over the given rows
    (rotary with rope_theta), launches back to back (graph replay), rotating
    through PREFILL_SETS copies of q, k, v so that the last-level cache holds
    no launch's inputs."""
    import torch

    from paper_2510_16292_amd import binding as B
    cu = torch.tensor(np.concatenate([[0], np.cumsum(lengths)]).astype(np.int32), device="cuda")
    out = torch.empty_like(q)
    sets = [(q, k, v)] + [(q.clone(), k.clone(), v.clone()) for _ in range(PREFILL_SETS - 1)]
    nxt = [0]

    def call(st):
        qq, kk, vv = sets[nxt[0] % PREFILL_SETS]
        nxt[0] += 1
        if rope_theta:
            B.check(B.qsvd_prefill_attention_rope(B.ptr(qq), B.ptr(kk), B.ptr(vv), len(lengths), B.ptr(cu),
                                                  max(lengths), n_q_heads, n_kv_heads, head_dim, 0.0, rope_theta,
                                                  B.ptr(out), st))
        else:
            B.check(B.qsvd_prefill_attention(B.ptr(qq), B.ptr(kk), B.ptr(vv), len(lengths), B.ptr(cu), max(lengths),
                                             n_q_heads, n_kv_heads, head_dim, 0.0, B.ptr(out), st))
    reps = max(reps // PREFILL_SETS, 1) * PREFILL_SETS
    t = replay_seconds(call, reps)
    del sets
    return t


def stack_layers(wl5):
    """The 13B-shaped stack: one layer per seeded rank, int4 weight codes and
    per-group scales drawn on the device (timing only; the stack's shapes,
    bits and groups are the configuration's, its values are not those of an
    SVD)."""
    from paper_2510_16292_amd import binding as B
    from workloads import gen
    L, G = wl5.layer, wl5.w_group
    ranks = gen.stack_ranks(wl5)
    layers = []
    for li, r in enumerate(ranks):
        a_t, s_a = gen.weight_codes_device(50000 + 2 * li, r, L.d, wl5.w_bits, L.d // G)
        b_t, s_b = gen.weight_codes_device(50001 + 2 * li, L.N, r, wl5.w_bits, r // G)
        layers.append(B.DeviceLayer.from_device(L.d, r, L.n_q_heads, L.n_kv_heads, L.head_dim, wl5.w_bits, G,
                                                a_t, s_a, b_t, s_b))
    return ranks, layers


def bench_stack_prefill(args, wl5, ranks, layers):
    """Prefill of 8 x (576 + 128) tokens through the 40 layers' quantized QKV
    projections (W4A4): per layer the 4-bit activation quantizer, X W^d with
    the latent quantization fused, Q(C) W^u into Q, K, V."""
    import torch

    from paper_2510_16292_amd import binding as B
    from workloads import gen
    L = wl5.layer
    M, d, nq, nkv = wl5.prefill_M, L.d, L.n_q, L.n_kv
    rmax = max(ranks)
    xs = [torch.from_numpy(gen.prefill_activations(wl5, layer=li)).cuda() for li in range(2)]
    xq = torch.empty((M, d // 2), dtype=torch.uint8, device="cuda")
    sx = torch.empty((M,), dtype=torch.float32, device="cuda")
    c_h = torch.empty((M, rmax), dtype=torch.float16, device="cuda")
    cq = torch.empty((M, rmax // 2), dtype=torch.uint8, device="cuda")
    sc = torch.empty((M,), dtype=torch.float32, device="cuda")
    q = torch.empty((M, nq), dtype=torch.float16, device="cuda")
    k = torch.empty((M, nkv), dtype=torch.float16, device="cuda")
    v = torch.empty((M, nkv), dtype=torch.float16, device="cuda")
    lib, s, P = B.lib(), B.stream_handle(), B.ptr
    xs_p = [P(x) for x in xs]

    # a pass: per layer the 4-bit activation quantizer, then the projection
    # (X W^d, Q(C), Q(C) W^u); the projections alone; the latent quantizations alone
    def stack_pass(st, quantize=True, project=True, latent_only=False):
        for li, dl in enumerate(layers):
            e = 0
            if quantize:
                e |= lib.qsvd_quantize_act(xs_p[li % 2], M, d, d, 4, 1.0, P(xq), P(sx), st)
            if project:
                e |= lib.qsvd_lowrank_qkv_prefill(dl.c, P(xq), P(sx), M, 4, 7, P(c_h), P(cq), P(sc), P(q), P(k),
                                                  P(v), 0, 0, 0, 0, st)
            if latent_only:
                e |= lib.qsvd_quantize_act(P(c_h), M, ranks[li], ranks[li], 4, 1.0, P(cq), P(sc), st)
            if e:
                raise B.QsvdError(e, B.last_error())

    passes = max(args.stack_passes, 1)
    pass_s = replay_seconds(stack_pass, 1, passes)
    proj_s = replay_seconds(lambda st: stack_pass(st, quantize=False), 1, passes)
    lq_s = replay_seconds(lambda st: stack_pass(st, quantize=False, project=False, latent_only=True), 1, passes)
    gemm_s = proj_s - lq_s
    ops = sum(2.0 * M * r * (d + L.N) for r in ranks)
    tops = ops / proj_s / 1e12
    lengths = [M // wl5.prefill_batch] * wl5.prefill_batch
    att_s = time_prefill_attention(q, k, v, lengths, L.n_q_heads, L.n_kv_heads, L.head_dim, 40)
    rope_s = time_prefill_attention(q, k, v, lengths, L.n_q_heads, L.n_kv_heads, L.head_dim, 40, rope_theta=10000.0)
    att_flops = causal_flops(lengths, L.n_q_heads, L.head_dim)
    attention = {"value": round(att_flops / att_s / 1e12, 1), "unit": "TFLOP/s", "us_per_layer": round(att_s * 1e6, 2),
                 "gflop_per_layer": round(att_flops / 1e9, 2), "lengths": lengths,
                 "rotary": {"us_per_layer": round(rope_s * 1e6, 2), "TFLOP/s": round(att_flops / rope_s / 1e12, 1),
                            "rope_theta": 10000.0},
                 "roofline": {"bound": "mfma", "achieved": round(att_flops / att_s / 1e12, 1),
                              "peak": F16_PEAK_TFLOPS, "unit": "TFLOP/s",
                              "frac": round(att_flops / att_s / 1e12 / F16_PEAK_TFLOPS, 4), "traffic": None,
                              "kernel": "prefill_flash_kernel (fp16)"}}
    del xs, xq, c_h, cq, q, k, v
    traffic = counted_traffic(STACK_GEMM_TRAFFIC_SUMMARY)
    return {"value": round(tops, 1), "unit": "TOPS", "timing": "graph replay of whole passes",
            "ms_per_pass": round(pass_s * 1e3, 3),
            "projection_ms_per_pass": round(proj_s * 1e3, 3), "gemm_ms_per_pass": round(gemm_s * 1e3, 3),
            "latent_quant_ms_per_pass": round(lq_s * 1e3, 3),
            "gemm_only_tops": round(ops / gemm_s / 1e12, 1), "call_tops": round(ops / pass_s / 1e12, 1),
            "tokens": M, "layers": len(ranks), "top_per_pass": round(ops / 1e12, 3), "attention": attention,
            "roofline": {"bound": "mfma", "achieved": round(tops, 1), "peak": INT8_PEAK_TOPS, "unit": "TOP/s",
                         "frac": round(tops / INT8_PEAK_TOPS, 4), "traffic": None if traffic is None else int(traffic),
                         "kernel": "gemm_q4_pipe (X W^d and Q(C) W^u, int4 x int4) + latent quantization Q(C)",
                         "launches": 3 * len(ranks) * passes}}


def bench_stack_decode(args, wl5, ranks, layers):
    """Decode through the 40-layer stack at batch 8 over 4096 cached tokens
    (int4 latent caches, W4A4 projections): per layer the 4-bit quantizer, the
    Q-only projection with the latent quantization fused, the append, and the
    absorbed attention (16-head blocks).  Timed eagerly and as one captured
    graph of the 40 layers replayed once per step."""
    import torch

    from paper_2510_16292_amd import binding as B
    from workloads import gen
    L = wl5.layer
    batch, ctx0, steps = wl5.decode_batch, wl5.decode_ctx, args.stack_steps
    d, nq = L.d, L.n_q
    rmax = max(ranks)
    cap = ctx0 + steps + 4
    caches = []
    for li, r in enumerate(ranks):
        c = B.DeviceCache(B.QSVD_CACHE_I4, batch, cap, r, [ctx0] * batch)
        gen.latent_codes_device(gen.with_rank(wl5, r), batch, ctx0, seed=3000 + li, codes=c.data, scales=c.scale,
                                bits=4)
        caches.append(c)
    xs = [torch.from_numpy(gen.decode_activations(wl5, t, batch=batch)).cuda() for t in range(8)]
    xq = torch.empty((batch, d // 2), dtype=torch.uint8, device="cuda")
    sx = torch.empty((batch,), dtype=torch.float32, device="cuda")
    c_h = torch.empty((batch, rmax), dtype=torch.float16, device="cuda")
    cq = torch.empty((batch, rmax // 2), dtype=torch.uint8, device="cuda")
    sc = torch.empty((batch,), dtype=torch.float32, device="cuda")
    q = torch.empty((batch, nq), dtype=torch.float16, device="cuda")
    out = torch.empty_like(q)
    for c in caches:
        c.c.max_len = cap - 1
    dws_b = max(B.qsvd_decode_workspace_size(l.c, c.c, 1, B.QSVD_ATTN_AUTO) for l, c in zip(layers, caches))
    dws = torch.empty((dws_b,), dtype=torch.uint8, device="cuda")
    lib, P = B.lib(), B.ptr
    xs_p = [P(x) for x in xs]

    def step_all(s):
        for li, (dl, c) in enumerate(zip(layers, caches)):
            st = lib.qsvd_decode_project_append(dl.c, c.c, xs_p[li % 8], d, 4, 1.0, P(xq), P(sx), P(c_h), P(cq),
                                                P(sc), P(q), s)
            st |= lib.qsvd_latent_decode_attention(dl.c, c.c, P(q), 1, B.QSVD_ATTN_AUTO, 0.0, P(out), P(dws), dws_b,
                                                   s)
            if st:
                raise B.QsvdError(st, B.last_error())

    def reset(max_len):
        torch.cuda.synchronize()
        for c in caches:
            c.seq_len.fill_(ctx0)
            c.c.max_len = max_len
        torch.cuda.synchronize()

    # Launch grids follow each cache's host max_len: holding it at the final
    # length makes every step (eager or replayed) use the same configuration;
    # chunks past a sequence's device length return at once.
    s = B.stream_handle()

    def eager_steps(profile):
        reset(ctx0 + steps - 1)
        if profile:
            B.profile_reset()
            B.profile_enable(True, "latent_attn")
        t0 = time.perf_counter()
        for _ in range(steps):
            step_all(s)
            for c in caches:
                c.c.max_len = ctx0 + steps - 1
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        B.profile_enable(False)
        return (t1 - t0) / steps

    reset(ctx0 + steps - 1)
    step_all(s)
    eager_s = eager_steps(False)
    eager_steps(True)
    kms, n = B.profile_read("latent_attn")
    B.profile_reset()
    ctx_mean = ctx0 + (steps + 1) / 2.0
    attn_bytes = sum(batch * ctx_mean * (r // 2 + 4) for r in ranks) * steps
    res = {"eager_ms_per_step": round(eager_s * 1e3, 4), "eager_tokens_per_s": round(batch / eager_s, 1),
           "steps": steps, "layers": len(ranks), "batch": batch, "mean_context": round(ctx0 + (steps + 1) / 2.0, 1)}
    if n:
        res["attn_kernel_us"] = round(kms * 1e-3 / n * 1e6, 2)
        achieved = attn_bytes / (kms * 1e-3) / 1e9
        traffic = counted_traffic(STACK_TRAFFIC_SUMMARY)
        res["roofline"] = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                           "frac": round(achieved / HBM_PEAK_GBS, 4),
                           "traffic": None if traffic is None else int(traffic),
                           "kernel": "latent_attn_h16_kernel (int4 cache)", "launches": n,
                           "bytes_per_launch": int(attn_bytes / n)}
    # the rotary variant of layer 0's attention (40 heads: the full-rebuild
    # form, K and V rebuilt from the int4 cache and K turned per position),
    # attention call alone over the final context, a few calls
    reset(ctx0 + steps - 1)
    rws_b = B.qsvd_decode_workspace_size(layers[0].c, caches[0].c, 1, B.QSVD_ATTN_RECONSTRUCT)
    rws = torch.empty((rws_b,), dtype=torch.uint8, device="cuda")
    rope_call = lambda: B.check(lib.qsvd_latent_decode_attention_rope(layers[0].c, caches[0].c, P(q), 1,
                                                                      B.QSVD_ATTN_AUTO, 0.0, 1.0e4, P(out), P(rws),
                                                                      rws_b, s))
    rope_call()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(3):
        rope_call()
    torch.cuda.synchronize()
    res["rotary_attention_us"] = {"us": round((time.perf_counter() - t0) * 1e6 / 3, 1), "rope_theta": 1.0e4,
                                  "form": "full rebuild (K, V from the int4 cache), 40 heads"}
    del rws
    if args.no_graph:
        res.update(value=res["eager_tokens_per_s"], unit="tokens/s", ms_per_step=res["eager_ms_per_step"],
                   us_per_layer_step=round(eager_s * 1e6 / len(ranks), 2), timing="eager")
        del caches
        torch.cuda.empty_cache()
        return res
    # the same step captured once as a graph of all layers, replayed per step
    reset(ctx0 + steps - 1)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step_all(B.stream_handle())
    reset(ctx0 + steps)
    g.replay()
    reset(ctx0 + steps)
    t0 = time.perf_counter()
    for _ in range(steps):
        g.replay()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    graph_s = (t1 - t0) / steps
    res.update(value=round(batch / graph_s, 1), unit="tokens/s", ms_per_step=round(graph_s * 1e3, 4),
               us_per_layer_step=round(graph_s * 1e6 / len(ranks), 2), timing="graph replay")
    del g, caches
    torch.cuda.empty_cache()
    return res


def bench_stack(args):
    from workloads import configs
    wl5 = configs.get(5)
    ranks, layers = stack_layers(wl5)
    out = {"workload": "llava-1.5-13b-shaped stack: 40 layers, d=5120, 40 heads x 128, per-layer ranks "
                       f"{min(ranks)}..{max(ranks)} (mean {sum(ranks) / len(ranks):.0f}), W4A4 with int4 "
                       "per-group-128 weights, int4 latent cache; weight codes drawn on the device",
           "prefill": bench_stack_prefill(args, wl5, ranks, layers)}
    print(f"[bench] stack prefill done: {out['prefill']['value']} TOPS", file=sys.stderr, flush=True)
    out["decode"] = bench_stack_decode(args, wl5, ranks, layers)
    return out


def cpu_baseline_decode(wl, factors):
    """The oracle, as it stands, on one full decode step of the 16-sequence
    batch at context 4096 (projection, append, attention in the plain
    reconstruct form); tokens/s of that step."""
    from oracle import qsvd_oracle as O
    from workloads import gen
    L = wl.layer
    U, s, V = factors
    A, Bm = O.split_beta(U, s, V.T, wl.beta)
    ol = O.make_layer(A, Bm, L.n_q_heads, L.n_kv_heads, L.head_dim, 8, 0)
    n_seq = DECODE_BATCH
    max_steps = 64
    oc = O.LatentCache(O.CACHE_F16, n_seq, CTX0 + max_steps, L.r)
    rows = gen.latent_rows(wl, n_seq, CTX0)
    for b in range(n_seq):
        oc.append(b, rows[b])
    # successive steps (each appends one token per sequence) until about
    # CPU_SAMPLE_S seconds of work
    steps = 0
    t0 = time.perf_counter()
    while steps < max_steps and (steps == 0 or time.perf_counter() - t0 < CPU_SAMPLE_S):
        O.decode_step(ol, oc, gen.decode_activations(wl, steps, batch=n_seq), 8)
        steps += 1
    dt = time.perf_counter() - t0
    return {"value": round(n_seq * steps / dt, 2), "unit": "tokens/s", "cores": cpu_threads(), "kind": "oracle",
            "sample": f"{steps} decode step{'s' if steps != 1 else ''} of all {n_seq} sequences from context {CTX0} (fp64 plain form), "
                      f"{dt:.1f} s", "host": cpu_host()}


def cpu_baseline_prefill(wl2, factors):
    from oracle import qsvd_oracle as O
    from workloads import gen
    L = wl2.layer
    U, s, V = factors
    A, Bm = O.split_beta(U, s, V.T, wl2.beta)
    ol = O.make_layer(A, Bm, L.n_q_heads, L.n_kv_heads, L.head_dim, 8, 0)
    X = gen.prefill_activations(wl2)
    seqs = [X[i:i + 640] for i in range(0, X.shape[0], 640)]
    # the batch's 640-token sequences in turn until about CPU_SAMPLE_S seconds of work
    calls, tokens = 0, 0
    t0 = time.perf_counter()
    while calls == 0 or time.perf_counter() - t0 < CPU_SAMPLE_S:
        Xs = seqs[calls % len(seqs)]
        O.prefill(ol, Xs, 8)
        calls += 1
        tokens += Xs.shape[0]
    dt = time.perf_counter() - t0
    ops = 2.0 * tokens * (L.d * L.r + L.r * L.N)
    return {"value": round(ops / dt / 1e12, 4), "unit": "TOPS", "cores": cpu_threads(), "kind": "oracle",
            "sample": f"{calls} prefill{'s' if calls != 1 else ''} of 640-token sequences of the 4 x 640 batch, {dt:.1f} s",
            "host": cpu_host()}


def cpu_baseline_other(factors2):
    """Further oracle samples (the oracle as it stands, each a few seconds):
    single-threaded tiny layer and LLaVA-7B-shaped prefill, the one-off
    rebuild of K and V for the 4096 cached tokens of one sequence, and decode
    steps / prefills of the Qwen2-VL-shaped and 13B-shaped layers on a subset
    of their sequences, each scaled to its unit."""
    from threadpoolctl import threadpool_limits

    from oracle import qsvd_oracle as O
    from workloads import configs, gen
    out = {}
    # tiny layer, end to end (64-token prefill, append, 16 decode steps), one thread
    wl1 = configs.get(1)
    L1 = wl1.layer
    A1, B1 = O.factors_from_weight(gen.weight_matrix(wl1), L1.r, wl1.beta)
    ol1 = O.make_layer(A1, B1, L1.n_q_heads, L1.n_kv_heads, L1.head_dim, 8, 0)
    X1 = gen.prefill_activations(wl1)

    def tiny(_):
        c = O.LatentCache(O.CACHE_F16, 1, 64 + 16, L1.r)
        O.cache_append_prefill(c, O.prefill(ol1, X1, 8), [64])
        for t in range(16):
            O.decode_step(ol1, c, gen.decode_activations(wl1, t), 8)
    with threadpool_limits(1):
        n, dt = timed_sample(tiny, 3.0, 50)
    out["tiny_end_to_end_1thread"] = {"value": round(16 * n / dt, 2), "unit": "decode tokens/s", "cores": 1,
                                      "sample": f"{n} runs of prefill (64 tokens) + 16 decode steps, {dt:.1f} s"}
    # LLaVA-7B-shaped prefill of one 640-token sequence, one thread
    wl2 = configs.get(2)
    L2 = wl2.layer
    U, sg, V = factors2
    A2, B2 = O.split_beta(U, sg, V.T, wl2.beta)
    ol2 = O.make_layer(A2, B2, L2.n_q_heads, L2.n_kv_heads, L2.head_dim, 8, 0)
    X2 = gen.prefill_activations(wl2)[:640]
    with threadpool_limits(1):
        n, dt = timed_sample(lambda i: O.prefill(ol2, X2, 8), 4.0, 20)
    ops = 2.0 * 640 * n * (L2.d * L2.r + L2.r * L2.N)
    out["llava7b_prefill_1thread"] = {"value": round(ops / dt / 1e12, 4), "unit": "TOPS", "cores": 1,
                                      "sample": f"{n} prefills of one 640-token sequence, {dt:.1f} s"}
    # the one-off rebuild K^, V^ = C W^u_k,v of one sequence's 4096 cached rows (fp64)
    rows = gen.latent_rows(configs.get(3), 1, CTX0)[0].astype(np.float64)
    Bh = ol2.B_hat()[:, L2.n_q:]
    n, dt = timed_sample(lambda i: rows @ Bh, 4.0, 10)
    out["llava7b_kv_rebuild"] = {"value": round(dt / n * DECODE_BATCH * 1e3, 1), "unit": "ms for 16 x 4096 tokens",
                                 "cores": cpu_threads(),
                                 "sample": f"{n} rebuilds of one sequence's {CTX0} rows, x{DECODE_BATCH} sequences"}
    # Qwen2-VL-shaped decode: 2 of the 32 sequences at context 8192 (int8 cache), scaled to 32
    wl4 = configs.get(4)
    L4 = wl4.layer
    U4, s4, V4 = gen.weight_factors(wl4)
    A4, B4 = O.split_beta(U4, s4, V4.T, wl4.beta)
    ol4 = O.make_layer(A4, B4, L4.n_q_heads, L4.n_kv_heads, L4.head_dim, 4, 128)
    c4 = O.LatentCache(O.CACHE_I8, 2, wl4.decode_ctx + 8, L4.r)
    lat = gen.latent_rows(wl4, 2, wl4.decode_ctx)
    for b in range(2):
        q8, sc8 = O.quantize_act(lat[b], 8)
        c4.append(b, None, q8, sc8)
    n, dt = timed_sample(lambda i: O.decode_step(ol4, c4, gen.decode_activations(wl4, i, batch=2), 8), 4.0, 8)
    out["qwen2vl_gqa_decode"] = {"value": round(2 * n / dt, 2), "unit": "tokens/s", "cores": cpu_threads(),
                                 "sample": f"{n} decode steps of 2 sequences from context {wl4.decode_ctx} (int8 "
                                           f"cache, W4A8); the batch of {wl4.decode_batch} takes "
                                           f"{wl4.decode_batch // 2}x as long per step"}
    # 13B-shaped layer at rank 2048 (W4A4, int4 cache): one 704-token prefill, and
    # decode steps of one of the 8 sequences at context 4096
    wl5 = gen.with_rank(configs.get(5), 2048)
    L5 = wl5.layer
    g = np.random.default_rng(5)
    A5 = g.standard_normal((L5.d, L5.r)) / np.sqrt(L5.d)
    B5 = g.standard_normal((L5.r, L5.N)) / np.sqrt(L5.r)
    ol5 = O.make_layer(A5, B5, L5.n_q_heads, L5.n_kv_heads, L5.head_dim, 4, 128)
    X5 = gen.prefill_activations(wl5, rows=704)
    n, dt = timed_sample(lambda i: O.prefill(ol5, X5, 4), 4.0, 10)
    ops = 2.0 * 704 * n * L5.r * (L5.d + L5.N)
    out["stack13b_layer_prefill"] = {"value": round(ops / dt / 1e12, 4), "unit": "TOPS", "cores": cpu_threads(),
                                     "sample": f"{n} prefills of one 704-token sequence through one layer at r=2048"}
    c5 = O.LatentCache(O.CACHE_I4, 1, wl5.decode_ctx + 8, L5.r)
    q4, sc4 = O.quantize_act(gen.latent_rows(wl5, 1, wl5.decode_ctx)[0], 4)
    c5.append(0, None, q4, sc4)
    n, dt = timed_sample(lambda i: O.decode_step(ol5, c5, gen.decode_activations(wl5, i, batch=1), 4), 4.0, 8)
    out["stack13b_layer_decode"] = {"value": round(n / dt, 2), "unit": "tokens/s per layer", "cores": cpu_threads(),
                                    "sample": f"{n} decode steps of 1 sequence from context {wl5.decode_ctx} through "
                                              "one layer at r=2048 (int4 cache); 40 layers and 8 sequences take "
                                              "320x as long per token"}
    return out


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py: the QSVD hot path is measured on one GPU only; multi-GPU runs are not supported "
              f"(asked for --gpus {args.gpus}).", file=sys.stderr)
        sys.exit(2)
    import torch

    from paper_2510_16292_amd import binding as B
    from workloads import configs
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    B.lib()
    wl2, wl3 = configs.get(2), configs.get(3)
    factors, host_layer = layer_weights(wl2)        # one 7B-shaped layer serves both legs
    legs = set(args.legs.split(","))
    if args.copy_probe:
        copy_probe(args.copy_probe)
    dec, pre = None, None
    if "decode" in legs:
        print(f"[bench] decode: {args.steps} steps, warmup {args.warmup}", file=sys.stderr, flush=True)
        dec = bench_decode(args, wl3, host_layer)
        print(f"[bench] decode done: {dec['ms_per_step']:.4f} ms/step", file=sys.stderr, flush=True)
    if "prefill" in legs:
        pre = bench_prefill(args, wl2, host_layer)
        print(f"[bench] prefill done: {pre['value']} TOPS", file=sys.stderr, flush=True)
    gqa = None
    if "gqa" in legs:
        gqa = bench_decode_gqa(args)
        print(f"[bench] gqa decode done: {gqa['ms_per_step']:.4f} ms/step", file=sys.stderr, flush=True)
    stack = None
    if "stack" in legs:
        stack = bench_stack(args)
        print(f"[bench] stack decode done: {stack['decode']['ms_per_step']:.4f} ms/step", file=sys.stderr, flush=True)
    if dec is None:
        print(json.dumps({k: v for k, v in (("prefill", pre), ("gqa_decode", gqa), ("stack13b", stack))
                          if v is not None}), flush=True)
        return
    line = {
        "metric": METRIC,
        "value": round(dec["tokens_per_s"], 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(dec["ms_per_step"], 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "i8+f16",
        "data": "synthetic",
        "config": {"workload": "llava-1.5-7b-shaped attention layer decode: batch 16, fp16 latent cache r=1536, "
                               f"context {dec['ctx_range'][0]}..{dec['ctx_range'][1]} after the append, W8A8 "
                               "projections, 32 rotated layers; value is tokens/s per layer step",
                   "d": 4096, "heads": 32, "head_dim": 128, "rank": 1536, "batch": DECODE_BATCH,
                   "mean_context": round(dec["mean_context"], 1), "attention": args.mode},
        "roofline": dec.get("roofline"),
        "attn_kernel_us": round(dec.get("attn_kernel_us", 0.0), 2),
        "graph_replay": graph_line(dec),
        "unfused_ms_per_step": round(dec["unfused_ms_per_step"], 5),
        "attention_form_us": dec["attention_form_us"],
        "prefill": pre,
    }
    if pre is None:
        line.pop("prefill")
    if gqa is not None:
        line["gqa_decode"] = gqa
    if stack is not None:
        line["stack13b"] = stack
    if not args.no_cpu_baseline:
        print("[bench] cpu baseline (oracle)", file=sys.stderr, flush=True)
        line["cpu_baseline"] = cpu_baseline_decode(wl3, factors)
        if pre is not None:
            line["prefill"]["cpu_baseline"] = cpu_baseline_prefill(wl2, factors)
        line["cpu_baseline"]["other_samples"] = cpu_baseline_other(factors)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
