"""Benchmark of the SpS verify step on one MI355X.

One "step" is one SpS verify step of the 70B-shaped target (d_model 8192,
80 layers, 64 heads x 128, GELU FFN 32768, vocab 32000, bf16, 129.9 GB of
weights resident in HBM): the transformer forward over the K+1 = 5 draft
positions of one sequence against a 2048-token KV cache, the softmax of the
5 target distributions and the fused modified rejection sampling. Inputs are
synthetic and already on the device when timing starts: random-init weights
N(0, 0.02), random bf16 prior keys/values, random tokens and draft
distributions. Lengths are not advanced by the verify step, so every timed
step sees the same context.

Printed: one JSON line with verify-step throughput (algorithmic HBM GB/s),
ms per step, the roofline of the dominant kernel (the weight-streaming GEMM,
timed with HIP events on its stream around every launch, each launch issued
8 times back to back so the event latency is amortised), SpS and ArS tokens/s
of the 70B target with its 3072-wide draft (prompt 2048, 128 new tokens,
K = 4, temperature 1) on a coupled pair whose draft agrees with the target
about as often as the paper's trained drafts (and on an unrelated random
pair beside it), and the CPU oracle timed on a bounded sample.

    python bench.py [--gpus 1] [--steps 20] [--warmup 3] [--K 4] [--B 1] [--ctx 2048]
    python bench.py --sweep | --accept-grid | --k-study | --draft-step | --softmax | --cpu-oracle
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "verify-step ms + HBM GB/s (70B-shape, K=4, bs=1); SpS tokens/sec at 1 GPU"
HBM_PEAK_GBS = 8000.0
GEMM_REPEATS = 8                 # back-to-back launches per event bracket in the roofline pass
CALIBRATION_BYTES = 1 << 30      # plain device copy whose HBM counters calibrate FETCH/WRITE_SIZE
# Sources of the single-tile GEMM kernel (the one the traffic counters were taken on).
GEMM_SOURCES = [os.path.join(ROOT, "paper_2302_01318_amd", "csrc", f)
                for f in ("gemm.hip", "gemm_epi.h", "common.h", "fp8.h")]
PROFILES = os.path.join(ROOT, "profiles")
CPU_BASELINE_SECONDS = 10.0     # CPU work the oracle baseline is timed over
STREAM_READ_BYTES = 8 << 30      # bytes of the packed weights read by the streaming-read ceiling


def source_digest(paths):
    import hashlib
    h = hashlib.sha256()
    for path in paths:
        with open(path, "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def _profile_file(kind, weights):
    """profiles/gemm_<kind>.json for bf16 weights, gemm_<kind>_fp8.json for FP8."""
    return os.path.join(PROFILES, "gemm_%s%s.json" % (kind, "_fp8" if weights == "fp8" else ""))


def measured_traffic(weights="bf16"):
    """HBM bytes per GEMM launch measured with rocprofv3 counters (see the
    profiles/ file), if they were taken on the current GEMM source."""
    try:
        with open(_profile_file("traffic", weights)) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("gemm_source_sha256_16") != source_digest(GEMM_SOURCES):
        return None
    return t.get("hbm_bytes_per_launch")


def measured_mfma(weights="bf16"):
    """MFMA utilisation of the GEMM launches from rocprofv3 counters (see the
    profiles/ file), if they were taken on the current GEMM source."""
    try:
        with open(_profile_file("mfma", weights)) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("gemm_source_sha256_16") != source_digest(GEMM_SOURCES):
        return None
    return {k: t[k] for k in ("mfma_busy_pct", "mfma_executed_tflops", "useful_tflops") if k in t}


def measured_trace(weights="bf16"):
    """Average GEMM launch duration from a rocprofv3 kernel trace of the
    benchmark (see the profiles/ file), if taken on the current GEMM source."""
    try:
        with open(_profile_file("trace", weights)) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("gemm_source_sha256_16") != source_digest(GEMM_SOURCES):
        return None
    return {k: t[k] for k in ("avg_launch_us", "achieved", "frac", "stream_read_gbs", "source") if k in t}


def profiled_figures(shape_name, weights, B, K, ctx):
    """The rocprofv3 figures of profiles/ (traffic, MFMA utilisation, traced
    launch average) for a run of the workload they were taken on -- the
    70B-shaped verify step at K = 4, B = 1, ctx 2048, in the run's weight
    format -- and None for any other workload, whose launches differ."""
    if shape_name != "70b" or (B, K, ctx) != (1, 4, 2048):
        return {"traffic": None, "mfma": None, "trace": None}
    return {"traffic": measured_traffic(weights), "mfma": measured_mfma(weights), "trace": measured_trace(weights)}


def _counter_rows(path):
    """rocprofv3 counter-collection CSV: {dispatch id: {name, grid, counters, seconds}}."""
    import csv
    import re
    d = {}
    for r in csv.DictReader(open(path)):
        k = int(r["Dispatch_Id"])
        e = d.setdefault(k, {"name": re.sub(r"\(.*", "", r["Kernel_Name"]).replace("void ", "").replace("sps::", ""),
                             "grid": int(r["Grid_Size"]),
                             "seconds": (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-9})
        e[r["Counter_Name"]] = e.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
    return d


def ingest_profiles(args):
    """Write profiles/gemm_{traffic,mfma,trace}[_fp8].json from rocprofv3
    output of this benchmark at its default workload (70B, K = 4, B = 1,
    ctx 2048, --weights as given), with the hash of the GEMM sources they
    were taken on (bench.py reports them only while it matches):
      traffic: FETCH_SIZE and WRITE_SIZE counter CSVs (two runs), scaled by
               the 1 GiB calibration copy + the embedding copy the benchmark
               performs;
      mfma:    a CSV of SQ_INSTS_VALU_MFMA_MOPS_BF16, SQ_VALU_MFMA_BUSY_CYCLES
               and GRBM_GUI_ACTIVE;
      trace:   a --kernel-trace CSV: the average gemm_kernel duration, and the
               streaming-read rate from the stream_read_kernel dispatches."""
    import csv
    import re
    from paper_2302_01318_amd import configs
    shape = configs.SEVENTY_B.with_(dtype=args.weights)
    alg = gemm_bytes_per_launch(shape, 5)
    dig = source_digest(GEMM_SOURCES)
    kind, paths = args.ingest[0], args.ingest[1:]
    base = {"workload": "70B-shaped verify step, K=4, B=1, ctx 2048 (321 GEMM launches per step)",
            "weights": args.weights, "gemm_source_sha256_16": dig}
    if kind == "traffic":
        fe, wr = _counter_rows(paths[0]), _counter_rows(paths[1])
        cbytes = (1 << 30) + shape.vocab * shape.d_model * 2          # calibration copy + embedding copy
        cp = [k for k in fe if "copyBuffer" in fe[k]["name"] and fe[k]["grid"] == 131072]
        fs = cbytes / (sum(fe[k]["FETCH_SIZE"] for k in cp) * 1024)
        ws = cbytes / (sum(wr[k]["WRITE_SIZE"] for k in cp) * 1024)
        g = [k for k in fe if fe[k]["name"].startswith("gemm_kernel")]
        per = sum(fe[k]["FETCH_SIZE"] * 1024 * fs + wr[k]["WRITE_SIZE"] * 1024 * ws for k in g) / len(g)
        out = dict(base, kernel="gemm_kernel, all launches of a step", fetch_scale=round(fs, 4),
                   write_scale=round(ws, 4), hbm_bytes_per_launch=int(round(per)),
                   algorithmic_bytes_per_launch=int(round(alg)), launches=len(g),
                   source="profiles/gemm_hbm_traffic_70b.md")
    elif kind == "mfma":
        d = _counter_rows(paths[0])
        busy = act = fl = dur = 0.0
        for r in d.values():
            if r["name"].startswith("gemm_kernel") and "SQ_VALU_MFMA_BUSY_CYCLES" in r:
                busy += r["SQ_VALU_MFMA_BUSY_CYCLES"]
                act += r["GRBM_GUI_ACTIVE"] / 8 * 1024          # 8 XCDs, 1024 SIMDs
                fl += r["SQ_INSTS_VALU_MFMA_MOPS_BF16"] * 512
                dur += r["seconds"]
        n = sum(1 for r in d.values() if r["name"].startswith("gemm_kernel") and "SQ_VALU_MFMA_BUSY_CYCLES" in r)
        HD, F_rows = shape.n_heads * shape.head_dim, shape.d_ff * (2 if shape.ffn == "swiglu" else 1)
        elems = shape.n_layers * (4 * HD * shape.d_model + F_rows * shape.d_model + shape.d_model * shape.d_ff) + \
            shape.vocab * shape.d_model
        useful = 2.0 * 5 * elems / (4 * shape.n_layers + 1) * n          # 5 real rows, every weight once
        out = dict(base, kernel="gemm_kernel, all launches of a step", mfma_busy_pct=round(100 * busy / act, 2),
                   mfma_executed_tflops=round(fl / dur / 1e12, 1), useful_tflops=round(useful / dur / 1e12, 1),
                   peak_tflops_bf16_dense=2500.0, launches=n, source="profiles/gemm_mfma_util_70b.md")
    else:
        rows = list(csv.DictReader(open(paths[0])))
        dur = lambda r: (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-9
        g = [dur(r) for r in rows if re.search(r"gemm_kernel", r["Kernel_Name"])]
        sr = [dur(r) for r in rows if "stream_read_kernel" in r["Kernel_Name"]]
        avg = sum(g) / len(g)
        out = dict(base, kernel="gemm_kernel, every dispatch of the run", dispatches=len(g),
                   avg_launch_us=round(avg * 1e6, 2), achieved=round(alg / avg / 1e9, 1),
                   frac=round(alg / avg / 1e9 / HBM_PEAK_GBS, 4),
                   stream_read_gbs=round(STREAM_READ_BYTES / sorted(sr)[len(sr) // 2] / 1e9, 1) if sr else None,
                   algorithmic_bytes_per_launch=int(round(alg)), source="profiles/verify_step_70b_kernel_trace.md")
    path = _profile_file(kind, args.weights)
    with open(path, "w") as f:
        json.dump(out, f, indent=1)
    print(json.dumps(out))


def stream_read_rate(sps, torch, buf, nbytes=STREAM_READ_BYTES, reps=10):
    """GB/s of the library's plain streaming read over the first `nbytes` of
    `buf` (the attainable HBM read rate on this device), median of `reps`."""
    sink = torch.zeros(1, dtype=torch.int32, device="cuda")
    sps.stream_read(buf, nbytes, sink)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(reps + 1)]
    ev[0].record()
    for i in range(reps):
        sps.stream_read(buf, nbytes, sink)
        ev[i + 1].record()
    torch.cuda.synchronize()
    t = sorted(ev[i].elapsed_time(ev[i + 1]) for i in range(reps))
    return nbytes / (t[reps // 2] * 1e-3) / 1e9


def round_up(x, m):
    return (x + m - 1) // m * m


def verify_bytes(shape, B, K, ctx):
    """Algorithmic HBM bytes of one verify step: every weight once, the KV
    cache of every sequence once (prior context plus the K+1 new positions),
    the new keys/values written once, the logits written and read once."""
    es = shape.act_bytes()
    M = B * (K + 1)
    HD = shape.n_heads * shape.head_dim
    weights = shape.n_layers * shape.matrix_bytes_per_layer() + shape.matrix_bytes(shape.vocab, shape.d_model)
    gains = (2 * shape.n_layers + 1) * shape.d_model * 4
    embed_rows = M * shape.d_model * es
    kv_read = shape.n_layers * B * 2 * HD * (ctx + K + 1) * es
    kv_write = shape.n_layers * M * 2 * HD * es
    logits = 2 * M * shape.vocab * 4
    return weights + gains + embed_rows + kv_read + kv_write + logits


def gemm_bytes_per_launch(shape, M):
    """Algorithmic bytes of one weight-streaming GEMM launch averaged over
    the launches of one forward at M rows: every weight (and FP8 row scale)
    once, the fp32 input activations and the fp32 outputs once -- the figure
    sps_profile_gemm_end accumulates per launch."""
    wes = 1 if shape.dtype == "fp8" else shape.act_bytes()
    HD, d, F = shape.n_heads * shape.head_dim, shape.d_model, shape.d_ff
    F_rows = 2 * F if shape.ffn == "swiglu" else F

    def one(rows_w, K, n_valid):
        return rows_w * K * wes + (4 * rows_w if shape.dtype == "fp8" else 0) + 4 * M * K + 4 * M * n_valid

    layer = one(3 * HD, d, 3 * HD) + one(d, HD, d) + one(F_rows, d, F) + one(d, F, d)
    return (shape.n_layers * layer + one(shape.vocab, d, shape.vocab)) / (4 * shape.n_layers + 1)


def model_shapes(configs, args):
    """Target (70B or 7B shape) and draft shapes, with FP8 projections when
    --weights fp8 (both models) or --draft-weights fp8 (the draft only)."""
    shape = configs.SEVENTY_B if args.shape == "70b" else configs.SEVEN_B
    dshape = configs.DRAFT_70B
    if args.weights == "fp8":
        shape, dshape = shape.with_(dtype="fp8"), dshape.with_(dtype="fp8")
    if getattr(args, "draft_weights", None) == "fp8":
        dshape = dshape.with_(dtype="fp8")
    return shape, dshape


def device_model(sps, synth, shape, seed):
    m = sps.Model(shape)
    for (name, layer), t in synth.device_weights(shape, seed):
        m.pack(name, layer, t)
    return m


E2E_CODE_PERT = 0.5       # draft logit perturbation of the end-to-end coupled pair


def coupled_model(sps, synth, shape, model_seed, code_pert, st, into=None):
    """One model of the coupled pair; packed into the buffers of `into` (a
    model of the same shape) when given. Reusing the buffers matters for
    timing: a generation right after the 70B target was freed and a new one
    allocated ran 28.0 instead of 27.3 ms per loop (the next one 27.3)."""
    m = into if into is not None else sps.Model(shape)
    for (name, layer), t in synth.coupled_device_weights(shape, st["pair_seed"], model_seed, st["layer_std"],
                                                         code_pert, st["logit_std"], st["rank"]):
        m.pack(name, layer, t)
    return m


def cpu_baseline(shape, K, ctx):
    """The oracle (fp64 numpy, as it stands) on a bounded sample: one
    full-width block of the benchmarked shape plus embedding and
    unembedding, K+1 positions of one sequence against a random ctx-token
    cache."""
    import numpy as np
    from oracle import model as om
    from paper_2302_01318_amd import synth
    one = shape.with_(n_layers=1)
    spec = _oracle_spec(one)
    W = _oracle_weights(shape, 1, 0)          # FP8: the oracle's own quantisation, outside the timed region
    cache = om.new_cache(spec, 1, ctx + K + 1)
    k, v = synth.kv_prior(one, 1, 0, 1, ctx)
    cache["k"][0, 0, :, :ctx] = k[0].double().numpy()
    cache["v"][0, 0, :, :ctx] = v[0].double().numpy()
    toks = synth.tokens(2, 1, K + 1, one.vocab)
    # Repeat the sample until ~10 s of CPU work (at least 4 runs).
    reps = 0
    t0 = time.perf_counter()
    while reps < 4 or time.perf_counter() - t0 < CPU_BASELINE_SECONDS:
        om.forward_cached(spec, W, cache, toks, np.array([ctx]))
        reps += 1
    dt = (time.perf_counter() - t0) / reps
    nbytes = verify_bytes(one, 1, K, ctx)
    host = host_info()
    threads = max([i["num_threads"] or 1 for i in host.get("blas", [])] or [host["affinity_cores"]])
    return {"value": nbytes / dt / 1e9, "unit": "GB/s", "cores": threads, "kind": "oracle",
            "seconds_per_sample": dt, "repeats": reps, "host": host,
            "sample": "oracle fp64 forward of one full-width %s-shaped block + embedding + unembedding, "
                      "K+1=%d positions, B=1, ctx %d (%.2f GB algorithmic)" % (shape.name, K + 1, ctx, nbytes / 1e9)}


def host_info():
    """The host the CPU oracle runs on: logical CPUs, the cores this process
    may use, RAM, and the BLAS library numpy calls with its thread count."""
    host = {"cpu_count": os.cpu_count(), "affinity_cores": len(os.sched_getaffinity(0))}
    try:
        host["ram_gb"] = round(os.sysconf("SC_PAGE_SIZE") * os.sysconf("SC_PHYS_PAGES") / 1e9, 1)
    except (ValueError, OSError):
        pass
    try:
        import numpy  # noqa: F401  (loads the BLAS numpy calls)
        from threadpoolctl import threadpool_info
        host["blas"] = [{"api": i.get("internal_api"), "num_threads": i.get("num_threads"),
                         "library": os.path.basename(i.get("filepath") or "")}
                        for i in threadpool_info() if i.get("user_api") == "blas"]
    except Exception:
        pass
    return host


def _oracle_weights(shape, n_layers, seed):
    """The oracle's weight dict (fp32 numpy) of the first n_layers layers of
    the synthetic model `shape` with weight seed `seed` (FP8 models: the
    oracle's own quantisation)."""
    f = lambda t: t.float().numpy()
    from paper_2302_01318_amd import synth
    one = shape.with_(n_layers=n_layers)
    w = {k: synth.weight(one, k[0], k[1], seed) for k in synth.tensor_shapes(one)}
    W = {"embed": f(w[("embed", -1)]), "final_norm": f(w[("final_norm", -1)]), "unembed": f(w[("unembed", -1)]),
         "layers": []}
    for l in range(n_layers):
        lw = {k: f(w[(k, l)]) for k in ("attn_norm", "wq", "wk", "wv", "wo", "ffn_norm")}
        if shape.ffn == "gelu":
            lw.update(w1=f(w[("w1", l)]), w2=f(w[("w2", l)]))
        else:
            lw.update(wg=f(w[("w1", l)]), wu=f(w[("w3", l)]), wd=f(w[("w2", l)]))
        W["layers"].append(lw)
    del w
    if shape.dtype == "fp8":
        from oracle import fp8
        W = fp8.fp8_weights(W)
    return W


def _oracle_spec(shape, n_layers=None):
    from oracle.model import ModelSpec
    return ModelSpec(shape.d_model, shape.n_layers if n_layers is None else n_layers, shape.n_heads, shape.head_dim,
                     shape.d_ff, shape.vocab, shape.ffn, "bf16" if shape.dtype == "fp8" else shape.dtype, shape.eps,
                     shape.rope_base)


def cpu_oracle(args):
    """The oracle's cost on the host's CPUs (numpy as it stands, BLAS threads
    as the host gives them), on bounded samples: the tiny fp32 pair's SpS
    and ArS generations end to end (prompt 32, 64 new tokens, K = 4, T = 1),
    and the verify step (K = 4, B = 1, ctx 2048) of the 7B and 70B shapes,
    timed on 1- and 2-layer models and extrapolated to all layers (the full
    fp32 models do not fit the host: 27 and 260 GB). Reported baselines,
    not targets."""
    import numpy as np
    from oracle import generate as ogen
    from oracle import model as om
    from paper_2302_01318_amd import configs, synth
    log = lambda *a: print(*a, file=sys.stderr, flush=True)
    out = {"metric": "oracle CPU time", "host": host_info()}
    # tiny pair end to end
    tgt, drf = configs.TINY_TARGET, configs.TINY_DRAFT
    Wt, Wd = _oracle_weights(tgt, tgt.n_layers, 100), _oracle_weights(drf, drf.n_layers, 101)
    prompt = synth.tokens(102, 1, 32, tgt.vocab)[0]
    t0 = time.perf_counter()
    toks, acc = ogen.sps_generate_one(_oracle_spec(tgt), Wt, _oracle_spec(drf), Wd, prompt, 64, 4, 1.0, 7)
    t_sps = time.perf_counter() - t0
    t0 = time.perf_counter()
    ogen.ars_generate_one(_oracle_spec(tgt), Wt, prompt, 64, 1.0, 7)
    t_ars = time.perf_counter() - t0
    out["tiny_e2e"] = {"sps_tokens_per_s": round(64 / t_sps, 2), "ars_tokens_per_s": round(64 / t_ars, 2),
                       "sps_seconds": round(t_sps, 3), "ars_seconds": round(t_ars, 3),
                       "sps_mean_accepted": round(float(np.mean(acc)), 3),
                       "note": "oracle generation recomputes the full prefix for every forward"}
    log("tiny e2e: sps %.2f tokens/s, ars %.2f tokens/s" % (64 / t_sps, 64 / t_ars))
    # verify step of the 7B and 70B shapes, from 1- and 2-layer models
    K, ctx = 4, 2048
    for shape in (configs.SEVEN_B, configs.SEVENTY_B):
        t = {}
        for n in (1, 2):
            W = _oracle_weights(shape, n, 0)
            spec = _oracle_spec(shape, n)
            cache = om.new_cache(spec, 1, ctx + K + 1)
            for l in range(n):
                k, v = synth.kv_prior(shape.with_(n_layers=n), 1, l, 1, ctx)
                cache["k"][l, 0, :, :ctx] = k[0].double().numpy()
                cache["v"][l, 0, :, :ctx] = v[0].double().numpy()
            toks = synth.tokens(2, 1, K + 1, shape.vocab)
            reps, t0 = 0, time.perf_counter()
            while reps < 2 or time.perf_counter() - t0 < CPU_BASELINE_SECONDS / 2:
                om.forward_cached(spec, W, cache, toks, np.array([ctx]))
                reps += 1
            t[n] = (time.perf_counter() - t0) / reps
            del W, cache
        per_layer = t[2] - t[1]
        total = t[1] + (shape.n_layers - 1) * per_layer
        nbytes = verify_bytes(shape, 1, K, ctx)
        out["verify_" + shape.name] = {"seconds_1_layer": round(t[1], 3), "seconds_2_layers": round(t[2], 3),
                                       "seconds_per_layer": round(per_layer, 3),
                                       "seconds_extrapolated": round(total, 2),
                                       "gbs_extrapolated": round(nbytes / total / 1e9, 3),
                                       "note": "extrapolated: 1-layer time + (L - 1) x per-layer time"}
        log("%s verify: %.3f s per layer, %.1f s extrapolated (%.3f GB/s)" % (shape.name, per_layer, total,
                                                                          nbytes / total / 1e9))
    return out


def cpu_baseline_accept(inputs, B, K, seed):
    """The oracle's accept / resample (numpy, as it stands) on host copies
    of one accept-grid input set; microseconds for one call."""
    from oracle import accept as oacc
    hp, hq, hd = (x.cpu().numpy() for x in inputs)
    hu = oacc.philox_uniforms(seed, 0, B, K)
    t0 = time.perf_counter()
    oacc.accept_resample(hp, hq, hd, hu)
    return (time.perf_counter() - t0) * 1e6


def timed(fn, steps, warmup):
    import torch
    for i in range(warmup):
        fn(i)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for i in range(steps):
        fn(i)
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / steps


def sweep(args):
    """The 70B-shaped verify step over K in {1,2,3,4,6,8}, B in {1,4,16}, KV
    context in {2048, 8192}, plus the accept stage on synthetic draft/target
    pairs with perturbation sigma in {0.1, 0.5, 1.0} and the SpS tokens/s those
    acceptance rates imply with the measured draft and verify times."""
    import torch
    from paper_2302_01318_amd import configs, sps, synth
    shape, dshape = model_shapes(configs, args)
    log = lambda *a: print(*a, file=sys.stderr, flush=True)
    target = device_model(sps, synth, shape, args.seed)
    rows = []
    verify_ms = {}
    for ctx in configs.SWEEP["ctx"]:
        for B in configs.SWEEP["B"]:
            T_cap = round_up(ctx + max(configs.SWEEP["K"]) + 1, 32)
            need = sps.lib.sps_kv_bytes(__import__("ctypes").byref(sps.config_of(shape)), B, T_cap)
            free = torch.cuda.mem_get_info()[0]
            if need + (4 << 30) > free:
                for K in configs.SWEEP["K"]:
                    rows.append({"ctx": ctx, "B": B, "K": K, "status": "OOM",
                                 "kv_gb": round(need / 1e9, 1), "free_gb": round(free / 1e9, 1)})
                log("ctx %d B %d: KV %.1f GB does not fit (%.1f GB free)" % (ctx, B, need / 1e9, free / 1e9))
                continue
            kv = sps.KVCache(shape, B, T_cap)
            kv.buf.view(torch.bfloat16).normal_()
            kv.lengths.fill_(ctx)
            for K in configs.SWEEP["K"]:
                p, _, drafts = synth.accept_case_device(args.seed + K, B, K, shape.vocab)
                first = torch.randint(0, shape.vocab, (B, 1), device="cuda", dtype=torch.int32)
                tokens = torch.cat([first, drafts], dim=1).contiguous()
                ws = sps.workspace(shape, B, K + 1, T_cap)
                out = torch.empty((B, K + 1), dtype=torch.int32, device="cuda")
                nacc = torch.empty(B, dtype=torch.int32, device="cuda")
                ms = timed(lambda i: sps.verify_step(target, kv, tokens, K, 1.0, ws, p_draft=p, rng=(args.seed, i),
                                                     out_tokens=out, n_accepted=nacc), 5, 2)
                nbytes = verify_bytes(shape, B, K, ctx)
                rows.append({"ctx": ctx, "B": B, "K": K, "status": "ok", "ms": round(ms, 3),
                             "gbs": round(nbytes / (ms * 1e-3) / 1e9, 1),
                             "frac": round(nbytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                             "tokens_scored_per_s": round(B * (K + 1) / (ms * 1e-3), 1)})
                verify_ms[(ctx, B, K)] = ms
                log("ctx %5d B %2d K %d: %.3f ms, %.0f GB/s" % (ctx, B, K, ms, rows[-1]["gbs"]))
                del ws, p, tokens
            del kv
            torch.cuda.empty_cache()
    # draft time per token (B = 1, ctx 2048)
    draft = device_model(sps, synth, dshape, args.seed + 10)
    T_cap = round_up(2048 + 16, 32)
    kvd = sps.KVCache(dshape, 1, T_cap)
    kvd.buf.view(torch.bfloat16).normal_()
    kvd.lengths.fill_(2048)
    wsd = sps.workspace(dshape, 1, 2, T_cap)
    ctx_tok = torch.randint(0, shape.vocab, (1, 2), device="cuda", dtype=torch.int32)
    draft_ms = {}
    for K in configs.SWEEP["K"]:
        toks = torch.empty((1, K + 1), dtype=torch.int32, device="cuda")
        pbuf = torch.empty((1, K, shape.vocab), device="cuda")
        draft_ms[K] = timed(lambda i: sps.draft_step(draft, kvd, ctx_tok, K, 1.0, (args.seed, i), toks, pbuf, wsd),
                            5, 2)
        log("draft step K %d: %.3f ms" % (K, draft_ms[K]))
    # accept stage acceptance for sigma_pert, and the implied SpS tokens/s at B = 1, ctx 2048
    proj = []
    for sig in configs.SWEEP["sigma_pert"]:
        for K in configs.SWEEP["K"]:
            Bs = 256
            p, q, drafts = synth.accept_case_device(args.seed + 100 + K, Bs, K, shape.vocab, 2.0, sig)
            _, nacc = sps.accept_resample(p, q, drafts, None, (args.seed, 7))
            a = float(nacc.float().mean().item())
            t_loop = draft_ms[K] + verify_ms[(2048, 1, K)]
            proj.append({"sigma_pert": sig, "K": K, "mean_accepted": round(a, 3),
                         "tokens_per_loop": round(a + 1, 3), "loop_ms": round(t_loop, 3),
                         "sps_tokens_per_s": round((a + 1) / (t_loop * 1e-3), 1)})
    return {"verify": rows, "draft_ms": {str(k): round(v, 3) for k, v in draft_ms.items()}, "projection": proj,
            "note": "SpS tokens/s projected from measured draft-step and verify-step times and the acceptance "
                    "the GPU accept kernel measures on synthetic pairs (z_q ~ N(0,4), z_p = z_q + N(0, sigma^2))"}


def draft_step_bench(args):
    """The draft side of one SpS loop: sps_draft_step (K draft tokens, each a
    forward of the 3072-wide, 24-layer draft over its pending tokens plus the
    softmax and draw) for B sequences at KV context ctx, with bf16 and with
    weight-only FP8 projections. Algorithmic bytes per draft token: the
    draft's weights once plus the KV cache it reads (verify_bytes with no
    lookahead); the first forward of a step runs two pending tokens. The
    draft's weights follow --weights."""
    import torch
    from paper_2302_01318_amd import configs, sps, synth
    log = lambda *a: print(*a, file=sys.stderr, flush=True)
    B, K, ctx = args.B, args.K, args.ctx
    rows = []
    for w in (args.weights,):
        dshape = configs.DRAFT_70B if w == "bf16" else configs.DRAFT_70B.with_(dtype="fp8")
        draft = device_model(sps, synth, dshape, args.seed + 10)
        T_cap = round_up(ctx + K + 2, 32)
        kv = sps.KVCache(dshape, B, T_cap)
        kv.buf.view(torch.bfloat16).normal_()
        kv.lengths.fill_(ctx)
        ws = sps.workspace(dshape, B, 2, T_cap)
        pending = torch.randint(0, dshape.vocab, (B, 2), device="cuda", dtype=torch.int32)
        toks = torch.empty((B, K + 1), dtype=torch.int32, device="cuda")
        pbuf = torch.empty((B, K, dshape.vocab), device="cuda")
        ms = timed(lambda i: sps.draft_step(draft, kv, pending, K, args.temperature, (args.seed, i), toks, pbuf, ws,
                                            top_k=args.top_k, top_p=args.top_p), args.steps, args.warmup)
        assert sps.device_error() == 0
        nbytes = verify_bytes(dshape, B, 0, ctx)
        gbs = nbytes / (ms / K * 1e-3) / 1e9
        rows.append({"weights": w, "ms_per_step": round(ms, 4), "ms_per_token": round(ms / K, 4),
                     "bytes_per_token": nbytes, "gbs": round(gbs, 1), "frac": round(gbs / HBM_PEAK_GBS, 4)})
        log("draft %s: %.3f ms per step of %d tokens, %.3f ms per token, %.0f GB/s" % (w, ms, K, ms / K, gbs))
        del draft, kv, ws
        torch.cuda.empty_cache()
    return {"metric": "draft step ms per draft token", "draft": configs.DRAFT_70B.name, "B": B, "K": K,
            "ctx": ctx, "temperature": args.temperature, "top_k": args.top_k, "top_p": args.top_p,
            "steps": args.steps, "warmup": args.warmup, "rows": rows}


def k_study(args):
    """Time to generate n_new tokens with SpS against K (a Figure 1
    analogue): the 70B target and the 3072-wide draft built as a coupled
    pair (synth.coupled_device_weights) whose draft logits are the target's
    plus N(0, code_pert^2) per entry; every point is `reps` real generations
    of n_new tokens from random prompts, each timed end to end (prefill
    excluded), against ArS on the same target and prompts."""
    import torch
    from paper_2302_01318_amd import configs, sps, synth
    st = configs.K_STUDY
    shape, dshape = model_shapes(configs, args)
    log = lambda *a: print(*a, file=sys.stderr, flush=True)
    Ks = [int(k) for k in args.k_study_K.split(",")] if args.k_study_K else list(st["K"])
    perts = [float(x) for x in args.k_study_pert.split(",")] if args.k_study_pert else list(st["code_pert"])
    reps = args.reps or st["reps"]
    n_new, plen = st["n_new"], st["prompt"]

    coupled = lambda shp, seed, pert, into=None: coupled_model(sps, synth, shp, seed, pert, st, into)

    target = coupled(shape, args.seed + 1, 0.0)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(args.seed + 5)
    prompts = [torch.randint(0, shape.vocab, (1, plen), generator=gen, device="cuda", dtype=torch.int32)
               for _ in range(reps)]
    T_cap = round_up(plen + n_new + 2 * (max(Ks) + 1), 32)

    def generations(draft, K):
        g = sps.Generator(target, draft, 1, T_cap, K)
        # Untimed warm-up on the timed runs' code path (accepted_log included:
        # its per-loop device ops are kernels too): first launches load code
        # objects.
        g.prefill(prompts[0])
        g.run(2 * (K + 1), args.temperature, args.seed + 999, accepted_log=[], top_k=args.top_k, top_p=args.top_p)
        times, accepted, loops = [], [], 0
        for r in range(reps):
            g.prefill(prompts[r])
            torch.cuda.synchronize()
            acc_log = []
            t0 = time.perf_counter()
            g.run(n_new, args.temperature, args.seed + 1000 * r + K, accepted_log=acc_log, top_k=args.top_k,
                  top_p=args.top_p)
            torch.cuda.synchronize()
            times.append(time.perf_counter() - t0)
            loops += g.loops
            accepted += [int(a[0]) for a, done in acc_log if not bool(done[0])]
        assert sps.device_error() == 0
        ts = sorted(times)
        q = lambda f: ts[min(len(ts) - 1, int(round(f * (len(ts) - 1))))]
        mean = sum(ts) / len(ts)
        return {"K": K, "reps": reps, "loops": loops, "mean_accepted": round(sum(accepted) / max(1, len(accepted)), 3),
                "accept_rate_per_draft": round(sum(accepted) / max(1, K * len(accepted)), 3) if K else None,
                "loop_ms": round(1e3 * sum(times) / loops, 3),
                "ms_per_token": round(1e3 * mean / n_new, 3),
                "time_s": {"mean": round(mean, 4), "std": round((sum((t - mean) ** 2 for t in ts) / len(ts)) ** 0.5, 4),
                           "p50": round(q(0.5), 4), "p90": round(q(0.9), 4), "max": round(ts[-1], 4)}}

    ars = generations(None, 0)
    log("ArS: %.2f ms/token" % ars["ms_per_token"])
    rows = []
    draft = None
    for i, sd in enumerate(perts):
        draft = coupled(dshape, args.seed + 2 + i, sd, draft)   # one set of draft buffers (see coupled_model)
        for K in Ks:
            r = generations(draft, K)
            r["code_pert"] = sd
            r["speedup_vs_ars"] = round(ars["ms_per_token"] / r["ms_per_token"], 3)
            rows.append(r)
            log("draft pert %.2f K %d: accepted %.2f per loop, %.2f ms/token, %.2fx ArS, time-to-%d p50 %.3f "
                "p90 %.3f s" % (sd, K, r["mean_accepted"], r["ms_per_token"], r["speedup_vs_ars"], n_new,
                                r["time_s"]["p50"], r["time_s"]["p90"]))
    del draft
    torch.cuda.empty_cache()
    return {"k_study": rows, "ars": ars, "layer_std": st["layer_std"], "prompt": plen,
            "n_new": n_new, "temperature": args.temperature, "top_k": args.top_k, "top_p": args.top_p,
            "target_weights": shape.dtype, "draft_weights": dshape.dtype,
            "note": "coupled synthetic pair: shared rank-%d bigram skip path, target logit spread %.1f, draft logits "
                    "= target logits + N(0, code_pert^2); times are wall-clock per generation of n_new tokens after "
                    "prefill" % (st["rank"], st["logit_std"])}


def accept_grid(args):
    """Accept/resample alone: V 32000, K in {1,2,4,8}, B in {1,8,64}, Philox
    uniforms drawn in the kernel; inputs resident in HBM, four input sets
    used in turn."""
    import torch
    from paper_2302_01318_amd import configs, sps, synth
    g = configs.ACCEPT_GRID
    rows = []
    for K in g["K"]:
        for B in g["B"]:
            # 4 input sets used in turn, so that the 256 MB MALL cannot serve a repeat
            sets = [synth.accept_case_device(args.seed + K * 100 + B + 7 * j, B, K, g["V"], g["sigma"],
                                             g["sigma_pert"]) for j in range(4)]
            out = torch.empty((B, K + 1), dtype=torch.int32, device="cuda")
            nacc = torch.empty(B, dtype=torch.int32, device="cuda")
            ms = timed(lambda i: sps.accept_resample(sets[i % 4][0], sets[i % 4][1], sets[i % 4][2], None,
                                                     (args.seed, i), out, nacc), 52, 4)
            naive = B * (2 * K + 1) * g["V"] * 4
            needed = B * (2 * g["V"] * 4 + 2 * K * 4 + (K + 1) * 4 + 4)
            cpu_us = cpu_baseline_accept(sets[0], B, K, args.seed)
            rows.append({"B": B, "K": K, "us": round(ms * 1e3, 2), "cpu_baseline_us": round(cpu_us, 1),
                         "gbs_needed_bytes": round(needed / (ms * 1e-3) / 1e9, 1),
                         "naive_bytes": naive, "needed_bytes": needed,
                         "mean_accepted": round(float(nacc.float().mean().item()), 3)})
            print("B %2d K %d: %.2f us" % (B, K, ms * 1e3), file=sys.stderr, flush=True)
    return {"accept": rows,
            "note": "needed bytes: one target row and one draft row of V fp32 per sequence (the residual or "
                    "bonus draw) plus the 2K gathered probabilities; naive: every p and q row; cpu_baseline_us: "
                    "the oracle (numpy, as it stands) on host copies of the same inputs, one call"}


def softmax_rows(args):
    """sps_softmax alone (one work-group per row) on 5 rows of 32000 logits
    ~ N(0, 2^2), the verify step's row count at K = 4: plain, nucleus 0.8
    and top-k 50 at --temperature; four input sets used in turn."""
    import torch
    from paper_2302_01318_amd import sps
    rows, V = 5, 32000
    gen = torch.Generator(device="cuda")
    gen.manual_seed(args.seed)
    sets = [torch.randn((rows, V), generator=gen, device="cuda") * 2.0 for _ in range(4)]
    out = torch.empty((rows, V), device="cuda")
    res = []
    for name, k, p in (("plain", 0, 1.0), ("nucleus 0.8", 0, 0.8), ("top-k 50", 50, 1.0)):
        ms = timed(lambda i: sps.softmax(sets[i % 4], args.temperature, k, p, out), 50, 5)
        assert sps.device_error() == 0
        res.append({"setting": name, "top_k": k, "top_p": p, "us": round(ms * 1e3, 2)})
        print("softmax %s: %.2f us" % (name, ms * 1e3), file=sys.stderr, flush=True)
    return {"metric": "sps_softmax us per call", "rows": rows, "V": V, "temperature": args.temperature,
            "softmax": res}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--K", type=int, default=4)
    ap.add_argument("--B", type=int, default=1)
    ap.add_argument("--ctx", type=int, default=2048)
    ap.add_argument("--n-new", type=int, default=128)
    ap.add_argument("--shape", default="70b", choices=["70b", "7b"])
    ap.add_argument("--weights", default="bf16", choices=["bf16", "fp8"],
                    help="projection weights of target and draft: bf16, or weight-only FP8 (E4M3)")
    ap.add_argument("--draft-weights", default=None, choices=["bf16", "fp8"],
                    help="the draft's projections (default: as --weights); for --k-study")
    ap.add_argument("--no-e2e", action="store_true")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--temperature", type=float, default=1.0)
    ap.add_argument("--top-k", type=int, default=0, help="top-k modifier of p and q (0: off)")
    ap.add_argument("--top-p", type=float, default=1.0, help="nucleus modifier of p and q (1: off)")
    ap.add_argument("--sweep", action="store_true", help="70B verify over K, B, ctx (+ accept-stage projection)")
    ap.add_argument("--accept-grid", action="store_true", help="accept/resample alone over the B x K grid")
    ap.add_argument("--cpu-oracle", action="store_true",
                    help="the oracle's CPU time: tiny pair end to end, 7B and 70B verify (extrapolated)")
    ap.add_argument("--softmax", action="store_true",
                    help="sps_softmax alone on 5 x 32000 rows: plain, nucleus 0.8, top-k 50")
    ap.add_argument("--draft-step", action="store_true",
                    help="the draft side alone: K draft tokens per step (draft weights per --weights)")
    ap.add_argument("--k-study", action="store_true",
                    help="SpS generation time vs K on a coupled 70B / draft pair (acceptance set by the draft's "
                         "logit perturbation)")
    ap.add_argument("--k-study-pert", default=None,
                    help="comma-separated draft logit perturbations for --k-study (default: the configured ones)")
    ap.add_argument("--k-study-K", default=None, help="comma-separated K values for --k-study")
    ap.add_argument("--reps", type=int, default=None, help="generations per point for --k-study")
    ap.add_argument("--ingest", nargs="+", default=None, metavar=("KIND", "CSV"),
                    help="write profiles/gemm_KIND[_fp8].json from rocprofv3 CSVs of this benchmark: "
                         "'traffic FETCH.csv WRITE.csv', 'mfma COUNTERS.csv' or 'trace KERNEL_TRACE.csv'")
    ap.add_argument("--no-roofline-pass", action="store_true",
                    help="skip the second pass that times every GEMM launch with events")
    args = ap.parse_args()
    if args.ingest:
        ingest_profiles(args)
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures the verify step on one GPU; there is no multi-GPU path "
              "(requested --gpus %d)" % args.gpus, file=sys.stderr)
        sys.exit(2)

    if args.cpu_oracle:
        print(json.dumps(cpu_oracle(args)), flush=True)
        return
    if args.sweep or args.accept_grid or args.k_study or args.draft_step or args.softmax:
        res = (sweep(args) if args.sweep else accept_grid(args) if args.accept_grid else
               draft_step_bench(args) if args.draft_step else softmax_rows(args) if args.softmax else
               k_study(args))
        print(json.dumps(res), flush=True)
        return

    import torch
    from paper_2302_01318_amd import configs, sps, synth

    shape, dshape = model_shapes(configs, args)
    B, K, ctx = args.B, args.K, args.ctx
    log = lambda *a: print(*a, file=sys.stderr, flush=True)

    # A plain copy of known size: its FETCH_SIZE / WRITE_SIZE counters scale the
    # counters of the library's kernels to HBM bytes (rocprofv3 --pmc runs).
    src = torch.empty(CALIBRATION_BYTES // 4, dtype=torch.float32, device="cuda").fill_(1.0)
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    del src, dst

    t0 = time.time()
    target = device_model(sps, synth, shape, args.seed)
    torch.cuda.synchronize()
    log("target packed: %.1f GB in %.1f s" % (target.packed.numel() / 1e9, time.time() - t0))
    read_gbs = stream_read_rate(sps, torch, target.packed)
    log("streaming read ceiling: %.1f GB/s" % read_gbs)

    # ---- verify step: timed region -------------------------------------------------
    T_cap = round_up(ctx + K + 1, 32)
    kv = sps.KVCache(shape, B, T_cap)
    kv.buf.view(torch.bfloat16).normal_()          # random prior keys / values
    kv.lengths.fill_(ctx)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(args.seed + 1)
    p, _, drafts = synth.accept_case_device(args.seed + 2, B, K, shape.vocab)
    first = torch.randint(0, shape.vocab, (B, 1), generator=gen, device="cuda", dtype=torch.int32)
    tokens = torch.cat([first, drafts], dim=1).contiguous()
    ws = sps.workspace(shape, B, K + 1, T_cap)
    out = torch.empty((B, K + 1), dtype=torch.int32, device="cuda")
    nacc = torch.empty(B, dtype=torch.int32, device="cuda")

    T, top_k, top_p = args.temperature, args.top_k, args.top_p

    def step(i):
        sps.verify_step(target, kv, tokens, K, T, ws, p_draft=p, rng=(args.seed, i), out_tokens=out,
                        n_accepted=nacc, top_k=top_k, top_p=top_p)

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    # One event between consecutive steps: the window gives the mean, the
    # per-step intervals the spread.
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    ev[0].record()
    for i in range(args.steps):
        step(i)
        ev[i + 1].record()
    torch.cuda.synchronize()
    ms = ev[0].elapsed_time(ev[-1]) / args.steps
    per_step = sorted(ev[i].elapsed_time(ev[i + 1]) for i in range(args.steps))
    pct = lambda f: per_step[min(len(per_step) - 1, int(round(f * (len(per_step) - 1))))]
    nbytes = verify_bytes(shape, B, K, ctx)
    gbs = nbytes / (ms * 1e-3) / 1e9
    log("verify step: %.3f ms, %.1f GB/s (%.1f%% of %.0f GB/s)" % (ms, gbs, 100 * gbs / HBM_PEAK_GBS, HBM_PEAK_GBS))

    # ---- roofline of the weight-streaming GEMM (events around every launch) --------
    roofline = None
    if not args.no_roofline_pass:
        sps.profile_gemm_begin(GEMM_REPEATS)
        for i in range(args.steps):
            step(i)
        g_ms, g_n, g_bytes = sps.profile_gemm_end()
        assert sps.device_error() == 0
        g_avg_ms = g_ms / g_n
        g_gbs = (g_bytes / g_n) / (g_avg_ms * 1e-3) / 1e9
        log("gemm: %d launches, avg %.1f us, %.1f GB/s" % (g_n, g_avg_ms * 1e3, g_gbs))
        prof = profiled_figures(args.shape, args.weights, B, K, ctx)
        roofline = {"bound": "hbm", "kernel": "gemm_kernel (weight-streaming skinny GEMM, all linear layers)",
                    "achieved": round(g_gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                    "frac": round(g_gbs / HBM_PEAK_GBS, 4), "traffic": prof["traffic"],
                    "launches_per_step": g_n // args.steps, "avg_launch_us": round(g_avg_ms * 1e3, 2),
                    "bytes_per_launch": g_bytes / g_n,
                    "frac_of_stream_read": round(g_gbs / read_gbs, 4), "mfma": prof["mfma"],
                    "trace": prof["trace"]}
    del kv, ws
    torch.cuda.empty_cache()     # the end-to-end caches differ in size from the timing cache

    # ---- SpS and ArS tokens/s end to end ---------------------------------------------
    # Two pairs: the coupled pair (draft logits = target logits + N(0, 0.5^2),
    # Sum min(p, q) ~ 0.81, the acceptance regime of the paper's trained
    # drafts) gives the SpS figure; the verify-timing target with an
    # unrelated random-init draft (they rarely agree) is reported beside it.
    e2e = {}
    if not args.no_e2e and args.shape == "70b":
        prompt = torch.randint(0, shape.vocab, (B, ctx), generator=gen, device="cuda", dtype=torch.int32)
        Tc = round_up(ctx + args.n_new + 2 * (K + 1), 32)

        def pair_run(tgt, dm, label, ars=True):
            out = {}
            for name, d_, k in (("sps", dm, K), ("ars", None, 0))[:2 if ars else 1]:
                g = sps.Generator(tgt, d_, B, Tc, k)
                # An untimed short generation first, on the timed run's code
                # path (accepted_log included: its per-loop device ops are
                # kernels too): the first launch of each kernel loads its code
                # object (up to ~0.16 s), which would otherwise land inside the
                # timed run.
                g.prefill(prompt)
                g.run(2 * (k + 1), T, args.seed + 999, accepted_log=[], top_k=top_k, top_p=top_p)
                g.prefill(prompt)
                torch.cuda.synchronize()
                acc_log = []
                t0 = time.perf_counter()
                g.run(args.n_new, T, args.seed, accepted_log=acc_log, top_k=top_k, top_p=top_p)
                torch.cuda.synchronize()
                dt = time.perf_counter() - t0
                accs = [int(a[0]) for a, done in acc_log if not bool(done[0])]
                out[name] = {"tokens_per_s": B * args.n_new / dt, "loops": g.loops, "seconds": dt,
                             "mean_accepted": sum(accs) / max(1, len(accs))}
                log("%s %s: %.1f tokens/s, %d loops, mean accepted %.2f" % (label, name, out[name]["tokens_per_s"],
                                                                            g.loops, out[name]["mean_accepted"]))
                del g
            assert sps.device_error() == 0
            return out

        t0 = time.time()
        draft = device_model(sps, synth, dshape, args.seed + 10)
        torch.cuda.synchronize()
        log("draft packed: %.1f GB in %.1f s" % (draft.packed.numel() / 1e9, time.time() - t0))
        e2e["unrelated"] = pair_run(target, draft, "unrelated pair")
        st = configs.K_STUDY
        coupled = lambda shp, seed, pert, into: coupled_model(sps, synth, shp, seed, pert, st, into)
        # The coupled pair goes into the same device buffers (see coupled_model).
        target = coupled(shape, args.seed + 1, 0.0, target)
        draft = coupled(dshape, args.seed + 2, E2E_CODE_PERT, draft)
        e2e["coupled"] = pair_run(target, draft, "coupled pair")
        if dshape.dtype != "fp8":
            # The same coupled pair with the draft's projections in weight-only
            # FP8: half the draft's bytes per token. The accepted tokens still
            # follow the bf16 target exactly (any draft does); only the
            # acceptance rate and the draft time change.
            draft8 = coupled(dshape.with_(dtype="fp8"), args.seed + 2, E2E_CODE_PERT, None)
            e2e["coupled_fp8_draft"] = pair_run(target, draft8, "coupled pair, fp8 draft", ars=False)
            del draft8
        del draft
        torch.cuda.empty_cache()

    result = {
        "metric": METRIC, "value": round(gbs, 1), "unit": "GB/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16",
        "weights": "fp8 e4m3, one fp32 scale per output row (exact bf16 conversion before the MFMA)"
                   if args.weights == "fp8" else "bf16",
        "data": "synthetic: verify timing on random-init weights N(0,0.02), random bf16 prior KV, random tokens "
                "and draft distributions; end to end on a seeded coupled target/draft pair (see e2e.pair)",
        "config": {"workload": "%s-shaped target verify step + softmax + fused accept/resample" % shape.name,
                   "K": K, "batch": B, "ctx": ctx, "temperature": T, "top_k": top_k, "top_p": top_p,
                   "bytes_per_step": nbytes,
                   "hbm_frac": round(gbs / HBM_PEAK_GBS, 4)},
        "stream_read_gbs": round(read_gbs, 1),
        "verify_frac_of_stream_read": round(gbs / read_gbs, 4),
        "verify_ms": round(ms, 4),
        "verify_ms_p10_median_p90": [round(pct(0.1), 4), round(pct(0.5), 4), round(pct(0.9), 4)],
    }
    if roofline is not None:
        result["roofline"] = roofline
    if e2e:
        c, u = e2e["coupled"], e2e["unrelated"]
        result["sps_tokens_per_s"] = round(c["sps"]["tokens_per_s"], 2)
        result["ars_tokens_per_s"] = round(c["ars"]["tokens_per_s"], 2)
        result["e2e"] = {"draft": dshape.name, "prompt": ctx, "n_new": args.n_new, "K": K, "temperature": T,
                         "top_k": top_k, "top_p": top_p,
                         "pair": "coupled synthetic pair: draft logits = target logits + N(0, %.1f^2) "
                                 "(Sum min(p, q) ~ 0.81)" % E2E_CODE_PERT,
                         "sps_mean_accepted": round(c["sps"]["mean_accepted"], 3),
                         "sps_loops": c["sps"]["loops"], "ars_loops": c["ars"]["loops"],
                         "speedup_vs_ars": round(c["sps"]["tokens_per_s"] / c["ars"]["tokens_per_s"], 3),
                         "fp8_draft": None if "coupled_fp8_draft" not in e2e else {
                             "sps_tokens_per_s": round(e2e["coupled_fp8_draft"]["sps"]["tokens_per_s"], 2),
                             "sps_mean_accepted": round(e2e["coupled_fp8_draft"]["sps"]["mean_accepted"], 3),
                             "sps_loops": e2e["coupled_fp8_draft"]["sps"]["loops"],
                             "speedup_vs_ars": round(e2e["coupled_fp8_draft"]["sps"]["tokens_per_s"]
                                                     / c["ars"]["tokens_per_s"], 3),
                             "note": "same coupled pair, draft projections in weight-only FP8 (target bf16)"},
                         "unrelated_pair": {"sps_tokens_per_s": round(u["sps"]["tokens_per_s"], 2),
                                            "ars_tokens_per_s": round(u["ars"]["tokens_per_s"], 2),
                                            "sps_mean_accepted": round(u["sps"]["mean_accepted"], 3)},
                         "paper_context": "Chinchilla 70B on 16 TPU v4: ArS 14.1 ms/token, SpS 1.92-2.46x "
                                          "(paper Table 1); not comparable hardware"}
    if not args.no_cpu_baseline:
        del target
        torch.cuda.empty_cache()
        log("cpu baseline (oracle) ...")
        result["cpu_baseline"] = cpu_baseline(shape, K, ctx)
        log("cpu baseline: %.3f GB/s in %.1f s" % (result["cpu_baseline"]["value"],
                                                    result["cpu_baseline"]["seconds_per_sample"]))
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
