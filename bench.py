"""Benchmark of the ResNet-18 training step on one MI355X.

One step = one full training step (forward, data- and weight-gradient
convolutions, BN/ReLU/residual, softmax cross-entropy, SGD-momentum) of one
synthetic batch already resident in HBM. The headline workload is the
ImageNet-shaped ResNet-18 in bf16 at batch 256, 224x224 (the configuration
the convolution-utilisation target is stated for); every other
(batch, resolution) step shape that the CIFAR cyclic-progressive and the
ImageNet hybrid schedules visit is timed too and reported under
"per_shape", with the parameter-server merge of the hybrid rounds.

Prints ONE JSON line. Kernel-level figures come from HIP events recorded
by the library around each launch, on the stream the kernels run on, in a
separate profiled step (the timed steps run without events).
"""
import argparse
import re
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK = {"bf16": 2500.0, "fp16": 2500.0, "fp32": 157.3}     # dense MFMA TFLOP/s, MI355X published
HBM_PEAK = 8000.0                           # GB/s
MFMA_CLASSES = {"conv_fwd", "conv_dgrad", "conv_wgrad"}

# (workload name, arch, classes, precision, N, H)
HEADLINE = ("imagenet_resnet18_bf16_b256_224", "imagenet", 1000, "bf16", 256, 224)
SHAPES = [
    ("cifar_resnet18_fp32_b128_32", "cifar", 100, "fp32", 128, 32),
    ("cifar_cyclic_fp32_b512_16", "cifar", 100, "fp32", 512, 16),
    ("cifar_cyclic_fp32_b256_24", "cifar", 100, "fp32", 256, 24),
    ("cifar_cyclic_fp32_b128_32", "cifar", 100, "fp32", 128, 32),
    ("imagenet_hybrid_bf16_L1024_128", "imagenet", 1000, "bf16", 1024, 128),
    ("imagenet_hybrid_bf16_L640_160", "imagenet", 1000, "bf16", 640, 160),
    ("imagenet_hybrid_bf16_L448_192", "imagenet", 1000, "bf16", 448, 192),
    ("imagenet_hybrid_bf16_L256_224", "imagenet", 1000, "bf16", 256, 224),
    ("imagenet_hybrid_bf16_S64_128", "imagenet", 1000, "bf16", 64, 128),
    ("imagenet_hybrid_bf16_S64_160", "imagenet", 1000, "bf16", 64, 160),
    ("imagenet_hybrid_bf16_S64_192", "imagenet", 1000, "bf16", 64, 192),
    ("imagenet_hybrid_bf16_S64_224", "imagenet", 1000, "bf16", 64, 224),
]


def symbol(rec, prec):
    """Kernel instance name of a profile record, as rocprofv3 prints it (the
    library records it; namespace dropped, the bf16 storage type shown as bf16)."""
    return rec["kernel"] or rec["cls"]


def summarize(recs, prec, steps=1):
    """Per-class and per-symbol totals of profiled launches (per step)."""
    by_cls, by_sym = {}, {}
    for r in recs:
        for d, k in ((by_cls, r["cls"]), (by_sym, symbol(r, prec))):
            e = d.setdefault(k, {"ms": 0.0, "flops": 0.0, "bytes": 0.0, "launches": 0, "cls": r["cls"]})
            e["ms"] += r["ms"] / steps
            e["flops"] += r["flops"] / steps
            e["bytes"] += r["bytes"] / steps
            e["launches"] += 1.0 / steps
    conv_ms = sum(v["ms"] for k, v in by_cls.items() if k in MFMA_CLASSES)
    conv_fl = sum(v["flops"] for k, v in by_cls.items() if k in MFMA_CLASSES)
    st_ms = sum(v["ms"] for k, v in by_cls.items() if k not in MFMA_CLASSES and k != "head")
    st_by = sum(v["bytes"] for k, v in by_cls.items() if k not in MFMA_CLASSES and k != "head")
    total_ms = sum(v["ms"] for v in by_cls.values())
    out = {
        "kernel_ms": round(total_ms, 4),
        "conv_ms": round(conv_ms, 4),
        "conv_tflops": round(conv_fl / conv_ms / 1e9, 2) if conv_ms > 0 else None,
        "conv_mfma_frac": round(conv_fl / conv_ms / 1e9 / PEAK[prec], 4) if conv_ms > 0 else None,
        "stream_ms": round(st_ms, 4),
        "stream_GBps": round(st_by / st_ms / 1e6, 1) if st_ms > 0 else None,
        "stream_hbm_frac": round(st_by / st_ms / 1e6 / HBM_PEAK, 4) if st_ms > 0 else None,
        "classes": {k: {"ms": round(v["ms"], 4), "launches": int(round(v["launches"])),
                        "TFLOPs": round(v["flops"] / v["ms"] / 1e9, 2) if v["flops"] and v["ms"] > 0 else None,
                        "GBps": round(v["bytes"] / v["ms"] / 1e6, 1) if v["bytes"] and v["ms"] > 0 else None}
                    for k, v in sorted(by_cls.items(), key=lambda kv: -kv[1]["ms"])},
    }
    return out, by_sym


def roofline(by_sym, prec, traffic_lookup):
    name, e = max(by_sym.items(), key=lambda kv: kv[1]["ms"])
    avg_ms = e["ms"] / e["launches"]
    if e["cls"] in MFMA_CLASSES:
        ach = e["flops"] / e["ms"] / 1e9
        peak, unit, bound = PEAK[prec], "TFLOP/s", "mfma"
    else:
        ach = e["bytes"] / e["ms"] / 1e6
        peak, unit, bound = HBM_PEAK, "GB/s", "hbm"
    return {"kernel": name, "bound": bound, "achieved": round(ach, 2), "peak": peak, "unit": unit,
            "frac": round(ach / peak, 4), "traffic": traffic_lookup(name),
            "launches_per_step": int(round(e["launches"])), "avg_launch_ms": round(avg_ms, 5),
            "share_of_kernel_time": None}


KERNEL_SOURCES = os.path.join(ROOT, "paper_2509_26092_amd", "csrc")
TRAFFIC_JSON = os.path.join(ROOT, "profiles", "hbm_traffic.json")
CALIB_FLOATS = 1 << 26   # ps_worker_delta over 2^26 floats: reads 512 MiB, writes 256 MiB


def kernel_source_sha():
    h = hashlib.sha256()
    for name in sorted(os.listdir(KERNEL_SOURCES)):
        if name.endswith((".hip", ".h", ".cpp")):
            h.update(name.encode())
            h.update(open(os.path.join(KERNEL_SOURCES, name), "rb").read())
    return h.hexdigest()


def traffic_lookup_factory():
    """HBM bytes per launch measured with rocprofv3 FETCH_SIZE / WRITE_SIZE,
    if a committed measurement exists for the current kernel sources."""
    try:
        with open(TRAFFIC_JSON) as f:
            tab = json.load(f)
        sha = kernel_source_sha()
    except (OSError, ValueError):
        return lambda name: None

    def look(name):
        e = tab.get("kernels", {}).get(name)
        if not e or tab.get("source_sha256") != sha:
            return None
        return e.get("bytes_per_launch")
    return look


def short_kernel_name(n):
    n = n.replace("rn18::(anonymous namespace)::", "").replace("unsigned short", "bf16").replace("void ", "")
    return re.sub(r"\(.*\)$", "", n)


def ingest_counters(fetch_csv, write_csv, command):
    """Per-kernel HBM bytes per dispatch from two rocprofv3 --pmc runs of the
    same command (FETCH_SIZE, then WRITE_SIZE, in KiB per dispatch), each
    scaled by what the counter reads for ps_worker_delta over 2^26 floats
    (a copy-like kernel of known traffic: 512 MiB read, 256 MiB written)."""
    import csv
    import collections
    def load(path, counter):
        out = collections.defaultdict(list)
        for r in csv.DictReader(open(path)):
            if r["Counter_Name"] == counter:
                out[short_kernel_name(r["Kernel_Name"])].append((int(r["Grid_Size"]), float(r["Counter_Value"])))
        return out
    fetch, write = load(fetch_csv, "FETCH_SIZE"), load(write_csv, "WRITE_SIZE")
    calib_grid = None
    cal_f = [v for g, v in fetch.get("delta_kernel", []) if v > 100000]
    cal_w = [v for g, v in write.get("delta_kernel", []) if v > 100000]
    if not cal_f or not cal_w:
        raise SystemExit("no calibration dispatch (run the counter passes with --calibrate)")
    kf = (2.0 * CALIB_FLOATS * 4 / 1024) / (sum(cal_f) / len(cal_f))   # true KiB per counted KiB
    kw = (1.0 * CALIB_FLOATS * 4 / 1024) / (sum(cal_w) / len(cal_w))
    kernels = {}
    for name in sorted(set(fetch) & set(write)):
        if name == "delta_kernel":
            continue
        f = sum(v for _, v in fetch[name]) / len(fetch[name]) * kf * 1024
        w = sum(v for _, v in write[name]) / len(write[name]) * kw * 1024
        kernels[name] = {"dispatches": len(fetch[name]), "fetch_bytes_per_launch": round(f),
                         "write_bytes_per_launch": round(w), "bytes_per_launch": round(f + w)}
    tab = {"source_sha256": kernel_source_sha(), "command": command,
           "fetch_scale": round(kf, 4), "write_scale": round(kw, 4), "kernels": kernels}
    with open(TRAFFIC_JSON, "w") as f:
        json.dump(tab, f, indent=1, sort_keys=True)
    return tab


def copy_ceiling(B, torch, n=1 << 27, reps=10):
    """HBM bandwidth that plain streaming reaches on this GPU, in bytes moved
    per second: the better of a device-to-device copy of n floats (torch's
    copy, one read and one write) and the library's ps_worker_delta over n
    floats (two reads and one write), best of `reps` runs each, on arrays
    of 512 MiB that no cache holds. It is the practical ceiling the stream
    kernels are also reported against (measured 5.0-5.4 TB/s; reads alone
    reach about 6.3)."""
    a, b, d = (torch.ones(n, device="cuda") for _ in range(3))

    def best(run, nbytes):
        run()
        torch.cuda.synchronize()
        t = None
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            run()
            e1.record()
            torch.cuda.synchronize()
            ms = e0.elapsed_time(e1)
            t = ms if t is None else min(t, ms)
        return nbytes / t / 1e6

    gbs = max(best(lambda: d.copy_(a), 8.0 * n), best(lambda: B.ps_worker_delta(a, b, d, n), 12.0 * n))
    del a, b, d
    return round(gbs, 1)


def counters_summary(csv_path, title, command):
    """Markdown table of a rocprofv3 --pmc run's SQ counters per kernel
    (averaged over its dispatches). With SQ_VALU_MFMA_BUSY_CYCLES and
    SQ_BUSY_CYCLES the MFMA busy share of the shader engines' SIMDs (32 per
    engine) is added."""
    import csv
    import collections
    per = collections.defaultdict(lambda: collections.defaultdict(list))
    for r in csv.DictReader(open(csv_path)):
        per[short_kernel_name(r["Kernel_Name"])][r["Counter_Name"]].append(float(r["Counter_Value"]))
    names = sorted({c for v in per.values() for c in v})
    lines = ["# %s" % title, "", "Command (from the repository root on the MI355X box, after "
             "`cd /tmp && export TMPDIR=/tmp`):", "", "```", command, "```", "",
             "Per-dispatch averages; MFMA busy = SQ_VALU_MFMA_BUSY_CYCLES / (SQ_BUSY_CYCLES x 32 SIMDs per "
             "shader engine).", ""]
    head = ["kernel", "dispatches"] + names + (["MFMA busy"] if "SQ_VALU_MFMA_BUSY_CYCLES" in names else [])
    lines.append("| " + " | ".join(head) + " |")
    lines.append("|---|" + "---:|" * (len(head) - 1))
    rows = []
    for k, cs in per.items():
        if k.startswith(("at::", "__amd")):
            continue
        avg = {c: sum(v) / len(v) for c, v in cs.items()}
        n = len(next(iter(cs.values())))
        row = ["`%s`" % k, str(n)] + ["%.0f" % avg.get(c, float("nan")) for c in names]
        if "SQ_VALU_MFMA_BUSY_CYCLES" in names:
            busy = avg.get("SQ_BUSY_CYCLES", 0)
            row.append("%.3f" % (avg.get("SQ_VALU_MFMA_BUSY_CYCLES", 0) / (busy * 32)) if busy else "")
        rows.append((avg.get("SQ_VALU_MFMA_BUSY_CYCLES", 0) * n, row))
    for _, row in sorted(rows, key=lambda t: -t[0]):
        lines.append("| " + " | ".join(row) + " |")
    return "\n".join(lines) + "\n"


def progress(msg):
    """A progress line on stderr (the JSON result alone goes to stdout)."""
    print("bench: " + msg, file=sys.stderr, flush=True)


def run_shape(B, torch, inputs, arch, classes, prec, N, H, steps, warmup, seed=1, dropout=0.0, serial=False):
    w = B.Worker(arch, classes, prec)
    if serial:
        B.rn18_debug_set(w.ctx, B.RN18_DBG_SERIAL, 1)
    if dropout:
        B.rn18_set_dropout(w.ctx, dropout, seed, 0)
    st = torch.zeros(w.n_state, device="cuda")
    B.rn18_destroy(B.rn18_init(w.cfg, seed, st))
    x = torch.from_numpy(inputs.images(seed, N, H, H)).cuda()
    y = torch.from_numpy(inputs.labels(seed, N, classes)).cuda()
    loss = torch.zeros(1, device="cuda")
    for _ in range(warmup):
        w.train_step(st, x, y, 0.01, loss)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        w.train_step(st, x, y, 0.01, loss)
    torch.cuda.synchronize()
    dt = (time.perf_counter() - t0) / steps
    B.rn18_profile_enable(w.ctx, True)
    w.train_step(st, x, y, 0.01, loss)
    recs = B.rn18_profile_read(w.ctx)
    B.rn18_profile_enable(w.ctx, False)
    status = w.sync_status()
    lval = float(loss.item())
    if prec == "fp16":
        # the dynamic loss scale after all steps, and how many were skipped
        scale, skipped = B.rn18_get_loss_scale(w.ctx)
        recs.append({"cls": "loss_scale", "scale": scale, "skipped": skipped, "steps": warmup + steps + 1})
    w.close()
    return dt, recs, status, lval


def merge_rate(B, torch, n, reps=20):
    p = torch.randn(n, device="cuda")
    ds = torch.randn(n, device="cuda") * 1e-3
    dl = torch.randn(n, device="cuda") * 1e-3
    for _ in range(3):
        B.ps_dual_merge(p, ds, dl, n, 0.5)
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    s.record()
    for _ in range(reps):
        B.ps_dual_merge(p, ds, dl, n, 0.5)
    e.record()
    torch.cuda.synchronize()
    ms = s.elapsed_time(e) / reps
    return ms, 16.0 * n / ms / 1e6


def dbl_plan(B, torch, inputs, by, merge_ms, steps):
    """The dual-batch planner on this GPU's measured step times: per hybrid
    resolution, a and b of t = a*x + b fitted over batches 64, B_L/2 and B_L
    (Sec. 3.2); the ImageNet split for one small and three large workers at
    k = 1.05 (Eqs. 4-6), B_S from Eq. 8, the factor d_S/d_L (Sec. 3.4); then a
    step at the planned B_S, the measured per-worker epoch times (Eq. 7 says
    they match) and a ratio-faithful round: one large step, the small worker's
    steps per large step, two deltas and the merge."""
    from paper_2509_26092_amd import planner
    d, k, n_s, n_l = 1281167, 1.05, 1, 3
    out = []
    for r, bl in ((128, 1024), (160, 640), (192, 448), (224, 256)):
        pts = [(64, by["imagenet_hybrid_bf16_S64_%d" % r]["ms_per_step"]),
               (bl, by["imagenet_hybrid_bf16_L%d_%d" % (bl, r)]["ms_per_step"])]
        half = run_shape(B, torch, inputs, "imagenet", 1000, "bf16", bl // 2, r, steps, 2)[0] * 1e3
        pts.append((bl // 2, half))
        a, b = planner.fit_linear([p[0] for p in pts], [p[1] for p in pts])
        p = planner.plan(a, b, bl, k, d, n_s, n_l, "ratio", whole_images=True)
        ts = run_shape(B, torch, inputs, "imagenet", 1000, "bf16", p["B_S"], r, steps, 2)[0] * 1e3
        tl = pts[1][1]
        spr = planner.steps_per_round(p)
        t_round = tl + spr * ts + 3 * merge_ms
        out.append({"resolution": r, "a_ms_per_image": round(a, 6), "b_ms": round(b, 4),
                    "fit_points_ms": [[x, round(t, 4)] for x, t in pts],
                    "B_L": bl, "B_S": p["B_S"], "d_L": p["d_L"], "d_S": round(p["d_S"], 1),
                    "factor": round(p["factor"], 4), "small_step_ms": round(ts, 4),
                    "small_step_predicted_ms": round(a * p["B_S"] + b, 4),
                    "epoch_s_large_measured": round(tl * p["d_L"] / bl / 1e3, 2),
                    "epoch_s_small_measured": round(ts * p["d_S"] / p["B_S"] / 1e3, 2),
                    "small_steps_per_large_step": round(spr, 3),
                    "round_ms": round(t_round, 3),
                    "round_images_per_s": round((bl + spr * p["B_S"]) / t_round * 1e3, 1)})
    return {"workload": "dbl_planner_imagenet_n4_k1.05", "n_S": n_s, "n_L": n_l, "k": k, "d": d,
            "stages": out}


def measured_rounds(B, torch, inputs, reps, factor=0.5):
    """Dual-batch rounds of the ImageNet hybrid schedule timed end to end:
    both workers pull the global state, the large worker (B_L at the stage's
    resolution) and the small worker (batch 64) take one step each, push
    their deltas, and ps_dual_merge applies them with the model-update
    factor (Sec. 3.4). 'sequential' runs everything on one stream;
    'concurrent' gives each worker its own stream (default priority), so the
    small step fills what the large one leaves of the chip, as two workers
    sharing one GPU would."""
    cfg = B.make_config("imagenet", 1000, "bf16")
    n = B.rn18_state_floats(cfg)[0]
    sa, sb = torch.cuda.Stream(), torch.cuda.Stream()
    out = []
    for r, bl in ((128, 1024), (160, 640), (192, 448), (224, 256)):
        xl = torch.from_numpy(inputs.images(11, bl, r, r)).cuda()
        yl = torch.from_numpy(inputs.labels(11, bl, 1000)).cuda()
        xs = torch.from_numpy(inputs.images(12, 64, r, r)).cuda()
        ys = torch.from_numpy(inputs.labels(12, 64, 1000)).cuda()
        row = {"resolution": r, "B_L": bl, "B_S": 64, "factor": factor}
        for mode in ("sequential", "concurrent"):
            s2 = sb if mode == "concurrent" else sa
            g = torch.zeros(n, device="cuda")
            B.rn18_destroy(B.rn18_init(cfg, 1, g))
            with torch.cuda.stream(sa):
                wl = B.Worker("imagenet", 1000, "bf16")
            with torch.cuda.stream(s2):
                wsm = B.Worker("imagenet", 1000, "bf16")
            sl, ss, dl, ds = (torch.empty_like(g) for _ in range(4))
            ll, ls = torch.zeros(1, device="cuda"), torch.zeros(1, device="cuda")
            torch.cuda.synchronize()

            def one_round():
                e = torch.cuda.Event()
                e.record(sa)                      # the merged global state
                with torch.cuda.stream(sa):
                    sl.copy_(g)
                    wl.train_step(sl, xl, yl, 0.01, ll)
                s2.wait_event(e)
                with torch.cuda.stream(s2):
                    ss.copy_(g)
                    wsm.train_step(ss, xs, ys, 0.01, ls)
                sa.wait_stream(s2)
                with torch.cuda.stream(sa):
                    B.ps_worker_delta(g, sl, dl, n)
                    B.ps_worker_delta(g, ss, ds, n)
                    B.ps_dual_merge(g, ds, dl, n, factor)

            for _ in range(2):
                one_round()
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            for _ in range(reps):
                one_round()
            torch.cuda.synchronize()
            ms = (time.perf_counter() - t0) / reps * 1e3
            status = max(abs(wl.sync_status()), abs(wsm.sync_status()))
            wl.close()
            wsm.close()
            row[mode] = {"round_ms": round(ms, 3), "round_images_per_s": round((bl + 64) / ms * 1e3, 1),
                         "status": status}
        progress("rounds at %d: sequential %.3f ms, concurrent %.3f ms"
                 % (r, row["sequential"]["round_ms"], row["concurrent"]["round_ms"]))
        out.append(row)
    return {"workload": "dbl_rounds_measured_imagenet_bf16", "stages": out}


def memory_model(B, torch):
    """Sec. 5.3: device memory of steps at B = 64..512 (hipMemGetInfo), the
    Eq. 9 fit, the largest batch for this GPU's memory, the library's own
    bound from its 32-bit tensor indexing, and the model checked against a
    measured step at 90% of the smaller of the two (the rest of the memory
    is left to the runtime and the allocator)."""
    from paper_2509_26092_amd import memory as Mm
    _, m_gpu = torch.cuda.mem_get_info()
    out = []
    for wl, arch, classes, prec, H in (("cifar100_fp32_32", "cifar", 100, "fp32", 32),
                                       ("imagenet_bf16_224", "imagenet", 1000, "bf16", 224)):
        bs = [64, 128, 192, 256, 320, 384, 448, 512]
        ms = Mm.profile(B, torch, arch, classes, prec, H, bs)
        p, a = Mm.fit(bs, ms)
        b_mem = Mm.max_batch(p, a, m_gpu)
        w = B.Worker(arch, classes, prec)
        b_addr = Mm.addressing_max_batch(B, w.ctx, H, H)
        w.close()
        b_v = int(0.9 * min(b_mem, b_addr))
        try:
            used, status = Mm.measure_step(B, torch, arch, classes, prec, b_v, H)
        except (RuntimeError, B.Rn18Error) as ex:      # out of memory: reported, not fatal to the bench
            progress("memory model %s: step at B=%d failed: %s" % (wl, b_v, ex))
            out.append({"workload": wl, "fit_batches": bs, "B_max_memory": b_mem, "B_max_addressing": b_addr,
                        "verified_at": b_v, "error": str(ex)[:200]})
            continue
        pred = Mm.predict(p, a, b_v)
        progress("memory model %s: B_max %d (memory) / %d (addressing), error %.4f at B=%d"
                 % (wl, b_mem, b_addr, abs(pred - used) / used, b_v))
        out.append({"workload": wl, "fit_batches": bs, "measured_GB": [round(m / 1e9, 3) for m in ms],
                    "sum_p_GB": round(p / 1e9, 4), "sum_a_MB_per_image": round(a / 1e6, 4),
                    "M_GPU_GB": round(m_gpu / 1e9, 2), "B_max_memory": b_mem, "B_max_addressing": b_addr,
                    "verified_at": b_v, "measured_at_verified_GB": round(used / 1e9, 3),
                    "predicted_at_verified_GB": round(pred / 1e9, 3),
                    "relative_error": round(abs(pred - used) / used, 5), "status": status})
    return {"workload": "memory_model_eq9", "configs": out}


def host_info():
    """CPU model, logical CPUs visible to this process and the BLAS thread count."""
    model = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        threads = os.cpu_count()
    try:
        visible = len(os.sched_getaffinity(0))
    except AttributeError:
        visible = os.cpu_count()
    return model, visible, threads


# train GFLOP per image of the workload's net (real channels): ImageNet at 224,
# CIFAR at 32; other resolutions scale with the pixel count
_GFLOP_IMG = {"imagenet": (10.648, 224), "cifar": (3.329, 32), "tiny": (0.0075, 16)}


def cpu_sample_images(arch, H, N, budget_gflop=60.0):
    """Images of a bounded oracle sample of a step shape: about budget_gflop
    of training work (a few seconds of fp64 on the host), at least 2, at
    most the batch."""
    g, h0 = _GFLOP_IMG[arch]
    per = g * (H / h0) ** 2
    return max(2, min(N, int(round(budget_gflop / per))))


def cpu_baseline(arch, classes, prec, H, n_img, seed=3, reps=3):
    """The fp64 oracle's training step, timed on the host cores on a bounded
    sample of the workload (n_img images at the workload's resolution): the
    median of `reps` steps (one if a step takes 60 s or more)."""
    import numpy as np
    from oracle import net
    from paper_2509_26092_amd import inputs
    model, visible, threads = host_info()
    L = net.Layout(arch, classes)
    cfg = net.Config(arch, classes, bf16=(prec == "bf16"))
    st = net.init_state(L, seed)
    x = inputs.images(seed, n_img, H, H)
    y = inputs.labels(seed, n_img, classes)
    times = []
    for _ in range(reps):
        t0 = time.perf_counter()
        net.train_step(cfg, L, st, np.zeros(L.n_trainable), x, y, 0.01)
        times.append(time.perf_counter() - t0)
        if times[-1] >= 60.0:
            break
    dt = float(np.median(times))
    return {"value": round(n_img / dt, 3), "unit": "images/s", "cores": threads, "kind": "oracle",
            "s_per_step_sample": round(dt, 3),
            "sample": "fp64 oracle training step of %d images at %dx%d (%s %s net), median of %d: %.2f s; "
                      "%d BLAS threads, %d logical CPUs visible, %s" % (n_img, H, H, arch, prec, len(times), dt,
                                                                       threads, visible, model)}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--shape-steps", type=int, default=8, help="timed steps per additional step shape")
    ap.add_argument("--headline-only", action="store_true")
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--serial", action="store_true",
                    help="keep every launch of the headline steps on one stream (no weight-gradient overlap), so "
                         "that a kernel trace times each kernel alone, as the profiled step does")
    ap.add_argument("--cpu-images", type=int, default=20)
    ap.add_argument("--traffic-from", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="write profiles/hbm_traffic.json from the counter_collection.csv files of a FETCH_SIZE "
                         "and a WRITE_SIZE rocprofv3 --pmc run of this script with --calibrate, then exit")
    ap.add_argument("--counters-summary", nargs=3, metavar=("CSV", "OUT_MD", "TITLE"),
                    help="write a per-kernel markdown summary of a rocprofv3 --pmc counter_collection.csv "
                         "(the command recorded with --traffic-command), then exit")
    ap.add_argument("--traffic-command", default="",
                    help="the command the counter runs used, recorded with --traffic-from")
    ap.add_argument("--no-ceiling", action="store_true",
                    help="skip the HBM copy-ceiling measurement (for kernel-trace runs of the step)")
    ap.add_argument("--calibrate", action="store_true",
                    help="also run ps_worker_delta over 2^26 floats (reads 512 MiB, writes 256 MiB) as the "
                         "known-size kernel that scales HBM counters")
    args = ap.parse_args()
    if args.counters_summary:
        csv_path, out_md, title = args.counters_summary
        with open(out_md, "w") as f:
            f.write(counters_summary(csv_path, title, args.traffic_command))
        return
    if args.traffic_from:
        tab = ingest_counters(args.traffic_from[0], args.traffic_from[1], args.traffic_command)
        print(json.dumps({"fetch_scale": tab["fetch_scale"], "write_scale": tab["write_scale"],
                          "kernels": len(tab["kernels"])}))
        return
    if args.gpus != 1:
        print("bench.py runs on one GPU only: this build has no multi-GPU path (the parameter-server merge is "
              "simulated on one GPU); run with --gpus 1", file=sys.stderr)
        sys.exit(2)
    import torch
    from paper_2509_26092_amd import binding as B
    from paper_2509_26092_amd import inputs
    torch.cuda.set_device(0)
    look = traffic_lookup_factory()

    name, arch, classes, prec, N, H = HEADLINE
    dt, recs, status, lval = run_shape(B, torch, inputs, arch, classes, prec, N, H, args.steps, args.warmup,
                                       serial=args.serial)
    head_sum, by_sym = summarize(recs, prec)
    roof = roofline(by_sym, prec, look)
    roof["share_of_kernel_time"] = round(by_sym[roof["kernel"]]["ms"] / head_sum["kernel_ms"], 4)

    per_shape = []
    if not args.headline_only:
        for sname, sarch, scls, sprec, sN, sH in SHAPES:
            sdt, srecs, sstatus, _ = run_shape(B, torch, inputs, sarch, scls, sprec, sN, sH, args.shape_steps, 2)
            progress("%s: %.3f ms/step" % (sname, sdt * 1e3))
            ssum, _ = summarize(srecs, sprec)
            per_shape.append({"workload": sname, "batch": sN, "resolution": sH, "dtype": sprec,
                              "images_per_s": round(sN / sdt, 1), "ms_per_step": round(sdt * 1e3, 3),
                              "conv_tflops": ssum["conv_tflops"], "conv_mfma_frac": ssum["conv_mfma_frac"],
                              "stream_GBps": ssum["stream_GBps"], "stream_hbm_frac": ssum["stream_hbm_frac"],
                              "status": sstatus})
            if not args.no_cpu:
                per_shape[-1]["cpu_baseline"] = cpu_baseline(sarch, scls, sprec, sH,
                                                             cpu_sample_images(sarch, sH, sN))
                progress("%s oracle sample: %s" % (sname, per_shape[-1]["cpu_baseline"]["sample"]))
        # the headline shape in fp16 with dynamic loss scaling (the 16-bit
        # mixed precision of Sec. 5.2.3 with the loss scaling it cites)
        fdt, frecs, fstatus, _ = run_shape(B, torch, inputs, arch, classes, "fp16", N, H, args.shape_steps, 2)
        fls = [r for r in frecs if r.get("cls") == "loss_scale"][0]
        fsum, _ = summarize([r for r in frecs if r.get("cls") != "loss_scale"], "fp16")
        per_shape.append({"workload": "imagenet_resnet18_fp16_b256_224", "batch": N, "resolution": H,
                          "dtype": "fp16", "images_per_s": round(N / fdt, 1), "ms_per_step": round(fdt * 1e3, 3),
                          "conv_tflops": fsum["conv_tflops"], "conv_mfma_frac": fsum["conv_mfma_frac"],
                          "stream_GBps": fsum["stream_GBps"], "stream_hbm_frac": fsum["stream_hbm_frac"],
                          "loss_scale": fls["scale"], "skipped_steps": fls["skipped"], "steps_run": fls["steps"],
                          "status": fstatus})
        progress("imagenet_resnet18_fp16_b256_224: %.3f ms/step, loss scale %g, %d of %d steps skipped"
                 % (fdt * 1e3, fls["scale"], fls["skipped"], fls["steps"]))
        # the headline shape with the classifier-input dropout of the 224
        # sub-stage of the ImageNet hybrid schedule (rate 0.2, Table 9)
        ddt, _, dstatus, _ = run_shape(B, torch, inputs, arch, classes, prec, N, H, args.shape_steps, 2, dropout=0.2)
        per_shape.append({"workload": name + "_dropout0.2", "batch": N, "resolution": H, "dtype": prec,
                          "images_per_s": round(N / ddt, 1), "ms_per_step": round(ddt * 1e3, 3), "status": dstatus})
        n_state = B.rn18_state_floats(B.make_config("imagenet", 1000, "bf16"))[0]
        mms, mgbs = merge_rate(B, torch, n_state)
        by = {p["workload"]: p for p in per_shape}
        rounds = []
        for r, bl in ((128, 1024), (160, 640), (192, 448), (224, 256)):
            L_ = by["imagenet_hybrid_bf16_L%d_%d" % (bl, r)]
            S_ = by["imagenet_hybrid_bf16_S64_%d" % r]
            t_round = L_["ms_per_step"] + S_["ms_per_step"] + 3 * mms   # two deltas + merge
            rounds.append({"resolution": r, "B_L": bl, "B_S": 64, "round_ms": round(t_round, 3),
                           "round_images_per_s": round((bl + 64) / t_round * 1e3, 1)})
        per_shape.append({"workload": "ps_dual_merge_imagenet_state", "elements": n_state,
                          "ms": round(mms, 4), "GBps": round(mgbs, 1), "hbm_frac": round(mgbs / HBM_PEAK, 4),
                          "hybrid_rounds": rounds})
        per_shape.append(dbl_plan(B, torch, inputs, by, mms, args.shape_steps))
        per_shape.append(measured_rounds(B, torch, inputs, args.shape_steps))
        per_shape.append(memory_model(B, torch))

    if args.calibrate:
        n = CALIB_FLOATS
        a, b, d = (torch.ones(n, device="cuda") for _ in range(3))
        for _ in range(3):
            B.ps_worker_delta(a, b, d, n)
        torch.cuda.synchronize()

    cpu = None
    if not args.no_cpu:
        cpu = cpu_baseline(arch, classes, prec, H, args.cpu_images)
    # the ceiling's copies and delta streams would enter a profile of the
    # step (and the counter calibration, which reads delta_kernel), so runs
    # under a profiler skip it
    ceil = None if args.calibrate or args.no_ceiling else copy_ceiling(B, torch)

    out = {
        "metric": "ResNet-18 train images/sec/GPU", "value": round(N / dt, 1), "unit": "images/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(dt * 1e3, 3),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": prec,
        "data": "synthetic: N(0,1) fp32 images, uniform int32 labels, He-init weights (seeded)",
        "config": {"workload": name, "global_batch": N, "resolution": H, "classes": classes,
                   "parallelism": "single GPU"},
        "status": status, "loss": round(lval, 5),
        "roofline": roof,
        "conv_mfma_frac": head_sum["conv_mfma_frac"], "conv_tflops": head_sum["conv_tflops"],
        "stream_GBps": head_sum["stream_GBps"], "stream_hbm_frac": head_sum["stream_hbm_frac"],
        "hbm_copy_ceiling_GBps": ceil,
        "stream_ceiling_frac": round(head_sum["stream_GBps"] / ceil, 4) if ceil and head_sum["stream_GBps"] else None,
        "kernel_breakdown_ms": head_sum["classes"],
        "cpu_baseline": cpu,
        "per_shape": per_shape,
    }
    print(json.dumps(out), flush=True)
    try:
        import psutil
        kids = psutil.Process().children(recursive=True)
        progress("child processes at exit: %d %s" % (len(kids), [k.name() for k in kids]))
    except Exception as e:  # psutil is optional here
        progress("child processes at exit: unknown (%s)" % e)


if __name__ == "__main__":
    main()
