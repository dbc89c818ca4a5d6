"""Benchmark: hit patches classified per second on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--config 3] [--precision fp32|bf16|fp16|fp8]

One step is one pass of the whole hot path — patch gather, conv, FC1, FC2 and
the heads — over one batch of synthetic input already resident in HBM:

* config 3 (default): an event of 18 planes (6 x (800, 800, 480) wires x 6000
  ticks, fp32 ADC) and 50,000 hits, classified by one pointid_classify_planes
  call;
* config 2: one 480 x 6000 plane and 3,000 hits (pointid_classify);
* config 1: one 128 x 512 plane and 128 hits (pointid_classify);
* config 4: a batch of pre-cut patches (pointid_classify_patches, --batch).

Prints one JSON line on stdout.  `roofline` describes the kernel that takes the
most time, timed with HIP events on its own stream inside the timed region;
`gather_roofline` does the same for the patch gather against HBM bandwidth;
for the event workload with a 16-bit path, `fp32` gives the same call at the
paper's precision (fp32), timed in the same run; `bf16_batches` times the
bf16 path on pre-cut batches of 16k and 64k patches; `board_power` reads the
socket power and clock (amd-smi) while the event runs back to back;
`cpu_baseline` times the fp64 CPU oracle on a bounded sample of the same
workload on this host's cores.  The default warmup (100 calls) is longer than
the chip's power controller takes to settle under full load (30-40 ms), so the
timed steps measure the sustained rate.
"""

from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "hit patches classified/sec on 1 MI355X; % MFMA peak (dense+conv)"
# Per-patch work of the network (paper §2.2).
CONV_MAC = 44 * 44 * 48 * 25            # 2,323,200
FC1_MAC = 92928 * 128                   # 11,894,784
TAIL_MAC = 128 * 32 + 32 * 4            # 4,224
# MI355X published peaks.
PEAK = {"mfma_bf16": 2500.0, "mfma_fp8": 5000.0, "mfma_fp32": 157.3, "alu_fp32": 157.3,
        "hbm": 8000.0}  # TFLOP/s, GB/s
# The 8-bit kernel runs FC1 on e4m3 MFMAs (5.0 PFLOP/s) and the conv on fp16
# ones (2.5): its peak is the rate at which both would finish together.
PEAK["mfma_fp8_conv16"] = round((CONV_MAC + FC1_MAC) / (FC1_MAC / PEAK["mfma_fp8"]
                                                       + CONV_MAC / PEAK["mfma_bf16"]), 1)

# Kernel name -> (model, source file).  Model gives algorithmic work per patch.
KERNELS = {
    "gather": ("bytes", "gather.hip"),
    "patches_to_16": ("bytes_cast", "gather.hip"),
    "conv_fc1_16": ("flops_conv_fc1", "conv_fc1_16.hip"),
    "conv_fc1_8": ("flops_conv_fc1_8", "conv_fc1_8.hip"),
    "conv_fc1_f32": ("flops_conv_fc1_f32", "conv_fc1_f32.hip"),
    "tail": ("bytes_tail", "tail.hip"),
    "bin_ticks": ("bytes_bin", "gather.hip"),
    "hits_mask": ("bytes_hits_mask", "hits.hip"),
    "hits_scan": ("bytes_hits_scan", "hits.hip"),
    "hits_emit": ("bytes_hits_emit", "hits.hip"),
}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None,
                    help="timed steps (default 100; 20 for --config 5)")
    ap.add_argument("--warmup", type=int, default=None,
                    help="untimed steps before them (default 100, about 0.14 s of the event: under "
                         "full load the chip's power controller settles over the first 30-40 ms, "
                         "during which the 16-bit fused kernel runs 5-15 %% slower; 3 for "
                         "--config 5, whose steps are whole serving runs)")
    ap.add_argument("--config", type=int, default=3, choices=[1, 2, 3, 4, 5])
    ap.add_argument("--precision", default="fp16", choices=["fp32", "bf16", "fp16", "fp8"])
    ap.add_argument("--batch", type=int, default=16384, help="config 4 batch size")
    ap.add_argument("--streams", type=int, default=64, help="config 5: request streams")
    ap.add_argument("--per-stream", type=int, default=32, help="config 5: requests per stream")
    ap.add_argument("--request-hits", type=int, nargs=2, default=[1000, 8000], metavar=("LO", "HI"),
                    help="config 5: hits per request, uniform in [LO, HI]")
    ap.add_argument("--batch-requests", type=int, default=0, metavar="K",
                    help="config 5: merge the requests, in arrival order, into "
                         "pointid_classify_requests calls of K requests (0: one call per request)")
    ap.add_argument("--clients", type=int, default=0, metavar="T",
                    help="config 5: T host threads, each classifying its share of the requests "
                         "one at a time and waiting for each (directly on its own stream, or "
                         "through the dynamic batcher when --batch-requests K > 0)")
    ap.add_argument("--server", action="store_true",
                    help="config 5: requests go through the local request server "
                         "(pointid_server_*, Unix socket) from --clients T client threads "
                         "(default 16), host hits in and host scores out; --batch-requests K "
                         "turns the server's dynamic batcher on")
    ap.add_argument("--patches", action="store_true",
                    help="config 5 with --server: clients send pre-cut fp32 patches "
                         "(9,216 B each, as the paper's clients do) instead of hits")
    ap.add_argument("--batch-delay-us", type=int, default=200,
                    help="config 5 with --clients: the batcher's longest wait for a fuller batch")
    ap.add_argument("--sort-hits", action="store_true",
                    help="config 3: hits in (plane, wire, tick) order, as a hit finder emits "
                         "them, instead of the generator's shuffled order")
    ap.add_argument("--ticks-per-column", type=int, default=1, metavar="D",
                    help="config 3: patches whose columns span D ticks "
                         "(pointid_classify_planes_ds; 1 = pointid_classify_planes)")
    ap.add_argument("--find-hits", type=float, default=None, metavar="THR",
                    help="config 3: time hit finding (pointid_find_hits) on the event's 18 "
                         "planes at threshold THR instead of classification")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-h2d", action="store_true", help="skip timing the host-to-device copies")
    ap.add_argument("--no-batch-block", action="store_true",
                    help="config 3: skip timing bf16 pre-cut batches of 16k and 64k patches")
    ap.add_argument("--sample-power", type=float, default=4.0, metavar="SECONDS",
                    help="config 3: read socket power and clock (amd-smi) while the call runs "
                         "back to back for this long after the timed region; 0 skips it")
    ap.add_argument("--no-fp32-block", action="store_true",
                    help="config 3: skip timing the same call at fp32 (the paper's precision)")
    ap.add_argument("--cpu-sample", type=int, default=24576, help="hits timed on the oracle (about 10 s)")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="first run 3 device-to-device copies of MIB MiB (a plain copy kernel of "
                         "known size, to scale rocprofv3 FETCH_SIZE/WRITE_SIZE)")
    args = ap.parse_args()
    light = args.config == 5 and args.find_hits is None
    if args.steps is None:
        args.steps = 20 if light else 100
    if args.warmup is None:
        args.warmup = 3 if light else 100
    return args


def source_sha(fname):
    p = os.path.join(ROOT, "paper_2009_04509_amd", "csrc", fname)
    return hashlib.sha256(open(p, "rb").read()).hexdigest()[:16]


def load_traffic(kernel, workload_tag):
    """HBM bytes per launch from a committed rocprofv3 counter summary, if it was
    taken on the current kernel source; else None."""
    path = os.path.join(ROOT, "profiles", f"traffic_{kernel}_{workload_tag}.txt")
    if not os.path.exists(path):
        return None
    kv = {}
    for line in open(path):
        if ":" in line and not line.startswith("#"):
            k, v = line.split(":", 1)
            kv[k.strip()] = v.strip()
    if kv.get("source_sha256_16") != source_sha(KERNELS[kernel][1]):
        return None
    try:
        return float(kv["hbm_bytes_per_dispatch"])
    except (KeyError, ValueError):
        return None


def make_workload(args, torch, pid):
    import synth
    dev = "cuda:0"
    if args.config == 3:
        planes, h3 = synth.config3()
        if args.sort_hits:
            h3 = np.ascontiguousarray(h3[np.lexsort((h3[:, 2], h3[:, 1], h3[:, 0]))])
        imgs = [torch.from_numpy(p.image).to(dev) for p in planes]
        hits = torch.from_numpy(h3).to(dev)
        n = len(h3)
        scores = torch.empty((n, 4), dtype=torch.float32, device=dev)
        D = args.ticks_per_column
        if D > 1:
            shapes = [(p.image.shape[0], -(-p.image.shape[1] // D)) for p in planes]
            cols = h3.copy()
            cols[:, 2] = np.floor_divide(cols[:, 2], D)
            footprint = _footprint(shapes, cols)

            def step(h):
                pid.pointid_classify_planes_ds(h, imgs, hits, D, scores)

            desc = {"workload": f"event: 18 planes (6x(800,800,480) wires x 6000 ticks fp32 ADC), "
                                f"50,000 hits, patch columns of {D} ticks, one "
                                "pointid_classify_planes_ds call (binning included)",
                    "hits": n, "planes": 18, "ticks": 6000, "ticks_per_column": D}
        else:
            footprint = _footprint([p.image.shape for p in planes], h3)

            def step(h):
                pid.pointid_classify_planes(h, imgs, hits, scores)

            desc = {"workload": "event: 18 planes (6x(800,800,480) wires x 6000 ticks fp32 ADC), "
                                "50,000 hits" + (" in (plane, wire, tick) order" if args.sort_hits
                                                 else "") + ", one pointid_classify_planes call",
                    "hits": n, "planes": 18, "ticks": 6000}
        sample = dict(kind="planes", images=[p.image for p in planes], hits=h3, D=D)
        hit_bytes = 12
    elif args.config in (1, 2):
        p = synth.config1() if args.config == 1 else synth.config2()
        img = torch.from_numpy(p.image).to(dev)
        hits = torch.from_numpy(p.hits).to(dev)
        n = len(p.hits)
        scores = torch.empty((n, 4), dtype=torch.float32, device=dev)
        h3 = np.c_[np.zeros(n, np.int32), p.hits]
        footprint = _footprint([p.image.shape], h3)

        def step(h):
            pid.pointid_classify(h, img, hits, scores)

        W, T = p.image.shape
        desc = {"workload": f"plane: {W} wires x {T} ticks fp32 ADC, {n:,} hits, one "
                            "pointid_classify call", "hits": n, "planes": 1, "ticks": T}
        sample = dict(kind="plane", image=p.image, hits=p.hits)
        hit_bytes = 8
    else:
        P = synth.config4_patches(args.batch)
        patches = torch.from_numpy(P).to(dev)
        n = args.batch
        scores = torch.empty((n, 4), dtype=torch.float32, device=dev)
        footprint = 0

        def step(h):
            pid.pointid_classify_patches(h, patches, scores)

        desc = {"workload": f"pre-cut patch batch of {n} (N(0,1) + one line each), one "
                            "pointid_classify_patches call", "hits": n}
        sample = dict(kind="patches", patches=P)
        hit_bytes = 0
    return step, n, desc, sample, footprint, hit_bytes


def _footprint(shapes, h3):
    """Distinct image pixels the hits' 48x48 windows touch (the gather's minimal read)."""
    total = 0
    for p, (W, T) in enumerate(shapes):
        sel = h3[h3[:, 0] == p]
        if not len(sel):
            continue
        mask = np.zeros((W + 48, T + 48), np.int8)
        for w, t in sel[:, 1:]:
            mask[w:w + 48, t:t + 48] = 1            # offset by 24 on both axes
        total += int(mask[24:24 + W, 24:24 + T].sum())
    return total


def host_facts():
    """Cores this process may run on, the BLAS thread count numpy uses, and
    the CPU model (from /proc/cpuinfo)."""
    cores = len(os.sched_getaffinity(0))
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        threads = None
    model = None
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return cores, threads, model


def cpu_baseline(sample, n_sample):
    import oracle
    import synth
    cores, threads, cpu_model = host_facts()
    w = synth.he_normal_weights()
    rng = np.random.default_rng(2024)
    if sample["kind"] == "planes":
        idx = np.sort(rng.choice(len(sample["hits"]), n_sample, replace=False))
        t0 = time.perf_counter()
        if sample.get("D", 1) > 1:
            oracle.classify_planes_ds(sample["images"], sample["hits"][idx], w, sample["D"])
            what = (f"{n_sample} hits sampled (seeded) from the 50,000-hit event, "
                    f"oracle.classify_planes_ds with D = {sample['D']} (binning included)")
        else:
            oracle.classify_planes(sample["images"], sample["hits"][idx], w)
            what = f"{n_sample} hits sampled (seeded) from the 50,000-hit event, oracle.classify_planes"
        if "what" in sample:
            what = f"{n_sample} {sample['what']}, oracle.classify_planes"
    elif sample["kind"] == "plane":
        idx = np.sort(rng.choice(len(sample["hits"]), min(n_sample, len(sample["hits"])), replace=False))
        t0 = time.perf_counter()
        oracle.classify(sample["image"], sample["hits"][idx], w)
        what = f"{len(idx)} hits sampled (seeded) from the plane, oracle.classify"
    else:
        idx = np.arange(min(n_sample, len(sample["patches"])))
        t0 = time.perf_counter()
        oracle.classify_patches(sample["patches"][idx], w)
        what = f"first {len(idx)} patches of the batch, oracle.classify_patches"
    dt = time.perf_counter() - t0
    return {"value": len(idx) / dt, "unit": "patches/s", "cores": int(cores), "kind": "oracle",
            "sample": f"{what}; {dt:.1f} s", "seconds": round(dt, 2),
            "blas_threads": threads, "cpu_model": cpu_model,
            "per_core": round(len(idx) / dt / cores, 2),
            "paper_context": "paper section 3.1: 213 s of single-process TensorFlow inference "
                             "for about 55,000 patches per event, about 258 patches/s per process "
                             "(other hardware; context only)"}


def env_info(torch, pid):
    """Versions and the device the line was measured on."""
    props = torch.cuda.get_device_properties(0)
    return {"device": props.name, "gcn_arch": getattr(props, "gcnArchName", None),
            "cus": props.multi_processor_count, "hip": torch.version.hip,
            "torch": torch.__version__, "libpointid": pid.pointid_version()}


def board_power(args, torch, pid, synth, step, precision):
    """Socket power and shader clock while the step runs back to back for
    args.sample_power seconds (a host sync every 8 calls), read with
    `amd-smi metric -p -c` (read-only) about every 0.1 s; samples of the first
    second (the ramp) are left out.  Shows whether the chip runs at its power
    cap or at its top clock under this load; the hotspot temperature before
    and just after the load is context for boxes whose sockets settle at
    different powers."""
    import shutil
    import subprocess
    import threading
    tool = shutil.which("amd-smi") or "/opt/rocm/bin/amd-smi"

    def read():
        r = subprocess.run([tool, "metric", "-p", "-c", "-g", "0", "--json"],
                           capture_output=True, text=True, timeout=20)
        d = json.loads(r.stdout)
        g = d["gpu_data"][0] if isinstance(d, dict) else d[0]
        clks = [v["clk"]["value"] for k, v in g["clock"].items()
                if k.startswith("gfx_") and isinstance(v, dict) and isinstance(v.get("clk"), dict)
                and isinstance(v["clk"].get("value"), (int, float))]
        return float(g["power"]["socket_power"]["value"]), (float(np.mean(clks)) if clks else None)

    def hotspot():
        # a separate query: the temperature is only context, so a missing
        # field costs nothing but this reading
        try:
            r = subprocess.run([tool, "metric", "-t", "-g", "0", "--json"],
                               capture_output=True, text=True, timeout=20)
            d = json.loads(r.stdout)
            g = d["gpu_data"][0] if isinstance(d, dict) else d[0]
            v = g["temperature"]["hotspot"]["value"]
            return float(v) if isinstance(v, (int, float)) else None
        except Exception:
            return None

    try:
        read()
    except Exception as exc:                       # no tool or no reading on this machine
        return {"tool": "amd-smi metric -p -c", "error": repr(exc)[:200]}
    h = pid.pointid_create(synth.he_normal_weights(), precision, 0)
    for _ in range(3):
        step(h)
    torch.cuda.synchronize()
    stop, samples = threading.Event(), []

    def sampler():
        while not stop.is_set():
            t = time.perf_counter()
            try:
                samples.append((t,) + read())
            except Exception:
                pass
            time.sleep(0.1)

    th = threading.Thread(target=sampler)
    t_idle = hotspot()
    t0 = time.perf_counter()
    th.start()
    calls = 0
    while time.perf_counter() - t0 < args.sample_power:
        for _ in range(8):
            step(h)
        calls += 8
        torch.cuda.synchronize()
    t_load = hotspot()                             # just after the last calls
    dt = time.perf_counter() - t0
    stop.set()
    th.join()
    h.close()
    kept = [x for x in samples if x[0] - t0 >= 1.0]
    pw = np.array([x[1] for x in kept])
    ck = np.array([x[2] for x in kept if x[2] is not None])
    out = {"tool": "amd-smi metric -p -c (socket power, mean gfx clock over XCDs); "
                   "metric -t (hotspot, before and just after the load)",
           "precision": precision, "seconds": round(dt, 2), "calls": calls,
           "ms_per_call": round(dt * 1e3 / max(calls, 1), 4), "samples": int(len(kept))}
    if len(pw):
        out["socket_power_w"] = {"median": float(np.median(pw)), "min": float(pw.min()), "max": float(pw.max())}
    if len(ck):
        out["gfx_clock_mhz"] = {"median": round(float(np.median(ck)), 1), "min": round(float(ck.min()), 1),
                                "max": round(float(ck.max()), 1)}
    out["hotspot_c"] = {"before": t_idle, "end": t_load}
    log(f"[bench] board power over {dt:.1f} s ({calls} calls): {out.get('socket_power_w')} W, "
        f"clock {out.get('gfx_clock_mhz')} MHz")
    return out


def transfer(args, torch, sample, n):
    """Host-to-device copies from pinned host memory, outside the timed region:
    the event's planes and hits (what this library's hit paths read), and the
    same hits' pre-cut fp32 patches (what the paper's clients transmit, its
    t_transmit).  Median of 5 copies each, HIP events on the current stream."""
    def time_copy(nbytes):
        src = torch.empty(nbytes // 4, dtype=torch.float32, pin_memory=True)
        dst = torch.empty(nbytes // 4, dtype=torch.float32, device="cuda:0")
        ms = []
        for _ in range(6):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            dst.copy_(src, non_blocking=True)
            e1.record()
            torch.cuda.synchronize()
            ms.append(e0.elapsed_time(e1))
        del src, dst
        return float(np.median(ms[1:]))
    if sample["kind"] == "planes":
        in_bytes = sum(im.nbytes for im in sample["images"]) + sample["hits"].nbytes
    elif sample["kind"] == "plane":
        in_bytes = sample["image"].nbytes + sample["hits"].nbytes
    else:
        in_bytes = 0
    out = {"note": "host-to-device copies from pinned memory, not in the timed region; "
                   "the analogue of the paper's t_transmit"}
    if in_bytes:
        ms = time_copy(in_bytes)
        out["planes_and_hits"] = {"bytes": int(in_bytes), "ms": round(ms, 4),
                                  "GB_per_s": round(in_bytes / (ms * 1e-3) / 1e9, 2)}
    pb = n * 9216
    ms = time_copy(pb)
    out["precut_fp32_patches"] = {"bytes": int(pb), "ms": round(ms, 4),
                                  "GB_per_s": round(pb / (ms * 1e-3) / 1e9, 2)}
    log(f"[bench] H2D: {out}")
    return out


def serving(args, torch, pid, synth):
    """Config 5: 8 resident config-2 planes; requests of 1,000-8,000 hits (or
    `--request-hits`) sent on `--streams` streams, `--per-stream` each, enqueued
    round-robin.  One step classifies every request, one call per request, or
    (`--batch-requests K`) K consecutive arrivals per batched call.  The value is
    hits per second of wall-clock time from the first enqueue to the completion
    of the last request (host enqueue cost included).  Per-request latency is
    the time between events recorded on the stream just before and just after
    the call that classified it.  With `--clients T`, T host threads each
    classify their share one request at a time and wait for it (the paper's
    many client processes), directly or through the dynamic batcher; latency
    is then the host time from the call (or submit) to the scores being ready."""
    dev = "cuda:0"
    lo_hits, hi_hits = args.request_hits
    planes, reqs = synth.config5_requests(n_planes=8, n_streams=args.streams,
                                          per_stream=args.per_stream, lo=lo_hits, hi=hi_hits)
    imgs = [torch.from_numpy(p.image).to(dev) for p in planes]
    hits = [[torch.from_numpy(x).to(dev) for (_, x) in rs] for rs in reqs]
    outs = [[torch.empty((len(x), 4), dtype=torch.float32, device=dev) for (_, x) in rs]
            for rs in reqs]
    streams = [torch.cuda.Stream() for _ in reqs]
    total = sum(len(x) for rs in reqs for (_, x) in rs)
    h = pid.pointid_create(synth.he_normal_weights(), args.precision, 0)

    K = args.batch_requests
    # arrival order: the k-th request of every stream, round-robin
    order = [(s, k) for k in range(args.per_stream) for s in range(len(reqs))]

    T = args.clients
    if args.server and T <= 0:
        T = 16
    batcher = pid.Batcher(h, imgs, max_requests=K, max_delay_us=args.batch_delay_us) \
        if (T > 0 and K > 0 and not args.server) else None
    server = None
    if args.server:
        import tempfile
        sock_dir = tempfile.mkdtemp(prefix="pointid_")
        sock_path = os.path.join(sock_dir, "bench.sock")
        server = pid.Server(h, imgs, sock_path, max_requests=K, max_delay_us=args.batch_delay_us)
        clients = [pid.Client(sock_path) for _ in range(T)]
        host_hits = [[x for (_, x) in rs] for rs in reqs]
        host_patches = None
        if args.patches:
            # the clients' pre-cut patches, made once before timing with the
            # library's own gather and kept in host memory
            host_patches = [[pid.pointid_gather(imgs[p], hits[s][k]).cpu().numpy()
                             for k, (p, _) in enumerate(rs)] for s, rs in enumerate(reqs)]
        server_ns = []

    def client_step():
        """T synchronous clients; per-request latency measured on the host."""
        import threading
        lat = [[] for _ in range(T)]

        def client(c):
            st = streams[c % len(streams)]
            for s, k in order[c::T]:
                t0 = time.perf_counter()
                if server is not None:
                    if host_patches is not None:
                        clients[c].classify_patches(host_patches[s][k])
                    else:
                        clients[c].classify(host_hits[s][k], plane=reqs[s][k][0])
                    server_ns.append(clients[c].server_ns)
                elif batcher is not None:
                    batcher.wait(batcher.submit(reqs[s][k][0], hits[s][k], outs[s][k]))
                else:
                    pid.pointid_classify(h, imgs[reqs[s][k][0]], hits[s][k], outs[s][k], stream=st)
                    st.synchronize()
                lat[c].append((time.perf_counter() - t0) * 1e3)

        ths = [threading.Thread(target=client, args=(c,)) for c in range(T)]
        for th in ths:
            th.start()
        for th in ths:
            th.join()
        return [x for l in lat for x in l]

    def one_step():
        if T > 0:
            return client_step()
        evs = []
        if K <= 0:
            for s, k in order:
                st = streams[s]
                e0 = torch.cuda.Event(enable_timing=True)
                e1 = torch.cuda.Event(enable_timing=True)
                e0.record(st)
                pid.pointid_classify(h, imgs[reqs[s][k][0]], hits[s][k], outs[s][k], stream=st)
                e1.record(st)
                evs.append((e0, e1))
            return evs
        # batched: consecutive arrivals share one call; the calls rotate over
        # the streams so that batches overlap as single requests do
        for b in range(0, len(order), K):
            st = streams[(b // K) % len(streams)]
            batch = [(reqs[s][k][0], hits[s][k], outs[s][k]) for s, k in order[b:b + K]]
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record(st)
            pid.pointid_classify_requests(h, imgs, batch, stream=st)
            e1.record(st)
            evs += [(e0, e1)] * len(batch)
        return evs

    log(f"[bench] serving: {args.streams} streams x {args.per_stream} requests, {total} hits; "
        f"warmup {args.warmup}")
    for _ in range(args.warmup):
        one_step()
    torch.cuda.synchronize()
    pid.pointid_timing_reset()
    pid.pointid_timing_enable(True)
    lat, walls = [], []
    for _ in range(args.steps):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        evs = one_step()
        torch.cuda.synchronize()
        walls.append(time.perf_counter() - t0)
        lat += evs if T > 0 else [a.elapsed_time(b) for a, b in evs]
    pid.pointid_timing_enable(False)
    wall = float(np.sum(walls))
    value = total * args.steps / wall
    lat = np.asarray(lat)
    log(f"[bench] {args.steps} steps: {wall / args.steps * 1e3:.2f} ms/step, "
        f"{value / 1e6:.2f} M patches/s; latency p50 {np.percentile(lat, 50):.3f} ms "
        f"p99 {np.percentile(lat, 99):.3f} ms")
    kern = {}
    for name in KERNELS:
        tot, cnt = pid.pointid_timing_query(name)
        if cnt:
            kern[name] = {"ms_per_step": round(tot / args.steps, 4), "launches": cnt,
                          "avg_launch_ms": round(tot / cnt, 4)}
    # the fused kernel over all launches of the timed steps (every request's
    # patches pass through it once).  When the batches run on one stream (a
    # batcher's) the launches are timed one by one; when requests run on many
    # streams at once their launches overlap, and the step's wall clock is the
    # time base instead.
    roof = None
    fused = [(k, pk) for k, pk in (("conv_fc1_16", "mfma_bf16"), ("conv_fc1_8", "mfma_fp8_conv16"),
                                    ("conv_fc1_f32", "mfma_fp32")) if k in kern]
    if fused:
        fk, pk = fused[0]
        one_stream = batcher is not None or (server is not None and K > 0)
        flop = total * args.steps * 2 * (CONV_MAC + FC1_MAC)
        base_s = (kern[fk]["ms_per_step"] * args.steps * 1e-3 if one_stream else wall)
        ach = flop / base_s / 1e12
        roof = {"kernel": fk, "bound": "mfma", "achieved": round(ach, 3),
                "peak": PEAK[pk], "unit": "TFLOP/s",
                "frac": round(ach / PEAK[pk], 4), "traffic": None,
                "time_base": "launch events on the batcher's stream" if one_stream else
                             "wall clock of the steps (launches on many streams overlap)",
                "avg_launch_ms": kern[fk]["avg_launch_ms"],
                "work_per_launch": flop / kern[fk]["launches"]}
    out = {
        "metric": METRIC, "value": round(value, 1), "unit": "patches/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(wall / args.steps * 1e3, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": args.precision, "data": "synthetic",
        "config": {"workload": f"serving: 8 resident planes (480 wires x 6000 ticks), "
                               f"{args.streams} streams x {args.per_stream} requests of "
                               f"{lo_hits:,}-{hi_hits:,} hits, " + (
                                   f"{T} client threads, each waiting for its request; " if T > 0
                                   else "") + (
                                   ("through the local request server (Unix socket, host " +
                                    ("patches" if args.patches else "hits") + " in, host scores "
                                    "out), ") if server is not None else "") + (
                                   (f"dynamic batcher (up to {K} requests, {args.batch_delay_us} us)"
                                    if T > 0 else
                                    f"batches of {K} requests per pointid_classify_requests call")
                                   if K > 0 else "one pointid_classify per request"),
                   "hits": total, "requests": args.streams * args.per_stream,
                   "batch_requests": K, "clients": T,
                   "precision": args.precision},
        "latency_ms": {"p50": round(float(np.percentile(lat, 50)), 4),
                       "p99": round(float(np.percentile(lat, 99)), 4),
                       "mean": round(float(lat.mean()), 4)},
        "roofline": roof,
        "kernels": kern,
    }
    if not args.no_cpu_baseline:
        # the oracle on a seeded sample of the requests' hits (each on its plane)
        rng = np.random.default_rng(2025)
        flat = [(p, x) for rs in reqs for (p, x) in rs]
        pick = rng.choice(len(flat), 6, replace=False)
        imgs_np = [pl.image for pl in planes]
        parts = []
        for r in pick:
            p, x = flat[r]
            parts.append(np.c_[np.full(len(x), p, np.int32), x])
        h3s = np.concatenate(parts)[:args.cpu_sample]
        out["cpu_baseline"] = cpu_baseline(dict(kind="planes", images=imgs_np, hits=h3s,
                                                what="hits of 6 seeded requests"), len(h3s))
    if server is not None:
        sn = np.asarray(server_ns, np.float64) / 1e6
        out["server_ms"] = {"p50": round(float(np.percentile(sn, 50)), 4),
                            "p99": round(float(np.percentile(sn, 99)), 4)}
        for c in clients:
            c.close()
        server.close()
    if batcher is not None:
        batcher.close()
    h.close()
    out["env"] = env_info(torch, pid)
    print(json.dumps(out), flush=True)


def hit_finding(args, torch, pid, synth):
    """Config 3 planes: one step finds every hit of the event's 18 planes
    (pointid_find_hits, three launches).  Algorithmic bytes of a step: the image
    read once, plus 12 B written per hit found."""
    import oracle
    dev = "cuda:0"
    thr = float(args.find_hits)
    planes, _ = synth.config3()
    imgs_np = [p.image for p in planes]
    imgs = [torch.from_numpy(a).to(dev) for a in imgs_np]
    image_bytes = sum(a.nbytes for a in imgs_np)
    rows = sum(a.shape[0] for a in imgs_np)
    h = pid.pointid_create(synth.he_normal_weights(), "fp16", 0)
    cap = 8 << 20
    out = torch.empty((cap, 3), dtype=torch.int32, device=dev)
    n_found = torch.empty((1,), dtype=torch.int64, device=dev)

    def step():
        pid.pointid_find_hits(h, imgs, thr, capacity=cap, hits_out=out, n_found=n_found)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    n_hits = int(n_found.item())
    pid.pointid_timing_reset()
    pid.pointid_timing_enable(True)
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    evs[0].record()
    for i in range(args.steps):
        step()
        evs[i + 1].record()
    torch.cuda.synchronize()
    pid.pointid_timing_enable(False)
    ms_step = evs[0].elapsed_time(evs[-1]) / args.steps
    per_step = np.array([evs[i].elapsed_time(evs[i + 1]) for i in range(args.steps)])
    mask_bytes = rows * 24 * 32
    work = {"hits_mask": image_bytes + mask_bytes + 4 * rows,
            "hits_scan": 4 * rows + 8 * rows + 8,
            "hits_emit": mask_bytes + 4 * rows + 8 * rows + 12 * n_hits}
    kern = {}
    for name, wb in work.items():
        tot, cnt = pid.pointid_timing_query(name)
        if cnt:
            kern[name] = {"ms_per_step": round(tot / args.steps, 4), "launches": cnt,
                          "avg_launch_ms": tot / cnt, "achieved": wb / (tot / cnt * 1e-3) / 1e9,
                          "unit": "GB/s", "work_per_launch": wb}
    d = kern["hits_mask"]
    value = (image_bytes + 12 * n_hits) / (ms_step * 1e-3) / 1e9
    log(f"[bench] find_hits thr {thr}: {n_hits} hits, {ms_step * 1e3:.1f} us/step, "
        f"{value:.0f} GB/s over the whole call")
    out_json = {
        "metric": "event hit finding: image bytes scanned + hits written per second",
        "value": round(value, 2), "unit": "GB/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_step, 4),
        "step_ms": {"median": round(float(np.median(per_step)), 4),
                    "min": round(float(per_step.min()), 4), "max": round(float(per_step.max()), 4)},
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": "event: 18 planes (6x(800,800,480) wires x 6000 ticks fp32 ADC), "
                               f"hits = ticks above {thr} that are local maxima along the wire, "
                               "one pointid_find_hits call", "threshold": thr,
                   "hits_found": n_hits, "image_bytes": image_bytes},
        "roofline": {"kernel": "hits_mask", "bound": "hbm", "achieved": round(d["achieved"], 2),
                     "peak": PEAK["hbm"], "unit": "GB/s",
                     "frac": round(d["achieved"] / PEAK["hbm"], 4),
                     "traffic": load_traffic("hits_mask", "config3_hits"),
                     "avg_launch_ms": round(d["avg_launch_ms"], 4),
                     "work_per_launch": d["work_per_launch"]},
        "kernels": {k: {"ms_per_step": v["ms_per_step"], "launches": v["launches"],
                        "achieved": round(v["achieved"], 2), "unit": "GB/s"}
                    for k, v in kern.items()},
    }
    if not args.no_cpu_baseline:
        cores, _threads, cpu_model = host_facts()
        t0 = time.perf_counter()
        ref = oracle.find_hits(imgs_np, thr)
        dt = time.perf_counter() - t0
        out_json["cpu_baseline"] = {"value": round((image_bytes + 12 * len(ref)) / dt / 1e9, 3),
                                    "unit": "GB/s", "cores": 1, "kind": "oracle",
                                    "sample": f"the whole event, oracle.find_hits (numpy, one "
                                              f"thread of the {cores} this process may use); {dt:.2f} s",
                                    "seconds": round(dt, 2), "cpu_model": cpu_model}
        got = out[:min(n_hits, cap)].cpu().numpy()
        out_json["matches_oracle"] = bool(len(ref) == n_hits and np.array_equal(got, ref))
    h.close()
    out_json["env"] = env_info(torch, pid)
    print(json.dumps(out_json), flush=True)


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py: measures one GPU only (got --gpus {args.gpus}); the per-hit "
              "path would shard by hits or planes, with no exchange between GPUs", file=sys.stderr)
        sys.exit(2)
    import torch
    from paper_2009_04509_amd import binding as pid
    import synth

    if not torch.cuda.is_available():
        raise SystemExit("bench.py needs a GPU")
    if args.calibrate_copy:
        src = torch.ones(args.calibrate_copy << 20, dtype=torch.uint8, device="cuda:0")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        log(f"[bench] calibration: 3 copies of {args.calibrate_copy} MiB")
        del src, dst
    if args.config == 5:
        serving(args, torch, pid, synth)
        return
    if args.find_hits is not None:
        if args.config != 3:
            raise SystemExit("--find-hits runs on the config 3 event planes")
        hit_finding(args, torch, pid, synth)
        return
    log(f"[bench] building config {args.config} workload")
    step, n, desc, sample, footprint, hit_bytes = make_workload(args, torch, pid)
    r = measure(args, torch, pid, synth, step, n, footprint, hit_bytes, args.precision)
    value = n / (r["ms_step"] * 1e-3)
    total_flop = n * 2 * (CONV_MAC + FC1_MAC + TAIL_MAC)
    out = {
        "metric": METRIC, "value": round(value, 1), "unit": "patches/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(r["ms_step"], 4),
        "step_ms": r["step_ms"],
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": args.precision, "data": "synthetic",
        "config": {**desc, "precision": args.precision},
        "roofline": r["roofline"],
        "network_tflops": round(total_flop / (r["ms_step"] * 1e-3) / 1e12, 3),
        "kernels": r["kernels"],
    }
    if "gather" in r["kern"]:
        g = r["kern"]["gather"]
        out["gather_roofline"] = {"kernel": "gather", "bound": "hbm", "achieved": round(g["achieved"], 2),
                                  "peak": PEAK["hbm"], "unit": "GB/s",
                                  "frac": round(g["achieved"] / PEAK["hbm"], 4),
                                  "traffic": load_traffic("gather", f"config{args.config}_{args.precision}"),
                                  "avg_launch_ms": round(g["avg_launch_ms"], 4),
                                  "work_per_launch": g["work_per_launch"]}
    if args.config == 3 and args.precision != "fp32" and not args.no_fp32_block:
        # the same call at the paper's precision (fp32 operands, fp32 MFMA),
        # timed in the same run; the headline stays the 16-bit path
        log("[bench] the same workload at fp32")
        r32 = measure(args, torch, pid, synth, step, n, footprint, hit_bytes, "fp32")
        out["fp32"] = {"dtype": "fp32", "value": round(n / (r32["ms_step"] * 1e-3), 1),
                       "unit": "patches/s", "ms_per_step": round(r32["ms_step"], 4),
                       "step_ms": r32["step_ms"], "roofline": r32["roofline"],
                       "kernels": r32["kernels"]}
    if args.config == 3 and args.precision in ("fp16", "bf16") and not args.no_batch_block:
        # the stated target's setting: bf16 operands on pre-cut batches of 16k
        # and 64k patches (the config-4 recipe), where the bf16 path also
        # meets the 2e-2 score bound against the fp64 oracle; timed in the same
        # run, the headline stays the event
        blk = {"dtype": "bf16", "workload": "pre-cut patch batches (N(0,1) + one line each), "
                                            "one pointid_classify_patches call each"}
        for b in (16384, 65536):
            a4 = argparse.Namespace(**vars(args))
            a4.config, a4.batch = 4, b
            log(f"[bench] bf16 batch of {b}")
            st4, n4, _, _, fp4, hb4 = make_workload(a4, torch, pid)
            r4 = measure(a4, torch, pid, synth, st4, n4, fp4, hb4, "bf16")
            blk[str(b)] = {"value": round(n4 / (r4["ms_step"] * 1e-3), 1), "unit": "patches/s",
                           "ms_per_step": round(r4["ms_step"], 4), "roofline": r4["roofline"]}
            del st4
            torch.cuda.empty_cache()
        out["bf16_batches"] = blk
    if args.sample_power > 0 and args.config == 3:
        out["board_power"] = board_power(args, torch, pid, synth, step, args.precision)
    if not args.no_h2d and args.config in (2, 3):
        out["h2d"] = transfer(args, torch, sample, n)
    if not args.no_cpu_baseline:
        log("[bench] cpu baseline (oracle)")
        out["cpu_baseline"] = cpu_baseline(sample, args.cpu_sample)
    out["env"] = env_info(torch, pid)
    print(json.dumps(out), flush=True)


def measure(args, torch, pid, synth, step, n, footprint, hit_bytes, precision):
    """Warm up, then time args.steps calls of `step` with a handle of
    `precision`: per-step events on the current stream bracket the timed
    region; the library's per-kernel events give each kernel's time."""
    h = pid.pointid_create(synth.he_normal_weights(), precision, 0)
    log(f"[bench] {precision}: warmup {args.warmup}")
    for _ in range(args.warmup):
        step(h)
    torch.cuda.synchronize()

    pid.pointid_timing_reset()
    pid.pointid_timing_enable(True)
    torch.cuda.synchronize()
    # one event per step boundary: the first and last bracket the timed region,
    # the others give the per-step distribution
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    t_wall = time.perf_counter()
    evs[0].record()
    for i in range(args.steps):
        step(h)
        evs[i + 1].record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_wall
    pid.pointid_timing_enable(False)
    ms = evs[0].elapsed_time(evs[-1])
    ms_step = ms / args.steps
    per_step = np.array([evs[i].elapsed_time(evs[i + 1]) for i in range(args.steps)])
    log(f"[bench] {args.steps} steps: {ms_step:.3f} ms/step (wall {wall * 1e3 / args.steps:.3f}; "
        f"median {np.median(per_step):.3f}, min {per_step.min():.3f}, max {per_step.max():.3f})")

    patch_bytes = 9216 if precision == "fp32" else 4608
    kern = {}
    for name, (model, _src) in KERNELS.items():
        tot, cnt = pid.pointid_timing_query(name)
        if cnt == 0:
            continue
        per_step_patches = n
        if model == "bytes":
            work = args.steps * (per_step_patches * (patch_bytes + hit_bytes) + footprint * 4)
            unit, rate = "GB/s", work / (tot * 1e-3) / 1e9
        elif model == "bytes_tail":
            work = args.steps * per_step_patches * (8 * 128 * 4 + 16)
            unit, rate = "GB/s", work / (tot * 1e-3) / 1e9
        elif model == "bytes_bin":
            img_bytes = 4 * 12480 * 6000
            work = args.steps * (img_bytes + img_bytes // args.ticks_per_column)
            unit, rate = "GB/s", work / (tot * 1e-3) / 1e9
        elif model == "bytes_cast":
            work = args.steps * per_step_patches * (9216 + 4608)
            unit, rate = "GB/s", work / (tot * 1e-3) / 1e9
        else:
            mac = {"flops_conv": CONV_MAC, "flops_fc1": FC1_MAC, "flops_conv_fc1": CONV_MAC + FC1_MAC,
                   "flops_conv_fc1_8": CONV_MAC + FC1_MAC, "flops_conv_fc1_f32": CONV_MAC + FC1_MAC}[model]
            work = args.steps * per_step_patches * 2 * mac
            unit, rate = "TFLOP/s", work / (tot * 1e-3) / 1e12
        kern[name] = {"ms_per_step": tot / args.steps, "launches": cnt,
                      "avg_launch_ms": tot / cnt, "achieved": rate, "unit": unit,
                      "work_per_launch": work / cnt}
        log(f"[bench] {name:10s} {tot / args.steps:8.3f} ms/step  {cnt} launches  {rate:9.2f} {unit}")
    h.close()

    dom = max(kern, key=lambda k: kern[k]["ms_per_step"])
    d = kern[dom]
    model = KERNELS[dom][0]
    if model == "flops_conv_fc1":
        bound, peak = "mfma", PEAK["mfma_bf16"]       # fp16 and bf16 MFMA share one peak
    elif model == "flops_conv_fc1_8":
        bound, peak = "mfma", PEAK["mfma_fp8_conv16"]
    elif model in ("flops_fc1", "flops_conv", "flops_conv_fc1_f32"):
        bound, peak = "mfma", PEAK["mfma_fp32"]
    elif model.startswith("flops"):
        bound, peak = "alu", PEAK["alu_fp32"]
    else:
        bound, peak = "hbm", PEAK["hbm"]
    tag = f"config{args.config}_{precision}"
    roof = {"kernel": dom, "bound": bound, "achieved": round(d["achieved"], 3), "peak": peak,
            "unit": d["unit"], "frac": round(d["achieved"] / peak, 4),
            "traffic": load_traffic(dom, tag), "avg_launch_ms": round(d["avg_launch_ms"], 4),
            "work_per_launch": d["work_per_launch"]}
    return {"ms_step": ms_step,
            "step_ms": {"median": round(float(np.median(per_step)), 4),
                        "min": round(float(per_step.min()), 4), "max": round(float(per_step.max()), 4)},
            "roofline": roof, "kern": kern,
            "kernels": {k: {"ms_per_step": round(v["ms_per_step"], 4), "launches": v["launches"],
                            "achieved": round(v["achieved"], 3), "unit": v["unit"]}
                        for k, v in kern.items()}}


if __name__ == "__main__":
    main()
