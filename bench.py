#!/usr/bin/env python3
"""Single-stream throughput of RVQ-position-aware speculative decoding on one GPU.

One step is one audio frame: the inner MultiCodeDecoder loop emitting the 15
residual codes c_1..c_15 of a frame after c_0 (prefix pass plus speculative
draft/verify rounds, Sec. 2.2 and Fig. 3 of the paper), decoded by the
library's persistent frame kernel through rvqsd_decode_frames_async (up to 1024
frames per launch, a grid barrier between frames) with every input already
resident in device memory.

Workload (default): the 1024-wide MultiCodeDecoder (5 layers, hidden 1024, GQA
16/8 heads of 128, SwiGLU FFN 3072, 15 codebooks of 2048, bf16 weights N(0,
0.02) seed 0), draft length 4, top-k 50, temperature 0.9, batch 1, 1000
frames.  Inputs are synthetic: frame hidden vectors N(0,1), c_0 uniform,
uniforms pre-drawn from seed 1.

With --streams S (2..16) the workload is S independent streams of the same
model verified together (S x (K + 1) rows per pass, stream i with frame seeds
2000 + i and uniform seeds 1000 + i, 500 frames per stream), run as one launch
of the batched kernel through rvqsd_decode_frames_batched_async; `value` is
then the aggregate codes/s of all streams.

With --pipeline the workload is the full per-frame pipeline: the 28-layer outer
CodeDecoder step (KV cache growing to the frame count, 3072-entry head, c_0
sampled with top-k 50) chained on the device with the inner loop (K = 4),
1500 frames through rvqsd_pipeline_frames_async; `value` is then 16 codes per
frame over the wall time.

Prints ONE JSON line.  `roofline` prices the frame kernel against HBM
bandwidth with the algorithmic bytes the device counts per frame (layer
weights per pass, the distinct LM heads a pass touches, gathered embedding
rows, KV cache) divided by the kernel duration from HIP events recorded on the
stream the kernel runs on.  `cpu_baseline` times the CPU oracle on a bounded
sample of the same frames on the host cores.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
METRIC = "RVQ codes/sec single-stream; accepted tok/call; verify-step GB/s vs roofline"
FRAMES_PER_LAUNCH = 1024  # frames per launch of the persistent frame kernel (rvqsd_decode_frames_async)
KERNEL_SOURCES = ("paper_2609_37007_amd/csrc/rvqsd_frame.hip", "paper_2609_37007_amd/csrc/rvqsd_device.h",
                  "paper_2609_37007_amd/csrc/rvqsd_internal.h")
PMC_SUMMARY = os.path.join(ROOT, "profiles", "frame_kernel_mcd1024_k4_fetch_write_counters.txt")

WORKLOADS = {
    # name: (shape, top-k, draft length, frames)
    "mcd1024": ("MCD_1024", 50, 4, 1000),
    "mcd1024-w8": ("MCD_1024_W8", 50, 4, 1000),  # the same model with W8A16 weights (Sec. 3.4)
    "tiny": ("TINY", 8, 3, 32),
}


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def measured_traffic():
    """Bytes per frame that the L2 caches fetched from and wrote to the memory fabric
    (rocprofv3 FETCH_SIZE + WRITE_SIZE of a launch, each scaled by a plain copy, over the
    launch's frames), from the committed counter summary, or None when the summary is
    absent or the kernel sources changed since it was taken. The counters see Infinity
    Cache (MALL) hits as fabric traffic."""
    if not os.path.exists(PMC_SUMMARY):
        return None
    kv = {}
    with open(PMC_SUMMARY) as fh:
        for line in fh:
            if ":" in line and not line.startswith(" "):
                k, v = line.split(":", 1)
                kv[k.strip()] = v.strip()
    if kv.get("kernel_source_sha256") != kernel_source_hash():
        return None
    try:
        return float(kv["fetch_write_bytes_per_frame"])
    except (KeyError, ValueError):
        return None


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None, help="timed frames (default: the workload's frame count)")
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", choices=sorted(WORKLOADS), default="mcd1024")
    ap.add_argument("--draft-len", type=int, default=None)
    ap.add_argument("--head-scale", type=float, default=1.0)
    ap.add_argument("--cpu-seconds", type=float, default=15.0, help="budget of the oracle timing sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--streams", type=int, default=1, help="independent streams verified together (1..16)")
    ap.add_argument("--frames-per-stream", type=int, default=500)
    ap.add_argument("--pipeline", action="store_true", help="outer CodeDecoder step + inner loop per frame")
    ap.add_argument("--offsets", default="seed", metavar="seed|zero|FILE.npy",
                    help="draft offsets: the blob's own N(0, 0.02) draw (seed), all zero (the reused heads of "
                         "Sec. 2.2), or a trained float32 [max_draft][hidden] array")
    ap.add_argument("--tree", default=None, metavar="FILE.json",
                    help="sparse-tree verification (Sec. 2.2, Fig. 2) with the packed tree of FILE (parents, ranks; "
                         "paper_2609_37007_amd/tree.py writes them); the frames then run through the batched "
                         "kernel's tree lane")
    ap.add_argument("--gemv", action="store_true",
                    help="projections and LM heads on the VALU GEMV instead of the matrix cores (cfg matrix_path 1)")
    ap.add_argument("--phases", action="store_true",
                    help="per-phase time of the frame kernel's passes from its per-workgroup clock trace")
    ap.add_argument("--residency", action="store_true",
                    help="only measure whether the weights stay in the Infinity Cache: warm against cold frames "
                         "(a 2 GiB sweep between frames) and a plain streaming read of a weight-sized buffer")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MB",
                    help="only run 5 plain device copies of MB MiB (the reference kernel for HBM byte counters)")
    return ap.parse_args()


def make_blob(S, s, a):
    """The workload's weight blob with the draft offsets chosen by --offsets."""
    import numpy as np
    if a.offsets == "seed":
        return S.make_weights(s, seed=0, head_scale=a.head_scale)
    if a.offsets == "zero":
        return S.make_weights(s, seed=0, head_scale=a.head_scale, offsets=np.zeros((s.max_draft, s.hidden)))
    path = a.offsets if os.path.isabs(a.offsets) else os.path.join(ROOT, a.offsets)
    ofs = np.load(path, allow_pickle=False)
    return S.make_weights(s, seed=0, head_scale=a.head_scale, offsets=ofs)


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def copy_calibration(mb: int) -> int:
    """Plain device-to-device copies of known size: rocprofv3 --pmc FETCH_SIZE / WRITE_SIZE of
    this run give the counter reading per byte moved, used to scale the frame kernel's readings."""
    import torch
    n = mb * (1 << 20) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_per_launch": n * 4, "launches": 5}), flush=True)
    return 0


def oracle_sample(blob, s, topk, temperature, K, f, c0, u, codes, seconds, order, one_thread_seconds=8.0,
                  tree=None):
    """Time the CPU oracle on frames `order` until `seconds` pass (all host threads), then on
    the next frames with one thread for `one_thread_seconds`; returns the cpu_baseline object."""
    from oracle import oracle as O
    orc = O.Oracle(blob, n_layers=s.n_layers, hidden=s.hidden, n_q_heads=s.n_q_heads, n_kv_heads=s.n_kv_heads,
                   head_dim=s.head_dim, ffn=s.ffn, n_codes=s.n_codes, vocab=s.vocab, max_draft=s.max_draft,
                   dtype=s.dtype, topk=topk, temperature=temperature, draft_len=K)
    threads = O.get_threads()
    otree = O.make_tree(*tree) if tree is not None else None
    print(f"[bench] oracle sample on {threads} threads, ~{seconds:.0f} s", file=sys.stderr, flush=True)

    def run(start, budget):
        done, same = 0, 0
        t0 = time.perf_counter()
        while start + done < len(order) and (time.perf_counter() - t0) < budget:
            i = order[start + done]
            if tree is None:
                oc, _, _ = orc.spec_frame(f[i], int(c0[i]), u[i])
            else:
                oc, _, _ = orc.tree_frame(otree, f[i], int(c0[i]), u[i])
            same += int((oc == codes[i]).all())
            done += 1
        return done, same, time.perf_counter() - t0

    done, same, c_el = run(0, seconds)
    one = None
    if one_thread_seconds > 0 and done < len(order):
        O.set_threads(1)
        d1, s1, e1 = run(done, one_thread_seconds)
        O.set_threads(threads)
        if d1:
            one = {"value": round(s.n_codes * d1 / e1, 3), "frames": d1, "seconds": round(e1, 1),
                   "identical_to_gpu": s1}
    orc.close()
    return {"value": round(s.n_codes * done / c_el, 3), "unit": "codes/s", "cores": threads, "kind": "oracle",
            "cpu_model": cpu_model(), "nproc": os.cpu_count(),
            "sample": f"{done} of the timed frames ({c_el:.1f} s on {threads} threads, fp64 full-recompute oracle, "
                      f"OpenMP over output rows); {same}/{done} frames give codes identical to the GPU's",
            "one_thread": one}


def run_pipeline(a) -> int:
    """Outer CodeDecoder step + inner speculative loop per frame, chained on the device."""
    import numpy as np
    import torch

    from oracle import oracle as O
    from paper_2609_37007_amd import rvqsd as R
    from paper_2609_37007_amd import synth as S

    R.lib()
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 1
    so, si = S.OUTER_1024, S.MCD_1024
    topk, K, temperature = 50, (4 if a.draft_len is None else a.draft_len), 0.9
    N = 1500 if a.steps is None else a.steps
    W = max(1, min(a.warmup, 8))
    nc = si.n_codes
    print(f"[bench] building outer and inner weights; {N} frames", file=sys.stderr, flush=True)
    oblob = S.make_weights(so, seed=0)
    iblob = S.make_weights(si, seed=0, head_scale=a.head_scale)
    tables = S.make_outer_tables(so, nc, si.vocab)
    ocfg = R.make_cfg(n_layers=so.n_layers, hidden=so.hidden, n_q_heads=so.n_q_heads, n_kv_heads=so.n_kv_heads,
                      head_dim=so.head_dim, ffn=so.ffn, n_codes=so.n_codes, vocab=so.vocab, max_draft=so.max_draft,
                      dtype=so.dtype, topk=topk, temperature=temperature, draft_len=0)
    icfg = R.make_cfg(n_layers=si.n_layers, hidden=si.hidden, n_q_heads=si.n_q_heads, n_kv_heads=si.n_kv_heads,
                      head_dim=si.head_dim, ffn=si.ffn, n_codes=nc, vocab=si.vocab, max_draft=si.max_draft,
                      dtype=si.dtype, topk=topk, temperature=temperature, draft_len=K)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    torch_stream = torch.cuda.current_stream(dev)
    omodel, imodel = R.Model(oblob, ocfg), R.Model(iblob, icfg)
    info = imodel.info()
    oinfo = omodel.info()
    stream = R.Stream(imodel, hip_stream=torch_stream.cuda_stream)
    outer = R.Outer(omodel, tables, nc, si.vocab, topk, temperature, max(N, W))
    t, u_c0 = S.pipeline_inputs(so, N)
    uni = S.uniforms(N, nc)
    d_t = torch.from_numpy(t).to(dev)
    d_u0 = torch.from_numpy(u_c0).to(dev)
    d_u = torch.from_numpy(np.ascontiguousarray(uni)).to(dev)
    d_codes = torch.full((N, 1 + nc), -1, dtype=torch.int32, device=dev)
    sb = R.STATS_DTYPE.itemsize
    d_st = torch.zeros(N * sb, dtype=torch.uint8, device=dev)

    def run(n):
        outer.pipeline_async(stream, n, d_t.data_ptr(), d_u0.data_ptr(), d_u.data_ptr(), d_codes.data_ptr(),
                             d_st.data_ptr())

    print(f"[bench] warmup {W} frames", file=sys.stderr, flush=True)
    run(W)
    torch.cuda.synchronize()
    outer.reset()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    print(f"[bench] timing {N} frames", file=sys.stderr, flush=True)
    t0 = time.perf_counter()
    ev0.record(torch_stream)
    run(N)
    ev1.record(torch_stream)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    gpu_ms = ev0.elapsed_time(ev1)
    st = np.frombuffer(d_st.cpu().numpy().tobytes(), dtype=R.STATS_DTYPE)
    codes = d_codes.cpu().numpy()
    if (st["status"] != 0).any() or (codes[:, 0] < 0).any():
        bad = int(np.argmax((st["status"] != 0) | (codes[:, 0] < 0)))
        print(f"[bench] frame {bad} failed with status {int(st['status'][bad])}", file=sys.stderr)
        return 1
    # algorithmic bytes: per frame the outer layers and head, the outer KV read (positions 0..i,
    # fp32 k and v), and the inner loop's own count
    H, L = so.hidden, so.n_layers
    outer_w = oinfo["layer_weight_bytes"] + oinfo["head_bytes"]
    kv_b = sum((i + 1) for i in range(N)) * L * so.n_kv_heads * so.head_dim * 2 * 4
    total_b = N * outer_w + kv_b + float(st["weight_bytes"].astype(np.float64).sum())
    achieved = total_b / (gpu_ms * 1e-3) / 1e9
    cpu = None
    if not a.no_cpu_baseline:
        oorc = O.Oracle(oblob, n_layers=so.n_layers, hidden=so.hidden, n_q_heads=so.n_q_heads,
                        n_kv_heads=so.n_kv_heads, head_dim=so.head_dim, ffn=so.ffn, n_codes=so.n_codes,
                        vocab=so.vocab, max_draft=so.max_draft, dtype=so.dtype, topk=topk,
                        temperature=temperature, draft_len=0)
        iorc = O.Oracle(iblob, n_layers=si.n_layers, hidden=si.hidden, n_q_heads=si.n_q_heads,
                        n_kv_heads=si.n_kv_heads, head_dim=si.head_dim, ffn=si.ffn, n_codes=nc, vocab=si.vocab,
                        max_draft=si.max_draft, dtype=si.dtype, topk=topk, temperature=temperature, draft_len=K)
        emb0 = S.unpack_weights(so, oblob)["emb0"]
        tab = S.unpack_outer_tables(so, tables, nc, si.vocab)
        threads = O.get_threads()
        print(f"[bench] oracle pipeline sample on {threads} threads, ~{a.cpu_seconds:.0f} s", file=sys.stderr,
              flush=True)
        done = min(N, 3)
        c_t0 = time.perf_counter()
        oc, _, _ = O.pipeline_frames(oorc, emb0, tab, iorc, t[:done], u_c0[:done], uni[:done], topk, temperature)
        c_el = time.perf_counter() - c_t0
        same = int(sum((oc[i] == codes[i]).all() for i in range(done)))
        oorc.close()
        iorc.close()
        cpu = {"value": round((nc + 1) * done / c_el, 3), "unit": "codes/s", "cores": threads, "kind": "oracle",
               "sample": f"the first {done} frames of the timed run through the fp64 oracle pipeline ({c_el:.1f} s, "
                         f"outer decoder recomputed over all earlier positions each frame); {same}/{done} frames give "
                         f"codes identical to the GPU's"}
    out = {
        "metric": METRIC,
        "value": round((nc + 1) * N / elapsed, 1),
        "unit": "codes/s",
        "n_gpus": 1,
        "steps": N,
        "warmup": W,
        "ms_per_step": round(elapsed * 1e3 / N, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (random-init weights, seeded text-side vectors and uniforms)",
        "config": {
            "workload": (f"pipeline: outer {so.n_layers}-layer CodeDecoder (hidden {so.hidden}, {so.n_q_heads}/"
                         f"{so.n_kv_heads} heads x {so.head_dim}, ffn {so.ffn}, {so.vocab}-entry head, KV to {N} "
                         f"positions, c0 top-k {topk}) + inner mcd1024 (draft length {K}, top-k {topk}), "
                         f"temperature {temperature}, batch 1, {N} frames"),
            "frames": N,
            "draft_len": K,
            "topk": topk,
            "temperature": temperature,
            "parallelism": "single GPU, one persistent launch per outer step and per inner frame",
        },
        "frames_per_s": round(N / elapsed, 2),
        "real_time_factor": round(N / elapsed / 12.5, 2),
        "frame_ms_mean": round(gpu_ms / N, 4),
        "accepted_tokens_per_call": round(nc * N / float(st["target_calls"].sum()), 4),
        "roofline": {
            "bound": "hbm",
            "achieved": round(achieved, 1),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4),
            "traffic": None,
            "kernel": "outer_flow_kernel + frame_kernel",
            "algorithmic_bytes_per_frame": round(total_b / N, 1),
        },
        "cpu_baseline": cpu,
        "device": torch.cuda.get_device_name(dev),
        "workgroups": info["workgroups"],
    }
    del d_t, d_u0, d_u, d_codes, d_st
    torch.cuda.synchronize()
    outer.close()
    stream.close()
    imodel.close()
    omodel.close()
    torch.cuda.empty_cache()
    print(json.dumps(out), flush=True)
    return 0


def run_streams(a) -> int:
    """S streams verified together by the batched kernel: one launch for all frames."""
    import numpy as np
    import torch

    from paper_2609_37007_amd import rvqsd as R
    from paper_2609_37007_amd import synth as S

    R.lib()
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 1
    s = S.MCD_1024
    topk, K = 50, (4 if a.draft_len is None else a.draft_len)
    temperature = 0.9
    ns, per = a.streams, a.frames_per_stream
    n = s.n_codes
    print(f"[bench] building weights; {ns} streams x {per} frames", file=sys.stderr, flush=True)
    blob = S.make_weights(s, seed=0, head_scale=a.head_scale)
    cfg = R.make_cfg(n_layers=s.n_layers, hidden=s.hidden, n_q_heads=s.n_q_heads, n_kv_heads=s.n_kv_heads,
                     head_dim=s.head_dim, ffn=s.ffn, n_codes=n, vocab=s.vocab, max_draft=s.max_draft,
                     dtype=s.dtype, topk=topk, temperature=temperature, draft_len=K, matrix_path=1 if a.gemv else 0)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    torch_stream = torch.cuda.current_stream(dev)
    model = R.Model(blob, cfg)
    info = model.info()
    stream = R.Stream(model, hip_stream=torch_stream.cuda_stream, max_streams=ns)
    # frame j of stream i is batched frame j * ns + i (lane i decodes stream i in order)
    N = ns * per
    f = np.zeros((N, s.hidden), dtype=np.float32)
    c0 = np.zeros(N, dtype=np.int32)
    u = np.zeros((N, n, 3), dtype=np.float32)
    for i in range(ns):
        fi, ci = S.frame_inputs(s, per, seed_hidden=2000 + i, seed_c0=3000 + i)
        f[i::ns], c0[i::ns], u[i::ns] = fi, ci, S.uniforms(per, n, seed=1000 + i)
    d_f = torch.from_numpy(f).to(dev)
    d_c0 = torch.from_numpy(c0).to(dev)
    d_u = torch.from_numpy(u).to(dev)
    d_codes = torch.full((N, n), -1, dtype=torch.int32, device=dev)
    sb = R.STATS_DTYPE.itemsize
    d_stats = torch.zeros(N * sb, dtype=torch.uint8, device=dev)

    def launch(count):
        stream.decode_frames_batched_async(count, d_f.data_ptr(), d_c0.data_ptr(), d_u.data_ptr(),
                                           d_codes.data_ptr(), d_stats.data_ptr())

    W = max(1, a.warmup) * ns
    print(f"[bench] warmup {min(W, N)} frames", file=sys.stderr, flush=True)
    launch(min(W, N))
    torch.cuda.synchronize()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    print(f"[bench] timing {N} frames", file=sys.stderr, flush=True)
    t0 = time.perf_counter()
    ev0.record(torch_stream)
    launch(N)
    ev1.record(torch_stream)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    launch_ms = ev0.elapsed_time(ev1)
    passes, nbytes = stream.batch_totals()
    st = np.frombuffer(d_stats.cpu().numpy().tobytes(), dtype=R.STATS_DTYPE)
    codes = d_codes.cpu().numpy()
    if (st["status"] != 0).any():
        bad = int(np.argmax(st["status"] != 0))
        print(f"[bench] frame {bad} failed with status {int(st['status'][bad])}", file=sys.stderr)
        return 1
    calls = int(st["target_calls"].sum())
    achieved = nbytes / (launch_ms * 1e-3) / 1e9
    cpu = None
    if not a.no_cpu_baseline:
        order = list(range(0, N, max(1, N // 64)))
        cpu = oracle_sample(blob, s, topk, temperature, K, f, c0, u, codes, a.cpu_seconds, order)
    out = {
        "metric": METRIC,
        "value": round(n * N / elapsed, 1),
        "unit": "codes/s",
        "n_gpus": 1,
        "steps": N,
        "warmup": min(W, N),
        "ms_per_step": round(elapsed * 1e3 / N, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (random-init weights, seeded frame inputs and uniforms per stream)",
        "config": {
            "workload": (f"mcd1024 x {ns} streams: {s.n_layers} layers, hidden {s.hidden}, {s.n_q_heads}/"
                         f"{s.n_kv_heads} heads x {s.head_dim}, ffn {s.ffn}, {n} codebooks of {s.vocab}, bf16 "
                         f"weights; draft length {K}, top-k {topk}, temperature {temperature}; {ns} independent "
                         f"streams verified together ({ns * max(K + 1, 2)} rows per pass), {per} frames each"),
            "frames": N,
            "streams": ns,
            "draft_len": K,
            "topk": topk,
            "temperature": temperature,
            "head_scale": a.head_scale,
            "parallelism": "single GPU, one persistent workgroup per compute unit, one launch for all frames",
        },
        "per_stream_codes_per_s": round(n * N / elapsed / ns, 1),
        "accepted_tokens_per_call": round(n * N / calls, 4),
        "passes": passes,
        "pass_us_mean": round(launch_ms * 1e3 / passes, 2),
        "roofline": {
            "bound": "hbm",
            "achieved": round(achieved, 1),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4),
            "traffic": None,
            "kernel": "batch_kernel",
            "algorithmic_bytes_per_launch": float(nbytes),
            "algorithmic_bytes_per_pass": round(nbytes / passes, 1),
            "launch_ms_mean": round(launch_ms, 4),
        },
        "cpu_baseline": cpu,
        "device": torch.cuda.get_device_name(dev),
        "workgroups": info["workgroups"],
    }
    del d_f, d_c0, d_u, d_codes, d_stats
    torch.cuda.synchronize()
    stream.close()
    model.close()
    torch.cuda.empty_cache()
    print(json.dumps(out), flush=True)
    return 0


def stream_read_rates(torch, dev, ts, nbytes, reps=20):
    """The box's own streaming-read rate: torch.sum over a buffer of nbytes, warm (read back
    to back, so it sits in the Infinity Cache when it fits) and cold (a 2 GiB read-and-write
    sweep of another buffer before each read). GB/s."""
    buf = torch.ones(nbytes // 4, dtype=torch.float32, device=dev)
    sweep = torch.ones(1 << 28, dtype=torch.float32, device=dev)
    out = torch.empty((), dtype=torch.float32, device=dev)

    def rate(evict, n):
        t = 0.0
        for _ in range(n):
            if evict:
                sweep.add_(1.0)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(ts)
            torch.sum(buf, dim=0, out=out)
            e1.record(ts)
            torch.cuda.synchronize()
            t += e0.elapsed_time(e1) * 1e-3
        return buf.numel() * 4 * n / t / 1e9

    rate(False, 3)
    res = {"bytes": buf.numel() * 4, "warm": round(rate(False, reps), 1), "cold": round(rate(True, reps), 1)}
    del buf, sweep, out
    torch.cuda.empty_cache()
    return res


def run_residency(a) -> int:
    """Whether the frame kernel's weights stay in the 256 MB Infinity Cache (MALL).

    * warm: frames back to back (the weights of one pass are the weights of the next);
    * cold: a 2 GiB read-and-write sweep of a separate buffer before each frame, so the
      frame's first pass reads its weights from HBM; every pass of a frame is clocked by
      the kernel's own trace (device clock at the end of each pass);
    * stream: plain torch reductions over a buffer of the round's weight bytes, warm
      (repeated) and cold (after the same sweep): the box's cache and HBM read rates."""
    import numpy as np
    import torch

    from paper_2609_37007_amd import rvqsd as R
    from paper_2609_37007_amd import synth as S

    R.lib()
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 1
    shape_name, topk, K_default, _ = WORKLOADS[a.workload]
    s = getattr(S, shape_name)
    K = K_default if a.draft_len is None else a.draft_len
    blob = make_blob(S, s, a)
    cfg = R.make_cfg(n_layers=s.n_layers, hidden=s.hidden, n_q_heads=s.n_q_heads, n_kv_heads=s.n_kv_heads,
                     head_dim=s.head_dim, ffn=s.ffn, n_codes=s.n_codes, vocab=s.vocab, max_draft=s.max_draft,
                     dtype=s.dtype, topk=topk, temperature=0.9, draft_len=K)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    ts = torch.cuda.current_stream(dev)
    model = R.Model(blob, cfg)
    stream = R.Stream(model, hip_stream=ts.cuda_stream)
    F = a.steps or 100
    f, c0 = S.frame_inputs(s, F)
    u = S.uniforms(F, s.n_codes)
    d_f, d_c0 = torch.from_numpy(f).to(dev), torch.from_numpy(c0).to(dev)
    d_u = torch.from_numpy(np.ascontiguousarray(u)).to(dev)
    n, H, sb = s.n_codes, s.hidden, R.STATS_DTYPE.itemsize
    d_codes = torch.zeros((F, n), dtype=torch.int32, device=dev)
    d_st = torch.zeros(F * sb, dtype=torch.uint8, device=dev)
    nph = 5 * s.n_layers + 5
    clk = torch.zeros((16, nph), dtype=torch.int64, device=dev)
    sweep = torch.ones(1 << 28, dtype=torch.float32, device=dev)  # 1 GiB, read and written: 2 GiB through the cache

    def frame(i, evict):
        if evict:
            sweep.add_(1.0)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        clk.zero_()
        stream.set_trace(0, 0, clk.data_ptr(), 16)
        e0.record(ts)
        stream.decode_frame_async(d_f.data_ptr() + i * H * 4, d_c0.data_ptr() + i * 4, d_u.data_ptr() + i * n * 12,
                                  d_codes.data_ptr() + i * n * 4, d_st.data_ptr() + i * sb)
        e1.record(ts)
        torch.cuda.synchronize()
        st = np.frombuffer(d_st[i * sb:(i + 1) * sb].cpu().numpy().tobytes(), dtype=R.STATS_DTYPE)[0]
        c = clk.cpu().numpy()[:int(st["target_calls"]), 5 * s.n_layers + 2].astype(np.float64)  # commit end
        start = float(st["clk_start"])
        passes = np.diff(np.concatenate([[start], c])) * 0.01  # 100 MHz clock -> us
        return e0.elapsed_time(e1) * 1e3, passes

    for i in range(5):
        frame(i, False)
    res = {}
    for mode, evict in (("warm", False), ("cold", True)):
        print(f"[bench] residency: {mode} frames", file=sys.stderr, flush=True)
        fr, p0, rest = [], [], []
        for i in range(F):
            us, passes = frame(i, evict)
            fr.append(us)
            p0.append(passes[0])
            rest.extend(passes[1:])
        res[mode] = {"frame_us_mean": round(float(np.mean(fr)), 2), "first_pass_us_mean": round(float(np.mean(p0)), 2),
                     "later_pass_us_mean": round(float(np.mean(rest)), 2), "frames": F}
    stream.set_trace()
    # plain streaming reads of a buffer the size of one round's weights
    wb = int(model.info()["layer_weight_bytes"] + 9 * model.info()["head_bytes"])
    del sweep
    res["stream_read_gbs"] = stream_read_rates(torch, dev, ts, wb)
    w, c = res["warm"], res["cold"]
    res["first_pass_extra_us_cold"] = round(c["first_pass_us_mean"] - w["first_pass_us_mean"], 2)
    res["later_pass_extra_us_cold"] = round(c["later_pass_us_mean"] - w["later_pass_us_mean"], 2)
    res["workload"] = f"{a.workload}, draft length {K}, offsets {a.offsets}"
    res["weight_bytes_per_round"] = wb
    stream.close()
    model.close()
    print(json.dumps({"residency": res}), flush=True)
    return 0


def run_phases(a) -> int:
    """Where a pass of the frame kernel spends its time, phase by phase.

    Every workgroup stamps the device clock (100 MHz) when the input of a phase is complete
    ("ready") and when it leaves the phase ("end"). Per phase and pass:
    * path: the increment of the latest end over all workgroups (the critical path);
    * wait: median over the phase's workgroups of ready minus that workgroup's previous end;
    * work: median of end minus ready;
    * exchange: ready minus the latest end among the workgroups that worked in the phase
      before (median and minimum over the consumers): the cost of handing the data over.
    Passes after the prefix pass of frames 5.. (the first frames warm the clocks up)."""
    import numpy as np
    import torch

    from paper_2609_37007_amd import rvqsd as R
    from paper_2609_37007_amd import synth as S

    R.lib()
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 1
    shape_name, topk, K_default, _ = WORKLOADS[a.workload]
    s = getattr(S, shape_name)
    K = K_default if a.draft_len is None else a.draft_len
    blob = make_blob(S, s, a)
    cfg = R.make_cfg(n_layers=s.n_layers, hidden=s.hidden, n_q_heads=s.n_q_heads, n_kv_heads=s.n_kv_heads,
                     head_dim=s.head_dim, ffn=s.ffn, n_codes=s.n_codes, vocab=s.vocab, max_draft=s.max_draft,
                     dtype=s.dtype, topk=topk, temperature=0.9, draft_len=K, matrix_path=1 if a.gemv else 0)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    ts = torch.cuda.current_stream(dev)
    model = R.Model(blob, cfg)
    nwg = int(model.info()["workgroups"])
    stream = R.Stream(model, hip_stream=ts.cuda_stream)
    F = a.steps or 60
    f, c0 = S.frame_inputs(s, F)
    u = S.uniforms(F, s.n_codes)
    L, n, H = s.n_layers, s.n_codes, s.hidden
    nph, MAXR = 5 * L + 5, 16
    names = [f"L{l}.{p}" for l in range(L) for p in ("qkv", "attn", "o", "gu", "down")] + ["heads", "sample", "commit"]
    wg = torch.zeros(MAXR * nph * nwg, dtype=torch.int64, device=dev)
    rd = torch.zeros(MAXR * nph * nwg, dtype=torch.int64, device=dev)
    stream.set_trace(wg_clock_ptr=wg.data_ptr(), wg_ready_ptr=rd.data_ptr(), max_rounds=MAXR)
    d_f, d_c0 = torch.from_numpy(f).to(dev), torch.from_numpy(c0).to(dev)
    d_u = torch.from_numpy(np.ascontiguousarray(u)).to(dev)
    sb = R.STATS_DTYPE.itemsize
    d_codes = torch.zeros((1, n), dtype=torch.int32, device=dev)
    d_st = torch.zeros(sb, dtype=torch.uint8, device=dev)
    nrow = len(names)
    path, wait, work, total = [[] for _ in range(nrow)], [[] for _ in range(nrow)], [[] for _ in range(nrow)], []
    # exchange: consumer input complete minus the last end of the previous phase's workers
    xmed, xmin = [[] for _ in range(nrow)], [[] for _ in range(nrow)]
    print(f"[bench] phase trace over {F} frames", file=sys.stderr, flush=True)
    for i in range(F):
        wg.zero_()
        rd.zero_()
        stream.decode_frame_async(d_f.data_ptr() + i * H * 4, d_c0.data_ptr() + i * 4, d_u.data_ptr() + i * n * 12,
                                  d_codes.data_ptr(), d_st.data_ptr())
        torch.cuda.synchronize()
        st = np.frombuffer(d_st.cpu().numpy().tobytes(), dtype=R.STATS_DTYPE)[0]
        if int(st["status"]) != 0:
            print(f"[bench] frame {i} failed with status {int(st['status'])}", file=sys.stderr)
            return 1
        if i < 5:
            continue
        w = wg.cpu().numpy().reshape(MAXR, nph, nwg).astype(np.int64)
        r = rd.cpu().numpy().reshape(MAXR, nph, nwg).astype(np.int64)
        for p in range(1, min(int(st["target_calls"]), MAXR)):
            prev_end = w[p - 1, nrow - 1]
            total.append((w[p, nrow - 1].max() - w[p - 1, nrow - 1].max()) * 0.01)
            for ph in range(nrow):
                e = w[p, ph]
                path[ph].append((e.max() - prev_end.max()) * 0.01)
                ok = r[p, ph] > 0
                if ok.any():
                    wait[ph].append(np.median((r[p, ph] - prev_end)[ok]) * 0.01)
                    work[ph].append(np.median((e - r[p, ph])[ok]) * 0.01)
                    workers = r[p, ph - 1] > 0 if ph > 0 else np.zeros(nwg, dtype=bool)
                    if workers.any():
                        last = prev_end[workers].max()
                        xmed[ph].append(np.median(r[p, ph][ok] - last) * 0.01)
                        xmin[ph].append(np.min(r[p, ph][ok] - last) * 0.01)
                prev_end = e
    stream.set_trace()
    stream.close()
    model.close()
    rows = []
    for ph in range(nrow):
        rows.append({"phase": names[ph], "path_us": round(float(np.mean(path[ph])), 2),
                     "wait_us": round(float(np.mean(wait[ph])), 2) if wait[ph] else None,
                     "work_us": round(float(np.mean(work[ph])), 2) if work[ph] else None,
                     "exchange_median_us": round(float(np.mean(xmed[ph])), 2) if xmed[ph] else None,
                     "exchange_min_us": round(float(np.mean(xmin[ph])), 2) if xmin[ph] else None})
    for row in rows:
        print(f"{row['phase']:8s} path {row['path_us']:6.2f}  wait {row['wait_us'] if row['wait_us'] is not None else '-':>6}"
              f"  work {row['work_us'] if row['work_us'] is not None else '-':>6}", file=sys.stderr)
    print(json.dumps({"phases": rows, "pass_us_mean": round(float(np.mean(total)), 2), "passes": len(total),
                      "workload": f"{a.workload}, draft length {K}"}), flush=True)
    return 0


def main() -> int:
    a = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if a.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: the decode of a stream runs on a single GPU and this library "
              "has no multi-GPU path (independent streams would shard across GPUs with no exchange). "
              "Run with --gpus 1.", file=sys.stderr)
        return 2
    if a.copy_calibration:
        return copy_calibration(a.copy_calibration)
    if a.streams > 1:
        return run_streams(a)
    if a.pipeline:
        return run_pipeline(a)
    if a.residency:
        return run_residency(a)
    if a.phases:
        return run_phases(a)

    import numpy as np
    import torch

    from paper_2609_37007_amd import rvqsd as R
    from paper_2609_37007_amd import synth as S

    R.lib()
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 1
    shape_name, topk, K_default, frames_default = WORKLOADS[a.workload]
    s = getattr(S, shape_name)
    K = K_default if a.draft_len is None else a.draft_len
    steps = frames_default if a.steps is None else a.steps
    W = a.warmup
    temperature = 0.9
    print(f"[bench] building {a.workload} weights", file=sys.stderr, flush=True)
    blob = make_blob(S, s, a)
    blob_sha = hashlib.sha256(blob).hexdigest()[:16]
    cfg = R.make_cfg(n_layers=s.n_layers, hidden=s.hidden, n_q_heads=s.n_q_heads, n_kv_heads=s.n_kv_heads,
                     head_dim=s.head_dim, ffn=s.ffn, n_codes=s.n_codes, vocab=s.vocab, max_draft=s.max_draft,
                     dtype=s.dtype, topk=topk, temperature=temperature, draft_len=K, matrix_path=1 if a.gemv else 0)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    torch_stream = torch.cuda.current_stream(dev)
    model = R.Model(blob, cfg)
    info = model.info()
    tree = None
    if a.tree:
        with open(a.tree if os.path.isabs(a.tree) else os.path.join(ROOT, a.tree)) as fh:
            tj = json.load(fh)
        tree = (tj["parents"], tj["ranks"])
    stream = R.Stream(model, hip_stream=torch_stream.cuda_stream, tree=tree)

    f, c0 = S.frame_inputs(s, steps)
    u = S.uniforms(steps, s.n_codes)
    d_f = torch.from_numpy(f).to(dev)
    d_c0 = torch.from_numpy(c0).to(dev)
    d_u = torch.from_numpy(np.ascontiguousarray(u)).to(dev)
    d_codes = torch.full((steps, s.n_codes), -1, dtype=torch.int32, device=dev)
    sb = R.STATS_DTYPE.itemsize
    d_stats = torch.zeros(steps * sb, dtype=torch.uint8, device=dev)
    H, n = s.hidden, s.n_codes

    def launch(i0, cnt):
        # frames i0 .. i0 + cnt - 1, up to 1024 per launch of the persistent kernel
        stream.decode_frames_async(cnt, d_f.data_ptr() + i0 * H * 4, d_c0.data_ptr() + i0 * 4,
                                   d_u.data_ptr() + i0 * n * 3 * 4, d_codes.data_ptr() + i0 * n * 4,
                                   d_stats.data_ptr() + i0 * sb)

    print(f"[bench] warmup {W} frames", file=sys.stderr, flush=True)
    for i0 in range(0, W, steps):
        launch(0, min(steps, W - i0))
    torch.cuda.synchronize()
    ws = np.frombuffer(d_stats.cpu().numpy().tobytes(), dtype=R.STATS_DTYPE)[:min(W, steps)]
    if (ws["status"] != 0).any():
        print(f"[bench] warmup frame failed: status {ws['status'].tolist()}", file=sys.stderr)
        return 1

    # a tree stream decodes through the batched kernel, one launch per frame
    fpl = 1 if tree else FRAMES_PER_LAUNCH
    n_launch = (steps + fpl - 1) // fpl
    ev0 = [torch.cuda.Event(enable_timing=True) for _ in range(n_launch)]
    ev1 = [torch.cuda.Event(enable_timing=True) for _ in range(n_launch)]
    print(f"[bench] timing {steps} frames in {n_launch} launch(es)", file=sys.stderr, flush=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for j in range(n_launch):
        i0 = j * fpl
        ev0[j].record(torch_stream)
        launch(i0, min(fpl, steps - i0))
        ev1[j].record(torch_stream)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    elapsed = t1 - t0

    st = np.frombuffer(d_stats.cpu().numpy().tobytes(), dtype=R.STATS_DTYPE)
    codes = d_codes.cpu().numpy()
    if (st["status"] != 0).any():
        bad = int(np.argmax(st["status"] != 0))
        print(f"[bench] frame {bad} failed with status {int(st['status'][bad])}", file=sys.stderr)
        return 1
    launch_ms = np.array([ev0[j].elapsed_time(ev1[j]) for j in range(n_launch)])
    calls = int(st["target_calls"].sum())
    rounds = int(st["rounds"].sum())
    frame_bytes = st["weight_bytes"].astype(np.float64)
    achieved = float(frame_bytes.sum() / (launch_ms.sum() * 1e-3) / 1e9)
    frames_per_launch = steps / n_launch
    # each frame's device time (its stats clock, 100 MHz)
    frame_ms = (st["clk_end"].astype(np.float64) - st["clk_start"].astype(np.float64)) / 1e5
    traffic = measured_traffic() if (a.workload == "mcd1024" and K == 4 and a.head_scale == 1.0 and not tree
                                     and a.offsets == "seed" and not a.gemv) else None
    if traffic is not None:
        traffic = round(traffic * frames_per_launch, 1)
    codes_per_s = n * steps / elapsed
    # the box's own read rates for a buffer of one launch's mean bytes per pass
    box = stream_read_rates(torch, dev, torch_stream, int(frame_bytes.sum() / calls) & ~255)

    cpu = None
    if not a.no_cpu_baseline:
        cpu = oracle_sample(blob, s, topk, temperature, K, f, c0, u, codes, a.cpu_seconds, list(range(steps)),
                            tree=tree)

    out = {
        "metric": METRIC,
        "value": round(codes_per_s, 1),
        "unit": "codes/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": W,
        "ms_per_step": round(elapsed * 1e3 / steps, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": {S.DTYPE_BF16: "bf16", S.DTYPE_I8: "int8 weights (W8A16), fp32 activations"}.get(s.dtype, "f32"),
        "data": "synthetic (random-init weights, seeded frame inputs and uniforms)",
        "config": {
            "workload": (f"{a.workload}: {s.n_layers} layers, hidden {s.hidden}, {s.n_q_heads}/{s.n_kv_heads} heads "
                         f"x {s.head_dim}, ffn {s.ffn}, {s.n_codes} codebooks of {s.vocab}, "
                         f"{ {S.DTYPE_BF16: 'bf16', S.DTYPE_I8: 'int8 (per-channel scales)'}.get(s.dtype, 'fp32')} weights; "
                         + (f"sparse tree of {len(tree[0])} nodes, depth {K}" if tree else f"draft length {K}")
                         + f", top-k {topk}, temperature {temperature}, batch 1"),
            "tree_nodes": len(tree[0]) if tree else 0,
            "frames": steps,
            "draft_len": K,
            "topk": topk,
            "temperature": temperature,
            "head_scale": a.head_scale,
            "offsets": a.offsets,
            "batch": 1,
            "weights_sha256_16": blob_sha,
            "parallelism": "single GPU, one persistent workgroup per compute unit",
            "matrix_path": "VALU GEMV" if a.gemv else "matrix cores when the pass has at most 8 rows",
        },
        "accepted_tokens_per_call": round(n * steps / calls, 4),
        "mean_tokens_per_round": round((n * steps - steps) / max(rounds, 1), 4),
        "accept_rate": round(float(st["accepted"].sum()) / max(int(st["drafted"].sum()), 1), 4),
        "target_calls_per_frame": round(calls / steps, 3),
        "frame_ms_p50": round(float(np.median(frame_ms)), 4),
        "pass_us_mean": round(float(launch_ms.sum() * 1e3 / calls), 2),
        "roofline": {
            "bound": "hbm",
            "achieved": round(achieved, 1),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4),
            "traffic": traffic,
            "kernel": "batch_kernel" if tree else "frame_kernel",
            "algorithmic_bytes_per_launch": round(float(frame_bytes.sum() / n_launch), 1),
            "launch_ms_mean": round(float(launch_ms.mean()), 5),
            "frames_per_launch": round(frames_per_launch, 2),
            "traffic_counts": "L2-to-fabric bytes (FETCH_SIZE + WRITE_SIZE, Infinity Cache hits included)",
            "box_read_gbs": {"warm": box["warm"], "cold": box["cold"], "bytes": box["bytes"],
                             "how": "torch.sum over one pass's bytes: warm = back to back (Infinity Cache), "
                                    "cold = after a 2 GiB sweep (HBM)"},
            "frac_of_box_warm_read": round(achieved / box["warm"], 4),
        },
        "cpu_baseline": cpu,
        "device": torch.cuda.get_device_name(dev),
        "workgroups": info["workgroups"],
    }
    # release device memory before the interpreter exits
    del ev0, ev1, d_f, d_c0, d_u, d_codes, d_stats
    torch.cuda.synchronize()
    stream.close()
    model.close()
    torch.cuda.empty_cache()
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    # success ends by returning from the script (a profiler attached to the
    # process then still writes its results); failures exit with their code
    rc = main()
    if rc:
        sys.exit(rc)
