#!/usr/bin/env python3
"""Benchmark of the fused quantized AdamW step on one MI355X.

Workload: the Llama-7B-shaped parameter list (291 tensors, 6,738,415,616
params): fp32 master params, bf16 grads N(0, 1e-3) with a fixed 1% exact-zero
mask (generated once, reused every step), AL8 second moment (block B_V) and
UF8 momentum (block 256), all resident in HBM. W warm-up steps, then K timed
steps with HIP events on the launch stream. The headline is B_V = 2048, the
second-moment block of the paper's AdamW configuration (Table 4); the
block-size sweep {64, 128, 256, 512, 1024, 2048} is reported alongside, as are the
measured streaming rates of the same byte mix (al_diag_stream: the step's access
shape, and the fastest shape found for the mix).

Prints ONE JSON line on stdout (progress goes to stderr).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "optimizer-step Gparams/s + achieved HBM GB/s (% of peak), AL8 AdamW"
PEAK_GBS = 8000.0
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "adamw_llama7b_traffic.json")
KERNEL_SOURCES = ("paper_2608_22322_amd/csrc/adamw.hip", "paper_2608_22322_amd/csrc/al_device.hpp")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def adamw_bytes_per_param(block_v: int, grad_bytes: int = 2, v_code_bytes: int = 1) -> float:
    """Algorithmic HBM bytes per parameter of one AdamW step: read+write p (fp32), read g, read+write m
    codes (1 B) and its absmax per 256, read+write v codes and its {l_min, delta} per B_V."""
    return 4 + 4 + grad_bytes + 1 + 1 + 2 * 4 / 256 + 2 * v_code_bytes + 2 * 8 / block_v


def kernel_hash() -> str:
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        h.update(open(os.path.join(ROOT, f), "rb").read())
    return h.hexdigest()[:16]


def measured_traffic(block_v: int):
    """Measured HBM bytes per launch (rocprofv3 FETCH_SIZE + WRITE_SIZE, calibrated on al_diag_stream), if the
    counters were taken on the current kernel source."""
    try:
        t = json.load(open(TRAFFIC_FILE))
    except (OSError, ValueError):
        return None
    if t.get("kernel_hash") != kernel_hash():
        return None
    return t.get("bytes_per_launch", {}).get(str(block_v))


def build_states(shapes, dev, block_v):
    import torch

    import paper_2608_22322_amd as al
    from paper_2608_22322_amd import data
    from paper_2608_22322_amd.workloads import workload_llama7b

    w = workload_llama7b()
    floor = al.log2_floor_of(1e-8 * 1e-8)
    states = []
    for i, s in enumerate(shapes):
        p = data.device_param(i, s, dev)
        g = data.device_grad_buffer(s, w, dev)
        data.fill_grad(g, i, s, w, 1)
        m, mm = al.alloc_state(s.n, al.Spec(al.UF8, 256), dev)
        v, vm = al.alloc_state(s.n, al.Spec(al.AL8, block_v, floor), dev)
        states.append(al.ParamState(p, g, s.rows, s.cols, m=m, m_meta=mm, v=v, v_meta=vm))
    torch.cuda.synchronize()
    return states


def time_adamw(states, block_v, steps, warmup):
    import torch

    import paper_2608_22322_amd as al

    floor = al.log2_floor_of(1e-8 * 1e-8)
    for st in states:  # fresh state for this block size
        st.m.zero_()
        st.m_meta.zero_()
        st.v.zero_()
        mf = al.meta_floats(al.AL8, st.rows * st.cols, block_v)
        if st.v_meta.numel() < mf:
            st.v_meta = torch.zeros(mf, dtype=torch.float32, device=st.v.device)
        else:
            st.v_meta.zero_()
    cfg = al.adamw_cfg(m=al.Spec(al.UF8, 256), v=al.Spec(al.AL8, block_v, floor))
    arr = al.tensor_array(states)
    ws = al.workspace(al.adamw_workspace_bytes(states, cfg, arr=arr))
    stream = torch.cuda.current_stream()
    t = 0
    for _ in range(warmup):
        t += 1
        al.adamw_step(states, cfg, t, ws, stream=stream, arr=arr)
    torch.cuda.synchronize()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    for k in range(steps):
        t += 1
        evs[k][0].record(stream)
        al.adamw_step(states, cfg, t, ws, stream=stream, arr=arr)
        evs[k][1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    ms = [a.elapsed_time(b) for a, b in evs]
    return ms, wall


def copy_ceiling(n, steps=10):
    """Streaming rates of the AdamW byte mix (al_diag_stream: read p/g/m/v, write p/m/v, no arithmetic) on flat
    buffers of n elements: the step's own access shape (ordinary and non-temporal) and the fastest shape found
    for the mix (4096-element chunks, 16 bytes per lane from every stream, all loads before any store)."""
    import torch

    import paper_2608_22322_amd as al

    n = n // 4096 * 4096
    p = torch.zeros(n, dtype=torch.float32, device="cuda")
    g = torch.zeros(n, dtype=torch.bfloat16, device="cuda")
    m = torch.zeros(n, dtype=torch.uint8, device="cuda")
    v = torch.zeros(n, dtype=torch.uint8, device="cuda")
    out = {}
    for name, nt, wide in (("step_shape", False, False), ("step_shape_nt", True, False), ("wide", True, True)):
        for _ in range(2):
            al.diag_stream(nt, p, g, m, v, wide=wide)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(steps):
            al.diag_stream(nt, p, g, m, v, wide=wide)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / steps
        out[name] = round(14 * n / (ms * 1e-3) / 1e9, 1)
    del p, g, m, v
    torch.cuda.empty_cache()
    out["bytes_per_elem"] = 14
    out["elems"] = n
    return out


def factored_bytes_per_param(shapes, came: bool):
    """(algorithmic, multi-pass schedule) HBM bytes per parameter of one Adafactor / CAME step on a tensor
    list: p read+write 8, g 2, (CAME) m codes read+write 2 plus its absmax per 256; the factored vectors add
    2 (rows + cols) x (code + meta) per 2-D tensor. The schedule re-reads g (Adafactor: marginals, RMS,
    update = 3x; CAME: 4x) and (CAME) m once more."""
    n = sum(s.n for s in shapes)
    vec = 0.0
    for s in shapes:
        if s.is_2d:
            k = 2 if came else 1  # CAME: V and confidence factors
            vec += k * 2 * (s.rows + s.cols) * (2 if came else 1)  # codes read + write (AL16 2 B, AL8 1 B)
        else:
            vec += 2 * s.n * (2 if came else 1)
    m = (2 + 8 / 256) if came else 0.0
    alg = 8 + 2 + m + vec / n
    sched = alg + (3 if came else 2) * 2 + (1 if came else 0)
    return alg, sched


def time_factored(came: bool, steps: int, warmup: int, llama7b: bool = False):
    """One Adafactor (AL8 B256 factored + 1-D, no zero mask) or CAME (AL16 B128 V and confidence, UF8 m,
    2% zeros) step over the TinyLlama-1.1B list (or the Llama-7B list), grads generated once."""
    import torch

    import paper_2608_22322_amd as al
    from paper_2608_22322_amd import data
    from paper_2608_22322_amd.workloads import Workload, llama7b_shapes, tinyllama_shapes, workload_tinyllama

    shapes = llama7b_shapes() if llama7b else tinyllama_shapes()
    w = (Workload("llama-7b", shapes, zero_frac=0.02 if came else 0.0, steps=20) if llama7b else
         workload_tinyllama(zero_frac=0.02 if came else 0.0))
    dev = torch.device("cuda:0")
    if came:
        cfg = al.came_cfg()
        vs, ms, cs = al.Spec(al.AL16, 128, al.log2_floor_of(1e-30)), al.Spec(al.UF8, 256), \
            al.Spec(al.AL16, 128, al.log2_floor_of(1e-16))
    else:
        cfg = al.adafactor_cfg()
        vs = al.Spec(al.AL8, 256, al.log2_floor_of(1e-30))
    states = []
    for i, s in enumerate(shapes):
        st = al.ParamState(data.device_param(i, s, dev), data.device_grad_buffer(s, w, dev), s.rows, s.cols)
        data.fill_grad(st.grad, i, s, w, 1)
        if s.is_2d:
            st.vr, st.vr_meta = al.alloc_state(s.rows, vs, dev)
            st.vc, st.vc_meta = al.alloc_state(s.cols, vs, dev)
            if came:
                st.cr, st.cr_meta = al.alloc_state(s.rows, cs, dev)
                st.cc, st.cc_meta = al.alloc_state(s.cols, cs, dev)
        else:
            st.v, st.v_meta = al.alloc_state(s.n, vs, dev)
        if came:
            st.m, st.m_meta = al.alloc_state(s.n, ms, dev)
        states.append(st)
    arr = al.tensor_array(states)
    nbytes = al.came_workspace_bytes(states, cfg, arr=arr) if came else al.adafactor_workspace_bytes(states, cfg,
                                                                                                        arr=arr)
    ws = torch.empty(nbytes, dtype=torch.uint8, device=dev)
    stepf = al.came_step if came else al.adafactor_step
    stream = torch.cuda.current_stream()
    t = 0
    for _ in range(warmup):
        t += 1
        stepf(states, cfg, t, ws, stream=stream, arr=arr)
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    torch.cuda.synchronize()
    for k in range(steps):
        t += 1
        evs[k][0].record(stream)
        stepf(states, cfg, t, ws, stream=stream, arr=arr)
        evs[k][1].record(stream)
    torch.cuda.synchronize()
    ms_ = [a.elapsed_time(b) for a, b in evs]
    mean = sum(ms_) / len(ms_)
    n = sum(s.n for s in shapes)
    alg, sched = factored_bytes_per_param(shapes, came)
    rec = {"workload": ("llama-7b list (291 tensors), " if llama7b else "tinyllama-1.1b list (201 tensors), ") +
                       ("CAME: AL16 B128 V and confidence, UF8 m B256, 2% zero grads" if came else
                        "Adafactor: AL8 B256 factored V and 1-D v"),
           "params": n, "ms_mean": round(mean, 4), "ms_min": round(min(ms_), 4),
           "gparams_s": round(n / (mean * 1e-3) / 1e9, 2),
           "algorithmic_bytes_per_param": round(alg, 4), "schedule_bytes_per_param": round(sched, 4),
           "algorithmic_gbs": round(alg * n / (mean * 1e-3) / 1e9, 1),
           "frac_of_peak": round(alg * n / (mean * 1e-3) / 1e9 / PEAK_GBS, 4),
           "workspace_bytes": nbytes}
    del states, ws
    torch.cuda.empty_cache()
    return rec


def time_apollo(steps: int, warmup: int):
    """One APOLLO step (rank 256, channel-wise scales, limiter 1.01; UF8 m B256 + AL8 v B2048) over the
    TinyLlama-1.1B list: the 154 layer matrices projected, the embedding, LM head and norms under AdamW with
    the same codes; bf16 grads N(0, 1e-3) with 2% zeros, generated once. The projection is the dense
    contraction of the step: 2 * rank flops per projected parameter, binary64 on the matrix cores."""
    import torch

    import paper_2608_22322_amd as al
    from paper_2608_22322_amd import apollo, data
    from paper_2608_22322_amd.workloads import tinyllama_shapes, workload_tinyllama

    shapes = tinyllama_shapes()
    w = workload_tinyllama(zero_frac=0.02)
    dev = torch.device("cuda:0")
    states = []
    for i, s in enumerate(shapes):
        st = al.ParamState(data.device_param(i, s, dev), data.device_grad_buffer(s, w, dev), s.rows, s.cols)
        data.fill_grad(st.grad, i, s, w, 1)
        states.append(st)
    cfg = al.apollo_cfg(rank=apollo.RANK, gamma=apollo.GAMMA)
    drv = apollo.ApolloStep(states, [s.name for s in shapes], cfg, device=dev)
    stream = torch.cuda.current_stream()
    t = 0
    for _ in range(warmup):
        t += 1
        drv.step(t, stream)
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    torch.cuda.synchronize()
    for k in range(steps):
        t += 1
        evs[k][0].record(stream)
        drv.step(t, stream)
        evs[k][1].record(stream)
    torch.cuda.synchronize()
    ms_ = [a.elapsed_time(b) for a, b in evs]
    mean = sum(ms_) / len(ms_)
    n = sum(s.n for s in shapes)
    nproj = sum(s.n for s in shapes if apollo.projected(s.name, s.rows, s.cols))
    flops = 2.0 * apollo.RANK * nproj
    rec = {"workload": "tinyllama-1.1b list (201 tensors), APOLLO rank 256: 154 layer matrices projected "
                       "(UF8 m B256 + AL8 v B2048 on the projected moments), embedding/head/norms AdamW "
                       "with the same codes, 2% zero grads",
           "params": n, "projected_params": nproj, "ms_mean": round(mean, 4), "ms_min": round(min(ms_), 4),
           "gparams_s": round(n / (mean * 1e-3) / 1e9, 2), "projection_gflop": round(flops / 1e9, 1),
           "projection_fp64_tflops_lower_bound": round(flops / (mean * 1e-3) / 1e12, 2),
           "fp64_mfma_peak_tflops": 78.6,
           "state_mib": round(apollo.state_bytes(shapes, apollo.RANK, al.Spec(al.UF8, 256),
                                                 al.Spec(al.AL8, 2048)) / 2**20, 1),
           "workspace_bytes": int(drv.ws.numel())}
    del states, drv
    torch.cuda.empty_cache()
    return rec


def _cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(shapes, block_v):
    """The oracle, untuned, on a bounded sample of the 7B list, one thread per tensor (parallel over tensors
    only, as the oracle's steps are per tensor): AdamW on layer 0's seven weight matrices (2 steps, AL8 B_V
    block_v + UF8), Adafactor on layer 0's q/k/v/o (1 step, AL8 B256 factors) and CAME on layer 0's q and k
    (1 step, AL16 B128 factors and confidence, UF8 m). Inputs for this timing-only leg are drawn with numpy's
    generator (params N(0, 0.02), bf16 grads N(0, 1e-3) with 1% zeros); bit-reproducible inputs are only
    needed for parity. Wall-clock throughput of each leg; ``value`` is the AdamW leg (the headline path)."""
    from concurrent.futures import ThreadPoolExecutor

    import numpy as np

    import oracle
    from paper_2608_22322_amd import synth

    host_cores = len(os.sched_getaffinity(0))
    rng = np.random.default_rng(921)
    fl32 = lambda x: float(np.float32(x))
    layer0 = {s.name.split(".", 1)[1]: s for s in shapes if s.name.startswith("layer0.") and s.is_2d}

    # one pool of draws, sliced per tensor (gradients are only read; each tensor gets its own params)
    pool_n = max(s.n for s in layer0.values())
    p_pool = rng.standard_normal(pool_n, dtype=np.float32) * np.float32(0.02)
    g_pool = rng.standard_normal(pool_n, dtype=np.float32) * np.float32(1e-3)
    g_pool[rng.random(pool_n, dtype=np.float32) < 0.01] = 0.0
    g_pool = synth.to_bf16_bits(g_pool)

    def inputs(s):
        return p_pool[: s.n].copy(), g_pool[: s.n]

    def touched(st):
        for a in (st.codes, st.meta, st.y):  # fault the pages in outside the timed region
            a.fill(0)
        return st

    def adamw(s):
        m = touched(oracle.State(oracle.UF8, s.n, 256))
        v = touched(oracle.State(oracle.AL8, s.n, block_v, fl32(2 * math.log2(1e-8))))

        def run(p, g):
            for t in (1, 2):
                oracle.adamw_step(p, g, m, v, t)
            return 2 * s.n
        return run

    def adafactor(s):
        f = fl32(math.log2(1e-30))
        vr, vc = touched(oracle.State(oracle.AL8, s.rows, 256, f)), touched(oracle.State(oracle.AL8, s.cols, 256, f))

        def run(p, g):
            oracle.adafactor_step(p, g, s.rows, s.cols, vr, vc, None, 1)
            return s.n
        return run

    def came(s):
        f1, f2 = fl32(math.log2(1e-30)), fl32(math.log2(1e-16))
        st = lambda n, f: touched(oracle.State(oracle.AL16, n, 128, f))
        m = touched(oracle.State(oracle.UF8, s.n, 256))
        vr, vc, cr, cc = st(s.rows, f1), st(s.cols, f1), st(s.rows, f2), st(s.cols, f2)

        def run(p, g):
            oracle.came_step(p, g, s.rows, s.cols, m, vr, vc, None, cr, cc, 1)
            return s.n
        return run

    legs = {}
    for name, make, names, what in (
            ("adamw", adamw, ("q", "k", "v", "o", "gate", "up", "down"),
             f"layer-0 weight matrices, 2 AdamW steps, AL8 B_V {block_v} + UF8"),
            ("adafactor", adafactor, ("q", "k", "v", "o"), "layer-0 q/k/v/o, 1 Adafactor step, AL8 B256 factors"),
            ("came", came, ("q", "k"), "layer-0 q/k, 1 CAME step, AL16 B128 factors + confidence, UF8 m")):
        sel = [layer0[k] for k in names]
        jobs = [(make(s), *inputs(s)) for s in sel]  # states and inputs built (and touched) before timing
        threads = min(host_cores, len(sel))
        t0 = time.perf_counter()
        with ThreadPoolExecutor(threads) as ex:
            n_done = sum(ex.map(lambda j: j[0](j[1], j[2]), jobs))
        secs = time.perf_counter() - t0
        legs[name] = {"value": n_done / secs / 1e9, "unit": "Gparams/s", "threads": threads,
                      "sample": f"{what} ({sum(s.n for s in sel):,} params)", "wall_s": round(secs, 2)}
        log(f"cpu oracle {name}: " + json.dumps(legs[name]))
        del jobs
    a = legs["adamw"]
    return {"value": a["value"], "unit": "Gparams/s", "cores": a["threads"], "kind": "oracle",
            "sample": f"Llama-7B {a['sample']}, binary64 C oracle, one thread per tensor; {a['wall_s']} s wall",
            "host_cores": host_cores, "cpu_model": _cpu_model(), "paths": legs}


PATHS = ("adafactor", "came", "adafactor_7b", "came_7b", "apollo")


def time_path(name: str, steps: int, warmup: int):
    """The other optimizer paths: Adafactor and CAME on the TinyLlama and Llama-7B lists, APOLLO on TinyLlama."""
    if name == "apollo":
        return time_apollo(steps, warmup)
    return time_factored(name.startswith("came"), steps, warmup, llama7b=name.endswith("_7b"))


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--block", type=int, default=2048, help="headline B_V (2048: the paper's AdamW configuration)")
    ap.add_argument("--sweep", default="64,128,256,512,1024,2048", help="B_V values to time ('' for headline only)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-paths", action="store_true", help="skip the Adafactor / CAME timings")
    ap.add_argument("--only-path", choices=PATHS, default=None,
                    help="time one of the other paths alone and print its record (for profiling; no headline)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU (asked for --gpus {args.gpus}): the optimizer step needs no collective; "
              f"on several GPUs each would step its own shard of the tensor list with no exchange inside the step.",
              file=sys.stderr)
        sys.exit(2)
    if args.only_path:
        print(json.dumps({"path": args.only_path, **time_path(args.only_path, args.steps, args.warmup)}), flush=True)
        return

    import torch

    import paper_2608_22322_amd as al
    from paper_2608_22322_amd.workloads import llama7b_shapes, total_params

    al.lib()
    dev = torch.device("cuda:0")
    shapes = llama7b_shapes()
    n = total_params(shapes)
    blocks = [int(b) for b in args.sweep.split(",") if b] if args.sweep else []
    if args.block not in blocks:
        blocks.append(args.block)
    blocks = [b for b in blocks if b != args.block] + [args.block]  # headline last
    log(f"building Llama-7B list: {len(shapes)} tensors, {n:,} params")
    states = build_states(shapes, dev, min(blocks))  # smallest block: largest metadata
    # al_adamw_step runs the whole list in one launch of the step kernel (include/al.h: several only beyond
    # 2^32 chunks of at least 1024 elements)
    assert n < 2**32 * 1024
    launches = 1
    sweep = []
    head = None
    for b in blocks:
        ms, wall = time_adamw(states, b, args.steps, args.warmup)
        mean = sum(ms) / len(ms)
        bpp = adamw_bytes_per_param(b)
        gbs = bpp * n / (mean * 1e-3) / 1e9
        rec = {"block_v": b, "ms_mean": round(mean, 4), "ms_min": round(min(ms), 4),
               "ms_median": round(sorted(ms)[len(ms) // 2], 4), "gparams_s": round(n / (mean * 1e-3) / 1e9, 2),
               "bytes_per_param": bpp, "gbs": round(gbs, 1), "frac_of_peak": round(gbs / PEAK_GBS, 4),
               "wall_s": round(wall, 3)}
        log(json.dumps(rec))
        sweep.append(rec)
        if b == args.block:
            head = (rec, ms, wall, bpp)
    rec, ms, wall, bpp = head
    del states
    torch.cuda.empty_cache()
    ceil = copy_ceiling(n // 4)
    log("copy ceiling: " + json.dumps(ceil))
    mean = rec["ms_mean"]
    traffic = measured_traffic(args.block)
    out = {
        "metric": METRIC,
        "value": rec["gparams_s"],
        "unit": "Gparams/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": mean,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f64 state / f32 param / u8 codes",
        "data": "synthetic (seeded counter-based generator; no dataset)",
        "config": {"workload": "llama-7b list, AdamW, AL8 v (B_V %d) + UF8 m (B 256), bf16 grads N(0,1e-3) "
                               "1%% zeros, fp32 params" % args.block,
                   "params": n, "tensors": len(shapes), "block_v": args.block, "block_m": 256,
                   "grad_dtype": "bf16", "parallelism": "none (1 GPU)"},
        # achieved = algorithmic bytes per launch / average launch duration (= per step / per step)
        "roofline": {"bound": "hbm", "achieved": round(bpp * n / (mean * 1e-3) / 1e9, 1), "peak": PEAK_GBS,
                     "unit": "GB/s", "frac": round(bpp * n / (mean * 1e-3) / 1e9 / PEAK_GBS, 4),
                     "traffic": traffic, "bytes_per_param": bpp, "launches_per_step": launches,
                     "avg_launch_ms": round(mean / launches, 4),
                     "algorithmic_bytes_per_launch": round(bpp * n / launches),
                     "kernel": "adamw_kernel<bf16, UF8, AL8, %d>" % args.block,
                     # best streaming rate measured for the step's byte mix (any access shape), and the rate of
                     # the step's own access shape without the arithmetic
                     "copy_ceiling_gbs": max(ceil["step_shape"], ceil["step_shape_nt"], ceil["wide"]),
                     "same_shape_stream_gbs": max(ceil["step_shape"], ceil["step_shape_nt"]),
                     "frac_of_copy_ceiling": round(bpp * n / (mean * 1e-3) / 1e9 / max(
                         ceil["step_shape"], ceil["step_shape_nt"], ceil["wide"]), 4)},
        "sweep": sweep,
    }
    if not args.no_paths:
        paths = {}
        for name in PATHS:
            paths[name] = time_path(name, args.steps, args.warmup)
            log(name + ": " + json.dumps(paths[name]))
        out["paths"] = paths
    if not args.no_cpu_baseline:
        log("timing the CPU oracle on a bounded sample ...")
        out["cpu_baseline"] = cpu_baseline(shapes, args.block)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
