"""Benchmark of the GNMR controller pass on one MI355X.

One step = one gnmr_step: the gradient pass over every unit (K1), the
Alg. 1 state update and risk (K2) and the Top_maxO selection with locks (K3),
over gradients already resident in HBM.  The default workload is the
LLaMA-2-13B-shaped bf16 gradient set (280 units, 25.38 GB per step).

Prints one JSON line: whole-step GB/s (algorithmic bytes = every gradient
byte once), ms and us per step, the dominant kernel's roofline position, and
the CPU oracle timed on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
# the sources of the gradient-pass kernel whose HBM counters profiles/ records
K1_SOURCES = ("k1_sumsq.hip", "k1_geometry.h")
METRIC = "GNMR step GB/s (frac. of HBM peak) + µs/step, 13B-shaped grads, 1 GPU"
# below this many gradient bytes per step the step is launch-bound, and the
# per-kernel events stay out of the timed steps
EVENT_FREE_BYTES = 1 << 30
# the controller's budget policies (gnmr_config.budget_mode)
BUDGET_MODES = {"active": 0, "admitted": 1, "static": 2}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


# Worker threads of the all-cores leg: the CPU share that a one-GPU job has on
# the GPU hosts this runs on is 16 threads, whatever the host's core count.
CPU_SHARE_THREADS = 16


def host_facts() -> dict:
    """The host the CPU oracle ran on: logical CPUs, the affinity mask, the CPU
    model and the BLAS thread pools NumPy would use."""
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    blas = None
    try:
        import numpy  # noqa: F401  (loads the BLAS whose pools are listed)
        from threadpoolctl import threadpool_info
        blas = [{"api": i.get("internal_api"), "threads": i.get("num_threads")}
                for i in threadpool_info()]
    except Exception:                                  # pragma: no cover
        pass
    return {"os_cpu_count": os.cpu_count(), "affinity_cpus": len(os.sched_getaffinity(0)),
            "cpu_model": model, "blas_pools_default": blas}


def cpu_baseline(torch, buf, lay, w, target_s: float = 12.0, max_units: int = 100000):
    """Oracle norm pass plus one oracle controller step, single-threaded, on a
    bounded sample of units copied off the device (copy not timed)."""
    import numpy as np

    from oracle import Controller as Oracle
    from oracle import sumsq

    try:
        from threadpoolctl import threadpool_limits
        limiter = threadpool_limits(limits=1)
    except Exception:                                  # pragma: no cover
        limiter = None
    order = np.random.default_rng(0).permutation(w.num_units)
    spent, nbytes, units = 0.0, 0, 0
    for b in order[:max_units]:
        s = int(lay.seg_byte_off[b])
        n = int(lay.seg_numel[b])
        esz = 2 if int(lay.seg_dtype[b]) == 1 else 4
        host = buf[s:s + n * esz].cpu().numpy()
        vals = host.view(np.uint16) if esz == 2 else host.view(np.float32)
        t0 = time.perf_counter()
        sumsq([(vals, int(lay.seg_dtype[b]))])
        spent += time.perf_counter() - t0
        nbytes += n * esz
        units += 1
        if spent >= target_s:
            break
    ora = Oracle(w.num_units, window=w.window, max_o=w.max_o, lock_len=w.lock_len, eps=w.eps)
    norms = np.ones(w.num_units)
    t0 = time.perf_counter()
    ora.step(norms, w.alpha(1), w.beta(1))
    logic_s = time.perf_counter() - t0
    if limiter is not None:
        limiter.unregister()
    gbs = nbytes / spent / 1e9
    step_s = w.bytes_per_step / (nbytes / spent) + logic_s
    return {"value": round(gbs, 4), "unit": "GB/s", "cores": 1, "kind": "oracle",
            "us_per_step": round(step_s * 1e6, 1), "host": host_facts(),
            "blas_threads_used": 1,
            "sample": f"float64 NumPy oracle norm pass over {units} of {w.num_units} units "
                      f"({nbytes / 1e9:.2f} GB, {spent:.1f} s) plus one oracle controller step "
                      f"over all units; us_per_step extrapolated to the full "
                      f"{w.bytes_per_step / 1e9:.2f} GB step"}


def cpu_baseline_all_cores(buf, lay, w, single_gbs: float, target_s: float = 10.0,
                           stage_bytes: float = 3e9):
    """The same oracle norm pass spread over the host's cores, one thread per
    core, each single-threaded inside NumPy (the oracle's float64 dot product
    releases the GIL).  A fixed set of units, about stage_bytes in all, is
    copied off the device once and swept repeatedly (copies not timed)."""
    from concurrent.futures import ThreadPoolExecutor

    import numpy as np

    from oracle import sumsq

    try:
        from threadpoolctl import threadpool_limits
        limiter = threadpool_limits(limits=1)
    except Exception:                                  # pragma: no cover
        limiter = None
    cores = max(1, min(CPU_SHARE_THREADS, len(os.sched_getaffinity(0))))
    order = np.random.default_rng(1).permutation(w.num_units)
    staged, nbytes = [], 0
    for b in order:
        s = int(lay.seg_byte_off[b])
        n = int(lay.seg_numel[b])
        esz = 2 if int(lay.seg_dtype[b]) == 1 else 4
        host = buf[s:s + n * esz].cpu().numpy()
        staged.append(((host.view(np.uint16) if esz == 2 else host.view(np.float32)),
                       int(lay.seg_dtype[b])))
        nbytes += n * esz
        if nbytes >= stage_bytes:
            break
    with ThreadPoolExecutor(max_workers=cores) as pool:
        # one untimed pilot sweep sizes the run: on small units the per-call
        # overhead, not the bytes, sets the time
        t0 = time.perf_counter()
        list(pool.map(lambda seg: sumsq([seg]), staged))
        pilot = time.perf_counter() - t0
        sweeps = max(1, min(int(round(single_gbs * 1e9 * cores * target_s / nbytes)),
                            int(target_s / max(pilot, 1e-6))))
        tasks = staged * sweeps
        t0 = time.perf_counter()
        list(pool.map(lambda seg: sumsq([seg]), tasks))
        spent = time.perf_counter() - t0
    if limiter is not None:
        limiter.unregister()
    total = nbytes * sweeps
    return {"value": round(total / spent / 1e9, 4), "unit": "GB/s", "cores": cores,
            "kind": "oracle", "host": host_facts(), "blas_threads_used": 1,
            "threads_rule": f"min(affinity CPUs, {CPU_SHARE_THREADS}): a one-GPU job's CPU "
                            "share on these hosts",
            "sample": f"float64 NumPy oracle norm pass, {cores} threads over {len(staged)} "
                      f"units ({nbytes / 1e9:.2f} GB) swept {sweeps} times "
                      f"({total / 1e9:.1f} GB, {spent:.1f} s)"}


def event_time(torch, fn, reps: int, stream=None, lead_in: int = 1) -> float:
    """Average ms of fn() over `reps` calls between two events on `stream`.
    `lead_in` untimed calls are queued right before the first event, with no
    synchronisation in between, so that the device is busy when the event is
    reached and a host delay before the first timed call is not counted."""
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    for _ in range(lead_in):
        fn()
    e0.record(stream)
    for _ in range(reps):
        fn()
    e1.record(stream)
    e1.synchronize()
    return e0.elapsed_time(e1) / reps


def library_reduce_probe(torch, buf, lay, w, reps: int = 5):
    """torch.linalg.vector_norm over the same gradient bytes viewed as one
    flat tensor of the workload's dtype: the library's own read-reduce, as a
    reference point for the gradient pass (a single-dtype workload only)."""
    dts = {int(d) for d in lay.seg_dtype}
    if len(dts) != 1:
        return None
    dt = torch.bfloat16 if dts.pop() == 1 else torch.float32
    x = buf[:w.bytes_per_step].view(dt)
    ms = event_time(torch, lambda: torch.linalg.vector_norm(x), reps, lead_in=2)
    return {"kind": "torch.linalg.vector_norm over the same bytes", "ms": round(ms, 4),
            "GBs": round(w.bytes_per_step / (ms * 1e-3) / 1e9, 1)}


def read_ceiling_probe(torch, buf, w, stream, reps: int = 5):
    """Plain read-reduce kernels over the same gradient bytes (grid-stride,
    and one 64 KiB block per workgroup in XCD-contiguous order): the read
    rate a minimal kernel reaches on this buffer in this run."""
    from synth.gpu import ReadProbe

    rp = ReadProbe()
    out = {}
    s = stream.cuda_stream
    for v, name in rp.VARIANTS.items():
        parts = torch.empty(rp.num_partials(w.bytes_per_step, v), dtype=torch.float32,
                            device="cuda")
        ms = event_time(torch, lambda: rp.run(buf.data_ptr(), w.bytes_per_step,
                                              parts.data_ptr(), v, s), reps, stream, lead_in=2)
        out[name] = {"ms": round(ms, 4), "GBs": round(w.bytes_per_step / (ms * 1e-3) / 1e9, 1)}
    return out


def measured_traffic(profile: str, sources, workload: str):
    """A kernel's HBM bytes per launch from its committed rocprofv3 counter
    summary (profiles/<profile>), or None when the summary is for another
    workload or the kernel source has changed since the counters were taken."""
    import hashlib

    path = os.path.join(ROOT, "profiles", profile)
    if not os.path.exists(path):
        return None
    kv = {}
    for line in open(path):
        if "=" in line and not line.startswith(("|", "#", "rocprofv3")):
            k, _, v = line.strip().partition("=")
            kv[k] = v
    src = b"".join(open(os.path.join(ROOT, "paper_2606_00539_amd", "csrc", f), "rb").read()
                   for f in sources)
    if kv.get("kernel_source_sha256_16") != hashlib.sha256(src).hexdigest()[:16]:
        return None
    if kv.get("workload") != workload:
        return None
    return int(kv["fetch_bytes_per_launch"]) + int(kv["write_bytes_per_launch"])


def copy_probe(torch, nbytes: int, steps: int, warmup: int) -> None:
    """Device-to-device copies of nbytes (read nbytes + write nbytes each)."""
    src = torch.empty(nbytes, dtype=torch.uint8, device="cuda").fill_(1)
    dst = torch.empty_like(src)
    for _ in range(warmup):
        dst.copy_(src)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        dst.copy_(src)
    torch.cuda.synchronize()
    dt = (time.perf_counter() - t0) / steps
    print(json.dumps({"probe": "copy", "bytes": nbytes, "ms": round(dt * 1e3, 4),
                      "read_plus_write_GBs": round(2 * nbytes / dt / 1e9, 1)}), flush=True)


def actuator_bench(torch, tokens: int, steps: int, warmup: int) -> None:
    """Saved activations of the 7 projections of each of 32 LLaMA-2-7B layers
    for `tokens` tokens (q, k, v, o, gate, up inputs: 4096 features; down:
    11008), all on the low-cost path (E2M1, in place): every byte is read and
    written once.  Also times the mixed case of 8 units on the BF16 path."""
    import numpy as np

    from paper_2606_00539_amd import GNMR_FMT_BF16, GNMR_FMT_E2M1, Actuator

    cols = [4096] * 6 + [11008]
    U = 32 * 7
    shapes = [(tokens, cols[b % 7]) for b in range(U)]
    total = sum(r * c for r, c in shapes)
    buf = torch.randn(total, dtype=torch.bfloat16, device="cuda")
    segs, off = [], 0
    for b, (r, c) in enumerate(shapes):
        p = buf.data_ptr() + 2 * off
        segs.append((p, p, r, c, b))
        off += r * c
    act = Actuator(segs, U)
    nbytes = act.info()["bytes"]
    results = {}
    for label, nrec in (("all_low_cost", 0), ("maxO8_bf16_in_place", 8)):
        mask = np.zeros(U, np.uint8)
        mask[np.random.default_rng(0).choice(U, nrec, replace=False)] = 1
        d_mask = torch.from_numpy(mask).to("cuda")
        ms = event_time(torch, lambda: act.apply(d_mask, GNMR_FMT_E2M1, GNMR_FMT_BF16), steps,
                        lead_in=max(warmup, 1))
        moved = 2 * sum(r * c * 2 for (r, c), m in zip(shapes, mask) if not m)
        results[label] = {"ms": round(ms, 4), "bytes_moved": moved,
                          "GBs": round(moved / (ms * 1e-3) / 1e9, 1)}
    a = results["all_low_cost"]
    # the read-and-write reference on the same bytes: a plain non-temporal copy
    from synth.gpu import ReadProbe

    rp = ReadProbe()
    dst = torch.empty_like(buf)
    nb = buf.numel() * 2 // 16 * 16
    copy_ms = event_time(torch, lambda: rp.copy(buf.data_ptr(), dst.data_ptr(), nb), 5,
                         lead_in=2)
    copy_gbs = 2 * nb / (copy_ms * 1e-3) / 1e9
    del dst
    print(json.dumps({
        "metric": "recovery actuator GB/s (bf16 read + write, per-token E2M1 fake quantisation)",
        "value": a["GBs"], "unit": "GB/s", "n_gpus": 1, "steps": steps, "warmup": warmup,
        "ms_per_step": a["ms"], "higher_is_better": True, "dtype": "f32", "data": "synthetic",
        "config": {"workload": f"LLaMA-2-7B-shaped saved activations, 224 units, {tokens} "
                               f"tokens, {nbytes / 1e9:.2f} GB bf16", "units": U,
                   "tokens": tokens, "activation_bytes": nbytes},
        "roofline": {"bound": "hbm", "achieved": a["GBs"], "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(a["GBs"] / HBM_PEAK_GBS, 4), "kernel": "k4_actuate",
                     "algorithmic_bytes": a["bytes_moved"],
                     "frac_of_copy_probe": round(a["GBs"] / copy_gbs, 4)},
        "copy_probe": {"kind": "plain non-temporal copy of the same bytes (read + write)",
                       "ms": round(copy_ms, 4), "GBs": round(copy_gbs, 1)},
        "cases": results}), flush=True)
    act.close()


def wgrad_bench(torch, tokens: int, steps: int, warmup: int) -> None:
    """The controller step with its gradient pass fused into the producer:
    the seven weight-gradient GEMMs of one LLaMA-2-13B layer (K5, the sum of
    squares in the epilogue) followed by K2 + K3 from the tile partials,
    against the unfused step: the same GEMMs by the vendor library
    (torch.mm -> hipBLASLt) followed by gnmr_step (K1 re-reads every
    gradient, then K2 + K3)."""
    import numpy as np

    from paper_2606_00539_amd import (Controller, gnmr_wgrad_num_tiles, gnmr_wgrad_sumsq,
                                      gnmr_wgrad_sumsq_batched)
    from synth import wgrad as SW

    L = SW.llama2_13b_layer(tokens)
    U = L.num_units
    t0 = time.perf_counter()
    dys, xs = [], []
    for b, (o, i) in enumerate(L.shapes):
        dy, x = SW.operands(L.seed, 1, b, tokens, o, i, dy_scale=L.dy_scale(1, b))
        dys.append(torch.from_numpy(dy.view(np.int16)).to("cuda").view(torch.bfloat16))
        xs.append(torch.from_numpy(x.view(np.int16)).to("cuda").view(torch.bfloat16))
    log(f"[bench] wgrad operands generated in {time.perf_counter() - t0:.1f} s")
    numel = [o * i for o, i in L.shapes]
    off = np.concatenate([[0], np.cumsum(numel)]).astype(np.int64)
    grads = torch.empty(int(off[-1]), dtype=torch.bfloat16, device="cuda")
    dws = [grads[int(off[b]):int(off[b + 1])].view(o, i) for b, (o, i) in enumerate(L.shapes)]
    tiles = [gnmr_wgrad_num_tiles(o, i) for o, i in L.shapes]
    poff = np.concatenate([[0], np.cumsum(tiles)]).astype(np.int64)
    parts = torch.empty(int(poff[-1]), dtype=torch.float32, device="cuda")
    psl = [parts[int(poff[b]):int(poff[b + 1])] for b in range(U)]
    ptrs = [d.data_ptr() for d in dws]
    stream = torch.cuda.current_stream()
    mk = lambda: Controller(U, 5, 2, 4, 1e-12, np.arange(U + 1), numel, [1] * U, ptrs,
                            stream=stream)
    fused, unfused = mk(), mk()
    fused.bind_partials(poff)

    problems = [(dys[b], xs[b], dws[b], tokens, o, i) for b, (o, i) in enumerate(L.shapes)]

    def fused_step(t):
        gnmr_wgrad_sumsq_batched(problems, parts, stream)
        fused.step_from_partials(parts, 1.5 if t == 1 else 1.1, 1.5, stream)

    def unfused_step(t):
        for b in range(U):
            torch.mm(dys[b].t(), xs[b], out=dws[b])
        unfused.step(1.5 if t == 1 else 1.1, 1.5, stream=stream)

    def gemms_only(kind):
        for b, (o, i) in enumerate(L.shapes):
            if kind == "k5":
                gnmr_wgrad_sumsq_batched(problems, parts, stream)
                break
            else:
                torch.mm(dys[b].t(), xs[b], out=dws[b])

    def timed(fn, n):
        calls = iter(range(1, n + 2))
        return event_time(torch, lambda: fn(next(calls)), n, stream)

    for k in range(warmup):
        fused_step(k + 1)
        unfused_step(k + 1)
    torch.cuda.synchronize()
    ms_fused = timed(fused_step, steps)
    ms_unfused = timed(unfused_step, steps)
    ms_k5 = timed(lambda _: gemms_only("k5"), steps)
    ms_blas = timed(lambda _: gemms_only("blas"), steps)
    # gradient accumulation over micro-batches: dw += dy^T x (K5's accumulate
    # flag; the library's beta = 1 product); the stored gradient is read too
    acc_problems = [p + (1,) for p in problems]
    ms_k5_acc = timed(lambda _: gnmr_wgrad_sumsq_batched(acc_problems, parts, stream), steps)

    def blas_acc(_):
        for b in range(U):
            dws[b].addmm_(dys[b].t(), xs[b])
    ms_blas_acc = timed(blas_acc, steps)
    # per-shape K5 and library GEMM times (the dominant kernel's roofline)
    per_shape = {}
    for b, (o, i) in enumerate(L.shapes[:1] + L.shapes[4:5] + L.shapes[6:7]):
        bb = L.shapes.index((o, i))
        f = 2.0 * tokens * o * i
        k5 = timed(lambda _: gnmr_wgrad_sumsq(dys[bb], xs[bb], dws[bb], tokens, o, i, psl[bb],
                                              stream), steps)
        bl = timed(lambda _: torch.mm(dys[bb].t(), xs[bb], out=dws[bb]), steps)
        per_shape[f"{o}x{i}"] = {"k5_ms": round(k5, 4), "k5_tflops": round(f / k5 / 1e9, 1),
                                 "hipblaslt_ms": round(bl, 4),
                                 "hipblaslt_tflops": round(f / bl / 1e9, 1)}
    out = fused.query(stream=stream)
    log(f"[bench] fused step stats {out['stats']}")
    tflops = L.flops / (ms_k5 * 1e-3) / 1e12
    print(json.dumps({
        "metric": "GNMR step fused into the weight-gradient GEMMs, LLaMA-2-13B layer "
                  "(GEMMs + controller step, TFLOP/s)",
        "value": round(L.flops / (ms_fused * 1e-3) / 1e12, 1), "unit": "TFLOP/s", "n_gpus": 1,
        "steps": steps, "warmup": warmup, "ms_per_step": round(ms_fused, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"LLaMA-2-13B decoder layer weight gradients, 7 units, "
                               f"{tokens} tokens, bf16", "units": U, "tokens": tokens,
                   "flops_per_step": L.flops, "grad_bytes": L.grad_bytes},
        "roofline": {"bound": "mfma", "achieved": round(tflops, 1), "peak": 2500.0,
                     "unit": "TFLOP/s", "frac": round(tflops / 2500.0, 4),
                     "traffic": measured_traffic("k5_wgrad_llama2-13b_layer.md", ("k5_wgrad.hip",),
                                                 L.name),
                     "traffic_unit": "bytes per launch (FETCH_SIZE + WRITE_SIZE, copy-calibrated)",
                     "algorithmic_bytes": L.operand_bytes + L.grad_bytes,
                     "kernel": "k5_wgrad", "kernel_ms_per_step": round(ms_k5, 4)},
        "unfused": {"ms_per_step": round(ms_unfused, 4),
                    "hipblaslt_gemms_ms": round(ms_blas, 4),
                    "gnmr_step_ms": round(ms_unfused - ms_blas, 4)},
        "fused_saving_ms": round(ms_unfused - ms_fused, 4),
        "accumulate": {"k5_ms": round(ms_k5_acc, 4),
                       "k5_tflops": round(L.flops / (ms_k5_acc * 1e-3) / 1e12, 1),
                       "hipblaslt_ms": round(ms_blas_acc, 4),
                       "hipblaslt_tflops": round(L.flops / (ms_blas_acc * 1e-3) / 1e12, 1)},
        "per_shape": per_shape}), flush=True)
    fused.close()
    unfused.close()


def qsim_bench(torch, tokens: int, steps: int, warmup: int) -> None:
    """The actuator inside a training step, on the seven projections of one
    LLaMA-2-13B layer at `tokens` tokens: forward and backward of bf16
    bias-free linear layers (a) as plain layers, (b) with their saved inputs
    quantised per token (QuantizedSavedInputs, E2M1), (c) as the
    quantisation-simulated operator (QuantSimLinears: x, w, y, dy, dx and dw
    quantised, E2M1).  Every unit is on the low-cost path (mask 0), the
    formats' most quantising case."""
    import numpy as np

    from paper_2606_00539_amd import GNMR_FMT_BF16, GNMR_FMT_E2M1
    from paper_2606_00539_amd.torch_units import (QuantizedSavedInputs, QuantSimLinears,
                                                  TorchUnits)

    d, ffn = 5120, 13824
    shapes = {"q_proj": (d, d), "k_proj": (d, d), "v_proj": (d, d), "o_proj": (d, d),
              "gate_proj": (ffn, d), "up_proj": (ffn, d), "down_proj": (d, ffn)}
    torch.manual_seed(0)
    layers = torch.nn.ModuleDict({n: torch.nn.Linear(i, o, bias=False)
                                  for n, (o, i) in shapes.items()}).to("cuda", torch.bfloat16)
    xs = {n: torch.randn(tokens, i, device="cuda").to(torch.bfloat16).requires_grad_(True)
          for n, (o, i) in shapes.items()}
    dys = {n: torch.randn(tokens, o, device="cuda").to(torch.bfloat16) * 1e-3
           for n, (o, i) in shapes.items()}
    flops = sum(3 * 2.0 * tokens * o * i for o, i in shapes.values())

    def layer_step(_):
        for n in shapes:
            y = layers[n](xs[n])
            y.backward(dys[n])
        layers.zero_grad(set_to_none=True)
        for x in xs.values():
            x.grad = None

    def timed():
        for k in range(warmup):
            layer_step(k)
        torch.cuda.synchronize()
        return event_time(torch, lambda: layer_step(0), steps)

    units = TorchUnits(layers.named_parameters(), max_o=1, lock_len=1,
                       unit_of=lambda n: n.split(".")[0])
    results = {"plain_bf16": timed()}
    saved = QuantizedSavedInputs(units, list(layers.named_children()), GNMR_FMT_E2M1,
                                 GNMR_FMT_BF16)
    results["saved_activations_e2m1"] = timed()
    saved.close()
    op = QuantSimLinears(units, list(layers.named_children()), low=(GNMR_FMT_E2M1,) * 2,
                         recovery=(3, 4))
    results["qsim_operator_e2m1"] = timed()
    op.close()
    units.close()
    base = results["plain_bf16"]
    # bytes K4 moves per layer step: the operator quantises x, w, y, dy, dx and dw
    # (read + write, bf16); the saved-activation path quantises x only
    act_bytes = {"saved_activations_e2m1": sum(2 * 2 * tokens * i for o, i in shapes.values()),
                 "qsim_operator_e2m1": sum(2 * 2 * (tokens * i + o * i + tokens * o) * 2
                                           for o, i in shapes.values())}
    print(json.dumps({
        "metric": "actuator inside a training step: one LLaMA-2-13B layer's seven projections, "
                  "forward + backward, ms (lower is better)",
        "value": round(results["qsim_operator_e2m1"], 4), "unit": "ms", "n_gpus": 1,
        "steps": steps, "warmup": warmup, "ms_per_step": round(results["qsim_operator_e2m1"], 4),
        "higher_is_better": False, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"LLaMA-2-13B decoder layer projections (q, k, v, o 5120x5120; "
                               f"gate, up 13824x5120; down 5120x13824), {tokens} tokens, bf16, "
                               "every unit on the E2M1 low-cost path", "tokens": tokens,
                   "gemm_flops_per_step": flops},
        "cases_ms": {k: round(v, 4) for k, v in results.items()},
        "overhead_vs_plain": {k: round(v / base - 1, 4) for k, v in results.items()
                              if k != "plain_bf16"},
        "k4_bytes_per_step": act_bytes,
        "plain_tflops": round(flops / (base * 1e-3) / 1e12, 1)}), flush=True)


def stream_steps(torch, np, w, lay, buf, ptrs, stream):
    """Every step of the workload's stream on a fresh controller, each timed
    by a pair of events right after its gradients were generated (the
    generation is not timed): the per-step spread of the whole stream."""
    from paper_2606_00539_amd import Controller
    from synth.gpu import Generator

    gen = Generator()
    us = []
    with Controller(w.num_units, w.window, w.max_o, w.lock_len, w.eps, lay.unit_seg_off,
                    lay.seg_numel, lay.seg_dtype, ptrs, stream=stream) as ctl:
        for t in range(1, w.steps + 1):
            gen.fill(lay, buf.data_ptr(), w.seed, t, w.scale32(t), stream=stream.cuda_stream)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            ctl.step(w.alpha(t), w.beta(t), stream=stream)
            e1.record(stream)
            e1.synchronize()
            us.append(e0.elapsed_time(e1) * 1e3)
    us = np.array(us)
    out = {q: round(float(np.percentile(us, p)), 1)
           for q, p in (("p10", 10), ("p50", 50), ("p90", 90))}
    out["steps"] = int(w.steps)
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="llama2-13b")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--graph", action="store_true",
                    help="time replays of one captured step (HIP graph) instead of eager steps; "
                         "kernel times still come from the eager steps timed before them")
    ap.add_argument("--actuator", action="store_true",
                    help="measure the recovery actuator (per-token fake quantisation of "
                         "LLaMA-2-7B-shaped saved activations) instead of the controller")
    ap.add_argument("--wgrad", action="store_true",
                    help="measure the gradient pass fused into the weight-gradient GEMMs of "
                         "one LLaMA-2-13B layer against library GEMMs + gnmr_step")
    ap.add_argument("--qsim", action="store_true",
                    help="measure the actuator inside a training step (saved activations, the "
                         "quantisation-simulated operator) against plain bf16 layers")
    ap.add_argument("--budget-mode", choices=sorted(BUDGET_MODES), default="active",
                    help="controller policy: the active-set cap (default), the admitted-only "
                         "budget, or the static baseline (ranked once after the warm-up)")
    ap.add_argument("--policy-warmup", type=int, default=None,
                    help="high-fidelity warm-up steps of the policy (default: 0; 3 for static)")
    ap.add_argument("--tokens", type=int, default=4096)
    ap.add_argument("--probe-copy-bytes", type=float, default=0,
                    help="instead of the controller, time device-to-device copies of this "
                         "many bytes (the known-size reference for HBM byte counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(the controller pass runs on a single MI355X)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2606_00539_amd import Controller
    from synth import layout as L
    from synth import recipe as R
    from synth.gpu import Generator

    assert torch.cuda.is_available(), "bench.py needs a HIP device"
    torch.cuda.set_device(0)
    if args.probe_copy_bytes:
        copy_probe(torch, int(args.probe_copy_bytes), args.steps, args.warmup)
        return
    if args.actuator:
        actuator_bench(torch, args.tokens, args.steps, args.warmup)
        return
    if args.wgrad:
        wgrad_bench(torch, args.tokens, args.steps, args.warmup)
        return
    if args.qsim:
        qsim_bench(torch, args.tokens, args.steps, args.warmup)
        return
    w = R.get(args.workload)
    lay = L.for_workload(w)
    log(f"[bench] {w.name}: {w.num_units} units, {w.bytes_per_step / 1e9:.3f} GB/step")
    buf = torch.empty(lay.total_bytes, dtype=torch.uint8, device="cuda")
    base = buf.data_ptr()
    ptrs = [base + int(o) for o in lay.seg_byte_off]
    Generator().fill(lay, base, w.seed, 1, w.scale32(1))
    stream = torch.cuda.current_stream()
    mode = BUDGET_MODES[args.budget_mode]
    policy_warmup = args.policy_warmup
    if policy_warmup is None:
        policy_warmup = 3 if args.budget_mode == "static" else 0
    ctl = Controller(w.num_units, w.window, w.max_o, w.lock_len, w.eps, lay.unit_seg_off,
                     lay.seg_numel, lay.seg_dtype, ptrs, stream=stream, budget_mode=mode,
                     warmup_steps=policy_warmup)
    info = ctl.info()
    t = 0
    for _ in range(args.warmup):
        t += 1
        ctl.step(w.alpha(t), w.beta(t), stream=stream)
    torch.cuda.synchronize()
    log(f"[bench] warmup {args.warmup} steps done")

    # The timed region: K steps, with the library's HIP events around each
    # kernel on the launch stream, so that the roofline's per-launch
    # durations come from these same steps.  The events cost nothing
    # measurable on a step of milliseconds, but each adds a few microseconds
    # to a launch-bound step: below EVENT_FREE_BYTES per step the timed steps
    # run without them and the kernel times come from a second pass.
    in_region = w.bytes_per_step >= EVENT_FREE_BYTES
    ctl.set_profiling(in_region)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        t += 1
        ctl.step(w.alpha(t), w.beta(t), stream=stream)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    if not in_region:
        ctl.set_profiling(True)
        for _ in range(args.steps):
            t += 1
            ctl.step(w.alpha(t), w.beta(t), stream=stream)
        torch.cuda.synchronize()
    prof = ctl.profile_read()
    ctl.set_profiling(False)
    if args.graph:
        # one step captured with the thresholds now in force, replayed K times
        graph = torch.cuda.CUDAGraph()
        side = torch.cuda.Stream()
        torch.cuda.synchronize()
        with torch.cuda.stream(side):
            with torch.cuda.graph(graph, stream=side):
                ctl.step(w.alpha(t + 1), w.beta(t + 1), stream=side)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(args.steps):
            graph.replay()
        torch.cuda.synchronize()
        elapsed = time.perf_counter() - t0
        log(f"[bench] {args.steps} graph replays in {elapsed:.6f} s")
    out = ctl.query(stream=stream)
    log(f"[bench] timed {args.steps} steps in {elapsed:.4f} s; stats {out['stats']}")
    # the spread of single steps, each between a pair of events (after the timed region)
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(args.steps)]
    for e0, e1 in evs:
        t += 1
        e0.record(stream)
        ctl.step(w.alpha(t), w.beta(t), stream=stream)
        e1.record(stream)
    torch.cuda.synchronize()
    step_us = np.array([e0.elapsed_time(e1) * 1e3 for e0, e1 in evs])
    spread = {q: round(float(np.percentile(step_us, p)), 1)
              for q, p in (("p10", 10), ("p50", 50), ("p90", 90))}
    stream_spread = stream_steps(torch, np, w, lay, buf, ptrs, stream)

    ms = elapsed * 1e3 / args.steps
    gbs = w.bytes_per_step / (elapsed / args.steps) / 1e9
    k1_ms = prof["ms_sumsq"] / max(prof["steps"], 1)
    k1_gbs = w.bytes_per_step / (k1_ms * 1e-3) / 1e9
    traffic = measured_traffic(f"k1_sumsq_{w.name}_bf16_traffic.md", K1_SOURCES, w.name)
    roofline = {"bound": "hbm", "achieved": round(k1_gbs, 1), "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": round(k1_gbs / HBM_PEAK_GBS, 4), "traffic": traffic,
                "traffic_unit": "bytes per launch (FETCH_SIZE + WRITE_SIZE, copy-calibrated)",
                "algorithmic_bytes": w.bytes_per_step,
                "kernel": "k1_sumsq", "kernel_ms": round(k1_ms, 4),
                "update_ms": round(prof["ms_update"] / max(prof["steps"], 1), 4),
                "select_ms": round(prof["ms_select"] / max(prof["steps"], 1), 4)}
    result = {
        "metric": METRIC, "value": round(gbs, 1), "unit": "GB/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 4),
        "us_per_step": round(ms * 1e3, 1), "frac_hbm_peak": round(gbs / HBM_PEAK_GBS, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": f"{w.name} gradients: {w.description}",
                   "units": w.num_units, "grad_dtype": "bf16" if w.dtypes[0] == 1 else "fp32",
                   "bytes_per_step": w.bytes_per_step, "max_o": w.max_o,
                   "lock_len": w.lock_len, "window": w.window,
                   "work_items": info["num_items"], "item_bytes": info["item_bytes"],
                   "launches_per_step": info["launches_per_step"],
                   "budget_mode": args.budget_mode, "policy_warmup_steps": policy_warmup,
                   "timing": ("graph replays; kernel times from eager steps before them"
                              if args.graph else
                              "eager steps; kernel times from HIP events in the same steps"
                              if in_region else
                              "eager steps (launch-bound: no events in them); kernel times "
                              "from a second pass with HIP events"),
                   "timed_loop": "steady loop: the warm-up and timed steps all read one "
                                 "resident buffer holding the stream's step-1 gradients "
                                 "(every byte each step); after its first steps the candidate "
                                 "pool is empty, so K3 does not rank. stream_step_us times every "
                                 "step of the workload's own stream, with its real pools, right "
                                 "after each step's gradients are generated"},
        "roofline": roofline,
        "step_us_spread": spread,
        "stream_step_us": stream_spread,
    }
    if w.bytes_per_step % 16 == 0:
        result["read_ceiling_probe"] = read_ceiling_probe(torch, buf, w, stream)
        best = max(v["GBs"] for v in result["read_ceiling_probe"].values())
        result["roofline"]["frac_of_read_probe"] = round(k1_gbs / best, 4)
    probe = library_reduce_probe(torch, buf, lay, w)
    if probe is not None:
        result["library_reduce_probe"] = probe
    if not args.no_cpu_baseline:
        log("[bench] timing the CPU oracle on a sample")
        result["cpu_baseline"] = cpu_baseline(torch, buf, lay, w)
        log("[bench] timing the CPU oracle on all host cores")
        result["cpu_baseline_all_cores"] = cpu_baseline_all_cores(
            buf, lay, w, result["cpu_baseline"]["value"])
    ctl.close()
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
