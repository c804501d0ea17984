"""Benchmark of the Approx-BP / MS-BP hot path on one MI355X.

A step is one pass of the whole hot path over one batch of the LLaMA-7B-shaped
workload (bf16 storage, fp32 arithmetic), in training order (the backward half
consumes the state saved by the previous step's forward, so all inputs are cold):

    MS-RMSNorm forward   on x    [4*2048, 4096]   -> z, rstd
    ReSiLU2 forward      on gate [4*2048, 11008]  -> SiLU(gate), 2-bit codes
    ReSiLU2 backward     dy, codes                -> d gate
    MS-RMSNorm backward  dz, z, rstd              -> dx

Inputs are seeded synthetic tensors already resident in HBM. The reported value
is the algorithmic HBM traffic of the step (bytes each kernel must read and
write) divided by the measured step time (K steps back to back between two HIP
events on the kernels' stream). Per-kernel launch durations come from a second
event-timed loop that launches each kernel back to back over rotating tensor
sets; the dominant kernel's figure feeds the roofline entry. The line also carries
the cold forward + backward GB/s of the MS-LN and ReGELU2 pairs on the ViT-B
batch-64 bf16 shapes (`pairs_vit_b_bs64_bf16`), and the CPU oracle's rate on the
same step (timed after the GPU legs).

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-cpu-baseline] [--swiglu] [--pairs]
                      [--linear] [--blocks] [--variants] [--workload NAME] [--graph]

--workload runs the same step on another configured workload (ViT-B fp32, ViT-B
batch 64 bf16 x 12 blocks, LLaMA-13B with outliers). --graph replays the timed
steps from one HIP graph instead of launching them from Python (for workloads
whose kernels are shorter than a Python launch); the JSON line names the mode
in "launch".
--linear adds the fused linear-layer + activation forward (TFLOP/s, against the
unfused library GEMM + activation kernel) on the ViT-B and LLaMA-7B MLP shapes.
--pairs adds, for every workload (ViT-B fp32, ViT-B batch 64 bf16 x 12 blocks,
LLaMA-7B and LLaMA-13B shapes), the forward + backward GB/s of the norm pair and
of the activation pair, cold and warm.
--blocks adds a bf16 training step of whole MLP blocks against torch's modules;
--variants the k-bit family kernels (k = 1..4, ReGELU2-d).
"""

import argparse
import gc
import hashlib
import json
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0            # MI355X HBM3E, AMD published peak
WORKLOAD = "llama7b_swiglu_bf16"
METRIC = "fwd+bwd HBM GB/s (% of peak) for ReGELU2/ReSiLU2/MS-LN; saved bytes/elt"
KERNEL_SOURCES = ("paper_2406_16282_amd/csrc/act_kernels.hip",
                  "paper_2406_16282_amd/csrc/act_codes.hpp",
                  "paper_2406_16282_amd/csrc/act_math.hpp",
                  "paper_2406_16282_amd/csrc/norm_kernels.hip",
                  "paper_2406_16282_amd/csrc/lmbp_device.hpp",
                  "paper_2406_16282_amd/csrc/gelu_poly.h")


def algorithmic_bytes(w, swiglu=False):
    """Bytes each kernel must move once (reads + writes), per launch."""
    eb = 2 if w.norm.dtype == "bf16" else 4
    rows, p = w.norm.rows, w.norm.cols
    n_norm = rows * p
    n_act = w.act.rows * w.act.cols
    ab = 2 if w.act.dtype == "bf16" else 4
    codes = 4 * ((n_act + 15) // 16)
    if swiglu:
        act = [("reswiglu2_fwd", 4 * n_act * ab + codes),          # g, u in; h, s out; codes out
               ("reswiglu2_bwd", 5 * n_act * ab + codes)]          # dh, u, s, codes in; dg, du out
    else:
        act = [(f"{w.act.op}_fwd", 2 * n_act * ab + codes),        # x in, y out, codes out
               (f"{w.act.op}_bwd", 2 * n_act * ab + codes)]        # dy, codes in, dx out
    return {
        f"{w.norm.op}_fwd": 2 * n_norm * eb + 4 * rows,            # x in, z out, rstd out
        act[0][0]: act[0][1],
        act[1][0]: act[1][1],
        f"{w.norm.op}_bwd": 3 * n_norm * eb + 4 * rows,            # dz, z, rstd in, dx out
    }


def source_hash():
    """SHA-256 of the kernel sources with comments removed and whitespace collapsed, so
    that only a change of the code itself invalidates the recorded counters."""
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(ROOT, rel)) as f:
            text = f.read()
        text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
        text = re.sub(r"//[^\n]*", " ", text)
        h.update(" ".join(text.split()).encode())
    return h.hexdigest()


def load_traffic(kernel, workload=WORKLOAD):
    """HBM traffic of `kernel` on `workload` from committed hardware-counter summaries, or
    None when there is none or the kernel sources changed since the counters were taken."""
    path = os.path.join(ROOT, "profiles", f"traffic_{kernel}_{workload}.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    if rec.get("source_sha256") != source_hash():
        return None
    return rec.get("traffic_bytes")


def _host_cpu():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def _oracle_step(spec, x, dz, g, dy, min_seconds):
    """Run the oracle's step on the given rows until `min_seconds` have passed; returns
    (passes, elapsed seconds). `spec` = (norm op, activation op, norm dtype, activation
    dtype, eps): plain values, so that worker processes need not import the package."""
    import oracle
    norm_op, act_op, dt_n, dt_a, eps = spec
    ofwd = {"msrms": oracle.msrms_fwd, "msln": oracle.msln_fwd}[norm_op]
    obwd = {"msrms": oracle.msrms_bwd, "msln": oracle.msln_bwd}[norm_op]
    afwd = {"resilu2": oracle.resilu2_fwd, "regelu2": oracle.regelu2_fwd}[act_op]
    abwd = {"resilu2": oracle.resilu2_bwd, "regelu2": oracle.regelu2_bwd}[act_op]
    passes = 0
    t0 = time.perf_counter()
    while True:
        z, r = ofwd(oracle.decode(x, dt_n), eps)
        z_s, r_s = oracle.encode(z, dt_n), r.astype(np.float32)
        y, codes = afwd(oracle.decode(g, dt_a))
        oracle.encode(y, dt_a)
        oracle.encode(abwd(oracle.decode(dy, dt_a), codes), dt_a)
        oracle.encode(obwd(oracle.decode(dz, dt_n), oracle.decode(z_s, dt_n), r_s), dt_n)
        passes += 1
        elapsed = time.perf_counter() - t0
        if elapsed >= min_seconds:
            return passes, elapsed


def _oracle_chunk(job):
    """Worker of the all-cores baseline: the oracle step on one row chunk."""
    spec, x, dz, g, dy, min_seconds = job
    return _oracle_step(spec, x, dz, g, dy, min_seconds)


def _spec(w):
    return (w.norm.op, w.act.op, w.norm.dtype, w.act.dtype, float(np.float32(w.norm.eps)))


def cpu_baseline(w, tensors, min_seconds=10.0):
    """The CPU oracle, as it stands, on the whole step (every row of every tensor),
    repeated until at least `min_seconds` of wall time; scaled to the same
    algorithmic-bytes unit as the GPU value. NumPy runs these elementwise and
    row-reduction ufuncs on one thread."""
    passes, elapsed = _oracle_step(_spec(w), *tensors, min_seconds)
    step_bytes = sum(algorithmic_bytes(w).values())
    return {
        "value": round(passes * step_bytes / elapsed / 1e9, 4),
        "unit": "GB/s",
        "cores": 1,
        "host_cpu": _host_cpu(),
        "host_cpus_visible": os.cpu_count(),
        "kind": "oracle",
        "sample": (f"{passes} full pass(es) of the step (all {w.norm.rows} rows of every tensor), "
                   f"fp64 NumPy, {elapsed:.2f} s wall"),
    }


def cpu_baseline_all_cores(w, tensors, pool, procs, min_seconds=5.0):
    """The same oracle on every host core at once: the step's rows split into `procs`
    chunks, one worker process each (the pool's processes are started before this
    process touches the GPU and never touch it), each repeating its chunk for
    `min_seconds`; rate = bytes of all chunk passes over the longest worker's wall time."""
    step_bytes = sum(algorithmic_bytes(w).values())
    x, dz, g, dy = tensors
    rn, ra = w.norm.rows, w.act.rows
    jobs = []
    for i in range(procs):
        a, b = rn * i // procs, rn * (i + 1) // procs
        c, d = ra * i // procs, ra * (i + 1) // procs
        jobs.append((_spec(w), x[a:b], dz[a:b], g[c:d], dy[c:d], min_seconds))
    res = pool.map(_oracle_chunk, jobs)
    # The chunks split the rows evenly (within one row), each 1/procs of the step.
    passes = sum(p for p, _ in res) / procs
    wall = max(e for _, e in res)
    return {
        "value": round(passes * step_bytes / wall / 1e9, 4),
        "unit": "GB/s",
        "cores": procs,
        "kind": "oracle",
        "sample": (f"{procs} worker processes, each {min_seconds:.0f}+ s of passes over 1/{procs} of the "
                   f"step's rows; {passes:.2f} step-equivalents in {wall:.2f} s"),
    }


def pair_report(torch, lmbp, inputs, dev, reps=40, cold_bytes=1 << 30, workloads=None):
    """Forward + backward GB/s of each op pair (norm, activation) on every workload:
    (B_fwd + B_bwd) / (t_fwd + t_bwd) with algorithmic bytes, per-launch durations
    from HIP-graph replays (launch-bound small kernels would otherwise measure the
    host), cold and warm.

    Cold: enough tensor sets (at most 64) that each kernel's launches cycle over at
    least `cold_bytes` of distinct memory, and at least the workload's blocks;
    forwards run over the sets in order, backwards in reverse (the training order).
    Warm: one set, relaunched (inputs partly resident in the 256 MB memory-side
    cache)."""
    out = {}
    mk = lambda: torch.cuda.Event(enable_timing=True)
    for name, w in inputs.WORKLOADS.items():
        if workloads is not None and name not in workloads:
            continue
        nb = algorithmic_bytes(w)
        names = list(nb)
        eps = float(np.float32(w.norm.eps))
        T = lambda a: inputs.storage_to_torch(a, dev)
        base = (T(w.norm_x()), T(w.norm_dz()), T(w.act_x()), T(w.act_dy()))
        set_bytes = sum(nb.values())
        nsets = max(w.blocks, 3, min(64, -(-cold_bytes // min(nb.values()))))
        nfwd = {"msrms": lmbp.msrms_fwd, "msln": lmbp.msln_fwd}[w.norm.op]
        nbwd = {"msrms": lmbp.msrms_bwd, "msln": lmbp.msln_bwd}[w.norm.op]
        afwd = {"resilu2": lmbp.resilu2_fwd, "regelu2": lmbp.regelu2_fwd}[w.act.op]
        abwd = {"resilu2": lmbp.resilu2_bwd, "regelu2": lmbp.regelu2_bwd}[w.act.op]
        # SiLU workloads (the LLaMA MLP) also time the fused SwiGLU pair on the gate shape:
        # u is the up projection, dy serves as dh; its codes are those of g, as above.
        glu = w.act.op == "resilu2"
        if glu:
            gb = algorithmic_bytes(w, swiglu=True)
            nb["reswiglu2_fwd"], nb["reswiglu2_bwd"] = gb["reswiglu2_fwd"], gb["reswiglu2_bwd"]
            names = list(nb)
            base = base + (T(w.act_u()),)

        def make_set(k):
            # Set k holds the block-0 tensors rotated by k * 4099 elements: same
            # values and distribution, distinct memory.
            x, dz, g, dy, *rest = (t if k == 0 else torch.roll(t.view(-1), k * 4099).view_as(t) for t in base)
            st = {"x": x, "dz": dz, "g": g, "dy": dy, "z": torch.empty_like(x),
                  "rstd": torch.empty(w.norm.rows, dtype=torch.float32, device=dev),
                  "h": torch.empty_like(g), "dg": torch.empty_like(dy), "dx": torch.empty_like(dz),
                  "codes": torch.empty(lmbp.codes_words(g.numel()), dtype=torch.int32, device=dev)}
            fns = [lambda: nfwd(st["x"], eps, z=st["z"], rstd=st["rstd"]),
                   lambda: afwd(st["g"], y=st["h"], codes=st["codes"]),
                   lambda: abwd(st["dy"], st["codes"], dx=st["dg"]),
                   lambda: nbwd(st["dz"], st["z"], st["rstd"], dx=st["dx"])]
            if glu:
                st.update(u=rest[0], s=torch.empty_like(g), du=torch.empty_like(g))
                fns += [lambda: lmbp.reswiglu2_fwd(st["g"], st["u"], h=st["h"], s=st["s"], codes=st["codes"]),
                        lambda: lmbp.reswiglu2_bwd(st["dy"], st["u"], st["s"], st["codes"], dg=st["dg"],
                                                   du=st["du"])]
            return fns

        sets = [make_set(k) for k in range(nsets)]
        for ks in sets:
            ks[0]()
            ks[1]()
            if glu:
                ks[4]()
        torch.cuda.synchronize()

        def launch_us(i, order):
            """Average duration of kernel i over `reps` launches cycling through `order`."""
            seq = [order[j % len(order)] for j in range(max(reps, len(order)))]
            side = torch.cuda.Stream()
            side.wait_stream(torch.cuda.current_stream())
            with torch.cuda.stream(side):
                for k in seq:
                    sets[k][i]()
            torch.cuda.current_stream().wait_stream(side)
            graph = torch.cuda.CUDAGraph()
            with torch.cuda.graph(graph):
                for k in seq:
                    sets[k][i]()
            graph.replay()
            a, b = mk(), mk()
            a.record()
            graph.replay()
            graph.replay()
            b.record()
            torch.cuda.synchronize()
            us = a.elapsed_time(b) * 1e3 / (2 * len(seq))
            del graph
            return us

        fwd_order = list(range(nsets))
        bwd_order = fwd_order[::-1]
        cold = {n: launch_us(i, bwd_order if n.endswith("_bwd") else fwd_order) for i, n in enumerate(names)}
        warm = {n: launch_us(i, [0]) for i, n in enumerate(names)}
        rec = {"sets": nsets, "set_bytes": set_bytes}
        pairs = [("norm", (names[0], names[3])), ("act", (names[1], names[2]))]
        if glu:
            pairs.append(("swiglu", (names[4], names[5])))
        for pair, (f, b) in pairs:
            byt = nb[f] + nb[b]
            gbs = byt / ((cold[f] + cold[b]) * 1e-6) / 1e9
            rec[pair] = {"op": f[:-4], "fwd_us": round(cold[f], 2), "bwd_us": round(cold[b], 2),
                         "bytes": byt, "GBps": round(gbs, 1), "pct_of_peak": round(100 * gbs / HBM_PEAK_GBS, 1),
                         "warm_GBps": round(byt / ((warm[f] + warm[b]) * 1e-6) / 1e9, 1)}
        out[name] = rec
        extra = f", swiglu {rec['swiglu']['GBps']} GB/s" if glu else ""
        print(f"[bench] pairs {name}: norm {rec['norm']['GBps']} GB/s, act {rec['act']['GBps']} GB/s"
              f"{extra} ({nsets} sets)", file=sys.stderr, flush=True)
        del sets, base
        torch.cuda.empty_cache()
    return out


def _graph_us(torch, fns, order, reps=48):
    """Average duration (us) of one launch over `reps` launches of fns[k] for k cycling
    through `order`, replayed from a HIP graph (launch-bound small kernels would
    otherwise measure the host)."""
    seq = [order[j % len(order)] for j in range(max(reps, len(order)))]
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        for k in seq:
            fns[k]()
    torch.cuda.current_stream().wait_stream(side)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        for k in seq:
            fns[k]()
    graph.replay()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    graph.replay()
    graph.replay()
    b.record()
    torch.cuda.synchronize()
    return a.elapsed_time(b) * 1e3 / (2 * len(seq))


def variants_report(torch, lmbp, inputs, dev, cold_bytes=1 << 30):
    """Forward + backward GB/s of the k-bit family kernels (stepact_fwd / stepact_bwd,
    k = 1, 2, 3, 4, and ReGELU2-d) next to the dedicated k = 2 kernels, on the ViT-B
    batch-64 GELU and LLaMA-7B gate SiLU activation shapes (bf16), cold: launches cycle
    over enough tensor sets to touch 1 GiB, forwards in set order, backwards reversed.
    Bytes per element: read x and write y (forward), read dy and write dx (backward),
    plus the k-bit codes both ways (floor(32 / k) codes per 32-bit word)."""
    from paper_2406_16282_amd import variants
    shapes = {"vit_b_bs64_bf16": ("gelu", 64 * 197, 3072, 1.5),
              "llama7b_gate_bf16": ("silu", 4 * 2048, 11008, 2.0)}
    out = {}
    for name, (act, rows, cols, std) in shapes.items():
        n = rows * cols
        x0 = inputs.storage_to_torch(inputs.normal((rows, cols), std, "bf16", tensor_id=2), dev)
        dy0 = inputs.storage_to_torch(inputs.normal((rows, cols), 1e-2, "bf16", tensor_id=3), dev)
        nsets = max(3, min(16, -(-cold_bytes // (4 * n))))
        sets = [(x0, dy0) if k == 0 else (torch.roll(x0.view(-1), k * 4099).view_as(x0),
                                          torch.roll(dy0.view(-1), k * 4099).view_as(dy0))
                for k in range(nsets)]
        outs = [(torch.empty_like(x0), torch.empty_like(x0)) for _ in range(nsets)]
        members = []
        span = 3.0 if act == "gelu" else 6.0
        for bits in (1, 2, 3, 4):
            m = (1 << bits) - 1
            c = [span * (2 * i / (m - 1) - 1) if m > 1 else 0.0 for i in range(m)]
            a = [1.0 / (m + 1)] * (m - 1)
            members.append((f"k{bits}_even", bits, c, variants.levels_of(a)))
        if act == "gelu":
            members.append(("regelu2_d", 2, list(variants.REGELU2D_C), variants.levels_of(variants.REGELU2D_A)))
        rec = {}
        for label, bits, c, lv in members + [("dedicated_k2", 2, None, None)]:
            words = int(lmbp.lib().lmbp_stepact_codes_bytes(bits, n)) // 4
            codes = [torch.empty(words, dtype=torch.int32, device=dev) for _ in range(nsets)]
            if c is None:
                fwd_op = lmbp.regelu2_fwd if act == "gelu" else lmbp.resilu2_fwd
                bwd_op = lmbp.regelu2_bwd if act == "gelu" else lmbp.resilu2_bwd
                fwd = [lambda k=k: fwd_op(sets[k][0], y=outs[k][0], codes=codes[k]) for k in range(nsets)]
                bwd = [lambda k=k: bwd_op(sets[k][1], codes[k], dx=outs[k][1]) for k in range(nsets)]
            else:
                fwd = [lambda k=k: lmbp.stepact_fwd(sets[k][0], act, c, bits, y=outs[k][0], codes=codes[k])
                       for k in range(nsets)]
                bwd = [lambda k=k: lmbp.stepact_bwd(sets[k][1], codes[k], lv, bits, dx=outs[k][1])
                       for k in range(nsets)]
            for f in fwd:
                f()
            torch.cuda.synchronize()
            order = list(range(nsets))
            tf = _graph_us(torch, fwd, order)
            tb = _graph_us(torch, bwd, order[::-1])
            byt = 2 * (2 * 2 * n + 4 * words)
            rec[label] = {"bits": bits, "stored_bits_per_elt": round(32 * words / n, 3),
                          "fwd_us": round(tf, 2), "bwd_us": round(tb, 2), "bytes": byt,
                          "GBps": round(byt / ((tf + tb) * 1e-6) / 1e9, 1),
                          "pct_of_peak": round(100 * byt / ((tf + tb) * 1e-6) / 1e9 / HBM_PEAK_GBS, 1)}
            del codes
        out[name] = rec
        print(f"[bench] variants {name}: " + ", ".join(f"{k} {v['GBps']}" for k, v in rec.items()),
              file=sys.stderr, flush=True)
        del sets, outs
        torch.cuda.empty_cache()
    return out


MFMA_BF16_PEAK_TFLOPS = 2500.0   # MI355X dense bf16 matrix peak, AMD published

LINEAR_SHAPES = {
    # name: (m, n, k, act, bias) -- the MLP's first projection feeding the activation
    "vit_b_bs64_fc1_bf16": (64 * 197, 3072, 768, "gelu", True),
    "llama7b_gate_bf16": (4 * 2048, 11008, 4096, "silu", False),
}


LINEAR_GLU_SHAPE = (4 * 2048, 11008, 4096)   # LLaMA-7B MLP: x [m, k], gate and up [n, k]


def _timed_all(torch, fns, reps, trials=5):
    """Median over `trials` of the mean duration (us) of `reps` back-to-back calls, the
    trials of the callables interleaved (so clock drift affects all alike), after a
    warm-up of the same length (the clocks ramp up under load)."""
    mk = lambda: torch.cuda.Event(enable_timing=True)
    for fn in fns:
        for _ in range(reps):
            fn()
    torch.cuda.synchronize()
    res = [[] for _ in fns]
    for _ in range(trials):
        for i, fn in enumerate(fns):
            a, b = mk(), mk()
            a.record()
            for _ in range(reps):
                fn()
            b.record()
            torch.cuda.synchronize()
            res[i].append(a.elapsed_time(b) * 1e3 / reps)
    return [float(np.median(r)) for r in res]


def linear_report(torch, lmbp, inputs, dev, reps):
    """Fused linear + ReGELU2 / ReSiLU2 forward against the unfused sequence (library
    GEMM through torch, i.e. hipBLASLt, writing z, then the activation kernel reading
    it), on the ViT-B and LLaMA-7B MLP shapes. Durations: HIP events around `reps`
    back-to-back launches on the current stream, median of five trials interleaved
    across the four variants after a warm-up of the same length."""
    out = {}
    timed_all = lambda fns: _timed_all(torch, fns, reps)

    for name, (m, n, k, act, has_bias) in LINEAR_SHAPES.items():
        T = lambda a: inputs.storage_to_torch(a, dev)
        x = T(inputs.normal((m, k), 1.0, "bf16", tensor_id=inputs.LIN_X))
        w = T(inputs.normal((n, k), k ** -0.5 * 2.0, "bf16", tensor_id=inputs.LIN_W))
        b = T(inputs.normal((n,), 0.1, "bf16", tensor_id=inputs.LIN_B)) if has_bias else None
        y = torch.empty((m, n), dtype=torch.bfloat16, device=dev)
        z = torch.empty((m, n), dtype=torch.bfloat16, device=dev)
        codes = torch.empty(lmbp.codes_words(m * n), dtype=torch.int32, device=dev)
        afwd = lmbp.regelu2_fwd if act == "gelu" else lmbp.resilu2_fwd
        wt = w.t()

        def gemm():
            if b is None:
                torch.matmul(x, wt, out=z)
            else:
                torch.addmm(b, x, wt, out=z)

        t_fused, t_gemm, t_act, t_unfused = timed_all([
            lambda: lmbp.linear_act_fwd(x, w, b, act=act, y=y, codes=codes),
            gemm,
            lambda: afwd(z, y=y, codes=codes),
            lambda: (gemm(), afwd(z, y=y, codes=codes)),
        ])
        flops = 2.0 * m * n * k
        tf = flops / (t_fused * 1e-6) / 1e12
        out[name] = {
            "m": m, "n": n, "k": k, "act": act, "bias": has_bias,
            "fused_us": round(t_fused, 1), "fused_TFLOPs": round(tf, 1),
            "unfused_us": round(t_unfused, 1), "library_gemm_us": round(t_gemm, 1),
            "act_kernel_us": round(t_act, 1),
            "library_gemm_TFLOPs": round(flops / (t_gemm * 1e-6) / 1e12, 1),
            "speedup_vs_unfused": round(t_unfused / t_fused, 3),
            "hbm_bytes_saved": 2 * 2 * m * n,   # z written by the GEMM and read by the activation
            "roofline": {"bound": "mfma", "achieved": round(tf, 1), "peak": MFMA_BF16_PEAK_TFLOPS,
                         "unit": "TFLOP/s", "frac": round(tf / MFMA_BF16_PEAK_TFLOPS, 4)},
        }
        print(f"[bench] linear {name}: fused {t_fused:.1f} us ({tf:.0f} TFLOP/s), unfused "
              f"{t_unfused:.1f} us (library GEMM {t_gemm:.1f} + activation {t_act:.1f})",
              file=sys.stderr, flush=True)
        del x, w, b, y, z, codes
        torch.cuda.empty_cache()

    # The gated form on the LLaMA-7B MLP: gate and up projections + ReSiLU2 inside SwiGLU.
    m, n, k = LINEAR_GLU_SHAPE
    name = "llama7b_mlp_swiglu_bf16"
    T = lambda a: inputs.storage_to_torch(a, dev)
    x = T(inputs.normal((m, k), 1.0, "bf16", tensor_id=inputs.LIN_X))
    wg = T(inputs.normal((n, k), k ** -0.5 * 2.0, "bf16", tensor_id=inputs.LIN_W))
    wu = T(inputs.normal((n, k), k ** -0.5, "bf16", tensor_id=inputs.LIN_B))
    h, s, u, g = (torch.empty((m, n), dtype=torch.bfloat16, device=dev) for _ in range(4))
    codes = torch.empty(lmbp.codes_words(m * n), dtype=torch.int32, device=dev)
    wgt, wut = wg.t(), wu.t()

    def unfused():
        torch.matmul(x, wgt, out=g)
        torch.matmul(x, wut, out=u)
        lmbp.reswiglu2_fwd(g, u, h=h, s=s, codes=codes)

    t_fused, t_unfused = timed_all([
        lambda: lmbp.linear_swiglu_fwd(x, wg, wu, h=h, s=s, u=u, codes=codes), unfused])
    flops = 4.0 * m * n * k
    tf = flops / (t_fused * 1e-6) / 1e12
    out[name] = {
        "m": m, "n": n, "k": k, "act": "silu (SwiGLU)", "bias": False,
        "fused_us": round(t_fused, 1), "fused_TFLOPs": round(tf, 1),
        "unfused_us": round(t_unfused, 1),
        "speedup_vs_unfused": round(t_unfused / t_fused, 3),
        "hbm_bytes_saved": 3 * 2 * m * n,   # g written and read, u read back by the activation
        "roofline": {"bound": "mfma", "achieved": round(tf, 1), "peak": MFMA_BF16_PEAK_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(tf / MFMA_BF16_PEAK_TFLOPS, 4)},
    }
    print(f"[bench] linear {name}: fused {t_fused:.1f} us ({tf:.0f} TFLOP/s), unfused "
          f"{t_unfused:.1f} us (two library GEMMs + SwiGLU activation)", file=sys.stderr, flush=True)

    # MS-RMSNorm in front of the same gated layer: the norm's statistics pass plus the GEMM
    # that also writes the norm's output z, against the norm kernel followed by the fused
    # gated layer on z (the same layer, the same saved z and rstd).
    name = "llama7b_msrms_mlp_swiglu_bf16"
    eps = float(np.float32(1e-5))
    xn = T(inputs.normal((m, k), 1.0, "bf16", tensor_id=inputs.NORM_X))
    zn = torch.empty_like(xn)
    rstd = torch.empty(m, dtype=torch.float32, device=dev)
    t_fused, t_unfused, t_norm = timed_all([
        lambda: lmbp.msrms_linear_swiglu_fwd(xn, wg, wu, eps, h=h, s=s, u=u, codes=codes, z=zn, rstd=rstd),
        lambda: (lmbp.msrms_fwd(xn, eps, z=zn, rstd=rstd),
                 lmbp.linear_swiglu_fwd(zn, wg, wu, h=h, s=s, u=u, codes=codes)),
        lambda: lmbp.msrms_fwd(xn, eps, z=zn, rstd=rstd)])
    tf = flops / (t_fused * 1e-6) / 1e12
    out[name] = {
        "m": m, "n": n, "k": k, "act": "silu (SwiGLU), MS-RMSNorm in front", "bias": False,
        "fused_us": round(t_fused, 1), "fused_TFLOPs": round(tf, 1),
        "unfused_us": round(t_unfused, 1), "norm_kernel_us": round(t_norm, 1),
        "speedup_vs_unfused": round(t_unfused / t_fused, 3),
        "roofline": {"bound": "mfma", "achieved": round(tf, 1), "peak": MFMA_BF16_PEAK_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(tf / MFMA_BF16_PEAK_TFLOPS, 4)},
    }
    print(f"[bench] linear {name}: fused {t_fused:.1f} us, unfused {t_unfused:.1f} us "
          f"(norm kernel {t_norm:.1f} + fused gated layer)", file=sys.stderr, flush=True)
    return out


BLOCK_SHAPES = {
    # name: (tokens, hidden p, MLP width F, architecture)
    "vit_b_bs64_mlp_bf16": (64 * 197, 768, 3072, "vit"),
    "llama7b_mlp_bf16": (4 * 2048, 4096, 11008, "llama"),
}


def block_report(torch, dev, reps):
    """Training step (forward + backward with input and weight gradients) of a whole MLP
    block in bf16, torch's modules against this library's: MS-LN / MS-RMSNorm (the norm's
    affine merged into the next layer), the first projection fused with ReGELU2 (ViT-B) or
    with ReSiLU2 inside SwiGLU (LLaMA-7B), then the library's plain second projection. Step
    time: median of interleaved trials of `reps` steps; memory: the bytes the forward leaves
    allocated for the backward (all saved activations, beyond the inputs and the output)."""
    from torch import nn
    from paper_2406_16282_amd.nn import LinearReGELU2, LinearReSwiGLU2, MSLayerNorm, MSRMSNorm
    bf = dict(device=dev, dtype=torch.bfloat16)
    out = {}
    for name, (tok, p, f, arch) in BLOCK_SHAPES.items():
        gen = torch.Generator(device=dev).manual_seed(0)
        x = torch.randn(tok, p, generator=gen, **bf)
        dy = torch.randn(tok, p, generator=gen, **bf) * 1e-2
        if arch == "vit":
            ln, fc1, fc2 = nn.LayerNorm(p, eps=1e-6, **bf), nn.Linear(p, f, **bf), nn.Linear(f, p, **bf)
            ms, fused, fc2b = MSLayerNorm(1e-6), LinearReGELU2(p, f, device=dev), nn.Linear(f, p, **bf)
            torch_block = lambda xi: fc2(nn.functional.gelu(fc1(ln(xi))))
            our_block = lambda xi: fc2b(fused(ms(xi)))
        else:
            rms = nn.RMSNorm(p, eps=1e-5, **bf)
            gate, up, down = (nn.Linear(p, f, bias=False, **bf), nn.Linear(p, f, bias=False, **bf),
                              nn.Linear(f, p, bias=False, **bf))
            ms, fused, downb = MSRMSNorm(1e-5), LinearReSwiGLU2(p, f, device=dev), nn.Linear(f, p, bias=False, **bf)

            def torch_block(xi):
                z = rms(xi)
                return down(nn.functional.silu(gate(z)) * up(z))
            our_block = lambda xi: downb(fused(ms(xi)))

        def step(block):
            xi = x.detach().requires_grad_(True)
            block(xi).backward(dy)

        def kept_bytes(block):
            step(block)                      # gradients allocated before the measurement
            torch.cuda.synchronize()
            xi = x.detach().requires_grad_(True)
            before = torch.cuda.memory_allocated()
            y = block(xi)
            torch.cuda.synchronize()
            kept = torch.cuda.memory_allocated() - before - y.numel() * y.element_size()
            del y, xi
            return kept

        mem_t, mem_o = kept_bytes(torch_block), kept_bytes(our_block)
        t_torch, t_ours = _timed_all(torch, [lambda: step(torch_block), lambda: step(our_block)], reps)
        out[name] = {
            "tokens": tok, "hidden": p, "mlp": f,
            "torch_step_us": round(t_torch, 1), "ours_step_us": round(t_ours, 1),
            "speedup": round(t_torch / t_ours, 3),
            "torch_kept_bytes_per_token": round(mem_t / tok, 1),
            "ours_kept_bytes_per_token": round(mem_o / tok, 1),
            "memory_ratio": round(mem_o / mem_t, 4),
        }
        print(f"[bench] block {name}: step {t_torch:.1f} us torch vs {t_ours:.1f} us ours; activations "
              f"{mem_t / tok:.0f} vs {mem_o / tok:.0f} B/token", file=sys.stderr, flush=True)
        torch.cuda.empty_cache()
    return out


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=1000)
    ap.add_argument("--warmup", type=int, default=200,
                    help="untimed steps first; a few hundred bring the clocks to their steady state")
    ap.add_argument("--workload", default=WORKLOAD,
                    help="the step's tensors (a name from inputs.WORKLOADS; the default is the "
                         "LLaMA-7B-shaped configuration the metric is quoted on)")
    ap.add_argument("--graph", action="store_true",
                    help="replay the timed steps and per-kernel loops from HIP graphs instead of launching "
                         "them from Python (for workloads whose kernels are shorter than a Python launch)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--swiglu", action="store_true",
                    help="use ReSiLU2 fused with the SwiGLU product (h = SiLU(g) * u) in the step")
    ap.add_argument("--pairs", action="store_true",
                    help="also report forward+backward GB/s of each op pair on every workload")
    ap.add_argument("--blocks", action="store_true",
                    help="also report the training step time and kept activation memory of whole "
                         "ViT-B and LLaMA-7B MLP blocks, torch modules against this library's")
    ap.add_argument("--variants", action="store_true",
                    help="also report the k-bit family kernels (k = 1..4, ReGELU2-d) against the "
                         "dedicated k = 2 kernels")
    ap.add_argument("--linear", action="store_true",
                    help="also report the fused linear + activation forward against the unfused "
                         "library GEMM + activation kernel")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU: the hot path is row- and element-local and runs "
              f"per GPU with no communication, so --gpus {args.gpus} is not supported.",
              file=sys.stderr)
        sys.exit(2)
    if args.steps < 1 or args.warmup < 0:
        sys.exit("--steps must be >= 1 and --warmup >= 0")

    from paper_2406_16282_amd import inputs

    wl = args.workload
    if wl not in inputs.WORKLOADS:
        sys.exit(f"--workload must be one of {', '.join(inputs.WORKLOADS)}")
    if args.swiglu and inputs.WORKLOADS[wl].act.op != "resilu2":
        sys.exit("--swiglu needs a SiLU workload")

    # The CPU oracle is timed after the GPU legs, so that the GPU is not left idle for the
    # oracle's tens of seconds right before its timed region. Its all-cores worker pool is
    # started here, before this process touches the GPU (a process that has initialised
    # the GPU does not start programs).
    run_cpu = not args.no_cpu_baseline and not args.swiglu
    pool = procs = None
    if run_cpu:
        import multiprocessing as mp
        procs = max(1, min(16, os.cpu_count() or 1))
        pool = mp.get_context("spawn").Pool(procs)

    import torch
    import paper_2406_16282_amd as lmbp

    if not torch.cuda.is_available():
        sys.exit("bench.py needs a GPU")
    dev = torch.device("cuda:0")
    w = inputs.WORKLOADS[wl]
    nb = algorithmic_bytes(w, args.swiglu)
    eps = float(np.float32(w.norm.eps))
    print(f"[bench] generating {wl} inputs", file=sys.stderr, flush=True)
    T = lambda a: inputs.storage_to_torch(a, dev)
    x, dz, g, dy = T(w.norm_x()), T(w.norm_dz()), T(w.act_x()), T(w.act_dy())
    u = T(w.act_u()) if args.swiglu else None
    nfwd = {"msrms": lmbp.msrms_fwd, "msln": lmbp.msln_fwd}[w.norm.op]
    nbwd = {"msrms": lmbp.msrms_bwd, "msln": lmbp.msln_bwd}[w.norm.op]
    afwd = {"resilu2": lmbp.resilu2_fwd, "regelu2": lmbp.regelu2_fwd}[w.act.op]
    abwd = {"resilu2": lmbp.resilu2_bwd, "regelu2": lmbp.regelu2_bwd}[w.act.op]
    stream = torch.cuda.current_stream(dev)
    names = list(nb.keys())

    class Set:
        """One full set of step tensors (inputs and saved state / outputs)."""
        def __init__(self, x, dz, g, dy, u):
            self.x, self.dz, self.g, self.dy, self.u = x, dz, g, dy, u
            self.z = torch.empty_like(x)
            self.rstd = torch.empty(w.norm.rows, dtype=torch.float32, device=dev)
            self.h = torch.empty_like(g)
            self.codes = torch.empty(lmbp.codes_words(g.numel()), dtype=torch.int32, device=dev)
            self.dg = torch.empty_like(dy)
            self.dx = torch.empty_like(dz)
            if u is not None:
                self.s = torch.empty_like(g)
                self.du = torch.empty_like(u)

        def kernels(self, stream):
            # stream None: the current stream (what a graph capture records).
            if self.u is None:
                act = [lambda: afwd(self.g, y=self.h, codes=self.codes, stream=stream),
                       lambda: abwd(self.dy, self.codes, dx=self.dg, stream=stream)]
            else:
                act = [lambda: lmbp.reswiglu2_fwd(self.g, self.u, h=self.h, s=self.s, codes=self.codes,
                                                  stream=stream),
                       lambda: lmbp.reswiglu2_bwd(self.dy, self.u, self.s, self.codes, dg=self.dg,
                                                  du=self.du, stream=stream)]
            return [lambda: nfwd(self.x, eps, z=self.z, rstd=self.rstd, stream=stream), act[0], act[1],
                    lambda: nbwd(self.dz, self.z, self.rstd, dx=self.dx, stream=stream)]

    # Python's garbage collector runs once here, before the tensor sets are built (GPU
    # copies), and is then off through the timed loops: a collection takes tens of ms, during
    # which the GPU would sit idle right before (or, inside the loops, within) the timed
    # region; the sets' copies and the priming launches run right before the warm-up.
    gc.collect()
    gc.disable()

    # Three tensor sets. Step k runs the forward kernels on set k % 3 and the backward
    # kernels on set (k - 1) % 3, i.e. the backward consumes saved state written one
    # full step (about 1.1 GB of traffic) earlier, as in training where a layer's
    # forward and backward are separated by the rest of the network: no kernel finds
    # its inputs in the 256 MB memory-side cache.
    clone = lambda t: None if t is None else t.clone()
    sets = [Set(x, dz, g, dy, u)] + [Set(x.clone(), dz.clone(), g.clone(), dy.clone(), clone(u))
                                     for _ in range(2)]
    ks = [st.kernels(stream) for st in sets]
    kc = [st.kernels(None) for st in sets]   # for graph capture

    def step(k, kl=ks):
        f, b = kl[k % 3], kl[(k - 1) % 3]
        f[0]()
        f[1]()
        b[2]()
        b[3]()

    def captured(fn):
        """A HIP graph of what fn() launches on the current stream (captured on a side
        stream after one eager pass there, as torch requires)."""
        side = torch.cuda.Stream(dev)
        side.wait_stream(stream)
        with torch.cuda.stream(side):
            fn()
        stream.wait_stream(side)
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            fn()
        torch.cuda.synchronize()
        return graph

    k0 = args.warmup
    graph = None if not args.graph else captured(lambda: [step(k0 + k, kc) for k in range(args.steps)])
    for st in ks:          # every set holds valid saved state before the first step
        st[0]()
        st[1]()
    for k in range(args.warmup):
        step(k)
    torch.cuda.synchronize()
    print(f"[bench] warmup {args.warmup} steps done; timing {args.steps}", file=sys.stderr, flush=True)

    # Timed region: K steps back to back, bracketed by events on the kernels' stream,
    # launched from Python; with --graph the K steps are replayed from one HIP graph (the
    # same launches without the host in the loop, which small workloads need; on this stack
    # a graph node costs slightly more GPU time than a back-to-back launch, so it is not the
    # default).
    mk = lambda: torch.cuda.Event(enable_timing=True)
    start, end = mk(), mk()
    t_wall0 = time.perf_counter()
    start.record(stream)
    if graph is None:
        for k in range(args.steps):
            step(k0 + k)
    else:
        graph.replay()
    end.record(stream)
    torch.cuda.synchronize()
    t_wall = time.perf_counter() - t_wall0
    ms_total = start.elapsed_time(end)
    ms_step = ms_total / args.steps
    del graph

    # Per-kernel launch duration: each kernel launched K times back to back, cycling over
    # the three tensor sets (consecutive launches do not share a working set), timed with
    # events around the launches on the same stream (replayed from a graph with --graph).
    print("[bench] per-kernel timing", file=sys.stderr, flush=True)
    per_kernel_ms = {}
    for i, n in enumerate(names):
        # two untimed rounds over the sets first, so that the host is well ahead of the
        # GPU when the timed launches start (otherwise the first of them can wait for it)
        for j in range(6):
            ks[j % 3][i]()
        g_i = None if not args.graph else captured(lambda: [kc[j % 3][i]() for j in range(args.steps)])
        a, b = mk(), mk()
        a.record(stream)
        if g_i is None:
            for j in range(args.steps):
                ks[j % 3][i]()
        else:
            g_i.replay()
        b.record(stream)
        torch.cuda.synchronize()
        per_kernel_ms[n] = a.elapsed_time(b) / args.steps
        del g_i
    del sets, ks, kc

    # Plain-copy reference of known size: the practical streaming ceiling, and the
    # calibration point for hardware byte counters.
    copy_bytes = 384 * 2 ** 20
    pairs = [(torch.ones(copy_bytes, dtype=torch.uint8, device=dev),
              torch.empty(copy_bytes, dtype=torch.uint8, device=dev)) for _ in range(3)]
    for src, dst in pairs:
        lmbp.copy_bytes(src, dst, stream=stream)
    a, b = mk(), mk()
    a.record(stream)
    for j in range(args.steps):
        src, dst = pairs[j % 3]
        lmbp.copy_bytes(src, dst, stream=stream)
    b.record(stream)
    torch.cuda.synchronize()
    copy_ms = a.elapsed_time(b) / args.steps
    del pairs

    # The same plain copy at each kernel's own size (half its bytes read, half written),
    # cold in the same way (three buffer pairs in rotation) and launched the same way as the
    # per-kernel loop (replayed from a graph with --graph): what pure streaming of that many
    # bytes costs per launch on this GPU, fixed per-launch cost included.
    print("[bench] same-size copies", file=sys.stderr, flush=True)
    copy_same_ms = {}
    for n in names:
        half = (nb[n] // 2) // 16 * 16
        pairs = [(torch.ones(half, dtype=torch.uint8, device=dev),
                  torch.empty(half, dtype=torch.uint8, device=dev)) for _ in range(3)]
        copy = lambda j, st: lmbp.copy_bytes(pairs[j % 3][0], pairs[j % 3][1], stream=st)
        for j in range(6):
            copy(j, stream)
        g_c = None if not args.graph else captured(lambda: [copy(j, None) for j in range(args.steps)])
        a, b = mk(), mk()
        a.record(stream)
        if g_c is None:
            for j in range(args.steps):
                copy(j, stream)
        else:
            g_c.replay()
        b.record(stream)
        torch.cuda.synchronize()
        copy_same_ms[n] = a.elapsed_time(b) / args.steps
        del g_c, pairs
    gc.enable()

    bytes_step = sum(nb.values())
    value = bytes_step / (ms_step * 1e-3) / 1e9
    per_kernel = {n: {"us": round(per_kernel_ms[n] * 1e3, 2),
                      "bytes": nb[n],
                      "GBps": round(nb[n] / (per_kernel_ms[n] * 1e-3) / 1e9, 1),
                      "copy_same_bytes_us": round(copy_same_ms[n] * 1e3, 2),
                      "copy_over_kernel": round(copy_same_ms[n] / per_kernel_ms[n], 3)}
                  for n in names}
    dominant = max(names, key=lambda n: per_kernel_ms[n])
    achieved = nb[dominant] / (per_kernel_ms[dominant] * 1e-3) / 1e9
    n_act = w.act.rows * w.act.cols
    out = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": wl + ("_fused" if args.swiglu else ""),
            "storage": w.act.dtype,
            "norm": f"{w.norm.op} [{w.norm.rows}x{w.norm.cols}] eps={w.norm.eps:g}",
            "act": (f"reswiglu2 (SiLU(g) * u) [{w.act.rows}x{w.act.cols}]" if args.swiglu
                    else f"{w.act.op} [{w.act.rows}x{w.act.cols}]"),
            "bytes_per_step": bytes_step,
            "elements_per_step": 2 * (n_act + w.norm.rows * w.norm.cols),
        },
        "pct_of_hbm_peak": round(100.0 * value / HBM_PEAK_GBS, 1),
        "elements_per_s": round(2 * (n_act + w.norm.rows * w.norm.cols) / (ms_step * 1e-3), 1),
        "saved_bytes_per_elt": {
            w.act.op: lmbp.codes_bytes(n_act) / n_act,
            w.norm.op: 4.0 / w.norm.cols,
            f"{w.act.op}_dense_reference": 2.0 if w.act.dtype == "bf16" else 4.0,
        },
        "per_kernel": per_kernel,
        "roofline": {
            "kernel": dominant,
            "bound": "hbm",
            "achieved": round(achieved, 1),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4),
            "traffic": load_traffic(dominant + ("_fused" if args.swiglu else ""), wl),
        },
        "copy_reference": {"bytes_moved": 2 * copy_bytes, "us": round(copy_ms * 1e3, 2),
                           "GBps": round(2 * copy_bytes / (copy_ms * 1e-3) / 1e9, 1)},
        # Step time minus the per-kernel durations measured in their own loops: the gaps
        # between launches (a few us; within run-to-run noise it can come out slightly negative).
        "step_minus_kernel_sum_us": round(ms_step * 1e3 - sum(per_kernel_ms.values()) * 1e3, 2),
        # The step's bytes over the sum of the four kernels' own launch durations (the pairs'
        # (B_fwd + B_bwd) / (t_fwd + t_bwd) summed over both pairs); `value` is the wall-clock rate.
        "kernels_only_GBps": round(bytes_step / (sum(per_kernel_ms.values()) * 1e-3) / 1e9, 1),
        "wall_s_timed": round(t_wall, 4),
        "launch": "hip_graph" if args.graph else "eager",
    }
    # The other ops the metric names, MS-LN and ReGELU2, on the ViT-B batch-64 bf16 shapes:
    # cold forward + backward GB/s of each pair, launches replayed from HIP graphs (as
    # --pairs reports them for every workload).
    if not args.pairs:
        print("[bench] MS-LN and ReGELU2 pairs on vit_b_bs64_bf16_x12", file=sys.stderr, flush=True)
        vit = pair_report(torch, lmbp, inputs, dev, workloads=("vit_b_bs64_bf16_x12",))["vit_b_bs64_bf16_x12"]
        out["pairs_vit_b_bs64_bf16"] = {rec["op"]: {k: rec[k] for k in ("fwd_us", "bwd_us", "bytes", "GBps",
                                                                      "pct_of_peak")}
                                        for rec in (vit["norm"], vit["act"])}
    if args.pairs:
        print("[bench] op pairs on every workload", file=sys.stderr, flush=True)
        out["pairs"] = pair_report(torch, lmbp, inputs, dev)
        out["pairs"]["copy_GBps"] = out["copy_reference"]["GBps"]
    if args.linear:
        print("[bench] fused linear + activation", file=sys.stderr, flush=True)
        out["linear"] = linear_report(torch, lmbp, inputs, dev, reps=max(10, min(args.steps, 50)))
    if args.variants:
        print("[bench] k-bit family", file=sys.stderr, flush=True)
        out["variants"] = variants_report(torch, lmbp, inputs, dev)
    if args.blocks:
        print("[bench] MLP blocks", file=sys.stderr, flush=True)
        out["blocks"] = block_report(torch, dev, reps=max(5, min(args.steps, 20)))
    if run_cpu:
        print("[bench] timing the CPU oracle on a bounded sample", file=sys.stderr, flush=True)
        tensors = (w.norm_x(), w.norm_dz(), w.act_x(), w.act_dy())
        out["cpu_baseline"] = cpu_baseline(w, tensors)
        print(f"[bench] timing the CPU oracle on {procs} processes", file=sys.stderr, flush=True)
        out["cpu_baseline_all_cores"] = cpu_baseline_all_cores(w, tensors, pool, procs)
        pool.close()
        pool.join()
    print(json.dumps(out))


if __name__ == "__main__":
    main()
