"""Benchmark of the MOSAIC hot path on one MI355X.

Workload (prefill-shaped masked products at 70B-layer shapes): M = 2048
tokens; (K, N) in {(8192, 8192), (8192, 28672), (28672, 8192)}; uniform int8
plaintext in [-127, 127] (seed 2); depth-1 LWE mask of rank r = 1536 with
discrete Gaussian error sigma = 0.5, |e| <= 4. Init W runs once per shape,
outside the timed region.

One step = for every shape, one full call of the protocol: Init X (sample R,
then [U_a | K_c] in one ring product), the mask pass (A' = A + U_a + E_a, in
digit layout), the server product ([Y' | Q] = A' Bext^T) and unmasking
(digits of Q, then Y = Y' - K_c - Q L^T). ``value`` counts the plaintext
product's ring operations, 2 M K N per shape, over the step time (ring-TOPS).

Printed as one JSON line. ``roofline`` covers the server product kernel
(per launch: 10 int8 MACs = 20 int8 ops per ring MAC, M K (N + r) ring MACs),
timed with HIP events on the stream it runs on. ``cpu_baseline`` times the
CPU oracle on a bounded sample of the same workload.
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

INT8_PEAK_TOPS = 5000.0     # MI355X dense int8 MFMA, TOP/s
HBM_PEAK_GBS = 8000.0
# Streaming benchmarks cycle through at least this many bytes of distinct
# operands, three times the 256 MB last-level cache, so repeated calls read
# them from HBM as a sequence of different layers would.
ROTATE_BYTES = 3 * 256 * 2 ** 20


def _graph_ms(step, reps: int) -> float:
    """Mean time per call of ``step(i)`` for i < reps, captured once as a HIP
    graph and replayed (one warm-up replay, three timed): the device time of
    the calls without the host's per-launch cost."""
    import torch
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        for i in range(reps):
            step(i)
    graph.replay()
    torch.cuda.synchronize()
    e0, e1 = _events(2)
    e0.record()
    for _ in range(3):
        graph.replay()
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / (3 * reps)


def _settle(step, seconds: float = 0.025) -> None:
    """Untimed calls of step(i) for some tens of milliseconds before a
    stand-alone pass is timed: an ALU-heavy kernel started after other work
    ran up to 25% slower for its first ~10 ms (the mask pass with noise drawn
    in the pass measured 104-112 us over its first 30-60 launches and 87-89 us
    after), a transient of the chip's clock and power control rather than of
    the kernel."""
    import torch
    t0, i = time.perf_counter(), 0
    while time.perf_counter() - t0 < seconds:
        for _ in range(10):
            step(i)
            i += 1
        torch.cuda.synchronize()


def _warm_up(dev, seconds: float = 2.0) -> None:
    """Runs fp32 matrix products for a few seconds before stand-alone timings:
    the GPU raises its clocks only after some time under load, and ALU-heavy
    kernels timed in the first seconds of a process (the samplers, the mask
    pass with noise drawn in the pass) measured up to 20% slower."""
    import torch
    a = torch.randn(4096, 4096, device=dev)
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < seconds:
        for _ in range(20):
            b = a @ a
        torch.cuda.synchronize()
    del a, b


def _rotation(bytes_per_copy: int) -> int:
    """Number of distinct copies (at least 2) that together reach ROTATE_BYTES."""
    return max(2, -(-ROTATE_BYTES // max(1, bytes_per_copy)))


def _profiled_traffic():
    """HBM bytes per server launch from the committed byte-counter profile,
    or None if the kernel source changed since the counters were taken."""
    import hashlib
    rec = os.path.join(ROOT, "profiles", "server_gemm_traffic.txt")
    src = os.path.join(ROOT, "paper_2607_29221_amd", "csrc", "ring_gemm.hip")
    try:
        kv = dict(line.split(": ", 1) for line in open(rec).read().splitlines() if ": " in line)
        sha = hashlib.sha256(open(src, "rb").read()).hexdigest()
    except OSError:
        return None
    if kv.get("ring_gemm_source_sha256") != sha:
        return None
    return float(kv["server_traffic_bytes_per_launch"])


def _events(n):
    import torch
    return [torch.cuda.Event(enable_timing=True) for _ in range(n)]


def run_gpu(steps: int, warmup: int, extras: bool):
    import torch

    from paper_2607_29221_amd import mosaic as m
    from paper_2607_29221_amd import protocol as gp
    from synthetic_inputs import PARAMS_PAPER_D1, PREFILL_KN, PREFILL_M, PREFILL_SEED, int8_operands

    torch.cuda.set_device(0)
    dev = torch.device("cuda", 0)
    params = PARAMS_PAPER_D1
    M = PREFILL_M
    seed = 0x6D6F736169630000 | PREFILL_SEED
    shapes = []
    init_w_ms = []
    for idx, (K, N) in enumerate(PREFILL_KN):
        A, W = int8_operands(M, K, N, PREFILL_SEED)
        Ad = torch.from_numpy(A).to(dev)
        Wd = torch.from_numpy(W).to(dev)
        torch.cuda.synchronize()
        e0, e1 = _events(2)
        e0.record()
        w = gp.MaskedWeight(Wd, params, seed, weight_id=idx)
        e1.record()
        torch.cuda.synchronize()
        init_w_ms.append(round(e0.elapsed_time(e1), 3))
        del Wd
        shapes.append((K, N, Ad, w, gp.alloc_call(w, M, dev)))
    torch.cuda.synchronize()

    phases = ("init_x", "mask", "server", "unmask")
    ev = {(s, p): [] for s in range(len(shapes)) for p in phases}

    def step(call_id, record):
        for si, (K, N, Ad, w, buf) in enumerate(shapes):
            fns = (lambda: gp.init_x(w, M, call_id, buf), lambda: gp.mask(w, Ad, call_id, buf),
                   lambda: gp.server(w, M, buf), lambda: gp.unmask(w, M, buf))
            for p, fn in zip(phases, fns):
                if record:
                    e0, e1 = _events(2)
                    e0.record()
                    fn()
                    e1.record()
                    ev[(si, p)].append((e0, e1))
                else:
                    fn()

    for i in range(warmup):
        step(1000 + i, False)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(steps):
        step(i, True)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0

    ms = {k: sum(a.elapsed_time(b) for a, b in v) / len(v) for k, v in ev.items()}
    r = params.ranks[0]
    ring_ops = sum(2.0 * M * K * N for K, N, *_ in shapes)
    server_ops = [20.0 * M * K * (N + w.R) for K, N, _, w, _ in shapes]
    server_ms = [ms[(s, "server")] for s in range(len(shapes))]
    achieved = sum(server_ops) / (sum(server_ms) * 1e-3) / 1e12
    per_shape = []
    for s, (K, N, _, w, _) in enumerate(shapes):
        per_shape.append({
            "K": K, "N": N,
            "ms": {p: round(ms[(s, p)], 4) for p in phases},
            "server_ring_tops": round(2.0 * M * K * (N + w.R) / (ms[(s, "server")] * 1e-3) / 1e12, 2),
            "server_int8_tops": round(server_ops[s] / (ms[(s, "server")] * 1e-3) / 1e12, 1),
            "mask_gbs": round((M * K * 9) / (ms[(s, "mask")] * 1e-3) / 1e9, 1),
            "init_w_ms_once": init_w_ms[s],
        })
    out = {
        "ms_per_step": elapsed / steps * 1e3,
        "value": ring_ops / (elapsed / steps) / 1e12,
        "roofline": {"bound": "mfma", "achieved": round(achieved, 1), "peak": INT8_PEAK_TOPS, "unit": "TOP/s",
                     "frac": round(achieved / INT8_PEAK_TOPS, 4), "traffic": _profiled_traffic(),
                     "kernel": "ring_gemm_kernel<0> (server product [Y'|Q] = A' Bext^T)",
                     "launch_ms": [round(x, 4) for x in server_ms]},
        "per_shape": per_shape,
        "rank": r,
    }
    if extras:
        out["extras"] = run_extras(dev)
        out["extras"]["decode"] = run_decode(dev)
        out["extras"]["lpn_client_cost"] = run_lpn_client_cost(dev)
        out["extras"]["decoder_stack"] = run_decoder_stack(dev)
        out["extras"]["integrity_check"] = run_integrity(dev)
        out["extras"]["matvec_sweep"] = run_matvec_sweep(dev)
        out["extras"]["vendor_int8_gemm"] = run_vendor_int8(dev)
        out["extras"]["client_overhead"] = run_client_overhead(dev)
    return out


def run_extras(dev):
    """Stand-alone passes at their own shapes: the rotation of a 4096 x 8192
    fp32 activation (forward), the rotations of a 4096 x 28672 activation
    (H_28 (x) H_1024 and the block-diagonal forms), the mask pass at the largest prefill shape
    (with and without E_a), the three samplers writing digits at that shape,
    and the quantisation of a 4096 x 8192 fp32 activation. Buffers rotate
    through more than the 256 MB last-level cache."""
    import torch

    from paper_2607_29221_amd import mosaic as m
    from paper_2607_29221_amd.mosaic import Digits

    res = {}
    rows, n = 4096, 8192
    nbuf = 3
    xs = [torch.randn(rows, n, device=dev) for _ in range(nbuf)]
    ys = [torch.empty_like(xs[0]) for _ in range(nbuf)]
    signs = torch.empty(n, dtype=torch.int8, device=dev)
    m.mosaic_sample_signs(m.rng(3, 0x70, 0, 0), n, signs)
    _settle(lambda i: m.mosaic_hadamard_rotate(xs[i % nbuf], ys[i % nbuf], signs=signs))
    reps = 30
    e0, e1 = _events(2)
    e0.record()
    for i in range(reps):
        m.mosaic_hadamard_rotate(xs[i % nbuf], ys[i % nbuf], signs=signs)
    e1.record()
    torch.cuda.synchronize()
    t = e0.elapsed_time(e1) / reps
    res["fwht_4096x8192_us"] = round(t * 1e3, 2)
    res["fwht_gbs"] = round(rows * n * 8 / (t * 1e-3) / 1e9, 1)
    res["fwht_hbm_frac"] = round(res["fwht_gbs"] / HBM_PEAK_GBS, 3)
    del xs, ys

    # n = 28672 = 28 x 1024: H_28 (x) H_1024 against the block-diagonal
    # rotations I_7 (x) H_4096 and I_28 (x) H_1024 (time, and the median
    # max/RMS ratio of outlier rows after each)
    from synthetic_inputs import outlier_activations
    n28 = 28672
    xs = [torch.randn(rows, n28, device=dev) for _ in range(2)]
    xs[0][:64] = torch.from_numpy(outlier_activations(64, n28, seed=3)).to(dev)
    ys = [torch.empty_like(xs[0]) for _ in range(2)]
    s28 = torch.empty(n28, dtype=torch.int8, device=dev)
    m.mosaic_sample_signs(m.rng(3, 0x70, 1, 0), n28, s28)
    variants = (("kron28", lambda a, b: m.mosaic_hadamard28_rotate(a, b, signs=s28)),
                ("blockdiag4096", lambda a, b: m.mosaic_hadamard_rotate(a, b, block=4096, signs=s28)),
                ("blockdiag1024", lambda a, b: m.mosaic_hadamard_rotate(a, b, block=1024, signs=s28)))
    res["rotation_28672"] = []
    for name, fn in variants:
        _settle(lambda i: fn(xs[i % 2], ys[i % 2]))
        e0, e1 = _events(2)
        e0.record()
        for i in range(reps):
            fn(xs[i % 2], ys[i % 2])
        e1.record()
        torch.cuda.synchronize()
        t = e0.elapsed_time(e1) / reps
        fn(xs[0], ys[0])
        v = ys[0][:64].double()
        peak = (v.abs().amax(dim=1) / v.pow(2).mean(dim=1).sqrt()).median().item()
        res["rotation_28672"].append({"variant": name, "us": round(t * 1e3, 2),
                                      "gbs": round(rows * n28 * 8 / (t * 1e-3) / 1e9, 1),
                                      "outlier_max_over_rms_median": round(peak, 3)})
    del xs, ys

    M, K = 2048, 28672
    A = [torch.randint(-127, 128, (M, K), dtype=torch.int8, device=dev) for _ in range(nbuf)]
    U = [torch.randint(-2 ** 31, 2 ** 31 - 1, (M, K), dtype=torch.int32, device=dev) for _ in range(nbuf)]
    D = [Digits.empty(M, K, dev) for _ in range(nbuf)]
    noise = m.rng(2, 0x50, 0, m.DIST_DGAUSS, sigma=0.5, bound=4)
    for with_noise in (False, True):
        _settle(lambda i: m.mosaic_mask(A[i % nbuf], U[i % nbuf], noise if with_noise else None, M, K,
                                        out_dig=D[i % nbuf]))
        e0, e1 = _events(2)
        e0.record()
        for i in range(reps):
            m.mosaic_mask(A[i % nbuf], U[i % nbuf], noise if with_noise else None, M, K, out_dig=D[i % nbuf])
        e1.record()
        torch.cuda.synchronize()
        t = e0.elapsed_time(e1) / reps
        key = "mask_in_pass_noise" if with_noise else "mask"
        res[key + "_us"] = round(t * 1e3, 2)
        res[key + "_gbs"] = round(M * K * 9 / (t * 1e-3) / 1e9, 1)
        res[key + "_hbm_frac"] = round(res[key + "_gbs"] / HBM_PEAK_GBS, 3)
    del A, U

    # samplers straight to digits (4 B written per element)
    for name, r in (("uniform", m.rng(2, 0x20, 0, m.DIST_UNIFORM)),
                    ("dgauss", m.rng(2, 0x50, 0, m.DIST_DGAUSS, sigma=0.5, bound=4)),
                    ("sparse", m.rng(2, 0x40, 0, m.DIST_SPARSE, log2_inv_density=6))):
        _settle(lambda i: m.mosaic_sample(r, M, K, out_dig=D[i % nbuf]))
        e0, e1 = _events(2)
        e0.record()
        for i in range(reps):
            m.mosaic_sample(r, M, K, out_dig=D[i % nbuf])
        e1.record()
        torch.cuda.synchronize()
        t = e0.elapsed_time(e1) / reps
        res[f"sample_{name}_us"] = round(t * 1e3, 2)
        res[f"sample_{name}_gbs"] = round(M * K * 4 / (t * 1e-3) / 1e9, 1)
    del D

    # quantisation of rotated activations: 4096 x 8192 fp32 -> int32 codes
    rows, n = 4096, 8192
    xs = [torch.randn(rows, n, device=dev) for _ in range(nbuf)]
    qs = [torch.empty((rows, n), dtype=torch.int32, device=dev) for _ in range(nbuf)]
    sc = torch.empty(rows, dtype=torch.float32, device=dev)
    _settle(lambda i: m.mosaic_quantize_rows(xs[i % nbuf], 1997, q=qs[i % nbuf], scale=sc))
    e0, e1 = _events(2)
    e0.record()
    for i in range(reps):
        m.mosaic_quantize_rows(xs[i % nbuf], 1997, q=qs[i % nbuf], scale=sc)
    e1.record()
    torch.cuda.synchronize()
    t = e0.elapsed_time(e1) / reps
    res["quantize_4096x8192_us"] = round(t * 1e3, 2)
    res["quantize_gbs"] = round(rows * n * 8 / (t * 1e-3) / 1e9, 1)

    # Pi_Sec-Linear input pass at the decoder shapes: rotation + quantisation
    # + mask (E_a drawn) as three passes and fused (12 algorithmic bytes per
    # element: x and U in, digits out)
    res["secure_input"] = []
    for n, block, qx in ((8192, 8192, 1997), (28672, 4096, 567)):
        xs = [torch.randn(rows, n, device=dev) for _ in range(2)]
        U = torch.randint(-2 ** 31, 2 ** 31 - 1, (rows, n), dtype=torch.int32, device=dev)
        Dg = Digits.empty(rows, n, dev)
        y = torch.empty_like(xs[0])
        q = torch.empty((rows, n), dtype=torch.int32, device=dev)
        sg = torch.empty(n, dtype=torch.int8, device=dev)
        m.mosaic_sample_signs(m.rng(3, 0x70, 0, 0), n, sg)
        nz = m.rng(2, 0x50, 0, m.DIST_DGAUSS, sigma=0.5, bound=4)

        def separate(i):
            m.mosaic_hadamard_rotate(xs[i % 2], y, block=block, signs=sg)
            m.mosaic_quantize_rows(y, qx, q=q, scale=sc)
            m.mosaic_mask(q, U, nz, rows, n, out_dig=Dg)

        def fused(i):
            m.mosaic_rotate_quantize_mask(xs[i % 2], qx, Dg, block=block, signs=sg, u=U, noise=nz, scale=sc)

        ts = []
        for fn in (separate, fused):
            _settle(fn)
            e0, e1 = _events(2)
            e0.record()
            for i in range(10):
                fn(i)
            e1.record()
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1) / 10)
        res["secure_input"].append({"rows": rows, "n": n, "block": block, "separate_us": round(ts[0] * 1e3, 1),
                                    "fused_us": round(ts[1] * 1e3, 1),
                                    "fused_gbs": round(rows * n * 12 / (ts[1] * 1e-3) / 1e9, 1)})
        del xs, U, Dg, y, q
    return res


def run_vendor_int8(dev):
    """Context for the MFMA figure: the vendor int8 GEMM (torch._int_mm, which
    calls hipBLASLt) on uniformly random int8 operands with the int8 work of
    the largest server launch as one plain GEMM (M = 2048, K = 4 x 8192 digit
    columns, N = 30208, B column-major), in int8 TOP/s. Not part of the
    product path."""
    import torch

    M, K, N = 2048, 4 * 8192, 30208
    g = torch.Generator(device=dev)
    g.manual_seed(7)
    a = torch.randint(-128, 128, (M, K), dtype=torch.int8, device=dev, generator=g)
    b = torch.randint(-128, 128, (N, K), dtype=torch.int8, device=dev, generator=g).t()
    for _ in range(2):
        torch._int_mm(a, b)
    reps = 10
    e0, e1 = _events(2)
    e0.record()
    for _ in range(reps):
        torch._int_mm(a, b)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    return {"M": M, "K": K, "N": N, "ms": round(ms, 3), "int8_tops": round(2.0 * M * K * N / (ms * 1e-3) / 1e12, 1),
            "operands": "uniform int8"}


def run_integrity(dev):
    """Cost of the integrity check (Freivalds' test, 32 check vectors) per
    prefill call: Init W with the check key (once, untimed), one honest call,
    then the check timed with HIP events (mean over 10) and compared with the
    call's server product. The check is timed twice: launched eagerly from
    Python (its six launches then wait on the interpreter) and replayed as a
    captured HIP graph, the form a serving loop would run it in; the graph's
    last replay must accept the call too."""
    import torch

    from paper_2607_29221_amd import protocol as gp
    from synthetic_inputs import PARAMS_PAPER_D1, PREFILL_KN, PREFILL_M, PREFILL_SEED, int8_operands

    M, t, reps = PREFILL_M, 32, 10
    out = []
    for idx, (K, N) in enumerate(PREFILL_KN):
        A, W = int8_operands(M, K, N, PREFILL_SEED)
        w = gp.MaskedWeight(torch.from_numpy(W).to(dev), PARAMS_PAPER_D1, 0x6D6F736169630000 | PREFILL_SEED,
                            weight_id=idx, check_vectors=t)
        buf = gp.run_call(w, torch.from_numpy(A).to(dev), call_id=1)
        ok = int(gp.verify(w, M, buf).item()) == 0
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            count = gp.verify(w, M, buf)
        torch.cuda.synchronize()
        e = _events(4)
        e[0].record()
        for _ in range(reps):
            gp.server(w, M, buf)
        e[1].record()
        for _ in range(reps):
            gp.verify(w, M, buf)
        e[2].record()
        for _ in range(reps):
            graph.replay()
        e[3].record()
        torch.cuda.synchronize()
        ok = ok and int(count.item()) == 0
        sv, ck, cg = (e[0].elapsed_time(e[1]) / reps, e[1].elapsed_time(e[2]) / reps,
                      e[2].elapsed_time(e[3]) / reps)
        out.append({"K": K, "N": N, "vectors": t, "honest_call_accepted": ok, "check_ms": round(cg, 4),
                    "check_ms_eager": round(ck, 4), "server_ms": round(sv, 4),
                    "check_over_server": round(cg / sv, 4)})
        del graph, count
        del w, buf
    return out


def run_matvec_sweep(dev):
    """One secure matrix-vector product (one token, W' n x n) for
    n in {4096, 8192, 16384, 36864}, depth-1 mask of rank 1536 with sigma =
    0.5: the server product ([Y' | Q]), the client's online steps (mask and
    unmask) and the input-independent Init X, HIP-event means over 20 calls
    that cycle through distinct masked weights (together beyond three times
    the last-level cache). The paper reports the same split for its own
    implementation (context only: other hardware and design)."""
    import torch

    from paper_2607_29221_amd import protocol as gp
    from synthetic_inputs import MATVEC_N, MATVEC_SEED, PARAMS_PAPER_D1, int8_matrix_device

    out, reps = [], 20
    for n in MATVEC_N:
        W = int8_matrix_device(n, n, MATVEC_SEED, dev)
        A = int8_matrix_device(1, n, MATVEC_SEED + 1, dev)
        Kp = 64 * ((n + 63) // 64)
        nrot = _rotation(4 * Kp * (n + sum(PARAMS_PAPER_D1.ranks)))
        wl = [gp.MaskedWeight(W, PARAMS_PAPER_D1, (0x6D6F736169630000 | MATVEC_SEED) + 0x10000 * j, weight_id=0)
              for j in range(nrot)]
        del W
        bl = [gp.alloc_call(w, 1, dev) for w in wl]
        for j in range(nrot):
            gp.run_call(wl[j], A, 100 + j, bl[j])
        torch.cuda.synchronize()
        e = _events(5)
        e[0].record()
        for i in range(reps):
            gp.init_x(wl[i % nrot], 1, 200 + i, bl[i % nrot])
        e[1].record()
        for i in range(reps):
            gp.mask(wl[i % nrot], A, 200 + i, bl[i % nrot])
        e[2].record()
        for i in range(reps):
            gp.server(wl[i % nrot], 1, bl[i % nrot])
        e[3].record()
        for i in range(reps):
            gp.unmask(wl[i % nrot], 1, bl[i % nrot])
        e[4].record()
        torch.cuda.synchronize()
        w = wl[0]
        t = [e[k].elapsed_time(e[k + 1]) / reps for k in range(4)]
        Kp = 64 * ((n + 63) // 64)
        byts = 4 * Kp * (1 + w.n_out) + 4 * w.n_out
        out.append({"n": n, "server_ms": round(t[2], 4), "server_gbs": round(byts / (t[2] * 1e-3) / 1e9, 1),
                    "client_online_ms": round(t[1] + t[3], 4), "init_x_ms": round(t[0], 4),
                    "total_ms": round(sum(t), 4), "weights_rotated": nrot})
        del w, wl, bl
    return out


def run_client_overhead(dev):
    """The paper's outsourcing-efficiency sweep on one GPU: for eight model
    shapes (attention output projection, MLP up, MLP down), the client's
    runtime per one-token call -- Init X batched over 512 calls and divided
    by 512, plus the online mask and unmask -- against computing W x
    locally on the same GPU, as a bf16 matrix-vector product (torch.mv) and
    as the same Z_2^32 product on plaintext digits (the local baseline is a
    reading: the paper does not state its arithmetic). Depth-1 mask of rank
    1536, sigma 0.5; HIP-event means over 20 calls. The online steps and
    both local products are also timed as replayed HIP graphs of 20 calls:
    eager, the smallest shapes measure the host's launch rate (about 11 us
    for the mask and 20 us for the unmask's two calls) rather than the GPU."""
    import torch

    from paper_2607_29221_amd import mosaic as m
    from paper_2607_29221_amd import protocol as gp
    from paper_2607_29221_amd.mosaic import Digits
    from synthetic_inputs import (OVERHEAD_BATCH, OVERHEAD_MODELS, OVERHEAD_SEED, PARAMS_PAPER_D1,
                                  int8_matrix_device)

    out, reps = [], 20
    for mi, (name, d, attn_in, f) in enumerate(OVERHEAD_MODELS):
        for kind, K, N in (("attn proj", attn_in, d), ("MLP up", d, f), ("MLP down", f, d)):
            W = int8_matrix_device(N, K, OVERHEAD_SEED + 3 * mi, dev)
            x = int8_matrix_device(1, K, OVERHEAD_SEED + 3 * mi + 1, dev)
            w = gp.MaskedWeight(W, PARAMS_PAPER_D1, 0x6D6F736169630000 | (OVERHEAD_SEED + mi), weight_id=mi)
            Wb = W.to(torch.bfloat16)
            xb = x[0].to(torch.bfloat16)
            Wd, xd = Digits.empty(N, K, dev), Digits.empty(1, K, dev)
            m.mosaic_mask(W, None, None, N, K, out_dig=Wd)
            m.mosaic_mask(x, None, None, 1, K, out_dig=xd)
            yr = torch.empty((1, N), dtype=torch.int32, device=dev)
            del W
            bufb = gp.alloc_call(w, OVERHEAD_BATCH, dev)
            buf1 = gp.alloc_call(w, 1, dev)
            gp.init_x(w, 1, 1, buf1)
            gp.init_x(w, OVERHEAD_BATCH, 2, bufb)
            _settle(lambda i: (gp.mask(w, x, 3, buf1), gp.unmask(w, 1, buf1), torch.mv(Wb, xb),
                               m.mosaic_masked_matmul(xd, Wd, 1, N, K, yr)))
            e = _events(6)
            e[0].record()
            for i in range(4):
                gp.init_x(w, OVERHEAD_BATCH, 10 + i, bufb)
            e[1].record()
            for i in range(reps):
                gp.mask(w, x, 20 + i, buf1)
            e[2].record()
            for i in range(reps):
                gp.unmask(w, 1, buf1)
            e[3].record()
            for i in range(reps):
                torch.mv(Wb, xb)
            e[4].record()
            for i in range(reps):
                m.mosaic_masked_matmul(xd, Wd, 1, N, K, yr)
            e[5].record()
            torch.cuda.synchronize()
            init_x = e[0].elapsed_time(e[1]) / 4 / OVERHEAD_BATCH
            online = e[1].elapsed_time(e[2]) / reps + e[2].elapsed_time(e[3]) / reps
            local = e[3].elapsed_time(e[4]) / reps
            local_ring = e[4].elapsed_time(e[5]) / reps
            online_g = _graph_ms(lambda i: (gp.mask(w, x, 40 + i, buf1), gp.unmask(w, 1, buf1)), reps)
            local_g = _graph_ms(lambda i: torch.mv(Wb, xb), reps)
            local_ring_g = _graph_ms(lambda i: m.mosaic_masked_matmul(xd, Wd, 1, N, K, yr), reps)
            out.append({"model": name, "matrix": kind, "K": K, "N": N, "init_x_ms_per_call": round(init_x, 5),
                        "online_ms": round(online, 5), "local_bf16_mv_ms": round(local, 5),
                        "local_ring_mv_ms": round(local_ring, 5),
                        "client_over_local": round((init_x + online) / local, 4),
                        "client_over_local_ring": round((init_x + online) / local_ring, 4),
                        "online_ms_graph": round(online_g, 5), "local_bf16_mv_ms_graph": round(local_g, 5),
                        "local_ring_mv_ms_graph": round(local_ring_g, 5),
                        "client_over_local_graph": round((init_x + online_g) / local_g, 4),
                        "client_over_local_ring_graph": round((init_x + online_g) / local_ring_g, 4)})
            del w, Wb, xb, bufb, buf1, Wd, xd, yr
    return out


def run_decode(dev):
    """Decode-shaped calls (M in {1, 8, 64} tokens; (K, N) in {4096^2,
    4096 x 14336, 14336 x 4096}; depth-2 mask of ranks (1536, 1024) with
    density-1/64 sparse LPN level, and the whole call also at depth 3 with
    ranks (1536, 1024, 652), sparse mode). Per shape and M: the server product
    ([Y' | Q], N + 2560 output columns) and the whole call (Init X, mask,
    server, unmask), HIP-event means over 20 calls; GB/s counts the server
    product's operand and output bytes once; ring-TOPS counts the plaintext
    product's 2 M K N ring ops over the server time. The server loop and the three
    whole-call loops are also timed as replayed HIP graphs of 20 calls (the
    device time without the host's per-launch cost). Calls cycle through distinct
    masked weights (independent masks of the same W) whose server matrices
    together exceed the last-level cache three times."""
    import torch

    from paper_2607_29221_amd import protocol as gp
    from synthetic_inputs import (DECODE_KN, DECODE_M, DECODE_SEED, PARAMS_DECODE_D2_NOISY, PARAMS_PAPER_D2_SPARSE,
                                  PARAMS_PAPER_D3_SPARSE, PARAMS_PAPER_D3_T80, int8_operands)

    res = []
    reps = 20
    for idx, (K, N) in enumerate(DECODE_KN):
        A, W = int8_operands(max(DECODE_M), K, N, DECODE_SEED)
        Wd = torch.from_numpy(W).to(dev)
        Kp = 64 * ((K + 63) // 64)
        nrot = _rotation(4 * Kp * (N + sum(PARAMS_PAPER_D2_SPARSE.ranks)))

        def weights(params, sparse):
            return [gp.MaskedWeight(Wd, params, 0xDEC0DE00 + 0x100 * j + idx, weight_id=idx, sparse_lpn=sparse)
                    for j in range(nrot)]

        wl = weights(PARAMS_PAPER_D2_SPARSE, False)        # dense LPN form only (the server loop)
        wal = weights(PARAMS_PAPER_D2_SPARSE, None)        # both forms, chosen per call by token count
        wsl = weights(PARAMS_PAPER_D2_SPARSE, True)
        w3l = weights(PARAMS_PAPER_D3_SPARSE, True)
        wnl = weights(PARAMS_DECODE_D2_NOISY, None)         # the same with sigma = 0.5 LWE error
        wtl = weights(PARAMS_PAPER_D3_T80, None)            # Example 4.1 in full (t = 80)
        w = wl[0]
        for M in DECODE_M:
            Ad = torch.from_numpy(A[:M].copy()).to(dev)
            bl = [gp.alloc_call(x, M, dev) for x in wl]
            bal = [gp.alloc_call(x, M, dev) for x in wal]
            bsl = [gp.alloc_call(x, M, dev) for x in wsl]
            b3l = [gp.alloc_call(x, M, dev) for x in w3l]
            bnl = [gp.alloc_call(x, M, dev) for x in wnl]
            btl = [gp.alloc_call(x, M, dev) for x in wtl]
            lists = ((wl, bl), (wal, bal), (wsl, bsl), (w3l, b3l), (wnl, bnl), (wtl, btl))
            for ws_, bs_ in lists:
                for j in range(nrot):
                    gp.run_call(ws_[j], Ad, 10_000 + j, bs_[j])
            torch.cuda.synchronize()
            extra_graph = {}
            for key, (ws_, bs_) in (("call_us_auto_lpn_graph", lists[1]), ("call_us_d2_noisy_graph", lists[4]),
                                    ("call_us_d3_t80_graph", lists[5])):
                extra_graph[key] = round(_graph_ms(lambda i: gp.run_call(ws_[i % nrot], Ad, 50_000 + i,
                                                                         bs_[i % nrot]), reps) * 1e3, 2)
            # the loops once more as replayed graphs: device time without the
            # host's per-launch cost (which bounds the eager whole-call loops)
            server_graph_ms = _graph_ms(lambda i: gp.server(wl[i % nrot], M, bl[i % nrot]), reps)
            call_graph_ms = _graph_ms(lambda i: gp.run_call(wl[i % nrot], Ad, 40_000 + i, bl[i % nrot]), reps)
            call_sparse_graph_ms = _graph_ms(lambda i: gp.run_call(wsl[i % nrot], Ad, 40_000 + i, bsl[i % nrot]),
                                             reps)
            call_d3_graph_ms = _graph_ms(lambda i: gp.run_call(w3l[i % nrot], Ad, 40_000 + i, b3l[i % nrot]), reps)
            e = _events(5)
            e[0].record()
            for i in range(reps):
                gp.server(wl[i % nrot], M, bl[i % nrot])
            e[1].record()
            for i in range(reps):
                gp.run_call(wl[i % nrot], Ad, 20_000 + i, bl[i % nrot])
            e[2].record()
            for i in range(reps):
                gp.run_call(wsl[i % nrot], Ad, 20_000 + i, bsl[i % nrot])
            e[3].record()
            for i in range(reps):
                gp.run_call(w3l[i % nrot], Ad, 20_000 + i, b3l[i % nrot])
            e[4].record()
            # phases of the sparse-mode call: Init X is input independent (it
            # can run ahead of the token); mask, server and unmask are online
            ph = _events(4)
            ph[0].record()
            for i in range(reps):
                gp.init_x(wsl[i % nrot], M, 30_000 + i, bsl[i % nrot])
            ph[1].record()
            for i in range(reps):
                ws_, bs_ = wsl[i % nrot], bsl[i % nrot]
                gp.mask(ws_, Ad, 30_000 + i, bs_)
                gp.server(ws_, M, bs_)
                gp.unmask(ws_, M, bs_)
            ph[2].record()
            torch.cuda.synchronize()
            server_ms = e[0].elapsed_time(e[1]) / reps
            call_ms = e[1].elapsed_time(e[2]) / reps
            call_sparse_ms = e[2].elapsed_time(e[3]) / reps
            call_d3_ms = e[3].elapsed_time(e[4]) / reps
            init_x_ms = ph[0].elapsed_time(ph[1]) / reps
            online_ms = ph[1].elapsed_time(ph[2]) / reps
            byts = 4 * Kp * (M + w.n_out) + 4 * M * w.n_out
            res.append({"K": K, "N": N, "M": M, "server_us": round(server_ms * 1e3, 2),
                        "server_gbs": round(byts / (server_ms * 1e-3) / 1e9, 1),
                        "server_hbm_frac": round(byts / (server_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 3),
                        "server_ring_tops": round(2.0 * M * K * N / (server_ms * 1e-3) / 1e12, 3),
                        "server_us_graph": round(server_graph_ms * 1e3, 2),
                        "server_hbm_frac_graph": round(byts / (server_graph_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 3),
                        "call_us": round(call_ms * 1e3, 2),
                        "call_us_sparse_lpn": round(call_sparse_ms * 1e3, 2),
                        "call_us_d3_sparse_lpn": round(call_d3_ms * 1e3, 2),
                        "call_us_graph": round(call_graph_ms * 1e3, 2),
                        "call_us_sparse_lpn_graph": round(call_sparse_graph_ms * 1e3, 2),
                        "call_us_d3_sparse_lpn_graph": round(call_d3_graph_ms * 1e3, 2),
                        "init_x_us_sparse_lpn": round(init_x_ms * 1e3, 2),
                        "online_us_sparse_lpn": round(online_ms * 1e3, 2), "weights_rotated": nrot,
                        **extra_graph})
            del bl, bal, bsl, b3l, bnl, btl
        del w, wl, wal, wsl, w3l, wnl, wtl
    return res


def run_lpn_client_cost(dev):
    """The client's share of a decode call for the three mask depths of
    Example 4.1 -- LWE only (r = 1536), + LPN-1 (r_2 = 1024, t_2 = 80),
    + LPN-2 (r_3 = 652, t_3 = 80), all with sigma = 0.5 -- at (K, N) = (4096,
    14336) for 1, 8 and 64 tokens: Init X, mask and unmask (no server
    product), sparse LPN form, device time of 20 calls replayed as a HIP
    graph, calls cycling through
    distinct masked weights. Table "lpn-tradeoff" puts the client's
    multiplications per (m + n) l at r_1 = 1536, r_2 + t_2 = 1104 and
    r_3 + t_2 + t_3 = 812 (ratios 1, 0.719, 0.529)."""
    import torch

    from paper_2607_29221_amd import protocol as gp
    from synthetic_inputs import (DECODE_SEED, PARAMS_PAPER_D1, PARAMS_PAPER_D2_T80, PARAMS_PAPER_D3_T80,
                                  int8_operands)

    K, N, reps = 4096, 14336, 20
    A, W = int8_operands(64, K, N, DECODE_SEED)
    Wd = torch.from_numpy(W).to(dev)
    cfgs = (("lwe_only", PARAMS_PAPER_D1), ("lpn1_t80", PARAMS_PAPER_D2_T80), ("lpn2_t80", PARAMS_PAPER_D3_T80))
    table = {"lwe_only": 1536, "lpn1_t80": 1104, "lpn2_t80": 812}
    rows = []
    for M in (1, 8, 64):
        Ad = torch.from_numpy(A[:M].copy()).to(dev)
        entry = {"M": M}
        for name, params in cfgs:
            nrot = _rotation(4 * K * (N + sum(params.ranks)))
            wl = [gp.MaskedWeight(Wd, params, 0xC11E0000 + 0x100 * j, weight_id=1, sparse_lpn=True)
                  for j in range(nrot)]
            bl = [gp.alloc_call(x, M, dev) for x in wl]
            for j in range(nrot):
                gp.run_call(wl[j], Ad, 60_000 + j, bl[j])

            def client(i):
                gp.init_x(wl[i % nrot], M, 70_000 + i, bl[i % nrot])
                gp.mask(wl[i % nrot], Ad, 70_000 + i, bl[i % nrot])
                gp.unmask(wl[i % nrot], M, bl[i % nrot])
            entry[name + "_us"] = round(_graph_ms(client, reps) * 1e3, 2)
            del wl, bl
        base = entry["lwe_only_us"]
        entry["ratio"] = [round(entry[n + "_us"] / base, 3) for n, _ in cfgs]
        rows.append(entry)
    return {"K": K, "N": N, "rows": rows,
            "table_per_row": [table[n] for n, _ in cfgs],
            "table_ratio": [round(table[n] / 1536, 3) for n, _ in cfgs],
            "summary": {"table_ratio": [round(table[n] / 1536, 3) for n, _ in cfgs],
                        **{f"M{r['M']}_ratio": r["ratio"] for r in rows}}}


def run_decoder_stack(dev):
    """Secure forward of the synthetic 70B-style stack (hidden 8192, 64/8
    heads, FFN 28672, 4 layers, 4096 tokens; int8 weights, depth-1 rank-1536
    mask, sigma = 0.5) against its float32 plaintext forward: per-layer
    relative l2 error and cosine similarity, forward times (Init W of the
    16 weight matrices is outside the timed region), and the time split of
    the secure forward by phase (Init X, input pass, server product, unmask
    with dequantisation, and everything else)."""
    import torch

    from paper_2607_29221_amd import decoder as dec
    from synthetic_inputs import DECODER, DECODER_LINEARS, DECODER_SEED, PARAMS_PAPER_D1, decoder_input, \
        decoder_weight

    prev = torch.backends.cuda.matmul.allow_tf32
    torch.backends.cuda.matmul.allow_tf32 = False
    try:
        weights = [{n: decoder_weight(l, n, dev) for n in DECODER_LINEARS} for l in range(DECODER["layers"])]
        x = decoder_input(dev)
        sd = dec.SecureDecoder(weights, DECODER, PARAMS_PAPER_D1, 0x6D6F736169630000 | DECODER_SEED)
        sd.forward(x)                                   # warm-up
        torch.cuda.synchronize()
        e = _events(3)
        e[0].record()
        got = sd.forward(x)
        e[1].record()
        ref = dec.plaintext_forward(x, weights, DECODER)
        e[2].record()
        torch.cuda.synchronize()
        errs = [dec.error_metrics(g, r) for g, r in zip(got, ref)]
        # time split of a further forward: the linear layers' phases from
        # events at their boundaries, the rest (norms, attention, SwiGLU,
        # residuals, buffer allocation) as the remainder
        marks = []
        for layer in sd.layers:
            for lin in layer.values():
                lin.phase_events = marks
        f0, f1 = _events(2)
        f0.record()
        sd.forward(x)
        f1.record()
        torch.cuda.synchronize()
        split = {"init_x": 0.0, "input": 0.0, "server": 0.0, "unmask": 0.0}
        for (_, a), (name, b) in zip(marks, marks[1:]):
            if name in split:
                split[name] += a.elapsed_time(b)
        total = f0.elapsed_time(f1)
        split = {k: round(v, 2) for k, v in split.items()}
        split["non_linear_and_other"] = round(total - sum(split.values()), 2)
        split["total"] = round(total, 2)
    finally:
        torch.backends.cuda.matmul.allow_tf32 = prev
    tokens = DECODER["batch"] * DECODER["seq"]
    macs = sum(a * b for a, b in (_shape(n) for n in DECODER_LINEARS)) * tokens * DECODER["layers"]
    secure_ms = e[0].elapsed_time(e[1])
    return {"layers": DECODER["layers"], "tokens": tokens,
            "secure_forward_ms": round(secure_ms, 2),
            "plaintext_fp32_forward_ms": round(e[1].elapsed_time(e[2]), 2),
            "secure_linear_ring_tops": round(2.0 * macs / (secure_ms * 1e-3) / 1e12, 2),
            "time_split_ms": split,
            "per_layer": [{"rel_l2": round(v["rel_l2"], 5), "cosine": round(v["cosine"], 6)} for v in errs]}


def _shape(name):
    from synthetic_inputs import decoder_linear_shape
    return decoder_linear_shape(name)


def _mfma_probe_tops(mode):
    """int8 TOP/s of the register-only MFMA probe (mosaic_probe_mfma_i8;
    mode 0 zero, 1 constant, 2 uniformly random operands): 0.5 s of the same
    load, then about 0.3 s timed."""
    import torch

    from paper_2607_29221_amd import mosaic as m

    out = torch.zeros(1, dtype=torch.int32, device=torch.device("cuda", 0))
    iters = 8192
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < 0.5:
        m.mosaic_probe_mfma_i8(mode, iters, out)
        torch.cuda.synchronize()
    e0, e1 = _events(2)
    e0.record()
    ops, n = 0, 0
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < 0.3 or n < 3:
        ops += m.mosaic_probe_mfma_i8(mode, iters, out)
        n += 1
    e1.record()
    torch.cuda.synchronize()
    return round(ops / (e0.elapsed_time(e1) * 1e-3) / 1e12, 1)


def run_mfma_ceiling():
    """The ceiling the server product runs under: the register-only MFMA
    probe (v_mfma_i32_32x32x32_i8, operands in registers, no memory traffic)
    on zero, constant and uniformly random operands, each timed for about
    0.3 s after 0.5 s of the same load; then the server product itself at
    the 8192 x 30208 x 8192 prefill server shape on uniform and on all-zero
    digits. int8 TOP/s."""
    import torch

    from paper_2607_29221_amd import mosaic as m
    from paper_2607_29221_amd.mosaic import Digits

    dev = torch.device("cuda", 0)
    res = {}
    for mode, name in ((0, "zero"), (1, "constant"), (2, "random")):
        res[f"register_{name}_tops"] = _mfma_probe_tops(mode)
    M, K, Np = 2048, 8192, 30208
    A, B = Digits.empty(M, K, dev), Digits.empty(Np, K, dev)
    C = torch.empty((M, Np), dtype=torch.int32, device=dev)
    for name in ("uniform", "zero"):
        if name == "uniform":
            m.mosaic_sample(m.rng(1, 1, 0, m.DIST_UNIFORM), M, K, out_dig=A)
            m.mosaic_sample(m.rng(1, 2, 0, m.DIST_UNIFORM), Np, K, out_dig=B)
        else:
            A.buf.zero_()
            B.buf.zero_()
        for _ in range(20):
            m.mosaic_masked_matmul(A, B, M, Np, K, C)
        e0, e1 = _events(2)
        e0.record()
        for _ in range(10):
            m.mosaic_masked_matmul(A, B, M, Np, K, C)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / 10
        res[f"server_{name}_digits_tops"] = round(20.0 * M * K * Np / ms / 1e9, 1)
    res["server_over_register_random"] = round(res["server_uniform_digits_tops"] / res["register_random_tops"], 3)
    res["server_over_register_zero"] = round(res["server_zero_digits_tops"] / res["register_zero_tops"], 3)
    return res


def run_product_only():
    """The server product alone (mosaic_masked_matmul) at the prefill server
    shapes, M = 2048, (N + 1536, K), on uniformly sampled digit operands:
    the kernel the roofline covers, without the rest of the call (used for
    counter runs)."""
    import torch

    from paper_2607_29221_amd import mosaic as m
    from paper_2607_29221_amd.mosaic import Digits
    from synthetic_inputs import PREFILL_KN, PREFILL_M

    dev = torch.device("cuda", 0)
    M, out = PREFILL_M, []
    for K, N in PREFILL_KN:
        Np = N + 1536
        A, B = Digits.empty(M, K, dev), Digits.empty(Np, K, dev)
        m.mosaic_sample(m.rng(1, 1, 0, m.DIST_UNIFORM), M, K, out_dig=A)
        m.mosaic_sample(m.rng(1, 2, 0, m.DIST_UNIFORM), Np, K, out_dig=B)
        C = torch.empty((M, Np), dtype=torch.int32, device=dev)
        for _ in range(2):
            m.mosaic_masked_matmul(A, B, M, Np, K, C)
        e0, e1 = _events(2)
        e0.record()
        for _ in range(5):
            m.mosaic_masked_matmul(A, B, M, Np, K, C)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / 5
        out.append({"K": K, "N_plus_r": Np, "ms": round(ms, 4), "int8_tops": round(20.0 * M * K * Np / ms / 1e9, 1)})
        del A, B, C
    return out


def _cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def run_cpu_baseline():
    """The oracle on the host cores of the machine that runs the benchmark
    (its plain C leg, OpenMP over output rows; ``cores`` is the thread count
    OpenMP uses), on bounded samples:

    * the whole prefill call at the first shape, M = 2048, (K, N) = (8192,
      8192), rank 1536: Init X, mask, server product with Q, unmasking (Init
      W prepared outside the timed region, as on the GPU). ``value`` counts
      every ring multiply-accumulate the call does (U_a, K_c, Y', Q and the
      unmask product) as two ring operations, so the counted operations
      equal the work done; ``plaintext_ring_tops`` counts only the 2 M K N of
      the plaintext product (the GPU line's definition);
    * the rotation of 4096 x 8192 float64 rows, forward and inverse, on all
      threads, and of 512 rows on one thread;
    * the single masked matmul (64 x 512 x 512, depth 1, rank 128) on one
      thread."""
    import os as _os

    import numpy as np

    from oracle import _cring
    from oracle import protocol as op
    from oracle.sampling import sample_signs
    from synthetic_inputs import (PARAMS_D1_SMALL_R128, PARAMS_PAPER_D1, PREFILL_SEED, int8_operands,
                                  outlier_activations)

    threads = _cring.threads()
    K, N, Ms, Ns, r = 8192, 8192, 2048, 8192, PARAMS_PAPER_D1.ranks[0]
    A, W = int8_operands(2048, K, N, PREFILL_SEED)
    seed = 0x6D6F736169630000 | PREFILL_SEED
    t0 = time.perf_counter()
    w = op.init_w_depth1_c(W[:Ns], PARAMS_PAPER_D1, seed, 0)
    init_w_s = time.perf_counter() - t0
    t0 = time.perf_counter()
    res = op.call_depth1_c(w, A[:Ms], PARAMS_PAPER_D1, seed, 1)
    dt = time.perf_counter() - t0
    assert res["Y"].shape == (Ms, Ns)
    macs = Ms * (r * K + r * Ns + K * (Ns + r) + r * Ns)

    x = outlier_activations(4096, 8192, 3)
    d = sample_signs(8192, 3, 0)
    t0 = time.perf_counter()
    y = _cring.rotate_rows(x, d)
    xb = _cring.rotate_rows(y, d, inverse=True)
    rot_s = time.perf_counter() - t0
    assert np.max(np.abs(xb - x)) < 1e-9 * np.max(np.abs(x))

    prev = _os.environ.get("OMP_NUM_THREADS")
    one = {}
    try:
        import ctypes
        ctypes.CDLL("libgomp.so.1").omp_set_num_threads(1)
        t0 = time.perf_counter()
        y1 = _cring.rotate_rows(x[:512], d)
        _cring.rotate_rows(y1, d, inverse=True)
        one["rotation_512x8192_fwd_inv_s"] = round(time.perf_counter() - t0, 3)
        A1, W1 = int8_operands(64, 512, 512, 0)
        t0 = time.perf_counter()
        w1 = op.init_w_depth1_c(W1, PARAMS_D1_SMALL_R128, 1234, 0)
        op.call_depth1_c(w1, A1, PARAMS_D1_SMALL_R128, 1234, 0)
        one["single_matmul_64x512x512_s"] = round(time.perf_counter() - t0, 4)
        one["threads"] = _cring.threads()
    finally:
        ctypes.CDLL("libgomp.so.1").omp_set_num_threads(threads)
        if prev is not None:
            _os.environ["OMP_NUM_THREADS"] = prev
    return {"value": round(2.0 * macs / dt / 1e12, 5), "unit": "ring-TOPS", "cores": threads,
            "kind": "oracle", "seconds": round(dt, 2),
            "plaintext_ring_tops": round(2.0 * Ms * K * Ns / dt / 1e12, 5),
            "sample": f"the whole call at M = {Ms}, (K, N) = ({K}, {Ns}), rank {r}: Init X, mask, "
                      f"server with Q, unmask ({macs:.3g} ring MACs, all counted); plain C ring loops "
                      f"(gcc -O2, OpenMP over rows); Init W {init_w_s:.1f} s untimed",
                      "host_cpus": _os.cpu_count(), "cpu_model": _cpu_model(),
            "rotation_4096x8192_fwd_inv_s": round(rot_s, 3),
            "rotation_gbs": round(2 * 4096 * 8192 * 16 / rot_s / 1e9, 2),
            "one_thread": one}


def _compact(ex):
    """The figures of the extras that the roofline targets name, as short
    top-level keys of the JSON line (the full extras go to a side file)."""
    out = {}
    p = {}
    p["fwht_4096x8192"] = {"us": ex["fwht_4096x8192_us"], "gbs": ex["fwht_gbs"], "hbm_frac": ex["fwht_hbm_frac"]}
    for key, name in (("mask", "mask_2048x28672"), ("mask_in_pass_noise", "mask_noise_2048x28672")):
        p[name] = {"us": ex[key + "_us"], "gbs": ex[key + "_gbs"], "hbm_frac": ex[key + "_hbm_frac"]}
    for si in ex.get("secure_input", []):
        p[f"fused_input_{si['rows']}x{si['n']}"] = {"us": si["fused_us"], "gbs": si["fused_gbs"],
                                                      "hbm_frac": round(si["fused_gbs"] / HBM_PEAK_GBS, 3)}
    out["passes"] = p
    if "decode" in ex:
        # device time of the server loop replayed as a graph (clear and
        # product; the eager loop's figure also holds the host's launch gaps)
        out["decode"] = [{"K": d["K"], "N": d["N"], "M": d["M"], "server_hbm_frac_graph": d["server_hbm_frac_graph"],
                          "call_us_graph": d["call_us_auto_lpn_graph"]} for d in ex["decode"]]
    if "lpn_client_cost" in ex:
        out["lpn_client_cost"] = ex["lpn_client_cost"]["summary"]
    if "integrity_check" in ex:
        out["integrity_check_over_server"] = [c["check_over_server"] for c in ex["integrity_check"]]
    if "decoder_stack" in ex:
        ds = ex["decoder_stack"]
        out["decoder_stack"] = {"secure_ms": ds["secure_forward_ms"], "plaintext_fp32_ms": ds["plaintext_fp32_forward_ms"],
                                "rel_l2_per_layer": [v["rel_l2"] for v in ds["per_layer"]]}
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extras", action="store_true")
    ap.add_argument("--extras-file", default=None,
                    help="also write every extra measurement (the JSON line keeps a compact summary) to this file")
    ap.add_argument("--product-only", action="store_true",
                    help="only time the server ring product on uniform digits (for counter runs)")
    ap.add_argument("--passes-only", action="store_true",
                    help="only time the stand-alone passes (rotation, mask, samplers, quantisation, fused input "
                         "pass; for counter runs)")
    ap.add_argument("--decode-only", action="store_true",
                    help="only time the decode-shaped calls (for kernel traces)")
    ap.add_argument("--mfma-ceiling", action="store_true",
                    help="only the register-only MFMA probe and the server product on uniform and zero digits")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only copy 1 GiB device-to-device three times (scale for HBM byte counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU: the masked product is benchmarked on a single MI355X "
              f"(--gpus {args.gpus} is not supported)", file=sys.stderr)
        sys.exit(2)

    if args.product_only:
        print(json.dumps({"product_only": run_product_only()}))
        return

    if args.mfma_ceiling:
        print(json.dumps({"mfma_ceiling": run_mfma_ceiling()}))
        return

    if args.passes_only:
        import torch
        _warm_up(torch.device("cuda:0"))
        print(json.dumps({"passes": run_extras(torch.device("cuda:0"))}))
        return

    if args.decode_only:
        import torch
        _warm_up(torch.device("cuda:0"))
        print(json.dumps({"decode": run_decode(torch.device("cuda:0")),
                          "lpn_client_cost": run_lpn_client_cost(torch.device("cuda:0"))}))
        return

    if args.copy_calibration:
        import torch
        src = torch.empty(1 << 28, dtype=torch.int32, device="cuda")
        dst = torch.empty_like(src)
        src.fill_(1)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_per_dispatch": 1 << 30, "dispatches": 3}))
        return

    gpu = run_gpu(args.steps, args.warmup, not args.no_extras)
    line = {
        "metric": "masked Z_2^32 matmul ring-TOPS (% int8 MFMA peak) at 70B-layer shapes",
        "value": round(gpu["value"], 2),
        "unit": "ring-TOPS",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(gpu["ms_per_step"], 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u32 ring (i8 MFMA digits)",
        "data": "synthetic",
        "config": {"workload": "prefill masked products, 70B-layer shapes, M=2048, "
                               "(K,N) in {8192x8192, 8192x28672, 28672x8192}, d=1 r=1536 sigma=0.5",
                   "M": 2048, "shapes": [[8192, 8192], [8192, 28672], [28672, 8192]], "rank": gpu["rank"]},
        "roofline": gpu["roofline"],
        "per_shape": gpu["per_shape"],
    }
    if "extras" in gpu:
        # the matrix cores' own limit on operands like the masked ones
        # (uniformly random, changing every instruction): the roofline's
        # kernel against it, next to its fraction of the datasheet peak
        ceil = _mfma_probe_tops(2)
        line["mfma_random_operand_ceiling"] = {"tops": ceil, "unit": "TOP/s",
                                               "kernel_frac_of_it": round(gpu["roofline"]["achieved"] / ceil, 3)}
        line.update(_compact(gpu["extras"]))
        if args.extras_file:
            path = os.path.abspath(args.extras_file)
            try:
                os.makedirs(os.path.dirname(path), exist_ok=True)
                with open(path, "w") as f:
                    json.dump(gpu["extras"], f, indent=1)
                line["extras_file"] = args.extras_file
            except OSError as err:
                print(f"extras not written to {path}: {err}", file=sys.stderr)
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = run_cpu_baseline()
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
