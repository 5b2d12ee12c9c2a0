"""SOAP optimizer-step throughput on one MI355X.

Workload: one 4096 x 14336 fp32 weight (MLP up-projection shape), low-rank
(rank 128) plus 10%-noise synthetic gradients, every step a full SOAP update
with per-step QR refresh of both eigenbases (R is 14336 x 14336).  Gradients
are generated and copied to HBM before the timed region.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-cpu-baseline]
                    [--calibration-copy-mib N] [--kl] [--refresh-every F] [--stale]
                    [--muon] [--workload {1,3,4}] [--group]

--kl times the KL-SOAP step instead (soap_kl_step, beta_kron 0.95): the
factors are accumulated by the KL-Shampoo rule, the rest of the step is the
same.  --refresh-every F refreshes the eigenbases only when t mod F = 0
(Algorithm 2's F; the paper uses 1), --stale takes the refresh from the
factors before the step's gradient (the ablation of Section 5.4.1).  --muon
times the Muon step of Algorithm 1 on the same weight instead (16
Newton-Schulz iterations; the paper's PolarExpress coefficients are not
printed, so the Taylor quintic (15/8, -5/4, 3/8) stands in: the cost does
not depend on the values).  --workload 1 / 3 / 4 time the SOAP step on the
other workloads instead: the 4096 x 4096 attention projection, the bank of 64
experts of 2048 x 768 through soap_step_batched, and the 24-layer model (96
matrices of four shapes; one soap_step per matrix from one host loop, or with
--group one soap_step_batched per shape).  These reuse one gradient per
matrix for every step.

Prints ONE JSON line.  `value` is steps/s of the whole step; `roofline`
describes the dominant kernel (timed with HIP events on the library's stream
through the soap_timing_* API); `cpu_baseline` times the fp64 oracle on a
bounded sample of the same workload.
"""
import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_FP32_MFMA_TFLOPS = 157.3   # MI355X dense fp32 matrix peak (256 CU x 256 flop/clk x 2.4 GHz)
PEAK_BF16_MFMA_TFLOPS = 2500.0  # MI355X dense bf16 matrix peak (datasheet, no sparsity)
PEAK_HBM_GBS = 8000.0
HP = dict(beta1=0.95, beta2=0.95, eps=1e-8, lr=1e-3, weight_decay=0.1)
BETA_KRON = 0.95   # KL-Shampoo accumulation coefficient (hyperparameter table of Section 5.4)


def step_flops(m: int, n: int) -> float:
    """Algorithmic flops of one SOAP step on an m x n weight: one triangle of
    each factor EMA, the two power products, Householder QR with explicit Q of
    both factors, and three rotation pairs (the Adam/momentum terms are O(mn))."""
    syrk = m * (m + 1) * n + n * (n + 1) * m
    power = 2.0 * (m ** 3 + n ** 3)
    qr = (8.0 / 3.0) * (m ** 3 + n ** 3)
    rot = 6.0 * m * n * (m + n)
    return syrk + power + qr + rot


def kl_step_flops(m: int, n: int) -> float:
    """step_flops plus the KL accumulation's extra products: Q^T F for the
    eigenvalue estimates of both factors and the projections Q_L^T G, G Q_R."""
    return step_flops(m, n) + 2.0 * (m ** 3 + n ** 3) + 2.0 * m * n * (m + n)


MUON_COEFFS = [(15 / 8, -5 / 4, 3 / 8)] * 16
MUON_HP = dict(beta1=0.9, lr=2e-2, weight_decay=0.1, eps=1e-7)


def muon_step_flops(m: int, n: int, iters: int = 16) -> float:
    """Per Newton-Schulz iteration on the smaller side d (other side e): one
    triangle of the Gram matrix d(d+1)e, the square 2d^3 and the product 2d^2e."""
    d, e = min(m, n), max(m, n)
    return iters * (d * (d + 1) * e + 2.0 * d ** 3 + 2.0 * d * d * e)


def bench_muon(args, soap, torch, sg):
    spec = sg.workload(2).matrices[0]
    m, n = spec.m, spec.n
    total = args.warmup + args.steps
    grads = [torch.from_numpy(G).cuda() for G in sg.make_matrix_stream(spec, 2, total)]
    W = torch.from_numpy(sg.initial_weight(spec, 2)).cuda()
    state = soap.MuonState(m, n)
    stream = torch.cuda.current_stream()
    bf = bool(args.bf16)
    for t in range(args.warmup):
        state.step(W, grads[t], MUON_COEFFS, bf16=bf, **MUON_HP)
    torch.cuda.synchronize()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for t in range(args.steps):
        state.step(W, grads[args.warmup + t], MUON_COEFFS, bf16=bf, stream=stream, **MUON_HP)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    # stage breakdown over separate steps (HIP events around every stage)
    soap.soap_timing_reset()
    soap.soap_timing_enable(True)
    for t in range(args.stage_steps):
        state.step(W, grads[(args.warmup + t) % total], MUON_COEFFS, bf16=bf, stream=stream,
                   **MUON_HP)
    torch.cuda.synchronize()
    soap.soap_timing_enable(False)
    soap.soap_timing_collect()
    stages = {}
    for i in range(soap.soap_timing_num_stages()):
        ms, launches, fl = soap.soap_timing_get(i)
        if launches:
            stages[soap.soap_timing_stage_name(i)] = (ms, launches, fl)
    ns_ms, ns_n, ns_fl = stages["muon_newton_schulz"]
    achieved = ns_fl / (ns_ms * 1e-3) / 1e12
    F = muon_step_flops(m, n)
    value = args.steps / elapsed
    peak = PEAK_BF16_MFMA_TFLOPS if bf else PEAK_FP32_MFMA_TFLOPS
    out = {
        "metric": "Muon steps/s per weight shape + achieved MFMA TFLOPS fraction (1 GPU)",
        "value": value, "unit": "steps/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": 1e3 * elapsed / args.steps,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16 (Newton-Schulz), f32 (rest)" if bf else "f32",
        "data": "synthetic (seeded low-rank + noise gradients, rank 128, 10% noise)",
        "config": {"workload": f"soap_muon_step on one {m}x{n} fp32 weight (MLP up-projection), "
                               f"16 Newton-Schulz iterations in {'bf16' if bf else 'fp32'}",
                   "m": m, "n": n, "rank": spec.rank, "global_batch": 1, "seq_len": None,
                   "parallelism": "none (1 GPU)"},
        "step_tflops": F * value / 1e12,
        "step_frac_of_fp32_mfma_peak": F * value / 1e12 / PEAK_FP32_MFMA_TFLOPS,
        "roofline": {"bound": "mfma", "kernel": "muon_newton_schulz (SYRK + two GEMMs per "
                                                "iteration)",
                     "achieved": achieved, "peak": peak, "unit": "TFLOP/s",
                     "frac": achieved / peak, "traffic": None,
                     "avg_launch_ms": ns_ms / ns_n},
        "stage_ms_per_step": {k: v[0] / max(1, args.stage_steps) for k, v in stages.items()},
    }
    if not args.no_cpu_baseline:
        import oracle
        ms_, ns_ = m // 4, n // 4
        sp = sg.MatrixSpec("cpu_sample", ms_, ns_, max(1, spec.rank // 4), "rel", 0.10)
        G = next(sg.make_matrix_stream(sp, 2, 1)).astype(np.float64)
        t1 = time.perf_counter()
        oracle.muon_step(np.zeros((ms_, ns_)), np.zeros((ms_, ns_)), G, coeffs=MUON_COEFFS,
                         **MUON_HP)
        dt = time.perf_counter() - t1
        ratio = muon_step_flops(m, n) / muon_step_flops(ms_, ns_)
        threads = int(os.environ.get("OMP_NUM_THREADS", "0") or 0) or len(os.sched_getaffinity(0))
        out["cpu_baseline"] = {
            "value": 1.0 / (dt * ratio), "unit": "steps/s", "cores": threads, "kind": "oracle",
            "sample": f"one fp64 oracle Muon step on a {ms_}x{ns_} matrix took {dt:.2f} s; "
                      f"scaled by the exact flop ratio {ratio:.1f}"}
    print(json.dumps(out), flush=True)


def bench_workload(args, soap, torch, sg):
    """Whole-workload SOAP step time on workload 1, 3 or 4 (information lines)."""
    wl = sg.workload(args.workload)
    specs = wl.matrices
    groups = {}
    for sp in specs:
        groups.setdefault((sp.m, sp.n), []).append(sp)
    scales = sg.expert_scales(0, 3, len(specs)) if args.workload == 3 else None
    calls = []   # (state, W, G) with W, G on the device; batched states take stacked tensors
    total_flops = sum(step_flops(sp.m, sp.n) for sp in specs)

    def grad(sp, i):
        g = next(sg.make_matrix_stream(sp, args.workload, 1))
        return g * np.float32(scales[i]) if scales is not None else g

    if args.workload == 3 or args.group:
        for (m, n), sps in groups.items():
            idx = [specs.index(sp) for sp in sps]
            W = torch.from_numpy(np.stack([sg.initial_weight(sp, args.workload) for sp in sps])).cuda()
            G = torch.from_numpy(np.stack([grad(sp, i) for sp, i in zip(sps, idx)])).cuda()
            st = soap.SoapState(m, n, batch=len(sps))
            calls.append((st, W, G))
    else:
        shared = {}
        for i, sp in enumerate(specs):
            key = (sp.m, sp.n)
            if key not in shared:
                shared[key] = soap.SoapState(sp.m, sp.n)
            st = shared[key]
            own = soap.SoapState.__new__(soap.SoapState)   # state tensors per matrix, shared workspace
            own.__dict__.update(st.__dict__)
            kw = dict(dtype=torch.float32, device="cuda")
            own.L = torch.empty((sp.m, sp.m), **kw); own.R = torch.empty((sp.n, sp.n), **kw)
            own.Q_L = torch.empty((sp.m, sp.m), **kw); own.Q_R = torch.empty((sp.n, sp.n), **kw)
            own.M = torch.empty((sp.m, sp.n), **kw); own.V = torch.empty((sp.m, sp.n), **kw)
            soap.soap_init_state(1, sp.m, sp.n, own.L, own.R, own.Q_L, own.Q_R, own.M, own.V)
            calls.append((own, torch.from_numpy(sg.initial_weight(sp, args.workload)).cuda(),
                          torch.from_numpy(grad(sp, i)).cuda()))
    stream = torch.cuda.current_stream()
    for t in range(1, args.warmup + 1):
        for st, W, G in calls:
            st.step(W, G, t, **HP)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for t in range(1, args.steps + 1):
        for st, W, G in calls:
            st.step(W, G, args.warmup + t, stream=stream, **HP)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    value = args.steps / elapsed
    desc = {1: "soap_step on one 4096x4096 fp32 weight (attention projection)",
            3: "soap_step_batched on 64 experts of 2048x768 (one call)",
            4: "the 24-layer dense model (hidden 2048, FFN 8192): 96 matrices, "
               + ("one soap_step_batched per shape" if args.group else "one soap_step per matrix")}
    out = {
        "metric": "SOAP steps/s of the whole workload (1 GPU)", "value": value, "unit": "steps/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": 1e3 * elapsed / args.steps, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32",
        "data": "synthetic (seeded low-rank + noise gradients; one gradient per matrix reused)",
        "config": {"workload": desc[args.workload], "matrices": len(specs),
                   "shapes": sorted(groups.keys()), "parallelism": "none (1 GPU)"},
        "step_tflops": total_flops * value / 1e12,
        "step_frac_of_fp32_mfma_peak": total_flops * value / 1e12 / PEAK_FP32_MFMA_TFLOPS,
    }
    print(json.dumps(out), flush=True)


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "power_product_R_4096x14336_traffic.json")
GEMM_SOURCE = os.path.join(ROOT, "paper_2607_20548_amd", "csrc", "gemm.hip")


def gemm_source_hash() -> str:
    with open(GEMM_SOURCE, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def measured_traffic():
    """HBM bytes per power-product launch from the committed counter summary,
    or None if there is none or it was taken on another GEMM source."""
    try:
        with open(TRAFFIC_FILE) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    if rec.get("gemm_source_sha256") != gemm_source_hash():
        return None
    return rec.get("bytes_per_launch")


def cpu_baseline(m: int, n: int, rank: int, scale: int = 4, kl: bool = False):
    """Times one fp64 oracle step on the workload shrunk by `scale` per side
    (same aspect ratio, rank and noise recipe) and scales the time by
    step_flops(m, n) / step_flops(m/scale, n/scale) (= scale^3: the step's work
    is a homogeneous cubic in the dimensions)."""
    import oracle
    from synth import gradients as sg
    ms, ns = m // scale, n // scale
    spec = sg.MatrixSpec("cpu_sample", ms, ns, max(1, rank // scale), "rel", 0.10)
    G = next(sg.make_matrix_stream(spec, 2, 1)).astype(np.float64)
    st = oracle.init_state(sg.initial_weight(spec, 2).astype(np.float64))
    t0 = time.perf_counter()
    if kl:
        oracle.kl_soap_step(st, G, 1, beta_kron=BETA_KRON, **HP)
    else:
        oracle.soap_step(st, G, 1, **HP)
    dt = time.perf_counter() - t0
    fl = kl_step_flops if kl else step_flops
    ratio = fl(m, n) / fl(ms, ns)
    threads = int(os.environ.get("OMP_NUM_THREADS", "0") or 0) or len(os.sched_getaffinity(0))
    return {
        "value": 1.0 / (dt * ratio), "unit": "steps/s", "cores": threads, "kind": "oracle",
        "sample": (f"one fp64 oracle {'KL-SOAP ' if kl else ''}step on a {ms}x{ns} matrix (the {m}x{n} workload at 1/{scale} "
                   f"per side, rank {spec.rank}, 10% noise) took {dt:.2f} s; scaled by the exact "
                   f"flop ratio {ratio:.1f}"),
    }


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--stage-steps", type=int, default=3,
                    help="steps run after the timed ones with per-stage HIP events")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calibration-copy-mib", type=int, default=0)
    ap.add_argument("--kl", action="store_true", help="time the KL-SOAP step")
    ap.add_argument("--refresh-every", type=int, default=1)
    ap.add_argument("--stale", action="store_true")
    ap.add_argument("--muon", action="store_true", help="time the Muon step instead")
    ap.add_argument("--bf16", action="store_true",
                    help="with --muon: Newton-Schulz in bfloat16 (the paper's precision)")
    ap.add_argument("--workload", type=int, default=2, choices=[1, 2, 3, 4])
    ap.add_argument("--group", action="store_true",
                    help="workload 4: one batched call per shape instead of one call per matrix")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the SOAP step of a "
              "matrix is independent of every other matrix and this build has no multi-GPU path.",
              file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2607_20548_amd as soap
    from synth import gradients as sg

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    if args.muon:
        return bench_muon(args, soap, torch, sg)
    if args.workload != 2:
        return bench_workload(args, soap, torch, sg)
    wl = sg.workload(2)
    spec = wl.matrices[0]
    m, n = spec.m, spec.n
    total = args.warmup + args.steps
    print(f"[bench] generating {total} gradients {m}x{n}", file=sys.stderr, flush=True)
    grads = [torch.from_numpy(G).cuda() for G in sg.make_matrix_stream(spec, 2, total)]
    W = torch.from_numpy(sg.initial_weight(spec, 2)).cuda()
    state = soap.SoapState(m, n, kl=args.kl)
    stream = torch.cuda.current_stream()
    extra = dict(beta_kron=BETA_KRON) if args.kl else {}
    extra.update(refresh_every=args.refresh_every, stale_refresh=args.stale)

    for t in range(1, args.warmup + 1):
        state.step(W, grads[t - 1], t, **extra, **HP)
    torch.cuda.synchronize()
    if args.calibration_copy_mib > 0:
        nel = args.calibration_copy_mib * (1 << 20) // 4
        src = torch.ones(nel, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        print(f"[bench] calibration copy of {args.calibration_copy_mib} MiB done", file=sys.stderr,
              flush=True)
        del src, dst
    soap.soap_init_state(1, m, n, state.L, state.R, state.Q_L, state.Q_R, state.M, state.V)
    torch.cuda.synchronize()
    print(f"[bench] warmup done; timing {args.steps} steps", file=sys.stderr, flush=True)

    # the timed steps run without stage events
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for t in range(1, args.steps + 1):
        state.step(W, grads[args.warmup + t - 1], t, stream=stream, **extra, **HP)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    print(f"[bench] timed {args.steps} steps: {1e3 * elapsed / args.steps:.2f} ms/step; "
          f"stage breakdown over {args.stage_steps} more", file=sys.stderr, flush=True)

    # stage breakdown (HIP events around every stage, on the stream that runs
    # it) over separate steps, continuing the same run
    soap.soap_timing_reset()
    soap.soap_timing_enable(True)
    for i in range(args.stage_steps):
        t = args.steps + 1 + i
        state.step(W, grads[(args.warmup + t - 1) % total], t, stream=stream, **extra, **HP)
    torch.cuda.synchronize()
    soap.soap_timing_enable(False)
    soap.soap_timing_collect()

    stages = {}
    for i in range(soap.soap_timing_num_stages()):
        ms, launches, fl = soap.soap_timing_get(i)
        stages[soap.soap_timing_stage_name(i)] = (ms, launches, fl)
    # dominant single-kernel stage among the MFMA GEMMs (the QR stages are
    # sequences of kernels and are reported separately)
    single = {k: v for k, v in stages.items() if k.startswith(("power", "factor", "rotate"))
              and v[1] > 0 and not k.startswith("rotate_in_QLt")}
    nst = max(1, args.stage_steps)
    roofline = None
    if single:
        dom = max(single, key=lambda k: single[k][0])
        d_ms, d_n, d_fl = single[dom]
        achieved = d_fl / (d_ms / d_n * 1e-3) / d_n / 1e12
        roofline = {"bound": "mfma", "kernel": dom, "achieved": achieved,
                    "peak": PEAK_FP32_MFMA_TFLOPS, "unit": "TFLOP/s",
                    "frac": achieved / PEAK_FP32_MFMA_TFLOPS,
                    "traffic": measured_traffic() if dom == "power_R" else None,
                    "traffic_unit": "HBM bytes per launch", "avg_launch_ms": d_ms / d_n}

    F = (kl_step_flops if args.kl else step_flops)(m, n)
    if args.refresh_every > 1:   # the power products and QRs run on 1 step in F
        F -= (1.0 - 1.0 / args.refresh_every) * (2.0 + 8.0 / 3.0) * (m ** 3 + n ** 3)
    value = args.steps / elapsed
    name = "KL-SOAP" if args.kl else "SOAP"
    out = {
        "metric": f"{name} steps/s per weight shape + achieved MFMA TFLOPS fraction (1 GPU)",
        "value": value,
        "unit": "steps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": 1e3 * elapsed / args.steps,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic (seeded low-rank + noise gradients, rank 128, 10% noise)",
        "config": {"workload": f"{'soap_kl_step' if args.kl else 'soap_step'} on one {m}x{n} fp32 "
                               f"weight (MLP up-projection), QR refresh of both factors every step"
                               + (f", KL-Shampoo factors (beta_kron {BETA_KRON})" if args.kl else "")
                               + (f", refresh every {args.refresh_every} steps"
                                  if args.refresh_every > 1 else "")
                               + (", stale refresh" if args.stale else ""),
                   "m": m, "n": n, "rank": spec.rank, "global_batch": 1, "seq_len": None,
                   "parallelism": "none (1 GPU)"},
        "step_tflops": F * value / 1e12,
        "step_frac_of_fp32_mfma_peak": F * value / 1e12 / PEAK_FP32_MFMA_TFLOPS,
        "roofline": roofline,
        "stage_ms_per_step": {k: v[0] / nst for k, v in stages.items() if v[1] > 0},
    }
    # The eigenbasis QR of the larger factor (n x n): a chain of latency-bound
    # block factorizations and MFMA updates, timed as one stage.
    # (square weights: both factors' QRs as one call, timed as "qr_L_R")
    qr_name = "qr_L_R" if stages.get("qr_L_R", (0, 0, 0))[1] else ("qr_R" if n >= m else "qr_L")
    q_ms, q_n, q_fl = stages[qr_name]
    if q_n and q_ms > 0:
        out["qr"] = {"stage": qr_name, "n": max(m, n), "ms": q_ms / q_n,
                     "tflops": q_fl / q_n / (q_ms / q_n * 1e-3) / 1e12,
                     "frac_of_fp32_mfma_peak": q_fl / q_n / (q_ms / q_n * 1e-3) / 1e12
                     / PEAK_FP32_MFMA_TFLOPS,
                     "share_of_step": (q_ms / nst) / (1e3 * elapsed / args.steps),
                     "flops": "(8/3) n^3 per factor: Householder factorization and explicit Q"}
    if not args.no_cpu_baseline:
        print("[bench] timing the oracle sample", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(m, n, spec.rank, kl=args.kl)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
