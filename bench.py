#!/usr/bin/env python3
"""Throughput of the GauS hot path on one MI355X.

One step = one iteration of the relaxed-schedule optimization for all B
restarts of a synthetic workload: CDFs and masses of every (restart, op,
step), folded usage and the capacity penalty, dependency / recurrence /
edge-length terms over the edges, the analytic gradient, Adam and the
multiplier update (gaus_step).  The timed region also runs one rounding +
legalization of every restart (gaus_legalize), so every step of the path is
inside it.  Inputs are resident in HBM before timing starts.

Prints one JSON line with the metric (op-step evaluations per second =
B*N*D / seconds per step), the roofline of the dominant kernel (timed with
HIP events on the library's stream) and the CPU oracle timed on a bounded
sample of the same workload.

  python bench.py [--steps K] [--warmup W] [--workload large]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
METRIC = "op-step evals/sec (fwd+bwd+Adam), ms/iteration, % roofline at 50k ops"

# VALU cost model of one iteration (per-unit algorithmic work):
#   per op-bin-edge (B*N*(D-1) units): 20 FMA-class instructions plus 2
#     transcendental evaluations (the CDF needs an exp and a reciprocal; the
#     Gaussian factor of the gradient shares the exp);
#   per edge-step (B*(E+E_B)*(D-1) units): 10 FMA-class instructions (the
#     products and sums of the edge terms and their derivatives, with both
#     end points' rows available).
# A transcendental occupies TRANS_WEIGHT FMA issue slots: the measured ratio of
# the v_fma_f32 to the v_exp_f32 rate on gfx950 (gaus_microbench:
# 101.7 vs 21.2 per clock per CU).  One slot = one fp32 FMA = 2 flops; the
# peak is MI355X's 157.3 TFLOP/s fp32 vector rate.
#
# The units of one launch of a kernel are the op-bin-edges and edge-steps it
# is responsible for: the chunk-polynomial kernel (k_poly) owns the (restart,
# op) pairs classified onto its path and the edges with both ends there
# (gaus_poly_census); the step-by-step kernel (k_ops) owns the rest of the
# forward edges and ops.  k_poly reaches its units through per-chunk
# polynomial expansions, so its figure is an effective rate of this per-unit
# model, not an instruction-issue rate.
FMA_PER_OP_STEP = 20.0
TRANS_PER_OP_STEP = 2.0
FMA_PER_EDGE_STEP = 10.0
FMA_LANES_PER_CLK_CU = 101.7
EXP_LANES_PER_CLK_CU = 21.2
TRANS_WEIGHT = FMA_LANES_PER_CLK_CU / EXP_LANES_PER_CLK_CU
PEAK_TFLOPS = 157.3
# issue-rate reference: the measured v_fma_f32 rate above
N_CU = 256
CLOCK_HZ = 2.4e9
CSRC = os.path.join(ROOT, "paper_2602_20427_amd", "csrc")
# the sources a kernel is built from (its file and the shared device headers)
KERNEL_SOURCES = {"k_poly": "gaus_poly.hip", "k_ops": "gaus_step.hip"}
SHARED_HEADERS = ("gaus_device.h", "gaus_internal.h", "gaus_erfcx_coeffs.h")
KERNEL_NAMES = {"ops": "k_ops", "poly": "k_poly"}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def kernel_source_hash(kernel: str) -> str:
    h = hashlib.sha256()
    for name in (KERNEL_SOURCES[kernel], *SHARED_HEADERS):
        with open(os.path.join(CSRC, name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def model_flops(units_op, units_edge):
    slots = units_op * (FMA_PER_OP_STEP + TRANS_PER_OP_STEP * TRANS_WEIGHT) + units_edge * FMA_PER_EDGE_STEP
    return 2.0 * slots


def pmc_value(kernel, profile, key):
    """A figure from the committed rocprofv3 counter summary
    profiles/<profile>_pmc.md, if it was taken on the kernel's current
    sources; else None."""
    path = os.path.join(ROOT, "profiles", f"{profile}_pmc.md")
    if not os.path.exists(path):
        return None
    txt = open(path).read()
    h = re.search(r"kernel_source_sha256:\s*([0-9a-f]+)", txt)
    v = re.search(key + r":\s*([0-9.eE+]+)", txt)
    if not h or not v or h.group(1) != kernel_source_hash(kernel):
        return None
    return float(v.group(1))


def pmc_traffic(kernel, profile):
    """HBM bytes per launch from the committed counter summary, or None."""
    return pmc_value(kernel, profile, "traffic_bytes_per_launch")


def pmc_issue(kernel, profile, kernel_ms):
    """VALU issue rate from the committed SQ-counter summary, against the
    measured v_fma_f32 issue rate of the chip; else None."""
    valu = pmc_value(kernel, profile, "valu_instructions_per_launch")
    if valu is None:
        return None
    lane_ops = valu * 64
    rate = lane_ops / (kernel_ms * 1e-3)
    peak = FMA_LANES_PER_CLK_CU * N_CU * CLOCK_HZ
    return {"valu_lane_ops_per_launch": lane_ops, "achieved_lane_ops_per_s": rate,
            "peak_lane_ops_per_s": peak, "frac": rate / peak}


def describe(cfg, prob):
    return (f"{cfg.name}: random layered DAG, {prob.n_ops} ops, {cfg.n_layers} layers, "
            f"out-degree Poisson({cfg.out_degree}), {prob.n_edges} edges, {prob.n_back} back edges, "
            f"{prob.n_types} resource types, D={prob.D}, II={prob.II}, B={cfg.B} restarts, "
            f"fp32, paper initialization (sigma = kappa*(ALAP-ASAP))" if cfg.init != "uniform" else
            f"{cfg.name}: random layered DAG, {prob.n_ops} ops, D={prob.D}, B={cfg.B}, mu~U[0,D), sigma={cfg.sigma0}")


def cpu_baseline(prob, mu, sigma, lam, hp, min_seconds):
    """The oracle as it stands: one fused iteration (loss, gradient, Adam) per
    restart of the workload, cycling through the restarts from the same state
    until at least min_seconds have passed (and at least one restart)."""
    import numpy as np
    import oracle
    oracle.build(force=False)
    oracle.set_family(hp.family)
    B = mu.shape[0]
    done = 0
    t0 = time.perf_counter()
    while done == 0 or time.perf_counter() - t0 < min_seconds:
        b = done % B
        _, _, gm, gs, _ = oracle.loss_grad(prob, mu[b:b + 1].astype(np.float64), sigma[b:b + 1].astype(np.float64),
                                           lam[b:b + 1].astype(np.float64), hp.alpha_com, hp.rho,
                                           beta=hp.beta_res, tau=hp.tau, gamma=hp.gamma_mem)
        z = np.zeros(prob.n_ops)
        oracle.adam(mu[b].astype(np.float64), z, z, gm[0], 1, hp.lr)
        oracle.adam(sigma[b].astype(np.float64), z, z, gs[0], 1, hp.lr)
        done += 1
    dt = time.perf_counter() - t0
    oracle.set_family("gaussian")
    return {"value": done * prob.n_ops * prob.D / dt, "unit": "op-step evals/s",
            "cores": oracle.num_threads(), "kind": "oracle",
            "sample": f"{done} restart-iterations (cycling over the {B} restarts of the same workload and state), "
                      f"one fused iteration (loss, gradient, Adam) each, fp64 C oracle with OpenMP; {dt:.2f} s"}


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="large")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="minimum CPU time of the oracle sample (whole restart-iterations)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--poly-chunk", type=int, default=0,
                    help="chunk width of the polynomial path: 0 = library's choice, -1 = off (every op step by step)")
    ap.add_argument("--lse-beta", type=float, default=0.0,
                    help="weight of the smooth peak usage term (LogSumExp, temperature --tau); 0 = off")
    ap.add_argument("--tau", type=float, default=1e-2)
    ap.add_argument("--mem-gamma", type=float, default=0.0,
                    help="weight of the smooth peak storage term (storage units of 1-32 bits per op and a "
                         "sink op are added to the workload); 0 = off")
    ap.add_argument("--family", default="gaussian", choices=["gaussian", "logistic", "laplace", "cauchy"],
                    help="distribution of the relaxed start times (App. D); the Laplace law runs every "
                         "op step by step")
    ap.add_argument("--sigma", type=float, default=0.0,
                    help="replace the initial widths by this sigma (a sharpened state like late iterations: "
                         "ops narrower than the polynomial threshold run step by step); 0 = paper init")
    ap.add_argument("--solve-check-every", type=int, default=0,
                    help="time the Alg. 1 driver (gaus_solve) with a legalization check every this many "
                         "iterations instead of plain steps + one legalization; 0 = off")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="after the run, copy this many MiB once (counter calibration)")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py: this build runs the scheduling hot path on one GPU; multi-GPU runs "
              "(--gpus > 1) are not supported", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    from paper_2602_20427_amd import binding as bd
    from paper_2602_20427_amd.workloads import CONFIGS, make_problem, restart_uniforms, uniform_state, with_storage

    assert torch.cuda.is_available(), "bench.py needs an MI355X"
    cfg = CONFIGS[args.workload]
    log(f"[bench] workload {cfg.name}: building problem")
    prob = make_problem(cfg, seed=0)
    if args.mem_gamma:
        prob = with_storage(prob, seed=1)
    B, N, D = cfg.B, prob.n_ops, prob.D
    hp = bd.default_hparams()
    hp.lr = cfg.lr
    hp.poly_chunk = args.poly_chunk
    hp.beta_res = args.lse_beta
    hp.tau = args.tau
    hp.gamma_mem = args.mem_gamma
    hp.family = bd.FAMILIES[args.family]
    dev = torch.device("cuda")
    ctx = bd.Context(prob, B, hp)
    mu = torch.zeros(B, N, device=dev)
    sigma = torch.zeros(B, N, device=dev)
    if cfg.init == "uniform":
        m0, s0 = uniform_state(N, D, B, seed=0, sigma0=cfg.sigma0)
        mu.copy_(torch.from_numpy(m0)); sigma.copy_(torch.from_numpy(s0))
    else:
        ctx.init_state(mu, sigma, restart_uniforms(N, B, seed=0))
    if args.sigma > 0:
        sigma.fill_(args.sigma)
    lam = torch.full((B, 3), hp.lambda0, device=dev)
    m = torch.zeros(2, B, N, device=dev)
    v = torch.zeros(2, B, N, device=dev)
    t = torch.zeros(1, dtype=torch.int32, device=dev)
    # state of the CPU-baseline sample: the timing state before any step
    mu0, sg0, lam0 = mu.cpu().numpy(), sigma.cpu().numpy(), lam.cpu().numpy()
    ctx.bind_state(mu, sigma, m, v, lam, t)
    terms = torch.zeros(B, bd.N_TERMS, device=dev)
    sched = torch.zeros(B, N, dtype=torch.int32, device=dev)

    log(f"[bench] warmup {args.warmup} steps")
    ctx.step(args.warmup, terms)
    ctx.sync()
    torch.cuda.synchronize()

    log(f"[bench] timing {args.steps} steps + 1 legalization")
    stream = torch.cuda.current_stream()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
    ctx.kernel_timing(True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    solve_stats = None
    if args.solve_check_every:
        best_cost = torch.zeros(B, bd.N_COST, dtype=torch.float64, device=dev)
        ev[0].record(stream)
        solve_stats = ctx.solve(sched, best_cost, max_iters=args.steps, check_every=args.solve_check_every)
        ev[1].record(stream)
        ev[2].record(stream)
        status = None
    else:
        ev[0].record(stream)
        ctx.step(args.steps, terms)
        ev[1].record(stream)
        status = ctx.legalize(mu, sched)
        ev[2].record(stream)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    if status is None:   # driver: 0 where the best schedule is legal
        status = (best_cost[:, 5] == 0).int().cpu().numpy()
    ktimes = ctx.kernel_timing_read()
    ctx.kernel_timing(False)
    census = ctx.poly_census()
    poly_cfg = ctx.poly_config()
    grids = ctx.poly_grids()
    for gr, n in zip(grids, ctx.poly_grid_census()):
        gr["ops"] = n
    step_ms_events = ev[0].elapsed_time(ev[1]) / args.steps
    legalize_ms = ev[1].elapsed_time(ev[2])
    ms_per_step = (t1 - t0) * 1e3 / args.steps
    tt = terms.cpu().numpy()

    # units of each per-step kernel (see the cost model above)
    E = prob.n_edges
    units = {"poly": (census["ops"] * (D - 1), census["edges"] * (D - 1)),
             "ops": ((B * N - census["ops"]) * (D - 1), (B * E - census["edges"]) * (D - 1))}
    kern = {}
    for k, (tot_ms, n) in ktimes.items():
        if n == 0:
            continue
        kms = tot_ms / n
        fl = model_flops(*units[k])
        kern[KERNEL_NAMES[k]] = {"ms": kms, "launches": n, "op_bin_edges": units[k][0],
                                 "edge_steps": units[k][1], "model_tflops": fl / 1e12,
                                 "achieved_tflops": fl / (kms * 1e-3) / 1e12}
    dom = max(kern, key=lambda k: kern[k]["ms"])
    log(f"[bench] {ms_per_step:.3f} ms/step wall; gaus_step {step_ms_events:.3f} ms/iter (events); "
        f"legalize {legalize_ms:.3f} ms; " +
        "; ".join(f"{k} {v['ms']:.3f} ms x {v['launches']}" for k, v in kern.items()))
    log(f"[bench] polynomial path: {census['ops']} of {B * N} (restart, op) pairs, "
        f"{census['edges']} of {B * E} (restart, edge) pairs; per grid (P, W, ops): " +
        ", ".join(f"({g['P']}, {g['W']}, {g['ops']})" for g in grids if g["on"]))
    log(f"[bench] last terms restart 0: L={tt[0, 0]:.6g} V_dep={tt[0, 1]:.6g} V_res={tt[0, 2]:.6g} "
        f"V_rec={tt[0, 3]:.6g} L_com={tt[0, 4]:.6g}; legalize status {status.tolist()}")

    value = B * N * D / (ms_per_step * 1e-3)
    achieved = kern[dom]["achieved_tflops"]
    # committed counter summary of this kernel and launch configuration
    profile = f"{dom}_{args.workload}" + ("" if args.poly_chunk == 0 else
                                          "_direct" if args.poly_chunk < 0 else f"_w{args.poly_chunk}")
    if args.lse_beta:
        profile += "_lse"
    if args.mem_gamma:
        profile += "_mem"
    if args.family != "gaussian":
        profile += "_" + args.family
    if args.sigma > 0:
        profile += f"_sigma{args.sigma:g}"
    whole = model_flops(B * N * (D - 1), B * (E + prob.n_back) * (D - 1))
    out = {
        "metric": METRIC, "value": value, "unit": "op-step evals/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_per_step,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": describe(cfg, prob), "B": B, "N": N, "E": E,
                   "n_back": prob.n_back, "D": D, "II": prob.II,
                   "objective": "alpha L_com + ALM(V_dep, V_res, V_rec)" +
                                (f" + {args.lse_beta:g} L_res (tau {args.tau:g})" if args.lse_beta else "") +
                                (f" + {args.mem_gamma:g} L_mem (tau {args.tau:g}; storage units and a sink op)"
                                 if args.mem_gamma else ""),
                   "family": args.family,
                   "state": "paper initialization" if args.sigma <= 0 else
                            f"paper initialization means, sigma = {args.sigma:g}"},
        "ms_per_iteration_events": step_ms_events, "legalize_ms": legalize_ms,
        "poly_path": dict(poly_cfg, ops=census["ops"], edges=census["edges"], grids=grids),
        "solve": solve_stats,
        "roofline": {"bound": "alu", "achieved": achieved, "peak": PEAK_TFLOPS, "unit": "TFLOP/s",
                     "frac": achieved / PEAK_TFLOPS,
                     "traffic": pmc_traffic(dom, profile),
                     "kernel": dom, "kernel_ms": kern[dom]["ms"],
                     "model": f"{FMA_PER_OP_STEP:g} FMA + {TRANS_PER_OP_STEP:g} transcendental "
                              f"(x{TRANS_WEIGHT:.2f} FMA slots) per op-bin-edge, {FMA_PER_EDGE_STEP:g} FMA per "
                              f"edge-step, 2 flops per FMA slot; units = those the kernel owns",
                     "note": "k_poly reaches its op-bin-edges through per-chunk polynomial expansions and "
                             "needs fewer operations than this per-step model charges, so frac can exceed 1; "
                             "'issue' gives its measured VALU issue rate"},
        "issue": pmc_issue(dom, profile, kern[dom]["ms"]),
        "kernels": kern,
        "iteration_model_tflops_per_s": whole / (step_ms_events * 1e-3) / 1e12,
    }
    if not args.no_cpu_baseline:
        log(f"[bench] CPU oracle for at least {args.cpu_seconds:g} s")
        out["cpu_baseline"] = cpu_baseline(prob, mu0, sg0, lam0, hp, args.cpu_seconds)
    if args.copy_probe_mib > 0:
        n = args.copy_probe_mib * (1 << 20) // 4
        a = torch.ones(n, device=dev)
        b = torch.empty_like(a)
        torch.cuda.synchronize()
        b.copy_(a)
        torch.cuda.synchronize()
        log(f"[bench] copy probe: {args.copy_probe_mib} MiB read + {args.copy_probe_mib} MiB written")
    ctx.close()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
