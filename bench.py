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

# Roofline of the dominant kernel.  Peaks are MI355X's published figures:
# fp32 vector 157.3 TFLOP/s = 256 CU x 128 FMA lanes per clock x 2.4 GHz x 2
# flops (7.86e13 FMA lane-operations/s), a transcendental (v_exp_f32,
# v_rcp_f32) issuing at a quarter of that rate (4 FMA slots), HBM 8 TB/s.
PEAK_TFLOPS = 157.3
N_CU = 256
CLOCK_HZ = 2.4e9
FMA_LANES_PER_CLK_CU = 128
PEAK_FMA_LANE_OPS = FMA_LANES_PER_CLK_CU * N_CU * CLOCK_HZ
TRANS_SLOTS = 4.0
PEAK_HBM_GBS = 8000.0

# (1) Chunk-polynomial kernel (k_poly): the work the method's sums require on
# a chunk of W steps at series degree d (NC = d + 1 coefficients per vector,
# the expansion carrying T_0 .. T_{d+2}), counted in FMA-class operations:
#   one CDF evaluation (tail and density of one z): the z value, |z|/sqrt(2),
#     z^2, the degree-8 rational form of erfc (8 FMA) and its products:
#     EVAL_FMA, plus 2 transcendentals (exp, reciprocal);
#   expansion at a chunk centre: one evaluation + 2 per Taylor coefficient
#     T_2 .. T_{d+2} (the three-term recursion with folded constants);
#   per (restart, op, chunk): the expansion at the centre, and for ops with
#     Lat != 1 a second one at the centre shifted by Lat - 1; the one-step mass
#     series (4 terms per coefficient) of both; dF/dmu one step back (5 terms
#     per coefficient); dF/dmu and dF/dsigma = z dF/dmu (3 per coefficient)
#     of both; the usage coefficients (1 per coefficient); six moment vectors
#     (H p)_k truncated at degree d (moments_fma(d) each);
#   per (restart, edge, chunk): the consumer's expansion, its dF/dmu,
#     dF/dsigma and mass (1 + 2 + 4 per coefficient) and ten dot products;
#   strip positions (per restart, SP = L0 + 2 of them): one evaluation per
#     op and position plus STRIP_OP_FMA for the derived rows, one evaluation
#     per edge and position plus STRIP_EDGE_FMA for its products.
EVAL_FMA = 14
STRIP_OP_FMA = 8
STRIP_EDGE_FMA = 12
TIER_DEGREE = {1: 8, 2: 6, 3: 5}


def moments_fma(d):
    """FMAs of one moment vector (H p)_k = sum_l H_{k+l} p_l over k + l <= d, k + l even."""
    return sum(t + 1 for t in range(0, d + 1, 2))


def expansion_fma(d):
    return EVAL_FMA + 2 * (d + 1)


def poly_op_chunk_fma(d, shifted):
    nc = d + 1
    per_expansion = expansion_fma(d) + 4 * nc + 3 * nc          # expansion, mass series, dF/dmu and dF/dsigma
    return (1 + shifted) * per_expansion + 5 * nc + nc + 6 * moments_fma(d)


def poly_edge_chunk_fma(d):
    nc = d + 1
    return expansion_fma(d) + 7 * nc + 10 * nc


def poly_model(tier_census, grids, shifted):
    """FMA-class operations and transcendentals of one k_poly launch from the
    census of (restart, op) pairs and polynomial edges per grid and tier;
    shifted = share of the ops whose delay is not 1."""
    fma = trans = 0.0
    for g, gr in enumerate(grids):
        if not gr["on"]:
            continue
        nc, sp = gr["chunks"], gr["L0"] + 2
        for t, d in TIER_DEGREE.items():
            ops, edges = float(tier_census[g][t][0]), float(tier_census[g][t][1])
            fma += ops * (nc * poly_op_chunk_fma(d, shifted) + sp * (EVAL_FMA + STRIP_OP_FMA))
            fma += edges * (nc * poly_edge_chunk_fma(d) + sp * (EVAL_FMA + STRIP_EDGE_FMA))
            trans += ops * (nc * 2 * (1 + shifted) + sp * 2) + edges * (nc * 2 + sp * 2)
    return fma, trans


# (2) Step-by-step op kernel (k_ops; the narrow regime, where each op's CDF
# differs from exactly 0 or 1 on a few steps only): bound by memory traffic
# and latency, priced against HBM with the bytes any split of the method
# must move across this kernel's boundary: per (restart, op) its mean and
# width in and four producer-side derivative pieces out (24 B); per
# (restart, edge) the consumer's mean and width in and four consumer-side
# pieces out (24 B); per (restart, type, step) one usage value out (4 B); the
# graph once (delay, type, row start per op, consumer per edge: 12 B + 4 B).
OPS_BYTES_PER_OP, OPS_BYTES_PER_EDGE, OPS_BYTES_PER_USAGE = 24, 24, 4

# (3) The per-step model of the whole iteration, kept as an effective rate
# (not a roofline): per op-bin-edge 20 FMA-class instructions and 2
# transcendentals, per edge-step 10; the chunk polynomials reach these units
# with far fewer operations, so this rate can exceed the fp32 peak.
FMA_PER_OP_STEP = 20.0
TRANS_PER_OP_STEP = 2.0
FMA_PER_EDGE_STEP = 10.0

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


def per_step_model_flops(units_op, units_edge):
    slots = units_op * (FMA_PER_OP_STEP + TRANS_PER_OP_STEP * TRANS_SLOTS) + units_edge * FMA_PER_EDGE_STEP
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
    """VALU issue rate (wave instructions x 64 lanes) from the committed
    SQ-counter summary, against the fp32 FMA lane rate of the spec
    (128 lanes per clock per CU); else None."""
    valu = pmc_value(kernel, profile, "valu_instructions_per_launch")
    if valu is None:
        return None
    lane_ops = valu * 64
    rate = lane_ops / (kernel_ms * 1e-3)
    return {"valu_lane_ops_per_launch": lane_ops, "achieved_lane_ops_per_s": rate,
            "peak_lane_ops_per_s": PEAK_FMA_LANE_OPS, "frac": rate / PEAK_FMA_LANE_OPS}


def describe(cfg, prob):
    return (f"{cfg.name}: random layered DAG, {prob.n_ops} ops, {cfg.n_layers} layers, "
            f"out-degree Poisson({cfg.out_degree}), {prob.n_edges} edges, {prob.n_back} back edges, "
            f"{prob.n_types} resource types, D={prob.D}, II={prob.II}, B={cfg.B} restarts, "
            f"fp32, paper initialization (sigma = kappa*(ALAP-ASAP))" if cfg.init != "uniform" else
            f"{cfg.name}: random layered DAG, {prob.n_ops} ops, D={prob.D}, B={cfg.B}, mu~U[0,D), sigma={cfg.sigma0}")


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def _oracle_iterations(prob, mu, sigma, lam, hp, min_seconds, max_iters=None):
    """Whole restart-iterations of the oracle (loss, gradient, Adam on mu and
    sigma) cycling over the restarts from the same state, until min_seconds
    have passed (at least one); returns (count, seconds)."""
    import numpy as np
    import oracle
    B = mu.shape[0]
    done = 0
    t0 = time.perf_counter()
    while done == 0 or (time.perf_counter() - t0 < min_seconds and (max_iters is None or done < max_iters)):
        b = done % B
        _, _, gm, gs, _ = oracle.loss_grad(prob, mu[b:b + 1].astype(np.float64), sigma[b:b + 1].astype(np.float64),
                                           lam[b:b + 1].astype(np.float64), hp.alpha_com, hp.rho,
                                           beta=hp.beta_res, tau=hp.tau, gamma=hp.gamma_mem)
        z = np.zeros(mu.shape[1])
        oracle.adam(mu[b].astype(np.float64), z, z, gm[0], 1, hp.lr)
        oracle.adam(sigma[b].astype(np.float64), z, z, gs[0], 1, hp.lr)
        done += 1
    return done, time.perf_counter() - t0


def cpu_baseline(prob, mu, sigma, lam, hp, min_seconds, single_ops, cfg=None):
    """The oracle as it stands, timed on the host's cores:
    * all threads: whole restart-iterations of the full workload from the
      benchmark's state, cycling over the B restarts, for at least
      min_seconds; value = op-step evals/s, plus ms per B-restart iteration;
    * one thread: one restart-iteration of the same generator and
      parameters at single_ops ops (same horizon, out-degree, delays, types,
      capacities), the bounded single-core sample."""
    import numpy as np
    import oracle
    oracle.build(force=False)
    oracle.set_family(hp.family)
    B, D = mu.shape[0], prob.D
    threads = oracle.num_threads()
    done, dt = _oracle_iterations(prob, mu, sigma, lam, hp, min_seconds)
    out = {"value": done * prob.n_ops * D / dt, "unit": "op-step evals/s", "cores": threads, "kind": "oracle",
           "cpu_model": cpu_model(),
           "ms_per_iteration": dt / done * B * 1e3,
           "sample": f"{done} restart-iterations of the full workload (cycling over its {B} restarts from the "
                     f"benchmark's state), each one fused iteration (loss, gradient, Adam), fp64 C oracle, "
                     f"OpenMP on {threads} threads; {dt:.2f} s; ms_per_iteration = the {B} restarts of one "
                     f"iteration"}
    if single_ops > 0 and cfg is not None:
        from paper_2602_20427_amd.workloads import make_problem, restart_uniforms
        n = min(single_ops, prob.n_ops)
        sub = make_problem(cfg, seed=0, n_ops=n)
        u = restart_uniforms(n, 1, seed=0)
        m1, s1, rc = oracle.init_state(sub, 1, u, kappa=float(hp.kappa), sigma_min=float(hp.sigma_min))
        oracle.set_num_threads(1)
        try:
            d1, t1 = _oracle_iterations(sub, m1.astype(np.float32), s1.astype(np.float32), lam[:1], hp, 0.0,
                                        max_iters=1)
        finally:
            oracle.set_num_threads(threads)
        rate1 = d1 * n * D / t1
        out["single_thread"] = {
            "value": rate1, "unit": "op-step evals/s", "cores": 1,
            "ms_per_iteration_scaled": B * prob.n_ops * D / rate1 * 1e3,
            "sample": f"{d1} restart-iteration (loss, gradient, Adam) of the same generator and parameters at "
                      f"{n} ops ({sub.n_edges} edges, D={D}, paper initialization), 1 thread; {t1:.2f} s; "
                      f"ms_per_iteration_scaled = B*N*D of the full workload at that rate"}
    oracle.set_family("gaussian")
    return out


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="large")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="minimum CPU time of the oracle sample (whole restart-iterations)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-single-ops", type=int, default=5000,
                    help="ops of the one-thread oracle sample (the same generator at this size); 0 = skip")
    ap.add_argument("--poly-chunk", type=int, default=0,
                    help="chunk width of the polynomial path: 0 = library's choice, -1 = off (every op step by step)")
    ap.add_argument("--lse-beta", type=float, default=0.0,
                    help="weight of the smooth peak usage term (LogSumExp, temperature --tau); 0 = off")
    ap.add_argument("--tau", type=float, default=1e-2)
    ap.add_argument("--mem-gamma", type=float, default=0.0,
                    help="weight of the smooth peak storage term (storage units of 1-32 bits per op and a "
                         "sink op are added to the workload); 0 = off")
    ap.add_argument("--family", default="gaussian", choices=["gaussian", "logistic", "laplace", "cauchy"],
                    help="distribution of the relaxed start times (App. E); the Laplace law runs every "
                         "op step by step")
    ap.add_argument("--sigma", type=float, default=0.0,
                    help="replace the initial widths by this sigma (a sharpened state like late iterations: "
                         "ops narrower than the polynomial threshold run step by step); 0 = paper init")
    ap.add_argument("--solve-check-every", type=int, default=0,
                    help="time the Alg. 1 driver (gaus_solve) with a legalization check every this many "
                         "iterations instead of plain steps + one legalization; 0 = off")
    ap.add_argument("--kernel-timing-every", type=int, default=10,
                    help="bracket the op and polynomial kernels of every n-th timed iteration with HIP events "
                         "(each event adds a few microseconds between launches; 1 = every iteration)")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="after the run, copy this many MiB once (counter calibration)")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py: the library runs the scheduling hot path on one GPU; multi-GPU runs "
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
    ctx.kernel_timing(max(1, args.kernel_timing_every))
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
    tier_census = ctx.poly_tier_census()
    poly_cfg = ctx.poly_config()
    grids = ctx.poly_grids()
    for gr, n in zip(grids, ctx.poly_grid_census()):
        gr["ops"] = n
    step_ms_events = ev[0].elapsed_time(ev[1]) / args.steps
    legalize_ms = ev[1].elapsed_time(ev[2])
    ms_per_step = (t1 - t0) * 1e3 / args.steps
    tt = terms.cpu().numpy()

    # per-step model units of each kernel (effective rates only)
    E = prob.n_edges
    units = {"poly": (census["ops"] * (D - 1), census["edges"] * (D - 1)),
             "ops": ((B * N - census["ops"]) * (D - 1), (B * E - census["edges"]) * (D - 1))}
    kern = {}
    for k, (tot_ms, n) in ktimes.items():
        if n == 0:
            continue
        kms = tot_ms / n
        fl = per_step_model_flops(*units[k])
        kern[KERNEL_NAMES[k]] = {"ms": kms, "launches": n, "op_bin_edges": units[k][0],
                                 "edge_steps": units[k][1],
                                 "per_step_model_tflops_per_s": fl / (kms * 1e-3) / 1e12}
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
    kms = kern[dom]["ms"]
    if dom == "k_poly":
        shifted = float(np.mean(np.asarray(prob.delay) != 1))
        fma, trans = poly_model(tier_census, grids, shifted)
        flops = 2.0 * (fma + TRANS_SLOTS * trans)
        achieved = flops / (kms * 1e-3) / 1e12
        roofline = {"bound": "alu", "achieved": achieved, "peak": PEAK_TFLOPS, "unit": "TFLOP/s",
                    "frac": achieved / PEAK_TFLOPS, "traffic": pmc_traffic(dom, profile),
                    "kernel": dom, "kernel_ms": kms,
                    "work_per_launch": {"fma": fma, "transcendental": trans, "flops": flops,
                                        "ops_by_grid_tier": tier_census.tolist()},
                    "model": "chunk-polynomial work of the method's sums per (restart, op, chunk) and "
                             "(restart, edge, chunk) at each op's series degree, plus the strip steps; "
                             "a transcendental = 4 FMA slots, 2 flops per slot"}
    else:
        n_ops_k = B * N - census["ops"]
        n_edges_k = B * E - census["edges"]
        alg = (n_ops_k * OPS_BYTES_PER_OP + n_edges_k * OPS_BYTES_PER_EDGE + B * prob.n_types * D *
               OPS_BYTES_PER_USAGE + 16 * N + 4 * E)
        achieved = alg / (kms * 1e-3) / 1e9
        roofline = {"bound": "hbm", "achieved": achieved, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                    "frac": achieved / PEAK_HBM_GBS, "traffic": pmc_traffic(dom, profile),
                    "kernel": dom, "kernel_ms": kms, "algorithmic_bytes_per_launch": alg,
                    "model": "per (restart, op) 24 B, per (restart, edge) 24 B, per (restart, type, step) 4 B, "
                             "graph 16 B per op + 4 B per edge"}
    whole = per_step_model_flops(B * N * (D - 1), B * (E + prob.n_back) * (D - 1))
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
        "kernel_timing_every": max(1, args.kernel_timing_every),
        "poly_path": dict(poly_cfg, ops=census["ops"], edges=census["edges"], grids=grids),
        "solve": solve_stats,
        "roofline": roofline,
        "issue": pmc_issue(dom, profile, kms),
        "kernels": kern,
        "per_step_model_tflops_per_s": {
            "iteration": whole / (step_ms_events * 1e-3) / 1e12,
            "note": "20 FMA + 2 transcendentals per op-bin-edge and 10 FMA per edge-step over B*N*(D-1) and "
                    "B*(E+E_B)*(D-1) units: an effective rate of the per-step formulation, not a roofline"},
    }
    if not args.no_cpu_baseline:
        log(f"[bench] CPU oracle for at least {args.cpu_seconds:g} s")
        out["cpu_baseline"] = cpu_baseline(prob, mu0, sg0, lam0, hp, args.cpu_seconds, args.cpu_single_ops, cfg)
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
