"""Throughput of the Spectral-LSH hot path on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload qwen7b_exact] [--no-cpu-baseline]

A step is one pass of the whole path over one prompt already resident in HBM:
feature map -> Lanczos (all steps) -> eigensolve + Ritz -> SimHash -> merge
(plus routing for the windowed adaptive workload).  The default workload is the
Qwen2.5-7B-shaped prompt (N=8192, D=3584) compressed to exactly N / 16 = 512
macro-tokens (rho = 16 with the exact-length adjustment).  Prints one JSON line.
"""
import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "compressed prompt tokens/sec at N=8192,D=3584,ρ=16; Lanczos matvec HBM GB/s"
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
BF16_PEAK_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
INFINITY_CACHE_BYTES = 256 * 2**20   # MI355X last-level (MALL) cache


PASS_REPS = 96                   # graph replays of the last step's pass over Phi


def measured_traffic(wl, resident):
    """HBM bytes per launch of the dominant Lanczos kernel from the committed
    counter summary: per pass of k_lz_step, or per run of k_lz_resident, if the
    summary was taken on the current kernel source and on this shape (one window
    of N=8192, m=2048, 96 steps); else None."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "lanczos_passes_qwen7b_traffic.md")
    src, key = (("k_lzres.hip", "traffic_bytes_per_run") if resident
                else ("k_lanczos.hip", "traffic_bytes_per_pass"))
    if (wl.N, wl.m, wl.n_it, wl.window) != (8192, 2048, 96, 0) or not os.path.exists(path):
        return None
    fields = {}
    for line in open(path):
        if ":" in line and not line.startswith(("|", "`", " ")):
            k, _, v = line.partition(":")
            fields[k.strip()] = v.strip()
    cur = hashlib.sha256(open(os.path.join(ROOT, "paper_2607_19368_amd", "csrc", src), "rb")
                         .read()).hexdigest()
    dev = hashlib.sha256(open(os.path.join(ROOT, "paper_2607_19368_amd", "csrc", "slh_device.h"),
                              "rb").read()).hexdigest()
    if (fields.get(src + " sha256") != cur or fields.get("slh_device.h sha256") != dev
            or key not in fields):
        return None
    return float(fields[key])


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="qwen7b_exact")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--timing", type=int, default=1, help="record per-stage HIP events")
    ap.add_argument("--resident", type=int, default=1,
                    help="SLH_OPT_RESIDENT: 1 lets a window whose Phi fits in the register files "
                         "run the whole Lanczos loop as one persistent kernel")
    return ap.parse_args()


def cpu_baseline(inp, min_seconds=10.0, max_reps=40, tau=None):
    """The oracle, untouched, on the same prompt: feature map .. merge (parameter
    drawing excluded, as on the GPU side where it happens in slh_create), repeated
    until about min_seconds of CPU work have been timed."""
    import numpy as np
    from oracle import params as OP
    from oracle import spectral_lsh as O
    blas = None
    try:
        from threadpoolctl import threadpool_info
        info = [d for d in threadpool_info() if d.get("user_api") == "blas"] or threadpool_info()
        cores = max((d.get("num_threads", 1) for d in info), default=1)
        if info:
            blas = f"{info[0].get('internal_api')} {info[0].get('version')}"
    except Exception:
        cores = len(os.sched_getaffinity(0))
    wl = inp.workload
    L = wl.window or wl.N
    W = OP.projection(0, wl.D, wl.m)
    psi = OP.phases(0, wl.m)
    R = OP.hyperplanes(0, wl.r, wl.bits)
    q1 = [OP.start_vector(0, L, w) for w in range(wl.N // L)]
    times = []
    stage = {k: 0.0 for k in ("route_chunk", "feature_map", "lanczos", "eigh_ritz", "simhash",
                              "merge", "adjust")}
    while len(times) < 2 or (sum(times) < min_seconds and len(times) < max_reps):
        t0 = time.perf_counter()
        for w in range(wl.N // L):
            ta = time.perf_counter()
            Xw = inp.x_float(slice(w * L, (w + 1) * L))
            if wl.adaptive and not O.route_window(L, O.redundancy_score(Xw), wl.rho, tau):
                O.chunk_pool(Xw, O.chunk_size(wl.rho), pos0=w * L)
                stage["route_chunk"] += time.perf_counter() - ta
                continue
            tb = time.perf_counter()
            Phi = O.feature_map(Xw, W, psi)
            if wl.normalise:
                Phi, _ = O.normalised_features(Phi)
            tc = time.perf_counter()
            lz = O.lanczos(Phi, q1[w], wl.n_it)
            td = time.perf_counter()
            _, Z, _, _ = O.ritz(lz, wl.r)
            te = time.perf_counter()
            codes = O.simhash(Z, R)
            tf = time.perf_counter()
            mg = O.merge(Xw, codes, positions=w * L + np.arange(L))
            tg = time.perf_counter()
            if wl.target and not wl.adaptive:
                O.merge_groups(Xw, O.adjust_to_target(mg.members, wl.target),
                               positions=w * L + np.arange(L))
            th = time.perf_counter()
            for k, (u, v) in zip(("route_chunk", "feature_map", "lanczos", "eigh_ritz", "simhash",
                                  "merge", "adjust"),
                                 ((ta, tb), (tb, tc), (tc, td), (td, te), (te, tf), (tf, tg), (tg, th))):
                stage[k] += v - u
        times.append(time.perf_counter() - t0)
    t = sum(times) / len(times)
    return {"value": wl.N / t, "unit": "tokens/s", "cores": int(cores), "kind": "oracle",
            "sample": f"the full {wl.name} prompt ({wl.N} tokens), feature map through merge"
                      + (" and the exact-length adjustment" if wl.target and not wl.adaptive else "")
                      + f", {len(times)} runs in {sum(times):.1f} s ({t:.2f} s each)",
            "seconds": t, "blas": blas,
            "stage_seconds": {k: v / len(times) for k, v in stage.items() if v > 0}}


def main():
    a = parse()
    if a.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py: the hot path runs on one GPU; multi-GPU sharding is not "
              "implemented, use --gpus 1", file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch
    import paper_2607_19368_amd as P
    from paper_2607_19368_amd import slh as B
    from workloads import make_inputs

    P.load()                                   # fails loudly if libslh.so is missing
    torch.cuda.set_device(0)
    inp = make_inputs(a.workload)
    wl = inp.workload
    L = wl.window or wl.N
    X = torch.from_numpy(inp.X.view(np.int16).copy()).view(torch.bfloat16).cuda() \
        if wl.x_dtype == "bf16" else torch.from_numpy(inp.X).cuda()

    ctx = P.slh_create(wl.N, wl.D, wl.m, wl.r, wl.bits, 0)
    if not a.resident:
        P.slh_set_option(ctx, B.SLH_OPT_RESIDENT, 0)
    if wl.keep_last:
        P.slh_set_option(ctx, B.SLH_OPT_KEEP_LAST, wl.keep_last)
    if wl.window:
        P.slh_set_option(ctx, B.SLH_OPT_WINDOW_LEN, wl.window)
    if wl.normalise:
        P.slh_set_option(ctx, B.SLH_OPT_NORMALIZE, 1)
    if wl.target:
        P.slh_set_option(ctx, B.SLH_OPT_TARGET_LEN, wl.target)
    tau = -1.0
    if wl.adaptive:
        # routing threshold: midpoint of the 32nd and 33rd largest window scores
        _, sc = P.slh_route(ctx, X, wl.rho, -1.0)
        s = np.sort(sc)[::-1]
        tau = 0.5 * (s[31] + s[32])
    cap = P.slh_merge_capacity(ctx) if not wl.window else wl.N
    if wl.adaptive and wl.target:
        P.slh_route(ctx, X, wl.rho, tau)           # budgets follow this routing
        cap = max(cap, P.slh_merge_capacity(ctx))
    # two sets of merge outputs: a step's merge is still running while the next
    # step is enqueued
    outs = [(torch.empty((cap, wl.D), dtype=torch.float32, device="cuda"),
             torch.empty(cap, dtype=torch.int32, device="cuda"),
             torch.empty(wl.N, dtype=torch.int32, device="cuda")) for _ in range(2)]

    def enqueue(k):
        if wl.adaptive:
            P.slh_route(ctx, X, wl.rho, tau)
        P.slh_feature_map(ctx, X)
        P.slh_lanczos(ctx, wl.n_it, want=False)
        P.slh_simhash(ctx)
        P.slh_merge_async(ctx, X, *outs[k & 1])

    def step():
        E, Pp, T2M = outs[0]
        if wl.adaptive:
            P.slh_route(ctx, X, wl.rho, tau)
        P.slh_feature_map(ctx, X)
        P.slh_lanczos(ctx, wl.n_it, want=False)
        P.slh_simhash(ctx)
        return P.slh_merge(ctx, X, E, Pp, T2M)[3]

    # timed region 1: the production path (Lanczos loop replayed as one HIP
    # graph).  Each step ends in a merge whose M the host reads; the host
    # enqueues step k + 1 before it waits for step k's M (slh_merge_async /
    # slh_merge_wait), so the GPU does not sit idle while the host returns from
    # one step and launches the next.  The intervals between the waits time the
    # steps.
    for k in range(a.warmup):
        enqueue(k)
        if k:
            M = P.slh_merge_wait(ctx)
    if a.warmup:
        M = P.slh_merge_wait(ctx)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    marks = [t0]
    for k in range(a.steps):
        enqueue(k)
        if k:
            M = P.slh_merge_wait(ctx)
            marks.append(time.perf_counter())
    M = P.slh_merge_wait(ctx)
    marks.append(time.perf_counter())
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    step_ms = [1e3 * (v - u) for u, v in zip(marks[:-1], marks[1:])]
    ms_per_step = 1e3 * dt / a.steps
    value = wl.N * a.steps / dt

    # timed region 2: the same steps with HIP events around every stage; the passes
    # over Phi are launched without the graph, each receiving its own kernel start /
    # end timestamps
    stage_sum = {k: 0.0 for k in B.STAGE_NAMES}
    ms2 = None
    if a.timing:
        P.slh_set_option(ctx, B.SLH_OPT_TIMING, 1)
        for _ in range(2):
            step()
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        for _ in range(a.steps):
            step()
            st = P.slh_stage_times(ctx)
            for k in stage_sum:
                stage_sum[k] += st[k]
        torch.cuda.synchronize()
        ms2 = 1e3 * (time.perf_counter() - t1) / a.steps

    out = {
        "metric": METRIC, "value": value, "unit": "tokens/s", "n_gpus": 1, "steps": a.steps,
        "warmup": a.warmup, "ms_per_step": ms_per_step, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f64",
        "data": "synthetic",
        "config": {
            "workload": f"{wl.name}: N={wl.N} D={wl.D} m={wl.m} n_it={wl.n_it} r={wl.r} "
                        f"bits={wl.bits} rho={wl.rho:g}" + (f" window={wl.window}" if wl.window else "")
                        + (" operator=row-normalised" if wl.normalise else "")
                        + (f" keep_last={wl.keep_last}" if wl.keep_last else "")
                        + (f" target={wl.target}" if wl.target else ""),
            "inputs": "Zipf(1.1) token ids over a seeded N(0,0.02) bf16 embedding table"
                      if wl.x_dtype == "bf16" else "seeded Gaussian mixture, fp32",
            "precision": "bf16 MFMA feature map with fp32 accumulation, fp32 Phi, fp64 Lanczos/"
                         "eigensolve/Ritz/SimHash, fp32 merge sums",
            "M": int(M), "rho_achieved": wl.N / max(1, int(M)),
        },
        "step_ms": {"median": float(np.median(step_ms)), "p10": float(np.percentile(step_ms, 10)),
                    "p90": float(np.percentile(step_ms, 90)), "n": len(step_ms)},
    }
    # measured ceilings, in the same job: a plain read of 1 GiB (four times the
    # Infinity Cache: HBM), a plain read of a buffer the size of Phi read over
    # and over (what the cache serves a buffer that fits in it), and a
    # register-only bf16 MFMA loop
    peaks = None
    if a.timing:
        phi_bytes = ctx.n_spectral * L * wl.m * 4
        big = torch.empty(2**30, dtype=torch.uint8, device="cuda")
        hbm = P.slh_peak_read(big, reps=10)
        small = big[:max(4096, (phi_bytes // 16) * 16)]
        cached = P.slh_peak_read(small, reps=50)
        del big, small
        mf = P.slh_peak_mfma(reps=5)
        peaks = {"read_1GiB_gbs": hbm, "read_phi_sized_gbs": cached, "mfma_bf16_tflops": mf,
                 "phi_bytes": phi_bytes,
                 "phi_fits_infinity_cache": bool(phi_bytes <= INFINITY_CACHE_BYTES)}
        out["measured_peaks"] = peaks
    if a.timing:
        K = a.steps
        n_win = ctx.n_spectral
        fm_ms = stage_sum["featmap_ms"] / K
        flops = 2.0 * n_win * L * wl.D * wl.m
        fm_tf = flops / (fm_ms * 1e-3) / 1e12
        out["featmap_mfma"] = {"bound": "mfma", "achieved": fm_tf, "peak": BF16_PEAK_TFLOPS,
                               "unit": "TFLOP/s", "frac": fm_tf / BF16_PEAK_TFLOPS,
                               "avg_launch_ms": fm_ms, "peak_measured": peaks["mfma_bf16_tflops"],
                               "frac_of_measured": fm_tf / peaks["mfma_bf16_tflops"]}
        out["stages_ms"] = {k: v / K for k, v in stage_sum.items() if k != "phi_pass_count"}
        out["stages_ms"]["ms_per_step_with_events"] = ms2
        if stage_sum["lanczos_resident"] > 0:
            # the resident kernel: one launch per run, all n_it steps; its duration
            # from slh_time_passes (PASS_REPS runs, each kernel between two events)
            run_ms = 1e-3 * P.slh_time_passes(ctx, PASS_REPS) * wl.n_it
            ev_ms = stage_sum["phi_pass_ms_sum"] / K
            # algorithmic bytes of the run: the matvec of every step j as the
            # streaming pass would move them (Phi once, t_j, Q_{j-1} and z1 in, q_j
            # and z1 out), 4 L m + 8 m + 8 L (j + 3), summed over j < n_it; the
            # kernel reads Phi from HBM once and keeps it in registers
            alg = n_win * sum(4.0 * L * wl.m + 8.0 * wl.m + 8.0 * L * (j + 3) for j in range(wl.n_it))
            ach = alg / (run_ms * 1e-3) / 1e9
            out["roofline"] = {"bound": "hbm", "achieved": ach, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                               "frac": ach / HBM_PEAK_GBS, "traffic": measured_traffic(wl, True),
                               "peak_measured_hbm_read": peaks["read_1GiB_gbs"],
                               "frac_of_measured_hbm_read": ach / peaks["read_1GiB_gbs"],
                               "peak_measured_phi_sized_read": peaks["read_phi_sized_gbs"],
                               "frac_of_measured_phi_sized_read": ach / peaks["read_phi_sized_gbs"],
                               "phi_fits_infinity_cache": peaks["phi_fits_infinity_cache"],
                               "traffic_unit": "HBM bytes per run (FETCH_SIZE + WRITE_SIZE, "
                                               "copy-calibrated; profiles/lanczos_passes_qwen7b_traffic.md)",
                               "kernel": "k_lz_resident (the whole Lanczos loop as one persistent "
                                         "kernel: rows of Phi held in registers, blocks exchanging "
                                         "step-tagged partial sums)",
                               "passes_per_step": 1,
                               "form": "resident: Phi read from HBM once per run; each step's matvec "
                                       "takes it from registers. achieved = the algorithmic bytes of "
                                       "every step's matvec over the kernel's duration",
                               "bytes_per_launch": alg, "avg_launch_ms": run_ms,
                               "steps_per_launch": wl.n_it,
                               "timing": f"slh_time_passes: {PASS_REPS} runs of the kernel, each "
                                         "between two events, the first excluded",
                               "avg_launch_ms_events": ev_ms,
                               "frac_events": alg / (ev_ms * 1e-3) / 1e9 / HBM_PEAK_GBS}
            out["stages_ms"]["lanczos_kernel_ms"] = ev_ms
        elif stage_sum["phi_pass_count"] > 0:
            ev_ms = stage_sum["phi_pass_ms_sum"] / stage_sum["phi_pass_count"]
            # the kernel duration: the last step's pass replayed PASS_REPS times as
            # one HIP graph between two events on the context stream (the per-launch
            # event pairs above add a dispatch overhead that varies by machine)
            pass_ms = 1e-3 * P.slh_time_passes(ctx, PASS_REPS)
            # algorithmic bytes of the pass of step j (both halves of the implicit
            # matvec of Eq. 4 on one read of Phi, plus the full re-orthogonalisation),
            # per window: Phi (4 B/elt), t_j in (fp64 m-vector), Q_{j-1} and z1 of
            # step j-1 in, q_j and z1 out (fp64 L-vectors): 4 L m + 8 m + 8 L (j + 3);
            # the replayed step is the last, j = n_it - 1
            j_last = wl.n_it - 1
            alg = n_win * (4.0 * L * wl.m + 8.0 * wl.m + 8.0 * L * (j_last + 3))
            ach = alg / (pass_ms * 1e-3) / 1e9
            out["roofline"] = {"bound": "hbm", "achieved": ach, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                               "frac": ach / HBM_PEAK_GBS, "traffic": measured_traffic(wl, False),
                               "peak_measured_hbm_read": peaks["read_1GiB_gbs"],
                               "frac_of_measured_hbm_read": ach / peaks["read_1GiB_gbs"],
                               "peak_measured_phi_sized_read": peaks["read_phi_sized_gbs"],
                               "frac_of_measured_phi_sized_read": ach / peaks["read_phi_sized_gbs"],
                               "phi_fits_infinity_cache": peaks["phi_fits_infinity_cache"],
                               "traffic_unit": "HBM bytes per pass (FETCH_SIZE + WRITE_SIZE, "
                                               "copy-calibrated; profiles/lanczos_passes_qwen7b_traffic.md)",
                               "kernel": "k_lz_step (u = Phi t_j, z1, Phi^T z1 partials, h2 partials)",
                               "passes_per_step": 1,
                               "form": "fused: one read of Phi per Lanczos step serves both products "
                                       "of the implicit matvec",
                               "bytes_per_launch": alg, "avg_launch_ms": pass_ms,
                               "timing": f"slh_time_passes: {PASS_REPS} x the pass of the last step "
                                         "as one HIP graph between two events",
                               "avg_launch_ms_events": ev_ms,
                               "frac_events": alg / (ev_ms * 1e-3) / 1e9 / HBM_PEAK_GBS}
            out["stages_ms"]["phi_pass_avg_ms"] = ev_ms
        else:
            # short windows: one launch runs Lanczos, Eigh and Ritz of every window.
            # Algorithmic bytes: Phi once, plus the basis, Ritz coordinates,
            # alpha/beta/theta and the start vector, fp64, per window
            lz_ms = stage_sum["lanczos_ms"] / K
            alg = n_win * (4.0 * L * wl.m + 8.0 * ((wl.n_it + 1) * L + L * wl.r + L
                                                   + 2 * wl.n_it + wl.r))
            ach = alg / (lz_ms * 1e-3) / 1e9
            loc = {"bound": "hbm", "achieved": ach, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                   "frac": ach / HBM_PEAK_GBS, "traffic": None,
                   "kernel": "k_local (Lanczos + Eigh + Ritz, one wavefront per window; "
                             "a serial chain of n_it dependent steps per window)",
                   "bytes_per_launch": alg, "avg_launch_ms": lz_ms}
            out["local_kernel"] = loc
            if lz_ms >= fm_ms:
                out["roofline"] = loc
            else:
                out["roofline"] = dict(out["featmap_mfma"], traffic=None,
                                       kernel="k_featmap (bf16 MFMA GEMM + cos epilogue)")
    # diagnostics of the last step (outside the timed regions): spectral-energy
    # fraction of the kept Ritz values and bucket purity (section 5 kill tests)
    if ctx.n_spectral:
        t0 = time.perf_counter()
        en = P.slh_spectral_energy(ctx)
        t1 = time.perf_counter()
        sim, tot = P.slh_bucket_purity(ctx, X, 0.7)
        t2 = time.perf_counter()
        out["diagnostics"] = {
            "spectral_energy_mean": float(np.mean(en)), "spectral_energy_min": float(np.min(en)),
            "bucket_purity": (sim / tot) if tot else None, "same_bucket_pairs": tot,
            "energy_ms": 1e3 * (t1 - t0), "purity_ms": 1e3 * (t2 - t1)}
    if not a.no_cpu_baseline:
        cb = cpu_baseline(inp, tau=tau if wl.adaptive else None)
        out["cpu_baseline"] = {k: cb[k] for k in ("value", "unit", "cores", "kind", "sample", "blas",
                                                  "stage_seconds")}
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
