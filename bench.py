"""Throughput of the multi-draft selection hot path on one MI355X.

One step = the whole path over one batch resident in HBM: induced distribution
r (K drafts), importance-weighted selection, accept / resample (Algorithm 1).
Default workload: V = 32000, K = 2, 256 positions of LLM-shaped synthetic
distributions.  Prints ONE JSON line.

  python bench.py [--gpus 1] [--steps K] [--warmup W] [--config llm32k] [--no-cpu]
"""
from __future__ import annotations

import argparse
import dataclasses
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

FP32_PEAK_TFLOPS = 157.3  # MI355X fp32 vector peak (packed FMA: 4 FLOP per lane and cycle)
FP32_NONPACKED_TFLOPS = 256 * 4 * 16 * 2 * 2.4e9 / 1e12  # 78.6: one FMA per lane and cycle (packed fp32 is not built)
HBM_PEAK_GBS = 8000.0     # MI355X HBM3E
R_REPS = 10               # r calls per graph in the r timing
# fp32 VALU issue without packed math: 256 CUs x 4 SIMDs x 16 lanes x 2.4 GHz = 39.3 T lane-instructions/s
ES_PEAK_SLOTS = 256 * 4 * 16 * 2.4e9
# Least work of the truncated quadrature per positive-weight token and law: the moments
# evaluate the nine nodes with a w in (1/4, 22.5] (mul, exp, fma) and an 8-term expansion
# for the nodes below (power sums: mul + add per term); the evaluation takes a token's
# nine node terms and its expansion as one degree-10 polynomial in a_k0 w (the map to t
# and ten fma).  In FLOP (fma 2, mul / add / exp 1): 9 * 4 + 8 * 2 + 2 + 10 * 2 = 74.
# In issue slots (exp takes two): 9 * 4 + 8 * 2 + 1 + 10 = 63.
ES_FLOPS_PER_TOKEN = 9 * 4 + 8 * 2 + 2 + 10 * 2
ES_SLOTS_PER_TOKEN = 9 * 4 + 8 * 2 + 11
METRIC = "positions/sec (V=32000, K=2) + % FP32 VALU peak (r) / % HBM BW (resample)"


def kernel_source_digest() -> str:
    """Digest of the device code and its build flags (the host-side argument checks
    of api.hip are left out: they launch nothing)."""
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2410_18234_amd", "csrc")
    files = sorted(f for f in os.listdir(csrc) if f.endswith((".h", ".hip")) and f != "api.hip")
    for f in [os.path.join("csrc", f) for f in files] + ["build.py"]:
        with open(os.path.join(ROOT, "paper_2410_18234_amd", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def counted_traffic(workload: str, kernels, digest: str):
    """HBM bytes per launch of a call (the sum over its kernels) from the committed PMC
    summary of this workload, only if every figure was taken on the current kernel
    sources (else None)."""
    path = os.path.join(ROOT, "profiles", "pmc_traffic.json")
    try:
        with open(path) as fh:
            d = json.load(fh)
    except (OSError, ValueError):
        return None
    total = 0
    for kernel in ([kernels] if isinstance(kernels, str) else kernels):
        e = d.get(workload, {}).get(kernel)
        if not e or e.get("source_digest") != digest:
            return None
        total += e.get("bytes_per_launch")
    return total


def pair_flops(q_np, K: int, q2_np=None) -> float:
    """Algorithmic work of r: K = 2: 6 FLOPs per unordered support pair (add,
    reciprocal, two FMAs) = 3 n (n - 1) per row; K = 3: 4 FLOPs per (query,
    unordered pair) = 2 n^2 (n + 1) per row.  Two drafts from different
    distributions: one denominator w1(y) + w2(x) per (y, x) in supp(q1) x
    supp(q2) serves both sums, 6 FLOPs each = 6 n1 n2 per row."""
    import numpy as np
    n = (q_np > 0).sum(1).astype(np.float64)
    if q2_np is not None:
        return float((6.0 * n * (q2_np > 0).sum(1)).sum())
    if K == 2:
        return float((3.0 * n * (n - 1.0)).sum())
    return float((2.0 * n * n * (n + 1.0)).sum())


def cpu_tlp_step(p, q1, q2, drafts, u, s, tail):
    """The truncated-LP path by the oracle: plan per row, selection, Algorithm 1."""
    import numpy as np

    import oracle
    from oracle import tlp
    B, V = p.shape
    r = np.empty((B, V), np.float32)
    om = np.full((B, s), -1, np.int32)
    betas = np.zeros((B, s, s))
    for b in range(B):
        res = tlp.plan_row(p[b], q1[b], None if q2 is None else q2[b], s=s, tail=tail)
        r[b] = res["r"].astype(np.float32)
        om[b, :len(res["omega1"])] = res["omega1"]
        betas[b, :len(res["omega1"]), :len(res["omega1"])] = res["beta"]
    _, stok, _ = tlp.select(p, q1, q2, drafts, u, om, betas, tail)
    return oracle.accept_resample(p, r, stok, u)


def expsum_evals(p_np, q_np, K: int, q2_np=None) -> float:
    """Nominal work of the exponential-sum r: every positive-weight token of a row
    meets every node of the row's grid once in the moments and once in the
    evaluation.  The grid (step 1/2 in t = ln a) spans from ln 1e-8 - ln D_max
    to ln ln 1e8 - ln D_min, D the denominators of the row (K i.i.d. drafts:
    K w_min (w_min alone when K >= 3 and some token has p = 0 < q) to K w_max;
    two laws: w1_min + w2_min to w1_max + w2_max)."""
    import math

    import numpy as np
    p64 = p_np.astype(np.float64)
    laws = [q_np] if q2_np is None else [q_np, q2_np]
    total = 0.0
    for b in range(p64.shape[0]):
        pos, wmin, wmax = [], [], []
        for qq in laws:
            q64 = qq[b].astype(np.float64)
            m = (q64 > 0) & (p64[b] > 0)
            pos.append(int(m.sum()))
            w = p64[b][m] / q64[m]
            wmin.append(w.min() if w.size else math.inf)
            wmax.append(w.max() if w.size else 0.0)
        if min(pos) == 0:
            continue
        if q2_np is None:
            q0 = float(q_np[b].astype(np.float64)[(q_np[b] > 0) & (p64[b] == 0)].sum())
            dmin = K * wmin[0] if (K == 2 or q0 == 0.0) else wmin[0]
            dmax = K * wmax[0]
        else:
            dmin, dmax = wmin[0] + wmin[1], wmax[0] + wmax[1]
        nk = math.ceil((math.log(math.log(1e8)) - math.log(dmin)) / 0.5) - \
            math.floor((math.log(1e-8) - math.log(dmax)) / 0.5) + 1
        total += 2.0 * sum(pos) * nk
    return total


def expsum_positive_tokens(p_np, q_np, q2_np=None, stages: int = 1) -> float:
    """Positive-weight tokens the quadrature takes (each law; successive stages: stage 1
    on q, each later stage on (r_(j-1), q), counted with q's support twice)."""
    import numpy as np
    pos = lambda qq: float(((p_np > 0) & (qq > 0)).sum())
    n1 = pos(q_np)
    total = n1 + (pos(q2_np) if q2_np is not None else 0.0)
    return total + (stages - 1) * 2.0 * n1


def succ_flops(q_np, K: int) -> float:
    """Successive pairwise selection: stage 1 is the K = 2 pair sum (3 n (n - 1)),
    each later stage a two-law pair sum over supp(r_{j-1}) x supp(q) = n x n (6 n^2)."""
    import numpy as np
    n = (q_np > 0).sum(1).astype(np.float64)
    return float((3.0 * n * (n - 1.0) + (K - 2) * 6.0 * n * n).sum())


def cpu_baseline(w, budget_rows: int):
    """The fp64 oracle (as it stands) on the first rows of the same workload."""
    import numpy as np

    import oracle
    cfg = w["config"]
    rows = min(budget_rows, w["p"].shape[0])
    p, q, d, u = (np.ascontiguousarray(w[k][:rows]) for k in ("p", "q", "drafts", "u"))
    q2 = np.ascontiguousarray(w["q2"][:rows]) if "q2" in w else None
    oracle.step(p[:1, :64], q[:1, :64], d[:1], u[:1])  # load the library outside the timing
    t0 = time.perf_counter()
    if cfg.alphabet:
        from oracle import alphabet
        pt, mass, inside = alphabet.truncate(p, cfg.alphabet)
        res = oracle.step(pt, q, d, u)
        alphabet.post(p, inside, mass, res["out_token"], np.ascontiguousarray(u[:, ::-1][:, :2]))  # timing only
    elif cfg.diag:
        from oracle import optimum
        for b in range(rows):
            optimum.prefix_optimum(p[b], q[b], 2)
        optimum.achieved(p, q)  # the proposal is an input of the step; any fp32 law costs the same
    elif cfg.tlp_s:
        cpu_tlp_step(p, q, q2, d, u, cfg.tlp_s, cfg.tlp_tail)
    elif cfg.successive:
        from oracle import successive
        successive.step(p, q, d, np.ascontiguousarray(u[:, :1].repeat(d.shape[1] - 1, 1)), u)
    elif q2 is not None:
        oracle.step_pair(p, q, q2, d, u)
    else:
        oracle.step(p, q, d, u)
    dt = time.perf_counter() - t0
    cores = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
    if cfg.alphabet:
        cores = min(cores, os.cpu_count() or cores, rows)
        what = ("truncation to Omega_0, r of the truncated target by enumeration of all ordered draft pairs, "
                "selection, accept/resample, post-processing")
    elif cfg.diag:
        cores = 1
        what = "P* by the prefix form (numpy sort and cumulative sums) and the acceptance sum per position"
    elif cfg.tlp_s:
        cores = 1  # numpy ranking and a HiGHS LP per position, one thread
        what = "truncated LP per position (numpy ranking, HiGHS LP), selection, accept/resample"
    elif cfg.successive:
        cores = min(cores, os.cpu_count() or cores, rows)
        what = "stage laws by enumeration of ordered pairs per stage, chained selection, accept/resample"
    else:
        cores = min(cores, os.cpu_count() or cores, rows)
        what = "r by enumeration of all ordered draft pairs, selection, accept/resample"
    return {"value": rows / dt, "unit": "positions/s", "cores": cores, "kind": "oracle",
            "sample": f"first {rows} positions of the same workload, whole path ({what}), {dt:.1f} s wall"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default="llm32k")
    ap.add_argument("--no-cpu", action="store_true", help="skip the oracle baseline leg")
    ap.add_argument("--no-graph", action="store_true", help="time eager launches instead of graph replays")
    ap.add_argument("--graph-steps", type=int, default=10,
                    help="steps captured back to back in each HIP graph (each graph launch leaves the GPU idle "
                         "for ~8 us; a serving loop captures the sampler inside its decode graph)")
    ap.add_argument("--cpu-rows", type=int, default=0, help="oracle sample size (0: one per core, 2 rounds)")
    ap.add_argument("--resample-reps", type=int, default=20)
    ap.add_argument("--tlp-tail", choices=["sorted", "half"], default=None,
                    help="truncated-LP workloads: Omega_2 sorted (Algorithm 2) or halves (its sort-free variant)")
    ap.add_argument("--method", choices=["expsum", "exact"], default="expsum",
                    help="induced distribution: exponential-sum quadrature (O(n) per node) or the exact pairwise "
                         "sums (O(n^2) for K=2, O(n^3) for K=3); the truncated LP, alphabet and optimum workloads "
                         "keep their own paths")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run one plain 256 MiB device copy (reference for HBM byte counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}); positions are independent, "
              "so several GPUs would each take a share of the rows with no exchange; run it with --gpus 1",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2410_18234_amd as mdss
    from workloads import CONFIGS, generate

    cfg = CONFIGS[args.config]
    w = generate(args.config)
    dev = torch.device("cuda:0")
    p = torch.from_numpy(w["p"]).to(dev)
    q = torch.from_numpy(w["q"]).to(dev)
    q2 = torch.from_numpy(w["q2"]).to(dev) if cfg.pair else None
    tlp_s, tail = cfg.tlp_s, cfg.tlp_tail
    if args.tlp_tail is not None:
        tail = 0 if args.tlp_tail == "sorted" else 1
        desc = cfg.describe.replace("sorted Omega_2", "sorted Omega_2" if tail == 0 else "Omega_2 pairs split in halves")
        cfg = dataclasses.replace(cfg, tlp_tail=tail, describe=desc)
        w["config"] = cfg
    if tlp_s:
        omega1 = torch.empty((p.shape[0], tlp_s), dtype=torch.int32, device=dev)
        wtab = torch.empty((p.shape[0], tlp_s, tlp_s), dtype=torch.float64, device=dev)
        acc_prob = torch.empty(p.shape[0], dtype=torch.float64, device=dev)
    drafts = torch.from_numpy(w["drafts"]).to(dev)
    u = torch.from_numpy(w["u"]).to(dev)
    B, V, K = p.shape[0], p.shape[1], cfg.K
    s_max = cfg.s_max
    r = torch.empty_like(p)
    status = torch.zeros(B, dtype=torch.int32, device=dev)
    use_es = args.method == "expsum" and not (tlp_s or cfg.alphabet or cfg.diag)
    # K >= 3 i.i.d. drafts from a top-s draft: the quadrature over each row's support
    use_topk = use_es and K >= 3 and bool(s_max) and not (cfg.successive or cfg.pair)
    # K i.i.d. drafts by the quadrature (tiled or top-s): r and Algorithm 1's residual sums in one pass,
    # then the selection and Algorithm 1 from those sums
    use_sums = use_es and not (cfg.successive or cfg.pair)
    if use_es and (cfg.successive or cfg.pair):
        ws_bytes = mdss.workspace_bytes_pair_expsum(B, V)
        if cfg.successive:
            r_stages = torch.empty((K - 1, B, V), dtype=torch.float32, device=dev)
            r = r_stages[K - 2]
            u_sel = torch.from_numpy(np.ascontiguousarray(w["u"][:, :1].repeat(K - 1, 1))).to(dev)
    elif use_topk:
        ws_bytes = 0  # the top-s call takes no workspace
    elif use_es:
        ws_bytes = mdss.workspace_bytes_expsum(B, V, K)
    elif tlp_s:
        ws_bytes = mdss.workspace_bytes_tlp(B, V, tail)
    elif cfg.successive:
        ws_bytes = mdss.workspace_bytes_successive(B, V)
        r_stages = torch.empty((K - 1, B, V), dtype=torch.float32, device=dev)
        r = r_stages[K - 2]
        u_sel = torch.from_numpy(np.ascontiguousarray(w["u"][:, :1].repeat(K - 1, 1))).to(dev)
    elif cfg.pair:
        ws_bytes = mdss.workspace_bytes_pair(B, V)
    else:
        ws_bytes = mdss.workspace_bytes(B, V, K, s_max)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    ws_acc = torch.empty(mdss.workspace_bytes_accept(B, V), dtype=torch.uint8, device=dev)  # step 2's scratch

    def induced():
        if use_es:
            if cfg.successive:
                mdss.induced_dist_successive_expsum(p, q, K, r_stages=r_stages, row_status=status, workspace=ws)
            elif cfg.pair:
                mdss.induced_dist_pair_expsum(p, q, q2, r=r, row_status=status, workspace=ws)
            elif use_topk:
                mdss.induced_dist_topk_expsum_sums(p, q, K, s_max, ws_acc, r=r, row_status=status)
            elif use_sums:
                mdss.induced_dist_expsum_sums(p, q, K, ws_acc, r=r, row_status=status, workspace=ws)
            else:
                mdss.induced_dist_expsum(p, q, K, r=r, row_status=status, workspace=ws)
        elif tlp_s:
            mdss.truncated_lp(p, q, q2, tlp_s, tail, r=r, omega1=omega1, w=wtab, accept=acc_prob,
                              row_status=status, workspace=ws)
        elif cfg.successive:
            mdss.induced_dist_successive(p, q, K, r_stages=r_stages, row_status=status, workspace=ws)
        elif cfg.pair:
            mdss.induced_dist_pair(p, q, q2, r=r, row_status=status, workspace=ws)
        else:
            mdss.induced_dist(p, q, K, s_max=s_max, r=r, row_status=status, workspace=ws)

    def select():
        if tlp_s:
            return mdss.select_truncated_lp(p, q, q2, drafts, omega1, wtab, tail, u, row_status=status)
        if cfg.successive:
            return mdss.select_successive(p, q, r_stages, drafts, u_sel, row_status=status)
        if cfg.pair:
            return mdss.select_intermediate_pair(p, q, q2, drafts, u, row_status=status)
        return mdss.select_intermediate(p, q, drafts, u, row_status=status)

    if cfg.alphabet:
        pt = torch.empty_like(p)
        mass0 = torch.empty(B, dtype=torch.float64, device=dev)
        u2 = None  # the post-processing draws its own uniforms (a Philox stream apart from Algorithm 1's)
    if cfg.diag:
        # the proposal whose share of the optimum is reported: the importance-weighted r, an input here
        mdss.induced_dist(p, q, K, r=r)
        ws_opt = torch.empty(mdss.workspace_bytes_optimum(B, V), dtype=torch.uint8, device=dev)

    def one_step(ev=None):
        if not use_sums:  # the summed form's r call sets the status words itself
            status.zero_()
        if ev is not None:
            ev[0].record()
        if cfg.alphabet:
            # p~ on the m most probable target tokens, the importance-weighted path with p~, the post-processing
            ptr, m0 = mdss.truncate_alphabet(p, cfg.alphabet, row_status=status)
            mdss.induced_dist(ptr, q, K, r=r, row_status=status, workspace=ws)
            if ev is not None:
                ev[1].record()
            _, sel_token = mdss.select_intermediate(ptr, q, drafts, u, row_status=status)
            z, acc, _, _ = mdss.accept_or_resample(ptr, r, sel_token, u, row_status=status, workspace=ws_acc)
            out, _ = mdss.alphabet_post(p, ptr, m0, z, u2)
            return out, acc
        if cfg.diag:
            pstar, _ = mdss.optimal_acceptance(p, q, 2, row_status=status, workspace=ws_opt)
            achieved = mdss.acceptance(p, r, row_status=status)
            if ev is not None:
                ev[1].record()
            return pstar, achieved
        if use_topk:
            # the top-s step in one launch: r, the residual sums, then the selection and Algorithm 1
            # (the eager events bracket the whole launch; r alone is timed on its own call below)
            _, _, _, out, acc, _ = mdss.step_topk_expsum(p, q, drafts, K, s_max, ws_acc, u, r=r, row_status=status)
            if ev is not None:
                ev[1].record()
            return out, acc
        induced()
        if ev is not None:
            ev[1].record()
        if not (tlp_s or cfg.successive):
            # selection and Algorithm 1 in one launch
            if cfg.pair:
                _, _, out, acc, _, _ = mdss.select_accept_pair(p, q, q2, r, drafts, u, row_status=status,
                                                                workspace=ws_acc)
            elif use_sums:
                _, _, out, acc, _ = mdss.select_accept_sums(p, q, r, drafts, ws_acc, u, row_status=status)
            else:
                _, _, out, acc, _, _ = mdss.select_accept(p, q, r, drafts, u, row_status=status, workspace=ws_acc)
            return out, acc
        _, sel_token = select()
        out, acc, _, _ = mdss.accept_or_resample(p, r, sel_token, u, row_status=status, workspace=ws_acc)
        return out, acc

    if args.copy_calibration:
        src = torch.ones(64 << 20, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    for _ in range(args.warmup):
        one_step()
    torch.cuda.synchronize()
    # r alone: HIP events around the induced-distribution call of eager steps
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        out, acc = one_step(evs[i])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    r_ms = float(np.mean([a.elapsed_time(b) for a, b in evs]))
    r_eager_ms = None
    ms_per_step = wall * 1e3 / args.steps
    ms_one_per_graph = None
    timing = "eager launches, HIP events around r in every step"
    if not args.no_graph:
        # the whole step (status clear, r, selection, accept/resample) in HIP graphs: no host
        # launch work or timing markers between the kernels.  Every graph is checked against
        # the eager step first.
        ref_out, ref_acc = out.clone(), acc.clone()
        ref_r = (r_stages if cfg.successive else r).clone()
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            one_step()
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        # graphs of n whole steps each, back to back on the same inputs (every step recomputes r, the
        # selection and Algorithm 1 from p, q, the drafts and u; the last step's outputs are kept)
        def capture(n):
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                for _ in range(n):
                    o = one_step()
            return g, o

        def check(g, o, what):
            for rep in range(3):
                g.replay()
                torch.cuda.synchronize()
                same = (torch.equal(o[0], ref_out) and torch.equal(o[1], ref_acc) and
                        torch.equal(r_stages if cfg.successive else r, ref_r) and int(status.abs().sum()) == 0)
                assert same, f"{what}: replay {rep} differs from the eager step"
                one_step()  # eager work between the replays
                torch.cuda.synchronize()

        def timed(graphs):
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            for g in graphs:
                g.replay()
            torch.cuda.synchronize()
            return (time.perf_counter() - t0) * 1e3 / args.steps

        # one step per graph: each replay pays the graph launch
        graph1, o1 = capture(1)
        check(graph1, o1, "one-step graph")
        for _ in range(args.warmup):
            graph1.replay()
        ms_one_per_graph = timed([graph1] * args.steps)
        # the timed form: K steps as replays of graphs of --graph-steps steps (a shorter graph for the rest)
        gs = max(1, min(args.graph_steps, args.steps))
        graph, g_o = capture(gs)
        check(graph, g_o, f"{gs}-step graph")
        plan = [graph] * (args.steps // gs)
        if args.steps % gs:
            tail, t_o = capture(args.steps % gs)
            check(tail, t_o, f"{args.steps % gs}-step graph")
            plan.append(tail)
        for _ in range(max(1, args.warmup // gs)):
            graph.replay()
        ms_per_step = timed(plan)
        out, acc = g_o
        del graph1
    if not args.no_graph and not (cfg.alphabet or cfg.diag):
        # r alone without host launch gaps: a graph of R_REPS back-to-back r calls, HIP events around replays
        # (the alphabet and optimum workloads time their own segments of the eager step instead)
        r_graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(r_graph):
            for _ in range(R_REPS):
                induced()
        r_graph.replay()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(args.steps):
            r_graph.replay()
        e1.record()
        torch.cuda.synchronize()
        r_eager_ms = r_ms
        r_ms = e0.elapsed_time(e1) / (args.steps * R_REPS)
        timing = (f"K steps as replays of HIP graphs of {min(args.graph_steps, args.steps)} whole steps each "
                  "(replays checked against the eager step); r by HIP events around replays of a graph of "
                  f"{R_REPS} back-to-back r calls")
    elif not args.no_graph:
        timing = (f"K steps as replays of HIP graphs of {min(args.graph_steps, args.steps)} whole steps each "
                  "(replays checked against the eager step); r by HIP events on eager steps")
    assert int(status.abs().sum()) == 0, "rows flagged during the bench"
    if cfg.diag:
        pstar_t, achieved_t = out, acc
        acc = torch.zeros(1, device=dev)
    accept_rate = float(acc.float().mean())
    # expected acceptance sum_y min(p, r) of the proposal, averaged over positions (measurement only)
    expected_acc = float(torch.minimum(p.double(), r.double()).sum(1).mean())

    digest = kernel_source_digest()
    if cfg.alphabet:
        # HBM-bound: read p (truncation) and p~, q (weights), write p~ and r
        nbytes = float(B) * V * 20
        gbs = nbytes / (r_ms * 1e-3) / 1e9
        roofline = {"bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                    "frac": round(gbs / HBM_PEAK_GBS, 4), "traffic": None,
                    "kernel": "mdss_truncate_alphabet + mdss_induced_dist with the truncated target",
                    "avg_ms": round(r_ms, 4), "bytes_per_launch": nbytes, "alphabet": cfg.alphabet}
    elif cfg.diag:
        # HBM-bound: P* reads p, q; the acceptance reads p, r (8 + 8 B/token)
        nbytes = float(B) * V * 16
        gbs = nbytes / (r_ms * 1e-3) / 1e9
        roofline = {"bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                    "frac": round(gbs / HBM_PEAK_GBS, 4), "traffic": None,
                    "kernel": "mdss_optimal_acceptance (rank_scan_kernel) + mdss_acceptance", "avg_ms": round(r_ms, 4),
                    "bytes_per_launch": nbytes}
    elif tlp_s:
        # HBM-bound: read p, q1 (and q2), write r once
        nbytes = float(B) * V * (16 if cfg.pair else 12)
        gbs = nbytes / (r_ms * 1e-3) / 1e9
        rank_name = "tlp_rank_sorted_kernel" if tail == 0 else "tlp_rank_half_kernel"
        roofline = {"bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                    "frac": round(gbs / HBM_PEAK_GBS, 4), "traffic": counted_traffic(cfg.name, rank_name, digest),
                    "kernel": f"mdss_truncated_lp ({rank_name} + tlp_lp_kernel)", "avg_ms": round(r_ms, 4),
                    "bytes_per_launch": nbytes, "s": tlp_s, "tail": "sorted" if tail == 0 else "half"}
    elif use_topk:
        # HBM-bound by design: one pass reads p and q (8 B/token) and writes r (4 B/token)
        nbytes = float(B) * V * 12
        gbs = nbytes / (r_ms * 1e-3) / 1e9
        ntok = expsum_positive_tokens(w["p"], w["q"])
        roofline = {"bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                    "frac": round(gbs / HBM_PEAK_GBS, 4),
                    "traffic": counted_traffic(cfg.name, ["es_topk_kernel<true, false>"], digest),
                    "kernel": "mdss_induced_dist_topk_expsum_sums (es_topk_kernel<true, false>, with the residual "
                              "sums of Algorithm 1; the step runs es_topk_kernel<true, true>, the same kernel with "
                              "the draw)", "avg_ms": round(r_ms, 4),
                    "bytes_per_launch": nbytes, "byte_basis": "p and q read once (8 B/token), r written once "
                                                             "(4 B/token), every token of the row",
                    "support_tokens_with_weight": ntok}
    elif use_es:
        stages = (K - 1) if cfg.successive else 1
        evals = expsum_evals(w["p"], w["q"], 2 if cfg.successive else K, w.get("q2"))
        if cfg.successive:  # later stages: two laws (the previous stage law, q); counted with q on both sides
            evals += (K - 2) * expsum_evals(w["p"], w["q"], 2, w["q"])
        ntok = expsum_positive_tokens(w["p"], w["q"], w.get("q2"), stages)
        flops = ES_FLOPS_PER_TOKEN * ntok
        slots = ES_SLOTS_PER_TOKEN * ntok
        achieved = flops / (r_ms * 1e-3) / 1e12
        api = ("mdss_induced_dist_successive_expsum" if cfg.successive else
               "mdss_induced_dist_pair_expsum" if cfg.pair else
               "mdss_induced_dist_expsum_sums" if use_sums else "mdss_induced_dist_expsum")
        eval_name = f"es_eval_kernel<{2 if cfg.pair else 1}, {'true' if use_sums else 'false'}>"
        roofline = {"bound": "alu", "achieved": round(achieved, 3), "peak": FP32_PEAK_TFLOPS,
                    "unit": "TFLOP/s", "frac": round(achieved / FP32_PEAK_TFLOPS, 4),
                    "traffic": counted_traffic(cfg.name, ["es_moments_kernel", f"es_coef_kernel<{2 if cfg.pair else 1}>",
                                                          eval_name], digest),
                    "kernel": f"{api} (es_moments_kernel + es_coef_kernel + es_eval_kernel"
                              f"{' with the residual sums of Algorithm 1' if use_sums else ''}"
                              f"{', per stage' if stages > 1 else ''})",
                    "avg_ms": round(r_ms, 4), "flops_per_launch": flops,
                    "flop_basis": f"{ES_FLOPS_PER_TOKEN} FLOP per positive-weight token and law, the least work of "
                                  "the truncated quadrature (moments: 9 node terms of mul, exp, fma and an 8-term "
                                  "expansion; evaluation: one degree-10 polynomial); fma 2, mul / add / exp 1",
                    "frac_of_nonpacked_fp32": round(achieved / FP32_NONPACKED_TFLOPS, 4),
                    "nonpacked_fp32_peak_tflops": round(FP32_NONPACKED_TFLOPS, 1),
                    "issue_slots": {"per_token": ES_SLOTS_PER_TOKEN, "per_launch": slots,
                                    "achieved_per_s": round(slots / (r_ms * 1e-3), 1), "peak_per_s": ES_PEAK_SLOTS,
                                    "frac": round(slots / (r_ms * 1e-3) / ES_PEAK_SLOTS, 4),
                                    "unit": "issue slots/s",
                                    "basis": "fp32 VALU issue without packed math (256 CU x 4 SIMD x 16 lanes x "
                                             "2.4 GHz); v_exp_f32 takes two slots"},
                    "nominal_node_evals": evals,
                    "nominal_node_eval_rate_per_s": round(evals / (r_ms * 1e-3), 1)}
    else:
        flops = succ_flops(w["q"], K) if cfg.successive else pair_flops(w["q"], K, w.get("q2"))
        achieved = flops / (r_ms * 1e-3) / 1e12
        sweep_name = "sweep_k2_mfma_kernel" if K == 2 or cfg.successive else "sweep_k3_kernel"
        roofline = {"bound": "alu", "achieved": round(achieved, 3), "peak": FP32_PEAK_TFLOPS, "unit": "TFLOP/s",
                    "frac": round(achieved / FP32_PEAK_TFLOPS, 4),
                    "traffic": counted_traffic(cfg.name, sweep_name, digest),
                    "kernel": f"{'mdss_induced_dist_successive' if cfg.successive else 'mdss_induced_dist_pair' if cfg.pair else 'mdss_induced_dist'} ({sweep_name} + "
                              "preparation)", "avg_ms": round(r_ms, 4), "flops_per_launch": flops}

    exact_pairwise = None
    if use_es:
        # the pairwise O(n^2) (K=2) / O(n^3) (K=3) sums the quadrature replaces, measured on the same rows
        flops_x = succ_flops(w["q"], K) if cfg.successive else pair_flops(w["q"], K, w.get("q2"))
        if cfg.successive:
            ws_x = torch.empty(mdss.workspace_bytes_successive(B, V), dtype=torch.uint8, device=dev)
            run_x = lambda: mdss.induced_dist_successive(p, q, K, row_status=status, workspace=ws_x)
        elif cfg.pair:
            ws_x = torch.empty(mdss.workspace_bytes_pair(B, V), dtype=torch.uint8, device=dev)
            run_x = lambda: mdss.induced_dist_pair(p, q, q2, row_status=status, workspace=ws_x)
        else:
            ws_x = torch.empty(mdss.workspace_bytes(B, V, K, s_max or 0), dtype=torch.uint8, device=dev)
            run_x = lambda: mdss.induced_dist(p, q, K, s_max=s_max, row_status=status, workspace=ws_x)
        run_x()
        torch.cuda.synchronize()
        xe = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(3)]
        for a, b in xe:
            a.record()
            run_x()
            b.record()
        torch.cuda.synchronize()
        x_ms = float(np.median([a.elapsed_time(b) for a, b in xe]))
        del ws_x
        exact_pairwise = {"avg_ms": round(x_ms, 4), "flops_per_launch": flops_x,
                          "achieved": round(flops_x / (x_ms * 1e-3) / 1e12, 3), "peak": FP32_PEAK_TFLOPS,
                          "unit": "TFLOP/s", "frac": round(flops_x / (x_ms * 1e-3) / 1e12 / FP32_PEAK_TFLOPS, 4),
                          "speedup_of_quadrature": round(x_ms / r_ms, 2),
                          "kernel": "mdss_induced_dist / _pair / _successive (pairwise sums; 6 FLOP per unordered "
                                    "pair, 4 per (query, pair) for K = 3)"}

    # accept / resample pass over every row with the residual written (12 B per token): on
    # the step's own buffers (the 98 MB of llm32k stay in the 256 MB Infinity Cache), and on
    # NC copies of (p, r, residual) taken in turn, so that every launch reads and writes
    # buffers last touched more than 256 MB of traffic ago (the HBM-bound figure)
    _, sel_token = select()
    import ctypes
    lib = mdss.load_library()
    stream = ctypes.c_void_p(torch.cuda.current_stream(dev).cuda_stream)
    res_bytes = 12.0 * B * V
    ncopy = max(2, int(np.ceil(3 * 256e6 / res_bytes)) + 1)  # footprint above three times the cache
    bufs = [(p if i == 0 else p.clone(), r if i == 0 else r.clone(), torch.empty_like(p),
             torch.empty(B, dtype=torch.float64, device=dev), torch.empty(B, dtype=torch.int32, device=dev),
             torch.empty(B, dtype=torch.uint8, device=dev)) for i in range(ncopy)]

    def resample_full(i):
        pp, rr, res, mass, out_t, acc_t = bufs[i]
        rc = lib.mdss_accept_or_resample(ctypes.c_void_p(pp.data_ptr()), ctypes.c_void_p(rr.data_ptr()),
                                         ctypes.c_void_p(sel_token.data_ptr()), ctypes.c_void_p(u.data_ptr()),
                                         ctypes.c_uint64(0), ctypes.c_uint64(0), B, V,
                                         ctypes.c_void_p(out_t.data_ptr()), ctypes.c_void_p(acc_t.data_ptr()),
                                         ctypes.c_void_p(res.data_ptr()), ctypes.c_void_p(mass.data_ptr()), None,
                                         ctypes.c_void_p(ws_acc.data_ptr()), ws_acc.numel(), stream)
        assert rc == 0

    def time_resample(copies, reps):
        for k in range(max(3, len(copies))):
            resample_full(copies[k % len(copies)])
        torch.cuda.synchronize()
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
        for k, (a, b) in enumerate(ev):
            a.record()
            resample_full(copies[k % len(copies)])
            b.record()
        torch.cuda.synchronize()
        return float(np.median([a.elapsed_time(b) for a, b in ev]))

    res_ms_hot = time_resample([0], args.resample_reps)
    res_ms = time_resample(list(range(ncopy)), max(args.resample_reps, 2 * ncopy))
    for i in range(1, ncopy):  # every copy computed the same outputs
        assert torch.equal(bufs[i][4], bufs[0][4]) and torch.equal(bufs[i][2], bufs[0][2])
    del bufs
    res_gbs = res_bytes / (res_ms * 1e-3) / 1e9
    res_gbs_hot = res_bytes / (res_ms_hot * 1e-3) / 1e9
    # L2 fetch and write bytes do not depend on where the line comes from (Infinity Cache or HBM):
    # the counted figure of the same kernels serves both placements
    res_traffic = counted_traffic(cfg.name, ["accept_seg_kernel<true>", "accept_draw_kernel<true, false, 1, 256>"], digest)
    roofline_resample = {"bound": "hbm", "achieved": round(res_gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                         "frac": round(res_gbs / HBM_PEAK_GBS, 4), "traffic": res_traffic,
                         "kernel": "mdss_accept_or_resample (accept_seg_kernel + accept_draw_kernel), residual and mass written for "
                                   "every row",
                         "avg_ms": round(res_ms, 4), "bytes_per_launch": res_bytes,
                         "buffers": f"{ncopy} copies of p, r and the residual ({ncopy * res_bytes / 1e6:.0f} MB) "
                                    "taken in turn: every launch misses the 256 MB Infinity Cache",
                         "cache_resident": {"avg_ms": round(res_ms_hot, 4), "achieved": round(res_gbs_hot, 1),
                                            "frac": round(res_gbs_hot / HBM_PEAK_GBS, 4),
                                            "traffic": res_traffic,
                                            "note": "the step's own buffers, %.1f MB per launch: %s the 256 MB "
                                                    "Infinity Cache" % (res_bytes / 1e6, "fit in" if res_bytes < 256e6
                                                                        else "exceed")}}

    line = {
        "metric": METRIC,
        "value": round(B / (ms_per_step * 1e-3), 2),
        "unit": "positions/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": f"{cfg.name}: {cfg.describe}", "B": B, "V": V, "K": K,
                   "s_max": s_max or None, "two_draft_distributions": cfg.pair,
                   "selection": "truncated LP" if tlp_s else ("successive pairwise, classical importance weights"
                                                              if cfg.successive else
                                                              f"classical importance weights, alphabet truncated to "
                                                              f"{cfg.alphabet} tokens" if cfg.alphabet else
                                                              "classical importance weights"),
                   "successive": cfg.successive, "accept_rate": None if cfg.diag else round(accept_rate, 4),
                   **({"mean_pstar": round(float(pstar_t.mean()), 5),
                       "mean_fraction_of_optimum": round(float((achieved_t / pstar_t).mean()), 5)} if cfg.diag else {}),
                   "expected_acceptance": round(expected_acc, 5)},
        "roofline": roofline,
        "roofline_resample": roofline_resample,
        "method": "exponential-sum quadrature" if use_es else "exact pairwise sums",
        "timing": timing,
        "ms_per_step_one_graph_each": None if ms_one_per_graph is None else round(ms_one_per_graph, 4),
        "r_eager_ms": None if r_eager_ms is None else round(r_eager_ms, 4),
        "exact_pairwise": exact_pairwise,
        "cpu_baseline": None,
        "kernel_source_digest": digest,
    }
    if not args.no_cpu:
        ncores = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
        rows = args.cpu_rows or (B if tlp_s or cfg.successive or cfg.diag else 2 * ncores)
        line["cpu_baseline"] = cpu_baseline(w, rows)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
