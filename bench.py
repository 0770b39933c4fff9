"""Benchmark of the CP tensor-product layer forward pass on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]
                    [--no-cpu-baseline] [--backward] [--eager] [--radius-graph]
                    [--ablation-atomics] [--ablations] [--attention] [--calibrate-copy]
                    [--no-comparator]
                    [--comparator-sweep] [--three-input]

One step is one call of tdn_cp_tp_forward on the headline workload (64
molecules x 50 atoms, 3200 nodes, ~151k edges within 6 A, L=4, C=128,
R=128, float32, edges pre-sorted by destination): segment offsets, the fused
harmonics/radial/Khatri-Rao MFMA edge pass with the per-node output factor,
and the shared channel-mix GEMM.  Inputs are resident in HBM before timing.
Prints one JSON line.  The metric is edge tensor products per second.  The
step is timed twice: launched eagerly (with per-kernel HIP events, which give
the roofline's kernel time) and captured once in a HIP graph and replayed
(every kernel of every step still runs, without per-launch host cost); value
and ms_per_step come from the replay, value_eager and ms_per_step_eager from
the eager loop (--eager times the eager step only).

The roofline object reports the dominant kernel (the edge pass): its
algorithmic flops per launch, E (2RdC + 2Rd + 17R + RC) + N 2dRC, over its
average launch time from HIP events recorded on its launch stream, against
the peak of the MFMA instruction its contraction executes: fp16 MFMA
(2.5 PFLOP/s) for fp32 problems, which run as three products of two-part
fp16 splits (fp32-level accuracy), and bf16 MFMA (2.5 PFLOP/s) for bfloat16
features.  Beside frac it gives the same rate against the fp32 MFMA peak
(frac_of_fp32_mfma_peak, which can pass 1) and against the ceiling of
emulated fp32 products, a third of the fp16 peak; "executed" gives the fp16
MFMA work the kernel actually issues (part products and padded degree rows
included) against the fp16 peak.  The CPU baseline times the oracle (the
plain float64 per-edge implementation) on a bounded sample of the same
workload on this host's cores.

The "exact_cg_comparator" object (fp32 workloads; --no-comparator skips it)
times tdn_dense_tp_forward, the exact CG tensor product with one radial
weight per path (Sec. 2, Sec. 3.2), on the same edges, features and channel
weight, and reports the CP edge pass's speed-up over it (edge kernel against
edge kernel, whole forward against whole forward, eager launches).  Its
algorithmic flops per launch are E (3 nnz(C) + 2 d^2 C): the per-edge matrix
K_e = C x2 (Y_e rho_e) and its product with the gathered features.
Its "unshared" object times tdn_dense_tp_forward_unshared, the exact
product without path-weight sharing (one channel matrix per path, the fully
connected product of Sec. 3.2): per-path edge sums (dense_edge_unshared) and
the per-path channel GEMMs (path_gemm), C <= 128.
--comparator-sweep adds the same comparison for L = 1..6 on the headline
graph (C = 128, R = 32 ceil(7 L^2 / 32) capped at 256, random factors):
the analogue of the paper's speed-up-against-degree figure (Sec. 4.5).
--ablations adds the forward with the factor blocks read from global memory,
with the harmonics read from a precomputed table, and with the contraction
on the vector ALUs (tdn_ablation_forward), each timed beside the product's
edge kernel (field "ablations"); --ablation-atomics the segmented sum
replaced by float atomics.
--attention adds the attention block (tdn_attention_forward: attention
weights from invariant edge inputs, softmax per destination and head, the
messages weighted per head inside the edge pass; 4 heads, 32 hidden units)
timed beside the plain forward (field "attention").
--three-input adds the three-input CP product (App. A, N = 3: source
features, edge harmonics, destination features; tdn_cp_tp3_forward) on the
same workload, timed beside the two-input forward.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "edge tensor products/sec, CP-TP fwd at L=4,C=128,R=128; % MFMA/HBM roofline"
PEAK_FP32_MFMA_TFLOPS = 157.3
PEAK_BF16_MFMA_TFLOPS = 2500.0
PEAK_FP16_MFMA_TFLOPS = 2500.0
FACTORS = os.path.join(ROOT, "tests", "golden", "factors")
CG_TABLES = os.path.join(ROOT, "tests", "golden", "cg")
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_cp_edge_fwd.json")


def edge_kernel_flops(N, E, d, C, R):
    return E * (2 * R * d * C + 2 * R * d + 17 * R + R * C) + N * 2 * d * R * C


def forward_flops(N, E, d, C, R):
    return edge_kernel_flops(N, E, d, C, R) + N * 2 * d * C * C


def kernel_source_hash():
    h = hashlib.sha256()
    for f in ("cp_edge_impl.hpp", "cp_edge.hip", "sh_device.hpp", "common.hpp"):
        h.update(open(os.path.join(ROOT, "paper_2507_01131_amd", "csrc", f), "rb").read())
    return h.hexdigest()[:16]


def traffic_for(workload):
    """HBM bytes per launch of the edge kernel from the committed rocprofv3
    counter summary, if it was taken on the current kernel source."""
    try:
        t = json.load(open(TRAFFIC_FILE))
    except (OSError, ValueError):
        return None
    if t.get("kernel_source_hash") != kernel_source_hash() or t.get("workload") != workload:
        return None
    return t.get("hbm_bytes_per_launch")


def time_calls(fn, torch, tdn, kernel, steps, warmup=3):
    """(average kernel ms from the library's HIP events, average ms per call)
    over `steps` eager calls."""
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    tdn.timer_enable(True)
    tdn.timer_read(kernel, reset=True)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        fn()
    e1.record()
    torch.cuda.synchronize()
    tdn.timer_enable(False)
    ms, n = tdn.timer_read(kernel, reset=True)
    return ms / max(1, n), e0.elapsed_time(e1) / steps


def exact_comparator(torch, tdn, L, x, vec, ei, W, r_cut, presorted, steps, n_radial, seed=0):
    """Times tdn_dense_tp_forward on these inputs with seeded path weights."""
    zc = np.load(os.path.join(CG_TABLES, f"cg_L{L}.npz"))
    tab = tdn.cg_table(zc["M"], zc["path"], x.device)
    rng = np.random.default_rng(seed)
    pw = torch.from_numpy((rng.standard_normal((n_radial, tab.n_path)) / np.sqrt(n_radial)).astype(np.float32))
    pw = pw.to(x.device)
    N, d, C = x.shape
    E = vec.shape[0]
    ws = torch.empty(tdn.workspace_size(tdn.make_problem(L, C, tab.n_path, N, E, r_cut, n_radial))[0],
                     dtype=torch.uint8, device=x.device)
    out = torch.empty((N, d, C), dtype=torch.float32, device=x.device)
    perm = torch.empty(E, dtype=torch.int32, device=x.device)
    off = torch.empty(N + 1, dtype=torch.int32, device=x.device)

    def call():
        return tdn.dense_forward(x, vec, ei, tab, pw, W, r_cut=r_cut, edges_sorted=presorted, workspace=ws,
                                 out=out, perm=perm, offsets=off)

    k_ms, f_ms = time_calls(call, torch, tdn, "dense_edge_fwd", steps)
    nnz = int(tab.col.shape[0])
    flops = E * (3 * nnz + 2 * d * d * C)
    return {"edge_kernel_ms": k_ms, "forward_ms": f_ms, "paths": tab.n_path, "cg_nnz": nnz,
            "flops_per_launch": flops, "achieved_tflops": flops / (k_ms * 1e-3) / 1e12}


def unshared_comparator(torch, tdn, L, x, vec, ei, r_cut, presorted, steps, n_radial, seed=0):
    """Times tdn_dense_tp_forward_unshared (one seeded channel matrix per
    path) on these inputs: the per-path edge sums and the path GEMM."""
    zc = np.load(os.path.join(CG_TABLES, f"cg_L{L}.npz"))
    tab = tdn.cg_table(zc["M"], zc["path"], x.device)
    rng = np.random.default_rng(seed)
    N, d, C = x.shape
    E = vec.shape[0]
    P = tab.n_path
    pw = torch.from_numpy((rng.standard_normal((n_radial, P)) / np.sqrt(n_radial)).astype(np.float32)).to(x.device)
    Wp = torch.from_numpy((rng.standard_normal((P, C, C)) / np.sqrt(C)).astype(np.float32)).to(x.device)
    out = torch.empty((N, d, C), dtype=torch.float32, device=x.device)
    perm = torch.empty(E, dtype=torch.int32, device=x.device)
    off = torch.empty(N + 1, dtype=torch.int32, device=x.device)
    ws = torch.empty(tdn.dense_unshared_workspace_size(tdn.make_problem(L, C, P, N, E, r_cut, n_radial)),
                     dtype=torch.uint8, device=x.device)

    def call():
        return tdn.dense_forward_unshared(x, vec, ei, tab, pw, Wp, r_cut=r_cut, edges_sorted=presorted,
                                          workspace=ws, out=out, perm=perm, offsets=off)

    k_ms, f_ms = time_calls(call, torch, tdn, "dense_edge_unshared", steps)
    g_ms, _ = time_calls(call, torch, tdn, "path_gemm", max(1, steps // 4))
    rows = sum(2 * l3 + 1 for l1 in range(L + 1) for l2 in range(L + 1)
               for l3 in range(abs(l1 - l2), min(l1 + l2, L) + 1))
    del Wp, ws
    return {"edge_kernel_ms": k_ms, "path_gemm_ms": g_ms, "forward_ms": f_ms, "paths": P, "path_rows": rows}


def cpu_model():
    try:
        for ln in open("/proc/cpuinfo"):
            if ln.startswith("model name"):
                return ln.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(w, A, B, D, budget_s=12.0):
    """The oracle's forward (float64, per-edge literal summation) on seeded
    batches of 64 destination nodes until about budget_s seconds of timed
    work; edges/s over the sample.  The stable sort by destination, the
    selection of each batch's edges and the gather of the rows they touch
    happen once per batch outside the timed region, so only the oracle's
    layer arithmetic is timed.  cores = threads the oracle's BLAS used, capped
    by the CPUs this process may run on."""
    from threadpoolctl import threadpool_info

    from oracle import layer

    N = w["N"]
    src, dst = np.asarray(w["edge_index"][0], np.int64), np.asarray(w["edge_index"][1], np.int64)
    perm, offsets = layer.stable_sort_by_key(dst, N)
    perm = perm.astype(np.int64)
    rng = np.random.default_rng(0)
    order = rng.permutation(N)
    edges = nodes = 0
    timed = 0.0
    for i in range(0, N, 64):
        batch = np.sort(order[i:i + 64])
        slots = np.concatenate([np.arange(offsets[t], offsets[t + 1]) for t in batch])
        ids = perm[slots]                      # the batch's edges in sorted order
        rows = np.unique(np.concatenate([src[ids], batch]))
        remap = np.full(N, -1, np.int64)
        remap[rows] = np.arange(rows.shape[0])
        ei = np.stack([remap[src[ids]], remap[dst[ids]]])
        xs, vec = np.ascontiguousarray(w["x"][rows]), np.ascontiguousarray(w["edge_vec"][ids])
        t0 = time.perf_counter()
        layer.forward(xs, ei, vec, A, B, D, w["W"], w["radial_w"], w["r_cut"], w["L"],
                      perm=np.arange(ids.shape[0]))
        timed += time.perf_counter() - t0
        edges += int(ids.shape[0])
        nodes += len(batch)
        if timed > budget_s:
            break
    affinity = len(os.sched_getaffinity(0))
    blas = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    return {"value": edges / timed, "unit": "edge tensor products/s", "cores": int(min(affinity, blas)),
            "kind": "oracle", "cpu_model": cpu_model(), "cpus_in_affinity": affinity, "blas_threads": int(blas),
            "sample": f"{nodes} of {N} destination nodes ({edges} of {w['E']} edges), float64 per-edge "
                      f"direct summation, {timed:.1f} s timed (sort and gathers untimed)"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="molecules3200_L4_C128_R128")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--backward", action="store_true",
                    help="also time tdn_cp_tp_backward with every gradient (x, W, edge vectors, radial weights; "
                         "extra field)")
    ap.add_argument("--attention", action="store_true",
                    help="time the attention block over the same messages (field 'attention')")
    ap.add_argument("--ablations", action="store_true",
                    help="time the forward with the factors read from global memory, the harmonics from a "
                         "precomputed table, and the contraction on the VALU (field 'ablations')")
    ap.add_argument("--ablation-atomics", action="store_true",
                    help="also time the atomic scatter-add forward (extra field; fp32 workloads with 2 <= L <= 4)")
    ap.add_argument("--eager", action="store_true",
                    help="time the eagerly launched step only (default: the step captured once in a HIP graph "
                         "and replayed, with the eager step timed beside it)")
    ap.add_argument("--radius-graph", action="store_true",
                    help="also time tdn_radius_graph on the workload's geometry (extra field)")
    ap.add_argument("--no-comparator", action="store_true",
                    help="skip timing the exact CG tensor product on the same edges")
    ap.add_argument("--comparator-sweep", action="store_true",
                    help="also compare the CP and exact forwards for L = 1..6 on this graph (extra field)")
    ap.add_argument("--three-input", action="store_true",
                    help="also time the three-input CP product on this workload (extra field; fp32, 2 <= L <= 4)")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="first run a plain 256 MiB device copy (reference for rocprofv3 byte counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for {args.gpus}); the multi-GPU layout is a design "
              "note, not a measured path", file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2507_01131_amd as tdn
    import workloads

    if not os.path.exists(tdn.LIB_PATH):
        from paper_2507_01131_amd import build as _b
        _b.build()
    dev = torch.device("cuda:0")
    w = workloads.make_workload(args.workload)
    z = np.load(os.path.join(FACTORS, f"cp_L{w['L']}_R{w['R']}.npz"))
    A, B, D = z["A"], z["B"], z["D"]
    N, E, d, C, R = w["N"], w["E"], w["d"], w["C"], w["R"]
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)  # noqa: E731
    if w["feat_dtype"] == "bf16":
        x = t(w["x_bf16"].view(np.int16)).view(torch.bfloat16)
        W = t(w["W_bf16"].view(np.int16)).view(torch.bfloat16)
    else:
        x, W = t(w["x"]), t(w["W"])
    vec, ei, rw = t(w["edge_vec"]), t(w["edge_index"]), t(w["radial_w"])
    At, Bt, Dt = t(A), t(B), t(D)
    p = tdn.make_problem(w["L"], C, R, N, E, w["r_cut"], w["n_radial"],
                         tdn.TDN_BF16 if w["feat_dtype"] == "bf16" else tdn.TDN_F32, w["presorted"])
    fwd_bytes, bwd_bytes = tdn.workspace_size(p)
    ws = torch.empty(fwd_bytes, dtype=torch.uint8, device=dev)
    out = torch.empty((N, d, C), dtype=torch.float32, device=dev)
    zsave = torch.empty((N, d, C), dtype=torch.float32, device=dev)
    perm = torch.empty(E, dtype=torch.int32, device=dev)
    offsets = torch.empty(N + 1, dtype=torch.int32, device=dev)

    def step():
        return tdn.forward(x, vec, ei, At, Bt, Dt, W, rw, L=w["L"], r_cut=w["r_cut"], edges_sorted=w["presorted"],
                           workspace=ws, out=out, z=zsave, perm=perm, offsets=offsets)

    if args.calibrate_copy:
        a = torch.empty(64 << 20, dtype=torch.float32, device=dev).fill_(1.0)
        b = torch.empty_like(a)
        for _ in range(3):
            b.copy_(a)
        torch.cuda.synchronize()
        del a, b
    for _ in range(args.warmup):
        res = step()
    torch.cuda.synchronize()
    tdn.timer_enable(True)
    fwd_kernels = ("cp_edge_fwd", "feature_layout", "node_gemm", "sort")
    for k in fwd_kernels:
        tdn.timer_read(k, reset=True)
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    ev0, ev1 = evs[0], evs[-1]
    torch.cuda.synchronize()
    for i in range(args.steps):
        evs[i].record()
        res = step()
    ev1.record()
    torch.cuda.synchronize()
    tdn.timer_enable(False)
    total_ms = ev0.elapsed_time(ev1)
    ms_step = total_ms / args.steps
    per_step = np.array([evs[i].elapsed_time(evs[i + 1]) for i in range(args.steps)])
    kern = {k: tdn.timer_read(k, reset=True) for k in fwd_kernels}
    edge_ms = kern["cp_edge_fwd"][0] / max(1, kern["cp_edge_fwd"][1])
    ms_step_eager = ms_step
    launch = "eager"
    if not args.eager:
        # The same step (offsets, feature layout, edge pass, node GEMM)
        # captured once in a HIP graph and replayed: every kernel of every step
        # still runs, without the per-launch host cost.  The eager loop above
        # gave the per-kernel durations.
        try:
            side = torch.cuda.Stream()
            side.wait_stream(torch.cuda.current_stream())
            with torch.cuda.stream(side):
                step()
            torch.cuda.current_stream().wait_stream(side)
            torch.cuda.synchronize()
            graph = torch.cuda.CUDAGraph()
            with torch.cuda.graph(graph):
                step()
            for _ in range(args.warmup):
                graph.replay()
            torch.cuda.synchronize()
            for i in range(args.steps):
                evs[i].record()
                graph.replay()
            ev1.record()
            torch.cuda.synchronize()
            ms_step = ev0.elapsed_time(ev1) / args.steps
            per_step = np.array([evs[i].elapsed_time(evs[i + 1]) for i in range(args.steps)])
            launch = "hip_graph_replay"
        except RuntimeError as exc:  # capture unavailable: report the eager step
            print(f"graph capture failed ({exc}); timing the eager step", file=sys.stderr)

    bf16 = w["feat_dtype"] == "bf16"
    f_edge = edge_kernel_flops(N, E, d, C, R)
    achieved = f_edge / (edge_ms * 1e-3) / 1e12
    # The peak of the MFMA instruction the edge contraction executes: bf16
    # features run it on bf16 MFMA, fp32 features on fp16 MFMA (three
    # products of two-part fp16 splits), both with fp32 accumulation.
    peak = PEAK_BF16_MFMA_TFLOPS if bf16 else PEAK_FP16_MFMA_TFLOPS
    line = {
        "metric": METRIC,
        "value": E / (ms_step * 1e-3),
        "unit": "edge tensor products/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "ms_per_step_p10_p50_p90": [float(np.percentile(per_step, q)) for q in (10, 50, 90)],
        "launch": launch,
        "ms_per_step_eager": ms_step_eager,
        "value_eager": E / (ms_step_eager * 1e-3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if bf16 else "f32",
        "data": "synthetic",
        "config": {"workload": w["name"], "N": N, "E": E, "L": w["L"], "d": d, "C": C, "R": R,
                   "edges_presorted": bool(w["presorted"]), "pass": "forward"},
        "roofline": {"bound": "mfma", "achieved": achieved, "peak": peak, "unit": "TFLOP/s",
                     "frac": achieved / peak, "traffic": traffic_for(w["name"]),
                     "kernel": "cp_edge_fwd", "kernel_ms": edge_ms, "flops_per_launch": f_edge,
                     "peak_instruction": "v_mfma_f32_32x32x16_bf16" if bf16 else "v_mfma_f32_32x32x16_f16"},
        "kernel_ms_per_step": {k: v[0] / max(1, v[1]) for k, v in kern.items()},
        # the paper's own speed figures (other hardware, other baselines): context, not targets
        "paper_reported": {
            "cp_tp_speedup_over_e3nn_fully_connected_cg_tp_by_L": {"1": 4.0, "2": 4.8, "3": 15.0, "4": 26.7,
                                                                  "5": 47.6, "6": 83.6},
            "cp_tp_speedup_source": "Sec. 4.5 (inference runtime figure); hardware not stated for it, the "
                                    "paper's experiments run on NVIDIA A100-80GB unless noted",
            "tdn_over_equiformer_structures_per_s": "2.47x to 8.44x, one NVIDIA A100-80GB, batch 128 (Sec. 4.5)",
            "training_time_reduction_ps_plus_cp": "about 78 % for TDN, about 74 % for NequIP, one NVIDIA "
                                                  "RTX A6000-48GB (Sec. 4.6)"},
        "forward_tflops": forward_flops(N, E, d, C, R) / (ms_step * 1e-3) / 1e12,
    }
    if not bf16:
        # fp16 MFMA work issued by the edge contraction: per edge, 32-channel
        # tile and 32-rank tile, the packed K-reduction of the three part
        # products, ceil(3 ceil(d/2) / 8) steps of 2*32*32*16 flops
        pk_blocks = (3 * ((d + 1) // 2) + 7) // 8
        executed = E * ((C + 31) // 32) * ((R + 31) // 32) * pk_blocks * 2 * 32 * 32 * 16
        # the same algorithmic rate against the fp32 MFMA peak (can pass 1,
        # since the work runs on fp16 MFMA) and against the ceiling of fp32
        # products emulated by three fp16 products (fp16 peak / 3)
        line["roofline"]["frac_of_fp32_mfma_peak"] = achieved / PEAK_FP32_MFMA_TFLOPS
        line["roofline"]["emulated_fp32_ceiling"] = PEAK_FP16_MFMA_TFLOPS / 3
        line["roofline"]["frac_of_emulated_fp32_ceiling"] = achieved / (PEAK_FP16_MFMA_TFLOPS / 3)
        line["roofline"]["executed"] = {
            "mfma": "v_mfma_f32_32x32x16_f16, three products of two-part fp16 splits per fp32 product, packed "
                    "into one K-reduction",
            "flops_per_launch": executed, "achieved": executed / (edge_ms * 1e-3) / 1e12,
            "peak": PEAK_FP16_MFMA_TFLOPS, "frac": executed / (edge_ms * 1e-3) / 1e12 / PEAK_FP16_MFMA_TFLOPS}
    if not bf16 and not args.no_comparator:
        # the exact CG tensor product on the same edges, features and W
        cmp_ = exact_comparator(torch, tdn, w["L"], x, vec, ei, W, w["r_cut"], w["presorted"], args.steps,
                                w["n_radial"])
        _, cp_fwd_ms = time_calls(step, torch, tdn, "cp_edge_fwd", args.steps)
        cmp_.update({"kernel": "dense_edge_fwd", "cp_edge_kernel_ms": edge_ms, "cp_forward_ms": cp_fwd_ms,
                     "cp_edge_kernel_speedup": cmp_["edge_kernel_ms"] / edge_ms,
                     "cp_forward_speedup": cmp_["forward_ms"] / cp_fwd_ms,
                     "frac_of_fp32_mfma_peak": cmp_["achieved_tflops"] / PEAK_FP32_MFMA_TFLOPS,
                     "launch": "eager"})
        if C <= 128:
            un = unshared_comparator(torch, tdn, w["L"], x, vec, ei, w["r_cut"], w["presorted"], args.steps,
                                     w["n_radial"])
            un.update({"kernel": "dense_edge_unshared", "cp_forward_speedup": un["forward_ms"] / cp_fwd_ms,
                       "cp_edge_kernel_speedup": un["edge_kernel_ms"] / edge_ms, "launch": "eager"})
            cmp_["unshared"] = un
        line["exact_cg_comparator"] = cmp_
    if args.comparator_sweep and not bf16:
        rng = np.random.default_rng(1)
        sweep = []
        for Ls in range(1, 7):
            ds = (Ls + 1) ** 2
            Rs = min(256, 32 * -(-7 * Ls * Ls // 32))
            Cs = 128
            xs_ = t(rng.standard_normal((N, ds, Cs)).astype(np.float32))
            Ws = t((rng.standard_normal((Cs, Cs)) / np.sqrt(Cs)).astype(np.float32))
            fac = [t((rng.standard_normal((ds, Rs)) / np.sqrt(ds)).astype(np.float32)) for _ in range(3)]
            rws = t((rng.standard_normal((w["n_radial"], Rs)) / np.sqrt(w["n_radial"])).astype(np.float32))

            def cp_call():
                return tdn.forward(xs_, vec, ei, fac[0], fac[1], fac[2], Ws, rws, L=Ls, r_cut=w["r_cut"],
                                   edges_sorted=w["presorted"], save_z=False)

            ck, cf = time_calls(cp_call, torch, tdn, "cp_edge_fwd", 20)
            ex = exact_comparator(torch, tdn, Ls, xs_, vec, ei, Ws, w["r_cut"], w["presorted"], 20, w["n_radial"])
            un = unshared_comparator(torch, tdn, Ls, xs_, vec, ei, w["r_cut"], w["presorted"], 5, w["n_radial"])
            sweep.append({"L": Ls, "d": ds, "C": Cs, "R": Rs, "paths": ex["paths"], "cg_nnz": ex["cg_nnz"],
                          "cp_edge_kernel_ms": ck, "exact_edge_kernel_ms": ex["edge_kernel_ms"],
                          "cp_forward_ms": cf, "exact_forward_ms": ex["forward_ms"],
                          "cp_edge_kernel_speedup": ex["edge_kernel_ms"] / ck,
                          "cp_forward_speedup": ex["forward_ms"] / cf,
                          "unshared_edge_kernel_ms": un["edge_kernel_ms"], "unshared_path_gemm_ms": un["path_gemm_ms"],
                          "unshared_forward_ms": un["forward_ms"],
                          "cp_forward_speedup_vs_unshared": un["forward_ms"] / cf})
            del xs_, Ws, fac, rws
        line["comparator_sweep"] = sweep
    if args.three_input and not bf16:
        A2t = t((np.random.default_rng(5).standard_normal((d, R)) / np.sqrt(d)).astype(np.float32))

        def step3():
            return tdn.forward3(x, vec, ei, At, A2t, Bt, Dt, W, rw, L=w["L"], r_cut=w["r_cut"],
                                edges_sorted=w["presorted"], workspace=ws, out=out, z=zsave, perm=perm,
                                offsets=offsets)

        k3, f3 = time_calls(step3, torch, tdn, "cp_edge_fwd_t3", args.steps)
        _, f2 = time_calls(step, torch, tdn, "cp_edge_fwd", args.steps)
        line["three_input"] = {"edge_kernel_ms": k3, "forward_ms": f3, "two_input_edge_kernel_ms": edge_ms,
                               "two_input_forward_ms": f2, "edge_kernel_ratio": k3 / edge_ms,
                               "value": E / (f3 * 1e-3), "launch": "eager"}
    if args.ablation_atomics:
        # the same forward with the segmented sum replaced by per-edge
        # application of D and float atomics into Z
        def step_atomic():
            return tdn.forward(x, vec, ei, At, Bt, Dt, W, rw, L=w["L"], r_cut=w["r_cut"],
                               edges_sorted=w["presorted"], workspace=ws, out=out, z=zsave, perm=perm,
                               offsets=offsets, atomics_ablation=True)

        for _ in range(3):
            step_atomic()
        torch.cuda.synchronize()
        tdn.timer_enable(True)
        tdn.timer_read("cp_edge_fwd_atomic", reset=True)
        ev0.record()
        for _ in range(args.steps):
            step_atomic()
        ev1.record()
        torch.cuda.synchronize()
        tdn.timer_enable(False)
        a_ms, a_n = tdn.timer_read("cp_edge_fwd_atomic", reset=True)
        a_step = ev0.elapsed_time(ev1) / args.steps
        line["ablation_atomics"] = {
            "edge_kernel_ms": a_ms / max(1, a_n), "segmented_edge_kernel_ms": edge_ms,
            "edge_kernel_slowdown": a_ms / max(1, a_n) / edge_ms,
            "ms_per_step": a_step, "value": E / (a_step * 1e-3)}
    if args.ablations and not bf16:
        # the other hot-path choices, each replaced in turn (tdn_ablation_forward)
        abl = {}
        for code, name in ((tdn.ABL_FACTORS_GLOBAL, "factors_global"), (tdn.ABL_Y_TABLE, "y_table"),
                           (tdn.ABL_VALU, "valu_contraction")):
            if code == tdn.ABL_VALU and (C > 128 or R > 128):
                continue
            pa = tdn.make_problem(w["L"], C, R, N, E, w["r_cut"], w["n_radial"], tdn.TDN_F32, w["presorted"])
            aws = torch.empty(tdn.ablation_workspace_size(pa, code), dtype=torch.uint8, device=x.device)

            def step_abl(code=code, aws=aws):
                return tdn.forward(x, vec, ei, At, Bt, Dt, W, rw, L=w["L"], r_cut=w["r_cut"],
                                   edges_sorted=w["presorted"], workspace=aws, out=out, z=zsave, perm=perm,
                                   offsets=offsets, ablation=code)

            k_ms, f_ms = time_calls(step_abl, torch, tdn, "cp_edge_fwd_ablation", args.steps)
            entry = {"edge_kernel_ms": k_ms, "ms_per_step": f_ms, "value": E / (f_ms * 1e-3),
                     "edge_kernel_slowdown": k_ms / edge_ms}
            if code == tdn.ABL_Y_TABLE:
                entry["table_kernel_ms"], _ = time_calls(step_abl, torch, tdn, "sh_table", max(1, args.steps // 4))
            abl[name] = entry
            del aws
        abl["segmented_edge_kernel_ms"] = edge_ms
        line["ablations"] = abl
    if args.attention and not bf16 and 1 <= w["L"] <= 4 and R <= 256 and C % 128 == 0:
        # the attention block over the same messages: 4 heads, 32 hidden units
        rng_a = np.random.default_rng(3)
        H_a, F_a = 4, 32
        W1a = t((rng_a.standard_normal((2 * C + w["n_radial"], F_a)) / np.sqrt(2 * C + w["n_radial"]))
                .astype(np.float32))
        w2a = t((rng_a.standard_normal((F_a, H_a)) / np.sqrt(F_a)).astype(np.float32))
        pa = tdn.make_problem(w["L"], C, R, N, E, w["r_cut"], w["n_radial"], tdn.TDN_F32, w["presorted"])
        aws = torch.empty(tdn.attention_workspace_size(pa, H_a, F_a), dtype=torch.uint8, device=x.device)
        alpha_a = torch.empty((E, H_a), dtype=torch.float32, device=x.device)

        def step_att():
            return tdn.attention_forward(x, vec, ei, At, Bt, Dt, W, rw, W1a, w2a, L=w["L"], r_cut=w["r_cut"],
                                         edges_sorted=w["presorted"], workspace=aws, out=out, alpha=alpha_a,
                                         perm=perm, offsets=offsets)

        k_ms, f_ms = time_calls(step_att, torch, tdn, "cp_edge_fwd_att", args.steps)
        w_ms, _ = time_calls(step_att, torch, tdn, "attention_weights", max(1, args.steps // 4))
        line["attention"] = {"heads": H_a, "hidden": F_a, "edge_kernel_ms": k_ms, "weights_ms": w_ms,
                             "ms_per_step": f_ms, "value": E / (f_ms * 1e-3),
                             "edge_kernel_vs_plain": k_ms / edge_ms, "launch": "eager"}
        del aws, alpha_a
    if args.radius_graph:
        # the edges of this workload rebuilt on the device from its atoms
        gi = workloads.graph_inputs(w["name"])
        per = gi["periodic"]
        gp, gg, gc = t(gi["pos"]), t(gi["graph_ptr"]), t(gi["cell"]) if any(per) else None
        first = tdn.radius_graph(gp, gg, r_cut=gi["r_cut"], cell=gc, periodic=per)
        E_rg = first.edge_index.shape[1]

        def build_graph():
            return tdn.radius_graph(gp, gg, r_cut=gi["r_cut"], cell=gc, periodic=per, capacity=E_rg)

        for _ in range(3):
            build_graph()
        torch.cuda.synchronize()
        tdn.timer_enable(True)
        tdn.timer_read("radius_graph", reset=True)
        t0 = time.perf_counter()
        for _ in range(args.steps):
            build_graph()
        torch.cuda.synchronize()
        wall = (time.perf_counter() - t0) / args.steps
        tdn.timer_enable(False)
        g_ms, g_n = tdn.timer_read("radius_graph", reset=True)
        n_at = gi["pos"].shape[0]
        line["radius_graph"] = {
            "atoms": n_at, "systems": len(gi["graph_ptr"]) - 1, "r_cut": gi["r_cut"], "periodic": list(per),
            "edges": E_rg, "edges_match_fixture": E_rg == E, "ms_per_call_wall": wall * 1e3,
            "ms_per_call_events": g_ms / max(1, g_n), "edges_per_s": E_rg / wall,
            "algorithmic_bytes": 12 * n_at + 20 * E_rg + 4 * (n_at + 1)}
    if args.backward:
        G = torch.from_numpy(w["grad_out"]).to(dev)
        wsb = torch.empty(bwd_bytes, dtype=torch.uint8, device=dev)
        for _ in range(3):
            tdn.backward(res, G, workspace=wsb, need_radial=True)
        torch.cuda.synchronize()
        bk = ("node_gemm", "gram", "channel_layout", "cp_bwd_dst", "radial_grad", "sort", "feature_layout",
              "cp_edge_bwd_src")
        tdn.timer_enable(True)
        for k in bk:
            tdn.timer_read(k, reset=True)
        ev0.record()
        for _ in range(10):
            tdn.backward(res, G, workspace=wsb, need_radial=True)
        ev1.record()
        torch.cuda.synchronize()
        tdn.timer_enable(False)
        line["backward_kernel_ms_per_step"] = {k: tdn.timer_read(k, reset=True)[0] / 10 for k in bk}
        line["backward_ms"] = ev0.elapsed_time(ev1) / 10
        line["backward_edges_per_s"] = E / (line["backward_ms"] * 1e-3)
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(w, A, B, D)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
