"""PARK sparse-attention forward benchmark: one DiT attention layer on one GPU.

A step is one park_forward call (recompute mode: query k-means, QRKC key
k-means, permutation, centroids, PAMA retrieval + selection, block-sparse
attention) over the whole layer, inputs already resident in HBM.

Prints one JSON line.  `value` is milliseconds per layer (lower is better);
the dense-equivalent TFLOP/s (4 N^2 d H / t) is reported beside it.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "ms per layer + dense-equiv TFLOP/s at 1 GPU; % of MFMA/HBM peak by stage"

# MI355X published peaks
PEAK = {"hbm": 8000.0,            # GB/s
        "mfma_bf16": 2500.0,      # TFLOP/s dense
        "alu_f32": 157.3,         # TFLOP/s vector fp32
        "alu_f64": 78.6}          # TFLOP/s vector fp64


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="hunyuan",
                    help="synthetic layer: tiny | medium | wan | hunyuan (default: the "
                         "HunyuanVideo-shaped layer, the largest single-GPU configuration)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-graph", action="store_true",
                    help="time eager launches only (no HIP graph replay)")
    ap.add_argument("--reuse", default="recompute", choices=["recompute", "clusters", "mask"],
                    help="recompute everything, or time the next diffusion step (Q, K drifted by "
                         "N(0, 0.05^2)) reusing the clustering (and the mask)")
    ap.add_argument("--topp", type=float, default=None, help="override: top-p selection mass")
    ap.add_argument("--ratio", type=float, default=None, help="override: top-k ratio")
    ap.add_argument("--block", type=int, default=None, help="override: mean block size B")
    ap.add_argument("--iters", type=int, default=None, help="override: k-means iterations T")
    ap.add_argument("--estimator", default="pama", choices=["pama", "qcentroid"],
                    help="block-importance estimate: PAMA, or the query-centroid estimate "
                         "(the 'w/o PAMA' ablation)")
    ap.add_argument("--blocks", default="cluster", choices=["cluster", "fixed"],
                    help="blocks = k-means clusters, or fixed chunks of the cluster order")
    ap.add_argument("--key-metric", default="qrkc", choices=["qrkc", "euclid"],
                    help="key clustering: QRKC, or Euclidean k-means (the 'w/o QRKC' ablation)")
    ap.add_argument("--alpha", type=float, default=0.05,
                    help="shrinkage of the key metric toward the isotropic one (App. D)")
    ap.add_argument("--cpu-heads", type=int, default=None,
                    help="heads of the layer the oracle runs for the CPU baseline (default: 4 "
                         "below 50k tokens per head, else 1: about 10-30 s of host work)")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="only run a plain elementwise copy of MIB MiB (float32 negation, "
                         "read once, written once) five times: the known-size kernel that "
                         "scales the FETCH_SIZE / WRITE_SIZE counters to bytes")
    return ap.parse_args()


CSRC = os.path.join(ROOT, "paper_2609_38978_amd", "csrc")


def kernel_source_digest(stage):
    """sha256 (16 hex) of the source file that launches `stage`, common.h and the build flags."""
    import hashlib
    tag = f'"{stage}"'
    h = hashlib.sha256()
    found = False
    for fn in sorted(os.listdir(CSRC)):
        if fn.endswith(".hip"):
            txt = open(os.path.join(CSRC, fn), "rb").read()
            if tag.encode() in txt:
                h.update(txt)
                found = True
    if not found:
        return None
    h.update(open(os.path.join(CSRC, "common.h"), "rb").read())
    h.update(open(os.path.join(ROOT, "paper_2609_38978_amd", "build.py"), "rb").read())
    return h.hexdigest()[:16]


def measured_traffic(workload, stage):
    """HBM bytes per launch of `stage` from the committed counter summary.

    The summary holds FETCH_SIZE and WRITE_SIZE (KiB per dispatch, averaged
    over the dispatches of the stage) scaled by what the same counters read for
    a plain copy of known size.  None when there is no summary for the stage or
    its source has changed since the counters were taken."""
    path = os.path.join(ROOT, "profiles", f"hbm_traffic_{workload}.md")
    if not os.path.exists(path):
        return None
    for line in open(path):
        cells = [c.strip() for c in line.strip().strip("|").split("|")]
        if len(cells) >= 6 and cells[0] == stage:
            if cells[2] != kernel_source_digest(stage):
                return None
            try:
                return float(cells[5])
            except ValueError:
                return None
    return None


def calibrate_copy(mib):
    import torch
    n = mib * (1 << 20) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(5):
        torch.neg(src, out=dst)
    torch.cuda.synchronize()
    print(json.dumps({"copy_kernel": "torch.neg float32", "bytes_read": 4 * n,
                      "bytes_written": 4 * n, "launches": 5}), flush=True)


def kernel_work(name, cfg, st, C):
    """Algorithmic work of ONE launch of kernel `name`: (bound, amount, unit, peak key)."""
    H, N, d = cfg.H, cfg.N, cfg.d
    eb = 2 if cfg.dtype == "bf16" else 4
    if name == "kmeans_assign64":
        return "alu", 2.0 * N * C * d * H, "flop", "alu_f64"
    if name == "kmeans_assign_fast":
        # algorithmic N*C*d multiply-adds; the hi/lo split issues twice that on MFMA
        return "mfma", 2.0 * N * C * d * H, "flop", "mfma_bf16"
    if name == "kmeans_assign_cand":
        # the filtered rounds score each token against its tile's candidate
        # union only (a few percent of the centroids): the gathered token rows
        # are the dominant traffic
        return "hbm", (1.0 * N * d * eb + 8.0 * N) * H, "byte", "hbm"
    if name == "kfilter_radius":  # token rows through perm, their norm bounds
        return "hbm", (1.0 * N * d * eb + 12.0 * N + C * d * 8.0) * H, "byte", "hbm"
    if name == "kfilter_cand":  # mu . w_v for every centroid pair, three split products
        return "mfma", 3.0 * 2.0 * C * C * d * H, "flop", "mfma_bf16"
    if name in ("pama_fast", "pama_fullk"):
        # one q.c product per (query, key block); the centroid split issues it 3x on MFMA
        # (the two-pass kernel twice, the single-sweep one once)
        return "mfma", 2.0 * N * C * d * H, "flop", "mfma_bf16"
    if name == "pama64":
        return "alu", 2.0 * N * C * d * H, "flop", "alu_f64"
    if name == "qcen64":  # one qbar_u . c_v product per (query block, key block)
        return "alu", 2.0 * C * C * d * H, "flop", "alu_f64"
    if name == "gram_partial":
        return "alu", 2.0 * N * d * d * H, "flop", "alu_f64"
    if name in ("attn_valu", "attn_mfma"):
        import numpy as np
        qo = st["q_offsets"].cpu().numpy()
        ko = st["k_offsets"].cpu().numpy()
        kvc = st["kv_count"].cpu().numpy()
        kvi = st["kv_index"].cpu().numpy()
        tot = 0.0
        for h in range(H):
            nk = np.diff(ko[h])
            nq = np.diff(qo[h])
            for u in range(len(nq)):
                if nq[u]:
                    tot += nq[u] * nk[kvi[h, u, :kvc[h, u]]].sum()
        peak = "mfma_bf16" if name == "attn_mfma" else "alu_f32"
        return ("mfma" if name == "attn_mfma" else "alu"), 4.0 * d * tot, "flop", peak
    if name == "gather_rows":  # one of the three gathers: rows read and written, perm read
        return "hbm", (2.0 * N * d * eb + 4.0 * N) * H, "byte", "hbm"
    if name == "segment_mean":  # rows read through perm, float64 means written
        return "hbm", (1.0 * N * d * eb + 4.0 * N + C * d * 8.0) * H, "byte", "hbm"
    if name == "sort_hist":
        return "hbm", 4.0 * N * H, "byte", "hbm"
    if name == "sort_scatter":
        return "hbm", 8.0 * N * H, "byte", "hbm"
    if name == "select_fast":  # the float W^ rows and their error bounds
        return "hbm", 4.0 * C * C * H, "byte", "hbm"
    return None


def attention_flops(ws, st, cfg, ms_attn):
    """Useful and issued MFMA flops of the block-sparse attention launch.

    useful = 4 d sum_u n_u sum_{v in sel(u)} n_v (each query row against the
    keys of its own block's selection).  The grouped kernel streams, per group
    of at most 128 rows (four wavefronts of 32), the union of its query
    blocks' selections in 32-key tiles (in chunks of at most 1024 key blocks)
    and every wavefront computes every tile, so issued = 4 d 128 32 x (tiles
    summed over groups).  The groups are read from the work plan the launch
    left in the workspace: after the 256-byte status region, order [H][CQ],
    row prefix [H][CQ+1] (int32), then the groups int4 [H][GPH] at 16-byte
    alignment, GPH = W + ceil((CQ + W) / 16) + 1, W = ceil(N / 128)."""
    import numpy as np
    H, N, d = cfg.H, cfg.N, cfg.d
    CQ = st["q_offsets"].shape[1] - 1
    qo = st["q_offsets"].cpu().numpy()
    ko = st["k_offsets"].cpu().numpy()
    kvc = st["kv_count"].cpu().numpy()
    kvi = st["kv_index"].cpu().numpy()
    W = -(-N // 128)
    GPH = W + -(-(CQ + W) // 16) + 1
    goff = ((H * CQ + H * (CQ + 1)) * 4 + 15) & ~15
    raw = ws[256:256 + goff + H * GPH * 16].cpu().numpy()
    order = raw[:H * CQ * 4].view(np.int32).reshape(H, CQ)
    grp = raw[goff:goff + H * GPH * 16].view(np.int32).reshape(H, GPH, 4)
    useful = 0.0
    tiles = 0
    for h in range(H):
        nk = np.diff(ko[h]).astype(np.int64)
        nq = np.diff(qo[h]).astype(np.int64)
        for u in range(CQ):
            if nq[u]:
                useful += float(nq[u] * nk[kvi[h, u, :kvc[h, u]]].sum())
        for g in range(GPH):
            r0, r1, i0, i1 = grp[h, g]
            if r1 <= r0 or i1 <= i0:
                continue
            blocks = order[h, i0:i1]
            blocks = blocks[(blocks >= 0) & (blocks < CQ)]
            sel = [kvi[h, u, :kvc[h, u]] for u in blocks]
            union = np.unique(np.concatenate(sel)) if sel else np.zeros(0, np.int64)
            union = union[(union >= 0) & (union < len(nk))]
            for c0 in range(0, len(union), 1024):
                tiles += int(-(-int(nk[union[c0:c0 + 1024]].sum()) // 32))
    useful *= 4.0 * d
    issued = 4.0 * d * 128 * 32 * tiles
    t = ms_attn * 1e-3
    return {"useful_tflop": round(useful / 1e12, 3), "issued_tflop": round(issued / 1e12, 3),
            "issued_over_useful": round(issued / max(useful, 1.0), 3),
            "useful_tflops": round(useful / t / 1e12, 2), "issued_tflops": round(issued / t / 1e12, 2),
            "useful_frac": round(useful / t / 1e12 / PEAK["mfma_bf16"], 4),
            "issued_frac": round(issued / t / 1e12 / PEAK["mfma_bf16"], 4)}


def host_info():
    """CPU model, logical CPUs, CPUs this process may run on, BLAS threads."""
    model = None
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    try:
        affinity = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        affinity = None
    try:
        from threadpoolctl import threadpool_info
        blas = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        blas = None
    return {"cpu_model": model, "os_cpu_count": os.cpu_count(), "affinity": affinity,
            "blas_threads": blas}


def cpu_baseline(cfg, q, k, v, nheads, variant):
    from oracle import park_oracle as O
    info = host_info()
    mode = cfg.select
    param = cfg.ratio if mode == "topk" else cfg.topp
    t0 = time.perf_counter()
    for h in range(nheads):
        O.park_head(q[h], k[h], v[h], cfg.C, cfg.C, cfg.iters, mode, param, seed=0, head=h,
                    **variant)
    dt = time.perf_counter() - t0
    ms_layer = dt * 1e3 * cfg.H / nheads
    cores = info["blas_threads"] or info["affinity"] or os.cpu_count()
    return {"value": round(ms_layer, 3), "unit": "ms per layer", "cores": int(cores),
            "kind": "oracle",
            "sample": f"{nheads} of {cfg.H} heads of the {cfg.name} layer (full N), "
                      f"whole PARK forward in float64 NumPy ({dt:.1f} s), scaled x{cfg.H / nheads:g}",
            **info}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); PARK shards by "
              f"head with no communication, see the design notes", file=sys.stderr)
        sys.exit(2)
    if args.calibrate_copy:
        calibrate_copy(args.calibrate_copy)
        return
    import numpy as np
    import torch

    from paper_2609_38978_amd import park as P
    from paper_2609_38978_amd import synth

    cfg = synth.CONFIGS[args.workload]
    over = {}
    if args.topp is not None:
        over.update(select="topp", topp=args.topp)
    if args.ratio is not None:
        over.update(select="topk", ratio=args.ratio)
    if args.block is not None:
        over["block"] = args.block
    if args.iters is not None:
        over["iters"] = args.iters
    cfg = cfg.with_(**over)
    q, k, v = synth.make_layer(cfg)
    tdt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    Q, K, V = (torch.from_numpy(a).to(tdt).cuda() for a in (q, k, v))
    C = cfg.C
    mode = cfg.select
    param = cfg.ratio if mode == "topk" else cfg.topp
    reuse = {"recompute": P.PARK_RECOMPUTE, "clusters": P.PARK_REUSE_CLUSTERS,
             "mask": P.PARK_REUSE_CLUSTERS_AND_MASK}[args.reuse]
    variant = {"estimator": args.estimator, "blocks": args.blocks, "key_metric": args.key_metric,
               "alpha": args.alpha}
    prm = P.make_params(C, C, T=cfg.iters, select=mode, ratio=param, topp=param, seed=0,
                        alpha=args.alpha,
                        out_dtype=P.PARK_BF16 if cfg.dtype == "bf16" else P.PARK_F32,
                        estimator={"pama": P.PARK_EST_PAMA,
                                   "qcentroid": P.PARK_EST_QCENTROID}[args.estimator],
                        block_mode={"cluster": P.PARK_BLOCKS_CLUSTER,
                                    "fixed": P.PARK_BLOCKS_FIXED}[args.blocks],
                        key_metric={"qrkc": P.PARK_METRIC_QRKC,
                                    "euclid": P.PARK_METRIC_EUCLID}[args.key_metric])
    ws = P.workspace(Q, C, C)
    st = P.make_state(Q, C, C)
    out = torch.empty(Q.shape, dtype=tdt, device="cuda")
    if reuse != P.PARK_RECOMPUTE:
        # this step's clustering/mask come from the previous step (Q, K); the
        # timed calls run on the drifted Q2, K2
        P.park_forward(Q, K, V, prm, state=st, out=out, ws=ws)
        q2, k2 = synth.perturb_layer(cfg, q, k)
        Q = torch.from_numpy(q2).to(tdt).cuda()
        K = torch.from_numpy(k2).to(tdt).cuda()
        del q2, k2

    def fwd():
        P.park_forward(Q, K, V, prm, reuse=reuse, state=st, out=out, ws=ws)

    for _ in range(args.warmup):
        fwd()
    P.park_check(ws)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)

    # (1) eager launches: the measured value
    stream = torch.cuda.current_stream()
    t0 = time.perf_counter()
    e0.record(stream)
    for _ in range(args.steps):
        fwd()
    e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_eager = e0.elapsed_time(e1) / args.steps
    P.park_check(ws)

    # (2) the same forward captured once in a HIP graph and replayed (reported
    # beside the eager time); every kernel of the layer runs in every replay
    ms_graph = None
    if not args.no_graph:
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            fwd()
        graph.replay()
        torch.cuda.synchronize()
        gs = torch.cuda.current_stream()
        e0.record(gs)
        for _ in range(args.steps):
            graph.replay()
        e1.record(gs)
        torch.cuda.synchronize()
        ms_graph = e0.elapsed_time(e1) / args.steps
        P.park_check(ws)
        del graph
    ms = ms_eager

    # (3) per-kernel HIP events on the launch stream (a separate eager pass)
    P.park_profile_reset()
    P.park_profile_enable(True)
    for _ in range(args.steps):
        fwd()
    torch.cuda.synchronize()
    P.park_profile_enable(False)
    prof = P.park_profile_read()
    P.park_check(ws)
    dense_flops = 4.0 * cfg.N * cfg.N * cfg.d * cfg.H

    # per-kernel share and roofline of the dominant kernel
    stages = {n: {"ms_per_step": round(r["ms"] / args.steps, 4),
                  "launches_per_step": r["launches"] // args.steps} for n, r in prof.items()}
    stage_roof = {}
    for n, r in prof.items():
        wk = kernel_work(n, cfg, st, C)
        if wk is None or not r["launches"]:
            continue
        b_, amt, unit_, pk_ = wk
        a_ms = r["ms"] / r["launches"]
        rate = amt / (a_ms * 1e-3) / (1e12 if unit_ == "flop" else 1e9)
        stage_roof[n] = {"bound": b_, "achieved": round(rate, 3),
                         "unit": "TFLOP/s" if unit_ == "flop" else "GB/s",
                         "frac": round(rate / PEAK[pk_], 4)}
    dom = max(prof, key=lambda n: prof[n]["ms"])
    avg_ms = prof[dom]["ms"] / prof[dom]["launches"]
    work = kernel_work(dom, cfg, st, C)
    roof = None
    if work is not None:
        bound, amount, unit, pk = work
        if unit == "flop":
            ach = amount / (avg_ms * 1e-3) / 1e12
            roof = {"bound": bound, "achieved": round(ach, 3), "peak": PEAK[pk],
                    "unit": "TFLOP/s", "frac": round(ach / PEAK[pk], 4), "traffic": None}
        else:
            ach = amount / (avg_ms * 1e-3) / 1e9
            roof = {"bound": bound, "achieved": round(ach, 2), "peak": PEAK[pk], "unit": "GB/s",
                    "frac": round(ach / PEAK[pk], 4), "traffic": None}
        tb = measured_traffic(cfg.name, dom)
        roof["traffic"] = None if tb is None else round(tb)
        roof["kernel"] = dom
        roof["avg_launch_ms"] = round(avg_ms, 4)

    res = {"metric": METRIC, "value": round(ms, 4), "unit": "ms/layer", "n_gpus": 1,
           "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 4),
           "higher_is_better": False, "scaling": "weak", "vs_baseline": None, "dtype": cfg.dtype,
           "data": "synthetic (seeded clustered-Gaussian DiT-shaped Q/K/V)",
           "config": {"workload": f"{cfg.name}: H={cfg.H} N={cfg.N} d={cfg.d} {cfg.dtype} "
                                  f"B={cfg.block} C={C} T={cfg.iters} {mode} {param}"
                                  + ("" if reuse == P.PARK_RECOMPUTE else f" reuse={args.reuse}")
                                  + "".join(f" {k}={v}" for k, v in variant.items()
                                            if v not in ("pama", "cluster", "qrkc", 0.05)),
                      "H": cfg.H, "N": cfg.N, "d": cfg.d, "B": cfg.block, "C": C, "T": cfg.iters,
                      "select": mode, "param": param, "reuse": args.reuse, **variant},
           "dense_equiv_tflops": round(dense_flops / (ms * 1e-3) / 1e12, 3),
           "timing": "eager park_forward calls, events on the launch stream",
           "graph_ms_per_step": None if ms_graph is None else round(ms_graph, 4),
           "wall_s": round(wall, 3), "stages": stages, "stage_roofline": stage_roof,
           "roofline": roof}
    if "attn_mfma" in prof and prof["attn_mfma"]["launches"]:
        res["attention_flops"] = attention_flops(ws, st, cfg, prof["attn_mfma"]["ms"] /
                                                 prof["attn_mfma"]["launches"])
    if not args.no_cpu_baseline:
        nh = args.cpu_heads if args.cpu_heads is not None else (4 if cfg.N < 50000 else 1)
        res["cpu_baseline"] = cpu_baseline(cfg, q, k, v, min(nh, cfg.H), variant)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
