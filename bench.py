#!/usr/bin/env python3
"""Memory-layer hot path throughput on one MI355X.

One step = one pass of the whole hot path over one batch of T tokens:
product-key search + softmax (mem_search), weighted EmbeddingBag forward
(mem_bag_forward) and backward with value / weight / score gradients
(mem_bag_backward).  Inputs are seeded synthetic tensors already resident in
HBM when the timed region starts; the value gradient accumulates across steps
(zeroing it is the caller's job, outside the step).

Prints one JSON line: throughput (tokens/s), per-stage and per-kernel times
from HIP events recorded inside the timed steps, the roofline of the dominant
kernel, the gather / scatter bandwidths, and the CPU oracle timed on a bounded
sample of the same workload.

    python bench.py [--gpus 1] [--steps 20] [--warmup 3] [--workload pk4m_d2048]
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
sys.path.insert(0, ROOT)

METRIC = "memory-layer tokens/s fwd+bwd (4M keys×2048 bf16); gather HBM GB/s vs peak"
HBM_PEAK_GBPS = 8000.0          # MI355X HBM3E, 8 TB/s
MFMA_BF16_PEAK_TFLOPS = 2500.0  # dense bf16
MFMA_F32_PEAK_TFLOPS = 157.3

KERNELS = ["score_topk", "cartesian", "bag_forward", "sort_by_row", "bag_backward_rows",
           "bag_backward_atomic", "softmax_backward", "search_backward", "topk_sort"]
KERNEL_SOURCES = {
    "score_topk": ["search.hip", "pk_device.h"],
    "topk_sort": ["search.hip", "pk_device.h"],
    "cartesian": ["search.hip", "pk_device.h"],
    "bag_forward": ["bag.hip", "pk_device.h"],
    "bag_backward_atomic": ["bag.hip", "pk_device.h"],
    "softmax_backward": ["bag.hip"],
    "sort_by_row": ["sorted.hip", "pk_device.h"],
    "bag_backward_rows": ["sorted.hip", "pk_device.h"],
    "search_backward": ["search_bwd.hip", "sorted.hip", "pk_device.h"],
    "bag_forward_gated": ["bag.hip", "pk_device.h"],
    "gate_backward": ["bag.hip", "pk_device.h"],
    "qnorm": ["search.hip", "pk_device.h"],
}


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def source_hash(kernel: str) -> str:
    """Hash of the kernel's source files with comments and whitespace removed,
    so a counter summary stays valid across comment-only edits."""
    h = hashlib.sha256()
    for f in KERNEL_SOURCES[kernel]:
        with open(os.path.join(ROOT, "paper_2412_09764_amd", "csrc", f)) as fh:
            src = fh.read()
        src = re.sub(r"/\*.*?\*/", " ", src, flags=re.S)
        src = re.sub(r"//[^\n]*", " ", src)
        h.update("".join(src.split()).encode())
    return h.hexdigest()[:16]


def measured_traffic(kernel: str, workload: str):
    """HBM bytes per launch from the committed rocprofv3 counter summary of this
    kernel and workload, if it was taken on the current kernel source."""
    path = os.path.join(ROOT, "profiles", f"{kernel}_{workload}_counters.txt")
    if not os.path.exists(path):
        return None
    txt = open(path).read()
    m_src = re.search(r"^source_sha256_16:\s*(\S+)", txt, re.M)
    m_b = re.search(r"^hbm_bytes_per_launch:\s*([0-9.eE+]+)", txt, re.M)
    if not m_src or not m_b or m_src.group(1) != source_hash(kernel):
        return None
    return float(m_b.group(1))


def alg_cost(kernel: str, wl, U: int, esz: int):
    """Algorithmic bytes (HBM-bound kernels) or flops (scoring) of one launch."""
    T, H, k, D, S, d = wl.T, wl.H, wl.k, wl.D, wl.S, wl.d
    L = T * H * k
    if kernel == "bag_forward":
        # selected value rows + output rows + (idx int64, w fp32) per lookup
        return "hbm", L * D * esz + T * D * esz + L * 12
    if kernel == "bag_backward_rows":
        # per touched row: value row read, segment start, and either the fp32 gradient
        # row read + write (dense) or written once with its row id (sparse);
        # per token: dy row; per lookup: sorted row key, lookup id, w, grad_w
        if wl.sparse_grad:
            return "hbm", U * D * (esz + 4) + U * (4 + 8) + T * D * esz + L * 16
        return "hbm", U * D * (esz + 8) + U * 4 + T * D * esz + L * 16
    if kernel == "bag_backward_atomic":
        # per lookup: value row read, fp32 gradient row read + write, (idx, w, grad_w); dy per token
        return "hbm", L * D * (esz + 8) + T * D * esz + L * 16
    if kernel == "bag_forward_gated":
        # the gather, plus the gate read and the gated and un-gated output rows
        return "hbm", L * D * esz + 3 * T * D * esz + L * 12
    if kernel == "gate_backward":
        # d_out, gate, un-gated bag read; dy (value dtype) and fp32 gate gradient written
        return "hbm", T * D * (4 * esz + 4)
    if kernel == "qnorm":
        # each query read once, its (mean, rstd) written
        return "hbm", T * H * wl.n * esz_q(wl) + T * H * 8
    if kernel == "score_topk":
        return "mfma", 2.0 * T * H * 2 * S * d
    if kernel == "sort_by_row":
        return "hbm", None
    return "hbm", None


def esz_q(wl):
    return 2 if wl.key_dtype == "bf16" else 4


def hbm_rate(alg_bytes, ms):
    ach = alg_bytes / (ms / 1e3) / 1e9
    return {"bound": "hbm", "achieved": round(ach, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
            "frac": round(ach / HBM_PEAK_GBPS, 4), "alg_bytes_per_launch": alg_bytes, "ms": round(ms, 4)}


def run_cpu_baseline(wl, q, K, V, dy, budget_s: float):
    """The fp64 oracle on the first tokens of the batch, until ~budget_s seconds
    of oracle time have been spent (at least 8 tokens).  One BLAS thread."""
    import numpy as np
    import torch
    from threadpoolctl import threadpool_info, threadpool_limits

    import oracle

    host_cores = len(os.sched_getaffinity(0))
    blas_default = max((i.get("num_threads", 0) for i in threadpool_info()
                        if i.get("user_api") == "blas"), default=None)
    Kh = K.float().cpu().double().numpy()
    spent = 0.0
    done = 0
    chunk = 8
    with threadpool_limits(limits=1):
        while done < wl.T and (spent < budget_s or done < 8):
            t0, t1 = done, min(wl.T, done + chunk)
            qh = q[t0:t1].float().cpu().double().numpy()
            dyh = dy[t0:t1].float().cpu().double().numpy()
            c0 = time.perf_counter()
            s = oracle.search(qh, Kh, wl.k)
            spent += time.perf_counter() - c0
            # the value rows this chunk selects (host copy, not timed)
            rows, inv = np.unique(s["idx"], return_inverse=True)
            Vh = V[torch.from_numpy(rows).to(V.device)].float().cpu().double().numpy()
            local = inv.reshape(s["idx"].shape)
            c0 = time.perf_counter()
            oracle.bag_forward(Vh, local.reshape(t1 - t0, -1), s["w"].reshape(t1 - t0, -1))
            oracle.bag_backward_rows(dyh, Vh, local, s["w"], wl.H, wl.k)
            spent += time.perf_counter() - c0
            done = t1
    return {"value": done / spent, "unit": "tokens/s", "cores": 1, "kind": "oracle",
            "host_cores_available": host_cores, "blas_threads_default": blas_default,
            "blas_threads_used": 1,
            "sample": (f"first {done} of {wl.T} tokens of {wl.name}: search + softmax + bag "
                       f"forward + bag backward (touched rows), fp64 NumPy, one BLAS thread, "
                       f"{spent:.1f} s")}


def bwd_sweep(args):
    """Both value-gradient strategies of Sec. 3.1.4 (lookups sorted by row, or
    fp32 atomic adds) timed over value widths D and token counts T at H = 4,
    k = 32 over a table of 2^20 rows, with uniformly drawn indices and
    softmax-like weights (seeded).  Each entry is the mean of `steps` calls of
    mem_bag_backward (dense accumulation, grad_w and grad_scores included)
    after one warm-up call, timed with events on the launch stream."""
    import torch

    import paper_2412_09764_amd as pk

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    N, H, k = 1 << 20, 4, 32
    g = torch.Generator(device=dev)
    rows = []
    for vdt, D in (("f32", 64), ("bf16", 64), ("bf16", 128), ("bf16", 256), ("bf16", 512),
                   ("bf16", 1024), ("bf16", 2048)):
        dt = torch.float32 if vdt == "f32" else torch.bfloat16
        g.manual_seed(D)
        V = (torch.randn((N, D), generator=g, device=dev) * 0.02).to(dt)
        gv = torch.zeros((N, D), dtype=torch.float32, device=dev)
        for T in (256, 1024, 2048, 4096, 8192, 16384):
            idx = torch.randint(0, N, (T, H, k), generator=g, device=dev)
            w = torch.softmax(torch.randn((T, H, k), generator=g, device=dev), dim=-1).contiguous()
            dy = torch.randn((T, D), generator=g, device=dev).to(dt)
            gw = torch.empty((T, H, k), dtype=torch.float32, device=dev)
            gz = torch.empty_like(gw)
            ent = {"dtype": vdt, "D": D, "T": T, "lookups": T * H * k}
            for mode in ("sorted", "atomic"):
                ws = torch.empty(max(1, pk.mem_bag_backward_workspace_size(T, H, k, N, D, mode)),
                                 dtype=torch.uint8, device=dev)
                run = lambda: pk.mem_bag_backward(dy, V, idx, w, grad_values=gv, grad_w=gw,  # noqa: E731
                                                  grad_scores=gz, mode=mode, workspace=ws)
                run()
                torch.cuda.synchronize()
                a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                a.record()
                for _ in range(args.steps):
                    run()
                b.record()
                torch.cuda.synchronize()
                ent[f"{mode}_ms"] = round(a.elapsed_time(b) / args.steps, 4)
                del ws
            ent["faster"] = "sorted" if ent["sorted_ms"] <= ent["atomic_ms"] else "atomic"
            log(f"[sweep] {ent}")
            rows.append(ent)
        del V, gv
        torch.cuda.empty_cache()
    print(json.dumps({"bwd_sweep": rows, "rows_N": N, "heads": H, "k": k,
                      "index_distribution": "uniform", "steps": args.steps}), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="pk4m_d2048")
    ap.add_argument("--bwd-mode", default="auto", choices=["auto", "atomic", "sorted"])
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="before the steps, run one plain device copy of this many MiB "
                         "(reference for scaling memory counters)")
    ap.add_argument("--bwd-sweep", action="store_true",
                    help="instead of the step: time both value-gradient strategies over a "
                         "grid of value widths and token counts (uniform indices), one JSON line")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: the library has no multi-GPU path "
              "(run with --gpus 1).", file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2412_09764_amd as pk
    from paper_2412_09764_amd.inputs import WORKLOADS, gen_dy, gen_queries, gen_subkeys, gen_values

    pk.load()
    if args.bwd_sweep:
        bwd_sweep(args)
        return
    wl = WORKLOADS[args.workload]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    esz = 2 if wl.value_dtype == "bf16" else 4
    T, H, k, N, D = wl.T, wl.H, wl.k, wl.N, wl.D
    log(f"[bench] workload {wl.name}: N={N} D={D} H={H} k={k} T={T}; generating inputs")

    q = gen_queries(wl, dev)
    K = gen_subkeys(wl, dev)
    V = gen_values(wl, dev)
    dy = gen_dy(wl, dev)
    idx = torch.empty((T, H, k), dtype=torch.int64, device=dev)
    w = torch.empty((T, H, k), dtype=torch.float32, device=dev)
    score = torch.empty((T, H, k), dtype=torch.float32, device=dev)
    y = torch.empty((T, D), dtype=V.dtype, device=dev)
    gw = torch.empty((T, H, k), dtype=torch.float32, device=dev)
    gz = torch.empty((T, H, k), dtype=torch.float32, device=dev)
    ws_s = torch.empty(pk.mem_search_workspace_size(T, H, wl.S, k), dtype=torch.uint8, device=dev)
    sparse = wl.sparse_grad
    mode = "sorted" if sparse else args.bwd_mode
    ws_b = torch.empty(max(1, pk.mem_bag_backward_workspace_size(T, H, k, N, D, mode)),
                       dtype=torch.uint8, device=dev)
    if sparse:
        cap = min(T * H * k, N)
        rows_out = torch.empty((cap,), dtype=torch.int64, device=dev)
        grows = torch.empty((cap, D), dtype=torch.float32, device=dev)
        gv = None
    else:
        gv = torch.zeros((N, D), dtype=torch.float32, device=dev)
    torch.cuda.synchronize()
    if args.copy_calibration_mib > 0:
        nfl = args.copy_calibration_mib * (1 << 20) // 4
        src = torch.ones(nfl, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
        log(f"[bench] copy calibration: {args.copy_calibration_mib} MiB read + written")
    # practical streaming peak of this machine: a plain 4 GiB device-to-device copy
    src = torch.empty(1 << 30, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    src.fill_(1.0)
    dst.copy_(src)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(5):
        dst.copy_(src)
    e1.record()
    torch.cuda.synchronize()
    copy_gbps = 5 * 2 * src.numel() * 4 / (e0.elapsed_time(e1) / 1e3) / 1e9
    # two streaming references with the backward's mix of reads and writes:
    # c = a + b over fp32 (two reads per write), and g += v with v bf16 and g
    # fp32 in place (the value-gradient update: 2 + 4 bytes read, 4 written)
    c = torch.empty_like(src)
    torch.add(src, dst, out=c)
    e0.record()
    for _ in range(5):
        torch.add(src, dst, out=c)
    e1.record()
    torch.cuda.synchronize()
    add_gbps = 5 * 3 * src.numel() * 4 / (e0.elapsed_time(e1) / 1e3) / 1e9
    del c
    vb = torch.ones(src.numel(), dtype=torch.bfloat16, device=dev)
    dst.add_(vb)
    e0.record()
    for _ in range(5):
        dst.add_(vb)
    e1.record()
    torch.cuda.synchronize()
    rmw_gbps = 5 * (2 + 4 + 4) * src.numel() / (e0.elapsed_time(e1) / 1e3) / 1e9
    del vb
    # the same in place over fp32 only (g += h: 4 + 4 bytes read, 4 written)
    dst.add_(src)
    e0.record()
    for _ in range(5):
        dst.add_(src)
    e1.record()
    torch.cuda.synchronize()
    rmw32_gbps = 5 * 3 * src.numel() * 4 / (e0.elapsed_time(e1) / 1e3) / 1e9
    del src, dst
    log(f"[bench] device copy: {copy_gbps:.0f} GB/s (read + write); a + b: {add_gbps:.0f} GB/s; "
        f"fp32 += bf16 in place: {rmw_gbps:.0f} GB/s; fp32 += fp32 in place: {rmw32_gbps:.0f} GB/s")
    log("[bench] inputs resident; warming up")

    L = pk.load()
    import ctypes
    st = torch.cuda.current_stream().cuda_stream
    BF = pk.BF16 if wl.value_dtype == "bf16" else pk.F32
    KDT = pk.BF16 if wl.key_dtype == "bf16" else pk.F32
    m = pk.BWD_MODES[mode]
    nrows = ctypes.c_int64(0)

    def step(ev=None):
        if ev is not None:
            ev[0].record()
        pk._check(L.mem_search(q.data_ptr(), KDT, K.data_ptr(), KDT, T, H, wl.n, wl.S, k,
                               idx.data_ptr(), w.data_ptr(), score.data_ptr(), None,
                               ws_s.data_ptr(), ws_s.numel(), st))
        if ev is not None:
            ev[1].record()
        pk._check(L.mem_bag_forward(V.data_ptr(), BF, N, D, idx.data_ptr(), w.data_ptr(), T,
                                    H * k, y.data_ptr(), st))
        if ev is not None:
            ev[2].record()
        if sparse:
            pk._check(L.mem_bag_backward_sparse(dy.data_ptr(), V.data_ptr(), BF, N, D,
                                                idx.data_ptr(), w.data_ptr(), T, H, k,
                                                rows_out.data_ptr(), grows.data_ptr(), cap,
                                                ctypes.addressof(nrows), gw.data_ptr(),
                                                gz.data_ptr(), ws_b.data_ptr(), ws_b.numel(), st))
        else:
            pk._check(L.mem_bag_backward(dy.data_ptr(), V.data_ptr(), BF, N, D, idx.data_ptr(),
                                         w.data_ptr(), T, H, k, gv.data_ptr(), gw.data_ptr(),
                                         gz.data_ptr(), m, ws_b.data_ptr(), ws_b.numel(), st))
        if ev is not None:
            ev[3].record()

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    log(f"[bench] timing {args.steps} steps")

    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
    pk.mem_timer_start(*KERNELS)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(evs[i])
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    pk.mem_timer_stop()
    launches = pk.mem_timer_read()
    # candidate records the scoring kernel wrote in the last step: the run
    # counts (one per run of 32 tokens, head and half) follow the candidate
    # slots in the search workspace (256 slots of 8 bytes per (token, head,
    # half) row, tokens rounded up to groups of 32, each region 256-byte
    # aligned)
    nruns = (T + 31) // 32 * H * 2
    cnt_off = (nruns * 32 * 256 * 8 + 255) // 256 * 256
    records = int(ws_s[cnt_off:cnt_off + nruns * 4].view(torch.int32).sum().item())
    ms_per_step = elapsed * 1e3 / args.steps
    log(f"[bench] {ms_per_step:.3f} ms/step")

    stages = {"search": 0.0, "bag_forward": 0.0, "bag_backward": 0.0}
    for e in evs:
        stages["search"] += e[0].elapsed_time(e[1])
        stages["bag_forward"] += e[1].elapsed_time(e[2])
        stages["bag_backward"] += e[2].elapsed_time(e[3])
    stages = {s: round(v / args.steps, 4) for s, v in stages.items()}
    per_kernel = {}
    for pos, ms in launches:
        per_kernel.setdefault(KERNELS[pos], []).append(ms)
    kernel_ms = {kname: round(sum(v) / len(v), 4) for kname, v in per_kernel.items()}

    # Search backward (gradients into queries and sub-keys): measured on its
    # own, after the timed steps; not part of the step's throughput.
    gq = torch.empty((T, H, wl.n), dtype=torch.float32, device=dev)
    gK = torch.zeros((H, 2, wl.S, wl.d), dtype=torch.float32, device=dev)
    ws_sb = torch.empty(max(1, pk.load().mem_search_backward_workspace_size(T, H, wl.S, k)),
                        dtype=torch.uint8, device=dev)
    def sbwd():
        pk._check(L.mem_search_backward(q.data_ptr(), KDT, K.data_ptr(), KDT, T, H, wl.n, wl.S, k,
                                        idx.data_ptr(), gz.data_ptr(), gq.data_ptr(),
                                        gK.data_ptr(), ws_sb.data_ptr(), ws_sb.numel(), st))
    sbwd()
    torch.cuda.synchronize()
    pk.mem_timer_start("search_backward")
    for _ in range(args.steps):
        sbwd()
    torch.cuda.synchronize()
    pk.mem_timer_stop()
    sb = [ms for _, ms in pk.mem_timer_read()]
    search_bwd_ms = sum(sb) / len(sb)
    del gq, gK, ws_sb

    # Both value-gradient strategies of Sec. 3.1.4 (sorted by row, fp32 atomic
    # adds) on the last step's selection, each timed on its own after the
    # steps with events on the launch stream: the evidence behind what
    # PKMEM_BWD_AUTO picks.  (The sparse gradient has the sorted form only.)
    strategies = None
    if not sparse:
        strategies = {}
        for mname in ("sorted", "atomic"):
            wsm = torch.empty(max(1, pk.mem_bag_backward_workspace_size(T, H, k, N, D, mname)),
                              dtype=torch.uint8, device=dev)
            mm = pk.BWD_MODES[mname]

            def bwd_once():
                pk._check(L.mem_bag_backward(dy.data_ptr(), V.data_ptr(), BF, N, D, idx.data_ptr(),
                                             w.data_ptr(), T, H, k, gv.data_ptr(), gw.data_ptr(),
                                             gz.data_ptr(), mm, wsm.data_ptr(), wsm.numel(), st))
            bwd_once()
            torch.cuda.synchronize()
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            for _ in range(args.steps):
                bwd_once()
            b.record()
            torch.cuda.synchronize()
            strategies[f"{mname}_ms"] = round(a.elapsed_time(b) / args.steps, 4)
            del wsm
        log(f"[bench] value-gradient strategies: {strategies}")

    # Memory+ gating (the gated gather and the gate backward): measured on
    # their own after the timed steps, on the last step's selection.
    gate = dy.clone()                       # N(0,1) gate pre-activation, value dtype
    g_out = torch.empty_like(dy)
    g_y = torch.empty_like(dy)
    g_dy = torch.empty_like(dy)
    g_dg = torch.empty((T, D), dtype=torch.float32, device=dev)
    idx2, w2 = idx.view(T, -1), w.view(T, -1)
    def gated():
        pk.mem_bag_forward_gated(V, idx2, w2, gate, out=g_out, y_out=g_y)
    def gate_bwd():
        pk.mem_gate_backward(dy, gate, g_y, dy_out=g_dy, grad_gate=g_dg)
    gplus = {}
    for name, fn in (("bag_forward", gated), ("gate_backward", gate_bwd)):
        fn()
        torch.cuda.synchronize()
        pk.mem_timer_start(name)
        for _ in range(args.steps):
            fn()
        torch.cuda.synchronize()
        pk.mem_timer_stop()
        v = [ms for _, ms in pk.mem_timer_read()]
        gplus[name] = sum(v) / len(v)
    del gate, g_out, g_y, g_dy, g_dg

    # Query normalisation fused into the search (and its backward), measured
    # on its own after the timed steps on the same queries.
    idx_qn, w_qn = torch.empty_like(idx), torch.empty_like(w)
    def search_qn():
        pk.mem_search_qnorm(q, K, k, 1e-5, idx_out=idx_qn, w_out=w_qn, want_score=False,
                            workspace=ws_s)
    search_qn()
    torch.cuda.synchronize()
    pk.mem_timer_start("qnorm", "score_topk", "cartesian", "topk_sort")
    for _ in range(args.steps):
        search_qn()
    torch.cuda.synchronize()
    pk.mem_timer_stop()
    qn = {}
    for pos, ms in pk.mem_timer_read():
        qn.setdefault(("qnorm", "score_topk", "cartesian", "topk_sort")[pos], []).append(ms)
    qn = {kn: sum(v) / len(v) for kn, v in qn.items()}
    gq = torch.empty((T, H, wl.n), dtype=torch.float32, device=dev)
    gK = torch.zeros((H, 2, wl.S, wl.d), dtype=torch.float32, device=dev)
    ws_sb = torch.empty(max(1, pk.load().mem_search_backward_workspace_size(T, H, wl.S, k)),
                        dtype=torch.uint8, device=dev)
    def sbwd_qn():
        pk.mem_search_backward_qnorm(q, K, idx_qn, gz, 1e-5, grad_q=gq, grad_subkeys=gK,
                                     workspace=ws_sb)
    sbwd_qn()
    torch.cuda.synchronize()
    pk.mem_timer_start("qnorm", "search_backward")
    for _ in range(args.steps):
        sbwd_qn()
    torch.cuda.synchronize()
    pk.mem_timer_stop()
    sbq = [ms for _, ms in pk.mem_timer_read()]
    search_bwd_qn_ms = sum(sbq) / args.steps
    del gq, gK, ws_sb, idx_qn, w_qn

    # Extra key-value pairs (16 per token and head) and the fixed sink pair,
    # each scored inside the cartesian kernel, and the sink's search backward
    # (its grad_q term and the deterministic grad_sink sum): measured on their
    # own after the timed steps on the same queries.
    def kernel_avg(fn, names):
        fn()
        torch.cuda.synchronize()
        pk.mem_timer_start(*names)
        for _ in range(args.steps):
            fn()
        torch.cuda.synchronize()
        pk.mem_timer_stop()
        acc = {}
        for pos, ms in pk.mem_timer_read():
            acc[names[pos]] = acc.get(names[pos], 0.0) + ms
        return {kn: v / args.steps for kn, v in acc.items()}

    r_ex = 16
    ex_idx = torch.randint(0, N, (T, H, r_ex), generator=torch.Generator().manual_seed(11),
                           dtype=torch.int64).to(dev)
    sink_keys = (torch.randn((H, wl.n), generator=torch.Generator().manual_seed(12)) / 16).to(q.dtype).to(dev)
    idx_x = torch.empty((T, H, k + r_ex), dtype=torch.int64, device=dev)
    w_x = torch.empty((T, H, k + r_ex), dtype=torch.float32, device=dev)
    extra_ms = kernel_avg(lambda: pk.mem_search_extra(q, K, k, ex_idx, idx_out=idx_x, w_out=w_x,
                                                      want_score=False, workspace=ws_s),
                          ("cartesian",))
    del idx_x, w_x, ex_idx
    idx_sk = torch.empty((T, H, k + 1), dtype=torch.int64, device=dev)
    w_sk = torch.empty((T, H, k + 1), dtype=torch.float32, device=dev)
    sink_ms = kernel_avg(lambda: pk.mem_search_sink(q, K, k, sink_keys, N, idx_out=idx_sk,
                                                    w_out=w_sk, want_score=False, workspace=ws_s),
                         ("cartesian",))
    gz_sk = (torch.randn((T, H, k + 1), generator=torch.Generator().manual_seed(13)) * 0.01).to(dev)
    gq = torch.empty((T, H, wl.n), dtype=torch.float32, device=dev)
    gK = torch.zeros((H, 2, wl.S, wl.d), dtype=torch.float32, device=dev)
    gS = torch.zeros((H, wl.n), dtype=torch.float32, device=dev)
    ws_sk = torch.empty(max(1, pk.load().mem_search_backward_sink_workspace_size(T, H, wl.n, wl.S, k)),
                        dtype=torch.uint8, device=dev)
    sink_bwd_ms = kernel_avg(lambda: pk.mem_search_backward_sink(q, K, idx_sk, gz_sk, sink_keys,
                                                                 grad_q=gq, grad_subkeys=gK,
                                                                 grad_sink=gS, workspace=ws_sk),
                             ("search_backward",))
    del idx_sk, w_sk, gz_sk, gq, gK, gS, ws_sk, sink_keys

    # touched rows of the last step's selection (outside the timed region)
    uniq, counts = torch.unique(idx.view(-1), return_counts=True)
    U = int(uniq.numel())
    max_mult = int(counts.max().item())

    def bw(kname):
        if kname not in kernel_ms:
            return None
        bound, cost = alg_cost(kname, wl, U, esz)
        if cost is None:
            return None
        sec = kernel_ms[kname] / 1e3
        if bound == "mfma":
            peak = MFMA_BF16_PEAK_TFLOPS if wl.key_dtype == "bf16" else MFMA_F32_PEAK_TFLOPS
            ach = cost / sec / 1e12
            return {"bound": "mfma", "achieved": round(ach, 2), "peak": peak, "unit": "TFLOP/s",
                    "frac": round(ach / peak, 4), "flops_per_launch": cost, "ms": kernel_ms[kname]}
        ach = cost / sec / 1e9
        return {"bound": "hbm", "achieved": round(ach, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                "frac": round(ach / HBM_PEAK_GBPS, 4), "alg_bytes_per_launch": cost,
                "ms": kernel_ms[kname]}

    dominant = max((kn for kn in kernel_ms if alg_cost(kn, wl, U, esz)[1] is not None),
                   key=lambda kn: kernel_ms[kn])
    roof = bw(dominant)
    traffic = measured_traffic(dominant, wl.name)
    roofline = {"kernel": dominant, "bound": roof["bound"], "achieved": roof["achieved"],
                "peak": roof["peak"], "unit": roof["unit"], "frac": roof["frac"],
                "traffic": traffic}

    # the scoring kernel computes the products of its first P1 sub-key chunks
    # twice (first threshold, then the final collection) and of the rest once:
    # P1 = an eighth of the chunks from 128 chunks up, a quarter from 32, else
    # half of them, all of them when k > 32 (2 sweeps); the MFMA work it
    # executes is that multiple of the algorithmic flops priced above
    search_roof = bw("score_topk")
    if search_roof and search_roof["bound"] == "mfma":
        search_roof = dict(search_roof, candidate_records=records,
                           candidates_per_row=round(records / (T * H * 2), 2))
        nch = -(-wl.S // 64)
        P = nch if wl.k > 32 else ((nch + 7) // 8 if nch >= 128 else (nch + 3) // 4 if nch >= 32 else (nch + 1) // 2)
        sweeps = (nch + P) / nch
        search_roof = dict(search_roof, sweeps=round(sweeps, 4),
                           executed_TFLOPs=round(sweeps * search_roof["achieved"], 2))

    scatter = bw("bag_backward_rows") or bw("bag_backward_atomic")
    if scatter:
        # against the in-place fp32 += bf16 stream measured above (the same mix of
        # reads and writes as the value-gradient update)
        scatter = dict(scatter, frac_of_stream_rmw=round(scatter["achieved"] / rmw_gbps, 4))

    cpu = None
    if not args.no_cpu_baseline:
        log("[bench] timing the CPU oracle on a sample")
        cpu = run_cpu_baseline(wl, q, K, V, dy, args.cpu_seconds)

    out = {
        "metric": METRIC,
        "value": round(T / (ms_per_step / 1e3), 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": wl.value_dtype,
        "data": "synthetic",
        "config": {"workload": wl.name, "keys": N, "sub_keys_per_half": wl.S, "heads": H,
                   "query_dim": wl.n, "value_dim": D, "k": k, "tokens": T,
                   "value_table_GiB": round(N * D * esz / 2**30, 2),
                   "value_grad": "sparse rows" if sparse else "dense fp32", "bwd_mode": mode},
        "roofline": roofline,
        "cpu_baseline": cpu,
        "stages_ms": stages,
        "kernels_ms": kernel_ms,
        "gather": bw("bag_forward"),
        "scatter": scatter,
        "bwd_strategies_ms": strategies,
        "search": search_roof,
        "search_backward_ms": round(search_bwd_ms, 4),
        "memory_plus": {
            "bag_forward_gated_ms": round(gplus["bag_forward"], 4),
            "gate_backward_ms": round(gplus["gate_backward"], 4),
            "gated_gather": dict(hbm_rate(alg_cost("bag_forward_gated", wl, U, esz)[1], gplus["bag_forward"]),
                                 traffic=measured_traffic("bag_forward_gated", wl.name)),
            "gate_backward": dict(hbm_rate(alg_cost("gate_backward", wl, U, esz)[1], gplus["gate_backward"]),
                                  traffic=measured_traffic("gate_backward", wl.name)),
        },
        "query_norm": {
            "qnorm_ms": round(qn["qnorm"], 4),
            "score_topk_ms": round(qn["score_topk"], 4),
            "topk_sort_ms": round(qn["topk_sort"], 4),
            "cartesian_ms": round(qn["cartesian"], 4),
            "search_backward_ms": round(search_bwd_qn_ms, 4),
            "qnorm": dict(hbm_rate(alg_cost("qnorm", wl, U, esz)[1], qn["qnorm"]),
                          traffic=measured_traffic("qnorm", wl.name)),
        },
        "extra_pairs": {"r": r_ex, "cartesian_ms": round(extra_ms["cartesian"], 4)},
        "sink_pair": {"cartesian_ms": round(sink_ms["cartesian"], 4),
                      "search_backward_ms": round(sink_bwd_ms["search_backward"], 4)},
        "stream_copy_GBps": round(copy_gbps, 1),
        "stream_add_GBps": round(add_gbps, 1),
        "stream_rmw_bf16_f32_GBps": round(rmw_gbps, 1),
        "stream_rmw_f32_GBps": round(rmw32_gbps, 1),
        "touched_rows": U,
        "max_row_multiplicity": max_mult,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
