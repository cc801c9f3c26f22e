"""Benchmark of the SAF3R global-attention hot path on one MI355X.

A step is one pass of the whole path over one layer: block pooling
(saf3r_estimate_blocks), selection (saf3r_select_blocks) and attention over
the kept blocks (saf3r_sparse_attention), inputs resident in HBM. Default
workload: 100 frames x 1374 tokens = 137400 tokens, 16 heads x 64, bf16,
table with 6 frame-local and 10 Top-K heads (target block sparsity 95%).

Prints one JSON line: dense-equivalent TFLOP/s (4 N^2 64 H per layer over
the measured step time) with ms per step, the attention kernel's roofline,
the estimation kernel's HBM rate, the dense baseline (every head dense: the
shared-tile dense kernel) and the CPU oracle timed on a bounded sample of the
same workload.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "ms per global-attn layer + dense-equiv TFLOP/s at S=100×1374 tok, 16 heads"
PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_F32_TFLOPS = 157.3     # MI355X fp32 matrix
PEAK_F64_TFLOPS = 78.6      # MI355X fp64 (matrix and vector)
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "attn_traffic.json")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def kept_flops(idx, cnt, table, n, nb):
    """Algorithmic attention FLOP: sum over kept (query block, key block)
    pairs of 4 * n_i * n_j * 64, counting valid tokens only."""
    last = n - (nb - 1) * 64
    rows = np.full(nb, 64, np.int64)
    rows[-1] = last
    total = 0
    for h, (pattern, _) in enumerate(table):
        if pattern == 0:
            total += 4 * n * n * 64
            continue
        c = cnt[h].astype(np.int64)
        listed = np.arange(idx.shape[2])[None, :] < c[:, None]
        has_last = ((idx[h] == nb - 1) & listed).any(axis=1)
        keys = 64 * c - (64 - last) * has_last
        total += int(4 * 64 * np.sum(rows * keys))
    return total


def source_sha(path):
    return hashlib.sha256(open(path, "rb").read()).hexdigest()[:16]


def recorded_traffic(workload):
    """HBM bytes per attention launch (for the 24-layer stack, the sum over
    the attention launches of one pass) from the committed rocprofv3 counter
    runs, if they were taken on the current kernel source."""
    try:
        rec = json.load(open(TRAFFIC_FILE))
    except (OSError, ValueError):
        return None
    cur = source_sha(os.path.join(ROOT, "paper_2607_03612_amd", "csrc", "attn.hip"))
    r = rec.get(workload)
    if not r or r.get("attn_source_sha") != cur:
        return None
    return r.get("bytes_per_launch")


def sample_rows(nb, rows_per_head, seed=0):
    """The seeded query blocks the oracle sample covers (the same for every head)."""
    return sorted(int(i) for i in np.random.default_rng(seed).choice(nb, size=min(rows_per_head, nb),
                                                                     replace=False))


def oracle_sample(w, q, k, v, table, rows_per_head, seed=0, results=None):
    """The fp64 oracle on a seeded sample of query blocks of every head.

    Per head, the full per-head work (widening to fp64, pooling every key
    block of a Top-K head) is timed once; the per-query-block work (probe,
    scores, selection, attention) is timed on the sample and scaled to all
    query blocks. Returns (estimated seconds per layer, sampled rows per head);
    with `results` (a dict), also keeps each sampled row's list, margin and
    output under (head, block)."""
    import oracle as O

    nb, n, T = w.nb, w.tokens, w.tokens_per_frame
    rows = sample_rows(nb, rows_per_head, seed)
    est = 0.0
    for h, (pattern, topk) in enumerate(table):
        t0 = time.perf_counter()
        qh, kh, vh = (O.to_f64(x[h], w.dtype) for x in (q, k, v))
        kbar = O.pool_blocks(kh, 64) if pattern == O.TOPK else None
        t1 = time.perf_counter()
        for i in rows:
            r = O.block_range(i, n, 64)
            srow = None
            if pattern == O.TOPK:
                qbar = O.pool_blocks(qh[r.start:r.stop], 64)
                srow = O.block_scores(qbar, kbar)[0]
                lst, margin = O.topk_row(srow, topk)
            elif pattern == O.FRAME_LOCAL:
                lst, margin = O.frame_local_row(i, n, T, 64), None
            else:
                lst, margin = np.arange(nb), None
            ref = O.attend_block(qh, kh, vh, i, lst, 64)
            if results is not None:
                results[(h, i)] = (lst, margin, ref[0], srow)
        t2 = time.perf_counter()
        est += (t1 - t0) + (t2 - t1) * nb / len(rows)
    return est, len(rows)


def parity_sample(res, sampled, out_sampled, idx_h, cnt_h, table, n, dtype, qkv):
    """The timed step's lists and outputs on the oracle sample's query blocks
    against the oracle. A list must equal the oracle's where its Top-K margin
    exceeds 1e-6; on a near-tie row (margin at most 1e-6) it must be a valid
    top-k of the oracle's scores (every kept score at least the k-th minus
    1e-6, every dropped one at most the (k+1)-th plus 1e-6), and the output
    is compared with the oracle's attention over the GPU's own list. Outputs
    within the dtype's bound."""
    import oracle as O
    from tests.parity import valid_topk

    offset, pos = {}, 0
    for i in sampled:
        offset[i] = pos
        pos += min(64, n - i * 64)
    equal = near = mismatch = 0
    err = 0.0
    for (h, i), (lst, margin, ref, srow) in res.items():
        if table[h][0] != 0:  # dense heads carry no list
            c = int(cnt_h[h, i])
            got_list = idx_h[h, i, :c]
            if np.array_equal(got_list, lst):
                equal += 1
            elif margin is not None and margin <= 1e-6 and valid_topk(got_list, srow, table[h][1]):
                near += 1
                qh, kh, vh = (O.to_f64(x[h], dtype) for x in qkv)
                ref = O.attend_block(qh, kh, vh, i, got_list, 64)[0]
            else:
                mismatch += 1
                continue
        got = out_sampled[h, offset[i]:offset[i] + ref.shape[0]]
        err = max(err, float(np.max(np.abs(got - ref))))
    return {"query_blocks": len(res), "lists_equal": equal, "near_ties_valid_differing": near,
            "list_mismatches": mismatch, "max_abs_err": err,
            "bound": 2e-2 if dtype == "bf16" else 1e-4}


def host_cpus():
    """(usable cores, CPU model) of the machine the oracle runs on."""
    try:
        usable = len(os.sched_getaffinity(0))
    except AttributeError:
        usable = os.cpu_count() or 1
    model = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return usable, model


def single_threaded():
    """A context in which the oracle's BLAS calls use one thread, so the
    baseline's core count is exact: the oracle's per-row Python loop is
    single-threaded, and only its small matrix products could fan out."""
    import contextlib

    try:
        import threadpoolctl

        return threadpoolctl.threadpool_limits(limits=1)
    except Exception:
        return contextlib.nullcontext()


def event_ms(torch, fn, reps):
    """Mean milliseconds of ``fn`` over ``reps`` launches. An untimed first
    launch is still running when the start event is queued, so the timed
    launches follow it back to back without host latency."""
    fn()
    torch.cuda.synchronize()
    fn()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(reps):
        fn()
    b.record()
    torch.cuda.synchronize()
    return a.elapsed_time(b) / reps


def measure_next_rows(P, torch, w, tq, tk, tv, out, table):
    H, N, nb, S, T = w.heads, w.tokens, w.nb, w.frames, w.tokens_per_frame
    dev = tq.device
    res = {}
    # uniform stride 7 on every head: 137400 queries x 19629 keys per head
    stride = 7
    st_tab = [(P.STRIDE, stride)] * H
    ms = event_ms(torch, lambda: P.sparse_attention(tq, tk, tv, st_tab, S, T, out=out), 2)
    flop = 4 * 64 * N * (-(-N // stride)) * H
    res["stride_attention"] = {"stride": stride, "ms": round(ms, 3),
                               "tflops": round(flop / (ms * 1e-3) / 1e12, 1)}
    # paper-literal global probe on the Top-K heads of the table
    g_tab = [(P.GLOBAL_PROBE, p) if c == P.TOPK else (c, p) for c, p in table]
    cap = P.index_capacity(g_tab, S, T)
    qp, kp = P.estimate_blocks(tq, tk, g_tab, S, T)
    idx = torch.empty((H, nb, cap), dtype=torch.int32, device=dev)
    cnt = torch.empty((H, nb), dtype=torch.int32, device=dev)
    ms = event_ms(torch, lambda: P.select_blocks(qp, kp, g_tab, S, T, cap, idx, cnt), 5)
    res["global_probe_select"] = {"heads": sum(c == P.GLOBAL_PROBE for c, _ in g_tab), "ms": round(ms, 4)}
    # per-frame cosine Top-K (2 key blocks per frame) on 1024-wide bf16 features
    dim = 1024
    feats = (torch.randn((N, dim), device=dev, generator=torch.Generator(device=dev).manual_seed(0))
             .to(torch.bfloat16))
    c_tab = [(P.COSINE_TOPK, 2)] * H
    ccap = P.index_capacity(c_tab, S, T)
    cidx = torch.empty((H, nb, ccap), dtype=torch.int32, device=dev)
    ccnt = torch.empty((H, nb), dtype=torch.int32, device=dev)
    ws = torch.empty(P.cosine_workspace_bytes(S, T, dim, H) // 8, dtype=torch.float64, device=dev)
    ms = event_ms(torch, lambda: P.cosine_select(feats, c_tab, S, T, cidx, ccnt, workspace=ws), 2)
    res["cosine_select"] = {"feat_dim": dim, "per_frame": 2, "ms": round(ms, 3),
                            "sim_fp64_tflops": round(2 * nb * nb * dim / (ms * 1e-3) / 1e12, 2)}
    del ws, feats
    # Eq. 1 error of two outputs of the layer
    other = out.clone()
    nws = torch.empty(P.nmse_workspace_bytes(w.heads, S, T) // 8, dtype=torch.float64, device=dev)
    nout = torch.empty(w.heads, dtype=torch.float64, device=dev)
    ms = event_ms(torch, lambda: P.nmse(out, other, S, T, out=nout, workspace=nws), 3)
    nbytes = 2 * out.numel() * out.element_size()
    res["nmse"] = {"ms": round(ms, 3), "gbps": round(nbytes / (ms * 1e-3) / 1e9, 1)}
    return res


def kept_flops_device(torch, idx, cnt, table, n, nb):
    """kept_flops computed on the device (the index lists of the stack's
    layers are hundreds of MB each); only per-head sums reach the host."""
    last = n - (nb - 1) * 64
    rows = torch.full((nb,), 64, dtype=torch.int64, device=cnt.device)
    rows[-1] = last
    slot = torch.arange(idx.shape[2], device=idx.device)
    total = 0
    for h, (pattern, _) in enumerate(table):
        if pattern == 0:
            total += 4 * n * n * 64
            continue
        c = cnt[h].to(torch.int64)
        has_last = ((idx[h] == nb - 1) & (slot[None, :] < c[:, None])).any(dim=1).to(torch.int64)
        keys = 64 * c - (64 - last) * has_last
        total += int(4 * 64 * (rows * keys).sum().item())
    return total


def run_stack(args, P, torch, w):
    """A stack of layers run end to end: every layer has fresh seeded Q/K/V
    and its own seeded pattern table, all resident in HBM; a step is
    estimation, selection and attention of every layer in order."""
    from concurrent.futures import ThreadPoolExecutor

    from workloads import layer_tau, make_qkv, make_table

    H, N, nb, S, T, L = w.heads, w.tokens, w.nb, w.frames, w.tokens_per_frame, w.layers
    code = P.BF16 if w.dtype == "bf16" else P.F32

    def up(x):
        if w.dtype == "bf16":
            return torch.from_numpy(x.view(np.int16)).cuda().view(torch.bfloat16)
        return torch.from_numpy(x).cuda()

    t0 = time.time()
    layers, host0 = [], None
    with ThreadPoolExecutor(2) as pool:
        futs = [pool.submit(make_qkv, w, l, args.seed) for l in range(L)]
        for l in range(L):
            q, k, v = futs[l].result()
            futs[l] = None
            table = make_table(w, l, seed=args.seed)
            layers.append({"q": up(q), "k": up(k), "v": up(v), "table": table,
                           "cap": P.index_capacity(table, S, T, code),
                           "tau": layer_tau(w, l, args.seed)})
            if l == 0:
                host0 = (q, k, v)
            del q, k, v
            log(f"[stack] layer {l}: tau {layers[-1]['tau']}% cap {layers[-1]['cap']} "
                f"({time.time() - t0:.1f}s)")
    dev = layers[0]["q"].device
    qp = torch.zeros((H, nb, 64), dtype=torch.float64, device=dev)
    kp = torch.zeros((H, 64, nb), dtype=torch.float64, device=dev)
    idx_buf = torch.empty(H * nb * max(x["cap"] for x in layers), dtype=torch.int32, device=dev)
    cnt = torch.empty((H, nb), dtype=torch.int32, device=dev)
    ws_bytes = max(P.select_workspace_bytes(x["table"], S, T, code) for x in layers)
    sel_ws = torch.empty(max(ws_bytes, 16) // 4, dtype=torch.int32, device=dev)
    att_bytes = max(P.attention_workspace_bytes(x["table"], S, T, code) for x in layers)
    att_ws = torch.empty(max(att_bytes, 16) // 4, dtype=torch.int32, device=dev) if args.split else None
    out = torch.empty_like(layers[0]["q"])

    def run_layer(x, ev=None):
        idx = idx_buf[: H * nb * x["cap"]].view(H, nb, x["cap"])
        if ev:
            ev[0].record()
        P.estimate_blocks(x["q"], x["k"], x["table"], S, T, qp, kp)
        if ev:
            ev[1].record()
        P.select_blocks(qp, kp, x["table"], S, T, x["cap"], idx, cnt, dtype=code, workspace=sel_ws)
        if ev:
            ev[2].record()
        P.sparse_attention(x["q"], x["k"], x["v"], x["table"], S, T, idx, cnt, out,
                           workspace=att_ws)
        if ev:
            ev[3].record()
        return idx

    # algorithmic FLOP and achieved sparsity of every layer, outside the timing;
    # layer 0's lists and outputs on the oracle sample's query blocks
    cpu_rows = min(args.cpu_rows, 16)
    sampled = sample_rows(nb, cpu_rows, args.seed) if cpu_rows > 0 else []
    for l, x in enumerate(layers):
        idx = run_layer(x)
        if l == 0 and sampled:
            tok = np.concatenate([np.arange(i * 64, min((i + 1) * 64, N)) for i in sampled])
            out0 = out[:, torch.from_numpy(tok).to(dev)].float().cpu().numpy().astype(np.float64)
            idx0, cnt0 = idx.cpu().numpy(), cnt.cpu().numpy()
        x["flop"] = kept_flops_device(torch, idx, cnt, x["table"], N, nb)
        c = cnt.to(torch.int64)
        x["pairs"] = sum(nb * nb if p == 0 else int(c[h].sum().item())
                         for h, (p, _) in enumerate(x["table"]))
    torch.cuda.synchronize()

    def step(evs=None):
        for l, x in enumerate(layers):
            run_layer(x, evs[l] if evs else None)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    evs = [[[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(L)]
           for _ in range(args.steps)]
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record()
    for s in range(args.steps):
        step(evs[s])
    end.record()
    torch.cuda.synchronize()
    ms_step = start.elapsed_time(end) / args.steps

    per_layer, att_total, flop_total, ph = [], 0.0, 0, np.zeros(3)
    for l, x in enumerate(layers):
        t = np.array([[e[l][i].elapsed_time(e[l][i + 1]) for i in range(3)] for e in evs]).mean(axis=0)
        ph += t
        att_total += t[2]
        flop_total += x["flop"]
        tab = x["table"]
        per_layer.append({"layer": l, "tau_percent": x["tau"],
                          "table": {"dense": sum(p == 0 for p, _ in tab),
                                    "frame_local": sum(p == 1 for p, _ in tab),
                                    "topk_blocks": sorted({k for p, k in tab if p == 2})},
                          "sparsity": round(1.0 - x["pairs"] / (H * nb * nb), 4),
                          "attention_workspace_bytes": P.attention_workspace_bytes(tab, S, T, code),
                          "ms": [round(float(v), 4) for v in t],
                          "attention_tflops": round(x["flop"] / (t[2] * 1e-3) / 1e12, 1)})
    flops_dense = 4 * N * N * 64 * H
    peak = PEAK_BF16_TFLOPS if w.dtype == "bf16" else PEAK_F32_TFLOPS
    att_tflops = flop_total / (att_total * 1e-3) / 1e12
    log(f"[stack] {L} layers: {ms_step:.2f} ms per step ({ms_step / L:.3f} ms per layer); "
        f"estimate {ph[0]:.2f}, select {ph[1]:.2f}, attention {ph[2]:.2f} ms; "
        f"attention {att_tflops:.1f} TFLOP/s")

    cpu = None
    parity = None
    if cpu_rows > 0:
        t0 = time.perf_counter()
        res = {}
        with single_threaded():
            sec, rows = oracle_sample(w, *host0, layers[0]["table"], cpu_rows, seed=args.seed, results=res)
        wall = time.perf_counter() - t0
        parity = parity_sample(res, sampled, out0, idx0, cnt0, layers[0]["table"], N, w.dtype, host0)
        parity["layer"] = 0
        log(f"[stack] parity on the oracle sample {parity}")
        usable, model = host_cpus()
        cpu = {"value": round(flops_dense / sec / 1e12, 6), "unit": "dense-equiv TFLOP/s",
               "cores": 1, "kind": "oracle", "host_cores": usable, "cpu_model": model,
               "ms_per_layer": round(sec * 1e3, 1),
               "sample": f"layer 0 only: {rows} of {nb} query blocks per head (seeded), all "
                         f"{H} heads; per-head work timed in full, per-block work scaled by "
                         f"{nb}/{rows}; {wall:.1f} s of CPU work"}
        log(f"[stack] cpu oracle {cpu}")

    result = {
        "metric": METRIC,
        "value": round(L * flops_dense / (ms_step * 1e-3) / 1e12, 2),
        "unit": "dense-equiv TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "ms_per_layer": round(ms_step / L, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic",
        "config": {"workload": w.name, "layers": L, "split_long_lists": bool(args.split),
                   "frames": S, "tokens_per_frame": T,
                   "tokens": N, "heads": H, "head_dim": 64, "block": 64, "key_blocks": nb,
                   "achieved_block_sparsity": round(
                       1.0 - sum(x["pairs"] for x in layers) / (L * H * nb * nb), 4)},
        "roofline": {
            "kernel": "attn_bf16_kernel" if w.dtype == "bf16" else "attn_f32_kernel",
            "bound": "mfma", "achieved": round(att_tflops, 2), "peak": peak, "unit": "TFLOP/s",
            "frac": round(att_tflops / peak, 4),
            # FETCH_SIZE + WRITE_SIZE of the 24 attention launches of one pass
            "traffic": recorded_traffic(w.name),
            "flop_per_step": flop_total, "attention_ms_per_step": round(att_total, 4),
        },
        "kernels_ms_per_step": {"estimate": round(float(ph[0]), 4), "select": round(float(ph[1]), 4),
                                "attention": round(float(ph[2]), 4)},
        "per_layer": per_layer,
        "cpu_baseline": cpu,
        "parity_sample": parity,
    }
    print(json.dumps(result), flush=True)


def other_config(P, torch, name, steps, warmup, seed=0):
    """One smaller configuration timed the way the main workload is (estimate
    -> select -> attention on one resident layer, HIP events on the launch
    stream), with the attention kernel against its dtype's matrix peak and,
    on every query block of a layer of at most 20000 tokens (else a seeded
    sample of 16 per head), its lists and outputs against the oracle."""
    import oracle as O
    from workloads import WORKLOADS, make_qkv, make_table

    w = WORKLOADS[name]
    q, k, v = make_qkv(w, seed=seed)
    table = make_table(w, seed=seed)
    code = P.BF16 if w.dtype == "bf16" else P.F32

    def up(x):
        if w.dtype == "bf16":
            return torch.from_numpy(x.view(np.int16)).cuda().view(torch.bfloat16)
        return torch.from_numpy(x).cuda()

    tq, tk, tv = up(q), up(k), up(v)
    H, N, nb, S, T = w.heads, w.tokens, w.nb, w.frames, w.tokens_per_frame
    dev = tq.device
    cap = P.index_capacity(table, S, T, code)
    qp = torch.zeros((H, nb, 64), dtype=torch.float64, device=dev)
    kp = torch.zeros((H, 64, nb), dtype=torch.float64, device=dev)
    idx = torch.empty((H, nb, cap), dtype=torch.int32, device=dev)
    cnt = torch.empty((H, nb), dtype=torch.int32, device=dev)
    out = torch.empty_like(tq)
    sel_ws = torch.empty(max(P.select_workspace_bytes(table, S, T, code), 16) // 4, dtype=torch.int32,
                         device=dev)
    att_ws = torch.empty(max(P.attention_workspace_bytes(table, S, T, code), 16) // 4,
                         dtype=torch.int32, device=dev)

    def step(ev=None):
        if ev:
            ev[0].record()
        P.estimate_blocks(tq, tk, table, S, T, qp, kp)
        if ev:
            ev[1].record()
        P.select_blocks(qp, kp, table, S, T, cap, idx, cnt, dtype=code, workspace=sel_ws)
        if ev:
            ev[2].record()
        P.sparse_attention(tq, tk, tv, table, S, T, idx, cnt, out, workspace=att_ws)
        if ev:
            ev[3].record()

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(steps)]
    a0, a1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a0.record()
    for st in range(steps):
        step(evs[st])
    a1.record()
    torch.cuda.synchronize()
    ms_step = a0.elapsed_time(a1) / steps
    ph = [float(np.mean([e[i].elapsed_time(e[i + 1]) for e in evs])) for i in range(3)]
    idx_h, cnt_h = idx.cpu().numpy(), cnt.cpu().numpy()
    flops = kept_flops(idx_h, cnt_h, table, N, nb)
    peak = PEAK_BF16_TFLOPS if w.dtype == "bf16" else PEAK_F32_TFLOPS
    att_tflops = flops / (ph[2] * 1e-3) / 1e12
    kept_pairs = sum(nb * nb if p == 0 else int(cnt_h[h].sum()) for h, (p, _) in enumerate(table))
    # parity: every query block of a small layer, a sample of a larger one
    rows = list(range(nb)) if N <= 20000 else sample_rows(nb, 16, seed)
    got = out.float().cpu().numpy().astype(np.float64)
    tol = 2e-2 if w.dtype == "bf16" else 1e-4
    equal = near = mismatch = 0
    err = 0.0
    from tests.parity import valid_topk

    for h, (pattern, param) in enumerate(table):
        qh, kh, vh = (O.to_f64(x[h], w.dtype) for x in (q, k, v))
        kbar = O.pool_blocks(kh, 64) if pattern == O.TOPK else None
        for i in rows:
            r = O.block_range(i, N, 64)
            lst = np.arange(nb)
            if pattern == O.TOPK:
                srow = O.block_scores(O.pool_blocks(qh[r.start:r.stop], 64), kbar)[0]
                lst, margin = O.topk_row(srow, param)
            elif pattern == O.FRAME_LOCAL:
                lst, margin = O.frame_local_row(i, N, T, 64), math.inf
            if pattern != O.DENSE:
                gl = idx_h[h, i, :int(cnt_h[h, i])]
                if np.array_equal(gl, lst):
                    equal += 1
                elif pattern == O.TOPK and margin <= 1e-6 and valid_topk(gl, srow, param):
                    near += 1
                    lst = gl
                else:
                    mismatch += 1
                    continue
            ref = O.attend_block(qh, kh, vh, i, lst, 64)[0]
            err = max(err, float(np.max(np.abs(got[h, r.start:r.stop] - ref))))
    res = {"workload": name, "dtype": w.dtype, "tokens": N, "key_blocks": nb,
           "ms_per_step": round(ms_step, 4),
           "dense_equiv_tflops": round(4 * N * N * 64 * H / (ms_step * 1e-3) / 1e12, 1),
           "kernels_ms": {"estimate": round(ph[0], 4), "select": round(ph[1], 4),
                          "attention": round(ph[2], 4)},
           "achieved_block_sparsity": round(1.0 - kept_pairs / (H * nb * nb), 4),
           "roofline": {"kernel": "attn_bf16_kernel" if w.dtype == "bf16" else "attn_f32_kernel",
                        "bound": "mfma", "achieved": round(att_tflops, 2), "peak": peak,
                        "unit": "TFLOP/s", "frac": round(att_tflops / peak, 4),
                        "flop_per_launch": flops},
           "parity": {"query_blocks_per_head": len(rows), "lists_equal": equal,
                      "near_ties_valid_differing": near, "list_mismatches": mismatch,
                      "max_abs_err": err, "bound": tol}}
    del tq, tk, tv, out, sel_ws, att_ws
    return res


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="S100xT1374-bf16")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--dense-reps", type=int, default=3)
    ap.add_argument("--cpu-rows", type=int, default=320,
                    help="query blocks per head in the oracle CPU sample (0 = skip)")
    ap.add_argument("--next-rows", type=int, default=1,
                    help="also time the stride, global-probe, cosine and NMSE kernels (0 = skip)")
    ap.add_argument("--other-configs", default="S4xT261-f32,S8xT1374-bf16,S32xT1374-bf16",
                    help="comma-separated smaller workloads also timed and checked (empty = none)")
    ap.add_argument("--split", type=int, default=1, choices=(0, 1),
                    help="1: pass the attention workspace, so lists of 384+ key blocks (on layers of 4096+ "
                         "key blocks) run split "
                         "into key ranges; 0: the unsplit launch (same work and results)")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run three device-to-device copies of MIB MiB (a plain copy "
                         "kernel of known size, to scale rocprofv3 FETCH_SIZE / WRITE_SIZE) and exit")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py runs on one GPU only; --gpus {args.gpus} is not supported "
              "(the heads of a layer would shard across GPUs with no exchange)", file=sys.stderr)
        sys.exit(2)

    import torch

    if args.copy_calibration > 0:
        nbytes = args.copy_calibration << 20
        src = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes": nbytes, "copies": 3}), flush=True)
        return

    import paper_2607_03612_amd as P
    from paper_2607_03612_amd import binding
    from workloads import WORKLOADS, make_qkv, make_table

    if not os.path.exists(binding.LIB_PATH):
        from paper_2607_03612_amd import build

        build.build()
    P.load()
    if not torch.cuda.is_available():
        raise SystemExit("no GPU visible: the HIP path needs an MI355X")

    w = WORKLOADS[args.workload]
    if w.layers > 1:
        run_stack(args, P, torch, w)
        return
    t0 = time.time()
    q, k, v = make_qkv(w, seed=args.seed)
    table = make_table(w, seed=args.seed)
    log(f"[bench] {w.name}: N={w.tokens} nb={w.nb} table={table} (gen {time.time() - t0:.1f}s)")
    code = P.BF16 if w.dtype == "bf16" else P.F32

    def up(x):
        if w.dtype == "bf16":
            return torch.from_numpy(x.view(np.int16)).cuda().view(torch.bfloat16)
        return torch.from_numpy(x).cuda()

    tq, tk, tv = up(q), up(k), up(v)
    H, N, nb, S, T = w.heads, w.tokens, w.nb, w.frames, w.tokens_per_frame
    dev = tq.device
    cap = P.index_capacity(table, S, T, code)
    qp = torch.zeros((H, nb, 64), dtype=torch.float64, device=dev)
    kp = torch.zeros((H, 64, nb), dtype=torch.float64, device=dev)
    idx = torch.empty((H, nb, cap), dtype=torch.int32, device=dev)
    cnt = torch.empty((H, nb), dtype=torch.int32, device=dev)
    out = torch.empty_like(tq)
    # Top-K scores go through a workspace (two launches, faster than the
    # single launch that keeps score rows in LDS; the same lists)
    sel_ws_bytes = P.select_workspace_bytes(table, S, T, code)
    sel_ws = torch.empty(max(sel_ws_bytes, 16) // 4, dtype=torch.int32, device=dev)
    # long lists (384+ key blocks, layers of 4096+) run split into key ranges through a
    # workspace; none at this layer's budget, the call takes it all the same
    att_ws_bytes = P.attention_workspace_bytes(table, S, T, code)
    att_ws = torch.empty(max(att_ws_bytes, 16) // 4, dtype=torch.int32, device=dev) if args.split else None

    def step(ev=None):
        if ev:
            ev[0].record()
        P.estimate_blocks(tq, tk, table, S, T, qp, kp)
        if ev:
            ev[1].record()
        P.select_blocks(qp, kp, table, S, T, cap, idx, cnt, dtype=code, workspace=sel_ws)
        if ev:
            ev[2].record()
        P.sparse_attention(tq, tk, tv, table, S, T, idx, cnt, out, workspace=att_ws)
        if ev:
            ev[3].record()

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record()
    for s in range(args.steps):
        step(evs[s])
    end.record()
    torch.cuda.synchronize()
    ms_step = start.elapsed_time(end) / args.steps
    est_ms = float(np.mean([e[0].elapsed_time(e[1]) for e in evs]))
    sel_ms = float(np.mean([e[1].elapsed_time(e[2]) for e in evs]))
    att_ms = float(np.mean([e[2].elapsed_time(e[3]) for e in evs]))

    idx_h, cnt_h = idx.cpu().numpy(), cnt.cpu().numpy()
    # the timed step's outputs on the query blocks the oracle sample covers
    # (later launches below reuse `out`)
    sampled = sample_rows(nb, args.cpu_rows, args.seed) if args.cpu_rows > 0 else []
    tok = np.concatenate([np.arange(i * 64, min((i + 1) * 64, N)) for i in sampled]) if sampled else None
    out_sampled = (out[:, torch.from_numpy(tok).to(dev)].float().cpu().numpy().astype(np.float64)
                   if sampled else None)
    flops_kept = kept_flops(idx_h, cnt_h, table, N, nb)
    flops_dense = 4 * N * N * 64 * H
    kept_pairs = sum(nb * nb if p == 0 else int(cnt_h[h].sum()) for h, (p, _) in enumerate(table))
    sparsity = 1.0 - kept_pairs / (H * nb * nb)
    esz = 2 if w.dtype == "bf16" else 4
    n_topk = sum(1 for p, _ in table if p == 2)
    est_read = 2 * n_topk * N * 64 * esz            # Q and K of the Top-K heads
    est_bytes = est_read + 2 * n_topk * nb * 64 * 8  # plus the pooled means (float64)
    peak = PEAK_BF16_TFLOPS if w.dtype == "bf16" else PEAK_F32_TFLOPS
    att_tflops = flops_kept / (att_ms * 1e-3) / 1e12
    value = flops_dense / (ms_step * 1e-3) / 1e12
    log(f"[bench] step {ms_step:.3f} ms (estimate {est_ms:.3f}, select {sel_ms:.3f}, "
        f"attention {att_ms:.3f}); sparsity {sparsity:.4f}; attention {att_tflops:.1f} TFLOP/s")

    # dense baseline: every head dense (the library's all-dense kernel)
    dense_tab = [(0, 0)] * H
    dense = None
    if args.dense_reps > 0:
        P.sparse_attention(tq, tk, tv, dense_tab, S, T, out=out)
        torch.cuda.synchronize()
        d0, d1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        d0.record()
        for _ in range(args.dense_reps):
            P.sparse_attention(tq, tk, tv, dense_tab, S, T, out=out)
        d1.record()
        torch.cuda.synchronize()
        dense_ms = d0.elapsed_time(d1) / args.dense_reps
        dense = {"ms": round(dense_ms, 3),
                 "tflops": round(flops_dense / (dense_ms * 1e-3) / 1e12, 1),
                 "mfma_frac": round(flops_dense / (dense_ms * 1e-3) / 1e12 / peak, 4),
                 "sparse_step_speedup": round(dense_ms / ms_step, 2)}
        log(f"[bench] dense baseline {dense}")

    # estimation kernel alone with a cold last-level cache: a read-only pass
    # over 768 MiB evicts Q and K from the 256 MB Infinity Cache without
    # leaving dirty lines whose write-back the timed kernel would pay for
    flush_buf = torch.ones((768 << 20) // 4, dtype=torch.float32, device=dev)
    sink = torch.zeros((), dtype=torch.float32, device=dev)

    def cold_ms(fn, reps=5):
        # The flush is queued on the same stream and the host does not wait
        # for it: the start event fires when the flush ends, by which time the
        # timed launch is already queued, so host launch latency stays out.
        ts = []
        for _ in range(reps):
            torch.cuda.synchronize()
            sink.copy_(flush_buf.sum())
            a0, a1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a0.record()
            fn()
            a1.record()
            torch.cuda.synchronize()
            ts.append(a0.elapsed_time(a1))
        return float(np.median(ts))

    est_cold_ms = cold_ms(lambda: P.estimate_blocks(tq, tk, table, S, T, qp, kp))
    del flush_buf

    # the other pattern classes and the profiler's error kernel on the same
    # layer: uniform stride (the profiling baseline at sparsity 0.85),
    # global-probe selection, per-frame cosine selection on 1024-wide
    # features, and the Eq. 1 error
    next_rows = None
    if args.next_rows:
        next_rows = measure_next_rows(P, torch, w, tq, tk, tv, out, table)
        log(f"[bench] next rows {next_rows}")

    cpu = None
    parity = None
    if args.cpu_rows > 0:
        t0 = time.perf_counter()
        res = {}
        with single_threaded():
            sec, rows = oracle_sample(w, q, k, v, table, args.cpu_rows, seed=args.seed, results=res)
        wall = time.perf_counter() - t0
        parity = parity_sample(res, sampled, out_sampled, idx_h, cnt_h, table, N, w.dtype, (q, k, v))
        log(f"[bench] parity on the oracle sample {parity}")
        usable, model = host_cpus()
        cpu = {"value": round(flops_dense / sec / 1e12, 6), "unit": "dense-equiv TFLOP/s",
               "cores": 1, "kind": "oracle", "host_cores": usable, "cpu_model": model,
               "ms_per_layer": round(sec * 1e3, 1),
               "sample": f"{rows} of {nb} query blocks per head (seeded), all 16 heads; per-head "
                         f"fp64 widening and key pooling timed in full, per-block probe/score/"
                         f"select/attention scaled by {nb}/{rows}; {wall:.1f} s of CPU work"}
        log(f"[bench] cpu oracle {cpu}")

    others = []
    for name in [x for x in args.other_configs.split(",") if x]:
        others.append(other_config(P, torch, name, steps=max(args.steps, 5), warmup=args.warmup,
                                   seed=args.seed))
        log(f"[bench] other config {others[-1]}")

    traffic = recorded_traffic(w.name)
    result = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "dense-equiv TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic",
        "config": {
            "workload": w.name, "frames": S, "tokens_per_frame": T, "tokens": N, "heads": H,
            "head_dim": 64, "block": 64, "key_blocks": nb,
            "table": {"dense": sum(p == 0 for p, _ in table), "frame_local": sum(p == 1 for p, _ in table),
                      "topk": n_topk, "topk_blocks": sorted({t for p, t in table if p == 2})},
            "achieved_block_sparsity": round(sparsity, 4),
        },
        "roofline": {
            "kernel": "attn_bf16_kernel" if w.dtype == "bf16" else "attn_f32_kernel",
            "bound": "mfma", "achieved": round(att_tflops, 2), "peak": peak, "unit": "TFLOP/s",
            "frac": round(att_tflops / peak, 4), "traffic": traffic,
            "flop_per_launch": flops_kept, "launch_ms": round(att_ms, 4),
        },
        "kernels_ms": {"estimate": round(est_ms, 4), "select": round(sel_ms, 4),
                       "attention": round(att_ms, 4)},
        "estimate_roofline": {
            "kernel": "pool_bf16_kernel" if w.dtype == "bf16" else "pool_f32_kernel",
            "bound": "hbm", "bytes_per_launch": est_bytes, "launch_ms_cold": round(est_cold_ms, 4),
            "achieved": round(est_bytes / (est_cold_ms * 1e-3) / 1e9, 1), "peak": PEAK_HBM_GBS,
            "unit": "GB/s", "frac": round(est_bytes / (est_cold_ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
            "read_bytes_per_launch": est_read,
            "read_frac": round(est_read / (est_cold_ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
        },
        "select_roofline": {
            # Top-K scores of every (query block, key block) pair in float64
            # on the matrix cores: 2 * nb^2 * 64 FLOP per Top-K head
            "kernel": "topk_score_kernel + topk_rows_kernel", "bound": "mfma-fp64",
            "flop_per_launch": 2 * nb * nb * 64 * n_topk, "launch_ms": round(sel_ms, 4),
            "achieved": round(2 * nb * nb * 64 * n_topk / (sel_ms * 1e-3) / 1e12, 2),
            "peak": PEAK_F64_TFLOPS, "unit": "TFLOP/s",
            "frac": round(2 * nb * nb * 64 * n_topk / (sel_ms * 1e-3) / 1e12 / PEAK_F64_TFLOPS, 4),
        },
        "dense_baseline": dense,
        "other_configs": others,
        "next_rows": next_rows,
        "cpu_baseline": cpu,
        "parity_sample": parity,
    }
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
