"""Benchmark of the fused block-scaled FP8 MoE layer on one MI355X.

    python bench.py [--steps K] [--warmup W] [--config decode|mid|prefill|skewed|...]

A step is one call of the whole layer (routing, permutation, GEMM1 + SwiGLU +
re-quantisation, GEMM2, combine) on one batch of seeded synthetic inputs
already resident in HBM.  By default the four DeepSeek-V3-shaped workloads of
the metric are timed in one run -- decode T=16, mid T=256, prefill T=4096 (32
of 256 experts resident) and skewed T=8192 (all 256 resident, 16 hot) -- each
with its own result object under "configs"; the line's `value` is the skewed
(largest) workload's µs per call over exactly --steps calls.  Activation
batches rotate over --rotate seeds (the resident expert weights stay fixed).
Each timed region starts behind a device spin long enough for the host to
enqueue all calls, so the calls run back to back; HIP events on the library's
stream give the per-kernel durations behind each roofline object.

Per workload also: the cold µs per call (median, p10, p90 of calls each
preceded, outside the timed interval, by a read-only sweep of 1 GiB that
evicts L2 and the 256 MB Infinity Cache without leaving dirty lines), P and
the touched experts, and the CPU oracle on a bounded token sample.  The line
carries the GPU clock read before and after the timed regions.

Extra legs (not `value`): `dsa_topk_indexer`, `dsa_sparse_attention` and
`router_projection` (see their functions).  --copy-calibration runs only a
plain 1 GiB device copy, the reference kernel for scaling the HBM byte
counters of rocprofv3.
"""
from __future__ import annotations

import argparse
import ctypes
import hashlib
import json
import os
import re
import sys
import time

import numpy as np
import torch

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import paper_2608_14560_amd as M  # noqa: E402
import workloads as W  # noqa: E402

METRIC = "fused FP8 MoE µs/call + effective TFLOP/s (% FP8 MFMA peak), T=16..8192"
HBM_PEAK_GBS = 8000.0
FP8_PEAK_TFLOPS = 5000.0
# fp32 fused multiply-adds without packed instructions (the kernels are built
# with packed fp32 disabled): 256 CUs x 4 SIMDs x 16 lanes x 2 FLOP x 2.4 GHz
FP32_FMA_PEAK_TFLOPS = 78.6
BF16_PEAK_TFLOPS = 2500.0  # dense bf16 MFMA
PROFILE_TRAFFIC = os.path.join(ROOT, "profiles", "gemm1_traffic_{cfg}.txt")


def flops_per_pair(cfg) -> int:
    return 2 * cfg.H * 2 * cfg.I + 2 * cfg.I * cfg.H


def small_tile_path(cfg) -> bool:
    """The library's choice of the column-split GEMM1 (plus a re-quantisation
    launch): batches with 16-row M-tiles (at most 16 expected rows per expert)."""
    return cfg.T * cfg.top_k / cfg.num_experts <= 16


def gemm1_bytes(cfg, P: int, touched: int) -> int:
    """Algorithmic HBM bytes of one GEMM1 launch: each touched expert's W13 and
    its scales once, each routed row of hidden (and scales) once, and its
    output once -- the FP8 intermediate with scales, or on the small-tile path
    the fp32 SwiGLU output that the re-quantisation launch reads."""
    H, I = cfg.H, cfg.I
    w = touched * (2 * I * H + 4 * (2 * I // 128) * (H // 128))
    a = P * (H + 4 * (H // 128))
    o = P * I * 4 if small_tile_path(cfg) else P * (I + 4 * (I // 128))
    return w + a + o


def layer_bytes(cfg, P: int, touched: int) -> int:
    """Algorithmic HBM bytes of the layer: weights of touched experts once, and
    per token its hidden row, scales, router logits and bf16 output."""
    H, I = cfg.H, cfg.I
    w = touched * (3 * I * H + 4 * ((2 * I // 128) * (H // 128) + (H // 128) * (I // 128)))
    per_tok = H + 4 * (H // 128) + 4 * cfg.num_experts + 2 * H
    return w + cfg.T * per_tok + 4 * cfg.num_experts


# The sources that decide the grouped GEMMs' kernels, their launch plan and
# their work-item order (the other operators' files are left out).
GEMM_SOURCES = ("api.cpp", "gemm.hip", "gemm_tile.hip", "moe_device.h", "permute.hip",
                "scatter_device.h")


def _code_only(text: str) -> str:
    """Source text without comments and without blank-line or spacing
    differences: what the digest of the GEMM kernels covers."""
    text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
    text = re.sub(r"//[^\n]*", "", text)
    return "\n".join(" ".join(line.split()) for line in text.splitlines() if line.strip())


def source_digest() -> str:
    """Digest of the GEMM kernel sources (their code, comments aside): a
    traffic measurement is reported only while it matches."""
    h = hashlib.sha256()
    d = os.path.join(ROOT, "paper_2608_14560_amd", "csrc")
    for f in GEMM_SOURCES:
        with open(os.path.join(d, f), encoding="utf-8") as fh:
            h.update(f.encode())
            h.update(_code_only(fh.read()).encode())
    return h.hexdigest()[:16]


def read_traffic(cfg_name: str):
    """Per-launch HBM bytes of GEMM1 measured with rocprofv3 counters (scaled by a
    plain copy), if taken on the current kernel source; else None."""
    path = PROFILE_TRAFFIC.format(cfg=cfg_name)
    if not os.path.exists(path):
        return None
    kv = {}
    with open(path) as f:
        for line in f:
            if "=" in line and not line.startswith("#"):
                k, v = line.split("=", 1)
                kv[k.strip()] = v.strip()
    if kv.get("source_digest") != source_digest():
        return None
    try:
        return int(float(kv["fetch_bytes_per_launch"]) + float(kv["write_bytes_per_launch"]))
    except (KeyError, ValueError):
        return None


def copy_calibration():
    n = 1 << 30
    src = torch.empty(n, dtype=torch.uint8, device="cuda").fill_(1)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_read": n, "copy_bytes_written": n, "launches": 3}))


def cpu_info() -> dict:
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        affinity = len(os.sched_getaffinity(0))
    except OSError:
        affinity = None
    return {"cpu_model": model, "nproc": os.cpu_count(), "cpus_available": affinity}


def cpu_baseline(cfg, batch, weights_dev, max_tokens: int, threads: int | None = None):
    """The CPU oracle on this host on one of the bench's batches (all tokens, or
    a seeded sample of max_tokens), scaled to microseconds per call by the
    resident-pair count (the oracle's time is proportional to it)."""
    import oracle
    oracle.build(force=False)
    before = oracle.num_threads()
    if threads:
        oracle.set_num_threads(threads)
    try:
        shape = oracle.shape_of(cfg)
        logits = batch["logits"].cpu().numpy()
        bias = batch["bias"].cpu().numpy()
        ids, _ = oracle.route(shape, logits, bias)
        le = ids - cfg.local_expert_offset
        local = (le >= 0) & (le < cfg.num_local_experts)
        pairs_all = int(local.sum())
        if cfg.T <= max_tokens:
            toks = np.arange(cfg.T, dtype=np.int32)
        else:
            toks = np.sort(np.random.default_rng(0).choice(cfg.T, max_tokens, replace=False)).astype(np.int32)
        need = sorted(set(int(e) for e in le[toks][local[toks]]))
        w13, s13, w2, s2 = weights_dev
        host = lambda t: [t[e].cpu().numpy() if e in need else None for e in range(cfg.num_local_experts)]
        hw = dict(w13=host(w13), w13_scale=host(s13), w2=host(w2), w2_scale=host(s2))
        hidden, hscale = batch["hidden"].cpu().numpy(), batch["hidden_scale"].cpu().numpy()
        used = oracle.num_threads()
        t0 = time.perf_counter()
        oracle.forward(shape, hidden, hscale, logits, bias, **hw, tokens=toks)
        wall = time.perf_counter() - t0
    finally:
        oracle.set_num_threads(before)
    done = int(local[toks].sum())
    per_call_s = wall * (pairs_all / max(done, 1))
    sample = (f"{'all' if cfg.T <= max_tokens else len(toks)} of {cfg.T} tokens ({done} of {pairs_all} "
              f"resident pairs), scaled to the call by resident pairs")
    return {"value": round(per_call_s * 1e6, 1), "unit": "us/call", "cores": used, "kind": "oracle",
            "sample": sample, "wall_s": round(wall, 3),
            "extrapolated": bool(cfg.T > max_tokens)}


def gpu_clock() -> dict:
    """The shader clock as the driver reports it (sysfs: the active DPM level)."""
    res = {}
    import glob
    for path in sorted(glob.glob("/sys/class/drm/card*/device/pp_dpm_sclk")):
        try:
            with open(path) as f:
                lines = f.read().split("\n")
        except OSError:
            continue
        cur = [ln for ln in lines if ln.strip().endswith("*")]
        if cur:
            res[path.split("/")[4]] = cur[0].split(":", 1)[1].replace("*", "").strip()
    return res


def router_projection_leg(cfg, shape, batches, weights, out, ws, stream, K, prefill):
    """µs per call of routing from the hidden rows (projection on the device)
    and from given logits, on the same batches, each K calls back to back.
    The projection's own cost is the difference; its roofline uses the
    projection's algorithmic work: the router weight, the hidden rows and
    scales read once, the block sums written and read once, and T*E*H fused
    multiply-adds."""
    wg = W.gen_router_weight(cfg, 0, device="cuda")
    ros = [M.alloc_route_out(shape) for _ in batches]

    def timed(fn):
        for i in range(3):
            fn(i)
        torch.cuda.synchronize()
        h0 = time.perf_counter()
        for i in range(K):
            fn(i)
        host_ms = (time.perf_counter() - h0) * 1e3
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        prefill(host_ms)
        a.record(stream)
        for i in range(K):
            fn(i)
        b.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(b) * 1e3 / K

    nb = len(batches)
    us_hidden = timed(lambda i: M.route_hidden(shape, batches[i % nb]["hidden"], batches[i % nb]["hidden_scale"],
                                               wg, batches[i % nb]["bias"], route_out=ros[i % nb],
                                               workspace=ws, stream=stream))
    us_logits = timed(lambda i: M.route(shape, batches[i % nb]["logits"], batches[i % nb]["bias"],
                                        route_out=ros[i % nb], workspace=ws, stream=stream))
    # context: the same projection unfused, as a caller without it would run
    # it (dequantise in torch, fp32 GEMM, then routing from the logits)
    wgt = wg.t().contiguous()

    def unfused(i):
        b = batches[i % nb]
        x = b["hidden"].view(torch.float8_e4m3fn).float() * b["hidden_scale"].repeat_interleave(128, dim=1)
        M.route(shape, x @ wgt, b["bias"], route_out=ros[i % nb], workspace=ws, stream=stream)

    us_unfused = timed(unfused)
    layer = [M.FusedCall(shape, b["hidden"], b["hidden_scale"], wg, b["bias"], *weights, out, ws,
                         stream=stream, router=True) for b in batches]
    us_layer = timed(lambda i: layer[i % nb]())
    T, E, H = cfg.T, cfg.num_experts, cfg.H
    KB = H // 128
    nbytes = 4 * E * H + T * H + 4 * T * KB + 2 * 4 * T * KB * E
    flop = 2.0 * T * E * H
    proj_us = max(us_hidden - us_logits, 1e-3)
    if nbytes / (HBM_PEAK_GBS * 1e9) >= flop / (FP32_FMA_PEAK_TFLOPS * 1e12):
        ach = nbytes / (proj_us * 1e-6) / 1e9
        roof = {"bound": "hbm", "achieved": round(ach, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(ach / HBM_PEAK_GBS, 4)}
    else:
        ach = flop / (proj_us * 1e-6) / 1e12
        roof = {"bound": "alu", "achieved": round(ach, 2), "peak": FP32_FMA_PEAK_TFLOPS,
                "unit": "TFLOP/s", "frac": round(ach / FP32_FMA_PEAK_TFLOPS, 4)}
    roof["algorithmic_bytes"] = int(nbytes)
    roof["flop"] = int(flop)
    return {"route_from_hidden_us": round(us_hidden, 2), "route_from_logits_us": round(us_logits, 2),
            "projection_us": round(proj_us, 2), "layer_with_projection_us": round(us_layer, 2),
            "unfused_torch_projection_then_route_us": round(us_unfused, 2),
            "roofline": roof}


def indexer_leg(K, prefill, with_cpu: bool):
    """µs per call of the DSA TopK indexer on two workloads, each K calls back to
    back; the score kernel alone (every sequence scored, dsa_debug_scores) gives
    the roofline: 2*64*128 FLOP per scored token (plain fp32 fused multiply-adds,
    the fixed sequence) and its key row (128 B + a 4-byte scale) read once."""
    res = {}
    for name in ("dsa_paper_long", "dsa_long"):
        cfg = W.INDEXER_CONFIGS[name]
        x = W.generate_indexer(cfg, 0, device="cuda")
        args = (x.q, x.weights, x.k_cache, x.k_scale, x.block_table, x.seq_lens)
        shape = M.dsa_shape(x.q, x.k_cache, x.block_table, cfg.topk)
        ws = torch.empty(max(M.dsa_workspace_size(shape), 256), dtype=torch.uint8, device="cuda")
        out = torch.empty(cfg.B, cfg.topk, dtype=torch.int32, device="cuda")
        scores = torch.empty(cfg.B, cfg.max_pages * cfg.page_size, dtype=torch.float32, device="cuda")

        def timed(fn):
            for _ in range(3):
                fn()
            torch.cuda.synchronize()
            h0 = time.perf_counter()
            for _ in range(K):
                fn()
            host_ms = (time.perf_counter() - h0) * 1e3
            torch.cuda.synchronize()
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            prefill(host_ms)
            a.record()
            for _ in range(K):
                fn()
            b.record()
            torch.cuda.synchronize()
            return a.elapsed_time(b) * 1e3 / K

        call_us = timed(lambda: M.dsa_topk_indexer(*args, topk=cfg.topk, out=out, workspace=ws))
        sc_shape = M.dsa_shape(x.q, x.k_cache, x.block_table, 1)
        ptrs = M._dsa_ptrs(*args)
        sc_ptr = scores.data_ptr()
        L = M.lib()
        scores_us = timed(lambda: L.dsa_debug_scores(ctypes.byref(sc_shape), *ptrs, sc_ptr, None))
        tokens = sum(cfg.seq_lens)
        flop = 2.0 * cfg.num_heads * cfg.head_dim * tokens
        nbytes = tokens * (cfg.head_dim + 4) + x.q.numel() + 4 * x.weights.numel() + 4 * tokens
        ach = flop / (scores_us * 1e-6) / 1e12
        rec = {"workload": f"{name}: B={cfg.B}, seq_lens={list(cfg.seq_lens)}, 64 heads x 128, "
                           f"page {cfg.page_size}, topk {cfg.topk}",
               "us_per_call": round(call_us, 2), "score_kernel_all_tokens_us": round(scores_us, 2),
               "roofline_score_kernel": {"bound": "alu", "achieved": round(ach, 2),
                                         "peak": FP32_FMA_PEAK_TFLOPS, "unit": "TFLOP/s",
                                         "frac": round(ach / FP32_FMA_PEAK_TFLOPS, 4),
                                         "flop": int(flop), "algorithmic_bytes": int(nbytes)}}
        if with_cpu:
            import oracle as O  # the CPU baseline: the oracle timed beside the GPU figure
            h = [t.cpu().numpy() for t in args]
            t0 = time.perf_counter()
            O.dsa_topk(*h, cfg.topk)
            rec["cpu_oracle_us"] = round((time.perf_counter() - t0) * 1e6, 1)
            rec["cpu_oracle_threads"] = int(O.lib().oracle_num_threads())
        res[name] = rec
    return res


def attention_leg(K, prefill, with_cpu: bool):
    """µs per call of the DSA sparse attention (both launches: the split kernel
    and the merge) on the paper's regimes, each K calls back to back.  Roofline
    over the whole call against HBM (the products run on the bf16 matrix cores,
    where 2*(576 + 512) FLOP per (token, head, valid entry) take a tenth of the
    time the bytes need at peak): algorithmic bytes = each valid entry's
    gathered row (1152 B) and its index once per token, the query rows, the
    bf16 output and the LSE."""
    res = {}
    for name in ("attn_long", "attn_two", "attn_one"):
        cfg = W.ATTENTION_CONFIGS[name]
        x = W.generate_attention(cfg, 0, device="cuda")
        args = (x.q_nope, x.q_pe, x.ckv, x.kpe, x.indices, x.sm_scale)
        shape = M.attention_shape(x.q_nope, x.ckv, x.indices, x.sm_scale)
        ws = torch.empty(max(M.dsa_attention_workspace_size(shape), 256), dtype=torch.uint8, device="cuda")
        out = torch.empty(cfg.T, cfg.num_heads, cfg.dc, dtype=torch.bfloat16, device="cuda")
        lse = torch.empty(cfg.T, cfg.num_heads, dtype=torch.float32, device="cuda")

        def fn():
            M.dsa_sparse_attention(*args, out=out, lse=lse, workspace=ws)

        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        h0 = time.perf_counter()
        for _ in range(K):
            fn()
        host_ms = (time.perf_counter() - h0) * 1e3
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        prefill(host_ms)
        a.record()
        for _ in range(K):
            fn()
        b.record()
        torch.cuda.synchronize()
        call_us = a.elapsed_time(b) * 1e3 / K
        valid = int((x.indices >= 0).sum().item())
        H = cfg.num_heads
        flop = 2.0 * (cfg.dc + cfg.dp) * H * valid + 2.0 * cfg.dc * H * valid
        nbytes = valid * 2 * (cfg.dc + cfg.dp) + 4 * x.indices.numel() + 2 * (x.q_nope.numel() + x.q_pe.numel()) \
            + 2 * out.numel() + 4 * lse.numel()
        gbs = nbytes / (call_us * 1e-6) / 1e9
        tf = flop / (call_us * 1e-6) / 1e12
        rec = {"workload": f"{name}: {cfg.T} tokens x {H} heads, topk {cfg.topk}, seq_lens "
                           f"{sorted(set(cfg.seq_lens))}, {cfg.pages} pages of {cfg.page_size}",
               "us_per_call": round(call_us, 2),
               "roofline_call": {"bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                                 "frac": round(gbs / HBM_PEAK_GBS, 4), "algorithmic_bytes": int(nbytes),
                                 "flop": int(flop), "tflops": round(tf, 2),
                                 "pct_bf16_mfma_peak": round(100 * tf / BF16_PEAK_TFLOPS, 3)}}
        if with_cpu:
            from oracle import dsa_attention as A  # the CPU baseline: the oracle timed beside the GPU figure
            h = [t.contiguous().cpu().view(torch.int16).numpy().view(np.uint16)
                 for t in (x.q_nope, x.q_pe, x.ckv, x.kpe)]
            idx = x.indices.cpu().numpy()
            t0 = time.perf_counter()
            A.sparse_attention(*h, idx, x.sm_scale)
            rec["cpu_oracle_us"] = round((time.perf_counter() - t0) * 1e6, 1)
            rec["cpu_oracle_threads"] = torch.get_num_threads()
        res[name] = rec
    return res


def run_config(cfg, steps: int, warmup: int, rotate: int, cold_calls: int, weights_rotated: bool,
               cpu_tokens: int, with_cpu: bool):
    """Times one workload; returns its result object (and the call closure data
    the extra legs reuse)."""
    shape = M.Shape.of(cfg)
    dev = "cuda"
    weights = W.gen_weights(cfg, 0, device=dev)
    _, bias, _ = W.gen_router(cfg, 0, device=dev)
    batches = []
    for seed in range(rotate):
        logits, _, _ = W.gen_router(cfg, seed, device=dev)
        hidden, hscale = W.gen_hidden(cfg, seed, device=dev)
        batches.append(dict(logits=logits, bias=bias, hidden=hidden, hidden_scale=hscale))
    ws = M.alloc_workspace(shape, dev)
    out = torch.empty(cfg.T, cfg.H, dtype=torch.bfloat16, device=dev)

    # work per batch (from the layer's own routing)
    Ps, touched = [], []
    for b in batches:
        ro = M.route(shape, b["logits"], b["bias"], workspace=ws)
        offs = ro["expert_offsets"].cpu().numpy()
        Ps.append(int(offs[-1]))
        touched.append(int((np.diff(offs) > 0).sum()))

    stream = torch.cuda.current_stream()
    nst = M.num_stages()
    calls = [M.FusedCall(shape, b["hidden"], b["hidden_scale"], b["logits"], b["bias"], *weights,
                         out, ws, stream=stream) for b in batches]

    def call(i, events=None):
        c = calls[i % len(calls)]
        if events is None:
            c()
        else:
            c.staged(events, nst + 1)

    for i in range(warmup):
        call(i)
    torch.cuda.synchronize()

    # The host enqueues a call (ctypes + one launch per kernel) more slowly
    # than the GPU runs small batches; each timed region starts behind a GPU
    # spin long enough for the host to enqueue all calls.
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    torch.cuda._sleep(10_000_000)
    e1.record(stream)
    torch.cuda.synchronize()
    cycles_per_ms = 10_000_000 / max(e0.elapsed_time(e1), 1e-3)

    K = steps
    h0 = time.perf_counter()
    for i in range(K):
        call(i)
    host_ms = (time.perf_counter() - h0) * 1e3
    torch.cuda.synchronize()

    def prefill(enqueue_ms=None):
        ms = host_ms if enqueue_ms is None else enqueue_ms
        torch.cuda._sleep(int((2.0 * ms + 2.0) * cycles_per_ms))

    # timed region 1: plain calls
    t_start = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    prefill()
    t_start.record(stream)
    for i in range(K):
        call(i)
    t_end.record(stream)
    enq_ms = (time.perf_counter() - wall0) * 1e3
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    ms_per_step = t_start.elapsed_time(t_end) / K

    # timed region 2: the same calls with a HIP event around every kernel
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(nst + 1)] for _ in range(K)]
    ev_arrays = [M.event_array(row) for row in evs]
    torch.cuda.synchronize()
    prefill()
    for i in range(K):
        call(i, ev_arrays[i])
    torch.cuda.synchronize()
    stage_ms = np.array([[evs[i][s].elapsed_time(evs[i][s + 1]) for s in range(nst)] for i in range(K)])
    stage_avg = stage_ms.mean(0)
    names = M.stage_names()

    P_avg = float(np.mean([Ps[i % len(Ps)] for i in range(K)]))
    T_avg = float(np.mean([touched[i % len(touched)] for i in range(K)]))
    flop = flops_per_pair(cfg) * P_avg
    lbytes = float(np.mean([layer_bytes(cfg, Ps[i % len(Ps)], touched[i % len(touched)]) for i in range(K)]))
    g1bytes = float(np.mean([gemm1_bytes(cfg, Ps[i % len(Ps)], touched[i % len(touched)]) for i in range(K)]))
    us = ms_per_step * 1e3
    tflops = flop / (ms_per_step * 1e-3) / 1e12
    gbs = lbytes / (ms_per_step * 1e-3) / 1e9

    g1 = names.index("gemm1_swiglu")
    g1_ms = float(stage_avg[g1])
    g1_flop = flop * (2 * cfg.H * 2 * cfg.I) / flops_per_pair(cfg)
    t_hbm = g1bytes / (HBM_PEAK_GBS * 1e9)
    t_mfma = g1_flop / (FP8_PEAK_TFLOPS * 1e12)
    if t_hbm >= t_mfma:
        ach = g1bytes / (g1_ms * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": round(ach, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(ach / HBM_PEAK_GBS, 4)}
    else:
        ach = g1_flop / (g1_ms * 1e-3) / 1e12
        roof = {"bound": "mfma", "achieved": round(ach, 2), "peak": FP8_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": round(ach / FP8_PEAK_TFLOPS, 4)}
    roof["traffic"] = read_traffic(cfg.name)
    roof["kernel"] = "gemm1_swiglu"
    roof["avg_launch_us"] = round(g1_ms * 1e3, 2)
    roof["algorithmic_bytes_per_launch"] = int(g1bytes)
    roof["flop_per_launch"] = int(g1_flop)

    # the calls alternating between two independent sets of expert weights (no
    # call finds its weights in the Infinity Cache left by the call before it)
    rotated = None
    if weights_rotated:
        weights2 = W.gen_weights(cfg, 1, device=dev)
        calls2 = [M.FusedCall(shape, b["hidden"], b["hidden_scale"], b["logits"], b["bias"], *weights2,
                              out, ws, stream=stream) for b in batches]
        sets = (calls, calls2)
        for i in range(2):
            sets[i % 2][i % len(calls)]()
        torch.cuda.synchronize()
        r0, r1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        prefill()
        r0.record(stream)
        for i in range(K):
            sets[i % 2][i % len(calls)]()
        r1.record(stream)
        torch.cuda.synchronize()
        rotated = round(r0.elapsed_time(r1) / K * 1e3, 2)
        del calls2, sets, weights2
        torch.cuda.empty_cache()

    # cold calls: a read-only sweep of 1 GiB before each (outside the timed
    # interval) evicts L2 and the Infinity Cache and leaves no dirty lines
    cold = None
    if cold_calls > 0:
        sweep = torch.ones(1 << 28, dtype=torch.float32, device=dev)
        times = []
        for i in range(cold_calls):
            sweep.sum()
            a0 = torch.cuda.Event(enable_timing=True)
            a1 = torch.cuda.Event(enable_timing=True)
            a0.record(stream)
            call(i)
            a1.record(stream)
            torch.cuda.synchronize()
            times.append(a0.elapsed_time(a1))
        cold = {"median": round(float(np.median(times)) * 1e3, 2),
                "p10": round(float(np.percentile(times, 10)) * 1e3, 2),
                "p90": round(float(np.percentile(times, 90)) * 1e3, 2), "calls": cold_calls}
        del sweep

    cpu = None
    if with_cpu:
        cpu = cpu_baseline(cfg, batches[0], weights, cpu_tokens)

    rec = {
        "workload": f"{cfg.name}: T={cfg.T}, H={cfg.H}, I={cfg.I}, {cfg.num_local_experts} of "
                    f"{cfg.num_experts} experts resident, top-{cfg.top_k} of {cfg.topk_group}/"
                    f"{cfg.n_group} groups" + (f", {cfg.hot_experts} hot experts (+{cfg.hot_bias} bias)"
                                               if cfg.hot_experts else ""),
        "us_per_call": round(us, 2),
        "ms_per_step": round(ms_per_step, 5),
        "steps": K,
        "tflops": round(tflops, 3),
        "pct_fp8_mfma_peak": round(100 * tflops / FP8_PEAK_TFLOPS, 3),
        "gbps": round(gbs, 1),
        "pct_hbm_peak": round(100 * gbs / HBM_PEAK_GBS, 2),
        "binding_roof": "mfma" if tflops / FP8_PEAK_TFLOPS > gbs / HBM_PEAK_GBS else "hbm",
        "pct_binding_roofline": round(100 * max(tflops / FP8_PEAK_TFLOPS, gbs / HBM_PEAK_GBS), 2),
        "resident_pairs_avg": P_avg,
        "touched_experts_avg": T_avg,
        "batches": rotate,
        "stage_us": {n: round(float(v) * 1e3, 2) for n, v in zip(names, stage_avg)},
        "roofline": roof,
        "us_per_call_cold": cold,
        "us_per_call_weights_rotated": rotated,
        "host_enqueue_us_per_call": round(host_ms * 1e3 / K, 1),
        "prefill_covered_enqueue": bool(enq_ms < 2.0 * host_ms + 2.0),
        "host_wall_s": round(wall, 3),
        "shader_clock_mhz_spin": round(cycles_per_ms / 1e3, 1),
        "cpu_baseline": cpu,
    }
    extras = dict(shape=shape, batches=batches, weights=weights, out=out, ws=ws, stream=stream,
                  prefill=prefill)
    return rec, extras


# the metric's workloads, in order; the last one is the line's `value`
METRIC_CONFIGS = ("decode", "mid", "prefill", "skewed")
# CPU oracle sample per workload: tokens (all threads); single-thread tokens
CPU_TOKENS = {"tiny": 8, "decode": 16, "mid": 256, "prefill": 1024, "skewed": 1152, "median": 64,
              "long": 1024}
CPU_TOKENS_1T = {"tiny": 8, "decode": 16, "mid": 16}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default=None, choices=sorted(W.CONFIGS),
                    help="time one workload only (default: decode, mid, prefill, skewed)")
    ap.add_argument("--rotate", type=int, default=4, help="distinct activation batches")
    ap.add_argument("--cold-calls", type=int, default=10)
    ap.add_argument("--no-weight-rotation", action="store_true",
                    help="skip the timing with two alternating sets of expert weights (decode)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration", action="store_true")
    ap.add_argument("--layer-only", action="store_true",
                    help="skip the router-projection, DSA-indexer and sparse-attention legs")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py: this build runs on one GPU only (no multi-GPU path; how the layer would "
              "shard by expert is described in the design notes); use --gpus 1", file=sys.stderr)
        sys.exit(2)
    if not torch.cuda.is_available():
        print("bench.py: no GPU visible", file=sys.stderr)
        sys.exit(2)
    if args.copy_calibration:
        copy_calibration()
        return

    names = (args.config,) if args.config else METRIC_CONFIGS
    clock_before = gpu_clock()
    configs = {}
    extras = None
    for name in names:
        cfg = W.CONFIGS[name]
        last = name == names[-1]
        K = args.steps if last else max(args.steps, 20)
        print(f"bench: {name} ...", file=sys.stderr, flush=True)
        rec, ex = run_config(cfg, K, args.warmup, args.rotate, args.cold_calls,
                             weights_rotated=(name == "decode" and not args.no_weight_rotation),
                             cpu_tokens=CPU_TOKENS.get(name, 16), with_cpu=not args.no_cpu_baseline)
        configs[name] = rec
        if name == "decode" or (extras is None and last):
            extras = (cfg, ex)
        else:
            del ex
        torch.cuda.empty_cache()
    clock_after = gpu_clock()

    router = indexer = attention = None
    if not args.layer_only:
        cfg0, ex = extras
        router = router_projection_leg(cfg0, ex["shape"], ex["batches"], ex["weights"], ex["out"], ex["ws"],
                                       ex["stream"], 20, ex["prefill"])
        indexer = indexer_leg(20, ex["prefill"], not args.no_cpu_baseline)
        attention = attention_leg(20, ex["prefill"], not args.no_cpu_baseline)

    head = configs[names[-1]]
    cpu = None
    if not args.no_cpu_baseline:
        cpu = dict(head["cpu_baseline"])
        cpu.update(cpu_info())
        cpu["per_config_us_per_call"] = {n: (c["cpu_baseline"] or {}).get("value") for n, c in configs.items()}
        # single-thread oracle on the small workloads (bounded samples)
        single = {}
        for n in ("tiny", "decode", "mid"):
            cfg = W.CONFIGS[n]
            wts = W.gen_weights(cfg, 0, device="cuda")
            lg, bs, _ = W.gen_router(cfg, 0, device="cuda")
            hq, hs = W.gen_hidden(cfg, 0, device="cuda")
            b = cpu_baseline(cfg, dict(logits=lg, bias=bs, hidden=hq, hidden_scale=hs), wts,
                             CPU_TOKENS_1T[n], threads=1)
            single[n] = {k: b[k] for k in ("value", "unit", "cores", "sample", "wall_s", "extrapolated")}
            del wts
        cpu["single_thread"] = single
        torch.cuda.empty_cache()

    rec = {
        "metric": METRIC,
        "value": head["us_per_call"],
        "unit": "us/call",
        "n_gpus": 1,
        "steps": head["steps"],
        "warmup": args.warmup,
        "ms_per_step": head["ms_per_step"],
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "fp8e4m3 (fp32 accumulate)",
        "data": "synthetic (seeded; DeepSeek-V3 shapes)",
        "config": {"workload": head["workload"], "configs_timed": list(names)},
        "tflops": head["tflops"],
        "pct_fp8_mfma_peak": head["pct_fp8_mfma_peak"],
        "gbps": head["gbps"],
        "pct_hbm_peak": head["pct_hbm_peak"],
        "roofline": head["roofline"],
        "cpu_baseline": cpu,
        "configs": configs,
        "gpu_clock_before": clock_before,
        "gpu_clock_after": clock_after,
        "router_projection": router,
        "dsa_topk_indexer": indexer,
        "dsa_sparse_attention": attention,
    }
    print(json.dumps(rec))


if __name__ == "__main__":
    main()
