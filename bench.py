#!/usr/bin/env python3
"""Benchmark of the block-sparse chunk-causal attention path on one MI355X.

One step = one chunk through the whole path, as a streaming SR DiT layer
would run it: evict the oldest non-pinned chunk (once the window is full),
append the new chunk's K and V, build the keep lists, run the attention of
the new chunk's queries.  Inputs are seeded synthetic N(0,1) bf16 tensors
already resident in HBM (a small rotating set of chunks); the keep lists
change every step because they are keyed on the current chunk's sequence
number.

Prints ONE JSON line.  ``value`` is kept-tile TFLOP/s over the whole step
(512 flop per kept, valid (query, key) pair: 4*D with D = 128), ``ms_per_step``
is milliseconds per chunk.  ``roofline`` prices the attention kernel alone
(its average duration from HIP events on the launch stream) against the bf16
dense MFMA peak.  ``cpu_baseline`` times the CPU oracle on a bounded sample of
the same workload on this host.

    python bench.py [--steps K] [--warmup W] [--config 1k] [--secondary 2k]
"""

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "ms per chunk + effective TFLOP/s (kept tiles) of sparse causal attn, 1K & 2K"
MFMA_BF16_PEAK_TFLOPS = 2516.6   # 256 CU x 4096 flop/clk x 2.4 GHz, dense
HBM_PEAK_GBPS = 8000.0
D = 128
# Measured HBM traffic of the attention kernel (rocprofv3 FETCH_SIZE / WRITE_SIZE,
# scaled by a plain copy of known size), valid only for the kernel sources it was
# measured on: their SHA-256 is recorded beside the figure.
TRAFFIC_PROFILE = os.path.join(ROOT, "profiles", "attn_fwd_tri_1k_traffic.md")
ATTN_SOURCES = ("paper_2606_09150_amd/csrc/kernels/attn_fwd_tri.hip",
                "paper_2606_09150_amd/csrc/kernels/attn_common.h",
                "paper_2606_09150_amd/csrc/kernels/kv_append.hip",
                "paper_2606_09150_amd/csrc/launch.h")


def attn_sources_sha256():
    import hashlib
    h = hashlib.sha256()
    for rel in ATTN_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def measured_traffic(config):
    """Bytes per attention launch from the committed counter summary, or None when the
    summary is missing, covers another workload, or the kernel sources changed since."""
    try:
        with open(TRAFFIC_PROFILE) as f:
            text = f.read()
    except OSError:
        return None
    fields = {}
    for line in text.splitlines():
        if line.startswith("- ") and ": " in line:
            k, v = line[2:].split(": ", 1)
            fields[k.strip()] = v.strip().strip("`")
    try:
        if fields["workload"] != config or fields["kernel_sources_sha256"] != attn_sources_sha256():
            return None
        return int(fields["traffic_bytes_per_launch"])
    except (KeyError, ValueError, OSError):
        return None


def _flops_of_lists(win, lists, nt, tail, T):
    """Kept-tile FLOPs of one list buffer: 4*D per kept valid (query, key) pair."""
    import torch
    counts, idx, _ = win.lists_views(lists)
    valid_k = torch.where(idx % nt == nt - 1, tail, T).to(torch.int64)
    valid_k = torch.where(idx >= 0, valid_k, torch.zeros_like(valid_k)).sum(-1)      # [B,H,NT]
    valid_q = torch.full((nt,), T, dtype=torch.int64, device=idx.device)
    valid_q[-1] = tail
    kept = int((valid_k * valid_q).sum().item()) * 4 * D
    padded = int(counts.to(torch.int64).sum().item()) * T * T * 4 * D
    return kept, padded


def run_workload(P, wl, steps, warmup, n_src=3, split=0):
    import torch
    import synth

    dev = torch.device("cuda", 0)
    B, L, H, T = wl.batch, wl.chunk_tokens, wl.heads, wl.tile
    nt = -(-L // T)
    tail = L - (nt - 1) * T
    win = P.KVWindow(B, H, L, T, wl.max_chunks, wl.pin_sink, device=dev)
    srcs = [{name: synth.chunk_tensor(wl, c, name, device="cuda") for name in ("k", "v", "q")}
            for c in range(n_src)]
    # window up to (but excluding) the current chunk
    for c in range(wl.window_chunks - 1):
        win.append(srcs[c % n_src]["k"], srcs[c % n_src]["v"])
    total = warmup + steps
    lists = [torch.empty(win.layout.total_bytes, dtype=torch.uint8, device=dev) for _ in range(total)]
    out = torch.empty((B, L, H, D), dtype=torch.bfloat16, device=dev)
    lse = torch.empty((B, H, L), dtype=torch.float32, device=dev)
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(total)]
    work = None
    n_cu = torch.cuda.get_device_properties(dev).multi_processor_count
    if split == "tail" or isinstance(split, tuple):
        pass   # sized in the first (warm-up) step, once the window is full: the plan depends on its length
    elif split:
        work = torch.empty(P.uf_attn_split_work_bytes(win.handle, split), dtype=torch.uint8, device=dev)
    scale = 1.0 / math.sqrt(D)
    stream = torch.cuda.current_stream(dev)

    def step(s):
        src = srcs[(wl.window_chunks - 1 + s) % n_src]
        if win.info().n_live == wl.max_chunks:
            win.evict(1)
        e = ev[s]
        e[0].record(stream)
        win.append(src["k"], src["v"])
        e[1].record(stream)
        win.lists = lists[s]
        win.build_lists(wl.seed, wl.p_prior)
        nonlocal work
        if (split == "tail" or isinstance(split, tuple)) and work is None:
            rows = P.uf_attn_tail_plan(win.handle, n_cu) if split == "tail" else split
            need = P.uf_attn_split_rows_work_bytes(win.handle, *rows)
            work = torch.empty(max(need, 16), dtype=torch.uint8, device=dev)
        e[2].record(stream)
        win.attention(src["q"], scale, out=out, lse=lse, split=split, work=work)
        e[3].record(stream)

    for s in range(warmup):
        step(s)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(warmup, total):
        step(s)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_step = (t1 - t0) * 1e3 / steps

    append_ms = [ev[s][0].elapsed_time(ev[s][1]) for s in range(warmup, total)]
    lists_ms = [ev[s][1].elapsed_time(ev[s][2]) for s in range(warmup, total)]
    attn_ms = [ev[s][2].elapsed_time(ev[s][3]) for s in range(warmup, total)]
    fl = [_flops_of_lists(win, lists[s], nt, tail, T) for s in range(warmup, total)]
    kept = sum(f[0] for f in fl) / steps
    padded = sum(f[1] for f in fl) / steps
    dense = 4 * D * B * H * L * (L * wl.window_chunks)
    attn_avg = sum(attn_ms) / steps
    attn_sorted = sorted(attn_ms)
    append_bytes = 2 * B * L * H * D * 2 + 2 * B * nt * T * H * D * 2 + B * nt * H * D * 4
    # unique bytes of one attention launch: Q, the window's K/V pages, O and LSE
    unique_bytes = B * L * H * D * 2 + wl.window_chunks * B * nt * H * 4 * T * D + B * L * H * D * 2 + B * H * L * 4
    res = {
        "workload": wl.name,
        "ms_per_step": ms_step,
        "value": kept / (ms_step * 1e-3) / 1e12,
        "attn_ms": attn_avg,
        "attn_ms_median": attn_sorted[len(attn_sorted) // 2],
        "attn_ms_p10": attn_sorted[len(attn_sorted) // 10],
        "attn_ms_p90": attn_sorted[(9 * len(attn_sorted)) // 10],
        "attn_tflops": kept / (attn_avg * 1e-3) / 1e12,
        "append_us": sum(append_ms) / steps * 1e3,
        "append_gbps": append_bytes / (sum(append_ms) / steps * 1e-3) / 1e9,
        "lists_us": sum(lists_ms) / steps * 1e3,
        "kept_tflop_per_step": kept / 1e12,
        "attn_unique_gbps": unique_bytes / (attn_avg * 1e-3) / 1e9,
        "kept_fraction": kept / dense,
        "padded_tile_tflop_per_step": padded / 1e12,
        "keys": L * wl.window_chunks,
    }
    # content-adaptive top-k lists (Eq. 4) on the final window, with the budget
    # that keeps the same expected number of earlier-chunk tiles as p_prior
    budget = int(wl.p_prior * wl.prior_chunks * nt)
    q_cur = srcs[(wl.window_chunks - 1 + total - 1) % n_src]["q"]
    tk = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    win.lists = torch.empty_like(lists[0])
    for _ in range(2):
        win.build_topk_lists(q_cur, budget)
    tk[0].record(stream)
    for _ in range(10):
        win.build_topk_lists(q_cur, budget)
    tk[1].record(stream)
    torch.cuda.synchronize()
    res["topk_budget"] = budget
    res["topk_lists_us"] = tk[0].elapsed_time(tk[1]) / 10 * 1e3
    last = total - 1
    win.lists = lists[last]
    state = {"win": win, "srcs": srcs, "n_src": n_src, "steps_done": total, "out": out, "lse": lse,
             "q": srcs[(wl.window_chunks - 1 + last) % n_src]["q"], "kept_flops": fl[-1][0], "scale": scale}
    return res, state


def run_backward(P, wl, state, reps=10, warmup=2):
    """dQ, dK, dV of the last step's attention (same window, lists, O and LSE).

    FLOPs are counted as the algorithmic backward over the kept (query, key)
    pairs: five D-long products per pair (S, dP, dV, dK, dQ), i.e. 2.5 times
    the forward's 4*D; the kernels recompute S and dP once more in the dQ pass
    (seven products per pair), which the count does not credit."""
    import torch
    import synth

    win = state["win"]
    dev = state["q"].device
    B, L, H = wl.batch, wl.chunk_tokens, wl.heads
    n_live = win.info().n_live
    do = synth.chunk_tensor(wl, 1000, "do", device="cuda")
    dq = torch.empty((B, L, H, D), dtype=torch.float32, device=dev)
    dk = torch.empty((n_live, B, L, H, D), dtype=torch.float32, device=dev)
    dv = torch.empty_like(dk)
    work = torch.empty(P.uf_attn_bwd_work_bytes(win.handle), dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream(dev)

    def once():
        P.uf_sparse_causal_attn_bwd(win.handle, state["q"], state["out"], do, state["lse"], win.lists,
                                    state["scale"], dq, dk, dv, work, None, stream)

    for _ in range(warmup):
        once()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    ev[0].record(stream)
    for _ in range(reps):
        once()
    ev[1].record(stream)
    torch.cuda.synchronize()
    ms = ev[0].elapsed_time(ev[1]) / reps
    flops = state["kept_flops"] * 10 // 4
    return {"bwd_ms": ms, "bwd_tflop": flops / 1e12, "bwd_tflops": flops / (ms * 1e-3) / 1e12,
            "bwd_roofline_frac": flops / (ms * 1e-3) / 1e12 / MFMA_BF16_PEAK_TFLOPS,
            "bwd_work_bytes": work.numel(), "bwd_reps": reps}


def run_blocked(P, wl, steps, warmup, local_r=9, block=(2, 8, 8), n_src=3):
    """The workload on 3-D blocks (the paper's (2, 8, 8) tiling, Sec. 2.3.1 (a)) with the
    local window M_local(r): per step, permute the chunk's K, V and Q from raster to
    block order, append, build Bernoulli lists intersected with M_local, attend, and
    permute O back to raster order."""
    import numpy as np
    import torch
    import synth

    dev = torch.device("cuda", 0)
    B, H = wl.batch, wl.heads
    geom = P.uf_block_geom(wl.frames, wl.grid_h, wl.grid_w, *block)
    padded, nb = P.uf_block_geom_tokens(geom)
    T = block[0] * block[1] * block[2]
    win = P.KVWindow(B, H, padded, T, wl.max_chunks, wl.pin_sink, device=dev)
    win.set_block_geom(wl.frames, wl.grid_h, wl.grid_w, *block)
    srcs = [{name: synth.chunk_tensor(wl, c, name, device="cuda") for name in ("k", "v", "q")}
            for c in range(n_src)]
    blk = {name: torch.empty((B, padded, H, D), dtype=torch.bfloat16, device=dev) for name in ("k", "v", "q", "o")}
    o_raster = torch.empty_like(srcs[0]["q"])
    lse = torch.empty((B, H, padded), dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream(dev)

    def permute(x, y, inverse):
        P.uf_block_permute(geom, B, H, x, y, inverse)

    for c in range(wl.window_chunks - 1):
        permute(srcs[c % n_src]["k"], blk["k"], 0)
        permute(srcs[c % n_src]["v"], blk["v"], 0)
        win.append(blk["k"], blk["v"])
    total = warmup + steps
    lists = [torch.empty(win.layout.total_bytes, dtype=torch.uint8, device=dev) for _ in range(total)]
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(6)] for _ in range(total)]

    def step(s):
        src = srcs[(wl.window_chunks - 1 + s) % n_src]
        if win.info().n_live == wl.max_chunks:
            win.evict(1)
        e = ev[s]
        e[0].record(stream)
        permute(src["k"], blk["k"], 0)
        permute(src["v"], blk["v"], 0)
        permute(src["q"], blk["q"], 0)
        e[1].record(stream)
        win.append(blk["k"], blk["v"])
        e[2].record(stream)
        win.lists = lists[s]
        win.build_lists(wl.seed, wl.p_prior, local_r=local_r)
        e[3].record(stream)
        win.attention(blk["q"], out=blk["o"], lse=lse)
        e[4].record(stream)
        permute(blk["o"], o_raster, 1)
        e[5].record(stream)

    for s in range(warmup):
        step(s)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(warmup, total):
        step(s)
    torch.cuda.synchronize()
    ms_step = (time.perf_counter() - t0) * 1e3 / steps
    span = lambda a, b: sum(ev[s][a].elapsed_time(ev[s][b]) for s in range(warmup, total)) / steps
    counts = np.zeros(nb, dtype=np.int64)
    for j in range(nb):   # valid tokens of block j (raster grid)
        nbh, nbw = -(-wl.grid_h // block[1]), -(-wl.grid_w // block[2])
        bti, bhi, bwi = j // (nbh * nbw), (j // nbw) % nbh, j % nbw
        counts[j] = (min(block[0], wl.frames - bti * block[0]) * min(block[1], wl.grid_h - bhi * block[1]) *
                     min(block[2], wl.grid_w - bwi * block[2]))
    cnt = torch.from_numpy(counts).to(dev)
    kept = 0
    for s in range(warmup, total):
        _, idx, _ = win.lists_views(lists[s])
        vk = torch.where(idx >= 0, cnt[idx.clamp(min=0) % nb], torch.zeros_like(idx, dtype=torch.int64)).sum(-1)
        kept += int((vk * cnt[None, None, :]).sum().item()) * 4 * D
    kept /= steps
    attn_ms = span(3, 4)
    dense = 4 * D * B * H * wl.chunk_tokens * (wl.chunk_tokens * wl.window_chunks)
    return {"workload": f"{wl.name} on ({block[0]}, {block[1]}, {block[2]}) blocks, local window r = {local_r}",
            "blocks_per_chunk": nb, "ms_per_step": ms_step, "attn_ms": attn_ms,
            "attn_tflops": kept / (attn_ms * 1e-3) / 1e12, "kept_fraction": kept / dense,
            "permute_in_us": span(0, 1) * 1e3, "append_us": span(1, 2) * 1e3, "lists_us": span(2, 3) * 1e3,
            "permute_out_us": span(4, 5) * 1e3}


def sparsity_sweep(wl, state, sparsities=(0.12, 0.35, 0.58, 0.72, 0.82), reps=10):
    """Attention time against sparsity on the final window of a run (the shape of the
    paper's sparsity-ratio ablation, App. L): pure top-k lists over the whole window
    (no forced chunks), budget = (1 - sparsity) * key tiles per row."""
    import torch

    win = state["win"]
    srcs, n_src = state["srcs"], state["n_src"]
    B, L, H, T = wl.batch, wl.chunk_tokens, wl.heads, wl.tile
    nt = -(-L // T)
    tail = L - (nt - 1) * T
    nk = win.info().nk_tiles
    q = srcs[(wl.window_chunks - 1 + state["steps_done"] - 1) % n_src]["q"]
    out = torch.empty((B, L, H, D), dtype=torch.bfloat16, device=q.device)
    lse = torch.empty((B, H, L), dtype=torch.float32, device=q.device)
    stream = torch.cuda.current_stream()
    dense = 4 * D * B * H * L * (L * win.info().n_live)
    rows = []
    for sp in sparsities:
        budget = int(round((1.0 - sp) * nk))
        win.build_topk_lists(q, budget, keep_sink=False, keep_current=False)
        for _ in range(2):
            win.attention(q, out=out, lse=lse)
        e = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        e[0].record(stream)
        for _ in range(reps):
            win.attention(q, out=out, lse=lse)
        e[1].record(stream)
        torch.cuda.synchronize()
        ms = e[0].elapsed_time(e[1]) / reps
        kept, _ = _flops_of_lists(win, win.lists, nt, tail, T)
        rows.append({"target_sparsity": sp, "budget": budget, "sparsity": 1.0 - kept / dense,
                     "attn_ms": ms, "tflops": kept / (ms * 1e-3) / 1e12})
    return rows


def run_stream(P, wl):
    """The streaming configuration: wl.stream_chunks chunks pushed one by one
    through the window (evict the oldest non-pinned chunk once it is full,
    append, build lists, attend), every chunk timed; the steady state is the
    chunks after the window first fills."""
    import torch
    import synth

    dev = torch.device("cuda", 0)
    B, L, H, T = wl.batch, wl.chunk_tokens, wl.heads, wl.tile
    nt = -(-L // T)
    tail = L - (nt - 1) * T
    win = P.KVWindow(B, H, L, T, wl.max_chunks, wl.pin_sink, device=dev)
    out = torch.empty((B, L, H, D), dtype=torch.bfloat16, device=dev)
    lse = torch.empty((B, H, L), dtype=torch.float32, device=dev)
    scale = 1.0 / math.sqrt(D)
    stream = torch.cuda.current_stream(dev)
    chunks = []
    for c in range(wl.stream_chunks):
        src = {name: synth.chunk_tensor(wl, c, name, device="cuda") for name in ("k", "v", "q")}
        torch.cuda.synchronize()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
        ev[0].record(stream)
        if win.info().n_live == wl.max_chunks:
            win.evict(1)
        win.append(src["k"], src["v"])
        win.build_lists(wl.seed, wl.p_prior)
        ev[1].record(stream)
        win.attention(src["q"], scale, out=out, lse=lse)
        ev[2].record(stream)
        torch.cuda.synchronize()
        kept, _ = _flops_of_lists(win, win.lists, nt, tail, T)
        attn = ev[1].elapsed_time(ev[2])
        chunks.append({"chunk": c, "n_live": win.info().n_live, "path_ms": ev[0].elapsed_time(ev[2]),
                       "attn_ms": attn, "attn_tflops": kept / (attn * 1e-3) / 1e12})
    steady = [x for x in chunks if x["chunk"] >= wl.max_chunks - 1]
    return {"workload": f"{wl.name}: {H} heads, {wl.stream_chunks} chunks through a {wl.max_chunks}-chunk window",
            "steady_state_chunks": f"{steady[0]['chunk']}..{steady[-1]['chunk']}",
            "steady_attn_ms": sum(x["attn_ms"] for x in steady) / len(steady),
            "steady_path_ms": sum(x["path_ms"] for x in steady) / len(steady),
            "steady_attn_tflops": sum(x["attn_tflops"] for x in steady) / len(steady),
            "per_chunk": [{k: (round(v, 4) if isinstance(v, float) else v) for k, v in x.items()} for x in chunks]}


def cpu_baseline(wl, state, target_s):
    """The oracle, as it stands, on a bounded sample: head 0 of the last window, leading q-tiles."""
    import numpy as np

    import oracle

    win = state["win"]
    srcs, n_src = state["srcs"], state["n_src"]
    B, L, H, T = wl.batch, wl.chunk_tokens, wl.heads, wl.tile
    nt = -(-L // T)
    tail = L - (nt - 1) * T
    info = win.info()
    seqs = [win.logical(p)[1] for p in range(info.n_live)]
    # chunk with sequence number s was appended from srcs[s % n_src]
    ring = oracle.RingModel(wl.max_chunks, wl.pin_sink)
    meta = oracle.RingModel(wl.max_chunks, wl.pin_sink)
    zeros = np.broadcast_to(np.zeros(1), (B, L, H, 1))
    for s in range(seqs[-1] + 1):
        if s in seqs:
            src = srcs[s % n_src]
            ring.live.append(oracle.ring.Chunk(s, wl.pin_sink and s == 0,
                                               src["k"][:, :, 0:1].double().cpu().numpy(),
                                               src["v"][:, :, 0:1].double().cpu().numpy()))
            meta.live.append(oracle.ring.Chunk(s, wl.pin_sink and s == 0, zeros, None))
    q = srcs[seqs[-1] % n_src]["q"][:, :, 0:1].double().cpu().numpy()
    bits = oracle.keep_bits(meta, T, oracle.KeepRule(wl.seed, wl.p_prior))[:, 0:1]
    scale = 1.0 / math.sqrt(D)

    def kept_flops(tiles):
        f = 0
        for i in tiles:
            vq = tail if i == nt - 1 else T
            for j in np.nonzero(bits[0, 0, i])[0]:
                f += vq * (tail if j % nt == nt - 1 else T)
        return f * 4 * D

    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info() if p.get("user_api") == "blas"] or [1])
    except Exception:   # threadpoolctl missing: report the affinity set
        threads = len(os.sched_getaffinity(0))
    t0 = time.perf_counter()
    oracle.sparse_causal_attention(ring, q, bits, T, scale, qtiles=[0])
    one = time.perf_counter() - t0
    n = max(1, min(nt - 1, int(target_s / max(one, 1e-3))))
    tiles = list(range(1, 1 + n))
    t0 = time.perf_counter()
    oracle.sparse_causal_attention(ring, q, bits, T, scale, qtiles=tiles)
    sec = time.perf_counter() - t0
    cpu_model = ""
    try:
        with open("/proc/cpuinfo") as f:
            cpu_model = next((ln.split(":", 1)[1].strip() for ln in f if ln.startswith("model name")), "")
    except OSError:
        pass
    return {
        "value": kept_flops(tiles) / sec / 1e12,
        "unit": "TFLOP/s",
        "cores": threads,
        "cpu_model": cpu_model,
        "kind": "oracle",
        "sample": f"{wl.name}: head 0, query tiles 1..{n} of {nt} ({n * T} queries x {L * info.n_live} keys, "
                  f"float64 numpy over each row's kept keys), {sec:.1f} s; throughput in kept-tile FLOP/s",
        "seconds": sec,
    }


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default="1k", choices=["tiny", "480p", "1k", "2k"])
    ap.add_argument("--secondary", default="2k", help="second workload reported in the same line ('' for none)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--split", type=int, default=0,
                    help="split-KV attention with this many list slices per row (0: whole rows)")
    ap.add_argument("--blocks", action="store_true",
                    help="also run the workload on (2, 8, 8) blocks with the local window r = 9")
    ap.add_argument("--no-bwd", action="store_true", help="skip timing the backward (dQ, dK, dV)")
    ap.add_argument("--no-others", action="store_true",
                    help="skip the other workloads (480p dense, tiny, the 40-head 1K stream)")
    ap.add_argument("--sweep", action="store_true",
                    help="also time the attention against sparsity (top-k lists, no forced chunks)")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="after the run, copy a buffer of this many MiB three times with a plain device copy "
                         "(reference dispatches for scaling hardware byte counters)")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py runs on one GPU only: the attention path has no multi-GPU variant here "
              "(heads would shard across GPUs with no exchange inside the kernel)", file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2606_09150_amd as P
    import synth

    P.load()
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)

    wl = synth.WORKLOADS[args.config]
    res, state = run_workload(P, wl, args.steps, args.warmup, split=args.split)
    if args.split:
        res["split"] = args.split
    line = {
        "metric": METRIC,
        "value": res["value"],
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": res["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"{wl.name}-shaped block-sparse chunk-causal attention",
                   "batch": wl.batch, "heads": wl.heads, "head_dim": D, "chunk_tokens": wl.chunk_tokens,
                   "grid": f"{wl.frames}x{wl.grid_h}x{wl.grid_w}", "tile": wl.tile,
                   "window_chunks": wl.window_chunks, "keys": res["keys"], "p_prior": wl.p_prior,
                   "pinned_first_chunk": wl.pin_sink},
    }
    for k in ("split",) if args.split else ():
        line[k] = res[k]
    for k in ("attn_ms", "attn_ms_median", "attn_ms_p10", "attn_ms_p90", "attn_tflops", "append_us", "append_gbps", "lists_us",
              "topk_budget", "topk_lists_us", "kept_tflop_per_step", "kept_fraction", "padded_tile_tflop_per_step"):
        line[k] = res[k]
    line["roofline"] = {
        "bound": "mfma",
        "achieved": res["attn_tflops"],
        "peak": MFMA_BF16_PEAK_TFLOPS,
        "unit": "TFLOP/s",
        "frac": res["attn_tflops"] / MFMA_BF16_PEAK_TFLOPS,
        "traffic": measured_traffic(wl.name),
    }
    if not args.no_bwd:
        line["backward"] = run_backward(P, wl, state)
    if args.sweep:
        line["sweep"] = sparsity_sweep(wl, state)
    if args.blocks:
        line["blocks"] = run_blocked(P, wl, max(5, args.steps // 2), args.warmup)
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(wl, state, args.cpu_seconds)
    del state
    torch.cuda.empty_cache()
    if args.secondary and args.secondary != args.config:
        wl2 = synth.WORKLOADS[args.secondary]
        res2, state2 = run_workload(P, wl2, max(5, args.steps // 2), args.warmup)
        res2["roofline_frac"] = res2["attn_tflops"] / MFMA_BF16_PEAK_TFLOPS
        if not args.no_bwd:
            res2["backward"] = run_backward(P, wl2, state2)
        line["secondary"] = res2
        del state2
        torch.cuda.empty_cache()
    if not args.no_others:
        others = {}
        for name in ("480p", "tiny"):
            r, st2 = run_workload(P, synth.WORKLOADS[name], 10, args.warmup)
            keep = ("workload", "ms_per_step", "attn_ms", "attn_ms_median", "attn_tflops", "attn_unique_gbps",
                    "append_us", "append_gbps", "lists_us", "kept_fraction")
            others[name] = {k: r[k] for k in keep}
            others[name]["roofline_frac"] = r["attn_tflops"] / MFMA_BF16_PEAK_TFLOPS
            if name == "tiny" and not args.no_bwd:
                others[name]["backward"] = run_backward(P, synth.WORKLOADS[name], st2, reps=20)
            del st2
            if name == "480p":
                # the same workload with the rows of the last, partly filled round split
                r, st2 = run_workload(P, synth.WORKLOADS[name], 10, args.warmup, split="tail")
                others[name]["tail_split"] = {k: r[k] for k in ("ms_per_step", "attn_ms", "attn_ms_median",
                                                                "attn_tflops")}
                others[name]["tail_split"]["roofline_frac"] = r["attn_tflops"] / MFMA_BF16_PEAK_TFLOPS
                n_cu = torch.cuda.get_device_properties(0).multi_processor_count
                others[name]["tail_split"]["plan"] = list(P.uf_attn_tail_plan(st2["win"].handle, n_cu))
                del st2
                # and rows 256.. (the last round on 256 CUs) in 4 slices, whether or not the plan takes it
                r, st2 = run_workload(P, synth.WORKLOADS[name], 10, args.warmup, split=(256, 4))
                others[name]["split_rows_256_4"] = {k: r[k] for k in ("ms_per_step", "attn_ms", "attn_ms_median",
                                                                      "attn_tflops")}
                del st2
        others["1k_stream"] = run_stream(P, synth.WORKLOADS["1k_stream"])
        line["others"] = others
        torch.cuda.empty_cache()
    if args.calib_copy_mib > 0:
        n = args.calib_copy_mib << 20
        src = torch.ones(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        line["calib_copy_bytes"] = n
        del src, dst
    line["context"] = ("paper (whole cascade, not this kernel): ~30 FPS at 1K and ~18 FPS at 2K on a single "
                       "B200, ~17 / ~10 FPS on a single H200")
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
