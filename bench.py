"""Benchmark of the ValueDiff eviction pass on one MI355X.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--no-cpu-baseline]

A step is one eviction pass (one ``vd_evict_step`` launch: mean, score, top-N,
gather for every unit) over one boundary of the workload, with its inputs
resident in HBM when timing starts.  The default workload is the
Llama-3-8B-shaped prefill eviction (1 sequence, 32 layers x 8 KV heads,
head_dim 128, bf16, budget 2048, block 512, prompt 32768: 60 evicting passes
at n = 2560).  Its pre-pass states are taken from the real block-processing
trajectory (untimed) and each timed pass consumes a fresh copy, so no pass
sees a cache the previous one already compacted.

Printed: ONE JSON line with passes/s (value), KV GB/s scanned, the roofline
of the pass kernel (algorithmic bytes per launch / mean launch time, against
8 TB/s) and the oracle's CPU throughput on a bounded sample.
"""
import argparse
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

from paper_2609_23314_amd import synth, vd  # noqa: E402

HBM_PEAK_GBPS = 8000.0
METRIC = "eviction passes/s + KV GB/s scanned (fraction of HBM peak), 1 MI355X"
KERNEL_SRC = os.path.join(ROOT, "paper_2609_23314_amd", "csrc", "vd_kernels.hip")
TRAFFIC_DIR = os.path.join(ROOT, "profiles")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def kernel_hash() -> str:
    """Hash of the kernel and host sources with comments and blank space
    removed, so that profiles stay tied to the code, not to its comments."""
    h = hashlib.sha256()
    for f in (KERNEL_SRC, os.path.join(ROOT, "paper_2609_23314_amd", "csrc", "vd_api.cpp")):
        with open(f, encoding="utf-8") as fh:
            text = fh.read()
        text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
        text = re.sub(r"//[^\n]*", " ", text)
        h.update(" ".join(text.split()).encode())
    return h.hexdigest()[:16]


# ---------------------------------------------------------------- trajectories

def prefill_states(w: synth.Workload, count: int, dev):
    """Pre-pass states (k, v, running_sum, n, movers per unit) of the first
    `count` evicting boundaries of sequence-synchronous block processing."""
    S, L, H, D, B = w.num_seqs, w.num_layers, w.num_kv_heads, w.head_dim, w.block
    C, U = w.capacity, w.units
    k, v = synth.empty_cache(w, dev)
    rs = torch.zeros((U, D + 1), dtype=torch.float64, device=dev)
    n = [0] * S
    states = []
    blk = 0
    while len(states) < count:
        for s in range(S):
            t0 = blk * B
            t1 = min(t0 + B, w.prompt[s])
            if t1 > t0:
                k[s, :, :, n[s]:n[s] + t1 - t0] = synth.block_rows(w, "k", s, blk, t0, t1, dev)
                v[s, :, :, n[s]:n[s] + t1 - t0] = synth.block_rows(w, "v", s, blk, t0, t1, dev)
                n[s] += t1 - t0
        blk += 1
        if blk * B >= max(w.prompt) and not any(a > b for a, b in zip(n, w.budget)):
            break
        if any(a > b for a, b in zip(n, w.budget)):
            keep = torch.zeros((U, C), dtype=torch.uint8, device=dev)
            snap = (k.clone(), v.clone(), rs.clone(), list(n))
            vd.vd_evict_step(k, v, n, w.budget, "l2", running_sum=rs, keep_out=keep)
            movers = []
            for s in range(S):
                N = w.budget[s]
                us = slice(s * L * H, (s + 1) * L * H)
                movers.append(int(keep[us, N:n[s]].sum().item()) if n[s] > N else 0)
            states.append(snap + (movers,))
            n = [min(a, b) for a, b in zip(n, w.budget)]
    return states


def algorithmic_bytes(w: synth.Workload, n, movers) -> int:
    """One read of every cached value row, K read + K write + V write per moved
    row, the running-sum state read and written; summed over units."""
    L, H, D = w.num_layers, w.num_kv_heads, w.head_dim
    row = w.row_bytes
    total = 0
    for s in range(w.num_seqs):
        if n[s] > w.budget[s]:
            total += L * H * n[s] * row + movers[s] * 3 * row
        total += L * H * 2 * (D + 1) * 8
    return total


def scanned_bytes(w, n) -> int:
    return sum(w.num_layers * w.num_kv_heads * n[s] * w.row_bytes
               for s in range(w.num_seqs) if n[s] > w.budget[s])


# ---------------------------------------------------------------- timing

def time_pool(w, states, steps, warmup, dev):
    """Times `steps` passes, each on a fresh copy of a pre-pass state.  The
    copies are made before each timed segment; inside a segment the passes run
    back to back on one stream, bracketed by two HIP events.  Returns (wall
    seconds of the timed segments, GPU milliseconds of the timed segments,
    per-launch algorithmic and scanned bytes)."""
    pool_n = min(len(states), max(steps, 1))
    work = [(st[0].clone(), st[1].clone(), st[2].clone()) for st in states[:pool_n]]

    def refill(i0, cnt):
        for j in range(cnt):
            st = states[(i0 + j) % len(states)]
            wk, wv, wr = work[j]
            wk.copy_(st[0])
            wv.copy_(st[1])
            wr.copy_(st[2])

    # The copies above leave up to a few hundred MB of dirty lines in L2 and
    # the MALL; a read of a buffer larger than both evicts them before each
    # timed segment, so that the passes do not pay for the copies' write-back.
    flush_buf = torch.zeros(1 << 28, dtype=torch.float32, device=dev)   # 1 GiB

    def flush():
        flush_buf.sum()

    stream = torch.cuda.current_stream(dev)
    done = 0
    for i in range(warmup):
        refill(i, 1)
        st = states[i % len(states)]
        vd.vd_evict_step(work[0][0], work[0][1], st[3], w.budget, "l2", running_sum=work[0][2])
    torch.cuda.synchronize()
    wall_s, gpu_ms, alg, scan = 0.0, 0.0, [], []
    while done < steps:
        seg = min(pool_n, steps - done)
        refill(done, seg)
        flush()
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        t0 = time.perf_counter()
        e0.record(stream)
        for j in range(seg):
            st = states[(done + j) % len(states)]
            vd.vd_evict_step(work[j][0], work[j][1], st[3], w.budget, "l2",
                             running_sum=work[j][2])
        e1.record(stream)
        torch.cuda.synchronize()
        wall_s += time.perf_counter() - t0
        gpu_ms += e0.elapsed_time(e1)
        for j in range(seg):
            st = states[(done + j) % len(states)]
            alg.append(algorithmic_bytes(w, st[3], st[4]))
            scan.append(scanned_bytes(w, st[3]))
        done += seg
    return wall_s, gpu_ms, alg, scan


def stream_read_gbps(dev, nbytes=2 << 30, reps=5):
    """Read bandwidth of the library's plain streaming read (vd_stream_read)
    over a 2 GiB buffer: the practical HBM read ceiling on this GPU, next to
    the 8 TB/s peak.  Best of `reps` timed runs, in GB/s."""
    buf = torch.ones(nbytes // 4, dtype=torch.float32, device=dev)
    sink = torch.zeros(1, dtype=torch.int32, device=dev)
    vd.vd_stream_read(buf, sink)
    torch.cuda.synchronize()
    best = float("inf")
    for _ in range(reps):
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record()
        vd.vd_stream_read(buf, sink)
        e1.record()
        torch.cuda.synchronize()
        best = min(best, e0.elapsed_time(e1) / 1e3)
    del buf
    return nbytes / best / 1e9


def decode_state(w: synth.Workload, dev):
    """A decode step of every sequence: N old tokens and one new token in the
    cache (n = N + 1), and the running sum of the N old rows."""
    S, L, H, D = w.num_seqs, w.num_layers, w.num_kv_heads, w.head_dim
    k, v = synth.empty_cache(w, dev)
    rs = torch.zeros((w.units, D + 1), dtype=torch.float64, device=dev)
    for s in range(S):
        N = w.budget[s]
        k[s, :, :, :N + 1] = synth.block_rows(w, "k", s, 0, 0, N + 1, dev, seq_seed=s)
        v[s, :, :, :N + 1] = synth.block_rows(w, "v", s, 0, 0, N + 1, dev, seq_seed=s)
        us = slice(s * L * H, (s + 1) * L * H)
        rs[us, :D] = v[s, :, :, :N].double().sum(dim=2).reshape(L * H, D)
        rs[us, D] = N
    return k, v, rs, [N + 1 for N in w.budget]


def time_in_place(w, k, v, rs, n, steps, warmup, dev):
    """Decode passes replayed on one cache: after a pass the valid slots are
    [0, N) and slot N still holds a row, so the next call with n = N + 1 is
    again a well-formed decode step (its new token is that row).  Returns
    (wall seconds, GPU milliseconds) of `steps` back-to-back passes."""
    for _ in range(warmup):
        vd.vd_evict_step(k, v, n, w.budget, "l2", running_sum=rs)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream(dev)
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record(stream)
    for _ in range(steps):
        vd.vd_evict_step(k, v, n, w.budget, "l2", running_sum=rs)
    e1.record(stream)
    torch.cuda.synchronize()
    return time.perf_counter() - t0, e0.elapsed_time(e1)


def decode_movers(w, k, v, rs, n, dev):
    """Moved rows per unit of one decode pass (run on copies, untimed)."""
    keep = torch.zeros((w.units, w.capacity), dtype=torch.uint8, device=dev)
    vd.vd_evict_step(k.clone(), v.clone(), n, w.budget, "l2", running_sum=rs.clone(),
                     keep_out=keep)
    L, H = w.num_layers, w.num_kv_heads
    out = []
    for s in range(w.num_seqs):
        N = w.budget[s]
        out.append(int(keep[s * L * H:(s + 1) * L * H, N].sum().item()))
    return out


# ---------------------------------------------------------------- oracle baseline

def cpu_baseline(w, state, budget_s=10.0, max_units=None):
    """The oracle on the host cores: whole passes over one pre-pass state, or
    over its first `max_units` units (then scaled to whole passes)."""
    import oracle
    k, v, _, n, _ = state
    S, L, H, C, D = k.shape
    U = S * L * H
    take = U if max_units is None else min(U, max_units)
    kn = to_np(k.reshape(U, C, D)[:take])
    vn = to_np(v.reshape(U, C, D)[:take])
    nu = np.repeat(np.asarray(n, np.int32), L * H)[:take]
    Nu = np.repeat(np.asarray(w.budget, np.int32), L * H)[:take]
    threads = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
    orc = oracle.load()
    elapsed, reps = 0.0, 0
    while elapsed < budget_s or reps == 0:
        kc, vc = kn.copy(), vn.copy()
        t0 = time.perf_counter()
        orc.evict_step(kc, vc, nu, Nu, "l2", nthreads=threads)
        elapsed += time.perf_counter() - t0
        reps += 1
    frac = take / U
    what = (f"{reps} whole passes of one {w.name} boundary ({U} units, n={max(n)})" if take == U
            else f"{reps} passes over {take} of the {U} units of one {w.name} step "
                 f"(n={max(n)}), scaled to whole passes")
    return {"value": reps * frac / elapsed, "unit": "passes/s", "cores": threads,
            "kind": "oracle", "sample": f"{what} in {elapsed:.1f} s",
            "gbps_scanned": reps * frac * scanned_bytes(w, n) / elapsed / 1e9}


def to_np(t):
    t = t.detach().contiguous().cpu()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


def load_traffic(workload: str):
    """HBM traffic per launch measured with rocprofv3 counters for this kernel
    source, or None when absent or taken on another kernel version."""
    path = os.path.join(TRAFFIC_DIR, f"traffic_{workload}.json")
    if not os.path.exists(path):
        return None
    with open(path) as fh:
        t = json.load(fh)
    if t.get("kernel_hash") != kernel_hash():
        return None
    return t.get("bytes_per_launch")


def geometry_bench(w, args, dev):
    """Times vd_geometry (sigma_K, sigma_V, mean distances and bos-cosim of
    every unit; Sec. 3.1, Sec. 4) over the workload's cache with every unit
    filled to capacity by the workload's generator.  The passes run back to
    back on one stream between two HIP events, after a read of a 1 GiB buffer
    that evicts the cache from L2 and the MALL.  Algorithmic bytes are one
    read of K and V (the kernel reads both twice: centroids, then distances)."""
    C = w.capacity
    log(f"bench: building the {w.name} cache at capacity ({w.units} units x {C} rows)")
    k, v = synth.empty_cache(w, dev)
    for s_ in range(w.num_seqs):
        k[s_] = synth.block_rows(w, "k", s_, 0, 0, C, dev)
        v[s_] = synth.block_rows(w, "v", s_, 0, 0, C, dev)
    n = [C] * w.num_seqs
    out = torch.empty((w.units, 5), dtype=torch.float64, device=dev)
    flush_buf = torch.zeros(1 << 28, dtype=torch.float32, device=dev)
    for _ in range(args.warmup):
        vd.vd_geometry(k, v, n, out)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream(dev)
    gpu_ms, wall_s, done = 0.0, 0.0, 0
    while done < args.steps:   # segments of at most 20 passes, each after a flush
        seg = min(20, args.steps - done)
        flush_buf.sum()
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        t0 = time.perf_counter()
        e0.record(stream)
        for _ in range(seg):
            vd.vd_geometry(k, v, n, out)
        e1.record(stream)
        torch.cuda.synchronize()
        wall_s += time.perf_counter() - t0
        gpu_ms += e0.elapsed_time(e1)
        done += seg
    alg = 2 * w.units * C * w.row_bytes
    traffic = load_traffic(f"geometry_{w.name}")
    us = gpu_ms / args.steps * 1e3
    alg_gbps = alg / (us * 1e-6) / 1e9
    log(f"bench: geometry {us:.2f} us per launch, {alg_gbps:.0f} GB/s algorithmic")
    res = {
        "metric": "geometry passes/s (sigma_K, sigma_V, mean distances, bos-cosim of every unit)",
        "value": round(args.steps / wall_s, 2),
        "unit": "passes/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(wall_s / args.steps * 1e3, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16" if w.dtype == torch.bfloat16 else "f32",
        "data": "synthetic (seeded generator; no model weights or datasets)",
        "config": {"workload": f"{w.name} cache at capacity", "seqs": w.num_seqs,
                   "layers": w.num_layers, "kv_heads": w.num_kv_heads,
                   "head_dim": w.head_dim, "n": C},
        "roofline": {"bound": "hbm", "achieved": round(alg_gbps, 1), "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s", "frac": round(alg_gbps / HBM_PEAK_GBPS, 4),
                     "traffic": None if traffic is None else int(traffic),
                     "traffic_over_alg": None if traffic is None else round(traffic / alg, 3),
                     "kernel": f"geometry_kernel<bf16,{w.head_dim}>",
                     "launch_us": round(us, 2), "alg_bytes_per_launch": alg,
                     "bytes_read_per_launch": 2 * alg},
    }
    if not args.no_cpu_baseline:
        log("bench: timing the oracle's geometry on the host ...")
        res["cpu_baseline"] = cpu_geometry(w, k, v, args.cpu_seconds)
    return res


def decode_attention_bench(args, dev):
    """Decode steps of the decode_b16 workload with the attention of the newest
    token fused to its eviction: per step one vd_decode_attention_evict call
    per layer (the layers of a model run one after another), each over the
    layer's 16 x 8 units at n = N + 1 = 4097, with that layer's running sum.
    The calls are replayed in place (after a call slot N still holds a row, so
    n = N + 1 is again a well-formed step).  Algorithmic bytes per call: one
    read of K and V, the moved rows (K and V read and written), the running
    sum read and written, q read and the output written."""
    w = synth.decode()
    S, L, H, D = w.num_seqs, w.num_layers, w.num_kv_heads, w.head_dim
    Hq, N = w.num_q_heads, w.budget[0]
    log(f"bench: building the {w.name} decode cache ({w.units} units)")
    k, v, rs, n = decode_state(w, dev)
    rs_l = [rs.view(S, L, H, D + 1)[:, l].reshape(S * H, D + 1).contiguous() for l in range(L)]
    g = torch.Generator(device=dev)
    g.manual_seed(1234)
    q_l = [torch.randn((S, 1, Hq, D), generator=g, device=dev) for _ in range(L)]
    out = torch.empty((S, 1, Hq, D), dtype=torch.float32, device=dev)
    kv_l = [(k[:, l:l + 1], v[:, l:l + 1]) for l in range(L)]
    ws = torch.zeros(vd.vd_decode_attention_workspace_size(kv_l[0][0], kv_l[0][1], Hq),
                     dtype=torch.uint8, device=dev)
    # moved rows of one call (untimed, on copies)
    pos = torch.arange(w.capacity, dtype=torch.int32, device=dev).repeat(S * H, 1).contiguous()
    vd.vd_decode_attention_evict(kv_l[0][0].clone(), kv_l[0][1].clone(), q_l[0], n, w.budget,
                                 rs_l[0].clone(), pos=pos, out=out, workspace=ws)
    movers = int((pos[:, :N] != torch.arange(N, dtype=torch.int32, device=dev)).any(dim=1).sum())

    def step():
        for l in range(L):
            vd.vd_decode_attention_evict(kv_l[l][0], kv_l[l][1], q_l[l], n, w.budget, rs_l[l],
                                         out=out, workspace=ws)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream(dev)
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record(stream)
    for _ in range(args.steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms = e0.elapsed_time(e1)
    calls = args.steps * L
    us_call = ms * 1e3 / calls
    units = S * H
    alg = (2 * units * (N + 1) * w.row_bytes + movers * 4 * w.row_bytes
           + units * (D + 1) * 16 + S * Hq * D * 8)
    gbps = alg / (us_call * 1e-6) / 1e9
    traffic = load_traffic("decode_attention_decode_b16")
    log(f"bench: {us_call:.2f} us per layer call, {gbps:.0f} GB/s algorithmic, {movers} movers of {units}")
    # the eviction pass alone over all layers (vd_evict_step), for context
    _, ev_ms = time_in_place(w, k, v, rs, n, 10, 2, dev)
    res = {
        "metric": "decode steps/s (attention of the newest token fused to its eviction, all layers)",
        "value": round(args.steps / wall, 2),
        "unit": "steps/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(wall / args.steps * 1e3, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded generator; no model weights or datasets)",
        "config": {"workload": "decode_b16 decode step, one call per layer", "seqs": S,
                   "layers": L, "kv_heads": H, "q_heads": Hq, "head_dim": D, "budget": N,
                   "n": N + 1},
        "roofline": {"bound": "hbm", "achieved": round(gbps, 1), "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s", "frac": round(gbps / HBM_PEAK_GBPS, 4),
                     "traffic": None if traffic is None else int(traffic),
                     "traffic_over_alg": None if traffic is None else round(traffic / alg, 3),
                     "kernel": "attn_split_kernel<bf16,128,4> + attn_combine_kernel (one call)",
                     "launch_us": round(us_call, 2), "alg_bytes_per_launch": alg},
        "evict_pass_alone_us": round(ev_ms * 1e3 / 10, 2),
    }
    if not args.no_cpu_baseline:
        log("bench: timing the oracle on the host ...")
        res["cpu_baseline"] = cpu_decode_attention(w, kv_l[0][0], kv_l[0][1], q_l[0], rs_l[0],
                                                   n, args.cpu_seconds)
    return res


def cpu_decode_attention(w, k, v, q, rs, n, budget_s):
    """The oracle's attention (every query head) and eviction for units of one
    layer, one at a time, for about budget_s seconds; scaled to whole steps
    (all layers) per second."""
    import oracle
    orc = oracle.load()
    S, H, D, C = w.num_seqs, w.num_kv_heads, w.head_dim, w.capacity
    G = w.num_q_heads // H
    kn = to_np(k).reshape(S * H, C, D)
    vn = to_np(v).reshape(S * H, C, D)
    qn = q.cpu().numpy().astype(np.float64).reshape(S * H, G, D)
    m = n[0]
    t0, done = time.perf_counter(), 0
    while done < S * H and time.perf_counter() - t0 < budget_s:
        for g in range(G):
            orc.attention(qn[done, g], kn[done, :m], vn[done, :m], D ** -0.5)
        kc, vc = kn[done:done + 1].copy(), vn[done:done + 1].copy()
        orc.evict_step(kc, vc, np.array([m], np.int32), np.array([w.budget[0]], np.int32), "l2")
        done += 1
    el = time.perf_counter() - t0
    return {"value": round(done / el / w.units, 4), "unit": "steps/s", "cores": 1,
            "kind": "oracle",
            "sample": f"{done} units of one layer (attention of {G} heads and eviction, n={m}), "
                      f"one thread, scaled to a step of {w.units} units"}


def cpu_geometry(w, k, v, budget_s):
    """The oracle's geometry of units 0, 1, 2, ... of sequence 0 until about
    budget_s seconds have passed, scaled to passes over every unit per second."""
    import oracle
    orc = oracle.load()
    ku = to_np(k[0]).reshape(-1, w.capacity, w.head_dim)
    vu = to_np(v[0]).reshape(-1, w.capacity, w.head_dim)
    t0, done = time.perf_counter(), 0
    while done < ku.shape[0] and time.perf_counter() - t0 < budget_s:
        orc.geometry(ku[done], vu[done])
        done += 1
    el = time.perf_counter() - t0
    return {"value": round(done / el / w.units, 4), "unit": "passes/s", "cores": 1,
            "kind": "oracle",
            "sample": f"{done} of {w.units} units of {w.capacity} rows, one thread"}


# ---------------------------------------------------------------- main

def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=60)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="llama3_8b_prefill",
                    choices=["llama3_8b_prefill", "wide_head_d256", "decode_b16",
                             "ragged_serving"],
                    help="the last two time decode steps (n = N + 1 in every sequence)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--geometry", action="store_true",
                    help="time the geometry diagnostics (vd_geometry) over the workload's "
                         "cache filled to capacity instead of the pass")
    ap.add_argument("--decode-attention", action="store_true",
                    help="time decode steps of the decode_b16 workload with attention fused "
                         "to the eviction (vd_decode_attention_evict), one call per layer")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 1 GiB device copy three times (reference for the "
                         "HBM byte counters) and exit")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the eviction pass has no cross-GPU step "
              "(units shard across GPUs with no exchange); run it with --gpus 1.",
              file=sys.stderr)
        sys.exit(2)
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.copy_calibration:
        src = torch.ones(1 << 28, dtype=torch.float32, device=dev)   # 1 GiB
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes": src.numel() * 4, "copies": 3}))
        return
    vd.load()
    w = synth.WORKLOADS[args.workload]()
    if args.geometry:
        print(json.dumps(geometry_bench(w, args, dev)), flush=True)
        return
    if args.decode_attention:
        print(json.dumps(decode_attention_bench(args, dev)), flush=True)
        return
    decode = args.workload in ("decode_b16", "ragged_serving")
    if decode:
        log(f"bench: building the {w.name} decode cache ({w.units} units) ...")
        k, v, rs, n = decode_state(w, dev)
        movers = decode_movers(w, k, v, rs, n, dev)
        log(f"bench: timing {args.steps} decode passes in place")
        total_s, gpu_ms = time_in_place(w, k, v, rs, n, args.steps, args.warmup, dev)
        alg = [algorithmic_bytes(w, n, movers)] * args.steps
        scan = [scanned_bytes(w, n)] * args.steps
        base_state = (k, v, rs, n, movers)
    else:
        pool = 60 if w.name == "llama3_8b_prefill" else 8
        log(f"bench: building {pool} pre-pass states of {w.name} ...")
        t0 = time.perf_counter()
        states = prefill_states(w, min(pool, max(args.steps, 1)), dev)
        log(f"bench: states ready in {time.perf_counter() - t0:.1f} s; timing {args.steps} passes")
        total_s, gpu_ms, alg, scan = time_pool(w, states, args.steps, args.warmup, dev)
        base_state = states[0]
    ms_launch = gpu_ms / args.steps          # launch to launch, back to back
    passes_per_s = args.steps / total_s
    kernel_s = gpu_ms / 1e3
    alg_gbps = sum(alg) / kernel_s / 1e9
    scan_gbps = sum(scan) / kernel_s / 1e9
    log(f"bench: {passes_per_s:.1f} passes/s wall, {ms_launch * 1e3:.2f} us per launch (HIP events)")
    traffic = load_traffic(w.name)
    evicting_units = sum(w.num_layers * w.num_kv_heads for s_ in range(w.num_seqs)
                         if base_state[3][s_] > w.budget[s_])
    stream_gbps = stream_read_gbps(dev)
    out = {
        "metric": METRIC,
        "value": round(passes_per_s, 2),
        "unit": "passes/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(total_s / args.steps * 1e3, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if w.dtype == torch.bfloat16 else "f32",
        "data": "synthetic (seeded generator; no model weights or datasets)",
        "config": {"workload": w.name, "seqs": w.num_seqs, "layers": w.num_layers,
                   "kv_heads": w.num_kv_heads, "q_heads": w.num_q_heads,
                   "head_dim": w.head_dim,
                   "budget": (w.budget[0] if len(set(w.budget)) == 1
                              else [min(w.budget), max(w.budget)]),
                   "block": w.block,
                   "prompt": max(w.prompt), "n": max(base_state[3]), "variant": "l2",
                   "running_sum": True, "parallelism": "single GPU"},
        "head_passes_per_s": round(passes_per_s * evicting_units, 1),
        "kv_gbps_scanned": round(scan_gbps, 1),
        "kv_scan_frac_of_hbm_peak": round(scan_gbps / HBM_PEAK_GBPS, 4),
        "stream_read_gbps": round(stream_gbps, 1),
        "alg_frac_of_stream_read": round(alg_gbps / stream_gbps, 4),
        "roofline": {"bound": "hbm", "achieved": round(alg_gbps, 1), "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s", "frac": round(alg_gbps / HBM_PEAK_GBPS, 4),
                     "traffic": None if traffic is None else int(traffic),
                     "traffic_over_alg": (None if traffic is None else
                                          round(traffic / (sum(alg) / len(alg)), 3)),
                     "kernel": f"step_kernel<bf16,{w.head_dim},L2>",
                     "launch_us": round(ms_launch * 1e3, 2),
                     "alg_bytes_per_launch": int(np.mean(alg))},
    }
    if not args.no_cpu_baseline:
        log("bench: timing the oracle on the host ...")
        out["cpu_baseline"] = cpu_baseline(w, base_state, args.cpu_seconds,
                                           max_units=64 if decode else None)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
