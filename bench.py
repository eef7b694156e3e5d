"""Benchmark of the ValueDiff eviction pass on one MI355X.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--variant V]
                    [--phase prefill|decode] [--no-cpu-baseline] [--launch auto|graph|eager]

A step is one eviction pass (one ``vd_evict_step`` launch: mean, score, top-N,
gather for every unit) over one boundary of the workload, with its inputs
resident in HBM when timing starts.  The default workload is the
Llama-3-8B-shaped prefill eviction (1 sequence, 32 layers x 8 KV heads,
head_dim 128, bf16, budget 2048, block 512, prompt 32768: 60 evicting passes
at n = 2560).  The pre-pass states of all 60 boundaries are taken from the
real block-processing trajectory (untimed); the K timed passes are spread
evenly over them (boundary floor(i * 60 / K) for pass i), and each timed pass
consumes a fresh copy of its state, so no pass sees a cache the previous one
already compacted.  The boundaries timed are printed with the result, and the
HBM byte counters of profiles/ are kept per boundary, so that the traffic
reported is the mean over exactly the boundaries timed.  The timed passes of
a segment are launched one by one, or, where a pass moves under 16 MB and
the host's ~30 us per launch would outlast the kernel (the tiny workload),
from a captured HIP graph (one host launch per segment); --launch chooses.
Graph-launched kernels of this size run about 1.5 us apart on this stack, so
the longer passes are timed from eager launches.

Printed: ONE JSON line with passes/s (value), KV GB/s scanned, the roofline
of the pass kernel (algorithmic bytes per launch / mean launch time, against
8 TB/s), the oracle's CPU throughput on a bounded sample (all host cores and
one core) and the near-tie count of a parity sample against the oracle.

Other modes (each prints one JSON line of the same form):
  --workload tiny | wide_head_d256     prefill boundaries of those workloads
  --workload decode_b16 | ragged_serving   decode steps (n = N + 1), in place
  --workload ragged_serving --phase prefill   the lock-step prefill calls
  --variant dir | norm | key_l2 | key_dir | key_norm   another score
  --geometry             vd_geometry over the workload's cache at capacity
  --decode-attention     the fused decode step (vd_decode_attention_evict)
  --copy-calibration     a plain 1 GiB copy, the reference of the counters
  --summarize-traces DIR / --summarize-counters DIR / --summarize-sq DIR
                         turn rocprofv3 CSV output into the summaries kept
                         in profiles/
"""
import argparse
import csv
import glob
import hashlib
import json
import math
import os
import re
import statistics
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
REL_TIE = 1e-5          # near-tie band of the parity rule (relative to the N-th score)
ALL_BOUNDARIES = {"llama3_8b_prefill": 1, "wide_head_d256": 6, "tiny": 1}  # keep every k-th


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


def spread(count: int, steps: int):
    """Indices of `steps` timed passes spread evenly over `count` states."""
    if steps <= count:
        return [i * count // steps for i in range(steps)]
    return [i % count for i in range(steps)]


# ---------------------------------------------------------------- trajectories

def prefill_states(w: synth.Workload, variant: str, dev, every: int = 1):
    """Pre-pass states (k, v, running_sum, n, movers per sequence, boundary
    index) of the evicting boundaries of sequence-synchronous block processing:
    every `every`-th evicting boundary and the last one are kept."""
    S, L, H, D, B = w.num_seqs, w.num_layers, w.num_kv_heads, w.head_dim, w.block
    C, U = w.capacity, w.units
    if w.name == "tiny":
        return tiny_states(w, variant, dev)
    k, v = synth.empty_cache(w, dev)
    rs = torch.zeros((U, D + 1), dtype=torch.float64, device=dev)
    n = [0] * S
    states, b_idx = [], 0
    nblocks = (max(w.prompt) + B - 1) // B
    n_evicting = sum(1 for blk in range(nblocks)
                     if any(min(w.budget[s], blk * B) + max(0, min(B, w.prompt[s] - blk * B))
                            > w.budget[s] for s in range(S)))
    for blk in range(nblocks):
        for s in range(S):
            t0 = blk * B
            t1 = min(t0 + B, w.prompt[s])
            if t1 > t0:
                k[s, :, :, n[s]:n[s] + t1 - t0] = synth.block_rows(w, "k", s, blk, t0, t1, dev)
                v[s, :, :, n[s]:n[s] + t1 - t0] = synth.block_rows(w, "v", s, blk, t0, t1, dev)
                n[s] += t1 - t0
        if any(a > b for a, b in zip(n, w.budget)):
            keep = torch.zeros((U, C), dtype=torch.uint8, device=dev)
            take = b_idx % every == 0 or b_idx == n_evicting - 1
            snap = (k.clone(), v.clone(), rs.clone(), list(n)) if take else None
            vd.vd_evict_step(k, v, n, w.budget, variant, running_sum=rs, keep_out=keep)
            if take:
                states.append(snap + (movers_of(w, keep, n), b_idx))
            b_idx += 1
        else:   # nothing evicts yet: the state absorbs the block, as in block processing
            vd.vd_evict_step(k, v, n, w.budget, variant, running_sum=rs)
        n = [min(a, b) for a, b in zip(n, w.budget)]
    return states


def tiny_states(w, variant, dev):
    """The 44 evicting passes of the tiny workload: 16 prefill blocks of 16
    tokens (12 evict, n = 80) and 32 decode steps (n = 65)."""
    K, V = synth.tiny_rows()
    C, N = w.capacity, w.budget[0]
    k = torch.zeros((1, 1, 1, C, 64), device=dev)
    v = torch.zeros((1, 1, 1, C, 64), device=dev)
    rs = torch.zeros((1, 65), dtype=torch.float64, device=dev)
    n, states = 0, []
    plan = [(16 * i, 16 * i + 16) for i in range(16)] + [(256 + t, 257 + t) for t in range(32)]
    for t0, t1 in plan:
        k[0, 0, 0, n:n + t1 - t0] = torch.from_numpy(K[t0:t1]).to(dev)
        v[0, 0, 0, n:n + t1 - t0] = torch.from_numpy(V[t0:t1]).to(dev)
        n += t1 - t0
        if n > N:
            keep = torch.zeros((1, C), dtype=torch.uint8, device=dev)
            snap = (k.clone(), v.clone(), rs.clone(), [n])
            vd.vd_evict_step(k, v, [n], [N], variant, running_sum=rs, keep_out=keep)
            states.append(snap + (movers_of(w, keep, [n]), len(states)))
        else:
            vd.vd_evict_step(k, v, [n], [N], variant, running_sum=rs)
        n = min(n, N)
    return states


def movers_of(w, keep, n):
    """Moved rows per sequence (kept slots at or above N), from a keep mask."""
    L, H = w.num_layers, w.num_kv_heads
    out = []
    for s in range(w.num_seqs):
        N = w.budget[s]
        us = slice(s * L * H, (s + 1) * L * H)
        out.append(int(keep[us, N:n[s]].sum().item()) if n[s] > N else 0)
    return out


def algorithmic_bytes(w: synth.Workload, n, movers) -> int:
    """One read of every cached row of the scored tensor, K read + K write +
    V write per moved row (the moved V row comes from LDS), the running-sum
    state read and written; summed over units."""
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

def time_pool(w, states, order, warmup, variant, dev, graph=True):
    """Times one pass per entry of `order` (indices into `states`), each on a
    fresh copy of its pre-pass state.  The copies of a segment are made before
    it; inside a segment the passes run back to back on one stream.

    With `graph` the passes of a segment are captured once in a HIP graph and
    launched by one replay: the host then queues one launch, not one per pass
    (about 30 us each through Python, which would keep the wall clock above
    the kernels' time), and the HIP events bracket the replay (the per-launch
    time carries the replay's one launch latency, spread over the segment).
    Without it the events start once the first pass is queued and take the
    rest.  The wall clock takes every pass either way.  Returns (wall seconds,
    GPU milliseconds, the positions in `order` the events took, "graph" or
    "eager")."""
    seg_max = len(states)
    work = [(states[0][0].clone(), states[0][1].clone(), states[0][2].clone())
            for _ in range(min(seg_max, len(order)))]

    def refill(idx):
        for j, i in enumerate(idx):
            wk, wv, wr = work[j]
            wk.copy_(states[i][0])
            wv.copy_(states[i][1])
            wr.copy_(states[i][2])

    def passes(idx):
        for j, i in enumerate(idx):
            vd.vd_evict_step(work[j][0], work[j][1], states[i][3], w.budget, variant,
                             running_sum=work[j][2])

    graphs = {}

    def segment_graph(idx):  # (capturing runs nothing: the buffers stay as they are)
        key = tuple(idx)
        if key not in graphs:
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                passes(idx)
            graphs[key] = g
        return graphs[key]

    # The copies above leave up to a few hundred MB of dirty lines in L2 and
    # the MALL; a read of a buffer larger than both evicts them before each
    # timed segment, so that the passes do not pay for the copies' write-back.
    flush_buf = torch.zeros(1 << 28, dtype=torch.float32, device=dev)   # 1 GiB
    stream = torch.cuda.current_stream(dev)
    for i in range(warmup):
        st = states[order[i % len(order)]]
        refill([order[i % len(order)]])
        vd.vd_evict_step(work[0][0], work[0][1], st[3], w.budget, variant, running_sum=work[0][2])
    torch.cuda.synchronize()
    if graph:
        try:
            segment_graph(order[:len(work)])
        except RuntimeError as exc:  # no capture on this stack: time the calls one by one
            log(f"bench: no HIP graph ({exc}); eager launches")
            graph = False
    wall_s, gpu_ms, done, timed = 0.0, 0.0, 0, []
    while done < len(order):
        idx = order[done:done + len(work)]
        g = segment_graph(idx) if graph else None
        refill(idx)
        flush_buf.sum()
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        t0 = time.perf_counter()
        if graph:
            e0.record(stream)
            g.replay()
        else:
            for j, i in enumerate(idx):
                vd.vd_evict_step(work[j][0], work[j][1], states[i][3], w.budget, variant,
                                 running_sum=work[j][2])
                if j == 0:
                    e0.record(stream)
        e1.record(stream)
        torch.cuda.synchronize()
        wall_s += time.perf_counter() - t0
        if graph:
            gpu_ms += e0.elapsed_time(e1)
            timed += list(range(done, done + len(idx)))
        elif len(idx) > 1:
            gpu_ms += e0.elapsed_time(e1)
            timed += list(range(done + 1, done + len(idx)))
        done += len(idx)
    return wall_s, gpu_ms, timed, "graph" if graph else "eager"


def hold(stream):
    """Keeps the GPU busy for about 200 us while the host enqueues a single
    timed launch, so that the start event fires only once the launch is
    queued (events over one launch would otherwise include the host's
    latency to it)."""
    with torch.cuda.stream(stream):
        torch.cuda._sleep(480000)  # the spin counts about 2.4 cycles per ns


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


def stream_read_us(dev, nbytes, reps=8):
    """Time per read of the plain streaming read (vd_stream_read) of `nbytes`:
    the read ceiling at a kernel's own size, where ramp-up and drain weigh more
    than at 2 GiB.  `reps` distinct buffers (one, read again, above 512 MiB),
    pushed out of the caches by 256 MiB of writes, are read back to back; the
    events take all but the first read, so that no launch latency enters (as
    for the kernels' own per-launch times).  In microseconds."""
    n = max((nbytes + 15) // 16, 1) * 4  # whole 16-byte words
    # above 512 MiB one buffer, read again and again, outgrows the caches by itself
    nbuf = reps + 1 if nbytes <= (512 << 20) else 1
    bufs = [torch.ones(n, dtype=torch.float32, device=dev) for _ in range(nbuf)]
    sink = torch.zeros(1, dtype=torch.int32, device=dev)
    flush = torch.empty(256 << 20, dtype=torch.uint8, device=dev)
    flush.fill_(1)
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    vd.vd_stream_read(bufs[0], sink)
    e0.record()
    for i in range(reps):
        vd.vd_stream_read(bufs[(i + 1) % nbuf], sink)
    e1.record()
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) * 1e3 / reps
    del bufs, flush
    return us


def decode_state(w: synth.Workload, dev, variant="l2"):
    """A decode step of every sequence: N old tokens and one new token in the
    cache (n = N + 1), and the running sum of the N old rows of the scored
    tensor (V, or K for a key-side score)."""
    S, L, H, D = w.num_seqs, w.num_layers, w.num_kv_heads, w.head_dim
    k, v = synth.empty_cache(w, dev)
    rs = torch.zeros((w.units, D + 1), dtype=torch.float64, device=dev)
    scored = k if variant.startswith("key") else v
    for s in range(S):
        N = w.budget[s]
        k[s, :, :, :N + 1] = synth.block_rows(w, "k", s, 0, 0, N + 1, dev, seq_seed=s)
        v[s, :, :, :N + 1] = synth.block_rows(w, "v", s, 0, 0, N + 1, dev, seq_seed=s)
        us = slice(s * L * H, (s + 1) * L * H)
        rs[us, :D] = scored[s, :, :, :N].double().sum(dim=2).reshape(L * H, D)
        rs[us, D] = N
    return k, v, rs, [N + 1 for N in w.budget]


def time_in_place(w, k, v, rs, n, steps, warmup, variant, dev):
    """Decode passes replayed on one cache: after a pass the valid slots are
    [0, N) and slot N still holds a row, so the next call with n = N + 1 is
    again a well-formed decode step (its new token is that row).  Returns
    (wall seconds, GPU milliseconds) of `steps` back-to-back passes."""
    for _ in range(warmup):
        vd.vd_evict_step(k, v, n, w.budget, variant, running_sum=rs)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream(dev)
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record(stream)
    for _ in range(steps):
        vd.vd_evict_step(k, v, n, w.budget, variant, running_sum=rs)
    e1.record(stream)
    torch.cuda.synchronize()
    return time.perf_counter() - t0, e0.elapsed_time(e1)


def ragged_prefill(w, variant, steps, dev):
    """The ragged workload's lock-step prefill in place: at call b every
    sequence whose prompt is not exhausted appends its block b (the last one
    partial), then one pass runs over all 64 sequences.  Only the passes are
    timed (HIP events around each evicting call); the appends are not, nor is
    the count of moved rows (vd_score and vd_select_topn on the pre-pass
    cache, which give the pass's own kept sets).  Returns (seconds of the
    timed passes, passes, algorithmic bytes, scanned bytes, and the pre-pass
    state of one sequence that evicts at the first evicting call, with the
    one-sequence workload it belongs to)."""
    import dataclasses
    S, L, H, D, B = w.num_seqs, w.num_layers, w.num_kv_heads, w.head_dim, w.block
    k, v = synth.empty_cache(w, dev)
    rs = torch.zeros((w.units, D + 1), dtype=torch.float64, device=dev)
    sc = torch.empty((w.units, w.capacity), dtype=torch.float32, device=dev)
    keep = torch.empty((w.units, w.capacity), dtype=torch.uint8, device=dev)
    n = [0] * S
    stream = torch.cuda.current_stream(dev)
    total_ms, passes, alg, scan, first, head = 0.0, 0, 0, 0, None, 0
    nblocks = (max(w.prompt) + B - 1) // B
    for blk in range(nblocks):
        for s in range(S):
            t0 = blk * B
            t1 = min(t0 + B, w.prompt[s])
            if t1 > t0:
                k[s, :, :, n[s]:n[s] + t1 - t0] = synth.block_rows(w, "k", s, blk, t0, t1, dev)
                v[s, :, :, n[s]:n[s] + t1 - t0] = synth.block_rows(w, "v", s, blk, t0, t1, dev)
                n[s] += t1 - t0
        if not any(a > b for a, b in zip(n, w.budget)):
            vd.vd_evict_step(k, v, n, w.budget, variant, running_sum=rs)  # only the state moves
            continue
        vd.vd_score(v, n, variant, scores=sc, k=k)
        vd.vd_select_topn(v, sc, n, w.budget, keep_mask=keep)
        mv = movers_of(w, keep, n)
        if first is None:
            s1 = next(s for s in range(S) if n[s] > w.budget[s])
            w1 = dataclasses.replace(w, num_seqs=1, prompt=[w.prompt[s1]], budget=[w.budget[s1]])
            us = slice(s1 * L * H, (s1 + 1) * L * H)
            first = ((k[s1:s1 + 1].clone(), v[s1:s1 + 1].clone(), rs[us].clone(), [n[s1]],
                      [mv[s1]], f"first evicting prefill call ({blk}), sequence {s1}"), w1)
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        hold(stream)
        e0.record(stream)
        vd.vd_evict_step(k, v, n, w.budget, variant, running_sum=rs)
        e1.record(stream)
        torch.cuda.synchronize()
        total_ms += e0.elapsed_time(e1)
        passes += 1
        alg += algorithmic_bytes(w, n, mv)
        scan += scanned_bytes(w, n)
        head += L * H * sum(1 for a, b in zip(n, w.budget) if a > b)
        n = [min(a, b) for a, b in zip(n, w.budget)]
        if passes >= steps:
            break
    return total_ms / 1e3, passes, alg, scan, first, head


# ---------------------------------------------------------------- oracle baseline

def to_np(t):
    t = t.detach().contiguous().cpu()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


def _oracle_pass(orc, w, state, variant, take, nthreads):
    k, v, _, n, _, _ = state
    S, L, H, C, D = k.shape
    U = S * L * H
    scored_k = variant.startswith("key")
    kn = to_np(k.reshape(U, C, D)[:take])
    vn = to_np(v.reshape(U, C, D)[:take])
    nu = np.repeat(np.asarray(n, np.int32), L * H)[:take]
    Nu = np.repeat(np.asarray(w.budget, np.int32), L * H)[:take]
    return kn, vn, nu, Nu, scored_k


def cpu_baseline(w, state, variant, budget_s=10.0, max_units=None, single_s=3.0):
    """The oracle on the host cores: whole passes over one pre-pass state (or
    over its first `max_units` units, scaled to whole passes), with every core
    and with one; plus the oracle's scores and kept sets of the first pass,
    for the parity sample."""
    import oracle
    k = state[0]
    S, L, H, C, D = k.shape
    U = S * L * H
    take = U if max_units is None else min(U, max_units)
    threads = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
    orc = oracle.load()
    kn, vn, nu, Nu, _ = _oracle_pass(orc, w, state, variant, take, threads)
    elapsed, reps, ref = 0.0, 0, None
    while elapsed < budget_s or reps == 0:
        kc, vc = kn.copy(), vn.copy()
        t0 = time.perf_counter()
        out = orc.evict_step(kc, vc, nu, Nu, variant, nthreads=threads)
        elapsed += time.perf_counter() - t0
        if ref is None:
            ref = out
        reps += 1
    frac = take / U
    n = state[3]
    what = (f"{reps} whole passes of one {w.name} boundary ({U} units, n={max(n)})" if take == U
            else f"{reps} passes over {take} of the {U} units of one {w.name} step "
                 f"(n={max(n)}), scaled to whole passes")
    # one core, on a smaller sample of units
    one = max(1, min(take, int(math.ceil(take / max(threads, 1)))))
    e1, r1 = 0.0, 0
    while e1 < single_s or r1 == 0:
        kc, vc = kn[:one].copy(), vn[:one].copy()
        t0 = time.perf_counter()
        orc.evict_step(kc, vc, nu[:one], Nu[:one], variant, nthreads=1)
        e1 += time.perf_counter() - t0
        r1 += 1
    res = {"value": reps * frac / elapsed, "unit": "passes/s", "cores": threads,
           "kind": "oracle", "sample": f"{what} in {elapsed:.1f} s, {threads} threads",
           "gbps_scanned": reps * frac * scanned_bytes(w, n) / elapsed / 1e9,
           "single_core": {"value": r1 * (one / U) / e1, "unit": "passes/s", "cores": 1,
                           "sample": f"{r1} passes over {one} of the {U} units in {e1:.1f} s, "
                                     f"scaled to whole passes"},
           "cpu_model": cpu_model(), "os_cpu_count": os.cpu_count()}
    return res, ref, take


def cpu_model():
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def parity_sample(w, state, variant, ref, take, dev):
    """Compares the GPU's pass on a copy of `state` with the oracle's pass on
    the same bytes (the first `take` units): identical kept sets, near-ties
    (sets that differ only on slots whose oracle scores lie within the
    relative 1e-5 band of the N-th score) and anything else, and the largest
    relative score error.  Counts only; the tests assert."""
    k, v, rs, n = state[0].clone(), state[1].clone(), state[2].clone(), state[3]
    U, C = w.units, k.shape[3]
    sc = torch.zeros((U, C), device=dev)
    kp = torch.zeros((U, C), dtype=torch.uint8, device=dev)
    vd.vd_evict_step(k, v, n, w.budget, variant, running_sum=rs, scores_out=sc, keep_out=kp)
    torch.cuda.synchronize()
    s_gpu = sc[:take].cpu().numpy().astype(np.float64)
    k_gpu = kp[:take].cpu().numpy()
    s_ref, k_ref, _ = ref
    L, H = w.num_layers, w.num_kv_heads
    nu = np.repeat(np.asarray(n, np.int32), L * H)[:take]
    Nu = np.repeat(np.asarray(w.budget, np.int32), L * H)[:take]
    same = ties = other = 0
    err = 0.0
    smallest = variant == "key_norm"
    for u in range(take):
        m, N = int(nu[u]), int(Nu[u])
        if m == 0:
            continue
        a, b, r = k_gpu[u, :m].astype(bool), k_ref[u, :m].astype(bool), s_ref[u, :m]
        top = np.abs(r).max()
        ok = np.abs(r) > 0
        if ok.any():
            err = max(err, float((np.abs(s_gpu[u, :m] - r)[ok] / np.abs(r[ok])).max()))
        if np.array_equal(a, b):
            same += 1
            continue
        order = np.sort(-r if smallest else r)[::-1]
        s_N = abs(order[min(N, m) - 1])
        band = REL_TIE * s_N + 1e-6 * top
        d = np.flatnonzero(a != b)
        if a.sum() == min(N, m) and np.all(np.abs(np.abs(r[d]) - s_N) <= band):
            ties += 1
        else:
            other += 1
    return {"units": int(take), "identical": same, "near_ties": ties, "outside_band": other,
            "max_rel_score_err": err, "state": f"boundary {state[5]}"}


# ---------------------------------------------------------------- counters

def load_traffic(name: str, boundaries):
    """HBM traffic per launch, measured with rocprofv3 counters on this
    kernel source, averaged over the given boundaries; None when absent, taken
    on another kernel version or not covering every boundary."""
    path = os.path.join(TRAFFIC_DIR, f"traffic_{name}.json")
    if not os.path.exists(path):
        return None
    with open(path) as fh:
        t = json.load(fh)
    if t.get("kernel_hash") != kernel_hash():
        return None
    per = t.get("bytes_per_boundary")
    if per is None:
        return t.get("bytes_per_launch") if boundaries is None else None
    if boundaries is None:
        return statistics.mean(per.values())
    if not all(str(b) in per for b in boundaries):
        return None
    return statistics.mean(per[str(b)] for b in boundaries)


def _csv_rows(d, kind):
    fs = sorted(glob.glob(os.path.join(d, "**", f"*{kind}.csv"), recursive=True))
    if not fs:
        raise SystemExit(f"no *{kind}.csv under {d}")
    with open(fs[0]) as fh:
        return list(csv.DictReader(fh))


def _counter_by_dispatch(d, match):
    by = {}
    for r in _csv_rows(d, "counter_collection"):
        if match in r["Kernel_Name"]:
            i = int(r["Dispatch_Id"])
            by[i] = by.get(i, 0.0) + float(r["Counter_Value"])
    return [by[i] for i in sorted(by)]


def summarize_counters(args):
    """Writes profiles/traffic_<name>.json from four rocprofv3 --pmc runs
    (FETCH_SIZE and WRITE_SIZE of the bench, then of --copy-calibration),
    each a directory under --summarize-counters, named fetch, write, cfetch,
    cwrite; the bench's JSON line is in <dir>/bench.json.  Counter values
    are scaled by what the same counter reads for the 1 GiB copy."""
    d = args.summarize_counters
    bench_line = json.loads(open(os.path.join(d, "bench.json")).read().strip().splitlines()[-1])
    cal = {"bytes": 1 << 30}
    for key in ("fetch", "write"):
        vals = _counter_by_dispatch(os.path.join(d, "c" + key), "opy")[-3:]
        cal[f"{key}_kib_raw"] = round(statistics.mean(vals), 3)
        cal[f"{key}_scale"] = (1 << 30) / (statistics.mean(vals) * 1024)
    kernels = [k.strip() for k in args.kernels.split(",")]
    order = bench_line.get("boundaries")
    K = args.last
    out = {"workload": args.name, "kernels": kernels, "kernel_hash": kernel_hash(),
           "copy_calibration": cal}
    per_kernel = {}
    for kern in kernels:
        f = _counter_by_dispatch(os.path.join(d, "fetch"), kern)[-K:]
        wv = _counter_by_dispatch(os.path.join(d, "write"), kern)[-K:]
        if len(f) != K or len(wv) != K:
            raise SystemExit(f"{kern}: {len(f)} / {len(wv)} dispatches, expected {K}")
        per_kernel[kern] = [a * 1024 * cal["fetch_scale"] + b * 1024 * cal["write_scale"]
                            for a, b in zip(f, wv)]
        out[kern] = {"fetch_bytes_per_launch": int(statistics.mean(f) * 1024 * cal["fetch_scale"]),
                     "write_bytes_per_launch": int(statistics.mean(wv) * 1024 * cal["write_scale"])}
    launches = [sum(per_kernel[kk][i] for kk in kernels) for i in range(K)]
    out["bytes_per_launch"] = int(statistics.mean(launches))
    if order is not None and len(order) * (K // max(len(order), 1)) == K:
        reps = K // len(order)
        per = {}
        for i, b in enumerate(order * reps):
            per.setdefault(str(b), []).append(launches[i])
        out["bytes_per_boundary"] = {b: int(statistics.mean(x)) for b, x in per.items()}
        out["boundaries"] = sorted({int(b) for b in order})
    # the counters take every launch, the events all but the first of a segment
    alg = bench_line["roofline"].get("alg_bytes_per_launch_all", bench_line["roofline"]["alg_bytes_per_launch"])
    out["alg_bytes_per_launch"] = alg
    out["traffic_over_alg"] = round(out["bytes_per_launch"] / alg, 4)
    out["dispatches_averaged"] = f"last {K} of each kernel: the timed launches"
    out["commands"] = args.commands.split(";;") if args.commands else []
    out["note"] = ("FETCH_SIZE / WRITE_SIZE count L2-to-fabric traffic (MALL hits included), "
                   "scaled by a plain 1 GiB copy measured the same way.")
    path = os.path.join(TRAFFIC_DIR, f"traffic_{args.name}.json")
    with open(path, "w") as fh:
        json.dump(out, fh, indent=1)
    print(json.dumps({"wrote": path, "bytes_per_launch": out["bytes_per_launch"],
                      "traffic_over_alg": out["traffic_over_alg"]}))


def summarize_sq(args):
    """Prints, per kernel of --kernels, the mean per dispatch of every counter
    of one rocprofv3 --pmc run (the directory under --summarize-sq) over its
    last --last dispatches, as a markdown table."""
    d = args.summarize_sq
    rows = _csv_rows(d, "counter_collection")
    lines = ["| kernel | counter | mean per dispatch |", "|---|---|---|"]
    for kern in [k.strip() for k in args.kernels.split(",")]:
        by = {}
        for r in rows:
            if kern in r["Kernel_Name"]:
                by.setdefault(r["Counter_Name"], {}).setdefault(int(r["Dispatch_Id"]), 0.0)
                by[r["Counter_Name"]][int(r["Dispatch_Id"])] += float(r["Counter_Value"])
        for name in sorted(by):
            vals = [by[name][i] for i in sorted(by[name])][-args.last:]
            lines.append(f"| `{kern}` | {name} | {statistics.mean(vals):.6g} |")
    print("\n".join(lines))


def summarize_traces(args):
    """Prints a markdown summary of one rocprofv3 --kernel-trace --stats run
    (the directory under --summarize-traces, with the bench's JSON line in
    <dir>/bench.json): per kernel of --kernels, the duration, gap and period
    of its last --last dispatches, then the run's top kernels."""
    d = args.summarize_traces
    tr = sorted(_csv_rows(d, "kernel_trace"), key=lambda r: int(r["Start_Timestamp"]))
    lines = []
    for kern in [k.strip() for k in args.kernels.split(",")]:
        idx = [i for i, r in enumerate(tr) if kern in r["Kernel_Name"]][-args.last:]
        dur, gap, per = [], [], []
        for i in idx:
            s, e = int(tr[i]["Start_Timestamp"]), int(tr[i]["End_Timestamp"])
            dur.append((e - s) / 1e3)
            if i + 1 < len(tr):
                ns = int(tr[i + 1]["Start_Timestamp"])
                gap.append((ns - e) / 1e3)
                per.append((ns - s) / 1e3)
        lines += [f"## `{kern}`: the last {len(idx)} launches", "",
                  "| quantity | mean | median | min | max |", "|---|---|---|---|---|"]
        for nm, xs in (("kernel duration (us)", dur), ("gap to the next dispatch (us)", gap),
                       ("dispatch period (us)", per)):
            if xs:
                lines.append(f"| {nm} | {statistics.mean(xs):.2f} | {statistics.median(xs):.2f} | "
                             f"{min(xs):.2f} | {max(xs):.2f} |")
        lines.append("")
    st = sorted(_csv_rows(d, "kernel_stats"), key=lambda r: -float(r["TotalDurationNs"]))[:8]
    lines += ["## All kernels of the run (setup included)", "",
              "| kernel | calls | avg us | min us | max us | % time |", "|---|---|---|---|---|---|"]
    for r in st:
        nm = r["Name"] if len(r["Name"]) <= 80 else r["Name"][:77] + "..."
        lines.append(f"| `{nm}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} | "
                     f"{float(r['MinNs']) / 1e3:.2f} | {float(r['MaxNs']) / 1e3:.2f} | "
                     f"{float(r['Percentage']):.1f} |")
    print("\n".join(lines))


# ---------------------------------------------------------------- other modes

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
    # the column sums of K and V over all rows, the state a caller keeps (the
    # pass keeps V's as its running sum): with them the centroids are known
    # and one read of K and V gives every distance
    D = w.head_dim
    sums = []
    for x in (k, v):
        t = torch.zeros((w.units, D + 1), dtype=torch.float64, device=dev)
        t[:, :D] = x.reshape(w.units, C, D).double().sum(dim=1)
        t[:, D] = C
        sums.append(t)
    stream = torch.cuda.current_stream(dev)

    def timed(with_sums):
        kw = dict(k_sum=sums[0], v_sum=sums[1]) if with_sums else {}
        for _ in range(args.warmup):
            vd.vd_geometry(k, v, n, out, **kw)
        torch.cuda.synchronize()
        gpu_ms, wall_s, done, timed = 0.0, 0.0, 0, 0
        while done < args.steps:   # segments of at most 20 passes, each after a flush
            seg = min(20, args.steps - done)
            flush_buf.sum()
            torch.cuda.synchronize()
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            t0 = time.perf_counter()
            for i in range(seg):
                vd.vd_geometry(k, v, n, out, **kw)
                if i == 0:
                    e0.record(stream)  # (the events take the launches after the first)
            e1.record(stream)
            torch.cuda.synchronize()
            wall_s += time.perf_counter() - t0
            if seg > 1:
                gpu_ms += e0.elapsed_time(e1)
                timed += seg - 1
            done += seg
        return gpu_ms / max(timed, 1), wall_s

    ms2, _ = timed(False)   # per launch
    ms1, wall_s = timed(True)
    alg = 2 * w.units * C * w.row_bytes + 2 * w.units * (D + 1) * 8
    traffic = load_traffic(f"geometry_{w.name}", None)
    us = ms1 * 1e3
    alg_gbps = alg / (us * 1e-6) / 1e9
    log(f"bench: geometry {us:.2f} us per launch with the sums ({alg_gbps:.0f} GB/s algorithmic), "
        f"{ms2 * 1e3:.2f} us without")
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
                   "head_dim": w.head_dim, "n": C, "column_sums_given": True},
        "roofline": {"bound": "hbm", "achieved": round(alg_gbps, 1), "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s", "frac": round(alg_gbps / HBM_PEAK_GBPS, 4),
                     "traffic": None if traffic is None else int(traffic),
                     "traffic_over_alg": None if traffic is None else round(traffic / alg, 3),
                     "kernel": f"geometry_kernel<bf16,{w.head_dim}>",
                     "launch_us": round(us, 2), "alg_bytes_per_launch": alg},
        "without_sums_launch_us": round(ms2 * 1e3, 2),
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
    variant = args.variant if args.variant in ("l2", "fastcaote") else "l2"
    log(f"bench: building the {w.name} decode cache ({w.units} units)")
    k, v, rs, n = decode_state(w, dev)
    rs_l = [rs.view(S, L, H, D + 1)[:, l].reshape(S * H, D + 1).contiguous() for l in range(L)]
    g = torch.Generator(device=dev)
    g.manual_seed(1234)
    q_l = [torch.randn((S, 1, Hq, D), generator=g, device=dev) for _ in range(L)]
    out = torch.empty((S, 1, Hq, D), dtype=torch.float32, device=dev)
    kv_l = [(k[:, l:l + 1], v[:, l:l + 1]) for l in range(L)]
    ws = torch.zeros(vd.vd_decode_attention_workspace_size(kv_l[0][0], kv_l[0][1], Hq, variant),
                     dtype=torch.uint8, device=dev)
    # moved rows of one call (untimed, on copies)
    pos = torch.arange(w.capacity, dtype=torch.int32, device=dev).repeat(S * H, 1).contiguous()
    vd.vd_decode_attention_evict(kv_l[0][0].clone(), kv_l[0][1].clone(), q_l[0], n, w.budget,
                                 rs_l[0].clone(), pos=pos, out=out, workspace=ws, variant=variant)
    movers = int((pos[:, :N] != torch.arange(N, dtype=torch.int32, device=dev)).any(dim=1).sum())

    def step():
        for l in range(L):
            vd.vd_decode_attention_evict(kv_l[l][0], kv_l[l][1], q_l[l], n, w.budget, rs_l[l],
                                         out=out, workspace=ws, variant=variant)

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
    traffic = load_traffic(f"decode_attention_{variant}_decode_b16", None)
    log(f"bench: {us_call:.2f} us per layer call, {gbps:.0f} GB/s algorithmic, {movers} movers of {units}")
    # the eviction pass alone over all layers (vd_evict_step), for context
    _, ev_ms = time_in_place(w, k, v, rs, n, 10, 2, "l2", dev)
    same_us = stream_read_us(dev, alg)
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
                   "n": N + 1, "variant": variant},
        "roofline": {"bound": "hbm", "achieved": round(gbps, 1), "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s", "frac": round(gbps / HBM_PEAK_GBPS, 4),
                     "traffic": None if traffic is None else int(traffic),
                     "traffic_over_alg": None if traffic is None else round(traffic / alg, 3),
                     "kernel": "attn_split_kernel<bf16,128,4> + attn_combine_kernel (one call)",
                     "launch_us": round(us_call, 2), "alg_bytes_per_launch": alg},
        "evict_pass_alone_us": round(ev_ms * 1e3 / 10, 2),
        "stream_read_same_bytes_us": round(same_us, 2),
        "call_over_stream_read_same_bytes": round(us_call / same_us, 3),
    }
    if not args.no_cpu_baseline:
        log("bench: timing the oracle on the host ...")
        res["cpu_baseline"] = cpu_decode_attention(w, kv_l[0][0], kv_l[0][1], q_l[0], rs_l[0],
                                                   n, args.cpu_seconds)
    return res


def _oracle_rate(fn, count, budget_s, threads):
    """Calls fn(i) for i = 0, 1, ... (cycling over count) on `threads` host
    threads (ctypes releases the GIL inside the oracle's C) for about budget_s
    seconds, `threads` calls at a time; returns (calls, seconds)."""
    from concurrent.futures import ThreadPoolExecutor
    t0, done = time.perf_counter(), 0
    with ThreadPoolExecutor(max_workers=threads) as ex:
        while done == 0 or time.perf_counter() - t0 < budget_s:
            list(ex.map(fn, [(done + i) % count for i in range(threads)]))
            done += threads
    return done, time.perf_counter() - t0


def cpu_decode_attention(w, k, v, q, rs, n, budget_s, single_s=3.0):
    """The oracle's attention (every query head) and eviction for units of one
    layer, one unit per call, with every core and with one, scaled to whole
    steps (all layers) per second."""
    import oracle
    orc = oracle.load()
    S, H, D, C = w.num_seqs, w.num_kv_heads, w.head_dim, w.capacity
    G = w.num_q_heads // H
    kn = to_np(k).reshape(S * H, C, D)
    vn = to_np(v).reshape(S * H, C, D)
    qn = q.cpu().numpy().astype(np.float64).reshape(S * H, G, D)
    m = n[0]
    threads = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))

    def unit(i):
        for g in range(G):
            orc.attention(qn[i, g], kn[i, :m], vn[i, :m], D ** -0.5)
        kc, vc = kn[i:i + 1].copy(), vn[i:i + 1].copy()
        orc.evict_step(kc, vc, np.array([m], np.int32), np.array([w.budget[0]], np.int32), "l2", nthreads=1)

    d1, e1 = _oracle_rate(unit, S * H, single_s, 1)
    dn, en = _oracle_rate(unit, S * H, budget_s, threads)
    what = f"attention of {G} heads and eviction, n={m}"
    return {"value": round(dn / en / w.units, 4), "unit": "steps/s", "cores": threads,
            "kind": "oracle",
            "sample": f"{dn} unit calls of one layer ({what}) in {en:.1f} s on {threads} threads, "
                      f"scaled to a step of {w.units} units",
            "single_core": {"value": round(d1 / e1 / w.units, 4), "unit": "steps/s", "cores": 1,
                            "sample": f"{d1} unit calls in {e1:.1f} s, scaled to a step"},
            "cpu_model": cpu_model(), "os_cpu_count": os.cpu_count()}


def cpu_geometry(w, k, v, budget_s, single_s=3.0):
    """The oracle's geometry of the units of sequence 0, one unit per call,
    with every core and with one, scaled to passes over every unit per second."""
    import oracle
    orc = oracle.load()
    ku = to_np(k[0]).reshape(-1, w.capacity, w.head_dim)
    vu = to_np(v[0]).reshape(-1, w.capacity, w.head_dim)
    threads = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))

    def unit(i):
        orc.geometry(ku[i], vu[i])

    d1, e1 = _oracle_rate(unit, ku.shape[0], single_s, 1)
    dn, en = _oracle_rate(unit, ku.shape[0], budget_s, threads)
    return {"value": round(dn / en / w.units, 4), "unit": "passes/s", "cores": threads,
            "kind": "oracle",
            "sample": f"{dn} unit calls ({w.capacity} rows of K and V each) in {en:.1f} s on "
                      f"{threads} threads, scaled to passes over all {w.units} units",
            "single_core": {"value": round(d1 / e1 / w.units, 4), "unit": "passes/s", "cores": 1,
                            "sample": f"{d1} unit calls in {e1:.1f} s, scaled to whole passes"},
            "cpu_model": cpu_model(), "os_cpu_count": os.cpu_count()}


# ---------------------------------------------------------------- main

def pass_bench(w, args, dev):
    variant = args.variant
    decode = args.workload in ("decode_b16", "ragged_serving") and args.phase != "prefill"
    order = None
    base_w = w
    if decode:
        log(f"bench: building the {w.name} decode cache ({w.units} units) ...")
        k, v, rs, n = decode_state(w, dev, variant)
        keep = torch.zeros((w.units, w.capacity), dtype=torch.uint8, device=dev)
        vd.vd_evict_step(k.clone(), v.clone(), n, w.budget, variant, running_sum=rs.clone(),
                         keep_out=keep)
        movers = movers_of(w, keep, n)
        del keep
        log(f"bench: timing {args.steps} decode passes in place")
        total_s, gpu_ms = time_in_place(w, k, v, rs, n, args.steps, args.warmup, variant, dev)
        timed, launch = list(range(args.steps)), "eager"

        alg = [algorithmic_bytes(w, n, movers)] * args.steps
        scan = [scanned_bytes(w, n)] * args.steps
        base_state = (k, v, rs, n, movers, "decode step")
        steps = args.steps
        head_passes = steps * w.units
    elif args.phase == "prefill" and w.name == "ragged_serving":
        log(f"bench: the {w.name} lock-step prefill in place (at most {args.steps} passes)")
        total_s, steps, a, sc, (base_state, base_w), head = ragged_prefill(w, variant, args.steps,
                                                                           dev)
        gpu_ms = total_s * 1e3
        timed, launch = list(range(steps)), "eager"
        alg, scan = [a / steps] * steps, [sc / steps] * steps
        head_passes = head
    else:
        every = ALL_BOUNDARIES.get(w.name, 1)
        log(f"bench: building the pre-pass states of {w.name} (every {every}. boundary) ...")
        t0 = time.perf_counter()
        states = prefill_states(w, variant, dev, every)
        order = spread(len(states), args.steps)
        log(f"bench: {len(states)} states ready in {time.perf_counter() - t0:.1f} s; "
            f"timing {args.steps} passes")
        small = np.mean([algorithmic_bytes(w, states[i][3], states[i][4]) for i in order]) < 16e6
        graph = args.launch == "graph" or (args.launch == "auto" and small)
        total_s, gpu_ms, timed, launch = time_pool(w, states, order, args.warmup, variant, dev,
                                                   graph=graph)
        alg = [algorithmic_bytes(w, states[i][3], states[i][4]) for i in order]
        scan = [scanned_bytes(w, states[i][3]) for i in order]
        base_state = states[0]
        steps = args.steps
        head_passes = sum(w.num_layers * w.num_kv_heads
                          for i in order for s_ in range(w.num_seqs)
                          if states[i][3][s_] > w.budget[s_])
        order = [states[i][5] for i in order]
    ms_launch = gpu_ms / len(timed)   # the launches the events took
    passes_per_s = steps / total_s
    kernel_s = gpu_ms / 1e3
    alg_gbps = sum(alg[i] for i in timed) / kernel_s / 1e9
    scan_gbps = sum(scan[i] for i in timed) / kernel_s / 1e9
    log(f"bench: {passes_per_s:.1f} passes/s wall, {ms_launch * 1e3:.2f} us per launch (HIP events)")
    tname = w.name + ("" if variant == "l2" else f"_{variant}") + (
        "_prefill" if args.phase == "prefill" and w.name == "ragged_serving" else "")
    traffic = load_traffic(tname, order)
    stream_gbps = stream_read_gbps(dev)
    alg_launch = sum(alg[i] for i in timed) / len(timed)
    same_us = stream_read_us(dev, int(alg_launch))
    out = {
        "metric": METRIC,
        "value": round(passes_per_s, 2),
        "unit": "passes/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": args.warmup,
        "ms_per_step": round(total_s / steps * 1e3, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if w.dtype == torch.bfloat16 else "f32",
        "data": "synthetic (seeded generator; no model weights or datasets)",
        "config": {"workload": w.name + (" (lock-step prefill)" if args.phase == "prefill" and
                                         w.name == "ragged_serving" else
                                         " (decode steps)" if decode else ""),
                   "seqs": w.num_seqs, "layers": w.num_layers,
                   "kv_heads": w.num_kv_heads, "q_heads": w.num_q_heads,
                   "head_dim": w.head_dim,
                   "budget": (w.budget[0] if len(set(w.budget)) == 1
                              else [min(w.budget), max(w.budget)]),
                   "block": w.block,
                   "prompt": max(w.prompt), "n": max(base_state[3]), "variant": variant,
                   "running_sum": True, "parallelism": "single GPU"},
        "boundaries": order,
        "launch": launch,
        "head_passes_per_s": round(head_passes / total_s, 1),
        "kv_gbps_scanned": round(scan_gbps, 1),
        "kv_scan_frac_of_hbm_peak": round(scan_gbps / HBM_PEAK_GBPS, 4),
        "stream_read_gbps": round(stream_gbps, 1),
        "alg_frac_of_stream_read": round(alg_gbps / stream_gbps, 4),
        "stream_read_same_bytes_us": round(same_us, 2),
        "launch_over_stream_read_same_bytes": round(ms_launch * 1e3 / same_us, 3),
        "roofline": {"bound": "hbm", "achieved": round(alg_gbps, 1), "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s", "frac": round(alg_gbps / HBM_PEAK_GBPS, 4),
                     "traffic": None if traffic is None else int(traffic),
                     "traffic_over_alg": (None if traffic is None else
                                          round(traffic / (sum(alg) / len(alg)), 3)),
                     "kernel": f"step_kernel<{'bf16' if w.dtype == torch.bfloat16 else 'f32'},"
                               f"{w.head_dim},{variant}>",
                     "launch_us": round(ms_launch * 1e3, 2),
                     "alg_bytes_per_launch": int(np.mean([alg[i] for i in timed])),
                     "alg_bytes_per_launch_all": int(np.mean(alg))},
    }
    if not args.no_cpu_baseline and base_state is not None:
        log("bench: timing the oracle on the host ...")
        max_units = 64 if decode or w.name == "ragged_serving" else None
        cb, ref, take = cpu_baseline(base_w, base_state, variant, args.cpu_seconds, max_units)
        out["cpu_baseline"] = cb
        out["parity_sample"] = parity_sample(base_w, base_state, variant, ref, take, dev)
    return out


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=60)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="llama3_8b_prefill",
                    choices=["tiny", "llama3_8b_prefill", "wide_head_d256", "decode_b16",
                             "ragged_serving"],
                    help="decode_b16 and ragged_serving time decode steps (n = N + 1) unless "
                         "--phase prefill")
    ap.add_argument("--phase", default=None, choices=["prefill", "decode"],
                    help="ragged_serving: the lock-step prefill calls or the decode steps")
    ap.add_argument("--variant", default="l2", choices=sorted(vd.VARIANTS))
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--launch", default="auto", choices=["auto", "graph", "eager"],
                    help="how the timed passes are launched: from a captured HIP graph, one by one, "
                         "or (auto) from a graph only where a pass moves under 16 MB (launch-bound)")
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
    ap.add_argument("--summarize-traces", metavar="DIR")
    ap.add_argument("--summarize-counters", metavar="DIR")
    ap.add_argument("--summarize-sq", metavar="DIR")
    ap.add_argument("--kernels", default="step_kernel<",
                    help="kernel name substrings for the summaries, comma separated")
    ap.add_argument("--last", type=int, default=60, help="dispatches the summaries average")
    ap.add_argument("--name", default="llama3_8b_prefill", help="traffic file name")
    ap.add_argument("--commands", default="", help="';;'-separated commands, recorded")
    args = ap.parse_args()
    if args.summarize_traces:
        summarize_traces(args)
        return
    if args.summarize_counters:
        summarize_counters(args)
        return
    if args.summarize_sq:
        summarize_sq(args)
        return
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
    if args.variant == "fastcaote":
        print("fastcaote is a score of the fused decode step: use --decode-attention",
              file=sys.stderr)
        sys.exit(2)
    print(json.dumps(pass_bench(w, args, dev)), flush=True)


if __name__ == "__main__":
    main()
