"""GPU parity on the five workloads at their full sizes, with the library
called as the benchmark calls it (running sum on, one launch per pass).

Inputs come from ``synth`` only; the oracle never sees a byte the HIP path
produced.  Where several passes run in a row (tiny trajectory, the llama
prefill boundaries), the oracle runs its own trajectory and the GPU is fed
the oracle's state before each pass ("oracle-forced"), so one benign
near-tie swap cannot make the two trajectories drift apart.  The large
workloads compare every unit (llama prefill) or a fixed sample of units
(decode, wide, ragged) that the oracle computes one by one.
"""
import numpy as np
import pytest
import torch

from paper_2609_23314_amd import synth, vd
from paper_2609_23314_amd.driver import EvictingCache
from parity import Report, compare_pass, from_np, per_unit, to_np, units

pytestmark = pytest.mark.gpu
DEV = "cuda"


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    vd.load()


def gpu_state(v5, count_per_seq, D):
    """Running-sum state of rows [0, count) of every unit, summed in fp64 on the
    GPU by torch (an input of the HIP path; exact for bf16 values)."""
    S, L, H, C, _ = v5.shape
    st = torch.zeros((S, L, H, D + 1), dtype=torch.float64, device=DEV)
    for s in range(S):
        c = int(count_per_seq[s])
        st[s, :, :, :D] = v5[s, :, :, :c].double().sum(dim=2)
        st[s, :, :, D] = c
    return st.reshape(S * L * H, D + 1).contiguous()


def sample_units(S, L, H, count, seed):
    rng = np.random.default_rng(seed)
    U = S * L * H
    ids = np.unique(np.concatenate([[0, U - 1], rng.choice(U, size=min(count, U), replace=False)]))
    return ids


def unit_rows(x5, ids, upto):
    """Oracle-form [len(ids), upto, D] copy of the given units' first rows."""
    S, L, H, C, D = x5.shape
    flat = x5.reshape(S * L * H, C, D)
    return to_np(flat[torch.as_tensor(ids, device=DEV), :upto])


# ------------------------------------------------------------------ tiny

def test_tiny_trajectory_matches_oracle_end_to_end(orc):
    """Tiny workload, free-running on both sides: 16 prefill blocks (12 evict)
    and 32 decode steps; every pass's kept set, scores and cache must agree."""
    w = synth.tiny()
    K, V = synth.tiny_rows()
    C = w.capacity
    cache = EvictingCache(1, 1, 1, 64, C, w.budget, dtype=torch.float32, device=DEV)
    ok, ov = np.zeros((1, C, 64), np.float32), np.zeros((1, C, 64), np.float32)
    opos = np.full((1, C), -1, np.int32)
    n_o = 0
    plan = [(16 * i, 16 * i + 16) for i in range(16)] + [(256 + t, 257 + t) for t in range(32)]
    evicting = 0
    for t0, t1 in plan:
        b = t1 - t0
        cache.append(0, torch.from_numpy(K[t0:t1]).view(1, 1, b, 64).to(DEV),
                     torch.from_numpy(V[t0:t1]).view(1, 1, b, 64).to(DEV))
        ok[0, n_o:n_o + b], ov[0, n_o:n_o + b] = K[t0:t1], V[t0:t1]
        opos[0, n_o:n_o + b] = np.arange(t0, t1)
        n_o += b
        sc = torch.zeros((1, C), device=DEV)
        kp = torch.zeros((1, C), dtype=torch.uint8, device=DEV)
        n_before = cache.n[0]
        cache.evict(scores_out=sc, keep_out=kp)
        torch.cuda.synchronize()
        rs, rk, _ = orc.evict_step(ok, ov, [n_o], [64], "l2", pos=opos)
        evicting += n_o > 64
        m = min(n_o, 64)
        assert n_before == n_o
        assert np.array_equal(to_np(kp)[0, :n_o], rk[0, :n_o]), f"kept set at token {t1}"
        assert np.allclose(to_np(sc)[0, :n_o], rs[0, :n_o], rtol=1e-5, atol=1e-6 * rs.max())
        assert np.array_equal(to_np(cache.v)[0, 0, 0, :m], ov[0, :m]), f"V at token {t1}"
        assert np.array_equal(to_np(cache.k)[0, 0, 0, :m], ok[0, :m]), f"K at token {t1}"
        assert np.array_equal(to_np(cache.pos)[0, :m], opos[0, :m]), f"pos at token {t1}"
        st = to_np(cache.running_sum)[0]
        assert st[64] == m and np.allclose(st[:64], ov[0, :m].astype(np.float64).sum(0),
                                           rtol=1e-12, atol=1e-12)
        n_o = m
    assert evicting == 12 + 32


# ------------------------------------------------------------------ llama prefill

def llama_boundary(w, seq_rows_old, n_old, block_idx):
    """Pre-pass cache at a block boundary: n_old old rows plus block `block_idx`."""
    B, D = w.block, w.head_dim
    k5, v5 = synth.empty_cache(w, DEV)
    k5[0, :, :, :n_old] = seq_rows_old[0]
    v5[0, :, :, :n_old] = seq_rows_old[1]
    t0 = block_idx * B
    k5[0, :, :, n_old:n_old + B] = synth.block_rows(w, "k", 0, block_idx, t0, t0 + B, DEV)
    v5[0, :, :, n_old:n_old + B] = synth.block_rows(w, "v", 0, block_idx, t0, t0 + B, DEV)
    return k5, v5


def test_llama_prefill_boundary_all_units(orc, parity_log):
    """One boundary of the Llama-3-8B-shaped prefill (256 units, n = 2560),
    every unit compared; the launch the benchmark times (no optional outputs)
    leaves bit-identical caches and state."""
    w = synth.llama_prefill()
    N, B, D = w.budget[0], w.block, w.head_dim
    old = (torch.cat([synth.block_rows(w, "k", 0, i, i * B, i * B + B, DEV) for i in range(4)], 2),
           torch.cat([synth.block_rows(w, "v", 0, i, i * B, i * B + B, DEV) for i in range(4)], 2))
    k5, v5 = llama_boundary(w, old, N, 4)
    U, C = w.units, w.capacity
    n = N + B
    k_b, v_b = k5.clone(), v5.clone()
    rs = gpu_state(v5, [N], D)
    rs_b = rs.clone()
    pre_k, pre_v = units(to_np(k5)), units(to_np(v5))
    sc = torch.zeros((U, C), device=DEV)
    kp = torch.zeros((U, C), dtype=torch.uint8, device=DEV)
    vd.vd_evict_step(k5, v5, [n], [N], "l2", running_sum=rs, scores_out=sc, keep_out=kp)
    vd.vd_evict_step(k_b, v_b, [n], [N], "l2", running_sum=rs_b)   # benchmark launch
    torch.cuda.synchronize()
    rep = compare_pass(orc, pre_k, pre_v, units(to_np(k5)), units(to_np(v5)),
                       np.full(U, n, np.int32), np.full(U, N, np.int32), "l2", w.dtype,
                       scores_gpu=to_np(sc), keep_gpu=to_np(kp), state=to_np(rs))
    parity_log("llama3_8b_prefill boundary 0, all 256 units (l2)", rep)
    assert rep.near_ties <= max(2, U // 100), rep
    assert torch.equal(k5.view(torch.int16), k_b.view(torch.int16))
    assert torch.equal(v5.view(torch.int16), v_b.view(torch.int16))
    assert torch.equal(rs, rs_b)


def test_llama_prefill_oracle_forced_boundaries(orc, parity_log):
    """The first three evicting boundaries of the prompt, oracle-forced, with
    the three value-side and the three key-side scores."""
    w = synth.llama_prefill()
    N, B, D = w.budget[0], w.block, w.head_dim
    U, C = w.units, w.capacity
    for variant in ("l2", "dir", "norm", "key_l2", "key_dir", "key_norm"):
        ok = np.zeros((U, C, D), np.uint16)
        ov = np.zeros((U, C, D), np.uint16)
        n_o = 0
        rep = Report()
        for blk in range(7):
            t0 = blk * B
            ok[:, n_o:n_o + B] = to_np(synth.block_rows(w, "k", 0, blk, t0, t0 + B, DEV)
                                       .reshape(U, B, D))
            ov[:, n_o:n_o + B] = to_np(synth.block_rows(w, "v", 0, blk, t0, t0 + B, DEV)
                                       .reshape(U, B, D))
            n = n_o + B
            if n > N:
                k5 = from_np(ok, w.dtype, DEV).view(1, 32, 8, C, D)
                v5 = from_np(ov, w.dtype, DEV).view(1, 32, 8, C, D)
                rs = gpu_state(k5 if variant.startswith("key") else v5, [n_o], D)
                sc = torch.zeros((U, C), device=DEV)
                kp = torch.zeros((U, C), dtype=torch.uint8, device=DEV)
                vd.vd_evict_step(k5, v5, [n], [N], variant, running_sum=rs, scores_out=sc,
                                 keep_out=kp)
                torch.cuda.synchronize()
                compare_pass(orc, ok, ov, units(to_np(k5)), units(to_np(v5)),
                             np.full(U, n, np.int32), np.full(U, N, np.int32), variant, w.dtype,
                             scores_gpu=to_np(sc), keep_gpu=to_np(kp), state=to_np(rs),
                             report=rep)
            orc.evict_step(ok, ov, np.full(U, n, np.int32), np.full(U, N, np.int32), variant)
            n_o = min(n, N)
        parity_log(f"llama3_8b_prefill boundaries 0-2, all 256 units ({variant})", rep)
        assert rep.units == 3 * U and rep.near_ties <= max(2, rep.units // 100), rep


def test_llama_prefill_whole_prompt_state_stays_exact():
    """The whole 32768-token prompt run free on the GPU (64 blocks, 60
    evicting passes, the running sum carried from pass to pass): after every
    pass the state equals the fp64 sum of the rows left in [0, N) and counts
    N, and every pass keeps exactly N rows.  A property of any correct pass,
    so it needs no oracle trajectory and holds at the full size."""
    w = synth.llama_prefill()
    N, B, D = w.budget[0], w.block, w.head_dim
    U, C = w.units, w.capacity
    k, v = synth.empty_cache(w, DEV)
    rs = torch.zeros((U, D + 1), dtype=torch.float64, device=DEV)
    keep = torch.zeros((U, C), dtype=torch.uint8, device=DEV)
    n_o, passes = 0, 0
    for blk in range(w.prompt[0] // B):
        t0 = blk * B
        k[0, :, :, n_o:n_o + B] = synth.block_rows(w, "k", 0, blk, t0, t0 + B, DEV)
        v[0, :, :, n_o:n_o + B] = synth.block_rows(w, "v", 0, blk, t0, t0 + B, DEV)
        n = n_o + B
        vd.vd_evict_step(k, v, [n], [N], "l2", running_sum=rs, keep_out=keep)
        n_o = min(n, N)
        if n > N:
            passes += 1
            assert int(keep[:, :n].sum().item()) == U * N, f"block {blk}"
        want = v[0, :, :, :n_o].double().sum(dim=2).reshape(U, D)
        got = rs[:, :D]
        scale = v[0, :, :, :n_o].double().abs().sum(dim=2).reshape(U, D).clamp_min(1.0)
        err = ((got - want).abs() / scale).max().item()
        assert err < 1e-12, f"block {blk}: state off by {err:.3g} (relative to the sum of |v|)"
        assert torch.all(rs[:, D] == n_o), f"block {blk}: count"
    assert passes == 60


# ------------------------------------------------------------------ decode

def test_decode_step_sampled_units(orc, parity_log):
    """Decode workload: 16 sequences x 256 units with a full cache of 4096
    tokens plus one new token (argmin path); 96 units checked."""
    w = synth.decode()
    N, D = w.budget[0], w.head_dim
    S, L, H = w.num_seqs, w.num_layers, w.num_kv_heads
    k5, v5 = synth.empty_cache(w, DEV)
    for s in range(S):
        k5[s, :, :, :N + 1] = synth.block_rows(w, "k", s, 0, 0, N + 1, DEV, seq_seed=s)
        v5[s, :, :, :N + 1] = synth.block_rows(w, "v", s, 0, 0, N + 1, DEV, seq_seed=s)
    ids = sample_units(S, L, H, 96, seed=3)
    pre_k, pre_v = unit_rows(k5, ids, N + 1), unit_rows(v5, ids, N + 1)
    rs = gpu_state(v5, [N] * S, D)
    U, C = w.units, w.capacity
    kp = torch.zeros((U, C), dtype=torch.uint8, device=DEV)
    sc = torch.zeros((U, C), device=DEV)
    vd.vd_evict_step(k5, v5, [N + 1] * S, [N] * S, "l2", running_sum=rs, keep_out=kp,
                     scores_out=sc)
    torch.cuda.synchronize()
    idx = torch.as_tensor(ids, device=DEV)
    rep = compare_pass(orc, pre_k, pre_v, unit_rows(k5, ids, N + 1), unit_rows(v5, ids, N + 1),
                       np.full(len(ids), N + 1, np.int32), np.full(len(ids), N, np.int32), "l2",
                       w.dtype, scores_gpu=to_np(sc[idx]), keep_gpu=to_np(kp[idx]),
                       state=to_np(rs[idx]), unit_ids=ids)
    parity_log(f"decode_b16 step 0, {len(ids)} sampled units (l2)", rep)
    assert to_np(kp.sum(dim=1)).tolist() == [N] * U


# ------------------------------------------------------------------ wide

def test_wide_head_boundary_sampled_units(orc, parity_log):
    """Wide-head workload (d = 256, Student-t values): 416 units at n = 5120;
    48 units checked."""
    w = synth.wide()
    N, B, D = w.budget[0], w.block, w.head_dim
    S, L, H = w.num_seqs, w.num_layers, w.num_kv_heads
    k5, v5 = synth.empty_cache(w, DEV)
    for s in range(S):
        for i in range(5):
            k5[s, :, :, i * B:(i + 1) * B] = synth.block_rows(w, "k", s, i, i * B, (i + 1) * B, DEV)
            v5[s, :, :, i * B:(i + 1) * B] = synth.block_rows(w, "v", s, i, i * B, (i + 1) * B, DEV)
    ids = sample_units(S, L, H, 48, seed=4)
    pre_k, pre_v = unit_rows(k5, ids, N + B), unit_rows(v5, ids, N + B)
    rs = gpu_state(v5, [N] * S, D)
    U, C = w.units, w.capacity
    kp = torch.zeros((U, C), dtype=torch.uint8, device=DEV)
    sc = torch.zeros((U, C), device=DEV)
    vd.vd_evict_step(k5, v5, [N + B] * S, [N] * S, "l2", running_sum=rs, keep_out=kp,
                     scores_out=sc)
    torch.cuda.synchronize()
    idx = torch.as_tensor(ids, device=DEV)
    rep = compare_pass(orc, pre_k, pre_v, unit_rows(k5, ids, N + B), unit_rows(v5, ids, N + B),
                       np.full(len(ids), N + B, np.int32), np.full(len(ids), N, np.int32), "l2",
                       w.dtype, scores_gpu=to_np(sc[idx]), keep_gpu=to_np(kp[idx]),
                       state=to_np(rs[idx]), unit_ids=ids)
    parity_log(f"wide_head_d256 boundary 0, {len(ids)} sampled units (l2)", rep)
    assert rep.near_ties <= max(2, rep.units // 100), rep


# ------------------------------------------------------------------ ragged

def test_ragged_serving_prefill_and_decode_sampled_units(orc, parity_log):
    """Ragged serving: 64 sequences of different prompt lengths and budgets, at
    lock-step block 40 (finished prompts are no-ops, others append a full or a
    partial block), then one decode step for all; 2 units per sequence checked."""
    w = synth.ragged()
    S, L, H, D, B = w.num_seqs, w.num_layers, w.num_kv_heads, w.head_dim, w.block
    blk = 40
    k5, v5 = synth.empty_cache(w, DEV)
    n_old, n_new = [], []
    for s in range(S):
        T, N = w.prompt[s], w.budget[s]
        no = min(N, blk * B)
        nn = max(0, min(B, T - blk * B))
        k5[s, :, :, :no] = synth.block_rows(w, "k", s, 1000, 0, no, DEV)
        v5[s, :, :, :no] = synth.block_rows(w, "v", s, 1000, 0, no, DEV)
        if nn:
            k5[s, :, :, no:no + nn] = synth.block_rows(w, "k", s, blk, blk * B, blk * B + nn, DEV)
            v5[s, :, :, no:no + nn] = synth.block_rows(w, "v", s, blk, blk * B, blk * B + nn, DEV)
        n_old.append(no)
        n_new.append(nn)
    n = [a + b for a, b in zip(n_old, n_new)]
    N = list(w.budget)
    rng = np.random.default_rng(5)
    ids = np.array(sorted({s * L * H + int(rng.integers(L * H)) for s in range(S)} |
                          {s * L * H + L * H - 1 for s in range(S)}))
    nu, Nu = per_unit(n, L, H)[ids], per_unit(N, L, H)[ids]
    C = w.capacity
    U = w.units
    idx = torch.as_tensor(ids, device=DEV)
    rs = gpu_state(v5, n_old, D)
    for phase in ("prefill", "decode"):
        pre_k, pre_v = unit_rows(k5, ids, C), unit_rows(v5, ids, C)
        kp = torch.zeros((U, C), dtype=torch.uint8, device=DEV)
        sc = torch.zeros((U, C), device=DEV)
        vd.vd_evict_step(k5, v5, n, N, "l2", running_sum=rs, keep_out=kp, scores_out=sc)
        torch.cuda.synchronize()
        rep = compare_pass(orc, pre_k, pre_v, unit_rows(k5, ids, C), unit_rows(v5, ids, C),
                           nu, Nu, "l2", w.dtype, scores_gpu=to_np(sc[idx]),
                           keep_gpu=to_np(kp[idx]), state=to_np(rs[idx]), unit_ids=ids)
        parity_log(f"ragged_serving block 40 {phase}, {len(ids)} sampled units (l2)", rep)
        assert rep.near_ties <= max(2, rep.units // 100), rep
        # next: one decode token for every sequence
        n = [min(a, b) for a, b in zip(n, N)]
        for s in range(S):
            k5[s, :, :, n[s]] = synth.block_rows(w, "k", s, 5000, 0, 1, DEV)[:, :, 0]
            v5[s, :, :, n[s]] = synth.block_rows(w, "v", s, 5000, 0, 1, DEV)[:, :, 0]
        n = [a + 1 for a in n]
        nu = per_unit(n, L, H)[ids]
