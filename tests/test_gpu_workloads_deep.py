"""GPU parity deep inside the large workloads' trajectories, at their full
sizes and in the launch shape the benchmark times.

The oracle runs its own trajectory (its own evictions, pass after pass) on
the compared units; at each checked pass the GPU's copy of those units is
first set to the oracle's pre-pass state ("oracle-forced"), so that a benign
near-tie swap earlier on cannot make the two trajectories drift apart.  The
units not compared run free on the GPU.  Each checked pass is a block
boundary of Sec. 2.2, Eq. block_processing (B = 1 for a decode step), and
the pass is Sec. 2.1, Eq. eviction with the scores of Sec. 3.2.

  decode_b16       decode steps 0, 1, 511 and 1023 of 1024 on a fixed 1/64
                   sample of the 4096 units
  wide_head_d256   every one of the 416 units at the first and the last of
                   the 60 evicting boundaries, for L2, Dir and Norm
  ragged_serving   the first evicting and the last lock-step prefill call,
                   then decode steps 0, 1023 and 2047 of 2048, on a fixed
                   sample of two units per sequence

Every comparison's counts (units, near-ties, largest relative score error)
are recorded through the parity_log fixture.
"""
import numpy as np
import pytest
import torch

from paper_2609_23314_amd import synth, vd
from parity import Report, compare_pass, from_np, to_np, units

pytestmark = pytest.mark.gpu
DEV = "cuda"


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    vd.load()


def fp64_state(x_units, count):
    """Running sum of rows [0, count[u]) of every unit of a [U, C, D] view,
    summed in fp64 by torch (an input of the HIP path; exact for bf16 values)."""
    U, _, D = x_units.shape
    st = torch.zeros((U, D + 1), dtype=torch.float64, device=DEV)
    for c in sorted(set(int(x) for x in count)):
        sel = torch.as_tensor([u for u in range(U) if int(count[u]) == c], device=DEV)
        st[sel, :D] = x_units[sel, :c].double().sum(dim=1)
        st[sel, D] = c
    return st


def force(k_u, v_u, pos, rs, ids, ok, ov, opos, count, dtype):
    """The GPU's compared units take the oracle's pre-pass rows, pos and a
    state covering their first count rows."""
    idx = torch.as_tensor(ids, device=DEV)
    upto = ok.shape[1]
    k_u[idx, :upto] = from_np(ok, dtype, DEV)
    v_u[idx, :upto] = from_np(ov, dtype, DEV)
    if pos is not None:
        pos[idx, :upto] = torch.from_numpy(opos).to(DEV)
    rs[idx] = fp64_state(v_u[idx], count)


# ------------------------------------------------------------------ decode

def test_decode_b16_deep_steps(orc, parity_log):
    """decode_b16: 16 sequences x 256 units, cache full at N = 4096; every
    decode step appends one token per sequence and evicts one per unit.
    Steps 0, 1, 511 and 1023 are compared on 64 fixed units (1/64)."""
    w = synth.decode()
    N, D = w.budget[0], w.head_dim
    S, L, H = w.num_seqs, w.num_layers, w.num_kv_heads
    U, C = w.units, w.capacity
    check = (0, 1, 511, 1023)
    k5, v5 = synth.empty_cache(w, DEV)
    for s in range(S):
        k5[s, :, :, :N + 1] = synth.block_rows(w, "k", s, 0, 0, N + 1, DEV, seq_seed=s)
        v5[s, :, :, :N + 1] = synth.block_rows(w, "v", s, 0, 0, N + 1, DEV, seq_seed=s)
    k_u, v_u = k5.view(U, C, D), v5.view(U, C, D)
    rs = fp64_state(v_u, [N] * U)
    pos = torch.arange(C, dtype=torch.int32, device=DEV).repeat(U, 1).contiguous()
    rng = np.random.default_rng(31)
    ids = np.sort(rng.choice(U, size=U // 64, replace=False))
    idx = torch.as_tensor(ids, device=DEV)
    ok, ov = to_np(k_u[idx]), to_np(v_u[idx])          # the oracle's trajectory
    opos = np.tile(np.arange(C, dtype=np.int32), (len(ids), 1))
    nu = np.full(len(ids), C, np.int32)
    Nu = np.full(len(ids), N, np.int32)
    rep = Report()
    for t in range(max(check) + 1):
        if t > 0:   # every sequence appends its token of step t at slot N
            kr = synth.decode_rows(w, "k", t, DEV).reshape(U, D)
            vr = synth.decode_rows(w, "v", t, DEV).reshape(U, D)
            k_u[:, N] = kr
            v_u[:, N] = vr
            pos[:, N] = N + t
            ok[:, N], ov[:, N] = to_np(kr[idx]), to_np(vr[idx])
            opos[:, N] = N + t
        if t in check:
            force(k_u, v_u, pos, rs, ids, ok, ov, opos, [N] * len(ids), w.dtype)
            sc = torch.zeros((U, C), device=DEV)
            kp = torch.zeros((U, C), dtype=torch.uint8, device=DEV)
            vd.vd_evict_step(k5, v5, [C] * S, [N] * S, "l2", running_sum=rs, pos=pos,
                             scores_out=sc, keep_out=kp)
            torch.cuda.synchronize()
            compare_pass(orc, ok, ov, to_np(k_u[idx]), to_np(v_u[idx]), nu, Nu, "l2", w.dtype,
                         scores_gpu=to_np(sc[idx]), keep_gpu=to_np(kp[idx]), pre_pos=opos,
                         post_pos=to_np(pos[idx]), state=to_np(rs[idx]), unit_ids=ids,
                         report=rep)
            assert torch.all(kp[:, :C].sum(dim=1) == N), f"step {t}: a unit did not keep N"
        else:
            vd.vd_evict_step(k5, v5, [C] * S, [N] * S, "l2", running_sum=rs, pos=pos)
        orc.evict_step(ok, ov, nu, Nu, "l2", pos=opos)   # the oracle's own step
    parity_log("decode_b16 steps 0,1,511,1023 (l2, 1/64 of the units)", rep)
    assert rep.units == len(check) * len(ids)
    assert rep.near_ties <= max(2, rep.units // 100), rep


# ------------------------------------------------------------------ wide

@pytest.mark.parametrize("variant", ["l2", "dir", "norm"])
def test_wide_head_first_and_last_boundary_all_units(orc, parity_log, variant):
    """wide_head_d256 (d = 256, Student-t values): the oracle processes the
    whole 65536-token prompt of all 416 units (64 blocks, 60 evicting
    passes); the first and the last evicting pass are compared on every unit."""
    w = synth.wide()
    N, B, D = w.budget[0], w.block, w.head_dim
    S, L, H = w.num_seqs, w.num_layers, w.num_kv_heads
    U, C = w.units, w.capacity
    ok = np.zeros((U, C, D), np.uint16)
    ov = np.zeros((U, C, D), np.uint16)
    n_o, passes = 0, 0
    nblocks = w.prompt[0] // B
    checked = (0, 59)
    rep = Report()
    for blk in range(nblocks):
        t0 = blk * B
        kb = torch.stack([synth.block_rows(w, "k", s, blk, t0, t0 + B, DEV) for s in range(S)])
        vb = torch.stack([synth.block_rows(w, "v", s, blk, t0, t0 + B, DEV) for s in range(S)])
        ok[:, n_o:n_o + B] = to_np(kb.reshape(U, B, D))
        ov[:, n_o:n_o + B] = to_np(vb.reshape(U, B, D))
        del kb, vb
        n = n_o + B
        if n <= N:
            n_o = n
            continue
        nu = np.full(U, n, np.int32)
        Nu = np.full(U, N, np.int32)
        if passes in checked:
            k5 = from_np(ok, w.dtype, DEV).view(S, L, H, C, D)
            v5 = from_np(ov, w.dtype, DEV).view(S, L, H, C, D)
            rs = fp64_state(v5.view(U, C, D), [n_o] * U)
            sc = torch.zeros((U, C), device=DEV)
            kp = torch.zeros((U, C), dtype=torch.uint8, device=DEV)
            vd.vd_evict_step(k5, v5, [n] * S, [N] * S, variant, running_sum=rs, scores_out=sc,
                             keep_out=kp)
            torch.cuda.synchronize()
            compare_pass(orc, ok, ov, units(to_np(k5)), units(to_np(v5)), nu, Nu, variant,
                         w.dtype, scores_gpu=to_np(sc), keep_gpu=to_np(kp), state=to_np(rs),
                         report=rep)
            del k5, v5, sc, kp, rs
        orc.evict_step(ok, ov, nu, Nu, variant)
        n_o = N
        passes += 1
    assert passes == 60
    parity_log(f"wide_head_d256 boundaries 0 and 59, all 416 units ({variant})", rep)
    assert rep.units == 2 * U
    assert rep.near_ties <= max(2, rep.units // 100), rep


# ------------------------------------------------------------------ ragged

def test_ragged_serving_prefill_and_decode_deep(orc, parity_log):
    """ragged_serving: 64 sequences of prompt lengths 4096..32768 and budgets
    of a quarter of them, blocks of 256 (the last partial), processed in lock
    step (a finished prompt appends nothing), then 2048 decode steps.  The
    first evicting and the last prefill call, and decode steps 0, 1023 and
    2047, are compared on two fixed units of every sequence."""
    w = synth.ragged()
    S, L, H, D, B = w.num_seqs, w.num_layers, w.num_kv_heads, w.head_dim, w.block
    U, C = w.units, w.capacity
    LH = L * H
    rng = np.random.default_rng(41)
    ids = np.array(sorted(s * LH + int(x) for s in range(S)
                          for x in rng.choice(LH, size=2, replace=False)))
    idx = torch.as_tensor(ids, device=DEV)
    seq_of = ids // LH
    k5, v5 = synth.empty_cache(w, DEV)
    k_u, v_u = k5.view(U, C, D), v5.view(U, C, D)
    rs = torch.zeros((U, D + 1), dtype=torch.float64, device=DEV)
    pos = torch.full((U, C), -1, dtype=torch.int32, device=DEV)
    ok = np.zeros((len(ids), C, D), np.uint16)
    ov = np.zeros((len(ids), C, D), np.uint16)
    opos = np.full((len(ids), C), -1, np.int32)
    n = [0] * S
    budget = list(w.budget)
    Nu = np.asarray(budget, np.int32)[seq_of]
    nblocks = (max(w.prompt) + B - 1) // B
    first_evicting = next(b for b in range(nblocks)
                          if any(min(budget[s], b * B) + max(0, min(B, w.prompt[s] - b * B))
                                 > budget[s] for s in range(S)))
    rep_p, rep_d = Report(), Report()

    def run(call_n, checked, rep):
        nu = np.asarray(call_n, np.int32)[seq_of]
        n_old_u = np.asarray(n_old, np.int32)[seq_of]
        if checked:
            force(k_u, v_u, pos, rs, ids, ok, ov, opos, n_old_u, w.dtype)
            sc = torch.zeros((U, C), device=DEV)
            kp = torch.zeros((U, C), dtype=torch.uint8, device=DEV)
            vd.vd_evict_step(k5, v5, call_n, budget, "l2", running_sum=rs, pos=pos,
                             scores_out=sc, keep_out=kp)
            torch.cuda.synchronize()
            compare_pass(orc, ok, ov, to_np(k_u[idx]), to_np(v_u[idx]), nu, Nu, "l2", w.dtype,
                         scores_gpu=to_np(sc[idx]), keep_gpu=to_np(kp[idx]), pre_pos=opos,
                         post_pos=to_np(pos[idx]), state=to_np(rs[idx]), unit_ids=ids,
                         report=rep)
        else:
            vd.vd_evict_step(k5, v5, call_n, budget, "l2", running_sum=rs, pos=pos)
        if (nu > Nu).any():
            orc.evict_step(ok, ov, nu, Nu, "l2", pos=opos)

    # lock-step prefill
    for blk in range(nblocks):
        n_old = list(n)
        for s in range(S):
            t0, t1 = blk * B, min(blk * B + B, w.prompt[s])
            if t1 <= t0:
                continue
            kr = synth.block_rows(w, "k", s, blk, t0, t1, DEV)
            vr = synth.block_rows(w, "v", s, blk, t0, t1, DEV)
            k5[s, :, :, n[s]:n[s] + t1 - t0] = kr
            v5[s, :, :, n[s]:n[s] + t1 - t0] = vr
            pos[s * LH:(s + 1) * LH, n[s]:n[s] + t1 - t0] = torch.arange(
                t0, t1, dtype=torch.int32, device=DEV)
            mine = np.flatnonzero(seq_of == s)
            loc = torch.as_tensor(ids[mine] - s * LH, device=DEV)
            ok[mine, n[s]:n[s] + t1 - t0] = to_np(kr.reshape(LH, t1 - t0, D)[loc])
            ov[mine, n[s]:n[s] + t1 - t0] = to_np(vr.reshape(LH, t1 - t0, D)[loc])
            opos[mine, n[s]:n[s] + t1 - t0] = np.arange(t0, t1, dtype=np.int32)
            n[s] += t1 - t0
        run(n, blk in (first_evicting, nblocks - 1), rep_p)
        n = [min(a, b) for a, b in zip(n, budget)]
    # decode: every sequence appends one token and evicts one
    check = (0, 1023, 2047)
    for t in range(w.decode_steps):
        n_old = list(n)
        kr = synth.decode_rows(w, "k", t + 1, DEV).reshape(U, D)
        vr = synth.decode_rows(w, "v", t + 1, DEV).reshape(U, D)
        slot = torch.as_tensor(np.repeat(np.asarray(n, np.int64), LH), device=DEV)
        ar = torch.arange(U, device=DEV)
        k_u[ar, slot] = kr
        v_u[ar, slot] = vr
        tok = torch.as_tensor(np.repeat(np.asarray(w.prompt, np.int64) + t, LH), device=DEV)
        pos[ar, slot] = tok.to(torch.int32)
        r = np.arange(len(ids))
        ns = np.asarray(n)[seq_of]
        ok[r, ns] = to_np(kr[idx])
        ov[r, ns] = to_np(vr[idx])
        opos[r, ns] = (np.asarray(w.prompt)[seq_of] + t).astype(np.int32)
        n = [a + 1 for a in n]
        run(n, t in check, rep_d)
        n = [min(a, b) for a, b in zip(n, budget)]
    parity_log("ragged_serving prefill calls first evicting and last (l2, 2 units/seq)", rep_p)
    parity_log("ragged_serving decode steps 0,1023,2047 (l2, 2 units/seq)", rep_d)
    assert rep_p.units == 2 * len(ids) and rep_d.units == 3 * len(ids)
    for rep in (rep_p, rep_d):
        assert rep.near_ties <= max(2, rep.units // 100), rep
