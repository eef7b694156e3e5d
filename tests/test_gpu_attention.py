"""GPU parity of the fused decode step (vd_decode_attention_evict) against the oracle.

Attention output: per query row, the oracle's fp64 softmax attention over the
unit's n rows before eviction (Sec. 2.1, Eq. attention).  The kernel works in
fp32: a logit z = scale * q . k carries a rounding error of at most about
(8 + 6) * 2^-24 relative to scale * sum_c |q_c k_c| (products of one lane,
then the tree over the lanes of a row), which for these inputs is below 1e-5
in absolute terms and changes each weight by a relative 1e-5 at most; each
lane group then adds at most a few hundred rows in fp32 (relative error below
300 * 2^-24 < 2e-5 of sum_j w_j |v_j|).  Hence the bar
|o_gpu - o_ref| <= 1e-4 * max_j |v_j| per column.

Eviction: the kept set, the compacted K, V and pos and the running sum follow
the bar of the pass (tests/parity.py): the GPU's kept set is read back from
the moved pos payload, and may differ from the oracle's only on a near-tie.

FastCAOTE (App. A, Eq. app_fastcaote): the evicted row must be the oracle's
argmin of s_j = a_j / (1 - a_j) ||v_j - v_bar||, or a row whose oracle score
lies within the near-tie band of that minimum.  The band follows the error of
the kernel's fp32 weights: a logit error dz (log2 units, at most 14 * 2^-24
of sum_c |q'_c k_c| with q' = q * scale * log2(e)) changes a weight by ln 2 *
dz relative, and the weight sum and the row's own weight enter the score, so
the band is 4 ln 2 * dz_max + 2e-5 relative to the minimum, plus an absolute
1e-6 of the largest finite score (weights that underflow fp32 score 0).
"""
import numpy as np
import pytest
import torch

from paper_2609_23314_amd import synth, vd
from parity import check_layout, compare_pass, per_unit, to_np, units, values_f64

pytestmark = pytest.mark.gpu
DEV = "cuda"
DTYPES = {"bf16": torch.bfloat16, "f32": torch.float32}
TOL_O = 1e-4


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    vd.load()


def make_cache(S, L, H, C, D, dtype, n, seed, same_rows=False):
    k = synth.random_rows((S, L, H, C, D), dtype, seed, DEV)
    v = synth.random_rows((S, L, H, C, D), dtype, seed + 1, DEV)
    if same_rows:
        v[:] = v[:, :, :, :1]
    for s in range(S):  # rows past n are never read
        k[s, :, :, n[s]:] = float("nan")
        v[s, :, :, n[s]:] = float("nan")
    return k, v


def state_covering(v_units, count):
    """Running sum over rows [0, count[u]) of every unit."""
    U, _, D = v_units.shape
    st = np.zeros((U, D + 1), np.float64)
    for u in range(U):
        c = int(count[u])
        st[u, :D] = values_f64(v_units[u, :c]).sum(axis=0)
        st[u, D] = c
    return torch.from_numpy(st).to(DEV)


def kept_from_pos(post_pos, n, N):
    """The GPU's kept set, read from the moved slot ids (pos starts as 0..C-1)."""
    keep = np.zeros(post_pos.shape[0], np.uint8)
    if n <= N:
        keep[:n] = 1
    else:
        keep[post_pos[:N]] = 1
    return keep


def compare_caote(orc, pre_k, pre_v, post_k, post_v, q_units, scale, n_unit, N_unit, keep_gpu,
                  pre_pos, post_pos, state):
    """FastCAOTE eviction of a decode step against the oracle (see the module
    docstring for the band); returns the number of near-tie units."""
    ties = 0
    for i in range(pre_v.shape[0]):
        n, N = int(n_unit[i]), int(N_unit[i])
        what = f"unit {i} (n={n}, N={N})"
        if n == 0:
            continue
        s_ref = orc.fastcaote_scores(q_units[i], pre_k[i, :n], pre_v[i, :n], scale)
        keep_ref = orc.select_topn(s_ref, N)
        kg = np.asarray(keep_gpu[i, :n]).astype(bool)
        m = min(n, N)
        if np.array_equal(kg, keep_ref.astype(bool)):
            ref_k, ref_v, ref_pos = pre_k[i].copy(), pre_v[i].copy(), pre_pos[i].copy()
            orc.compact(ref_k, ref_v, n, N, keep_ref, ref_pos)
            assert np.array_equal(post_v[i, :m], ref_v[:m]), f"{what}: V differs"
            assert np.array_equal(post_k[i, :m], ref_k[:m]), f"{what}: K differs"
            assert np.array_equal(post_pos[i, :m], ref_pos[:m]), f"{what}: pos differs"
        else:
            assert kg.sum() == m, what
            j_o = int(np.flatnonzero(~keep_ref.astype(bool))[0])
            j_g = int(np.flatnonzero(~kg)[0])
            qk = np.abs(q_units[i] * scale * np.log2(np.e)) @ np.abs(values_f64(pre_k[i, :n])).T
            dz = 14 * 2.0 ** -24 * qk.max()
            fin = s_ref[np.isfinite(s_ref)]
            band = (4 * np.log(2) * dz + 2e-5) * s_ref[j_o] + 1e-6 * (fin.max() if fin.size else 0)
            assert s_ref[j_g] - s_ref[j_o] <= band, (f"{what}: GPU evicted {j_g} (s={s_ref[j_g]!r}), "
                                                     f"oracle {j_o} (s={s_ref[j_o]!r}), band {band:.3g}")
            ties += 1
            for post, pre in ((post_v, pre_v), (post_k, pre_k), (post_pos, pre_pos)):
                check_layout(post[i], pre[i], kg, n, N, what)
        want = values_f64(post_v[i, :m]).sum(axis=0)
        assert state[i, -1] == m, what
        tol = 1e-12 * np.abs(values_f64(post_v[i, :m])).sum(axis=0) + 1e-300
        assert np.all(np.abs(state[i, :-1] - want) <= tol), f"{what}: running sum differs"
    return ties


def run_case(orc, S, L, H, G, C, D, dtype, n, N, seed, qscale=1.0, same_rows=False,
             sample=None, count=None, k_ramp=None, variant="l2"):
    k, v = make_cache(S, L, H, C, D, dtype, n, seed, same_rows)
    if k_ramp is not None:
        # every key row is slot 0's row times (1 + k_ramp * slot)
        j = torch.arange(C, device=DEV, dtype=torch.float32).view(1, 1, 1, C, 1)
        k.copy_((k[:, :, :, :1].float() * (1.0 + k_ramp * j)).to(dtype))
        for s in range(S):
            k[s, :, :, n[s]:] = float("nan")
    U = S * L * H
    n_u, N_u = per_unit(n, L, H), per_unit(N, L, H)
    cnt = np.maximum(n_u - 1, 0) if count is None else per_unit(count, L, H)
    idx = np.arange(U) if sample is None else np.asarray(sample)
    pre_k = units(to_np(k))[idx]
    pre_v = units(to_np(v))[idx]
    rs = state_covering(units(to_np(v)), cnt)
    pos = torch.arange(C, dtype=torch.int32, device=DEV).repeat(U, 1).contiguous()
    g = torch.Generator(device=DEV)
    g.manual_seed(seed + 7)
    q = torch.randn((S, L, H * G, D), generator=g, device=DEV) * qscale
    scale = D ** -0.5
    out = vd.vd_decode_attention_evict(k, v, q, n, N, rs, scale=scale, pos=pos, variant=variant)
    torch.cuda.synchronize()
    o = out.cpu().numpy().reshape(U, G, D)
    qn = q.cpu().numpy().astype(np.float64).reshape(U, G, D)
    for i, u in enumerate(idx):
        m = int(n_u[u])
        if m == 0:
            assert np.all(o[u] == 0.0), f"unit {u}: output of an empty unit"
            continue
        vmax = np.abs(values_f64(pre_v[i, :m])).max()
        for gg in range(G):
            ref = orc.attention(qn[u, gg], pre_k[i, :m], pre_v[i, :m], scale)
            err = np.abs(o[u, gg] - ref).max()
            assert err <= TOL_O * vmax, f"unit {u} head {gg}: attention error {err:.3g} (max |v| {vmax:.3g})"
    post_pos = to_np(pos)[idx]
    keep = np.stack([kept_from_pos(post_pos[i], int(n_u[u]), int(N_u[u]))
                     for i, u in enumerate(idx)])
    if variant == "fastcaote":
        ties = compare_caote(orc, pre_k, pre_v, units(to_np(k))[idx], units(to_np(v))[idx],
                             qn[idx], scale, n_u[idx], N_u[idx], keep,
                             np.arange(C, dtype=np.int32)[None].repeat(len(idx), 0), post_pos,
                             to_np(rs)[idx])
        return ties, k, v, rs, pos
    rep = compare_pass(orc, pre_k, pre_v, units(to_np(k))[idx], units(to_np(v))[idx],
                       n_u[idx], N_u[idx], "l2", dtype, keep_gpu=keep,
                       pre_pos=np.arange(C, dtype=np.int32)[None].repeat(len(idx), 0),
                       post_pos=post_pos, state=to_np(rs)[idx])
    return rep, k, v, rs, pos


@pytest.mark.parametrize("dt", list(DTYPES))
@pytest.mark.parametrize("D", [64, 128, 256])
@pytest.mark.parametrize("G", [1, 2, 4])
def test_decode_step_matches_oracle(orc, dt, D, G):
    # a unit that evicts at a tail of several tiles, a shorter one, and one
    # under its budget (attention only; the state takes the newest row)
    rep, *_ = run_case(orc, 3, 2, 2, G, 320, D, DTYPES[dt], [300, 201, 150], [299, 200, 200],
                       seed=500 + D + G)
    print(rep)


def test_decode_step_tiny_units(orc):
    # n = 0, n = 1 under budget, n = 2 over a budget of 1
    rep, *_ = run_case(orc, 3, 1, 2, 2, 8, 64, torch.float32, [0, 1, 2], [1, 1, 1], seed=61)
    print(rep)


def test_decode_step_equal_scores_evict_newest(orc):
    # identical value rows: every score is 0, the highest slot (the newest
    # row) goes and nothing moves
    rep, k, v, rs, pos = run_case(orc, 1, 1, 2, 4, 130, 128, torch.bfloat16, [129], [128], seed=62,
                                  same_rows=True)
    assert torch.equal(pos[:, :128].cpu(), torch.arange(128, dtype=torch.int32).repeat(2, 1))


def test_decode_step_sharp_softmax(orc):
    # large queries: the softmax is nearly one-hot
    rep, *_ = run_case(orc, 2, 1, 2, 4, 520, 128, torch.bfloat16, [513, 400], [512, 399],
                       seed=63, qscale=30.0)
    print(rep)


def test_decode_step_rising_logits(orc):
    # keys along one direction with a growing length: for the query heads that
    # face it the logits rise along the slots, so each lane group raises its
    # softmax reference again and again, by steps above and below 2^8; 128
    # units give 6 splits of 6 tiles per lane group
    S, H = 16, 8
    rep, *_ = run_case(orc, S, 1, H, 4, 1040, 128, torch.bfloat16, [1025] * S, [1024] * S,
                       seed=67, qscale=2.0, k_ramp=0.05)
    print(rep)


def test_decode_step_stale_state_is_recounted(orc):
    # a state covering fewer rows than n - 1: the rows it does not cover are
    # added by every workgroup; results as before
    rep, *_ = run_case(orc, 2, 1, 2, 2, 200, 64, torch.float32, [190, 120], [189, 119], seed=64,
                       count=[150, 0])
    print(rep)


def test_decode_step_many_sequences(orc):
    n = [(29 * s) % 41 + 1 for s in range(300)]
    N = [max(1, x - (s % 2)) for s, x in enumerate(n)]
    rep, *_ = run_case(orc, 300, 1, 1, 2, 48, 64, torch.bfloat16, n, N, seed=65)
    print(rep)


@pytest.mark.parametrize("dt", list(DTYPES))
@pytest.mark.parametrize("D", [64, 128, 256])
@pytest.mark.parametrize("G", [1, 2, 4])
def test_fastcaote_decode_step_matches_oracle(orc, dt, D, G):
    """FastCAOTE in the fused decode step (App. A, Eq. app_fastcaote): the
    attention output as for ValueDiff, and the eviction of the row with the
    lowest a_j / (1 - a_j) ||v_j - v_bar||."""
    ties, *_ = run_case(orc, 3, 2, 2, G, 320, D, DTYPES[dt], [300, 201, 150], [299, 200, 200],
                        seed=540 + D + G, variant="fastcaote")
    assert ties <= 1, ties


def test_fastcaote_uniform_attention_evicts_like_valuediff(orc):
    """Zero queries weigh every row 1/n, so FastCAOTE's scores are the L2
    scores / (n - 1) and it evicts the row ValueDiff evicts (App. A: the
    max-entropy limit); identical caches, identical results."""
    S, L, H, G, C, D = 2, 1, 4, 4, 700, 128
    n, N = [700, 513], [699, 512]
    k, v = make_cache(S, L, H, C, D, torch.bfloat16, n, seed=550)
    U = S * L * H
    cnt = np.repeat(np.asarray(n) - 1, L * H)
    outs = []
    for variant in ("l2", "fastcaote"):
        kk, vv = k.clone(), v.clone()
        rs = state_covering(units(to_np(vv)), cnt)
        pos = torch.arange(C, dtype=torch.int32, device=DEV).repeat(U, 1).contiguous()
        q = torch.zeros((S, L, H * G, D), device=DEV)
        vd.vd_decode_attention_evict(kk, vv, q, n, N, rs, pos=pos, variant=variant)
        torch.cuda.synchronize()
        outs.append((kk, vv, rs, pos))
    for a, b in zip(outs[0], outs[1]):   # bit patterns: the tail rows hold NaN
        assert torch.equal(a.contiguous().view(torch.uint8), b.contiguous().view(torch.uint8))


def test_fastcaote_sharp_and_rising_logits(orc):
    """Nearly one-hot softmax (large queries), and logits that rise along the
    slots: rows that take almost all the weight score near +infinity, rows
    whose weight underflows fp32 score 0 (the highest such slot goes)."""
    # (rows whose weight underflows fp32 in every head tie at 0 on the GPU, so
    # near-ties are expected here; compare_caote checks each against the band)
    run_case(orc, 2, 1, 2, 4, 520, 128, torch.bfloat16, [513, 400], [512, 399],
             seed=563, qscale=30.0, variant="fastcaote")
    run_case(orc, 16, 1, 8, 4, 1040, 128, torch.bfloat16, [1025] * 16, [1024] * 16,
             seed=567, qscale=2.0, k_ramp=0.05, variant="fastcaote")


def test_fastcaote_decode_workload_layer(orc):
    """The decode workload's shape, one layer per call (16 x 8 units, 32 query
    heads, n = 4097, N = 4096, 6 row splits per unit), 12 sampled units."""
    S, H, G, D, N = 16, 8, 4, 128, 4096
    rng = np.random.default_rng(571)
    idx = np.sort(rng.choice(S * H, size=12, replace=False))
    ties, *_ = run_case(orc, S, 1, H, G, N + 1, D, torch.bfloat16, [N + 1] * S, [N] * S,
                        seed=572, sample=idx, variant="fastcaote")
    assert ties <= 1


def test_decode_steps_in_a_row(orc):
    # three decode steps: each appends a new row at slot N and evicts one
    S, L, H, G, C, D, N = 2, 2, 2, 4, 260, 128, 256
    k, v = make_cache(S, L, H, C, D, torch.bfloat16, [N + 1] * S, seed=66)
    U = S * L * H
    rs = state_covering(units(to_np(v)), [N] * U)
    pos = torch.arange(C, dtype=torch.int32, device=DEV).repeat(U, 1).contiguous()
    for step in range(3):
        new_k = synth.random_rows((S, L, H, D), torch.bfloat16, 700 + step, DEV)
        new_v = synth.random_rows((S, L, H, D), torch.bfloat16, 800 + step, DEV)
        if step > 0:
            k[:, :, :, N] = new_k
            v[:, :, :, N] = new_v
            pos.view(S, L, H, C)[:, :, :, N] = 1000 + step
        pre_k, pre_v, pre_pos = units(to_np(k)), units(to_np(v)), to_np(pos)
        g = torch.Generator(device=DEV)
        g.manual_seed(900 + step)
        q = torch.randn((S, L, H * G, D), generator=g, device=DEV)
        out = vd.vd_decode_attention_evict(k, v, q, [N + 1] * S, [N] * S, rs, pos=pos)
        torch.cuda.synchronize()
        o = out.cpu().numpy().reshape(U, G, D)
        qn = q.cpu().numpy().astype(np.float64).reshape(U, G, D)
        for u in range(U):
            vmax = np.abs(values_f64(pre_v[u, :N + 1])).max()
            for gg in range(G):
                ref = orc.attention(qn[u, gg], pre_k[u, :N + 1], pre_v[u, :N + 1], D ** -0.5)
                assert np.abs(o[u, gg] - ref).max() <= TOL_O * vmax, (step, u, gg)
        post_pos = to_np(pos)
        # the kept set, by original slot: slots whose pos payload survived in [0, N)
        keep = np.stack([np.isin(pre_pos[u, :N + 1], post_pos[u, :N]).astype(np.uint8)
                         for u in range(U)])
        compare_pass(orc, pre_k, pre_v, units(to_np(k)), units(to_np(v)),
                     np.full(U, N + 1), np.full(U, N), "l2", torch.bfloat16, keep_gpu=keep,
                     pre_pos=pre_pos, post_pos=post_pos, state=to_np(rs))


@pytest.mark.parametrize("per_layer", [True, False])
def test_decode_workload_sampled(orc, per_layer):
    # the decode workload's shape: 16 sequences x 32 layers x 8 KV heads, 32
    # query heads, n = 4097, N = 4096; one layer per call (128 units, 6 row
    # splits per unit) or all layers in one call (one split per unit)
    S, L, H, G, D, N = 16, 32, 8, 4, 128, 4096
    C = N + 1
    layers = [5] if per_layer else list(range(L))
    Lc = len(layers)
    k = synth.random_rows((S, Lc, H, C, D), torch.bfloat16, 71, DEV)
    v = synth.random_rows((S, Lc, H, C, D), torch.bfloat16, 72, DEV)
    U = S * Lc * H
    rng = np.random.default_rng(5)
    idx = np.sort(rng.choice(U, size=10, replace=False))
    kv_u = v.view(U, C, D)
    ku_u = k.view(U, C, D)
    st = torch.zeros((U, D + 1), dtype=torch.float64, device=DEV)
    for a in range(0, U, 256):
        st[a:a + 256, :D] = kv_u[a:a + 256, :N].to(torch.float64).sum(dim=1)
    st[:, D] = N
    pre_k = to_np(ku_u[idx])
    pre_v = to_np(kv_u[idx])
    pos = torch.arange(C, dtype=torch.int32, device=DEV).repeat(U, 1).contiguous()
    g = torch.Generator(device=DEV)
    g.manual_seed(73)
    q = torch.randn((S, Lc, H * G, D), generator=g, device=DEV)
    out = vd.vd_decode_attention_evict(k, v, q, [C] * S, [N] * S, st, pos=pos)
    torch.cuda.synchronize()
    o = out.view(U, G, D)[idx].cpu().numpy()
    qn = q.view(U, G, D)[idx].cpu().numpy().astype(np.float64)
    for i in range(len(idx)):
        vmax = np.abs(values_f64(pre_v[i])).max()
        for gg in range(G):
            ref = orc.attention(qn[i, gg], pre_k[i], pre_v[i], D ** -0.5)
            assert np.abs(o[i, gg] - ref).max() <= TOL_O * vmax, (int(idx[i]), gg)
    post_pos = to_np(pos[idx])
    keep = np.stack([kept_from_pos(post_pos[i], C, N) for i in range(len(idx))])
    rep = compare_pass(orc, pre_k, pre_v, to_np(ku_u[idx]), to_np(kv_u[idx]),
                       np.full(len(idx), C), np.full(len(idx), N), "l2", torch.bfloat16,
                       keep_gpu=keep, pre_pos=np.arange(C, dtype=np.int32)[None].repeat(len(idx), 0),
                       post_pos=post_pos, state=to_np(st[idx]))
    print(rep)
    # every unit evicted exactly one row and kept N
    assert torch.all(st[:, D] == N)
