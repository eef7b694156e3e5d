"""GPU parity of the HIP path against the oracle, through the C ABI.

Small cases span several row tiles of the kernels plus a ragged tail; edge
cases cover no-op units, the decode argmin path, crossing fill, ties, zero
rows, duplicate rows, strided layouts, more sequences than one launch takes,
and rows past n holding NaN (which must never be read).
"""
import numpy as np
import pytest
import torch

from paper_2609_23314_amd import synth, vd
from parity import (check_scores, compare_pass, per_unit, score_scale, to_np, units,
                    values_f64)

pytestmark = pytest.mark.gpu
DEV = "cuda"
VARIANTS = ["l2", "dir", "norm"]
KEY_VARIANTS = ["key_l2", "key_dir", "key_norm"]   # the same forms on K; KeyNorm keeps smallest
ALL_VARIANTS = VARIANTS + KEY_VARIANTS
DTYPES = {"bf16": torch.bfloat16, "f32": torch.float32}


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    vd.load()


def make_cache(S, L, H, C, D, dtype, n, seed, layout="hnd", dist="normal", nan_tail=True):
    """Seeded K/V caches as [S, L, H, C, D] views; slots >= n hold NaN."""
    if layout == "hnd":
        k = synth.random_rows((S, L, H, C, D), dtype, seed, DEV, dist)
        v = synth.random_rows((S, L, H, C, D), dtype, seed + 1, DEV, dist)
    else:  # per-layer [S, L, C, H, D] storage seen through a permuted view
        k = synth.random_rows((S, L, C, H, D), dtype, seed, DEV, dist).permute(0, 1, 3, 2, 4)
        v = synth.random_rows((S, L, C, H, D), dtype, seed + 1, DEV, dist).permute(0, 1, 3, 2, 4)
    if nan_tail:
        for s in range(S):
            k[s, :, :, n[s]:] = float("nan")
            v[s, :, :, n[s]:] = float("nan")
    return k, v


def state_for(v_np_units, count_unit, D):
    """Running-sum state describing rows [0, count) of every unit."""
    U = v_np_units.shape[0]
    st = np.zeros((U, D + 1), np.float64)
    for u in range(U):
        c = int(count_unit[u])
        st[u, :D] = values_f64(v_np_units[u, :c]).sum(axis=0)
        st[u, D] = c
    return torch.from_numpy(st).to(DEV)


def run_step_case(orc, S, L, H, C, D, dtype, n, N, variant, seed, state="none",
                  count=None, layout="hnd", dist="normal", k_present=True):
    k, v = make_cache(S, L, H, C, D, dtype, n, seed, layout, dist)
    U = S * L * H
    pre_k, pre_v = units(to_np(k)), units(to_np(v))
    pos = torch.arange(C, dtype=torch.int32, device=DEV).repeat(U, 1).contiguous()
    pre_pos = to_np(pos)
    scores = torch.full((U, C), -1.0, device=DEV)
    keep = torch.full((U, C), 7, dtype=torch.uint8, device=DEV)
    rs = None
    if state == "zero":
        rs = torch.zeros((U, D + 1), dtype=torch.float64, device=DEV)
    elif state == "incremental":
        rs = state_for(pre_k if variant.startswith("key") else pre_v, per_unit(count, L, H), D)
    vd.vd_evict_step(k if k_present else None, v, n, N, variant, running_sum=rs, pos=pos,
                     scores_out=scores, keep_out=keep)
    torch.cuda.synchronize()
    rep = compare_pass(orc, pre_k if k_present else None, pre_v, units(to_np(k)),
                       units(to_np(v)), per_unit(n, L, H), per_unit(N, L, H), variant, dtype,
                       scores_gpu=to_np(scores), keep_gpu=to_np(keep), pre_pos=pre_pos,
                       post_pos=to_np(pos), state=to_np(rs) if rs is not None else None)
    return rep


# ------------------------------------------------------------------ vd_score

@pytest.mark.parametrize("dt", list(DTYPES))
@pytest.mark.parametrize("D", [64, 128, 256])
@pytest.mark.parametrize("variant", ALL_VARIANTS)
def test_score_matches_oracle(orc, dt, D, variant):
    dtype = DTYPES[dt]
    S, L, H, C = 2, 2, 3, 1400
    n = [1400, 777]
    k, v = make_cache(S, L, H, C, D, dtype, n, seed=10 + D, dist="shifted")
    U = S * L * H
    scores = torch.full((U, C), -1.0, device=DEV)
    mean = torch.zeros((U, D), device=DEV)
    vd.vd_score(v, n, variant, scores, mean, k=k)
    torch.cuda.synchronize()
    pre_v = units(to_np(k if variant.startswith("key") else v))   # the scored rows
    sg, mg = to_np(scores), to_np(mean)
    nu = per_unit(n, L, H)
    for u in range(U):
        s_ref, m_ref = orc.score(pre_v[u, :nu[u]], variant)
        check_scores(sg[u, :nu[u]], s_ref, dtype, f"unit {u}",
                     score_scale(pre_v[u, :nu[u]], variant))
        assert np.all(np.abs(mg[u] - m_ref) <= 1e-6 * np.abs(m_ref) + 1e-7), f"mean of unit {u}"
        assert np.all(sg[u, nu[u]:] == -1.0), "wrote past n"


# ------------------------------------------------------------------ vd_select_topn

@pytest.mark.parametrize("ties", [False, True])
def test_select_matches_oracle_exactly(orc, ties):
    """Selection on given fp32 scores is an integer decision: bit-exact."""
    S, L, H, C, D = 3, 2, 2, 2100, 64
    n, N = [2100, 513, 1], [1000, 512, 1]
    v = torch.zeros((S, L, H, C, D), dtype=torch.float32, device=DEV)
    U = S * L * H
    sc = torch.stack([synth.random_scores(C, 100 + u, ties, DEV) for u in range(U)])
    keep = torch.full((U, C), 7, dtype=torch.uint8, device=DEV)
    vd.vd_select_topn(v, sc, n, N, keep)
    torch.cuda.synchronize()
    kg, s64 = to_np(keep), to_np(sc).astype(np.float64)
    nu, Nu = per_unit(n, L, H), per_unit(N, L, H)
    for u in range(U):
        want = orc.select_topn(s64[u, :nu[u]], int(Nu[u]))
        assert np.array_equal(kg[u, :nu[u]], want), f"unit {u}"
        assert np.all(kg[u, nu[u]:] == 7)


@pytest.mark.parametrize("ties", [False, True])
def test_select_slot_runs(orc, ties):
    """Slot counts where every wave takes the same number of 64-slot blocks
    (n = 2048), where all but one take one block more (n = 3000, 47 blocks)
    and the largest capacity (16384 slots, 16 blocks a wave), with the
    threshold deep in the order and at its edges."""
    S, L, H, C, D = 3, 1, 2, 16384, 64
    n, N = [2048, 3000, 16384], [1500, 2999, 9000]
    v = torch.zeros((S, L, H, C, D), dtype=torch.float32, device=DEV)
    U = S * L * H
    sc = torch.stack([synth.random_scores(C, 300 + u, ties, DEV) for u in range(U)])
    keep = torch.full((U, C), 7, dtype=torch.uint8, device=DEV)
    vd.vd_select_topn(v, sc, n, N, keep)
    torch.cuda.synchronize()
    kg, s64 = to_np(keep), to_np(sc).astype(np.float64)
    nu, Nu = per_unit(n, L, H), per_unit(N, L, H)
    for u in range(U):
        want = orc.select_topn(s64[u, :nu[u]], int(Nu[u]))
        assert np.array_equal(kg[u, :nu[u]], want), f"unit {u} (n = {nu[u]})"
        assert np.all(kg[u, nu[u]:] == 7)


def test_select_negative_scores_and_signed_zeros(orc):
    """Scores of any sign (a caller's own ranking), with +0 and -0 mixed: the
    two zeros are one value, so they tie and the lower slot wins."""
    S, L, H, C, D = 1, 1, 4, 1500, 64
    n, N = [1500], [700]
    v = torch.zeros((S, L, H, C, D), dtype=torch.float32, device=DEV)
    rng = np.random.default_rng(37)
    rows = []
    for u in range(4):
        x = rng.standard_normal(C).astype(np.float32) * (10.0 ** (u - 1))
        x[rng.random(C) < 0.3] = 0.0
        x[rng.random(C) < 0.3] = -0.0
        if u == 3:
            x[:] = np.where(rng.random(C) < 0.5, np.float32(0.0), np.float32(-0.0))  # all zero
        rows.append(x)
    sc = torch.from_numpy(np.stack(rows)).to(DEV)
    keep = torch.full((4, C), 7, dtype=torch.uint8, device=DEV)
    vd.vd_select_topn(v, sc, n, N, keep)
    torch.cuda.synchronize()
    kg = to_np(keep)
    for u in range(4):
        want = orc.select_topn(rows[u][:n[0]].astype(np.float64), N[0])
        assert np.array_equal(kg[u, :n[0]], want), f"unit {u}"
    assert np.array_equal(kg[3, :n[0]], (np.arange(n[0]) < N[0]).astype(np.uint8))


# ------------------------------------------------------------------ vd_compact

@pytest.mark.parametrize("dt", list(DTYPES))
@pytest.mark.parametrize("D", [64, 256])
def test_compact_matches_oracle_exactly(orc, dt, D):
    dtype = DTYPES[dt]
    S, L, H, C = 2, 2, 2, 1500
    n, N = [1500, 700], [900, 699]
    k, v = make_cache(S, L, H, C, D, dtype, n, seed=33)
    U = S * L * H
    nu, Nu = per_unit(n, L, H), per_unit(N, L, H)
    keep = torch.zeros((U, C), dtype=torch.uint8)
    for u in range(U):
        keep[u, :nu[u]] = synth.random_keep(int(nu[u]), int(Nu[u]), 200 + u)
    keep = keep.to(DEV)
    pos = torch.arange(C, dtype=torch.int32, device=DEV).repeat(U, 1).contiguous()
    pre_k, pre_v, pre_pos = units(to_np(k)), units(to_np(v)), to_np(pos)
    vd.vd_compact(k, v, keep, n, N, pos)
    torch.cuda.synchronize()
    post_k, post_v, post_pos = units(to_np(k)), units(to_np(v)), to_np(pos)
    kn = to_np(keep)
    for u in range(U):
        rk, rv, rp = pre_k[u].copy(), pre_v[u].copy(), pre_pos[u].copy()
        orc.compact(rk, rv, int(nu[u]), int(Nu[u]), kn[u, :nu[u]], rp)
        assert np.array_equal(post_k[u].view(np.uint8), rk.view(np.uint8)), f"K of unit {u}"
        assert np.array_equal(post_v[u].view(np.uint8), rv.view(np.uint8)), f"V of unit {u}"
        assert np.array_equal(post_pos[u], rp), f"pos of unit {u}"


def test_compact_with_unbalanced_masks(orc):
    """Masks that keep more or fewer than N slots: only min(#holes, #movers)
    rows move, the rest of the slab stays as it was."""
    S, L, H, C, D = 1, 2, 2, 1200, 128
    n, N = [1200], [800]
    k, v = make_cache(S, L, H, C, D, torch.bfloat16, n, seed=34)
    U = S * L * H
    rng = np.random.default_rng(35)
    frac = [0.2, 0.5, 0.9, 1.0]   # of slots kept: few movers ... no holes
    keep = torch.zeros((U, C), dtype=torch.uint8)
    for u in range(U):
        keep[u, :n[0]] = torch.from_numpy((rng.random(n[0]) < frac[u]).astype(np.uint8))
    keep = keep.to(DEV)
    pos = torch.arange(C, dtype=torch.int32, device=DEV).repeat(U, 1).contiguous()
    pre_k, pre_v, pre_pos = units(to_np(k)), units(to_np(v)), to_np(pos)
    vd.vd_compact(k, v, keep, n, N, pos)
    torch.cuda.synchronize()
    post_k, post_v, post_pos = units(to_np(k)), units(to_np(v)), to_np(pos)
    kn = to_np(keep)
    for u in range(U):
        rk, rv, rp = pre_k[u].copy(), pre_v[u].copy(), pre_pos[u].copy()
        orc.compact(rk, rv, n[0], N[0], kn[u, :n[0]], rp)
        assert np.array_equal(post_k[u].view(np.uint8), rk.view(np.uint8)), f"K of unit {u}"
        assert np.array_equal(post_v[u].view(np.uint8), rv.view(np.uint8)), f"V of unit {u}"
        assert np.array_equal(post_pos[u], rp), f"pos of unit {u}"


# ------------------------------------------------------------------ vd_evict_step

@pytest.mark.parametrize("dt", list(DTYPES))
@pytest.mark.parametrize("D", [64, 128, 256])
@pytest.mark.parametrize("variant", ALL_VARIANTS)
def test_step_matches_oracle(orc, dt, D, variant):
    """Prefill boundary, decode step and no-op units in one launch."""
    dtype = DTYPES[dt]
    rep = run_step_case(orc, 3, 2, 2, 1300, D, dtype, n=[1300, 801, 300], N=[1000, 800, 400],
                        variant=variant, seed=40 + D)
    assert rep.near_ties <= 2, rep


@pytest.mark.parametrize("dt", list(DTYPES))
@pytest.mark.parametrize("state", ["zero", "incremental"])
@pytest.mark.parametrize("variant", ALL_VARIANTS)
def test_step_with_running_sum(orc, dt, state, variant):
    dtype = DTYPES[dt]
    n, N = [1300, 801, 300, 650], [1000, 800, 400, 640]
    count = [1000, 800, 200, 600]   # crossing fill in the last sequence
    rep = run_step_case(orc, 4, 2, 2, 1300, 128, dtype, n, N, variant, seed=60,
                        state=state, count=count)
    assert rep.near_ties <= 2, rep


@pytest.mark.parametrize("dt,shift", [("f32", 1.0e4), ("f32", -3.0e5), ("bf16", 256.0)])
@pytest.mark.parametrize("state", ["none", "incremental"])
def test_l2_far_from_the_origin(orc, dt, shift, state):
    """L2 scores are invariant under a common shift of the value rows (Sec.
    3.2, Eq. vd): with every row moved far from the origin the GPU's scores
    still meet the relative bar with the absolute floor at 1e-6 of the largest
    score, because the mean is subtracted as a pair of fp32 numbers (an fp32
    mean alone would be off by 2^-24 * |shift| per channel, about 1e-4 of a
    score here)."""
    dtype = DTYPES[dt]
    S, L, H, C, D = 2, 1, 3, 1200, 128
    n, N, count = [1200, 1001], [1000, 1000], [1000, 1000]
    k, v = make_cache(S, L, H, C, D, dtype, n, seed=150)
    v[:] = (v.float() + shift).to(dtype)   # rows past n stay NaN
    U = S * L * H
    pre_k, pre_v = units(to_np(k)), units(to_np(v))
    rs = None if state == "none" else state_for(pre_v, per_unit(count, L, H), D)
    scores = torch.full((U, C), -1.0, device=DEV)
    keep = torch.zeros((U, C), dtype=torch.uint8, device=DEV)
    vd.vd_evict_step(k, v, n, N, "l2", running_sum=rs, scores_out=scores, keep_out=keep)
    torch.cuda.synchronize()
    rep = compare_pass(orc, pre_k, pre_v, units(to_np(k)), units(to_np(v)), per_unit(n, L, H),
                       per_unit(N, L, H), "l2", dtype, scores_gpu=to_np(scores),
                       keep_gpu=to_np(keep), state=to_np(rs) if rs is not None else None)
    assert rep.near_ties <= 2, rep


@pytest.mark.parametrize("dt,D,variant", [("bf16", 128, "l2"), ("f32", 256, "dir"), ("bf16", 64, "norm"),
                                         ("bf16", 128, "key_norm")])
def test_step_at_maximum_capacity(orc, dt, D, variant):
    """n at the ABI's slot limit (16384): every wave's selection segment is
    full, the keys fill 64 KB of LDS and nothing is staged; one unit evicts a
    quarter, one keeps all but one (decode argmin), one crosses the fill."""
    C = vd.MAX_CAPACITY
    n, N = [C, C, C], [12288, C - 1, 16000]
    rep = run_step_case(orc, 3, 1, 1, C, D, DTYPES[dt], n, N, variant, seed=130 + D,
                        state="incremental", count=[12288, C - 1, 9000])
    assert rep.near_ties <= 2, rep


@pytest.mark.parametrize("dt", list(DTYPES))
@pytest.mark.parametrize("state", ["none", "incremental"])
@pytest.mark.parametrize("variant", ALL_VARIANTS)
def test_step_partial_staging(orc, dt, state, variant):
    """Rows to stage (the appended part, or all n rows without a state) that do
    not all fit in LDS at head_dim 256: the first ones are staged and the rest
    is streamed twice (for the mean, then for the scores)."""
    n, N, count = [600, 450], [400, 300], [300, 100]
    rep = run_step_case(orc, 2, 1, 2, 600, 256, DTYPES[dt], n, N, variant, seed=140,
                        state=state, count=count if state != "none" else None)
    assert rep.near_ties <= 2, rep


def test_step_without_k_and_nhd_layout(orc):
    run_step_case(orc, 2, 3, 4, 700, 128, torch.bfloat16, [700, 650], [512, 600], "l2",
                  seed=71, layout="nhd")
    run_step_case(orc, 2, 1, 2, 700, 64, torch.float32, [700, 650], [512, 600], "dir",
                  seed=72, k_present=False)


def test_step_many_sequences(orc):
    """More sequences than one launch carries (the library splits the batch)."""
    S = 300
    n = [(s * 7) % 50 + 1 for s in range(S)]
    N = [max(1, (s * 3) % 40) for s in range(S)]
    run_step_case(orc, S, 1, 2, 50, 64, torch.float32, n, N, "l2", seed=80,
                  state="incremental", count=[min(x, y) for x, y in zip(n, N)])


@pytest.mark.parametrize("variant", VARIANTS)
def test_step_ties_zero_and_duplicate_rows(orc, variant):
    S, L, H, C, D = 1, 1, 3, 900, 128
    n, N = [900], [600]
    k, v = make_cache(S, L, H, C, D, torch.bfloat16, n, seed=90)
    v[0, 0, 0] = v[0, 0, 0, 5]           # unit 0: all rows equal -> keeps [0, N)
    v[0, 0, 1, ::3] = 0.0                # unit 1: zero rows (Dir convention)
    v[0, 0, 2, 1::2] = v[0, 0, 2, 0::2][: v[0, 0, 2, 1::2].shape[0]]  # unit 2: pairs of duplicates
    U = S * L * H
    pre_k, pre_v = units(to_np(k)), units(to_np(v))
    scores = torch.zeros((U, C), device=DEV)
    keep = torch.zeros((U, C), dtype=torch.uint8, device=DEV)
    vd.vd_evict_step(k, v, n, N, variant, scores_out=scores, keep_out=keep)
    torch.cuda.synchronize()
    kg = to_np(keep)
    assert np.array_equal(np.flatnonzero(kg[0, :900]), np.arange(600)), "all-equal rows"
    sg = to_np(scores)
    # duplicates score identically and the lower slot of an equal pair is never evicted alone
    assert np.array_equal(sg[2, 0:898:2], sg[2, 1:899:2])
    assert not np.any((kg[2, 1:899:2] == 1) & (kg[2, 0:898:2] == 0))
    compare_pass(orc, pre_k, pre_v, units(to_np(k)), units(to_np(v)), per_unit(n, L, H),
                 per_unit(N, L, H), variant, torch.bfloat16, scores_gpu=sg, keep_gpu=kg)


@pytest.mark.parametrize("variant", ["l2", "norm"])
def test_step_clustered_scores_with_outliers(orc, variant):
    """A few huge and tiny rows stretch the key range, so the bin holding the
    threshold after the first histogram pass still holds hundreds of keys and
    the selection narrows it again."""
    S, L, H, C, D = 1, 1, 2, 2000, 128
    n, N = [2000], [1000]
    k, v = make_cache(S, L, H, C, D, torch.float32, n, seed=97, nan_tail=False)
    g = torch.Generator(device="cpu").manual_seed(98)
    big = (torch.randn(5, D, generator=g) * 1e3).to(DEV)
    v[0, 0, 0, 0:10:2] = big                 # +x and -x pairs keep the mean small
    v[0, 0, 0, 1:10:2] = -big
    v[0, 0, 0, 10:15] = (torch.randn(5, D, generator=g) * 1e-4).to(DEV)
    U = S * L * H
    pre_k, pre_v = units(to_np(k)), units(to_np(v))
    scores = torch.zeros((U, C), device=DEV)
    keep = torch.zeros((U, C), dtype=torch.uint8, device=DEV)
    vd.vd_evict_step(k, v, n, N, variant, scores_out=scores, keep_out=keep)
    torch.cuda.synchronize()
    kg = to_np(keep)
    assert kg[0, :10].all(), "the outlier rows score highest"
    compare_pass(orc, pre_k, pre_v, units(to_np(k)), units(to_np(v)), per_unit(n, L, H),
                 per_unit(N, L, H), variant, torch.float32, scores_gpu=to_np(scores),
                 keep_gpu=kg)


def test_step_tiny_units(orc):
    """n = 0, n = 1, N = 1 and n == N in one launch."""
    run_step_case(orc, 5, 1, 1, 8, 64, torch.float32, n=[0, 1, 2, 8, 5], N=[1, 1, 1, 8, 2],
                  variant="l2", seed=95, state="zero")


@pytest.mark.parametrize("variant", KEY_VARIANTS)
def test_key_side_reads_keys_and_moves_values_along(orc, variant):
    """A key-side pass scores K (V holds rows that would keep another set) and
    moves V, K and pos together; KeyNorm at n = N + 1 evicts the largest key
    norm, the highest slot among equal ones."""
    S, L, H, C, D = 2, 1, 2, 900, 128
    n, N = [900, 801], [700, 800]
    k, v = make_cache(S, L, H, C, D, torch.bfloat16, n, seed=160)
    v[:, :, :, :, 0] = v[:, :, :, :, 0] * 50.0   # value scores would differ wildly
    k[1, 0, 1, 3] = k[1, 0, 1, 3] * 4.0          # unit 3: the largest key norm at slot 3 ...
    k[1, 0, 1, 800] = k[1, 0, 1, 3]              # ... and an equal one at the new slot 800
    U = S * L * H
    pre_k, pre_v = units(to_np(k)), units(to_np(v))
    pos = torch.arange(C, dtype=torch.int32, device=DEV).repeat(U, 1).contiguous()
    scores = torch.zeros((U, C), device=DEV)
    keep = torch.zeros((U, C), dtype=torch.uint8, device=DEV)
    vd.vd_evict_step(k, v, n, N, variant, pos=pos, scores_out=scores, keep_out=keep)
    torch.cuda.synchronize()
    rep = compare_pass(orc, pre_k, pre_v, units(to_np(k)), units(to_np(v)), per_unit(n, L, H),
                       per_unit(N, L, H), variant, torch.bfloat16, scores_gpu=to_np(scores),
                       keep_gpu=to_np(keep), pre_pos=np.tile(np.arange(C, dtype=np.int32), (U, 1)),
                       post_pos=to_np(pos))
    assert rep.near_ties == 0, rep
    if variant == "key_norm":   # unit 3: the highest slot of the two largest norms goes
        kg = to_np(keep)[3, :801]
        assert kg[3] == 1 and kg[800] == 0 and kg.sum() == 800


def test_key_norm_fused_equals_separate_calls_on_negated_scores(orc):
    """KeyNorm through the separate calls: vd_score gives the norms, and
    vd_select_topn on their negatives keeps the smallest (equal norms to the
    lower slot), so that vd_compact then leaves the fused pass's caches."""
    S, L, H, C, D = 2, 2, 2, 1100, 64
    n, N = [1100, 901], [800, 900]
    k1, v1 = make_cache(S, L, H, C, D, torch.float32, n, seed=170)
    k1[:, :, :, 5] = k1[:, :, :, 9]   # equal norms
    k2, v2 = k1.clone(), v1.clone()
    U = S * L * H
    s1 = torch.zeros((U, C), device=DEV)
    kp1 = torch.zeros((U, C), dtype=torch.uint8, device=DEV)
    vd.vd_evict_step(k1, v1, n, N, "key_norm", scores_out=s1, keep_out=kp1)
    s2, _ = vd.vd_score(v2, n, "key_norm", k=k2)
    kp2 = vd.vd_select_topn(v2, (-s2).contiguous(), n, N)
    vd.vd_compact(k2, v2, kp2, n, N)
    torch.cuda.synchronize()
    nu = per_unit(n, L, H)
    for u in range(U):
        assert torch.equal(s1[u, :nu[u]], s2[u, :nu[u]])
        assert torch.equal(kp1[u, :nu[u]], kp2[u, :nu[u]])
    assert torch.equal(k1.view(torch.int32), k2.view(torch.int32))   # bits: tails hold NaN
    assert torch.equal(v1.view(torch.int32), v2.view(torch.int32))


def test_fused_equals_separate_calls(orc):
    S, L, H, C, D = 2, 2, 2, 1100, 128
    n, N = [1100, 900], [800, 899]
    k1, v1 = make_cache(S, L, H, C, D, torch.bfloat16, n, seed=110)
    k2, v2 = k1.clone(), v1.clone()
    U = S * L * H
    s1 = torch.zeros((U, C), device=DEV)
    kp1 = torch.zeros((U, C), dtype=torch.uint8, device=DEV)
    vd.vd_evict_step(k1, v1, n, N, "l2", scores_out=s1, keep_out=kp1)
    s2, _ = vd.vd_score(v2, n, "l2")
    kp2 = vd.vd_select_topn(v2, s2, n, N)
    vd.vd_compact(k2, v2, kp2, n, N)
    torch.cuda.synchronize()
    nu = per_unit(n, L, H)
    for u in range(U):
        assert torch.equal(s1[u, :nu[u]], s2[u, :nu[u]])
        assert torch.equal(kp1[u, :nu[u]], kp2[u, :nu[u]])
    assert torch.equal(k1.view(torch.int16), k2.view(torch.int16))
    assert torch.equal(v1.view(torch.int16), v2.view(torch.int16))


def test_repeat_runs_are_bitwise_identical():
    S, L, H, C, D = 2, 4, 2, 2600, 128
    n, N = [2600, 2049], [2048, 2048]
    outs = []
    for _ in range(2):
        k, v = make_cache(S, L, H, C, D, torch.bfloat16, n, seed=120)
        rs = torch.zeros((S * L * H, D + 1), dtype=torch.float64, device=DEV)
        sc = torch.zeros((S * L * H, C), device=DEV)
        vd.vd_evict_step(k, v, n, N, "l2", running_sum=rs, scores_out=sc)
        torch.cuda.synchronize()
        outs.append((k.clone(), v.clone(), rs.clone(), sc.clone()))
    for a, b in zip(*outs):
        assert torch.equal(a.view(torch.uint8) if a.dtype == torch.bfloat16 else a,
                           b.view(torch.uint8) if b.dtype == torch.bfloat16 else b)


def test_stream_read_reads_every_word():
    # the sink is written iff the XOR of all words read is a fixed constant
    magic = 0x9E3779B9
    for words, planted in ((4, True), (4 * 1000003, True), (4 * 1000003, False)):
        buf = torch.zeros(words, dtype=torch.int32, device=DEV)
        if planted:
            buf[-1] = magic - (1 << 32)      # the last word carries the constant
        buf[0] = buf[words // 2] = 12345      # equal words in two places cancel
        sink = torch.zeros(1, dtype=torch.int32, device=DEV)
        vd.vd_stream_read(buf, sink)
        torch.cuda.synchronize()
        assert (int(sink.item()) & 0xFFFFFFFF) == (magic if planted else 0)
