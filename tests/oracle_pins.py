"""Pins of the C oracle: checks against what the paper and the mathematics fix.

None of these checks reuses the oracle's own arithmetic.  Each check takes an
``oracle.Oracle`` so that the same checks also run against deliberately
mutated builds of ``oracle/vdref.c`` (see ``test_oracle_mutants.py``): every
plausible mistake planted there must fail at least one check here.

Pins and what they fix:
  worked examples     hand-derived exact values, Sec. 3.2 Eq. vd / Sec. 2.1 Eq. eviction
  min. disturbance    (n-1)^2 ||o* - o*_{\\j}||^2 = s_j^2, Sec. 3.3 Eq. recon_error
  law of cosines      links L2, Dir and Norm, Sec. 3.2 Eq. decomp
  Dirichlet           Monte Carlo of App. A Eq. app_claim (closed form with C(n))
  invariances         translation (L2), scale, permutation (Sec. 3.3, symmetric point)
  selection           stable sort, brute force over subsets, n = N + 1, n <= N
  compaction          row multiset / pairing / slot-reuse layout properties
  decoding            bf16 and fp32 element values against torch's conversion
  geometry            sigma_K / sigma_V / bos-cosim (Sec. 3.1, Sec. 4): hand values,
                      closed forms, invariances and special cases
  attention           decode attention (Sec. 2.1, Eq. attention): zero query = mean,
                      one row, hand weights 1/4 and 3/4, scale, overflow-free one-hot,
                      key shift, permutation, bf16
  key side            the three scores on the key rows (Sec. 4, Baselines): hand kept
                      sets with values that would keep other sets, KeyNorm keeping the
                      smallest norms, the law of cosines on K, K and V moved together
  FastCAOTE           App. A, Eq. app_fastcaote: uniform attention collapses to the
                      L2 score / (n - 1) (App. A, the max-entropy limit), hand values
                      with weights 1/4 and 3/4 and a two-head mean, one-hot, key shift,
                      permutation, scale, bf16
"""
import itertools
import json
import os
from fractions import Fraction

import numpy as np

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden",
                      "worked_examples.json")


# ---------------------------------------------------------------- helpers

def _f32(a):
    return np.ascontiguousarray(np.asarray(a, dtype=np.float32))


def _rel_close(a, b, rtol, atol=0.0):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    return np.all(np.abs(a - b) <= rtol * np.abs(b) + atol)


def _frac(s: str) -> float:
    if "sqrt2" in s:  # only the form "1-1/sqrt2" appears
        assert s == "1-1/sqrt2"
        return 1.0 - 1.0 / np.sqrt(2.0)
    return float(Fraction(s))


def _kept_list(keep):
    return sorted(int(j) for j in np.flatnonzero(np.asarray(keep)))


def check_decode(orc):
    """bf16 / fp32 elements decode to the values torch's own conversion gives."""
    import torch
    rng = np.random.default_rng(11)
    bits = rng.integers(0, 1 << 16, size=4096, dtype=np.uint32).astype(np.uint16)
    bits = bits[(bits & 0x7F80) != 0x7F80]  # finite values only
    bits = np.concatenate([bits, np.array([0x3F80, 0xC000, 0x0001, 0x8000, 0x7F7F],
                                          dtype=np.uint16)])
    got = orc.decode_elems(bits)
    ref = torch.from_numpy(bits.view(np.int16).copy()).view(torch.bfloat16).double().numpy()
    assert np.array_equal(got, ref), "bf16 decoding differs from torch"
    assert got[-5] == 1.0 and got[-4] == -2.0
    f = rng.standard_normal(257).astype(np.float32)
    assert np.array_equal(orc.decode_elems(f), f.astype(np.float64))


def check_mean_library(orc):
    """The mean is numpy's mean of the decoded rows (a library routine)."""
    rng = np.random.default_rng(12)
    for n, d in ((1, 3), (7, 5), (300, 64)):
        v = _f32(rng.standard_normal((n, d)) * 3.0)
        assert _rel_close(orc.mean(v), v.astype(np.float64).mean(axis=0), 1e-12, 1e-14)
        b = (v.view(np.uint32) >> 16).astype(np.uint16)
        vb = (b.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
        assert _rel_close(orc.mean(b), vb.mean(axis=0), 1e-12, 1e-14)


def check_worked_examples(orc):
    """Hand-worked examples W1-W5 (exact values derived from the definitions)."""
    with open(GOLDEN) as fh:
        ex = json.load(fh)["examples"]
    for e in ex:
        v = _f32(e["v"])
        n = v.shape[0]
        s, m = orc.score(v, "l2")
        assert _rel_close(m, [_frac(x) for x in e["mean"]], 1e-15, 1e-15), e["name"]
        assert _rel_close(s ** 2, [_frac(x) for x in e["l2_sq"]], 1e-13, 1e-15), e["name"]
        if "norm_sq" in e:
            sn, _ = orc.score(v, "norm")
            assert _rel_close(sn ** 2, [_frac(x) for x in e["norm_sq"]], 1e-13, 1e-15)
        if "dir_one_minus_cos" in e:
            sd, _ = orc.score(v, "dir")
            assert _rel_close(sd, [_frac(x) for x in e["dir_one_minus_cos"]], 1e-12, 1e-12)
        ties = e.get("exact_tie", {})
        for variant, by_n in e["kept"].items():
            sv, _ = orc.score(v, variant)
            for N_s, want in by_n.items():
                got = _kept_list(orc.select_topn(sv, int(N_s)))
                tie = ties.get(variant, {}).get(N_s)
                if tie is None:
                    assert got == want, (e["name"], variant, N_s, got, want)
                else:  # exact tie at 0 in exact arithmetic: fp64 may order it either way
                    common = sorted(set(want) - set(tie))
                    assert set(common) <= set(got) and len(got) == len(want), (e["name"], got)
                    assert len(set(got) & set(tie)) == len(set(want) & set(tie))
        if "uniform_disturbance_times_n_minus_1_sq" in e:
            assert _rel_close(s ** 2, [_frac(x) for x in
                                       e["uniform_disturbance_times_n_minus_1_sq"]], 1e-13)
        if "post_v" in e:
            N = e["N"]
            k = _f32(np.stack([np.arange(n), -np.arange(n)], axis=1))
            vv = v.copy()
            pos = np.arange(n, dtype=np.int32)
            kk, vv2, pp = k[None].copy(), vv[None].copy(), pos[None].copy()
            _, keep, _ = orc.evict_step(kk, vv2, [n], [N], "l2", pos=pp)
            assert np.array_equal(vv2[0, :N], _f32(e["post_v"])), e["name"]
            assert pp[0, :N].tolist() == e["post_pos"], e["name"]
            assert kk[0, :N, 0].tolist() == e["post_pos"], e["name"]
            assert _kept_list(keep[0, :n]) == e["kept"]["l2"][str(N)]


def check_minimal_disturbance(orc):
    """Sec. 3.3, Eqs. uniform_outputs / recon_error by brute force: evict each
    token in turn, take the uniform-attention output (the mean) before and after,
    and compare (n-1)^2 ||o* - o*_{\\j}||^2 with s_j^2; the argmin is the
    ValueDiff argmin (Prop. vdiff_optimum)."""
    rng = np.random.default_rng(13)
    for trial in range(40):
        n = int(rng.integers(2, 14))
        d = int(rng.integers(1, 6))
        v = _f32(rng.standard_normal((n, d)) * rng.uniform(0.1, 10.0) + rng.normal(0, 3, d))
        x = v.astype(np.float64)
        s, _ = orc.score(v, "l2")
        o_all = x.sum(axis=0) / n
        dist = np.empty(n)
        for j in range(n):
            rest = np.delete(x, j, axis=0)
            o_j = rest.sum(axis=0) / (n - 1)
            dist[j] = ((o_all - o_j) ** 2).sum() * (n - 1) ** 2
        assert _rel_close(s ** 2, dist, 1e-9, 1e-12 * dist.max()), trial
        if np.sort(dist)[1] > np.sort(dist)[0] * (1 + 1e-6):
            assert int(np.argmin(s)) == int(np.argmin(dist))


def check_law_of_cosines(orc):
    """Sec. 3.2 Eq. decomp: s_L2^2 = s_Norm^2 - 2 s_Norm ||v_bar|| (1 - s_Dir) + ||v_bar||^2."""
    rng = np.random.default_rng(14)
    for trial in range(30):
        n = int(rng.integers(2, 40))
        d = int(rng.choice([1, 2, 3, 8, 64]))
        v = _f32(rng.standard_normal((n, d)) + rng.normal(0, 2, d))
        if trial % 5 == 0:
            v[0] = 0.0  # exercises the zero-norm convention for Dir
        s2, m = orc.score(v, "l2")
        sd, _ = orc.score(v, "dir")
        sn, _ = orc.score(v, "norm")
        mn = np.sqrt((m ** 2).sum())
        rhs = sn ** 2 - 2.0 * sn * mn * (1.0 - sd) + mn ** 2
        scale = (sn ** 2 + mn ** 2).max()
        assert np.all(np.abs(s2 ** 2 - rhs) <= 1e-11 * scale), trial


def check_dirichlet(orc):
    """App. A Eq. app_claim by Monte Carlo: with alpha ~ Dirichlet(1,...,1),
    E[(a_j/(1-a_j))^2 ||v_j - o(a)||^2] = 2/(n(n-1)) s_j^2 + C(n),
    C(n) = 2 (S_2 - n ||v_bar||^2) / (n^2 (n-1)(n+1))."""
    rng = np.random.default_rng(15)
    n, d, M = 6, 3, 400_000
    v = _f32(rng.standard_normal((n, d)) * 2.0 + 1.0)
    x = v.astype(np.float64)
    s, m = orc.score(v, "l2")
    S2 = (x ** 2).sum()
    C = 2.0 * (S2 - n * (m ** 2).sum()) / (n ** 2 * (n - 1) * (n + 1))
    want = 2.0 / (n * (n - 1)) * s ** 2 + C
    alpha = rng.dirichlet(np.ones(n), size=M)          # [M, n]
    o = alpha @ x                                       # [M, d]
    for j in range(n):
        w = (alpha[:, j] / (1.0 - alpha[:, j])) ** 2
        g = w * ((x[j] - o) ** 2).sum(axis=1)
        se = g.std() / np.sqrt(M)
        assert abs(g.mean() - want[j]) < 6.0 * se + 1e-12, (j, g.mean(), want[j], se)


def check_invariances(orc):
    """Translation invariance of L2 scores, scale behaviour of all three
    variants, permutation equivariance (integer-valued fp32 data: exact)."""
    rng = np.random.default_rng(16)
    for trial in range(20):
        n = int(rng.integers(2, 30))
        d = int(rng.integers(1, 9))
        v = _f32(rng.integers(-8, 9, size=(n, d)))
        c = _f32(rng.integers(-50, 51, size=d))
        s, _ = orc.score(v, "l2")
        st, _ = orc.score(_f32(v + c), "l2")
        assert _rel_close(st, s, 1e-12, 1e-12), trial
        for a in (2.0, -3.0):
            for var, f in (("l2", abs(a)), ("norm", abs(a)), ("dir", 1.0)):
                s0, _ = orc.score(v, var)
                s1, _ = orc.score(_f32(v * a), var)
                assert _rel_close(s1, f * s0, 1e-12, 1e-12), (trial, var, a)
        perm = rng.permutation(n)
        for var in ("l2", "dir", "norm"):
            s0, _ = orc.score(v, var)
            s1, _ = orc.score(_f32(v[perm]), var)
            assert _rel_close(s1, s0[perm], 1e-12, 1e-12), (trial, var)


def check_select_vs_sort(orc):
    """Top-N equals the first N of a stable sort by descending score (Python's
    sorted is stable, so equal scores keep ascending slot order)."""
    rng = np.random.default_rng(17)
    for trial in range(60):
        n = int(rng.integers(1, 200))
        N = int(rng.integers(1, n + 3))
        s = rng.integers(0, 6, size=n).astype(np.float64) if trial % 2 else rng.random(n)
        order = sorted(range(n), key=lambda j: -s[j])
        want = sorted(order[:min(N, n)])
        assert _kept_list(orc.select_topn(s, N)) == want, trial


def check_select_bruteforce(orc):
    """For n <= 9: the kept set is the N-subset of largest score sum, and among
    those the one whose sorted slot list is lexicographically smallest."""
    rng = np.random.default_rng(18)
    for trial in range(40):
        n = int(rng.integers(2, 10))
        s = rng.integers(0, 4, size=n).astype(np.float64)
        for N in range(1, n):
            best = None
            for sub in itertools.combinations(range(n), N):
                key = (-sum(s[list(sub)]), list(sub))
                if best is None or key < best:
                    best = key
            assert _kept_list(orc.select_topn(s, N)) == best[1], (trial, N)


def check_select_special(orc):
    """n = N + 1 evicts the argmin, the highest slot among equal minima;
    n <= N keeps everything; all-equal scores keep slots [0, N)."""
    rng = np.random.default_rng(19)
    for trial in range(30):
        n = int(rng.integers(2, 50))
        s = rng.integers(0, 3, size=n).astype(np.float64)
        keep = orc.select_topn(s, n - 1)
        evicted = [j for j in range(n) if not keep[j]]
        mins = [j for j in range(n) if s[j] == s.min()]
        assert evicted == [max(mins)], trial
        assert orc.select_topn(s, n).all() and orc.select_topn(s, n + 5).all()
        eq = orc.select_topn(np.full(n, 2.5), n // 2 + 1)
        assert _kept_list(eq) == list(range(n // 2 + 1))
    v = _f32(np.tile([1.0, -2.0, 0.5], (9, 1)))
    for var in ("l2", "dir", "norm"):
        s, _ = orc.score(v, var)
        assert _kept_list(orc.select_topn(s, 4)) == [0, 1, 2, 3], var


def _check_layout(pre_ids, post_ids, keep, n, N):
    """Slot-reuse layout properties for one unit; ids identify original slots."""
    kept = [j for j in range(n) if keep[j]]
    if n <= N:
        assert list(post_ids[:n]) == list(pre_ids[:n])
        return
    assert len(kept) == N
    assert sorted(post_ids[:N]) == sorted(pre_ids[j] for j in kept)
    holes = [j for j in range(N) if not keep[j]]
    movers = [j for j in range(N, n) if keep[j]]
    assert len(holes) == len(movers)
    for j in range(N):
        if keep[j]:
            assert post_ids[j] == pre_ids[j]  # surviving old slots stay put
    for h, m in zip(holes, movers):
        assert post_ids[h] == pre_ids[m]


def check_compact(orc):
    """Compaction invariants on random masks; K, V and pos stay paired."""
    rng = np.random.default_rng(20)
    for trial in range(50):
        n = int(rng.integers(1, 80))
        N = int(rng.integers(1, n + 3))
        d = int(rng.integers(1, 5))
        keep = np.zeros(n, np.uint8)
        keep[rng.permutation(n)[:min(N, n)]] = 1
        ids = np.arange(n)
        k = _f32(np.repeat(ids[:, None], d, axis=1) * 2.0)
        v = _f32(np.repeat(ids[:, None], d, axis=1) * -1.0)
        pos = (ids + 1000).astype(np.int32)
        orc.compact(k, v, n, N, keep, pos)
        _check_layout(ids, (k[:, 0] / 2).astype(int), keep, n, N)
        _check_layout(ids, (-v[:, 0]).astype(int), keep, n, N)
        _check_layout(ids, pos - 1000, keep, n, N)
        assert np.all(k[:, :1] == k) and np.all(v[:, :1] == v)


def check_evict_step_batch(orc):
    """The batched pass: per-unit n and N, ragged units, both dtypes; kept sets
    follow the scores, the layout follows the slot-reuse rule, units stay apart."""
    rng = np.random.default_rng(21)
    for dt in ("f32", "bf16"):
        U, cap, d = 7, 40, 6
        x = rng.standard_normal((U, cap, d)).astype(np.float32)
        v = x if dt == "f32" else (x.view(np.uint32) >> 16).astype(np.uint16)
        v = np.ascontiguousarray(v)
        n_unit = rng.integers(0, cap + 1, size=U).astype(np.int32)
        n_unit[0], n_unit[1] = cap, 1
        N_unit = rng.integers(1, cap, size=U).astype(np.int32)
        ids = np.broadcast_to(np.arange(cap, dtype=np.int32), (U, cap)).copy()
        k = np.ascontiguousarray(np.broadcast_to(ids[:, :, None], (U, cap, d))
                                 .astype(np.float32))
        if dt == "bf16":
            k = (k.view(np.uint32) >> 16).astype(np.uint16)  # small ints are exact
        v_pre = v.copy()
        pos = ids.copy()
        scores, keep, means = orc.evict_step(k, v, n_unit, N_unit, "l2", pos=pos)
        for u in range(U):
            n, N = int(n_unit[u]), int(N_unit[u])
            if n == 0:
                continue
            s_u, m_u = orc.score(v_pre[u, :n], "l2")
            assert np.array_equal(scores[u, :n], s_u)
            assert np.array_equal(means[u], m_u)
            assert np.array_equal(keep[u, :n], orc.select_topn(s_u, N))
            _check_layout(np.arange(cap), pos[u], keep[u], n, N)
            kd = orc.decode_elems(k[u, :, 0]).astype(int)
            assert np.array_equal(kd, pos[u])
            for slot in range(min(n, N)):
                assert np.array_equal(v[u, slot], v_pre[u, pos[u, slot]])
            assert np.array_equal(v[u, n:], v_pre[u, n:])  # beyond n: untouched


def check_geometry(orc):
    """sigma_X = std_i ||x_i - x_bar|| (population std) and bos-cosim =
    cos(k_0, mean of k_1..k_{n-1}) against values derived by hand and
    properties that fix them."""
    r2 = np.sqrt(2.0)
    # W1 rows as V, W2 rows as K: distances V [r2, 1, 1, 2 r2], K [1, 1, 0, r2];
    # content mean of K = (1, 4/3), so bos-cosim = 1 / (5/3)
    V = _f32([[0, 0], [1, 0], [0, 1], [3, 3]])
    K = _f32([[1, 0], [0, 1], [1, 1], [2, 2]])
    mu_v, mu_k = (2 + 3 * r2) / 4, (2 + r2) / 4
    want = [np.sqrt(1.0 - mu_k ** 2), np.sqrt(3.0 - mu_v ** 2), mu_k, mu_v, 0.6]
    assert _rel_close(orc.geometry(K, V), want, 1e-12), orc.geometry(K, V)
    # one channel, rows -2, -1, 1, 2: distances 2, 1, 1, 2 -> mean 1.5, population std 0.5
    x = _f32([[-2], [-1], [1], [2]])
    g = orc.geometry(x, x)
    assert _rel_close(g[:4], [0.5, 0.5, 1.5, 1.5], 1e-12), g
    # two rows: both at half their distance from the mean, so sigma = 0
    g = orc.geometry(_f32([[0, 0], [3, 4]]), _f32([[1, 1], [1, 1]]))
    assert _rel_close(g[:4], [0.0, 0.0, 2.5, 0.0], 1e-12, 1e-12), g
    # one token: nothing spreads and there is no content mean
    assert np.all(orc.geometry(_f32([[1, 2]]), _f32([[3, 4]])) == 0.0)
    # bos-cosim: k_0 against the content mean, along it, opposite, zero
    c = _f32([[1, 2], [3, 1], [2, 3]])   # content mean (2, 2)
    for k0, cos in (([4, 4], 1.0), ([-1, -1], -1.0), ([0, 0], 0.0), ([2, -2], 0.0)):
        g = orc.geometry(_f32(np.vstack([k0, c])), _f32(np.vstack([k0, c])))
        assert abs(g[4] - cos) < 1e-12, (k0, g[4])
    # invariances: translation and permutation keep sigma and the mean distance,
    # scaling by a multiplies them by |a| and keeps bos-cosim
    rng = np.random.default_rng(31)
    k = _f32(rng.standard_normal((40, 6)))
    v = _f32(rng.standard_normal((40, 6)) * 3.0)
    g = orc.geometry(k, v)
    t = _f32(k + rng.standard_normal(6).astype(np.float32) * 0.5)
    u = _f32(v + rng.standard_normal(6).astype(np.float32) * 0.5)
    assert _rel_close(orc.geometry(t, u)[:4], g[:4], 1e-5)
    perm = np.concatenate([[0], 1 + rng.permutation(39)])
    assert _rel_close(orc.geometry(k[perm], v[perm]), g, 1e-12, 1e-15)
    for a in (2.0, -0.5):
        ga = orc.geometry(_f32(k * a), _f32(v * a))
        assert _rel_close(ga[:4], np.abs(a) * g[:4], 1e-6)
        assert abs(ga[4] - g[4]) < 1e-6
    # bf16 rows give the same statistics as their fp32 values
    kb = (k.view(np.uint32) >> 16).astype(np.uint16)
    vb = (v.view(np.uint32) >> 16).astype(np.uint16)
    kf = _f32((kb.astype(np.uint32) << 16).view(np.float32))
    vf = _f32((vb.astype(np.uint32) << 16).view(np.float32))
    assert _rel_close(orc.geometry(kb, vb), orc.geometry(kf, vf), 1e-12, 1e-15)


def check_attention(orc):
    """Decode attention o = sum_j softmax_j(scale * q . k_j) v_j (Sec. 2.1,
    Eq. attention) against hand values and properties that fix it."""
    rng = np.random.default_rng(41)
    k = _f32(rng.standard_normal((30, 8)))
    v = _f32(rng.standard_normal((30, 8)) * 2.0)
    v64 = v.astype(np.float64)
    # a zero query weighs every row alike: the output is the plain mean of the rows
    o = orc.attention(np.zeros(8), k, v, 0.35)
    assert _rel_close(o, v64.sum(axis=0) / 30.0, 1e-12, 1e-14), o
    # one row: the output is that row
    assert np.array_equal(orc.attention(rng.standard_normal(8), k[:1], v[:1], 0.35), v64[0])
    # two rows with logits 0 and ln 3 weigh 1/4 and 3/4: (4, -8)/4 + 3 (0, 8)/4 = (1, 4)
    o = orc.attention(np.array([np.log(3.0), 5.0]), _f32([[0, 0], [1, 0]]),
                      _f32([[4, -8], [0, 8]]), 1.0)
    assert _rel_close(o, [1.0, 4.0], 1e-12, 1e-12), o
    # the scale multiplies the logits
    q = rng.standard_normal(8)
    a = orc.attention(q, k, v, 0.7)
    assert _rel_close(a, orc.attention(0.7 * q, k, v, 1.0), 1e-12, 1e-14)
    assert not _rel_close(a, orc.attention(q, k, v, 1.0), 1e-6)
    # one logit 1000 above the others: exactly that row, with no overflow
    big = np.zeros(8)
    big[0] = 1000.0
    kk = np.zeros((5, 8), np.float32)
    kk[2, 0] = 1.0
    assert np.array_equal(orc.attention(big, kk, v[:5], 1.0), v64[2])
    # the same shift of every key moves every logit alike: no change (integer
    # keys, so that the shifted keys are exact)
    ki = _f32(rng.integers(-4, 5, (30, 8)))
    ks = _f32(ki + rng.integers(-3, 4, 8))
    assert _rel_close(orc.attention(q, ks, v, 0.3), orc.attention(q, ki, v, 0.3), 1e-11, 1e-13)
    # rows permuted together with their values: no change
    perm = rng.permutation(30)
    assert _rel_close(orc.attention(q, k[perm], v[perm], 0.5), orc.attention(q, k, v, 0.5),
                      1e-12, 1e-14)
    # bf16 rows give the output of their fp32 values
    kb = (k.view(np.uint32) >> 16).astype(np.uint16)
    vb = (v.view(np.uint32) >> 16).astype(np.uint16)
    kf = _f32((kb.astype(np.uint32) << 16).view(np.float32))
    vf = _f32((vb.astype(np.uint32) << 16).view(np.float32))
    assert _rel_close(orc.attention(q, kb, vb, 0.5), orc.attention(q, kf, vf, 0.5), 1e-12, 1e-15)


def check_key_side(orc):
    """Key-side scores (Sec. 4, Baselines, key geometry): L2, Dir and Norm on
    the key rows, KeyNorm keeping the smallest norms, through the batched pass.
    K holds W1's rows (scores: L2 [r2, 1, 1, 2 r2], Dir [1, 1-1/r2, 1-1/r2, 0],
    norms [0, 1, 1, 3 r2]); the value rows would keep other sets."""
    K = _f32([[0, 0], [1, 0], [0, 1], [3, 3]])
    V = _f32([[1, 1], [1, 1], [0, 0], [1, 1]])
    r2 = np.sqrt(2.0)
    want_s = {"key_l2": [r2, 1, 1, 2 * r2], "key_dir": [1, 1 - 1 / r2, 1 - 1 / r2, 0],
              "key_norm": [0, 1, 1, 3 * r2]}
    want_keep = {("key_l2", 2): [0, 3], ("key_l2", 3): [0, 1, 3], ("key_dir", 2): [0, 1],
                 ("key_dir", 3): [0, 1, 2], ("key_norm", 2): [0, 1], ("key_norm", 3): [0, 1, 2]}
    for (var, N), want in want_keep.items():
        k, v = K[None].copy(), V[None].copy()
        pos = np.arange(4, dtype=np.int32)[None].copy()
        s, keep, _ = orc.evict_step(k, v, [4], [N], var, pos=pos)
        assert _rel_close(s[0, :4], want_s[var], 1e-12, 1e-12), (var, s[0, :4])
        assert _kept_list(keep[0, :4]) == want, (var, N, _kept_list(keep[0, :4]))
        for slot in range(N):   # K and V rows stay paired with their slot id
            assert np.array_equal(k[0, slot], K[pos[0, slot]]), (var, N)
            assert np.array_equal(v[0, slot], V[pos[0, slot]]), (var, N)
    # KeyNorm: n = N + 1 evicts the largest norm, the highest slot among equals
    k = _f32([[3, 4], [0, 1], [4, 3], [1, 0]])[None].copy()
    _, keep, _ = orc.evict_step(k, k.copy(), [4], [3], "key_norm")
    assert _kept_list(keep[0, :4]) == [0, 1, 3]
    # law of cosines on K (Sec. 3.2, Eq. decomp on the key side), random rows
    rng = np.random.default_rng(51)
    for trial in range(10):
        n, d = int(rng.integers(3, 40)), int(rng.choice([2, 5, 16]))
        k = _f32(rng.standard_normal((1, n, d)) + rng.normal(0, 2, d))
        v = _f32(rng.standard_normal((1, n, d)) * 3.0)
        out = {var: orc.evict_step(k.copy(), v.copy(), [n], [n], var)
               for var in ("key_l2", "key_dir", "key_norm")}
        s2, sd, sn = out["key_l2"][0][0, :n], out["key_dir"][0][0, :n], out["key_norm"][0][0, :n]
        mn = np.sqrt((out["key_l2"][2][0] ** 2).sum())
        rhs = sn ** 2 - 2.0 * sn * mn * (1.0 - sd) + mn ** 2
        assert np.all(np.abs(s2 ** 2 - rhs) <= 1e-11 * (sn ** 2 + mn ** 2).max()), trial
        assert _rel_close(out["key_l2"][2][0], k[0].astype(np.float64).mean(axis=0), 1e-12, 1e-14)


def check_fastcaote(orc):
    """FastCAOTE, s_j = a_j / (1 - a_j) * ||v_j - v_bar|| (App. A, Eq.
    app_fastcaote), a_j the softmax weight of row j averaged over the heads."""
    rng = np.random.default_rng(61)
    # uniform attention (zero queries): a_j = 1/n, so s_j = ||v_j - v_bar|| / (n - 1),
    # the ValueDiff score up to a factor that leaves its ranking unchanged (App. A)
    for n, G in ((2, 1), (7, 3), (40, 4)):
        k = _f32(rng.standard_normal((n, 5)))
        v = _f32(rng.standard_normal((n, 5)) * 2.0 + 1.0)
        s = orc.fastcaote_scores(np.zeros((G, 5)), k, v, 0.3)
        l2, _ = orc.score(v, "l2")
        assert _rel_close(s, l2 / (n - 1), 1e-12, 1e-15), (n, G)
    # two rows, logits 0 and ln 3: weights 1/4 and 3/4, ratios 1/3 and 3; the
    # values (0,0) and (2,0) lie at distance 1 from their mean (1,0)
    K = _f32([[0, 0], [1, 0]])
    V = _f32([[0, 0], [2, 0]])
    q1 = np.array([[np.log(3.0), 0.0]])
    assert _rel_close(orc.fastcaote_scores(q1, K, V, 1.0), [1 / 3, 3.0], 1e-12)
    # two heads, uniform and (1/4, 3/4): mean weights 3/8 and 5/8, ratios 3/5 and 5/3
    q2 = np.array([[0.0, 0.0], [np.log(3.0), 0.0]])
    assert _rel_close(orc.fastcaote_scores(q2, K, V, 1.0), [0.6, 5 / 3], 1e-12)
    # one logit 1000 above the rest: that row takes all the weight (+inf), the others none
    kk = np.zeros((5, 4), np.float32)
    kk[2, 0] = 1.0
    vv = _f32(rng.standard_normal((5, 4)))
    s = orc.fastcaote_scores(np.array([[1000.0, 0, 0, 0]]), kk, vv, 1.0)
    assert np.isinf(s[2]) and s[2] > 0 and np.all(s[[0, 1, 3, 4]] == 0.0), s
    # logits near 800 (past fp64's exp range) give the weights of the same
    # logits less 800 (offsets in sixteenths: exact in fp32)
    off = _f32(np.zeros((12, 3)))
    off[:, 0] = rng.integers(0, 48, 12) / 16.0
    hi = _f32(off + np.array([800.0, 0, 0], np.float32))
    vv = _f32(rng.standard_normal((12, 3)))
    qq = np.array([[1.0, 0.3, -0.2]])
    s_hi = orc.fastcaote_scores(qq, hi, vv, 1.0)
    assert np.all(np.isfinite(s_hi)), s_hi
    assert _rel_close(s_hi, orc.fastcaote_scores(qq, off, vv, 1.0), 1e-12, 1e-15)
    # the scale multiplies the logits
    q = rng.standard_normal((2, 6)) * 0.5
    kx = _f32(rng.standard_normal((20, 6)))
    vx = _f32(rng.standard_normal((20, 6)))
    a = orc.fastcaote_scores(q, kx, vx, 0.7)
    assert _rel_close(a, orc.fastcaote_scores(0.7 * q, kx, vx, 1.0), 1e-12, 1e-15)
    assert not _rel_close(a, orc.fastcaote_scores(q, kx, vx, 1.0), 1e-6)
    # invariances: a common key shift (integer keys: exact), rows permuted
    # together, values scaled by a (scores scale by |a|)
    ki = _f32(rng.integers(-3, 4, (30, 6)))
    vi = _f32(rng.standard_normal((30, 6)))
    s0 = orc.fastcaote_scores(q, ki, vi, 0.4)
    ks = _f32(ki + rng.integers(-2, 3, 6))
    assert _rel_close(orc.fastcaote_scores(q, ks, vi, 0.4), s0, 1e-10, 1e-15)
    perm = rng.permutation(30)
    assert _rel_close(orc.fastcaote_scores(q, ki[perm], vi[perm], 0.4), s0[perm], 1e-12, 1e-15)
    assert _rel_close(orc.fastcaote_scores(q, ki, _f32(vi * -2.0), 0.4), 2.0 * s0, 1e-12, 1e-15)
    # bf16 rows give the scores of their fp32 values
    kb = (ki.view(np.uint32) >> 16).astype(np.uint16)
    vb = (vi.view(np.uint32) >> 16).astype(np.uint16)
    kf = _f32((kb.astype(np.uint32) << 16).view(np.float32))
    vf = _f32((vb.astype(np.uint32) << 16).view(np.float32))
    assert _rel_close(orc.fastcaote_scores(q, kb, vb, 0.4), orc.fastcaote_scores(q, kf, vf, 0.4),
                      1e-12, 1e-15)


ALL_CHECKS = [
    check_decode, check_mean_library, check_worked_examples,
    check_minimal_disturbance, check_law_of_cosines, check_dirichlet,
    check_invariances, check_select_vs_sort, check_select_bruteforce,
    check_select_special, check_compact, check_evict_step_batch, check_geometry,
    check_attention, check_key_side, check_fastcaote,
]


def run_all(lib_path: str, fail_fast: bool = False) -> int:
    """Runs every check against one build; returns the number that failed."""
    import sys
    sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
    from oracle.vdref import Oracle
    orc = Oracle(lib_path)
    failed = 0
    for chk in ALL_CHECKS:
        try:
            chk(orc)
        except Exception as exc:  # noqa: BLE001 -- any failure counts
            failed += 1
            print(f"FAIL {chk.__name__}: {type(exc).__name__}: {str(exc)[:200]}")
            if fail_fast:
                break
    return failed


if __name__ == "__main__":
    import sys
    raise SystemExit(min(run_all(sys.argv[1], fail_fast="--fail-fast" in sys.argv), 100))
