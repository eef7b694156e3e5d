"""Helpers of the GPU parity tests: moving tensors to the oracle's numpy form
and comparing one pass of the HIP path with the oracle's pass on the same
inputs.

Bar (per unit):
  kept set    identical to the oracle's, except when the oracle's boundary is a
              near-tie: every slot on which the two sets differ must then have
              an oracle score within REL_TIE * s_(N) + atol of the N-th largest
              score s_(N); such units are counted and reported.
  caches      when the kept sets are identical, K, V and pos after the pass are
              bit-identical to the oracle's; otherwise they must hold exactly
              the rows the GPU kept, in the slot-reuse layout.
  scores      |s_gpu - s_ref| <= rtol * s_ref + atol, rtol = 1e-3 (bf16) or
              1e-5 (fp32), atol = 1e-6 * max(max_j s_ref, scale), where scale is
              1 for Dir (1 - cos is dimensionless, at most 2) and 0 for L2 and
              Norm.  (The kernels subtract the mean as a pair of fp32 numbers,
              so an L2 score keeps fp32 accuracy relative to itself however
              far the mean lies from the origin.)
  state       the running sum equals the fp64 sum of the kept rows of the
              scored tensor (V; K for a key-side score).
"""
import numpy as np
import torch

REL_TIE = 1e-5
RTOL = {torch.bfloat16: 1e-3, torch.float32: 1e-5}


def to_np(t: torch.Tensor) -> np.ndarray:
    """bf16 -> uint16 bit patterns, fp32 -> float32, other dtypes as they are."""
    t = t.detach().contiguous().cpu()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16).copy()
    return t.numpy().copy()


def from_np(a: np.ndarray, dtype, device) -> torch.Tensor:
    if dtype == torch.bfloat16:
        return torch.from_numpy(a.view(np.int16).copy()).view(torch.bfloat16).to(device)
    return torch.from_numpy(a.copy()).to(device)


def values_f64(a: np.ndarray) -> np.ndarray:
    """Element values of oracle-form rows, as float64."""
    if a.dtype == np.uint16:
        return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return a.astype(np.float64)


def units(a: np.ndarray) -> np.ndarray:
    """[S, L, H, C, D] -> [U, C, D] (C-contiguous copy)."""
    S, L, H, C, D = a.shape
    return np.ascontiguousarray(a.reshape(S * L * H, C, D))


def per_unit(vals, L, H):
    return np.repeat(np.asarray(vals, dtype=np.int32), L * H)


class Report:
    def __init__(self):
        self.units = 0
        self.near_ties = 0
        self.max_score_err = 0.0

    def __repr__(self):
        return (f"Report(units={self.units}, near_ties={self.near_ties}, "
                f"max_rel_score_err={self.max_score_err:.3g})")


def score_scale(rows, variant):
    """The `scale` of the score tolerance for one unit's rows (oracle form)."""
    return 1.0 if variant in ("dir", "key_dir") else 0.0


def check_scores(s_gpu, s_ref, dtype, what="", scale=0.0):
    s_gpu = np.asarray(s_gpu, np.float64)
    s_ref = np.asarray(s_ref, np.float64)
    atol = 1e-6 * max(np.abs(s_ref).max() if s_ref.size else 0.0, scale)
    err = np.abs(s_gpu - s_ref)
    bad = err > RTOL[dtype] * np.abs(s_ref) + atol
    assert not bad.any(), (f"{what}: {bad.sum()} scores out of tolerance; worst "
                           f"j={int(np.argmax(err))} gpu={s_gpu[np.argmax(err)]!r} "
                           f"ref={s_ref[np.argmax(err)]!r}")
    return float((err / np.maximum(np.abs(s_ref), atol + 1e-300)).max()) if s_ref.size else 0.0


def keep_agrees(keep_gpu, keep_ref, s_ref, N, what="", scale=0.0, smallest=False):
    """True if identical; False for a tolerated near-tie; asserts otherwise.
    `smallest`: the N lowest scores are kept (KeyNorm)."""
    keep_gpu = np.asarray(keep_gpu).astype(bool)
    keep_ref = np.asarray(keep_ref).astype(bool)
    if np.array_equal(keep_gpu, keep_ref):
        return True
    n = keep_ref.size
    assert keep_gpu.sum() == min(N, n), f"{what}: GPU kept {keep_gpu.sum()} of {n}, budget {N}"
    s_sorted = np.sort(s_ref) if smallest else np.sort(s_ref)[::-1]
    s_N = s_sorted[min(N, n) - 1]
    band = REL_TIE * abs(s_N) + 1e-6 * max(np.abs(s_ref).max(), scale)
    diff = np.flatnonzero(keep_gpu != keep_ref)
    far = diff[np.abs(s_ref[diff] - s_N) > band]
    assert far.size == 0, (f"{what}: kept sets differ outside the near-tie band at slots "
                           f"{far[:8].tolist()} (s={s_ref[far[:8]].tolist()}, s_N={s_N})")
    return False


def check_layout(post_rows, pre_rows, keep, n, N, what=""):
    """post_rows[:min(n,N)] hold the kept pre rows in the slot-reuse layout."""
    keep = np.asarray(keep).astype(bool)
    if n <= N:
        assert np.array_equal(post_rows[:n], pre_rows[:n]), f"{what}: rows moved without eviction"
        return
    holes = [j for j in range(N) if not keep[j]]
    movers = [j for j in range(N, n) if keep[j]]
    assert len(holes) == len(movers), what
    expect = pre_rows[:N].copy()
    for h, m in zip(holes, movers):
        expect[h] = pre_rows[m]
    assert np.array_equal(post_rows[:N], expect), f"{what}: layout differs"


def compare_pass(orc, pre_k, pre_v, post_k, post_v, n_unit, N_unit, variant, dtype,
                 scores_gpu=None, keep_gpu=None, pre_pos=None, post_pos=None,
                 state=None, unit_ids=None, report=None):
    """Runs the oracle on the pre-pass units and compares with the GPU's results.

    pre_k/pre_v/post_k/post_v : [U', C, D] oracle-form arrays of the compared units
    n_unit/N_unit             : [U'] per-unit n and N
    scores_gpu/keep_gpu       : [U', C] GPU outputs or None
    state                     : [U', D + 1] GPU running sum after the pass or None
    """
    report = report if report is not None else Report()
    ref_k = pre_k.copy() if pre_k is not None else None
    ref_v = pre_v.copy()
    ref_pos = pre_pos.copy() if pre_pos is not None else None
    ref_scores, ref_keep, _ = orc.evict_step(ref_k, ref_v, n_unit, N_unit, variant, pos=ref_pos)
    for i in range(pre_v.shape[0]):
        u = i if unit_ids is None else int(unit_ids[i])
        n, N = int(n_unit[i]), int(N_unit[i])
        what = f"unit {u} (n={n}, N={N})"
        report.units += 1
        if n == 0:
            continue
        key_side = variant.startswith("key")
        scored_pre = pre_k if key_side else pre_v
        scored_post = post_k if key_side else post_v
        scale = score_scale(scored_pre[i, :n], variant)
        if scores_gpu is not None:
            e = check_scores(scores_gpu[i, :n], ref_scores[i, :n], dtype, what, scale)
            report.max_score_err = max(report.max_score_err, e)
        if keep_gpu is not None:
            same = keep_agrees(keep_gpu[i, :n], ref_keep[i, :n], ref_scores[i, :n], N, what,
                               scale, smallest=variant == "key_norm")
            kept = keep_gpu[i, :n]
        else:
            same = True
            kept = ref_keep[i, :n]
        if not same:
            report.near_ties += 1
        m = min(n, N)
        if same:
            assert np.array_equal(post_v[i, :m], ref_v[i, :m]), f"{what}: V differs"
            if pre_k is not None:
                assert np.array_equal(post_k[i, :m], ref_k[i, :m]), f"{what}: K differs"
            if pre_pos is not None:
                assert np.array_equal(post_pos[i, :m], ref_pos[i, :m]), f"{what}: pos differs"
        else:
            check_layout(post_v[i], pre_v[i], kept, n, N, what + " V")
            if pre_k is not None:
                check_layout(post_k[i], pre_k[i], kept, n, N, what + " K")
            if pre_pos is not None:
                check_layout(post_pos[i], pre_pos[i], kept, n, N, what + " pos")
        if state is not None:   # the sum of the kept rows of the scored tensor
            want = values_f64(scored_post[i, :m]).sum(axis=0)
            got = state[i, :-1]
            assert state[i, -1] == m, f"{what}: state count {state[i, -1]} != {m}"
            tol = 1e-12 * np.abs(values_f64(scored_post[i, :m])).sum(axis=0) + 1e-300
            assert np.all(np.abs(got - want) <= tol), f"{what}: running sum differs"
    return report
