"""GPU parity of the geometry diagnostics (vd_geometry) against the oracle.

Per unit the HIP path returns sigma_K, sigma_V, the mean distances to the
centroid and bos-cosim (Sec. 3.1; Sec. 4).  Centroids and every sum over rows
are fp64 on both sides; the kernel forms each distance in fp32 from the
difference to an fp32 (hi + lo) centroid, which bounds its relative error by a
few fp32 units in the last place: rounding of the differences and squares
(about 2^-24 each) and of a sum of at most 8 terms per lane followed by a tree
of at most 6 levels, so at most about 15 * 2^-24 < 1e-6.  Hence the bar:

  mean distance   |mu_gpu - mu_ref| <= TOL * max_i d_i
  sigma           |sigma_gpu - sigma_ref| <= TOL * max_i d_i  (the standard
                  deviation moves by at most the largest change of one distance)
  bos-cosim       |c_gpu - c_ref| <= 1e-10 (fp64 throughout)

with TOL = 2e-6 and d_i the fp64 distances of the rows to their centroid.
"""
import numpy as np
import pytest
import torch

from paper_2609_23314_amd import synth, vd
from parity import to_np, units, values_f64

pytestmark = pytest.mark.gpu
DEV = "cuda"
DTYPES = {"bf16": torch.bfloat16, "f32": torch.float32}
TOL = 2e-6
BOS_TOL = 1e-10


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    vd.load()


def dmax(rows):
    x = values_f64(rows)
    if x.shape[0] == 0:
        return 0.0
    return float(np.sqrt(((x - x.mean(axis=0)) ** 2).sum(axis=1)).max())


def column_sums(x, count_unit):
    """[U, D + 1]: fp64 column sums of the first count rows of every unit and
    the count (torch on the GPU: an input of the HIP path, exact for bf16)."""
    S, L, H, C, D = x.shape
    xu = x.reshape(S * L * H, C, D)
    t = torch.zeros((S * L * H, D + 1), dtype=torch.float64, device=DEV)
    for u in range(S * L * H):
        c = int(count_unit[u])
        t[u, :D] = xu[u, :c].double().sum(dim=0)
        t[u, D] = c
    return t


def check_units(orc, k, v, n_seq, L, H, sample=None, sums=None):
    """Runs vd_geometry on [S, L, H, C, D] caches and compares every unit (or
    the sampled ones) with the oracle; `sums` = (k_sum, v_sum) or None."""
    kw = {} if sums is None else dict(k_sum=sums[0], v_sum=sums[1])
    out = vd.vd_geometry(k, v, n_seq, **kw)
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    ku, vu = units(to_np(k)), units(to_np(v))
    n_unit = np.repeat(np.asarray(n_seq, np.int64), L * H)
    idx = range(ku.shape[0]) if sample is None else sample
    for u in idx:
        n = int(n_unit[u])
        ref = orc.geometry(ku[u, :n], vu[u, :n])
        sk, sv = dmax(ku[u, :n]), dmax(vu[u, :n])
        g = got[u]
        assert abs(g[0] - ref[0]) <= TOL * sk, (u, n, "sigma_K", g[0], ref[0])
        assert abs(g[1] - ref[1]) <= TOL * sv, (u, n, "sigma_V", g[1], ref[1])
        assert abs(g[2] - ref[2]) <= TOL * sk, (u, n, "mean dist K", g[2], ref[2])
        assert abs(g[3] - ref[3]) <= TOL * sv, (u, n, "mean dist V", g[3], ref[3])
        assert abs(g[4] - ref[4]) <= BOS_TOL, (u, n, "bos-cosim", g[4], ref[4])
    return got


def make(S, L, H, C, D, dtype, n, seed, dist="normal", layout="hnd", scale=1.0):
    if layout == "hnd":
        k = synth.random_rows((S, L, H, C, D), dtype, seed, DEV, dist, scale)
        v = synth.random_rows((S, L, H, C, D), dtype, seed + 1, DEV, dist, scale)
    else:
        k = synth.random_rows((S, L, C, H, D), dtype, seed, DEV, dist, scale).permute(0, 1, 3, 2, 4)
        v = synth.random_rows((S, L, C, H, D), dtype, seed + 1, DEV, dist, scale).permute(0, 1, 3, 2, 4)
    for s in range(S):  # rows past n are never read
        k[s, :, :, n[s]:] = float("nan")
        v[s, :, :, n[s]:] = float("nan")
    return k, v


@pytest.mark.parametrize("dt", list(DTYPES))
@pytest.mark.parametrize("D", [64, 128, 256])
def test_geometry_matches_oracle(orc, dt, D):
    # several row tiles of the kernel plus a ragged tail, and a short unit
    n = [1000, 333]
    k, v = make(2, 2, 2, 1024, D, DTYPES[dt], n, seed=300 + D)
    check_units(orc, k, v, n, 2, 2)


@pytest.mark.parametrize("dt", list(DTYPES))
@pytest.mark.parametrize("D", [64, 128, 256])
def test_geometry_with_column_sums(orc, dt, D):
    """Column sums of K and V covering exactly the n rows give the centroids
    up front and one read of the rows; a unit whose sums cover fewer rows
    (here the second sequence's) takes its centroids from the rows.  Both
    meet the oracle's bar, and with bf16 rows (exact fp64 sums) the results
    equal those computed without sums bit for bit."""
    n = [1000, 333]
    k, v = make(2, 2, 2, 1024, D, DTYPES[dt], n, seed=310 + D)
    count = np.repeat([1000, 300], 4)
    sums = (column_sums(k, count), column_sums(v, count))
    got = check_units(orc, k, v, n, 2, 2, sums=sums)
    plain = vd.vd_geometry(k, v, n).cpu().numpy()
    if dt == "bf16":
        assert np.array_equal(got, plain)
    # the one-read path also on a centroid far from the origin
    k2, v2 = make(1, 1, 2, 800, 128, DTYPES[dt], [777], seed=43, dist="shifted", scale=0.05)
    c2 = np.repeat([777], 2)
    check_units(orc, k2, v2, [777], 1, 2, sums=(column_sums(k2, c2), column_sums(v2, c2)))


@pytest.mark.parametrize("dt", list(DTYPES))
def test_geometry_far_centroid(orc, dt):
    # rows far from the origin: the fp32 distance must not lose the spread
    n = [777]
    k, v = make(1, 1, 2, 800, 128, DTYPES[dt], n, seed=41, dist="shifted", scale=0.05)
    check_units(orc, k, v, n, 1, 2)


def test_geometry_tiny_and_empty_units(orc):
    n = [0, 1, 2, 3, 65]
    k, v = make(5, 1, 2, 80, 64, torch.float32, n, seed=7)
    got = check_units(orc, k, v, n, 1, 2)
    assert np.all(got[:2] == 0.0)          # n = 0: all five zero
    assert np.all(got[2:4, 4] == 0.0)      # n = 1: no bos-cosim
    assert np.all(got[2:4, :4] == 0.0)     # n = 1: the row is its centroid


def test_geometry_degenerate_rows(orc):
    # identical rows (sigma and mean distance zero), a zero first key (bos 0),
    # and a first key that is a large outlier
    S, L, H, C, D = 1, 1, 3, 300, 128
    k = torch.zeros((S, L, H, C, D), dtype=torch.bfloat16, device=DEV)
    v = torch.zeros_like(k)
    row = synth.random_rows((D,), torch.bfloat16, 5, DEV)
    k[0, 0, 0] = row
    v[0, 0, 0] = row
    k[0, 0, 1] = synth.random_rows((C, D), torch.bfloat16, 6, DEV)
    k[0, 0, 1, 0] = 0.0
    v[0, 0, 1] = synth.random_rows((C, D), torch.bfloat16, 8, DEV)
    k[0, 0, 2] = synth.random_rows((C, D), torch.bfloat16, 9, DEV, "shifted")
    k[0, 0, 2, 0] = k[0, 0, 2, 0] * 64.0
    v[0, 0, 2] = synth.random_rows((C, D), torch.bfloat16, 10, DEV)
    got = check_units(orc, k, v, [C], L, H)
    assert np.all(got[0, :4] == 0.0)
    assert got[1, 4] == 0.0


def test_geometry_strided_and_many_sequences(orc):
    # a per-layer [S, L, C, H, D] layout seen through a permuted view, and more
    # sequences than one launch takes
    S = 300
    n = [(37 * s) % 97 for s in range(S)]
    k, v = make(S, 1, 2, 96, 64, torch.bfloat16, n, seed=11, layout="nhd")
    check_units(orc, k, v, n, 1, 2)


def test_geometry_llama_prompt_sampled(orc):
    # the prefill workload's cache at the boundary (32 layers, 8 KV heads,
    # 2560 rows of 128 bf16 channels per unit, with its outlier tokens);
    # sampled units against the oracle, every unit's results finite
    w = synth.llama_prefill()
    C = w.capacity
    k, v = synth.empty_cache(w, DEV)
    k[0] = synth.block_rows(w, "k", 0, 0, 0, C, DEV)
    v[0] = synth.block_rows(w, "v", 0, 0, 0, C, DEV)
    rng = np.random.default_rng(3)
    sample = sorted(rng.choice(w.units, size=12, replace=False).tolist())
    got = check_units(orc, k, v, [C], w.num_layers, w.num_kv_heads, sample=sample)
    assert np.all(np.isfinite(got)) and np.all(got[:, :4] > 0.0)


def test_geometry_repeat_is_bitwise_identical():
    n = [900, 500]
    k, v = make(2, 2, 2, 1024, 128, torch.bfloat16, n, seed=17)
    a = vd.vd_geometry(k, v, n).cpu()
    b = vd.vd_geometry(k, v, n).cpu()
    assert torch.equal(a.view(torch.int64), b.view(torch.int64))
