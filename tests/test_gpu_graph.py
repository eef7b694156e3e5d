"""The fused pass launched from a captured HIP graph (how bench.py times back
to back passes) against the same calls made one by one: every replay, with
the inputs restored between replays and the program's own eager work in
between, must leave K, V, pos and the running sum bit-identical to the eager
calls.  The passes run in steady state (the state covers the N old rows), at
a decode step (n = N + 1) and with a crossing fill, two sequences each."""
import pytest
import torch

from paper_2609_23314_amd import synth, vd

DEV = "cuda"


def _case(S, L, H, C, D, n, N, dtype, seed, count):
    k = synth.random_rows((S, L, H, C, D), dtype, seed, DEV)
    v = synth.random_rows((S, L, H, C, D), dtype, seed + 1, DEV)
    U = S * L * H
    st = torch.zeros((U, D + 1), dtype=torch.float64, device=DEV)
    vu = v.view(U, C, D)
    for s in range(S):
        us = slice(s * L * H, (s + 1) * L * H)
        c = count[s]
        st[us, :D] = vu[us, :c].double().sum(dim=1)
        st[us, D] = c
    pos = torch.arange(C, dtype=torch.int32, device=DEV).repeat(U, 1).contiguous()
    return k, v, st, pos


def _bits(t):
    return t.contiguous().view(torch.uint8)


CASES = [
    # steady state, several tiles and a ragged tail
    dict(S=2, L=2, H=2, C=1280, D=128, n=[1280, 1100], N=[1024, 900], count=[1024, 900],
         dtype=torch.bfloat16, seed=801),
    # a decode step (one token leaves)
    dict(S=2, L=1, H=4, C=513, D=64, n=[513, 400], N=[512, 399], count=[512, 399],
         dtype=torch.bfloat16, seed=811),
    # crossing fill without a state covering N rows, fp32
    dict(S=2, L=1, H=2, C=700, D=128, n=[700, 650], N=[600, 640], count=[300, 0],
         dtype=torch.float32, seed=821),
]


@pytest.mark.gpu
@pytest.mark.parametrize("case", CASES, ids=["steady", "decode", "crossing"])
def test_graph_replays_match_eager_calls(case):
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    vd.load()
    c = case
    k, v, st, pos = _case(c["S"], c["L"], c["H"], c["C"], c["D"], c["n"], c["N"], c["dtype"],
                          c["seed"], c["count"])
    # eager reference
    ke, ve, ste, pose = k.clone(), v.clone(), st.clone(), pos.clone()
    vd.vd_evict_step(ke, ve, c["n"], c["N"], "l2", running_sum=ste, pos=pose)
    torch.cuda.synchronize()
    # static buffers of the graph
    kg, vg, stg, posg = k.clone(), v.clone(), st.clone(), pos.clone()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):  # one call before the capture, as the capture API asks
        vd.vd_evict_step(kg, vg, c["n"], c["N"], "l2", running_sum=stg, pos=posg)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        vd.vd_evict_step(kg, vg, c["n"], c["N"], "l2", running_sum=stg, pos=posg)
    for rep in range(3):
        for dst, src in ((kg, k), (vg, v), (stg, st), (posg, pos)):
            dst.copy_(src)
        scratch = torch.randn(1 << 20, device=DEV).sum()  # eager work between the replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        what = f"replay {rep}: n={c['n']} N={c['N']} {c['dtype']}"
        print("graph:", what, float(scratch), flush=True)
        for got, want, name in ((kg, ke, "k"), (vg, ve, "v"), (stg, ste, "state"), (posg, pose, "pos")):
            assert torch.equal(_bits(got), _bits(want)), f"{name} differs after {what}"
