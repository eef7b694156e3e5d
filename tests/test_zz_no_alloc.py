"""The allocation-free fused decode step (vd_decode_attention_evict_noalloc)
against the fused decode step with a caller's workspace
(vd_decode_attention_evict): both run the same kernels on the same split plan,
so attention outputs, K, V, pos and the running sum must be bit-identical.
Two calls in a row on the static scratch, the second on a smaller input; and
the size limit, which is checked on the host before anything is queued."""
import ctypes

import numpy as np
import pytest
import torch

from paper_2609_23314_amd import synth, vd

DEV = "cuda"


def _case(S, L, H, G, C, D, n, N, dtype, seed):
    k = synth.random_rows((S, L, H, C, D), dtype, seed, DEV)
    v = synth.random_rows((S, L, H, C, D), dtype, seed + 1, DEV)
    U = S * L * H
    st = torch.zeros((U, D + 1), dtype=torch.float64, device=DEV)
    vu = v.view(U, C, D)
    for s in range(S):   # the state covers every row but the newest
        us = slice(s * L * H, (s + 1) * L * H)
        st[us, :D] = vu[us, :n[s] - 1].double().sum(dim=1)
        st[us, D] = n[s] - 1
    pos = torch.arange(C, dtype=torch.int32, device=DEV).repeat(U, 1).contiguous()
    g = torch.Generator(device=DEV)
    g.manual_seed(seed + 7)
    q = torch.randn((S, L, H * G, D), generator=g, device=DEV)
    return k, v, st, pos, q


def _bits(t):
    return t.contiguous().view(torch.uint8)


@pytest.mark.gpu
def test_noalloc_matches_workspace_call_twice():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    vd.load()
    cases = [  # the second call is the smaller input
        dict(S=3, L=2, H=4, G=4, C=2049, D=128, n=[2049, 1500, 7], N=[2048, 2048, 2048],
             dtype=torch.bfloat16, seed=501),
        dict(S=2, L=1, H=2, G=2, C=300, D=64, n=[300, 120], N=[299, 119],
             dtype=torch.float32, seed=601),
    ]
    for c in cases:
        k, v, st, pos, q = _case(c["S"], c["L"], c["H"], c["G"], c["C"], c["D"], c["n"], c["N"],
                                 c["dtype"], c["seed"])
        kb, vb, stb, posb = k.clone(), v.clone(), st.clone(), pos.clone()
        out_a = torch.full(q.shape, float("nan"), device=DEV)
        out_b = torch.full(q.shape, float("nan"), device=DEV)
        vd.vd_decode_attention_evict(k, v, q, c["n"], c["N"], st, pos=pos, out=out_a)
        vd.vd_decode_attention_evict_noalloc(kb, vb, q, c["n"], c["N"], stb, out_b, pos=posb)
        torch.cuda.synchronize()
        what = f"S={c['S']} D={c['D']} n={c['n']}"
        print("noalloc:", what, flush=True)
        assert torch.isfinite(out_b).all(), what
        assert torch.equal(_bits(out_a), _bits(out_b)), what
        assert torch.equal(_bits(k), _bits(kb)) and torch.equal(_bits(v), _bits(vb)), what
        assert torch.equal(pos, posb), what
        assert torch.equal(_bits(st), _bits(stb)), what
        # the step evicted where n = N + 1 and kept everything elsewhere
        U = st.shape[0]
        L, H = c["L"], c["H"]
        for s in range(c["S"]):
            us = slice(s * L * H, (s + 1) * L * H)
            assert torch.all(stb[us, -1] == min(c["n"][s], c["N"][s])), what


def test_noalloc_rejects_a_call_beyond_its_scratch():
    """A call whose workspace would exceed the static array is refused on the
    host (the pointers below are never dereferenced)."""
    lib = vd.load()
    limit = vd.vd_decode_attention_noalloc_max_bytes()
    assert limit == 32 << 20
    fake = 0x7F0000000000
    d = vd.VdCacheDesc()
    d.k, d.v = fake, fake + (1 << 36)
    d.dtype = vd.VD_DTYPE_BF16
    d.num_seqs, d.num_layers, d.num_kv_heads, d.num_q_heads = 64, 32, 8, 32
    d.head_dim, d.capacity = 128, 4097
    d.stride_slot, d.stride_head = 128, 4097 * 128
    d.stride_layer, d.stride_seq = 8 * 4097 * 128, 32 * 8 * 4097 * 128
    need = lib.vd_decode_attention_workspace_size(ctypes.byref(d), 0)
    assert need > limit
    S = 64
    n = (ctypes.c_int32 * S)(*([4097] * S))
    N = (ctypes.c_int32 * S)(*([4096] * S))
    st = lib.vd_decode_attention_evict_noalloc(ctypes.byref(d), fake, 0.1, n, N, 0, fake, None,
                                               fake, None)
    assert st == vd.VD_ERR_WORKSPACE
    # and a call that fits passes the size check (then fails on a null q
    # before anything is queued)
    d.num_seqs = 1
    assert lib.vd_decode_attention_workspace_size(ctypes.byref(d), 0) <= limit
    st = lib.vd_decode_attention_evict_noalloc(ctypes.byref(d), None, 0.1, n, N, 0, fake, None,
                                               fake, None)
    assert st == vd.VD_ERR_INVALID_ARG
