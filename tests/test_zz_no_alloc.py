"""rv_attend_frame_noalloc (the entry point for callers that cannot allocate) against
rv_attend_frame through the C ABI: two calls in a row on one GPU, the second with a
smaller frame and memory, each compared with rv_attend_frame's outputs on the same
inputs -- out, LSE and saliency within the oracle acceptance bounds (and bit for bit:
both take the same work plan) -- and the first call's outputs also against the oracle on
sampled rows."""
import ctypes

import numpy as np
import pytest

import oracle
from paper_2609_23286_amd import synth
from util import LSE_ATOL, OUT_ATOL, SAL_RTOL, bf16_to_f64, to_dev, to_host_u16

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def rv():
    from paper_2609_23286_amd import rv as _rv
    _rv.init()
    return _rv


def call(rv, fn, Qd, Kd, Vd, mem, qs, H, N):
    import torch
    vp = ctypes.c_void_p
    out = torch.full((N, H, 64), 3, dtype=torch.int16, device="cuda")
    lse = torch.full((H, N), -9.0, dtype=torch.float32, device="cuda")
    sal = torch.full((H, N), -9.0, dtype=torch.float32, device="cuda")
    mk, mv, hs = mem.view()
    q = rv.rv_qsub(*qs)
    st = getattr(rv.lib(), fn)(vp(Qd.data_ptr()), vp(Kd.data_ptr()), vp(Vd.data_ptr()), N, vp(mk), vp(mv),
                               mem.len, hs, H, 64, ctypes.byref(q), vp(out.data_ptr()), vp(lse.data_ptr()),
                               vp(sal.data_ptr()), vp(torch.cuda.current_stream().cuda_stream))
    assert st == rv.RV_OK, rv.lib().rv_last_error()
    rv.device_status()
    return (bf16_to_f64(to_host_u16(out)), lse.cpu().numpy().astype(np.float64),
            sal.cpu().numpy().astype(np.float64))


@pytest.mark.parametrize("order", ["large_then_small"])
def test_noalloc_matches_attend_frame_on_consecutive_calls(rv, order):
    import torch
    cases = [(1041, 16, 3000, (28, 37, 5, 2)), (300, 4, 500, (10, 30, 0, 2))]
    for i, (N, H, M, qs) in enumerate(cases):
        print(f"noalloc call {i}: N={N} H={H} M={M}", flush=True)
        Q, K, V = (synth.normal_bf16(600 + i, 0, 0, tag, (N, H, 64), 0.125) for tag in range(3))
        memK = synth.normal_bf16(610 + i, 1, 0, synth.TAG_MEMK, (H, M, 64), 0.125)
        memV = synth.normal_bf16(610 + i, 1, 0, synth.TAG_MEMV, (H, M, 64), 0.125)
        mem = rv.Memory(H, reserve_tokens=M, max_tokens=M)
        mem.write(torch.from_numpy(memK.view(np.int16)), torch.from_numpy(memV.view(np.int16)))
        Qd, Kd, Vd = to_dev(Q), to_dev(K), to_dev(V)
        got = call(rv, "rv_attend_frame_noalloc", Qd, Kd, Vd, mem, qs, H, N)
        ref = call(rv, "rv_attend_frame", Qd, Kd, Vd, mem, qs, H, N)
        assert np.abs(got[0] - ref[0]).max() <= OUT_ATOL
        assert np.abs(got[1] - ref[1]).max() <= LSE_ATOL
        assert (np.abs(got[2] - ref[2]) <= SAL_RTOL * ref[2]).all()
        for x, y in zip(got, ref):
            assert (x == y).all()
        if i == 0:
            rows = np.arange(0, N, 61, dtype=np.int32)
            out_o, lse_o = oracle.attend(Q, K, V, memK, memV, M, rows=rows)
            assert np.abs(got[0][rows] - out_o).max() <= OUT_ATOL
            assert np.abs(got[1][:, rows] - lse_o).max() <= LSE_ATOL
        mem.close()


def test_noalloc_refuses_a_plan_beyond_its_static_array(rv, monkeypatch):
    """A forced work plan with more partial slots than the static array holds is refused
    before anything is enqueued: the outputs keep their contents."""
    import torch
    N, H, M = 1041, 16, 3000
    monkeypatch.setenv("RV_ATTN_SPLIT", "64")
    monkeypatch.setenv("RV_ATTN_MIN_CHUNK", "1")
    Q = torch.zeros((N, H, 64), dtype=torch.int16, device="cuda")
    mem = rv.Memory(H, reserve_tokens=M, max_tokens=M)
    z = torch.zeros((H, M, 64), dtype=torch.int16)
    mem.write(z, z)
    out = torch.full((N, H, 64), 3, dtype=torch.int16, device="cuda")
    lse = torch.full((H, N), -9.0, dtype=torch.float32, device="cuda")
    mk, mv, hs = mem.view()
    vp = ctypes.c_void_p
    st = rv.lib().rv_attend_frame_noalloc(vp(Q.data_ptr()), vp(Q.data_ptr()), vp(Q.data_ptr()), N, vp(mk), vp(mv),
                                          M, hs, H, 64, None, vp(out.data_ptr()), vp(lse.data_ptr()), None,
                                          vp(torch.cuda.current_stream().cuda_stream))
    assert st == rv.RV_ERR_CAPACITY and b"static" in rv.lib().rv_last_error()
    torch.cuda.synchronize()
    assert (out == 3).all() and (lse == -9.0).all()
    mem.close()
