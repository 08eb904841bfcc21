"""GPU parity, kernel by kernel: librv through its C ABI against the fp64 oracle on the
same seeded inputs.  Shapes span several tiles with ragged tails, empty and one-row
memories, one-token frames, and the ViT-L frame (1041 tokens x 16 heads)."""
import os

import numpy as np
import pytest

import oracle
from paper_2609_23286_amd import synth
from util import (LSE_ATOL, OUT_ATOL, SAL_RTOL, bf16_to_f64, check_index_sets, out_error_bound,
                  to_dev, to_host_u16)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def rv():
    from paper_2609_23286_amd import rv as _rv
    _rv.init()
    return _rv


def frame(seed, N, H, sigma=0.125):
    return tuple(synth.normal_bf16(seed, 0, 0, tag, (N, H, 64), sigma) for tag in range(3))


def memory_rows(seed, H, M, sigma=0.125):
    K = synth.normal_bf16(seed, 1, 0, synth.TAG_MEMK, (H, M, 64), sigma)
    V = synth.normal_bf16(seed, 1, 0, synth.TAG_MEMV, (H, M, 64), sigma)
    return K, V


def qsub_for(N):
    if N == 1041:
        return (28, 37, 5, 2)
    return (1, N, 0, 2)   # a 1 x N strip: every other token


def run_attend(rv, Q, K, V, memK, memV, qs, with_saliency=True):
    import torch
    N, H, _ = Q.shape
    M = memK.shape[1]
    mem = rv.Memory(H, reserve_tokens=M + 7, max_tokens=M + 64)
    if M:
        mem.write(torch.from_numpy(memK.view(np.int16)), torch.from_numpy(memV.view(np.int16)))
    Qd, Kd, Vd = to_dev(Q), to_dev(K), to_dev(V)
    out = torch.empty((N, H, 64), dtype=torch.int16, device="cuda")
    lse = torch.empty((H, N), dtype=torch.float32, device="cuda")
    sal = torch.empty((H, N), dtype=torch.float32, device="cuda") if with_saliency else None
    rv.attend_frame(Qd, Kd, Vd, mem, out, lse, sal, qs)
    rv.device_status()
    res = (bf16_to_f64(to_host_u16(out)), lse.cpu().numpy().astype(np.float64),
           None if sal is None else sal.cpu().numpy().astype(np.float64))
    mem.close()
    return res


ATTEND_CASES = [  # (N, H, M, sigma)
    (1, 1, 0, 0.125),
    (1, 1, 1, 0.125),
    (17, 2, 0, 0.125),
    (64, 2, 0, 0.125),
    (64, 2, 1, 0.125),
    (65, 2, 63, 0.5),
    (130, 2, 65, 0.125),
    (200, 3, 1000, 0.125),
    (300, 2, 700, 2.0),       # logits of a few units: running-max raises and rescales
    (1041, 16, 0, 0.125),
    (1041, 16, 257, 0.125),
]


@pytest.mark.parametrize("N,H,M,sigma", ATTEND_CASES)
def test_attend_and_saliency_match_oracle(rv, N, H, M, sigma):
    print(f"attend N={N} H={H} M={M} sigma={sigma}", flush=True)
    Q, K, V = frame(100 + N + M, N, H, sigma)
    memK, memV = memory_rows(200 + N + M, H, M, sigma)
    qs = qsub_for(N)
    out, lse, sal = run_attend(rv, Q, K, V, memK, memV, qs)
    out_o, lse_o = oracle.attend(Q, K, V, memK, memV, M)
    qidx = oracle.qsub_index(*qs)
    sal_o = oracle.saliency(Q, K, lse_o, qidx)
    assert np.isfinite(out).all() and np.isfinite(lse).all() and np.isfinite(sal).all()
    err = np.abs(out - out_o).max()
    vmax = max(np.abs(bf16_to_f64(V)).max(), np.abs(bf16_to_f64(memV)).max() if M else 0.0)
    assert err <= out_error_bound(out_o, vmax)
    if sigma <= 0.125:      # the workloads' scale: the 2e-2 acceptance bound applies
        assert err <= OUT_ATOL
    assert np.abs(lse - lse_o).max() <= LSE_ATOL
    assert (np.abs(sal - sal_o) <= SAL_RTOL * sal_o).all()


PLANS = [  # (workgroups per CU, minimum chunk, split: -1 auto, 0 stream-K, k > 0 k-way,
           #  per cent of a later stream-K chunk's tiles given to a first-dispatched one;
           #  "" the default: the unit-aligned share where one exists, as at 1041 x 16, M = 3000)
    ("1", "1", "0", "140"), ("2", "2", "0", "140"), ("4", "1", "0", "140"), ("1", "100000", "0", "140"),
    ("2", "2", "-1", "140"), ("1", "1", "1", "140"), ("2", "1", "7", "140"), ("2", "1", "64", "140"),
    ("4", "3", "-1", "140"), ("2", "1", "0", "100"), ("2", "1", "0", "101"), ("2", "2", "0", "400"),
    ("4", "1", "0", "250"), ("2", "2", "0", ""), ("2", "2", "-1", ""),
]


@pytest.mark.parametrize("wg_per_cu,min_chunk,split,first_pct", PLANS)
def test_work_plans_agree_with_oracle(rv, wg_per_cu, min_chunk, split, first_pct, monkeypatch):
    """Work plans (stream-K chunks of one key tile, of a few, whole units, with the
    first-dispatched chunks as long as the others or longer, or the unit-aligned form;
    aligned k-way splits with k = 1, several, more pieces than tiles) change only the
    rounding order of the partial merges."""
    monkeypatch.setenv("RV_ATTN_WG_PER_CU", wg_per_cu)
    monkeypatch.setenv("RV_ATTN_MIN_CHUNK", min_chunk)
    monkeypatch.setenv("RV_ATTN_SPLIT", split)
    monkeypatch.setenv("RV_ATTN_FIRST_PCT", first_pct)
    for N, H, M in ((333, 4, 1500), (1041, 16, 3000), (65, 1, 0)):
        print(f"plan {wg_per_cu}/{min_chunk}/{split}/{first_pct}: N={N} H={H} M={M}", flush=True)
        rv.reserve_workspace(N, H, M)   # a forced plan may need more partial slots than the default
        Q, K, V = frame(7 + N, N, H)
        memK, memV = memory_rows(8 + N, H, M)
        out, lse, _ = run_attend(rv, Q, K, V, memK, memV, qsub_for(N), with_saliency=False)
        out_o, lse_o = oracle.attend(Q, K, V, memK, memV, M)
        assert np.abs(out - out_o).max() <= OUT_ATOL
        assert np.abs(lse - lse_o).max() <= LSE_ATOL


def test_empty_query_subset_gives_zero_saliency(rv):
    """A query-subset descriptor with no window (grid_h = 0: every token is a special
    token) is valid: every saliency is the empty sum 0 (as the oracle's definition
    gives), so the selection takes the lowest indices.  Through rv_attend_frame and
    through the deferred rv_admit_layers."""
    import torch
    N, H, M, budget = 1041, 16, 300, 10
    qs = (0, 37, N, 2)
    qidx = oracle.qsub_index(*qs)
    assert len(qidx) == 0
    Q, K, V = frame(21, N, H)
    memK, memV = memory_rows(22, H, M)
    out, lse, sal = run_attend(rv, Q, K, V, memK, memV, qs)
    out_o, lse_o = oracle.attend(Q, K, V, memK, memV, M)
    sal_o = oracle.saliency(Q, K, lse_o, qidx)
    assert (sal_o == 0).all() and (sal == 0).all()
    assert np.abs(out - out_o).max() <= OUT_ATOL and np.abs(lse - lse_o).max() <= LSE_ATOL
    mem = rv.Memory(H, reserve_tokens=M, max_tokens=M + budget)
    mem.write(torch.from_numpy(memK.view(np.int16)), torch.from_numpy(memV.view(np.int16)))
    sal_d = torch.full((H, N), -1.0, dtype=torch.float32, device="cuda")
    idx = torch.full((H, budget), -1, dtype=torch.int32, device="cuda")
    rv.admit_layers([to_dev(Q)], [to_dev(K)], [to_dev(V)], [to_dev(lse.astype(np.float32))], qs, budget,
                    [mem], 4, [sal_d], [idx])
    rv.device_status()
    assert (sal_d.cpu().numpy() == 0).all()
    assert (idx.cpu().numpy() == oracle.topk(sal_o, budget)).all()
    assert (idx.cpu().numpy() == np.arange(budget)).all()
    mem.close()


def test_attend_frame_neither_allocates_nor_synchronises(rv, monkeypatch):
    """rv_attend_frame returns while earlier work on its stream is still running (no
    implicit device synchronisation), and a work plan that needs more partial slots than
    the workspace holds is refused with RV_ERR_CAPACITY -- nothing enqueued, outputs
    untouched -- instead of allocating; after rv_reserve_workspace the same call runs."""
    import torch
    N, H, M = 1041, 16, 2000
    Q, K, V = frame(31, N, H)
    memK, memV = memory_rows(32, H, M)
    mem = rv.Memory(H, reserve_tokens=M, max_tokens=M)
    mem.write(torch.from_numpy(memK.view(np.int16)), torch.from_numpy(memV.view(np.int16)))
    Qd, Kd, Vd = to_dev(Q), to_dev(K), to_dev(V)
    out = torch.full((N, H, 64), 7, dtype=torch.int16, device="cuda")
    lse = torch.full((H, N), 5.0, dtype=torch.float32, device="cuda")
    torch.cuda.synchronize()
    if hasattr(torch.cuda, "_sleep"):          # keeps the stream busy for a bounded while
        torch.cuda._sleep(200_000_000)
    else:
        a = torch.full((4096, 4096), 1e-3, device="cuda")
        for _ in range(40):
            a = a @ a
    busy = torch.cuda.Event()
    busy.record()
    rv.attend_frame(Qd, Kd, Vd, mem, out, lse)
    returned_early = not busy.query()
    torch.cuda.synchronize()
    assert returned_early, "rv_attend_frame waited for earlier work on the device"
    out_o, lse_o = oracle.attend(Q, K, V, memK, memV, M, rows=np.arange(0, N, 97, dtype=np.int32))
    assert np.abs(bf16_to_f64(to_host_u16(out))[::97] - out_o).max() <= OUT_ATOL
    # every tile its own chunk, at a memory length no other test reserves for
    monkeypatch.setenv("RV_ATTN_SPLIT", "100000")
    monkeypatch.setenv("RV_ATTN_MIN_CHUNK", "1")
    big = 40000
    memK2 = np.zeros((H, big, 64), dtype=np.uint16)
    mem2 = rv.Memory(H, reserve_tokens=big, max_tokens=big)
    mem2.write(torch.from_numpy(memK2.view(np.int16)), torch.from_numpy(memK2.view(np.int16)))
    out.fill_(7)
    lse.fill_(5.0)
    torch.cuda.synchronize()
    with pytest.raises(rv.RVError) as e:
        rv.attend_frame(Qd, Kd, Vd, mem2, out, lse)
    assert e.value.status == rv.RV_ERR_CAPACITY
    torch.cuda.synchronize()
    assert (out == 7).all() and (lse == 5.0).all()
    monkeypatch.setenv("RV_ATTN_SPLIT", "40")
    rv.reserve_workspace(N, H, M)
    rv.attend_frame(Qd, Kd, Vd, mem, out, lse)
    rv.device_status()
    assert np.abs(bf16_to_f64(to_host_u16(out))[::97] - out_o).max() <= OUT_ATOL
    mem.close()
    mem2.close()


def test_saliency_is_bit_reproducible(rv):
    N, H, M = 1041, 16, 500
    Q, K, V = frame(3, N, H)
    memK, memV = memory_rows(4, H, M)
    a = run_attend(rv, Q, K, V, memK, memV, qsub_for(N))
    b = run_attend(rv, Q, K, V, memK, memV, qsub_for(N))
    for x, y in zip(a, b):
        assert (x == y).all()


SELECT_CASES = [  # (N, H, budget, values): "ties" = nine levels, "spread" = continuous
    (1, 1, 0, "ties"), (1, 1, 1, "ties"), (64, 2, 1, "ties"), (100, 3, 7, "ties"),
    (1041, 16, 10, "ties"), (1041, 16, 10, "spread"), (1041, 4, 1040, "ties"),
    (1041, 2, 1041, "ties"), (1374, 4, 13, "spread"), (300, 2, 33, "ties"),
    (2048, 2, 32, "ties"), (2048, 2, 32, "spread"), (2049, 2, 32, "ties"), (3000, 1, 20, "spread"),
    (5000, 2, 50, "ties"), (16384, 1, 163, "ties"),
]


@pytest.mark.parametrize("N,H,budget,values", SELECT_CASES)
def test_admit_matches_oracle_topk_on_given_saliency(rv, N, H, budget, values):
    """rv_admit on a given saliency (full of exact ties, or continuous): the index set,
    its order, the appended rows and their provenance must equal the oracle's exactly
    (both wave-level and radix selection paths, on both sides of their boundary)."""
    import torch
    print(f"admit N={N} H={H} budget={budget} {values}", flush=True)
    rng = np.random.default_rng(N + budget)
    if values == "ties":
        sal = (rng.integers(0, 9, size=(H, N)).astype(np.float32) / 9.0)
    else:
        sal = rng.random(size=(H, N)).astype(np.float32) * np.float32(0.05)
    K, V, _ = frame(11, N, H)
    mem = rv.Memory(H, reserve_tokens=3, max_tokens=budget + 10)
    pre = memory_rows(12, H, 3)
    mem.write(torch.from_numpy(pre[0].view(np.int16)), torch.from_numpy(pre[1].view(np.int16)), frame_id=-1)
    idx = torch.full((H, budget), -7, dtype=torch.int32, device="cuda")
    rv.admit(to_dev(sal), budget, to_dev(K), to_dev(V), mem, 42, idx)
    rv.device_status()
    ref = oracle.topk(sal.astype(np.float64), budget)
    got = idx.cpu().numpy()
    assert (got == ref).all()
    assert mem.len == 3 + budget
    mk, mv, prov = mem.read()
    mk, mv, prov = mk.numpy().view(np.uint16), mv.numpy().view(np.uint16), prov.numpy()
    assert (mk[:, :3] == pre[0]).all() and (mv[:, :3] == pre[1]).all()
    for h in range(H):
        assert (mk[h, 3:] == K[ref[h], h]).all()
        assert (mv[h, 3:] == V[ref[h], h]).all()
        assert (prov[h, 3:, 0] == 42).all() and (prov[h, 3:, 1] == ref[h]).all()
    mem.close()


def test_admit_capacity_error_leaves_memory_unchanged(rv):
    import torch
    N, H = 64, 2
    K, V, _ = frame(5, N, H)
    sal = to_dev(np.linspace(1, 2, N * H, dtype=np.float32).reshape(H, N))
    mem = rv.Memory(H, reserve_tokens=0, max_tokens=15)
    rv.admit(sal, 10, to_dev(K), to_dev(V), mem, 0)
    before = [t.clone() for t in mem.read()]
    with pytest.raises(rv.RVError) as e:
        rv.admit(sal, 10, to_dev(K), to_dev(V), mem, 1)
    assert e.value.status == rv.RV_ERR_CAPACITY
    assert mem.len == 10
    after = mem.read()
    assert all((x == y).all() for x, y in zip(before, after))
    mem.close()


def test_bad_shapes_are_rejected(rv):
    import torch
    Q = torch.zeros((10, 2, 64), dtype=torch.int16, device="cuda")
    out = torch.zeros_like(Q)
    lse = torch.zeros((2, 10), dtype=torch.float32, device="cuda")
    with pytest.raises(ValueError):
        rv.attend_frame(Q, Q, Q[:9], None, out, lse)
    with pytest.raises(rv.RVError) as e:
        rv.attend_frame(Q, Q, Q, None, out, lse, lse, qs=(3, 3, 0, 2))
    assert e.value.status == rv.RV_ERR_INVALID


@pytest.mark.parametrize("L", [3, 26])
def test_admit_layers_is_bit_identical_to_per_layer_calls(rv, L):
    """Deferred, layer-batched admission == per-layer saliency + admit, bit for bit (26
    layers: two launches, of 24 layers and of 2)."""
    import torch
    N, H, M, budget = 300, 4, 200, 5
    print(f"admit_layers L={L}", flush=True)
    qs = (10, 30, 0, 2)
    results = []
    for batched in (False, True):
        mems, sals, idxs = [], [], []
        for l in range(L):
            Q, K, V = frame(50 + l, N, H)
            memK, memV = memory_rows(60 + l, H, M)
            mem = rv.Memory(H, reserve_tokens=M, max_tokens=M + budget)
            mem.write(torch.from_numpy(memK.view(np.int16)), torch.from_numpy(memV.view(np.int16)))
            Qd, Kd, Vd = to_dev(Q), to_dev(K), to_dev(V)
            out = torch.empty_like(Qd)
            lse = torch.empty((H, N), dtype=torch.float32, device="cuda")
            sal = torch.empty((H, N), dtype=torch.float32, device="cuda")
            idx = torch.empty((H, budget), dtype=torch.int32, device="cuda")
            if batched:
                rv.attend_frame(Qd, Kd, Vd, mem, out, lse)
            else:
                rv.attend_frame(Qd, Kd, Vd, mem, out, lse, sal, qs)
                rv.admit(sal, budget, Kd, Vd, mem, 9, idx)
            mems.append((mem, Qd, Kd, Vd, lse))
            sals.append(sal)
            idxs.append(idx)
        if batched:
            rv.admit_layers([m[1] for m in mems], [m[2] for m in mems], [m[3] for m in mems],
                            [m[4] for m in mems], qs, budget, [m[0] for m in mems], 9, sals, idxs)
        torch.cuda.synchronize()
        results.append(([s.cpu() for s in sals], [i.cpu() for i in idxs],
                        [m[0].read() for m in mems]))
        for m in mems:
            m[0].close()
    (sa, ia, ma), (sb, ib, mb) = results
    for l in range(L):
        assert (sa[l] == sb[l]).all()
        assert (ia[l] == ib[l]).all()
        assert all((x == y).all() for x, y in zip(ma[l], mb[l]))


def test_gpu_generator_matches_cpu_generator(rv):
    """The benchmark's GPU-side generator reproduces the CPU generator's bits."""
    import torch
    for name, frame_id in (("tiny", 3), ("vitl_layer", 17)):
        cfg = synth.CONFIGS[name]
        out = torch.empty((cfg.n_layers, 3, cfg.n_tokens, cfg.n_heads, 64), dtype=torch.int16, device="cuda")
        rv.gpu_frame_qkv(cfg, frame_id, out)
        torch.cuda.synchronize()
        got = out.cpu().numpy().view(np.uint16)
        Q, K, V = synth.frame_qkv(cfg, 0, frame_id)
        assert (got[0, 0] == Q).all() and (got[0, 2] == V).all()
        assert (got[0, 1] == K).all()


def test_gpu_generator_heavy_tailed_keys(rv):
    """The square-resolution stream's log-normal key scales on the GPU: Q and V bit for bit
    the CPU generator's; K too except where the two fp64 exponentials differ in their last
    bit, which can move an element by one bf16 step (rare, and never more)."""
    import torch
    cfg = synth.CONFIGS["square_2000"]
    out = torch.empty((2, 3, cfg.n_tokens, cfg.n_heads, 64), dtype=torch.int16, device="cuda")
    rv.gpu_frame_qkv(cfg, 41, out, layer0=5, n_layers=2)
    torch.cuda.synchronize()
    got = out.cpu().numpy().view(np.uint16)
    for i, layer in enumerate((5, 6)):
        Q, K, V = synth.frame_qkv(cfg, layer, 41)
        assert (got[i, 0] == Q).all() and (got[i, 2] == V).all()
        diff = np.abs(got[i, 1].astype(np.int32) - K.astype(np.int32))   # bf16 steps (same sign)
        assert diff.max() <= 1 and (diff > 0).mean() < 1e-4
        # the planted rows carry the scaled norms: the keys really are heavy-tailed
        norms = np.linalg.norm(bf16_to_f64(K), axis=2)
        assert norms.max() / np.median(norms) > 3.0


def test_memory_snapshot_round_trip(rv, tmp_path):
    """rv_mem_save / rv_mem_load: rows and provenance survive a round trip into a fresh
    memory (which grows to fit); a mismatched head count, an oversized snapshot, a
    truncated file and a foreign file are refused and leave the target unchanged."""
    import torch
    H, N, k = 3, 200, 7
    mem = rv.Memory(H, reserve_tokens=4, max_tokens=100)
    for t in range(5):
        K, V, _ = frame(40 + t, N, H)
        sal = torch.rand((H, N), device="cuda")
        rv.admit(sal, k, to_dev(K), to_dev(V), mem, t)
    rv.device_status()
    path = tmp_path / "mem.rvm"
    mem.save(path)
    ref = [x.numpy().copy() for x in mem.read()]
    fresh = rv.Memory(H, reserve_tokens=0, max_tokens=100)
    fresh.load(path)
    assert fresh.len == mem.len == 5 * k
    for a, b in zip(ref, fresh.read()):
        assert (a == b.numpy()).all()
    small = rv.Memory(H, reserve_tokens=0, max_tokens=10)
    other = rv.Memory(H + 1, reserve_tokens=0, max_tokens=100)
    with pytest.raises(rv.RVError) as e:
        small.load(path)
    assert e.value.status == rv.RV_ERR_CAPACITY and small.len == 0
    with pytest.raises(rv.RVError) as e:
        other.load(path)
    assert e.value.status == rv.RV_ERR_INVALID and other.len == 0
    data = path.read_bytes()
    (tmp_path / "cut.rvm").write_bytes(data[:-5])
    (tmp_path / "foreign.rvm").write_bytes(b"not a snapshot at all")
    for bad in ("cut.rvm", "foreign.rvm", "missing.rvm"):
        with pytest.raises(rv.RVError) as e:
            fresh.load(tmp_path / bad)
        assert e.value.status == rv.RV_ERR_IO
    assert fresh.len == 5 * k
    for a, b in zip(ref, fresh.read()):
        assert (a == b.numpy()).all()
    for m in (mem, fresh, small, other):
        m.close()


def test_head_averaged_admission(rv):
    """rv_admit_layers_shared: one selection per layer on the head-summed saliency, the
    same tokens appended to every head.  The saliency itself is the head-specific one;
    the selection must equal a CPU re-selection of the GPU's head sum (fp32, head order)
    exactly, and the oracle's head-mean selection under the band rule."""
    import torch
    L, N, H, M, budget = 2, 1041, 16, 300, 10
    qs = (28, 37, 5, 2)
    qidx = oracle.qsub_index(*qs)
    layers = []
    for l in range(L):
        Q, K, V = frame(70 + l, N, H)
        memK, memV = memory_rows(80 + l, H, M)
        mem = rv.Memory(H, reserve_tokens=M, max_tokens=M + budget)
        mem.write(torch.from_numpy(memK.view(np.int16)), torch.from_numpy(memV.view(np.int16)))
        Qd, Kd, Vd = to_dev(Q), to_dev(K), to_dev(V)
        out = torch.empty_like(Qd)
        lse = torch.empty((H, N), dtype=torch.float32, device="cuda")
        rv.attend_frame(Qd, Kd, Vd, mem, out, lse)
        layers.append((Q, K, V, memK, memV, mem, Qd, Kd, Vd, lse))
    sals = [torch.empty((H, N), dtype=torch.float32, device="cuda") for _ in range(L)]
    idxs = [torch.empty((H, budget), dtype=torch.int32, device="cuda") for _ in range(L)]
    rv.admit_layers([x[6] for x in layers], [x[7] for x in layers], [x[8] for x in layers],
                    [x[9] for x in layers], qs, budget, [x[5] for x in layers], 3, sals, idxs, shared=True)
    rv.device_status()
    for l, (Q, K, V, memK, memV, mem, *_rest) in enumerate(layers):
        idx = idxs[l].cpu().numpy()
        assert (idx == idx[0]).all()                      # one selection for every head
        sal = sals[l].cpu().numpy()
        head_sum = np.zeros(N, dtype=np.float32)
        for h in range(H):
            head_sum += sal[h]
        assert (idx[0] == oracle.topk(head_sum[None].astype(np.float64), budget)[0]).all()
        _, lse_o = oracle.attend(Q, K, V, memK, memV, M)
        sal_o = oracle.saliency(Q, K, lse_o, qidx)
        assert (np.abs(sal - sal_o) <= SAL_RTOL * sal_o).all()
        check_index_sets(idx[:1], sal_o.mean(axis=0, keepdims=True), budget)
        mk, mv, prov = (x.numpy() for x in mem.read())
        for h in range(H):
            assert (mk[h, M:].view(np.uint16) == K[idx[0], h]).all()
            assert (mv[h, M:].view(np.uint16) == V[idx[0], h]).all()
            assert (prov[h, M:, 0] == 3).all() and (prov[h, M:, 1] == idx[0]).all()
        mem.close()


@pytest.mark.parametrize("stride", [1, 3, 4])
def test_query_downsampling_factors(rv, stride):
    """Saliency with s x s query windows (Table 6's factors 1, 3, 4 beside the default 2):
    the sampled subset follows the same top-left rule, and saliency and selection match
    the oracle."""
    import torch
    N, H, M, budget = 1041, 16, 700, 10
    qs = (28, 37, 5, stride)
    qidx = oracle.qsub_index(*qs)
    print(f"stride {stride}: {len(qidx)} sampled queries", flush=True)
    Q, K, V = frame(90 + stride, N, H)
    memK, memV = memory_rows(95 + stride, H, M)
    out, lse, sal = run_attend(rv, Q, K, V, memK, memV, qs)
    _, lse_o = oracle.attend(Q, K, V, memK, memV, M)
    sal_o = oracle.saliency(Q, K, lse_o, qidx)
    assert (np.abs(sal - sal_o) <= SAL_RTOL * sal_o).all()
    mem = rv.Memory(H, reserve_tokens=budget, max_tokens=budget)
    idx = torch.empty((H, budget), dtype=torch.int32, device="cuda")
    rv.admit(to_dev(sal.astype(np.float32)), budget, to_dev(K), to_dev(V), mem, 0, idx)
    rv.device_status()
    idx = idx.cpu().numpy()
    assert (idx == oracle.topk(sal, budget)).all()
    check_index_sets(idx, sal_o, budget)
    mem.close()


STAGED_CASES = [  # (N, H, M, budget): ragged tails, empty memory, tile-aligned and
                  # unaligned memories, budgets whose selected rows overlap their
                  # destinations during the in-place compaction
    (1, 1, 0, 1), (65, 2, 0, 30), (130, 3, 257, 5), (300, 4, 200, 150), (300, 2, 64, 300),
    (200, 2, 128, 199), (1041, 16, 1000, 10), (1041, 16, 1024, 10),
]


@pytest.mark.parametrize("N,H,M,budget", STAGED_CASES)
def test_staged_frame_matches_oracle_and_frame_path(rv, N, H, M, budget):
    """A frame staged in the arena (rv_mem_stage_frame, rv_attend_staged): out, LSE and
    saliency within the oracle tolerances, and bit for bit the frame path's when M is a
    multiple of 64.  rv_admit_staged_layers (in-place compaction) against rv_admit_layers
    on the same LSE: saliency, selection, arena rows and provenance bit for bit."""
    import torch
    print(f"staged N={N} H={H} M={M} budget={budget}", flush=True)
    L = 2
    qs = qsub_for(N)
    qidx = oracle.qsub_index(*qs)
    staged_mems, frame_mems, Qs, Ks, Vs, lses = [], [], [], [], [], []
    for l in range(L):
        Q, K, V = frame(300 + l + N, N, H)
        memK, memV = memory_rows(400 + l + M, H, M)
        pair = []
        for _ in range(2):
            mem = rv.Memory(H, reserve_tokens=M + 3, max_tokens=M + N + 64)
            if M:
                mem.write(torch.from_numpy(memK.view(np.int16)), torch.from_numpy(memV.view(np.int16)))
            pair.append(mem)
        Qd, Kd, Vd = to_dev(Q), to_dev(K), to_dev(V)
        out = torch.empty_like(Qd)
        lse = torch.empty((H, N), dtype=torch.float32, device="cuda")
        sal = torch.empty((H, N), dtype=torch.float32, device="cuda")
        pair[0].stage_frame(Kd, Vd)   # grows the arena (reserve was M + 3)
        rv.attend_staged(Qd, pair[0], out, lse, sal, qs)
        rv.device_status()
        out_o, lse_o = oracle.attend(Q, K, V, memK, memV, M)
        sal_o = oracle.saliency(Q, K, lse_o, qidx)
        out_h = bf16_to_f64(to_host_u16(out))
        lse_h = lse.cpu().numpy().astype(np.float64)
        sal_h = sal.cpu().numpy().astype(np.float64)
        assert np.abs(out_h - out_o).max() <= OUT_ATOL
        assert np.abs(lse_h - lse_o).max() <= LSE_ATOL
        assert (np.abs(sal_h - sal_o) <= SAL_RTOL * sal_o).all()
        if M % 64 == 0:
            out_f = torch.empty_like(Qd)
            lse_f = torch.empty_like(lse)
            sal_f = torch.empty_like(sal)
            rv.attend_frame(Qd, Kd, Vd, pair[1], out_f, lse_f, sal_f, qs)
            torch.cuda.synchronize()
            assert (out_f == out).all() and (lse_f == lse).all() and (sal_f == sal).all()
        staged_mems.append(pair[0]); frame_mems.append(pair[1])
        Qs.append(Qd); Ks.append(Kd); Vs.append(Vd); lses.append(lse)
    res = []
    for staged in (True, False):
        sals = [torch.empty((H, N), dtype=torch.float32, device="cuda") for _ in range(L)]
        idxs = [torch.empty((H, budget), dtype=torch.int32, device="cuda") for _ in range(L)]
        if staged:
            rv.admit_staged_layers(Qs, lses, qs, budget, staged_mems, 7, sals, idxs)
            mems = staged_mems
        else:
            rv.admit_layers(Qs, Ks, Vs, lses, qs, budget, frame_mems, 7, sals, idxs)
            mems = frame_mems
        rv.device_status()
        res.append(([x.cpu() for x in sals], [x.cpu() for x in idxs], [m.read() for m in mems],
                    [m.len for m in mems]))
    for l in range(L):
        assert (res[0][0][l] == res[1][0][l]).all()
        assert (res[0][1][l] == res[1][1][l]).all()
        assert res[0][3][l] == res[1][3][l] == M + budget
        assert all((x == y).all() for x, y in zip(res[0][2][l], res[1][2][l]))
    # the compacted rows are the selected frame rows (layer 0)
    Q, K, V = frame(300 + N, N, H)
    Kr, Vr, prov = res[0][2][0]
    sel = res[0][1][0].numpy()
    for h in range(H):
        assert (Kr[h, M:].numpy().view(np.uint16) == K[sel[h], h]).all()
        assert (Vr[h, M:].numpy().view(np.uint16) == V[sel[h], h]).all()
        assert (prov[h, M:, 0].numpy() == 7).all() and (prov[h, M:, 1].numpy() == sel[h]).all()
    for m in staged_mems + frame_mems:
        m.close()


def test_staged_calls_need_a_staged_frame(rv):
    """rv_attend_staged / rv_admit_staged_layers refuse a memory with no room staged."""
    import torch
    H, N = 2, 64
    mem = rv.Memory(H, reserve_tokens=0, max_tokens=1000)
    Q = torch.zeros((N, H, 64), dtype=torch.int16, device="cuda")
    out = torch.empty_like(Q)
    lse = torch.empty((H, N), dtype=torch.float32, device="cuda")
    with pytest.raises(rv.RVError) as e:
        rv.attend_staged(Q, mem, out, lse)
    assert e.value.status == rv.RV_ERR_INVALID
    with pytest.raises(rv.RVError):
        rv.admit_staged_layers([Q], [lse], (1, N, 0, 2), 1, [mem], 0)
    assert mem.len == 0
    k, v, hs = mem.stage(N)
    assert k and v and hs >= N and mem.len == 0
    mem.close()


def test_staged_frames_in_one_launch_equal_per_layer_staging(rv):
    """rv_mem_stage_frames (26 layers: launches of 24 and 2) stages what rv_mem_stage_frame
    stages layer by layer, over memories with and without room for the frame: the
    lengths stay put, the staged attention gives the same bits, and after the staged
    admission (in-place compaction of the chosen staged rows) the arenas hold the same
    bytes."""
    import torch
    L, H, N, M, budget = 26, 3, 130, 70, 4
    qs = (10, 13, 0, 2)
    print(f"stage_frames L={L} H={H} N={N} M={M}", flush=True)
    runs = []
    for batched in (False, True):
        mems, frames = [], []
        for l in range(L):
            Q, K, V = frame(90 + l, N, H)
            mem = rv.Memory(H, reserve_tokens=M + (N if l % 2 else 0), max_tokens=M + N + 8)
            memK, memV = memory_rows(95 + l, H, M)
            mem.write(torch.from_numpy(memK.view(np.int16)), torch.from_numpy(memV.view(np.int16)))
            mems.append(mem)
            frames.append((to_dev(Q), to_dev(K), to_dev(V)))
        if batched:
            rv.stage_frames(mems, [f[1] for f in frames], [f[2] for f in frames])
        else:
            for mem, f in zip(mems, frames):
                mem.stage_frame(f[1], f[2])
        assert all(m.len == M for m in mems)
        outs, lses = [], []
        for mem, f in zip(mems, frames):
            out = torch.empty_like(f[0])
            lse = torch.empty((H, N), dtype=torch.float32, device="cuda")
            rv.attend_staged(f[0], mem, out, lse)
            outs.append(out)
            lses.append(lse)
        sals = [torch.empty((H, N), dtype=torch.float32, device="cuda") for _ in range(L)]
        rv.admit_staged_layers([f[0] for f in frames], lses, qs, budget, mems, 3, sals)
        rv.device_status()
        runs.append(([o.cpu() for o in outs], [x.cpu() for x in lses], [m.read() for m in mems]))
        assert all(m.len == M + budget for m in mems)
        for m in mems:
            m.close()
    (oa, la, ma), (ob, lb, mb) = runs
    for l in range(L):
        assert (oa[l] == ob[l]).all() and (la[l] == lb[l]).all(), f"layer {l}"
        assert all((x == y).all() for x, y in zip(ma[l], mb[l])), f"layer {l}"


FUSED_CASES = [  # (N, H, M, qs, plan overrides): ragged blocks, empty memory, a block with no
                 # sampled query, every query sampled, units covered whole by one chunk
    (1041, 16, 0, (28, 37, 5, 2), {}),
    (1041, 16, 2500, (28, 37, 5, 2), {}),
    (1041, 16, 700, (28, 37, 5, 1), {}),
    (300, 4, 700, (1, 300, 0, 2), {}),
    (130, 3, 1000, (10, 13, 0, 3), {}),
    (65, 2, 63, (5, 13, 0, 2), {}),
    (1, 1, 0, (1, 1, 0, 1), {}),
    (400, 2, 200, (0, 10, 400, 2), {}),                     # empty subset: every row 0
    (333, 4, 1500, (9, 37, 0, 2), {"RV_ATTN_WG_PER_CU": "1", "RV_ATTN_MIN_CHUNK": "100000"}),
]


@pytest.mark.parametrize("N,H,M,qs,env", FUSED_CASES)
def test_fused_saliency_matches_oracle(rv, N, H, M, qs, env, monkeypatch):
    """rv_attend_frame_fused (saliency in the attention epilogue, per 128-query block) and
    rv_admit_layers_tiled: out and LSE bit for bit rv_attend_frame's and within the oracle
    bounds; every block's row against the oracle's column mass over that block's sampled
    queries; the summed saliency against the oracle's; the selection exact on the GPU's own
    saliency and under the band rule on the oracle's; the appended rows."""
    import torch
    for k_, v_ in env.items():
        monkeypatch.setenv(k_, v_)
    print(f"fused N={N} H={H} M={M} qs={qs} {env}", flush=True)
    budget = min(10, N)
    Q, K, V = frame(500 + N + M, N, H)
    memK, memV = memory_rows(510 + N + M, H, M)
    mem = rv.Memory(H, reserve_tokens=M + budget, max_tokens=M + budget)
    if M:
        mem.write(torch.from_numpy(memK.view(np.int16)), torch.from_numpy(memV.view(np.int16)))
    Qd, Kd, Vd = to_dev(Q), to_dev(K), to_dev(V)
    nb = -(-N // 128)
    out = torch.empty_like(Qd)
    lse = torch.empty((H, N), dtype=torch.float32, device="cuda")
    tiles = torch.full((H, nb, N), -1.0, dtype=torch.float32, device="cuda")
    rv.attend_frame_fused(Qd, Kd, Vd, mem, out, lse, tiles, qs)
    out_f = torch.empty_like(Qd)
    lse_f = torch.empty_like(lse)
    rv.attend_frame(Qd, Kd, Vd, mem, out_f, lse_f)
    rv.device_status()
    assert (out == out_f).all() and (lse == lse_f).all()
    out_o, lse_o = oracle.attend(Q, K, V, memK, memV, M)
    assert np.abs(bf16_to_f64(to_host_u16(out)) - out_o).max() <= OUT_ATOL
    assert np.abs(lse.cpu().numpy() - lse_o).max() <= LSE_ATOL
    qidx = oracle.qsub_index(*qs)
    t_h = tiles.cpu().numpy().astype(np.float64)
    for b in range(nb):
        sel = qidx[(qidx >= 128 * b) & (qidx < 128 * (b + 1))]
        ref = oracle.column_mass(Q, sel, lse_o[:, sel], K, "frame")
        assert (np.abs(t_h[:, b] - ref) <= SAL_RTOL * ref).all(), f"block {b}"
    sal_o = oracle.saliency(Q, K, lse_o, qidx)
    sal = torch.full((H, N), -1.0, dtype=torch.float32, device="cuda")
    idx = torch.full((H, budget), -1, dtype=torch.int32, device="cuda")
    rv.admit_layers_tiled([tiles], budget, [Kd], [Vd], [mem], 6, [sal], [idx])
    rv.device_status()
    s_h = sal.cpu().numpy().astype(np.float64)
    assert (np.abs(s_h - sal_o) <= SAL_RTOL * sal_o).all()
    acc = t_h[:, 0].astype(np.float32)
    for b in range(1, nb):
        acc = acc + t_h[:, b].astype(np.float32)
    assert (acc == s_h.astype(np.float32)).all()              # the rows summed in block order
    i_h = idx.cpu().numpy()
    assert (i_h == oracle.topk(s_h, budget)).all()
    check_index_sets(i_h, sal_o, budget)
    mk, mv, prov = (x.numpy() for x in mem.read())
    for h in range(H):
        assert (mk[h, M:].view(np.uint16) == K[i_h[h], h]).all()
        assert (mv[h, M:].view(np.uint16) == V[i_h[h], h]).all()
        assert (prov[h, M:, 0] == 6).all() and (prov[h, M:, 1] == i_h[h]).all()
    mem.close()
