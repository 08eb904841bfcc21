"""GPU parity over whole streams and at the benchmark's full size.

* Free-running streams (tiny: 8 frames; one ViT-L layer: its first frames): the GPU and
  the oracle each keep their own memory; every frame's output, LSE, saliency, admitted
  set (band rule) and memory bytes are compared.  Should a near-tie inside the band let
  the two admit different tokens, the GPU memory is re-synchronised from the oracle's
  (the oracle never takes GPU state).
* Full size, in the launch configuration the benchmark times (24-layer ViT-L stack,
  1041 tokens x 16 heads, memory of 9,990 rows = frame 1000): the oracle computes the
  sampled queries row by row (all 266 saliency queries plus tile-edge rows); saliency,
  the admitted sets and the appended rows are compared in full -- per layer, and for the
  benchmark's one admission launch over all 24 layers.
"""
import numpy as np
import pytest

import oracle
from paper_2609_23286_amd import synth
from util import (LSE_ATOL, OUT_ATOL, SAL_RTOL, bf16_to_f64, check_index_sets, to_dev,
                  to_host_u16)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def rv():
    from paper_2609_23286_amd import rv as _rv
    _rv.init()
    return _rv


def gpu_frame_step(rv, mem, Q, K, V, qs, budget, frame_id):
    import torch
    N, H, _ = Q.shape
    Qd, Kd, Vd = to_dev(Q), to_dev(K), to_dev(V)
    out = torch.empty_like(Qd)
    lse = torch.empty((H, N), dtype=torch.float32, device="cuda")
    sal = torch.empty((H, N), dtype=torch.float32, device="cuda")
    idx = torch.empty((H, budget), dtype=torch.int32, device="cuda")
    rv.attend_frame(Qd, Kd, Vd, mem, out, lse, sal, qs)
    rv.admit(sal, budget, Kd, Vd, mem, frame_id, idx)
    rv.device_status()
    return (bf16_to_f64(to_host_u16(out)), lse.cpu().numpy().astype(np.float64),
            sal.cpu().numpy().astype(np.float64), idx.cpu().numpy())


def run_free_stream(rv, cfg, n_frames, anchor=False, row_sample=None, reserve=None):
    """Free-running stream: the GPU and the oracle each keep their own memory.  With
    row_sample, the oracle computes only the sampled queries (all of them, for the
    saliency) and the given output rows -- the rest of the attention is not needed for
    the admission -- and outputs are compared on those rows.  reserve: rows the GPU
    memory starts with (default: the whole stream's), so that smaller values make it
    grow inside the admissions."""
    import torch
    H, N, k = cfg.n_heads, cfg.n_tokens, cfg.budget
    qs = (cfg.grid_h, cfg.grid_w, cfg.n_special, cfg.stride)
    qidx = oracle.qsub_index(*qs)
    rows = None
    if row_sample is not None:
        rows = np.unique(np.concatenate([qidx, np.asarray(row_sample, dtype=np.int32)])).astype(np.int32)
        pos = np.searchsorted(rows, qidx)
    cap = (N if anchor else 0) + n_frames * k + 8
    mem = rv.Memory(H, reserve_tokens=cap if reserve is None else reserve, max_tokens=cap)
    omem = oracle.Memory(H, cfg.head_dim, cap)
    resyncs = 0
    for t in range(n_frames):
        print(f"{cfg.name} frame {t} (memory {mem.len})", flush=True)
        Q, K, V = synth.frame_qkv(cfg, 0, t)
        budget = N if (anchor and t == 0) else k
        out, lse, sal, idx = gpu_frame_step(rv, mem, Q, K, V, qs, budget, t)
        if rows is None:
            ref = oracle.step(omem, Q, K, V, qidx, budget)
        else:
            out_o, lse_o = oracle.attend(Q, K, V, omem.K, omem.V, omem.len, rows=rows)
            sal_o = oracle.column_mass(Q, qidx, lse_o[:, pos], K, "frame")
            idx_o = oracle.topk(sal_o, budget)
            omem.append(K, V, idx_o)
            ref = {"out": out_o, "lse": lse_o, "sal": sal_o, "idx": idx_o}
            out, lse = out[rows], lse[:, rows]
        assert np.abs(out - ref["out"]).max() <= OUT_ATOL
        assert np.abs(lse - ref["lse"]).max() <= LSE_ATOL
        assert (np.abs(sal - ref["sal"]) <= SAL_RTOL * ref["sal"]).all()
        # the GPU's top-k of its own saliency is exact
        assert (idx == oracle.topk(sal, budget)).all()
        check_index_sets(idx, ref["sal"], budget)
        assert mem.len == omem.len
        mk, mv, prov = (x.numpy() for x in mem.read())
        if (idx == ref["idx"]).all():
            assert (mk.view(np.uint16) == omem.K[:, :omem.len]).all()
            assert (mv.view(np.uint16) == omem.V[:, :omem.len]).all()
            assert (prov[:, -budget:, 0] == t).all() and (prov[:, -budget:, 1] == idx).all()
        else:
            resyncs += 1
            mem.write(torch.from_numpy(omem.K[:, :omem.len].view(np.int16).copy()),
                      torch.from_numpy(omem.V[:, :omem.len].view(np.int16).copy()))
    # memory growth formula (Eq. 4 and 6)
    assert mem.len == (N if anchor else k) + (n_frames - 1) * k
    mem.close()
    return resyncs


def test_tiny_stream_free_running(rv):
    assert run_free_stream(rv, synth.CONFIGS["tiny"], 8) == 0


def test_tiny_stream_with_anchor_frame(rv):
    assert run_free_stream(rv, synth.CONFIGS["tiny"], 8, anchor=True) == 0


def test_vitl_layer_stream_free_running(rv):
    """The whole 100-frame single-layer ViT-L stream, free-running from an empty memory
    to 1,000 rows: every frame's saliency, admitted set and memory bytes against the
    oracle's own stream, outputs and LSE on every sampled query plus tile-edge and
    scattered rows."""
    cfg = synth.CONFIGS["vitl_layer"]
    N = cfg.n_tokens
    sample = np.array([0, 1, 4, 5, 31, 32, 63, 64, 127, 128, 129, 511, 512, N - 2, N - 1], dtype=np.int32)
    sample = np.concatenate([sample, np.arange(3, N, 53, dtype=np.int32)])
    assert run_free_stream(rv, cfg, cfg.n_frames, row_sample=sample) == 0


def test_memory_grows_in_stream_order_on_a_side_stream(rv):
    """The first 60 frames of the single-layer ViT-L stream from a memory created empty,
    every call on a non-default stream: the arenas grow inside the admissions (0 -> 256
    -> 512 -> 608 rows, allocation, copy and release all stream-ordered, no host
    synchronisation) and every frame still matches the oracle's own stream, memory bytes
    included."""
    import torch
    cfg = synth.CONFIGS["vitl_layer"]
    N = cfg.n_tokens
    sample = np.array([0, 1, 63, 64, 511, 512, N - 1], dtype=np.int32)
    side = torch.cuda.Stream()
    with torch.cuda.stream(side):
        assert run_free_stream(rv, cfg, 60, row_sample=sample, reserve=0) == 0
    side.synchronize()


def test_stream_continues_bit_identically_after_restore(rv, tmp_path):
    """Checkpoint / resume: a memory saved after frame t and loaded into a fresh memory
    continues the stream exactly as the uninterrupted one -- outputs, LSE, saliency,
    admitted indices and memory bytes equal bit for bit for the frames that follow."""
    cfg = synth.CONFIGS["vitl_layer"]
    H, k = cfg.n_heads, cfg.budget
    qs = (cfg.grid_h, cfg.grid_w, cfg.n_special, cfg.stride)
    cap = 12 * k
    mem = rv.Memory(H, reserve_tokens=cap, max_tokens=cap)
    for t in range(6):
        gpu_frame_step(rv, mem, *synth.frame_qkv(cfg, 0, t), qs, k, t)
    path = tmp_path / "layer0.rvm"
    mem.save(path)
    restored = rv.Memory(H, reserve_tokens=0, max_tokens=cap)
    restored.load(path)
    for t in range(6, 12):
        frame = synth.frame_qkv(cfg, 0, t)
        a = gpu_frame_step(rv, mem, *frame, qs, k, t)
        b = gpu_frame_step(rv, restored, *frame, qs, k, t)
        for x, y in zip(a, b):
            assert (x == y).all(), f"frame {t} differs after the restore"
    assert mem.len == restored.len == 12 * k
    for x, y in zip(mem.read(), restored.read()):
        assert (x.numpy() == y.numpy()).all()
    mem.close()
    restored.close()


def test_stream_is_deterministic(rv):
    cfg = synth.CONFIGS["tiny"]
    qs = (cfg.grid_h, cfg.grid_w, cfg.n_special, cfg.stride)
    runs = []
    for _ in range(2):
        mem = rv.Memory(cfg.n_heads, reserve_tokens=64, max_tokens=64)
        outs = []
        for t in range(cfg.n_frames):
            outs.append(gpu_frame_step(rv, mem, *synth.frame_qkv(cfg, 0, t), qs, cfg.budget, t))
        outs.append(tuple(x.numpy() for x in mem.read()))
        runs.append(outs)
        mem.close()
    for a, b in zip(*runs):
        for x, y in zip(a, b):
            assert (x == y).all()


FULL_CASES = [  # (config, layer, memory rows)
    ("vitl_stack_1000", 5, 9990),     # last frame of the 1000-frame stream
    ("vitl_stack_1000", 23, 4000),
    ("square_2000", 11, 26000),       # 1374 tokens, heavy-tailed key norms, late frame
    ("long_memory_52k", 0, 52000),    # long-memory stress
]


@pytest.mark.parametrize("name,layer,M", FULL_CASES)
def test_full_size_frame_sampled_rows(rv, name, layer, M):
    import torch
    cfg = synth.CONFIGS[name]
    H, N, k = cfg.n_heads, cfg.n_tokens, cfg.budget
    print(f"full-size {name} layer {layer} M={M}", flush=True)
    qs = (cfg.grid_h, cfg.grid_w, cfg.n_special, cfg.stride)
    qidx = oracle.qsub_index(*qs)
    Q, K, V = synth.frame_qkv(cfg, layer, M // max(k, 1))
    memK, memV = synth.memory_prefill(cfg, layer, M)
    mem = rv.Memory(H, reserve_tokens=M + k, max_tokens=M + k)
    mem.write(torch.from_numpy(memK.view(np.int16)), torch.from_numpy(memV.view(np.int16)))
    out, lse, sal, idx = gpu_frame_step(rv, mem, Q, K, V, qs, k, 7)

    edge = [0, 1, 31, 32, 127, 128, N - 2, N - 1]
    rows = np.unique(np.concatenate([qidx, np.array(edge, dtype=np.int32)])).astype(np.int32)
    out_o, lse_o = oracle.attend(Q, K, V, memK, memV, M, rows=rows)
    assert np.abs(out[rows] - out_o).max() <= OUT_ATOL
    assert np.abs(lse[:, rows] - lse_o).max() <= LSE_ATOL
    pos = np.searchsorted(rows, qidx)
    sal_o = oracle.column_mass(Q, qidx, lse_o[:, pos], K, "frame")
    assert (np.abs(sal - sal_o) <= SAL_RTOL * sal_o).all()
    assert (idx == oracle.topk(sal, k)).all()
    check_index_sets(idx, sal_o, k)
    mk, mv, _ = (x.numpy().view(np.uint16) if x.dtype != torch.int32 else x.numpy() for x in mem.read())
    for h in range(H):
        assert (mk[h, M:] == K[idx[h], h]).all() and (mv[h, M:] == V[idx[h], h]).all()
    mem.close()


def test_layer_batched_admission_at_benchmark_shape(rv):
    """The admission launch the benchmark times: rv_admit_layers over all 24 layers of the
    ViT-L stack (1041 tokens x 16 heads, 266 sampled queries, budget 10; two saliency
    workgroups per (layer, head), 768 in the launch) on each layer's GPU attention LSE,
    against the oracle layer by layer: every key's saliency within SAL_RTOL of the
    column mass the oracle forms from its own LSE of the sampled queries, the selection
    the exact top-k of the GPU saliency and valid under the band rule, the appended rows
    bit for bit."""
    import torch
    cfg = synth.CONFIGS["vitl_stack_1000"]
    L, H, N, k = cfg.n_layers, cfg.n_heads, cfg.n_tokens, cfg.budget
    print(f"layer-batched admission L={L} H={H} N={N} budget={k}", flush=True)
    qs = (cfg.grid_h, cfg.grid_w, cfg.n_special, cfg.stride)
    qidx = oracle.qsub_index(*qs)
    frames = [synth.frame_qkv(cfg, l, 500) for l in range(L)]
    Qd, Kd, Vd, lse, sal, idx, mems = [], [], [], [], [], [], []
    for Q, K, V in frames:
        mem = rv.Memory(H, reserve_tokens=k, max_tokens=k)
        q, kk, v = to_dev(Q), to_dev(K), to_dev(V)
        out = torch.empty_like(q)
        ls = torch.empty((H, N), dtype=torch.float32, device="cuda")
        rv.attend_frame(q, kk, v, mem, out, ls)
        Qd.append(q), Kd.append(kk), Vd.append(v), lse.append(ls), mems.append(mem)
        sal.append(torch.empty((H, N), dtype=torch.float32, device="cuda"))
        idx.append(torch.empty((H, k), dtype=torch.int32, device="cuda"))
    rv.admit_layers(Qd, Kd, Vd, lse, qs, k, mems, 500, sal, idx)
    rv.device_status()
    for l, (Q, K, V) in enumerate(frames):
        _, lse_o = oracle.attend(Q, K, V, rows=qidx)
        sal_o = oracle.column_mass(Q, qidx, lse_o, K, "frame")
        s = sal[l].cpu().numpy().astype(np.float64)
        ix = idx[l].cpu().numpy()
        assert (np.abs(s - sal_o) <= SAL_RTOL * sal_o).all(), f"layer {l}"
        assert (ix == oracle.topk(s, k)).all(), f"layer {l}"
        check_index_sets(ix, sal_o, k)
        mk, mv, _ = (x.numpy().view(np.uint16) if x.dtype != torch.int32 else x.numpy() for x in mems[l].read())
        for h in range(H):
            assert (mk[h] == K[ix[h], h]).all() and (mv[h] == V[ix[h], h]).all(), f"layer {l} head {h}"
        mems[l].close()


def test_largest_frame_sampled_rows(rv):
    """The largest frame the boundary accepts (16384 tokens, a 128 x 128 grid, 2 heads)
    over a 3000-row memory: the 4096 sampled queries do not fit the saliency
    workgroup's LDS (rows read from memory), the budget of 163 takes the radix
    selection, and the key range spans 304 tiles.  Sampled rows against the oracle."""
    import torch
    H, N, M, k = 2, 16384, 3000, 163
    print(f"largest frame N={N} H={H} M={M} budget={k}", flush=True)
    qs = (128, 128, 0, 2)
    qidx = oracle.qsub_index(*qs)
    Q, K, V = (synth.normal_bf16(77, 0, 0, tag, (N, H, 64), 0.125) for tag in range(3))
    memK = synth.normal_bf16(78, 1, 0, synth.TAG_MEMK, (H, M, 64), 0.125)
    memV = synth.normal_bf16(78, 1, 0, synth.TAG_MEMV, (H, M, 64), 0.125)
    mem = rv.Memory(H, reserve_tokens=M + k, max_tokens=M + k)
    mem.write(torch.from_numpy(memK.view(np.int16)), torch.from_numpy(memV.view(np.int16)))
    out, lse, sal, idx = gpu_frame_step(rv, mem, Q, K, V, qs, k, 3)

    rng = np.random.default_rng(5)
    extra = rng.choice(N, 48, replace=False)
    edge = [0, 1, 63, 64, 127, 128, N - 65, N - 64, N - 2, N - 1]
    rows = np.unique(np.concatenate([qidx, extra, np.array(edge)])).astype(np.int32)
    out_o, lse_o = oracle.attend(Q, K, V, memK, memV, M, rows=rows)
    assert np.abs(out[rows] - out_o).max() <= OUT_ATOL
    assert np.abs(lse[:, rows] - lse_o).max() <= LSE_ATOL
    pos = np.searchsorted(rows, qidx)
    sal_o = oracle.column_mass(Q, qidx, lse_o[:, pos], K, "frame")
    assert (np.abs(sal - sal_o) <= SAL_RTOL * sal_o).all()
    assert (idx == oracle.topk(sal, k)).all()
    check_index_sets(idx, sal_o, k)
    mk, mv, _ = (x.numpy().view(np.uint16) if x.dtype != torch.int32 else x.numpy() for x in mem.read())
    for h in range(H):
        assert (mk[h, M:] == K[idx[h], h]).all() and (mv[h, M:] == V[idx[h], h]).all()
    mem.close()


def test_layer_policy_stream(rv):
    """The paper's layer partition (Sec. 3.3 Eq. 4-5, Sec. 4.1): the first frame is kept
    whole in every layer (global anchor); afterwards only the regulated layers admit
    tokens, the others attend over the anchor and the current frame alone.  Three layers
    of the tiny stream, the middle one regulated, eight frames, against the oracle."""
    import torch
    cfg = synth.CONFIGS["tiny"]
    H, N, k, L, T = cfg.n_heads, cfg.n_tokens, cfg.budget, 3, 8
    regulated = {1}
    qs = (cfg.grid_h, cfg.grid_w, cfg.n_special, cfg.stride)
    qidx = oracle.qsub_index(*qs)
    cap = N + T * k
    mems = [rv.Memory(H, reserve_tokens=cap, max_tokens=cap) for _ in range(L)]
    omems = [oracle.Memory(H, cfg.head_dim, cap) for _ in range(L)]
    for t in range(T):
        for l in range(L):
            Q, K, V = synth.frame_qkv(cfg, l, t)
            admit = t == 0 or l in regulated
            budget = N if t == 0 else k
            if admit:
                out, lse, sal, idx = gpu_frame_step(rv, mems[l], Q, K, V, qs, budget, t)
                ref = oracle.step(omems[l], Q, K, V, qidx, budget)
                assert (np.abs(sal - ref["sal"]) <= SAL_RTOL * ref["sal"]).all()
                check_index_sets(idx, ref["sal"], budget)
            else:
                Qd, Kd, Vd = to_dev(Q), to_dev(K), to_dev(V)
                outd = torch.empty_like(Qd)
                lsed = torch.empty((H, N), dtype=torch.float32, device="cuda")
                rv.attend_frame(Qd, Kd, Vd, mems[l], outd, lsed)
                rv.device_status()
                out = bf16_to_f64(to_host_u16(outd))
                lse = lsed.cpu().numpy().astype(np.float64)
                om = omems[l]
                ro, rl = oracle.attend(Q, K, V, om.K, om.V, om.len)
                ref = {"out": ro, "lse": rl}
            assert np.abs(out - ref["out"]).max() <= OUT_ATOL
            assert np.abs(lse - ref["lse"]).max() <= LSE_ATOL
    for l in range(L):
        assert mems[l].len == omems[l].len == (N + (T - 1) * k if l in regulated else N)
        mems[l].close()
