"""Python binding of librv (include/rv.h): argument marshalling only.

Every step of the hot path runs in librv's HIP kernels; this module checks tensor
shapes/dtypes/devices the C ABI cannot see (it receives raw pointers), converts
handles, and raises RVError on any non-zero rv_status.  Tensors are torch CUDA
(HIP) tensors; bf16 tensors may be any 2-byte dtype (bfloat16, int16, uint16) since
only their bits matter.  PyTorch supplies device memory and streams, nothing else.
There is no fallback: if librv.so is missing the import of this module fails.
"""
import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "librv.so")
SYNTH_LIB_PATH = os.path.join(_HERE, "librv_synth.so")

RV_OK, RV_ERR_INVALID, RV_ERR_OOM, RV_ERR_CAPACITY, RV_ERR_HIP, RV_ERR_IO = range(6)
HEAD_DIM = 64


class RVError(RuntimeError):
    def __init__(self, status, message):
        super().__init__(f"librv status {status}: {message}")
        self.status = status


class rv_qsub(ctypes.Structure):
    _fields_ = [("grid_h", ctypes.c_int32), ("grid_w", ctypes.c_int32),
                ("n_special", ctypes.c_int32), ("stride", ctypes.c_int32)]


class rv_attn_plan(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("n_units", "q_tiles", "T", "U", "E", "E1", "n_first",
                                               "n_queues", "grid", "total_chunks")] + [
        ("unit_base", ctypes.c_int32 * 17), ("n_chunks", ctypes.c_int32 * 16), ("chunk_base", ctypes.c_int32 * 16)]


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build() "
                          "(hipcc --offload-arch=gfx950)")
    lib = ctypes.CDLL(LIB_PATH)
    vp, i32, i64 = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64
    P = ctypes.POINTER
    sigs = {
        "rv_last_error": ([], ctypes.c_char_p),
        "rv_version": ([], ctypes.c_char_p),
        "rv_init": ([], i32),
        "rv_mem_create": ([i32, i32, i64, i64, P(vp)], i32),
        "rv_mem_destroy": ([vp], i32),
        "rv_mem_len": ([vp], i64),
        "rv_mem_capacity": ([vp], i64),
        "rv_mem_view": ([vp, P(vp), P(vp), P(i64)], i32),
        "rv_mem_reserve": ([vp, i64, vp], i32),
        "rv_mem_reset": ([vp], i32),
        "rv_mem_truncate": ([vp, i64], i32),
        "rv_mem_write": ([vp, vp, vp, i64, i32, vp], i32),
        "rv_mem_read": ([vp, vp, vp, vp, vp], i32),
        "rv_mem_save": ([vp, ctypes.c_char_p], i32),
        "rv_mem_load": ([vp, ctypes.c_char_p], i32),
        "rv_attend_frame": ([vp, vp, vp, i32, vp, vp, i64, i64, i32, i32, P(rv_qsub), vp, vp, vp, vp], i32),
        "rv_attend_frame_fused": ([vp, vp, vp, i32, vp, vp, i64, i64, i32, i32, P(rv_qsub), vp, vp, vp, vp], i32),
        "rv_admit_layers_tiled": ([i32, P(vp), i32, i32, P(vp), P(vp), P(vp), i32, P(vp), P(vp), vp], i32),
        "rv_attend_frame_noalloc": ([vp, vp, vp, i32, vp, vp, i64, i64, i32, i32, P(rv_qsub), vp, vp, vp, vp],
                                    i32),
        "rv_admit": ([vp, i32, vp, vp, i32, vp, i32, vp, vp], i32),
        "rv_admit_layers": ([i32, P(vp), P(vp), P(vp), P(vp), i32, P(rv_qsub), i32, P(vp), i32, P(vp), P(vp), vp], i32),
        "rv_admit_layers_shared": ([i32, P(vp), P(vp), P(vp), P(vp), i32, P(rv_qsub), i32, P(vp), i32, P(vp), P(vp),
                                    vp], i32),
        "rv_mem_stage": ([vp, i32, P(vp), P(vp), P(i64), vp], i32),
        "rv_mem_stage_frame": ([vp, vp, vp, i32, vp], i32),
        "rv_mem_stage_frames": ([i32, P(vp), P(vp), P(vp), i32, vp], i32),
        "rv_attend_staged": ([vp, i32, vp, P(rv_qsub), vp, vp, vp, vp], i32),
        "rv_admit_staged_layers": ([i32, P(vp), P(vp), i32, P(rv_qsub), i32, P(vp), i32, P(vp), P(vp), vp], i32),
        "rv_reserve_workspace": ([i32, i32, i64, i32], i32),
        "rv_attention_plan": ([i32, i32, i64, i32, i32, i32, P(rv_attn_plan)], i32),
        "rv_device_status": ([], i32),
    }
    for name, (args, res) in sigs.items():
        f = getattr(lib, name)
        f.argtypes = args
        f.restype = res
    return lib


_lib = _load()


def lib():
    return _lib


def _check(status):
    if status != RV_OK:
        raise RVError(status, _lib.rv_last_error().decode(errors="replace"))


def _stream(stream):
    if stream is None:
        return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    if isinstance(stream, torch.cuda.Stream):
        return ctypes.c_void_p(stream.cuda_stream)
    return ctypes.c_void_p(int(stream))


def _ptr(t, shape=None, itemsize=None, what="tensor"):
    if t is None:
        return None
    if isinstance(t, int):
        return ctypes.c_void_p(t)
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{what}: expected a torch tensor")
    if not t.is_cuda:
        raise ValueError(f"{what}: must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{what}: must be contiguous")
    if itemsize is not None and t.element_size() != itemsize:
        raise TypeError(f"{what}: element size {t.element_size()}, expected {itemsize}")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{what}: shape {tuple(t.shape)}, expected {tuple(shape)}")
    return ctypes.c_void_p(t.data_ptr())


def version():
    return _lib.rv_version().decode()


def qsub(grid_h, grid_w, n_special, stride):
    return rv_qsub(grid_h, grid_w, n_special, stride)


def init():
    """rv_init: set up librv on the current device (limits, XCD count, workspace)."""
    _check(_lib.rv_init())


def reserve_workspace(n_tokens, n_heads, max_mem_len=0, n_layers=1):
    """rv_reserve_workspace: partial slots for forced work plans up to max_mem_len memory
    rows, saliency staging for n_layers layers."""
    _check(_lib.rv_reserve_workspace(n_tokens, n_heads, max_mem_len, n_layers))


def attention_plan(n_tokens, n_fkeys, mem_len, n_heads, n_cus, n_queues):
    """The attention work plan for a frame on a device of n_cus CUs and n_queues XCDs
    (rv_attention_plan; no device work), as an rv_attn_plan structure."""
    out = rv_attn_plan()
    _check(_lib.rv_attention_plan(n_tokens, n_fkeys, mem_len, n_heads, n_cus, n_queues, ctypes.byref(out)))
    return out


def device_status():
    """Synchronise the device; raise RVError if a kernel raised a status bit."""
    _check(_lib.rv_device_status())


class Memory:
    """One layer's regulated KV memory (rv_mem)."""

    def __init__(self, n_heads, head_dim=HEAD_DIM, reserve_tokens=0, max_tokens=1 << 31):
        h = ctypes.c_void_p()
        _check(_lib.rv_mem_create(n_heads, head_dim, reserve_tokens, max_tokens, ctypes.byref(h)))
        self.handle = h
        self.n_heads = n_heads

    def close(self):
        if self.handle:
            _lib.rv_mem_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    @property
    def len(self):
        return _lib.rv_mem_len(self.handle)

    @property
    def capacity(self):
        return _lib.rv_mem_capacity(self.handle)

    def view(self):
        """(memK pointer, memV pointer, head stride in tokens)."""
        k, v, s = ctypes.c_void_p(), ctypes.c_void_p(), ctypes.c_int64()
        _check(_lib.rv_mem_view(self.handle, ctypes.byref(k), ctypes.byref(v), ctypes.byref(s)))
        return k.value or 0, v.value or 0, s.value

    def reserve(self, tokens, stream=None):
        _check(_lib.rv_mem_reserve(self.handle, tokens, _stream(stream)))

    def reset(self):
        _check(_lib.rv_mem_reset(self.handle))

    def truncate(self, n_rows):
        """rv_mem_truncate: drop the newest rows (host-side length change only)."""
        _check(_lib.rv_mem_truncate(self.handle, n_rows))

    def write(self, K, V, frame_id=-1, stream=None):
        """Overwrite rows 0..n-1 with K, V ([H, n, 64], 2-byte elements, host or device)."""
        if K.shape != V.shape or K.shape[0] != self.n_heads or K.shape[2] != HEAD_DIM:
            raise ValueError("K, V must both be [n_heads, n_rows, 64]")
        kp, vp = _host_or_dev_ptr(K), _host_or_dev_ptr(V)
        _check(_lib.rv_mem_write(self.handle, kp, vp, K.shape[1], frame_id, _stream(stream)))

    def read(self, stream=None):
        """(K, V, prov) of the valid rows as CPU torch tensors (int16 bits / int32)."""
        n = self.len
        K = torch.empty((self.n_heads, n, HEAD_DIM), dtype=torch.int16, pin_memory=True)
        V = torch.empty_like(K, pin_memory=True)
        prov = torch.empty((self.n_heads, n, 2), dtype=torch.int32, pin_memory=True)
        _check(_lib.rv_mem_read(self.handle, ctypes.c_void_p(K.data_ptr()), ctypes.c_void_p(V.data_ptr()),
                                ctypes.c_void_p(prov.data_ptr()), _stream(stream)))
        return K, V, prov

    def stage(self, n_tokens, stream=None):
        """rv_mem_stage: room for a frame of n_tokens rows past the valid ones; returns
        (K_tail, V_tail, head_stride) device addresses / row stride."""
        k, v, hs = ctypes.c_void_p(), ctypes.c_void_p(), ctypes.c_int64()
        _check(_lib.rv_mem_stage(self.handle, n_tokens, ctypes.byref(k), ctypes.byref(v), ctypes.byref(hs),
                                 _stream(stream)))
        return k.value, v.value, hs.value

    def stage_frame(self, K, V, stream=None):
        """rv_mem_stage_frame: stage a frame given as [N, H, 64] bf16 K, V tensors."""
        N = K.shape[0]
        shp = (N, self.n_heads, HEAD_DIM)
        _check(_lib.rv_mem_stage_frame(self.handle, _ptr(K, shp, 2, "K"), _ptr(V, shp, 2, "V"), N,
                                       _stream(stream)))

    def save(self, path):
        """Write a snapshot (rows and provenance) to `path`."""
        _check(_lib.rv_mem_save(self.handle, os.fsencode(path)))

    def load(self, path):
        """Replace the contents with a snapshot written by save()."""
        _check(_lib.rv_mem_load(self.handle, os.fsencode(path)))


def _host_or_dev_ptr(t):
    if not isinstance(t, torch.Tensor) or not t.is_contiguous() or t.element_size() != 2:
        raise TypeError("expected a contiguous torch tensor with 2-byte elements")
    return ctypes.c_void_p(t.data_ptr())


def attend_frame(Q, K, V, mem, out, lse, saliency=None, qs=None, stream=None,
                 memK=None, memV=None, mem_len=None, head_stride=None):
    """rv_attend_frame.  Q, K, V, out: [N, H, 64] bf16; lse/saliency: [H, N] fp32.

    The memory is given either as a Memory (``mem``) or, with mem=None, as raw
    ``memK``/``memV`` device pointers (int or tensor), ``mem_len`` and ``head_stride``."""
    N, H, d = Q.shape
    if mem is not None:
        mk, mv, hs = mem.view()
        ml = mem.len
    else:
        mk = memK.data_ptr() if isinstance(memK, torch.Tensor) else (memK or 0)
        mv = memV.data_ptr() if isinstance(memV, torch.Tensor) else (memV or 0)
        ml, hs = int(mem_len or 0), int(head_stride or 0)
    shp = (N, H, d)
    q = qs if qs is None or isinstance(qs, rv_qsub) else rv_qsub(*qs)
    _check(_lib.rv_attend_frame(
        _ptr(Q, shp, 2, "Q"), _ptr(K, shp, 2, "K"), _ptr(V, shp, 2, "V"), N,
        ctypes.c_void_p(mk), ctypes.c_void_p(mv), ml, hs, H, d,
        ctypes.byref(q) if q is not None else None,
        _ptr(out, shp, 2, "out"), _ptr(lse, (H, N), 4, "lse"),
        _ptr(saliency, (H, N), 4, "saliency"), _stream(stream)))


QUERY_BLOCK = 128


def attend_frame_fused(Q, K, V, mem, out, lse, sal_tiles, qs, stream=None):
    """rv_attend_frame_fused: attention with the saliency formed in its epilogue, per
    128-query block: sal_tiles [H, ceil(N / 128), N] fp32."""
    N, H, d = Q.shape
    mk, mv, hs = mem.view()
    shp = (N, H, d)
    q = qs if isinstance(qs, rv_qsub) else rv_qsub(*qs)
    _check(_lib.rv_attend_frame_fused(
        _ptr(Q, shp, 2, "Q"), _ptr(K, shp, 2, "K"), _ptr(V, shp, 2, "V"), N, ctypes.c_void_p(mk),
        ctypes.c_void_p(mv), mem.len, hs, H, d, ctypes.byref(q), _ptr(out, shp, 2, "out"),
        _ptr(lse, (H, N), 4, "lse"), _ptr(sal_tiles, (H, -(-N // QUERY_BLOCK), N), 4, "sal_tiles"),
        _stream(stream)))


def admit_layers_tiled(sal_tiles, budget, K, V, mems, frame_id, saliency_out=None, idx_out=None, stream=None):
    """rv_admit_layers_tiled over lists of per-layer sal_tiles [H, ceil(N / 128), N], K, V
    [N, H, 64] and Memory objects."""
    L = len(mems)
    N, H, d = K[0].shape
    arr = ctypes.c_void_p * L

    def pack(ts, shape, itemsize, what):
        return arr(*[_ptr(t, shape, itemsize, f"{what}[{i}]") for i, t in enumerate(ts)])

    sal = pack(saliency_out, (H, N), 4, "saliency_out") if saliency_out is not None else None
    idx = pack(idx_out, (H, budget), 4, "idx_out") if idx_out is not None else None
    _check(_lib.rv_admit_layers_tiled(
        L, pack(sal_tiles, (H, -(-N // QUERY_BLOCK), N), 4, "sal_tiles"), N, budget, pack(K, (N, H, d), 2, "K"),
        pack(V, (N, H, d), 2, "V"), arr(*[m.handle for m in mems]), frame_id, sal, idx, _stream(stream)))


def attend_staged(Q, mem, out, lse, saliency=None, qs=None, stream=None):
    """rv_attend_staged: attention of Q [N, H, 64] over mem's rows and its staged frame."""
    N, H, d = Q.shape
    q = qs if qs is None or isinstance(qs, rv_qsub) else rv_qsub(*qs)
    _check(_lib.rv_attend_staged(
        _ptr(Q, (N, H, d), 2, "Q"), N, mem.handle, ctypes.byref(q) if q is not None else None,
        _ptr(out, (N, H, d), 2, "out"), _ptr(lse, (H, N), 4, "lse"), _ptr(saliency, (H, N), 4, "saliency"),
        _stream(stream)))


def admit_staged_layers(Q, lse, qs, budget, mems, frame_id, saliency_out=None, idx_out=None, stream=None):
    """rv_admit_staged_layers over lists of per-layer Q [N, H, 64], lse [H, N] and Memory
    objects whose frames are staged."""
    L = len(mems)
    N, H, d = Q[0].shape
    arr = ctypes.c_void_p * L

    def pack(ts, shape, itemsize, what):
        return arr(*[_ptr(t, shape, itemsize, f"{what}[{i}]") for i, t in enumerate(ts)])

    q = qs if isinstance(qs, rv_qsub) else rv_qsub(*qs)
    sal = pack(saliency_out, (H, N), 4, "saliency_out") if saliency_out is not None else None
    idx = pack(idx_out, (H, budget), 4, "idx_out") if idx_out is not None else None
    _check(_lib.rv_admit_staged_layers(
        L, pack(Q, (N, H, d), 2, "Q"), pack(lse, (H, N), 4, "lse"), N, ctypes.byref(q), budget,
        arr(*[m.handle for m in mems]), frame_id, sal, idx, _stream(stream)))


def admit(saliency, budget, K, V, mem, frame_id, idx_out=None, stream=None):
    """rv_admit: per-head top-`budget` of saliency [H, N], append K/V rows to mem."""
    N, H, d = K.shape
    _check(_lib.rv_admit(_ptr(saliency, (H, N), 4, "saliency"), budget, _ptr(K, (N, H, d), 2, "K"),
                         _ptr(V, (N, H, d), 2, "V"), N, mem.handle, frame_id,
                         _ptr(idx_out, (H, budget), 4, "idx_out"), _stream(stream)))


def admit_layers(Q, K, V, lse, qs, budget, mems, frame_id, saliency_out=None, idx_out=None,
                 stream=None, shared=False):
    """rv_admit_layers (shared=False: head-specific retention) or rv_admit_layers_shared
    (shared=True: one selection per layer on the head-summed saliency) over lists of
    per-layer tensors and Memory objects."""
    L = len(mems)
    N, H, d = K[0].shape
    shp = (N, H, d)
    arr = ctypes.c_void_p * L

    def pack(ts, shape, itemsize, what):
        return arr(*[_ptr(t, shape, itemsize, f"{what}[{i}]") for i, t in enumerate(ts)])

    q = qs if isinstance(qs, rv_qsub) else rv_qsub(*qs)
    sal = pack(saliency_out, (H, N), 4, "saliency_out") if saliency_out is not None else None
    idx = pack(idx_out, (H, budget), 4, "idx_out") if idx_out is not None else None
    fn = _lib.rv_admit_layers_shared if shared else _lib.rv_admit_layers
    _check(fn(
        L, pack(Q, shp, 2, "Q"), pack(K, shp, 2, "K"), pack(V, shp, 2, "V"), pack(lse, (H, N), 4, "lse"),
        N, ctypes.byref(q), budget, arr(*[m.handle for m in mems]), frame_id, sal, idx, _stream(stream)))



def stage_frames(mems, K, V, stream=None):
    """rv_mem_stage_frames: stage each layer's frame (K[l], V[l]: [N, H, 64] bf16) in
    mems[l], one copy launch for up to 24 layers."""
    L = len(mems)
    N = K[0].shape[0]
    shp = (N, mems[0].n_heads, HEAD_DIM)
    arr = ctypes.c_void_p * L
    _check(_lib.rv_mem_stage_frames(L, arr(*[m.handle for m in mems]),
                                    arr(*[_ptr(k, shp, 2, f"K[{i}]") for i, k in enumerate(K)]),
                                    arr(*[_ptr(v, shp, 2, f"V[{i}]") for i, v in enumerate(V)]), N,
                                    _stream(stream)))

# ---- seeded stream generator on the GPU (benchmark inputs) -------------------------
_synth = None


def _load_synth():
    global _synth
    if _synth is None:
        if not os.path.exists(SYNTH_LIB_PATH):
            raise ImportError(f"{SYNTH_LIB_PATH} is not built; run __graft_entry__.build()")
        s = ctypes.CDLL(SYNTH_LIB_PATH)
        s.rvs_frame_qkv.argtypes = [ctypes.c_uint64, ctypes.c_uint32, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                    ctypes.c_int, ctypes.c_int, ctypes.c_float, ctypes.c_int, ctypes.c_double,
                                    ctypes.c_double, ctypes.c_void_p, ctypes.c_void_p]
        s.rvs_frame_qkv.restype = ctypes.c_int
        s.rvs_normal_bf16.argtypes = [ctypes.c_uint64, ctypes.c_uint32, ctypes.c_int, ctypes.c_int,
                                      ctypes.c_int64, ctypes.c_float, ctypes.c_void_p, ctypes.c_void_p]
        s.rvs_normal_bf16.restype = ctypes.c_int
        _synth = s
    return _synth


def gpu_frame_qkv(cfg, frame, out, layer0=0, n_layers=None, stream=None):
    """Fill out = [n_layers, 3, N, H, 64] (2-byte) with frame `frame` of cfg's stream."""
    n_layers = cfg.n_layers if n_layers is None else n_layers
    shape = (n_layers, 3, cfg.n_tokens, cfg.n_heads, cfg.head_dim)
    rc = _load_synth().rvs_frame_qkv(cfg.seed, frame & 0xFFFFFFFF, layer0, n_layers, cfg.n_tokens, cfg.n_heads,
                                     cfg.head_dim, cfg.sigma, cfg.n_plant, cfg.alpha, cfg.lognormal_sigma,
                                     _ptr(out, shape, 2, "out"), _stream(stream))
    if rc != 0:
        raise RVError(rc, "rvs_frame_qkv failed")


def gpu_normal(seed, frame, layer, tag, out, sigma, stream=None):
    rc = _load_synth().rvs_normal_bf16(seed, frame & 0xFFFFFFFF, layer, tag, out.numel(), sigma,
                                       _ptr(out, None, 2, "out"), _stream(stream))
    if rc != 0:
        raise RVError(rc, "rvs_normal_bf16 failed")
