"""Seeded synthetic token streams (numpy) -- the one module both sides read inputs from.

Holds no arithmetic of the method: it only draws Q/K/V tensors of the paper's token
shapes (ViT-L aggregator: 16 heads x 64, a 28x37 or 37x37 patch grid plus 5 special
tokens) with a counter-based generator, so that any frame of any layer can be drawn on
its own, on the CPU here or on the GPU by the library's generator, with the same bits.

Recipe (stated once; the GPU generator follows it step for step):

* Philox4x32-10 (Salmon, Moraes, Dror, Shaw: "Parallel random numbers: as easy as
  1, 2, 3", SC'11): 10 rounds, multipliers 0xD2511F53 / 0xCD9E8D57, Weyl key
  increments 0x9E3779B9 / 0xBB67AE85.
  key = (seed & 0xffffffff, seed >> 32);
  counter = (element index low 32 bits, element index high 32 bits, frame,
             layer << 8 | tag).
* Near-Gaussian value per element: the eight 16-bit halves of the four output words are
  summed (Irwin-Hall of order 8: mean 262140, variance 8 (2^32 - 1) / 12), centred
  and scaled by sigma / sd in fp32 (one IEEE multiply), then rounded to bf16
  (round-to-nearest-even).  Exact integer arithmetic up to the one multiply, so CPU
  and GPU agree bit for bit.  It matches N(0, sigma^2) in mean and variance; its
  tails stop at about 4.9 sd.
* Planted salient keys: per (layer, frame, head), ``n_plant`` distinct token positions
  drawn by a partial Fisher-Yates shuffle (Philox words, tag 3, reduced modulo the
  remaining count).  Key row j becomes alpha * |k_j| * qbar / |qbar|, with qbar the
  sum of the frame's queries of that head (fp64, exact for bf16 inputs of this range),
  norms summed over the head dimension in order in fp64, then ratio * qbar[e]
  rounded to fp32 then to bf16.
* Heavy-tailed key norms (square-resolution stream only, CPU side): every key row is
  multiplied by exp(sigma_ln * xi), xi a near-Gaussian from tag 6, before planting.
* Memory prefill rows (long-memory stress): tags 4 (K) and 5 (V), frame field
  0xFFFFFFFF, layout [H, rows, d].
"""
from dataclasses import dataclass, field
import math
import os

import numpy as np

M0, M1 = 0xD2511F53, 0xCD9E8D57
W0, W1 = 0x9E3779B9, 0xBB67AE85
MASK32 = 0xFFFFFFFF

TAG_Q, TAG_K, TAG_V, TAG_PLANT, TAG_MEMK, TAG_MEMV, TAG_LOGN = 0, 1, 2, 3, 4, 5, 6
PREFILL_FRAME = 0xFFFFFFFF

IH_MEAN = 262140                       # 8 * 65535 / 2
IH_SD = math.sqrt(8.0 * (65536.0 ** 2 - 1.0) / 12.0)


def philox4x32_10(c0, c1, c2, c3, k0, k1):
    """Philox4x32 with 10 rounds on uint32 arrays (broadcast); returns 4 uint32 arrays."""
    u64 = np.uint64
    c0, c1, c2, c3 = (np.asarray(x, dtype=np.uint64) & u64(MASK32) for x in (c0, c1, c2, c3))
    k0, k1 = int(k0) & MASK32, int(k1) & MASK32
    m32, sh = u64(MASK32), u64(32)
    for r in range(10):
        if r:
            k0 = (k0 + W0) & MASK32
            k1 = (k1 + W1) & MASK32
        p0 = c0 * u64(M0)
        p1 = c2 * u64(M1)
        c0 = (p1 >> sh) ^ c1 ^ u64(k0)
        c1 = p1 & m32
        c2 = (p0 >> sh) ^ c3 ^ u64(k1)
        c3 = p0 & m32
    c0, c1, c2, c3 = np.broadcast_arrays(c0, c1, c2, c3)
    return [x.astype(np.uint32) for x in (c0, c1, c2, c3)]


def f32_to_bf16_bits(x):
    """Round fp32 to bf16, nearest-even, on the bit pattern (no NaN input expected)."""
    u = np.asarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    r = (u + np.uint64(0x7FFF) + ((u >> np.uint64(16)) & np.uint64(1))) >> np.uint64(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(b):
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


_CHUNK = 1 << 18


def _normal_chunk(e0, e1, frame, stream_id, k0, k1, scale, out):
    """Elements e0..e1-1 of one counter stream -> bf16 bits into out[e0:e1]."""
    e = np.arange(e0, e1, dtype=np.uint64)
    w = philox4x32_10(e & np.uint64(MASK32), e >> np.uint64(32), np.uint64(frame),
                      np.uint64(stream_id), k0, k1)
    s = np.zeros(e.shape, dtype=np.int64)
    for x in w:
        x = x.astype(np.int64)
        s += (x & 0xFFFF) + (x >> 16)
    s -= IH_MEAN
    out[e0:e1] = f32_to_bf16_bits(s.astype(np.float32) * scale)


def _irwin_hall_stream(seed, frame, layer, tag, n):
    """Centred order-8 Irwin-Hall integers of one counter stream (length n)."""
    w = _stream_words(seed, frame, layer, tag, n)
    return irwin_hall8(w)


def _stream_words(seed, frame, layer, tag, n):
    e = np.arange(n, dtype=np.uint64)
    return philox4x32_10(e & np.uint64(MASK32), e >> np.uint64(32), np.uint64(frame & MASK32),
                         np.uint64(((layer << 8) | tag) & MASK32), seed & MASK32, seed >> 32)


def irwin_hall8(words):
    s = np.zeros(words[0].shape, dtype=np.int64)
    for w in words:
        w = w.astype(np.int64)
        s += (w & 0xFFFF) + (w >> 16)
    return s - IH_MEAN


def normal_bf16(seed, frame, layer, tag, shape, sigma):
    """Near-Gaussian N(0, sigma^2) tensor as bf16 bit patterns (see module recipe).
    Large tensors are drawn in independent chunks on a thread pool (numpy releases
    the GIL); the bits do not depend on the chunking."""
    n = int(np.prod(shape))
    scale = np.float32(sigma / IH_SD)
    out = np.empty(n, dtype=np.uint16)
    args = (frame & MASK32, ((layer << 8) | tag) & MASK32, seed & MASK32, seed >> 32, scale, out)
    bounds = [(a, min(n, a + _CHUNK)) for a in range(0, n, _CHUNK)]
    if len(bounds) <= 1:
        for a, b in bounds:
            _normal_chunk(a, b, *args)
    else:
        from concurrent.futures import ThreadPoolExecutor
        with ThreadPoolExecutor(max_workers=min(16, os.cpu_count() or 1)) as ex:
            list(ex.map(lambda ab: _normal_chunk(ab[0], ab[1], *args), bounds))
    return out.reshape(shape)


def plant_positions(seed, frame, layer, n_heads, n_tokens, n_plant):
    """[H, n_plant] distinct positions per head, partial Fisher-Yates on Philox words."""
    out = np.zeros((n_heads, n_plant), dtype=np.int32)
    if n_plant == 0:
        return out
    blocks = (n_plant + 3) // 4
    h = np.repeat(np.arange(n_heads, dtype=np.uint64), blocks)
    b = np.tile(np.arange(blocks, dtype=np.uint64), n_heads)
    w = philox4x32_10(h, b, np.uint64(frame & MASK32),
                      np.uint64(((layer << 8) | TAG_PLANT) & MASK32), seed & MASK32, seed >> 32)
    words = np.stack(w, axis=1).reshape(n_heads, blocks * 4)
    for hh in range(n_heads):
        perm = np.arange(n_tokens, dtype=np.int64)
        for i in range(n_plant):
            j = i + int(words[hh, i]) % (n_tokens - i)
            perm[i], perm[j] = perm[j], perm[i]
        out[hh] = perm[:n_plant]
    return out


def plant_keys(Q, K, pos, alpha):
    """Rewrite planted key rows in place: alpha * |k_j| * qbar / |qbar| (module recipe)."""
    n, H, d = Q.shape
    q = bf16_bits_to_f32(Q).astype(np.float64)
    qbar = q.sum(axis=0)                     # exact: bf16 values of this range
    for h in range(H):
        nq2 = 0.0
        for e in range(d):
            nq2 = nq2 + qbar[h, e] * qbar[h, e]
        if nq2 == 0.0:
            continue
        for j in pos[h]:
            k = bf16_bits_to_f32(K[j, h]).astype(np.float64)
            nk2 = 0.0
            for e in range(d):
                nk2 = nk2 + k[e] * k[e]
            ratio = (alpha * math.sqrt(nk2)) / math.sqrt(nq2)
            K[j, h] = f32_to_bf16_bits((ratio * qbar[h]).astype(np.float32))
    return K


@dataclass(frozen=True)
class StreamConfig:
    """One synthetic stream: per-layer token shapes and the generator's parameters."""
    name: str
    n_layers: int
    n_heads: int
    head_dim: int
    grid_h: int
    grid_w: int
    n_special: int
    stride: int
    budget: int
    n_frames: int
    seed: int
    sigma: float = 0.125
    n_plant: int = 0
    alpha: float = 3.0
    lognormal_sigma: float = 0.0
    prefill: int = 0
    extra: dict = field(default_factory=dict, compare=False, hash=False)

    @property
    def n_tokens(self):
        return self.grid_h * self.grid_w + self.n_special


CONFIGS = {
    # tiny CPU-checkable stream: 1 layer, 2 heads, 8 frames x 64 tokens, top-1
    "tiny": StreamConfig("tiny", 1, 2, 64, 8, 8, 0, 2, 1, 8, seed=0, n_plant=2, alpha=4.0),
    # one ViT-L-shaped layer, 100 frames
    "vitl_layer": StreamConfig("vitl_layer", 1, 16, 64, 28, 37, 5, 2, 10, 100, seed=1,
                               n_plant=10, alpha=3.0),
    # full 24-layer stack, 1000 frames: the throughput workload
    "vitl_stack_1000": StreamConfig("vitl_stack_1000", 24, 16, 64, 28, 37, 5, 2, 10, 1000,
                                    seed=2, n_plant=10, alpha=3.0),
    # square-resolution long stream, heavy-tailed key norms
    "square_2000": StreamConfig("square_2000", 24, 16, 64, 37, 37, 5, 2, 13, 2000, seed=3,
                                n_plant=13, alpha=3.0, lognormal_sigma=0.5),
    # 52k-token memory prefill, 50 frames
    "long_memory_52k": StreamConfig("long_memory_52k", 24, 16, 64, 28, 37, 5, 2, 10, 50,
                                    seed=5, n_plant=10, alpha=3.0, prefill=52000),
}


def frame_qkv(cfg: StreamConfig, layer: int, frame: int):
    """Q, K, V of one frame of one layer: uint16 [n_tokens, n_heads, head_dim] each."""
    shape = (cfg.n_tokens, cfg.n_heads, cfg.head_dim)
    Q = normal_bf16(cfg.seed, frame, layer, TAG_Q, shape, cfg.sigma)
    K = normal_bf16(cfg.seed, frame, layer, TAG_K, shape, cfg.sigma)
    V = normal_bf16(cfg.seed, frame, layer, TAG_V, shape, cfg.sigma)
    if cfg.lognormal_sigma > 0.0:
        xi = _irwin_hall_stream(cfg.seed, frame, layer, TAG_LOGN, cfg.n_tokens * cfg.n_heads) / IH_SD
        s = np.exp(cfg.lognormal_sigma * xi).astype(np.float32).reshape(cfg.n_tokens, cfg.n_heads, 1)
        K = f32_to_bf16_bits(bf16_bits_to_f32(K) * s)
    if cfg.n_plant > 0:
        pos = plant_positions(cfg.seed, frame, layer, cfg.n_heads, cfg.n_tokens, cfg.n_plant)
        plant_keys(Q, K, pos, cfg.alpha)
    return Q, K, V


def memory_prefill(cfg: StreamConfig, layer: int, rows: int, capacity: int = None):
    """Prefilled memory rows, uint16 [H, capacity, d] each (rows beyond ``rows`` zero)."""
    capacity = rows if capacity is None else capacity
    shape = (cfg.n_heads, rows, cfg.head_dim)
    K = np.zeros((cfg.n_heads, capacity, cfg.head_dim), dtype=np.uint16)
    V = np.zeros_like(K)
    K[:, :rows] = normal_bf16(cfg.seed, PREFILL_FRAME, layer, TAG_MEMK, shape, cfg.sigma)
    V[:, :rows] = normal_bf16(cfg.seed, PREFILL_FRAME, layer, TAG_MEMV, shape, cfg.sigma)
    return K, V
