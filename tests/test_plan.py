"""The attention work plan (host logic, no device): every queue's iterations are cut
into chunks that cover them exactly once, whatever the shape, device and overrides.

The kernel derives a chunk's iteration range from the plan alone (chunk_range below
restates the rule `include/rv.h` documents for rv_attention_plan), so a partition
failure here would mean keys attended twice or never."""
import itertools

import pytest

from paper_2609_23286_amd import rv

SHAPES = [  # (n_tokens, n_fkeys, mem_len, n_heads)
    (1041, 1041, 0, 16), (1041, 1041, 1000, 16), (1041, 1041, 5000, 16), (1041, 1041, 9990, 16),
    (1041, 1041, 52000, 16), (1041, 0, 11031, 16), (1374, 1374, 26000, 16), (16384, 16384, 3000, 2),
    (65, 65, 0, 1), (333, 333, 1500, 4), (1, 1, 0, 1), (1, 1, 63, 3), (128, 128, 64, 1),
]
DEVICES = [(256, 8), (304, 8), (80, 2), (32, 1), (120, 3)]  # (CUs, XCDs)
OVERRIDES = [  # RV_ATTN_SPLIT, RV_ATTN_FIRST_PCT, RV_ATTN_WG_PER_CU, RV_ATTN_MIN_CHUNK
    {}, {"RV_ATTN_SPLIT": "0"}, {"RV_ATTN_SPLIT": "3"}, {"RV_ATTN_SPLIT": "1"},
    {"RV_ATTN_SPLIT": "0", "RV_ATTN_FIRST_PCT": "100"}, {"RV_ATTN_SPLIT": "0", "RV_ATTN_FIRST_PCT": "101"},
    {"RV_ATTN_SPLIT": "0", "RV_ATTN_FIRST_PCT": "400"}, {"RV_ATTN_WG_PER_CU": "1"},
    {"RV_ATTN_WG_PER_CU": "4", "RV_ATTN_MIN_CHUNK": "1"}, {"RV_ATTN_MIN_CHUNK": "100000"},
    {"RV_ATTN_SPLIT": "0", "RV_ATTN_FIRST_PCT": "133", "RV_ATTN_MIN_CHUNK": "1"},
]
ENV_KEYS = ("RV_ATTN_SPLIT", "RV_ATTN_FIRST_PCT", "RV_ATTN_WG_PER_CU", "RV_ATTN_MIN_CHUNK", "RV_ATTN_SPLIT_SLACK")


def chunk_range(p, c, units):
    """Iterations [first, end) of chunk c of a queue of `units` units (the rule of include/rv.h)."""
    def cut(c):  # lengths in 1/256 iterations
        return (c * p.E if c < p.n_first else p.n_first * p.E + (c - p.n_first) * p.E1) // 256
    return cut(c), min(cut(c + 1), units * p.U)


def check_plan(p, n_tokens, n_fkeys, mem_len, n_heads, n_queues):
    q_tiles = -(-n_tokens // 128)
    T = -(-mem_len // 64) + -(-n_fkeys // 64)
    assert (p.q_tiles, p.n_units, p.T, p.n_queues) == (q_tiles, q_tiles * n_heads, T, n_queues)
    assert p.U >= p.T and p.E >= 256 and p.E1 >= 256 and p.E >= p.E1
    assert p.U == p.T or (p.E % 256 == 0 and p.U % (p.E // 256) == 0 and p.n_first == 0 and p.E1 == p.E)
    base = list(p.unit_base)[: n_queues + 1]
    assert base[0] == 0 and base[-1] == p.n_units and base == sorted(base)
    per_queue = p.grid // n_queues
    assert p.grid % n_queues == 0 and 0 <= p.n_first <= per_queue
    total = 0
    for q in range(n_queues):
        iters = (base[q + 1] - base[q]) * p.U
        n = p.n_chunks[q]
        assert p.chunk_base[q] == total and 0 <= n <= per_queue
        total += n
        if iters == 0:
            assert n == 0
            continue
        ranges = [chunk_range(p, c, base[q + 1] - base[q]) for c in range(n)]
        # consecutive, non-empty chunks from iteration 0 whose last one reaches the end
        assert ranges[0][0] == 0 and ranges[-1][1] == iters
        assert all(a < b for a, b in ranges) and all(r[1] == s[0] for r, s in zip(ranges, ranges[1:]))
    assert total == p.total_chunks


@pytest.mark.parametrize("shape", SHAPES)
def test_chunks_partition_every_queue(shape, monkeypatch):
    for k in ENV_KEYS:
        monkeypatch.delenv(k, raising=False)
    for (n_cus, n_queues), env in itertools.product(DEVICES, OVERRIDES):
        with monkeypatch.context() as m:
            for k, v in env.items():
                m.setenv(k, v)
            p = rv.attention_plan(*shape, n_cus, n_queues)
            check_plan(p, *shape, n_queues)


def test_first_dispatched_chunks_are_longer_in_stream_k(monkeypatch):
    """At the benchmark's long contexts the plan is stream-K in its unit-aligned form: the
    later chunks are a quarter of a unit (T/4 tiles, so four of them end exactly on each
    unit boundary of the queue's last 8 of 18 units) and the first chunk of each CU's pair
    shares the first 10 units with the other 31 (125 % of a later chunk's tiles); the
    fractional lengths give every one of the 512 workgroup slots a chunk of one of two
    neighbouring integer lengths.  With RV_ATTN_FIRST_PCT set, the share is that per cent
    (rounded up, in 1/256 tiles)."""
    for k in ENV_KEYS:
        monkeypatch.delenv(k, raising=False)
    p = rv.attention_plan(1041, 1041, 9990, 16, 256, 8)
    assert p.U == p.T == 174 and p.n_first == 32
    assert p.E1 * 4 == p.T * 256 and p.E * 32 == 10 * p.T * 256 and p.E * 100 == p.E1 * 125
    assert p.grid == 512
    units = p.unit_base[1] - p.unit_base[0]
    lengths = [b - a for a, b in (chunk_range(p, c, units) for c in range(p.n_chunks[0]))]
    assert set(lengths[:32]) <= {p.E // 256, -(-p.E // 256)}
    assert set(lengths[32:-1]) <= {p.E1 // 256, -(-p.E1 // 256)} and 1 <= lengths[-1] <= -(-p.E1 // 256)
    monkeypatch.setenv("RV_ATTN_FIRST_PCT", "140")
    p = rv.attention_plan(1041, 1041, 9990, 16, 256, 8)
    assert p.n_first == 32 and p.E == -(-p.E1 * 140 // 100) and p.grid == 512


@pytest.mark.parametrize("M", [1500, 2500, 4990, 7770, 9990])
def test_aligned_plans_start_every_unit_at_a_chunk_boundary(M, monkeypatch):
    """In the unit-aligned form no later chunk holds tiles of two units, and the first
    chunks end on a unit boundary (for every queue, including those with fewer units)."""
    for k in ENV_KEYS:
        monkeypatch.delenv(k, raising=False)
    p = rv.attention_plan(1041, 1041, M, 16, 256, 8)
    assert p.U == p.T and p.n_first == 32 and (p.T * 256) % p.E1 == 0
    assert p.n_first * p.E % (p.T * 256) == 0
    for q in range(8):
        units = p.unit_base[q + 1] - p.unit_base[q]
        for c in range(p.n_first, p.n_chunks[q]):
            a, b = chunk_range(p, c, units)
            if b > a:
                assert a // p.T == (b - 1) // p.T, (q, c, a, b)


def test_plan_rejects_bad_sizes():
    for args in ((0, 0, 0, 16, 256, 8), (1041, 1042, 0, 16, 256, 8), (1041, 1041, -1, 16, 256, 8),
                 (1041, 1041, 0, 0, 256, 8), (1041, 1041, 0, 16, 0, 8), (1041, 1041, 0, 16, 256, 17)):
        with pytest.raises(rv.RVError):
            rv.attention_plan(*args)
