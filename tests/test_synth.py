"""The seeded input generator: Philox known answers, distribution and planting."""
import os

import numpy as np

from paper_2609_23286_amd import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_philox_known_answers():
    rows = [l.split() for l in open(os.path.join(GOLDEN, "philox4x32_10_kat.txt"))
            if l.strip() and not l.startswith("#")]
    assert len(rows) == 3
    for r in rows:
        v = [int(x, 16) for x in r]
        out = synth.philox4x32_10(*v[:6])
        assert [int(o) for o in out] == v[6:]


def test_bf16_rounding_is_nearest_even():
    x = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, 1.0 + 2 ** -9, -2.5, 0.0],
                 dtype=np.float32)
    # 1+2^-8 is a tie between 1 and 1+2^-7 -> even (1); 1+3*2^-8 ties up to 1+2^-6
    back = synth.bf16_bits_to_f32(synth.f32_to_bf16_bits(x))
    assert back.tolist() == [1.0, 1.0, 1.0 + 2 ** -6, 1.0, -2.5, 0.0]


def test_normal_moments_and_determinism():
    a = synth.normal_bf16(7, 3, 2, synth.TAG_K, (4096, 64), 0.125)
    b = synth.normal_bf16(7, 3, 2, synth.TAG_K, (4096, 64), 0.125)
    c = synth.normal_bf16(7, 4, 2, synth.TAG_K, (4096, 64), 0.125)
    assert (a == b).all() and not (a == c).all()
    x = synth.bf16_bits_to_f32(a).astype(np.float64)
    assert abs(x.mean()) < 3e-3 and abs(x.std() - 0.125) < 2e-3
    assert np.abs(x).max() < 0.125 * 4.95


def test_planted_rows_follow_mean_query_direction():
    cfg = synth.CONFIGS["vitl_layer"]
    Q, K, _ = synth.frame_qkv(cfg, 0, 5)
    pos = synth.plant_positions(cfg.seed, 5, 0, cfg.n_heads, cfg.n_tokens, cfg.n_plant)
    assert all(len(set(p)) == cfg.n_plant for p in pos)
    qbar = synth.bf16_bits_to_f32(Q).astype(np.float64).sum(0)
    for h in (0, 15):
        for j in pos[h]:
            k = synth.bf16_bits_to_f32(K[j, h]).astype(np.float64)
            cos = k @ qbar[h] / np.linalg.norm(k) / np.linalg.norm(qbar[h])
            assert cos > 0.9999
            assert 2.0 < np.linalg.norm(k) < 4.5       # ~3x the ~1.0 norm of a key
