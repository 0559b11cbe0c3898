"""The seeded generator is deterministic and produces the documented shapes."""
import numpy as np

from paper_2609_38978_amd import synth


def test_shapes_and_determinism():
    cfg = synth.CONFIGS["tiny"]
    a = synth.make_head(cfg, 0)
    b = synth.make_head(cfg, 0)
    for x, y in zip(a, b):
        assert x.shape == (4096, 64) and x.dtype == np.float32
        assert np.array_equal(x.view(np.uint32), y.view(np.uint32))
    assert not np.array_equal(a[0], a[1])  # independent noise per tensor


def test_bf16_rounding_is_rne_and_representable():
    x = np.array([1.0, 1.00390625, 1.01171875, -2.0 ** -130, 3.0e38], np.float32)
    r = synth.bf16_round(x)
    assert np.all((r.view(np.uint32) & 0xFFFF) == 0)
    # 1 + 2^-8 is a tie between 1 and 1 + 2^-7: even mantissa -> 1.0
    assert r[1] == 1.0
    # 1 + 3*2^-8 ties between 1+2^-7 and 1+2^-6 -> even -> 1 + 2^-6
    assert r[2] == np.float32(1.015625)
    cfg = synth.CONFIGS["medium"]
    q, k, v = synth.make_head(cfg.with_(grid=(2, 8, 8)), 1)
    for t in (q, k, v):
        assert np.all((t.view(np.uint32) & 0xFFFF) == 0)


def test_config_sizes():
    C = synth.CONFIGS
    assert (C["tiny"].N, C["tiny"].C) == (4096, 64)
    assert (C["medium"].N, C["medium"].C) == (16384, 256)
    assert (C["wan"].N, C["wan"].C) == (75600, 1182)
    assert (C["hunyuan"].N, C["hunyuan"].C) == (119056, 1861)


def test_text_tokens_and_q_scale():
    cfg = synth.CONFIGS["hunyuan"].with_(grid=(1, 4, 8))
    q, k, v = synth.make_head(cfg, 0)
    assert q.shape == (32 + 256, 128)
    w = synth.CONFIGS["wan"].with_(grid=(1, 4, 8))
    w1 = w.with_(q_scale=None)
    qa, ka, _ = synth.make_head(w, 3)
    qb, kb, _ = synth.make_head(w1, 3)
    assert np.array_equal(ka, kb)
    ratio = np.median(np.abs(qa) / np.maximum(np.abs(qb), 1e-3))
    assert 0.45 < ratio < 2.05
