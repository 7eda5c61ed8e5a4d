"""The seeded input generators: deterministic per (config, head), right shapes,
bf16-exact values for bf16 workloads."""
import numpy as np

from synth import CONFIGS, bf16_round, keep_to_k, make_config, mixture_inputs, field_inputs


def test_bf16_round_is_rne_and_idempotent():
    x = np.array([1.0, 1.00390625, 1.005859375, -2.5, 3.0e-39, 65504.0], dtype=np.float32)
    r = bf16_round(x)
    assert (r.view(np.uint32) & 0xFFFF == 0).all()
    assert r[1] == 1.0  # halfway, ties to even
    assert r[2] == np.float32(1.0078125)
    assert np.array_equal(bf16_round(r), r)


def test_mixture_deterministic_and_head_independent():
    a = mixture_inputs(3, 2, 100, 8, "bf16")
    b = mixture_inputs(3, 2, 100, 8, "bf16")
    for x, y in zip(a, b):
        assert np.array_equal(x, y)
        assert x.shape == (2, 100, 8) and x.dtype == np.float32
        assert np.array_equal(bf16_round(x), x)
    c = mixture_inputs(4, 2, 100, 8, "bf16")
    assert not np.array_equal(a[0], c[0])


def test_field_shapes_and_correlation():
    q, k, v = field_inputs(0, 1, (6, 8, 10), 4, "f32", corr_len=2.0)
    assert q.shape == (1, 480, 4)
    # queries and keys share the field: strongly correlated per channel
    cor = np.corrcoef(q[0, :, 0], k[0, :, 0])[0, 1]
    assert cor > 0.8


def test_named_config_subset_of_heads():
    q, k, v = make_config(1)
    assert q.shape == (1, 1024, 64) and q.dtype == np.float32
    q2, _, _ = make_config(1, heads=[0])
    assert np.array_equal(q, q2)
    cfg = CONFIGS[5]
    assert cfg.params["grid"] == (21, 45, 80) and cfg.n == 21 * 45 * 80


def test_keep_to_k():
    assert keep_to_k(1 / 8, 512) == 64
    assert keep_to_k(1 / 4, 1182) == 296
    assert keep_to_k(1 / 16, 591) == 37
    assert keep_to_k(1.0, 16) == 16
