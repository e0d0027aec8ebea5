"""CPU tests of the attention latency model (the alpha_2 B S^2 term of Eq. (9), Section IV-B)."""
import numpy as np
import pytest

from paper_2607_01701_amd.costmodel import AttentionCostModel, fit, relative_errors


def _synthetic(model, shapes):
    return [(l, h, d, model.predict_lengths(l, h, d)) for l, h, d in shapes]


SHAPES = [([s] * b, h, d) for s in (1024, 4096, 16384) for b in (1, 4) for h, d in ((24, 128), (30, 64))]


def test_fit_recovers_exact_coefficients():
    true = AttentionCostModel(beta2=2.1e-12, beta1=3.3e-9, c0=0.05)
    m, stats = fit(_synthetic(true, SHAPES))
    assert m.beta2 == pytest.approx(true.beta2, rel=1e-9)
    assert m.beta1 == pytest.approx(true.beta1, rel=1e-6)
    assert m.c0 == pytest.approx(true.c0, rel=1e-6, abs=1e-9)
    assert stats["max_rel_err"] < 1e-9


def test_fit_minimises_relative_error_under_noise():
    rng = np.random.default_rng(3)
    true = AttentionCostModel(beta2=2.0e-12, beta1=1.0e-9, c0=0.02)
    samples = [(l, h, d, t * (1 + 0.01 * rng.standard_normal())) for l, h, d, t in _synthetic(true, SHAPES)]
    m, stats = fit(samples)
    assert m.beta2 == pytest.approx(true.beta2, rel=0.02)
    assert stats["rms_rel_err"] < 0.02


def test_bucket_and_pack_forms_agree():
    """B clips of length S in a pack give the paper's alpha_2 B S^2 + alpha_1 B S (k = 1)."""
    m = AttentionCostModel(beta2=1.5e-12, beta1=2e-9, c0=0.1)
    for b, s in ((1, 75600), (8, 4096), (64, 1024)):
        assert m.predict_lengths([s] * b, 24, 128) == pytest.approx(m.predict_bucket(b, s, 24, 128))
        assert m.alpha2(24, 128) * b * s * s + m.alpha1(24, 128) * b * s + m.c0 == pytest.approx(
            m.predict_bucket(b, s, 24, 128))


def test_parallel_degree_divides_compute_term():
    m = AttentionCostModel(beta2=1.5e-12, beta1=2e-9, c0=0.0)
    assert m.predict_bucket(2, 8192, 24, 128, k=4) == pytest.approx(m.predict_bucket(2, 8192, 24, 128) / 4)


def test_zero_length_clips_cost_nothing_and_order_is_irrelevant():
    m = AttentionCostModel(beta2=1.5e-12, beta1=2e-9, c0=0.1)
    a = m.predict_lengths([6912, 0, 1280, 20280], 24, 128)
    b = m.predict_lengths([20280, 1280, 6912], 24, 128)
    assert a == pytest.approx(b)


def test_relative_errors_sign():
    m = AttentionCostModel(beta2=1e-12, beta1=0.0, c0=0.0)
    t = m.predict_lengths([4096], 24, 128)
    e = relative_errors(m, [([4096], 24, 128, 2 * t)])
    assert e[0] == pytest.approx(-0.5)


def test_fit_rejects_too_few_or_bad_samples():
    with pytest.raises(ValueError):
        fit([([1024], 24, 128, 1.0)])
    with pytest.raises(ValueError):
        fit([([1024], 24, 128, 1.0), ([2048], 24, 128, 0.0), ([4096], 24, 128, 3.0)])
