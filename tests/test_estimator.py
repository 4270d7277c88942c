"""Section 5 estimators: the fits recover the coefficients of the paper's
time forms from noise-free samples of those forms (closed forms written out
here, not by the estimator), and the KV memory bound is mu + 2 sigma."""
import numpy as np
import pytest

from paper_2504_03651_amd.estimator import (DecodeModel, Estimator, MixedModel, PrefillModel,
                                            kv_memory_bound)


def test_prefill_fit_recovers_the_quadratic_and_the_floor():
    alpha, beta, c = 2.0e-8, 3.0e-5, 0.02
    l = np.array([16, 32, 64, 128, 256, 512, 1024, 2048, 4096, 8192], float)
    t = np.maximum(alpha * l * l + beta * l, c)
    m = PrefillModel.fit(l, t)
    assert m.c == pytest.approx(c, rel=1e-12)
    assert m.alpha == pytest.approx(alpha, rel=1e-6) and m.beta == pytest.approx(beta, rel=1e-6)
    # below the knee the floor, above it the polynomial
    assert m.predict(16) == pytest.approx(c) and m.predict(8192) == pytest.approx(t[-1])


def test_decode_fit_per_batch_size():
    rng = np.random.default_rng(0)
    truth = {16: (1e-6, 2e-5), 64: (5e-7, 8e-5), 256: (0.0, 3e-4)}
    batches, times = [], []
    for n, (g, d) in truth.items():
        for _ in range(6):
            L = rng.integers(64, 4096, size=n)
            L[0] = int(rng.integers(4096, 32768))
            batches.append(L)
            times.append(g * L.max() + d * L.mean())
    m = DecodeModel.fit(batches, times)
    assert m.sizes == [16, 64, 256]
    for n, (g, d) in truth.items():
        gg, dd, ee = m.coef(n)
        assert ee == 0.0
        assert gg == pytest.approx(g, abs=1e-12) and dd == pytest.approx(d, rel=1e-6)
    # delta interpolates linearly between calibrated sizes
    assert m.coef(40)[1] == pytest.approx((2e-5 + 8e-5) / 2, rel=1e-6)


def test_mixed_fit_and_composition():
    tp = np.array([0.1, 0.5, 1.0, 2.0])
    td = np.array([0.4, 0.3, 0.2, 1.5])
    lam = 0.7
    tb = lam * np.maximum(tp, td) + (1 - lam) * np.minimum(tp, td)
    m = MixedModel.fit(tp, td, tb)
    assert m.lam == pytest.approx(lam, rel=1e-12)
    est = Estimator(PrefillModel(0.0, 1e-3, 0.0), DecodeModel([8], [0.0], [1e-3]), m)
    # prefill requests run one after another; decode alone; both by lam
    assert est.batch_time([100, 200], []) == pytest.approx(0.3)
    assert est.batch_time([], [10] * 8) == pytest.approx(0.01)
    assert est.batch_time([100], [10] * 8) == pytest.approx(0.7 * 0.1 + 0.3 * 0.01)
    d = Estimator.from_dict(est.to_dict())
    assert d.batch_time([100], [10] * 8) == pytest.approx(est.batch_time([100], [10] * 8))


def test_kv_memory_bound_is_mean_plus_two_sigma():
    x = np.array([10.0, 12.0, 14.0, 16.0, 18.0])   # mean 14, population sigma sqrt(8)
    assert kv_memory_bound(x) == pytest.approx(14 + 2 * np.sqrt(8.0))
    rng = np.random.default_rng(1)
    y = rng.normal(100.0, 5.0, size=200000)
    frac = float(np.mean(y <= kv_memory_bound(y)))
    assert abs(frac - 0.97725) < 0.003   # one-sided normal quantile at 2 sigma


def test_decode_intercept_form():
    rng = np.random.default_rng(2)
    batches = [rng.integers(64, 4096, size=32) for _ in range(8)]
    t = [4e-7 * b.max() + 6e-5 * b.mean() + 0.04 for b in batches]
    m = DecodeModel.fit(batches, t, intercept=True)
    g, d, e = m.coef(32)
    assert g == pytest.approx(4e-7, rel=1e-6) and d == pytest.approx(6e-5, rel=1e-6)
    assert e == pytest.approx(0.04, rel=1e-9)
    assert DecodeModel.fit(batches, t).coef(32)[2] == 0.0   # the paper's form: no constant


def test_mixed_sum_form():
    tp = np.array([0.1, 0.5, 1.0])
    td = np.array([0.4, 0.3, 0.2])
    m = MixedModel.fit(tp, td, tp + td - 0.03, form="sum")
    assert m.kappa == pytest.approx(0.03) and m.predict(0.2, 0.1) == pytest.approx(0.27)


def test_kernel_reading_of_the_forms():
    est = Estimator(PrefillModel(1e-6, 1e-3, 0.05),
                    DecodeModel([8, 32], [1e-4, 2e-4], [1e-3, 3e-3], [0.01, 0.02]),
                    MixedModel(kappa=0.005, form="sum"))
    # one whole prompt, no sharing: the paper's forms exactly
    assert est.batch_time_kernel([(300, 0)], []) == pytest.approx(est.batch_time([300], []))
    L = [100, 200, 300, 400] * 4
    assert est.batch_time_kernel([], L, sum(L)) == pytest.approx(est.batch_time([], L))
    assert est.batch_time_kernel([(300, 0)], L) == pytest.approx(est.batch_time([300], L))
    # chunks share one launch: the floor is paid once, work terms add
    assert est.batch_time_kernel([(10, 0), (10, 0)], []) == pytest.approx(0.05)
    assert est.batch_time([10, 10], []) == pytest.approx(0.10)
    # a chunk after cached context: n ctx + n^2 / 2 pairs at 2 alpha each
    assert est.batch_time_kernel([(100, 1000)], []) == pytest.approx(
        max(1e-6 * (100 * 100 + 2 * 100 * 1000) + 1e-3 * 100, 0.05))
    # shared prefix blocks read once: the mean term takes distinct tokens per row
    g, d, e = est.decode.coef(16)
    assert est.batch_time_kernel([], L, 1000) == pytest.approx(g * 400 + d * 1000 / 16 + e)


def test_prefill_fit_on_batches_of_chunks_recovers_known_coefficients():
    # several chunks per batch, some after cached context, priced by the
    # kernel reading: alpha sum(n^2 + 2 n ctx) + beta sum(n), floor once
    from paper_2504_03651_amd.calibrate import PREFILL_BATCHES
    alpha, beta, c = 3.0e-9, 2.0e-5, 0.025
    batches = [[(l, ctx)] * k for k, l, ctx in PREFILL_BATCHES]
    t = [max(sum(alpha * (n * n + 2 * n * x) + beta * n for n, x in b), c) for b in batches]
    m = PrefillModel.fit_chunks(batches, t)
    assert m.alpha == pytest.approx(alpha, rel=1e-6) and m.beta == pytest.approx(beta, rel=1e-6)
    assert m.c == pytest.approx(c)
    # one prompt of l tokens from scratch is the paper's alpha l^2 + beta l
    assert m.predict_chunks([(4096, 0)]) == pytest.approx(float(m.predict(4096)))
