"""The Sec. 4.1 cost model's fitting, on the CPU: exact recovery of known
coefficients from noiseless samples on the paper's power-of-two grid, both
interaction forms, the swap model, and how an iteration combines them."""

import numpy as np
import pytest

from paper_2504_09590_amd import costmodel as cm


def _samples(phase, a0, a1, b, form, grid):
    out = []
    for batch, n in grid:
        ln = batch * n if phase == "prefill" else batch
        la = ln if phase == "prefill" else batch * n
        pairs = batch * n * n if phase == "prefill" else batch * n
        inter = ln * la if form == "paper" else pairs
        out.append(cm.Sample(phase, ln, la, pairs, a0 * ln + a1 * inter + b, batch))
    return out


def test_power_grid():
    assert cm.power_grid(128, 4096) == [128, 256, 512, 1024, 2048, 4096]
    assert cm.power_grid(3, 2) == []


@pytest.mark.parametrize("form", cm.FORMS)
@pytest.mark.parametrize("phase", ["prefill", "decode"])
def test_fit_recovers_coefficients(form, phase):
    grid = [(b, n) for n in cm.power_grid(128, 4096) for b in cm.power_grid(1, 8)]
    true = (0.013, 2.5e-6, 7.0)
    s = _samples(phase, *true, form, grid)
    coef = cm.fit(s, form)
    assert np.allclose(coef, true, rtol=1e-9, atol=1e-9)
    model = cm.CostModel(coef={f"{phase}/{form}": coef})
    assert cm.relative_errors(model, s, form).max() < 1e-9


def test_forms_agree_for_one_request():
    # one request: Ln * La equals n * a, so the two forms are the same model
    for n in (64, 512):
        assert np.allclose(cm.features("paper", n, n, n * n), cm.features("per_request", n, n, n * n))


def test_swap_fit_and_iteration():
    sizes = [2 ** k for k in range(16, 29)]
    t_d2h = [s / 50e3 + 12.0 for s in sizes]          # 50 GB/s = 5e4 bytes per us, 12 us fixed
    coef = cm.fit_swap(sizes, t_d2h)
    assert np.allclose(coef, [1 / 50e3, 12.0], rtol=1e-9)
    model = cm.CostModel(coef={"prefill/paper": [0.01, 0.0, 5.0], "decode/paper": [0.1, 0.0, 2.0]},
                         swap={"d2h": list(coef), "h2d": list(coef)})
    t_exec = 0.01 * 2048 + 5.0 + 0.1 * 128 + 2.0
    t_swap = 2 * ((1 << 22) / 50e3 + 12.0)
    got_serial = model.iteration_us(prefill=(2048, 2048, 0), decode=(128, 10 ** 6, 0),
                                    nbytes_out=1 << 22, nbytes_in=1 << 22)
    got_overlap = model.iteration_us(prefill=(2048, 2048, 0), decode=(128, 10 ** 6, 0),
                                     nbytes_out=1 << 22, nbytes_in=1 << 22, overlap=True)
    assert got_serial == pytest.approx(t_exec + t_swap)
    assert got_overlap == pytest.approx(max(t_exec, t_swap))
    assert model.iteration_us() == 0.0


def test_json_round_trip():
    m = cm.CostModel(coef={"decode/paper": [1.0, 2.0, 3.0]}, swap={"d2h": [1e-5, 4.0]})
    m2 = cm.CostModel.from_json(m.to_json())
    assert m2.coef == m.coef and m2.swap == m.swap
    assert float(m2.predict("decode", 10, 20)) == pytest.approx(1 * 10 + 2 * 200 + 3)


def test_fit_keeps_every_term_non_negative():
    # a decode profile whose time barely grows with the batch: an unconstrained
    # fit gives the per-request term a small negative value, the fit clamps it
    grid = [(b, c) for b in cm.power_grid(8, 256) for c in cm.power_grid(256, 8192)]
    s = []
    for b, c in grid:
        t = 22.0 + 6.0e-4 * b * c - 0.002 * b
        s.append(cm.Sample("decode", b, b * c, b * c, t, b))
    free, *_ = np.linalg.lstsq(cm.features("per_request", [x.ln for x in s], [x.la for x in s],
                                           [x.pairs for x in s]) / np.array([x.t_us for x in s])[:, None],
                               np.ones(len(s)), rcond=None)
    assert free[0] < 0
    coef = cm.fit(s, "per_request")
    assert np.all(coef >= 0) and coef[0] == 0.0
    model = cm.CostModel(coef={"decode/per_request": coef})
    assert cm.relative_errors(model, s, "per_request").max() < 0.02
