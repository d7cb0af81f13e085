"""The seeded generator: reproducible, and the stated distributions."""
import numpy as np
import torch

from paper_2604_11947_amd import inputs as I


def test_reproducible_and_seed_sensitive():
    a = I.make_inputs(64, 128, 8, "normal", seed=3)
    b = I.make_inputs(64, 128, 8, "normal", seed=3)
    c = I.make_inputs(64, 128, 8, "normal", seed=4)
    for k in ("x_attn", "z", "W_e", "W_d", "g_zt", "g_id"):
        assert torch.equal(a[k], b[k])
        assert not torch.equal(a[k], c[k])
    assert a["x_attn"].dtype == torch.bfloat16 and a["W_e"].dtype == torch.float32
    assert a["W_e"].shape == (128, 8) and a["W_d"].shape == (8, 128)


def test_chunking_does_not_change_the_draw(monkeypatch):
    a = I.make_inputs(50, 64, 4, "token_lognormal", seed=1)
    monkeypatch.setattr(I, "_CHUNK_ROWS", 7)
    b = I.make_inputs(50, 64, 4, "token_lognormal", seed=1)
    for k in ("x_attn", "z", "g_zt", "g_id"):
        assert torch.equal(a[k], b[k])


def test_distributions():
    T, n, r = 2048, 512, 8
    d = I.make_inputs(T, n, r, "student_t3", seed=0)
    for k in ("x_attn", "z"):
        x = d[k].double()
        assert abs(float(x.pow(2).mean().sqrt()) - 1.0) < 1e-2
        assert float(x.abs().max()) > 10.0            # heavy tail
    W = d["W_e"].double()
    assert abs(float(W.var()) * n - 1.0) < 0.05
    assert abs(float(d["W_d"].double().var()) * r - 1.0) < 0.05
    assert abs(float(d["g_zt"].double().std()) - 0.1) < 2e-3

    o = I.make_inputs(256, 2048, 16, "outliers", seed=0)
    ch = o["meta"]["outlier_channels"]
    assert len(ch) == 20 and len(set(ch)) == 20
    col_std = o["z"].double().std(dim=0)
    assert float(col_std[ch].min()) > 10.0
    mask = torch.ones(2048, dtype=torch.bool)
    mask[ch] = False
    assert float(col_std[mask].max()) < 2.0

    g = I.make_inputs(512, 1024, 8, "token_lognormal", seed=0)
    rx = g["x_attn"].double().pow(2).mean(dim=1).sqrt()
    rz = g["z"].double().pow(2).mean(dim=1).sqrt()
    # same per-token factor in both tensors
    assert float(torch.corrcoef(torch.stack([rx.log(), rz.log()]))[0, 1]) > 0.95
    assert abs(float(rx.log().std()) - 0.5) < 0.06


def test_workloads_table():
    w = I.WORKLOADS[I.HEADLINE]
    assert (w.n, w.r, w.tokens) == (4096, 32, 16384)
    for w in I.WORKLOADS.values():
        assert w.n % w.r == 0
    assert I.make_inputs(0, 64, 4)["z"].shape == (0, 64)


def test_bf16_widening_is_exact():
    x = torch.tensor([1.0078125, -3.5, 2 ** -130], dtype=torch.bfloat16)
    np.testing.assert_array_equal(I.bf16_to_f64(x), [1.0078125, -3.5, 2 ** -130])
