"""Determinism and shape of the seeded input generators."""
import numpy as np

from paper_2609_24802_amd import synth


def test_chunked_streams_are_deterministic(monkeypatch):
    a = synth.normal_f32((1 << 24) + 12345, (7, 1))
    monkeypatch.setattr(synth, "_threads", lambda: 1)
    b = synth.normal_f32((1 << 24) + 12345, (7, 1))
    assert synth.fingerprint(a) == synth.fingerprint(b)
    c = synth.randint_i32(1000, 50, (7, 2))
    assert c.min() >= 0 and c.max() < 50


def test_zipf_degrees():
    deg = synth.zipf_degrees(100_000, 1_600_000, 2.1, 10_000, (8,))
    assert deg.sum() == 1_600_000 and deg.max() <= 10_000 and deg.min() >= 1
    deg2 = synth.zipf_degrees(100_000, 1_600_000, 2.1, 10_000, (8,))
    assert np.array_equal(deg, deg2)
    # heavy tail: most rows short, a large share of edges in long rows
    assert np.mean(deg <= 8) > 0.6
    assert deg[deg >= 64].sum() > 0.4 * deg.sum()


def test_uniform_small_config():
    g = synth.csr_uniform_small()
    rp, col = g["row_ptr"], g["col"]
    assert rp.shape == (1025,) and rp[-1] == 8192 and col.shape == (8192,)
    assert g["x"].min() >= -1 and g["x"].max() < 1 and g["w"].min() >= 0 and g["w"].max() < 1
    h = synth.csr_uniform_small()
    assert synth.fingerprint(rp, col, g["w"], g["x"]) == synth.fingerprint(h["row_ptr"], h["col"], h["w"], h["x"])
