"""Pins for the oracle's online-softmax attention (Section 5.2 and the appendix on causal attention).

Each check comes from something other than the oracle's own formula: the IEEE definitions (through
numpy's own conversions), closed forms, the combine law of the online-softmax state printed in
Section 5.2, invariances of the softmax, and the relation's structure (the triangular row i is the
dense relation over the first i + 1 tokens)."""
import math

import numpy as np
import pytest

import oracle
from paper_2609_24802_amd import synth


def bits(a, dtype="f16"):
    return synth.f32_to_half_bits(np.asarray(a, np.float32), dtype)


def test_f16_widening_all_patterns():
    allb = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    got = oracle.half_to_double(allb, "f16")
    ref = allb.view(np.float16).astype(np.float64)
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], ref[~nan])
    # signed zeros keep their sign
    assert math.copysign(1.0, got[0x8000]) == -1.0


def test_bf16_widening_all_patterns():
    allb = np.arange(1 << 16, dtype=np.uint32)
    got = oracle.half_to_double(allb.astype(np.uint16), "bf16")
    ref = (allb << 16).astype(np.uint32).view(np.float32).astype(np.float64)
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], ref[~nan])


@pytest.mark.parametrize("dtype", ["f16", "bf16"])
def test_first_token_reads_only_itself(dtype):
    d = synth.attention_inputs(37, 3, 64, dtype)
    y, ya, lse = oracle.attention_fwd(d["q"], d["k"], d["v"], d["scale"], dtype, "triangular", pts=[0])
    v0 = oracle.half_to_double(d["v"][:, 0, :], dtype).reshape(3, 64)
    assert np.array_equal(y[0], v0)
    assert np.array_equal(ya[0], np.abs(v0))
    q0 = oracle.half_to_double(d["q"][:, 0, :], dtype).reshape(3, 64)
    k0 = oracle.half_to_double(d["k"][:, 0, :], dtype).reshape(3, 64)
    s00 = (q0 * k0).sum(1) * float(d["scale"])
    assert np.allclose(lse[0], s00, rtol=1e-14, atol=1e-14)


@pytest.mark.parametrize("relation", ["triangular", "dense"])
def test_zero_query_gives_the_mean_of_the_values(relation):
    n, H, D = 40, 2, 64
    d = synth.attention_inputs(n, H, D, "f16")
    q = np.zeros_like(d["q"])
    y, _, lse = oracle.attention_fwd(q, d["k"], d["v"], d["scale"], "f16", relation)
    v = oracle.half_to_double(d["v"], "f16").reshape(H, n, D)
    for i in range(n):
        last = i if relation == "triangular" else n - 1
        np.testing.assert_allclose(y[i], v[:, :last + 1].mean(1), rtol=1e-12, atol=1e-14)
        np.testing.assert_allclose(lse[i], math.log(last + 1), rtol=1e-13)


def test_two_token_closed_form_and_head_separation():
    # head 0: q1 = (1, 0), k0 = (2, 0), k1 = (0, 3), scale 0.5 -> s10 = 1, s11 = 0
    # head 1: q and k swap roles, so a kernel that used <k_i, q_j> gets head 0 wrong
    D = 2
    q = np.array([[[0, 1], [1, 0]], [[2, 0], [0, 3]]], np.float32)
    k = np.array([[[2, 0], [0, 3]], [[0, 1], [1, 0]]], np.float32)
    v = np.array([[[1, 2], [-3, 4]], [[5, -6], [7, 8]]], np.float32)
    y, ya, lse = oracle.attention_fwd(bits(q), bits(k), bits(v), 0.5, "f16", "triangular")
    v = v.astype(np.float64)
    e = math.e
    # head 0, token 1: weights (e, 1) / (e + 1) on v0, v1
    np.testing.assert_allclose(y[1, 0], (e * v[0, 0] + v[0, 1]) / (e + 1), rtol=1e-14)
    np.testing.assert_allclose(lse[1, 0], math.log(e + 1), rtol=1e-14)
    # head 1, token 1: q1 = (0, 3), k0 = (0, 1), k1 = (1, 0) -> s10 = 1.5, s11 = 0
    w0 = math.exp(1.5)
    np.testing.assert_allclose(y[1, 1], (w0 * v[1, 0] + v[1, 1]) / (w0 + 1), rtol=1e-14)
    np.testing.assert_allclose(ya[1, 1], (w0 * np.abs(v[1, 0]) + np.abs(v[1, 1])) / (w0 + 1), rtol=1e-14)
    # dense: token 0 also reads token 1; head 0: q0 = (0, 1): s00 = 0, s01 = 1.5
    yd, _, _ = oracle.attention_fwd(bits(q), bits(k), bits(v), 0.5, "f16", "dense")
    np.testing.assert_allclose(yd[0, 0], (v[0, 0] + w0 * v[0, 1]) / (1 + w0), rtol=1e-14)


@pytest.mark.parametrize("dtype", ["f16", "bf16"])
def test_online_softmax_combine_law(dtype):
    """Section 5.2: two nonempty states (m, l, o) over disjoint key sets combine by rescaling into
    the common maximum.  With the finalized state of a set being (lse, 1, y), combining the states
    of halves A and B must give the state of A u B."""
    nA, nB, H, D = 23, 41, 2, 64
    d = synth.attention_inputs(nA + nB, H, D, dtype, sigma=2.0)
    q, k, v = d["q"], d["k"], d["v"]
    qq = np.repeat(q[:, :1], nA + nB, axis=1)          # every query row is the same vector

    def state(lo, hi):
        yy, _, ll = oracle.attention_fwd(qq[:, lo:hi], k[:, lo:hi], v[:, lo:hi], d["scale"], dtype, "dense",
                                         pts=[0])
        return yy[0], ll[0]

    yA, lA = state(0, nA)
    yB, lB = state(nA, nA + nB)
    yAB, lAB = state(0, nA + nB)
    m = np.maximum(lA, lB)
    l = np.exp(lA - m) + np.exp(lB - m)
    o = (np.exp(lA - m)[:, None] * yA + np.exp(lB - m)[:, None] * yB) / l[:, None]
    np.testing.assert_allclose(yAB, o, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(lAB, m + np.log(l), rtol=1e-13)


def test_shift_of_all_keys_leaves_outputs_unchanged():
    """Adding one vector c to every key shifts row i's scores by scale * <q_i, c>, the same for all j,
    which the softmax cancels.  Small integers keep every input exact in binary16."""
    rng = np.random.default_rng(5)
    n, H, D = 30, 2, 16
    q = rng.integers(-2, 3, (H, n, D)).astype(np.float32)
    k = rng.integers(-2, 3, (H, n, D)).astype(np.float32)
    v = rng.integers(-4, 5, (H, n, D)).astype(np.float32)
    c = rng.integers(-3, 4, (H, 1, D)).astype(np.float32)
    sc = 0.25
    for rel in ("triangular", "dense"):
        y0, _, l0 = oracle.attention_fwd(bits(q), bits(k), bits(v), sc, "f16", rel)
        y1, _, l1 = oracle.attention_fwd(bits(q), bits(k + c), bits(v), sc, "f16", rel)
        np.testing.assert_allclose(y1, y0, rtol=1e-12, atol=1e-12)
        shift = sc * np.einsum("hnd,hd->nh", q, c[:, 0])
        np.testing.assert_allclose(l1, l0 + shift, rtol=1e-12, atol=1e-12)


def test_triangular_row_is_dense_over_its_prefix():
    n, H, D = 33, 2, 64
    d = synth.attention_inputs(n, H, D, "bf16")
    yt, at, lt = oracle.attention_fwd(d["q"], d["k"], d["v"], d["scale"], "bf16", "triangular")
    for i in (0, 1, 7, 32):
        yd, ad, ld = oracle.attention_fwd(d["q"][:, :i + 1], d["k"][:, :i + 1], d["v"][:, :i + 1], d["scale"],
                                          "bf16", "dense", pts=[i])
        assert np.array_equal(yt[i], yd[0]) and np.array_equal(lt[i], ld[0]) and np.array_equal(at[i], ad[0])


def test_dominant_key_selects_its_value():
    rng = np.random.default_rng(9)
    n, H, D = 12, 1, 8
    q = np.ones((H, n, D), np.float32)
    k = rng.integers(-1, 2, (H, n, D)).astype(np.float32)
    k[0, 4] = 16.0                          # s_i4 - s_ij >= 0.5 * 8 * (16 - 1) = 60 for every j != 4
    v = rng.integers(-4, 5, (H, n, D)).astype(np.float32)
    y, _, _ = oracle.attention_fwd(bits(q), bits(k), bits(v), 0.5, "f16", "dense")
    np.testing.assert_allclose(y[:, 0], np.broadcast_to(v[0, 4], (n, D)), rtol=0, atol=1e-20)
    yt, _, _ = oracle.attention_fwd(bits(q), bits(k), bits(v), 0.5, "f16", "triangular")
    np.testing.assert_allclose(yt[4:, 0], np.broadcast_to(v[0, 4], (n - 4, D)), rtol=0, atol=1e-20)


def test_constant_values_are_reproduced():
    n, H, D = 50, 2, 64
    d = synth.attention_inputs(n, H, D, "f16", sigma=3.0)
    v = bits(np.full((H, n, D), -1.5, np.float32))
    y, ya, _ = oracle.attention_fwd(d["q"], d["k"], v, d["scale"], "f16", "triangular")
    np.testing.assert_allclose(y, -1.5, rtol=1e-14)
    np.testing.assert_allclose(ya, 1.5, rtol=1e-14)


def test_rejects_unknown_relation():
    d = synth.attention_inputs(4, 1, 64, "f16")
    with pytest.raises(KeyError):
        oracle.attention_fwd(d["q"], d["k"], d["v"], d["scale"], "f16", "banded")
