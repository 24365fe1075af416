"""GPU parity of the online-softmax attention path (triangular and dense relations) against the oracle.

Tolerance, per output element, from the arithmetic of the path:
  - the normalized weights enter the value product rounded to the 16-bit input type:
    |error| <= u * sum_j p_ij |v_jd| = u * yabs  (u = 2^-11 for binary16, 2^-8 for bfloat16);
  - the output is rounded once to the same type: <= u * |y| <= u * yabs;
  - fp32 scores (exact products, fp32 sums over the width), exp2 and fp32 mass/accumulator sums:
    well under 1e-4 * yabs at these widths and score ranges;
  - absolute floors: 2^-24 for outputs in the binary16 subnormal range, and n * 2^-25 * max|v| for
    binary16 weights rounded into its subnormal range.
so |y_gpu - y_oracle| <= (2u + 1e-4) * yabs + floors.  The mass is summed from the same rounded
weights as the numerator, so lse = m + log(sum of rounded weights) carries up to u of absolute error
from that rounding: |lse error| <= u + 1e-4 * (1 + |lse|).
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_24802_amd import synth

pytestmark = pytest.mark.gpu

U = {"f16": 2.0 ** -11, "bf16": 2.0 ** -8}
TORCH_DT = {"f16": torch.float16, "bf16": torch.bfloat16}


def dev(bits, dtype):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).cuda().view(TORCH_DT[dtype])


def to_f64(t):
    return t.float().cpu().numpy().astype(np.float64)


def check(y, lse, ref, yabs, ref_lse, n, vmax, dtype, what):
    u = U[dtype]
    floor = 2.0 ** -24 + (n * 2.0 ** -25 * vmax if dtype == "f16" else 0.0)
    err = np.abs(y - ref)
    bound = (2 * u + 1e-4) * yabs + floor
    bad = err > bound
    if bad.any():
        k = np.unravel_index(np.argmax(np.where(bad, err - bound, -np.inf)), err.shape)
        raise AssertionError(f"{what}: {int(bad.sum())} of {err.size} exceed the bound; worst at {k}: got {y[k]!r} "
                             f"ref {ref[k]!r} yabs {yabs[k]!r}")
    if lse is not None:
        lerr = np.abs(lse - ref_lse)
        assert (lerr <= u + 1e-4 * (1 + np.abs(ref_lse))).all(), f"{what}: lse max error {lerr.max()}"
    return float((err / (yabs + 1e-30)).max())


def run(lib, inp, relation, pts=None, layout="hnd"):
    dt = inp["dtype"]
    q, k, v = (dev(inp[a], dt) for a in ("q", "k", "v"))
    if layout == "nhd":
        q, k, v = (t.permute(1, 0, 2) for t in (q, k, v))
    y, lse = lib.tiga_mp_attention_fwd(q, k, v, float(inp["scale"]), relation, want_lse=True, layout=layout)
    torch.cuda.synchronize()
    if layout == "nhd":
        y = y.permute(1, 0, 2)
    y, lse = to_f64(y), lse.cpu().numpy().astype(np.float64)      # [H, n, D], [H, n]
    if pts is not None:
        y, lse = y[:, pts], lse[:, pts]
    return y.transpose(1, 0, 2), lse.T                              # [npts, H, D], [npts, H]


def compare(lib, inp, relation, pts=None, what=""):
    y, lse = run(lib, inp, relation, pts)
    ref, yabs, ref_lse = oracle.attention_fwd(inp["q"], inp["k"], inp["v"], inp["scale"], inp["dtype"], relation,
                                              pts=pts)
    vmax = float(np.abs(oracle.half_to_double(inp["v"].reshape(-1)[:4096], inp["dtype"])).max()) * 8
    return check(y, lse, ref, yabs, ref_lse, inp["q"].shape[1], vmax, inp["dtype"], what)


def test_paper_example_shape(lib):
    """The appendix's runnable check: 65 tokens (a partial tile), two heads of width 64, binary16."""
    inp = synth.attention_inputs(65, 2, 64, "f16")
    compare(lib, inp, "triangular", what="n=65 H=2 D=64 f16")


CASES = [
    (1, 1, 64, "f16", "triangular"), (2, 2, 64, "bf16", "dense"), (17, 3, 128, "f16", "triangular"),
    (64, 1, 128, "bf16", "triangular"), (127, 2, 64, "f16", "dense"), (128, 2, 128, "f16", "triangular"),
    (129, 1, 64, "bf16", "triangular"), (300, 3, 128, "bf16", "dense"), (1000, 2, 64, "f16", "triangular"),
    (1000, 1, 128, "f16", "dense"), (2049, 2, 128, "f16", "triangular"), (2049, 1, 64, "bf16", "triangular"),
    (777, 4, 128, "bf16", "triangular"), (513, 2, 64, "f16", "dense"),
]


@pytest.mark.parametrize("n,H,D,dtype,relation", CASES)
def test_attention_against_oracle(lib, n, H, D, dtype, relation):
    inp = synth.attention_inputs(n, H, D, dtype, cfg=60)
    compare(lib, inp, relation, what=f"n={n} H={H} D={D} {dtype} {relation}")


@pytest.mark.parametrize("dtype", ["f16", "bf16"])
@pytest.mark.parametrize("relation", ["triangular", "dense"])
def test_large_scores(lib, dtype, relation):
    """Scores spanning about +-60: the running maximum must keep every exponent in range."""
    inp = synth.attention_inputs(600, 2, 128, dtype, cfg=61, sigma=2.5)
    compare(lib, inp, relation, what=f"large scores {dtype} {relation}")


@pytest.mark.parametrize("dtype", ["f16", "bf16"])
def test_rising_maximum_rescales(lib, dtype):
    """Scores that grow along the key axis raise every query's maximum tile after tile, so the
    accumulator is rescaled many times."""
    n, H, D = 1500, 2, 64
    rng = np.random.default_rng(3)
    q = np.ones((H, n, D), np.float32)
    k = (np.linspace(-1.5, 1.5, n, dtype=np.float32)[None, :, None] * np.ones((H, 1, D), np.float32)
         + 0.01 * rng.standard_normal((H, n, D)).astype(np.float32))
    v = rng.standard_normal((H, n, D)).astype(np.float32)
    inp = dict(q=synth.f32_to_half_bits(q, dtype), k=synth.f32_to_half_bits(k, dtype),
               v=synth.f32_to_half_bits(v, dtype), scale=np.float32(D ** -0.5), dtype=dtype)
    for rel in ("triangular", "dense"):
        compare(lib, inp, rel, what=f"rising {dtype} {rel}")


@pytest.mark.parametrize("D", [64, 128])
@pytest.mark.parametrize("dtype", ["f16", "bf16"])
def test_tile_mass_above_cap(lib, dtype, D):
    """Keys 128..255 score about 7 (log2 units) above keys 0..127: a later key tile (the kernel's
    tiles hold 64 or 128 keys) whose weights all stay inside the 16-bit range, but whose mass
    (at least 64 * 2^7) exceeds the fast path's cap, so the reference point must still move
    before the value product."""
    n, H = 300, 2
    rng = np.random.default_rng(12 + D)
    q = np.ones((H, n, D), np.float32)
    unit = np.float32(np.log(2.0) / np.sqrt(D))      # scale * <q, k> = ln 2 per unit of lift
    lift = np.zeros(n, np.float32)
    lift[128:256] = 7.0 * unit
    lift[256:] = 3.5 * unit
    k = lift[None, :, None] + 0.02 * rng.standard_normal((H, n, D)).astype(np.float32) / np.sqrt(D)
    v = rng.standard_normal((H, n, D)).astype(np.float32)
    inp = dict(q=synth.f32_to_half_bits(q, dtype), k=synth.f32_to_half_bits(k, dtype),
               v=synth.f32_to_half_bits(v, dtype), scale=np.float32(D ** -0.5), dtype=dtype)
    for rel in ("triangular", "dense"):
        compare(lib, inp, rel, what=f"tile mass {dtype} D={D} {rel}")


def test_paper_layout_view(lib):
    """The logical (n, heads, width) view of head-major storage gives the same bits as [heads, n, width]."""
    inp = synth.attention_inputs(333, 3, 64, "f16", cfg=62)
    y1, l1 = run(lib, inp, "triangular")
    y2, l2 = run(lib, inp, "triangular", layout="nhd")
    assert np.array_equal(y1, y2) and np.array_equal(l1, l2)


def test_repeated_calls_are_bit_identical(lib):
    inp = synth.attention_inputs(1111, 2, 128, "bf16", cfg=63)
    y1, l1 = run(lib, inp, "dense")
    y2, l2 = run(lib, inp, "dense")
    assert np.array_equal(y1, y2) and np.array_equal(l1, l2)


def test_constant_values(lib):
    """Every weight is positive and they are normalized: constant values come back exactly
    (the constant is a 16-bit value; the weights sum, divided by their own total, to 1)."""
    n, H, D = 700, 2, 128
    inp = synth.attention_inputs(n, H, D, "f16", cfg=64)
    inp["v"] = synth.f32_to_half_bits(np.full((H, n, D), 0.75, np.float32), "f16")
    y, _ = run(lib, inp, "triangular")
    assert np.abs(y - 0.75).max() <= 2 * U["f16"] * 0.75


def test_empty_and_unsupported(lib):
    z = torch.empty(2, 0, 64, dtype=torch.float16, device="cuda")
    y = lib.tiga_mp_attention_fwd(z, z, z)
    assert y.shape == (2, 0, 64)
    bad = torch.zeros(1, 8, 96, dtype=torch.float16, device="cuda")
    with pytest.raises(lib.TigaError) as e:
        lib.tiga_mp_attention_fwd(bad, bad, bad)
    assert e.value.code == lib.TIGA_EUNSUPPORTED


def test_full_size_sampled(lib):
    """The measured workload (16 heads, 16384 tokens, width 128, binary16, triangular), checked on
    sampled query rows: the first and last rows, rows at tile boundaries and random rows, all heads."""
    n, H, D = 16384, 16, 128
    inp = synth.attention_inputs(n, H, D, "f16", cfg=6)
    rng = np.random.default_rng(11)
    pts = np.unique(np.concatenate([[0, 1, 63, 64, 127, 128, 129, n - 129, n - 128, n - 2, n - 1],
                                    rng.integers(0, n, 21)]))
    compare(lib, inp, "triangular", pts=pts, what="16k x 16 heads x 128 sampled")
