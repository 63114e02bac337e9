"""GPU parity of the kinds with the random-orthogonal Kronecker pre-conditioner
(QKH: eq. straight on the flattened layer; AFJLQ: eq. frikadel with H_N -> Q;
AFFDQ: eq. bami with both H_N -> Q)
through the C ABI, against the fp64 oracle.  Same error metric and fp32
tolerance as the other kinds: per batch row max_i |y_i - o_i| / max(|o_i|, rms(o)).

The cases cover every contraction order of the library: layers with fewer live
rows than D / 1024 (Qt first), one slab (P = 1), two and four slabs (fold
inside the contraction), sixteen slabs (separate fold), D = 2048 (two kept rows
of factor K - 2), D = 2^16 and 2^20, ragged tails, bf16 inputs and outputs,
theta0, streaming with accumulate, and the full-size GPT-2-small layer set on
sampled batch rows."""
import numpy as np
import pytest
import torch

import oracle as O

pytestmark = pytest.mark.gpu

TOL = 1e-5


@pytest.fixture(scope="module")
def dev():
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    from paper_2402_03994_amd import _lib
    _lib.load()
    return torch.device("cuda", 0)


def rel_err(y, o):
    y = np.asarray(y, dtype=np.float64).reshape(len(y), -1)
    o = np.asarray(o, dtype=np.float64).reshape(len(o), -1)
    rms = np.sqrt((o ** 2).mean(axis=1, keepdims=True))
    den = np.maximum(np.abs(o), rms)
    den[den == 0] = 1.0
    return float((np.abs(y - o) / den).max())


def inputs(shapes, batch, seed, dtype=torch.float32):
    g = torch.Generator().manual_seed(seed)
    xs = [torch.randn((batch, r * c), generator=g) for r, c in shapes]
    return [x.to(dtype) for x in xs]


def as_oracle(x):
    if x.dtype == torch.bfloat16:
        return x.view(torch.int16).numpy().view(np.uint16), "bf16"
    return x.numpy(), "f32"


def sketch(kind, shapes, D, seed, dev):
    from paper_2402_03994_amd import Sketch
    return Sketch(kind, shapes, D, seed, device=dev)


CASES = [
    # D = 4096 (D_m = 4): Qt-first layers (1 and 3 live rows), P = 1 with 4 rows, P = 2, P = 4
    ([(1, 768), (3, 1000), (64, 64), (1, 2 ** 21 - 5), (1, 3 * 2 ** 20 + 7)], 4096),
    # sixteen slabs (separate fold) and a tiny layer
    ([(1, 2 ** 23 + 3), (1, 5)], 4096),
    # D = 2048: two kept rows, ragged K in the transposed contraction
    ([(7, 300), (1, 2 ** 20 + 1), (1, 2048)], 2048),
    # D = 2^16 (D_m = 64): GPT-2-like mix
    ([(1, 768), (768, 2304), (1, 2304), (768, 768)], 65536),
]


@pytest.mark.parametrize("kind", ["qkh", "afjlq"])
@pytest.mark.parametrize("case", range(len(CASES)))
def test_forward_parity(kind, case, dev):
    shapes, D = CASES[case]
    seed = 300 + case
    xs = inputs(shapes, 3, seed)
    s = sketch(kind, shapes, D, seed, dev)
    y = s.apply([x.to(dev) for x in xs]).cpu().numpy()
    ref = O.apply(kind, shapes, D, seed, [x.numpy() for x in xs])
    assert rel_err(y, ref) < TOL


@pytest.mark.parametrize("kind", ["qkh", "afjlq"])
@pytest.mark.parametrize("case", range(len(CASES)))
def test_transpose_parity(kind, case, dev):
    shapes, D = CASES[case]
    seed = 400 + case
    g = torch.Generator().manual_seed(seed)
    z = torch.randn((2, D), generator=g)
    th = [None if i == 0 else torch.randn(r * c, generator=g) * 0.02 for i, (r, c) in enumerate(shapes)]
    s = sketch(kind, shapes, D, seed, dev)
    outs = s.apply_T(z.to(dev), theta0=[None if t is None else t.to(dev) for t in th])
    refs = O.apply_T(kind, shapes, D, seed, z.numpy().astype(np.float64),
                     theta0=[None if t is None else t.numpy() for t in th])
    for o, r in zip(outs, refs):
        assert rel_err(o.cpu().numpy(), r) < TOL


@pytest.mark.parametrize("kind", ["qkh", "afjlq"])
def test_bf16_input_and_output(kind, dev):
    shapes, D = CASES[0]
    xs = inputs(shapes, 2, 7, torch.bfloat16)
    s = sketch(kind, shapes, D, 7, dev)
    y = s.apply([x.to(dev) for x in xs]).cpu().numpy()
    ins = [as_oracle(x) for x in xs]
    ref = O.apply(kind, shapes, D, 7, [a for a, _ in ins], dtype="bf16")
    assert rel_err(y, ref) < TOL  # bf16 values are exact in fp32
    z = torch.randn((2, D), generator=torch.Generator().manual_seed(8))
    outs = s.apply_T(z.to(dev), out_dtype=torch.bfloat16)
    refs = O.apply_T(kind, shapes, D, 7, z.numpy().astype(np.float64))
    for o, r in zip(outs, refs):
        assert rel_err(o.float().cpu().numpy(), r) < 2 ** -8  # one bf16 rounding of the output


@pytest.mark.parametrize("kind", ["qkh", "afjlq"])
def test_streaming_accumulate_and_determinism(kind, dev):
    shapes, D = CASES[2]
    xs = [x.to(dev) for x in inputs(shapes, 4, 12)]
    s = sketch(kind, shapes, D, 13, dev)
    y1 = s.apply(xs)
    assert torch.equal(y1, s.apply(xs))
    out = torch.zeros_like(y1)
    for l, x in enumerate(xs):
        s.apply([x], out=out, first_layer=l, accumulate=True)
    ref = O.apply(kind, shapes, D, 13, [x.cpu().numpy() for x in xs])
    assert rel_err(out.cpu().numpy(), ref) < TOL


def test_d_2_20(dev):
    """D = 2^20: factor K - 2 kept whole (D_m = 1024)."""
    shapes, D = [(1, 2 ** 20 - 3), (1, 1000)], 2 ** 20
    xs = inputs(shapes, 2, 21)
    s = sketch("afjlq", shapes, D, 21, dev)
    y = s.apply([x.to(dev) for x in xs]).cpu().numpy()
    ref = O.apply("afjlq", shapes, D, 21, [x.numpy() for x in xs])
    assert rel_err(y, ref) < TOL


def test_gpt2_small_full_size_sampled_rows(dev):
    """All 148 GPT-2-small tensors at D = 2^16 and batch 8 on the GPU; rows 0 and 7 against the oracle."""
    import workloads as W
    shapes = W.CONFIGS["c2"]["shapes"]
    D, seed, batch = 65536, 1, 8
    g = torch.Generator(device=dev).manual_seed(5)
    xs = [torch.randn((batch, r * c), generator=g, device=dev) * 1e-2 for r, c in shapes]
    s = sketch("afjlq", shapes, D, seed, dev)
    y = s.apply(xs).cpu().numpy()
    rows = [0, batch - 1]
    ref = O.apply("afjlq", shapes, D, seed, [x[rows].cpu().numpy() for x in xs])
    assert rel_err(y[rows], ref) < TOL


# AFFDQ: dense per slab, so smaller cases (live slabs 1 .. 2, Qt-first-sized small layers, D = 2048 .. 2^16)
AFFDQ_CASES = [
    ([(1, 768), (3, 1000), (64, 64), (1, 2 ** 21 - 5)], 4096),
    ([(7, 300), (1, 2 ** 20 + 1)], 2048),
    ([(1, 768), (768, 768)], 65536),
]


@pytest.mark.parametrize("case", range(len(AFFDQ_CASES)))
def test_affdq_forward_parity(case, dev):
    shapes, D = AFFDQ_CASES[case]
    seed = 500 + case
    xs = inputs(shapes, 2, seed)
    s = sketch("affdq", shapes, D, seed, dev)
    y = s.apply([x.to(dev) for x in xs]).cpu().numpy()
    ref = O.apply("affdq", shapes, D, seed, [x.numpy() for x in xs])
    assert rel_err(y, ref) < TOL


@pytest.mark.parametrize("case", range(len(AFFDQ_CASES)))
def test_affdq_transpose_parity(case, dev):
    shapes, D = AFFDQ_CASES[case]
    seed = 600 + case
    g = torch.Generator().manual_seed(seed)
    z = torch.randn((2, D), generator=g)
    th = [None if i == 0 else torch.randn(r * c, generator=g) * 0.02 for i, (r, c) in enumerate(shapes)]
    s = sketch("affdq", shapes, D, seed, dev)
    outs = s.apply_T(z.to(dev), theta0=[None if t is None else t.to(dev) for t in th])
    refs = O.apply_T("affdq", shapes, D, seed, z.numpy().astype(np.float64),
                     theta0=[None if t is None else t.numpy() for t in th])
    for o, r in zip(outs, refs):
        assert rel_err(o.cpu().numpy(), r) < TOL


def test_affdq_bf16_streaming(dev):
    shapes, D = AFFDQ_CASES[1]
    xs = [x.to(dev) for x in inputs(shapes, 2, 31, torch.bfloat16)]
    s = sketch("affdq", shapes, D, 32, dev)
    y1 = s.apply(xs)
    assert torch.equal(y1, s.apply(xs))
    out = torch.zeros_like(y1)
    for l, x in enumerate(xs):
        s.apply([x], out=out, first_layer=l, accumulate=True)
    ins = [as_oracle(x.cpu()) for x in xs]
    ref = O.apply("affdq", shapes, D, 32, [a for a, _ in ins], dtype="bf16")
    assert rel_err(out.cpu().numpy(), ref) < TOL
