"""GPU parity of the Fourier pre-conditioner kind AFJLF (eq. frikadel with H_N replaced by the FFT, Sec. 3
"Alternative pre-conditioners") against the fp64 oracle (oracle/fourier.py), through the C ABI.

Cases cover the one-kernel path (layers with N' = D and at most 16384 entries), the two-pass path over the whole
range of Q = N'/(D/2) (2 .. 2048, rows of R = N'/256 once Q exceeds 256) and of the outputs per residue (4 .. 16384),
several layers per launch, ragged rows, bf16 inputs and outputs, theta0, streaming with accumulate and bitwise
determinism.  Same metric and bounds as the
other kinds: max_i |y_i - o_i| / max(|o_i|, rms(o)) <= 1e-5.
"""
import numpy as np
import pytest
import torch

import oracle as O

pytestmark = pytest.mark.gpu

TOL_F32 = 1e-5
TOL_BF16 = 2e-2


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


def inputs(shapes, batch, seed, dtype=torch.float32, scale=1.0):
    g = torch.Generator().manual_seed(seed)
    xs = [torch.randn((batch, r * c), generator=g) * scale for r, c in shapes]
    return [x.to(dtype) for x in xs]


def host(x):
    if x.dtype == torch.bfloat16:
        return x.view(torch.int16).numpy().view(np.uint16), "bf16"
    return x.numpy(), "f32"


LAYERS = [(1, 30), (7, 111), (3, 1500), (1, 5003), (33, 1024), (1, 16)]
CASES = [
    (LAYERS, 2048),                                   # small path, P = 8 and 64 (J = 128, 16)
    (LAYERS, 4096),
    ([(1, 70000), (3, 500)], 4096),                   # P = 64, J = 32
    ([(1, 1 << 20)], 2048),                           # N'/M = 1024: rows of R = 4M (P = 256), J = 4
    ([(1, 3 * 2 ** 20 + 5), (2, 999)], 4096),         # N'/M = 2048: P = 256, R = 2^14, J = 8, two q-blocks
    ([(1, 3 * 2 ** 20 + 11)], 1 << 16),               # P = 128, J = 256, two q-blocks
    ([(1, 768), (1, 2304), (96, 1024), (1, 3072), (2, 3000), (1, 8200), (1, 20000)], 1 << 16),  # P = 2 .. 4
    ([(1, 2 ** 22 - 9), (5, 999)], 1 << 17),          # P = 64, J = 1024
    ([(1, 2 ** 25 + 5), (2, 4097)], 1 << 20),         # P = 128, J = 4096; small path with 64 c-groups
]


@pytest.mark.parametrize("case", range(len(CASES)))
def test_afjlf_forward(case, dev):
    from paper_2402_03994_amd import Sketch
    shapes, D = CASES[case]
    seed = 600 + case
    xs = inputs(shapes, 3, seed)
    s = Sketch("afjlf", shapes, D, seed, device=dev)
    y = s.apply([x.to(dev) for x in xs]).cpu().numpy()
    ref = O.apply("afjlf", shapes, D, seed, [x.numpy() for x in xs])
    assert rel_err(y, ref) < TOL_F32
    s.close()


@pytest.mark.parametrize("case", range(len(CASES)))
def test_afjlf_transpose(case, dev):
    from paper_2402_03994_amd import Sketch
    shapes, D = CASES[case]
    seed = 700 + case
    g = torch.Generator().manual_seed(seed)
    z = torch.randn((2, D), generator=g)
    th = [torch.randn(r * c, generator=g) * 0.02 if i % 2 else None for i, (r, c) in enumerate(shapes)]
    s = Sketch("afjlf", shapes, D, seed, device=dev)
    outs = s.apply_T(z.to(dev), theta0=[None if t is None else t.to(dev) for t in th])
    refs = O.apply_T("afjlf", shapes, D, seed, z.numpy().astype(np.float64),
                     theta0=[None if t is None else t.numpy() for t in th])
    for o, r in zip(outs, refs):
        assert rel_err(o.cpu().numpy(), r) < TOL_F32
    s.close()


def test_afjlf_bf16_inputs_and_outputs(dev):
    from paper_2402_03994_amd import Sketch
    shapes, D = CASES[5]
    seed = 801
    xs = inputs(shapes, 2, seed, dtype=torch.bfloat16, scale=0.01)
    s = Sketch("afjlf", shapes, D, seed, device=dev)
    y = s.apply([x.to(dev) for x in xs]).cpu().numpy()
    ref = O.apply("afjlf", shapes, D, seed, [host(x)[0] for x in xs], dtype="bf16")
    assert rel_err(y, ref) < TOL_F32  # bf16 inputs are widened exactly
    z = torch.randn((2, D), generator=torch.Generator().manual_seed(seed))
    outs = s.apply_T(z.to(dev), out_dtype=torch.bfloat16)
    refs = O.apply_T("afjlf", shapes, D, seed, z.numpy().astype(np.float64))
    for o, r in zip(outs, refs):
        assert rel_err(o.float().cpu().numpy(), r) < TOL_BF16
    s.close()


def test_afjlf_streaming_accumulate_and_determinism(dev):
    from paper_2402_03994_amd import Sketch
    shapes, D = CASES[0]
    xs = [x.to(dev) for x in inputs(shapes, 4, 9)]
    s = Sketch("afjlf", shapes, D, 11, device=dev)
    y1 = s.apply(xs)
    y2 = s.apply(xs)
    assert torch.equal(y1, y2)
    out = torch.zeros_like(y1)
    for l, x in enumerate(xs):
        s.apply([x], out=out, first_layer=l, accumulate=True)
    ref = O.apply("afjlf", shapes, D, 11, [x.cpu().numpy() for x in xs])
    assert rel_err(out.cpu().numpy(), ref) < TOL_F32
    s.close()


def test_afjlf_small_workspace_tiles(dev, monkeypatch):
    """A 16 MB workspace: the 2^22-entry layer's pass buffer holds one vector at a time (vector tiles), the
    other layers go through in separate groups; same result as the default workspace."""
    from paper_2402_03994_amd import Sketch
    shapes, D = [(1, 3 * 2 ** 20 + 11), (33, 1024), (1, 300)], 1 << 16
    seed = 803
    xs = inputs(shapes, 3, seed)
    ref = O.apply("afjlf", shapes, D, seed, [x.numpy() for x in xs])
    big = Sketch("afjlf", shapes, D, seed, device=dev)
    yb = big.apply([x.to(dev) for x in xs]).cpu().numpy()
    big.close()
    monkeypatch.setenv("SK_WORKSPACE_MB", "40")
    small = Sketch("afjlf", shapes, D, seed, device=dev)
    ys = small.apply([x.to(dev) for x in xs]).cpu().numpy()
    small.close()
    assert rel_err(yb, ref) < TOL_F32
    assert rel_err(ys, ref) < TOL_F32
