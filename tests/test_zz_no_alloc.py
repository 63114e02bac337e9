"""The allocation-free forward entry point (sketch_apply_noalloc, scratch in the library's static device array)
against sketch_apply on the same handle: two calls in a row, the second with a smaller batch, for every kind whose
per-vector scratch fits, plus a batch that goes through the static scratch in several chunks, and the rejection of
a layer range that does not fit."""
import numpy as np
import pytest
import torch

import oracle as O

pytestmark = pytest.mark.gpu

TOL_F32 = 1e-5


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


def inputs(shapes, batch, seed):
    g = torch.Generator().manual_seed(seed)
    return [torch.randn((batch, s[0] * s[1]), generator=g) for s in shapes]


LAYERS = [(1, 30), (7, 111), (3, 1500), (1, 5003), (33, 1024), (1, 16)]
CASES = [("afjl", LAYERS, 1024), ("afjl", [(768, 3072), (1, 768), (50, 1024)], 1 << 16),
         ("fjl", [(1, 1 << 20)], 4096), ("ffd", LAYERS, 256), ("affd", LAYERS, 4096),
         ("affd", [(96, 1024), (1, 3072), (2, 3000)], 1 << 16),
         ("qk", [(40, 70, 4, 5), (64, 33, 8, 2), (256, 512, 32, 16)], 20 + 16 + 512)]


@pytest.mark.parametrize("case", range(len(CASES)))
def test_noalloc_matches_apply_two_calls(case, dev):
    from paper_2402_03994_amd import Sketch
    kind, shapes, D = CASES[case]
    seed = 500 + case
    s = Sketch(kind, shapes, D, seed, device=dev)
    for batch in (6, 2):  # the second call with a smaller input
        xs = inputs(shapes, batch, seed + batch)
        xd = [x.to(dev) for x in xs]
        ref = s.apply(xd).cpu().numpy()
        out = torch.full((batch, D), float("nan"), device=dev)
        s.apply(xd, out=out, noalloc=True)
        y = out.cpu().numpy()
        assert rel_err(y, ref) <= TOL_F32
        assert rel_err(y, O.apply(kind, shapes, D, seed, [x.numpy() for x in xs])) <= TOL_F32
    s.close()


def test_noalloc_chunks_and_accumulate(dev):
    """FJL with N' = 2^22 (16 MiB of scratch per vector): a batch of 9 goes through the 64 MiB static scratch in
    chunks; then a streamed call with accumulate over a layer range."""
    from paper_2402_03994_amd import Sketch
    shapes, D, seed = [(1, (1 << 22) - 5), (3, 700)], 8192, 77
    s = Sketch("fjl", shapes, D, seed, device=dev)
    xs = inputs(shapes, 9, seed)
    xd = [x.to(dev) for x in xs]
    ref = s.apply(xd).cpu().numpy()
    out = torch.zeros((9, D), device=dev)
    s.apply(xd[:1], out=out, first_layer=0, noalloc=True)
    s.apply(xd[1:], out=out, first_layer=1, accumulate=True, noalloc=True)
    y = out.cpu().numpy()
    assert rel_err(y, ref) <= TOL_F32
    assert rel_err(y, O.apply("fjl", shapes, D, seed, [x.numpy() for x in xs])) <= TOL_F32
    s.close()


def test_noalloc_rejects_layers_beyond_the_scratch(dev):
    from paper_2402_03994_amd import Sketch
    from paper_2402_03994_amd._lib import SketchError
    s = Sketch("fjl", [(1, (1 << 24) + 1)], 4096, 3, device=dev)
    x = torch.zeros((1, (1 << 24) + 1), device=dev)
    out = torch.full((1, 4096), 7.0, device=dev)
    with pytest.raises(SketchError) as e:
        s.apply([x], out=out, noalloc=True)
    assert e.value.code == -5 and "static scratch" in str(e.value)
    assert torch.all(out == 7.0)
    s.close()
