"""GPU parity: the HIP library (through its C ABI) against the fp64 oracle.

Error metric per batch row: max_i |y_i - o_i| / max(|o_i|, rms(o)), bounded by
1e-5 for fp32 inputs and 2e-2 for bf16 inputs (fp32 arithmetic on the GPU);
random signs, sample positions and permutations must match bit for bit.
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
    _lib.load()  # fail loudly if the HIP library is missing
    return torch.device("cuda", 0)


def sk(kind, shapes, D, seed, dev):
    from paper_2402_03994_amd import Sketch
    return Sketch(kind, shapes, D, seed, device=dev)


def rel_err(y, o):
    y = np.asarray(y, dtype=np.float64)
    o = np.asarray(o, dtype=np.float64)
    o2 = o.reshape(o.shape[0], -1)
    y2 = y.reshape(y.shape[0], -1)
    rms = np.sqrt((o2**2).mean(axis=1, keepdims=True))
    den = np.maximum(np.abs(o2), rms)
    den[den == 0] = 1.0
    return float((np.abs(y2 - o2) / den).max())


def rand_inputs(shapes, batch, seed, dtype=torch.float32, scale=1.0):
    g = torch.Generator().manual_seed(seed)
    xs = [torch.randn((batch, s[0] * s[1]), generator=g, dtype=torch.float32) * scale for s in shapes]
    if dtype == torch.bfloat16:
        xs = [x.to(torch.bfloat16) for x in xs]
    return xs


def oracle_in(x):
    if x.dtype == torch.bfloat16:
        return x.view(torch.int16).numpy().view(np.uint16), "bf16"
    return x.numpy(), "f32"


# shapes spanning several tiles, ragged tails, n < D and n not a multiple of 4
LAYERS = [(1, 30), (7, 111), (3, 1500), (1, 5003), (33, 1024), (1, 16)]
CASES = [(LAYERS, 16), (LAYERS, 256), (LAYERS, 1024), (LAYERS, 4096), ([(1, 70000), (3, 500)], 65536),
         ([(1, 2 ** 20 + 3), (1, 9)], 2048), ([(1, 3 * 2 ** 20 + 11)], 65536),
         # transformer-like mix: small layers grouped (N' = D, <= 8 rows), a
         # two-digit layer with 128 rows and one with 9 source rows
         ([(1, 768), (1, 2304), (96, 1024), (1, 3072), (2, 3000), (1, 8200)], 65536)]


@pytest.mark.parametrize("kind", ["afjl", "affd", "fjl", "ffd"])
@pytest.mark.parametrize("case", range(len(CASES)))
def test_forward_parity_f32(kind, case, dev):
    shapes, D = CASES[case]
    seed = 100 + case
    xs = rand_inputs(shapes, 3, seed)
    s = sk(kind, shapes, D, seed, dev)
    y = s.apply([x.to(dev) for x in xs]).cpu().numpy()
    ref = O.apply(kind, shapes, D, seed, [x.numpy() for x in xs])
    assert rel_err(y, ref) < TOL_F32


@pytest.mark.parametrize("mtab", [True, False])
@pytest.mark.parametrize("shapes", [[(3, 2 ** 20 + 77), (1, 5000)], [(1, 9 * 2 ** 20 + 5)], [(37, 2 ** 20)]])
def test_affd_mtab_parity(shapes, mtab, dev):
    """AFFD layers on the transposed path (one to sixteen top slabs), with the
    stored M tables and with the Gaussians regenerated per call."""
    from paper_2402_03994_amd import Sketch
    D, seed, batch = 65536, 21, 5
    s = Sketch("affd", shapes, D, seed, device=dev, flags=0 if mtab else Sketch.AFFD_NO_MTAB)
    xs = rand_inputs(shapes, batch, 99)
    y = s.apply([x.to(dev) for x in xs])
    o = O.apply("affd", shapes, D, seed, [oracle_in(x)[0] for x in xs])
    assert rel_err(y.cpu().numpy(), o) <= TOL_F32
    s.close()


def test_affd_slab_groups_small_workspace(dev, monkeypatch):
    """A ten-slab transposed-path layer under an 80 MB workspace: the live
    slabs go through the row and top kernels one group at a time with F
    carried between the groups; the result matches the oracle and the default
    single-group schedule."""
    from paper_2402_03994_amd import Sketch
    shapes = [(1, 9 * 2 ** 20 + 5), (1, 3000)]
    D, seed, batch = 65536, 29, 11
    xs = rand_inputs(shapes, batch, 97)
    o = O.apply("affd", shapes, D, seed, [oracle_in(x)[0] for x in xs])
    big = Sketch("affd", shapes, D, seed, device=dev)
    y_big = big.apply([x.to(dev) for x in xs]).cpu().numpy()
    big.close()
    monkeypatch.setenv("SK_WORKSPACE_MB", "80")
    small = Sketch("affd", shapes, D, seed, device=dev)
    y_small = small.apply([x.to(dev) for x in xs]).cpu().numpy()
    small.close()
    assert rel_err(y_small, o) <= TOL_F32
    assert rel_err(y_big, o) <= TOL_F32
    assert rel_err(y_small, y_big.astype(np.float64)) <= TOL_F32


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_affd_transposed_vector_loads(dtype, dev):
    """Transposed-path AFFD layers whose length is a multiple of 4 (16- or
    8-byte row loads) with a partial last source row, in fp32 and bf16.  The
    oracle reads the same bf16 values exactly and the kernels compute in fp32,
    so both dtypes are held to the fp32 bound."""
    from paper_2402_03994_amd import Sketch
    shapes = [(1, 2 ** 21 + 1000), (5, 2 ** 18 + 4)]
    D, seed, batch = 65536, 23, 4
    s = Sketch("affd", shapes, D, seed, device=dev)
    xs = rand_inputs(shapes, batch, 98, dtype=dtype)
    y = s.apply([x.to(dev) for x in xs])
    o = O.apply("affd", shapes, D, seed, [oracle_in(x)[0] for x in xs], dtype=oracle_in(xs[0])[1])
    assert rel_err(y.cpu().numpy(), o) <= TOL_F32
    s.close()


@pytest.mark.parametrize("kind", ["afjl", "affd", "fjl", "ffd"])
@pytest.mark.parametrize("case", [1, 3, 4])
def test_transpose_parity(kind, case, dev):
    shapes, D = CASES[case]
    seed = 200 + case
    g = torch.Generator().manual_seed(seed)
    z = torch.randn((2, D), generator=g)
    th = [torch.randn(s[0] * s[1], generator=g) * 0.02 for s in shapes]
    th[0] = None
    s = sk(kind, shapes, D, seed, dev)
    outs = s.apply_T(z.to(dev), theta0=[None if t is None else t.to(dev) for t in th])
    refs = O.apply_T(kind, shapes, D, seed, z.numpy().astype(np.float64),
                     theta0=[None if t is None else t.numpy() for t in th])
    for o, r in zip(outs, refs):
        assert rel_err(o.cpu().numpy(), r) < TOL_F32


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_ffd_large_D(dtype, dev):
    """FFD with D = 2^20 (rows/cols kernels over transposed intermediates):
    forward over three blocks with a ragged tail and a one-block layer, and
    theta0 + S^T z with fp32 and bf16 outputs."""
    shapes, D, seed = [(1, 2 ** 21 + 5), (3, 1000)], 2 ** 20, 41
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    xs = rand_inputs(shapes, 3, seed, dtype=tdt)
    s = sk("ffd", shapes, D, seed, dev)
    y = s.apply([x.to(dev) for x in xs]).cpu().numpy()
    ref = O.apply("ffd", shapes, D, seed, [oracle_in(x)[0] for x in xs], dtype=dtype)
    assert rel_err(y, ref) < TOL_F32
    g = torch.Generator().manual_seed(seed)
    z = torch.randn((2, D), generator=g)
    th = [torch.randn(sh[0] * sh[1], generator=g) * 0.02 for sh in shapes]
    outs = s.apply_T(z.to(dev), out_dtype=tdt, theta0=[t.to(dev) for t in th])
    refs = O.apply_T("ffd", shapes, D, seed, z.numpy().astype(np.float64), theta0=[t.numpy() for t in th])
    for o, r in zip(outs, refs):
        assert rel_err(o.float().cpu().numpy(), r) < (TOL_BF16 if dtype == "bf16" else TOL_F32)


@pytest.mark.parametrize("batch,dtype", [(4, "f32"), (8, "bf16")])
def test_ffd_large_D_groups(batch, dtype, dev):
    """FFD with D = 2^20 on a batch that is a multiple of four: the four-vector
    groups with interleaved intermediates.  Forward over three blocks with a
    ragged tail plus a one-block layer (accumulated into the same output), and
    theta0 + S^T z with fp32 or bf16 outputs."""
    shapes, D, seed = [(1, 2 ** 21 + 5), (3, 1000)], 2 ** 20, 43
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    xs = rand_inputs(shapes, batch, seed, dtype=tdt)
    s = sk("ffd", shapes, D, seed, dev)
    y = s.apply([x.to(dev) for x in xs]).cpu().numpy()
    ref = O.apply("ffd", shapes, D, seed, [oracle_in(x)[0] for x in xs], dtype=dtype)
    assert rel_err(y, ref) < TOL_F32
    g = torch.Generator().manual_seed(seed)
    z = torch.randn((batch, D), generator=g)
    th = [torch.randn(sh[0] * sh[1], generator=g) * 0.02 for sh in shapes]
    if batch == 8:
        th[1] = None  # a layer without theta0
    outs = s.apply_T(z.to(dev), out_dtype=tdt, theta0=[None if t is None else t.to(dev) for t in th])
    refs = O.apply_T("ffd", shapes, D, seed, z.numpy().astype(np.float64),
                     theta0=[None if t is None else t.numpy() for t in th])
    for o, r in zip(outs, refs):
        assert rel_err(o.float().cpu().numpy(), r) < (TOL_BF16 if dtype == "bf16" else TOL_F32)


@pytest.mark.parametrize("shapes", [[(1, 2 ** 21 + 5), (3, 1000)], [(1, 8 * 2 ** 20 - 5)]])
def test_ffd_large_D_groups_gather(shapes, dev, monkeypatch):
    """The four-vector groups without the bucket tables (SK_FFD_BUCKET_MB=0):
    the permutation gathers one 16-byte word per coordinate; forward and
    transpose against the oracle, and equal to the bucketed path bit for bit
    (both place the same values, the sums run in the same order).  Eight
    blocks (one group) take the XCD-grouped workgroup order."""
    D, seed = 2 ** 20, 47
    xs = rand_inputs(shapes, 4, seed)
    g = torch.Generator().manual_seed(seed)
    z = torch.randn((4, D), generator=g)
    th = [torch.randn(sh[0] * sh[1], generator=g) * 0.02 for sh in shapes]
    s_b = sk("ffd", shapes, D, seed, dev)
    yb = s_b.apply([x.to(dev) for x in xs]).cpu().numpy()
    ob = [o.cpu().numpy() for o in s_b.apply_T(z.to(dev), theta0=[t.to(dev) for t in th])]
    monkeypatch.setenv("SK_FFD_BUCKET_MB", "0")
    s_g = sk("ffd", shapes, D, seed, dev)
    y = s_g.apply([x.to(dev) for x in xs]).cpu().numpy()
    ref = O.apply("ffd", shapes, D, seed, [x.numpy() for x in xs])
    assert rel_err(y, ref) < TOL_F32
    assert np.array_equal(y, yb)
    outs = [o.cpu().numpy() for o in s_g.apply_T(z.to(dev), theta0=[t.to(dev) for t in th])]
    refs = O.apply_T("ffd", shapes, D, seed, z.numpy().astype(np.float64), theta0=[t.numpy() for t in th])
    for o, r, o2 in zip(outs, refs, ob):
        assert rel_err(o, r) < TOL_F32
        assert np.array_equal(o, o2)


@pytest.mark.parametrize("kind", ["afjl", "affd", "fjl", "ffd"])
def test_forward_parity_bf16(kind, dev):
    shapes, D = CASES[3]
    seed = 300
    xs = rand_inputs(shapes, 2, seed, dtype=torch.bfloat16, scale=0.01)
    s = sk(kind, shapes, D, seed, dev)
    y = s.apply([x.to(dev) for x in xs]).cpu().numpy()
    ins = [oracle_in(x)[0] for x in xs]
    ref = O.apply(kind, shapes, D, seed, ins, dtype="bf16")
    # bf16 inputs are widened exactly, so the fp32 bound holds too
    assert rel_err(y, ref) < TOL_F32


@pytest.mark.parametrize("kind", ["afjl", "affd", "fjl", "ffd"])
def test_transpose_bf16_output(kind, dev):
    shapes, D = CASES[1]
    g = torch.Generator().manual_seed(5)
    z = torch.randn((2, D), generator=g)
    s = sk(kind, shapes, D, 5, dev)
    outs = s.apply_T(z.to(dev), out_dtype=torch.bfloat16)
    refs = O.apply_T(kind, shapes, D, 5, z.numpy().astype(np.float64))
    for o, r in zip(outs, refs):
        assert rel_err(o.float().cpu().numpy(), r) < TOL_BF16


@pytest.mark.parametrize("kind", ["afjl", "affd", "fjl", "ffd", "qk"])
def test_streaming_accumulate_and_determinism(kind, dev):
    if kind == "qk":
        shapes, D = [(40, 70, 4, 5), (64, 33, 8, 2), (1, 300, 1, 9)], 20 + 16 + 9
    else:
        shapes, D = LAYERS, 1024
    xs = [x.to(dev) for x in rand_inputs(shapes, 4, 9)]
    s = sk(kind, shapes, D, 11, dev)
    y1 = s.apply(xs)
    y2 = s.apply(xs)
    assert torch.equal(y1, y2)  # bitwise deterministic
    out = torch.zeros_like(y1)
    for l, x in enumerate(xs):
        s.apply([x], out=out, first_layer=l, accumulate=True)
    ref = O.apply(kind, shapes, D, 11, [x.cpu().numpy() for x in xs])
    assert rel_err(out.cpu().numpy(), ref) < TOL_F32


def test_debug_streams_bit_exact(dev):
    seed = 0xDEADBEEF12345
    shapes = [(1, 3000), (1, 70000)]
    for kind in ["afjl", "affd", "fjl"]:
        s = sk(kind, shapes, 1024, seed, dev)
        for layer, (r, c) in enumerate(shapes):
            np_len = O.padded(r * c, 1024)
            cnt = min(20000, np_len - 5)
            assert np.array_equal(s.debug_stream(layer, "sign", 5, cnt), O.signs(seed, layer, 5, cnt))
            g = s.debug_stream(layer, "gauss", 0, 8192).astype(np.float64)
            go = O.gauss(seed, layer, "gauss", 0, 8192)
            assert np.abs(g - go).max() < 1e-5
            if kind == "fjl":
                assert np.array_equal(s.debug_stream(layer, "index", 0, 1024), O.indices(seed, layer, 0, 1024, np_len))
            else:
                assert np.array_equal(s.debug_stream(layer, "pi1", 0, np_len), O.digit_perm(seed, layer, "pi1", np_len))
            if kind == "affd":
                assert np.array_equal(s.debug_stream(layer, "pi2", 0, np_len), O.digit_perm(seed, layer, "pi2", np_len))
    s = sk("ffd", [(1, 5000)], 4096, seed, dev)
    for b in [0, 1]:
        assert np.array_equal(s.debug_stream(0, "ffdperm", 0, 4096, aux=b), O.perm(seed, 0, "ffdperm", b, 12))
    s = sk("ffd", [(1, 5000)], 1 << 20, seed, dev)
    assert np.array_equal(s.debug_stream(0, "ffdperm", 0, 1 << 20, aux=3), O.perm(seed, 0, "ffdperm", 3, 20))


@pytest.mark.parametrize("shapes,D", [([(40, 70, 4, 5), (64, 33, 8, 2), (1, 300, 1, 9)], 45),
                                      ([(256, 512, 32, 16), (300, 200, 16, 32)], 32 * 16 * 2),
                                      ([(2048, 2048, 32, 16), (512, 1024, 32, 128), (1024, 256, 128, 32),
                                        (208, 384, 64, 48)], 512 + 4096 + 4096 + 3072),
                                      # dA < dB: the A-first contraction, one to four 16-row tiles of A
                                      ([(64, 512, 48, 64), (128, 256, 16, 32), (192, 768, 64, 80)],
                                       48 * 64 + 16 * 32 + 64 * 80),
                                      # A-first with columns a multiple of 512: eight columns per lane,
                                      # one and two 16-row tiles of A
                                      ([(64, 512, 16, 32), (128, 1024, 32, 48)], 16 * 32 + 32 * 48),
                                      # B first with four and five 16-column tiles of B (two 16-row
                                      # tiles per wave), stacked rows ragged against the workgroup
                                      ([(256, 512, 128, 64), (208, 256, 96, 80)], 128 * 64 + 96 * 80)])
def test_qk_parity(shapes, D, dev):
    seed = 21
    xs = rand_inputs(shapes, 3, seed, dtype=torch.bfloat16, scale=0.01)
    s = sk("qk", shapes, D, seed, dev)
    y = s.apply([x.to(dev) for x in xs]).cpu().numpy()
    ins = [oracle_in(x)[0] for x in xs]
    exact = O.apply("qk", shapes, D, seed, ins, dtype="bf16")
    # bound of the configuration for bf16 inputs; the matrix-core path
    # multiplies by B to ~16 mantissa bits, so the error is far below it
    assert rel_err(y, exact) < TOL_BF16
    assert rel_err(y, exact) < 1e-4
    # the transpose multiplies by the fp32 factors: the fp32 bound
    g = torch.Generator().manual_seed(3)
    z = torch.randn((2, D), generator=g)
    outs = s.apply_T(z.to(dev))
    refs = O.apply_T("qk", shapes, D, seed, z.numpy().astype(np.float64))
    for o, r in zip(outs, refs):
        assert rel_err(o.cpu().numpy(), r) < TOL_F32
    # fp32 inputs take the fp32 factors too
    xf = rand_inputs(shapes, 2, seed + 1)
    yf = s.apply([x.to(dev) for x in xf]).cpu().numpy()
    assert rel_err(yf, O.apply("qk", shapes, D, seed, [x.numpy() for x in xf])) < TOL_F32


@pytest.mark.parametrize("ws_mb", [None, 16])
def test_afjl_transpose_layer_groups(ws_mb, dev, monkeypatch):
    """AFJL transposes run in groups of layers per launch (at most 64, fewer when the workspace holds fewer
    D-vectors per batch): 71 layers, a call over a sub-range, theta0 on some layers, and a 16 MB workspace
    that forces groups of 21 layers at D = 2^16, batch 3."""
    from paper_2402_03994_amd import Sketch
    if ws_mb is not None:
        monkeypatch.setenv("SK_WORKSPACE_MB", str(ws_mb))
    shapes = [(1, 37 + 11 * i) for i in range(70)] + [(3, 5000)]
    D, seed, f, cnt = (1 << 16, 31, 0, 71) if ws_mb else (1024, 30, 5, 66)
    s = Sketch("afjl", shapes, D, seed, device=dev)
    g = torch.Generator().manual_seed(seed)
    z = torch.randn((3, D), generator=g)
    th = [torch.randn(r * c, generator=g) * 0.02 if i % 3 == 0 else None for i, (r, c) in enumerate(shapes)]
    sub = th[f:f + cnt]
    outs = s.apply_T(z.to(dev), theta0=[None if t is None else t.to(dev) for t in sub], first_layer=f, n_layers=cnt)
    refs = O.apply_T("afjl", shapes[f:f + cnt], D, seed, z.numpy().astype(np.float64), layer0=f,
                     theta0=[None if t is None else t.numpy() for t in sub])
    for o, r in zip(outs, refs):
        assert rel_err(o.cpu().numpy(), r) < TOL_F32
    s.close()


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("aligned", [True, False])
def test_afjl_single_vector(dtype, aligned, dev):
    """One vector (the single-vector fold kernel: shared sign blocks, deeper prefetch): 16-byte and scalar
    loads, fp32 and bf16, ragged rows, a layer of 1025 source rows (several fold items), D = 4096."""
    from paper_2402_03994_amd import Sketch
    shapes = [(1, 3000), (64, 1024), (1025, 1024)] if aligned else [(1, 3001), (7, 1001), (1, 2 ** 20 + 3)]
    D, seed = 4096, 77
    xs = rand_inputs(shapes, 1, seed, dtype=dtype, scale=0.01)
    s = Sketch("afjl", shapes, D, seed, device=dev)
    y = s.apply([x.to(dev) for x in xs]).cpu().numpy()
    ref = O.apply("afjl", shapes, D, seed, [oracle_in(x)[0] for x in xs], dtype=oracle_in(xs[0])[1])
    assert rel_err(y, ref) < TOL_F32
    s.close()


@pytest.mark.parametrize("D", [16, 64, 4096, 8192])
def test_ffd_small_D_vector_tiles(D, dev):
    """FFD with D <= 2^13 (one workgroup per block group and tile of vectors, the block's permutation,
    Gaussians and signs built once in LDS): 5 vectors (a partial tile), ragged tail, blocks of D < 128
    that do not start on a 128-coordinate boundary, forward and theta0 + S^T z."""
    shapes = [(1, 5 * D + 7), (3, D // 2 + 1)]
    seed = 60 + D
    xs = rand_inputs(shapes, 5, seed)
    s = sk("ffd", shapes, D, seed, dev)
    y = s.apply([x.to(dev) for x in xs]).cpu().numpy()
    ref = O.apply("ffd", shapes, D, seed, [x.numpy() for x in xs])
    assert rel_err(y, ref) < TOL_F32
    g = torch.Generator().manual_seed(seed)
    z = torch.randn((5, D), generator=g)
    th = [torch.randn(r * c, generator=g) * 0.02 for r, c in shapes]
    outs = s.apply_T(z.to(dev), theta0=[t.to(dev) for t in th])
    refs = O.apply_T("ffd", shapes, D, seed, z.numpy().astype(np.float64), theta0=[t.numpy() for t in th])
    for o, r in zip(outs, refs):
        assert rel_err(o.cpu().numpy(), r) < TOL_F32
    s.close()


@pytest.mark.parametrize("shapes,D", [([(1, 5000), (1, 20000), (1, 9)], 16384), ([(1, 2 ** 20), (2, 3)], 16)])
def test_fjl_transpose_tiles(shapes, D, dev):
    """FJL transpose with the sample scatter fused into the first transform pass (a per-tile range of
    the position-sorted sample list): layers shorter than D padded to N' = D (D samples over D positions,
    so many positions take several samples, summed in id order), empty tiles (16 samples over the 128
    tiles of 2^13 entries of an N' = 2^20 layer), tiny layers (n = 9 and 6), three vectors, theta0."""
    seed = 77 + D
    g = torch.Generator().manual_seed(seed)
    z = torch.randn((3, D), generator=g)
    th = [torch.randn(r * c, generator=g) * 0.02 for r, c in shapes]
    s = sk("fjl", shapes, D, seed, dev)
    outs = s.apply_T(z.to(dev), theta0=[t.to(dev) for t in th])
    refs = O.apply_T("fjl", shapes, D, seed, z.numpy().astype(np.float64), theta0=[t.numpy() for t in th])
    for o, r in zip(outs, refs):
        assert rel_err(o.cpu().numpy(), r) < TOL_F32
    s.close()


def test_ffd_partials_reduction_many_slots(dev):
    """FFD forward with D = 64 over 2^16 + 5 coordinates: 513 partial sums per output reduced in
    16-byte pieces (32 residues per workgroup, combined in a fixed order), accumulated over two layers;
    the result is bitwise the same in one batch and in two."""
    shapes = [(1, 2 ** 16 + 5), (4, 33)]
    D = 64
    xs = rand_inputs(shapes, 6, 91)
    s = sk("ffd", shapes, D, 91, dev)
    y = s.apply([x.to(dev) for x in xs]).cpu()
    ref = O.apply("ffd", shapes, D, 91, [x.numpy() for x in xs])
    assert rel_err(y.numpy(), ref) < TOL_F32
    y2 = torch.cat([s.apply([x[:2].to(dev) for x in xs]).cpu(), s.apply([x[2:].to(dev) for x in xs]).cpu()])
    assert torch.equal(y, y2)
    s.close()


# D above 2^16 (Sec. 4 sketches Hessians with AFFD at D = 2^20; the gradient benchmarks of the appendix use
# D in [2^17, 2^22]): AFFD's transposed-slab path with R = D / 1024 kept rows of the second digit (128, 256 and
# 1024) over layers of 8 and 64 slabs (N' = 2^23, 2^26), layers with N' = D, and FJL's sample gather and
# scatter over N' up to 2^26.
LARGE_D = [(2 ** 17, [(1, 5 * 2 ** 20 + 7), (1, 2 ** 17 - 3), (3, 1000)]),
           (2 ** 18, [(1, 2 ** 25 + 5), (7, 3001)]),
           (2 ** 20, [(1, 2 ** 25 + 5), (1, 2 ** 20 - 1), (2, 4097)])]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("case", range(len(LARGE_D)))
@pytest.mark.parametrize("kind", ["affd", "fjl"])
def test_large_D_forward(kind, case, dtype, dev):
    D, shapes = LARGE_D[case]
    seed = 400 + case
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    xs = rand_inputs(shapes, 3, seed, dtype=tdt, scale=0.01)
    s = sk(kind, shapes, D, seed, dev)
    y = s.apply([x.to(dev) for x in xs]).cpu().numpy()
    ref = O.apply(kind, shapes, D, seed, [oracle_in(x)[0] for x in xs], dtype=dtype)
    # bf16 inputs are widened exactly: the fp32 bound holds for both
    assert rel_err(y, ref) < TOL_F32
    s.close()


@pytest.mark.parametrize("case", range(len(LARGE_D)))
@pytest.mark.parametrize("kind", ["affd", "fjl"])
def test_large_D_transpose(kind, case, dev):
    D, shapes = LARGE_D[case]
    seed = 410 + case
    g = torch.Generator().manual_seed(seed)
    z = torch.randn((2, D), generator=g)
    th = [None] * (len(shapes) - 1) + [torch.randn(shapes[-1][0] * shapes[-1][1], generator=g) * 0.02]
    s = sk(kind, shapes, D, seed, dev)
    outs = s.apply_T(z.to(dev), theta0=[None if t is None else t.to(dev) for t in th])
    refs = O.apply_T(kind, shapes, D, seed, z.numpy().astype(np.float64),
                     theta0=[None if t is None else t.numpy() for t in th])
    for o, r in zip(outs, refs):
        assert rel_err(o.cpu().numpy(), r) < TOL_F32
    s.close()


def test_affd_large_D_regenerated_gaussians(dev):
    """AFFD at D = 2^20 with the Gaussians regenerated per call (no stored M tables) over a 64-slab layer,
    against the oracle and the default (stored-table) sketch."""
    from paper_2402_03994_amd import Sketch
    D, shapes = LARGE_D[2]
    seed = 420
    xs = rand_inputs(shapes, 2, seed, scale=0.01)
    ref = O.apply("affd", shapes, D, seed, [x.numpy() for x in xs])
    for flags in (Sketch.AFFD_NO_MTAB, 0):
        s = Sketch("affd", shapes, D, seed, device=dev, flags=flags)
        y = s.apply([x.to(dev) for x in xs]).cpu().numpy()
        assert rel_err(y, ref) < TOL_F32
        s.close()


@pytest.mark.parametrize("kind", ["fjl", "ffd"])
def test_d8192_parity(kind, dev):
    """D = 2^13, the widest small-D FFD blocks (32 values per thread) and the one-pass FJL with 32
    samples per thread (the transpose's products gathered from global memory): an N' = 2^21 layer
    (B = 5 low bits per tile row), an N' = 2^14 layer (B = 12) and one padded to N' = D, which keeps
    the pass-based path; forward, then the transpose with theta0."""
    shapes, D = [(1, 2 ** 20 + 3), (3, 5000), (1, 9)], 8192
    seed = 88
    xs = rand_inputs(shapes, 3, seed)
    s = sk(kind, shapes, D, seed, dev)
    y = s.apply([x.to(dev) for x in xs]).cpu().numpy()
    ref = O.apply(kind, shapes, D, seed, [x.numpy() for x in xs])
    assert rel_err(y, ref) < TOL_F32
    g = torch.Generator().manual_seed(seed)
    z = torch.randn((2, D), generator=g)
    th = [torch.randn(r * c, generator=g) * 0.02 for r, c in shapes]
    outs = s.apply_T(z.to(dev), theta0=[t.to(dev) for t in th])
    refs = O.apply_T(kind, shapes, D, seed, z.numpy().astype(np.float64), theta0=[t.numpy() for t in th])
    for o, r in zip(outs, refs):
        assert rel_err(o.cpu().numpy(), r) < TOL_F32
    s.close()
