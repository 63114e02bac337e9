"""Synthetic workloads of the benchmark and the full-size parity tests.

Shapes of the parameter tensors the sketches are applied to, and seeded input
generators.  Nothing here computes any part of a sketch; both the benchmark
(GPU inputs) and the tests (the same inputs handed to the oracle) take their
inputs from this module.

The paper measures real per-example gradients of fine-tuned language models;
no checkpoint or dataset is available here, so model-shaped tensors with
Gaussian (or heavy-tailed) entries stand in for them.
"""
from __future__ import annotations

import math

import torch


def gpt2_small_shapes():
    """GPT-2 small (N = 124,439,808): wte, wpe, 12 blocks, ln_f, in module order."""
    s = [(50257, 768), (1024, 768)]
    for _ in range(12):
        s += [(1, 768), (1, 768),            # ln_1 weight, bias
              (768, 2304), (1, 2304),        # attn.c_attn
              (768, 768), (1, 768),          # attn.c_proj
              (1, 768), (1, 768),            # ln_2
              (768, 3072), (1, 3072),        # mlp.c_fc
              (3072, 768), (1, 768)]         # mlp.c_proj
    s += [(1, 768), (1, 768)]                # ln_f
    return s


def decoder_1p3b_qk_shapes():
    """Weight matrices of a 1.3B-shaped decoder (24 layers, d=2048, ffn 8192,
    vocab 50304) with their QK output blocks (dA, dB); sum dA*dB = 2^18."""
    s = [(50304, 2048, 256, 64)]
    for _ in range(24):
        s += [(2048, 2048, 32, 16)] * 4     # q, k, v, o
        s += [(2048, 8192, 32, 128),        # fc1
              (8192, 2048, 128, 32)]        # fc2
    return s


def llama3_8b_shapes():
    """Llama-3-8B parameter tensors (N = 8,030,261,248) in module order."""
    s = [(128256, 4096)]
    for _ in range(32):
        s += [(4096, 4096), (1024, 4096), (1024, 4096), (4096, 4096),   # q, k, v, o
              (14336, 4096), (14336, 4096), (4096, 14336),              # gate, up, down
              (1, 4096), (1, 4096)]                                     # input / post-attention RMSNorm
    s += [(1, 4096), (128256, 4096)]                                     # final norm, lm_head
    return s


def llama3_8b_stream_groups():
    """Layer ranges (first, count) of the streamed calls: embedding, one call per
    transformer block, then final norm + lm_head."""
    g = [(0, 1)]
    for b in range(32):
        g.append((1 + 9 * b, 9))
    g.append((1 + 9 * 32, 2))
    return g


CONFIGS = {
    "c1": dict(kinds=("fjl", "ffd"), shapes=[(1, 1 << 20)], D=4096, batch=8, seed=0, dtype="f32"),
    "c2": dict(kinds=("afjl", "affd"), shapes=gpt2_small_shapes(), D=1 << 16, batch=64, seed=1, dtype="f32"),
    "c3": dict(kinds=("qk",), shapes=decoder_1p3b_qk_shapes(), D=1 << 18, batch=256, seed=0, dtype="bf16"),
    "c4": dict(kinds=("ffd",), shapes=[(1, 100_000_000)], D=1 << 20, batch=4, seed=0, dtype="f32"),
    "c5": dict(kinds=("afjl",), shapes=llama3_8b_shapes(), D=1 << 20, batch=8, seed=7, dtype="bf16"),
    # the C2 gradients through the sketches with the random-orthogonal pre-conditioner Q
    "c6": dict(kinds=("afjlq", "qkh"), shapes=gpt2_small_shapes(), D=1 << 16, batch=64, seed=1, dtype="f32"),
    # the C2 gradients through the sketch with the Fourier pre-conditioner (eq. frikadel, H_N -> FFT)
    "c10": dict(kinds=("afjlf",), shapes=gpt2_small_shapes(), D=1 << 16, batch=64, seed=1, dtype="f32"),
    # AFFD with Q (dense: ~4.3 GFLOP per vector and 2^20-element slab each way) on C1's vectors
    "c7": dict(kinds=("affdq",), shapes=[(1, 1 << 20)], D=4096, batch=8, seed=0, dtype="f32"),
    # sketched Hessian eigenvalues: Arnoldi (64 steps) on v -> S H S^T v, GPT-2-small parameters, a
    # synthetic rank-16 spiked Hessian (c8_hessian), AFJL sketch to D = 2^16
    "c8": dict(kinds=("afjl",), shapes=gpt2_small_shapes(), D=1 << 16, batch=1, seed=1, dtype="f32", krylov=64),
    # intrinsic-dimension search: FFD on C4's 1e8-entry vector (padded to 2^27), D_max = 2^20, on the
    # quadratic 1/2 theta^T H theta of a rank-8 synthetic Hessian (c9_problem)
    "c9": dict(kinds=("ffd",), shapes=[(1, 100_000_000)], D=1 << 20, batch=1, seed=0, dtype="f32", d_min=2,
               tau_target=0.9, delta=0.02, cg_steps=8, max_rounds=16),
}
# the objective of c9: 8 spikes, no bulk; theta0 = V V^T x (x ~ N(0, 1)) lies in their span
C9_LAMBDAS = (8.0, 6.0, 5.0, 4.0, 3.0, 2.5, 2.0, 1.5)
C9_HSEED = 99
# the synthetic Hessian of c8: 14 positive outliers, 2 negative ones, a flat bulk of 1e-5
C8_LAMBDAS = (20.0, 15.0, 11.0, 8.5, 6.5, 5.0, 4.0, 3.0, 2.5, 2.0, 1.6, 1.3, 1.1, 1.0, -3.0, -1.5)
C8_SHIFT = 1e-5
C8_HSEED = 4242
INPUT_SEED = {"c1": 1001, "c2": 1002, "c3": 1003, "c4": 1004, "c5": 1005, "c6": 1002, "c7": 1001, "c8": 1008,
              "c9": 1009, "c10": 1002}
# variance of the gradient entries (N(0, var)); C4's forward input is Student-t(3)
GRAD_VAR = {"c1": 1.0, "c2": 1e-4, "c3": 1e-4, "c4": None, "c5": 1e-5, "c6": 1e-4, "c7": 1.0, "c10": 1e-4}


def gaussian(shape, var: float, gen: torch.Generator, device, dtype=torch.float32) -> torch.Tensor:
    """Entries N(0, var); bf16 tensors are drawn in fp32 (one leading index at a
    time) and rounded to nearest even."""
    if dtype == torch.float32:
        return torch.randn(shape, generator=gen, device=device, dtype=torch.float32).mul_(math.sqrt(var))
    out = torch.empty(shape, device=device, dtype=dtype)
    for i in range(shape[0]):
        out[i] = torch.randn(shape[1:], generator=gen, device=device, dtype=torch.float32).mul_(math.sqrt(var))
    return out


def student_t3(shape, gen: torch.Generator, device) -> torch.Tensor:
    """Student-t with 3 degrees of freedom: Z / sqrt(chi2_3 / 3) (heavy-tailed, HVP-like)."""
    z = torch.randn(shape, generator=gen, device=device, dtype=torch.float32)
    chi2 = torch.zeros(shape, device=device, dtype=torch.float32)
    for _ in range(3):
        e = torch.randn(shape, generator=gen, device=device, dtype=torch.float32)
        chi2.add_(e * e)
    return z.div_(torch.sqrt(chi2.div_(3.0)))


def bf16_bits(x):
    """float32 numpy array -> bf16 bit patterns (uint16), rounded to nearest even."""
    import numpy as np

    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return u.astype(np.uint16)


def generator(cfg: str, device) -> torch.Generator:
    return torch.Generator(device=device).manual_seed(INPUT_SEED[cfg])


def c8_hessian(device):
    """The synthetic Hessian of c8 on `device` and its parameters as the oracle takes them."""
    import numpy as np

    from paper_2402_03994_amd import SyntheticHessian

    lam = np.array(C8_LAMBDAS, dtype=np.float32)
    H = SyntheticHessian(CONFIGS["c8"]["shapes"], len(lam), lam, C8_SHIFT, C8_HSEED, max_batch=1, device=device)
    return H, dict(rank=len(lam), lambdas=lam, shift=float(np.float32(C8_SHIFT)), seed=C8_HSEED)


def c9_x(device) -> torch.Tensor:
    """The seeded vector x ~ N(0, 1) ([1, n]) that c9's theta0 = V V^T x projects."""
    shapes = CONFIGS["c9"]["shapes"]
    return torch.randn((1, shapes[0][0] * shapes[0][1]), generator=generator("c9", device), device=device)


def c9_problem(device):
    """The objective's Hessian of c9 on `device`, its parameters as the oracle takes them, and theta0
    = V V^T x with x ~ N(0, 1) seeded (built with a unit-weight Hessian on the same sign vectors)."""
    import numpy as np

    from paper_2402_03994_amd import SyntheticHessian

    shapes = CONFIGS["c9"]["shapes"]
    lam = np.array(C9_LAMBDAS, dtype=np.float32)
    H = SyntheticHessian(shapes, len(lam), lam, 0.0, C9_HSEED, device=device)
    unit = SyntheticHessian(shapes, len(lam), np.ones(len(lam), dtype=np.float32), 0.0, C9_HSEED, device=device)
    theta0 = unit.apply([c9_x(device)])[0].reshape(-1)
    unit.close()
    return H, dict(rank=len(lam), lambdas=lam, shift=0.0, seed=C9_HSEED), [theta0]
