"""Seeded synthetic inputs for the convolution path.

This module holds shapes and random-number recipes only -- none of the
convolution's arithmetic -- so that the tests, the smoke check and the
benchmark can feed the same tensors to both the HIP path and the oracle.

Shapes follow the layer table of the paper's evaluation (Table 1: ResNet-18
and similar layers, NCHW inputs, KCRS kernels), written as valid (unpadded)
stride-1 correlations, with H and W the *input* extents.  The paper uses no
dataset, only these shapes; values are uniform on [-1, 1) from a seeded CPU
generator.
"""
from dataclasses import dataclass

import torch


@dataclass(frozen=True)
class ConvShape:
    name: str
    N: int
    C: int
    K: int
    H: int
    W: int
    R: int
    S: int
    dtype: str = "f32"  # "f32", or "bf16" (bf16 In/Ker, fp32 accumulate and Out)
    seed: int = 0
    stride: int = 1     # strided, zero-padded layers (conv_fwd_ex); square
    pad: int = 0

    @property
    def P(self):
        return (self.H + 2 * self.pad - self.R) // self.stride + 1

    @property
    def Q(self):
        return (self.W + 2 * self.pad - self.S) // self.stride + 1

    def key(self):
        return (self.N, self.C, self.K, self.H, self.W, self.R, self.S)


# The five layer configurations.  Index 0 is the small case the CPU oracle
# finishes in well under a second; index 1 is the pointwise layer the headline
# benchmark line is quoted on.
CONFIGS = (
    ConvShape("conv3x3_n1_c64_k64_in58", 1, 64, 64, 58, 58, 3, 3, "f32", 1000),
    ConvShape("conv1x1_n32_c256_k64_in56", 32, 256, 64, 56, 56, 1, 1, "f32", 2000),
    ConvShape("conv3x3_n32_c128_k128_in30", 32, 128, 128, 30, 30, 3, 3, "f32", 3000),
    ConvShape("conv3x3_n32_c512_k512_in9", 32, 512, 512, 9, 9, 3, 3, "f32", 4000),
    ConvShape("conv3x3_bf16_n16_c32_k64_in226", 16, 32, 64, 226, 226, 3, 3, "bf16", 5000),
)

# Strided, "same"-padded layers of Table 1 (ResNet-18 R1*, R4*, R5*) at batch
# 32, for the strided path (conv_fwd_ex); not part of the five
# configurations above.
STRIDED_CONFIGS = (
    ConvShape("conv7x7s2p3_n32_c3_k64_in224", 32, 3, 64, 224, 224, 7, 7, "f32", 6000, 2, 3),
    ConvShape("conv3x3s2p1_n32_c64_k128_in56", 32, 64, 128, 56, 56, 3, 3, "f32", 7000, 2, 1),
    ConvShape("conv1x1s2_n32_c64_k128_in56", 32, 64, 128, 56, 56, 1, 1, "f32", 8000, 2, 0),
)

# Table 1's conv2d layers (Yolo-9000 and ResNet-18) at batch 1, fp32, with
# the table's stride and "same" padding (R // 2 on each side), as the
# networks use them.  MobileNet's depth-wise layers are not an instance of
# Eq. (1) and are left out.  (K, C, H = W, R = S, stride) per layer.
_TABLE1 = (
    ("Y0", 32, 3, 544, 3, 1), ("Y2", 64, 32, 272, 3, 1), ("Y4", 128, 64, 136, 3, 1),
    ("Y5", 64, 128, 136, 1, 1), ("Y8", 256, 128, 68, 3, 1), ("Y9", 128, 256, 68, 1, 1),
    ("Y12", 512, 256, 34, 3, 1), ("Y13", 256, 512, 34, 1, 1), ("Y18", 1024, 512, 17, 3, 1),
    ("Y19", 512, 1024, 17, 1, 1), ("Y23", 28269, 1024, 17, 1, 1),
    ("R1", 64, 3, 224, 7, 2), ("R2", 64, 64, 56, 3, 1), ("R3", 64, 64, 56, 1, 1),
    ("R4", 128, 64, 56, 3, 2), ("R5", 128, 64, 56, 1, 2), ("R6", 128, 128, 28, 3, 1),
    ("R7", 256, 128, 28, 3, 2), ("R8", 256, 128, 28, 3, 1), ("R9", 256, 256, 14, 3, 1),
    ("R10", 512, 256, 14, 3, 2), ("R11", 512, 256, 14, 1, 2), ("R12", 512, 512, 7, 3, 1),
)
TABLE1 = tuple(ConvShape(f"table1_{name}", 1, C, K, HW, HW, RS, RS, "f32", 9000 + i, st, RS // 2)
               for i, (name, K, C, HW, RS, st) in enumerate(_TABLE1))

BY_NAME = {c.name: c for c in CONFIGS + STRIDED_CONFIGS + TABLE1}


def make_inputs(shape, seed=None, kind="uniform"):
    """Host (CPU) tensors (In [N,C,H,W], Ker [K,C,R,S]).

    kind = "uniform": U[-1, 1) float32, In drawn before Ker from one generator.
    kind = "int":     integers in [-4, 4] (exact in fp32 and bf16; every
                      partial sum of a small layer stays an exact integer).
    For dtype "bf16" the float32 draws are rounded to bfloat16 (round to
    nearest even, torch's conversion).
    """
    g = torch.Generator(device="cpu")
    g.manual_seed(shape.seed if seed is None else seed)
    ish = (shape.N, shape.C, shape.H, shape.W)
    ksh = (shape.K, shape.C, shape.R, shape.S)
    if kind == "uniform":
        In = torch.rand(ish, generator=g, dtype=torch.float32) * 2 - 1
        Ker = torch.rand(ksh, generator=g, dtype=torch.float32) * 2 - 1
    elif kind == "int":
        In = torch.randint(-4, 5, ish, generator=g).to(torch.float32)
        Ker = torch.randint(-4, 5, ksh, generator=g).to(torch.float32)
    else:
        raise ValueError(kind)
    if shape.dtype == "bf16":
        In = In.to(torch.bfloat16)
        Ker = Ker.to(torch.bfloat16)
    return In.contiguous(), Ker.contiguous()
