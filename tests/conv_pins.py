"""Checks that pin a CPU implementation of Eq. (1) to things other than itself.

Each ``pin_*`` takes ``conv(In, Ker) -> float64 ndarray [N,K,P,Q]`` (In, Ker
float32 numpy arrays in NCHW / KCRS) and raises AssertionError on a mismatch.
They are used on the oracle itself and, with planted mistakes, on mutated
copies of it (to show that a plausible slip fails at least one pin).
"""
import numpy as np
import torch

# Tiny shapes (N, C, K, H, W, R, S): asymmetric H/W and R/S so that a swapped
# index or a transposed operand changes the result; R == H and S == W edges.
TINY_SHAPES = (
    (2, 3, 4, 7, 5, 3, 2),
    (1, 2, 5, 4, 9, 4, 3),
    (2, 4, 3, 6, 6, 1, 1),
    (1, 1, 1, 1, 1, 1, 1),
    (3, 2, 2, 3, 5, 3, 1),
    (1, 5, 2, 6, 4, 2, 4),
)


def rand_inputs(shape, rng):
    N, C, K, H, W, R, S = shape
    In = rng.uniform(-1, 1, (N, C, H, W)).astype(np.float32)
    Ker = rng.uniform(-1, 1, (K, C, R, S)).astype(np.float32)
    return In, Ker


def im2col_reference(In, Ker):
    """Independent fp64 reference: explicit im2col matrix times the kernel matrix."""
    N, C, H, W = In.shape
    K, _, R, S = Ker.shape
    P, Q = H - R + 1, W - S + 1
    cols = np.empty((N, C, R, S, P, Q), dtype=np.float64)
    x = In.astype(np.float64)
    for r in range(R):
        for s in range(S):
            cols[:, :, r, s] = x[:, :, r:r + P, s:s + Q]
    A = Ker.astype(np.float64).reshape(K, C * R * S)
    B = cols.reshape(N, C * R * S, P * Q)
    return np.matmul(A[None], B).reshape(N, K, P, Q)


def _close(a, b, rtol=1e-12):
    scale = max(1.0, float(np.max(np.abs(b))) if b.size else 1.0)
    assert a.shape == b.shape, (a.shape, b.shape)
    err = float(np.max(np.abs(a - b))) if a.size else 0.0
    assert err <= rtol * scale, f"max err {err} vs scale {scale}"


def pin_im2col(conv, seed=1):
    rng = np.random.default_rng(seed)
    for shape in TINY_SHAPES:
        In, Ker = rand_inputs(shape, rng)
        _close(conv(In, Ker), im2col_reference(In, Ker))


def pin_torch(conv, seed=2):
    """Eq. (1) is exactly torch's conv2d (a correlation) with no padding."""
    rng = np.random.default_rng(seed)
    for shape in TINY_SHAPES:
        In, Ker = rand_inputs(shape, rng)
        ref = torch.nn.functional.conv2d(torch.from_numpy(In).double(),
                                         torch.from_numpy(Ker).double(), padding=0).numpy()
        _close(conv(In, Ker), ref)


def pin_ones(conv):
    """All-ones In and Ker: every output equals C*R*S exactly."""
    for (N, C, K, H, W, R, S) in TINY_SHAPES:
        out = conv(np.ones((N, C, H, W), np.float32), np.ones((K, C, R, S), np.float32))
        assert out.shape == (N, K, H - R + 1, W - S + 1)
        assert np.all(out == C * R * S), "all-ones closed form"


def pin_delta(conv, seed=3):
    """A one-hot kernel per output channel selects one shifted input channel."""
    rng = np.random.default_rng(seed)
    for (N, C, K, H, W, R, S) in TINY_SHAPES:
        In, _ = rand_inputs((N, C, K, H, W, R, S), rng)
        Ker = np.zeros((K, C, R, S), np.float32)
        sel = []
        for k in range(K):
            c0, r0, s0 = (3 * k + 1) % C, k % R, (k // R + 1) % S
            Ker[k, c0, r0, s0] = 1.0
            sel.append((c0, r0, s0))
        out = conv(In, Ker)
        P, Q = H - R + 1, W - S + 1
        for k, (c0, r0, s0) in enumerate(sel):
            expect = In[:, c0, r0:r0 + P, s0:s0 + Q].astype(np.float64)
            assert np.array_equal(out[:, k], expect), f"delta kernel k={k}"


def pin_shift(conv, seed=4):
    """Shift equivariance: shifting In by one column shifts Out by one column."""
    rng = np.random.default_rng(seed)
    In, Ker = rand_inputs((2, 3, 4, 7, 8, 3, 2), rng)
    In2 = np.zeros_like(In)
    In2[..., 1:] = In[..., :-1]
    a, b = conv(In, Ker), conv(In2, Ker)
    assert np.array_equal(b[..., 1:], a[..., :-1]), "shift equivariance (w)"
    In3 = np.zeros_like(In)
    In3[..., 1:, :] = In[..., :-1, :]
    c = conv(In3, Ker)
    assert np.array_equal(c[..., 1:, :], a[..., :-1, :]), "shift equivariance (h)"


def pin_integer(conv, seed=5):
    """Integer inputs: the fp64 sum is exact, equal to an int64 brute force."""
    rng = np.random.default_rng(seed)
    for (N, C, K, H, W, R, S) in TINY_SHAPES:
        In = rng.integers(-4, 5, (N, C, H, W))
        Ker = rng.integers(-4, 5, (K, C, R, S))
        P, Q = H - R + 1, W - S + 1
        ref = np.zeros((N, K, P, Q), np.int64)
        for r in range(R):
            for s in range(S):
                ref += np.einsum("nchw,kc->nkhw", In[:, :, r:r + P, s:s + Q], Ker[:, :, r, s])
        out = conv(In.astype(np.float32), Ker.astype(np.float32))
        assert np.array_equal(out, ref.astype(np.float64)), "integer exactness"


ALL_PINS = (pin_im2col, pin_torch, pin_ones, pin_delta, pin_shift, pin_integer)


# ---------------------------------------------------------------------------
# Pins of the strided, zero-padded form (row f2).  Each takes
# ``conv_ex(In, Ker, stride, pad) -> float64 [N,K,P,Q]``.

# (N, C, K, H, W, R, S, (sh, sw), (ph, pw)): stride 1-3, unequal strides and
# pads, 1x1 and 7x7 taps, outputs down to 1x1.
STRIDED_SHAPES = (
    (2, 3, 4, 9, 7, 3, 3, (2, 2), (1, 1)),
    (1, 2, 3, 8, 11, 3, 2, (2, 3), (1, 0)),
    (2, 4, 3, 6, 6, 1, 1, (2, 2), (0, 0)),
    (1, 3, 2, 11, 11, 7, 7, (2, 2), (3, 3)),
    (1, 2, 2, 5, 4, 3, 3, (1, 1), (2, 1)),
    (2, 1, 3, 4, 4, 4, 4, (3, 3), (0, 0)),
    (1, 3, 2, 7, 9, 2, 3, (3, 2), (1, 2)),
)


def _ex_extents(H, W, R, S, st, pd):
    return (H + 2 * pd[0] - R) // st[0] + 1, (W + 2 * pd[1] - S) // st[1] + 1


def pin_ex_torch(conv_ex, seed=21):
    """The strided, padded form equals torch's conv2d with stride and padding."""
    rng = np.random.default_rng(seed)
    for (N, C, K, H, W, R, S, st, pd) in STRIDED_SHAPES:
        In, Ker = rand_inputs((N, C, K, H, W, R, S), rng)
        ref = torch.nn.functional.conv2d(torch.from_numpy(In).double(), torch.from_numpy(Ker).double(),
                                         stride=st, padding=pd).numpy()
        _close(conv_ex(In, Ker, st, pd), ref)


def pin_ex_reduces_to_eq1(conv_ex, seed=22):
    """Stride 1 and no padding is Eq. (1) (the im2col reference)."""
    rng = np.random.default_rng(seed)
    for shape in TINY_SHAPES:
        In, Ker = rand_inputs(shape, rng)
        _close(conv_ex(In, Ker, (1, 1), (0, 0)), im2col_reference(In, Ker))


def pin_ex_subsample_of_padded(conv_ex, seed=23):
    """Closed form: the strided output is every sh-th row and sw-th column of
    the stride-1 correlation of the explicitly zero-padded input."""
    rng = np.random.default_rng(seed)
    for (N, C, K, H, W, R, S, st, pd) in STRIDED_SHAPES:
        In, Ker = rand_inputs((N, C, K, H, W, R, S), rng)
        Xp = np.pad(In, ((0, 0), (0, 0), (pd[0], pd[0]), (pd[1], pd[1])))
        full = im2col_reference(Xp, Ker)
        P, Q = _ex_extents(H, W, R, S, st, pd)
        _close(conv_ex(In, Ker, st, pd), full[:, :, ::st[0], ::st[1]][:, :, :P, :Q])


def pin_ex_hand_example(conv_ex):
    """The worked example in tests/golden/strided_hand_example.json."""
    import json
    import os
    g = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "strided_hand_example.json")))
    H, W = g["input_hw"]
    R, S = g["kernel_rs"]
    In = np.arange(1, H * W + 1, dtype=np.float32).reshape(1, 1, H, W)
    Ker = np.ones((1, 1, R, S), np.float32)
    out = conv_ex(In, Ker, tuple(g["stride"]), tuple(g["pad"]))
    assert np.array_equal(out[0, 0], np.array(g["expected"], np.float64)), out


def pin_ex_integer_brute_force(conv_ex, seed=24):
    """Integer inputs: exact against a pure-Python brute force of the definition."""
    rng = np.random.default_rng(seed)
    for (N, C, K, H, W, R, S, st, pd) in STRIDED_SHAPES[:4]:
        In = rng.integers(-3, 4, (N, C, H, W))
        Ker = rng.integers(-3, 4, (K, C, R, S))
        P, Q = _ex_extents(H, W, R, S, st, pd)
        ref = np.zeros((N, K, P, Q), np.int64)
        for n in range(N):
            for k in range(K):
                for h in range(P):
                    for w in range(Q):
                        acc = 0
                        for c in range(C):
                            for r in range(R):
                                for s in range(S):
                                    y, x = h * st[0] + r - pd[0], w * st[1] + s - pd[1]
                                    if 0 <= y < H and 0 <= x < W:
                                        acc += int(In[n, c, y, x]) * int(Ker[k, c, r, s])
                        ref[n, k, h, w] = acc
        out = conv_ex(In.astype(np.float32), Ker.astype(np.float32), st, pd)
        assert np.array_equal(out, ref.astype(np.float64)), "integer brute force"


STRIDED_PINS = (pin_ex_torch, pin_ex_reduces_to_eq1, pin_ex_subsample_of_padded, pin_ex_hand_example,
                pin_ex_integer_brute_force)
