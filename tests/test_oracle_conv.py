"""The Eq. (1) oracle against its pins (CPU only)."""
import ctypes
import os
import shutil
import subprocess

import numpy as np
import pytest

from oracle import conv as oconv
from tests import conv_pins


@pytest.mark.parametrize("pin", conv_pins.ALL_PINS, ids=lambda p: p.__name__)
def test_oracle_pins(pin):
    pin(oconv.conv_fwd)


def test_points_match_full():
    rng = np.random.default_rng(11)
    In, Ker = conv_pins.rand_inputs((3, 5, 6, 9, 8, 3, 2), rng)
    full = oconv.conv_fwd(In, Ker)
    idx = rng.integers(0, full.size, 200)
    assert np.array_equal(oconv.conv_fwd_points(In, Ker, idx), full.reshape(-1)[idx])


def test_rejects_undefined_shapes():
    with pytest.raises(ValueError):
        oconv.conv_fwd(np.zeros((1, 1, 2, 2), np.float32), np.zeros((1, 1, 3, 1), np.float32))
    with pytest.raises(ValueError):
        oconv.conv_fwd(np.zeros((1, 2, 4, 4), np.float32), np.zeros((1, 3, 1, 1), np.float32))
    with pytest.raises(ValueError):
        oconv.conv_fwd_points(np.zeros((1, 1, 4, 4), np.float32),
                              np.zeros((1, 1, 1, 1), np.float32), np.array([16]))


# Plausible slips, planted in a copy of the oracle's C source; every one of
# them must fail at least one pin.
MUTATIONS = {
    "wrong_tap_index": ("(h + r)) * W + (w + s)", "(h + r)) * W + (w + (s + 1) % S)"),
    "kernel_flip": ("((size_t)c * R + r) * S + s]", "((size_t)c * R + (R - 1 - r)) * S + (S - 1 - s)]"),
    "drop_last_tap": ("for (int s = 0; s < S; ++s)", "for (int s = 0; s < S - 1; ++s)"),
    "input_channel_fixed": ("In_n[((size_t)c * H", "In_n[((size_t)0 * H"),
    "transposed_output": ("Out_nk[(size_t)h * Q + w]", "Out_nk[(size_t)w * P + h]"),
    "float_accumulator": ("double acc = 0.0;", "float acc = 0.0f;"),
    "sign_flip": ("acc += (double)In_n", "acc -= (double)In_n"),
    "channel_stride_kernel": ("Ker + (size_t)k * C * R * S", "Ker + (size_t)k * R * S"),
}


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_pins_catch_planted_mistake(name, tmp_path):
    if shutil.which("gcc") is None:
        pytest.skip("no host C compiler")
    src = open(os.path.join(os.path.dirname(oconv.__file__), "conv_ref.c")).read()
    old, new = MUTATIONS[name]
    assert old in src, f"mutation anchor not found: {old}"
    mutated = tmp_path / "mut.c"
    mutated.write_text(src.replace(old, new))
    lib_path = tmp_path / "libmut.so"
    subprocess.run(["gcc", "-O1", "-fopenmp", "-fPIC", "-shared", str(mutated), "-o", str(lib_path)],
                   check=True)
    lib = ctypes.CDLL(str(lib_path))
    fp, dp = ctypes.POINTER(ctypes.c_float), ctypes.POINTER(ctypes.c_double)
    lib.oracle_conv_fwd.argtypes = [ctypes.c_int] * 7 + [fp, fp, dp]
    lib.oracle_conv_fwd.restype = ctypes.c_int

    def mutant(In, Ker):
        In = np.ascontiguousarray(In, np.float32)
        Ker = np.ascontiguousarray(Ker, np.float32)
        N, C, H, W = In.shape
        K, _, R, S = Ker.shape
        out = np.zeros((N, K, H - R + 1, W - S + 1), np.float64)
        lib.oracle_conv_fwd(N, C, K, H, W, R, S, In.ctypes.data_as(fp), Ker.ctypes.data_as(fp),
                            out.ctypes.data_as(dp))
        return out

    failed = []
    for pin in conv_pins.ALL_PINS:
        try:
            pin(mutant)
        except AssertionError:
            failed.append(pin.__name__)
    assert failed, f"mutation {name} passed every pin"


# ---------------------------------------------------------------------------
# The strided, zero-padded form (row f2)

@pytest.mark.parametrize("pin", conv_pins.STRIDED_PINS, ids=lambda p: p.__name__)
def test_oracle_strided_pins(pin):
    pin(oconv.conv_fwd_ex)


def test_strided_points_match_full():
    rng = np.random.default_rng(12)
    In, Ker = conv_pins.rand_inputs((2, 3, 4, 11, 9, 3, 3), rng)
    full = oconv.conv_fwd_ex(In, Ker, (2, 2), (1, 1))
    idx = rng.integers(0, full.size, 100)
    assert np.array_equal(oconv.conv_fwd_ex_points(In, Ker, idx, (2, 2), (1, 1)), full.reshape(-1)[idx])


def test_strided_rejects_undefined_shapes():
    x, k = np.zeros((1, 1, 4, 4), np.float32), np.zeros((1, 1, 3, 3), np.float32)
    for st, pd in (((0, 1), (0, 0)), ((1, 1), (-1, 0)), ((1, 1), (0, 0))):
        if st == (1, 1) and pd == (0, 0):
            continue
        with pytest.raises(ValueError):
            oconv.conv_fwd_ex(x, k, st, pd)
    with pytest.raises(ValueError):
        oconv.conv_fwd_ex(np.zeros((1, 1, 2, 2), np.float32), np.zeros((1, 1, 5, 1), np.float32), (1, 1), (1, 0))


STRIDED_MUTATIONS = {
    "stride_swapped": ("const int y = h * sh + r - ph, x = w * sw + s - pw;",
                       "const int y = h * sw + r - ph, x = w * sh + s - pw;"),
    "pad_sign": ("const int y = h * sh + r - ph, x = w * sw + s - pw;",
                 "const int y = h * sh + r + ph, x = w * sw + s - pw;"),
    "padding_not_zero": ("if (y < 0 || y >= H || x < 0 || x >= W) continue;",
                         "if (y < 0 || y >= H || x < 0 || x >= W) { acc += 1.0; continue; }"),
    "edge_off_by_one": ("if (y < 0 || y >= H || x < 0 || x >= W) continue;",
                        "if (y < 0 || y >= H - 1 || x < 0 || x >= W) continue;"),
    "extent_ignores_pad": ("*P = (H + 2 * ph - R) / sh + 1;", "*P = (H - R) / sh + 1;"),
    "stride_not_applied": ("const int y = h * sh + r - ph, x = w * sw + s - pw;",
                           "const int y = h + r - ph, x = w * sw + s - pw;"),
}


@pytest.mark.parametrize("name", sorted(STRIDED_MUTATIONS))
def test_strided_pins_catch_planted_mistake(name, tmp_path):
    if shutil.which("gcc") is None:
        pytest.skip("no host C compiler")
    src = open(os.path.join(os.path.dirname(oconv.__file__), "conv_ref.c")).read()
    old, new = STRIDED_MUTATIONS[name]
    assert old in src, f"mutation anchor not found: {old}"
    mutated = tmp_path / "mut.c"
    mutated.write_text(src.replace(old, new))
    lib_path = tmp_path / "libmut.so"
    subprocess.run(["gcc", "-O1", "-fopenmp", "-fPIC", "-shared", str(mutated), "-o", str(lib_path)],
                   check=True)
    lib = ctypes.CDLL(str(lib_path))
    fp, dp = ctypes.POINTER(ctypes.c_float), ctypes.POINTER(ctypes.c_double)
    lib.oracle_conv_fwd_ex.argtypes = [ctypes.c_int] * 11 + [fp, fp, dp]
    lib.oracle_conv_fwd_ex.restype = ctypes.c_int

    def mutant(In, Ker, st, pd):
        In = np.ascontiguousarray(In, np.float32)
        Ker = np.ascontiguousarray(Ker, np.float32)
        N, C, H, W = In.shape
        K, _, R, S = Ker.shape
        P, Q = oconv.ex_extents(H, W, R, S, st, pd)
        out = np.zeros((N, K, P, Q), np.float64)
        rc = lib.oracle_conv_fwd_ex(N, C, K, H, W, R, S, st[0], st[1], pd[0], pd[1], In.ctypes.data_as(fp),
                                    Ker.ctypes.data_as(fp), out.ctypes.data_as(dp))
        assert rc == 0
        return out

    failed = []
    for pin in conv_pins.STRIDED_PINS:
        try:
            pin(mutant)
        except AssertionError:
            failed.append(pin.__name__)
    assert failed, f"mutation {name} passed every strided pin"
