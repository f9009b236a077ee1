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
