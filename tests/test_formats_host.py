"""The library's E2M1 / E4M3 rounding (csrc/formats.h, __host__ __device__),
compiled for the host and compared with the oracle on dense sweeps."""
import ctypes as C
import os
import subprocess

import numpy as np
import pytest

import oracle
from paper_2608_13966_amd import build as B

HERE = os.path.dirname(os.path.abspath(__file__))


@pytest.fixture(scope="module")
def hostlib(tmp_path_factory):
    out = str(tmp_path_factory.mktemp("fmt") / "libformats_host.so")
    cmd = [B.hipcc(), "-O2", "-std=c++17", "-fPIC", "-shared", "-ffp-contract=off", "--offload-arch=gfx950",
           f"-I{B.CSRC}", os.path.join(HERE, "host", "formats_host.hip"), "-o", out]
    subprocess.check_call(cmd, stdout=subprocess.DEVNULL, stderr=subprocess.DEVNULL)
    L = C.CDLL(out)
    L.host_e2m1_round.argtypes = [C.c_float]
    L.host_e2m1_round.restype = C.c_float
    L.host_e2m1_code_of.argtypes = [C.c_float]
    L.host_e2m1_code_of.restype = C.c_uint
    L.host_e4m3_round.argtypes = [C.c_double, C.POINTER(C.c_uint)]
    L.host_e4m3_round.restype = C.c_double
    L.host_e4m3_round_f32.argtypes = [C.c_float, C.POINTER(C.c_uint)]
    L.host_e4m3_round_f32.restype = C.c_float
    return L


def test_e2m1_matches_oracle(hostlib):
    pts = list(np.linspace(-9, 9, 90001, dtype=np.float32))
    for m in (0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0, 6.0, 7.0):
        for s in (1.0, -1.0):
            x = np.float32(s * m)
            pts += [x, np.nextafter(x, np.float32(np.inf)), np.nextafter(x, np.float32(-np.inf))]
    pts += [np.float32(v) for v in (1e-38, -1e-38, 1e-45, 0.0, 3.0e38, -3.0e38, 1e30, 65504.0)]
    for y in pts:
        q = hostlib.host_e2m1_round(float(y))
        code = hostlib.host_e2m1_code_of(q)
        ref = oracle.e2m1_code(float(y))
        assert code == ref, (float(y), q, code, ref)
        mag = oracle.E2M1_MAGNITUDES[ref & 7]
        assert abs(q) == mag and (q == 0 or (q < 0) == (y < 0))


def test_e4m3_matches_oracle(hostlib):
    rng = np.random.default_rng(4)
    xs = list(np.exp(rng.uniform(np.log(1e-6), np.log(600), 20000)))
    for v in range(0x7F):
        val = oracle.e4m3_value(v)
        xs += [val, val * (1 + 1e-12), val * (1 - 1e-12)]
    for a, b in zip([oracle.e4m3_value(v) for v in range(0x7E)], [oracle.e4m3_value(v) for v in range(1, 0x7F)]):
        xs += [(a + b) / 2, np.nextafter((a + b) / 2, 0), np.nextafter((a + b) / 2, 1e9)]
    xs += [0.0, -1.0, 448.0, 464.0, 1e300, 2.0 ** -10, 1.5 * 2.0 ** -9]
    code = C.c_uint(0)
    for x in xs:
        val = hostlib.host_e4m3_round(float(x), C.byref(code))
        ref = oracle.e4m3_code(float(x))
        assert code.value == ref, (x, code.value, ref)
        assert val == oracle.e4m3_value(ref)


def test_e4m3_from_fp32_matches_oracle(hostlib):
    """fp32 inputs are exact in fp64, so the fp32 routine must agree with the
    oracle's fp64 rounding on every one of them (ties and saturation included)."""
    rng = np.random.default_rng(5)
    xs = list(np.exp(rng.uniform(np.log(1e-6), np.log(600), 20000)).astype(np.float32))
    vals = [oracle.e4m3_value(v) for v in range(0x7F)]
    for a, b in zip(vals[:-1], vals[1:]):
        m = np.float32((a + b) / 2)
        xs += [m, np.nextafter(m, np.float32(0)), np.nextafter(m, np.float32(1e9)), np.float32(a)]
    xs += [np.float32(v) for v in (0.0, -1.0, 448.0, 464.0, 500.0, 3e38, 2.0 ** -10, 1.5 * 2.0 ** -9, 1e-45)]
    code = C.c_uint(0)
    for x in xs:
        val = hostlib.host_e4m3_round_f32(float(x), C.byref(code))
        ref = oracle.e4m3_code(float(x))
        assert code.value == ref, (float(x), code.value, ref)
        assert val == np.float32(oracle.e4m3_value(ref))
