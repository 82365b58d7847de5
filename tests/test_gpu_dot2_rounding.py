"""The rounding model that the envelope kinds' bound pass (score_kernel, kQuestBound ..
kRectifiedBound) assumes of v_dot2c_f32_bf16, d = a.lo b.lo + a.hi b.hi + c: at most 4 units of
2^-24 (|a.lo b.lo| + |a.hi b.hi| + |c|) from the exact sum, plus at most 3 * 2^-126 for subnormal
operands, products and results flushed to zero.  The bound's error budget allows 8 units; the
instruction has measured at most 2.76.  The probe runs one instruction per element
(tests/probes/dot2_probe.hip); the exact sums come from the host (a product of two bf16 values is
exact in fp64, the three-term sum is taken in long double)."""
import ctypes
import os

import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu
LIB = os.path.join(os.path.dirname(os.path.abspath(__file__)), "probes", "libdot2probe.so")
N = 1 << 20


def _bf16(x):
    """bf16 bit patterns of float32 values (truncated: any bf16 value will do) and their values."""
    bits = (np.asarray(x, np.float32).view(np.uint32) >> 16).astype(np.uint32)
    return bits, (bits << 16).view(np.float32).astype(np.float64)


def _operands(regime, rng):
    u = lambda: rng.uniform(-1.0, 1.0, N)
    scale = {"unit": lambda: 1.0,
             "wide": lambda: np.exp2(rng.integers(-30, 30, N)),
             "cancel": lambda: 1.0,
             "tiny": lambda: np.exp2(-rng.integers(118, 140, N).astype(np.float64))}[regime]
    (a0, v_a0), (a1, v_a1) = _bf16(u() * scale()), _bf16(u() * scale())
    (b0, v_b0), (b1, v_b1) = _bf16(u() * scale()), _bf16(u() * scale())
    if regime == "cancel":                 # c cancels the first product up to a small remainder
        c = (-(v_a0 * v_b0) + u() * 2.0 ** -10).astype(np.float32)
    elif regime == "tiny":
        c = (u() * np.exp2(-rng.integers(126, 136, N).astype(np.float64))).astype(np.float32)
    else:
        c = (u() * scale()).astype(np.float32)
    return a0 | (a1 << 16), b0 | (b1 << 16), c, v_a0 * v_b0, v_a1 * v_b1


@pytest.mark.parametrize("regime", ["unit", "wide", "cancel", "tiny"])
def test_dot2_bf16_error_model(regime):
    assert os.path.exists(LIB), "tests/probes/libdot2probe.so is not built (run __graft_entry__.build())"
    lib = ctypes.CDLL(LIB)
    lib.vxt_dot2_bf16.restype = ctypes.c_int
    lib.vxt_dot2_bf16.argtypes = [ctypes.c_void_p] * 4 + [ctypes.c_int, ctypes.c_void_p]
    rng = np.random.default_rng({"unit": 1, "wide": 2, "cancel": 3, "tiny": 4}[regime])
    a, b, c, p0, p1 = _operands(regime, rng)
    ta = torch.from_numpy(a.view(np.int32)).cuda()
    tb = torch.from_numpy(b.view(np.int32)).cuda()
    tc = torch.from_numpy(c).cuda()
    td = torch.full((N,), float("nan"), dtype=torch.float32, device="cuda")
    rc = lib.vxt_dot2_bf16(ta.data_ptr(), tb.data_ptr(), tc.data_ptr(), td.data_ptr(), N,
                           ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert rc == 0
    torch.cuda.synchronize()
    d = td.cpu().numpy().astype(np.longdouble)
    exact = p0.astype(np.longdouble) + p1.astype(np.longdouble) + c.astype(np.longdouble)
    S = np.abs(p0) + np.abs(p1) + np.abs(c.astype(np.float64))
    err = np.abs(d - exact)
    allowed = 4.0 * 2.0 ** -24 * S.astype(np.longdouble) + 3.0 * 2.0 ** -126
    worst = int(np.argmax(err - allowed))
    assert (err <= allowed).all(), (regime, worst, float(p0[worst]), float(p1[worst]), float(c[worst]),
                                    float(d[worst]), float(exact[worst]))
    if regime != "tiny":
        ratio = float(np.max(err / (2.0 ** -24 * S)))
        print(f"[dot2] {regime}: max error {ratio:.3f} units of 2^-24 (|p0| + |p1| + |c|)")
