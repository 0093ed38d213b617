"""Measured MFMA accumulation error against the certificate's model.

The certificate (Section 5.2's verification, with Theorem 1's (1 + eps) model
of each floating-point operation) assumes that an MFMA chain
    acc = C0;  acc += A_c B_c  (v_mfma_f32_32x32x16_{f16,bf16}, c = 0 .. kc-1)
returns, for each output, the exact sum of its t = 16 kc + 1 terms (the
exact fp16 / bf16 products and the seed C0) within
    gamma_{t+1} * sum |terms| + 16 kc * 2^-120,   gamma_t = t u / (1 - t u),
with u = 2^-23 per addition (twice the fp32 unit roundoff: room for
truncating adders) and the last term for products below the fp32 normal
range.  This test measures the error of the hardware on inputs chosen to
stress that model (random, heavy cancellation, a wide exponent spread,
products near the fp32 underflow threshold, and the folded seed of rows of
at most 8 elements) and asserts the bound, printing the largest ratio of
error to bound.  The exact sums are math.fsum of the fp64 products, which
are exact for fp16 and bf16 operands."""
import ctypes
import math
import os
import sys

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

HERE = os.path.dirname(os.path.abspath(__file__))
LIB = os.path.join(HERE, "hip", "libmfma_probe.so")
U = 2.0 ** -23


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def env():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a visible MI355X"
    if not os.path.exists(LIB):
        pytest.fail("tests/hip/libmfma_probe.so is not built (tests/hip/build_probe.py)")
    lib = ctypes.CDLL(LIB)
    lib.probe_mfma_chain.argtypes = [ctypes.c_int] + [ctypes.c_void_p] * 4 + [ctypes.c_int,
                                                                               ctypes.c_void_p]
    lib.probe_mfma_chain.restype = ctypes.c_int
    return torch, lib


def to_bf16_bits(x):
    """Round fp32 values to bf16 (nearest, ties to even); returns the bits."""
    b = np.asarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    b = (b + 0x7FFF + ((b >> 16) & 1)) >> 16
    return b.astype(np.uint16)


def bits_to_f64(bits, bf16):
    if bf16:
        return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return bits.view(np.float16).astype(np.float64)


def quantise(x, bf16):
    if bf16:
        return to_bf16_bits(x)
    return np.asarray(x, dtype=np.float16).view(np.uint16)


def run(env, bf16, abits, bbits, c0):
    """C = C0 + A B on the GPU; abits [32, K], bbits [K, 32] uint16, c0 [32, 32] fp32."""
    torch, lib = env
    K = abits.shape[1]
    assert abits.shape == (32, K) and bbits.shape == (K, 32) and K % 16 == 0
    a = torch.from_numpy(abits.astype(np.int16).copy()).cuda()
    b = torch.from_numpy(bbits.astype(np.int16).copy()).cuda()
    c = torch.from_numpy(np.ascontiguousarray(c0, dtype=np.float32)).cuda()
    out = torch.empty((32, 32), dtype=torch.float32, device="cuda")
    st = lib.probe_mfma_chain(int(bf16), a.data_ptr(), b.data_ptr(), c.data_ptr(),
                              out.data_ptr(), K // 16, None)
    assert st == 0
    torch.cuda.synchronize()
    return out.cpu().numpy().astype(np.float64)


def check(env, bf16, abits, bbits, c0, what, t=None):
    """Assert the error model on all 1,024 outputs; return the worst ratio.
    t: the number of terms the bound counts (default K + 1, every product
    and the seed; a layout whose zero products add nothing may pass fewer)."""
    got = run(env, bf16, abits, bbits, c0)
    A = bits_to_f64(abits, bf16)
    B = bits_to_f64(bbits, bf16)
    K = A.shape[1]
    c0 = np.asarray(c0, dtype=np.float32).astype(np.float64)
    if t is None:
        t = K + 1
    gam = (t + 1) * U / (1 - (t + 1) * U)
    worst = 0.0
    worst24 = 0.0
    for i in range(32):
        prods = A[i][:, None] * B  # [K, 32], exact
        for j in range(32):
            terms = np.concatenate(([c0[i, j]], prods[:, j]))
            exact = math.fsum(terms)
            mag = math.fsum(np.abs(terms))
            err = abs(got[i, j] - exact)
            bound = gam * mag + K * 2.0 ** -120
            assert err <= bound, "%s: C[%d,%d] = %r, exact %r, error %g > bound %g" % (
                what, i, j, got[i, j], exact, err, bound)
            if bound > 0:
                worst = max(worst, err / bound)
            g24 = (t + 1) * 2.0 ** -24
            if mag > 0:
                worst24 = max(worst24, err / (g24 * mag))
    say("%-34s worst error / bound (u = 2^-23): %.4f   (/ u = 2^-24 bound: %.4f)"
        % (what, worst, worst24))
    return worst


@pytest.mark.parametrize("bf16", [0, 1], ids=["f16", "bf16"])
@pytest.mark.parametrize("K", [16, 64, 512])
def test_random(env, bf16, K):
    rng = np.random.default_rng(9000 + K + bf16)
    scale = 2.0 ** 12 if not bf16 else 1.0
    for rep in range(4):
        a = quantise(rng.standard_normal((32, K)) * scale, bf16)
        b = quantise(rng.standard_normal((K, 32)) * scale, bf16)
        c0 = (-0.5 * rng.standard_normal((32, 32)) ** 2 * K * scale * scale).astype(np.float32)
        check(env, bf16, a, b, c0, "random K=%d rep %d" % (K, rep))


@pytest.mark.parametrize("bf16", [0, 1], ids=["f16", "bf16"])
def test_cancellation(env, bf16):
    """Pairs of terms that cancel to a small remainder, and a seed that cancels
    the rest: the sum is tiny next to the sum of magnitudes."""
    rng = np.random.default_rng(9100 + bf16)
    K = 512
    x = rng.standard_normal((32, K // 2)) * (2.0 ** 10 if not bf16 else 1.0)
    a = np.repeat(x, 2, axis=1)
    y = rng.standard_normal((K // 2, 32)) * (2.0 ** 10 if not bf16 else 1.0)
    b = np.empty((K, 32))
    b[0::2] = y
    b[1::2] = -y * (1.0 + 2.0 ** -6 * rng.standard_normal((K // 2, 32)))
    ab, bb = quantise(a, bf16), quantise(b, bf16)
    A, B = bits_to_f64(ab, bf16), bits_to_f64(bb, bf16)
    c0 = -(A @ B) * (1.0 + 2.0 ** -10)
    check(env, bf16, ab, bb, c0.astype(np.float32), "cancellation")


@pytest.mark.parametrize("bf16", [0, 1], ids=["f16", "bf16"])
def test_wide_exponent_spread(env, bf16):
    rng = np.random.default_rng(9200 + bf16)
    K = 256
    span = 12 if not bf16 else 50
    for rep in range(4):
        ea = rng.integers(-span, span + 1, (32, K))
        eb = rng.integers(-span, span + 1, (K, 32))
        a = np.sign(rng.standard_normal((32, K))) * (1 + rng.random((32, K))) * 2.0 ** ea
        b = np.sign(rng.standard_normal((K, 32))) * (1 + rng.random((K, 32))) * 2.0 ** eb
        c0 = rng.standard_normal((32, 32)) * 2.0 ** (2 * span - 4)
        check(env, bf16, quantise(a, bf16), quantise(b, bf16), c0.astype(np.float32),
              "exponent spread rep %d" % rep)


def test_near_underflow_bf16(env):
    """bf16 products around the fp32 normal threshold 2^-126 (fp16 operands,
    normal or zero after the quantiser's flush, cannot get there)."""
    rng = np.random.default_rng(9300)
    K = 128
    a = rng.standard_normal((32, K)) * 2.0 ** -63
    b = rng.standard_normal((K, 32)) * 2.0 ** -63
    c0 = np.zeros((32, 32), dtype=np.float32)
    check(env, 1, quantise(a, 1), quantise(b, 1), c0, "near underflow")


@pytest.mark.parametrize("bf16", [0, 1], ids=["f16", "bf16"])
def test_folded_seed(env, bf16):
    """Rows of at most 8 elements: one 16-wide k-step whose columns 8..11
    carry the seed -N_j / (2 c) as four parts (each the rounding of what the
    earlier parts left) and the queries the constant c there, so that
    acc = <xq, xr> - N_j / 2 comes out of the single MFMA.  Checked against
    the certificate's count t = d + 6 (the four zero columns add nothing)."""
    rng = np.random.default_rng(9400 + bf16)
    c = 32768.0 if not bf16 else 1.0
    scale = 2.0 ** 13 if not bf16 else 1.0
    r = rng.uniform(-1, 1, (32, 8)) * scale
    q = rng.uniform(-1, 1, (8, 32)) * scale
    rb = quantise(r, bf16)
    R = bits_to_f64(rb, bf16)
    a = np.zeros((32, 16))
    a[:, :8] = R
    for i in range(32):
        rest = -float(np.sum(R[i] * R[i])) / 2.0 / c
        for p in range(4):
            part = bits_to_f64(quantise(np.array([rest]), bf16), bf16)[0]
            a[i, 8 + p] = part
            rest -= part
    b = np.zeros((16, 32))
    b[:8] = q
    b[8:12] = c
    check(env, bf16, quantise(a, bf16), quantise(b, bf16), np.zeros((32, 32), np.float32),
          "folded seed", t=8 + 6)


@pytest.mark.parametrize("bf16", [0, 1], ids=["f16", "bf16"])
@pytest.mark.parametrize("d", [32, 512])
def test_seed_product(env, bf16, d):
    """Rows of more than 8 elements: the sub-tile's chain starts with a seed
    k-step whose columns 0..3 carry the four parts of -N_j / (2 c) against
    the constant c (the other twelve columns zero), followed by the d / 16
    data k-steps.  Checked against the certificate's own count for this
    layout, t = d + 6 (d products, four parts, a spare; the zero products add
    nothing), with the scale the planner gives fp16 rows of d elements
    (d 2^(2E) <= 2^31)."""
    rng = np.random.default_rng(9500 + bf16 + d)
    c = 32768.0 if not bf16 else 1.0
    lg = (d - 1).bit_length()
    scale = 2.0 ** min(14, (31 - lg) // 2) if not bf16 else 1.0
    r = rng.uniform(-1, 1, (32, d)) * scale
    q = rng.uniform(-1, 1, (d, 32)) * scale
    R = bits_to_f64(quantise(r, bf16), bf16)
    a = np.zeros((32, 16 + d))
    a[:, 16:] = R
    for i in range(32):
        rest = -float(np.sum(R[i] * R[i])) / 2.0 / c
        for p in range(4):
            part = bits_to_f64(quantise(np.array([rest]), bf16), bf16)[0]
            assert math.isfinite(part)
            a[i, p] = part
            rest -= part
    b = np.zeros((16 + d, 32))
    b[:4] = c
    b[16:] = q
    check(env, bf16, quantise(a, bf16), quantise(b, bf16), np.zeros((32, 32), np.float32),
          "seed product, d = %d" % d, t=d + 6)


@pytest.mark.parametrize("bf16", [0, 1], ids=["f16", "bf16"])
def test_absorption(env, bf16):
    """Every product below half an ulp of a large seed: sequential fp32
    additions rounded to nearest would drop each of them (error = their sum,
    about a fifth of the bound); wider internal sums drop less."""
    K = 512
    a = np.full((32, K), 0.75)
    b = np.full((K, 32), 0.5)  # products 0.375 < 1 = half an ulp of 2^24
    c0 = np.full((32, 32), 2.0 ** 24, dtype=np.float32)
    c0[::2] *= -1  # and the same below zero
    check(env, bf16, quantise(a, bf16), quantise(b, bf16), c0, "absorption")
