"""Pins for the oracle's RoPE and bf16 rounding, checked against closed forms,
textbook identities and library routines (not against the oracle itself).

RoPE is the positional encoding the repositioning relies on (paper, Related
work); its frequency schedule and pairing are the standard ones the paper's
GQA models use, as read in the oracle header.
"""
import math
import os

import numpy as np
import pytest
import torch

from paper_2606_17107_amd import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def f32_bits_to_bf16_bits(x):
    return synth.to_numpy_bits(torch.from_numpy(np.asarray(x, dtype=np.float32)).to(torch.bfloat16))


def bf16_bits_to_f64(b):
    return (np.asarray(b, dtype=np.uint32) << 16).view(np.float32).astype(np.float64)


# ---- bf16 rounding ---------------------------------------------------------

def _load_golden_rounding():
    rows = []
    with open(os.path.join(GOLDEN, "bf16_rounding.txt")) as f:
        for line in f:
            line = line.split("#")[0].strip()
            if line:
                x, bits = line.split()
                rows.append((float.fromhex(x), int(bits, 16)))
    return rows


def test_round_bf16_golden(ref):
    """Hand-derived IEEE cases: ties to even, carries, subnormals, overflow,
    and a value that double rounding (fp64 -> fp32 -> bf16) would get wrong."""
    rows = _load_golden_rounding()
    assert len(rows) >= 12
    for x, bits in rows:
        assert ref.round_bf16(x) == bits, (x.hex(), hex(ref.round_bf16(x)), hex(bits))


def test_round_bf16_matches_torch_on_fp32_values(ref):
    """For fp32-representable inputs, one RNE rounding equals torch's fp32->bf16 cast."""
    g = torch.Generator().manual_seed(1)
    x = torch.randn(20000, generator=g) * torch.exp(torch.randn(20000, generator=g) * 8)
    x = torch.cat([x, torch.tensor([0.0, -0.0, 1e-40, -3e-39, 3.3e38, -3.39e38])])
    want = synth.to_numpy_bits(x.to(torch.bfloat16))
    got = np.array([ref.round_bf16(float(v)) for v in x.numpy().astype(np.float64)], dtype=np.uint16)
    np.testing.assert_array_equal(got, want)


# ---- frequencies -----------------------------------------------------------

def test_omega_closed_form(ref):
    """theta = 10^4, r = 8: omega_i = 10^4^(-2i/8) = 10^-i exactly in the reals."""
    with open(os.path.join(GOLDEN, "rope_omega_theta1e4_r8.txt")) as f:
        want = [float(l.split("#")[0]) for l in f if l.split("#")[0].strip()]
    got = [ref.rope_omega(10000.0, 8, i) for i in range(4)]
    np.testing.assert_allclose(got, want, rtol=1e-15, atol=0)


def test_omega_pair0_is_one_for_any_theta(ref):
    for theta in (10.0, 1e4, 5e5, 1e6):
        for r in (2, 64, 128):
            assert ref.rope_omega(theta, r, 0) == 1.0


# ---- pairing, sign and angle ---------------------------------------------

@pytest.mark.parametrize("style", [0, 1])
@pytest.mark.parametrize("offset,r,d", [(0, 8, 8), (4, 8, 16), (512, 64, 576)])
def test_unit_vector_rotates_in_its_pair_plane(ref, style, offset, r, d):
    """A unit vector on the first channel of pair i moves only within pair i's
    plane, by the angle p*omega_i, counter-clockwise: (1, 0) -> (cos, sin)."""
    theta = 10000.0
    p = 7
    for i in range(r // 2):
        a = offset + (i if style == 0 else 2 * i)
        b = offset + (i + r // 2 if style == 0 else 2 * i + 1)
        x = np.zeros((1, d), dtype=np.float32)
        x[0, a] = 1.0
        y = ref.rope_rows(x, np.array([p], np.int32), theta, r, offset, style)
        ang = p * theta ** (-2.0 * i / r)
        mask = np.ones(d, bool)
        mask[[a, b]] = False
        assert np.all(y[0, mask] == 0)
        assert abs(y[0, a] - math.cos(ang)) < 1e-7
        assert abs(y[0, b] - math.sin(ang)) < 1e-7


def test_rope_dim2_is_complex_multiplication(ref):
    """r = 2: the single pair has omega = 1 and rotation by p is multiplication
    by exp(i p), independent of theta (textbook complex rotation)."""
    g = torch.Generator().manual_seed(2)
    x = torch.randn(64, 2, generator=g).numpy().astype(np.float32)
    pos = np.arange(-32, 32, dtype=np.int32) * 37
    z = (x[:, 0].astype(np.float64) + 1j * x[:, 1]) * np.exp(1j * pos.astype(np.float64))
    for theta in (10000.0, 123.0):
        y = ref.rope_rows(x, pos, theta, 2, 0, 0)
        np.testing.assert_allclose(y[:, 0], z.real, atol=1e-6, rtol=1e-6)
        np.testing.assert_allclose(y[:, 1], z.imag, atol=1e-6, rtol=1e-6)


def test_matches_rotate_half_formulation(ref):
    """HALF pairing equals the rotate-half formulation (x*cos + rotate_half(x)*sin
    with frequencies 1/theta^(arange(0, r, 2)/r)), computed here in fp64 torch."""
    g = torch.Generator().manual_seed(3)
    d, theta = 128, 500000.0
    x = torch.randn(40, d, generator=g, dtype=torch.float64).float()
    pos = torch.randint(0, 60000, (40,), generator=g, dtype=torch.int32)
    inv = 1.0 / theta ** (torch.arange(0, d, 2, dtype=torch.float64) / d)
    ang = pos.double()[:, None] * inv[None, :]
    emb = torch.cat([ang, ang], dim=-1)
    xd = x.double()
    rot_half = torch.cat([-xd[:, d // 2:], xd[:, : d // 2]], dim=-1)
    want = (xd * emb.cos() + rot_half * emb.sin()).float().numpy()
    got = ref.rope_rows(x.numpy(), pos.numpy(), theta, d, 0, 0)
    np.testing.assert_allclose(got, want, rtol=0, atol=1e-6)


# ---- rotation-group identities --------------------------------------------

@pytest.mark.parametrize("style", [0, 1])
def test_composition_and_relative_position(ref, style):
    """R(a) R(b) = R(a + b) within 1e-5 relative (fp32 storage), and
    <R(m) q, R(n) k> depends only on m - n."""
    g = torch.Generator().manual_seed(4)
    d, theta = 128, 1e6
    x = torch.randn(32, d, generator=g).numpy()
    p = torch.randint(0, 40000, (32,), generator=g, dtype=torch.int32).numpy()
    delta = torch.randint(-20000, 20000, (32,), generator=g, dtype=torch.int32).numpy()
    two_step = ref.rope_rows(ref.rope_rows(x, p, theta, d, 0, style), delta, theta, d, 0, style)
    direct = ref.rope_rows(x, p + delta, theta, d, 0, style)
    rel = np.linalg.norm(two_step - direct, axis=1) / np.linalg.norm(direct, axis=1)
    assert rel.max() <= 1e-5
    # relative position: shift both positions by the same amount
    q = x[:16].astype(np.float32)
    k = x[16:].astype(np.float32)
    m = p[:16]
    n = p[16:]
    s0 = np.einsum("ij,ij->i", ref.rope_rows(q, m, theta, d, 0, style).astype(np.float64),
                   ref.rope_rows(k, n, theta, d, 0, style).astype(np.float64))
    s1 = np.einsum("ij,ij->i", ref.rope_rows(q, m + 999, theta, d, 0, style).astype(np.float64),
                   ref.rope_rows(k, n + 999, theta, d, 0, style).astype(np.float64))
    np.testing.assert_allclose(s0, s1, rtol=1e-5, atol=1e-4)


def test_zero_position_is_identity_and_norm_preserved(ref):
    g = torch.Generator().manual_seed(5)
    x = torch.randn(64, 64, generator=g).to(torch.bfloat16)
    xb = synth.to_numpy_bits(x)
    y = ref.rope_rows(xb, np.zeros(64, np.int32), 10000.0, 64, 0, 0)
    np.testing.assert_array_equal(y, xb)
    y = ref.rope_rows(xb, np.full(64, 12345, np.int32), 10000.0, 64, 0, 0)
    n0 = np.linalg.norm(bf16_bits_to_f64(xb), axis=1)
    n1 = np.linalg.norm(bf16_bits_to_f64(y), axis=1)
    np.testing.assert_allclose(n1, n0, rtol=8e-3)
    assert not np.array_equal(y, xb)
