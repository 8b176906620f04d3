"""Pins for the oracle's explicit-frequency reposition (paper, Related work:
repositioning relies on rotary embeddings and their extensions; Sec. 8
"Multimodal" and Fig. "attention-variant adapters" (b): moving an image
re-rotates only the temporal M-RoPE channels, in the sectioned and the
interleaved layout).

Checked against the plain theta schedule (bit for bit), direct fp64 pair
rotations written here, the rotation group law, and an M-RoPE definition
written out here with three position axes (an image's tokens share one
temporal position and differ in height and width)."""
import numpy as np
import pytest

from paper_2606_17107_amd import synth


def f32(shape, seed):
    return np.random.default_rng(seed).standard_normal(shape).astype(np.float32)


def bf16(shape, seed):
    x = f32(shape, seed)
    return synth.to_numpy_bits(synth.from_numpy_bits(x).to(__import__("torch").bfloat16))


def pair_channels(style, r, i, o=0):
    return (o + i, o + i + r // 2) if style == 0 else (o + 2 * i, o + 2 * i + 1)


def rotate_np(x, angle_per_pair, style, r, o=0):
    """Rotate the rotary pairs of rows x (fp64) by the given per-pair angles (broadcast over rows)."""
    y = x.astype(np.float64).copy()
    for i in range(r // 2):
        ca, cb = pair_channels(style, r, i, o)
        a, b = x[..., ca].astype(np.float64), x[..., cb].astype(np.float64)
        c, s = np.cos(angle_per_pair[..., i]), np.sin(angle_per_pair[..., i])
        y[..., ca] = a * c - b * s
        y[..., cb] = a * s + b * c
    return y


@pytest.mark.parametrize("style,r,o", [(0, 128, 0), (1, 128, 0), (0, 64, 32), (1, 64, 512)])
def test_theta_table_equals_default(ref, style, r, o):
    d = max(128, o + r)
    k = bf16((2, 3, 40, d), 1)
    dst_a = bf16((2, 3, 100, d), 2)
    dst_b = dst_a.copy()
    src = np.arange(40, dtype=np.int32) + 7
    dst = np.arange(40, dtype=np.int32) * 2 + 3
    ref.reposition_splice(k, None, dst_a, None, src, dst, 5e5, r, o, style)
    ref.reposition_splice(k, None, dst_b, None, src, dst, 5e5, r, o, style, omega=synth.rope_omega(5e5, r))
    assert np.array_equal(dst_a, dst_b)


@pytest.mark.parametrize("style", [0, 1])
def test_zero_frequencies_copy_and_others_rotate(ref, style):
    r, d, n = 64, 64, 30
    w = np.abs(np.random.default_rng(3).standard_normal(r // 2)) * 0.3
    w[::3] = 0.0
    k = f32((1, 2, n, d), 4)
    out = np.zeros((1, 2, 200, d), np.float32)
    src = np.arange(n, dtype=np.int32)
    dst = src + 111
    ref.reposition_splice(k, None, out, None, src, dst, 1e4, r, 0, style, omega=w)
    got = out[:, :, dst]
    for i in range(r // 2):
        ca, cb = pair_channels(style, r, i)
        if w[i] == 0.0:
            assert np.array_equal(got[..., ca], k[..., ca]) and np.array_equal(got[..., cb], k[..., cb])
    want = rotate_np(k, np.broadcast_to(111.0 * w, k.shape[:-1] + (r // 2,)), style, r)
    np.testing.assert_allclose(got, want, rtol=0, atol=2e-6)


def test_table_group_law(ref):
    """R_w(a) R_w(b) = R_w(a + b) for an arbitrary table (fp32 storage, two roundings)."""
    r, d, n = 128, 128, 25
    w = np.random.default_rng(5).uniform(0, 2, r // 2)
    k = f32((1, 1, n, d), 6)
    zero = np.zeros(n, np.int32)
    mid = np.zeros((1, 1, n, d), np.float32)
    two = np.zeros((1, 1, n, d), np.float32)
    one = np.zeros((1, 1, n, d), np.float32)
    idx = np.arange(n, dtype=np.int32)
    ref.reposition_splice(k, None, mid, None, zero, zero + 700, 1e4, r, omega=w, dst_slot=idx)
    ref.reposition_splice(mid, None, two, None, zero + 700, zero + 1900, 1e4, r, omega=w, dst_slot=idx)
    ref.reposition_splice(k, None, one, None, zero, zero + 1900, 1e4, r, omega=w, dst_slot=idx)
    err = np.linalg.norm(two - one, axis=-1) / np.linalg.norm(one, axis=-1)
    assert err.max() < 1e-6


def test_table_helpers():
    w = synth.rope_omega(1e4, 8)
    np.testing.assert_allclose(w, [1.0, 0.1, 0.01, 0.001], rtol=1e-15)
    sec = synth.mrope_axes(128, (16, 24, 24), "sectioned")
    assert list(np.bincount(sec)) == [16, 24, 24] and (sec[:16] == 0).all() and (sec[16:40] == 1).all()
    inter = synth.mrope_axes(128, (24, 20, 20), "interleaved")
    assert list(np.bincount(inter)) == [24, 20, 20]
    assert list(inter[:9]) == [0, 1, 2] * 3 and (inter[60:] == 0).all()
    tw = synth.mrope_temporal_omega(1e6, 128, (16, 24, 24), "sectioned")
    assert (tw[16:] == 0).all() and np.array_equal(tw[:16], synth.rope_omega(1e6, 128)[:16])
    l31 = synth.llama31_omega(5e5, 128)
    base = synth.rope_omega(5e5, 128)
    wl = 2 * np.pi / base
    assert np.array_equal(l31[wl < 2048], base[wl < 2048])               # high frequencies kept
    np.testing.assert_allclose(l31[wl > 8192], base[wl > 8192] / 8.0, rtol=1e-15)   # low ones / factor
    assert np.all(np.diff(l31) < 0)                                       # still a decreasing schedule


def mrope_np(x, t, h, w_, theta, r, axes, style=0):
    """M-RoPE written out: pair i turns by pos[axis(i)] * theta^(-2i/r), pos = (t, h, w) per row."""
    om = theta ** (-2.0 * np.arange(r // 2) / r)
    pos = np.stack([t, h, w_], axis=-1).astype(np.float64)                 # [..., 3]
    ang = np.take_along_axis(pos[..., None, :], np.broadcast_to(axes[:, None], pos.shape[:-1] + (r // 2, 1)),
                             axis=-1)[..., 0] * om
    return rotate_np(x, ang, style, r)


@pytest.mark.parametrize("layout,sections", [("sectioned", (16, 24, 24)), ("interleaved", (24, 20, 20))])
def test_mrope_temporal_transplant_equals_recompute(ref, layout, sections):
    """An image's keys cached at temporal position t0 and moved to t0 + delta with the temporal table
    equal M-RoPE recomputed at (t0 + delta, h, w); height/width channels come through bit-exact."""
    theta, r, d = 1e6, 128, 128
    axes = synth.mrope_axes(r, sections, layout)
    hh, ww = np.meshgrid(np.arange(4), np.arange(6), indexing="ij")
    hh, ww = hh.reshape(-1).astype(np.int32), ww.reshape(-1).astype(np.int32)
    n = hh.size
    t0, delta = 37, 161
    k_pre = f32((2, 2, n, d), 7)
    src_keys = mrope_np(k_pre, np.full(n, t0), hh + t0, ww + t0, theta, r, axes).astype(np.float32)
    want = mrope_np(k_pre, np.full(n, t0 + delta), hh + t0, ww + t0, theta, r, axes)
    out = np.zeros((2, 2, 300, d), np.float32)
    slots = np.arange(n, dtype=np.int32) + 100
    ref.reposition_splice(src_keys, None, out, None, np.full(n, t0, np.int32), np.full(n, t0 + delta, np.int32),
                          theta, r, omega=synth.mrope_temporal_omega(theta, r, sections, layout), dst_slot=slots)
    got = out[:, :, slots]
    err = np.linalg.norm(got - want, axis=-1) / np.linalg.norm(want, axis=-1)
    assert err.max() < 1e-6
    for i in np.nonzero(axes != 0)[0]:
        for c in pair_channels(0, r, i):
            assert np.array_equal(got[..., c], src_keys[..., c])
    # without the table (all pairs moved) the spatial channels would be wrong
    wrong = np.zeros_like(out)
    ref.reposition_splice(src_keys, None, wrong, None, np.full(n, t0, np.int32), np.full(n, t0 + delta, np.int32),
                          theta, r, dst_slot=slots)
    assert np.linalg.norm(wrong[:, :, slots] - want) > 1e-2 * np.linalg.norm(want)


def test_llama31_scaled_transplant_equals_recompute(ref):
    theta, r = 5e5, 128
    w = synth.llama31_omega(theta, r)
    k_pre = f32((1, 4, 50, r), 8)
    src = np.arange(50, dtype=np.int32) + 1000
    dst = np.arange(50, dtype=np.int32) + 21000
    at_src = ref.rope_rows(k_pre, np.broadcast_to(src, (1, 4, 50)), theta, r, omega=w)
    direct = rotate_np(k_pre, np.broadcast_to(dst[:, None] * w, (1, 4, 50, r // 2)), 0, r)
    out = np.zeros((1, 4, 21050, r), np.float32)
    ref.reposition_splice(at_src, None, out, None, src, dst, theta, r, omega=w)
    got = out[:, :, dst]
    err = np.linalg.norm(got - direct, axis=-1) / np.linalg.norm(direct, axis=-1)
    assert err.max() < 1e-6
