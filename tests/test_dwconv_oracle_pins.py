"""Pins of the depthwise 3D convolution oracle (MegaSlide-DiT, Section 5.2, Eq. (1) first term;
Section 5.3, the offset network's depthwise nn.Conv3d with groups = channels).

The oracle is trusted only through these checks, each independent of its code:
  * torch.nn.functional.conv3d with groups = C (the layer Section 5.3 names) in fp64 on the
    CPU, and its autograd for dx, dw and dbias;
  * a delta filter reproduces a zero-filled shift of the input (numpy slicing);
  * the adjoint identity <conv(x), dy> = <x, dx(dy)> (dx is the transpose of the forward);
  * dw[c, tap] = <dy, x shifted by the tap> and dbias = sum of dy, written with slicing;
  * bf16 inputs are read exactly.
"""
import numpy as np
import pytest

import oracle
import testgen

torch = pytest.importorskip("torch")

KERNELS = [(1, 1, 1), (3, 3, 3), (1, 3, 5), (3, 5, 5), (5, 3, 1)]


def rand(shape, seed):
    return np.random.default_rng(seed).standard_normal(shape).astype(np.float32)


def torch_conv(x, w, bias):
    """x [B,T,H,W,C] -> torch NCDHW depthwise conv with 'same' zero padding, back to channels last."""
    C = x.shape[-1]
    kt, kh, kw = w.shape[1:]
    xt = torch.from_numpy(np.asarray(x, np.float64)).permute(0, 4, 1, 2, 3).requires_grad_(True)
    wt = torch.from_numpy(np.asarray(w, np.float64)).reshape(C, 1, kt, kh, kw).requires_grad_(True)
    bt = None if bias is None else torch.from_numpy(np.asarray(bias, np.float64)).requires_grad_(True)
    y = torch.nn.functional.conv3d(xt, wt, bt, padding=((kt - 1) // 2, (kh - 1) // 2, (kw - 1) // 2),
                                   groups=C)
    return xt, wt, bt, y.permute(0, 2, 3, 4, 1)


@pytest.mark.parametrize("k", KERNELS, ids=lambda k: "x".join(map(str, k)))
def test_forward_matches_torch_conv3d_groups(k):
    B, T, H, W, C = 2, 4, 5, 6, 3
    x = rand((B, T, H, W, C), 1)
    w = rand((C,) + k, 2)
    bias = rand((C,), 3)
    shape = (B, T, H, W, C) + k
    _, _, _, ref = torch_conv(x, w, bias)
    got = oracle.dwconv_forward(shape, "f32", x, w, bias)
    np.testing.assert_allclose(got, ref.detach().numpy(), rtol=0, atol=1e-12)
    # frame window
    got2 = oracle.dwconv_forward(shape, "f32", x, w, None, frames=(1, 3))
    _, _, _, ref2 = torch_conv(x, w, None)
    np.testing.assert_allclose(got2, ref2.detach().numpy()[:, 1:3], rtol=0, atol=1e-12)


@pytest.mark.parametrize("k", KERNELS, ids=lambda k: "x".join(map(str, k)))
def test_backward_matches_torch_autograd(k):
    B, T, H, W, C = 2, 4, 5, 6, 3
    x = rand((B, T, H, W, C), 4)
    w = rand((C,) + k, 5)
    bias = rand((C,), 6)
    dy = rand((B, T, H, W, C), 7)
    shape = (B, T, H, W, C) + k
    xt, wt, bt, y = torch_conv(x, w, bias)
    y.backward(torch.from_numpy(dy.astype(np.float64)))
    dx, dw, db = oracle.dwconv_backward(shape, "f32", x, w, dy)
    np.testing.assert_allclose(dx, xt.grad.permute(0, 2, 3, 4, 1).numpy(), rtol=0, atol=1e-11)
    np.testing.assert_allclose(dw, wt.grad.reshape((C,) + k).numpy(), rtol=0, atol=1e-10)
    np.testing.assert_allclose(db, bt.grad.numpy(), rtol=0, atol=1e-11)
    dx2, dw2, db2 = oracle.dwconv_backward(shape, "f32", x, w, dy, frames=(2, 4),
                                           weight_grads=False)
    np.testing.assert_allclose(dx2, dx[:, 2:4], rtol=0, atol=1e-14)
    assert dw2 is None and db2 is None


def shifted(x, dt, dh, dw_):
    """s[b,t,i,j,c] = x[b, t+dt, i+dh, j+dw, c], zero where that is outside the grid."""
    s = np.zeros_like(x, dtype=np.float64)
    T, H, W = x.shape[1:4]

    def rng(n, d):
        lo, hi = max(0, -d), min(n, n - d)
        return slice(lo, hi), slice(lo + d, hi + d)

    (ot, it), (oh, ih), (ow, iw) = rng(T, dt), rng(H, dh), rng(W, dw_)
    s[:, ot, oh, ow] = x[:, it, ih, iw]
    return s


def test_delta_filter_is_a_shift():
    B, T, H, W, C = 1, 5, 4, 7, 2
    k = (3, 5, 3)
    x = rand((B, T, H, W, C), 8)
    for tap in [(0, 0, 0), (2, 4, 2), (1, 2, 1), (0, 3, 2)]:
        w = np.zeros((C,) + k, np.float32)
        w[:, tap[0], tap[1], tap[2]] = 1.0
        y = oracle.dwconv_forward((B, T, H, W, C) + k, "f32", x, w)
        ref = shifted(x, tap[0] - 1, tap[1] - 2, tap[2] - 1)
        np.testing.assert_array_equal(y, ref)


def test_adjoint_identity_and_weight_gradient_by_shifts():
    B, T, H, W, C = 2, 4, 6, 5, 3
    k = (3, 3, 5)
    shape = (B, T, H, W, C) + k
    x = rand((B, T, H, W, C), 9)
    w = rand((C,) + k, 10)
    dy = rand((B, T, H, W, C), 11)
    y = oracle.dwconv_forward(shape, "f32", x, w)
    dx, dw, db = oracle.dwconv_backward(shape, "f32", x, w, dy)
    lhs = float(np.sum(y * dy))
    rhs = float(np.sum(x.astype(np.float64) * dx))
    assert abs(lhs - rhs) <= 1e-10 * max(1.0, abs(lhs))
    for a in range(k[0]):
        for e in range(k[1]):
            for f in range(k[2]):
                s = shifted(x, a - 1, e - 1, f - 2)
                ref = np.sum(dy.astype(np.float64) * s, axis=(0, 1, 2, 3))
                np.testing.assert_allclose(dw[:, a, e, f], ref, rtol=0, atol=1e-10)
    np.testing.assert_allclose(db, dy.astype(np.float64).sum(axis=(0, 1, 2, 3)), rtol=0,
                               atol=1e-11)


def test_bf16_inputs_are_read_exactly():
    B, T, H, W, C = 1, 3, 4, 4, 4
    k = (3, 3, 3)
    xf = rand((B, T, H, W, C), 12)
    xb = testgen.f32_to_bf16(xf)
    x_exact = testgen.bf16_to_f32(xb)
    w = rand((C,) + k, 13)
    dyb = testgen.f32_to_bf16(rand((B, T, H, W, C), 14))
    shape = (B, T, H, W, C) + k
    np.testing.assert_array_equal(oracle.dwconv_forward(shape, "bf16", xb, w),
                                  oracle.dwconv_forward(shape, "f32", x_exact, w))
    a = oracle.dwconv_backward(shape, "bf16", xb, w, dyb)
    b = oracle.dwconv_backward(shape, "f32", x_exact, w, testgen.bf16_to_f32(dyb))
    for u, v in zip(a, b):
        np.testing.assert_array_equal(u, v)


def test_malformed_problems_are_rejected():
    x = np.zeros((1, 2, 2, 2, 1), np.float32)
    w = np.zeros((1, 2, 3, 3), np.float32)
    with pytest.raises(ValueError):
        oracle.dwconv_forward((1, 2, 2, 2, 1, 2, 3, 3), "f32", x, w)
