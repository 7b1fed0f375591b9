"""Pins of the predicted-weights oracle (MegaSlide-DiT, Section 5.2: the module learns offsets
and attention weights; in this variant the weights are a softmax over per-point logits that a
linear layer predicts, with no q and no K).

Each check is independent of the oracle's code:
  * the grid_sample route of Section 5.3 in fp64 torch (5D bilinear sampling with zero
    padding) followed by softmax over the logits, with autograd for every gradient;
  * integer offsets: plain row gathers, no interpolation;
  * softmax facts: adding a constant to a row's logits changes nothing, the logit gradient of a
    row sums to zero, equal logits give the mean of the samples;
  * bf16 V is read exactly.
"""
import numpy as np
import pytest

import oracle
import testgen
from tests.test_oracle_pins import base_grid, positions_f32

torch = pytest.importorskip("torch")


def case(seed, B, T, H, W, M, D, kt, kh, kw, off_std=1.0):
    rng = np.random.default_rng(seed)
    P = kt * kh * kw
    v = rng.standard_normal((B, T, H, W, M, D)).astype(np.float32)
    # on a 2^-12 grid, so that adding a small constant to a row is exact in fp32
    logits = (np.round(2.0 * rng.standard_normal((B, T, H, W, M, P)) * 4096) / 4096).astype(np.float32)
    off = (off_std * rng.standard_normal((B, T, H, W, M, P, 3))).astype(np.float32)
    dout = rng.standard_normal((B, T, H, W, M, D)).astype(np.float32)
    return v, logits, off, dout


def torch_route(v, logits, off, kt, kh, kw, dout):
    B, T, H, W, M, D = v.shape
    P = kt * kh * kw
    vt = torch.tensor(v, dtype=torch.float64, requires_grad=True)
    lt = torch.tensor(logits, dtype=torch.float64, requires_grad=True)
    ot = torch.tensor(off, dtype=torch.float64, requires_grad=True)
    pos = torch.tensor(positions_f32(T, H, W, M, off, kt, kh, kw)) + (ot - ot.detach())
    size = torch.tensor([W, H, T], dtype=torch.float64)
    grid_n = (2.0 * pos + 1.0) / size - 1.0
    outs, lses = [], []
    for m in range(M):
        g = grid_n[:, :, :, :, m].reshape(B, T, H, W * P, 3)
        V5 = vt[:, :, :, :, m].permute(0, 4, 1, 2, 3)
        vs = torch.nn.functional.grid_sample(V5, g, mode="bilinear", padding_mode="zeros",
                                             align_corners=False)
        vs = vs.reshape(B, D, T, H, W, P).permute(0, 2, 3, 4, 5, 1)
        a = torch.softmax(lt[:, :, :, :, m], -1)
        outs.append((a[..., None] * vs).sum(-2))
        lses.append(torch.logsumexp(lt[:, :, :, :, m], -1))
    out = torch.stack(outs, 4)
    lse = torch.stack(lses, 4)
    (out * torch.tensor(dout, dtype=torch.float64)).sum().backward()
    return out.detach().numpy(), lse.detach().numpy(), lt.grad.numpy(), vt.grad.numpy(), \
        ot.grad.numpy()


@pytest.mark.parametrize("kern", [(1, 1, 1), (3, 3, 3), (1, 3, 5)], ids=lambda k: "x".join(map(str, k)))
def test_matches_grid_sample_route_with_autograd(kern):
    B, T, H, W, M, D = 2, 3, 4, 5, 2, 8
    v, logits, off, dout = case(1, B, T, H, W, M, D, *kern)
    shape = (B, T, H, W, M, D) + kern
    ro, rl, rdl, rdv, rdo = torch_route(v, logits, off, *kern, dout)
    out, lse = oracle.pw_forward(shape, "f32", logits, v, off)
    np.testing.assert_allclose(out.reshape(ro.shape), ro, rtol=0, atol=1e-12)
    np.testing.assert_allclose(lse.reshape(rl.shape), rl, rtol=0, atol=1e-12)
    dl, dv, do = oracle.pw_backward(shape, "f32", logits, v, off, dout)
    np.testing.assert_allclose(dl, rdl, rtol=0, atol=1e-11)
    np.testing.assert_allclose(dv, rdv, rtol=0, atol=1e-11)
    np.testing.assert_allclose(do, rdo, rtol=0, atol=1e-10)


def test_integer_offsets_are_weighted_row_gathers():
    B, T, H, W, M, D, kt, kh, kw = 1, 4, 5, 6, 2, 4, 3, 3, 3
    rng = np.random.default_rng(2)
    v, logits, _, _ = case(3, B, T, H, W, M, D, kt, kh, kw)
    ioff = rng.integers(-2, 3, (B, T, H, W, M, kt * kh * kw, 3))
    out, _ = oracle.pw_forward((B, T, H, W, M, D, kt, kh, kw), "f32", logits, v,
                               ioff.astype(np.float32))
    g = base_grid(kt, kh, kw)
    l64 = logits.astype(np.float64)
    a = np.exp(l64 - l64.max(-1, keepdims=True))
    a /= a.sum(-1, keepdims=True)
    ref = np.zeros((B, T, H, W, M, D))
    for t in range(T):
        for i in range(H):
            for j in range(W):
                for m in range(M):
                    for p in range(len(g)):
                        x, y, z = (np.array([j, i, t]) + g[p] + ioff[0, t, i, j, m, p])
                        if 0 <= x < W and 0 <= y < H and 0 <= z < T:
                            ref[0, t, i, j, m] += a[0, t, i, j, m, p] * v[0, z, y, x, m]
    np.testing.assert_allclose(out.reshape(ref.shape), ref, rtol=0, atol=1e-12)


def test_softmax_facts():
    B, T, H, W, M, D, kt, kh, kw = 1, 3, 4, 4, 2, 8, 3, 3, 3
    shape = (B, T, H, W, M, D, kt, kh, kw)
    v, logits, off, dout = case(4, B, T, H, W, M, D, kt, kh, kw)
    out, lse = oracle.pw_forward(shape, "f32", logits, v, off)
    shifted = (logits + np.float32(3.0)).astype(np.float32)
    out2, lse2 = oracle.pw_forward(shape, "f32", shifted, v, off)
    np.testing.assert_allclose(out2, out, rtol=0, atol=1e-12)
    dl, _, _ = oracle.pw_backward(shape, "f32", logits, v, off, dout)
    np.testing.assert_allclose(dl.sum(-1), 0.0, rtol=0, atol=1e-12)
    # equal logits: the plain mean of the P samples (zero offsets: integer gathers)
    zero = np.zeros_like(logits)
    out3, lse3 = oracle.pw_forward(shape, "f32", zero, v, np.zeros_like(off))
    np.testing.assert_allclose(lse3, np.log(kt * kh * kw), rtol=0, atol=1e-12)
    g = base_grid(kt, kh, kw)
    ref = np.zeros((T, H, W, M, D))
    for t in range(T):
        for i in range(H):
            for j in range(W):
                for p in range(len(g)):
                    x, y, z = np.array([j, i, t]) + g[p]
                    if 0 <= x < W and 0 <= y < H and 0 <= z < T:
                        ref[t, i, j] += v[0, z, y, x].astype(np.float64) / len(g)
    np.testing.assert_allclose(out3.reshape(ref.shape), ref, rtol=0, atol=1e-12)


def test_bf16_values_are_read_exactly():
    B, T, H, W, M, D, kt, kh, kw = 1, 3, 4, 5, 2, 8, 3, 3, 3
    shape = (B, T, H, W, M, D, kt, kh, kw)
    v, logits, off, dout = case(5, B, T, H, W, M, D, kt, kh, kw)
    vb, gb = testgen.f32_to_bf16(v), testgen.f32_to_bf16(dout)
    a = oracle.pw_forward(shape, "bf16", logits, vb, off)
    b = oracle.pw_forward(shape, "f32", logits, testgen.bf16_to_f32(vb), off)
    for x, y in zip(a, b):
        np.testing.assert_array_equal(x, y)
    a = oracle.pw_backward(shape, "bf16", logits, vb, off, gb)
    b = oracle.pw_backward(shape, "f32", logits, testgen.bf16_to_f32(vb), off,
                           testgen.bf16_to_f32(gb))
    np.testing.assert_array_equal(a[0], b[0])   # dlogits: per query, fixed order
    np.testing.assert_array_equal(a[2], b[2])   # d_offsets
    # dV is scattered by OpenMP threads with atomic adds: only the summation order may differ
    np.testing.assert_allclose(a[1], b[1], rtol=0, atol=1e-12)


def test_minus_infinity_logits_drop_their_points():
    """A logit of -inf takes its point out of the softmax (weight exactly 0), here for the
    leading points of every row (1 to 3 of them) and for one point in the middle; the
    result is the grid_sample route's, whose softmax gives those points weight 0."""
    B, T, H, W, M, D, kt, kh, kw = 1, 3, 4, 5, 2, 8, 3, 3, 3
    shape = (B, T, H, W, M, D, kt, kh, kw)
    v, logits, off, dout = case(6, B, T, H, W, M, D, kt, kh, kw)
    lead = 1 + np.arange(B * T * H * W * M).reshape(B, T, H, W, M) % 3
    for p in range(3):
        logits[..., p][lead > p] = -np.inf
    logits[..., 13] = -np.inf
    ro, rl, rdl, rdv, rdo = torch_route(v, logits, off, kt, kh, kw, dout)
    out, lse = oracle.pw_forward(shape, "f32", logits, v, off)
    assert np.all(np.isfinite(out)) and np.all(np.isfinite(lse))
    np.testing.assert_allclose(out.reshape(ro.shape), ro, rtol=0, atol=1e-12)
    np.testing.assert_allclose(lse.reshape(rl.shape), rl, rtol=0, atol=1e-12)
    dl, dv, do = oracle.pw_backward(shape, "f32", logits, v, off, dout)
    np.testing.assert_allclose(dl, rdl, rtol=0, atol=1e-11)
    np.testing.assert_allclose(dv, rdv, rtol=0, atol=1e-11)
    np.testing.assert_allclose(do, rdo, rtol=0, atol=1e-10)
