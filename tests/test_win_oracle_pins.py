"""Pins of the shifted-window attention oracle (the Swin-DiT baseline, Section 6.2: windows of
3 x 16 x 16 tokens, shifted-window attention).

Independent of the oracle's code:
  * Swin's own procedure in fp64 torch: pad the grid to whole windows, roll by -shift,
    partition into windows, label the regions the roll joined with slices of the padded grid,
    mask across regions and padding, softmax, un-partition, roll back, crop; autograd for
    dq, dk, dv;
  * a window covering the whole grid without shift is global attention (plain torch matmuls);
  * a 1 x 1 x 1 window returns v and LSE = scale <q, k> of the token itself;
  * bf16 inputs are read exactly.
"""
import math

import numpy as np
import pytest

import oracle
import testgen

torch = pytest.importorskip("torch")


def rand(shape, seed):
    return np.random.default_rng(seed).standard_normal(shape).astype(np.float32)


def axis_labels(n, win, shift):
    """Region label of each rolled coordinate along one axis (Swin's three slices)."""
    lab = torch.zeros(n, dtype=torch.int64)
    if shift > 0:
        lab[n - win:n - shift] = 1
        lab[n - shift:] = 2
    return lab


def torch_swin(q, k, v, win, shift, scale, dout):
    B, T, H, W, M, D = q.shape
    wt, wh, ww = win
    st, sh, sw = shift
    Tp, Hp, Wp = (math.ceil(T / wt) * wt, math.ceil(H / wh) * wh, math.ceil(W / ww) * ww)
    ts = [torch.tensor(a, dtype=torch.float64, requires_grad=True) for a in (q, k, v)]

    def prep(x):  # pad, roll, partition: [nwin, wt*wh*ww, M, D] with nwin = B*nT*nH*nW
        x = torch.nn.functional.pad(x, (0, 0, 0, 0, 0, Wp - W, 0, Hp - H, 0, Tp - T))
        x = torch.roll(x, shifts=(-st, -sh, -sw), dims=(1, 2, 3))
        x = x.reshape(B, Tp // wt, wt, Hp // wh, wh, Wp // ww, ww, M, D)
        return x.permute(0, 1, 3, 5, 2, 4, 6, 7, 8).reshape(-1, wt * wh * ww, M, D)

    valid = torch.zeros(B, Tp, Hp, Wp, dtype=torch.bool)
    valid[:, :T, :H, :W] = True
    valid = torch.roll(valid, shifts=(-st, -sh, -sw), dims=(1, 2, 3))
    lab = (axis_labels(Tp, wt, st)[:, None, None] * 9 + axis_labels(Hp, wh, sh)[None, :, None] * 3
           + axis_labels(Wp, ww, sw)[None, None, :])
    lab = lab[None].expand(B, Tp, Hp, Wp)

    def part(x):
        x = x.reshape(B, Tp // wt, wt, Hp // wh, wh, Wp // ww, ww)
        return x.permute(0, 1, 3, 5, 2, 4, 6).reshape(-1, wt * wh * ww)

    vw, lw = part(valid), part(lab)
    mask = (lw[:, :, None] == lw[:, None, :]) & vw[:, None, :]
    qw, kw_, vw_ = (prep(t) for t in ts)
    s = scale * torch.einsum("nqmd,nkmd->nmqk", qw, kw_)
    s = s.masked_fill(~mask[:, None], float("-inf"))
    lse = torch.logsumexp(s, -1)
    a = torch.exp(s - lse[..., None])
    a = torch.nan_to_num(a)  # fully masked rows (padding queries) are dropped below
    ow = torch.einsum("nmqk,nkmd->nqmd", a, vw_)

    def unprep(x, last):
        x = x.reshape(B, Tp // wt, Hp // wh, Wp // ww, wt, wh, ww, *last)
        nd = len(last)
        x = x.permute(0, 1, 4, 2, 5, 3, 6, *range(7, 7 + nd)).reshape(B, Tp, Hp, Wp, *last)
        x = torch.roll(x, shifts=(st, sh, sw), dims=(1, 2, 3))
        return x[:, :T, :H, :W]

    out = unprep(ow, (M, D))
    lse_g = unprep(lse.permute(0, 2, 1), (M,))
    (out * torch.tensor(dout, dtype=torch.float64)).sum().backward()
    return out.detach().numpy(), lse_g.detach().numpy(), tuple(t.grad.numpy() for t in ts)


CASES = [
    # (grid T, H, W), window, shift
    ((3, 8, 8), (3, 4, 4), (0, 0, 0)),
    ((6, 8, 8), (3, 4, 4), (1, 2, 2)),
    ((5, 7, 9), (3, 4, 4), (1, 2, 2)),      # padding on every axis
    ((4, 6, 10), (2, 3, 5), (0, 1, 3)),     # shift on two axes only
]


@pytest.mark.parametrize("grid,win,shift", CASES, ids=lambda c: "x".join(map(str, c)))
def test_matches_swin_procedure_with_autograd(grid, win, shift):
    B, M, D = 2, 2, 8
    T, H, W = grid
    q, k, v, dout = (rand((B, T, H, W, M, D), s) for s in (1, 2, 3, 4))
    scale = 0.35
    ro, rl, (rdq, rdk, rdv) = torch_swin(q, k, v, win, shift, scale, dout)
    shape = (B, T, H, W, M, D) + win + shift
    out, lse = oracle.win_forward(shape, "f32", q, k, v, scale=scale)
    np.testing.assert_allclose(out, ro, rtol=0, atol=1e-12)
    np.testing.assert_allclose(lse, rl, rtol=0, atol=1e-12)
    dq, dk, dv = oracle.win_backward(shape, "f32", q, k, v, dout, scale=scale)
    np.testing.assert_allclose(dq, rdq, rtol=0, atol=1e-11)
    np.testing.assert_allclose(dk, rdk, rtol=0, atol=1e-11)
    np.testing.assert_allclose(dv, rdv, rtol=0, atol=1e-11)
    out2, _ = oracle.win_forward(shape, "f32", q, k, v, frames=(1, 3), scale=scale)
    np.testing.assert_allclose(out2, out[:, 1:3], rtol=0, atol=1e-14)


def test_whole_grid_window_is_global_attention():
    B, T, H, W, M, D = 1, 2, 3, 4, 2, 8
    q, k, v = (rand((B, T, H, W, M, D), s) for s in (5, 6, 7))
    out, lse = oracle.win_forward((B, T, H, W, M, D, T, H, W, 0, 0, 0), "f32", q, k, v)
    q2, k2, v2 = (torch.tensor(a, dtype=torch.float64).reshape(B, -1, M, D) for a in (q, k, v))
    s = torch.einsum("bqmd,bkmd->bmqk", q2, k2) / math.sqrt(D)
    ref = torch.einsum("bmqk,bkmd->bqmd", torch.softmax(s, -1), v2).reshape(out.shape)
    np.testing.assert_allclose(out, ref.numpy(), rtol=0, atol=1e-12)
    np.testing.assert_allclose(lse, torch.logsumexp(s, -1).permute(0, 2, 1).reshape(lse.shape).numpy(),
                               rtol=0, atol=1e-12)


def test_unit_window_returns_v():
    B, T, H, W, M, D = 1, 2, 3, 3, 2, 4
    q, k, v = (rand((B, T, H, W, M, D), s) for s in (8, 9, 10))
    out, lse = oracle.win_forward((B, T, H, W, M, D, 1, 1, 1, 0, 0, 0), "f32", q, k, v, scale=0.5)
    np.testing.assert_allclose(out, v.astype(np.float64), rtol=0, atol=0)
    np.testing.assert_allclose(lse, 0.5 * np.sum(q.astype(np.float64) * k, -1), rtol=0, atol=1e-12)


def test_bf16_inputs_are_read_exactly():
    B, T, H, W, M, D = 1, 3, 5, 6, 2, 8
    shape = (B, T, H, W, M, D, 3, 4, 4, 1, 2, 2)
    raw = [rand((B, T, H, W, M, D), s) for s in (11, 12, 13, 14)]
    bf = [testgen.f32_to_bf16(a) for a in raw]
    ex = [testgen.bf16_to_f32(a) for a in bf]
    a = oracle.win_forward(shape, "bf16", *bf[:3])
    b = oracle.win_forward(shape, "f32", *ex[:3])
    for x, y in zip(a, b):
        np.testing.assert_array_equal(x, y)
    ga = oracle.win_backward(shape, "bf16", *bf)
    gb = oracle.win_backward(shape, "f32", *ex)
    np.testing.assert_array_equal(ga[0], gb[0])   # dq: per query
    for x, y in zip(ga[1:], gb[1:]):              # dk, dv: OpenMP atomic summation order
        np.testing.assert_allclose(x, y, rtol=0, atol=1e-12)


def test_backward_frame_range_is_exact_on_whole_regions():
    """With shift 1 and windows of 3 frames the temporal regions are frames [0,1), [1,4), [4,6):
    the backward over the queries of [1, 4) gives the full dq there, and the full dk, dv of keys
    in those frames (their queries all lie in the same frames)."""
    B, T, H, W, M, D = 1, 6, 5, 6, 2, 4
    shape = (B, T, H, W, M, D, 3, 4, 4, 1, 2, 2)
    q, k, v, dout = (rand((B, T, H, W, M, D), s) for s in (15, 16, 17, 18))
    full = oracle.win_backward(shape, "f32", q, k, v, dout)
    part = oracle.win_backward(shape, "f32", q, k, v, dout, frames=(1, 4))
    for a, b in zip(part, full):
        assert a.shape == (B, 3, H, W, M, D)
        np.testing.assert_allclose(a, b[:, 1:4], rtol=0, atol=1e-12)
