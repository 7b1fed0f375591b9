"""CPU checks of the tensor-level calls (paper_2607_22696_amd.ops): a tensor of the wrong
shape, dtype or layout raises ValueError naming it before anything reaches the C ABI (which
sees raw pointers only and could not tell).  The tensors here live on the CPU, so every call
also reports that q is not a CUDA tensor; each test checks that the planted problem is
reported too."""
import pytest
import torch

from paper_2607_22696_amd import ops

B, T, H, W, M, D, P = 1, 2, 3, 4, 2, 32, 27
Q = (B, T, H, W, M, D)


def bf(shape=Q):
    return torch.zeros(shape, dtype=torch.bfloat16)


def f32(shape):
    return torch.zeros(shape, dtype=torch.float32)


def fwd_args(**over):
    a = dict(q=bf(), k=bf(), v=bf(), offsets=f32(Q[:5] + (P, 3)))
    a.update(over)
    return a


def raises(fn, *want, **kw):
    with pytest.raises(ValueError) as e:
        fn(**kw)
    msg = str(e.value)
    for w in want:
        assert w in msg, (w, msg)
    return msg


def test_forward_checks_every_tensor():
    raises(ops.forward, "q: not a CUDA tensor", **fwd_args())
    raises(ops.forward, "k: shape", **fwd_args(k=bf((B, T, H, W, M, 64))))
    raises(ops.forward, "v: dtype", **fwd_args(v=f32(Q)))
    raises(ops.forward, "offsets: shape", **fwd_args(offsets=f32(Q[:5] + (26, 3))))
    raises(ops.forward, "offsets: dtype", **fwd_args(offsets=torch.zeros(Q[:5] + (P, 3),
                                                                          dtype=torch.float64)))
    raises(ops.forward, "out: dtype", **fwd_args(out=f32(Q)))
    raises(ops.forward, "lse: shape", **fwd_args(lse=f32(Q[:4])))
    raises(ops.forward, "k: not contiguous", **fwd_args(k=bf((B, T, H, W, D, M)).transpose(4, 5)))
    raises(ops.forward, "offsets: shape", kernel=(3, 5, 5), **fwd_args())
    raises(ops.forward, "q: expected [B, T, H, W, heads, head_dim]", **fwd_args(q=bf(Q[:5])))
    raises(ops.forward, "q: unsupported dtype", **fwd_args(q=torch.zeros(Q, dtype=torch.float16)))


def bwd_args(**over):
    a = dict(q=bf(), k=bf(), v=bf(), offsets=f32(Q[:5] + (P, 3)), lse=f32(Q[:5]), dout=bf())
    a.update(over)
    return a


def test_backward_checks_every_tensor():
    raises(ops.backward, "q: not a CUDA tensor", **bwd_args())
    raises(ops.backward, "dout: dtype", **bwd_args(dout=f32(Q)))
    raises(ops.backward, "lse: shape", **bwd_args(lse=f32(Q)))
    raises(ops.backward, "lse: dtype", **bwd_args(lse=bf(Q[:5])))
    raises(ops.backward, "offsets: shape", **bwd_args(offsets=f32(Q[:5] + (P,))))
    raises(ops.backward, "out: shape", **bwd_args(out=bf((B, T, H, W, M, 64))))
    good = (f32(Q), f32(Q), f32(Q), f32(Q[:5] + (P, 3)))
    raises(ops.backward, "dk: dtype", grads=(good[0], bf(), good[2], good[3]), **bwd_args())
    raises(ops.backward, "d_offsets: shape", grads=good[:3] + (f32(Q[:5] + (P,)),), **bwd_args())
    raises(ops.backward, "grads: expected", grads=good[:3], **bwd_args())
    raises(ops.backward, "workspace: dtype", workspace=f32((16,)), **bwd_args())


def test_predicted_weights_checks():
    args = dict(logits=f32(Q[:5] + (P,)), v=bf(), offsets=f32(Q[:5] + (P, 3)))
    raises(ops.pw_forward, "v: not a CUDA tensor", **args)
    raises(ops.pw_forward, "logits: shape", **dict(args, logits=f32(Q[:5] + (P + 1,))))
    raises(ops.pw_forward, "logits: dtype", **dict(args, logits=bf(Q[:5] + (P,))))
    bargs = dict(args, lse=f32(Q[:5]), dout=bf())
    raises(ops.pw_backward, "dout: dtype", **dict(bargs, dout=f32(Q)))
    raises(ops.pw_backward, "lse: shape", **dict(bargs, lse=f32(Q[:4])))
    raises(ops.pw_backward, "dlogits: shape",
           grads=(f32(Q[:5]), f32(Q), f32(Q[:5] + (P, 3))), **bargs)


def test_conv_checks():
    x = bf((B, T, H, W, 64))
    w = f32((64, 3, 3, 3))
    raises(ops.dwconv3d_forward, "x: not a CUDA tensor", x=x, weight=w)
    raises(ops.dwconv3d_forward, "weight: dtype", x=x, weight=bf((64, 3, 3, 3)))
    raises(ops.dwconv3d_forward, "weight: shape", x=x, weight=f32((32, 3, 3, 3)))
    raises(ops.dwconv3d_forward, "bias: shape", x=x, weight=w, bias=f32((63,)))
    raises(ops.dwconv3d_forward, "accumulate needs", x=x, weight=w, accumulate=True)
    raises(ops.dwconv3d_backward, "dy: dtype", x=x, weight=w, dy=f32(x.shape))
    raises(ops.dwconv3d_backward, "dx: dtype", x=x, weight=w, dy=bf(x.shape), dx=bf(x.shape))


def test_window_attention_checks():
    args = dict(q=bf(), k=bf(), v=bf())
    raises(ops.win_forward, "q: not a CUDA tensor", **args)
    raises(ops.win_forward, "q: unsupported dtype", **dict(args, q=f32(Q)))
    raises(ops.win_forward, "out_res: dtype", out_res=f32(Q), **args)
    bargs = dict(args, out=bf(), out_res=None, lse=f32(Q[:5]), dout=bf())
    raises(ops.win_backward, "out: shape", **dict(bargs, out=bf(Q[:5])))
    raises(ops.win_backward, "dq: dtype", grads=(bf(), f32(Q), f32(Q)), **bargs)
