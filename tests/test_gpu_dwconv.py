"""GPU-vs-oracle parity of the depthwise 3D convolution (DWConv3D term of Eq. (1), Section 5.2;
the offset network's depthwise conv, Section 5.3), through the C ABI.

Tolerances
  * fp32 data: max-abs <= 1e-5 on y and dx.  The weight and bias gradients are sums over the
    whole grid whose size grows like sqrt(tokens); fp32 summation of n terms errs by about
    sqrt(n) u (u = 2^-24) of that size, so they are held to max |g - r| <= 1e-5 rms(r).
  * bf16 x / dy (fp32 accumulate): max over elements of |g - r| / max(|r|, 1e-2 rms(r)) <= 2e-2
    for y (stored in bf16), dx, dw and dbias, against the fp64 oracle on the same bf16 inputs.
Small grids are compared element by element (several 128-channel chunks, ragged channel and
token tails, filter rows reaching past every border); the full-size grids on whole frames
(y, dx) and, on the 130,560-token grid, on every weight and bias gradient.
"""
import numpy as np
import pytest

import oracle
import testgen
from tests.util import max_abs, rel_err, say, to_device, to_host

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

F32_TOL = 1e-5
BF16_TOL = 2e-2


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2607_22696_amd as dsa
    dsa.load()
    yield


def check(name, got, ref, bf16, reduction=False):
    if bf16:
        e = rel_err(got, ref)
        say(f"  {name}: rel {e:.3e} (max-abs {max_abs(got, ref):.3e})")
        assert e <= BF16_TOL, name
    elif reduction:
        rms = float(np.sqrt(np.mean(np.asarray(ref, np.float64) ** 2)))
        e = max_abs(got, ref)
        say(f"  {name}: max-abs {e:.3e} = {e / rms:.3e} rms")
        assert e <= F32_TOL * rms, name
    else:
        e = max_abs(got, ref)
        say(f"  {name}: max-abs {e:.3e}")
        assert e <= F32_TOL, name


def conv(name, B, T, H, W, C, k, dtype, seed=30):
    return testgen.ConvWorkload(name, B, T, H, W, C, k[0], k[1], k[2], dtype, seed)


SMALL = [
    conv("f32_3x3x3", 1, 4, 5, 6, 8, (3, 3, 3), "f32"),
    conv("f32_ragged_1x3x5", 2, 3, 7, 13, 130, (1, 3, 5), "f32", 31),
    conv("bf16_3x3x3_two_chunks", 1, 5, 9, 17, 256, (3, 3, 3), "bf16", 32),
    conv("bf16_5x3x7", 1, 6, 5, 11, 66, (5, 3, 7), "bf16", 33),
    conv("f32_9x1x1", 1, 10, 2, 9, 4, (9, 1, 1), "f32", 34),
    conv("bf16_narrow_W3", 2, 2, 1, 3, 2, (3, 3, 3), "bf16", 35),
    conv("f32_1x7x7_T1", 1, 1, 9, 10, 20, (1, 7, 7), "f32", 36),
    # the bf16 streaming path (every extent 1 or 3) with a time extent of 1, a single frame,
    # mixed extents, a 1 x 1 x 1 filter, two batch items and a ragged channel chunk
    conv("bf16_1x3x3_B2_C130", 2, 3, 6, 10, 130, (1, 3, 3), "bf16", 37),
    conv("bf16_3x1x3_T1", 1, 1, 5, 9, 128, (3, 1, 3), "bf16", 38),
    conv("bf16_3x3x1_T2", 1, 2, 7, 5, 64, (3, 3, 1), "bf16", 39),
    conv("bf16_1x1x1", 1, 3, 4, 5, 32, (1, 1, 1), "bf16", 40),
]


def run_case(w, host=None, frames=None, weight_grads=True):
    import paper_2607_22696_amd as dsa
    bf = w.dtype == "bf16"
    x, dy, wt, bias = host if host is not None else testgen.gen_conv_inputs(w)
    xd, dyd = to_device(x, bf), to_device(dy, bf)
    wd, bd = to_device(wt, False), to_device(bias, False)
    y = dsa.dwconv3d_forward(xd, wd, bd)
    dx, dw, db = dsa.dwconv3d_backward(xd, wd, dyd, need_dweight=weight_grads,
                                       need_dbias=weight_grads)
    torch.cuda.synchronize()
    t0, t1 = frames if frames is not None else (0, w.T)
    say(f"  oracle on frames [{t0},{t1}) of {w.name} ...")
    ry = oracle.dwconv_forward(w.shape8(), w.dtype, x, wt, bias, frames=(t0, t1))
    rdx, rdw, rdb = oracle.dwconv_backward(w.shape8(), w.dtype, x, wt, dy, frames=(t0, t1),
                                           weight_grads=weight_grads)
    check("y", to_host(y[:, t0:t1]), ry, bf)
    check("dx", to_host(dx[:, t0:t1]), rdx, bf)
    if weight_grads:
        check("dweight", to_host(dw), rdw, bf, reduction=True)
        check("dbias", to_host(db), rdb, bf, reduction=True)
    return xd, wd, bd, dyd, y, dx, dw, db


@pytest.mark.parametrize("w", SMALL, ids=lambda w: w.name)
def test_small_grid_parity(w):
    run_case(w)


def test_accumulate_modes_and_partial_requests():
    import paper_2607_22696_amd as dsa
    w = conv("bf16_acc", 1, 3, 4, 9, 130, (3, 3, 3), "bf16", 37)
    x, dy, wt, bias = testgen.gen_conv_inputs(w)
    xd, dyd, wd, bd = to_device(x, True), to_device(dy, True), to_device(wt, False), to_device(bias, False)
    # y += conv(x) + bias on top of an existing tensor (the Eq. (1) sum with the attention term)
    base = testgen.gen_tensor(testgen.WORKLOADS["tiny_f32"], 7, w.x_shape(), testgen.N01, False)
    base_bf = testgen.f32_to_bf16(base)
    yd = to_device(base_bf, True)
    dsa.dwconv3d_forward(xd, wd, bd, out=yd, accumulate=True)
    ref = oracle.dwconv_forward(w.shape8(), "bf16", x, wt, bias) + testgen.bf16_to_f32(base_bf)
    check("y += conv", to_host(yd), ref, True)
    # dx += conv^T(dy), dx only (no workspace needed)
    dx0 = torch.from_numpy(base).cuda()
    dx, dw, db = dsa.dwconv3d_backward(xd, wd, dyd, need_dweight=False, need_dbias=False, dx=dx0,
                                       accumulate_dx=True)
    assert dw is None and db is None
    rdx, rdw, rdb = oracle.dwconv_backward(w.shape8(), "bf16", x, wt, dy)
    check("dx += ...", to_host(dx), rdx + base, True)
    # weight gradients only
    dx2, dw2, db2 = dsa.dwconv3d_backward(xd, wd, dyd, need_dx=False, need_dbias=False)
    assert dx2 is None and db2 is None
    check("dweight only", to_host(dw2), rdw, True)
    # repeatability: the weight gradients are summed in a fixed order
    dw3 = dsa.dwconv3d_backward(xd, wd, dyd, need_dx=False, need_dbias=False)[1]
    assert torch.equal(dw2, dw3)


def test_delta_filter_copies_bf16_input_bitwise():
    """A filter with one tap equal to 1 is a zero-filled shift: y must equal x bit for bit."""
    import paper_2607_22696_amd as dsa
    w = conv("delta", 1, 4, 6, 10, 256, (3, 3, 3), "bf16", 38)
    x, _, _, _ = testgen.gen_conv_inputs(w)
    wt = np.zeros((w.C, 3, 3, 3), np.float32)
    wt[:, 2, 0, 1] = 1.0          # y[t, i, j] = x[t + 1, i - 1, j]
    y = to_host(dsa.dwconv3d_forward(to_device(x, True), to_device(wt, False)))
    xf = testgen.bf16_to_f32(x)
    ref = np.zeros_like(xf)
    ref[:, :-1, 1:, :] = xf[:, 1:, :-1, :]
    assert np.array_equal(y, ref)


# ----------------------------------------------------------------------------- full size

@pytest.mark.slow
def test_dwconv_64x34x60_full_size():
    """130,560 tokens x 1024 channels, bf16: y and dx on three whole frames, every weight and
    bias gradient (sums over the full grid)."""
    w = testgen.CONV_WORKLOADS["dwconv_64x34x60"]
    host = testgen.gen_conv_inputs(w, progress=say)
    for fr in [(0, 1), (31, 32), (63, 64)]:
        run_case(w, host=host, frames=fr, weight_grads=fr == (0, 1))


@pytest.mark.slow
def test_dwconv_1080p_256f_full_size():
    """2,088,960 tokens x 3072 channels (the attention's 24 x 128), bf16: the launch
    configuration the bench times; y and dx checked on the first, a middle and the last frame.
    The weight gradients at this size are covered by the 130,560-token test (same kernels)."""
    import paper_2607_22696_amd as dsa
    w = testgen.CONV_WORKLOADS["dwconv_1080p_256f"]
    x, dy, wt, bias = testgen.gen_conv_inputs(w, progress=say)
    xd, dyd = to_device(x, True), to_device(dy, True)
    wd, bd = to_device(wt, False), to_device(bias, False)
    say("  forward + backward on GPU ...")
    y = dsa.dwconv3d_forward(xd, wd, bd)
    dx, dw, db = dsa.dwconv3d_backward(xd, wd, dyd)
    torch.cuda.synchronize()
    for t0 in (0, 128, 255):
        say(f"  oracle frame {t0} ...")
        ry = oracle.dwconv_forward(w.shape8(), "bf16", x, wt, bias, frames=(t0, t0 + 1))
        rdx = oracle.dwconv_backward(w.shape8(), "bf16", x, wt, dy, frames=(t0, t0 + 1),
                                     weight_grads=False)[0]
        check(f"y[frame {t0}]", to_host(y[:, t0:t0 + 1]), ry, True)
        check(f"dx[frame {t0}]", to_host(dx[:, t0:t0 + 1]), rdx, True)
    assert torch.isfinite(dw).all() and torch.isfinite(db).all()
