"""GPU-vs-oracle parity of the fixed / shifted window attention (the Swin-DiT baseline,
Section 6.2: 3 x 16 x 16 windows, shifted windows), through the C ABI.

bf16 q, k, v, dout with fp32 accumulation, against the fp64 oracle on the same bf16 inputs:
max over elements of |g - r| / max(|r|, 1e-2 rms(r)) <= 2e-2 for out, lse, dq, dk and dv.
Small grids are compared element by element (several query and key tiles per box, ragged
boxes at every border, padding windows, windows larger than 768 tokens); the full-size grids
on whole frames (out, lse) and on whole temporal regions (dq, dk, dv).
"""
import numpy as np
import pytest

import oracle
import testgen
from tests.util import max_abs, rel_err, say, to_device, to_host

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

BF16_TOL = 2e-2


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2607_22696_amd as dsa
    dsa.load()
    yield


def check(name, got, ref):
    e = rel_err(got, ref)
    say(f"  {name}: rel {e:.3e} (max-abs {max_abs(got, ref):.3e})")
    assert e <= BF16_TOL, name


def win(name, B, T, H, W, heads, D, window, shift, seed):
    return testgen.WinWorkload(name, B, T, H, W, heads, D, window, shift, seed)


def run(w, host, backward=True, residual=True):
    import paper_2607_22696_amd as dsa
    q, k, v, dout = (to_device(a, True) for a in host)
    kw = dict(window=w.window, shift=w.shift)
    out, lse, res = dsa.win_forward(q, k, v, need_residual=residual, **kw)
    grads = dsa.win_backward(q, k, v, out, res, lse, dout, **kw) if backward else None
    torch.cuda.synchronize()
    return out, lse, grads


SMALL = [
    # shifted Swin-DiT windows: 768-token boxes (6 query tiles, 12 key tiles) and ragged ones
    win("d64_3x16x16_shifted", 1, 6, 20, 24, 2, 64, (3, 16, 16), (1, 8, 8), 50),
    # plain windows with padding on every axis, two batch items, head_dim 128
    win("d128_3x16x16_padded", 2, 4, 18, 20, 2, 128, (3, 16, 16), (0, 0, 0), 51),
    # small windows, odd shifts, three heads
    win("d64_2x3x5_shift_1x1x2", 1, 5, 7, 11, 3, 64, (2, 3, 5), (1, 1, 2), 52),
    # 1024-token windows (boxes beyond the 768 of the paper's windows)
    win("d128_4x8x32_shifted", 1, 8, 10, 40, 1, 128, (4, 8, 32), (2, 4, 16), 53),
    # window larger than the grid on every axis: each box is a piece of the grid
    win("d64_window_exceeds_grid", 1, 2, 5, 7, 2, 64, (3, 16, 16), (1, 8, 8), 54),
]


@pytest.mark.parametrize("w", SMALL, ids=lambda w: w.name)
def test_small_grid_parity(w):
    host = testgen.gen_win_inputs(w)
    out, lse, (dq, dk, dv) = run(w, host)
    q, k, v, dout = host
    ro, rl = oracle.win_forward(w.shape12(), "bf16", q, k, v)
    rdq, rdk, rdv = oracle.win_backward(w.shape12(), "bf16", q, k, v, dout)
    check("out", to_host(out), ro)
    check("lse", to_host(lse), rl)
    check("dq", to_host(dq), rdq)
    check("dk", to_host(dk), rdk)
    check("dv", to_host(dv), rdv)


def test_unit_window_copies_v_bitwise():
    """1 x 1 x 1 windows: every token attends only to itself, so out is v bit for bit; the
    gradients (dv = dout, dq = dk = 0) within the tolerance (alpha is recomputed from lse)."""
    w = win("unit", 1, 3, 5, 6, 2, 64, (1, 1, 1), (0, 0, 0), 55)
    host = testgen.gen_win_inputs(w)
    out, lse, (dq, dk, dv) = run(w, host)
    q, k, v, dout = host
    assert np.array_equal(to_host(out), testgen.bf16_to_f32(v))
    check("dv", to_host(dv), testgen.bf16_to_f32(dout))
    check("dq", to_host(dq), np.zeros(dq.shape))
    check("dk", to_host(dk), np.zeros(dk.shape))


def test_backward_without_residual():
    """Without out_res, Delta = <dout, out> takes the bf16 rounding of out (|O - out| <= 2^-9 |O|
    elementwise), so dq and dk may move by at most scale |Delta error| max|k| and
    scale |Delta error| max|q| per row; dv does not depend on Delta and is bitwise that of the
    call with the residual."""
    import paper_2607_22696_amd as dsa
    w = win("nores", 1, 6, 20, 24, 2, 64, (3, 16, 16), (1, 8, 8), 57)
    host = testgen.gen_win_inputs(w)
    q, k, v, dout = host
    qd, kd, vd, gd = (to_device(a, True) for a in host)
    kw = dict(window=w.window, shift=w.shift)
    out, lse, res = dsa.win_forward(qd, kd, vd, **kw)
    g_res = dsa.win_backward(qd, kd, vd, out, res, lse, gd, **kw)
    g_nor = dsa.win_backward(qd, kd, vd, out, None, lse, gd, **kw)
    torch.cuda.synchronize()
    assert torch.equal(g_res[2], g_nor[2])
    ro, _ = oracle.win_forward(w.shape12(), "bf16", q, k, v)
    rdq, rdk, _ = oracle.win_backward(w.shape12(), "bf16", q, k, v, dout)
    g64 = testgen.bf16_to_f32(dout).astype(np.float64)
    ddelta = 2.0 ** -9 * np.sum(np.abs(g64) * np.abs(ro), axis=-1, keepdims=True)
    scale = 1.0 / np.sqrt(w.head_dim)
    kmax = np.abs(testgen.bf16_to_f32(k)).max()
    qmax = np.abs(testgen.bf16_to_f32(q)).max()
    # dq of a query moves by at most scale |dDelta_query| max|k|; dk of a key by
    # scale max|dDelta| max|q| times the key's alpha summed over its box's queries (a softmax
    # column sum, near 1 for N(0, 1) logits; 32 bounds it with a wide margin)
    slack = 1e-4 * np.sqrt(np.mean(rdq ** 2))
    assert np.all(np.abs(to_host(g_nor[0]) - rdq) <= scale * ddelta * kmax + slack)
    assert np.all(np.abs(to_host(g_nor[1]) - rdk) <= 32 * scale * ddelta.max() * qmax + slack)


def test_repeatable_and_scale_argument():
    import paper_2607_22696_amd as dsa
    w = win("rep", 1, 3, 16, 16, 2, 128, (3, 16, 16), (0, 0, 0), 56)
    host = testgen.gen_win_inputs(w)
    q, k, v, dout = (to_device(a, True) for a in host)
    kw = dict(window=w.window, shift=w.shift, scale=0.05)
    out, lse, res = dsa.win_forward(q, k, v, **kw)
    g1 = dsa.win_backward(q, k, v, out, res, lse, dout, **kw)
    g2 = dsa.win_backward(q, k, v, out, res, lse, dout, **kw)
    torch.cuda.synchronize()
    for a, b in zip(g1, g2):
        assert torch.equal(a, b)
    ro, rl = oracle.win_forward(w.shape12(), "bf16", *host[:3], scale=0.05)
    check("out (scale 0.05)", to_host(out), ro)
    rg = oracle.win_backward(w.shape12(), "bf16", *host, scale=0.05)
    for name, a, b in zip(("dq", "dk", "dv"), g1, rg):
        check(f"{name} (scale 0.05)", to_host(a), b)


# ----------------------------------------------------------------------------- full size

@pytest.mark.slow
def test_swin_64x34x60_full_size():
    """130,560 tokens x 16 heads x 64, shifted 3 x 16 x 16 windows: out and lse on three whole
    frames, dq, dk, dv on two whole temporal regions (frames [1, 4) and [61, 64))."""
    w = testgen.WIN_WORKLOADS["swin_64x34x60"]
    host = testgen.gen_win_inputs(w, progress=say)
    out, lse, (dq, dk, dv) = run(w, host)
    q, k, v, dout = host
    for f in (0, 31, 63):
        say(f"  oracle forward, frame {f} ...")
        ro, rl = oracle.win_forward(w.shape12(), "bf16", q, k, v, frames=(f, f + 1))
        check(f"out[frame {f}]", to_host(out[:, f:f + 1]), ro)
        check(f"lse[frame {f}]", to_host(lse[:, f:f + 1]), rl)
    for t0, t1 in ((1, 4), (61, 64)):
        say(f"  oracle backward, frames [{t0},{t1}) ...")
        rdq, rdk, rdv = oracle.win_backward(w.shape12(), "bf16", q, k, v, dout, frames=(t0, t1))
        check(f"dq[{t0}:{t1}]", to_host(dq[:, t0:t1]), rdq)
        check(f"dk[{t0}:{t1}]", to_host(dk[:, t0:t1]), rdk)
        check(f"dv[{t0}:{t1}]", to_host(dv[:, t0:t1]), rdv)


# 51 GB of bf16 inputs are generated on the host and two 3-frame backward regions go
# through the fp64 oracle: about two minutes of host work besides the GPU run.
@pytest.mark.slow
@pytest.mark.timeout(420)
def test_swin_1080p_256f_full_size():
    """2,088,960 tokens x 24 heads x 128, shifted 3 x 16 x 16 windows (Swin-DiT's attention on
    256 frames of 1080p): the launch configuration the bench times; out and lse on the first, a
    middle and the last frame, dq, dk, dv on the first and the last full temporal regions."""
    w = testgen.WIN_WORKLOADS["swin_1080p_256f"]
    host = testgen.gen_win_inputs(w, progress=say)
    say("  forward + backward on GPU ...")
    out, lse, (dq, dk, dv) = run(w, host)
    q, k, v, dout = host
    for f in (0, 128, 255):
        say(f"  oracle forward, frame {f} ...")
        ro, rl = oracle.win_forward(w.shape12(), "bf16", q, k, v, frames=(f, f + 1))
        check(f"out[frame {f}]", to_host(out[:, f:f + 1]), ro)
        check(f"lse[frame {f}]", to_host(lse[:, f:f + 1]), rl)
    for t0, t1 in ((1, 4), (253, 256)):
        say(f"  oracle backward, frames [{t0},{t1}) ...")
        rdq, rdk, rdv = oracle.win_backward(w.shape12(), "bf16", q, k, v, dout, frames=(t0, t1))
        check(f"dq[{t0}:{t1}]", to_host(dq[:, t0:t1]), rdq)
        check(f"dk[{t0}:{t1}]", to_host(dk[:, t0:t1]), rdk)
        check(f"dv[{t0}:{t1}]", to_host(dv[:, t0:t1]), rdv)
