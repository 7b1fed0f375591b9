"""GPU-vs-oracle parity of the HIP path, through the C ABI.

Tolerances
  * fp32 data: max-abs <= 1e-5 on out and lse, and on every gradient.
  * bf16 q/k/v/dout (fp32 accumulate, fp32 gradients): max over elements of
    |g - r| / max(|r|, 1e-2 rms(r)) <= 2e-2 for out, lse and every gradient, against the
    fp64 oracle on the same bf16 inputs.
Small grids are compared element by element (several tiles, ragged tails); the full-size
workloads are compared on sampled query rows (forward, dq, d_offsets) and on frame slabs of
dk/dv whose every contributing query is recomputed by the oracle.
"""
import math

import numpy as np
import pytest

import oracle
import testgen
from tests.util import io_as_f32, max_abs, rel_err, reach_frames, say, shape9, to_device, to_host

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


def run_forward(w, q, k, v, off):
    import paper_2607_22696_amd as dsa
    bf = w.dtype == "bf16"
    qd, kd, vd = (to_device(a, bf) for a in (q, k, v))
    od = to_device(off, False)
    out, lse = dsa.forward(qd, kd, vd, od, kernel=(w.kt, w.kh, w.kw))
    torch.cuda.synchronize()
    return qd, kd, vd, od, out, lse


def run_backward(w, dev, out, lse, dout):
    import paper_2607_22696_amd as dsa
    qd, kd, vd, od = dev
    gd = to_device(dout, w.dtype == "bf16")
    grads = dsa.backward(qd, kd, vd, od, lse, gd, kernel=(w.kt, w.kh, w.kw))
    torch.cuda.synchronize()
    return grads


def check(name, got, ref, bf16):
    if bf16:
        e = rel_err(got, ref)
        say(f"  {name}: rel {e:.3e} (max-abs {max_abs(got, ref):.3e})")
        assert e <= BF16_TOL, (name, e)
    else:
        e = max_abs(got, ref)
        say(f"  {name}: max-abs {e:.3e}")
        assert e <= F32_TOL, (name, e)


def full_case(w, seed_override=None, off_override=None, check_bwd=True):
    """Element-by-element forward (and backward) parity on a small workload."""
    say(f"case {w.name}: grid {w.T}x{w.H}x{w.W} B={w.B} heads={w.heads} D={w.head_dim} "
        f"kernel {w.kt}x{w.kh}x{w.kw} {w.dtype}")
    q, k, v, off, dout = testgen.gen_inputs(w)
    if off_override is not None:
        off = off_override(off)
    if dout is None:
        dout = testgen.gen_tensor(w, testgen.TID_DOUT, w.qkv_shape(), w.dout, True)
    bf = w.dtype == "bf16"
    qd, kd, vd, od, out, lse = run_forward(w, q, k, v, off)
    ref_out, ref_lse = oracle.forward(shape9(w), w.dtype, q, k, v, off)
    check("out", to_host(out).reshape(-1, w.head_dim), ref_out, bf)
    check("lse", to_host(lse).reshape(-1), ref_lse, bf)
    if not check_bwd:
        return
    dq, dk, dv, doff = run_backward(w, (qd, kd, vd, od), out, lse, dout)
    rq, rk, rv, roff = oracle.backward(shape9(w), w.dtype, q, k, v, off, dout)
    check("dq", to_host(dq), rq, bf)
    check("dk", to_host(dk), rk, bf)
    check("dv", to_host(dv), rv, bf)
    check("doff", to_host(doff), roff, bf)


# ----------------------------------------------------------------------------- small grids

def small(name, **kw):
    base = testgen.WORKLOADS["tiny_f32"]
    return base.with_grid(name=name, **kw)


SMALL_CASES = [
    # tiny fp32 workload as specified (256 tokens, 2 heads x 32, 3x3x3, offsets N(0, 0.5))
    testgen.WORKLOADS["tiny_f32"],
    small("ragged_f32_d64", T=5, H=7, W=9, heads=3, head_dim=64, seed=10),
    small("ragged_f32_d128", T=3, H=5, W=11, heads=2, head_dim=128, seed=11),
    small("ragged_bf16_d32", T=5, H=7, W=9, heads=3, head_dim=32, dtype="bf16", seed=12),
    small("ragged_bf16_d64", T=6, H=9, W=10, heads=4, head_dim=64, dtype="bf16", seed=13,
          offsets=testgen.Dist(testgen.UNIFORM, -2.0, 2.0)),
    small("ragged_bf16_d128", T=4, H=6, W=13, heads=3, head_dim=128, dtype="bf16", seed=14,
          offsets=testgen.Dist(testgen.NORMAL, 0.0, 1.0, -3.0, 3.0)),
    small("batch2_bf16", B=2, T=3, H=5, W=6, heads=2, head_dim=64, dtype="bf16", seed=15),
    small("k355_bf16", T=5, H=8, W=9, heads=2, head_dim=128, kt=3, kh=5, kw=5, dtype="bf16",
          seed=16, offsets=testgen.Dist(testgen.UNIFORM, -8.0, 8.0)),
    small("k377_bf16", T=4, H=9, W=9, heads=2, head_dim=64, kt=3, kh=7, kw=7, dtype="bf16",
          seed=17),
    small("k377_f32", T=3, H=8, W=8, heads=1, head_dim=32, kt=3, kh=7, kw=7, seed=18),
    small("k111_f32", T=3, H=4, W=5, heads=2, head_dim=32, kt=1, kh=1, kw=1, seed=19),
    small("k135_f32", T=2, H=6, W=7, heads=2, head_dim=64, kt=1, kh=3, kw=5, seed=20),
    small("grid_1x1x1", T=1, H=1, W=1, heads=2, head_dim=32, seed=21),
    small("t1_bf16", T=1, H=9, W=17, heads=2, head_dim=64, dtype="bf16", seed=22),
    small("w1_f32", T=6, H=7, W=1, heads=2, head_dim=32, seed=23),
    # bf16 with degenerate and mixed-size kernels (1 to 315 points) against the dK/dV
    # matrix-core gather's 4 x 2 x 2 voxel blocks and 32-entry batches
    small("k111_bf16_d128", T=3, H=4, W=5, heads=2, head_dim=128, kt=1, kh=1, kw=1,
          dtype="bf16", seed=26),
    small("k135_bf16_d64", T=2, H=6, W=7, heads=3, head_dim=64, kt=1, kh=3, kw=5, dtype="bf16",
          seed=27),
    small("k377_bf16_d128", T=3, H=7, W=6, heads=2, head_dim=128, kt=3, kh=7, kw=7,
          dtype="bf16", seed=28, offsets=testgen.Dist(testgen.UNIFORM, -3.0, 3.0)),
    small("k579_bf16_d64", T=5, H=7, W=9, heads=2, head_dim=64, kt=5, kh=7, kw=9, dtype="bf16",
          seed=29),
    # the K pass holds a row's (alpha_p, A_p) in registers up to 5 chunks of L = D s / 16
    # points and goes through the records beyond: 5 chunks of 8 with a ragged last one, 6 of 8,
    # 6 of 16 (the chunk after 3x5x5's five), 4 of 4
    small("k157_bf16_d64", T=4, H=7, W=9, heads=2, head_dim=64, kt=1, kh=5, kw=7, dtype="bf16",
          seed=53),
    small("k335_bf16_d64", T=4, H=6, W=7, heads=2, head_dim=64, kt=3, kh=3, kw=5, dtype="bf16",
          seed=54),
    small("k339_bf16_d128", T=4, H=6, W=11, heads=2, head_dim=128, kt=3, kh=3, kw=9,
          dtype="bf16", seed=55, offsets=testgen.Dist(testgen.UNIFORM, -3.0, 3.0)),
    small("k135_bf16_d32", T=3, H=6, W=7, heads=2, head_dim=32, kt=1, kh=3, kw=5, dtype="bf16",
          seed=56),
    # fp32 rows take twice the lanes: 3 chunks of 32 (ragged), 5 of 16, 6 of 8
    small("k355_f32_d128", T=3, H=5, W=6, heads=1, head_dim=128, kt=3, kh=5, kw=5, seed=57,
          offsets=testgen.Dist(testgen.UNIFORM, -3.0, 3.0)),
    small("k355_f32_d64", T=3, H=6, W=7, heads=2, head_dim=64, kt=3, kh=5, kw=5, seed=58),
    small("k335_f32_d32", T=4, H=6, W=7, heads=2, head_dim=32, kt=3, kh=3, kw=5, seed=59),
    # grids thinner than one 4 x 2 x 2 gather block (a block with 2-4 cell columns, no second
    # row or plane)
    small("thin_bf16_d64", T=3, H=1, W=3, heads=2, head_dim=64, dtype="bf16", seed=50),
    small("line_bf16_d32", T=2, H=2, W=1, heads=2, head_dim=32, dtype="bf16", seed=51),
    small("grid_1x1x1_bf16_d128", T=1, H=1, W=1, heads=2, head_dim=128, dtype="bf16", seed=52),
    # 32 heads x 512-byte fp32 rows: a token's rows exceed the buffer record stride limit, so
    # every corner takes the global-load path
    small("wide_token_f32", T=2, H=4, W=5, heads=32, head_dim=128, seed=25,
          offsets=testgen.Dist(testgen.UNIFORM, -2.0, 2.0)),
]


@pytest.mark.parametrize("w", SMALL_CASES, ids=lambda w: w.name)
def test_small_grid_parity(w):
    full_case(w)


def test_medium_bf16_forward_full():
    """16,384 tokens, 8 heads x 64, every output element."""
    full_case(testgen.WORKLOADS["medium_bf16"], check_bwd=False)


def test_zero_offsets_fixed_window():
    """Zero offsets (fixed local window, Section 9.1)."""
    w = small("zero_off_bf16", T=5, H=7, W=8, heads=2, head_dim=64, dtype="bf16", seed=24)
    full_case(w, off_override=lambda o: np.zeros_like(o))


def test_single_point_integer_offsets_copy_rows_bitwise():
    """1x1x1 kernel with integer offsets: alpha = 1 and one corner of weight 1, so out must be
    exactly the shifted V row (zero outside the grid), in both dtypes."""
    for dtype, seed in (("f32", 30), ("bf16", 31)):
        w = small(f"int_copy_{dtype}", T=4, H=5, W=6, heads=2, head_dim=64, kt=1, kh=1, kw=1,
                  dtype=dtype, seed=seed)
        q, k, v, off, _ = testgen.gen_inputs(w)
        rng = np.random.default_rng(seed)
        off = rng.integers(-2, 3, off.shape).astype(np.float32)
        _, _, _, _, out, _ = run_forward(w, q, k, v, off)
        got = to_host(out)
        vf = io_as_f32(v)
        want = np.zeros_like(got)
        for t in range(w.T):
            for i in range(w.H):
                for j in range(w.W):
                    for m in range(w.heads):
                        dx, dy, dz = off[0, t, i, j, m, 0].astype(int)
                        x, y, z = j + dx, i + dy, t + dz
                        if 0 <= x < w.W and 0 <= y < w.H and 0 <= z < w.T:
                            want[0, t, i, j, m] = vf[0, z, y, x, m]
        bad = np.argwhere(got != want)
        assert bad.size == 0, (dtype, len(bad), bad[:5].tolist(),
                               float(np.max(np.abs(got - want))), got[tuple(bad[0])],
                               want[tuple(bad[0])])


@pytest.mark.parametrize("dtype,dim", [("f32", 32), ("bf16", 64), ("bf16", 128)])
def test_non_finite_and_huge_offsets_are_safe(dtype, dim):
    """Offsets of +-1e30, +-inf and NaN put every corner outside the grid: no fault, and the
    result is the all-outside one (logit 0 everywhere: out = 0, lse = ln P)."""
    w = small(f"huge_offsets_{dtype}_{dim}", T=3, H=4, W=5, heads=2, head_dim=dim, dtype=dtype,
              seed=32)
    q, k, v, off, _ = testgen.gen_inputs(w)
    vals = np.array([1e30, -1e30, np.inf, -np.inf, np.nan], dtype=np.float32)
    off = vals[np.arange(off.size) % len(vals)].reshape(off.shape)
    _, _, _, _, out, lse = run_forward(w, q, k, v, off)
    assert np.array_equal(to_host(out), np.zeros(q.shape, np.float32))
    np.testing.assert_allclose(to_host(lse), math.log(w.P), rtol=0, atol=1e-6)
    ref_out, ref_lse = oracle.forward(shape9(w), w.dtype, q, k, v, off)
    assert np.all(ref_out == 0.0)


def test_backward_repeatability():
    """dq and d_offsets are query-owned (bitwise repeatable); dk/dv sum each bin in the order
    its points claimed their slots, so repeated runs may differ only by summation order."""
    w = small("repeat_bf16", T=4, H=8, W=8, heads=2, head_dim=64, dtype="bf16", seed=33,
              offsets=testgen.Dist(testgen.UNIFORM, -1.0, 1.0))
    q, k, v, off, _ = testgen.gen_inputs(w)
    dout = testgen.gen_tensor(w, testgen.TID_DOUT, w.qkv_shape(), w.dout, True)
    qd, kd, vd, od, out, lse = run_forward(w, q, k, v, off)
    runs = [[to_host(t) for t in run_backward(w, (qd, kd, vd, od), out, lse, dout)]
            for _ in range(4)]
    for r in runs[1:]:
        assert np.array_equal(r[0], runs[0][0])  # dq is query-owned: bitwise
        assert np.array_equal(r[3], runs[0][3])  # d_offsets too
        for a in (1, 2):
            assert rel_err(r[a], runs[0][a]) < 1e-4


def test_backward_timed_matches_untimed_and_marks_every_phase():
    import paper_2607_22696_amd as dsa
    w = small("timed_bf16", T=5, H=9, W=11, heads=2, head_dim=64, dtype="bf16", seed=34,
              offsets=testgen.Dist(testgen.UNIFORM, -2.0, 2.0))
    q, k, v, off, _ = testgen.gen_inputs(w)
    dout = testgen.gen_tensor(w, testgen.TID_DOUT, w.qkv_shape(), w.dout, True)
    qd, kd, vd, od, out, lse = run_forward(w, q, k, v, off)
    gd = to_device(dout, True)
    kern = (w.kt, w.kh, w.kw)
    plain = [to_host(t) for t in dsa.backward(qd, kd, vd, od, lse, gd, kernel=kern)]
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(dsa.DSA3D_BACKWARD_PHASES + 1)]
    for e in evs:  # creates the underlying HIP events
        e.record()
    timed = dsa.backward(qd, kd, vd, od, lse, gd, kernel=kern, phase_events=evs)
    torch.cuda.synchronize()
    timed = [to_host(t) for t in timed]
    assert np.array_equal(timed[0], plain[0]) and np.array_equal(timed[3], plain[3])
    for a in (1, 2):
        assert rel_err(timed[a], plain[a]) < 1e-4
    ms = [evs[i].elapsed_time(evs[i + 1]) for i in range(dsa.DSA3D_BACKWARD_PHASES)]
    say(f"  phase ms {ms}")
    assert all(t > 0.0 for t in ms)


# ----------------------------------------------------------------------------- full size

def sampled_rows(w, n, rng):
    rows = rng.choice(w.queries, size=n, replace=False)
    # always include the first and last token of the grid for every head
    extra = [m for m in range(w.heads)] + [(w.N - 1) * w.heads + m for m in range(w.heads)]
    return np.unique(np.concatenate([rows, np.array(extra, dtype=np.int64)]))


def frame_rows(w, frames):
    """Every (token, head) row of the given frames (all heads)."""
    HW = w.H * w.W
    per = HW * w.heads
    return np.concatenate([np.arange(f * per, (f + 1) * per, dtype=np.int64) for f in frames])


def full_size_forward(w, nsamp, frames=()):
    """The whole grid on the GPU; the oracle on `nsamp` random rows plus every row of
    `frames`."""
    say(f"full-size {w.name}: generating {w.queries} rows ...")
    q, k, v, off, dout = testgen.gen_inputs(w, progress=say)
    say("  forward on GPU ...")
    qd, kd, vd, od, out, lse = run_forward(w, q, k, v, off)
    rng = np.random.default_rng(w.seed)
    rows = sampled_rows(w, nsamp, rng)
    if len(frames):
        rows = np.unique(np.concatenate([rows, frame_rows(w, frames)]))
    say(f"  oracle on {rows.size} rows ({nsamp} sampled, frames {list(frames)}) ...")
    ref_out, ref_lse = oracle.forward(shape9(w), w.dtype, q, k, v, off, rows=rows)
    sel = torch.from_numpy(rows).cuda()
    out_h = to_host(out.view(-1, w.head_dim)[sel])
    lse_h = to_host(lse.view(-1)[sel])
    check("out", out_h, ref_out, True)
    check("lse", lse_h, ref_lse, True)
    return (q, k, v, off, dout), (qd, kd, vd, od), out, lse, rows


def full_size_backward(w, host, dev, out, lse, rows, slab_frames, slab_heads):
    q, k, v, off, dout = host
    say("  backward on GPU ...")
    dq, dk, dv, doff = run_backward(w, dev, out, lse, dout)
    B, T, H, W, M, D = w.qkv_shape()
    P = w.P
    # dq and d_offsets: query-owned, compare on the sampled rows
    sel = torch.from_numpy(rows).cuda()
    dq_h = to_host(dq.view(-1, D)[sel])
    doff_h = to_host(doff.view(-1, P * 3)[sel])
    R = reach_frames(w, float(np.max(np.abs(off[..., 2])))) if slab_frames else 0
    for m in slab_heads:
        for f in slab_frames:
            t0, t1 = max(0, f - R), min(T, f + 1 + R)
            say(f"  oracle backward head {m}, frames [{t0},{t1}) for dk/dv at frame {f} ...")
            rq, roff, rk, rv = oracle.backward_slab(shape9(w), w.dtype, q, k, v, off, dout, 0, m,
                                                    t0, t1)
            check(f"dk[frame {f}, head {m}]", to_host(dk[0, f, :, :, m]), rk[f], True)
            check(f"dv[frame {f}, head {m}]", to_host(dv[0, f, :, :, m]), rv[f], True)
            # dq/doff of the slab's queries come for free
            check(f"dq[frames {t0}-{t1}, head {m}]", to_host(dq[0, t0:t1, :, :, m]), rq, True)
            check(f"doff[frames {t0}-{t1}, head {m}]", to_host(doff[0, t0:t1, :, :, m]), roff, True)
    # sampled rows, all heads
    say(f"  oracle backward on {rows.size} sampled rows ...")
    rq, roff = oracle.backward_rows(shape9(w), w.dtype, q, k, v, off, dout, rows)
    check("dq[sampled rows]", dq_h, rq, True)
    check("doff[sampled rows]", doff_h, roff.reshape(-1, P * 3), True)


@pytest.mark.slow
@pytest.mark.timeout(900)
def test_full_scale_1080p_256f_forward_sampled():
    """2,088,960 tokens x 24 heads x 128, 3x3x3 kernel: the full grid runs on the GPU in the
    bench's launch configuration; every row of frames 0, 1, 128 and 255 (all 24 heads: the
    first, last and an interior frame, and one whose corners reach across frame 0) plus 65,536
    random rows are checked."""
    full_size_forward(testgen.WORKLOADS["full_1080p_256f"], 65536, frames=(0, 1, 128, 255))


@pytest.mark.slow
@pytest.mark.timeout(900)
def test_paper_3x7x7_1080p_256f_forward_sampled():
    """The paper's 3x7x7 kernel (147 points) on the 256-frame 1080p grid, the forward the
    bench profiles at that size: 4,096 random rows plus every row of frames 0 and 255."""
    full_size_forward(testgen.WORKLOADS["paper_3x7x7_1080p_256f"], 4096, frames=(0, 255))


@pytest.mark.slow
def test_window_fallback_large_temporal_offsets():
    """K and V of 5 GB each: the buffer window covers 85 of the 100 frames, and offsets up to
    +-60 tokens put many in-grid corners outside it, where the global-load path takes over."""
    base = testgen.WORKLOADS["full_1080p_256f"]
    w = base.with_grid(name="window_fallback", T=100, offsets=testgen.Dist(testgen.UNIFORM, -60.0, 60.0),
                       seed=40, backward=True)
    host, dev, out, lse, rows = full_size_forward(w, 4096)
    q, k, v, off, dout = host
    if dout is None:
        dout = testgen.gen_tensor(w, testgen.TID_DOUT, w.qkv_shape(), w.dout, True)
    full_size_backward(w, (q, k, v, off, dout), dev, out, lse, rows, slab_frames=[], slab_heads=[])


@pytest.mark.slow
def test_fwdbwd_64x34x60_full_size():
    w = testgen.WORKLOADS["fwdbwd_64x34x60"]
    host, dev, out, lse, rows = full_size_forward(w, 8192)
    full_size_backward(w, host, dev, out, lse, rows, slab_frames=[0, 31, 63], slab_heads=[0, 9])


@pytest.mark.slow
@pytest.mark.timeout(900)
def test_wide_64x68x120_p75_full_size():
    """The bench's default workload: 4,096 sampled rows plus all of frame 63 (forward, dq,
    d_offsets) and dK / dV frame slabs of three heads."""
    w = testgen.WORKLOADS["wide_64x68x120_p75"]
    host, dev, out, lse, rows = full_size_forward(w, 4096, frames=(63,))
    full_size_backward(w, host, dev, out, lse, rows, slab_frames=[0, 37],
                       slab_heads=[0, 5, 23])


@pytest.mark.slow
def test_paper_3x7x7_64x68x120_full_size():
    """The paper's 3x7x7 kernel (147 points) on the 64-frame 1080p grid, forward and
    backward at full size; sampled rows plus dK/dV frame slabs are checked."""
    w = testgen.WORKLOADS["paper_3x7x7_64x68x120"]
    host, dev, out, lse, rows = full_size_forward(w, 2048)
    full_size_backward(w, host, dev, out, lse, rows, slab_frames=[0, 40], slab_heads=[11])
