"""Pins of the oracle's sub-range entry points against its pinned full-grid ones.

The full-size GPU parity tests compare the kernels with oracle results for parts of a
grid: the forward and the backward of a list of scattered query rows, the backward of the
queries of one (batch, head) and frame range [t0, t1) with t0 > 0 (dq, d_offsets and their
contributions to dK / dV), and the same for the predicted-weights variant.  Each of those
oracle calls decodes a flat row index or a position inside its frame range into
(b, t, i, j, head) by itself.  Here they are checked against the full-grid calls (every
row, frames [0, T)), which tests/test_oracle_pins.py and tests/test_pw_oracle_pins.py pin
against F.grid_sample with autograd (Section 5.3), finite differences and closed forms, so
that a slip in those decodes (a dropped t0, a transposed H and W, a wrong head or batch
stride) fails here.  The same arithmetic runs on both sides, so the bar is 1e-12.
"""
import numpy as np
import pytest

import oracle
import testgen

TOL = 1e-12

# grids with B > 1, T, H, W and heads all different, and a non-cubic kernel, so that any
# mix-up of the axes in a decode lands on another query
CASES = [
    # (name, dtype, B, T, H, W, heads, D, kt, kh, kw, offset std)
    ("f32_k333", "f32", 2, 6, 4, 5, 3, 8, 3, 3, 3, 1.5),
    ("bf16_k135", "bf16", 2, 7, 5, 3, 2, 16, 1, 3, 5, 1.0),
    ("f32_k355_wide", "f32", 1, 5, 6, 7, 2, 8, 3, 5, 5, 3.0),
]


def make_case(seed, dtype, B, T, H, W, M, D, kt, kh, kw, off_std):
    rng = np.random.default_rng(seed)
    P = kt * kh * kw
    q, k, v, dout = (rng.standard_normal((B, T, H, W, M, D)).astype(np.float32) for _ in range(4))
    off = (off_std * rng.standard_normal((B, T, H, W, M, P, 3))).astype(np.float32)
    if dtype == "bf16":
        q, k, v, dout = (testgen.f32_to_bf16(a) for a in (q, k, v, dout))
    return q, k, v, off, dout


def close(got, want, what):
    got, want = np.asarray(got), np.asarray(want)
    assert got.shape == want.shape, (what, got.shape, want.shape)
    if want.size == 0:
        return
    err = float(np.max(np.abs(got - want)))
    assert err <= TOL * max(1.0, float(np.max(np.abs(want)))), (what, err)


def scattered_rows(rng, nrows_total, heads, n=48):
    rows = rng.choice(nrows_total, size=min(n, nrows_total), replace=False)
    edge = np.array([0, heads - 1, nrows_total - heads, nrows_total - 1], dtype=np.int64)
    return np.unique(np.concatenate([rows.astype(np.int64), edge]))


def frame_windows(T):
    """A partition of [0, T) into windows, most of them starting past frame 0, with one
    empty window."""
    cuts = [0, 1, 1, 3, T - 1, T] if T > 4 else [0, 1, 1, T]
    return [(a, b) for a, b in zip(cuts[:-1], cuts[1:])]


@pytest.mark.parametrize("case", CASES, ids=lambda c: c[0])
def test_forward_rows_match_the_full_grid(case):
    name, dtype, B, T, H, W, M, D, kt, kh, kw, sd = case
    shape = (B, T, H, W, M, D, kt, kh, kw)
    q, k, v, off, _ = make_case(1, dtype, B, T, H, W, M, D, kt, kh, kw, sd)
    out, lse = oracle.forward(shape, dtype, q, k, v, off)
    rows = scattered_rows(np.random.default_rng(2), B * T * H * W * M, M)
    o_r, l_r = oracle.forward(shape, dtype, q, k, v, off, rows=rows)
    close(o_r, out[rows], "out")
    close(l_r, lse[rows], "lse")


@pytest.mark.parametrize("case", CASES, ids=lambda c: c[0])
def test_backward_rows_match_the_full_grid(case):
    name, dtype, B, T, H, W, M, D, kt, kh, kw, sd = case
    shape = (B, T, H, W, M, D, kt, kh, kw)
    P = kt * kh * kw
    q, k, v, off, dout = make_case(3, dtype, B, T, H, W, M, D, kt, kh, kw, sd)
    dq, dk, dv, doff = oracle.backward(shape, dtype, q, k, v, off, dout)
    rows = scattered_rows(np.random.default_rng(4), B * T * H * W * M, M)
    dq_r, doff_r = oracle.backward_rows(shape, dtype, q, k, v, off, dout, rows)
    close(dq_r, dq.reshape(-1, D)[rows], "dq")
    close(doff_r, doff.reshape(-1, P, 3)[rows], "doff")


@pytest.mark.parametrize("case", CASES, ids=lambda c: c[0])
def test_backward_frame_slabs_match_the_full_grid(case):
    """dq and d_offsets of a slab [t0, t1) are the full result's frames t0..t1-1; the
    slabs' dK / dV contributions, summed over a partition of [0, T), are the full dK / dV."""
    name, dtype, B, T, H, W, M, D, kt, kh, kw, sd = case
    shape = (B, T, H, W, M, D, kt, kh, kw)
    q, k, v, off, dout = make_case(5, dtype, B, T, H, W, M, D, kt, kh, kw, sd)
    dq, dk, dv, doff = oracle.backward(shape, dtype, q, k, v, off, dout)
    for b in range(B):
        for m in range(M):
            acc_k = np.zeros((T, H, W, D))
            acc_v = np.zeros((T, H, W, D))
            for t0, t1 in frame_windows(T):
                sq, so, _, _ = oracle.backward_slab(shape, dtype, q, k, v, off, dout, b, m, t0, t1,
                                                    dk=acc_k, dv=acc_v)
                close(sq, dq[b, t0:t1, :, :, m], f"dq b{b} m{m} [{t0},{t1})")
                close(so, doff[b, t0:t1, :, :, m], f"doff b{b} m{m} [{t0},{t1})")
            close(acc_k, dk[b, :, :, :, m], f"dk b{b} m{m}")
            close(acc_v, dv[b, :, :, :, m], f"dv b{b} m{m}")


@pytest.mark.parametrize("case", CASES[:2], ids=lambda c: c[0])
def test_pw_rows_and_slabs_match_the_full_grid(case):
    name, dtype, B, T, H, W, M, D, kt, kh, kw, sd = case
    shape = (B, T, H, W, M, D, kt, kh, kw)
    P = kt * kh * kw
    _, _, v, off, dout = make_case(6, dtype, B, T, H, W, M, D, kt, kh, kw, sd)
    logits = (1.5 * np.random.default_rng(7).standard_normal((B, T, H, W, M, P))).astype(np.float32)
    out, lse = oracle.pw_forward(shape, dtype, logits, v, off)
    rows = scattered_rows(np.random.default_rng(8), B * T * H * W * M, M)
    o_r, l_r = oracle.pw_forward(shape, dtype, logits, v, off, rows=rows)
    close(o_r, out[rows], "pw out")
    close(l_r, lse[rows], "pw lse")
    dlog, dv, doff = oracle.pw_backward(shape, dtype, logits, v, off, dout)
    for b in range(B):
        for m in range(M):
            acc_v = np.zeros((T, H, W, D))
            for t0, t1 in frame_windows(T):
                sl, so, _ = oracle.pw_backward_slab(shape, dtype, logits, v, off, dout, b, m, t0,
                                                    t1, dv=acc_v)
                close(sl, dlog[b, t0:t1, :, :, m], f"dlogits b{b} m{m} [{t0},{t1})")
                close(so, doff[b, t0:t1, :, :, m], f"pw doff b{b} m{m} [{t0},{t1})")
            close(acc_v, dv[b, :, :, :, m], f"pw dv b{b} m{m}")


def test_a_planted_t0_slip_is_caught():
    """The check above fails for a slab decoded from frame 0 instead of t0: the frames
    [t0, t1) of the full result differ from frames [0, t1 - t0) (what a dropped t0 would
    return)."""
    dtype, B, T, H, W, M, D, kt, kh, kw, sd = CASES[0][1:]
    shape = (B, T, H, W, M, D, kt, kh, kw)
    q, k, v, off, dout = make_case(9, dtype, B, T, H, W, M, D, kt, kh, kw, sd)
    sq, _, _, _ = oracle.backward_slab(shape, dtype, q, k, v, off, dout, 1, 2, 0, 2)
    sq3, _, _, _ = oracle.backward_slab(shape, dtype, q, k, v, off, dout, 1, 2, 3, 5)
    assert float(np.max(np.abs(sq - sq3))) > 1e-3
