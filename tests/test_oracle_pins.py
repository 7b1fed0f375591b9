"""Pins of the CPU oracle against what the paper and the mathematics fix.

None of these re-types the oracle's own formula: each compares it with an
independent route to the same quantity.

  * hand-derived worked examples (closed forms, tests/golden/)
  * zero offsets reduce the operator to fixed-window local attention
    (Section 9.1), checked against an integer-gather implementation that has
    no interpolation code
  * integer offsets give exact gathers (every trilinear weight is 0 or 1)
  * brute-force trilinear interpolation as a sum over the whole grid of
    hat-function weights (tiny grids)
  * the paper's own implementation route, F.grid_sample in 5D with zero
    padding (Section 5.3), with torch autograd giving every gradient
  * central finite differences of the forward for every gradient
  * invariants: softmax normalisation, head/batch independence, linearity in
    V, point-order permutation, logit-scale folding, translation
    equivariance, no causal mask (Section 5.3)
"""
import json
import math
import os

import numpy as np
import pytest
import torch

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "worked_examples.json")


# ----------------------------------------------------------------------------- helpers

def rand_case(rng, B, T, H, W, M, D, kt, kh, kw, off_std=1.0, off_unif=None, grid_step=None):
    P = kt * kh * kw
    q = rng.standard_normal((B, T, H, W, M, D)).astype(np.float32)
    k = rng.standard_normal((B, T, H, W, M, D)).astype(np.float32)
    v = rng.standard_normal((B, T, H, W, M, D)).astype(np.float32)
    if off_unif is not None:
        off = rng.uniform(-off_unif, off_unif, (B, T, H, W, M, P, 3)).astype(np.float32)
    else:
        off = (off_std * rng.standard_normal((B, T, H, W, M, P, 3))).astype(np.float32)
    if grid_step is not None:  # values on a dyadic grid so that +-h steps are exact in fp32
        q, k, v, off = (np.round(a / grid_step) * grid_step for a in (q, k, v, off))
        q, k, v, off = (a.astype(np.float32) for a in (q, k, v, off))
    return q, k, v, off


def shape_of(q, kt, kh, kw):
    return tuple(q.shape) + (kt, kh, kw)


def base_grid(kt, kh, kw):
    """Query-centred kernel cells, enumerated row-major over (it, ih, iw)."""
    g = []
    for it in range(kt):
        for ih in range(kh):
            for iw in range(kw):
                g.append((iw - kw // 2, ih - kh // 2, it - kt // 2))
    return np.array(g, dtype=np.int64)  # [P, 3] as (x, y, z)


def positions_f32(T, H, W, M, off, kt, kh, kw):
    """pos = (float)(token + base cell) + offset, in fp32 (one rounding), as float64."""
    g = base_grid(kt, kh, kw)
    tt, ii, jj = np.meshgrid(np.arange(T), np.arange(H), np.arange(W), indexing="ij")
    base = np.stack([jj, ii, tt], -1)[None, :, :, :, None, None, :] + g[None, None, None, None, None]
    pos = base.astype(np.float32) + off
    return pos.astype(np.float64)


def slide_attention_integer(q, k, v, ioff, kt, kh, kw, scale):
    """Local attention with integer sample positions: plain gathers, zero rows outside.

    Written without any interpolation: row (t+dz, i+dy, j+dx) of K and V is
    read directly, or taken as zero when it falls outside the grid."""
    B, T, H, W, M, D = q.shape
    g = base_grid(kt, kh, kw)
    P = len(g)
    q64, k64, v64 = (a.astype(np.float64) for a in (q, k, v))
    bb, tt, ii, jj, mm = np.meshgrid(np.arange(B), np.arange(T), np.arange(H), np.arange(W),
                                     np.arange(M), indexing="ij")
    logits = np.empty((B, T, H, W, M, P))
    vals = np.empty((B, T, H, W, M, P, D))
    for p in range(P):
        x = jj + g[p, 0] + ioff[..., p, 0]
        y = ii + g[p, 1] + ioff[..., p, 1]
        z = tt + g[p, 2] + ioff[..., p, 2]
        inside = (x >= 0) & (x < W) & (y >= 0) & (y < H) & (z >= 0) & (z < T)
        xc, yc, zc = np.clip(x, 0, W - 1), np.clip(y, 0, H - 1), np.clip(z, 0, T - 1)
        krow = k64[bb, zc, yc, xc, mm] * inside[..., None]
        vrow = v64[bb, zc, yc, xc, mm] * inside[..., None]
        logits[..., p] = scale * np.sum(q64 * krow, -1)
        vals[..., p, :] = vrow
    mx = logits.max(-1, keepdims=True)
    e = np.exp(logits - mx)
    alpha = e / e.sum(-1, keepdims=True)
    out = np.einsum("...p,...pd->...d", alpha, vals)
    lse = (mx[..., 0] + np.log(e.sum(-1)))
    return out, lse


def hat_sample(F, pos):
    """Trilinear sample as sum over all grid points of prod max(0, 1 - |pos - x|); F is [T,H,W,D]."""
    T, H, W, D = F.shape
    wx = np.maximum(0.0, 1.0 - np.abs(pos[0] - np.arange(W)))
    wy = np.maximum(0.0, 1.0 - np.abs(pos[1] - np.arange(H)))
    wz = np.maximum(0.0, 1.0 - np.abs(pos[2] - np.arange(T)))
    return np.einsum("t,h,w,thwd->d", wz, wy, wx, F)


def torch_reference(q, k, v, off, kt, kh, kw, scale, dout=None):
    """3D-DSA through torch.nn.functional.grid_sample (5D, bilinear = trilinear, zero padding,
    align_corners=False), the route Section 5.3 describes; fp64 on the CPU, autograd for the
    gradients.  Positions carry the fp32 rounding of the operator's definition."""
    B, T, H, W, M, D = q.shape
    P = kt * kh * kw
    qt = torch.tensor(q, dtype=torch.float64, requires_grad=True)
    kt_ = torch.tensor(k, dtype=torch.float64, requires_grad=True)
    vt = torch.tensor(v, dtype=torch.float64, requires_grad=True)
    ot = torch.tensor(off, dtype=torch.float64, requires_grad=True)
    pos32 = torch.tensor(positions_f32(T, H, W, M, off, kt, kh, kw))
    pos = pos32 + (ot - ot.detach())  # value: the fp32 position; derivative: 1 w.r.t. the offset
    size = torch.tensor([W, H, T], dtype=torch.float64)
    grid_n = (2.0 * pos + 1.0) / size - 1.0  # [B,T,H,W,M,P,3] normalised, (x,y,z)
    outs, lses = [], []
    for m in range(M):
        g = grid_n[:, :, :, :, m].reshape(B, T, H, W * P, 3)
        K5 = kt_[:, :, :, :, m].permute(0, 4, 1, 2, 3)
        V5 = vt[:, :, :, :, m].permute(0, 4, 1, 2, 3)
        ks = torch.nn.functional.grid_sample(K5, g, mode="bilinear", padding_mode="zeros",
                                             align_corners=False)
        vs = torch.nn.functional.grid_sample(V5, g, mode="bilinear", padding_mode="zeros",
                                             align_corners=False)
        ks = ks.reshape(B, D, T, H, W, P).permute(0, 2, 3, 4, 5, 1)  # [B,T,H,W,P,D]
        vs = vs.reshape(B, D, T, H, W, P).permute(0, 2, 3, 4, 5, 1)
        s = scale * (qt[:, :, :, :, m, None, :] * ks).sum(-1)
        a = torch.softmax(s, -1)
        outs.append((a[..., None] * vs).sum(-2))
        lses.append(torch.logsumexp(s, -1))
    out = torch.stack(outs, 4)
    lse = torch.stack(lses, 4)
    grads = None
    if dout is not None:
        (out * torch.tensor(dout, dtype=torch.float64)).sum().backward()
        grads = tuple(t.grad.numpy() for t in (qt, kt_, vt, ot))
    return out.detach().numpy(), lse.detach().numpy(), grads


def oracle_full_forward(q, k, v, off, kt, kh, kw, scale):
    out, lse = oracle.forward(shape_of(q, kt, kh, kw), "f32", q, k, v, off, scale=scale)
    return out.reshape(q.shape), lse.reshape(q.shape[:5])


# ----------------------------------------------------------------------------- worked examples

def _golden():
    with open(GOLDEN) as f:
        return json.load(f)["examples"]


@pytest.mark.parametrize("ex", _golden(), ids=lambda e: e["name"])
def test_worked_examples(ex):
    T, H, W = ex["grid"]
    D = ex["D"]
    kt, kh, kw = ex["kernel"]
    P = kt * kh * kw
    q = np.array(ex["q"], dtype=np.float32).reshape(1, T, H, W, 1, D)
    k = np.array(ex["k"], dtype=np.float32).reshape(1, T, H, W, 1, D)
    v = np.array(ex["v"], dtype=np.float32).reshape(1, T, H, W, 1, D)
    off = np.zeros((1, T, H, W, 1, P, 3), dtype=np.float32)
    t, i, j = ex["query"]
    if "offset" in ex:
        off[0, t, i, j, 0, 0] = ex["offset"]
    shape = (1, T, H, W, 1, D, kt, kh, kw)
    row = ((t * H + i) * W + j)
    out, lse = oracle.forward(shape, "f32", q, k, v, off, rows=[row], scale=ex["scale"])
    np.testing.assert_allclose(out[0], ex["out"], rtol=0, atol=1e-12)
    assert abs(lse[0] - ex["lse"]) < 1e-12
    if "doff" in ex:
        dout = np.zeros_like(q)
        dout[0, t, i, j, 0] = ex["dout"]
        dq, dk, dv, doff = oracle.backward(shape, "f32", q, k, v, off, dout, scale=ex["scale"])
        np.testing.assert_allclose(doff[0, t, i, j, 0, 0], ex["doff"], atol=1e-12)
        np.testing.assert_allclose(dq[0, t, i, j, 0], ex["dq"], atol=1e-12)
        for (zz, yy, xx, val) in ex["dv_at"]:
            assert abs(dv[0, zz, yy, xx, 0, 0] - val) < 1e-12
        for (zz, yy, xx, val) in ex["dk_at"]:
            assert abs(dk[0, zz, yy, xx, 0, 0] - val) < 1e-12


# ----------------------------------------------------------------------------- special cases

@pytest.mark.parametrize("kern", [(3, 3, 3), (1, 3, 5), (3, 5, 5), (3, 7, 7)])
def test_zero_offsets_equal_fixed_window_attention(kern):
    """Section 9.1: offsets frozen at zero give fixed local attention over the kernel."""
    rng = np.random.default_rng(11)
    kt, kh, kw = kern
    q, k, v, _ = rand_case(rng, 2, 4, 5, 6, 2, 8, kt, kh, kw)
    off = np.zeros((2, 4, 5, 6, 2, kt * kh * kw, 3), np.float32)
    scale = 1.0 / math.sqrt(8)
    out, lse = oracle_full_forward(q, k, v, off, kt, kh, kw, scale)
    ref, ref_lse = slide_attention_integer(q, k, v, off.astype(np.int64), kt, kh, kw, scale)
    np.testing.assert_allclose(out, ref, rtol=0, atol=1e-12)
    np.testing.assert_allclose(lse, ref_lse, rtol=0, atol=1e-12)


def test_integer_offsets_are_exact_gathers():
    rng = np.random.default_rng(12)
    kt, kh, kw = 3, 3, 3
    q, k, v, _ = rand_case(rng, 1, 5, 6, 7, 3, 16, kt, kh, kw)
    ioff = rng.integers(-3, 4, (1, 5, 6, 7, 3, 27, 3))
    scale = 0.3
    out, lse = oracle_full_forward(q, k, v, ioff.astype(np.float32), kt, kh, kw, scale)
    ref, ref_lse = slide_attention_integer(q, k, v, ioff, kt, kh, kw, scale)
    np.testing.assert_allclose(out, ref, rtol=0, atol=1e-12)
    np.testing.assert_allclose(lse, ref_lse, rtol=0, atol=1e-12)


def test_single_point_integer_offset_copies_the_row():
    """1x1x1 kernel: alpha = 1, so out is exactly V at the shifted position (or 0 outside);
    also fixes the offset component order (x = w, y = h, z = t)."""
    rng = np.random.default_rng(13)
    q, k, v, _ = rand_case(rng, 1, 3, 4, 5, 1, 4, 1, 1, 1)
    for comp, (dx, dy, dz) in enumerate([(1, 0, 0), (0, 1, 0), (0, 0, 1)]):
        off = np.zeros((1, 3, 4, 5, 1, 1, 3), np.float32)
        off[..., 0, :] = (dx, dy, dz)
        out, _ = oracle_full_forward(q, k, v, off, 1, 1, 1, 1.0)
        for t in range(3):
            for i in range(4):
                for j in range(5):
                    z, y, x = t + dz, i + dy, j + dx
                    want = v[0, z, y, x, 0] if (z < 3 and y < 4 and x < 5) else np.zeros(4)
                    assert np.array_equal(out[0, t, i, j, 0], want.astype(np.float64))


def test_bruteforce_hat_function_interpolation():
    """Sum over every grid voxel of prod_d max(0, 1 - |pos_d - x_d|), including positions far
    outside the grid, against the oracle's floor/frac corner form."""
    rng = np.random.default_rng(14)
    kt, kh, kw = 3, 3, 3
    B, T, H, W, M, D = 1, 3, 4, 5, 2, 6
    q, k, v, off = rand_case(rng, B, T, H, W, M, D, kt, kh, kw, off_std=2.5)
    scale = 0.5
    out, lse = oracle_full_forward(q, k, v, off, kt, kh, kw, scale)
    pos = positions_f32(T, H, W, M, off, kt, kh, kw)
    k64, v64, q64 = k.astype(np.float64), v.astype(np.float64), q.astype(np.float64)
    for t in range(T):
        for i in range(H):
            for j in range(W):
                for m in range(M):
                    kp = np.array([hat_sample(k64[0, :, :, :, m], pos[0, t, i, j, m, p]) for p in range(27)])
                    vp = np.array([hat_sample(v64[0, :, :, :, m], pos[0, t, i, j, m, p]) for p in range(27)])
                    s = scale * kp @ q64[0, t, i, j, m]
                    a = np.exp(s - s.max())
                    np.testing.assert_allclose(out[0, t, i, j, m], (a / a.sum()) @ vp, rtol=0, atol=1e-12)
                    assert abs(lse[0, t, i, j, m] - (s.max() + np.log(a.sum()))) < 1e-12


@pytest.mark.parametrize("kern,off_std", [((1, 1, 1), 1.5), ((3, 3, 3), 1.0), ((3, 5, 5), 3.0)])
def test_matches_grid_sample_route_with_autograd(kern, off_std):
    """Section 5.3's implementation (grid_sample on 5D tensors, zero padding) in fp64 torch,
    forward and every gradient through autograd."""
    rng = np.random.default_rng(15)
    kt, kh, kw = kern
    q, k, v, off = rand_case(rng, 2, 3, 4, 5, 2, 8, kt, kh, kw, off_std=off_std)
    dout = rng.standard_normal(q.shape).astype(np.float32)
    scale = 1.0 / math.sqrt(8)
    ref, ref_lse, (gq, gk, gv, goff) = torch_reference(q, k, v, off, kt, kh, kw, scale, dout)
    out, lse = oracle_full_forward(q, k, v, off, kt, kh, kw, scale)
    np.testing.assert_allclose(out, ref, rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(lse, ref_lse, rtol=1e-10, atol=1e-12)
    dq, dk, dv, doff = oracle.backward(shape_of(q, kt, kh, kw), "f32", q, k, v, off, dout, scale=scale)
    for name, a, b in (("dq", dq, gq), ("dk", dk, gk), ("dv", dv, gv), ("doff", doff, goff)):
        np.testing.assert_allclose(a, b, rtol=1e-9, atol=1e-10, err_msg=name)


def test_bf16_inputs_are_read_exactly():
    """bf16 storage: the oracle must see exactly the fp32 value of each bf16 pattern."""
    import testgen
    rng = np.random.default_rng(16)
    q, k, v, off = rand_case(rng, 1, 3, 4, 4, 2, 8, 3, 3, 3)
    qb, kb, vb = (testgen.f32_to_bf16(a) for a in (q, k, v))
    qf, kf, vf = (testgen.bf16_to_f32(a) for a in (qb, kb, vb))
    shape = shape_of(q, 3, 3, 3)
    o1, l1 = oracle.forward(shape, "bf16", qb, kb, vb, off)
    o2, l2 = oracle.forward(shape, "f32", qf, kf, vf, off)
    assert np.array_equal(o1, o2) and np.array_equal(l1, l2)


# ----------------------------------------------------------------------------- finite differences

def test_finite_differences_all_inputs():
    """Central differences of L = sum(out * dout) in fp64 (inputs on a 2^-12 grid, step 2^-10,
    both exact in fp32), skipping offset components within one step of an integer position."""
    rng = np.random.default_rng(17)
    kt, kh, kw = 3, 3, 3
    B, T, H, W, M, D = 1, 3, 3, 4, 2, 4
    h = 2.0 ** -10
    q, k, v, off = rand_case(rng, B, T, H, W, M, D, kt, kh, kw, off_std=1.2, grid_step=2.0 ** -12)
    dout = rng.standard_normal(q.shape).astype(np.float32)
    scale = 0.7
    shape = shape_of(q, kt, kh, kw)
    dq, dk, dv, doff = oracle.backward(shape, "f32", q, k, v, off, dout, scale=scale)

    def loss(qq, kk, vv, oo):
        out, _ = oracle.forward(shape, "f32", qq, kk, vv, oo, scale=scale)
        return float(np.sum(out.reshape(q.shape) * dout.astype(np.float64)))

    pos = positions_f32(T, H, W, M, off, kt, kh, kw)
    frac = pos - np.floor(pos)
    checked = 0
    for which, arr, grad in (("q", q, dq), ("k", k, dk), ("v", v, dv), ("off", off, doff)):
        flat_idx = rng.choice(arr.size, size=40, replace=False)
        for fi in flat_idx:
            idx = np.unravel_index(fi, arr.shape)
            if which == "off":
                fr = frac[idx]
                if min(fr, 1.0 - fr) <= 2 * h:
                    continue
            args = {"q": q, "k": k, "v": v, "off": off}
            plus = {n: a.copy() for n, a in args.items()}
            minus = {n: a.copy() for n, a in args.items()}
            plus[which][idx] += np.float32(h)
            minus[which][idx] -= np.float32(h)
            assert plus[which][idx] - minus[which][idx] == np.float32(2 * h)
            fd = (loss(plus["q"], plus["k"], plus["v"], plus["off"])
                  - loss(minus["q"], minus["k"], minus["v"], minus["off"])) / (2 * h)
            an = grad[idx]
            assert abs(fd - an) <= 2e-6 * (1.0 + abs(an)), (which, idx, fd, an)
            checked += 1
    assert checked > 120


# ----------------------------------------------------------------------------- invariants

def test_softmax_normalisation():
    rng = np.random.default_rng(18)
    kt, kh, kw = 3, 3, 3
    B, T, H, W, M, D = 1, 6, 6, 6, 2, 8
    q, k, _, off = rand_case(rng, B, T, H, W, M, D, kt, kh, kw, off_unif=0.4)
    # V == 1 and every sample strictly inside -> out == 1 (checked on interior queries)
    v = np.ones_like(q)
    out, _ = oracle_full_forward(q, k, v, off, kt, kh, kw, 0.5)
    np.testing.assert_allclose(out[:, 2:4, 2:4, 2:4], 1.0, rtol=0, atol=1e-13)
    # q == 0 -> alpha == 1/P: out is the mean of the sampled values and LSE = ln P
    q0 = np.zeros_like(q)
    vrand = rng.standard_normal(q.shape).astype(np.float32)
    out0, lse0 = oracle_full_forward(q0, k, vrand, off, kt, kh, kw, 0.5)
    np.testing.assert_allclose(lse0, math.log(27), rtol=0, atol=1e-13)
    out_one = oracle_full_forward(q0, k, np.ones_like(q), off, kt, kh, kw, 0.5)[0]
    pos = positions_f32(T, H, W, M, off, kt, kh, kw)
    # with V == 1 the sampled value is the in-grid trilinear weight mass of each point
    for (t, i, j, m) in [(0, 0, 0, 0), (5, 5, 5, 1), (2, 3, 1, 0)]:
        mass = np.mean([hat_sample(np.ones((T, H, W, 1)), pos[0, t, i, j, m, p])[0] for p in range(27)])
        assert abs(out_one[0, t, i, j, m, 0] - mass) < 1e-13


def test_heads_and_batch_items_are_independent():
    rng = np.random.default_rng(19)
    q, k, v, off = rand_case(rng, 2, 3, 4, 5, 3, 8, 3, 3, 3)
    out, lse = oracle_full_forward(q, k, v, off, 3, 3, 3, 0.4)
    k2, v2, off2 = k.copy(), v.copy(), off.copy()
    k2[:, :, :, :, 1] += 1.0
    v2[:, :, :, :, 1] *= -2.0
    off2[:, :, :, :, 1] += 0.5
    k2[1] += 3.0
    out2, lse2 = oracle_full_forward(q, k2, v2, off2, 3, 3, 3, 0.4)
    for m in (0, 2):
        assert np.array_equal(out[0, :, :, :, m], out2[0, :, :, :, m])
        assert np.array_equal(lse[0, :, :, :, m], lse2[0, :, :, :, m])
    assert not np.allclose(out[0, :, :, :, 1], out2[0, :, :, :, 1])
    assert not np.allclose(out[1], out2[1])


def test_linear_in_v_and_scale_folding():
    rng = np.random.default_rng(20)
    q, k, v, off = rand_case(rng, 1, 3, 4, 5, 2, 8, 3, 3, 3)
    v2 = rng.standard_normal(v.shape).astype(np.float32)
    o1, _ = oracle_full_forward(q, k, v, off, 3, 3, 3, 0.4)
    o2, _ = oracle_full_forward(q, k, v2, off, 3, 3, 3, 0.4)
    o12, _ = oracle_full_forward(q, k, v + v2, off, 3, 3, 3, 0.4)
    # v + v2 is rounded to fp32, so compare against the exactly-representable sum
    o_sum_ref, _ = oracle_full_forward(q, k, (v.astype(np.float64) + v2).astype(np.float32), off, 3, 3, 3, 0.4)
    np.testing.assert_allclose(o12, o_sum_ref, atol=0)
    np.testing.assert_allclose(o1 + o2, o12, atol=1e-6)
    # (2q, scale/2) gives the same logits exactly
    o3, l3 = oracle_full_forward(2 * q, k, v, off, 3, 3, 3, 0.2)
    o4, l4 = oracle_full_forward(q, k, v, off, 3, 3, 3, 0.4)
    np.testing.assert_allclose(o3, o4, rtol=0, atol=1e-14)
    np.testing.assert_allclose(l3, l4, rtol=0, atol=1e-14)


def test_point_order_permutation():
    """Relabelling points (moving offsets with their positions) permutes nothing in the output
    and permutes the offset gradients with the points."""
    rng = np.random.default_rng(21)
    kt, kh, kw = 3, 3, 3
    q, k, v, off = rand_case(rng, 1, 3, 4, 5, 1, 8, kt, kh, kw, grid_step=2.0 ** -10)
    g = base_grid(kt, kh, kw).astype(np.float32)
    perm = rng.permutation(27)
    # point p of the new labelling samples where point perm[p] sampled before
    off_new = (off[..., perm, :] + (g[perm] - g)[None, None, None, None, None]).astype(np.float32)
    o1, l1 = oracle_full_forward(q, k, v, off, kt, kh, kw, 0.4)
    o2, l2 = oracle_full_forward(q, k, v, off_new, kt, kh, kw, 0.4)
    np.testing.assert_allclose(o1, o2, rtol=0, atol=1e-13)
    np.testing.assert_allclose(l1, l2, rtol=0, atol=1e-13)
    dout = rng.standard_normal(q.shape).astype(np.float32)
    shape = shape_of(q, kt, kh, kw)
    g1 = oracle.backward(shape, "f32", q, k, v, off, dout, scale=0.4)
    g2 = oracle.backward(shape, "f32", q, k, v, off_new, dout, scale=0.4)
    np.testing.assert_allclose(g1[3][..., perm, :], g2[3], rtol=0, atol=1e-12)
    for a, b in zip(g1[:3], g2[:3]):
        np.testing.assert_allclose(a, b, rtol=0, atol=1e-12)


def test_translation_equivariance_in_the_interior():
    """Shifting every input by one token along each axis shifts the output of queries whose
    samples stay inside the grid (index or axis mix-ups break this)."""
    rng = np.random.default_rng(22)
    kt, kh, kw = 3, 3, 3
    B, T, H, W, M, D = 1, 7, 8, 9, 1, 4
    q, k, v, off = rand_case(rng, B, T, H, W, M, D, kt, kh, kw, off_unif=0.45, grid_step=2.0 ** -10)
    out, _ = oracle_full_forward(q, k, v, off, kt, kh, kw, 0.5)
    for axis in (1, 2, 3):
        sh = [np.roll(a, 1, axis=axis) for a in (q, k, v, off)]
        out_s, _ = oracle_full_forward(*sh, kt, kh, kw, 0.5)
        ref = np.roll(out, 1, axis=axis)
        np.testing.assert_allclose(out_s[:, 3:5, 3:5, 3:6], ref[:, 3:5, 3:5, 3:6], rtol=0, atol=1e-12)


def test_no_causal_mask():
    """Section 5.3: no causal masking -- a later frame's keys change an earlier frame's output."""
    rng = np.random.default_rng(23)
    q, k, v, off = rand_case(rng, 1, 4, 4, 4, 1, 8, 3, 3, 3, off_unif=0.3)
    o1, _ = oracle_full_forward(q, k, v, off, 3, 3, 3, 0.5)
    k2 = k.copy()
    k2[0, 2] += 1.0
    o2, _ = oracle_full_forward(q, k2, v, off, 3, 3, 3, 0.5)
    assert np.max(np.abs(o1[0, 1] - o2[0, 1])) > 1e-3
    assert np.array_equal(o1[0, 0][..., :], o1[0, 0])  # frame 0 samples frames <= 1 only here
