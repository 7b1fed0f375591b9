"""The no-allocation backward (dsa3d_backward_noalloc, which runs in the library's fixed
scratch array) against dsa3d_backward with a caller workspace, through the C ABI.

Two calls in a row, the second on a smaller problem, so that the second one runs on the
scratch contents the first left behind.  dq and d_offsets are query-owned and must match
bit for bit; dK and dV sum each trilinear bin in the order its points claimed their slots,
which may differ between calls, so they are held to 1e-4 of the relative metric; all four
are also checked against the oracle at the bf16 bar (2e-2).
"""
import numpy as np
import pytest

import oracle
import testgen
from tests.util import rel_err, say, shape9, to_device, to_host

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2607_22696_amd as dsa
    dsa.load()
    yield


def cases():
    base = testgen.WORKLOADS["tiny_f32"]
    return [
        base.with_grid(name="noalloc_first", T=6, H=17, W=23, heads=3, head_dim=64, dtype="bf16",
                       seed=60, offsets=testgen.Dist(testgen.UNIFORM, -2.0, 2.0)),
        base.with_grid(name="noalloc_second_smaller", T=3, H=5, W=7, heads=2, head_dim=128,
                       dtype="bf16", seed=61),
    ]


def test_noalloc_backward_matches_the_workspace_backward_on_two_calls():
    import paper_2607_22696_amd as dsa
    for w in cases():
        say(f"case {w.name}: grid {w.T}x{w.H}x{w.W} heads={w.heads} D={w.head_dim}")
        q, k, v, off, _ = testgen.gen_inputs(w)
        dout = testgen.gen_tensor(w, testgen.TID_DOUT, w.qkv_shape(), w.dout, True)
        qd, kd, vd, gd = (to_device(a, True) for a in (q, k, v, dout))
        od = to_device(off, False)
        kern = (w.kt, w.kh, w.kw)
        out, lse = dsa.forward(qd, kd, vd, od, kernel=kern)
        ref = [to_host(t) for t in dsa.backward(qd, kd, vd, od, lse, gd, kernel=kern)]
        desc = dsa.make_desc(w.B, w.T, w.H, w.W, w.heads, w.head_dim, *kern, "bf16")
        assert dsa.dsa3d_backward_workspace_size(desc) <= dsa._binding.DSA3D_NOALLOC_SCRATCH_BYTES
        f32 = dict(dtype=torch.float32, device=qd.device)
        dq, dk, dv = (torch.full(q.shape, float("nan"), **f32) for _ in range(3))
        doff = torch.full(off.shape, float("nan"), **f32)
        dsa.dsa3d_backward_noalloc(desc, qd, kd, vd, od, out, lse, gd, dq, dk, dv, doff)
        torch.cuda.synchronize()
        got = [to_host(t) for t in (dq, dk, dv, doff)]
        assert np.array_equal(got[0], ref[0]), "dq"
        assert np.array_equal(got[3], ref[3]), "d_offsets"
        for i, name in ((1, "dk"), (2, "dv")):
            e = rel_err(got[i], ref[i])
            say(f"  {name} vs workspace backward: rel {e:.2e}")
            assert e <= 1e-4, name
        rq, rk, rv, roff = oracle.backward(shape9(w), w.dtype, q, k, v, off, dout)
        for g, r, name in zip(got, (rq, rk, rv, roff), ("dq", "dk", "dv", "d_offsets")):
            e = rel_err(g, r)
            say(f"  {name} vs oracle: rel {e:.2e}")
            assert e <= 2e-2, name
