"""CPU-side checks of the C ABI: the library loads, exports every declared entry point, and
every validation error returns its status before anything is launched (all pointers here
are fake host addresses; no call in this file reaches the GPU)."""
import ctypes
import os
import re

import pytest

import paper_2607_22696_amd as dsa
from paper_2607_22696_amd import _binding as B

INCLUDE = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include")


def declared_functions():
    names = set()
    for h in sorted(os.listdir(INCLUDE)):
        if h.endswith(".h"):
            src = open(os.path.join(INCLUDE, h)).read()
            src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
            names |= set(re.findall(r"\b(dsa3d_[a-z0-9_]+)\s*\(", src))
    return sorted(names)


def test_library_exports_every_declared_function():
    lib = ctypes.CDLL(B.LIB_PATH)
    names = declared_functions()
    assert set(names) == set(B.EXPORTED), names
    for n in names:
        assert hasattr(lib, n), n


def test_abi_version_and_status_strings():
    assert dsa.dsa3d_abi_version() == 1
    for s in range(0, 9):
        assert isinstance(dsa.status_string(s), str) and dsa.status_string(s)
    assert dsa.status_string(99) == "unknown status"


def test_desc_layout_matches_header():
    # 9 int32 dims + float scale + enum dtype
    assert ctypes.sizeof(B.dsa3d_desc) == 11 * 4


A = 1 << 20  # fake, well-aligned, non-overlapping "device" addresses (never dereferenced)


def ptrs(n, stride=1 << 34, base=1 << 40):
    return [base + i * stride for i in range(n)]


def fwd(desc, **over):
    q, k, v, off, out, lse = ptrs(6)
    args = dict(q=q, k=k, v=v, offsets=off, out=out, lse=lse)
    args.update(over)
    return dsa.dsa3d_forward(desc, args["q"], args["k"], args["v"], args["offsets"], args["out"],
                             args["lse"], stream=0, check=False)


BWD_NAMES = ["q", "k", "v", "offsets", "out", "lse", "dout", "dq", "dk", "dv", "d_offsets",
             "workspace"]


def bwd(desc, **over):
    names = BWD_NAMES
    args = dict(zip(names, ptrs(len(names))))
    args["workspace_bytes"] = 1 << 33
    args.update(over)
    return dsa.dsa3d_backward(desc, *[args[n] for n in names[:-1]], workspace=args["workspace"],
                              workspace_bytes=args["workspace_bytes"], stream=0, check=False)


def good_desc(**kw):
    d = dict(B=1, T=4, H=8, W=8, heads=2, head_dim=32, kt=3, kh=3, kw=3, dtype="f32", scale=0.0)
    d.update(kw)
    return dsa.make_desc(d["B"], d["T"], d["H"], d["W"], d["heads"], d["head_dim"], d["kt"],
                         d["kh"], d["kw"], d["dtype"], d["scale"])


@pytest.mark.parametrize("kw,status", [
    (dict(B=0), B.DSA3D_ERR_INVALID_SHAPE),
    (dict(T=-1), B.DSA3D_ERR_INVALID_SHAPE),
    (dict(heads=0), B.DSA3D_ERR_INVALID_SHAPE),
    (dict(kt=2), B.DSA3D_ERR_INVALID_SHAPE),
    (dict(kw=4), B.DSA3D_ERR_INVALID_SHAPE),
    (dict(kh=0), B.DSA3D_ERR_INVALID_SHAPE),
    (dict(scale=float("nan")), B.DSA3D_ERR_INVALID_SHAPE),
    (dict(scale=float("inf")), B.DSA3D_ERR_INVALID_SHAPE),
    (dict(T=1 << 16, H=1 << 16, W=2), B.DSA3D_ERR_INVALID_SHAPE),        # 2^33 tokens
    (dict(T=1 << 12, H=1 << 10, W=1 << 8, heads=2), B.DSA3D_ERR_INVALID_SHAPE),  # 2^31 rows
    (dict(head_dim=48), B.DSA3D_ERR_UNSUPPORTED),
    (dict(head_dim=256), B.DSA3D_ERR_UNSUPPORTED),
    (dict(kt=11, kh=11, kw=11), B.DSA3D_ERR_UNSUPPORTED),                 # P = 1331 > 1024
])
def test_descriptor_errors(kw, status):
    d = good_desc(**kw)
    assert fwd(d) == status
    assert bwd(d) == status


def test_bad_dtype():
    d = good_desc()
    d.dtype = 7
    assert fwd(d) == B.DSA3D_ERR_UNSUPPORTED


def test_null_pointers():
    assert dsa.dsa3d_forward(None, *ptrs(6), stream=0, check=False) == B.DSA3D_ERR_NULL_POINTER
    d = good_desc()
    for name in ["q", "k", "v", "offsets", "out"]:
        assert fwd(d, **{name: None}) == B.DSA3D_ERR_NULL_POINTER, name
    for name in ["q", "k", "v", "offsets", "lse", "dout", "dq", "dk", "dv", "d_offsets"]:
        assert bwd(d, **{name: None}) == B.DSA3D_ERR_NULL_POINTER, name


def test_misaligned_pointers():
    d = good_desc()
    for name in ["q", "k", "v", "out"]:
        p = ptrs(8)[7] + 8
        assert fwd(d, **{name: p}) == B.DSA3D_ERR_MISALIGNED, name
    assert fwd(d, offsets=ptrs(8)[7] + 2) == B.DSA3D_ERR_MISALIGNED
    assert fwd(d, lse=ptrs(8)[7] + 1) == B.DSA3D_ERR_MISALIGNED
    for name in ["q", "k", "v", "dout", "dq", "dk", "dv"]:
        assert bwd(d, **{name: ptrs(16)[15] + 4}) == B.DSA3D_ERR_MISALIGNED, name
    for name in ["offsets", "lse", "d_offsets"]:
        assert bwd(d, **{name: ptrs(16)[15] + 2}) == B.DSA3D_ERR_MISALIGNED, name


def test_overlapping_outputs():
    d = good_desc()
    q = ptrs(1)[0]
    assert fwd(d, out=q) == B.DSA3D_ERR_ALIAS
    assert fwd(d, out=q + 256) == B.DSA3D_ERR_ALIAS      # partial overlap of q's range
    assert fwd(d, lse=q + 1024) == B.DSA3D_ERR_ALIAS
    names = ptrs(12)
    assert bwd(d, dk=names[7]) == B.DSA3D_ERR_ALIAS      # dk == dq
    assert bwd(d, d_offsets=names[0] + 64) == B.DSA3D_ERR_ALIAS
    assert bwd(d, dv=names[4] + 256) == B.DSA3D_ERR_ALIAS   # dv inside out


def test_backward_out_is_optional_but_checked_when_given():
    """out (the forward's output) is not read by the backward: NULL is accepted, a given
    pointer must be aligned and must not overlap an output or the workspace."""
    d = good_desc()
    need = dsa.dsa3d_backward_workspace_size(d)
    names = ptrs(12)
    # NULL out passes the pointer checks: the call stops at the (later) workspace check
    assert bwd(d, out=None, workspace_bytes=need - 1) == B.DSA3D_ERR_WORKSPACE
    assert bwd(d, out=ptrs(16)[15] + 8) == B.DSA3D_ERR_MISALIGNED
    assert bwd(d, out=names[7]) == B.DSA3D_ERR_ALIAS            # out == dq
    assert bwd(d, out=names[11] + 1024) == B.DSA3D_ERR_ALIAS    # out inside the workspace
    assert bwd_timed(d, out=names[8]) == B.DSA3D_ERR_ALIAS      # out == dk


def noalloc(desc, **over):
    names = BWD_NAMES[:-1]
    args = dict(zip(names, ptrs(len(names))))
    args.update(over)
    return dsa.dsa3d_backward_noalloc(desc, *[args[n] for n in names], stream=0, check=False)


def test_noalloc_backward_checks_before_touching_the_device():
    """The no-allocation backward validates like dsa3d_backward (minus the workspace) and
    rejects a problem whose workspace exceeds its fixed scratch, all on the host."""
    d = good_desc()
    assert noalloc(good_desc(kt=2)) == B.DSA3D_ERR_INVALID_SHAPE
    assert noalloc(d, dq=None) == B.DSA3D_ERR_NULL_POINTER
    assert noalloc(d, dk=ptrs(16)[15] + 4) == B.DSA3D_ERR_MISALIGNED
    assert noalloc(d, dv=ptrs(1)[0]) == B.DSA3D_ERR_ALIAS            # dv == q
    big = good_desc(T=16, H=64, W=64, heads=2, head_dim=64, kt=3, kh=3, kw=3)
    assert dsa.dsa3d_backward_workspace_size(big) > B.DSA3D_NOALLOC_SCRATCH_BYTES
    assert noalloc(big) == B.DSA3D_ERR_SCRATCH
    fits = good_desc(T=8, H=32, W=32, heads=2, head_dim=64)
    assert dsa.dsa3d_backward_workspace_size(fits) <= B.DSA3D_NOALLOC_SCRATCH_BYTES
    src = open(os.path.join(INCLUDE, "dsa3d.h")).read()
    assert re.search(r"DSA3D_NOALLOC_SCRATCH_BYTES \(128u << 20\)", src)
    assert B.DSA3D_NOALLOC_SCRATCH_BYTES == 128 << 20


def test_status_codes_match_the_header():
    src = open(os.path.join(INCLUDE, "dsa3d.h")).read()
    codes = dict((n, int(v)) for n, v in re.findall(r"\b(DSA3D_(?:OK|ERR_[A-Z_]+))\s*=\s*(\d+)", src))
    assert codes == {"DSA3D_OK": 0, "DSA3D_ERR_NULL_POINTER": 1, "DSA3D_ERR_INVALID_SHAPE": 2,
                     "DSA3D_ERR_UNSUPPORTED": 3, "DSA3D_ERR_MISALIGNED": 4,
                     "DSA3D_ERR_WORKSPACE": 5, "DSA3D_ERR_DEVICE": 6, "DSA3D_ERR_ALIAS": 7,
                     "DSA3D_ERR_SCRATCH": 8}
    for n, v in codes.items():
        assert getattr(B, n) == v, n


def test_workspace_size_follows_the_documented_formula():
    for kw in (dict(), dict(B=2, T=5, H=7, W=9, heads=3, kt=3, kh=5, kw=5)):
        d = good_desc(**kw)
        rows = d.batch * d.frames * d.height * d.width * d.heads
        P = d.kt * d.kh * d.kw
        cells = d.batch * d.heads * (d.frames + 1) * (d.height + 1) * (d.width + 1)
        ws = dsa.dsa3d_backward_workspace_size(d)
        assert ws % 256 == 0
        lo = 60 * rows * P + 12 * cells + 4 * rows
        assert lo <= ws <= lo + 9 * 256 + 4 * (cells // 4096 + 1) + 4
    assert dsa.dsa3d_backward_workspace_size(good_desc(kt=2)) == 0


def test_workspace_errors():
    d = good_desc()
    need = dsa.dsa3d_backward_workspace_size(d)
    assert bwd(d, workspace=None) == B.DSA3D_ERR_WORKSPACE
    assert bwd(d, workspace_bytes=need - 1) == B.DSA3D_ERR_WORKSPACE
    assert bwd(d, workspace=ptrs(16)[15] + 128) == B.DSA3D_ERR_MISALIGNED
    names = ptrs(12)
    assert bwd(d, workspace=names[7]) == B.DSA3D_ERR_ALIAS          # workspace == dq
    assert bwd(d, workspace=names[0], workspace_bytes=need) == B.DSA3D_ERR_ALIAS  # == q


def test_backward_index_range_limit():
    # 2^22 rows x 729 points > 2^31 (row, point) pairs: the forward accepts it, the
    # backward's 32-bit bins do not.
    d2 = good_desc(T=1 << 7, H=1 << 7, W=1 << 6, heads=2, kt=7, kh=7, kw=7)  # 2^21 rows, P=343
    assert dsa.dsa3d_backward_workspace_size(d2) > 0  # 2^21 * 343 < 2^31
    d3 = good_desc(T=1 << 8, H=1 << 7, W=1 << 6, heads=2, kt=9, kh=9, kw=9)  # 2^22 rows, P=729
    assert dsa.dsa3d_backward_workspace_size(d3) == 0
    assert bwd(d3) == B.DSA3D_ERR_INVALID_SHAPE


def bwd_timed(desc, events=None, **over):
    names = BWD_NAMES
    args = dict(zip(names, ptrs(len(names))))
    args["workspace_bytes"] = 1 << 33
    args.update(over)
    return dsa.dsa3d_backward_timed(desc, *[args[n] for n in names[:-1]],
                                    workspace=args["workspace"],
                                    workspace_bytes=args["workspace_bytes"], stream=0,
                                    events=events, check=False)


def test_timed_backward_validates_like_backward():
    d = good_desc()
    need = dsa.dsa3d_backward_workspace_size(d)
    names = ptrs(12)
    cases = [dict(q=None), dict(d_offsets=None), dict(dq=ptrs(16)[15] + 4),
             dict(workspace=None), dict(workspace_bytes=need - 1), dict(dk=names[7]),
             dict(out=names[9])]
    fake_events = list(range(1 << 12, (1 << 12) + B.DSA3D_BACKWARD_PHASES + 1))
    for over in cases:
        want = bwd(d, **over)
        assert want != B.DSA3D_OK
        assert bwd_timed(d, **over) == want, over
        # the events are only touched after every check has passed
        assert bwd_timed(d, events=fake_events, **over) == want, over
    bad = good_desc(kt=2)
    assert bwd_timed(bad, events=fake_events) == B.DSA3D_ERR_INVALID_SHAPE


def test_timed_backward_needs_one_event_per_phase_boundary():
    with pytest.raises(ValueError):
        bwd_timed(good_desc(), events=[1, 2, 3])


# ----------------------------------------------------------------------------- depthwise conv

def good_conv(**kw):
    d = dict(B=1, T=4, H=5, W=6, C=8, kt=3, kh=3, kw=3, dtype="f32")
    d.update(kw)
    return dsa.make_conv_desc(d["B"], d["T"], d["H"], d["W"], d["C"], d["kt"], d["kh"], d["kw"],
                              d["dtype"])


def conv_fwd(desc, **over):
    x, w, b, y = ptrs(4)
    args = dict(x=x, weight=w, bias=b, y=y)
    args.update(over)
    return dsa.dsa3d_dwconv3d_forward(desc, args["x"], args["weight"], args["bias"], args["y"],
                                      stream=0, check=False)


def conv_bwd(desc, **over):
    names = ["x", "weight", "dy", "dx", "dweight", "dbias", "workspace"]
    args = dict(zip(names, ptrs(len(names))))
    args["workspace_bytes"] = 1 << 33
    args.update(over)
    return dsa.dsa3d_dwconv3d_backward(desc, args["x"], args["weight"], args["dy"], args["dx"],
                                       args["dweight"], args["dbias"], args["workspace"],
                                       args["workspace_bytes"], stream=0, check=False)


def test_conv_desc_layout_matches_header():
    assert ctypes.sizeof(B.dsa3d_dwconv_desc) == 9 * 4


@pytest.mark.parametrize("kw,status", [
    (dict(T=0), B.DSA3D_ERR_INVALID_SHAPE), (dict(C=0), B.DSA3D_ERR_INVALID_SHAPE),
    (dict(C=7), B.DSA3D_ERR_INVALID_SHAPE), (dict(kt=2), B.DSA3D_ERR_INVALID_SHAPE),
    (dict(kw=4), B.DSA3D_ERR_INVALID_SHAPE), (dict(kh=9), B.DSA3D_ERR_UNSUPPORTED),
    (dict(kt=3, kh=7, kw=7), B.DSA3D_ERR_UNSUPPORTED),          # 147 taps
    (dict(kt=9, kh=3, kw=3), B.DSA3D_OK),                       # 81 taps, kt free
    (dict(B=1 << 16, T=1 << 8, H=1 << 4, W=1 << 3), B.DSA3D_ERR_INVALID_SHAPE),  # 2^31 tokens
])
def test_conv_descriptor_errors(kw, status):
    assert conv_fwd(good_conv(**kw), x=None if status == B.DSA3D_OK else ptrs(1)[0]) == (
        B.DSA3D_ERR_NULL_POINTER if status == B.DSA3D_OK else status)


def test_conv_bad_dtype_and_null_pointers():
    d = good_conv()
    d.dtype = 5
    assert conv_fwd(d) == B.DSA3D_ERR_UNSUPPORTED
    assert dsa.dsa3d_dwconv3d_forward(None, *ptrs(4), stream=0, check=False) == \
        B.DSA3D_ERR_NULL_POINTER
    d = good_conv()
    for name in ["x", "weight", "y"]:
        assert conv_fwd(d, **{name: None}) == B.DSA3D_ERR_NULL_POINTER, name
    for name in ["x", "weight", "dy"]:
        assert conv_bwd(d, **{name: None}) == B.DSA3D_ERR_NULL_POINTER, name
    assert conv_bwd(d, dx=None, dweight=None, dbias=None) == B.DSA3D_ERR_NULL_POINTER


def test_conv_alignment_and_aliasing():
    d = good_conv()
    far = ptrs(16)[15]
    assert conv_fwd(d, x=far + 4) == B.DSA3D_ERR_MISALIGNED      # fp32 pair needs 8 bytes
    # bf16 needs only 4 bytes: with a NULL weight the call stops at the pointer check instead
    assert conv_fwd(good_conv(dtype="bf16"), x=far + 4, weight=None) == B.DSA3D_ERR_NULL_POINTER
    assert conv_fwd(good_conv(dtype="bf16"), y=far + 2) == B.DSA3D_ERR_MISALIGNED
    assert conv_fwd(d, weight=far + 2) == B.DSA3D_ERR_MISALIGNED
    assert conv_bwd(d, dx=far + 4) == B.DSA3D_ERR_MISALIGNED
    assert conv_bwd(d, workspace=far + 128) == B.DSA3D_ERR_MISALIGNED
    x = ptrs(1)[0]
    assert conv_fwd(d, y=x) == B.DSA3D_ERR_ALIAS
    assert conv_fwd(d, y=x + 64) == B.DSA3D_ERR_ALIAS
    names = ptrs(7)
    assert conv_bwd(d, dweight=names[3]) == B.DSA3D_ERR_ALIAS     # dweight == dx
    assert conv_bwd(d, dx=names[2]) == B.DSA3D_ERR_ALIAS          # dx == dy
    assert conv_bwd(d, workspace=names[5]) == B.DSA3D_ERR_ALIAS   # workspace == dbias


def test_conv_workspace_size_and_errors():
    for kw in (dict(), dict(B=2, T=7, H=300, W=9, C=258, kt=5, kh=1, kw=7),
               dict(T=2, H=3, W=9, C=4000, kt=3)):
        d = good_conv(**kw)
        chunks = -(-d.channels // 128)
        strips = -(-d.width // 8)
        sg = min(strips, 5)
        tiles_per_bc = -(-strips // sg) * sg * d.frames * -(-d.height // 4)
        blocks = min(max(768 // (chunks * d.kt), 1), d.batch * tiles_per_bc)
        taps = d.kt * d.kh * d.kw
        slots = blocks * 4
        r256 = lambda n: -(-n // 256) * 256
        assert dsa.dsa3d_dwconv3d_backward_workspace_size(d) == \
            r256(slots * d.channels * taps * 4) + r256(slots * d.channels * 4)
    assert dsa.dsa3d_dwconv3d_backward_workspace_size(good_conv(kt=2)) == 0
    d = good_conv()
    need = dsa.dsa3d_dwconv3d_backward_workspace_size(d)
    assert conv_bwd(d, workspace=None) == B.DSA3D_ERR_WORKSPACE
    assert conv_bwd(d, workspace_bytes=need - 1) == B.DSA3D_ERR_WORKSPACE
    # dx alone needs no workspace: the call passes validation up to the (absent) device,
    # so only check that the workspace is not what fails
    assert conv_bwd(d, workspace=None, dweight=None, dbias=None, dx=None) == \
        B.DSA3D_ERR_NULL_POINTER



# ----------------------------------------------------------------------------- predicted weights

def pw_fwd(desc, **over):
    lg, v, off, out, lse = ptrs(5)
    args = dict(logits=lg, v=v, offsets=off, out=out, lse=lse)
    args.update(over)
    return dsa.dsa3d_pw_forward(desc, args["logits"], args["v"], args["offsets"], args["out"],
                                args["lse"], stream=0, check=False)


def pw_bwd(desc, **over):
    names = ["logits", "v", "offsets", "lse", "dout", "dlogits", "dv", "d_offsets", "workspace"]
    args = dict(zip(names, ptrs(len(names))))
    args["workspace_bytes"] = 1 << 33
    args.update(over)
    return dsa.dsa3d_pw_backward(desc, *[args[n] for n in names[:-1]], workspace=args["workspace"],
                                 workspace_bytes=args["workspace_bytes"], stream=0, check=False)


def test_pw_validation():
    d = good_desc()
    assert pw_fwd(good_desc(kt=2)) == B.DSA3D_ERR_INVALID_SHAPE
    assert pw_fwd(good_desc(scale=0.5)) == B.DSA3D_ERR_INVALID_SHAPE   # logits are used as given
    assert pw_fwd(good_desc(scale=1.0), logits=None) == B.DSA3D_ERR_NULL_POINTER
    for name in ["logits", "v", "offsets", "out"]:
        assert pw_fwd(d, **{name: None}) == B.DSA3D_ERR_NULL_POINTER, name
    far = ptrs(16)[15]
    assert pw_fwd(d, v=far + 8) == B.DSA3D_ERR_MISALIGNED
    assert pw_fwd(d, logits=far + 2) == B.DSA3D_ERR_MISALIGNED
    assert pw_fwd(d, out=ptrs(1)[0] + 256) == B.DSA3D_ERR_ALIAS        # out inside logits
    for name in ["logits", "v", "offsets", "lse", "dout", "dlogits", "dv", "d_offsets"]:
        assert pw_bwd(d, **{name: None}) == B.DSA3D_ERR_NULL_POINTER, name
    names = ptrs(9)
    assert pw_bwd(d, dv=names[5]) == B.DSA3D_ERR_ALIAS                 # dv == dlogits
    assert pw_bwd(d, workspace=None) == B.DSA3D_ERR_WORKSPACE
    assert pw_bwd(d, workspace=far + 128) == B.DSA3D_ERR_MISALIGNED
    assert pw_bwd(d, dlogits=far + 2) == B.DSA3D_ERR_MISALIGNED


def test_pw_workspace_is_the_backward_binning():
    for kw in (dict(), dict(B=2, T=5, H=7, W=9, heads=3, kt=3, kh=5, kw=5)):
        d = good_desc(**kw)
        assert dsa.dsa3d_pw_backward_workspace_size(d) == dsa.dsa3d_backward_workspace_size(d) > 0
    assert dsa.dsa3d_pw_backward_workspace_size(good_desc(scale=2.0)) == 0


# ----------------------------------------------------------------------------- window attention

def good_win(**over):
    kw = dict(B=1, T=6, H=20, W=24, heads=2, head_dim=64, window=(3, 16, 16), shift=(1, 8, 8))
    kw.update(over)
    return dsa.make_win_desc(kw["B"], kw["T"], kw["H"], kw["W"], kw["heads"], kw["head_dim"],
                             kw["window"], kw["shift"], kw.get("dtype", "bf16"), kw.get("scale", 0.0))


def win_fwd(desc, **over):
    q, k, v, out, res, lse = ptrs(6)
    args = dict(q=q, k=k, v=v, out=out, out_res=res, lse=lse)
    args.update(over)
    return dsa.dsa3d_win_forward(desc, args["q"], args["k"], args["v"], args["out"],
                                 args["out_res"], args["lse"], stream=0, check=False)


def win_bwd(desc, **over):
    names = ["q", "k", "v", "out", "out_res", "lse", "dout", "dq", "dk", "dv", "workspace"]
    args = dict(zip(names, ptrs(len(names))))
    args["workspace_bytes"] = 1 << 33
    args.update(over)
    return dsa.dsa3d_win_backward(desc, *[args[n] for n in names[:-1]], workspace=args["workspace"],
                                  workspace_bytes=args["workspace_bytes"], stream=0, check=False)


def test_win_desc_layout_matches_header():
    # 12 int32 dims + float scale + enum dtype
    assert ctypes.sizeof(B.dsa3d_win_desc) == 14 * 4


@pytest.mark.parametrize("over,status", [
    (dict(T=0), B.DSA3D_ERR_INVALID_SHAPE),
    (dict(heads=0), B.DSA3D_ERR_INVALID_SHAPE),
    (dict(window=(0, 16, 16)), B.DSA3D_ERR_INVALID_SHAPE),
    (dict(shift=(3, 8, 8)), B.DSA3D_ERR_INVALID_SHAPE),      # shift must be below the window
    (dict(shift=(-1, 0, 0)), B.DSA3D_ERR_INVALID_SHAPE),
    (dict(scale=-1.0), B.DSA3D_ERR_INVALID_SHAPE),
    (dict(scale=float("nan")), B.DSA3D_ERR_INVALID_SHAPE),
    (dict(window=(2, 256, 256), shift=(0, 0, 0)), B.DSA3D_ERR_INVALID_SHAPE),  # > 65536 tokens
    (dict(B=1 << 12, T=1 << 10, H=1 << 5, W=1 << 4, heads=1), B.DSA3D_ERR_INVALID_SHAPE),  # 2^31 rows
    (dict(W=1 << 24, H=1, T=1), B.DSA3D_ERR_INVALID_SHAPE),
    (dict(dtype="f32"), B.DSA3D_ERR_UNSUPPORTED),
    (dict(head_dim=32), B.DSA3D_ERR_UNSUPPORTED),
    (dict(head_dim=96), B.DSA3D_ERR_UNSUPPORTED),
])
def test_win_descriptor_errors(over, status):
    d = good_win(**over)
    assert win_fwd(d) == status
    assert win_bwd(d) == status
    assert dsa.dsa3d_win_backward_workspace_size(d) == 0


def test_win_pointer_checks():
    d = good_win()
    assert win_fwd(None) == B.DSA3D_ERR_NULL_POINTER
    for name in ["q", "k", "v", "out"]:
        assert win_fwd(d, **{name: None}) == B.DSA3D_ERR_NULL_POINTER, name
    for name in ["q", "k", "v", "out", "lse", "dout", "dq", "dk", "dv"]:
        assert win_bwd(d, **{name: None}) == B.DSA3D_ERR_NULL_POINTER, name
    far = ptrs(16)[15]
    for name in ["q", "k", "v", "out", "out_res"]:
        assert win_fwd(d, **{name: far + 8}) == B.DSA3D_ERR_MISALIGNED, name
    assert win_fwd(d, lse=far + 2) == B.DSA3D_ERR_MISALIGNED
    for name in ["out_res", "dout", "dq", "dk", "dv"]:
        assert win_bwd(d, **{name: far + 8}) == B.DSA3D_ERR_MISALIGNED, name
    assert win_bwd(d, workspace=far + 128) == B.DSA3D_ERR_MISALIGNED
    f = ptrs(6)
    assert win_fwd(d, out=f[0] + 256) == B.DSA3D_ERR_ALIAS               # out inside q
    assert win_fwd(d, lse=f[3] + 64) == B.DSA3D_ERR_ALIAS                # lse inside out
    assert win_fwd(d, out_res=f[3]) == B.DSA3D_ERR_ALIAS                 # out_res == out
    assert win_fwd(d, out_res=f[1] + 16) == B.DSA3D_ERR_ALIAS            # out_res inside k
    names = ptrs(11)
    assert win_bwd(d, dk=names[7]) == B.DSA3D_ERR_ALIAS                  # dk == dq
    assert win_bwd(d, dv=names[6]) == B.DSA3D_ERR_ALIAS                  # dv == dout
    assert win_bwd(d, dq=names[4]) == B.DSA3D_ERR_ALIAS                  # dq == out_res
    assert win_bwd(d, workspace=names[9]) == B.DSA3D_ERR_ALIAS           # workspace == dv


def test_win_workspace_size_and_errors():
    for over in (dict(), dict(B=2, T=5, H=7, W=9, heads=3, head_dim=128, window=(2, 3, 5),
                                 shift=(1, 1, 2))):
        d = good_win(**over)
        rows = d.batch * d.frames * d.height * d.width * d.heads
        assert dsa.dsa3d_win_backward_workspace_size(d) == -(-rows * 4 // 256) * 256
    d = good_win()
    need = dsa.dsa3d_win_backward_workspace_size(d)
    assert win_bwd(d, workspace=None) == B.DSA3D_ERR_WORKSPACE
    assert win_bwd(d, workspace_bytes=need - 1) == B.DSA3D_ERR_WORKSPACE


def test_gather_probe_library_exports_its_entry_point():
    """The gather microbenchmark bench.py reports its ceiling from is built beside bench.py
    (not into the library) and exports its one C entry point (running it needs a GPU)."""
    import os
    lib = os.path.join(os.path.dirname(INCLUDE), "libgather_probe.so")
    assert os.path.exists(lib), lib
    assert hasattr(ctypes.CDLL(lib), "dsa3d_probe_gather")
