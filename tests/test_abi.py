"""C-ABI tests that need no GPU: the library loads, exports every entry point
declared in include/flex.h, and rejects invalid arguments with a status code
before any device work."""
import ctypes
import os
import re

import pytest

import paper_2606_27748_amd as F

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "flex.h")

# Fake, 16-byte aligned, never dereferenced pointers: every call below must be
# rejected by validation before any launch.  They are only used where no GPU
# is visible, so a validation bug cannot turn into a device access.
FAKE = ctypes.c_void_p(0x10000)
NO_GPU = not os.path.exists("/dev/kfd")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(flex_[a-z_]+)\s*\(", text)))


def test_exports_match_header():
    lib = F.load()
    names = declared_functions()
    assert set(names) == set(F.EXPORTS), names
    for n in names:
        assert hasattr(lib, n), n
    assert lib.flex_abi_version() == 7


def test_status_strings():
    for s in range(5):
        assert F.status_string(s)
    assert F.status_string(99) == "unknown status"


def _ws(desc, p=F.FLEX_PASS_FWD):
    n = ctypes.c_size_t(123)
    st = F.load().flex_workspace_size(ctypes.byref(desc) if desc is not None else None, p,
                                      ctypes.byref(n))
    return st, n.value


def test_workspace_size():
    d = F.make_desc(2, 16, 8192, 64, 128, "nonstationary", True, "bf16")
    st, n = _ws(d)
    assert st == F.FLEX_OK and n > 0
    st, nb = _ws(d, F.FLEX_PASS_BWD)
    assert st == F.FLEX_OK and nb > n
    st, n0 = _ws(d, F.FLEX_PASS_FEATURE_MAP)
    assert st == F.FLEX_OK and n0 == 0
    assert _ws(None)[0] == F.FLEX_ERR_INVALID_ARG
    assert _ws(d, 7)[0] == F.FLEX_ERR_INVALID_ARG
    # d = 128, m = 256 runs as frequency groups; both passes have a workspace
    d5 = F.make_desc(2, 16, 8192, 128, 256, "nonstationary", True, "bf16")
    assert _ws(d5)[0] == F.FLEX_OK and _ws(d5, F.FLEX_PASS_BWD)[0] == F.FLEX_OK
    # an unsupported shape is reported for both passes
    d6 = F.make_desc(2, 16, 8192, 96, 128, "nonstationary", True, "bf16")
    assert _ws(d6)[0] == F.FLEX_ERR_UNSUPPORTED and _ws(d6, F.FLEX_PASS_BWD)[0] == F.FLEX_ERR_UNSUPPORTED


@pytest.mark.parametrize("io,d,m,ok", [
    ("bf16", 32, 128, True), ("bf16", 32, 256, True), ("bf16", 64, 192, True), ("bf16", 64, 256, True),
    ("bf16", 128, 64, True), ("bf16", 128, 192, True), ("f32", 32, 256, True),
    ("bf16", 64, 96, True), ("bf16", 64, 16, True), ("bf16", 128, 208, True), ("f32", 32, 48, True),
    ("bf16", 64, 320, False), ("bf16", 64, 40, False), ("bf16", 64, 0, False), ("f32", 64, 64, False),
])
def test_attention_shape_set(io, d, m, ok):
    """The attention passes and the standalone feature map take d in
    {32, 64, 128} (fp32: 32) and m a multiple of 16 up to 256 (frequency groups
    or slices where no one kernel covers the shape)."""
    want = F.FLEX_OK if ok else (F.FLEX_ERR_INVALID_ARG if m <= 0 else F.FLEX_ERR_UNSUPPORTED)
    dd = F.make_desc(1, 2, 100, d, m, "nonstationary", True, io)
    assert _ws(dd)[0] == want and _ws(dd, F.FLEX_PASS_BWD)[0] == want
    if m > 0:
        assert _ws(dd, F.FLEX_PASS_FEATURE_MAP)[0] == (F.FLEX_OK if ok else F.FLEX_ERR_UNSUPPORTED)


def test_padded_group_workspace():
    """A last frequency group that 64 does not fill adds its zero-padded rows
    of W1 and W2 to both workspaces."""
    full = F.make_desc(1, 4, 1000, 64, 64, "nonstationary", True, "bf16")
    part = F.make_desc(1, 4, 1000, 64, 48, "nonstationary", True, "bf16")
    pad = 2 * 4 * 64 * 64 * 4
    for p in (F.FLEX_PASS_FWD, F.FLEX_PASS_BWD):
        assert _ws(part, p)[1] == _ws(full, p)[1] + pad


def test_awd_workspace_size():
    """The distillation loss pass: non-causal only, its own shape set."""
    d = F.make_desc(32, 8, 512, 64, 64, "nonstationary", False, "bf16")
    st, n = _ws(d, F.FLEX_PASS_AWD)
    assert st == F.FLEX_OK
    # at least the two feature blocks and the two feature gradients (bf16)
    assert n >= 32 * 8 * 512 * 128 * (2 + 2 + 2 + 2)
    dc = F.make_desc(32, 8, 512, 64, 64, "nonstationary", True, "bf16")
    assert _ws(dc, F.FLEX_PASS_AWD)[0] == F.FLEX_ERR_UNSUPPORTED
    d5 = F.make_desc(2, 16, 8192, 128, 256, "nonstationary", False, "bf16")
    assert _ws(d5, F.FLEX_PASS_AWD)[0] == F.FLEX_ERR_UNSUPPORTED
    df = F.make_desc(2, 2, 100, 32, 64, "stationary", False, "f32")
    assert _ws(df, F.FLEX_PASS_AWD)[0] == F.FLEX_OK


@pytest.mark.parametrize("field,value,status", [
    ("B", 0, F.FLEX_ERR_INVALID_ARG), ("N", -1, F.FLEX_ERR_INVALID_ARG),
    ("variant", 2, F.FLEX_ERR_INVALID_ARG), ("causal", 3, F.FLEX_ERR_INVALID_ARG),
    ("io_dtype", 5, F.FLEX_ERR_INVALID_ARG), ("sigma", 0.0, F.FLEX_ERR_INVALID_ARG),
    ("sigma", float("nan"), F.FLEX_ERR_INVALID_ARG), ("chunk", 48, F.FLEX_ERR_UNSUPPORTED),
    ("chunk", 128, F.FLEX_ERR_UNSUPPORTED), ("chunk", 8, F.FLEX_ERR_UNSUPPORTED),
    ("chunk", -16, F.FLEX_ERR_INVALID_ARG), ("chunk", 16, F.FLEX_OK), ("chunk", 32, F.FLEX_OK),
    ("chunk", 64, F.FLEX_OK),
    ("d", 48, F.FLEX_ERR_UNSUPPORTED), ("m", 100, F.FLEX_ERR_UNSUPPORTED), ("m", 96, F.FLEX_OK),
    ("dv", 32, F.FLEX_OK), ("dv", 128, F.FLEX_OK), ("dv", 48, F.FLEX_ERR_UNSUPPORTED),
    ("dv", 256, F.FLEX_ERR_UNSUPPORTED), ("grad_dtype", 1, F.FLEX_ERR_UNSUPPORTED),
])
def test_descriptor_validation(field, value, status):
    d = F.make_desc(1, 2, 100, 64, 128, "nonstationary", True, "bf16")
    setattr(d, field, value)
    assert _ws(d)[0] == status


@pytest.mark.parametrize("field,value", [("dv", 0), ("dv", 48), ("causal", 7), ("chunk", 48),
                                         ("segments", -1), ("grad_dtype", 9)])
def test_feature_map_ignores_attention_fields(field, value):
    """The feature map has no values, mask, chunks, segments or gradients: it
    accepts any value of those descriptor fields (its workspace is empty)."""
    d = F.make_desc(1, 2, 100, 64, 128, "nonstationary", True, "bf16")
    setattr(d, field, value)
    assert _ws(d, F.FLEX_PASS_FEATURE_MAP) == (F.FLEX_OK, 0)
    d.d = 48   # the shape itself is still checked
    assert _ws(d, F.FLEX_PASS_FEATURE_MAP)[0] == F.FLEX_ERR_UNSUPPORTED


@pytest.mark.parametrize("d,dv", [(64, 32), (128, 64), (128, 32), (32, 64), (64, 128), (32, 128)])
def test_value_width_workspace(d, dv):
    """d_v != d runs at width max(d, d_v) on zero-padded copies: its workspace
    is the padded shape's plus the copies (Q, K, W and their gradients when
    d_v > d; V, O, dO and dV when d_v < d)."""
    for causal in (False, True):
        for variant in ("stationary", "nonstationary"):
            desc = F.make_desc(2, 3, 300, d, 128, variant, causal, "bf16", dv=dv)
            w = max(d, dv)
            pad = F.make_desc(2, 3, 300, w, 128, variant, causal, "bf16")
            rows, hm = 2 * 3 * 300, 3 * 128
            nmat = 2 if variant == "nonstationary" else 1
            for pas in (F.FLEX_PASS_FWD, F.FLEX_PASS_BWD):
                st, n = _ws(desc, pas)
                st0, n0 = _ws(pad, pas)
                assert st == F.FLEX_OK and st0 == F.FLEX_OK
                if dv > d:
                    copies = 2 * rows * w * 2 + nmat * hm * w * 4
                    if pas == F.FLEX_PASS_BWD:
                        copies += 2 * rows * w * 4 + nmat * hm * w * 4
                else:
                    copies = 2 * rows * w * 2
                    if pas == F.FLEX_PASS_BWD:
                        copies += rows * w * 2 + rows * w * 4
                assert n0 + copies <= n <= n0 + copies + 256 * 8


def test_value_width_limits():
    """fp32 has d = d_v = 32 only, and d_v is one of the head widths."""
    assert _ws(F.make_desc(1, 1, 64, 32, 64, "stationary", True, "f32", dv=64))[0] == F.FLEX_ERR_UNSUPPORTED
    assert _ws(F.make_desc(1, 1, 64, 64, 64, "stationary", True, "bf16", dv=48))[0] == F.FLEX_ERR_UNSUPPORTED


def test_fp32_large_shapes_unsupported():
    d = F.make_desc(1, 1, 64, 64, 128, "stationary", False, "f32")
    assert _ws(d)[0] == F.FLEX_ERR_UNSUPPORTED


@pytest.mark.skipif(not NO_GPU, reason="fake pointers are only passed where no GPU is visible")
def test_entry_points_reject_bad_arguments():
    lib = F.load()
    dn = F.make_desc(1, 2, 100, 64, 128, "nonstationary", True, "bf16")
    ds = F.make_desc(1, 2, 100, 64, 128, "stationary", True, "bf16")
    P = FAKE
    big = ctypes.c_size_t(1 << 40)
    # NULL descriptor / pointers
    assert lib.flex_linattn_fwd(None, P, P, P, P, P, P, P, P, P, big, None) == F.FLEX_ERR_INVALID_ARG
    assert lib.flex_linattn_fwd(ctypes.byref(dn), None, P, P, P, P, P, P, P, P, big, None) == 1
    # W2 must be given exactly for the nonstationary variant
    assert lib.flex_linattn_fwd(ctypes.byref(dn), P, P, P, P, None, P, P, P, P, big, None) == 1
    assert lib.flex_linattn_fwd(ctypes.byref(ds), P, P, P, P, P, P, P, P, P, big, None) == 1
    # misaligned pointer
    assert lib.flex_linattn_fwd(ctypes.byref(dn), ctypes.c_void_p(0x10002), P, P, P, P, P, P, P,
                                P, big, None) == 1
    # workspace missing or too small
    assert lib.flex_linattn_fwd(ctypes.byref(dn), P, P, P, P, P, P, P, P, None, big, None) == 3
    assert lib.flex_linattn_fwd(ctypes.byref(dn), P, P, P, P, P, P, P, P, P, 16, None) == 3
    # backward: den, dO and dW2 are required, dW2 must be NULL for stationary
    args = [P] * 15
    nofwd = [None, 0]
    a = list(args); a[7] = None  # den
    assert lib.flex_linattn_bwd(ctypes.byref(dn), *a, *nofwd, P, 16, None) == 1
    a = list(args); a[13] = None  # dW2 missing for nonstationary
    assert lib.flex_linattn_bwd(ctypes.byref(dn), *a, *nofwd, P, big, None) == 1
    a = list(args); a[4] = None  # W2 NULL, stationary, but dW2 given
    assert lib.flex_linattn_bwd(ctypes.byref(ds), *a, *nofwd, P, big, None) == 1
    assert lib.flex_linattn_bwd(ctypes.byref(dn), *args, *nofwd, P, 16, None) == F.FLEX_ERR_WORKSPACE
    # a forward workspace smaller than the forward needs
    assert lib.flex_linattn_bwd(ctypes.byref(dn), *args, P, 16, P, big, None) == F.FLEX_ERR_WORKSPACE
    # the forward without a workspace: the same argument checks, and a forward
    # workspace beyond the static scratch is refused before any device work
    assert lib.flex_linattn_fwd_noalloc(None, P, P, P, P, P, P, P, P, None) == F.FLEX_ERR_INVALID_ARG
    assert lib.flex_linattn_fwd_noalloc(ctypes.byref(dn), P, P, P, P, None, P, P, P, None) == 1
    assert lib.flex_linattn_fwd_noalloc(ctypes.byref(ds), P, P, P, P, P, P, P, P, None) == 1
    d5 = F.make_desc(2, 16, 8192, 128, 256, "nonstationary", True, "bf16")
    assert lib.flex_linattn_fwd_noalloc(ctypes.byref(d5), P, P, P, P, P, P, P, P, None) == 3
    # prefill: causal only, state required, workspace checked
    nc = F.make_desc(1, 2, 100, 64, 128, "nonstationary", False, "bf16")
    assert lib.flex_linattn_prefill(ctypes.byref(nc), P, P, P, P, P, P, P, P, P, P, big, None) == 2
    assert lib.flex_linattn_prefill(ctypes.byref(dn), P, P, P, P, P, P, P, P, None, P, big, None) == 1
    assert lib.flex_linattn_prefill(ctypes.byref(dn), P, P, P, P, P, P, P, P, P, P, 16, None) == 3
    # feature map
    assert lib.flex_feature_map(ctypes.byref(dn), None, P, P, P, P, None, 0, None) == 1
    assert lib.flex_feature_map(ctypes.byref(ds), P, P, P, P, P, None, 0, None) == 1
    # distillation loss: loss is required, W2 matches the variant, dW2 is
    # required with gradients of the nonstationary variant, non-causal only,
    # and the workspace is checked
    an = F.make_desc(1, 2, 100, 64, 128, "nonstationary", False, "bf16")
    ast = F.make_desc(1, 2, 100, 64, 128, "stationary", False, "bf16")
    assert lib.flex_awd_loss(ctypes.byref(an), P, P, P, P, P, None, P, P, P, P, big, None) == 1
    assert lib.flex_awd_loss(ctypes.byref(an), P, P, P, None, P, P, P, P, P, P, big, None) == 1
    assert lib.flex_awd_loss(ctypes.byref(ast), P, P, P, P, P, P, P, None, P, P, big, None) == 1
    assert lib.flex_awd_loss(ctypes.byref(an), P, P, P, P, P, P, P, None, P, P, big, None) == 1
    assert lib.flex_awd_loss(ctypes.byref(dn), P, P, P, P, P, P, P, P, P, P, big, None) == 2
    assert lib.flex_awd_loss(ctypes.byref(an), P, P, P, P, P, P, P, P, P, P, 16, None) == 3
    assert lib.flex_awd_loss(ctypes.byref(an), P, P, P, P, P, P, None, None, None, None, big, None) == 3
