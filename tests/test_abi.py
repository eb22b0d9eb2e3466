"""C-ABI checks that need no GPU: the library loads, exports every declared
function, sizes workspaces, and rejects bad arguments before any launch."""

import ctypes

import pytest

from paper_2607_14530_amd import xhc as X


def test_binding_signatures_match_header():
    """Each bound function passes as many arguments as the header declares."""
    import re
    text = re.sub(r"/\*.*?\*/", "", open(X.HEADER).read(), flags=re.S)
    for name, (_, args) in X._SIGS.items():
        m = re.search(name + r"\s*\(([^;]*)\)\s*;", text)
        assert m, name
        params = [a for a in m.group(1).split(",") if a.strip() and a.strip() != "void"]
        assert len(params) == len(args), (name, len(params), len(args))


def test_library_exports_every_declared_symbol():
    L = X.lib()
    names = X.declared_functions()
    assert "xhc_pre" in names and "xhc_post" in names
    for n in names:
        assert hasattr(L, n), n


def test_packed_and_workspace_sizes():
    d = X.make_dims(T=16384, N=16, k=4, m=2, C=4096, Kr=4, S=8192)
    # 65536 rows x 32 columns of bf16 in 1 KiB fragments, plus column sums
    assert X.xhc_packed_full_bytes(d, 1) == 65536 // 32 * 2 * 1024 + 256
    # [W_post | W_res] = 16 + 16 columns over 4 * 4096 rows
    assert X.xhc_packed_active_bytes(d, 4, 1) == 16384 // 32 * 2 * 1024
    assert X.xhc_workspace_bytes(d, X.XHC_OP_PRE) > 0
    assert X.xhc_workspace_bytes(d, X.XHC_OP_POST) > 0
    d1 = X.make_dims(T=64, N=4, k=4, m=4, C=256, Kr=1)
    assert X.xhc_workspace_bytes(d1, X.XHC_OP_POST) == 0


FAKE = 1 << 20  # a 16-byte aligned non-null address; never dereferenced below


def _pre_status(d, ws_bytes=1 << 40, null_at=None):
    ptrs = [FAKE] * 13 + [None, FAKE]      # saved (14th) is optional
    if null_at is not None:
        ptrs[null_at if null_at < 13 else 14] = None
    return X.lib().xhc_pre(ctypes.byref(d), *ptrs, ws_bytes, None)


def _post_status(d, conv=True, ws_bytes=1 << 40, F=FAKE + 4096):
    return X.lib().xhc_post(ctypes.byref(d), FAKE, F, FAKE if conv else None, FAKE, FAKE, FAKE, FAKE, None,
                            FAKE, ws_bytes, None)


@pytest.mark.parametrize("kw,status", [
    (dict(k=5, N=4), X.XHC_EINVAL),          # k > N
    (dict(m=5), X.XHC_EINVAL),               # m > k
    (dict(T=100, S=30), X.XHC_EINVAL),       # T % S != 0
    (dict(C=48), X.XHC_EUNSUPPORTED),        # C % 32 != 0
    (dict(N=65, k=4), X.XHC_EUNSUPPORTED),   # N above the supported maximum
    (dict(k=9, N=16), X.XHC_EUNSUPPORTED),   # k above the supported maximum
    (dict(Kr=5), X.XHC_EUNSUPPORTED),
    (dict(eps=0.0), X.XHC_EINVAL),
])
def test_invalid_dims_rejected_before_launch(kw, status):
    base = dict(T=64, N=16, k=4, m=2, C=256, Kr=1, S=64)
    base.update(kw)
    d = X.make_dims(**base)
    assert _pre_status(d) == status
    assert _post_status(d, conv=False) == status


def test_unknown_router_rejected():
    d = X.make_dims(T=64, N=16, k=4, m=2, C=256, Kr=1, S=64)
    d.router = 2
    assert _pre_status(d) == X.XHC_EINVAL


def test_dims_struct_fields_match_header():
    """The binding's xhc_dims fields follow the header's, in order."""
    import re
    text = re.sub(r"/\*.*?\*/", "", open(X.HEADER).read(), flags=re.S)
    body = re.search(r"typedef struct xhc_dims \{(.*?)\} xhc_dims;", text, flags=re.S).group(1)
    names = re.findall(r"\b(\w+)\s*(?:\[\d+\])?\s*;", body)
    assert names == [f[0] for f in X.Dims._fields_]


def test_null_pointer_and_workspace_errors():
    d = X.make_dims(T=64, N=16, k=4, m=2, C=256, Kr=1)
    for i in range(14):
        assert _pre_status(d, null_at=i) == X.XHC_EINVAL, i
    assert _pre_status(d, ws_bytes=16) == X.XHC_EWORKSPACE
    d4 = X.make_dims(T=64, N=16, k=4, m=2, C=256, Kr=4)
    assert _post_status(d4, conv=False) == X.XHC_EINVAL      # conv_w required when Kr > 1
    assert _post_status(d, conv=True) == X.XHC_EINVAL        # and forbidden when Kr == 1
    assert _post_status(d4, ws_bytes=16) == X.XHC_EWORKSPACE
    assert _post_status(d, conv=False, F=FAKE) == X.XHC_EINVAL   # F aliasing X


def test_misaligned_pointers_rejected():
    d = X.make_dims(T=64, N=16, k=4, m=2, C=256, Kr=1)
    ptrs = [FAKE] * 13 + [None, FAKE]
    ptrs[0] = FAKE + 2
    assert X.lib().xhc_pre(ctypes.byref(d), *ptrs, 1 << 40, None) == X.XHC_EUNSUPPORTED


def test_empty_batch_is_a_no_op():
    d = X.make_dims(T=0, N=16, k=4, m=2, C=256, Kr=1, S=1)
    assert _pre_status(d) == X.XHC_OK
    assert _post_status(d, conv=False) == X.XHC_OK


def test_forced_fused_path_rejects_uncovered_shapes():
    d = X.make_dims(T=64, N=8, k=4, m=2, C=256, Kr=1, impl=X.XHC_IMPL_FUSED)
    assert _pre_status(d) == X.XHC_EUNSUPPORTED
    d = X.make_dims(T=64, N=16, k=4, m=2, C=96, Kr=1, impl=X.XHC_IMPL_FUSED)
    assert _pre_status(d) == X.XHC_EUNSUPPORTED
    d = X.make_dims(T=64, N=16, k=4, m=2, C=256, Kr=1, impl=7)
    assert _pre_status(d) == X.XHC_EINVAL


def test_post_noalloc_rejects_shapes_beyond_its_scratch_before_any_work():
    """xhc_post_noalloc refuses a shape whose scratch exceeds the static array
    (XHC_NOALLOC_SCRATCH_BYTES) before touching any pointer or the device."""
    d = X.make_dims(1 << 20, 16, 4, 2, 4096, Kr=4, S=8192)
    assert X.xhc_workspace_bytes(d, X.XHC_OP_POST) > X.NOALLOC_SCRATCH_BYTES
    st = X.lib().xhc_post_noalloc(ctypes.byref(d), 16, 16, 16, 16, 16, 16, 16, None, None)
    assert st == X.XHC_EWORKSPACE
