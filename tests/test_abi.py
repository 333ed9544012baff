"""CPU checks of the C ABI: the library loads, exports every declared entry
point, and rejects bad arguments on the host before anything is launched.

Every call here fails validation by construction (the pointers are fake), so
none of them reaches a kernel launch.
"""

import ctypes
import os
import re

import pytest

# a missing or unloadable library fails this module (no skip): the binding
# raises ImportError when libmicromix.so is absent
from paper_2508_02343_amd import binding as b

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "micromix.h")


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(mm_[a-z_]+)\s*\(", text)))


def test_header_declares_the_calls():
    names = _declared_functions()
    for n in ("mm_quantize_act", "mm_quantize_weight", "mm_gemm", "mm_calibrate", "mm_calibrate_workspace_size", "mm_calibrate_no_alloc",
              "mm_rmsnorm_quantize_act",
              "mm_status_str", "mm_last_error", "mm_abi_version"):
        assert n in names


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(b.LIB_PATH)
    for n in _declared_functions():
        assert hasattr(lib, n), n
    assert b.lib.mm_abi_version() == 6


def test_status_strings():
    for code, name in b.STATUS_NAMES.items():
        assert b.lib.mm_status_str(code).decode() == name


FAKE = 0x10000  # 16-byte aligned, never dereferenced: validation fails first


def _tensor(rows=4, K=128, split=(64, 32, 32), ptr=FAKE):
    d = b.MMTensor()
    d.rows, d.K = rows, K
    d.split = b.MMSplit(*split)
    for name, p in zip(("q4", "q6", "q8"), split):
        setattr(d, name, ptr if p else None)
    d.sc = ptr
    return d


def _q(d, x=FAKE, ldx=None, perm=FAKE):
    return b.lib.mm_quantize_act(ctypes.c_void_p(x), ldx if ldx is not None else d.K, ctypes.c_void_p(perm),
                                 ctypes.byref(d), None)


@pytest.mark.parametrize(
    "mutate,expect",
    [
        (lambda d: setattr(d, "split", b.MMSplit(64, 16, 48)), "MM_ERR_SPLIT"),
        (lambda d: setattr(d, "split", b.MMSplit(64, 32, 64)), "MM_ERR_SPLIT"),
        (lambda d: setattr(d, "split", b.MMSplit(-32, 96, 64)), "MM_ERR_SPLIT"),
        (lambda d: setattr(d, "K", 100), "MM_ERR_SHAPE"),
        (lambda d: setattr(d, "rows", 0), "MM_ERR_SHAPE"),
        (lambda d: setattr(d, "q4", None), "MM_ERR_NULL"),
        (lambda d: setattr(d, "sc", None), "MM_ERR_NULL"),
        (lambda d: setattr(d, "q6", FAKE + 8), "MM_ERR_ALIGN"),
        (lambda d: setattr(d, "sc", FAKE + 4), "MM_ERR_ALIGN"),
        (lambda d: setattr(d, "formats", b.MMFormats(2, 0)), "MM_ERR_FORMAT"),
        (lambda d: setattr(d, "formats", b.MMFormats(0, -1)), "MM_ERR_FORMAT"),
    ],
)
def test_quantize_rejects_bad_descriptors(mutate, expect):
    d = _tensor()
    mutate(d)
    st = _q(d)
    assert b.STATUS_NAMES[st] == expect, b.lib.mm_last_error()
    assert b.lib.mm_last_error().decode()


def test_quantize_rejects_bad_inputs():
    d = _tensor()
    assert b.STATUS_NAMES[_q(d, x=0)] == "MM_ERR_NULL"
    assert b.STATUS_NAMES[_q(d, perm=0)] == "MM_ERR_NULL"
    assert b.STATUS_NAMES[_q(d, ldx=64)] == "MM_ERR_SHAPE"
    assert b.STATUS_NAMES[_q(d, ldx=132)] == "MM_ERR_ALIGN"
    assert b.STATUS_NAMES[_q(d, x=FAKE + 2)] == "MM_ERR_ALIGN"
    assert b.STATUS_NAMES[_q(d, perm=FAKE + 4)] == "MM_ERR_ALIGN"
    big = _tensor(K=65536, split=(65536, 0, 0))
    assert b.STATUS_NAMES[_q(big)] == "MM_ERR_SHAPE"
    assert b.STATUS_NAMES[b.lib.mm_quantize_act(None, 128, None, None, None)] == "MM_ERR_NULL"


def test_empty_groups_may_be_null_but_rest_is_checked():
    d = _tensor(split=(128, 0, 0))
    assert d.q6 is None and d.q8 is None
    d.q4 = FAKE + 8  # misaligned: proves validation still runs
    assert b.STATUS_NAMES[_q(d)] == "MM_ERR_ALIGN"


def _g(a, w, y=FAKE, ldy=None):
    return b.lib.mm_gemm(ctypes.byref(a), ctypes.byref(w), ctypes.c_void_p(y),
                         ldy if ldy is not None else w.rows, None)


def test_gemm_rejects_mismatched_operands():
    a, w = _tensor(rows=8), _tensor(rows=16, K=160, split=(64, 32, 64))
    assert b.STATUS_NAMES[_g(a, w)] == "MM_ERR_SHAPE"
    w = _tensor(rows=16, split=(32, 64, 32))
    assert b.STATUS_NAMES[_g(a, w)] == "MM_ERR_SHAPE"
    w = _tensor(rows=16)
    assert b.STATUS_NAMES[_g(a, w, y=0)] == "MM_ERR_NULL"
    assert b.STATUS_NAMES[_g(a, w, ldy=8)] == "MM_ERR_SHAPE"
    assert b.STATUS_NAMES[_g(a, w, ldy=20)] == "MM_ERR_ALIGN"
    assert b.STATUS_NAMES[_g(a, w, y=FAKE + 4)] == "MM_ERR_ALIGN"
    bad = _tensor(rows=8, split=(64, 32, 16))
    assert b.STATUS_NAMES[_g(bad, w)] == "MM_ERR_SPLIT"


@pytest.mark.parametrize("rows,K,split,want", [
    # rows padded to 32; steps of 4 blocks: E2M1 3 blocks -> 1 step, E3M2 5 -> 2, E4M3 3 -> 1
    (5, 352, (96, 160, 96), {"q4": 1 * 32 * 64, "q6": 2 * 32 * 96, "q8": 1 * 32 * 128, "sc": 4 * 32 * 4}),
    (33, 4096, (3072, 768, 256), {"q4": 24 * 64 * 64, "q6": 6 * 64 * 96, "q8": 2 * 64 * 128, "sc": 32 * 64 * 4}),
    (64, 64, (64, 0, 0), {"q4": 64 * 64, "q6": 0, "q8": 0, "sc": 64 * 4}),
])
def test_layout_sizes(rows, K, split, want):
    assert b.layout_sizes(rows, K, split) == want
    from tests import packed_layout as L

    assert L.geometry(rows, split)["bytes"] == [want[k] for k in ("q4", "q6", "q8", "sc")]


def test_layout_sizes_rejects_bad_shapes():
    with pytest.raises(b.MMError):
        b.layout_sizes(4, 96, (64, 16, 16))
    with pytest.raises(b.MMError):
        b.layout_sizes(0, 64, (64, 0, 0))
    assert b.lib.mm_mx_layout_sizes(4, 64, b.MMSplit(64, 0, 0), None) == 1


def test_binding_descriptor_fields():
    t = b.MXTensor.empty(5, 352, (96, 160, 96), device="cpu")
    d = t.descriptor()
    assert (d.rows, d.K, d.split.p4, d.split.p6, d.split.p8) == (5, 352, 96, 160, 96)
    assert d.q4 == t.q4.data_ptr() and d.q6 == t.q6.data_ptr() and d.q8 == t.q8.data_ptr()
    assert d.sc == t.sc.data_ptr()
    assert t.q4.numel() == 2048 and t.sc.numel() == 512
    e = b.MXTensor.empty(3, 64, (64, 0, 0), device="cpu").descriptor()
    assert e.q6 is None and e.q8 is None


def test_descriptor_layout_matches_the_header():
    """The ctypes mirror has the C struct's size and field offsets (checked
    against a C compiler's view of include/micromix.h)."""
    import subprocess
    import tempfile

    src = (f'#include "{HEADER}"\n#include <stddef.h>\n#include <stdio.h>\nint main(void) {{\n'
           'printf("%zu %zu %zu %zu %zu\\n", sizeof(mm_mx_tensor), offsetof(mm_mx_tensor, split),'
           ' offsetof(mm_mx_tensor, formats), offsetof(mm_mx_tensor, q4), offsetof(mm_mx_tensor, sc));\n'
           'return 0; }\n')
    with tempfile.TemporaryDirectory() as d:
        c = os.path.join(d, "t.c")
        open(c, "w").write(src)
        exe = os.path.join(d, "t")
        subprocess.run(["gcc", "-std=c99", "-o", exe, c], check=True)
        got = tuple(int(v) for v in subprocess.run([exe], check=True, capture_output=True, text=True).stdout.split())
    M = b.MMTensor
    assert got == (ctypes.sizeof(M), M.split.offset, M.formats.offset, M.q4.offset, M.sc.offset)


def test_gemm_rejects_mixed_formats():
    a, w = _tensor(), _tensor()
    w.formats = b.MMFormats(1, 0)
    st = b.lib.mm_gemm(ctypes.byref(a), ctypes.byref(w), ctypes.c_void_p(FAKE), 128, None)
    assert b.STATUS_NAMES[st] == "MM_ERR_FORMAT"


def _ws(rows, K):
    n = ctypes.c_int64(-1)
    st = b.lib.mm_calibrate_workspace_size(rows, K, ctypes.byref(n))
    return b.STATUS_NAMES[st], n.value


@pytest.mark.parametrize("rows,K", [(1, 32), (16, 32), (17, 4096), (2048, 4096), (4096, 14336), (8192, 32768),
                                    (100000, 512)])
def test_calibrate_workspace_size(rows, K):
    st, n = _ws(rows, K)
    assert st == "MM_OK"
    doubles, rem = divmod(n - 2048 - 4 * K * -(-K // 256), 8 * K)  # (chunks + 1) * K doubles: partial sums and means
    chunks = doubles - 1
    assert rem == 0 and 1 <= chunks <= 128
    assert chunks - 1 <= (rows - 1) // 64  # at least 64 rows per chunk, except a single chunk
    if rows == 1:
        assert chunks == 1


def test_calibrate_workspace_size_rejects():
    assert _ws(0, 64)[0] == "MM_ERR_SHAPE"
    assert _ws(4, 100)[0] == "MM_ERR_SHAPE"
    assert _ws(4, 65536)[0] == "MM_ERR_SHAPE"
    assert b.STATUS_NAMES[b.lib.mm_calibrate_workspace_size(4, 64, None)] == "MM_ERR_NULL"


def _cal(rows=64, K=128, ldx=None, fm=(0, 0), x=FAKE, ws=FAKE, wsb=None, perm=FAKE, split=FAKE):
    if wsb is None:
        wsb = _ws(rows, K)[1] if _ws(rows, K)[0] == "MM_OK" else 1 << 30
    st = b.lib.mm_calibrate(ctypes.c_void_p(x), rows, K, ldx if ldx is not None else K, b.MMFormats(*fm),
                            ctypes.c_void_p(ws), wsb, ctypes.c_void_p(perm), ctypes.c_void_p(split), None)
    return b.STATUS_NAMES[st]


def test_calibrate_rejects_bad_arguments():
    assert _cal(x=0) == "MM_ERR_NULL"
    assert _cal(ws=0) == "MM_ERR_NULL"
    assert _cal(perm=0) == "MM_ERR_NULL"
    assert _cal(split=0) == "MM_ERR_NULL"
    assert _cal(rows=0) == "MM_ERR_SHAPE"
    assert _cal(K=96 + 8) == "MM_ERR_SHAPE"
    assert _cal(K=65536) == "MM_ERR_SHAPE"
    assert _cal(ldx=96) == "MM_ERR_SHAPE"
    assert _cal(fm=(2, 0)) == "MM_ERR_FORMAT"
    assert _cal(fm=(0, 5)) == "MM_ERR_FORMAT"
    assert _cal(wsb=_ws(64, 128)[1] - 8) == "MM_ERR_WORKSPACE"
    assert _cal(x=FAKE + 2) == "MM_ERR_ALIGN"
    assert _cal(ldx=132) == "MM_ERR_ALIGN"
    assert _cal(ws=FAKE + 8) == "MM_ERR_ALIGN"
    assert _cal(perm=FAKE + 4) == "MM_ERR_ALIGN"
    assert _cal(split=FAKE + 2) == "MM_ERR_ALIGN"
    assert b.lib.mm_last_error().decode()


def _nq(d, x=FAKE, gamma=FAKE, eps=1e-5, perm=FAKE):
    st = b.lib.mm_rmsnorm_quantize_act(ctypes.c_void_p(x), d.K, ctypes.c_void_p(gamma), ctypes.c_float(eps),
                                       ctypes.c_void_p(perm), ctypes.byref(d), None)
    return b.STATUS_NAMES[st]


def test_rmsnorm_quantize_rejects_bad_arguments():
    d = _tensor()
    assert _nq(d, gamma=0) == "MM_ERR_NULL"
    assert _nq(d, x=0) == "MM_ERR_NULL"
    assert _nq(d, perm=0) == "MM_ERR_NULL"
    for eps in (0.0, -1e-5, float("inf"), float("nan")):
        assert _nq(d, eps=eps) == "MM_ERR_VALUE", eps
    assert _nq(d, gamma=FAKE + 1) == "MM_ERR_ALIGN"
    assert _nq(d, gamma=FAKE + 8) == "MM_ERR_ALIGN"
    assert _nq(_tensor(split=(64, 16, 48))) == "MM_ERR_SPLIT"
    bad = _tensor()
    bad.formats = b.MMFormats(7, 0)
    assert _nq(bad) == "MM_ERR_FORMAT"
    assert b.lib.mm_last_error().decode()


def _cal_na(rows=64, K=128, ldx=None, fm=(0, 0), x=FAKE, perm=FAKE, split=FAKE):
    st = b.lib.mm_calibrate_no_alloc(ctypes.c_void_p(x), rows, K, ldx if ldx is not None else K, b.MMFormats(*fm),
                                     ctypes.c_void_p(perm), ctypes.c_void_p(split), None)
    return b.STATUS_NAMES[st]


def test_calibrate_no_alloc_rejects_bad_arguments():
    """The no-allocation variant validates like mm_calibrate, and rejects a
    plan beyond its 16 MiB static scratch before touching the device."""
    assert _cal_na(x=0) == "MM_ERR_NULL"
    assert _cal_na(perm=0) == "MM_ERR_NULL"
    assert _cal_na(split=0) == "MM_ERR_NULL"
    assert _cal_na(rows=0) == "MM_ERR_SHAPE"
    assert _cal_na(K=96 + 8) == "MM_ERR_SHAPE"
    assert _cal_na(ldx=96) == "MM_ERR_SHAPE"
    assert _cal_na(fm=(2, 0)) == "MM_ERR_FORMAT"
    # the largest plan that fits: K = 31488 at any row count (reaches the alignment check)
    st, n = _ws(1 << 20, 31488)
    assert st == "MM_OK" and n <= 16 << 20
    assert _cal_na(rows=1 << 20, K=31488, x=FAKE + 2) == "MM_ERR_ALIGN"
    # one step wider no longer fits
    st, n = _ws(1 << 20, 31520)
    assert st == "MM_OK" and n > 16 << 20
    assert _cal_na(rows=1 << 20, K=31520) == "MM_ERR_WORKSPACE"
    msg = b.lib.mm_last_error().decode()
    assert "static" in msg and str(16 << 20) in msg
    assert _cal_na(rows=1 << 20, K=32768) == "MM_ERR_WORKSPACE"
    assert _cal_na(x=FAKE + 2) == "MM_ERR_ALIGN"
    assert _cal_na(perm=FAKE + 4) == "MM_ERR_ALIGN"
    assert _cal_na(split=FAKE + 2) == "MM_ERR_ALIGN"
