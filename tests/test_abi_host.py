"""Host-side tests of the C ABI (no GPU needed): the library loads, exports
every function include/kf355.h declares, and rejects bad arguments on the
host before any HIP call.  Only argument errors and zero-element no-ops are
exercised here, so nothing is ever launched; fake device addresses are never
dereferenced."""
import ctypes
import os
import re

import pytest

from paper_2607_24762_amd import kf355

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "kf355.h")

F32, BF16, F16 = 0, 1, 2
OK, NULLP, SHAPE, DTYPE, ARG, LAYOUT, WS, HIP = range(8)
FAKE = 0x7F0000000000          # a 256-byte aligned "device" address, never touched


@pytest.fixture(scope="module")
def lib():
    import torch
    # The fake addresses below must never reach a real device: these tests
    # only run where no GPU is visible.
    if torch.cuda.is_available():
        pytest.skip("host-only ABI tests use fake device addresses")
    if not os.path.exists(kf355.LIB_PATH):
        pytest.skip("libkf355.so not built (run __graft_entry__.build())")
    return kf355.lib()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(kf_\w+)\s*\(", text)))


def test_header_and_binding_agree():
    assert declared_functions() == sorted(kf355._SIGNATURES)


def test_every_declared_symbol_is_exported(lib):
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_version_and_status_names(lib):
    assert lib.kf_abi_version() == 1
    for code, name in kf355.STATUS_NAMES.items():
        assert lib.kf_status_name(code).decode() == name
    assert lib.kf_status_name(99).decode() == "KF_UNKNOWN"


def arr(vals):
    return (ctypes.c_int64 * max(len(vals), 1))(*vals)


def softmax(lib, x=FAKE, xt=F32, y=FAKE + (1 << 30), yt=F32, shape=(4, 8), xs=None, ys=None, dim=-1, ndim=None):
    nd = len(shape) if ndim is None else ndim
    return lib.kf_softmax(ctypes.c_void_p(x), xt, ctypes.c_void_p(y), yt, nd,
                          arr(shape) if shape is not None else None,
                          arr(xs) if xs else None, arr(ys) if ys else None, dim, None)


def err(lib):
    return lib.kf_last_error().decode()


def test_softmax_rejections(lib):
    assert softmax(lib, ndim=9, shape=(1,) * 9) == SHAPE
    assert softmax(lib, ndim=2, shape=None) == NULLP
    assert softmax(lib, shape=(4, -1)) == SHAPE
    assert softmax(lib, xt=7) == DTYPE
    assert softmax(lib, xt=F32, yt=BF16) == DTYPE          # narrowing is not softmax's dtype=
    assert softmax(lib, dim=2) == ARG and "dim" in err(lib)
    assert softmax(lib, dim=-3) == ARG
    assert softmax(lib, x=0) == NULLP
    assert softmax(lib, x=FAKE + 2) == ARG                 # fp32 needs 4-byte alignment
    assert softmax(lib, xs=(1, 4)) == LAYOUT               # transposed view
    assert softmax(lib, y=FAKE + 64) == ARG                # partial overlap
    assert softmax(lib, y=FAKE, xt=BF16, yt=F32) == ARG    # in place needs equal dtypes
    assert softmax(lib, shape=(4, 2**62, 4)) == SHAPE      # element count overflows


def test_softmax_zero_elements_is_a_noop(lib):
    assert softmax(lib, shape=(0, 8)) == OK
    assert lib.kf_last_variant().decode() == "noop"
    assert softmax(lib, x=0, y=0, shape=(5, 0)) == OK      # nothing to touch, NULL allowed
    assert softmax(lib, shape=(0,), dim=0) == OK


def test_softmax_size_one_dims_may_have_any_stride(lib):
    # [1, 0] has no elements; a size-1 leading dim with an odd stride is dense.
    assert softmax(lib, shape=(1, 0), xs=(12345, 1)) == OK


def split(lib, shape=(1, 8, 1, 32768), xt=BF16, yt=F32, x=FAKE, y=FAKE + (1 << 30), ws=FAKE + (2 << 30),
          wsb=1 << 20, dim=-1, xs=None):
    return lib.kf_softmax_split(ctypes.c_void_p(x), xt, ctypes.c_void_p(y), yt, len(shape), arr(shape),
                                arr(xs) if xs else None, None, dim, ctypes.c_void_p(ws), wsb, None)


def split_ws(lib, shape, xt=BF16, yt=F32, dim=-1):
    n = ctypes.c_size_t(0)
    st = lib.kf_softmax_split_workspace_bytes(xt, yt, len(shape), arr(shape), dim, ctypes.byref(n))
    return st, n.value


def test_softmax_split_rejections(lib):
    # The argument checks are kf_softmax's ...
    assert split(lib, xt=F32, yt=BF16) == DTYPE
    assert split(lib, dim=4) == ARG
    assert split(lib, x=0) == NULLP
    assert split(lib, xs=(262144, 32768, 32768, 2)) == LAYOUT
    assert split(lib, y=FAKE + 64) == ARG
    # ... plus the workspace, on a view that is split.
    assert split(lib, ws=0) == WS
    assert split(lib, wsb=64) == WS and "needed" in err(lib)
    assert split(lib, ws=FAKE + (2 << 30) + 128) == WS     # not 256-byte aligned
    assert split(lib, ws=FAKE + 256) == ARG                # overlaps x
    assert split(lib, shape=(1, 8, 1, 0), ws=0, wsb=0) == OK
    assert lib.kf_last_variant().decode() == "noop"


def test_softmax_split_workspace_query(lib):
    # 8 rows of 32768 bf16 -> fp32 (192 KiB of traffic each): the smallest
    # parts that leave at most 16 per row, 16 parts of 2048 elements: the
    # 256-byte status block, 8-byte (m, s) partials (1024 bytes, a whole
    # number of 256-byte lines), one 256-byte counter line per row.
    assert split_ws(lib, (1, 8, 1, 32768)) == (OK, 256 + 1024 + 8 * 256)
    # The same rows with bf16 output move 128 KiB each: not split.
    assert split_ws(lib, (1, 8, 1, 32768), yt=BF16) == (OK, 0)
    # A row that does not start on a 16-byte boundary spans one more vector:
    # 40001 elements take 10 parts of 4096.
    assert split_ws(lib, (3, 40001)) == (OK, 256 + 256 + 3 * 256)
    # Rows of partial vectors beyond 16384 elements are split at any size
    # (the per-row path would stream them twice): 16385 -> 9 parts of 2048.
    assert split_ws(lib, (2, 16385), yt=BF16) == (OK, 256 + 256 + 2 * 256)
    assert split_ws(lib, (2, 16384), yt=BF16) == (OK, 0)
    # 127 rows of 70000: 9 parts of 8192 (the first size with at most 16 per
    # row) would make 1143 workgroups, so parts of 16384 (5 per row).
    assert split_ws(lib, (127, 70000)) == (OK, ((127 * 5 * 8 + 255) // 256) * 256 + 127 * 256 + 256)
    assert split_ws(lib, (4096, 4096)) == (OK, 0)          # many rows: not split
    assert split_ws(lib, (4, 1000), xt=F32, yt=F32) == (OK, 0)
    assert split_ws(lib, (1, 32768 * 4, 8), dim=1) == (OK, 0)  # not the last dim
    assert split_ws(lib, (0, 32768)) == (OK, 0)
    assert split_ws(lib, (4, 8), dim=2)[0] == ARG
    assert split_ws(lib, (4, 8), xt=9)[0] == DTYPE
    assert split_ws(lib, (4, 8), yt=9)[0] == DTYPE
    assert lib.kf_softmax_split_workspace_bytes(BF16, F32, 2, arr((2, 4)), -1, None) == NULLP


def causal(lib, shape=(2, 4, 8), scale=0.5, x=FAKE, y=FAKE + (1 << 30), xt=F32, yt=F32, xs=None):
    return lib.kf_softmax_causal(ctypes.c_void_p(x), xt, ctypes.c_void_p(y), yt, len(shape), arr(shape),
                                 arr(xs) if xs else None, None, scale, None)


def test_softmax_causal_rejections(lib):
    assert causal(lib, shape=(8,)) == SHAPE               # needs [..., q, k]
    assert causal(lib, scale=float("nan")) == ARG
    assert causal(lib, scale=float("inf")) == ARG
    assert causal(lib, xt=F32, yt=F16) == DTYPE
    assert causal(lib, x=0) == NULLP
    assert causal(lib, xs=(32, 1, 4)) == LAYOUT
    assert causal(lib, y=FAKE + 4) == ARG
    assert causal(lib, shape=(2, 0, 8)) == OK and lib.kf_last_variant().decode() == "noop"


def ln(lib, shape=(4, 64), nd=1, w=None, b=None, at=F32, eps=1e-5, x=FAKE, y=FAKE + (1 << 30), xt=F32, xs=None):
    return lib.kf_layer_norm(ctypes.c_void_p(x), xt, ctypes.c_void_p(y), len(shape), arr(shape),
                             arr(xs) if xs else None, None, nd, ctypes.c_void_p(w), ctypes.c_void_p(b), at, eps, None)


def test_layer_norm_rejections(lib):
    assert ln(lib, nd=0) == ARG
    assert ln(lib, nd=3) == ARG
    assert ln(lib, eps=-1.0) == ARG
    assert ln(lib, xt=BF16, w=FAKE + (3 << 30), at=F16) == DTYPE
    assert ln(lib, x=0) == NULLP
    assert ln(lib, xs=(1, 4)) == LAYOUT
    assert ln(lib, y=FAKE + 8) == ARG
    assert ln(lib, w=FAKE + (1 << 30) + 4) == ARG          # weight inside y
    assert ln(lib, w=FAKE + (3 << 30) + 2) == ARG          # fp32 weight not 4-byte aligned
    assert ln(lib, shape=(0, 64)) == OK and lib.kf_last_variant().decode() == "noop"


def gn(lib, shape=(2, 8, 4, 4), groups=4, w=None, b=None, at=F32, eps=1e-5, ws=FAKE + (2 << 30), wsb=1 << 20,
       xt=F32, x=FAKE, y=FAKE + (1 << 30), xs=None):
    return lib.kf_group_norm(ctypes.c_void_p(x), xt, ctypes.c_void_p(y), len(shape), arr(shape),
                             arr(xs) if xs else None, None, groups, ctypes.c_void_p(w), ctypes.c_void_p(b), at,
                             eps, ctypes.c_void_p(ws), wsb, None)


def gn_ws(lib, shape, groups, xt=BF16):
    n = ctypes.c_size_t(0)
    st = lib.kf_group_norm_workspace_bytes(xt, len(shape), arr(shape), groups, ctypes.byref(n))
    return st, n.value


def test_group_norm_rejections(lib):
    assert gn(lib, shape=(8,)) == SHAPE
    assert gn(lib, groups=3) == ARG and "divisible" in err(lib)
    assert gn(lib, groups=0) == ARG
    assert gn(lib, eps=-1.0) == ARG
    assert gn(lib, eps=float("nan")) == ARG
    assert gn(lib, xt=BF16, w=FAKE + (3 << 30), at=F16) == DTYPE
    assert gn(lib, ws=0) == WS
    assert gn(lib, wsb=16) == WS
    assert gn(lib, ws=FAKE + (2 << 30) + 64) == WS         # not 256-byte aligned
    assert gn(lib, xs=(128, 16, 4, 2)) == LAYOUT          # not dense in any layout
    assert gn(lib, xs=(128, 1, 32, 8)) == LAYOUT and "channels last" in err(lib)  # channels-last x, NCHW y
    assert gn(lib, y=FAKE + 128) == ARG                   # partial overlap
    assert gn(lib, w=FAKE + (1 << 30) + 64) == ARG        # weight inside y
    assert gn(lib, ws=FAKE) == ARG                        # workspace overlaps x


def test_group_norm_zero_elements_and_workspace_query(lib):
    assert gn(lib, shape=(0, 8, 4, 4), ws=0, wsb=0) == OK
    st, n = gn_ws(lib, (0, 8, 4), 2)
    assert st == OK and n == 0
    st, n = gn_ws(lib, (1, 512, 128, 128), 32)
    # The query sizes for every path this shape may take: channels last in
    # 16 bits, 32 groups x 64 parts (tiles of 256 pixels): the 256-byte
    # status block, one 8-byte published word per part, each on a 128-byte
    # line of its own, then one 256-byte counter line per group.  NCHW uses
    # 16 packed words per group.
    assert st == OK and n == 256 + 32 * 64 * 128 + 32 * 256
    # The same in fp32: no tile kernel, 16 chunks of 16384 elements per group.
    st, n = gn_ws(lib, (1, 512, 128, 128), 32, xt=F32)
    assert st == OK and n == 256 + 32 * 16 * 8 + 32 * 256
    # 12-channel groups: 3 chunks of 16384 elements per group, partials
    # padded to 256 bytes.
    st, n = gn_ws(lib, (1, 24, 64, 64), 2)
    assert st == OK and n == 256 + 256 + 2 * 256
    st, _ = gn_ws(lib, (1, 6, 4), 4)
    assert st == ARG
    assert lib.kf_group_norm_workspace_bytes(F32, 2, arr((2, 4)), 2, None) == NULLP


def gn_static(lib, shape=(2, 8, 4, 4), groups=4, xt=F32, x=FAKE, y=FAKE + (1 << 30), eps=1e-5):
    return lib.kf_group_norm_static(ctypes.c_void_p(x), xt, ctypes.c_void_p(y), len(shape), arr(shape), None, None,
                                    groups, None, None, xt, eps, None)


def test_group_norm_static_rejections(lib):
    # The allocation-free GroupNorm runs the same checks as kf_group_norm,
    # all before its scratch array is looked up on the device.
    assert gn_static(lib, shape=(0, 8, 4, 4)) == OK
    assert lib.kf_last_variant().decode() == "noop"
    assert gn_static(lib, x=0) == NULLP
    assert gn_static(lib, groups=3) == ARG
    assert gn_static(lib, eps=-1.0) == ARG
    assert gn_static(lib, xt=7) == DTYPE
    assert gn_static(lib, y=FAKE + 16) == ARG                  # partial overlap
    # One-chunk groups of 16384 elements: 96000 of them need 256 + 768000 +
    # 96000 * 256 bytes of exchange workspace, beyond the 1 MiB array.
    assert gn_static(lib, shape=(3000, 32, 128, 128), groups=32, y=FAKE + (1 << 40)) == WS
    assert "static scratch array holds 1048576" in err(lib)
    st, n = gn_ws(lib, (3000, 32, 128, 128), 32, xt=F32)
    assert st == OK and n > 1 << 20
    # The SD3.5 VAE block fits in either layout (the query's 270592 bytes
    # cover channels last; NCHW needs 12544).
    st, n = gn_ws(lib, (1, 512, 128, 128), 32)
    assert st == OK and n == 270592 <= 1 << 20


def test_binding_workspace_query_is_the_abi_query(lib):
    # kf355.kf_group_norm_workspace_bytes marshals the same query (shape and
    # dtype only: a CPU tensor serves), and repeats it per shape from its cache.
    import torch
    x = torch.empty((1, 512, 128, 128), dtype=torch.bfloat16)
    assert kf355.kf_group_norm_workspace_bytes(x, 32) == gn_ws(lib, (1, 512, 128, 128), 32)[1] == 270592
    assert kf355.kf_group_norm_workspace_bytes(x, 32) == 270592
    y = torch.empty((2, 96, 32, 32), dtype=torch.float16)
    assert kf355.kf_group_norm_workspace_bytes(y, 4) == gn_ws(lib, (2, 96, 32, 32), 4, xt=F16)[1]


def ap(lib, shape=(2, 3, 7, 7), oh=1, ow=1, x=FAKE, y=FAKE + (1 << 30), xt=F32, xs=None, ys=None):
    return lib.kf_adaptive_avgpool2d(ctypes.c_void_p(x), xt, ctypes.c_void_p(y), len(shape), arr(shape),
                                     arr(xs) if xs else None, arr(ys) if ys else None, oh, ow, None)


def test_avgpool_rejections(lib):
    assert ap(lib, shape=(7, 7)) == SHAPE
    assert ap(lib, shape=(1, 2, 3, 4, 5)) == SHAPE
    assert ap(lib, shape=(2, 3, 0, 7)) == SHAPE
    assert ap(lib, oh=0) == ARG
    assert ap(lib, y=FAKE + 64) == ARG                    # overlaps x
    assert ap(lib, xs=(147, 1, 21, 3)) == LAYOUT          # channels-last x, NCHW y
    assert ap(lib, xs=(147, 49, 1, 7)) == LAYOUT          # neither layout
    assert ap(lib, xt=5) == DTYPE
    assert ap(lib, x=0) == NULLP


def test_avgpool_zero_planes_is_a_noop(lib):
    assert ap(lib, shape=(0, 3, 7, 7)) == OK
    assert lib.kf_last_variant().decode() == "noop"


def mp(lib, shape=(2, 3, 9, 9), win=(3, 3, 2, 2, 1, 1, 1, 1), ceil=0, x=FAKE, y=FAKE + (1 << 30), idx=None, xt=F32,
       xs=None, ys=None):
    return lib.kf_max_pool2d(ctypes.c_void_p(x), xt, ctypes.c_void_p(y), ctypes.c_void_p(idx), len(shape),
                             arr(shape), arr(xs) if xs else None, arr(ys) if ys else None,
                             arr(win) if win is not None else None, ceil, None)


def mp_size(lib, h, w, win, ceil=0):
    out = arr([0, 0])
    st = lib.kf_max_pool2d_output_size(h, w, arr(win), ceil, out)
    return st, (out[0], out[1])


def test_max_pool2d_rejections(lib):
    assert mp(lib, shape=(9, 9)) == SHAPE
    assert mp(lib, win=None) == NULLP
    assert mp(lib, win=(0, 3, 1, 1, 0, 0, 1, 1)) == ARG
    assert mp(lib, win=(3, 3, 0, 1, 0, 0, 1, 1)) == ARG
    assert mp(lib, win=(3, 3, 1, 1, 2, 0, 1, 1)) == ARG and "padding" in err(lib)
    assert mp(lib, win=(3, 3, 1, 1, 0, 0, 0, 1)) == ARG
    assert mp(lib, shape=(1, 1, 2, 2), win=(3, 3, 1, 1, 0, 0, 1, 1)) == SHAPE   # empty output
    assert mp(lib, xt=4) == DTYPE
    assert mp(lib, x=0) == NULLP
    assert mp(lib, idx=FAKE + (2 << 30) + 4) == ARG                              # int64 alignment
    assert mp(lib, y=FAKE + 8) == ARG                                            # overlaps x
    assert mp(lib, idx=FAKE + 16) == ARG                                         # indices overlap x
    assert mp(lib, xs=(1, 2, 3, 4)) == LAYOUT
    assert mp(lib, xs=(243, 1, 27, 3)) == LAYOUT and "channels last" in err(lib)  # y not in x's layout
    assert mp(lib, shape=(0, 3, 9, 9)) == OK and lib.kf_last_variant().decode() == "noop"


def test_max_pool2d_output_size(lib):
    assert mp_size(lib, 112, 112, (3, 3, 2, 2, 1, 1, 1, 1)) == (OK, (56, 56))   # ResNet-50 stem
    assert mp_size(lib, 5, 7, (2, 2, 2, 2, 0, 0, 1, 1)) == (OK, (2, 3))
    assert mp_size(lib, 5, 7, (2, 2, 2, 2, 0, 0, 1, 1), ceil=1) == (OK, (3, 4))
    assert mp_size(lib, 6, 6, (3, 3, 2, 2, 1, 1, 2, 2)) == (OK, (2, 2))
    assert mp_size(lib, 2, 2, (3, 3, 1, 1, 0, 0, 1, 1))[0] == SHAPE
    # The dilated kernel (9) is longer than the input (7): floor mode has no
    # window, ceil mode one (its span rounds toward -infinity, as PyTorch's).
    assert mp_size(lib, 7, 7, (5, 5, 3, 3, 0, 0, 2, 2))[0] == SHAPE
    assert mp_size(lib, 7, 7, (5, 5, 3, 3, 0, 0, 2, 2), ceil=1) == (OK, (1, 1))
    assert mp_size(lib, 0, 4, (1, 1, 1, 1, 0, 0, 1, 1))[0] == SHAPE
    assert lib.kf_max_pool2d_output_size(4, 4, arr((1, 1, 1, 1, 0, 0, 1, 1)), 0, None) == NULLP


def test_binding_refuses_cpu_tensors(lib):
    import torch
    with pytest.raises(ValueError):
        kf355.kf_softmax(torch.zeros(4, 4))


def test_stream_copy_rejections(lib):
    # The calibration copy checks its arguments on the host like the operators.
    assert lib.kf_stream_copy(FAKE, FAKE + (1 << 30), 0, None) == OK          # no-op
    assert lib.kf_stream_copy(FAKE, FAKE + (1 << 30), 24, None) == SHAPE      # not a multiple of 16
    assert lib.kf_stream_copy(FAKE, FAKE + (1 << 30), -16, None) == SHAPE
    assert lib.kf_stream_copy(None, FAKE, 64, None) == NULLP
    assert lib.kf_stream_copy(FAKE + 4, FAKE + (1 << 30), 64, None) == ARG    # misaligned
    assert lib.kf_stream_copy(FAKE, FAKE + 32, 64, None) == ARG               # overlap


def test_stream_read_rejections(lib):
    # The calibration read checks its arguments on the host like the operators.
    assert lib.kf_stream_read(FAKE, 0, FAKE + (1 << 30), None) == OK          # no-op
    assert lib.kf_stream_read(FAKE, 24, FAKE + (1 << 30), None) == SHAPE      # not a multiple of 16
    assert lib.kf_stream_read(FAKE, -16, FAKE + (1 << 30), None) == SHAPE
    assert lib.kf_stream_read(None, 64, FAKE, None) == NULLP
    assert lib.kf_stream_read(FAKE, 64, None, None) == NULLP
    assert lib.kf_stream_read(FAKE, 64, FAKE + (1 << 30) + 4, None) == ARG    # dst not 8-byte aligned
    assert lib.kf_stream_read(FAKE + 8, 64, FAKE + (1 << 30), None) == ARG    # src not 16-byte aligned
    assert lib.kf_stream_read(FAKE, 8192, FAKE + 4096, None) == ARG           # output inside the input
    assert lib.kf_stream_read(FAKE, 4096, FAKE + 4080, None) == ARG           # output (two 8-byte words) on the input's end
