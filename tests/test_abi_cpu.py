"""The C ABI without a GPU: the library loads, exports every symbol the header
declares, sizes the workspace, and rejects malformed calls on the host before
anything is launched (fake, never-dereferenced device addresses are enough)."""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2608_12700_amd import gdn

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def header_functions():
    src = open(os.path.join(ROOT, "include", "gdn.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(gdn_[a-z_]+)\s*\(", src)))


def test_library_exports_every_declared_function():
    lib = gdn.load()
    declared = header_functions()
    assert set(declared) == set(gdn.EXPORTED)
    for name in declared:
        assert hasattr(lib, name), name


def test_status_strings_and_version():
    assert "gfx950" in gdn.gdn_version()
    for code in range(0, -11, -1):
        assert gdn.gdn_status_str(code) != "unknown status"


FAKE = 0x7f0000000000  # never dereferenced: validation fails first or nothing runs


def fake(i):
    return ctypes.c_void_p(FAKE + (i << 32))


NO_WS = object()  # pass a NULL workspace pointer


def call_fwd(p, ptrs=None, ws_bytes=None, ws=None, **over):
    args = dict(q=fake(1), k=fake(2), v=fake(3), g=fake(4), beta=fake(5), S0=None, o=fake(6),
                S_T=fake(7), states=fake(8))
    if p.variant == 1:
        args["g"] = None
    if p.variant == 2:
        args["beta"] = None
    args.update(over)
    wsb = gdn.gdn_fwd_workspace_size(p) if ws_bytes is None else ws_bytes
    return gdn.gdn_fwd(p, args["q"], args["k"], args["v"], args["g"], args["beta"], args["S0"],
                       args["o"], args["S_T"], args["states"],
                       None if ws is NO_WS else (fake(9) if ws is None else ws), wsb, None)


def call_bwd(p, **over):
    args = dict(q=fake(1), k=fake(2), v=fake(3), g=fake(4), beta=fake(5), st=fake(6), dO=fake(7),
                dST=None, dq=fake(10), dk=fake(11), dv=fake(12), dg=fake(13), db=fake(14),
                dS0=fake(15))
    if p.variant == 1:
        args["g"] = args["dg"] = None
    if p.variant == 2:
        args["beta"] = args["db"] = None
    args.update(over)
    return gdn.gdn_bwd(p, args["q"], args["k"], args["v"], args["g"], args["beta"], args["st"],
                       args["dO"], args["dST"], args["dq"], args["dk"], args["dv"], args["dg"],
                       args["db"], args["dS0"], fake(20), gdn.gdn_bwd_workspace_size(p), None)


def test_unsupported_dims_and_chunk():
    for dk, dv in [(32, 64), (96, 128), (128, 512), (256, 128)]:
        p = gdn.make_problem(1, 64, 1, dk, dv)
        assert call_fwd(p) == -3
        assert gdn.gdn_fwd_workspace_size(p) == 0
    p = gdn.make_problem(1, 64, 1, 64, 64, chunk=32)
    assert call_fwd(p) == -3


def test_head_stride_limit():
    # row strides H * max(d_k, d_v) must stay below 2^24 elements
    p = gdn.make_problem(1, 64, (1 << 24) // 256, 64, 256)
    assert call_fwd(p) == -3 and call_bwd(p) == -3
    assert gdn.gdn_fwd_workspace_size(p) == 0
    p = gdn.make_problem(1, 64, (1 << 24) // 256 - 1, 64, 256)
    assert gdn.gdn_fwd_workspace_size(p) > 0


def test_bad_shape_dtype_variant():
    assert call_fwd(gdn.make_problem(-1, 64, 1, 64, 64)) == -2
    assert call_fwd(gdn.make_problem(1, 64, 1, 64, 64, io_dtype=7)) == -4
    assert call_fwd(gdn.make_problem(1, 64, 1, 64, 64, variant=5)) == -9
    p = gdn.make_problem(2, 64, 1, 64, 64)
    p.num_seqs = 3
    assert call_fwd(p) == -2


def test_gate_pointers_must_match_variant():
    p = gdn.make_problem(1, 64, 1, 64, 64, variant="delta")
    assert call_fwd(p, g=fake(4)) == -9
    p = gdn.make_problem(1, 64, 1, 64, 64, variant="decay_only")
    assert call_fwd(p, beta=fake(5)) == -9
    p = gdn.make_problem(1, 64, 1, 64, 64)
    assert call_fwd(p, g=None) == -9
    assert call_bwd(p, dg=None) == -9


def test_null_pointers():
    p = gdn.make_problem(1, 64, 2, 64, 64)
    assert call_fwd(p, q=None) == -1
    assert call_fwd(p, states=None) == -1
    assert call_bwd(p, dq=None) == -1
    assert call_bwd(p, st=None) == -1


def test_workspace_checks():
    p = gdn.make_problem(1, 64, 2, 64, 64)
    need = gdn.gdn_fwd_workspace_size(p)
    assert need > 0 and need % 256 == 0
    assert call_fwd(p, ws_bytes=need - 1) == -5
    assert call_fwd(p, ws=ctypes.c_void_p(FAKE + 128)) == -5  # misaligned
    assert call_fwd(p, ws=NO_WS, ws_bytes=need) == -5         # NULL workspace
    assert call_fwd(p, ws=NO_WS, ws_bytes=0) == -5


def test_alias_rejected():
    p = gdn.make_problem(1, 64, 2, 64, 64)
    assert call_fwd(p, o=fake(1)) == -6          # o on top of q
    assert call_fwd(p, S_T=fake(6)) == -6        # two outputs overlap
    assert call_bwd(p, dv=fake(3)) == -6
    assert call_bwd(p, dS0=fake(15), dq=fake(15)) == -6


def test_packed_offsets_validated():
    good = np.array([0, 5, 70, 70, 200], np.int32)
    p = gdn.make_problem(1, 200, 2, 64, 64, cu_host=good, cu_dev_ptr=FAKE + (30 << 32))
    assert gdn.gdn_num_chunks(p) == 1 + 2 + 0 + 3
    for bad in ([1, 5, 70, 70, 200], [0, 70, 5, 70, 200], [0, 5, 70, 70, 199]):
        b = np.array(bad, np.int32)
        p = gdn.make_problem(1, 200, 2, 64, 64, cu_host=b, cu_dev_ptr=FAKE + (30 << 32))
        assert call_fwd(p) == -7
    p = gdn.make_problem(2, 200, 2, 64, 64, cu_host=good, cu_dev_ptr=FAKE + (30 << 32))
    assert call_fwd(p) == -7
    p = gdn.make_problem(1, 200, 2, 64, 64, cu_host=good, cu_dev_ptr=None)
    assert call_fwd(p) == -1


def test_chunk_count_and_workspace_grow_with_size():
    small = gdn.make_problem(1, 256, 2, 64, 64, io_dtype=0)
    big = gdn.make_problem(4, 4096, 16, 128, 128)
    assert gdn.gdn_num_chunks(small) == 4
    assert gdn.gdn_num_chunks(big) == 256
    assert gdn.gdn_fwd_workspace_size(big) > gdn.gdn_fwd_workspace_size(small)
    assert gdn.gdn_bwd_workspace_size(big) > gdn.gdn_bwd_workspace_size(small)
    assert gdn.gdn_num_chunks(gdn.make_problem(1, 0, 2, 64, 64)) == 0


# ---------------------------------------------------------------- channel-wise entry points

def call_cw_fwd(p, ws_bytes=None, **over):
    args = dict(q=fake(1), k=fake(2), v=fake(3), g=fake(4), b=fake(5), w=fake(16), S0=None, o=fake(6),
                S_T=fake(7), states=fake(8))
    args.update(over)
    wsb = gdn.gdn_cw_fwd_workspace_size(p) if ws_bytes is None else ws_bytes
    return gdn.gdn_cw_fwd(p, args["q"], args["k"], args["v"], args["g"], args["b"], args["w"], args["S0"],
                          args["o"], args["S_T"], args["states"], fake(9), wsb, None)


def call_cw_bwd(p, **over):
    args = dict(q=fake(1), k=fake(2), v=fake(3), g=fake(4), b=fake(5), w=fake(16), st=fake(6), dO=fake(7),
                dST=None, dq=fake(10), dk=fake(11), dv=fake(12), dg=fake(13), db=fake(14), dw=fake(17),
                dS0=fake(15))
    args.update(over)
    return gdn.gdn_cw_bwd(p, args["q"], args["k"], args["v"], args["g"], args["b"], args["w"], args["st"],
                          args["dO"], args["dST"], args["dq"], args["dk"], args["dv"], args["dg"], args["db"],
                          args["dw"], args["dS0"], fake(20), gdn.gdn_cw_bwd_workspace_size(p), None)


def test_channelwise_bf16_activations_fp32_gates():
    pb = gdn.make_problem(1, 64, 2, 64, 64, io_dtype=gdn.GDN_BF16)
    pf = gdn.make_problem(1, 64, 2, 64, 64, io_dtype=gdn.GDN_F32)
    # the scans' operands follow the activation dtype; the gradient kernels' are fp32
    assert 0 < gdn.gdn_cw_fwd_workspace_size(pb) < gdn.gdn_cw_fwd_workspace_size(pf)
    assert 0 < gdn.gdn_cw_bwd_workspace_size(pb) < gdn.gdn_cw_bwd_workspace_size(pf)
    # gates are sized as fp32 also with bf16 activations: an output 16 KiB past
    # g's start (the bf16 size of q) still lies inside g (32 KiB)
    o_in_g = ctypes.c_void_p(FAKE + (4 << 32) + 64 * 2 * 64 * 2)
    assert call_cw_fwd(pb, o=o_in_g) == -6


def test_channelwise_gradients_follow_the_gates():
    p = gdn.make_problem(1, 64, 2, 64, 64, io_dtype=gdn.GDN_F32)
    assert call_cw_bwd(p, dg=None) == -9
    assert call_cw_bwd(p, b=None) == -9
    assert call_cw_bwd(p, dw=None) == -9


def test_channelwise_null_alias_and_workspace():
    p = gdn.make_problem(1, 64, 2, 64, 64, io_dtype=gdn.GDN_F32)
    need = gdn.gdn_cw_fwd_workspace_size(p)
    assert need > 0 and need % 256 == 0
    assert call_cw_fwd(p, q=None) == -1
    assert call_cw_fwd(p, ws_bytes=need - 1) == -5
    assert call_cw_fwd(p, o=fake(4)) == -6           # o on top of g
    assert call_cw_bwd(p, dw=fake(16)) == -6         # dw on top of w
    assert call_cw_bwd(p, dS0=None) == -1
    # a larger problem needs more workspace, the backward more than the forward
    big = gdn.make_problem(2, 640, 4, 128, 128, io_dtype=gdn.GDN_F32)
    assert gdn.gdn_cw_fwd_workspace_size(big) > need
    assert gdn.gdn_cw_bwd_workspace_size(big) > gdn.gdn_cw_fwd_workspace_size(big)


def test_noalloc_rejects_oversized_problems_on_the_host():
    # the size check runs before any HIP call: no GPU is needed to see it
    big = gdn.make_problem(4, 4096, 16, 128, 128)
    assert gdn.gdn_fwd_workspace_size(big) > gdn.NOALLOC_SCRATCH_BYTES
    args = [fake(i) for i in range(1, 6)] + [None] + [fake(i) for i in range(6, 9)]
    assert gdn.gdn_fwd_noalloc(big, *args, None) == -10
    bad = gdn.make_problem(1, 64, 1, 96, 64)
    assert gdn.gdn_fwd_noalloc(bad, *args, None) == -3
