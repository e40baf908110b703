"""The C-ABI library loads, exports every declared symbol, and rejects bad
arguments on the host before any launch (no GPU needed for these paths)."""
import ctypes
import os
import re

import pytest

import paper_2609_23169_amd as ut

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include",
                      "ultratex.h")

FAKE = ctypes.c_void_p(0x10000)        # aligned, never dereferenced on these paths
MISALIGNED = ctypes.c_void_p(0x10002)


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"\b(ut_[a-z_0-9]+)\s*\(", text)))


def test_header_and_binding_agree():
    assert declared_functions() == sorted(ut.EXPORTS)


def test_library_exports_every_declared_symbol():
    lib = ut.lib()
    for name in declared_functions():
        assert hasattr(lib, name), name
    assert lib.ut_abi_version() == 3


def test_trace_switch_and_empty_read():
    lib = ut.lib()
    assert lib.ut_trace_enable(1) == ut.UT_OK
    assert lib.ut_trace_enable(0) == ut.UT_OK
    assert ut.trace_read() == []          # nothing launched on this host
    assert lib.ut_trace_read(None, 0) == 0


def test_diag_library_exports_its_header():
    diag = os.path.join(os.path.dirname(HEADER), "ultratex_diag.h")
    names = sorted(set(re.findall(r"\b(ut_[a-z_0-9]+)\s*\(", open(diag).read())))
    assert names == ["ut_diag_mfma_rate"]
    lib = ctypes.CDLL(os.path.join(os.path.dirname(ut.__file__), "libutdiag.so"))
    for n in names:
        assert hasattr(lib, n), n
    f = lib.ut_diag_mfma_rate
    f.argtypes = [ctypes.c_int] * 3 + [ctypes.c_void_p] * 4
    assert f(2, 10, 4, FAKE, FAKE, FAKE, None) == -1       # unknown shape: nothing launched
    assert f(0, 0, 4, FAKE, FAKE, FAKE, None) == -1
    assert f(1, 10, 4, None, FAKE, FAKE, None) == -1


def test_workspace_sizes():
    assert ut.ut_drop_background_workspace_size(212992) == 52 * 4
    assert ut.ut_drop_background_workspace_size(1) == 4
    assert ut.ut_drop_background_workspace_size(0) == 0
    assert ut.ut_bsattn_bwd_workspace_size(1, 77586, 24) == 77586 * 24 * 8
    assert ut.ut_bsattn_bwd_varlen_workspace_size(77586, 24) == 77586 * 24 * 8
    assert ut.ut_bsattn_bwd_varlen_workspace_size(0, 24) == 0


def test_stored_ds_workspace_sizes():
    # statistics planes, a flag per query block row, the entry -> tile map and
    # the tiles of 2 block^2 bytes, each part padded to 256 bytes
    pad = lambda x: -(-x // 256) * 256
    rows = 1 * 3 * 8                      # B H ceil(1000 / 128)
    head = pad(1000 * 3 * 8) + pad(rows * 4)
    assert ut.ut_bsattn_bwd_workspace_size_stored(1, 1000, 3, 128, 0) == head
    assert ut.ut_bsattn_bwd_workspace_size_stored(1, 1000, 3, 128, 10) == head + pad(40) + 10 * 32768
    rows64 = 1 * 3 * 16
    assert (ut.ut_bsattn_bwd_workspace_size_stored(1, 1000, 3, 64, 10)
            == pad(1000 * 3 * 8) + pad(rows64 * 4) + pad(40) + 10 * 8192)
    # the 2K training workload at rho = 0.1: 882,792 pairs of 32 KiB
    big = ut.ut_bsattn_bwd_workspace_size_stored(1, 77060, 24, 128, 882792)
    assert big == pad(77060 * 24 * 8) + pad(24 * 603 * 4) + pad(882792 * 4) + 882792 * 32768
    for args in [(1, 1000, 3, 96, 10), (1, 1000, 3, 128, -1), (0, 1000, 3, 128, 10),
                 (1, 0, 3, 128, 10), (1, 1000, 3, 0, 10)]:
        assert ut.ut_bsattn_bwd_workspace_size_stored(*args) == 0, args
    # packed samples: B = 2, max_seqlen 700 -> 6 blocks per sample
    assert (ut.ut_bsattn_bwd_varlen_workspace_size_stored(2, 1000, 700, 3, 128, 10)
            == pad(1000 * 3 * 8) + pad(2 * 3 * 6 * 4) + pad(40) + 10 * 32768)
    assert ut.ut_bsattn_bwd_varlen_workspace_size_stored(2, 0, 700, 3, 128, 10) == 0
    assert ut.ut_bsattn_bwd_varlen_workspace_size_stored(0, 1000, 700, 3, 128, 10) == 0


def _fwd(**kw):
    a = dict(q=FAKE, k=FAKE, v=FAKE, o=FAKE, lse=FAKE, B=1, N=100, H=2, D=128, block=128,
             rowptr=FAKE, cols=FAKE, scale=0.1)
    a.update(kw)
    return ut.lib().ut_bsattn_fwd(a["q"], a["k"], a["v"], a["o"], a["lse"], a["B"], a["N"], a["H"],
                                  a["D"], a["block"], a["rowptr"], a["cols"], a["scale"], None)


@pytest.mark.parametrize("kw,status,msg", [
    (dict(D=96), ut.UT_ERR_UNSUPPORTED, "head_dim"),
    (dict(block=32), ut.UT_ERR_UNSUPPORTED, "block"),
    (dict(N=0), ut.UT_ERR_INVALID_ARG, "must be >= 1"),
    (dict(H=0), ut.UT_ERR_INVALID_ARG, "must be >= 1"),
    (dict(q=None), ut.UT_ERR_INVALID_ARG, "q is NULL"),
    (dict(v=MISALIGNED), ut.UT_ERR_INVALID_ARG, "aligned"),
    (dict(cols=None), ut.UT_ERR_INVALID_ARG, "q_cols is NULL"),
    (dict(scale=float("nan")), ut.UT_ERR_INVALID_ARG, "finite"),
    (dict(scale=0.0), ut.UT_ERR_INVALID_ARG, "> 0"),
    (dict(scale=-0.088), ut.UT_ERR_INVALID_ARG, "> 0"),
    # one sample's tensor of 2 GiB: 131072 x 64 x 128 bf16 (32-bit load ranges)
    (dict(N=131072, H=64), ut.UT_ERR_UNSUPPORTED, "2 GiB"),
])
def test_fwd_rejects_bad_arguments(kw, status, msg):
    assert _fwd(**kw) == status
    assert msg in ut.last_error()


def test_bwd_rejects_missing_workspace():
    lib = ut.lib()
    args = [FAKE] * 9 + [1, 100, 2, 128, 128] + [FAKE] * 4 + [0.1]
    st = lib.ut_bsattn_bwd(*args, None, 0, None)
    assert st == ut.UT_ERR_WORKSPACE and "workspace" in ut.last_error()
    st = lib.ut_bsattn_bwd(*args, FAKE, 100 * 2 * 8 - 4, None)
    assert st == ut.UT_ERR_WORKSPACE
    args[2] = None
    assert lib.ut_bsattn_bwd(*args, FAKE, 1600, None) == ut.UT_ERR_INVALID_ARG
    args[2] = FAKE
    args[10], args[11] = 131072, 64   # N, H: one sample's tensor reaches 2 GiB
    assert lib.ut_bsattn_bwd(*args, FAKE, 131072 * 64 * 8, None) == ut.UT_ERR_UNSUPPORTED
    assert "2 GiB" in ut.last_error()


def test_bwd_rejects_non_positive_scale():
    lib = ut.lib()
    for scale in (0.0, -0.088, float("inf")):
        args = [FAKE] * 9 + [1, 100, 2, 128, 128] + [FAKE] * 4 + [scale]
        assert lib.ut_bsattn_bwd(*args, FAKE, 1600, None) == ut.UT_ERR_INVALID_ARG
        assert "softmax_scale" in ut.last_error()
        vargs = [FAKE] * 10 + [3, 300, 128, 2, 128, 128] + [FAKE] * 4 + [scale]
        assert lib.ut_bsattn_bwd_varlen(*vargs, FAKE, 4800, None) == ut.UT_ERR_INVALID_ARG
        assert "softmax_scale" in ut.last_error()


def test_bwd_noalloc_rejects_problems_beyond_its_scratch():
    lib = ut.lib()
    args = [FAKE] * 9
    tail = [FAKE] * 4 + [0.0883883476]
    # 1 x 24 x 174763 = 4,194,312 query rows > 4,194,304 (32 MiB of 8-byte rows)
    st = lib.ut_bsattn_bwd_noalloc(*args, 1, 174763, 24, 128, 128, *tail, None)
    assert st == ut.UT_ERR_WORKSPACE and "built-in scratch" in ut.last_error()
    st = lib.ut_bsattn_bwd_noalloc(*args, 2, 100000, 24, 128, 128, *tail, None)
    assert st == ut.UT_ERR_WORKSPACE
    # the usual checks come first
    assert lib.ut_bsattn_bwd_noalloc(*args, 1, 100, 2, 96, 128, *tail, None) == ut.UT_ERR_UNSUPPORTED
    args[6] = None
    assert lib.ut_bsattn_bwd_noalloc(*args, 1, 100, 2, 128, 128, *tail, None) == ut.UT_ERR_INVALID_ARG
    assert "dq is NULL" in ut.last_error()


def _fwd_varlen(**kw):
    a = dict(q=FAKE, k=FAKE, v=FAKE, o=FAKE, lse=FAKE, cu=FAKE, B=3, T=300, maxlen=128, H=2, D=128,
             block=128, rowptr=FAKE, cols=FAKE, scale=0.1)
    a.update(kw)
    return ut.lib().ut_bsattn_fwd_varlen(a["q"], a["k"], a["v"], a["o"], a["lse"], a["cu"], a["B"],
                                         a["T"], a["maxlen"], a["H"], a["D"], a["block"], a["rowptr"],
                                         a["cols"], a["scale"], None)


@pytest.mark.parametrize("kw,status,msg", [
    (dict(cu=None), ut.UT_ERR_INVALID_ARG, "cu_seqlens is NULL"),
    (dict(T=-1), ut.UT_ERR_INVALID_ARG, "outside [0, 2^31)"),
    (dict(T=1 << 31), ut.UT_ERR_INVALID_ARG, "outside [0, 2^31)"),
    (dict(maxlen=0), ut.UT_ERR_INVALID_ARG, "must be >= 1"),
    (dict(B=0), ut.UT_ERR_INVALID_ARG, "must be >= 1"),
    (dict(D=96), ut.UT_ERR_UNSUPPORTED, "head_dim"),
    (dict(q=None), ut.UT_ERR_INVALID_ARG, "q is NULL"),
    (dict(lse=MISALIGNED), ut.UT_ERR_INVALID_ARG, "aligned"),
    (dict(maxlen=131072, H=64, T=131072), ut.UT_ERR_UNSUPPORTED, "2 GiB"),
    (dict(scale=0.0), ut.UT_ERR_INVALID_ARG, "> 0"),
    (dict(scale=-1.0), ut.UT_ERR_INVALID_ARG, "> 0"),
])
def test_fwd_varlen_rejects_bad_arguments(kw, status, msg):
    assert _fwd_varlen(**kw) == status
    assert msg in ut.last_error()


def test_varlen_with_no_tokens_launches_nothing():
    # T = 0: checked, then nothing to do (the fake pointers are never touched)
    assert _fwd_varlen(T=0, q=None) == ut.UT_OK
    lib = ut.lib()
    args = [FAKE] * 10 + [3, 0, 128, 2, 128, 128] + [FAKE] * 4 + [0.1]
    assert lib.ut_bsattn_bwd_varlen(*args, None, 0, None) == ut.UT_OK


def test_bwd_varlen_rejects_missing_workspace():
    lib = ut.lib()
    args = [FAKE] * 10 + [3, 300, 128, 2, 128, 128] + [FAKE] * 4 + [0.1]
    assert lib.ut_bsattn_bwd_varlen(*args, None, 0, None) == ut.UT_ERR_WORKSPACE
    assert lib.ut_bsattn_bwd_varlen(*args, FAKE, 300 * 2 * 8 - 1, None) == ut.UT_ERR_WORKSPACE
    args[9] = None
    assert lib.ut_bsattn_bwd_varlen(*args, FAKE, 4800, None) == ut.UT_ERR_INVALID_ARG
    assert "cu_seqlens" in ut.last_error()


def test_drop_background_rejects_bad_arguments():
    lib = ut.lib()
    ws = ut.ut_drop_background_workspace_size(1000)
    call = lambda **kw: lib.ut_drop_background(
        kw.get("mask", FAKE), kw.get("L", 1000), kw.get("xf", FAKE), kw.get("rb", 6144),
        kw.get("xp", FAKE), kw.get("cap", 1000), kw.get("kept", FAKE), kw.get("inv", None),
        kw.get("n", FAKE), None, kw.get("ws", FAKE), kw.get("wsb", ws), None)
    assert call(L=0) == ut.UT_ERR_INVALID_ARG
    assert call(L=1 << 31) == ut.UT_ERR_INVALID_ARG
    assert call(rb=100) == ut.UT_ERR_INVALID_ARG and "multiple of 16" in ut.last_error()
    assert call(xp=None) == ut.UT_ERR_INVALID_ARG
    assert call(xf=MISALIGNED) == ut.UT_ERR_INVALID_ARG
    assert call(mask=None) == ut.UT_ERR_INVALID_ARG
    assert call(cap=-1) == ut.UT_ERR_INVALID_ARG
    assert call(wsb=ws - 1) == ut.UT_ERR_WORKSPACE
    assert call(ws=None) == ut.UT_ERR_WORKSPACE


def test_scatter_and_block_index_reject_bad_arguments():
    lib = ut.lib()
    assert lib.ut_scatter_foreground(FAKE, FAKE, 10, 24, FAKE, None) == ut.UT_ERR_INVALID_ARG
    assert lib.ut_scatter_foreground(FAKE, FAKE, -1, 32, FAKE, None) == ut.UT_ERR_INVALID_ARG
    assert lib.ut_scatter_foreground(None, None, 0, 32, None, None) == ut.UT_OK   # no-op
    assert lib.ut_scatter_foreground(FAKE, FAKE, 10, 32, MISALIGNED, None) == ut.UT_ERR_INVALID_ARG
    bi = lambda B=1, H=2, Nq=5, Nk=5, mask=FAKE, rp=FAKE, cap=50: lib.ut_build_block_index(
        mask, B, H, Nq, Nk, rp, FAKE, FAKE, FAKE, cap, None, None, 0, None)
    assert bi(Nq=0) == ut.UT_ERR_INVALID_ARG
    assert bi(mask=None) == ut.UT_ERR_INVALID_ARG
    assert bi(rp=MISALIGNED) == ut.UT_ERR_INVALID_ARG
    assert bi(cap=-1) == ut.UT_ERR_INVALID_ARG
    assert bi(B=300, H=300) == ut.UT_ERR_INVALID_ARG and "65535" in ut.last_error()
    # 2^31 mask entries would wrap the int32 list offsets
    assert bi(B=1, H=2, Nq=32768, Nk=32768) == ut.UT_ERR_INVALID_ARG
    assert "2^31" in ut.last_error()
    assert bi(B=1, H=2, Nq=32768, Nk=32767, mask=None) == ut.UT_ERR_INVALID_ARG   # just below


def test_block_index_needs_no_workspace():
    for shape in ((1, 24, 603, 603), (1, 1, 1, 1), (2, 2, 70, 65)):
        assert ut.ut_build_block_index_workspace_size(*shape) == 0
    lib = ut.lib()
    # a NULL workspace of 0 bytes passes the checks (a NULL mask is then the error)
    st = lib.ut_build_block_index(None, 1, 2, 5, 5, FAKE, FAKE, FAKE, FAKE, 50, None, None, 0, None)
    assert st == ut.UT_ERR_INVALID_ARG and "block_mask is NULL" in ut.last_error()


def test_binding_refuses_host_tensors():
    import torch
    q = torch.zeros((1, 64, 1, 64), dtype=torch.bfloat16)
    idx = torch.zeros(2, dtype=torch.int32)
    with pytest.raises(ValueError):
        ut.ut_bsattn_fwd(q, q, q, q, torch.zeros(64), 64, idx, idx, 0.125)


def test_topk_block_mask_rejects_bad_arguments():
    lib = ut.lib()
    assert ut.ut_topk_block_mask_workspace_size(1, 77060, 24, 128, 128) == 2 * 24 * 603 * 128 * 4
    assert ut.ut_topk_block_mask_workspace_size(1, 0, 24, 128, 128) == 0
    ws = ut.ut_topk_block_mask_workspace_size(1, 1000, 2, 64, 64)
    call = lambda **kw: lib.ut_topk_block_mask(
        kw.get("q", FAKE), kw.get("k", FAKE), kw.get("B", 1), kw.get("N", 1000), kw.get("H", 2),
        kw.get("D", 64), kw.get("block", 64), kw.get("kk", 3), kw.get("P", 0), kw.get("m", FAKE),
        kw.get("ws", FAKE), kw.get("wsb", ws), None)
    for kw, status, msg in [
        (dict(N=0), ut.UT_ERR_INVALID_ARG, ">= 1"),
        (dict(block=0), ut.UT_ERR_INVALID_ARG, ">= 1"),
        (dict(D=60), ut.UT_ERR_INVALID_ARG, "multiple of 8"),
        (dict(D=520), ut.UT_ERR_INVALID_ARG, "multiple of 8"),
        (dict(kk=0), ut.UT_ERR_INVALID_ARG, "k_keep"),
        (dict(P=-1), ut.UT_ERR_INVALID_ARG, "prefix_blocks"),
        (dict(P=17), ut.UT_ERR_INVALID_ARG, "prefix_blocks"),
        (dict(B=70000), ut.UT_ERR_INVALID_ARG, "65535"),
        (dict(q=None), ut.UT_ERR_INVALID_ARG, "q is NULL"),
        (dict(k=MISALIGNED), ut.UT_ERR_INVALID_ARG, "aligned"),
        (dict(m=None), ut.UT_ERR_INVALID_ARG, "block_mask is NULL"),
        (dict(ws=None), ut.UT_ERR_WORKSPACE, "workspace"),
        (dict(wsb=ws - 1), ut.UT_ERR_WORKSPACE, "workspace"),
        # 20000 blocks of one token: a score row of 80 KB does not fit one workgroup
        (dict(N=20000, block=1, wsb=1 << 40), ut.UT_ERR_UNSUPPORTED, "do not fit"),
    ]:
        assert call(**kw) == status, kw
        assert msg in ut.last_error(), (kw, ut.last_error())


def test_foreground_step_calls_reject_bad_arguments():
    lib = ut.lib()
    assert ut.ut_fg_flow_loss_workspace_size() == 1024 * 8
    eu = lambda **kw: lib.ut_euler_update_foreground(
        kw.get("z", FAKE), kw.get("L", 1000), kw.get("C", 64), kw.get("v", FAKE), kw.get("vt", ut.UT_BF16),
        kw.get("kept", FAKE), kw.get("n", 10), kw.get("dt", -0.1), None)
    for kw, msg in [(dict(L=0), "L must"), (dict(C=6), "multiple of 4"), (dict(C=0), "multiple of 4"),
                    (dict(n=-1), "n_kept"), (dict(n=1001), "n_kept"), (dict(vt=7), "dtype"),
                    (dict(dt=float("inf")), "finite"), (dict(z=None), "z is NULL"),
                    (dict(z=MISALIGNED), "aligned"), (dict(kept=None), "kept_idx is NULL"),
                    (dict(v=ctypes.c_void_p(0x10004), vt=ut.UT_F32), "aligned")]:
        assert eu(**kw) == ut.UT_ERR_INVALID_ARG, kw
        assert msg in ut.last_error(), (kw, ut.last_error())
    assert eu(n=0, z=None, kept=None, v=None) == ut.UT_OK      # nothing to do
    ws = ut.ut_fg_flow_loss_workspace_size()
    lo = lambda **kw: lib.ut_fg_flow_loss(
        kw.get("v", FAKE), kw.get("vt", ut.UT_BF16), kw.get("e", FAKE), kw.get("z0", FAKE),
        kw.get("xt", ut.UT_F32), kw.get("L", 1000), kw.get("C", 64), kw.get("kept", FAKE), kw.get("n", 10),
        kw.get("loss", FAKE), kw.get("grad", None), kw.get("ws", FAKE), kw.get("wsb", ws), None)
    for kw, status, msg in [(dict(xt=5), ut.UT_ERR_INVALID_ARG, "dtype"),
                            (dict(loss=None), ut.UT_ERR_INVALID_ARG, "loss is NULL"),
                            (dict(e=None), ut.UT_ERR_INVALID_ARG, "eps is NULL"),
                            (dict(grad=MISALIGNED), ut.UT_ERR_INVALID_ARG, "aligned"),
                            (dict(ws=None), ut.UT_ERR_WORKSPACE, "workspace"),
                            (dict(wsb=ws - 8), ut.UT_ERR_WORKSPACE, "workspace")]:
        assert lo(**kw) == status, kw
        assert msg in ut.last_error(), (kw, ut.last_error())


def test_composite_and_token_mask_reject_bad_arguments():
    lib = ut.lib()
    co = lambda **kw: lib.ut_composite_latent(
        kw.get("xp", FAKE), kw.get("n", 10), kw.get("inv", FAKE), kw.get("L", 100), kw.get("bg", FAKE),
        kw.get("P", 16), kw.get("rb", 256), kw.get("out", FAKE), None)
    for kw, msg in [(dict(L=0), "L must"), (dict(P=0), "bg_rows"), (dict(n=101), "n_kept"),
                    (dict(rb=100), "multiple of 16"), (dict(xp=None), "x_packed is NULL"),
                    (dict(inv=None), "inv_idx is NULL"), (dict(out=MISALIGNED), "aligned")]:
        assert co(**kw) == ut.UT_ERR_INVALID_ARG, kw
        assert msg in ut.last_error(), (kw, ut.last_error())
    assert ut.ut_token_mask_workspace_size(7, 2048, 2048, 16) == 7 * 128 * 128
    tm = lambda **kw: lib.ut_token_mask_from_alpha(
        kw.get("a", FAKE), kw.get("V", 2), kw.get("H", 64), kw.get("W", 96), kw.get("p", 16),
        kw.get("t", 0), kw.get("r", 1), kw.get("m", FAKE), kw.get("ws", FAKE), kw.get("wsb", 2 * 4 * 6), None)
    for kw, status, msg in [(dict(p=8), ut.UT_ERR_INVALID_ARG, "patch"),
                            (dict(W=100), ut.UT_ERR_INVALID_ARG, "patch"),
                            (dict(t=256), ut.UT_ERR_INVALID_ARG, "threshold"),
                            (dict(r=-1), ut.UT_ERR_INVALID_ARG, "radius"),
                            (dict(a=MISALIGNED), ut.UT_ERR_INVALID_ARG, "aligned"),
                            (dict(m=None), ut.UT_ERR_INVALID_ARG, "token_mask is NULL"),
                            (dict(wsb=47), ut.UT_ERR_WORKSPACE, "workspace")]:
        assert tm(**kw) == status, kw
        assert msg in ut.last_error(), (kw, ut.last_error())
