"""Host-side tests of the C ABI (no GPU): the library loads, exports every symbol the
header declares, and every argument / shape / order / alignment / workspace error
is returned before any HIP call.  Workspace sizes do not depend on V."""
import ctypes
import os
import re

import pytest

import paper_2609_14306_amd as vp

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "vpce.h")

pytestmark = pytest.mark.skipif(not os.path.exists(vp.LIB_PATH),
                                reason="libvpce.so not built (run __graft_entry__.build())")

FAKE = 0x100000  # an aligned, never-dereferenced pointer value for validation tests


def declared_functions():
    src = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:vp_status|const char\*|int)\s+(vp_\w+)\s*\(", src, re.M)))


def test_header_declarations_match_binding():
    assert declared_functions() == sorted(vp.EXPORTED)


def test_library_exports_every_declared_symbol():
    lib = vp.load_library()
    for name in declared_functions():
        assert hasattr(lib, name), name
    assert vp.vp_abi_version() == 1


def test_status_strings():
    for s in range(10):
        assert vp.vp_status_str(s)
    assert vp.vp_status_str(0) == "ok"


def _prob(**kw):
    base = dict(T=4096, d=2880, shard_rows=[25136] * 8, dtype=vp.VP_BF16)
    base.update(kw)
    return vp.Problem(**base)


def test_workspace_size_independent_of_V():
    sizes = set()
    for V in (32768, 65536, 131072, 201088, 262144):
        rows = [V // 8] * 8
        sizes.add(vp.vp_ce_workspace_size(_prob(T=32768, shard_rows=rows)))
    assert len(sizes) == 1, sizes
    fwd, bwd = sizes.pop()
    T, d, eb = 32768, 2880, 2
    # forward: per-split (m, s) and the target logit per token
    assert 0 < fwd <= (2 * 32 + 1) * T * 4 + 4096
    # backward: two strip layouts, double buffered (default budget 100 Mi elements
    # each), H^T and one vocabulary chunk of W^T (at most 32768 rows)
    assert 0 < bwd <= 4 * (100 << 20) * eb + T * d * eb + d * 32768 * eb + 8192


def _forward_splits(T, d, dtype, shard_rows=(25136,) * 8):
    """The forward's vocabulary split count S, read back from its workspace size:
    256 header bytes, S partial maxima and sums per token, one target logit per token."""
    fwd, _ = vp.vp_ce_workspace_size(_prob(T=T, d=d, dtype=dtype, shard_rows=list(shard_rows)))
    a256 = lambda x: (x + 255) // 256 * 256
    body = fwd - 256 - a256(T * 4)
    S = body // 2 // (T * 4)
    assert 2 * a256(S * T * 4) == body
    return S


@pytest.mark.parametrize("T, d, dtype, S", [
    (256, 256, vp.VP_F32, 32),        # one token block: splits fill the CUs, at most 32
    (4096, 2880, vp.VP_BF16, 16),     # 16 token blocks: 16 splits fill 256 CUs
    (32768, 2880, vp.VP_BF16, 4),     # at least 4: 32 concurrent tiles share 12 panels
    (16384, 7168, vp.VP_BF16, 8),     # 64 H panels of 3.7 MB would overflow the cache budget
    (65536, 4096, vp.VP_BF16, 4),     # 64 H panels of 2 MB fit; 2 splits would not
    (16384, 7168, vp.VP_F32, 16),     # float32 panels are twice the bytes
])
def test_forward_split_rule(T, d, dtype, S):
    assert _forward_splits(T, d, dtype) == S


def test_largest_accepted_shapes():
    fwd, bwd = vp.vp_ce_workspace_size(_prob(T=(1 << 23) - 256))
    assert fwd > 0 and bwd > 0
    fwd, bwd = vp.vp_ce_workspace_size(_prob(T=16, d=1 << 22))
    assert fwd > 0 and bwd > 0


def test_plan_info():
    # long-context shape: 8192-token strips, shards of 25136 rows cut in two chunks
    info = vp.vp_ce_plan_info(_prob(T=32768))
    assert info["Tc"] == 8192 and info["Vc"] == 12800
    assert info["strips"] == 8 * 2 * 4 and info["stage_launches"] == 65
    assert vp.vp_ce_plan_info(_prob(T=0))["stage_launches"] == 0
    one = vp.vp_ce_plan_info(_prob(T=1, shard_rows=[100, 0, 5]))
    assert one["strips"] == 2 and one["stage_launches"] == 3
    with pytest.raises(vp.VpError):
        vp.vp_ce_plan_info(_prob(T=-1))
    lib = vp.load_library()
    assert lib.vp_ce_plan_info(ctypes.byref(_prob().c), None) == vp.VP_ERR_NULL


def test_workspace_respects_strip_budget():
    T, d = 4096, 2880
    _, small = vp.vp_ce_workspace_size(_prob(T=T, d=d, strip_elems=1 << 20))
    _, big = vp.vp_ce_workspace_size(_prob(T=T, d=d, strip_elems=1 << 26))
    fixed = T * d * 2  # H^T
    assert small < big
    # strips (2 layouts x 2 buffers x budget) plus W^T of a chunk (at most
    # budget / 256 rows here) plus H^T
    assert small - fixed <= 4 * (1 << 21) + d * ((1 << 20) // 256) * 2 + 8192


@pytest.mark.parametrize("kw,status", [
    (dict(T=-1), vp.VP_ERR_SHAPE),
    (dict(d=0), vp.VP_ERR_SHAPE),
    (dict(d=12), vp.VP_ERR_SHAPE),
    (dict(T=(1 << 23) - 255), vp.VP_ERR_SHAPE),
    (dict(d=(1 << 22) + 8), vp.VP_ERR_SHAPE),
    (dict(shard_rows=[]), vp.VP_ERR_SHAPE),
    (dict(shard_rows=[1] * 65), vp.VP_ERR_SHAPE),
    (dict(shard_rows=[0, 0]), vp.VP_ERR_SHAPE),
    (dict(shard_rows=[5, -1]), vp.VP_ERR_SHAPE),
    (dict(dtype=7), vp.VP_ERR_DTYPE),
    (dict(shard_rows=[4, 4], order=[0, 0]), vp.VP_ERR_ORDER),
    (dict(shard_rows=[4, 4], order=[0, 2]), vp.VP_ERR_ORDER),
    (dict(strip_elems=-5), vp.VP_ERR_SHAPE),
])
def test_invalid_problem(kw, status):
    with pytest.raises(vp.VpError) as e:
        vp.vp_ce_workspace_size(_prob(**kw))
    assert e.value.status == status


def _fwd(prob, H=FAKE, W=(FAKE,), t=FAKE, loss=FAKE, lse=FAKE, ws=FAKE, ws_bytes=None):
    lib = vp.load_library()
    fwd_b, _ = vp.vp_ce_workspace_size(prob)
    arr = (ctypes.c_void_p * max(len(W), 1))(*W)
    return lib.vp_ce_forward(ctypes.byref(prob.c), H, arr, t, loss, lse, ws,
                             fwd_b if ws_bytes is None else ws_bytes, 0)


def _bwd(prob, H=FAKE, W=(FAKE,), t=FAKE, lse=FAKE, g=FAKE, dH=FAKE, dW=(FAKE,), ws=FAKE,
         ws_bytes=None):
    lib = vp.load_library()
    _, bwd_b = vp.vp_ce_workspace_size(prob)
    Wa = (ctypes.c_void_p * max(len(W), 1))(*W)
    dWa = (ctypes.c_void_p * max(len(dW), 1))(*dW)
    return lib.vp_ce_backward(ctypes.byref(prob.c), H, Wa, t, lse, g, dH, dWa, ws,
                              bwd_b if ws_bytes is None else ws_bytes, 0)


def test_forward_argument_errors_before_launch():
    p = _prob(shard_rows=[100])
    assert _fwd(p, ws=None) == vp.VP_ERR_WORKSPACE
    assert _fwd(p, ws_bytes=16) == vp.VP_ERR_WORKSPACE
    assert _fwd(p, ws=FAKE + 8) == vp.VP_ERR_ALIGN
    assert _fwd(p, H=FAKE + 2) == vp.VP_ERR_ALIGN
    assert _fwd(p, W=(FAKE + 4,)) == vp.VP_ERR_ALIGN
    assert _fwd(p, W=(None,)) == vp.VP_ERR_NULL
    assert _fwd(p, H=None) == vp.VP_ERR_NULL
    assert _fwd(p, t=None) == vp.VP_ERR_NULL
    assert _fwd(p, loss=None) == vp.VP_ERR_NULL
    assert _fwd(p, lse=None) == vp.VP_ERR_NULL
    lib = vp.load_library()
    assert lib.vp_ce_forward(None, FAKE, None, FAKE, FAKE, FAKE, FAKE, 1 << 30, 0) == vp.VP_ERR_NULL
    arr = (ctypes.c_void_p * 1)(FAKE)
    assert lib.vp_ce_forward(ctypes.byref(p.c), FAKE, None, FAKE, FAKE, FAKE, FAKE, 1 << 30,
                             0) == vp.VP_ERR_NULL
    del arr


def test_backward_argument_errors_before_launch():
    p = _prob(shard_rows=[100, 0])
    W = (FAKE, None)
    dW = (FAKE, None)
    assert _bwd(p, W=W, dW=dW, ws=None) == vp.VP_ERR_WORKSPACE
    assert _bwd(p, W=W, dW=dW, ws_bytes=255) == vp.VP_ERR_WORKSPACE
    assert _bwd(p, W=W, dW=(FAKE + 4, None)) == vp.VP_ERR_ALIGN
    assert _bwd(p, W=W, dW=(None, None)) == vp.VP_ERR_NULL
    assert _bwd(p, W=W, dW=dW, dH=None) == vp.VP_ERR_NULL
    assert _bwd(p, W=W, dW=dW, lse=None) == vp.VP_ERR_NULL
    assert _bwd(p, W=W, dW=dW, g=None) == vp.VP_ERR_NULL
    assert _bwd(p, W=W, dW=dW, dH=FAKE + 4) == vp.VP_ERR_ALIGN
    bad_order = _prob(shard_rows=[100, 0], order=[1, 1])
    lib = vp.load_library()
    Wa = (ctypes.c_void_p * 2)(*W)
    assert lib.vp_ce_backward(ctypes.byref(bad_order.c), FAKE, Wa, FAKE, FAKE, FAKE, FAKE, Wa, FAKE,
                              1 << 30, 0) == vp.VP_ERR_ORDER


def test_fold_argument_errors_before_launch():
    lib = vp.load_library()
    assert lib.vp_ce_state_init(FAKE, -1, 0) == vp.VP_ERR_SHAPE
    assert lib.vp_ce_state_init(None, 5, 0) == vp.VP_ERR_NULL
    assert lib.vp_ce_state_init(FAKE + 2, 5, 0) == vp.VP_ERR_ALIGN
    assert lib.vp_ce_state_init(None, 0, 0) == vp.VP_OK

    shard = _prob(shard_rows=[1000])
    fwd_b, _ = vp.vp_ce_workspace_size(shard)

    def fold(prob, off=0, H=FAKE, W=FAKE, t=FAKE, state=FAKE, ws=FAKE, ws_bytes=fwd_b):
        return lib.vp_ce_fold_shard(ctypes.byref(prob.c), off, H, W, t, state, ws, ws_bytes, 0)

    assert fold(_prob(shard_rows=[500, 500])) == vp.VP_ERR_SHAPE  # one shard per meeting
    assert fold(shard, off=-1) == vp.VP_ERR_SHAPE
    assert fold(shard, off=(1 << 31) - 1000) == vp.VP_ERR_SHAPE
    assert fold(shard, ws=None) == vp.VP_ERR_WORKSPACE
    assert fold(shard, ws_bytes=16) == vp.VP_ERR_WORKSPACE
    assert fold(shard, ws=FAKE + 8) == vp.VP_ERR_ALIGN
    assert fold(shard, H=None) == vp.VP_ERR_NULL
    assert fold(shard, W=None) == vp.VP_ERR_NULL
    assert fold(shard, t=None) == vp.VP_ERR_NULL
    assert fold(shard, state=None) == vp.VP_ERR_NULL
    assert fold(shard, state=FAKE + 2) == vp.VP_ERR_ALIGN
    assert fold(shard, W=FAKE + 4) == vp.VP_ERR_ALIGN
    # an empty shard or an empty batch is a no-op: nothing is launched, and no workspace
    # is needed (its size depends on T, d and dtype, which a caller may not have sized for)
    assert fold(_prob(shard_rows=[0]), W=None) == vp.VP_OK
    assert fold(_prob(shard_rows=[0]), W=None, ws=None, ws_bytes=0) == vp.VP_OK
    assert fold(_prob(T=0, shard_rows=[1000]), H=None, t=None, state=None) == vp.VP_OK
    assert fold(_prob(T=0, shard_rows=[1000]), H=None, t=None, state=None, ws=None,
                ws_bytes=0) == vp.VP_OK
    # the forward workspace depends on d and dtype as well as T (the split count does)
    f_small, _ = vp.vp_ce_workspace_size(_prob(T=65536, d=8, shard_rows=[1000]))
    f_wide, _ = vp.vp_ce_workspace_size(_prob(T=65536, d=7168, shard_rows=[1000]))
    assert f_small != f_wide
    assert fold(_prob(shard_rows=[0, 0])) == vp.VP_ERR_SHAPE

    full = _prob(shard_rows=[1000, 24])
    fin = lambda t=FAKE, state=FAKE, loss=FAKE, lse=FAKE, ws=FAKE, ws_bytes=256: \
        lib.vp_ce_fold_finalize(ctypes.byref(full.c), t, state, loss, lse, ws, ws_bytes, 0)
    assert fin(ws=None) == vp.VP_ERR_WORKSPACE
    assert fin(ws_bytes=255) == vp.VP_ERR_WORKSPACE
    assert fin(state=None) == vp.VP_ERR_NULL
    assert fin(t=None) == vp.VP_ERR_NULL
    assert fin(loss=None) == vp.VP_ERR_NULL
    assert fin(state=FAKE + 1) == vp.VP_ERR_ALIGN


def test_check_null_workspace():
    lib = vp.load_library()
    assert lib.vp_ce_check(None, None, None) == vp.VP_ERR_NULL


def test_forward_noalloc_refusals_before_launch():
    lib = vp.load_library()

    def call(prob, H=FAKE, W=None, t=FAKE, loss=FAKE, lse=FAKE):
        Wa = (ctypes.c_void_p * max(prob.P, 1))(*(W or [FAKE] * prob.P))
        return lib.vp_ce_forward_noalloc(ctypes.byref(prob.c), H, Wa, t, loss, lse, 0)

    # the problem's forward workspace exceeds the library's 16 MiB buffer
    big = _prob(T=(1 << 23) - 256, shard_rows=[1000])
    assert vp.vp_ce_workspace_size(big)[0] > 16 << 20
    assert call(big) == vp.VP_ERR_WORKSPACE
    p = _prob(shard_rows=[100])
    assert call(p, H=None) == vp.VP_ERR_NULL
    assert call(p, loss=None) == vp.VP_ERR_NULL
    assert call(p, H=FAKE + 2) == vp.VP_ERR_ALIGN
    assert call(p, W=[FAKE + 4]) == vp.VP_ERR_ALIGN
    assert lib.vp_ce_forward_noalloc(None, FAKE, None, FAKE, FAKE, FAKE, 0) == vp.VP_ERR_NULL
    assert call(_prob(shard_rows=[100], order=[1])) == vp.VP_ERR_ORDER
