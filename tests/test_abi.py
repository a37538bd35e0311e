"""C-ABI tests that need no GPU: the library loads, exports every symbol that
include/sparstar.h declares, and rejects invalid arguments on the host before
any HIP call (the fake device pointers below are never dereferenced)."""
import ctypes
import os
import re

import pytest

from paper_2608_10519_amd import sparstar as S

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "sparstar.h")

FAKE = 0x10000  # a 256-byte aligned, never-dereferenced "device" address


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(S.LIB_PATH):
        pytest.fail("libsparstar.so is not built (run __graft_entry__.build())")
    return S.load()


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(sparstar_[a-z_]+)\s*\(", text)))


def test_exports_every_declared_symbol(lib):
    names = _declared()
    assert {"sparstar_score_blocks", "sparstar_sparse_attn_fwd", "sparstar_dense_attn_fwd",
            "sparstar_score_workspace_bytes", "sparstar_attn_workspace_bytes", "sparstar_kv_stride",
            "sparstar_last_error"} <= set(names)
    for n in names:
        assert hasattr(lib, n), n


def test_workspace_bytes(lib):
    # 720p: qbar 24*1125*128*4, kbar 24*2258*128*4, their scales 24*1125*4 and
    # 24*2258*4, S 24*1125*2272*4 (rows of 2258 floats padded to 2272;
    # 256-aligned regions)
    al = lambda x: (x + 255) // 256 * 256
    want = (al(24 * 1125 * 128 * 4) + al(24 * 2258 * 128 * 4) + al(24 * 1125 * 4) + al(24 * 2258 * 4)
            + al(24 * 1125 * 2272 * 4))
    assert S.sparstar_score_workspace_bytes(1, 24, 72_000, 144_512, 128, 64) == want
    assert S.sparstar_score_workspace_bytes(1, 24, 72_000, 144_512, 96, 64) == 0
    assert S.sparstar_score_workspace_bytes(0, 24, 72_000, 144_512, 128, 64) == 0


@pytest.mark.parametrize("H,Lk,b,budget,keep,want", [
    (24, 144_512, 64, 0.25, [(72_000, 72_512)], 8 + 563),
    (24, 144_512, 64, 0.10, [(72_000, 72_512)], 8 + 225),
    (24, 144_512, 64, 0.14, [(72_000, 72_512)], 8 + 315),       # 0.14 * 2250 = 315.00000000000006 in binary
    (24, 144_512, 128, 0.25, [(72_000, 72_512)], 5 + 281),      # n_k = 1129, 5 straddling text blocks, n_sel 1124
    (2, 1152, 64, 0.25, [(512, 640)], 2 + 4),
    (2, 1152, 64, 0.25, [(512, 640), (0, 512)], 10 + 2),         # clip 1: text + reference
    (3, 1152, 64, [0.0, 1.0, 0.5], [(512, 640)], 2 + 16),        # per-head: max k = 16
    (1, 1152, 64, 0.5, [(0, 1152)], 18 + 0),                     # n_sel = 0
    (1, 1152, 64, 0.5, [], 0 + 9),
])
def test_kv_stride_matches_eq3_to_5(lib, H, Lk, b, budget, keep, want):
    assert S.sparstar_kv_stride(H, Lk, b, budget, keep) == want


def _score(lib, **over):
    a = dict(q=FAKE, k=FAKE, B=1, H=2, Lq=512, Lk=1152, D=64, block=64, budget=[0.25], keep=[(512, 640)],
             num=FAKE, idx=FAKE, stride=6, scores=None, ws=FAKE,
             ws_bytes=S.sparstar_score_workspace_bytes(1, 2, 512, 1152, 64, 64))
    a.update(over)
    bud = None if a["budget"] is None else (ctypes.c_double * len(a["budget"]))(*a["budget"])
    nb = over.get("n_budget", 0 if a["budget"] is None else len(a["budget"]))
    kr = (S.Range * max(1, len(a["keep"])))(*[S.Range(x, y) for x, y in a["keep"]]) if a["keep"] else None
    nk = over.get("n_keep", len(a["keep"]))
    return lib.sparstar_score_blocks(a["q"], a["k"], a["B"], a["H"], a["Lq"], a["Lk"], a["D"], a["block"], bud, nb,
                                     kr, nk, a["num"], a["idx"], a["stride"], a["scores"], a["ws"], a["ws_bytes"],
                                     None)


@pytest.mark.parametrize("over,code,msg", [
    (dict(q=None), S.ERR_INVALID_ARG, "non-null"),
    (dict(q=FAKE + 2), S.ERR_INVALID_ARG, "aligned"),
    (dict(num=None), S.ERR_INVALID_ARG, "kv_num_blocks"),
    (dict(D=96), S.ERR_UNSUPPORTED, "head dim"),
    (dict(block=32), S.ERR_UNSUPPORTED, "block size"),
    (dict(B=0), S.ERR_INVALID_ARG, "B and H"),
    (dict(H=300, budget=[0.25]), S.ERR_UNSUPPORTED, "H must be"),
    (dict(Lk=0), S.ERR_INVALID_ARG, "Lk"),
    (dict(Lq=-1), S.ERR_INVALID_ARG, "Lq"),
    (dict(budget=[1.5]), S.ERR_INVALID_ARG, "outside [0, 1]"),
    (dict(budget=[-0.1]), S.ERR_INVALID_ARG, "outside [0, 1]"),
    (dict(budget=[float("nan")]), S.ERR_INVALID_ARG, "outside [0, 1]"),
    (dict(budget=None), S.ERR_INVALID_ARG, "budget"),
    (dict(budget=[0.1, 0.2, 0.3]), S.ERR_INVALID_ARG, "n_budget"),
    (dict(keep=[(600, 500)]), S.ERR_INVALID_ARG, "keep[0]"),
    (dict(keep=[(0, 2000)]), S.ERR_INVALID_ARG, "keep[0]"),
    (dict(keep=[(-1, 5)]), S.ERR_INVALID_ARG, "keep[0]"),
    (dict(keep=[(0, 1)] * 9), S.ERR_INVALID_ARG, "n_keep"),
    (dict(keep=[], n_keep=2), S.ERR_INVALID_ARG, "keep is null"),
    (dict(stride=5), S.ERR_INVALID_ARG, "kv_stride"),
    (dict(ws=None), S.ERR_WORKSPACE, "workspace"),
    (dict(ws=FAKE + 16), S.ERR_WORKSPACE, "256-byte"),
    (dict(ws_bytes=100), S.ERR_WORKSPACE, "required"),
])
def test_score_blocks_rejects_invalid_arguments(lib, over, code, msg):
    assert _score(lib, **over) == code
    assert msg in S.last_error()


def _score_fused(lib, **over):
    a = dict(q=FAKE, k=FAKE, B=1, H=2, Lq=512, Lk=1152, D=64, block=64, budget=[0.25], keep=[(0, 128)], num=FAKE,
             idx=FAKE, stride=6, ws=FAKE, ws_bytes=1 << 40)
    a.update(over)
    bud = (ctypes.c_double * len(a["budget"]))(*a["budget"])
    kr = (S.Range * len(a["keep"]))(*[S.Range(x, y) for x, y in a["keep"]])
    return lib.sparstar_score_blocks_fused(a["q"], a["k"], a["B"], a["H"], a["Lq"], a["Lk"], a["D"], a["block"],
                                           bud, len(a["budget"]), kr, len(a["keep"]), a["num"], a["idx"],
                                           a["stride"], a["ws"], a["ws_bytes"], None)


@pytest.mark.parametrize("over,code,msg", [
    (dict(D=96), S.ERR_UNSUPPORTED, "head dim"),
    (dict(stride=5), S.ERR_INVALID_ARG, "kv_stride"),
    (dict(ws=None), S.ERR_WORKSPACE, "workspace"),
    # one key block past the fused kernel's LDS rows
    (dict(Lk=64 * S.FUSED_MAX_BLOCKS + 1, stride=1000), S.ERR_UNSUPPORTED, "at most 2304"),
])
def test_score_blocks_fused_rejects_invalid_arguments(lib, over, code, msg):
    assert _score_fused(lib, **over) == code
    assert msg in S.last_error()


def _score_static(lib, **over):
    a = dict(q=FAKE, k=FAKE, B=1, H=2, Lq=512, Lk=1152, D=64, block=64, budget=[0.25], keep=[(0, 128)], num=FAKE,
             idx=FAKE, stride=6, scores=None)
    a.update(over)
    bud = (ctypes.c_double * len(a["budget"]))(*a["budget"]) if a["budget"] is not None else None
    kr = (S.Range * max(1, len(a["keep"])))(*[S.Range(x, y) for x, y in a["keep"]])
    return lib.sparstar_score_blocks_static(a["q"], a["k"], a["B"], a["H"], a["Lq"], a["Lk"], a["D"], a["block"],
                                            bud, len(a["budget"]) if a["budget"] is not None else 1, kr,
                                            a.get("n_keep", len(a["keep"])), a["num"], a["idx"], a["stride"],
                                            a["scores"], None)


@pytest.mark.parametrize("over,code,msg", [
    (dict(D=96), S.ERR_UNSUPPORTED, "head dim"),
    (dict(q=FAKE + 2), S.ERR_INVALID_ARG, "16-byte"),
    (dict(budget=[1.5]), S.ERR_INVALID_ARG, "outside [0, 1]"),
    (dict(keep=[(0, 2000)]), S.ERR_INVALID_ARG, "keep[0]"),
    (dict(stride=5), S.ERR_INVALID_ARG, "kv_stride"),
    (dict(scores=FAKE + 2), S.ERR_INVALID_ARG, "scores"),
    # the 720p shape (24 heads, 72,000 queries, 144,512 keys, D 128): qbar + kbar, scales and S = 287 MB
    (dict(H=24, Lq=72_000, Lk=144_512, D=128, keep=[(72_000, 72_512)], stride=571), S.ERR_WORKSPACE,
     "more than the 67108864 bytes"),
])
def test_score_blocks_static_rejects_before_any_hip_call(lib, over, code, msg):
    """Every argument, the static scratch's size included, is checked on the host
    first: without a GPU these calls return their own error, never a HIP one."""
    assert _score_static(lib, **over) == code
    assert msg in S.last_error()


def test_score_blocks_static_scratch_limit():
    """With `scores` given, S stays out of the static scratch: at the 720p shape
    qbar + kbar and their scales (41.9 MB) fit, which the next check (a too-small
    stride) shows."""
    lib = S.load()
    big = dict(H=24, Lq=72_000, Lk=144_512, D=128, keep=[(72_000, 72_512)])
    assert _score_static(lib, **big, stride=5, scores=FAKE) == S.ERR_INVALID_ARG
    assert "kv_stride" in S.last_error()
    assert _score_static(lib, **big, stride=571) == S.ERR_WORKSPACE
    # an empty query side is a no-op that makes no HIP call
    assert _score_static(lib, Lq=0) == S.OK and S.last_error() == ""


def test_score_blocks_fused_takes_the_limit_on_an_empty_query_side(lib):
    # Lq = 0 is a no-op that touches no device memory, after the size checks
    assert _score_fused(lib, Lq=0, Lk=64 * S.FUSED_MAX_BLOCKS, stride=1000) == S.OK


def _attn(lib, dense=False, **over):
    a = dict(q=FAKE, k=FAKE, v=FAKE, B=1, H=2, Lq=512, Lk=1152, D=64, block=64, num=FAKE, idx=FAKE, stride=6,
             scale=0.0, o=FAKE, lse=None, ws=None, ws_bytes=0)
    a.update(over)
    if dense:
        return lib.sparstar_dense_attn_fwd(a["q"], a["k"], a["v"], a["B"], a["H"], a["Lq"], a["Lk"], a["D"],
                                           a["block"], a["scale"], a["o"], a["lse"], a["ws"], a["ws_bytes"], None)
    return lib.sparstar_sparse_attn_fwd(a["q"], a["k"], a["v"], a["B"], a["H"], a["Lq"], a["Lk"], a["D"], a["block"],
                                        a["num"], a["idx"], a["stride"], a["scale"], a["o"], a["lse"], a["ws"],
                                        a["ws_bytes"], None)


def test_attn_workspace_bytes(lib):
    # 720p: 24 heads x 1125 query blocks x 16 key ranges x 64 rows: fp16 partial P V [.., 128] + four fp32
    # per row (running max, the two row sums, the row's scale exponent)
    rows = 24 * 1125 * 16 * 64
    want = (rows * 128 * 2 + 255) // 256 * 256 + rows * 16
    assert S.sparstar_attn_workspace_bytes(1, 24, 72_000, 144_512, 128, 64) == want
    # fewer than 16 key blocks: no split, no workspace
    assert S.sparstar_attn_workspace_bytes(1, 2, 512, 960, 64, 64) == 0
    assert S.sparstar_attn_workspace_bytes(1, 2, 512, 1152, 64, 64) > 0


@pytest.mark.parametrize("dense", [False, True])
@pytest.mark.parametrize("over", [dict(ws=FAKE, ws_bytes=100), dict(ws=FAKE + 16, ws_bytes=1 << 30)])
def test_attention_rejects_bad_workspace(lib, dense, over):
    assert _attn(lib, dense=dense, **over) == S.ERR_WORKSPACE
    assert "workspace" in S.last_error()


@pytest.mark.parametrize("dense", [False, True])
@pytest.mark.parametrize("over,code", [
    (dict(v=None), S.ERR_INVALID_ARG),
    (dict(o=FAKE + 8), S.ERR_INVALID_ARG),
    (dict(lse=FAKE + 2), S.ERR_INVALID_ARG),
    (dict(D=256), S.ERR_UNSUPPORTED),
    (dict(block=256), S.ERR_UNSUPPORTED),
    (dict(scale=float("inf")), S.ERR_INVALID_ARG),
    (dict(scale=float("nan")), S.ERR_INVALID_ARG),
    (dict(H=0), S.ERR_INVALID_ARG),
])
def test_attention_rejects_invalid_arguments(lib, dense, over, code):
    assert _attn(lib, dense=dense, **over) == code
    assert S.last_error()


@pytest.mark.parametrize("over", [dict(num=None), dict(idx=None), dict(stride=0)])
def test_sparse_attention_needs_lists(lib, over):
    assert _attn(lib, **over) == S.ERR_INVALID_ARG


def test_python_binding_raises_without_library(tmp_path):
    with pytest.raises(RuntimeError, match="not found"):
        S.load(str(tmp_path / "missing.so"))


def test_last_error_is_cleared_by_success(lib):
    assert _score(lib, q=None) == S.ERR_INVALID_ARG
    assert S.last_error()
    assert S.sparstar_kv_stride(2, 1152, 64, 0.25, [(512, 640)]) == 6
    assert S.last_error() == ""


def test_token_topk_workspace_bytes(lib):
    # fp32 logits [B, H, n_rows, Lk]
    assert S.sparstar_token_topk_workspace_bytes(1, 24, 144_512, 8) == 24 * 8 * 144_512 * 4
    assert S.sparstar_token_topk_workspace_bytes(1, 2, 100, 0) == 0
    assert S.sparstar_token_topk_workspace_bytes(1, 2, 100, S.MAX_MASS_ROWS + 1) == 0
    assert S.sparstar_token_topk_workspace_bytes(300, 300, 100, 1) == 0  # B * H above 65535


def _topk(lib, **over):
    import ctypes

    a = dict(q=FAKE, k=FAKE, B=1, H=2, Lq=512, Lk=1152, D=64, rows=[0, 5, 511], ntok=FAKE, lse=FAKE, scale=0.0,
             mass=FAKE, ws=FAKE, ws_bytes=1 << 30)
    a.update(over)
    rows = a["rows"]
    arr = (ctypes.c_int64 * max(1, len(rows)))(*rows) if rows is not None else None
    return lib.sparstar_token_topk_mass(a["q"], a["k"], a["B"], a["H"], a["Lq"], a["Lk"], a["D"], arr,
                                        len(rows) if rows is not None else 1, a["ntok"], a["lse"], a["scale"],
                                        a["mass"], a["ws"], a["ws_bytes"], None)


@pytest.mark.parametrize("over,code,msg", [
    (dict(q=None), S.ERR_INVALID_ARG, "non-null"),
    (dict(rows=None), S.ERR_INVALID_ARG, "non-null"),
    (dict(ntok=None), S.ERR_INVALID_ARG, "non-null"),
    (dict(k=FAKE + 8), S.ERR_INVALID_ARG, "16-byte"),
    (dict(lse=FAKE + 2), S.ERR_INVALID_ARG, "4-byte"),
    (dict(rows=[0, 512]), S.ERR_INVALID_ARG, "outside"),
    (dict(rows=[-1]), S.ERR_INVALID_ARG, "outside"),
    (dict(rows=[]), S.ERR_INVALID_ARG, "n_rows"),
    (dict(rows=list(range(17))), S.ERR_INVALID_ARG, "n_rows"),
    (dict(D=96), S.ERR_UNSUPPORTED, "head dim"),
    (dict(Lq=0), S.ERR_INVALID_ARG, "Lq"),
    (dict(scale=float("nan")), S.ERR_INVALID_ARG, "finite"),
    (dict(ws=None), S.ERR_WORKSPACE, "null"),
    (dict(ws_bytes=100), S.ERR_WORKSPACE, "required"),
])
def test_token_topk_mass_rejects_invalid_arguments(lib, over, code, msg):
    assert _topk(lib, **over) == code
    assert msg in S.last_error()


@pytest.mark.parametrize("args,msg", [
    ((FAKE, FAKE, -1, FAKE), ">= 0"),
    ((None, FAKE, 4, FAKE), "non-null"),
    ((FAKE, FAKE, 4, FAKE + 2), "4-byte"),
])
def test_retained_mass_rejects_invalid_arguments(lib, args, msg):
    assert lib.sparstar_retained_mass(*args, None) == S.ERR_INVALID_ARG
    assert msg in S.last_error()


def test_retained_mass_empty_is_noop(lib):
    # n = 0 launches nothing, so it succeeds without a device
    assert lib.sparstar_retained_mass(None, None, 0, None, None) == S.OK
