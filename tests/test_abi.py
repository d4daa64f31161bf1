"""The C ABI without a GPU: the library loads, exports every symbol the header
declares, and rejects invalid arguments on the host before any HIP call."""
import ctypes
import os
import re

import pytest

import paper_2309_00754_amd as H
from paper_2309_00754_amd import _binding as Bd

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "hydra.h")

pytestmark = pytest.mark.skipif(not os.path.exists(H.LIB_PATH), reason="libhydra.so not built")

# Fake device addresses: never dereferenced, because every call below fails
# validation first.
P = 0x10000      # 16-byte aligned
P8 = 0x10008     # only 8-byte aligned


def _declared_functions():
    txt = open(HEADER).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"\b(hydra_[a-z0-9_]+)\s*\(", txt)))


def test_every_declared_symbol_is_exported():
    L = H.lib()
    declared = _declared_functions()
    assert sorted(Bd.EXPORTED) == declared
    for name in declared:
        assert hasattr(L, name), name


def test_abi_version_and_status_strings():
    assert H.lib().hydra_abi_version() == 1
    for code in (0, -1, -2, -3, -4, -5, -6):
        s = H.status_string(code)
        assert s.startswith("HYDRA_")
    assert "unknown" in H.status_string(7)


def _lin(x=P, W=P, A=P, B=P, s=2.0, M=32, N=64, K=64, r=8, y_off=P, y_on=P + 0x1000):
    return H.lib().hydra_lora_linear(x, W, A, B, s, M, N, K, r, y_off, y_on, None)


@pytest.mark.parametrize("kw,code", [
    (dict(x=None), H.HYDRA_ERR_NULL),
    (dict(W=None), H.HYDRA_ERR_NULL),
    (dict(y_off=None, y_on=None), H.HYDRA_ERR_NULL),
    (dict(A=None), H.HYDRA_ERR_NULL),
    (dict(B=None), H.HYDRA_ERR_NULL),
    (dict(M=0), H.HYDRA_ERR_SHAPE),
    (dict(N=-3), H.HYDRA_ERR_SHAPE),
    (dict(K=0), H.HYDRA_ERR_SHAPE),
    (dict(K=60), H.HYDRA_ERR_SHAPE),
    (dict(K=(1 << 21) + 8), H.HYDRA_ERR_SHAPE),
    (dict(M=1 << 31), H.HYDRA_ERR_SHAPE),
    (dict(r=-1), H.HYDRA_ERR_SHAPE),
    (dict(r=129), H.HYDRA_ERR_SHAPE),
    (dict(y_on=P), H.HYDRA_ERR_SHAPE),          # aliased outputs
    (dict(x=P8), H.HYDRA_ERR_ALIGN),
    (dict(W=P + 4), H.HYDRA_ERR_ALIGN),
    (dict(A=P8), H.HYDRA_ERR_ALIGN),
    (dict(B=P + 1), H.HYDRA_ERR_ALIGN),
    (dict(y_off=P + 2), H.HYDRA_ERR_ALIGN),
])
def test_lora_linear_rejects(kw, code):
    assert _lin(**kw) == code


def test_lora_linear_lora_pointers_unused_without_y_on():
    # With y_on == NULL the adapter is not needed: A/B NULL passes validation of
    # the adapter; the call is then only rejected here because x is misaligned.
    assert _lin(A=None, B=None, y_on=None, x=P8) == H.HYDRA_ERR_ALIGN


def _score(h=P, W=P, A=P, B=P, tok=P, w_rm=P, n_seq=4, seq_len=8, K=64, V=1000, r=8,
           lp_on=P, lp_off=P, kl=P, reward=P, lse_on=None, lse_off=None, ws=P, ws_bytes=None, err=None):
    if ws_bytes is None:
        ws_bytes = H.hydra_score_workspace_bytes(n_seq * seq_len, V) if n_seq > 0 and seq_len > 0 else 0
    return H.lib().hydra_score(h, W, A, B, 2.0, tok, w_rm, n_seq, seq_len, K, V, r, lp_on, lp_off, kl, reward,
                               lse_on, lse_off, ws, ws_bytes, err, None)


@pytest.mark.parametrize("kw,code", [
    (dict(h=None), H.HYDRA_ERR_NULL),
    (dict(tok=None), H.HYDRA_ERR_NULL),
    (dict(kl=None), H.HYDRA_ERR_NULL),
    (dict(A=None), H.HYDRA_ERR_NULL),
    (dict(n_seq=0, ws_bytes=0), H.HYDRA_ERR_SHAPE),
    (dict(V=0, ws_bytes=0), H.HYDRA_ERR_SHAPE),
    (dict(K=12), H.HYDRA_ERR_SHAPE),
    (dict(r=129), H.HYDRA_ERR_SHAPE),
    (dict(n_seq=1 << 20, seq_len=1 << 12, ws_bytes=1), H.HYDRA_ERR_SHAPE),
    (dict(ws=None), H.HYDRA_ERR_WORKSPACE),
    (dict(ws_bytes=16), H.HYDRA_ERR_WORKSPACE),
    (dict(h=P8), H.HYDRA_ERR_ALIGN),
    (dict(ws=P8), H.HYDRA_ERR_ALIGN),
    (dict(lp_on=P + 2), H.HYDRA_ERR_ALIGN),
    (dict(w_rm=P + 1), H.HYDRA_ERR_ALIGN),
])
def test_score_rejects(kw, code):
    assert _score(**kw) == code


def _score2(h_act=P, **kw):
    a = dict(h=P, W=P, A=P, B=P, tok=P, w_rm=P, n_seq=4, seq_len=8, K=64, V=1000, r=8, lp_on=P, lp_off=P, kl=P,
             reward=P, lse_on=None, lse_off=None, ws=P, ws_bytes=None, err=None)
    a.update(kw)
    if a["ws_bytes"] is None:
        a["ws_bytes"] = H.hydra_score_workspace_bytes(a["n_seq"] * a["seq_len"], a["V"])
    return H.lib().hydra_score_two_input(h_act, a["h"], a["W"], a["A"], a["B"], 2.0, a["tok"], a["w_rm"], a["n_seq"],
                                         a["seq_len"], a["K"], a["V"], a["r"], a["lp_on"], a["lp_off"], a["kl"],
                                         a["reward"], a["lse_on"], a["lse_off"], a["ws"], a["ws_bytes"], a["err"], None)


@pytest.mark.parametrize("kw,code", [
    (dict(h_act=None), H.HYDRA_ERR_NULL),
    (dict(h=None), H.HYDRA_ERR_NULL),
    (dict(A=None), H.HYDRA_ERR_NULL),
    (dict(K=12), H.HYDRA_ERR_SHAPE),
    (dict(h_act=P8), H.HYDRA_ERR_ALIGN),
    (dict(h=P8), H.HYDRA_ERR_ALIGN),
    (dict(ws=None), H.HYDRA_ERR_WORKSPACE),
    (dict(ws_bytes=16), H.HYDRA_ERR_WORKSPACE),
    # twice the one-input tile grid: 2048 x 4096 row x column tiles of 256 would reach 2^24 x 256 work-items
    (dict(n_seq=1 << 11, seq_len=1 << 8, V=1 << 20, K=64, ws_bytes=1 << 40), H.HYDRA_ERR_SHAPE),
])
def test_score_two_input_rejects(kw, code):
    assert _score2(**kw) == code


def test_score_two_input_grid_limit_is_twice_the_one_input_one():
    """The same sizes that the one-input call accepts up to its grid limit are halved here (fake pointers; the call
    then fails only on a planted misalignment)."""
    assert _score(n_seq=1 << 11, seq_len=1 << 8, V=1 << 20, K=64, ws_bytes=1 << 40, h=P8) == H.HYDRA_ERR_ALIGN
    assert _score2(n_seq=1 << 10, seq_len=1 << 8, V=1 << 20, K=64, ws_bytes=1 << 40, h=P8) == H.HYDRA_ERR_ALIGN


def _score_na(h=P, W=P, A=P, B=P, tok=P, w_rm=P, n_seq=4, seq_len=8, K=64, V=1000, r=8,
              lp_on=P, lp_off=P, kl=P, reward=P, lse_on=None, lse_off=None, err=None):
    return H.lib().hydra_score_noalloc(h, W, A, B, 2.0, tok, w_rm, n_seq, seq_len, K, V, r, lp_on, lp_off, kl,
                                       reward, lse_on, lse_off, err, None)


@pytest.mark.parametrize("kw,code", [
    (dict(h=None), H.HYDRA_ERR_NULL),
    (dict(tok=None), H.HYDRA_ERR_NULL),
    (dict(A=None), H.HYDRA_ERR_NULL),
    (dict(n_seq=0), H.HYDRA_ERR_SHAPE),
    (dict(K=12), H.HYDRA_ERR_SHAPE),
    (dict(r=129), H.HYDRA_ERR_SHAPE),
    (dict(h=P8), H.HYDRA_ERR_ALIGN),
    (dict(lp_on=P + 2), H.HYDRA_ERR_ALIGN),
    # beyond the scratch: 8192 tokens over a 50272-entry vocabulary need 86 MB of workspace
    (dict(n_seq=16, seq_len=512, V=50272, K=2048), H.HYDRA_ERR_WORKSPACE),
    (dict(n_seq=16, seq_len=512, V=50272, K=2048, h=P8), H.HYDRA_ERR_ALIGN),   # argument errors come first
])
def test_score_noalloc_rejects(kw, code):
    """Every argument error and the scratch limit are reported before any HIP call (the pointers are fake)."""
    assert _score_na(**kw) == code


def test_score_noalloc_limit_covers_the_scoring_workloads():
    """The scratch holds the workspace of the Llama-7B (2048 x 32000) and OPT-1.3b (4096 x 50272) scoring passes;
    calls up to the limit pass the size check (then fail on a planted misalignment)."""
    cap = H.HYDRA_SCORE_NOALLOC_MAX_BYTES
    assert cap == 48 << 20
    assert H.hydra_score_workspace_bytes(2048, 32000) <= cap
    assert H.hydra_score_workspace_bytes(4096, 50272) <= cap
    assert _score_na(n_seq=8, seq_len=512, V=50272, K=2048, h=P8) == H.HYDRA_ERR_ALIGN
    assert H.hydra_score_workspace_bytes(8192, 50272) > cap


def _ws(M, V):
    # one float4 partial per (row, 256-column tile), two floats per row (the
    # gathered token logits), then, 16-byte aligned, 2 x 128 bf16 per row (the
    # hi and lo parts of s * h A^T at the largest rank) and 128 bf16 per
    # vocabulary row (B zero padded to the padded rank)
    # then, 16-byte aligned, the LoRA pre-pass's partial sums (8 K chunks x 128 fp32 per row)
    tiles = (V + 255) // 256
    zt_end = M * tiles * 16 + M * 8
    bp_end = ((zt_end + 15) // 16) * 16 + M * 2 * 128 * 2 + V * 128 * 2
    return ((bp_end + 15) // 16) * 16 + 8 * M * 128 * 4


def test_score_workspace_bytes():
    assert H.hydra_score_workspace_bytes(2048, 32000) == _ws(2048, 32000) == 5160960 + 32000 * 256 + 8 * 2048 * 512
    assert H.hydra_score_workspace_bytes(3, 257) == _ws(3, 257) == 1664 + 257 * 256 + 8 * 3 * 512
    out = ctypes.c_size_t(0)
    assert H.lib().hydra_score_workspace_bytes(0, 10, ctypes.byref(out)) == H.HYDRA_ERR_SHAPE
    assert H.lib().hydra_score_workspace_bytes(10, 10, None) == H.HYDRA_ERR_NULL


@pytest.mark.parametrize("kw,code", [
    (dict(on=None), H.HYDRA_ERR_NULL),
    (dict(tok=None), H.HYDRA_ERR_NULL),
    (dict(M=0), H.HYDRA_ERR_SHAPE),
    (dict(V=-1), H.HYDRA_ERR_SHAPE),
    (dict(on=P8), H.HYDRA_ERR_ALIGN),
    (dict(lp_on=P + 1), H.HYDRA_ERR_ALIGN),
])
def test_score_logits_rejects(kw, code):
    a = dict(on=P, off=P, tok=P, M=8, V=1000, lp_on=P, lp_off=P, kl=P)
    a.update(kw)
    assert H.lib().hydra_score_logits(a["on"], a["off"], a["tok"], a["M"], a["V"], a["lp_on"], a["lp_off"],
                                      a["kl"], None, None, None, None) == code


def test_binding_raises_typed_error():
    with pytest.raises(H.HydraError) as ei:
        Bd._check(H.HYDRA_ERR_SHAPE, "probe")
    assert ei.value.status == H.HYDRA_ERR_SHAPE


def _grp(G=2, xs=(P, P), Ws=(P, P), As=(P, P), Bs=(P, P), ss=(2.0, 2.0), M=4, N=64, K=64, r=8,
         yo=(P, P), yn=(P + 0x1000, P + 0x1000)):
    def arr(v):
        if v is None:
            return None
        a = (ctypes.c_void_p * len(v))()
        for i, p in enumerate(v):
            a[i] = p
        return a
    svals = None if ss is None else (ctypes.c_float * len(ss))(*ss)
    return H.lib().hydra_lora_linear_group(G, arr(xs), arr(Ws), arr(As), arr(Bs), svals, M, N, K, r,
                                           arr(yo), arr(yn), None)


@pytest.mark.parametrize("kw,code", [
    (dict(G=0), H.HYDRA_ERR_SHAPE),
    (dict(G=9), H.HYDRA_ERR_SHAPE),
    (dict(xs=None), H.HYDRA_ERR_NULL),
    (dict(ss=None), H.HYDRA_ERR_NULL),
    (dict(yo=None, yn=None), H.HYDRA_ERR_NULL),
    (dict(xs=(P, None)), H.HYDRA_ERR_NULL),
    (dict(yo=(P, None), yn=(P + 0x1000, None)), H.HYDRA_ERR_NULL),
    (dict(As=(P, None)), H.HYDRA_ERR_NULL),
    (dict(K=20), H.HYDRA_ERR_SHAPE),
    (dict(Ws=(P, P8)), H.HYDRA_ERR_ALIGN),
    (dict(yo=(P, P), yn=(P + 0x1000, P)), H.HYDRA_ERR_SHAPE),
])
def test_lora_linear_group_rejects(kw, code):
    assert _grp(**kw) == code


def test_linear_workspace_bytes():
    # ts: 2 RP bf16 per row, then (16-byte aligned) bp: RP bf16 per output row, then (16-byte aligned) the
    # pre-pass partial sums: 8 K chunks x RP fp32 per row; RP = r rounded up to 16/32/64/128
    def lws(M, N, rp):
        a16 = lambda v: (v + 15) // 16 * 16
        return a16(a16(M * 4 * rp) + N * 2 * rp) + 8 * M * rp * 4
    assert H.hydra_lora_linear_workspace_bytes(2048, 4096, 16) == lws(2048, 4096, 16) == 2048 * 64 + 4096 * 32 + 2048 * 512
    assert H.hydra_lora_linear_workspace_bytes(2048, 11008, 128) == lws(2048, 11008, 128)
    assert H.hydra_lora_linear_workspace_bytes(3, 5, 33) == lws(3, 5, 64)
    assert H.hydra_lora_linear_workspace_bytes(7, 9, 0) == 0
    out = ctypes.c_size_t(0)
    L = H.lib()
    assert L.hydra_lora_linear_workspace_bytes(0, 5, 16, ctypes.byref(out)) == H.HYDRA_ERR_SHAPE
    assert L.hydra_lora_linear_workspace_bytes(5, 5, 129, ctypes.byref(out)) == H.HYDRA_ERR_SHAPE
    assert L.hydra_lora_linear_workspace_bytes(5, 5, 16, None) == H.HYDRA_ERR_NULL


def _lws(x=P, W=P, A=P, B=P, s=2.0, M=64, N=64, K=64, r=128, y_off=P + 0x2000, y_on=P + 0x3000,
         ws=P + 0x10000, nbytes=1 << 20):
    return H.lib().hydra_lora_linear_ws(x, W, A, B, s, M, N, K, r, y_off, y_on, ws, nbytes, None)


@pytest.mark.parametrize("kw,code", [
    (dict(x=None), H.HYDRA_ERR_NULL),
    (dict(y_off=None, y_on=None), H.HYDRA_ERR_NULL),
    (dict(A=None), H.HYDRA_ERR_NULL),
    (dict(ws=None), H.HYDRA_ERR_NULL),                     # GEMM update needs the workspace
    (dict(nbytes=100), H.HYDRA_ERR_WORKSPACE),
    (dict(ws=P + 0x10008), H.HYDRA_ERR_ALIGN),
    (dict(r=129), H.HYDRA_ERR_SHAPE),
    (dict(K=20), H.HYDRA_ERR_SHAPE),
    (dict(y_on=P + 0x2000), H.HYDRA_ERR_SHAPE),            # y_on == y_off
    (dict(W=P8), H.HYDRA_ERR_ALIGN),
])
def test_lora_linear_ws_rejects(kw, code):
    assert _lws(**kw) == code


def test_rank_above_64_needs_the_workspace_in_the_gemm():
    """hydra_lora_linear (and the group call) at M > 16 with r > 64 and y_on: HYDRA_ERR_WORKSPACE, nothing launched."""
    L = H.lib()
    assert L.hydra_lora_linear(P, P, P, P, 2.0, 64, 64, 64, 100, P + 0x2000, P + 0x3000, None) == \
        H.HYDRA_ERR_WORKSPACE
    assert _grp(M=64, r=100, G=2) == H.HYDRA_ERR_WORKSPACE


def _grp_ws(G=2, xs=(P, P), Ws=(P, P), As=(P, P), Bs=(P, P), ss=(2.0, 2.0), M=4, N=64, K=64, r=8,
            yo=(P + 0x1000, P + 0x2000), yn=(P + 0x3000, P + 0x4000), ws=P + 0x10000, nbytes=None):
    def arr(v):
        if v is None:
            return None
        a = (ctypes.c_void_p * len(v))()
        for i, p in enumerate(v):
            a[i] = p
        return a
    if nbytes is None:
        nbytes = H.hydra_lora_linear_group_workspace_bytes(min(max(G, 1), 8), min(max(M, 1), 1 << 20), max(N, 1),
                                                            min(max(r, 0), 128))
    svals = None if ss is None else (ctypes.c_float * len(ss))(*ss)
    return H.lib().hydra_lora_linear_group_ws(G, arr(xs), arr(Ws), arr(As), arr(Bs), svals, M, N, K, r,
                                              arr(yo), arr(yn), ws, nbytes, None)


@pytest.mark.parametrize("kw,code", [
    (dict(G=0), H.HYDRA_ERR_SHAPE),
    (dict(G=9), H.HYDRA_ERR_SHAPE),
    (dict(xs=None), H.HYDRA_ERR_NULL),
    (dict(As=(P, None)), H.HYDRA_ERR_NULL),
    (dict(K=20), H.HYDRA_ERR_SHAPE),
    (dict(r=129), H.HYDRA_ERR_SHAPE),
    (dict(M=(1 << 20) + 1), H.HYDRA_ERR_SHAPE),
    (dict(xs=(P, P8)), H.HYDRA_ERR_ALIGN),
    (dict(ws=None), H.HYDRA_ERR_NULL),
    (dict(nbytes=H.HYDRA_GROUP_WS_CONTROL_BYTES - 1, r=0), H.HYDRA_ERR_WORKSPACE),
    (dict(ws=P + 8), H.HYDRA_ERR_ALIGN),
    (dict(M=2048, r=128, nbytes=4096), H.HYDRA_ERR_WORKSPACE),     # rank 128 above 16 rows: the pre-pass body
])
def test_group_ws_rejects(kw, code):
    """Argument and workspace errors of the workspace group call, all before any HIP call (fake pointers)."""
    assert _grp_ws(**kw) == code


def test_group_ws_workspace_bytes():
    """The control words, the tagged T region and the tagged LoRA-off output region (fixed sizes, so calls of any
    shape find only their own or older tags there), then above 16 rows at padded rank 128 one pre-pass workspace of
    hydra_lora_linear_ws per member."""
    gb = H.hydra_lora_linear_group_workspace_bytes
    C = H.HYDRA_GROUP_WS_CONTROL_BYTES
    T = H.HYDRA_GROUP_WS_T_BYTES
    Y = H.HYDRA_GROUP_WS_Y_BYTES
    assert C == 34 * 128  # a line with the caller's bound word, a spare line, 32 bucket lines
    assert T == 8 * 8 * 128 * 8  # up to 8 members x 8 rows x rank 128, 64-bit tagged entries
    assert Y == 2 << 20  # 64-bit tagged entries of G x N x (rows padded to 1, 2, 4 or 8)
    for args in ((4, 4, 4096, 16), (4, 6, 2048, 128), (1, 1, 10, 0), (8, 16, 100, 9), (3, 2048, 4096, 16)):
        assert gb(*args) == C + T + Y, args
    for G in (1, 3, 8):
        assert gb(G, 2048, 4096, 128) == C + T + Y + G * H.hydra_lora_linear_workspace_bytes(2048, 4096, 128)
    out = ctypes.c_size_t(0)
    assert H.lib().hydra_lora_linear_group_workspace_bytes(9, 4, 10, 0, ctypes.byref(out)) == H.HYDRA_ERR_SHAPE
    assert H.lib().hydra_lora_linear_group_workspace_bytes(1, 4, 10, 129, ctypes.byref(out)) == H.HYDRA_ERR_SHAPE
    assert H.lib().hydra_lora_linear_group_workspace_bytes(1, 4, 10, 8, None) == H.HYDRA_ERR_NULL


def test_header_constants_match_the_binding():
    """Every integer #define of include/hydra.h has the same value in the Python binding."""
    txt = open(HEADER).read()
    pat = r"#define\s+(HYDRA_[A-Z0-9_]+)\s+\(?([0-9]+)u?(?:\s*<<\s*([0-9]+))?"
    defs = {m[0]: int(m[1]) << int(m[2] or 0) for m in re.findall(pat, txt)}
    assert "HYDRA_GROUP_WS_T_BYTES" in defs and "HYDRA_GROUP_WS_CONTROL_BYTES" in defs
    for name, val in defs.items():
        assert getattr(Bd, name) == val, name


def _multi(x_off=P, W=P, n_on=2, xs=(P, P), As=(P, P), Bs=(P, P), ss=(2.0, 2.0), M=4, N=64, K=64, r=8,
           y_off=P + 0x2000, yn=(P + 0x3000, P + 0x4000)):
    def arr(v):
        if v is None:
            return None
        a = (ctypes.c_void_p * max(len(v), 1))()
        for i, p in enumerate(v):
            a[i] = p
        return a
    svals = None if ss is None else (ctypes.c_float * max(len(ss), 1))(*ss)
    return H.lib().hydra_lora_linear_multi(x_off, W, n_on, arr(xs), arr(As), arr(Bs), svals, M, N, K, r, y_off,
                                           arr(yn), None)


@pytest.mark.parametrize("kw,code", [
    (dict(W=None), H.HYDRA_ERR_NULL),
    (dict(n_on=-1), H.HYDRA_ERR_SHAPE),
    (dict(n_on=5), H.HYDRA_ERR_SHAPE),
    (dict(y_off=None), H.HYDRA_ERR_NULL),                       # x_off without y_off
    (dict(x_off=None), H.HYDRA_ERR_NULL),                       # y_off without x_off
    (dict(x_off=None, y_off=None, n_on=0), H.HYDRA_ERR_NULL),   # nothing to compute
    (dict(xs=None), H.HYDRA_ERR_NULL),
    (dict(ss=None), H.HYDRA_ERR_NULL),
    (dict(As=None), H.HYDRA_ERR_NULL),
    (dict(xs=(P, None)), H.HYDRA_ERR_NULL),
    (dict(Bs=(P, None)), H.HYDRA_ERR_NULL),
    (dict(yn=(P + 0x3000, None)), H.HYDRA_ERR_NULL),
    (dict(K=20), H.HYDRA_ERR_SHAPE),
    (dict(r=129), H.HYDRA_ERR_SHAPE),
    (dict(M=0), H.HYDRA_ERR_SHAPE),
    (dict(W=P8), H.HYDRA_ERR_ALIGN),
    (dict(x_off=P8), H.HYDRA_ERR_ALIGN),
    (dict(xs=(P, P8)), H.HYDRA_ERR_ALIGN),
    (dict(As=(P8, P)), H.HYDRA_ERR_ALIGN),
    (dict(yn=(P + 0x3000, P + 0x4002)), H.HYDRA_ERR_ALIGN),
    (dict(yn=(P + 0x2000, P + 0x4000)), H.HYDRA_ERR_SHAPE),    # y_on[0] == y_off
    (dict(yn=(P + 0x3000, P + 0x3000)), H.HYDRA_ERR_SHAPE),    # y_on[0] == y_on[1]
])
def test_lora_linear_multi_rejects(kw, code):
    assert _multi(**kw) == code


def test_lora_linear_multi_rank_above_64_rejected_before_any_launch():
    """M > 16 with adapters of padded rank 128: HYDRA_ERR_WORKSPACE from the host checks, before the LoRA-off output
    is launched (the pointers here are fake: a launch would fault or report HYDRA_ERR_HIP)."""
    assert _multi(M=32, r=100) == H.HYDRA_ERR_WORKSPACE
    assert _multi(M=4096, r=128, n_on=1, xs=(P,), As=(P,), Bs=(P,), ss=(2.0,), yn=(P + 0x3000,)) == \
        H.HYDRA_ERR_WORKSPACE
    # without adapters (LoRA-off input alone) the rank plays no part
    assert _multi(M=32, r=100, n_on=0, xs=None, As=None, Bs=None, ss=None, yn=None, W=P8) == H.HYDRA_ERR_ALIGN
    # decode sizes take rank 128 (the rows go through the stream and update kernels)
    assert _multi(M=16, r=128, W=P8) == H.HYDRA_ERR_ALIGN


def _multi_ws(ws=P + 0x10000, nbytes=None, **kw):
    args = dict(x_off=P, W=P, n_on=2, xs=(P, P), As=(P, P), Bs=(P, P), ss=(2.0, 2.0), M=4, N=64, K=64, r=8,
                y_off=P + 0x2000, yn=(P + 0x3000, P + 0x4000))
    args.update(kw)

    def arr(v):
        if v is None:
            return None
        a = (ctypes.c_void_p * max(len(v), 1))()
        for i, p in enumerate(v):
            a[i] = p
        return a
    if nbytes is None:
        nbytes = H.hydra_lora_linear_multi_workspace_bytes(min(max(args["M"], 1), 1 << 20), max(args["N"], 1),
                                                           min(max(args["r"], 0), 128))
    ss = args["ss"]
    svals = None if ss is None else (ctypes.c_float * max(len(ss), 1))(*ss)
    return H.lib().hydra_lora_linear_multi_ws(args["x_off"], args["W"], args["n_on"], arr(args["xs"]),
                                              arr(args["As"]), arr(args["Bs"]), svals, args["M"], args["N"],
                                              args["K"], args["r"], args["y_off"], arr(args["yn"]), ws, nbytes, None)


@pytest.mark.parametrize("kw,code", [
    (dict(W=None), H.HYDRA_ERR_NULL),
    (dict(n_on=5), H.HYDRA_ERR_SHAPE),
    (dict(yn=(P + 0x3000, P + 0x3000)), H.HYDRA_ERR_SHAPE),
    (dict(ws=None), H.HYDRA_ERR_NULL),
    (dict(ws=P + 8), H.HYDRA_ERR_ALIGN),
    (dict(M=2048, r=128, nbytes=4096), H.HYDRA_ERR_WORKSPACE),   # rank 128 above 16 rows: the pre-pass workspace
    (dict(M=2048, r=128, x_off=P8), H.HYDRA_ERR_ALIGN),
])
def test_lora_linear_multi_ws_rejects(kw, code):
    """Argument and workspace errors of the workspace multi-input call, all before any HIP call (fake pointers)."""
    assert _multi_ws(**kw) == code


def test_lora_linear_multi_ws_workspace_bytes():
    """The workspace of hydra_lora_linear_ws for the same M, N, r (the adapters share it in turn); a rank-128 call
    above 16 rows accepts exactly that size (validation then fails only on the deliberate bad alignment)."""
    for M, N, r in ((2048, 4096, 128), (130, 300, 100), (4, 64, 8)):
        assert H.hydra_lora_linear_multi_workspace_bytes(M, N, r) == H.hydra_lora_linear_workspace_bytes(M, N, r)
    need = H.hydra_lora_linear_multi_workspace_bytes(2048, 64, 128)
    assert _multi_ws(M=2048, r=128, nbytes=need, W=P8) == H.HYDRA_ERR_ALIGN
    assert _multi_ws(M=2048, r=128, nbytes=need - 1) == H.HYDRA_ERR_WORKSPACE


def test_lora_linear_multi_adapters_unused_at_rank_zero():
    """r == 0: A and B may be NULL arrays; validation then fails only on the deliberate bad alignment."""
    assert _multi(r=0, As=None, Bs=None, W=P8) == H.HYDRA_ERR_ALIGN


@pytest.mark.parametrize("kw,code", [
    (dict(h=None), H.HYDRA_ERR_NULL),
    (dict(values=None), H.HYDRA_ERR_NULL),
    (dict(M=0), H.HYDRA_ERR_SHAPE),
    (dict(K=12), H.HYDRA_ERR_SHAPE),
    (dict(K=(1 << 21) + 8), H.HYDRA_ERR_SHAPE),
    (dict(h=P8), H.HYDRA_ERR_ALIGN),
    (dict(w=P + 4), H.HYDRA_ERR_ALIGN),
    (dict(values=P + 2), H.HYDRA_ERR_ALIGN),
])
def test_value_head_rejects(kw, code):
    a = dict(h=P, w=P, M=16, K=64, values=P + 0x1000)
    a.update(kw)
    assert H.lib().hydra_value_head(a["h"], a["w"], a["M"], a["K"], a["values"], None) == code


@pytest.mark.parametrize("kw,code", [
    (dict(kl=None), H.HYDRA_ERR_NULL),
    (dict(adv=None), H.HYDRA_ERR_NULL),
    (dict(n_seq=0), H.HYDRA_ERR_SHAPE),
    (dict(seq_len=0), H.HYDRA_ERR_SHAPE),
    (dict(n_seq=1 << 20, seq_len=1 << 12), H.HYDRA_ERR_SHAPE),
    (dict(start=-1), H.HYDRA_ERR_SHAPE),
    (dict(start=8), H.HYDRA_ERR_SHAPE),
    (dict(adv=P + 0x300), H.HYDRA_ERR_SHAPE),          # advantages written over values
    (dict(ret=P + 0x400), H.HYDRA_ERR_SHAPE),          # returns == advantages
    (dict(rew=P + 0x500), H.HYDRA_ERR_SHAPE),          # rewards == returns
    (dict(kl=P + 2), H.HYDRA_ERR_ALIGN),
    (dict(rew=P + 0x602), H.HYDRA_ERR_ALIGN),
])
def test_ppo_advantages_rejects(kw, code):
    a = dict(kl=P + 0x100, reward=P + 0x200, values=P + 0x300, n_seq=4, seq_len=8, start=0,
             rew=P + 0x600, adv=P + 0x400, ret=P + 0x500)
    a.update(kw)
    assert H.lib().hydra_ppo_advantages(a["kl"], a["reward"], a["values"], a["n_seq"], a["seq_len"], a["start"],
                                        0.02, 1.0, 0.95, a["rew"], a["adv"], a["ret"], None) == code


@pytest.mark.parametrize("kw,code", [
    (dict(lp_new=None), H.HYDRA_ERR_NULL),
    (dict(losses=None), H.HYDRA_ERR_NULL),
    (dict(n_seq=0), H.HYDRA_ERR_SHAPE),
    (dict(start=8), H.HYDRA_ERR_SHAPE),
    (dict(start=-1), H.HYDRA_ERR_SHAPE),
    (dict(eps=1.0), H.HYDRA_ERR_SHAPE),
    (dict(eps=-0.1), H.HYDRA_ERR_SHAPE),
    (dict(eps=float("nan")), H.HYDRA_ERR_SHAPE),
    (dict(d_lp=P), H.HYDRA_ERR_SHAPE),                  # gradient written over lp_new
    (dict(d_v=P + 0x600), H.HYDRA_ERR_SHAPE),           # d_v == d_lp
    (dict(losses=P + 0x600), H.HYDRA_ERR_SHAPE),        # losses == d_lp
    (dict(values=P + 2), H.HYDRA_ERR_ALIGN),
    (dict(d_v=P + 0x702), H.HYDRA_ERR_ALIGN),
])
def test_ppo_loss_rejects(kw, code):
    a = dict(lp_new=P, lp_old=P + 0x100, adv=P + 0x200, values=P + 0x300, returns=P + 0x400, n_seq=2, seq_len=8,
             start=0, eps=0.2, losses=P + 0x500, d_lp=P + 0x600, d_v=P + 0x700)
    a.update(kw)
    assert H.lib().hydra_ppo_loss(a["lp_new"], a["lp_old"], a["adv"], a["values"], a["returns"], a["n_seq"],
                                  a["seq_len"], a["start"], a["eps"], a["losses"], a["d_lp"], a["d_v"],
                                  None) == code


# ------------------------------------------------------------------ backward of the LoRA linear, transpose

def _bwd(x=P, Wt=P + 0x100, A=P + 0x200, B=P + 0x300, s=2.0, dy=P + 0x400, M=64, N=64, K=64, r=16,
         dx=P + 0x1000, dA=P + 0x2000, dB=P + 0x3000, ws=P + 0x10000, nbytes=1 << 24):
    return H.lib().hydra_lora_linear_backward(x, Wt, A, B, s, dy, M, N, K, r, dx, dA, dB, ws, nbytes, None)


@pytest.mark.parametrize("kw,code", [
    (dict(dy=None), H.HYDRA_ERR_NULL),
    (dict(dx=None, dA=None, dB=None), H.HYDRA_ERR_NULL),
    (dict(r=0, dx=None), H.HYDRA_ERR_NULL),               # dA, dB are empty at rank 0: no output left
    (dict(Wt=None), H.HYDRA_ERR_NULL),                    # dx needs W^T
    (dict(A=None), H.HYDRA_ERR_NULL),
    (dict(B=None), H.HYDRA_ERR_NULL),
    (dict(x=None), H.HYDRA_ERR_NULL),                     # dA, dB need x
    (dict(ws=None), H.HYDRA_ERR_NULL),
    (dict(nbytes=1000), H.HYDRA_ERR_WORKSPACE),
    (dict(M=0), H.HYDRA_ERR_SHAPE),
    (dict(M=(1 << 24) + 1), H.HYDRA_ERR_SHAPE),
    (dict(N=12), H.HYDRA_ERR_SHAPE),
    (dict(K=20), H.HYDRA_ERR_SHAPE),
    (dict(K=(1 << 21) + 8), H.HYDRA_ERR_SHAPE),
    (dict(N=(1 << 21) + 8), H.HYDRA_ERR_SHAPE),
    (dict(r=129), H.HYDRA_ERR_SHAPE),
    (dict(r=-1), H.HYDRA_ERR_SHAPE),
    (dict(dA=P + 0x1000), H.HYDRA_ERR_SHAPE),             # dA == dx
    (dict(dB=P + 0x2000), H.HYDRA_ERR_SHAPE),             # dB == dA
    (dict(dy=P8), H.HYDRA_ERR_ALIGN),
    (dict(x=P8), H.HYDRA_ERR_ALIGN),
    (dict(Wt=P8 + 0x100), H.HYDRA_ERR_ALIGN),
    (dict(A=P8 + 0x200), H.HYDRA_ERR_ALIGN),
    (dict(B=P + 0x301), H.HYDRA_ERR_ALIGN),
    (dict(dB=P + 0x3002), H.HYDRA_ERR_ALIGN),
    (dict(ws=P + 0x10008), H.HYDRA_ERR_ALIGN),
])
def test_lora_linear_backward_rejects(kw, code):
    assert _bwd(**kw) == code


def test_lora_linear_backward_optional_inputs():
    """Pointers an output does not need may be NULL (W^T without dx, x without dA / dB, A / B and the
    workspace at rank 0); the checks that remain still fire, so the call is rejected for the one left."""
    assert _bwd(Wt=None, dx=None, x=P8) == H.HYDRA_ERR_ALIGN             # Wt unused, x still checked
    assert _bwd(x=None, dA=None, dB=None, Wt=P8) == H.HYDRA_ERR_ALIGN     # x unused, Wt still checked
    assert _bwd(r=0, A=None, B=None, ws=None, nbytes=0, dy=P8) == H.HYDRA_ERR_ALIGN


def _outer_chunks(M, C):
    tiles = -(-C // 256)
    want = max(1, -(-256 // tiles))
    rows = -(-M // want)
    rows = max(128, -(-rows // 32) * 32)
    return -(-M // rows)


def _bwd_ws(M, N, K, rp):
    if rp == 0:
        return 0
    up = lambda v: -(-v // 256) * 256  # noqa: E731
    Mp = -(-M // 32) * 32
    oa = _outer_chunks(M, K) * rp * K
    ob = _outer_chunks(M, N) * rp * N
    return (up(rp * N * 2) + up(K * rp * 2) + up(M * 2 * rp * 2) + 2 * up(2 * rp * Mp * 2) + 2 * up(8 * M * rp * 4)
            + up(oa * 4) + up(ob * 4))


def test_backward_workspace_bytes():
    for M, N, K, r, rp in [(2048, 4096, 4096, 16, 16), (2048, 11008, 4096, 16, 16), (2048, 4096, 11008, 128, 128),
                           (3, 8, 16, 33, 64), (1, 8, 8, 1, 16)]:
        assert H.hydra_lora_linear_backward_workspace_bytes(M, N, K, r) == _bwd_ws(M, N, K, rp)
    assert H.hydra_lora_linear_backward_workspace_bytes(7, 8, 8, 0) == 0
    # the outer-product partials stay near 2 x 4 MiB however the shape grows (about 256 workgroups' worth each)
    assert H.hydra_lora_linear_backward_workspace_bytes(65536, 4096, 4096, 16) == _bwd_ws(65536, 4096, 4096, 16)
    assert _outer_chunks(65536, 4096) * 16 * 4096 * 4 <= 5 << 20
    L = H.lib()
    out = ctypes.c_size_t(0)
    assert L.hydra_lora_linear_backward_workspace_bytes(0, 8, 8, 16, ctypes.byref(out)) == H.HYDRA_ERR_SHAPE
    assert L.hydra_lora_linear_backward_workspace_bytes(8, 12, 8, 16, ctypes.byref(out)) == H.HYDRA_ERR_SHAPE
    assert L.hydra_lora_linear_backward_workspace_bytes(8, 8, 8, 129, ctypes.byref(out)) == H.HYDRA_ERR_SHAPE
    assert L.hydra_lora_linear_backward_workspace_bytes(8, 8, 8, 16, None) == H.HYDRA_ERR_NULL


@pytest.mark.parametrize("src,R,C,dst,code", [
    (None, 4, 4, P + 0x100, H.HYDRA_ERR_NULL),
    (P, 4, 4, None, H.HYDRA_ERR_NULL),
    (P, 0, 4, P + 0x100, H.HYDRA_ERR_SHAPE),
    (P, 4, (1 << 21) + 1, P + 0x100, H.HYDRA_ERR_SHAPE),
    (P, 4, 4, P, H.HYDRA_ERR_SHAPE),                      # in place
    (P + 1, 4, 4, P + 0x100, H.HYDRA_ERR_ALIGN),
])
def test_transpose_rejects(src, R, C, dst, code):
    assert H.lib().hydra_transpose_bf16(src, R, C, dst, None) == code


# ------------------------------------------------------------------ launch-size limits
# A dispatch counts work-items in 32 bits; the calls bound M (2^20 rows), N / V (2^21) and the MFMA tile grids so
# that every launch fits, and reject larger sizes on the host.

def test_row_and_width_limits():
    big = 1 << 20
    assert _lin(M=big + 1, y_on=None) == H.HYDRA_ERR_SHAPE
    assert _lin(N=(1 << 21) + 1, y_on=None) == H.HYDRA_ERR_SHAPE
    # within the row and width limits but a GEMM tile grid of 8192 x 8192 x 512 threads: too large for a dispatch
    assert _lin(M=big, N=1 << 21, y_on=None) == H.HYDRA_ERR_SHAPE
    assert _lin(M=big, N=1 << 21, y_on=None, x=P8) == H.HYDRA_ERR_SHAPE     # shape is checked before alignment
    assert _lws(M=big + 1) == H.HYDRA_ERR_SHAPE
    assert _grp(M=big + 1) == H.HYDRA_ERR_SHAPE
    assert _multi(M=big + 1) == H.HYDRA_ERR_SHAPE
    out = ctypes.c_size_t(0)
    L = H.lib()
    assert L.hydra_lora_linear_workspace_bytes(big + 1, 8, 16, ctypes.byref(out)) == H.HYDRA_ERR_SHAPE
    assert L.hydra_score_workspace_bytes(8, (1 << 21) + 1, ctypes.byref(out)) == H.HYDRA_ERR_SHAPE
    assert _score(V=(1 << 21) + 1, ws_bytes=1 << 40) == H.HYDRA_ERR_SHAPE
    assert _score(n_seq=1 << 10, seq_len=(1 << 10) + 1, ws_bytes=1 << 40) == H.HYDRA_ERR_SHAPE
    assert L.hydra_score_logits(P, P, P, big + 1, 1000, P, P, P, None, None, None, None) == H.HYDRA_ERR_SHAPE
    assert L.hydra_score_logits(P, P, P, 8, (1 << 21) + 1, P, P, P, None, None, None, None) == H.HYDRA_ERR_SHAPE
    assert L.hydra_value_head(P, P, big + 1, 64, P + 0x1000, None) == H.HYDRA_ERR_SHAPE
    assert L.hydra_ppo_advantages(P, P + 0x100, P + 0x200, 1 << 26, 1, 0, 0.02, 1.0, 0.95, None, P + 0x300,
                                  P + 0x400, None) == H.HYDRA_ERR_SHAPE
    # the PPO calls bound M = n_seq * seq_len (and so seq_len) by the same 2^20 rows
    for n_seq, seq_len in ((1, big + 1), (1 << 10, (1 << 10) + 1), (big + 1, 1)):
        assert L.hydra_ppo_advantages(P, P + 0x100, P + 0x200, n_seq, seq_len, 0, 0.02, 1.0, 0.95, None, P + 0x300,
                                      P + 0x400, None) == H.HYDRA_ERR_SHAPE
        assert L.hydra_ppo_loss(P, P + 0x100, P + 0x200, P + 0x300, P + 0x400, n_seq, seq_len, 0, 0.2, P + 0x500,
                                None, None, None) == H.HYDRA_ERR_SHAPE
    # M = 2^20 exactly passes the size checks (then fails on a planted misalignment)
    for n_seq, seq_len in ((1, big), (1 << 10, 1 << 10)):
        assert L.hydra_ppo_advantages(P + 2, P + 0x100, P + 0x200, n_seq, seq_len, 0, 0.02, 1.0, 0.95, None,
                                      P + 0x300, P + 0x400, None) == H.HYDRA_ERR_ALIGN
        assert L.hydra_ppo_loss(P + 2, P + 0x100, P + 0x200, P + 0x300, P + 0x400, n_seq, seq_len, 0, 0.2,
                                P + 0x500, None, None, None) == H.HYDRA_ERR_ALIGN
    assert L.hydra_transpose_bf16(P, 1 << 21, 1 << 21, P + 0x100, None) == H.HYDRA_ERR_SHAPE
    assert _bwd(M=big + 1) == H.HYDRA_ERR_SHAPE
    assert _bwd(M=big, K=1 << 21, N=64) == H.HYDRA_ERR_SHAPE                   # dx's tile grid


def test_limits_admit_the_largest_realistic_shapes():
    """At the limits that matter in practice the checks pass (the call then fails only on a planted misalignment):
    a million rows through a Llama-7B MLP linear, the 32000-entry head on a million tokens."""
    big = 1 << 20
    assert _lin(M=big, N=11008, K=4096, y_on=None, x=P8) == H.HYDRA_ERR_ALIGN
    assert _score(n_seq=1 << 11, seq_len=1 << 9, V=32000, K=4096, ws_bytes=1 << 40, h=P8) == H.HYDRA_ERR_ALIGN
    assert _bwd(M=big, N=11008, K=4096, dy=P8, nbytes=1 << 40) == H.HYDRA_ERR_ALIGN
    assert H.lib().hydra_transpose_bf16(P + 1, 32000, 4096, P + 0x100, None) == H.HYDRA_ERR_ALIGN
