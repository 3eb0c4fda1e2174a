"""The C ABI on the host: symbols, status codes, workspace sizing and every
argument check that fires before anything is enqueued.

No compute call is made here (no GPU is needed): every call below is
rejected by host-side validation, so fake but well-aligned pointer values
are enough.
"""

import os
import re
import subprocess

import pytest

from paper_2607_21535_amd import wmtp as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "wmtp.h")

P = 0x10000  # a fake, 256-byte aligned "device pointer" (never dereferenced)


def _gpu_present():
    import torch
    return torch.cuda.is_available()


# The fake pointers above must never reach a real device: if a check were
# missing, a GPU would run a kernel on them.  These host-validation tests
# therefore only run where no GPU is visible.
fake_pointers = pytest.mark.skipif(_gpu_present(), reason="fake-pointer validation tests run without a GPU")


@pytest.fixture(scope="module")
def lib():
    return W.load_library()


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(wmtp_[a-z0-9_]+)\s*\(", text)))


def test_header_declares_the_binding_symbols():
    assert _declared_functions() == sorted(W.EXPORTED_SYMBOLS)


def test_library_exports_every_declared_symbol(lib):
    out = subprocess.run(["nm", "-D", "--defined-only", W.lib_path()], capture_output=True, text=True)
    exported = set(re.findall(r"\sT\s+(wmtp_\w+)", out.stdout))
    for name in _declared_functions():
        assert name in exported, name
        assert hasattr(lib, name)


def test_abi_version_and_status_strings(lib):
    assert lib.wmtp_abi_version() == (2 << 16) | 2
    # the header, the library and the binding's signatures agree
    with open(os.path.join(ROOT, "include", "wmtp.h")) as f:
        m = re.search(r"#define WMTP_ABI_VERSION \(\(2 << 16\) \| (\d+)\)", f.read())
    assert m is not None and W.ABI_VERSION == (2 << 16) | int(m.group(1)) == lib.wmtp_abi_version()
    for code in range(6):
        assert W.status_string(code).startswith("WMTP_")
    assert "unknown" in W.status_string(99)


def test_workspace_bytes_shapes():
    full = W.workspace_bytes(1, 32, 2, 256, 1 << 20, variant=W.VARIANT_FULL)
    win = W.workspace_bytes(1, 32, 2, 256, 1 << 20, 2048, 4, variant=W.VARIANT_WINDOWED)
    ring = W.workspace_bytes(1, 32, 2, 256, 0, 2048, 4, variant=W.VARIANT_RING)
    assert full > win > 0
    assert win == ring  # windowed and ring share one split plan
    # windowed workspace does not grow with the cache length
    assert W.workspace_bytes(1, 32, 2, 256, 1 << 17, 2048, 4, variant=W.VARIANT_WINDOWED) == win
    assert W.workspace_bytes(1, 32, 2, 256, 0, variant=W.VARIANT_FULL) == 0
    assert W.workspace_bytes(0, 32, 2, 256, 1000, variant=W.VARIANT_FULL) == 0
    # invalid shapes size to 0
    assert W.workspace_bytes(1, 32, 3, 256, 1000, variant=W.VARIANT_FULL) == 0
    assert W.workspace_bytes(1, 32, 2, 96, 1000, variant=W.VARIANT_FULL) == 0
    assert W.workspace_bytes(1, 32, 2, 256, 1000, variant=7) == 0
    assert W.workspace_bytes(1, 32, 2, 256, 1000, 0, 4, variant=W.VARIANT_WINDOWED) == 0


def test_extend_workspace_bytes():
    """The full-context extend's per-sequence items need room for up to
    q_max times more partials; other variants and single rows size as
    workspace_bytes of B * q_max rows."""
    for B, q, S in [(1, 8, 1 << 20), (1, 8, 1 << 17), (3, 5, 20000), (2, 1, 5000)]:
        rows = W.workspace_bytes(B * q, 32, 2, 256, S, variant=W.VARIANT_FULL)
        ext = W.extend_workspace_bytes(B, q, 32, 2, 256, S)
        assert ext >= rows > 0
        assert (ext > rows) == (q > 1)
        for var, S_, w in [(W.VARIANT_WINDOWED, S, 2048), (W.VARIANT_RING, 2048 + q + 4, 2048)]:
            assert W.extend_workspace_bytes(B, q, 32, 2, 256, S_, w, 4, variant=var) == \
                W.workspace_bytes(B * q, 32, 2, 256, S_, w, 4, variant=var)
    # the finer items are at most q_max * T + rows partials (T = one per CU and KV head)
    one = W.extend_workspace_bytes(1, 8, 32, 2, 256, 1 << 20)
    assert one <= 2 * W.workspace_bytes(8 * 8, 32, 2, 256, 1 << 20, variant=W.VARIANT_FULL)
    # rejected shapes size to 0
    assert W.extend_workspace_bytes(1, 0, 32, 2, 256, 1000) == 0
    assert W.extend_workspace_bytes(1, 8, 32, 3, 256, 1000) == 0
    assert W.extend_workspace_bytes(1, 4097, 32, 2, 256, 1000) == 0
    assert W.extend_workspace_bytes(0, 8, 32, 2, 256, 1000) == 0


def _full(lib, **kw):
    a = dict(q=P, k=P, v=P, lens=P, out=P, lse=None, B=1, Hq=16, Hkv=2, d=128, S_max=100,
             scale=0.1, ws=P, ws_bytes=1 << 30, err=None, stream=None)
    a.update(kw)
    return lib.wmtp_draft_attn_full(*a.values())


def _win(lib, **kw):
    a = dict(q=P, k=P, v=P, lens=P, out=P, lse=None, B=1, Hq=16, Hkv=2, d=128, S_max=100, W=8,
             sink=4, scale=0.1, ws=P, ws_bytes=1 << 30, err=None, stream=None)
    a.update(kw)
    return lib.wmtp_draft_attn_windowed(*a.values())


def _ring(lib, **kw):
    a = dict(q=P, k=P, v=P, lens=P, out=P, lse=None, B=1, Hq=16, Hkv=2, d=128, W=8, sink=4, R_w=8,
             scale=0.1, ws=P, ws_bytes=1 << 30, err=None, stream=None)
    a.update(kw)
    return lib.wmtp_ring_attn(*a.values())


@fake_pointers
@pytest.mark.parametrize("call", [_full, _win, _ring])
def test_attention_argument_checks(lib, call):
    assert call(lib, d=96) == W.EUNSUPPORTED
    assert call(lib, d=512) == W.EUNSUPPORTED
    assert call(lib, Hq=64, Hkv=2) == W.EUNSUPPORTED  # G = 32 > 16
    assert call(lib, d=0) == W.EINVAL
    assert call(lib, Hq=16, Hkv=3) == W.EINVAL
    assert call(lib, Hkv=0) == W.EINVAL
    assert call(lib, B=-1) == W.EINVAL
    assert call(lib, q=None) == W.EINVAL
    assert call(lib, k=None) == W.EINVAL
    assert call(lib, lens=None) == W.EINVAL
    assert call(lib, out=None) == W.EINVAL
    assert call(lib, q=P + 2) == W.EINVAL  # bf16 tensors need 16-byte alignment
    assert call(lib, out=P + 8) == W.EINVAL
    assert call(lib, lens=P + 2) == W.EINVAL
    assert call(lib, ws=P + 64) == W.EINVAL  # workspace needs 256-byte alignment
    assert call(lib, ws=None) == W.EINVAL
    assert call(lib, ws_bytes=1) == W.EWORKSPACE
    assert call(lib, scale=float("nan")) == W.EINVAL
    assert call(lib, scale=float("inf")) == W.EINVAL
    assert call(lib, B=0, q=None, k=None, v=None, lens=None, out=None) == W.OK  # nothing to do


@fake_pointers
def test_full_specific_checks(lib):
    assert _full(lib, S_max=-1) == W.EINVAL
    assert W.workspace_bytes(1, 16, 2, 128, 0, variant=W.VARIANT_FULL) == 0


@fake_pointers
@pytest.mark.parametrize("d,Hq,cap", [(256, 32, 16384), (128, 16, 4096), (64, 8, 4096)])
def test_full_one_launch_workspace(lib, monkeypatch, d, Hq, cap):
    """Full-context calls of at most four query rows x KV heads over a cache
    of at most `cap` rows take the one-launch kernel: their workspace holds
    its records (sized otherwise than the split partials), a byte less is
    refused, and one row more of capacity (or the override
    WMTP_WIN_FULL_MAX_KEYS=0) gives the split layout."""
    monkeypatch.delenv("WMTP_WIN_FULL_MAX_KEYS", raising=False)
    monkeypatch.delenv("WMTP_WIN_ONE_LAUNCH_ROWS", raising=False)
    one = W.workspace_bytes(1, Hq, 2, d, cap, variant=W.VARIANT_FULL)
    assert _full(lib, Hq=Hq, d=d, S_max=cap, ws_bytes=one - 1) == W.EWORKSPACE
    monkeypatch.setenv("WMTP_WIN_FULL_MAX_KEYS", "0")
    split = W.workspace_bytes(1, Hq, 2, d, cap, variant=W.VARIANT_FULL)
    assert split > 0 and split != one
    monkeypatch.delenv("WMTP_WIN_FULL_MAX_KEYS")
    assert W.workspace_bytes(1, Hq, 2, d, cap + 1, variant=W.VARIANT_FULL) != one
    # three sequences (six rows x KV heads) keep split + merge at any capacity
    monkeypatch.setenv("WMTP_WIN_FULL_MAX_KEYS", "0")
    split3 = W.workspace_bytes(3, Hq, 2, d, cap, variant=W.VARIANT_FULL)
    monkeypatch.delenv("WMTP_WIN_FULL_MAX_KEYS")
    assert W.workspace_bytes(3, Hq, 2, d, cap, variant=W.VARIANT_FULL) == split3


@fake_pointers
@pytest.mark.parametrize("call", [_win, _ring])
def test_window_argument_checks(lib, call):
    assert call(lib, W=0) == W.EINVAL
    assert call(lib, W=-3) == W.EINVAL
    assert call(lib, sink=-1) == W.EINVAL


@fake_pointers
def test_ring_specific_checks(lib):
    assert _ring(lib, R_w=7) == W.EINVAL  # R_w < W cannot hold the window
    assert _ring(lib, R_w=0) == W.EINVAL


def _rapp(lib, **kw):
    a = dict(k=P, v=P, kn=P, vn=P, n_new=P, lens=P, B=2, Hkv=2, d=256, sink=4, R_w=16, n_max=8,
             err=None, stream=None)
    a.update(kw)
    return lib.wmtp_ring_append(*a.values())


def _capp(lib, **kw):
    a = dict(k=P, v=P, kn=P, vn=P, n_new=P, lens=P, B=2, Hkv=2, d=256, S_max=100, n_max=8,
             err=None, stream=None)
    a.update(kw)
    return lib.wmtp_cache_append(*a.values())


@fake_pointers
@pytest.mark.parametrize("call", [_rapp, _capp])
def test_append_argument_checks(lib, call):
    assert call(lib, d=96) == W.EUNSUPPORTED
    assert call(lib, d=-1) == W.EINVAL
    assert call(lib, Hkv=0) == W.EINVAL
    assert call(lib, n_max=-1) == W.EINVAL
    assert call(lib, k=None) == W.EINVAL
    assert call(lib, lens=None) == W.EINVAL
    assert call(lib, n_new=None) == W.EINVAL
    assert call(lib, kn=None) == W.EINVAL
    assert call(lib, kn=P + 4) == W.EINVAL
    assert call(lib, lens=P + 1) == W.EINVAL
    assert call(lib, B=0, k=None, v=None, kn=None, vn=None, n_new=None, lens=None) == W.OK


@fake_pointers
def test_ring_append_specific_checks(lib):
    assert _rapp(lib, R_w=0) == W.EINVAL
    assert _rapp(lib, sink=-2) == W.EINVAL


@fake_pointers
def test_cache_append_specific_checks(lib):
    assert _capp(lib, S_max=-1) == W.EINVAL
    assert _capp(lib, S_max=1 << 40) == W.EINVAL


@fake_pointers
def test_select_argument_checks(lib):
    sel = lib.wmtp_select_indices
    assert sel(P, 2, 0, 4, 8, P, P, P, None, None) == W.EINVAL  # W < 1
    assert sel(P, 2, 8, -1, 8, P, P, P, None, None) == W.EINVAL
    assert sel(P, 2, 8, 4, 7, P, P, P, None, None) == W.EINVAL  # slots need R_w >= W
    assert sel(None, 2, 8, 4, 8, P, P, P, None, None) == W.EINVAL
    assert sel(P, 2, 8, 4, 8, None, P, P, None, None) == W.EINVAL
    assert sel(P, 2, 8, 4, 8, P, P, None, None, None) == W.EINVAL
    assert sel(P + 2, 2, 8, 4, 8, P, P, P, None, None) == W.EINVAL
    assert sel(P, 0, 8, 4, 8, None, None, None, None, None) == W.OK


def test_binding_rejects_host_tensors():
    import torch
    q = torch.zeros(1, 16, 128, dtype=torch.bfloat16)
    k = torch.zeros(1, 10, 2, 128, dtype=torch.bfloat16)
    lens = torch.zeros(1, dtype=torch.int32)
    with pytest.raises(ValueError, match="HIP device"):
        W.draft_attn_full(q, k, k, lens)


def _ext(lib, which, fp8=False, **kw):
    base = dict(q=P, k=P, v=P, lens=P, n_q=P, out=P, lse=None, B=1, q_max=4, Hq=16, Hkv=2, d=128)
    if which == "full":
        base.update(S_max=100)
    elif which == "windowed":
        base.update(S_max=100, W=8, sink=4)
    else:
        base.update(W=8, sink=4, R_w=11)
    base.update(scale=0.1)
    if fp8:
        base.update(k_scale=0.5, v_scale=2.0)
    base.update(ws=P, ws_bytes=1 << 30, err=None, stream=None)
    base.update(kw)
    name = {"full": "wmtp_draft_extend_full", "windowed": "wmtp_draft_extend_windowed",
            "ring": "wmtp_ring_extend"}[which] + ("_fp8" if fp8 else "")
    return getattr(lib, name)(*base.values())


@fake_pointers
@pytest.mark.parametrize("which", ["full", "windowed", "ring"])
def test_fp8_extend_argument_checks(lib, which):
    def call(**kw):
        return _ext(lib, which, fp8=True, **kw)
    assert call(q_max=0) == W.EINVAL
    assert call(d=96) == W.EUNSUPPORTED
    assert call(k=P + 8) == W.EINVAL
    assert call(ws_bytes=1) == W.EWORKSPACE
    for bad in (0.0, float("nan")):
        assert call(k_scale=bad) == W.EINVAL
        assert call(v_scale=bad) == W.EINVAL
    if which == "ring":
        assert call(R_w=10) == W.EINVAL
    assert call(B=0, q=None, k=None, v=None, lens=None, n_q=None, out=None) == W.OK


@fake_pointers
@pytest.mark.parametrize("which", ["full", "windowed", "ring"])
def test_extend_argument_checks(lib, which):
    assert _ext(lib, which, q_max=0) == W.EINVAL
    assert _ext(lib, which, q_max=5000) == W.EINVAL
    assert _ext(lib, which, n_q=P + 2) == W.EINVAL
    assert _ext(lib, which, d=96) == W.EUNSUPPORTED
    assert _ext(lib, which, ws_bytes=1) == W.EWORKSPACE
    assert _ext(lib, which, q=None) == W.EINVAL


@fake_pointers
def test_ring_extend_needs_room_for_the_earliest_row(lib):
    assert _ext(lib, "ring", R_w=10) == W.EINVAL  # W + q_max - 1 = 11
    assert _ext(lib, "ring", q_max=1, R_w=8, ws_bytes=1) == W.EWORKSPACE  # R_w = W is enough for one row


def _full8(lib, **kw):
    a = dict(q=P, k=P, v=P, lens=P, out=P, lse=None, B=1, Hq=16, Hkv=2, d=128, S_max=100,
             scale=0.1, k_scale=0.5, v_scale=2.0, ws=P, ws_bytes=1 << 30, err=None, stream=None)
    a.update(kw)
    return lib.wmtp_draft_attn_full_fp8(*a.values())


def _win8(lib, **kw):
    a = dict(q=P, k=P, v=P, lens=P, out=P, lse=None, B=1, Hq=16, Hkv=2, d=128, S_max=100, W=8,
             sink=4, scale=0.1, k_scale=0.5, v_scale=2.0, ws=P, ws_bytes=1 << 30, err=None, stream=None)
    a.update(kw)
    return lib.wmtp_draft_attn_windowed_fp8(*a.values())


def _ring8(lib, **kw):
    a = dict(q=P, k=P, v=P, lens=P, out=P, lse=None, B=1, Hq=16, Hkv=2, d=128, W=8, sink=4, R_w=8,
             scale=0.1, k_scale=0.5, v_scale=2.0, ws=P, ws_bytes=1 << 30, err=None, stream=None)
    a.update(kw)
    return lib.wmtp_ring_attn_fp8(*a.values())


@fake_pointers
@pytest.mark.parametrize("call", [_full8, _win8, _ring8])
def test_fp8_attention_argument_checks(lib, call):
    for bad in (0.0, -1.0, float("nan"), float("inf")):
        assert call(lib, k_scale=bad) == W.EINVAL
        assert call(lib, v_scale=bad) == W.EINVAL
    assert call(lib, scale=1e30, k_scale=1e30) == W.EINVAL  # folded logit scale overflows
    assert call(lib, d=96) == W.EUNSUPPORTED
    assert call(lib, Hq=16, Hkv=3) == W.EINVAL
    assert call(lib, k=P + 8) == W.EINVAL  # caches need 16-byte alignment
    assert call(lib, q=None) == W.EINVAL
    assert call(lib, ws_bytes=1) == W.EWORKSPACE
    assert call(lib, B=0, q=None, k=None, v=None, lens=None, out=None) == W.OK


def _paged(lib, fp8, windowed, **kw):
    a = dict(q=P, k=P, v=P, table=P, lens=P, out=P, lse=None, B=2, Hq=16, Hkv=2, d=128, pool_rows=1000,
             table_stride=100)
    if windowed:
        a.update(W=8, sink=4)
    a.update(scale=0.1)
    if fp8:
        a.update(k_scale=0.5, v_scale=2.0)
    a.update(ws=P, ws_bytes=1 << 30, err=None, stream=None)
    a.update(kw)
    name = "wmtp_paged_attn_" + ("windowed" if windowed else "full") + ("_fp8" if fp8 else "")
    return getattr(lib, name)(*a.values())


@fake_pointers
@pytest.mark.parametrize("fp8", [False, True])
@pytest.mark.parametrize("windowed", [False, True])
def test_paged_attention_argument_checks(lib, fp8, windowed):
    def call(**kw):
        return _paged(lib, fp8, windowed, **kw)
    assert call(table=None) == W.EINVAL
    assert call(table=P + 2) == W.EINVAL  # int32 table, 4-byte alignment
    assert call(pool_rows=0) == W.EINVAL
    assert call(table_stride=-1) == W.EINVAL
    assert call(d=96) == W.EUNSUPPORTED
    assert call(Hq=64, Hkv=2) == W.EUNSUPPORTED
    assert call(k=P + 8) == W.EINVAL
    assert call(ws_bytes=1) == W.EWORKSPACE
    if windowed:
        assert call(W=0) == W.EINVAL
    if fp8:
        for bad in (0.0, -1.0, float("nan")):
            assert call(k_scale=bad) == W.EINVAL
            assert call(v_scale=bad) == W.EINVAL
    assert call(B=0, q=None, k=None, v=None, table=None, lens=None, out=None) == W.OK


def _rapp8(lib, **kw):
    a = dict(k=P, v=P, kn=P, vn=P, n_new=P, lens=P, B=2, Hkv=2, d=256, sink=4, R_w=16, n_max=8,
             k_scale=1.0, v_scale=1.0, err=None, stream=None)
    a.update(kw)
    return lib.wmtp_ring_append_fp8(*a.values())


def _capp8(lib, **kw):
    a = dict(k=P, v=P, kn=P, vn=P, n_new=P, lens=P, B=2, Hkv=2, d=256, S_max=100, n_max=8,
             k_scale=1.0, v_scale=1.0, err=None, stream=None)
    a.update(kw)
    return lib.wmtp_cache_append_fp8(*a.values())


@fake_pointers
@pytest.mark.parametrize("call", [_rapp8, _capp8])
def test_fp8_append_argument_checks(lib, call):
    for bad in (0.0, -2.0, float("nan"), float("inf")):
        assert call(lib, k_scale=bad) == W.EINVAL
        assert call(lib, v_scale=bad) == W.EINVAL
    assert call(lib, d=96) == W.EUNSUPPORTED
    assert call(lib, kn=P + 4) == W.EINVAL
    assert call(lib, B=0, k=None, v=None, kn=None, vn=None, n_new=None, lens=None) == W.OK


@fake_pointers
def test_fp8_conversion_argument_checks(lib):
    q, dq = lib.wmtp_fp8_quantize, lib.wmtp_fp8_dequantize
    assert q(P, 12, 1.0, P, None) == W.EINVAL  # n a multiple of 8
    assert q(P, -8, 1.0, P, None) == W.EINVAL
    assert q(P, 16, 0.0, P, None) == W.EINVAL
    assert q(P + 8, 16, 1.0, P, None) == W.EINVAL  # bf16 input 16-byte aligned
    assert q(P, 16, 1.0, P + 4, None) == W.EINVAL  # codes 8-byte aligned
    assert q(None, 16, 1.0, P, None) == W.EINVAL
    assert q(None, 0, 1.0, None, None) == W.OK
    assert dq(P, 12, P, None) == W.EINVAL
    assert dq(P + 4, 16, P, None) == W.EINVAL
    assert dq(P, 16, P + 8, None) == W.EINVAL
    assert dq(None, 0, None, None) == W.OK


def _tattn(lib, **kw):
    a = dict(q=P, kr=P, vr=P, kb=P, vb=P, lens=P, depth=P, out=P, lse=None, B=2, width=3, Hq=16, Hkv=2,
             d=128, W=8, sink=4, R_w=12, dd=4, scale=0.1, ws=P, ws_bytes=1 << 30, err=None, stream=None)
    a.update(kw)
    return lib.wmtp_tree_attn(*a.values())


def _tapp(lib, **kw):
    a = dict(kr=P, vr=P, kb=P, vb=P, kn=P, vn=P, lens=P, depth=P, B=2, width=3, Hkv=2, d=128, W=8, sink=4,
             R_w=12, dd=4, err=None, stream=None)
    a.update(kw)
    return lib.wmtp_tree_append(*a.values())


@fake_pointers
@pytest.mark.parametrize("call", [_tattn, _tapp])
def test_tree_argument_checks(lib, call):
    assert call(lib, R_w=11) == W.EINVAL  # the ring needs W + depth_max window slots
    assert call(lib, dd=0) == W.EINVAL
    assert call(lib, width=0) == W.EINVAL
    assert call(lib, W=0) == W.EINVAL
    assert call(lib, depth=None) == W.EINVAL
    assert call(lib, kb=None) == W.EINVAL  # candidates 1.. need private runs
    assert call(lib, kb=P + 8) == W.EINVAL
    assert call(lib, d=96) == W.EUNSUPPORTED
    assert call(lib, B=0, kr=None, vr=None, kb=None, vb=None, lens=None, depth=None) == W.OK


@fake_pointers
def test_tree_attn_specific_checks(lib):
    assert _tattn(lib, ws_bytes=1) == W.EWORKSPACE
    assert _tattn(lib, q=None) == W.EINVAL
    assert _tattn(lib, Hq=64, Hkv=2) == W.EUNSUPPORTED
    assert W.workspace_bytes(6, 16, 2, 128, 0, 8, 4, variant=W.VARIANT_TREE) == \
        W.workspace_bytes(6, 16, 2, 128, 12, 8, 4, variant=W.VARIANT_RING)


@fake_pointers
def test_rollback_argument_checks(lib):
    rb, rs = lib.wmtp_ring_rollback, lib.wmtp_tree_reset
    assert rb(None, P, 2, None, None) == W.EINVAL
    assert rb(P, None, 2, None, None) == W.EINVAL
    assert rb(P + 2, P, 2, None, None) == W.EINVAL
    assert rb(P, P, -1, None, None) == W.EINVAL
    assert rb(None, None, 0, None, None) == W.OK
    assert rs(None, 2, None) == W.EINVAL
    assert rs(P + 1, 2, None) == W.EINVAL
    assert rs(None, 0, None) == W.OK


def _step(lib, fn, **kw):
    if fn == "ring":
        a = dict(q=P, k=P, v=P, kn=P, vn=P, nn=P, li=P, lo=P + 256, out=P, lse=None, B=2, Hq=16, Hkv=2, d=128,
                 W=8, sink=4, R_w=8, n_max=2, scale=0.1, ws=P, ws_bytes=1 << 30, err=None, stream=None)
        a.update(kw)
        return lib.wmtp_ring_step(*a.values())
    a = dict(q=P, k=P, v=P, kn=P, vn=P, nn=P, li=P, lo=P + 256, out=P, lse=None, B=2, Hq=16, Hkv=2, d=128,
             S_max=100, n_max=2)
    if fn == "windowed":
        a.update(W=8, sink=4)
    a.update(scale=0.1, ws=P, ws_bytes=1 << 30, err=None, stream=None)
    a.update(kw)
    f = lib.wmtp_draft_step_full if fn == "full" else lib.wmtp_draft_step_windowed
    return f(*a.values())


@fake_pointers
@pytest.mark.parametrize("fn", ["full", "windowed", "ring"])
def test_step_argument_checks(lib, fn):
    assert _step(lib, fn, lo=P) == W.EINVAL  # lens_out must not alias lens_in
    assert _step(lib, fn, lo=None) == W.EINVAL
    assert _step(lib, fn, lo=P + 2) == W.EINVAL
    assert _step(lib, fn, nn=None) == W.EINVAL
    assert _step(lib, fn, kn=None) == W.EINVAL
    assert _step(lib, fn, vn=P + 8) == W.EINVAL
    assert _step(lib, fn, n_max=-1) == W.EINVAL
    assert _step(lib, fn, d=96) == W.EUNSUPPORTED
    assert _step(lib, fn, ws_bytes=1) == W.EWORKSPACE
    assert _step(lib, fn, B=0, q=None, k=None, v=None, kn=None, vn=None, nn=None, li=None, lo=None,
                 out=None) == W.OK
    if fn == "ring":
        assert _step(lib, fn, R_w=7) == W.EINVAL
    if fn == "windowed":  # the fused path numbers the new rows after the cache's: int32
        assert _step(lib, fn, S_max=(1 << 31) - 2, n_max=4) == W.EINVAL


@fake_pointers
def test_read_probe_argument_checks(lib):
    probe = lib.wmtp_hbm_read_probe
    assert probe(P, 24, P, None) == W.EINVAL  # a multiple of 16 bytes
    assert probe(P, -16, P, None) == W.EINVAL
    assert probe(P + 8, 32, P, None) == W.EINVAL  # 16-byte aligned buffer
    assert probe(None, 32, P, None) == W.EINVAL
    assert probe(P, 32, None, None) == W.EINVAL
    assert probe(None, 0, None, None) == W.OK  # nothing to read: no launch


# ----------------------------------------------------- allocation-free call
def _noalloc(lib, B=1, Hq=32, Hkv=2, d=256, S_max=1 << 20, W_=2048, sink=4, q=P, out=P):
    return lib.wmtp_draft_attn_windowed_noalloc(q, P, P, P, out, None, B, Hq, Hkv, d, S_max, W_, sink,
                                                0.0625, None, None)


@fake_pointers
def test_noalloc_host_checks(lib):
    # argument errors come first, as for the workspace form
    assert _noalloc(lib, d=96) == W.EUNSUPPORTED
    assert _noalloc(lib, Hkv=3) == W.EINVAL
    assert _noalloc(lib, W_=0) == W.EINVAL
    assert _noalloc(lib, q=None) == W.EINVAL
    assert _noalloc(lib, out=P + 2) == W.EINVAL
    assert _noalloc(lib, B=0) == W.OK
    # a batch whose partials exceed the static array is rejected, nothing enqueued
    for B in (4096, 1 << 16):
        need = W.workspace_bytes(B, 32, 2, 256, 1 << 20, 2048, 4, variant=W.VARIANT_WINDOWED)
        assert need > W.NOALLOC_SCRATCH_BYTES
        assert _noalloc(lib, B=B) == W.ESCRATCH
    assert "static" in W.status_string(W.ESCRATCH)


def test_noalloc_limit_matches_header():
    text = open(HEADER).read()
    m = re.search(r"#define WMTP_NOALLOC_SCRATCH_BYTES \((\d+)u << (\d+)\)", text)
    assert m is not None and int(m.group(1)) << int(m.group(2)) == W.NOALLOC_SCRATCH_BYTES
    # the 1M workload's windowed call and a 32-sequence batch fit the array
    for B in (1, 8, 32):
        assert W.workspace_bytes(B, 32, 2, 256, 1 << 20, 2048, 4, variant=W.VARIANT_WINDOWED) <= \
            W.NOALLOC_SCRATCH_BYTES
