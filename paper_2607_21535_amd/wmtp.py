"""Python binding of libwmtp.so (ctypes): argument marshalling only.

Every function here checks tensor dtypes, devices and shapes, allocates
outputs/workspace with torch when the caller passes none, and calls the C ABI
(include/wmtp.h) with raw device pointers on torch's current HIP stream.
All computation happens in the library's HIP kernels; there is no fallback:
if libwmtp.so is missing or fails to load, every call raises.
"""

from __future__ import annotations

import ctypes
import math
import os

import torch

__all__ = [
    "WmtpError",
    "VARIANT_FULL",
    "VARIANT_WINDOWED",
    "VARIANT_RING",
    "VARIANT_PAGED_FULL",
    "VARIANT_PAGED_WINDOWED",
    "VARIANT_TREE",
    "DERR_LEN_RANGE",
    "DERR_NNEW_RANGE",
    "DERR_CAPACITY",
    "DERR_SLOT_RANGE",
    "DERR_DEPTH",
    "lib_path",
    "load_library",
    "workspace_bytes",
    "draft_attn_full",
    "draft_attn_windowed",
    "draft_attn_windowed_noalloc",
    "NOALLOC_SCRATCH_BYTES",
    "ring_attn",
    "draft_extend_full",
    "draft_extend_windowed",
    "ring_extend",
    "paged_attn_full",
    "paged_attn_windowed",
    "build_kv_indices",
    "ring_append",
    "cache_append",
    "select_indices",
    "draft_attn_full_fp8",
    "draft_attn_windowed_fp8",
    "ring_attn_fp8",
    "paged_attn_full_fp8",
    "paged_attn_windowed_fp8",
    "draft_extend_full_fp8",
    "draft_extend_windowed_fp8",
    "ring_extend_fp8",
    "cache_append_fp8",
    "ring_append_fp8",
    "fp8_quantize",
    "fp8_dequantize",
    "draft_step_full",
    "draft_step_windowed",
    "ring_step",
    "ring_rollback",
    "tree_append",
    "tree_attn",
    "tree_reset",
    "hbm_read_probe",
    "PROBE_BLOCKS",
    "status_string",
    "EXPORTED_SYMBOLS",
]

VARIANT_FULL, VARIANT_WINDOWED, VARIANT_RING = 0, 1, 2
VARIANT_PAGED_FULL, VARIANT_PAGED_WINDOWED, VARIANT_TREE = 3, 4, 5
DERR_LEN_RANGE, DERR_NNEW_RANGE, DERR_CAPACITY, DERR_SLOT_RANGE, DERR_DEPTH = 0x1, 0x2, 0x4, 0x8, 0x10
OK, EINVAL, EUNSUPPORTED, EWORKSPACE, ELAUNCH, ESCRATCH = 0, 1, 2, 3, 4, 5
NOALLOC_SCRATCH_BYTES = 16 << 20  # WMTP_NOALLOC_SCRATCH_BYTES
PROBE_BLOCKS = 512  # WMTP_PROBE_BLOCKS

EXPORTED_SYMBOLS = (
    "wmtp_workspace_bytes",
    "wmtp_extend_workspace_bytes",
    "wmtp_draft_attn_full",
    "wmtp_draft_attn_windowed",
    "wmtp_draft_attn_windowed_noalloc",
    "wmtp_ring_attn",
    "wmtp_draft_extend_full",
    "wmtp_draft_extend_windowed",
    "wmtp_ring_extend",
    "wmtp_paged_attn_full",
    "wmtp_paged_attn_windowed",
    "wmtp_kv_indices_capacity",
    "wmtp_build_kv_indices",
    "wmtp_ring_append",
    "wmtp_cache_append",
    "wmtp_select_indices",
    "wmtp_draft_attn_full_fp8",
    "wmtp_draft_attn_windowed_fp8",
    "wmtp_ring_attn_fp8",
    "wmtp_draft_extend_full_fp8",
    "wmtp_draft_extend_windowed_fp8",
    "wmtp_ring_extend_fp8",
    "wmtp_paged_attn_full_fp8",
    "wmtp_paged_attn_windowed_fp8",
    "wmtp_ring_append_fp8",
    "wmtp_cache_append_fp8",
    "wmtp_fp8_quantize",
    "wmtp_fp8_dequantize",
    "wmtp_draft_step_full",
    "wmtp_draft_step_windowed",
    "wmtp_ring_step",
    "wmtp_ring_rollback",
    "wmtp_tree_append",
    "wmtp_tree_attn",
    "wmtp_tree_reset",
    "wmtp_hbm_read_probe",
    "wmtp_status_string",
    "wmtp_abi_version",
)

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB = None

_P = ctypes.c_void_p
_I = ctypes.c_int
_I64 = ctypes.c_int64
_F = ctypes.c_float
_SZ = ctypes.c_size_t

_SIGNATURES = {
    "wmtp_workspace_bytes": (_SZ, [_I, _I, _I, _I, _I64, _I, _I, _I]),
    "wmtp_extend_workspace_bytes": (_SZ, [_I, _I, _I, _I, _I, _I64, _I, _I, _I]),
    "wmtp_draft_attn_full": (_I, [_P, _P, _P, _P, _P, _P, _I, _I, _I, _I, _I64, _F, _P, _SZ, _P, _P]),
    "wmtp_draft_attn_windowed": (_I, [_P, _P, _P, _P, _P, _P, _I, _I, _I, _I, _I64, _I, _I, _F, _P, _SZ, _P, _P]),
    "wmtp_draft_attn_windowed_noalloc": (_I, [_P, _P, _P, _P, _P, _P, _I, _I, _I, _I, _I64, _I, _I, _F, _P, _P]),
    "wmtp_ring_attn": (_I, [_P, _P, _P, _P, _P, _P, _I, _I, _I, _I, _I, _I, _I, _F, _P, _SZ, _P, _P]),
    "wmtp_draft_extend_full": (_I, [_P, _P, _P, _P, _P, _P, _P, _I, _I, _I, _I, _I, _I64, _F, _P, _SZ, _P, _P]),
    "wmtp_draft_extend_windowed": (_I, [_P, _P, _P, _P, _P, _P, _P, _I, _I, _I, _I, _I, _I64, _I, _I, _F, _P, _SZ, _P, _P]),
    "wmtp_ring_extend": (_I, [_P, _P, _P, _P, _P, _P, _P, _I, _I, _I, _I, _I, _I, _I, _I, _F, _P, _SZ, _P, _P]),
    "wmtp_paged_attn_full": (_I, [_P, _P, _P, _P, _P, _P, _P, _I, _I, _I, _I, _I64, _I64, _F, _P, _SZ, _P, _P]),
    "wmtp_paged_attn_windowed": (_I, [_P, _P, _P, _P, _P, _P, _P, _I, _I, _I, _I, _I64, _I64, _I, _I, _F, _P, _SZ, _P, _P]),
    "wmtp_kv_indices_capacity": (_I64, [_I, _I, _I64, _I, _I]),
    "wmtp_build_kv_indices": (_I, [_P, _P, _I, _I64, _I, _I, _I, _P, _P, _I64, _P, _P]),
    "wmtp_ring_append": (_I, [_P, _P, _P, _P, _P, _P, _I, _I, _I, _I, _I, _I, _P, _P]),
    "wmtp_cache_append": (_I, [_P, _P, _P, _P, _P, _P, _I, _I, _I, _I64, _I, _P, _P]),
    "wmtp_select_indices": (_I, [_P, _I, _I, _I, _I, _P, _P, _P, _P, _P]),
    "wmtp_draft_attn_full_fp8": (_I, [_P, _P, _P, _P, _P, _P, _I, _I, _I, _I, _I64, _F, _F, _F, _P, _SZ, _P, _P]),
    "wmtp_draft_attn_windowed_fp8": (_I, [_P, _P, _P, _P, _P, _P, _I, _I, _I, _I, _I64, _I, _I, _F, _F, _F, _P, _SZ,
                                          _P, _P]),
    "wmtp_ring_attn_fp8": (_I, [_P, _P, _P, _P, _P, _P, _I, _I, _I, _I, _I, _I, _I, _F, _F, _F, _P, _SZ, _P, _P]),
    "wmtp_draft_extend_full_fp8": (_I, [_P, _P, _P, _P, _P, _P, _P, _I, _I, _I, _I, _I, _I64, _F, _F, _F, _P, _SZ,
                                        _P, _P]),
    "wmtp_draft_extend_windowed_fp8": (_I, [_P, _P, _P, _P, _P, _P, _P, _I, _I, _I, _I, _I, _I64, _I, _I, _F, _F,
                                            _F, _P, _SZ, _P, _P]),
    "wmtp_ring_extend_fp8": (_I, [_P, _P, _P, _P, _P, _P, _P, _I, _I, _I, _I, _I, _I, _I, _I, _F, _F, _F, _P, _SZ,
                                  _P, _P]),
    "wmtp_paged_attn_full_fp8": (_I, [_P, _P, _P, _P, _P, _P, _P, _I, _I, _I, _I, _I64, _I64, _F, _F, _F, _P, _SZ, _P,
                                      _P]),
    "wmtp_paged_attn_windowed_fp8": (_I, [_P, _P, _P, _P, _P, _P, _P, _I, _I, _I, _I, _I64, _I64, _I, _I, _F, _F, _F,
                                          _P, _SZ, _P, _P]),
    "wmtp_ring_append_fp8": (_I, [_P, _P, _P, _P, _P, _P, _I, _I, _I, _I, _I, _I, _F, _F, _P, _P]),
    "wmtp_cache_append_fp8": (_I, [_P, _P, _P, _P, _P, _P, _I, _I, _I, _I64, _I, _F, _F, _P, _P]),
    "wmtp_fp8_quantize": (_I, [_P, _I64, _F, _P, _P]),
    "wmtp_fp8_dequantize": (_I, [_P, _I64, _P, _P]),
    "wmtp_ring_rollback": (_I, [_P, _P, _I, _P, _P]),
    "wmtp_draft_step_full": (_I, [_P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _I, _I, _I, _I, _I64, _I, _F, _P, _SZ,
                                  _P, _P]),
    "wmtp_draft_step_windowed": (_I, [_P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _I, _I, _I, _I, _I64, _I, _I, _I, _F,
                                      _P, _SZ, _P, _P]),
    "wmtp_ring_step": (_I, [_P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _I, _I, _I, _I, _I, _I, _I, _I, _F, _P, _SZ,
                            _P, _P]),
    "wmtp_tree_append": (_I, [_P, _P, _P, _P, _P, _P, _P, _P, _I, _I, _I, _I, _I, _I, _I, _I, _P, _P]),
    "wmtp_tree_attn": (_I, [_P, _P, _P, _P, _P, _P, _P, _P, _P, _I, _I, _I, _I, _I, _I, _I, _I, _I, _F, _P, _SZ,
                            _P, _P]),
    "wmtp_tree_reset": (_I, [_P, _I, _P]),
    "wmtp_hbm_read_probe": (_I, [_P, _I64, _P, _P]),
    "wmtp_status_string": (ctypes.c_char_p, [_I]),
    "wmtp_abi_version": (_I, []),
}


class WmtpError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {status_string(status)} (status {status})")


# The version of include/wmtp.h these signatures follow, (major << 16) | minor:
# a library of another major version, or an older minor one, is refused.
ABI_VERSION = (2 << 16) | 2


def lib_path() -> str:
    return os.environ.get("WMTP_LIB", os.path.join(_HERE, "libwmtp.so"))


def load_library():
    """Load libwmtp.so (once).  Raises OSError when it is missing."""
    global _LIB
    if _LIB is None:
        path = lib_path()
        if not os.path.exists(path):
            raise OSError(f"{path} not found: build it with `python -m paper_2607_21535_amd.build`")
        lib = ctypes.CDLL(path)
        lib.wmtp_abi_version.restype = ctypes.c_int
        lib.wmtp_abi_version.argtypes = []
        v = int(lib.wmtp_abi_version())
        if v >> 16 != ABI_VERSION >> 16 or (v & 0xFFFF) < (ABI_VERSION & 0xFFFF):
            raise OSError(f"{path} has ABI {v >> 16}.{v & 0xFFFF}; this binding needs "
                          f"{ABI_VERSION >> 16}.{ABI_VERSION & 0xFFFF} (rebuild the library)")
        for name, (res, args) in _SIGNATURES.items():
            fn = getattr(lib, name)
            fn.restype = res
            fn.argtypes = args
        _LIB = lib
    return _LIB


def status_string(status: int) -> str:
    return load_library().wmtp_status_string(int(status)).decode()


def _check(status: int, where: str):
    if status != OK:
        raise WmtpError(status, where)


def _ptr(t):
    return None if t is None else t.data_ptr()


def _stream(device) -> int:
    return torch.cuda.current_stream(device).cuda_stream


def _need(t, name, dtype, ndim=None, device=None):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_cuda:
        raise ValueError(f"{name} must be on a HIP device")
    if device is not None and t.device != device:
        raise ValueError(f"{name} is on {t.device}, expected {device}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if ndim is not None and t.dim() != ndim:
        raise ValueError(f"{name} must have {ndim} dims, got {tuple(t.shape)}")


def workspace_bytes(B, Hq, Hkv, d, S_max=0, W=1, sink=0, variant=VARIANT_FULL) -> int:
    """wmtp_workspace_bytes: bytes of the workspace one attention call of
    this variant and shape needs (zero-filled once before its first use)."""
    return int(load_library().wmtp_workspace_bytes(B, Hq, Hkv, d, S_max, W, sink, variant))


def extend_workspace_bytes(B, q_max, Hq, Hkv, d, S_max=0, W=1, sink=0, variant=VARIANT_FULL) -> int:
    """wmtp_extend_workspace_bytes: workspace bytes with which a draft-extend
    call of B sequences and q_max rows spreads each sequence's keys over the
    whole device (full context); other variants: as workspace_bytes(B * q_max)."""
    return int(load_library().wmtp_extend_workspace_bytes(B, q_max, Hq, Hkv, d, S_max, W, sink, variant))


def _workspace(ws, nbytes, device, alloc=None):
    """The caller's workspace (checked for size), or a new zero-filled one of
    `alloc` bytes (default nbytes)."""
    if ws is None:
        alloc = nbytes if alloc is None else alloc
        if alloc == 0:
            return None
        return torch.zeros(alloc, dtype=torch.uint8, device=device)
    if ws.numel() * ws.element_size() < nbytes:
        raise WmtpError(EWORKSPACE, "workspace")
    return ws


_FP8_DTYPES = (torch.uint8, torch.float8_e4m3fn)


def _need_kv(t, name, fp8, ndim, device):
    """A K/V cache: bf16, or (fp8) E4M3 codes as uint8 or float8_e4m3fn."""
    if not fp8:
        return _need(t, name, torch.bfloat16, ndim, device)
    if not isinstance(t, torch.Tensor) or t.dtype not in _FP8_DTYPES:
        raise TypeError(f"{name} must be a uint8 / float8_e4m3fn tensor of E4M3 codes")
    _need(t, name, t.dtype, ndim, device)


def _attn_io(q, k, v, lens, out, lse, fp8=False):
    _need(q, "q", torch.bfloat16, 3)
    dev = q.device
    _need_kv(k, "k", fp8, 4, dev)
    _need_kv(v, "v", fp8, 4, dev)
    _need(lens, "lens", torch.int32, 1, dev)
    B, Hq, d = q.shape
    if k.shape != v.shape or k.shape[0] != B or k.shape[3] != d or lens.shape[0] != B:
        raise ValueError(f"shape mismatch: q {tuple(q.shape)} k {tuple(k.shape)} v {tuple(v.shape)} lens {tuple(lens.shape)}")
    if out is None:
        out = torch.empty_like(q)
    else:
        _need(out, "out", torch.bfloat16, 3, dev)
        if out.shape != q.shape:
            raise ValueError("out must have q's shape")
    if lse is not None:
        _need(lse, "lse", torch.float32, 2, dev)
        if tuple(lse.shape) != (B, Hq):
            raise ValueError("lse must be [B, Hq]")
    return dev, B, Hq, d, out


def draft_attn_full(q, k, v, lens, out=None, lse=None, scale=None, ws=None, err=None):
    """Full-context draft decode attention; returns out [B, Hq, d] bf16."""
    dev, B, Hq, d, out = _attn_io(q, k, v, lens, out, lse)
    S_max, Hkv = k.shape[1], k.shape[2]
    scale = 1.0 / math.sqrt(d) if scale is None else float(scale)
    nb = workspace_bytes(B, Hq, Hkv, d, S_max, variant=VARIANT_FULL)
    ws = _workspace(ws, nb, dev)
    st = load_library().wmtp_draft_attn_full(
        _ptr(q), _ptr(k), _ptr(v), _ptr(lens), _ptr(out), _ptr(lse), B, Hq, Hkv, d, S_max, scale,
        _ptr(ws), 0 if ws is None else ws.numel() * ws.element_size(), _ptr(err), _stream(dev))
    _check(st, "wmtp_draft_attn_full")
    return out


def draft_attn_windowed(q, k, v, lens, W, sink, out=None, lse=None, scale=None, ws=None, err=None):
    """Sink + recent-window draft decode attention over a dense cache."""
    dev, B, Hq, d, out = _attn_io(q, k, v, lens, out, lse)
    S_max, Hkv = k.shape[1], k.shape[2]
    scale = 1.0 / math.sqrt(d) if scale is None else float(scale)
    nb = workspace_bytes(B, Hq, Hkv, d, S_max, W, sink, variant=VARIANT_WINDOWED)
    ws = _workspace(ws, nb, dev)
    st = load_library().wmtp_draft_attn_windowed(
        _ptr(q), _ptr(k), _ptr(v), _ptr(lens), _ptr(out), _ptr(lse), B, Hq, Hkv, d, S_max, W, sink,
        scale, _ptr(ws), 0 if ws is None else ws.numel() * ws.element_size(), _ptr(err), _stream(dev))
    _check(st, "wmtp_draft_attn_windowed")
    return out


def draft_attn_windowed_noalloc(q, k, v, lens, W, sink, out, lse=None, scale=None, err=None):
    """draft_attn_windowed with the library's static scratch instead of a
    workspace (wmtp_draft_attn_windowed_noalloc): the call allocates nothing,
    so `out` must be given.  Raises WmtpError (ESCRATCH) for shapes whose
    partials exceed NOALLOC_SCRATCH_BYTES."""
    if out is None:
        raise ValueError("the allocation-free call needs a preallocated out")
    dev, B, Hq, d, out = _attn_io(q, k, v, lens, out, lse)
    S_max, Hkv = k.shape[1], k.shape[2]
    scale = 1.0 / math.sqrt(d) if scale is None else float(scale)
    st = load_library().wmtp_draft_attn_windowed_noalloc(
        _ptr(q), _ptr(k), _ptr(v), _ptr(lens), _ptr(out), _ptr(lse), B, Hq, Hkv, d, S_max, W, sink,
        scale, _ptr(err), _stream(dev))
    _check(st, "wmtp_draft_attn_windowed_noalloc")
    return out


def ring_attn(q, k_ring, v_ring, lens, W, sink, R_w, out=None, lse=None, scale=None, ws=None, err=None):
    """Windowed draft decode attention over the compact ring [B, sink+R_w, Hkv, d]."""
    dev, B, Hq, d, out = _attn_io(q, k_ring, v_ring, lens, out, lse)
    if k_ring.shape[1] != sink + R_w:
        raise ValueError(f"ring must hold sink + R_w = {sink + R_w} rows, has {k_ring.shape[1]}")
    Hkv = k_ring.shape[2]
    scale = 1.0 / math.sqrt(d) if scale is None else float(scale)
    nb = workspace_bytes(B, Hq, Hkv, d, sink + R_w, W, sink, variant=VARIANT_RING)
    ws = _workspace(ws, nb, dev)
    st = load_library().wmtp_ring_attn(
        _ptr(q), _ptr(k_ring), _ptr(v_ring), _ptr(lens), _ptr(out), _ptr(lse), B, Hq, Hkv, d, W, sink,
        R_w, scale, _ptr(ws), 0 if ws is None else ws.numel() * ws.element_size(), _ptr(err), _stream(dev))
    _check(st, "wmtp_ring_attn")
    return out


def _extend_io(q, k, v, lens, n_q, out, lse, fp8=False):
    _need(q, "q", torch.bfloat16, 4)
    dev = q.device
    cache_dtype = torch.uint8 if fp8 else torch.bfloat16
    _need(k, "k", cache_dtype, 4, dev)
    _need(v, "v", cache_dtype, 4, dev)
    _need(lens, "lens", torch.int32, 1, dev)
    B, q_max, Hq, d = q.shape
    if k.shape != v.shape or k.shape[0] != B or k.shape[3] != d or lens.shape[0] != B:
        raise ValueError(f"shape mismatch: q {tuple(q.shape)} k {tuple(k.shape)} lens {tuple(lens.shape)}")
    if n_q is not None:
        _need(n_q, "n_q", torch.int32, 1, dev)
        if n_q.shape[0] != B:
            raise ValueError("n_q must be [B]")
    if out is None:
        out = torch.empty_like(q)
    else:
        _need(out, "out", torch.bfloat16, 4, dev)
        if out.shape != q.shape:
            raise ValueError("out must have q's shape")
    if lse is not None:
        _need(lse, "lse", torch.float32, 3, dev)
        if tuple(lse.shape) != (B, q_max, Hq):
            raise ValueError("lse must be [B, q_max, Hq]")
    return dev, B, q_max, Hq, d, out


def _wsize(ws):
    return 0 if ws is None else ws.numel() * ws.element_size()


def draft_extend_full(q, k, v, lens, n_q=None, out=None, lse=None, scale=None, ws=None, err=None):
    """Causal multi-row draft attention over the full context.

    q [B, q_max, Hq, d]; lens counts the cached rows including the new ones;
    row t of sequence b sees lens[b] - n_q[b] + t + 1 rows.
    """
    dev, B, q_max, Hq, d, out = _extend_io(q, k, v, lens, n_q, out, lse)
    S_max, Hkv = k.shape[1], k.shape[2]
    scale = 1.0 / math.sqrt(d) if scale is None else float(scale)
    ws = _workspace(ws, workspace_bytes(B * q_max, Hq, Hkv, d, S_max, variant=VARIANT_FULL), dev,
                    extend_workspace_bytes(B, q_max, Hq, Hkv, d, S_max))
    st = load_library().wmtp_draft_extend_full(
        _ptr(q), _ptr(k), _ptr(v), _ptr(lens), _ptr(n_q), _ptr(out), _ptr(lse), B, q_max, Hq, Hkv, d,
        S_max, scale, _ptr(ws), _wsize(ws), _ptr(err), _stream(dev))
    _check(st, "wmtp_draft_extend_full")
    return out


def draft_extend_windowed(q, k, v, lens, W, sink, n_q=None, out=None, lse=None, scale=None, ws=None,
                          err=None):
    """Causal multi-row draft attention, each row under its own sink + window."""
    dev, B, q_max, Hq, d, out = _extend_io(q, k, v, lens, n_q, out, lse)
    S_max, Hkv = k.shape[1], k.shape[2]
    scale = 1.0 / math.sqrt(d) if scale is None else float(scale)
    ws = _workspace(ws, workspace_bytes(B * q_max, Hq, Hkv, d, S_max, W, sink, variant=VARIANT_WINDOWED), dev)
    st = load_library().wmtp_draft_extend_windowed(
        _ptr(q), _ptr(k), _ptr(v), _ptr(lens), _ptr(n_q), _ptr(out), _ptr(lse), B, q_max, Hq, Hkv, d,
        S_max, W, sink, scale, _ptr(ws), _wsize(ws), _ptr(err), _stream(dev))
    _check(st, "wmtp_draft_extend_windowed")
    return out


def ring_extend(q, k_ring, v_ring, lens, W, sink, R_w, n_q=None, out=None, lse=None, scale=None,
                ws=None, err=None):
    """Causal multi-row windowed draft attention over the ring (R_w >= W + q_max - 1)."""
    dev, B, q_max, Hq, d, out = _extend_io(q, k_ring, v_ring, lens, n_q, out, lse)
    if k_ring.shape[1] != sink + R_w:
        raise ValueError(f"ring must hold sink + R_w = {sink + R_w} rows, has {k_ring.shape[1]}")
    Hkv = k_ring.shape[2]
    scale = 1.0 / math.sqrt(d) if scale is None else float(scale)
    ws = _workspace(ws, workspace_bytes(B * q_max, Hq, Hkv, d, sink + R_w, W, sink, variant=VARIANT_RING), dev)
    st = load_library().wmtp_ring_extend(
        _ptr(q), _ptr(k_ring), _ptr(v_ring), _ptr(lens), _ptr(n_q), _ptr(out), _ptr(lse), B, q_max, Hq,
        Hkv, d, W, sink, R_w, scale, _ptr(ws), _wsize(ws), _ptr(err), _stream(dev))
    _check(st, "wmtp_ring_extend")
    return out


def _paged_io(q, k_pool, v_pool, table, lens, out, lse, fp8=False):
    _need(q, "q", torch.bfloat16, 3)
    dev = q.device
    pool_dtype = torch.uint8 if fp8 else torch.bfloat16
    _need(k_pool, "k_pool", pool_dtype, 3, dev)
    _need(v_pool, "v_pool", pool_dtype, 3, dev)
    _need(table, "req_to_token", torch.int32, 2, dev)
    _need(lens, "lens", torch.int32, 1, dev)
    B, Hq, d = q.shape
    if (k_pool.shape != v_pool.shape or k_pool.shape[2] != d or table.shape[0] != B
            or lens.shape[0] != B):
        raise ValueError(f"shape mismatch: q {tuple(q.shape)} pool {tuple(k_pool.shape)} "
                         f"table {tuple(table.shape)} lens {tuple(lens.shape)}")
    if out is None:
        out = torch.empty_like(q)
    else:
        _need(out, "out", torch.bfloat16, 3, dev)
    if lse is not None:
        _need(lse, "lse", torch.float32, 2, dev)
    return dev, B, Hq, d, out


def paged_attn_full(q, k_pool, v_pool, req_to_token, lens, out=None, lse=None, scale=None, ws=None,
                    err=None):
    """Full-context draft attention over a token pool [P, Hkv, d] read through req_to_token [B, C]."""
    dev, B, Hq, d, out = _paged_io(q, k_pool, v_pool, req_to_token, lens, out, lse)
    P, Hkv = k_pool.shape[0], k_pool.shape[1]
    C = req_to_token.shape[1]
    scale = 1.0 / math.sqrt(d) if scale is None else float(scale)
    ws = _workspace(ws, workspace_bytes(B, Hq, Hkv, d, C, variant=VARIANT_PAGED_FULL), dev)
    st = load_library().wmtp_paged_attn_full(
        _ptr(q), _ptr(k_pool), _ptr(v_pool), _ptr(req_to_token), _ptr(lens), _ptr(out), _ptr(lse), B, Hq,
        Hkv, d, P, C, scale, _ptr(ws), _wsize(ws), _ptr(err), _stream(dev))
    _check(st, "wmtp_paged_attn_full")
    return out


def paged_attn_windowed(q, k_pool, v_pool, req_to_token, lens, W, sink, out=None, lse=None, scale=None,
                        ws=None, err=None):
    """Sink + window draft attention over a token pool read through req_to_token."""
    dev, B, Hq, d, out = _paged_io(q, k_pool, v_pool, req_to_token, lens, out, lse)
    P, Hkv = k_pool.shape[0], k_pool.shape[1]
    C = req_to_token.shape[1]
    scale = 1.0 / math.sqrt(d) if scale is None else float(scale)
    ws = _workspace(ws, workspace_bytes(B, Hq, Hkv, d, C, W, sink, variant=VARIANT_PAGED_WINDOWED), dev)
    st = load_library().wmtp_paged_attn_windowed(
        _ptr(q), _ptr(k_pool), _ptr(v_pool), _ptr(req_to_token), _ptr(lens), _ptr(out), _ptr(lse), B, Hq,
        Hkv, d, P, C, W, sink, scale, _ptr(ws), _wsize(ws), _ptr(err), _stream(dev))
    _check(st, "wmtp_paged_attn_windowed")
    return out


def build_kv_indices(req_to_token, lens, variant, W=1, sink=0, indptr=None, indices=None, err=None):
    """Packed index list (kv_indptr [B+1], kv_indices) of the kept keys' pool rows."""
    _need(req_to_token, "req_to_token", torch.int32, 2)
    dev = req_to_token.device
    _need(lens, "lens", torch.int32, 1, dev)
    B, C = req_to_token.shape
    cap = int(load_library().wmtp_kv_indices_capacity(variant, B, C, W, sink))
    if indptr is None:
        indptr = torch.empty(B + 1, dtype=torch.int32, device=dev)
    if indices is None:
        indices = torch.empty(max(cap, 1), dtype=torch.int32, device=dev)
    st = load_library().wmtp_build_kv_indices(
        _ptr(req_to_token), _ptr(lens), B, C, variant, W, sink, _ptr(indptr), _ptr(indices),
        indices.numel(), _ptr(err), _stream(dev))
    _check(st, "wmtp_build_kv_indices")
    return indptr, indices


def _append_io(k, v, k_new, v_new, n_new, lens, fp8=False):
    if not isinstance(k, torch.Tensor):
        raise TypeError("k must be a torch.Tensor")
    dev = k.device
    _need_kv(k, "k", fp8, 4, dev)
    _need_kv(v, "v", fp8, 4, dev)
    _need(k_new, "k_new", torch.bfloat16, 4, dev)
    _need(v_new, "v_new", torch.bfloat16, 4, dev)
    _need(n_new, "n_new", torch.int32, 1, dev)
    _need(lens, "lens", torch.int32, 1, dev)
    B, _, Hkv, d = k.shape
    if (v.shape != k.shape or k_new.shape != v_new.shape or k_new.shape[0] != B
            or tuple(k_new.shape[2:]) != (Hkv, d) or n_new.shape[0] != B or lens.shape[0] != B):
        raise ValueError("append shape mismatch")
    return dev, B, Hkv, d, k_new.shape[1]


def ring_append(k_ring, v_ring, k_new, v_new, n_new, lens, sink, R_w, err=None):
    """Append n_new[b] rows per sequence to the ring; lens += n_new on the device."""
    dev, B, Hkv, d, n_max = _append_io(k_ring, v_ring, k_new, v_new, n_new, lens)
    if k_ring.shape[1] != sink + R_w:
        raise ValueError("ring must hold sink + R_w rows")
    st = load_library().wmtp_ring_append(
        _ptr(k_ring), _ptr(v_ring), _ptr(k_new), _ptr(v_new), _ptr(n_new), _ptr(lens), B, Hkv, d, sink,
        R_w, n_max, _ptr(err), _stream(dev))
    _check(st, "wmtp_ring_append")


def cache_append(k, v, k_new, v_new, n_new, lens, err=None):
    """Append n_new[b] rows per sequence to a dense cache; lens += n_new on the device."""
    dev, B, Hkv, d, n_max = _append_io(k, v, k_new, v_new, n_new, lens)
    st = load_library().wmtp_cache_append(
        _ptr(k), _ptr(v), _ptr(k_new), _ptr(v_new), _ptr(n_new), _ptr(lens), B, Hkv, d, k.shape[1],
        n_max, _ptr(err), _stream(dev))
    _check(st, "wmtp_cache_append")


def select_indices(lens, W, sink, R_w=None, err=None):
    """Kept positions [B, sink+W] (-1 padded), ring slots (if R_w) and counts [B]."""
    _need(lens, "lens", torch.int32, 1)
    dev = lens.device
    B = lens.shape[0]
    pos = torch.empty((B, sink + W), dtype=torch.int32, device=dev)
    slot = None if R_w is None else torch.empty_like(pos)
    n_sel = torch.empty(B, dtype=torch.int32, device=dev)
    st = load_library().wmtp_select_indices(
        _ptr(lens), B, W, sink, W if R_w is None else R_w, _ptr(pos), _ptr(slot), _ptr(n_sel),
        _ptr(err), _stream(dev))
    _check(st, "wmtp_select_indices")
    return pos, slot, n_sel


def _scales(k_scale, v_scale):
    return float(k_scale), float(v_scale)


def draft_attn_full_fp8(q, k, v, lens, k_scale=1.0, v_scale=1.0, out=None, lse=None, scale=None, ws=None,
                        err=None):
    """Full-context draft attention over an fp8 (E4M3) cache [B, S_max, Hkv, d]."""
    dev, B, Hq, d, out = _attn_io(q, k, v, lens, out, lse, fp8=True)
    S_max, Hkv = k.shape[1], k.shape[2]
    scale = 1.0 / math.sqrt(d) if scale is None else float(scale)
    ws = _workspace(ws, workspace_bytes(B, Hq, Hkv, d, S_max, variant=VARIANT_FULL), dev)
    st = load_library().wmtp_draft_attn_full_fp8(
        _ptr(q), _ptr(k), _ptr(v), _ptr(lens), _ptr(out), _ptr(lse), B, Hq, Hkv, d, S_max, scale,
        *_scales(k_scale, v_scale), _ptr(ws), _wsize(ws), _ptr(err), _stream(dev))
    _check(st, "wmtp_draft_attn_full_fp8")
    return out


def draft_attn_windowed_fp8(q, k, v, lens, W, sink, k_scale=1.0, v_scale=1.0, out=None, lse=None, scale=None,
                            ws=None, err=None):
    """Sink + window draft attention over an fp8 (E4M3) dense cache."""
    dev, B, Hq, d, out = _attn_io(q, k, v, lens, out, lse, fp8=True)
    S_max, Hkv = k.shape[1], k.shape[2]
    scale = 1.0 / math.sqrt(d) if scale is None else float(scale)
    ws = _workspace(ws, workspace_bytes(B, Hq, Hkv, d, S_max, W, sink, variant=VARIANT_WINDOWED), dev)
    st = load_library().wmtp_draft_attn_windowed_fp8(
        _ptr(q), _ptr(k), _ptr(v), _ptr(lens), _ptr(out), _ptr(lse), B, Hq, Hkv, d, S_max, W, sink, scale,
        *_scales(k_scale, v_scale), _ptr(ws), _wsize(ws), _ptr(err), _stream(dev))
    _check(st, "wmtp_draft_attn_windowed_fp8")
    return out


def ring_attn_fp8(q, k_ring, v_ring, lens, W, sink, R_w, k_scale=1.0, v_scale=1.0, out=None, lse=None,
                  scale=None, ws=None, err=None):
    """Windowed draft attention over an fp8 (E4M3) ring [B, sink + R_w, Hkv, d]."""
    dev, B, Hq, d, out = _attn_io(q, k_ring, v_ring, lens, out, lse, fp8=True)
    if k_ring.shape[1] != sink + R_w:
        raise ValueError(f"ring must hold sink + R_w = {sink + R_w} rows, has {k_ring.shape[1]}")
    Hkv = k_ring.shape[2]
    scale = 1.0 / math.sqrt(d) if scale is None else float(scale)
    ws = _workspace(ws, workspace_bytes(B, Hq, Hkv, d, sink + R_w, W, sink, variant=VARIANT_RING), dev)
    st = load_library().wmtp_ring_attn_fp8(
        _ptr(q), _ptr(k_ring), _ptr(v_ring), _ptr(lens), _ptr(out), _ptr(lse), B, Hq, Hkv, d, W, sink, R_w,
        scale, *_scales(k_scale, v_scale), _ptr(ws), _wsize(ws), _ptr(err), _stream(dev))
    _check(st, "wmtp_ring_attn_fp8")
    return out


def paged_attn_full_fp8(q, k_pool, v_pool, req_to_token, lens, k_scale=1.0, v_scale=1.0, out=None, lse=None,
                        scale=None, ws=None, err=None):
    """Full-context draft attention over an fp8 (E4M3) token pool [P, Hkv, d] read through req_to_token."""
    dev, B, Hq, d, out = _paged_io(q, k_pool, v_pool, req_to_token, lens, out, lse, fp8=True)
    P, Hkv = k_pool.shape[0], k_pool.shape[1]
    C = req_to_token.shape[1]
    scale = 1.0 / math.sqrt(d) if scale is None else float(scale)
    ws = _workspace(ws, workspace_bytes(B, Hq, Hkv, d, C, variant=VARIANT_PAGED_FULL), dev)
    st = load_library().wmtp_paged_attn_full_fp8(
        _ptr(q), _ptr(k_pool), _ptr(v_pool), _ptr(req_to_token), _ptr(lens), _ptr(out), _ptr(lse), B, Hq,
        Hkv, d, P, C, scale, *_scales(k_scale, v_scale), _ptr(ws), _wsize(ws), _ptr(err), _stream(dev))
    _check(st, "wmtp_paged_attn_full_fp8")
    return out


def paged_attn_windowed_fp8(q, k_pool, v_pool, req_to_token, lens, W, sink, k_scale=1.0, v_scale=1.0, out=None,
                            lse=None, scale=None, ws=None, err=None):
    """Sink + window draft attention over an fp8 (E4M3) token pool read through req_to_token."""
    dev, B, Hq, d, out = _paged_io(q, k_pool, v_pool, req_to_token, lens, out, lse, fp8=True)
    P, Hkv = k_pool.shape[0], k_pool.shape[1]
    C = req_to_token.shape[1]
    scale = 1.0 / math.sqrt(d) if scale is None else float(scale)
    ws = _workspace(ws, workspace_bytes(B, Hq, Hkv, d, C, W, sink, variant=VARIANT_PAGED_WINDOWED), dev)
    st = load_library().wmtp_paged_attn_windowed_fp8(
        _ptr(q), _ptr(k_pool), _ptr(v_pool), _ptr(req_to_token), _ptr(lens), _ptr(out), _ptr(lse), B, Hq,
        Hkv, d, P, C, W, sink, scale, *_scales(k_scale, v_scale), _ptr(ws), _wsize(ws), _ptr(err), _stream(dev))
    _check(st, "wmtp_paged_attn_windowed_fp8")
    return out


def draft_extend_full_fp8(q, k, v, lens, k_scale=1.0, v_scale=1.0, n_q=None, out=None, lse=None, scale=None,
                          ws=None, err=None):
    """Causal multi-row draft attention over the full context of an fp8 (E4M3) cache."""
    dev, B, q_max, Hq, d, out = _extend_io(q, k, v, lens, n_q, out, lse, fp8=True)
    S_max, Hkv = k.shape[1], k.shape[2]
    scale = 1.0 / math.sqrt(d) if scale is None else float(scale)
    ws = _workspace(ws, workspace_bytes(B * q_max, Hq, Hkv, d, S_max, variant=VARIANT_FULL), dev,
                    extend_workspace_bytes(B, q_max, Hq, Hkv, d, S_max))
    st = load_library().wmtp_draft_extend_full_fp8(
        _ptr(q), _ptr(k), _ptr(v), _ptr(lens), _ptr(n_q), _ptr(out), _ptr(lse), B, q_max, Hq, Hkv, d,
        S_max, scale, *_scales(k_scale, v_scale), _ptr(ws), _wsize(ws), _ptr(err), _stream(dev))
    _check(st, "wmtp_draft_extend_full_fp8")
    return out


def draft_extend_windowed_fp8(q, k, v, lens, W, sink, k_scale=1.0, v_scale=1.0, n_q=None, out=None, lse=None,
                              scale=None, ws=None, err=None):
    """Causal multi-row draft attention over an fp8 (E4M3) cache, each row under its own sink + window."""
    dev, B, q_max, Hq, d, out = _extend_io(q, k, v, lens, n_q, out, lse, fp8=True)
    S_max, Hkv = k.shape[1], k.shape[2]
    scale = 1.0 / math.sqrt(d) if scale is None else float(scale)
    ws = _workspace(ws, workspace_bytes(B * q_max, Hq, Hkv, d, S_max, W, sink, variant=VARIANT_WINDOWED), dev)
    st = load_library().wmtp_draft_extend_windowed_fp8(
        _ptr(q), _ptr(k), _ptr(v), _ptr(lens), _ptr(n_q), _ptr(out), _ptr(lse), B, q_max, Hq, Hkv, d,
        S_max, W, sink, scale, *_scales(k_scale, v_scale), _ptr(ws), _wsize(ws), _ptr(err), _stream(dev))
    _check(st, "wmtp_draft_extend_windowed_fp8")
    return out


def ring_extend_fp8(q, k_ring, v_ring, lens, W, sink, R_w, k_scale=1.0, v_scale=1.0, n_q=None, out=None,
                    lse=None, scale=None, ws=None, err=None):
    """Causal multi-row windowed draft attention over an fp8 (E4M3) ring (R_w >= W + q_max - 1)."""
    dev, B, q_max, Hq, d, out = _extend_io(q, k_ring, v_ring, lens, n_q, out, lse, fp8=True)
    if k_ring.shape[1] != sink + R_w:
        raise ValueError(f"ring must hold sink + R_w = {sink + R_w} rows, has {k_ring.shape[1]}")
    Hkv = k_ring.shape[2]
    scale = 1.0 / math.sqrt(d) if scale is None else float(scale)
    ws = _workspace(ws, workspace_bytes(B * q_max, Hq, Hkv, d, sink + R_w, W, sink, variant=VARIANT_RING), dev)
    st = load_library().wmtp_ring_extend_fp8(
        _ptr(q), _ptr(k_ring), _ptr(v_ring), _ptr(lens), _ptr(n_q), _ptr(out), _ptr(lse), B, q_max, Hq,
        Hkv, d, W, sink, R_w, scale, *_scales(k_scale, v_scale), _ptr(ws), _wsize(ws), _ptr(err), _stream(dev))
    _check(st, "wmtp_ring_extend_fp8")
    return out


def cache_append_fp8(k, v, k_new, v_new, n_new, lens, k_scale=1.0, v_scale=1.0, err=None):
    """Quantise and append n_new[b] bf16 rows per sequence to an fp8 dense cache; lens += n_new."""
    dev, B, Hkv, d, n_max = _append_io(k, v, k_new, v_new, n_new, lens, fp8=True)
    st = load_library().wmtp_cache_append_fp8(
        _ptr(k), _ptr(v), _ptr(k_new), _ptr(v_new), _ptr(n_new), _ptr(lens), B, Hkv, d, k.shape[1], n_max,
        *_scales(k_scale, v_scale), _ptr(err), _stream(dev))
    _check(st, "wmtp_cache_append_fp8")


def ring_append_fp8(k_ring, v_ring, k_new, v_new, n_new, lens, sink, R_w, k_scale=1.0, v_scale=1.0, err=None):
    """Quantise and append n_new[b] bf16 rows per sequence to an fp8 ring; lens += n_new."""
    dev, B, Hkv, d, n_max = _append_io(k_ring, v_ring, k_new, v_new, n_new, lens, fp8=True)
    if k_ring.shape[1] != sink + R_w:
        raise ValueError("ring must hold sink + R_w rows")
    st = load_library().wmtp_ring_append_fp8(
        _ptr(k_ring), _ptr(v_ring), _ptr(k_new), _ptr(v_new), _ptr(n_new), _ptr(lens), B, Hkv, d, sink, R_w,
        n_max, *_scales(k_scale, v_scale), _ptr(err), _stream(dev))
    _check(st, "wmtp_ring_append_fp8")


def fp8_quantize(x, scale=1.0, out=None):
    """E4M3 codes (uint8, x's shape) of bf16 x stored with per-tensor `scale` (the appends' rule)."""
    _need(x, "x", torch.bfloat16)
    if x.numel() % 8:
        raise ValueError("x must hold a multiple of 8 elements")
    if out is None:
        out = torch.empty(x.shape, dtype=torch.uint8, device=x.device)
    else:
        _need(out, "out", torch.uint8, None, x.device)
        if out.numel() != x.numel():
            raise ValueError("out must have x's size")
    st = load_library().wmtp_fp8_quantize(_ptr(x), x.numel(), float(scale), _ptr(out), _stream(x.device))
    _check(st, "wmtp_fp8_quantize")
    return out


def hbm_read_probe(buf, sink=None):
    """One streaming read pass over the bytes of the contiguous device tensor
    `buf` (a measurement helper: timed, it gives the HBM read ceiling).
    Returns sink, int32[PROBE_BLOCKS]: the XOR of the words each workgroup read."""
    if not isinstance(buf, torch.Tensor) or not buf.is_cuda or not buf.is_contiguous():
        raise ValueError("buf must be a contiguous device tensor")
    nbytes = buf.numel() * buf.element_size()
    if nbytes % 16 or buf.data_ptr() % 16:
        raise ValueError("buf must be 16-byte aligned and a multiple of 16 bytes")
    if sink is None:
        sink = torch.empty(PROBE_BLOCKS, dtype=torch.int32, device=buf.device)
    else:
        _need(sink, "sink", torch.int32, 1, buf.device)
        if sink.numel() < PROBE_BLOCKS:
            raise ValueError(f"sink must hold {PROBE_BLOCKS} words")
    st = load_library().wmtp_hbm_read_probe(_ptr(buf), nbytes, _ptr(sink), _stream(buf.device))
    _check(st, "wmtp_hbm_read_probe")
    return sink


def fp8_dequantize(codes, out=None):
    """bf16 values (codes' shape) of E4M3 codes, as the attention kernels widen them."""
    if not isinstance(codes, torch.Tensor) or codes.dtype not in _FP8_DTYPES:
        raise TypeError("codes must be a uint8 / float8_e4m3fn tensor")
    _need(codes, "codes", codes.dtype)
    if codes.numel() % 8:
        raise ValueError("codes must hold a multiple of 8 elements")
    if out is None:
        out = torch.empty(codes.shape, dtype=torch.bfloat16, device=codes.device)
    else:
        _need(out, "out", torch.bfloat16, None, codes.device)
        if out.numel() != codes.numel():
            raise ValueError("out must have codes' size")
    st = load_library().wmtp_fp8_dequantize(_ptr(codes), codes.numel(), _ptr(out), _stream(codes.device))
    _check(st, "wmtp_fp8_dequantize")
    return out


def ring_rollback(lens, n_drop, err=None):
    """Discard rejected speculative rows of a chain: lens -= n_drop on the device."""
    _need(lens, "lens", torch.int32, 1)
    _need(n_drop, "n_drop", torch.int32, 1, lens.device)
    if n_drop.shape != lens.shape:
        raise ValueError("n_drop must have lens' shape")
    st = load_library().wmtp_ring_rollback(_ptr(lens), _ptr(n_drop), lens.shape[0], _ptr(err), _stream(lens.device))
    _check(st, "wmtp_ring_rollback")


def _tree_store(k_ring, v_ring, k_branch, v_branch, width, depth_max, sink, R_w):
    _need(k_ring, "k_ring", torch.bfloat16, 4)
    dev = k_ring.device
    _need(v_ring, "v_ring", torch.bfloat16, 4, dev)
    B, rows, Hkv, d = k_ring.shape
    if v_ring.shape != k_ring.shape or rows != sink + R_w:
        raise ValueError(f"ring must be [B, sink + R_w = {sink + R_w}, Hkv, d]")
    if width > 1:
        _need(k_branch, "k_branch", torch.bfloat16, 4, dev)
        _need(v_branch, "v_branch", torch.bfloat16, 4, dev)
        if tuple(k_branch.shape) != (B, (width - 1) * depth_max, Hkv, d) or v_branch.shape != k_branch.shape:
            raise ValueError(f"private runs must be [B, (width - 1) * depth_max, Hkv, d], got {tuple(k_branch.shape)}")
    return dev, B, Hkv, d


def tree_append(k_ring, v_ring, k_branch, v_branch, k_new, v_new, lens, depth, W, sink, R_w, depth_max, err=None):
    """One draft row per candidate (k_new [B, width, Hkv, d]) at position lens + depth; depth += 1."""
    _need(k_new, "k_new", torch.bfloat16, 4)
    width = k_new.shape[1]
    dev, B, Hkv, d = _tree_store(k_ring, v_ring, k_branch, v_branch, width, depth_max, sink, R_w)
    _need(v_new, "v_new", torch.bfloat16, 4, dev)
    _need(lens, "lens", torch.int32, 1, dev)
    _need(depth, "depth", torch.int32, 1, dev)
    if tuple(k_new.shape) != (B, width, Hkv, d) or v_new.shape != k_new.shape:
        raise ValueError("k_new / v_new must be [B, width, Hkv, d]")
    st = load_library().wmtp_tree_append(
        _ptr(k_ring), _ptr(v_ring), _ptr(k_branch), _ptr(v_branch), _ptr(k_new), _ptr(v_new), _ptr(lens), _ptr(depth),
        B, width, Hkv, d, W, sink, R_w, depth_max, _ptr(err), _stream(dev))
    _check(st, "wmtp_tree_append")


def tree_attn(q, k_ring, v_ring, k_branch, v_branch, lens, depth, W, sink, R_w, depth_max, out=None, lse=None,
              scale=None, ws=None, err=None):
    """Windowed draft attention of every speculation candidate: q, out [B, width, Hq, d]."""
    _need(q, "q", torch.bfloat16, 4)
    B, width, Hq, d = q.shape
    dev, B2, Hkv, d2 = _tree_store(k_ring, v_ring, k_branch, v_branch, width, depth_max, sink, R_w)
    if B2 != B or d2 != d:
        raise ValueError("q and the ring disagree on B or d")
    _need(lens, "lens", torch.int32, 1, dev)
    _need(depth, "depth", torch.int32, 1, dev)
    if out is None:
        out = torch.empty_like(q)
    else:
        _need(out, "out", torch.bfloat16, 4, dev)
        if out.shape != q.shape:
            raise ValueError("out must have q's shape")
    if lse is not None:
        _need(lse, "lse", torch.float32, 3, dev)
        if tuple(lse.shape) != (B, width, Hq):
            raise ValueError("lse must be [B, width, Hq]")
    scale = 1.0 / math.sqrt(d) if scale is None else float(scale)
    ws = _workspace(ws, workspace_bytes(B * width, Hq, Hkv, d, 0, W, sink, variant=VARIANT_TREE), dev)
    st = load_library().wmtp_tree_attn(
        _ptr(q), _ptr(k_ring), _ptr(v_ring), _ptr(k_branch), _ptr(v_branch), _ptr(lens), _ptr(depth), _ptr(out),
        _ptr(lse), B, width, Hq, Hkv, d, W, sink, R_w, depth_max, scale, _ptr(ws), _wsize(ws), _ptr(err), _stream(dev))
    _check(st, "wmtp_tree_attn")
    return out


def tree_reset(depth):
    """Speculative depth back to 0 for every request (after the verify)."""
    _need(depth, "depth", torch.int32, 1)
    st = load_library().wmtp_tree_reset(_ptr(depth), depth.shape[0], _stream(depth.device))
    _check(st, "wmtp_tree_reset")


def _step_io(q, k, v, k_new, v_new, n_new, lens_in, lens_out, out, lse):
    dev, B, Hq, d, out = _attn_io(q, k, v, lens_in, out, lse)
    _need(k_new, "k_new", torch.bfloat16, 4, dev)
    _need(v_new, "v_new", torch.bfloat16, 4, dev)
    _need(n_new, "n_new", torch.int32, 1, dev)
    _need(lens_out, "lens_out", torch.int32, 1, dev)
    Hkv = k.shape[2]
    if (k_new.shape != v_new.shape or k_new.shape[0] != B or tuple(k_new.shape[2:]) != (Hkv, d)
            or n_new.shape[0] != B or lens_out.shape[0] != B):
        raise ValueError("step shape mismatch")
    if lens_out.data_ptr() == lens_in.data_ptr():
        raise ValueError("lens_out must be a different array from lens_in")
    return dev, B, Hq, Hkv, d, k_new.shape[1], out


def draft_step_full(q, k, v, k_new, v_new, n_new, lens_in, lens_out, out=None, lse=None, scale=None, ws=None,
                    err=None):
    """Append n_new rows at lens_in, attend the full context; lens_out = lens_in + n_new."""
    dev, B, Hq, Hkv, d, n_max, out = _step_io(q, k, v, k_new, v_new, n_new, lens_in, lens_out, out, lse)
    S_max = k.shape[1]
    scale = 1.0 / math.sqrt(d) if scale is None else float(scale)
    ws = _workspace(ws, workspace_bytes(B, Hq, Hkv, d, S_max, variant=VARIANT_FULL), dev)
    st = load_library().wmtp_draft_step_full(
        _ptr(q), _ptr(k), _ptr(v), _ptr(k_new), _ptr(v_new), _ptr(n_new), _ptr(lens_in), _ptr(lens_out), _ptr(out),
        _ptr(lse), B, Hq, Hkv, d, S_max, n_max, scale, _ptr(ws), _wsize(ws), _ptr(err), _stream(dev))
    _check(st, "wmtp_draft_step_full")
    return out


def draft_step_windowed(q, k, v, k_new, v_new, n_new, lens_in, lens_out, W, sink, out=None, lse=None, scale=None,
                        ws=None, err=None):
    """Append n_new rows at lens_in, attend sink + window; lens_out = lens_in + n_new."""
    dev, B, Hq, Hkv, d, n_max, out = _step_io(q, k, v, k_new, v_new, n_new, lens_in, lens_out, out, lse)
    S_max = k.shape[1]
    scale = 1.0 / math.sqrt(d) if scale is None else float(scale)
    ws = _workspace(ws, workspace_bytes(B, Hq, Hkv, d, S_max, W, sink, variant=VARIANT_WINDOWED), dev)
    st = load_library().wmtp_draft_step_windowed(
        _ptr(q), _ptr(k), _ptr(v), _ptr(k_new), _ptr(v_new), _ptr(n_new), _ptr(lens_in), _ptr(lens_out), _ptr(out),
        _ptr(lse), B, Hq, Hkv, d, S_max, n_max, W, sink, scale, _ptr(ws), _wsize(ws), _ptr(err), _stream(dev))
    _check(st, "wmtp_draft_step_windowed")
    return out


def ring_step(q, k_ring, v_ring, k_new, v_new, n_new, lens_in, lens_out, W, sink, R_w, out=None, lse=None,
              scale=None, ws=None, err=None):
    """Append n_new rows to the ring at lens_in, attend sink + window; lens_out = lens_in + n_new."""
    dev, B, Hq, Hkv, d, n_max, out = _step_io(q, k_ring, v_ring, k_new, v_new, n_new, lens_in, lens_out, out, lse)
    if k_ring.shape[1] != sink + R_w:
        raise ValueError(f"ring must hold sink + R_w = {sink + R_w} rows, has {k_ring.shape[1]}")
    scale = 1.0 / math.sqrt(d) if scale is None else float(scale)
    ws = _workspace(ws, workspace_bytes(B, Hq, Hkv, d, sink + R_w, W, sink, variant=VARIANT_RING), dev)
    st = load_library().wmtp_ring_step(
        _ptr(q), _ptr(k_ring), _ptr(v_ring), _ptr(k_new), _ptr(v_new), _ptr(n_new), _ptr(lens_in), _ptr(lens_out),
        _ptr(out), _ptr(lse), B, Hq, Hkv, d, W, sink, R_w, n_max, scale, _ptr(ws), _wsize(ws), _ptr(err),
        _stream(dev))
    _check(st, "wmtp_ring_step")
    return out
