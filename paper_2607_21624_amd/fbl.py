"""ctypes binding of libfbl.so (the C ABI in include/fbl.h).

Argument marshalling only: every step of the attention path runs in the HIP
kernels behind the C ABI.  torch is used for device memory (allocating outputs
and the workspace) and for the current stream.  If libfbl.so is missing the
import fails; there is no fallback implementation.
"""
from __future__ import annotations

import ctypes
import math
import os
from typing import Optional, Tuple

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libfbl.so")

FBL_OK = 0
FBL_ERR_NULL = 1
FBL_ERR_SHAPE = 2
FBL_ERR_DTYPE = 3
FBL_ERR_LAYOUT = 4
FBL_ERR_ALIGN = 5
FBL_ERR_UNSUPPORTED = 6
FBL_ERR_WORKSPACE = 7
FBL_ERR_HIP = 8
FBL_ERR_ARG = 9

FBL_F32 = 0
FBL_BF16 = 1
FBL_MASK_CAUSAL = 1
FBL_MASK_KEY_PADDING = 2

FBL_BWD_PREP = 1
FBL_BWD_KV = 2
FBL_BWD_Q = 4
FBL_BWD_ALL = 7

FBL_PROJ_FWD = 0
FBL_PROJ_BWD_DATA = 1
FBL_PROJ_BWD_WEIGHT = 2
FBL_GEMM_TILE_AUTO = -1
FBL_GEMM_TILE_128x128 = 0
FBL_GEMM_TILE_128x64 = 1
FBL_GEMM_TILE_64x128 = 2
FBL_GEMM_TILE_64x64 = 3
FBL_TUNE_TIME = 0
FBL_TUNE_GFLOPS_X_MEMEFF = 1

FBL_ATTN_FWD = 0
FBL_ATTN_BWD_KV = 1
FBL_ATTN_BWD_DQ = 2
FBL_ATTN_TILE_AUTO = -1

EXPORTED = ("fbl_layout_desc", "fbl_layout_packed_qkv", "fbl_layout_offset", "fbl_layout_map_device", "fbl_attn_fwd",
            "fbl_attn_bwd_workspace", "fbl_attn_bwd_workspace_min", "fbl_attn_bwd", "fbl_attn_bwd_phases",
            "fbl_attn_bwd_noalloc", "fbl_attn_fwd_tiled", "fbl_attn_bwd_tiled", "fbl_attn_bwd_launches", "fbl_attn_tile_count",
            "fbl_attn_tile_info", "fbl_attn_candidates", "fbl_attn_auto_tiles", "fbl_attn_tune", "fbl_attn_tuned_tile",
            "fbl_attn_tune_reset", "fbl_proj", "fbl_proj_dt",
            "fbl_gemm_tile_count", "fbl_gemm_tile_info", "fbl_proj_candidates", "fbl_proj_tune", "fbl_proj_tuned_tile", "fbl_proj_auto_tile",
            "fbl_proj_tune_reset", "fbl_status_str")


class Layout(ctypes.Structure):
    """Mirror of fbl_layout."""
    _fields_ = [("dtype", ctypes.c_int32), ("reserved0", ctypes.c_int32), ("tile_d", ctypes.c_int32),
                ("reserved1", ctypes.c_int32),
                ("B", ctypes.c_int64), ("S", ctypes.c_int64), ("H", ctypes.c_int64), ("D", ctypes.c_int64),
                ("sb", ctypes.c_int64), ("ss", ctypes.c_int64), ("sh", ctypes.c_int64), ("sd", ctypes.c_int64)]

    def __repr__(self):
        return (f"Layout(dtype={self.dtype}, B={self.B}, S={self.S}, H={self.H}, D={self.D}, "
                f"sb={self.sb}, ss={self.ss}, sh={self.sh}, sd={self.sd}, tile_d={self.tile_d})")


class Mask(ctypes.Structure):
    """Mirror of fbl_mask."""
    _fields_ = [("kind", ctypes.c_uint32), ("reserved", ctypes.c_uint32), ("kv_len", ctypes.c_void_p)]


class FblError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {status_str(status)} (status {status})")


def _load() -> ctypes.CDLL:
    # torch bundles its own HIP runtime (soname libamdhip64.so.7).  Loading it
    # first makes libfbl.so bind to that same runtime instead of pulling in a
    # second copy from /opt/rocm: one runtime owns the device memory and the
    # streams that torch hands over.
    import torch  # noqa: F401
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"libfbl.so not built at {LIB_PATH}; run __graft_entry__.build() "
                          "or python paper_2607_21624_amd/build.py")
    lib = ctypes.CDLL(LIB_PATH)
    P = ctypes.POINTER
    vp = ctypes.c_void_p
    lib.fbl_layout_desc.argtypes = [P(Layout), ctypes.c_int32] + [ctypes.c_int64] * 7
    lib.fbl_layout_desc.restype = ctypes.c_int
    lib.fbl_layout_packed_qkv.argtypes = [P(Layout), P(Layout), P(Layout), P(ctypes.c_int64), P(ctypes.c_int64),
                                          ctypes.c_int32] + [ctypes.c_int64] * 7
    lib.fbl_layout_packed_qkv.restype = ctypes.c_int
    lib.fbl_layout_offset.argtypes = [P(Layout)] + [ctypes.c_int64] * 4
    lib.fbl_layout_offset.restype = ctypes.c_int64
    lib.fbl_layout_map_device.argtypes = [P(Layout), vp, vp]
    lib.fbl_layout_map_device.restype = ctypes.c_int
    lib.fbl_attn_fwd.argtypes = [P(Layout), vp, P(Layout), vp, P(Layout), vp, P(Layout), vp, vp,
                                 ctypes.c_float, Mask, vp]
    lib.fbl_attn_fwd.restype = ctypes.c_int
    lib.fbl_attn_bwd_workspace.argtypes = [P(Layout), P(Layout), P(ctypes.c_size_t)]
    lib.fbl_attn_bwd_workspace.restype = ctypes.c_int
    lib.fbl_attn_bwd_workspace_min.argtypes = [P(Layout), P(Layout), P(ctypes.c_size_t)]
    lib.fbl_attn_bwd_workspace_min.restype = ctypes.c_int
    lib.fbl_attn_bwd.argtypes = [P(Layout), vp, P(Layout), vp, P(Layout), vp, P(Layout), vp, P(Layout), vp,
                                 vp, ctypes.c_float, Mask, P(Layout), vp, P(Layout), vp, P(Layout), vp,
                                 vp, ctypes.c_size_t, vp]
    lib.fbl_attn_bwd.restype = ctypes.c_int
    lib.fbl_attn_bwd_phases.argtypes = [ctypes.c_uint32] + lib.fbl_attn_bwd.argtypes
    lib.fbl_attn_bwd_phases.restype = ctypes.c_int
    lib.fbl_attn_bwd_noalloc.argtypes = lib.fbl_attn_bwd.argtypes[:19] + [vp]
    lib.fbl_attn_bwd_noalloc.restype = ctypes.c_int
    lib.fbl_attn_fwd_tiled.argtypes = lib.fbl_attn_fwd.argtypes[:11] + [ctypes.c_int32, vp]
    lib.fbl_attn_fwd_tiled.restype = ctypes.c_int
    lib.fbl_attn_bwd_tiled.argtypes = [ctypes.c_uint32] + lib.fbl_attn_bwd.argtypes[:21] + [ctypes.c_int32,
                                                                                         ctypes.c_int32, vp]
    lib.fbl_attn_bwd_tiled.restype = ctypes.c_int
    lib.fbl_attn_tile_count.argtypes = []
    lib.fbl_attn_tile_count.restype = ctypes.c_int32
    lib.fbl_attn_tile_info.argtypes = [ctypes.c_int32, ctypes.c_int64, P(ctypes.c_int32)]
    lib.fbl_attn_tile_info.restype = ctypes.c_int
    lib.fbl_attn_candidates.argtypes = [ctypes.c_uint32, P(Layout), P(Layout), P(ctypes.c_int32), ctypes.c_int32,
                                        P(ctypes.c_int32)]
    lib.fbl_attn_candidates.restype = ctypes.c_int
    lib.fbl_attn_auto_tiles.argtypes = [P(Layout), P(Layout), ctypes.c_uint32, P(ctypes.c_int32)]
    lib.fbl_attn_auto_tiles.restype = ctypes.c_int
    lib.fbl_attn_bwd_launches.argtypes = [ctypes.c_uint32, P(Layout), P(Layout), ctypes.c_uint32, ctypes.c_size_t,
                                          ctypes.c_int32, ctypes.c_int32, P(ctypes.c_int32)]
    lib.fbl_attn_bwd_launches.restype = ctypes.c_int
    lib.fbl_attn_tune.argtypes = ([P(Layout), vp, P(Layout), vp, P(Layout), vp, P(Layout), vp, vp, P(Layout), vp,
                                   ctypes.c_float, Mask, P(Layout), vp, P(Layout), vp, P(Layout), vp, vp,
                                   ctypes.c_size_t, ctypes.c_uint32, ctypes.c_int32, P(ctypes.c_float),
                                   P(ctypes.c_int32), vp])
    lib.fbl_attn_tune.restype = ctypes.c_int
    lib.fbl_attn_tuned_tile.argtypes = [ctypes.c_uint32, P(Layout), P(Layout), ctypes.c_uint32]
    lib.fbl_attn_tuned_tile.restype = ctypes.c_int32
    lib.fbl_attn_tune_reset.argtypes = []
    lib.fbl_attn_tune_reset.restype = None
    lib.fbl_proj.argtypes = [ctypes.c_uint32] + [ctypes.c_int64] * 3 + [vp, ctypes.c_int64, vp, ctypes.c_int64, vp,
                                                                        ctypes.c_int64, ctypes.c_int32, vp]
    lib.fbl_proj.restype = ctypes.c_int
    lib.fbl_proj_dt.argtypes = [ctypes.c_uint32, ctypes.c_int32] + [ctypes.c_int64] * 3 + [vp, ctypes.c_int64, vp,
                                                                                   ctypes.c_int64, vp, ctypes.c_int64,
                                                                                   ctypes.c_int32, vp]
    lib.fbl_proj_dt.restype = ctypes.c_int
    lib.fbl_gemm_tile_count.argtypes = []
    lib.fbl_gemm_tile_count.restype = ctypes.c_int32
    lib.fbl_gemm_tile_info.argtypes = [ctypes.c_int32, P(ctypes.c_int32)]
    lib.fbl_gemm_tile_info.restype = ctypes.c_int
    lib.fbl_proj_candidates.argtypes = [ctypes.c_uint32] + [ctypes.c_int64] * 3 + [P(ctypes.c_int32), ctypes.c_int32,
                                                                                 P(ctypes.c_int32)]
    lib.fbl_proj_candidates.restype = ctypes.c_int
    lib.fbl_proj_tune.argtypes = lib.fbl_proj.argtypes[:10] + [ctypes.c_uint32, ctypes.c_int32, P(ctypes.c_float),
                                                              P(ctypes.c_int32), vp]
    lib.fbl_proj_tune.restype = ctypes.c_int
    lib.fbl_proj_tuned_tile.argtypes = [ctypes.c_uint32] + [ctypes.c_int64] * 3
    lib.fbl_proj_tuned_tile.restype = ctypes.c_int32
    lib.fbl_proj_auto_tile.argtypes = [ctypes.c_uint32] + [ctypes.c_int64] * 3 + [ctypes.POINTER(ctypes.c_int32)]
    lib.fbl_proj_auto_tile.restype = ctypes.c_int
    lib.fbl_proj_tune_reset.argtypes = []
    lib.fbl_proj_tune_reset.restype = None
    lib.fbl_status_str.argtypes = [ctypes.c_int]
    lib.fbl_status_str.restype = ctypes.c_char_p
    return lib


LIB = _load()


def status_str(status: int) -> str:
    return LIB.fbl_status_str(int(status)).decode()


def _check(status: int, where: str) -> None:
    if status != FBL_OK:
        raise FblError(status, where)


# ------------------------------------------------------------------ layouts
def fbl_layout_desc(dtype: int, B: int, S: int, H: int, D: int, row_stride: int = 0, batch_stride: int = 0,
                    tile_d: int = 0) -> Layout:
    out = Layout()
    _check(LIB.fbl_layout_desc(ctypes.byref(out), dtype, B, S, H, D, row_stride, batch_stride, tile_d),
           "fbl_layout_desc")
    return out


def fbl_layout_desc_status(dtype: int, B: int, S: int, H: int, D: int, row_stride: int = 0,
                           batch_stride: int = 0, tile_d: int = 0) -> Tuple[int, Layout]:
    """Like fbl_layout_desc but returns (status, layout) instead of raising."""
    out = Layout()
    st = LIB.fbl_layout_desc(ctypes.byref(out), dtype, B, S, H, D, row_stride, batch_stride, tile_d)
    return st, out


def fbl_layout_packed_qkv(dtype: int, B: int, S: int, Hq: int, Hkv: int, D: int, batch_stride: int = 0,
                          tile_d: int = 0):
    """Descriptors of Q, K, V inside one packed [B, S, (Hq + 2 Hkv) D] projection
    output: returns (lq, lk, lv, k_off, v_off), offsets in elements."""
    lq, lk, lv = Layout(), Layout(), Layout()
    ko, vo = ctypes.c_int64(0), ctypes.c_int64(0)
    _check(LIB.fbl_layout_packed_qkv(ctypes.byref(lq), ctypes.byref(lk), ctypes.byref(lv), ctypes.byref(ko),
                                     ctypes.byref(vo), dtype, B, S, Hq, Hkv, D, batch_stride, tile_d),
           "fbl_layout_packed_qkv")
    return lq, lk, lv, int(ko.value), int(vo.value)


def fbl_layout_offset(l: Layout, b: int, h: int, s: int, i: int) -> int:
    return LIB.fbl_layout_offset(ctypes.byref(l), b, h, s, i)


def _ptr(x) -> Optional[int]:
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def fbl_layout_map_device(l: Layout, out, stream=None) -> None:
    _check(LIB.fbl_layout_map_device(ctypes.byref(l), _ptr(out), _stream(stream)), "fbl_layout_map_device")


def _mask(causal: bool, kv_len) -> Mask:
    kind = (FBL_MASK_CAUSAL if causal else 0) | (FBL_MASK_KEY_PADDING if kv_len is not None else 0)
    return Mask(kind, 0, _ptr(kv_len))


def fbl_attn_fwd_raw(lq, q, lk, k, lv, v, lo, o, lse, scale, mask: Mask, stream=None,
                     tile: int = FBL_ATTN_TILE_AUTO) -> int:
    """Direct call of fbl_attn_fwd (tile AUTO) or fbl_attn_fwd_tiled; returns the status code."""
    ref = lambda l: ctypes.byref(l) if l is not None else None
    args = (ref(lq), _ptr(q), ref(lk), _ptr(k), ref(lv), _ptr(v), ref(lo), _ptr(o), _ptr(lse), float(scale), mask)
    st = _stream(stream) if stream != 0 else None
    if tile == FBL_ATTN_TILE_AUTO:
        return LIB.fbl_attn_fwd(*args, st)
    return LIB.fbl_attn_fwd_tiled(*args, int(tile), st)


def fbl_attn_bwd_workspace(lq: Layout, lk: Layout) -> int:
    n = ctypes.c_size_t(0)
    _check(LIB.fbl_attn_bwd_workspace(ctypes.byref(lq), ctypes.byref(lk), ctypes.byref(n)), "fbl_attn_bwd_workspace")
    return int(n.value)


def fbl_attn_bwd_workspace_min(lq: Layout, lk: Layout) -> int:
    n = ctypes.c_size_t(0)
    _check(LIB.fbl_attn_bwd_workspace_min(ctypes.byref(lq), ctypes.byref(lk), ctypes.byref(n)),
           "fbl_attn_bwd_workspace_min")
    return int(n.value)


def fbl_attn_bwd_raw(lq, q, lk, k, lv, v, lo, o, ldo, do, lse, scale, mask: Mask, ldq, dq, ldk, dk, ldv, dv,
                     ws, ws_bytes, stream=None, phases: int = FBL_BWD_ALL, kv_tile: int = FBL_ATTN_TILE_AUTO,
                     dq_tile: int = FBL_ATTN_TILE_AUTO) -> int:
    """Direct call of fbl_attn_bwd (phases == FBL_BWD_ALL, AUTO tiles), fbl_attn_bwd_phases (AUTO
    tiles) or fbl_attn_bwd_tiled (an explicit tile); returns the status."""
    ref = lambda l: ctypes.byref(l) if l is not None else None
    args = (ref(lq), _ptr(q), ref(lk), _ptr(k), ref(lv), _ptr(v), ref(lo), _ptr(o), ref(ldo), _ptr(do), _ptr(lse),
            float(scale), mask, ref(ldq), _ptr(dq), ref(ldk), _ptr(dk), ref(ldv), _ptr(dv), _ptr(ws), int(ws_bytes))
    st = _stream(stream) if stream != 0 else None
    if kv_tile != FBL_ATTN_TILE_AUTO or dq_tile != FBL_ATTN_TILE_AUTO:
        return LIB.fbl_attn_bwd_tiled(phases, *args, int(kv_tile), int(dq_tile), st)
    if phases == FBL_BWD_ALL:
        return LIB.fbl_attn_bwd(*args, st)
    return LIB.fbl_attn_bwd_phases(phases, *args, st)


# ------------------------------------------------------- torch-tensor helpers
def _dtype_code(t) -> int:
    import torch
    if t.dtype == torch.bfloat16:
        return FBL_BF16
    if t.dtype == torch.float32:
        return FBL_F32
    raise FblError(FBL_ERR_DTYPE, f"unsupported tensor dtype {t.dtype}")


_LAYOUTS = {}


def _layout(t, H: int) -> Layout:
    """layout_of for the calls below, cached per (dtype, shape, strides, H): the
    descriptor only depends on those, and building it costs a library call per
    tensor per launch.  The cached objects are passed read-only (const) and
    never handed out."""
    key = (t.dtype, tuple(t.shape), t.stride(), H)
    l = _LAYOUTS.get(key)
    if l is None:
        l = layout_of(t, H)
        if len(_LAYOUTS) < 4096:
            _LAYOUTS[key] = l
    return l


def layout_of(t, H: int) -> Layout:
    """Descriptor of a token-major [B, S, H*D] tensor (or a strided view of one:
    inner stride 1, arbitrary row and batch strides).  No data is touched."""
    if t.dim() != 3:
        raise FblError(FBL_ERR_SHAPE, "expected a [B, S, H*D] tensor")
    B, S, HD = t.shape
    if HD % H:
        raise FblError(FBL_ERR_SHAPE, f"last dim {HD} not divisible by heads {H}")
    if t.stride(2) != 1:
        raise FblError(FBL_ERR_LAYOUT, "innermost stride must be 1")
    return fbl_layout_desc(_dtype_code(t), B, S, H, HD // H, row_stride=t.stride(1),
                           batch_stride=t.stride(0) if B > 1 else 0)


def _check_kv_len(kv_len, B: int, where: str) -> None:
    """kv_len must be an int32 tensor of at least B entries with unit stride:
    the kernels read kv_len[b] as a 32-bit integer from device memory."""
    if kv_len is None:
        return
    import torch
    if not isinstance(kv_len, torch.Tensor):
        raise FblError(FBL_ERR_ARG, f"{where}: kv_len must be a torch tensor")
    if kv_len.dtype != torch.int32:
        raise FblError(FBL_ERR_DTYPE, f"{where}: kv_len must be int32, got {kv_len.dtype}")
    if kv_len.dim() != 1 or (kv_len.numel() > 1 and kv_len.stride(0) != 1):
        raise FblError(FBL_ERR_LAYOUT, f"{where}: kv_len must be a 1-D tensor with unit stride")
    if kv_len.numel() < B:
        raise FblError(FBL_ERR_SHAPE, f"{where}: kv_len has {kv_len.numel()} entries, needs {B}")


def _check_lse(lse, B: int, Hq: int, S: int, where: str) -> None:
    """lse must be a contiguous float32 [B, Hq, S_q] tensor: the kernels read and
    write it as B*Hq*S_q consecutive floats."""
    if lse is None:
        return
    import torch
    if not isinstance(lse, torch.Tensor):
        raise FblError(FBL_ERR_ARG, f"{where}: lse must be a torch tensor")
    if lse.dtype != torch.float32:
        raise FblError(FBL_ERR_DTYPE, f"{where}: lse must be float32, got {lse.dtype}")
    if tuple(lse.shape) != (B, Hq, S):
        raise FblError(FBL_ERR_SHAPE, f"{where}: lse has shape {tuple(lse.shape)}, needs {(B, Hq, S)}")
    if not lse.is_contiguous():
        raise FblError(FBL_ERR_LAYOUT, f"{where}: lse must be contiguous")


def _check_workspace(ws, where: str) -> None:
    """The workspace is handed over as one span of numel * element_size bytes."""
    if ws is None:
        return
    import torch
    if not isinstance(ws, torch.Tensor):
        raise FblError(FBL_ERR_ARG, f"{where}: workspace must be a torch tensor")
    if not ws.is_contiguous():
        raise FblError(FBL_ERR_LAYOUT, f"{where}: workspace must be contiguous")


def _check_device(where: str, stream, **tensors) -> None:
    """Every tensor argument lives on one GPU, the device the launch stream
    belongs to: the kernels dereference each pointer on that device."""
    import torch
    dev = None
    for name, t in tensors.items():
        if t is None:
            continue
        if not t.is_cuda:
            raise FblError(FBL_ERR_ARG, f"{where}: {name} is on {t.device}, not on a GPU")
        if dev is None:
            dev = t.device
        elif t.device != dev:
            raise FblError(FBL_ERR_ARG, f"{where}: {name} is on {t.device}, the other tensors on {dev}")
    if dev is None or isinstance(stream, int) or stream == 0:
        return
    sdev = torch.cuda.current_device() if stream is None else stream.device.index
    if sdev != dev.index:
        raise FblError(FBL_ERR_ARG, f"{where}: tensors are on {dev}, the stream on cuda:{sdev}")


def attn_fwd(q, k, v, Hq: int, Hkv: int, scale: Optional[float] = None, causal: bool = False, kv_len=None,
             out=None, lse=None, stream=None, tile: int = FBL_ATTN_TILE_AUTO):
    """Forward on token-major tensors.  Returns (O, LSE); O has q's shape and dtype
    (allocated contiguous unless `out` is given), LSE is float32 [B, Hq, S]."""
    import torch
    _check_kv_len(kv_len, q.shape[0], "attn_fwd")
    _check_device("attn_fwd", stream, q=q, k=k, v=v, kv_len=kv_len, out=out, lse=lse)
    if q.dim() == 3:
        _check_lse(lse, q.shape[0], Hq, q.shape[1], "attn_fwd")
    lq, lk, lv = _layout(q, Hq), _layout(k, Hkv), _layout(v, Hkv)
    if scale is None:
        scale = 1.0 / math.sqrt(lq.D)
    B, S = q.shape[0], q.shape[1]
    if out is None:
        out = torch.empty((B, S, q.shape[2]), dtype=q.dtype, device=q.device)
    if lse is None:
        lse = torch.empty((B, Hq, S), dtype=torch.float32, device=q.device)
    lo = _layout(out, Hq)
    _check(fbl_attn_fwd_raw(lq, q, lk, k, lv, v, lo, out, lse, scale, _mask(causal, kv_len), stream, tile),
           "fbl_attn_fwd")
    return out, lse


def attn_bwd(q, k, v, o, do, lse, Hq: int, Hkv: int, scale: Optional[float] = None, causal: bool = False,
             kv_len=None, dq=None, dk=None, dv=None, workspace=None, stream=None, phases: int = FBL_BWD_ALL,
             kv_tile: int = FBL_ATTN_TILE_AUTO, dq_tile: int = FBL_ATTN_TILE_AUTO):
    """Backward.  Returns (dQ, dK, dV) with the shapes/dtypes of q, k, v."""
    import torch
    _check_kv_len(kv_len, q.shape[0], "attn_bwd")
    _check_device("attn_bwd", stream, q=q, k=k, v=v, o=o, do=do, lse=lse, kv_len=kv_len, dq=dq, dk=dk, dv=dv,
                  workspace=workspace)
    if q.dim() == 3:
        _check_lse(lse, q.shape[0], Hq, q.shape[1], "attn_bwd")
    _check_workspace(workspace, "attn_bwd")
    lq, lk, lv = _layout(q, Hq), _layout(k, Hkv), _layout(v, Hkv)
    lo, ldo = _layout(o, Hq), _layout(do, Hq)
    if scale is None:
        scale = 1.0 / math.sqrt(lq.D)
    if dq is None:
        dq = torch.empty(q.shape, dtype=q.dtype, device=q.device)
    if dk is None:
        dk = torch.empty(k.shape, dtype=k.dtype, device=k.device)
    if dv is None:
        dv = torch.empty(v.shape, dtype=v.dtype, device=v.device)
    if workspace is None:
        need = fbl_attn_bwd_workspace(lq, lk)
        workspace = torch.empty(need, dtype=torch.uint8, device=q.device)
    ldq, ldk, ldv = _layout(dq, Hq), _layout(dk, Hkv), _layout(dv, Hkv)
    _check(fbl_attn_bwd_raw(lq, q, lk, k, lv, v, lo, o, ldo, do, lse, scale, _mask(causal, kv_len), ldq, dq, ldk,
                            dk, ldv, dv, workspace, workspace.numel() * workspace.element_size(), stream,
                            phases, kv_tile, dq_tile), "fbl_attn_bwd")
    return dq, dk, dv


# ------------------------------------------------------- attention tiles
def attn_tiles(D: int):
    """Every attention tile configuration at head dim D:
    {id: dict(pass, rows, cols, waves, per_wave, occupancy, lds_bytes, legal)}."""
    keys = ("pass", "rows", "cols", "waves", "per_wave", "occupancy", "lds_bytes", "legal")
    out = {}
    for t in range(LIB.fbl_attn_tile_count()):
        info = (ctypes.c_int32 * 8)()
        _check(LIB.fbl_attn_tile_info(t, D, info), "fbl_attn_tile_info")
        out[t] = dict(zip(keys, list(info)))
    return out


def attn_candidates(pass_: int, lq: Layout, lk: Layout):
    """Candidate tile ids of one attention pass for these shapes (C1/C2/C3)."""
    n = ctypes.c_int32()
    cap = LIB.fbl_attn_tile_count()
    ids = (ctypes.c_int32 * cap)()
    _check(LIB.fbl_attn_candidates(pass_, ctypes.byref(lq), ctypes.byref(lk), ids, cap, ctypes.byref(n)),
           "fbl_attn_candidates")
    return list(ids[:n.value])


def attn_auto_tiles(lq: Layout, lk: Layout, mask_kind: int):
    """(forward, kv, dQ) tile ids FBL_ATTN_TILE_AUTO resolves to."""
    t = (ctypes.c_int32 * 3)()
    _check(LIB.fbl_attn_auto_tiles(ctypes.byref(lq), ctypes.byref(lk), mask_kind, t), "fbl_attn_auto_tiles")
    return tuple(t)


def attn_bwd_launches(lq: Layout, lk: Layout, mask_kind: int, ws_bytes: int, phases: int = FBL_BWD_ALL,
                      kv_tile: int = FBL_ATTN_TILE_AUTO, dq_tile: int = FBL_ATTN_TILE_AUTO) -> int:
    """Kernel launches a backward call with these shapes, mask bits, workspace
    size and tiles enqueues (1: the one-launch backward)."""
    n = ctypes.c_int32()
    _check(LIB.fbl_attn_bwd_launches(phases, ctypes.byref(lq), ctypes.byref(lk), mask_kind, ws_bytes, kv_tile,
                                     dq_tile, ctypes.byref(n)), "fbl_attn_bwd_launches")
    return n.value


def attn_tune(q, k, v, do, Hq: int, Hkv: int, scale: Optional[float] = None, causal: bool = False, kv_len=None,
              o=None, lse=None, dq=None, dk=None, dv=None, workspace=None, objective: int = FBL_TUNE_TIME,
              reps: int = 10, stream=None):
    """Measured tile selection for this attention shape (fbl_attn_tune).  Returns
    ((fwd, kv, dq) chosen ids, {id: average ms}, outputs (o, lse, dq, dk, dv)
    computed with the chosen tiles)."""
    import torch
    _check_kv_len(kv_len, q.shape[0], "attn_tune")
    _check_device("attn_tune", stream, q=q, k=k, v=v, do=do, kv_len=kv_len, o=o, lse=lse, dq=dq, dk=dk, dv=dv,
                  workspace=workspace)
    if q.dim() == 3:
        _check_lse(lse, q.shape[0], Hq, q.shape[1], "attn_tune")
    _check_workspace(workspace, "attn_tune")
    lq, lk, lv, ldo = _layout(q, Hq), _layout(k, Hkv), _layout(v, Hkv), _layout(do, Hq)
    if scale is None:
        scale = 1.0 / math.sqrt(lq.D)
    B, S = q.shape[0], q.shape[1]
    o = torch.empty(q.shape, dtype=q.dtype, device=q.device) if o is None else o
    lse = torch.empty((B, Hq, S), dtype=torch.float32, device=q.device) if lse is None else lse
    dq = torch.empty(q.shape, dtype=q.dtype, device=q.device) if dq is None else dq
    dk = torch.empty(k.shape, dtype=k.dtype, device=k.device) if dk is None else dk
    dv = torch.empty(v.shape, dtype=v.dtype, device=v.device) if dv is None else dv
    if workspace is None:
        workspace = torch.empty(fbl_attn_bwd_workspace(lq, lk), dtype=torch.uint8, device=q.device)
    lo, ldq, ldk, ldv = _layout(o, Hq), _layout(dq, Hq), _layout(dk, Hkv), _layout(dv, Hkv)
    cap = LIB.fbl_attn_tile_count()
    ms = (ctypes.c_float * cap)()
    best = (ctypes.c_int32 * 3)()
    ref = ctypes.byref
    _check(LIB.fbl_attn_tune(ref(lq), _ptr(q), ref(lk), _ptr(k), ref(lv), _ptr(v), ref(lo), _ptr(o), _ptr(lse),
                             ref(ldo), _ptr(do), float(scale), _mask(causal, kv_len), ref(ldq), _ptr(dq), ref(ldk),
                             _ptr(dk), ref(ldv), _ptr(dv), _ptr(workspace),
                             workspace.numel() * workspace.element_size(), objective, reps, ms, best,
                             _stream(stream) if stream != 0 else None), "fbl_attn_tune")
    return tuple(best), {t: ms[t] for t in range(cap) if ms[t] >= 0}, (o, lse, dq, dk, dv)


def attn_tuned_tile(pass_: int, lq: Layout, lk: Layout, mask_kind: int) -> int:
    """The tile fbl_attn_tune chose for this pass and shape in this process, or -1."""
    return LIB.fbl_attn_tuned_tile(pass_, ctypes.byref(lq), ctypes.byref(lk), mask_kind)


def attn_tune_reset() -> None:
    LIB.fbl_attn_tune_reset()


NOALLOC_SCRATCH_BYTES = 64 << 20  # FBL_NOALLOC_SCRATCH_BYTES


def fbl_attn_bwd_noalloc_raw(lq, q, lk, k, lv, v, lo, o, ldo, do, lse, scale, mask: Mask, ldq, dq, ldk, dk, ldv,
                             dv, stream=None) -> int:
    """Direct call of fbl_attn_bwd_noalloc; returns the status."""
    ref = lambda l: ctypes.byref(l) if l is not None else None
    return LIB.fbl_attn_bwd_noalloc(ref(lq), _ptr(q), ref(lk), _ptr(k), ref(lv), _ptr(v), ref(lo), _ptr(o), ref(ldo),
                                    _ptr(do), _ptr(lse), float(scale), mask, ref(ldq), _ptr(dq), ref(ldk), _ptr(dk),
                                    ref(ldv), _ptr(dv), _stream(stream) if stream != 0 else None)


def attn_bwd_noalloc(q, k, v, o, do, lse, Hq: int, Hkv: int, dq, dk, dv, scale: Optional[float] = None,
                     causal: bool = False, kv_len=None, stream=None):
    """Backward through fbl_attn_bwd_noalloc: the library's own device scratch
    replaces the workspace, so nothing is allocated; dq, dk, dv are the
    caller's preallocated outputs (shapes and dtypes of q, k, v)."""
    _check_kv_len(kv_len, q.shape[0], "attn_bwd_noalloc")
    _check_device("attn_bwd_noalloc", stream, q=q, k=k, v=v, o=o, do=do, lse=lse, kv_len=kv_len, dq=dq, dk=dk,
                  dv=dv)
    if q.dim() == 3:
        _check_lse(lse, q.shape[0], Hq, q.shape[1], "attn_bwd_noalloc")
    lq, lk, lv = _layout(q, Hq), _layout(k, Hkv), _layout(v, Hkv)
    lo, ldo = _layout(o, Hq), _layout(do, Hq)
    ldq, ldk, ldv = _layout(dq, Hq), _layout(dk, Hkv), _layout(dv, Hkv)
    if scale is None:
        scale = 1.0 / math.sqrt(lq.D)
    _check(fbl_attn_bwd_noalloc_raw(lq, q, lk, k, lv, v, lo, o, ldo, do, lse, scale, _mask(causal, kv_len), ldq, dq,
                                    ldk, dk, ldv, dv, stream), "fbl_attn_bwd_noalloc")
    return dq, dk, dv


# ------------------------------------------------- packed QKV projection output
def _packed(qkv, Hq: int, Hkv: int):
    import torch
    if qkv.dim() != 3 or qkv.stride(2) != 1 or qkv.stride(1) != qkv.shape[2]:
        raise FblError(FBL_ERR_LAYOUT, "expected a [B, S, (Hq + 2 Hkv) D] tensor with contiguous rows")
    B, S, W = qkv.shape
    if W % (Hq + 2 * Hkv):
        raise FblError(FBL_ERR_SHAPE, f"row width {W} not divisible by Hq + 2 Hkv = {Hq + 2 * Hkv}")
    D = W // (Hq + 2 * Hkv)
    lq, lk, lv, ko, vo = fbl_layout_packed_qkv(_dtype_code(qkv), B, S, Hq, Hkv, D,
                                               batch_stride=qkv.stride(0) if B > 1 else 0)
    es = qkv.element_size()
    base = qkv.data_ptr()
    return lq, lk, lv, base, base + ko * es, base + vo * es


def attn_fwd_packed(qkv, Hq: int, Hkv: int, scale: Optional[float] = None, causal: bool = False, kv_len=None,
                    out=None, lse=None, stream=None):
    """Forward on a packed QKV projection output [B, S, (Hq + 2 Hkv) D]: Q, K and
    V are read in place through fbl_layout_packed_qkv descriptors.  Returns
    (O [B, S, Hq D], LSE [B, Hq, S])."""
    import torch
    _check_kv_len(kv_len, qkv.shape[0], "attn_fwd_packed")
    _check_device("attn_fwd_packed", stream, qkv=qkv, kv_len=kv_len, out=out, lse=lse)
    if qkv.dim() == 3:
        _check_lse(lse, qkv.shape[0], Hq, qkv.shape[1], "attn_fwd_packed")
    lq, lk, lv, pq, pk, pv = _packed(qkv, Hq, Hkv)
    if scale is None:
        scale = 1.0 / math.sqrt(lq.D)
    B, S = qkv.shape[0], qkv.shape[1]
    if out is None:
        out = torch.empty((B, S, Hq * lq.D), dtype=qkv.dtype, device=qkv.device)
    if lse is None:
        lse = torch.empty((B, Hq, S), dtype=torch.float32, device=qkv.device)
    lo = _layout(out, Hq)
    _check(fbl_attn_fwd_raw(lq, pq, lk, pk, lv, pv, lo, out, lse, scale, _mask(causal, kv_len), stream),
           "fbl_attn_fwd")
    return out, lse


def attn_bwd_packed(qkv, o, do, lse, Hq: int, Hkv: int, scale: Optional[float] = None, causal: bool = False,
                    kv_len=None, dqkv=None, workspace=None, stream=None):
    """Backward on a packed QKV projection output: dQ, dK, dV are written into
    one packed gradient tensor shaped like ``qkv`` (allocated unless given)."""
    import torch
    _check_kv_len(kv_len, qkv.shape[0], "attn_bwd_packed")
    _check_device("attn_bwd_packed", stream, qkv=qkv, o=o, do=do, lse=lse, kv_len=kv_len, dqkv=dqkv,
                  workspace=workspace)
    if qkv.dim() == 3:
        _check_lse(lse, qkv.shape[0], Hq, qkv.shape[1], "attn_bwd_packed")
    _check_workspace(workspace, "attn_bwd_packed")
    lq, lk, lv, pq, pk, pv = _packed(qkv, Hq, Hkv)
    if scale is None:
        scale = 1.0 / math.sqrt(lq.D)
    if dqkv is None:
        dqkv = torch.empty(qkv.shape, dtype=qkv.dtype, device=qkv.device)
    if dqkv.shape != qkv.shape or dqkv.stride() != qkv.stride() or dqkv.dtype != qkv.dtype:
        raise FblError(FBL_ERR_SHAPE, "dqkv must have qkv's shape, strides and dtype")
    _, _, _, gq, gk, gv = _packed(dqkv, Hq, Hkv)
    lo, ldo = _layout(o, Hq), _layout(do, Hq)
    if workspace is None:
        workspace = torch.empty(fbl_attn_bwd_workspace(lq, lk), dtype=torch.uint8, device=qkv.device)
    _check(fbl_attn_bwd_raw(lq, pq, lk, pk, lv, pv, lo, o, ldo, do, lse, scale, _mask(causal, kv_len), lq, gq, lk,
                            gk, lv, gv, workspace, workspace.numel() * workspace.element_size(), stream),
           "fbl_attn_bwd")
    return dqkv


# ------------------------------------------------------- projection products
def fbl_proj_raw(op, M, K, N, a, lda, b, ldb, c, ldc, tile=FBL_GEMM_TILE_AUTO, stream=None) -> int:
    """Direct call of fbl_proj; returns the status code."""
    return LIB.fbl_proj(op, M, K, N, _ptr(a), lda, _ptr(b), ldb, _ptr(c), ldc, tile,
                        _stream(stream) if stream != 0 else None)


def _rows(t, name):
    if t.dim() != 2 or t.stride(1) != 1:
        raise FblError(FBL_ERR_LAYOUT, f"{name}: expected a 2-D row-major tensor (inner stride 1)")
    return t.shape[0], t.shape[1], t.stride(0)


def _proj_shape(op, a, b):
    ra, wa, lda = _rows(a, "a")
    rb, wb, ldb = _rows(b, "b")
    if op == FBL_PROJ_FWD:
        M, K, N, shape = ra, wa, wb, (ra, wb)
    elif op == FBL_PROJ_BWD_DATA:
        M, N, K, shape = ra, wa, rb, (ra, rb)
    else:
        M, K, N, shape = ra, wa, wb, (wa, wb)
    return M, K, N, shape, lda, ldb


def proj(op: int, a, b, out=None, tile: int = FBL_GEMM_TILE_AUTO, stream=None):
    """One projection product on 2-D bf16 or fp32 tensors (row-major, any row stride):
    FBL_PROJ_FWD (a = X [M, K], b = W [K, N]) -> Y [M, N];
    FBL_PROJ_BWD_DATA (a = dY [M, N], b = W [K, N]) -> dX [M, K];
    FBL_PROJ_BWD_WEIGHT (a = X [M, K], b = dY [M, N]) -> dW [K, N]."""
    import torch
    _check_device("proj", stream, a=a, b=b, out=out)
    M, K, N, shape, lda, ldb = _proj_shape(op, a, b)
    if out is None:
        out = torch.empty(shape, dtype=a.dtype, device=a.device)
    _, _, ldc = _rows(out, "out")
    if not (a.dtype == b.dtype == out.dtype):
        raise FblError(FBL_ERR_DTYPE, f"proj: operand dtypes differ ({a.dtype}, {b.dtype}, {out.dtype})")
    if a.dtype == torch.float32:
        _check(LIB.fbl_proj_dt(op, FBL_F32, M, K, N, _ptr(a), lda, _ptr(b), ldb, _ptr(out), ldc, tile,
                               _stream(stream) if stream != 0 else None), "fbl_proj_dt")
    else:
        _check(fbl_proj_raw(op, M, K, N, a, lda, b, ldb, out, ldc, tile, stream), "fbl_proj")
    return out


def gemm_tiles():
    """Every tile configuration: {id: dict(bm, bn, bk, stages, wm, wn, wk, lds_bytes)}."""
    keys = ("bm", "bn", "bk", "stages", "wm", "wn", "wk", "lds_bytes")
    out = {}
    for t in range(LIB.fbl_gemm_tile_count()):
        info = (ctypes.c_int32 * 8)()
        _check(LIB.fbl_gemm_tile_info(t, info), "fbl_gemm_tile_info")
        out[t] = dict(zip(keys, list(info)))
    return out


def proj_candidates(op: int, M: int, K: int, N: int):
    """Candidate tile ids of one product shape (the C1/C2/C3 filters)."""
    n = ctypes.c_int32()
    cap = LIB.fbl_gemm_tile_count()
    ids = (ctypes.c_int32 * cap)()
    _check(LIB.fbl_proj_candidates(op, M, K, N, ids, cap, ctypes.byref(n)), "fbl_proj_candidates")
    return list(ids[:n.value])


def proj_tune(op: int, a, b, out, objective: int = FBL_TUNE_TIME, reps: int = 10, stream=None):
    """Measured tile selection for one product (fbl_proj_tune).  Returns
    (chosen id, {id: average ms} over the candidates); `out` then holds the
    product computed with the chosen tile."""
    _check_device("proj_tune", stream, a=a, b=b, out=out)
    M, K, N, _, lda, ldb = _proj_shape(op, a, b)
    _, _, ldc = _rows(out, "out")
    cap = LIB.fbl_gemm_tile_count()
    ms = (ctypes.c_float * cap)()
    best = ctypes.c_int32(-1)
    _check(LIB.fbl_proj_tune(op, M, K, N, _ptr(a), lda, _ptr(b), ldb, _ptr(out), ldc, objective, reps, ms,
                             ctypes.byref(best), _stream(stream) if stream != 0 else None), "fbl_proj_tune")
    return best.value, {t: ms[t] for t in range(cap) if ms[t] >= 0}


def proj_tuned_tile(op: int, M: int, K: int, N: int) -> int:
    """The tile fbl_proj_tune chose for this shape in this process, or -1."""
    return LIB.fbl_proj_tuned_tile(op, M, K, N)


def proj_auto_tile(op: int, M: int, K: int, N: int) -> int:
    """The tile id FBL_GEMM_TILE_AUTO resolves to for this bf16 product."""
    t = ctypes.c_int32(-1)
    _check(LIB.fbl_proj_auto_tile(op, M, K, N, ctypes.byref(t)), "fbl_proj_auto_tile")
    return t.value


def proj_tune_reset() -> None:
    LIB.fbl_proj_tune_reset()
