"""ctypes binding of libdecode_attn.so: argument marshalling only.

Every function has the name of the C entry point it calls.  torch supplies
device memory (tensors), their data pointers and the current HIP stream;
every step of the computation runs in the library's HIP kernels.  torch is
imported before the library is loaded so that both resolve the same HIP
runtime (libamdhip64.so.7).  A missing library raises; there is no fallback.
"""

from __future__ import annotations

import ctypes
import os
from typing import Dict, List, Optional, Sequence, Tuple

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libdecode_attn.so")
HEAD_DIM = 128
MAX_SPLITS = 64

DA_OK = 0
DA_ERR_NULL = -1
DA_ERR_SHAPE = -2
DA_ERR_UNSUPPORTED = -3
DA_ERR_SPLITS = -4
DA_ERR_ALIGN = -5
DA_ERR_WORKSPACE = -6
DA_ERR_HIP = -7
DA_ERR_ARG = -8

POLICY_MI355X = 0
POLICY_PAPER = 1
POLICY_EVOLVED = 2
POLICY_STREAMED = 3
POLICY_TABLE = 4
POLICY_TABLE_STREAMED = 5

# Every symbol include/decode_attn.h declares.
EXPORTS = (
    "da_choose_splits", "da_model_time", "da_make_plan", "da_workspace_bytes", "da_split_bounds", "da_decode_attn",
    "da_decode_attn_planned", "da_decode_attn_noalloc", "da_decode_attn_paged", "da_decode_attn_paged_planned", "da_schedule_max_bytes",
    "da_make_schedule", "da_schedule_workspace_bytes",
    "da_decode_attn_scheduled", "da_split_partials", "da_combine_splits", "da_device_info", "da_strerror",
    "da_last_error",
)


class DaPlan(ctypes.Structure):
    _fields_ = [
        ("num_splits", ctypes.c_int32),
        ("pack_gqa", ctypes.c_int32),
        ("heads_per_tile", ctypes.c_int32),
        ("tiles", ctypes.c_int32),
        ("grid", ctypes.c_int32),
        ("num_cus", ctypes.c_int32),
        ("group_waves", ctypes.c_int32),
        ("kv_fetch", ctypes.c_int32),
        ("kv_nontemporal", ctypes.c_int32),
        ("v_slices", ctypes.c_int32),
        ("combine", ctypes.c_int32),
        ("wg_per_cu", ctypes.c_int32),
    ]

    def as_dict(self) -> dict:
        return {name: int(getattr(self, name)) for name, _ in self._fields_}


class DaSchedule(ctypes.Structure):
    _fields_ = [(name, ctypes.c_int32) for name in (
        "B", "H_Q", "H_KV", "L_K_max", "pack_gqa", "heads_per_tile", "tiles", "num_items", "chunk_tiles",
        "max_splits", "state_rows", "num_cus", "kv_fetch", "seq_offset", "meta_bytes", "kv_nontemporal",
        "combine")]

    def as_dict(self) -> dict:
        return {name: int(getattr(self, name)) for name, _ in self._fields_}


class DecodeAttnError(RuntimeError):
    def __init__(self, code: int, message: str):
        super().__init__(f"{message} (code {code})")
        self.code = code


_lib: Optional[ctypes.CDLL] = None

_I = ctypes.c_int
_P = ctypes.c_void_p
_F = ctypes.c_float
_Z = ctypes.c_size_t


def _hip_runtimes_loaded() -> List[str]:
    paths = set()
    try:
        with open("/proc/self/maps") as f:
            for line in f:
                if "libamdhip64.so" in line:
                    paths.add(line.split()[-1])
    except OSError:
        pass
    return sorted(paths)


def load() -> ctypes.CDLL:
    """Load the built library (once).  Raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2604_00028_amd.build` "
                           "(there is no fallback implementation)")
    lib = ctypes.CDLL(LIB_PATH)
    runtimes = _hip_runtimes_loaded()
    if len(runtimes) > 1:
        raise RuntimeError(f"two HIP runtimes are loaded ({runtimes}); torch must be imported first")
    lib.da_choose_splits.argtypes = [_I, _I, _I, _I, _I, _I, _I, _I, ctypes.POINTER(DaPlan)]
    lib.da_choose_splits.restype = _I
    lib.da_model_time.argtypes = [_I] * 10
    lib.da_model_time.restype = ctypes.c_double
    lib.da_make_plan.argtypes = [_I, _I, _I, _I, _I, _I, _I, _I, _I, _I, ctypes.POINTER(DaPlan)]
    lib.da_make_plan.restype = _I
    lib.da_workspace_bytes.argtypes = [_I, _I, _I, _I]
    lib.da_workspace_bytes.restype = _Z
    lib.da_split_bounds.argtypes = [_I, _I, ctypes.POINTER(ctypes.c_int32)]
    lib.da_split_bounds.restype = _I
    lib.da_decode_attn.argtypes = [_P, _P, _P, _P, _P, _P, _I, _I, _I, _I, _I, _F, _I, _I, _P, _Z, _P]
    lib.da_decode_attn.restype = _I
    lib.da_decode_attn_planned.argtypes = [_P, _P, _P, _P, _P, _P, _I, _I, _I, _I, _I, _F, ctypes.POINTER(DaPlan),
                                           _P, _Z, _P]
    lib.da_decode_attn_planned.restype = _I
    lib.da_decode_attn_noalloc.argtypes = [_P, _P, _P, _P, _P, _P, _I, _I, _I, _I, _I, _F, _I, _I, _P]
    lib.da_decode_attn_noalloc.restype = _I
    lib.da_decode_attn_paged.argtypes = [_P, _P, _P, _P, _P, _P, _P, _I, _I, _I, _I, _I, _I, _I, _I, _F, _I, _I,
                                         _P, _Z, _P]
    lib.da_decode_attn_paged.restype = _I
    lib.da_decode_attn_paged_planned.argtypes = [_P, _P, _P, _P, _P, _P, _P, _I, _I, _I, _I, _I, _I, _I, _I, _F,
                                                 ctypes.POINTER(DaPlan), _P, _Z, _P]
    lib.da_decode_attn_paged_planned.restype = _I
    lib.da_schedule_max_bytes.argtypes = [_I, _I, _I, _I]
    lib.da_schedule_max_bytes.restype = _Z
    lib.da_make_schedule.argtypes = [_P, _I, _I, _I, _I, _I, _I, _I, _I, _I, _P, _Z, ctypes.POINTER(DaSchedule)]
    lib.da_make_schedule.restype = _I
    lib.da_schedule_workspace_bytes.argtypes = [ctypes.POINTER(DaSchedule)]
    lib.da_schedule_workspace_bytes.restype = _Z
    lib.da_decode_attn_scheduled.argtypes = [_P, _P, _P, _P, _P, _P, _I, _I, _I, _P, _P, _I, _F,
                                             ctypes.POINTER(DaSchedule), _P, _P, _Z, _P]
    lib.da_decode_attn_scheduled.restype = _I
    lib.da_split_partials.argtypes = [_P, _P, _P, _P, _P, _P, _P, _I, _I, _I, _I, _I, _F, _I, _I, _P]
    lib.da_split_partials.restype = _I
    lib.da_combine_splits.argtypes = [_P, _P, _P, _P, _P, _I, _I, _I, _I, _P]
    lib.da_combine_splits.restype = _I
    lib.da_device_info.argtypes = [ctypes.POINTER(_I), ctypes.POINTER(_I)]
    lib.da_device_info.restype = _I
    lib.da_strerror.argtypes = [_I]
    lib.da_strerror.restype = ctypes.c_char_p
    lib.da_last_error.argtypes = []
    lib.da_last_error.restype = ctypes.c_char_p
    _lib = lib
    return lib


def _check(rc: int) -> None:
    if rc != DA_OK:
        lib = load()
        msg = (lib.da_last_error() or b"").decode() or lib.da_strerror(rc).decode()
        raise DecodeAttnError(rc, msg)


def da_strerror(code: int) -> str:
    return load().da_strerror(code).decode()


def da_last_error() -> str:
    return (load().da_last_error() or b"").decode()


def da_device_info() -> Tuple[int, bool]:
    cus, is950 = _I(0), _I(0)
    _check(load().da_device_info(ctypes.byref(cus), ctypes.byref(is950)))
    return cus.value, bool(is950.value)


def da_choose_splits(B: int, H_Q: int, H_KV: int, L_K_max: int, d: int = HEAD_DIM, num_cus: int = 0,
                     cu_margin: int = 0, policy: int = POLICY_MI355X) -> DaPlan:
    plan = DaPlan()
    _check(load().da_choose_splits(B, H_Q, H_KV, L_K_max, d, num_cus, cu_margin, policy, ctypes.byref(plan)))
    return plan


def da_model_time(policy: int, B: int, H_Q: int, H_KV: int, L_K: int, heads_per_tile: int, num_splits: int,
                  v_slices: int = 1, combine: int = 0, num_cus: int = 256) -> float:
    """The planner's modelled microseconds per call (-1 for no launch)."""
    return float(load().da_model_time(policy, B, H_Q, H_KV, L_K, heads_per_tile, num_splits, v_slices, combine,
                                      num_cus))


def da_make_plan(B: int, H_Q: int, H_KV: int, L_K_max: int, d: int = HEAD_DIM, num_splits: int = 0,
                 pack_gqa: int = -1, num_cus: int = 0, cu_margin: int = 0, policy: int = POLICY_MI355X) -> DaPlan:
    plan = DaPlan()
    _check(load().da_make_plan(B, H_Q, H_KV, L_K_max, d, num_splits, pack_gqa, num_cus, cu_margin, policy,
                               ctypes.byref(plan)))
    return plan


def da_workspace_bytes(B: int, H_Q: int, d: int, num_splits: int) -> int:
    return int(load().da_workspace_bytes(B, H_Q, d, num_splits))


def da_split_bounds(L: int, num_splits: int) -> List[int]:
    cuts = (ctypes.c_int32 * (num_splits + 1))() if num_splits >= 0 else None
    _check(load().da_split_bounds(L, num_splits, cuts))
    return list(cuts)


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    # an empty tensor has no storage: NULL (the library reads nothing there)
    return None if t is None or t.numel() == 0 else t.data_ptr()


def _stream(dev: torch.device, stream) -> int:
    if stream is None:
        return torch.cuda.current_stream(dev).cuda_stream
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def _shapes(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, cu: Optional[torch.Tensor],
            L_K_max: Optional[int]) -> Tuple[int, int, int, int, int]:
    for name, t in (("q", q), ("k", k), ("v", v)):
        if t.dtype != torch.bfloat16 or not t.is_contiguous() or not t.is_cuda:
            raise ValueError(f"{name} must be a contiguous bfloat16 CUDA tensor")
    if k.shape != v.shape:
        raise ValueError("k and v shapes differ")
    B, H_Q, d = q.shape
    if cu is None:
        if k.dim() != 4 or k.shape[0] != B or k.shape[3] != d:
            raise ValueError("k must be [B, L_K, H_KV, d]")
        L = k.shape[1]
        H_KV = k.shape[2]
        if L_K_max is not None and L_K_max != L:
            raise ValueError("L_K_max must equal k.shape[1] for the fixed layout")
        L_K_max = L
    else:
        if cu.dtype != torch.int32 or not cu.is_contiguous() or cu.numel() != B + 1 or not cu.is_cuda:
            raise ValueError("cu_seqlens_k must be a contiguous int32 CUDA tensor of B+1 entries")
        if k.dim() != 3 or k.shape[2] != d:
            raise ValueError("varlen k must be [sum L_b, H_KV, d]")
        H_KV = k.shape[1]
        if L_K_max is None:
            raise ValueError("L_K_max (the host-known longest sequence) is required with cu_seqlens_k")
    return B, H_Q, H_KV, int(L_K_max), d


_workspaces: Dict[Tuple[int, int], torch.Tensor] = {}
# Workspaces replaced by a larger one.  They are never freed: a HIP graph
# captured earlier keeps their addresses, and kernels queued on a stream
# other than torch's current one may still be using them, so returning them
# to the caching allocator could hand live memory to another tensor.
_retired: List[torch.Tensor] = []


def workspace_for(dev: torch.device, stream_handle: int, nbytes: int) -> torch.Tensor:
    """A workspace of at least nbytes, cached per (device, stream).  Calls on
    one stream run in order, so they can share it.  It is zero-filled when
    allocated: the chunk-state regions need no initialisation (every call
    writes what it reads), and the arrival counters of single-launch plans
    start at zero and are left at zero by every call.  A cache that has to
    grow keeps its old buffer alive for the life of the process."""
    index = dev.index if dev.index is not None else (torch.cuda.current_device() if dev.type == "cuda" else -1)
    key = (index, stream_handle)
    ws = _workspaces.get(key)
    if ws is None or ws.numel() < nbytes:
        if ws is not None:
            _retired.append(ws)
        ws = torch.zeros(max(nbytes, 256), dtype=torch.uint8, device=dev)
        _workspaces[key] = ws
    return ws


def da_decode_attn(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, cu_seqlens_k: Optional[torch.Tensor] = None,
                   out: Optional[torch.Tensor] = None, lse_out: Optional[torch.Tensor] = None, *,
                   L_K_max: Optional[int] = None, softmax_scale: float = 0.0, num_splits: int = 0,
                   pack_gqa: int = -1, workspace: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """O = softmax(scale q K^T) V for one decode step; returns `out`."""
    B, H_Q, H_KV, L, d = _shapes(q, k, v, cu_seqlens_k, L_K_max)
    dev = q.device
    if out is None:
        out = torch.empty((B, H_Q, d), dtype=torch.bfloat16, device=dev)
    s_handle = _stream(dev, stream)
    if workspace is None:
        plan = da_make_plan(B, H_Q, H_KV, L, d, num_splits, pack_gqa)
        nbytes = da_workspace_bytes(B, H_Q, d, plan.num_splits)
        if nbytes:
            workspace = workspace_for(dev, s_handle, nbytes)
    ws_ptr = _ptr(workspace)
    ws_bytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    _check(load().da_decode_attn(_ptr(q), _ptr(k), _ptr(v), _ptr(cu_seqlens_k), _ptr(out), _ptr(lse_out),
                                 B, H_Q, H_KV, L, d, float(softmax_scale), int(num_splits), int(pack_gqa),
                                 ws_ptr, ws_bytes, s_handle))
    return out


def da_decode_attn_planned(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, plan: DaPlan,
                           cu_seqlens_k: Optional[torch.Tensor] = None, out: Optional[torch.Tensor] = None,
                           lse_out: Optional[torch.Tensor] = None, *, L_K_max: Optional[int] = None,
                           softmax_scale: float = 0.0, workspace: Optional[torch.Tensor] = None,
                           stream=None) -> torch.Tensor:
    """da_decode_attn with a plan made beforehand (da_make_plan /
    da_choose_splits, any policy or cu_margin), run exactly as it is."""
    B, H_Q, H_KV, L, d = _shapes(q, k, v, cu_seqlens_k, L_K_max)
    dev = q.device
    if out is None:
        out = torch.empty((B, H_Q, d), dtype=torch.bfloat16, device=dev)
    s_handle = _stream(dev, stream)
    if workspace is None:
        nbytes = da_workspace_bytes(B, H_Q, d, plan.num_splits)
        if nbytes:
            workspace = workspace_for(dev, s_handle, nbytes)
    ws_ptr = _ptr(workspace)
    ws_bytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    _check(load().da_decode_attn_planned(_ptr(q), _ptr(k), _ptr(v), _ptr(cu_seqlens_k), _ptr(out), _ptr(lse_out),
                                         B, H_Q, H_KV, L, d, float(softmax_scale), ctypes.byref(plan),
                                         ws_ptr, ws_bytes, s_handle))
    return out


def da_decode_attn_noalloc(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor,
                           cu_seqlens_k: Optional[torch.Tensor] = None, out: Optional[torch.Tensor] = None,
                           lse_out: Optional[torch.Tensor] = None, *, L_K_max: Optional[int] = None,
                           softmax_scale: float = 0.0, num_splits: int = 0, pack_gqa: int = -1,
                           stream=None) -> torch.Tensor:
    """da_decode_attn with no workspace: the library's fixed per-device
    scratch holds the chunk states.  Pass `out` to make the call allocate
    nothing at all."""
    B, H_Q, H_KV, L, d = _shapes(q, k, v, cu_seqlens_k, L_K_max)
    if out is None:
        out = torch.empty((B, H_Q, d), dtype=torch.bfloat16, device=q.device)
    _check(load().da_decode_attn_noalloc(_ptr(q), _ptr(k), _ptr(v), _ptr(cu_seqlens_k), _ptr(out), _ptr(lse_out),
                                         B, H_Q, H_KV, L, d, float(softmax_scale), int(num_splits), int(pack_gqa),
                                         _stream(q.device, stream)))
    return out


def _paged_args(q, k_cache, v_cache, block_table, seq_lens):
    """Check a paged call's tensors; (B, H_Q, H_KV, d, page_size, max_pages, num_pages)."""
    for name, t in (("q", q), ("k_cache", k_cache), ("v_cache", v_cache)):
        if t.dtype != torch.bfloat16 or not t.is_contiguous() or not t.is_cuda:
            raise ValueError(f"{name} must be a contiguous bfloat16 CUDA tensor")
    for name, t in (("block_table", block_table), ("seq_lens", seq_lens)):
        if t.dtype != torch.int32 or not t.is_contiguous() or not t.is_cuda:
            raise ValueError(f"{name} must be a contiguous int32 CUDA tensor")
    if k_cache.shape != v_cache.shape or k_cache.dim() != 4:
        raise ValueError("k_cache and v_cache must both be [num_pages, page_size, H_KV, d]")
    B, H_Q, d = q.shape
    num_pages, page_size, H_KV, dk = k_cache.shape
    if dk != d or block_table.dim() != 2 or block_table.shape[0] != B or seq_lens.numel() != B:
        raise ValueError("block_table must be [B, max_pages], seq_lens [B], and the head dims must agree")
    return B, H_Q, H_KV, d, page_size, block_table.shape[1], num_pages


def da_decode_attn_paged(q: torch.Tensor, k_cache: torch.Tensor, v_cache: torch.Tensor, block_table: torch.Tensor,
                         seq_lens: torch.Tensor, L_K_max: int, out: Optional[torch.Tensor] = None,
                         lse_out: Optional[torch.Tensor] = None, *, softmax_scale: float = 0.0, num_splits: int = 0,
                         pack_gqa: int = -1, workspace: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """Decode attention over a paged KV cache; returns `out`.
    k_cache, v_cache: [num_pages, page_size, H_KV, d] bf16; block_table: [B, max_pages] int32;
    seq_lens: [B] int32; L_K_max: host-known longest sequence."""
    B, H_Q, H_KV, d, page_size, max_pages, num_pages = _paged_args(q, k_cache, v_cache, block_table, seq_lens)
    dev = q.device
    if out is None:
        out = torch.empty((B, H_Q, d), dtype=torch.bfloat16, device=dev)
    s_handle = _stream(dev, stream)
    if workspace is None:
        plan = da_make_plan(B, H_Q, H_KV, int(L_K_max), d, num_splits, pack_gqa)
        nbytes = da_workspace_bytes(B, H_Q, d, plan.num_splits)
        if nbytes:
            workspace = workspace_for(dev, s_handle, nbytes)
    ws_bytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    _check(load().da_decode_attn_paged(_ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(block_table), _ptr(seq_lens),
                                       _ptr(out), _ptr(lse_out), B, H_Q, H_KV, page_size, max_pages, num_pages,
                                       int(L_K_max), d, float(softmax_scale), int(num_splits), int(pack_gqa),
                                       _ptr(workspace), ws_bytes, s_handle))
    return out


def da_decode_attn_paged_planned(q: torch.Tensor, k_cache: torch.Tensor, v_cache: torch.Tensor,
                                 block_table: torch.Tensor, seq_lens: torch.Tensor, L_K_max: int, plan: DaPlan,
                                 out: Optional[torch.Tensor] = None, lse_out: Optional[torch.Tensor] = None, *,
                                 softmax_scale: float = 0.0, workspace: Optional[torch.Tensor] = None,
                                 stream=None) -> torch.Tensor:
    """da_decode_attn_paged with a plan made beforehand, run exactly as it is."""
    B, H_Q, H_KV, d, page_size, max_pages, num_pages = _paged_args(q, k_cache, v_cache, block_table, seq_lens)
    dev = q.device
    if out is None:
        out = torch.empty((B, H_Q, d), dtype=torch.bfloat16, device=dev)
    s_handle = _stream(dev, stream)
    if workspace is None:
        nbytes = da_workspace_bytes(B, H_Q, d, plan.num_splits)
        if nbytes:
            workspace = workspace_for(dev, s_handle, nbytes)
    ws_bytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    _check(load().da_decode_attn_paged_planned(_ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(block_table),
                                               _ptr(seq_lens), _ptr(out), _ptr(lse_out), B, H_Q, H_KV, page_size,
                                               max_pages, num_pages, int(L_K_max), d, float(softmax_scale),
                                               ctypes.byref(plan), _ptr(workspace), ws_bytes, s_handle))
    return out


def da_schedule_max_bytes(B: int, H_Q: int, H_KV: int, pack_gqa: int = -1) -> int:
    return int(load().da_schedule_max_bytes(B, H_Q, H_KV, pack_gqa))


def da_make_schedule(seq_lens: Sequence[int], H_Q: int, H_KV: int, L_K_max: Optional[int] = None,
                     d: int = HEAD_DIM, pack_gqa: int = -1, num_cus: int = 0, cu_margin: int = 0,
                     chunk_tiles: int = 0) -> Tuple[DaSchedule, torch.Tensor]:
    """Per-sequence schedule from host-known lengths: (DaSchedule, metadata
    bytes as a CPU uint8 tensor to copy to the device)."""
    lens = torch.as_tensor(list(seq_lens) if not isinstance(seq_lens, torch.Tensor) else seq_lens.cpu(),
                           dtype=torch.int32).contiguous()
    B = lens.numel()
    if L_K_max is None:
        L_K_max = int(lens.max()) if B else 0
    cap = da_schedule_max_bytes(B, H_Q, H_KV, pack_gqa)
    meta = torch.zeros(max(cap, 16), dtype=torch.uint8)
    sched = DaSchedule()
    _check(load().da_make_schedule(lens.data_ptr() if B else None, B, H_Q, H_KV, int(L_K_max), d, pack_gqa,
                                   num_cus, cu_margin, chunk_tiles, meta.data_ptr(), meta.numel(),
                                   ctypes.byref(sched)))
    return sched, meta[: sched.meta_bytes].clone()


def da_schedule_workspace_bytes(sched: DaSchedule) -> int:
    return int(load().da_schedule_workspace_bytes(ctypes.byref(sched)))


def da_decode_attn_scheduled(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, sched: DaSchedule,
                             meta_dev: torch.Tensor, cu_seqlens_k: Optional[torch.Tensor] = None,
                             block_table: Optional[torch.Tensor] = None, seq_lens: Optional[torch.Tensor] = None,
                             out: Optional[torch.Tensor] = None, lse_out: Optional[torch.Tensor] = None, *,
                             softmax_scale: float = 0.0, workspace: Optional[torch.Tensor] = None,
                             stream=None) -> torch.Tensor:
    """Decode attention driven by a per-sequence schedule; returns `out`.
    Contiguous K/V (fixed, or varlen with cu_seqlens_k) when block_table is
    None, else paged: k, v [num_pages, page_size, H_KV, d] with block_table
    [B, max_pages] and seq_lens [B]."""
    for name, t in (("q", q), ("k", k), ("v", v)):
        if t.dtype != torch.bfloat16 or not t.is_contiguous() or not t.is_cuda:
            raise ValueError(f"{name} must be a contiguous bfloat16 CUDA tensor")
    if meta_dev.dtype != torch.uint8 or not meta_dev.is_cuda or meta_dev.numel() < sched.meta_bytes:
        raise ValueError("meta_dev must be a CUDA uint8 tensor holding the schedule's metadata")
    B, H_Q, d = q.shape
    if B != sched.B or H_Q != sched.H_Q:
        raise ValueError("q does not match the schedule")
    page_size = max_pages = num_pages = 0
    if block_table is not None:
        for name, t in (("block_table", block_table), ("seq_lens", seq_lens)):
            if t is None or t.dtype != torch.int32 or not t.is_contiguous() or not t.is_cuda:
                raise ValueError(f"{name} must be a contiguous int32 CUDA tensor")
        num_pages, page_size = k.shape[0], k.shape[1]
        max_pages = block_table.shape[1]
    dev = q.device
    if out is None:
        out = torch.empty((B, H_Q, d), dtype=torch.bfloat16, device=dev)
    s_handle = _stream(dev, stream)
    if workspace is None:
        nbytes = da_schedule_workspace_bytes(sched)
        if nbytes:
            workspace = workspace_for(dev, s_handle, nbytes)
    ws_bytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    _check(load().da_decode_attn_scheduled(_ptr(q), _ptr(k), _ptr(v), _ptr(cu_seqlens_k), _ptr(block_table),
                                           _ptr(seq_lens), page_size, max_pages, num_pages, _ptr(out),
                                           _ptr(lse_out), d, float(softmax_scale), ctypes.byref(sched),
                                           _ptr(meta_dev), _ptr(workspace), ws_bytes, s_handle))
    return out


def da_split_partials(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor,
                      cu_seqlens_k: Optional[torch.Tensor] = None, o_part: Optional[torch.Tensor] = None,
                      m_part: Optional[torch.Tensor] = None, l_part: Optional[torch.Tensor] = None, *,
                      num_splits: int, pack_gqa: int, L_K_max: Optional[int] = None,
                      softmax_scale: float = 0.0, stream=None):
    """Per-chunk partial states (o_part [s,B,H_Q,d], m_part, l_part [s,B,H_Q])."""
    B, H_Q, H_KV, L, d = _shapes(q, k, v, cu_seqlens_k, L_K_max)
    dev = q.device
    if o_part is None:
        o_part = torch.empty((num_splits, B, H_Q, d), dtype=torch.float32, device=dev)
    if m_part is None:
        m_part = torch.empty((num_splits, B, H_Q), dtype=torch.float32, device=dev)
    if l_part is None:
        l_part = torch.empty((num_splits, B, H_Q), dtype=torch.float32, device=dev)
    _check(load().da_split_partials(_ptr(q), _ptr(k), _ptr(v), _ptr(cu_seqlens_k), _ptr(o_part), _ptr(m_part),
                                    _ptr(l_part), B, H_Q, H_KV, L, d, float(softmax_scale), int(num_splits),
                                    int(pack_gqa), _stream(dev, stream)))
    return o_part, m_part, l_part


def da_combine_splits(o_part: torch.Tensor, m_part: torch.Tensor, l_part: torch.Tensor,
                      out: Optional[torch.Tensor] = None, lse_out: Optional[torch.Tensor] = None, *,
                      stream=None) -> torch.Tensor:
    """Log-sum-exp merge of partial states; returns `out` (bf16 [B,H_Q,d])."""
    for name, t in (("o_part", o_part), ("m_part", m_part), ("l_part", l_part)):
        if t.dtype != torch.float32 or not t.is_contiguous() or not t.is_cuda:
            raise ValueError(f"{name} must be a contiguous float32 CUDA tensor")
    s, B, H_Q, d = o_part.shape
    if tuple(m_part.shape) != (s, B, H_Q) or tuple(l_part.shape) != (s, B, H_Q):
        raise ValueError("m_part and l_part must be [s, B, H_Q]")
    dev = o_part.device
    if out is None:
        out = torch.empty((B, H_Q, d), dtype=torch.bfloat16, device=dev)
    _check(load().da_combine_splits(_ptr(o_part), _ptr(m_part), _ptr(l_part), _ptr(out), _ptr(lse_out), s, B, H_Q,
                                    d, _stream(dev, stream)))
    return out
