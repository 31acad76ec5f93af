"""Python binding of libcomem_attn.so (ctypes): argument marshalling only.

The functions named like the C entry points pass plain integers (device
pointers, strides, sizes) straight through and raise ``ComemError`` on a
non-OK status. ``DecodeAttention`` is a convenience wrapper that takes torch
tensors, reads their pointers and strides, and owns a zero-filled workspace;
torch is used only for device memory and the current stream. Every step of
the computation runs in the HIP kernels of the library: when the library has
not been built this module raises instead of computing anything else.
"""

from __future__ import annotations

import ctypes
import os
from typing import Optional, Tuple

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libcomem_attn.so")
PROBE_LIB_PATH = os.path.join(PKG, "libcomem_probe.so")

OK, ERR_NULL_POINTER, ERR_INVALID_SHAPE, ERR_UNSUPPORTED, ERR_MISALIGNED = 0, 1, 2, 3, 4
ERR_WORKSPACE_TOO_SMALL, ERR_BAD_HANDLE, ERR_HIP, ERR_NO_DEVICE, ERR_SCRATCH_LIMIT = 5, 6, 7, 8, 9
F32, BF16, FP8_E4M3 = 0, 1, 2
DTYPES = {"f32": F32, "bf16": BF16, "fp8": FP8_E4M3}
VARIANT_AUTO, VARIANT_VALU, VARIANT_MFMA, VARIANT_MFMA_GRID = 0, 1, 2, 3
NO_DEVICE = -1

EXPORTED = (
    "comem_decode_attn_init", "comem_decode_attn_destroy", "comem_status_string",
    "comem_decode_attn_plan_splits", "comem_decode_attn", "comem_decode_attn_paged",
    "comem_kv_append", "comem_kv_append_paged", "comem_append_decode_attn", "comem_append_decode_attn_paged",
    "comem_prefill_attn", "comem_prefill_attn_paged", "comem_decode_attn_device_errors",
    "comem_decode_attn_noalloc",
)
NOALLOC_SCRATCH_BYTES = 32 << 20  # COMEM_NOALLOC_SCRATCH_BYTES
FLAG_DEBUG_CHECKS = 1
DEVICE_ERR_CTX_LEN, DEVICE_ERR_BLOCK_TABLE = 1, 2
PROBE_EXPORTED = ("comem_probe_read", "comem_probe_copy", "comem_probe_read_kv_heads")
COST_EXPORTED = (
    "comem_cost_kv_bytes_per_token", "comem_cost_decode_time", "comem_cost_decode_saving",
    "comem_cost_prefill_time", "comem_cost_net_saving", "comem_cost_max_compression_ratio",
)


class Config(ctypes.Structure):
    _fields_ = [
        ("num_q_heads", ctypes.c_int32),
        ("num_kv_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("dtype", ctypes.c_int32),
        ("scale", ctypes.c_float),
        ("max_batch", ctypes.c_int32),
        ("max_ctx_len", ctypes.c_int64),
        ("chunk_tokens", ctypes.c_int32),
        ("variant", ctypes.c_int32),
        ("k_scale", ctypes.c_float),
        ("v_scale", ctypes.c_float),
        ("flags", ctypes.c_uint32),
    ]


class CostInputs(ctypes.Structure):
    """S (KV bytes per token), W (bytes/s), P (prefill tokens/s), Y (generated tokens)."""

    _fields_ = [
        ("kv_bytes_per_token", ctypes.c_double),
        ("hbm_bytes_per_s", ctypes.c_double),
        ("prefill_tokens_per_s", ctypes.c_double),
        ("generated_tokens", ctypes.c_double),
    ]


class ComemError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: status {status} ({status_string(status)})")


_lib = None


def _hip_runtime_first() -> None:
    """Load torch (and with it the HIP runtime it ships) before the library.

    The library links the system HIP runtime; torch ships its own, and which
    one the process uses depends on what loads first. With the library opened
    first, the library's device queries failed once torch was imported; with
    torch first, everything here runs.
    """
    try:
        import torch  # noqa: F401
    except ImportError:
        pass


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load the built library once; raise if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} not found: build it with `python -m paper_2605_30842_amd.build`")
    _hip_runtime_first()
    lib = ctypes.CDLL(path)
    vp, i32, i64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    lib.comem_decode_attn_init.argtypes = [ctypes.POINTER(Config), ctypes.c_int, ctypes.POINTER(vp),
                                           ctypes.POINTER(sz)]
    lib.comem_decode_attn_init.restype = ctypes.c_int
    lib.comem_decode_attn_destroy.argtypes = [vp]
    lib.comem_decode_attn_destroy.restype = ctypes.c_int
    lib.comem_status_string.argtypes = [ctypes.c_int]
    lib.comem_status_string.restype = ctypes.c_char_p
    lib.comem_decode_attn_plan_splits.argtypes = [vp, i32, i64, sz, ctypes.POINTER(i32), ctypes.POINTER(i32)]
    lib.comem_decode_attn_plan_splits.restype = ctypes.c_int
    lib.comem_decode_attn_device_errors.argtypes = [vp, vp, sz, ctypes.POINTER(ctypes.c_uint32), vp]
    lib.comem_decode_attn_device_errors.restype = ctypes.c_int
    lib.comem_decode_attn.argtypes = [vp, vp, vp, vp, i64, i64, vp, vp, i32, i64, vp, vp, vp, sz, vp]
    lib.comem_decode_attn.restype = ctypes.c_int
    lib.comem_decode_attn_noalloc.argtypes = [vp, vp, vp, vp, i64, i64, vp, vp, i32, i64, vp, vp, vp]
    lib.comem_decode_attn_noalloc.restype = ctypes.c_int
    lib.comem_decode_attn_paged.argtypes = [vp, vp, vp, vp, i64, i64, i64, i32, i64, vp, i32, vp, i32, i64,
                                            vp, vp, vp, sz, vp]
    lib.comem_decode_attn_paged.restype = ctypes.c_int
    lib.comem_kv_append.argtypes = [vp, vp, vp, vp, vp, i64, i64, vp, vp, i32, i64, vp]
    lib.comem_kv_append.restype = ctypes.c_int
    lib.comem_kv_append_paged.argtypes = [vp, vp, vp, vp, vp, i64, i64, i64, i32, i64, vp, i32, vp, i32, i64, vp]
    lib.comem_kv_append_paged.restype = ctypes.c_int
    dp, cp, f64 = ctypes.POINTER(ctypes.c_double), ctypes.POINTER(CostInputs), ctypes.c_double
    lib.comem_cost_kv_bytes_per_token.argtypes = [i32, i32, i32, i32, dp]
    lib.comem_cost_decode_time.argtypes = [cp, f64, dp]
    lib.comem_cost_decode_saving.argtypes = [cp, f64, f64, dp]
    lib.comem_cost_prefill_time.argtypes = [cp, f64, dp]
    lib.comem_cost_net_saving.argtypes = [cp, f64, f64, dp]
    lib.comem_cost_max_compression_ratio.argtypes = [cp, dp]
    for name in COST_EXPORTED:
        getattr(lib, name).restype = ctypes.c_int
    lib.comem_append_decode_attn.argtypes = [vp, vp, vp, vp, vp, vp, i64, i64, vp, vp, i32, i64, vp, vp, vp, sz, vp]
    lib.comem_append_decode_attn.restype = ctypes.c_int
    lib.comem_append_decode_attn_paged.argtypes = [vp, vp, vp, vp, vp, vp, i64, i64, i64, i32, i64, vp, i32, vp,
                                                   i32, i64, vp, vp, vp, sz, vp]
    lib.comem_append_decode_attn_paged.restype = ctypes.c_int
    lib.comem_prefill_attn.argtypes = [vp, vp, vp, vp, i32, vp, vp, i64, i64, vp, vp, i32, i64, vp, vp, vp]
    lib.comem_prefill_attn.restype = ctypes.c_int
    lib.comem_prefill_attn_paged.argtypes = [vp, vp, vp, vp, i32, vp, vp, i64, i64, i64, i32, i64, vp, i32, vp,
                                             i32, i64, vp, vp, vp]
    lib.comem_prefill_attn_paged.restype = ctypes.c_int
    _lib = lib
    return lib


_probe = None


def load_probe_library(path: str = PROBE_LIB_PATH) -> ctypes.CDLL:
    """The measurement kernels (streaming read, copy); raise if not built."""
    global _probe
    if _probe is not None:
        return _probe
    if not os.path.exists(path):
        raise RuntimeError(f"{path} not found: build it with `python -m paper_2605_30842_amd.build`")
    _hip_runtime_first()
    lib = ctypes.CDLL(path)
    vp, sz = ctypes.c_void_p, ctypes.c_size_t
    lib.comem_probe_read.argtypes = [vp, sz, vp, ctypes.c_int, vp]
    lib.comem_probe_read.restype = ctypes.c_int
    lib.comem_probe_copy.argtypes = [vp, vp, sz, ctypes.c_int, vp]
    lib.comem_probe_copy.restype = ctypes.c_int
    i32, i64 = ctypes.c_int32, ctypes.c_int64
    lib.comem_probe_read_kv_heads.argtypes = [vp, vp, i64, i32, i32, i64, i32, vp, vp]
    lib.comem_probe_read_kv_heads.restype = ctypes.c_int
    _probe = lib
    return lib


def comem_probe_read(src, nbytes, sink, blocks, stream) -> None:
    err = load_probe_library().comem_probe_read(src, nbytes, sink, blocks, stream)
    if err != 0:
        raise RuntimeError(f"comem_probe_read: HIP error {err}")


def comem_probe_copy(src, dst, nbytes, blocks, stream) -> None:
    err = load_probe_library().comem_probe_copy(src, dst, nbytes, blocks, stream)
    if err != 0:
        raise RuntimeError(f"comem_probe_copy: HIP error {err}")


def comem_probe_read_kv_heads(k, v, tokens, kv_heads, head_bytes, stride_token, chunk, sink, stream) -> None:
    err = load_probe_library().comem_probe_read_kv_heads(k, v, tokens, kv_heads, head_bytes, stride_token, chunk,
                                                         sink, stream)
    if err != 0:
        raise RuntimeError(f"comem_probe_read_kv_heads: HIP error {err}")


def status_string(status: int) -> str:
    return load_library().comem_status_string(int(status)).decode()


def _check(status: int, where: str) -> None:
    if status != OK:
        raise ComemError(status, where)


# ------------------------------------------------------------ C entry points


def comem_decode_attn_init(cfg: Config, device: int) -> Tuple[int, int]:
    """Create a plan; returns (plan handle, workspace bytes)."""
    plan = ctypes.c_void_p()
    ws = ctypes.c_size_t()
    _check(load_library().comem_decode_attn_init(ctypes.byref(cfg), int(device), ctypes.byref(plan),
                                                 ctypes.byref(ws)), "comem_decode_attn_init")
    return plan.value, ws.value


def comem_decode_attn_destroy(plan: int) -> None:
    _check(load_library().comem_decode_attn_destroy(plan), "comem_decode_attn_destroy")


def comem_decode_attn_device_errors(plan: int, workspace: int, workspace_bytes: int, stream: Optional[int]) -> int:
    """COMEM_DEVICE_ERR_* bits recorded by calls using this workspace since the last read (then cleared)."""
    word = ctypes.c_uint32()
    _check(load_library().comem_decode_attn_device_errors(plan, workspace, workspace_bytes, ctypes.byref(word),
                                                          stream), "comem_decode_attn_device_errors")
    return word.value


def comem_decode_attn_plan_splits(plan: int, batch: int, max_ctx_len: int, workspace_bytes: int) -> Tuple[int, int]:
    chunk, splits = ctypes.c_int32(), ctypes.c_int32()
    _check(load_library().comem_decode_attn_plan_splits(plan, batch, max_ctx_len, workspace_bytes,
                                                        ctypes.byref(chunk), ctypes.byref(splits)),
           "comem_decode_attn_plan_splits")
    return chunk.value, splits.value


def comem_decode_attn(plan, q, k, v, stride_token, stride_head, seq_start, ctx_lens, batch, max_ctx_len,
                      out, lse, workspace, workspace_bytes, stream) -> None:
    _check(load_library().comem_decode_attn(plan, q, k, v, stride_token, stride_head, seq_start, ctx_lens,
                                            batch, max_ctx_len, out, lse, workspace, workspace_bytes, stream),
           "comem_decode_attn")


def comem_decode_attn_noalloc(plan, q, k, v, stride_token, stride_head, seq_start, ctx_lens, batch, max_ctx_len,
                              out, lse, stream) -> None:
    _check(load_library().comem_decode_attn_noalloc(plan, q, k, v, stride_token, stride_head, seq_start, ctx_lens,
                                                    batch, max_ctx_len, out, lse, stream),
           "comem_decode_attn_noalloc")


def comem_decode_attn_paged(plan, q, k_pages, v_pages, stride_page, stride_token, stride_head, page_size,
                            num_pages, block_table, max_pages_per_seq, ctx_lens, batch, max_ctx_len, out, lse,
                            workspace, workspace_bytes, stream) -> None:
    _check(load_library().comem_decode_attn_paged(plan, q, k_pages, v_pages, stride_page, stride_token,
                                                  stride_head, page_size, num_pages, block_table,
                                                  max_pages_per_seq, ctx_lens, batch, max_ctx_len, out, lse,
                                                  workspace, workspace_bytes, stream),
           "comem_decode_attn_paged")


def comem_kv_append(plan, new_k, new_v, k, v, stride_token, stride_head, seq_start, ctx_lens, batch,
                    max_ctx_len, stream) -> None:
    _check(load_library().comem_kv_append(plan, new_k, new_v, k, v, stride_token, stride_head, seq_start,
                                          ctx_lens, batch, max_ctx_len, stream), "comem_kv_append")


def comem_kv_append_paged(plan, new_k, new_v, k_pages, v_pages, stride_page, stride_token, stride_head,
                          page_size, num_pages, block_table, max_pages_per_seq, ctx_lens, batch, max_ctx_len,
                          stream) -> None:
    _check(load_library().comem_kv_append_paged(plan, new_k, new_v, k_pages, v_pages, stride_page, stride_token,
                                                stride_head, page_size, num_pages, block_table, max_pages_per_seq,
                                                ctx_lens, batch, max_ctx_len, stream),
           "comem_kv_append_paged")


def comem_append_decode_attn(plan, q, new_k, new_v, k, v, stride_token, stride_head, seq_start, ctx_lens, batch,
                             max_ctx_len, out, lse, workspace, workspace_bytes, stream) -> None:
    _check(load_library().comem_append_decode_attn(plan, q, new_k, new_v, k, v, stride_token, stride_head,
                                                   seq_start, ctx_lens, batch, max_ctx_len, out, lse, workspace,
                                                   workspace_bytes, stream), "comem_append_decode_attn")


def comem_append_decode_attn_paged(plan, q, new_k, new_v, k_pages, v_pages, stride_page, stride_token, stride_head,
                                   page_size, num_pages, block_table, max_pages_per_seq, ctx_lens, batch,
                                   max_ctx_len, out, lse, workspace, workspace_bytes, stream) -> None:
    _check(load_library().comem_append_decode_attn_paged(plan, q, new_k, new_v, k_pages, v_pages, stride_page,
                                                         stride_token, stride_head, page_size, num_pages,
                                                         block_table, max_pages_per_seq, ctx_lens, batch,
                                                         max_ctx_len, out, lse, workspace, workspace_bytes, stream),
           "comem_append_decode_attn_paged")


def comem_prefill_attn(plan, q, q_start, q_lens, max_q_len, k, v, stride_token, stride_head, seq_start, ctx_lens,
                       batch, max_ctx_len, out, lse, stream) -> None:
    _check(load_library().comem_prefill_attn(plan, q, q_start, q_lens, max_q_len, k, v, stride_token, stride_head,
                                             seq_start, ctx_lens, batch, max_ctx_len, out, lse, stream),
           "comem_prefill_attn")


def comem_prefill_attn_paged(plan, q, q_start, q_lens, max_q_len, k_pages, v_pages, stride_page, stride_token,
                             stride_head, page_size, num_pages, block_table, max_pages_per_seq, ctx_lens, batch,
                             max_ctx_len, out, lse, stream) -> None:
    _check(load_library().comem_prefill_attn_paged(plan, q, q_start, q_lens, max_q_len, k_pages, v_pages,
                                                   stride_page, stride_token, stride_head, page_size, num_pages,
                                                   block_table, max_pages_per_seq, ctx_lens, batch, max_ctx_len,
                                                   out, lse, stream),
           "comem_prefill_attn_paged")


def _cost_call(name, *args) -> float:
    out = ctypes.c_double()
    _check(getattr(load_library(), name)(*args, ctypes.byref(out)), name)
    return out.value


def comem_cost_kv_bytes_per_token(num_layers, num_kv_heads, head_dim, elem_bytes) -> float:
    return _cost_call("comem_cost_kv_bytes_per_token", num_layers, num_kv_heads, head_dim, elem_bytes)


def comem_cost_decode_time(inputs: CostInputs, ctx_tokens) -> float:
    return _cost_call("comem_cost_decode_time", ctypes.byref(inputs), float(ctx_tokens))


def comem_cost_decode_saving(inputs: CostInputs, l_full, l_sum) -> float:
    return _cost_call("comem_cost_decode_saving", ctypes.byref(inputs), float(l_full), float(l_sum))


def comem_cost_prefill_time(inputs: CostInputs, l_sum) -> float:
    return _cost_call("comem_cost_prefill_time", ctypes.byref(inputs), float(l_sum))


def comem_cost_net_saving(inputs: CostInputs, l_full, l_sum) -> float:
    return _cost_call("comem_cost_net_saving", ctypes.byref(inputs), float(l_full), float(l_sum))


def comem_cost_max_compression_ratio(inputs: CostInputs) -> float:
    return _cost_call("comem_cost_max_compression_ratio", ctypes.byref(inputs))


def _torch_dtypes(dtype: str):
    """(query dtypes, cache dtypes) a plan of `dtype` accepts as torch dtypes."""
    import torch

    if dtype == "f32":
        return (torch.float32,), (torch.float32,)
    if dtype == "bf16":
        return (torch.bfloat16,), (torch.bfloat16,)
    fp8 = tuple(t for t in (getattr(torch, "float8_e4m3fn", None),) if t is not None)
    return (torch.bfloat16,), (torch.uint8,) + fp8


def _need(cond: bool, msg: str) -> None:
    if not cond:
        raise ValueError(msg)


def _check_tensor(name, t, dtypes, device, shape=None, ndim=None, contiguous=True):
    """Raise ValueError unless t is a tensor on `device` with one of `dtypes`, the given shape (None entries
    match any size) or rank, and (if asked) contiguous."""
    import torch

    _need(isinstance(t, torch.Tensor), f"{name} must be a torch tensor, got {type(t).__name__}")
    _need(t.device == device, f"{name} is on {t.device}, expected {device}")
    _need(t.dtype in dtypes, f"{name} has dtype {t.dtype}, expected {' or '.join(str(d) for d in dtypes)}")
    if shape is not None:
        _need(t.dim() == len(shape) and all(w is None or w == g for w, g in zip(shape, t.shape)),
              f"{name} has shape {tuple(t.shape)}, expected {tuple('*' if w is None else w for w in shape)}")
    if ndim is not None:
        _need(t.dim() == ndim, f"{name} must have {ndim} dimensions, got {t.dim()}")
    if contiguous:
        _need(t.is_contiguous(), f"{name} must be contiguous")


# ------------------------------------------------------------ torch wrapper


# Placement of V relative to K that the C header recommends
# (COMEM_V_BASE_OFFSET_BYTES modulo COMEM_V_BASE_OFFSET_MODULUS).
V_BASE_OFFSET_BYTES = 256
V_BASE_OFFSET_MODULUS = 512


def kv_cache_pair(shape, dtype, device):
    """Empty K and V caches of `shape` carved from one allocation, with V's base
    at K's base plus V_BASE_OFFSET_BYTES modulo V_BASE_OFFSET_MODULUS (whatever
    the allocation's own alignment). Both are contiguous tensors."""
    import math

    import torch

    esize = torch.empty((), dtype=dtype).element_size()
    n = math.prod(shape)
    nbytes = n * esize
    gap = (V_BASE_OFFSET_BYTES - nbytes) % V_BASE_OFFSET_MODULUS  # bytes between K's end and V's start
    if gap % esize != 0:
        raise ValueError(f"element size {esize} does not divide the placement gap {gap}")
    g = gap // esize
    buf = torch.empty(2 * n + g, dtype=dtype, device=device)
    k = buf[:n].view(shape)
    v = buf[n + g:2 * n + g].view(shape)
    if (v.data_ptr() - k.data_ptr()) % V_BASE_OFFSET_MODULUS != V_BASE_OFFSET_BYTES:
        raise RuntimeError("K/V placement not reached (allocation misaligned)")
    return k, v


class DecodeAttention:
    """A plan plus its workspace, called with torch device tensors.

    q: [B, Hq, D]; contiguous k, v: [T, Hkv, D] (any strides with d
    contiguous); paged k, v: [P, page_size, Hkv, D]. Outputs are float32
    [B, Hq, D] and [B, Hq] (natural-log lse). dtype "fp8": q is bf16, K and V
    are uint8 tensors of OCP FP8 E4M3 codes with per-tensor k_scale, v_scale.
    """

    def __init__(self, num_q_heads: int, num_kv_heads: int, head_dim: int, dtype: str, scale: float,
                 max_batch: int, max_ctx_len: int, chunk_tokens: int = 0, variant: str = "auto",
                 device: int = 0, k_scale: float = 1.0, v_scale: float = 1.0, debug_checks: bool = False):
        import torch

        self.cfg = Config(num_q_heads, num_kv_heads, head_dim, DTYPES[dtype], float(scale),
                          max_batch, max_ctx_len, chunk_tokens,
                          {"auto": VARIANT_AUTO, "valu": VARIANT_VALU, "mfma": VARIANT_MFMA,
                           "mfma_grid": VARIANT_MFMA_GRID}[variant], float(k_scale), float(v_scale),
                          FLAG_DEBUG_CHECKS if debug_checks else 0)
        self.device = device
        self.dtype = dtype
        self.num_q_heads, self.num_kv_heads, self.head_dim = num_q_heads, num_kv_heads, head_dim
        self._torch_device = torch.device("cuda", device)
        self._q_dtypes, self._kv_dtypes = _torch_dtypes(dtype)
        self.plan, self.workspace_bytes = comem_decode_attn_init(self.cfg, device)
        self.workspace = torch.zeros(max(self.workspace_bytes, 256), dtype=torch.uint8, device=f"cuda:{device}")

    def close(self) -> None:
        if self.plan:
            comem_decode_attn_destroy(self.plan)
            self.plan = None

    def __del__(self):
        try:
            self.close()
        except Exception:  # noqa: BLE001 - interpreter shutdown
            pass

    def splits(self, batch: int, max_ctx_len: int) -> Tuple[int, int]:
        return comem_decode_attn_plan_splits(self.plan, batch, max_ctx_len, self.workspace_bytes)

    def device_errors(self, stream=None) -> int:
        """Contract-violation bits (debug_checks=True) since the last read; waits for the stream."""
        return comem_decode_attn_device_errors(self.plan, self.workspace.data_ptr(), self.workspace_bytes,
                                               self._stream(stream))

    # Checks of every tensor against the plan, before any pointer reaches the library.

    def _check_q_out(self, q, out, lse, rows=None):
        Hq, D = self.num_q_heads, self.head_dim
        _check_tensor("q", q, self._q_dtypes, self._torch_device, shape=(rows, Hq, D))
        R = q.shape[0]
        import torch

        if out is not None:
            _check_tensor("out", out, (torch.float32,), self._torch_device, shape=(R, Hq, D))
        if lse is not None:
            _check_tensor("lse", lse, (torch.float32,), self._torch_device, shape=(R, Hq))

    def _check_cache(self, k, v, paged: bool):
        dims = 4 if paged else 3
        for name, t in (("k", k), ("v", v)):
            _check_tensor(name, t, self._kv_dtypes, self._torch_device, ndim=dims, contiguous=False)
            _need(t.shape[-2] == self.num_kv_heads and t.shape[-1] == self.head_dim,
                  f"{name} has shape {tuple(t.shape)}, expected [..., {self.num_kv_heads}, {self.head_dim}]")
            _need(t.stride(-1) == 1, f"{name} must have a contiguous last dimension")
        _need(k.shape == v.shape and k.stride() == v.stride(), "k and v must have the same shape and strides")
        _need(k.dtype == v.dtype, "k and v must have the same dtype")

    def _check_lengths(self, ctx_lens, batch, seq_start=None, block_table=None):
        import torch

        _check_tensor("ctx_lens", ctx_lens, (torch.int32,), self._torch_device, shape=(batch,))
        if seq_start is not None:
            _check_tensor("seq_start", seq_start, (torch.int64,), self._torch_device, shape=(batch,))
        if block_table is not None:
            _check_tensor("block_table", block_table, (torch.int32,), self._torch_device, shape=(batch, None))

    def _check_new_rows(self, new_k, new_v, k, batch):
        for name, t in (("new_k", new_k), ("new_v", new_v)):
            _check_tensor(name, t, (k.dtype,), self._torch_device, shape=(batch, self.num_kv_heads, self.head_dim))

    @staticmethod
    def _check_bound(max_ctx_len, name="max_ctx_len"):
        import numbers

        _need(isinstance(max_ctx_len, numbers.Integral) and not isinstance(max_ctx_len, bool),
              f"{name} must be an integer, got {type(max_ctx_len).__name__}")

    def _outputs(self, q, out, lse):
        import torch

        B, Hq, D = q.shape
        if out is None:
            out = torch.empty((B, Hq, D), dtype=torch.float32, device=q.device)
        return out, lse

    @staticmethod
    def _stream(stream):
        import torch

        return (stream if stream is not None else torch.cuda.current_stream()).cuda_stream

    def forward(self, q, k, v, seq_start, ctx_lens, max_ctx_len: int, out=None, lse=None, stream=None):
        self._check_q_out(q, out, lse)
        self._check_cache(k, v, paged=False)
        self._check_lengths(ctx_lens, q.shape[0], seq_start=seq_start)
        self._check_bound(max_ctx_len)
        out, lse = self._outputs(q, out, lse)
        comem_decode_attn(self.plan, q.data_ptr(), k.data_ptr(), v.data_ptr(), k.stride(0), k.stride(1),
                          seq_start.data_ptr(), ctx_lens.data_ptr(), q.shape[0], int(max_ctx_len),
                          out.data_ptr(), None if lse is None else lse.data_ptr(), self.workspace.data_ptr(),
                          self.workspace_bytes, self._stream(stream))
        return out, lse

    def append(self, new_k, new_v, k, v, seq_start, ctx_lens, max_ctx_len: int, stream=None) -> None:
        """Store new_k/new_v [B, Hkv, D] as token ctx_lens[b] - 1 of each sequence (in place)."""
        self._check_cache(k, v, paged=False)
        self._check_new_rows(new_k, new_v, k, None)
        self._check_lengths(ctx_lens, new_k.shape[0], seq_start=seq_start)
        self._check_bound(max_ctx_len)
        comem_kv_append(self.plan, new_k.data_ptr(), new_v.data_ptr(), k.data_ptr(), v.data_ptr(), k.stride(0),
                        k.stride(1), seq_start.data_ptr(), ctx_lens.data_ptr(), new_k.shape[0], int(max_ctx_len),
                        self._stream(stream))

    def append_paged(self, new_k, new_v, k_pages, v_pages, block_table, ctx_lens, max_ctx_len: int,
                     stream=None) -> None:
        self._check_cache(k_pages, v_pages, paged=True)
        self._check_new_rows(new_k, new_v, k_pages, None)
        self._check_lengths(ctx_lens, new_k.shape[0], block_table=block_table)
        self._check_bound(max_ctx_len)
        comem_kv_append_paged(self.plan, new_k.data_ptr(), new_v.data_ptr(), k_pages.data_ptr(),
                              v_pages.data_ptr(), k_pages.stride(0), k_pages.stride(1), k_pages.stride(2),
                              k_pages.shape[1], k_pages.shape[0], block_table.data_ptr(), block_table.shape[1],
                              ctx_lens.data_ptr(), new_k.shape[0], int(max_ctx_len), self._stream(stream))

    def append_forward(self, q, new_k, new_v, k, v, seq_start, ctx_lens, max_ctx_len: int, out=None, lse=None,
                       stream=None):
        """Store the new rows as token ctx_lens[b] - 1 and attend, in one launch."""
        self._check_q_out(q, out, lse)
        self._check_cache(k, v, paged=False)
        self._check_new_rows(new_k, new_v, k, q.shape[0])
        self._check_lengths(ctx_lens, q.shape[0], seq_start=seq_start)
        self._check_bound(max_ctx_len)
        out, lse = self._outputs(q, out, lse)
        comem_append_decode_attn(self.plan, q.data_ptr(), new_k.data_ptr(), new_v.data_ptr(), k.data_ptr(),
                                 v.data_ptr(), k.stride(0), k.stride(1), seq_start.data_ptr(), ctx_lens.data_ptr(),
                                 q.shape[0], int(max_ctx_len), out.data_ptr(),
                                 None if lse is None else lse.data_ptr(), self.workspace.data_ptr(),
                                 self.workspace_bytes, self._stream(stream))
        return out, lse

    def append_forward_paged(self, q, new_k, new_v, k_pages, v_pages, block_table, ctx_lens, max_ctx_len: int,
                             out=None, lse=None, stream=None):
        self._check_q_out(q, out, lse)
        self._check_cache(k_pages, v_pages, paged=True)
        self._check_new_rows(new_k, new_v, k_pages, q.shape[0])
        self._check_lengths(ctx_lens, q.shape[0], block_table=block_table)
        self._check_bound(max_ctx_len)
        out, lse = self._outputs(q, out, lse)
        comem_append_decode_attn_paged(self.plan, q.data_ptr(), new_k.data_ptr(), new_v.data_ptr(),
                                       k_pages.data_ptr(), v_pages.data_ptr(), k_pages.stride(0), k_pages.stride(1),
                                       k_pages.stride(2), k_pages.shape[1], k_pages.shape[0], block_table.data_ptr(),
                                       block_table.shape[1], ctx_lens.data_ptr(), q.shape[0], int(max_ctx_len),
                                       out.data_ptr(), None if lse is None else lse.data_ptr(),
                                       self.workspace.data_ptr(), self.workspace_bytes, self._stream(stream))
        return out, lse

    def forward_paged(self, q, k_pages, v_pages, block_table, ctx_lens, max_ctx_len: int, out=None, lse=None,
                      stream=None):
        self._check_q_out(q, out, lse)
        self._check_cache(k_pages, v_pages, paged=True)
        self._check_lengths(ctx_lens, q.shape[0], block_table=block_table)
        self._check_bound(max_ctx_len)
        out, lse = self._outputs(q, out, lse)
        comem_decode_attn_paged(self.plan, q.data_ptr(), k_pages.data_ptr(), v_pages.data_ptr(),
                                k_pages.stride(0), k_pages.stride(1), k_pages.stride(2), k_pages.shape[1],
                                k_pages.shape[0], block_table.data_ptr(), block_table.shape[1],
                                ctx_lens.data_ptr(), q.shape[0], int(max_ctx_len), out.data_ptr(),
                                None if lse is None else lse.data_ptr(), self.workspace.data_ptr(),
                                self.workspace_bytes, self._stream(stream))
        return out, lse

    def _check_prefill(self, q, q_start, q_lens, max_q_len, ctx_lens, out, lse, max_ctx_len):
        import torch

        _check_tensor("ctx_lens", ctx_lens, (torch.int32,), self._torch_device, ndim=1)
        batch = ctx_lens.shape[0]
        self._check_q_out(q, out, lse)
        _check_tensor("q_start", q_start, (torch.int64,), self._torch_device, shape=(batch,))
        _check_tensor("q_lens", q_lens, (torch.int32,), self._torch_device, shape=(batch,))
        self._check_bound(max_q_len, "max_q_len")
        self._check_bound(max_ctx_len)

    def _prefill_outputs(self, q, out, lse):
        import torch

        if out is None:
            out = torch.empty(q.shape, dtype=torch.float32, device=q.device)
        return out, lse

    def prefill(self, q, q_start, q_lens, max_q_len: int, k, v, seq_start, ctx_lens, max_ctx_len: int, out=None,
                lse=None, stream=None):
        """Prefill attention of the packed new tokens q [total, Hq, D] over a contiguous cache."""
        self._check_prefill(q, q_start, q_lens, max_q_len, ctx_lens, out, lse, max_ctx_len)
        self._check_cache(k, v, paged=False)
        self._check_lengths(ctx_lens, ctx_lens.shape[0], seq_start=seq_start)
        out, lse = self._prefill_outputs(q, out, lse)
        comem_prefill_attn(self.plan, q.data_ptr(), q_start.data_ptr(), q_lens.data_ptr(), int(max_q_len),
                           k.data_ptr(), v.data_ptr(), k.stride(0), k.stride(1), seq_start.data_ptr(),
                           ctx_lens.data_ptr(), ctx_lens.shape[0], int(max_ctx_len), out.data_ptr(),
                           None if lse is None else lse.data_ptr(), self._stream(stream))
        return out, lse

    def prefill_paged(self, q, q_start, q_lens, max_q_len: int, k_pages, v_pages, block_table, ctx_lens,
                      max_ctx_len: int, out=None, lse=None, stream=None):
        self._check_prefill(q, q_start, q_lens, max_q_len, ctx_lens, out, lse, max_ctx_len)
        self._check_cache(k_pages, v_pages, paged=True)
        self._check_lengths(ctx_lens, ctx_lens.shape[0], block_table=block_table)
        out, lse = self._prefill_outputs(q, out, lse)
        comem_prefill_attn_paged(self.plan, q.data_ptr(), q_start.data_ptr(), q_lens.data_ptr(), int(max_q_len),
                                 k_pages.data_ptr(), v_pages.data_ptr(), k_pages.stride(0), k_pages.stride(1),
                                 k_pages.stride(2), k_pages.shape[1], k_pages.shape[0], block_table.data_ptr(),
                                 block_table.shape[1], ctx_lens.data_ptr(), ctx_lens.shape[0], int(max_ctx_len),
                                 out.data_ptr(), None if lse is None else lse.data_ptr(), self._stream(stream))
        return out, lse
