"""Thin Python binding of ``libkvattn.so`` (argument marshalling only).

Every computation runs in the HIP library; this module passes device
pointers, sizes and the current HIP stream through ``ctypes``. PyTorch is
used for device memory (outputs, workspaces) and streams. If the library has
not been built the functions raise: there is no fallback path.
"""
from __future__ import annotations

import ctypes
import math
import os
import re
from typing import Optional

import numpy as np
import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libkvattn.so")
HEADER = os.path.join(os.path.dirname(HERE), "include", "kvattn.h")
PROBES_HEADER = os.path.join(os.path.dirname(HERE), "include", "kvattn_probes.h")

KV_OK, KV_ERR_INVALID, KV_ERR_UNSUPPORTED, KV_ERR_HIP, KV_ERR_OOM, KV_ERR_STATE = 0, -1, -2, -3, -4, -5
KV_F32, KV_BF16 = 0, 1
_STATUS = {0: "KV_OK", -1: "KV_ERR_INVALID", -2: "KV_ERR_UNSUPPORTED", -3: "KV_ERR_HIP",
           -4: "KV_ERR_OOM", -5: "KV_ERR_STATE"}

_lib = None

POOL_STEPS = ("commit_create_ms", "commit_copy_ms", "commit_map_ms", "commit_access_ms",
              "commit_release_ms", "decommit_sync_ms", "decommit_create_ms",
              "decommit_copy_ms", "decommit_unmap_ms", "decommit_map_ms",
              "decommit_access_ms", "decommit_release_ms")


class KvPoolSteps(ctypes.Structure):
    """``kvpool_steps``: host ms of each step of a pool's last commit and decommit."""
    _fields_ = [(n, ctypes.c_double) for n in POOL_STEPS]


class KvAttnError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{_STATUS.get(code, code)}: {msg}")
        self.code = code


def _c(fn, restype, *argtypes):
    fn.restype = restype
    fn.argtypes = list(argtypes)
    return fn


def lib() -> ctypes.CDLL:
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                           "`python -m paper_2608_23658_amd.build`")
    L = ctypes.CDLL(LIB_PATH)
    vp, i32, sz, f32, dp = (ctypes.c_void_p, ctypes.c_int, ctypes.c_size_t, ctypes.c_float,
                            ctypes.POINTER(ctypes.c_double))
    _c(L.kv_last_error, ctypes.c_char_p)
    _c(L.kvattn_abi_version, i32)
    _c(L.kvattn_decode_workspace_bytes, sz, i32, i32, i32, i32)
    _c(L.kvattn_decode_split_tokens, i32, i32)
    _c(L.kvattn_decode, i32, vp, vp, i32, vp, vp, vp, i32, i32, i32, i32, i32, i32, i32, f32,
       i32, vp, sz, vp)
    _c(L.kvattn_decode_noalloc_max_scratch_bytes, sz)
    _c(L.kvattn_decode_noalloc, i32, vp, vp, i32, vp, vp, vp, i32, i32, i32, i32, i32, i32, i32,
       f32, i32, vp)
    _c(L.kvattn_decode_two_tensor, i32, vp, vp, i32, vp, i32, vp, vp, vp, i32, i32, i32, i32,
       i32, i32, i32, f32, i32, vp, sz, vp)
    _c(L.kvattn_prefill_workspace_bytes, sz, i32, i32, i32, i32)
    _c(L.kvattn_prefill_chunk, i32, vp, vp, i32, vp, vp, vp, vp, i32, i32, i32, i32, i32, i32,
       i32, i32, i32, f32, i32, vp, sz, vp)
    _c(L.kvattn_kv_append, i32, vp, vp, vp, vp, i32, i32, i32, i32, i32, i32, vp)
    _c(L.kvpool_granularity, i32, i32, ctypes.POINTER(ctypes.c_size_t))
    _c(L.kvpool_create, i32, i32, i32, sz, sz, ctypes.POINTER(vp))
    _c(L.kvpool_layer_ptr, i32, vp, i32, ctypes.POINTER(vp))
    _c(L.kvpool_is_committed, i32, vp)
    _c(L.kvpool_commit_elastic, i32, vp, dp)
    _c(L.kvpool_decommit_elastic, i32, vp, dp)
    _c(L.kvpool_sizes, i32, vp, ctypes.POINTER(i32), ctypes.POINTER(ctypes.c_size_t),
       ctypes.POINTER(ctypes.c_size_t))
    _c(L.kvpool_last_toggle_breakdown, i32, vp, dp, dp, dp, dp, dp)
    _c(L.kvpool_destroy, None, vp)
    _c(L.kvpool_commit_whole, i32, vp, dp)
    _c(L.kvpool_last_toggle_steps, i32, vp, ctypes.POINTER(KvPoolSteps))
    _c(L.kvpool_time_single_handle, i32, i32, sz, dp, dp, dp, dp)
    ip = ctypes.POINTER(ctypes.c_int32)
    _c(L.kvblocks_create, i32, i32, i32, ctypes.POINTER(vp))
    _c(L.kvblocks_destroy, None, vp)
    _c(L.kvblocks_set_elastic, i32, vp, i32)
    _c(L.kvblocks_is_admitted, i32, vp)
    _c(L.kvblocks_alloc, i32, vp, i32, ip)
    _c(L.kvblocks_free, i32, vp, i32, ip)
    _c(L.kvblocks_num_free, i32, vp)
    _c(L.kvblocks_num_admitted, i32, vp)
    _c(L.kvblocks_live_elastic, i32, vp)
    _c(L.kvblocks_plan_drain, i32, vp, i32, ip, ip, ctypes.POINTER(i32))
    _c(L.kvattn_copy_blocks, i32, ctypes.POINTER(vp), i32, i32, sz, vp, vp, i32, vp)
    _c(L.kvctl_create, i32, vp, vp, i32, ctypes.POINTER(vp))
    _c(L.kvctl_destroy, None, vp)
    _c(L.kvctl_before_step, i32, vp, i32, ctypes.POINTER(i32), dp)
    _c(L.kvctl_would_commit, i32, vp, i32)
    _c(L.kvctl_is_committed, i32, vp)
    _c(L.kvctl_counts, i32, vp, ctypes.POINTER(i32), ctypes.POINTER(i32))
    _c(L.kvattn_trace_begin, i32, ctypes.POINTER(vp), i32)
    _c(L.kvattn_trace_end, i32, ctypes.POINTER(i32))
    _c(L.kvattn_trace_kernel_name, ctypes.c_char_p, i32)
    _c(L.kvattn_probe_mfma_threads, i32)
    _c(L.kvattn_probe_mfma, i32, vp, vp, i32, i32, vp)
    _c(L.kvattn_probe_read_blocks_waves, i32, i32, i32, i32)
    _c(L.kvattn_probe_read_blocks, i32, vp, i32, vp, vp, i32, i32, i32, i32, i32, i32, vp, vp)
    _lib = L
    return L


def declared_symbols() -> list:
    """Function names declared in include/kvattn.h and include/kvattn_probes.h."""
    names = set()
    for path in (HEADER, PROBES_HEADER):
        text = re.sub(r"/\*.*?\*/", "", open(path).read(), flags=re.S)
        names.update(re.findall(r"\b(kv\w+)\s*\(", text))
    return sorted(names)


def last_error() -> str:
    return lib().kv_last_error().decode()


def check(rc: int) -> None:
    if rc != KV_OK:
        raise KvAttnError(rc, last_error())


def _dtype_code(t: torch.dtype) -> int:
    if t == torch.bfloat16:
        return KV_BF16
    if t == torch.float32:
        return KV_F32
    raise ValueError(f"unsupported dtype {t}")


def _ptr(x) -> int:
    if x is None:
        return 0
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _stream(stream) -> int:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _require_cuda(*ts):
    """Tensors reach the library as bare pointers, so they must be contiguous
    (checked first, which also runs without a GPU) and on the GPU."""
    for t in ts:
        if isinstance(t, torch.Tensor) and not t.is_contiguous():
            raise ValueError("tensors must be contiguous")
    for t in ts:
        if isinstance(t, torch.Tensor) and not t.is_cuda:
            raise ValueError("tensors must be on the GPU")


def _require_int32(**named):
    for name, t in named.items():
        if t.dtype != torch.int32:
            raise ValueError(f"{name} must be int32, not {t.dtype}")
    bt = named.get("block_table")
    if bt is not None and bt.dim() != 2:
        raise ValueError("block_table must be [num_seqs, max_blocks_per_seq]")


def _require_rows(num_seqs: int, block_table, seq_lens, cu_seqlens_q=None):
    """The per-sequence tensors reach the kernels as bare pointers: their
    lengths must match the batch, or the kernels would read past them."""
    if tuple(seq_lens.shape) != (num_seqs,):
        raise ValueError(f"seq_lens must be [{num_seqs}], not {tuple(seq_lens.shape)}")
    if block_table.shape[0] != num_seqs:
        raise ValueError(f"block_table must have {num_seqs} rows, not {block_table.shape[0]}")
    if cu_seqlens_q is not None and tuple(cu_seqlens_q.shape) != (num_seqs + 1,):
        raise ValueError(f"cu_seqlens_q must be [{num_seqs + 1}], "
                         f"not {tuple(cu_seqlens_q.shape)}")


def _require_out(out, q):
    if out is not None and (out.dtype != q.dtype or out.shape != q.shape):
        raise ValueError("out must have q's shape and dtype")


def decode_workspace_bytes(num_seqs: int, num_q_heads: int, head_dim: int, max_seq_len: int) -> int:
    return int(lib().kvattn_decode_workspace_bytes(num_seqs, num_q_heads, head_dim, max_seq_len))


def decode_split_tokens(max_seq_len: int) -> int:
    return int(lib().kvattn_decode_split_tokens(max_seq_len))


def decode_two_tensor(q: torch.Tensor, kv_base, num_base: int, kv_elastic, num_elastic: int,
                      block_table: torch.Tensor, seq_lens: torch.Tensor, *, num_kv_heads: int,
                      max_seq_len: int, block_size: int = 16, scale: Optional[float] = None,
                      out: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None,
                      stream=None) -> torch.Tensor:
    """Decode over a layer split into two tensors (ids >= num_base in the second)."""
    B, Hq, d = q.shape
    _require_int32(block_table=block_table, seq_lens=seq_lens)
    _require_rows(B, block_table, seq_lens)
    _require_out(out, q)
    _require_cuda(q, kv_base, kv_elastic, block_table, seq_lens, out, ws)
    if out is None:
        out = torch.empty_like(q)
    if ws is None:
        ws = workspace(decode_workspace_bytes(B, Hq, d, max_seq_len), q.device)
    scale = 1.0 / math.sqrt(d) if scale is None else scale
    rc = lib().kvattn_decode_two_tensor(_ptr(q), _ptr(kv_base), int(num_base), _ptr(kv_elastic),
                                        int(num_elastic), _ptr(block_table), _ptr(seq_lens),
                                        _ptr(out), B, Hq, int(num_kv_heads), d, int(block_size),
                                        int(block_table.shape[1]), int(max_seq_len),
                                        float(scale), _dtype_code(q.dtype), _ptr(ws),
                                        ws.numel(), _stream(stream))
    check(rc)
    return out


def prefill_workspace_bytes(num_seqs: int, total_q_tokens: int, num_q_heads: int,
                            head_dim: int) -> int:
    return int(lib().kvattn_prefill_workspace_bytes(num_seqs, total_q_tokens, num_q_heads,
                                                    head_dim))


def workspace(nbytes: int, device=None) -> torch.Tensor:
    return torch.empty(max(int(nbytes), 256), dtype=torch.uint8,
                       device=device if device is not None else "cuda")


def decode(q: torch.Tensor, kv_layer, num_blocks: int, block_table: torch.Tensor,
           seq_lens: torch.Tensor, *, num_kv_heads: int, max_seq_len: int,
           block_size: int = 16, scale: Optional[float] = None,
           out: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None,
           stream=None) -> torch.Tensor:
    """Paged decode: ``q`` [B, Hq, d] -> out [B, Hq, d] (same dtype).

    ``kv_layer`` is a tensor or a device address of the layer base.
    """
    B, Hq, d = q.shape
    _require_int32(block_table=block_table, seq_lens=seq_lens)
    _require_rows(B, block_table, seq_lens)
    _require_out(out, q)
    _require_cuda(q, kv_layer, block_table, seq_lens, out, ws)
    if out is None:
        out = torch.empty_like(q)
    if ws is None:
        ws = workspace(decode_workspace_bytes(B, Hq, d, max_seq_len), q.device)
    scale = 1.0 / math.sqrt(d) if scale is None else scale
    rc = lib().kvattn_decode(_ptr(q), _ptr(kv_layer), int(num_blocks), _ptr(block_table),
                             _ptr(seq_lens), _ptr(out), B, Hq, int(num_kv_heads), d,
                             int(block_size), int(block_table.shape[1]), int(max_seq_len),
                             float(scale), _dtype_code(q.dtype), _ptr(ws), ws.numel(),
                             _stream(stream))
    check(rc)
    return out


def decode_noalloc_max_scratch_bytes() -> int:
    return int(lib().kvattn_decode_noalloc_max_scratch_bytes())


def decode_noalloc(q: torch.Tensor, kv_layer, num_blocks: int, block_table: torch.Tensor,
                   seq_lens: torch.Tensor, out: torch.Tensor, *, num_kv_heads: int,
                   max_seq_len: int, block_size: int = 16, scale: Optional[float] = None,
                   stream=None) -> torch.Tensor:
    """Paged decode through ``kvattn_decode_noalloc``: no workspace, and the
    caller passes ``out`` so that nothing is allocated by the call."""
    B, Hq, d = q.shape
    _require_int32(block_table=block_table, seq_lens=seq_lens)
    _require_rows(B, block_table, seq_lens)
    if out is None:
        raise ValueError("decode_noalloc needs a caller-provided out")
    _require_out(out, q)
    _require_cuda(q, kv_layer, block_table, seq_lens, out)
    scale = 1.0 / math.sqrt(d) if scale is None else scale
    rc = lib().kvattn_decode_noalloc(_ptr(q), _ptr(kv_layer), int(num_blocks), _ptr(block_table),
                                     _ptr(seq_lens), _ptr(out), B, Hq, int(num_kv_heads), d,
                                     int(block_size), int(block_table.shape[1]),
                                     int(max_seq_len), float(scale), _dtype_code(q.dtype),
                                     _stream(stream))
    check(rc)
    return out


def prefill_chunk(q: torch.Tensor, kv_layer, num_blocks: int, block_table: torch.Tensor,
                  seq_lens: torch.Tensor, cu_seqlens_q: torch.Tensor, *, num_kv_heads: int,
                  max_seq_len: int, max_num_batched_tokens: Optional[int] = None,
                  block_size: int = 16, scale: Optional[float] = None,
                  out: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None,
                  stream=None) -> torch.Tensor:
    """Chunked prefill: ``q`` [T, Hq, d] bf16, chunks given by ``cu_seqlens_q``."""
    T, Hq, d = q.shape
    _require_int32(block_table=block_table, seq_lens=seq_lens, cu_seqlens_q=cu_seqlens_q)
    B = int(seq_lens.shape[0])
    _require_rows(B, block_table, seq_lens, cu_seqlens_q)
    _require_out(out, q)
    _require_cuda(q, kv_layer, block_table, seq_lens, cu_seqlens_q, out, ws)
    if out is None:
        out = torch.empty_like(q)
    if ws is None:
        ws = workspace(prefill_workspace_bytes(B, T, Hq, d), q.device)
    scale = 1.0 / math.sqrt(d) if scale is None else scale
    budget = T if max_num_batched_tokens is None else int(max_num_batched_tokens)
    rc = lib().kvattn_prefill_chunk(_ptr(q), _ptr(kv_layer), int(num_blocks), _ptr(block_table),
                                    _ptr(seq_lens), _ptr(cu_seqlens_q), _ptr(out), B, T, budget,
                                    Hq, int(num_kv_heads), d, int(block_size),
                                    int(block_table.shape[1]), int(max_seq_len), float(scale),
                                    _dtype_code(q.dtype), _ptr(ws), ws.numel(), _stream(stream))
    check(rc)
    return out


def kv_append(k_new: torch.Tensor, v_new: torch.Tensor, slot_mapping: torch.Tensor, kv_layer,
              num_blocks: int, *, block_size: int = 16, stream=None) -> None:
    """Write ``k_new``/``v_new`` [T, Hkv, d] into the layer's slots ``slot_mapping`` [T] int32."""
    T, Hkv, d = k_new.shape
    if v_new.shape != k_new.shape or v_new.dtype != k_new.dtype:
        raise ValueError("k_new and v_new must have the same shape and dtype")
    if slot_mapping.dtype != torch.int32 or tuple(slot_mapping.shape) != (T,):
        raise ValueError("slot_mapping must be int32 [num_tokens]")
    _require_cuda(k_new, v_new, slot_mapping, kv_layer)
    rc = lib().kvattn_kv_append(_ptr(k_new), _ptr(v_new), _ptr(slot_mapping), _ptr(kv_layer),
                                int(num_blocks), T, Hkv, d, int(block_size),
                                _dtype_code(k_new.dtype), _stream(stream))
    check(rc)


class KernelTrace:
    """Per-kernel HIP-event timing of the library's launches on this thread.

    ``with KernelTrace(n) as tr: ...`` then ``tr.durations()`` gives a list of
    (kernel name, milliseconds) for the traced launches."""

    def __init__(self, max_kernels: int):
        self.events = [torch.cuda.Event(enable_timing=True) for _ in range(2 * max_kernels)]
        for e in self.events:
            e.record()          # materialise the underlying hipEvent_t
        torch.cuda.synchronize()
        self._arr = (ctypes.c_void_p * len(self.events))(*[e.cuda_event for e in self.events])
        self.used = 0
        self.names = []

    def __enter__(self):
        check(lib().kvattn_trace_begin(self._arr, len(self.events)))
        return self

    def __exit__(self, *exc):
        n = ctypes.c_int()
        check(lib().kvattn_trace_end(ctypes.byref(n)))
        self.used = n.value
        self.names = [lib().kvattn_trace_kernel_name(i).decode() for i in range(self.used // 2)]
        return False

    def durations(self):
        torch.cuda.synchronize()
        return [(self.names[i], self.events[2 * i].elapsed_time(self.events[2 * i + 1]))
                for i in range(self.used // 2)]


class _DeviceBytes:
    """A raw device range exposed to torch through __cuda_array_interface__."""

    def __init__(self, ptr: int, nbytes: int):
        self.__cuda_array_interface__ = {"shape": (int(nbytes),), "typestr": "|u1",
                                         "data": (int(ptr), False), "version": 3,
                                         "strides": None}


def device_view(ptr: int, nbytes: int, dtype: torch.dtype = torch.uint8,
                device: int = 0) -> torch.Tensor:
    """A torch tensor over ``nbytes`` of device memory at ``ptr`` (no copy).
    The memory stays owned by whoever allocated it."""
    with torch.cuda.device(device):
        t = torch.as_tensor(_DeviceBytes(ptr, nbytes), device=f"cuda:{device}")
    return t.view(dtype)


class ElasticPool:
    """Per-layer KV ranges of base + elastic bytes (kvpool_* in the C ABI)."""

    def __init__(self, num_layers: int, base_bytes: int, elastic_bytes: int, device: int = 0):
        L = lib()
        h = ctypes.c_void_p()
        check(L.kvpool_create(device, num_layers, base_bytes, elastic_bytes, ctypes.byref(h)))
        self._h = h
        self.device = device
        self.num_layers = num_layers
        self.base_bytes = base_bytes
        self.elastic_bytes = elastic_bytes

    @staticmethod
    def granularity(device: int = 0) -> int:
        g = ctypes.c_size_t()
        check(lib().kvpool_granularity(device, ctypes.byref(g)))
        return int(g.value)

    def layer_ptr(self, layer: int) -> int:
        p = ctypes.c_void_p()
        check(lib().kvpool_layer_ptr(self._h, layer, ctypes.byref(p)))
        return int(p.value)

    def layer_view(self, layer: int, committed_part: bool = True,
                   dtype: torch.dtype = torch.uint8) -> torch.Tensor:
        """torch view of a layer: base only, or base + elastic (must be committed)."""
        n = self.base_bytes + (self.elastic_bytes if committed_part else 0)
        if committed_part and self.elastic_bytes and not self.is_committed:
            raise KvAttnError(KV_ERR_STATE, "elastic range is not committed")
        return device_view(self.layer_ptr(layer), n, dtype, self.device)

    @property
    def is_committed(self) -> bool:
        rc = lib().kvpool_is_committed(self._h)
        if rc < 0:
            check(rc)
        return rc == 1

    def commit(self, empty_cache: bool = True) -> float:
        """Commit the elastic sub-ranges; returns host wall ms of the commit call.
        The torch caching allocator is emptied first so memory it holds from
        earlier work is free for the physical handles."""
        if empty_cache:
            torch.cuda.empty_cache()
        ms = ctypes.c_double()
        check(lib().kvpool_commit_elastic(self._h, ctypes.byref(ms)))
        return ms.value

    def decommit(self) -> float:
        ms = ctypes.c_double()
        check(lib().kvpool_decommit_elastic(self._h, ctypes.byref(ms)))
        return ms.value

    def last_breakdown(self) -> dict:
        v = [ctypes.c_double() for _ in range(5)]
        check(lib().kvpool_last_toggle_breakdown(self._h, *[ctypes.byref(x) for x in v]))
        return dict(zip(["create_ms", "map_ms", "access_ms", "sync_ms", "unmap_ms"],
                        [x.value for x in v]))

    def commit_whole(self, empty_cache: bool = True) -> float:
        """The naive toggle: one whole handle per layer over base + elastic,
        base contents copied in; returns host wall ms."""
        if empty_cache:
            torch.cuda.empty_cache()
        ms = ctypes.c_double()
        check(lib().kvpool_commit_whole(self._h, ctypes.byref(ms)))
        return ms.value

    def last_steps(self) -> dict:
        st = KvPoolSteps()
        check(lib().kvpool_last_toggle_steps(self._h, ctypes.byref(st)))
        return {n: getattr(st, n) for n in POOL_STEPS}

    @staticmethod
    def time_single_handle(nbytes: int, device: int = 0) -> dict:
        """Create + map + access + release of one handle of nbytes (host ms)."""
        v = [ctypes.c_double() for _ in range(4)]
        check(lib().kvpool_time_single_handle(device, int(nbytes), *[ctypes.byref(x) for x in v]))
        return dict(zip(["create_ms", "map_ms", "access_ms", "release_ms"], [x.value for x in v]))

    def close(self) -> None:
        if self._h is not None and self._h.value:
            lib().kvpool_destroy(self._h)
        self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def _ids(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.int32))


def _iptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))


class BlockPool:
    """Block-id allocator with the elastic gate (kvblocks_* in the C ABI)."""

    def __init__(self, num_base: int, num_elastic: int):
        h = ctypes.c_void_p()
        check(lib().kvblocks_create(int(num_base), int(num_elastic), ctypes.byref(h)))
        self._h = h
        self.num_base = int(num_base)
        self.num_elastic = int(num_elastic)

    def alloc(self, n: int) -> np.ndarray:
        out = np.empty(int(n), dtype=np.int32)
        check(lib().kvblocks_alloc(self._h, int(n), _iptr(out)))
        return out

    def free(self, ids) -> None:
        a = _ids(ids)
        check(lib().kvblocks_free(self._h, a.size, _iptr(a)))

    def set_elastic(self, admit: bool) -> None:
        check(lib().kvblocks_set_elastic(self._h, int(bool(admit))))

    @property
    def admitted(self) -> bool:
        return self._int(lib().kvblocks_is_admitted(self._h)) == 1

    @property
    def num_free(self) -> int:
        return self._int(lib().kvblocks_num_free(self._h))

    @property
    def num_admitted(self) -> int:
        return self._int(lib().kvblocks_num_admitted(self._h))

    @property
    def live_elastic(self) -> int:
        return self._int(lib().kvblocks_live_elastic(self._h))

    def plan_drain(self):
        """(from, to) int32 arrays: each live elastic id and the base id it moves to."""
        cap = self.live_elastic
        f = np.empty(max(cap, 1), dtype=np.int32)
        t = np.empty(max(cap, 1), dtype=np.int32)
        n = ctypes.c_int()
        check(lib().kvblocks_plan_drain(self._h, cap, _iptr(f), _iptr(t), ctypes.byref(n)))
        return f[:n.value].copy(), t[:n.value].copy()

    @staticmethod
    def _int(rc: int) -> int:
        if rc < 0:
            check(rc)
        return rc

    def close(self) -> None:
        if self._h is not None and self._h.value:
            lib().kvblocks_destroy(self._h)
        self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def copy_blocks(layers, num_blocks: int, block_bytes: int, src: torch.Tensor, dst: torch.Tensor,
                stream=None) -> None:
    """Copy blocks src[i] -> dst[i] (device int32) in every layer (device pointers)."""
    _require_cuda(src, dst, *layers)
    if src.dtype != torch.int32 or dst.dtype != torch.int32 or src.shape != dst.shape:
        raise ValueError("src and dst must be int32 tensors of one shape")
    ptrs = (ctypes.c_void_p * len(layers))(*[_ptr(x) for x in layers])
    check(lib().kvattn_copy_blocks(ptrs, len(layers), int(num_blocks), int(block_bytes),
                                   _ptr(src), _ptr(dst), int(src.numel()), _stream(stream)))


KVCTL_NONE, KVCTL_COMMIT, KVCTL_DECOMMIT = 0, 1, 2


class Controller:
    """One-step-ahead commit/decommit controller (kvctl_* in the C ABI).

    ``pool`` may be None: the state machine runs without a device."""

    def __init__(self, pool: Optional["ElasticPool"], blocks: BlockPool, hysteresis: int):
        h = ctypes.c_void_p()
        check(lib().kvctl_create(pool._h if pool is not None else None, blocks._h,
                                 int(hysteresis), ctypes.byref(h)))
        self._h = h
        self.pool = pool
        self.blocks = blocks

    def before_step(self, next_has_prefill: bool):
        """Returns (action, host ms). Empties torch's cache first when the call
        is about to commit, so memory it holds is free for the elastic handles."""
        if self.pool is not None and lib().kvctl_would_commit(self._h, int(bool(next_has_prefill))):
            torch.cuda.empty_cache()
        act = ctypes.c_int()
        ms = ctypes.c_double()
        check(lib().kvctl_before_step(self._h, int(bool(next_has_prefill)), ctypes.byref(act),
                                      ctypes.byref(ms)))
        return act.value, ms.value

    @property
    def committed(self) -> bool:
        rc = lib().kvctl_is_committed(self._h)
        if rc < 0:
            check(rc)
        return rc == 1

    def counts(self):
        c, d = ctypes.c_int(), ctypes.c_int()
        check(lib().kvctl_counts(self._h, ctypes.byref(c), ctypes.byref(d)))
        return c.value, d.value

    def close(self) -> None:
        if self._h is not None and self._h.value:
            lib().kvctl_destroy(self._h)
        self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


# ---------------------------------------------------------------------------
# Rate probes (include/kvattn_probes.h): what the chip sustains for the
# resource each kernel is bound by, in that kernel's launch shape.

def probe_mfma_flops(num_workgroups: int, iters: int) -> int:
    """FLOP of one probe_mfma call: 8 wavefronts x 8 * iters matrix
    instructions of 32 x 32 x 16 (32768 FLOP) per workgroup."""
    return num_workgroups * 8 * 8 * iters * 32768


def probe_mfma(num_workgroups: int, iters: int, out: Optional[torch.Tensor] = None,
               clocks: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """Run the matrix-unit probe; returns each thread's accumulator sum. With
    ``clocks`` (int64 [num_workgroups * 8 * 4]) each wavefront also records
    its shader-clock and real-time counters around its loop."""
    n = num_workgroups * int(lib().kvattn_probe_mfma_threads())
    if out is None:
        out = torch.empty(n, dtype=torch.float32, device="cuda")
    if out.dtype != torch.float32 or out.numel() < n:
        raise ValueError(f"out must hold {n} float32")
    if clocks is not None and (clocks.dtype != torch.int64 or
                               clocks.numel() < num_workgroups * 8 * 4):
        raise ValueError(f"clocks must hold {num_workgroups * 8 * 4} int64")
    _require_cuda(out, clocks)
    check(lib().kvattn_probe_mfma(_ptr(out), _ptr(clocks), int(num_workgroups), int(iters),
                                  _stream(stream)))
    return out


def probe_mfma_clock(clocks: torch.Tensor, iters: int, tflops: Optional[float] = None) -> dict:
    """From the counters ``probe_mfma`` recorded: the matrix pipes' busy
    fraction over each wavefront's loop in shader-clock cycles (two
    wavefronts per SIMD, 32 cycles per instruction), and the shader clock
    against the real-time counter taken at 100 MHz. With ``tflops`` (the
    probe's measured rate) also the clock that rate implies at that busy
    fraction, 256 CUs x 4096 FLOP per cycle; the real-time counter's rate
    has disagreed with it by up to 15% on some boxes, so the implied clock is
    the one to use."""
    c = clocks.view(-1, 4).cpu().double()
    dt, dr = c[:, 1] - c[:, 0], c[:, 3] - c[:, 2]
    ok = dr > 0
    ghz = (dt[ok] / dr[ok] * 0.1).median().item()
    busy = (2 * 8 * iters * 32 / dt[ok]).median().item()
    r = {"matrix_busy_median": round(busy, 4), "clock_ghz_realtime_median": round(ghz, 3)}
    if tflops is not None:
        r["clock_ghz_implied"] = round(tflops / (256 * 4096 * busy) * 1e3, 3)
    return r


def probe_read_blocks_waves(num_seqs: int, num_kv_heads: int, max_seq_len: int) -> int:
    return int(lib().kvattn_probe_read_blocks_waves(num_seqs, num_kv_heads, max_seq_len))


def probe_read_blocks(kv_layer, num_blocks: int, block_table: torch.Tensor,
                      seq_lens: torch.Tensor, *, num_kv_heads: int, head_dim: int,
                      dtype: torch.dtype, max_seq_len: int,
                      out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """Read the K/V tiles a decode batch reads (one 32-bit word sum per lane
    of each wavefront); returns out, int32 [waves * 64]."""
    B = int(seq_lens.shape[0])
    _require_int32(block_table=block_table, seq_lens=seq_lens)
    _require_rows(B, block_table, seq_lens)
    waves = probe_read_blocks_waves(B, num_kv_heads, max_seq_len)
    if waves <= 0:
        raise ValueError("invalid or too large batch for the read probe")
    if out is None:
        out = torch.empty(waves * 64, dtype=torch.int32, device="cuda")
    if out.dtype != torch.int32 or out.numel() < waves * 64:
        raise ValueError(f"out must hold {waves * 64} int32")
    _require_cuda(kv_layer, block_table, seq_lens, out)
    check(lib().kvattn_probe_read_blocks(_ptr(kv_layer), int(num_blocks), _ptr(block_table),
                                         _ptr(seq_lens), B, int(num_kv_heads), int(head_dim),
                                         _dtype_code(dtype), int(block_table.shape[1]),
                                         int(max_seq_len), _ptr(out), _stream(stream)))
    return out
