"""Python binding of the ACP-SGD compressor library (argument marshalling only).

``Acp`` owns one C context (``acp_init``) and the device state block it needs (a torch
uint8 tensor handed to ``acp_bind_state``); its methods carry the C names without the
``acp_`` prefix and pass torch device pointers and the current HIP stream through.  Every
computation happens in libacp.so's kernels.
"""

from __future__ import annotations

import ctypes as C
from typing import Optional, Sequence, Tuple

import numpy as np

from . import _lib as L


def _check(status: int, lib, ctx, where: str):
    if status != L.ACP_OK:
        detail = lib.acp_last_error(ctx).decode() if ctx else ""
        raise L.AcpError(status, where, detail)


def _stream_ptr(stream) -> Optional[int]:
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return s.cuda_stream


def _fptr(t) -> int:
    import torch
    if t.dtype != torch.float32 or not t.is_cuda or not t.is_contiguous():
        raise ValueError("expected a contiguous float32 device tensor")
    return t.data_ptr()


class Acp:
    """One model replica's compressor state (see include/acp.h)."""

    def __init__(self, shapes: Sequence[Sequence[int]], rank: int, seed: int = 0,
                 cap_bytes: int = 25 * 1024 * 1024, world_size: int = 1, ef: bool = True,
                 device=None, bind: bool = True, reuse: bool = True, powersgd: bool = False):
        self.lib = L.load()
        self.shapes = [tuple(int(d) for d in s) for s in shapes]
        ndims = (C.c_int32 * len(self.shapes))(*[len(s) for s in self.shapes])
        flat = [d for s in self.shapes for d in s]
        dims = (C.c_int64 * len(flat))(*flat)
        flags = ((L.ACP_FLAG_REUSE if reuse else 0) | (L.ACP_FLAG_EF if ef else 0) |
                 (L.ACP_FLAG_POWERSGD if powersgd else 0))
        ctx = C.c_void_p()
        st = self.lib.acp_init(C.byref(ctx), len(self.shapes), ndims, dims, rank, seed, cap_bytes,
                               world_size, flags)
        if st != L.ACP_OK:
            raise L.AcpError(st, "acp_init")
        self.ctx = ctx
        self.rank, self.world_size, self.ef = rank, world_size, ef
        self.reuse, self.powersgd = reuse, powersgd
        self.state = None
        if bind:
            self.bind_state(device)

    # ---- setup
    def state_bytes(self) -> int:
        v = C.c_int64()
        _check(self.lib.acp_state_bytes(self.ctx, C.byref(v)), self.lib, self.ctx, "acp_state_bytes")
        return v.value

    def bind_state(self, device=None, stream=None):
        import torch
        dev = torch.device("cuda", torch.cuda.current_device()) if device is None else torch.device(device)
        with torch.cuda.device(dev):
            nbytes = self.state_bytes()
            self.state = torch.empty(nbytes, dtype=torch.uint8, device=dev)
            _check(self.lib.acp_bind_state(self.ctx, self.state.data_ptr(), nbytes, _stream_ptr(stream)),
                   self.lib, self.ctx, "acp_bind_state")

    # ---- layout
    def num_buckets(self) -> int:
        return self.lib.acp_num_buckets(self.ctx)

    def bucket_info(self, b: int) -> Tuple[int, int, int, int]:
        nt, ge, fp, fq = C.c_int32(), C.c_int64(), C.c_int64(), C.c_int64()
        _check(self.lib.acp_bucket_info(self.ctx, b, C.byref(nt), C.byref(ge), C.byref(fp), C.byref(fq)),
               self.lib, self.ctx, "acp_bucket_info")
        return nt.value, ge.value, fp.value, fq.value

    def layout(self, b: int):
        nt = self.bucket_info(b)[0]
        tids = np.zeros(nt, np.int32)
        go, fp, fq = (np.zeros(nt, np.int64) for _ in range(3))
        comp = np.zeros(nt, np.int32)
        P32, P64 = C.POINTER(C.c_int32), C.POINTER(C.c_int64)
        _check(self.lib.acp_layout(self.ctx, b, tids.ctypes.data_as(P32), go.ctypes.data_as(P64),
                                   fp.ctypes.data_as(P64), fq.ctypes.data_as(P64), comp.ctypes.data_as(P32)),
               self.lib, self.ctx, "acp_layout")
        return tids, go, fp, fq, comp

    def tensor_info(self, tid: int):
        c, n, m, b = C.c_int32(), C.c_int64(), C.c_int64(), C.c_int32()
        _check(self.lib.acp_tensor_info(self.ctx, tid, C.byref(c), C.byref(n), C.byref(m), C.byref(b)),
               self.lib, self.ctx, "acp_tensor_info")
        return bool(c.value), n.value, m.value, b.value

    def fusion_groups(self, which: str):
        """Compressed-buffer fusion groups of a P-step ('P') or Q-step ('Q'): (group index of
        every tensor in registration order, number of groups)."""
        g = np.zeros(len(self.shapes), np.int32)
        ng = C.c_int32()
        _check(self.lib.acp_fusion_groups(self.ctx, L.ACP_FACTOR_P if which == "P" else L.ACP_FACTOR_Q,
                                          g.ctypes.data_as(C.POINTER(C.c_int32)), C.byref(ng)),
               self.lib, self.ctx, "acp_fusion_groups")
        return g, ng.value

    def init_factor(self, tid: int, which: str) -> np.ndarray:
        comp, n, m, _ = self.tensor_info(tid)
        rows = n if which == "P" else m
        out = np.zeros((rows, self.rank), np.float32)
        _check(self.lib.acp_init_factor(self.ctx, tid, L.ACP_FACTOR_P if which == "P" else L.ACP_FACTOR_Q,
                                        out.ctypes.data, out.size), self.lib, self.ctx, "acp_init_factor")
        return out

    # ---- the step
    def compress(self, step: int, b: int, grad, factor_buf, stream=None):
        _check(self.lib.acp_compress(self.ctx, step, b, _fptr(grad), _fptr(factor_buf), _stream_ptr(stream)),
               self.lib, self.ctx, "acp_compress")

    def compress_noalloc(self, step: int, b: int, grad, factor_buf, stream=None):
        _check(self.lib.acp_compress_noalloc(self.ctx, step, b, _fptr(grad), _fptr(factor_buf),
                                             _stream_ptr(stream)),
               self.lib, self.ctx, "acp_compress_noalloc")

    def decompress(self, step: int, b: int, agg_factor, out, stream=None):
        _check(self.lib.acp_decompress(self.ctx, step, b, _fptr(agg_factor), _fptr(out), _stream_ptr(stream)),
               self.lib, self.ctx, "acp_decompress")

    def _ptrs(self, tensors):
        """Host array of one device pointer per bucket (the library reads acp_num_buckets() of them)."""
        if len(tensors) != self.num_buckets():
            raise ValueError(f"expected {self.num_buckets()} buffers (one per bucket), got {len(tensors)}")
        return (C.c_void_p * len(tensors))(*[_fptr(x) for x in tensors])

    def compress_all(self, step: int, grads, factor_bufs, stream=None):
        """One step for every bucket: ``grads`` / ``factor_bufs`` are lists of device tensors."""
        g, f = self._ptrs(grads), self._ptrs(factor_bufs)
        _check(self.lib.acp_compress_all(self.ctx, step, g, f, _stream_ptr(stream)), self.lib, self.ctx,
               "acp_compress_all")

    def decompress_all(self, step: int, aggs, outs, stream=None):
        a, o = self._ptrs(aggs), self._ptrs(outs)
        _check(self.lib.acp_decompress_all(self.ctx, step, a, o, _stream_ptr(stream)), self.lib, self.ctx,
               "acp_decompress_all")

    # ---- Power-SGD (a context made with powersgd=True)
    def powersgd_p(self, step: int, b: int, grad, p_buf, stream=None):
        _check(self.lib.acp_powersgd_p(self.ctx, step, b, _fptr(grad), _fptr(p_buf), _stream_ptr(stream)),
               self.lib, self.ctx, "acp_powersgd_p")

    def powersgd_q(self, step: int, b: int, grad, p_agg, q_buf, stream=None):
        _check(self.lib.acp_powersgd_q(self.ctx, step, b, _fptr(grad), _fptr(p_agg), _fptr(q_buf),
                                       _stream_ptr(stream)), self.lib, self.ctx, "acp_powersgd_q")

    def powersgd_decompress(self, step: int, b: int, q_agg, out, stream=None):
        _check(self.lib.acp_powersgd_decompress(self.ctx, step, b, _fptr(q_agg), _fptr(out), _stream_ptr(stream)),
               self.lib, self.ctx, "acp_powersgd_decompress")

    def powersgd_p_all(self, step: int, grads, p_bufs, stream=None):
        _check(self.lib.acp_powersgd_p_all(self.ctx, step, self._ptrs(grads), self._ptrs(p_bufs),
                                           _stream_ptr(stream)), self.lib, self.ctx, "acp_powersgd_p_all")

    def powersgd_q_all(self, step: int, grads, p_aggs, q_bufs, stream=None):
        _check(self.lib.acp_powersgd_q_all(self.ctx, step, self._ptrs(grads), self._ptrs(p_aggs),
                                           self._ptrs(q_bufs), _stream_ptr(stream)),
               self.lib, self.ctx, "acp_powersgd_q_all")

    def powersgd_decompress_all(self, step: int, q_aggs, outs, stream=None):
        _check(self.lib.acp_powersgd_decompress_all(self.ctx, step, self._ptrs(q_aggs), self._ptrs(outs),
                                                    _stream_ptr(stream)),
               self.lib, self.ctx, "acp_powersgd_decompress_all")

    # ---- inspection and checkpoint
    def error(self, b: int, e_out, stream=None):
        _check(self.lib.acp_error(self.ctx, b, _fptr(e_out), _stream_ptr(stream)), self.lib, self.ctx, "acp_error")

    def factor(self, tid: int, which: str, out, stream=None):
        w = L.ACP_FACTOR_P if which == "P" else L.ACP_FACTOR_Q
        _check(self.lib.acp_factor(self.ctx, tid, w, _fptr(out), _stream_ptr(stream)), self.lib, self.ctx,
               "acp_factor")

    def checkpoint_bytes(self) -> int:
        v = C.c_int64()
        _check(self.lib.acp_checkpoint_bytes(self.ctx, C.byref(v)), self.lib, self.ctx, "acp_checkpoint_bytes")
        return v.value

    def get_state(self) -> bytes:
        buf = C.create_string_buffer(self.checkpoint_bytes())
        _check(self.lib.acp_get_state(self.ctx, buf, len(buf)), self.lib, self.ctx, "acp_get_state")
        return buf.raw

    def set_state(self, blob: bytes):
        buf = C.create_string_buffer(blob, len(blob))
        _check(self.lib.acp_set_state(self.ctx, buf, len(blob)), self.lib, self.ctx, "acp_set_state")

    def profile_start(self, family: int, max_launches: int = 4096):
        _check(self.lib.acp_profile_start(self.ctx, family, max_launches), self.lib, self.ctx,
               "acp_profile_start")

    def profile_stop(self):
        """(timed launches, seconds, algorithmic bytes) since profile_start."""
        n, sec, by = C.c_int64(), C.c_double(), C.c_double()
        _check(self.lib.acp_profile_stop(self.ctx, C.byref(n), C.byref(sec), C.byref(by)), self.lib,
               self.ctx, "acp_profile_stop")
        return n.value, sec.value, by.value

    def close(self):
        if getattr(self, "ctx", None):
            self.lib.acp_destroy(self.ctx)
            self.ctx = None
        self.state = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
