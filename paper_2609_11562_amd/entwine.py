"""ctypes binding of libentwine.so (C ABI in include/entwine.h).

Argument marshalling only: torch CUDA tensors are turned into device
pointers and leading dimensions, torch streams into hipStream_t handles.
Every step of the computation runs in the HIP library; if the library is
missing this module raises instead of computing anything on the host.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libentwine.so")
_lib = None

OK, EINVAL, EUNSUPPORTED, ENOMEM, EHIP, ETIMEOUT = range(6)
ORDER_INTERLEAVED, ORDER_ROW_MAJOR, ORDER_M_MAJOR = 0, 1, 2
GEMM_256x256, GEMM_256x128, GEMM_128x256, GEMM_128x128 = 0, 1, 2, 3
# release_blocks values other than a block count g >= 1
RELEASE_AT_END, RELEASE_PARTITION, RELEASE_OUTPUT = -1, -2, -3
GEMM_SHAPES = {GEMM_256x256: (256, 256), GEMM_256x128: (256, 128), GEMM_128x256: (128, 256),
               GEMM_128x128: (128, 128)}
DEST_ALL = -1
MAX_P = 8
TILE = 128


class EntwineError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{_status_name(status)}: {msg}")
        self.status = status


class Config(ctypes.Structure):
    """Mirror of entwine_config; zero / -1 fields mean the library default."""

    _fields_ = [("order", ctypes.c_int32), ("gemm_cfg", ctypes.c_int32),
                ("reduce_wgs", ctypes.c_int32), ("reduce_threads", ctypes.c_int32),
                ("timeout_us", ctypes.c_int32), ("withhold_peer", ctypes.c_int32),
                ("record_timing", ctypes.c_int32), ("group_m", ctypes.c_int32),
                ("gemm_wgs", ctypes.c_int32), ("launch", ctypes.c_int32),
                ("release_blocks", ctypes.c_int32), ("store_mode", ctypes.c_int32)]

    @classmethod
    def make(cls, **kw) -> "Config":
        c = cls()
        lib().entwine_config_default(ctypes.byref(c))
        for k, v in kw.items():
            if v is not None:
                setattr(c, k, int(v))
        return c


_i32, _i64, _vp = ctypes.c_int32, ctypes.c_int64, ctypes.c_void_p
_P32 = ctypes.POINTER(ctypes.c_int32)
_PROTOS = {
    "entwine_config_default": (None, [ctypes.POINTER(Config)]),
    "entwine_ctx_create": (_i32, [ctypes.POINTER(_vp), _i32, _i64, _i64, _i64, _i32]),
    "entwine_ctx_destroy": (_i32, [_vp]),
    "entwine_gemm_rs": (_i32, [_vp, _vp, _i64, _vp, _i64, ctypes.POINTER(_vp), _i64, _i32, _vp, _i64,
                               _vp, _i64, ctypes.POINTER(Config), _vp, _vp]),
    "entwine_gemm_rs_rmsnorm": (_i32, [_vp, _vp, _i64, _vp, _i64, ctypes.POINTER(_vp), _i64, _i32, _vp, _i64, _vp,
                                       ctypes.c_float, _vp, _i64, _vp, _i64, _vp, _i64, ctypes.POINTER(Config),
                                       _vp]),
    "entwine_gemm_only": (_i32, [_vp, _vp, _i64, _vp, _i64, _vp, _i64, ctypes.POINTER(Config), _vp]),
    "entwine_reduce_only": (_i32, [_vp, _vp, _i64, ctypes.POINTER(_vp), _i64, _i32, _vp, _i64,
                                   ctypes.POINTER(Config), _vp]),
    "entwine_query_status": (_i32, [_vp, _P32, _P32, _P32]),
    "entwine_last_timing": (_i32, [_vp, _i32, ctypes.POINTER(ctypes.c_float),
                                   ctypes.POINTER(ctypes.c_float), ctypes.POINTER(ctypes.c_float)]),
    "entwine_last_stamps": (_i32, [_vp, _i32, ctypes.POINTER(ctypes.c_uint64), _i32, _P32, _P32,
                                   ctypes.POINTER(ctypes.c_double)]),
    "entwine_last_clock": (_i32, [_vp, _i32, ctypes.POINTER(ctypes.c_double)]),
    "entwine_validate": (_i32, [_i64, _i64, _i64, _i32, _i32, ctypes.POINTER(Config)]),
    "entwine_tile_schedule": (_i32, [_i32, _i64, _i64, _i32, _i32, _i32, _i32, _P32, _P32]),
    "entwine_consumer_tasks": (_i32, [_i32, _i32, _i32, _i32, _i32, _P32, _P32, _i32, _P32]),
    "entwine_status_string": (ctypes.c_char_p, [_i32]),
    "entwine_last_error": (ctypes.c_char_p, [_vp]),
    "entwine_abi_version": (_i32, []),
}


def lib_path() -> str:
    return _LIB_PATH


def lib():
    """Load libentwine.so (once).  Raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise ImportError(f"libentwine.so not found at {_LIB_PATH}; build it with "
                              "`python -m paper_2609_11562_amd.build` (no host fallback exists)")
        L = ctypes.CDLL(_LIB_PATH)
        for name, (res, args) in _PROTOS.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def _status_name(s: int) -> str:
    try:
        return lib().entwine_status_string(s).decode()
    except Exception:  # noqa: BLE001 - only used while formatting an error
        return f"status {s}"


def _check(status: int, ctx=None):
    if status != OK:
        msg = lib().entwine_last_error(ctx).decode(errors="replace")
        raise EntwineError(status, msg)


def validate(M, N, K, P, dest, cfg: Config | None = None) -> int:
    """Host-only argument check; returns the status code."""
    return lib().entwine_validate(M, N, K, P, dest, ctypes.byref(cfg) if cfg else None)


def tile_schedule(order: int, M: int, N: int, P: int, BM: int, BN: int, group_m: int = 1):
    """Traversal as computed by the library: (blocks[p] = (d, l, mb, nb),
    tiles[tile_row, tile_col] = (d, t))."""
    nb = (M // BM) * (N // BN)
    blocks = np.zeros((nb, 4), np.int32)
    tiles = np.zeros((M // TILE, N // TILE, 2), np.int32)
    _check(lib().entwine_tile_schedule(order, M, N, P, BM, BN, group_m, blocks.ctypes.data_as(_P32),
                                       tiles.ctypes.data_as(_P32)))
    return blocks, tiles


def consumer_tasks(dest: int, P: int, Q: int, x: int, j: int):
    cap = Q + 1
    buf = np.zeros(cap, np.int32)
    part, count = ctypes.c_int32(), ctypes.c_int32()
    _check(lib().entwine_consumer_tasks(dest, P, Q, x, j, ctypes.byref(part), buf.ctypes.data_as(_P32),
                                        cap, ctypes.byref(count)))
    return part.value, buf[:count.value].tolist()


def _stream_handle(stream) -> int | None:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _mat(t, rows: int, cols: int, name: str):
    import torch
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a CUDA tensor")
    if t.dtype not in (torch.bfloat16, torch.int16, torch.uint16):
        raise TypeError(f"{name} must hold bfloat16 values")
    if t.dim() != 2 or t.shape[0] != rows or t.shape[1] != cols or t.stride(1) != 1:
        raise ValueError(f"{name} must be a row-major {rows}x{cols} matrix, got {tuple(t.shape)} "
                         f"strides {tuple(t.stride())}")
    return t.data_ptr(), t.stride(0)


class Context:
    """One problem shape (M, N, K, P) on one device; owns flags and events."""

    def __init__(self, M: int, N: int, K: int, P: int, device: int = 0):
        self.M, self.N, self.K, self.P, self.device = M, N, K, P, device
        h = _vp()
        _check(lib().entwine_ctx_create(ctypes.byref(h), device, M, N, K, P))
        self._h = h

    def close(self):
        if getattr(self, "_h", None):
            lib().entwine_ctx_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:  # noqa: BLE001 - interpreter shutdown
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    def _peers(self, peers):
        if self.P == 1:
            return None, 0
        if peers is None or len(peers) != self.P - 1:
            raise ValueError(f"need {self.P - 1} peer partials")
        ptrs, ld = [], None
        for q, t in enumerate(peers):
            p, l = _mat(t, self.M, self.N, f"peer {q}")
            if ld is not None and l != ld:
                raise ValueError("peers must share one leading dimension")
            ptrs.append(p)
            ld = l
        return (_vp * len(ptrs))(*ptrs), ld

    def out_rows(self, dest: int) -> int:
        return self.M if dest == DEST_ALL else self.M // self.P

    def gemm_rs(self, A, B, peers, dest: int, out=None, partial=None, cfg: Config | None = None,
                gemm_stream=None, reduce_stream=None):
        """Fused GEMM + tile reduce; returns ``out``.  With reduce_stream None
        a second stream is required for overlap: pass one explicitly, or the
        reducer runs on gemm_stream after the GEMM."""
        import torch
        a, lda = _mat(A, self.M, self.K, "A")
        b, ldb = _mat(B, self.K, self.N, "B")
        if out is None:
            out = torch.empty(self.out_rows(dest), self.N, dtype=torch.bfloat16, device=A.device)
        o, ldo = _mat(out, self.out_rows(dest), self.N, "out")
        c, ldc = (0, 0) if partial is None else _mat(partial, self.M, self.N, "partial")
        parr, ldp = self._peers(peers)
        gs = _stream_handle(gemm_stream)
        rs = gs if reduce_stream is None else _stream_handle(reduce_stream)
        _check(lib().entwine_gemm_rs(self._h, a, lda, b, ldb, parr, ldp, dest, o, ldo, c or None, ldc,
                                     ctypes.byref(cfg) if cfg else None, gs, rs), self._h)
        return out

    def gemm_rs_rmsnorm(self, A, B, peers, dest: int, residual, gamma, eps: float, h_out=None, y_out=None,
                        partial=None, cfg: Config | None = None, stream=None):
        """Fused GEMM + tile reduce + residual addition + RMSNorm (one
        launch); returns ``(h_out, y_out)``."""
        import torch
        a, lda = _mat(A, self.M, self.K, "A")
        b, ldb = _mat(B, self.K, self.N, "B")
        rows = self.out_rows(dest)
        if h_out is None:
            h_out = torch.empty(rows, self.N, dtype=torch.bfloat16, device=A.device)
        if y_out is None:
            y_out = torch.empty(rows, self.N, dtype=torch.bfloat16, device=A.device)
        h, ldh = _mat(h_out, rows, self.N, "h_out")
        y, ldy = _mat(y_out, rows, self.N, "y_out")
        r, ldr = _mat(residual, rows, self.N, "residual")
        g, _ = _mat(gamma.view(1, -1), 1, self.N, "gamma")
        c, ldc = (0, 0) if partial is None else _mat(partial, self.M, self.N, "partial")
        parr, ldp = self._peers(peers)
        _check(lib().entwine_gemm_rs_rmsnorm(self._h, a, lda, b, ldb, parr, ldp, dest, r, ldr, g, float(eps), h, ldh,
                                             y, ldy, c or None, ldc, ctypes.byref(cfg) if cfg else None,
                                             _stream_handle(stream)), self._h)
        return h_out, y_out

    def gemm_only(self, A, B, partial=None, cfg: Config | None = None, stream=None):
        import torch
        a, lda = _mat(A, self.M, self.K, "A")
        b, ldb = _mat(B, self.K, self.N, "B")
        if partial is None:
            partial = torch.empty(self.M, self.N, dtype=torch.bfloat16, device=A.device)
        c, ldc = _mat(partial, self.M, self.N, "partial")
        _check(lib().entwine_gemm_only(self._h, a, lda, b, ldb, c, ldc, ctypes.byref(cfg) if cfg else None,
                                       _stream_handle(stream)), self._h)
        return partial

    def reduce_only(self, partial, peers, dest: int, out=None, cfg: Config | None = None, stream=None):
        import torch
        c, ldc = _mat(partial, self.M, self.N, "partial")
        if out is None:
            out = torch.empty(self.out_rows(dest), self.N, dtype=torch.bfloat16, device=partial.device)
        o, ldo = _mat(out, self.out_rows(dest), self.N, "out")
        parr, ldp = self._peers(peers)
        _check(lib().entwine_reduce_only(self._h, c, ldc, parr, ldp, dest, o, ldo,
                                         ctypes.byref(cfg) if cfg else None, _stream_handle(stream)), self._h)
        return out

    def query_status(self):
        """(status, tile, src) of the device status word; clears it."""
        code, tile, src = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int32()
        s = lib().entwine_query_status(self._h, ctypes.byref(code), ctypes.byref(tile), ctypes.byref(src))
        if s not in (OK, ETIMEOUT):
            _check(s, self._h)
        return s, tile.value, src.value

    def last_stamps(self, back: int = 0):
        """Per-workgroup timeline of a single-launch call made with
        record_timing=1: (stamps, nproducers) with stamps an (nwgs, 4) float
        array of microseconds since the first workgroup's start, columns
        start, producer end, first reduction task ready (NaN if none), end."""
        import numpy as np
        n, g, tpu = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_double()
        _check(lib().entwine_last_stamps(self._h, back, None, 0, ctypes.byref(n), ctypes.byref(g), ctypes.byref(tpu)),
               self._h)
        buf = (ctypes.c_uint64 * (4 * n.value))()
        _check(lib().entwine_last_stamps(self._h, back, buf, len(buf), None, None, None), self._h)
        raw = np.frombuffer(buf, dtype=np.uint64).reshape(n.value, 4)
        t0 = raw[:, 0].min()
        us = (raw.astype(np.float64) - float(t0)) / tpu.value
        us[raw[:, 2] == 0, 2] = np.nan
        return us, g.value

    def last_clock(self, back: int = 0) -> float:
        """Engine clock (GHz) the producer role ran at during a single-launch
        call made with record_timing=1."""
        ghz = ctypes.c_double()
        _check(lib().entwine_last_clock(self._h, back, ctypes.byref(ghz)), self._h)
        return ghz.value

    def last_timing(self, back: int = 0):
        """(gemm_ms, reduce_ms, e2e_ms) of a call made with record_timing=1."""
        g, r, e = ctypes.c_float(), ctypes.c_float(), ctypes.c_float()
        _check(lib().entwine_last_timing(self._h, back, ctypes.byref(g), ctypes.byref(r), ctypes.byref(e)),
               self._h)
        return g.value, r.value, e.value
