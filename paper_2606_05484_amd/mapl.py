"""ctypes binding of libmapl (include/mapl.h): argument marshalling only.

Every entry point takes device pointers -- torch tensors (their data_ptr()),
plain integers, or None -- and the HIP stream to enqueue on (default: torch's
current stream on the current device).  All computation happens in the HIP
kernels of libmapl.so; this module never computes a result itself and raises
MaplError when the library is missing or a call fails.
"""
import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libmapl.so")

MAPL_OK = 0
STATUS = {0: "MAPL_OK", -1: "MAPL_E_NULL", -2: "MAPL_E_SHAPE", -3: "MAPL_E_DTYPE", -4: "MAPL_E_RANGE",
          -5: "MAPL_E_ALIGN", -6: "MAPL_E_ALIAS", -7: "MAPL_E_WORKSPACE", -8: "MAPL_E_UNSUPPORTED",
          -9: "MAPL_E_HIP"}
F32, BF16, U8, U16 = 0, 1, 2, 3
AMBIENT, COORD = 0, 1
CALL_ENCODE, CALL_DECODE, CALL_DECODE_BWD, CALL_ENCODE_BWD, CALL_STIEFEL = range(5)
SENDER, RECEIVER = 0, 1
_DT = {"f32": F32, "bf16": BF16, "u8": U8, "u16": U16}
_SPACE = {"ambient": AMBIENT, "coord": COORD}


class MaplError(RuntimeError):
    def __init__(self, status, message):
        super().__init__("%s (%d): %s" % (STATUS.get(status, "?"), status, message))
        self.status = status


class CodecDesc(ctypes.Structure):
    _fields_ = [("T", ctypes.c_int64), ("d", ctypes.c_int64), ("r", ctypes.c_int64), ("V", ctypes.c_int64),
                ("k", ctypes.c_int64), ("anchor_space", ctypes.c_int32), ("L", ctypes.c_int32),
                ("K", ctypes.c_int32), ("x_dtype", ctypes.c_int32), ("ab_dtype", ctypes.c_int32),
                ("code_dtype", ctypes.c_int32), ("group_dim", ctypes.c_int32)]


_lib = None
_P = ctypes.c_void_p
_SIG = {
    "mapl_encode": [ctypes.POINTER(CodecDesc)] + [_P] * 7 + [_P, ctypes.c_size_t, _P],
    "mapl_encode_noalloc": [ctypes.POINTER(CodecDesc)] + [_P] * 7 + [_P],
    "mapl_codebook_pack": [ctypes.c_int32, ctypes.c_int32, ctypes.c_int64, _P, _P, ctypes.c_int32, _P, _P],
    "mapl_codebook_unpack": [ctypes.c_int32, ctypes.c_int32, ctypes.c_int64, _P, _P, ctypes.c_int32, _P, _P],
    "mapl_decode": [ctypes.POINTER(CodecDesc)] + [_P] * 7 + [_P, ctypes.c_size_t, _P],
    "mapl_decode_bwd": [ctypes.POINTER(CodecDesc)] + [_P] * 9 + [ctypes.c_int, _P, ctypes.c_size_t, _P],
    "mapl_encode_bwd": [ctypes.POINTER(CodecDesc)] + [_P] * 8 + [ctypes.c_int, _P, ctypes.c_size_t, _P],
    "mapl_decode_bwd_q": [ctypes.POINTER(CodecDesc)] + [_P] * 7 + [ctypes.c_int32] * 3 + [_P] * 3 +
                         [ctypes.c_int, _P, ctypes.c_size_t, _P],
    "mapl_decode_bwd_q_workspace_bytes": [ctypes.POINTER(CodecDesc), ctypes.c_int32, ctypes.c_int32],
    "mapl_anchor_bwd": [ctypes.POINTER(CodecDesc), ctypes.c_int] + [_P] * 5 + [ctypes.c_int, _P, ctypes.c_size_t,
                                                                              _P],
    "mapl_anchor_bwd_workspace_bytes": [ctypes.POINTER(CodecDesc), ctypes.c_int],
    "mapl_grad_dequantize": [ctypes.c_int64, ctypes.c_int64] + [ctypes.c_int32] * 3 + [_P, _P, ctypes.c_int32,
                                                                                        _P, _P],
    "mapl_stiefel_step": [ctypes.c_int64] * 3 + [_P] * 3 + [ctypes.c_float, ctypes.c_float, ctypes.c_int,
                                                            ctypes.c_int, _P, ctypes.c_size_t, _P],
    "mapl_workspace_bytes": [ctypes.POINTER(CodecDesc), ctypes.c_int, ctypes.c_int64, ctypes.c_int64,
                             ctypes.c_int64],
    "mapl_last_error": [],
    "mapl_version": [],
    "mapl_profile": [ctypes.c_int],
    "mapl_profile_report": [ctypes.c_char_p, ctypes.c_size_t],
}
_RES = {"mapl_workspace_bytes": ctypes.c_size_t, "mapl_decode_bwd_q_workspace_bytes": ctypes.c_size_t,
        "mapl_anchor_bwd_workspace_bytes": ctypes.c_size_t,
        "mapl_last_error": ctypes.c_char_p}
EXPORTS = tuple(_SIG)


def lib():
    """Load libmapl.so (built in-tree by paper_2606_05484_amd.build)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise MaplError(-8, "libmapl.so not built at %s (run paper_2606_05484_amd.build)" % LIB_PATH)
        L = ctypes.CDLL(LIB_PATH)
        for name, args in _SIG.items():
            fn = getattr(L, name)
            fn.argtypes = args
            fn.restype = _RES.get(name, ctypes.c_int)
        _lib = L
    return _lib


def last_error():
    return lib().mapl_last_error().decode()


def _check(status):
    if status != MAPL_OK:
        raise MaplError(status, last_error())


def _ptr(x):
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def desc(T, d, r, V=0, k=0, L=0, K=0, x_dtype="bf16", anchor_space="ambient", code_dtype=None, group_dim=0):
    """Build a mapl_codec_desc; code_dtype defaults to u8 for K <= 256, else u16."""
    if code_dtype is None:
        code_dtype = "u8" if K <= 256 else "u16"
    dt = _DT[x_dtype] if isinstance(x_dtype, str) else x_dtype
    return CodecDesc(T, d, r, V, k, _SPACE[anchor_space] if isinstance(anchor_space, str) else anchor_space,
                     L, K, dt, dt, _DT[code_dtype] if isinstance(code_dtype, str) else code_dtype, group_dim)


def payload_bytes_per_token(D):
    """Bytes that cross the pipeline link per token (ids excluded)."""
    if D.L == 0:
        return D.r * (4 if D.x_dtype == F32 else 2)
    if D.group_dim == 2:
        return D.L * (D.r // 2)
    return D.L * (1 if D.code_dtype == U8 else 2)


def workspace_bytes(D, call, P=0, d=0, r=0):
    n = lib().mapl_workspace_bytes(ctypes.byref(D) if D is not None else None, call, P, d, r)
    if n == 0 and last_error():
        raise MaplError(-2, last_error())
    return n


def workspace(nbytes, device=None):
    """A device byte buffer for the workspace (torch's allocator aligns to 512 B)."""
    import torch
    return torch.empty(max(int(nbytes), 1), dtype=torch.uint8, device=device or "cuda")


def encode(D, X, ids, U, A_s, B_s, C, payload, ws, ws_bytes=None, stream=None):
    wb = ws_bytes if ws_bytes is not None else (ws.numel() if ws is not None else 0)
    _check(lib().mapl_encode(ctypes.byref(D), _ptr(X), _ptr(ids), _ptr(U), _ptr(A_s), _ptr(B_s), _ptr(C),
                             _ptr(payload), _ptr(ws), wb, _stream(stream)))


def encode_noalloc(D, X, ids, U, A_s, B_s, C, payload, stream=None):
    """mapl_encode on the library's static device scratch (no workspace)."""
    _check(lib().mapl_encode_noalloc(ctypes.byref(D), _ptr(X), _ptr(ids), _ptr(U), _ptr(A_s), _ptr(B_s), _ptr(C),
                                     _ptr(payload), _stream(stream)))


NOALLOC_SCRATCH_BYTES = 16 << 20


def decode(D, payload, ids, U, A_r, B_r, C, Xhat, ws, ws_bytes=None, stream=None):
    wb = ws_bytes if ws_bytes is not None else (ws.numel() if ws is not None else 0)
    _check(lib().mapl_decode(ctypes.byref(D), _ptr(payload), _ptr(ids), _ptr(U), _ptr(A_r), _ptr(B_r), _ptr(C),
                             _ptr(Xhat), _ptr(ws), wb, _stream(stream)))


def decode_bwd(D, dXhat, payload, ids, U, A_r, B_r, C, dZ, dU, accumulate_dU, ws, ws_bytes=None, stream=None):
    wb = ws_bytes if ws_bytes is not None else (ws.numel() if ws is not None else 0)
    _check(lib().mapl_decode_bwd(ctypes.byref(D), _ptr(dXhat), _ptr(payload), _ptr(ids), _ptr(U), _ptr(A_r),
                                 _ptr(B_r), _ptr(C), _ptr(dZ), _ptr(dU), int(accumulate_dU), _ptr(ws), wb,
                                 _stream(stream)))


def decode_bwd_q(D, dXhat, payload, ids, U, A_r, B_r, C, Lg, Kg, Cg, gcodes, dU, accumulate_dU, ws,
                 ws_bytes=None, stream=None, gcode_dtype=None):
    """decode_bwd with the returned gradient RVQ-encoded into gcodes [T,Lg]."""
    wb = ws_bytes if ws_bytes is not None else (ws.numel() if ws is not None else 0)
    gdt = (U8 if Kg <= 256 else U16) if gcode_dtype is None else _DT.get(gcode_dtype, gcode_dtype)
    _check(lib().mapl_decode_bwd_q(ctypes.byref(D), _ptr(dXhat), _ptr(payload), _ptr(ids), _ptr(U), _ptr(A_r),
                                   _ptr(B_r), _ptr(C), Lg, Kg, gdt, _ptr(Cg), _ptr(gcodes), _ptr(dU),
                                   int(accumulate_dU), _ptr(ws), wb, _stream(stream)))


def decode_bwd_q_workspace_bytes(D, Lg, Kg):
    n = lib().mapl_decode_bwd_q_workspace_bytes(ctypes.byref(D), Lg, Kg)
    if n == 0 and last_error():
        raise MaplError(-2, last_error())
    return n


def anchor_bwd(D, side, dY, ids, U, B, dA, accumulate, ws, ws_bytes=None, stream=None):
    """Gradient of the sender's (side 0) or receiver's (side 1) anchor table."""
    wb = ws_bytes if ws_bytes is not None else (ws.numel() if ws is not None else 0)
    _check(lib().mapl_anchor_bwd(ctypes.byref(D), int(side), _ptr(dY), _ptr(ids), _ptr(U), _ptr(B), _ptr(dA),
                                 int(accumulate), _ptr(ws), wb, _stream(stream)))


def anchor_bwd_workspace_bytes(D, side):
    n = lib().mapl_anchor_bwd_workspace_bytes(ctypes.byref(D), int(side))
    if n == 0 and last_error():
        raise MaplError(-2, last_error())
    return n


def grad_dequantize(T, r, Lg, Kg, gcodes, Cg, dZ, out_dtype="bf16", stream=None, gcode_dtype=None):
    """dZ[t] = sum_l Cg[l, gcodes[t, l]] as bf16 or fp32."""
    gdt = (U8 if Kg <= 256 else U16) if gcode_dtype is None else _DT.get(gcode_dtype, gcode_dtype)
    _check(lib().mapl_grad_dequantize(T, r, Lg, Kg, gdt, _ptr(gcodes), _ptr(Cg), _DT.get(out_dtype, out_dtype),
                                      _ptr(dZ), _stream(stream)))


def encode_bwd(D, dZ, X, ids, U, A_s, B_s, dX, dU, accumulate_dU, ws, ws_bytes=None, stream=None):
    wb = ws_bytes if ws_bytes is not None else (ws.numel() if ws is not None else 0)
    _check(lib().mapl_encode_bwd(ctypes.byref(D), _ptr(dZ), _ptr(X), _ptr(ids), _ptr(U), _ptr(A_s), _ptr(B_s),
                                 _ptr(dX), _ptr(dU), int(accumulate_dU), _ptr(ws), wb, _stream(stream)))


def stiefel_step(P, d, r, U, G, M, lr, beta, lmo_steps, retract_steps, ws, ws_bytes=None, stream=None):
    wb = ws_bytes if ws_bytes is not None else (ws.numel() if ws is not None else 0)
    _check(lib().mapl_stiefel_step(P, d, r, _ptr(U), _ptr(G), _ptr(M), lr, beta, lmo_steps, retract_steps,
                                   _ptr(ws), wb, _stream(stream)))


def codebook_pack(L, K, r, C, rows, n, buf, stream=None):
    """Sender side of the streaming codebook sync: buf[l, i] = C[l, rows[l, i]]."""
    _check(lib().mapl_codebook_pack(L, K, r, _ptr(C), _ptr(rows), n, _ptr(buf), _stream(stream)))


def codebook_unpack(L, K, r, buf, rows, n, C, stream=None):
    """Receiver side: C[l, rows[l, i]] = buf[l, i]."""
    _check(lib().mapl_codebook_unpack(L, K, r, _ptr(buf), _ptr(rows), n, _ptr(C), _stream(stream)))


def profile(enable):
    """Per-kernel event tracing: 0 off, 1 (True) on, 2 also RVQ decision
    counters (see mapl_profile_report)."""
    _check(lib().mapl_profile(int(enable)))


def profile_report():
    """{kernel name: (launches, total_ms)} for the launches since the last report."""
    buf = ctypes.create_string_buffer(1 << 16)
    _check(lib().mapl_profile_report(buf, len(buf)))
    out = {}
    for line in buf.value.decode().splitlines():
        name, n, ms = line.split()
        out[name] = (int(n), float(ms))
    return out
