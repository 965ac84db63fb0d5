"""ctypes binding of libgsrq.so (the C ABI in include/gsrq.h).

Argument marshalling only: every step of the GSRQ path runs in the HIP
kernels of the library.  torch supplies device memory and the stream; a torch
tensor is passed as its data pointer.  If the library is not built, importing
functions from here raises instead of falling back to anything else.
"""
from __future__ import annotations

import ctypes
import math
import os
from dataclasses import dataclass
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libgsrq.so")

GSRQ_OK, GSRQ_E_ARG, GSRQ_E_UNSUPPORTED, GSRQ_E_WORKSPACE, GSRQ_E_HIP = range(5)
GSRQ_F32, GSRQ_F16 = 0, 1
GSRQ_RESUME, GSRQ_ASSIGN_IN, GSRQ_NO_EARLY_STOP, GSRQ_KMEANS, GSRQ_CHECK_INPUTS = 1, 2, 4, 8, 16


class GsrqError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {status_string(status)} (status {status})")


class Shape(ctypes.Structure):
    _fields_ = [("N", ctypes.c_int64), ("D", ctypes.c_int32), ("d", ctypes.c_int32),
                ("K", ctypes.c_int32), ("M", ctypes.c_int32)]


class AttnShape(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int32), ("cap", ctypes.c_int32), ("Hq", ctypes.c_int32),
                ("Hkv", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("rope_base", ctypes.c_float), ("scale", ctypes.c_float),
                ("flags", ctypes.c_uint32)]


_lib = None
_vp = ctypes.c_void_p


def load_library(path: str = LIB_PATH):
    """Load libgsrq.so once; raise if it is missing (no fallback exists)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is not built; run `python -c 'import __graft_entry__ as g; g.build()'`")
    # torch first: the library then binds to the HIP runtime torch ships and
    # uses, instead of loading a second runtime that cannot see torch's
    # device memory
    _torch()
    lib = ctypes.CDLL(path)
    SP = ctypes.POINTER(Shape)
    lib.gsrq_status_string.restype = ctypes.c_char_p
    lib.gsrq_status_string.argtypes = [ctypes.c_int]
    lib.gsrq_code_words.restype = ctypes.c_size_t
    lib.gsrq_code_words.argtypes = [SP]
    lib.gsrq_bits_per_element.restype = ctypes.c_double
    lib.gsrq_bits_per_element.argtypes = [SP]
    lib.gsrq_train_workspace_bytes.restype = ctypes.c_int
    lib.gsrq_train_workspace_bytes.argtypes = [SP, ctypes.POINTER(ctypes.c_size_t)]
    lib.gsrq_encode_workspace_bytes.restype = ctypes.c_int
    lib.gsrq_encode_workspace_bytes.argtypes = [SP, ctypes.POINTER(ctypes.c_size_t)]
    lib.gsrq_train_stage.restype = ctypes.c_int
    lib.gsrq_train_stage.argtypes = [SP, _vp, ctypes.c_int, ctypes.c_int64, _vp, ctypes.c_int32,
                                     _vp, ctypes.c_uint32, _vp, _vp, _vp, _vp, _vp, _vp,
                                     _vp, ctypes.c_size_t, _vp]
    lib.gsrq_encode.restype = ctypes.c_int
    lib.gsrq_encode.argtypes = [SP, _vp, ctypes.c_int, ctypes.c_int64, _vp, _vp, _vp, _vp,
                                _vp, ctypes.c_size_t, _vp]
    lib.gsrq_prepared_bytes.restype = ctypes.c_int
    lib.gsrq_prepared_bytes.argtypes = [SP, ctypes.POINTER(ctypes.c_size_t)]
    lib.gsrq_encode_prepare.restype = ctypes.c_int
    lib.gsrq_encode_prepare.argtypes = [SP, _vp, _vp, _vp, ctypes.c_size_t, _vp]
    lib.gsrq_encode_prepared.restype = ctypes.c_int
    lib.gsrq_encode_prepared.argtypes = [SP, _vp, ctypes.c_int, ctypes.c_int64, _vp, _vp, _vp,
                                         _vp]
    lib.gsrq_decode.restype = ctypes.c_int
    lib.gsrq_decode.argtypes = [SP, _vp, ctypes.c_int32, _vp, _vp, _vp, ctypes.c_int,
                                ctypes.c_int64, _vp]
    lib.gsrq_row_weights.restype = ctypes.c_int
    lib.gsrq_row_weights.argtypes = [_vp, ctypes.c_int, ctypes.c_int64, ctypes.c_int32,
                                     ctypes.c_int64, ctypes.c_float, _vp, _vp, _vp, _vp]
    AP = ctypes.POINTER(AttnShape)
    lib.gsrq_attn_workspace_bytes.restype = ctypes.c_int
    lib.gsrq_attn_workspace_bytes.argtypes = [AP, ctypes.POINTER(ctypes.c_size_t)]
    lib.gsrq_attn_workspace_bytes_kv.restype = ctypes.c_int
    lib.gsrq_attn_workspace_bytes_kv.argtypes = [AP, SP, ctypes.POINTER(ctypes.c_size_t)]
    lib.gsrq_attn_decode.restype = ctypes.c_int
    lib.gsrq_attn_decode.argtypes = [AP, SP, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp,
                                     ctypes.c_int, _vp, _vp, ctypes.c_size_t, _vp]
    lib.gsrq_attn_decode_noalloc.restype = ctypes.c_int
    lib.gsrq_attn_decode_noalloc.argtypes = [AP, SP, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp,
                                             ctypes.c_int, _vp, _vp]
    lib.gsrq_timing_enable.restype = ctypes.c_int
    lib.gsrq_timing_enable.argtypes = [ctypes.c_int]
    lib.gsrq_timing_enable_kinds.restype = ctypes.c_int
    lib.gsrq_timing_enable_kinds.argtypes = [ctypes.c_uint32]
    lib.gsrq_timing_read.restype = ctypes.c_int
    lib.gsrq_timing_read.argtypes = [ctypes.POINTER(ctypes.c_double),
                                     ctypes.POINTER(ctypes.c_int64), ctypes.c_int]
    _lib = lib
    return lib


KERNEL_KINDS = ("assign", "finalize", "encode", "decode", "transpose", "accumulate",
                "fragments", "exact", "attention")


def timing_enable(on: bool = True, kinds=None):
    """Bracket kernel launches with HIP events on their stream (measurement):
    every kind, or only the named ones (names from KERNEL_KINDS)."""
    if kinds is None:
        _check(load_library().gsrq_timing_enable(1 if on else 0), "gsrq_timing_enable")
        return
    mask = 0
    for k in kinds:
        mask |= 1 << KERNEL_KINDS.index(k)
    _check(load_library().gsrq_timing_enable_kinds(ctypes.c_uint32(mask if on else 0)),
           "gsrq_timing_enable_kinds")


def timing_read():
    """{kind: (total_ms, launches)} for the launches recorded since enabling."""
    n = len(KERNEL_KINDS)
    ms = (ctypes.c_double * n)()
    cnt = (ctypes.c_int64 * n)()
    _check(load_library().gsrq_timing_read(ms, cnt, n), "gsrq_timing_read")
    return {k: (float(ms[i]), int(cnt[i])) for i, k in enumerate(KERNEL_KINDS)}


def status_string(status: int) -> str:
    return load_library().gsrq_status_string(int(status)).decode()


def _check(status: int, where: str):
    if status != GSRQ_OK:
        raise GsrqError(status, where)


def make_shape(N, D, d, K, M=1) -> Shape:
    return Shape(int(N), int(D), int(d), int(K), int(M))


def code_words(N, D, d, K, M) -> int:
    return int(load_library().gsrq_code_words(ctypes.byref(make_shape(N, D, d, K, M))))


def bits_per_element(d, K, M, D=None) -> float:
    D = d if D is None else D
    return float(load_library().gsrq_bits_per_element(ctypes.byref(make_shape(1, D, d, K, M))))


def train_workspace_bytes(N, D, d, K) -> int:
    n = ctypes.c_size_t(0)
    _check(load_library().gsrq_train_workspace_bytes(ctypes.byref(make_shape(N, D, d, K, 1)),
                                                      ctypes.byref(n)), "train_workspace_bytes")
    return int(n.value)


def encode_workspace_bytes(N, D, d, K, M) -> int:
    n = ctypes.c_size_t(0)
    _check(load_library().gsrq_encode_workspace_bytes(ctypes.byref(make_shape(N, D, d, K, M)),
                                                       ctypes.byref(n)), "encode_workspace_bytes")
    return int(n.value)


# ------------------------------------------------------------ torch plumbing

def _torch():
    import torch
    return torch


def _ptr(t) -> Optional[int]:
    return None if t is None else int(t.data_ptr())


def _stream_handle(stream) -> Optional[int]:
    torch = _torch()
    s = torch.cuda.current_stream() if stream is None else stream
    return int(s.cuda_stream) or None


def _dtype_code(t) -> int:
    torch = _torch()
    if t.dtype == torch.float16:
        return GSRQ_F16
    if t.dtype == torch.float32:
        return GSRQ_F32
    raise TypeError(f"unsupported dtype {t.dtype}; float16 or float32 expected")


def _rows(X):
    if X.dim() != 2 or X.stride(1) != 1:
        raise ValueError("X must be a 2-D tensor with unit column stride")
    return X.shape[0], X.shape[1], X.stride(0)


def _need(t, name, dtypes, device, shape=None):
    """Check a tensor argument passed as a dense pointer: dtype, device,
    contiguity and (optionally) shape; None passes."""
    if t is None:
        return
    if t.dtype not in dtypes:
        raise TypeError(f"{name} must be {' or '.join(str(d) for d in dtypes)}, not {t.dtype}")
    if t.device != device:
        raise ValueError(f"{name} is on {t.device}, expected {device}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if shape is not None and t.numel() != int(np.prod(shape)):
        raise ValueError(f"{name} has {t.numel()} elements, expected {tuple(shape)}")


def _workspace(nbytes, device, workspace):
    torch = _torch()
    if workspace is not None:
        if workspace.numel() * workspace.element_size() < nbytes:
            raise ValueError("workspace too small")
        return workspace
    # torch's caching allocator returns 512-byte aligned blocks
    return torch.empty(max(nbytes, 256), dtype=torch.uint8, device=device)


@dataclass
class TrainResult:
    gain: object          # [G, K] float32
    shape: object         # [G, K, d] float32
    assign: object        # [G, N] int16 holding uint16 codes
    iters: object         # [G] int32
    trace: object         # [G, T] float64 or None
    residual: object      # [N, D] float32 or None
    seed_rows: object = None  # host table kept alive with the results


def train_stage(X, d, K, T, seed_rows=None, w=None, *, gain=None, shape=None, assign=None,
                resume=False, assign_in=False, no_early_stop=False, residual=False,
                trace=True, kmeans=False, check_inputs=False, workspace=None,
                stream=None) -> TrainResult:
    """One stage of weighted GSKM on device tensor X [N, D] (see gsrq_train_stage).

    residual: True for a new R_next tensor, or an [N, D] float32 tensor to
    write it into.  kmeans: the K-means baseline (GSRQ_KMEANS) instead of
    GSKM; its centroids are gain[:, :, None] * shape.  check_inputs: the
    device check of GSRQ_CHECK_INPUTS (weights, finite X, nonzero seeds;
    the call then waits for the stream)."""
    torch = _torch()
    lib = load_library()
    N, D, ldx = _rows(X)
    G = D // d if d > 0 and D % d == 0 else 0
    dev = X.device
    _need(w, "w", (torch.float32,), dev, (N,))
    _need(gain, "gain", (torch.float32,), dev, (G, K))
    _need(shape, "shape", (torch.float32,), dev, (G, K, d))
    _need(assign, "assign", (torch.int16, torch.uint16), dev, (G, N))
    if residual is not True and residual is not False and residual is not None:
        _need(residual, "residual", (torch.float32,), dev, (N, D))
    if gain is None:
        gain = torch.empty((max(G, 1), K), dtype=torch.float32, device=dev)
    if shape is None:
        shape = torch.empty((max(G, 1), K, d), dtype=torch.float32, device=dev)
    if assign is None:
        assign = torch.empty((max(G, 1), N), dtype=torch.int16, device=dev)
    iters = torch.empty(max(G, 1), dtype=torch.int32, device=dev)
    tr = torch.empty((max(G, 1), max(T, 1)), dtype=torch.float64, device=dev) if trace and T > 0 else None
    if residual is True:
        res = torch.empty((N, D), dtype=torch.float32, device=dev)
    else:   # False / None, or an [N, D] float32 output tensor
        res = residual if residual is not False else None
    seeds = None
    if seed_rows is not None:
        seeds = np.ascontiguousarray(np.asarray(seed_rows), dtype=np.int32)
    flags = ((GSRQ_RESUME if resume else 0) | (GSRQ_ASSIGN_IN if assign_in else 0)
             | (GSRQ_NO_EARLY_STOP if no_early_stop else 0) | (GSRQ_KMEANS if kmeans else 0)
             | (GSRQ_CHECK_INPUTS if check_inputs else 0))
    sh = make_shape(N, D, d, K, 1)
    n = ctypes.c_size_t(0)
    st = lib.gsrq_train_workspace_bytes(ctypes.byref(sh), ctypes.byref(n))
    _check(st, "gsrq_train_workspace_bytes")
    ws = _workspace(n.value, dev, workspace)
    st = lib.gsrq_train_stage(
        ctypes.byref(sh), _ptr(X), _dtype_code(X), ldx, _ptr(w), int(T),
        None if seeds is None else seeds.ctypes.data, flags, _ptr(gain), _ptr(shape),
        _ptr(res), _ptr(assign), _ptr(iters), _ptr(tr), _ptr(ws),
        ws.numel() * ws.element_size(), _stream_handle(stream))
    _check(st, "gsrq_train_stage")
    return TrainResult(gain, shape, assign, iters, tr, res, seeds)


def encode(X, gain, shape, *, codes=None, residual=False, workspace=None, stream=None):
    """Stage-fused encode of device tensor X [N, D] with codebooks
    gain [M, G, K], shape [M, G, K, d].  Returns (codes [N, W] int32 words
    holding uint32 bit fields, residual [N, D] float32 or None)."""
    torch = _torch()
    lib = load_library()
    N, D, ldx = _rows(X)
    M, G, K = gain.shape
    d = shape.shape[-1]
    _need(gain, "gain", (torch.float32,), X.device)
    _need(shape, "shape", (torch.float32,), X.device, (M, G, K, d))
    sh = make_shape(N, D, d, K, M)
    W = int(lib.gsrq_code_words(ctypes.byref(sh)))
    _need(codes, "codes", (torch.int32, torch.uint32), X.device, (N, max(W, 1)))
    if codes is None:
        codes = torch.empty((N, max(W, 1)), dtype=torch.int32, device=X.device)
    res = torch.empty((N, D), dtype=torch.float32, device=X.device) if residual else None
    n = ctypes.c_size_t(0)
    _check(lib.gsrq_encode_workspace_bytes(ctypes.byref(sh), ctypes.byref(n)),
           "gsrq_encode_workspace_bytes")
    ws = _workspace(n.value, X.device, workspace)
    st = lib.gsrq_encode(ctypes.byref(sh), _ptr(X), _dtype_code(X), ldx, _ptr(gain),
                         _ptr(shape), _ptr(codes), _ptr(res), _ptr(ws),
                         ws.numel() * ws.element_size(), _stream_handle(stream))
    _check(st, "gsrq_encode")
    return codes, res


@dataclass
class Prepared:
    """A prepared codebook (gsrq_encode_prepare): the device buffer and the
    shape it was built for."""
    buf: object
    D: int
    d: int
    K: int
    M: int


def prepare_codebook(gain, shape, *, stream=None) -> Prepared:
    """Prepared codebook of gain [M, G, K], shape [M, G, K, d] (narrow
    family, d <= 8, K <= 256) for encode_prepared."""
    torch = _torch()
    lib = load_library()
    M, G, K = gain.shape
    d = shape.shape[-1]
    _need(gain, "gain", (torch.float32,), gain.device)
    _need(shape, "shape", (torch.float32,), gain.device, (M, G, K, d))
    sh = make_shape(1, G * d, d, K, M)
    n = ctypes.c_size_t(0)
    _check(lib.gsrq_prepared_bytes(ctypes.byref(sh), ctypes.byref(n)), "gsrq_prepared_bytes")
    buf = torch.empty(n.value, dtype=torch.uint8, device=gain.device)
    _check(lib.gsrq_encode_prepare(ctypes.byref(sh), _ptr(gain), _ptr(shape), _ptr(buf), n.value,
                                   _stream_handle(stream)), "gsrq_encode_prepare")
    return Prepared(buf, G * d, d, K, M)


def encode_prepared(X, prep: Prepared, *, codes=None, residual=False, stream=None):
    """encode() with a prepared codebook (no operand-table build per call)."""
    torch = _torch()
    lib = load_library()
    N, D, ldx = _rows(X)
    if D != prep.D:
        raise ValueError("X does not match the prepared codebook's vector length")
    sh = make_shape(N, D, prep.d, prep.K, prep.M)
    W = int(lib.gsrq_code_words(ctypes.byref(sh)))
    if codes is None:
        codes = torch.empty((N, max(W, 1)), dtype=torch.int32, device=X.device)
    _need(codes, "codes", (torch.int32, torch.uint32), X.device, (N, max(W, 1)))
    res = torch.empty((N, D), dtype=torch.float32, device=X.device) if residual else None
    st = lib.gsrq_encode_prepared(ctypes.byref(sh), _ptr(X), _dtype_code(X), ldx, _ptr(prep.buf),
                                  _ptr(codes), _ptr(res), _stream_handle(stream))
    _check(st, "gsrq_encode_prepared")
    return codes, res


def decode(codes, gain, shape, D, M_use=None, *, out_dtype=None, out=None, stream=None):
    """Gather-sum decode of packed codes [N, W] with codebooks gain [M, G, K],
    shape [M, G, K, d] into [N, D] (float16 by default)."""
    torch = _torch()
    lib = load_library()
    M, G, K = gain.shape
    d = shape.shape[-1]
    N = codes.shape[0]
    M_use = M if M_use is None else int(M_use)
    dev = codes.device
    _need(codes, "codes", (torch.int32, torch.uint32), dev)
    _need(gain, "gain", (torch.float32,), dev)
    _need(shape, "shape", (torch.float32,), dev, (M, G, K, d))
    if out is None:
        out = torch.empty((N, D), dtype=out_dtype or torch.float16, device=dev)
    elif out.dim() != 2 or out.stride(1) != 1 or out.device != dev or tuple(out.shape) != (N, D):
        raise ValueError("out must be an [N, D] tensor with unit column stride on the codes' device")
    sh = make_shape(N, D, d, K, M)
    st = lib.gsrq_decode(ctypes.byref(sh), _ptr(codes), M_use, _ptr(gain), _ptr(shape),
                         _ptr(out), _dtype_code(out), out.stride(0), _stream_handle(stream))
    _check(st, "gsrq_decode")
    return out


def row_weights(grad=None, *, norms=None, tau=1.0, stream=None):
    """Per-token weights of Sec. 5.3 / Appendix B (see gsrq_row_weights):
    from gradient rows grad [N, D] (float16/float32), or from precomputed
    norms [N] float32 when grad is None.  Returns (w [N], norms [N],
    stats [2] float64 = (median, lambda))."""
    torch = _torch()
    lib = load_library()
    if grad is not None:
        N, D, ldg = _rows(grad)
        dev = grad.device
        if norms is None:
            norms = torch.empty(N, dtype=torch.float32, device=dev)
        dt = _dtype_code(grad)
    else:
        if norms is None:
            raise ValueError("either grad or norms is needed")
        N, D, ldg, dev, dt = norms.shape[0], 0, 0, norms.device, GSRQ_F32
    w = torch.empty(N, dtype=torch.float32, device=dev)
    stats = torch.empty(2, dtype=torch.float64, device=dev)
    st = lib.gsrq_row_weights(_ptr(grad), dt, N, D, ldg, float(tau), _ptr(norms), _ptr(w),
                              _ptr(stats), _stream_handle(stream))
    _check(st, "gsrq_row_weights")
    return w, norms, stats


GSRQ_ATTN_TABLES_READY = 1


def make_attn_shape(B, cap, Hq, Hkv, head_dim=128, rope_base=500000.0, scale=None,
                    flags=0) -> AttnShape:
    scale = 1.0 / math.sqrt(head_dim) if scale is None else float(scale)
    return AttnShape(int(B), int(cap), int(Hq), int(Hkv), int(head_dim), float(rope_base), scale,
                     int(flags))


def attn_workspace_bytes(B, cap, Hq, Hkv, head_dim=128, *, d=8, M=1) -> int:
    """Workspace of gsrq_attn_decode for codes of subvector length d and M
    stages (d = 8, M = 1: the 1-bit layout; d = head_dim: residual-coded)."""
    n = ctypes.c_size_t()
    sh = make_attn_shape(B, cap, Hq, Hkv, head_dim)
    kv = make_shape(B * cap, Hkv * head_dim, d, 256, M)
    _check(load_library().gsrq_attn_workspace_bytes_kv(ctypes.byref(sh), ctypes.byref(kv),
                                                       ctypes.byref(n)),
           "gsrq_attn_workspace_bytes_kv")
    return int(n.value)


ATTN_NOALLOC_BYTES = 16 << 20


def attn_decode(k_codes, v_codes, seq_len, k_gain, k_shape, v_gain, v_shape, q, *,
                rope_base=500000.0, scale=None, out=None, workspace=None, stream=None,
                tables_ready=False, noalloc=False):
    """One decoding step of attention over coded caches (see gsrq_attn_decode).
    k_codes, v_codes [B, cap, W] packed codes; seq_len [B] int32; codebooks
    [M, G, 256] / [M, G, 256, d] (the 1-bit layout d = 8, M = 1, or the
    residual-coded one d = 128, M <= 16); q [B, Hq, 128] (float16/float32).  Returns
    out [B, Hq, 128] float32.  tables_ready: the given workspace holds the
    tables of these codebooks from an earlier call (GSRQ_ATTN_TABLES_READY).
    noalloc: gsrq_attn_decode_noalloc (the library's per-GPU scratch instead
    of a workspace; workspace must then be None)."""
    torch = _torch()
    lib = load_library()
    B, cap, W = k_codes.shape
    Hq, hd = q.shape[1], q.shape[2]
    M, G, K = k_gain.shape
    d = k_shape.shape[-1]
    D = G * d
    Hkv = D // hd
    for t in (k_codes, v_codes, seq_len, k_gain, k_shape, v_gain, v_shape, q):
        if not t.is_contiguous():
            raise ValueError("attn_decode expects contiguous tensors")
    if tuple(v_codes.shape) != (B, cap, W) or q.shape[0] != B or seq_len.numel() != B:
        raise ValueError("inconsistent shapes")
    if seq_len.dtype != torch.int32:
        raise TypeError("seq_len must be int32")
    ash = make_attn_shape(B, cap, Hq, Hkv, hd, rope_base, scale,
                          GSRQ_ATTN_TABLES_READY if tables_ready else 0)
    sh = make_shape(B * cap, D, d, K, M)
    if out is None:
        out = torch.empty((B, Hq, hd), dtype=torch.float32, device=q.device)
    if noalloc:
        if workspace is not None:
            raise ValueError("noalloc takes no workspace")
        st = lib.gsrq_attn_decode_noalloc(
            ctypes.byref(ash), ctypes.byref(sh), _ptr(k_codes), _ptr(v_codes), _ptr(seq_len),
            _ptr(k_gain), _ptr(k_shape), _ptr(v_gain), _ptr(v_shape), _ptr(q), _dtype_code(q),
            _ptr(out), _stream_handle(stream))
        _check(st, "gsrq_attn_decode_noalloc")
        return out
    n = ctypes.c_size_t()
    _check(lib.gsrq_attn_workspace_bytes_kv(ctypes.byref(ash), ctypes.byref(sh), ctypes.byref(n)),
           "gsrq_attn_workspace_bytes_kv")
    ws = _workspace(n.value, q.device, workspace)
    st = lib.gsrq_attn_decode(ctypes.byref(ash), ctypes.byref(sh), _ptr(k_codes), _ptr(v_codes),
                              _ptr(seq_len), _ptr(k_gain), _ptr(k_shape), _ptr(v_gain),
                              _ptr(v_shape), _ptr(q), _dtype_code(q), _ptr(out), _ptr(ws),
                              ws.numel() * ws.element_size(), _stream_handle(stream))
    _check(st, "gsrq_attn_decode")
    return out
