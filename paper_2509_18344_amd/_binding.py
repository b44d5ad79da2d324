"""ctypes binding of libsubspec.so: one Python function per C entry point, with the
same name and argument order.  Tensors are passed as their data pointers; a
``stream`` of None means torch's current stream on the current device."""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_NAME = "libsubspec.so"

SUBSPEC_PATH_AUTO = 0
SUBSPEC_PATH_GEMV = 1
SUBSPEC_PATH_MFMA = 2
SUBSPEC_PATH_MFMA16 = 3
SUBSPEC_PATH_MFMA32 = 4
SUBSPEC_NOALLOC_SCRATCH_BYTES = 32 << 20  # the fixed per-device scratch of subspec_qlinear_noalloc

_STATUS = {0: "OK", -1: "EINVAL", -2: "EUNSUPPORTED", -3: "EHIP", -4: "ECAPTURE"}


class SubspecError(RuntimeError):
    def __init__(self, fn: str, status: int, message: str):
        super().__init__(f"{fn} failed with {_STATUS.get(status, status)}: {message}")
        self.status = status
        self.message = message


class _Plan(ctypes.Structure):
    _fields_ = [("path", ctypes.c_int), ("mfma_rows", ctypes.c_int), ("rows", ctypes.c_int),
                ("tiles_per_wave", ctypes.c_int),
                ("waves", ctypes.c_int),
                ("chunk_blocks", ctypes.c_int), ("ring_chunks", ctypes.c_int), ("col_groups", ctypes.c_int),
                ("full_groups", ctypes.c_int),
                ("splits", ctypes.c_int), ("blocks_per_split", ctypes.c_int),
                ("grid", ctypes.c_int), ("workspace_bytes", ctypes.c_size_t),
                ("teams", ctypes.c_int), ("row_blocks", ctypes.c_int)]


class SubspecProj(ctypes.Structure):
    _fields_ = [("x", ctypes.c_void_p), ("qweight", ctypes.c_void_p), ("scales", ctypes.c_void_p),
                ("zeros", ctypes.c_void_p), ("y", ctypes.c_void_p), ("N", ctypes.c_int),
                ("K", ctypes.c_int)]


_lib = None


def library_path() -> str:
    return os.path.join(_HERE, _LIB_NAME)


def load_library():
    """Load libsubspec.so (once).  Raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    path = library_path()
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with __graft_entry__.build() "
                           "(or python -m paper_2509_18344_amd.build)")
    lib = ctypes.CDLL(path)
    P, I, S = ctypes.c_void_p, ctypes.c_int, ctypes.c_size_t
    sig = {
        "subspec_qpack_bytes": (S, [I, I, I]),
        "subspec_quantize": (I, [P, I, I, I, I, P, P, P, P]),
        "subspec_qpack": (I, [P, I, I, I, P, P]),
        "subspec_quantize_hqq": (I, [P, I, I, I, I, P, P, P, P]),
        "subspec_qpack_host": (I, [P, I, I, I, P]),
        "subspec_qlinear": (I, [P, P, P, P, I, I, I, I, I, P, P]),
        "subspec_qlinear_path": (I, [P, P, P, P, I, I, I, I, I, P, I, P]),
        "subspec_qlinear_noalloc": (I, [P, P, P, P, I, I, I, I, I, P, P]),
        "subspec_qlinear_plan": (I, [I, I, I, I, I, I, ctypes.POINTER(_Plan)]),
        "subspec_qdequant": (I, [P, P, P, I, I, I, I, P, P, P]),
        "subspec_reserve": (I, [S]),
        "subspec_workspace_info": (I, [ctypes.POINTER(ctypes.c_size_t), ctypes.POINTER(ctypes.c_int),
                                       ctypes.POINTER(ctypes.c_ulonglong)]),
        "subspec_stack_forward": (I, [ctypes.POINTER(SubspecProj), I, I, I, I, P]),
        "subspec_stack_capture": (I, [ctypes.POINTER(SubspecProj), I, I, I, I, P,
                                      ctypes.POINTER(ctypes.c_void_p)]),
        "subspec_graph_launch": (I, [P, P]),
        "subspec_graph_destroy": (I, [P]),
        "subspec_tree_expand": (I, [P, P, I, I, ctypes.c_float, I, P, P, P, P]),
        "subspec_tree_workspace_bytes": (S, [I, I, I]),
        "subspec_tree_plan": (I, [I, I, I, P, P, P]),
        "subspec_tree_attention": (I, [P, P, P, P, P, P, I, I, I, I, I, I, ctypes.c_float, P, P]),
        "subspec_tree_attention_workspace_bytes": (S, [I, I, I, I, I]),
        "subspec_tree_attention_plan": (I, [I, I, I, I, I, P, P]),
        "subspec_prefetch_create": (I, [S, I, ctypes.POINTER(ctypes.c_void_p)]),
        "subspec_prefetch_destroy": (I, [P]),
        "subspec_prefetch_begin": (I, [P, P, S, ctypes.POINTER(ctypes.c_longlong)]),
        "subspec_prefetch_acquire": (I, [P, ctypes.c_longlong, P, ctypes.POINTER(ctypes.c_void_p)]),
        "subspec_prefetch_release": (I, [P, ctypes.c_longlong, P]),
        "subspec_last_error": (ctypes.c_char_p, []),
    }
    for name, (res, args) in sig.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    _lib = lib
    return lib


def _ptr(t):
    """Data pointer of a torch tensor / numpy array, or an int address, or None."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    if hasattr(t, "data_ptr"):
        return t.data_ptr()
    if hasattr(t, "ctypes"):
        return t.ctypes.data
    raise TypeError(f"cannot take the address of {type(t)}")


def _stream(s):
    if s is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(s, int):
        return s
    return s.cuda_stream


def _check(fn: str, status: int) -> int:
    if status != 0:
        raise SubspecError(fn, status, subspec_last_error())
    return status


def subspec_last_error() -> str:
    return load_library().subspec_last_error().decode()


def subspec_qpack_bytes(bits: int, N: int, K: int) -> int:
    return int(load_library().subspec_qpack_bytes(bits, N, K))


def subspec_quantize(w, bits, group, N, K, codes, scales, zeros, stream=None) -> int:
    return _check("subspec_quantize", load_library().subspec_quantize(
        _ptr(w), bits, group, N, K, _ptr(codes), _ptr(scales), _ptr(zeros), _stream(stream)))


def subspec_quantize_hqq(w, bits, group, N, K, codes, scales, zeros, stream=None) -> int:
    return _check("subspec_quantize_hqq", load_library().subspec_quantize_hqq(
        _ptr(w), bits, group, N, K, _ptr(codes), _ptr(scales), _ptr(zeros), _stream(stream)))


def subspec_qpack(codes, bits, N, K, qweight, stream=None) -> int:
    return _check("subspec_qpack", load_library().subspec_qpack(
        _ptr(codes), bits, N, K, _ptr(qweight), _stream(stream)))


def subspec_qpack_host(codes, bits, N, K, qweight) -> int:
    return _check("subspec_qpack_host", load_library().subspec_qpack_host(
        _ptr(codes), bits, N, K, _ptr(qweight)))


def subspec_qlinear(x, qweight, scales, zeros, bits, group, M, N, K, y, stream=None) -> int:
    return _check("subspec_qlinear", load_library().subspec_qlinear(
        _ptr(x), _ptr(qweight), _ptr(scales), _ptr(zeros), bits, group, M, N, K, _ptr(y),
        _stream(stream)))


def subspec_qlinear_noalloc(x, qweight, scales, zeros, bits, group, M, N, K, y, stream=None) -> int:
    return _check("subspec_qlinear_noalloc", load_library().subspec_qlinear_noalloc(
        _ptr(x), _ptr(qweight), _ptr(scales), _ptr(zeros), bits, group, M, N, K, _ptr(y), _stream(stream)))


def subspec_qlinear_path(x, qweight, scales, zeros, bits, group, M, N, K, y, path,
                         stream=None) -> int:
    return _check("subspec_qlinear_path", load_library().subspec_qlinear_path(
        _ptr(x), _ptr(qweight), _ptr(scales), _ptr(zeros), bits, group, M, N, K, _ptr(y), path,
        _stream(stream)))


def subspec_qlinear_plan(M, N, K, bits, group, path=SUBSPEC_PATH_AUTO) -> dict:
    p = _Plan()
    _check("subspec_qlinear_plan", load_library().subspec_qlinear_plan(
        M, N, K, bits, group, path, ctypes.byref(p)))
    return {name: getattr(p, name) for name, _ in _Plan._fields_}


def subspec_qdequant(qweight, scales, zeros, bits, group, N, K, w_f32, w_bf16,
                     stream=None) -> int:
    return _check("subspec_qdequant", load_library().subspec_qdequant(
        _ptr(qweight), _ptr(scales), _ptr(zeros), bits, group, N, K, _ptr(w_f32), _ptr(w_bf16),
        _stream(stream)))


def subspec_reserve(nbytes: int) -> int:
    return _check("subspec_reserve", load_library().subspec_reserve(nbytes))


def subspec_workspace_info() -> dict:
    """The calling device's workspace: bytes, retired buffers held, allocations so far."""
    b, r, a = ctypes.c_size_t(), ctypes.c_int(), ctypes.c_ulonglong()
    _check("subspec_workspace_info", load_library().subspec_workspace_info(
        ctypes.byref(b), ctypes.byref(r), ctypes.byref(a)))
    return {"bytes": int(b.value), "retired": int(r.value), "allocations": int(a.value)}


def _projs(projs):
    """A ctypes array of subspec_proj from dicts with keys x, qweight, scales, zeros,
    y, N, K (tensors or addresses)."""
    arr = (SubspecProj * len(projs))()
    for i, p in enumerate(projs):
        arr[i] = SubspecProj(_ptr(p["x"]), _ptr(p["qweight"]), _ptr(p["scales"]), _ptr(p["zeros"]),
                             _ptr(p["y"]), int(p["N"]), int(p["K"]))
    return arr


def subspec_stack_forward(projs, bits, group, M, stream=None) -> int:
    arr = _projs(projs)
    return _check("subspec_stack_forward", load_library().subspec_stack_forward(
        arr, len(projs), bits, group, M, _stream(stream)))


def subspec_stack_capture(projs, bits, group, M, stream) -> int:
    """Returns the graph handle (an address) of the captured sequence."""
    arr = _projs(projs)
    h = ctypes.c_void_p()
    _check("subspec_stack_capture", load_library().subspec_stack_capture(
        arr, len(projs), bits, group, M, _stream(stream), ctypes.byref(h)))
    return h.value


def subspec_graph_launch(graph, stream=None) -> int:
    return _check("subspec_graph_launch", load_library().subspec_graph_launch(graph, _stream(stream)))


def subspec_graph_destroy(graph) -> int:
    return _check("subspec_graph_destroy", load_library().subspec_graph_destroy(graph))


def subspec_tree_expand(logits, parent_logp, R, V, temperature, k, parent_out, token_out,
                        score_out, stream=None) -> int:
    return _check("subspec_tree_expand", load_library().subspec_tree_expand(
        _ptr(logits), _ptr(parent_logp), R, V, float(temperature), k, _ptr(parent_out),
        _ptr(token_out), _ptr(score_out), _stream(stream)))


def subspec_tree_workspace_bytes(R, V, k) -> int:
    return int(load_library().subspec_tree_workspace_bytes(R, V, k))


def subspec_tree_attention(q, k_cache, v_cache, k_new, v_new, mask, M, Hq, Hkv, S, P, T, scale, out,
                           stream=None):
    return _check("subspec_tree_attention", load_library().subspec_tree_attention(
        _ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(k_new), _ptr(v_new), _ptr(mask), M, Hq, Hkv, S, P, T,
        scale, _ptr(out), _stream(stream)))


def subspec_tree_attention_workspace_bytes(M, Hq, Hkv, P, T) -> int:
    return int(load_library().subspec_tree_attention_workspace_bytes(M, Hq, Hkv, P, T))


def subspec_tree_attention_plan(M, Hq, Hkv, P, T):
    """(splits, tiles_per_split) of the tree-attention launch."""
    s, t = ctypes.c_int(), ctypes.c_int()
    _check("subspec_tree_attention_plan", load_library().subspec_tree_attention_plan(
        M, Hq, Hkv, P, T, ctypes.byref(s), ctypes.byref(t)))
    return s.value, t.value


class Prefetcher:
    """The library's cross-layer weight prefetcher (a ring of `slots` device buffers of
    `slot_bytes`, one copy stream): begin(host) -> ticket, acquire(ticket, stream) ->
    device address, release(ticket, stream).  Host sources must be pinned."""

    def __init__(self, slot_bytes: int, slots: int):
        h = ctypes.c_void_p()
        _check("subspec_prefetch_create", load_library().subspec_prefetch_create(slot_bytes, slots, ctypes.byref(h)))
        self._h = h.value

    def begin(self, host, nbytes=None) -> int:
        if nbytes is None:
            nbytes = host.numel() * host.element_size()
        t = ctypes.c_longlong()
        _check("subspec_prefetch_begin", load_library().subspec_prefetch_begin(self._h, _ptr(host), nbytes,
                                                                               ctypes.byref(t)))
        return t.value

    def acquire(self, ticket: int, stream=None) -> int:
        p = ctypes.c_void_p()
        _check("subspec_prefetch_acquire", load_library().subspec_prefetch_acquire(self._h, ticket, _stream(stream),
                                                                                   ctypes.byref(p)))
        return p.value

    def release(self, ticket: int, stream=None) -> None:
        _check("subspec_prefetch_release", load_library().subspec_prefetch_release(self._h, ticket, _stream(stream)))

    def close(self) -> None:
        if self._h:
            _check("subspec_prefetch_destroy", load_library().subspec_prefetch_destroy(self._h))
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def subspec_tree_plan(R, V, k):
    """(chunks, chunk_len, list_len) of the expansion launch for (R, V, k)."""
    c, n, l = ctypes.c_int(), ctypes.c_int(), ctypes.c_int()
    _check("subspec_tree_plan", load_library().subspec_tree_plan(
        R, V, k, ctypes.byref(c), ctypes.byref(n), ctypes.byref(l)))
    return c.value, n.value, l.value
