"""Thin ctypes binding of libchronostitch.so (argument marshalling only).

Every function has the name of the C entry point it calls.  Device buffers
are torch tensors (their data_ptr() is passed through); host arrays are numpy
arrays; the stream is torch's current stream unless one is given.  All the
computation happens in the library's HIP kernels: if the library cannot be
loaded, every call raises.
"""
import ctypes
import os

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "lib", "libchronostitch.so")

CS_OK, CS_ERR_INVALID_ARGUMENT, CS_ERR_UNSUPPORTED, CS_ERR_WORKSPACE_TOO_SMALL, CS_ERR_HIP = range(5)
CS_F32, CS_BF16 = 0, 1
EXPORTS = ("compose_rebase_k", "score_deviation_topk_workspace", "score_deviation_topk",
           "selective_attend_scatter_workspace", "selective_attend_scatter", "cs_last_error",
           "cs_trace_enable", "cs_trace_only", "cs_trace_collect", "cs_trace_count", "cs_trace_get",
           "cs_trace_reset")


class CsError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"chronostitch error {code}: {msg}")
        self.code = code


class Geometry(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("n_q_heads", ctypes.c_int32),
                ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("sections", ctypes.c_int32 * 3), ("dtype", ctypes.c_int32),
                ("rope_base", ctypes.c_double), ("inv_freq", ctypes.POINTER(ctypes.c_double)),
                ("n_tokens", ctypes.c_int64), ("n_chunks", ctypes.c_int32),
                ("chunk_start", ctypes.POINTER(ctypes.c_int64))]


_lib = None


def lib():
    """The loaded library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build()")
        L = ctypes.CDLL(LIB_PATH)
        vp, i32, i64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
        G = ctypes.POINTER(Geometry)
        L.compose_rebase_k.argtypes = [G, vp, vp, vp, vp, vp]
        L.compose_rebase_k_tokens.argtypes = [G, vp, vp, vp]
        L.score_deviation_topk_workspace.argtypes = [G, ctypes.POINTER(sz)]
        L.score_deviation_topk.argtypes = [G, vp, i32, vp, ctypes.c_double, vp, vp,
                                           ctypes.POINTER(i64), vp, sz, vp]
        L.selective_attend_scatter_workspace.argtypes = [G, i64, i32, ctypes.POINTER(sz)]
        L.selective_attend_scatter_rope_workspace.argtypes = [G, i64, i32, ctypes.POINTER(sz)]
        L.selective_attend_scatter_rope.argtypes = [G, vp, vp, i32, i32, vp, i64, vp, vp, vp, vp, vp, vp,
                                                    vp, sz, vp]
        L.selective_attend_scatter.argtypes = [G, vp, vp, i32, i32, vp, i64, vp, vp, vp, vp, vp,
                                               vp, sz, vp]
        L.selective_attend_scatter_noalloc.argtypes = [G, vp, vp, i32, i32, vp, i64, vp, vp, vp, vp, vp, vp]
        L.compose_rebase_k_paged.argtypes = [G, vp, vp, vp, vp, vp]
        L.compose_rebase_k_tokens_paged.argtypes = [G, vp, vp, vp]
        L.compose_load_rebase_k_paged.argtypes = [G, vp, vp, vp, vp, vp, vp, vp]
        L.score_deviation_topk_paged.argtypes = [G, vp, i32, vp, ctypes.c_double, vp, vp,
                                                 ctypes.POINTER(i64), vp, sz, vp]
        L.selective_attend_scatter_paged.argtypes = [G, vp, vp, i32, i32, vp, i64, vp, vp, vp, vp, vp,
                                                     vp, sz, vp]
        L.selective_attend_scatter_rope_paged.argtypes = [G, vp, vp, i32, i32, vp, i64, vp, vp, vp, vp, vp,
                                                          vp, vp, sz, vp]
        L.cs_last_error.restype = ctypes.c_char_p
        L.cs_trace_enable.argtypes = [i32]
        L.cs_trace_only.argtypes = [ctypes.c_char_p]
        L.cs_trace_get.argtypes = [i32, ctypes.POINTER(ctypes.c_char_p), ctypes.POINTER(i64),
                                   ctypes.POINTER(ctypes.c_double)]
        L.cs_trace_count.restype = i32
        for name in ("compose_rebase_k", "compose_rebase_k_tokens", "score_deviation_topk_workspace",
                     "score_deviation_topk",
                     "selective_attend_scatter_workspace", "selective_attend_scatter",
                     "selective_attend_scatter_noalloc",
                     "selective_attend_scatter_rope_workspace", "selective_attend_scatter_rope",
                     "compose_rebase_k_paged", "compose_rebase_k_tokens_paged", "score_deviation_topk_paged",
                     "compose_load_rebase_k_paged",
                     "selective_attend_scatter_paged", "selective_attend_scatter_rope_paged",
                     "cs_trace_enable", "cs_trace_only", "cs_trace_collect", "cs_trace_get"):
            getattr(L, name).restype = ctypes.c_int
        _lib = L
    return _lib


def _check(code):
    if code != CS_OK:
        raise CsError(code, lib().cs_last_error().decode())


class Geo:
    """Owns a cs_geometry and the host arrays it points to."""

    def __init__(self, n_layers, n_q_heads, n_kv_heads, head_dim, sections, dtype, chunk_start,
                 rope_base=1.0e6, inv_freq=None):
        self.chunk_start = np.ascontiguousarray(chunk_start, dtype=np.int64)
        self.inv_freq = None if inv_freq is None else np.ascontiguousarray(inv_freq, dtype=np.float64)
        self.g = Geometry()
        self.g.n_layers, self.g.n_q_heads, self.g.n_kv_heads, self.g.head_dim = (
            n_layers, n_q_heads, n_kv_heads, head_dim)
        self.g.sections = (ctypes.c_int32 * 3)(*sections)
        self.g.dtype = {"bf16": CS_BF16, "f32": CS_F32}.get(dtype, dtype)
        self.g.rope_base = rope_base
        self.g.inv_freq = (self.inv_freq.ctypes.data_as(ctypes.POINTER(ctypes.c_double))
                           if self.inv_freq is not None else None)
        self.g.n_tokens = int(self.chunk_start[-1])
        self.g.n_chunks = len(self.chunk_start) - 1
        self.g.chunk_start = self.chunk_start.ctypes.data_as(ctypes.POINTER(ctypes.c_int64))

    @classmethod
    def from_workload(cls, w):
        return cls(w.n_layers, w.n_q_heads, w.n_kv_heads, w.head_dim, w.sections, w.dtype,
                   w.chunk_start, w.base)

    @property
    def ref(self):
        return ctypes.byref(self.g)


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is not None:
        return ctypes.c_void_p(stream)
    import torch
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def compose_rebase_k(geo, k_cache, chunk_offsets, local_coords=None, want_global=False, stream=None):
    """Re-base k_cache in place; returns global coords [T,3] (int32) when asked."""
    off = np.ascontiguousarray(chunk_offsets, dtype=np.int32)
    loc = None if local_coords is None else np.ascontiguousarray(local_coords, dtype=np.int32)
    glob = np.empty_like(loc) if (want_global and loc is not None) else None
    _check(lib().compose_rebase_k(geo.ref, _ptr(k_cache), off.ctypes.data_as(ctypes.c_void_p),
                                  None if loc is None else loc.ctypes.data_as(ctypes.c_void_p),
                                  None if glob is None else glob.ctypes.data_as(ctypes.c_void_p),
                                  _stream(stream)))
    return glob


def compose_rebase_k_tokens(geo, k_cache, token_offsets, stream=None):
    """Re-base k_cache in place by a per-token offset (DEVICE int32 [T, 3] tensor)."""
    _check(lib().compose_rebase_k_tokens(geo.ref, _ptr(k_cache), _ptr(token_offsets), _stream(stream)))


def score_deviation_topk_workspace(geo):
    n = ctypes.c_size_t(0)
    _check(lib().score_deviation_topk_workspace(geo.ref, ctypes.byref(n)))
    return n.value


def score_deviation_topk(geo, k_cache, score_layer, k_fresh, rho, scores, sel_idx, workspace=None,
                         stream=None):
    """Scores later-chunk tokens and selects the top rho; returns n_sel."""
    k = ctypes.c_int64(0)
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib().score_deviation_topk(geo.ref, _ptr(k_cache), int(score_layer), _ptr(k_fresh),
                                      float(rho), _ptr(scores), _ptr(sel_idx), ctypes.byref(k),
                                      _ptr(workspace), ws_bytes, _stream(stream)))
    return k.value


def selective_attend_scatter_workspace(geo, n_sel, n_layers_per_call):
    n = ctypes.c_size_t(0)
    _check(lib().selective_attend_scatter_workspace(geo.ref, int(n_sel), int(n_layers_per_call),
                                                    ctypes.byref(n)))
    return n.value


def selective_attend_scatter(geo, k_cache, v_cache, layer_begin, layer_end, sel_idx, n_sel, q_fresh,
                             k_fresh, v_fresh, out, lse=None, workspace=None, stream=None):
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib().selective_attend_scatter(geo.ref, _ptr(k_cache), _ptr(v_cache), int(layer_begin),
                                          int(layer_end), _ptr(sel_idx), int(n_sel), _ptr(q_fresh),
                                          _ptr(k_fresh), _ptr(v_fresh), _ptr(out), _ptr(lse),
                                          _ptr(workspace), ws_bytes, _stream(stream)))


def selective_attend_scatter_noalloc(geo, k_cache, v_cache, layer_begin, layer_end, sel_idx, n_sel, q_fresh,
                                     k_fresh, v_fresh, out, lse=None, stream=None):
    """selective_attend_scatter with the library's own per-GPU scratch array (no workspace)."""
    _check(lib().selective_attend_scatter_noalloc(geo.ref, _ptr(k_cache), _ptr(v_cache), int(layer_begin),
                                                  int(layer_end), _ptr(sel_idx), int(n_sel), _ptr(q_fresh),
                                                  _ptr(k_fresh), _ptr(v_fresh), _ptr(out), _ptr(lse),
                                                  _stream(stream)))


# ---------------------------------------------------------------- tracing
def cs_trace_enable(on=True):
    _check(lib().cs_trace_enable(1 if on else 0))


def cs_trace_only(names=None):
    """Trace only the kernels named (an iterable of names, or None for all)."""
    _check(lib().cs_trace_only(None if names is None else ",".join(names).encode()))


def cs_trace_reset():
    lib().cs_trace_reset()


def cs_trace_collect():
    """Synchronises pending trace events; returns {kernel: (launches, total_ms)}."""
    L = lib()
    _check(L.cs_trace_collect())
    out = {}
    for i in range(L.cs_trace_count()):
        name = ctypes.c_char_p()
        n = ctypes.c_int64()
        ms = ctypes.c_double()
        _check(L.cs_trace_get(i, ctypes.byref(name), ctypes.byref(n), ctypes.byref(ms)))
        out[name.value.decode()] = (n.value, ms.value)
    return out


def selective_attend_scatter_rope_workspace(geo, n_sel, n_layers_per_call):
    n = ctypes.c_size_t(0)
    _check(lib().selective_attend_scatter_rope_workspace(geo.ref, int(n_sel), int(n_layers_per_call),
                                                         ctypes.byref(n)))
    return n.value


def selective_attend_scatter_rope(geo, k_cache, v_cache, layer_begin, layer_end, sel_idx, n_sel, q_pre, k_pre,
                                  v_fresh, coords, out, lse=None, workspace=None, stream=None):
    """selective_attend_scatter on pre-rotary fresh Q/K, rotated at the global coordinates (DEVICE int32 [T, 3])."""
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib().selective_attend_scatter_rope(geo.ref, _ptr(k_cache), _ptr(v_cache), int(layer_begin),
                                               int(layer_end), _ptr(sel_idx), int(n_sel), _ptr(q_pre), _ptr(k_pre),
                                               _ptr(v_fresh), _ptr(coords), _ptr(out), _ptr(lse), _ptr(workspace),
                                               ws_bytes, _stream(stream)))


# ---------------------------------------------------------------- paged cache
def _chunks(ts):
    """HOST array of the chunk tensors' device pointers (None stays NULL)."""
    if ts is None:
        return None
    arr = (ctypes.c_void_p * max(1, len(ts)))(*[None if t is None else t.data_ptr() for t in ts])
    return arr


def compose_rebase_k_paged(geo, k_chunks, chunk_offsets, local_coords=None, want_global=False, stream=None):
    """compose_rebase_k on a cache held as one tensor per chunk ([L, H_kv, len_c, D] each)."""
    off = np.ascontiguousarray(chunk_offsets, dtype=np.int32)
    loc = None if local_coords is None else np.ascontiguousarray(local_coords, dtype=np.int32)
    glob = np.empty_like(loc) if (want_global and loc is not None) else None
    _check(lib().compose_rebase_k_paged(geo.ref, _chunks(k_chunks), off.ctypes.data_as(ctypes.c_void_p),
                                        None if loc is None else loc.ctypes.data_as(ctypes.c_void_p),
                                        None if glob is None else glob.ctypes.data_as(ctypes.c_void_p),
                                        _stream(stream)))
    return glob


def compose_load_rebase_k_paged(geo, k_chunks, v_chunks, k_host, v_host, chunk_offsets, copy_stream=None,
                                stream=None):
    """Copy each chunk's K and V from host tensors (page-locked for overlap) into the device chunk
    tensors on copy_stream, re-basing each chunk's keys on stream as soon as they have landed."""
    off = np.ascontiguousarray(chunk_offsets, dtype=np.int32)
    _check(lib().compose_load_rebase_k_paged(geo.ref, _chunks(k_chunks), _chunks(v_chunks), _chunks(k_host),
                                             _chunks(v_host), off.ctypes.data_as(ctypes.c_void_p),
                                             None if copy_stream is None else ctypes.c_void_p(copy_stream),
                                             _stream(stream)))


def compose_rebase_k_tokens_paged(geo, k_chunks, token_offsets, stream=None):
    _check(lib().compose_rebase_k_tokens_paged(geo.ref, _chunks(k_chunks), _ptr(token_offsets), _stream(stream)))


def score_deviation_topk_paged(geo, k_chunks, score_layer, k_fresh, rho, scores, sel_idx, workspace=None,
                               stream=None):
    k = ctypes.c_int64(0)
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib().score_deviation_topk_paged(geo.ref, _chunks(k_chunks), int(score_layer), _ptr(k_fresh),
                                            float(rho), _ptr(scores), _ptr(sel_idx), ctypes.byref(k),
                                            _ptr(workspace), ws_bytes, _stream(stream)))
    return k.value


def selective_attend_scatter_paged(geo, k_chunks, v_chunks, layer_begin, layer_end, sel_idx, n_sel, q_fresh,
                                   k_fresh, v_fresh, out, lse=None, workspace=None, stream=None):
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib().selective_attend_scatter_paged(geo.ref, _chunks(k_chunks), _chunks(v_chunks), int(layer_begin),
                                                int(layer_end), _ptr(sel_idx), int(n_sel), _ptr(q_fresh),
                                                _ptr(k_fresh), _ptr(v_fresh), _ptr(out), _ptr(lse),
                                                _ptr(workspace), ws_bytes, _stream(stream)))


def selective_attend_scatter_rope_paged(geo, k_chunks, v_chunks, layer_begin, layer_end, sel_idx, n_sel, q_pre,
                                        k_pre, v_fresh, coords, out, lse=None, workspace=None, stream=None):
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib().selective_attend_scatter_rope_paged(geo.ref, _chunks(k_chunks), _chunks(v_chunks),
                                                     int(layer_begin), int(layer_end), _ptr(sel_idx), int(n_sel),
                                                     _ptr(q_pre), _ptr(k_pre), _ptr(v_fresh), _ptr(coords),
                                                     _ptr(out), _ptr(lse), _ptr(workspace), ws_bytes,
                                                     _stream(stream)))
