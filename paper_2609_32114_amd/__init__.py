"""MI355X (gfx950) chunkwise delta-rule linear-attention prefill: GDN and KDA.

Thin Python binding over the C ABI of ``include/hagdn.h`` (``libhagdn.so``,
built in-tree by ``paper_2609_32114_amd.build``).  This module only marshals
arguments: it allocates outputs and the workspace with torch, passes raw device
pointers and torch's current HIP stream, and raises on a non-OK status.  Every
step of the computation runs in the library's HIP kernels; there is no CPU or
PyTorch fallback, and calls fail loudly when the library is missing.

    o, s_final = gdn_prefill(q, k, v, g, beta, initial_state=None,
                             cu_seqlens=None, scale=1.0, preprocess=0)
    o = gdn_decode(q1, k1, v1, g1, beta1, state_pool, slots=None, scale=1.0)

Layouts: q, k [T, Hqk, Dk]; v [T, Hv, Dv] (bf16 or fp32, all the same dtype);
g [T, Hv] fp32 (KDA: [T, Hv, Dk]); beta [T, Hv] fp32; initial_state
[N, Hv, Dk, Dv] fp32; cu_seqlens int32 [N+1] on the device (None: one
sequence of length T).  Returns o [T, Hv, Dv] in the input dtype and the final
state [N, Hv, Dk, Dv] fp32.  ``preprocess`` (PRE_* flags) makes the kernels
normalise raw q/k and map raw gate / beta projections as they load them.
The decode entry points advance one token per sequence and update a state
pool in place.
"""

from __future__ import annotations

import ctypes
import os

__all__ = ["gdn_prefill", "kda_prefill", "gdn_decode", "kda_decode", "workspace_size",
           "device_status", "library_path", "load_library", "profile_begin", "profile_end", "kernel_names", "set_segment_chunks",
           "set_overlap", "overlap_for",
           "segment_chunks", "segment_chunks_for", "workspace_region", "measure_copy", "measure_mfma",
           "HagdnError"]

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libhagdn.so")
_lib = None

HAGDN_F32, HAGDN_BF16 = 0, 1
DEV_OK, DEV_BAD_SEQLENS, DEV_WAIT_TIMEOUT = 0, 1, 2
# preprocessing flags (hagdn_pre_flags)
PRE_QK_L2NORM, PRE_GATE_SOFTPLUS, PRE_BETA_SIGMOID = 1, 2, 4
PRE_ALL = 7

_PREFILL_ARGS = ([ctypes.c_void_p] * 7 + [ctypes.c_int] * 6 + [ctypes.c_float, ctypes.c_int])
_PREFILL_TAIL = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]
_DECODE_ARGS = ([ctypes.c_void_p] * 7 + [ctypes.c_int] * 6 +
                [ctypes.c_float, ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p])

_SYMBOLS = {
    # name: (restype, argtypes)
    "gdn_prefill_workspace_size": (ctypes.c_size_t, [ctypes.c_int] * 7),
    "kda_prefill_workspace_size": (ctypes.c_size_t, [ctypes.c_int] * 7),
    "gdn_prefill": (ctypes.c_int, _PREFILL_ARGS + _PREFILL_TAIL),
    "kda_prefill": (ctypes.c_int, _PREFILL_ARGS + _PREFILL_TAIL),
    "gdn_prefill_ex": (ctypes.c_int, _PREFILL_ARGS + [ctypes.c_int] + _PREFILL_TAIL),
    "kda_prefill_ex": (ctypes.c_int, _PREFILL_ARGS + [ctypes.c_int] + _PREFILL_TAIL),
    "gdn_decode": (ctypes.c_int, _DECODE_ARGS),
    "kda_decode": (ctypes.c_int, _DECODE_ARGS),
    "hagdn_last_error": (ctypes.c_char_p, []),
    "hagdn_device_status": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p,
                                           ctypes.POINTER(ctypes.c_int)]),
    "hagdn_profile_begin": (ctypes.c_int, [ctypes.c_int]),
    "hagdn_profile_end": (ctypes.c_int, [ctypes.POINTER(ctypes.c_double), ctypes.c_int,
                                         ctypes.POINTER(ctypes.c_int)]),
    "hagdn_kernel_count": (ctypes.c_int, []),
    "hagdn_kernel_name": (ctypes.c_char_p, [ctypes.c_int]),
    "hagdn_version": (ctypes.c_int, []),
    "hagdn_set_segment_chunks": (ctypes.c_int, [ctypes.c_int]),
    "hagdn_set_overlap": (ctypes.c_int, [ctypes.c_int]),
    "hagdn_overlap_for": (ctypes.c_int, [ctypes.c_int] * 8),
    "hagdn_segment_chunks": (ctypes.c_int, [ctypes.c_int] * 6),
    "hagdn_segment_chunks_for": (ctypes.c_int, [ctypes.c_int] * 7),
    "hagdn_workspace_region": (ctypes.c_int, [ctypes.c_int] * 9 + [ctypes.POINTER(ctypes.c_size_t)] * 2),
    "hagdn_prefill_noalloc": (ctypes.c_int, [ctypes.c_int] + [ctypes.c_void_p] * 7 + [ctypes.c_int] * 6 +
                              [ctypes.c_float, ctypes.c_int, ctypes.c_int, ctypes.c_void_p,
                               ctypes.c_void_p, ctypes.c_void_p]),
    "hagdn_prefill_noalloc_capacity": (ctypes.c_size_t, []),
    "hagdn_measure_copy": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]),
    "hagdn_measure_mfma": (ctypes.c_int, [ctypes.c_int, ctypes.c_void_p, ctypes.c_size_t,
                                          ctypes.POINTER(ctypes.c_double), ctypes.c_void_p]),
}

# workspace regions (hagdn_ws_region)
WS_NM, WS_B, WS_QP, WS_OLOC, WS_DECAY, WS_SEG_A, WS_SEG_B = range(7)


class HagdnError(RuntimeError):
    """A non-OK status from the library (message from hagdn_last_error)."""

    def __init__(self, code, msg):
        super().__init__(f"hagdn status {code}: {msg}")
        self.code = code


def library_path() -> str:
    return _LIB_PATH


def load_library():
    """Load libhagdn.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        # torch first: the library then binds to the HIP runtime torch loaded,
        # so that both share one runtime (and device context) in the process
        import torch  # noqa: F401
        if not os.path.exists(_LIB_PATH):
            raise RuntimeError(f"{_LIB_PATH} is missing: build it with "
                               "`python -m paper_2609_32114_amd.build`")
        lib = ctypes.CDLL(_LIB_PATH)
        for name, (res, args) in _SYMBOLS.items():
            fn = getattr(lib, name)
            fn.restype = res
            fn.argtypes = args
        _lib = lib
    return _lib


def _err(lib):
    m = lib.hagdn_last_error()
    return m.decode() if m else ""


def _dtype_code(t):
    import torch
    if t == torch.bfloat16:
        return HAGDN_BF16
    if t == torch.float32:
        return HAGDN_F32
    raise TypeError(f"unsupported dtype {t}; use torch.bfloat16 or torch.float32")


def workspace_size(kind, N, T, Hqk, Hv, Dk, Dv, dtype_code) -> int:
    lib = load_library()
    fn = lib.gdn_prefill_workspace_size if kind == "gdn" else lib.kda_prefill_workspace_size
    n = fn(N, T, Hqk, Hv, Dk, Dv, dtype_code)
    if n == 0:
        raise HagdnError(1, _err(lib))
    return int(n)


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _check_buffer(name, t, device, dtype, shape):
    """A caller-supplied buffer the kernels write or read through a raw pointer:
    on the call's GPU, of the expected dtype, shape and contiguous layout."""
    if not t.is_cuda or t.device != device:
        raise ValueError(f"{name} must be on {device} (got {t.device})")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype} (got {t.dtype})")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)} (got {tuple(t.shape)})")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _prefill(kind, q, k, v, g, beta, initial_state, cu_seqlens, scale, output_final_state,
             workspace, out, final_out, preprocess=0):
    import torch
    lib = load_library()
    if not (q.is_cuda and k.is_cuda and v.is_cuda and g.is_cuda and beta.is_cuda):
        raise ValueError("all tensors must be on the GPU")
    if not all(t.device == q.device for t in (k, v, g, beta)):
        raise ValueError("q, k, v, g and beta must be on one device")
    if not (q.dtype == k.dtype == v.dtype):
        raise TypeError("q, k, v must share one dtype")
    dt = _dtype_code(q.dtype)
    if g.dtype != torch.float32 or beta.dtype != torch.float32:
        raise TypeError("g and beta must be float32")
    for name, t in (("q", q), ("k", k), ("v", v), ("g", g), ("beta", beta)):
        if not t.is_contiguous():
            raise ValueError(f"{name} must be contiguous")
    T, Hqk, Dk = q.shape
    Hv, Dv = v.shape[1], v.shape[2]
    if k.shape != q.shape or v.shape[0] != T:
        raise ValueError("shape mismatch between q, k, v")
    gshape = (T, Hv) if kind == "gdn" else (T, Hv, Dk)
    if tuple(g.shape) != gshape or tuple(beta.shape) != (T, Hv):
        raise ValueError(f"g must be {gshape} and beta {(T, Hv)}")
    dev = q.device
    if cu_seqlens is None:
        cu_seqlens = torch.tensor([0, T], dtype=torch.int32, device=dev)
    if cu_seqlens.dtype != torch.int32 or not cu_seqlens.is_cuda or not cu_seqlens.is_contiguous():
        raise TypeError("cu_seqlens must be a contiguous int32 GPU tensor")
    if cu_seqlens.device != dev or cu_seqlens.dim() != 1:
        raise ValueError(f"cu_seqlens must be a 1-D tensor on {dev}")
    N = cu_seqlens.shape[0] - 1
    state_shape = (N, Hv, Dk, Dv)
    if initial_state is not None:
        _check_buffer("initial_state", initial_state, dev, torch.float32, state_shape)
    if out is not None:
        _check_buffer("out", out, dev, q.dtype, (T, Hv, Dv))
    o = out if out is not None else torch.empty((T, Hv, Dv), dtype=q.dtype, device=dev)
    sf = None
    if output_final_state:
        if final_out is not None:
            _check_buffer("final_out", final_out, dev, torch.float32, state_shape)
        sf = final_out if final_out is not None else torch.empty(state_shape, dtype=torch.float32,
                                                                 device=dev)
    need = workspace_size(kind, N, T, Hqk, Hv, Dk, Dv, dt)
    if workspace is None:
        workspace = torch.empty(need, dtype=torch.uint8, device=dev)
    elif not workspace.is_cuda or workspace.device != dev or not workspace.is_contiguous():
        raise ValueError(f"workspace must be a contiguous tensor on {dev}")
    stream = torch.cuda.current_stream(dev).cuda_stream
    fn = lib.gdn_prefill_ex if kind == "gdn" else lib.kda_prefill_ex
    rc = fn(_ptr(q), _ptr(k), _ptr(v), _ptr(g), _ptr(beta), _ptr(initial_state), _ptr(cu_seqlens),
            N, T, Hqk, Hv, Dk, Dv, float(scale), dt, int(preprocess), _ptr(o), _ptr(sf),
            _ptr(workspace), workspace.numel() * workspace.element_size(), ctypes.c_void_p(stream))
    if rc != 0:
        raise HagdnError(rc, _err(lib))
    return o, sf


def gdn_prefill(q, k, v, g, beta, initial_state=None, cu_seqlens=None, scale=1.0,
                output_final_state=True, workspace=None, out=None, final_out=None, preprocess=0):
    """Gated DeltaNet prefill.  Returns (o, final_state or None).

    preprocess: a mask of PRE_* flags; q, k, g and beta then hold raw
    projections that the kernels normalise / map as they load them."""
    return _prefill("gdn", q, k, v, g, beta, initial_state, cu_seqlens, scale, output_final_state,
                    workspace, out, final_out, preprocess)


def kda_prefill(q, k, v, g, beta, initial_state=None, cu_seqlens=None, scale=1.0,
                output_final_state=True, workspace=None, out=None, final_out=None, preprocess=0):
    """KDA prefill (per-key-channel log-gate g [T, Hv, Dk]).  Returns (o, final_state or None)."""
    return _prefill("kda", q, k, v, g, beta, initial_state, cu_seqlens, scale, output_final_state,
                    workspace, out, final_out, preprocess)


def _decode(kind, q, k, v, g, beta, state, slots, scale, preprocess, out):
    import torch
    lib = load_library()
    for name, t in (("q", q), ("k", k), ("v", v), ("g", g), ("beta", beta), ("state", state)):
        if not t.is_cuda or not t.is_contiguous() or t.device != q.device:
            raise ValueError(f"{name} must be a contiguous tensor on {q.device}")
    if not (q.dtype == k.dtype == v.dtype):
        raise TypeError("q, k, v must share one dtype")
    dt = _dtype_code(q.dtype)
    if g.dtype != torch.float32 or beta.dtype != torch.float32 or state.dtype != torch.float32:
        raise TypeError("g, beta and state must be float32")
    N, Hqk, Dk = q.shape
    Hv, Dv = v.shape[1], v.shape[2]
    if k.shape != q.shape or v.shape[0] != N:
        raise ValueError("shape mismatch between q, k, v")
    gshape = (N, Hv) if kind == "gdn" else (N, Hv, Dk)
    if tuple(g.shape) != gshape or tuple(beta.shape) != (N, Hv):
        raise ValueError(f"g must be {gshape} and beta {(N, Hv)}")
    if state.dim() != 4 or tuple(state.shape[1:]) != (Hv, Dk, Dv):
        raise ValueError(f"state must be [slots, {Hv}, {Dk}, {Dv}]")
    if slots is None:
        if state.shape[0] < N:
            raise ValueError("without slots the state pool needs one state per sequence")
    elif slots.dtype != torch.int32 or not slots.is_cuda or tuple(slots.shape) != (N,) \
            or not slots.is_contiguous() or slots.device != q.device:
        raise TypeError(f"slots must be a contiguous int32 tensor of length N on {q.device}")
    if out is not None:
        _check_buffer("out", out, q.device, q.dtype, (N, Hv, Dv))
    o = out if out is not None else torch.empty((N, Hv, Dv), dtype=q.dtype, device=q.device)
    stream = torch.cuda.current_stream(q.device).cuda_stream
    fn = lib.gdn_decode if kind == "gdn" else lib.kda_decode
    rc = fn(_ptr(q), _ptr(k), _ptr(v), _ptr(g), _ptr(beta), _ptr(state), _ptr(slots),
            int(state.shape[0]), N, Hqk, Hv, Dk, Dv, float(scale), dt, int(preprocess), _ptr(o),
            ctypes.c_void_p(stream))
    if rc != 0:
        raise HagdnError(rc, _err(lib))
    return o


def gdn_decode(q, k, v, g, beta, state, slots=None, scale=1.0, preprocess=0, out=None):
    """One GDN decode step: q, k [N, Hqk, Dk], v [N, Hv, Dv], g, beta [N, Hv].
    Updates the fp32 state pool [S, Hv, Dk, Dv] in place (sequence n in slot
    slots[n], or n) and returns o [N, Hv, Dv]."""
    return _decode("gdn", q, k, v, g, beta, state, slots, scale, preprocess, out)


def kda_decode(q, k, v, g, beta, state, slots=None, scale=1.0, preprocess=0, out=None):
    """One KDA decode step (g [N, Hv, Dk]); see gdn_decode."""
    return _decode("kda", q, k, v, g, beta, state, slots, scale, preprocess, out)


def device_status(workspace) -> int:
    """Device status word of the last call that used ``workspace`` (synchronises)."""
    import torch
    lib = load_library()
    code = ctypes.c_int(-1)
    stream = torch.cuda.current_stream(workspace.device).cuda_stream
    rc = lib.hagdn_device_status(_ptr(workspace), workspace.numel(), ctypes.c_void_p(stream),
                                 ctypes.byref(code))
    if rc != 0:
        raise HagdnError(rc, _err(lib))
    return code.value


def set_segment_chunks(chunks: int):
    """Force the state chain's segment length (in 64-token chunks) for every later
    call in this process; 0 restores the automatic choice.  Workspace sizes
    depend on it: query them after setting."""
    lib = load_library()
    rc = lib.hagdn_set_segment_chunks(int(chunks))
    if rc != 0:
        raise HagdnError(rc, _err(lib))


def set_overlap(on: bool = True, force: bool = False):
    """The overlapped launch for later calls: where it pays (on, the default),
    wherever it can run (force; for tests and measurements), or never (off)."""
    lib = load_library()
    rc = lib.hagdn_set_overlap(0 if not on else (2 if force else 1))
    if rc != 0:
        raise HagdnError(rc, _err(lib))


def overlap_for(N: int, T: int, Hv: int, Dk: int, Dv: int, dtype_code: int, kind: str = "gdn",
                cus: int = 256) -> bool:
    """Whether a call with these sizes takes the overlapped launch on a device
    of `cus` compute units (host logic only)."""
    lib = load_library()
    r = lib.hagdn_overlap_for(int(N), int(T), int(Hv), int(Dk), int(Dv), int(dtype_code),
                              int(kind == "kda"), int(cus))
    if r < 0:
        raise HagdnError(1, _err(lib))
    return bool(r)


def segment_chunks(N: int, T: int, Hv: int, Dv: int, dtype=None, kind: str = "gdn") -> int:
    """Segment length a gdn_prefill (kind "gdn") or kda_prefill ("kda") call
    with these sizes and I/O dtype (torch.bfloat16, the default, or
    torch.float32) would use now."""
    import torch
    lib = load_library()
    code = _dtype_code(torch.bfloat16 if dtype is None else dtype)
    if kind not in ("gdn", "kda"):
        raise ValueError(f"kind must be 'gdn' or 'kda', not {kind!r}")
    L = lib.hagdn_segment_chunks(int(N), int(T), int(Hv), int(Dv), code, int(kind == "kda"))
    if L < 0:
        raise HagdnError(1, _err(lib))
    return L


def workspace_region(kind, N, T, Hqk, Hv, Dk, Dv, dtype_code, region):
    """(byte offset, bytes) of a workspace region (WS_*) for a call with these sizes."""
    lib = load_library()
    off, n = ctypes.c_size_t(), ctypes.c_size_t()
    rc = lib.hagdn_workspace_region(int(kind == "kda"), N, T, Hqk, Hv, Dk, Dv, dtype_code, int(region),
                                    ctypes.byref(off), ctypes.byref(n))
    if rc != 0:
        raise HagdnError(rc, _err(lib))
    return off.value, n.value


def measure_copy(src, dst):
    """Enqueue the library's streaming copy of src into dst (same byte size) on
    torch's current stream."""
    import torch
    lib = load_library()
    n = src.numel() * src.element_size()
    if dst.numel() * dst.element_size() != n or not (src.is_cuda and dst.is_cuda):
        raise ValueError("src and dst must be GPU tensors of one byte size")
    rc = lib.hagdn_measure_copy(_ptr(src), _ptr(dst), n,
                                ctypes.c_void_p(torch.cuda.current_stream(src.device).cuda_stream))
    if rc != 0:
        raise HagdnError(rc, _err(lib))


def measure_mfma(iterations, sink):
    """Enqueue the library's bf16 MFMA loop on torch's current stream; returns
    the FLOPs it performs.  sink: a float32 GPU tensor of >= 16 x CUs elements."""
    import torch
    lib = load_library()
    flops = ctypes.c_double()
    rc = lib.hagdn_measure_mfma(int(iterations), _ptr(sink), sink.numel(), ctypes.byref(flops),
                                ctypes.c_void_p(torch.cuda.current_stream(sink.device).cuda_stream))
    if rc != 0:
        raise HagdnError(rc, _err(lib))
    return flops.value


def segment_chunks_for(N: int, T: int, Hv: int, Dv: int, cus: int, dtype=None,
                       kind: str = "gdn") -> int:
    """The automatic segment length for a device of ``cus`` compute units (host
    rule only, no device query; a forced length applies here too)."""
    import torch
    lib = load_library()
    code = _dtype_code(torch.bfloat16 if dtype is None else dtype)
    if kind not in ("gdn", "kda"):
        raise ValueError(f"kind must be 'gdn' or 'kda', not {kind!r}")
    L = lib.hagdn_segment_chunks_for(int(N), int(T), int(Hv), int(Dv), code, int(kind == "kda"),
                                     int(cus))
    if L < 0:
        raise HagdnError(1, _err(lib))
    return L


def kernel_names():
    lib = load_library()
    return [lib.hagdn_kernel_name(i).decode() for i in range(lib.hagdn_kernel_count())]


def profile_begin(max_calls: int):
    lib = load_library()
    rc = lib.hagdn_profile_begin(int(max_calls))
    if rc != 0:
        raise HagdnError(rc, _err(lib))


def profile_end():
    """Returns ({kernel name: mean ms}, calls timed)."""
    lib = load_library()
    n = lib.hagdn_kernel_count()
    arr = (ctypes.c_double * n)()
    calls = ctypes.c_int(0)
    rc = lib.hagdn_profile_end(arr, n, ctypes.byref(calls))
    if rc != 0:
        raise HagdnError(rc, _err(lib))
    return dict(zip(kernel_names(), list(arr))), calls.value
