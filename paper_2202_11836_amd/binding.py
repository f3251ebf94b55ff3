"""Thin ctypes binding of the C ABI of libskystage.so: the encoder stage
(include/stage.h) and the host-side layer allocator (include/alloc.h).

Argument marshalling only: torch tensors supply device memory and the HIP
stream (torch.cuda.current_stream()); every step of the stage runs in the
HIP kernels of libskystage.so.  There is no fallback: if the library is not
built, loading fails with an error.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libskystage.so")

STAGE_OK, STAGE_EINVAL, STAGE_ESTATE, STAGE_ENOMEM, STAGE_EHIP = range(5)
STAGE_F32, STAGE_BF16 = 0, 1
PARAM_NAMES = ("W_qkv", "b_qkv", "W_o", "b_o", "g1", "be1",
               "W_1", "b_1", "W_2", "b_2", "g2", "be2")
SAVED_NAMES = ("X", "QKV", "CTX", "H1", "GD", "G")  # GD = GELU'(U)
KIND_PARAM, KIND_GRAD, KIND_SAVED, KIND_RECORDED_GRAD = 0, 1, 2, 3
STATUS_NAMES = {0: "OK", 1: "EINVAL", 2: "ESTATE", 3: "ENOMEM", 4: "EHIP"}

ALLOC_OK, ALLOC_EINVAL, ALLOC_ENOFIT = range(3)
ALLOC_CT_PER_LAYER, ALLOC_CT_PER_DEVICE = 0, 1
ALLOC_STATUS_NAMES = {0: "OK", 1: "EINVAL", 2: "ENOFIT"}

EXPORTED = ("alloc_coarse", "alloc_fine", "alloc_workloads", "stage_init", "stage_init_units",
            "stage_set_stream", "stage_forward", "stage_backward", "stage_param",
            "stage_grad", "stage_set_param", "stage_read", "stage_tensor_bytes",
            "stage_trace_site", "stage_trace_mask", "stage_trace_read", "stage_site_count",
            "stage_site_name", "stage_device_bytes", "stage_memory_model",
            "stage_memory_model_units", "stage_mfma_peak", "stage_record_grads",
            "stage_backward_noalloc",
            "stage_last_error", "stage_destroy")

_lib = None


class AllocError(RuntimeError):
    def __init__(self, status: int, pi=None):
        super().__init__(ALLOC_STATUS_NAMES.get(status, str(status)))
        self.status = status
        self.pi = pi  # last partition index (ENOFIT)


class StageError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {msg}")
        self.status = status


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libskystage.so and declare the C signatures."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is not built; run __graft_entry__.build() first")
    # torch ships its own HIP runtime (same soname as /opt/rocm's).  Load it
    # first so that the library binds to the runtime that owns torch's
    # device memory and streams, never to a second copy in the process.
    import torch  # noqa: F401
    lib = ctypes.CDLL(path)
    vp, i32, i64, u64, sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_uint64, ctypes.c_size_t
    lib.stage_init.argtypes = [i32, i32, i32, i32, u64, i32, vp, ctypes.POINTER(vp)]
    lib.stage_init.restype = i32
    lib.stage_init_units.argtypes = [i32, i32, i32, i32, i32, u64, i32, vp, ctypes.POINTER(vp)]
    lib.stage_init_units.restype = i32
    lib.stage_set_stream.argtypes = [vp, vp]
    lib.stage_set_stream.restype = i32
    lib.stage_forward.argtypes = [vp, vp, vp, i32, i32, vp]
    lib.stage_forward.restype = i32
    lib.stage_backward.argtypes = [vp, vp, vp]
    lib.stage_backward.restype = i32
    lib.stage_backward_noalloc.argtypes = [vp, vp, vp]
    lib.stage_backward_noalloc.restype = i32
    lib.stage_param.argtypes = [vp, i32, i32, ctypes.POINTER(vp), ctypes.POINTER(i64), ctypes.POINTER(i32)]
    lib.stage_param.restype = i32
    lib.stage_grad.argtypes = [vp, i32, i32, ctypes.POINTER(vp), ctypes.POINTER(i64)]
    lib.stage_grad.restype = i32
    lib.stage_set_param.argtypes = [vp, i32, i32, vp, sz]
    lib.stage_set_param.restype = i32
    lib.stage_read.argtypes = [vp, i32, i32, i32, vp, sz]
    lib.stage_read.restype = i32
    lib.stage_tensor_bytes.argtypes = [vp, i32, i32, i32]
    lib.stage_tensor_bytes.restype = sz
    lib.stage_trace_site.argtypes = [vp, i32]
    lib.stage_trace_site.restype = i32
    lib.stage_trace_mask.argtypes = [vp, u64]
    lib.stage_trace_mask.restype = i32
    lib.stage_trace_read.argtypes = [vp, ctypes.POINTER(i32), ctypes.POINTER(ctypes.c_double)]
    lib.stage_trace_read.restype = i32
    lib.stage_site_count.argtypes = []
    lib.stage_site_count.restype = i32
    lib.stage_site_name.argtypes = [i32]
    lib.stage_site_name.restype = ctypes.c_char_p
    lib.stage_last_error.argtypes = [vp]
    lib.stage_last_error.restype = ctypes.c_char_p
    lib.stage_destroy.argtypes = [vp]
    lib.stage_destroy.restype = None
    lib.stage_device_bytes.argtypes = [vp, ctypes.POINTER(i64)]
    lib.stage_device_bytes.restype = i32
    lib.stage_memory_model.argtypes = [i32, i32, i32, i32, i32, i32, ctypes.POINTER(i64),
                                       ctypes.POINTER(i64)]
    lib.stage_memory_model.restype = i32
    lib.stage_memory_model_units.argtypes = [i32, i32, i32, i32, i32, i32, ctypes.POINTER(i64),
                                             ctypes.POINTER(i64), ctypes.POINTER(i64)]
    lib.stage_memory_model_units.restype = i32
    lib.stage_mfma_peak.argtypes = [vp, i32, ctypes.POINTER(ctypes.c_double),
                                    ctypes.POINTER(ctypes.c_double)]
    lib.stage_mfma_peak.restype = i32
    lib.stage_record_grads.argtypes = [vp, i32]
    lib.stage_record_grads.restype = i32
    dp, ip = ctypes.POINTER(ctypes.c_double), ctypes.POINTER(i32)
    lib.alloc_coarse.argtypes = [i32, i32, dp, dp, ip, ip]
    lib.alloc_coarse.restype = i32
    lib.alloc_fine.argtypes = [i32, i32, dp, dp, dp, dp, dp, i32, ip, ip]
    lib.alloc_fine.restype = i32
    lib.alloc_workloads.argtypes = [i32, i32, dp, dp, dp, ip, i32, dp]
    lib.alloc_workloads.restype = i32
    _lib = lib
    return lib


def _check(handle, status: int):
    if status != STAGE_OK:
        msg = ""
        if handle:
            raw = load_library().stage_last_error(handle)
            msg = raw.decode() if raw else ""
        raise StageError(status, msg)


def _current_stream():
    import torch
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


# ---------------------------------------------------------------------------
# Same names as the C ABI (argument marshalling only)
# ---------------------------------------------------------------------------

def stage_init(L: int, hidden: int, heads: int, ffn: int, seed: int, dtype: int,
               stream=None) -> ctypes.c_void_p:
    lib = load_library()
    out = ctypes.c_void_p()
    st = lib.stage_init(L, hidden, heads, ffn, seed, dtype,
                        stream if stream is not None else _current_stream(), ctypes.byref(out))
    if st != STAGE_OK:
        raise StageError(st, "stage_init: " + (lib.stage_last_error(None) or b"").decode())
    return out


def stage_init_units(first_unit: int, n_units: int, hidden: int, heads: int, ffn: int, seed: int,
                     dtype: int, stream=None) -> ctypes.c_void_p:
    lib = load_library()
    out = ctypes.c_void_p()
    st = lib.stage_init_units(first_unit, n_units, hidden, heads, ffn, seed, dtype,
                              stream if stream is not None else _current_stream(),
                              ctypes.byref(out))
    if st != STAGE_OK:
        raise StageError(st, "stage_init_units: " + (lib.stage_last_error(None) or b"").decode())
    return out


def stage_set_stream(handle, stream) -> None:
    _check(handle, load_library().stage_set_stream(handle, stream))


def stage_forward(handle, x, key_mask, batch: int, seq: int, y) -> None:
    _check(handle, load_library().stage_forward(handle, _ptr(x), _ptr(key_mask), batch, seq, _ptr(y)))


def stage_backward(handle, dy, dx) -> None:
    _check(handle, load_library().stage_backward(handle, _ptr(dy), _ptr(dx)))


def stage_backward_noalloc(handle, dy, dx) -> None:
    _check(handle, load_library().stage_backward_noalloc(handle, _ptr(dy), _ptr(dx)))


def stage_param(handle, layer: int, which: int):
    p, n, d = ctypes.c_void_p(), ctypes.c_int64(), ctypes.c_int()
    _check(handle, load_library().stage_param(handle, layer, which, ctypes.byref(p), ctypes.byref(n),
                                              ctypes.byref(d)))
    return p.value, n.value, d.value


def stage_grad(handle, layer: int, which: int):
    p, n = ctypes.c_void_p(), ctypes.c_int64()
    _check(handle, load_library().stage_grad(handle, layer, which, ctypes.byref(p), ctypes.byref(n)))
    return p.value, n.value


def stage_set_param(handle, layer: int, which: int, src) -> None:
    nbytes = src.numel() * src.element_size()
    _check(handle, load_library().stage_set_param(handle, layer, which, src.data_ptr(), nbytes))


def stage_read(handle, kind: int, layer: int, which: int, dst) -> None:
    nbytes = dst.numel() * dst.element_size()
    _check(handle, load_library().stage_read(handle, kind, layer, which, dst.data_ptr(), nbytes))


def stage_record_grads(handle, on: int) -> None:
    _check(handle, load_library().stage_record_grads(handle, int(on)))


def stage_tensor_bytes(handle, kind: int, layer: int, which: int) -> int:
    return load_library().stage_tensor_bytes(handle, kind, layer, which)


def stage_trace_site(handle, site: int) -> None:
    _check(handle, load_library().stage_trace_site(handle, site))


def stage_trace_mask(handle, mask: int) -> None:
    _check(handle, load_library().stage_trace_mask(handle, mask))


def stage_trace_read(handle):
    n, ms = ctypes.c_int(), ctypes.c_double()
    _check(handle, load_library().stage_trace_read(handle, ctypes.byref(n), ctypes.byref(ms)))
    return n.value, ms.value


def stage_site_count() -> int:
    return load_library().stage_site_count()


def stage_site_name(site: int) -> str:
    return load_library().stage_site_name(site).decode()


def stage_device_bytes(handle) -> int:
    v = ctypes.c_int64(0)
    _check(handle, load_library().stage_device_bytes(handle, ctypes.byref(v)))
    return v.value


def stage_memory_model(hidden: int, heads: int, ffn: int, batch: int, seq: int, dtype: int):
    """(per_layer, shared) device bytes of a stage after a forward of batch x seq."""
    a, b = ctypes.c_int64(0), ctypes.c_int64(0)
    _check(None, load_library().stage_memory_model(hidden, heads, ffn, batch, seq, dtype,
                                                   ctypes.byref(a), ctypes.byref(b)))
    return a.value, b.value


def stage_memory_model_units(hidden: int, heads: int, ffn: int, batch: int, seq: int, dtype: int):
    """(attn_unit, ffn_unit, shared) device bytes per half-layer unit."""
    a, b, c = ctypes.c_int64(0), ctypes.c_int64(0), ctypes.c_int64(0)
    _check(None, load_library().stage_memory_model_units(hidden, heads, ffn, batch, seq, dtype,
                                                         ctypes.byref(a), ctypes.byref(b),
                                                         ctypes.byref(c)))
    return a.value, b.value, c.value


def stage_mfma_peak(iters: int = 20000, stream=None):
    """(TFLOP/s, GHz): achievable dense bf16 MFMA rate and the shader clock
    held meanwhile, on the current device and stream."""
    t, g = ctypes.c_double(0.0), ctypes.c_double(0.0)
    st = stream if stream is not None else _current_stream()
    _check(None, load_library().stage_mfma_peak(st, iters, ctypes.byref(t), ctypes.byref(g)))
    return t.value, g.value


def stage_last_error(handle) -> str:
    raw = load_library().stage_last_error(handle)
    return raw.decode() if raw else ""


def stage_destroy(handle) -> None:
    if handle:
        load_library().stage_destroy(handle)


# ---------------------------------------------------------------------------
# Convenience wrapper
# ---------------------------------------------------------------------------

class Stage:
    """One stage of L encoder layers on the current GPU, or, with
    first_unit / n_units, of the half-layer units [first_unit, first_unit +
    n_units) (unit 2j: attention half of layer j, unit 2j+1: its
    feed-forward half; L is then the number of layers they touch)."""

    def __init__(self, L: Optional[int], hidden: int, heads: int, ffn: int, seed: int = 0,
                 dtype: str = "bf16", first_unit: int = 0, n_units: Optional[int] = None):
        import torch
        self.hidden, self.heads, self.ffn = hidden, heads, ffn
        self.dtype_name = dtype
        self.code = STAGE_BF16 if dtype == "bf16" else STAGE_F32
        self.torch_dtype = torch.bfloat16 if dtype == "bf16" else torch.float32
        if n_units is None:
            self.first_unit, self.n_units = 0, 2 * L
            self.handle = stage_init(L, hidden, heads, ffn, seed, self.code)
        else:
            self.first_unit, self.n_units = first_unit, n_units
            self.handle = stage_init_units(first_unit, n_units, hidden, heads, ffn, seed, self.code)
            L = (first_unit + n_units - 1) // 2 - first_unit // 2 + 1
        self.L = L

    def _sync_stream(self):
        stage_set_stream(self.handle, _current_stream())

    def forward(self, x, key_mask=None, out=None):
        import torch
        B, S, h = x.shape
        assert h == self.hidden and x.dtype == self.torch_dtype and x.is_cuda and x.is_contiguous()
        if key_mask is not None:
            assert key_mask.dtype == torch.uint8 and key_mask.shape == (B, S) and key_mask.is_contiguous()
        y = torch.empty_like(x) if out is None else out
        self._sync_stream()
        stage_forward(self.handle, x, key_mask, B, S, y)
        return y

    def backward(self, dy, out=None):
        import torch
        assert dy.dtype == self.torch_dtype and dy.is_cuda and dy.is_contiguous()
        dx = torch.empty_like(dy) if out is None else out
        self._sync_stream()
        stage_backward(self.handle, dy, dx)
        return dx

    def backward_noalloc(self, dy, out):
        """Backward with the partial results in the library's static
        scratch (stage_backward_noalloc); out must be given."""
        import torch
        assert dy.dtype == self.torch_dtype and dy.is_cuda and dy.is_contiguous()
        assert out is not None and out.dtype == dy.dtype and out.shape == dy.shape
        self._sync_stream()
        stage_backward_noalloc(self.handle, dy, out)
        return out

    def _param_shape(self, which: int):
        h, f = self.hidden, self.ffn
        return {0: (3 * h, h), 1: (3 * h,), 2: (h, h), 3: (h,), 4: (h,), 5: (h,), 6: (f, h),
                7: (f,), 8: (h, f), 9: (h,), 10: (h,), 11: (h,)}[which]

    def param(self, layer: int, which: int):
        import torch
        _, n, d = stage_param(self.handle, layer, which)
        dt = torch.bfloat16 if d == STAGE_BF16 else torch.float32
        out = torch.empty(self._param_shape(which), dtype=dt, device="cuda")
        self._sync_stream()
        stage_read(self.handle, KIND_PARAM, layer, which, out)
        return out

    def grad(self, layer: int, which: int):
        import torch
        out = torch.empty(self._param_shape(which), dtype=torch.float32, device="cuda")
        self._sync_stream()
        stage_read(self.handle, KIND_GRAD, layer, which, out)
        return out

    def set_param(self, layer: int, which: int, value):
        import torch
        _, n, d = stage_param(self.handle, layer, which)
        dt = torch.bfloat16 if d == STAGE_BF16 else torch.float32
        v = value.to(dtype=dt).contiguous()
        assert v.numel() == n
        self._sync_stream()
        stage_set_param(self.handle, layer, which, v)

    def saved(self, layer: int, which: int, tokens: int):
        import torch
        width = {0: self.hidden, 1: 3 * self.hidden, 2: self.hidden, 3: self.hidden,
                 4: self.ffn, 5: self.ffn}[which]
        out = torch.empty((tokens, width), dtype=self.torch_dtype, device="cuda")
        self._sync_stream()
        stage_read(self.handle, KIND_SAVED, layer, which, out)
        return out

    def record_grads(self, on: bool = True):
        """Record the gradient reaching each layer's output in later
        backward passes (from the next forward on)."""
        stage_record_grads(self.handle, 1 if on else 0)

    def recorded_grad(self, layer: int, tokens: int):
        """fp32 [tokens, hidden] gradient that reached `layer`'s output in
        the latest backward."""
        import torch
        out = torch.empty((tokens, self.hidden), dtype=torch.float32, device="cuda")
        self._sync_stream()
        stage_read(self.handle, KIND_RECORDED_GRAD, layer, 0, out)
        return out

    def trace(self, site_names):
        """Trace every launch of the named kernel site(s) (None: off)."""
        if site_names is None:
            site_names = []
        elif isinstance(site_names, str):
            site_names = [site_names]
        names = [stage_site_name(i) for i in range(stage_site_count())]
        mask = 0
        for n in site_names:
            mask |= 1 << names.index(n)
        self._sync_stream()
        stage_trace_mask(self.handle, mask)

    def device_bytes(self) -> int:
        return stage_device_bytes(self.handle)

    def trace_read(self):
        """(launches, total_ms) of the traced site since trace() / the last read."""
        self._sync_stream()
        return stage_trace_read(self.handle)

    def close(self):
        if getattr(self, "handle", None):
            stage_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


# ---------------------------------------------------------------------------
# Layer allocator (host code; include/alloc.h)
# ---------------------------------------------------------------------------
def _dvec(v):
    v = [float(x) for x in v]
    return (ctypes.c_double * max(len(v), 1))(*v), len(v)


def _ivec(v, n=None):
    v = [int(x) for x in v] if v is not None else [0] * n
    return (ctypes.c_int * max(len(v), 1))(*v)


def alloc_coarse(lm, dm):
    """Algorithm 1: returns (pi, sweeps); raises AllocError (with .pi, the
    last partition index, for ENOFIT)."""
    a_lm, L = _dvec(lm)
    a_dm, D = _dvec(dm)
    pi = _ivec(None, D + 1)
    n = ctypes.c_int(0)
    st = load_library().alloc_coarse(L, D, a_lm, a_dm, pi, ctypes.byref(n))
    if st != ALLOC_OK:
        raise AllocError(st, list(pi) if st == ALLOC_ENOFIT else None)
    return list(pi), n.value


def alloc_fine(dt, dm, ct, lf, lm, pi, max_iter: int):
    """Algorithm 2 from partition pi: returns (tuned pi, rounds)."""
    a_dt, D = _dvec(dt)
    a_dm, _ = _dvec(dm)
    a_ct, _ = _dvec(ct)
    a_lf, L = _dvec(lf)
    a_lm, _ = _dvec(lm)
    p = _ivec(pi)
    if len(pi) != D + 1 or len(dm) != D or len(ct) != D or len(lm) != L:
        raise AllocError(ALLOC_EINVAL)
    n = ctypes.c_int(0)
    st = load_library().alloc_fine(L, D, a_dt, a_dm, a_ct, a_lf, a_lm, int(max_iter), p,
                                   ctypes.byref(n))
    if st != ALLOC_OK:
        raise AllocError(st)
    return list(p), n.value


def alloc_workloads(dt, ct, lf, pi, mode: int = ALLOC_CT_PER_LAYER):
    """Workload of every device under partition pi."""
    a_dt, D = _dvec(dt)
    a_ct, _ = _dvec(ct)
    a_lf, L = _dvec(lf)
    if len(pi) != D + 1 or len(ct) != D:
        raise AllocError(ALLOC_EINVAL)
    out = (ctypes.c_double * D)()
    st = load_library().alloc_workloads(L, D, a_dt, a_ct, a_lf, _ivec(pi), int(mode), out)
    if st != ALLOC_OK:
        raise AllocError(st)
    return list(out)
