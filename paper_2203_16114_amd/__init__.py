"""Python binding of libtrace: TRACE's batched next-byte estimator and its
controller-gated online update on one MI355X (gfx950).

This module only marshals arguments for the C ABI declared in include/trace.h;
every step of the estimator runs in the HIP kernels of libtrace.so.  PyTorch
supplies device memory and the current stream.  There is no fallback: if the
library is missing, loading it raises.
"""
from __future__ import annotations

import ctypes
import os
from ctypes import POINTER, byref, c_double, c_float, c_int32, c_int64, c_uint32, c_uint64, c_void_p

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libtrace.so")

TRACE_OK, TRACE_EINVAL, TRACE_ENOMEM, TRACE_EHIP, TRACE_ESTATE, TRACE_ENONFINITE, TRACE_EUNSUPPORTED = 0, -1, -2, -3, -4, -5, -6
TRACE_FP32, TRACE_BF16 = 0, 1
TRACE_KEEP_ACTS, TRACE_TOKEN_ATTN = 1, 2
TRACE_ATTN_SOFTMAX, TRACE_ATTN_PERFORMER = 0, 1

EXPORTS = ("trace_create", "trace_destroy", "trace_param_count", "trace_init_weights", "trace_init_flat_host", "trace_set_features",
           "trace_forward_bits", "trace_forward_bits_noalloc", "trace_adapt_step", "trace_controller_init", "trace_controller_decide",
           "trace_gated_run",
           "trace_get_state", "trace_set_state", "trace_get_grads", "trace_quant_table", "trace_quantize",
           "trace_rc_encode", "trace_rc_decode", "trace_compress", "trace_decompress",
           "trace_debug_gemm", "trace_debug_kept_tokens", "trace_debug_kv_wgrad",
           "trace_set_timing",
           "trace_read_timing", "trace_strerror", "trace_last_error")
KINDS = ("attn", "ffn_head", "step_ce", "backward", "adam", "refresh")


class TraceError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{msg} (code {code})")
        self.code = code


class TraceConfig(ctypes.Structure):
    _fields_ = [("W", c_int32), ("e", c_int32), ("g", c_int32), ("H", c_int32), ("F", c_int32), ("k", c_int32),
                ("dtype", c_int32), ("use_pos", c_int32), ("max_windows", c_int64), ("max_keep", c_int64),
                ("lr", c_double), ("beta1", c_double), ("beta2", c_double), ("eps", c_double),
                ("untied_ffn", c_int32), ("attention", c_int32), ("n_features", c_int32), ("layers", c_int32),
                ("reserved_", c_int32)]


class TraceControllerState(ctypes.Structure):
    _fields_ = [("t", c_int32), ("count", c_int32), ("head", c_int32), ("pad_", c_int32),
                ("delta", c_double), ("sum", c_double), ("ring", c_double * 256)]


_lib = None


def lib():
    """Loads libtrace.so (built by build.py); raises if it is missing."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                              "or python paper_2203_16114_amd/build.py")
        # PyTorch's HIP runtime first: loaded after the library's, it finds no
        # GPU; loaded first, the library and PyTorch share it
        try:
            import torch  # noqa: F401
        except ImportError:
            pass
        L = ctypes.CDLL(LIB_PATH)
        P = c_void_p
        sig = {
            "trace_create": (c_int32, [POINTER(TraceConfig), POINTER(c_void_p)]),
            "trace_destroy": (None, [P]),
            "trace_param_count": (c_int32, [POINTER(TraceConfig), POINTER(c_int64)]),
            "trace_init_weights": (c_int32, [P, c_uint64, c_double, P]),
            "trace_init_flat_host": (c_int32, [POINTER(TraceConfig), c_uint64, c_double, P, c_int64]),
            "trace_set_features": (c_int32, [P, P, c_int64]),
            "trace_forward_bits": (c_int32, [P, P, c_int64, c_int32, c_int64, c_int32, P, P, P, c_uint32, P]),
            "trace_forward_bits_noalloc": (c_int32, [P, P, c_int64, c_int32, c_int64, c_int32, P, P, P, c_uint32, P]),
            "trace_adapt_step": (c_int32, [P, P]),
            "trace_controller_init": (c_int32, [POINTER(TraceControllerState), c_int32, c_double]),
            "trace_controller_decide": (c_int32, [POINTER(TraceControllerState), c_double, POINTER(c_int32)]),
            "trace_gated_run": (c_int32, [P, P, c_int64, c_int32, c_int64, c_int32, c_int32, c_int32, c_double,
                                          c_int32, P, P, POINTER(c_int64), P]),
            "trace_get_state": (c_int32, [P, P, P, P, POINTER(c_int64), c_int64]),
            "trace_set_state": (c_int32, [P, P, P, P, c_int64, c_int64]),
            "trace_get_grads": (c_int32, [P, P, c_int64]),
            "trace_quant_table": (c_int32, [P]),
            "trace_quantize": (c_int32, [P, c_int64, P, P]),
            "trace_rc_encode": (c_int32, [P, c_int64, P, c_int64, P, c_int64, POINTER(c_int64)]),
            "trace_rc_decode": (c_int32, [P, c_int64, P, c_int64, c_int64, P]),
            "trace_compress": (c_int32, [P, P, c_int64, c_int32, c_int64, c_int32, c_int32, c_double, P, c_int64,
                                         P, POINTER(c_int64), P]),
            "trace_decompress": (c_int32, [P, P, c_int64, P, c_int32, c_int64, c_int32, c_int32, c_double, P,
                                           c_int64, POINTER(c_int64), P]),
            "trace_debug_gemm": (c_int32, [c_int32, c_int32, c_int32, P, c_int32, c_int32, P, c_int32, c_int32, P,
                                           c_int32, c_int32, P, c_int64, P]),
            "trace_debug_kept_tokens": (c_int32, [P, P, P]),
            "trace_debug_kv_wgrad": (c_int32, [P, P, P, P]),
            "trace_set_timing": (c_int32, [P, c_int32]),
            "trace_read_timing": (c_int32, [P, P, P, POINTER(c_int64)]),
            "trace_strerror": (ctypes.c_char_p, [c_int32]),
            "trace_last_error": (ctypes.c_char_p, []),
        }
        for name, (res, args) in sig.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def check(rc: int):
    if rc != TRACE_OK:
        L = lib()
        raise TraceError(rc, f"{L.trace_strerror(rc).decode()}: {L.trace_last_error().decode()}")


def make_config(W, e, g, H, F, k, dtype="fp32", use_pos=True, max_windows=1 << 16, max_keep=0,
                lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, untied_ffn=False, attention="softmax",
                n_features=0, layers=1) -> TraceConfig:
    dt = {"fp32": TRACE_FP32, "bf16": TRACE_BF16}[dtype] if isinstance(dtype, str) else int(dtype)
    att = {"softmax": TRACE_ATTN_SOFTMAX, "performer": TRACE_ATTN_PERFORMER}[attention]
    return TraceConfig(W, e, g, H, F, k, dt, int(bool(use_pos)), int(max_windows), int(max_keep),
                       float(lr), float(beta1), float(beta2), float(eps), int(bool(untied_ffn)), att,
                       int(n_features), int(layers), 0)


def param_count(cfg: TraceConfig) -> int:
    n = c_int64()
    check(lib().trace_param_count(byref(cfg), byref(n)))
    return n.value


def init_flat_host(cfg: TraceConfig, seed: int, std: float = 0.02) -> np.ndarray:
    out = np.empty(param_count(cfg), np.float32)
    check(lib().trace_init_flat_host(byref(cfg), c_uint64(seed & ((1 << 64) - 1)), float(std),
                                     out.ctypes.data, out.size))
    return out


class Controller:
    """The back-prop controller (host only; see trace_controller_decide)."""

    def __init__(self, t: int = 16, delta: float = 0.05):
        self.state = TraceControllerState()
        check(lib().trace_controller_init(byref(self.state), int(t), float(delta)))

    def decide(self, e: float) -> int:
        u = c_int32()
        check(lib().trace_controller_decide(byref(self.state), float(e), byref(u)))
        return u.value


def _stream_ptr(stream=None):
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return c_void_p(s.cuda_stream)


def _dptr(t):
    return c_void_p(t.data_ptr()) if t is not None else None


def debug_gemm(A, B, M: int, N: int, K: int, a_kc: bool, mode_a: int, b_kc: bool, mode_b: int,
               half_c: bool = False, kernel: int = 1, ws_floats: int = 1 << 22, stream=None):
    """One update-step product on the bf16 GEMM kernels (trace_debug_gemm).  A, B:
    CUDA tensors (fp32, or int16 holding bf16 bits for mode 2), laid out as that
    entry point describes; returns C [M][N] (fp32, or int16 bf16 bits)."""
    import torch
    C = torch.empty(M, N, dtype=torch.int16 if half_c else torch.float32, device=A.device)
    ws = torch.empty(max(1, ws_floats), dtype=torch.float32, device=A.device)
    check(lib().trace_debug_gemm(int(M), int(N), int(K), _dptr(A), int(bool(a_kc)), int(mode_a), _dptr(B),
                                 int(bool(b_kc)), int(mode_b), _dptr(C), int(bool(half_c)), int(kernel), _dptr(ws),
                                 int(ws_floats), _stream_ptr(stream)))
    return C


MODE_NEVER, MODE_GATED, MODE_ALWAYS = 0, 1, 2


def quant_table() -> np.ndarray:
    """T[j] = round(2^31 2^(-j/256)) of trace_quantize, uint32[256]."""
    t = np.empty(256, np.uint32)
    check(lib().trace_quant_table(t.ctypes.data))
    return t


def quantize(logits, freq=None, stream=None):
    """Integer frequencies (trace_quantize) of CUDA fp32 logits [n][256]:
    a CUDA int16 tensor [n][256] holding the uint16 values."""
    import torch
    if logits.dtype != torch.float32 or not logits.is_cuda or not logits.is_contiguous():
        raise TypeError("logits must be a contiguous float32 CUDA tensor")
    n = logits.numel() // 256
    if freq is None:
        freq = torch.empty(n, 256, dtype=torch.int16, device=logits.device)
    check(lib().trace_quantize(_dptr(logits), n, _dptr(freq), _stream_ptr(stream)))
    return freq


def _freq_arg(freq, n):
    if freq is None:
        return None, 0, None
    f = np.ascontiguousarray(freq, np.uint16).reshape(-1, 256)
    if f.shape[0] < n:
        raise ValueError("one frequency row per symbol")
    return f.ctypes.data, 256, f


def rc_encode(freq, sym) -> bytes:
    """One range code (trace_rc_encode) of uint8 symbols under frequency rows
    [n][256] (uint16), or under 1/256 when freq is None."""
    x = np.ascontiguousarray(sym, np.uint8)
    fp, fs, keep = _freq_arg(freq, x.size)
    cap = 2 * x.size + 16
    out = np.empty(cap, np.uint8)
    size = c_int64()
    check(lib().trace_rc_encode(fp, fs, x.ctypes.data, x.size, out.ctypes.data, cap, byref(size)))
    return out[:size.value].tobytes()


def rc_decode(freq, data: bytes, n: int) -> np.ndarray:
    fp, fs, keep = _freq_arg(freq, n)
    buf = np.frombuffer(data, np.uint8) if len(data) else np.zeros(1, np.uint8)
    out = np.empty(max(n, 1), np.uint8)
    check(lib().trace_rc_decode(fp, fs, buf.ctypes.data, len(data), n, out.ctypes.data))
    return out[:n]


class TraceModel:
    """One model on the current HIP device (see include/trace.h)."""

    def __init__(self, W, e, g, H, F, k, dtype="fp32", use_pos=True, max_windows=1 << 16, max_keep=0,
                 lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, untied_ffn=False, attention="softmax", n_features=0,
                 layers=1):
        self.cfg = make_config(W, e, g, H, F, k, dtype, use_pos, max_windows, max_keep, lr, beta1, beta2, eps,
                               untied_ffn, attention, n_features, layers)
        self.layers = layers
        self.attention = attention
        self.W, self.e, self.g, self.H, self.F, self.k = W, e, g, H, F, k
        self.T, self.d = W // g, g * e
        self.dtype = dtype
        self.n_params = param_count(self.cfg)
        h = c_void_p()
        check(lib().trace_create(byref(self.cfg), byref(h)))
        self._h = h

    def close(self):
        if getattr(self, "_h", None):
            lib().trace_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def init_weights(self, seed: int, std: float = 0.02, flat: np.ndarray | None = None):
        if flat is not None:
            flat = np.ascontiguousarray(flat, np.float32)
            if flat.size != self.n_params:
                raise ValueError("flat has the wrong length")
        check(lib().trace_init_weights(self._h, c_uint64(seed & ((1 << 64) - 1)), float(std),
                                       None if flat is None else flat.ctypes.data))

    def forward_bits(self, streams, pos0: int, n_steps: int, bits=None, logits=None, step_ce=None,
                     keep: bool = False, n_streams: int | None = None, stride: int | None = None, stream=None,
                     token_attn: bool = False, noalloc: bool = False):
        """streams: uint8 CUDA tensor [B][L] (row stride = L) or flat with n_streams/stride given.
        bits/logits/step_ce: preallocated CUDA tensors, or True to allocate (logits, step_ce).
        token_attn: TRACE_TOKEN_ATTN; noalloc: through trace_forward_bits_noalloc."""
        import torch
        if streams.dtype != torch.uint8 or not streams.is_cuda:
            raise TypeError("streams must be a uint8 CUDA tensor")
        if n_streams is None:
            if streams.dim() != 2 or not streams.is_contiguous():
                raise ValueError("streams must be a contiguous [B][L] tensor, or give n_streams and stride")
            n_streams, stride = streams.shape[0], streams.shape[1]
        dev = streams.device
        N = n_streams * n_steps
        if bits is None:
            bits = torch.empty(N, dtype=torch.float32, device=dev)
        if logits is True:
            logits = torch.empty(N, 256, dtype=torch.float32, device=dev)
        if step_ce is True:
            step_ce = torch.empty(n_steps, dtype=torch.float64, device=dev)
        for t, n in ((bits, N), (logits, N * 256), (step_ce, n_steps)):
            if t is not None and (not t.is_cuda or not t.is_contiguous() or t.numel() < n):
                raise ValueError("output buffers must be contiguous CUDA tensors of the right size")
        fn = lib().trace_forward_bits_noalloc if noalloc else lib().trace_forward_bits
        check(fn(self._h, _dptr(streams), int(stride), int(n_streams), int(pos0), int(n_steps),
                 _dptr(bits), _dptr(logits) if logits is not None else None,
                 _dptr(step_ce) if step_ce is not None else None,
                 (TRACE_KEEP_ACTS if keep else 0) | (TRACE_TOKEN_ATTN if token_attn else 0), _stream_ptr(stream)))
        return {"bits": bits, "logits": logits, "step_ce": step_ce}

    def set_features(self, omega: np.ndarray):
        """The Performer's random projection omega [n_features][d/H] (trace_set_features)."""
        om = np.ascontiguousarray(omega, np.float32)
        check(lib().trace_set_features(self._h, om.ctypes.data, om.size))

    def compress(self, streams, mode: int = MODE_NEVER, t: int = 16, delta: float = 0.05, length=None,
                 stream=None):
        """The compressor of Alg. 1 (trace_compress) over a contiguous uint8
        CUDA tensor [B][stride], coding the first `length` bytes of each row
        (all by default): (list of B codes, number of updates)."""
        import torch
        if streams.dtype != torch.uint8 or not streams.is_cuda or streams.dim() != 2 or not streams.is_contiguous():
            raise TypeError("streams must be a contiguous uint8 CUDA tensor [B][L]")
        B, stride = streams.shape
        L = stride if length is None else int(length)
        cap = 2 * L + 16
        out = np.empty((B, cap), np.uint8)
        sizes = np.empty(B, np.int64)
        nupd = c_int64()
        check(lib().trace_compress(self._h, _dptr(streams), stride, B, L, int(mode), int(t), float(delta),
                                   out.ctypes.data, cap, sizes.ctypes.data, byref(nupd), _stream_ptr(stream)))
        return [out[b, :sizes[b]].tobytes() for b in range(B)], nupd.value

    def decompress(self, codes, length: int, mode: int = MODE_NEVER, t: int = 16, delta: float = 0.05,
                   out=None, stream=None):
        """Inverse of compress for a model in the encoder's starting state:
        (uint8 CUDA tensor [B][length], number of updates)."""
        import torch
        B = len(codes)
        cs = max([len(c) for c in codes] + [1])
        buf = np.zeros((B, cs), np.uint8)
        for b, c in enumerate(codes):
            buf[b, :len(c)] = np.frombuffer(c, np.uint8)
        sizes = np.array([len(c) for c in codes], np.int64)
        if out is None:
            out = torch.empty(B, max(int(length), 1), dtype=torch.uint8, device="cuda")
        nupd = c_int64()
        check(lib().trace_decompress(self._h, buf.ctypes.data, cs, sizes.ctypes.data, B, int(length), int(mode),
                                     int(t), float(delta), _dptr(out), out.shape[1], byref(nupd),
                                     _stream_ptr(stream)))
        return out[:, :length], nupd.value

    def gated_run(self, streams, pos0: int, n_steps: int, mode: int = MODE_GATED, t: int = 16,
                  delta: float = 0.05, max_spec: int = 64, stream=None):
        """Alg. 1 with the controller of Alg. 2 (trace_gated_run) over a
        contiguous uint8 CUDA tensor [B][L]: (step_ce [n_steps] float64,
        decisions [n_steps] int32, number of updates)."""
        import torch
        if streams.dtype != torch.uint8 or not streams.is_cuda or streams.dim() != 2 or not streams.is_contiguous():
            raise TypeError("streams must be a contiguous uint8 CUDA tensor [B][L]")
        B, L = streams.shape
        ce = np.empty(max(n_steps, 1), np.float64)
        dec = np.empty(max(n_steps, 1), np.int32)
        nupd = c_int64()
        check(lib().trace_gated_run(self._h, _dptr(streams), L, B, int(pos0), int(n_steps), int(mode), int(t),
                                    float(delta), int(max_spec), ce.ctypes.data, dec.ctypes.data, byref(nupd),
                                    _stream_ptr(stream)))
        return ce[:n_steps], dec[:n_steps], nupd.value

    def adapt_step(self, stream=None):
        check(lib().trace_adapt_step(self._h, _stream_ptr(stream)))

    def get_state(self):
        n = self.n_params
        th, m, v = (np.empty(n, np.float32) for _ in range(3))
        step = c_int64()
        check(lib().trace_get_state(self._h, th.ctypes.data, m.ctypes.data, v.ctypes.data, byref(step), n))
        return th, m, v, step.value

    def set_state(self, theta, adam_m=None, adam_v=None, step: int = 0):
        n = self.n_params
        arrs = [None if a is None else np.ascontiguousarray(a, np.float32) for a in (theta, adam_m, adam_v)]
        for a in arrs:
            if a is not None and a.size != n:
                raise ValueError("state arrays must have trace_param_count entries")
        check(lib().trace_set_state(self._h, *[None if a is None else a.ctypes.data for a in arrs], int(step), n))

    def grads(self) -> np.ndarray:
        out = np.empty(self.n_params, np.float32)
        check(lib().trace_get_grads(self._h, out.ctypes.data, self.n_params))
        return out

    def set_timing(self, enable: bool):
        check(lib().trace_set_timing(self._h, int(bool(enable))))

    def read_timing(self):
        """{kind: (total ms, launches)} since the last read (synchronises)."""
        ms = np.zeros(len(KINDS), np.float64)
        n = np.zeros(len(KINDS), np.int64)
        ov = c_int64()
        check(lib().trace_read_timing(self._h, ms.ctypes.data, n.ctypes.data, byref(ov)))
        out = {k: (float(ms[i]), int(n[i])) for i, k in enumerate(KINDS)}
        out["overflow"] = ov.value
        return out

    def debug_kv_wgrad(self, stream=None):
        """dWk and dWv of the last update recomputed twice by the rank-one
        weight-gradient kernel (trace_debug_kv_wgrad): from the gathered token
        rows and with the rows gathered in the kernel.  Two CUDA tensors
        [2][d][d] fp32 (gathered in the kernel, from the rows)."""
        import torch
        a = torch.empty(2, self.d, self.d, dtype=torch.float32, device="cuda")
        b = torch.empty_like(a)
        check(lib().trace_debug_kv_wgrad(self._h, _dptr(a), _dptr(b), _stream_ptr(stream)))
        return a, b

    def debug_kept_tokens(self, n_windows: int, stream=None):
        """Byte-embedding part of the kept batch's tokens, from the update's
        gather (trace_debug_kept_tokens): CUDA tensor [n_windows][T][d], fp32
        or int16 holding bf16 bits."""
        import torch
        dt = torch.int16 if self.dtype == "bf16" else torch.float32
        X = torch.empty(n_windows, self.T, self.d, dtype=dt, device="cuda")
        check(lib().trace_debug_kept_tokens(self._h, _dptr(X), _stream_ptr(stream)))
        return X
