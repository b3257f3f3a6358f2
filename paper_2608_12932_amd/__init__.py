"""MI355X (gfx950) W4A8 linear layer: Python binding of libw4a8.so.

The functions carry the names of the C ABI in include/w4a8.h and only
marshal arguments: they check dtypes and shapes of torch tensors, allocate
outputs with torch (device memory is the one thing torch is used for here),
and pass raw pointers plus torch's current HIP stream to the library.  Every
step of the computation runs in the HIP kernels; there is no fallback, and
loading fails loudly when the library has not been built.
"""
from __future__ import annotations

import contextlib
import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libw4a8.so")

W4A8_OK, W4A8_EINVAL, W4A8_EUNSUPPORTED, W4A8_ERANGE, W4A8_EHIP = 0, 1, 2, 3, 4
SCALE_CHANNEL_F32, SCALE_GROUP_F16 = 0, 1
IN_BF16, IN_I8 = 0, 1
OUT_BF16, OUT_F32, OUT_I32_ACC = 0, 1, 2
GROUP_SIZE = 128

EXPORTS = ("w4a8_status_string", "w4a8_packed_weight_bytes", "w4a8_pack_weights",
           "w4a8_quantize_act", "w4a8_linear_workspace_bytes", "w4a8_linear",
           "w4a8_linear_describe", "w4a8_linear_swiglu", "w4a8_linear_swiglu_workspace_bytes",
           "w4a8_linear_swiglu_describe", "w4a8_rmsnorm_quantize_act", "w4a8_stream_attention",
           "w4a8_stream_attention_workspace_bytes", "w4a8_flow_schedule", "w4a8_flow_step",
           "w4a8_linear_noalloc")
NOALLOC_SCRATCH_BYTES = 32 << 20

_OUT_DTYPE = {OUT_BF16: torch.bfloat16, OUT_F32: torch.float32, OUT_I32_ACC: torch.int32}


class W4A8Error(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        super().__init__(f"{what}: {status_string(status)} (status {status})")


_lib = None


def lib() -> ctypes.CDLL:
    """Load libw4a8.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                               "(hipcc, gfx950) before using the W4A8 kernels")
        L = ctypes.CDLL(LIB_PATH)
        P, I64, I, SZ = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_size_t
        L.w4a8_status_string.argtypes = [I]
        L.w4a8_status_string.restype = ctypes.c_char_p
        L.w4a8_packed_weight_bytes.argtypes = [I64, I64]
        L.w4a8_packed_weight_bytes.restype = SZ
        L.w4a8_pack_weights.argtypes = [P, I64, I64, P, P]
        L.w4a8_pack_weights.restype = I
        L.w4a8_quantize_act.argtypes = [P, I64, I64, P, P, P]
        L.w4a8_quantize_act.restype = I
        L.w4a8_rmsnorm_quantize_act.argtypes = [P, P, ctypes.c_float, I64, I64, P, P, P]
        L.w4a8_rmsnorm_quantize_act.restype = I
        L.w4a8_stream_attention.argtypes = [P, P, P, P, P, P, P, I64, I64, I64, I64, I64, I64, ctypes.c_float, P,
                                            P, SZ, P]
        L.w4a8_stream_attention.restype = I
        L.w4a8_stream_attention_workspace_bytes.argtypes = [I64, I64, I64]
        L.w4a8_stream_attention_workspace_bytes.restype = SZ
        L.w4a8_flow_schedule.argtypes = [I64, I64, P]
        L.w4a8_flow_schedule.restype = I
        L.w4a8_flow_step.argtypes = [P, P, P, I64, I64, ctypes.c_float, I64, P, P]
        L.w4a8_flow_step.restype = I
        L.w4a8_linear_workspace_bytes.argtypes = [I64, I64, I64, I, I]
        L.w4a8_linear_workspace_bytes.restype = SZ
        L.w4a8_linear.argtypes = [P, I, P, I64, I64, P, P, I, I64, P, I, P, SZ, P]
        L.w4a8_linear.restype = I
        L.w4a8_linear_noalloc.argtypes = [P, I, P, I64, I64, P, P, I, I64, P, I, P]
        L.w4a8_linear_noalloc.restype = I
        L.w4a8_linear_describe.argtypes = [I64, I64, I64, I, I, I]
        L.w4a8_linear_describe.restype = ctypes.c_char_p
        L.w4a8_linear_swiglu_workspace_bytes.argtypes = [I64, I64, I64, I, I]
        L.w4a8_linear_swiglu_workspace_bytes.restype = SZ
        L.w4a8_linear_swiglu.argtypes = [P, I, P, I64, I64, P, P, I, I64, P, I, P, SZ, P]
        L.w4a8_linear_swiglu.restype = I
        L.w4a8_linear_swiglu_describe.argtypes = [I64, I64, I64, I, I]
        L.w4a8_linear_swiglu_describe.restype = ctypes.c_char_p
        _lib = L
    return _lib


def status_string(status: int) -> str:
    return lib().w4a8_status_string(int(status)).decode()


def _torch_stream(stream=None, device=None) -> torch.cuda.Stream:
    return torch.cuda.current_stream(device) if stream is None else stream


def _stream(stream=None) -> int:
    return _torch_stream(stream).cuda_stream


def _alloc_on(stream):
    """Context for allocating a call's outputs: on the call's stream when it
    is not torch's current one, so that the caching allocator orders their
    reuse after the call's kernels."""
    return contextlib.nullcontext() if stream is None else torch.cuda.stream(stream)


def _dev(t: torch.Tensor, name: str, dtype: torch.dtype) -> int:
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a device tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t.data_ptr()


def _check(rc: int, what: str) -> None:
    if rc != W4A8_OK:
        raise W4A8Error(rc, what)


def w4a8_packed_weight_bytes(N: int, K: int) -> int:
    return int(lib().w4a8_packed_weight_bytes(N, K))


def w4a8_pack_weights(w: torch.Tensor, out: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """w: int8 [N][K] device tensor with values in [-8, 7] -> packed uint8 (N*K/2)."""
    N, K = w.shape
    nbytes = w4a8_packed_weight_bytes(N, K)
    if nbytes == 0:
        raise W4A8Error(W4A8_EINVAL, f"w4a8_pack_weights: shape {N}x{K}")
    if out is None:
        with _alloc_on(stream):
            out = torch.empty(nbytes, dtype=torch.uint8, device=w.device)
    elif out.numel() != nbytes:
        raise ValueError(f"out must hold {nbytes} bytes")
    rc = lib().w4a8_pack_weights(_dev(w, "w", torch.int8), N, K, _dev(out, "out", torch.uint8),
                                 _stream(stream))
    _check(rc, "w4a8_pack_weights")
    return out


def w4a8_quantize_act(x: torch.Tensor, stream=None):
    """x: bf16 [M][K] device tensor -> (codes int8 [M][K], scales fp32 [M])."""
    M, K = x.shape
    with _alloc_on(stream):
        q = torch.empty((M, K), dtype=torch.int8, device=x.device)
        s = torch.empty((M,), dtype=torch.float32, device=x.device)
    rc = lib().w4a8_quantize_act(_dev(x, "x", torch.bfloat16), M, K, _dev(q, "q", torch.int8),
                                 _dev(s, "s", torch.float32), _stream(stream))
    _check(rc, "w4a8_quantize_act")
    return q, s


def w4a8_rmsnorm_quantize_act(x: torch.Tensor, gamma: torch.Tensor, eps: float, stream=None):
    """RMSNorm (gain gamma bf16 [K], eps > 0) of bf16 x [M][K] then the
    per-token int8 quantize of the fp32 result -> (codes int8 [M][K],
    scales fp32 [M]), the int8 input of w4a8_linear."""
    M, K = x.shape
    x_ptr = _dev(x, "x", torch.bfloat16)
    g_ptr = _dev(gamma, "gamma", torch.bfloat16)
    if tuple(gamma.shape) != (K,):
        raise ValueError(f"gamma must be [{K}]")
    with _alloc_on(stream):
        q = torch.empty((M, K), dtype=torch.int8, device=x.device)
        s = torch.empty((M,), dtype=torch.float32, device=x.device)
    rc = lib().w4a8_rmsnorm_quantize_act(x_ptr, g_ptr, float(eps), M, K, q.data_ptr(), s.data_ptr(), _stream(stream))
    _check(rc, "w4a8_rmsnorm_quantize_act")
    return q, s


def w4a8_flow_schedule(n_steps: int, n_reuse: int) -> list:
    """Per step of an n_steps flow-matching solve: True where the action
    network is evaluated, False where the cached velocity is reused."""
    import ctypes

    buf = (ctypes.c_int32 * max(int(n_steps), 1))()
    _check(lib().w4a8_flow_schedule(n_steps, n_reuse, buf), "w4a8_flow_schedule")
    return [bool(buf[i]) for i in range(n_steps)]


def w4a8_flow_step(x: torch.Tensor, v_new, v_cache: torch.Tensor, dt: float, stats: bool = False, stream=None,
                   repeat: int = 1):
    """Euler step x += dt v of the flow-matching solve, in place on fp32 x
    [B][n], applied `repeat` times (consecutive steps with the same
    velocity).  v_new bf16 [B][n] (an evaluated step: the cache becomes
    v_new) or None (a reused step: v = v_cache).  With stats (evaluated
    steps only) returns fp64 [B][4] = (v.c, v.v, c.c, |v - c|^2) against
    the cache before the step, else None."""
    B, n = x.shape
    x_ptr = _dev(x, "x", torch.float32)
    c_ptr = _dev(v_cache, "v_cache", torch.bfloat16)
    v_ptr = None if v_new is None else _dev(v_new, "v_new", torch.bfloat16)
    for name, t in (("v_cache", v_cache), ("v_new", v_new)):
        if t is not None and tuple(t.shape) != (B, n):
            raise ValueError(f"{name} must be [{B}][{n}]")
    with _alloc_on(stream):
        st = torch.empty((B, 4), dtype=torch.float64, device=x.device) if stats else None
    rc = lib().w4a8_flow_step(x_ptr, v_ptr, c_ptr, B, n, float(dt), int(repeat),
                              None if st is None else st.data_ptr(), _stream(stream))
    _check(rc, "w4a8_flow_step")
    return st


def w4a8_linear_workspace_bytes(M: int, N: int, K: int, scale_mode: int = SCALE_CHANNEL_F32,
                                in_kind: int = IN_BF16) -> int:
    return int(lib().w4a8_linear_workspace_bytes(M, N, K, scale_mode, in_kind))


def w4a8_linear_describe(M: int, N: int, K: int, scale_mode: int = SCALE_CHANNEL_F32,
                         in_kind: int = IN_BF16, out_kind: int = OUT_BF16) -> str:
    return lib().w4a8_linear_describe(M, N, K, scale_mode, in_kind, out_kind).decode()


class Workspace:
    """A zero-filled device buffer reused across w4a8_linear calls (the calls
    leave its counters at zero).  Grows on demand.  Calls that share one
    Workspace must not overlap: use it from one stream at a time.

    get(nbytes, stream) returns the buffer ordered for work on `stream`: a
    grown buffer is allocated and zero-filled on that stream, and the
    caching allocator keeps every buffer (also a replaced one) from reuse
    until the work already queued on the streams that used it is done."""

    def __init__(self, device="cuda"):
        self.device = torch.device(device)
        self.buf = torch.zeros(0, dtype=torch.uint8, device=self.device)

    def get(self, nbytes: int, stream: torch.cuda.Stream | None = None) -> torch.Tensor:
        s = _torch_stream(stream, self.device)
        if nbytes > self.buf.numel():
            old = self.buf
            with torch.cuda.stream(s):
                self.buf = torch.zeros(max(nbytes, 2 * old.numel()), dtype=torch.uint8, device=self.device)
            if old.numel():
                old.record_stream(s)
        elif self.buf.numel():
            self.buf.record_stream(s)
        return self.buf


def _workspace_ptr(workspace, need: int, device, stream):
    """(pointer, bytes) of a workspace of at least `need` bytes for a call on
    `stream`: a Workspace, a caller's uint8 tensor, or None for a temporary
    buffer zero-filled on that stream (and released to the allocator on it,
    so later work on the stream cannot see it reused early)."""
    if need == 0:
        return None, 0
    s = _torch_stream(stream, device)
    if workspace is None:
        with torch.cuda.stream(s):
            buf = torch.zeros(need, dtype=torch.uint8, device=device)
    elif isinstance(workspace, Workspace):
        buf = workspace.get(need, s)
    else:
        buf = workspace
    return _dev(buf, "workspace", torch.uint8), buf.numel()


def _linear_call(entry: str, x, w_packed, w_scale, N, out_cols, x_scale, scale_mode, out_kind, out,
                 workspace, stream):
    M, K = x.shape
    if x.dtype == torch.bfloat16:
        in_kind = IN_BF16
        xs_ptr = None
    elif x.dtype == torch.int8:
        in_kind = IN_I8
        if x_scale is None:
            raise ValueError("int8 input needs x_scale")
        xs_ptr = _dev(x_scale, "x_scale", torch.float32)
    else:
        raise TypeError("x must be bf16 or int8")
    x_ptr = _dev(x, "x", x.dtype)
    wp_ptr = _dev(w_packed, "w_packed", torch.uint8)
    if w_scale is None:
        ws_ptr = None
    else:
        ws_ptr = _dev(w_scale, "w_scale", torch.float32 if scale_mode == SCALE_CHANNEL_F32 else torch.float16)
    if out is None:
        with _alloc_on(stream):
            out = torch.empty((M, out_cols), dtype=_OUT_DTYPE[out_kind], device=x.device)
    elif tuple(out.shape) != (M, out_cols):
        raise ValueError(f"out must be [{M}][{out_cols}]")
    y_ptr = _dev(out, "out", _OUT_DTYPE[out_kind])
    need = int(getattr(lib(), entry + "_workspace_bytes")(M, N, K, scale_mode, in_kind))
    wk_ptr, wk_bytes = _workspace_ptr(workspace, need, x.device, stream)
    rc = getattr(lib(), entry)(x_ptr, in_kind, xs_ptr, M, K, wp_ptr, ws_ptr, scale_mode, N, y_ptr,
                               out_kind, wk_ptr, wk_bytes, _stream(stream))
    _check(rc, entry)
    return out


def w4a8_linear(x: torch.Tensor, w_packed: torch.Tensor, w_scale: torch.Tensor | None, N: int, *,
                x_scale: torch.Tensor | None = None, scale_mode: int = SCALE_CHANNEL_F32,
                out_kind: int = OUT_BF16, out: torch.Tensor | None = None,
                workspace: Workspace | torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """y[M][N] = dequant(quant8(x) . W^T).

    x is bf16 [M][K] (quantized inside the call) or int8 codes [M][K] with
    x_scale fp32 [M].  w_scale is fp32 [N] (SCALE_CHANNEL_F32) or fp16
    [K/128][N] (SCALE_GROUP_F16).  Returns bf16, fp32 or int32 [M][N].
    """
    return _linear_call("w4a8_linear", x, w_packed, w_scale, N, N, x_scale, scale_mode, out_kind, out,
                        workspace, stream)


def w4a8_linear_noalloc(x: torch.Tensor, w_packed: torch.Tensor, w_scale: torch.Tensor | None, N: int, *,
                        x_scale: torch.Tensor | None = None, scale_mode: int = SCALE_CHANNEL_F32,
                        out_kind: int = OUT_BF16, out: torch.Tensor, stream=None) -> torch.Tensor:
    """w4a8_linear without a workspace, into a caller-given `out`: the call's
    scratch memory is the library's own per-GPU array (at most
    NOALLOC_SCRATCH_BYTES of workspace), so nothing is allocated.  Calls that
    may overlap on one GPU must not be issued."""
    M, K = x.shape
    if x.dtype == torch.bfloat16:
        in_kind, xs_ptr = IN_BF16, None
    elif x.dtype == torch.int8:
        if x_scale is None:
            raise ValueError("int8 input needs x_scale")
        in_kind, xs_ptr = IN_I8, _dev(x_scale, "x_scale", torch.float32)
    else:
        raise TypeError("x must be bf16 or int8")
    if tuple(out.shape) != (M, N):
        raise ValueError(f"out must be [{M}][{N}]")
    ws_ptr = None if w_scale is None else _dev(
        w_scale, "w_scale", torch.float32 if scale_mode == SCALE_CHANNEL_F32 else torch.float16)
    rc = lib().w4a8_linear_noalloc(_dev(x, "x", x.dtype), in_kind, xs_ptr, M, K,
                                   _dev(w_packed, "w_packed", torch.uint8), ws_ptr, scale_mode, N,
                                   _dev(out, "out", _OUT_DTYPE[out_kind]), out_kind, _stream(stream))
    _check(rc, "w4a8_linear_noalloc")
    return out


def w4a8_linear_swiglu_workspace_bytes(M: int, N: int, K: int, scale_mode: int = SCALE_CHANNEL_F32,
                                       in_kind: int = IN_BF16) -> int:
    return int(lib().w4a8_linear_swiglu_workspace_bytes(M, N, K, scale_mode, in_kind))


def w4a8_linear_swiglu_describe(M: int, N: int, K: int, scale_mode: int = SCALE_CHANNEL_F32,
                                in_kind: int = IN_BF16) -> str:
    return lib().w4a8_linear_swiglu_describe(M, N, K, scale_mode, in_kind).decode()


def w4a8_linear_swiglu(x: torch.Tensor, w_packed: torch.Tensor, w_scale: torch.Tensor | None, N: int, *,
                       x_scale: torch.Tensor | None = None, scale_mode: int = SCALE_CHANNEL_F32,
                       out_kind: int = OUT_BF16, out: torch.Tensor | None = None,
                       workspace: Workspace | torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """Fused gate+up projection with its gated activation, M <= 64:
    y[M][N/2] = silu(g) * u, where g and u are the fp32 outputs of
    w4a8_linear over weight rows [0, N/2) (gate) and [N/2, N) (up) of the
    same packed weight.  Arguments as for w4a8_linear; out_kind bf16 or fp32.
    """
    return _linear_call("w4a8_linear_swiglu", x, w_packed, w_scale, N, N // 2, x_scale, scale_mode, out_kind,
                        out, workspace, stream)


def w4a8_stream_attention(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, pos_q: torch.Tensor,
                          pos_k: torch.Tensor, rope_cos: torch.Tensor, rope_sin: torch.Tensor, scale: float,
                          out: torch.Tensor | None = None, workspace: Workspace | torch.Tensor | None = None,
                          stream=None) -> torch.Tensor:
    """Streaming prefill attention: q bf16 [H][Nq][128] and the pre-RoPE
    cache k, v bf16 [Hkv][Nk][128], int32 window positions pos_q [Nq] and
    pos_k [Nk], fp32 rotary tables [n_pos][64] -> bf16 [H][Nq][128]; key j is
    visible to query i iff pos_k[j] <= pos_q[i]."""
    H, Nq, D = q.shape
    Hkv, Nk, Dk = k.shape
    if tuple(v.shape) != (Hkv, Nk, Dk) or Dk != D:
        raise ValueError("k and v must be [Hkv][Nk][D] with q's D")
    if tuple(pos_q.shape) != (Nq,) or tuple(pos_k.shape) != (Nk,):
        raise ValueError("positions must be [Nq] and [Nk]")
    if rope_cos.shape != rope_sin.shape or rope_cos.dim() != 2 or rope_cos.shape[1] != D // 2:
        raise ValueError("rotary tables must be [n_pos][D/2]")
    if out is None:
        with _alloc_on(stream):
            out = torch.empty((H, Nq, D), dtype=torch.bfloat16, device=q.device)
    elif tuple(out.shape) != (H, Nq, D):
        raise ValueError(f"out must be [{H}][{Nq}][{D}]")
    need = int(lib().w4a8_stream_attention_workspace_bytes(H, Nq, Nk)) if Nq else 0
    wk_ptr, wk_bytes = _workspace_ptr(workspace, need, q.device, stream)
    rc = lib().w4a8_stream_attention(_dev(q, "q", torch.bfloat16), _dev(k, "k", torch.bfloat16),
                                     _dev(v, "v", torch.bfloat16), _dev(pos_q, "pos_q", torch.int32),
                                     _dev(pos_k, "pos_k", torch.int32), _dev(rope_cos, "rope_cos", torch.float32),
                                     _dev(rope_sin, "rope_sin", torch.float32), rope_cos.shape[0], H, Hkv, Nq, Nk, D,
                                     float(scale), _dev(out, "out", torch.bfloat16), wk_ptr, wk_bytes, _stream(stream))
    _check(rc, "w4a8_stream_attention")
    return out


def w4a8_stream_attention_workspace_bytes(H: int, Nq: int, Nk: int) -> int:
    return int(lib().w4a8_stream_attention_workspace_bytes(H, Nq, Nk))
