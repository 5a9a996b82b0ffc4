"""Python binding of liblayerdrop (MI355X / gfx950 layer-dropout hot path).

Argument marshalling only: every function here has the name of a C entry
point in include/layerdrop.h, converts torch tensors to device pointers and
the current torch stream to a hipStream_t, calls the library, and raises
LdError on a non-zero status.  All computation happens in the HIP kernels;
there is no fallback -- importing fails loudly when the library is not built.
"""

import ctypes as C
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liblayerdrop.so")

LD_F32, LD_BF16 = 0, 1
LD_GRAN_LAYER_SEQ, LD_GRAN_SUBLAYER_SEQ, LD_GRAN_LAYER_BATCH, LD_GRAN_SUBLAYER_BATCH = 0, 1, 2, 3
UNIFORM, ILD, ALD = 0, 1, 2
CONSTANT, ITS, DTS = 0, 1, 2

WEIGHT_KEYS = ("g_attn", "w_qkv", "w_o", "g_mlp", "w_gate_up", "w_down")


class LdError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"{status_name(status)}: {msg}")
        self.status = status


class ld_config(C.Structure):
    _fields_ = [("batch", C.c_int32), ("seq", C.c_int32), ("d_model", C.c_int32),
                ("n_heads", C.c_int32), ("d_ff", C.c_int32), ("dtype", C.c_int32),
                ("rms_eps", C.c_float), ("rescale", C.c_int32), ("res_scale", C.c_float),
                ("block_kind", C.c_int32), ("granularity", C.c_int32)]


class ld_weights(C.Structure):
    _fields_ = [(k, C.c_void_p) for k in WEIGHT_KEYS]


class ld_grads(C.Structure):
    _fields_ = [(k, C.c_void_p) for k in WEIGHT_KEYS]


if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is not built; run `python paper_2609_05275_amd/build.py`")
_lib = C.CDLL(LIB_PATH)

_vp, _i32, _i64, _u64, _f32, _sz = C.c_void_p, C.c_int32, C.c_int64, C.c_uint64, C.c_float, C.c_size_t
_PCFG = C.POINTER(ld_config)
_SIGS = {
    "ld_status_string": (C.c_char_p, [C.c_int]),
    "ld_last_error": (C.c_char_p, []),
    "ld_schedule_p": (C.c_int, [_i32, _i32, _f32, _i32, _i32, _i64, _i64, C.POINTER(_f32)]),
    "ld_masks": (C.c_int, [_i32, _i32, C.POINTER(_f32), _i32, _u64, _u64, _vp, _vp, _vp, _vp]),
    "ld_masks_granular": (C.c_int, [_i32, _i32, _i32, C.POINTER(_f32), _i32, _u64, _u64, _vp, _vp,
                                    _vp, _vp]),
    "ld_gather_rows": (C.c_int, [_PCFG, _vp, _vp, _vp, _vp, _vp]),
    "ld_scatter_add_rows": (C.c_int, [_PCFG, _vp, _vp, _f32, _vp, _vp, _vp]),
    "ld_layer_ctx_bytes": (_sz, [_PCFG]),
    "ld_layer_ws_bytes": (_sz, [_PCFG]),
    "ld_stack_ws_bytes": (_sz, [_PCFG, _i32]),
    "ld_layer_fwd": (C.c_int, [_PCFG, C.POINTER(ld_weights), _i32, _f32, _u64, _u64, _vp, _vp,
                               _vp, _sz, _vp, _vp]),
    "ld_layer_bwd": (C.c_int, [_PCFG, C.POINTER(ld_weights), _vp, _vp, C.POINTER(ld_grads), _vp,
                               _sz, _vp]),
    "ld_stack_step": (C.c_int, [_PCFG, _i32, C.POINTER(ld_weights), C.POINTER(_f32), _u64, _u64,
                                _vp, _vp, C.POINTER(ld_grads), _vp, _sz, _vp, _vp, _vp, _vp, _vp]),
    "ld_rmsnorm_fwd": (C.c_int, [_i32, _i32, _i32, _f32, _vp, _vp, _vp, _vp, _vp]),
    "ld_rmsnorm_bwd_ws_bytes": (_sz, [_i32, _i32]),
    "ld_rmsnorm_bwd": (C.c_int, [_i32, _i32, _i32, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _sz,
                                 _vp]),
    "ld_relu2_fwd": (C.c_int, [_i32, _i32, _i32, _vp, _vp, _vp]),
    "ld_relu2_bwd": (C.c_int, [_i32, _i32, _i32, _vp, _vp, _vp, _vp]),
    "ld_alibi_slope": (C.c_float, [_i32, _i32]),
    "ld_swiglu_fwd": (C.c_int, [_i32, _i32, _i32, _vp, _vp, _vp]),
    "ld_swiglu_bwd": (C.c_int, [_i32, _i32, _i32, _vp, _vp, _vp, _vp]),
    "ld_gemm_ws_bytes": (_sz, [_i32, _i32, _i32, _i32, _i32, _i32, _i32, _i32]),
    "ld_gemm": (C.c_int, [_i32, _i32, _i32, _i32, _i32, _i32, _vp, _i32, _vp, _i32, _vp, _i32,
                          _i32, _f32, _vp, _i32, _vp, _sz, _vp]),
    "ld_attn_fwd": (C.c_int, [_i32, _i32, _i32, _i32, _i32, _i32, _vp, _vp, _vp, _vp]),
    "ld_attn_bwd_ws_bytes": (_sz, [_i32, _i32, _i32]),
    "ld_attn_bwd": (C.c_int, [_i32, _i32, _i32, _i32, _i32, _i32, _vp, _vp, _vp, _vp, _vp, _vp,
                              _sz, _vp]),
    "ld_attn_bwd_noalloc": (C.c_int, [_i32, _i32, _i32, _i32, _i32, _i32, _vp, _vp, _vp, _vp, _vp,
                                      _vp]),
    "ld_eval_ws_bytes": (_sz, [_PCFG]),
    "ld_stack_eval": (C.c_int, [_PCFG, _i32, C.POINTER(ld_weights), _vp, _vp, _vp, _vp, _i32, _vp,
                                _sz, _vp]),
    "ld_decode_ws_bytes": (_sz, [_PCFG, _i32, _i32]),
    "ld_stack_decode": (C.c_int, [_PCFG, _i32, C.POINTER(ld_weights), _vp, _vp, _vp, _vp, _i32,
                                  _i32, _i32, _vp, _sz, _vp]),
    "ld_gemm_skinny_ws_bytes": (_sz, [_i32, _i32, _i32]),
    "ld_gemm_skinny": (C.c_int, [_i32, _i32, _i32, _vp, _i32, _vp, _i32, _vp, _i32, _f32, _vp, _i32,
                                 _vp, _sz, _vp]),
    "ld_gemm_dec": (C.c_int, [_i32, _i32, _i32, _vp, _i32, _vp, _f32, _vp, _i32, _vp, _i32, _f32, _vp, _i32,
                              _i32, _vp]),
    "ld_kv_store": (C.c_int, [_i32, _i32, _i32, _i32, _vp, _vp, _i32, _vp]),
    "ld_attn_decode_ws_bytes": (_sz, [_i32, _i32, _i32, _i32]),
    "ld_attn_decode": (C.c_int, [_i32, _i32, _i32, _i32, _i32, _i32, _vp, _vp, _i32, _vp, _vp, _sz,
                                 _vp]),
    "ld_prof_start": (C.c_int, [C.c_char_p]),
    "ld_prof_stop": (C.c_int, []),
    "ld_prof_result": (C.c_int, [C.POINTER(_i64), C.POINTER(C.c_double), C.POINTER(C.c_double),
                                 C.POINTER(C.c_double)]),
}
for _name, (_res, _args) in _SIGS.items():
    _fn = getattr(_lib, _name)
    _fn.restype = _res
    _fn.argtypes = _args

EXPORTED = tuple(_SIGS)


def status_name(status):
    return _lib.ld_status_string(status).decode()


def last_error():
    return _lib.ld_last_error().decode()


def _check(status):
    if status != 0:
        raise LdError(status, last_error())


def _ptr(t, name="tensor", inner=False):
    """Device address of t.  A torch tensor must live on the GPU and be
    contiguous (with inner=True, for calls that take a leading dimension,
    only its last dimension must be); anything else -- a raw address (int) or
    an object with data_ptr() -- is passed through for the library to check."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    if isinstance(t, torch.Tensor):
        if not t.is_cuda:
            raise ValueError(f"{name}: a device tensor is required, got one on {t.device}")
        if inner:
            if t.dim() and t.stride(-1) != 1 and t.numel() > 1:
                raise ValueError(f"{name}: the last dimension must be contiguous")
        elif not t.is_contiguous():
            raise ValueError(f"{name}: a contiguous tensor is required")
    return t.data_ptr()


_TORCH_OF = {LD_F32: torch.float32, LD_BF16: torch.bfloat16}


def _need(t, name, dtype=None, numel=None, min_bytes=None):
    """Checks a torch tensor argument against what the call reads or writes
    (dtype, element count, byte size) before anything is launched; other
    objects pass through to the library's own checks."""
    if not isinstance(t, torch.Tensor):
        return
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name}: dtype {t.dtype}, expected {dtype}")
    if numel is not None and t.numel() != numel:
        raise ValueError(f"{name}: {t.numel()} elements, expected {numel}")
    if min_bytes is not None and t.numel() * t.element_size() < min_bytes:
        raise ValueError(f"{name}: {t.numel() * t.element_size()} bytes, at least {min_bytes} needed")


def _n_masks(cfg):
    return 2 if cfg.granularity & LD_GRAN_SUBLAYER_SEQ else 1


def _weight_numel(cfg):
    d, f = cfg.d_model, cfg.d_ff
    return dict(g_attn=d, w_qkv=3 * d * d, w_o=d * d, g_mlp=d,
                w_gate_up=(2 if cfg.block_kind == 0 else 1) * f * d, w_down=d * f)


def _check_layer_tensors(cfg, w=None, dw=None, acts=()):
    dt = _TORCH_OF.get(cfg.dtype)
    n = _weight_numel(cfg)
    for k in WEIGHT_KEYS:
        if w is not None:
            _need(w[k], k, dt, n[k])
        if dw is not None:
            _need(dw[k], "grad " + k, torch.float32, n[k])
    for name, t in acts:
        _need(t, name, dt, cfg.batch * cfg.seq * cfg.d_model)


def _stream(stream):
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _dtype_code(t):
    if t.dtype == torch.bfloat16:
        return LD_BF16
    if t.dtype == torch.float32:
        return LD_F32
    raise TypeError(f"unsupported dtype {t.dtype}")


def config(batch, seq, d_model, n_heads, d_ff, dtype=LD_BF16, rms_eps=1e-5, rescale=True,
           res_scale=1.0, block_kind=0, granularity=0):
    return ld_config(batch, seq, d_model, n_heads, d_ff, dtype, rms_eps, int(bool(rescale)),
                     res_scale, block_kind, granularity)


def weights(w):
    """ld_weights from a dict of device tensors keyed by WEIGHT_KEYS."""
    return ld_weights(*[_ptr(w[k], k) for k in WEIGHT_KEYS])


def grads(g):
    return ld_grads(*[_ptr(g[k], "grad " + k) for k in WEIGHT_KEYS])


# ------------------------------------------------------------------ entry points

def ld_schedule_p(dist, sched, p_max, layer, n_layers, t, n_steps):
    out = C.c_float()
    _check(_lib.ld_schedule_p(dist, sched, p_max, layer, n_layers, t, n_steps, C.byref(out)))
    return out.value


def ld_masks(p, seed, step, keep, idx, count, first_layer=0, stream=None):
    n = len(p)
    arr = (C.c_float * n)(*[float(v) for v in p])
    B = keep.shape[-1]
    _need(keep, "keep", torch.uint8, n * B)
    _need(idx, "idx", torch.int32, n * B)
    _need(count, "count", torch.int32, n)
    _check(_lib.ld_masks(n, B, arr, first_layer, seed, step, _ptr(keep, "keep"), _ptr(idx, "idx"),
                         _ptr(count, "count"), _stream(stream)))


def ld_masks_granular(granularity, p, seed, step, keep, idx, count, first_layer=0, stream=None):
    n = len(p)
    arr = (C.c_float * n)(*[float(v) for v in p])
    B = keep.shape[-1]
    nm = 2 if granularity in (LD_GRAN_SUBLAYER_SEQ, LD_GRAN_SUBLAYER_BATCH) else 1
    _need(keep, "keep", torch.uint8, n * nm * B)
    _need(idx, "idx", torch.int32, n * nm * B)
    _need(count, "count", torch.int32, n * nm)
    _check(_lib.ld_masks_granular(granularity, n, B, arr, first_layer, seed, step,
                                  _ptr(keep, "keep"), _ptr(idx, "idx"), _ptr(count, "count"),
                                  _stream(stream)))


def ld_gather_rows(cfg, idx, count, x, xk, stream=None):
    _need(idx, "idx", torch.int32, cfg.batch)
    _need(count, "count", torch.int32, 1)
    _check_layer_tensors(cfg, acts=(("x", x), ("xk", xk)))
    _check(_lib.ld_gather_rows(C.byref(cfg), _ptr(idx, "idx"), _ptr(count, "count"), _ptr(x, "x"),
                               _ptr(xk, "xk"), _stream(stream)))


def ld_scatter_add_rows(cfg, idx, count, r, yk, x, stream=None):
    _need(idx, "idx", torch.int32, cfg.batch)
    _need(count, "count", torch.int32, 1)
    _check_layer_tensors(cfg, acts=(("yk", yk), ("x", x)))
    _check(_lib.ld_scatter_add_rows(C.byref(cfg), _ptr(idx, "idx"), _ptr(count, "count"), r,
                                    _ptr(yk, "yk"), _ptr(x, "x"), _stream(stream)))


def ld_layer_ctx_bytes(cfg):
    return _lib.ld_layer_ctx_bytes(C.byref(cfg))


def ld_layer_ws_bytes(cfg):
    return _lib.ld_layer_ws_bytes(C.byref(cfg))


def ld_stack_ws_bytes(cfg, n_layers):
    return _lib.ld_stack_ws_bytes(C.byref(cfg), n_layers)


def ld_layer_fwd(cfg, w, layer, p, seed, step, x, ctx, ws=None, keep_override=None, stream=None):
    _check_layer_tensors(cfg, w=w, acts=(("x", x),))
    _need(ctx, "ctx", min_bytes=ld_layer_ctx_bytes(cfg))
    _need(keep_override, "keep_override", torch.uint8, _n_masks(cfg) * cfg.batch)
    wb = weights(w)
    ws_bytes = 0 if ws is None else ws.numel() * ws.element_size()
    _check(_lib.ld_layer_fwd(C.byref(cfg), C.byref(wb), layer, p, seed, step, _ptr(x), _ptr(ctx),
                             _ptr(ws), ws_bytes, _ptr(keep_override), _stream(stream)))


def ld_layer_bwd(cfg, w, ctx, dx, dw, ws, stream=None):
    _check_layer_tensors(cfg, w=w, dw=dw, acts=(("dx", dx),))
    _need(ctx, "ctx", min_bytes=ld_layer_ctx_bytes(cfg))
    wb, gb = weights(w), grads(dw)
    _check(_lib.ld_layer_bwd(C.byref(cfg), C.byref(wb), _ptr(ctx), _ptr(dx), C.byref(gb),
                             _ptr(ws), ws.numel() * ws.element_size(), _stream(stream)))


def ld_stack_step(cfg, ws_list, p, seed, step, x, dx, dw_list, ws, keep_override=None,
                  keep_out=None, idx_out=None, count_out=None, stream=None):
    L = len(ws_list)
    if len(dw_list) != L or len(p) != L:
        raise ValueError(f"{L} layers of weights, {len(dw_list)} of gradients, {len(p)} rates")
    for l in range(L):
        _check_layer_tensors(cfg, w=ws_list[l], dw=dw_list[l])
    _check_layer_tensors(cfg, acts=(("x", x), ("dx", dx)))
    nmb = L * _n_masks(cfg) * cfg.batch
    _need(keep_override, "keep_override", torch.uint8, nmb)
    _need(keep_out, "keep_out", torch.uint8, nmb)
    _need(idx_out, "idx_out", torch.int32, nmb)
    _need(count_out, "count_out", torch.int32, L * _n_masks(cfg))
    wa = (ld_weights * L)(*[weights(w) for w in ws_list])
    ga = (ld_grads * L)(*[grads(g) for g in dw_list])
    pa = (C.c_float * L)(*[float(v) for v in p])
    _check(_lib.ld_stack_step(C.byref(cfg), L, wa, pa, seed, step, _ptr(x), _ptr(dx), ga, _ptr(ws),
                              ws.numel() * ws.element_size(), _ptr(keep_override), _ptr(keep_out),
                              _ptr(idx_out), _ptr(count_out), _stream(stream)))


def _u8_array(v, n):
    if v is None:
        return None
    return (C.c_uint8 * n)(*[1 if a else 0 for a in v])


def _f32_array(v, n):
    if v is None:
        return None
    if isinstance(v, (int, float)):
        v = [v] * n
    return (C.c_float * n)(*[float(a) for a in v])


def _ptr_array(v, n):
    if v is None:
        return None
    return (C.c_void_p * n)(*[_ptr(t) for t in v])


def ld_eval_ws_bytes(cfg):
    return _lib.ld_eval_ws_bytes(C.byref(cfg))


def ld_stack_eval(cfg, ws_list, x, ws, active=None, r_eval=None, kv=None, s_max=0, stream=None):
    """Forward-only evaluation form over the active layers; kv: list of
    per-layer caches (None entries allowed for inactive layers)."""
    L = len(ws_list)
    wa = (ld_weights * L)(*[weights(w) for w in ws_list])
    act, rr, kk = _u8_array(active, L), _f32_array(r_eval, L), _ptr_array(kv, L)
    _check(_lib.ld_stack_eval(C.byref(cfg), L, wa, act, rr, _ptr(x), kk, s_max, _ptr(ws),
                              ws.numel() * ws.element_size(), _stream(stream)))


def ld_decode_ws_bytes(cfg, n_new, s_max):
    return _lib.ld_decode_ws_bytes(C.byref(cfg), n_new, s_max)


def ld_stack_decode(cfg, ws_list, x, kv, s_max, pos, n_new, ws, active=None, r_eval=None,
                    stream=None):
    L = len(ws_list)
    wa = (ld_weights * L)(*[weights(w) for w in ws_list])
    act, rr, kk = _u8_array(active, L), _f32_array(r_eval, L), _ptr_array(kv, L)
    _check(_lib.ld_stack_decode(C.byref(cfg), L, wa, act, rr, _ptr(x), kk, s_max, pos, n_new,
                                _ptr(ws), ws.numel() * ws.element_size(), _stream(stream)))


def ld_gemm_skinny_ws_bytes(M, N, K):
    return _lib.ld_gemm_skinny_ws_bytes(M, N, K)


def ld_gemm_skinny(A, W, C_out, alpha=1.0, R=None, ws=None, stream=None):
    M, K = A.shape
    N = W.shape[0]
    _check(_lib.ld_gemm_skinny(M, N, K, _ptr(A, "A", inner=True), A.stride(0),
                               _ptr(W, "W", inner=True), W.stride(0), _ptr(C_out, "C_out", inner=True),
                               C_out.stride(0), alpha, _ptr(R, "R", inner=True),
                               0 if R is None else R.stride(0), _ptr(ws, "ws"),
                               0 if ws is None else ws.numel() * ws.element_size(), _stream(stream)))


DEC_ACT_NONE, DEC_ACT_SWIGLU, DEC_ACT_RELU2 = 0, 1, 2


def ld_gemm_dec(A, W, C_out, g=None, eps=1e-5, alpha=1.0, R=None, act=DEC_ACT_NONE, stream=None):
    """Fused decoding projection (M <= 8 rows): C = act(R + alpha A' W^T), A'
    the RMSNorm of A's rows with gain g when g is given; with SwiGLU W holds
    the gate rows then the up rows and C has half as many columns."""
    M, K = A.shape
    N = C_out.shape[1]
    _check(_lib.ld_gemm_dec(M, N, K, _ptr(A, "A", inner=True), A.stride(0), _ptr(g, "g"), eps,
                            _ptr(W, "W", inner=True), W.stride(0), _ptr(C_out, "C_out", inner=True),
                            C_out.stride(0), alpha, _ptr(R, "R", inner=True),
                            0 if R is None else R.stride(0), act, _stream(stream)))


def ld_kv_store(n_seq, n_new, d_model, pos, qkv, kv, s_max, stream=None):
    _check(_lib.ld_kv_store(n_seq, n_new, d_model, pos, _ptr(qkv), _ptr(kv), s_max, _stream(stream)))


def ld_attn_decode_ws_bytes(n_seq, n_heads, d_head, s_max):
    return _lib.ld_attn_decode_ws_bytes(n_seq, n_heads, d_head, s_max)


def ld_attn_decode(n_seq, n_heads, d_head, pos, n_new, qkv, kv, s_max, o, ws, alibi=0, stream=None):
    _check(_lib.ld_attn_decode(n_seq, n_heads, d_head, alibi, pos, n_new, _ptr(qkv), _ptr(kv), s_max,
                               _ptr(o), _ptr(ws), ws.numel() * ws.element_size(), _stream(stream)))


def ld_rmsnorm_fwd(x, g, y, rstd, eps=1e-5, stream=None):
    rows, d = x.shape
    _check(_lib.ld_rmsnorm_fwd(_dtype_code(x), rows, d, eps, _ptr(x), _ptr(g), _ptr(y), _ptr(rstd),
                               _stream(stream)))


def ld_rmsnorm_bwd_ws_bytes(rows, d):
    return _lib.ld_rmsnorm_bwd_ws_bytes(rows, d)


def ld_rmsnorm_bwd(x, g, rstd, gy, gres, gx, dg, ws, stream=None):
    rows, d = x.shape
    _check(_lib.ld_rmsnorm_bwd(_dtype_code(x), rows, d, _ptr(x), _ptr(g), _ptr(rstd), _ptr(gy),
                               _ptr(gres), _ptr(gx), _ptr(dg), _ptr(ws),
                               ws.numel() * ws.element_size(), _stream(stream)))


def ld_relu2_fwd(u, s, stream=None):
    rows, f = u.shape
    _check(_lib.ld_relu2_fwd(_dtype_code(u), rows, f, _ptr(u), _ptr(s), _stream(stream)))


def ld_relu2_bwd(u, gs, gu, stream=None):
    rows, f = u.shape
    _check(_lib.ld_relu2_bwd(_dtype_code(u), rows, f, _ptr(u), _ptr(gs), _ptr(gu),
                             _stream(stream)))


def ld_alibi_slope(h, n_heads):
    return _lib.ld_alibi_slope(h, n_heads)


def ld_swiglu_fwd(uv, s, stream=None):
    rows, f2 = uv.shape
    _check(_lib.ld_swiglu_fwd(_dtype_code(uv), rows, f2 // 2, _ptr(uv), _ptr(s), _stream(stream)))


def ld_swiglu_bwd(uv, gs, guv, stream=None):
    rows, f2 = uv.shape
    _check(_lib.ld_swiglu_bwd(_dtype_code(uv), rows, f2 // 2, _ptr(uv), _ptr(gs), _ptr(guv),
                              _stream(stream)))


def ld_gemm_ws_bytes(dtype, a_kcontig, b_kcontig, M, N, K, ldc, c_f32):
    return _lib.ld_gemm_ws_bytes(dtype, int(a_kcontig), int(b_kcontig), M, N, K, ldc, int(c_f32))


def ld_gemm(a_kcontig, b_kcontig, M, N, K, A, lda, B, ldb, Cm, ldc, alpha=1.0, R=None, ldr=0,
            c_f32=False, dtype=None, ws=None, stream=None):
    dt = _dtype_code(A) if dtype is None else dtype
    ws_bytes = 0 if ws is None else ws.numel() * ws.element_size()
    _check(_lib.ld_gemm(dt, int(a_kcontig), int(b_kcontig), M, N, K, _ptr(A, "A", inner=True), lda,
                        _ptr(B, "B", inner=True), ldb, _ptr(Cm, "C", inner=True), ldc, int(c_f32), alpha,
                        _ptr(R, "R", inner=True), ldr, _ptr(ws, "ws"), ws_bytes, _stream(stream)))


def ld_attn_fwd(n_seq, seq, n_heads, d_head, qkv, o, lse, stream=None, alibi=0):
    _check(_lib.ld_attn_fwd(_dtype_code(qkv), n_seq, seq, n_heads, d_head, int(alibi), _ptr(qkv),
                            _ptr(o), _ptr(lse), _stream(stream)))


def ld_attn_bwd_ws_bytes(n_seq, seq, n_heads):
    return _lib.ld_attn_bwd_ws_bytes(n_seq, seq, n_heads)


def ld_attn_bwd(n_seq, seq, n_heads, d_head, qkv, o, lse, go, gqkv, ws, stream=None, alibi=0):
    _check(_lib.ld_attn_bwd(_dtype_code(qkv), n_seq, seq, n_heads, d_head, int(alibi), _ptr(qkv),
                            _ptr(o), _ptr(lse), _ptr(go), _ptr(gqkv), _ptr(ws),
                            ws.numel() * ws.element_size(), _stream(stream)))


def ld_attn_bwd_noalloc(n_seq, seq, n_heads, d_head, qkv, o, lse, go, gqkv, stream=None, alibi=0):
    _check(_lib.ld_attn_bwd_noalloc(_dtype_code(qkv), n_seq, seq, n_heads, d_head, int(alibi),
                                    _ptr(qkv, "qkv"), _ptr(o, "o"), _ptr(lse, "lse"), _ptr(go, "go"),
                                    _ptr(gqkv, "gqkv"), _stream(stream)))


def ld_prof_start(kernel_name):
    _check(_lib.ld_prof_start(kernel_name.encode()))


def ld_prof_stop():
    _check(_lib.ld_prof_stop())


def ld_prof_result():
    n, ms, fl, by = C.c_int64(), C.c_double(), C.c_double(), C.c_double()
    _check(_lib.ld_prof_result(C.byref(n), C.byref(ms), C.byref(fl), C.byref(by)))
    return dict(launches=n.value, ms=ms.value, flops=fl.value, bytes=by.value)
