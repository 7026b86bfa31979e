"""Python binding of libtfm (include/tfm.h): argument marshalling only.

Every function has the name of the C entry point it calls, takes and returns
torch tensors on the current HIP device, enqueues on torch's current stream
and raises ``TfmError`` with the library's status text when the library
rejects a call.  Nothing here computes any part of the method: all of it runs
in the HIP kernels of libtfm.so, which must have been built (see
``__graft_entry__.build``); ``lib()`` raises if it is missing.
"""
import ctypes
import math
import os

import torch

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libtfm.so")

TFM_F32 = 0
TFM_BF16 = 1
_DTYPES = {torch.float32: TFM_F32, torch.bfloat16: TFM_BF16}

# Query-scale modes of tfm_icl_options.q_scale_mode.
Q_SCALE_MODES = {"shared": 0, "per_call": 1, "joint": 2}


class tfm_icl_options(ctypes.Structure):
    _fields_ = [("q_scale_mode", ctypes.c_int), ("test_kv_heads", ctypes.c_int)]


def _opts(q_scale_mode="shared", test_kv_heads=0):
    """A tfm_icl_options by reference; an unknown mode name raises ValueError here,
    anything else the library checks."""
    if q_scale_mode not in Q_SCALE_MODES:
        raise ValueError("q_scale_mode must be one of %s" % sorted(Q_SCALE_MODES))
    return ctypes.byref(tfm_icl_options(Q_SCALE_MODES[q_scale_mode], int(test_kv_heads or 0)))

# name -> (restype, argtypes), in the order of include/tfm.h
_c_int, _c_size, _c_float, _p = ctypes.c_int, ctypes.c_size_t, ctypes.c_float, ctypes.c_void_p
_o = ctypes.POINTER(tfm_icl_options)
SIGNATURES = {
    "tfm_status_string": (ctypes.c_char_p, [_c_int]),
    "tfm_version": (_c_int, []),
    "tfm_quantize_workspace_bytes": (_c_size, [_c_int, _c_int]),
    "tfm_quantize_qkv_per_head": (_c_int, [_c_int, _o] + [_c_int] * 5 + [_p] * 13 + [_c_size, _p]),
    "tfm_icl_attention_fp8_workspace_bytes": (_c_size, [_c_int] * 5),
    "tfm_icl_attention_fp8": (_c_int, [_c_int, _c_int, _o] + [_c_int] * 5 + [_c_float] + [_p] * 7 + [_c_size, _p]),
    "tfm_icl_attention_fp8_quantize": (_c_int, [_c_int, _o] + [_c_int] * 5 + [_p] * 5 + [_c_size, _p]),
    "tfm_icl_attention_fp8_attend": (_c_int, [_c_int, _o] + [_c_int] * 5 + [_c_float] + [_p] * 3 + [_c_size, _p]),
    "tfm_icl_attention_fp8_prequantized_workspace_bytes": (_c_size, [_c_int] * 4),
    "tfm_icl_attention_fp8_prequantized": (_c_int, [_c_int, _o] + [_c_int] * 5 + [_c_float] + [_p] * 11
                                           + [_c_size, _p]),
    "tfm_icl_attention_fp8_block_kv": (_c_int, [_c_int]),
    "tfm_icl_attention_bf16": (_c_int, [_c_int, _c_int, _o] + [_c_int] * 5 + [_c_float] + [_p] * 6 + [_p]),
    "tfm_icl_attention_workspace_bytes": (_c_size, [_c_int] * 6),
    "tfm_icl_attention": (_c_int, [_c_int, _c_int, _o] + [_c_int] * 5 + [_c_float] + [_p] * 6
                          + [_c_int, ctypes.POINTER(_c_int), _p, _c_size, _p]),
    "tfm_icl_attention_fp8_noalloc": (_c_int, [_c_int, _c_int, _o] + [_c_int] * 5 + [_c_float] + [_p] * 6 + [_p]),
    "tfm_icl_attention_fp8_fit": (_c_int, [_c_int, _c_int, _o] + [_c_int] * 4 + [_c_float] + [_p] * 5
                                  + [_c_size, _p]),
    "tfm_icl_attention_fp8_predict": (_c_int, [_c_int, _c_int, _o] + [_c_int] * 5 + [_c_float] + [_p] * 3
                                      + [_c_size, _p]),
    "tfm_noise_per_head_workspace_bytes": (_c_size, [_c_int] * 4),
    "tfm_noise_per_head": (_c_int, [_c_int] * 6 + [_p, _p, _c_float, _p, _p, _p, _c_size, _p]),
}


class TfmError(RuntimeError):
    def __init__(self, status, where):
        self.status = status
        super().__init__("%s: %s" % (where, lib().tfm_status_string(status).decode()))


_lib = None


def lib():
    """The loaded libtfm (ctypes.CDLL); raises if the library has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError("libtfm.so not found at %s: build it with __graft_entry__.build()" % LIB_PATH)
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            f = getattr(L, name)
            f.restype, f.argtypes = res, args
        _lib = L
    return _lib


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _call(name, *args):
    st = getattr(lib(), name)(*args)
    if st != 0:
        raise TfmError(st, name)


def _shape_bnhd(x, what):
    if x.dim() != 4:
        raise ValueError("%s must be (B, rows, H, D)" % what)
    return x.shape


def _check_inputs(tensors, dtype=None):
    dev = None
    for name, t in tensors.items():
        if t is None:
            continue
        if not t.is_cuda:
            raise ValueError("%s must be a GPU tensor" % name)
        if not t.is_contiguous():
            raise ValueError("%s must be contiguous" % name)
        if dtype is not None and t.dtype != dtype:
            raise ValueError("%s must be %s" % (name, dtype))
        if dev is None:
            dev = t.device
        elif t.device != dev:
            raise ValueError("all tensors must be on one device")
    if dev is not None and dev.index is not None and dev.index != torch.cuda.current_device():
        raise ValueError("tensors must be on the current device (the library enqueues on its current stream)")
    return dev


def _qkv_dims(q_train, k, v, q_test):
    B, N, H, D = _shape_bnhd(q_train, "q_train")
    if tuple(k.shape) != (B, N, H, D) or tuple(v.shape) != (B, N, H, D):
        raise ValueError("k and v must have the shape of q_train")
    M = 0
    if q_test is not None:
        Bt, M, Ht, Dt = _shape_bnhd(q_test, "q_test")
        if (Bt, Ht, Dt) != (B, H, D):
            raise ValueError("q_test must be (B, M, H, D)")
        if M == 0:
            q_test = None
    return B, H, D, N, M, q_test


def _alpha(alpha, D):
    return float(1.0 / math.sqrt(D)) if alpha is None else float(alpha)


def tfm_version():
    return lib().tfm_version()


def tfm_icl_attention_fp8_block_kv(D):
    return lib().tfm_icl_attention_fp8_block_kv(int(D))


def tfm_quantize_workspace_bytes(B, H):
    return lib().tfm_quantize_workspace_bytes(B, H)


def tfm_icl_attention_fp8_workspace_bytes(B, H, D, N, M):
    return lib().tfm_icl_attention_fp8_workspace_bytes(B, H, D, N, M)


def tfm_icl_attention_fp8_prequantized_workspace_bytes(B, H, D, N):
    return lib().tfm_icl_attention_fp8_prequantized_workspace_bytes(B, H, D, N)


def tfm_quantize_qkv_per_head(q_train, k, v, q_test=None, q_scale_mode="shared"):
    """Eq. (2) per (b, h): returns dict q8_train, k8, v8, q8_test ((B,H,rows,D) uint8) and s_q, s_k, s_v,
    s_q_test ((B,H) fp32; s_q_test is the scale the test queries were quantized with)."""
    B, H, D, N, M, q_test = _qkv_dims(q_train, k, v, q_test)
    if q_train.dtype not in _DTYPES:
        raise ValueError("inputs must be float32 or bfloat16")
    dev = _check_inputs({"q_train": q_train, "k": k, "v": v, "q_test": q_test}, q_train.dtype)
    u8 = dict(dtype=torch.uint8, device=dev)
    out = {"q8_train": torch.empty((B, H, N, D), **u8), "k8": torch.empty((B, H, N, D), **u8),
           "v8": torch.empty((B, H, N, D), **u8),
           "q8_test": torch.empty((B, H, M, D), **u8) if M else None,
           "s_q": torch.empty((B, H), dtype=torch.float32, device=dev),
           "s_k": torch.empty((B, H), dtype=torch.float32, device=dev),
           "s_v": torch.empty((B, H), dtype=torch.float32, device=dev),
           "s_q_test": torch.empty((B, H), dtype=torch.float32, device=dev)}
    nws = tfm_quantize_workspace_bytes(B, H)
    ws = torch.empty(nws, **u8)
    _call("tfm_quantize_qkv_per_head", _DTYPES[q_train.dtype], _opts(q_scale_mode), B, H, D, N, M, _ptr(q_train),
          _ptr(k), _ptr(v), _ptr(q_test), _ptr(out["q8_train"]), _ptr(out["k8"]), _ptr(out["v8"]),
          _ptr(out["q8_test"]), _ptr(out["s_q"]), _ptr(out["s_k"]), _ptr(out["s_v"]), _ptr(out["s_q_test"]),
          _ptr(ws), nws, _stream())
    if out["q8_test"] is None:
        out["q8_test"] = torch.empty((B, H, 0, D), **u8)
    return out


def _outputs(B, H, D, N, M, out_dtype, dev, out):
    if out is not None:
        o_tr, o_te = out
        if o_te is None:
            o_te = torch.empty((B, 0, H, D), dtype=out_dtype, device=dev)
        for t, rows in ((o_tr, N), (o_te, M)):
            if tuple(t.shape) != (B, rows, H, D) or t.dtype != out_dtype or not t.is_contiguous():
                raise ValueError("output tensors must be contiguous (B, rows, H, D) of the output dtype")
    else:
        o_tr = torch.empty((B, N, H, D), dtype=out_dtype, device=dev)
        o_te = torch.empty((B, M, H, D), dtype=out_dtype, device=dev)
    return o_tr, o_te


def tfm_icl_attention_fp8(q_train, k, v, q_test=None, alpha=None, out_dtype=torch.float32, out=None, workspace=None,
                          q_scale_mode="shared", test_kv_heads=0):
    """Quantize (Eq. (2)) and run both ICL calls in FP8; returns (o_train (B,N,H,D), o_test (B,M,H,D)).

    q_scale_mode: "shared" (test queries on the train-query scale), "per_call" (their own
    scale) or "joint" (one scale over train and test queries).  test_kv_heads G (0 = H):
    test queries of head h attend to K/V head h // (H // G)."""
    B, H, D, N, M, q_test = _qkv_dims(q_train, k, v, q_test)
    if q_train.dtype not in _DTYPES or out_dtype not in _DTYPES:
        raise ValueError("inputs and outputs must be float32 or bfloat16")
    dev = _check_inputs({"q_train": q_train, "k": k, "v": v, "q_test": q_test}, q_train.dtype)
    o_tr, o_te = _outputs(B, H, D, N, M, out_dtype, dev, out)
    nws = tfm_icl_attention_fp8_workspace_bytes(B, H, D, N, M)
    ws = workspace if workspace is not None else torch.empty(nws, dtype=torch.uint8, device=dev)
    _call("tfm_icl_attention_fp8", _DTYPES[q_train.dtype], _DTYPES[out_dtype], _opts(q_scale_mode, test_kv_heads),
          B, H, D, N, M, _alpha(alpha, D),
          _ptr(q_train), _ptr(k), _ptr(v), _ptr(q_test), _ptr(o_tr), _ptr(o_te if M else None), _ptr(ws),
          ws.numel(), _stream())
    return o_tr, o_te


def tfm_icl_attention_fp8_noalloc(q_train, k, v, q_test=None, alpha=None, out_dtype=torch.float32, out=None,
                                  q_scale_mode="shared", test_kv_heads=0):
    """tfm_icl_attention_fp8 on the library's fixed scratch (no workspace); the outputs are
    allocated here unless ``out`` gives them."""
    B, H, D, N, M, q_test = _qkv_dims(q_train, k, v, q_test)
    if q_train.dtype not in _DTYPES or out_dtype not in _DTYPES:
        raise ValueError("inputs and outputs must be float32 or bfloat16")
    dev = _check_inputs({"q_train": q_train, "k": k, "v": v, "q_test": q_test}, q_train.dtype)
    o_tr, o_te = _outputs(B, H, D, N, M, out_dtype, dev, out)
    _call("tfm_icl_attention_fp8_noalloc", _DTYPES[q_train.dtype], _DTYPES[out_dtype],
          _opts(q_scale_mode, test_kv_heads), B, H, D, N, M, _alpha(alpha, D),
          _ptr(q_train), _ptr(k), _ptr(v), _ptr(q_test), _ptr(o_tr), _ptr(o_te if M else None), _stream())
    return o_tr, o_te


def tfm_icl_attention_fp8_quantize(q_train, k, v, q_test=None, workspace=None, q_scale_mode="shared"):
    """First stage of tfm_icl_attention_fp8: quantize into a workspace (returned)."""
    B, H, D, N, M, q_test = _qkv_dims(q_train, k, v, q_test)
    if q_train.dtype not in _DTYPES:
        raise ValueError("inputs must be float32 or bfloat16")
    dev = _check_inputs({"q_train": q_train, "k": k, "v": v, "q_test": q_test}, q_train.dtype)
    nws = tfm_icl_attention_fp8_workspace_bytes(B, H, D, N, M)
    ws = workspace if workspace is not None else torch.empty(nws, dtype=torch.uint8, device=dev)
    _call("tfm_icl_attention_fp8_quantize", _DTYPES[q_train.dtype], _opts(q_scale_mode), B, H, D, N, M,
          _ptr(q_train), _ptr(k), _ptr(v), _ptr(q_test), _ptr(ws), ws.numel(), _stream())
    return ws


def tfm_icl_attention_fp8_attend(workspace, B, H, D, N, M, alpha=None, out_dtype=torch.float32, out=None,
                                 test_kv_heads=0):
    """Second stage of tfm_icl_attention_fp8: both ICL calls from a quantized workspace."""
    if out_dtype not in _DTYPES:
        raise ValueError("outputs must be float32 or bfloat16")
    dev = _check_inputs({"workspace": workspace}, torch.uint8)
    o_tr, o_te = _outputs(B, H, D, N, M, out_dtype, dev, out)
    _call("tfm_icl_attention_fp8_attend", _DTYPES[out_dtype], _opts("shared", test_kv_heads), B, H, D, N, M,
          _alpha(alpha, D), _ptr(o_tr),
          _ptr(o_te if M else None), _ptr(workspace), workspace.numel(), _stream())
    return o_tr, o_te


def tfm_icl_attention_fp8_prequantized(q8_train, k8, v8, q8_test, s_q, s_k, s_v, alpha=None,
                                       out_dtype=torch.float32, out=None, workspace=None, s_q_test=None,
                                       test_kv_heads=0):
    """Both ICL calls on codes/scales from tfm_quantize_qkv_per_head; returns (o_train, o_test).

    s_q_test (None = s_q) is the scale of the test-query codes."""
    B, H, N, D = q8_train.shape
    M = 0 if q8_test is None else q8_test.shape[2]
    if M == 0:
        q8_test = None
    dev = _check_inputs({"q8_train": q8_train, "k8": k8, "v8": v8, "q8_test": q8_test}, torch.uint8)
    _check_inputs({"s_q": s_q, "s_k": s_k, "s_v": s_v, "s_q_test": s_q_test}, torch.float32)
    for name, t in (("k8", k8), ("v8", v8)):
        if tuple(t.shape) != (B, H, N, D):
            raise ValueError("%s must be (B, H, N, D)" % name)
    o_tr, o_te = _outputs(B, H, D, N, M, out_dtype, dev, out)
    nws = tfm_icl_attention_fp8_prequantized_workspace_bytes(B, H, D, N)
    ws = workspace if workspace is not None else torch.empty(nws, dtype=torch.uint8, device=dev)
    _call("tfm_icl_attention_fp8_prequantized", _DTYPES[out_dtype], _opts("shared", test_kv_heads), B, H, D, N, M,
          _alpha(alpha, D), _ptr(q8_train), _ptr(k8), _ptr(v8), _ptr(q8_test), _ptr(s_q), _ptr(s_k), _ptr(s_v),
          _ptr(s_q_test), _ptr(o_tr),
          _ptr(o_te if M else None), _ptr(ws), ws.numel(), _stream())
    return o_tr, o_te


def tfm_icl_attention_bf16(q_train, k, v, q_test=None, alpha=None, out_dtype=torch.float32, out=None,
                           test_kv_heads=0):
    """The 16-bit baseline of both ICL calls (bf16, or fp32 rounded to bf16 on load); returns (o_train, o_test)."""
    B, H, D, N, M, q_test = _qkv_dims(q_train, k, v, q_test)
    if q_train.dtype not in _DTYPES or out_dtype not in _DTYPES:
        raise ValueError("inputs and outputs must be float32 or bfloat16")
    dev = _check_inputs({"q_train": q_train, "k": k, "v": v, "q_test": q_test}, q_train.dtype)
    o_tr, o_te = _outputs(B, H, D, N, M, out_dtype, dev, out)
    _call("tfm_icl_attention_bf16", _DTYPES[q_train.dtype], _DTYPES[out_dtype], _opts("shared", test_kv_heads),
          B, H, D, N, M, _alpha(alpha, D),
          _ptr(q_train), _ptr(k), _ptr(v), _ptr(q_test), _ptr(o_tr), _ptr(o_te if M else None), _stream())
    return o_tr, o_te


def tfm_icl_attention_fp8_fit(q_train, k, v, alpha=None, out_dtype=torch.float32, m_max=0, out=None,
                              workspace=None, q_scale_mode="shared"):
    """Quantize the train rows and run the train-train call; returns (o_train, workspace).

    The workspace holds the fit state for tfm_icl_attention_fp8_predict, sized for test batches of up
    to m_max rows (or pass a larger workspace)."""
    B, N, H, D = _shape_bnhd(q_train, "q_train")
    if tuple(k.shape) != (B, N, H, D) or tuple(v.shape) != (B, N, H, D):
        raise ValueError("k and v must have the shape of q_train")
    if q_train.dtype not in _DTYPES or out_dtype not in _DTYPES:
        raise ValueError("inputs and outputs must be float32 or bfloat16")
    dev = _check_inputs({"q_train": q_train, "k": k, "v": v}, q_train.dtype)
    o_tr = out if out is not None else torch.empty((B, N, H, D), dtype=out_dtype, device=dev)
    if tuple(o_tr.shape) != (B, N, H, D) or o_tr.dtype != out_dtype or not o_tr.is_contiguous():
        raise ValueError("out must be a contiguous (B, N, H, D) tensor of the output dtype")
    nws = tfm_icl_attention_fp8_workspace_bytes(B, H, D, N, int(m_max))
    ws = workspace if workspace is not None else torch.empty(nws, dtype=torch.uint8, device=dev)
    _call("tfm_icl_attention_fp8_fit", _DTYPES[q_train.dtype], _DTYPES[out_dtype], _opts(q_scale_mode), B, H, D, N,
          _alpha(alpha, D), _ptr(q_train), _ptr(k), _ptr(v), _ptr(o_tr), _ptr(ws), ws.numel(), _stream())
    return o_tr, ws


def tfm_icl_attention_fp8_predict(workspace, q_test, N, alpha=None, out_dtype=torch.float32, out=None,
                                  q_scale_mode="shared", test_kv_heads=0):
    """The test-train call for q_test (B, M, H, D) against the fit state in workspace (N train rows)."""
    B, M, H, D = _shape_bnhd(q_test, "q_test")
    if q_test.dtype not in _DTYPES or out_dtype not in _DTYPES:
        raise ValueError("inputs and outputs must be float32 or bfloat16")
    dev = _check_inputs({"q_test": q_test if M else None, "workspace": workspace})
    o_te = out if out is not None else torch.empty((B, M, H, D), dtype=out_dtype, device=dev)
    if tuple(o_te.shape) != (B, M, H, D) or o_te.dtype != out_dtype or not o_te.is_contiguous():
        raise ValueError("out must be a contiguous (B, M, H, D) tensor of the output dtype")
    _call("tfm_icl_attention_fp8_predict", _DTYPES[q_test.dtype], _DTYPES[out_dtype],
          _opts(q_scale_mode, test_kv_heads), B, H, D, int(N), M, _alpha(alpha, D), _ptr(q_test if M else None),
          _ptr(o_te if M else None), _ptr(workspace), workspace.numel(), _stream())
    return o_te


FP8_MIN_TRAIN_ROWS_DEFAULT = 8192


def tfm_icl_attention(q_train, k, v, q_test=None, alpha=None, out_dtype=torch.float32, fp8_min_train_rows=-1,
                      out=None, workspace=None, q_scale_mode="shared", test_kv_heads=0):
    """Gated ICL attention: FP8 when N > fp8_min_train_rows (default 8192), else the 16-bit path.

    Returns (o_train, o_test, used_fp8)."""
    B, H, D, N, M, q_test = _qkv_dims(q_train, k, v, q_test)
    if q_train.dtype not in _DTYPES or out_dtype not in _DTYPES:
        raise ValueError("inputs and outputs must be float32 or bfloat16")
    dev = _check_inputs({"q_train": q_train, "k": k, "v": v, "q_test": q_test}, q_train.dtype)
    o_tr, o_te = _outputs(B, H, D, N, M, out_dtype, dev, out)
    nws = lib().tfm_icl_attention_workspace_bytes(B, H, D, N, M, int(fp8_min_train_rows))
    ws = workspace if workspace is not None else (torch.empty(nws, dtype=torch.uint8, device=dev) if nws else None)
    used = ctypes.c_int(-1)
    _call("tfm_icl_attention", _DTYPES[q_train.dtype], _DTYPES[out_dtype], _opts(q_scale_mode, test_kv_heads),
          B, H, D, N, M, _alpha(alpha, D),
          _ptr(q_train), _ptr(k), _ptr(v), _ptr(q_test), _ptr(o_tr), _ptr(o_te if M else None),
          int(fp8_min_train_rows), ctypes.byref(used), _ptr(ws), 0 if ws is None else ws.numel(), _stream())
    return o_tr, o_te, bool(used.value)


def tfm_noise_per_head_workspace_bytes(B, H, S, D):
    return lib().tfm_noise_per_head_workspace_bytes(B, H, S, D)


def tfm_noise_per_head(x, z, eps, out=None, workspace=None):
    """Eq. (3): x + eps * rho * z per (table, head), rho the head's RMS; returns (out, rho (B,H) fp32).

    x and z are (B, S, H, D) float32 or bfloat16 (z may differ from x); out has the type of x
    and may be x itself (in place)."""
    B, S, H, D = _shape_bnhd(x, "x")
    if tuple(z.shape) != (B, S, H, D):
        raise ValueError("z must have the shape of x")
    if x.dtype not in _DTYPES or z.dtype not in _DTYPES:
        raise ValueError("x and z must be float32 or bfloat16")
    dev = _check_inputs({"x": x, "z": z})
    if out is None:
        out = torch.empty_like(x)
    elif tuple(out.shape) != (B, S, H, D) or out.dtype != x.dtype or not out.is_contiguous():
        raise ValueError("out must be a contiguous tensor of the shape and type of x")
    rho = torch.empty((B, H), dtype=torch.float32, device=dev)
    nws = tfm_noise_per_head_workspace_bytes(B, H, S, D)
    ws = workspace if workspace is not None else torch.empty(max(nws, 1), dtype=torch.uint8, device=dev)
    _call("tfm_noise_per_head", _DTYPES[x.dtype], _DTYPES[z.dtype], B, H, S, D, _ptr(x), _ptr(z), float(eps),
          _ptr(out), _ptr(rho), _ptr(ws), ws.numel(), _stream())
    return out, rho
