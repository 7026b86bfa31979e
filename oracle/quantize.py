"""Per-head dynamic absmax quantization to e4m3fn (test oracle).

Eq. (2) of the paper (Sec. 3): for each head h of a tensor X,
    s_X^(h) = max_{i,j} |X^(h)_ij| / 448,
    X_8     = rn_fp8( clamp(X / s_X, -448, 448) ),
with an FP32 dequantization scale, so that X ~= s_X * X_8.  The scale is
computed from the tensor itself (no calibration).  In the ICL layer keys and
values come from the train rows only, and the test queries are quantized
with the scale of the *train* queries, which makes test predictions
independent of the test batch (Sec. 3, paragraph after Eq. (2); Table 1,
last row).  Two other query-scale choices the paper evaluates are modes of
``quantize_qkv_per_head``: "per_call" gives the test queries their own
per-head scale (Table 1, "both, per-call query scale"), and "joint" takes one
per-head scale over train and test queries together, as a single attention
call over all rows does (the appendix's TabICLv2 experiments).

Readings where the paper is silent (each also listed in the design notes):
* granularity: one scale per (table b, head h), over all rows and channels;
* ``s = fl32(amax / 448)`` and ``y = fl32(x / s)`` are IEEE fp32 divisions
  (round to nearest even) -- the formula read literally;
* the clamp is applied before rounding, so values beyond the train amax
  (possible only for test queries) saturate to +-448;
* ``amax == 0`` (or an amax whose quotient underflows to 0) uses s = 1, which
  maps the whole head to zero codes;
* negative values that round to zero keep their sign (code 0x80).

Layouts: inputs are (B, S, H, D) row-major (rows, heads, head_dim per table,
as the paper writes activations X in R^{S x H x d}); codes are returned as
(B, H, S, D) uint8 and scales as (B, H) float32.
"""
import numpy as np

from .e4m3 import encode_rne, MAX_FINITE

F32_448 = np.float32(448.0)


def absmax_per_head(x):
    """max |x| over rows and channels, per (b, h): (B,S,H,D) -> (B,H) float32."""
    x = np.asarray(x, dtype=np.float32)
    if x.shape[1] == 0:
        return np.zeros((x.shape[0], x.shape[2]), dtype=np.float32)
    return np.abs(x).max(axis=(1, 3)).astype(np.float32)


def scale_from_amax(amax):
    """Dequantization scale s = fl32(amax / 448); s = 1 where that is 0."""
    s = np.divide(np.asarray(amax, dtype=np.float32), F32_448, dtype=np.float32)
    return np.where(s == 0, np.float32(1.0), s).astype(np.float32)


def quantize_with_scale(x, s):
    """Codes rn_fp8(clamp(fl32(x / s), -448, 448)): (B,S,H,D), (B,H) -> (B,H,S,D) uint8."""
    x = np.asarray(x, dtype=np.float32)
    s = np.asarray(s, dtype=np.float32)
    # a value far outside the scale's range (test queries on the train-query scale)
    # overflows fp32 to +-inf here; the clamp then saturates it to +-448
    with np.errstate(over="ignore"):
        y = np.divide(x, s[:, None, :, None], dtype=np.float32)
    np.clip(y, np.float32(-MAX_FINITE), np.float32(MAX_FINITE), out=y)
    codes = encode_rne(y)
    return np.ascontiguousarray(codes.transpose(0, 2, 1, 3))


Q_SCALE_MODES = ("shared", "per_call", "joint")


def quantize_qkv_per_head(q_train, k, v, q_test=None, q_scale_mode="shared"):
    """Eq. (2) applied to the ICL layer's tensors.

    K and V get their own per-head scales.  The queries' scales follow
    ``q_scale_mode``:
      "shared"   -- s_q from Q_train; Q_test is quantized with s_q as well;
      "per_call" -- s_q from Q_train, s_q_test from Q_test alone;
      "joint"    -- one scale s_q = s_q_test from the absmax over Q_train and
                    Q_test together.
    A missing or empty Q_test has absmax 0.  Returns a dict with the codes
    ``q8_train, k8, v8, q8_test`` ((B,H,S,D) uint8) and the scales
    ``s_q, s_k, s_v, s_q_test`` ((B,H) float32).
    """
    if q_scale_mode not in Q_SCALE_MODES:
        raise ValueError("q_scale_mode must be one of %s" % (Q_SCALE_MODES,))
    a_q = absmax_per_head(q_train)
    if q_test is None:
        a_qt = np.zeros_like(a_q)
    else:
        a_qt = absmax_per_head(q_test)
    if q_scale_mode == "joint":
        s_q = scale_from_amax(np.maximum(a_q, a_qt))
    else:
        s_q = scale_from_amax(a_q)
    s_q_test = scale_from_amax(a_qt) if q_scale_mode == "per_call" else s_q
    s_k = scale_from_amax(absmax_per_head(k))
    s_v = scale_from_amax(absmax_per_head(v))
    out = {
        "q8_train": quantize_with_scale(q_train, s_q),
        "k8": quantize_with_scale(k, s_k),
        "v8": quantize_with_scale(v, s_v),
        "s_q": s_q, "s_k": s_k, "s_v": s_v, "s_q_test": s_q_test,
    }
    if q_test is not None:
        out["q8_test"] = quantize_with_scale(q_test, s_q_test)
    return out
