"""Plausible mistakes, planted one at a time in the oracle on the CPU.

Each mutation rewrites one expression in the source of one oracle function
(the text must occur exactly once, so a mutation cannot silently stop
applying as the oracle evolves) and re-binds the function wherever the
oracle's modules refer to it.  The oracle's pin tests (tests/test_oracle_*.py:
worked values, closed forms, library routines, brute force, bounds) must fail
under every mutation; ``tests/test_oracle_mutations.py`` checks that, running
them in a subprocess with ORACLE_MUTATION set, which ``tests/conftest.py``
applies before any test module imports the oracle.
"""
import importlib
import inspect
import sys
import textwrap

import numpy as np

# name: (module, function, old text, new text, the mistake)
MUTATIONS = {
    # ---- e4m3 codec (format definition) ----
    "decode_bias": ("oracle.e4m3", "_decode_codes", "np.exp2(e - 7.0)", "np.exp2(e - 8.0)",
                    "exponent bias 8 instead of 7"),
    "decode_subnormal_step": ("oracle.e4m3", "_decode_codes", "m * 2.0 ** -9", "m * 2.0 ** -10",
                              "subnormal step 2^-10"),
    "decode_nan_code": ("oracle.e4m3", "_decode_codes", "(c & 0x7F) == 0x7F", "(c & 0x7F) == 0x7E",
                        "448 taken for the NaN code"),
    "encode_ties_away": ("oracle.e4m3", "_encode_block", "q = np.rint(np.ldexp(a[nrm], 3 - e))",
                         "q = np.floor(np.ldexp(a[nrm], 3 - e) + 0.5)", "ties away from zero (normal range)"),
    "encode_truncate": ("oracle.e4m3", "_encode_block", "q = np.rint(np.ldexp(a[nrm], 3 - e))",
                        "q = np.floor(np.ldexp(a[nrm], 3 - e))", "truncation instead of rounding"),
    "encode_subnormal_ties_away": ("oracle.e4m3", "_encode_block", "np.rint(a[sub] * 2.0 ** 9)",
                                   "np.floor(a[sub] * 2.0 ** 9 + 0.5)", "ties away from zero (subnormals)"),
    "encode_subnormal_boundary": ("oracle.e4m3", "_encode_block", "sub = a < 2.0 ** -6", "sub = a < 2.0 ** -7",
                                  "subnormal range ends one binade early"),
    "encode_negative_zero": ("oracle.e4m3", "_encode_block", "np.signbit(y)", "y < 0",
                             "negative values rounding to zero lose their sign"),
    "encode_no_carry": ("oracle.e4m3", "_encode_block", "carry = q == 16", "carry = q > 16",
                        "mantissa carry not moved to the next binade"),
    # ---- quantizer, Eq. (2) ----
    "scale_constant": ("oracle.quantize", "scale_from_amax", "F32_448", "np.float32(256.0)",
                       "scale amax / 256"),
    "scale_zero_rule": ("oracle.quantize", "scale_from_amax", "np.where(s == 0, np.float32(1.0), s)", "s",
                        "no scale of 1 for an all-zero head"),
    "reciprocal_multiply": ("oracle.quantize", "quantize_with_scale",
                            "np.divide(x, s[:, None, :, None], dtype=np.float32)",
                            "x * (np.float32(1.0) / s)[:, None, :, None]",
                            "multiply by the fp32 reciprocal instead of dividing"),
    "no_clamp": ("oracle.quantize", "quantize_with_scale",
                 "np.clip(y, np.float32(-MAX_FINITE), np.float32(MAX_FINITE), out=y)", "y",
                 "no clamp to [-448, 448] before rounding"),
    "codes_reshaped": ("oracle.quantize", "quantize_with_scale", "codes.transpose(0, 2, 1, 3)",
                       "codes.reshape(codes.shape[0], codes.shape[2], codes.shape[1], codes.shape[3])",
                       "(B,S,H,D) codes reshaped instead of transposed to (B,H,S,D)"),
    "amax_over_tables": ("oracle.quantize", "absmax_per_head", "max(axis=(1, 3))", "max(axis=(0, 1, 3))[None]",
                         "absmax over all tables of a head"),
    "test_queries_own_scale": ("oracle.quantize", "quantize_qkv_per_head",
                               'scale_from_amax(a_qt) if q_scale_mode == "per_call" else s_q',
                               'scale_from_amax(a_qt) if q_scale_mode != "joint" else s_q',
                               "test queries on their own scale in the shared mode"),
    "joint_ignores_test": ("oracle.quantize", "quantize_qkv_per_head", "scale_from_amax(np.maximum(a_q, a_qt))",
                           "scale_from_amax(a_q)", "joint scale without the test queries"),
    # ---- attention, Eq. (1), and the one-pass kernel model ----
    "softmax_no_alpha": ("oracle.attention", "softmax_attention", "float(alpha) * (q[r0:r0 + chunk_rows] @ k.T)",
                         "(q[r0:r0 + chunk_rows] @ k.T)", "softmax scale dropped"),
    "softmax_column_sum": ("oracle.attention", "softmax_attention", "p /= p.sum(axis=1, keepdims=True)",
                           "p /= p.sum(axis=0, keepdims=True)", "softmax normalised over the wrong axis"),
    "grouped_head_mod": ("oracle.attention", "grouped_kv_head", "return h // (H // G)", "return h % G",
                         "grouped test heads interleaved instead of contiguous"),
    "dequant_scale_head0": ("oracle.attention", "dequantize", "[:, :, None, None]", "[:, :1, None, None]",
                            "every head dequantized with head 0's scale"),
    "kernel_lift_2_7": ("oracle.attention", "one_pass_fp8_attention", "+ P_LIFT_LOG2)", "+ P_LIFT_LOG2 - 1)",
                        "row maximum lifted to 2^7"),
    "kernel_no_rescale": ("oracle.attention", "one_pass_fp8_attention",
                          "np.exp2(c * (np.where(first, m_new, m) - m_new))", "1.0",
                          "state not rescaled when the max grows"),
    "kernel_first_block_rescale": ("oracle.attention", "one_pass_fp8_attention",
                                   "r = np.where(first, 0.0, np.exp2(c * (np.where(first, m_new, m) - m_new)))",
                                   "r = np.exp2(c * (m - m_new))",
                                   "the empty state rescaled by 2^(c (-inf)), NaN when c is 0"),
    "kernel_max_over_rows": ("oracle.attention", "one_pass_fp8_attention",
                             "m_new = np.maximum(m, s.max(axis=1))", "m_new = np.maximum(m, s.max())",
                             "one running max shared by all rows"),
    "kernel_global_max": ("oracle.attention", "one_pass_fp8_attention",
                          "m_new = np.maximum(m, s.max(axis=1))", "m_new = (q8 @ k8.T).max(axis=1)",
                          "lift relative to the row's final max instead of the running max"),
    "kernel_unrounded_pv": ("oracle.attention", "one_pass_fp8_attention",
                            "acc = acc * r[:, None] + p8 @ v8[j0:j0 + block_kv]",
                            "acc = acc * r[:, None] + p @ v8[j0:j0 + block_kv]", "P V with the unrounded P"),
    "kernel_no_sv": ("oracle.attention", "one_pass_fp8_attention", "o = acc * float(s_v) / l[:, None]",
                     "o = acc / l[:, None]", "V scale not applied"),
    "kernel_rowsum_unrounded": ("oracle.attention", "one_pass_fp8_attention",
                                'l = l * r + (p8 if row_sum == "p8" else p).sum(axis=1)', "l = l * r + p.sum(axis=1)",
                                "row sum of the unrounded P under the p8 reading"),
    "kernel_natural_exp": ("oracle.attention", "one_pass_fp8_attention",
                           "np.exp2(c * (s - m_new[:, None]) + P_LIFT_LOG2)",
                           "np.exp(c * (s - m_new[:, None])) * 2.0 ** P_LIFT_LOG2",
                           "natural exp of a base-2 logit"),
    "kernel_test_scale": ("oracle.attention", "icl_attention_fp8_kernel_model", "re, s_q_test[b, h], hk)",
                          're, qz["s_q"][b, h], hk)', "test call on the train-query scale in every mode"),
    # ---- noise, Eq. (3) ----
    "rms_no_d": ("oracle.noise", "rms_per_head", "/ (S * D)", "/ S", "mean over rows only"),
    "rms_no_sqrt": ("oracle.noise", "rms_per_head", "np.sqrt(np.einsum(", "(np.einsum(", "mean square, no root"),
    "noise_global_rho": ("oracle.noise", "perturb_per_head", "rho[:, None, :, None]", "rho.max()",
                         "one perturbation scale for every head"),
}


def apply(name):
    """Plant mutation `name` in the imported oracle modules."""
    mod_name, fn_name, old, new, _ = MUTATIONS[name]
    mod = importlib.import_module(mod_name)
    fn = getattr(mod, fn_name)
    src = textwrap.dedent(inspect.getsource(fn))
    if src.count(old) != 1:
        raise RuntimeError("mutation %s: %r occurs %d times in %s.%s" % (name, old, src.count(old), mod_name, fn_name))
    exec(compile(src.replace(old, new), "<mutation %s>" % name, "exec"), mod.__dict__)
    mutated = mod.__dict__[fn_name]
    for m in list(sys.modules.values()):
        if getattr(m, "__name__", "").startswith("oracle"):
            for k, v in list(vars(m).items()):
                if v is fn:
                    setattr(m, k, mutated)
    if fn_name == "_decode_codes":      # the decode table is built from it at import
        mod._VALUES = mutated(np.arange(256, dtype=np.int64))
