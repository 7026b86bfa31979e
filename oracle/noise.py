"""Per-head RMS-scaled Gaussian perturbation, Eq. (3) (test oracle).

The appendix's noise experiment replaces quantization with an explicit
perturbation of a tensor X in R^{S x H x d}: for every head h independently,

    X~^(h) = X^(h) + eps * rho^(h) * Z^(h),
    rho^(h) = sqrt( (1 / (S d)) * sum_{i,j} (X^(h)_ij)^2 ),

with Z^(h) a field of iid standard normal values.  The head's own RMS sets
the size of its perturbation, as the head's absmax sets its scale in Eq. (2),
so heads of very different magnitude are perturbed by the same relative
amount.

Readings (each also listed in the design notes):
* the random field Z is an input (the caller draws it from its seeded
  generator), so both the oracle and the GPU path apply the same field;
* the RMS runs over the S rows and d channels of one (table b, head h), like
  the quantization scales;
* S = 0 gives rho = 0 and an empty result.

Layouts: X and Z are (B, S, H, D); rho is (B, H).  Arithmetic is fp64.
"""
import numpy as np


def rms_per_head(x):
    """rho per (b, h) of a (B,S,H,D) tensor, fp64; 0 for S = 0."""
    x = np.asarray(x, dtype=np.float64)
    B, S, H, D = x.shape
    if S == 0:
        return np.zeros((B, H))
    return np.sqrt(np.einsum("bshd,bshd->bh", x, x) / (S * D))


def perturb_per_head(x, z, eps):
    """Eq. (3): x + eps * rho * z per head, fp64, returned with rho as (x_tilde, rho)."""
    x = np.asarray(x, dtype=np.float64)
    z = np.asarray(z, dtype=np.float64)
    if x.shape != z.shape:
        raise ValueError("x and z must have the same (B, S, H, D) shape")
    rho = rms_per_head(x)
    return x + float(eps) * rho[:, None, :, None] * z, rho
