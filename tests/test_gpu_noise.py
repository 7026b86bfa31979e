"""GPU parity of tfm_noise_per_head with the Eq. (3) oracle.

rho: within one fp32 rounding of the fp64 RMS.  out: within the rounding of
the stated fp32 arithmetic, fmaf(fl32(eps * rho), z, x) (and one bf16
rounding for bf16 outputs), elementwise on every element or, at full size, on
sampled rows (each output element depends only on its own x, z and its
head's rho, and rho is checked over the whole tensor)."""
import numpy as np
import pytest
import torch

from oracle import noise as NZ
from paper_2609_13031_amd import tfm
from parity import sample_rows

pytestmark = pytest.mark.gpu
U = 2.0 ** -24          # fp32 unit roundoff
TORCH = {"f32": torch.float32, "bf16": torch.bfloat16}


def draw(B, S, H, D, seed, spread=True):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((B, S, H, D)).astype(np.float32)
    if spread:
        x *= (10.0 ** rng.uniform(-3, 3, size=(B, 1, H, 1))).astype(np.float32)
    return x, rng.standard_normal((B, S, H, D)).astype(np.float32)


def on_gpu(a, dt):
    return torch.from_numpy(np.ascontiguousarray(a)).to(TORCH[dt]).cuda()


def as_f64(t):
    return t.float().cpu().numpy().astype(np.float64)


def check(out, rho, x64, z64, eps, out_dt, rows=None):
    """rho and out against the oracle; rows: the sampled rows of out (all by default)."""
    ref_rho = NZ.rms_per_head(x64)
    # one fp32 rounding of an fp64 sum whose own error is far below 1e-9 relative
    assert np.all(np.abs(rho - ref_rho) <= (U + 1e-9) * ref_rho), np.max(np.abs(rho - ref_rho) / ref_rho)
    e = np.float64(np.float32(eps))
    sel = (slice(None), slice(None) if rows is None else rows)
    ref = x64[sel] + e * ref_rho[:, None, :, None] * z64[sel]
    # fl32(eps * rho32) is within 2U of eps * rho; the fma and the final fp32 rounding add U of |y|
    delta = 2.03 * U * e * ref_rho[:, None, :, None] * np.abs(z64[sel]) + 1.0001 * U * np.abs(ref) + 1e-44
    if out_dt == "bf16":
        delta = delta + 2.0 ** -8 * (np.abs(ref) + delta)      # bf16 unit roundoff (8 significant bits)
    err = np.abs(out - ref)
    assert np.all(err <= delta), np.max(err / delta)


@pytest.mark.parametrize("B,S,H,D", [(1, 1, 1, 8), (2, 300, 6, 64), (1, 1000, 3, 128), (3, 77, 5, 24),
                                     (1, 200, 8, 512), (2, 33, 1, 16384), (1, 40000, 2, 64)])
@pytest.mark.parametrize("xd,zd", [("f32", "f32"), ("bf16", "bf16"), ("bf16", "f32"), ("f32", "bf16")])
def test_noise_matches_oracle(B, S, H, D, xd, zd):
    print("noise", B, S, H, D, xd, zd, flush=True)
    x, z = draw(B, S, H, D, seed=B * 7 + S + H * D)
    gx, gz = on_gpu(x, xd), on_gpu(z, zd)
    eps = 0.0265 * 3
    out, rho = tfm.tfm_noise_per_head(gx, gz, eps)
    torch.cuda.synchronize()
    check(as_f64(out), rho.cpu().numpy().astype(np.float64), as_f64(gx), as_f64(gz), eps, xd)


def test_noise_in_place_deterministic_and_degenerate_heads():
    B, S, H, D = 2, 5000, 4, 64
    x, z = draw(B, S, H, D, seed=3)
    x[1, :, 2] = 0.0                                       # a zero head: rho = 0, output = x
    gx, gz = on_gpu(x, "bf16"), on_gpu(z, "bf16")
    a, ra = tfm.tfm_noise_per_head(gx, gz, 0.1)
    b, rb = tfm.tfm_noise_per_head(gx, gz, 0.1)
    assert torch.equal(a, b) and torch.equal(ra, rb)      # fixed-order reduction: bitwise reproducible
    assert ra[1, 2].item() == 0.0 and torch.equal(a[1, :, 2], gx[1, :, 2])
    c = gx.clone()
    c2, rc = tfm.tfm_noise_per_head(c, gz, 0.1, out=c)    # in place
    assert c2.data_ptr() == c.data_ptr() and torch.equal(c, a) and torch.equal(rc, ra)
    e0, _ = tfm.tfm_noise_per_head(gx, gz, 0.0)            # eps = 0: identity, bit for bit
    assert torch.equal(e0, gx)
    empty = torch.empty((2, 0, 4, 64), dtype=torch.bfloat16, device="cuda")
    o, r = tfm.tfm_noise_per_head(empty, empty, 0.5)
    assert o.shape == (2, 0, 4, 64) and torch.equal(r, torch.zeros((2, 4), device="cuda"))


def test_noise_full_size_keys_sampled_rows():
    # the K (or V) tensor of the 65536-train-row workload: B=2, S=65536, H=6, D=64, bf16
    B, S, H, D = 2, 65536, 6, 64
    x, z = draw(B, S, H, D, seed=11)
    gx, gz = on_gpu(x, "bf16"), on_gpu(z, "bf16")
    out, rho = tfm.tfm_noise_per_head(gx, gz, 0.0265)
    torch.cuda.synchronize()
    rows = sample_rows(S, 512, 12)
    x64, z64 = as_f64(gx), as_f64(gz)
    check(as_f64(out[:, torch.from_numpy(rows).cuda()]), rho.cpu().numpy().astype(np.float64), x64, z64, 0.0265,
          "bf16", rows=rows)
    # relative perturbation per head is about eps (Z standard normal), whatever the head's magnitude
    d = (out.float() - gx.float()).double().pow(2).sum(dim=(1, 3)).sqrt()
    n = gx.double().pow(2).sum(dim=(1, 3)).sqrt()
    rel = (d / n).cpu().numpy()
    assert np.all(np.abs(rel / 0.0265 - 1) < 0.1), rel


def test_noise_beyond_4_gib():
    # 8.6 G elements per tensor (B=2, S=2^21, H=16, D=128, bf16, drawn on the GPU): element and
    # byte offsets pass 2^32.  rho of two heads (the first and the last) against the oracle over
    # the whole head, and their outputs on sampled rows.
    B, S, H, D = 2, 1 << 21, 16, 128
    gen = torch.Generator(device="cuda").manual_seed(66)
    gx = torch.randn((B, S, H, D), generator=gen, device="cuda", dtype=torch.bfloat16)
    gx *= (10.0 ** (torch.rand((B, 1, H, 1), generator=gen, device="cuda") * 4 - 2)).to(torch.bfloat16)
    gz = torch.randn((B, S, H, D), generator=gen, device="cuda", dtype=torch.bfloat16)
    assert gx.numel() > 2 ** 32
    eps = 0.05
    out, rho = tfm.tfm_noise_per_head(gx, gz, eps)
    torch.cuda.synchronize()
    rows = sample_rows(S, 64, 67)
    ri = torch.from_numpy(rows).cuda()
    e = np.float64(np.float32(eps))
    for b, h in ((0, 0), (1, 15)):
        ref_rho = NZ.rms_per_head(gx[b, :, h].double().cpu().numpy()[None, :, None, :])[0, 0]
        assert abs(rho[b, h].item() - ref_rho) <= (U + 1e-9) * ref_rho, (b, h)
        x64, z64 = gx[b, ri, h].double().cpu().numpy(), gz[b, ri, h].double().cpu().numpy()
        ref = x64 + e * ref_rho * z64
        delta = 2.03 * U * e * ref_rho * np.abs(z64) + 1.0001 * U * np.abs(ref) + 1e-44
        delta = delta + 2.0 ** -8 * (np.abs(ref) + delta)
        assert np.all(np.abs(out[b, ri, h].double().cpu().numpy() - ref) <= delta), (b, h)
    del gx, gz, out
    torch.cuda.empty_cache()
