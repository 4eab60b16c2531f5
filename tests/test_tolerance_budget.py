"""The parity tolerances are attainable: a NumPy emulation of the GPU's
arithmetic (bf16 operands, fp32 scores, probabilities rounded to bf16 with
the reference maximum lagging by up to the lazy-rescale slack of 2^8, fp32
accumulation, bf16 output; fp8 K/V decoded exactly) stays well inside them
against the fp64 definition (CPU only).  This is the analysis behind the
bounds the GPU parity tests use: bf16 max 2e-2 / mean 2e-3, fp8 max 3e-2."""
import numpy as np
import pytest

from oracle import formats, paged


def bf16(x):
    return formats.bf16_bits_to_f64(formats.bf16_bits_from_f32(np.asarray(x, np.float32)))


def emulate(q, k, v, scale, lag):
    """One query row over keys k, v (already in the precision they are stored
    in); lag: how far below the true maximum the reference maximum sits."""
    s = (k.astype(np.float32) @ q.astype(np.float32)).astype(np.float64)  # fp32 products and sums
    t = s * (scale * np.log2(np.e))
    m = t.max() - lag
    p = bf16(np.exp2(t - m))          # what the PV MFMA consumes
    l = np.float32(p.astype(np.float32).sum())
    o = (p.astype(np.float32) @ v.astype(np.float32)) / l
    return bf16(o)


@pytest.mark.parametrize("kv", ["bf16", "fp8"])
@pytest.mark.parametrize("L", [64, 4096, 47000])
def test_emulated_pipeline_error_is_well_inside_the_tolerance(kv, L):
    rng = np.random.default_rng(L + (7 if kv == "fp8" else 0))
    D, rows = 128, 24
    scale = 1.0 / np.sqrt(D)
    k = bf16(rng.standard_normal((L, D)))
    v = bf16(rng.standard_normal((L, D)))
    if kv == "fp8":  # per-block scales s = amax / 448, codes decoded exactly
        for x in (k, v):
            for b0 in range(0, L, 64):
                blk = x[b0:b0 + 64]
                s = np.float32(np.abs(blk).max() / 448.0)
                x[b0:b0 + 64] = formats.e4m3_to_f64(formats.fp8_quantize(blk.astype(np.float32), s)) * s
    errs = []
    for r in range(rows):
        q = bf16(rng.standard_normal(D))
        ref = paged.attend(q[None, None, :], np.array([L - 1]), k[:, None, :], v[:, None, :], scale)[0, 0]
        for lag in (0.0, 8.0):  # fresh maximum, and one lagging by the full slack
            errs.append(np.abs(emulate(q, k, v, scale, lag) - ref))
    err = np.stack(errs)
    bound_max, bound_mean = (3e-2, 2e-3) if kv == "fp8" else (2e-2, 2e-3)
    # the emulation uses a fraction of each bound
    assert err.max() <= 0.5 * bound_max
    assert err.mean() <= 0.5 * bound_mean
