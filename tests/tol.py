"""Parity tolerance shared by the GPU tests.

Bar for bf16 inputs with fp32 accumulation, per output tensor:
    max_i (|got_i - ref_i| - BF16_REL * |ref_i|)  <= 2e-2
    ||got - ref||_F / ||ref||_F                  <= 1e-2
The 2e-2 absolute bar applies to the arithmetic error on top of the output's
own representation error: a bf16 output x carries a rounding error of up to
2^-9 |x| (round to nearest even), which alone exceeds 2e-2 once |x| > 10, and
the probabilities / score gradients are rounded to bf16 once more before
their fp32-accumulated products; BF16_REL = 2^-8 covers both roundings.
Weight gradients reduce over the whole sequence, so their entries grow like
sqrt(S); for them the max-abs criterion is applied to err / max(1, rms(ref)).
"""

import numpy as np

MAX_ABS = 2e-2
REL_FROB = 1e-2
BF16_REL = 2.0 ** -8


def as64(t):
    try:
        import torch
        if isinstance(t, torch.Tensor):
            return t.detach().float().cpu().double().numpy()
    except ImportError:  # pragma: no cover
        pass
    return np.asarray(t, np.float64)


def errors(got, ref, rms_scaled=False):
    got, ref = as64(got), as64(ref)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    err = got - ref
    excess = np.abs(err) - BF16_REL * np.abs(ref)
    max_abs = float(excess.max()) if err.size else 0.0
    if rms_scaled:
        rms = float(np.sqrt(np.mean(ref * ref))) if ref.size else 0.0
        max_abs /= max(1.0, rms)
    nref = float(np.linalg.norm(ref))
    nerr = float(np.linalg.norm(err))
    rel = nerr / nref if nref > 0 else nerr
    return max_abs, rel


def assert_close(name, got, ref, rms_scaled=False):
    max_abs, rel = errors(got, ref, rms_scaled)
    raw = float(np.abs(as64(got) - as64(ref)).max()) if as64(ref).size else 0.0
    print(f"  {name}: max_abs={raw:.3e} excess={max_abs:.3e} rel_frob={rel:.3e}")
    assert np.all(np.isfinite(as64(got))), f"{name}: non-finite values"
    assert max_abs <= MAX_ABS and rel <= REL_FROB, (
        f"{name}: max_abs={max_abs:.3e} (<= {MAX_ABS}) "
        f"rel_frob={rel:.3e} (<= {REL_FROB})")
    return max_abs, rel
