"""Sampler schedule and the clean-cache renoise/emit updates (Section 3.4, Equations 1-3, and
the appendix's shift-five schedule).

Schedule: n equally spaced raw coordinates u_i = 1000 (n - i) / n are mapped by the shift
map sigma_i = s u_i / (1000 + (s - 1) u_i) (s = 5 in the paper) to noise levels, and the DiT
label is t_i = 1000 sigma_i; the map keeps the endpoints 1000 and 0.  Evaluated in float64
(the paper keeps the schedule tables in float64).

Updates around one DiT evaluation v = f(x_tilde, t) at noise level sigma:
    renoise  x_tilde = (1 - sigma) x + sigma eps      (Equation 1; eps ~ N(0, I) is an input)
    emit     x_next  = x_tilde - sigma v              (Equation 3)
The clean-cache pass uses sigma = 0.02 (UnStep) where the original sampler uses 0, which
makes both updates identities.

Rounding contract (the paper fixes float64 for the schedule, not the operation order): the
inputs are bf16 latents; each product and the sum/difference are IEEE float64 operations
(no fused multiply-add), the result is rounded to binary32 and then to bf16, both to
nearest-even.  1 - sigma is formed in float64.

Test infrastructure: nothing in the library imports this module.
"""
from __future__ import annotations

import numpy as np

from .numerics import bf16_to_f64, f32_to_bf16_bits, round_f32

SIGMA_CLEAN_UNSTEP = 0.02


def shift_schedule(n_steps: int = 4, shift: float = 5.0):
    """(u, sigma, t) float64 arrays of the n-step shifted schedule."""
    if n_steps < 1 or not shift > 0:
        raise ValueError("n_steps >= 1 and shift > 0 required")
    u = np.array([1000.0 * (n_steps - i) / n_steps for i in range(n_steps)])
    sigma = shift * u / (1000.0 + (shift - 1.0) * u)
    return u, sigma, 1000.0 * sigma


def renoise_bf16(x_bits: np.ndarray, eps_bits: np.ndarray, sigma: float) -> np.ndarray:
    """Equation 1 on bf16 latents; bf16 bits out (contract in the module docstring)."""
    x = bf16_to_f64(x_bits)
    e = bf16_to_f64(eps_bits)
    return f32_to_bf16_bits(round_f32((1.0 - sigma) * x + sigma * e))


def emit_bf16(xt_bits: np.ndarray, v_bits: np.ndarray, sigma: float) -> np.ndarray:
    """Equation 3 on bf16 latents; bf16 bits out."""
    return f32_to_bf16_bits(round_f32(bf16_to_f64(xt_bits) - sigma * bf16_to_f64(v_bits)))
