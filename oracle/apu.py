"""Oracle: efficiency bookkeeping of Sec. 2.2 and Sec. 2.3. Test infrastructure only.

Sec. 2.2 defines the average parameters used per token,
    APU = (n_sparse * C_sparse + C_full) / n_AAL,
and, dividing by C_full with I = C_sparse / C_full, the effective density
    (n_sparse * I + 1) / n_AAL,  or with a period n_period = n_sparse + 1,
    ((n_period - 1) * I + 1) / n_AAL.
Sec. 2.3 uses the speculative-decoding expectation of accepted tokens at
acceptance rate alpha and draft length gamma,
    AAL = (1 - alpha^(gamma + 1)) / (1 - alpha).
"""

from __future__ import annotations


def sd_aal(alpha: float, gamma: int) -> float:
    """Expected advance per verification of speculative decoding (Sec. 2.3)."""
    if alpha == 1.0:
        return float(gamma + 1)
    return (1.0 - alpha ** (gamma + 1)) / (1.0 - alpha)


def apu(n_sparse: float, c_sparse: float, c_full: float, n_aal: float) -> float:
    """Average parameters used per token (Sec. 2.2, first equation)."""
    return (n_sparse * c_sparse + c_full) / n_aal


def effective_density(n_period: float, global_density: float, n_aal: float) -> float:
    """APU / C_full written with the period (Sec. 2.2, last equation)."""
    return ((n_period - 1) * global_density + 1.0) / n_aal
