"""Memory model (Section 3.3) and decode-time cost model (Appendix B).

All counts are per layer and per sequence (the paper omits the batch axis),
in stored scalar elements (memory) or multiply-accumulate units (cost).
"""

import math


def k_from_rho(L, W, rho):
    """Global budget k = max(floor(rho*L) - W, 0) (3.2.3)."""
    return max(int(math.floor(rho * L)) - W, 0)


def m_from_rho(L, W, rho):
    """m_t = W + max(floor(rho*L) - W, 0) = max(W, floor(rho*L)) (3.3)."""
    return W + k_from_rho(L, W, rho)


def mem_full(L, s, Dp):
    """M_full(t) = 2 (s + L) Dp."""
    return 2 * (s + L) * Dp


def mem_s4r(L, s, Dp, r, G, W):
    """M_S4R(t) = 2 s Dp + 2 L r + G W r + 2 Dp r."""
    return 2 * s * Dp + 2 * L * r + G * W * r + 2 * Dp * r


def mem_ratio(L, s, Dp, r, G, W):
    """Eq. memory_ratio: (s Dp + L r + G W r / 2 + Dp r) / ((s + L) Dp)."""
    return (s * Dp + L * r + 0.5 * G * W * r + Dp * r) / ((s + L) * Dp)


def mem_work(m, Dp):
    """M_work(t) = 2 m_t Dp (the reconstructed key/value buffer)."""
    return 2 * m * Dp


def rank_for_ratio(eta, L, s, Dp, G, W):
    """Real r solving Eq. memory_ratio = eta (the ratio is affine in r)."""
    return (eta * (s + L) * Dp - s * Dp) / (L + 0.5 * G * W + Dp)


# Appendix B: per-step costs with the common factor L removed.

def full_rec_coeff(r, Dp, G):
    """C_full-rec / L = r Dp + G Dp (Eq. full_reconstruction_complexity)."""
    return r * Dp + G * Dp


def s4r_coeff(r, Dp, G, W, rho):
    """C_S4R / L = G W r + rho r Dp + rho G Dp (Eq. s4r_decoding_complexity_compact)."""
    return G * W * r + rho * r * Dp + rho * G * Dp


def s4r_beneficial(r, Dp, G, W, rho):
    """Eq. s4r_beneficial_condition: G W r < (1 - rho) Dp (r + G)."""
    return G * W * r < (1.0 - rho) * Dp * (r + G)


def step_terms(L, s, Dp, r, G, W, m):
    """Un-normalised per-step cost terms of Appendix B.2 (MAC units)."""
    return {
        "update": (G + 2) * Dp * r,
        "scoring": G * W * L * r,
        "reconstruction": 2 * m * r * Dp,
        "attention": G * (s + m) * Dp,
    }
