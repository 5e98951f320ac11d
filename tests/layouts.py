"""Element offsets of the fragment-ordered page layouts documented in include/forkkv.h (page
size 16, head dim 128), for tests that read pools back on the host.  Test infrastructure."""


def k_off(t, i):
    """Key (token t, dim i) inside a (page, K, head) block."""
    return (i // 32) * 512 + (t + 16 * ((i % 16) // 4)) * 8 + 4 * ((i % 32) // 16) + i % 4


def v_off(t, i):
    """Value (token t, dim i) inside a (page, V, head) block."""
    return (i // 32) * 512 + (i % 16 + 16 * (t // 4)) * 8 + 4 * ((i // 16) % 2) + t % 4


def ck_off(t, rho):
    """C_K (token t, rank rho) inside a residual page."""
    return (rho // 16) * 512 + (16 * ((rho % 16) // 4) + t) * 8 + rho % 4


def cv_off(t, rho):
    """C_V (token t, rank rho) inside a residual page."""
    return (rho // 16) * 512 + (16 * (t // 4) + rho % 16) * 8 + 4 + t % 4
