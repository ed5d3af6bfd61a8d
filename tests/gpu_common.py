"""Shared helpers of the GPU parity tests."""
import sys

import numpy as np

UNB = 0x7FFFFFFF


def announce(*what):
    """Name the case on stderr before touching the GPU (survives a lost box)."""
    print("[gpu case]", *what, file=sys.stderr, flush=True)


def assert_iterates_close(x_gpu, x_ref, rel=1e-12):
    """Normwise: ||x_gpu - x_ref||_inf <= rel * ||x_ref||_inf."""
    err = float(np.abs(x_gpu - x_ref).max()) if x_ref.size else 0.0
    scale = float(np.abs(x_ref).max()) if x_ref.size else 0.0
    assert err <= rel * scale, "max|dx| = %.3e, ||x||_inf = %.3e" % (err, scale)
    return err


def assert_rho_close(rho_gpu, rho_ref, floor):
    """|rho_gpu - rho_ref| <= 1e-12 rho_ref + 32 u floor (u = 2^-53)."""
    u = 2.0 ** -53
    tol = 1e-12 * np.abs(rho_ref) + 32 * u * floor
    bad = np.nonzero(np.abs(rho_gpu - rho_ref) > tol)[0]
    assert bad.size == 0, "rho mismatch at t=%s: gpu %s ref %s" % (
        bad[:5], rho_gpu[bad[:5]], rho_ref[bad[:5]])
