"""Shared test utilities: the parity bar and device upload helpers."""
import re
import os

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "nsd.h")

# Parity bar for floating-point outputs: |got - ref| <= TOL * mag, where mag
# is the oracle's evaluation of the same expression on absolute values (it
# bounds the rounding error of any summation order).  Where mag == 0 the
# output must be exactly 0.  TOL is the 1e-4 relative bound.
TOL = 1e-4


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(nsd_\w+)\s*\(", text, flags=re.M)))


def mag_err(got, ref, mag):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    mag = np.asarray(mag, dtype=np.float64)
    diff = np.abs(got - ref)
    err = np.where(mag > 0, diff / np.where(mag > 0, mag, 1.0), np.where(diff > 0, np.inf, 0.0))
    return err


def assert_mag_close(got, ref, mag, tol=TOL, what=""):
    err = mag_err(got, ref, mag)
    worst = float(err.max()) if err.size else 0.0
    if not worst <= tol:
        i = int(np.argmax(err.ravel()))
        raise AssertionError(
            f"{what}: max |got-ref|/mag = {worst:.3e} > {tol:.0e} at flat index {i}: "
            f"got {np.ravel(got)[i]!r} ref {np.ravel(ref)[i]!r} mag {np.ravel(mag)[i]!r}")
    return worst
