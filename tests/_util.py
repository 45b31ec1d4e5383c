"""Shared helpers of the test suite (no method arithmetic)."""

import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

U32 = 2.0 ** -24  # float32 unit roundoff


def gamma(n, u=U32):
    """Higham's gamma_n = n u / (1 - n u) (rounding-error bound of a length-n
    dot product accumulated in a format with unit roundoff u)."""
    return n * u / (1 - n * u)


def rel_inf(y, ref):
    """||y - ref||_inf / ||ref||_inf over the whole tensor."""
    y = np.asarray(y, np.float64)
    ref = np.asarray(ref, np.float64)
    den = np.abs(ref).max() if ref.size else 0.0
    return float(np.abs(y - ref).max() / den) if den > 0 else float(np.abs(y - ref).max() if y.size else 0.0)


def row_rel(y, ref, floor_frac=1e-3):
    """Per-row max error over max(max|ref_row|, floor_frac * rms(ref))."""
    y = np.asarray(y, np.float64)
    ref = np.asarray(ref, np.float64)
    if not ref.size:
        return 0.0
    floor = floor_frac * np.sqrt(np.mean(ref ** 2))
    den = np.maximum(np.abs(ref).max(axis=1), floor)
    return float((np.abs(y - ref).max(axis=1) / den).max())


def ensure_built():
    """Build the library only when nothing is built yet."""
    from paper_2609_38823_amd import abi, build
    if not os.path.exists(abi.LIB_PATH):
        build.build()
    return abi.load()
