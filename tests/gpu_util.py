"""Helpers shared by the GPU tests (comparison metrics and problem setup)."""
import numpy as np


def colscaled_max_rel_err(X, Xref):
    """max over features t of max_i |X - Xref|_{it} / max_i |Xref|_{it}.

    The tolerance of 1e-3 on W and H after one outer iteration is read this way:
    a per-feature scale, so entries near zero do not blow up the ratio."""
    X = np.asarray(X, dtype=np.float64)
    Xref = np.asarray(Xref, dtype=np.float64)
    scale = np.abs(Xref).max(axis=0)
    scale[scale == 0] = 1.0
    return float((np.abs(X - Xref).max(axis=0) / scale).max())


def gpu_available():
    try:
        import torch
        return torch.cuda.is_available()
    except Exception:
        return False
