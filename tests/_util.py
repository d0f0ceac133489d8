"""Helpers shared by the tests (error measures only; no method arithmetic)."""
import numpy as np


def normwise_rel_err(got, ref, axes=None):
    """max over systems of ||got - ref||_inf / ||ref||_inf.

    The leading axis indexes independent systems (the batch) unless ``axes``
    is None and the arrays have no batch, in which case the whole tensor is
    one system."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    if got.size == 0:
        return 0.0
    if axes == "all" or got.ndim == 1:
        den = np.max(np.abs(ref))
        num = np.max(np.abs(got - ref))
        return float(num / den) if den > 0 else float(num)
    g = got.reshape(got.shape[0], -1)
    r = ref.reshape(ref.shape[0], -1)
    num = np.max(np.abs(g - r), axis=1)
    den = np.max(np.abs(r), axis=1)
    den = np.where(den > 0, den, 1.0)
    return float(np.max(num / den))


def per_layer_rel_err(got, ref, floor=1e-6, layer_axis=1):
    """Worst normwise error over single layers: for each layer (and system,
    where the arrays have a batch axis before ``layer_axis``), max|got - ref|
    over max|ref| of that layer, for the layers whose reference norm is at
    least ``floor`` times the largest layer norm of the same system.
    Returns (worst error, index of that layer as a tuple)."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    lead = got.shape[:layer_axis + 1]
    g = got.reshape(lead + (-1,))
    r = ref.reshape(lead + (-1,))
    num = np.max(np.abs(g - r), axis=-1)
    den = np.max(np.abs(r), axis=-1)
    top = np.max(den, axis=layer_axis, keepdims=True)
    keep = (den >= floor * top) & (den > 0)
    err = np.where(keep, num / np.where(den > 0, den, 1.0), 0.0)
    idx = np.unravel_index(int(np.argmax(err)), err.shape)
    return float(err[idx]), tuple(int(i) for i in idx)
