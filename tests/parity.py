"""Comparison rules shared by the GPU parity tests.

The library and the oracle compute distances as squared L2 accumulated in
double and rounded once to float, in different summation orders; the double
sums differ by ~1e-16 relative, so after rounding the floats agree except in
rare cases where they are one float ulp apart.  Search trajectories are then
identical and results must match exactly: same ids, bit-identical distances.
The residual rule covers the rare ulp case: a query whose rows differ must
agree on every distance within 1e-4 relative, and may differ in ids only
inside runs of near-tied distances (|delta| <= 1e-4 relative) of the oracle's
row.  At most `max_residual` such queries are tolerated.
"""
import numpy as np

REL = 1e-4


def _tie_runs(d):
    """Group positions of a sorted distance row into runs of near ties."""
    runs = []
    start = 0
    for i in range(1, len(d) + 1):
        if i == len(d) or not (np.isfinite(d[i]) and abs(float(d[i]) - float(d[i - 1])) <= REL * max(abs(float(d[i])), 1e-30)):
            runs.append((start, i))
            start = i
    return runs


def compare_rows(g_ids, g_d, o_ids, o_d):
    """Returns 'exact', 'tie' or a string describing the failure."""
    if (g_ids == o_ids).all() and (g_d.view(np.uint32) == o_d.view(np.uint32)).all():
        return "exact"
    fin = np.isfinite(o_d)
    if not (np.isfinite(g_d) == fin).all():
        return f"padding differs: gpu {g_ids.tolist()} oracle {o_ids.tolist()}"
    if not np.allclose(g_d[fin], o_d[fin], rtol=REL, atol=0):
        return f"distances differ: gpu {g_d.tolist()} oracle {o_d.tolist()}"
    for a, b in _tie_runs(o_d[fin]):
        if sorted(g_ids[a:b].tolist()) != sorted(o_ids[a:b].tolist()):
            # ids may leave a run only at the row's end (the k-th slot tie)
            if b != fin.sum():
                return f"ids differ outside a tie run: gpu {g_ids.tolist()} oracle {o_ids.tolist()}"
    return "tie"


def assert_parity(g_ids, g_d, o_ids, o_d, max_residual=1):
    g_ids = np.asarray(g_ids)
    g_d = np.asarray(g_d, dtype=np.float32)
    o_ids = np.asarray(o_ids)
    o_d = np.asarray(o_d, dtype=np.float32)
    assert g_ids.shape == o_ids.shape and g_d.shape == o_d.shape
    residual = []
    for i in range(g_ids.shape[0]):
        res = compare_rows(g_ids[i], g_d[i], o_ids[i], o_d[i])
        if res == "exact":
            continue
        assert res == "tie", f"query {i}: {res}"
        residual.append(i)
    assert len(residual) <= max_residual, f"{len(residual)} queries differ within ties: {residual[:10]}"
    return residual
