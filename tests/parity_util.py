"""Comparison rules shared by the GPU parity tests.

Integer outputs (queue ids, boundaries, counts, sums) must match the oracle
bit for bit.  Scores are binary32 on the GPU against the oracle's binary64
definition rounded once to binary32: they must agree to 1e-5 relative.  The
admitted sets may differ only in requests whose oracle score lies within
1e-5 (relative) of the oracle's B-th admitted score.
"""
import numpy as np

SCORE_RTOL = 1e-5


def check_scores(gpu, ref, rtol=SCORE_RTOL):
    gpu = np.asarray(gpu, np.float32)
    ref = np.asarray(ref, np.float32)
    assert gpu.shape == ref.shape
    assert np.array_equal(np.isnan(gpu), np.isnan(ref)), "NaN (empty-slot) positions differ"
    fin = np.isfinite(ref)
    assert np.array_equal(np.isinf(gpu) & (gpu < 0), np.isinf(ref) & (ref < 0))
    g, r = gpu[fin].astype(np.float64), ref[fin].astype(np.float64)
    err = np.abs(g - r) / np.maximum(np.abs(r), 1e-30)
    worst = float(err.max()) if err.size else 0.0
    assert worst <= rtol, f"score relative error {worst:.3e} > {rtol}"
    return worst


def check_admission(gpu_ids, gpu_top, gpu_nsel, ref_ids, ref_top, ref_nsel, ref_scores, rtol=SCORE_RTOL):
    """One parameter vector.  ref_scores: the oracle's full score row."""
    gpu_ids = np.asarray(gpu_ids)
    ref_ids = np.asarray(ref_ids)
    assert int(gpu_nsel) == int(ref_nsel), f"n_sel {gpu_nsel} != {ref_nsel}"
    n = int(ref_nsel)
    assert np.all(gpu_ids[n:] == -1) and np.all(np.isnan(np.asarray(gpu_top)[n:]))
    if n == 0:
        return 0
    g = gpu_ids[:n]
    assert len(set(g.tolist())) == n, "duplicate admitted id"
    kB = float(ref_top[n - 1])
    diff = set(g.tolist()) ^ set(ref_ids[:n].tolist())
    for i in diff:
        s = float(ref_scores[i])
        assert abs(s - kB) <= rtol * max(abs(kB), 1e-30), f"id {i} (score {s}) differs away from the cut {kB}"
    # reported scores belong to the ids and are in (score desc, id asc) order
    top = np.asarray(gpu_top[:n], np.float64)
    rs = np.asarray(ref_scores, np.float64)[g]
    ok = np.isclose(top, rs, rtol=rtol, atol=0) | (np.isinf(top) & np.isinf(rs))
    assert np.all(ok), "reported scores do not match the admitted ids"
    for a in range(n - 1):
        assert top[a] > top[a + 1] or (top[a] == top[a + 1] and g[a] < g[a + 1]), "admission order broken"
    return len(diff)


def check_table(gpu_tab: dict, ref) -> None:
    """Bit-exact comparison of a GPU queue table with an oracle Table."""
    assert gpu_tab["k"] == ref.k, f"k {gpu_tab['k']} != {ref.k}"
    assert np.array_equal(gpu_tab["bounds"], ref.bounds), "bounds differ"
    assert np.array_equal(gpu_tab["count"], ref.count), "counts differ"
    assert np.array_equal(gpu_tab["sum"], ref.sum), "sums differ"
    assert np.array_equal(gpu_tab["lo"], ref.lo) and np.array_equal(gpu_tab["hi"], ref.hi), "lo/hi differ"
    assert np.array_equal(gpu_tab["mean"].view(np.uint64), ref.mean.view(np.uint64)), "means differ"
    assert gpu_tab["n_distinct"] == ref.n_distinct
    assert gpu_tab["n_coarse"] == ref.n_coarse
    assert gpu_tab["n_leaves"] == ref.n_leaves
