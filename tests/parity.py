"""Comparison rules between the HIP path and the fp64 oracle.

Selection (block ids are integers decided by floating-point scores; the kernel
ranks fp32 scores, the oracle fp64 scores): the per-(head, group) count must match
exactly and the id sets must match exactly, except at an oracle near-tie -- when
the oracle's K-th and (K+1)-th candidate scores differ by less than
1e-4 * max(|s_K|, |s_K+1|) + 1e-6 * mean |s| over Omega.  Then every id in the
symmetric difference must lie inside that band around s_K.  Candidate sets not
larger than K must match exactly.

Attention outputs: bf16 inputs -- max-abs <= 2e-2 and mean-abs <= 2e-3 against the
fp64 oracle on the same rounded inputs; fp32 inputs -- max-abs <= 1e-5.
"""
from __future__ import annotations

import sys

import numpy as np

BF16_MAX_ABS, BF16_MEAN_ABS = 2e-2, 2e-3
F32_MAX_ABS = 1e-5
TIE_RTOL, TIE_FLOOR = 1e-4, 1e-6


def say(*args):
    print(*args, flush=True)
    sys.stdout.flush()


def check_selection(idx, cnt, ref, heads=None):
    """idx [H,R,K], cnt [H,R] from the GPU; ref = oracle.select(..., want_all_scores=True).
    Returns the number of (h, r) rows that differed inside the near-tie band."""
    idx = np.asarray(idx)
    cnt = np.asarray(cnt)
    H, R, K = ref["idx"].shape
    heads = range(H) if heads is None else heads
    ties = 0
    for h in heads:
        for r in range(R):
            c = int(ref["cnt"][h, r])
            assert int(cnt[h, r]) == c, f"count differs at h={h} r={r}: gpu {cnt[h, r]} oracle {c}"
            g = idx[h, r]
            assert (g[c:] == -1).all(), f"padding not -1 at h={h} r={r}"
            assert (np.diff(g[:c]) > 0).all(), f"ids not strictly ascending at h={h} r={r}: {g[:c]}"
            gset, oset = set(g[:c].tolist()), set(ref["idx"][h, r, :c].tolist())
            if gset == oset:
                continue
            s = ref["all_scores"][h, r]
            omega = ~np.isnan(s)
            assert all(omega[b] for b in gset), f"gpu selected a non-candidate block at h={h} r={r}"
            ids = np.nonzero(omega)[0]
            assert len(ids) > K, f"id sets differ with |Omega| <= K at h={h} r={r}"
            order = ids[np.lexsort((ids, -s[ids]))]
            sK, sK1 = s[order[K - 1]], s[order[K]]
            band = TIE_RTOL * max(abs(sK), abs(sK1)) + TIE_FLOOR * float(np.mean(np.abs(s[ids])))
            assert abs(sK - sK1) < band, (f"id sets differ outside a near-tie at h={h} r={r}: "
                                          f"gap {abs(sK - sK1):.3g} band {band:.3g} diff {sorted(gset ^ oset)}")
            for b in gset ^ oset:
                assert abs(s[b] - sK) <= band, f"mismatched id {b} outside the tie band at h={h} r={r}"
            ties += 1
    return ties


def errors(got, ref):
    got = np.asarray(got, dtype=np.float64)
    err = np.abs(got - ref)
    return float(err.max()) if err.size else 0.0, float(err.mean()) if err.size else 0.0


def check_bf16(got, ref, what):
    mx, mean = errors(got, ref)
    say(f"  {what}: max-abs {mx:.3e} mean-abs {mean:.3e} over {np.asarray(ref).size} values")
    assert np.isfinite(np.asarray(got, dtype=np.float64)).all(), f"{what}: non-finite output"
    assert mx <= BF16_MAX_ABS and mean <= BF16_MEAN_ABS, f"{what}: max-abs {mx:.3e} mean-abs {mean:.3e}"
    return mx, mean


def check_f32(got, ref, what):
    mx, mean = errors(got, ref)
    say(f"  {what}: max-abs {mx:.3e} mean-abs {mean:.3e} over {np.asarray(ref).size} values")
    assert mx <= F32_MAX_ABS, f"{what}: max-abs {mx:.3e}"
    return mx, mean


def check_lse(got, ref, what, tol):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    inf_ref = np.isneginf(ref)
    assert (np.isneginf(got) == inf_ref).all(), f"{what}: -inf pattern differs"
    err = np.abs(got[~inf_ref] - ref[~inf_ref])
    mx = float(err.max()) if err.size else 0.0
    say(f"  {what}: max |dLSE| {mx:.3e}")
    assert mx <= tol, f"{what}: |dLSE| {mx:.3e}"
