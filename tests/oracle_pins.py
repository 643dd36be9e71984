"""Pins for the fp64 oracle: each function checks the oracle against something the
paper or the mathematics fixes -- a worked example printed in the paper, a
hand-enumerated case of Eq. 2 / Eq. 3, a closed form, an identity, brute force on
tiny inputs, or a textbook special case computed by a library routine.

The functions are plain callables raising AssertionError, so that
``test_oracle_pins.py`` runs them against the oracle as built, and
``test_oracle_mutants.py`` runs the same battery against deliberately broken
builds of the oracle and requires every broken build to fail at least one pin.
"""
from __future__ import annotations

import itertools
import json
import math
import os

import numpy as np
import scipy.special as sps

import oracle as O

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def _case(seed, n=5, S=10, H=2, d=8, Lq=12):
    rng = np.random.default_rng(seed)
    q = rng.standard_normal((Lq, H, d))
    k = rng.standard_normal((n, S, H, d))
    v = rng.standard_normal((n, S, H, d))
    return q, k, v


def _block_tokens(b, S, B):
    """Chunk and chunk-local token range of block b (Alg. 1: c = b div Bpc, o = b mod Bpc)."""
    Bpc = -(-S // B)
    c, o = divmod(int(b), Bpc)
    return c, range(o * B, min(o * B + B, S))


def _library_attention(qv, keys, vals, scale):
    """Textbook softmax attention by library routines (scipy), one query."""
    logits = scale * (keys @ qv)
    return sps.softmax(logits) @ vals, float(sps.logsumexp(logits))


# --------------------------------------------------------------- worked examples

def pin_local_window_blocks():
    g = _golden("local_window_blocks.json")
    Bpc = O.blocks_per_chunk(g["S"], g["B"])
    assert g["N_w"] * Bpc == g["window_blocks"], (Bpc, g)
    n = 10
    omega, awe = O.candidates(n, Bpc, 4, g["N_w"], 3)
    assert awe
    assert int((~omega).sum()) == g["window_blocks"]
    assert not omega[-g["window_blocks"]:].any() and omega[: -g["window_blocks"]].all()


def pin_awe_tiny_config():
    g = _golden("awe_tiny_config.json")
    Bpc = O.blocks_per_chunk(g["S"], g["B"])
    for n_str, want in g["awe_by_history"].items():
        n = int(n_str)
        got = O.awe_active(n, g["window_chunks"], g["awe_min_outside_chunks"], g["top_k"], Bpc)
        assert got == want, (n, got, want)
        omega, awe = O.candidates(n, Bpc, g["top_k"], g["window_chunks"], g["awe_min_outside_chunks"])
        assert awe == want
        assert int(omega.sum()) == ((n - g["window_chunks"]) * Bpc if want else n * Bpc)


def pin_awe_block_guard():
    # Eq. 2's own guard: exclusion needs |H \ W| >= K blocks outside the window.
    Bpc = 4
    assert O.awe_active(10, 1, 0, 36, Bpc)        # 9 chunks * 4 = 36 blocks outside
    assert not O.awe_active(10, 1, 0, 37, Bpc)
    assert not O.awe_active(3, 3, 0, 1, Bpc)      # whole history inside the window
    assert not O.awe_active(2, 3, 0, 1, Bpc)
    assert O.awe_active(4, 0, 4, 1, Bpc) and not O.awe_active(3, 0, 4, 1, Bpc)


def pin_hand_selection():
    g = _golden("hand_selection.json")
    n = len(g["keys"])
    k = np.array(g["keys"], dtype=np.float64).reshape(n, 1, 1, g["d"])
    q = np.array(g["queries"], dtype=np.float64).reshape(-1, 1, g["d"])
    for case in g["cases"]:
        res = O.select(q, k, g["B"], case["K"], case["G_q"], case["E"], case["T_out"], 1.0,
                       resident=np.array(case["resident"], dtype=bool), want_all_scores=True)
        assert res["awe"] == case["awe"], case
        assert res["idx"][0].tolist() == case["idx"], (case, res["idx"])
        assert res["cnt"][0].tolist() == case["cnt"], (case, res["cnt"])
    res = O.select(q, k, 1, 1, 2, 1, 4, 1.0, want_all_scores=True)
    assert np.allclose(res["all_scores"][0, 0], g["proxy_scores_group_of_2"], atol=0, rtol=0)


def pin_hand_attention():
    g = _golden("hand_selection.json")
    n = len(g["keys"])
    k = np.array(g["keys"], dtype=np.float64).reshape(n, 1, 1, g["d"])
    v = np.array(g["values"], dtype=np.float64).reshape(n, 1, 1, g["d"])
    q = np.array(g["queries"], dtype=np.float64).reshape(-1, 1, g["d"])
    e = math.e
    # selection {0}: both queries see only token 0 -> O = v0, LSE = q.k0 = 1
    out, lse, _, _ = O.sparse_attn(q, k, v, 1, [[[0, -1]]], [[1]], 2, 1.0)
    assert np.allclose(out, [[10, 0], [10, 0]], atol=1e-14) and np.allclose(lse, [1, 1], atol=1e-14)
    # selection {0, 1}: query (1,1) has logits [1, 1]; query (1,-1) has logits [1, -1]
    out, lse, _, _ = O.sparse_attn(q, k, v, 1, [[[0, 1]]], [[2]], 2, 1.0)
    w = np.array([e, 1 / e]) / (e + 1 / e)
    assert np.allclose(out[0], [5, 5], atol=1e-13) and abs(lse[0] - (1 + math.log(2))) < 1e-13
    assert np.allclose(out[1], [10 * w[0], 10 * w[1]], atol=1e-13)
    assert abs(lse[1] - math.log(e + 1 / e)) < 1e-13


def pin_cross_query_union():
    g = _golden("cross_query_union.json")
    m = g["queries"]
    k = np.eye(m).reshape(m, 1, 1, m)          # one single-token block per chunk, keys e_j
    q = 3.0 * np.eye(m).reshape(m, 1, m)       # query j prefers block j
    res = O.select(q, k, 1, g["per_query_budget"], 1, 0, 0, 1.0)
    assert res["idx"][0, :, 0].tolist() == list(range(m))
    per, tot = O.union(res["idx"], res["cnt"], m)
    assert tot == g["union_blocks"] == g["history_blocks"] and per.tolist() == [g["union_blocks"]]
    # one shared group (Eq. 3): the union shrinks to R*K = 1 block
    res = O.select(q, k, 1, g["per_query_budget"], m, 0, 0, 1.0)
    per, tot = O.union(res["idx"], res["cnt"], m)
    assert tot == 1 and res["idx"].shape == (1, 1, 1)


def pin_union_bounds():
    rng = np.random.default_rng(7)
    H, R, K, nb = 5, 6, 4, 40
    idx = np.full((H, R, K), -1, dtype=np.int32)
    cnt = rng.integers(0, K + 1, size=(H, R)).astype(np.int32)
    for h in range(H):
        for r in range(R):
            idx[h, r, : cnt[h, r]] = np.sort(rng.choice(nb, cnt[h, r], replace=False))
    per, tot = O.union(idx, cnt, nb)
    sets = [set(idx[h][idx[h] >= 0].tolist()) for h in range(H)]
    assert per.tolist() == [len(s) for s in sets]
    assert tot == len(set().union(*sets))
    assert all(p <= min(R * K, nb) for p in per) and max(per) <= tot <= min(H * R * K, nb)


# ------------------------------------------------------------------ closed forms

def pin_pooling_closed_form():
    n, S, H, d, B = 3, 10, 2, 3, 4          # blocks of 4, 4, 2 tokens per chunk
    c, t, h, j = np.meshgrid(np.arange(n), np.arange(S), np.arange(H), np.arange(d), indexing="ij")
    k = (c * S + t) + 100.0 * h + 0.25 * j   # affine in the token index
    kbar = O.pool_keys(k, B)
    Bpc = 3
    for b in range(n * Bpc):
        cc, toks = _block_tokens(b, S, B)
        mid = cc * S + (toks[0] + toks[-1]) / 2.0   # mean of an arithmetic run
        for hh in range(H):
            assert np.allclose(kbar[hh, b], mid + 100.0 * hh + 0.25 * np.arange(d), atol=1e-12), (b, hh)
    # B = 1: pooling is the identity
    k2 = np.random.default_rng(3).standard_normal((2, 5, 2, 4))
    assert np.array_equal(O.pool_keys(k2, 1), k2.reshape(10, 2, 4).transpose(1, 0, 2))


def pin_group_mean_queries():
    rng = np.random.default_rng(11)
    q = rng.standard_normal((13, 2, 3))
    qbar = O.proxy_queries(q, 5)                  # groups of 5, 5, 3 rows
    assert qbar.shape == (2, 3, 3)
    for r, (a, b) in enumerate([(0, 5), (5, 10), (10, 13)]):
        assert np.allclose(qbar[:, r], q[a:b].sum(axis=0) / (b - a), atol=1e-14)
    assert np.allclose(O.proxy_queries(q, 1), q.transpose(1, 0, 2), atol=0)


def pin_scores_linearity():
    # Eq. 3: the group average of the per-query scores of Eq. 2 is what the
    # proxy-query form of the selection ranks.
    q, k, _ = _case(5, n=4, S=10, H=2, d=6, Lq=12)
    B, G, scale = 4, 5, 0.37
    per_q = O.query_scores(q, k, B, scale)         # [H, Lq, N_b]
    res = O.select(q, k, B, 3, G, 1, 100, scale, want_all_scores=True)
    for r, (a, b) in enumerate([(0, 5), (5, 10), (10, 12)]):
        assert np.allclose(res["all_scores"][:, r], per_q[:, a:b].mean(axis=1), atol=1e-12)


def pin_topk_brute_force():
    # The chosen set is the K-subset of Omega with the largest score sum; scores
    # are recomputed here from numpy means of the token slices.
    for seed in range(6):
        q, k, _ = _case(100 + seed, n=4, S=7, H=2, d=5, Lq=6)
        B, K, G, E, T, scale = 3, 3, 4, 1, 2, 0.5
        Bpc = 3
        resident = np.ones(4 * Bpc, dtype=bool)
        resident[seed % 12] = False
        res = O.select(q, k, B, K, G, E, T, scale, resident=resident)
        awe = (4 - E >= T) and ((4 - E) * Bpc >= K)
        assert res["awe"] == awe
        cand = [b for b in range(4 * Bpc) if resident[b] and not (awe and b // Bpc >= 4 - E)]
        for h in range(2):
            for r, (a, z) in enumerate([(0, 4), (4, 6)]):
                qb = q[a:z, h].mean(axis=0)
                sc = {}
                for b in cand:
                    c, toks = _block_tokens(b, 7, B)
                    sc[b] = scale * float(qb @ k[c, list(toks), h].mean(axis=0))
                best = max(itertools.combinations(cand, K), key=lambda s: sum(sc[b] for b in s))
                assert res["idx"][h, r].tolist() == sorted(best), (seed, h, r)
                assert res["cnt"][h, r] == K
                assert np.allclose(res["score"][h, r], [sc[b] for b in sorted(best)], atol=1e-12)


def pin_topk_ties_and_padding():
    # identical blocks tie exactly: the lower id wins; short candidate sets pad with -1
    k = np.ones((3, 4, 1, 2))                       # every block has the same pooled key
    q = np.ones((2, 1, 2))
    res = O.select(q, k, 2, 3, 2, 1, 0, 1.0)        # AWE on: Omega = blocks 0..3
    assert res["awe"] and res["idx"][0, 0].tolist() == [0, 1, 2]
    res = O.select(q, k, 2, 9, 2, 1, 0, 1.0)        # |H\W| = 4 < 9: AWE off, all 6 blocks
    assert not res["awe"] and res["idx"][0, 0].tolist() == [0, 1, 2, 3, 4, 5, -1, -1, -1]
    assert res["cnt"][0, 0] == 6 and np.isneginf(res["score"][0, 0, 6:]).all()
    res = O.select(q, np.zeros((0, 4, 1, 2)), 2, 3, 2, 1, 0, 1.0)   # empty history
    assert res["cnt"][0, 0] == 0 and res["idx"][0, 0].tolist() == [-1, -1, -1]


# ------------------------------------------------------------- attention pins

def pin_dense_vs_library():
    q, k, v = _case(21, n=3, S=10, H=2, d=8, Lq=9)
    scale = 1 / math.sqrt(8)
    for c0, c1 in [(0, 3), (2, 3), (1, 3)]:
        out, lse, hs, qs = O.dense_attn(q, k, v, 4, c0, c1, scale)
        for i, (h, qi) in enumerate(zip(hs, qs)):
            keys = k[c0:c1, :, h].reshape(-1, 8)
            vals = v[c0:c1, :, h].reshape(-1, 8)
            ref, ref_lse = _library_attention(q[qi, h], keys, vals, scale)
            assert np.allclose(out[i], ref, atol=1e-12) and abs(lse[i] - ref_lse) < 1e-12, (c0, c1, h, qi)


def pin_sparse_vs_library():
    q, k, v = _case(22, n=4, S=10, H=2, d=8, Lq=10)
    B, G, K, scale = 4, 4, 5, 0.3
    Bpc, R = 3, 3
    rng = np.random.default_rng(1)
    idx = np.full((2, R, K), -1, dtype=np.int32)
    cnt = np.zeros((2, R), dtype=np.int32)
    for h in range(2):
        for r in range(R):
            cnt[h, r] = rng.integers(1, K + 1)
            idx[h, r, : cnt[h, r]] = rng.integers(0, 4 * Bpc, size=cnt[h, r])   # duplicates allowed
    out, lse, hs, qs = O.sparse_attn(q, k, v, B, idx, cnt, G, scale)
    for i, (h, qi) in enumerate(zip(hs, qs)):
        r = qi // G
        rows_k, rows_v = [], []
        for b in idx[h, r, : cnt[h, r]]:
            c, toks = _block_tokens(b, 10, B)
            rows_k.append(k[c, list(toks), h])
            rows_v.append(v[c, list(toks), h])
        ref, ref_lse = _library_attention(q[qi, h], np.concatenate(rows_k), np.concatenate(rows_v), scale)
        assert np.allclose(out[i], ref, atol=1e-12) and abs(lse[i] - ref_lse) < 1e-12, (h, qi)


def pin_sparse_all_blocks_equals_dense():
    # With K covering every block (exclusion then off), selection attention is full attention.
    q, k, v = _case(23, n=3, S=10, H=2, d=8, Lq=8)
    B, scale = 4, 0.35
    res = O.select(q, k, B, 9, 8, 1, 3, scale)
    assert not res["awe"] and (res["cnt"] == 9).all()
    o1, l1, _, _ = O.sparse_attn(q, k, v, B, res["idx"], res["cnt"], 8, scale)
    o2, l2, _, _ = O.dense_attn(q, k, v, B, 0, 3, scale)
    assert np.allclose(o1, o2, atol=1e-12) and np.allclose(l1, l2, atol=1e-12)


def pin_cmp_constant_blocks_equals_full():
    # Compression attention (Eq. 1's CMP branch over App. C's pooled history): with
    # every token of a block equal and every block full (S a multiple of B), a
    # block's pooled token is that token, and full attention gives each block B equal
    # logits, so the softmax weights of the two agree and their LSEs differ by ln B.
    rng = np.random.default_rng(61)
    n, S, H, d, B = 3, 8, 2, 5, 4
    k = np.repeat(rng.standard_normal((n, S // B, H, d)), B, axis=1)
    v = np.repeat(rng.standard_normal((n, S // B, H, d)), B, axis=1)
    q = rng.standard_normal((6, H, d))
    kc, vc = O.cmp_cache(k, v, B)
    assert kc.shape == (H, n * S // B, d)
    o1, l1, _, _ = O.cmp_attn(q, kc, vc, 0.4)
    o2, l2, _, _ = O.dense_attn(q, k, v, B, 0, n, 0.4)
    assert np.allclose(o1, o2, atol=1e-12) and np.allclose(l1 + math.log(B), l2, atol=1e-12)


def pin_cmp_vs_library():
    # Pooled tokens as numpy block means (partial tail blocks included), then
    # textbook softmax attention by library routines over them.
    q, k, v = _case(62, n=3, S=10, H=2, d=6, Lq=5)
    B, scale = 4, 0.45
    kc, vc = O.cmp_cache(k, v, B)
    out, lse, hs, qs = O.cmp_attn(q, kc, vc, scale)
    nb = 3 * O.blocks_per_chunk(10, B)
    for i, (h, qi) in enumerate(zip(hs, qs)):
        keys = np.stack([k[c, list(t), h].mean(axis=0) for c, t in (_block_tokens(b, 10, B) for b in range(nb))])
        vals = np.stack([v[c, list(t), h].mean(axis=0) for c, t in (_block_tokens(b, 10, B) for b in range(nb))])
        ref, ref_lse = _library_attention(q[qi, h], keys, vals, scale)
        assert np.allclose(out[i], ref, atol=1e-12) and abs(lse[i] - ref_lse) < 1e-12, (h, qi)
    # no history: O = 0, LSE = -inf
    out, lse, _, _ = O.cmp_attn(q, kc[:, :0], vc[:, :0], scale)
    assert np.all(out == 0) and np.all(np.isneginf(lse))


def pin_bf16_rounding():
    # bfloat16 keeps 8 significant bits; ties go to the even significand.
    one = 1.0
    cases = {one + 2.0 ** -8: one,                       # tie, even below
             one + 3 * 2.0 ** -8: one + 2.0 ** -6,       # tie, even above
             one + 2.0 ** -8 + 2.0 ** -20: one + 2.0 ** -7,
             -(2.0 + 2.0 ** -7): -2.0,                   # tie at a larger exponent
             255.5: 256.0, 0.0: 0.0}
    for x, want in cases.items():
        assert O.round_bf16(x) == want, (x, O.round_bf16(x), want)
    # against a library conversion on values that fp32 holds exactly
    import torch
    x = np.random.default_rng(63).standard_normal(4096).astype(np.float32).astype(np.float64)
    lib = torch.from_numpy(x).to(torch.float32).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(O.round_bf16(x), lib)


def pin_prob_scores_where_readings_differ():
    # A worked case where the probability-averaged score and the mean-logit score
    # (reading R1) rank differently.  One-hot pooled keys make the logits the query
    # entries: query 1 strongly prefers block 1, query 2 mildly prefers block 0.
    # Mean logits (1, -5, 0) pick block 0; mean probabilities pick block 1.
    q = np.array([[[0.0, 10.0, 0.0]], [[2.0, -20.0, 0.0]]])      # [Lq=2, H=1, d=3]
    k = np.eye(3).reshape(3, 1, 1, 3)                            # 3 chunks of one 1-token block
    logit = O.select(q, k, 1, 1, 2, 0, 0, 1.0)
    assert logit["idx"].tolist() == [[[0]]], logit
    kc = O.pool_keys(k, 1)
    prob = O.select_prob(q, kc, 3, 1, 1, 2, 0, 0, 1.0, want_all_scores=True)
    assert prob["idx"].tolist() == [[[1]]], prob
    want = (sps.softmax(q[0, 0]) + sps.softmax(q[1, 0])) / 2     # library softmax per query
    assert np.allclose(prob["all_scores"][0, 0], want, rtol=1e-14, atol=0), (prob["all_scores"], want)
    assert prob["score"][0, 0, 0] == prob["all_scores"][0, 0, 1]


def pin_prob_scores_vs_library():
    # Library softmax of numpy logits over every pooled key, averaged over each
    # group's rows (ragged last group), on random inputs; window excluded by AWE.
    q, k, _ = _case(71, n=5, S=10, H=2, d=6, Lq=11)
    B, G, scale = 4, 3, 0.6
    Bpc = O.blocks_per_chunk(10, B)
    kc = O.pool_keys(k, B)
    got = O.select_prob(q, kc, 5, Bpc, 3, G, 1, 2, scale, want_all_scores=True)
    assert got["awe"]
    omega, _ = O.candidates(5, Bpc, 3, 1, 2)
    for h in range(2):
        p = sps.softmax(scale * (q[:, h] @ kc[h].T), axis=1)     # [Lq, N]
        for r in range(-(-11 // G)):
            want = p[r * G: min(r * G + G, 11)].mean(axis=0)
            have = got["all_scores"][h, r]
            assert np.all(np.isnan(have[~omega])), (h, r)
            assert np.allclose(have[omega], want[omega], rtol=1e-12, atol=0), (h, r)
            top = sorted(np.flatnonzero(omega), key=lambda b: (-want[b], b))[:3]
            assert got["idx"][h, r].tolist() == sorted(top), (h, r)


def pin_prob_scores_invariants():
    # (a) Without exclusion each group's scores are a mean of probability vectors, so
    #     they sum to 1 over the blocks.
    # (b) Adding one vector c to every pooled key shifts each query's logits by a
    #     constant, which its softmax removes: the scores do not change.
    # (c) Softmax is monotone, so with one query per group, or groups of identical
    #     rows, the top-K equals the mean-logit selection (reading R1).
    q, k, _ = _case(72, n=4, S=9, H=3, d=5, Lq=10)
    B, scale = 3, 0.7
    Bpc = O.blocks_per_chunk(9, B)
    kc = O.pool_keys(k, B)
    a = O.select_prob(q, kc, 4, Bpc, 4, 3, 0, 0, scale, want_all_scores=True)
    assert np.allclose(a["all_scores"].sum(axis=-1), 1.0, rtol=0, atol=1e-12), a["all_scores"].sum(axis=-1)
    c = np.random.default_rng(73).standard_normal(5)
    b = O.select_prob(q, kc + c, 4, Bpc, 4, 3, 0, 0, scale, want_all_scores=True)
    assert np.allclose(a["all_scores"], b["all_scores"], rtol=1e-11, atol=1e-15)
    assert np.array_equal(a["idx"], b["idx"])
    resident = np.ones(4 * Bpc, dtype=bool)
    resident[[1, 5]] = False
    for E, T_out in ((0, 0), (1, 2), (2, 0)):
        one = O.select_prob(q, kc, 4, Bpc, 3, 1, E, T_out, scale, resident=resident)
        ref = O.select(q, k, B, 3, 1, E, T_out, scale, resident=resident)
        assert np.array_equal(one["idx"], ref["idx"]) and np.array_equal(one["cnt"], ref["cnt"]), (E, T_out)
        assert one["awe"] == ref["awe"]
    G = 4
    rep = np.repeat(q[::G], G, axis=0)[:10]                      # rows of each group identical
    same = O.select_prob(rep, kc, 4, Bpc, 3, G, 1, 2, scale, resident=resident)
    ref = O.select(rep, k, B, 3, G, 1, 2, scale, resident=resident)
    assert np.array_equal(same["idx"], ref["idx"]) and np.array_equal(same["cnt"], ref["cnt"])


def pin_gated_combine():
    # Eq. 1 with sigmoid gates: a saturated gate keeps or drops a branch exactly,
    # a zero logit weighs a branch by 1/2, and sigmoid(x) + sigmoid(-x) = 1.
    rng = np.random.default_rng(64)
    a, b, c = (rng.standard_normal((5, 2, 4)) for _ in range(3))
    big = np.full((5, 2, 3), -800.0)
    only = big.copy()
    only[..., 1] = 800.0                                       # SLC alone
    assert np.array_equal(O.gated_combine(a, b, c, only), b)
    half = np.zeros((5, 2, 3))
    assert np.allclose(O.gated_combine(a, b, c, half), (a + b + c) / 2, atol=1e-15)
    x = rng.standard_normal((5, 2))
    sym = np.stack([x, -x, np.full_like(x, -800.0)], axis=-1)
    assert np.allclose(O.gated_combine(a, a, c, sym), a, atol=1e-15)
    # a missing branch contributes nothing
    assert np.allclose(O.gated_combine(None, b, c, only), b, atol=0)
    g = rng.standard_normal((5, 2, 3))
    assert np.allclose(O.gated_combine(a, b, None, g) + O.gated_combine(None, None, c, g),
                       O.gated_combine(a, b, c, g), atol=1e-14)
    # Finite logits: sigmoid(ln 3) = 3/4 and sigmoid(-ln 3) = 1/4 exactly, since
    # 1 / (1 + e^{-ln 3}) = 1 / (1 + 1/3).  A slip such as sigmoid(2x) = (1 + tanh x) / 2
    # keeps every property above but fails these.
    ones = np.ones((1, 1, 1))
    three = np.full((1, 1, 3), -800.0)
    three[..., 0] = math.log(3.0)
    assert abs(O.gated_combine(ones, None, None, three)[0, 0, 0] - 0.75) < 1e-15
    three[..., 0] = -math.log(3.0)
    assert abs(O.gated_combine(ones, None, None, three)[0, 0, 0] - 0.25) < 1e-15
    # Random logits over the whole range against the library logistic function.
    g = rng.standard_normal((5, 2, 3)) * 6.0
    ref = sps.expit(g[..., 0:1]) * a + sps.expit(g[..., 1:2]) * b + sps.expit(g[..., 2:3]) * c
    assert np.allclose(O.gated_combine(a, b, c, g), ref, rtol=1e-14, atol=1e-15)


def pin_attention_special_cases():
    rng = np.random.default_rng(31)
    n, S, H, d = 2, 6, 1, 4
    q = rng.standard_normal((3, H, d))
    k = rng.standard_normal((n, S, H, d))
    v = np.broadcast_to(np.array([1.5, -2.0, 0.25, 3.0]), (n, S, H, d)).copy()
    out, _, _, _ = O.dense_attn(q, k, v, 4, 0, n, 0.7)               # constant V -> O = V
    assert np.allclose(out, v[0, 0, 0], atol=1e-13)
    k_eq = np.broadcast_to(rng.standard_normal(d), (n, S, H, d)).copy()
    v2 = rng.standard_normal((n, S, H, d))
    out, lse, hs, qs = O.dense_attn(q, k_eq, v2, 4, 0, n, 0.7)       # equal keys -> mean of V
    assert np.allclose(out, v2.reshape(-1, d).mean(axis=0), atol=1e-13)
    assert np.allclose(lse, 0.7 * (q[qs, 0] @ k_eq[0, 0, 0]) + math.log(n * S), atol=1e-12)
    # a selected block holding one token returns that token's value (B = 1)
    out, lse, _, _ = O.sparse_attn(q, k, v2, 1, [[[7, -1]]], [[1]], 3, 0.7)
    assert np.allclose(out, v2[1, 1, 0], atol=0)


def pin_lse_merge_and_order():
    q, k, v = _case(41, n=4, S=10, H=1, d=6, Lq=4)
    B, scale = 4, 0.4
    full = np.array([[[0, 4, 7, 9, 11]]], dtype=np.int32)
    o, l, _, _ = O.sparse_attn(q, k, v, B, full, [[5]], 4, scale)
    oa, la, _, _ = O.sparse_attn(q, k, v, B, full[:, :, :2], [[2]], 4, scale)
    ob, lb, _, _ = O.sparse_attn(q, k, v, B, full[:, :, 2:], [[3]], 4, scale)
    lm = np.logaddexp(la, lb)
    om = (np.exp(la - lm)[:, None] * oa + np.exp(lb - lm)[:, None] * ob)
    assert np.allclose(l, lm, atol=1e-12) and np.allclose(o, om, atol=1e-12)
    perm = np.array([[[11, 0, 9, 4, 7]]], dtype=np.int32)              # list order is irrelevant
    op, lp, _, _ = O.sparse_attn(q, k, v, B, perm, [[5]], 4, scale)
    assert np.allclose(op, o, atol=1e-12) and np.allclose(lp, l, atol=1e-12)


def pin_residency_and_empty():
    q, k, v = _case(51, n=3, S=10, H=2, d=4, Lq=5)
    B, scale = 4, 0.5
    resident = np.ones(9, dtype=bool)
    resident[[2, 4]] = False
    lst = np.array([[[1, 2, 4, 6]], [[1, 2, 4, 6]]], dtype=np.int32)
    o1, l1, _, _ = O.sparse_attn(q, k, v, B, lst, [[4], [4]], 5, scale, resident=resident)
    lst2 = np.array([[[1, 6]], [[1, 6]]], dtype=np.int32)
    o2, l2, _, _ = O.sparse_attn(q, k, v, B, lst2, [[2], [2]], 5, scale)
    assert np.allclose(o1, o2, atol=0) and np.allclose(l1, l2, atol=0)
    res = O.select(q, k, B, 9, 5, 0, 0, scale, resident=resident)
    assert res["cnt"].tolist() == [[7], [7]] and not np.isin(res["idx"], [2, 4]).any()
    # dense attention skips non-resident blocks too
    od, ld, _, _ = O.dense_attn(q, k, v, B, 0, 3, scale, resident=resident)
    keep = [b for b in range(9) if resident[b]]
    os_, ls_, _, _ = O.sparse_attn(q, k, v, B, np.tile(np.array(keep, np.int32), (2, 1, 1)), [[7], [7]], 5, scale)
    assert np.allclose(od, os_, atol=1e-12) and np.allclose(ld, ls_, atol=1e-12)
    # empty list: O = 0, LSE = -inf
    o0, l0, _, _ = O.sparse_attn(q, k, v, B, np.full((2, 1, 3), -1, np.int32), [[0], [0]], 5, scale)
    assert (o0 == 0).all() and np.isneginf(l0).all()


def pin_permutation_equivariance():
    # Prop. J.1 (App. J): jointly permuting cache tokens leaves each query's output
    # unchanged, and permuting the queries permutes the outputs.
    q, k, v = _case(61, n=3, S=8, H=2, d=6, Lq=7)
    scale = 0.45
    o, l, hs, qs = O.dense_attn(q, k, v, 4, 0, 3, scale)
    rng = np.random.default_rng(2)
    pk = rng.permutation(24)
    kp = k.reshape(24, 2, 6)[pk].reshape(3, 8, 2, 6)
    vp = v.reshape(24, 2, 6)[pk].reshape(3, 8, 2, 6)
    o2, l2, _, _ = O.dense_attn(q, kp, vp, 4, 0, 3, scale)
    assert np.allclose(o, o2, atol=1e-12) and np.allclose(l, l2, atol=1e-12)
    pq = rng.permutation(7)
    o3, l3, hs3, qs3 = O.dense_attn(q[pq], k, v, 4, 0, 3, scale)
    ref = {(h, qi): i for i, (h, qi) in enumerate(zip(hs, qs))}
    for i, (h, qi) in enumerate(zip(hs3, qs3)):
        j = ref[(h, pq[qi])]
        assert np.allclose(o3[i], o[j], atol=1e-12) and abs(l3[i] - l[j]) < 1e-12


def pin_widening_of_stored_types():
    # fp32 and bf16 inputs are widened exactly: results equal the float64 run on the same values.
    import torch
    q, k, v = _case(71, n=2, S=10, H=2, d=8, Lq=6)
    qb = torch.from_numpy(q).to(torch.bfloat16)
    kb = torch.from_numpy(k).to(torch.bfloat16)
    vb = torch.from_numpy(v).to(torch.bfloat16)
    o1, l1, _, _ = O.dense_attn(qb, kb, vb, 4, 0, 2, 0.3)
    o2, l2, _, _ = O.dense_attn(qb.double().numpy(), kb.double().numpy(), vb.double().numpy(), 4, 0, 2, 0.3)
    assert np.array_equal(o1, o2) and np.array_equal(l1, l2)
    o3, l3, _, _ = O.dense_attn(qb.float(), kb.float(), vb.float(), 4, 0, 2, 0.3)
    assert np.array_equal(o1, o3) and np.array_equal(l1, l3)


def pin_lru_policy():
    # The textbook page-replacement example (Silberschatz, Galvin and Gagne,
    # "Operating System Concepts", the LRU example on 3 frames): this reference string
    # gives 12 faults under LRU (15 under FIFO, 9 under the optimal policy).
    ref = [7, 0, 1, 2, 0, 3, 0, 4, 2, 3, 0, 3, 2, 1, 2, 0, 1, 7, 0, 1]
    r = O.lru_simulate([[c] for c in ref], 3)
    assert (r["misses"], r["hits"], r["evictions"]) == (12, 8, 9), r
    # with one chunk per request, LRU keeps exactly the last `slots` distinct chunks
    # requested (scanning the history backwards)
    rng = np.random.default_rng(81)
    for slots in (1, 2, 4):
        seq = rng.integers(0, 7, 40).tolist()
        for t in range(1, len(seq) + 1):
            r = O.lru_simulate([[c] for c in seq[:t]], slots)
            last = []
            for c in reversed(seq[:t]):
                if c not in last:
                    last.append(c)
                if len(last) == slots:
                    break
            assert set(r["slot_of"]) == set(last), (slots, t)
    # enough slots: only the first use of each chunk misses; slots fill from 0
    r = O.lru_simulate([[4, 1], [1, 9], [4], [2, 9]], 5)
    assert (r["misses"], r["hits"], r["evictions"]) == (4, 3, 0)
    assert r["slot_of"] == {1: 0, 4: 1, 9: 2, 2: 3}
    # a request's chunks are all resident afterwards, and the evicted chunk is the
    # least recently used one the request does not name: after [0,1], [2,3], [1],
    # the order is 0, 2, 3, 1; [0, 5] keeps 0 (a hit) and evicts 2
    r = O.lru_simulate([[0, 1], [2, 3], [1], [0, 5]], 4)
    assert set(r["slot_of"]) == {0, 1, 3, 5} and r["slot_of"][5] == 2 and r["per_request"][-1] == (1, 1)
    # hits refresh recency: after [0], [1], [0], a new chunk evicts 1 (not 0)
    r = O.lru_simulate([[0], [1], [0], [2]], 2)
    assert set(r["slot_of"]) == {0, 2} and r["slot_of"][2] == 1


ALL_PINS = [obj for name, obj in sorted(globals().items()) if name.startswith("pin_") and callable(obj)]
