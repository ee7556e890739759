"""Pins of the CPU oracle against what the paper and mathematics fix (no GPU needed).

Each test checks the oracle against something other than itself: closed forms, invariants, special
cases that reduce to a library routine (torch / numpy), or brute force on tiny inputs.
"""
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle
import synth
from helpers import from_bits, rng, to_bits


# ------------------------------------------------------------------------ rules of the method
def test_window_rows_follow_static_eviction_setup():
    # App. F: last 20% of the prompt, 10% beyond 24k tokens (rounded down).
    assert [oracle.window_rows(T) for T in (512, 2048, 8192)] == [102, 409, 1638]
    assert [oracle.window_rows(T) for T in (32768, 131072)] == [3276, 13107]
    assert oracle.window_rows(24576) == 4915      # 20% at exactly 24k
    assert oracle.window_rows(24577) == 2457      # 10% just above
    assert oracle.window_rows(3) == 1


def test_owner_layer_skips_first_two_layers():
    # Sec. 3.4: pairs of adjacent layers share, the first two layers never do.
    assert [oracle.owner_layer(l, 2, 2) for l in range(12)] == [0, 1, 2, 2, 4, 4, 6, 6, 8, 8, 10, 10]
    got = [oracle.owner_layer(l, 4, 2) for l in range(12)]
    assert got == [0, 1, 2, 2, 2, 2, 6, 6, 6, 6, 10, 10]
    # Alg. 3's literal "l % 2" pairing is start = 0.
    assert [oracle.owner_layer(l, 2, 0) for l in range(6)] == [0, 0, 2, 2, 4, 4]
    assert [oracle.owner_layer(l, 1, 2) for l in range(5)] == list(range(5))


@pytest.mark.parametrize("name", ["C1", "C2", "C3", "C4", "C5", "X1"])
def test_workload_integers_follow_the_rules(name):
    w = synth.get(name)
    assert w.window == oracle.window_rows(w.T)
    assert w.keep == oracle.keep_tokens(w.T, w.static_ratio, w.cluster)
    C = -(-w.keep // w.cluster)
    S = -(-C // w.fanout)
    assert w.k_super == oracle.level1_keep(S, w.dynamic_ratio)
    assert w.k_clusters == oracle.level2_keep(w.keep, w.dynamic_ratio, w.cluster, w.k_super * w.fanout)


def test_level2_budget_of_the_prompt_reading():
    # The Fig. 9 caption, which calls eta the final budget of the KV cache, reads it against the prompt: at the GPT-2 workload
    # (T = 2048, static ratio 50%, eta = 12.5%, s = 16) that is 2048 / 8 / 16 = 16 clusters, twice
    # the 8 clusters of the post-eviction reading.
    w = synth.get("C2")
    assert oracle.level2_keep(w.keep, w.dynamic_ratio, w.cluster, w.k_super * w.fanout) == 8
    assert oracle.level2_keep_of_prompt(w.T, w.dynamic_ratio, w.cluster, w.k_super * w.fanout) == 16
    # 128K GQA: 2% of 131072 tokens in clusters of 64 = 40.96 -> 40 clusters (10 under the other reading)
    assert oracle.level2_keep_of_prompt(131072, 0.02, 64, 256) == 40
    # rounding down, at least one cluster, at most the candidates
    assert oracle.level2_keep_of_prompt(1000, 0.001, 16, 8) == 1
    assert oracle.level2_keep_of_prompt(8192, 0.5, 32, 64) == 64
    for name in ("C2", "C3", "C4", "C5", "X1"):
        w = synth.get(name)
        k = oracle.level2_keep_of_prompt(w.T, w.dynamic_ratio, w.cluster, w.k_super * w.fanout)
        # the selected tokens are the largest whole-cluster count within eta * T
        assert k * w.cluster <= w.dynamic_ratio * w.T < (k + 1) * w.cluster
        assert synth.get(name + "-T").k_clusters == k
        # with static ratio r the prompt reading selects about 1 / r times as many clusters
        assert abs(k / w.k_clusters - 1 / w.static_ratio) <= 1 / w.k_clusters * (1 + 1 / w.static_ratio)
    assert synth.get("C1-T").k_clusters == synth.get("C1").k_clusters == 8


def test_workload_derived_sizes():
    # cluster / super-cluster counts and owner-layer counts of the five workloads
    exp = {"C1": (16, 4, 1), "C2": (64, 16, 7), "C3": (128, 16, 10), "C4": (307, 39, 10),
           "C5": (512, 64, 10), "X1": (128, 64, 17)}
    for name, (C, S, n_own) in exp.items():
        w = synth.get(name)
        assert -(-w.keep // w.cluster) == C
        assert -(-C // w.fanout) == S
        owners = {oracle.owner_layer(l, w.share_period, w.share_start) for l in range(w.n_layers)}
        assert len(owners) == n_own


def test_hierarchy_ratios_match_table3():
    # Table 3 (20% overall): level-1 keep ratio x level-2 keep ratio of the surviving clusters = 0.2
    for r1, r2 in [(0.9, 0.22), (0.7, 0.28), (0.5, 0.40), (0.3, 0.67)]:
        assert abs(r1 * r2 - 0.2) < 0.005
    # Our level-2 budget is taken against the kept cache, so with half the coarse clusters kept the
    # fine level keeps 0.2 / 0.5 = 0.4 of its candidates, up to rounding down to whole clusters.
    C, f = 64, 4
    k1 = oracle.level1_keep(C // f, 0.2)
    k2 = oracle.level2_keep(C * 16, 0.2, 16, k1 * f)
    assert k1 * f == C // 2 and 0 <= 0.4 * k1 * f - k2 < 1


# ------------------------------------------------------------------------ static scoring (A2)
def _rand_bits(shape, dtype, seed, scale=1.0):
    return to_bits(rng(seed).standard_normal(shape) * scale, dtype)


def _torch_scores(qw, k, sm, causal):
    """Brute force: dense masked softmax with torch (fp64), column sums over rows and heads."""
    q = torch.from_numpy(qw)  # [G][W][d]
    kk = torch.from_numpy(k)  # [T][d]
    G, W, _ = q.shape
    T = kk.shape[0]
    s = sm * (q @ kk.T)  # [G][W][T]
    if causal:
        pos = torch.arange(T - W, T).view(W, 1)
        s = s.masked_fill(torch.arange(T).view(1, T) > pos, float("-inf"))
    return torch.softmax(s, dim=-1).sum(dim=(0, 1)).numpy()


@pytest.mark.parametrize("dtype", ["fp32", "bf16", "fp16"])
@pytest.mark.parametrize("causal", [True, False])
def test_token_scores_brute_force(dtype, causal):
    G, W, T, d = 3, 5, 17, 8
    qw = _rand_bits((G, W, d), dtype, 1)
    k = _rand_bits((T, d), dtype, 2)
    sm = 0.35
    got = oracle.token_scores(qw, k, dtype, sm, causal)
    ref = _torch_scores(from_bits(qw, dtype), from_bits(k, dtype), float(np.float32(sm)), causal)
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-15)


def test_token_scores_rows_sum_to_one():
    G, W, T, d = 2, 9, 40, 16
    qw = _rand_bits((G, W, d), "bf16", 3, 2.0)
    k = _rand_bits((T, d), "bf16", 4, 2.0)
    got = oracle.token_scores(qw, k, "bf16", 1 / 4, True)
    assert abs(got.sum() - G * W) < 1e-12 * G * W
    assert np.all(got[:T - W + 1] > 0)


def test_token_scores_uniform_keys_closed_form():
    # Identical keys: every causal row is uniform over its prefix, p = 1/(pos+1).
    G, W, T, d = 2, 4, 10, 4
    qw = _rand_bits((G, W, d), "fp32", 5)
    k = np.tile(np.float32([0.5, -1.0, 2.0, 0.25]), (T, 1))
    got = oracle.token_scores(qw, k, "fp32", 0.5, True)
    exp = []
    for j in range(T):
        s = sum(Fraction(1, p + 1) for p in range(T - W, T) if p >= j)
        exp.append(float(G * s))
    np.testing.assert_allclose(got, exp, rtol=1e-13)
    # non-causal: uniform over all T keys
    got_nc = oracle.token_scores(qw, k, "fp32", 0.5, False)
    np.testing.assert_allclose(got_nc, np.full(T, G * W / T), rtol=1e-13)


def test_token_scores_dominant_key_takes_all_mass():
    G, W, T, d = 1, 3, 12, 4
    q = np.float32([1, 0, 0, 0])
    qw = np.tile(q, (G, W, 1)).astype(np.float32)
    k = _rand_bits((T, d), "fp32", 6, 0.1)
    k[2] = np.float32([400, 0, 0, 0])
    got = oracle.token_scores(qw, k, "fp32", 1.0, True)
    assert abs(got[2] - G * W) < 1e-9
    assert got.sum() - got[2] < 1e-9


def test_token_scores_scale_invariance():
    # scaling q by 2 and the softmax scale by 1/2 leaves the scores unchanged (catches a dropped
    # or doubly applied scale)
    G, W, T, d = 2, 3, 9, 4
    qw = _rand_bits((G, W, d), "fp32", 7)
    k = _rand_bits((T, d), "fp32", 8)
    a = oracle.token_scores(qw, k, "fp32", 0.5, True)
    b = oracle.token_scores((qw * 2).astype(np.float32), k, "fp32", 0.25, True)
    np.testing.assert_allclose(a, b, rtol=1e-13)


def test_row_lse_matches_torch():
    G, W, T, d = 1, 6, 30, 8
    qw = _rand_bits((G, W, d), "bf16", 9)
    k = _rand_bits((T, d), "bf16", 10)
    _, lse = oracle.token_scores(qw, k, "bf16", 0.3, True, with_lse=True)
    qf, kf = from_bits(qw, "bf16"), from_bits(k, "bf16")
    sm = float(np.float32(0.3))
    for t in range(W):
        n = T - W + t + 1
        ref = torch.logsumexp(torch.from_numpy(sm * kf[:n] @ qf[0, t]), 0).item()
        assert abs(lse[0, t] - ref) < 1e-12
        assert abs(oracle.row_lse(qw[0, t], t, W, k, "bf16", 0.3) - ref) < 1e-12


# ------------------------------------------------------------------------ static top-k
def _lexsort_topk(score, k):
    order = np.lexsort((np.arange(len(score)), -np.asarray(score)))
    return order[:k]


def test_static_topk_matches_lexsort_with_ties():
    r = rng(11)
    for T, keep, local in [(50, 20, 5), (64, 64, 8), (33, 10, 0), (40, 6, 10)]:
        score = r.integers(0, 6, T).astype(np.float64)  # many ties
        kept = oracle.static_topk(score, keep, local)
        loc = min(local, keep)
        exp = np.sort(np.concatenate([_lexsort_topk(score[:T - loc], keep - loc), np.arange(T - loc, T)]))
        np.testing.assert_array_equal(kept, exp)
        assert np.all(np.diff(kept) > 0)


def test_static_topk_identity_and_equal_scores():
    np.testing.assert_array_equal(oracle.static_topk(np.ones(16), 16, 4), np.arange(16))
    # all equal: lowest indices first, plus the recent window
    np.testing.assert_array_equal(oracle.static_topk(np.zeros(20), 6, 2), [0, 1, 2, 3, 18, 19])


# ------------------------------------------------------------------------ clusters (A3, A4)
def test_cluster_bounds_match_numpy_with_partial_tail():
    k = _rand_bits((37, 8), "bf16", 12)
    kf = from_bits(k, "bf16")
    for first, count in [(0, 16), (16, 16), (32, 16)]:
        rmax, rmin = oracle.cluster_bounds(k, "bf16", first, count)
        np.testing.assert_array_equal(rmax, kf[first:first + count].max(0))
        np.testing.assert_array_equal(rmin, kf[first:first + count].min(0))


def test_centroid_fp32_rounding_and_alpha_limits():
    r = rng(13)
    vals = from_bits(to_bits(r.standard_normal((500, 2)) * 10, "bf16"), "bf16")
    for a in (0.6, 0.3, 0.9):
        a32 = np.float32(a)
        b32 = np.float32(1) - a32
        for rmax, rmin in vals:
            exp = np.float32(a32 * np.float32(rmax)) + np.float32(b32 * np.float32(rmin))
            assert np.float32(oracle.centroid(rmax, rmin, a)) == np.float32(exp)
    for rmax, rmin in vals[:50]:
        assert oracle.centroid(rmax, rmin, 1.0) == np.float32(rmax)  # alpha = 1 -> r^max
        assert oracle.centroid(rmax, rmin, 0.0) == np.float32(rmin)  # alpha = 0 -> r^min


def test_super_bounds_equal_member_bounds():
    L, B, H, Ts, d, s, f = 1, 1, 2, 80, 8, 8, 3     # C = 10, S = 4 with a tail of 1
    k = _rand_bits((L, B, H, Ts, d), "fp16", 14)
    cent, scent = oracle.build_clusters(k, "fp16", cluster=s, fanout=f, alpha=1.0)
    kf = from_bits(k, "fp16")
    C = 10
    assert cent.shape[3] == C and scent.shape[3] == 4
    for h in range(H):
        cmax = np.stack([kf[0, 0, h, c * s:(c + 1) * s].max(0) for c in range(C)])
        np.testing.assert_array_equal(cent[0, 0, h], cmax.astype(np.float32))
        for sc in range(4):
            np.testing.assert_array_equal(scent[0, 0, h, sc], cmax[sc * f:(sc + 1) * f].max(0).astype(np.float32))


def test_linear_score_below_mp_bound_above_true_max():
    # Eq. 2 and the linearisation: for alpha in [0,1], sum q_i (a r^max + (1-a) r^min) <=
    # sum max(q_i r^max, q_i r^min) >= max_k q.k
    r = rng(15)
    for trial in range(50):
        d, s = 16, 8
        kf = from_bits(to_bits(r.standard_normal((s, d)) * 3, "bf16"), "bf16")
        q = to_bits(r.standard_normal((1, d)), "bf16")
        qf = from_bits(q, "bf16")[0]
        rmax, rmin = kf.max(0), kf.min(0)
        cent = np.float32([oracle.centroid(a, b, 0.6) for a, b in zip(rmax, rmin)])
        lin = oracle.cluster_scores(q, cent[None], "bf16")[0]
        mp = oracle.mp_bound(qf, rmax, rmin)
        true_max = (kf @ qf).max()
        tol = 1e-6 * np.abs(qf) @ np.maximum(np.abs(rmax), np.abs(rmin))
        assert lin <= mp + tol
        assert mp >= true_max - 1e-12


def test_unit_cluster_score_is_dot_product():
    # s = 1, alpha = 1: the representative is the key itself, the score is q.k (exact in fp64)
    r = rng(16)
    k = to_bits(r.standard_normal((20, 8)), "bf16")
    q = to_bits(r.standard_normal((2, 8)), "bf16")
    cent = np.float32([[oracle.centroid(x, x, 1.0) for x in row] for row in from_bits(k, "bf16")])
    got = oracle.cluster_scores(q, cent, "bf16")
    exp = from_bits(k, "bf16") @ from_bits(q, "bf16").sum(0)
    np.testing.assert_array_equal(got, exp)


def test_cluster_mean_matches_exact_sum():
    # the average representative: fp64 sum of the exact key values / count (math.fsum is exact)
    import math
    k = _rand_bits((37, 8), "bf16", 21)
    kf = from_bits(k, "bf16")
    for first, count in [(0, 16), (16, 16), (32, 16)]:
        got = oracle.cluster_mean(k, "bf16", first, count)
        rows = kf[first:first + count]
        exp = np.array([math.fsum(rows[:, i]) / len(rows) for i in range(8)])
        np.testing.assert_array_equal(got, exp)


@pytest.mark.parametrize("similarity", ["linear", "maxprod", "mean"])
def test_representatives_of_each_similarity(similarity):
    # linear: alpha r^max + (1-alpha) r^min rounded as in Eq. "sim"; max-product: the two bound rows
    # (Eq. 2); average: the fp32-rounded mean -- for clusters and for super-clusters (all tokens)
    L, B, H, Ts, d, s, f = 1, 1, 2, 80, 8, 8, 3     # C = 10, S = 4 with a tail of 1
    k = _rand_bits((L, B, H, Ts, d), "fp16", 22)
    kf = from_bits(k, "fp16")
    cent, scent = oracle.build_clusters(k, "fp16", cluster=s, fanout=f, alpha=0.6, similarity=similarity)
    for h in range(H):
        for rep, blocks in ((cent[0, 0, h], [(c * s, s) for c in range(10)]),
                            (scent[0, 0, h], [(u * f * s, f * s) for u in range(4)])):
            for j, (first, count) in enumerate(blocks):
                rows = kf[0, 0, h, first:first + count]
                if similarity == "maxprod":
                    np.testing.assert_array_equal(rep[j, 0], rows.max(0).astype(np.float32))
                    np.testing.assert_array_equal(rep[j, 1], rows.min(0).astype(np.float32))
                elif similarity == "mean":
                    np.testing.assert_array_equal(rep[j], (rows.sum(0) / len(rows)).astype(np.float32))
                else:
                    exp = [oracle.centroid(a, b, 0.6) for a, b in zip(rows.max(0), rows.min(0))]
                    np.testing.assert_array_equal(rep[j], np.float32(exp))


def test_maxprod_score_bounds_true_max_and_every_linear_score():
    # Eq. 2: sum_i max(q_i r^max_i, q_i r^min_i) >= max_k q.k, and >= the linear score for every
    # alpha in [0, 1]; summed over the group's heads
    r = rng(23)
    for trial in range(40):
        G, d, s = 2, 16, 8
        k = to_bits(r.standard_normal((s, d)) * 3, "bf16")
        kf = from_bits(k, "bf16")
        q = to_bits(r.standard_normal((G, d)), "bf16")
        qf = from_bits(q, "bf16")
        rep = np.stack([kf.max(0), kf.min(0)]).astype(np.float32)
        mp = oracle.cluster_scores(q, rep[None], "bf16", "maxprod")[0]
        brute = sum((kf @ qf[g]).max() for g in range(G))
        assert mp >= brute - 1e-12
        for a in (0.0, 0.3, 0.6, 1.0):
            lin = sum(np.sum(np.maximum(qf[g] * rep[0], qf[g] * rep[1])) for g in range(G))
            assert abs(mp - lin) <= 1e-12 * max(1.0, abs(lin))  # the bound itself, by numpy
            cen = qf.sum(0) @ (a * rep[0].astype(np.float64) + (1 - a) * rep[1].astype(np.float64))
            assert cen <= mp + 1e-9


def test_single_token_clusters_score_the_dot_product_in_every_mode():
    # s = 1: r^max = r^min = mean = k, so every representative scores q.k exactly (alpha = 1 for
    # the linear form, whose fp32 products are exact then)
    r = rng(24)
    k = to_bits(r.standard_normal((1, 1, 1, 20, 8)), "bf16")
    q = to_bits(r.standard_normal((2, 8)), "bf16")
    exp = from_bits(k, "bf16")[0, 0, 0] @ from_bits(q, "bf16").sum(0)
    for sim in ("linear", "maxprod", "mean"):
        cent, _ = oracle.build_clusters(k, "bf16", cluster=1, fanout=4, alpha=1.0, similarity=sim)
        got = oracle.cluster_scores(q, cent[0, 0, 0], "bf16", sim)
        np.testing.assert_array_equal(got, exp)


def test_maxprod_equals_alpha_one_linear_for_nonnegative_queries():
    # with q >= 0 every max picks q_i r^max_i: the bound is the alpha = 1 linear score, term by term
    r = rng(25)
    k = to_bits(r.standard_normal((1, 1, 1, 64, 16)), "bf16")
    q = to_bits(np.abs(r.standard_normal((3, 16))), "bf16")
    lin, _ = oracle.build_clusters(k, "bf16", cluster=8, fanout=2, alpha=1.0)
    mp, _ = oracle.build_clusters(k, "bf16", cluster=8, fanout=2, similarity="maxprod")
    np.testing.assert_array_equal(oracle.cluster_scores(q, lin[0, 0, 0], "bf16"),
                                  oracle.cluster_scores(q, mp[0, 0, 0], "bf16", "maxprod"))


def test_average_dilutes_a_single_important_token():
    # the paper's argument against the average (Sec. 3.3 opening; appendix comparison): a cluster
    # holding one key aligned with q among opposed keys ranks below a uniformly mild cluster under
    # the average, but above it under the max-product bound and the alpha = 0.6 linear form, which
    # follow the true maximum dot product
    d, s = 8, 16
    q = np.zeros((1, d)); q[0, 0] = 1.0
    a = np.full((s, d), 0.0); a[:, 0] = -1.0; a[0, 0] = 8.0       # one key with q.k = 8, the rest -1
    b = np.full((s, d), 0.0); b[:, 0] = 1.0                         # every key q.k = 1
    k = to_bits(np.concatenate([a, b])[None, None, None], "fp32")
    qb = to_bits(q, "fp32")
    true_max = [8.0, 1.0]
    for sim, winner in (("maxprod", 0), ("linear", 0), ("mean", 1)):
        cent, _ = oracle.build_clusters(k, "fp32", cluster=s, fanout=2, alpha=0.6, similarity=sim)
        sc = oracle.cluster_scores(qb, cent[0, 0, 0], "fp32", sim)
        assert int(np.argmax(sc)) == winner, (sim, sc)
    assert int(np.argmax(true_max)) == 0


# ------------------------------------------------------------------------ selection (A5-A7)
def test_topk_matches_lexsort():
    r = rng(17)
    s = r.integers(0, 4, 30).astype(np.float64)
    np.testing.assert_array_equal(oracle.topk(s, 12), _lexsort_topk(s, 12))


def _select_case(seed, L=6, B=1, Hq=4, Hkv=2, Ts=200, d=16, s=8, f=4, dtype="bf16", similarity="linear"):
    r = rng(seed)
    k = to_bits(r.standard_normal((L, B, Hkv, Ts, d)), dtype)
    q = to_bits(r.standard_normal((L, B, Hq, d)), dtype)
    cent, scent = oracle.build_clusters(k, dtype, cluster=s, fanout=f, similarity=similarity)
    return k, q, cent, scent


@pytest.mark.parametrize("similarity", ["linear", "maxprod", "mean"])
def test_full_budget_selects_every_cluster(similarity):
    k, q, cent, scent = _select_case(18, Ts=200, s=8, f=4, similarity=similarity)  # C = 25, S = 7 (tail 1)
    sel, _ = oracle.select_clusters(q, cent, scent, "bf16", Ts=200, cluster=8, fanout=4, k_super=7,
                                    k_clusters=25, similarity=similarity)
    assert np.all(sel == np.arange(25))


@pytest.mark.parametrize("similarity", ["maxprod", "mean"])
def test_hierarchical_selection_of_other_similarities_matches_independent_ranking(similarity):
    # the two levels rank by the mode's score recomputed here with numpy from the key values
    Ts, s, f, ks, kc, G, C = 200, 8, 4, 3, 5, 2, 25
    k, q, cent, scent = _select_case(26, Ts=Ts, s=s, f=f, similarity=similarity)
    sel, score = oracle.select_clusters(q, cent, scent, "bf16", Ts=Ts, cluster=s, fanout=f, k_super=ks,
                                        k_clusters=kc, similarity=similarity)
    qf, kf = from_bits(q, "bf16"), from_bits(k, "bf16")

    def sc(qg, rows):  # rows [n_tok][d] of one representative
        if similarity == "mean":
            return qg.sum(0) @ (rows.sum(0) / len(rows)).astype(np.float32).astype(np.float64)
        return sum(np.sum(np.maximum(qh * rows.max(0), qh * rows.min(0))) for qh in qg)

    for l in range(q.shape[0]):
        for h in range(2):
            qg = qf[l, 0, h * G:(h + 1) * G]
            kh = kf[l, 0, h]
            s1 = np.array([sc(qg, kh[u * f * s:(u + 1) * f * s]) for u in range(7)])
            sup = np.sort(_lexsort_topk(s1, ks))
            cand = np.array([c for x in sup for c in range(x * f, min(C, (x + 1) * f))])
            s2 = np.array([sc(qg, kh[c * s:(c + 1) * s]) for c in cand])
            exp = np.sort(cand[_lexsort_topk(s2, kc)])
            np.testing.assert_array_equal(sel[l, 0, h], exp)
            np.testing.assert_allclose(score[l, 0, h], s2[np.searchsorted(cand, exp)], rtol=1e-12)


def test_hierarchical_selection_matches_independent_ranking():
    Ts, s, f, ks, kc = 200, 8, 4, 3, 5
    k, q, cent, scent = _select_case(19, Ts=Ts, s=s, f=f)
    sel, score = oracle.select_clusters(q, cent, scent, "bf16", Ts=Ts, cluster=s, fanout=f, k_super=ks,
                                        k_clusters=kc)
    G = 2
    qf = from_bits(q, "bf16")
    C = 25
    for l in range(q.shape[0]):
        for h in range(2):
            qs = qf[l, 0, h * G:(h + 1) * G].sum(0)
            s1 = scent[l, 0, h].astype(np.float64) @ qs
            sup = np.sort(_lexsort_topk(s1, ks))
            cand = np.array([c for x in sup for c in range(x * f, min(C, (x + 1) * f))])
            s2 = cent[l, 0, h, cand].astype(np.float64) @ qs
            exp = np.sort(cand[_lexsort_topk(s2, kc)])
            np.testing.assert_array_equal(sel[l, 0, h], exp)
            np.testing.assert_allclose(score[l, 0, h], cent[l, 0, h, exp].astype(np.float64) @ qs, rtol=1e-12)


def test_index_sharing_copies_owner_selection():
    Ts, s, f = 200, 8, 4
    k, q, cent, scent = _select_case(20, L=8, Ts=Ts, s=s, f=f)
    kw = dict(Ts=Ts, cluster=s, fanout=f, k_super=3, k_clusters=4)
    shared, _ = oracle.select_clusters(q, cent, scent, "bf16", share_period=2, **kw)
    alone, _ = oracle.select_clusters(q, cent, scent, "bf16", share_period=1, **kw)
    for l in range(8):
        o = oracle.owner_layer(l, 2, 2)
        np.testing.assert_array_equal(shared[l], alone[o])
    # owners outside the block: the caller's selection is kept
    prev = np.full((3, 1, 2, 4), 7, np.int32)
    sel, _ = oracle.select_clusters(q[3:6], cent[3:6], scent[3:6], "bf16", layer0=3, share_period=2,
                                    sel_in=prev, **kw)
    assert np.all(sel[0] == 7)                      # layer 3's owner is layer 2
    np.testing.assert_array_equal(sel[1], alone[4])  # layer 4 owns
    np.testing.assert_array_equal(sel[2], alone[4])  # layer 5 follows layer 4


# ------------------------------------------------------------------------ grouped query heads
def _head_scores(qh, rep, similarity):
    """numpy score of one query head [d] against representatives [n][R][d] (or [n][d])."""
    rep = rep.astype(np.float64)
    if similarity == "maxprod":
        return np.maximum(qh * rep[:, 0], qh * rep[:, 1]).sum(-1)
    return rep @ qh


@pytest.mark.parametrize("similarity", ["linear", "maxprod", "mean"])
def test_group_max_score_is_the_largest_head_score(similarity):
    r = rng(41)
    G, d, n = 4, 16, 9
    q = to_bits(r.standard_normal((G, d)), "fp16")
    R = oracle.rep_rows(similarity)
    rep = r.standard_normal((n, R, d) if R > 1 else (n, d)).astype(np.float32)
    qf = from_bits(q, "fp16")
    per_head = np.stack([_head_scores(qf[g], rep, similarity) for g in range(G)])
    np.testing.assert_allclose(oracle.cluster_scores(q, rep, "fp16", similarity, group="max"), per_head.max(0),
                               rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(oracle.cluster_scores(q, rep, "fp16", similarity, group="sum"), per_head.sum(0),
                               rtol=1e-12, atol=1e-12)
    # one head: the two rules coincide
    np.testing.assert_array_equal(oracle.cluster_scores(q[:1], rep, "fp16", similarity, group="max"),
                                  oracle.cluster_scores(q[:1], rep, "fp16", similarity, group="sum"))


def _two_level(s1_fn, s2_fn, S, C, f, ks, kc):
    """Two-level selection by independent numpy ranking: s1_fn() -> [S], s2_fn(cand) -> [len(cand)]."""
    s1 = s1_fn()
    sup = np.sort(_lexsort_topk(s1, ks))
    cand = np.array([c for x in sup for c in range(x * f, min(C, (x + 1) * f))])
    s2 = s2_fn(cand)
    return np.sort(cand[_lexsort_topk(s2, kc)])


@pytest.mark.parametrize("similarity", ["linear", "maxprod"])
@pytest.mark.parametrize("group", ["max", "head"])
def test_grouped_selection_matches_independent_ranking(similarity, group):
    Ts, s, f, ks, kc, G, C, S = 200, 8, 4, 3, 5, 2, 25, 7
    k, q, cent, scent = _select_case(42, Ts=Ts, s=s, f=f, similarity=similarity)
    sel, _ = oracle.select_clusters(q, cent, scent, "bf16", Ts=Ts, cluster=s, fanout=f, k_super=ks, k_clusters=kc,
                                    similarity=similarity, group=group)
    qf = from_bits(q, "bf16")
    L, Hkv = q.shape[0], 2
    assert sel.shape == ((L, 1, 2 * G, kc) if group == "head" else (L, 1, Hkv, kc))
    for l in range(L):
        for h in range(sel.shape[2]):
            kvh = h // G if group == "head" else h
            heads = [h] if group == "head" else list(range(h * G, (h + 1) * G))

            def score(rep):
                return np.max([_head_scores(qf[l, 0, g], rep, similarity) for g in heads], axis=0)

            exp = _two_level(lambda: score(scent[l, 0, kvh]), lambda cand: score(cent[l, 0, kvh, cand]), S, C, f,
                             ks, kc)
            np.testing.assert_array_equal(sel[l, 0, h], exp)


def test_single_head_groups_select_alike_in_every_rule():
    Ts, s, f = 200, 8, 4
    r = rng(43)
    k = to_bits(r.standard_normal((3, 2, 3, Ts, 16)), "fp16")
    q = to_bits(r.standard_normal((3, 2, 3, 16)), "fp16")
    cent, scent = oracle.build_clusters(k, "fp16", cluster=s, fanout=f)
    kw = dict(Ts=Ts, cluster=s, fanout=f, k_super=4, k_clusters=6)
    ref, _ = oracle.select_clusters(q, cent, scent, "fp16", group="sum", **kw)
    for group in ("max", "head"):
        got, _ = oracle.select_clusters(q, cent, scent, "fp16", group=group, **kw)
        np.testing.assert_array_equal(got, ref)


def test_per_head_selection_is_shared_across_layers():
    Ts, s, f = 200, 8, 4
    k, q, cent, scent = _select_case(44, L=8, Ts=Ts, s=s, f=f)
    kw = dict(Ts=Ts, cluster=s, fanout=f, k_super=3, k_clusters=4, group="head")
    shared, _ = oracle.select_clusters(q, cent, scent, "bf16", share_period=2, **kw)
    alone, _ = oracle.select_clusters(q, cent, scent, "bf16", share_period=1, **kw)
    for l in range(8):
        np.testing.assert_array_equal(shared[l], alone[oracle.owner_layer(l, 2, 2)])


def test_per_head_sparse_attention_uses_each_heads_clusters():
    L, B, Hq, Hkv, Ts, d, s = 1, 2, 4, 2, 40, 8, 8   # C = 5
    r = rng(45)
    k = to_bits(r.standard_normal((L, B, Hkv, Ts, d)), "bf16")
    v = to_bits(r.standard_normal((L, B, Hkv, Ts, d)), "bf16")
    q = to_bits(r.standard_normal((L, B, Hq, d)), "bf16")
    sel = np.array([[[[0, 3], [1, 4], [2, 3], [0, 1]], [[1, 2], [3, 4], [0, 4], [2, 3]]]], np.int32)
    out, _ = oracle.sparse_decode_attn(q, k, v, sel, "bf16", cluster=s, sm_scale=0.35)
    qf, kf, vf = (from_bits(x, "bf16") for x in (q, k, v))
    for b in range(B):
        for h in range(Hq):
            rows = [t for c in sel[0, b, h] for t in range(c * s, (c + 1) * s)]
            ref = _sdpa(qf[0, b, h], kf[0, b, h // 2, rows], vf[0, b, h // 2, rows], float(np.float32(0.35)))
            np.testing.assert_allclose(out[0, b, h], ref, rtol=1e-12, atol=1e-13)


# ------------------------------------------------------------------------ commonality (Sec. 3, Obs. 3)
def test_commonality_worked_cases():
    idx = np.array([[[1, 2]], [[2, 3]], [[3, 4]]], np.int32)  # layers {1,2}, {2,3}, {3,4}
    assert oracle.commonality(idx, 1)[0] == 0.5   # (1 + 1) / (2 * 2)
    assert oracle.commonality(idx, 2)[0] == 0.0   # empty triple intersection
    assert oracle.commonality(idx, 0)[0] == 1.0   # every set with itself
    same = np.tile(np.array([5, 1, 9], np.int32), (6, 2, 1))
    assert np.all(oracle.commonality(same, 4) == 1.0)
    disjoint = np.arange(5 * 3, dtype=np.int32).reshape(5, 1, 3)
    assert oracle.commonality(disjoint, 1)[0] == 0.0


def test_commonality_matches_set_intersections():
    r = rng(46)
    L, U, k, n = 7, 5, 6, 12
    idx = np.stack([np.stack([r.choice(n, k, replace=False) for _ in range(U)]) for _ in range(L)]).astype(np.int32)
    for m in (1, 2, 3):
        got = oracle.commonality(idx, m)
        for u in range(U):
            tot = sum(len(set.intersection(*[set(idx[i, u].tolist()) for i in range(l, l + m + 1)]))
                      for l in range(L - m))
            assert got[u] == float(Fraction(tot, k * (L - m)))


# ------------------------------------------------------------------------ attention (A9, A12)
def _sdpa(q, k, v, sm):
    """torch scaled_dot_product_attention in fp64 on the CPU: q [d], k/v [n][d]."""
    out = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q)[None, None, None], torch.from_numpy(k)[None, None],
        torch.from_numpy(v)[None, None], scale=sm)
    return out[0, 0, 0].numpy()


@pytest.mark.parametrize("dtype", ["fp32", "fp16", "bf16"])
def test_full_budget_sparse_equals_dense_equals_sdpa(dtype):
    L, B, Hq, Hkv, Ts, d, s = 2, 1, 4, 2, 40, 8, 8   # C = 5
    r = rng(21)
    k = to_bits(r.standard_normal((L, B, Hkv, Ts, d)), dtype)
    v = to_bits(r.standard_normal((L, B, Hkv, Ts, d)), dtype)
    q = to_bits(r.standard_normal((L, B, Hq, d)), dtype)
    sm = 1 / np.sqrt(d)
    sel = np.tile(np.arange(5, dtype=np.int32), (L, B, Hkv, 1))
    sp, lse_s = oracle.sparse_decode_attn(q, k, v, sel, dtype, cluster=s, sm_scale=sm)
    dn, lse_d = oracle.dense_decode_attn(q, k, v, dtype, sm_scale=sm)
    np.testing.assert_allclose(sp, dn, rtol=1e-13, atol=1e-14)
    np.testing.assert_allclose(lse_s, lse_d, rtol=1e-13)
    sm32 = float(np.float32(sm))
    qf, kf, vf = (from_bits(x, dtype) for x in (q, k, v))
    for l in range(L):
        for h in range(Hq):
            ref = _sdpa(qf[l, 0, h], kf[l, 0, h // 2], vf[l, 0, h // 2], sm32)
            np.testing.assert_allclose(dn[l, 0, h], ref, rtol=1e-12, atol=1e-13)
            lref = torch.logsumexp(torch.from_numpy(sm32 * kf[l, 0, h // 2] @ qf[l, 0, h]), 0).item()
            assert abs(lse_d[l, 0, h] - lref) < 1e-12


def test_sparse_attention_gathers_selected_clusters_with_partial_tail():
    L, B, Hq, Hkv, Ts, d, s = 1, 1, 2, 1, 45, 8, 8   # C = 6, last cluster has 5 tokens
    r = rng(22)
    k = to_bits(r.standard_normal((L, B, Hkv, Ts, d)), "bf16")
    v = to_bits(r.standard_normal((L, B, Hkv, Ts, d)), "bf16")
    q = to_bits(r.standard_normal((L, B, Hq, d)), "bf16")
    sel = np.array([[[[1, 3, 5]]]], np.int32)
    out, _ = oracle.sparse_decode_attn(q, k, v, sel, "bf16", cluster=s, sm_scale=0.3)
    rows = list(range(8, 16)) + list(range(24, 32)) + list(range(40, 45))
    qf, kf, vf = (from_bits(x, "bf16") for x in (q, k, v))
    for h in range(Hq):
        ref = _sdpa(qf[0, 0, h], kf[0, 0, 0, rows], vf[0, 0, 0, rows], float(np.float32(0.3)))
        np.testing.assert_allclose(out[0, 0, h], ref, rtol=1e-12, atol=1e-13)


# ------------------------------------------------------------------------ decode-time growth (App. A.3)
def test_tail_rows_join_the_attended_tokens():
    # clusters 0 and 2 of Ts = 32 (s = 8) plus a tail of 5 appended rows: softmax attention over
    # exactly those 21 rows, checked against torch's attention on the gathered rows
    L, B, Hq, Hkv, Ts, n_tail, d, s = 1, 2, 4, 2, 32, 5, 8, 8
    r = rng(31)
    k = to_bits(r.standard_normal((L, B, Hkv, Ts + n_tail, d)), "fp16")
    v = to_bits(r.standard_normal((L, B, Hkv, Ts + n_tail, d)), "fp16")
    q = to_bits(r.standard_normal((L, B, Hq, d)), "fp16")
    sel = np.tile(np.array([0, 2], np.int32), (L, B, Hkv, 1))
    out, lse = oracle.sparse_decode_attn(q, k, v, sel, "fp16", cluster=s, sm_scale=0.4, n_tail=n_tail)
    rows = list(range(0, 8)) + list(range(16, 24)) + list(range(32, 37))
    qf, kf, vf = (from_bits(x, "fp16") for x in (q, k, v))
    sm32 = float(np.float32(0.4))
    for b in range(B):
        for h in range(Hq):
            kk, vv = kf[0, b, h // 2, rows], vf[0, b, h // 2, rows]
            np.testing.assert_allclose(out[0, b, h], _sdpa(qf[0, b, h], kk, vv, sm32), rtol=1e-12, atol=1e-13)
            lref = torch.logsumexp(torch.from_numpy(sm32 * kk @ qf[0, b, h]), 0).item()
            assert abs(lse[0, b, h] - lref) < 1e-12


def test_full_budget_with_tail_is_dense_attention_over_the_grown_cache():
    # every cluster selected + the tail = the decode attention of App. A.3 over the whole cache
    L, B, Hq, Hkv, Ts, n_tail, d, s = 2, 1, 2, 2, 24, 7, 8, 8
    r = rng(32)
    k = to_bits(r.standard_normal((L, B, Hkv, Ts + n_tail, d)), "bf16")
    v = to_bits(r.standard_normal((L, B, Hkv, Ts + n_tail, d)), "bf16")
    q = to_bits(r.standard_normal((L, B, Hq, d)), "bf16")
    sel = np.tile(np.arange(3, dtype=np.int32), (L, B, Hkv, 1))
    sp, lse_s = oracle.sparse_decode_attn(q, k, v, sel, "bf16", cluster=s, sm_scale=0.3, n_tail=n_tail)
    dn, lse_d = oracle.dense_decode_attn(q, k, v, "bf16", sm_scale=0.3)
    np.testing.assert_allclose(sp, dn, rtol=1e-13, atol=1e-14)
    np.testing.assert_allclose(lse_s, lse_d, rtol=1e-13)


@pytest.mark.parametrize("s", [1, 4, 16])
def test_append_state_walk(s):
    # from (Ts0, 0), n appends leave Ts0 + n rows, the newest n_tail in [1, s] of them unclustered,
    # and the clustered count a multiple of s above Ts0: clusters are sealed only when full
    Ts0 = 3 * s
    Ts, nt = Ts0, 0
    for n in range(1, 5 * s + 3):
        Ts, nt = oracle.append_state(Ts, nt, s)
        assert Ts + nt == Ts0 + n
        assert 1 <= nt <= s
        assert Ts == Ts0 + s * ((n - 1) // s)
    with pytest.raises(oracle.OracleError):
        oracle.append_state(0, s + 1, s)


def test_sealed_cluster_is_the_cluster_of_the_longer_cache():
    # sealing is the cluster build over the first Ts + s rows: the earlier clusters and the
    # super-clusters that do not hold the new cluster keep their representatives
    L, B, Hkv, d, s, f = 1, 1, 1, 8, 4, 2
    r = rng(33)
    k = to_bits(r.standard_normal((L, B, Hkv, 28, d)), "bf16")
    before = oracle.build_clusters(k[:, :, :, :20], "bf16", cluster=s, fanout=f)   # C = 5, S = 3
    after = oracle.build_clusters(k[:, :, :, :24], "bf16", cluster=s, fanout=f)    # C = 6, S = 3
    np.testing.assert_array_equal(after[0][..., :5, :], before[0])
    np.testing.assert_array_equal(after[1][..., :2, :], before[1][..., :2, :])
    # the grown super-cluster 2 now bounds clusters 4 and 5
    kf = from_bits(k, "bf16")[0, 0, 0, 16:24]
    np.testing.assert_array_equal(after[1][0, 0, 0, 2], [oracle.centroid(hi, lo, 0.6) for hi, lo in
                                                         zip(kf.max(axis=0), kf.min(axis=0))])


# ------------------------------------------------------------------------ whole static eviction
def test_static_evict_identity_sharing_and_gather():
    L, B, Hq, Hkv, T, W, d = 4, 1, 4, 2, 48, 9, 8
    r = rng(23)
    qw = to_bits(r.standard_normal((L, B, Hq, W, d)), "bf16")
    k = to_bits(r.standard_normal((L, B, Hkv, T, d)), "bf16")
    v = to_bits(r.standard_normal((L, B, Hkv, T, d)), "bf16")
    kept, ko, vo = oracle.static_evict(qw, k, v, "bf16", keep=T, local_keep=4, sm_scale=0.35)
    assert np.all(kept == np.arange(T))
    np.testing.assert_array_equal(ko, k)
    kept, ko, vo, sc = oracle.static_evict(qw, k, v, "bf16", keep=20, local_keep=4, sm_scale=0.35,
                                           share_period=2, with_scores=True)
    for l in range(L):
        o = oracle.owner_layer(l, 2, 2)
        np.testing.assert_array_equal(kept[l], kept[o])
        for h in range(Hkv):
            np.testing.assert_array_equal(ko[l, 0, h], k[l, 0, h, kept[l, 0, h]])
            np.testing.assert_array_equal(vo[l, 0, h], v[l, 0, h, kept[l, 0, h]])
    # owner layers: kept = recent window + best scores by lexsort
    for l in (0, 1, 2):
        for h in range(Hkv):
            exp = np.sort(np.concatenate([_lexsort_topk(sc[l, 0, h, :T - 4], 16), np.arange(T - 4, T)]))
            np.testing.assert_array_equal(kept[l, 0, h], exp)
            assert abs(sc[l, 0, h].sum() - 2 * W) < 1e-11


def test_planted_tokens_survive_static_eviction_tiny():
    # Sanity on the tiny workload: sinks and heavy hitters are the most attended tokens.
    w = synth.get("C1")
    qw, k, v = synth.prefill_host(w, 0)
    kept, _, _ = oracle.static_evict(qw[None], k[None], v[None], w.dtype, keep=w.keep,
                                     local_keep=w.local_keep, sm_scale=float(1 / np.sqrt(w.head_dim)))
    sp = synth.spec(w)
    for h in range(w.n_kv_heads):
        ks = set(kept[0, 0, h].tolist())
        assert {0, 1, 2, 3} <= ks
        hh = synth.hh_starts(sp, 0, 0, h)
        assert sum(int(x) in ks for x in hh) >= 14
