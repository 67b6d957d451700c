"""Pins of the CPU oracle against what the paper and the mathematics fix.

None of these compares the oracle with itself: each check is a hand-derived value
(tests/golden), a special case that reduces to a library routine, brute force on
tiny inputs, or an identity that a dropped term, a wrong sign or index, or a
transposed operand would break.
"""
import itertools
import json
import os

import numpy as np
import pytest
import scipy.special
import torch

import oracle as O
from paper_2508_06024_amd import workload as W
from tests._expr import value

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rand_gate(rng, T, d, M, K, scale=1.0):
    x = rng.standard_normal((T, d))
    wl = rng.standard_normal((M, d)) * scale / np.sqrt(d)
    bl = rng.standard_normal(M) * 0.3
    wg = rng.standard_normal((K, d)) * scale / np.sqrt(d)
    bg = rng.standard_normal(K) * 0.3
    return x, wg, bg, wl, bl


def _random_mask(rng, M, n_keep):
    keep = rng.choice(M, n_keep, replace=False)
    return W.mask_words(sorted(keep), M), sorted(int(e) for e in keep)


# ----------------------------------------------------------------------------- gate, Eq. (4)-(7)

def _load(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


@pytest.mark.parametrize("case", _load("gate_hand.json")["cases"], ids=lambda c: c["name"])
def test_gate_hand_examples(case):
    ev = lambda a: np.array([[value(e) for e in row] for row in a]) if isinstance(a[0], list) \
        else np.array([value(e) for e in a])
    x, wl, bl, wg, bg = (ev(case[k]) for k in ("x", "w_local", "b_local", "w_global", "b_global"))
    M = wl.shape[0]
    mask = W.mask_words(case["candidates"], M)
    renorm = case.get("renormalize", True)
    idx, w, g = O.group_gate(x, wg, bg, wl, bl, mask, case["n_groups"], case["top_k"], renorm)
    np.testing.assert_allclose(g[0], [value(e) for e in case["g"]], rtol=0, atol=1e-14)
    assert idx[0].tolist() == case["idx"]
    np.testing.assert_allclose(w[0], [value(e) for e in case["w"]], rtol=0, atol=1e-14)


def test_gate_single_group_is_plain_softmax_gate():
    """K = 1: the fused gate is the traditional single-layer softmax gate over the
    candidates (scipy's softmax)."""
    rng = np.random.default_rng(10)
    x, wg, bg, wl, bl = _rand_gate(rng, 32, 24, 8, 1)
    mask, cand = _random_mask(rng, 8, 5)
    g = O.group_gate_probs(x, wg, bg, wl, bl, mask, 1)
    ref = scipy.special.softmax((x @ wl.T + bl)[:, cand], axis=1)
    np.testing.assert_allclose(g[:, cand], ref, rtol=1e-13, atol=1e-15)
    assert np.all(g[:, [e for e in range(8) if e not in cand]] == 0)


def test_gate_one_expert_per_group_is_global_softmax():
    """K = M: every in-group softmax is over one expert, so g is the global softmax over
    the candidate groups."""
    rng = np.random.default_rng(11)
    x, wg, bg, wl, bl = _rand_gate(rng, 32, 24, 8, 8)
    mask, cand = _random_mask(rng, 8, 6)
    g = O.group_gate_probs(x, wg, bg, wl, bl, mask, 8)
    ref = scipy.special.softmax((x @ wg.T + bg)[:, cand], axis=1)
    np.testing.assert_allclose(g[:, cand], ref, rtol=1e-13, atol=1e-15)


@pytest.mark.parametrize("M,K,keep", [(8, 2, 6), (16, 4, 12), (64, 8, 48), (64, 8, 16), (12, 3, 5)])
def test_gate_distribution_sums_to_one_over_candidates(M, K, keep):
    rng = np.random.default_rng(M * 100 + keep)
    x, wg, bg, wl, bl = _rand_gate(rng, 40, 32, M, K, scale=3.0)
    mask, cand = _random_mask(rng, M, keep)
    g = O.group_gate_probs(x, wg, bg, wl, bl, mask, K)
    np.testing.assert_allclose(g.sum(axis=1), 1.0, rtol=0, atol=1e-13)
    non = [e for e in range(M) if e not in cand]
    assert np.all(g[:, non] == 0)
    assert np.all(g[:, cand] > 0)


def test_gate_zero_weights_reproduce_zipf_popularity():
    """With zero gate weights and biases b_global,k = log(sum of z over group k),
    b_local,i = log z_i - log(sum of z over i's group), Eq. (5)-(7) give g = z."""
    cfg = W.CONFIGS["finegrained"]
    z = W.zipf_popularity(cfg, cfg.seed)
    M, K, Mk = cfg.n_experts, cfg.n_groups, cfg.group_size
    zg = z.reshape(K, Mk).sum(axis=1)
    bg = np.log(zg)
    bl = np.log(z) - np.repeat(np.log(zg), Mk)
    d = 16
    x = np.random.default_rng(0).standard_normal((5, d))
    g = O.group_gate_probs(x, np.zeros((K, d)), bg, np.zeros((M, d)), bl,
                           W.mask_words(range(M), M), K)
    np.testing.assert_allclose(g, np.broadcast_to(z, g.shape), rtol=1e-12, atol=0)
    # Zipf(1.1) over 64 experts: the most popular expert carries about a quarter
    assert abs(z.max() - 0.2497) < 1e-3


def test_gate_scale_invariance_of_in_group_softmax():
    """Adding a constant to every local logit of one group leaves g unchanged, while
    adding it to a group logit moves mass between groups: pins which logits enter
    which softmax."""
    rng = np.random.default_rng(12)
    x, wg, bg, wl, bl = _rand_gate(rng, 8, 10, 8, 2)
    mask = W.mask_words(range(8), 8)
    g0 = O.group_gate_probs(x, wg, bg, wl, bl, mask, 2)
    bl2 = bl.copy()
    bl2[4:] += 5.0
    np.testing.assert_allclose(O.group_gate_probs(x, wg, bg, wl, bl2, mask, 2), g0, rtol=1e-12)
    bg2 = bg.copy()
    bg2[1] += np.log(3.0)
    g2 = O.group_gate_probs(x, wg, bg2, wl, bl, mask, 2)
    # odds of group 1 vs group 0 multiply by exactly 3
    r0 = g0[:, 4:].sum(1) / g0[:, :4].sum(1)
    r2 = g2[:, 4:].sum(1) / g2[:, :4].sum(1)
    np.testing.assert_allclose(r2 / r0, 3.0, rtol=1e-12)


# ----------------------------------------------------------------------------- top-k

def _brute_topk(g_row, cand, k):
    """Exhaustive search over all k-subsets of the candidates: largest sum of g, ties to
    the lexicographically smallest index tuple; then order by (-g, index)."""
    best, best_key = None, None
    for sub in itertools.combinations(sorted(cand), k):
        key = (-sum(g_row[i] for i in sub), sub)
        if best_key is None or key < best_key:
            best, best_key = sub, key
    return sorted(best, key=lambda i: (-g_row[i], i))


@pytest.mark.parametrize("seed", range(40))
def test_topk_matches_exhaustive_search(seed):
    rng = np.random.default_rng(seed)
    M = int(rng.integers(2, 9))
    k = int(rng.integers(1, M + 1))
    keep = int(rng.integers(k, M + 1))
    cand = sorted(rng.choice(M, keep, replace=False).tolist())
    # coarse values make exact ties common
    g = rng.integers(0, 4, M).astype(np.float64) / 4.0
    assert O.topk_select(g, cand, k) == _brute_topk(g, cand, k)
    # counting rule: i is selected iff fewer than k candidates beat it
    sel = set(O.topk_select(g, cand, k))
    for i in cand:
        beat = sum(1 for j in cand if g[j] > g[i] or (g[j] == g[i] and j < i))
        assert (i in sel) == (beat < k)


def test_topk_never_selects_a_non_candidate():
    rng = np.random.default_rng(3)
    for _ in range(50):
        M = 16
        mask, cand = _random_mask(rng, M, 5)
        x, wg, bg, wl, bl = _rand_gate(rng, 6, 8, M, 4, scale=4.0)
        idx, _, _ = O.group_gate(x, wg, bg, wl, bl, mask, 4, 3)
        assert set(idx.ravel().tolist()) <= set(cand)


def test_topk_too_few_candidates_is_an_error():
    rng = np.random.default_rng(4)
    x, wg, bg, wl, bl = _rand_gate(rng, 2, 8, 8, 2)
    with pytest.raises(O.TooFewCandidates):
        O.group_gate(x, wg, bg, wl, bl, W.mask_words([1], 8), 2, 2)


def test_renormalised_weights():
    rng = np.random.default_rng(5)
    x, wg, bg, wl, bl = _rand_gate(rng, 64, 16, 16, 4, scale=2.0)
    mask = W.mask_words(range(16), 16)
    _, w, g = O.group_gate(x, wg, bg, wl, bl, mask, 4, 3)
    np.testing.assert_allclose(w.sum(1), 1.0, rtol=0, atol=4e-16)
    assert np.all(w[:, :-1] >= w[:, 1:])
    _, w1, _ = O.group_gate(x, wg, bg, wl, bl, mask, 4, 1)
    assert np.all(w1 == 1.0)
    idx_raw, w_raw, _ = O.group_gate(x, wg, bg, wl, bl, mask, 4, 3, renormalize=False)
    np.testing.assert_array_equal(w_raw, np.take_along_axis(g, idx_raw.astype(np.int64), 1))


# ----------------------------------------------------------------------------- permutation

def _brute_segments(idx, M):
    """Scan experts in order and, for each, the assignments in order."""
    flat = [int(e) for e in np.asarray(idx).ravel()]
    k = np.asarray(idx).shape[1]
    seg, perm_src, inv = [0], [], [0] * len(flat)
    for e in range(M):
        for a, ea in enumerate(flat):
            if ea == e:
                inv[a] = len(perm_src)
                perm_src.append(a // k)
        seg.append(len(perm_src))
    return seg, perm_src, inv


@pytest.mark.parametrize("T,M,k,keep,skew", [(37, 8, 2, 6, 0.0), (100, 16, 3, 12, 1.1),
                                              (64, 64, 6, 48, 1.1), (5, 4, 4, 4, 0.0),
                                              (1, 8, 1, 3, 0.0)])
def test_permutation_matches_brute_force(T, M, k, keep, skew):
    rng = np.random.default_rng(T + M)
    cand = sorted(rng.choice(M, keep, replace=False).tolist())
    idx, _ = W.gen_routing(T, M, k, cand, seed=T * M, skew=skew)
    seg, perm_src, inv = O.permute(idx, M)
    bseg, bsrc, binv = _brute_segments(idx, M)
    assert seg.tolist() == bseg
    assert perm_src.tolist() == bsrc
    assert inv.tolist() == binv
    assert seg[-1] == T * k
    for e in range(M):
        if e not in cand:
            assert seg[e] == seg[e + 1]


# ----------------------------------------------------------------------------- unequal groups, group pruning

def test_unequal_groups_hand_example():
    c = _load("gate_unequal_hand.json")
    M, K, d = 4, 2, c["d"]
    x = np.ones((1, d))
    z = lambda *shape: np.zeros(shape)
    for top_groups in (0, 1, 2):
        idx, w, g = O.group_gate(x, z(K, d), z(K), z(M, d), z(M), [0b1111], K, c["top_k"],
                                 group_sizes=c["group_sizes"], top_groups=top_groups)
        np.testing.assert_allclose(g[0], [value(v) for v in c["g"]], rtol=1e-15)
        assert idx[0].tolist() == c["idx"]
        np.testing.assert_allclose(w[0], [value(v) for v in c["w"]], rtol=1e-15)


def test_unequal_groups_reduce_to_known_cases():
    rng = np.random.default_rng(40)
    T, d, M, K = 9, 24, 12, 3
    x, wg, bg, wl, bl = _rand_gate(rng, T, d, M, K)
    mask, _ = _random_mask(rng, M, 10)
    # equal sizes given explicitly: the default grouping
    a = O.group_gate_probs(x, wg, bg, wl, bl, mask, K)
    b = O.group_gate_probs(x, wg, bg, wl, bl, mask, K, group_sizes=[4, 4, 4])
    np.testing.assert_array_equal(a, b)
    # one group of all experts: scipy's softmax over the candidates
    g1 = O.group_gate_probs(x, wg[:1], bg[:1], wl, bl, mask, 1, group_sizes=[M])
    cand = O.candidate_set(mask, M)
    ref = scipy.special.softmax(x @ wl[cand].T + bl[cand], axis=1)
    np.testing.assert_allclose(g1[:, cand], ref, rtol=1e-12)
    # sizes (5, 2, 5): each group's g sums to its p_group; in-group odds are exp(logit gaps)
    sizes = [5, 2, 5]
    g = O.group_gate_probs(x, wg, bg, wl, bl, W.mask_words(range(M), M), K, group_sizes=sizes)
    pg = scipy.special.softmax(x @ wg.T + bg, axis=1)
    starts = np.cumsum([0] + sizes)
    for k in range(K):
        np.testing.assert_allclose(g[:, starts[k]:starts[k + 1]].sum(1), pg[:, k], rtol=1e-12)
    l = x @ wl.T + bl
    np.testing.assert_allclose(g[:, 6] / g[:, 5], np.exp(l[:, 6] - l[:, 5]), rtol=1e-12)
    with pytest.raises(ValueError):
        O.group_gate_probs(x, wg, bg, wl, bl, mask, K, group_sizes=[5, 5, 5])


def test_group_pruning_keeps_all_groups_when_g_covers_them():
    rng = np.random.default_rng(41)
    T, d, M, K, k = 20, 16, 16, 4, 3
    x, wg, bg, wl, bl = _rand_gate(rng, T, d, M, K)
    mask, _ = _random_mask(rng, M, 13)
    dense = O.group_gate(x, wg, bg, wl, bl, mask, K, k)
    for G in (K, K + 3):
        pruned = O.group_gate(x, wg, bg, wl, bl, mask, K, k, top_groups=G)
        for a, b in zip(dense, pruned):
            np.testing.assert_array_equal(a, b)


def test_top1_group_is_the_in_group_softmax():
    """top_groups = 1 and a top group with at least k candidates: the selected experts come from
    the group with the largest p_group, and their renormalised weights are the in-group
    softmax's (p_group cancels)."""
    rng = np.random.default_rng(42)
    T, d, M, K, k = 30, 20, 24, 4, 2
    x, wg, bg, wl, bl = _rand_gate(rng, T, d, M, K, scale=3.0)
    mask = W.mask_words(range(M), M)
    idx, w, g = O.group_gate(x, wg, bg, wl, bl, mask, K, k, top_groups=1)
    top = np.argmax(x @ wg.T + bg, axis=1)
    l = x @ wl.T + bl
    for t in range(T):
        members = np.arange(top[t] * 6, top[t] * 6 + 6)
        assert set(idx[t].tolist()) <= set(members.tolist())
        pl = scipy.special.softmax(l[t, members])
        best = members[np.argsort(-pl, kind="stable")[:k]]
        assert idx[t].tolist() == best.tolist()
        np.testing.assert_allclose(w[t], pl[best - top[t] * 6] / pl[best - top[t] * 6].sum(), rtol=1e-12)
        assert np.count_nonzero(g[t]) == 6
        # p_group stays the softmax over all groups: the kept group's g sums to its p_group
        np.testing.assert_allclose(g[t].sum(), scipy.special.softmax(x[t] @ wg.T + bg)[top[t]], rtol=1e-12)


def test_group_pruning_extends_until_k_candidates():
    """The kept groups are taken in p_group order until they hold k candidates; ties between
    groups go to the lower group index."""
    rng = np.random.default_rng(43)
    T, d, M, K, k = 25, 12, 16, 8, 5
    x, wg, bg, wl, bl = _rand_gate(rng, T, d, M, K)
    wg[5] = wg[2]
    bg[5] = bg[2]  # groups 2 and 5 always tie
    keep = [0, 2, 3, 4, 5, 9, 10, 11, 12, 14]  # candidates per group of 2: 1 2 2 0 1 2 1 1
    mask = W.mask_words(keep, M)
    idx, w, g = O.group_gate(x, wg, bg, wl, bl, mask, K, k, top_groups=2)
    gl = x @ wg.T + bg
    cand_g = {kk: [i for i in keep if i // 2 == kk] for kk in range(K)}
    active = [kk for kk in range(K) if cand_g[kk]]
    for t in range(T):
        order = sorted(active, key=lambda kk: (-gl[t, kk], kk))
        kept, held = [], 0
        for kk in order:
            if len(kept) >= 2 and held >= k:
                break
            kept.append(kk)
            held += len(cand_g[kk])
        assert {int(i) // 2 for i in idx[t]} <= set(kept)
        assert {int(i) // 2 for i in np.nonzero(g[t])[0]} == set(kept)
        if 2 in kept and 5 in kept:
            continue
        assert not (5 in kept and 2 not in kept), "tie between groups 2 and 5 must keep group 2 first"


# ----------------------------------------------------------------------------- experts, Eq. (1)

def test_silu_pins():
    z = np.linspace(-30, 30, 301)
    # silu(z) - silu(-z) = z(sigma(z) + sigma(-z)) = z
    np.testing.assert_allclose(O.silu(z) - O.silu(-z), z, rtol=0, atol=1e-12)
    assert O.silu(np.array(0.0)) == 0.0
    np.testing.assert_allclose(O.silu(z), torch.nn.functional.silu(torch.tensor(z)).numpy(),
                               rtol=1e-14, atol=1e-300)


def test_swiglu_gate_and_up_order():
    c = _load("swiglu_hand.json")
    y = O.swiglu_expert(np.array(c["x"]), np.array(c["w_gate_up"][0]), np.array(c["w_down"][0]))
    np.testing.assert_allclose(y[0, 0], value(c["y"]), rtol=1e-14)


def _torch_dense_swiglu(x, wgu, wd):
    H = wd.shape[1]
    xt, g, u, dn = (torch.tensor(a, dtype=torch.float64) for a in (x, wgu[:H], wgu[H:], wd))
    f = torch.nn.functional
    return f.linear(f.silu(f.linear(xt, g)) * f.linear(xt, u), dn).numpy()


def test_one_expert_moe_is_dense_ffn():
    rng = np.random.default_rng(6)
    T, d, H = 23, 16, 40
    x = rng.standard_normal((T, d))
    wgu = rng.standard_normal((1, 2 * H, d)) * 0.3
    wd = rng.standard_normal((1, d, H)) * 0.3
    wg, bg, wl, bl = np.zeros((1, d)), np.zeros(1), rng.standard_normal((1, d)), np.zeros(1)
    idx, w, _ = O.group_gate(x, wg, bg, wl, bl, [1], 1, 1)
    assert np.all(idx == 0) and np.all(w == 1.0)
    y = O.moe_forward(x, idx, w, wgu, wd)
    np.testing.assert_allclose(y, _torch_dense_swiglu(x, wgu[0], wd[0]), rtol=1e-12, atol=1e-12)


def test_identical_experts_equal_dense_ffn_for_any_routing():
    rng = np.random.default_rng(7)
    T, d, H, M, k = 31, 12, 20, 8, 3
    x = rng.standard_normal((T, d))
    one_gu = rng.standard_normal((2 * H, d)) * 0.3
    one_dn = rng.standard_normal((d, H)) * 0.3
    wgu = np.stack([one_gu] * M)
    wd = np.stack([one_dn] * M)
    idx, w = W.gen_routing(T, M, k, range(M), seed=1, skew=1.1)
    w = w.astype(np.float64)
    w /= w.sum(1, keepdims=True)
    y = O.moe_forward(x, idx, w, wgu, wd)
    np.testing.assert_allclose(y, _torch_dense_swiglu(x, one_gu, one_dn), rtol=1e-12, atol=1e-12)


def test_combine_matches_per_token_sum():
    """Permutation + expert segments + combine against the definition token by token."""
    rng = np.random.default_rng(8)
    T, d, H, M, k = 29, 8, 12, 6, 2
    x = rng.standard_normal((T, d))
    wgu = rng.standard_normal((M, 2 * H, d)) * 0.4
    wd = rng.standard_normal((M, d, H)) * 0.4
    idx, w = W.gen_routing(T, M, k, [0, 1, 3, 4, 5], seed=2)
    y = O.moe_forward(x, idx, w, wgu, wd)
    for t in range(T):
        ref = sum(float(w[t, j]) * _torch_dense_swiglu(x[t:t + 1], wgu[idx[t, j]], wd[idx[t, j]])[0]
                  for j in range(k))
        np.testing.assert_allclose(y[t], ref, rtol=1e-12, atol=1e-12)


def test_top1_combine_is_a_gather_and_zero_rows_stay_zero():
    rng = np.random.default_rng(9)
    T, d, H, M = 16, 8, 10, 4
    x = rng.standard_normal((T, d))
    x[3] = 0.0
    wgu = rng.standard_normal((M, 2 * H, d))
    wd = rng.standard_normal((M, d, H))
    idx, _ = W.gen_routing(T, M, 1, range(M), seed=3)
    w = np.ones((T, 1))
    y_perm, seg, perm_src, inv = O.expert_outputs(x, idx, wgu, wd)
    y = O.combine(y_perm, inv, w)
    np.testing.assert_array_equal(y, y_perm[inv])
    assert np.all(y[3] == 0.0)


# ----------------------------------------------------------------------------- ReLU experts

def test_relu_expert_hand_example():
    c = _load("relu_hand.json")
    y = O.relu_expert(np.array(c["x"]), np.array(c["w_in"][0]), np.array(c["w_down"][0]))
    np.testing.assert_array_equal(y[0], np.array(c["y"]))
    # the same through the MoE path: one expert, top-1, weight 1
    y2 = O.moe_forward(np.array(c["x"]), np.zeros((1, 1), np.int32), np.ones((1, 1)),
                       np.array(c["w_in"]), np.array(c["w_down"]), activation="relu")
    np.testing.assert_array_equal(y2[0], np.array(c["y"]))


def test_one_expert_relu_moe_is_dense_relu_ffn():
    """A 1-expert ReLU MoE (gate forced by a one-expert candidate set) equals a dense
    ReLU FFN built from torch's linear and relu."""
    rng = np.random.default_rng(16)
    T, d, H = 19, 24, 56
    x = rng.standard_normal((T, d))
    w_in = rng.standard_normal((1, H, d)) * 0.3
    wd = rng.standard_normal((1, d, H)) * 0.3
    wg, bg, wl, bl = np.zeros((1, d)), np.zeros(1), rng.standard_normal((1, d)), np.zeros(1)
    idx, w, _ = O.group_gate(x, wg, bg, wl, bl, [1], 1, 1)
    y = O.moe_forward(x, idx, w, w_in, wd, activation="relu")
    f = torch.nn.functional
    xt, wi, wdn = (torch.tensor(a, dtype=torch.float64) for a in (x, w_in[0], wd[0]))
    np.testing.assert_allclose(y, f.linear(f.relu(f.linear(xt, wi)), wdn).numpy(), rtol=1e-12, atol=1e-12)


def test_relu_expert_identities():
    """relu(z) - relu(-z) = z, so E(x) - E(-x) = W_down W_in x; and E(a x) = a E(x) for
    a > 0 (positive homogeneity of a bias-free ReLU network)."""
    rng = np.random.default_rng(17)
    T, d, H = 13, 10, 30
    x = rng.standard_normal((T, d))
    w_in = rng.standard_normal((H, d))
    wd = rng.standard_normal((d, H))
    e_pos, e_neg = O.relu_expert(x, w_in, wd), O.relu_expert(-x, w_in, wd)
    np.testing.assert_allclose(e_pos - e_neg, x @ (wd @ w_in).T, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(O.relu_expert(2.5 * x, w_in, wd), 2.5 * e_pos, rtol=1e-13, atol=1e-13)
    # a row whose every hidden unit is negative gives a zero output
    x1 = -np.abs(rng.standard_normal((1, d)))
    np.testing.assert_array_equal(O.relu_expert(x1, np.abs(w_in), wd), np.zeros((1, d)))


def test_relu_top1_moe_matches_per_token_definition():
    """Top-1 routing over ReLU experts, token by token against Eq. (1) with one term."""
    rng = np.random.default_rng(18)
    T, d, H, M = 27, 8, 16, 5
    x = rng.standard_normal((T, d))
    w_in = rng.standard_normal((M, H, d)) * 0.5
    wd = rng.standard_normal((M, d, H)) * 0.5
    idx, w = W.gen_routing(T, M, 1, [0, 2, 3, 4], seed=4)
    y = O.moe_forward(x, idx, w, w_in, wd, activation="relu")
    for t in range(T):
        e = int(idx[t, 0])
        h = np.maximum(w_in[e] @ x[t], 0.0)
        np.testing.assert_allclose(y[t], float(w[t, 0]) * (wd[e] @ h), rtol=1e-12, atol=1e-12)


def test_switch_workloads_follow_the_parameter_selection():
    """4 x 256 tokens, top-1, 8/16/32/64 experts, candidate set at most 40% of them."""
    for n in W.SWITCH_ORDER:
        cfg = W.CONFIGS[n]
        assert cfg.n_tokens == 4 * 256 and cfg.top_k == 1 and cfg.codec_slices == 4
        assert cfg.n_experts in (8, 16, 32, 64) and cfg.activation == "relu"
        x, mask = W.gen_call(cfg)
        kept = W.mask_members(mask, cfg.n_experts)
        assert len(kept) == int(0.4 * cfg.n_experts) and len(kept) <= 0.4 * cfg.n_experts
        assert cfg.w_in_rows == cfg.ffn_hidden


# ----------------------------------------------------------------------------- codec

def test_codec_full_rank_round_trip():
    """A rank-d orthonormal codec (U, V square orthogonal) reconstructs X exactly
    (up to rounding): the tiny workload's shape, T=64 tokens, d=128."""
    cfg = W.CONFIGS["tiny"]
    x = W.to_f64(W.gen_call(cfg)[0], cfg.dtype)
    u = W.haar_orthonormal(5, (1,), cfg.n_tokens, cfg.n_tokens)
    v = W.haar_orthonormal(5, (2,), cfg.d_model, cfg.d_model)
    z = O.lowrank_encode(x, u, v)
    xh = O.lowrank_decode(z, u, v)
    np.testing.assert_allclose(xh, x, rtol=0, atol=1e-14)


def test_codec_projection_identities():
    rng = np.random.default_rng(13)
    T, d, rh, rw = 48, 80, 12, 20
    x = rng.standard_normal((T, d))
    u = W.haar_orthonormal(1, (1,), T, rh)
    v = W.haar_orthonormal(1, (2,), d, rw)
    z = O.lowrank_encode(x, u, v)
    assert z.shape == (rh, rw)
    xh = O.lowrank_decode(z, u, v)
    # decode(encode(.)) is the orthogonal projection P_U X P_V: idempotent
    np.testing.assert_allclose(O.lowrank_decode(O.lowrank_encode(xh, u, v), u, v), xh, atol=1e-12)
    # Pythagoras: ||Z|| = ||X_hat|| and ||X||^2 = ||X_hat||^2 + ||X - X_hat||^2
    np.testing.assert_allclose(np.linalg.norm(z), np.linalg.norm(xh), rtol=1e-12)
    np.testing.assert_allclose(np.sum(x * x), np.sum(xh * xh) + np.sum((x - xh) ** 2), rtol=1e-12)
    # U = I reduces to the one-sided product X V
    zi = O.lowrank_encode(x, np.eye(T), v)
    np.testing.assert_allclose(zi, x @ v, rtol=1e-13, atol=1e-13)


def test_layer_codes_each_slice_separately():
    """c slices: every slice s of X is projected on its own, X_hat[s] = U U^T X[s] V V^T,
    and a full-rank codec round-trips every slice."""
    rng = np.random.default_rng(15)
    c, h, d, M, H = 3, 8, 6, 4, 8
    x = rng.standard_normal((c * h, d))
    u = W.haar_orthonormal(2, (1,), h, 5)
    v = W.haar_orthonormal(2, (2,), d, 4)
    w_in = rng.standard_normal((M, H, d))
    wd = rng.standard_normal((M, d, H))
    wl = rng.standard_normal((M, d))
    out = O.layer(x, [0b1111], np.zeros((2, d)), np.zeros(2), wl, np.zeros(M), w_in, wd,
                  u, v, u, v, 2, 1, activation="relu", codec_slices=c)
    assert out["z"].shape == (c, 5, 4)
    for s in range(c):
        xs = x[s * h:(s + 1) * h]
        np.testing.assert_allclose(out["z"][s], u.T @ xs @ v, rtol=1e-12, atol=1e-12)
        np.testing.assert_allclose(out["x_hat"][s * h:(s + 1) * h], u @ u.T @ xs @ v @ v.T, atol=1e-12)
    uf, vf = W.haar_orthonormal(3, (1,), h, h), W.haar_orthonormal(3, (2,), d, d)
    full = O.layer(x, [0b1111], np.zeros((2, d)), np.zeros(2), wl, np.zeros(M), w_in, wd,
                   uf, vf, uf, vf, 2, 1, activation="relu", codec_slices=c)
    np.testing.assert_allclose(full["x_hat"], x, atol=1e-13)


def test_codec_eckart_young():
    """With U, V the top singular vectors of X, the codec error is the tail of the
    singular values (numpy's SVD)."""
    rng = np.random.default_rng(14)
    T, d, r = 40, 70, 9
    x = rng.standard_normal((T, d)) @ np.diag(np.linspace(3, 0.1, d))
    uu, s, vt = np.linalg.svd(x, full_matrices=False)
    z = O.lowrank_encode(x, uu[:, :r], vt[:r].T)
    np.testing.assert_allclose(np.diag(z), s[:r], rtol=1e-12)
    xh = O.lowrank_decode(z, uu[:, :r], vt[:r].T)
    np.testing.assert_allclose(np.sum((x - xh) ** 2), np.sum(s[r:] ** 2), rtol=1e-10)


# ----------------------------------------------------------------------------- layer

def test_layer_routes_on_x_and_runs_experts_on_reconstruction():
    cfg = W.CONFIGS["tiny"]
    inp = W.gen_layer(cfg)
    f = inp.f64
    out = O.layer(f("x"), inp.mask, f("w_global"), inp.b_global, f("w_local"), inp.b_local,
                  f("w_gate_up"), f("w_down"), f("u"), f("v"), f("u"), f("v"),
                  cfg.n_groups, cfg.top_k)
    idx, w, _ = O.group_gate(f("x"), f("w_global"), inp.b_global, f("w_local"), inp.b_local,
                             inp.mask, cfg.n_groups, cfg.top_k)
    np.testing.assert_array_equal(out["idx"], idx)
    xh = f("u") @ (f("u").T @ f("x") @ f("v")) @ f("v").T
    np.testing.assert_allclose(out["x_hat"], xh, atol=1e-14)
    assert out["y"].shape == (cfg.n_tokens, cfg.d_model)
    assert not set(out["idx"].ravel().tolist()) & set(cfg.masked_out)
    # Eq. 1 token by token on the reconstruction X_hat = U U^T X V V^T, with the routing the
    # gate took on X: y[t] = sum_j w[t, j] E_{idx[t, j]}(x_hat[t]), each expert a dense SwiGLU
    # FFN evaluated by torch (not the oracle's permuted expert path)
    gu, dn = f("w_gate_up"), f("w_down")
    for t in range(cfg.n_tokens):
        ref = sum(float(w[t, j]) * _torch_dense_swiglu(xh[t:t + 1], gu[idx[t, j]], dn[idx[t, j]])[0]
                  for j in range(cfg.top_k))
        np.testing.assert_allclose(out["y"][t], ref, rtol=1e-12, atol=1e-15)
    # the experts see X_hat, not X: below full rank (16 of 64 tokens, 16 of 128 features) the
    # two outputs differ by far more than rounding
    y_on_x = np.stack([sum(float(w[t, j]) * _torch_dense_swiglu(f("x")[t:t + 1], gu[idx[t, j]], dn[idx[t, j]])[0]
                           for j in range(cfg.top_k)) for t in range(cfg.n_tokens)])
    assert np.max(np.abs(out["y"] - y_on_x)) > 0.1 * np.max(np.abs(y_on_x))


# ----------------------------------------------------------------------------- codec fitting (Eq. 8, lambda = 0)

def _spectrum_matrix(rng, h, w, sv):
    """X = P diag(sv) Q^T with Haar P [h][n], Q [w][n]."""
    p = W.haar_orthonormal(int(rng.integers(1 << 30)), (1,), h, len(sv))
    q = W.haar_orthonormal(int(rng.integers(1 << 30)), (2,), w, len(sv))
    return (p * np.asarray(sv)) @ q.T


def test_fit_one_slice_reaches_eckart_young():
    rng = np.random.default_rng(50)
    h, w, r = 40, 56, 7
    sv = np.linspace(5.0, 0.2, 30)
    x = _spectrum_matrix(rng, h, w, sv)
    u, v = O.codec_fit_hosvd(x[None], r, r)
    xh = O.lowrank_decode(O.lowrank_encode(x, u, v), u, v)
    np.testing.assert_allclose(np.sum((x - xh) ** 2), np.sum(sv[r:] ** 2), rtol=1e-10)
    np.testing.assert_allclose(u.T @ u, np.eye(r), atol=1e-12)
    np.testing.assert_allclose(v.T @ v, np.eye(r), atol=1e-12)


def test_fit_recovers_low_rank_slices_exactly():
    """Slices sharing row and column spaces of rank <= r are reconstructed exactly."""
    rng = np.random.default_rng(51)
    c, h, w, r = 3, 30, 44, 6
    p = W.haar_orthonormal(3, (1,), h, 4)
    q = W.haar_orthonormal(3, (2,), w, 5)
    xs = np.stack([p @ rng.standard_normal((4, 5)) @ q.T for _ in range(c)])
    for u, v in (O.codec_fit_hosvd(xs, r, r),
                 O.codec_fit_subspace(xs, rng.standard_normal((h, r)), rng.standard_normal((w, r)), 2)):
        for s in range(c):
            xh = O.lowrank_decode(O.lowrank_encode(xs[s], u, v), u, v)
            np.testing.assert_allclose(xh, xs[s], atol=1e-10)


def test_subspace_iteration_converges_to_the_hosvd_subspace():
    rng = np.random.default_rng(52)
    c, h, w, r = 2, 48, 64, 5
    sv = np.concatenate([np.linspace(10, 6, r), np.linspace(1.0, 0.1, 20)])  # gap after r
    # slices sharing their singular vectors (per-slice scales): the Gram sums keep the gap
    p = W.haar_orthonormal(7, (1,), h, sv.size)
    q = W.haar_orthonormal(7, (2,), w, sv.size)
    xs = np.stack([(p * (sv * rng.uniform(0.9, 1.1, sv.size))) @ q.T for _ in range(c)])
    u0, v0 = O.codec_fit_hosvd(xs, r, r)
    u, v = O.codec_fit_subspace(xs, rng.standard_normal((h, r)), rng.standard_normal((w, r)), 12)
    np.testing.assert_allclose(u @ u.T, u0 @ u0.T, atol=1e-9)
    np.testing.assert_allclose(v @ v.T, v0 @ v0.T, atol=1e-9)
    np.testing.assert_allclose(u.T @ u, np.eye(r), atol=1e-12)


@pytest.mark.parametrize("iters", [0, 1, 3])
def test_subspace_iteration_takes_the_asked_power_steps(iters):
    """Closed form: one slice X = diag(sqrt(a)) has A = B = diag(a), and from a start block of
    ones (rank 1) the i-th iterate is A^i 1 / ||A^i 1||: U = V = a^iters normalised."""
    a = np.array([4.0, 3.0, 2.0, 1.5, 1.0, 0.5])
    x = np.diag(np.sqrt(a))
    ones = np.ones((a.size, 1))
    u, v = O.codec_fit_subspace(x[None], ones, ones, iters)
    want = a ** iters / np.linalg.norm(a ** iters)
    np.testing.assert_allclose(u[:, 0], want, rtol=1e-12)
    np.testing.assert_allclose(v[:, 0], want, rtol=1e-12)


def test_orthonormal_basis_is_the_positive_diagonal_qr():
    rng = np.random.default_rng(53)
    y = rng.standard_normal((30, 6))
    q = O.orthonormal_basis(y)
    r = q.T @ y
    np.testing.assert_allclose(np.tril(r, -1), 0.0, atol=1e-12)
    assert np.all(np.diag(r) > 0)
    # Gram-Schmidt by hand on the first two columns
    e1 = y[:, 0] / np.linalg.norm(y[:, 0])
    t = y[:, 1] - (e1 @ y[:, 1]) * e1
    np.testing.assert_allclose(q[:, 0], e1, atol=1e-12)
    np.testing.assert_allclose(q[:, 1], t / np.linalg.norm(t), atol=1e-12)
