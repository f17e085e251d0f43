"""Pins of the oracle's AdaKV allocation (App. B: BACON on the AdaKV backbone
keeps its head-wise budgets and changes only the score within each head).

The allocation read here: each KV head keeps its top f = floor(alpha K)
positions by the backbone score A; the layer's other H (K - f) slots go to the
highest A over the union of every head's remaining positions (ties: score
desc, head asc, position asc); K_h = f + the head's share.  Each pin reaches
the budgets by a route that shares nothing with the oracle's code: worked
examples by hand, the plain union top-(H K) at alpha = 0, and a threshold
walk over all entries (K_h = max(f, n_h) at the union's boundary entry).
"""
import numpy as np
import pytest

from paper_2606_14782_amd import inputs


def _walk(A, K, alpha):
    """Budgets by walking every entry in union order (score desc, head asc,
    position asc) and stopping where the heads' counts beyond their floors
    reach H (K - f); a head's budget is then max(f, its count)."""
    H, n = A.shape
    if K >= n:
        return np.full(H, K)
    f = int(np.floor(alpha * K))
    R = H * (K - f)
    hs, ps = np.meshgrid(np.arange(H), np.arange(n), indexing="ij")
    order = np.lexsort((ps.ravel(), hs.ravel(), -A.ravel()))
    cnt = np.zeros(H, np.int64)
    for e in order:
        cnt[hs.ravel()[e]] += 1
        if np.maximum(cnt - f, 0).sum() == R:
            break
    return np.maximum(cnt, f)


def test_worked_examples(oracle):
    # f = 1: each head's best is reserved; the union of the rest gives its
    # two best (0.8 in head 0, 0.25 in head 1) one slot each
    A = np.array([[0.9, 0.8, 0.1, 0.05], [0.3, 0.2, 0.25, 0.1]])
    assert oracle.adaptive_budgets(A, 2, 0.5).tolist() == [2, 2]
    # head 1's remaining scores are all below head 0's: both union slots go to head 0
    A = np.array([[0.9, 0.8, 0.1, 0.05], [0.3, 0.02, 0.01, 0.0]])
    assert oracle.adaptive_budgets(A, 2, 0.5).tolist() == [3, 1]
    # no floor: the top H K = 2 of the union are head 0's two tied 0.5's
    # (lower head first), and head 1 gets none
    A = np.array([[0.5, 0.5, 0.1], [0.5, 0.5, 0.1]])
    assert oracle.adaptive_budgets(A, 1, 0.0).tolist() == [2, 0]
    # f = 1 reserves position 0 of each head; the union's two 0.5's at
    # position 1 go one to each head
    assert oracle.adaptive_budgets(A, 2, 0.5).tolist() == [2, 2]
    # with a third tied 0.5 per head, the union's top two are head 0's
    # positions 1 and 2 (lower head first)
    A = np.array([[0.5, 0.5, 0.5, 0.1], [0.5, 0.5, 0.5, 0.1]])
    assert oracle.adaptive_budgets(A, 2, 0.5).tolist() == [3, 1]
    # K >= n: every head keeps all its candidates
    assert oracle.adaptive_budgets(A, 4, 0.2).tolist() == [4, 4]


def test_full_floor_is_uniform(oracle):
    rng = np.random.default_rng(1)
    A = rng.random((6, 50))
    for K in (1, 7, 49):
        assert oracle.adaptive_budgets(A, K, 1.0).tolist() == [K] * 6


@pytest.mark.parametrize("seed", range(6))
def test_no_floor_is_the_union_top(oracle, seed):
    """alpha = 0: K_h is the number of head h's entries among the plain top
    H K of all heads' scores (a full lexsort)."""
    rng = np.random.default_rng(seed)
    H, n, K = 4, 40, int(rng.integers(1, 39))
    A = np.round(rng.random((H, n)), 1)       # many ties across heads
    hs, ps = np.meshgrid(np.arange(H), np.arange(n), indexing="ij")
    top = np.lexsort((ps.ravel(), hs.ravel(), -A.ravel()))[:H * K]
    want = np.bincount(hs.ravel()[top], minlength=H)
    assert oracle.adaptive_budgets(A, K, 0.0).tolist() == want.tolist()


@pytest.mark.parametrize("seed", range(10))
def test_threshold_walk_and_invariants(oracle, seed):
    rng = np.random.default_rng(100 + seed)
    H, n = int(rng.integers(1, 7)), int(rng.integers(2, 60))
    K = int(rng.integers(1, n + 3))
    alpha = float(rng.choice([0.0, 0.1, 0.2, 0.5, 0.9, 1.0]))
    levels = int(rng.choice([3, 10, 1000]))
    A = rng.integers(0, levels, size=(H, n)) / levels
    got = oracle.adaptive_budgets(A, K, alpha)
    assert got.tolist() == _walk(A, K, alpha).tolist()
    if K < n:
        f = int(np.floor(alpha * K))
        assert got.sum() == H * K and got.min() >= f and got.max() <= n


def test_heads_permute_with_their_scores(oracle):
    rng = np.random.default_rng(7)
    A = rng.random((5, 30))                   # distinct scores: no cross-head ties
    perm = rng.permutation(5)
    a = oracle.adaptive_budgets(A, 6, 0.2)
    b = oracle.adaptive_budgets(A[perm], 6, 0.2)
    assert b.tolist() == a[perm].tolist()


def test_layer_on_the_adakv_backbone(oracle):
    """Prompt.layer_adaptive: alpha = 1 is the uniform layer; otherwise the
    budgets are the allocation of the pooled B over each sequence's
    candidates, and each head keeps its K_{b,h} best of S."""
    wl = inputs.Workload("pin", 3, 4, 2, 16, 4, 3, "fp32", (70, 45), (8, 6),
                         ((5, 40), (5, 30)), 1, 99)
    xs = [inputs.layer_inputs(wl, l) for l in range(wl.num_layers)]
    u = oracle.Prompt.for_workload(wl)
    a1 = oracle.Prompt.for_workload(wl)
    a2 = oracle.Prompt.for_workload(wl)
    for l, x in enumerate(xs):
        ru = u.layer(l, x["q_win"], x["k"])
        r1 = a1.layer_adaptive(l, x["q_win"], x["k"], 1.0)
        assert np.array_equal(r1["idx"], ru["idx"]) and np.array_equal(r1["S"], ru["S"])
        r2 = a2.layer_adaptive(l, x["q_win"], x["k"], 0.2)
        for b, (s0, s1) in enumerate(zip(wl.cu_seqlens[:-1], wl.cu_seqlens[1:])):
            nc = (s1 - s0) - wl.window
            A = np.stack([_box(r2["B"][h, s0:s0 + nc], wl.pool_kernel)
                          for h in range(wl.num_kv_heads)])
            K = wl.budgets[b]
            assert r2["alloc_budgets"][b].tolist() == _walk(A, K, 0.2).tolist()
            for h in range(wl.num_kv_heads):
                kh = int(r2["alloc_budgets"][b, h])
                S = r2["S_pool"][h, s0:s0 + nc]
                best = np.lexsort((np.arange(nc), -S))[:min(kh, nc)]
                assert np.array_equal(a2.idx_of(r2, b, h), np.sort(best))


def _box(x, k):
    n, h, ones = len(x), k // 2, np.ones(k)
    num = np.convolve(x, ones, mode="full")[h:h + n]
    den = np.convolve(np.ones(n), ones, mode="full")[h:h + n]
    return num / den


def test_zero_budget_head(oracle):
    """A head the allocation leaves without slots keeps nothing (lambda 0:
    its scale-matching set is empty); the other heads select as with their
    own budgets everywhere."""
    wl = inputs.Workload("pin", 2, 4, 2, 16, 4, 3, "fp32", (70, 45), (8, 6),
                         ((5, 40), (5, 30)), 1, 98)
    hb = np.array([[0, 5], [3, 0]], np.int32)
    p = oracle.Prompt.for_workload(wl)
    u = oracle.Prompt.for_workload(wl.with_(budgets=(5, 3)))
    for l in range(wl.num_layers):
        x = inputs.layer_inputs(wl, l)
        r = p.layer(l, x["q_win"], x["k"], head_budgets=hb)
        ru = u.layer(l, x["q_win"], x["k"])
        assert r["n_kept"][0, 0] == 0 and r["n_kept"][1, 1] == 0
        assert r["lambda"][0, 0] == 0.0 and r["m_count"][0, 0] == 0
        assert np.array_equal(p.idx_of(r, 0, 1), u.idx_of(ru, 0, 1))
        assert np.array_equal(p.idx_of(r, 1, 0), u.idx_of(ru, 1, 0))
