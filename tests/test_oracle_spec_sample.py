"""Pins for the oracle's acceptance of sampled drafts (Sec. 4.3 with the
speculative-sampling rule), CPU only.  What the pins rest on, other than the
oracle itself:

  - the rule's defining property: whatever the draft distribution, every
    emitted token is distributed as the target's distribution at its
    position, and the first draft is kept with probability
    sum_x min(p(x), q(x)); checked by chi-square and binomial tests over many
    sequences whose drafts are drawn from q here with numpy;
  - hand-worked draws at the exact boundaries of the inverse-CDF sampling;
  - the degenerate cases the readings fix (tokens outside the vocabulary,
    NaN and out-of-range weights, all-zero residuals).
"""
import numpy as np
import pytest
from scipy import stats

import oracle


def emitted(acc, nxt, drafts, pos):
    """Token emitted at position pos (None where the sequence stopped before)."""
    return np.where(acc > pos, drafts[:, pos] if pos < drafts.shape[1] else -1,
                    np.where(acc == pos, nxt, -1))


@pytest.mark.parametrize("seed", [1, 2])
def test_emitted_tokens_follow_the_target(seed):
    rng = np.random.default_rng(seed)
    B, k, V = 200_000, 2, 6
    p_rows = rng.dirichlet(np.ones(V) * 0.8, size=k + 1).astype(np.float32)
    q_rows = rng.dirichlet(np.ones(V) * 0.8, size=k).astype(np.float32)
    p = np.broadcast_to(p_rows, (B, k + 1, V))
    q = np.broadcast_to(q_rows, (B, k, V))
    drafts = np.stack([rng.choice(V, size=B, p=q_rows[i] / q_rows[i].sum()) for i in range(k)], axis=1)
    u = rng.random((B, k + 1), dtype=np.float32)
    acc, nxt = oracle.accept_sample(p, q, drafts, u)
    assert acc.min() >= 0 and acc.max() <= k
    # first draft kept with probability sum_x min(p, q)
    keep = float(np.minimum(p_rows[0], q_rows[0]).sum())
    n_keep = int((acc >= 1).sum())
    assert stats.binomtest(n_keep, B, keep).pvalue > 1e-4
    for pos in range(k + 1):
        tok = emitted(acc, nxt, drafts, pos)
        tok = tok[tok >= 0]
        want = p_rows[pos].astype(np.float64)
        want /= want.sum()
        counts = np.bincount(tok, minlength=V)
        assert stats.chisquare(counts, want * len(tok)).pvalue > 1e-4, (pos, counts, want * len(tok))


def test_draws_at_the_boundaries_by_hand():
    """Bonus draw over p_k = [0.25, 0.5, 0.25, 0] (drafts all kept: u = 0):
    S = 2^40 and t = floor(S U / 2^32), so U = u 2^32 gives t = u S; the token
    is the first whose inclusive prefix (2^38, 3 2^38, 2^40, 2^40) exceeds t."""
    k, V = 1, 4
    p = np.array([[[0.5, 0.5, 0, 0], [0.25, 0.5, 0.25, 0.0]]], np.float32)
    q = np.array([[[0.5, 0.5, 0, 0]]], np.float32)
    cases = [(0.0, 0), (0.2499999, 0), (0.25, 1), (0.5, 1), (0.7499999, 1), (0.75, 2),
             (0.9999999, 2), (1.0, 2), (7.0, 2), (-1.0, 0), (float("nan"), 0)]
    for uf, want in cases:
        acc, nxt = oracle.accept_sample(p, q, np.array([[1]]), np.array([[0.0, uf]], np.float32))
        assert acc[0] == 1 and nxt[0] == want, (uf, nxt[0], want)


def test_rejection_and_residual_by_hand():
    """p_0 = [0.1, 0.9], q_0 = [0.6, 0.4], draft 0: kept iff 0.6 u <= 0.1
    (u <= 1/6); on rejection the residual is [0, 0.5], so the next token is 1
    whatever the draw.  Draft 1 (0.4 u <= 0.9) is always kept for u < 1."""
    p = np.array([[[0.1, 0.9], [0.3, 0.7]]], np.float32)
    q = np.array([[[0.6, 0.4]]], np.float32)
    for u0, want_acc in [(0.0, 1), (0.16, 1), (0.17, 0), (0.5, 0), (0.99, 0)]:
        for uf in (0.0, 0.5, 0.99):
            acc, nxt = oracle.accept_sample(p, q, np.array([[0]]), np.array([[u0, uf]], np.float32))
            assert acc[0] == want_acc
            if want_acc == 0:
                assert nxt[0] == 1
            else:   # bonus from p_1 = [0.3, 0.7]
                assert nxt[0] == (0 if uf < 0.3 else 1)
    for u0 in (0.0, 0.5, 0.99):
        acc, _ = oracle.accept_sample(p, q, np.array([[1]]), np.array([[u0, 0.5]], np.float32))
        assert acc[0] == 1


def test_degenerate_cases():
    V = 3
    p = np.array([[[0.2, 0.3, 0.5], [0.0, 1.0, 0.0]]], np.float32)
    q = np.array([[[0.2, 0.3, 0.5]]], np.float32)
    # tokens outside the vocabulary are never kept; p = q leaves no residual,
    # so the draw falls back to p_0
    for bad in (-1, V, 1 << 30):
        acc, nxt = oracle.accept_sample(p, q, np.array([[bad]]), np.array([[0.0, 0.6]], np.float32))
        assert acc[0] == 0 and nxt[0] == 2   # prefix 0.2, 0.5, 1.0 > 0.6 at token 2
    # an all-zero row: next_token -1
    z = np.zeros((1, 2, V), np.float32)
    zq = np.array([[[0.5, 0.5, 0.0]]], np.float32)
    acc, nxt = oracle.accept_sample(z, zq, np.array([[0]]), np.array([[0.5, 0.5]], np.float32))
    assert acc[0] == 0 and nxt[0] == -1
    # NaN, negative and above-one weights count as 0, 0 and 1
    pn = np.array([[[0.5, 0.5, 0.0], [np.nan, -3.0, 5.0]]], np.float32)
    qn = np.array([[[0.5, 0.5, 0.0]]], np.float32)
    acc, nxt = oracle.accept_sample(pn, qn, np.array([[0]]), np.array([[0.0, 0.0]], np.float32))
    assert acc[0] == 1 and nxt[0] == 2


def test_longest_prefix_and_independence_of_later_drafts():
    """Drafts after the first one not kept change nothing."""
    rng = np.random.default_rng(4)
    B, k, V = 500, 5, 50
    p = rng.dirichlet(np.ones(V), size=(B, k + 1)).astype(np.float32)
    q = rng.dirichlet(np.ones(V), size=(B, k)).astype(np.float32)
    drafts = rng.integers(0, V, size=(B, k))
    u = rng.random((B, k + 1), dtype=np.float32)
    acc, nxt = oracle.accept_sample(p, q, drafts, u)
    d2 = drafts.copy()
    for b in range(B):
        d2[b, acc[b] + 1:] = rng.integers(0, V, size=k - acc[b] - 1) if acc[b] + 1 < k else d2[b, acc[b] + 1:]
    acc2, nxt2 = oracle.accept_sample(p, q, d2, u)
    assert np.array_equal(acc, acc2) and np.array_equal(nxt, nxt2)
