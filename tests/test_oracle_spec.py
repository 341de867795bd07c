"""Pins for the oracle's greedy acceptance of drafted tokens, CPU only.

Sec. 4.3: verification keeps the longest prefix of the drafts that the target
model agrees with and corrects the first divergence.  The pins are worked
examples computed by hand (each states its answer and why), the tie rule
(lowest vocabulary index among equal scores), and the defining properties of
the result on random inputs.
"""
import numpy as np
import pytest

import oracle


def logits_with_choices(choices, V, rng=None, fill=0.0):
    """[len(choices)][V] logits whose unique maximum sits at each choice."""
    out = np.full((len(choices), V), fill, np.float32)
    if rng is not None:
        out = rng.standard_normal((len(choices), V)).astype(np.float32)
    for i, c in enumerate(choices):
        out[i, c] = np.abs(out[i]).max() + 1.0
    return out


def test_all_drafts_kept_gives_bonus_token():
    # target choices 3, 1, 4 at the two draft positions and the one after:
    # both drafts (3, 1) agree, so 2 are kept and the bonus token is 4
    logits = logits_with_choices([3, 1, 4], V=6)[None]
    acc, nxt = oracle.accept_greedy(logits, np.array([[3, 1]]))
    assert acc.tolist() == [2] and nxt.tolist() == [4]


def test_first_divergence_is_corrected():
    # target choices 2, 5, 0, 1; drafts 2, 5, 3: the third differs (0 vs 3),
    # so 2 are kept and the correction is the target's 0
    logits = logits_with_choices([2, 5, 0, 1], V=8)[None]
    acc, nxt = oracle.accept_greedy(logits, np.array([[2, 5, 3]]))
    assert acc.tolist() == [2] and nxt.tolist() == [0]


def test_divergence_at_the_first_draft():
    # target choice 7 at position 0, draft 6: nothing kept, correction 7
    logits = logits_with_choices([7, 6], V=9)[None]
    acc, nxt = oracle.accept_greedy(logits, np.array([[6]]))
    assert acc.tolist() == [0] and nxt.tolist() == [7]


def test_ties_take_the_lowest_index():
    # position 0 scores [1, 5, 5, 2]: indices 1 and 2 tie, the choice is 1;
    # a draft of 2 is therefore rejected and corrected to 1
    logits = np.array([[[1, 5, 5, 2], [0, 0, 0, 1]]], np.float32)
    acc, nxt = oracle.accept_greedy(logits, np.array([[2]]))
    assert acc.tolist() == [0] and nxt.tolist() == [1]
    # ... and a draft of 1 is kept, the bonus being position 1's choice 3
    acc, nxt = oracle.accept_greedy(logits, np.array([[1]]))
    assert acc.tolist() == [1] and nxt.tolist() == [3]


def test_negative_scores():
    # all scores negative: the maximum is the least negative (-0.5 at index 2)
    logits = np.array([[[-3.0, -1.0, -0.5, -2.0], [-1.0, -4.0, -9.0, -1.5]]], np.float32)
    acc, nxt = oracle.accept_greedy(logits, np.array([[2]]))
    assert acc.tolist() == [1] and nxt.tolist() == [0]


@pytest.mark.parametrize("seed", range(5))
def test_defining_properties(seed):
    """For every sequence: the first `accepted` drafts equal the target's
    choices, the next draft (if any) does not, and next_token is the target's
    choice at position `accepted`."""
    rng = np.random.default_rng(seed)
    B, k, V = 16, 8, 50
    logits = rng.standard_normal((B, k + 1, V)).astype(np.float32)
    choices = logits.argmax(axis=2)
    # drafts copy the target's choices up to a random divergence point
    drafts = choices[:, :k].copy()
    cut = rng.integers(0, k + 1, B)
    for b in range(B):
        if cut[b] < k:
            drafts[b, cut[b]] = (choices[b, cut[b]] + 1 + rng.integers(0, V - 1)) % V
    acc, nxt = oracle.accept_greedy(logits, drafts)
    assert np.array_equal(acc, cut)
    for b in range(B):
        assert all(drafts[b, i] == choices[b, i] for i in range(acc[b]))
        if acc[b] < k:
            assert drafts[b, acc[b]] != choices[b, acc[b]]
        assert nxt[b] == choices[b, acc[b]]
