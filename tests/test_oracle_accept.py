"""CPU pins of the oracle's tolerant acceptance (Sec. 3.2, the Top-3 rule):
a hand-worked window, brute force by sorting, top-1 = greedy, and torch's
topk on rows without ties."""
import numpy as np
import pytest
import torch

from oracle import kap_oracle as O


def test_hand_worked_window():
    # row ranks: token 1 (5) is 0, token 3 (5, later index) 1, token 2 (3) 2,
    # token 5 (2) 3, token 0 (1) 4, token 4 (0) 5 -> top-3 = {1, 3, 2}
    row = np.array([1.0, 5.0, 3.0, 5.0, 0.0, 2.0])
    assert [O.token_rank(row, d) for d in range(6)] == [4, 0, 2, 1, 5, 3]
    logits = np.stack([row, row[::-1], row, row])[None]       # window of 4: 3 drafts
    # draft 0 = token 2 (rank 2: accepted); draft 1 = token 1 in the reversed
    # row (values 2,0,5,3,5,1: rank of token 1 is 5: rejected) -> m = 1
    m, carry = O.accept_top_k(logits, np.array([[2, 1, 3]]), 3)
    assert m[0] == 1
    assert carry[0] == 2          # argmax of the reversed row: 5 at index 2 (before index 4)
    m, carry = O.accept_top_k(logits, np.array([[3, 2, 1]]), 3)
    assert m[0] == 3 and carry[0] == 1            # all accepted; carry from the last row
    m, _ = O.accept_top_k(logits, np.array([[7, 2, 1]]), 3)
    assert m[0] == 0                              # out-of-range draft is never accepted


@pytest.mark.parametrize("seed", range(5))
def test_rank_matches_sorting(seed):
    rng = np.random.default_rng(seed)
    row = rng.integers(-3, 4, 200).astype(np.float64)          # many ties
    order = sorted(range(200), key=lambda j: (-row[j], j))
    for d in rng.integers(0, 200, 30):
        assert O.token_rank(row, int(d)) == order.index(int(d))


def test_top1_is_greedy():
    rng = np.random.default_rng(7)
    logits = rng.integers(0, 5, (6, 5, 40)).astype(np.float64)
    drafts = rng.integers(0, 40, (6, 4))
    drafts[:, 0] = np.argmax(logits[:, 0], axis=1)            # first draft always greedy
    m, carry = O.accept_top_k(logits, drafts, 1)
    for b in range(6):
        want = 0
        while want < 4 and drafts[b, want] == np.argmax(logits[b, want]):
            want += 1
        assert m[b] == want and m[b] >= 1
        assert carry[b] == np.argmax(logits[b, want])


def test_matches_torch_topk_without_ties():
    rng = np.random.default_rng(8)
    logits = rng.standard_normal((4, 6, 1000))
    drafts = rng.integers(0, 1000, (4, 5))
    top = torch.topk(torch.from_numpy(logits), 3, dim=-1).indices.numpy()
    drafts[:, :3] = top[:, :3, 1]                             # second-best: accepted
    m, carry = O.accept_top_k(logits, drafts, 3)
    for b in range(4):
        want = 0
        while want < 5 and drafts[b, want] in top[b, want]:
            want += 1
        assert m[b] == want and m[b] >= 3
        assert carry[b] == top[b, want, 0]


def test_planted_tie_break_mistake_is_caught(monkeypatch):
    def no_tie_break(row, d):
        x = np.asarray(row, dtype=np.float64)
        return int(np.sum(x > x[d]))
    monkeypatch.setattr(O, "token_rank", no_tie_break)
    with pytest.raises(AssertionError):
        test_hand_worked_window()
