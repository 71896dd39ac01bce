"""Prefix-tree packing of a rollout's model calls (Sec. 3.2.1): pins of the oracle, and parity of
the library's host implementation (rlk_tree_pack, through the C ABI) with it."""
import numpy as np
import pytest

import oracle as O


def path_tokens(r, p):
    out = []
    while p >= 0:
        out.append(int(r["token"][p]))
        p = int(r["parent"][p])
    return out[::-1]


def random_calls(rng, n_calls=8, vocab=6):
    """A rollout's calls: mostly extensions of the latest history, some retries (same context,
    new or identical response) and some restarts from a shortened context (compaction)."""
    calls = []
    hist = list(rng.integers(0, vocab, size=rng.integers(2, 6)))   # the task prompt
    ctx = hist
    for _ in range(n_calls):
        kind = rng.random()
        if calls and kind < 0.2:          # retry of the previous call (maybe the same response)
            x, y = calls[-1][0], (calls[-1][1] if rng.random() < 0.5 else list(rng.integers(0, vocab, 3)))
        elif calls and kind < 0.35:       # compaction: a shortened context plus a summary
            keep = rng.integers(1, max(2, len(ctx)))
            x = ctx[:keep] + list(rng.integers(0, vocab, size=rng.integers(1, 4)))
            y = list(rng.integers(0, vocab, size=rng.integers(1, 5)))
        else:                             # extension: tool output appended to the latest history
            x = ctx + list(rng.integers(0, vocab, size=rng.integers(0, 4)))
            y = list(rng.integers(0, vocab, size=rng.integers(1, 5)))
        calls.append((list(map(int, x)), list(map(int, y))))
        ctx = list(map(int, x)) + list(map(int, y))
    return calls


# ------------------------------------------------------------------- oracle pins
def test_linear_rollout_is_one_path():
    calls = [([1, 2, 3], [4, 5]), ([1, 2, 3, 4, 5, 9], [6]), ([1, 2, 3, 4, 5, 9, 6, 7], [8, 8])]
    r = O.tree_pack([calls])
    assert r["token"].tolist() == [1, 2, 3, 4, 5, 9, 6, 7, 8, 8]
    assert r["parent"].tolist() == list(range(-1, 9))
    assert r["row_mask"].tolist() == [0, 0, 1, 1, 0, 1, 0, 1, 1]       # rows predict tokens 1..9
    assert r["row_target"].tolist() == [2, 3, 4, 5, 9, 6, 7, 8, 8]
    assert r["leaves"].tolist() == [1]


def test_every_call_is_spelled_by_its_root_path_and_shared_prefixes_are_stored_once():
    rng = np.random.default_rng(5)
    for _ in range(30):
        calls = random_calls(rng)
        r = O.tree_pack([calls])
        # each call's x + y is the token path from the root to some position
        paths = {tuple(path_tokens(r, p)) for p in range(len(r["token"]))}
        for x, y in calls:
            assert tuple(x + y) in paths
        # no two positions share (parent, token, mask) -> every shared prefix is stored once
        keys = {}
        for p in range(len(r["token"])):
            m = -1 if r["parent"][p] < 0 else None
            keys.setdefault((int(r["parent"][p]), int(r["token"][p])), []).append(p)
        dup = [v for v in keys.values() if len(v) > 1]
        for v in dup:   # allowed only when the nodes differ in trainability (harness vs model token)
            assert len({path_tokens(r, q)[-1] for q in v}) == 1
        # rows: one per non-root position, src is the parent, depth grows by one
        n_roots = int((r["parent"] < 0).sum())
        assert len(r["row_src"]) == len(r["token"]) - n_roots
        nonroot = np.flatnonzero(r["parent"] >= 0)
        assert np.array_equal(r["row_src"], r["parent"][nonroot])
        assert np.array_equal(r["row_target"], r["token"][nonroot])
        assert np.all(r["depth"][nonroot] == r["depth"][r["parent"][nonroot]] + 1)


def test_duplicate_calls_do_not_change_the_packing():
    rng = np.random.default_rng(6)
    for _ in range(20):
        calls = random_calls(rng)
        dup = []
        for c in calls:
            dup.append(c)
            if rng.random() < 0.4:
                dup.append(c)                 # the proxy recorded the same call twice
        a, b = O.tree_pack([calls]), O.tree_pack([dup])
        for k in a:
            np.testing.assert_array_equal(a[k], b[k], err_msg=k)


def test_fork_shares_the_prefix_once():
    # a compaction restart: the second segment starts from the prompt plus a summary
    calls = [([1, 2], [3, 4]), ([1, 2, 3, 4, 7], [5]), ([1, 2, 9], [6, 6])]
    r = O.tree_pack([calls])
    assert r["leaves"].tolist() == [2]
    assert r["token"].tolist() == [1, 2, 3, 4, 7, 5, 9, 6, 6]
    assert r["parent"].tolist() == [-1, 0, 1, 2, 3, 4, 1, 6, 7]
    # both continuations of the shared "1 2" are predicted from the same hidden state (position 1)
    assert r["row_src"].tolist().count(1) == 2
    assert int(r["row_mask"].sum()) == 5


def test_batch_offsets_concatenate_rollouts():
    rng = np.random.default_rng(7)
    rolls = [random_calls(rng, n_calls=int(rng.integers(1, 6))) for _ in range(5)]
    r = O.tree_pack(rolls)
    for i, calls in enumerate(rolls):
        one = O.tree_pack([calls])
        a, b = r["pos_off"][i], r["pos_off"][i + 1]
        np.testing.assert_array_equal(r["token"][a:b], one["token"])
        shift = lambda v: np.where(v >= 0, v + a, v)
        np.testing.assert_array_equal(r["parent"][a:b], shift(one["parent"]))
        c0, c1 = r["row_cu"][i], r["row_cu"][i + 1]
        np.testing.assert_array_equal(r["row_src"][c0:c1], one["row_src"] + a)


# ------------------------------------------------------------- library parity
def test_library_tree_pack_matches_oracle():
    import paper_2608_16798_amd as rlk

    rng = np.random.default_rng(8)
    for trial in range(25):
        rolls = [random_calls(rng, n_calls=int(rng.integers(0, 12)), vocab=int(rng.integers(2, 9)))
                 for _ in range(int(rng.integers(1, 7)))]
        want = O.tree_pack(rolls)
        got = rlk.tree_pack(rolls)
        for k in want:
            np.testing.assert_array_equal(np.asarray(got[k]), want[k], err_msg=f"{k} (trial {trial})")


def test_library_tree_pack_capacity_and_sizes():
    import paper_2608_16798_amd as rlk

    calls = [[([1, 2, 3], [4, 5]), ([1, 2, 3, 4, 5, 9], [6])]]
    n_pos, n_rows = rlk.tree_pack_sizes(calls)
    assert (n_pos, n_rows) == (7, 6)
    with pytest.raises(rlk.RlkError):
        rlk.tree_pack(calls, cap_pos=6)
