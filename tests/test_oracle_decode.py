"""Pins for oracle.decode: top-1 rule, acceptance, commit and page allocation."""
import json
import os

import numpy as np
import pytest

from oracle import decode as od
from paper_2609_26638_amd import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _sorted_first(row):
    # independent formulation: sort (value descending, index ascending)
    return sorted(range(len(row)), key=lambda i: (-float(row[i]), i))[0]


def test_top1_tie_and_signed_zero():
    assert od.top1(np.array([1.0, 3.0, 2.0, 3.0])) == 1
    assert od.top1(np.array([-0.0, 0.0, -1.0])) == 0
    assert od.top1(np.array([-1.0, 0.0, -0.0])) == 1
    assert od.top1(np.array([-5.0, -0.0, -3.0, 0.0])) == 1
    with pytest.raises(ValueError):
        od.top1(np.array([0.0, np.nan]))
    with pytest.raises(ValueError):
        od.top1(np.array([0.0, np.inf]))


def test_top1_matches_sort_definition_on_ties():
    x = synth.tied_logits(3, 4, 6, 37).astype(np.float64)
    am = od.top1_rows(x)
    for s in range(4):
        for r in range(6):
            assert am[s, r] == _sorted_first(x[s, r])


def test_top1_planted_logits():
    li = synth.make_logit_inputs(5, 3, 4, 4, 2048, 4.0, 0.5)
    x = synth.bf16_to_f64(li.logits)
    am = od.top1_rows(x)
    np.testing.assert_array_equal(am[:, :4], li.planted)


def test_accept_length_rule():
    a = np.array([4, 5, 6, 7, 8])
    assert od.accept_length(a, np.array([4, 5, 6, 7])) == 4     # full match
    assert od.accept_length(a, np.array([4, 5, 9, 7])) == 2     # first mismatch at j=3
    assert od.accept_length(a, np.array([1, 5, 6, 7])) == 0
    assert od.accept_length(a, np.array([], dtype=int)) == 0     # B=1: nothing to check
    # a later match after a mismatch does not count (longest *prefix*)
    assert od.accept_length(a, np.array([4, 0, 6, 7])) == 1


def test_match_probability_gives_expected_acceptance():
    # drafts copy the verify top-1 w.p. p independently: E[A] = sum_{k=1}^{n} p^k
    S, B, p = 400, 8, 0.8
    li = synth.make_logit_inputs(8, S, B, B, 64, 4.0, p)
    am = od.top1_rows(synth.bf16_to_f64(li.logits))
    A = od.accept(am, li.draft, B)
    expect = sum(p ** k for k in range(1, B))
    assert abs(A.mean() - expect) < 4 * np.sqrt(B * B / S)
    assert A.min() >= 0 and A.max() <= B - 1


def _state_from(d):
    S = len(d["kv_len"])
    max_pages = len(d["page_table"][0])
    st = synth.PagedState(
        kv_len=np.array(d["kv_len"], np.int32),
        page_table=np.array(d["page_table"], np.int32),
        num_pages=np.array(d["num_pages"], np.int32),
        free_stack=np.array(d["free_stack"], np.int32),
        free_top=int(d["free_top"]),
        boundary=np.array(d["boundary"], np.int32),
        draft=np.array(d["draft"], np.int32),
        out_tokens=np.full((S, 16), -1, np.int32),
        out_count=np.zeros(S, np.int32),
        finished=np.zeros(S, np.int32),
        pool_pages=len(d["free_stack"]), max_pages=max_pages)
    return st


def test_commit_golden_example():
    g = json.load(open(os.path.join(GOLDEN, "commit_example.json")))
    st = _state_from(g["before"])
    am = np.array(g["before"]["argmax"], np.int32)
    A = od.accept(am, st.draft, g["n_causal"])
    np.testing.assert_array_equal(A, g["after"]["accept_len"])
    err = od.kv_commit(st, A, am, g["n_causal"], g["n_mask"], eos_id=g["eos_id"],
                       page_size=g["page_size"])
    assert err == 0
    a = g["after"]
    np.testing.assert_array_equal(st.kv_len, a["kv_len"])
    np.testing.assert_array_equal(st.page_table, a["page_table"])
    np.testing.assert_array_equal(st.num_pages, a["num_pages"])
    assert st.free_top == a["free_top"]
    np.testing.assert_array_equal(st.free_stack[:st.free_top], a["free_stack_live"])
    np.testing.assert_array_equal(st.boundary, a["boundary"])
    np.testing.assert_array_equal(st.draft, a["draft"])
    np.testing.assert_array_equal(st.finished, a["finished"])
    for s, toks in enumerate(a["out_tokens"]):
        assert list(st.out_tokens[s, :st.out_count[s]]) == toks


def test_literal_round_commit_hand_example():
    # Two-forward round, B = 2: the verify window is [a0, d_1, d_2] (3 causal
    # rows), kv_len already counts x0, the run is a0, d_1..d_A, a_{A+1} and
    # the pages must cover the next round's [L', L' + B + 2).  Page size 4.
    # seq0: L0 = 5 (kv_len 6), a0 = 40, d = [7, 8], verify top-1 [7, 50, 60]:
    #   a_1 = 7 = d_1, a_2 = 50 != 8 -> A = 1; run [40, 7, 50]; L' = 6 + 3 - 1 = 8;
    #   boundary 50; needs ceil((8 + 4) / 4) = 3 pages, holds 3.
    # seq1: L0 = 2 (kv_len 3), a0 = 41, d = [9, 10], top-1 [9, 10, 61]: A = 2;
    #   run [41, 9, 10, 61]; L' = 3 + 4 - 1 = 6; boundary 61; needs ceil(10 / 4)
    #   = 3, holds 2 -> pops the stack top (page 42) into logical page 2.
    st = _state_from({
        "kv_len": [6, 3], "page_table": [[10, 11, 12, -1], [20, 21, -1, -1]],
        "num_pages": [3, 2], "free_stack": [40, 41, 42, -1], "free_top": 3,
        "boundary": [100, 200], "draft": [[7, 8], [9, 10]]})
    am = np.array([[7, 50, 60], [9, 10, 61]], np.int32)
    A = od.accept(am, st.draft, 3)
    np.testing.assert_array_equal(A, [1, 2])
    err = od.kv_commit(st, A, am, 3, 0, page_size=4, lead=np.array([40, 41]), window=4)
    assert err == 0
    np.testing.assert_array_equal(st.kv_len, [8, 6])
    np.testing.assert_array_equal(st.boundary, [50, 61])
    assert list(st.out_tokens[0, :st.out_count[0]]) == [40, 7, 50]
    assert list(st.out_tokens[1, :st.out_count[1]]) == [41, 9, 10, 61]
    np.testing.assert_array_equal(st.page_table, [[10, 11, 12, -1], [20, 21, 42, -1]])
    np.testing.assert_array_equal(st.num_pages, [3, 3])
    assert st.free_top == 2
    np.testing.assert_array_equal(st.draft, [[7, 8], [9, 10]])   # no mask rows: unchanged


def test_commit_max_new_truncates():
    g = json.load(open(os.path.join(GOLDEN, "commit_example.json")))
    st = _state_from(g["before"])
    am = np.array(g["before"]["argmax"], np.int32)
    A = od.accept(am, st.draft, 2)
    err = od.kv_commit(st, A, am, 2, 2, max_new=1, page_size=4)
    assert err == 0
    assert list(st.out_count) == [1, 1, 1, 1]
    assert list(st.finished) == [1, 1, 1, 1]
    assert list(st.kv_len) == [6, 3, 8, 1]
    # a finished sequence is frozen on the next step
    before = st.copy()
    err = od.kv_commit(st, A, am, 2, 2, page_size=4)
    assert err == 0
    np.testing.assert_array_equal(st.kv_len, before.kv_len)
    np.testing.assert_array_equal(st.out_tokens, before.out_tokens)


def test_commit_errors_leave_state_unchanged():
    g = json.load(open(os.path.join(GOLDEN, "commit_example.json")))
    st = _state_from(g["before"])
    st.free_top = 0                       # nothing free; seq1 pushes 2, seq2+seq3 pop 2
    st.num_pages[1] = 2; st.page_table[1, 2:] = -1   # remove seq1's surplus
    am = np.array(g["before"]["argmax"], np.int32)
    A = od.accept(am, st.draft, 2)
    before = st.copy()
    err = od.kv_commit(st, A, am, 2, 2, eos_id=77, page_size=4)
    assert err == od.ERR_POOL_EXHAUSTED
    for f in ("kv_len", "page_table", "num_pages", "free_stack", "boundary", "draft",
              "out_tokens", "out_count", "finished"):
        np.testing.assert_array_equal(getattr(st, f), getattr(before, f))
    st = _state_from(g["before"])
    st.max_pages = 3
    err = od.kv_commit(st, A, am, 2, 2, eos_id=77, page_size=4)
    assert err & od.ERR_MAX_PAGES


def _check_conservation(st, R, page_size):
    live = []
    for s in range(st.kv_len.shape[0]):
        n = int(st.num_pages[s])
        assert n == (int(st.kv_len[s]) + R + page_size - 1) // page_size
        assert np.all(st.page_table[s, :n] >= 0) and np.all(st.page_table[s, n:] == -1)
        live += list(st.page_table[s, :n])
    free = list(st.free_stack[:st.free_top])
    allp = live + free
    assert len(allp) == len(set(allp)) == st.pool_pages


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_commit_random_steps_conserve_pages(seed):
    rng = np.random.default_rng(seed)
    S, B, V = 6, 5, 7
    R = 2 * B
    L = rng.integers(0, 40, size=S)
    st = synth.make_paged_state(rng, L, R, max_pages=64, scatter=True, slack=0.5,
                                extra_pages=40, n_causal=B)
    _check_conservation(st, R, 16)
    for step in range(30):
        am = rng.integers(0, V, size=(S, R)).astype(np.int32)
        st.draft[:] = np.where(rng.random((S, B - 1)) < 0.7, am[:, :B - 1], st.draft)
        A = od.accept(am, st.draft, B)
        L0, c0 = st.kv_len.copy(), st.out_count.copy()
        err = od.kv_commit(st, A, am, B, B, eos_id=3 if step > 20 else -1)
        assert err == 0
        k = st.out_count - c0
        live = st.finished == 0
        assert np.all((k >= 1) | (st.finished == 1) | (c0 == st.out_count))
        assert np.all(k <= B)
        np.testing.assert_array_equal(st.kv_len - L0, k)
        # every committed token is the verifier's top-1 at its position
        for s in range(S):
            for i in range(int(k[s])):
                assert st.out_tokens[s, c0[s] + i] == am[s, i]
        _check_conservation(st, R, 16)
