"""Pins for the per-acceptance multi-draft step (oracle).

The paper's round redrafts from the true boundary after every acceptance
(appendix "Self-Speculative Decoding and KV-Cache Update", item Next round);
the structured-mask AR-diffusion hybrids its related work cites draft one
block per possible acceptance length inside the verifying forward.  Here the
mask rows are B groups of B rows; group k assumes A = k: it sits right after
d_k, sees the cache, the causal rows 0..k and itself, and supplies the next
draft when A = k.

Pins:
* the grouped visibility and the row positions against hand-written tables;
* one group is the hybrid mask (``visible_hi``), with positions L + r;
* group k equals the mask block of a step that verifies only x0, d_1..d_k
  (a forward with k + 1 causal rows and B mask rows from the same state);
* B = 1 is the fused step; every committed token is greedy AR's (the paper's
  AR-equivalence argument holds for any draft);
* a draft equal to the AR continuation is fully accepted and the next draft
  is group B-1's, which equals the fused step's next draft;
* after a partial acceptance the next draft is group A's top-1.
"""
import copy

import numpy as np
import pytest

from oracle import attention as oa
from oracle import decode as od
from oracle import model as om
from paper_2609_26638_amd import synth


def test_grouped_visibility_hand_table():
    # L = 2, two causal rows (x0, d_1), two groups of two mask rows
    vis = oa.visible_mask(2, 2, 4, group=2)
    #        cache  c0 c1  g0 g0  g1 g1
    want = [[1, 1,  1, 0,  0, 0,  0, 0],    # causal row 0
            [1, 1,  1, 1,  0, 0,  0, 0],    # causal row 1
            [1, 1,  1, 0,  1, 1,  0, 0],    # group 0 (A = 0): sees x0 only
            [1, 1,  1, 0,  1, 1,  0, 0],
            [1, 1,  1, 1,  0, 0,  1, 1],    # group 1 (A = 1): sees x0, d_1
            [1, 1,  1, 1,  0, 0,  1, 1]]
    np.testing.assert_array_equal(vis, np.array(want, dtype=bool))
    np.testing.assert_array_equal(oa.window_positions(2, 2, 4, group=2), [2, 3, 3, 4, 4, 5])


@pytest.mark.parametrize("L,nc,nm", [(0, 3, 3), (5, 4, 4), (17, 1, 6), (9, 6, 0), (3, 0, 5)])
def test_one_group_is_the_hybrid_mask(L, nc, nm):
    vis = oa.visible_mask(L, nc, nm)
    hi = oa.visible_hi(L, nc, nm)
    np.testing.assert_array_equal(vis, np.arange(L + nc + nm)[None, :] <= hi[:, None])
    np.testing.assert_array_equal(oa.window_positions(L, nc, nm), L + np.arange(nc + nm))


def _model(seed, V=13, B=3, S=2, P=7, std=0.7):
    w = synth.make_model_weights(seed, V, 32, 4, 2, 8, 2, 48, std=std, gain_std=0.2)
    pool = 96
    kp = [np.zeros((pool, 2, 16, 8), np.float32) for _ in range(2)]
    vp = [np.zeros((pool, 2, 8, 16), np.float32) for _ in range(2)]
    m = om.OracleModel(w, kp, vp)
    rng = np.random.default_rng(seed)
    R = B + B * B
    st = synth.make_paged_state(rng, np.zeros(S, np.int64), P + R, max_pages=40, scatter=True,
                                slack=0.0, extra_pages=pool - S * ((P + R + 15) // 16),
                                n_causal=B, max_new=256)
    m.prefill(st, rng.standard_normal((S, P, w.H)), B)
    return m, st


def _clone(m):
    c = copy.copy(m)
    c.k_pools = [a.copy() for a in m.k_pools]
    c.v_pools = [a.copy() for a in m.v_pools]
    return c


@pytest.mark.parametrize("seed,B", [(1, 3), (2, 4)])
def test_group_k_is_the_draft_of_a_step_verifying_k_drafts(seed, B):
    m, st = _model(seed, B=B)
    st.draft[:] = np.random.default_rng(seed).integers(0, m.V, size=st.draft.shape)
    S = st.kv_len.shape[0]
    tok = np.empty((S, B + B * B), np.int64)
    tok[:, 0] = st.boundary
    tok[:, 1:B] = st.draft[:, :B - 1]
    tok[:, B:] = m.mask_id
    full = _clone(m).forward(m.embed[tok], st, B, B * B, group=B)
    for k in range(B):
        sub = np.concatenate([tok[:, :k + 1], np.full((S, B), m.mask_id)], axis=1)
        ref = _clone(m).forward(m.embed[sub], st, k + 1, B)
        got = full[:, B + k * B:B + (k + 1) * B]
        np.testing.assert_allclose(got, ref[:, k + 1:], rtol=0, atol=1e-12 * np.abs(ref).max())
        # ... and the causal rows equal that step's causal rows
        np.testing.assert_allclose(full[:, :k + 1], ref[:, :k + 1], rtol=0,
                                   atol=1e-12 * np.abs(ref).max())


def test_b1_is_the_fused_step():
    m, st = _model(5, B=1)
    a, sa = _clone(m), st.copy()
    b, sb = _clone(m), st.copy()
    for _ in range(4):
        la, ama, Aa, ea = a.multidraft_step(sa, 1)
        lb, amb, Ab, eb = b.fused_step(sb, 1)
        assert ea == eb == 0
        np.testing.assert_allclose(la, lb, rtol=0, atol=1e-12 * np.abs(lb).max())
        np.testing.assert_array_equal(ama, amb)
        for f in ("kv_len", "page_table", "boundary", "draft", "out_tokens", "out_count"):
            np.testing.assert_array_equal(getattr(sa, f), getattr(sb, f))


def _ar(m, st, n):
    m, st = _clone(m), st.copy()
    for _ in range(n):
        m.ar_step(st)
    return [list(st.out_tokens[s, :st.out_count[s]]) for s in range(st.kv_len.shape[0])]


@pytest.mark.parametrize("seed,B", [(7, 2), (8, 3), (9, 4)])
def test_stream_equals_greedy_ar(seed, B):
    m, st = _model(seed, B=B)
    n = 20
    ar = _ar(m, st, n)
    ms, ss = _clone(m), st.copy()
    while min(ss.out_count) < n + 1:
        _, am, A, err = ms.multidraft_step(ss, B)
        assert err == 0 and np.all((A >= 0) & (A <= B - 1))
    for s in range(ss.kv_len.shape[0]):
        got = list(ss.out_tokens[s, :ss.out_count[s]])
        L = min(len(got), len(ar[s]))
        assert got[:L] == ar[s][:L]


@pytest.mark.parametrize("seed", [11, 12])
def test_full_acceptance_and_next_draft_from_the_accepted_group(seed):
    B = 3
    m, st = _model(seed, B=B)
    ar = _ar(m, st, B + 1)
    S = st.kv_len.shape[0]
    full = st.copy()
    for s in range(S):
        full.draft[s] = ar[s][1:B]
    # fully accepted: A = B-1, and the next draft is group B-1's, which is the
    # fused step's mask block
    a, sa = _clone(m), full.copy()
    _, am, A, err = a.multidraft_step(sa, B)
    assert err == 0 and list(A) == [B - 1] * S
    b, sb = _clone(m), full.copy()
    _, amb, Ab, _ = b.fused_step(sb, B)
    np.testing.assert_array_equal(A, Ab)
    np.testing.assert_array_equal(sa.draft, sb.draft)
    np.testing.assert_array_equal(sa.out_tokens, sb.out_tokens)
    # partial acceptance: d_1 right, d_2 wrong -> A = 1, the draft is group 1's
    part = full.copy()
    for s in range(S):
        part.draft[s, 1] = (ar[s][2] + 1) % m.V
    c, sc = _clone(m), part.copy()
    _, amc, Ac, err = c.multidraft_step(sc, B)
    assert err == 0 and list(Ac) == [1] * S
    np.testing.assert_array_equal(sc.draft, amc[:, B + B:B + B + B - 1])
    np.testing.assert_array_equal(sc.kv_len, part.kv_len + 2)
    for s in range(S):
        assert list(sc.out_tokens[s, :sc.out_count[s]]) == ar[s][:3]
