"""Pins for oracle.model.

Layers: RMSNorm and SiLU against torch's library routines; RoPE against a
complex-number formulation and its relative-position property.  Decoding:
the paper's AR-equivalence argument (committed stream of self-speculative
decoding == greedy AR, in exact arithmetic) on small random-init models,
B=1 reducing to AR, a draft equal to the AR continuation being fully
accepted, and every draft over a tiny vocabulary committing the AR tokens.
The paper's two-forward round: its stream equals greedy AR, and its
accounting (a round commits A + 2 tokens in two forwards, so tokens per
forward = (A + 2) / 2) matches the acceptance / TPF pairs the paper prints.
"""
import json
import os
import itertools

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import model as om
from paper_2609_26638_amd import synth


def test_rmsnorm_matches_torch():
    rng = np.random.default_rng(0)
    x = rng.standard_normal((3, 5, 24)); g = rng.standard_normal(24)
    ref = F.rms_norm(torch.from_numpy(x), (24,), torch.from_numpy(g), eps=1e-6).numpy()
    np.testing.assert_allclose(om.rmsnorm(x, g, 1e-6), ref, rtol=1e-13, atol=1e-14)


def test_silu_matches_torch():
    x = np.linspace(-9, 9, 101)
    np.testing.assert_allclose(om.silu(x), F.silu(torch.from_numpy(x)).numpy(), rtol=1e-14)


def test_rope_complex_form_and_relative_position():
    rng = np.random.default_rng(1)
    D, theta = 16, 10000.0
    x = rng.standard_normal((4, 3, D))
    pos = np.array([0, 5, 17, 1000])
    got = om.rope(x, pos, theta)
    # complex form: z_i = x_i + i x_{i+D/2} multiplied by exp(i pos w_i)
    w = theta ** (-np.arange(D // 2) * 2.0 / D)
    z = (x[..., :D // 2] + 1j * x[..., D // 2:]) * np.exp(1j * pos[:, None, None] * w)
    np.testing.assert_allclose(got, np.concatenate([z.real, z.imag], -1), rtol=1e-12, atol=1e-12)
    np.testing.assert_array_equal(om.rope(x[:1], np.array([0]), theta), x[:1])
    # <rope(q, m), rope(k, n)> depends only on m - n
    q = rng.standard_normal((1, 1, D)); k = rng.standard_normal((1, 1, D))
    def dot(m, n):
        return float(np.sum(om.rope(q, np.array([m]), theta) * om.rope(k, np.array([n]), theta)))
    assert abs(dot(7, 3) - dot(104, 100)) < 1e-10
    assert abs(dot(7, 3) - dot(8, 3)) > 1e-6


def _tiny_model(seed, V=11, H=32, Hq=4, Hkv=2, D=8, n_layers=2, ffn=48, std=0.5, pool=64):
    w = synth.make_model_weights(seed, V, H, Hq, Hkv, D, n_layers, ffn, std=std)
    rng = np.random.default_rng(seed)
    kp = [np.zeros((pool, Hkv, 16, D), np.float32) for _ in range(n_layers)]
    vp = [np.zeros((pool, Hkv, D, 16), np.float32) for _ in range(n_layers)]
    return w, kp, vp, rng


def _prefilled(seed, S=2, P=9, B=4, n_causal=None, **kw):
    w, kp, vp, rng = _tiny_model(seed, **kw)
    m = om.OracleModel(w, kp, vp)
    rows = P + max(2 * B, B + 2)
    st = synth.make_paged_state(rng, np.zeros(S, np.int64), rows, max_pages=32,
                                scatter=True, slack=0.0, extra_pages=kp[0].shape[0] - S * 2
                                - rows // 16 * S, n_causal=B if n_causal is None else n_causal,
                                max_new=256)
    x = rng.standard_normal((S, P, w.H))
    m.prefill(st, x, B)
    return m, st


def _ar_tokens(m, st, n):
    st = st.copy()
    m = _clone(m)
    for _ in range(n):
        m.ar_step(st)
    return [list(st.out_tokens[s, :st.out_count[s]]) for s in range(st.kv_len.shape[0])]


def _clone(m):
    import copy
    c = copy.copy(m)
    c.k_pools = [a.copy() for a in m.k_pools]
    c.v_pools = [a.copy() for a in m.v_pools]
    return c


@pytest.mark.parametrize("seed,B", [(0, 4), (1, 3), (2, 6), (3, 1)])
def test_selfspec_stream_equals_greedy_ar(seed, B):
    m, st = _prefilled(seed, B=B)
    n = 30
    ar = _ar_tokens(m, st, n)
    ms, ss = _clone(m), st.copy()
    steps = 0
    while min(ss.out_count) < n + 1:
        _, _, A, err = ms.fused_step(ss, B)
        assert err == 0
        steps += 1
    for s in range(ss.kv_len.shape[0]):
        got = list(ss.out_tokens[s, :ss.out_count[s]])
        L = min(len(got), len(ar[s]))
        assert got[:L] == ar[s][:L]
    assert steps <= n + 1


@pytest.mark.parametrize("seed", [4, 5])
def test_ar_continuation_draft_fully_accepted(seed):
    B = 5
    m, st = _prefilled(seed, B=B)
    ar = _ar_tokens(m, st, B + 2)
    ss = st.copy()
    for s in range(ss.kv_len.shape[0]):
        # stream so far is [x0]; the AR continuation after x0 is ar[s][1:]
        ss.draft[s] = ar[s][1:B]
    _, _, A, err = _clone(m).fused_step(ss, B)
    assert err == 0
    assert list(A) == [B - 1] * ss.kv_len.shape[0]
    for s in range(ss.kv_len.shape[0]):
        assert list(ss.out_tokens[s, :ss.out_count[s]]) == ar[s][:B + 1]
    np.testing.assert_array_equal(ss.kv_len, st.kv_len + B)


def test_every_draft_over_tiny_vocab_commits_ar_tokens():
    V, B = 5, 3
    m, st = _prefilled(6, S=1, V=V, B=B, std=0.8)
    ar = _ar_tokens(m, st, B + 1)[0]
    seen_A = set()
    for d in itertools.product(range(V), repeat=B - 1):
        ss = st.copy()
        ss.draft[0] = d
        _, _, A, err = _clone(m).fused_step(ss, B)
        assert err == 0
        got = list(ss.out_tokens[0, :ss.out_count[0]])
        k = len(got) - 1
        assert k == A[0] + 1
        assert got == ar[:len(got)]
        # A is exactly the number of leading draft tokens equal to AR's
        lead = 0
        for j in range(B - 1):
            if d[j] != ar[1 + j]:
                break
            lead += 1
        assert A[0] == lead
        seen_A.add(int(A[0]))
    assert seen_A == set(range(B))


def test_b1_step_is_ar_step():
    m, st = _prefilled(7, B=1)
    ar = _ar_tokens(m, st, 6)
    ss, ms = st.copy(), _clone(m)
    for _ in range(6):
        _, _, A, err = ms.fused_step(ss, 1)
        assert err == 0 and list(A) == [0, 0]
    for s in range(2):
        assert list(ss.out_tokens[s, :ss.out_count[s]]) == ar[s]


@pytest.mark.parametrize("seed,B", [(10, 4), (11, 3), (12, 1), (13, 6)])
def test_literal_round_stream_equals_greedy_ar(seed, B):
    m, st = _prefilled(seed, B=B, n_causal=B + 1)
    n = 30
    ar = _ar_tokens(m, st, n)
    ms, ss = _clone(m), st.copy()
    rounds = 0
    while min(ss.out_count) < n + 1:
        before = ss.out_count.copy()
        _, _, _, A, err = ms.literal_round(ss, B)
        assert err == 0
        assert np.all((A >= 0) & (A <= B))
        # a round commits a0, d_1..d_A and a_{A+1}
        np.testing.assert_array_equal(ss.out_count - before, A + 2)
        rounds += 1
    for s in range(ss.kv_len.shape[0]):
        got = list(ss.out_tokens[s, :ss.out_count[s]])
        L = min(len(got), len(ar[s]))
        assert got[:L] == ar[s][:L]
        # KV holds every committed token but the boundary: the prompt, x0 and
        # the committed run up to its last token
        assert ss.kv_len[s] == st.kv_len[s] + ss.out_count[s] - 1
    assert rounds <= (n + 1) // 2 + 1


def test_literal_round_accounting_gives_tokens_per_forward():
    B = 4
    m, st = _prefilled(14, B=B, n_causal=B + 1, std=0.9)
    ms, ss = _clone(m), st.copy()
    As, committed = [], 0
    for _ in range(8):
        before = int(ss.out_count.sum())
        _, _, _, A, err = ms.literal_round(ss, B)
        assert err == 0
        As.extend(int(a) for a in A)
        committed += int(ss.out_count.sum()) - before
    forwards = 2 * 8 * ss.kv_len.shape[0]         # two forwards per round and sequence
    assert committed / forwards == (np.mean(As) + 2) / 2


def test_tpf_identity_against_printed_table():
    g = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "tpf_by_content_type.json")))
    for row in g["rows"]:
        # the paper prints one decimal: the identity must agree to that digit
        assert abs((row["accepted"] + 2) / 2 - row["tpf"]) <= 0.05 + 1e-12, row


@pytest.mark.parametrize("seed,B,tau_d", [(30, 4, 0.05), (31, 3, 0.3), (32, 6, 1.01)])
def test_refined_draft_round_stream_equals_greedy_ar(seed, B, tau_d):
    """Multi-step drafting (experiments, "Draft Schedule") changes only the
    draft, so the committed stream is still greedy AR's; a refinement takes
    1..B+1 draft forwards and reveals at least one prediction per forward."""
    m, st = _prefilled(seed, B=B, n_causal=B + 1)
    n = 24
    ar = _ar_tokens(m, st, n)
    ms, ss = _clone(m), st.copy()
    while min(ss.out_count) < n + 1:
        _, _, _, A, err = ms.literal_round(ss, B, tau_d=tau_d)
        assert err == 0
        assert 1 <= ms.draft_steps <= B + 1
        if tau_d > 1:
            assert ms.draft_steps == B + 1
    for s in range(ss.kv_len.shape[0]):
        got = list(ss.out_tokens[s, :ss.out_count[s]])
        L = min(len(got), len(ar[s]))
        assert got[:L] == ar[s][:L]


def test_refined_draft_with_zero_threshold_is_one_shot():
    B = 5
    m, st = _prefilled(33, B=B, n_causal=B + 1)
    a, sa = _clone(m), st.copy()
    b, sb = _clone(m), st.copy()
    for _ in range(3):
        _, lv_a, _, A_a, _ = a.literal_round(sa, B)
        _, lv_b, _, A_b, _ = b.literal_round(sb, B, tau_d=0.0)
        assert b.draft_steps == 1
        np.testing.assert_array_equal(A_a, A_b)
        np.testing.assert_array_equal(lv_a, lv_b)
        np.testing.assert_array_equal(sa.draft, sb.draft)
        np.testing.assert_array_equal(sa.out_tokens, sb.out_tokens)
