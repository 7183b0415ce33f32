"""Pins for the oracle's direct block-diffusion decoder (appendix "Direct
Block-Diffusion Decoding").

* Confidence: closed forms (uniform logits give 1/V, two logits ln 3 and 0
  give 3/4), shift invariance, and scipy's softmax on random rows.
* Reveal: hand-derived cases in ``golden/reveal_cases.json``.
* Decoding: B = 1 reduces to greedy AR (the boundary row predicts the only
  position, one reveal per block, the cache-write forward keeps x0), so the
  stream must equal the AR stream; the first position of every block is
  predicted by the causal boundary row, so it equals the AR token from the
  same state; tau_c = 0 reveals a whole block in one forward and a
  threshold above 1 exactly one position per forward; revealed tokens never
  change and every forward reveals at least one; a stop token truncates the
  output and freezes the sequence.
"""
import copy
import json
import os

import numpy as np
import pytest
import scipy.special

from oracle import decode as odec
from oracle import model as om
from paper_2609_26638_amd import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "reveal_cases.json")


def _model(seed, V=11, H=32, Hq=4, Hkv=2, D=8, n_layers=2, ffn=48, std=0.5, pool=96):
    w = synth.make_model_weights(seed, V, H, Hq, Hkv, D, n_layers, ffn, std=std)
    kp = [np.zeros((pool, Hkv, 16, D), np.float32) for _ in range(n_layers)]
    vp = [np.zeros((pool, Hkv, D, 16), np.float32) for _ in range(n_layers)]
    return w, kp, vp, np.random.default_rng(seed)


def _prefilled(seed, S=2, P=9, B=4, **kw):
    w, kp, vp, rng = _model(seed, **kw)
    m = om.OracleModel(w, kp, vp)
    rows = P + B + 1
    st = synth.make_paged_state(rng, np.zeros(S, np.int64), rows, max_pages=32, scatter=True,
                                slack=0.0, extra_pages=kp[0].shape[0] - S * 2 - rows // 16 * S,
                                n_causal=B + 1, max_new=256)
    m.prefill(st, rng.standard_normal((S, P, w.H)), B)
    return m, st


def _clone(m):
    c = copy.copy(m)
    c.k_pools = [a.copy() for a in m.k_pools]
    c.v_pools = [a.copy() for a in m.v_pools]
    return c


def _ar_stream(m, st, n):
    m, st = _clone(m), st.copy()
    for _ in range(n):
        m.ar_step(st)
    return [list(st.out_tokens[s, :st.out_count[s]]) for s in range(st.kv_len.shape[0])]


def test_confidence_closed_forms_and_softmax():
    V = 37
    t, c = odec.top1_confidence(np.zeros(V))
    assert t == 0 and abs(c - 1.0 / V) < 1e-15
    t, c = odec.top1_confidence(np.array([0.0, np.log(3.0)]))
    assert t == 1 and abs(c - 0.75) < 1e-15
    rng = np.random.default_rng(0)
    for _ in range(20):
        z = rng.standard_normal(V) * rng.uniform(0.1, 8.0)
        t, c = odec.top1_confidence(z)
        p = scipy.special.softmax(z)
        assert t == int(np.argmax(p))
        assert abs(c - p.max()) < 1e-14
        assert abs(odec.top1_confidence(z + 123.25)[1] - c) < 1e-13


def test_reveal_golden_cases():
    cases = json.load(open(GOLDEN))["cases"]
    for cs in cases:
        block = np.array([cs["block"]])
        out = odec.reveal(block, np.array([cs["am"]]), np.array([cs["conf"]]), cs["tau_c"],
                          np.array([cs["finished"]]))
        assert list(out[0]) == cs["expect"], cs["name"]
        assert list(block[0]) == cs["block"]          # input untouched


@pytest.mark.parametrize("seed", [20, 21])
def test_b1_diffusion_is_greedy_ar(seed):
    m, st = _prefilled(seed, B=1)
    n = 12
    ar = _ar_stream(m, st, n)
    ms, ss = _clone(m), st.copy()
    for _ in range(n):
        block, steps, err = ms.diffusion_block(ss, 1, tau_c=0.9)
        assert err == 0 and steps == 1
    for s in range(2):
        assert list(ss.out_tokens[s, :ss.out_count[s]]) == ar[s]
        assert ss.kv_len[s] == st.kv_len[s] + n


@pytest.mark.parametrize("seed,B,tau", [(22, 4, 0.3), (23, 6, 0.15), (24, 3, 0.5)])
def test_block_structure_and_first_position_is_ar(seed, B, tau):
    m, st = _prefilled(seed, B=B)
    ms, ss = _clone(m), st.copy()
    for _ in range(4):
        ar_next = _ar_stream(ms, ss, 1)
        before = ss.copy()
        # denoise by hand to watch every step
        block = np.full((2, B), -1, dtype=np.int64)
        steps = 0
        mm = _clone(ms)
        while (block < 0).any():
            _, am, conf, nb = mm.diffusion_denoise(ss, block, tau)
            kept = block >= 0
            assert np.array_equal(nb[kept], block[kept])           # revealed stay fixed
            open_ = (block < 0).any(1)
            assert np.all((nb >= 0).sum(1)[open_] > (block >= 0).sum(1)[open_])  # >= 1 reveal
            np.testing.assert_array_equal(nb[~open_], block[~open_])
            block = nb
            steps += 1
        assert steps <= B
        got, steps2, err = ms.diffusion_block(ss, B, tau)
        assert err == 0 and steps2 == steps
        np.testing.assert_array_equal(got, block)
        for s in range(2):
            assert got[s, 0] == ar_next[s][-1]                      # position 1 == AR token
            new = list(ss.out_tokens[s, before.out_count[s]:ss.out_count[s]])
            assert new == list(got[s])
            assert ss.boundary[s] == got[s, -1]
        np.testing.assert_array_equal(ss.kv_len, before.kv_len + B)


def test_threshold_extremes():
    B = 5
    m, st = _prefilled(25, B=B)
    a, sa = _clone(m), st.copy()
    _, steps, err = a.diffusion_block(sa, B, tau_c=0.0)
    assert err == 0 and steps == 1
    b, sb = _clone(m), st.copy()
    _, steps, err = b.diffusion_block(sb, B, tau_c=1.01)
    assert err == 0 and steps == B
    # tau_c = 0: the block is the top-1 of one forward over [x0, [M] x B],
    # the same forward the two-forward round drafts with
    c, sc = _clone(m), st.copy()
    logits_d, _, _, _, _ = c.literal_round(sc, B)
    draft_top1 = odec.top1_rows(logits_d)[:, :B]
    np.testing.assert_array_equal(sa.out_tokens[:, st.out_count[0]:st.out_count[0] + B],
                                  draft_top1)


def test_stop_token_truncates_and_freezes():
    B = 4
    m, st = _prefilled(26, B=B)
    probe, sp = _clone(m), st.copy()
    blocks = [probe.diffusion_block(sp, B, 0.3)[0] for _ in range(3)]
    # a stop token from the second block of sequence 0 that the first
    # committed token is not
    stream = np.concatenate([blocks[0][0], blocks[1][0]])
    x0 = int(st.out_tokens[0, 0])
    eos = next(int(t) for t in blocks[1][0] if int(t) != x0)
    first = next(i for i, t in enumerate(stream) if t == eos)
    ms, ss = _clone(m), st.copy()
    for _ in range(3):
        _, _, err = ms.diffusion_block(ss, B, 0.3, eos_id=eos)
        assert err == 0
    got = list(ss.out_tokens[0, :ss.out_count[0]])
    assert got == [x0] + list(stream[:first + 1])
    assert ss.finished[0] == 1
