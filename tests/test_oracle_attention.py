"""Pins for oracle.attention against library routines and invariants.

* causal rows == torch SDPA with a bottom-right-aligned causal mask
  (``causal_lower_right``) over cache + causal rows only;
* mask rows == unmasked torch SDPA over cache + all window rows (they see
  every key: the whole cache, all causal rows, the whole mask block);
* grouped-query mapping == torch SDPA's ``enable_gqa``;
* paging: any physical page permutation gives identical outputs, and the
  append writes the window's K/V at [L, L+R).
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F
from torch.nn.attention.bias import causal_lower_right

from oracle import attention as oa
from paper_2609_26638_amd import synth


def _dense(ai, s):
    L = int(ai.state.kv_len[s])
    kp, vp = ai.as_f64("k_pool"), ai.as_f64("v_pool")
    ck = oa.gather_cache(kp, ai.state.page_table[s], L, 16)
    cv = oa.gather_cache(vp, ai.state.page_table[s], L, 16, slot_last=True)
    return ck, cv


def _sdpa(q, k, v, scale, mask=None):
    # q [Rq, Hq, D], k/v [T, Hkv, D] -> [Rq, Hq, D]; float64 CPU library routine
    qt = torch.from_numpy(q).permute(1, 0, 2)[None]
    kt = torch.from_numpy(k).permute(1, 0, 2)[None]
    vt = torch.from_numpy(v).permute(1, 0, 2)[None]
    o = F.scaled_dot_product_attention(qt, kt, vt, attn_mask=mask, scale=scale, enable_gqa=True)
    return o[0].permute(1, 0, 2).numpy()


@pytest.mark.parametrize("seed,S,L,Vc,Vm,Hq,Hkv,D", [
    (11, 2, [37, 5], 4, 4, 4, 2, 16),
    (12, 1, [64], 3, 5, 6, 3, 8),
    (13, 3, [1, 17, 33], 8, 8, 8, 2, 32),
    (14, 1, [40], 1, 0, 4, 1, 16),      # plain AR decode row
    (15, 1, [40], 0, 6, 4, 4, 16),      # mask block only
    (16, 2, [0, 9], 2, 3, 2, 2, 8),     # empty cache
])
def test_hybrid_matches_sdpa(seed, S, L, Vc, Vm, Hq, Hkv, D):
    ai = synth.make_attn_inputs(seed, S, L, Vc, Vm, Hq, Hkv, D, "f32", scatter=True)
    q, kn, vn = ai.as_f64("q"), ai.as_f64("k_new"), ai.as_f64("v_new")
    kp, vp = ai.as_f64("k_pool"), ai.as_f64("v_pool")
    dense = [_dense(ai, s) for s in range(S)]
    out = oa.attn_hybrid_block(q, kn, vn, kp, vp, ai.state.page_table, ai.state.kv_len,
                               Vc, Vm, ai.scale)
    for s in range(S):
        ck, cv = dense[s]
        Ls = int(ai.state.kv_len[s])
        if Vc:
            k = np.concatenate([ck, kn[s, :Vc]]); v = np.concatenate([cv, vn[s, :Vc]])
            ref = _sdpa(q[s, :Vc], k, v, ai.scale, causal_lower_right(Vc, Ls + Vc))
            np.testing.assert_allclose(out[s, :Vc], ref, rtol=1e-12, atol=1e-13)
        if Vm:
            k = np.concatenate([ck, kn[s]]); v = np.concatenate([cv, vn[s]])
            ref = _sdpa(q[s, Vc:], k, v, ai.scale, None)
            np.testing.assert_allclose(out[s, Vc:], ref, rtol=1e-12, atol=1e-13)


def test_visible_hi_rule():
    hi = oa.visible_hi(100, 3, 4)
    assert list(hi) == [100, 101, 102, 106, 106, 106, 106]


def test_append_writes_window_kv():
    ai = synth.make_attn_inputs(3, 2, [20, 7], 4, 4, 4, 2, 8, "f32")
    kp, vp = ai.as_f64("k_pool"), ai.as_f64("v_pool")
    kn, vn = ai.as_f64("k_new"), ai.as_f64("v_new")
    oa.attn_hybrid_block(ai.as_f64("q"), kn, vn, kp, vp, ai.state.page_table,
                         ai.state.kv_len, 4, 4, ai.scale)
    for s in range(2):
        L = int(ai.state.kv_len[s])
        got = oa.gather_cache(kp, ai.state.page_table[s], L + 8, 16)[L:]
        np.testing.assert_array_equal(got, kn[s])
        got = oa.gather_cache(vp, ai.state.page_table[s], L + 8, 16, slot_last=True)[L:]
        np.testing.assert_array_equal(got, vn[s])


def test_page_permutation_invariance():
    ai = synth.make_attn_inputs(5, 2, [50, 23], 4, 4, 4, 2, 8, "f32", scatter=False)
    q, kn, vn = ai.as_f64("q"), ai.as_f64("k_new"), ai.as_f64("v_new")
    kp, vp = ai.as_f64("k_pool"), ai.as_f64("v_pool")
    out1 = oa.attn_hybrid_block(q, kn, vn, kp.copy(), vp.copy(), ai.state.page_table,
                                ai.state.kv_len, 4, 4, ai.scale)
    perm = np.random.default_rng(0).permutation(kp.shape[0])
    inv = np.argsort(perm)
    kp2, vp2 = kp[perm], vp[perm]      # physical page p moves to slot inv[p]
    pt2 = np.where(ai.state.page_table >= 0, inv[np.maximum(ai.state.page_table, 0)], -1)
    out2 = oa.attn_hybrid_block(q, kn, vn, kp2, vp2, pt2, ai.state.kv_len, 4, 4, ai.scale)
    np.testing.assert_array_equal(out1, out2)


def test_sampled_rows_equal_full():
    ai = synth.make_attn_inputs(7, 3, [31, 64, 2], 5, 3, 4, 2, 16, "f32")
    q, kn, vn = ai.as_f64("q"), ai.as_f64("k_new"), ai.as_f64("v_new")
    kp, vp = ai.as_f64("k_pool"), ai.as_f64("v_pool")
    samples = [(0, 0, 0), (1, 4, 3), (2, 7, 1), (1, 5, 2)]
    sm = oa.attn_sampled(q, kn, vn, kp, vp, ai.state.page_table, ai.state.kv_len, 5, 3,
                         ai.scale, samples)
    out = oa.attn_hybrid_block(q, kn, vn, kp, vp, ai.state.page_table, ai.state.kv_len,
                               5, 3, ai.scale)
    for (s, r, h) in samples:
        np.testing.assert_allclose(sm[(s, r, h)], out[s, r, h], rtol=1e-13, atol=1e-14)
    # pools kept in bf16 bits and decoded page by page give the same rows
    bi = synth.make_attn_inputs(7, 3, [31, 64, 2], 5, 3, 4, 2, 16, "bf16")
    full = oa.attn_sampled(bi.as_f64("q"), bi.as_f64("k_new"), bi.as_f64("v_new"),
                           bi.as_f64("k_pool"), bi.as_f64("v_pool"), bi.state.page_table,
                           bi.state.kv_len, 5, 3, bi.scale, samples)
    lazy = oa.attn_sampled(bi.as_f64("q"), bi.as_f64("k_new"), bi.as_f64("v_new"),
                           bi.k_pool, bi.v_pool, bi.state.page_table, bi.state.kv_len, 5, 3,
                           bi.scale, samples, decode=synth.bf16_to_f64)
    for key in samples:
        np.testing.assert_array_equal(full[key], lazy[key])


def test_constant_values_give_constant_output():
    # softmax weights sum to one: if every visible V row is the same vector c,
    # the output is c whatever the scores.
    ai = synth.make_attn_inputs(9, 1, [13], 3, 3, 2, 1, 8, "f32")
    q, kn = ai.as_f64("q"), ai.as_f64("k_new")
    c = np.linspace(-1, 1, 8)
    kp = ai.as_f64("k_pool")
    vp = np.broadcast_to(c[:, None], ai.v_pool.shape).copy()   # [P, Hkv, D, 16]
    vn = np.broadcast_to(c, ai.v_new.shape).copy()
    out = oa.attn_hybrid_block(q, kn, vn, kp, vp, ai.state.page_table, ai.state.kv_len,
                               3, 3, ai.scale)
    np.testing.assert_allclose(out, np.broadcast_to(c, out.shape), rtol=0, atol=1e-14)


def test_causal_rows_ignore_mask_rows():
    ai = synth.make_attn_inputs(21, 1, [29], 4, 4, 4, 2, 8, "f32")
    q, kn, vn = ai.as_f64("q"), ai.as_f64("k_new"), ai.as_f64("v_new")
    kp, vp = ai.as_f64("k_pool"), ai.as_f64("v_pool")
    o1 = oa.attn_hybrid_block(q, kn, vn, kp.copy(), vp.copy(), ai.state.page_table,
                              ai.state.kv_len, 4, 4, ai.scale)
    kn2, vn2, q2 = kn.copy(), vn.copy(), q.copy()
    kn2[:, 4:] += 3.0; vn2[:, 4:] -= 2.0; q2[:, 4:] *= -1
    o2 = oa.attn_hybrid_block(q2, kn2, vn2, kp.copy(), vp.copy(), ai.state.page_table,
                              ai.state.kv_len, 4, 4, ai.scale)
    np.testing.assert_array_equal(o1[:, :4], o2[:, :4])
    assert not np.allclose(o1[:, 4:], o2[:, 4:])
