"""Pins for the oracle's decoder composition and prefill.

``OracleModel.forward`` composes pre-norm attention and MLP sub-layers with
residuals, rotary positions, the hybrid-mask attention over a paged cache, a
final norm and the LM head (the layer reading of the decoder, the paper
leaving the architecture open; the mask token is an extra embedding row,
Method "AR-to-Diffusion Conversion").  The AR-equivalence pins hold for any
causal model, so they cannot see a wrong composition; these tests compare the
oracle against an independent torch composition built from library
routines: ``F.rms_norm`` with its weight, rotary embedding in complex form
(``torch.polar``), ``F.scaled_dot_product_attention`` with an explicit
boolean hybrid mask over keys gathered by page-table indexing, ``F.silu``
and plain matmuls.  Gains are drawn away from one, so a swapped or dropped
gain, an LM head on the un-normed stream or a residual taken after the norm
all fail.

Prefill (appendix item State: the first boundary is produced by prefill):
its boundary is the top-1 of row P-1 of a causal-only forward of the prefix,
the mask rows do not change the prefix rows' logits, and the first draft is
the top-1 of the mask rows.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import decode as od
from oracle import model as om
from paper_2609_26638_amd import synth

PAGE = 16


def _weights(seed, V=37, H=48, Hq=4, Hkv=2, D=12, n_layers=2, ffn=40):
    # large weights and gains N(1, 0.3): every term of the composition moves the logits
    return synth.make_model_weights(seed, V, H, Hq, Hkv, D, n_layers, ffn, std=0.4,
                                    gain_std=0.3)


def _state_and_pools(w, seed, kv_lens, R):
    rng = np.random.default_rng(seed)
    st = synth.make_paged_state(rng, np.asarray(kv_lens, np.int64), R, max_pages=16,
                                scatter=True, slack=0.2, n_causal=2)
    P = st.pool_pages
    kp = [rng.standard_normal((P, w.Hkv, PAGE, w.D)) for _ in range(w.n_layers)]
    vp = [rng.standard_normal((P, w.Hkv, w.D, PAGE)) for _ in range(w.n_layers)]
    return st, kp, vp


def _t(a):
    return torch.from_numpy(np.asarray(a, dtype=np.float64))


def _rope_complex(x, pos, theta):
    """x [n, h, D] rotated at positions pos [n]: pairs (x_i, x_{i+D/2}) as one
    complex number times exp(i * pos * theta^(-2i/D))."""
    D = x.shape[-1]
    w = theta ** (-torch.arange(D // 2, dtype=torch.float64) * 2.0 / D)
    rot = torch.polar(torch.ones_like(pos[:, None] * w), pos[:, None].double() * w)  # [n, D/2]
    z = torch.complex(x[..., :D // 2], x[..., D // 2:]) * rot[:, None, :]
    return torch.cat([z.real, z.imag], dim=-1)


def _torch_forward(w, kp, vp, st, x, n_causal, n_mask, mistake=None):
    """Independent composition: returns logits [S, R, V] (pools not modified).
    ``mistake`` plants one error, to show the pin rejects it."""
    S, R, H = x.shape
    G = w.Hq // w.Hkv
    out = []
    for s in range(S):
        L = int(st.kv_len[s])
        pages = torch.from_numpy(st.page_table[s, :(L + PAGE - 1) // PAGE].astype(np.int64))
        pos = torch.arange(L, L + R)
        # hybrid mask: causal row r sees keys <= L + r; mask rows see all L + R keys
        keys = torch.arange(L + R)
        hi = torch.where(torch.arange(R) < n_causal, L + torch.arange(R),
                         torch.full((R,), L + R - 1))
        allowed = keys[None, :] <= hi[:, None]                       # [R, L + R]
        h_res = _t(x[s])
        for l in range(w.n_layers):
            hn = F.rms_norm(h_res, (H,), _t(w.g_attn[l]), eps=w.eps)
            q = (hn @ _t(w.wq[l])).view(R, w.Hq, w.D)
            k = (hn @ _t(w.wk[l])).view(R, w.Hkv, w.D)
            v = (hn @ _t(w.wv[l])).view(R, w.Hkv, w.D)
            q = _rope_complex(q, pos, w.rope_theta)
            k = _rope_complex(k, pos, w.rope_theta)
            # cache rows by page-table indexing: [pages, Hkv, 16, D] -> [L, Hkv, D]
            kc = _t(kp[l])[pages].permute(0, 2, 1, 3).reshape(-1, w.Hkv, w.D)[:L]
            vc = _t(vp[l])[pages].permute(0, 3, 1, 2).reshape(-1, w.Hkv, w.D)[:L]
            K = torch.cat([kc, k], 0).repeat_interleave(G, dim=1)   # [L+R, Hq, D]
            Vv = torch.cat([vc, v], 0).repeat_interleave(G, dim=1)
            o = F.scaled_dot_product_attention(q.transpose(0, 1), K.transpose(0, 1),
                                               Vv.transpose(0, 1), attn_mask=allowed)
            base = hn if mistake == "residual_after_norm" else h_res
            h_res = base + o.transpose(0, 1).reshape(R, w.Hq * w.D) @ _t(w.wo[l])
            hm = F.rms_norm(h_res, (H,), _t(w.g_mlp[l]), eps=w.eps)
            h_res = h_res + (F.silu(hm @ _t(w.w_gate[l])) * (hm @ _t(w.w_up[l]))) @ _t(w.w_down[l])
        y = F.rms_norm(h_res, (H,), _t(w.g_final), eps=w.eps)
        if mistake == "lm_head_unnormed":
            y = h_res
        out.append((y @ _t(w.lm_head)).numpy())
    return np.stack(out)


@pytest.mark.parametrize("seed,kv_lens,n_causal,n_mask", [
    (0, [37, 5], 3, 3),      # fused step shape (B causal + B mask rows), ragged cache
    (1, [0, 20], 1, 4),      # the paper's draft forward (1, B), one empty cache
    (2, [33], 5, 0),         # the paper's verify forward (B + 1, 0)
    (3, [16, 47], 1, 0),     # one AR row
])
def test_forward_equals_torch_composition(seed, kv_lens, n_causal, n_mask):
    w = _weights(seed)
    R = n_causal + n_mask
    st, kp, vp = _state_and_pools(w, seed, kv_lens, R)
    rng = np.random.default_rng(100 + seed)
    tok = rng.integers(0, w.V + 1, size=(len(kv_lens), R))       # includes the mask row V
    x = w.embed[tok].astype(np.float64)
    ref = _torch_forward(w, kp, vp, st, x, n_causal, n_mask)
    m = om.OracleModel(w, kp, vp)
    got = m.forward(x, st, n_causal, n_mask)
    np.testing.assert_allclose(got, ref, rtol=0, atol=1e-12 * np.abs(ref).max())
    # the forward appended the window K/V at [L, L + R) of every layer's pools
    for l in range(w.n_layers):
        for s, L in enumerate(kv_lens):
            p = st.page_table[s, (L + R - 1) // PAGE]
            assert np.any(m.k_pools[l][p] != kp[l][p])


def test_composition_pin_sees_plausible_mistakes():
    """The comparison above is sharp enough to reject the mistakes it is for:
    each mistaken composition, run through the torch side, misses by far
    more than the tolerance."""
    w = _weights(7)
    st, kp, vp = _state_and_pools(w, 7, [29, 11], 6)
    x = w.embed[np.random.default_rng(7).integers(0, w.V + 1, size=(2, 6))].astype(np.float64)
    good = om.OracleModel(w, kp, vp).forward(x, st.copy(), 3, 3)
    tol = 1e-12 * np.abs(good).max()
    import copy
    # g_mlp used for g_attn
    w1 = copy.copy(w); w1.g_attn = w.g_mlp
    # final norm gain dropped
    w2 = copy.copy(w); w2.g_final = np.ones_like(w.g_final)
    for bad in (w1, w2):
        assert np.abs(_torch_forward(bad, kp, vp, st, x, 3, 3) - good).max() > 1e3 * tol
    for mistake in ("residual_after_norm", "lm_head_unnormed"):
        bad = _torch_forward(w, kp, vp, st, x, 3, 3, mistake=mistake)
        assert np.abs(bad - good).max() > 1e3 * tol, mistake
    # mask rows attending causally (as if n_causal = R) changes the mask rows only
    bad = _torch_forward(w, kp, vp, st, x, 6, 0)
    np.testing.assert_allclose(bad[:, :3], good[:, :3], rtol=0, atol=tol)
    assert np.abs(bad[:, 3:] - good[:, 3:]).max() > 1e3 * tol


@pytest.mark.parametrize("seed,P,B", [(11, 9, 4), (12, 21, 3)])
def test_prefill_boundary_is_causal_prefix_top1(seed, P, B):
    w = _weights(seed)
    S = 2
    rows = P + 2 * B
    rng = np.random.default_rng(seed)
    st = synth.make_paged_state(rng, np.zeros(S, np.int64), rows, max_pages=16, scatter=True,
                                slack=0.3, n_causal=B, max_new=64)
    kp = [np.zeros((st.pool_pages, w.Hkv, PAGE, w.D)) for _ in range(w.n_layers)]
    vp = [np.zeros((st.pool_pages, w.Hkv, w.D, PAGE)) for _ in range(w.n_layers)]
    x = rng.standard_normal((S, P, w.H))
    # causal-only forward of the prefix alone, by the independent composition
    causal = _torch_forward(w, kp, vp, st, x, P, 0)
    m = om.OracleModel(w, kp, vp)
    ps = st.copy()
    logits = m.prefill(ps, x, B)
    # mask rows appended after the prefix leave the prefix rows' logits unchanged
    np.testing.assert_allclose(logits[:, :P], causal, rtol=0, atol=1e-12 * np.abs(causal).max())
    np.testing.assert_array_equal(ps.boundary, od.top1_rows(causal)[:, P - 1])
    np.testing.assert_array_equal(ps.kv_len, [P] * S)
    for s in range(S):
        assert ps.out_count[s] == 1 and ps.out_tokens[s, 0] == ps.boundary[s]
    # the first draft: top-1 of the mask rows of the (P, B) forward
    xm = np.concatenate([x, np.broadcast_to(w.embed[w.V], (S, B, w.H))], axis=1)
    full = _torch_forward(w, kp, vp, st, xm, P, B)
    np.testing.assert_array_equal(ps.draft, od.top1_rows(full)[:, P:P + ps.draft.shape[1]])
