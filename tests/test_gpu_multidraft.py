"""GPU: the per-acceptance multi-draft step (grouped-mask attention and
multidraft_step) against the oracle.

Mask rows in B groups of B rows; group k sits after d_k, sees the cache, the
causal rows 0..k and itself, and supplies the next draft when A = k (the
structured-mask AR-diffusion hybrid of the paper's related work, applied to
the fused step).  Tolerances as the other parity tests: attention 2e-2 (bf16)
and 1e-5 (fp32) max relative error per output vector, fp32 model logits 1e-4
of the row's largest logit; integers bit for bit.
"""
import copy

import numpy as np
import pytest
import torch

from oracle import attention as oa
from oracle import decode as od
from oracle.model import OracleModel
from paper_2609_26638_amd import dvs, synth
from tests.gpu_util import dev_attn, max_rel_err, to_f64

pytestmark = pytest.mark.gpu

TOL = {"bf16": 2e-2, "f32": 1e-5}
LOGIT_TOL_F32 = 1e-4

ATTN_CASES = [
    # name, seed, S, L, n_causal, n_mask, group, Hq, Hkv, D, dtype, chunk
    ("aligned_b4", 71, 2, [100, 300], 4, 16, 4, 16, 4, 128, "bf16", 256),
    ("balanced_b4", 72, 3, [0, 77, 700], 4, 16, 4, 16, 4, 128, "bf16", 0),
    ("producer_consumer_b8", 73, 2, [900, 2100], 8, 64, 8, 16, 4, 128, "bf16", 0),
    ("d96_b3", 74, 2, [40, 500], 3, 9, 3, 16, 4, 96, "bf16", 64),
    ("fp32_b3", 75, 2, [17, 100], 3, 9, 3, 8, 2, 64, "f32", 0),
    ("two_groups_of_five", 76, 2, [30, 130], 6, 10, 5, 8, 2, 64, "bf16", 128),
]


@pytest.mark.parametrize("case", ATTN_CASES, ids=[c[0] for c in ATTN_CASES])
def test_grouped_attention_matches_oracle(case):
    name, seed, S, L, nc, nm, grp, Hq, Hkv, D, dt, chunk = case
    print(f"[grouped attn] {name}", flush=True)
    ai = synth.make_attn_inputs(seed, S, L, nc, nm, Hq, Hkv, D, dt, std=1.0, scatter=True)
    d = dev_attn(ai)
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    out = dvs.attn_hybrid_block_grouped(d["q"], d["k_new"], d["v_new"], d["k_pool"], d["v_pool"],
                                        d["page_table"], d["kv_len"], nc, nm, grp, ai.scale,
                                        err=err, chunk_keys=chunk)
    torch.cuda.synchronize()
    kp, vp = ai.as_f64("k_pool"), ai.as_f64("v_pool")
    ref = oa.attn_hybrid_block(ai.as_f64("q"), ai.as_f64("k_new"), ai.as_f64("v_new"), kp, vp,
                               ai.state.page_table, ai.state.kv_len, nc, nm, ai.scale, group=grp)
    e = max_rel_err(to_f64(out), ref)
    print(f"[err] {name}: max rel err {e:.3e}", flush=True)
    assert e <= TOL[dt] and int(err.item()) == 0
    np.testing.assert_array_equal(to_f64(d["k_pool"]), kp)
    np.testing.assert_array_equal(to_f64(d["v_pool"]), vp)


def _fp32_model(seed, B, L=(256,), n_layers=1, ffn=0):
    w = synth.make_model_weights(seed, 1024, 256, 4, 4, 64, n_layers, ffn, std=0.02)
    ai = synth.make_attn_inputs(seed, len(L), list(L), B, B * B, 4, 4, 64, "f32", std=0.02,
                                scatter=True, extra_pages=16)
    kps, vps = [ai.k_pool], [ai.v_pool]
    for l in range(1, n_layers):
        o = synth.make_attn_inputs(seed + 10 * l, len(L), list(L), B, B * B, 4, 4, 64, "f32",
                                   std=0.02, scatter=True, extra_pages=16)
        kps.append(o.k_pool)
        vps.append(o.v_pool)
    host = ai.state.copy()
    rng = np.random.default_rng(seed)
    host.boundary[:] = rng.integers(0, w.V, size=len(L))
    host.draft[:] = rng.integers(0, w.V, size=host.draft.shape)
    host.out_tokens = np.full((len(L), 64), -1, np.int32)
    return w, kps, vps, host


def test_tiny_fp32_multidraft_steps_match_oracle():
    """Three steps of the fp32 single-layer model (L = 256, 4 heads x 64,
    B = 4, so 4 + 16 window rows): logits within 1e-4 of the oracle's from
    the same state, and the integer stages (top-1, A, commit with the next
    draft from group A) replayed through the oracle bit for bit.  The second
    step's draft has its first token right and its second wrong, so A = 1
    and the next draft is group 1's."""
    B = 4
    w, kps, vps, host = _fp32_model(0, B, L=(256, 97))
    S, R = 2, B + B * B
    om = OracleModel(w, [k.copy() for k in kps], [v.copy() for v in vps])
    dm = dvs.DeviceModel(w, [torch.from_numpy(k).cuda() for k in kps],
                         [torch.from_numpy(v).cuda() for v in vps], "f32")
    st = dvs.DeviceState(host)
    ref = host.copy()
    logits = torch.empty((S * R, w.V), dtype=torch.float32, device="cuda")
    am = torch.empty((S, R), dtype=torch.int32, device="cuda")
    acc = torch.empty((S,), dtype=torch.int32, device="cuda")
    for step in range(3):
        if step == 1:
            # a_1 = the causal prediction after x0 (an AR step from the same state)
            probe = copy.copy(om)
            probe.k_pools = [a.copy() for a in om.k_pools]
            probe.v_pools = [a.copy() for a in om.v_pools]
            lp = probe.forward(om.embed[ref.boundary[:, None].astype(np.int64)], ref.copy(), 1, 0)
            a1 = od.top1_rows(lp)[:, 0]
            srt = np.sort(lp[:, 0], axis=-1)
            clear = (srt[:, -1] - srt[:, -2]) > 4 * LOGIT_TOL_F32 * np.abs(lp[:, 0]).max(-1)
            ref.draft[:, 0] = a1
            ref.draft[:, 1] = (a1 + 1) % w.V
            st.draft.copy_(torch.from_numpy(ref.draft))
        tok = np.empty((S, R), np.int64)
        tok[:, 0] = ref.boundary
        tok[:, 1:B] = ref.draft[:, :B - 1]
        tok[:, B:] = w.V
        before = ref.copy()
        lref = om.forward(om.embed[tok], before.copy(), B, B * B, group=B)
        dvs.multidraft_step(dm, st, B, chunk_keys=64, logits_out=logits, argmax_out=am,
                            accept_out=acc)
        torch.cuda.synchronize()
        assert int(st.err.item()) == 0
        lg = logits.cpu().numpy().reshape(S, R, w.V).astype(np.float64)
        e = max_rel_err(lg, lref)
        print(f"[multidraft] step {step}: logit max rel err {e:.2e}", flush=True)
        assert e <= LOGIT_TOL_F32
        am_gpu = am.cpu().numpy()
        A = od.accept(am_gpu, before.draft, B)
        np.testing.assert_array_equal(acc.cpu().numpy(), A)
        if step == 1:
            assert all(A[s] == 1 for s in range(S) if clear[s])
        assert od.kv_commit(ref, A, am_gpu, B, B * B, draft_group=B) == 0
        got = st.to_host(ref)
        for f in ("kv_len", "page_table", "num_pages", "boundary", "draft", "out_tokens",
                  "out_count", "finished"):
            np.testing.assert_array_equal(getattr(got, f), getattr(ref, f), err_msg=f)
        assert got.free_top == ref.free_top
        for s in range(S):
            np.testing.assert_array_equal(ref.draft[s], am_gpu[s, B + A[s] * B:B + A[s] * B + B - 1])


def test_group_k_equals_a_fused_call_verifying_k_drafts():
    """On the GPU, group k of a multi-draft step equals the mask rows of a
    fused call with causal rows x0, d_1..d_k from the same state (fp32, two
    layers with an MLP; the two calls place the keys in different slots, so
    they agree to rounding)."""
    B = 4
    w, kps, vps, host = _fp32_model(3, B, L=(300, 40), n_layers=2, ffn=128)
    S, R = 2, B + B * B

    def fresh():
        return dvs.DeviceModel(w, [torch.from_numpy(k).cuda() for k in kps],
                               [torch.from_numpy(v).cuda() for v in vps], "f32")

    full = torch.empty((S * R, w.V), dtype=torch.float32, device="cuda")
    dvs.multidraft_step(fresh(), dvs.DeviceState(host), B, chunk_keys=64, logits_out=full)
    full_np = full.cpu().numpy().reshape(S, R, w.V)
    for k in range(B):
        part = torch.empty((S * (k + 1 + B), w.V), dtype=torch.float32, device="cuda")
        dvs.draft_verify_step(fresh(), dvs.DeviceState(host), k + 1, B, chunk_keys=64,
                              logits_out=part)
        torch.cuda.synchronize()
        p = part.cpu().numpy().reshape(S, k + 1 + B, w.V).astype(np.float64)
        g = full_np[:, B + k * B:B + (k + 1) * B].astype(np.float64)
        assert max_rel_err(g, p[:, k + 1:]) <= LOGIT_TOL_F32, k
        assert max_rel_err(full_np[:, :k + 1].astype(np.float64), p[:, :k + 1]) <= LOGIT_TOL_F32


def _bf16_model(seed, B, L=(37, 300, 129)):
    w = synth.make_model_weights(seed, 512, 256, 4, 2, 64, 2, 512, std=0.08)
    base = synth.make_attn_inputs(seed, len(L), list(L), B, B * B, 4, 2, 64, "bf16", std=0.5,
                                  scatter=True, extra_pages=64)
    other = synth.make_attn_inputs(seed + 100, len(L), list(L), B, B * B, 4, 2, 64, "bf16",
                                   std=0.5, scatter=True, extra_pages=64)
    host = base.state.copy()
    host.out_tokens = np.full((len(L), 256), -1, np.int32)
    rng = np.random.default_rng(seed)
    host.boundary[:] = rng.integers(0, w.V, size=len(L))
    host.draft[:] = rng.integers(0, w.V, size=host.draft.shape)

    def fresh():
        pools = lambda arrs: [torch.from_numpy(np.ascontiguousarray(a).view(np.int16))
                              .view(torch.bfloat16).cuda() for a in arrs]
        return dvs.DeviceModel(w, pools([base.k_pool, other.k_pool]),
                               pools([base.v_pool, other.v_pool]), "bf16")
    return w, host, fresh


def test_b1_multidraft_is_the_fused_step_bit_for_bit():
    w, host, fresh = _bf16_model(8, 1)
    S = host.kv_len.shape[0]
    a_m, a_st = fresh(), dvs.DeviceState(host)
    b_m, b_st = fresh(), dvs.DeviceState(host)
    la = torch.empty((S * 2, w.V), dtype=torch.float32, device="cuda")
    lb = torch.empty_like(la)
    for _ in range(5):
        dvs.multidraft_step(a_m, a_st, 1, chunk_keys=64, logits_out=la)
        dvs.draft_verify_step(b_m, b_st, 1, 1, chunk_keys=64, logits_out=lb)
        torch.cuda.synchronize()
        assert torch.equal(la, lb)
    ha, hb = a_st.to_host(host), b_st.to_host(host)
    for f in ("kv_len", "page_table", "boundary", "draft", "out_tokens", "out_count"):
        np.testing.assert_array_equal(getattr(ha, f), getattr(hb, f), err_msg=f)


@pytest.mark.parametrize("B", [3, 4])
def test_multidraft_stream_equals_greedy_ar_on_gpu(B):
    """bf16, two layers: the committed stream of multi-draft steps equals
    greedy AR bit for bit; the first draft is the AR continuation, so the
    first step accepts every draft."""
    N = 40
    w, host, fresh = _bf16_model(9, B)
    S = host.kv_len.shape[0]
    ar_st = dvs.DeviceState(host)
    ar_m = fresh()
    for _ in range(N):
        dvs.draft_verify_step(ar_m, ar_st, 1, 0, chunk_keys=64)
    torch.cuda.synchronize()
    ar = ar_st.to_host(host)
    ss_host = host.copy()
    ss_host.draft[:] = ar.out_tokens[:, :B - 1]
    st, m = dvs.DeviceState(ss_host), fresh()
    acc = torch.empty((S,), dtype=torch.int32, device="cuda")
    dvs.multidraft_step(m, st, B, chunk_keys=64, accept_out=acc)
    torch.cuda.synchronize()
    assert acc.cpu().numpy().tolist() == [B - 1] * S
    steps = 1
    while int(st.out_count.min().item()) < N:
        dvs.multidraft_step(m, st, B, chunk_keys=64)
        steps += 1
        assert steps < 10 * N
    torch.cuda.synchronize()
    assert int(st.err.item()) == 0
    ss = st.to_host(ss_host)
    for s in range(S):
        n = min(int(ss.out_count[s]), int(ar.out_count[s]))
        assert n >= N
        np.testing.assert_array_equal(ss.out_tokens[s, :n], ar.out_tokens[s, :n])
