"""GPU: draft_verify_step (decoder layers + hot path) against the oracle, and
GPU self-speculative decoding == GPU greedy AR decoding, token for token."""
import numpy as np
import pytest
import torch

from oracle import decode as od
from oracle.model import OracleModel
from paper_2609_26638_amd import dvs, synth
from tests.gpu_util import max_rel_err

pytestmark = pytest.mark.gpu

# fp32 logits vs the float64 oracle: a handful of fp32 roundings per layer on
# O(1)-normalised activations; 1e-4 of the row's largest logit is ~100x the
# expected error.
LOGIT_TOL_F32 = 1e-4


def _states_equal(dev, host, fields=("kv_len", "page_table", "num_pages", "boundary", "draft",
                                     "out_tokens", "out_count", "finished")):
    got = dev.to_host(host)
    for f in fields:
        np.testing.assert_array_equal(getattr(got, f), getattr(host, f), err_msg=f)
    assert got.free_top == host.free_top


def test_tiny_fp32_single_layer_step_matches_oracle():
    w, ai = synth.tiny_step_inputs(0)
    B, V = ai.n_causal, w.V
    om = OracleModel(w, [ai.k_pool], [ai.v_pool])
    st_ref = ai.state.copy()
    logits_ref, am_ref, A_ref, err = om.fused_step(st_ref, B)
    assert err == 0
    dm = dvs.DeviceModel(w, [ai.k_pool], [ai.v_pool], "f32")
    st = dvs.DeviceState(ai.state)
    logits = torch.empty((2 * B, V), dtype=torch.float32, device="cuda")
    am = torch.empty((1, 2 * B), dtype=torch.int32, device="cuda")
    acc = torch.empty((1,), dtype=torch.int32, device="cuda")
    dvs.draft_verify_step(dm, st, B, B, logits_out=logits, argmax_out=am, accept_out=acc)
    torch.cuda.synchronize()
    assert int(st.err.item()) == 0
    lg = logits.cpu().numpy().reshape(1, 2 * B, V)
    assert max_rel_err(lg.astype(np.float64), logits_ref) <= LOGIT_TOL_F32
    # replay: the integer stages on the GPU's own logits are bit-exact
    am_gpu = am.cpu().numpy()
    np.testing.assert_array_equal(am_gpu, od.top1_rows(lg.astype(np.float64)))
    A_gpu = od.accept(am_gpu, ai.state.draft, B)
    np.testing.assert_array_equal(acc.cpu().numpy(), A_gpu)
    replay = ai.state.copy()
    assert od.kv_commit(replay, A_gpu, am_gpu, B, B) == 0
    _states_equal(st, replay)
    # and the tokens equal the float64 oracle's wherever its top-2 margin is
    # above the logit tolerance
    srt = np.sort(logits_ref, axis=-1)
    margin = srt[..., -1] - srt[..., -2]
    scale = np.abs(logits_ref).max(axis=-1)
    clear = margin > 4 * LOGIT_TOL_F32 * scale
    assert np.array_equal(am_gpu[clear], am_ref[clear])
    # the appended window K/V (first layer's pools) agree with the oracle
    kp = dm.k_pools[0].cpu().numpy()
    np.testing.assert_allclose(kp, om.k_pools[0], rtol=1e-4, atol=1e-6)


def _small_model(seed, dtype, n_layers=2, ffn=512, L=(37, 300, 129), std=0.08):
    w = synth.make_model_weights(seed, 512, 256, 4, 2, 64, n_layers, ffn, std=std)
    S = len(L)
    base = synth.make_attn_inputs(seed, S, list(L), 8, 8, 4, 2, 64, dtype, std=0.5,
                                  scatter=True, extra_pages=64)
    kps, vps = [base.k_pool], [base.v_pool]
    for l in range(1, n_layers):
        other = synth.make_attn_inputs(seed + 100 * l, S, list(L), 8, 8, 4, 2, 64, dtype, std=0.5,
                                       scatter=True, extra_pages=64)
        kps.append(other.k_pool)
        vps.append(other.v_pool)
    return w, base, kps, vps


def _dev_pools(arrs, dtype):
    out = []
    for a in arrs:
        if dtype == "bf16":
            out.append(torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda())
        else:
            out.append(torch.from_numpy(np.ascontiguousarray(a)).cuda())
    return out


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_selfspec_equals_greedy_ar_on_gpu(dtype):
    """Committed streams of fused self-speculative steps equal greedy AR steps,
    bit for bit (the paper's AR-equivalence argument, on the GPU's own
    arithmetic: rows never depend on the other rows of the call)."""
    B, N, CH = 8, 40, 64
    w, base, kps, vps = _small_model(3, dtype)
    S = base.S
    host = base.state.copy()
    host.out_tokens = np.full((S, 256), -1, np.int32)
    rng = np.random.default_rng(1)
    host.boundary[:] = rng.integers(0, w.V, size=S)
    host.draft[:] = rng.integers(0, w.V, size=(S, B - 1))

    # greedy AR
    ar_m = dvs.DeviceModel(w, _dev_pools(kps, dtype), _dev_pools(vps, dtype), dtype)
    ar_st = dvs.DeviceState(host)
    for _ in range(N):
        dvs.draft_verify_step(ar_m, ar_st, 1, 0, chunk_keys=CH)
    torch.cuda.synchronize()
    assert int(ar_st.err.item()) == 0
    ar = ar_st.to_host(host)

    # self-speculative, first draft = the AR continuation (fully accepted)
    ss_host = host.copy()
    ss_host.draft[:] = ar.out_tokens[:, :B - 1]
    ss_m = dvs.DeviceModel(w, _dev_pools(kps, dtype), _dev_pools(vps, dtype), dtype)
    ss_st = dvs.DeviceState(ss_host)
    acc = torch.empty((S,), dtype=torch.int32, device="cuda")
    dvs.draft_verify_step(ss_m, ss_st, B, B, chunk_keys=CH, accept_out=acc)
    torch.cuda.synchronize()
    assert acc.cpu().numpy().tolist() == [B - 1] * S
    steps = 1
    while int(ss_st.out_count.min().item()) < N:
        dvs.draft_verify_step(ss_m, ss_st, B, B, chunk_keys=CH)
        steps += 1
        assert steps < 10 * N
    torch.cuda.synchronize()
    assert int(ss_st.err.item()) == 0
    ss = ss_st.to_host(ss_host)
    for s in range(S):
        n = min(int(ss.out_count[s]), int(ar.out_count[s]))
        assert n >= N
        np.testing.assert_array_equal(ss.out_tokens[s, :n], ar.out_tokens[s, :n])
    assert steps < N   # the full-acceptance first step already saved B-1 steps


def test_bf16_model_step_matches_oracle_replay():
    """Multi-layer bf16 step: logits close to the float64 oracle, integer
    stages bit-exact when replayed on the GPU's logits."""
    B = 8
    w, base, kps, vps = _small_model(5, "bf16")
    st_host = base.state.copy()
    rng = np.random.default_rng(2)
    st_host.boundary[:] = rng.integers(0, w.V, size=base.S)
    st_host.draft[:] = rng.integers(0, w.V, size=(base.S, B - 1))
    wb = synth.ModelWeights(**{**w.__dict__})
    for name in ("embed", "g_final", "lm_head"):
        setattr(wb, name, synth.f32_to_bf16_bits(getattr(w, name)))
    for name in ("wq", "wk", "wv", "wo", "g_attn", "g_mlp", "w_gate", "w_up", "w_down"):
        setattr(wb, name, [synth.f32_to_bf16_bits(a) for a in getattr(w, name)])
    om = OracleModel(wb, kps, vps, bf16_bits=True)
    ref_st = st_host.copy()
    logits_ref, am_ref, A_ref, err = om.fused_step(ref_st, B)
    dm = dvs.DeviceModel(w, _dev_pools(kps, "bf16"), _dev_pools(vps, "bf16"), "bf16")
    st = dvs.DeviceState(st_host)
    M = base.S * 2 * B
    logits = torch.empty((M, w.V), dtype=torch.float32, device="cuda")
    am = torch.empty((base.S, 2 * B), dtype=torch.int32, device="cuda")
    dvs.draft_verify_step(dm, st, B, B, logits_out=logits, argmax_out=am)
    torch.cuda.synchronize()
    lg = logits.cpu().numpy().reshape(base.S, 2 * B, w.V).astype(np.float64)
    # bf16 activations between the layers: relative logit error of a few 1e-3
    assert max_rel_err(lg, logits_ref) <= 5e-2
    am_gpu = am.cpu().numpy()
    np.testing.assert_array_equal(am_gpu, od.top1_rows(lg))
    replay = st_host.copy()
    A_gpu = od.accept(am_gpu, st_host.draft, B)
    assert od.kv_commit(replay, A_gpu, am_gpu, B, B) == 0
    _states_equal(st, replay)
