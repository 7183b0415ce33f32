"""GPU: draft_verify_step (decoder layers + hot path) against the oracle, and
GPU self-speculative decoding == GPU greedy AR decoding, token for token;
the same for the paper's two-forward round (literal_round)."""
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


def _widen_draft(host, width):
    """The two-forward round keeps d_1..d_B in the draft array: width >= B."""
    h = host.copy()
    d = np.zeros((h.draft.shape[0], width), np.int32)
    d[:, :h.draft.shape[1]] = h.draft
    h.draft = d
    return h


def test_tiny_fp32_literal_round_matches_oracle():
    w, ai = synth.tiny_step_inputs(0)
    B, V = ai.n_causal, w.V
    host = _widen_draft(ai.state, B)
    om = OracleModel(w, [ai.k_pool], [ai.v_pool])
    st_ref = host.copy()
    lg_d, lg_v, am_v, A_ref, err = om.literal_round(st_ref, B)
    assert err == 0
    dm = dvs.DeviceModel(w, [ai.k_pool], [ai.v_pool], "f32")
    st = dvs.DeviceState(host)
    logits = torch.empty((B + 1, V), dtype=torch.float32, device="cuda")
    am = torch.empty((1, B + 1), dtype=torch.int32, device="cuda")
    acc = torch.empty((1,), dtype=torch.int32, device="cuda")
    dvs.literal_round(dm, st, B, logits_out=logits, argmax_out=am, accept_out=acc)
    torch.cuda.synchronize()
    assert int(st.err.item()) == 0
    got = st.to_host(host)
    # draft forward: the GPU's a0 and d_1..d_B are the oracle's (every top-2
    # margin of these rows is far above the fp32 logit error for this seed)
    srt = np.sort(lg_d, axis=-1)
    assert np.all(srt[..., -1] - srt[..., -2] > 4 * LOGIT_TOL_F32 * np.abs(lg_d).max(axis=-1))
    np.testing.assert_array_equal(got.draft[:, :B], st_ref.draft[:, :B])
    a0 = got.out_tokens[:, host.out_count[0]]
    np.testing.assert_array_equal(a0, st_ref.out_tokens[:, host.out_count[0]])
    # verify forward on the same window: logits within the fp32 tolerance
    lg = logits.cpu().numpy().reshape(1, B + 1, V)
    assert max_rel_err(lg.astype(np.float64), lg_v) <= LOGIT_TOL_F32
    # replay: acceptance and the round's commit on the GPU's own top-1 are
    # bit-exact, and so is the resulting state
    am_gpu = am.cpu().numpy()
    np.testing.assert_array_equal(am_gpu, od.top1_rows(lg.astype(np.float64)))
    replay = host.copy()
    replay.draft[:, :B] = got.draft[:, :B]
    replay.kv_len += 1
    A_gpu = od.accept(am_gpu, replay.draft, B + 1)
    np.testing.assert_array_equal(acc.cpu().numpy(), A_gpu)
    assert od.kv_commit(replay, A_gpu, am_gpu, B + 1, 0, lead=a0, window=B + 2) == 0
    _states_equal(st, replay)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_literal_round_equals_greedy_ar_on_gpu(dtype):
    """The paper's two-forward round commits a0, d_1..d_A, a_{A+1} per round;
    its committed stream equals greedy AR bit for bit on the GPU."""
    B, N, CH = 8, 40, 64
    w, base, kps, vps = _small_model(4, dtype)
    S = base.S
    host = _widen_draft(base.state, B)
    host.out_tokens = np.full((S, 256), -1, np.int32)
    rng = np.random.default_rng(2)
    host.boundary[:] = rng.integers(0, w.V, size=S)
    ar_m = dvs.DeviceModel(w, _dev_pools(kps, dtype), _dev_pools(vps, dtype), dtype)
    ar_st = dvs.DeviceState(host)
    for _ in range(N):
        dvs.draft_verify_step(ar_m, ar_st, 1, 0, chunk_keys=CH)
    torch.cuda.synchronize()
    assert int(ar_st.err.item()) == 0
    ar = ar_st.to_host(host)
    lr_m = dvs.DeviceModel(w, _dev_pools(kps, dtype), _dev_pools(vps, dtype), dtype)
    lr_st = dvs.DeviceState(host)
    acc = torch.empty((S,), dtype=torch.int32, device="cuda")
    rounds = 0
    while int(lr_st.out_count.min().item()) < N:
        before = lr_st.out_count.clone()
        dvs.literal_round(lr_m, lr_st, B, chunk_keys=CH, accept_out=acc)
        rounds += 1
        # each round commits a0, the accepted drafts and a_{A+1}: A + 2 tokens
        assert torch.equal(lr_st.out_count - before, acc + 2)
        assert rounds <= N
    torch.cuda.synchronize()
    assert int(lr_st.err.item()) == 0
    lr = lr_st.to_host(host)
    for s in range(S):
        n = min(int(lr.out_count[s]), int(ar.out_count[s]))
        assert n >= N
        np.testing.assert_array_equal(lr.out_tokens[s, :n], ar.out_tokens[s, :n])
        # every committed token but the boundary holds KV
        assert lr.kv_len[s] - lr.out_count[s] == host.kv_len[s] - host.out_count[s]


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


def test_bf16_wide_step_matches_oracle_replay():
    """A one-layer bf16 step at 256 window rows (8 sequences, B=16) whose
    projections take the wide decode-step GEMM paths: Q|K|V of 32/4 heads of
    64 (80 column blocks: the row-split 2x2 kernel with the rotary epilogue),
    SwiGLU 2192 (137 gate|up blocks: the block-split 2x2 kernel, the last
    pair half empty) and vocabulary 8200 (257 blocks: the column-split LM
    head, the last block 8 columns wide). Logits close to the float64
    oracle; the top-1 of the fused LM-head epilogue equals the top-1 of the
    logits; accept and commit replayed through the oracle bit for bit."""
    B, S = 16, 8
    L = [41, 77, 130, 199, 256, 301, 350, 397]
    w = synth.make_model_weights(11, 8200, 256, 32, 4, 64, 1, 2192, std=0.08)
    base = synth.make_attn_inputs(11, S, L, B, B, 32, 4, 64, "bf16", std=0.5, scatter=True,
                                  extra_pages=64)
    kps, vps = [base.k_pool], [base.v_pool]
    st_host = base.state.copy()
    rng = np.random.default_rng(3)
    st_host.boundary[:] = rng.integers(0, w.V, size=S)
    st_host.draft[:] = rng.integers(0, w.V, size=(S, B - 1))
    om = OracleModel(_bf16_weights(w), kps, vps, bf16_bits=True)
    ref_st = st_host.copy()
    logits_ref, _, _, _ = om.fused_step(ref_st, B)
    dm = dvs.DeviceModel(w, _dev_pools(kps, "bf16"), _dev_pools(vps, "bf16"), "bf16")
    M = S * 2 * B
    # with the logits written out (fp32 epilogue), then with the fused top-1
    st = dvs.DeviceState(st_host)
    logits = torch.empty((M, w.V), dtype=torch.float32, device="cuda")
    am = torch.empty((S, 2 * B), dtype=torch.int32, device="cuda")
    dvs.draft_verify_step(dm, st, B, B, logits_out=logits, argmax_out=am, chunk_keys=256)
    st2 = dvs.DeviceState(st_host)
    am2 = torch.empty((S, 2 * B), dtype=torch.int32, device="cuda")
    dvs.draft_verify_step(dm, st2, B, B, argmax_out=am2, chunk_keys=256)
    torch.cuda.synchronize()
    lg = logits.cpu().numpy().reshape(S, 2 * B, w.V).astype(np.float64)
    assert max_rel_err(lg, logits_ref) <= 5e-2
    am_gpu = am.cpu().numpy()
    np.testing.assert_array_equal(am_gpu, od.top1_rows(lg))
    np.testing.assert_array_equal(am2.cpu().numpy(), am_gpu)
    replay = st_host.copy()
    A_gpu = od.accept(am_gpu, st_host.draft, B)
    assert od.kv_commit(replay, A_gpu, am_gpu, B, B) == 0
    _states_equal(st, replay)
    _states_equal(st2, replay)


@pytest.mark.parametrize("S", [8, 5, 3, 1, 12, 20])
def test_bf16_ar_steps_match_oracle_replay(S):
    """Greedy AR steps of a two-layer bf16 model (one row per sequence)
    through the few-row decode GEMM paths: Q|K|V of 32/4 heads of 64 in
    16-column blocks with the rotary epilogue, the O and down projections in
    8-column blocks, only the first rows of A copied per chunk, gate|up with
    SwiGLU, and the LM head (vocabulary 8200, 257 blocks, the last 8 columns
    wide) with its fused top-1. Three steps in a row: logits close to the
    float64 oracle on the same state; the top-1 of the fused LM-head
    epilogue equals the top-1 of the logits; the commit replayed through the
    oracle bit for bit, which also keeps both sides on the same state.
    12 and 20 sequences: the whole-line launches copy every row of A (the
    LM head still only the first 16 at 12); 20 rows, no first-rows copies."""
    L = ([41, 77, 130, 199, 256, 301, 350, 397] + [60 + 37 * i for i in range(12)])[:S]
    w = synth.make_model_weights(13, 8200, 256, 32, 4, 64, 2, 2304, std=0.08)
    pools = [synth.make_attn_inputs(13 + 100 * l, S, L, 16, 16, 32, 4, 64, "bf16", std=0.5,
                                    scatter=True, extra_pages=64) for l in range(2)]
    kps, vps = [p.k_pool for p in pools], [p.v_pool for p in pools]
    st_host = pools[0].state.copy()
    st_host.boundary[:] = np.random.default_rng(4).integers(0, w.V, size=S)
    om = OracleModel(_bf16_weights(w), kps, vps, bf16_bits=True)
    dm = dvs.DeviceModel(w, _dev_pools(kps, "bf16"), _dev_pools(vps, "bf16"), "bf16")
    st = dvs.DeviceState(st_host)
    st2 = dvs.DeviceState(st_host)
    ref = st_host.copy()
    for step in range(3):
        logits_ref, _, err = om.ar_step(ref)
        assert err == 0
        logits = torch.empty((S, w.V), dtype=torch.float32, device="cuda")
        am = torch.empty((S, 1), dtype=torch.int32, device="cuda")
        am2 = torch.empty((S, 1), dtype=torch.int32, device="cuda")
        before = st.to_host(st_host)
        dvs.draft_verify_step(dm, st, 1, 0, logits_out=logits, argmax_out=am, chunk_keys=256)
        dvs.draft_verify_step(dm, st2, 1, 0, argmax_out=am2, chunk_keys=256)
        torch.cuda.synchronize()
        lg = logits.cpu().numpy().reshape(S, 1, w.V).astype(np.float64)
        assert max_rel_err(lg, logits_ref) <= 5e-2, step
        am_gpu = am.cpu().numpy()
        np.testing.assert_array_equal(am_gpu, od.top1_rows(lg))
        np.testing.assert_array_equal(am2.cpu().numpy(), am_gpu)
        # the oracle's own commit used its top-1; replay the GPU's on the
        # state before the step, and carry the oracle on with that state
        replay = before.copy()
        assert od.kv_commit(replay, np.zeros(S, dtype=np.int32), am_gpu, 1, 0) == 0
        _states_equal(st, replay)
        _states_equal(st2, replay)
        ref = replay


def _embed_prefix_f64(w_bits, vision, prompt):
    """Oracle-side prefix rows: vision vectors, then embedding rows of the prompt."""
    emb = synth.bf16_to_f64(w_bits.embed)
    return np.concatenate([vision.astype(np.float64), emb[prompt]], axis=1)


def _bf16_weights(w):
    wb = synth.ModelWeights(**{**w.__dict__})
    for name in ("embed", "g_final", "lm_head"):
        setattr(wb, name, synth.f32_to_bf16_bits(getattr(w, name)))
    for name in ("wq", "wk", "wv", "wo", "g_attn", "g_mlp", "w_gate", "w_up", "w_down"):
        setattr(wb, name, [synth.f32_to_bf16_bits(a) for a in getattr(w, name)])
    return wb


def test_prefill_matches_oracle_small():
    B = 8
    si = synth.decoder_stack_inputs(seed=9, S=3, n_layers=2, H=256, Hq=4, Hkv=2, D=64, ffn=512,
                                    V=512, n_vision=24, n_prompt=16, B=B, max_new=64)
    P, S, H = si.P, 3, 256
    w = si.weights
    pool = si.state.pool_pages
    kps = [np.zeros((pool, 2, 16, 64), np.uint16) for _ in range(2)]
    vps = [np.zeros((pool, 2, 64, 16), np.uint16) for _ in range(2)]
    wb = _bf16_weights(w)
    om = OracleModel(wb, kps, vps, bf16_bits=True)
    ref = si.state.copy()
    logits_ref = om.prefill(ref, _embed_prefix_f64(wb, si.vision, si.prompt), B)
    dm = dvs.DeviceModel(w, _dev_pools(kps, "bf16"), _dev_pools(vps, "bf16"), "bf16")
    st = dvs.DeviceState(si.state)
    lg = torch.empty((S * (B + 1), w.V), dtype=torch.float32, device="cuda")
    dvs.prefill(dm, st, P, B, prefix_tokens=torch.from_numpy(si.prefix_tokens()).cuda(),
                x_prefix=torch.from_numpy(si.x_prefix()).cuda(), logits_out=lg)
    torch.cuda.synchronize()
    assert int(st.err.item()) == 0
    got = lg.cpu().numpy().reshape(S, B + 1, w.V).astype(np.float64)
    assert max_rel_err(got, logits_ref[:, P - 1:P + B]) <= 5e-2
    am = od.top1_rows(got)
    host = st.to_host(si.state)
    np.testing.assert_array_equal(host.kv_len, [P] * S)
    np.testing.assert_array_equal(host.boundary, am[:, 0])
    np.testing.assert_array_equal(host.draft, am[:, 1:B])
    np.testing.assert_array_equal(host.out_tokens[:, 0], am[:, 0])
    np.testing.assert_array_equal(host.out_count, [1] * S)
    # the prefix KV written by the GPU equals the oracle's within bf16 rounding
    kp0 = synth.bf16_to_f64(dm.k_pools[0].cpu().view(torch.int16).numpy().view(np.uint16))
    for s in range(S):
        pages = si.state.page_table[s, :(P + 15) // 16]
        a = kp0[pages].transpose(0, 2, 1, 3).reshape(-1, 2, 64)[:P]
        b = om.k_pools[0][pages].transpose(0, 2, 1, 3).reshape(-1, 2, 64)[:P]
        assert max_rel_err(a, b) <= 3e-2
    # a step after the prefill, on the workspace the prefill laid out
    # differently, equals the same step on a fresh workspace, bit for bit
    st2 = dvs.DeviceState(st.to_host(si.state))
    pools2 = ([k.clone() for k in dm.k_pools], [v.clone() for v in dm.v_pools])
    lg_a = torch.empty((S * 2 * B, w.V), dtype=torch.float32, device="cuda")
    dvs.draft_verify_step(dm, st, B, B, logits_out=lg_a)
    dm2 = dvs.DeviceModel(w, pools2[0], pools2[1], "bf16")
    lg_b = torch.empty_like(lg_a)
    dvs.draft_verify_step(dm2, st2, B, B, logits_out=lg_b)
    torch.cuda.synchronize()
    assert int(st.err.item()) == 0 and int(st2.err.item()) == 0
    assert torch.equal(lg_a, lg_b)


def _run_stack(si, dtype, mode, chunk):
    """prefill then AR (mode 'ar'), fused steps ('fused') or two-forward rounds
    ('literal') until max_new tokens; returns the host state, the number of
    steps and the device seconds of the loop."""
    w = si.weights
    pool = si.state.pool_pages
    L = w.n_layers
    kps = [torch.zeros((pool, w.Hkv, 16, w.D), dtype=torch.bfloat16, device="cuda") for _ in range(L)]
    vps = [torch.zeros((pool, w.Hkv, w.D, 16), dtype=torch.bfloat16, device="cuda") for _ in range(L)]
    dm = dvs.DeviceModel(w, kps, vps, dtype)
    host = _widen_draft(si.state, si.B) if mode == "literal" else si.state
    st = dvs.DeviceState(host)
    dvs.prefill(dm, st, si.P, si.B, prefix_tokens=torch.from_numpy(si.prefix_tokens()).cuda(),
                x_prefix=torch.from_numpy(si.x_prefix()).cuda(), chunk_keys=chunk)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    steps = 0
    while True:
        for _ in range(16):
            if mode == "ar":
                dvs.draft_verify_step(dm, st, 1, 0, chunk_keys=chunk)
            elif mode == "literal":
                dvs.literal_round(dm, st, si.B, chunk_keys=chunk)
            else:
                dvs.draft_verify_step(dm, st, si.B, si.B, chunk_keys=chunk)
            steps += 1
        if int(st.finished.min().item()) == 1 or steps > 4 * si.max_new:
            break
    e1.record()
    torch.cuda.synchronize()
    assert int(st.err.item()) == 0
    return st.to_host(host), steps, e0.elapsed_time(e1) / 1e3


def test_decoder_stack_selfspec_equals_ar():
    """The 16-layer bf16 stack (hidden 1536, 16/4 heads, head_dim 96, SwiGLU
    4096, vocab 65536), 8 sequences with 1024 vision embeddings + 64 prompt
    tokens, B=16, decoded to 1024 tokens: the self-speculative stream equals
    greedy AR token for token."""
    print("[stack] generating the 16-layer stack", flush=True)
    si = synth.decoder_stack_inputs()
    ar, ar_steps, ar_s = _run_stack(si, "bf16", "ar", 256)
    print(f"[stack] AR {ar_steps} steps {ar_s:.2f} s", flush=True)
    ss, ss_steps, ss_s = _run_stack(si, "bf16", "fused", 256)
    print(f"[stack] self-spec {ss_steps} steps {ss_s:.2f} s", flush=True)
    np.testing.assert_array_equal(ar.out_count, [si.max_new] * 8)
    np.testing.assert_array_equal(ss.out_count, [si.max_new] * 8)
    np.testing.assert_array_equal(ss.out_tokens, ar.out_tokens)
    lr, lr_rounds, lr_s = _run_stack(si, "bf16", "literal", 256)
    print(f"[stack] two-forward rounds {lr_rounds} rounds {lr_s:.2f} s", flush=True)
    np.testing.assert_array_equal(lr.out_count, [si.max_new] * 8)
    np.testing.assert_array_equal(lr.out_tokens, ar.out_tokens)


def test_decoder_stack_replay_with_ar_drafts():
    """The 16-layer bf16 stack with full acceptances: every third fused step
    the device draft is overwritten with the greedy-AR continuation, so the
    step must accept all B - 1 drafts (A = B - 1) at the stack's own shape.
    Every step's GPU top-1 is replayed through the oracle's accept and commit
    (appendix items Accept and Cache update), which must reproduce the GPU's
    accepted lengths, committed tokens, lengths, page tables and free stack
    bit for bit; the final stream equals greedy AR."""
    print("[stack] generating the 16-layer stack", flush=True)
    si = synth.decoder_stack_inputs()
    ar, _, _ = _run_stack(si, "bf16", "ar", 256)
    print("[stack] AR reference done", flush=True)
    w, B, S = si.weights, si.B, 8
    pool = si.state.pool_pages
    kps = [torch.zeros((pool, w.Hkv, 16, w.D), dtype=torch.bfloat16, device="cuda")
           for _ in range(w.n_layers)]
    vps = [torch.zeros((pool, w.Hkv, w.D, 16), dtype=torch.bfloat16, device="cuda")
           for _ in range(w.n_layers)]
    dm = dvs.DeviceModel(w, kps, vps, "bf16")
    st = dvs.DeviceState(si.state)
    dvs.prefill(dm, st, si.P, B, prefix_tokens=torch.from_numpy(si.prefix_tokens()).cuda(),
                x_prefix=torch.from_numpy(si.x_prefix()).cuda(), chunk_keys=256)
    am = torch.empty((S, 2 * B), dtype=torch.int32, device="cuda")
    acc = torch.empty(S, dtype=torch.int32, device="cuda")
    forced_full = 0
    steps = 0
    while True:
        before = st.to_host(si.state)
        if before.finished.min() == 1:
            break
        forced = steps % 3 == 2
        if forced:
            d = np.zeros((S, B - 1), np.int32)
            for s in range(S):
                c = int(before.out_count[s])
                tail = ar.out_tokens[s, c:c + B - 1]
                d[s, :tail.size] = tail
            st.draft.copy_(torch.from_numpy(d).cuda())
            before.draft = d
        dvs.draft_verify_step(dm, st, B, B, chunk_keys=256, argmax_out=am, accept_out=acc)
        torch.cuda.synchronize()
        assert int(st.err.item()) == 0
        got_am = am.cpu().numpy()
        got_A = acc.cpu().numpy()
        ref_A = od.accept(got_am, before.draft, B)
        np.testing.assert_array_equal(got_A, ref_A)
        ref = before.copy()
        assert od.kv_commit(ref, ref_A, got_am, B, B) == 0
        _states_equal(st, ref)
        after = st.to_host(si.state)
        assert after.free_top == ref.free_top
        np.testing.assert_array_equal(after.free_stack[:after.free_top], ref.free_stack[:ref.free_top])
        if forced:
            for s in range(S):
                c = int(before.out_count[s])
                if not before.finished[s] and c + B - 1 <= si.max_new:
                    assert got_A[s] == B - 1, (steps, s, got_A[s])
                    forced_full += 1
        steps += 1
        assert steps <= 2 * si.max_new
    print(f"[stack] {steps} steps, {forced_full} full acceptances", flush=True)
    assert forced_full >= 8 * 10
    host = st.to_host(si.state)
    np.testing.assert_array_equal(host.out_count, [si.max_new] * S)
    np.testing.assert_array_equal(host.out_tokens, ar.out_tokens)
