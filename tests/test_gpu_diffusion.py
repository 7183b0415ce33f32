"""GPU: direct block-diffusion decoding (top1_confidence, diffusion_denoise,
diffusion_block, kv_commit_block) against the oracle.

* top1_confidence: top-1 bit-exact, confidence within 1e-5 relative of the
  float64 softmax probability: each thread sums up to 256 fp32 terms in
  order (rounding bound 256 x 2^-24 = 1.5e-5, typically ~1e-6), then a tree
  over the threads; an all-equal row of 65,536 logits sums exactly, so a
  dropped or doubled term shows there.
* diffusion_denoise: logits within the fp32 tolerance of the oracle's; the
  reveal replayed by the oracle on the GPU's own top-1 and confidence (taken
  in fp32 on both sides) is bit-exact.
* diffusion_block: blocks, denoising step counts and the decode state equal
  the oracle's over several blocks, with the threshold placed so that every
  reveal decision has a margin far above the fp32 confidence error.
* B = 1 is greedy AR: the GPU streams are bit-identical (bf16 and fp32).
"""
import numpy as np
import pytest
import torch

from oracle import decode as od
from oracle.model import OracleModel
from paper_2609_26638_amd import dvs, synth
from tests.gpu_util import max_rel_err
from tests.test_gpu_model_step import LOGIT_TOL_F32, _dev_pools, _small_model, _states_equal

pytestmark = pytest.mark.gpu

CONF_TOL = 1e-5


def _logit_rows(seed, rows, V, scale):
    rng = np.random.default_rng(seed)
    x = (rng.standard_normal((rows, V)) * scale).astype(np.float32)
    x[0, :] = 0.0                                  # all equal: top-1 0, conf 1/V
    if rows > 1:
        x[1, V // 3] = x[1, (2 * V) // 3] = x[1].max() + 1.0   # tie: the lower index wins
    return x


@pytest.mark.parametrize("V,dtype,scale", [(65536, "f32", 4.0), (65536, "bf16", 4.0),
                                           (1000, "f32", 30.0), (1, "f32", 1.0),
                                           (517, "bf16", 0.5)])
def test_top1_confidence_matches_oracle(V, dtype, scale):
    x = _logit_rows(V + len(dtype), 37, V, scale)
    if dtype == "bf16":
        bits = synth.f32_to_bf16_bits(x)
        ref = synth.bf16_to_f64(bits)
        t = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).cuda()
    else:
        ref = x.astype(np.float64)
        t = torch.from_numpy(x).cuda()
    am, conf = dvs.top1_confidence(t)
    torch.cuda.synchronize()
    am, conf = am.cpu().numpy(), conf.cpu().numpy().astype(np.float64)
    for r in range(x.shape[0]):
        tr, cr = od.top1_confidence(ref[r])
        assert am[r] == tr, r
        assert abs(conf[r] - cr) <= CONF_TOL * cr, (r, conf[r], cr)


def _model_and_state(dtype, B, seed=4):
    w, base, kps, vps = _small_model(seed, dtype)
    host = base.state.copy()
    host.out_tokens = np.full((base.S, 256), -1, np.int32)
    rng = np.random.default_rng(seed + 1)
    host.boundary[:] = rng.integers(0, w.V, size=base.S)
    return w, host, kps, vps


def test_denoise_step_matches_oracle():
    B = 8
    w, host, kps, vps = _model_and_state("f32", B)
    S = host.kv_len.shape[0]
    om = OracleModel(w, kps, vps)
    dm = dvs.DeviceModel(w, _dev_pools(kps, "f32"), _dev_pools(vps, "f32"), "f32")
    rng = np.random.default_rng(9)
    block = np.full((S, B), -1, np.int64)
    block[rng.random((S, B)) < 0.3] = 7                # some positions already revealed
    lg_ref, am_ref, conf_ref, _ = om.diffusion_denoise(host.copy(), block, 0.0)
    st = dvs.DeviceState(host)
    for tau in (float(np.median(conf_ref)), 0.0, 1.01):
        tau32 = float(np.float32(tau))
        blk = torch.from_numpy(block.astype(np.int32)).cuda()
        logits = torch.empty((S * (B + 1), w.V), dtype=torch.float32, device="cuda")
        am = torch.empty(S * (B + 1), dtype=torch.int32, device="cuda")
        conf = torch.empty(S * (B + 1), dtype=torch.float32, device="cuda")
        n_open = dvs.diffusion_denoise(dm, st, blk, tau32, logits_out=logits, argmax_out=am,
                                       conf_out=conf)
        torch.cuda.synchronize()
        assert int(st.err.item()) == 0
        lg = logits.cpu().numpy().astype(np.float64).reshape(S, B + 1, w.V)
        err = max_rel_err(lg, lg_ref)
        print(f"[err] denoise logits tau={tau32:.4g}: {err:.3e}")
        assert err <= LOGIT_TOL_F32
        am_g = am.cpu().numpy().reshape(S, B + 1)
        conf_g = conf.cpu().numpy().astype(np.float64).reshape(S, B + 1)
        np.testing.assert_array_equal(am_g, od.top1_rows(lg).reshape(S, B + 1))
        np.testing.assert_allclose(conf_g[:, :B], conf_ref, rtol=1e-4)
        # the reveal on the GPU's own predictions: bit-exact
        expect = od.reveal(block, am_g[:, :B], conf_g[:, :B], tau32, host.finished)
        np.testing.assert_array_equal(blk.cpu().numpy(), expect)
        assert int(n_open.item()) == int(np.sum((expect < 0).any(axis=1)))
        _states_equal(st, host)                           # a denoising step commits nothing


def _oracle_blocks(om, st, B, tau, n_blocks):
    """Oracle blocks, plus the smallest margin of any reveal decision."""
    out, margin = [], np.inf
    S = st.kv_len.shape[0]
    for _ in range(n_blocks):
        block = np.full((S, B), -1, np.int64)
        steps = 0
        while np.any((block < 0).any(axis=1) & (st.finished == 0)):
            _, _, conf, nb = om.diffusion_denoise(st, block, tau)
            for s in range(S):
                masked = conf[s][block[s] < 0]
                if masked.size:
                    margin = min(margin, float(np.min(np.abs(masked - tau))))
                    if np.all(masked <= tau) and masked.size > 1:
                        top2 = np.sort(masked)[-2:]
                        margin = min(margin, float(top2[1] - top2[0]) + (top2[1] == top2[0]))
            block = nb
            steps += 1
        tok = np.concatenate([st.boundary[:, None], np.where(block[:, :B - 1] < 0, om.mask_id,
                                                            block[:, :B - 1])], axis=1)
        om.forward(om.embed[tok], st, B, 0)
        assert od.kv_commit(st, None, None, B, 0, window=B + 1, block_runs=block) == 0
        out.append((block.copy(), steps, st.copy()))
    return out, margin


def test_diffusion_blocks_match_oracle():
    B, n_blocks = 8, 3
    w, host, kps, vps = _model_and_state("f32", B, seed=6)
    om = OracleModel(w, kps, vps)
    # a threshold between two confidences of the first forward, so that some
    # positions clear it and some do not
    _, _, conf0, _ = om.diffusion_denoise(host.copy(), np.full((host.kv_len.shape[0], B), -1), 0.0)
    c = np.sort(conf0.ravel())
    i = int(0.3 * len(c))
    tau = float(np.float32(0.5 * (c[i] + c[i + 1])))
    ref, margin = _oracle_blocks(om, host.copy(), B, tau, n_blocks)
    print(f"[margin] tau={tau:.4g} smallest reveal margin {margin:.3e}")
    assert margin > 1e-4 * max(tau, 1e-3)
    dm = dvs.DeviceModel(w, _dev_pools(kps, "f32"), _dev_pools(vps, "f32"), "f32")
    st = dvs.DeviceState(host)
    multi = 0
    for blk_ref, steps_ref, st_ref in ref:
        blk, steps = dvs.diffusion_block(dm, st, B, tau)
        torch.cuda.synchronize()
        assert int(st.err.item()) == 0
        np.testing.assert_array_equal(blk.cpu().numpy(), blk_ref)
        assert steps == steps_ref
        multi += steps < B
        _states_equal(st, st_ref)
    assert multi >= 1          # at least one block revealed several positions at once


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_b1_diffusion_equals_greedy_ar_on_gpu(dtype):
    N, CH = 24, 64
    w, host, kps, vps = _model_and_state(dtype, 1)
    ar_m = dvs.DeviceModel(w, _dev_pools(kps, dtype), _dev_pools(vps, dtype), dtype)
    ar_st = dvs.DeviceState(host)
    for _ in range(N):
        dvs.draft_verify_step(ar_m, ar_st, 1, 0, chunk_keys=CH)
    df_m = dvs.DeviceModel(w, _dev_pools(kps, dtype), _dev_pools(vps, dtype), dtype)
    df_st = dvs.DeviceState(host)
    for _ in range(N):
        _, steps = dvs.diffusion_block(df_m, df_st, 1, 0.9, chunk_keys=CH)
        assert steps == 1
    torch.cuda.synchronize()
    assert int(ar_st.err.item()) == 0 and int(df_st.err.item()) == 0
    ar, df = ar_st.to_host(host), df_st.to_host(host)
    # (page counts differ: a diffusion commit keeps pages for a 2-row window)
    for f in ("out_tokens", "out_count", "kv_len", "boundary", "finished"):
        np.testing.assert_array_equal(getattr(df, f), getattr(ar, f), err_msg=f)


def test_block_commit_rejects_open_block():
    B = 4
    w, host, kps, vps = _model_and_state("f32", B)
    st = dvs.DeviceState(host)
    block = torch.full((host.kv_len.shape[0], B), 5, dtype=torch.int32, device="cuda")
    block[1, 2] = -1
    dvs.kv_commit_block(st, block)
    torch.cuda.synchronize()
    assert int(st.err.item()) & 16
    _states_equal(st, host)


def _top2_margin_ok(logits):
    srt = np.sort(logits, axis=-1)
    return bool(np.all(srt[..., -1] - srt[..., -2] > 4 * LOGIT_TOL_F32 * np.abs(logits).max(axis=-1)))


def test_refined_draft_round_matches_oracle(monkeypatch):
    """literal_round_refined (multi-step drafting) against the oracle's round
    with the same tau_d: draft forwards, drafts and the committed state.
    Every reveal decision of the oracle is recorded to check its margin."""
    B = 6
    margin = [np.inf]
    reveal = od.reveal

    def recording_reveal(block, am, conf, tau_c, finished):
        for s in range(block.shape[0]):
            m = conf[s][block[s] < 0]
            if finished[s] or not m.size:
                continue
            margin[0] = min(margin[0], float(np.min(np.abs(m - tau_c))))
            if np.all(m <= tau_c) and m.size > 1:
                t2 = np.sort(m)[-2:]
                margin[0] = min(margin[0], float(t2[1] - t2[0]) + float(t2[1] == t2[0]))
        return reveal(block, am, conf, tau_c, finished)

    monkeypatch.setattr(od, "reveal", recording_reveal)
    w, host, kps, vps = _model_and_state("f32", B, seed=15)
    host.draft = np.zeros((host.kv_len.shape[0], B), np.int32)
    om = OracleModel(w, kps, vps)
    probe = OracleModel(w, kps, vps)
    lg0 = probe.forward(probe.embed[np.concatenate(
        [host.boundary[:, None], np.full((host.kv_len.shape[0], B), probe.mask_id)], 1)],
        host.copy(), 1, B)
    c = np.sort([od.top1_confidence(r)[1] for r in lg0.reshape(-1, w.V)])
    i = int(0.5 * len(c))
    tau = float(np.float32(0.5 * (c[i] + c[i + 1])))
    dm = dvs.DeviceModel(w, _dev_pools(kps, "f32"), _dev_pools(vps, "f32"), "f32")
    st = dvs.DeviceState(host)
    ref = host.copy()
    for rnd in range(2):
        lg_d, lg_v, _, _, err = om.literal_round(ref, B, tau_d=tau)
        assert err == 0
        assert _top2_margin_ok(lg_d) and _top2_margin_ok(lg_v)
        steps = dvs.literal_round_refined(dm, st, B, tau)
        torch.cuda.synchronize()
        assert int(st.err.item()) == 0
        print(f"[round {rnd}] tau_d={tau:.4g} draft forwards gpu {steps} oracle {om.draft_steps}")
        assert steps == om.draft_steps
        _states_equal(st, ref)
    print(f"[margin] smallest reveal margin {margin[0]:.3e}")
    assert margin[0] > 1e-4 * tau


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_refined_draft_round_equals_greedy_ar_on_gpu(dtype):
    B, N, CH, TAU = 8, 32, 64, 0.05
    w, host, kps, vps = _model_and_state(dtype, B)
    host.draft = np.zeros((host.kv_len.shape[0], B), np.int32)
    ar_m = dvs.DeviceModel(w, _dev_pools(kps, dtype), _dev_pools(vps, dtype), dtype)
    ar_st = dvs.DeviceState(host)
    for _ in range(N):
        dvs.draft_verify_step(ar_m, ar_st, 1, 0, chunk_keys=CH)
    rm = dvs.DeviceModel(w, _dev_pools(kps, dtype), _dev_pools(vps, dtype), dtype)
    rs = dvs.DeviceState(host)
    rounds, multi = 0, 0
    while int(rs.out_count.min().item()) < N:
        steps = dvs.literal_round_refined(rm, rs, B, TAU, chunk_keys=CH)
        assert 1 <= steps <= B + 1
        multi += steps > 1
        rounds += 1
        assert rounds <= N
    torch.cuda.synchronize()
    assert int(ar_st.err.item()) == 0 and int(rs.err.item()) == 0
    ar, rr = ar_st.to_host(host), rs.to_host(host)
    for s in range(host.kv_len.shape[0]):
        n = min(int(rr.out_count[s]), int(ar.out_count[s]))
        assert n >= N
        np.testing.assert_array_equal(rr.out_tokens[s, :n], ar.out_tokens[s, :n])
    assert multi >= 1
