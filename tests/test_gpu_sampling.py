"""GPU: the two-forward round under sampling (literal_round_sampled) against
the oracle's sampled_round, on the same uniforms.

Every sampling and acceptance decision is a float comparison; the test
records the oracle's margin for each (distance of u * total to the nearest
CDF boundary, relative to the total; |u q - p| relative to max(p, q)) and
requires them far above the fp32 logit error, then asks for identical
drafts, acceptance lengths, final tokens and state.  At T -> 0 sampling is
the top-1, so the sampled round's stream equals the GPU's greedy AR stream
(bf16 and fp32)."""
import numpy as np
import pytest
import torch

from oracle import decode as od
from oracle.model import OracleModel
from paper_2609_26638_amd import dvs
from tests.test_gpu_diffusion import _model_and_state
from tests.test_gpu_model_step import _dev_pools, _states_equal

pytestmark = pytest.mark.gpu


def _cdf_margin(w, u):
    c = np.cumsum(w)
    t = u * c[-1]
    i = od.sample_index(w, u)
    lo = c[i - 1] if i > 0 else 0.0
    return min(t - lo, c[i] - t) / c[-1]


def _decision_margin(lg_d, lg_v, st_before, B, T, u):
    """Smallest relative margin of the oracle's decisions in one round."""
    S = lg_d.shape[0]
    mg = np.inf
    for s in range(S):
        q = [od.softmax_t(lg_d[s, r], T) for r in range(B + 1)]
        p = [od.softmax_t(lg_v[s, r], T) for r in range(B + 1)]
        d = [od.sample_index(q[r], u[s, r]) for r in range(B + 1)]
        for r in range(B + 1):
            mg = min(mg, _cdf_margin(q[r], u[s, r]))
        A = od.stochastic_accept(np.array(p[:B]), np.array(q[1:]), np.array(d[1:]),
                                 u[s, B + 1:2 * B + 1])
        for j in range(1, min(A + 1, B) + 1):
            pj, qj = p[j - 1][d[j]], q[j][d[j]]
            mg = min(mg, abs(u[s, B + j] * qj - pj) / max(pj, qj))
        w = od.resample_weights(p[A], None if A == B else q[A + 1])
        mg = min(mg, _cdf_margin(w, u[s, 2 * B + 1]))
    return mg


def test_sampled_round_matches_oracle():
    B, T = 6, 1.0
    w, host, kps, vps = _model_and_state("f32", B, seed=17)
    host.draft = np.zeros((host.kv_len.shape[0], B), np.int32)
    S = host.kv_len.shape[0]
    om = OracleModel(w, kps, vps)
    dm = dvs.DeviceModel(w, _dev_pools(kps, "f32"), _dev_pools(vps, "f32"), "f32")
    st = dvs.DeviceState(host)
    ref = host.copy()
    rng = np.random.default_rng(3)
    acc = torch.empty(S, dtype=torch.int32, device="cuda")
    for rnd in range(2):
        u = rng.random((S, 2 * B + 2))
        u32 = u.astype(np.float32)
        before = ref.copy()
        lg_d, lg_v, A, final, err = om.sampled_round(ref, B, T, u32.astype(np.float64))
        assert err == 0
        mg = _decision_margin(lg_d, lg_v, before, B, T, u32.astype(np.float64))
        print(f"[round {rnd}] A={list(A)} smallest decision margin {mg:.3e}")
        # fp32 logits are within ~2e-6 of the row's largest |logit| (~1 here),
        # so at T = 1 a weight moves by ~2e-6 relative: 1.5e-5 leaves 7x
        assert mg > 1.5e-5
        dvs.literal_round_sampled(dm, st, B, T, torch.from_numpy(u32).cuda(), accept_out=acc)
        torch.cuda.synchronize()
        assert int(st.err.item()) == 0
        np.testing.assert_array_equal(acc.cpu().numpy(), A)
        _states_equal(st, ref)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_low_temperature_sampled_round_equals_greedy_ar_on_gpu(dtype):
    B, N, CH, T = 8, 32, 64, 1e-4
    w, host, kps, vps = _model_and_state(dtype, B)
    host.draft = np.zeros((host.kv_len.shape[0], B), np.int32)
    S = host.kv_len.shape[0]
    ar_m = dvs.DeviceModel(w, _dev_pools(kps, dtype), _dev_pools(vps, dtype), dtype)
    ar_st = dvs.DeviceState(host)
    for _ in range(N):
        dvs.draft_verify_step(ar_m, ar_st, 1, 0, chunk_keys=CH)
    sm = dvs.DeviceModel(w, _dev_pools(kps, dtype), _dev_pools(vps, dtype), dtype)
    ss = dvs.DeviceState(host)
    gen = torch.Generator(device="cuda").manual_seed(5)
    rounds = 0
    while int(ss.out_count.min().item()) < N:
        u = torch.rand((S, 2 * B + 2), device="cuda", generator=gen)
        dvs.literal_round_sampled(sm, ss, B, T, u, chunk_keys=CH)
        rounds += 1
        assert rounds <= N
    torch.cuda.synchronize()
    assert int(ar_st.err.item()) == 0 and int(ss.err.item()) == 0
    ar, sr = ar_st.to_host(host), ss.to_host(host)
    for s in range(S):
        n = min(int(sr.out_count[s]), int(ar.out_count[s]))
        assert n >= N
        np.testing.assert_array_equal(sr.out_tokens[s, :n], ar.out_tokens[s, :n])
