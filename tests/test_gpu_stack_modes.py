"""GPU: the decoding modes beside the fused step on the 16-layer bf16 stack at
the benchmark's shape (8 sequences, 1024 vision + 64 prompt tokens, B = 16,
vocab 65536, chunk 256), checked by properties that hold at any size:

* direct block diffusion with B = 1 is greedy AR (identical streams);
* with B = 16 at tau_c = 0.9 (the benchmark's setting) the first position of
  a block is predicted by the causal boundary row, so it is the AR token;
  a block takes 1..16 denoising forwards and commits 16 tokens;
* the refined-draft round (tau_d = 0.9) and the sampled round at T = 1e-4
  commit the greedy AR stream (any draft is verified exactly; at T -> 0
  sampling is the top-1).
"""
import numpy as np
import pytest
import torch

from paper_2609_26638_amd import dvs, synth
from tests.test_gpu_model_step import _widen_draft

pytestmark = pytest.mark.gpu

CH = 256
N = 40


@pytest.fixture(scope="module")
def stack():
    print("[stack-modes] generating the 16-layer stack", flush=True)
    return synth.decoder_stack_inputs()


def _prefilled(si, wide=False):
    w = si.weights
    pool = si.state.pool_pages
    kps = [torch.zeros((pool, w.Hkv, 16, w.D), dtype=torch.bfloat16, device="cuda")
           for _ in range(w.n_layers)]
    vps = [torch.zeros((pool, w.Hkv, w.D, 16), dtype=torch.bfloat16, device="cuda")
           for _ in range(w.n_layers)]
    dm = dvs.DeviceModel(w, kps, vps, "bf16")
    host = _widen_draft(si.state, si.B) if wide else si.state
    st = dvs.DeviceState(host)
    dvs.prefill(dm, st, si.P, si.B, prefix_tokens=torch.from_numpy(si.prefix_tokens()).cuda(),
                x_prefix=torch.from_numpy(si.x_prefix()).cuda(), chunk_keys=CH)
    return dm, st, host


def _ar_stream(si):
    dm, st, host = _prefilled(si)
    for _ in range(N):
        dvs.draft_verify_step(dm, st, 1, 0, chunk_keys=CH)
    torch.cuda.synchronize()
    assert int(st.err.item()) == 0
    return st.to_host(host)


def _same_prefix(got, ar, n):
    for s in range(ar.out_count.shape[0]):
        assert int(got.out_count[s]) >= n
        np.testing.assert_array_equal(got.out_tokens[s, :n], ar.out_tokens[s, :n])


def test_stack_diffusion_properties(stack):
    si = stack
    ar = _ar_stream(si)
    print("[stack-modes] AR reference done", flush=True)
    dm, st, host = _prefilled(si, wide=True)
    for _ in range(N):
        _, steps = dvs.diffusion_block(dm, st, 1, 0.9, chunk_keys=CH)
        assert steps == 1
    torch.cuda.synchronize()
    assert int(st.err.item()) == 0
    _same_prefix(st.to_host(host), ar, N + 1)
    print("[stack-modes] B=1 diffusion == AR", flush=True)
    dm, st, host = _prefilled(si, wide=True)
    before = st.to_host(host)
    for blk in range(2):
        block, steps = dvs.diffusion_block(dm, st, si.B, 0.9, chunk_keys=CH)
        torch.cuda.synchronize()
        assert int(st.err.item()) == 0
        assert 1 <= steps <= si.B
        got = st.to_host(host)
        np.testing.assert_array_equal(got.out_count, before.out_count + si.B * (blk + 1))
        np.testing.assert_array_equal(got.kv_len, before.kv_len + si.B * (blk + 1))
        if blk == 0:
            np.testing.assert_array_equal(block.cpu().numpy()[:, 0], ar.out_tokens[:, 1])
    print("[stack-modes] B=16 diffusion blocks checked", flush=True)


@pytest.mark.parametrize("mode", ["refined", "sampled"])
def test_stack_rounds_commit_the_ar_stream(stack, mode):
    si = stack
    ar = _ar_stream(si)
    dm, st, host = _prefilled(si, wide=True)
    gen = torch.Generator(device="cuda").manual_seed(7)
    rounds = 0
    while int(st.out_count.min().item()) < N + 1:
        if mode == "refined":
            steps = dvs.literal_round_refined(dm, st, si.B, 0.9, chunk_keys=CH)
            assert 1 <= steps <= si.B + 1
        else:
            u = torch.rand((st.kv_len.shape[0], 2 * si.B + 2), device="cuda", generator=gen)
            dvs.literal_round_sampled(dm, st, si.B, 1e-4, u, chunk_keys=CH)
        rounds += 1
        assert rounds <= N
    torch.cuda.synchronize()
    assert int(st.err.item()) == 0
    _same_prefix(st.to_host(host), ar, N + 1)
    print(f"[stack-modes] {mode}: {rounds} rounds == AR", flush=True)


def test_stack_multidraft_commits_the_ar_stream(stack):
    """The per-acceptance multi-draft step at the stack's shape (B = 16: 16
    causal rows and 16 groups of 16 mask rows, 272 window rows per
    sequence): the first draft is the AR continuation, so the first step
    accepts all 15 drafts, and the committed stream equals greedy AR."""
    si = stack
    ar = _ar_stream(si)
    w, B = si.weights, si.B
    pool_state = synth.stack_state(3, 8, si.P, B, si.max_new, B + B * B)
    pool = pool_state.pool_pages
    kps = [torch.zeros((pool, w.Hkv, 16, w.D), dtype=torch.bfloat16, device="cuda")
           for _ in range(w.n_layers)]
    vps = [torch.zeros((pool, w.Hkv, w.D, 16), dtype=torch.bfloat16, device="cuda")
           for _ in range(w.n_layers)]
    dm = dvs.DeviceModel(w, kps, vps, "bf16")
    st = dvs.DeviceState(pool_state)
    dvs.prefill(dm, st, si.P, B, prefix_tokens=torch.from_numpy(si.prefix_tokens()).cuda(),
                x_prefix=torch.from_numpy(si.x_prefix()).cuda(), chunk_keys=CH)
    st.draft.copy_(torch.from_numpy(np.ascontiguousarray(ar.out_tokens[:, 1:B])))
    acc = torch.empty((8,), dtype=torch.int32, device="cuda")
    dvs.multidraft_step(dm, st, B, chunk_keys=CH, accept_out=acc)
    torch.cuda.synchronize()
    assert acc.cpu().numpy().tolist() == [B - 1] * 8
    steps = 1
    while int(st.out_count.min().item()) < N + 1:
        dvs.multidraft_step(dm, st, B, chunk_keys=CH)
        steps += 1
        assert steps <= N
    torch.cuda.synchronize()
    assert int(st.err.item()) == 0
    _same_prefix(st.to_host(pool_state), ar, N + 1)
    print(f"[stack-modes] multidraft: {steps} steps == AR", flush=True)
