"""GPU parity: argmax_accept and kv_commit vs the oracle, bit for bit."""
import json
import os

import numpy as np
import pytest
import torch

from oracle import decode as od
from paper_2609_26638_amd import dvs, synth
from tests.gpu_util import to_dev

pytestmark = pytest.mark.gpu
GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _argmax(logits_np, dtype, n_causal, draft_np):
    lg = to_dev(logits_np, dtype)
    dr = torch.from_numpy(np.ascontiguousarray(draft_np, dtype=np.int32)).cuda()
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    am, A = dvs.argmax_accept(lg, n_causal, dr, err=err)
    torch.cuda.synchronize()
    return am.cpu().numpy(), A.cpu().numpy(), int(err.item())


@pytest.mark.parametrize("S,B,V,p", [(32, 16, 65536, 0.9), (3, 8, 1001, 0.7), (5, 4, 8, 0.5)])
def test_argmax_accept_planted_bf16(S, B, V, p):
    li = synth.make_logit_inputs(7, S, B, B, V, 4.0, p)
    am, A, err = _argmax(li.logits, "bf16", B, li.draft)
    ref_am = od.top1_rows(synth.bf16_to_f64(li.logits))
    np.testing.assert_array_equal(am, ref_am)
    np.testing.assert_array_equal(A, od.accept(ref_am, li.draft, B))
    assert err == 0


@pytest.mark.parametrize("dtype,V,levels", [("f32", 37, 4), ("f32", 4096, 4), ("bf16", 37, 4), ("bf16", 4099, 4),
                                            ("bf16", 65536, 4), ("f32", 16384, 4), ("bf16", 65536, 2),
                                            ("f32", 16384, 2)])
def test_argmax_ties_and_signed_zero(dtype, V, levels):
    x = synth.tied_logits(11, 4, 6, V, levels=levels)
    if dtype == "bf16":
        x = synth.f32_to_bf16_bits(x)
        ref = od.top1_rows(synth.bf16_to_f64(x))
    else:
        ref = od.top1_rows(x.astype(np.float64))
    draft = np.zeros((4, 2), np.int32)
    am, _, err = _argmax(x, dtype, 3, draft)
    np.testing.assert_array_equal(am, ref)
    assert err == 0


def test_argmax_all_negative_and_extremes():
    x = -np.abs(np.random.default_rng(2).standard_normal((2, 3, 777))).astype(np.float32) - 1
    x[0, 1, 500] = -0.5
    x[1, 2, 3] = np.float32(3.4e38)
    x[1, 2, 700] = np.float32(3.4e38)
    am, _, err = _argmax(x, "f32", 1, np.zeros((2, 0), np.int32))
    np.testing.assert_array_equal(am, od.top1_rows(x.astype(np.float64)))
    assert am[1, 2] == 3 and err == 0


def test_argmax_nonfinite_flagged():
    x = np.zeros((1, 2, 64), np.float32)
    x[0, 1, 9] = np.nan
    _, _, err = _argmax(x, "f32", 1, np.zeros((1, 0), np.int32))
    assert err & dvs.ERR_NONFINITE


@pytest.mark.parametrize("bits", [0x7FC0, 0xFFC0, 0x7F80, 0xFF80], ids=["nan", "neg_nan", "inf", "neg_inf"])
def test_argmax_nonfinite_flagged_long_bf16_row(bits):
    """A NaN or an infinity deep inside a vocabulary-sized bf16 row (the
    batched vector path) raises the flag."""
    x = synth.f32_to_bf16_bits(np.random.default_rng(3).standard_normal((1, 2, 65536)).astype(np.float32))
    x[0, 1, 40001] = bits
    _, _, err = _argmax(x, "bf16", 1, np.zeros((1, 0), np.int32))
    assert err & dvs.ERR_NONFINITE


def _expected_degenerate(row):
    """The header's rule for a row with no value above -inf: the lowest index
    holding -inf, or 0 when every value is NaN (NaN never wins)."""
    idx = np.flatnonzero(row == -np.inf)
    return int(idx[0]) if idx.size else 0


@pytest.mark.parametrize("dtype,V", [("f32", 777), ("bf16", 65536), ("bf16", 37), ("f32", 16384)])
def test_argmax_rows_without_a_finite_value_give_vocabulary_indices(dtype, V):
    """All -inf, all NaN, NaN then -inf, and a row whose only non-NaN values
    are -inf deep inside it: every result is an index in [0, V) by the rule
    above, and every such row raises DVS_ERR_NONFINITE.  A row with NaNs
    among finite values takes the top-1 of the finite values."""
    x = np.full((1, 5, V), -np.inf, np.float32)
    x[0, 1] = np.nan
    x[0, 2, :3] = np.nan
    x[0, 3] = np.nan
    x[0, 3, V - 2] = -np.inf
    x[0, 4] = np.random.default_rng(8).standard_normal(V).astype(np.float32)
    x[0, 4, ::7] = np.nan
    x[0, 4, V // 2 + 3] = 9.0
    xx = synth.f32_to_bf16_bits(x) if dtype == "bf16" else x
    for r in range(4):   # each degenerate row alone, to see its own flag
        am, _, err = _argmax(xx[:, r:r + 1], dtype, 1, np.zeros((1, 0), np.int32))
        assert int(am[0, 0]) == _expected_degenerate(x[0, r]), r
        assert err & dvs.ERR_NONFINITE
    am, _, err = _argmax(xx, dtype, 1, np.zeros((1, 0), np.int32))
    assert [int(v) for v in am[0]] == [0, 0, 3, V - 2, V // 2 + 3]
    lg = to_dev(xx.reshape(5, V), dtype)
    top = torch.zeros(5, dtype=torch.int32, device="cuda")
    conf = torch.zeros(5, dtype=torch.float32, device="cuda")
    e2 = torch.zeros(1, dtype=torch.int32, device="cuda")
    dvs.top1_confidence(lg, top, conf, err=e2)
    torch.cuda.synchronize()
    assert top.cpu().tolist() == [0, 0, 3, V - 2, V // 2 + 3]
    assert int(e2.item()) & dvs.ERR_NONFINITE


def test_argmax_ties_in_vectorized_path_bf16():
    """Equal maxima planted at two positions of 65536-wide rows: in one 16-byte
    vector, in one thread's batch, across threads, across batches, at the row
    ends.  The lowest index must win."""
    pairs = [(100, 103), (8 * 5, 8 * (5 + 256)), (8 * 7 + 2, 8 * 8 + 1), (8 * 9, 8 * (9 + 2048)),
             (3, 65535), (0, 65535), (8 * 2047 + 7, 8 * 4095 + 7)]
    rng = np.random.default_rng(4)
    x = np.clip(rng.standard_normal((1, len(pairs), 65536)), -6, 6).astype(np.float32)
    for r, (a, b) in enumerate(pairs):
        x[0, r, a] = 7.5
        x[0, r, b] = 7.5
    xb = synth.f32_to_bf16_bits(x)
    am, _, err = _argmax(xb, "bf16", 1, np.zeros((1, 0), np.int32))
    ref = od.top1_rows(synth.bf16_to_f64(xb))
    np.testing.assert_array_equal(am, ref)
    assert [int(v) for v in am[0]] == [min(a, b) for a, b in pairs] and err == 0


def _dev_state(st):
    return dvs.DeviceState(st)


def _assert_state_equal(dev, host):
    got = dev.to_host(host)
    for f in ("kv_len", "page_table", "num_pages", "boundary", "draft", "out_tokens",
              "out_count", "finished"):
        np.testing.assert_array_equal(getattr(got, f), getattr(host, f), err_msg=f)
    assert got.free_top == host.free_top
    np.testing.assert_array_equal(got.free_stack[:got.free_top], host.free_stack[:host.free_top])


def test_commit_eos_push_pop_mix_matches_oracle():
    """The golden example's state (EOS stop, surplus pages, pops) with its
    lengths scaled to the library's 16-token pages, against the oracle."""
    g = json.load(open(os.path.join(GOLDEN, "commit_example.json")))
    b = g["before"]
    S = len(b["kv_len"])
    st = synth.PagedState(
        kv_len=np.array(b["kv_len"], np.int32) * 4, page_table=np.array(b["page_table"], np.int32),
        num_pages=np.array(b["num_pages"], np.int32),
        free_stack=np.array(b["free_stack"], np.int32), free_top=int(b["free_top"]),
        boundary=np.array(b["boundary"], np.int32), draft=np.array(b["draft"], np.int32),
        out_tokens=np.full((S, 16), -1, np.int32), out_count=np.zeros(S, np.int32),
        finished=np.zeros(S, np.int32), pool_pages=8, max_pages=4)
    am = np.array(b["argmax"], np.int32)
    ref = st.copy()
    A = od.accept(am, ref.draft, 2)
    # window of 2 causal + 14 mask rows keeps R = 16 (one page), drafts width 1
    am16 = np.concatenate([am[:, :2], np.repeat(am[:, 2:3], 14, axis=1)], axis=1)
    err_ref = od.kv_commit(ref, A, am16, 2, 14, eos_id=77)
    dev = _dev_state(st)
    dvs.kv_commit(dev, torch.from_numpy(A).cuda(), torch.from_numpy(am16).cuda(), 2, 14, eos_id=77)
    torch.cuda.synchronize()
    assert err_ref == 0 and int(dev.err.item()) == 0
    _assert_state_equal(dev, ref)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_commit_random_steps_match_oracle(seed):
    rng = np.random.default_rng(seed)
    S, B, V = 37, 6, 9
    R = 2 * B
    L = rng.integers(0, 300, size=S)
    st = synth.make_paged_state(rng, L, R, max_pages=64, scatter=True, slack=0.3,
                                extra_pages=20, n_causal=B, max_new=64)
    dev = _dev_state(st)
    for step in range(25):
        am = rng.integers(0, V, size=(S, R)).astype(np.int32)
        st.draft[:] = np.where(rng.random((S, B - 1)) < 0.8, am[:, :B - 1], st.draft)
        dev.draft.copy_(torch.from_numpy(st.draft))
        A = od.accept(am, st.draft, B)
        e = od.kv_commit(st, A, am, B, B, eos_id=4 if step > 10 else -1)
        dvs.kv_commit(dev, torch.from_numpy(A).cuda(), torch.from_numpy(am).cuda(), B, B,
                      eos_id=4 if step > 10 else -1)
        torch.cuda.synchronize()
        assert e == int(dev.err.item())
        _assert_state_equal(dev, st)


@pytest.mark.parametrize("seed,B", [(0, 6), (1, 32), (2, 17)])
def test_accept_commit_random_steps_match_oracle(seed, B):
    """accept_commit (acceptance inside the commit kernel) against the
    oracle's accept then kv_commit over random steps: drafts that match the
    top-1 with probability 0.9 (long accepted runs at B = 32: four run
    chunks), EOS stops, budget truncation, finished sequences."""
    rng = np.random.default_rng(200 + seed)
    S, V = 41, 9
    R = 2 * B
    L = rng.integers(0, 300, size=S)
    # pool: enough free pages for every sequence to reach its 200-token budget
    st = synth.make_paged_state(rng, L, R, max_pages=96, scatter=True, slack=0.3,
                                extra_pages=S * 14, n_causal=B, max_new=200)
    dev = _dev_state(st)
    accepted = []
    for step in range(25):
        am = rng.integers(0, V, size=(S, R)).astype(np.int32)
        st.draft[:] = np.where(rng.random((S, B - 1)) < 0.9, am[:, :B - 1], st.draft)
        dev.draft.copy_(torch.from_numpy(st.draft))
        A = od.accept(am, st.draft, B)
        live = st.finished == 0
        eos = 4 if step > 15 else -1
        e = od.kv_commit(st, A, am, B, B, eos_id=eos)
        got_A = dvs.accept_commit(dev, torch.from_numpy(am).cuda(), B, B, eos_id=eos)
        torch.cuda.synchronize()
        assert e == int(dev.err.item()) == 0
        np.testing.assert_array_equal(got_A.cpu().numpy(), np.where(live, A, 0))
        _assert_state_equal(dev, st)
        accepted.extend(A[live].tolist())
    assert max(accepted) == B - 1 and st.finished.sum() > 0


@pytest.mark.parametrize("seed", [0, 1])
def test_commit_round_random_steps_match_oracle(seed):
    """kv_commit_round (two-forward round: lead a0, then d_1..d_A, a_{A+1};
    kv_len already counts x0; pages for the next B + 2 window) against the
    oracle over random rounds, with EOS stops, budget truncation and
    finished sequences."""
    rng = np.random.default_rng(100 + seed)
    S, B, V = 29, 5, 7
    L = rng.integers(0, 300, size=S)
    st = synth.make_paged_state(rng, L, B + 2, max_pages=64, scatter=True, slack=0.3,
                                extra_pages=20, n_causal=B + 1, max_new=60)
    dev = _dev_state(st)
    for step in range(25):
        am = rng.integers(0, V, size=(S, B + 1)).astype(np.int32)
        lead = rng.integers(0, V, size=S).astype(np.int32)
        live = st.finished == 0
        # the draft forward's effect: d_1..d_B written, x0's KV kept
        d = np.where(rng.random((S, B)) < 0.8, am[:, :B], rng.integers(0, V, size=(S, B)))
        st.draft[live] = d[live]
        st.kv_len[live] += 1
        dev.draft.copy_(torch.from_numpy(st.draft))
        dev.kv_len.copy_(torch.from_numpy(st.kv_len))
        A = od.accept(am, st.draft, B + 1)
        eos = 4 if step > 10 else -1
        e = od.kv_commit(st, A, am, B + 1, 0, eos_id=eos, lead=lead, window=B + 2)
        dvs.kv_commit_round(dev, B, torch.from_numpy(lead).cuda(), torch.from_numpy(A).cuda(),
                            torch.from_numpy(am).cuda(), eos_id=eos)
        torch.cuda.synchronize()
        assert e == int(dev.err.item()) == 0
        _assert_state_equal(dev, st)
    assert st.finished.sum() > 0


def test_commit_switching_window_size_pushes_pages():
    rng = np.random.default_rng(3)
    S = 9
    L = rng.integers(0, 100, size=S)
    st = synth.make_paged_state(rng, L, 64, max_pages=16, scatter=True, slack=0.0,
                                n_causal=32, max_new=32)
    dev = _dev_state(st)
    am = rng.integers(0, 50, size=(S, 1)).astype(np.int32)
    A = np.zeros(S, np.int32)
    # an AR step (1 row): every sequence drops to ceil((L+2)/16) pages
    st.draft = np.zeros((S, 0), np.int32)
    dev = _dev_state(st)
    od.kv_commit(st, A, am, 1, 0)
    dvs.kv_commit(dev, torch.from_numpy(A).cuda(), torch.from_numpy(am).cuda(), 1, 0)
    torch.cuda.synchronize()
    _assert_state_equal(dev, st)


def test_commit_pool_exhausted_leaves_state():
    rng = np.random.default_rng(4)
    S, B = 4, 16
    st = synth.make_paged_state(rng, np.array([15, 31, 47, 63]), 2 * B, max_pages=16,
                                scatter=True, slack=0.0, n_causal=B, max_new=64)
    assert st.free_top == 0
    dev = _dev_state(st)
    am = np.tile(np.arange(2 * B, dtype=np.int32), (S, 1))
    st.draft[:] = am[:, :B - 1]
    dev.draft.copy_(torch.from_numpy(st.draft))
    A = od.accept(am, st.draft, B)
    ref = st.copy()
    e = od.kv_commit(ref, A, am, B, B)
    assert e == od.ERR_POOL_EXHAUSTED
    dvs.kv_commit(dev, torch.from_numpy(A).cuda(), torch.from_numpy(am).cuda(), B, B)
    torch.cuda.synchronize()
    assert int(dev.err.item()) == dvs.ERR_POOL_EXHAUSTED
    _assert_state_equal(dev, st)
