"""GPU parity: attn_hybrid_block (HIP) vs the float64 oracle.

Tolerances: max over output vectors of ||o - o_ref||_inf / ||o_ref||_inf,
2e-2 for bf16 inputs (fp32 accumulation) and 1e-5 in fp32 mode.  Integer-like
effects (the K/V append) and invariances are checked bit for bit.
"""
import numpy as np
import pytest
import torch

from oracle import attention as oa
from paper_2609_26638_amd import dvs, synth
from tests.gpu_util import dev_attn, max_rel_err, to_f64

pytestmark = pytest.mark.gpu

TOL = {"bf16": 2e-2, "f32": 1e-5}


def _run(ai, chunk_keys=0, ws=None, err=None):
    d = dev_attn(ai)
    out = dvs.attn_hybrid_block(d["q"], d["k_new"], d["v_new"], d["k_pool"], d["v_pool"],
                                d["page_table"], d["kv_len"], ai.n_causal, ai.n_mask, ai.scale,
                                chunk_keys=chunk_keys, workspace=ws, err=err)
    torch.cuda.synchronize()
    return out, d


def _oracle(ai):
    kp, vp = ai.as_f64("k_pool"), ai.as_f64("v_pool")
    out = oa.attn_hybrid_block(ai.as_f64("q"), ai.as_f64("k_new"), ai.as_f64("v_new"), kp, vp,
                               ai.state.page_table, ai.state.kv_len, ai.n_causal, ai.n_mask,
                               ai.scale)
    return out, kp, vp


CASES = [
    # name, seed, S, L, Vc, Vm, Hq, Hkv, D, dtype, chunk
    ("tiny_fp32_single_layer", 0, 1, [256], 8, 8, 4, 4, 64, "f32", 0),
    ("one_layer_bf16_kv2048", 1, 1, [2048], 16, 16, 16, 4, 128, "bf16", 0),
    ("ragged_multichunk", 21, 3, [0, 77, 1000], 16, 16, 16, 4, 128, "bf16", 256),
    ("ragged_b8_d96", 22, 4, [5, 64, 130, 700], 8, 8, 16, 4, 96, "bf16", 128),
    ("mha_d64", 23, 2, [300, 31], 4, 4, 4, 4, 64, "bf16", 64),
    ("ar_row", 24, 3, [1, 63, 2000], 1, 0, 16, 4, 128, "bf16", 512),
    ("mask_block_only", 25, 2, [100, 1], 0, 16, 8, 2, 128, "bf16", 0),
    ("two_row_tiles", 26, 2, [90, 500], 40, 40, 16, 4, 128, "bf16", 256),
    ("b32_long", 27, 2, [4100, 3000], 32, 32, 16, 4, 128, "bf16", 1024),
    ("fp32_gqa_ragged", 28, 3, [0, 40, 333], 4, 4, 8, 2, 128, "f32", 0),
    ("fp32_d96", 29, 2, [17, 100], 3, 5, 6, 3, 96, "f32", 0),
    # head_dim 96 at every wave count: AR rows (1 wave), a B=16 window (4
    # waves), and a prefill-shaped window (no cache, hundreds of causal rows)
    ("ar_row_d96", 30, 3, [1, 63, 1100], 1, 0, 16, 4, 96, "bf16", 64),
    ("ar_row_d96_balanced", 33, 3, [1, 63, 1100], 1, 0, 16, 4, 96, "bf16", 0),
    ("window_d96_4waves", 32, 2, [1088, 500], 16, 16, 16, 4, 96, "bf16", 0),
    ("prefill_d96", 31, 2, [0, 0], 300, 16, 16, 4, 96, "bf16", 64),
    ("prefill_d128_balanced", 34, 2, [0, 0], 200, 8, 8, 2, 128, "bf16", 0),
    ("d64_wide", 35, 2, [300, 77], 32, 32, 8, 2, 64, "bf16", 0),
    ("d64_wide_aligned", 36, 3, [5, 300, 1200], 16, 16, 8, 2, 64, "bf16", 128),
    ("d128_aligned_narrow", 37, 2, [700, 33], 4, 4, 8, 2, 128, "bf16", 256),
    # wide windows in the balanced split (the producer/consumer kernel):
    # ragged lengths incl. an empty cache, head_dim 96, two row tiles with a
    # partly filled second one
    ("pc_d128_ragged", 38, 3, [0, 77, 5000], 32, 32, 16, 4, 128, "bf16", 0),
    ("pc_d96_wide", 39, 2, [1500, 3000], 48, 16, 16, 4, 96, "bf16", 0),
    ("pc_d128_two_row_tiles", 40, 2, [900, 2100], 40, 40, 16, 4, 128, "bf16", 0),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_attention_matches_oracle(case):
    name, seed, S, L, Vc, Vm, Hq, Hkv, D, dt, chunk = case
    print(f"[attn] {name}", flush=True)
    ai = synth.make_attn_inputs(seed, S, L, Vc, Vm, Hq, Hkv, D, dt, std=1.0, scatter=True)
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    out, d = _run(ai, chunk, err=err)
    ref, kp, vp = _oracle(ai)
    e = max_rel_err(to_f64(out), ref)
    print(f"[err] {name}: max rel err {e:.3e}", flush=True)
    assert e <= TOL[dt], f"{name}: max rel err {e:.3e}"
    assert int(err.item()) == 0
    # the append wrote exactly the window's K/V (bit for bit, full pools)
    np.testing.assert_array_equal(to_f64(d["k_pool"]), kp)
    np.testing.assert_array_equal(to_f64(d["v_pool"]), vp)


def test_deterministic_and_page_permutation_invariant():
    ai = synth.make_attn_inputs(31, 3, [700, 33, 1500], 16, 16, 16, 4, 128, "bf16", scatter=True)
    o1, _ = _run(ai, 256)
    o2, _ = _run(ai, 256)
    assert torch.equal(o1.view(torch.int16), o2.view(torch.int16))
    # same logical cache, different physical pages
    ai2 = synth.make_attn_inputs(31, 3, [700, 33, 1500], 16, 16, 16, 4, 128, "bf16", scatter=True)
    rng = np.random.default_rng(5)
    P = ai2.k_pool.shape[0]
    perm = rng.permutation(P)
    inv = np.argsort(perm)
    ai2.k_pool = ai2.k_pool[perm].copy()
    ai2.v_pool = ai2.v_pool[perm].copy()
    pt = ai2.state.page_table
    ai2.state.page_table = np.where(pt >= 0, inv[np.maximum(pt, 0)], -1).astype(np.int32)
    o3, _ = _run(ai2, 256)
    assert torch.equal(o1.view(torch.int16), o3.view(torch.int16))


@pytest.mark.parametrize("dt", ["bf16", "f32"])
def test_causal_row_equals_ar_call(dt):
    """Verify row i gives bit-identical output to a plain AR call (1 causal
    row) at committed length L + i: rows do not influence each other."""
    B, L = 16, 1234
    ai = synth.make_attn_inputs(41, 1, [L], B, B, 16, 4, 128, dt, scatter=True)
    out, d = _run(ai, 512)
    for i in (0, 1, 7, B - 1):
        kvl = torch.tensor([L + i], dtype=torch.int32, device="cuda")
        oi = dvs.attn_hybrid_block(d["q"][:, i:i + 1].contiguous(), d["k_new"][:, i:i + 1].contiguous(),
                                   d["v_new"][:, i:i + 1].contiguous(), d["k_pool"], d["v_pool"],
                                   d["page_table"], kvl, 1, 0, ai.scale, chunk_keys=512)
        torch.cuda.synchronize()
        assert torch.equal(oi[:, 0].view(torch.int32 if dt == "f32" else torch.int16),
                           out[:, i].view(torch.int32 if dt == "f32" else torch.int16)), i


def test_mask_rows_do_not_change_causal_rows():
    B = 8
    ai = synth.make_attn_inputs(43, 2, [300, 90], B, B, 8, 2, 128, "bf16", scatter=True)
    o1, _ = _run(ai, 128)
    ai.q[:, B:] = ai.q[:, B:][:, ::-1]
    ai.k_new[:, B:] = ai.k_new[:, B:][:, ::-1] ^ 0x0001
    ai.v_new[:, B:] = 0x3F80  # 1.0
    o2, _ = _run(ai, 128)
    assert torch.equal(o1[:, :B].view(torch.int16), o2[:, :B].view(torch.int16))
    assert not torch.equal(o1[:, B:].view(torch.int16), o2[:, B:].view(torch.int16))


def test_bad_page_reported_without_fault():
    ai = synth.make_attn_inputs(44, 2, [200, 64], 4, 4, 8, 2, 64, "bf16", scatter=True)
    ai.state.page_table[1, 1] = 10 ** 6
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    _run(ai, 0, err=err)
    assert int(err.item()) & dvs.ERR_BAD_PAGE


def test_bad_page_reported_without_fault_wide_window():
    ai = synth.make_attn_inputs(46, 2, [900, 64], 32, 32, 8, 2, 128, "bf16", scatter=True)
    ai.state.page_table[0, 3] = -5
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    _run(ai, 0, err=err)
    assert int(err.item()) & dvs.ERR_BAD_PAGE


def test_too_long_sequence_reported():
    ai = synth.make_attn_inputs(45, 2, [200, 64], 4, 4, 8, 2, 64, "bf16", scatter=True)
    ai.state.kv_len[0] = ai.state.page_table.shape[1] * 16     # L + R > max_pages * 16
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    _run(ai, 0, err=err)
    assert int(err.item()) & dvs.ERR_MAX_PAGES


@pytest.fixture(scope="module")
def long_doc():
    print("[attn] generating the 64-sequence KV 4k-16k workload", flush=True)
    ai, li = synth.long_document_inputs()
    return ai, li


def test_long_document_sampled_rows(long_doc):
    """64 sequences, KV 4k-16k, 16/4 heads, D=128, B=32: the benchmark's launch
    configuration, checked on sampled (s, r, h) rows against the oracle."""
    ai, _ = long_doc
    out, d = _run(ai, 0)
    o = to_f64(out)
    rng = np.random.default_rng(0)
    S, R = ai.S, ai.R
    samples = {(int(rng.integers(S)), int(rng.integers(R)), int(rng.integers(16))) for _ in range(24)}
    samples |= {(0, 0, 0), (S - 1, R - 1, 15), (3, 31, 5), (5, 32, 9)}
    ref = oa.attn_sampled(ai.as_f64("q"), ai.as_f64("k_new"), ai.as_f64("v_new"),
                          ai.k_pool, ai.v_pool, ai.state.page_table, ai.state.kv_len,
                          ai.n_causal, ai.n_mask, ai.scale, sorted(samples),
                          decode=synth.bf16_to_f64)
    worst = 0.0
    for key, v in ref.items():
        s, r, h = key
        e = max_rel_err(o[s, r, h][None], v[None])
        worst = max(worst, e)
        assert e <= 2e-2, (key, e)
    print(f"[err] long-document sampled rows: max rel err {worst:.3e}", flush=True)
    assert np.all(np.isfinite(o))
