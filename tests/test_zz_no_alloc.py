"""GPU: attn_hybrid_block_noalloc (the library's scratch array as workspace)
against attn_hybrid_block with a caller workspace, through the C ABI.

Two calls in a row on the same GPU, the second with a smaller input and a
different kernel, so the second call runs on the array the first one left
behind: outputs and the appended pools must be bit-identical to the
workspace entry point's (the same kernels and the same deterministic split),
and within the bf16 bound (2e-2 max relative error per output vector) of the
oracle.
"""
import numpy as np
import pytest
import torch

from oracle import attention as oa
from paper_2609_26638_amd import dvs, synth
from tests.gpu_util import dev_attn, max_rel_err, to_f64

pytestmark = pytest.mark.gpu

CASES = [
    # seed, S, L, n_causal, n_mask, Hq, Hkv, D, chunk_keys
    (61, 4, [0, 300, 5000, 9000], 32, 32, 16, 4, 128, 0),   # producer/consumer kernel, split items
    (62, 2, [100, 700], 16, 16, 16, 4, 128, 0),             # smaller: 4-wave balanced kernel
    (63, 2, [40, 1300], 8, 8, 16, 4, 96, 256),              # smaller still: aligned chunks
]


def _pair(case):
    seed, S, L, nc, nm, Hq, Hkv, D, ck = case
    print(f"[noalloc] seed={seed} S={S} L={L} rows={nc}+{nm} D={D} chunk={ck}", flush=True)
    ai = synth.make_attn_inputs(seed, S, L, nc, nm, Hq, Hkv, D, "bf16", std=1.0, scatter=True)
    a, b = dev_attn(ai), dev_attn(ai)
    err_a = torch.zeros(1, dtype=torch.int32, device="cuda")
    err_b = torch.zeros(1, dtype=torch.int32, device="cuda")
    out_a = dvs.attn_hybrid_block(a["q"], a["k_new"], a["v_new"], a["k_pool"], a["v_pool"],
                                  a["page_table"], a["kv_len"], nc, nm, ai.scale, err=err_a,
                                  chunk_keys=ck)
    out_b = dvs.attn_hybrid_block_noalloc(b["q"], b["k_new"], b["v_new"], b["k_pool"], b["v_pool"],
                                          b["page_table"], b["kv_len"], nc, nm, ai.scale,
                                          err=err_b, chunk_keys=ck)
    torch.cuda.synchronize()
    return ai, a, b, out_a, out_b, err_a, err_b


def test_noalloc_equals_workspace_entry_point_on_consecutive_calls():
    for case in CASES:
        ai, a, b, out_a, out_b, err_a, err_b = _pair(case)
        assert int(err_a.item()) == 0 and int(err_b.item()) == 0
        assert torch.equal(out_a.view(torch.int16), out_b.view(torch.int16))
        assert torch.equal(a["k_pool"].view(torch.int16), b["k_pool"].view(torch.int16))
        assert torch.equal(a["v_pool"].view(torch.int16), b["v_pool"].view(torch.int16))
        ref = oa.attn_hybrid_block(ai.as_f64("q"), ai.as_f64("k_new"), ai.as_f64("v_new"),
                                   ai.as_f64("k_pool"), ai.as_f64("v_pool"), ai.state.page_table,
                                   ai.state.kv_len, ai.n_causal, ai.n_mask, ai.scale)
        e = max_rel_err(to_f64(out_b), ref)
        print(f"[noalloc] max rel err vs oracle {e:.3e}", flush=True)
        assert e <= 2e-2


def test_noalloc_rejects_shapes_beyond_its_scratch():
    # aligned 64-key chunks over 64 long sequences need far more than the array
    S, R, Hq, Hkv, D, max_pages = 64, 64, 16, 4, 128, 1030
    need = dvs.attn_workspace_bytes(S, 32, 32, Hq, Hkv, D, max_pages, 64, dvs.DVS_BF16)
    assert need > (64 << 20)
    q = torch.zeros((S, R, Hq, D), dtype=torch.bfloat16, device="cuda")
    kn = torch.zeros((S, R, Hkv, D), dtype=torch.bfloat16, device="cuda")
    kp = torch.zeros((4, Hkv, 16, D), dtype=torch.bfloat16, device="cuda")
    vp = torch.zeros((4, Hkv, D, 16), dtype=torch.bfloat16, device="cuda")
    pt = torch.zeros((S, max_pages), dtype=torch.int32, device="cuda")
    kl = torch.zeros(S, dtype=torch.int32, device="cuda")
    with pytest.raises(dvs.DvsError, match="scratch"):
        dvs.attn_hybrid_block_noalloc(q, kn, kn, kp, vp, pt, kl, 32, 32, 0.1, chunk_keys=64)
