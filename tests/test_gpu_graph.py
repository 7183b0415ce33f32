"""GPU: decode steps captured into a HIP graph and replayed.

A step's inputs all live in device memory, so a replay of a captured fused
step (or AR step, or two-forward round) is the next step.  Each replay is
checked against the same step run eagerly on a second copy of the model and
state (same kernels, so bit-identical), with eager work and host
synchronisations between replays."""
import numpy as np
import pytest
import torch

from paper_2609_26638_amd import dvs
from tests.test_gpu_model_step import _dev_pools, _small_model, _widen_draft

pytestmark = pytest.mark.gpu

FIELDS = ("kv_len", "page_table", "num_pages", "boundary", "draft", "out_tokens", "out_count",
          "finished")


@pytest.mark.parametrize("mode", ["fused", "ar", "literal"])
def test_graph_replays_equal_eager_steps(mode):
    B, CH, REPLAYS = 8, 64, 6
    dtype = "bf16"
    w, base, kps, vps = _small_model(5, dtype)
    host = _widen_draft(base.state, B) if mode == "literal" else base.state.copy()
    host.out_tokens = np.full((base.S, 256), -1, np.int32)

    def make():
        m = dvs.DeviceModel(w, _dev_pools(kps, dtype), _dev_pools(vps, dtype), dtype)
        return m, dvs.DeviceState(host)

    def step(m, st):
        if mode == "literal":
            dvs.literal_round(m, st, B, chunk_keys=CH)
        elif mode == "fused":
            dvs.draft_verify_step(m, st, B, B, chunk_keys=CH)
        else:
            dvs.draft_verify_step(m, st, 1, 0, chunk_keys=CH)

    em, es = make()
    gm, gs = make()
    # one eager step on each allocates the workspaces
    step(em, es)
    step(gm, gs)
    torch.cuda.synchronize()
    g = dvs.capture(lambda: step(gm, gs))
    torch.cuda.synchronize()
    # capturing launches nothing: the graph state is still one step in
    a, b = es.to_host(host), gs.to_host(host)
    for f in FIELDS:
        np.testing.assert_array_equal(getattr(a, f), getattr(b, f), err_msg=f)
    for i in range(REPLAYS):
        g.replay()
        step(em, es)
        scratch = torch.randn(1 << 20, device="cuda").sum()   # unrelated eager work
        torch.cuda.synchronize()
        assert float(scratch) == float(scratch)
        assert int(gs.err.item()) == 0 and int(es.err.item()) == 0
        a, b = es.to_host(host), gs.to_host(host)
        for f in FIELDS:
            np.testing.assert_array_equal(getattr(b, f), getattr(a, f), err_msg=f"replay {i}: {f}")
        assert a.free_top == b.free_top
    assert int(b.out_count.min()) > int(host.out_count.min()) + REPLAYS
