"""Helpers for GPU parity tests: move seeded inputs to the device and compare."""
import numpy as np
import torch

from paper_2609_26638_amd import synth


def to_dev(a: np.ndarray, dtype: str):
    """float32 array or uint16 bf16 bits -> device tensor."""
    if dtype == "bf16":
        t = torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16)
    else:
        t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    return t.cuda()


def to_f64(t: torch.Tensor) -> np.ndarray:
    if t.dtype == torch.bfloat16:
        return synth.bf16_to_f64(t.cpu().view(torch.int16).numpy().view(np.uint16))
    return t.cpu().double().numpy()


def dev_attn(ai):
    d = ai.dtype
    return dict(q=to_dev(ai.q, d), k_new=to_dev(ai.k_new, d), v_new=to_dev(ai.v_new, d),
                k_pool=to_dev(ai.k_pool, d), v_pool=to_dev(ai.v_pool, d),
                page_table=torch.from_numpy(ai.state.page_table).cuda(),
                kv_len=torch.from_numpy(ai.state.kv_len).cuda())


def max_rel_err(got: np.ndarray, ref: np.ndarray) -> float:
    """max over output vectors (last axis) of ||got - ref||_inf / ||ref||_inf."""
    num = np.abs(got - ref).max(axis=-1)
    den = np.abs(ref).max(axis=-1)
    return float((num / np.maximum(den, 1e-30)).max())
