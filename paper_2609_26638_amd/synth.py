"""Seeded synthetic inputs for the draft-verify step.

This module only draws random numbers and lays them out; it performs none of
the method's arithmetic (no attention, no argmax, no acceptance, no commit).
Both the CPU oracle's tests and the HIP path's tests/benchmark take their
inputs from here, so the two sides always see identical arrays.

Conventions
-----------
* Every tensor gets its own PCG64 stream spawned from ``SeedSequence(seed)``,
  in a fixed order, so adding a tensor never perturbs the others.
* bf16 tensors are produced in float32 and rounded to bf16 once, with
  round-to-nearest-even, and are carried as ``uint16`` bit patterns.
  ``bf16_to_f64`` expands them exactly.
* ``N(m, s)`` means mean ``m`` and standard deviation ``s``.

Workload shapes (document-OCR decoding: long vision+prompt prefix, short
draft blocks) follow the configurations used for parity tests and the
benchmark: tiny fp32 single layer; one bf16 layer at KV 2048; a 32-sequence
bf16 batch at KV 1k-8k; a 64-sequence bf16 batch at KV 4k-16k.
"""
from __future__ import annotations

import dataclasses
import math
import os

import numpy as np

PAGE_SIZE = 16


# ----------------------------------------------------------------------------
# bf16 helpers (bit-level; no rounding other than the one RNE conversion)
# ----------------------------------------------------------------------------

def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 -> bf16 with round-to-nearest-even; returns uint16 bits."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    out = np.empty(x.shape, dtype=np.uint16)
    flat_in = x.reshape(-1)
    flat_out = out.reshape(-1)
    step = 1 << 24
    for i in range(0, flat_in.size, step):
        u = flat_in[i:i + step].view(np.uint32)
        lsb = (u >> np.uint32(16)) & np.uint32(1)
        r = (u + np.uint32(0x7FFF) + lsb) >> np.uint32(16)
        flat_out[i:i + step] = r.astype(np.uint16)
    return out


def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    return (bits.astype(np.uint32) << np.uint32(16)).view(np.float32)


def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    return bf16_to_f32(bits).astype(np.float64)


_CHUNK = 1 << 22


def _normal(rng: np.random.Generator, shape, std: float, mean: float = 0.0,
            bf16: bool = False) -> np.ndarray:
    """N(mean, std) float32 (or RNE-rounded bf16 bits), drawn in fixed 4M-element
    chunks, each from its own child stream of ``rng``, in parallel threads."""
    n = int(np.prod(shape)) if len(shape) else 1
    out = np.empty(n, dtype=np.uint16 if bf16 else np.float32)
    nchunk = (n + _CHUNK - 1) // _CHUNK
    seeds = rng.bit_generator.seed_seq.spawn(nchunk) if nchunk else []

    def work(i):
        lo, hi = i * _CHUNK, min(n, (i + 1) * _CHUNK)
        g = np.random.Generator(np.random.PCG64(seeds[i]))
        x = g.standard_normal(hi - lo, dtype=np.float32)
        if std != 1.0:
            x *= np.float32(std)
        if mean != 0.0:
            x += np.float32(mean)
        out[lo:hi] = f32_to_bf16_bits(x) if bf16 else x

    if nchunk > 1:
        import concurrent.futures as cf
        with cf.ThreadPoolExecutor(max_workers=min(16, os.cpu_count() or 1)) as ex:
            list(ex.map(work, range(nchunk)))
    elif nchunk == 1:
        work(0)
    return out.reshape(shape)


# ----------------------------------------------------------------------------
# Paged KV state
# ----------------------------------------------------------------------------

@dataclasses.dataclass
class PagedState:
    """Integer decode state for S sequences over a shared page pool.

    kv_len[s]        committed KV length L_s (positions [0, L_s) hold KV)
    page_table[s, i] physical page of logical page i (-1 where unused)
    num_pages[s]     pages held by sequence s (= ceil((L_s + R) / 16))
    free_stack[0:free_top] physical pages that are free (top at the end)
    boundary[s]      last committed token x0 (no KV yet)
    draft[s, j]      draft token d_{j+1}, j in [0, n_causal-1)
    out_tokens, out_count, finished: committed output stream per sequence
    """
    kv_len: np.ndarray
    page_table: np.ndarray
    num_pages: np.ndarray
    free_stack: np.ndarray
    free_top: int
    boundary: np.ndarray
    draft: np.ndarray
    out_tokens: np.ndarray
    out_count: np.ndarray
    finished: np.ndarray
    pool_pages: int
    max_pages: int

    def copy(self) -> "PagedState":
        return PagedState(**{f.name: (getattr(self, f.name).copy()
                                      if isinstance(getattr(self, f.name), np.ndarray)
                                      else getattr(self, f.name))
                             for f in dataclasses.fields(self)})


def make_paged_state(rng_pages: np.random.Generator, kv_len: np.ndarray, n_rows: int,
                     max_pages: int, scatter: bool, slack: float = 0.10,
                     extra_pages: int = 0, n_causal: int = 1, max_new: int = 4096) -> PagedState:
    """Reserve ceil((L_s + n_rows)/16) pages per sequence from a pool.

    The pool holds ``ceil(sum * (1 + slack)) + extra_pages`` pages.  With
    ``scatter`` the physical ids are a seeded random permutation; otherwise
    sequences take consecutive ids.  Unreserved pages form the free stack, in
    the order drawn.
    """
    S = kv_len.shape[0]
    need = [(int(L) + n_rows + PAGE_SIZE - 1) // PAGE_SIZE for L in kv_len]
    total = sum(need)
    pool = int(math.ceil(total * (1.0 + slack))) + extra_pages
    ids = rng_pages.permutation(pool).astype(np.int32) if scatter else np.arange(pool, dtype=np.int32)
    pt = np.full((S, max_pages), -1, dtype=np.int32)
    off = 0
    for s in range(S):
        if need[s] > max_pages:
            raise ValueError("max_pages too small for the generated KV length")
        pt[s, :need[s]] = ids[off:off + need[s]]
        off += need[s]
    free = np.full(pool, -1, dtype=np.int32)
    rest = ids[off:]
    free[:rest.size] = rest
    return PagedState(
        kv_len=kv_len.astype(np.int32).copy(),
        page_table=pt,
        num_pages=np.array(need, dtype=np.int32),
        free_stack=free,
        free_top=int(rest.size),
        boundary=np.zeros(S, dtype=np.int32),
        draft=np.zeros((S, max(n_causal - 1, 0)), dtype=np.int32),
        out_tokens=np.full((S, max_new), -1, dtype=np.int32),
        out_count=np.zeros(S, dtype=np.int32),
        finished=np.zeros(S, dtype=np.int32),
        pool_pages=pool,
        max_pages=max_pages,
    )


# ----------------------------------------------------------------------------
# Attention-step inputs (single layer, given Q/K/V)
# ----------------------------------------------------------------------------

@dataclasses.dataclass
class AttnInputs:
    dtype: str            # "f32" or "bf16"
    S: int
    n_causal: int
    n_mask: int
    Hq: int
    Hkv: int
    D: int
    q: np.ndarray          # [S, R, Hq, D]   float32 or uint16 bf16 bits
    k_new: np.ndarray      # [S, R, Hkv, D]
    v_new: np.ndarray      # [S, R, Hkv, D]
    k_pool: np.ndarray     # [pool, Hkv, 16, D]   (slot-major pages)
    v_pool: np.ndarray     # [pool, Hkv, D, 16]   (head-dim-major pages)
    state: PagedState
    scale: float

    @property
    def R(self) -> int:
        return self.n_causal + self.n_mask

    def as_f64(self, name: str) -> np.ndarray:
        a = getattr(self, name)
        return bf16_to_f64(a) if self.dtype == "bf16" else a.astype(np.float64)


def make_attn_inputs(seed: int, S: int, kv_lens, n_causal: int, n_mask: int, Hq: int,
                     Hkv: int, D: int, dtype: str, std: float = 1.0, scatter: bool = True,
                     max_pages: int | None = None, slack: float = 0.10,
                     extra_pages: int = 0) -> AttnInputs:
    """Q, block K/V and a paged KV cache, all ~N(0, std); cache in a shared pool.

    ``kv_lens`` is either an explicit list or a (lo, hi) pair for U{lo..hi}.
    """
    ss = np.random.SeedSequence(seed)
    r_len, r_pages, r_q, r_k, r_v, r_kp, r_vp = [np.random.Generator(np.random.PCG64(c))
                                                 for c in ss.spawn(7)]
    if isinstance(kv_lens, tuple):
        lo, hi = kv_lens
        L = r_len.integers(lo, hi + 1, size=S).astype(np.int32)
    else:
        L = np.asarray(kv_lens, dtype=np.int32)
        assert L.shape == (S,)
    R = n_causal + n_mask
    if max_pages is None:
        max_pages = (int(L.max()) + 4 * R + PAGE_SIZE - 1) // PAGE_SIZE + 2
    st = make_paged_state(r_pages, L, R, max_pages, scatter, slack=slack,
                          extra_pages=extra_pages, n_causal=n_causal)
    P = st.pool_pages
    arrs = []
    for rng, shape in ((r_q, (S, R, Hq, D)), (r_k, (S, R, Hkv, D)), (r_v, (S, R, Hkv, D)),
                       (r_kp, (P, Hkv, PAGE_SIZE, D)), (r_vp, (P, Hkv, D, PAGE_SIZE))):
        arrs.append(_normal(rng, shape, std, bf16=(dtype == "bf16")))
    return AttnInputs(dtype, S, n_causal, n_mask, Hq, Hkv, D, *arrs, state=st,
                      scale=1.0 / math.sqrt(D))


# ----------------------------------------------------------------------------
# Logits + drafts for the argmax / acceptance stage
# ----------------------------------------------------------------------------

PLANT_VALUE = 32.0        # exactly representable in bf16
PLANT_CLAMP = 31.75       # every other logit is clamped below the planted one


@dataclasses.dataclass
class LogitInputs:
    logits: np.ndarray     # [S, R, V] uint16 bf16 bits (or float32)
    planted: np.ndarray    # [S, n_causal] token whose logit was raised (-1 = none)
    draft: np.ndarray      # [S, n_causal - 1] previous draft d_1..d_{B-1}
    dtype: str


def make_logit_inputs(seed: int, S: int, n_causal: int, n_mask: int, V: int, std: float,
                      match_p: float, dtype: str = "bf16", plant: bool = True) -> LogitInputs:
    """Logits ~N(0, std) and drafts that equal the verify-row top-1 w.p. match_p.

    To know each verify row's top-1 without computing an argmax here, one
    uniformly drawn token per verify row gets the value 32.0 and every other
    logit of that row is clamped to at most 31.75 (a 8-sigma value at std 4,
    so the clamp does not change the draw in practice).  Draft d_j copies the
    planted token of verify row j-1 with probability ``match_p`` and is
    otherwise uniform over the other V-1 tokens.  Mask rows are left as drawn,
    so exact ties occur among them naturally in bf16.
    """
    ss = np.random.SeedSequence([seed, 0x10917])
    r_log, r_plant, r_match, r_other = [np.random.Generator(np.random.PCG64(c))
                                        for c in ss.spawn(4)]
    R = n_causal + n_mask
    x = _normal(r_log, (S, R, V), std)
    planted = np.full((S, n_causal), -1, dtype=np.int32)
    if plant:
        tau = r_plant.integers(0, V, size=(S, n_causal)).astype(np.int32)
        np.minimum(x[:, :n_causal, :], np.float32(PLANT_CLAMP), out=x[:, :n_causal, :])
        si, ri = np.meshgrid(np.arange(S), np.arange(n_causal), indexing="ij")
        x[si, ri, tau] = np.float32(PLANT_VALUE)
        planted = tau
    nd = max(n_causal - 1, 0)
    match = r_match.random(size=(S, nd)) < match_p
    u = r_other.integers(0, V - 1, size=(S, nd)).astype(np.int32)
    base = planted[:, :nd] if plant else np.zeros((S, nd), np.int32)
    other = u + (u >= base).astype(np.int32)
    draft = np.where(match, base, other).astype(np.int32)
    logits = f32_to_bf16_bits(x) if dtype == "bf16" else x
    return LogitInputs(logits=logits, planted=planted, draft=draft, dtype=dtype)


def tied_logits(seed: int, S: int, R: int, V: int, levels: int = 4) -> np.ndarray:
    """float32 logits drawn from a handful of values (with +0.0 and -0.0),
    so that exact ties and signed zeros are frequent."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 0x71E5])))
    vals = np.array([-0.0, 0.0, 1.5, -2.25, 3.0, 0.5][:max(levels, 2)], dtype=np.float32)
    return vals[rng.integers(0, vals.size, size=(S, R, V))]


# ----------------------------------------------------------------------------
# Random-init single/multi-layer decoder weights
# ----------------------------------------------------------------------------

@dataclasses.dataclass
class ModelWeights:
    """Decoder weights (float32 masters; bf16 variants derive by RNE).

    embed has V+1 rows: rows [0, V) are the vocabulary, row V is the mask
    token [M] (mean-resized: per-dimension normal fitted to the other rows).
    Linear maps are stored [in, out] and applied as ``x @ W``.
    """
    V: int
    H: int
    Hq: int
    Hkv: int
    D: int
    n_layers: int
    ffn: int                      # 0 = no MLP
    embed: np.ndarray             # [V+1, H]
    wq: list
    wk: list
    wv: list
    wo: list
    g_attn: list                  # RMSNorm gains, N(1, gain_std)
    g_mlp: list
    w_gate: list
    w_up: list
    w_down: list
    g_final: np.ndarray
    lm_head: np.ndarray           # [H, V]
    rope_theta: float = 10000.0
    eps: float = 1e-6

    @property
    def mask_id(self) -> int:
        return self.V


def make_model_weights(seed: int, V: int, H: int, Hq: int, Hkv: int, D: int,
                       n_layers: int, ffn: int, std: float = 0.02,
                       gain_std: float = 0.1) -> ModelWeights:
    ss = np.random.SeedSequence([seed, 0x3E16])
    rngs = [np.random.Generator(np.random.PCG64(c)) for c in ss.spawn(4 + 7 * n_layers)]
    it = iter(rngs)
    emb = _normal(next(it), (V + 1, H), std)
    mu = emb[:V].mean(axis=0, dtype=np.float64)
    sd = emb[:V].std(axis=0, dtype=np.float64)
    emb[V] = (mu + sd * next(it).standard_normal(H)).astype(np.float32)
    wq, wk, wv, wo, wg, wu, wd = [], [], [], [], [], [], []
    for _ in range(n_layers):
        wq.append(_normal(next(it), (H, Hq * D), std))
        wk.append(_normal(next(it), (H, Hkv * D), std))
        wv.append(_normal(next(it), (H, Hkv * D), std))
        wo.append(_normal(next(it), (Hq * D, H), std))
        if ffn:
            wg.append(_normal(next(it), (H, ffn), std))
            wu.append(_normal(next(it), (H, ffn), std))
            wd.append(_normal(next(it), (ffn, H), std))
        else:
            for _ in range(3):
                next(it)
    lm = _normal(next(it), (H, V), std)
    # RMSNorm gains: N(1, gain_std) per element (a trained model's gains are
    # not all one; distinct gains make a swapped or dropped gain visible).
    gss = np.random.SeedSequence([seed, 0x6A1E])
    g_rng = [np.random.Generator(np.random.PCG64(c)) for c in gss.spawn(2 * n_layers + 1)]
    g_attn = [_normal(g_rng[2 * l], (H,), gain_std, mean=1.0) for l in range(n_layers)]
    g_mlp = [_normal(g_rng[2 * l + 1], (H,), gain_std, mean=1.0) for l in range(n_layers)]
    g_final = _normal(g_rng[-1], (H,), gain_std, mean=1.0)
    return ModelWeights(V=V, H=H, Hq=Hq, Hkv=Hkv, D=D, n_layers=n_layers, ffn=ffn,
                        embed=emb, wq=wq, wk=wk, wv=wv, wo=wo,
                        g_attn=g_attn, g_mlp=g_mlp,
                        w_gate=wg, w_up=wu, w_down=wd,
                        g_final=g_final, lm_head=lm)


# ----------------------------------------------------------------------------
# Named workloads
# ----------------------------------------------------------------------------

def tiny_step_inputs(seed: int = 0):
    """Tiny fp32 single-layer step: 1 sequence, L=256, 4 heads x 64, B=8,
    vocab 1024; weights and KV ~N(0, 0.02); x0 and drafts uniform."""
    V, H, Hq, Hkv, D, B, L = 1024, 256, 4, 4, 64, 8, 256
    w = make_model_weights(seed, V, H, Hq, Hkv, D, n_layers=1, ffn=0, std=0.02)
    ai = make_attn_inputs(seed, 1, [L], B, B, Hq, Hkv, D, "f32", std=0.02,
                          scatter=False, extra_pages=4)
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 0x70C])))
    ai.state.boundary[:] = rng.integers(0, V, size=1)
    ai.state.draft[:] = rng.integers(0, V, size=(1, B - 1))
    return w, ai


def one_layer_attn_inputs(seed: int = 1) -> AttnInputs:
    """One bf16 decoder-layer attention: batch 1, KV 2048 (1536 vision + 512
    text), 16 q / 4 kv heads, head_dim 128, B=16 -> 32 rows, 16-token pages."""
    return make_attn_inputs(seed, 1, [2048], 16, 16, 16, 4, 128, "bf16", std=1.0,
                            scatter=False)


def batched_serving_inputs(seed: int = 2, S: int = 32, kv=(1024, 8192), B: int = 16,
                           V: int = 65536, match_p: float = 0.9):
    ai = make_attn_inputs(seed, S, kv, B, B, 16, 4, 128, "bf16", std=1.0, scatter=True)
    li = make_logit_inputs(seed, S, B, B, V, 4.0, match_p)
    ai.state.draft[:] = li.draft
    return ai, li


def long_document_inputs(seed: int = 4, S: int = 64, kv=(4096, 16384), B: int = 32,
                         V: int = 65536, match_p: float = 0.95):
    ai = make_attn_inputs(seed, S, kv, B, B, 16, 4, 128, "bf16", std=1.0, scatter=True)
    li = make_logit_inputs(seed, S, B, B, V, 4.0, match_p)
    ai.state.draft[:] = li.draft
    return ai, li


@dataclasses.dataclass
class StackInputs:
    weights: ModelWeights
    vision: np.ndarray        # [S, n_vision, H] float32 ~N(0, 1)
    prompt: np.ndarray        # [S, n_prompt] int32 uniform over the vocabulary
    state: PagedState         # kv_len = 0, pages for the prefill window and growth
    B: int
    max_new: int

    @property
    def P(self) -> int:
        return self.vision.shape[1] + self.prompt.shape[1]

    def prefix_tokens(self) -> np.ndarray:
        """[S, P] ids: -1 for the vision rows (take the given vectors), then the prompt."""
        S = self.vision.shape[0]
        ids = np.full((S, self.P), -1, dtype=np.int32)
        ids[:, self.vision.shape[1]:] = self.prompt
        return ids

    def x_prefix(self) -> np.ndarray:
        """[S, P, H] float32: the vision vectors, zeros for the prompt rows."""
        S, nv, H = self.vision.shape
        x = np.zeros((S, self.P, H), dtype=np.float32)
        x[:, :nv] = self.vision
        return x


def stack_state(seed: int, S: int, P: int, B: int, max_new: int, window: int) -> PagedState:
    """Fresh decode state for a prefix of P rows (kv_len = 0): pages for the
    prefill and a window of `window` rows, scattered, and a pool with room
    for max_new tokens of growth per sequence."""
    ss = np.random.SeedSequence([seed, 0x5AC4])
    r_pages = np.random.Generator(np.random.PCG64(ss.spawn(3)[2]))
    max_pages = (P + max_new + window + PAGE_SIZE - 1) // PAGE_SIZE + 2
    growth = S * ((max_new + window + PAGE_SIZE - 1) // PAGE_SIZE + 2)
    st = make_paged_state(r_pages, np.full(S, P, dtype=np.int64), window, max_pages, scatter=True,
                          slack=0.0, extra_pages=growth, n_causal=B, max_new=max_new)
    st.kv_len[:] = 0
    return st


def decoder_stack_inputs(seed: int = 3, S: int = 8, n_layers: int = 16, H: int = 1536,
                         Hq: int = 16, Hkv: int = 4, D: int = 96, ffn: int = 4096, V: int = 65536,
                         n_vision: int = 1024, n_prompt: int = 64, B: int = 16,
                         max_new: int = 1024) -> StackInputs:
    """Random-init decoder stack (weights N(0, 0.02)), a prefix of synthetic
    vision embeddings N(0, 1) plus uniform prompt tokens, block size B."""
    w = make_model_weights(seed, V, H, Hq, Hkv, D, n_layers, ffn, std=0.02)
    ss = np.random.SeedSequence([seed, 0x5AC4])
    r_vis, r_prompt, _ = [np.random.Generator(np.random.PCG64(c)) for c in ss.spawn(3)]
    vision = _normal(r_vis, (S, n_vision, H), 1.0)
    prompt = r_prompt.integers(0, V, size=(S, n_prompt)).astype(np.int32)
    P = n_vision + n_prompt
    st = stack_state(seed, S, P, B, max_new, 2 * B)
    return StackInputs(weights=w, vision=vision, prompt=prompt, state=st, B=B, max_new=max_new)
