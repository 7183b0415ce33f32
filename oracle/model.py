"""Oracle: a random-init decoder, greedy AR decoding and fused self-speculative
decoding (float64).

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__``).

The paper fixes the decoding algorithm but not the decoder architecture; the
layers below are a plain pre-norm decoder, read as follows:

* RMSNorm: ``x / sqrt(mean(x^2) + eps) * g``.
* Linear maps without bias, stored [in, out], applied as ``x @ W``.
* Rotary position embedding, rotate-half over the whole head dimension:
  pairs ``(x_i, x_{i + D/2})`` are rotated by angle ``pos * theta^(-2i/D)``.
* Attention: the hybrid-mask block attention of ``oracle.attention``.
* Optional SwiGLU MLP: ``(silu(h Wg) * (h Wu)) Wd``.
* Final RMSNorm, untied LM head over the V vocabulary rows.
* Input rows are embedding rows; the mask token [M] is the extra embedding
  row V (Method "AR-to-Diffusion Conversion": the only architectural
  addition is a learned embedding for [M]).

Decoders (all from a given committed state, see ``oracle.decode``):

* ``ar_step``   one greedy AR step: window ``[x0]`` (1 causal row), commit
  its top-1 (Preliminaries, eq. ``eq:ar`` under greedy decoding).
* ``fused_step`` one self-speculative step: window ``[x0, d_1..d_{B-1}]``
  (causal) followed by B ``[M]`` rows (bidirectional within the block);
  accept, commit, roll back (``oracle.decode``).
* ``diffusion_block`` direct block-diffusion decoding of one block
  (appendix "Direct Block-Diffusion Decoding", see ``oracle.decode``):
  denoising forwards over ``[x0, b_1..b_B]`` until every position is
  revealed, then a cache-write forward over ``[x0, b_1..b_{B-1}]`` and the
  commit of the block.
* ``prefill``   the prefix as causal rows, plus B ``[M]`` rows whose top-1
  tokens are the first draft; the last prefix row's top-1 is the first
  committed token and boundary (appendix item State: the initial boundary is
  produced by prefill).

The committed streams of ``ar_step`` and ``fused_step`` loops coincide in
exact arithmetic (appendix "AR-Equivalence and Equality Testing", Argument).
"""
from __future__ import annotations

import numpy as np

from . import attention as oattn
from . import decode as odec


def rmsnorm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * g


def rope(x: np.ndarray, pos: np.ndarray, theta: float) -> np.ndarray:
    """x [..., n, D] rotated by positions pos [...] (broadcast over heads)."""
    D = x.shape[-1]
    half = D // 2
    i = np.arange(half, dtype=np.float64)
    inv = theta ** (-2.0 * i / D)                       # [half]
    ang = pos[..., None, None].astype(np.float64) * inv  # [..., 1, half]
    c, s = np.cos(ang), np.sin(ang)
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x1 * s + x2 * c], axis=-1)


def silu(x: np.ndarray) -> np.ndarray:
    return x / (1.0 + np.exp(-x))


class OracleModel:
    """float64 copy of the weights plus per-layer paged KV pools."""

    def __init__(self, w, k_pools, v_pools, page_size: int = 16, bf16_bits: bool = False):
        """w: synth.ModelWeights-like (float32 or, with bf16_bits, uint16 arrays).
        k_pools: per layer [P, Hkv, page_size, D]; v_pools: per layer
        [P, Hkv, D, page_size] (copied)."""
        cv = (lambda a: (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)) \
            if bf16_bits else (lambda a: np.asarray(a, dtype=np.float64))
        self.V, self.H, self.Hq, self.Hkv, self.D = w.V, w.H, w.Hq, w.Hkv, w.D
        self.n_layers, self.ffn = w.n_layers, w.ffn
        self.theta, self.eps = w.rope_theta, w.eps
        self.embed = cv(w.embed)
        self.wq = [cv(a) for a in w.wq]
        self.wk = [cv(a) for a in w.wk]
        self.wv = [cv(a) for a in w.wv]
        self.wo = [cv(a) for a in w.wo]
        self.g_attn = [cv(a) for a in w.g_attn]
        self.g_mlp = [cv(a) for a in w.g_mlp]
        self.w_gate = [cv(a) for a in w.w_gate]
        self.w_up = [cv(a) for a in w.w_up]
        self.w_down = [cv(a) for a in w.w_down]
        self.g_final = cv(w.g_final)
        self.lm_head = cv(w.lm_head)
        self.k_pools = [cv(a).copy() for a in k_pools]
        self.v_pools = [cv(a).copy() for a in v_pools]
        self.page_size = page_size

    @property
    def mask_id(self) -> int:
        return self.V

    def forward(self, x: np.ndarray, st, n_causal: int, n_mask: int,
                group: int = 0) -> np.ndarray:
        """Rows x [S, R, H] (already embedded) at positions kv_len[s] + r
        (``group`` > 0: mask rows in groups, at the positions of
        ``attention.window_positions``, attending with the grouped mask).

        Appends every layer's window K/V to the pools (window row r at slot
        kv_len[s] + r) and returns logits [S, R, V].
        """
        S, R, _ = x.shape
        pos = np.stack([oattn.window_positions(int(L), n_causal, n_mask, group)
                        for L in st.kv_len])
        scale = 1.0 / np.sqrt(self.D)
        for l in range(self.n_layers):
            h = rmsnorm(x, self.g_attn[l], self.eps)
            q = (h @ self.wq[l]).reshape(S, R, self.Hq, self.D)
            k = (h @ self.wk[l]).reshape(S, R, self.Hkv, self.D)
            v = (h @ self.wv[l]).reshape(S, R, self.Hkv, self.D)
            q = rope(q, pos, self.theta)
            k = rope(k, pos, self.theta)
            o = oattn.attn_hybrid_block(q, k, v, self.k_pools[l], self.v_pools[l],
                                        st.page_table, st.kv_len, n_causal, n_mask, scale,
                                        self.page_size, group=group)
            x = x + o.reshape(S, R, self.Hq * self.D) @ self.wo[l]
            if self.ffn:
                h2 = rmsnorm(x, self.g_mlp[l], self.eps)
                x = x + (silu(h2 @ self.w_gate[l]) * (h2 @ self.w_up[l])) @ self.w_down[l]
        y = rmsnorm(x, self.g_final, self.eps)
        return y @ self.lm_head

    def window_tokens(self, st, B: int) -> np.ndarray:
        """Fused-step inputs: [x0, d_1..d_{B-1}] then B copies of [M]."""
        S = st.kv_len.shape[0]
        tok = np.empty((S, 2 * B), dtype=np.int64)
        tok[:, 0] = st.boundary
        tok[:, 1:B] = st.draft[:, :B - 1]
        tok[:, B:] = self.mask_id
        return tok

    def fused_step(self, st, B: int, eos_id: int = -1, max_new=None):
        """One self-speculative step; returns (logits, argmax, accept_len, err)."""
        tok = self.window_tokens(st, B)
        logits = self.forward(self.embed[tok], st, B, B)
        am = odec.top1_rows(logits)
        A = odec.accept(am, st.draft, B)
        err = odec.kv_commit(st, A, am, B, B, eos_id=eos_id, max_new=max_new,
                             page_size=self.page_size)
        return logits, am, A, err

    def multidraft_step(self, st, B: int, eos_id: int = -1, max_new=None):
        """One self-speculative step with a draft per possible acceptance
        (the structured-mask AR-diffusion hybrid the paper cites in its
        related work): window [x0, d_1..d_{B-1}] (causal) followed by B groups
        of B [M] rows.  Group k assumes A = k: its rows sit right after d_k
        (at L + k + 1 + i, the first standing in for the unknown a_{k+1}),
        see the cache, the causal rows 0..k and their own group.  After
        acceptance A the next draft is group A's top-1 (rows 0..B-2 of the
        group), so it is conditioned on the accepted tokens only.  Pages must
        cover [L, L + B + B*B).  Returns (logits, argmax, accept_len, err)."""
        S = st.kv_len.shape[0]
        tok = np.empty((S, B + B * B), dtype=np.int64)
        tok[:, 0] = st.boundary
        tok[:, 1:B] = st.draft[:, :B - 1]
        tok[:, B:] = self.mask_id
        logits = self.forward(self.embed[tok], st, B, B * B, group=B)
        am = odec.top1_rows(logits)
        A = odec.accept(am, st.draft, B)
        err = odec.kv_commit(st, A, am, B, B * B, eos_id=eos_id, max_new=max_new,
                             page_size=self.page_size, draft_group=B)
        return logits, am, A, err

    def literal_round(self, st, B: int, eos_id: int = -1, max_new=None, tau_d=None):
        """The paper's two-forward round (appendix "Self-Speculative Decoding
        and KV-Cache Update"); see oracle.decode.  Pages must cover
        [L, L + B + 2).  Returns (draft logits, verify logits, verify top-1,
        accept_len, err).

        tau_d (experiments, "Draft Schedule"): the draft is refined over
        several forwards instead of one.  The B + 1 predictions of the draft
        window (a0 from the boundary row, d_j from mask row j) are revealed
        like a diffusion block (``decode.reveal`` with threshold tau_d);
        revealed a0, d_1..d_{B-1} replace the [M] inputs of mask rows 1..B in
        the next draft forward (d_B has no input slot).  ``self.draft_steps``
        records the draft forwards of the last call; tau_d = None is the
        one-shot draft (one forward)."""
        S = st.kv_len.shape[0]
        live = st.finished == 0
        # draft forward(s): [x0, [M] x B] (revealed tokens in place of [M])
        block = np.full((S, B + 1), -1, dtype=np.int64)
        steps = 0
        while True:
            tok = np.empty((S, B + 1), dtype=np.int64)
            tok[:, 0] = st.boundary
            tok[:, 1:] = np.where(block[:, :B] < 0, self.mask_id, block[:, :B])
            logits_d = self.forward(self.embed[tok], st, 1, B)
            steps += 1
            if tau_d is None:
                block = odec.top1_rows(logits_d).astype(np.int64)
                break
            am = np.zeros((S, B + 1), dtype=np.int32)
            conf = np.zeros((S, B + 1), dtype=np.float64)
            for s in range(S):
                for r in range(B + 1):
                    am[s, r], conf[s, r] = odec.top1_confidence(logits_d[s, r])
            block = odec.reveal(block, am, conf, tau_d, st.finished)
            if not np.any((block < 0).any(axis=1) & live):
                break
        self.draft_steps = steps
        a0 = block[:, 0].copy()
        st.draft[live, :B] = block[live, 1:B + 1]
        st.kv_len[live] += 1                      # x0's causal KV is kept
        # verify forward: [a0, d_1..d_B] under causal attention from L + 1
        tok_v = np.empty((S, B + 1), dtype=np.int64)
        tok_v[:, 0] = a0
        tok_v[:, 1:] = st.draft[:, :B]
        logits_v = self.forward(self.embed[tok_v], st, B + 1, 0)
        am_v = odec.top1_rows(logits_v)
        A = odec.accept(am_v, st.draft, B + 1)
        err = odec.kv_commit(st, A, am_v, B + 1, 0, eos_id=eos_id, max_new=max_new,
                             page_size=self.page_size, lead=a0, window=B + 2)
        return logits_d, logits_v, am_v, A, err

    def sampled_round(self, st, B: int, T: float, u: np.ndarray, eos_id: int = -1,
                      max_new=None):
        """The two-forward round under sampling at temperature T with the
        standard acceptance-rejection rule (see oracle.decode).  u [S, 2B + 2]
        uniforms: u[:, 0] samples a0, u[:, j] samples d_j (j = 1..B),
        u[:, B + j] tests d_j, u[:, 2B + 1] samples the final token.  Pages
        must cover [L, L + B + 2).  Returns (draft logits, verify logits, A,
        final tokens, err)."""
        S = st.kv_len.shape[0]
        live = st.finished == 0
        tok = np.empty((S, B + 1), dtype=np.int64)
        tok[:, 0] = st.boundary
        tok[:, 1:] = self.mask_id
        logits_d = self.forward(self.embed[tok], st, 1, B)
        q = np.array([[odec.softmax_t(logits_d[s, r], T) for r in range(B + 1)] for s in range(S)])
        drafted = np.array([[odec.sample_index(q[s, r], u[s, r]) for r in range(B + 1)]
                            for s in range(S)], dtype=np.int64)
        a0 = drafted[:, 0].copy()
        st.draft[live, :B] = drafted[live, 1:]
        st.kv_len[live] += 1
        tok_v = np.empty((S, B + 1), dtype=np.int64)
        tok_v[:, 0] = a0
        tok_v[:, 1:] = st.draft[:, :B]
        logits_v = self.forward(self.embed[tok_v], st, B + 1, 0)
        A = np.zeros(S, dtype=np.int32)
        final = np.zeros(S, dtype=np.int32)
        am = np.zeros((S, B + 1), dtype=np.int32)
        for s in range(S):
            p = np.array([odec.softmax_t(logits_v[s, r], T) for r in range(B + 1)])
            A[s] = odec.stochastic_accept(p[:B], q[s, 1:], st.draft[s, :B], u[s, B + 1:2 * B + 1])
            w = odec.resample_weights(p[A[s]], None if A[s] == B else q[s, A[s] + 1])
            final[s] = odec.sample_index(w, u[s, 2 * B + 1])
            am[s, A[s]] = final[s]
        err = odec.kv_commit(st, A, am, B + 1, 0, eos_id=eos_id, max_new=max_new,
                             page_size=self.page_size, lead=a0, window=B + 2)
        return logits_d, logits_v, A, final, err

    def diffusion_denoise(self, st, block: np.ndarray, tau_c: float):
        """One denoising forward over [x0, b_1..b_B] (1 causal row, B block
        rows; -1 = [M]) and its reveal.  kv_len is unchanged.  Returns
        (logits [S, B+1, V], top-1 [S, B], confidence [S, B], new block):
        column p-1 of the last three is block position p, from row p-1."""
        S, B = block.shape
        tok = np.empty((S, B + 1), dtype=np.int64)
        tok[:, 0] = st.boundary
        tok[:, 1:] = np.where(block < 0, self.mask_id, block)
        logits = self.forward(self.embed[tok], st, 1, B)
        am = np.zeros((S, B), dtype=np.int32)
        conf = np.zeros((S, B), dtype=np.float64)
        for s in range(S):
            for p in range(B):
                am[s, p], conf[s, p] = odec.top1_confidence(logits[s, p])
        return logits, am, conf, odec.reveal(block, am, conf, tau_c, st.finished)

    def diffusion_block(self, st, B: int, tau_c: float, eos_id: int = -1, max_new=None):
        """Decode one block by direct block diffusion.  Pages must cover
        [L, L + B + 1) on entry (the commit leaves them so).  Returns
        (block [S, B], denoising forwards, err); the block costs that many
        forwards plus one cache-write forward."""
        S = st.kv_len.shape[0]
        block = np.full((S, B), -1, dtype=np.int64)
        steps = 0
        while np.any((block < 0).any(axis=1) & (st.finished == 0)):
            _, _, _, block = self.diffusion_denoise(st, block, tau_c)
            steps += 1
            assert steps <= B, "a denoising step revealed nothing"
        # cache-write forward: x0 and b_1..b_{B-1} as causal rows
        tok = np.empty((S, B), dtype=np.int64)
        tok[:, 0] = st.boundary
        tok[:, 1:] = np.where(block[:, :B - 1] < 0, self.mask_id, block[:, :B - 1])
        self.forward(self.embed[tok], st, B, 0)
        err = odec.kv_commit(st, None, None, B, 0, eos_id=eos_id, max_new=max_new,
                             page_size=self.page_size, window=B + 1, block_runs=block)
        return block, steps, err

    def ar_step(self, st, eos_id: int = -1, max_new=None):
        """One greedy AR step: window [x0]; commits its top-1."""
        tok = st.boundary[:, None].astype(np.int64)
        logits = self.forward(self.embed[tok], st, 1, 0)
        am = odec.top1_rows(logits)
        A = np.zeros(st.kv_len.shape[0], dtype=np.int32)
        err = odec.kv_commit(st, A, am, 1, 0, eos_id=eos_id, max_new=max_new,
                             page_size=self.page_size)
        return logits, am, err

    def prefill(self, st, x_prefix: np.ndarray, B: int) -> np.ndarray:
        """Prefix rows x_prefix [S, P, H] at positions 0..P-1 (kv_len must be 0),
        plus B [M] rows.  Sets kv_len=P, boundary = top-1 of row P-1 (committed
        as the first output token), draft = top-1 of mask rows 0..B-2.
        Pages must already cover P + B positions.  Returns the logits."""
        S, P, _ = x_prefix.shape
        assert np.all(st.kv_len == 0)
        xm = np.broadcast_to(self.embed[self.mask_id], (S, B, self.H))
        x = np.concatenate([x_prefix, xm], axis=1)
        logits = self.forward(x, st, P, B)
        am = odec.top1_rows(logits)
        st.kv_len[:] = P
        st.boundary[:] = am[:, P - 1]
        if st.draft.shape[1]:
            st.draft[:] = am[:, P:P + st.draft.shape[1]]
        for s in range(S):
            st.out_tokens[s, st.out_count[s]] = am[s, P - 1]
            st.out_count[s] += 1
        return logits
