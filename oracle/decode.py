"""Oracle: top-1 selection, greedy acceptance, commit and KV rollback.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__``).

The fused step
--------------
The paper's serving round uses two forwards: a draft forward over
``[x0, [M] x B]`` and a causal verify forward over ``[a0, d_1..d_B]``
(appendix "Self-Speculative Decoding and KV-Cache Update").  The step
implemented here carries both in one forward of ``n_causal + n_mask`` rows:

* causal rows r = 0..n_causal-1 take ``[x0, d_1, ..., d_{n_causal-1}]`` and
  row r predicts position ``L + r + 1`` (shifted prediction: the logit at
  position p-1 gives token p; Method "Joint AR-Diffusion Training", and the
  appendix's "Direct Block-Diffusion Decoding").  So ``a_j = top1(row j-1)``.
* mask rows r = n_causal..R-1 take ``[M]`` and their top-1 tokens form the
  next draft: ``d'_j = top1(row n_causal + j - 1)``, j = 1..W, where W is the
  draft width (n_causal - 1 in the fused step).  A window without mask rows
  (plain AR) leaves the draft unchanged.  Which draft to carry after a
  partial acceptance is not fixed by the paper (its round always redrafts
  from the true boundary); reusing the mask rows unconditionally is this
  implementation's reading, and its content is parity unpinned beyond
  oracle == GPU and the invariants that hold for any draft.

Acceptance (Method "Self-Speculative Decoding"; appendix item Accept): A is
the length of the longest prefix with ``d_j == a_j``; with n_causal verify
rows the drafts that can be checked are d_1..d_{n_causal-1}, so
``0 <= A <= n_causal - 1``.  The step commits ``d_1..d_A`` and ``a_{A+1}``
(the verifier's own prediction), i.e. 1..n_causal tokens.

Cache update (appendix item Cache update): the causal KV of x0 and the
accepted drafts is kept, so ``L' = L + A + 1``; every other slot written by
the window, in particular every mask-row slot, is rolled back.  The new
boundary is the last committed token (item Next round).  A stop condition
(EOS or the output budget) truncates the committed run at that token and
freezes the sequence (item Next round, last sentence).

The paper's own round (two forwards)
------------------------------------
The appendix round is also kept here, as written: a draft forward over
``[x0, [M] x B]`` (1 causal row, B mask rows) gives ``a0`` from the boundary
row and ``d_j`` from mask row j (j = 1..B); x0's causal KV from that forward
is kept (``kv_len`` + 1); a verify forward over ``[a0, d_1..d_B]`` (B + 1
causal rows, no mask rows) at positions ``L + 1 ..`` overwrites the draft's
mask-row slots and gives ``a_j = top1(row j-1)``, j = 1..B+1; A in 0..B is the
longest prefix with ``d_j == a_j``; the round commits ``a0, d_1..d_A,
a_{A+1}`` (2..B+2 tokens).  Its commit is ``kv_commit`` with ``lead = a0``:
the run starts with the lead token and, since the kept x0 is already in
``kv_len``, the new length is ``kv_len + k - 1``; the pages cover the next
round's windows, ``[L', L' + B + 2)`` (``window = B + 2``).

Direct block-diffusion decoding
-------------------------------
The appendix's diagnostic decoder ("Direct Block-Diffusion Decoding") fills
one block of B positions after the boundary by repeated denoising: every
forward runs over ``[x0, b_1..b_B]`` (1 causal row, B bidirectional block
rows) where ``b_p`` is the revealed token or ``[M]``; the prediction for
block position p is the top-1 of row p-1 (the shifted convention: position 1
is predicted by the boundary row, the final position of the preceding
block), its confidence the softmax probability of that top-1 token.  Every
still-masked position whose confidence exceeds tau_c (strictly) is
revealed; if none does, the single most confident masked position is
(readings: ties go to the lowest position; only masked positions are
candidates, revealed tokens never change).  When no position is masked, one
more forward over ``[x0, b_1..b_{B-1}]`` as causal rows writes the block's KV
without predicting anything, and the block ``b_1..b_B`` is committed: its
last token is the new boundary, ``kv_len`` grows by B, and the pages cover
the next denoising window ``[L', L' + B + 1)``.  A stop token truncates the
committed run at that token and ends the sequence (the output is cut at its
first EOS, and no later block is generated).  ``kv_commit`` takes the block
as the explicit run of each sequence (``block_runs``).

Multi-step drafting (experiments, "Draft Schedule": a draft-side
threshold tau_d sets how many denoising forwards build the draft) is the
two-forward round with its draft refined like a diffusion block: the B + 1
predictions of the draft window are revealed with ``reveal`` at tau_d, and
revealed a0, d_1..d_{B-1} are fed back as the inputs of mask rows 1..B (a
reading: d_B, predicted by the last row, has no input slot but is revealed
like the others).  tau_d = 0 is the one-shot draft.

Stochastic acceptance
---------------------
Under sampling, the draft is accepted by the standard acceptance-rejection
rule of speculative decoding, which keeps the committed tokens distributed
as the verifier's own samples (Preliminaries, "Speculative Decoding"; the
rule is that of Leviathan et al. 2023 and Chen et al. 2023).  For the
two-forward round at temperature T: p_j = softmax(z_j / T) of verify row
j-1 and q_j = softmax of draft row j; a0 is sampled from the boundary row
(the verifier's own distribution), d_j from q_j; d_j is accepted while
``u_j * q_j(d_j) < p_j(d_j)`` (probability min(1, p/q)); at the first
rejection the token is sampled from ``max(0, p_j - q_j)`` (normalised), and
after B acceptances from p_{B+1}.  Every random number is an input.
Sampling from weights w with a uniform u takes the smallest index whose
running sum (index order) exceeds ``u * sum(w)``.

Top-1 rule: the maximum logit wins; among equal maxima the lowest vocabulary
index wins; -0.0 and +0.0 are equal.  Non-finite logits are an error.

Pages (a reading: the paper does not describe a paged cache).  Every
sequence holds exactly ``ceil((L + R) / page_size)`` pages so that the next
window's slots exist.  After a commit, sequences that need fewer pages push
their surplus logical pages onto the free stack (sequences in order, each
from its highest logical page down); then sequences that need more pop pages
from the top of the stack (sequences in order, logical pages ascending).  If
the pops cannot be served, or a table would exceed ``max_pages``, nothing is
committed and the error word records why (1 = pool exhausted,
2 = max_pages exceeded).
"""
from __future__ import annotations

import numpy as np

ERR_POOL_EXHAUSTED = 1
ERR_MAX_PAGES = 2
ERR_NONFINITE = 4


def top1(row: np.ndarray) -> int:
    """Index of the largest value, lowest index among ties.

    numpy's argmax returns the first maximal index, and its comparisons treat
    -0.0 == +0.0.  Values must be finite.
    """
    if not np.all(np.isfinite(row)):
        raise ValueError("non-finite logit")
    return int(np.argmax(row))


def top1_rows(logits: np.ndarray) -> np.ndarray:
    """top1 over the last axis for every leading index; returns int32."""
    lead = logits.shape[:-1]
    flat = logits.reshape(-1, logits.shape[-1])
    out = np.empty(flat.shape[0], dtype=np.int32)
    for i in range(flat.shape[0]):
        out[i] = top1(flat[i])
    return out.reshape(lead)


def top1_confidence(row: np.ndarray) -> tuple:
    """(top-1 index, softmax probability of that token) of one logit row.

    The probability of the largest logit z_m is exp(z_m) / sum_i exp(z_i)
    = 1 / sum_i exp(z_i - z_m) (appendix "Direct Block-Diffusion Decoding":
    a prediction's confidence is its token probability).
    """
    t = top1(row)
    z = np.asarray(row, dtype=np.float64)
    return t, float(1.0 / np.sum(np.exp(z - z[t])))


def reveal(block: np.ndarray, am: np.ndarray, conf: np.ndarray, tau_c: float,
           finished: np.ndarray) -> np.ndarray:
    """One denoising step's reveal (appendix "Direct Block-Diffusion Decoding").

    block [S, B] int: revealed token of position p (column p-1), or -1 while
    masked.  am, conf [S, B]: top-1 and its confidence of window row p-1,
    i.e. the prediction for position p.  Every masked position with
    conf > tau_c is revealed; if there is none, the masked position of
    largest confidence (lowest position among ties).  Finished sequences and
    complete blocks are left alone.  Returns the new block.
    """
    out = block.copy()
    S, B = block.shape
    for s in range(S):
        if finished[s]:
            continue
        masked = [p for p in range(B) if block[s, p] < 0]
        if not masked:
            continue
        chosen = [p for p in masked if conf[s, p] > tau_c]
        if not chosen:
            best = masked[0]
            for p in masked[1:]:
                if conf[s, p] > conf[s, best]:
                    best = p
            chosen = [best]
        for p in chosen:
            out[s, p] = am[s, p]
    return out


def softmax_t(z: np.ndarray, T: float) -> np.ndarray:
    """softmax(z / T) of one row, float64."""
    z = np.asarray(z, dtype=np.float64)
    w = np.exp((z - z.max()) / T)
    return w / w.sum()


def sample_index(w: np.ndarray, u: float) -> int:
    """Inverse-CDF sample: the smallest i with w_0 + ... + w_i > u * sum(w)
    (w >= 0, not all zero; 0 <= u < 1)."""
    c = np.cumsum(np.asarray(w, dtype=np.float64))
    i = int(np.searchsorted(c, u * c[-1], side="right"))
    return min(i, len(c) - 1)


def stochastic_accept(p: np.ndarray, q: np.ndarray, d: np.ndarray, u_acc: np.ndarray) -> int:
    """A = number of leading drafts accepted: d_j (j = 1..B) is accepted
    while u_acc[j-1] * q[j-1, d_j] < p[j-1, d_j].  p, q: [B, V]."""
    A = 0
    for j in range(len(d)):
        if not (u_acc[j] * q[j, d[j]] < p[j, d[j]]):
            break
        A = j + 1
    return A


def resample_weights(p: np.ndarray, q: np.ndarray | None) -> np.ndarray:
    """max(0, p - q) after a rejection, p itself after full acceptance."""
    return p.copy() if q is None else np.maximum(p - q, 0.0)


def accept_length(a: np.ndarray, d: np.ndarray) -> int:
    """Longest k such that d_j == a_j for every j <= k (1-based j).

    ``a[j-1]`` is a_j and ``d[j-1]`` is d_j; only positions present in d count.
    """
    k = 0
    for j in range(1, d.shape[0] + 1):
        if d[j - 1] != a[j - 1]:
            break
        k = j
    return k


def accept(argmax: np.ndarray, draft: np.ndarray, n_causal: int) -> np.ndarray:
    """A_s for every sequence.  argmax [S, R] (row r's top-1), draft [S, n_causal-1]."""
    S = argmax.shape[0]
    A = np.zeros(S, dtype=np.int32)
    for s in range(S):
        a = argmax[s, :n_causal]               # a_1..a_{n_causal}
        A[s] = accept_length(a, draft[s, :n_causal - 1])
    return A


def committed_run(argmax_row: np.ndarray, draft_row: np.ndarray, A: int, lead=None) -> list:
    """The tokens a step commits before any stop rule: d_1..d_A then a_{A+1},
    after the lead token a0 in the two-forward round."""
    run = [int(draft_row[j - 1]) for j in range(1, A + 1)] + [int(argmax_row[A])]
    return run if lead is None else [int(lead)] + run


def kv_commit(st, accept_len: np.ndarray, argmax: np.ndarray, n_causal: int, n_mask: int,
              eos_id: int = -1, max_new: int | None = None, page_size: int = 16,
              lead: np.ndarray | None = None, window: int | None = None,
              block_runs: np.ndarray | None = None, draft_group: int = 0) -> int:
    """Apply one step's commit to ``st`` (a synth.PagedState-like object) in place.

    ``lead`` (two-forward round): per-sequence a0, committed first; the
    boundary's KV is then already in ``kv_len``.  ``window``: rows of the next
    window the pages must cover (default n_causal + n_mask).  ``block_runs``
    [S, n] (direct block diffusion): the whole row is each sequence's run,
    in place of the accepted drafts and the verifier's token (accept_len and
    argmax are then unused).  ``draft_group`` > 0 (per-acceptance drafts): the
    mask rows are n_causal groups of that many rows, and the next draft comes
    from group A (the continuation that kept exactly the accepted drafts).
    Returns the error word (0 on success; on error ``st`` is unchanged).
    """
    S = st.kv_len.shape[0]
    R = n_causal + n_mask if window is None else window
    W = st.draft.shape[1]
    if n_mask > 0 and n_mask < W:
        raise ValueError("mask rows must cover the draft width")
    if max_new is None:
        max_new = st.out_tokens.shape[1]
    max_new = min(max_new, st.out_tokens.shape[1])

    new_len = st.kv_len.copy()
    new_bound = st.boundary.copy()
    new_draft = st.draft.copy()
    new_fin = st.finished.copy()
    runs = [[] for _ in range(S)]
    for s in range(S):
        if st.finished[s]:
            continue
        if block_runs is not None:
            run = [int(t) for t in block_runs[s]]
        else:
            run = committed_run(argmax[s], st.draft[s], int(accept_len[s]),
                                None if lead is None else lead[s])
        kept = []
        stop = False
        for tok in run:
            if st.out_count[s] + len(kept) >= max_new:
                stop = True
                break
            kept.append(tok)
            if eos_id >= 0 and tok == eos_id:
                stop = True
                break
        if st.out_count[s] + len(kept) >= max_new:
            stop = True
        runs[s] = kept
        new_len[s] = st.kv_len[s] + len(kept) - (0 if lead is None else 1)
        if kept:
            new_bound[s] = kept[-1]
        if n_mask > 0:
            W = st.draft.shape[1]
            first = n_causal + (int(accept_len[s]) * draft_group if draft_group else 0)
            new_draft[s] = argmax[s, first:first + W]
        new_fin[s] = 1 if stop else 0

    need = np.array([(int(new_len[s]) + R + page_size - 1) // page_size for s in range(S)],
                    dtype=np.int64)
    err = 0
    if np.any(need > st.max_pages):
        err |= ERR_MAX_PAGES
    pushes = int(sum(max(int(st.num_pages[s]) - int(need[s]), 0) for s in range(S)))
    pops = int(sum(max(int(need[s]) - int(st.num_pages[s]), 0) for s in range(S)))
    if pops > st.free_top + pushes:
        err |= ERR_POOL_EXHAUSTED
    if err:
        return err

    # pushes: sequences in order, surplus logical pages from the highest down
    top = st.free_top
    for s in range(S):
        for i in range(int(st.num_pages[s]) - 1, int(need[s]) - 1, -1):
            st.free_stack[top] = st.page_table[s, i]
            st.page_table[s, i] = -1
            top += 1
    # pops: sequences in order, missing logical pages ascending
    for s in range(S):
        for i in range(int(st.num_pages[s]), int(need[s])):
            top -= 1
            st.page_table[s, i] = st.free_stack[top]
            st.free_stack[top] = -1
    st.free_top = top
    st.num_pages[:] = need

    for s in range(S):
        for tok in runs[s]:
            st.out_tokens[s, st.out_count[s]] = tok
            st.out_count[s] += 1
    st.kv_len[:] = new_len
    st.boundary[:] = new_bound
    st.draft[:] = new_draft
    st.finished[:] = new_fin
    return 0
