// kv_commit: commit the accepted run and roll back the rest of the window's
// KV (appendix "Self-Speculative Decoding and KV-Cache Update", items Accept,
// Cache update, Next round).
//
// One workgroup, one thread per sequence.  The committed run of sequence s
// is d_1..d_A followed by the verifier's a_{A+1} = argmax[s, A].  A stop token
// or the output budget truncates it; the KV of x0 and the kept drafts stays
// (kv_len += k), every other window slot is dropped.
//
// The paper's two-forward round commits through the same kernel with a lead
// token: the run is a0, d_1..d_A, a_{A+1}, kv_len already counts the kept x0
// (so kv_len += k - 1), and the pages cover the next round's windows.
//
// Direct block diffusion commits a whole block b_1..b_B through the same
// kernel (no accept length): the run is the block, kv_len += k (the
// cache-write forward wrote x0 and b_1..b_{B-1}), and the pages cover the
// next denoising window of B + 1 rows.  A masked (negative) token in a live
// block is an error.
//
// Pages: each sequence ends holding ceil((kv_len + W) / 16) pages, W the
// window of the next call (R, or B + 2 in the two-forward round).  Two
// exclusive scans over the sequences give every surplus page its slot on the
// free stack (pushes, sequences in order, highest logical page first) and
// every missing page its slot below the new top (pops, sequences in order,
// logical pages ascending), so the result is independent of thread timing.
// Feasibility is decided before anything is written: on failure the whole
// state is left untouched and the error bit is set.
//
// accept_commit runs the acceptance in the same kernel: each thread first
// finds its sequence's longest accepted prefix A (draft against the
// verifier's top-1), then commits as above -- one launch for accept, commit
// and rollback.
#include "dvs_common.h"

namespace dvs {

constexpr int COMMIT_THREADS = 1024;
constexpr int RUN_CHUNK = 8;

__device__ __forceinline__ int block_exclusive_scan(int v, int* sh, int& total) {
  // Hillis-Steele over the block in shared memory (S <= 1024; runs once).
  const int tid = threadIdx.x;
  sh[tid] = v;
  __syncthreads();
  for (int off = 1; off < (int)blockDim.x; off <<= 1) {
    const int add = tid >= off ? sh[tid - off] : 0;
    __syncthreads();
    sh[tid] += add;
    __syncthreads();
  }
  const int incl = sh[tid];
  total = sh[blockDim.x - 1];
  __syncthreads();
  return incl - v;
}

struct CommitParams {
  int S, n_causal, n_mask, R, window, max_pages, pool_pages, draft_width, max_new, eos_id;
  const int32_t* lead;   // two-forward round: a0 per sequence, committed first (else NULL)
  const int32_t* accept_len;   // NULL: the run is the first n_causal tokens of argmax
  int accept_here;             // 1: A computed in this kernel from argmax and draft
  int32_t* accept_out;         // accept_here: A per sequence (may be NULL)
  int draft_group;             // > 0: next draft from mask group A (groups of this many rows)
  const int32_t* argmax;
  int32_t* kv_len;
  int32_t* page_table;
  int32_t* num_pages;
  int32_t* free_stack;
  int32_t* free_top;
  int32_t* boundary;
  int32_t* draft;
  int32_t* out_tokens;
  int32_t* out_count;
  int32_t* finished;
  int32_t* err;
};

// j-th token of the committed run: [a0,] d_1..d_A, a_{A+1}.
__device__ __forceinline__ int run_token(const CommitParams& p, int s, int A, int j) {
  if (p.lead) {
    if (j == 0) return p.lead[s];
    --j;
  }
  return j < A ? p.draft[(size_t)s * p.draft_width + j] : p.argmax[(size_t)s * p.R + A];
}

// FAST: acceptance here, no lead token, no draft groups, at most
// COMMIT_FAST_W causal rows and draft slots.  A sequence's whole draft row,
// its verify rows' top-1 and the next draft's rows are loaded at once, with
// its state and the free-stack top, so the acceptance, the run and the next
// draft come from registers (one memory round trip instead of one per chunk
// and per dependent step); the results are the general path's.
constexpr int COMMIT_FAST_W = 32;

template <bool FAST>
__global__ void __launch_bounds__(COMMIT_THREADS) kv_commit_kernel(CommitParams p) {
  __shared__ int sh[COMMIT_THREADS];
  __shared__ int s_err;
  const int s = threadIdx.x;
  const bool live_seq = s < p.S;
  if (s == 0) s_err = 0;
  __syncthreads();

  int L = 0, n = 0, k = 0, need = 0, cnt = 0, A = 0;
  bool fin = false, stop = false;
  int last_tok = 0;
  constexpr int FW = FAST ? COMMIT_FAST_W : 1;
  int dv[FW], av[FW], nx[FW];   // FAST: draft row, verify top-1, next draft
  int top0 = 0;
  if (FAST) top0 = *p.free_top;
  if (FAST && live_seq) {
    const int nd = p.n_causal - 1;
    const int32_t* drow = p.draft + (size_t)s * p.draft_width;
    const int32_t* arow = p.argmax + (size_t)s * p.R;
    L = p.kv_len[s];
    n = p.num_pages[s];
    cnt = p.out_count[s];
    fin = p.finished[s] != 0;
#pragma unroll
    for (int j = 0; j < FW; ++j) {
      dv[j] = j < nd ? drow[j] : 0;
      av[j] = j < p.n_causal ? arow[j] : 0;
      nx[j] = (p.n_mask > 0 && j < p.draft_width) ? arow[p.n_causal + j] : 0;
    }
    if (!fin) {
      bool go = true;
#pragma unroll
      for (int j = 0; j < FW; ++j) {
        if (j < nd && go && dv[j] == av[j]) A = j + 1;
        else go = false;
      }
    }
    if (p.accept_out) p.accept_out[s] = fin ? 0 : A;
    if (!fin) {
      // run = d_1..d_A, a_{A+1}; keep up to the first stop token / budget
      bool done = false;
#pragma unroll
      for (int j = 0; j < FW; ++j) {
        if (done || j > A) continue;
        const int tk = j < A ? dv[j] : av[j];
        if (cnt + k >= p.max_new) {
          stop = done = true;
        } else {
          if (tk < 0) atomicOr(&s_err, DVS_ERR_OPEN_BLOCK);
          ++k;
          last_tok = tk;
          if (p.eos_id >= 0 && tk == p.eos_id) stop = done = true;
        }
      }
      if (cnt + k >= p.max_new) stop = true;
    }
    need = (L + k + p.window + DVS_PAGE_SIZE - 1) / DVS_PAGE_SIZE;
    if (need > p.max_pages || n < 0 || n > p.max_pages || L < 0)
      atomicOr(&s_err, DVS_ERR_MAX_PAGES);
  } else if (!FAST && live_seq) {
    L = p.kv_len[s];
    n = p.num_pages[s];
    cnt = p.out_count[s];
    fin = p.finished[s] != 0;
    if (!fin && p.accept_here) {
      // longest prefix with d_j == a_j = argmax[s, j-1], j <= n_causal - 1,
      // compared RUN_CHUNK positions at a time (independent loads first)
      const int nd = p.n_causal - 1;
      bool go = true;
      for (int j0 = 0; j0 < nd && go; j0 += RUN_CHUNK) {
        int dv[RUN_CHUNK], av[RUN_CHUNK];
#pragma unroll
        for (int u = 0; u < RUN_CHUNK; ++u) {
          const int j = min(j0 + u, nd - 1);
          dv[u] = p.draft[(size_t)s * p.draft_width + j];
          av[u] = p.argmax[(size_t)s * p.R + j];
        }
#pragma unroll
        for (int u = 0; u < RUN_CHUNK; ++u) {
          if (!go || j0 + u >= nd) continue;
          if (dv[u] == av[u]) A = j0 + u + 1;
          else go = false;
        }
      }
    }
    if (live_seq && p.accept_here && p.accept_out) p.accept_out[s] = fin ? 0 : A;
    if (!fin) {
      if (!p.accept_here) A = p.accept_len ? p.accept_len[s] : p.n_causal - 1;
      A = A < 0 ? 0 : (A > p.n_causal - 1 ? p.n_causal - 1 : A);
      // run = [a0,] d_1..d_A, a_{A+1} (last index jl); keep up to the first
      // stop token / budget.  Tokens are fetched RUN_CHUNK at a time
      // (independent loads, one memory round trip per chunk), then scanned in
      // order.
      const int jl = A + (p.lead ? 1 : 0);
      bool done = false;
      for (int j0 = 0; j0 <= jl && !done; j0 += RUN_CHUNK) {
        int tk[RUN_CHUNK];
#pragma unroll
        for (int u = 0; u < RUN_CHUNK; ++u) tk[u] = run_token(p, s, A, min(j0 + u, jl));
#pragma unroll
        for (int u = 0; u < RUN_CHUNK; ++u) {
          if (done || j0 + u > jl) continue;
          if (cnt + k >= p.max_new) {
            stop = done = true;
          } else {
            if (!p.accept_len && tk[u] < 0) atomicOr(&s_err, DVS_ERR_OPEN_BLOCK);
            ++k;
            last_tok = tk[u];
            if (p.eos_id >= 0 && tk[u] == p.eos_id) stop = done = true;
          }
        }
      }
      if (cnt + k >= p.max_new) stop = true;
    }
    // new length: + k, or + k - 1 when kv_len already counts the kept x0
    need = (L + k - (p.lead && !fin ? 1 : 0) + p.window + DVS_PAGE_SIZE - 1) / DVS_PAGE_SIZE;
    if (need > p.max_pages || n < 0 || n > p.max_pages || L < 0)
      atomicOr(&s_err, DVS_ERR_MAX_PAGES);
  }
  const int push = live_seq && n > need ? n - need : 0;
  const int pop = live_seq && need > n ? need - n : 0;
  int tot_push = 0, tot_pop = 0;
  const int push_off = block_exclusive_scan(push, sh, tot_push);
  const int pop_off = block_exclusive_scan(pop, sh, tot_pop);
  if (!FAST) top0 = *p.free_top;
  if (s == 0) {
    if (tot_pop > top0 + tot_push) atomicOr(&s_err, DVS_ERR_POOL_EXHAUSTED);
    if (top0 + tot_push > p.pool_pages || top0 < 0) atomicOr(&s_err, DVS_ERR_POOL_EXHAUSTED);
  }
  __syncthreads();
  if (s_err) {
    if (s == 0) set_err(p.err, s_err);
    return;
  }

  int32_t* row = p.page_table + (size_t)s * p.max_pages;
  for (int i = 0; i < push; ++i) {            // logical n-1, n-2, ... need
    p.free_stack[top0 + push_off + i] = row[n - 1 - i];
    row[n - 1 - i] = -1;
  }
  __threadfence_block();
  __syncthreads();
  const int top1 = top0 + tot_push;
  for (int j = 0; j < pop; ++j) {             // logical n, n+1, ... need-1
    const int slot = top1 - 1 - (pop_off + j);
    row[n + j] = p.free_stack[slot];
    p.free_stack[slot] = -1;
  }
  if (s == 0) *p.free_top = top1 - tot_pop;

  if (FAST && live_seq) {
    p.num_pages[s] = need;
    if (!fin) {
      int32_t* ot = p.out_tokens + (size_t)s * p.max_new + cnt;
#pragma unroll
      for (int j = 0; j < FW; ++j)
        if (j < k) ot[j] = j < A ? dv[j] : av[j];
      p.out_count[s] = cnt + k;
      p.kv_len[s] = L + k;
      if (k > 0) p.boundary[s] = last_tok;
      if (p.n_mask > 0) {
        int32_t* drow = p.draft + (size_t)s * p.draft_width;
#pragma unroll
        for (int j = 0; j < FW; ++j)
          if (j < p.draft_width) drow[j] = nx[j];
      }
      p.finished[s] = stop ? 1 : 0;
    }
  } else if (!FAST && live_seq) {
    p.num_pages[s] = need;
    if (!fin) {
      int32_t* ot = p.out_tokens + (size_t)s * p.max_new;
      for (int j0 = 0; j0 < k; j0 += RUN_CHUNK) {   // loads of a chunk first, then its stores
        int tk[RUN_CHUNK];
#pragma unroll
        for (int u = 0; u < RUN_CHUNK; ++u) tk[u] = run_token(p, s, A, min(j0 + u, k - 1));
#pragma unroll
        for (int u = 0; u < RUN_CHUNK; ++u)
          if (j0 + u < k) ot[cnt + j0 + u] = tk[u];
      }
      p.out_count[s] = cnt + k;
      p.kv_len[s] = L + k - (p.lead ? 1 : 0);
      if (k > 0) p.boundary[s] = last_tok;
      if (p.n_mask > 0) {
        for (int j0 = 0; j0 < p.draft_width; j0 += RUN_CHUNK) {
          int tk[RUN_CHUNK];
#pragma unroll
          for (int u = 0; u < RUN_CHUNK; ++u)
            tk[u] = p.argmax[(size_t)s * p.R + p.n_causal + A * p.draft_group +
                             min(j0 + u, p.draft_width - 1)];
#pragma unroll
          for (int u = 0; u < RUN_CHUNK; ++u)
            if (j0 + u < p.draft_width) p.draft[(size_t)s * p.draft_width + j0 + u] = tk[u];
        }
      }
      p.finished[s] = stop ? 1 : 0;
    }
  }
}

}  // namespace dvs

using namespace dvs;

static int launch_commit(const char* who, int32_t S, int32_t n_causal, int32_t n_mask,
                         int32_t window, const int32_t* lead, const int32_t* accept_len,
                         int accept_here, int32_t* accept_out, int32_t draft_group,
                         const int32_t* argmax, int32_t* kv_len, int32_t* page_table,
                         int32_t* num_pages, int32_t max_pages, int32_t* free_stack,
                         int32_t* free_top, int32_t num_pool_pages, int32_t* boundary,
                         int32_t* draft, int32_t draft_width, int32_t* out_tokens,
                         int32_t* out_count, int32_t max_new, int32_t eos_id, int32_t* finished,
                         int32_t* err_word, void* stream) {
  DVS_CHECK_ARG(argmax && kv_len && page_table && num_pages && free_stack &&
                    free_top && boundary && out_tokens && out_count && finished,
                "%s: NULL array argument", who);
  DVS_CHECK_ARG(S >= 1 && S <= COMMIT_THREADS, "%s: need 1 <= S <= %d", who, COMMIT_THREADS);
  DVS_CHECK_ARG(n_causal >= 1 && n_mask >= 0, "%s: need n_causal >= 1, n_mask >= 0", who);
  DVS_CHECK_ARG(draft_width >= 0 && (draft || draft_width == 0), "%s: bad draft", who);
  DVS_CHECK_ARG(draft_width >= n_causal - 1, "%s: draft_width < n_causal - 1", who);
  DVS_CHECK_ARG(n_mask == 0 || n_mask >= draft_width,
                "%s: mask rows (%d) must cover the draft width (%d)", who, n_mask, draft_width);
  DVS_CHECK_ARG(max_pages >= 1 && num_pool_pages >= 1 && max_new >= 1,
                "%s: need max_pages, num_pool_pages, max_new >= 1", who);
  DVS_CHECK_ARG(window >= n_causal + n_mask, "%s: window (%d) < n_causal + n_mask", who, window);
  CommitParams p{};
  p.S = S; p.n_causal = n_causal; p.n_mask = n_mask; p.R = n_causal + n_mask; p.window = window;
  p.lead = lead;
  p.max_pages = max_pages; p.pool_pages = num_pool_pages; p.draft_width = draft_width;
  p.max_new = max_new; p.eos_id = eos_id;
  DVS_CHECK_ARG(draft_group >= 0 && (draft_group == 0 ||
                                     (n_mask == n_causal * draft_group && draft_group >= draft_width)),
                "%s: mask rows must be n_causal groups of draft_group >= draft_width rows", who);
  p.accept_len = accept_len; p.accept_here = accept_here; p.accept_out = accept_out;
  p.draft_group = draft_group;
  p.argmax = argmax; p.kv_len = kv_len; p.page_table = page_table;
  p.num_pages = num_pages; p.free_stack = free_stack; p.free_top = free_top;
  p.boundary = boundary; p.draft = draft; p.out_tokens = out_tokens; p.out_count = out_count;
  p.finished = finished; p.err = err_word;
  // one thread per sequence, in whole waves: the block scans and barriers
  // cost as many steps as the block has threads' log2
  const int threads = ((S + 63) / 64) * 64;
  const bool fast = accept_here && !lead && draft_group == 0 && n_causal <= COMMIT_FAST_W &&
                    draft_width <= COMMIT_FAST_W;
  if (fast)
    hipLaunchKernelGGL(kv_commit_kernel<true>, dim3(1), dim3(threads), 0, (hipStream_t)stream, p);
  else
    hipLaunchKernelGGL(kv_commit_kernel<false>, dim3(1), dim3(threads), 0, (hipStream_t)stream, p);
  return launch_status(who);
}

extern "C" int kv_commit(int32_t S, int32_t n_causal, int32_t n_mask, const int32_t* accept_len,
                         const int32_t* argmax, int32_t* kv_len, int32_t* page_table,
                         int32_t* num_pages, int32_t max_pages, int32_t* free_stack,
                         int32_t* free_top, int32_t num_pool_pages, int32_t* boundary,
                         int32_t* draft, int32_t draft_width, int32_t* out_tokens,
                         int32_t* out_count, int32_t max_new, int32_t eos_id, int32_t* finished,
                         int32_t* err_word, void* stream) {
  clear_error();
  DVS_CHECK_ARG(accept_len != nullptr, "kv_commit: NULL accept_len");
  return launch_commit("kv_commit", S, n_causal, n_mask, n_causal + n_mask, nullptr, accept_len,
                       0, nullptr, 0, argmax, kv_len, page_table, num_pages, max_pages, free_stack, free_top,
                       num_pool_pages, boundary, draft, draft_width, out_tokens, out_count, max_new,
                       eos_id, finished, err_word, stream);
}

extern "C" int kv_commit_round(int32_t S, int32_t B, const int32_t* lead, const int32_t* accept_len,
                               const int32_t* argmax, int32_t* kv_len, int32_t* page_table,
                               int32_t* num_pages, int32_t max_pages, int32_t* free_stack,
                               int32_t* free_top, int32_t num_pool_pages, int32_t* boundary,
                               int32_t* draft, int32_t draft_width, int32_t* out_tokens,
                               int32_t* out_count, int32_t max_new, int32_t eos_id,
                               int32_t* finished, int32_t* err_word, void* stream) {
  clear_error();
  DVS_CHECK_ARG(lead != nullptr && accept_len != nullptr, "kv_commit_round: NULL lead/accept_len");
  DVS_CHECK_ARG(B >= 1, "kv_commit_round: need B >= 1");
  return launch_commit("kv_commit_round", S, B + 1, 0, B + 2, lead, accept_len, 0, nullptr, 0,
                       argmax, kv_len,
                       page_table, num_pages, max_pages, free_stack, free_top, num_pool_pages,
                       boundary, draft, draft_width, out_tokens, out_count, max_new, eos_id,
                       finished, err_word, stream);
}

extern "C" int kv_commit_block(int32_t S, int32_t B, const int32_t* block, int32_t* kv_len,
                               int32_t* page_table, int32_t* num_pages, int32_t max_pages,
                               int32_t* free_stack, int32_t* free_top, int32_t num_pool_pages,
                               int32_t* boundary, int32_t* out_tokens, int32_t* out_count,
                               int32_t max_new, int32_t eos_id, int32_t* finished,
                               int32_t* err_word, void* stream) {
  clear_error();
  DVS_CHECK_ARG(block != nullptr, "kv_commit_block: NULL block");
  DVS_CHECK_ARG(B >= 1, "kv_commit_block: need B >= 1");
  // run token j < B - 1 comes from the draft slot j, the last from argmax[B - 1]:
  // both are the block row
  return launch_commit("kv_commit_block", S, B, 0, B + 1, nullptr, nullptr, 0, nullptr, 0,
                       block, kv_len,
                       page_table, num_pages, max_pages, free_stack, free_top, num_pool_pages,
                       boundary, const_cast<int32_t*>(block), B, out_tokens, out_count, max_new,
                       eos_id, finished, err_word, stream);
}

extern "C" int accept_commit(int32_t S, int32_t n_causal, int32_t n_mask, int32_t draft_group,
                             const int32_t* argmax, int32_t* accept_out, int32_t* kv_len, int32_t* page_table,
                             int32_t* num_pages, int32_t max_pages, int32_t* free_stack,
                             int32_t* free_top, int32_t num_pool_pages, int32_t* boundary,
                             int32_t* draft, int32_t draft_width, int32_t* out_tokens,
                             int32_t* out_count, int32_t max_new, int32_t eos_id, int32_t* finished,
                             int32_t* err_word, void* stream) {
  clear_error();
  DVS_CHECK_ARG(draft || n_causal == 1, "accept_commit: NULL draft");
  return launch_commit("accept_commit", S, n_causal, n_mask, n_causal + n_mask, nullptr, nullptr,
                       1, accept_out, draft_group, argmax, kv_len, page_table, num_pages, max_pages,
                       free_stack, free_top, num_pool_pages, boundary, draft, draft_width,
                       out_tokens, out_count, max_new, eos_id, finished, err_word, stream);
}
