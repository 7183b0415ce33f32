// attn_hybrid_block: append the window's K/V to the paged cache and attend
// with the block-causal (hybrid) mask.
//
// Visibility rule (Preliminaries "Block Diffusion"; Method "Joint
// AR-Diffusion Training"; appendix items Draft forward / Verify forward):
// window row r of a sequence with committed length L sits at position L + r;
// a causal row (r < n_causal) sees keys <= L + r, a mask row sees every key
// up to L + R - 1.  Keys below L are visible to every row, so only the tiles
// that reach the window need a mask.
//
// bf16 path (MFMA, gfx950)
//   Work items are (sequence, KV head, row tile); an item's keys are cut into
//   64-key tiles.  All G query heads of the KV head and all R window rows (up
//   to 256 "query rows", 32 per wave) share every K/V tile staged in LDS, so
//   the cache is read from HBM once per KV head.  Per tile and wave:
//     S^T[key, row] = K Q^T   v_mfma_f32_32x32x16_bf16, A = K from LDS,
//                             B = Q held in registers for the whole segment;
//     the C layout puts one query row per lane, so the online-softmax row max
//     and sum are in-lane plus one exchange with lane^32, and the O rescale
//     touches only the lane's own row;
//     O^T[d, row] += V^T P^T  A = V^T slice of the head-dim-major V tile,
//                             B = P packed to bf16 straight from the scores.
//   A workgroup first appends the window keys of its own tiles ([L, T) from
//   k_new / v_new) to their pool slots; then every tile, cache or window, is
//   copied HBM -> LDS with direct 16-byte loads through a 3-stage ring.  The
//   tiles that reach L are masked; in the tile that runs past T the keys >= T
//   read the sequence's last page again and their V values are zeroed before
//   the products (their weights are zero, and a non-finite stale value would
//   otherwise make them NaN).
//
//   Two ways to cut the work (both deterministic):
//   * aligned (chunk_keys > 0): workgroup = one chunk of one item, chunks at
//     absolute multiples of chunk_keys, so a row's arithmetic never depends
//     on the other rows or on the batch (a causal row equals a plain AR call
//     at its position, bit for bit);
//   * balanced (chunk_keys == 0): the items' tiles are concatenated and every
//     workgroup takes an equal contiguous share, so the grid finishes together
//     whatever the length mix; only shares that split an item publish
//     partials.
//   A split item's partials ((m, l) in fp32; O/l in bf16) are merged in
//   segment order by the last workgroup to count in; the count-in is an
//   agent-scope release atomic add on the item's counter, and the workgroup
//   that counts in last takes an agent-scope acquire fence: the count-ins
//   form one release sequence, so every workgroup's partial stores are
//   ordered before the merging workgroup's loads.
//
// fp32 path: a plain per-(sequence, row, head) workgroup, fp32 throughout.
#include <math.h>

#include <mutex>

#include "dvs_common.h"

namespace dvs {

constexpr int KT = 64;                 // keys per tile
constexpr int NSTAGE = 4;              // LDS ring depth for cache tiles
constexpr int SUB_TILES = 256;         // tiles whose page ids are staged at once
constexpr int MAX_CHUNK_KEYS = 16384;
constexpr int BAL_MAX_SEGS = 16;       // balanced mode: segments per item (bound)
constexpr int BAL_MAX_SEQS = 1024;     // balanced mode: sequences per call
constexpr float RESCALE_LOG2 = 8.f;

// Partial slot of segment k of a split item whose segment 0 is held by
// workgroup wg0.  Aligned chunks: one slot per (item, chunk).  Balanced
// shares: an item's segments sit in consecutive workgroups, and a workgroup
// holds at most two segments of split items -- the continuation of an item
// begun earlier (its first segment, k > 0) and the start of an item that runs
// on past its share (its last segment, k == 0) -- so two slots per
// workgroup suffice, whatever the length mix.
__device__ __forceinline__ size_t part_slot(int balanced, int it, int max_segs, int wg0, int k) {
  return balanced ? (size_t)(wg0 + k) * 2 + (k == 0 ? 1 : 0) : (size_t)it * max_segs + k;
}

struct AttnParams {
  const void* q;
  const void* k_new;
  const void* v_new;
  void* k_pool;
  void* v_pool;
  const int32_t* page_table;
  const int32_t* kv_len;
  void* out;
  float* part_o;
  float* part_ml;
  int32_t* counters;
  int32_t* err;
  int S, n_causal, n_mask, R, Hq, Hkv, G, max_pages, pool_pages;
  int rows_total, n_row_tiles, n_items;
  int balanced;      // 0: aligned chunks, 1: balanced shares
  int chunk_tiles;   // aligned: tiles per chunk
  int n_chunks_max;  // aligned: grid rows
  int share_min;     // balanced: minimum tiles per workgroup
  int max_segs;      // partial slots per item
  int group;         // mask rows per group (0: one block of n_mask rows)
  int n_groups;      // n_mask / group
  float scale_log2;
  float scale;
};

// Second visible interval of window row r (beside keys <= hi): the slots of
// its own mask group when the mask rows come in groups.  Row i of mask group
// g sees the cache, the causal rows 0 .. n_causal - n_groups + g (so hi =
// L + n_causal - n_groups + g) and the slots [lo2, hi2] of its group.  Empty
// (lo2 > hi2) for causal rows and for one group, where hi covers the whole
// window.
struct Vis2 {
  int lo2, hi2;
};
__device__ __forceinline__ Vis2 group_interval(const AttnParams& p, int L, int r) {
  if (p.group == 0 || r < p.n_causal) return Vis2{1 << 30, -1};
  const int g = (r - p.n_causal) / p.group;
  const int lo = L + p.n_causal + g * p.group;
  return Vis2{lo, lo + p.group - 1};
}
__device__ __forceinline__ int row_hi(const AttnParams& p, int L, int r) {
  if (r < p.n_causal) return L + r;
  if (p.group == 0) return L + p.R - 1;
  return L + p.n_causal - p.n_groups + (r - p.n_causal) / p.group;
}

// ---------------------------------------------------------------------------
// LDS layouts of one 64-key tile (bf16)
//
// K: 64 rows of D*2 bytes (row = key); the 16-byte chunks of row r are
//    XOR-swizzled by kswz(r) so the A-operand reads (8 rows per LDS phase)
//    hit distinct banks.
// V: 4 pages x D rows x 32 bytes (row = head-dim element, 16 keys) - the
//    layout of a head-dim-major V page of the pool, so cache tiles are plain
//    copies; the two 16-byte halves swap on every other group of 4 rows.
// Both tiles are built from 1 KB wave segments, and a page of one KV head is
// a whole number of segments (4 KB / 3 KB / 2 KB for D = 128 / 96 / 64), so
// every direct-load instruction reads a single, wave-uniform page.
//
// Key permutation: QK^T A-operand lane m (0..31 within a 32-key group) is fed
// key kperm(m) (bits 2 and 3 of m swapped).  With the 32x32 MFMA C layout,
// lane (row, hh) then holds in score registers 0..7 the keys 8*hh + 0..7 and
// in registers 8..15 the keys 16 + 8*hh + 0..7: exactly the B-operand layout
// of two 16-key PV k-steps, whose A operand is one 16-byte half of a V page
// row.
// ---------------------------------------------------------------------------
__device__ __forceinline__ int kperm(int m) {
  return (m & 0x13) | ((m & 4) << 1) | ((m & 8) >> 1);
}

// Chunk swizzles.  K (16 chunks per row): a bijection of the row's low 4 bits
// (bits 2 and 3 swapped) so that the 8 rows kperm(0..7) and the 16 rows
// kperm(0..15) read by consecutive lanes land on distinct 16-byte bank groups
// whether the LDS serves 8 or 16 lanes per cycle.  V: halves swap with bit 2
// xor bit 3 of the row, distinct over 8 and over 16 consecutive rows.
template <int CPR>
__device__ __forceinline__ int kswz(int row) {
  if constexpr (CPR % 16 == 0) return (row & 3) | ((row >> 1) & 4) | ((row & 4) << 1);
  else if constexpr (CPR % 8 == 0) return (row & 3) | ((row >> 1) & 4);
  else return row & 3;
}

__device__ __forceinline__ int vswz(int d) { return ((d >> 2) ^ (d >> 3)) & 1; }

// s_waitcnt vmcnt(n), other counters untouched (gfx9 encoding; n <= 63).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// Wait until at most `tiles_after` cache tiles (NPL loads per lane each) are
// still in flight (tiles_after in [0, NSTAGE - 2]).  A bound above 63 is
// clamped, which only waits longer.
template <int N>
__device__ __forceinline__ void wait_vmcnt_clamped() {
  wait_vmcnt<(N < 63 ? N : 63)>();
}

template <int NPL>
__device__ __forceinline__ void wait_tiles(int tiles_after) {
  static_assert(NSTAGE >= 2 && NSTAGE <= 4, "wait_tiles covers up to 2 tiles in flight");
  if (NSTAGE >= 4 && tiles_after >= 2) wait_vmcnt_clamped<2 * NPL>();
  else if (NSTAGE >= 3 && tiles_after >= 1) wait_vmcnt_clamped<NPL>();
  else wait_vmcnt<0>();
}

// ---------------------------------------------------------------------------
// Append the window keys [a, b) (L <= a < b <= T) of item (sequence s, KV
// head kvh) to their pool slots: K rows from k_new, and in the head-dim-major
// V pages one 32-byte row (the 16 slots of a page) per (page, head-dim
// element), merged with the slots outside [a, b), which keep their values.
// A workgroup appends exactly the keys of its own tiles before it streams
// them, so the window tiles then go through the same direct loads as cache
// tiles.  Tiles start at multiples of 64 keys, so every page belongs to one
// tile, and workgroups of different row tiles of one item write identical
// bytes.  Every load of a thread is issued before its stores (a pool store
// could alias a pool load as far as the compiler can tell).  Slots whose page
// id is invalid are skipped (the page staging reports them).
// ---------------------------------------------------------------------------
template <int D, int NT>
__device__ __forceinline__ void append_window(int tid, int a, int b, int L, int s, int R, int Hkv,
                                              int kvh, const int32_t* __restrict__ pt, int pool_pages,
                                              char* __restrict__ kpb, char* __restrict__ vpb,
                                              const char* __restrict__ knb,
                                              const char* __restrict__ vnb) {
  constexpr int CPR = D / 8;
  constexpr int KROWB = D * 2;
  constexpr int PAGE_K = 16 * KROWB;
  constexpr int PAGE_V = D * 32;
  // K: (b - a) rows of CPR 16-byte chunks, two chunks per thread per batch
  const int nk = (b - a) * CPR;
#pragma unroll 1
  for (int i0 = tid; i0 < nk; i0 += 2 * NT) {
    u32x4 x[2];
    int pg[2];
#pragma unroll
    for (int e = 0; e < 2; ++e) {
      const int i = i0 + e * NT;
      const bool live = i < nk;
      const int key = a + (live ? i / CPR : 0), cc = live ? i % CPR : 0;
      pg[e] = live ? pt[key >> 4] : -1;
      x[e] = *(const u32x4*)(knb + (((size_t)s * R + (key - L)) * Hkv + kvh) * KROWB + cc * 16);
    }
#pragma unroll
    for (int e = 0; e < 2; ++e) {
      const int i = i0 + e * NT;
      if (i >= nk || pg[e] < 0 || pg[e] >= pool_pages) continue;
      const int key = a + i / CPR, cc = i % CPR;
      *(u32x4*)(kpb + ((size_t)pg[e] * Hkv + kvh) * PAGE_K + (key & 15) * KROWB + cc * 16) = x[e];
    }
  }
  // V: pages [a / 16, (b - 1) / 16], one (page, head-dim element) row per thread
  const int p0 = a >> 4;
  const int nv = (((b - 1) >> 4) - p0 + 1) * D;
#pragma unroll 1
  for (int i = tid; i < nv; i += NT) {
    const int pi = p0 + i / D, d = i % D;
    const int pg = pt[pi];
    if (pg < 0 || pg >= pool_pages) continue;
    char* row = vpb + ((size_t)pg * Hkv + kvh) * PAGE_V + d * 32;
    const int lo = max(a, pi * 16) - pi * 16, hi = min(b, pi * 16 + 16) - pi * 16;   // new slots [lo, hi)
    u32x4 o0 = u32x4{0, 0, 0, 0}, o1 = u32x4{0, 0, 0, 0};
    if (lo > 0 || hi < 16) {
      o0 = *(const u32x4*)row;
      o1 = *(const u32x4*)(row + 16);
    }
    uint16_t nvv[16];
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int key = pi * 16 + (e >= lo && e < hi ? e : lo);
      nvv[e] = *(const uint16_t*)(vnb + (((size_t)s * R + (key - L)) * Hkv + kvh) * KROWB + d * 2);
    }
    uint32_t w[8] = {o0[0], o0[1], o0[2], o0[3], o1[0], o1[1], o1[2], o1[3]};
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      if (e >= lo && e < hi) {
        const int sh = 16 * (e & 1);
        w[e >> 1] = (w[e >> 1] & ~(0xffffu << sh)) | ((uint32_t)nvv[e] << sh);
      }
    }
    *(u32x4*)row = u32x4{w[0], w[1], w[2], w[3]};
    *(u32x4*)(row + 16) = u32x4{w[4], w[5], w[6], w[7]};
  }
}

// A V fragment of the 8 keys key0 .. key0 + 7 (bf16, in key order) with the
// keys >= T zeroed: past T the pool holds whatever the slots last held (a
// non-finite value there would turn its zero weight into NaN).
__device__ __forceinline__ bf16x8 v_keys_below(const bf16x8& f, int key0, int T) {
  const int nz = T - key0;
  u32x4 w = __builtin_bit_cast(u32x4, f);
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const uint32_t m = (2 * j + 1 < nz) ? 0xffffffffu : ((2 * j < nz) ? 0x0000ffffu : 0u);
    w[j] &= m;
  }
  return __builtin_bit_cast(bf16x8, w);
}

__device__ __forceinline__ uint32_t lds_addr(const void* ptr) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)ptr;
}

// MFMA operand fragments of the producer/consumer kernel are read from LDS
// with explicit waits: the compiler's wait insertion cannot tell the ring
// slot being read from the slots in-flight direct loads are filling, and
// would drain all of them before every read.  LDS reads complete in order,
// so "at most N LDS operations outstanding" completes every read but the N
// youngest; operations the compiler adds only make the wait longer.  The
// wait names the fragment as an in/out operand, so no use of it can be
// scheduled above the wait.
template <int OFF>
__device__ __forceinline__ bf16x8 lds_read16(uint32_t addr) {
  static_assert(OFF >= 0 && OFF < 65536, "ds offset field");
  bf16x8 r;
  asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(r) : "v"(addr), "n"(OFF) : "memory");
  return r;
}

template <int N>
__device__ __forceinline__ void lds_wait(bf16x8& frag) {
  static_assert(N >= 0 && N < 16, "lgkmcnt range");
  asm volatile("s_waitcnt lgkmcnt(%1)" : "+v"(frag) : "n"(N) : "memory");
}

// Issue the N reads rd(n) in order with DEPTH in flight; hand read n to
// use(n, fragment) once it has arrived.  A ring slot is refilled one use
// after it was consumed.
template <int N, int DEPTH, typename RD, typename USE>
__device__ __forceinline__ void lds_pipeline(RD&& rd, USE&& use) {
  constexpr int RING = DEPTH + 1;
  constexpr int PRE = DEPTH < N ? DEPTH : N;
  bf16x8 ring[RING];
  static_for<0, PRE>([&](auto c) { ring[decltype(c)::value % RING] = rd(c); });
  static_for<0, N>([&](auto c) {
    constexpr int n = decltype(c)::value;
    constexpr int issued = (n + DEPTH < N) ? n + DEPTH : N;
    lds_wait<issued - (n + 1)>(ring[n % RING]);
    use(c, ring[n % RING]);
    if constexpr (n + DEPTH < N) ring[(n + DEPTH) % RING] = rd(IC<n + DEPTH>{});
  });
}

// Barrier for the producer/consumer kernel: completes this wave's LDS
// operations (P hand-off writes, fragment reads) and meets the other waves.
// Inline, so no compiler-inserted wait for in-flight direct loads rides on it.
__device__ __forceinline__ void pc_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

template <int D, int NW>
__global__ void __launch_bounds__(NW * 64, 1) attn_bf16_kernel(AttnParams p) {
  constexpr int NT = NW * 64;
  constexpr int CPR = D / 8;
  constexpr int KROWB = D * 2;
  constexpr int KTILE_B = KT * KROWB;
  constexpr int VTILE_B = KT * D * 2;
  constexpr int STAGE_B = KTILE_B + VTILE_B;
  constexpr int K_INS = KTILE_B / (NT * 16);
  constexpr int V_INS = VTILE_B / (NT * 16);
  constexpr int NPL = K_INS + V_INS;
  constexpr int KS = D / 16;
  constexpr int DG = D / 32;
  constexpr int KG = KT / 32;
  constexpr int RPW = NW * 32;
  constexpr int PAGE_K = 16 * KROWB;
  constexpr int PAGE_V = D * 32;
  constexpr int SEGPP_K = PAGE_K / 1024;
  constexpr int SEGPP_V = PAGE_V / 1024;
  constexpr bool KXOR = (KROWB & (KROWB - 1)) == 0;   // row stride a power of two
  static_assert(KTILE_B % (NT * 16) == 0 && VTILE_B % (NT * 16) == 0, "tile / wave mismatch");
  static_assert(PAGE_K % 1024 == 0 && PAGE_V % 1024 == 0, "page / segment mismatch");
  constexpr int NREG = DG * 16;

  __shared__ __attribute__((aligned(1024))) char smem[NSTAGE * STAGE_B];
  __shared__ int s_pages[SUB_TILES * 4 + 4];
  __shared__ int s_seq[BAL_MAX_SEQS + 1];   // balanced: tile prefix over sequences
  __shared__ int s_flag[2];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = tid >> 6;
  const int hh = lane >> 5;
  const int l32 = lane & 31;
  const int R = p.R;
  const int HN = p.Hkv * p.n_row_tiles;   // items per sequence

  const __bf16* __restrict__ q = (const __bf16*)p.q;
  const char* __restrict__ knb = (const char*)p.k_new;
  const char* __restrict__ vnb = (const char*)p.v_new;
  char* __restrict__ kpb = (char*)p.k_pool;
  char* __restrict__ vpb = (char*)p.v_pool;
  __bf16* __restrict__ out = (__bf16*)p.out;

  // ---- per-lane constant offsets of the direct loads (within a page)
  uint32_t koff[K_INS], voff[V_INS];
#pragma unroll
  for (int j = 0; j < K_INS; ++j) {
    const int off = (w * K_INS + j) * 1024 + lane * 16;
    const int row = off / KROWB;
    const int cc = ((off % KROWB) >> 4) ^ kswz<CPR>(row);
    koff[j] = (uint32_t)((row & 15) * KROWB + cc * 16);
  }
#pragma unroll
  for (int j = 0; j < V_INS; ++j) {
    const int off = (w * V_INS + j) * 1024 + lane * 16;
    const int rem = off % PAGE_V;
    const int d = rem >> 5;
    const int hc = ((rem >> 4) & 1) ^ vswz(d);
    voff[j] = (uint32_t)(d * 32 + hc * 16);
  }
  // per-lane fragment offsets within a stage buffer
  int kfrag[KG];
#pragma unroll
  for (int kg = 0; kg < KG; ++kg) {
    const int row = kg * 32 + kperm(l32);
    kfrag[kg] = row * KROWB + (KXOR ? ((hh ^ kswz<CPR>(row)) << 4) : 0);
  }
  const int ksw = kswz<CPR>(kperm(l32));   // same for kg = 0, 1 (row differs by 32)
  const int vfrag = KTILE_B + l32 * 32 + ((hh ^ vswz(l32)) << 4);

  // ---- work decomposition
  // segments: (item, tile range [j0, j1), segment index k, segments nseg)
  int u = 0, u_end = 0;          // balanced: global tile range of this workgroup
  int share = 0;
  int it_a = 0, c_a = 0;         // aligned: item and chunk
  if (p.balanced) {
    // tile prefix over sequences (invalid sequences contribute no tiles)
    if (tid == 0) s_flag[0] = 0;
    for (int s0 = 0; s0 < p.S; s0 += NT) {
      __syncthreads();
      int t = 0;
      const int s = s0 + tid;
      if (s < p.S) {
        const int L = p.kv_len[s];
        const int T = L + R;
        if (L < 0 || T > p.max_pages * 16) {
          s_flag[0] = 1;
        } else {
          t = (T + KT - 1) / KT;
        }
      }
      // inclusive scan of t over this block of sequences (Hillis-Steele)
      s_seq[1 + tid + s0] = t;   // s0 + NT <= BAL_MAX_SEQS guaranteed by the host
      __syncthreads();
      for (int off = 1; off < NT; off <<= 1) {
        const int v = (tid >= off && s0 + tid < p.S) ? s_seq[1 + s0 + tid - off] : 0;
        __syncthreads();
        if (s0 + tid < p.S) s_seq[1 + s0 + tid] += v;
        __syncthreads();
      }
      if (s0 > 0 && s0 + tid < p.S) s_seq[1 + s0 + tid] += s_seq[s0];
      // (the carry read above sees the previous block's final value)
    }
    if (tid == 0) s_seq[0] = 0;
    __syncthreads();
    if (blockIdx.x == 0 && tid == 0 && s_flag[0]) set_err(p.err, DVS_ERR_MAX_PAGES);
    const int U = s_seq[p.S] * HN;
    share = max((U + (int)gridDim.x - 1) / (int)gridDim.x, p.share_min);
    u = (int)blockIdx.x * share;
    u_end = min(u + share, U);
    if (u >= u_end) return;
  } else {
    int idx = blockIdx.x;
    it_a = idx % p.n_items;
    c_a = idx / p.n_items;
  }

  bool first_segment = true;
  int s_cur = 0;                 // balanced: sequence cursor
  while (true) {
    int s, kvh, rt, it, j0, j1, k, nseg, L;
    if (p.balanced) {
      if (u >= u_end) break;
      while (s_seq[s_cur + 1] * HN <= u) ++s_cur;
      s = s_cur;
      L = p.kv_len[s];
      const int tiles = s_seq[s + 1] - s_seq[s];
      const int local = u - s_seq[s] * HN;
      const int qi = local / tiles;
      j0 = local - qi * tiles;
      j1 = min(tiles, j0 + (u_end - u));
      it = s * HN + qi;
      kvh = qi / p.n_row_tiles;
      rt = qi - kvh * p.n_row_tiles;
      const int P0 = s_seq[s] * HN + qi * tiles;     // first unit of the item
      k = (int)blockIdx.x - P0 / share;
      nseg = (P0 + tiles - 1) / share - P0 / share + 1;
      u += j1 - j0;
    } else {
      if (!first_segment) break;
      it = it_a;
      s = it / HN;
      const int qi = it - s * HN;
      kvh = qi / p.n_row_tiles;
      rt = qi - kvh * p.n_row_tiles;
      L = p.kv_len[s];
      const int T = L + R;
      if (L < 0 || T > p.max_pages * 16) {
        if (c_a == 0 && qi == 0 && tid == 0) set_err(p.err, DVS_ERR_MAX_PAGES);
        return;
      }
      const int tiles = (T + KT - 1) / KT;
      nseg = (tiles + p.chunk_tiles - 1) / p.chunk_tiles;
      if (c_a >= nseg) return;
      k = c_a;
      j0 = c_a * p.chunk_tiles;
      j1 = min(tiles, j0 + p.chunk_tiles);
    }
    if (!first_segment) __syncthreads();   // previous segment fully done with LDS
    first_segment = false;
    const int T = L + R;
    const int32_t* __restrict__ pt = p.page_table + (size_t)s * p.max_pages;
    const int n_valid = (T + 15) >> 4;    // pages the sequence holds
    // the page ids of the segment's first sub-range, loaded together with Q
    // (one wait for both)
    int pg_pre = 0;
    if (tid < min(j1, j0 + SUB_TILES) * 4 - j0 * 4) pg_pre = pt[min(j0 * 4 + tid, n_valid - 1)];

    // ---- rows of this lane: Q fragments (B operand), visibility limit
    const int n = rt * RPW + w * 32 + l32;
    const bool rvalid = n < p.rows_total;
    const int r = n / p.G;
    const int h = kvh * p.G + (n - r * p.G);
    const int hi = !rvalid ? -1 : row_hi(p, L, r);
    bf16x8 qf[KS];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      qf[ks] = rvalid ? *(const bf16x8*)(q + (((size_t)s * R + r) * p.Hq + h) * D + ks * 16 + hh * 8)
                      : bf16x8{};
    // Complete the Q loads here, then re-define the fragments through an empty
    // asm: the waitcnt pass otherwise cannot prove inside the tile loop that
    // they are complete and waits for every in-flight cache-tile load.
    wait_vmcnt<0>();
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) asm volatile("" : "+v"(qf[ks]));

    f32x16 o[DG];
#pragma unroll
    for (int dg = 0; dg < DG; ++dg) o[dg] = f32x16{};
    float m = -INFINITY, lsum = 0.f;

    // ---- one tile of compute from LDS
    auto compute_tile = [&](const char* stage, int key0, bool masked) {
      f32x16 sacc[KG];
#pragma unroll
      for (int kg = 0; kg < KG; ++kg) sacc[kg] = f32x16{};
      // K fragments are read one k-step ahead of the MFMAs that use them
      auto kload = [&](int ks, int kg) {
        const int off = KXOR ? (kfrag[kg] ^ (ks << 5))
                             : (kfrag[kg] + ((((ks << 1) | hh) ^ ksw) << 4));
        return *(const bf16x8*)(stage + off);
      };
      bf16x8 ka[2][KG];
#pragma unroll
      for (int kg = 0; kg < KG; ++kg) ka[0][kg] = kload(0, kg);
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        if (ks + 1 < KS) {
#pragma unroll
          for (int kg = 0; kg < KG; ++kg) ka[(ks + 1) & 1][kg] = kload(ks + 1, kg);
        }
#pragma unroll
        for (int kg = 0; kg < KG; ++kg)
          sacc[kg] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka[ks & 1][kg], qf[ks], sacc[kg], 0, 0, 0);
      }
      if (masked) {
        const Vis2 v2 = rvalid ? group_interval(p, L, r) : Vis2{1 << 30, -1};
#pragma unroll
        for (int kg = 0; kg < KG; ++kg)
#pragma unroll
          for (int i = 0; i < 16; ++i) {
            const int key = key0 + kg * 32 + 16 * (i >> 3) + 8 * hh + (i & 7);
            if (key > hi && (key < v2.lo2 || key > v2.hi2)) sacc[kg][i] = -INFINITY;
          }
      }
      // tile max: a tree over the lane's 16*KG scores, then lane^32
      float mx[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) mx[j] = fmaxf(sacc[0][2 * j], sacc[0][2 * j + 1]);
#pragma unroll
      for (int kg = 1; kg < KG; ++kg)
#pragma unroll
        for (int j = 0; j < 8; ++j) mx[j] = fmaxf(mx[j], fmaxf(sacc[kg][2 * j], sacc[kg][2 * j + 1]));
      float tmax = fmaxf(fmaxf(fmaxf(mx[0], mx[1]), fmaxf(mx[2], mx[3])),
                         fmaxf(fmaxf(mx[4], mx[5]), fmaxf(mx[6], mx[7])));
      {
        const f32x2 hp = halves_pair(tmax);
        tmax = fmaxf(hp[0], hp[1]);
      }
      // The row's reference maximum m only moves when the tile maximum exceeds
      // it by more than 2^RESCALE_LOG2 (weights stay <= 2^RESCALE_LOG2 and the
      // final division by l is exact about it); the wave skips the O rescale
      // when no row moved.  The decision is per row.
      const float cand = tmax * p.scale_log2;
      const bool move = cand > m + RESCALE_LOG2;
      if (__ballot(move)) {
        const float alpha = move ? __builtin_amdgcn_exp2f(m - cand) : 1.f;
        lsum *= alpha;
#pragma unroll
        for (int dg = 0; dg < DG; ++dg) o[dg] *= alpha;
      }
      if (move) m = cand;
      const float msafe = (m == -INFINITY) ? 0.f : m;
      bf16x8 pf[KT / 16];
      float psum[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int t = 0; t < KT / 16; ++t) {
        uint32_t pk[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int i0 = 8 * (t & 1) + 2 * e;
          const float a0 = __builtin_amdgcn_exp2f(fmaf(sacc[t >> 1][i0], p.scale_log2, -msafe));
          const float a1 = __builtin_amdgcn_exp2f(fmaf(sacc[t >> 1][i0 + 1], p.scale_log2, -msafe));
          psum[e] += a0 + a1;
          pk[e] = __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{a0, a1}, bf16x2));
        }
        pf[t] = __builtin_bit_cast(bf16x8, u32x4{pk[0], pk[1], pk[2], pk[3]});
      }
      lsum += (psum[0] + psum[1]) + (psum[2] + psum[3]);
      // V fragments are read one k-step ahead of the MFMAs that use them;
      // in the tile that runs past T (TAIL), keys >= T are zeroed
      auto pv = [&](auto tail) {
        constexpr bool TAIL = decltype(tail)::value != 0;
        bf16x8 va[2][DG];
#pragma unroll
        for (int dg = 0; dg < DG; ++dg) va[0][dg] = *(const bf16x8*)(stage + vfrag + dg * 32 * 32);
#pragma unroll
        for (int t = 0; t < KT / 16; ++t) {
          if (t + 1 < KT / 16) {
#pragma unroll
            for (int dg = 0; dg < DG; ++dg)
              va[(t + 1) & 1][dg] = *(const bf16x8*)(stage + vfrag + ((t + 1) * D + dg * 32) * 32);
          }
#pragma unroll
          for (int dg = 0; dg < DG; ++dg) {
            bf16x8 vf = va[t & 1][dg];
            if constexpr (TAIL) vf = v_keys_below(vf, key0 + t * 16 + 8 * hh, T);
            o[dg] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[t], o[dg], 0, 0, 0);
          }
        }
      };
      if (key0 + KT > T) pv(IC<1>{});
      else pv(IC<0>{});
    };

    // ---- the window keys of the segment's tiles go to their pool slots
    // first; then every tile streams through the direct-load ring
    {
      const int wa = max(L, j0 * KT), wb = min(T, j1 * KT);
      if (wa < wb) {
        append_window<D, NT>(tid, wa, wb, L, s, R, p.Hkv, kvh, pt, p.pool_pages, kpb, vpb, knb, vnb);
        wait_vmcnt<0>();
        __syncthreads();
      }
    }
    // ---- the segment's tiles, in sub-ranges whose page ids fit in LDS
    for (int ja = j0; ja < j1; ja += SUB_TILES) {
      const int jb = min(j1, ja + SUB_TILES);
      const int pg_lo = ja * 4;
      const int pg_hi = jb * 4;
      if (ja != j0) __syncthreads();
      if (tid == 0) s_flag[1] = 0;
      __syncthreads();
      for (int i = tid; i < pg_hi - pg_lo; i += NT) {
        // pages past the last one of the sequence (in the tile that runs
        // past T) repeat the last page: their keys are masked
        int pg = (ja == j0 && i == tid) ? pg_pre : pt[min(pg_lo + i, n_valid - 1)];
        if (pg < 0 || pg >= p.pool_pages) {
          pg = 0;
          s_flag[1] = 1;
        }
        s_pages[i] = pg;
      }
      __syncthreads();   // also completes the Q loads
      if (tid == 0 && s_flag[1]) set_err(p.err, DVS_ERR_BAD_PAGE);

      // every tile through the direct-load ring; tiles that reach L are masked
      const int n_main = jb - ja;
      auto issue = [&](int i) {
        char* stage = smem + (i % NSTAGE) * STAGE_B;
        const int pbase = i * 4;          // first page of tile ja+i, relative to pg_lo
#pragma unroll
        for (int j = 0; j < K_INS; ++j) {
          const int seg = w * K_INS + j;
          const int pg = __builtin_amdgcn_readfirstlane(s_pages[pbase + seg / SEGPP_K]);
          const char* base = kpb + ((size_t)pg * p.Hkv + kvh) * PAGE_K;
          __builtin_amdgcn_global_load_lds((const void*)(base + koff[j]),
              (__attribute__((address_space(3))) void*)(stage + seg * 1024), 16, 0, 0);
        }
#pragma unroll
        for (int j = 0; j < V_INS; ++j) {
          const int seg = w * V_INS + j;
          const int pg = __builtin_amdgcn_readfirstlane(s_pages[pbase + seg / SEGPP_V]);
          const char* base = vpb + ((size_t)pg * p.Hkv + kvh) * PAGE_V;
          __builtin_amdgcn_global_load_lds((const void*)(base + voff[j]),
              (__attribute__((address_space(3))) void*)(stage + KTILE_B + seg * 1024), 16, 0, 0);
        }
      };
#pragma unroll
      for (int i = 0; i < NSTAGE - 1; ++i)
        if (i < n_main) issue(i);
      for (int i = 0; i < n_main; ++i) {
        wait_tiles<NPL>(min(NSTAGE - 2, n_main - 1 - i));
        __builtin_amdgcn_s_barrier();     // tile i complete for every wave; tile i-1 consumed
        if (i + NSTAGE - 1 < n_main) issue(i + NSTAGE - 1);
        compute_tile(smem + (i % NSTAGE) * STAGE_B, (ja + i) * KT, ja + i >= L / KT);
      }
    }

    // ---- finish the segment
    {
      const f32x2 hp = halves_pair(lsum);
      lsum = hp[0] + hp[1];
    }
    auto write_out = [&](const f32x16* ov, float inv) {
      if (!rvalid) return;
      __bf16* orow = out + (((size_t)s * R + r) * p.Hq + h) * D;
#pragma unroll
      for (int dg = 0; dg < DG; ++dg)
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) {
          const int d = dg * 32 + 8 * g4 + 4 * hh;
          const f32x2 v01 = f32x2{ov[dg][4 * g4 + 0] * inv, ov[dg][4 * g4 + 1] * inv};
          const f32x2 v23 = f32x2{ov[dg][4 * g4 + 2] * inv, ov[dg][4 * g4 + 3] * inv};
          const uint32_t w0 = __builtin_bit_cast(uint32_t, __builtin_convertvector(v01, bf16x2));
          const uint32_t w1 = __builtin_bit_cast(uint32_t, __builtin_convertvector(v23, bf16x2));
          *(u32x2*)(orow + d) = u32x2{w0, w1};
        }
    };
    if (nseg == 1) {
      write_out(o, lsum > 0.f ? 1.f / lsum : 0.f);
      continue;
    }
    // Publish the partial: O / l in bf16 (16-byte words of 8 values, word j
    // of every thread side by side, so that each store and load of a wave
    // covers 1 KB in one piece) and (m, l) in fp32 per thread; wait for the
    // stores, then count in; the workgroup that completes the item merges.
    const int wg0 = (int)blockIdx.x - k;
    const size_t slot = part_slot(p.balanced, it, p.max_segs, wg0, k);
    // a wave whose 32 rows all lie past the item's rows has nothing to
    // publish or merge (few-row calls run four waves for the copies)
    const bool wave_rows = rt * RPW + w * 32 < p.rows_total;
    constexpr int NWD = NREG / 8;   // 16-byte words of a thread's partial
    if (wave_rows) {
      uint32_t* po = (uint32_t*)p.part_o + slot * (size_t)(NT * NREG / 2) + (size_t)tid * 4;
      float* pml = p.part_ml + slot * (size_t)(NT * 2) + (size_t)tid * 2;
      *(f32x2*)pml = f32x2{m, lsum};
      const float inv = lsum > 0.f ? 1.f / lsum : 0.f;
#pragma unroll
      for (int jw = 0; jw < NWD; ++jw) {
        u32x4 v;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int f0 = 8 * jw + 2 * e;   // element f of the thread: o[f / 16][f % 16]
          const f32x2 pr = f32x2{o[f0 / 16][f0 % 16] * inv, o[(f0 + 1) / 16][(f0 + 1) % 16] * inv};
          v[e] = __builtin_bit_cast(uint32_t, __builtin_convertvector(pr, bf16x2));
        }
        *(u32x4*)(po + jw * (NT * 4)) = v;
      }
    }
    wait_vmcnt<0>();
    __syncthreads();
    // The count-in is a release (the partials written by every thread of the
    // workgroup, ordered before it by the barrier, become visible at agent
    // scope first); the count-ins form one release sequence, so the last
    // workgroup's acquire fence after its own count-in makes every other
    // workgroup's partials visible to its loads below (the barrier extends it
    // to all its threads).  Only that workgroup pays for the acquire.
    if (tid == 0) {
      const bool last = __hip_atomic_fetch_add(&p.counters[it], 1, __ATOMIC_RELEASE,
                                               __HIP_MEMORY_SCOPE_AGENT) == nseg - 1;
      if (last) __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
      s_flag[0] = last;
    }
    __syncthreads();
    if (!s_flag[0]) continue;
    if (tid == 0) __hip_atomic_store(&p.counters[it], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (!wave_rows) continue;
    // Partials are read in batches issued in full before any of it is used,
    // so the loads overlap instead of each one waiting for the previous.
    auto ml_of = [&](int c) {
      return *(const f32x2*)(p.part_ml + part_slot(p.balanced, it, p.max_segs, wg0, c) * (NT * 2) +
                             (size_t)tid * 2);
    };
    // SB segments per batch (eight where the registers allow), added in
    // segment order: O += exp2(m_c - M) l_c (O_c / l_c), l += exp2(m_c - M) l_c.
    // M, the largest m_c, is found in a first pass over the (m, l) pairs,
    // or from the batch itself when one batch holds every segment (one
    // round of loads instead of two).
    constexpr int SB = NREG <= 48 ? 8 : 4;
    float M = -INFINITY;
    if (nseg > SB) {
      for (int c0 = 0; c0 < nseg; c0 += 8) {
        f32x2 mv[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) mv[j] = ml_of(min(c0 + j, nseg - 1));
#pragma unroll
        for (int j = 0; j < 8; ++j) M = fmaxf(M, mv[j][0]);   // repeats of the last segment are harmless
      }
    }
    float Ms = (M == -INFINITY) ? 0.f : M;
    f32x16 acc[DG];
#pragma unroll
    for (int dg = 0; dg < DG; ++dg) acc[dg] = f32x16{};
    float lt = 0.f;
    for (int c0 = 0; c0 < nseg; c0 += SB) {
      u32x4 pv[SB][NWD];
      f32x2 mlc[SB];
#pragma unroll
      for (int b = 0; b < SB; ++b) {
        const int c = min(c0 + b, nseg - 1);
        const uint32_t* src = (const uint32_t*)p.part_o +
                              part_slot(p.balanced, it, p.max_segs, wg0, c) * (NT * NREG / 2) +
                              (size_t)tid * 4;
#pragma unroll
        for (int jw = 0; jw < NWD; ++jw) pv[b][jw] = *(const u32x4*)(src + jw * (NT * 4));
        mlc[b] = ml_of(c);
      }
      if (nseg <= SB) {
#pragma unroll
        for (int b = 0; b < SB; ++b) M = fmaxf(M, mlc[b][0]);   // repeats of the last segment are harmless
        Ms = (M == -INFINITY) ? 0.f : M;
      }
#pragma unroll
      for (int b = 0; b < SB; ++b) {
        if (c0 + b >= nseg) break;
        const float wgt = __builtin_amdgcn_exp2f(mlc[b][0] - Ms) * mlc[b][1];
        lt += wgt;
#pragma unroll
        for (int jw = 0; jw < NWD; ++jw)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int f0 = 8 * jw + 2 * e;
            const uint32_t wd = pv[b][jw][e];
            acc[f0 / 16][f0 % 16] += wgt * __uint_as_float(wd << 16);
            acc[(f0 + 1) / 16][(f0 + 1) % 16] += wgt * __uint_as_float(wd & 0xffff0000u);
          }
      }
    }
    write_out(acc, lt > 0.f ? 1.f / lt : 0.f);
  }
}

// ---------------------------------------------------------------------------
// bf16, balanced work split, wide windows (>= 128 query rows per KV head):
// producer/consumer wave pairs.
//
// Pair k owns 64 query rows as two 32-row groups.  Its producer wave computes
// S^T = K Q^T for both groups (every K fragment read from LDS feeds two
// MFMAs) and the online softmax, and hands P (bf16, already in the PV MFMA's
// B-operand order) and the rescale factors to its consumer wave through LDS.
// The consumer wave accumulates O^T += V^T P^T for both groups (every V
// fragment feeds two MFMAs) and issues all direct cache loads.  Tile i of a
// segment takes one period of two halves:
//     producer:  QK(i)               | softmax(i), P(i) -> LDS
//     consumer:  P(i-1) -> registers, | O rescale, PV(i-1)
//                loads of group i    |
// so the consumer's MFMAs run under the producer's vector-ALU softmax (the
// two waves of a pair share a SIMD).  K and V tiles live in separate 3-slot
// rings: group g(i) = {K(i+2), V(i+1)} is issued in period i into the slots
// of K(i-1) and V(i-2), whose last readers finished in period i-1; period i
// waits for g(i-2) = {K(i), V(i-1)}.  A group's K part past the last tile
// re-reads the last tile into a dead slot, so every group has the same load
// count.  Producer and consumer keep their state in separate branches (the
// two roles' registers are not live at the same time), and both walk the
// same sequence of barriers.
// ---------------------------------------------------------------------------
constexpr int PC_NSTAGE = 3;
// Producer/consumer kernel, balanced split: cost units of a tile.  A tile
// that reaches the window streams like a cache tile but adds the masking, and
// the segment holding it first appends the window's K/V to the pool.
constexpr int PC_WM = 4;    // units of a cache tile (keys below L)
constexpr int PC_WW = 5;    // units of a window tile
// units added to the last tile of an item: the end of a segment there (the
// partial's publication, the next item's page staging and, for the last
// workgroup to finish the item, the merge)
constexpr int PC_WE = 24;
constexpr int PC_LDS_DEPTH = 6;

template <int D, int NP>
__global__ void __launch_bounds__(NP * 128, 1) attn_bf16_pc_kernel(AttnParams p) {
  constexpr int NC = NP * 64;            // threads per role
  constexpr int CPR = D / 8;
  constexpr int KROWB = D * 2;
  constexpr int KTILE_B = KT * KROWB;
  constexpr int VTILE_B = KT * D * 2;
  constexpr int K_INS = KTILE_B / (NC * 16);
  constexpr int V_INS = VTILE_B / (NC * 16);
  constexpr int NPL = K_INS + V_INS;
  constexpr int KS = D / 16;
  constexpr int DG = D / 32;
  constexpr int RPWG = NP * 64;
  constexpr int PAGE_K = 16 * KROWB;
  constexpr int PAGE_V = D * 32;
  constexpr int SEGPP_K = PAGE_K / 1024;
  constexpr int SEGPP_V = PAGE_V / 1024;
  constexpr bool KXOR = (KROWB & (KROWB - 1)) == 0;
  constexpr int NS = PC_NSTAGE;
  constexpr int OREG = 2 * DG * 16;      // partial O floats per consumer thread
  static_assert(KTILE_B % (NC * 16) == 0 && VTILE_B % (NC * 16) == 0, "tile / wave mismatch");
  static_assert(PAGE_K % 1024 == 0 && PAGE_V % 1024 == 0, "page / segment mismatch");
  static_assert(NPL < 64, "vmcnt range");
  static_assert(NP == 4 && K_INS == SEGPP_K && V_INS == SEGPP_V, "consumer wave k copies page k of a tile");

  __shared__ __attribute__((aligned(1024))) char kring[NS * KTILE_B];
  __shared__ __attribute__((aligned(1024))) char vring[NS * VTILE_B];
  __shared__ u32x4 s_P[NP][2][4][64];    // P of a pair: [group][16-key step][lane]
  __shared__ float s_alpha[NP][2][32];
  __shared__ int s_resc[NP];
  __shared__ int s_pages[SUB_TILES * 4 + 4];
  __shared__ int s_seq[BAL_MAX_SEQS + 1];
  __shared__ int s_flag[2];

  const int tid = threadIdx.x;
  // wave-uniform role (an SGPR), so the role branch is a real branch: its
  // two sides run different barrier sequences and keep separate registers
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const bool prod = w < NP;
  const int kp = prod ? w : w - NP;      // pair
  const int R = p.R;
  const int HN = p.Hkv * p.n_row_tiles;

  const __bf16* __restrict__ q = (const __bf16*)p.q;
  const char* __restrict__ knb = (const char*)p.k_new;
  const char* __restrict__ vnb = (const char*)p.v_new;
  char* __restrict__ kpb = (char*)p.k_pool;
  char* __restrict__ vpb = (char*)p.v_pool;
  __bf16* __restrict__ out = (__bf16*)p.out;

  // ---- balanced split: cost-unit prefix over sequences (every item of a
  // sequence has the same tiles), equal shares of units; a tile belongs to
  // the workgroup whose share holds its first unit
  if (tid == 0) s_flag[0] = 0;
  for (int s0 = 0; s0 < p.S; s0 += NP * 128) {
    __syncthreads();
    int t = 0;
    const int s = s0 + tid;
    if (s < p.S) {
      const int L = p.kv_len[s];
      const int T = L + R;
      if (L < 0 || T > p.max_pages * 16) s_flag[0] = 1;
      else t = PC_WM * (L / KT) + PC_WW * ((T + KT - 1) / KT - L / KT) + PC_WE;
    }
    s_seq[1 + tid + s0] = t;
    __syncthreads();
    for (int off = 1; off < NP * 128; off <<= 1) {
      const int v = (tid >= off && s0 + tid < p.S) ? s_seq[1 + s0 + tid - off] : 0;
      __syncthreads();
      if (s0 + tid < p.S) s_seq[1 + s0 + tid] += v;
      __syncthreads();
    }
    if (s0 > 0 && s0 + tid < p.S) s_seq[1 + s0 + tid] += s_seq[s0];
  }
  if (tid == 0) s_seq[0] = 0;
  __syncthreads();
  if (blockIdx.x == 0 && tid == 0 && s_flag[0]) set_err(p.err, DVS_ERR_MAX_PAGES);
  const int U = s_seq[p.S] * HN;
  const int share = max((U + (int)gridDim.x - 1) / (int)gridDim.x, p.share_min);
  const int u0 = (int)blockIdx.x * share;
  const int u_end = min(u0 + share, U);
  if (u0 >= u_end) return;

  // The two roles run separate copies of the segment loop (the same
  // segments and the same barrier sequence), so the register allocation of
  // one role never sees the other's live values.
  auto segments = [&](auto role) {
    constexpr bool PROD = decltype(role)::value != 0;
    bool first_segment = true;
    int s_cur = 0;
    int u = u0;
    while (u < u_end) {
      // Per-lane values are derived every segment from an opaque copy of the
      // thread index: hoisted out of the loop they would stay live across the
      // code of both roles.
      int tidv = tid;
      asm volatile("" : "+v"(tidv));
      const int lane = tidv & 63;
      const int hh = lane >> 5;
      const int l32 = lane & 31;
      const int ct = tidv - NC;            // consumer thread index (consumers only)
      while (s_seq[s_cur + 1] * HN <= u) ++s_cur;
      const int s = s_cur;
      const int L = p.kv_len[s];
      const int iu = s_seq[s + 1] - s_seq[s];            // units of one item
      const int qi = (u - s_seq[s] * HN) / iu;
      const int P0 = s_seq[s] * HN + qi * iu;             // first unit of the item
      const int nm = L / KT;                              // cache tiles
      const int tiles = (L + R + KT - 1) / KT;
      // first tile whose first unit is >= x (x in [0, iu]; iu maps to tiles)
      auto tile_at = [&](int x) {
        return x <= PC_WM * nm ? (x + PC_WM - 1) / PC_WM
                               : min(tiles, nm + (x - PC_WM * nm + PC_WW - 1) / PC_WW);
      };
      auto owner = [&](int j) {   // workgroup holding tile j's first unit
        return (P0 + (j <= nm ? PC_WM * j : PC_WM * nm + PC_WW * (j - nm))) / share;
      };
      const int j0 = tile_at(u - P0);
      const int j1 = tile_at(min(u_end, P0 + iu) - P0);
      u = P0 + iu;
      // (share >= PC_WW + PC_WE, the longest span of a tile: every workgroup
      // between an item's first and last owners holds at least one of its tiles)
      if (j0 >= j1) continue;
      const int it = s * HN + qi;
      const int kvh = qi / p.n_row_tiles;
      const int rt = qi - kvh * p.n_row_tiles;
      const int kseg = (int)blockIdx.x - owner(0);
      const int nseg = owner(tiles - 1) - owner(0) + 1;
      if (!first_segment) __syncthreads();
      first_segment = false;
      const int T = L + R;
      const int32_t* __restrict__ pt = p.page_table + (size_t)s * p.max_pages;

      // the lane's two rows (one per group) and their visibility limits
      bool rvalid[2];
      int rr[2], hq[2], hi[2];
#pragma unroll
      for (int g = 0; g < 2; ++g) {
        const int n = rt * RPWG + kp * 64 + g * 32 + l32;
        rvalid[g] = n < p.rows_total;
        rr[g] = n / p.G;
        hq[g] = kvh * p.G + (n - rr[g] * p.G);
        hi[g] = !rvalid[g] ? -1 : row_hi(p, L, rr[g]);
      }

      const int n_valid = (T + 15) >> 4;    // pages the sequence holds
      auto stage_pages = [&](int ja, int jb) {
        const int pg_lo = ja * 4;
        const int pg_hi = jb * 4;
        if (ja != j0) __syncthreads();
        if (tid == 0) s_flag[1] = 0;
        __syncthreads();
        for (int i = tidv; i < pg_hi - pg_lo; i += NP * 128) {
          // pages past the last one of the sequence (in the tile that runs
          // past T) repeat the last page: their keys are masked
          int pg = pt[min(pg_lo + i, n_valid - 1)];
          if (pg < 0 || pg >= p.pool_pages) {
            pg = 0;
            s_flag[1] = 1;
          }
          s_pages[i] = pg;
        }
        __syncthreads();
        if (tid == 0 && s_flag[1]) set_err(p.err, DVS_ERR_BAD_PAGE);
      };
      const int wg0 = owner(0);
      const size_t slot = part_slot(1, it, p.max_segs, wg0, kseg);
      // Merge of a split item by its last workgroup, all 512 threads: rows'
      // segment weights exp2(m_c - M) l_c / sum_c exp2(m_c - M) l_c go to LDS
      // (the K ring is idle by then), then every thread combines whole runs
      // of 4 output columns of one row, in segment order, with batched
      // coherent loads, and stores them as 8 bf16 bytes.
      auto merge_all = [&]() {
        const uint32_t* pob = (const uint32_t*)p.part_o;
        float* s_w = (float*)kring;   // [BAL_MAX_SEGS][RPWG]
        if (tid < RPWG) {
          float mv[BAL_MAX_SEGS], lv[BAL_MAX_SEGS];
#pragma unroll
          for (int c = 0; c < BAL_MAX_SEGS; ++c) {
            const int cc = min(c, nseg - 1);
            const float* src = p.part_ml + part_slot(1, it, p.max_segs, wg0, cc) * (2 * RPWG);
            mv[c] = __hip_atomic_load(src + tid, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            lv[c] = __hip_atomic_load(src + RPWG + tid, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          }
          float M = -INFINITY;
#pragma unroll
          for (int c = 0; c < BAL_MAX_SEGS; ++c) M = fmaxf(M, mv[c]);   // repeats of the last segment are harmless
          const float Ms = (M == -INFINITY) ? 0.f : M;
          float lt = 0.f;
#pragma unroll
          for (int c = 0; c < BAL_MAX_SEGS; ++c)
            if (c < nseg) lt += __builtin_amdgcn_exp2f(mv[c] - Ms) * lv[c];
          const float inv = lt > 0.f ? 1.f / lt : 0.f;
#pragma unroll
          for (int c = 0; c < BAL_MAX_SEGS; ++c)
            if (c < nseg) s_w[c * RPWG + tid] = __builtin_amdgcn_exp2f(mv[c] - Ms) * lv[c] * inv;
        }
        __syncthreads();
        // thread -> (row lane ct of the partial layout, half of its 4-column runs)
        const int ct = tid & (NC - 1);
        const int half = tid / NC;
        const int mkp = ct >> 6, mlane = ct & 63, ml32 = mlane & 31, mhh = mlane >> 5;
        constexpr int NQ = 2 * DG * 4;           // 4-column runs per row lane
        constexpr int QB = (NQ / 2) % 8 == 0 ? 8 : 4;   // runs per batch (two words each)
        static_assert((NQ / 2) % QB == 0, "merge batches");
#pragma unroll 1
        for (int q0 = 0; q0 < NQ / 2; q0 += QB) {
          float acc[QB][4];
#pragma unroll
          for (int b = 0; b < QB; ++b)
#pragma unroll
            for (int j = 0; j < 4; ++j) acc[b][j] = 0.f;
          // SBM segments' words in flight at once, then added in segment order
          constexpr int SBM = 2;
#pragma unroll 1
          for (int c0 = 0; c0 < nseg; c0 += SBM) {
            uint32_t v[SBM][QB][2];
#pragma unroll
            for (int sb = 0; sb < SBM; ++sb) {
              // opaque offset: the addresses are formed here, not hoisted
              int off = (int)part_slot(1, it, p.max_segs, wg0, min(c0 + sb, nseg - 1)) * (NC * OREG / 2) + ct;
              asm volatile("" : "+v"(off));
#pragma unroll
              for (int b = 0; b < QB; ++b) {
                const int q = half + 2 * (q0 + b);     // run index: g, dg, i4
                const int base_w = (q >> 2) * 8 + (q & 3) * 2;   // (g * DG + dg) * 8 + 2 * i4
#pragma unroll
                for (int j = 0; j < 2; ++j)
                  v[sb][b][j] = __hip_atomic_load(pob + off + (base_w + j) * NC, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
              }
            }
#pragma unroll
            for (int sb = 0; sb < SBM; ++sb) {
              const int c = c0 + sb;
              if (c >= nseg) break;
#pragma unroll
              for (int b = 0; b < QB; ++b) {
                const int q = half + 2 * (q0 + b);
                const int g = q / (DG * 4);
                const float wc = s_w[c * RPWG + mkp * 64 + g * 32 + ml32];
#pragma unroll
                for (int j = 0; j < 4; ++j)
                  acc[b][j] += wc * __uint_as_float((j & 1) ? (v[sb][b][j >> 1] & 0xffff0000u) : (v[sb][b][j >> 1] << 16));
              }
            }
          }
#pragma unroll
          for (int b = 0; b < QB; ++b) {
            const int q = half + 2 * (q0 + b);
            const int g = q / (DG * 4), dg = (q / 4) % DG, i4 = q & 3;
            const int n = rt * RPWG + mkp * 64 + g * 32 + ml32;
            if (n >= p.rows_total) continue;
            const int r = n / p.G;
            const int h = kvh * p.G + (n - r * p.G);
            const int d = dg * 32 + 8 * i4 + 4 * mhh;
            const uint32_t w0 = __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{acc[b][0], acc[b][1]}, bf16x2));
            const uint32_t w1 = __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{acc[b][2], acc[b][3]}, bf16x2));
            *(u32x2*)(out + (((size_t)s * R + r) * p.Hq + h) * D + d) = u32x2{w0, w1};
          }
        }
      };

      // the window keys of this segment's tiles go to their pool slots first;
      // then every tile streams through the direct-load rings
      {
        const int wa = max(L, j0 * KT), wb = min(T, j1 * KT);
        if (wa < wb) {
          int tidw = tidv;   // opaque: nothing of the append is hoisted out of it
          asm volatile("" : "+v"(tidw));
          append_window<D, NP * 128>(tidw, wa, wb, L, s, R, p.Hkv, kvh, pt, p.pool_pages, kpb, vpb, knb, vnb);
          wait_vmcnt<0>();
          __syncthreads();
        }
      }

      if constexpr (PROD) {
        // =================== producer: QK and softmax ===================
        bf16x8 qf[2][KS];
#pragma unroll
        for (int g = 0; g < 2; ++g)
#pragma unroll
          for (int ks = 0; ks < KS; ++ks)
            qf[g][ks] = rvalid[g]
                            ? *(const bf16x8*)(q + (((size_t)s * R + rr[g]) * p.Hq + hq[g]) * D + ks * 16 + hh * 8)
                            : bf16x8{};
        wait_vmcnt<0>();
#pragma unroll
        for (int g = 0; g < 2; ++g)
#pragma unroll
          for (int ks = 0; ks < KS; ++ks) asm volatile("" : "+v"(qf[g][ks]));
        const int krow = kperm(l32);
        const int kfrag = krow * KROWB + (KXOR ? ((hh ^ kswz<CPR>(krow)) << 4) : 0);
        const int ksw = kswz<CPR>(krow);
        float m[2] = {-INFINITY, -INFINITY}, lsum[2] = {0.f, 0.f};
        f32x16 sacc[2][2];

        auto qk = [&](const char* kst) {
          const uint32_t kb = lds_addr(kst);
#pragma unroll
          for (int g = 0; g < 2; ++g)
#pragma unroll
            for (int kg = 0; kg < 2; ++kg) sacc[g][kg] = f32x16{};
          // read n = ks * 2 + kg: K rows of key group kg, head-dim step ks
          lds_pipeline<KS * 2, PC_LDS_DEPTH>(
              [&](auto c) {
                constexpr int n = decltype(c)::value;
                constexpr int ks = n / 2, kg = n % 2;
                const int row_off = kg * 32 * KROWB;
                const uint32_t a = KXOR ? (kb + (uint32_t)(row_off + (kfrag ^ (ks << 5))))
                                        : (kb + (uint32_t)(row_off + kfrag + ((((ks << 1) | hh) ^ ksw) << 4)));
                return lds_read16<0>(a);
              },
              [&](auto c, const bf16x8& kf) {
                constexpr int n = decltype(c)::value;
                constexpr int ks = n / 2, kg = n % 2;
                sacc[0][kg] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[0][ks], sacc[0][kg], 0, 0, 0);
                sacc[1][kg] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[1][ks], sacc[1][kg], 0, 0, 0);
              });
        };
        // softmax of both groups; P (bf16, B-operand order), the rescale
        // factors and the "some row moved" flag go to the pair's LDS slots
        auto softmax_out = [&](bool masked, int key0) {
          bool any_move = false;
#pragma unroll
          for (int g = 0; g < 2; ++g) {
            if (masked) {
              const Vis2 v2 = rvalid[g] ? group_interval(p, L, rr[g]) : Vis2{1 << 30, -1};
#pragma unroll
              for (int kg = 0; kg < 2; ++kg)
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                  const int key = key0 + kg * 32 + 16 * (i >> 3) + 8 * hh + (i & 7);
                  if (key > hi[g] && (key < v2.lo2 || key > v2.hi2)) sacc[g][kg][i] = -INFINITY;
                }
            }
            // tile max: two running max3 chains (one per 32-key group); a
            // chain keeps the compiler's NaN canonicalization to its head
            float ma = sacc[g][0][0], mb = sacc[g][1][0];
#pragma unroll
            for (int i = 1; i < 16; ++i) {
              ma = fmaxf(ma, sacc[g][0][i]);
              mb = fmaxf(mb, sacc[g][1][i]);
            }
            float tmax = fmaxf(ma, mb);
            {
              const f32x2 hp = halves_pair(tmax);
              tmax = fmaxf(hp[0], hp[1]);
            }
            // lazy rescale: the reference maximum moves only by more than
            // 2^RESCALE_LOG2; the consumer rescales O and l before its next PV
            const float cand = tmax * p.scale_log2;
            const bool move = cand > m[g] + RESCALE_LOG2;
            const float alpha = move ? __builtin_amdgcn_exp2f(m[g] - cand) : 1.f;
            if (move) m[g] = cand;
            any_move |= move;
            if (hh == 0) s_alpha[kp][g][l32] = alpha;
            const float msafe = (m[g] == -INFINITY) ? 0.f : m[g];
#pragma unroll
            for (int t = 0; t < KT / 16; ++t) {
              uint32_t pk[4];
#pragma unroll
              for (int e = 0; e < 4; ++e) {
                const int i0 = 8 * (t & 1) + 2 * e;
                const float a0 = __builtin_amdgcn_exp2f(fmaf(sacc[g][t >> 1][i0], p.scale_log2, -msafe));
                const float a1 = __builtin_amdgcn_exp2f(fmaf(sacc[g][t >> 1][i0 + 1], p.scale_log2, -msafe));
                pk[e] = __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{a0, a1}, bf16x2));
              }
              s_P[kp][g][t][lane] = u32x4{pk[0], pk[1], pk[2], pk[3]};
            }
          }
          const bool anyw = __ballot(any_move) != 0;
          if (lane == 0) s_resc[kp] = anyw ? 1 : 0;
        };

        for (int ja = j0; ja < j1; ja += SUB_TILES) {
          const int jb = min(j1, ja + SUB_TILES);
          stage_pages(ja, jb);
          const int n_main = jb - ja;
          // tiles below L, then the tiles that reach L (masked) and the
          // drain period: one period per tile plus one, as the consumer's
          const int n_c = min(max(nm - ja, 0), n_main);
          if (n_main > 0) {
            for (int i = 0; i < n_c; ++i) {
              pc_barrier();   // A: K(i) landed, P(i-1) taken
              qk(kring + (i % NS) * KTILE_B);
              pc_barrier();   // B: consumers hold P(i-1)
              softmax_out(false, 0);
            }
            for (int i = n_c; i <= n_main; ++i) {
              pc_barrier();
              // tile i-1 runs past T: its V entries of keys >= T are zeroed
              // in LDS before the consumer's products of this period read
              // them (their weights are zero; a stale non-finite value would
              // make the product NaN)
              if (i >= 1 && (ja + i) * KT > T) {
                char* vst = vring + ((i - 1) % NS) * VTILE_B;
                const int nk = T - (ja + i - 1) * KT;
                for (int e = tidv; e < (KT - nk) * D; e += NC) {
                  const int kk = nk + e / D, d = e % D;
                  const int tp = kk >> 4, kin = kk & 15;
                  *(uint16_t*)(vst + (tp * D + d) * 32 + ((((kin >> 3) ^ vswz(d)) << 4) | ((kin & 7) * 2))) = 0;
                }
              }
              if (i < n_main) qk(kring + (i % NS) * KTILE_B);
              pc_barrier();
              if (i < n_main) softmax_out(true, (ja + i) * KT);
            }
          }
        }
        // segment-final m (l is the consumer's)
        __syncthreads();                                     // F1
        if (nseg == 1) continue;
        float* pml = p.part_ml + slot * (size_t)(2 * RPWG);
        if (hh == 0) {
#pragma unroll
          for (int g = 0; g < 2; ++g)
            __hip_atomic_store(pml + kp * 64 + g * 32 + l32, m[g], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        wait_vmcnt<0>();
        __syncthreads();                                     // F2
        // release count-in; the acquire fence only in the last workgroup
        // (the count-ins form one release sequence)
        if (tid == 0) {
          const bool last = __hip_atomic_fetch_add(&p.counters[it], 1, __ATOMIC_RELEASE,
                                                   __HIP_MEMORY_SCOPE_AGENT) == nseg - 1;
          if (last) __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
          s_flag[0] = last;
        }
        __syncthreads();                                     // F3
        if (s_flag[0]) {
          if (tid == 0) __hip_atomic_store(&p.counters[it], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          merge_all();
        }
        continue;
      } else {
        // =================== consumer: loads, O rescale, PV ===================
        const int vfrag = l32 * 32 + ((hh ^ vswz(l32)) << 4);
        f32x16 o[2][DG];
#pragma unroll
        for (int g = 0; g < 2; ++g)
#pragma unroll
          for (int dg = 0; dg < DG; ++dg) o[g][dg] = f32x16{};
        // l of the lane's two rows over the lane's half of every tile's keys:
        // the sum of the bf16 weights the PV products use
        float lrow[2] = {0.f, 0.f};
        // P of one tile as handed over by the producer (declared per period so
        // that it is not carried around the tile loop)
        struct Hand {
          u32x4 pf[2][4];
          float alpha[2];
          int resc;
        };
        auto take_p = [&](Hand& hd) {   // P, rescale factors and flag of the producer's last tile
#pragma unroll
          for (int g = 0; g < 2; ++g) {
#pragma unroll
            for (int t = 0; t < 4; ++t) hd.pf[g][t] = s_P[kp][g][t][lane];
            hd.alpha[g] = s_alpha[kp][g][l32];
          }
          hd.resc = s_resc[kp];
          __builtin_amdgcn_s_waitcnt(0xc07f);   // lgkmcnt(0): the P reads are done before the barrier
        };
        // l: rescale, then add the tile's weights (a bf16 word widens to fp32
        // exactly: it is the high half).  Plain vector-ALU work, placed where
        // the pair's SIMD is busy with the producer's matrix products (a dot2
        // against (1, 1) was slower here: it competed with those products).
        auto add_l = [&](const Hand& hd) {
#pragma unroll
          for (int g = 0; g < 2; ++g) {
            float acc = 0.f;
#pragma unroll
            for (int t = 0; t < 4; ++t)
#pragma unroll
              for (int e = 0; e < 4; ++e)
                acc += __uint_as_float(hd.pf[g][t][e] << 16) + __uint_as_float(hd.pf[g][t][e] & 0xffff0000u);
            lrow[g] = fmaf(lrow[g], hd.alpha[g], acc);
          }
        };
        auto pv = [&](const Hand& hd, const char* vst) {
          if (hd.resc) {
#pragma unroll
            for (int g = 0; g < 2; ++g)
#pragma unroll
              for (int dg = 0; dg < DG; ++dg) o[g][dg] *= hd.alpha[g];
          }
          const uint32_t vb = lds_addr(vst) + (uint32_t)vfrag;
          // read n = t * DG + dg: V^T rows dg*32.. of key step t
          lds_pipeline<(KT / 16) * DG, PC_LDS_DEPTH>(
              [&](auto c) {
                constexpr int n = decltype(c)::value;
                constexpr int t = n / DG, dg = n % DG;
                return lds_read16<(t * D + dg * 32) * 32>(vb);
              },
              [&](auto c, const bf16x8& vf) {
                constexpr int n = decltype(c)::value;
                constexpr int t = n / DG, dg = n % DG;
                o[0][dg] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, __builtin_bit_cast(bf16x8, hd.pf[0][t]), o[0][dg], 0, 0, 0);
                o[1][dg] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, __builtin_bit_cast(bf16x8, hd.pf[1][t]), o[1][dg], 0, 0, 0);
              });
        };

        for (int ja = j0; ja < j1; ja += SUB_TILES) {
          const int jb = min(j1, ja + SUB_TILES);
          stage_pages(ja, jb);
          const int n_main = jb - ja;
          // With 4 pairs, consumer wave k copies page k of every 4-page tile
          // (its K_INS / V_INS 1 KB segments are exactly that page).
          int kpg = 0, vpg = 0;
          // page ids of group gi = {K(gi+2), V(gi+1)} (clamped), read in two
          // halves so that the LDS reads can share a wait with other reads
          int kraw = 0, vraw = 0;
          auto read_pages = [&](int gi) {
            const int ik = max(0, min(gi + 2, n_main - 1));
            const int iv = max(0, min(gi + 1, n_main - 1));
            kraw = s_pages[ik * 4 + kp];
            vraw = s_pages[iv * 4 + kp];
          };
          auto take_pages = [&]() {
            kpg = __builtin_amdgcn_readfirstlane(kraw);
            vpg = __builtin_amdgcn_readfirstlane(vraw);
          };
          auto fetch_pages = [&](int gi) {
            read_pages(gi);
            take_pages();
          };
          auto issue_k = [&](int gi) {   // K(gi + 2)
            // page bases are wave-uniform; the per-lane offsets are made opaque
            // here so that base + offset stays a scalar base plus a 32-bit
            // vector offset instead of hoisted 64-bit per-lane pointers
            // (the lane's source offsets within the page are recomputed per group
            // from an opaque lane index: cheaper than 2 * 4 registers held
            // across the tile loop)
            int ln = lane;
            asm volatile("" : "+v"(ln));
            {
              const char* base = kpb + ((size_t)kpg * p.Hkv + kvh) * PAGE_K;
              char* dst = kring + ((gi + 2 + NS) % NS) * KTILE_B + kp * (K_INS * 1024);
              // byte offset within the page of the lane's chunk of segment 0; when
              // a 1 KB segment holds whole rows, segment j's rows are 1024/KROWB*j
              // above segment 0's (their low bits are the lane's) and kswz is a
              // bit selection, so segment j's offset is segment 0's XOR a constant
              constexpr bool KLIN = (1024 % KROWB) == 0;
              constexpr uint32_t RPK = KLIN ? 1024 / KROWB : 1;
              const uint32_t off0 = (uint32_t)ln * 16u;
              const uint32_t row0 = off0 / (uint32_t)KROWB;
              const uint32_t src0 = row0 * (uint32_t)KROWB +
                  ((((off0 % (uint32_t)KROWB) >> 4) ^ (uint32_t)kswz<CPR>((int)row0)) << 4);
#pragma unroll
              for (int j = 0; j < K_INS; ++j) {
                uint32_t src;
                if constexpr (KLIN) {
                  src = (uint32_t)j * 1024u + (src0 ^ ((uint32_t)kswz<CPR>((int)(RPK * j)) << 4));
                } else {
                  // unsigned: the row division by a constant stays a mul_hi
                  const uint32_t off = (uint32_t)j * 1024u + off0;
                  const uint32_t row = off / (uint32_t)KROWB;
                  const uint32_t cc = ((off % (uint32_t)KROWB) >> 4) ^ (uint32_t)kswz<CPR>((int)row);
                  src = row * (uint32_t)KROWB + cc * 16u;
                }
                __builtin_amdgcn_global_load_lds((const void*)(base + src),
                    (__attribute__((address_space(3))) void*)(dst + j * 1024), 16, 0, 0);
              }
            }
          };
          auto issue_v = [&](int gi) {   // V(gi + 1)
            int ln = lane;
            asm volatile("" : "+v"(ln));
            {
              const char* base = vpb + ((size_t)vpg * p.Hkv + kvh) * PAGE_V;
              char* dst = vring + ((gi + 1 + NS) % NS) * VTILE_B + kp * (V_INS * 1024);
#pragma unroll
              for (int j = 0; j < V_INS; ++j) {
                const uint32_t off = (uint32_t)j * 1024u + (uint32_t)ln * 16u;
                const uint32_t d = off >> 5;
                const uint32_t hc = ((off >> 4) & 1u) ^ (uint32_t)vswz((int)d);
                const uint32_t src = d * 32u + hc * 16u;
                __builtin_amdgcn_global_load_lds((const void*)(base + src),
                    (__attribute__((address_space(3))) void*)(dst + j * 1024), 16, 0, 0);
              }
            }
          };
          auto issue_group = [&](int gi) {   // prologue groups
            issue_k(gi);
            issue_v(gi);
          };
          if (n_main > 0) {
            // g(-2) = {K(0), V(-1) re-reading tile 0 into the dead slot}, g(-1);
            // older stores (a previous segment's output) are drained first so
            // the counted waits below only count this ring's loads
            wait_vmcnt<0>();
            fetch_pages(-2);
            issue_group(-2);
            fetch_pages(-1);
            issue_group(-1);
            if (n_main >= 2) fetch_pages(0);
          }
          for (int i = 0; n_main > 0 && i <= n_main; ++i) {
            // g(i-1) is in flight (issued) iff i <= n_main - 1
            if (i <= n_main - 1) wait_vmcnt<NPL>();
            else wait_vmcnt<0>();
            pc_barrier();   // A
            Hand hd;
            // the next group's page ids are read with the hand-off (one wait)
            const bool nxt = i + 1 <= n_main - 2;
            if (nxt) read_pages(i + 1);
            if (i >= 1) take_p(hd);
            if (i >= 1) {
              add_l(hd);
              // keep the sums on this side of the barrier (they would
              // otherwise sink into the matrix-product phase)
              asm volatile("" ::"v"(lrow[0]), "v"(lrow[1]));
            }
            pc_barrier();   // B
            // The copies go out in phase 2, around the products: issuing 8
            // direct loads stalls the wave while the load path drains them,
            // which here overlaps the producer's softmax instead of delaying
            // barrier B; K (needed first) before the products, V after them.
            // Slots: K(i+2) replaces K(i-1) (read by QK(i-1) before barrier
            // A), V(i+1) replaces V(i-2) (read by PV(i-2) last period).
            if (i <= n_main - 2) issue_k(i);
            if (i >= 1) pv(hd, vring + ((i - 1) % NS) * VTILE_B);
            if (i <= n_main - 2) issue_v(i);
            if (nxt) take_pages();
          }
        }
        __syncthreads();                                       // F1
#pragma unroll
        for (int g = 0; g < 2; ++g) {
          const f32x2 hp = halves_pair(lrow[g]);
          lrow[g] = hp[0] + hp[1];
        }
        auto write_cols = [&](int g, int dg, const f32x16& ov, float inv) {   // columns dg*32..+31
          if (!rvalid[g]) return;
          __bf16* orow = out + (((size_t)s * R + rr[g]) * p.Hq + hq[g]) * D;
#pragma unroll
          for (int g4 = 0; g4 < 4; ++g4) {
            const int d = dg * 32 + 8 * g4 + 4 * hh;
            const f32x2 v01 = f32x2{ov[4 * g4 + 0] * inv, ov[4 * g4 + 1] * inv};
            const f32x2 v23 = f32x2{ov[4 * g4 + 2] * inv, ov[4 * g4 + 3] * inv};
            const uint32_t w0 = __builtin_bit_cast(uint32_t, __builtin_convertvector(v01, bf16x2));
            const uint32_t w1 = __builtin_bit_cast(uint32_t, __builtin_convertvector(v23, bf16x2));
            *(u32x2*)(orow + d) = u32x2{w0, w1};
          }
        };
        if (nseg == 1) {
#pragma unroll
          for (int g = 0; g < 2; ++g)
#pragma unroll
            for (int dg = 0; dg < DG; ++dg) write_cols(g, dg, o[g][dg], lrow[g] > 0.f ? 1.f / lrow[g] : 0.f);
          continue;
        }
        {
          // the segment's partial output O / l in bf16 (pairs of registers
          // in one word), m and l in fp32
          uint32_t* po = (uint32_t*)p.part_o + slot * (size_t)(NC * OREG / 2);
          if (hh == 0) {
            float* pml = p.part_ml + slot * (size_t)(2 * RPWG);
#pragma unroll
            for (int g = 0; g < 2; ++g)
              __hip_atomic_store(pml + RPWG + kp * 64 + g * 32 + l32, lrow[g], __ATOMIC_RELAXED,
                                 __HIP_MEMORY_SCOPE_AGENT);
          }
#pragma unroll
          for (int g = 0; g < 2; ++g) {
            const float inv = lrow[g] > 0.f ? 1.f / lrow[g] : 0.f;
#pragma unroll
            for (int dg = 0; dg < DG; ++dg)
#pragma unroll
              for (int i = 0; i < 16; i += 2) {
                const uint32_t w = __builtin_bit_cast(
                    uint32_t, __builtin_convertvector(f32x2{o[g][dg][i] * inv, o[g][dg][i + 1] * inv}, bf16x2));
                __hip_atomic_store(po + ((g * DG + dg) * 8 + i / 2) * NC + ct, w, __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
              }
          }
        }
        wait_vmcnt<0>();
        __syncthreads();                                       // F2
        __syncthreads();                                       // F3 (counter decided)
        if (s_flag[0]) merge_all();
      }
    }
  };
  if (prod) segments(IC<1>{});
  else segments(IC<0>{});
}

// ---------------------------------------------------------------------------
// fp32: one workgroup per (sequence, window row, query head); 256 threads.
// Scores for a 256-key tile in LDS, online softmax over tiles, thread d
// accumulates output element d.
// ---------------------------------------------------------------------------
template <int D>
__global__ void __launch_bounds__(256) attn_f32_kernel(AttnParams p) {
  __shared__ float sq[D];
  __shared__ float sp[256];
  __shared__ float sred[8];
  int idx = blockIdx.x;
  const int h = idx % p.Hq;
  idx /= p.Hq;
  const int r = idx % p.R;
  const int s = idx / p.R;
  const int tid = threadIdx.x;
  const int kvh = h / p.G;
  const int L = p.kv_len[s];
  const int R = p.R;
  const int T = L + R;
  if (L < 0 || T > p.max_pages * 16) {
    if (r == 0 && h == 0 && tid == 0) set_err(p.err, DVS_ERR_MAX_PAGES);
    return;
  }
  const int hi = row_hi(p, L, r);
  const Vis2 v2 = group_interval(p, L, r);
  const int hend = v2.hi2 > hi ? v2.hi2 : hi;   // last visible key
  const float* q = (const float*)p.q;
  const float* kn = (const float*)p.k_new;
  const float* vn = (const float*)p.v_new;
  float* kp = (float*)p.k_pool;
  float* vp = (float*)p.v_pool;
  const int32_t* pt = p.page_table + (size_t)s * p.max_pages;

  // append this row's K/V once per KV head (by the group's first query head)
  if (h % p.G == 0 && tid < D) {
    const int pos = L + r;
    const int pg = pt[pos >> 4];
    if (pg >= 0 && pg < p.pool_pages) {
      const size_t src = (((size_t)s * R + r) * p.Hkv + kvh) * D + tid;
      kp[(((size_t)pg * p.Hkv + kvh) * 16 + (pos & 15)) * D + tid] = kn[src];
      vp[(((size_t)pg * p.Hkv + kvh) * D + tid) * 16 + (pos & 15)] = vn[src];
    } else {
      set_err(p.err, DVS_ERR_BAD_PAGE);
    }
  }
  if (tid < D) sq[tid] = q[(((size_t)s * R + r) * p.Hq + h) * D + tid];
  __syncthreads();

  float m = -INFINITY, l = 0.f, acc = 0.f;
  bool bad = false;
  for (int t0 = 0; t0 <= hend; t0 += 256) {
    const int k = t0 + tid;
    float sc = -INFINITY;
    if (k <= hi || (k >= v2.lo2 && k <= v2.hi2)) {
      const float* krow = nullptr;
      if (k < L) {
        const int pg = pt[k >> 4];
        if (pg >= 0 && pg < p.pool_pages)
          krow = kp + (((size_t)pg * p.Hkv + kvh) * 16 + (k & 15)) * D;
        else
          bad = true;
      } else {
        krow = kn + (((size_t)s * R + (k - L)) * p.Hkv + kvh) * D;
      }
      if (krow) {
        float dot = 0.f;
        for (int d = 0; d < D; ++d) dot = fmaf(sq[d], krow[d], dot);
        sc = dot * p.scale;
      }
    }
    // tile max
    float v = sc;
    for (int off = 32; off > 0; off >>= 1) v = fmaxf(v, __shfl_xor(v, off));
    if ((tid & 63) == 0) sred[tid >> 6] = v;
    __syncthreads();
    const float tmax = fmaxf(fmaxf(sred[0], sred[1]), fmaxf(sred[2], sred[3]));
    __syncthreads();
    const float mnew = fmaxf(m, tmax);
    const float alpha = (m == -INFINITY) ? 0.f : expf(m - mnew);
    const float pe = (sc == -INFINITY) ? 0.f : expf(sc - mnew);
    sp[tid] = pe;
    float ps = pe;
    for (int off = 32; off > 0; off >>= 1) ps += __shfl_xor(ps, off);
    if ((tid & 63) == 0) sred[4 + (tid >> 6)] = ps;
    __syncthreads();
    l = l * alpha + ((sred[4] + sred[5]) + (sred[6] + sred[7]));
    m = mnew;
    if (tid < D) {
      float a = acc * alpha;
      const int nk = min(256, hend + 1 - t0);
      for (int j = 0; j < nk; ++j) {
        const int kk = t0 + j;
        float vv;
        if (kk < L) {
          const int pg = pt[kk >> 4];
          if (pg < 0 || pg >= p.pool_pages) continue;
          vv = vp[(((size_t)pg * p.Hkv + kvh) * D + tid) * 16 + (kk & 15)];
        } else {
          vv = vn[(((size_t)s * R + (kk - L)) * p.Hkv + kvh) * D + tid];
        }
        a = fmaf(sp[j], vv, a);
      }
      acc = a;
    }
    __syncthreads();
  }
  if (bad) set_err(p.err, DVS_ERR_BAD_PAGE);
  if (tid < D) ((float*)p.out)[(((size_t)s * R + r) * p.Hq + h) * D + tid] = acc / l;
}

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------
__global__ void attn_zero_kernel(int32_t* __restrict__ p, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0;
}

struct AttnPlan {
  int nw, rows_total, rows_per_wg, n_row_tiles, n_items, balanced, pc;
  int chunk_tiles, n_chunks_max, share_min, max_segs, grid;
  size_t off_counters, off_ml, off_o, bytes;
};

static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }


static AttnPlan plan_attn(int S, int R, int Hq, int Hkv, int D, int max_pages, int chunk_keys,
                          int dtype) {
  AttnPlan pl{};
  const int G = Hq / Hkv;
  pl.rows_total = R * G;
  pl.balanced = (chunk_keys == 0 && S <= BAL_MAX_SEQS) ? 1 : 0;
  if (dtype == DVS_BF16) {
    const int groups = (pl.rows_total + 31) / 32;   // 32-row MFMA groups
    pl.nw = groups >= 8 ? 8 : (groups >= 4 ? 4 : (groups >= 2 ? 2 : 1));
    if (D == 96 && pl.nw > 4) pl.nw = 4;   // a 96-wide tile splits over at most 4 waves
    // wide windows in the balanced split: producer/consumer pairs, 4 pairs
    // (8 waves, one producer and one consumer per SIMD) over 256 rows
    pl.pc = (pl.balanced && pl.rows_total > 128) ? 1 : 0;
    if (pl.pc) pl.nw = 8;
    // aligned chunks with few rows (decode steps): four waves all the same,
    // so that a chunk's copies are spread over them (a row's arithmetic does
    // not depend on the wave count)
    if (!pl.balanced && pl.nw < 4) pl.nw = 4;
  } else {
    pl.nw = 4;
  }
  pl.rows_per_wg = pl.nw * 32;
  pl.n_row_tiles = (pl.rows_total + pl.rows_per_wg - 1) / pl.rows_per_wg;
  pl.n_items = S * Hkv * pl.n_row_tiles;
  const int max_tiles = (max_pages * DVS_PAGE_SIZE + KT - 1) / KT;
  if (pl.balanced) {
    if (pl.pc) {
      // in cost units; an item has at most (R + KT - 1) / KT + 1 window tiles
      const int R = pl.rows_total / G;
      const int nwin = (R + KT - 1) / KT + 1;
      const int max_units = PC_WM * max_tiles + (PC_WW - PC_WM) * nwin + PC_WE;
      pl.share_min = std::max((max_units + BAL_MAX_SEGS - 2) / (BAL_MAX_SEGS - 1), PC_WW + PC_WE);
    } else {
      pl.share_min = (max_tiles + BAL_MAX_SEGS - 2) / (BAL_MAX_SEGS - 1);
    }
    if (pl.share_min < 1) pl.share_min = 1;
    pl.max_segs = BAL_MAX_SEGS;
    pl.grid = device_cus();
  } else {
    int C = chunk_keys > 0 ? chunk_keys : 4096;
    pl.chunk_tiles = C / KT;
    pl.n_chunks_max = (max_tiles + pl.chunk_tiles - 1) / pl.chunk_tiles;
    pl.max_segs = pl.n_chunks_max;
    pl.grid = pl.n_chunks_max * pl.n_items;
  }
  const int NT = pl.nw * 64;
  // partial slots: two per workgroup in the balanced split, one per (item,
  // chunk) in the aligned one (part_slot)
  const size_t slots = pl.balanced ? (size_t)2 * pl.grid : (size_t)pl.n_items * pl.max_segs;
  if (dtype == DVS_BF16) {
    // per slot: m and l of every query row (fp32), and O / l in bf16 -- per
    // thread and register in attn_bf16_kernel, as pairs per consumer thread
    // in the producer/consumer kernel (4 pairs, 256 rows)
    const size_t ml_b = pl.pc ? (size_t)2 * 256 * sizeof(float) : (size_t)NT * 2 * sizeof(float);
    const size_t o_b = pl.pc ? (size_t)256 * (2 * (D / 32) * 16) * 2
                             : (size_t)NT * (D / 32) * 16 * 2;
    pl.off_counters = 0;
    pl.off_ml = align256((size_t)pl.n_items * sizeof(int32_t));
    pl.off_o = pl.off_ml + align256(slots * ml_b);
    pl.bytes = pl.off_o + align256(slots * o_b);
  } else {
    pl.bytes = 256;
  }
  return pl;
}

template <int D>
static void launch_bf16(const AttnPlan& pl, const AttnParams& prm, hipStream_t st) {
  if (pl.pc) {
    hipLaunchKernelGGL((attn_bf16_pc_kernel<D, 4>), dim3(pl.grid), dim3(512), 0, st, prm);
    return;
  }
  switch (pl.nw) {
    case 8:
      if constexpr (D != 96)
        hipLaunchKernelGGL((attn_bf16_kernel<D, 8>), dim3(pl.grid), dim3(512), 0, st, prm);
      break;
    case 4: hipLaunchKernelGGL((attn_bf16_kernel<D, 4>), dim3(pl.grid), dim3(256), 0, st, prm); break;
    case 2: hipLaunchKernelGGL((attn_bf16_kernel<D, 2>), dim3(pl.grid), dim3(128), 0, st, prm); break;
    default: hipLaunchKernelGGL((attn_bf16_kernel<D, 1>), dim3(pl.grid), dim3(64), 0, st, prm); break;
  }
}

size_t attn_counter_bytes(int S, int R, int Hq, int Hkv, int D, int max_pages, int chunk_keys,
                          int dtype) {
  if (dtype != DVS_BF16) return 0;
  const AttnPlan pl = plan_attn(S, R, Hq, Hkv, D, max_pages, chunk_keys, dtype);
  return pl.off_ml - pl.off_counters;
}

}  // namespace dvs

using namespace dvs;

extern "C" size_t dvs_attn_workspace_bytes(int32_t S, int32_t n_causal, int32_t n_mask,
                                           int32_t Hq, int32_t Hkv, int32_t D, int32_t max_pages,
                                           int32_t chunk_keys, int32_t dtype) {
  if (S < 1 || n_causal < 0 || n_mask < 0 || n_causal + n_mask < 1 || Hkv < 1 || Hq < Hkv ||
      Hq % Hkv != 0 || max_pages < 1 || chunk_keys < 0)
    return 0;
  return plan_attn(S, n_causal + n_mask, Hq, Hkv, D, max_pages, chunk_keys, dtype).bytes;
}

// Host check and launch shared by attn_hybrid_block and
// attn_hybrid_block_noalloc.  `scratch_cap` > 0 marks the scratch-array
// variant: the workspace is the library's own array of that many bytes, and
// the split counters are cleared by a kernel at the start of every call.
static int attn_launch(const void* q, const void* k_new, const void* v_new, void* k_pool,
                       void* v_pool, const int32_t* page_table, const int32_t* kv_len, int32_t S,
                       int32_t n_causal, int32_t n_mask, int32_t Hq, int32_t Hkv, int32_t D,
                       int32_t max_pages, int32_t num_pool_pages, float softmax_scale,
                       int32_t dtype, int32_t chunk_keys, void* out, int32_t* err_word,
                       void* workspace, size_t ws_bytes, void* stream, size_t scratch_cap,
                       bool check_only = false, int32_t mask_group = 0) {
  DVS_CHECK_ARG(q && k_new && v_new && k_pool && v_pool && page_table && kv_len && out,
                "attn_hybrid_block: NULL array argument");
  DVS_CHECK_ARG(S >= 1 && n_causal >= 0 && n_mask >= 0 && n_causal + n_mask >= 1,
                "attn_hybrid_block: need S >= 1 and n_causal + n_mask >= 1");
  DVS_CHECK_ARG(Hkv >= 1 && Hq >= Hkv && Hq % Hkv == 0, "attn_hybrid_block: Hq %% Hkv != 0");
  DVS_CHECK_ARG(max_pages >= 1 && num_pool_pages >= 1, "attn_hybrid_block: empty page table/pool");
  DVS_CHECK_ARG(softmax_scale > 0.f && isfinite(softmax_scale),
                "attn_hybrid_block: softmax_scale must be positive");
  DVS_CHECK_ARG(chunk_keys >= 0 && chunk_keys % KT == 0 && chunk_keys <= MAX_CHUNK_KEYS,
                "attn_hybrid_block: chunk_keys must be a multiple of 64 and <= %d", MAX_CHUNK_KEYS);
  DVS_CHECK_SUPPORTED(dtype == DVS_F32 || dtype == DVS_BF16, "attn_hybrid_block: dtype %d", dtype);
  DVS_CHECK_SUPPORTED(D == 64 || D == 96 || D == 128, "attn_hybrid_block: head_dim %d", D);
  DVS_CHECK_ARG(mask_group >= 0 && (mask_group == 0 || n_mask % mask_group == 0),
                "attn_hybrid_block: mask_group must divide n_mask");
  const int n_groups = mask_group > 0 ? n_mask / mask_group : 1;
  DVS_CHECK_ARG(n_groups <= 1 || n_groups <= n_causal,
                "attn_hybrid_block: %d mask groups need as many causal rows", n_groups);
  const int R = n_causal + n_mask;
  AttnPlan pl = plan_attn(S, R, Hq, Hkv, D, max_pages, chunk_keys, dtype);
  if (scratch_cap > 0 && dtype == DVS_BF16 && pl.bytes > scratch_cap) {
    set_error("attn_hybrid_block_noalloc: this shape needs %zu bytes of scratch, the library's "
              "array holds %zu (use attn_hybrid_block with a workspace)", pl.bytes, scratch_cap);
    return DVS_EWORKSPACE;
  }
  if (check_only) return DVS_OK;
  if (dtype == DVS_BF16 && (!workspace || ws_bytes < pl.bytes)) {
    set_error("attn_hybrid_block: workspace needs %zu bytes, got %zu", pl.bytes, ws_bytes);
    return DVS_EWORKSPACE;
  }
  AttnParams prm{};
  prm.q = q; prm.k_new = k_new; prm.v_new = v_new; prm.k_pool = k_pool; prm.v_pool = v_pool;
  prm.page_table = page_table; prm.kv_len = kv_len; prm.out = out; prm.err = err_word;
  prm.S = S; prm.n_causal = n_causal; prm.n_mask = n_mask; prm.R = R; prm.Hq = Hq;
  prm.Hkv = Hkv; prm.G = Hq / Hkv; prm.max_pages = max_pages; prm.pool_pages = num_pool_pages;
  prm.rows_total = pl.rows_total; prm.n_row_tiles = pl.n_row_tiles; prm.n_items = pl.n_items;
  prm.balanced = pl.balanced; prm.chunk_tiles = pl.chunk_tiles;
  prm.n_chunks_max = pl.n_chunks_max; prm.share_min = pl.share_min; prm.max_segs = pl.max_segs;
  prm.group = n_groups > 1 ? mask_group : 0;
  prm.n_groups = n_groups;
  prm.scale = softmax_scale;
  prm.scale_log2 = softmax_scale * 1.4426950408889634f;
  hipStream_t st = (hipStream_t)stream;
  if (dtype == DVS_BF16) {
    char* ws = (char*)workspace;
    prm.counters = (int32_t*)(ws + pl.off_counters);
    prm.part_ml = (float*)(ws + pl.off_ml);
    prm.part_o = (float*)(ws + pl.off_o);
    DVS_CHECK_SUPPORTED((long long)pl.grid < (1LL << 31), "attn_hybrid_block: grid too large");
    if (scratch_cap > 0) {
      // the array keeps the previous call's contents: clear the counters
      const int nw = (int)((pl.off_ml - pl.off_counters) / sizeof(int32_t));
      hipLaunchKernelGGL(attn_zero_kernel, dim3((nw + 255) / 256), dim3(256), 0, st, prm.counters, nw);
    }
    if (D == 128) launch_bf16<128>(pl, prm, st);
    else if (D == 96) launch_bf16<96>(pl, prm, st);
    else launch_bf16<64>(pl, prm, st);
  } else {
    const long long grid = (long long)S * R * Hq;
    DVS_CHECK_SUPPORTED(grid < (1LL << 31), "attn_hybrid_block: grid too large");
    if (D == 128) hipLaunchKernelGGL(attn_f32_kernel<128>, dim3(grid), dim3(256), 0, st, prm);
    else if (D == 96) hipLaunchKernelGGL(attn_f32_kernel<96>, dim3(grid), dim3(256), 0, st, prm);
    else hipLaunchKernelGGL(attn_f32_kernel<64>, dim3(grid), dim3(256), 0, st, prm);
  }
  return launch_status("attn_hybrid_block");
}

extern "C" int attn_hybrid_block(const void* q, const void* k_new, const void* v_new,
                                 void* k_pool, void* v_pool, const int32_t* page_table,
                                 const int32_t* kv_len, int32_t S, int32_t n_causal,
                                 int32_t n_mask, int32_t Hq, int32_t Hkv, int32_t D,
                                 int32_t max_pages, int32_t num_pool_pages, float softmax_scale,
                                 int32_t dtype, int32_t chunk_keys, void* out,
                                 int32_t* err_word, void* workspace, size_t ws_bytes,
                                 void* stream) {
  clear_error();
  return attn_launch(q, k_new, v_new, k_pool, v_pool, page_table, kv_len, S, n_causal, n_mask,
                     Hq, Hkv, D, max_pages, num_pool_pages, softmax_scale, dtype, chunk_keys, out,
                     err_word, workspace, ws_bytes, stream, 0);
}

extern "C" int attn_hybrid_block_grouped(const void* q, const void* k_new, const void* v_new,
                                         void* k_pool, void* v_pool, const int32_t* page_table,
                                         const int32_t* kv_len, int32_t S, int32_t n_causal,
                                         int32_t n_mask, int32_t mask_group, int32_t Hq,
                                         int32_t Hkv, int32_t D, int32_t max_pages,
                                         int32_t num_pool_pages, float softmax_scale,
                                         int32_t dtype, int32_t chunk_keys, void* out,
                                         int32_t* err_word, void* workspace, size_t ws_bytes,
                                         void* stream) {
  clear_error();
  return attn_launch(q, k_new, v_new, k_pool, v_pool, page_table, kv_len, S, n_causal, n_mask,
                     Hq, Hkv, D, max_pages, num_pool_pages, softmax_scale, dtype, chunk_keys, out,
                     err_word, workspace, ws_bytes, stream, 0, false, mask_group);
}

// ---------------------------------------------------------------------------
// attn_hybrid_block_noalloc: the same call with the library's own scratch
// array as its workspace, for callers that cannot allocate device memory.
// `scratch` is a device-side symbol: host code never passes its name to a
// kernel; it uses the address hipGetSymbolAddress gives for the current
// device, looked up once per device on that device's first call.
// ---------------------------------------------------------------------------
static __device__ __align__(256) char scratch[DVS_ATTN_SCRATCH_BYTES];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};
}  // namespace

static int scratch_for_current_device(void** out_ptr) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
    set_error("attn_hybrid_block_noalloc: no current device (or device id >= %d)", kMaxDevices);
    return DVS_EHIP;
  }
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !ptr) {
      set_error("attn_hybrid_block_noalloc: hipGetSymbolAddress failed on device %d: %s", dev,
                hipGetErrorString(e));
      return DVS_EHIP;
    }
    g_scratch_ptr[dev] = ptr;
  }
  *out_ptr = g_scratch_ptr[dev];
  return DVS_OK;
}

extern "C" int attn_hybrid_block_noalloc(const void* q, const void* k_new, const void* v_new,
                                         void* k_pool, void* v_pool, const int32_t* page_table,
                                         const int32_t* kv_len, int32_t S, int32_t n_causal,
                                         int32_t n_mask, int32_t Hq, int32_t Hkv, int32_t D,
                                         int32_t max_pages, int32_t num_pool_pages,
                                         float softmax_scale, int32_t dtype, int32_t chunk_keys,
                                         void* out, int32_t* err_word, void* stream) {
  clear_error();
  // every argument and the scratch size are checked before anything is
  // launched or the device array is looked up
  int rc = attn_launch(q, k_new, v_new, k_pool, v_pool, page_table, kv_len, S, n_causal, n_mask,
                       Hq, Hkv, D, max_pages, num_pool_pages, softmax_scale, dtype, chunk_keys,
                       out, err_word, nullptr, 0, stream, DVS_ATTN_SCRATCH_BYTES, true);
  if (rc != DVS_OK) return rc;
  void* ws = nullptr;
  if (dtype == DVS_BF16) {
    rc = scratch_for_current_device(&ws);
    if (rc != DVS_OK) return rc;
  }
  return attn_launch(q, k_new, v_new, k_pool, v_pool, page_table, kv_len, S, n_causal, n_mask,
                     Hq, Hkv, D, max_pages, num_pool_pages, softmax_scale, dtype, chunk_keys, out,
                     err_word, ws, DVS_ATTN_SCRATCH_BYTES, stream, DVS_ATTN_SCRATCH_BYTES);
}
