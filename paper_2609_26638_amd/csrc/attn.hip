// attn_hybrid_block: append the window's K/V to the paged cache and attend
// with the block-causal (hybrid) mask.
//
// Visibility rule (Preliminaries "Block Diffusion"; Method "Joint
// AR-Diffusion Training"; appendix items Draft forward / Verify forward):
// window row r of a sequence with committed length L sits at position L + r;
// a causal row (r < n_causal) sees keys <= L + r, a mask row sees every key
// up to L + R - 1.  Keys below L are visible to every row, so only the tile
// that reaches the window needs a mask.
//
// bf16 path (MFMA, gfx950)
//   One workgroup per (key chunk, row tile, sequence, KV head).  All G query
//   heads of the KV head and all R window rows (R*G "query rows", up to 256
//   per workgroup) share each K/V tile staged in LDS, so the cache is read
//   from HBM once per KV head.  Per 64-key tile:
//     S^T[key, row] = K Q^T   v_mfma_f32_32x32x16_bf16, A = K from LDS,
//                             B = Q held in registers for the whole chunk;
//     the C layout puts one query row per lane (16 keys per 32-key group), so
//     the row max / sum of the online softmax are in-lane plus one exchange
//     with lane^32, and the rescale of O touches only the lane's own row;
//     O^T[d, row] += V^T P^T  A = V^T read from a transposed, XOR-swizzled
//                             LDS copy of V, B = P (bf16) straight from the
//                             score registers (same key permutation).
//   Chunks begin at absolute multiples of chunk_keys.  A sequence spanning
//   several chunks writes fp32 partials (m, l, O); the last workgroup of the
//   (sequence, KV head, row tile) to finish merges them in chunk order, so
//   results are deterministic and a row's arithmetic does not depend on the
//   other rows of the window.
//   The window's own K/V (positions [L, L+R)) are read from k_new / v_new and
//   written to the pool by the workgroup whose chunk covers them.
//
// fp32 path: a plain per-(sequence, row, head) workgroup, fp32 throughout.
#include <math.h>

#include "dvs_common.h"

namespace dvs {

constexpr int KT = 64;  // keys per tile

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
  int chunk_keys, n_chunks_max, rows_total, n_row_tiles;
  float scale_log2;
  float scale;
};

// ---------------------------------------------------------------------------
// LDS layouts of one 64-key tile (bf16)
//
// K: 64 rows of D*2 bytes (row = key), 16-byte chunks XOR-swizzled by kswz(row)
//    so the A-operand reads (8 rows per LDS phase) hit distinct banks.
// V: KT/16 pages x D rows x 32 bytes (row = head-dim element, 16 keys): the
//    same layout as a head-dim-major V page of the pool, so cache tiles are a
//    straight copy; the two 16-byte halves are swapped on every other group of
//    4 rows, again for conflict-free operand reads.
//
// Key permutation: the QK^T A-operand lane m (m = 0..31 within a 32-key group)
// is fed key kperm(m) (bits 2 and 3 of m swapped).  With the 32x32 MFMA C
// layout, lane (row, hh) then holds in registers 0..7 the scores of keys
// 8*hh + 0..7 and in registers 8..15 those of keys 16 + 8*hh + 0..7, which is
// exactly the B-operand layout of a 16-key k-step of the PV product, and the
// matching A-operand (V^T) slice is one 16-byte chunk of a V page row.
// ---------------------------------------------------------------------------
__device__ __forceinline__ int kperm(int m) {
  return (m & 0x13) | ((m & 4) << 1) | ((m & 8) >> 1);
}

template <int CPR>
__device__ __forceinline__ int kswz(int row) {
  return (CPR % 8 == 0) ? ((row & 3) | ((row >> 1) & 4)) : (row & 3);
}

__device__ __forceinline__ int vswz(int d) { return (d >> 2) & 1; }

// s_waitcnt vmcnt(n) with the other counters left alone (gfx9 encoding).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

constexpr int MAX_CHUNK_KEYS = 16384;
constexpr float RESCALE_LOG2 = 8.f;
constexpr int NSTAGE = 3;

template <int D, int NW, int RG>
__global__ void __launch_bounds__(NW * 64, 1) attn_bf16_kernel(AttnParams p) {
  constexpr int NT = NW * 64;
  constexpr int CPR = D / 8;              // 16-byte chunks per K row
  constexpr int KROWB = D * 2;
  constexpr int KTILE_B = KT * KROWB;
  constexpr int VTILE_B = KT * D * 2;
  constexpr int STAGE_B = KTILE_B + VTILE_B;
  constexpr int K_INS = KTILE_B / (NT * 16);   // DMA instructions per lane per tile
  constexpr int V_INS = VTILE_B / (NT * 16);
  constexpr int NPL = K_INS + V_INS;
  constexpr int KS = D / 16;
  constexpr int DG = D / 32;
  constexpr int KG = KT / 32;
  constexpr int RPW = NW * RG * 32;
  static_assert(KTILE_B % (NT * 16) == 0 && VTILE_B % (NT * 16) == 0, "tile / wave mismatch");

  __shared__ __attribute__((aligned(1024))) char smem[NSTAGE * STAGE_B];
  __shared__ int s_pages[MAX_CHUNK_KEYS / 16 + 1];
  __shared__ int s_flag;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = tid >> 6;
  const int hh = lane >> 5;
  const int l32 = lane & 31;

  int idx = blockIdx.x;
  const int kvh = idx % p.Hkv;
  idx /= p.Hkv;
  const int s = idx % p.S;
  idx /= p.S;
  const int rt = idx % p.n_row_tiles;
  const int c = idx / p.n_row_tiles;

  const int L = p.kv_len[s];
  const int R = p.R;
  const int T = L + R;
  if (L < 0 || T > p.max_pages * 16) {
    if (c == 0 && rt == 0 && kvh == 0 && tid == 0) set_err(p.err, DVS_ERR_MAX_PAGES);
    return;
  }
  const int C = p.chunk_keys;
  const int n_chunks = (T + C - 1) / C;
  if (c >= n_chunks) return;
  const int k0 = c * C;
  const int k1 = min(k0 + C, T);
  const int pg0 = k0 >> 4;

  const __bf16* __restrict__ q = (const __bf16*)p.q;
  const char* __restrict__ knb = (const char*)p.k_new;
  const char* __restrict__ vnb = (const char*)p.v_new;
  char* __restrict__ kpb = (char*)p.k_pool;
  char* __restrict__ vpb = (char*)p.v_pool;
  const int32_t* __restrict__ pt = p.page_table + (size_t)s * p.max_pages;

  // ---- page ids of this chunk (invalid ids are replaced by page 0 and reported)
  if (tid == 0) s_flag = 0;
  __syncthreads();
  for (int i = tid; i < ((k1 + 15) >> 4) - pg0; i += NT) {
    int pg = pt[pg0 + i];
    if (pg < 0 || pg >= p.pool_pages) {
      pg = 0;
      s_flag = 1;
    }
    s_pages[i] = pg;
  }
  __syncthreads();
  if (tid == 0 && s_flag) set_err(p.err, DVS_ERR_BAD_PAGE);

  // ---- query rows of this lane: Q fragments (B operand) and visibility limit
  bf16x8 qf[RG][KS];
  int hi[RG], rowr[RG], rowh[RG];
  bool rvalid[RG];
#pragma unroll
  for (int rg = 0; rg < RG; ++rg) {
    const int n = rt * RPW + w * RG * 32 + rg * 32 + l32;
    rvalid[rg] = n < p.rows_total;
    const int r = n / p.G;
    const int h = kvh * p.G + (n - r * p.G);
    rowr[rg] = r;
    rowh[rg] = h;
    hi[rg] = !rvalid[rg] ? -1 : (r < p.n_causal ? L + r : T - 1);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      qf[rg][ks] = rvalid[rg]
          ? *(const bf16x8*)(q + (((size_t)s * R + r) * p.Hq + h) * D + ks * 16 + hh * 8)
          : bf16x8{};
  }

  f32x16 o[RG][DG];
  float m[RG], lsum[RG];
#pragma unroll
  for (int rg = 0; rg < RG; ++rg) {
    m[rg] = -INFINITY;
    lsum[rg] = 0.f;
#pragma unroll
    for (int dg = 0; dg < DG; ++dg) o[rg][dg] = f32x16{};
  }

  // ---- cache tiles (all 64 keys below L): direct global -> LDS copies
  auto issue_tile = [&](int t0, char* buf) {
#pragma unroll
    for (int j = 0; j < K_INS; ++j) {
      const int seg = w * K_INS + j;
      const int off = seg * 1024 + lane * 16;
      const int row = off / KROWB;
      const int cc = ((off % KROWB) >> 4) ^ kswz<CPR>(row);
      const int key = t0 + row;
      const int pg = s_pages[(key >> 4) - pg0];
      const char* src = kpb + ((((size_t)pg * p.Hkv + kvh) * 16 + (key & 15)) * D) * 2 + cc * 16;
      __builtin_amdgcn_global_load_lds((const void*)src,
                                       (__attribute__((address_space(3))) void*)(buf + seg * 1024),
                                       16, 0, 0);
    }
#pragma unroll
    for (int j = 0; j < V_INS; ++j) {
      const int seg = w * V_INS + j;
      const int off = seg * 1024 + lane * 16;
      const int tp = off / (D * 32);
      const int d = (off % (D * 32)) >> 5;
      const int hc = ((off >> 4) & 1) ^ vswz(d);
      const int pg = s_pages[(t0 >> 4) + tp - pg0];
      const char* src = vpb + ((((size_t)pg * p.Hkv + kvh) * D + d) * 16) * 2 + hc * 16;
      __builtin_amdgcn_global_load_lds((const void*)src,
                                       (__attribute__((address_space(3))) void*)(buf + KTILE_B + seg * 1024),
                                       16, 0, 0);
    }
  };

  // ---- one tile of compute from LDS
  auto compute_tile = [&](const char* kb, int t0, bool masked) {
    const char* vb = kb + KTILE_B;
    f32x16 sacc[KG][RG];
#pragma unroll
    for (int kg = 0; kg < KG; ++kg)
#pragma unroll
      for (int rg = 0; rg < RG; ++rg) sacc[kg][rg] = f32x16{};
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
#pragma unroll
      for (int kg = 0; kg < KG; ++kg) {
        const int row = kg * 32 + kperm(l32);
        const bf16x8 a = *(const bf16x8*)(kb + row * KROWB + (((2 * ks + hh) ^ kswz<CPR>(row)) << 4));
#pragma unroll
        for (int rg = 0; rg < RG; ++rg)
          sacc[kg][rg] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[rg][ks], sacc[kg][rg], 0, 0, 0);
      }
    }
    if (masked) {
#pragma unroll
      for (int kg = 0; kg < KG; ++kg)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int key = t0 + kg * 32 + 16 * (i >> 3) + 8 * hh + (i & 7);
#pragma unroll
          for (int rg = 0; rg < RG; ++rg)
            if (key > hi[rg]) sacc[kg][rg][i] = -INFINITY;
        }
    }
    bf16x8 pf[RG][KT / 16];
#pragma unroll
    for (int rg = 0; rg < RG; ++rg) {
      float tmax = -INFINITY;
#pragma unroll
      for (int kg = 0; kg < KG; ++kg)
#pragma unroll
        for (int i = 0; i < 16; ++i) tmax = fmaxf(tmax, sacc[kg][rg][i]);
      tmax = fmaxf(tmax, __shfl_xor(tmax, 32));
      // The row's reference maximum m only moves when the tile maximum exceeds
      // it by more than 2^RESCALE_LOG2 (weights stay <= 2^RESCALE_LOG2, exact
      // after the final division by l); the wave skips the O rescale when no
      // row moved.  The decision is per row, so rows stay independent.
      const float cand = tmax * p.scale_log2;
      const bool move = cand > m[rg] + RESCALE_LOG2;
      if (__ballot(move)) {
        const float alpha = move ? __builtin_amdgcn_exp2f(m[rg] - cand) : 1.f;
        lsum[rg] *= alpha;
#pragma unroll
        for (int dg = 0; dg < DG; ++dg) o[rg][dg] *= alpha;
      }
      if (move) m[rg] = cand;
      const float msafe = (m[rg] == -INFINITY) ? 0.f : m[rg];
      float ps = 0.f;
#pragma unroll
      for (int t = 0; t < KT / 16; ++t) {
        uint32_t pk[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int i0 = 8 * (t & 1) + 2 * e;
          const float a0 = __builtin_amdgcn_exp2f(fmaf(sacc[t >> 1][rg][i0], p.scale_log2, -msafe));
          const float a1 = __builtin_amdgcn_exp2f(fmaf(sacc[t >> 1][rg][i0 + 1], p.scale_log2, -msafe));
          ps += a0 + a1;
          pk[e] = __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{a0, a1}, bf16x2));
        }
        pf[rg][t] = __builtin_bit_cast(bf16x8, u32x4{pk[0], pk[1], pk[2], pk[3]});
      }
      lsum[rg] += ps;
    }
#pragma unroll
    for (int t = 0; t < KT / 16; ++t) {
#pragma unroll
      for (int dg = 0; dg < DG; ++dg) {
        const int d = dg * 32 + l32;
        const bf16x8 a = *(const bf16x8*)(vb + (t * D + d) * 32 + ((hh ^ vswz(d)) << 4));
#pragma unroll
        for (int rg = 0; rg < RG; ++rg)
          o[rg][dg] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pf[rg][t], o[rg][dg], 0, 0, 0);
      }
    }
  };

  // main (pure cache) tiles: [k0, kmain)
  const int lfloor = (L / KT) * KT;
  const int kmain = min(k1, max(k0, lfloor));
  const int n_main = (kmain - k0) / KT;

  // prologue: the Q loads were issued first; start NSTAGE-1 tiles, then wait
  // only for Q (loads complete in issue order).
#pragma unroll
  for (int i = 0; i < NSTAGE - 1; ++i)
    if (i < n_main) issue_tile(k0 + i * KT, smem + i * STAGE_B);
  // (waiting for "at most 63 outstanding" is still enough: the Q loads are older)
  if (n_main >= 2) wait_vmcnt<(2 * NPL < 63 ? 2 * NPL : 63)>();
  else if (n_main == 1) wait_vmcnt<NPL>();
  else wait_vmcnt<0>();

  for (int i = 0; i < n_main; ++i) {
    if (i + 1 < n_main) wait_vmcnt<NPL>();   // tile i landed (this wave's part)
    else wait_vmcnt<0>();
    __builtin_amdgcn_s_barrier();             // ... every wave's part; tile i-1 consumed
    if (i + NSTAGE - 1 < n_main)
      issue_tile(k0 + (i + NSTAGE - 1) * KT, smem + ((i + NSTAGE - 1) % NSTAGE) * STAGE_B);
    compute_tile(smem + (i % NSTAGE) * STAGE_B, k0 + i * KT, false);
  }

  // ---- tiles that reach the window or run past T: staged through registers.
  // Keys < L come from the pool, keys in [L, T) from k_new / v_new (and are
  // appended to the pool by row tile 0), keys >= T are zero.
  bool bad_new = false;
  for (int t0 = kmain; t0 < k1; t0 += KT) {
    __syncthreads();
    char* kb = smem;
    char* vb = smem + KTILE_B;
    for (int ci = tid; ci < KT * CPR; ci += NT) {
      const int kk = ci / CPR;
      const int cc = ci - kk * CPR;
      const int key = t0 + kk;
      u32x4 val = u32x4{0, 0, 0, 0};
      if (key < L) {
        const int pg = s_pages[(key >> 4) - pg0];
        val = *(const u32x4*)(kpb + ((((size_t)pg * p.Hkv + kvh) * 16 + (key & 15)) * D) * 2 + cc * 16);
      } else if (key < T) {
        val = *(const u32x4*)(knb + ((((size_t)s * R + (key - L)) * p.Hkv + kvh) * D) * 2 + cc * 16);
        if (rt == 0) {
          const int pg = s_pages[(key >> 4) - pg0];
          *(u32x4*)(kpb + ((((size_t)pg * p.Hkv + kvh) * 16 + (key & 15)) * D) * 2 + cc * 16) = val;
        }
      }
      *(u32x4*)(kb + kk * KROWB + ((cc ^ kswz<CPR>(kk)) << 4)) = val;
    }
    for (int ci = tid; ci < KT / 16 * D * 2; ci += NT) {
      const int tp = ci / (D * 2);
      const int d = (ci >> 1) % D;
      const int hc = ci & 1;
      const int kbase = t0 + tp * 16 + hc * 8;
      u32x4 val = u32x4{0, 0, 0, 0};
      if (kbase + 8 <= L) {
        const int pg = s_pages[(kbase >> 4) - pg0];
        val = *(const u32x4*)(vpb + ((((size_t)pg * p.Hkv + kvh) * D + d) * 16) * 2 + hc * 16);
      } else {
        uint16_t e16[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int key = kbase + e;
          uint16_t x = 0;
          if (key < L) {
            const int pg = s_pages[(key >> 4) - pg0];
            x = ((const uint16_t*)vpb)[(((size_t)pg * p.Hkv + kvh) * D + d) * 16 + (key & 15)];
          } else if (key < T) {
            x = ((const uint16_t*)vnb)[(((size_t)s * R + (key - L)) * p.Hkv + kvh) * D + d];
            if (rt == 0) {
              const int pg = s_pages[(key >> 4) - pg0];
              ((uint16_t*)vpb)[(((size_t)pg * p.Hkv + kvh) * D + d) * 16 + (key & 15)] = x;
            }
          }
          e16[e] = x;
        }
        val = u32x4{e16[0] | ((uint32_t)e16[1] << 16), e16[2] | ((uint32_t)e16[3] << 16),
                    e16[4] | ((uint32_t)e16[5] << 16), e16[6] | ((uint32_t)e16[7] << 16)};
      }
      *(u32x4*)(vb + (tp * D + d) * 32 + ((hc ^ vswz(d)) << 4)) = val;
    }
    __syncthreads();
    compute_tile(kb, t0, true);
  }
  (void)bad_new;

#pragma unroll
  for (int rg = 0; rg < RG; ++rg) lsum[rg] += __shfl_xor(lsum[rg], 32);

  __bf16* __restrict__ out = (__bf16*)p.out;
  auto write_out = [&](int rg, const f32x16* ov, float inv) {
    if (!rvalid[rg]) return;
    __bf16* orow = out + (((size_t)s * R + rowr[rg]) * p.Hq + rowh[rg]) * D;
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

  if (n_chunks == 1) {
#pragma unroll
    for (int rg = 0; rg < RG; ++rg) write_out(rg, o[rg], lsum[rg] > 0.f ? 1.f / lsum[rg] : 0.f);
    return;
  }

  // ---- split key range: publish partials, the last workgroup merges in order
  constexpr int NREG = RG * DG * 16;
  const size_t item = ((size_t)s * p.Hkv + kvh) * p.n_row_tiles + rt;
  {
    f32x4* po = (f32x4*)(p.part_o + (item * p.n_chunks_max + c) * (size_t)(NT * NREG));
    f32x2* pml = (f32x2*)(p.part_ml + (item * p.n_chunks_max + c) * (size_t)(NT * RG * 2));
#pragma unroll
    for (int rg = 0; rg < RG; ++rg) {
      pml[rg * NT + tid] = f32x2{m[rg], lsum[rg]};
#pragma unroll
      for (int dg = 0; dg < DG; ++dg)
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
          const f32x16& v = o[rg][dg];
          po[((rg * DG + dg) * 4 + q4) * NT + tid] = f32x4{v[4 * q4], v[4 * q4 + 1], v[4 * q4 + 2], v[4 * q4 + 3]};
        }
    }
  }
  __threadfence();
  __syncthreads();
  if (tid == 0) s_flag = (atomicAdd(&p.counters[item], 1) == n_chunks - 1);
  __syncthreads();
  if (!s_flag) return;
  __threadfence();

  const f32x4* pob = (const f32x4*)(p.part_o + item * p.n_chunks_max * (size_t)(NT * NREG));
  const f32x2* pmlb = (const f32x2*)(p.part_ml + item * p.n_chunks_max * (size_t)(NT * RG * 2));
#pragma unroll
  for (int rg = 0; rg < RG; ++rg) {
    float M = -INFINITY;
    for (int cc = 0; cc < n_chunks; ++cc) M = fmaxf(M, pmlb[(size_t)cc * NT * RG + rg * NT + tid].x);
    const float Ms = (M == -INFINITY) ? 0.f : M;
    f32x16 acc[DG];
#pragma unroll
    for (int dg = 0; dg < DG; ++dg) acc[dg] = f32x16{};
    float lt = 0.f;
    for (int cc = 0; cc < n_chunks; ++cc) {
      const f32x2 ml = pmlb[(size_t)cc * NT * RG + rg * NT + tid];
      const float wgt = __builtin_amdgcn_exp2f(ml.x - Ms);
      lt += wgt * ml.y;
      const f32x4* src = pob + (size_t)cc * NT * NREG / 4;
#pragma unroll
      for (int dg = 0; dg < DG; ++dg)
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
          const f32x4 v = src[((rg * DG + dg) * 4 + q4) * NT + tid];
          acc[dg][4 * q4 + 0] += wgt * v.x;
          acc[dg][4 * q4 + 1] += wgt * v.y;
          acc[dg][4 * q4 + 2] += wgt * v.z;
          acc[dg][4 * q4 + 3] += wgt * v.w;
        }
    }
    write_out(rg, acc, lt > 0.f ? 1.f / lt : 0.f);
  }
  if (tid == 0) p.counters[item] = 0;
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
  const int hi = r < p.n_causal ? L + r : T - 1;
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
  for (int t0 = 0; t0 <= hi; t0 += 256) {
    const int k = t0 + tid;
    float sc = -INFINITY;
    if (k <= hi) {
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
      const int nk = min(256, hi + 1 - t0);
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
struct AttnPlan {
  int nw, rg, rows_total, rows_per_wg, n_row_tiles, chunk, n_chunks_max;
  size_t off_counters, off_ml, off_o, bytes;
};

static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

static AttnPlan plan_attn(int S, int R, int Hq, int Hkv, int D, int max_pages, int chunk_keys,
                          int dtype) {
  AttnPlan pl{};
  const int G = Hq / Hkv;
  pl.rows_total = R * G;
  if (dtype == DVS_BF16) {
    const int groups = (pl.rows_total + 31) / 32;  // 32-row MFMA groups
    if (groups >= 8) {
      pl.nw = 4; pl.rg = 2;
    } else if (groups >= 4) {
      pl.nw = 2; pl.rg = 2;
    } else if (groups >= 2) {
      pl.nw = 1; pl.rg = 2;
    } else {
      pl.nw = 1; pl.rg = 1;
    }
  } else {
    pl.nw = 4; pl.rg = 1;
  }
  pl.rows_per_wg = pl.nw * pl.rg * 32;
  pl.n_row_tiles = (pl.rows_total + pl.rows_per_wg - 1) / pl.rows_per_wg;
  const long long max_keys = (long long)max_pages * DVS_PAGE_SIZE;
  int C = chunk_keys;
  if (C <= 0) {
    const long long items = (long long)S * Hkv * pl.n_row_tiles;
    long long want = (max_keys * items + 1535) / 1536;
    want = (want + KT - 1) / KT * KT;
    if (want < 256) want = 256;
    if (want > MAX_CHUNK_KEYS) want = MAX_CHUNK_KEYS;
    C = (int)want;
  }
  pl.chunk = C;
  pl.n_chunks_max = (int)((max_keys + C - 1) / C);
  const int NT = pl.nw * 64;
  const size_t items = (size_t)S * Hkv * pl.n_row_tiles;
  if (dtype == DVS_BF16) {
    const size_t nreg = (size_t)pl.rg * (D / 32) * 16;
    pl.off_counters = 0;
    pl.off_ml = align256(items * sizeof(int32_t));
    pl.off_o = pl.off_ml + align256(items * pl.n_chunks_max * (size_t)NT * pl.rg * 2 * sizeof(float));
    pl.bytes = pl.off_o + align256(items * pl.n_chunks_max * (size_t)NT * nreg * sizeof(float));
  } else {
    pl.bytes = 256;
  }
  return pl;
}

template <int D>
static void launch_bf16(const AttnPlan& pl, const AttnParams& prm, int grid, hipStream_t st) {
  if (pl.nw == 4)
    hipLaunchKernelGGL((attn_bf16_kernel<D, 4, 2>), dim3(grid), dim3(256), 0, st, prm);
  else if (pl.nw == 2)
    hipLaunchKernelGGL((attn_bf16_kernel<D, 2, 2>), dim3(grid), dim3(128), 0, st, prm);
  else if (pl.rg == 2)
    hipLaunchKernelGGL((attn_bf16_kernel<D, 1, 2>), dim3(grid), dim3(64), 0, st, prm);
  else
    hipLaunchKernelGGL((attn_bf16_kernel<D, 1, 1>), dim3(grid), dim3(64), 0, st, prm);
}

}  // namespace dvs

using namespace dvs;

extern "C" size_t dvs_attn_workspace_bytes(int32_t S, int32_t n_causal, int32_t n_mask,
                                           int32_t Hq, int32_t Hkv, int32_t D, int32_t max_pages,
                                           int32_t chunk_keys, int32_t dtype) {
  if (S < 1 || n_causal < 0 || n_mask < 0 || n_causal + n_mask < 1 || Hkv < 1 || Hq < Hkv ||
      Hq % Hkv != 0 || max_pages < 1)
    return 0;
  return plan_attn(S, n_causal + n_mask, Hq, Hkv, D, max_pages, chunk_keys, dtype).bytes;
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
  const int R = n_causal + n_mask;
  AttnPlan pl = plan_attn(S, R, Hq, Hkv, D, max_pages, chunk_keys, dtype);
  if (dtype == DVS_BF16 && (!workspace || ws_bytes < pl.bytes)) {
    set_error("attn_hybrid_block: workspace needs %zu bytes, got %zu", pl.bytes, ws_bytes);
    return DVS_EWORKSPACE;
  }
  AttnParams prm{};
  prm.q = q; prm.k_new = k_new; prm.v_new = v_new; prm.k_pool = k_pool; prm.v_pool = v_pool;
  prm.page_table = page_table; prm.kv_len = kv_len; prm.out = out; prm.err = err_word;
  prm.S = S; prm.n_causal = n_causal; prm.n_mask = n_mask; prm.R = R; prm.Hq = Hq;
  prm.Hkv = Hkv; prm.G = Hq / Hkv; prm.max_pages = max_pages; prm.pool_pages = num_pool_pages;
  prm.chunk_keys = pl.chunk; prm.n_chunks_max = pl.n_chunks_max; prm.rows_total = pl.rows_total;
  prm.n_row_tiles = pl.n_row_tiles;
  prm.scale = softmax_scale;
  prm.scale_log2 = softmax_scale * 1.4426950408889634f;
  hipStream_t st = (hipStream_t)stream;
  if (dtype == DVS_BF16) {
    char* ws = (char*)workspace;
    prm.counters = (int32_t*)(ws + pl.off_counters);
    prm.part_ml = (float*)(ws + pl.off_ml);
    prm.part_o = (float*)(ws + pl.off_o);
    const long long grid = (long long)pl.n_chunks_max * pl.n_row_tiles * S * Hkv;
    DVS_CHECK_SUPPORTED(grid < (1LL << 31), "attn_hybrid_block: grid too large");
    if (D == 128) launch_bf16<128>(pl, prm, (int)grid, st);
    else if (D == 96) launch_bf16<96>(pl, prm, (int)grid, st);
    else launch_bf16<64>(pl, prm, (int)grid, st);
  } else {
    const long long grid = (long long)S * R * Hq;
    DVS_CHECK_SUPPORTED(grid < (1LL << 31), "attn_hybrid_block: grid too large");
    if (D == 128) hipLaunchKernelGGL(attn_f32_kernel<128>, dim3(grid), dim3(256), 0, st, prm);
    else if (D == 96) hipLaunchKernelGGL(attn_f32_kernel<96>, dim3(grid), dim3(256), 0, st, prm);
    else hipLaunchKernelGGL(attn_f32_kernel<64>, dim3(grid), dim3(256), 0, st, prm);
  }
  return launch_status("attn_hybrid_block");
}
