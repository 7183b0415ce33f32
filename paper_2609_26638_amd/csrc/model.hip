// draft_verify_step: one fused self-speculative step of a decoder.
//
// Row inputs (Method "AR-to-Diffusion Conversion": the only architectural
// addition is the embedding of the mask token [M]):
//   causal rows r = 0..n_causal-1 : [x0, d_1, .., d_{n_causal-1}]
//   mask rows                     : [M] (embedding row `vocab`)
// then per layer: RMSNorm -> Q/K/V projections -> rotary positions at
// kv_len + r -> attn_hybrid_block (appends the window's K/V) -> O projection
// + residual -> [RMSNorm -> SwiGLU MLP + residual], final RMSNorm, LM head,
// and the hot-path tail argmax_accept -> kv_commit.
//
// Every matrix product is C[m, n] = sum_k A[m, k] * W[n, k] with weights laid
// out [out, in] so both MFMA operands are contiguous along k.  One wave owns
// 32 output columns for ALL rows: it streams its weight rows exactly once, in
// ascending k, and accumulates every 32-row group of A against them.  A row's
// result therefore never depends on how many rows the call carries, so an AR
// call (1 row) and a fused call (2B rows) produce bit-identical rows.
#include <algorithm>
#include <math.h>

#include "dvs_common.h"

namespace dvs {

// ---------------------------------------------------------------------------
// small element-wise kernels
// ---------------------------------------------------------------------------
template <typename T> __device__ __forceinline__ float to_f(T v);
template <> __device__ __forceinline__ float to_f<float>(float v) { return v; }
template <> __device__ __forceinline__ float to_f<__bf16>(__bf16 v) { return (float)v; }
template <typename T> __device__ __forceinline__ T from_f(float v);
template <> __device__ __forceinline__ float from_f<float>(float v) { return v; }
template <> __device__ __forceinline__ __bf16 from_f<__bf16>(float v) { return (__bf16)v; }

// x[m, :] = embed[token(m), :] (fp32 residual stream)
template <typename T>
__global__ void embed_rows_kernel(const T* __restrict__ embed, int H, int vocab, int R, int n_causal,
                                  const int32_t* __restrict__ boundary,
                                  const int32_t* __restrict__ draft, int draft_width,
                                  float* __restrict__ x) {
  const int mrow = blockIdx.x;
  const int s = mrow / R, r = mrow - s * R;
  int tok = vocab;  // [M]
  if (r < n_causal) tok = (r == 0) ? boundary[s] : draft[(size_t)s * draft_width + (r - 1)];
  if (tok < 0 || tok > vocab) tok = vocab;
  const T* e = embed + (size_t)tok * H;
  for (int i = threadIdx.x; i < H; i += blockDim.x) x[(size_t)mrow * H + i] = to_f(e[i]);
}

// out[m, :] = x[m, :] / sqrt(mean(x^2) + eps) * g   (one workgroup per row)
template <typename T>
__global__ void __launch_bounds__(256) rmsnorm_kernel(const float* __restrict__ x, const T* __restrict__ g,
                                                      int H, float eps, T* __restrict__ out) {
  __shared__ float red[4];
  const int mrow = blockIdx.x;
  const float* xr = x + (size_t)mrow * H;
  float ss = 0.f;
  for (int i = threadIdx.x; i < H; i += 256) ss = fmaf(xr[i], xr[i], ss);
  for (int off = 32; off > 0; off >>= 1) ss += __shfl_xor(ss, off);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
  __syncthreads();
  const float tot = (red[0] + red[1]) + (red[2] + red[3]);
  const float inv = 1.0f / sqrtf(tot / (float)H + eps);
  for (int i = threadIdx.x; i < H; i += 256)
    out[(size_t)mrow * H + i] = from_f<T>(xr[i] * inv * to_f(g[i]));
}

// rotate-half rotary embedding, in place, position kv_len[s] + r; angles in
// double precision (positions reach thousands of radians).
template <typename T>
__global__ void rope_kernel(T* __restrict__ x, int M, int R, int nh, int D, double log2_theta,
                            const int32_t* __restrict__ kv_len) {
  const int half = D / 2;
  const long long idx = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (long long)M * nh * half) return;
  const int i = (int)(idx % half);
  const long long mh = idx / half;
  const int mrow = (int)(mh / nh);
  const int s = mrow / R, r = mrow - s * R;
  const double pos = (double)(kv_len[s] + r);
  const double inv = exp2(-2.0 * i / D * log2_theta);
  double sn, cs;
  sincos(pos * inv, &sn, &cs);
  T* v = x + mh * D;
  const float x1 = to_f(v[i]), x2 = to_f(v[i + half]);
  v[i] = from_f<T>((float)(x1 * cs - x2 * sn));
  v[i + half] = from_f<T>((float)(x1 * sn + x2 * cs));
}

// Prefill rows: row r < P of sequence s takes embed[tokens[s, r]] when that
// id is >= 0 and otherwise the given vector x_prefix[s, r, :] (e.g. a vision
// encoder output); rows r >= P are mask tokens.
template <typename T>
__global__ void embed_prefill_kernel(const T* __restrict__ embed, int H, int vocab, int R, int P,
                                     const int32_t* __restrict__ tokens,
                                     const float* __restrict__ x_prefix, float* __restrict__ x) {
  const int mrow = blockIdx.x;
  const int s = mrow / R, r = mrow - s * R;
  int tok = vocab;
  const float* src = nullptr;
  if (r < P) {
    tok = tokens ? tokens[(size_t)s * P + r] : -1;
    if (tok < 0 || tok >= vocab) {
      tok = -1;
      if (x_prefix) src = x_prefix + ((size_t)s * P + r) * H;
      else tok = vocab;
    }
  }
  for (int i = threadIdx.x; i < H; i += blockDim.x)
    x[(size_t)mrow * H + i] = src ? src[i] : to_f(embed[(size_t)tok * H + i]);
}

// dst[s*n + j, :] = src[s*R + r0 + j, :]  (rows whose logits are needed)
template <typename T>
__global__ void gather_rows_kernel(const T* __restrict__ src, int H, int R, int r0, int n,
                                   T* __restrict__ dst) {
  const int row = blockIdx.x;
  const int s = row / n, j = row - s * n;
  const T* a = src + ((size_t)s * R + r0 + j) * H;
  for (int i = threadIdx.x; i < H; i += blockDim.x) dst[(size_t)row * H + i] = a[i];
}

// After a prefill of P rows: kv_len = P, the top-1 of row P-1 is the first
// committed token and boundary, the mask rows' top-1 tokens the first draft.
// am holds per sequence the top-1 of rows P-1 .. P+n_mask-1.
__global__ void prefill_commit_kernel(int S, int P, int n_mask, const int32_t* __restrict__ am,
                                      int32_t* kv_len, int32_t* boundary, int32_t* draft,
                                      int draft_width, int32_t* out_tokens, int32_t* out_count,
                                      int max_new, int eos_id, int32_t* finished) {
  const int s = blockIdx.x * blockDim.x + threadIdx.x;
  if (s >= S) return;
  const int n = n_mask + 1;
  const int first = am[(size_t)s * n];
  kv_len[s] = P;
  boundary[s] = first;
  for (int j = 0; j < draft_width && j < n_mask; ++j) draft[(size_t)s * draft_width + j] = am[(size_t)s * n + 1 + j];
  const int c = out_count[s];
  if (c < max_new) {
    out_tokens[(size_t)s * max_new + c] = first;
    out_count[s] = c + 1;
  }
  finished[s] = ((eos_id >= 0 && first == eos_id) || c + 1 >= max_new) ? 1 : 0;
}

template <typename T>
__global__ void silu_mul_kernel(const T* __restrict__ gate, const T* __restrict__ up, long long n,
                                T* __restrict__ out) {
  const long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const float g = to_f(gate[i]);
  out[i] = from_f<T>(g / (1.0f + expf(-g)) * to_f(up[i]));
}

// ---------------------------------------------------------------------------
// GEMM: C[m, n] (=, or += into an fp32 residual) sum_k A[m, k] W[n, k]
// One wave per 32 output columns; it walks k in ascending order, loading each
// weight fragment once and applying it to every 32-row group of A (up to
// MG_MAX groups, the rest in further passes).
// ---------------------------------------------------------------------------
constexpr int MG_MAX = 8;   // 32-row groups per pass (256 rows)

// bf16: v_mfma_f32_32x32x16_bf16, A lane = row, W lane = column, 8 k each
__global__ void __launch_bounds__(256) gemm_bf16_kernel(const __bf16* __restrict__ A,
                                                        const __bf16* __restrict__ W, int M, int N,
                                                        int K, void* __restrict__ C, int c_f32,
                                                        int accumulate) {
  float* __restrict__ Cf = c_f32 ? (float*)C : nullptr;
  __bf16* __restrict__ Cb = c_f32 ? nullptr : (__bf16*)C;
  const int lane = threadIdx.x & 63;
  const int wave = blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6);
  const int n0 = wave * 32;
  if (n0 >= N) return;
  const int l32 = lane & 31, hh = lane >> 5;
  const int ncol = n0 + l32;
  const bool nvalid = ncol < N;
  const __bf16* wrow = W + (size_t)(nvalid ? ncol : n0) * K;
  for (int m0 = 0; m0 < M; m0 += MG_MAX * 32) {
    const int ng = min(MG_MAX, (M - m0 + 31) / 32);
    f32x16 acc[MG_MAX];
#pragma unroll
    for (int g = 0; g < MG_MAX; ++g) acc[g] = f32x16{};
    for (int k0 = 0; k0 < K; k0 += 16) {
      const bf16x8 b = nvalid ? *(const bf16x8*)(wrow + k0 + hh * 8) : bf16x8{};
#pragma unroll
      for (int g = 0; g < MG_MAX; ++g) {
        if (g < ng) {
          const int mrow = m0 + g * 32 + l32;
          const bf16x8 a = mrow < M ? *(const bf16x8*)(A + (size_t)mrow * K + k0 + hh * 8) : bf16x8{};
          acc[g] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[g], 0, 0, 0);
        }
      }
    }
    if (!nvalid) continue;
#pragma unroll
    for (int g = 0; g < MG_MAX; ++g) {
      if (g >= ng) break;
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int mrow = m0 + g * 32 + 8 * (i >> 2) + 4 * hh + (i & 3);
        if (mrow >= M) continue;
        const size_t o = (size_t)mrow * N + ncol;
        if (Cf) {
          if (accumulate) Cf[o] += acc[g][i];
          else Cf[o] = acc[g][i];
        } else {
          Cb[o] = (__bf16)acc[g][i];
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------
// bf16 GEMM for the decoder stack: C[m, n] (=, or += into the fp32 residual)
// sum_k A[m, k] W[n, k].  The weights are streamed once; the row count is
// small (8..256 window rows) or a long prefill.
//
// A workgroup owns 32 output columns and a K range; its 4 waves split that
// range in four, each accumulating all rows of a 256-row pass with
// v_mfma_f32_32x32x16_bf16 (A lane = row, W lane = column, 8 k each).  The
// four partial tiles are summed through LDS in wave order.  When the column
// count alone cannot fill the chip, the K range is further split over
// `ksplit` workgroups: each publishes its fp32 tile with write-through stores
// and the last one to finish (counter) sums the tiles in split order.
// Every output element is therefore reduced in an order fixed by (N, K)
// alone: a row's result does not depend on how many rows the call carries,
// which keeps a fused step's causal rows bit-identical to AR steps.
// ---------------------------------------------------------------------------
constexpr int GK_ROWS = 256;   // rows per pass
constexpr int GK_MAXSPLIT = 32;

// MG: 32-row groups per pass (1, 2, 4 or 8); KU: k-steps whose operands are
// loaded before their MFMAs are issued.
template <int MG>
__global__ void __launch_bounds__(256, 1) gemm_bf16_sk_kernel(
    const __bf16* __restrict__ A, const __bf16* __restrict__ W, int M, int N, int K, void* C,
    int c_f32, int accumulate, int ksplit, float* __restrict__ part, int32_t* __restrict__ counters) {
  constexpr int KU = MG >= 4 ? 2 : 4;
  constexpr int PR = MG * 32;   // rows per pass
  __shared__ float red[4][PR][33];
  __shared__ int s_last;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int l32 = lane & 31, hh = lane >> 5;
  const int NB = (N + 31) / 32;
  const int nb = blockIdx.x % NB;
  const int ks = blockIdx.x / NB;
  const int n0 = nb * 32;
  const int kc = K / ksplit, kw = kc / 4;
  const int kbeg = ks * kc + w * kw;
  const int ncol = n0 + l32;
  const bool nvalid = ncol < N;
  const __bf16* wrow = W + (size_t)(nvalid ? ncol : 0) * K;
  float* Cf = c_f32 ? (float*)C : nullptr;
  __bf16* Cb = c_f32 ? nullptr : (__bf16*)C;
  for (int m0 = 0; m0 < M; m0 += PR) {
    f32x16 acc[MG];
#pragma unroll
    for (int g = 0; g < MG; ++g) acc[g] = f32x16{};
    const __bf16* arow[MG];
    bool avalid[MG];
#pragma unroll
    for (int g = 0; g < MG; ++g) {
      const int mrow = m0 + g * 32 + l32;
      avalid[g] = mrow < M;
      arow[g] = A + (size_t)(avalid[g] ? mrow : 0) * K;
    }
    int k0 = kbeg;
    for (; k0 + 16 * KU <= kbeg + kw; k0 += 16 * KU) {
      bf16x8 bf[KU], af[KU][MG];
#pragma unroll
      for (int u = 0; u < KU; ++u) {
        bf[u] = nvalid ? *(const bf16x8*)(wrow + k0 + 16 * u + hh * 8) : bf16x8{};
#pragma unroll
        for (int g = 0; g < MG; ++g)
          af[u][g] = avalid[g] ? *(const bf16x8*)(arow[g] + k0 + 16 * u + hh * 8) : bf16x8{};
      }
#pragma unroll
      for (int u = 0; u < KU; ++u)
#pragma unroll
        for (int g = 0; g < MG; ++g) acc[g] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[u][g], bf[u], acc[g], 0, 0, 0);
    }
    for (; k0 < kbeg + kw; k0 += 16) {
      const bf16x8 b = nvalid ? *(const bf16x8*)(wrow + k0 + hh * 8) : bf16x8{};
#pragma unroll
      for (int g = 0; g < MG; ++g) {
        const bf16x8 a = avalid[g] ? *(const bf16x8*)(arow[g] + k0 + hh * 8) : bf16x8{};
        acc[g] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[g], 0, 0, 0);
      }
    }
    // C layout: lane (col l32, hh), register i holds row 8*(i>>2) + 4*hh + (i&3)
#pragma unroll
    for (int g = 0; g < MG; ++g)
#pragma unroll
      for (int i = 0; i < 16; ++i) red[w][g * 32 + 8 * (i >> 2) + 4 * hh + (i & 3)][l32] = acc[g][i];
    __syncthreads();
    // thread t sums column t&31 of rows (t>>5) + 8j over the four waves, in
    // order; a residual being accumulated into is read in one batch first
    const int col = tid & 31, n = n0 + col;
    float cur[PR / 8];
    if (ksplit == 1 && Cf && accumulate) {
#pragma unroll
      for (int j = 0; j < PR / 8; ++j) {
        const int mrow = m0 + (tid >> 5) + 8 * j;
        cur[j] = (mrow < M && n < N) ? Cf[(size_t)mrow * N + n] : 0.f;
      }
    }
#pragma unroll
    for (int j = 0; j < PR / 8; ++j) {
      const int r = (tid >> 5) + 8 * j;
      const float v = ((red[0][r][col] + red[1][r][col]) + red[2][r][col]) + red[3][r][col];
      const int mrow = m0 + r;
      if (mrow >= M || n >= N) continue;
      if (ksplit > 1) {
        __hip_atomic_store(part + ((size_t)ks * M + mrow) * N + n, v, __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
      } else {
        const size_t o = (size_t)mrow * N + n;
        if (Cf) Cf[o] = accumulate ? cur[j] + v : v;
        else Cb[o] = (__bf16)v;
      }
    }
    __syncthreads();   // red is reused by the next pass
  }
  if (ksplit == 1) return;
  // split K (M <= PR here): the last workgroup of the column block sums the
  // splits in order; the loads of one split are issued together
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (tid == 0)
    s_last = __hip_atomic_fetch_add(&counters[nb], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
             ksplit - 1;
  __syncthreads();
  if (!s_last) return;
  const int col = tid & 31, n = n0 + col;
  float sum[PR / 8];
#pragma unroll
  for (int j = 0; j < PR / 8; ++j) sum[j] = 0.f;
  for (int sp = 0; sp < ksplit; ++sp) {
    float v[PR / 8];
#pragma unroll
    for (int j = 0; j < PR / 8; ++j) {
      const int mrow = (tid >> 5) + 8 * j;
      v[j] = (mrow < M && n < N)
                 ? __hip_atomic_load(part + ((size_t)sp * M + mrow) * N + n, __ATOMIC_RELAXED,
                                     __HIP_MEMORY_SCOPE_AGENT)
                 : 0.f;
    }
#pragma unroll
    for (int j = 0; j < PR / 8; ++j) sum[j] += v[j];
  }
  float cur[PR / 8];
  if (Cf && accumulate) {
#pragma unroll
    for (int j = 0; j < PR / 8; ++j) {
      const int mrow = (tid >> 5) + 8 * j;
      cur[j] = (mrow < M && n < N) ? Cf[(size_t)mrow * N + n] : 0.f;
    }
  }
#pragma unroll
  for (int j = 0; j < PR / 8; ++j) {
    const int mrow = (tid >> 5) + 8 * j;
    if (mrow >= M || n >= N) continue;
    const size_t o = (size_t)mrow * N + n;
    if (Cf) Cf[o] = accumulate ? cur[j] + sum[j] : sum[j];
    else Cb[o] = (__bf16)sum[j];
  }
  if (tid == 0) __hip_atomic_store(&counters[nb], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// fp32: v_mfma_f32_32x32x2_f32; lane (row|col, hh) takes k = k0 + 4*hh + j in
// MFMA j, so one 16-byte load per operand feeds 4 MFMAs.
__global__ void __launch_bounds__(256) gemm_f32_kernel(const float* __restrict__ A,
                                                       const float* __restrict__ W, int M, int N,
                                                       int K, float* __restrict__ Cf, int accumulate) {
  const int lane = threadIdx.x & 63;
  const int wave = blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6);
  const int n0 = wave * 32;
  if (n0 >= N) return;
  const int l32 = lane & 31, hh = lane >> 5;
  const int ncol = n0 + l32;
  const bool nvalid = ncol < N;
  const float* wrow = W + (size_t)(nvalid ? ncol : n0) * K;
  for (int m0 = 0; m0 < M; m0 += MG_MAX * 32) {
    const int ng = min(MG_MAX, (M - m0 + 31) / 32);
    f32x16 acc[MG_MAX];
#pragma unroll
    for (int g = 0; g < MG_MAX; ++g) acc[g] = f32x16{};
    for (int k0 = 0; k0 < K; k0 += 8) {
      const f32x4 b = nvalid ? *(const f32x4*)(wrow + k0 + hh * 4) : f32x4{};
#pragma unroll
      for (int g = 0; g < MG_MAX; ++g) {
        if (g < ng) {
          const int mrow = m0 + g * 32 + l32;
          const f32x4 a = mrow < M ? *(const f32x4*)(A + (size_t)mrow * K + k0 + hh * 4) : f32x4{};
#pragma unroll
          for (int j = 0; j < 4; ++j)
            acc[g] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[j], b[j], acc[g], 0, 0, 0);
        }
      }
    }
    if (!nvalid) continue;
#pragma unroll
    for (int g = 0; g < MG_MAX; ++g) {
      if (g >= ng) break;
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int mrow = m0 + g * 32 + 8 * (i >> 2) + 4 * hh + (i & 3);
        if (mrow >= M) continue;
        const size_t o = (size_t)mrow * N + ncol;
        if (accumulate) Cf[o] += acc[g][i];
        else Cf[o] = acc[g][i];
      }
    }
  }
}

// ---------------------------------------------------------------------------
// host orchestration
// ---------------------------------------------------------------------------
struct StepLayout {
  size_t x, h, hsel, q, k, v, att, gate, up, act, logits, am, acc, attn_ws, total, attn_bytes,
      attn_counters, gemm_part, gemm_part_bytes, gemm_counters, n_gemm_counters;
};

// K splits of a bf16 GEMM over workgroups: enough column blocks x splits to
// fill the chip, a split being a multiple of 64 of K.  A function of (N, K)
// for every call of up to 256 rows (so row results do not depend on the row
// count); longer calls (prefill) have rows enough and do not split.
static int gemm_ksplit(int M, int N, int K) {
  if (M > GK_ROWS || K % 64 != 0) return 1;
  static_assert(GK_MAXSPLIT >= 1, "split bound");
  const int nb = (N + 31) / 32;
  const int target = (256 + nb - 1) / nb;
  if (target <= 1) return 1;
  const int units = K / 64;
  for (int d = target; d <= units && d <= GK_MAXSPLIT; ++d)
    if (units % d == 0) return d;
  for (int d = std::min(units, GK_MAXSPLIT); d > 1; --d)
    if (units % d == 0) return d;
  return 1;
}

__global__ void zero_words_kernel(int32_t* __restrict__ p, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0;
}

static size_t al(size_t v) { return (v + 255) & ~(size_t)255; }

static bool model_ok(const dvs_model* m) {
  return m && (m->dtype == DVS_F32 || m->dtype == DVS_BF16) && m->n_layers >= 1 && m->vocab >= 1 &&
         m->hidden >= 1 && m->n_kv_heads >= 1 && m->n_heads >= m->n_kv_heads &&
         m->n_heads % m->n_kv_heads == 0 && m->embed && m->g_final && m->lm_head && m->layers &&
         m->hidden % 16 == 0 && (m->ffn == 0 || m->ffn % 16 == 0);
}

// logit_rows: rows that get LM-head logits (every window row for a step;
// the last prefix row and the mask rows for a prefill)
static StepLayout step_layout(const dvs_model* m, int S, int n_causal, int n_mask, int max_pages,
                              int chunk_keys, size_t logit_rows) {
  StepLayout L{};
  const size_t M = (size_t)S * (n_causal + n_mask);
  const size_t es = m->dtype == DVS_BF16 ? 2 : 4;
  const size_t qd = (size_t)m->n_heads * m->head_dim, kd = (size_t)m->n_kv_heads * m->head_dim;
  size_t off = 0;
  L.x = off; off += al(M * m->hidden * 4);
  L.h = off; off += al(M * m->hidden * es);
  L.hsel = off; off += al(logit_rows * m->hidden * es);
  L.q = off; off += al(M * qd * es);
  L.k = off; off += al(M * kd * es);
  L.v = off; off += al(M * kd * es);
  L.att = off; off += al(M * qd * es);
  L.gate = off; off += al(M * (size_t)m->ffn * es);
  L.up = off; off += al(M * (size_t)m->ffn * es);
  L.act = off; off += al(M * (size_t)m->ffn * es);
  L.logits = off; off += al(logit_rows * (size_t)m->vocab * 4);
  L.am = off; off += al(logit_rows * 4);
  L.acc = off; off += al((size_t)S * 4);
  L.attn_bytes = dvs_attn_workspace_bytes(S, n_causal, n_mask, m->n_heads, m->n_kv_heads,
                                          m->head_dim, max_pages, chunk_keys, m->dtype);
  L.attn_counters = attn_counter_bytes(S, n_causal + n_mask, m->n_heads, m->n_kv_heads,
                                       m->head_dim, max_pages, chunk_keys, m->dtype);
  L.attn_ws = off; off += al(L.attn_bytes);
  // split-K partials and counters of the largest bf16 GEMM of the call
  if (m->dtype == DVS_BF16) {
    const int H = m->hidden;
    const int shapes[6][3] = {{(int)M, (int)qd, H}, {(int)M, (int)kd, H}, {(int)M, H, (int)qd},
                              {(int)M, m->ffn, H}, {(int)M, H, m->ffn}, {(int)logit_rows, m->vocab, H}};
    size_t part = 0, cnt = 0;
    for (const auto& sh : shapes) {
      if (sh[1] <= 0) continue;
      const int ksp = gemm_ksplit(sh[0], sh[1], sh[2]);
      if (ksp > 1) {
        part = std::max(part, (size_t)ksp * sh[0] * sh[1] * 4);
        cnt = std::max(cnt, (size_t)(sh[1] + 31) / 32);
      }
    }
    L.gemm_part = off; off += al(part); L.gemm_part_bytes = part;
    L.gemm_counters = off; off += al(cnt * 4); L.n_gemm_counters = cnt;
  }
  L.total = off;
  return L;
}

// C = A W^T (or C += for the fp32 residual).  `c_f32` selects an fp32 output
// for bf16 models (residual stream, logits); fp32 models always write fp32.
static int gemm(const StepLayout& L, char* ws, int dtype, const void* A, const void* W, int M,
                int N, int K, void* C, int c_f32, int accumulate, hipStream_t st) {
  const int waves = (N + 31) / 32;
  const int blocks = (waves + 3) / 4;
  if (dtype == DVS_BF16 && K % 64 == 0) {
    const int ksp = gemm_ksplit(M, N, K);
    const int nb = (N + 31) / 32;
    if (ksp > 1 && ((size_t)ksp * M * N * 4 > L.gemm_part_bytes || (size_t)nb > L.n_gemm_counters)) {
      set_error("draft_verify_step: GEMM split workspace too small");
      return DVS_EWORKSPACE;
    }
    float* part = (float*)(ws + L.gemm_part);
    int32_t* cnt = (int32_t*)(ws + L.gemm_counters);
    const dim3 grid(nb * ksp), blk(256);
    // rows per pass: the smallest power-of-two number of 32-row groups
    // covering M (up to 256 rows); the reduction order does not depend on it
    if (M <= 32)
      hipLaunchKernelGGL(gemm_bf16_sk_kernel<1>, grid, blk, 0, st, (const __bf16*)A, (const __bf16*)W, M, N, K, C, c_f32, accumulate, ksp, part, cnt);
    else if (M <= 64)
      hipLaunchKernelGGL(gemm_bf16_sk_kernel<2>, grid, blk, 0, st, (const __bf16*)A, (const __bf16*)W, M, N, K, C, c_f32, accumulate, ksp, part, cnt);
    else if (M <= 128)
      hipLaunchKernelGGL(gemm_bf16_sk_kernel<4>, grid, blk, 0, st, (const __bf16*)A, (const __bf16*)W, M, N, K, C, c_f32, accumulate, ksp, part, cnt);
    else
      hipLaunchKernelGGL(gemm_bf16_sk_kernel<8>, grid, blk, 0, st, (const __bf16*)A, (const __bf16*)W, M, N, K, C, c_f32, accumulate, ksp, part, cnt);
  } else if (dtype == DVS_BF16)
    hipLaunchKernelGGL(gemm_bf16_kernel, dim3(blocks), dim3(256), 0, st, (const __bf16*)A,
                       (const __bf16*)W, M, N, K, C, c_f32, accumulate);
  else
    hipLaunchKernelGGL(gemm_f32_kernel, dim3(blocks), dim3(256), 0, st, (const float*)A,
                       (const float*)W, M, N, K, (float*)C, accumulate);
  return launch_status("draft_verify_step(gemm)");
}

// The decoder stack on the rows in x (fp32, [M, hidden]); leaves the final
// RMSNorm output in h.  The window is (n_causal, n_mask) rows per sequence.
template <typename T>
static int forward_layers(const dvs_model* m, const dvs_state* st, int n_causal, int n_mask,
                          int chunk_keys, const StepLayout& L, char* ws, hipStream_t stream) {
  const int S = st->S, R = n_causal + n_mask, M = S * R;
  const int H = m->hidden, D = m->head_dim, Hq = m->n_heads, Hkv = m->n_kv_heads;
  const int dt = m->dtype;
  float* x = (float*)(ws + L.x);
  T* h = (T*)(ws + L.h);
  T* q = (T*)(ws + L.q);
  T* k = (T*)(ws + L.k);
  T* v = (T*)(ws + L.v);
  T* att = (T*)(ws + L.att);
  T* gate = (T*)(ws + L.gate);
  T* up = (T*)(ws + L.up);
  T* act = (T*)(ws + L.act);
  int rc;
  // The workspace may carry another call shape's data where this shape keeps
  // the attention's split counters: clear them once; every attention call
  // leaves them zero for the next layer.
  if (L.attn_counters) {
    const int nw = (int)(L.attn_counters / 4);
    hipLaunchKernelGGL(zero_words_kernel, dim3((nw + 255) / 256), dim3(256), 0, stream,
                       (int32_t*)(ws + L.attn_ws), nw);
  }
  if (L.n_gemm_counters) {
    const int nw = (int)L.n_gemm_counters;
    hipLaunchKernelGGL(zero_words_kernel, dim3((nw + 255) / 256), dim3(256), 0, stream,
                       (int32_t*)(ws + L.gemm_counters), nw);
  }
  const double log2_theta = log2((double)m->rope_theta);
  for (int l = 0; l < m->n_layers; ++l) {
    const dvs_layer& ly = m->layers[l];
    hipLaunchKernelGGL(rmsnorm_kernel<T>, dim3(M), dim3(256), 0, stream, x, (const T*)ly.g_attn, H,
                       m->rms_eps, h);
    if ((rc = gemm(L, ws, dt, h, ly.wq, M, Hq * D, H, q, 0, 0, stream))) return rc;
    if ((rc = gemm(L, ws, dt, h, ly.wk, M, Hkv * D, H, k, 0, 0, stream))) return rc;
    if ((rc = gemm(L, ws, dt, h, ly.wv, M, Hkv * D, H, v, 0, 0, stream))) return rc;
    const long long nq = (long long)M * Hq * (D / 2), nk = (long long)M * Hkv * (D / 2);
    hipLaunchKernelGGL(rope_kernel<T>, dim3((unsigned)((nq + 255) / 256)), dim3(256), 0, stream, q, M,
                       R, Hq, D, log2_theta, st->kv_len);
    hipLaunchKernelGGL(rope_kernel<T>, dim3((unsigned)((nk + 255) / 256)), dim3(256), 0, stream, k, M,
                       R, Hkv, D, log2_theta, st->kv_len);
    if ((rc = launch_status("draft_verify_step(rope)"))) return rc;
    rc = attn_hybrid_block(q, k, v, ly.k_pool, ly.v_pool, st->page_table, st->kv_len, S, n_causal,
                           n_mask, Hq, Hkv, D, st->max_pages, st->num_pool_pages,
                           (float)(1.0 / sqrt((double)D)), dt, chunk_keys, att, st->err_word,
                           ws + L.attn_ws, L.attn_bytes, stream);
    if (rc) return rc;
    if ((rc = gemm(L, ws, dt, att, ly.wo, M, H, Hq * D, x, 1, 1, stream))) return rc;
    if (m->ffn > 0) {
      hipLaunchKernelGGL(rmsnorm_kernel<T>, dim3(M), dim3(256), 0, stream, x, (const T*)ly.g_mlp,
                         H, m->rms_eps, h);
      if ((rc = gemm(L, ws, dt, h, ly.w_gate, M, m->ffn, H, gate, 0, 0, stream))) return rc;
      if ((rc = gemm(L, ws, dt, h, ly.w_up, M, m->ffn, H, up, 0, 0, stream))) return rc;
      const long long n = (long long)M * m->ffn;
      hipLaunchKernelGGL(silu_mul_kernel<T>, dim3((unsigned)((n + 255) / 256)), dim3(256), 0,
                         stream, gate, up, n, act);
      if ((rc = launch_status("draft_verify_step(silu)"))) return rc;
      if ((rc = gemm(L, ws, dt, act, ly.w_down, M, H, m->ffn, x, 1, 1, stream))) return rc;
    }
  }
  hipLaunchKernelGGL(rmsnorm_kernel<T>, dim3(M), dim3(256), 0, stream, x, (const T*)m->g_final, H,
                     m->rms_eps, h);
  return launch_status("draft_verify_step(final norm)");
}

template <typename T>
static int run_step(const dvs_model* m, const dvs_state* st, int n_causal, int n_mask,
                    int chunk_keys, const StepLayout& L, char* ws, float* logits_out,
                    int32_t* argmax_out, int32_t* accept_out, hipStream_t stream) {
  const int S = st->S, R = n_causal + n_mask, M = S * R;
  float* logits = logits_out ? logits_out : (float*)(ws + L.logits);
  int32_t* am = argmax_out ? argmax_out : (int32_t*)(ws + L.am);
  int32_t* acc = accept_out ? accept_out : (int32_t*)(ws + L.acc);
  hipLaunchKernelGGL(embed_rows_kernel<T>, dim3(M), dim3(256), 0, stream, (const T*)m->embed,
                     m->hidden, m->vocab, R, n_causal, st->boundary, st->draft, st->draft_width,
                     (float*)(ws + L.x));
  int rc;
  if ((rc = launch_status("draft_verify_step(embed)"))) return rc;
  if ((rc = forward_layers<T>(m, st, n_causal, n_mask, chunk_keys, L, ws, stream))) return rc;
  if ((rc = gemm(L, ws, m->dtype, ws + L.h, m->lm_head, M, m->vocab, m->hidden, logits, 1, 0, stream)))
    return rc;
  rc = argmax_accept(logits, DVS_F32, S, R, m->vocab, n_causal, st->draft, st->draft_width, am, acc,
                     st->err_word, stream);
  if (rc) return rc;
  return kv_commit(S, n_causal, n_mask, acc, am, st->kv_len, st->page_table, st->num_pages,
                   st->max_pages, st->free_stack, st->free_top, st->num_pool_pages, st->boundary,
                   st->draft, st->draft_width, st->out_tokens, st->out_count, st->max_new, st->eos_id,
                   st->finished, st->err_word, stream);
}

template <typename T>
static int run_prefill(const dvs_model* m, const dvs_state* st, int P, int n_mask,
                       const int32_t* tokens, const float* x_prefix, int chunk_keys,
                       const StepLayout& L, char* ws, float* logits_out, hipStream_t stream) {
  const int S = st->S, R = P + n_mask, M = S * R, nsel = n_mask + 1;
  hipLaunchKernelGGL(embed_prefill_kernel<T>, dim3(M), dim3(256), 0, stream, (const T*)m->embed,
                     m->hidden, m->vocab, R, P, tokens, x_prefix, (float*)(ws + L.x));
  int rc;
  if ((rc = launch_status("dvs_prefill(embed)"))) return rc;
  if ((rc = forward_layers<T>(m, st, P, n_mask, chunk_keys, L, ws, stream))) return rc;
  // LM head only for rows P-1 .. P+n_mask-1 (the first token and the draft)
  T* hsel = (T*)(ws + L.hsel);
  hipLaunchKernelGGL(gather_rows_kernel<T>, dim3(S * nsel), dim3(256), 0, stream,
                     (const T*)(ws + L.h), m->hidden, R, P - 1, nsel, hsel);
  float* logits = logits_out ? logits_out : (float*)(ws + L.logits);
  if ((rc = gemm(L, ws, m->dtype, hsel, m->lm_head, S * nsel, m->vocab, m->hidden, logits, 1, 0, stream)))
    return rc;
  int32_t* am = (int32_t*)(ws + L.am);
  int32_t* acc = (int32_t*)(ws + L.acc);
  rc = argmax_accept(logits, DVS_F32, S, nsel, m->vocab, 1, nullptr, 0, am, acc, st->err_word, stream);
  if (rc) return rc;
  hipLaunchKernelGGL(prefill_commit_kernel, dim3((S + 255) / 256), dim3(256), 0, stream, S, P,
                     n_mask, am, st->kv_len, st->boundary, st->draft, st->draft_width,
                     st->out_tokens, st->out_count, st->max_new, st->eos_id, st->finished);
  return launch_status("dvs_prefill(commit)");
}

}  // namespace dvs

using namespace dvs;

extern "C" size_t dvs_step_workspace_bytes(const dvs_model* m, int32_t S, int32_t n_causal,
                                           int32_t n_mask, int32_t max_pages, int32_t chunk_keys) {
  if (!model_ok(m) || S < 1 || n_causal < 1 || n_mask < 0 || max_pages < 1) return 0;
  return step_layout(m, S, n_causal, n_mask, max_pages, chunk_keys,
                     (size_t)S * (n_causal + n_mask)).total;
}

extern "C" int draft_verify_step(const dvs_model* m, const dvs_state* st, int32_t n_causal,
                                 int32_t n_mask, int32_t chunk_keys, float* logits_out,
                                 int32_t* argmax_out, int32_t* accept_out, void* workspace,
                                 size_t ws_bytes, void* stream) {
  clear_error();
  DVS_CHECK_ARG(model_ok(m), "draft_verify_step: invalid model description");
  DVS_CHECK_ARG(st && st->S >= 1 && st->kv_len && st->page_table && st->num_pages &&
                    st->free_stack && st->free_top && st->boundary && st->out_tokens &&
                    st->out_count && st->finished,
                "draft_verify_step: invalid state description");
  DVS_CHECK_ARG(n_causal >= 1 && n_mask >= 0, "draft_verify_step: need n_causal >= 1");
  DVS_CHECK_ARG(st->draft_width >= n_causal - 1 && (st->draft || st->draft_width == 0),
                "draft_verify_step: draft narrower than n_causal - 1");
  for (int l = 0; l < m->n_layers; ++l) {
    const dvs_layer& ly = m->layers[l];
    DVS_CHECK_ARG(ly.wq && ly.wk && ly.wv && ly.wo && ly.g_attn && ly.k_pool && ly.v_pool,
                  "draft_verify_step: layer %d incomplete", l);
    DVS_CHECK_ARG(m->ffn == 0 || (ly.g_mlp && ly.w_gate && ly.w_up && ly.w_down),
                  "draft_verify_step: layer %d MLP incomplete", l);
  }
  DVS_CHECK_SUPPORTED(m->head_dim == 64 || m->head_dim == 96 || m->head_dim == 128,
                      "draft_verify_step: head_dim %d", m->head_dim);
  const StepLayout L = step_layout(m, st->S, n_causal, n_mask, st->max_pages, chunk_keys,
                                   (size_t)st->S * (n_causal + n_mask));
  if (!workspace || ws_bytes < L.total) {
    set_error("draft_verify_step: workspace needs %zu bytes, got %zu", L.total, ws_bytes);
    return DVS_EWORKSPACE;
  }
  hipStream_t s = (hipStream_t)stream;
  if (m->dtype == DVS_BF16)
    return run_step<__bf16>(m, st, n_causal, n_mask, chunk_keys, L, (char*)workspace, logits_out,
                            argmax_out, accept_out, s);
  return run_step<float>(m, st, n_causal, n_mask, chunk_keys, L, (char*)workspace, logits_out,
                         argmax_out, accept_out, s);
}

extern "C" size_t dvs_prefill_workspace_bytes(const dvs_model* m, int32_t S, int32_t P,
                                              int32_t n_mask, int32_t max_pages,
                                              int32_t chunk_keys) {
  if (!model_ok(m) || S < 1 || P < 1 || n_mask < 0 || max_pages < 1) return 0;
  return step_layout(m, S, P, n_mask, max_pages, chunk_keys, (size_t)S * (n_mask + 1)).total;
}

extern "C" int dvs_prefill(const dvs_model* m, const dvs_state* st, int32_t P, int32_t n_mask,
                           const int32_t* prefix_tokens, const float* x_prefix, int32_t chunk_keys,
                           float* logits_out, void* workspace, size_t ws_bytes, void* stream) {
  clear_error();
  DVS_CHECK_ARG(model_ok(m), "dvs_prefill: invalid model description");
  DVS_CHECK_ARG(st && st->S >= 1 && st->kv_len && st->page_table && st->boundary &&
                    st->out_tokens && st->out_count && st->finished,
                "dvs_prefill: invalid state description");
  DVS_CHECK_ARG(P >= 1 && n_mask >= 0, "dvs_prefill: need P >= 1, n_mask >= 0");
  DVS_CHECK_ARG(prefix_tokens || x_prefix, "dvs_prefill: no prefix inputs");
  DVS_CHECK_ARG(n_mask >= st->draft_width && (st->draft || st->draft_width == 0),
                "dvs_prefill: mask rows (%d) must cover the draft width (%d)", n_mask,
                st->draft_width);
  DVS_CHECK_SUPPORTED(m->head_dim == 64 || m->head_dim == 96 || m->head_dim == 128,
                      "dvs_prefill: head_dim %d", m->head_dim);
  const StepLayout L = step_layout(m, st->S, P, n_mask, st->max_pages, chunk_keys,
                                   (size_t)st->S * (n_mask + 1));
  if (!workspace || ws_bytes < L.total) {
    set_error("dvs_prefill: workspace needs %zu bytes, got %zu", L.total, ws_bytes);
    return DVS_EWORKSPACE;
  }
  hipStream_t s = (hipStream_t)stream;
  if (m->dtype == DVS_BF16)
    return run_prefill<__bf16>(m, st, P, n_mask, prefix_tokens, x_prefix, chunk_keys, L,
                               (char*)workspace, logits_out, s);
  return run_prefill<float>(m, st, P, n_mask, prefix_tokens, x_prefix, chunk_keys, L,
                            (char*)workspace, logits_out, s);
}
