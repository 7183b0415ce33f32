// draft_verify_step: one fused self-speculative step of a decoder.
//
// Row inputs (Method "AR-to-Diffusion Conversion": the only architectural
// addition is the embedding of the mask token [M]):
//   causal rows r = 0..n_causal-1 : [x0, d_1, .., d_{n_causal-1}]
//   mask rows                     : [M] (embedding row `vocab`)
// then per layer: RMSNorm -> Q/K/V projections -> rotary positions at
// kv_len + r -> attn_hybrid_block (appends the window's K/V) -> O projection
// + residual -> [RMSNorm -> SwiGLU MLP + residual], final RMSNorm, LM head,
// and the hot-path tail argmax_accept -> accept_commit.
//
// Every matrix product is C[m, n] = sum_k A[m, k] * W[n, k] with weights laid
// out [out, in] so both MFMA operands are contiguous along k.  K is cut into
// a fixed number of logical splits that depends on K only; each output is the
// in-order sum of the splits' in-order MFMA accumulations, whichever kernel
// computes it (gemm_ws_kernel for calls of up to 256 rows, gemm_rt_kernel for
// longer ones).  A row's result therefore never depends on how many rows the
// call carries, so an AR call (1 row) and a fused call (2B rows) produce
// bit-identical rows.
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

// The RMS norm of a row held in registers by a 256-thread workgroup:
// thread t holds elements 8t .. 8t+7 (xa, xb; zeros where t >= H/8 = nrun),
// and writes them normalized (H/8 <= 256).  rmsnorm_kernel's arithmetic for
// such a row; shared so that every caller gets the same bits.
template <typename T>
__device__ __forceinline__ void rms_row_held(f32x4 xa, f32x4 xb, const T* __restrict__ g, int H,
                                             float eps, T* __restrict__ orow, float* red) {
  const int t = threadIdx.x;
  float ss = 0.f;
#pragma unroll
  for (int e = 0; e < 4; ++e) ss = fmaf(xa[e], xa[e], ss);
#pragma unroll
  for (int e = 0; e < 4; ++e) ss = fmaf(xb[e], xb[e], ss);
  for (int off = 32; off > 0; off >>= 1) ss += __shfl_xor(ss, off);
  if ((t & 63) == 0) red[t >> 6] = ss;
  __syncthreads();
  const float tot = (red[0] + red[1]) + (red[2] + red[3]);
  const float inv = 1.0f / sqrtf(tot / (float)H + eps);
  if (t < H / 8) {
#pragma unroll
    for (int e = 0; e < 8; ++e)
      orow[8 * t + e] = from_f<T>((e < 4 ? xa[e] : xb[e - 4]) * inv * to_f(g[8 * t + e]));
  }
}

// x[m, :] = embed[token(m), :] (fp32 residual stream); with `h` set (bf16,
// H <= 2048, 256 threads) also h[m, :] = the RMS norm of that row with gain
// g0 (rms_row_held: the first layer's norm, bit for bit, without a launch)
template <typename T>
__global__ void embed_rows_kernel(const T* __restrict__ embed, int H, int vocab, int R, int n_causal,
                                  const int32_t* __restrict__ boundary,
                                  const int32_t* __restrict__ draft, int draft_width,
                                  const int32_t* __restrict__ block, int block_stride,
                                  float* __restrict__ x, const T* __restrict__ g0 = nullptr,
                                  float eps = 0.f, T* __restrict__ h = nullptr) {
  const int mrow = blockIdx.x;
  const int s = mrow / R, r = mrow - s * R;
  int tok = vocab;  // [M]
  if (r < n_causal) tok = (r == 0) ? boundary[s] : draft[(size_t)s * draft_width + (r - 1)];
  else if (block) tok = block[(size_t)s * block_stride + (r - n_causal)];  // -1: [M]
  if (tok < 0 || tok > vocab) tok = vocab;
  const T* e = embed + (size_t)tok * H;
  float* xr = x + (size_t)mrow * H;
  if constexpr (sizeof(T) == 2) {
    if (h) {
      // one run of 8 per thread, kept in registers for the norm
      __shared__ float red[4];
      const int t = threadIdx.x;
      f32x4 xa = f32x4{0.f, 0.f, 0.f, 0.f}, xb = xa;
      if (t < H / 8) {
        const bf16x8 v = *(const bf16x8*)(e + 8 * t);
        xa = f32x4{(float)v[0], (float)v[1], (float)v[2], (float)v[3]};
        xb = f32x4{(float)v[4], (float)v[5], (float)v[6], (float)v[7]};
        *(f32x4*)(xr + 8 * t) = xa;
        *(f32x4*)(xr + 8 * t + 4) = xb;
      }
      rms_row_held<T>(xa, xb, g0, H, eps, h + (size_t)mrow * H, red);
      return;
    }
    // runs of 8 (H is a multiple of 16): one 16-byte read, two 16-byte writes
    for (int c = threadIdx.x; c < H / 8; c += blockDim.x) {
      const bf16x8 v = *(const bf16x8*)(e + 8 * c);
      *(f32x4*)(xr + 8 * c) = f32x4{(float)v[0], (float)v[1], (float)v[2], (float)v[3]};
      *(f32x4*)(xr + 8 * c + 4) = f32x4{(float)v[4], (float)v[5], (float)v[6], (float)v[7]};
    }
  } else {
    for (int i = threadIdx.x; i < H; i += blockDim.x) xr[i] = to_f(e[i]);
  }
}

// Two-forward round, between the forwards (appendix "Self-Speculative
// Decoding and KV-Cache Update", item Draft forward): a0 = top-1 of the
// boundary row, d_j = top-1 of mask row j (j = 1..B), and the causal KV the
// draft forward wrote for x0 is kept (kv_len + 1).  Finished sequences keep
// their state.  am: [S, B + 1].
__global__ void round_draft_kernel(int S, int B, const int32_t* __restrict__ am,
                                   const int32_t* __restrict__ finished, int32_t* __restrict__ kv_len,
                                   int32_t* __restrict__ lead, int32_t* __restrict__ draft,
                                   int draft_width) {
  const int s = blockIdx.x * blockDim.x + threadIdx.x;
  if (s >= S) return;
  const int R = B + 1;
  lead[s] = am[(size_t)s * R];
  if (finished[s]) return;
  for (int j = 0; j < B; ++j) draft[(size_t)s * draft_width + j] = am[(size_t)s * R + 1 + j];
  kv_len[s] += 1;
}

// Reveal of one denoising step (appendix "Direct Block-Diffusion
// Decoding"): every masked block position p whose prediction (top-1 of
// window row p-1) has confidence above tau_c takes that token; when no
// position qualifies, the most confident masked one does (lowest position
// among ties).  Revealed positions never change.  One 64-lane wave per
// sequence, lane = position mod 64; a sequence whose block stays open adds
// one to *n_open.  block: [S, B] (-1 = masked); am, conf: [S, R], R > B-1
// (row p-1 predicts position p).  The refined draft of the two-forward round
// uses B = R: its last prediction has no input slot.
__global__ void __launch_bounds__(64) reveal_kernel(int B, int R, float tau_c,
                                                    const int32_t* __restrict__ am,
                                                    const float* __restrict__ conf,
                                                    const int32_t* __restrict__ finished,
                                                    int32_t* __restrict__ block,
                                                    int32_t* __restrict__ n_open) {
  const int s = blockIdx.x, lane = threadIdx.x;
  if (finished[s]) return;
  int32_t* b = block + (size_t)s * B;
  const int32_t* a = am + (size_t)s * R;
  const float* c = conf + (size_t)s * R;
  constexpr int NONE = 0x7fffffff;
  int hits = 0, bp = NONE;
  float bc = 0.f;
  for (int p = lane; p < B; p += 64) {
    if (b[p] >= 0) continue;
    const float cp = c[p];
    if (cp > tau_c) {
      b[p] = a[p];
      ++hits;
    } else if (bp == NONE || cp > bc) {   // positions ascend: the first of equals stays
      bc = cp;
      bp = p;
    }
  }
  if (!__any(hits)) {
    // (larger confidence, then smaller position) over the wave
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
      const float oc = __shfl_xor(bc, off);
      const int op = __shfl_xor(bp, off);
      if (op != NONE && (bp == NONE || oc > bc || (oc == bc && op < bp))) {
        bc = oc;
        bp = op;
      }
    }
    if (bp != NONE && (bp & 63) == lane) b[bp] = a[bp];
  }
  int left = 0;
  for (int p = lane; p < B; p += 64) left |= b[p] < 0;
  if (__any(left) && lane == 0) atomicAdd(n_open, 1);
}

__global__ void fill_words_kernel(int32_t* __restrict__ p, int n, int32_t v) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

// out[m, :] = x[m, :] / sqrt(mean(x^2) + eps) * g   (one workgroup per row).
// Thread t takes the runs of 8 elements 8(t + 256c) .. 8(t + 256c) + 7,
// c = 0, 1, ... (16-byte loads; the sum of squares in that order), then a
// butterfly over its wave, then (w0 + w1) + (w2 + w3).  H is a multiple of
// 8; a row of up to 2048 elements is loaded once before the reduction, with
// no per-element branch around the loads (the per-element form waited for
// each load in turn: 4.5 -> about 2.5 us per launch).
template <typename T>
__global__ void __launch_bounds__(256) rmsnorm_kernel(const float* __restrict__ x, const T* __restrict__ g,
                                                      int H, float eps, T* __restrict__ out) {
  __shared__ float red[4];
  const int mrow = blockIdx.x, t = threadIdx.x;
  const float* xr = x + (size_t)mrow * H;
  T* orow = out + (size_t)mrow * H;
  const int nrun = H / 8;
  if (nrun <= 256) {
    // the row in one pass, loaded before the reduction
    f32x4 xa = f32x4{0.f, 0.f, 0.f, 0.f}, xb = xa;
    if (t < nrun) {
      xa = *(const f32x4*)(xr + 8 * t);
      xb = *(const f32x4*)(xr + 8 * t + 4);
    }
    rms_row_held<T>(xa, xb, g, H, eps, orow, red);
    return;
  }
  float ss = 0.f;
  for (int c = t; c < nrun; c += 256) {
    const f32x4 a = *(const f32x4*)(xr + 8 * c), b = *(const f32x4*)(xr + 8 * c + 4);
#pragma unroll
    for (int e = 0; e < 4; ++e) ss = fmaf(a[e], a[e], ss);
#pragma unroll
    for (int e = 0; e < 4; ++e) ss = fmaf(b[e], b[e], ss);
  }
  for (int off = 32; off > 0; off >>= 1) ss += __shfl_xor(ss, off);
  if ((t & 63) == 0) red[t >> 6] = ss;
  __syncthreads();
  const float tot = (red[0] + red[1]) + (red[2] + red[3]);
  const float inv = 1.0f / sqrtf(tot / (float)H + eps);
  for (int c = t; c < nrun; c += 256) {
    const f32x4 a = *(const f32x4*)(xr + 8 * c), b = *(const f32x4*)(xr + 8 * c + 4);
#pragma unroll
    for (int e = 0; e < 8; ++e)
      orow[8 * c + e] = from_f<T>((e < 4 ? a[e] : b[e - 4]) * inv * to_f(g[8 * c + e]));
  }
}

// Position of window row r relative to kv_len: r, except for mask rows cut
// into groups of `group` rows (G = n_mask / group groups), where row i of
// group g sits right after the last causal row the group sees:
// n_causal - G + g + 1 + i (one group gives r again).
__device__ __forceinline__ int window_offset(int r, int n_causal, int n_mask, int group) {
  if (r < n_causal || group <= 0) return r;
  const int n_groups = n_mask / group;
  const int g = (r - n_causal) / group, i = (r - n_causal) - g * group;
  return n_causal - n_groups + g + 1 + i;
}

// Rotate-half rotary embedding: pair (x1 = element i, x2 = element i + D/2
// of a head) at position pos turns by the angle pos * theta^(-2i/D),
// computed in double precision (positions reach thousands of radians).  One
// definition for the standalone kernel and the per-step table the Q|K|V
// GEMM epilogue reads, so both round alike.
__device__ __forceinline__ void rope_cs_sn(int i, int D, double log2_theta, double pos, double& cs,
                                           double& sn) {
  const double inv = exp2(-2.0 * i / D * log2_theta);
  sincos(pos * inv, &sn, &cs);
}
__device__ __forceinline__ void rope_rotate(float x1, float x2, double cs, double sn, float& o1,
                                            float& o2) {
  o1 = (float)(x1 * cs - x2 * sn);
  o2 = (float)(x1 * sn + x2 * cs);
}

// (cos, sin) of every (row, i < D/2) of a step: row s * R + r at position
// kv_len[s] + window_offset(r); the same for every layer of the step.  The
// first zero_blocks workgroups clear zero[0 .. n_zero) instead (the
// attention's split counters), so that both take one launch.
__global__ void rope_table_kernel(double2* __restrict__ tab, int M, int R, int D, double log2_theta,
                                  const int32_t* __restrict__ kv_len, int n_causal, int n_mask,
                                  int group, int32_t* __restrict__ zero, int n_zero,
                                  int zero_blocks) {
  if ((int)blockIdx.x < zero_blocks) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n_zero) zero[i] = 0;
    return;
  }
  const int half = D / 2;
  const int idx = (blockIdx.x - zero_blocks) * blockDim.x + threadIdx.x;
  if (idx >= M * half) return;
  const int mrow = idx / half, i = idx - mrow * half;
  const int s = mrow / R, r = mrow - s * R;
  const double pos = (double)(kv_len[s] + window_offset(r, n_causal, n_mask, group));
  double cs, sn;
  rope_cs_sn(i, D, log2_theta, pos, cs, sn);
  tab[idx] = double2{cs, sn};
}

// rotate-half rotary embedding, in place, at position kv_len[s] +
// window_offset(r)
template <typename T>
__global__ void rope_kernel(T* __restrict__ xq, int nhq, T* __restrict__ xk, int nhk, int M, int R,
                            int D, double log2_theta, const int32_t* __restrict__ kv_len,
                            int n_causal, int n_mask, int group) {
  // one launch for the query and the key heads: indices below M*nhq*D/2
  // rotate q, the rest k
  const int half = D / 2;
  long long idx = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  const long long nq = (long long)M * nhq * half;
  T* x = xq;
  int nh = nhq;
  if (idx >= nq) {
    idx -= nq;
    x = xk;
    nh = nhk;
  }
  if (idx >= (long long)M * nh * half) return;
  const int i = (int)(idx % half);
  const long long mh = idx / half;
  const int mrow = (int)(mh / nh);
  const int s = mrow / R, r = mrow - s * R;
  const double pos = (double)(kv_len[s] + window_offset(r, n_causal, n_mask, group));
  T* v = x + mh * D;
  double cs, sn;
  rope_cs_sn(i, D, log2_theta, pos, cs, sn);
  float o1, o2;
  rope_rotate(to_f(v[i]), to_f(v[i + half]), cs, sn, o1, o2);
  v[i] = from_f<T>(o1);
  v[i + half] = from_f<T>(o2);
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
// Generic GEMM: C[m, n] (=, or += into an fp32 residual) sum_k A[m, k] W[n, k]
// for the fp32 model and for bf16 shapes whose K is not a multiple of 64
// (small test models).  One wave per 32 output columns; it walks k in
// ascending order, loading each weight fragment once and applying it to every
// 32-row group of A (up to MG_MAX groups, the rest in further passes), so a
// row's result does not depend on the row count here either.
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
// bf16 GEMMs of the decoder stack.  C[m, n] = sum_k A[m, k] W[n, k] (bf16
// operands, fp32 accumulation).
//
// Row invariance.  K is cut into KS logical splits (KS = 4 when K is a
// multiple of 256, else 1; a function of K only).  Every output element is
//     ((0 + p_0) + p_1) + ... + p_{KS-1}      (fp32, in this order)
// where p_s is the in-order accumulation of v_mfma_f32_32x32x16_bf16 over the
// 16-wide k-steps of split s (lane half hh holds k values 8*hh .. 8*hh+7 of a
// step in both operands).  Both kernels below compute exactly that, so a
// row's result never depends on how many rows a call carries: a fused step's
// causal rows, a two-forward round's verify rows and AR rows agree bit for
// bit.
//   * gemm_ws_kernel (calls of at most WS_MAX_ROWS rows: every decode step
//     of the benchmark shapes): wave s of a workgroup computes split s of a
//     (row tile x 32 columns) tile straight from global memory and the four
//     splits are added through LDS in order -- no partials leave the
//     workgroup;
//   * gemm_rt_kernel (longer calls: prefill, wide multi-draft windows): LDS-
//     staged tiles of MT rows x 128 columns, the splits' products added to a
//     running sum in registers.
// ---------------------------------------------------------------------------
constexpr int GK_SPLITS = 4;        // logical K splits when K % 256 == 0
constexpr int WS_MAX_ROWS = 256;    // calls up to this many rows use gemm_ws_kernel
constexpr int WS_NARROW_NB = 128;   // few-row calls below this many 32-column blocks take narrow blocks
constexpr int WS_WIDE_MIN_WG = 256; // 64-row calls take 2 blocks per wave while the grid keeps this many

static int gemm_ksplit(int K) { return K % (64 * GK_SPLITS) == 0 ? GK_SPLITS : 1; }

// ---------------------------------------------------------------------------
// gemm_ws_kernel<MT, NARROW, CB, EPI, WK>: weight-streaming GEMM for
// decode-step row counts.
//
// Workgroup = 4 waves = one (row tile of MT rows, group of CB 32-column
// blocks); wave s computes split s (K/4 consecutive k) for the whole tile.
// Each wave copies its K chunks (the blocks' weight rows and MT rows of A)
// with direct global -> LDS 16-byte loads, fully coalesced, into a private
// ring ahead of its products, and feeds the MFMAs from there (no barriers
// between the waves until the split sums).  Each weight element is read
// once per row tile; the row tiles of a column group are dispatched back to
// back on one XCD (blockIdx mod 8), so the second and later ones find the
// group's weights in that XCD's L2.  The splits meet in LDS and are added in
// order, then the epilogue EPI writes the tile:
//   EPI_BF16       C (bf16) of the column block's segment (fused projections:
//                  up to three weight matrices side by side, e.g. Wq|Wk|Wv,
//                  each output into its own array; with a rotary table the
//                  first two leave rotated);
//   EPI_F32_ADD    C (fp32) += tile (the residual stream);
//   EPI_F32        C (fp32) = tile (logits);
//   EPI_SWIGLU     columns 0..15 of a block are gate rows, 16..31 the same up
//                  rows: act = bf16(silu(bf16 gate) * bf16 up), 16 outputs per
//                  row (the same roundings as separate gate, up and silu*up
//                  passes);
//   EPI_ARGMAX     per row the block's largest logit and its lowest index,
//                  packed (order-preserving key, 0x7fffffff - index) for a
//                  64-bit max (NaN never wins; non-finite values set
//                  DVS_ERR_NONFINITE); argmax_rows_kernel takes the max over
//                  a row's blocks, so the logits never reach memory.
// ---------------------------------------------------------------------------
enum { EPI_BF16 = 0, EPI_F32 = 1, EPI_F32_ADD = 2, EPI_SWIGLU = 3, EPI_ARGMAX = 4 };

struct GemmSeg {
  const __bf16* W;   // [n, K] rows of this segment
  void* C;           // output of this segment, row stride = n (EPI_SWIGLU: the act array)
  int n0, n;         // columns [n0, n0 + n) of the fused output
};

struct GemmArgs {
  const __bf16* A;
  int M, K, ncols;   // ncols: total output columns (EPI_SWIGLU: 2 * ffn)
  GemmSeg seg[3];
  int nseg, epi, n_rt;
  uint64_t* part;    // EPI_ARGMAX: [M, ncols / 32]
  int32_t* err;
  // EPI_BF16 with rope_tab set: segments 0 and 1 (Q and K, heads of rope_D)
  // leave rotated by the rotary embedding, (cos, sin) of (row, i) at
  // rope_tab[row * rope_D / 2 + i] (rope_table_kernel)
  const double2* rope_tab;
  int rope_D;
};

__device__ __forceinline__ uint64_t pack_logit(float v, int idx, bool& nonfinite) {
  uint32_t u = __float_as_uint(v);
  if ((u & 0x7f800000u) == 0x7f800000u) nonfinite = true;
  if (v != v) return 0;                        // NaN: never the top-1
  if ((u & 0x7fffffffu) == 0) u = 0;           // -0 == +0
  const uint32_t key = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return ((uint64_t)key << 32) | (uint32_t)(0x7fffffff - idx);
}

// s_waitcnt vmcnt(n) with the other counters untouched (gfx9 encoding).
template <int N>
__device__ __forceinline__ void ws_wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// The epilogue of a weight-streaming GEMM tile (MT rows x CB 32-column
// blocks of CW kept columns): s_red holds NSP planes [NSP][MT][CB * 32] of
// fp32 partial sums (the splits, or one plane already summed in order),
// added in plane order as ((0 + p0) + p1) + ...; then EPI writes the tile.
// EPI_F32_ADD: the residual values of the tile's whole 4-column runs, loaded
// when the kernel starts (the tile is written only by its own epilogue), so
// that the epilogue does not wait for them; unit u0 + tid of the epilogue's
// loop is cpre[u0 / 256].
template <int MT, int CB, int CW>
__device__ __forceinline__ void ws_residual_prefetch(const GemmArgs& g, int tid, int m0, int cg, int si,
                                                     f32x4* cpre) {
  constexpr int TW = CB * 32;
  constexpr int UNITS = MT * TW / 4;
  const GemmSeg sg = g.seg[si];
  const bool vec = (sg.n & 3) == 0;
#pragma unroll
  for (int u0 = 0; u0 < UNITS; u0 += 256) {
    const int u = u0 + tid;
    const int r = u / (TW / 4), cc = (u % (TW / 4)) * 4;
    const int c = cc & 31;
    const int row = m0 + r;
    const int col = (cg * CB + (cc >> 5)) * CW + c - sg.n0;
    cpre[u0 / 256] = f32x4{0.f, 0.f, 0.f, 0.f};
    if (u < UNITS && row < g.M && c < CW && vec && col + 4 <= sg.n)
      cpre[u0 / 256] = *(const f32x4*)((const float*)sg.C + (size_t)row * sg.n + col);
  }
}

template <int MT, int CB, int CW, int EPI, int NSP>
__device__ __forceinline__ void ws_epilogue(const GemmArgs& g, const float* __restrict__ s_red,
                                            int tid, int lane, int m0, int cg, int si, int NB,
                                            bool rope, const f32x4* cpre = nullptr) {
  constexpr int TW = CB * 32;
  // the tile's sums, 4 adjacent columns at a time: ((0 + p0) + p1) + ...
  // per element, the split planes in order
  auto sum4 = [&](int r, int cc) {
    f32x4 t = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int sp = 0; sp < NSP; ++sp) t += *(const f32x4*)(s_red + sp * (MT * TW) + r * TW + cc);
    return t;
  };
  if (EPI == EPI_BF16 && rope) {
    // a unit: column j < P of a block (dim i of a head) and its partner
    // column P + j (dim i + D/2), each rounded to bf16 as the projection
    // writes it, then rotated
    const GemmSeg sg = g.seg[si];
    constexpr int P = CW / 2;
    constexpr int UNITS = MT * CB * P;
    const int D = g.rope_D, half = D / 2;
#pragma unroll
    for (int u0 = 0; u0 < UNITS; u0 += 256) {
      const int u = u0 + tid;
      const int r = u / (CB * P), b = (u / P) % CB, j = u % P;
      const int row = m0 + r;
      const int cs = (cg * CB + b) * CW - sg.n0;   // the block's first column in the segment
      if (u >= UNITS || row >= g.M || cs >= sg.n) continue;
      const int hd = cs / D, i = (cs - hd * D) / CW * P + j;
      float t1 = 0.f, t2 = 0.f;
#pragma unroll
      for (int sp = 0; sp < NSP; ++sp) {
        t1 += s_red[sp * (MT * TW) + r * TW + b * 32 + j];
        t2 += s_red[sp * (MT * TW) + r * TW + b * 32 + P + j];
      }
      const double2 cssn = g.rope_tab[(size_t)row * half + i];
      float o1, o2;
      rope_rotate((float)(__bf16)t1, (float)(__bf16)t2, cssn.x, cssn.y, o1, o2);
      __bf16* dst = (__bf16*)sg.C + (size_t)row * sg.n + hd * D + i;
      dst[0] = (__bf16)o1;
      dst[half] = (__bf16)o2;
    }
  } else if constexpr (EPI == EPI_BF16 || EPI == EPI_F32 || EPI == EPI_F32_ADD) {
    const GemmSeg sg = g.seg[si];
    const bool vec = (sg.n & 3) == 0;    // whole 4-column runs are aligned
    constexpr int UNITS = MT * TW / 4;
#pragma unroll
    for (int u0 = 0; u0 < UNITS; u0 += 256) {
      const int u = u0 + tid;
      const int r = u / (TW / 4), cc = (u % (TW / 4)) * 4;
      const int c = cc & 31;
      const int row = m0 + r;
      const int col = (cg * CB + (cc >> 5)) * CW + c - sg.n0;   // column in the segment
      if (u >= UNITS || row >= g.M || c >= CW || col >= sg.n) continue;
      const f32x4 t = sum4(r, cc);
      const size_t o = (size_t)row * sg.n + col;
      if (vec && col + 4 <= sg.n) {
        if constexpr (EPI == EPI_BF16) {
          const bf16x2 lo = __builtin_convertvector(f32x2{t[0], t[1]}, bf16x2);
          const bf16x2 hi = __builtin_convertvector(f32x2{t[2], t[3]}, bf16x2);
          *(u32x2*)((__bf16*)sg.C + o) =
              u32x2{__builtin_bit_cast(uint32_t, lo), __builtin_bit_cast(uint32_t, hi)};
        } else if constexpr (EPI == EPI_F32_ADD) {
          f32x4 v = cpre ? cpre[u0 / 256] : *(const f32x4*)((float*)sg.C + o);
          v += t;
          *(f32x4*)((float*)sg.C + o) = v;
        } else {
          *(f32x4*)((float*)sg.C + o) = t;
        }
      } else {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          if (col + i >= sg.n) break;
          if constexpr (EPI == EPI_BF16) ((__bf16*)sg.C)[o + i] = (__bf16)t[i];
          else if constexpr (EPI == EPI_F32_ADD) ((float*)sg.C)[o + i] += t[i];
          else ((float*)sg.C)[o + i] = t[i];
        }
      }
    }
  } else if constexpr (EPI == EPI_SWIGLU) {
    // a unit: 4 gate columns of a block and the 4 up columns 16 further on
    const GemmSeg sg = g.seg[0];
    constexpr int UNITS = MT * CB * 4;
#pragma unroll
    for (int u0 = 0; u0 < UNITS; u0 += 256) {
      const int u = u0 + tid;
      const int r = u / (CB * 4), b = (u / 4) % CB, c = (u % 4) * 4;
      const int row = m0 + r;
      const int f = (cg * CB + b) * 16 + c;
      if (u >= UNITS || row >= g.M || f >= sg.n) continue;
      const f32x4 gt = sum4(r, b * 32 + c), upv = sum4(r, b * 32 + 16 + c);
      __bf16 act[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float v = (float)(__bf16)gt[i];        // gate and up, rounded as their own outputs
        const float o = (float)(__bf16)upv[i];
        act[i] = (__bf16)(v / (1.0f + expf(-v)) * o);
      }
      __bf16* dst = (__bf16*)sg.C + (size_t)row * sg.n + f;
      if ((sg.n & 3) == 0 && f + 4 <= sg.n) {
        *(u32x2*)dst = __builtin_bit_cast(u32x2, act);
      } else {
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (f + i < sg.n) dst[i] = act[i];
      }
    }
  } else {
    // EPI_ARGMAX: a unit is 8 columns of a block's row; the 4 units of a
    // block row are adjacent lanes (the key max is exact and the keys are
    // distinct, so the order of the max does not matter)
    bool nonfinite = false;
    constexpr int UNITS = MT * CB * 4;
    static_assert(UNITS % 256 == 0 || UNITS < 256, "whole lane quads");
#pragma unroll
    for (int u0 = 0; u0 < UNITS; u0 += 256) {
      const int u = u0 + tid;
      const int r = u / (CB * 4), b = (u / 4) % CB, q = u % 4;
      const int row = m0 + r;
      const int cb = cg * CB + b;
      const bool live = u < UNITS && row < g.M && cb < NB;
      uint64_t kv = 0;
      if (live) {
        const f32x4 t0 = sum4(r, b * 32 + q * 8), t1 = sum4(r, b * 32 + q * 8 + 4);
        const int col0 = cb * CW + q * 8;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const int col = col0 + i;
          const uint64_t k = col < g.ncols ? pack_logit(i < 4 ? t0[i] : t1[i - 4], col, nonfinite) : 0;
          kv = k > kv ? k : kv;
        }
      }
#pragma unroll
      for (int off = 1; off < 4; off <<= 1) {
        const uint32_t lo = __shfl_xor((uint32_t)kv, off);
        const uint32_t hi = __shfl_xor((uint32_t)(kv >> 32), off);
        const uint64_t o = ((uint64_t)hi << 32) | lo;
        kv = o > kv ? o : kv;
      }
      if (live && q == 0) g.part[(size_t)row * NB + cb] = kv;
    }
    if (__any(nonfinite) && lane == 0) set_err(g.err, DVS_ERR_NONFINITE);
  }
}

// Narrow blocks (CWT 16 or 8; few-row calls with few blocks, plain
// epilogues): only CWT weight rows are copied per chunk; the products still
// span 32 columns, of which the columns past CWT read stale LDS rows and are
// discarded -- each kept column's arithmetic is exactly the 32-column
// block's -- so the chip gets two or four times the workgroups and each
// streams a half or a quarter of the weights.
// CB: column blocks per wave (wider calls): each wave computes its split for
// CB adjacent 32-column blocks, so one A chunk feeds CB blocks' products
// (A is re-read once per CB blocks instead of once per block); per element
// the arithmetic is the single block's.
template <int MT, int CWT, int CB, int EPI, bool WK, bool FEW = false>
__global__ void __launch_bounds__(256, WK ? 1 : 2) gemm_ws_kernel(GemmArgs g) {
  constexpr int CW = CWT;                  // output columns per block (32, or 16 or 8: narrow)
  constexpr bool NARROW = CWT < 32;
  // k per chunk.  WK (calls of at most one workgroup per CU): 64, so that a
  // copy takes whole 128-byte lines of a row (copies of half lines, the
  // other half taken by the next chunk, moved 1.6x fewer useful bytes per
  // CU in a measurement), in rings of up to 144 KB.  Otherwise 32, in
  // rings that leave room for two workgroups per CU.
  constexpr int KC = WK ? 64 : 32;
  constexpr int RB = KC * 2;               // bytes of a row in a chunk
  constexpr int RPI = 1024 / RB;           // rows per 1 KB copy
  constexpr int WI = CW / RPI;             // weight copies per block and chunk
  static_assert(CW % RPI == 0, "a block's weight rows fill whole copies");
  constexpr int RG = MT / 32;              // 32-row groups per wave
  // ring stages per wave: WK three (two for tiles of two blocks); otherwise
  // four for the few-row calls (64 KB), three for 64-row tiles of one block
  // (72 KB), two for tiles of two blocks (64 KB)
  constexpr int NS = WK ? (CB == 2 ? 2 : 3) : (MT == 32 ? 4 : (CB == 2 ? 2 : 3));
  constexpr int WB = 32 * RB;              // W part of a block's chunk: 32 rows
  constexpr int CHB = CB * WB + MT * RB;   // chunk bytes (CB blocks' W rows, then A rows)
  // FEW: calls of at most RPI rows copy only the first RPI rows of A (one
  // copy per chunk); the tile's other rows read stale LDS and their outputs
  // are discarded
  constexpr int AI = FEW ? 1 : MT / RPI;   // A copies per chunk and wave
  constexpr int NPL = CB * WI + AI;        // 1 KB copies per chunk and wave
  constexpr int TW = CB * 32;              // tile width in the split sums
  static_assert(NPL * (NS - 1) < 64, "vmcnt range");
  static_assert(!NARROW || (MT == 32 && CB == 1), "narrow blocks serve few-row calls");
  static_assert(!NARROW || EPI == EPI_BF16 || EPI == EPI_F32 || EPI == EPI_F32_ADD,
                "narrow blocks take plain epilogues");
  static_assert(4 * NS * CHB >= GK_SPLITS * MT * TW * 4, "the split sums reuse the rings");
  __shared__ __attribute__((aligned(1024))) char s_ring[4 * NS * CHB];
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l32 = lane & 31, hh = lane >> 5;
  const int NB = (g.ncols + CW - 1) / CW;  // blocks
  const int NG = (NB + CB - 1) / CB;       // groups of CB blocks
  // XCD-aware order: groups b, b + 8, b + 16, ... share an XCD; the row
  // tiles of one group are consecutive among them
  const int x = blockIdx.x & 7, j = blockIdx.x >> 3;
  const int cg = (j / g.n_rt) * 8 + x, rt = j % g.n_rt;
  if (cg >= NG) return;
  const int m0 = rt * MT;
  char* ring = s_ring + w * NS * CHB;

  // Copies: instruction i of a block's chunk moves 1 KB, RPI rows of RB
  // bytes; lane L takes row RPI*i + L/(RB/16) and 16-byte chunk
  // (L mod RB/16) ^ sw(row), sw(row) = (row / 2) & 7 for 128-byte rows and
  // (row / 4) & 3 for 64-byte rows, so LDS slot c of a row holds its chunk
  // c ^ sw(row): the 16 rows an MFMA operand read serves at once hit
  // distinct banks.  The blocks of a group lie in one segment (the host
  // checks it).
  const int crow = lane / (RB / 16), cchk = lane % (RB / 16);
  auto sw = [](int row) { return KC == 64 ? (row >> 1) & 7 : (row >> 2) & 3; };
  int si = 0;
  if (EPI != EPI_SWIGLU)
    while (si + 1 < g.nseg && cg * CB * CW >= g.seg[si + 1].n0) ++si;
  const bool rope = EPI == EPI_BF16 && g.rope_tab != nullptr && si < 2;
  f32x4 cpre[(MT * CB * 32 / 4 + 255) / 256];
  if constexpr (EPI == EPI_F32_ADD) ws_residual_prefetch<MT, CB, CW>(g, tid, m0, cg, si, cpre);
  const __bf16* wsrc[CB][WI];  // this lane's weight rows (block b, tile rows 8i + L/8)
#pragma unroll
  for (int b = 0; b < CB; ++b)
#pragma unroll
    for (int i = 0; i < WI; ++i) {
      const int cb = cg * CB + b, c0 = cb * CW;
      const int r = RPI * i + crow;
      const __bf16* base;
      bool valid;
      int rowi;
      if (EPI == EPI_SWIGLU) {
        rowi = cb * 16 + (r & 15);
        valid = rowi < g.seg[0].n;
        base = r < 16 ? g.seg[0].W : g.seg[1].W;
      } else {
        rowi = c0 - g.seg[si].n0 + r;
        if (rope) {
          // block bh of a head holds dims bh*P .. bh*P+P-1 and their
          // rotate-half partners D/2 + bh*P ..
          const int hd = rowi / g.rope_D, cp = rowi - hd * g.rope_D;
          const int bh = cp / CW, c = cp - bh * CW;
          rowi = hd * g.rope_D + (c < CW / 2 ? bh * (CW / 2) + c : g.rope_D / 2 + bh * (CW / 2) + c - CW / 2);
        }
        valid = rowi < g.seg[si].n;
        base = g.seg[si].W;
      }
      wsrc[b][i] = base + (size_t)(valid ? rowi : 0) * g.K + ((cchk ^ sw(r)) << 3);
    }
  const __bf16* asrc[AI];
#pragma unroll
  for (int i = 0; i < AI; ++i) {
    const int r = RPI * i + crow;
    asrc[i] = g.A + (size_t)min(m0 + r, g.M - 1) * g.K + ((cchk ^ sw(r)) << 3);
  }
  const int kq = g.K / GK_SPLITS;
  const int kw = w * kq;               // this wave's split
  const int nch = kq / KC;
  auto issue = [&](int t) {
    char* dst = ring + (t % NS) * CHB;
    const int k0 = kw + t * KC;
#pragma unroll
    for (int b = 0; b < CB; ++b)
#pragma unroll
      for (int i = 0; i < WI; ++i)
        __builtin_amdgcn_global_load_lds((const void*)(wsrc[b][i] + k0),
                                         (__attribute__((address_space(3))) void*)(dst + b * WB + i * 1024), 16, 0, 0);
#pragma unroll
    for (int i = 0; i < AI; ++i)
      __builtin_amdgcn_global_load_lds((const void*)(asrc[i] + k0),
                                       (__attribute__((address_space(3))) void*)(dst + CB * WB + i * 1024), 16, 0, 0);
  };

  f32x16 acc[RG][CB];
#pragma unroll
  for (int a = 0; a < RG; ++a)
#pragma unroll
    for (int b = 0; b < CB; ++b) acc[a][b] = f32x16{};
  static_for<0, NS - 1>([&](auto c) {
    if (decltype(c)::value < nch) issue(decltype(c)::value);
  });
  // chunk t complete while the `later` chunks after it may still be in flight
  auto wait_chunk = [&](int later) {
    static_for<0, NS>([&](auto c) {
      constexpr int n = NS - 1 - decltype(c)::value;
      if (later == n) ws_wait_vmcnt<n * NPL>();
    });
  };
  for (int t = 0; t < nch; ++t) {
    if (t + NS - 1 < nch) issue(t + NS - 1);
    wait_chunk(min(NS - 1, nch - 1 - t));
    const char* src = ring + (t % NS) * CHB;
    // every operand of the chunk from LDS first, then the products
    bf16x8 bw[KC / 16][CB], ba[KC / 16][RG];
#pragma unroll
    for (int ks = 0; ks < KC / 16; ++ks) {
      const int q = 2 * ks + hh;   // the lane's 16-byte chunk of the row
#pragma unroll
      for (int b = 0; b < CB; ++b)
        bw[ks][b] = *(const bf16x8*)(src + b * WB + l32 * RB + ((q ^ sw(l32)) << 4));
#pragma unroll
      for (int a = 0; a < RG; ++a) {
        const int r = a * 32 + l32;
        ba[ks][a] = *(const bf16x8*)(src + CB * WB + r * RB + ((q ^ sw(r)) << 4));
      }
    }
    // every read issued before the first product: the fragments pass
    // through an empty asm that the products depend on (left to itself the
    // scheduler interleaves reads and products and waits for each in turn)
#pragma unroll
    for (int ks = 0; ks < KC / 16; ++ks) {
#pragma unroll
      for (int b = 0; b < CB; ++b) asm volatile("" : "+v"(bw[ks][b]));
#pragma unroll
      for (int a = 0; a < RG; ++a) asm volatile("" : "+v"(ba[ks][a]));
    }
#pragma unroll
    for (int ks = 0; ks < KC / 16; ++ks)
#pragma unroll
      for (int a = 0; a < RG; ++a)
#pragma unroll
        for (int b = 0; b < CB; ++b)
          acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ba[ks][a], bw[ks][b], acc[a][b], 0, 0, 0);
  }

  // splits in order through LDS (the rings are free once every wave is done);
  // rows of W past the segment end were read from row 0: their columns are 0
  __syncthreads();
  float* s_red = (float*)s_ring;
#pragma unroll
  for (int b = 0; b < CB; ++b) {
    const int cb = cg * CB + b, c0 = cb * CW;
    bool wvalid;
    if (EPI == EPI_SWIGLU) wvalid = cb * 16 + (l32 & 15) < g.seg[0].n;
    else wvalid = l32 < CW && c0 - g.seg[si].n0 + l32 < g.seg[si].n;
#pragma unroll
    for (int a = 0; a < RG; ++a)
#pragma unroll
      for (int i = 0; i < 16; ++i)
        s_red[w * (MT * TW) + (a * 32 + 8 * (i >> 2) + 4 * hh + (i & 3)) * TW + b * 32 + l32] =
            wvalid ? acc[a][b][i] : 0.f;
  }
  __syncthreads();
  ws_epilogue<MT, CB, CW, EPI, GK_SPLITS>(g, s_red, tid, lane, m0, cg, si, NB, rope,
                                         EPI == EPI_F32_ADD ? cpre : nullptr);
}

// gemm_ns_kernel<EPI, MT, NS>: the weight-streaming GEMM with the waves
// split over columns instead of K.  Workgroup = 4 waves = one (row tile of
// MT rows, group of 4 32-column blocks); wave w computes block w for all of
// K, keeping the four splits' sums apart (acc[s] is the in-order MFMA
// accumulation over split s's K range, exactly gemm_ws_kernel's p_s), and
// adds them in order at the end, so every output element is bit-identical
// to gemm_ws_kernel's.  The A chunk (MT rows x 64 k, whole 128-byte lines)
// is copied once per workgroup and read by all four waves, so A is re-read
// once per 128 output columns; each wave copies its block's weight rows.
// MT = 64 with a 3-stage ring of 24 KB stages (72 KB) leaves room for two
// workgroups per CU.  Used for the 64-row LM head (top-1 or fp32 logits):
// 14% faster there; for gate|up (256 workgroups, one per CU, each walking
// all of K with a barrier per chunk) it was slower than gemm_ws_kernel at
// 64 or 32 rows and three or four stages.
constexpr int NS_BLOCKS = 4;   // 32-column blocks per workgroup
template <int EPI, int MT, int NS>
__global__ void __launch_bounds__(256, NS * (MT * 128 + NS_BLOCKS * 4096) <= 81920 ? 2 : 1)
gemm_ns_kernel(GemmArgs g) {
  constexpr int RG = MT / 32, CW = 32, KC = 64, RB = KC * 2;
  constexpr int AB = MT * RB;                   // A part of a stage: 4 or 8 KB
  constexpr int WB = 32 * RB;                   // one block's weight rows: 4 KB
  constexpr int STB = AB + NS_BLOCKS * WB;
  constexpr int TW = NS_BLOCKS * 32;
  constexpr int AI = MT / 32;                   // A copies per wave and chunk (MT/8 rows-copies over 4 waves)
  constexpr int NPL = AI + 4;                   // 1 KB copies per wave and chunk (A rows, own W)
  static_assert(NS * STB >= MT * TW * 4, "the summed tile reuses the ring");
  __shared__ __attribute__((aligned(1024))) char s_ring[NS * STB];
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l32 = lane & 31, hh = lane >> 5;
  const int NB = (g.ncols + CW - 1) / CW;
  const int NG = (NB + NS_BLOCKS - 1) / NS_BLOCKS;
  // XCD-aware order, as in gemm_ws_kernel
  const int x = blockIdx.x & 7, j = blockIdx.x >> 3;
  const int cg = (j / g.n_rt) * 8 + x, rt = j % g.n_rt;
  if (cg >= NG) return;
  const int m0 = rt * MT;

  // copies (whole lines): 8 rows of 128 bytes per 1 KB instruction, lane L
  // takes row 8i + L/8 and 16-byte chunk (L & 7) ^ sw(row)
  const int crow = lane >> 3, cchk = lane & 7;
  auto sw = [](int row) { return (row >> 1) & 7; };
  int si = 0;
  if (EPI != EPI_SWIGLU)
    while (si + 1 < g.nseg && cg * NS_BLOCKS * CW >= g.seg[si + 1].n0) ++si;
  const int cb = cg * NS_BLOCKS + w;            // this wave's block
  const __bf16* wsrc[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int r = 8 * i + crow;
    const __bf16* base;
    bool valid;
    int rowi;
    if (EPI == EPI_SWIGLU) {
      rowi = cb * 16 + (r & 15);
      valid = rowi < g.seg[0].n;
      base = r < 16 ? g.seg[0].W : g.seg[1].W;
    } else {
      rowi = cb * CW - g.seg[si].n0 + r;
      valid = rowi < g.seg[si].n;
      base = g.seg[si].W;
    }
    wsrc[i] = base + (size_t)(valid ? rowi : 0) * g.K + ((cchk ^ sw(r)) << 3);
  }
  const __bf16* asrc[AI];                       // A rows 8(AI w + i) + L/8
#pragma unroll
  for (int i = 0; i < AI; ++i) {
    const int r = 8 * (AI * w + i) + crow;
    asrc[i] = g.A + (size_t)min(m0 + r, g.M - 1) * g.K + ((cchk ^ sw(r)) << 3);
  }
  const int nch = g.K / KC;                     // a multiple of 4 (K % 256 == 0)
  const int cps = nch / GK_SPLITS;              // chunks per split
  auto issue = [&](int t) {
    char* stage = s_ring + (t % NS) * STB;
    const int k0 = t * KC;
#pragma unroll
    for (int i = 0; i < AI; ++i)
      __builtin_amdgcn_global_load_lds((const void*)(asrc[i] + k0),
                                       (__attribute__((address_space(3))) void*)(stage + (AI * w + i) * 1024), 16, 0, 0);
#pragma unroll
    for (int i = 0; i < 4; ++i)
      __builtin_amdgcn_global_load_lds((const void*)(wsrc[i] + k0),
                                       (__attribute__((address_space(3))) void*)(stage + AB + w * WB + i * 1024), 16, 0, 0);
  };
  auto wait_chunk = [&](int later) {
    static_for<0, NS>([&](auto c) {
      constexpr int n = NS - 1 - decltype(c)::value;
      if (later == n) ws_wait_vmcnt<n * NPL>();
    });
  };

  f32x16 acc[GK_SPLITS][RG];
#pragma unroll
  for (int sp = 0; sp < GK_SPLITS; ++sp)
#pragma unroll
    for (int a = 0; a < RG; ++a) acc[sp][a] = f32x16{};
  static_for<0, NS - 1>([&](auto c) {
    if (decltype(c)::value < nch) issue(decltype(c)::value);
  });
  static_for<0, GK_SPLITS>([&](auto spc) {
    constexpr int sp = decltype(spc)::value;
    for (int tt = 0; tt < cps; ++tt) {
      const int t = sp * cps + tt;
      // this wave's copies of chunk t are in; the barrier makes everyone's
      // (the A rows are shared) and frees the slot chunk t-1 used
      wait_chunk(min(NS - 2, nch - 1 - t));
      __syncthreads();
      if (t + NS - 1 < nch) issue(t + NS - 1);
      const char* stage = s_ring + (t % NS) * STB;
      bf16x8 bw[KC / 16], ba[KC / 16][RG];
#pragma unroll
      for (int ks = 0; ks < KC / 16; ++ks) {
        const int q = 2 * ks + hh;
        bw[ks] = *(const bf16x8*)(stage + AB + w * WB + l32 * RB + ((q ^ sw(l32)) << 4));
#pragma unroll
        for (int a = 0; a < RG; ++a) {
          const int r = a * 32 + l32;
          ba[ks][a] = *(const bf16x8*)(stage + r * RB + ((q ^ sw(r)) << 4));
        }
      }
#pragma unroll
      for (int ks = 0; ks < KC / 16; ++ks) {
        asm volatile("" : "+v"(bw[ks]));
#pragma unroll
        for (int a = 0; a < RG; ++a) asm volatile("" : "+v"(ba[ks][a]));
      }
#pragma unroll
      for (int ks = 0; ks < KC / 16; ++ks)
#pragma unroll
        for (int a = 0; a < RG; ++a)
          acc[sp][a] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ba[ks][a], bw[ks], acc[sp][a], 0, 0, 0);
    }
  });

  // the splits in order, in registers; rows of W past the segment end were
  // read from row 0: their columns are 0.  The summed tile goes to LDS (the
  // ring is free once every wave is done) for the shared epilogue.
  bool wvalid;
  if (EPI == EPI_SWIGLU) wvalid = cb * 16 + (l32 & 15) < g.seg[0].n;
  else wvalid = cb * CW - g.seg[si].n0 + l32 < g.seg[si].n;
  __syncthreads();
  float* s_sum = (float*)s_ring;
#pragma unroll
  for (int a = 0; a < RG; ++a)
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      float t = 0.f;
#pragma unroll
      for (int sp = 0; sp < GK_SPLITS; ++sp) t += wvalid ? acc[sp][a][i] : 0.f;
      s_sum[(a * 32 + 8 * (i >> 2) + 4 * hh + (i & 3)) * TW + w * 32 + l32] = t;
    }
  __syncthreads();
  ws_epilogue<MT, NS_BLOCKS, CW, EPI, 1>(g, s_sum, tid, lane, m0, cg, si, NB, false);
}

// gemm_nk_kernel<EPI, SPLIT_M>: 64-row tiles with the four waves split 2 x
// 2, each over one K half, that is splits 2h and 2h+1, whose sums it keeps
// apart (each the in-order MFMA accumulation over its K range, exactly
// gemm_ws_kernel's p_s):
//   SPLIT_M = false: two 32-column blocks; wave w takes block w & 1 over K
//     half w >> 1, and the two waves of a half share its A chunk;
//   SPLIT_M = true: one 32-column block; wave w takes rows 32 (w & 1) ..
//     over K half w >> 1, and the two waves of a half share its weight
//     chunk (and the Q|K|V projection's rotary epilogue is available).
// Chunks are 64 k wide (whole 128-byte lines) in rings that leave room for
// two workgroups per CU (2 stages of 32 KB, or 3 of 24 KB).  The four split
// sums meet in LDS and the shared epilogue adds them in order:
// bit-identical to gemm_ws_kernel.
template <int EPI, bool SPLIT_M>
__global__ void __launch_bounds__(256, 2) gemm_nk_kernel(GemmArgs g) {
  constexpr int MT = 64, CW = 32, KC = 64, RB = KC * 2;
  constexpr int CB = SPLIT_M ? 1 : 2;           // blocks per tile
  constexpr int RG = SPLIT_M ? 1 : 2;           // 32-row groups per wave
  constexpr int AB = MT * RB;                   // one K half's A chunk: 8 KB
  constexpr int WB = 32 * RB;                   // one block's weight rows: 4 KB
  constexpr int STB = 2 * AB + 2 * CB * WB;     // A of both halves, W of (block, half)
  constexpr int NS = SPLIT_M ? 3 : 2;
  constexpr int TW = CB * 32;
  constexpr int AI = 4;                         // A copies per wave and chunk (32 rows)
  constexpr int WIW = SPLIT_M ? 2 : 4;          // W copies per wave and chunk
  constexpr int NPL = AI + WIW;
  static_assert(NS * STB >= GK_SPLITS * MT * TW * 4, "the split sums reuse the ring");
  static_assert(NS * STB <= 81920, "two workgroups per CU");
  __shared__ __attribute__((aligned(1024))) char s_ring[NS * STB];
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l32 = lane & 31, hh = lane >> 5;
  const int wl = w & 1, kh = w >> 1;            // block (or row group) and K half of this wave
  const int NB = (g.ncols + CW - 1) / CW;
  const int NG = (NB + CB - 1) / CB;
  const int x = blockIdx.x & 7, j = blockIdx.x >> 3;
  const int cg = (j / g.n_rt) * 8 + x, rt = j % g.n_rt;
  if (cg >= NG) return;
  const int m0 = rt * MT;
  const int crow = lane >> 3, cchk = lane & 7;
  auto sw = [](int row) { return (row >> 1) & 7; };
  int si = 0;
  if (EPI != EPI_SWIGLU)
    while (si + 1 < g.nseg && cg * CB * CW >= g.seg[si + 1].n0) ++si;
  const bool rope = EPI == EPI_BF16 && g.rope_tab != nullptr && si < 2;
  const int cb = cg * CB + (SPLIT_M ? 0 : wl);  // this wave's block
  // weight rows this wave copies: all 32 of its block (SPLIT_M = false), or
  // rows 16 (w & 1) .. + 15 of the shared block (SPLIT_M = true)
  const __bf16* wsrc[WIW];
#pragma unroll
  for (int i = 0; i < WIW; ++i) {
    const int r = (SPLIT_M ? 16 * wl : 0) + 8 * i + crow;
    const __bf16* base;
    bool valid;
    int rowi;
    if (EPI == EPI_SWIGLU) {
      rowi = cb * 16 + (r & 15);
      valid = rowi < g.seg[0].n;
      base = r < 16 ? g.seg[0].W : g.seg[1].W;
    } else {
      rowi = cb * CW - g.seg[si].n0 + r;
      if (rope) {
        // block bh of a head holds dims bh*16 .. bh*16+15 and their
        // rotate-half partners D/2 + bh*16 ..
        const int hd = rowi / g.rope_D, cp = rowi - hd * g.rope_D;
        const int bh = cp / CW, c = cp - bh * CW;
        rowi = hd * g.rope_D + (c < CW / 2 ? bh * (CW / 2) + c : g.rope_D / 2 + bh * (CW / 2) + c - CW / 2);
      }
      valid = rowi < g.seg[si].n;
      base = g.seg[si].W;
    }
    wsrc[i] = base + (size_t)(valid ? rowi : 0) * g.K + ((cchk ^ sw(r)) << 3);
  }
  const __bf16* asrc[AI];                       // A rows 32 (w & 1) + 8i + L/8 of half kh
#pragma unroll
  for (int i = 0; i < AI; ++i) {
    const int r = 32 * wl + 8 * i + crow;
    asrc[i] = g.A + (size_t)min(m0 + r, g.M - 1) * g.K + ((cchk ^ sw(r)) << 3);
  }
  const int kh0 = kh * (g.K / 2);               // first k of this wave's half
  const int nch = g.K / 2 / KC;                 // chunks per half (even: K % 256 == 0)
  const int cps = nch / 2;                      // chunks per split
  // stage layout: A of half 0, A of half 1, then W of (block or half) slots
  auto wslot = [&](int blk, int half) { return 2 * AB + (SPLIT_M ? half : 2 * half + blk) * WB; };
  auto issue = [&](int t) {
    char* stage = s_ring + (t % NS) * STB;
    const int k0 = kh0 + t * KC;
#pragma unroll
    for (int i = 0; i < AI; ++i)
      __builtin_amdgcn_global_load_lds((const void*)(asrc[i] + k0),
                                       (__attribute__((address_space(3))) void*)(stage + kh * AB + (4 * wl + i) * 1024), 16, 0, 0);
#pragma unroll
    for (int i = 0; i < WIW; ++i)
      __builtin_amdgcn_global_load_lds((const void*)(wsrc[i] + k0),
                                       (__attribute__((address_space(3))) void*)(stage + wslot(wl, kh) + ((SPLIT_M ? 2 * wl : 0) + i) * 1024), 16, 0, 0);
  };
  auto wait_chunk = [&](int later) {
    static_for<0, NS>([&](auto c) {
      constexpr int n = NS - 1 - decltype(c)::value;
      if (later == n) ws_wait_vmcnt<n * NPL>();
    });
  };
  f32x16 acc[2][RG];
#pragma unroll
  for (int sp = 0; sp < 2; ++sp)
#pragma unroll
    for (int a = 0; a < RG; ++a) acc[sp][a] = f32x16{};
  static_for<0, NS - 1>([&](auto c) {
    if (decltype(c)::value < nch) issue(decltype(c)::value);
  });
  static_for<0, 2>([&](auto spc) {
    constexpr int sp = decltype(spc)::value;
    for (int tt = 0; tt < cps; ++tt) {
      const int t = sp * cps + tt;
      // this wave's copies of chunk t are in; the barrier makes the
      // partner's, and frees the slot chunk t-1 used
      wait_chunk(min(NS - 2, nch - 1 - t));
      __syncthreads();
      if (t + NS - 1 < nch) issue(t + NS - 1);
      const char* stage = s_ring + (t % NS) * STB;
      const char* wsl = stage + wslot(wl, kh);
      bf16x8 bwf[KC / 16], ba[KC / 16][RG];
#pragma unroll
      for (int ks = 0; ks < KC / 16; ++ks) {
        const int q = 2 * ks + hh;
        bwf[ks] = *(const bf16x8*)(wsl + l32 * RB + ((q ^ sw(l32)) << 4));
#pragma unroll
        for (int a = 0; a < RG; ++a) {
          const int r = (SPLIT_M ? 32 * wl : a * 32) + l32;
          ba[ks][a] = *(const bf16x8*)(stage + kh * AB + r * RB + ((q ^ sw(r)) << 4));
        }
      }
#pragma unroll
      for (int ks = 0; ks < KC / 16; ++ks) {
        asm volatile("" : "+v"(bwf[ks]));
#pragma unroll
        for (int a = 0; a < RG; ++a) asm volatile("" : "+v"(ba[ks][a]));
      }
#pragma unroll
      for (int ks = 0; ks < KC / 16; ++ks)
#pragma unroll
        for (int a = 0; a < RG; ++a)
          acc[sp][a] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ba[ks][a], bwf[ks], acc[sp][a], 0, 0, 0);
    }
  });

  // the four split sums to LDS as planes [split][row][TW] (the ring is free
  // once every wave is done); rows of W past the segment end were read from
  // row 0: their columns are 0
  bool wvalid;
  if (EPI == EPI_SWIGLU) wvalid = cb * 16 + (l32 & 15) < g.seg[0].n;
  else wvalid = cb * CW - g.seg[si].n0 + l32 < g.seg[si].n;
  __syncthreads();
  float* s_red = (float*)s_ring;
#pragma unroll
  for (int sp = 0; sp < 2; ++sp)
#pragma unroll
    for (int a = 0; a < RG; ++a)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int row = (SPLIT_M ? 32 * wl : a * 32) + 8 * (i >> 2) + 4 * hh + (i & 3);
        s_red[(2 * kh + sp) * (MT * TW) + row * TW + (SPLIT_M ? 0 : wl * 32) + l32] =
            wvalid ? acc[sp][a][i] : 0.f;
      }
  __syncthreads();
  ws_epilogue<MT, CB, CW, EPI, GK_SPLITS>(g, s_red, tid, lane, m0, cg, si, NB, rope);
}

// Top-1 of each row from its column blocks' packed (key, index) maxima: one
// workgroup per row, every load of a thread in flight at once (a clamped
// index repeats the last block, which leaves the maximum unchanged), a
// 64-bit max over the lanes and then the waves; the lowest index wins among
// equal maxima; a row whose values were all NaN gives 0.
__global__ void __launch_bounds__(256) argmax_rows_kernel(const uint64_t* __restrict__ part, int M,
                                                          int NB, int32_t* __restrict__ out) {
  __shared__ uint64_t s_b[4];
  const int row = blockIdx.x, tid = threadIdx.x, lane = tid & 63;
  if (row >= M) return;
  const uint64_t* p = part + (size_t)row * NB;
  uint64_t b = 0;
  for (int i0 = 0; i0 < NB; i0 += 256 * 8) {
    uint64_t v[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) v[j] = p[min(i0 + tid + 256 * j, NB - 1)];
#pragma unroll
    for (int j = 0; j < 8; ++j) b = v[j] > b ? v[j] : b;
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    const uint32_t lo = __shfl_xor((uint32_t)b, off);
    const uint32_t hi = __shfl_xor((uint32_t)(b >> 32), off);
    const uint64_t o = ((uint64_t)hi << 32) | lo;
    b = o > b ? o : b;
  }
  if (lane == 0) s_b[tid >> 6] = b;
  __syncthreads();
  if (tid == 0) {
    b = s_b[0];
#pragma unroll
    for (int i = 1; i < 4; ++i) b = s_b[i] > b ? s_b[i] : b;
    out[row] = b == 0 ? 0 : 0x7fffffff - (int)(uint32_t)(b & 0xffffffffu);
  }
}

// ---------------------------------------------------------------------------
// gemm_rt_kernel<MT>: C[M, N] = A[M, K] W[N, K]^T for long calls, tiles of MT
// rows x 128 columns staged through LDS; all KS splits of a tile in one
// workgroup, each split's product added to a running sum in registers.
//
// Waves: MT = 32 -> 1 x 4 (each wave 32 rows x 32 columns); MT >= 64 ->
// 2 x 2 (each wave MT/2 rows x 64 columns).  Per 64-wide K chunk all 256
// threads copy the A tile (MT x 64) and the W tile (128 x 64) into a
// double-buffered LDS pair (16-byte chunks XOR-swizzled by row so the MFMA
// operand reads are conflict-free); the global loads of the next P - 1
// chunks are in flight while the current chunk is multiplied.
// ---------------------------------------------------------------------------
constexpr int RT_NT = 128;   // columns per tile
constexpr int RT_KC = 64;    // K per LDS chunk

// SPLITS = false: one logical split only (KS == 1), no running sum kept.
template <int MT, bool SPLITS>
__global__ void __launch_bounds__(256, 1) gemm_rt_kernel(
    const __bf16* __restrict__ A, const __bf16* __restrict__ W, int M, int N, int K, void* C,
    int c_f32, int accumulate, int KS, uint64_t* __restrict__ part, int32_t* err) {
  constexpr bool WIDE = MT >= 64;
  constexpr int RG = WIDE ? MT / 64 : 1;   // 32-row groups per wave
  constexpr int CG = WIDE ? 2 : 1;         // 32-column groups per wave
  constexpr int A_LD = MT * RT_KC / 8 / 256;      // 16-byte A chunks per thread per K chunk
  constexpr int W_LD = RT_NT * RT_KC / 8 / 256;   // 16-byte W chunks per thread per K chunk
  static_assert(A_LD >= 1 && W_LD >= 1, "tile / threads");
  __shared__ __attribute__((aligned(16))) char s_a[2][MT * RT_KC * 2];
  __shared__ __attribute__((aligned(16))) char s_w[2][RT_NT * RT_KC * 2];

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int l32 = lane & 31, hh = lane >> 5;
  const int NBK = (N + RT_NT - 1) / RT_NT;
  const int nb = blockIdx.x % NBK;
  const int rt = blockIdx.x / NBK;
  const int n0 = nb * RT_NT;
  const int m0 = rt * MT;
  const int kc = K / KS;
  const int wr = WIDE ? (w >> 1) : 0, wc = WIDE ? (w & 1) : w;
  const int row_w = wr * (MT / (WIDE ? 2 : 1));   // first tile row of the wave
  const int col_w = wc * (CG * 32);               // first tile column of the wave

  // global -> register staging of K chunks, P - 1 chunks ahead of the one
  // being multiplied (ring slot = chunk index mod P)
  constexpr int P = MT <= 64 ? 4 : 2;
  u32x4 ra[P][A_LD], rw[P][W_LD];
  auto load_chunk = [&](int k0, u32x4 (&xa)[A_LD], u32x4 (&xw)[W_LD]) {
#pragma unroll
    for (int j = 0; j < A_LD; ++j) {
      const int idx = tid + j * 256;
      const int r = idx >> 3, c = idx & 7;
      // unconditional loads (rows past the end re-read the last row and are
      // zeroed after), so that the wait counts stay exact across the ring
      const int mrow = m0 + r;
      const u32x4 x = *(const u32x4*)(A + (size_t)min(mrow, M - 1) * K + k0 + c * 8);
      xa[j] = mrow < M ? x : u32x4{0, 0, 0, 0};
    }
#pragma unroll
    for (int j = 0; j < W_LD; ++j) {
      const int idx = tid + j * 256;
      const int r = idx >> 3, c = idx & 7;
      const int n = n0 + r;
      const u32x4 x = *(const u32x4*)(W + (size_t)min(n, N - 1) * K + k0 + c * 8);
      xw[j] = n < N ? x : u32x4{0, 0, 0, 0};
    }
  };
  auto store_chunk = [&](int buf, const u32x4 (&xa)[A_LD], const u32x4 (&xw)[W_LD]) {
#pragma unroll
    for (int j = 0; j < A_LD; ++j) {
      const int idx = tid + j * 256;
      const int r = idx >> 3, c = idx & 7;
      *(u32x4*)(s_a[buf] + r * 128 + ((c ^ (r & 7)) << 4)) = xa[j];
    }
#pragma unroll
    for (int j = 0; j < W_LD; ++j) {
      const int idx = tid + j * 256;
      const int r = idx >> 3, c = idx & 7;
      *(u32x4*)(s_w[buf] + r * 128 + ((c ^ (r & 7)) << 4)) = xw[j];
    }
  };

  f32x16 acc[RG][CG], sum[SPLITS ? RG : 1][SPLITS ? CG : 1];
  if constexpr (SPLITS) {
#pragma unroll
    for (int a = 0; a < RG; ++a)
#pragma unroll
      for (int b = 0; b < CG; ++b) sum[a][b] = f32x16{};
  }

  const int nch = kc / RT_KC;
  const int total = KS * nch;
  auto chunk_k0 = [&](int t) { return (t / nch) * kc + (t % nch) * RT_KC; };
  static_for<0, P - 1>([&](auto c) {
    constexpr int i = decltype(c)::value;
    load_chunk(chunk_k0(min(i, total - 1)), ra[i], rw[i]);
  });
  store_chunk(0, ra[0], rw[0]);
  __syncthreads();
  // one chunk: acc reset at a split start, the next-but-(P-2) chunk's loads
  // (clamped to the last chunk: a harmless re-read), the products, the
  // ordered split sum, the next chunk into the other LDS buffer
  auto step = [&](int t, auto cs) {
    constexpr int sl = decltype(cs)::value;   // ring slot of chunk t
    const int ch = t % nch;
    if (ch == 0) {
#pragma unroll
      for (int a = 0; a < RG; ++a)
#pragma unroll
        for (int b = 0; b < CG; ++b) acc[a][b] = f32x16{};
    }
    load_chunk(chunk_k0(min(t + P - 1, total - 1)), ra[(sl + P - 1) % P], rw[(sl + P - 1) % P]);
    const char* sa = s_a[t & 1];
    const char* sw = s_w[t & 1];
#pragma unroll
    for (int ks = 0; ks < RT_KC / 16; ++ks) {
      const int ch16 = ks * 2 + hh;   // 16-byte chunk of the row holding this lane's 8 k values
      bf16x8 af[RG], bf[CG];
#pragma unroll
      for (int a = 0; a < RG; ++a) {
        const int r = row_w + a * 32 + l32;
        af[a] = *(const bf16x8*)(sa + r * 128 + ((ch16 ^ (r & 7)) << 4));
      }
#pragma unroll
      for (int b = 0; b < CG; ++b) {
        const int r = col_w + b * 32 + l32;
        bf[b] = *(const bf16x8*)(sw + r * 128 + ((ch16 ^ (r & 7)) << 4));
      }
#pragma unroll
      for (int a = 0; a < RG; ++a)
#pragma unroll
        for (int b = 0; b < CG; ++b)
          acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[a], bf[b], acc[a][b], 0, 0, 0);
    }
    if (SPLITS && ch == nch - 1) {   // split complete: ordered running sum
#pragma unroll
      for (int a = 0; a < RG; ++a)
#pragma unroll
        for (int b = 0; b < CG; ++b) sum[a][b] += acc[a][b];
    }
    store_chunk((t + 1) & 1, ra[(sl + 1) % P], rw[(sl + 1) % P]);
    __syncthreads();
  };
  // whole groups of P chunks keep the ring slots compile-time; the tail runs
  // the same steps one by one
  int t0 = 0;
  for (; t0 + P <= total; t0 += P) static_for<0, P>([&](auto c) { step(t0 + decltype(c)::value, c); });
  static_for<0, P - 1>([&](auto c) {
    if (t0 + decltype(c)::value < total) step(t0 + decltype(c)::value, c);
  });

  // element (a, b, i) of this lane: row m0 + row_w + 32a + 8(i>>2) + 4hh + (i&3),
  // column n0 + col_w + 32b + l32
  float* Cf = c_f32 ? (float*)C : nullptr;
  __bf16* Cb = c_f32 ? nullptr : (__bf16*)C;
  auto write_out = [&](f32x16 (&v)[RG][CG]) {
#pragma unroll
    for (int a = 0; a < RG; ++a)
#pragma unroll
      for (int b = 0; b < CG; ++b) {
        const int n = n0 + col_w + b * 32 + l32;
        float cur[16];
        if (Cf && accumulate) {
#pragma unroll
          for (int i = 0; i < 16; ++i) {
            const int mrow = m0 + row_w + a * 32 + 8 * (i >> 2) + 4 * hh + (i & 3);
            cur[i] = (mrow < M && n < N) ? Cf[(size_t)mrow * N + n] : 0.f;
          }
        }
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int mrow = m0 + row_w + a * 32 + 8 * (i >> 2) + 4 * hh + (i & 3);
          if (mrow >= M || n >= N) continue;
          const size_t o = (size_t)mrow * N + n;
          if (Cf) Cf[o] = accumulate ? cur[i] + v[a][b][i] : v[a][b][i];
          else Cb[o] = (__bf16)v[a][b][i];
        }
      }
  };
  // top-1 epilogue (part != NULL): per row and 32-column group the largest
  // value and its lowest index, packed as gemm_ws_kernel's EPI_ARGMAX; the 32
  // lanes of a lane half hold one row's 32 columns
  auto write_top1 = [&](f32x16 (&v)[RG][CG]) {
    const int NB = (N + 31) / 32;
    bool nonfinite = false;
#pragma unroll
    for (int a = 0; a < RG; ++a)
#pragma unroll
      for (int b = 0; b < CG; ++b) {
        const int n = n0 + col_w + b * 32 + l32;
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int mrow = m0 + row_w + a * 32 + 8 * (i >> 2) + 4 * hh + (i & 3);
          uint64_t kv = (mrow < M && n < N) ? pack_logit(v[a][b][i], n, nonfinite) : 0;
#pragma unroll
          for (int off = 16; off > 0; off >>= 1) {
            const uint32_t lo = __shfl_xor((uint32_t)kv, off);
            const uint32_t hi = __shfl_xor((uint32_t)(kv >> 32), off);
            const uint64_t o = ((uint64_t)hi << 32) | lo;
            kv = o > kv ? o : kv;
          }
          if (l32 == 0 && mrow < M) part[(size_t)mrow * NB + (n0 + col_w + b * 32) / 32] = kv;
        }
      }
    if (__any(nonfinite) && lane == 0) set_err(err, DVS_ERR_NONFINITE);
  };
  if constexpr (!SPLITS) {
    // 0 + p_0, as in the split paths (keeps the sign of a zero sum alike)
#pragma unroll
    for (int a = 0; a < RG; ++a)
#pragma unroll
      for (int b = 0; b < CG; ++b) acc[a][b] = f32x16{} + acc[a][b];
    if (part) write_top1(acc);
    else write_out(acc);
  } else {
    if (part) write_top1(sum);
    else write_out(sum);
  }
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
  size_t x, h, hsel, q, k, v, att, gate, up, act, logits, am, conf, nopen, blk, acc, lead, part,
      attn_ws, rope, total, attn_bytes, attn_counters;
};

// Rows per tile when all splits run in one workgroup (more than 32 rows):
// the largest tile that still gives 256 workgroups, else 32.
static int gemm_rows_per_tile(int M, int N) {
  const long long nb = (N + RT_NT - 1) / RT_NT;
  for (int mt = 256; mt >= 64; mt >>= 1)
    if (mt / 2 < M && nb * ((M + mt - 1) / mt) >= 256) return mt;
  return 32;
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
  L.conf = off; off += al(logit_rows * 4);
  L.nopen = off; off += al(4);
  L.blk = off; off += al(M * 4);
  L.acc = off; off += al((size_t)S * 4);
  L.lead = off; off += al((size_t)S * 4);
  // the LM head's per-column-block maxima (fused top-1)
  L.part = off; off += al(std::max(M, logit_rows) * (size_t)((m->vocab + 31) / 32) * 8);
  L.attn_bytes = dvs_attn_workspace_bytes(S, n_causal, n_mask, m->n_heads, m->n_kv_heads,
                                          m->head_dim, max_pages, chunk_keys, m->dtype);
  L.attn_counters = attn_counter_bytes(S, n_causal + n_mask, m->n_heads, m->n_kv_heads,
                                       m->head_dim, max_pages, chunk_keys, m->dtype);
  L.attn_ws = off; off += al(L.attn_bytes);
  // the step's rotary (cos, sin) table, for calls whose Q|K|V projection
  // takes the rotation in its epilogue (up to WS_MAX_ROWS rows)
  L.rope = off; off += al(M <= (size_t)WS_MAX_ROWS ? M * (m->head_dim / 2) * 16 : 0);
  L.total = off;
  return L;
}

template <int MT, int CWT, int CB, bool WK, bool FEW>
static void launch_ws_epi(const GemmArgs& g, dim3 gr, hipStream_t st) {
  const dim3 blk(256);
  switch (g.epi) {
    case EPI_BF16: hipLaunchKernelGGL((gemm_ws_kernel<MT, CWT, CB, EPI_BF16, WK, FEW>), gr, blk, 0, st, g); break;
    case EPI_F32: hipLaunchKernelGGL((gemm_ws_kernel<MT, CWT, CB, EPI_F32, WK, FEW>), gr, blk, 0, st, g); break;
    case EPI_F32_ADD: hipLaunchKernelGGL((gemm_ws_kernel<MT, CWT, CB, EPI_F32_ADD, WK, FEW>), gr, blk, 0, st, g); break;
    default:
      if constexpr (CWT == 32) {
        if (g.epi == EPI_SWIGLU) hipLaunchKernelGGL((gemm_ws_kernel<MT, 32, CB, EPI_SWIGLU, WK, FEW>), gr, blk, 0, st, g);
        else hipLaunchKernelGGL((gemm_ws_kernel<MT, 32, CB, EPI_ARGMAX, WK, FEW>), gr, blk, 0, st, g);
      }
      break;
  }
}

template <int MT, int CWT, int CB>
static void launch_ws_k(const GemmArgs& g, dim3 gr, bool wk, hipStream_t st) {
  if constexpr (CWT == 8) {
    // 8-column blocks: whole-line chunks only (one copy of 8 weight rows)
    if constexpr (MT == 32) {
      if (g.M <= 8) launch_ws_epi<MT, 8, CB, true, true>(g, gr, st);
      else launch_ws_epi<MT, 8, CB, true, false>(g, gr, st);
    }
    return;
  } else {
    if constexpr (MT == 32) {
      // calls whose rows fit one copy of A rows (8 rows in 64-k chunks, 16
      // in 32-k chunks)
      if (g.M <= (wk ? 8 : 16)) {
        if (wk) launch_ws_epi<MT, CWT, CB, true, true>(g, gr, st);
        else launch_ws_epi<MT, CWT, CB, false, true>(g, gr, st);
        return;
      }
    }
    if (wk) launch_ws_epi<MT, CWT, CB, true, false>(g, gr, st);
    else launch_ws_epi<MT, CWT, CB, false, false>(g, gr, st);
  }
}

static int launch_ws(GemmArgs& g, hipStream_t st) {
  const int MT = g.M <= 32 ? 32 : 64;
  // few-row calls with few 32-column blocks and a plain epilogue: narrow
  // blocks of 16 or 8 columns (more workgroups)
  const bool narrow = MT == 32 && (g.ncols + 31) / 32 < WS_NARROW_NB &&
                      (g.epi == EPI_BF16 || g.epi == EPI_F32 || g.epi == EPI_F32_ADD);
  g.n_rt = (g.M + MT - 1) / MT;
  // narrow calls whose 8-column blocks still fit one workgroup per CU take
  // 8-column blocks (whole-line chunks), else 16-column ones
  int cw = 32;
  if (narrow) cw = (long long)((g.ncols + 7) / 8) * g.n_rt <= device_cus() ? 8 : 16;
  if (narrow) {
    for (int i = 0; i < g.nseg; ++i)
      if (g.seg[i].n0 % cw) cw = 16;
  }
  const int NB = (g.ncols + cw - 1) / cw;
  // wider calls: CB blocks per wave while that still gives the chip enough
  // workgroups, and every segment starts on a group boundary
  int CB = 1;
  if (MT == 64) {
    auto groups_ok = [&](int cb) {
      for (int i = 0; i < g.nseg; ++i)
        if (g.seg[i].n0 % (32 * cb)) return false;
      return true;
    };
    if ((NB / 2) * g.n_rt >= WS_WIDE_MIN_WG && groups_ok(2)) CB = 2;
  }
  // 64-row calls with many 128-column groups and a top-1 or fp32 epilogue
  // (the LM head): the column-split kernel (one A chunk per four blocks)
  if (MT == 64 && !narrow && (g.epi == EPI_ARGMAX || g.epi == EPI_F32)) {
    const int NGn = (NB + NS_BLOCKS - 1) / NS_BLOCKS;
    bool ok = (long long)NGn * g.n_rt >= WS_WIDE_MIN_WG;
    for (int i = 0; i < g.nseg; ++i)
      if (g.seg[i].n0 % (32 * NS_BLOCKS)) ok = false;
    if (ok) {
      const long long gridn = (long long)((NGn + 7) / 8) * 8 * g.n_rt;
      DVS_CHECK_SUPPORTED(gridn < (1LL << 31), "draft_verify_step: GEMM grid too large");
      const dim3 grn((unsigned)gridn), blk(256);
      if (g.epi == EPI_ARGMAX) hipLaunchKernelGGL((gemm_ns_kernel<EPI_ARGMAX, 64, 3>), grn, blk, 0, st, g);
      else hipLaunchKernelGGL((gemm_ns_kernel<EPI_F32, 64, 3>), grn, blk, 0, st, g);
      return launch_status("draft_verify_step(gemm)");
    }
  }
  const int NG = (NB + CB - 1) / CB;
  const long long grid = (long long)((NG + 7) / 8) * 8 * g.n_rt;
  DVS_CHECK_SUPPORTED(grid < (1LL << 31), "draft_verify_step: GEMM grid too large");
  const dim3 gr((unsigned)grid);
  // calls of at most one workgroup per CU: whole-line chunks, deeper rings
  const bool wk = (long long)NG * g.n_rt <= device_cus();
  // 64-row calls of more than one workgroup per CU: whole-line chunks with
  // the waves split 2 x 2 (two blocks or two row groups, two K halves), so
  // that the rings still leave room for two workgroups per CU (gate|up
  // 20.8 -> 18.6 us per launch at 256 rows)
  if (MT == 64 && CB == 2 && !wk && g.epi == EPI_SWIGLU) {
    hipLaunchKernelGGL((gemm_nk_kernel<EPI_SWIGLU, false>), gr, dim3(256), 0, st, g);
    return launch_status("draft_verify_step(gemm)");
  }
  if (MT == 64 && CB == 1 && !wk && g.epi == EPI_BF16) {
    hipLaunchKernelGGL((gemm_nk_kernel<EPI_BF16, true>), gr, dim3(256), 0, st, g);
    return launch_status("draft_verify_step(gemm)");
  }
  if (cw == 8) launch_ws_k<32, 8, 1>(g, gr, wk, st);
  else if (narrow) launch_ws_k<32, 16, 1>(g, gr, wk, st);
  else if (MT == 32) launch_ws_k<32, 32, 1>(g, gr, wk, st);
  else if (CB == 2) launch_ws_k<64, 32, 2>(g, gr, wk, st);
  else launch_ws_k<64, 32, 1>(g, gr, wk, st);
  return launch_status("draft_verify_step(gemm)");
}

// gemm_ws_kernel serves a call when it computes the same splits as
// gemm_rt_kernel would (bf16, K a multiple of 256) and the rows are few.
static bool use_ws(int dtype, int M, int K) {
  return dtype == DVS_BF16 && K % (64 * GK_SPLITS) == 0 && M <= WS_MAX_ROWS;
}

// C = A W^T (or C += for the fp32 residual).  `c_f32` selects an fp32 output
// for bf16 models (residual stream, logits); fp32 models always write fp32.
static int gemm(const StepLayout& L, char* ws, int dtype, const void* A, const void* W, int M,
                int N, int K, void* C, int c_f32, int accumulate, hipStream_t st) {
  (void)L; (void)ws;
  const int waves = (N + 31) / 32;
  const int blocks = (waves + 3) / 4;
  if (use_ws(dtype, M, K)) {
    GemmArgs g{};
    g.A = (const __bf16*)A; g.M = M; g.K = K; g.ncols = N;
    g.seg[0] = GemmSeg{(const __bf16*)W, C, 0, N};
    g.nseg = 1;
    g.epi = c_f32 ? (accumulate ? EPI_F32_ADD : EPI_F32) : EPI_BF16;
    return launch_ws(g, st);
  }
  if (dtype == DVS_BF16 && K % 64 == 0) {
    const int ksp = gemm_ksplit(K);
    int mt = M <= 32 ? 32 : gemm_rows_per_tile(M, N);
    if (mt == 256 && ksp > 1) mt = 128;   // the 256-row tile keeps no running split sum
    const int nb = (N + RT_NT - 1) / RT_NT;
    const long long grid = (long long)nb * ((M + mt - 1) / mt);
    DVS_CHECK_SUPPORTED(grid < (1LL << 31), "draft_verify_step: GEMM grid too large");
    const dim3 g((unsigned)grid), blk(256);
    const __bf16* a = (const __bf16*)A;
    const __bf16* wt = (const __bf16*)W;
    switch (mt) {
      case 256: hipLaunchKernelGGL((gemm_rt_kernel<256, false>), g, blk, 0, st, a, wt, M, N, K, C, c_f32, accumulate, ksp, nullptr, nullptr); break;
      case 128: hipLaunchKernelGGL((gemm_rt_kernel<128, true>), g, blk, 0, st, a, wt, M, N, K, C, c_f32, accumulate, ksp, nullptr, nullptr); break;
      case 64: hipLaunchKernelGGL((gemm_rt_kernel<64, true>), g, blk, 0, st, a, wt, M, N, K, C, c_f32, accumulate, ksp, nullptr, nullptr); break;
      default: hipLaunchKernelGGL((gemm_rt_kernel<32, true>), g, blk, 0, st, a, wt, M, N, K, C, c_f32, accumulate, ksp, nullptr, nullptr); break;
    }
  } else if (dtype == DVS_BF16)
    hipLaunchKernelGGL(gemm_bf16_kernel, dim3(blocks), dim3(256), 0, st, (const __bf16*)A,
                       (const __bf16*)W, M, N, K, C, c_f32, accumulate);
  else
    hipLaunchKernelGGL(gemm_f32_kernel, dim3(blocks), dim3(256), 0, st, (const float*)A,
                       (const float*)W, M, N, K, (float*)C, accumulate);
  return launch_status("draft_verify_step(gemm)");
}

// LM head with the top-1 fused into its epilogue (no logits in memory), for
// the rows in h; the result is argmax_kernel's (same values, same order).
static int lm_head_top1(const dvs_model* m, const StepLayout& L, char* ws, const void* h, int M,
                        int32_t* am, int32_t* err, hipStream_t st) {
  GemmArgs g{};
  g.A = (const __bf16*)h; g.M = M; g.K = m->hidden; g.ncols = m->vocab;
  g.seg[0] = GemmSeg{(const __bf16*)m->lm_head, nullptr, 0, m->vocab};
  g.nseg = 1;
  g.epi = EPI_ARGMAX;
  g.part = (uint64_t*)(ws + L.part);
  g.err = err;
  // (calls of more than 32 rows take two 32-column blocks per wave, so each
  // A chunk serves 64 columns)
  int rc = launch_ws(g, st);
  if (rc) return rc;
  const int NB = (m->vocab + 31) / 32;
  hipLaunchKernelGGL(argmax_rows_kernel, dim3((unsigned)M), dim3(256), 0, st, g.part,
                     M, NB, am);
  return launch_status("draft_verify_step(lm head top-1)");
}

// The decoder stack on the rows in x (fp32, [M, hidden]); leaves the final
// RMSNorm output in h.  The window is (n_causal, n_mask) rows per sequence.
template <typename T>
// first_norm_done: the embedding launch already wrote layer 0's norm to h
static int forward_layers(const dvs_model* m, const dvs_state* st, int n_causal, int n_mask,
                          int chunk_keys, const StepLayout& L, char* ws, hipStream_t stream,
                          int group = 0, bool first_norm_done = false) {
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
  const double log2_theta = log2((double)m->rope_theta);
  const bool rope_fused = use_ws(dt, M, H) && D % 32 == 0;
  const int nw = (int)(L.attn_counters / 4);
  if (rope_fused) {
    // the rotary table, with the counters' clearing in the same launch
    const int zb = (nw + 255) / 256;
    hipLaunchKernelGGL(rope_table_kernel, dim3(zb + (M * (D / 2) + 255) / 256), dim3(256), 0, stream,
                       (double2*)(ws + L.rope), M, R, D, log2_theta, st->kv_len, n_causal, n_mask,
                       group, (int32_t*)(ws + L.attn_ws), nw, zb);
    if ((rc = launch_status("draft_verify_step(rope table)"))) return rc;
  } else if (nw) {
    hipLaunchKernelGGL(zero_words_kernel, dim3((nw + 255) / 256), dim3(256), 0, stream,
                       (int32_t*)(ws + L.attn_ws), nw);
  }
  for (int l = 0; l < m->n_layers; ++l) {
    const dvs_layer& ly = m->layers[l];
    if (l > 0 || !first_norm_done)
      hipLaunchKernelGGL(rmsnorm_kernel<T>, dim3(M), dim3(256), 0, stream, x, (const T*)ly.g_attn, H,
                         m->rms_eps, h);
    if (use_ws(dt, M, H)) {
      // Q, K and V in one launch (the same splits as three separate calls)
      GemmArgs g{};
      g.A = (const __bf16*)h; g.M = M; g.K = H; g.ncols = (Hq + 2 * Hkv) * D;
      g.seg[0] = GemmSeg{(const __bf16*)ly.wq, q, 0, Hq * D};
      g.seg[1] = GemmSeg{(const __bf16*)ly.wk, k, Hq * D, Hkv * D};
      g.seg[2] = GemmSeg{(const __bf16*)ly.wv, v, (Hq + Hkv) * D, Hkv * D};
      g.nseg = 3;
      g.epi = EPI_BF16;
      // the rotary embedding in the epilogue (heads split evenly into
      // 16- or 32-column blocks)
      if (rope_fused) {
        g.rope_tab = (const double2*)(ws + L.rope);
        g.rope_D = D;
      }
      if ((rc = launch_ws(g, stream))) return rc;
    } else {
      if ((rc = gemm(L, ws, dt, h, ly.wq, M, Hq * D, H, q, 0, 0, stream))) return rc;
      if ((rc = gemm(L, ws, dt, h, ly.wk, M, Hkv * D, H, k, 0, 0, stream))) return rc;
      if ((rc = gemm(L, ws, dt, h, ly.wv, M, Hkv * D, H, v, 0, 0, stream))) return rc;
    }
    if (!rope_fused) {
      const long long nqk = (long long)M * (Hq + Hkv) * (D / 2);
      hipLaunchKernelGGL(rope_kernel<T>, dim3((unsigned)((nqk + 255) / 256)), dim3(256), 0, stream,
                         q, Hq, k, Hkv, M, R, D, log2_theta, st->kv_len, n_causal, n_mask, group);
      if ((rc = launch_status("draft_verify_step(rope)"))) return rc;
    }
    rc = attn_hybrid_block_grouped(q, k, v, ly.k_pool, ly.v_pool, st->page_table, st->kv_len, S,
                                   n_causal, n_mask, group, Hq, Hkv, D, st->max_pages,
                                   st->num_pool_pages, (float)(1.0 / sqrt((double)D)), dt,
                                   chunk_keys, att, st->err_word, ws + L.attn_ws, L.attn_bytes,
                                   stream);
    if (rc) return rc;
    if ((rc = gemm(L, ws, dt, att, ly.wo, M, H, Hq * D, x, 1, 1, stream))) return rc;
    if (m->ffn > 0) {
      hipLaunchKernelGGL(rmsnorm_kernel<T>, dim3(M), dim3(256), 0, stream, x, (const T*)ly.g_mlp,
                         H, m->rms_eps, h);
      if (use_ws(dt, M, H)) {
        // gate and up in one launch, silu(gate) * up in its epilogue
        GemmArgs g{};
        g.A = (const __bf16*)h; g.M = M; g.K = H; g.ncols = 32 * ((m->ffn + 15) / 16);
        g.seg[0] = GemmSeg{(const __bf16*)ly.w_gate, act, 0, m->ffn};
        g.seg[1] = GemmSeg{(const __bf16*)ly.w_up, nullptr, 0, m->ffn};
        g.nseg = 2;
        g.epi = EPI_SWIGLU;
        if ((rc = launch_ws(g, stream))) return rc;
      } else {
        if ((rc = gemm(L, ws, dt, h, ly.w_gate, M, m->ffn, H, gate, 0, 0, stream))) return rc;
        if ((rc = gemm(L, ws, dt, h, ly.w_up, M, m->ffn, H, up, 0, 0, stream))) return rc;
        const long long n = (long long)M * m->ffn;
        hipLaunchKernelGGL(silu_mul_kernel<T>, dim3((unsigned)((n + 255) / 256)), dim3(256), 0,
                           stream, gate, up, n, act);
        if ((rc = launch_status("draft_verify_step(silu)"))) return rc;
      }
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
                    int32_t* argmax_out, int32_t* accept_out, hipStream_t stream,
                    int group = 0) {
  const int S = st->S, R = n_causal + n_mask, M = S * R;
  float* logits = logits_out ? logits_out : (float*)(ws + L.logits);
  int32_t* am = argmax_out ? argmax_out : (int32_t*)(ws + L.am);
  int32_t* acc = accept_out ? accept_out : (int32_t*)(ws + L.acc);
  // bf16 rows of at most 2048: the embedding launch also writes layer 0's
  // norm (rms_row_held, the same bits as the norm launch it replaces)
  const bool embed_norm = m->dtype == DVS_BF16 && m->hidden <= 2048;
  hipLaunchKernelGGL(embed_rows_kernel<T>, dim3(M), dim3(256), 0, stream, (const T*)m->embed,
                     m->hidden, m->vocab, R, n_causal, st->boundary, st->draft, st->draft_width,
                     nullptr, 0, (float*)(ws + L.x),
                     embed_norm ? (const T*)m->layers[0].g_attn : nullptr, m->rms_eps,
                     embed_norm ? (T*)(ws + L.h) : nullptr);
  int rc;
  if ((rc = launch_status("draft_verify_step(embed)"))) return rc;
  if ((rc = forward_layers<T>(m, st, n_causal, n_mask, chunk_keys, L, ws, stream, group, embed_norm)))
    return rc;
  if (!logits_out && use_ws(m->dtype, M, m->hidden)) {
    // top-1 in the LM head's epilogue: the logits never reach memory
    if ((rc = lm_head_top1(m, L, ws, ws + L.h, M, am, st->err_word, stream))) return rc;
  } else {
    if ((rc = gemm(L, ws, m->dtype, ws + L.h, m->lm_head, M, m->vocab, m->hidden, logits, 1, 0,
                   stream)))
      return rc;
    rc = argmax_accept(logits, DVS_F32, S, R, m->vocab, n_causal, st->draft, st->draft_width, am,
                       nullptr, st->err_word, stream);
    if (rc) return rc;
  }
  // acceptance inside the commit kernel
  return accept_commit(S, n_causal, n_mask, group, am, acc, st->kv_len, st->page_table, st->num_pages,
                       st->max_pages, st->free_stack, st->free_top, st->num_pool_pages,
                       st->boundary, st->draft, st->draft_width, st->out_tokens, st->out_count,
                       st->max_new, st->eos_id, st->finished, st->err_word, stream);
}

// The paper's two-forward round: draft forward over [x0, [M] x B], then a
// causal verify forward over [a0, d_1..d_B] from position L + 1 (its K/V
// overwrites the draft's mask-row slots), then acceptance against d_1..d_B
// and the commit of a0, d_1..d_A, a_{A+1}.  Both forwards carry B + 1 rows.
template <typename T>
static int run_round(const dvs_model* m, const dvs_state* st, int B, int chunk_keys,
                     const StepLayout& L, char* ws, float* logits_out, int32_t* argmax_out,
                     int32_t* accept_out, hipStream_t stream) {
  const int S = st->S, R = B + 1, M = S * R;
  float* logits = logits_out ? logits_out : (float*)(ws + L.logits);
  int32_t* am = argmax_out ? argmax_out : (int32_t*)(ws + L.am);
  int32_t* acc = accept_out ? accept_out : (int32_t*)(ws + L.acc);
  int32_t* lead = (int32_t*)(ws + L.lead);
  int rc;
  // draft forward
  hipLaunchKernelGGL(embed_rows_kernel<T>, dim3(M), dim3(256), 0, stream, (const T*)m->embed,
                     m->hidden, m->vocab, R, 1, st->boundary, st->draft, st->draft_width,
                     nullptr, 0, (float*)(ws + L.x));
  if ((rc = launch_status("literal_round(embed)"))) return rc;
  if ((rc = forward_layers<T>(m, st, 1, B, chunk_keys, L, ws, stream))) return rc;
  if ((rc = gemm(L, ws, m->dtype, ws + L.h, m->lm_head, M, m->vocab, m->hidden, logits, 1, 0, stream)))
    return rc;
  rc = argmax_accept(logits, DVS_F32, S, R, m->vocab, 1, st->draft, st->draft_width, am, acc,
                     st->err_word, stream);
  if (rc) return rc;
  hipLaunchKernelGGL(round_draft_kernel, dim3((S + 255) / 256), dim3(256), 0, stream, S, B, am,
                     st->finished, st->kv_len, lead, st->draft, st->draft_width);
  if ((rc = launch_status("literal_round(draft)"))) return rc;
  // verify forward
  hipLaunchKernelGGL(embed_rows_kernel<T>, dim3(M), dim3(256), 0, stream, (const T*)m->embed,
                     m->hidden, m->vocab, R, R, lead, st->draft, st->draft_width, nullptr, 0,
                     (float*)(ws + L.x));
  if ((rc = launch_status("literal_round(embed)"))) return rc;
  if ((rc = forward_layers<T>(m, st, R, 0, chunk_keys, L, ws, stream))) return rc;
  if ((rc = gemm(L, ws, m->dtype, ws + L.h, m->lm_head, M, m->vocab, m->hidden, logits, 1, 0, stream)))
    return rc;
  rc = argmax_accept(logits, DVS_F32, S, R, m->vocab, R, st->draft, st->draft_width, am, acc,
                     st->err_word, stream);
  if (rc) return rc;
  return kv_commit_round(S, B, lead, acc, am, st->kv_len, st->page_table, st->num_pages,
                         st->max_pages, st->free_stack, st->free_top, st->num_pool_pages,
                         st->boundary, st->draft, st->draft_width, st->out_tokens, st->out_count,
                         st->max_new, st->eos_id, st->finished, st->err_word, stream);
}

// One denoising forward of direct block diffusion: [x0, b_1..b_B] with the
// boundary row causal and the block rows bidirectional (masked positions
// carry [M]); top-1 and confidence of every row; the reveal.  kv_len is
// unchanged (the window's K/V slots are rewritten by the next forward).
// npos: block positions, B (direct diffusion) or B + 1 (the refined draft of
// the two-forward round, whose last prediction has no input slot).
template <typename T>
static int run_denoise(const dvs_model* m, const dvs_state* st, int B, int npos, float tau_c,
                       int32_t* block, int32_t* n_open, int chunk_keys, const StepLayout& L,
                       char* ws, float* logits_out, int32_t* argmax_out, float* conf_out,
                       hipStream_t stream) {
  const int S = st->S, R = B + 1, M = S * R;
  float* logits = logits_out ? logits_out : (float*)(ws + L.logits);
  int32_t* am = argmax_out ? argmax_out : (int32_t*)(ws + L.am);
  float* conf = conf_out ? conf_out : (float*)(ws + L.conf);
  hipLaunchKernelGGL(embed_rows_kernel<T>, dim3(M), dim3(256), 0, stream, (const T*)m->embed,
                     m->hidden, m->vocab, R, 1, st->boundary, st->draft, st->draft_width, block,
                     npos, (float*)(ws + L.x));
  int rc;
  if ((rc = launch_status("diffusion_denoise(embed)"))) return rc;
  if ((rc = forward_layers<T>(m, st, 1, B, chunk_keys, L, ws, stream))) return rc;
  if ((rc = gemm(L, ws, m->dtype, ws + L.h, m->lm_head, M, m->vocab, m->hidden, logits, 1, 0, stream)))
    return rc;
  if ((rc = top1_confidence(logits, DVS_F32, M, m->vocab, am, conf, st->err_word, stream))) return rc;
  hipLaunchKernelGGL(zero_words_kernel, dim3(1), dim3(256), 0, stream, n_open, 1);
  hipLaunchKernelGGL(reveal_kernel, dim3(S), dim3(64), 0, stream, npos, R, tau_c, am, conf,
                     st->finished, block, n_open);
  return launch_status("diffusion_denoise(reveal)");
}

// The block's cache-write forward (x0 and b_1..b_{B-1} as causal rows, no
// LM head) and its commit.
template <typename T>
static int run_block_commit(const dvs_model* m, const dvs_state* st, int B, const int32_t* block,
                            int chunk_keys, const StepLayout& L, char* ws, hipStream_t stream) {
  const int S = st->S, M = S * B;
  hipLaunchKernelGGL(embed_rows_kernel<T>, dim3(M), dim3(256), 0, stream, (const T*)m->embed,
                     m->hidden, m->vocab, B, B, st->boundary, block, B, nullptr, 0,
                     (float*)(ws + L.x));
  int rc;
  if ((rc = launch_status("diffusion_block(embed)"))) return rc;
  if ((rc = forward_layers<T>(m, st, B, 0, chunk_keys, L, ws, stream))) return rc;
  return kv_commit_block(S, B, block, st->kv_len, st->page_table, st->num_pages, st->max_pages,
                         st->free_stack, st->free_top, st->num_pool_pages, st->boundary,
                         st->out_tokens, st->out_count, st->max_new, st->eos_id, st->finished,
                         st->err_word, stream);
}

// The two-forward round with a refined draft: draft forwards over
// [x0, b_1..b_B] until every one of the B + 1 predictions (a0, d_1..d_B) is
// revealed at threshold tau_d (b_p: revealed prediction p, else [M]); then
// the verify forward and commit of run_round.  Ld and Lv (layouts of the
// (1, B) and (B + 1, 0) windows) agree below the attention workspace, where
// the block and the lead tokens live.
template <typename T>
static int run_round_refined(const dvs_model* m, const dvs_state* st, int B, float tau_d,
                             int chunk_keys, const StepLayout& Ld, const StepLayout& Lv, char* ws,
                             float* logits_out, int32_t* argmax_out, int32_t* accept_out,
                             int* draft_steps, hipStream_t stream) {
  const int S = st->S, R = B + 1, M = S * R;
  int32_t* blk = (int32_t*)(ws + Ld.blk);
  int32_t* n_open = (int32_t*)(ws + Ld.nopen);
  int32_t* lead = (int32_t*)(ws + Lv.lead);
  hipLaunchKernelGGL(fill_words_kernel, dim3((M + 255) / 256), dim3(256), 0, stream, blk, M, -1);
  int rc;
  if ((rc = launch_status("literal_round_refined(fill)"))) return rc;
  int steps = 0, open = 1;
  while (open && steps < R) {
    if ((rc = run_denoise<T>(m, st, B, R, tau_d, blk, n_open, chunk_keys, Ld, ws, nullptr, nullptr,
                             nullptr, stream)))
      return rc;
    ++steps;
    if (hipMemcpyAsync(&open, n_open, sizeof(int32_t), hipMemcpyDeviceToHost, stream) != hipSuccess ||
        hipStreamSynchronize(stream) != hipSuccess) {
      set_error("literal_round_refined: reading the open-draft count failed");
      return DVS_EHIP;
    }
  }
  if (open) {
    set_error("literal_round_refined: %d drafts still open after %d forwards", open, steps);
    return DVS_EHIP;
  }
  if (draft_steps) *draft_steps = steps;
  hipLaunchKernelGGL(round_draft_kernel, dim3((S + 255) / 256), dim3(256), 0, stream, S, B, blk,
                     st->finished, st->kv_len, lead, st->draft, st->draft_width);
  if ((rc = launch_status("literal_round_refined(draft)"))) return rc;
  float* logits = logits_out ? logits_out : (float*)(ws + Lv.logits);
  int32_t* am = argmax_out ? argmax_out : (int32_t*)(ws + Lv.am);
  int32_t* acc = accept_out ? accept_out : (int32_t*)(ws + Lv.acc);
  hipLaunchKernelGGL(embed_rows_kernel<T>, dim3(M), dim3(256), 0, stream, (const T*)m->embed,
                     m->hidden, m->vocab, R, R, lead, st->draft, st->draft_width, nullptr, 0,
                     (float*)(ws + Lv.x));
  if ((rc = launch_status("literal_round_refined(embed)"))) return rc;
  if ((rc = forward_layers<T>(m, st, R, 0, chunk_keys, Lv, ws, stream))) return rc;
  if ((rc = gemm(Lv, ws, m->dtype, ws + Lv.h, m->lm_head, M, m->vocab, m->hidden, logits, 1, 0,
                 stream)))
    return rc;
  rc = argmax_accept(logits, DVS_F32, S, R, m->vocab, R, st->draft, st->draft_width, am, acc,
                     st->err_word, stream);
  if (rc) return rc;
  return kv_commit_round(S, B, lead, acc, am, st->kv_len, st->page_table, st->num_pages,
                         st->max_pages, st->free_stack, st->free_top, st->num_pool_pages,
                         st->boundary, st->draft, st->draft_width, st->out_tokens, st->out_count,
                         st->max_new, st->eos_id, st->finished, st->err_word, stream);
}

// The two-forward round under sampling at temperature T (stochastic
// acceptance): the draft forward's rows are sampled (a0 from the boundary
// row, d_j from mask row j) with u[s, 0..B]; the verify forward's rows give
// p_j; acceptance and the final sample use u[s, B+1..2B+1].  Draft logits and
// both rows' statistics live past the larger of the two forwards' layouts.
template <typename T>
static int run_round_sampled(const dvs_model* m, const dvs_state* st, int B, float T_,
                             const float* u, int chunk_keys, const StepLayout& Ld,
                             const StepLayout& Lv, size_t extra, char* ws, float* logits_out,
                             int32_t* accept_out, hipStream_t stream) {
  const int S = st->S, R = B + 1, M = S * R, V = m->vocab, us = 2 * B + 2;
  const float invT = 1.f / T_;
  float* zd = (float*)(ws + extra);
  float2* sd = (float2*)(ws + extra + al((size_t)M * V * 4));
  float2* sv = sd + M;
  float* zv = logits_out ? logits_out : (float*)(ws + Lv.logits);
  int32_t* tok = (int32_t*)(ws + Lv.am);
  int32_t* acc = accept_out ? accept_out : (int32_t*)(ws + Lv.acc);
  int32_t* lead = (int32_t*)(ws + Lv.lead);
  int rc;
  hipLaunchKernelGGL(embed_rows_kernel<T>, dim3(M), dim3(256), 0, stream, (const T*)m->embed,
                     m->hidden, V, R, 1, st->boundary, st->draft, st->draft_width, nullptr, 0,
                     (float*)(ws + Ld.x));
  if ((rc = launch_status("literal_round_sampled(embed)"))) return rc;
  if ((rc = forward_layers<T>(m, st, 1, B, chunk_keys, Ld, ws, stream))) return rc;
  if ((rc = gemm(Ld, ws, m->dtype, ws + Ld.h, m->lm_head, M, V, m->hidden, zd, 1, 0, stream)))
    return rc;
  if ((rc = launch_row_stats(zd, M, V, invT, sd, st->err_word, stream))) return rc;
  if ((rc = launch_sample_rows(zd, sd, V, invT, u, us, S, R, tok, stream))) return rc;
  hipLaunchKernelGGL(round_draft_kernel, dim3((S + 255) / 256), dim3(256), 0, stream, S, B, tok,
                     st->finished, st->kv_len, lead, st->draft, st->draft_width);
  if ((rc = launch_status("literal_round_sampled(draft)"))) return rc;
  hipLaunchKernelGGL(embed_rows_kernel<T>, dim3(M), dim3(256), 0, stream, (const T*)m->embed,
                     m->hidden, V, R, R, lead, st->draft, st->draft_width, nullptr, 0,
                     (float*)(ws + Lv.x));
  if ((rc = launch_status("literal_round_sampled(embed)"))) return rc;
  if ((rc = forward_layers<T>(m, st, R, 0, chunk_keys, Lv, ws, stream))) return rc;
  if ((rc = gemm(Lv, ws, m->dtype, ws + Lv.h, m->lm_head, M, V, m->hidden, zv, 1, 0, stream)))
    return rc;
  if ((rc = launch_row_stats(zv, M, V, invT, sv, st->err_word, stream))) return rc;
  if ((rc = launch_accept_final(S, B, V, invT, zv, sv, zd, sd, st->draft, st->draft_width, u, us,
                                acc, tok, stream)))
    return rc;
  return kv_commit_round(S, B, lead, acc, tok, st->kv_len, st->page_table, st->num_pages,
                         st->max_pages, st->free_stack, st->free_top, st->num_pool_pages,
                         st->boundary, st->draft, st->draft_width, st->out_tokens, st->out_count,
                         st->max_new, st->eos_id, st->finished, st->err_word, stream);
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

static int check_model_state(const dvs_model* m, const dvs_state* st, const char* who);

extern "C" int multidraft_step(const dvs_model* m, const dvs_state* st, int32_t B,
                               int32_t chunk_keys, float* logits_out, int32_t* argmax_out,
                               int32_t* accept_out, void* workspace, size_t ws_bytes,
                               void* stream) {
  clear_error();
  DVS_CHECK_ARG(model_ok(m), "multidraft_step: invalid model description");
  DVS_CHECK_ARG(B >= 1 && B <= 64, "multidraft_step: need 1 <= B <= 64");
  int rc = check_model_state(m, st, "multidraft_step");
  if (rc) return rc;
  DVS_CHECK_ARG(st->draft_width >= B - 1 && st->draft_width <= B,
                "multidraft_step: draft width must be B - 1 or B");
  const int n_mask = B * B;
  const StepLayout L = step_layout(m, st->S, B, n_mask, st->max_pages, chunk_keys,
                                   (size_t)st->S * (B + n_mask));
  if (!workspace || ws_bytes < L.total) {
    set_error("multidraft_step: workspace needs %zu bytes, got %zu", L.total, ws_bytes);
    return DVS_EWORKSPACE;
  }
  hipStream_t s = (hipStream_t)stream;
  if (m->dtype == DVS_BF16)
    return run_step<__bf16>(m, st, B, n_mask, chunk_keys, L, (char*)workspace, logits_out,
                            argmax_out, accept_out, s, B);
  return run_step<float>(m, st, B, n_mask, chunk_keys, L, (char*)workspace, logits_out, argmax_out,
                         accept_out, s, B);
}

extern "C" int literal_round(const dvs_model* m, const dvs_state* st, int32_t B,
                             int32_t chunk_keys, float* logits_out, int32_t* argmax_out,
                             int32_t* accept_out, void* workspace, size_t ws_bytes, void* stream) {
  clear_error();
  DVS_CHECK_ARG(model_ok(m), "literal_round: invalid model description");
  DVS_CHECK_ARG(st && st->S >= 1 && st->kv_len && st->page_table && st->num_pages &&
                    st->free_stack && st->free_top && st->boundary && st->out_tokens &&
                    st->out_count && st->finished,
                "literal_round: invalid state description");
  DVS_CHECK_ARG(B >= 1, "literal_round: need B >= 1");
  DVS_CHECK_ARG(st->draft && st->draft_width >= B, "literal_round: draft narrower than B");
  for (int l = 0; l < m->n_layers; ++l) {
    const dvs_layer& ly = m->layers[l];
    DVS_CHECK_ARG(ly.wq && ly.wk && ly.wv && ly.wo && ly.g_attn && ly.k_pool && ly.v_pool,
                  "literal_round: layer %d incomplete", l);
    DVS_CHECK_ARG(m->ffn == 0 || (ly.g_mlp && ly.w_gate && ly.w_up && ly.w_down),
                  "literal_round: layer %d MLP incomplete", l);
  }
  DVS_CHECK_SUPPORTED(m->head_dim == 64 || m->head_dim == 96 || m->head_dim == 128,
                      "literal_round: head_dim %d", m->head_dim);
  const StepLayout L = step_layout(m, st->S, B + 1, 0, st->max_pages, chunk_keys,
                                   (size_t)st->S * (B + 1));
  if (!workspace || ws_bytes < L.total) {
    set_error("literal_round: workspace needs %zu bytes, got %zu", L.total, ws_bytes);
    return DVS_EWORKSPACE;
  }
  hipStream_t s = (hipStream_t)stream;
  if (m->dtype == DVS_BF16)
    return run_round<__bf16>(m, st, B, chunk_keys, L, (char*)workspace, logits_out, argmax_out,
                             accept_out, s);
  return run_round<float>(m, st, B, chunk_keys, L, (char*)workspace, logits_out, argmax_out,
                          accept_out, s);
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

static int check_model_state(const dvs_model* m, const dvs_state* st, const char* who) {
  DVS_CHECK_ARG(model_ok(m), "%s: invalid model description", who);
  DVS_CHECK_ARG(st && st->S >= 1 && st->kv_len && st->page_table && st->num_pages &&
                    st->free_stack && st->free_top && st->boundary && st->out_tokens &&
                    st->out_count && st->finished,
                "%s: invalid state description", who);
  for (int l = 0; l < m->n_layers; ++l) {
    const dvs_layer& ly = m->layers[l];
    DVS_CHECK_ARG(ly.wq && ly.wk && ly.wv && ly.wo && ly.g_attn && ly.k_pool && ly.v_pool,
                  "%s: layer %d incomplete", who, l);
    DVS_CHECK_ARG(m->ffn == 0 || (ly.g_mlp && ly.w_gate && ly.w_up && ly.w_down),
                  "%s: layer %d MLP incomplete", who, l);
  }
  DVS_CHECK_SUPPORTED(m->head_dim == 64 || m->head_dim == 96 || m->head_dim == 128,
                      "%s: head_dim %d", who, m->head_dim);
  return DVS_OK;
}

extern "C" size_t dvs_diffusion_workspace_bytes(const dvs_model* m, int32_t S, int32_t B,
                                                int32_t max_pages, int32_t chunk_keys) {
  if (!model_ok(m) || S < 1 || B < 1 || max_pages < 1) return 0;
  return std::max(step_layout(m, S, 1, B, max_pages, chunk_keys, (size_t)S * (B + 1)).total,
                  step_layout(m, S, B, 0, max_pages, chunk_keys, 0).total);
}

extern "C" int diffusion_denoise(const dvs_model* m, const dvs_state* st, int32_t B, float tau_c,
                                 int32_t* block, int32_t* n_open, int32_t chunk_keys,
                                 float* logits_out, int32_t* argmax_out, float* conf_out,
                                 void* workspace, size_t ws_bytes, void* stream) {
  clear_error();
  int rc = check_model_state(m, st, "diffusion_denoise");
  if (rc) return rc;
  DVS_CHECK_ARG(B >= 1 && block && n_open, "diffusion_denoise: need B >= 1, block, n_open");
  const StepLayout L = step_layout(m, st->S, 1, B, st->max_pages, chunk_keys,
                                   (size_t)st->S * (B + 1));
  if (!workspace || ws_bytes < L.total) {
    set_error("diffusion_denoise: workspace needs %zu bytes, got %zu", L.total, ws_bytes);
    return DVS_EWORKSPACE;
  }
  hipStream_t s = (hipStream_t)stream;
  if (m->dtype == DVS_BF16)
    return run_denoise<__bf16>(m, st, B, B, tau_c, block, n_open, chunk_keys, L,
                               (char*)workspace, logits_out, argmax_out, conf_out, s);
  return run_denoise<float>(m, st, B, B, tau_c, block, n_open, chunk_keys, L, (char*)workspace,
                            logits_out, argmax_out, conf_out, s);
}

extern "C" int diffusion_block(const dvs_model* m, const dvs_state* st, int32_t B, float tau_c,
                               int32_t* block, int32_t chunk_keys, int32_t* steps_out,
                               void* workspace, size_t ws_bytes, void* stream) {
  clear_error();
  int rc = check_model_state(m, st, "diffusion_block");
  if (rc) return rc;
  DVS_CHECK_ARG(B >= 1 && block, "diffusion_block: need B >= 1 and a block array");
  const int S = st->S;
  const StepLayout Ld = step_layout(m, S, 1, B, st->max_pages, chunk_keys, (size_t)S * (B + 1));
  const StepLayout Lc = step_layout(m, S, B, 0, st->max_pages, chunk_keys, 0);
  const size_t need = std::max(Ld.total, Lc.total);
  if (!workspace || ws_bytes < need) {
    set_error("diffusion_block: workspace needs %zu bytes, got %zu", need, ws_bytes);
    return DVS_EWORKSPACE;
  }
  hipStream_t s = (hipStream_t)stream;
  char* ws = (char*)workspace;
  int32_t* n_open = (int32_t*)(ws + Ld.nopen);
  hipLaunchKernelGGL(fill_words_kernel, dim3((S * B + 255) / 256), dim3(256), 0, s, block, S * B,
                     -1);
  if ((rc = launch_status("diffusion_block(fill)"))) return rc;
  // every step reveals at least one position of every open block
  int steps = 0, open = 1;
  while (open && steps < B) {
    rc = m->dtype == DVS_BF16
             ? run_denoise<__bf16>(m, st, B, B, tau_c, block, n_open, chunk_keys, Ld, ws, nullptr,
                                   nullptr, nullptr, s)
             : run_denoise<float>(m, st, B, B, tau_c, block, n_open, chunk_keys, Ld, ws, nullptr,
                                  nullptr, nullptr, s);
    if (rc) return rc;
    ++steps;
    if (hipMemcpyAsync(&open, n_open, sizeof(int32_t), hipMemcpyDeviceToHost, s) != hipSuccess ||
        hipStreamSynchronize(s) != hipSuccess) {
      set_error("diffusion_block: reading the open-block count failed");
      return DVS_EHIP;
    }
  }
  if (open) {
    set_error("diffusion_block: %d blocks still open after %d steps", open, steps);
    return DVS_EHIP;
  }
  if (steps_out) *steps_out = steps;
  return m->dtype == DVS_BF16 ? run_block_commit<__bf16>(m, st, B, block, chunk_keys, Lc, ws, s)
                              : run_block_commit<float>(m, st, B, block, chunk_keys, Lc, ws, s);
}

extern "C" int literal_round_refined(const dvs_model* m, const dvs_state* st, int32_t B,
                                     float tau_d, int32_t chunk_keys, float* logits_out,
                                     int32_t* argmax_out, int32_t* accept_out,
                                     int32_t* draft_steps_out, void* workspace, size_t ws_bytes,
                                     void* stream) {
  clear_error();
  int rc = check_model_state(m, st, "literal_round_refined");
  if (rc) return rc;
  DVS_CHECK_ARG(B >= 1, "literal_round_refined: need B >= 1");
  DVS_CHECK_ARG(st->draft && st->draft_width >= B, "literal_round_refined: draft narrower than B");
  const int S = st->S;
  const StepLayout Ld = step_layout(m, S, 1, B, st->max_pages, chunk_keys, (size_t)S * (B + 1));
  const StepLayout Lv = step_layout(m, S, B + 1, 0, st->max_pages, chunk_keys, (size_t)S * (B + 1));
  const size_t need = std::max(Ld.total, Lv.total);
  if (!workspace || ws_bytes < need) {
    set_error("literal_round_refined: workspace needs %zu bytes, got %zu", need, ws_bytes);
    return DVS_EWORKSPACE;
  }
  int steps = 0;
  hipStream_t s = (hipStream_t)stream;
  rc = m->dtype == DVS_BF16
           ? run_round_refined<__bf16>(m, st, B, tau_d, chunk_keys, Ld, Lv, (char*)workspace,
                                       logits_out, argmax_out, accept_out, &steps, s)
           : run_round_refined<float>(m, st, B, tau_d, chunk_keys, Ld, Lv, (char*)workspace,
                                      logits_out, argmax_out, accept_out, &steps, s);
  if (draft_steps_out) *draft_steps_out = steps;
  return rc;
}

// Workspace of the sampled round: the larger of the two forwards' layouts,
// then the draft logits [S(B+1), V] fp32 and two [S(B+1)] float2 statistics.
static size_t sampled_extra(const dvs_model* m, int S, int B, int max_pages, int chunk_keys,
                            StepLayout* Ld, StepLayout* Lv) {
  *Ld = step_layout(m, S, 1, B, max_pages, chunk_keys, (size_t)S * (B + 1));
  *Lv = step_layout(m, S, B + 1, 0, max_pages, chunk_keys, (size_t)S * (B + 1));
  return al(std::max(Ld->total, Lv->total));
}

extern "C" size_t dvs_sampled_round_workspace_bytes(const dvs_model* m, int32_t S, int32_t B,
                                                    int32_t max_pages, int32_t chunk_keys) {
  if (!model_ok(m) || S < 1 || B < 1 || max_pages < 1) return 0;
  StepLayout Ld, Lv;
  const size_t M = (size_t)S * (B + 1);
  return sampled_extra(m, S, B, max_pages, chunk_keys, &Ld, &Lv) + al(M * m->vocab * 4) +
         2 * al(M * 8);
}

extern "C" int literal_round_sampled(const dvs_model* m, const dvs_state* st, int32_t B,
                                     float temperature, const float* u, int32_t chunk_keys,
                                     float* logits_out, int32_t* accept_out, void* workspace,
                                     size_t ws_bytes, void* stream) {
  clear_error();
  int rc = check_model_state(m, st, "literal_round_sampled");
  if (rc) return rc;
  DVS_CHECK_ARG(B >= 1 && u, "literal_round_sampled: need B >= 1 and uniforms");
  DVS_CHECK_ARG(temperature > 0.f && temperature < 1e30f,
                "literal_round_sampled: temperature must be positive and finite");
  DVS_CHECK_ARG(st->draft && st->draft_width >= B, "literal_round_sampled: draft narrower than B");
  const size_t need = dvs_sampled_round_workspace_bytes(m, st->S, B, st->max_pages, chunk_keys);
  if (!workspace || ws_bytes < need) {
    set_error("literal_round_sampled: workspace needs %zu bytes, got %zu", need, ws_bytes);
    return DVS_EWORKSPACE;
  }
  StepLayout Ld, Lv;
  const size_t extra = sampled_extra(m, st->S, B, st->max_pages, chunk_keys, &Ld, &Lv);
  hipStream_t s = (hipStream_t)stream;
  return m->dtype == DVS_BF16
             ? run_round_sampled<__bf16>(m, st, B, temperature, u, chunk_keys, Ld, Lv, extra,
                                         (char*)workspace, logits_out, accept_out, s)
             : run_round_sampled<float>(m, st, B, temperature, u, chunk_keys, Ld, Lv, extra,
                                        (char*)workspace, logits_out, accept_out, s);
}
