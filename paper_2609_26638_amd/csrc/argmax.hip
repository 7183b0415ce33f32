// argmax_accept: vocabulary top-1 per window row, then greedy acceptance.
//
// Top-1 (the verifier's greedy prediction; appendix "AR-Equivalence and
// Equality Testing" uses top-1 decoding): the largest logit wins, the lowest
// index among equal maxima, -0.0 == +0.0.  Each thread keeps its first
// maximum (values compared as floats); the per-thread winners are mapped to
// order-preserving unsigned keys (sign-magnitude -> two's-complement order,
// -0.0 folded onto +0.0) and reduced with "larger key, then smaller index"
// packed into one 64-bit max.
//
// Acceptance (method "Self-Speculative Decoding"; appendix item Accept):
// a_j = top1(row j-1); A = longest prefix of the draft with d_j == a_j.
//
// The argmax is a pure HBM stream: one workgroup of 512 threads per row,
// 16-byte loads with 8 in flight per thread (interleaved A/B: 256 threads
// with 8 or 16 in flight read 5% / 2% slower, 512 with 16 17% slower), about
// two vector instructions per element (max3 chain, NaN/infinity probe),
// wavefront shuffles, then LDS across the eight waves.
#include "dvs_common.h"

namespace dvs {

__device__ __forceinline__ uint32_t key_f32(uint32_t u, bool& nonfinite) {
  if ((u & 0x7fffffffu) == 0) u = 0;
  if ((u & 0x7f800000u) == 0x7f800000u) nonfinite = true;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Larger key first, then smaller index: pack (key, 0x7fffffff - index).
__device__ __forceinline__ uint64_t pack_ki(uint32_t key, int idx) {
  return ((uint64_t)key << 32) | (uint32_t)(0x7fffffff - idx);
}

__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t v, int m) {
  const uint32_t lo = __shfl_xor((uint32_t)v, m);
  const uint32_t hi = __shfl_xor((uint32_t)(v >> 32), m);
  return ((uint64_t)hi << 32) | lo;
}

template <bool BF16>
__device__ __forceinline__ float elem_f(const u32x4& x, int e) {
  if constexpr (BF16) {
    const uint32_t w = x[e >> 1];
    return __uint_as_float((e & 1) ? (w & 0xffff0000u) : (w << 16));   // bf16 -> fp32 is exact
  } else {
    return __uint_as_float(x[e]);
  }
}

// A row with no value above -inf (every value -inf or NaN): the top-1 is the
// lowest index holding -inf (the largest comparable value), or 0 when every
// value is NaN, so the result is always a vocabulary index.  Block-wide scan
// (NT threads); runs only for such rows, which also set DVS_ERR_NONFINITE.
template <bool BF16, int NT>
__device__ __forceinline__ int first_neg_inf(const char* base, int V, int tid, int* s_first) {
  if (tid == 0) *s_first = 0x7fffffff;
  __syncthreads();
  int first = 0x7fffffff;
  for (int i = tid; i < V; i += NT) {
    const float f = BF16 ? __uint_as_float((uint32_t)((const uint16_t*)base)[i] << 16)
                         : ((const float*)base)[i];
    if (f == -INFINITY) { first = i; break; }
  }
  if (first != 0x7fffffff) atomicMin(s_first, first);
  __syncthreads();
  return *s_first == 0x7fffffff ? 0 : *s_first;
}

template <bool BF16>
__global__ void __launch_bounds__(512) argmax_kernel(const void* __restrict__ logits, int V,
                                                     int32_t* __restrict__ argmax_out,
                                                     int32_t* err) {
  constexpr int EPV = BF16 ? 8 : 4;   // elements per 16-byte vector
  constexpr int UNR = 8;              // vectors in flight per thread
  __shared__ uint64_t sred[8];
  __shared__ int s_first;
  const size_t row = blockIdx.x;
  const int tid = threadIdx.x;
  const char* base = (const char*)logits + row * (size_t)V * (BF16 ? 2 : 4);
  // Every thread visits its elements in increasing index order, so its first
  // maximum is kept by a strict comparison.  Values are compared as floats
  // (-0.0 == +0.0); a NaN never wins a comparison, and x * 0 turns any NaN or
  // infinity into a NaN in `nf`, which flags the row.
  float best = -INFINITY;
  int bi = 0x7fffffff;
  float nf = 0.f;

  // vectorised body when the row start is 16-byte aligned: per batch of UNR
  // vectors, a running max3 chain; only a batch that beats the thread's best
  // is scanned again for the position of its first maximum
  const bool aligned = ((((uintptr_t)base) & 15) == 0);
  const int nvec = aligned ? V / EPV : 0;
  int v0 = 0;
  for (; v0 + UNR * 512 <= nvec; v0 += UNR * 512) {
    u32x4 buf[UNR];
#pragma unroll
    for (int u = 0; u < UNR; ++u) buf[u] = ((const u32x4*)base)[v0 + u * 512 + tid];
    float bm = -INFINITY;
#pragma unroll
    for (int u = 0; u < UNR; ++u)
#pragma unroll
      for (int e = 0; e < EPV; ++e) {
        const float x = elem_f<BF16>(buf[u], e);
        bm = fmaxf(bm, x);
        nf = fmaf(x, 0.f, nf);
      }
    if (bm > best) {
      int at = 0x7fffffff;
#pragma unroll
      for (int u = UNR - 1; u >= 0; --u)
#pragma unroll
        for (int e = EPV - 1; e >= 0; --e)
          if (elem_f<BF16>(buf[u], e) == bm) at = (v0 + u * 512 + tid) * EPV + e;
      best = bm;
      bi = at;
    }
  }
  for (int vi = v0 + tid; vi < nvec; vi += 512) {
    const u32x4 x = ((const u32x4*)base)[vi];
#pragma unroll
    for (int e = 0; e < EPV; ++e) {
      const float f = elem_f<BF16>(x, e);
      nf = fmaf(f, 0.f, nf);
      if (f > best) { best = f; bi = vi * EPV + e; }
    }
  }
  // scalar tail (and the whole row when unaligned)
  for (int i = nvec * EPV + tid; i < V; i += 512) {
    const float f = BF16 ? __uint_as_float((uint32_t)((const uint16_t*)base)[i] << 16)
                         : ((const float*)base)[i];
    nf = fmaf(f, 0.f, nf);
    if (f > best) { best = f; bi = i; }
  }

  bool nonfinite = nf != nf;
  uint64_t bp = (bi == 0x7fffffff) ? 0 : pack_ki(key_f32(__float_as_uint(best), nonfinite), bi);
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    const uint64_t o = shfl_xor_u64(bp, off);
    bp = o > bp ? o : bp;
  }
  if ((tid & 63) == 0) sred[tid >> 6] = bp;
  if (nonfinite) set_err(err, DVS_ERR_NONFINITE);
  __syncthreads();
  uint64_t b = sred[0];
  for (int i = 1; i < 8; ++i) b = sred[i] > b ? sred[i] : b;
  if (b == 0) {   // no value above -inf anywhere in the row (uniform branch)
    const int i0 = first_neg_inf<BF16, 512>(base, V, tid, &s_first);
    if (tid == 0) argmax_out[row] = i0;
  } else if (tid == 0) {
    argmax_out[row] = 0x7fffffff - (int)(uint32_t)(b & 0xffffffffu);
  }
}

// Top-1 and its softmax probability (appendix "Direct Block-Diffusion
// Decoding": a prediction's confidence is its token probability), in one
// pass over the row: every thread keeps its first maximum m and the sum
// sum_i exp(x_i - m) of what it has read, rescaled when m grows; the threads
// then merge (m, sum, index) pairs, the lowest index among equal maxima.
// conf = 1 / sum.  fp32 arithmetic; one workgroup per row, 16-byte loads
// with UNR in flight per thread as in argmax_kernel.
template <bool BF16>
__global__ void __launch_bounds__(256) top1_conf_kernel(const void* __restrict__ logits, int V,
                                                        int32_t* __restrict__ argmax_out,
                                                        float* __restrict__ conf_out,
                                                        int32_t* err) {
  constexpr int EPV = BF16 ? 8 : 4;   // elements per 16-byte vector
  constexpr int UNR = 8;              // vectors in flight per thread
  __shared__ float sm[4], ss[4];
  __shared__ int si[4];
  __shared__ int s_first;
  const size_t row = blockIdx.x;
  const int tid = threadIdx.x;
  const char* base = (const char*)logits + row * (size_t)V * (BF16 ? 2 : 4);
  float m = -INFINITY, sum = 0.f, nf = 0.f;
  int bi = 0x7fffffff;
  // elementwise update, in increasing index order per thread
  auto visit = [&](float f, int i) {
    nf = fmaf(f, 0.f, nf);
    if (f > m) {
      sum = (m == -INFINITY ? 0.f : sum * __expf(m - f)) + 1.f;
      m = f;
      bi = i;
    } else if (m != -INFINITY) {
      sum += __expf(f - m);
    }
  };
  // vectorised body (16-byte aligned rows): per batch of UNR vectors, the
  // batch maximum first (one rescale of the running sum per batch), then the
  // batch's terms
  const bool aligned = ((((uintptr_t)base) & 15) == 0);
  const int nvec = aligned ? V / EPV : 0;
  int v0 = 0;
  for (; v0 + UNR * 256 <= nvec; v0 += UNR * 256) {
    u32x4 buf[UNR];
#pragma unroll
    for (int u = 0; u < UNR; ++u) buf[u] = ((const u32x4*)base)[v0 + u * 256 + tid];
    float bm = -INFINITY;
#pragma unroll
    for (int u = 0; u < UNR; ++u)
#pragma unroll
      for (int e = 0; e < EPV; ++e) {
        const float x = elem_f<BF16>(buf[u], e);
        bm = fmaxf(bm, x);
        nf = fmaf(x, 0.f, nf);
      }
    if (bm > m) {
      int at = 0x7fffffff;
#pragma unroll
      for (int u = UNR - 1; u >= 0; --u)
#pragma unroll
        for (int e = EPV - 1; e >= 0; --e)
          if (elem_f<BF16>(buf[u], e) == bm) at = (v0 + u * 256 + tid) * EPV + e;
      sum = m == -INFINITY ? 0.f : sum * __expf(m - bm);
      m = bm;
      bi = at;
    }
    if (m != -INFINITY) {
#pragma unroll
      for (int u = 0; u < UNR; ++u)
#pragma unroll
        for (int e = 0; e < EPV; ++e) sum += __expf(elem_f<BF16>(buf[u], e) - m);
    }
  }
  for (int vi = v0 + tid; vi < nvec; vi += 256) {
    const u32x4 x = ((const u32x4*)base)[vi];
#pragma unroll
    for (int e = 0; e < EPV; ++e) visit(elem_f<BF16>(x, e), vi * EPV + e);
  }
  for (int i = nvec * EPV + tid; i < V; i += 256)
    visit(BF16 ? __uint_as_float((uint32_t)((const uint16_t*)base)[i] << 16)
               : ((const float*)base)[i],
          i);
  // wave merge
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    const float om = __shfl_xor(m, off);
    const float os = __shfl_xor(sum, off);
    const int oi = __shfl_xor(bi, off);
    const float M = fmaxf(m, om);
    const float a = m == -INFINITY ? 0.f : sum * __expf(m - M);
    const float b = om == -INFINITY ? 0.f : os * __expf(om - M);
    bi = (om > m || (om == m && oi < bi)) ? oi : bi;
    m = M;
    sum = a + b;
  }
  if ((tid & 63) == 0) { sm[tid >> 6] = m; ss[tid >> 6] = sum; si[tid >> 6] = bi; }
  if (nf != nf) set_err(err, DVS_ERR_NONFINITE);
  __syncthreads();
  if (si[0] == 0x7fffffff && si[1] == 0x7fffffff && si[2] == 0x7fffffff && si[3] == 0x7fffffff) {
    // no value above -inf anywhere in the row (uniform branch)
    const int i0 = first_neg_inf<BF16, 256>(base, V, tid, &s_first);
    if (tid == 0) {
      argmax_out[row] = i0;
      conf_out[row] = 0.f;
    }
    return;
  }
  if (tid == 0) {
    float M = sm[0], S = ss[0];
    int I = si[0];
    for (int w = 1; w < 4; ++w) {
      const float nm = fmaxf(M, sm[w]);
      const float a = M == -INFINITY ? 0.f : S * __expf(M - nm);
      const float b = sm[w] == -INFINITY ? 0.f : ss[w] * __expf(sm[w] - nm);
      if (sm[w] > M || (sm[w] == M && si[w] < I)) I = si[w];
      M = nm;
      S = a + b;
    }
    argmax_out[row] = I;
    conf_out[row] = 1.f / S;
  }
}

__global__ void accept_kernel(const int32_t* __restrict__ argmax_out, int S, int R, int n_causal,
                              const int32_t* __restrict__ draft, int draft_width,
                              int32_t* __restrict__ accept_len) {
  const int s = blockIdx.x * blockDim.x + threadIdx.x;
  if (s >= S) return;
  int A = 0;
  for (int j = 1; j <= n_causal - 1; ++j) {
    if (draft[(size_t)s * draft_width + (j - 1)] != argmax_out[(size_t)s * R + (j - 1)]) break;
    A = j;
  }
  accept_len[s] = A;
}

}  // namespace dvs

using namespace dvs;

extern "C" int top1_confidence(const void* logits, int32_t dtype, int32_t rows, int32_t V,
                               int32_t* argmax_out, float* conf_out, int32_t* err_word,
                               void* stream) {
  clear_error();
  DVS_CHECK_ARG(logits && argmax_out && conf_out, "top1_confidence: NULL array argument");
  DVS_CHECK_ARG(rows >= 1 && V >= 1, "top1_confidence: need rows, V >= 1");
  DVS_CHECK_SUPPORTED(dtype == DVS_F32 || dtype == DVS_BF16, "top1_confidence: dtype %d", dtype);
  hipStream_t st = (hipStream_t)stream;
  if (dtype == DVS_BF16)
    hipLaunchKernelGGL(top1_conf_kernel<true>, dim3((unsigned)rows), dim3(256), 0, st, logits, V,
                       argmax_out, conf_out, err_word);
  else
    hipLaunchKernelGGL(top1_conf_kernel<false>, dim3((unsigned)rows), dim3(256), 0, st, logits, V,
                       argmax_out, conf_out, err_word);
  return launch_status("top1_confidence");
}

extern "C" int argmax_accept(const void* logits, int32_t dtype, int32_t S, int32_t R, int32_t V,
                             int32_t n_causal, const int32_t* draft, int32_t draft_width,
                             int32_t* argmax_out, int32_t* accept_len, int32_t* err_word,
                             void* stream) {
  clear_error();
  DVS_CHECK_ARG(logits && argmax_out, "argmax_accept: NULL array argument");
  DVS_CHECK_ARG(S >= 1 && R >= 1 && V >= 1, "argmax_accept: need S, R, V >= 1");
  DVS_CHECK_ARG(n_causal >= 1 && n_causal <= R, "argmax_accept: need 1 <= n_causal <= R");
  DVS_CHECK_ARG(draft_width >= n_causal - 1, "argmax_accept: draft_width < n_causal - 1");
  DVS_CHECK_ARG(draft || n_causal == 1, "argmax_accept: NULL draft");
  DVS_CHECK_SUPPORTED(dtype == DVS_F32 || dtype == DVS_BF16, "argmax_accept: dtype %d", dtype);
  const long long rows = (long long)S * R;
  DVS_CHECK_SUPPORTED(rows < (1LL << 31), "argmax_accept: too many rows");
  hipStream_t st = (hipStream_t)stream;
  if (dtype == DVS_BF16)
    hipLaunchKernelGGL(argmax_kernel<true>, dim3((unsigned)rows), dim3(512), 0, st, logits, V,
                       argmax_out, err_word);
  else
    hipLaunchKernelGGL(argmax_kernel<false>, dim3((unsigned)rows), dim3(512), 0, st, logits, V,
                       argmax_out, err_word);
  int rc = launch_status("argmax_accept(argmax)");
  if (rc || !accept_len) return rc;
  hipLaunchKernelGGL(accept_kernel, dim3((S + 255) / 256), dim3(256), 0, st, argmax_out, S, R,
                     n_causal, draft, draft_width, accept_len);
  return launch_status("argmax_accept(accept)");
}
