// argmax_accept: vocabulary top-1 per window row, then greedy acceptance.
//
// Top-1 (the verifier's greedy prediction; appendix "AR-Equivalence and
// Equality Testing" uses top-1 decoding): the largest logit wins, the lowest
// index among equal maxima, -0.0 == +0.0.  Each value is mapped to an
// order-preserving unsigned key (sign-magnitude -> two's-complement order)
// after folding -0.0 onto +0.0; (key, index) pairs are reduced with
// "larger key, then smaller index" packed into one 64-bit max.
//
// Acceptance (method "Self-Speculative Decoding"; appendix item Accept):
// a_j = top1(row j-1); A = longest prefix of the draft with d_j == a_j.
//
// The argmax is a pure HBM stream: one workgroup per row, 16-byte loads with
// several in flight per thread, wavefront shuffles, then LDS across waves.
#include "dvs_common.h"

namespace dvs {

__device__ __forceinline__ uint32_t key_bf16(uint32_t b, bool& nonfinite) {
  b &= 0xffffu;
  if ((b & 0x7fffu) == 0) b = 0;                        // -0.0 -> +0.0
  if ((b & 0x7f80u) == 0x7f80u) nonfinite = true;
  return (b & 0x8000u) ? (~b & 0xffffu) : (b | 0x8000u);
}

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
__global__ void __launch_bounds__(256) argmax_kernel(const void* __restrict__ logits, int V,
                                                     int32_t* __restrict__ argmax_out,
                                                     int32_t* err) {
  constexpr int EPV = BF16 ? 8 : 4;   // elements per 16-byte vector
  constexpr int UNR = 8;              // vectors in flight per thread
  __shared__ uint64_t sred[4];
  const size_t row = blockIdx.x;
  const int tid = threadIdx.x;
  const char* base = (const char*)logits + row * (size_t)V * (BF16 ? 2 : 4);
  bool nonfinite = false;
  uint32_t bk = 0;
  int bi = 0x7fffffff;

  // vectorised body when the row start is 16-byte aligned
  const bool aligned = ((((uintptr_t)base) & 15) == 0);
  const int nvec = aligned ? V / EPV : 0;
  int v0 = 0;
  for (; v0 + UNR * 256 <= nvec; v0 += UNR * 256) {
    u32x4 buf[UNR];
#pragma unroll
    for (int u = 0; u < UNR; ++u) buf[u] = ((const u32x4*)base)[v0 + u * 256 + tid];
#pragma unroll
    for (int u = 0; u < UNR; ++u) {
      const int e0 = (v0 + u * 256 + tid) * EPV;
#pragma unroll
      for (int e = 0; e < EPV; ++e) {
        const uint32_t w = buf[u][BF16 ? (e >> 1) : e];
        const uint32_t bits = BF16 ? ((e & 1) ? (w >> 16) : (w & 0xffffu)) : w;
        const uint32_t k = BF16 ? key_bf16(bits, nonfinite) : key_f32(bits, nonfinite);
        if (k > bk) { bk = k; bi = e0 + e; }
      }
    }
  }
  for (int vi = v0 + tid; vi < nvec; vi += 256) {
    const u32x4 x = ((const u32x4*)base)[vi];
#pragma unroll
    for (int e = 0; e < EPV; ++e) {
      const uint32_t w = x[BF16 ? (e >> 1) : e];
      const uint32_t bits = BF16 ? ((e & 1) ? (w >> 16) : (w & 0xffffu)) : w;
      const uint32_t k = BF16 ? key_bf16(bits, nonfinite) : key_f32(bits, nonfinite);
      if (k > bk) { bk = k; bi = vi * EPV + e; }
    }
  }
  // scalar tail (and the whole row when unaligned)
  for (int i = nvec * EPV + tid; i < V; i += 256) {
    uint32_t k;
    if (BF16) k = key_bf16(((const uint16_t*)base)[i], nonfinite);
    else k = key_f32(((const uint32_t*)base)[i], nonfinite);
    if (k > bk || (k == bk && i < bi)) { bk = k; bi = i; }
  }

  uint64_t best = (bi == 0x7fffffff) ? 0 : pack_ki(bk, bi);
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    const uint64_t o = shfl_xor_u64(best, off);
    best = o > best ? o : best;
  }
  if ((tid & 63) == 0) sred[tid >> 6] = best;
  if (nonfinite) set_err(err, DVS_ERR_NONFINITE);
  __syncthreads();
  if (tid == 0) {
    uint64_t b = sred[0];
    for (int i = 1; i < 4; ++i) b = sred[i] > b ? sred[i] : b;
    argmax_out[row] = 0x7fffffff - (int)(uint32_t)(b & 0xffffffffu);
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

extern "C" int argmax_accept(const void* logits, int32_t dtype, int32_t S, int32_t R, int32_t V,
                             int32_t n_causal, const int32_t* draft, int32_t draft_width,
                             int32_t* argmax_out, int32_t* accept_len, int32_t* err_word,
                             void* stream) {
  clear_error();
  DVS_CHECK_ARG(logits && argmax_out && accept_len, "argmax_accept: NULL array argument");
  DVS_CHECK_ARG(S >= 1 && R >= 1 && V >= 1, "argmax_accept: need S, R, V >= 1");
  DVS_CHECK_ARG(n_causal >= 1 && n_causal <= R, "argmax_accept: need 1 <= n_causal <= R");
  DVS_CHECK_ARG(draft_width >= n_causal - 1, "argmax_accept: draft_width < n_causal - 1");
  DVS_CHECK_ARG(draft || n_causal == 1, "argmax_accept: NULL draft");
  DVS_CHECK_SUPPORTED(dtype == DVS_F32 || dtype == DVS_BF16, "argmax_accept: dtype %d", dtype);
  const long long rows = (long long)S * R;
  DVS_CHECK_SUPPORTED(rows < (1LL << 31), "argmax_accept: too many rows");
  hipStream_t st = (hipStream_t)stream;
  if (dtype == DVS_BF16)
    hipLaunchKernelGGL(argmax_kernel<true>, dim3((unsigned)rows), dim3(256), 0, st, logits, V,
                       argmax_out, err_word);
  else
    hipLaunchKernelGGL(argmax_kernel<false>, dim3((unsigned)rows), dim3(256), 0, st, logits, V,
                       argmax_out, err_word);
  int rc = launch_status("argmax_accept(argmax)");
  if (rc) return rc;
  hipLaunchKernelGGL(accept_kernel, dim3((S + 255) / 256), dim3(256), 0, st, argmax_out, S, R,
                     n_causal, draft, draft_width, accept_len);
  return launch_status("argmax_accept(accept)");
}
