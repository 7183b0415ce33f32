// Stochastic acceptance for the two-forward round (Preliminaries,
// "Speculative Decoding": under sampling, the standard acceptance-rejection
// rule keeps the committed tokens distributed as the verifier's samples).
//
// At temperature T every row has the distribution softmax(z / T).  Three
// kernels serve the round:
//   row_stats_kernel    m = max z and Z = sum exp((z - m) / T) per row, one
//                       pass (running sum rescaled when m grows);
//   sample_rows_kernel  an inverse-CDF sample per row from a given uniform:
//                       the smallest index whose running weight (index
//                       order) exceeds u * total;
//   accept_sampled_kernel / final_sample_kernel
//                       d_j is accepted while u * q_j(d_j) < p_j(d_j); the
//                       final token is sampled from max(0, p - q) after a
//                       rejection, from p after B acceptances.
// Every random number is an input.  Sampling: thread t of a row's workgroup
// owns the contiguous chunk [t C, (t + 1) C), C = ceil(V / 256); chunk sums
// are scanned across the threads, the owner of u * total walks its chunk.
#include "dvs_common.h"

namespace dvs {

constexpr int SMP_THREADS = 256;

__device__ __forceinline__ void stats_merge(float& m, float& s, float om, float os, float invT) {
  const float M = fmaxf(m, om);
  const float a = m == -INFINITY ? 0.f : s * __expf((m - M) * invT);
  const float b = om == -INFINITY ? 0.f : os * __expf((om - M) * invT);
  m = M;
  s = a + b;
}

__global__ void __launch_bounds__(SMP_THREADS) row_stats_kernel(const float* __restrict__ logits,
                                                               int V, float invT,
                                                               float2* __restrict__ stats,
                                                               int32_t* err) {
  __shared__ float sm[SMP_THREADS / 64], ss[SMP_THREADS / 64];
  const float* z = logits + (size_t)blockIdx.x * V;
  const int tid = threadIdx.x;
  float m = -INFINITY, s = 0.f, nf = 0.f;
  for (int i = tid; i < V; i += SMP_THREADS) {
    const float f = z[i];
    nf = fmaf(f, 0.f, nf);
    if (f > m) {
      s = (m == -INFINITY ? 0.f : s * __expf((m - f) * invT)) + 1.f;
      m = f;
    } else if (m != -INFINITY) {
      s += __expf((f - m) * invT);
    }
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    const float om = __shfl_xor(m, off), os = __shfl_xor(s, off);
    stats_merge(m, s, om, os, invT);
  }
  if ((tid & 63) == 0) { sm[tid >> 6] = m; ss[tid >> 6] = s; }
  if (nf != nf) set_err(err, DVS_ERR_NONFINITE);
  __syncthreads();
  if (tid == 0) {
    for (int w = 1; w < SMP_THREADS / 64; ++w) stats_merge(m, s, sm[w], ss[w], invT);
    stats[blockIdx.x] = make_float2(m, s);
  }
}

// Weight of index k: p_k = exp((za_k - ma) / T) / Za, minus q_k of the second
// row (clipped at 0) when zb is given.
struct RowWeights {
  const float* za;
  float2 sa;
  const float* zb;
  float2 sb;
  float invT;
  __device__ __forceinline__ float operator()(int k) const {
    float w = __expf((za[k] - sa.x) * invT) / sa.y;
    if (zb) w = fmaxf(w - __expf((zb[k] - sb.x) * invT) / sb.y, 0.f);
    return w;
  }
};

// Inverse-CDF sample of one row by the whole workgroup; every thread returns
// the index.
__device__ int sample_row(const RowWeights& wgt, int V, float u, float* sh, int* pick) {
  const int tid = threadIdx.x;
  const int C = (V + SMP_THREADS - 1) / SMP_THREADS;
  const int lo = min(V, tid * C), hi = min(V, lo + C);
  float part = 0.f;
  int last_pos = -1;
  for (int k = lo; k < hi; ++k) {
    const float w = wgt(k);
    part += w;
    if (w > 0.f) last_pos = k;
  }
  if (tid == 0) { pick[0] = 0x7fffffff; pick[1] = -1; }
  sh[tid] = part;
  __syncthreads();
  for (int off = 1; off < SMP_THREADS; off <<= 1) {   // inclusive scan of chunk sums
    const float v = tid >= off ? sh[tid - off] : 0.f;
    __syncthreads();
    sh[tid] += v;
    __syncthreads();
  }
  const float incl = sh[tid], excl = tid ? sh[tid - 1] : 0.f, total = sh[SMP_THREADS - 1];
  const float t = u * total;
  if (part > 0.f && t >= excl && t < incl) {
    float run = excl;
    int k = lo, found = -1;
    for (; k < hi; ++k) {
      run += wgt(k);
      if (run > t) { found = k; break; }
    }
    atomicMin(&pick[0], found >= 0 ? found : last_pos);
  }
  if (last_pos >= 0) atomicMax(&pick[1], last_pos);   // fallback: t rounded past the total
  __syncthreads();
  const int r = pick[0] != 0x7fffffff ? pick[0] : (pick[1] >= 0 ? pick[1] : 0);
  __syncthreads();
  return r;
}

// One workgroup per row of [S, R] rows; u[s * u_stride + r].
__global__ void __launch_bounds__(SMP_THREADS) sample_rows_kernel(
    const float* __restrict__ logits, const float2* __restrict__ stats, int V, float invT,
    const float* __restrict__ u, int u_stride, int R, int32_t* __restrict__ tok_out) {
  __shared__ float sh[SMP_THREADS];
  __shared__ int pick[2];
  const int row = blockIdx.x, s = row / R, r = row - s * R;
  RowWeights wgt{logits + (size_t)row * V, stats[row], nullptr, make_float2(0.f, 1.f), invT};
  const int k = sample_row(wgt, V, u[(size_t)s * u_stride + r], sh, pick);
  if (threadIdx.x == 0) tok_out[row] = k;
}

// A_s: drafts d_j (draft[s, j-1], j = 1..B) accepted while
// u[s, B + j] * q_j(d_j) < p_j(d_j); p_j from verify row j-1, q_j from draft
// row j (rows of R = B + 1 per sequence).
__global__ void accept_sampled_kernel(int S, int B, int V, float invT,
                                      const float* __restrict__ zv, const float2* __restrict__ sv,
                                      const float* __restrict__ zd, const float2* __restrict__ sd,
                                      const int32_t* __restrict__ draft, int draft_width,
                                      const float* __restrict__ u, int u_stride,
                                      int32_t* __restrict__ accept_len) {
  const int s = blockIdx.x * blockDim.x + threadIdx.x;
  if (s >= S) return;
  const int R = B + 1;
  int A = 0;
  for (int j = 1; j <= B; ++j) {
    const int d = draft[(size_t)s * draft_width + j - 1];
    if (d < 0 || d >= V) break;
    const size_t rv = (size_t)s * R + j - 1, rd = (size_t)s * R + j;
    const float p = __expf((zv[rv * V + d] - sv[rv].x) * invT) / sv[rv].y;
    const float q = __expf((zd[rd * V + d] - sd[rd].x) * invT) / sd[rd].y;
    if (!(u[(size_t)s * u_stride + B + j] * q < p)) break;
    A = j;
  }
  accept_len[s] = A;
}

// The final token of sequence s: from max(0, p_{A+1} - q_{A+1}) when A < B,
// from p_{B+1} when A = B; written to am[s, A] (the verifier-token slot the
// round's commit reads).
__global__ void __launch_bounds__(SMP_THREADS) final_sample_kernel(
    int B, int V, float invT, const float* __restrict__ zv, const float2* __restrict__ sv,
    const float* __restrict__ zd, const float2* __restrict__ sd,
    const int32_t* __restrict__ accept_len, const float* __restrict__ u, int u_stride,
    int32_t* __restrict__ am) {
  __shared__ float sh[SMP_THREADS];
  __shared__ int pick[2];
  const int s = blockIdx.x, R = B + 1;
  int A = accept_len[s];
  A = A < 0 ? 0 : (A > B ? B : A);
  const size_t rv = (size_t)s * R + A;
  RowWeights wgt{zv + rv * V, sv[rv], nullptr, make_float2(0.f, 1.f), invT};
  if (A < B) {
    wgt.zb = zd + (rv + 1) * V;
    wgt.sb = sd[rv + 1];
  }
  const int k = sample_row(wgt, V, u[(size_t)s * u_stride + 2 * B + 1], sh, pick);
  if (threadIdx.x == 0) am[rv] = k;
}

int launch_row_stats(const float* logits, int rows, int V, float invT, float2* stats,
                     int32_t* err, hipStream_t st) {
  hipLaunchKernelGGL(row_stats_kernel, dim3(rows), dim3(SMP_THREADS), 0, st, logits, V, invT,
                     stats, err);
  return launch_status("sampled round (row stats)");
}

int launch_sample_rows(const float* logits, const float2* stats, int V, float invT,
                       const float* u, int u_stride, int S, int R, int32_t* tok,
                       hipStream_t st) {
  hipLaunchKernelGGL(sample_rows_kernel, dim3(S * R), dim3(SMP_THREADS), 0, st, logits, stats, V,
                     invT, u, u_stride, R, tok);
  return launch_status("sampled round (draft samples)");
}

int launch_accept_final(int S, int B, int V, float invT, const float* zv, const float2* sv,
                        const float* zd, const float2* sd, const int32_t* draft, int draft_width,
                        const float* u, int u_stride, int32_t* accept_len, int32_t* am,
                        hipStream_t st) {
  hipLaunchKernelGGL(accept_sampled_kernel, dim3((S + 255) / 256), dim3(256), 0, st, S, B, V,
                     invT, zv, sv, zd, sd, draft, draft_width, u, u_stride, accept_len);
  int rc = launch_status("sampled round (accept)");
  if (rc) return rc;
  hipLaunchKernelGGL(final_sample_kernel, dim3(S), dim3(SMP_THREADS), 0, st, B, V, invT, zv, sv,
                     zd, sd, accept_len, u, u_stride, am);
  return launch_status("sampled round (final sample)");
}

}  // namespace dvs
