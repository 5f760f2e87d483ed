// Acceptance-profile statistics of verified blocks (Section 3.2, Eq.
// nonuniform_tpf and Eq. brisk_weighting; Appendix "Brisk Backbone", Eq.
// idlm_tpf_instantiation).
//
// From the accepted-prefix lengths L_b in [0, M] of many verified blocks:
// a_i = 1 - rejected_i / reached_i (block b reaches positions 1..L_b + 1 and
// is rejected at L_b + 1 when L_b < M), survival A_k = prod_{j<=k} a_j, the
// ISD tokens per forward TPF = (2 + sum_{k=1}^{M-1} A_k) / (2 - A_M) and
// FPT = 1 / TPF, the position sensitivities w_raw_i = -dFPT/dz_i under the
// log-odds z_i = log(a_i / (1 - a_i)), and the mean-one weights
// w_i = M w_raw_i / (sum_j w_raw_j + eps).
//
// Two launches: workgroups histogram disjoint slices of the lengths into
// private partial histograms (no atomics on global memory, so the counts do
// not depend on scheduling), then one workgroup adds the partials and
// evaluates the closed forms in fp64.
#include "device_common.h"
#include "kernels.h"

namespace brisk {

namespace {

constexpr int kHistThreads = 256;
constexpr int kMaxHistGroups = 256;
constexpr int kBlocksPerGroup = 4096;

int hist_groups(int n_blocks) {
  const int g = (n_blocks + kBlocksPerGroup - 1) / kBlocksPerGroup;
  return g < 1 ? 1 : (g > kMaxHistGroups ? kMaxHistGroups : g);
}

__global__ __launch_bounds__(kHistThreads) void accept_hist_kernel(const int32_t* __restrict__ len,
                                                                   int n_blocks, int M,
                                                                   uint32_t* __restrict__ part) {
  // M < 64: every thread owns a private column of counters (no atomics, no
  // conflicting updates); otherwise one shared histogram with LDS atomics
  extern __shared__ uint32_t h[];
  const bool priv = M < kWave;
  const int cols = priv ? kHistThreads : 1;
  for (int j = threadIdx.x; j < (M + 1) * cols; j += kHistThreads) h[j] = 0;
  __syncthreads();
  const int per = (n_blocks + gridDim.x - 1) / gridDim.x;
  const int b0 = blockIdx.x * per;
  const int b1 = min(b0 + per, n_blocks);
  constexpr int BATCH = 8;
  for (int bb = b0; bb < b1; bb += kHistThreads * BATCH) {
    int Ls[BATCH];
#pragma unroll
    for (int q = 0; q < BATCH; ++q) {
      const int b = bb + q * kHistThreads + threadIdx.x;
      Ls[q] = b < b1 ? len[b] : -1;
    }
#pragma unroll
    for (int q = 0; q < BATCH; ++q) {
      const int b = bb + q * kHistThreads + threadIdx.x;
      if (b >= b1) continue;
      const int L = Ls[q] < 0 ? 0 : (Ls[q] > M ? M : Ls[q]);
      if (priv) h[L * kHistThreads + threadIdx.x] += 1u;
      else atomicAdd(&h[L], 1u);
    }
  }
  __syncthreads();
  if (priv) {
    // bin j: sum of the 256 private counters (each thread adds its row of 4)
    for (int j = 0; j <= M; ++j) {
      uint32_t v = h[j * kHistThreads + threadIdx.x];
      v += __shfl_xor(v, 1, kWave);
      v += __shfl_xor(v, 2, kWave);
      v += __shfl_xor(v, 4, kWave);
      v += __shfl_xor(v, 8, kWave);
      v += __shfl_xor(v, 16, kWave);
      v += __shfl_xor(v, 32, kWave);
      __syncthreads();
      if ((threadIdx.x & 63) == 0) h[j * kHistThreads + threadIdx.x] = v;  // wave totals in place
      __syncthreads();
      if (threadIdx.x == 0)
        part[static_cast<size_t>(blockIdx.x) * (M + 1) + j] =
            h[j * kHistThreads] + h[j * kHistThreads + 64] + h[j * kHistThreads + 128] + h[j * kHistThreads + 192];
    }
  } else {
    for (int j = threadIdx.x; j <= M; j += kHistThreads)
      part[static_cast<size_t>(blockIdx.x) * (M + 1) + j] = h[j];
  }
}

__global__ __launch_bounds__(kHistThreads) void accept_profile_kernel(const uint32_t* __restrict__ part,
                                                                      int groups, int M, double eps,
                                                                      double* __restrict__ a_out,
                                                                      double* __restrict__ raw_out,
                                                                      double* __restrict__ w_out,
                                                                      double* __restrict__ tpf_fpt) {
  extern __shared__ double sm[];
  double* cnt = sm;              // [M + 1] block counts per accepted length
  __shared__ uint32_t c32[1025];
  double* a = cnt + (M + 1);     // [M]
  double* A = a + M;             // [M + 1] survival
  double* S = A + (M + 1);       // [M + 1] S_i = sum_{k=i}^{M-1} A_k
  double* R = S + (M + 1);       // [M] raw sensitivities
  __shared__ double s_num, s_den, s_sum;
  // add the partial histograms: every (group, length) entry is one load, a
  // batch of loads in flight per thread, integer LDS atomics (order-free)
  for (int j = threadIdx.x; j <= M; j += kHistThreads) c32[j] = 0;
  __syncthreads();
  const int n_ent = groups * (M + 1);
  constexpr int BATCH = 8;
  for (int e0 = 0; e0 < n_ent; e0 += kHistThreads * BATCH) {
    uint32_t v[BATCH];
#pragma unroll
    for (int q = 0; q < BATCH; ++q) {
      const int e = e0 + q * kHistThreads + threadIdx.x;
      v[q] = e < n_ent ? part[e] : 0u;
    }
#pragma unroll
    for (int q = 0; q < BATCH; ++q) {
      const int e = e0 + q * kHistThreads + threadIdx.x;
      if (e < n_ent && v[q]) atomicAdd(&c32[e % (M + 1)], v[q]);
    }
  }
  __syncthreads();
  for (int j = threadIdx.x; j <= M; j += kHistThreads) cnt[j] = static_cast<double>(c32[j]);
  __syncthreads();
  if (threadIdx.x == 0) {
    // reached_i = #{L >= i-1}, rejected_i = #{L = i-1}
    double reach = 0.0;
    for (int j = 0; j <= M; ++j) reach += cnt[j];
    for (int i = 1; i <= M; ++i) {
      const double rej = cnt[i - 1];
      a[i - 1] = reach > 0.0 ? 1.0 - rej / reach : 1.0;
      reach -= rej;
    }
    A[0] = 1.0;
    for (int k = 1; k <= M; ++k) A[k] = A[k - 1] * a[k - 1];
    double num = 2.0;
    for (int k = 1; k <= M - 1; ++k) num += A[k];
    S[M] = 0.0;
    for (int i = M - 1; i >= 1; --i) S[i] = S[i + 1] + A[i];
    s_num = num;
    s_den = 2.0 - A[M];
  }
  __syncthreads();
  const double num = s_num, den = s_den;
  for (int i = 1 + threadIdx.x; i <= M; i += kHistThreads) {
    const double Si = i <= M - 1 ? S[i] : 0.0;
    const double r = (1.0 - a[i - 1]) * (A[M] * num + den * Si) / (num * num);
    raw_out[i - 1] = r;
    a_out[i - 1] = a[i - 1];
    R[i - 1] = r;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    double sum = 0.0;
    for (int i = 0; i < M; ++i) sum += R[i];
    s_sum = sum;
    tpf_fpt[0] = num / den;
    tpf_fpt[1] = den / num;
  }
  __syncthreads();
  for (int i = threadIdx.x; i < M; i += kHistThreads) w_out[i] = M * R[i] / (s_sum + eps);
}

}  // namespace

size_t accept_profile_workspace_bytes(int n_blocks, int M) {
  return static_cast<size_t>(hist_groups(n_blocks)) * (M + 1) * sizeof(uint32_t);
}

void launch_accept_profile(const int32_t* accept_len, int n_blocks, int M, double eps, double* a,
                           double* w_raw, double* w, double* tpf_fpt, void* ws, hipStream_t s) {
  const int groups = hist_groups(n_blocks);
  uint32_t* part = static_cast<uint32_t*>(ws);
  const size_t hist_lds = (M + 1) * sizeof(uint32_t) * (M < kWave ? kHistThreads : 1);
  hipLaunchKernelGGL(accept_hist_kernel, dim3(groups), dim3(kHistThreads), hist_lds, s,
                     accept_len, n_blocks, M, part);
  hipLaunchKernelGGL(accept_profile_kernel, dim3(1), dim3(kHistThreads), (5 * M + 3) * sizeof(double), s,
                     part, groups, M, eps, a, w_raw, w, tpf_fpt);
}

}  // namespace brisk
