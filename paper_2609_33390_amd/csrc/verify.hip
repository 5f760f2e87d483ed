// Greedy verification (Section 2.2 accepted prefix; Section 3.3 acceptance
// rule at temperature zero; Algorithm 1(b) verify and commit): the accepted
// prefix ends at the first position where the proposal differs from the
// verifier's argmax; the verifier's token there is the correction.
#include "device_common.h"
#include "kernels.h"

namespace brisk {

namespace {

// One wavefront per block: 64 positions per ballot, the first set bit of the
// mismatch mask is the first rejection.
__global__ __launch_bounds__(256) void verify_kernel(const int32_t* __restrict__ proposal,
                                                     const int32_t* __restrict__ verifier, int B,
                                                     int L, int32_t* __restrict__ accept_len,
                                                     int32_t* __restrict__ correction) {
  const int lane = threadIdx.x & 63;
  const int b = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (b >= B) return;
  const size_t base = static_cast<size_t>(b) * L;
  int accept = L;
  for (int c = 0; c < L; c += 64) {
    const int i = c + lane;
    const bool bad = i < L && proposal[base + i] != verifier[base + i];
    const uint64_t mask = __ballot(bad);
    if (mask) {
      accept = c + __builtin_ctzll(mask);
      break;
    }
  }
  if (lane == 0) {
    accept_len[b] = accept;
    if (correction) correction[b] = accept < L ? verifier[base + accept] : -1;
  }
}

// Commit (Algorithm 1(b), verify and commit): the accepted prefix followed
// by the verifier's token at the first mismatch, padded with -1 to L + 1.
__global__ __launch_bounds__(256) void commit_kernel(const int32_t* __restrict__ proposal,
                                                     const int32_t* __restrict__ verifier, int B,
                                                     int L, int32_t* __restrict__ accept_len,
                                                     int32_t* __restrict__ committed,
                                                     int32_t* __restrict__ n_committed) {
  const int lane = threadIdx.x & 63;
  const int b = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (b >= B) return;
  const size_t base = static_cast<size_t>(b) * L;
  int accept = L;
  for (int c = 0; c < L; c += 64) {
    const int i = c + lane;
    const bool bad = i < L && proposal[base + i] != verifier[base + i];
    const uint64_t mask = __ballot(bad);
    if (mask) {
      accept = c + __builtin_ctzll(mask);
      break;
    }
  }
  const int n = accept < L ? accept + 1 : L;
  int32_t* out = committed + static_cast<size_t>(b) * (L + 1);
  for (int i = lane; i <= L; i += 64)
    out[i] = i < accept ? proposal[base + i] : (i == accept && accept < L ? verifier[base + i] : -1);
  if (lane == 0) {
    if (accept_len) accept_len[b] = accept;
    n_committed[b] = n;
  }
}

}  // namespace

void launch_commit(const int32_t* proposal, const int32_t* verifier, int B, int L,
                   int32_t* accept_len, int32_t* committed, int32_t* n_committed, hipStream_t s) {
  hipLaunchKernelGGL(commit_kernel, dim3((B + 3) / 4), dim3(256), 0, s, proposal, verifier, B, L,
                     accept_len, committed, n_committed);
}

void launch_verify(const int32_t* proposal, const int32_t* verifier, int B, int L,
                   int32_t* accept_len, int32_t* correction, hipStream_t s) {
  hipLaunchKernelGGL(verify_kernel, dim3((B + 3) / 4), dim3(256), 0, s, proposal, verifier, B, L,
                     accept_len, correction);
}

}  // namespace brisk
