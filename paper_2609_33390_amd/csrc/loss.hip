// Corrector training loss, forward (Appendix "Candidate-Refinement Head
// Details", Eq. head_training_loss; Algorithm 1(a), corrector training).
//
// At position j of a block with candidate set S_j: p_S = the verifier
// distribution restricted to S_j and renormalised, q_S = the base proposal
// distribution restricted to S_j, r = softmax of the refined logits;
// l_j = CE(p_S, r) + beta KL(q_S || r).  Only the positions whose
// verification is reached count: the accepted prefix and the first rejected
// position (every position of a fully accepted block).  The loss is the mean
// of l_j over those positions.
//
// One workgroup per position: its four wavefronts take the verifier logits
// <E_out[v_k], h_j> of the candidates (dot products over d), then wavefront 0
// holds candidate k in lane k for the three log-softmaxes.  A second launch
// adds the per-position losses in a fixed order.
#include "device_common.h"
#include "kernels.h"

namespace brisk {

namespace {

__device__ __forceinline__ bool reached(const int32_t* accept_len, int r, int L) {
  const int b = r / L, j = r % L;
  return j <= accept_len[b];
}

__global__ __launch_bounds__(256) void loss_pos_kernel(const uint16_t* __restrict__ Hv,
                                                       const uint16_t* __restrict__ W,
                                                       const int32_t* __restrict__ cand_id,
                                                       const float* __restrict__ cand_logit,
                                                       const float* __restrict__ refined,
                                                       const int32_t* __restrict__ accept_len, int L,
                                                       int K, int d, int V, float beta,
                                                       float* __restrict__ loss_pos,
                                                       float* __restrict__ ce_out,
                                                       float* __restrict__ kl_out) {
  __shared__ float s_lp[64];
  const int r = blockIdx.x;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (!reached(accept_len, r, L)) {
    if (threadIdx.x == 0) {
      loss_pos[r] = 0.f;
      if (ce_out) ce_out[r] = 0.f;
      if (kl_out) kl_out[r] = 0.f;
    }
    return;
  }
  const uint16_t* h = Hv + static_cast<size_t>(r) * d;
  for (int k = wave; k < K; k += 4) {
    const uint16_t* w = W + static_cast<size_t>(clamp_id(cand_id[static_cast<size_t>(r) * K + k], V)) * d;
    float s = 0.f;
    for (int c = lane * 8; c < d; c += 64 * 8) {
      const uint4 a = *reinterpret_cast<const uint4*>(w + c);
      const uint4 b = *reinterpret_cast<const uint4*>(h + c);
      s += bf16_lo(a.x) * bf16_lo(b.x) + bf16_hi(a.x) * bf16_hi(b.x);
      s += bf16_lo(a.y) * bf16_lo(b.y) + bf16_hi(a.y) * bf16_hi(b.y);
      s += bf16_lo(a.z) * bf16_lo(b.z) + bf16_hi(a.z) * bf16_hi(b.z);
      s += bf16_lo(a.w) * bf16_lo(b.w) + bf16_hi(a.w) * bf16_hi(b.w);
    }
    s = wave_sum(s);
    if (lane == 0) s_lp[k] = s;
  }
  __syncthreads();
  if (wave != 0) return;
  const bool on = lane < K;
  const float lp = on ? s_lp[lane] : -INFINITY;
  const float lq = on ? cand_logit[static_cast<size_t>(r) * K + lane] : -INFINITY;
  const float lr = on ? refined[static_cast<size_t>(r) * K + lane] : -INFINITY;
  // log-softmax over the K lanes of each of the three logit vectors
  const float mp = wave_allmax(lp), mq = wave_allmax(lq), mr = wave_allmax(lr);
  const float zp = wave_allsum(on ? __expf(lp - mp) : 0.f);
  const float zq = wave_allsum(on ? __expf(lq - mq) : 0.f);
  const float zr = wave_allsum(on ? __expf(lr - mr) : 0.f);
  const float log_p = lp - mp - __logf(zp), log_q = lq - mq - __logf(zq), log_r = lr - mr - __logf(zr);
  const float ce = wave_allsum(on ? -__expf(log_p) * log_r : 0.f);
  const float kl = wave_allsum(on ? __expf(log_q) * (log_q - log_r) : 0.f);
  if (lane == 0) {
    loss_pos[r] = ce + beta * kl;
    if (ce_out) ce_out[r] = ce;
    if (kl_out) kl_out[r] = kl;
  }
}

// mean over the reached positions: per-thread strided partial sums, then a
// fixed-order tree, so the result does not depend on scheduling
__global__ __launch_bounds__(256) void loss_mean_kernel(const float* __restrict__ loss_pos,
                                                        const int32_t* __restrict__ accept_len,
                                                        int rows, int L, float* __restrict__ out) {
  __shared__ double s_sum[256];
  __shared__ int s_cnt[256];
  double sum = 0.0;
  int cnt = 0;
  for (int r = threadIdx.x; r < rows; r += 256) {
    if (reached(accept_len, r, L)) {
      sum += loss_pos[r];
      ++cnt;
    }
  }
  s_sum[threadIdx.x] = sum;
  s_cnt[threadIdx.x] = cnt;
  __syncthreads();
  for (int s = 128; s >= 1; s >>= 1) {
    if (static_cast<int>(threadIdx.x) < s) {
      s_sum[threadIdx.x] += s_sum[threadIdx.x + s];
      s_cnt[threadIdx.x] += s_cnt[threadIdx.x + s];
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    out[0] = s_cnt[0] > 0 ? static_cast<float>(s_sum[0] / s_cnt[0]) : 0.f;
    out[1] = static_cast<float>(s_cnt[0]);
  }
}

}  // namespace

void launch_corrector_loss(const uint16_t* ver_hidden, const uint16_t* lm_head, const int32_t* cand_id,
                           const float* cand_logit, const float* refined, const int32_t* accept_len,
                           int B, int L, int K, int d, int V, float beta, float* loss_pos, float* ce,
                           float* kl, float* loss_mean, hipStream_t s) {
  const int rows = B * L;
  hipLaunchKernelGGL(loss_pos_kernel, dim3(rows), dim3(256), 0, s, ver_hidden, lm_head, cand_id,
                     cand_logit, refined, accept_len, L, K, d, V, beta, loss_pos, ce, kl);
  hipLaunchKernelGGL(loss_mean_kernel, dim3(1), dim3(256), 0, s, loss_pos, accept_len, rows, L,
                     loss_mean);
}

}  // namespace brisk
