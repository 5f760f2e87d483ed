// LM-head projection with a fused streaming top-K, and the top-K merge.
//
// Proposal logits l[r, v] = <hidden[r], lm_head[v]> (Section 3.3, Algorithm
// 1(b) first step) are produced tile by tile on bf16 MFMA with fp32
// accumulation and consumed in the same kernel: every tile is folded into
// per-(row, slice) top-K lists of 64-bit keys, so the [rows, V] logits are
// never written.  A second kernel merges the lists of one row into the
// ordered candidate set C_i = TopK(q_i, K) (Section 3.3; Appendix head
// details): logit descending, token id ascending among equal logits.
#include "device_common.h"
#include "kernels.h"

namespace brisk {

namespace {

constexpr int BK = 64;                // reduction slice staged per step
constexpr int LDS_STRIDE = BK + 8;    // bf16 per staged row: 144 B breaks bank aliasing

// Tile geometry.  The vocabulary runs along the MFMA M dimension (A = lm_head
// rows) and the block positions along N (B = hidden rows), so one lane's four
// accumulator values are four consecutive vocabulary ids of one position.
template <int BV_, int BR_, int WAVES_V_, int WAVES_R_, int EPI_V_>
struct TileCfg {
  static constexpr int BV = BV_, BR = BR_, WAVES_V = WAVES_V_, WAVES_R = WAVES_R_;
  static constexpr int EPI_V = EPI_V_;
  static constexpr int NT = 64 * WAVES_V * WAVES_R;
  static constexpr int WV = BV / WAVES_V, WR = BR / WAVES_R;
  static constexpr int TV = WV / 16, TR = WR / 16;
  static constexpr int TPP = NT / BR;  // epilogue threads per position
  static constexpr int STAGE_BYTES = (BV + BR) * LDS_STRIDE * 2;
  static constexpr int EPI_BYTES = BR * (EPI_V + 1) * 4;
  static constexpr int LDS_BYTES = STAGE_BYTES > EPI_BYTES ? STAGE_BYTES : EPI_BYTES;
  static constexpr int W_CHUNKS = BV * BK / 8, H_CHUNKS = BR * BK / 8;
  static constexpr int W_PER_T = (W_CHUNKS + NT - 1) / NT, H_PER_T = (H_CHUNKS + NT - 1) / NT;
  static_assert(WV % 16 == 0 && WR % 16 == 0, "wave tile must be a multiple of 16");
  static_assert(NT % BR == 0, "threads must cover the positions evenly");
  static_assert(BV % EPI_V == 0 && WV % 16 == 0, "epilogue chunking");
};

// XCD-aware block order.  Consecutive workgroup ids are dealt round-robin to
// the 8 XCDs; remapping gives each XCD a contiguous range of logical tiles so
// the row tiles that share one lm_head tile run on the same L2.
__device__ __forceinline__ int xcd_remap(int bid, int nblocks) {
  constexpr int NXCD = 8;
  const int per = nblocks / NXCD;
  const int full = per * NXCD;
  if (bid >= full) return bid;
  return (bid % NXCD) * per + bid / NXCD;
}

// Whether the per-position lists fit in the kernel's LDS for the in-workgroup merge.
template <class C, int KP>
constexpr bool kWgMerge = C::TPP > 1 && C::NT * KP * 8 <= C::LDS_BYTES;

template <class C, int KP>
__global__ __launch_bounds__(C::NT) void lmhead_topk_kernel(
    const uint16_t* __restrict__ H, const uint16_t* __restrict__ W, int rows, int d, int V,
    int n_rtiles, int n_vtiles, int tiles_per_group, uint64_t* __restrict__ partial,
    int n_parts) {
  __shared__ __align__(16) unsigned char smem[C::LDS_BYTES];
  uint16_t* sW = reinterpret_cast<uint16_t*>(smem);
  uint16_t* sH = sW + C::BV * LDS_STRIDE;
  float* sL = reinterpret_cast<float*>(smem);

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wv = wave % C::WAVES_V, wr = wave / C::WAVES_V;
  const int logical = xcd_remap(blockIdx.x, gridDim.x);
  const int rt = logical % n_rtiles;         // row tile fastest: row tiles of one
  const int group = logical / n_rtiles;      // vocabulary group run side by side
  const int r0 = rt * C::BR;

  const int ep = tid % C::BR, esub = tid / C::BR;
  uint64_t list[KP];
#pragma unroll
  for (int j = 0; j < KP; ++j) list[j] = 0;

  const int vt_begin = group * tiles_per_group;
  const int vt_end = min(vt_begin + tiles_per_group, n_vtiles);
  for (int vt = vt_begin; vt < vt_end; ++vt) {
    const int v0 = vt * C::BV;
    floatx4 acc[C::TV][C::TR];
#pragma unroll
    for (int a = 0; a < C::TV; ++a)
#pragma unroll
      for (int b = 0; b < C::TR; ++b) acc[a][b] = floatx4{0.f, 0.f, 0.f, 0.f};

    uint4 rw[C::W_PER_T], rh[C::H_PER_T];
    auto load = [&](int k0) {
#pragma unroll
      for (int i = 0; i < C::W_PER_T; ++i) {
        const int c = tid + i * C::NT;
        const int row = c / (BK / 8), col = (c % (BK / 8)) * 8;
        const int v = v0 + row, k = k0 + col;
        uint4 val = make_uint4(0, 0, 0, 0);
        if (c < C::W_CHUNKS && v < V && k < d)
          val = *reinterpret_cast<const uint4*>(W + static_cast<size_t>(v) * d + k);
        rw[i] = val;
      }
#pragma unroll
      for (int i = 0; i < C::H_PER_T; ++i) {
        const int c = tid + i * C::NT;
        const int row = c / (BK / 8), col = (c % (BK / 8)) * 8;
        const int r = r0 + row, k = k0 + col;
        uint4 val = make_uint4(0, 0, 0, 0);
        if (c < C::H_CHUNKS && r < rows && k < d)
          val = *reinterpret_cast<const uint4*>(H + static_cast<size_t>(r) * d + k);
        rh[i] = val;
      }
    };
    auto store = [&]() {
#pragma unroll
      for (int i = 0; i < C::W_PER_T; ++i) {
        const int c = tid + i * C::NT;
        if (c < C::W_CHUNKS)
          *reinterpret_cast<uint4*>(sW + (c / (BK / 8)) * LDS_STRIDE + (c % (BK / 8)) * 8) = rw[i];
      }
#pragma unroll
      for (int i = 0; i < C::H_PER_T; ++i) {
        const int c = tid + i * C::NT;
        if (c < C::H_CHUNKS)
          *reinterpret_cast<uint4*>(sH + (c / (BK / 8)) * LDS_STRIDE + (c % (BK / 8)) * 8) = rh[i];
      }
    };

    load(0);
    __syncthreads();  // LDS readers of the previous tile's epilogue are done
    store();
    __syncthreads();
    for (int k0 = 0; k0 < d; k0 += BK) {
      const bool more = k0 + BK < d;
      if (more) load(k0 + BK);
#pragma unroll
      for (int kk = 0; kk < BK; kk += 32) {
        bf16x8 a[C::TV], b[C::TR];
        const int koff = kk + (lane >> 4) * 8;
#pragma unroll
        for (int t = 0; t < C::TV; ++t)
          a[t] = *reinterpret_cast<const bf16x8*>(
              sW + (wv * C::WV + t * 16 + (lane & 15)) * LDS_STRIDE + koff);
#pragma unroll
        for (int t = 0; t < C::TR; ++t)
          b[t] = *reinterpret_cast<const bf16x8*>(
              sH + (wr * C::WR + t * 16 + (lane & 15)) * LDS_STRIDE + koff);
#pragma unroll
        for (int x = 0; x < C::TV; ++x)
#pragma unroll
          for (int y = 0; y < C::TR; ++y)
            acc[x][y] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[x], b[y], acc[x][y], 0, 0, 0);
      }
      __syncthreads();
      if (more) store();
      __syncthreads();
    }

    // Fused top-K: stage EPI_V vocabulary columns of the tile at a time as
    // fp32 [position][column] in LDS; every thread folds the columns of its
    // position into its running list.
#pragma unroll
    for (int c0 = 0; c0 < C::BV; c0 += C::EPI_V) {
#pragma unroll
      for (int x = 0; x < C::TV; ++x) {
        const int vbase = wv * C::WV + x * 16;
        if (vbase >= c0 && vbase < c0 + C::EPI_V) {
#pragma unroll
          for (int y = 0; y < C::TR; ++y) {
            const int p = wr * C::WR + y * 16 + (lane & 15);
            const int vl = vbase - c0 + (lane >> 4) * 4;
#pragma unroll
            for (int q = 0; q < 4; ++q) sL[p * (C::EPI_V + 1) + vl + q] = acc[x][y][q];
          }
        }
      }
      __syncthreads();
      for (int col = esub; col < C::EPI_V; col += C::TPP) {
        const int v = v0 + c0 + col;
        if (v < V) {
          const uint64_t key = make_key(sL[ep * (C::EPI_V + 1) + col], static_cast<uint32_t>(v));
          if (key > list[KP - 1]) list_insert(list, key);
        }
      }
      __syncthreads();
    }
  }

  // Merge the TPP lists of each position inside the workgroup (pairwise
  // tree through LDS) so one list per (row, vocabulary group) leaves the
  // kernel.  Lists are stored [slot][thread] so neighbouring threads touch
  // neighbouring words.
  const int r = r0 + ep;
  if constexpr (kWgMerge<C, KP>) {
    uint64_t* sk = reinterpret_cast<uint64_t*>(smem);
    __syncthreads();
#pragma unroll
    for (int j = 0; j < KP; ++j) sk[j * C::NT + tid] = list[j];
    __syncthreads();
#pragma unroll
    for (int s = C::TPP / 2; s >= 1; s >>= 1) {
      if (esub < s) {
        const int other = (esub + s) * C::BR + ep;
#pragma unroll
        for (int j = 0; j < KP; ++j) {
          const uint64_t key = sk[j * C::NT + other];
          if (key > list[KP - 1]) list_insert(list, key);
        }
#pragma unroll
        for (int j = 0; j < KP; ++j) sk[j * C::NT + tid] = list[j];
      }
      __syncthreads();
    }
    if (esub == 0 && r < rows) {
      uint64_t* dst = partial + (static_cast<size_t>(r) * n_parts + group) * KP;
#pragma unroll
      for (int j = 0; j < KP; ++j) dst[j] = list[j];
    }
  } else {
    if (r < rows) {
      uint64_t* dst =
          partial + (static_cast<size_t>(r) * n_parts + static_cast<size_t>(group) * C::TPP + esub) * KP;
#pragma unroll
      for (int j = 0; j < KP; ++j) dst[j] = list[j];
    }
  }
}

// One workgroup per row: every thread folds a strided share of the row's
// partial keys into a private list, then the lists are merged pairwise through
// LDS; thread 0's list is the row's ordered top-KP.
template <int KP>
__global__ __launch_bounds__(256) void topk_merge_kernel(const uint64_t* __restrict__ partial,
                                                         int rows, int n_keys, int K,
                                                         float* __restrict__ cand_logit,
                                                         int32_t* __restrict__ cand_id) {
  constexpr int NT = 256, BATCH = 4;
  __shared__ uint64_t sk[KP * NT];
  const int tid = threadIdx.x;
  const int row = blockIdx.x;
  const uint64_t* src = partial + static_cast<size_t>(row) * n_keys;
  uint64_t list[KP];
#pragma unroll
  for (int j = 0; j < KP; ++j) list[j] = 0;
  for (int i0 = tid; i0 < n_keys; i0 += NT * BATCH) {
    uint64_t kb[BATCH];
#pragma unroll
    for (int q = 0; q < BATCH; ++q) {
      const int i = i0 + q * NT;
      kb[q] = i < n_keys ? src[i] : 0ull;
    }
#pragma unroll
    for (int q = 0; q < BATCH; ++q)
      if (kb[q] > list[KP - 1]) list_insert(list, kb[q]);
  }
#pragma unroll
  for (int j = 0; j < KP; ++j) sk[j * NT + tid] = list[j];
  __syncthreads();
  for (int s = NT / 2; s >= 1; s >>= 1) {
    if (tid < s) {
#pragma unroll
      for (int j = 0; j < KP; ++j) {
        const uint64_t key = sk[j * NT + tid + s];
        if (key > list[KP - 1]) list_insert(list, key);
      }
#pragma unroll
      for (int j = 0; j < KP; ++j) sk[j * NT + tid] = list[j];
    }
    __syncthreads();
  }
  if (tid < K) {
    const uint64_t key = sk[tid * NT];
    cand_logit[static_cast<size_t>(row) * K + tid] = key_logit(key);
    cand_id[static_cast<size_t>(row) * K + tid] = key_id(key);
  }
}

using SmallRows = TileCfg<256, 32, 4, 1, 256>;   // <= 32 rows: weight streaming
using MidRows = TileCfg<256, 64, 4, 1, 128>;     // <= 64 rows
using LargeRows = TileCfg<256, 128, 2, 2, 64>;   // many rows: MFMA bound

struct Plan {
  int cfg;        // 0 small, 1 mid, 2 large
  int BV, BR, TPP;
  int n_rtiles, n_vtiles, tiles_per_group, n_groups, n_parts, KP;
};

template <class C>
Plan make_plan_for(int cfg, int rows, int V, int K) {
  Plan p{};
  p.cfg = cfg;
  p.BV = C::BV;
  p.BR = C::BR;
  p.TPP = C::TPP;
  p.n_rtiles = (rows + C::BR - 1) / C::BR;
  p.n_vtiles = (V + C::BV - 1) / C::BV;
  p.tiles_per_group = 1;
  p.n_groups = (p.n_vtiles + p.tiles_per_group - 1) / p.tiles_per_group;
  p.KP = K <= 4 ? 4 : K <= 8 ? 8 : K <= 16 ? 16 : K <= 32 ? 32 : 64;
  const bool wg_merge = p.KP == 4    ? kWgMerge<C, 4>
                        : p.KP == 8  ? kWgMerge<C, 8>
                        : p.KP == 16 ? kWgMerge<C, 16>
                        : p.KP == 32 ? kWgMerge<C, 32>
                                     : kWgMerge<C, 64>;
  p.n_parts = p.n_groups * (wg_merge ? 1 : C::TPP);
  return p;
}

Plan make_plan(int rows, int V, int K) {
  if (rows <= 32) return make_plan_for<SmallRows>(0, rows, V, K);
  if (rows <= 64) return make_plan_for<MidRows>(1, rows, V, K);
  return make_plan_for<LargeRows>(2, rows, V, K);
}

template <class C, int KP>
void launch_tile(const Plan& p, const uint16_t* H, const uint16_t* W, int rows, int d, int V,
                 uint64_t* partial, hipStream_t s) {
  const int nblocks = p.n_rtiles * p.n_groups;
  hipLaunchKernelGGL((lmhead_topk_kernel<C, KP>), dim3(nblocks), dim3(C::NT), 0, s, H, W, rows, d,
                     V, p.n_rtiles, p.n_vtiles, p.tiles_per_group, partial, p.n_parts);
}

template <int KP>
void launch_kp(const Plan& p, const uint16_t* H, const uint16_t* W, int rows, int d, int V, int K,
               uint64_t* partial, float* cand_logit, int32_t* cand_id, hipStream_t s) {
  switch (p.cfg) {
    case 0: launch_tile<SmallRows, KP>(p, H, W, rows, d, V, partial, s); break;
    case 1: launch_tile<MidRows, KP>(p, H, W, rows, d, V, partial, s); break;
    default: launch_tile<LargeRows, KP>(p, H, W, rows, d, V, partial, s); break;
  }
  hipLaunchKernelGGL((topk_merge_kernel<KP>), dim3(rows), dim3(256), 0, s, partial, rows,
                     p.n_parts * KP, K, cand_logit, cand_id);
}

}  // namespace

size_t propose_workspace_bytes(int rows, int V, int K) {
  const Plan p = make_plan(rows, V, K);
  return static_cast<size_t>(rows) * p.n_parts * p.KP * sizeof(uint64_t);
}

void launch_propose(const uint16_t* H, const uint16_t* W, int rows, int d, int V, int K,
                    float* cand_logit, int32_t* cand_id, void* ws, hipStream_t s) {
  const Plan p = make_plan(rows, V, K);
  uint64_t* partial = static_cast<uint64_t*>(ws);
  switch (p.KP) {
    case 4: launch_kp<4>(p, H, W, rows, d, V, K, partial, cand_logit, cand_id, s); break;
    case 8: launch_kp<8>(p, H, W, rows, d, V, K, partial, cand_logit, cand_id, s); break;
    case 16: launch_kp<16>(p, H, W, rows, d, V, K, partial, cand_logit, cand_id, s); break;
    case 32: launch_kp<32>(p, H, W, rows, d, V, K, partial, cand_logit, cand_id, s); break;
    default: launch_kp<64>(p, H, W, rows, d, V, K, partial, cand_logit, cand_id, s); break;
  }
}

}  // namespace brisk
