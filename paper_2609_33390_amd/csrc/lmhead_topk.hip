// LM-head projection with a fused streaming top-K, and the top-K merge.
//
// Proposal logits l[r, v] = <hidden[r], lm_head[v]> (Section 3.3, Algorithm
// 1(b) first step) are produced tile by tile on bf16 MFMA with fp32
// accumulation and consumed in the same kernel: every tile is folded into
// per-(row, vocabulary group) top-K lists of 64-bit keys, so the [rows, V]
// logits are never written.  A second kernel merges the lists of one row into
// the ordered candidate set C_i = TopK(q_i, K) (Section 3.3; Appendix head
// details): logit descending, token id ascending among equal logits.
//
// Pipeline.  Each workgroup owns one row tile and a contiguous group of
// vocabulary tiles, and streams the reduction slices of all its tiles as one
// continuous sequence of stages: global memory is copied straight into LDS
// (global_load_lds, no staging registers), STAGES slices deep, so the loads
// of the next tile's first slices are already in flight while the current
// tile's top-K epilogue runs.  Each thread waits only for its own copies of
// the slice about to be read (an explicit vmcnt that leaves the younger
// slices in flight) and then meets the workgroup at a barrier.  Staged rows
// are dense with their 16-byte chunks XOR-swizzled, which keeps the MFMA
// operand reads (16 lanes, 16 rows, one chunk) free of bank conflicts.
#include "device_common.h"
#include "kernels.h"

namespace brisk {

namespace {

template <int BV_, int BR_, int WAVES_V_, int WAVES_R_, int BK_, int STAGES_>
struct TileCfg {
  static constexpr int BV = BV_, BR = BR_, WAVES_V = WAVES_V_, WAVES_R = WAVES_R_, BK = BK_;
  static constexpr int STAGES = STAGES_;
  // the epilogue stages one 16-column accumulator block of every wave at a time
  static constexpr int EPI_V = 16 * WAVES_V;
  static constexpr int NW = WAVES_V * WAVES_R, NT = 64 * NW;
  static constexpr int WV = BV / WAVES_V, WR = BR / WAVES_R, TV = WV / 16, TR = WR / 16;
  static constexpr int CPR = BK / 8;            // 16-byte chunks per staged row
  static constexpr int RPI = 64 / CPR;          // staged rows one DMA instruction fills
  static constexpr int ROWS = BV + BR;          // staged rows per stage: lm_head tile, then hidden tile
  static constexpr int NDMA = ROWS / RPI / NW;  // DMA instructions per wave per stage
  static constexpr int STAGE_BYTES = ROWS * BK * 2;
  static constexpr int TPP = NT / BR;           // epilogue threads per position
  static constexpr int EPI_BYTES = BR * EPI_V * 4;  // staged logits, [BR][EPI_V] fp32
  // The epilogue reuses the stage buffer of the slice just consumed when it
  // fits (no copy targets that buffer until the next slice begins).
  static constexpr bool EPI_ALIAS = EPI_BYTES <= STAGE_BYTES;
  static constexpr int LDS_BYTES = STAGES * STAGE_BYTES + (EPI_ALIAS ? 0 : EPI_BYTES);
  static_assert(ROWS % (RPI * NW) == 0 && BV % RPI == 0, "DMA instructions must tile the stage");
  static_assert(WV % 16 == 0 && WR % 16 == 0, "wave tile must be a multiple of 16");
  static_assert(NT % BR == 0 && (TPP & (TPP - 1)) == 0, "epilogue thread mapping");
  static_assert(BK % 32 == 0 && (CPR == 4 || CPR == 8), "reduction slice");
  static_assert(EPI_V % (4 * TPP) == 0 && EPI_V >= 32, "epilogue chunking");
  static_assert((STAGES - 2) * NDMA <= 63, "vmcnt range");
  static_assert(LDS_BYTES <= 160 * 1024, "LDS budget");
};

// 16-byte slot that holds chunk c of staged row r (an involution in c).  A
// 128-bit LDS read is served 8 lanes at a time; the MFMA operand reads put 8
// consecutive rows at one chunk in such a group, so the eight rows of every
// aligned run of 8 must land on eight different 16-byte bank groups (rows are
// CPR * 16 bytes long, so a bank line of 128 bytes holds 8 / CPR rows).
template <int CPR>
__device__ __forceinline__ int swz(int r, int c) {
  return c ^ ((r / (8 / CPR)) & (CPR - 1));
}

// 16-byte slot of chunk c (four logits) in staged logit row p: rows are
// EPI_V * 4 bytes long, and the eight rows of an aligned run of 8 put a given
// chunk on eight different bank groups (writes come 16 rows per chunk, reads
// one row per thread).
__device__ __forceinline__ int epi_slot(int p, int c) { return c ^ (p & 7); }

// Wait until at most N vector-memory operations of this thread are
// outstanding and all its LDS operations are done, then barrier.
template <int N>
__device__ __forceinline__ void stage_sync() {
  __builtin_amdgcn_s_waitcnt((N & 15) | (((N >> 4) & 3) << 14) | (7 << 4) | (0 << 8));
  asm volatile("s_barrier" ::: "memory");
}
__device__ __forceinline__ void lds_sync() { stage_sync<63>(); }

typedef __attribute__((address_space(3))) void* lds_ptr_t;

// XCD-aware block order.  Consecutive workgroup ids are dealt round-robin to
// the 8 XCDs; remapping gives each XCD a contiguous range of logical ids so
// the row tiles that share lm_head tiles run on the same L2.
__device__ __forceinline__ int xcd_remap(int bid, int nblocks) {
  constexpr int NXCD = 8;
  const int per = nblocks / NXCD;
  const int full = per * NXCD;
  if (bid >= full) return bid;
  return (bid % NXCD) * per + bid / NXCD;
}

// Whether the per-position lists fit in LDS for the in-workgroup merge (the
// stage buffers are idle by then).
template <class C, int KP>
constexpr bool kWgMerge = C::TPP > 1 && C::NT * KP * 8 <= C::LDS_BYTES;

// One workgroup per compute unit (the LDS footprint allows no more), so the
// compiler may split the whole register file among the workgroup's waves.
template <class C, int KP>
__global__ __launch_bounds__(C::NT) __attribute__((amdgpu_waves_per_eu(C::NW / 4, C::NW / 4))) void lmhead_topk_kernel(
    const uint16_t* __restrict__ H, const uint16_t* __restrict__ W, int rows, int d, int V,
    int n_rtiles, int n_vtiles, int tiles_per_group, uint64_t* __restrict__ partial, int n_parts) {
  __shared__ __align__(16) unsigned char smem[C::LDS_BYTES];

  const int tid = threadIdx.x, lane = tid & 63;
  // the wave index is uniform per wave; saying so keeps LDS bases in scalars
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wv = wave % C::WAVES_V, wr = wave / C::WAVES_V;
  const int logical = xcd_remap(blockIdx.x, gridDim.x);
  const int rt = logical % n_rtiles;
  const int group = logical / n_rtiles;
  const int r0 = rt * C::BR;
  const int vt_begin = group * tiles_per_group;
  const int n_tiles = min(tiles_per_group, n_vtiles - vt_begin);
  const int nk = (d + C::BK - 1) / C::BK;
  const int tail = (d % C::BK) / 8;  // valid chunks of the last slice (0: slice is full)

  // ---- copy issue: stage g = (tile g / nk, slice g % nk); past the end the
  // last slice is re-read so every wave issues the same number of copies.
  // Buffer resources bound-check every copy: lm_head rows >= V and hidden
  // rows >= rows read as zeros.  Byte offsets fit in 32 bits (checked on the
  // host).
  const __amdgpu_buffer_rsrc_t rw = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(W), static_cast<short>(0), static_cast<int>(static_cast<unsigned>(V) * d * 2u), 0x00020000);
  const __amdgpu_buffer_rsrc_t rh = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(H), static_cast<short>(0), static_cast<int>(static_cast<unsigned>(rows) * d * 2u), 0x00020000);
  const unsigned row_bytes = static_cast<unsigned>(d) * 2u;
  // lane part of a copy's byte offset: row lane / CPR of the instruction's
  // rows, and the chunk its slot holds (the swizzle repeats every 8 rows, so
  // it does not depend on the instruction)
  const unsigned lane_voff = static_cast<unsigned>(lane / C::CPR) * row_bytes +
                             static_cast<unsigned>(swz<C::CPR>(lane / C::CPR, lane % C::CPR)) * 16u;
  auto issue = [&](int g) {
    int tl = g / nk, kt = g % nk;
    if (tl >= n_tiles) {
      tl = n_tiles - 1;
      kt = nk - 1;
    }
    const unsigned v0 = static_cast<unsigned>((vt_begin + tl) * C::BV), k0b = static_cast<unsigned>(kt * C::BK) * 2u;
    unsigned char* base = smem + (g % C::STAGES) * C::STAGE_BYTES;
#pragma unroll
    for (int i = 0; i < C::NDMA; ++i) {
      const int j = i * C::NW + wave;
      const unsigned lv = lane_voff;
      if (j * C::RPI < C::BV) {
        const unsigned off = lv + (v0 + static_cast<unsigned>(j * C::RPI)) * row_bytes + k0b;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rw, (lds_ptr_t)(base + j * 1024), 16, off, 0, 0, 0);
      } else {
        const unsigned off = lv + static_cast<unsigned>(r0 + j * C::RPI - C::BV) * row_bytes + k0b;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rh, (lds_ptr_t)(base + j * 1024), 16, off, 0, 0, 0);
      }
    }
  };

  // per-lane parts of the MFMA operand addresses (see swz: independent of the 16-row block)
  const int l15 = lane & 15;
  int lane_off[C::BK / 32];
#pragma unroll
  for (int kk = 0; kk < C::BK / 32; ++kk)
    lane_off[kk] = (l15 * C::CPR + swz<C::CPR>(l15, kk * 4 + (lane >> 4))) * 16;

  const int ep = tid % C::BR, esub = tid / C::BR;
  uint64_t list[KP];
#pragma unroll
  for (int j = 0; j < KP; ++j) list[j] = 0;
  float thr = -INFINITY;  // logits below this cannot enter the list

  floatx4 acc[C::TV][C::TR];
#pragma unroll
  for (int a = 0; a < C::TV; ++a)
#pragma unroll
    for (int b = 0; b < C::TR; ++b) acc[a][b] = floatx4{0.f, 0.f, 0.f, 0.f};

#pragma unroll
  for (int st = 0; st < C::STAGES - 1; ++st) issue(st);

  for (int tl = 0; tl < n_tiles; ++tl) {
    for (int kt = 0; kt < nk; ++kt) {
      const int g = tl * nk + kt;
      stage_sync<(C::STAGES - 2) * C::NDMA>();  // slice g landed; everyone is done with slice g-1
      issue(g + C::STAGES - 1);                  // refills the buffer slice g-1 used
      const unsigned char* sb = smem + (g % C::STAGES) * C::STAGE_BYTES;
      if (tail && kt == nk - 1) {
        // chunks past d hold re-read data: zero them in the lm_head tile
        unsigned char* wb = smem + (g % C::STAGES) * C::STAGE_BYTES;
        const int nz = C::CPR - tail;
        for (int idx = tid; idx < C::BV * nz; idx += C::NT) {
          const int R = idx / nz, c = tail + idx % nz;
          *reinterpret_cast<uint4*>(wb + (R * C::CPR + swz<C::CPR>(R, c)) * 16) = make_uint4(0, 0, 0, 0);
        }
        lds_sync();
      }
#pragma unroll
      for (int kk = 0; kk < C::BK / 32; ++kk) {
        // all operand fragments of this 32-wide slice first, then the MFMAs,
        // so LDS latency overlaps the first products instead of every row
        bf16x8 b[C::TR], a[C::TV];
#pragma unroll
        for (int y = 0; y < C::TR; ++y)
          b[y] = *reinterpret_cast<const bf16x8*>(sb + (C::BV + wr * C::WR + y * 16) * C::CPR * 16 + lane_off[kk]);
#pragma unroll
        for (int x = 0; x < C::TV; ++x)
          a[x] = *reinterpret_cast<const bf16x8*>(sb + (wv * C::WV + x * 16) * C::CPR * 16 + lane_off[kk]);
#pragma unroll
        for (int x = 0; x < C::TV; ++x)
#pragma unroll
          for (int y = 0; y < C::TR; ++y)
            acc[x][y] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[x], b[y], acc[x][y], 0, 0, 0);
        // keep that order: every fragment read issued before the products
        __builtin_amdgcn_sched_group_barrier(0x100, C::TV + C::TR, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, C::TV * C::TR, 0);
      }
    }

    // Fused top-K over this tile.  Chunk x stages accumulator block x of
    // every wave as fp32 [position][wave_v * 16 + column]; each thread then
    // folds its position's columns into its running list.
    const int v0 = (vt_begin + tl) * C::BV;
    float* sE;
    if constexpr (C::EPI_ALIAS) {
      sE = reinterpret_cast<float*>(smem + ((tl * nk + nk - 1) % C::STAGES) * C::STAGE_BYTES);
      lds_sync();  // every wave has finished reading that slice
    } else {
      sE = reinterpret_cast<float*>(smem + C::STAGES * C::STAGE_BYTES);
    }
#pragma unroll
    for (int x = 0; x < C::TV; ++x) {
#pragma unroll
      for (int y = 0; y < C::TR; ++y) {
        const int p = wr * C::WR + y * 16 + l15;
        *reinterpret_cast<floatx4*>(sE + p * C::EPI_V + epi_slot(p, wv * 4 + (lane >> 4)) * 4) = acc[x][y];
        acc[x][y] = floatx4{0.f, 0.f, 0.f, 0.f};
      }
      lds_sync();
#pragma unroll
      for (int col = esub * 4; col < C::EPI_V; col += C::TPP * 4) {
        const floatx4 v = *reinterpret_cast<const floatx4*>(sE + ep * C::EPI_V + epi_slot(ep, col >> 2) * 4);
        // common case: none of the four logits reaches the list's smallest
        // entry, which one float compare decides; only then build keys
        const float m = fmaxf(fmaxf(v[0], v[1]), fmaxf(v[2], v[3]));
        if (m >= thr) {
          const int vid0 = v0 + (col >> 4) * C::WV + x * 16 + (col & 15);
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int vid = vid0 + q;
            const uint64_t key = make_key(v[q], static_cast<uint32_t>(vid));
            if (vid < V && key > list[KP - 1]) list_insert(list, key);
          }
          thr = list_floor(list[KP - 1]);
        }
      }
      lds_sync();
    }
  }
  stage_sync<0>();  // the trailing copies have landed; LDS is free

  // Merge the TPP lists of each position inside the workgroup (pairwise
  // tree through LDS) so one list per (row, vocabulary group) leaves.
  const int r = r0 + ep;
  if constexpr (kWgMerge<C, KP>) {
    uint64_t* sk = reinterpret_cast<uint64_t*>(smem);
#pragma unroll
    for (int j = 0; j < KP; ++j) sk[j * C::NT + tid] = list[j];
    lds_sync();
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
      lds_sync();
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

// One workgroup per row: every lane folds a strided share of the row's
// partial keys into a private sorted list, then the lists meet in butterflies
// (inside each wavefront, then across the four wavefronts through LDS).  At
// each level a lane and its partner hold sorted lists a and b; c_j =
// max(a_j, b_{KP-1-j}) is a bitonic sequence holding the KP largest keys of
// both, and a bitonic half-cleaner network sorts it, so both lanes leave the
// level with the same merged list.
__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t v, int m) {
  const uint32_t lo = __shfl_xor(static_cast<uint32_t>(v), m, kWave);
  const uint32_t hi = __shfl_xor(static_cast<uint32_t>(v >> 32), m, kWave);
  return (static_cast<uint64_t>(hi) << 32) | lo;
}

template <int KP>
__device__ __forceinline__ void butterfly_merge(uint64_t (&list)[KP], int m) {
  uint64_t c[KP];
#pragma unroll
  for (int j = 0; j < KP; ++j) {
    const uint64_t o = shfl_xor_u64(list[KP - 1 - j], m);
    c[j] = list[j] > o ? list[j] : o;
  }
#pragma unroll
  for (int s = KP / 2; s >= 1; s >>= 1) {
#pragma unroll
    for (int i = 0; i < KP; ++i) {
      if ((i & s) == 0) {
        const uint64_t hi = c[i] > c[i + s] ? c[i] : c[i + s];
        const uint64_t lo = c[i] > c[i + s] ? c[i + s] : c[i];
        c[i] = hi;
        c[i + s] = lo;
      }
    }
  }
#pragma unroll
  for (int j = 0; j < KP; ++j) list[j] = c[j];
}

// Rows below rows_prop are proposal rows (K candidates out); the rows after
// them are verifier rows, whose argmax (the top key) goes to ver_token.
template <int KP>
__global__ __launch_bounds__(256) void topk_merge_kernel(const uint64_t* __restrict__ partial,
                                                         int rows, int n_keys, int K, int rows_prop,
                                                         float* __restrict__ cand_logit,
                                                         int32_t* __restrict__ cand_id,
                                                         int32_t* __restrict__ ver_token) {
  constexpr int NT = 256, NW = NT / kWave, BATCH = 8;
  __shared__ uint64_t sk[NW][KP];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
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
  for (int m = 1; m < kWave; m <<= 1) butterfly_merge(list, m);
  if (lane == 0) {
#pragma unroll
    for (int j = 0; j < KP; ++j) sk[wave][j] = list[j];
  }
  __syncthreads();
  if (wave != 0) return;
  // lane l < NW takes wave l's list; two more levels leave the row's list in lane 0
#pragma unroll
  for (int j = 0; j < KP; ++j) list[j] = lane < NW ? sk[lane][j] : 0ull;
#pragma unroll
  for (int m = 1; m < NW; m <<= 1) butterfly_merge(list, m);
  if (lane == 0) {
    if (row >= rows_prop) {
      ver_token[row - rows_prop] = key_id(list[0]);
    } else {
#pragma unroll
      for (int j = 0; j < KP; ++j) {
        if (j < K) {
          cand_logit[static_cast<size_t>(row) * K + j] = key_logit(list[j]);
          cand_id[static_cast<size_t>(row) * K + j] = key_id(list[j]);
        }
      }
    }
  }
}

using SmallRows = TileCfg<256, 32, 4, 1, 64, 3>;    // <= 32 rows: weight streaming
using MidRows = TileCfg<256, 64, 4, 1, 64, 3>;      // <= 64 rows
using LargeRows = TileCfg<256, 256, 4, 2, 64, 2>;   // many rows: MFMA bound

constexpr int kTargetWorkgroups = 256;  // one persistent workgroup per compute unit

struct Plan {
  int cfg;  // 0 small, 1 mid, 2 large
  int n_rtiles, n_vtiles, tiles_per_group, n_groups, n_parts, KP;
};

template <class C>
Plan make_plan_for(int cfg, int rows, int V, int K) {
  Plan p{};
  p.cfg = cfg;
  p.n_rtiles = (rows + C::BR - 1) / C::BR;
  p.n_vtiles = (V + C::BV - 1) / C::BV;
  int want = kTargetWorkgroups / p.n_rtiles;
  want = want < 1 ? 1 : (want > p.n_vtiles ? p.n_vtiles : want);
  p.tiles_per_group = (p.n_vtiles + want - 1) / want;
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
               int rows_prop, uint64_t* partial, float* cand_logit, int32_t* cand_id,
               int32_t* ver_token, hipStream_t s) {
  switch (p.cfg) {
    case 0: launch_tile<SmallRows, KP>(p, H, W, rows, d, V, partial, s); break;
    case 1: launch_tile<MidRows, KP>(p, H, W, rows, d, V, partial, s); break;
    default: launch_tile<LargeRows, KP>(p, H, W, rows, d, V, partial, s); break;
  }
  hipLaunchKernelGGL((topk_merge_kernel<KP>), dim3(rows), dim3(256), 0, s, partial, rows,
                     p.n_parts * KP, K, rows_prop, cand_logit, cand_id, ver_token);
}

}  // namespace

size_t propose_workspace_bytes(int rows, int V, int K) {
  const Plan p = make_plan(rows, V, K);
  return static_cast<size_t>(rows) * p.n_parts * p.KP * sizeof(uint64_t);
}

void launch_propose(const uint16_t* H, const uint16_t* W, int rows, int d, int V, int K,
                    int rows_prop, float* cand_logit, int32_t* cand_id, int32_t* ver_token,
                    void* ws, hipStream_t s) {
  const Plan p = make_plan(rows, V, K);
  uint64_t* partial = static_cast<uint64_t*>(ws);
  switch (p.KP) {
    case 4: launch_kp<4>(p, H, W, rows, d, V, K, rows_prop, partial, cand_logit, cand_id, ver_token, s); break;
    case 8: launch_kp<8>(p, H, W, rows, d, V, K, rows_prop, partial, cand_logit, cand_id, ver_token, s); break;
    case 16: launch_kp<16>(p, H, W, rows, d, V, K, rows_prop, partial, cand_logit, cand_id, ver_token, s); break;
    case 32: launch_kp<32>(p, H, W, rows, d, V, K, rows_prop, partial, cand_logit, cand_id, ver_token, s); break;
    default: launch_kp<64>(p, H, W, rows, d, V, K, rows_prop, partial, cand_logit, cand_id, ver_token, s); break;
  }
}

}  // namespace brisk
