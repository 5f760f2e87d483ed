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
#include <mutex>

#include "device_common.h"
#include "kernels.h"

// Fixed scratch of the propose call that allocates nothing
// (brisk_propose_block_noalloc): the per-(row, vocabulary group) key lists
// live here instead of in a caller's workspace.  Each GPU holds its own copy
// for the life of the process; host code never uses this name as an address
// (it is a host-side stand-in), only the device address that
// hipGetSymbolAddress returns for it on each device.
static __device__ __align__(256) unsigned char scratch[BRISK_NOALLOC_SCRATCH_BYTES];

namespace brisk {

namespace {

template <int BV_, int BR_, int WAVES_V_, int WAVES_R_, int BK_, int STAGES_, bool SPLIT_ = true>
struct TileCfg {
  static constexpr int BV = BV_, BR = BR_, WAVES_V = WAVES_V_, WAVES_R = WAVES_R_, BK = BK_;
  static constexpr int STAGES = STAGES_;
  // the epilogue stages one 16-column accumulator block of every wave at a time
  static constexpr int EPI_V = 16 * WAVES_V;
  static constexpr int NW = WAVES_V * WAVES_R, NT = 64 * NW;
  // Small row tiles defer a tile's top-K into the next tile's reduction
  // loop: the whole tile of logits waits in its own buffer, [TV][BR][EPI_V]
  // fp32, while the copies of the next tile stream.
  static constexpr bool DEFER = BR <= 32;
  // There the top-K runs on wavefronts of its own (SPLIT_): NCW consumer
  // waves own the key lists and fold the staged tile while the NW compute
  // waves issue the next tile's copies and products, one of each per SIMD.
  // Folded by the compute waves, the fold sat on the copy loop's path: the
  // sampling pass spent 40 of its 221 us at 32 rows on it.  NTA threads in
  // all; NC own lists.
  static constexpr int NCW = DEFER && SPLIT_ ? NW : 0;
  static constexpr int NTA = 64 * (NW + NCW);
  static constexpr int NC = NCW ? 64 * NCW : NT;
  static constexpr int WV = BV / WAVES_V, WR = BR / WAVES_R, TV = WV / 16, TR = WR / 16;
  static constexpr int CPR = BK / 8;            // 16-byte chunks per staged row
  static constexpr int RPI = 64 / CPR;          // staged rows one DMA instruction fills
  static constexpr int ROWS = BV + BR;          // staged rows per stage: lm_head tile, then hidden tile
  static constexpr int NDMA = ROWS / RPI / NW;  // DMA instructions per wave per stage
  static constexpr int STAGE_BYTES = ROWS * BK * 2;
  static constexpr int TPP = NC / BR;           // epilogue threads per position
  static constexpr int EPI_BYTES = BR * EPI_V * 4;  // staged logits, [BR][EPI_V] fp32
  // The epilogue reuses the stage buffer of the slice just consumed when it
  // fits (no copy targets that buffer until the next slice begins).
  static constexpr bool EPI_ALIAS = EPI_BYTES <= STAGE_BYTES;
  static constexpr int DEF_BYTES = DEFER ? BR * BV * 4 : 0;
  // the epilogue's list floors, [BR][TPP] fp32, follow the buffers (one
  // LDS object for the whole kernel: a second one makes the compiler wait
  // for every outstanding LDS copy before each LDS read)
  static constexpr int THR_OFF = STAGES * STAGE_BYTES + (DEFER ? DEF_BYTES : (EPI_ALIAS ? 0 : EPI_BYTES));
  // Per-position thresholds, queue counters and an overflow flag of the
  // filtered epilogue (see the kernel), after the floors.
  static constexpr int POS_OFF = THR_OFF + NC * 4;
  // Filtered epilogue: the list of the second thread of every position as
  // floats, [BR][16], read by the first to bound the position's KP-th key.
  static constexpr int U_OFF = POS_OFF + BR * 8 + 16;
  static constexpr int U_BYTES = BR >= 128 ? BR * 16 * 4 : 0;
  static constexpr int LDS_BYTES = U_OFF + U_BYTES;
  // Sampling pass: each thread keeps up to CKR candidate ids of its row in
  // registers, so testing a token against them touches no memory (a global
  // load there waits for every copy in flight, and so does an LDS read, which
  // the compiler cannot tell apart from the copies' destinations).
  static constexpr int CKR = BR <= 64 ? 16 : 8;
  // survivors a position's queue holds per tile (the queues use the stage
  // buffer the epilogue aliases)
  static constexpr int QCAP = STAGE_BYTES / (BR * 8);
  static_assert(ROWS % (RPI * NW) == 0 && BV % RPI == 0, "DMA instructions must tile the stage");
  static_assert(WV % 16 == 0 && WR % 16 == 0, "wave tile must be a multiple of 16");
  static_assert(NT % BR == 0 && (TPP & (TPP - 1)) == 0, "epilogue thread mapping");
  static_assert(BK % 32 == 0 && (CPR == 4 || CPR == 8 || CPR == 16 || CPR == 32), "reduction slice");
  static_assert(EPI_V % (4 * TPP) == 0 && EPI_V >= 32, "epilogue chunking");
  static_assert(!DEFER || TPP % 4 == 0, "row floors of the deferred fold are read as float4");
  static_assert((STAGES - 2) * NDMA <= 63, "vmcnt range");
  static_assert(LDS_BYTES <= 160 * 1024, "LDS budget");
};

// 16-byte slot that holds chunk c of staged row r (an involution in c).  A
// 128-bit LDS read is served 16 lanes a cycle (256 bytes, 16 slots of 16
// bytes): lanes l..l+7 with l+16..l+23, as the LDS counters of these tiles
// show (four busy cycles a read and no conflicts with 128-byte rows, eight
// with 512-byte rows and r & 7 below).  The MFMA operand reads put in such a
// group rows r..r+7 (r a multiple of 8) at chunks c and c + 1, c even, so
// those 16 accesses must fall on 16 different slots of a 256-byte line.
// Rows of 8 chunks: two rows share a line, and c ^ (r & 7) puts chunks c and
// c + 1 of a row on slots of opposite parity, each row pair on its own half.
// Rows of 16 chunks or more all start a line: c ^ 2 (r & 7) spreads the
// eight rows over the even slots, and c + 1 = c ^ 1 takes the odd ones.
// (Rows shorter than 8 chunks: 8 / CPR rows share a 128-byte run.)
template <int CPR>
__device__ __forceinline__ int swz(int r, int c) {
  if constexpr (CPR >= 16) return c ^ ((r & 7) << 1);
  else if constexpr (CPR == 8) return c ^ (r & 7);
  else return c ^ ((r / (8 / CPR)) & (CPR - 1));
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

// Row tile and vocabulary group of a logical workgroup.  The workgroups of
// one XCD run in near lockstep over the reduction, so per slice the XCD's L2
// fetches one hidden-state slice per row tile and one lm_head slice per group
// among them, and serves every other request: 32 workgroups as 8 row tiles x
// 4 groups fetch 12 slices, against 18 as 16 x 2 (4096 rows: 1 -> 0.98 of
// the pass time).  Other grids take row tiles fastest.
__device__ __forceinline__ void tile_of(int logical, int nblocks, int n_rtiles, int n_groups, int& rt, int& group) {
  rt = logical % n_rtiles;
  group = logical / n_rtiles;
  if (nblocks == 8 * 32 && n_rtiles % 8 == 0 && n_groups % 4 == 0) {
    const int i = logical % 32, blk = logical / 32, nrb = n_rtiles / 8;
    rt = (blk % nrb) * 8 + i % 8;
    group = (blk / nrb) * 4 + i / 8;
  }
}

// Equal vocabulary shares for weight-streaming shapes, and list floors shared
// among the epilogue threads of a row (both described where they are used).
constexpr bool kEvenShares = true;
constexpr bool kRowThreshold = true;  // where TPP <= 2, and in the deferred fold

// Whether the per-position lists fit in LDS for the in-workgroup merge (the
// stage buffers are idle by then).
template <class C, int KP>
constexpr bool kWgMerge = C::TPP > 1 && C::NC * KP * 8 + C::NC * 8 <= C::LDS_BYTES;

// Bitonic sort of N floats into descending order, in registers.
template <int N>
__device__ __forceinline__ void sort_desc(float (&a)[N]) {
#pragma unroll
  for (int k = 2; k <= N; k <<= 1)
#pragma unroll
    for (int j = k >> 1; j > 0; j >>= 1)
#pragma unroll
      for (int i = 0; i < N; ++i) {
        const int l = i ^ j;
        if (l > i) {
          const float hi = fmaxf(a[i], a[l]), lo = fminf(a[i], a[l]);
          const bool down = (i & k) == 0;
          a[i] = down ? hi : lo;
          a[l] = down ? lo : hi;
        }
      }
}

// R-th largest (R >= 1) of the union of two descending lists of N floats:
// taking j entries from a and R - j from b, min(a[j-1], b[R-j-1]) has at
// least R entries at or above it, and the best split reaches the R-th.
template <int N, int R>
__device__ __forceinline__ float union_rank(const float (&a)[N], const float (&b)[N]) {
  static_assert(R >= 1 && R <= 2 * N, "rank within the union");
  float t = -INFINITY;
#pragma unroll
  for (int j = (R > N ? R - N : 0); j <= (R < N ? R : N); ++j) {
    const float x = j > 0 ? a[j > 0 ? j - 1 : 0] : INFINITY;
    const float y = R - j > 0 ? b[R - j > 0 ? R - j - 1 : 0] : INFINITY;
    t = fmaxf(t, fminf(x, y));
  }
  return t;
}

// Verifier rows of stochastic verification: logits are scaled by 1/T, each
// thread also keeps a running log-sum-exp (max, scaled sum) of its logits,
// and the keys rank s + G (a Gumbel variate per token from Philox4x32-10
// keyed by (key0, key1), counter (token / 4, row, 0, 0), word token % 4).
struct SampleArgs {
  float inv_T;
  uint32_t key0, key1;
  float2* lse_part;         // [rows, n_parts] (max, sum of exp(s - max))
  const int32_t* cand_id;   // [rows, K]: tokens kept out of the key lists
  int K;
};

// Candidate filter of a row: bit (id mod 64) of a 64-bit mask is set for
// every candidate id (clamped into [0, V) as everywhere else), so a clear bit
// rules a token out at once; a set bit is settled against the ids themselves,
// loaded eight at a time so one memory latency covers eight of them.
__device__ __forceinline__ uint64_t candidate_mask(const SampleArgs& sa, int r, int V) {
  const int32_t* ids = sa.cand_id + static_cast<size_t>(r) * sa.K;
  uint64_t m = 0;
  for (int k0 = 0; k0 < sa.K; k0 += 8) {
    int32_t t[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) t[q] = k0 + q < sa.K ? ids[k0 + q] : -1;
#pragma unroll
    for (int q = 0; q < 8; ++q)
      if (k0 + q < sa.K) m |= 1ull << (clamp_id(t[q], V) & 63);
  }
  return m;
}

__device__ __forceinline__ bool is_candidate(const SampleArgs& sa, uint64_t mask, int r, int v, int V) {
  if (!((mask >> (v & 63)) & 1ull)) return false;
  const int32_t* ids = sa.cand_id + static_cast<size_t>(r) * sa.K;
  int hit = 0;
  for (int k0 = 0; k0 < sa.K; k0 += 8) {
    int32_t t[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) t[q] = k0 + q < sa.K ? ids[k0 + q] : -1;
#pragma unroll
    for (int q = 0; q < 8; ++q) hit |= (k0 + q < sa.K) & (clamp_id(t[q], V) == v);
  }
  return hit != 0;
}

// The same test against the row's ids held in registers (already clamped;
// unused slots hold -1).
template <int N>
__device__ __forceinline__ bool is_candidate_reg(const int (&ids)[N], uint64_t mask, int v) {
  if (!((mask >> (v & 63)) & 1ull)) return false;
  int hit = 0;
#pragma unroll
  for (int k = 0; k < N; ++k) hit |= ids[k] == v;
  return hit != 0;
}

// One workgroup per compute unit (the LDS footprint allows no more), so the
// compiler may split the whole register file among the workgroup's waves.
template <class C, int KP, bool SAMPLE = false>
__global__ __launch_bounds__(C::NTA) __attribute__((amdgpu_waves_per_eu(C::NTA / 256, C::NTA / 256))) void lmhead_topk_kernel(
    const uint16_t* __restrict__ H, const uint16_t* __restrict__ W, int rows, int d, int V,
    int n_rtiles, int n_groups, int tiles_per_group, int even, uint64_t* __restrict__ partial,
    int n_parts, SampleArgs sa) {
  __shared__ __align__(16) unsigned char smem[C::LDS_BYTES];
  float* const s_thr = reinterpret_cast<float*>(smem + C::THR_OFF);  // list floors, [position][TPP]
  // Filtered epilogue (large-row tiles, plain pass): each lane tests its own
  // accumulators against its positions' thresholds (lower bounds of each
  // position's KP-th largest logit: the KP-th of the position's two lists,
  // raised on the first two tiles by a seed from the tile itself) and
  // queues only the survivors, which the
  // position's list owners then fold.  A tile whose queues overflow, and a
  // first tile that is not whole, take the full path.  Lists of up to 16
  // keys; longer lists keep the full path on every tile.
  constexpr bool kFilt = !SAMPLE && C::BR >= 128 && C::EPI_ALIAS && KP <= 16;
  constexpr bool kSeed = kFilt;
  float* const s_pthr = reinterpret_cast<float*>(smem + C::POS_OFF);        // [BR]
  int* const s_cnt = reinterpret_cast<int*>(smem + C::POS_OFF + C::BR * 4);  // [BR]
  int* const s_flag = reinterpret_cast<int*>(smem + C::POS_OFF + C::BR * 8);

  const int tid = threadIdx.x, lane = tid & 63;
  // the wave index is uniform per wave; saying so keeps LDS bases in scalars
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wv = wave % C::WAVES_V, wr = wave / C::WAVES_V;
  const int logical = xcd_remap(blockIdx.x, gridDim.x);
  int rt, group;
  tile_of(logical, static_cast<int>(gridDim.x), n_rtiles, n_groups, rt, group);
  const int r0 = rt * C::BR;
  // Vocabulary rows [vb, ve) of this group: runs of whole tiles, or (even)
  // equal shares cut at multiples of 16, so that every compute unit streams
  // the same number of rows; the last tile of a share is partly masked.
  int vb, ve;
  if (even) {
    vb = group == 0 ? 0 : static_cast<int>(static_cast<long long>(group) * V / n_groups) & ~15;
    ve = group + 1 == n_groups ? V : static_cast<int>(static_cast<long long>(group + 1) * V / n_groups) & ~15;
  } else {
    vb = group * tiles_per_group * C::BV;
    ve = min(V, vb + tiles_per_group * C::BV);
  }
  // Tiles of the share: runs of BV rows, the last one partial.  (A short
  // extra tile at the end, to shorten the top-K that cannot overlap with
  // copies, costs more: a slice takes time whether or not its rows exist.)
  const int n_tiles = (ve - vb + C::BV - 1) / C::BV;
  auto tile_start = [&](int t) { return vb + t * C::BV; };
  auto tile_end = [&](int t) { return min(ve, vb + (t + 1) * C::BV); };
  const int nk = (d + C::BK - 1) / C::BK;
  const int tail = (d % C::BK) / 8;  // valid chunks of the last slice (0: slice is full)

  // ---- copy issue: stage g = (tile g / nk, slice g % nk); nothing past the
  // last slice.  Buffer resources bound-check every copy: the lm_head
  // resource starts at row vb and ends at row ve, so rows past the group's
  // share read as zeros without touching memory, and hidden rows >= rows
  // read as zeros.  Byte offsets fit in 32 bits (checked on the host).
  const __amdgpu_buffer_rsrc_t rw = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(W + static_cast<size_t>(vb) * d), static_cast<short>(0),
      static_cast<int>(static_cast<unsigned>(ve - vb) * d * 2u), 0x00020000);
  const __amdgpu_buffer_rsrc_t rh = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(H), static_cast<short>(0), static_cast<int>(static_cast<unsigned>(rows) * d * 2u), 0x00020000);
  const unsigned row_bytes = static_cast<unsigned>(d) * 2u;
  // lane part of a copy's byte offset: row lane / CPR of the instruction's
  // rows, and the chunk its slot holds.  The swizzle repeats every 8 rows, so
  // it does not depend on the instruction when one covers 8 rows or more;
  // with fewer (slices of 128 bytes per row or more) it depends on the
  // instruction's first row modulo 8.
  const unsigned lane_voff = static_cast<unsigned>(lane / C::CPR) * row_bytes +
                             static_cast<unsigned>(swz<C::CPR>(lane / C::CPR, lane % C::CPR)) * 16u;
  auto lane_voff_of = [&](int j) -> unsigned {
    if constexpr (C::RPI >= 8) {
      return lane_voff;
    } else {
      const int r = j * C::RPI + lane / C::CPR;
      return static_cast<unsigned>(lane / C::CPR) * row_bytes +
             static_cast<unsigned>(swz<C::CPR>(r, lane % C::CPR)) * 16u;
    }
  };
  auto issue = [&](int g) {
    const int tl = g / nk, kt = g % nk;
    if (tl >= n_tiles) return;
    const unsigned v0 = static_cast<unsigned>(tl * C::BV), k0b = static_cast<unsigned>(kt * C::BK) * 2u;
    unsigned char* base = smem + (g % C::STAGES) * C::STAGE_BYTES;
#pragma unroll
    for (int i = 0; i < C::NDMA; ++i) {
      const int j = i * C::NW + wave;
      const unsigned lv = lane_voff_of(j);
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

  // roles (see TileCfg::NCW); without consumer waves every wave does both
  const bool computer = C::NCW == 0 || wave < C::NW;
  const bool consumer = C::NCW == 0 || wave >= C::NW;
  const int ctid = C::NCW ? (consumer ? tid - C::NT : 0) : tid;  // index among the list owners
  const int ep = ctid % C::BR, esub = ctid / C::BR;
  uint64_t list[KP];
#pragma unroll
  for (int j = 0; j < KP; ++j) list[j] = 0;
  float thr = -INFINITY;  // logits below this cannot enter the list
  float lse_m = -INFINITY, lse_s = 0.f;  // SAMPLE: running log-sum-exp
  // The sampling epilogue keeps at most two generator blocks live (one in
  // the large-row tile), and so does a 64-key list: unrolled further, the
  // large-row tile runs out of registers and the others outgrow the full
  // unroll of the chunk loop, whose accumulator indexing must stay static.
  constexpr int kColFull = C::EPI_V / (C::TPP * 4);
  constexpr int kColTwo = kColFull < 2 ? kColFull : 2;
  constexpr int kColUnroll = SAMPLE ? (C::BR >= 128 ? 1 : kColTwo) : (KP >= 64 ? kColTwo : kColFull);
  const bool row_ok = r0 + ep < rows;
  uint64_t cmask = 0;
  constexpr int kCandRegs = SAMPLE ? C::CKR : 1;
  int cid_reg[kCandRegs];
#pragma unroll
  for (int k = 0; k < kCandRegs; ++k) cid_reg[k] = -1;
  const bool cand_reg = SAMPLE && sa.K <= C::CKR;
  if constexpr (SAMPLE) {
    if (consumer && row_ok) {
      cmask = candidate_mask(sa, r0 + ep, V);
      if (cand_reg) {
#pragma unroll
        for (int k = 0; k < kCandRegs; ++k)
          if (k < sa.K) cid_reg[k] = clamp_id(sa.cand_id[static_cast<size_t>(r0 + ep) * sa.K + k], V);
      }
    }
  }

  // One float4 of staged logits (columns col..col+3 of chunk x) of this
  // thread's position folded into its list.
  auto consume = [&](const float* buf, int x, int col, int v0, int vend) {
    const int vid0 = v0 + (col >> 4) * C::WV + x * 16 + (col & 15);  // a multiple of 4
    if (vid0 >= vend) return;  // columns past the tile's last row
    floatx4 v = *reinterpret_cast<const floatx4*>(buf + ep * C::EPI_V + epi_slot(ep, col >> 2) * 4);
    if constexpr (SAMPLE) {
      float m4 = -INFINITY;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        v[q] *= sa.inv_T;
        if (vid0 + q < vend) m4 = fmaxf(m4, v[q]);
      }
      if (m4 > lse_m) {
        lse_s *= __expf(lse_m - m4);
        lse_m = m4;
      }
      const uint4 w = philox4x32_10(make_uint4(static_cast<uint32_t>(vid0) >> 2, static_cast<uint32_t>(r0 + ep), 0u, 0u),
                                    sa.key0, sa.key1);
      const uint32_t wq[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        if (vid0 + q < vend) lse_s += __expf(v[q] - lse_m);
        v[q] += gumbel_of(wq[q]);
      }
    }
    // common case: none of the four logits reaches the list's smallest
    // entry, which one float compare decides; only then build keys
    const float m = fmaxf(fmaxf(v[0], v[1]), fmaxf(v[2], v[3]));
    if (m >= thr) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int vid = vid0 + q;
        const uint64_t key = make_key(v[q], static_cast<uint32_t>(vid));
        if (vid < vend && v[q] >= thr && key > list[KP - 1]) {
          // sampling keeps candidates out: their draws use exact weights
          if constexpr (SAMPLE) {
            if (!row_ok) continue;
            if (cand_reg ? is_candidate_reg(cid_reg, cmask, vid) : is_candidate(sa, cmask, r0 + ep, vid, V))
              continue;
          }
          list_insert(list, key);
        }
      }
      thr = fmaxf(thr, list_floor(list[KP - 1]));
    }
  };
  // deferred top-K: item i is float4 (i % kColFull) of chunk i / kColFull
  constexpr int kItems = C::TV * kColFull;
  float* const sD = reinterpret_cast<float*>(smem + C::STAGES * C::STAGE_BYTES);
  int pend = kItems, pend_v0 = 0, pend_end = 0;
  auto consume_item = [&](int i) {
    if (!consumer) return;
    if constexpr (kRowThreshold) {
      // Every list's floor bounds its row's KP-th key from below, so the
      // largest floor the row's lists have published filters this one too
      // (a floor being replaced is still a bound: no barrier needed).  Once
      // the lists are full, far fewer logits reach the shared floor than a
      // list's own, and the fold skips their keys and candidate tests.
      const floatx4* f = reinterpret_cast<const floatx4*>(s_thr + ep * C::TPP);
#pragma unroll
      for (int e = 0; e < C::TPP / 4; ++e) {
        const floatx4 t = f[e];
        thr = fmaxf(thr, fmaxf(fmaxf(t[0], t[1]), fmaxf(t[2], t[3])));
      }
    }
    const int x = i / kColFull;
    consume(sD + x * C::BR * C::EPI_V, x, esub * 4 + (i % kColFull) * C::TPP * 4, pend_v0, pend_end);
    if constexpr (kRowThreshold) s_thr[ep * C::TPP + esub] = thr;
  };

  // Filtered epilogue: the position's threshold for the tile, the KP-th
  // largest key of its two lists together after the previous tile (every
  // list entry is a logit of the position, so the KP-th of any of them bounds
  // the KP-th of the whole vocabulary from below); the first owner also
  // clears the position's queue counter there.
  // The second list owner publishes its floors at the end of a tile; the
  // first takes the bound at the start of the next tile's epilogue, before
  // the barrier that opens it (the next tile's slice barriers order the two,
  // so no barrier of its own is needed).
  float* const s_u = reinterpret_cast<float*>(smem + C::U_OFF);
  auto publish_floors = [&]() {
    if (esub == 1) {
#pragma unroll
      for (int j = 0; j < KP; ++j) s_u[ep * 16 + j] = list_floor(list[j]);
    }
  };
  auto take_bound = [&]() {
    if (esub == 0) {
      float a[KP], b[KP];
#pragma unroll
      for (int j = 0; j < KP; ++j) {
        a[j] = list_floor(list[j]);
        b[j] = s_u[ep * 16 + j];
      }
      thr = fmaxf(thr, union_rank<KP, KP>(a, b));
      s_pthr[ep] = row_ok ? thr : INFINITY;  // padding rows (all logits 0) queue nothing
      s_cnt[ep] = 0;
    }
  };

  if constexpr (C::DEFER && kRowThreshold) {
    for (int i = tid; i < C::NC; i += C::NTA) s_thr[i] = -INFINITY;
  }
  if constexpr (kFilt) {
    static_assert(!kFilt || (C::TPP == 2 && KP <= 16 && C::WAVES_V == 4), "filtered epilogue layout");
    for (int i = tid; i < C::BR; i += C::NTA) {
      s_pthr[i] = -INFINITY;
      s_cnt[i] = 0;
    }
    if (tid == 0) s_flag[0] = 0;  // first read after the pipeline's barriers
  }

  floatx4 acc[C::TV][C::TR];
#pragma unroll
  for (int a = 0; a < C::TV; ++a)
#pragma unroll
    for (int b = 0; b < C::TR; ++b) acc[a][b] = floatx4{0.f, 0.f, 0.f, 0.f};

  if (computer) {
#pragma unroll
    for (int st = 0; st < C::STAGES - 1; ++st) issue(st);
  }

  for (int tl = 0; tl < n_tiles; ++tl) {
    for (int kt = 0; kt < nk; ++kt) {
      const int g = tl * nk + kt;
      // slice g landed; everyone is done with slice g-1 (in the last slices
      // fewer younger copies exist, so wait for all)
      if (g + C::STAGES - 2 < n_tiles * nk) stage_sync<(C::STAGES - 2) * C::NDMA>();
      else stage_sync<0>();
      if (computer) issue(g + C::STAGES - 1);    // refills the buffer slice g-1 used
      const unsigned char* sb = smem + (g % C::STAGES) * C::STAGE_BYTES;
      if (tail && kt == nk - 1) {
        // chunks past d hold re-read data: zero them in the lm_head tile
        unsigned char* wb = smem + (g % C::STAGES) * C::STAGE_BYTES;
        const int nz = C::CPR - tail;
        for (int idx = tid; idx < C::BV * nz; idx += C::NTA) {
          const int R = idx / nz, c = tail + idx % nz;
          *reinterpret_cast<uint4*>(wb + (R * C::CPR + swz<C::CPR>(R, c)) * 16) = make_uint4(0, 0, 0, 0);
        }
        lds_sync();
      }
      if (computer) {
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
      if constexpr (C::DEFER) {
        // the previous tile's top-K, spread evenly over this tile's slices
        while (pend < kItems && kt * kItems >= pend * nk) consume_item(pend++);
      }
    }

    // Fused top-K over this tile.  Chunk x stages accumulator block x of
    // every wave as fp32 [position][wave_v * 16 + column]; each thread then
    // folds its position's columns into its running list.
    const int v0 = tile_start(tl), vend = tile_end(tl);
    if constexpr (C::DEFER) {
      while (pend < kItems) consume_item(pend++);  // tiles shorter than kItems slices
      lds_sync();  // every thread has finished with the previous tile's logits
      if (computer) {
#pragma unroll
        for (int x = 0; x < C::TV; ++x) {
#pragma unroll
          for (int y = 0; y < C::TR; ++y) {
            const int p = wr * C::WR + y * 16 + l15;
            *reinterpret_cast<floatx4*>(sD + (x * C::BR + p) * C::EPI_V + epi_slot(p, wv * 4 + (lane >> 4)) * 4) =
                acc[x][y];
            acc[x][y] = floatx4{0.f, 0.f, 0.f, 0.f};
          }
        }
      }
      lds_sync();
      pend = 0;
      pend_v0 = v0;
      pend_end = vend;
      if (tl == n_tiles - 1) {
        while (pend < kItems) consume_item(pend++);
      }
      continue;
    }
    if constexpr (kFilt) {
      if (tl > 0) take_bound();  // published by the barrier below
    }
    float* sE;
    if constexpr (C::EPI_ALIAS) {
      sE = reinterpret_cast<float*>(smem + ((tl * nk + nk - 1) % C::STAGES) * C::STAGE_BYTES);
      lds_sync();  // every wave has finished reading that slice
    } else {
      sE = reinterpret_cast<float*>(smem + C::STAGES * C::STAGE_BYTES);
    }
    if constexpr (kFilt) {
      const bool whole = vend - v0 == C::BV;
      // seed the first two tiles; after them the two lists bound tightly
      const bool seed = kSeed && whole && tl < 2;
      if (tl > 0 || seed) {
        // lane l holds, for position wr*WR + y*16 + l%16, the logits of
        // vocabulary rows wv*WV + x*16 + 4*(l/16) + q of the tile
        uint64_t* const sq = reinterpret_cast<uint64_t*>(sE);
        // Queue entry i of position p: the slot XORed with the position, so
        // that the lanes of 16 positions storing (or the list owners
        // reading) the same entry index hit different banks (rows of the
        // queue are 256 bytes apart).
        static_assert((C::QCAP & (C::QCAP - 1)) == 0, "queue slots");
        auto qslot = [](int p, int i) { return p * C::QCAP + (i ^ (p & (C::QCAP - 1))); };
        if (seed) {
          // Seed from the tile itself: each of the 16 lanes that hold a
          // position's 256 logits offers its M largest, and the KP-th
          // largest of those 16 * M logits bounds the position's KP-th from
          // below.  With M = 2 for 16 keys (one otherwise) about KP + 2
          // logits of normally spread rows pass it, well inside the queues,
          // whatever the earlier tiles left; an unlucky position only sends
          // the tile down the full path.
          constexpr int M = KP > 8 ? 2 : 1;
          float* const s_seed = sE;  // [BR][16 * M], slots permuted per position
          const int h = wv * 4 + (lane >> 4);
#pragma unroll
          for (int y = 0; y < C::TR; ++y) {
            float t1 = -INFINITY, t2 = -INFINITY;
#pragma unroll
            for (int x = 0; x < C::TV; ++x)
#pragma unroll
              for (int q = 0; q < 4; ++q) {
                const float v = acc[x][y][q];
                if constexpr (M == 2) t2 = fmaxf(t2, fminf(t1, v));
                t1 = fmaxf(t1, v);
              }
            const int p = wr * C::WR + y * 16 + l15;
            const int slot = h ^ (p & 15);  // spreads a store's 16 positions over the banks
            if constexpr (M == 2) *reinterpret_cast<float2*>(s_seed + p * 32 + slot * 2) = make_float2(t1, t2);
            else s_seed[p * 16 + slot] = t1;
          }
          lds_sync();
          if (esub == 0) {
            float a[8 * M], b[8 * M];
            const floatx4* src = reinterpret_cast<const floatx4*>(s_seed + ep * 16 * M);
#pragma unroll
            for (int c = 0; c < 4 * M; ++c) {
              const floatx4 f = src[c];
#pragma unroll
              for (int q = 0; q < 4; ++q) {
                if (c < 2 * M) a[c * 4 + q] = f[q];
                else b[(c - 2 * M) * 4 + q] = f[q];
              }
            }
            sort_desc(a);
            sort_desc(b);
            thr = fmaxf(thr, union_rank<8 * M, KP>(a, b));
            s_pthr[ep] = row_ok ? thr : INFINITY;
          }
          lds_sync();
        }
        float pt[C::TR];
#pragma unroll
        for (int y = 0; y < C::TR; ++y) pt[y] = s_pthr[wr * C::WR + y * 16 + l15];
        const int vl0 = v0 + wv * C::WV + 4 * (lane >> 4);
        if (vend - v0 < C::BV) {  // the share's last tile: rows past its end never enter
#pragma unroll
          for (int x = 0; x < C::TV; ++x)
#pragma unroll
            for (int q = 0; q < 4; ++q)
              if (vl0 + x * 16 + q >= vend)
#pragma unroll
                for (int y = 0; y < C::TR; ++y) acc[x][y][q] = -3.0e38f;
        }
        // Per position of the lane, without branches: how many of its 16
        // logits reach the threshold, the last of them and the largest logit.
        // (Branching per block of logits made the whole wavefront walk every
        // block some lane had a survivor in: about 2000 instructions a tile.)
        int cnt[C::TR], last[C::TR];
        float mx[C::TR];
#pragma unroll
        for (int y = 0; y < C::TR; ++y) {
          int c = 0, li = 0;
          float m = acc[0][y][0];
#pragma unroll
          for (int x = 0; x < C::TV; ++x)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              const float v = acc[x][y][q];
              const bool ge = v >= pt[y];
              c += ge ? 1 : 0;
              li = ge ? x * 16 + q : li;
              m = fmaxf(m, v);
            }
          cnt[y] = c;
          last[y] = li;
          mx[y] = m;
        }
        // One queue reservation per position, issued back to back (adding 0
        // where the lane has no survivor), then the survivors stored as
        // (logit bits, id): the list owners build the keys of survivors
        // only, where here every slot would pay for it.  A lane whose
        // survivors do not all fit stores none and flags the overflow, which
        // sends the whole tile down the full path.
        int base[C::TR];
#pragma unroll
        for (int y = 0; y < C::TR; ++y) base[y] = atomicAdd(&s_cnt[wr * C::WR + y * 16 + l15], cnt[y]);
        uint2* const sq2 = reinterpret_cast<uint2*>(sq);
#pragma unroll
        for (int y = 0; y < C::TR; ++y) {
          const int p = wr * C::WR + y * 16 + l15;
          const bool fits = base[y] + cnt[y] <= C::QCAP;
          if (!fits) s_flag[0] = 1;
          if (fits && cnt[y] == 1) {  // the only survivor is the largest logit
            sq2[qslot(p, base[y])] = make_uint2(__float_as_uint(mx[y]), static_cast<uint32_t>(vl0 + last[y]));
          } else if (fits && cnt[y] > 1) {
            int idx = base[y];
#pragma unroll
            for (int x = 0; x < C::TV; ++x)
#pragma unroll
              for (int q = 0; q < 4; ++q) {
                if (acc[x][y][q] >= pt[y]) {
                  sq2[qslot(p, idx)] = make_uint2(__float_as_uint(acc[x][y][q]), static_cast<uint32_t>(vl0 + x * 16 + q));
                  ++idx;
                }
              }
          }
        }
        lds_sync();
        if (s_flag[0] == 0) {  // uniform: every thread reads the same flag
          const int n = min(s_cnt[ep], C::QCAP);
          for (int i = esub; i < n; i += C::TPP) {
            const uint2 e = reinterpret_cast<const uint2*>(sq)[qslot(ep, i)];
            const uint64_t key = make_key(__uint_as_float(e.x), e.y);
            if (key > list[KP - 1]) list_insert(list, key);
          }
#pragma unroll
          for (int x = 0; x < C::TV; ++x)
#pragma unroll
            for (int y = 0; y < C::TR; ++y) acc[x][y] = floatx4{0.f, 0.f, 0.f, 0.f};
          publish_floors();
          continue;  // the next slice's barrier ends every read of the queues
        }
        // a queue overflowed: the whole tile takes the full path below
      }
      thr = fmaxf(thr, s_pthr[ep]);  // the position's bound skips logits early
    }
    // Large-row tile: one copy of the consume loop, run once per accumulator
    // block (its LDS store keeps static register indices); on this tile the
    // path runs after an overflow, on a first tile that is not whole and for
    // lists longer than 16 keys, and unrolling it per block made the kernel
    // several times larger.  Smaller tiles unroll it.
    constexpr bool kOneConsume = C::BR >= 128;
#pragma unroll (kOneConsume ? 1 : C::TV)
    for (int x = 0; x < C::TV; ++x) {
#pragma unroll
      for (int xs = 0; xs < C::TV; ++xs) {
        if (xs == x) {
#pragma unroll
          for (int y = 0; y < C::TR; ++y) {
            const int p = wr * C::WR + y * 16 + l15;
            *reinterpret_cast<floatx4*>(sE + p * C::EPI_V + epi_slot(p, wv * 4 + (lane >> 4)) * 4) = acc[xs][y];
            acc[xs][y] = floatx4{0.f, 0.f, 0.f, 0.f};
          }
        }
      }
      lds_sync();
#pragma unroll (kOneConsume ? 1 : kColUnroll)
      for (int col = esub * 4; col < C::EPI_V; col += C::TPP * 4)
        consume(sE, x, col, v0, vend);
      // Share the floors of a row's TPP lists: each thread's floor bounds the
      // row's KP-th largest key from below, so the largest of them filters
      // every list of the row.  It pays on the large-row tile (two lists per
      // row, long streams); with eight lists per row and short streams the
      // exchange costs more than the insertions it saves.
      if constexpr (kRowThreshold && C::TPP == 2) s_thr[ep * C::TPP + esub] = thr;
      lds_sync();
      if constexpr (kRowThreshold && C::TPP == 2) {
#pragma unroll
        for (int e = 0; e < C::TPP; ++e) thr = fmaxf(thr, s_thr[ep * C::TPP + e]);
      }
    }
    if constexpr (kFilt) {
      // thresholds for the next tile; counters and flag cleared (the flag
      // was read by every thread before the barriers above)
      publish_floors();
      if (tid == 0) s_flag[0] = 0;
    }
  }
  stage_sync<0>();  // the trailing copies have landed; LDS is free

  // Merge the TPP lists of each position inside the workgroup (pairwise
  // tree through LDS) so one list per (row, vocabulary group) leaves.
  const int r = r0 + ep;
  if constexpr (kWgMerge<C, KP>) {
    uint64_t* sk = reinterpret_cast<uint64_t*>(smem);
    float2* sl = reinterpret_cast<float2*>(smem + C::NC * KP * 8);
    if (consumer) {
#pragma unroll
      for (int j = 0; j < KP; ++j) sk[j * C::NC + ctid] = list[j];
      if constexpr (SAMPLE) sl[ctid] = make_float2(lse_m, lse_s);
    }
    lds_sync();
#pragma unroll
    for (int s = C::TPP / 2; s >= 1; s >>= 1) {
      if (consumer && esub < s) {
        const int other = (esub + s) * C::BR + ep;
#pragma unroll
        for (int j = 0; j < KP; ++j) {
          const uint64_t key = sk[j * C::NC + other];
          if (key > list[KP - 1]) list_insert(list, key);
        }
#pragma unroll
        for (int j = 0; j < KP; ++j) sk[j * C::NC + ctid] = list[j];
        if constexpr (SAMPLE) {
          lse_combine(lse_m, lse_s, sl[other]);
          sl[ctid] = make_float2(lse_m, lse_s);
        }
      }
      lds_sync();
    }
    if (consumer && esub == 0 && r < rows) {
      uint64_t* dst = partial + (static_cast<size_t>(r) * n_parts + group) * KP;
#pragma unroll
      for (int j = 0; j < KP; ++j) dst[j] = list[j];
      if constexpr (SAMPLE) sa.lse_part[static_cast<size_t>(r) * n_parts + group] = make_float2(lse_m, lse_s);
    }
  } else {
    if (consumer && r < rows) {
      const size_t part = static_cast<size_t>(r) * n_parts + static_cast<size_t>(group) * C::TPP + esub;
      uint64_t* dst = partial + part * KP;
#pragma unroll
      for (int j = 0; j < KP; ++j) dst[j] = list[j];
      if constexpr (SAMPLE) sa.lse_part[part] = make_float2(lse_m, lse_s);
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
// Partner exchange of the butterfly levels, all on the VALU: M = 1, 2 swap
// lanes inside quads, M = 4 and 8 pair each lane with its mirror in its
// half-row and row (lane ^ 7, lane ^ 15), and M = 16, 32 use the gfx950
// lane swaps (lane ^ 16, lane ^ 32).  Applied in the order 1, 2, 4, 8, 16,
// 32, each level joins disjoint groups of 1, 2, 4, ... lanes, as xor
// partners would.
template <int M>
__device__ __forceinline__ uint32_t lane_xchg(uint32_t v) {
  if constexpr (M == 1 || M == 2 || M == 4 || M == 8) {
    constexpr int ctrl = M == 1 ? 0xB1 : M == 2 ? 0x4E : M == 4 ? 0x141 : 0x140;
    return static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(v), ctrl, 0xF, 0xF, false));
  } else if constexpr (M == 16) {
    const auto r = __builtin_amdgcn_permlane16_swap(v, v, false, false);
    return r[0] == v ? r[1] : r[0];  // one result is the lane's own word
  } else {
    static_assert(M == 32, "partner distance");
    const auto r = __builtin_amdgcn_permlane32_swap(v, v, false, false);
    return r[0] == v ? r[1] : r[0];
  }
}

template <int M>
__device__ __forceinline__ uint64_t lane_xchg_u64(uint64_t v) {
  const uint32_t lo = lane_xchg<M>(static_cast<uint32_t>(v));
  const uint32_t hi = lane_xchg<M>(static_cast<uint32_t>(v >> 32));
  return (static_cast<uint64_t>(hi) << 32) | lo;
}

// Top KP of two descending lists a (in place) and b: c_j = max(a_j,
// b_{KP-1-j}) is bitonic and holds the KP largest keys of the pair; a bitonic
// half-cleaner network sorts it.
template <int KP>
__device__ __forceinline__ void merge_sorted(uint64_t (&a)[KP], const uint64_t (&b)[KP]) {
  uint64_t c[KP];
#pragma unroll
  for (int j = 0; j < KP; ++j) c[j] = a[j] > b[KP - 1 - j] ? a[j] : b[KP - 1 - j];
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
  for (int j = 0; j < KP; ++j) a[j] = c[j];
}

template <int M, int KP>
__device__ __forceinline__ void butterfly_merge(uint64_t (&list)[KP]) {
  uint64_t o[KP];
#pragma unroll
  for (int j = 0; j < KP; ++j) o[j] = lane_xchg_u64<M>(list[j]);
  merge_sorted(list, o);
}

// All 64 lanes end with the wavefront's top KP.
template <int KP>
__device__ __forceinline__ void wave_merge(uint64_t (&list)[KP]) {
  butterfly_merge<1>(list);
  butterfly_merge<2>(list);
  butterfly_merge<4>(list);
  butterfly_merge<8>(list);
  butterfly_merge<16>(list);
  butterfly_merge<32>(list);
}

// Fold parts pt = first, first + step, ... of a row (each a descending list
// of KP keys, as the LM-head pass writes them) into the thread's list.
template <int KP>
__device__ __forceinline__ void fold_parts(uint64_t (&list)[KP], const uint64_t* src, int n_parts, int first,
                                           int step) {
  static_assert(KP % 2 == 0, "16-byte loads");
  for (int pt = first; pt < n_parts; pt += step) {
    const uint4* p = reinterpret_cast<const uint4*>(src + static_cast<size_t>(pt) * KP);
    uint64_t kb[KP];
#pragma unroll
    for (int q = 0; q < KP / 2; ++q) {
      const uint4 u = p[q];
      kb[2 * q] = (static_cast<uint64_t>(u.y) << 32) | u.x;
      kb[2 * q + 1] = (static_cast<uint64_t>(u.w) << 32) | u.z;
    }
    merge_sorted(list, kb);
  }
}

// Rows below rows_prop are proposal rows (K candidates out); the rows after
// them are verifier rows, whose argmax (the top key) goes to ver_token.
// NW wavefronts per row: one when a row has at most 256 parts (each lane
// folds up to four, and no cross-wave stage is needed), four above that.
template <int KP, int NW>
__global__ __launch_bounds__(64 * NW) void topk_merge_kernel(const uint64_t* __restrict__ partial,
                                                             int rows, int n_keys, int K, int rows_prop,
                                                             float* __restrict__ cand_logit,
                                                             int32_t* __restrict__ cand_id,
                                                             int32_t* __restrict__ ver_token) {
  constexpr int NT = NW * kWave;
  static_assert(NW == 1 || NW == 4, "one wavefront, or two cross-wave levels");
  __shared__ uint64_t sk[NW][KP];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int row = blockIdx.x;
  const uint64_t* src = partial + static_cast<size_t>(row) * n_keys;
  uint64_t list[KP];
#pragma unroll
  for (int j = 0; j < KP; ++j) list[j] = 0;
  fold_parts(list, src, n_keys / KP, tid, NT);
  if constexpr (NW == 1) {
    // parts sit in lanes 0..n_parts-1 (and their repeats 64 apart); levels
    // past the highest occupied lane group would merge empty lists
    const int n_parts = n_keys / KP;
    butterfly_merge<1>(list);
    butterfly_merge<2>(list);
    butterfly_merge<4>(list);
    butterfly_merge<8>(list);
    if (n_parts > 16) butterfly_merge<16>(list);
    if (n_parts > 32) butterfly_merge<32>(list);
  } else {
    wave_merge(list);
  }
  if constexpr (NW == 4) {
    if (lane == 0) {
#pragma unroll
      for (int j = 0; j < KP; ++j) sk[wave][j] = list[j];
    }
    __syncthreads();
    if (wave != 0) return;
    // lane l < NW takes wave l's list; two more levels leave the row's list in lane 0
#pragma unroll
    for (int j = 0; j < KP; ++j) list[j] = lane < NW ? sk[lane][j] : 0ull;
    butterfly_merge<1>(list);
    butterfly_merge<2>(list);
  }
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

// <= 32 rows: weight streaming.  64-row tiles of 256-wide slices read each
// lm_head row in 512-byte runs, which streams about 3% faster than 256-row
// tiles of 64-wide slices (128-byte runs) and leaves more tiles for the
// deferred top-K to hide behind.
using SmallRows = TileCfg<64, 32, 4, 1, 256, 3>;
// 64-key lists take 128 registers: at two waves per SIMD they would spill,
// so that case keeps the fold in the compute waves.
using SmallRowsUnsplit = TileCfg<64, 32, 4, 1, 256, 3, false>;
using MidRows = TileCfg<256, 64, 4, 1, 64, 3>;      // <= 64 rows
using LargeRows = TileCfg<256, 256, 4, 2, 64, 2>;   // many rows: MFMA bound

constexpr int kTargetWorkgroups = 256;  // one persistent workgroup per compute unit
// The plain pass at 32 rows or fewer streams lm_head as fast from 224
// compute units (28 per XCD) as from 256 (169-170 against 172 us at 32
// rows; 192 units: 186 us) and leaves 32 free for work on another stream
// (brisk_rerank_hoist): a whole 44 us rerank beside it ends 8 us after the
// pass's 170, where beside a 256-unit pass the two took 229 us.  The
// sampling pass keeps every unit (it is 1-7 us slower on 224).
constexpr int kSmallRowsWorkgroups = 224;

struct Plan {
  int cfg;  // 0 small, 1 mid, 2 large
  int n_rtiles, n_vtiles, tiles_per_group, n_groups, n_parts, KP;
  int even;  // equal vocabulary shares instead of runs of whole tiles
};

template <class C>
Plan make_plan_for(int cfg, int rows, int V, int K, int target = kTargetWorkgroups) {
  Plan p{};
  p.cfg = cfg;
  p.n_rtiles = (rows + C::BR - 1) / C::BR;
  p.n_vtiles = (V + C::BV - 1) / C::BV;
  int want = target / p.n_rtiles;
  want = want < 1 ? 1 : (want > p.n_vtiles ? p.n_vtiles : want);
  p.tiles_per_group = (p.n_vtiles + want - 1) / want;
  p.n_groups = (p.n_vtiles + p.tiles_per_group - 1) / p.tiles_per_group;
  // Weight-streaming shapes: when runs of whole tiles leave compute units
  // idle, cut the vocabulary into one equal share per compute unit instead
  // (the partly masked last tile costs MFMA time, which these shapes have
  // to spare, but no memory traffic).
  const int want_all = target / p.n_rtiles < 1 ? 1 : target / p.n_rtiles;
  p.even = 0;
  if (kEvenShares && cfg != 2 && p.n_groups < want_all && V / want_all >= C::BV / 2) {
    p.even = 1;
    p.n_groups = want_all;
    p.tiles_per_group = (V / want_all + 16 + C::BV - 1) / C::BV;
  }
  p.KP = K <= 4 ? 4 : K <= 8 ? 8 : K <= 16 ? 16 : K <= 32 ? 32 : 64;
  const bool wg_merge = p.KP == 4    ? kWgMerge<C, 4>
                        : p.KP == 8  ? kWgMerge<C, 8>
                        : p.KP == 16 ? kWgMerge<C, 16>
                        : p.KP == 32 ? kWgMerge<C, 32>
                                     : kWgMerge<C, 64>;
  p.n_parts = p.n_groups * (wg_merge ? 1 : C::TPP);
  return p;
}

Plan make_plan(int rows, int V, int K, bool sample = false) {
  if (rows <= 32) return make_plan_for<SmallRows>(0, rows, V, K, sample ? kTargetWorkgroups : kSmallRowsWorkgroups);
  if (rows <= 64) return make_plan_for<MidRows>(1, rows, V, K);
  return make_plan_for<LargeRows>(2, rows, V, K);
}

template <class C, int KP, bool SAMPLE = false>
void launch_tile(const Plan& p, const uint16_t* H, const uint16_t* W, int rows, int d, int V,
                 uint64_t* partial, hipStream_t s, SampleArgs sa = SampleArgs{}) {
  const int nblocks = p.n_rtiles * p.n_groups;
  hipLaunchKernelGGL((lmhead_topk_kernel<C, KP, SAMPLE>), dim3(nblocks), dim3(C::NTA), 0, s, H, W, rows,
                     d, V, p.n_rtiles, p.n_groups, p.tiles_per_group, p.even, partial, p.n_parts, sa);
}

// ---------------------------------------------------------------------------
// Stochastic speculative verification (Section 3.3): per verifier row r, the
// accept test of the proposal x_r against min{1, p_r(x_r) / pi_r(x_r)} and a
// draw y_r from [p_r - pi_r]_+ by Gumbel-max.  Only the K candidates carry
// proposal mass, so every other token competes with score s + G - lse
// (s = logit / T): the LM-head pass leaves, per (row, group), the largest
// keys of s + G over the non-candidate tokens and a log-sum-exp partial.  One
// workgroup per row: merge keys and partials, take the verifier logits of the
// candidates and of x_r by dot products, then decide.
// ---------------------------------------------------------------------------
template <int KP>
__global__ __launch_bounds__(256) void spec_row_kernel(
    const uint64_t* __restrict__ partial, const float2* __restrict__ lse_part, int n_parts,
    const uint16_t* __restrict__ Hv, const uint16_t* __restrict__ W, int d, int V, int K,
    const int32_t* __restrict__ proposal, const int32_t* __restrict__ cand_id,
    const float* __restrict__ cand_prob, const float* __restrict__ u_accept, float inv_T,
    uint32_t key0, uint32_t key1, int32_t* __restrict__ row_accept, int32_t* __restrict__ row_resample) {
  constexpr int NT = 256, NW = NT / kWave;
  static_assert(NW == 4, "two cross-wave levels");
  // the first NPF tokens of each wavefront have their rows in flight before
  // anything waits (rows of up to CH * 512 elements in one batch)
  constexpr int NPF = 3, CH = 8;
  __shared__ uint64_t sk[NW][KP];
  __shared__ float2 s_lse[NW];
  __shared__ float s_logit[kWave + 1];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int row = blockIdx.x;
  const uint16_t* h = Hv + static_cast<size_t>(row) * d;
  const int x = clamp_id(proposal[row], V);
  auto token = [&](int k) { return k < K ? clamp_id(cand_id[static_cast<size_t>(row) * K + k], V) : x; };
  auto dot8 = [](float& acc, uint4 a, uint4 b) {
    acc += bf16_lo(a.x) * bf16_lo(b.x) + bf16_hi(a.x) * bf16_hi(b.x);
    acc += bf16_lo(a.y) * bf16_lo(b.y) + bf16_hi(a.y) * bf16_hi(b.y);
    acc += bf16_lo(a.z) * bf16_lo(b.z) + bf16_hi(a.z) * bf16_hi(b.z);
    acc += bf16_lo(a.w) * bf16_lo(b.w) + bf16_hi(a.w) * bf16_hi(b.w);
  };

  // (0) loads of the verifier-logit rows: the candidates (k < K) and the
  // proposal (k = K), token k on wavefront k % NW
  uint4 hv[CH], wv[NPF][CH];
#pragma unroll
  for (int i = 0; i < CH; ++i) {
    const int c = lane * 8 + i * kWave * 8;
    hv[i] = c < d ? *reinterpret_cast<const uint4*>(h + c) : make_uint4(0, 0, 0, 0);
  }
#pragma unroll
  for (int t = 0; t < NPF; ++t) {
    const int k = wave + t * NW;
    const uint16_t* w = W + static_cast<size_t>(k <= K ? token(k) : x) * d;
#pragma unroll
    for (int i = 0; i < CH; ++i) {
      const int c = lane * 8 + i * kWave * 8;
      wv[t][i] = k <= K && c < d ? *reinterpret_cast<const uint4*>(w + c) : make_uint4(0, 0, 0, 0);
    }
  }

  // (1) keys of s + G: per-lane lists, wave butterflies, then across waves
  const int n_keys = n_parts * KP;
  const uint64_t* src = partial + static_cast<size_t>(row) * n_keys;
  uint64_t list[KP];
#pragma unroll
  for (int j = 0; j < KP; ++j) list[j] = 0;
  fold_parts(list, src, n_parts, tid, NT);
  // (2) log-sum-exp partials, combined in a fixed order: strided per thread,
  // then a butterfly within the wavefront, then the wavefronts in order
  float m = -INFINITY, sm = 0.f;
  for (int i = tid; i < n_parts; i += NT) lse_combine(m, sm, lse_part[static_cast<size_t>(row) * n_parts + i]);
  wave_merge(list);
  if (lane == 0) {
#pragma unroll
    for (int j = 0; j < KP; ++j) sk[wave][j] = list[j];
  }
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1)
    lse_combine(m, sm, make_float2(__shfl_xor(m, off, kWave), __shfl_xor(sm, off, kWave)));
  if (lane == 0) s_lse[wave] = make_float2(m, sm);

  // (3) the dot products: the prefetched tokens, then any further ones
#pragma unroll
  for (int t = 0; t < NPF; ++t) {
    const int k = wave + t * NW;
    if (k > K) break;
    float acc = 0.f;
#pragma unroll
    for (int i = 0; i < CH; ++i) dot8(acc, wv[t][i], hv[i]);
    const uint16_t* w = W + static_cast<size_t>(token(k)) * d;
    for (int c = lane * 8 + CH * kWave * 8; c < d; c += kWave * 8)
      dot8(acc, *reinterpret_cast<const uint4*>(w + c), *reinterpret_cast<const uint4*>(h + c));
    acc = wave_sum(acc);
    if (lane == 0) s_logit[k] = acc;
  }
  for (int k = wave + NPF * NW; k <= K; k += NW) {
    const uint16_t* w = W + static_cast<size_t>(token(k)) * d;
    float acc = 0.f;
    for (int c = lane * 8; c < d; c += kWave * 8)
      dot8(acc, *reinterpret_cast<const uint4*>(w + c), *reinterpret_cast<const uint4*>(h + c));
    acc = wave_sum(acc);
    if (lane == 0) s_logit[k] = acc;
  }
  __syncthreads();
  if (wave != 0) return;
  float2 tot = s_lse[0];
#pragma unroll
  for (int w = 1; w < NW; ++w) lse_combine(tot.x, tot.y, s_lse[w]);
#pragma unroll
  for (int j = 0; j < KP; ++j) list[j] = lane < NW ? sk[lane][j] : 0ull;
  butterfly_merge<1>(list);
  butterfly_merge<2>(list);

  // (4) decisions with the accurate exp / log: where p_r and pi_r nearly
  // cancel, the residual weight needs every bit fp32 has
  const float lse = tot.x + logf(tot.y);
  const int32_t* ids = cand_id + static_cast<size_t>(row) * K;
  // no cand_prob: the proposal is the greedy choice, pi_r = point mass at x_r
  const float* pis = cand_prob ? cand_prob + static_cast<size_t>(row) * K : nullptr;
  auto pi_of = [&](int k, int v) { return pis ? pis[k] : (v == x ? 1.f : 0.f); };
  // residual draw: candidate k scored by lane k from its exact weight,
  // everyone else from the best key (no candidate enters the lists; score
  // s + G - lse); the best score wins, the lower id on ties
  float best = -INFINITY;
  int best_id = 0x7FFFFFFF;
  for (int k = lane; k < K; k += kWave) {
    const int v = clamp_id(ids[k], V);
    const float w = fminf(1.f, expf(s_logit[k] * inv_T - lse)) - pi_of(k, v);
    if (w <= 0.f) continue;
    const uint4 g4 = philox4x32_10(make_uint4(static_cast<uint32_t>(v) >> 2, static_cast<uint32_t>(row), 0u, 0u),
                                   key0, key1);
    const uint32_t gw[4] = {g4.x, g4.y, g4.z, g4.w};
    const float sc = logf(w) + gumbel_of(gw[v & 3]);
    if (sc > best || (sc == best && v < best_id)) {
      best = sc;
      best_id = v;
    }
  }
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    const float ob = __shfl_xor(best, off, kWave);
    const int oi = __shfl_xor(best_id, off, kWave);
    if (ob > best || (ob == best && oi < best_id)) {
      best = ob;
      best_id = oi;
    }
  }
  if (lane != 0) return;
  float pi_x = 0.f;
  for (int k = 0; k < K; ++k) {
    const int v = clamp_id(ids[k], V);
    if (v == x) pi_x += pi_of(k, v);
  }
  // p <= 1 holds exactly; the clamp keeps rounding (the dot products and the
  // log-sum-exp add in different orders) from giving weight to pi = 1
  const float p_x = fminf(1.f, expf(s_logit[K] * inv_T - lse));
  const bool accept = pi_x <= 0.f || u_accept[row] < fminf(1.f, p_x / pi_x);
  if (list[0] != 0) {
    const int v = key_id(list[0]);
    const float sc = key_logit(list[0]) - lse;
    if (sc > best || (sc == best && v < best_id)) {
      best = sc;
      best_id = v;
    }
  }
  row_accept[row] = accept ? 1 : 0;
  row_resample[row] = best_id == 0x7FFFFFFF ? x : best_id;
}

// First rejected position of each block and the token drawn there.
__global__ __launch_bounds__(256) void spec_commit_kernel(const int32_t* __restrict__ row_accept,
                                                          const int32_t* __restrict__ row_resample,
                                                          int B, int L, int32_t* __restrict__ accept_len,
                                                          int32_t* __restrict__ correction) {
  const int lane = threadIdx.x & 63;
  const int b = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (b >= B) return;
  const size_t base = static_cast<size_t>(b) * L;
  int a = L;
  for (int c = 0; c < L; c += 64) {
    const int i = c + lane;
    const uint64_t mask = __ballot(i < L && row_accept[base + i] == 0);
    if (mask) {
      a = c + __builtin_ctzll(mask);
      break;
    }
  }
  if (lane == 0) {
    accept_len[b] = a;
    if (correction) correction[b] = a < L ? row_resample[base + a] : -1;
  }
}

template <int KP>
void launch_kp_pass(const Plan& p, const uint16_t* H, const uint16_t* W, int rows, int d, int V,
                    uint64_t* partial, hipStream_t s) {
  switch (p.cfg) {
    case 0:
      if constexpr (KP >= 64) launch_tile<SmallRowsUnsplit, KP>(p, H, W, rows, d, V, partial, s);
      else launch_tile<SmallRows, KP>(p, H, W, rows, d, V, partial, s);
      break;
    case 1: launch_tile<MidRows, KP>(p, H, W, rows, d, V, partial, s); break;
    default: launch_tile<LargeRows, KP>(p, H, W, rows, d, V, partial, s); break;
  }
}

template <int KP>
void launch_kp_merge(const Plan& p, int rows, int K, int rows_prop, const uint64_t* partial,
                     float* cand_logit, int32_t* cand_id, int32_t* ver_token, hipStream_t s) {
  if (p.n_parts <= 4 * kWave)
    hipLaunchKernelGGL((topk_merge_kernel<KP, 1>), dim3(rows), dim3(kWave), 0, s, partial, rows,
                       p.n_parts * KP, K, rows_prop, cand_logit, cand_id, ver_token);
  else
    hipLaunchKernelGGL((topk_merge_kernel<KP, 4>), dim3(rows), dim3(4 * kWave), 0, s, partial, rows,
                       p.n_parts * KP, K, rows_prop, cand_logit, cand_id, ver_token);
}

template <int KP>
void launch_spec_kp(const Plan& p, const uint16_t* Hv, const uint16_t* W, int B, int L, int d, int V, int K,
                    const int32_t* proposal, const int32_t* cand_id, const float* cand_prob,
                    const float* u_accept, SampleArgs sa, uint64_t* partial, int32_t* row_accept,
                    int32_t* row_resample, int32_t* accept_len, int32_t* correction, hipStream_t s) {
  const int rows = B * L;
  switch (p.cfg) {
    case 0: launch_tile<SmallRows, KP, true>(p, Hv, W, rows, d, V, partial, s, sa); break;
    case 1: launch_tile<MidRows, KP, true>(p, Hv, W, rows, d, V, partial, s, sa); break;
    default: launch_tile<LargeRows, KP, true>(p, Hv, W, rows, d, V, partial, s, sa); break;
  }
  hipLaunchKernelGGL((spec_row_kernel<KP>), dim3(rows), dim3(256), 0, s, partial, sa.lse_part, p.n_parts,
                     Hv, W, d, V, K, proposal, cand_id, cand_prob, u_accept, sa.inv_T, sa.key0, sa.key1,
                     row_accept, row_resample);
  hipLaunchKernelGGL(spec_commit_kernel, dim3((B + 3) / 4), dim3(256), 0, s, row_accept, row_resample, B,
                     L, accept_len, correction);
}

struct SpecLayout {
  Plan plan;
  size_t keys, lse, rows_acc, rows_res, total;
};

SpecLayout spec_layout(int B, int L, int V, int K) {
  SpecLayout l{};
  const int rows = B * L;
  l.plan = make_plan(rows, V, 1, true);  // the best non-candidate key per row
  auto up = [](size_t n) { return (n + 255) / 256 * 256; };
  l.keys = 0;
  l.lse = up(static_cast<size_t>(rows) * l.plan.n_parts * l.plan.KP * sizeof(uint64_t));
  l.rows_acc = l.lse + up(static_cast<size_t>(rows) * l.plan.n_parts * sizeof(float2));
  l.rows_res = l.rows_acc + up(static_cast<size_t>(rows) * sizeof(int32_t));
  l.total = l.rows_res + up(static_cast<size_t>(rows) * sizeof(int32_t));
  return l;
}

}  // namespace

size_t spec_verify_workspace_bytes(int B, int L, int V, int K) { return spec_layout(B, L, V, K).total; }

void launch_spec_verify(const uint16_t* Hv, const uint16_t* W, int B, int L, int d, int V, int K,
                        const int32_t* proposal, const int32_t* cand_id, const float* cand_prob,
                        const float* u_accept, uint64_t seed, float temperature, int32_t* accept_len,
                        int32_t* correction, int32_t* row_accept, int32_t* row_resample, void* ws,
                        hipStream_t s) {
  const SpecLayout l = spec_layout(B, L, V, K);
  char* base = static_cast<char*>(ws);
  SampleArgs sa{1.0f / temperature, static_cast<uint32_t>(seed), static_cast<uint32_t>(seed >> 32),
                reinterpret_cast<float2*>(base + l.lse), cand_id, K};
  uint64_t* partial = reinterpret_cast<uint64_t*>(base + l.keys);
  int32_t* ra = row_accept ? row_accept : reinterpret_cast<int32_t*>(base + l.rows_acc);
  int32_t* rr = row_resample ? row_resample : reinterpret_cast<int32_t*>(base + l.rows_res);
  launch_spec_kp<4>(l.plan, Hv, W, B, L, d, V, K, proposal, cand_id, cand_prob, u_accept, sa, partial, ra, rr,
                    accept_len, correction, s);
}

size_t propose_workspace_bytes(int rows, int V, int K) {
  const Plan p = make_plan(rows, V, K);
  return static_cast<size_t>(rows) * p.n_parts * p.KP * sizeof(uint64_t);
}

void launch_propose_pass(const uint16_t* H, const uint16_t* W, int rows, int d, int V, int K, void* ws,
                         hipStream_t s) {
  const Plan p = make_plan(rows, V, K);
  uint64_t* partial = static_cast<uint64_t*>(ws);
  switch (p.KP) {
    case 4: launch_kp_pass<4>(p, H, W, rows, d, V, partial, s); break;
    case 8: launch_kp_pass<8>(p, H, W, rows, d, V, partial, s); break;
    case 16: launch_kp_pass<16>(p, H, W, rows, d, V, partial, s); break;
    case 32: launch_kp_pass<32>(p, H, W, rows, d, V, partial, s); break;
    default: launch_kp_pass<64>(p, H, W, rows, d, V, partial, s); break;
  }
}

void launch_propose_merge(int rows, int V, int K, int rows_prop, float* cand_logit, int32_t* cand_id,
                          int32_t* ver_token, const void* ws, hipStream_t s) {
  const Plan p = make_plan(rows, V, K);
  const uint64_t* partial = static_cast<const uint64_t*>(ws);
  switch (p.KP) {
    case 4: launch_kp_merge<4>(p, rows, K, rows_prop, partial, cand_logit, cand_id, ver_token, s); break;
    case 8: launch_kp_merge<8>(p, rows, K, rows_prop, partial, cand_logit, cand_id, ver_token, s); break;
    case 16: launch_kp_merge<16>(p, rows, K, rows_prop, partial, cand_logit, cand_id, ver_token, s); break;
    case 32: launch_kp_merge<32>(p, rows, K, rows_prop, partial, cand_logit, cand_id, ver_token, s); break;
    default: launch_kp_merge<64>(p, rows, K, rows_prop, partial, cand_logit, cand_id, ver_token, s); break;
  }
}

void launch_propose(const uint16_t* H, const uint16_t* W, int rows, int d, int V, int K,
                    int rows_prop, float* cand_logit, int32_t* cand_id, int32_t* ver_token,
                    void* ws, hipStream_t s) {
  launch_propose_pass(H, W, rows, d, V, K, ws, s);
  launch_propose_merge(rows, V, K, rows_prop, cand_logit, cand_id, ver_token, ws, s);
}

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch[kMaxDevices];  // device address of `scratch` on each device, once looked up

// Device address of `scratch` on device `dev`, looked up on the first call
// for that device with the device current (restored afterwards).
void* scratch_on(int dev) {
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch[dev]) return g_scratch[dev];
  int cur = -1;
  if (hipGetDevice(&cur) != hipSuccess) return nullptr;
  if (cur != dev && hipSetDevice(dev) != hipSuccess) return nullptr;
  void* p = nullptr;
  const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
  if (cur != dev) (void)hipSetDevice(cur);
  if (e != hipSuccess || !p) return nullptr;
  g_scratch[dev] = p;
  return p;
}

}  // namespace

size_t noalloc_scratch_bytes() { return BRISK_NOALLOC_SCRATCH_BYTES; }

int launch_propose_noalloc(const uint16_t* H, const uint16_t* W, int rows, int d, int V, int K,
                           float* cand_logit, int32_t* cand_id, hipStream_t s) {
  int dev = -1;
  if (s) {
    hipDevice_t sd;
    if (hipStreamGetDevice(s, &sd) != hipSuccess) return -1;
    dev = static_cast<int>(sd);
  } else if (hipGetDevice(&dev) != hipSuccess) {
    return -1;
  }
  if (dev < 0 || dev >= kMaxDevices) return -1;
  void* ws = scratch_on(dev);
  if (!ws) return -1;
  // every (row, group) list is written by the pass before the merge reads
  // it, so nothing left by an earlier call needs clearing
  launch_propose(H, W, rows, d, V, K, rows, cand_logit, cand_id, nullptr, ws, s);
  return 0;
}

}  // namespace brisk
