// Prefix-conditioned corrector (Section 3.3 Eq. inference_head_state and
// Eq. candidate_residual; Appendix head details, Eq. head_residual_logits;
// Algorithm 1(b) loop).
//
// The recurrence is sequential over the L block positions, but almost all of
// its arithmetic does not depend on which candidate gets selected.  Because
// the step input x_hat_i is a concatenation and every map applied to it is
// linear, W_z x_hat_i splits into a per-row part (hidden state and position),
// a per-previous-token part and a 5-wide feature part; the residual
// <W_s u_i, W_c E_out(v)> re-associates to <u_i, W_s^T W_c E_out(v)>.  All of
// those pieces are computed up front for every row and every candidate
// (kernels gather_proj, which also forms the cross logits, and lift); the
// scan then carries only
// the selection-dependent chain: features, gate, state update, K dot products
// and an argmax per step, one wavefront per sequence.
#include <algorithm>

#include "device_common.h"
#include "kernels.h"

namespace brisk {

namespace {

// ---------------------------------------------------------------------------
// gather_proj: out[n, j] = sum_k table[row(n), k] * wt[j, k]   (bf16 in, fp32 out)
// row(n) = idx[n] (clamped into [0, n_table)) or n when idx is null.
// MFMA: A = wt rows (M = j), B = gathered rows (N = n).  The reduction over
// d is split into `splits` slices (grid z) so that small batches still fill
// the GPU; slice s writes its partial sums to out + s * n * J and the
// consumers add the slices in order, which keeps the result deterministic.
// ---------------------------------------------------------------------------
struct ProjJob {
  const uint16_t* table;
  const int32_t* idx;
  int n, J, n_table;
  const uint16_t* wt;
  float* out;           // slice s, row n, column j at out[s * slice_stride + n * J + j]
  size_t slice_stride;  // floats between consecutive slices
};
constexpr int kMaxProjJobs = 6;
// The cross logits ride in the same launch as one more job row: dot product n
// < NC is candidate k of row r against hidden row r+1 (0 on the last row of a
// block); n >= NC is the anchor token x_0 against the block's first row.
struct CrossJob {
  const uint16_t* W;
  const uint16_t* H;
  const int32_t* cand_id;
  const int32_t* anchor;
  int B, L, K, V;
  float* X;
  int group;  // candidates per wavefront, 1..8
};
// Table rows into the step blocks (with the per-token tables): for every
// candidate its EH, TZ and TH rows, for every anchor its TZ and TH rows; one
// wavefront per row, rows first..n_vec-1 in steps of `step`.
struct FillArgs {
  const float* tables;   // [3][V][vs]: EH, TZ, TH
  const int32_t* cand_id;
  const int32_t* anchor;
  float* SB;             // [rows][2 + 3K][vs]
  float* TZA;            // [B][ds]
  float* THA;
  int rows, K, B, V, ds, vs;  // rows = B = 0: nothing to copy
};

// Vector n: the candidates' EH, TZ and TH rows first, then the anchors' TZ
// and TH rows.  fill_id gives its token id; fill_vec its source, destination
// and length for that id.
struct FillVec {
  const float* src;
  float* dst;
  int len;
};
__device__ __forceinline__ int fill_id(const FillArgs& a, int n) {
  const int n_cand = a.rows * 3 * a.K;
  if (n < n_cand) {
    const int r = n / (3 * a.K), k = n % (3 * a.K) % a.K;
    return clamp_id(a.cand_id[static_cast<size_t>(r) * a.K + k], a.V);
  }
  return clamp_id(a.anchor[(n - n_cand) % a.B], a.V);
}
__device__ __forceinline__ FillVec fill_vec(const FillArgs& a, int n, int v) {
  const int n_cand = a.rows * 3 * a.K;
  if (n < n_cand) {
    const int r = n / (3 * a.K), f = n % (3 * a.K), kind = f / a.K;
    return {a.tables + (static_cast<size_t>(kind) * a.V + v) * a.vs,
            a.SB + (static_cast<size_t>(r) * (2 + 3 * a.K) + 2 + f) * a.vs, a.vs};
  }
  const int m = n - n_cand, b = m % a.B, kind = 1 + m / a.B;  // TZ, then TH
  return {a.tables + (static_cast<size_t>(kind) * a.V + v) * a.vs,
          (kind == 1 ? a.TZA : a.THA) + static_cast<size_t>(b) * a.ds, a.ds};
}

// A wavefront copies kFillBatch consecutive vectors at a time: lane g loads
// vector g's token id (one load for the batch), then every lane loads its 16
// bytes of each source row before the first store, so the batch waits for
// two memory latencies instead of two per vector.  With 256-float table rows
// (d_state <= 256) the row loads are unconditional (a table row is never
// shorter) and only the stores into rows of d_state floats are masked; other
// strides copy vector by vector.
constexpr int kFillBatch = 4;
__device__ void fill_rows(const FillArgs& a, int first, int step) {
  const int lane = threadIdx.x & 63;
  const int n_all = a.rows * 3 * a.K + 2 * a.B;
  // the batch index is wave-uniform
  for (int n0 = __builtin_amdgcn_readfirstlane(first * kFillBatch); n0 < n_all; n0 += step * kFillBatch) {
    const int my_id = fill_id(a, min(n0 + min(lane, kFillBatch - 1), n_all - 1));
    if (a.vs == 256 && (a.ds & 3) == 0) {
      // named, not arrays, so that nothing is staged through memory; a batch
      // past the last vector repeats it (the same bytes to the same place)
      static_assert(kFillBatch == 4, "the batch below is written out for four vectors");
      const FillVec f0 = fill_vec(a, min(n0 + 0, n_all - 1), __builtin_amdgcn_readlane(my_id, 0));
      const FillVec f1 = fill_vec(a, min(n0 + 1, n_all - 1), __builtin_amdgcn_readlane(my_id, 1));
      const FillVec f2 = fill_vec(a, min(n0 + 2, n_all - 1), __builtin_amdgcn_readlane(my_id, 2));
      const FillVec f3 = fill_vec(a, min(n0 + 3, n_all - 1), __builtin_amdgcn_readlane(my_id, 3));
      const float4 v0 = *reinterpret_cast<const float4*>(f0.src + lane * 4);
      const float4 v1 = *reinterpret_cast<const float4*>(f1.src + lane * 4);
      const float4 v2 = *reinterpret_cast<const float4*>(f2.src + lane * 4);
      const float4 v3 = *reinterpret_cast<const float4*>(f3.src + lane * 4);
      if (lane * 4 < f0.len) *reinterpret_cast<float4*>(f0.dst + lane * 4) = v0;
      if (lane * 4 < f1.len) *reinterpret_cast<float4*>(f1.dst + lane * 4) = v1;
      if (lane * 4 < f2.len) *reinterpret_cast<float4*>(f2.dst + lane * 4) = v2;
      if (lane * 4 < f3.len) *reinterpret_cast<float4*>(f3.dst + lane * 4) = v3;
      continue;
    }
    for (int g = 0; g < kFillBatch && n0 + g < n_all; ++g) {
      const FillVec f = fill_vec(a, n0 + g, __builtin_amdgcn_readlane(my_id, g));
      if ((f.len & 3) == 0) {
        for (int e = lane * 4; e < f.len; e += 256)
          *reinterpret_cast<float4*>(f.dst + e) = *reinterpret_cast<const float4*>(f.src + e);
      } else {
        for (int e = lane; e < f.len; e += 64) f.dst[e] = f.src[e];
      }
    }
  }
}

__global__ __launch_bounds__(256) void fill_kernel(FillArgs a) {
  fill_rows(a, blockIdx.x * 4 + (threadIdx.x >> 6), gridDim.x * 4);
}

// One launch: the projection jobs (grid rows 0..kMaxProjJobs-1), the cross
// logits (row kMaxProjJobs) and the table rows (row kMaxProjJobs + 1), which
// all read nothing the others write.
struct ProjJobs {
  ProjJob job[kMaxProjJobs];
  CrossJob cross;
  FillArgs fill;
  int d, splits;
};

// Tiles are PJ_BN gathered rows x BJ outputs (BJ = 64 or 128, a template
// argument).  A job with J outputs gathers each of its rows once per output
// tile, and neighbouring workgroups run on different XCDs, so those re-reads
// miss in L2: with J = 128, 128-wide tiles halve the gathered traffic, which
// decides the batched shapes.  Small batches split d instead and keep 64-wide
// tiles, which give twice as many workgroups.
constexpr int PJ_BN = 64, PJ_BK = 64, PJ_STRIDE = PJ_BK + 8;
constexpr int PJ_CPR = PJ_BK / 8;        // 16-byte pieces per staged row
constexpr int PJ_NPB = PJ_BN * PJ_CPR / 256;  // gathered-row pieces per thread
static_assert(PJ_NPB >= 1 && PJ_BN * PJ_CPR % 256 == 0, "staging map");
constexpr int PJ_PF = 2;  // reduction chunks in flight per thread

// One wavefront per row and group of up to `group` of its candidates: the
// hidden row m_{r+1} is read once for all of them, two 512-element chunks of
// every operand in flight per lane.  Anchors take one wavefront each.  Groups
// of eight when there are many dots (the hidden row is re-read less); one
// candidate per wavefront when there are few, which keeps more wavefronts
// in flight (32 rows: 257 wavefronts instead of 33).
__device__ __forceinline__ float dot8_bf16(uint4 a, uint4 c, float s) {
  s += bf16_lo(a.x) * bf16_lo(c.x) + bf16_hi(a.x) * bf16_hi(c.x);
  s += bf16_lo(a.y) * bf16_lo(c.y) + bf16_hi(a.y) * bf16_hi(c.y);
  s += bf16_lo(a.z) * bf16_lo(c.z) + bf16_hi(a.z) * bf16_hi(c.z);
  s += bf16_lo(a.w) * bf16_lo(c.w) + bf16_hi(a.w) * bf16_hi(c.w);
  return s;
}

// G candidates a wavefront at most, U 512-element chunks of each operand in
// flight per lane.  One candidate a wavefront takes eight chunks, so a 4096-
// long dot is one round of loads instead of four, and groups of four take
// four chunks, two rounds (the accumulation order over k is the same).
template <int G, int U>
__device__ void cross_dots(const CrossJob& cj, int d) {
  const int lane = threadIdx.x & 63;
  const int rows = cj.B * cj.L, NC = rows * cj.K;
  const int g = cj.group;
  const int nkb = (cj.K + g - 1) / g;
  const int items = rows * nkb + cj.B;
  const int waves = gridDim.x * gridDim.z * 4;
  for (int it = (blockIdx.z * gridDim.x + blockIdx.x) * 4 + (threadIdx.x >> 6); it < items; it += waves) {
    int hrow, nk;
    float* xo;
    const uint16_t* w[G];
    if (it < rows * nkb) {
      const int r = it / nkb, k0 = (it % nkb) * g;
      nk = min(g, cj.K - k0);
      xo = cj.X + static_cast<size_t>(r) * cj.K + k0;
      if (r % cj.L == cj.L - 1) {  // the last row of a block has no next row
        if (lane < nk) xo[lane] = 0.f;
        continue;
      }
      hrow = r + 1;
#pragma unroll
      for (int q = 0; q < G; ++q) {
        const int v = clamp_id(cj.cand_id[static_cast<size_t>(r) * cj.K + k0 + min(q, nk - 1)], cj.V);
        w[q] = cj.W + static_cast<size_t>(v) * d;
      }
    } else {
      const int b = it - rows * nkb;
      nk = 1;
      xo = cj.X + NC + b;
      hrow = b * cj.L;
      const int v = clamp_id(cj.anchor[b], cj.V);
#pragma unroll
      for (int q = 0; q < G; ++q) w[q] = cj.W + static_cast<size_t>(v) * d;
    }
    const uint16_t* h = cj.H + static_cast<size_t>(hrow) * d;
    float acc[G];
#pragma unroll
    for (int q = 0; q < G; ++q) acc[q] = 0.f;
    for (int k0 = lane * 8; k0 < d; k0 += 512 * U) {
      uint4 hv[U], wv[G][U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int k = k0 + u * 512;
        hv[u] = k < d ? *reinterpret_cast<const uint4*>(h + k) : make_uint4(0, 0, 0, 0);
#pragma unroll
        for (int q = 0; q < G; ++q)
          wv[q][u] = k < d && q < nk ? *reinterpret_cast<const uint4*>(w[q] + k) : make_uint4(0, 0, 0, 0);
      }
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int q = 0; q < G; ++q) acc[q] = dot8_bf16(wv[q][u], hv[u], acc[q]);
    }
#pragma unroll
    for (int q = 0; q < G; ++q) {
      const float sq = wave_sum(acc[q]);
      if (lane == 0 && q < nk) xo[q] = sq;
    }
  }
}

template <int BJ>
__global__ __launch_bounds__(256) void gather_proj_kernel(ProjJobs jobs) {
  static_assert(BJ == 64 || BJ == 128, "output tile");
  constexpr int NPA = BJ * PJ_CPR / 256;  // weight-row pieces per thread
  constexpr int WJ = BJ / 2, TJ = WJ / 16;  // a wave's outputs and 16-wide fragments
  const int d = jobs.d;
  if (blockIdx.y == kMaxProjJobs) {
    if (jobs.cross.group == 1) cross_dots<1, 8>(jobs.cross, d);
    else if (jobs.cross.group == 4) cross_dots<4, 4>(jobs.cross, d);
    else cross_dots<8, 2>(jobs.cross, d);
    return;
  }
  if (blockIdx.y == kMaxProjJobs + 1) {
    fill_rows(jobs.fill, (blockIdx.z * gridDim.x + blockIdx.x) * 4 + (threadIdx.x >> 6), gridDim.x * gridDim.z * 4);
    return;
  }
  const ProjJob& jb = jobs.job[blockIdx.y];
  const int n_jt = (jb.J + BJ - 1) / BJ;
  const int n_nt = (jb.n + PJ_BN - 1) / PJ_BN;
  if (static_cast<int>(blockIdx.x) >= n_jt * n_nt) return;
  const int jt = blockIdx.x % n_jt, nt = blockIdx.x / n_jt;
  const int j0 = jt * BJ, n0 = nt * PJ_BN;
  const int chunks = (d + PJ_BK - 1) / PJ_BK;
  const int per = (chunks + jobs.splits - 1) / jobs.splits;
  const int c_begin = min(static_cast<int>(blockIdx.z) * per, chunks);
  const int n_ch = min(c_begin + per, chunks) - c_begin;

  __shared__ __align__(16) uint16_t sA[BJ * PJ_STRIDE];
  __shared__ __align__(16) uint16_t sB[PJ_BN * PJ_STRIDE];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wj = wave & 1, wn = wave >> 1;  // 2 x 2 waves, WJ x 32 each

  // Each thread stages NPA + PJ_NPB 16-byte pieces per chunk; its
  // rows are fixed, so the gathered table rows are resolved once.  PJ_PF
  // chunks are in flight in registers, so a workgroup with a short slice of
  // the reduction waits about one memory latency, not one per chunk.  Every
  // load is unconditional and reads valid memory, so the compiler counts the
  // loads in flight exactly and waits only for the chunk being staged: rows
  // past J or n read a valid row whose outputs are never stored, and pieces
  // past d or past the slice (the tail of the last group re-reads the slice's
  // last chunk) are staged as zeros.
  // every piece of a thread has the same column, since 256 is a multiple of
  // the pieces per row
  const int col = (tid % PJ_CPR) * 8;
  int arow[NPA], brow[PJ_NPB];
#pragma unroll
  for (int i = 0; i < NPA; ++i) {
    const int row = (tid + i * 256) / PJ_CPR;
    arow[i] = j0 + row < jb.J ? j0 + row : 0;
  }
#pragma unroll
  for (int i = 0; i < PJ_NPB; ++i) {
    const int n = n0 + (tid + i * 256) / PJ_CPR;
    brow[i] = n < jb.n ? (jb.idx ? clamp_id(jb.idx[n], jb.n_table) : n) : 0;
  }
  uint4 ra[PJ_PF][NPA], rb[PJ_PF][PJ_NPB];
  auto load = [&](uint4 (&A)[NPA], uint4 (&Bv)[PJ_NPB], int ch) {
    const int cc = c_begin + max(min(ch, n_ch - 1), 0);
    const int k = cc * PJ_BK + col;
    const int kc = k < d ? k : 0;
#pragma unroll
    for (int i = 0; i < NPA; ++i)
      A[i] = *reinterpret_cast<const uint4*>(jb.wt + static_cast<size_t>(arow[i]) * d + kc);
#pragma unroll
    for (int i = 0; i < PJ_NPB; ++i)
      Bv[i] = *reinterpret_cast<const uint4*>(jb.table + static_cast<size_t>(brow[i]) * d + kc);
  };
  auto store = [&](const uint4 (&A)[NPA], const uint4 (&Bv)[PJ_NPB], int ch) {
    const uint32_t m = ch < n_ch && (c_begin + ch) * PJ_BK + col < d ? ~0u : 0u;
#pragma unroll
    for (int i = 0; i < NPA; ++i) {
      const int row = (tid + i * 256) / PJ_CPR;
      *reinterpret_cast<uint4*>(sA + row * PJ_STRIDE + col) =
          make_uint4(A[i].x & m, A[i].y & m, A[i].z & m, A[i].w & m);
    }
#pragma unroll
    for (int i = 0; i < PJ_NPB; ++i) {
      const int row = (tid + i * 256) / PJ_CPR;
      *reinterpret_cast<uint4*>(sB + row * PJ_STRIDE + col) =
          make_uint4(Bv[i].x & m, Bv[i].y & m, Bv[i].z & m, Bv[i].w & m);
    }
  };

  floatx4 acc[TJ][2];
#pragma unroll
  for (int a = 0; a < TJ; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b) acc[a][b] = floatx4{0.f, 0.f, 0.f, 0.f};

  // the scheduling barriers keep the loads in chunk order, which is what
  // lets each staging step wait for its own chunk only
#pragma unroll
  for (int p = 0; p < PJ_PF; ++p) {
    load(ra[p], rb[p], p);
    __builtin_amdgcn_sched_barrier(0);
  }
  for (int g = 0; g < n_ch; g += PJ_PF) {
#pragma unroll
    for (int p = 0; p < PJ_PF; ++p) {
      const int ch = g + p;
      store(ra[p], rb[p], ch);
      __syncthreads();
      __builtin_amdgcn_sched_barrier(0);
      load(ra[p], rb[p], ch + PJ_PF);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int kk = 0; kk < PJ_BK; kk += 32) {
        const int koff = kk + (lane >> 4) * 8;
        bf16x8 a[TJ], b[2];
#pragma unroll
        for (int t = 0; t < TJ; ++t)
          a[t] = *reinterpret_cast<const bf16x8*>(sA + (wj * WJ + t * 16 + (lane & 15)) * PJ_STRIDE + koff);
#pragma unroll
        for (int t = 0; t < 2; ++t)
          b[t] = *reinterpret_cast<const bf16x8*>(sB + (wn * 32 + t * 16 + (lane & 15)) * PJ_STRIDE + koff);
#pragma unroll
        for (int x = 0; x < TJ; ++x)
#pragma unroll
          for (int y = 0; y < 2; ++y)
            acc[x][y] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[x], b[y], acc[x][y], 0, 0, 0);
      }
      __syncthreads();
    }
  }
  float* out = jb.out + static_cast<size_t>(blockIdx.z) * jb.slice_stride;
#pragma unroll
  for (int x = 0; x < TJ; ++x)
#pragma unroll
    for (int y = 0; y < 2; ++y) {
      const int n = n0 + wn * 32 + y * 16 + (lane & 15);
      const int jb0 = j0 + wj * WJ + x * 16 + (lane >> 4) * 4;
      if (n < jb.n) {
        float* o = out + static_cast<size_t>(n) * jb.J + jb0;
        if (jb0 + 4 <= jb.J && (reinterpret_cast<uintptr_t>(o) & 15u) == 0) {
          *reinterpret_cast<float4*>(o) = make_float4(acc[x][y][0], acc[x][y][1], acc[x][y][2], acc[x][y][3]);
        } else {
#pragma unroll
          for (int q = 0; q < 4; ++q)
            if (jb0 + q < jb.J) o[q] = acc[x][y][q];
        }
      }
    }
}

// ---------------------------------------------------------------------------
// lift: out[n, j] = sum over terms T of sum_c M_T(j, c) in_T(n, c), j < ds.
// A term reads its input either as fp32 (the projections above, split-K
// slices already summed) or as bf16 (the position table, the feature map
// P_phi), with arbitrary strides and an optional row period (position index
// = row mod L); M_T(j, c) = m[j * m_rs + c * m_cs] is a bf16 slice of a
// corrector matrix.
//
// MFMA with a three-term split of the fp32 input: x = x0 + x1 + x2 + e with
// x0 = bf16(x), x1 = bf16(x - x0), x2 = bf16(x - x0 - x1) and |e| <= 2^-27
// |x|, so M x = M x0 + M x1 + M x2 goes through bf16 products with fp32
// accumulation at full fp32 input precision (the matrices are bf16
// already).  Tiles of 64 rows x 64 outputs (wave w owns outputs
// 16w..16w+15 of the tile); the reduction is staged in LDS 64 columns at a
// time with the next columns already loading.  Vectors stored with a stride
// beyond d_state are zero-filled up to the stride.
// ---------------------------------------------------------------------------
struct LiftTerm {
  const void* in;      // fp32 or bf16
  int in_bf16;
  int rs, cs, period;  // in(n, c) = in[(period ? n % period : n) * rs + c * cs]
  int C;
  const uint16_t* m;
  int m_rs, m_cs;
  int vec;    // fp32 input rows may be read as 16-byte vectors along c
  int mvec;   // the matrix may be read as 16-byte vectors along its contiguous index
};
struct LiftJob {
  LiftTerm t[2];       // second term optional (C = 0)
  int n;
  float* out;          // row n -> out + (n / grp) * blk + (n % grp) * vs
  int grp;
  size_t blk, vs;
};
constexpr int kMaxLiftJobs = 9;
struct LiftJobs {
  LiftJob job[kMaxLiftJobs];
  int ds;
};
constexpr int LT_BN = 64, LT_BJ = 64, LT_BC = 64, LT_ROW = LT_BC + 8;  // LDS row: 144 bytes

__device__ __forceinline__ uint16_t bf16_rne(float x) {
  uint32_t u = __float_as_uint(x);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return static_cast<uint16_t>(u >> 16);
}

__device__ __forceinline__ float lift_in(const LiftTerm& t, int n, int c) {
  const size_t idx = static_cast<size_t>(t.period ? n % t.period : n) * t.rs + static_cast<size_t>(c) * t.cs;
  return t.in_bf16 ? bf16_to_f32(static_cast<const uint16_t*>(t.in)[idx]) : static_cast<const float*>(t.in)[idx];
}

// LT_BUFS staging buffers.  With two, the next chunk is staged while the
// current one's products run; with one, a barrier separates them, but twice
// as many workgroups fit in a compute unit's LDS, which pays off when there
// are many of them (37 KB against 74 KB: 39 against 50 us at 2048 rows; at
// 32 rows two buffers are 0.7 us faster).
template <int LT_BUFS>
__global__ __launch_bounds__(256) void lift_kernel(LiftJobs jobs) {
  const LiftJob& jb = jobs.job[blockIdx.z];
  const int n0 = blockIdx.x * LT_BN, j0 = blockIdx.y * LT_BJ;
  const int ds = jobs.ds;
  const int jend = static_cast<int>(jb.vs) > ds ? static_cast<int>(jb.vs) : ds;
  if (n0 >= jb.n || j0 >= jend) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  auto out_row = [&](int n) {
    return jb.out + static_cast<size_t>(n / jb.grp) * jb.blk + static_cast<size_t>(n % jb.grp) * jb.vs;
  };
  if (j0 >= ds) {  // zero padding only
    for (int e = tid; e < LT_BN * LT_BJ; e += 256) {
      const int n = n0 + e / LT_BJ, j = j0 + e % LT_BJ;
      if (n < jb.n && j < jend) out_row(n)[j] = 0.f;
    }
    return;
  }

  __shared__ __align__(16) uint16_t s_x[3][LT_BUFS][LT_BN * LT_ROW];
  __shared__ __align__(16) uint16_t s_m[LT_BUFS][LT_BJ * LT_ROW];

  // Term 0 fills chunks [0, nc0) and term 1 the rest, so the term of a chunk
  // is uniform across the workgroup.
  const int nc0 = (jb.t[0].C + LT_BC - 1) / LT_BC;
  const int nch = nc0 + (jb.t[1].C + LT_BC - 1) / LT_BC;
  // staging map: 16 consecutive columns of one row per thread
  const int sr = tid >> 2, sc = (tid & 3) * 16;
  // Raw words of the thread's input and matrix runs, as loaded.  Every load
  // is unconditional and reads valid memory (an element outside the term or
  // the tile reads index 0); masking and unpacking wait until the run is
  // staged, so a chunk's loads stay in flight across the previous chunk's
  // products.  Runs that are contiguous and 16-byte aligned (the host sets
  // vec / mvec) load as vectors.
  enum { kF32 = 0, kBf16Pairs = 1, kBf16 = 2 };
  uint32_t rw[16], mw[16];
  uint32_t in_ok = 0, m_ok = 0;  // bit q: element q of the run is inside its term and tile
  int in_mode = kF32;
  bool m_pairs = false, mt = false;
  auto load = [&](int ch) {
    const bool second = ch >= nc0;
    const LiftTerm t = second ? jb.t[1] : jb.t[0];
    const int cbase = (second ? ch - nc0 : ch) * LT_BC;  // first column of the chunk in the term
    const int n = n0 + sr;
    const int nv = n < jb.n ? n : 0;
    const size_t rbase = static_cast<size_t>(t.period ? nv % t.period : nv) * t.rs;
    const int c = cbase + sc;
    if (t.vec) {  // cs == 1 and C % 16 == 0: the run is wholly inside the term or wholly outside
      const bool ok = n < jb.n && c + 16 <= t.C;
      in_ok = ok ? 0xFFFFu : 0u;
      const size_t off = rbase + (ok ? c : 0);
      if (t.in_bf16) {
        in_mode = kBf16Pairs;
        const uint4* p = reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(t.in) + off);
        const uint4 u0 = p[0], u1 = p[1];
        rw[0] = u0.x; rw[1] = u0.y; rw[2] = u0.z; rw[3] = u0.w;
        rw[4] = u1.x; rw[5] = u1.y; rw[6] = u1.z; rw[7] = u1.w;
      } else {
        in_mode = kF32;
        const uint4* p = reinterpret_cast<const uint4*>(static_cast<const float*>(t.in) + off);
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const uint4 x = p[v];
          rw[4 * v] = x.x; rw[4 * v + 1] = x.y; rw[4 * v + 2] = x.z; rw[4 * v + 3] = x.w;
        }
      }
    } else {
      in_mode = t.in_bf16 ? kBf16 : kF32;
      in_ok = 0;
      size_t idx[16];
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        const bool ok = n < jb.n && c + q < t.C;
        in_ok |= ok ? 1u << q : 0u;
        idx[q] = ok ? rbase + static_cast<size_t>(c + q) * t.cs : 0;
      }
      if (t.in_bf16) {
#pragma unroll
        for (int q = 0; q < 16; ++q) rw[q] = static_cast<const uint16_t*>(t.in)[idx[q]];
      } else {
#pragma unroll
        for (int q = 0; q < 16; ++q) rw[q] = static_cast<const uint32_t*>(t.in)[idx[q]];
      }
    }
    // matrix run: along c when m_cs == 1, along j when m_rs == 1 (mt)
    mt = t.m_rs == 1;
    const int j = j0 + (mt ? sc : sr), cm = cbase + (mt ? sr : sc);
    m_pairs = t.mvec != 0;
    if (t.mvec) {
      const bool ok = mt ? (j + 16 <= ds && cm < t.C) : (j < ds && cm + 16 <= t.C);
      m_ok = ok ? 0xFFFFu : 0u;
      const uint4* p = reinterpret_cast<const uint4*>(
          t.m + (ok ? static_cast<size_t>(j) * t.m_rs + static_cast<size_t>(cm) * t.m_cs : 0));
      const uint4 u0 = p[0], u1 = p[1];
      mw[0] = u0.x; mw[1] = u0.y; mw[2] = u0.z; mw[3] = u0.w;
      mw[4] = u1.x; mw[5] = u1.y; mw[6] = u1.z; mw[7] = u1.w;
    } else {
      m_ok = 0;
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        const int jq = mt ? j + q : j, cq = mt ? cm : cm + q;
        const bool ok = jq < ds && cq < t.C;
        m_ok |= ok ? 1u << q : 0u;
        mw[q] = t.m[ok ? static_cast<size_t>(jq) * t.m_rs + static_cast<size_t>(cq) * t.m_cs : 0];
      }
    }
  };
  auto pack = [](const uint16_t* h) {
    return make_uint4(h[0] | (static_cast<uint32_t>(h[1]) << 16), h[2] | (static_cast<uint32_t>(h[3]) << 16),
                      h[4] | (static_cast<uint32_t>(h[5]) << 16), h[6] | (static_cast<uint32_t>(h[7]) << 16));
  };
  auto store = [&](int buf) {
    // decode (uniform branches), then mask with the per-element bits
    uint32_t bits[16], h[16];
    if (in_mode == kBf16Pairs) {
#pragma unroll
      for (int q = 0; q < 16; ++q) bits[q] = q & 1 ? rw[q >> 1] & 0xFFFF0000u : rw[q >> 1] << 16;
    } else if (in_mode == kBf16) {
#pragma unroll
      for (int q = 0; q < 16; ++q) bits[q] = rw[q] << 16;
    } else {
#pragma unroll
      for (int q = 0; q < 16; ++q) bits[q] = rw[q];
    }
    if (m_pairs) {
#pragma unroll
      for (int q = 0; q < 16; ++q) h[q] = q & 1 ? mw[q >> 1] >> 16 : mw[q >> 1] & 0xFFFFu;
    } else {
#pragma unroll
      for (int q = 0; q < 16; ++q) h[q] = mw[q] & 0xFFFFu;
    }
    float rin[16];
    uint16_t rm[16];
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      rin[q] = __uint_as_float(bits[q] & (0u - ((in_ok >> q) & 1u)));
      rm[q] = static_cast<uint16_t>(h[q] & (0u - ((m_ok >> q) & 1u)));
    }
    uint16_t x[3][16];
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      x[0][q] = bf16_rne(rin[q]);
      const float r1 = rin[q] - bf16_to_f32(x[0][q]);
      x[1][q] = bf16_rne(r1);
      x[2][q] = bf16_rne(r1 - bf16_to_f32(x[1][q]));
    }
#pragma unroll
    for (int t = 0; t < 3; ++t) {
      uint4* dst = reinterpret_cast<uint4*>(&s_x[t][buf][sr * LT_ROW + sc]);
      dst[0] = pack(x[t]);
      dst[1] = pack(x[t] + 8);
    }
    if (mt) {
#pragma unroll
      for (int q = 0; q < 16; ++q) s_m[buf][(sc + q) * LT_ROW + sr] = rm[q];
    } else {
      uint4* dst = reinterpret_cast<uint4*>(&s_m[buf][sr * LT_ROW + sc]);
      dst[0] = pack(rm);
      dst[1] = pack(rm + 8);
    }
  };

  floatx4 acc[4];
#pragma unroll
  for (int b = 0; b < 4; ++b) acc[b] = floatx4{0.f, 0.f, 0.f, 0.f};
  load(0);
  store(0);
  __syncthreads();
  for (int ch = 0; ch < nch; ++ch) {
    const int buf = LT_BUFS == 2 ? ch & 1 : 0;
    if (ch + 1 < nch) load(ch + 1);
#pragma unroll
    for (int kk = 0; kk < LT_BC; kk += 32) {
      const int koff = kk + (lane >> 4) * 8;
      const bf16x8 a = *reinterpret_cast<const bf16x8*>(&s_m[buf][(wave * 16 + (lane & 15)) * LT_ROW + koff]);
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        const int row = (b * 16 + (lane & 15)) * LT_ROW + koff;
#pragma unroll
        for (int t = 0; t < 3; ++t) {
          const bf16x8 x = *reinterpret_cast<const bf16x8*>(&s_x[t][buf][row]);
          acc[b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, x, acc[b], 0, 0, 0);
        }
      }
    }
    if (ch + 1 < nch) {
      if constexpr (LT_BUFS == 1) __syncthreads();  // every wave is done with the buffer
      store(LT_BUFS == 2 ? buf ^ 1 : 0);
    }
    __syncthreads();
  }
  // lane holds outputs j = 16 wave + 4 (lane / 16) + q of row 16 b + lane % 16
  const int jq = j0 + wave * 16 + (lane >> 4) * 4;
#pragma unroll
  for (int b = 0; b < 4; ++b) {
    const int n = n0 + b * 16 + (lane & 15);
    if (n >= jb.n) continue;
    float* o = out_row(n);
    if (jq + 4 <= ds && (reinterpret_cast<uintptr_t>(o + jq) & 15u) == 0) {
      // four consecutive outputs of the row in one 16-byte store
      *reinterpret_cast<float4*>(o + jq) = make_float4(acc[b][0], acc[b][1], acc[b][2], acc[b][3]);
      continue;
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int j = jq + q;
      if (j < ds) o[j] = acc[b][q];
      else if (j < jend) o[j] = 0.f;
    }
  }
}

// ---------------------------------------------------------------------------
// slice_sum: in-place, in-order sum of the split-K slices into slice 0.
// ---------------------------------------------------------------------------
struct SliceArr {
  float* p;
  size_t n;       // elements per slice (a multiple of 4)
  size_t stride;  // floats between slices
};
constexpr int kMaxSliceArrs = 4, kMaxSplits = 16;
struct SliceArrs {
  SliceArr arr[kMaxSliceArrs];
  int splits;
};

__global__ __launch_bounds__(256) void slice_sum_kernel(SliceArrs sa) {
  const SliceArr& A = sa.arr[blockIdx.y];
  const size_t i = (static_cast<size_t>(blockIdx.x) * 256 + threadIdx.x) * 4;
  if (i >= A.n) return;
  float4 v[kMaxSplits];
#pragma unroll
  for (int s = 0; s < kMaxSplits; ++s)
    if (s < sa.splits) v[s] = *reinterpret_cast<const float4*>(A.p + s * A.stride + i);
  float4 t = v[0];
#pragma unroll
  for (int s = 1; s < kMaxSplits; ++s)
    if (s < sa.splits) {
      t.x += v[s].x;
      t.y += v[s].y;
      t.z += v[s].z;
      t.w += v[s].w;
    }
  *reinterpret_cast<float4*>(A.p + i) = t;
}

// ---------------------------------------------------------------------------
// scan: one workgroup per sequence, one 64-wide slice of the state per wave.
//
// The lift kernel leaves each row's step inputs in one contiguous "step
// block" of F = 2 + 3K vectors of length ds: [AZ, AH, EH_0..EH_{K-1},
// TZ_0..TZ_{K-1}, TH_0..TH_{K-1}] (TZ_k/TH_k: what candidate k of this row
// feeds into the next step).  A step therefore loads with buffer
// instructions whose only per-field arithmetic is a scalar offset.
//
// The loads for the next D-1 rows are in flight while a step runs: D
// statically indexed buffers are rotated by unrolling the step loop D times,
// loads are unconditional (indices clamped, never masked at load time) and
// outputs are staged in LDS, so the loop holds no stores and the compiler can
// wait for exactly the buffer a step consumes.
//
// Reductions: the K residual dot products and the gate product are summed
// inside each 16-lane row with DPP (all values interleaved), the row sums of
// every wave go to LDS, and after one barrier every lane adds the 4 * waves
// row sums of its value in a fixed order, so all waves take the same decision.
// ---------------------------------------------------------------------------
struct ScanArgs {
  int B, L, K, ds, vs;  // vs: floats between the vectors of a step block (>= ds)
  const float* U0;   // [2, B, ds]  A_h h_c, A_e E(x_0)
  const float* X;    // [NC + B]
  const float* SB;   // [rows, F, ds] step blocks
  const float* TZA;  // [B, ds] anchor-token inputs of step 0
  const float* THA;
  const float* FZ;   // [5, ds] W_z[:, feat] P_phi
  const float* FH;   // [5, ds] W_h[:, feat] P_phi
  const uint16_t* w_g;
  float alpha, b_g;
  const float* cand_logit;
  const int32_t* cand_id;
  const int32_t* anchor;
  int32_t* selected;
  float* refined;
  float* gamma;
  float* resid;
  float* dump;       // [B, 64] sink for output lanes with nothing to write
  // optional verification in the same pass (single-wave scan only): the
  // verifier's tokens [B, L] and the accepted-prefix length / correction [B]
  const int32_t* verifier;
  int32_t* accept_len;
  int32_t* correction;
  // optional per-token tables [EH; TZ; TH] (single-wave scan only): the
  // candidates' and the anchor's vectors are read from them by token id,
  // and the step blocks hold only AZ and AH
  const float* tables;
  int V;
};

template <int KM>
struct StepData {
  float az, ah;
  float eh[KM];
  float tz[KM], th[KM];
  float cl, xs;
  int ci;
};

__device__ __forceinline__ float buf_ld(__amdgpu_buffer_rsrc_t r, int voff, int soff) {
  return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, voff, soff, 0));
}

// Loads of step i (row clamped into the block).  Candidates k >= K read a
// duplicate of candidate K-1 and lanes past ds read element ds-1; consumers
// ignore those values (k >= K is never selected or used, lanes past ds hold
// u = 0, lanes >= K are masked where scores are formed).
template <int KM>
__device__ __forceinline__ void load_step(StepData<KM>& s, const ScanArgs& a,
                                          __amdgpu_buffer_rsrc_t rsb, int voff, int b, int i,
                                          int lane) {
  const int ii = i < a.L ? i : a.L - 1;
  const int F = 2 + 3 * a.K;
  const int vb = a.vs * 4;                // bytes per vector
  const int base = ii * F * vb;           // this row's step block inside the sequence
  s.az = buf_ld(rsb, voff, base);
  s.ah = buf_ld(rsb, voff, base + vb);
#pragma unroll
  for (int k = 0; k < KM; ++k) {
    const int kk = k < a.K ? k : a.K - 1;
    s.eh[k] = buf_ld(rsb, voff, base + (2 + kk) * vb);
    s.tz[k] = buf_ld(rsb, voff, base + (2 + a.K + kk) * vb);
    s.th[k] = buf_ld(rsb, voff, base + (2 + 2 * a.K + kk) * vb);
  }
  const size_t nl = (static_cast<size_t>(b) * a.L + ii) * a.K + (lane < a.K ? lane : a.K - 1);
  s.cl = a.cand_logit[nl];
  s.xs = a.X[nl];
  s.ci = a.cand_id[nl];
}

constexpr int kScanOutChunk = 32;  // steps whose outputs are staged in LDS at once
constexpr int kScanMaxWaves = 8;

template <int KM, int D>
__global__ __launch_bounds__(512) void scan_kernel(ScanArgs a) {
  constexpr int NV = KM + 1;                 // K residual sums + the gate sum
  constexpr int NQ = kScanMaxWaves * 4;      // row sums per value
  __shared__ __align__(16) float red[2][NV][NQ];
  __shared__ float o_ref[kScanOutChunk][KM], o_res[kScanOutChunk][KM], o_gam[kScanOutChunk];
  __shared__ int o_sel[kScanOutChunk];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int nw = blockDim.x >> 6;
  const int nq = nw * 4;
  const int b = blockIdx.x;
  const int ds = a.ds, K = a.K, L = a.L;
  const int NC = a.B * L * K;
  const int e = w * 64 + lane;
  const bool ok = e < ds;
  const int ec = ok ? e : ds - 1;
  const int F = 2 + 3 * K;
  const __amdgpu_buffer_rsrc_t rsb = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<float*>(a.SB + static_cast<size_t>(b) * L * F * a.vs), static_cast<short>(0),
      L * F * a.vs * 4, 0x00020000);
  const int voff = ec * 4;

  float fz[5], fh[5];
  const float u0a = a.U0[static_cast<size_t>(b) * ds + ec];
  const float u0b = a.U0[static_cast<size_t>(a.B + b) * ds + ec];
  const float wg_e = bf16_to_f32(a.w_g[ec]);
#pragma unroll
  for (int f = 0; f < 5; ++f) {
    fz[f] = a.FZ[f * ds + ec];
    fh[f] = a.FH[f * ds + ec];
  }
  float u = ok ? tanhf(u0a + u0b) : 0.f;
  const float wgu = ok ? wg_e : 0.f;
  float wgphi[5];
#pragma unroll
  for (int f = 0; f < 5; ++f) wgphi[f] = bf16_to_f32(a.w_g[ds + f]);
  const float sig_alpha = sigmoidf_(a.alpha);

  float prev_tz = a.TZA[static_cast<size_t>(b) * ds + ec];
  float prev_th = a.THA[static_cast<size_t>(b) * ds + ec];
  float prev_x = a.X[NC + b];
  int prev_tok = a.anchor[b];
  const int my_v = lane < K ? lane : 0;  // the residual sum this lane assembles

  auto flush = [&](int i0, int n) {
    __syncthreads();
    if (w == 0) {
      for (int t = 0; t < n; ++t) {
        const size_t r = static_cast<size_t>(b) * L + i0 + t;
        if (lane < K) {
          if (a.refined) a.refined[r * K + lane] = o_ref[t][lane];
          if (a.resid) a.resid[r * K + lane] = o_res[t][lane];
        }
        if (lane == 0) {
          a.selected[r] = o_sel[t];
          if (a.gamma) a.gamma[r] = o_gam[t];
        }
      }
    }
    __syncthreads();
  };

  auto step = [&](const StepData<KM>& c, int i) {
    const float c0 = readlane_f32(c.cl, 0), c1 = readlane_f32(c.cl, 1), c3 = readlane_f32(c.cl, 3);
    const int id0 = __builtin_amdgcn_readlane(c.ci, 0);
    const bool in4 = __ballot(lane < 4 && c.ci == prev_tok) != 0;
    float phi[5];
    phi[0] = c0 - c1;
    phi[1] = c0 - c3;
    phi[2] = prev_tok == id0 ? 1.f : 0.f;
    phi[3] = in4 ? 1.f : 0.f;
    phi[4] = c0 - prev_x;

    float gz = c.az + prev_tz, gh = c.ah + prev_th;
#pragma unroll
    for (int f = 0; f < 5; ++f) {
      gz += fz[f] * phi[f];
      gh += fh[f] * phi[f];
    }
    const float z = sigmoidf_(gz);
    u = ok ? (1.f - z) * u + z * gh : 0.f;

    float v[NV];
#pragma unroll
    for (int k = 0; k < KM; ++k) v[k] = u * c.eh[k];
    v[KM] = u * wgu;
#pragma unroll
    for (int k = 0; k < NV; ++k) v[k] += dpp_f32<0xB1>(v[k]);
#pragma unroll
    for (int k = 0; k < NV; ++k) v[k] += dpp_f32<0x4E>(v[k]);
#pragma unroll
    for (int k = 0; k < NV; ++k) v[k] += dpp_f32<0x141>(v[k]);
#pragma unroll
    for (int k = 0; k < NV; ++k) v[k] += dpp_f32<0x140>(v[k]);
    const int buf = i & 1;
    if ((lane & 15) == 0) {
      const int q = w * 4 + (lane >> 4);
#pragma unroll
      for (int k = 0; k < NV; ++k) red[buf][k][q] = v[k];
    }
    __syncthreads();
    float my_d = 0.f, s = 0.f;
    for (int q = 0; q < nq; q += 4) {
      const float4 rd = *reinterpret_cast<const float4*>(&red[buf][my_v][q]);
      const float4 rg = *reinterpret_cast<const float4*>(&red[buf][KM][q]);
      my_d += (rd.x + rd.y) + (rd.z + rd.w);
      s += (rg.x + rg.y) + (rg.z + rg.w);
    }
    s += a.b_g;
#pragma unroll
    for (int f = 0; f < 5; ++f) s += wgphi[f] * phi[f];
    const float g = sig_alpha * sigmoidf_(s);
    my_d = lane < K ? my_d : 0.f;
    const float lt = c.cl + g * my_d;
    const float m = wave_allmax(lane < K ? lt : -INFINITY);
    const uint64_t hit = __ballot(lane < K && lt == m);
    const int kstar = hit ? __builtin_ctzll(hit) : 0;
    const int sel = __builtin_amdgcn_readlane(c.ci, kstar);
    const int t = i % kScanOutChunk;
    if (w == 0) {
      if (lane < K) {
        o_ref[t][lane] = lt;
        o_res[t][lane] = my_d;
      }
      if (lane == 0) {
        o_sel[t] = sel;
        o_gam[t] = g;
      }
    }
    float tz = c.tz[0], th = c.th[0];
#pragma unroll
    for (int k = 1; k < KM; ++k) {
      tz = k == kstar ? c.tz[k] : tz;
      th = k == kstar ? c.th[k] : th;
    }
    prev_tz = tz;
    prev_th = th;
    prev_x = readlane_f32(c.xs, kstar);
    prev_tok = sel;
    if (t == kScanOutChunk - 1 || i == L - 1) flush(i - t, t + 1);
  };

  StepData<KM> q[D];
#pragma unroll
  for (int t = 0; t < D; ++t) load_step<KM>(q[t], a, rsb, voff, b, t, lane);
  for (int i = 0; i < L; i += D) {
#pragma unroll
    for (int t = 0; t < D; ++t) {
      if (i + t < L) step(q[t], i + t);
      load_step<KM>(q[t], a, rsb, voff, b, i + t + D, lane);
    }
  }
}

// ---------------------------------------------------------------------------
// scan_pc: one sequence per workgroup of two wavefronts (d_state <= 256).
// Wave 1 is a copy engine: it streams the step blocks of the next rows into a
// ring of D LDS slots with buffer-to-LDS DMA (one instruction per 1 KiB
// vector, and 64-word vectors for the candidate logits, ids and cross
// logits), waiting only for the row the recurrence is about to use.  Wave 0
// runs the recurrence; lane l holds state elements 4l..4l+3.  One workgroup
// barrier per row hands a filled slot to wave 0 and a consumed slot back to
// wave 1, so the copies of later rows overlap the arithmetic of the current
// one and neither wave spends issue slots on the other's work.
// Step-block vectors are zero beyond d_state, so the padded state elements
// stay zero without any masking in the loop.
// ---------------------------------------------------------------------------
template <int KM>
struct LdsStage {
  static constexpr int NVEC = 2 + 3 * KM;       // AZ, AH, EH_k, TZ_k, TH_k
  static constexpr int NDMA = NVEC + 3;         // + candidate logits, ids, cross logits
  static constexpr int FLOATS = NVEC * 256 + 3 * 64;
};

// s_waitcnt vmcnt(N), leaving the other counters unconstrained.
template <int N>
__device__ __forceinline__ void wait_vm() {
  __builtin_amdgcn_s_waitcnt((N & 15) | (((N >> 4) & 3) << 14) | (7 << 4) | (15 << 8));
}

// Workgroup barrier that is also a compiler barrier for memory accesses (the
// LDS reads after it must not be moved above it).
__device__ __forceinline__ void wg_barrier() { asm volatile("s_barrier" ::: "memory"); }

typedef __attribute__((address_space(3))) void* lds_vptr_t;
typedef float f4_t __attribute__((ext_vector_type(4)));

// DPP row broadcast into the rows selected by ROWMASK (others receive 0).
template <int CTRL, int ROWMASK>
__device__ __forceinline__ float dpp_rows(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, ROWMASK, 0xF, false));
}

__device__ __forceinline__ float sigmoid_rcp(float x) {
  return __builtin_amdgcn_rcpf(1.0f + __expf(-x));
}

// `ids` is the candidate-id array again, as a kernel argument of its own: read
// only and unaliased, so the copy engine's wave-uniform reads of it become
// scalar loads, which leave the vector-memory counter to the row copies.
template <int KM, int D, bool TAB>
__global__ __launch_bounds__(128) void scan_pc_kernel(ScanArgs a, const int32_t* __restrict__ ids_in) {
  using S = LdsStage<KM>;
  static_assert((D - 2) * S::NDMA <= 63, "vmcnt range");
  static_assert(2 * KM <= 62, "output lanes");
  __shared__ __align__(16) float ring[D * S::FLOATS];
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int b = blockIdx.x;
  const int ds = a.ds, K = a.K, L = a.L;
  const int F = 2 + 3 * K;
  const size_t row0 = static_cast<size_t>(b) * L;

  if (wave == 1) {
    // ---- copy engine --------------------------------------------------------
    const __amdgpu_buffer_rsrc_t rsb = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float*>(a.SB + row0 * F * 256), static_cast<short>(0), L * F * 1024, 0x00020000);
    const __amdgpu_buffer_rsrc_t rcl = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float*>(a.cand_logit + row0 * K), static_cast<short>(0), L * K * 4, 0x00020000);
    const __amdgpu_buffer_rsrc_t rci = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<int32_t*>(a.cand_id + row0 * K), static_cast<short>(0), L * K * 4, 0x00020000);
    const __amdgpu_buffer_rsrc_t rxs = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float*>(a.X + row0 * K), static_cast<short>(0), L * K * 4, 0x00020000);
    // the tables' byte size fits 32 bits (checked on the host)
    constexpr bool tab = TAB;
    const __amdgpu_buffer_rsrc_t rtb = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float*>(tab ? a.tables : a.SB), static_cast<short>(0),
        tab ? static_cast<int>(3u * static_cast<unsigned>(a.V) * 1024u) : 0, 0x00020000);
    // Token ids of the candidates of row i, wave-uniform (scalar loads),
    // fetched one row before the row's copies are issued.
    int ids[KM];
    auto load_ids = [&](int i) {
      const int ii = i < L ? i : L - 1;
      const int32_t* src = ids_in + (row0 + ii) * K;
      // all loads first, one wait for them
#pragma unroll
      for (int k = 0; k < KM; ++k) ids[k] = src[k < K ? k : K - 1];
    };
    auto clamp_ids = [&] {
#pragma unroll
      for (int k = 0; k < KM; ++k) ids[k] = __builtin_amdgcn_readfirstlane(clamp_id(ids[k], a.V));
    };
    // Copies of row i (clamped to the block) into slot i % D.  Candidate slots
    // k >= K repeat candidate K-1, so every row issues exactly NDMA copies and
    // vmcnt(n * NDMA) always means "every row but the n last issued landed".
    auto issue = [&](int i) {
      const int ii = i < L ? i : L - 1;
      float* st = ring + (i % D) * S::FLOATS;
      const unsigned rb = static_cast<unsigned>(ii * F) * 1024u;
      if constexpr (tab) clamp_ids();
#pragma unroll
      for (int v = 0; v < S::NVEC; ++v) {
        if (tab && v >= 2) {
          // table kind (EH, TZ, TH) and candidate slot of vector v
          const int kind = (v - 2) / KM, k = (v - 2) % KM;
          const unsigned off = (static_cast<unsigned>(kind) * static_cast<unsigned>(a.V) +
                                static_cast<unsigned>(ids[k])) * 1024u;
          __builtin_amdgcn_raw_ptr_buffer_load_lds(rtb, (lds_vptr_t)(st + v * 256), 16, lane * 16, off, 0, 0);
          continue;
        }
        int f;
        if (v < 2) f = v;
        else if (v < 2 + KM) f = 2 + min(v - 2, K - 1);
        else if (v < 2 + 2 * KM) f = 2 + K + min(v - 2 - KM, K - 1);
        else f = 2 + 2 * K + min(v - 2 - 2 * KM, K - 1);
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rsb, (lds_vptr_t)(st + v * 256), 16, lane * 16,
                                                 rb + static_cast<unsigned>(f) * 1024u, 0, 0);
      }
      const unsigned cb = static_cast<unsigned>(ii * K) * 4u;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rcl, (lds_vptr_t)(st + S::NVEC * 256), 4, lane * 4, cb, 0, 0);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rci, (lds_vptr_t)(st + S::NVEC * 256 + 64), 4, lane * 4, cb, 0, 0);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rxs, (lds_vptr_t)(st + S::NVEC * 256 + 128), 4, lane * 4, cb, 0, 0);
    };
    // The gate terms that depend on the row alone (features 0 and 1, and
    // the candidate-logit half of feature 4) are folded into AZ and AH in
    // the slot before the recurrence reads it, and the row's part of the
    // selection gate's pre-activation goes to word 63 of the logit vector
    // (a lane >= K, which nothing else reads).
    float cz[4][3], ch[4][3];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const bool ok = 4 * lane + j < ds;
      const int e = ok ? 4 * lane + j : ds - 1;
#pragma unroll
      for (int q = 0; q < 3; ++q) {
        const int f = q < 2 ? q : 4;
        const float z = a.FZ[f * ds + e], h = a.FH[f * ds + e];
        cz[j][q] = ok ? z : 0.f;
        ch[j][q] = ok ? h : 0.f;
      }
    }
    float wphi[3];
#pragma unroll
    for (int q = 0; q < 3; ++q) wphi[q] = bf16_to_f32(a.w_g[ds + (q < 2 ? q : 4)]);
    auto prep = [&](int r) {
      float* st = ring + (r % D) * S::FLOATS;
      f4_t* sv = reinterpret_cast<f4_t*>(st) + lane;
      float* sc = st + S::NVEC * 256;
      const float c0 = sc[0], p0 = c0 - sc[1], p1 = c0 - sc[3];
      f4_t az = sv[0], ah = sv[64];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        az[j] += cz[j][0] * p0 + cz[j][1] * p1 + cz[j][2] * c0;
        ah[j] += ch[j][0] * p0 + ch[j][1] * p1 + ch[j][2] * c0;
      }
      sv[0] = az;
      sv[64] = ah;
      if (lane == 63) sc[63] = a.b_g + wphi[0] * p0 + wphi[1] * p1 + wphi[2] * c0;
    };
    // LDS writes complete before the barrier that hands the row over
    auto handover = [] { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); };
#pragma unroll
    for (int t = 0; t < D - 1; ++t) {
      if constexpr (tab) load_ids(t);
      issue(t);
    }
    if constexpr (tab) load_ids(D - 1);
    wait_vm<(D - 2) * S::NDMA>();  // row 0 has landed
    prep(0);
    for (int i = 0; i < L; ++i) {
      wait_vm<(D - 3) * S::NDMA>();  // row i + 1 has landed
      prep(i + 1);
      handover();                    // hand slot i over; slot (i-1) % D is free again
      issue(i + D - 1);
      if constexpr (tab) load_ids(i + D);  // the next row's ids, used at the next step
    }
    wait_vm<0>();  // no copy may land after the workgroup's LDS is released
    return;
  }

  // ---- recurrence (wave 0) ---------------------------------------------------
  float u[4], wgu[4], fz[4][5], fh[4][5];
  f4_t ptz, pth;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const bool ok = 4 * lane + j < ds;
    const int e = ok ? 4 * lane + j : ds - 1;
    const float u0a = a.U0[static_cast<size_t>(b) * ds + e];
    const float u0b = a.U0[static_cast<size_t>(a.B + b) * ds + e];
    u[j] = ok ? tanhf(u0a + u0b) : 0.f;
    wgu[j] = ok ? bf16_to_f32(a.w_g[e]) : 0.f;
    float tz, th;
    if constexpr (TAB) {  // the anchor's rows of the TZ and TH tables
      const size_t x0 = static_cast<size_t>(clamp_id(a.anchor[b], a.V));
      tz = a.tables[(static_cast<size_t>(a.V) + x0) * 256 + e];
      th = a.tables[(2 * static_cast<size_t>(a.V) + x0) * 256 + e];
    } else {
      tz = a.TZA[static_cast<size_t>(b) * ds + e];
      th = a.THA[static_cast<size_t>(b) * ds + e];
    }
    ptz[j] = ok ? tz : 0.f;
    pth[j] = ok ? th : 0.f;
#pragma unroll
    for (int f = 0; f < 5; ++f) {
      const float z = a.FZ[f * ds + e], h = a.FH[f * ds + e];
      fz[j][f] = ok ? z : 0.f;
      fh[j][f] = ok ? h : 0.f;
    }
  }
  float wgphi[5];
#pragma unroll
  for (int f = 0; f < 5; ++f) wgphi[f] = bf16_to_f32(a.w_g[ds + f]);
  const float sig_alpha = sigmoidf_(a.alpha);
  float prev_x = a.X[static_cast<size_t>(a.B) * L * K + b];
  int prev_tok = a.anchor[b];

  // Each lane stores one value per row: lanes < K the refined logits, lanes
  // K..2K-1 the residuals, lane 62 the gate, lane 63 the selected id; lanes
  // without an output (or whose output was not requested) write to a sink.
  const bool want = a.refined != nullptr || a.resid != nullptr;
  // Verification on the fly: step i's selection sits in lane i % 64; at the
  // end of every 64 steps a ballot against the verifier's tokens of those
  // steps (loaded a chunk ahead) finds the first mismatch.
  const bool fuse = a.verifier != nullptr;
  int mysel = 0, first_mis = L, corr_tok = -1;
  auto load_ver = [&](int c0) {
    const int i = c0 + lane;
    return fuse && i < L ? a.verifier[row0 + i] : 0;
  };
  int vchunk = load_ver(0);
  const int kd = lane < K ? lane : lane - K;
  // reduce-scatter keep rules and the candidate each lane ends up holding
  const bool kb0 = lane & 1, kb1 = lane & 2, kb2 = lane & 4, kb3 = lane & 8;
  const bool kc0 = kb0 != kb2, kc1 = kb1 != kb2;
  const int my_cand = KM == 16 ? 8 * kc0 + 4 * kc1 + 2 * kb2 + kb3 : 4 * kc0 + 2 * kc1 + kb2;
  // a lane holding candidate kd (bpermute address)
  int out_src;
  {
    const int o = kd < KM ? kd : 0;
    int ob0, ob1, ob2, ob3 = 0;
    if (KM == 16) {
      ob3 = o & 1;
      ob2 = (o >> 1) & 1;
      ob1 = ((o >> 2) & 1) ^ ob2;
      ob0 = ((o >> 3) & 1) ^ ob2;
    } else {
      ob2 = o & 1;
      ob1 = ((o >> 1) & 1) ^ ob2;
      ob0 = ((o >> 2) & 1) ^ ob2;
    }
    out_src = 4 * (ob0 + 2 * ob1 + 4 * ob2 + 8 * ob3);
  }
  float* obase = a.dump + static_cast<size_t>(b) * 64 + lane;
  size_t ostride = 0;
  if (lane < K && a.refined) { obase = a.refined + lane; ostride = K; }
  else if (lane >= K && lane < 2 * K && a.resid) { obase = a.resid + (lane - K); ostride = K; }
  else if (lane == 62 && a.gamma) { obase = a.gamma; ostride = 1; }
  else if (lane == 63) { obase = reinterpret_cast<float*>(a.selected); ostride = 1; }

  for (int i = 0; i < L; ++i) {
    // The copy wave refills the slot of row i - 1 once this barrier passes,
    // so the reads of that slot (the previous-token vectors, the last ones
    // of step i - 1) must have returned first.
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    wg_barrier();  // row i is in slot i % D
    const float* st = ring + (i % D) * S::FLOATS;
    const f4_t* sv = reinterpret_cast<const f4_t*>(st) + lane;  // vector v of the row at sv[64 v]
    const float* sc = st + S::NVEC * 256;                          // logits, ids, cross logits
    const f4_t az = sv[0], ah = sv[64];
    f4_t eh[KM];
#pragma unroll
    for (int k = 0; k < KM; ++k) eh[k] = sv[64 * (2 + k)];
    const float cl_l = sc[lane], xs_l = sc[128 + lane], cl_mine = sc[my_cand];
    const int ci_l = __float_as_int(sc[64 + lane]);
    const float s_row = sc[63];
    int idu[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) idu[k] = __float_as_int(sc[64 + k]);

    // AZ and AH arrive with the row-only feature terms folded in; features 2
    // and 3 (the previous token is the top candidate / among the top four)
    // and the previous cross logit remain
    float phi[5];
    phi[2] = prev_tok == idu[0] ? 1.f : 0.f;
    phi[3] = (prev_tok == idu[0] || prev_tok == idu[1] || prev_tok == idu[2] || prev_tok == idu[3]) ? 1.f : 0.f;

#pragma unroll
    for (int j = 0; j < 4; ++j) {
      float gz = az[j] + ptz[j], gh = ah[j] + pth[j];
      gz += fz[j][2] * phi[2] + fz[j][3] * phi[3] - fz[j][4] * prev_x;
      gh += fh[j][2] * phi[2] + fh[j][3] * phi[3] - fh[j][4] * prev_x;
      const float z = sigmoid_rcp(gz);
      u[j] = (1.f - z) * u[j] + z * gh;
    }

    float v[KM + 1];
#pragma unroll
    for (int k = 0; k < KM; ++k) v[k] = u[0] * eh[k][0] + u[1] * eh[k][1] + u[2] * eh[k][2] + u[3] * eh[k][3];
    v[KM] = u[0] * wgu[0] + u[1] * wgu[1] + u[2] * wgu[2] + u[3] * wgu[3];
    // 64-lane sums of the KM candidate partials as a reduce-scatter: at each
    // level a lane keeps one half of its values, adds its partner's copy of
    // that half and hands the other half over, so the number of values per
    // lane halves.  The keep rules (bit0^bit2, bit1^bit2, bit2, bit3) make the
    // half-mirror partner hold the same half as the lane, and the last
    // levels (rotate by 8 in the row, then swaps across 16 and 32 lanes) pair
    // lanes with the same index.  Every lane ends with the full sum of
    // candidate my_cand; the gate partial is summed whole.
    float w[KM / 2];
#pragma unroll
    for (int m = 0; m < KM / 2; ++m) {
      const float keep = kc0 ? v[m + KM / 2] : v[m], send = kc0 ? v[m] : v[m + KM / 2];
      w[m] = keep + dpp_f32<0xB1>(send);  // quad_perm [1,0,3,2]: lane ^ 1
    }
    float x[KM / 4];
#pragma unroll
    for (int m = 0; m < KM / 4; ++m) {
      const float keep = kc1 ? w[m + KM / 4] : w[m], send = kc1 ? w[m] : w[m + KM / 4];
      x[m] = keep + dpp_f32<0x4E>(send);  // quad_perm [2,3,0,1]: lane ^ 2
    }
    float y[KM / 8];
#pragma unroll
    for (int m = 0; m < KM / 8; ++m) {
      const float keep = kb2 ? x[m + KM / 8] : x[m], send = kb2 ? x[m] : x[m + KM / 8];
      y[m] = keep + dpp_f32<0x141>(send);  // row_half_mirror: lane ^ 7 in each 8
    }
    float dsum;
    if constexpr (KM == 16) {
      const float keep = kb3 ? y[1] : y[0], send = kb3 ? y[0] : y[1];
      dsum = keep + dpp_f32<0x128>(send);  // row_ror 8: lane ^ 8
    } else {
      dsum = y[0] + dpp_f32<0x128>(y[0]);
    }
    dsum = swap16_sum(dsum);
    dsum = swap32_sum(dsum);
    float gsum = row_sum16(v[KM]);
    gsum = swap32_sum(swap16_sum(gsum));
    // the row's part of the pre-activation (b_g and features 0, 1 and the
    // logit half of 4) waits in word 63 of the slot's logit vector
    const float s = gsum + s_row + wgphi[2] * phi[2] + wgphi[3] * phi[3] - wgphi[4] * prev_x;
    const float g = sig_alpha * sigmoid_rcp(s);

    // refined logits and their argmax (the first maximum: smallest k on
    // ties); every row holds all KM candidates, so row-wide reductions do
    const float lt = my_cand < K ? __builtin_fmaf(g, dsum, cl_mine) : -INFINITY;
    const float best = row_max16(lt);
    int key = my_cand < K && lt == best ? my_cand : KM;
    key = min(key, dpp_i32<0xB1>(key));
    key = min(key, dpp_i32<0x4E>(key));
    key = min(key, dpp_i32<0x141>(key));
    key = min(key, dpp_i32<0x140>(key));
    const int kstar = __builtin_amdgcn_readfirstlane(key);
    const int sel = __builtin_amdgcn_readlane(ci_l, kstar);
    prev_x = readlane_f32(xs_l, kstar);
    ptz = sv[64 * (2 + KM + kstar)];
    pth = sv[64 * (2 + 2 * KM + kstar)];
    prev_tok = sel;

    float ov = g;
    if (want) {
      // candidate kd's sum from a lane that holds it
      const float dl = __int_as_float(__builtin_amdgcn_ds_bpermute(out_src, __float_as_int(dsum)));
      ov = lane < K ? __builtin_fmaf(g, dl, cl_l) : (lane < 2 * K ? dl : g);
    }
    ov = lane == 63 ? __int_as_float(sel) : ov;
    obase[(row0 + i) * ostride] = ov;
    if (fuse) {
      mysel = lane == (i & 63) ? sel : mysel;
      if ((i & 63) == 63 || i == L - 1) {
        const int c0 = i & ~63;
        const uint64_t mis = __ballot(c0 + lane <= i && mysel != vchunk);
        if (first_mis == L && mis) {
          first_mis = c0 + static_cast<int>(__builtin_ctzll(mis));
          corr_tok = __builtin_amdgcn_readlane(vchunk, first_mis - c0);
        }
        if (i + 1 < L) vchunk = load_ver(c0 + 64);
      }
    }
  }
  if (fuse && lane == 0) {
    a.accept_len[b] = first_mis;
    if (a.correction) a.correction[b] = first_mis < L ? corr_tok : -1;
  }
}

// ---------------------------------------------------------------------------
// Step blocks from the per-token tables (brisk_corrector_prepare): for row r
// and candidate k the vectors EH_k, TZ_k, TH_k are rows c_{r,k} of the EH, TZ
// and TH tables, and the anchor lifts TZA, THA are rows x_0 of TZ and TH.
// One wavefront copies one vector, 16 bytes per lane.
// ---------------------------------------------------------------------------
// Vector stride of the step blocks: one 256-float vector per field when the
// state fits (the single-wave scan copies whole 1 KiB vectors), else d_state.
size_t step_vec_stride(int ds) { return ds <= 256 ? 256 : static_cast<size_t>(ds); }

struct Layout {
  size_t PE, PC, PH, U0, X, SB, TZA, THA, FZ, FH, DUMP, total;
  size_t sPE, sPC, sPH, sU0;  // floats between split-K slices (multiples of 64)
  int splits;
};

int proj_tiles(int n, int J, int bj = 64) { return ((J + bj - 1) / bj) * ((n + PJ_BN - 1) / PJ_BN); }

// Split the gather projections' reduction so that about 1024 workgroups run
// even when the batch is small; never more than 16 slices.  Only the jobs
// that run count: with the per-token tables the candidates' and anchors'
// projections are not computed, and the hidden-state projection alone would
// otherwise run unsplit on a few dozen workgroups (at 4096 rows it was the
// longest part of the launch).
int proj_splits(const brisk_corrector& c, int B, int L, int K, bool tab) {
  const int rows = B * L, NC = rows * K;
  int tiles = proj_tiles(rows, c.d_hproj) + 2 * proj_tiles(B, c.d_state);
  if (!tab) tiles += proj_tiles(NC, c.d_tproj) + proj_tiles(B, c.d_tproj) + proj_tiles(NC, c.rank);
  int sp = 1024 / (tiles > 0 ? tiles : 1);
  return sp < 1 ? 1 : (sp > 16 ? 16 : sp);
}

Layout rerank_layout(const brisk_corrector& c, int B, int L, int K, bool tab) {
  const size_t rows = static_cast<size_t>(B) * L, NC = rows * K, NP = NC + B;
  const size_t ds = c.d_state;
  Layout l{};
  l.splits = proj_splits(c, B, L, K, tab);
  const size_t S = l.splits;
  auto pad = [](size_t n) { return (n + 63) / 64 * 64; };
  // with the tables no candidate or anchor is projected
  l.sPE = tab ? 0 : pad(NP * c.d_tproj);
  l.sPC = tab ? 0 : pad(NC * c.rank);
  l.sPH = pad(rows * c.d_hproj);
  l.sU0 = pad(2 * static_cast<size_t>(B) * ds);
  size_t off = 0;
  auto take = [&](size_t floats) {
    const size_t o = off;
    off += (floats * sizeof(float) + 255) / 256 * 256;
    return o;
  };
  l.PE = take(S * l.sPE);
  l.PC = take(S * l.sPC);
  l.PH = take(S * l.sPH);
  l.U0 = take(S * l.sU0);
  l.X = take(NP);
  l.SB = take(rows * (2 + 3 * static_cast<size_t>(K)) * step_vec_stride(ds));
  l.TZA = take(static_cast<size_t>(B) * ds);
  l.THA = take(static_cast<size_t>(B) * ds);
  l.FZ = take(5 * ds);
  l.FH = take(5 * ds);
  l.DUMP = take(static_cast<size_t>(B) * 64);
  l.total = off;
  return l;
}

template <int KM, int D>
void launch_scan(const ScanArgs& sa, int B, int nw, hipStream_t s) {
  hipLaunchKernelGGL((scan_kernel<KM, D>), dim3(B), dim3(64 * nw), 0, s, sa);
}

}  // namespace

// Large enough for either path, so a workspace sized before the tables were
// prepared (or after they were dropped) still fits.
size_t rerank_workspace_bytes(const brisk_corrector& c, int B, int L, int K) {
  return std::max(rerank_layout(c, B, L, K, false).total, rerank_layout(c, B, L, K, true).total);
}

void launch_rerank(const brisk_corrector& c, const uint16_t* hidden, const uint16_t* ctx_hidden,
                   const int32_t* anchor_tok, const uint16_t* lm_head, const uint16_t* tok_embed,
                   const float* cand_logit, const int32_t* cand_id, int B, int L, int K, int d,
                   int V, int32_t* selected, float* refined, float* gamma, float* resid,
                   const int32_t* verifier, int32_t* accept_len, int32_t* correction, void* ws,
                   hipStream_t s, RerankPart part) {
  const bool tab = c.tables != nullptr;
  // The hoisted part: the hidden-state, context and A_e anchor projections,
  // the sums of their split slices and their lifts (with the feature maps).
  // The rest reads candidates, or (without the tables) shares the PE array
  // and its slice sum with them: the candidate and anchor P_e projections,
  // the W_c projections, the cross logits, their lifts, the table rows, the
  // scan and the verification.
  const bool hoist = part != RerankPart::kFinish, finish = part != RerankPart::kHoist;
  const Layout lay = rerank_layout(c, B, L, K, tab);
  char* base = static_cast<char*>(ws);
  auto F = [&](size_t off) { return reinterpret_cast<float*>(base + off); };
  const int rows = B * L, NC = rows * K, NP = NC + B;
  const int ds = c.d_state;
  const int d_in = c.d_hproj + c.d_tproj + c.d_pos + c.d_feat;
  const int tp_off = c.d_hproj, pos_off = c.d_hproj + c.d_tproj, feat_off = pos_off + c.d_pos;
  const int S = lay.splits;

  // Slices of PE are [NP, d_tproj]: candidate rows, then anchor rows.
  // Slices of U0 are [2, B, ds]: A_h h_c, then A_e E(x_0).
  const size_t sPE = lay.sPE, sPC = lay.sPC, sPH = lay.sPH, sU0 = lay.sU0;
  // With the per-token tables, every per-candidate and per-anchor lift is a
  // table row: the projections of candidates and anchors are not computed.
  const int n_cand = tab ? 0 : NC, n_anch = tab ? 0 : B;
  const int fc = finish ? n_cand : 0, fa = finish ? n_anch : 0;  // rows of the finishing jobs
  const int hr = hoist ? rows : 0, hb = hoist ? B : 0;             // and of the hoisted ones
  ProjJobs pj{};
  pj.d = d;
  pj.splits = S;
  pj.job[0] = ProjJob{tok_embed, cand_id, fc, c.d_tproj, V, c.P_e, F(lay.PE), sPE};
  pj.job[1] = ProjJob{tok_embed, anchor_tok, fa, c.d_tproj, V, c.P_e, F(lay.PE) + static_cast<size_t>(NC) * c.d_tproj, sPE};
  pj.job[2] = ProjJob{lm_head, cand_id, fc, c.rank, V, c.W_c, F(lay.PC), sPC};
  pj.job[3] = ProjJob{hidden, nullptr, hr, c.d_hproj, rows, c.P_h, F(lay.PH), sPH};
  pj.job[4] = ProjJob{ctx_hidden, nullptr, hb, ds, B, c.A_h, F(lay.U0), sU0};
  pj.job[5] = ProjJob{tok_embed, anchor_tok, hb, ds, V, c.A_e, F(lay.U0) + static_cast<size_t>(B) * ds, sU0};
  // unsplit (batched) shapes take 128-wide output tiles
  const int bj = S == 1 ? 128 : 64;
  int max_tiles = 0;
  for (int j = 0; j < kMaxProjJobs; ++j) {
    const int t = proj_tiles(pj.job[j].n, pj.job[j].J, bj);
    max_tiles = t > max_tiles ? t : max_tiles;
  }
  // Candidates per cross-logit wavefront.  Below 4096 dots, one (more
  // wavefronts win).  Up to 32768 the gather waits on latency: groups of
  // four with four chunks in flight (two rounds of loads per 4096-long dot)
  // took 83-85 against 90-93 us after the LM-head launch at 2048 rows x 8
  // keys and 92 against 97 us at 512 x 16.  From 32768 dots (268 MB of
  // lm_head rows at 4096 x 8) it streams near the HBM limit, and groups of
  // eight, which read each hidden row half as often, were 2 us faster.
  const int group = NC >= 32768 ? 8 : NC >= 4096 ? 4 : 1;
  // (no sequences: no cross logits in the hoisted part)
  pj.cross = CrossJob{lm_head, hidden, cand_id, anchor_tok, finish ? B : 0, L, K, V, F(lay.X), group};
  // the cross-logit row needs a wavefront per row and group of candidates,
  // and one per anchor, four to a workgroup (each loops over more when the
  // grid is capped at about 4096 workgroups)
  const int cross_items = finish ? rows * ((K + group - 1) / group) + B : 0;
  const int cross_x = std::min(((cross_items + 3) / 4 + S - 1) / S, (4096 + S - 1) / S);
  const bool pc = ds <= 256 && K <= 16;  // the single-wave scan, which can verify in the same pass
  // Who brings the table rows to the scan.  The single-wave scan can gather
  // them itself (its copy wave issues each row's copies three rows ahead), but
  // random 1 KiB reads from the tables outlast that lead: at 32 rows the scan
  // took 40 instead of 23 us, with 16 keys (two rows of lead) 72 instead of
  // 36 us.  Copying the rows into the step blocks first is a parallel,
  // bandwidth-bound pass whose cost grows with the batch (5 us at 32 rows,
  // 17 us at 2048, 32 us at 4096), against a latency the gathering scan pays
  // once per step whatever the batch: the whole rerank took 89.5 against
  // 76.3 us with gathering at 64 x 32 rows, and 165 against 140 us at
  // 256 x 16, so the scan gathers from 64 sequences on.
  const bool scan_gathers = tab && pc && K <= 8 && B >= 64;
  // Without it the scan reads whole step blocks and the table rows are
  // copied in, kFillBatch rows a wavefront at a time.  Up to 4096 rows
  // (4 MiB) the projection launch copies them, which saves a launch
  // (32 rows: 2.5 us of a rerank's 43); more would stretch that launch
  // (512 x 16 rows: 24 us against 15 + 8 us for two launches).
  const size_t vsz = step_vec_stride(ds);
  float* SB = F(lay.SB);
  const bool fill = finish && tab && !scan_gathers;
  const int n_vec = fill ? rows * 3 * K + 2 * B : 0;
  const bool fill_here = fill && n_vec <= 4096;
  const FillArgs fargs{c.tables, cand_id, anchor_tok, SB, F(lay.TZA), F(lay.THA), fill ? rows : 0, K,
                       fill ? B : 0, V, ds, static_cast<int>(vsz)};
  if (fill_here) pj.fill = fargs;
  const int fill_x =
      fill_here ? std::min(((n_vec + 4 * kFillBatch - 1) / (4 * kFillBatch) + S - 1) / S, (4096 + S - 1) / S) : 0;
  const int gx = std::max(max_tiles, std::max(cross_x, fill_x));
  const int gy = kMaxProjJobs + (fill_here ? 2 : 1);  // the table-row row only when it copies
  if (gx > 0) {
    if (bj == 128)
      hipLaunchKernelGGL(gather_proj_kernel<128>, dim3(gx, gy, S), dim3(256), 0, s, pj);
    else
      hipLaunchKernelGGL(gather_proj_kernel<64>, dim3(gx, gy, S), dim3(256), 0, s, pj);
  }
  if (fill && !fill_here)
    hipLaunchKernelGGL(fill_kernel, dim3((n_vec + 4 * kFillBatch - 1) / (4 * kFillBatch)), dim3(256), 0, s, fargs);

  if (S > 1) {
    SliceArrs sl{};
    sl.splits = S;
    sl.arr[0] = SliceArr{F(lay.PE), tab || !finish ? 0 : sPE, sPE};
    sl.arr[1] = SliceArr{F(lay.PC), tab || !finish ? 0 : sPC, sPC};
    sl.arr[2] = SliceArr{F(lay.PH), hoist ? sPH : 0, sPH};
    sl.arr[3] = SliceArr{F(lay.U0), hoist ? sU0 : 0, sU0};
    size_t mx = 0;
    for (int a = 0; a < kMaxSliceArrs; ++a) mx = sl.arr[a].n > mx ? sl.arr[a].n : mx;
    const int blocks = static_cast<int>((mx / 4 + 255) / 256);
    if (blocks > 0) hipLaunchKernelGGL(slice_sum_kernel, dim3(blocks, kMaxSliceArrs), dim3(256), 0, s, sl);
  }

  // Step blocks: row r holds F = 2 + 3K vectors [AZ, AH, EH_k, TZ_k, TH_k].
  const int FB = 2 + 3 * K;
  const size_t blk = static_cast<size_t>(FB) * vsz;
  LiftJobs lj{};
  lj.ds = ds;
  const float* PEa = F(lay.PE) + static_cast<size_t>(NC) * c.d_tproj;
  // A term's input runs load as vectors when they are contiguous (cs == 1),
  // whole (C % 16 == 0) and 16-byte aligned; its matrix runs likewise along
  // c (m_cs == 1, C % 16 == 0) or along j (m_rs == 1, d_state % 16 == 0).
  auto term = [&](const void* in, int bf16, int rs, int cs, int period, int C, const uint16_t* m,
                  int m_rs, int m_cs) {
    const int per16 = bf16 ? 8 : 4;  // elements per 16 bytes
    const bool a16 = (reinterpret_cast<uintptr_t>(in) & 15u) == 0 && cs == 1 && C % 16 == 0 &&
                     rs % per16 == 0;
    const bool m16 = (reinterpret_cast<uintptr_t>(m) & 15u) == 0 &&
                     (m_cs == 1 ? m_rs % 8 == 0 && C % 16 == 0 : m_rs == 1 && m_cs % 8 == 0 && ds % 16 == 0);
    return LiftTerm{in, bf16, rs, cs, period, C, m, m_rs, m_cs, a16 ? 1 : 0, m16 ? 1 : 0};
  };
  // fp32 inputs: the projections, their split-K slices already summed
  auto fterm = [&](const float* in, int C, const uint16_t* m, int m_rs, int m_cs) {
    return term(in, 0, C, 1, 0, C, m, m_rs, m_cs);
  };
  const LiftTerm none{nullptr, 0, 0, 0, 0, 0, nullptr, 0, 0, 0, 0};
  const LiftTerm posz = term(c.pos_emb, 1, c.d_pos, 1, L, c.d_pos, c.W_z + pos_off, d_in, 1);
  const LiftTerm posh = term(c.pos_emb, 1, c.d_pos, 1, L, c.d_pos, c.W_h + pos_off, d_in, 1);
  const size_t vds = static_cast<size_t>(ds);
  lj.job[0] = LiftJob{{fterm(F(lay.PE), c.d_tproj, c.W_z + tp_off, d_in, 1), none}, fc, SB + (2 + K) * vsz, K, blk, vsz};
  lj.job[1] = LiftJob{{fterm(F(lay.PE), c.d_tproj, c.W_h + tp_off, d_in, 1), none}, fc, SB + (2 + 2 * K) * vsz, K, blk, vsz};
  lj.job[2] = LiftJob{{fterm(F(lay.PC), c.rank, c.W_s, 1, ds), none}, fc, SB + 2 * vsz, K, blk, vsz};
  lj.job[3] = LiftJob{{fterm(F(lay.PH), c.d_hproj, c.W_z, d_in, 1), posz}, hr, SB, 1, blk, vsz};
  lj.job[4] = LiftJob{{fterm(F(lay.PH), c.d_hproj, c.W_h, d_in, 1), posh}, hr, SB + vsz, 1, blk, vsz};
  lj.job[5] = LiftJob{{fterm(PEa, c.d_tproj, c.W_z + tp_off, d_in, 1), none}, fa, F(lay.TZA), 1, vds, vds};
  lj.job[6] = LiftJob{{fterm(PEa, c.d_tproj, c.W_h + tp_off, d_in, 1), none}, fa, F(lay.THA), 1, vds, vds};
  // feature maps W_z[:, feat] P_phi and W_h[:, feat] P_phi as [5, ds]: input row f is column f of P_phi
  lj.job[7] = LiftJob{{term(c.P_phi, 1, 1, 5, 0, c.d_feat, c.W_z + feat_off, d_in, 1), none}, hoist ? 5 : 0, F(lay.FZ), 1, vds, vds};
  lj.job[8] = LiftJob{{term(c.P_phi, 1, 1, 5, 0, c.d_feat, c.W_h + feat_off, d_in, 1), none}, hoist ? 5 : 0, F(lay.FH), 1, vds, vds};
  const int lift_cols = static_cast<int>(vsz > vds ? vsz : vds);
  int lift_rows = 0;
  for (int j = 0; j < kMaxLiftJobs; ++j) lift_rows = lj.job[j].n > lift_rows ? lj.job[j].n : lift_rows;
  const dim3 lift_grid((lift_rows + LT_BN - 1) / LT_BN, (lift_cols + LT_BJ - 1) / LT_BJ, kMaxLiftJobs);
  // Tiles of the candidate jobs and of the two hidden-state jobs: two or
  // more per compute unit -> one buffer, which fits twice as many
  // workgroups (the same choice in both parts of a split rerank).  At 4096
  // rows with the tables, 512 hidden-state tiles: the step after the LM-head
  // launch took 112.7 against 115.5 us with one buffer.
  const bool many_tiles =
      (3 * ((n_cand + LT_BN - 1) / LT_BN) + 2 * ((rows + LT_BN - 1) / LT_BN)) * ((ds + LT_BJ - 1) / LT_BJ) >= 512;
  if (lift_rows > 0) {
    if (many_tiles) hipLaunchKernelGGL(lift_kernel<1>, lift_grid, dim3(256), 0, s, lj);
    else hipLaunchKernelGGL(lift_kernel<2>, lift_grid, dim3(256), 0, s, lj);
  }
  if (!finish) return;

  ScanArgs sa{};
  sa.B = B; sa.L = L; sa.K = K; sa.ds = ds; sa.vs = static_cast<int>(vsz);
  sa.U0 = F(lay.U0); sa.X = F(lay.X); sa.SB = SB; sa.TZA = F(lay.TZA); sa.THA = F(lay.THA);
  sa.FZ = F(lay.FZ); sa.FH = F(lay.FH); sa.w_g = c.w_g;
  sa.alpha = c.alpha; sa.b_g = c.b_g;
  sa.cand_logit = cand_logit; sa.cand_id = cand_id; sa.anchor = anchor_tok;
  sa.selected = selected; sa.refined = refined; sa.gamma = gamma; sa.resid = resid;
  sa.dump = F(lay.DUMP);
  if (scan_gathers) {  // the single-wave scan gathers the table rows itself
    sa.tables = c.tables;
    sa.V = V;
  }
  if (verifier && pc) {
    sa.verifier = verifier;
    sa.accept_len = accept_len;
    sa.correction = correction;
  }
  const int nw = (ds + 63) / 64;
  if (scan_gathers)
    hipLaunchKernelGGL((scan_pc_kernel<8, 4, true>), dim3(B), dim3(128), 0, s, sa, cand_id);
  else if (ds <= 256 && K <= 8)
    hipLaunchKernelGGL((scan_pc_kernel<8, 4, false>), dim3(B), dim3(128), 0, s, sa, cand_id);
  else if (ds <= 256 && K <= 16)
    hipLaunchKernelGGL((scan_pc_kernel<16, 3, false>), dim3(B), dim3(128), 0, s, sa, cand_id);
  else if (K <= 8) launch_scan<8, 4>(sa, B, nw, s);
  else if (K <= 16) launch_scan<16, 3>(sa, B, nw, s);
  else launch_scan<64, 1>(sa, B, nw, s);
  if (verifier && !pc) launch_verify(selected, verifier, B, L, accept_len, correction, s);
}

size_t corrector_tables_bytes(const brisk_corrector& c, int V) {
  return 3 * static_cast<size_t>(V) * step_vec_stride(c.d_state) * sizeof(float);
}

size_t corrector_prepare_ws_bytes(const brisk_corrector& c, int V) {
  return static_cast<size_t>(V) * (c.d_tproj + c.rank) * sizeof(float);
}

// The per-token tables: P_e E(v) and W_c E_out(v) for every token (the
// gathered projections with the identity as row map), then their lifts
// TZ = W_z[:, t] P_e E(v), TH = W_h[:, t] P_e E(v) and EH = W_s^T W_c E_out(v),
// each row zero-padded to the step-vector stride.
void launch_corrector_prepare(const brisk_corrector& c, const uint16_t* lm_head, const uint16_t* tok_embed,
                              int V, int d, float* tables, void* ws, hipStream_t s) {
  const int ds = c.d_state;
  const int d_in = c.d_hproj + c.d_tproj + c.d_pos + c.d_feat;
  const int tp_off = c.d_hproj;
  const size_t vsz = step_vec_stride(ds);
  float* PE = static_cast<float*>(ws);
  float* PC = PE + static_cast<size_t>(V) * c.d_tproj;
  ProjJobs pj{};
  pj.d = d;
  pj.splits = 1;
  pj.job[0] = ProjJob{tok_embed, nullptr, V, c.d_tproj, V, c.P_e, PE, static_cast<size_t>(V) * c.d_tproj};
  pj.job[2] = ProjJob{lm_head, nullptr, V, c.rank, V, c.W_c, PC, static_cast<size_t>(V) * c.rank};
  int gx = 0;
  for (int j = 0; j < kMaxProjJobs; ++j) gx = std::max(gx, proj_tiles(pj.job[j].n, pj.job[j].J, 128));
  hipLaunchKernelGGL(gather_proj_kernel<128>, dim3(gx, kMaxProjJobs + 1, 1), dim3(256), 0, s, pj);

  auto fterm = [&](const float* in, int C, const uint16_t* m, int m_rs, int m_cs) {
    const bool a16 = (reinterpret_cast<uintptr_t>(in) & 15u) == 0 && C % 16 == 0;
    const bool m16 = (reinterpret_cast<uintptr_t>(m) & 15u) == 0 &&
                     (m_cs == 1 ? m_rs % 8 == 0 && C % 16 == 0 : m_rs == 1 && m_cs % 8 == 0 && ds % 16 == 0);
    return LiftTerm{in, 0, C, 1, 0, C, m, m_rs, m_cs, a16 ? 1 : 0, m16 ? 1 : 0};
  };
  const LiftTerm none{nullptr, 0, 0, 0, 0, 0, nullptr, 0, 0, 0, 0};
  const size_t tstride = static_cast<size_t>(V) * vsz;
  LiftJobs lj{};
  lj.ds = ds;
  lj.job[0] = LiftJob{{fterm(PC, c.rank, c.W_s, 1, ds), none}, V, tables, 1, vsz, vsz};
  lj.job[1] = LiftJob{{fterm(PE, c.d_tproj, c.W_z + tp_off, d_in, 1), none}, V, tables + tstride, 1, vsz, vsz};
  lj.job[2] = LiftJob{{fterm(PE, c.d_tproj, c.W_h + tp_off, d_in, 1), none}, V, tables + 2 * tstride, 1, vsz, vsz};
  const dim3 grid((V + LT_BN - 1) / LT_BN, static_cast<int>((vsz + LT_BJ - 1) / LT_BJ), kMaxLiftJobs);
  hipLaunchKernelGGL(lift_kernel<1>, grid, dim3(256), 0, s, lj);
}

}  // namespace brisk
