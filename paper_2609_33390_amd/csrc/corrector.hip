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
// (kernels gather_proj, cross_dot and lift); the scan then carries only
// the selection-dependent chain: features, gate, state update, K dot products
// and an argmax per step, one wavefront per sequence.
#include "device_common.h"
#include "kernels.h"

namespace brisk {

namespace {

// ---------------------------------------------------------------------------
// gather_proj: out[n, j] = sum_k table[row(n), k] * wt[j, k]   (bf16 in, fp32 out)
// row(n) = idx[n] (clamped into [0, n_table)) or n when idx is null.
// MFMA: A = wt rows (M = j), B = gathered rows (N = n).
// ---------------------------------------------------------------------------
struct ProjJob {
  const uint16_t* table;
  const int32_t* idx;
  int n, J, n_table;
  const uint16_t* wt;
  float* out;  // [n, J]
};
constexpr int kMaxProjJobs = 6;
struct ProjJobs {
  ProjJob job[kMaxProjJobs];
  int d;
};

constexpr int PJ_BN = 64, PJ_BJ = 64, PJ_BK = 64, PJ_STRIDE = PJ_BK + 8;

__global__ __launch_bounds__(256) void gather_proj_kernel(ProjJobs jobs) {
  const ProjJob& jb = jobs.job[blockIdx.y];
  const int d = jobs.d;
  const int n_jt = (jb.J + PJ_BJ - 1) / PJ_BJ;
  const int n_nt = (jb.n + PJ_BN - 1) / PJ_BN;
  if (static_cast<int>(blockIdx.x) >= n_jt * n_nt) return;
  const int jt = blockIdx.x % n_jt, nt = blockIdx.x / n_jt;
  const int j0 = jt * PJ_BJ, n0 = nt * PJ_BN;

  __shared__ __align__(16) uint16_t sA[PJ_BJ * PJ_STRIDE];
  __shared__ __align__(16) uint16_t sB[PJ_BN * PJ_STRIDE];
  __shared__ int srow[PJ_BN];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wj = wave & 1, wn = wave >> 1;  // 2 x 2 waves, 32 x 32 each
  if (tid < PJ_BN) {
    const int n = n0 + tid;
    int r = -1;
    if (n < jb.n) r = jb.idx ? clamp_id(jb.idx[n], jb.n_table) : n;
    srow[tid] = r;
  }
  __syncthreads();

  floatx4 acc[2][2];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b) acc[a][b] = floatx4{0.f, 0.f, 0.f, 0.f};

  for (int k0 = 0; k0 < d; k0 += PJ_BK) {
    // 64 rows x 64 cols of each operand = 512 16-byte chunks each, 2 per thread.
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int c = tid + i * 256;
      const int row = c >> 3, col = (c & 7) * 8;
      const int k = k0 + col;
      uint4 va = make_uint4(0, 0, 0, 0), vb = make_uint4(0, 0, 0, 0);
      const int j = j0 + row;
      if (j < jb.J && k < d) va = *reinterpret_cast<const uint4*>(jb.wt + static_cast<size_t>(j) * d + k);
      const int r = srow[row];
      if (r >= 0 && k < d) vb = *reinterpret_cast<const uint4*>(jb.table + static_cast<size_t>(r) * d + k);
      *reinterpret_cast<uint4*>(sA + row * PJ_STRIDE + col) = va;
      *reinterpret_cast<uint4*>(sB + row * PJ_STRIDE + col) = vb;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < PJ_BK; kk += 32) {
      const int koff = kk + (lane >> 4) * 8;
      bf16x8 a[2], b[2];
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        a[t] = *reinterpret_cast<const bf16x8*>(sA + (wj * 32 + t * 16 + (lane & 15)) * PJ_STRIDE + koff);
        b[t] = *reinterpret_cast<const bf16x8*>(sB + (wn * 32 + t * 16 + (lane & 15)) * PJ_STRIDE + koff);
      }
#pragma unroll
      for (int x = 0; x < 2; ++x)
#pragma unroll
        for (int y = 0; y < 2; ++y)
          acc[x][y] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[x], b[y], acc[x][y], 0, 0, 0);
    }
    __syncthreads();
  }
#pragma unroll
  for (int x = 0; x < 2; ++x)
#pragma unroll
    for (int y = 0; y < 2; ++y) {
      const int n = n0 + wn * 32 + y * 16 + (lane & 15);
      const int jb0 = j0 + wj * 32 + x * 16 + (lane >> 4) * 4;
      if (n < jb.n) {
#pragma unroll
        for (int q = 0; q < 4; ++q)
          if (jb0 + q < jb.J) jb.out[static_cast<size_t>(n) * jb.J + jb0 + q] = acc[x][y][q];
      }
    }
}

// ---------------------------------------------------------------------------
// cross_dot: the full-vocabulary logit of every possible previous token at the
// next position.  n < NC: candidate k of row r against hidden row r+1 (0 on
// the last row of a block); n >= NC: anchor token x_0 against the block's
// first row.  One wavefront per dot product.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void cross_dot_kernel(const uint16_t* __restrict__ W,
                                                        const uint16_t* __restrict__ H,
                                                        const int32_t* __restrict__ cand_id,
                                                        const int32_t* __restrict__ anchor, int B,
                                                        int L, int K, int d, int V,
                                                        float* __restrict__ X) {
  const int lane = threadIdx.x & 63;
  const int n = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int NC = B * L * K;
  if (n >= NC + B) return;
  int v, hrow;
  if (n < NC) {
    const int r = n / K;
    if (r % L == L - 1) {
      if (lane == 0) X[n] = 0.f;
      return;
    }
    v = clamp_id(cand_id[n], V);
    hrow = r + 1;
  } else {
    const int b = n - NC;
    v = clamp_id(anchor[b], V);
    hrow = b * L;
  }
  const uint16_t* w = W + static_cast<size_t>(v) * d;
  const uint16_t* h = H + static_cast<size_t>(hrow) * d;
  float s = 0.f;
  for (int k = lane * 8; k < d; k += 64 * 8) {
    const uint4 a = *reinterpret_cast<const uint4*>(w + k);
    const uint4 c = *reinterpret_cast<const uint4*>(h + k);
    s += bf16_lo(a.x) * bf16_lo(c.x) + bf16_hi(a.x) * bf16_hi(c.x);
    s += bf16_lo(a.y) * bf16_lo(c.y) + bf16_hi(a.y) * bf16_hi(c.y);
    s += bf16_lo(a.z) * bf16_lo(c.z) + bf16_hi(a.z) * bf16_hi(c.z);
    s += bf16_lo(a.w) * bf16_lo(c.w) + bf16_hi(a.w) * bf16_hi(c.w);
  }
  s = wave_sum(s);
  if (lane == 0) X[n] = s;
}

// ---------------------------------------------------------------------------
// lift: out[n, j] = sum_c M(j, c) in[n, c] (+ sum_c M2(j, c) pos[n mod L, c])
// for j < ds, with M(j, c) = m[j * m_rs + c * m_cs] (bf16) and fp32 inputs.
// ---------------------------------------------------------------------------
struct LiftJob {
  const float* in;
  int n, C;
  const uint16_t* m;
  int m_rs, m_cs;
  const uint16_t* m2;   // nullable: position term
  const uint16_t* pos;  // [max_L, C2]
  int C2, L;
  float* out;           // [n, ds]
};
constexpr int kMaxLiftJobs = 5;
struct LiftJobs {
  LiftJob job[kMaxLiftJobs];
  int ds, m2_rs;
};
constexpr int LT_N = 16;
constexpr int LT_MAXC = 256;

__global__ __launch_bounds__(256) void lift_kernel(LiftJobs jobs) {
  const LiftJob& jb = jobs.job[blockIdx.y];
  const int n0 = blockIdx.x * LT_N;
  if (n0 >= jb.n) return;
  __shared__ float s_in[LT_N * LT_MAXC];
  const int tid = threadIdx.x;
  for (int e = tid; e < LT_N * jb.C; e += 256) {
    const int n = n0 + e / jb.C;
    s_in[e] = n < jb.n ? jb.in[static_cast<size_t>(n) * jb.C + e % jb.C] : 0.f;
  }
  __syncthreads();
  for (int j = tid; j < jobs.ds; j += 256) {
    float acc[LT_N];
#pragma unroll
    for (int q = 0; q < LT_N; ++q) acc[q] = 0.f;
    for (int c = 0; c < jb.C; ++c) {
      const float mv = bf16_to_f32(jb.m[static_cast<size_t>(j) * jb.m_rs + static_cast<size_t>(c) * jb.m_cs]);
#pragma unroll
      for (int q = 0; q < LT_N; ++q) acc[q] += mv * s_in[q * jb.C + c];
    }
    if (jb.m2) {
      for (int c = 0; c < jb.C2; ++c) {
        const float mv = bf16_to_f32(jb.m2[static_cast<size_t>(j) * jobs.m2_rs + c]);
#pragma unroll
        for (int q = 0; q < LT_N; ++q) {
          const int n = n0 + q;
          acc[q] += mv * bf16_to_f32(jb.pos[(n % jb.L) * jb.C2 + c]);
        }
      }
    }
#pragma unroll
    for (int q = 0; q < LT_N; ++q) {
      const int n = n0 + q;
      if (n < jb.n) jb.out[static_cast<size_t>(n) * jobs.ds + j] = acc[q];
    }
  }
}

// ---------------------------------------------------------------------------
// scan: one wavefront per sequence, the L dependent steps in order.
// Lane `lane` owns state elements e = lane + 64 j, j < PL.
// ---------------------------------------------------------------------------
struct ScanArgs {
  int B, L, K, ds, d_in, feat_off, df;
  const float* U0;   // [2, B, ds]  A_h h_c, A_e E(x_0)
  const float* X;    // [NC + B]
  const float* TZ;   // [NC + B, ds]
  const float* TH;
  const float* EH;   // [NC, ds]
  const float* AZ;   // [rows, ds]
  const float* AH;
  const uint16_t* W_z;
  const uint16_t* W_h;
  const uint16_t* P_phi;
  const uint16_t* w_g;
  float alpha, b_g;
  const float* cand_logit;
  const int32_t* cand_id;
  const int32_t* anchor;
  int32_t* selected;
  float* refined;
  float* gamma;
  float* resid;
};

template <int PL>
__global__ __launch_bounds__(256) void scan_kernel(ScanArgs a) {
  const int lane = threadIdx.x & 63;
  const int b = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (b >= a.B) return;
  const int ds = a.ds, K = a.K, L = a.L;
  const int NC = a.B * L * K;

  float u[PL], wgu[PL], fz[PL][5], fh[PL][5];
#pragma unroll
  for (int j = 0; j < PL; ++j) {
    const int e = lane + 64 * j;
    const bool ok = e < ds;
    u[j] = ok ? tanhf(a.U0[static_cast<size_t>(b) * ds + e] + a.U0[static_cast<size_t>(a.B + b) * ds + e]) : 0.f;
    wgu[j] = ok ? bf16_to_f32(a.w_g[e]) : 0.f;
#pragma unroll
    for (int f = 0; f < 5; ++f) {
      float sz = 0.f, sh = 0.f;
      if (ok) {
        for (int q = 0; q < a.df; ++q) {
          const float p = bf16_to_f32(a.P_phi[q * 5 + f]);
          sz += bf16_to_f32(a.W_z[static_cast<size_t>(e) * a.d_in + a.feat_off + q]) * p;
          sh += bf16_to_f32(a.W_h[static_cast<size_t>(e) * a.d_in + a.feat_off + q]) * p;
        }
      }
      fz[j][f] = sz;
      fh[j][f] = sh;
    }
  }
  float wgphi[5];
#pragma unroll
  for (int f = 0; f < 5; ++f) wgphi[f] = bf16_to_f32(a.w_g[ds + f]);
  const float sig_alpha = sigmoidf_(a.alpha);

  int prev_n = NC + b;
  int prev_tok = a.anchor[b];
  for (int i = 0; i < L; ++i) {
    const int r = b * L + i;
    const float cl = lane < K ? a.cand_logit[static_cast<size_t>(r) * K + lane] : 0.f;
    const int ci = lane < K ? a.cand_id[static_cast<size_t>(r) * K + lane] : -1;
    const float c0 = __shfl(cl, 0), c1 = __shfl(cl, 1), c3 = __shfl(cl, 3);
    const int id0 = __shfl(ci, 0);
    const bool in4 = __ballot(lane < 4 && ci == prev_tok) != 0;
    float phi[5];
    phi[0] = c0 - c1;
    phi[1] = c0 - c3;
    phi[2] = prev_tok == id0 ? 1.f : 0.f;
    phi[3] = in4 ? 1.f : 0.f;
    phi[4] = c0 - a.X[prev_n];

    float gs = 0.f;
#pragma unroll
    for (int j = 0; j < PL; ++j) {
      const int e = lane + 64 * j;
      if (e < ds) {
        float gz = a.AZ[static_cast<size_t>(r) * ds + e] + a.TZ[static_cast<size_t>(prev_n) * ds + e];
        float gh = a.AH[static_cast<size_t>(r) * ds + e] + a.TH[static_cast<size_t>(prev_n) * ds + e];
#pragma unroll
        for (int f = 0; f < 5; ++f) {
          gz += fz[j][f] * phi[f];
          gh += fh[j][f] * phi[f];
        }
        const float z = sigmoidf_(gz);
        u[j] = (1.f - z) * u[j] + z * gh;
        gs += u[j] * wgu[j];
      }
    }
    float s = wave_sum(gs) + a.b_g;
#pragma unroll
    for (int f = 0; f < 5; ++f) s += wgphi[f] * phi[f];
    const float g = sig_alpha * sigmoidf_(s);

    float my_d = 0.f;
    for (int k = 0; k < K; ++k) {
      const float* eh = a.EH + (static_cast<size_t>(r) * K + k) * ds;
      float p = 0.f;
#pragma unroll
      for (int j = 0; j < PL; ++j) {
        const int e = lane + 64 * j;
        if (e < ds) p += u[j] * eh[e];
      }
      p = wave_sum(p);
      if (lane == k) my_d = p;
    }
    const float lt = cl + g * my_d;
    const uint64_t key = lane < K ? make_key(lt, static_cast<uint32_t>(lane)) : 0ull;
    const int kstar = key_id(wave_max_u64(key));
    const int sel = __shfl(ci, kstar);
    if (lane < K) {
      if (a.refined) a.refined[static_cast<size_t>(r) * K + lane] = lt;
      if (a.resid) a.resid[static_cast<size_t>(r) * K + lane] = my_d;
    }
    if (lane == 0) {
      a.selected[r] = sel;
      if (a.gamma) a.gamma[r] = g;
    }
    prev_n = r * K + kstar;
    prev_tok = sel;
  }
}

struct Layout {
  size_t PE, PC, PH, U0, X, TZ, TH, EH, AZ, AH, total;
};

Layout rerank_layout(const brisk_corrector& c, int B, int L, int K) {
  const size_t rows = static_cast<size_t>(B) * L, NC = rows * K, NP = NC + B;
  const size_t ds = c.d_state;
  Layout l{};
  size_t off = 0;
  auto take = [&](size_t floats) {
    const size_t o = off;
    off += (floats * sizeof(float) + 255) / 256 * 256;
    return o;
  };
  l.PE = take(NP * c.d_tproj);
  l.PC = take(NC * c.rank);
  l.PH = take(rows * c.d_hproj);
  l.U0 = take(2 * static_cast<size_t>(B) * ds);
  l.X = take(NP);
  l.TZ = take(NP * ds);
  l.TH = take(NP * ds);
  l.EH = take(NC * ds);
  l.AZ = take(rows * ds);
  l.AH = take(rows * ds);
  l.total = off;
  return l;
}

}  // namespace

size_t rerank_workspace_bytes(const brisk_corrector& c, int B, int L, int K) {
  return rerank_layout(c, B, L, K).total;
}

void launch_rerank(const brisk_corrector& c, const uint16_t* hidden, const uint16_t* ctx_hidden,
                   const int32_t* anchor_tok, const uint16_t* lm_head, const uint16_t* tok_embed,
                   const float* cand_logit, const int32_t* cand_id, int B, int L, int K, int d,
                   int V, int32_t* selected, float* refined, float* gamma, float* resid, void* ws,
                   hipStream_t s) {
  const Layout lay = rerank_layout(c, B, L, K);
  char* base = static_cast<char*>(ws);
  auto F = [&](size_t off) { return reinterpret_cast<float*>(base + off); };
  const int rows = B * L, NC = rows * K, NP = NC + B;
  const int ds = c.d_state;
  const int d_in = c.d_hproj + c.d_tproj + c.d_pos + c.d_feat;
  const int tp_off = c.d_hproj, pos_off = c.d_hproj + c.d_tproj, feat_off = pos_off + c.d_pos;

  ProjJobs pj{};
  pj.d = d;
  pj.job[0] = ProjJob{tok_embed, cand_id, NC, c.d_tproj, V, c.P_e, F(lay.PE)};
  pj.job[1] = ProjJob{tok_embed, anchor_tok, B, c.d_tproj, V, c.P_e, F(lay.PE) + static_cast<size_t>(NC) * c.d_tproj};
  pj.job[2] = ProjJob{lm_head, cand_id, NC, c.rank, V, c.W_c, F(lay.PC)};
  pj.job[3] = ProjJob{hidden, nullptr, rows, c.d_hproj, rows, c.P_h, F(lay.PH)};
  pj.job[4] = ProjJob{ctx_hidden, nullptr, B, ds, B, c.A_h, F(lay.U0)};
  pj.job[5] = ProjJob{tok_embed, anchor_tok, B, ds, V, c.A_e, F(lay.U0) + static_cast<size_t>(B) * ds};
  int max_tiles = 0;
  for (int j = 0; j < kMaxProjJobs; ++j) {
    const int t = ((pj.job[j].J + PJ_BJ - 1) / PJ_BJ) * ((pj.job[j].n + PJ_BN - 1) / PJ_BN);
    max_tiles = t > max_tiles ? t : max_tiles;
  }
  hipLaunchKernelGGL(gather_proj_kernel, dim3(max_tiles, kMaxProjJobs), dim3(256), 0, s, pj);

  hipLaunchKernelGGL(cross_dot_kernel, dim3((NP + 3) / 4), dim3(256), 0, s, lm_head, hidden, cand_id,
                     anchor_tok, B, L, K, d, V, F(lay.X));

  LiftJobs lj{};
  lj.ds = ds;
  lj.m2_rs = d_in;
  lj.job[0] = LiftJob{F(lay.PE), NP, c.d_tproj, c.W_z + tp_off, d_in, 1, nullptr, nullptr, 0, L, F(lay.TZ)};
  lj.job[1] = LiftJob{F(lay.PE), NP, c.d_tproj, c.W_h + tp_off, d_in, 1, nullptr, nullptr, 0, L, F(lay.TH)};
  lj.job[2] = LiftJob{F(lay.PC), NC, c.rank, c.W_s, 1, ds, nullptr, nullptr, 0, L, F(lay.EH)};
  lj.job[3] = LiftJob{F(lay.PH), rows, c.d_hproj, c.W_z, d_in, 1, c.W_z + pos_off, c.pos_emb, c.d_pos, L, F(lay.AZ)};
  lj.job[4] = LiftJob{F(lay.PH), rows, c.d_hproj, c.W_h, d_in, 1, c.W_h + pos_off, c.pos_emb, c.d_pos, L, F(lay.AH)};
  hipLaunchKernelGGL(lift_kernel, dim3((NP + LT_N - 1) / LT_N, kMaxLiftJobs), dim3(256), 0, s, lj);

  ScanArgs sa{};
  sa.B = B; sa.L = L; sa.K = K; sa.ds = ds; sa.d_in = d_in; sa.feat_off = feat_off; sa.df = c.d_feat;
  sa.U0 = F(lay.U0); sa.X = F(lay.X); sa.TZ = F(lay.TZ); sa.TH = F(lay.TH); sa.EH = F(lay.EH);
  sa.AZ = F(lay.AZ); sa.AH = F(lay.AH);
  sa.W_z = c.W_z; sa.W_h = c.W_h; sa.P_phi = c.P_phi; sa.w_g = c.w_g;
  sa.alpha = c.alpha; sa.b_g = c.b_g;
  sa.cand_logit = cand_logit; sa.cand_id = cand_id; sa.anchor = anchor_tok;
  sa.selected = selected; sa.refined = refined; sa.gamma = gamma; sa.resid = resid;
  const dim3 grid((B + 3) / 4), block(256);
  if (ds <= 64) hipLaunchKernelGGL(scan_kernel<1>, grid, block, 0, s, sa);
  else if (ds <= 128) hipLaunchKernelGGL(scan_kernel<2>, grid, block, 0, s, sa);
  else if (ds <= 256) hipLaunchKernelGGL(scan_kernel<4>, grid, block, 0, s, sa);
  else hipLaunchKernelGGL(scan_kernel<8>, grid, block, 0, s, sa);
}

}  // namespace brisk
