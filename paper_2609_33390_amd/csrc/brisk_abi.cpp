// C ABI of the decoding hot path: argument validation, workspace sizing and
// kernel launches.  Every check runs on the host before the first HIP call, so
// an error return has launched nothing and touched no output.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "brisk.h"
#include "kernels.h"

namespace {

constexpr int kAbiVersion = 10;
constexpr int32_t kMaxRows = 1 << 20;
constexpr int32_t kMaxD = 65536;
constexpr int32_t kMaxTableV = 1 << 24;

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
bool aligned4(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 3u) == 0; }
bool aligned2(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 1u) == 0; }
bool aligned8(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 7u) == 0; }

constexpr int32_t kMaxProfileM = 1024;
constexpr int32_t kMaxProfileBlocks = 1 << 30;

// hidden [rows, d] x lm_head [V, d]: shapes, alignment and the 32-bit byte
// offsets the LM-head kernel addresses both matrices with
int lmhead_check(const uint16_t* hidden, const uint16_t* lm_head, int32_t rows, int32_t d, int32_t V,
                 int32_t K) {
  if (!hidden || !lm_head) return BRISK_ERR_NULL;
  if (rows < 1 || rows > kMaxRows || d < 8 || d > kMaxD || K < 1 || K > 64 || V < K)
    return BRISK_ERR_SHAPE;
  if (d % 8 != 0 || !aligned16(hidden) || !aligned16(lm_head)) return BRISK_ERR_UNSUPPORTED;
  if (static_cast<uint64_t>(V) * d * 2 >= (uint64_t{1} << 32) ||
      static_cast<uint64_t>(rows) * d * 2 >= (uint64_t{1} << 32))
    return BRISK_ERR_UNSUPPORTED;
  return BRISK_OK;
}

int propose_check(const uint16_t* hidden, const uint16_t* lm_head, int32_t rows, int32_t d,
                  int32_t V, int32_t K, const float* cand_logit, const int32_t* cand_id) {
  if (!hidden || !lm_head || !cand_logit || !cand_id) return BRISK_ERR_NULL;
  const int st = lmhead_check(hidden, lm_head, rows, d, V, K);
  if (st != BRISK_OK) return st;
  if (!aligned4(cand_logit) || !aligned4(cand_id)) return BRISK_ERR_UNSUPPORTED;
  return BRISK_OK;
}

int corrector_check(const brisk_corrector* c) {
  if (!c) return BRISK_ERR_NULL;
  if (!c->A_h || !c->A_e || !c->P_h || !c->P_e || !c->pos_emb || !c->P_phi || !c->W_z ||
      !c->W_h || !c->W_s || !c->W_c || !c->w_g)
    return BRISK_ERR_NULL;
  if (c->d_state < 1 || c->d_state > 512 || c->d_hproj < 1 || c->d_hproj > 256 ||
      c->d_tproj < 1 || c->d_tproj > 256 || c->rank < 1 || c->rank > 256 || c->d_pos < 1 ||
      c->d_pos > 64 || c->d_feat < 1 || c->d_feat > 64 || c->max_L < 1)
    return BRISK_ERR_SHAPE;
  if (!aligned16(c->A_h) || !aligned16(c->A_e) || !aligned16(c->P_h) || !aligned16(c->P_e) ||
      !aligned16(c->W_c) || !aligned2(c->pos_emb) || !aligned2(c->P_phi) || !aligned2(c->W_z) ||
      !aligned2(c->W_h) || !aligned2(c->W_s) || !aligned2(c->w_g))
    return BRISK_ERR_UNSUPPORTED;
  return BRISK_OK;
}

int rerank_shape_check(const brisk_corrector* c, int32_t B, int32_t L, int32_t K) {
  if (B < 1 || L < 1 || L > c->max_L || K < 4 || K > 64) return BRISK_ERR_SHAPE;
  if (static_cast<int64_t>(B) * L > kMaxRows) return BRISK_ERR_SHAPE;
  return BRISK_OK;
}

int launch_status() {
  return hipGetLastError() == hipSuccess ? BRISK_OK : BRISK_ERR_HIP;
}

}  // namespace

extern "C" {

const char* brisk_status_str(int status) {
  switch (status) {
    case BRISK_OK: return "ok";
    case BRISK_ERR_NULL: return "a required pointer is NULL";
    case BRISK_ERR_SHAPE: return "a size is out of range or inconsistent";
    case BRISK_ERR_UNSUPPORTED: return "unsupported alignment or divisibility (16-byte pointers, d % 8 == 0)";
    case BRISK_ERR_WORKSPACE: return "workspace missing or too small";
    case BRISK_ERR_HIP: return "a HIP launch failed";
    case BRISK_ERR_SCRATCH: return "the shape needs more scratch than the fixed no-alloc buffer holds";
    default: return "unknown status";
  }
}

int brisk_abi_version(void) { return kAbiVersion; }

int brisk_propose_workspace_size(int32_t rows, int32_t d, int32_t V, int32_t K, size_t* bytes) {
  if (!bytes) return BRISK_ERR_NULL;
  if (rows < 1 || rows > kMaxRows || d < 8 || d > kMaxD || K < 1 || K > 64 || V < K)
    return BRISK_ERR_SHAPE;
  *bytes = brisk::propose_workspace_bytes(rows, V, K);
  return BRISK_OK;
}

int brisk_propose_block(const uint16_t* hidden, const uint16_t* lm_head, int32_t rows, int32_t d,
                        int32_t V, int32_t K, float* cand_logit, int32_t* cand_id, void* ws,
                        size_t ws_bytes, void* stream) {
  const int st = propose_check(hidden, lm_head, rows, d, V, K, cand_logit, cand_id);
  if (st != BRISK_OK) return st;
  const size_t need = brisk::propose_workspace_bytes(rows, V, K);
  if (ws_bytes < need || (need > 0 && !ws)) return BRISK_ERR_WORKSPACE;
  if (!aligned16(ws)) return BRISK_ERR_UNSUPPORTED;
  brisk::launch_propose(hidden, lm_head, rows, d, V, K, rows, cand_logit, cand_id, nullptr, ws,
                        static_cast<hipStream_t>(stream));
  return launch_status();
}

int brisk_propose_block_noalloc(const uint16_t* hidden, const uint16_t* lm_head, int32_t rows, int32_t d,
                                int32_t V, int32_t K, float* cand_logit, int32_t* cand_id, void* stream) {
  const int st = propose_check(hidden, lm_head, rows, d, V, K, cand_logit, cand_id);
  if (st != BRISK_OK) return st;
  if (brisk::propose_workspace_bytes(rows, V, K) > brisk::noalloc_scratch_bytes()) return BRISK_ERR_SCRATCH;
  if (brisk::launch_propose_noalloc(hidden, lm_head, rows, d, V, K, cand_logit, cand_id,
                                    static_cast<hipStream_t>(stream)) != 0)
    return BRISK_ERR_HIP;
  return launch_status();
}

int brisk_propose_lmhead(const uint16_t* hidden, const uint16_t* lm_head, int32_t rows, int32_t d,
                         int32_t V, int32_t K, void* ws, size_t ws_bytes, void* stream) {
  const int st = lmhead_check(hidden, lm_head, rows, d, V, K);
  if (st != BRISK_OK) return st;
  const size_t need = brisk::propose_workspace_bytes(rows, V, K);
  if (ws_bytes < need || (need > 0 && !ws)) return BRISK_ERR_WORKSPACE;
  if (!aligned16(ws)) return BRISK_ERR_UNSUPPORTED;
  brisk::launch_propose_pass(hidden, lm_head, rows, d, V, K, ws, static_cast<hipStream_t>(stream));
  return launch_status();
}

int brisk_propose_merge(int32_t rows, int32_t V, int32_t K, float* cand_logit, int32_t* cand_id,
                        const void* ws, size_t ws_bytes, void* stream) {
  if (!cand_logit || !cand_id) return BRISK_ERR_NULL;
  if (rows < 1 || rows > kMaxRows || K < 1 || K > 64 || V < K) return BRISK_ERR_SHAPE;
  if (!aligned4(cand_logit) || !aligned4(cand_id)) return BRISK_ERR_UNSUPPORTED;
  const size_t need = brisk::propose_workspace_bytes(rows, V, K);
  if (ws_bytes < need || (need > 0 && !ws)) return BRISK_ERR_WORKSPACE;
  if (!aligned16(ws)) return BRISK_ERR_UNSUPPORTED;
  brisk::launch_propose_merge(rows, V, K, rows, cand_logit, cand_id, nullptr, ws,
                              static_cast<hipStream_t>(stream));
  return launch_status();
}

int brisk_propose_verify_workspace_size(int32_t rows_prop, int32_t rows_ver, int32_t d, int32_t V,
                                        int32_t K, size_t* bytes) {
  if (!bytes) return BRISK_ERR_NULL;
  const int64_t rows = static_cast<int64_t>(rows_prop) + rows_ver;
  if (rows_prop < 0 || rows_ver < 0 || rows < 1 || rows > kMaxRows || d < 8 || d > kMaxD || K < 1 ||
      K > 64 || V < K)
    return BRISK_ERR_SHAPE;
  *bytes = brisk::propose_workspace_bytes(static_cast<int>(rows), V, K);
  return BRISK_OK;
}

int brisk_propose_verify(const uint16_t* hidden, const uint16_t* lm_head, int32_t rows_prop,
                         int32_t rows_ver, int32_t d, int32_t V, int32_t K, float* cand_logit,
                         int32_t* cand_id, int32_t* ver_token, void* ws, size_t ws_bytes,
                         void* stream) {
  if (!hidden || !lm_head || (rows_prop > 0 && (!cand_logit || !cand_id)) || (rows_ver > 0 && !ver_token))
    return BRISK_ERR_NULL;
  const int64_t rows64 = static_cast<int64_t>(rows_prop) + rows_ver;
  if (rows_prop < 0 || rows_ver < 0 || rows64 < 1 || rows64 > kMaxRows) return BRISK_ERR_SHAPE;
  const int32_t rows = static_cast<int32_t>(rows64);
  const int st = lmhead_check(hidden, lm_head, rows, d, V, K);
  if (st != BRISK_OK) return st;
  if (!aligned4(cand_logit) || !aligned4(cand_id) || !aligned4(ver_token)) return BRISK_ERR_UNSUPPORTED;
  const size_t need = brisk::propose_workspace_bytes(rows, V, K);
  if (ws_bytes < need || !ws) return BRISK_ERR_WORKSPACE;
  if (!aligned16(ws)) return BRISK_ERR_UNSUPPORTED;
  brisk::launch_propose(hidden, lm_head, rows, d, V, K, rows_prop, cand_logit, cand_id, ver_token, ws,
                        static_cast<hipStream_t>(stream));
  return launch_status();
}

int brisk_rerank_workspace_size(const brisk_corrector* c, int32_t B, int32_t L, int32_t K,
                                size_t* bytes) {
  if (!bytes || !c) return BRISK_ERR_NULL;
  if (c->d_state < 1 || c->d_state > 512 || c->d_hproj < 1 || c->d_hproj > 256 ||
      c->d_tproj < 1 || c->d_tproj > 256 || c->rank < 1 || c->rank > 256)
    return BRISK_ERR_SHAPE;
  if (B < 1 || L < 1 || K < 4 || K > 64 || static_cast<int64_t>(B) * L > kMaxRows)
    return BRISK_ERR_SHAPE;
  *bytes = brisk::rerank_workspace_bytes(*c, B, L, K);
  return BRISK_OK;
}

namespace {

int rerank_impl(brisk::RerankPart part, const brisk_corrector* c, const uint16_t* hidden,
                const uint16_t* ctx_hidden, const int32_t* anchor_tok, const uint16_t* lm_head,
                const uint16_t* tok_embed, const float* cand_logit, const int32_t* cand_id,
                const int32_t* verifier, int32_t B, int32_t L, int32_t K, int32_t d, int32_t V,
                int32_t* selected, float* refined, float* gamma, float* resid, int32_t* accept_len,
                int32_t* correction, void* ws, size_t ws_bytes, void* stream) {
  int st = corrector_check(c);
  if (st != BRISK_OK) return st;
  if (!hidden || !ctx_hidden || !anchor_tok || !tok_embed) return BRISK_ERR_NULL;
  // the hoisted part reads no LM head, candidates or outputs
  if (part != brisk::RerankPart::kHoist && (!lm_head || !cand_logit || !cand_id || !selected))
    return BRISK_ERR_NULL;
  st = rerank_shape_check(c, B, L, K);
  if (st != BRISK_OK) return st;
  if (d < 8 || d > kMaxD || V < K) return BRISK_ERR_SHAPE;
  // the scan addresses one sequence's step vectors with 32-bit byte offsets;
  // each vector is padded to at least 256 floats
  const uint64_t vec = c->d_state <= 256 ? 256 : static_cast<uint64_t>(c->d_state);
  if (static_cast<uint64_t>(L) * (2 + 3 * static_cast<uint64_t>(K)) * vec * 4 >= (uint64_t{1} << 31))
    return BRISK_ERR_UNSUPPORTED;
  if (d % 8 != 0 || !aligned16(hidden) || !aligned16(ctx_hidden) || !aligned16(lm_head) ||
      !aligned16(tok_embed) || !aligned4(anchor_tok) || !aligned4(cand_logit) ||
      !aligned4(cand_id) || !aligned4(selected) || !aligned4(refined) || !aligned4(gamma) ||
      !aligned4(resid))
    return BRISK_ERR_UNSUPPORTED;
  if (c->tables && (c->tables_V != V)) return BRISK_ERR_SHAPE;
  // the scan addresses the tables with 32-bit byte offsets
  if (c->tables && 3 * static_cast<uint64_t>(V) * vec * 4 >= (uint64_t{1} << 31)) return BRISK_ERR_UNSUPPORTED;
  if (!aligned16(c->tables)) return BRISK_ERR_UNSUPPORTED;
  const size_t need = brisk::rerank_workspace_bytes(*c, B, L, K);
  if (ws_bytes < need || !ws) return BRISK_ERR_WORKSPACE;
  if (!aligned16(ws)) return BRISK_ERR_UNSUPPORTED;
  brisk::launch_rerank(*c, hidden, ctx_hidden, anchor_tok, lm_head, tok_embed, cand_logit, cand_id,
                       B, L, K, d, V, selected, refined, gamma, resid, verifier, accept_len,
                       correction, ws, static_cast<hipStream_t>(stream), part);
  return launch_status();
}

}  // namespace

int brisk_rerank(const brisk_corrector* c, const uint16_t* hidden, const uint16_t* ctx_hidden,
                 const int32_t* anchor_tok, const uint16_t* lm_head, const uint16_t* tok_embed,
                 const float* cand_logit, const int32_t* cand_id, int32_t B, int32_t L, int32_t K,
                 int32_t d, int32_t V, int32_t* selected, float* refined, float* gamma,
                 float* resid, void* ws, size_t ws_bytes, void* stream) {
  return rerank_impl(brisk::RerankPart::kAll, c, hidden, ctx_hidden, anchor_tok, lm_head, tok_embed,
                     cand_logit, cand_id, nullptr, B, L, K, d, V, selected, refined, gamma, resid,
                     nullptr, nullptr, ws, ws_bytes, stream);
}

int brisk_rerank_verify(const brisk_corrector* c, const uint16_t* hidden, const uint16_t* ctx_hidden,
                        const int32_t* anchor_tok, const uint16_t* lm_head, const uint16_t* tok_embed,
                        const float* cand_logit, const int32_t* cand_id, const int32_t* verifier,
                        int32_t B, int32_t L, int32_t K, int32_t d, int32_t V, int32_t* selected,
                        float* refined, float* gamma, float* resid, int32_t* accept_len,
                        int32_t* correction, void* ws, size_t ws_bytes, void* stream) {
  if (!verifier || !accept_len) return BRISK_ERR_NULL;
  if (!aligned4(verifier) || !aligned4(accept_len) || !aligned4(correction)) return BRISK_ERR_UNSUPPORTED;
  return rerank_impl(brisk::RerankPart::kAll, c, hidden, ctx_hidden, anchor_tok, lm_head, tok_embed,
                     cand_logit, cand_id, verifier, B, L, K, d, V, selected, refined, gamma, resid,
                     accept_len, correction, ws, ws_bytes, stream);
}

int brisk_rerank_hoist(const brisk_corrector* c, const uint16_t* hidden, const uint16_t* ctx_hidden,
                       const int32_t* anchor_tok, const uint16_t* tok_embed, int32_t B, int32_t L,
                       int32_t K, int32_t d, int32_t V, void* ws, size_t ws_bytes, void* stream) {
  return rerank_impl(brisk::RerankPart::kHoist, c, hidden, ctx_hidden, anchor_tok, nullptr, tok_embed,
                     nullptr, nullptr, nullptr, B, L, K, d, V, nullptr, nullptr, nullptr, nullptr,
                     nullptr, nullptr, ws, ws_bytes, stream);
}

int brisk_rerank_finish(const brisk_corrector* c, const uint16_t* hidden, const uint16_t* ctx_hidden,
                        const int32_t* anchor_tok, const uint16_t* lm_head, const uint16_t* tok_embed,
                        const float* cand_logit, const int32_t* cand_id, const int32_t* verifier,
                        int32_t B, int32_t L, int32_t K, int32_t d, int32_t V, int32_t* selected,
                        float* refined, float* gamma, float* resid, int32_t* accept_len,
                        int32_t* correction, void* ws, size_t ws_bytes, void* stream) {
  if (verifier && !accept_len) return BRISK_ERR_NULL;
  if (!aligned4(verifier) || !aligned4(accept_len) || !aligned4(correction)) return BRISK_ERR_UNSUPPORTED;
  return rerank_impl(brisk::RerankPart::kFinish, c, hidden, ctx_hidden, anchor_tok, lm_head, tok_embed,
                     cand_logit, cand_id, verifier, B, L, K, d, V, selected, refined, gamma, resid,
                     verifier ? accept_len : nullptr, verifier ? correction : nullptr, ws, ws_bytes,
                     stream);
}

int brisk_corrector_tables_size(const brisk_corrector* c, int32_t V, size_t* table_bytes, size_t* ws_bytes) {
  if (!table_bytes || !ws_bytes) return BRISK_ERR_NULL;
  const int st = corrector_check(c);
  if (st != BRISK_OK) return st;
  if (V < 1 || V > kMaxTableV) return BRISK_ERR_SHAPE;
  *table_bytes = brisk::corrector_tables_bytes(*c, V);
  *ws_bytes = brisk::corrector_prepare_ws_bytes(*c, V);
  return BRISK_OK;
}

int brisk_corrector_prepare(const brisk_corrector* c, const uint16_t* lm_head, const uint16_t* tok_embed,
                            int32_t V, int32_t d, float* tables, size_t table_bytes, void* ws,
                            size_t ws_bytes, void* stream) {
  int st = corrector_check(c);
  if (st != BRISK_OK) return st;
  if (!lm_head || !tok_embed || !tables) return BRISK_ERR_NULL;
  if (V < 1 || V > kMaxTableV || d < 8 || d > kMaxD) return BRISK_ERR_SHAPE;
  if (d % 8 != 0 || !aligned16(lm_head) || !aligned16(tok_embed) || !aligned16(tables)) return BRISK_ERR_UNSUPPORTED;
  if (table_bytes < brisk::corrector_tables_bytes(*c, V)) return BRISK_ERR_WORKSPACE;
  if (ws_bytes < brisk::corrector_prepare_ws_bytes(*c, V) || !ws) return BRISK_ERR_WORKSPACE;
  if (!aligned16(ws)) return BRISK_ERR_UNSUPPORTED;
  brisk::launch_corrector_prepare(*c, lm_head, tok_embed, V, d, tables, ws, static_cast<hipStream_t>(stream));
  return launch_status();
}

int brisk_verify_accept(const int32_t* proposal, const int32_t* verifier, int32_t B, int32_t L,
                        int32_t* accept_len, int32_t* correction, void* stream) {
  if (!proposal || !verifier || !accept_len) return BRISK_ERR_NULL;
  if (B < 1 || L < 1 || static_cast<int64_t>(B) * L > (int64_t{1} << 30)) return BRISK_ERR_SHAPE;
  if (!aligned4(proposal) || !aligned4(verifier) || !aligned4(accept_len) || !aligned4(correction))
    return BRISK_ERR_UNSUPPORTED;
  brisk::launch_verify(proposal, verifier, B, L, accept_len, correction,
                       static_cast<hipStream_t>(stream));
  return launch_status();
}

int brisk_verify_commit(const int32_t* proposal, const int32_t* verifier, int32_t B, int32_t L,
                        int32_t* accept_len, int32_t* committed, int32_t* n_committed, void* stream) {
  if (!proposal || !verifier || !committed || !n_committed) return BRISK_ERR_NULL;
  if (B < 1 || L < 1 || static_cast<int64_t>(B) * (L + 1) > (int64_t{1} << 30)) return BRISK_ERR_SHAPE;
  if (!aligned4(proposal) || !aligned4(verifier) || !aligned4(accept_len) || !aligned4(committed) ||
      !aligned4(n_committed))
    return BRISK_ERR_UNSUPPORTED;
  brisk::launch_commit(proposal, verifier, B, L, accept_len, committed, n_committed,
                       static_cast<hipStream_t>(stream));
  return launch_status();
}

int brisk_spec_verify_workspace_size(int32_t B, int32_t L, int32_t V, int32_t K, size_t* bytes) {
  if (!bytes) return BRISK_ERR_NULL;
  if (B < 1 || L < 1 || static_cast<int64_t>(B) * L > kMaxRows || K < 1 || K > 64 || V <= K)
    return BRISK_ERR_SHAPE;
  *bytes = brisk::spec_verify_workspace_bytes(B, L, V, K);
  return BRISK_OK;
}

int brisk_spec_verify(const uint16_t* ver_hidden, const uint16_t* lm_head, const int32_t* proposal,
                      const int32_t* cand_id, const float* cand_prob, const float* u_accept,
                      uint64_t seed, float temperature, int32_t B, int32_t L, int32_t K, int32_t d,
                      int32_t V, int32_t* accept_len, int32_t* correction, int32_t* row_accept,
                      int32_t* row_resample, void* ws, size_t ws_bytes, void* stream) {
  if (!proposal || !cand_id || !u_accept || !accept_len) return BRISK_ERR_NULL;
  if (B < 1 || L < 1 || static_cast<int64_t>(B) * L > kMaxRows || K < 1 || K > 64 || V <= K ||
      !(temperature > 0.f) || temperature > 3.0e38f)
    return BRISK_ERR_SHAPE;
  const int st = lmhead_check(ver_hidden, lm_head, B * L, d, V, 1);
  if (st != BRISK_OK) return st;
  if (!aligned4(proposal) || !aligned4(cand_id) || !aligned4(cand_prob) || !aligned4(u_accept) ||
      !aligned4(accept_len) || !aligned4(correction) || !aligned4(row_accept) || !aligned4(row_resample))
    return BRISK_ERR_UNSUPPORTED;
  const size_t need = brisk::spec_verify_workspace_bytes(B, L, V, K);
  if (ws_bytes < need || !ws) return BRISK_ERR_WORKSPACE;
  if (!aligned16(ws)) return BRISK_ERR_UNSUPPORTED;
  brisk::launch_spec_verify(ver_hidden, lm_head, B, L, d, V, K, proposal, cand_id, cand_prob, u_accept,
                            seed, temperature, accept_len, correction, row_accept, row_resample, ws,
                            static_cast<hipStream_t>(stream));
  return launch_status();
}

int brisk_corrector_loss(const uint16_t* ver_hidden, const uint16_t* lm_head, const int32_t* cand_id,
                         const float* cand_logit, const float* refined, const int32_t* accept_len,
                         int32_t B, int32_t L, int32_t K, int32_t d, int32_t V, float beta,
                         float* loss_pos, float* ce, float* kl, float* loss_mean, void* stream) {
  if (!ver_hidden || !lm_head || !cand_id || !cand_logit || !refined || !accept_len || !loss_pos ||
      !loss_mean)
    return BRISK_ERR_NULL;
  if (B < 1 || L < 1 || static_cast<int64_t>(B) * L > kMaxRows || K < 1 || K > 64 || V < K || d < 8 ||
      d > kMaxD)
    return BRISK_ERR_SHAPE;
  if (d % 8 != 0 || !aligned16(ver_hidden) || !aligned16(lm_head) || !aligned4(cand_id) ||
      !aligned4(cand_logit) || !aligned4(refined) || !aligned4(accept_len) || !aligned4(loss_pos) ||
      !aligned4(ce) || !aligned4(kl) || !aligned4(loss_mean))
    return BRISK_ERR_UNSUPPORTED;
  brisk::launch_corrector_loss(ver_hidden, lm_head, cand_id, cand_logit, refined, accept_len, B, L, K, d,
                               V, beta, loss_pos, ce, kl, loss_mean, static_cast<hipStream_t>(stream));
  return launch_status();
}

int brisk_accept_profile_workspace_size(int32_t n_blocks, int32_t M, size_t* bytes) {
  if (!bytes) return BRISK_ERR_NULL;
  if (M < 1 || M > kMaxProfileM || n_blocks < 0 || n_blocks > kMaxProfileBlocks) return BRISK_ERR_SHAPE;
  *bytes = brisk::accept_profile_workspace_bytes(n_blocks, M);
  return BRISK_OK;
}

int brisk_accept_profile(const int32_t* accept_len, int32_t n_blocks, int32_t M, double eps,
                         double* a, double* w_raw, double* w, double* tpf_fpt, void* ws,
                         size_t ws_bytes, void* stream) {
  if (!a || !w_raw || !w || !tpf_fpt || (n_blocks > 0 && !accept_len)) return BRISK_ERR_NULL;
  if (M < 1 || M > kMaxProfileM || n_blocks < 0 || n_blocks > kMaxProfileBlocks) return BRISK_ERR_SHAPE;
  if (!aligned4(accept_len) || !aligned8(a) || !aligned8(w_raw) || !aligned8(w) || !aligned8(tpf_fpt))
    return BRISK_ERR_UNSUPPORTED;
  const size_t need = brisk::accept_profile_workspace_bytes(n_blocks, M);
  if (ws_bytes < need || !ws) return BRISK_ERR_WORKSPACE;
  if (!aligned16(ws)) return BRISK_ERR_UNSUPPORTED;
  brisk::launch_accept_profile(accept_len, n_blocks, M, eps, a, w_raw, w, tpf_fpt, ws,
                               static_cast<hipStream_t>(stream));
  return launch_status();
}

}  // extern "C"
