// Launchers of the gfx950 kernels (host side, internal to the library).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "brisk.h"

namespace brisk {

// ---- propose: LM head + fused top-K + merge --------------------------------
size_t propose_workspace_bytes(int rows, int V, int K);
// rows = proposal rows (K candidates each) followed by verifier rows (argmax
// each): rows_prop of them are proposal rows.
// The two launches of launch_propose: the LM-head pass (per-group ordered
// keys into ws) and the merge of those keys into candidates.
void launch_propose_pass(const uint16_t* H, const uint16_t* W, int rows, int d, int V, int K, void* ws,
                         hipStream_t s);
void launch_propose_merge(int rows, int V, int K, int rows_prop, float* cand_logit, int32_t* cand_id,
                          int32_t* ver_token, const void* ws, hipStream_t s);
void launch_propose(const uint16_t* H, const uint16_t* W, int rows, int d, int V, int K,
                    int rows_prop, float* cand_logit, int32_t* cand_id, int32_t* ver_token,
                    void* ws, hipStream_t s);

// The propose call on the library's fixed per-device scratch (the array
// `scratch` in lmhead_topk.hip) instead of a caller's workspace; the caller
// has checked that propose_workspace_bytes fits.  Returns 0, or -1 when the
// stream's device or the scratch address cannot be determined (nothing is
// launched then).
size_t noalloc_scratch_bytes();
int launch_propose_noalloc(const uint16_t* H, const uint16_t* W, int rows, int d, int V, int K,
                           float* cand_logit, int32_t* cand_id, hipStream_t s);

// ---- stochastic speculative verification ------------------------------------
size_t spec_verify_workspace_bytes(int B, int L, int V, int K);
void launch_spec_verify(const uint16_t* Hv, const uint16_t* W, int B, int L, int d, int V, int K,
                        const int32_t* proposal, const int32_t* cand_id, const float* cand_prob,
                        const float* u_accept, uint64_t seed, float temperature, int32_t* accept_len,
                        int32_t* correction, int32_t* row_accept, int32_t* row_resample, void* ws,
                        hipStream_t s);

// ---- rerank: hoisted projections + sequential scan -------------------------
size_t rerank_workspace_bytes(const brisk_corrector& c, int B, int L, int K);
// What one launch_rerank call queues: the whole rerank; only the work that
// does not read the candidates (projections of the hidden states, the
// context and the anchors' embeddings, their lifts), which may run while the
// LM-head pass that makes the candidates streams; or only the rest, on a
// workspace the hoisted part filled.  Split or not, the results are the same
// bits.
enum class RerankPart { kAll, kHoist, kFinish };
void launch_rerank(const brisk_corrector& c, const uint16_t* hidden, const uint16_t* ctx_hidden,
                   const int32_t* anchor_tok, const uint16_t* lm_head, const uint16_t* tok_embed,
                   const float* cand_logit, const int32_t* cand_id, int B, int L, int K, int d,
                   int V, int32_t* selected, float* refined, float* gamma, float* resid,
                   const int32_t* verifier, int32_t* accept_len, int32_t* correction, void* ws,
                   hipStream_t s, RerankPart part = RerankPart::kAll);

// Per-token tables [EH; TZ; TH], each [V][step vector stride] fp32, and the
// scratch their preparation needs.
size_t corrector_tables_bytes(const brisk_corrector& c, int V);
size_t corrector_prepare_ws_bytes(const brisk_corrector& c, int V);
void launch_corrector_prepare(const brisk_corrector& c, const uint16_t* lm_head, const uint16_t* tok_embed,
                              int V, int d, float* tables, void* ws, hipStream_t s);

// ---- verify -----------------------------------------------------------------
void launch_verify(const int32_t* proposal, const int32_t* verifier, int B, int L,
                   int32_t* accept_len, int32_t* correction, hipStream_t s);
void launch_commit(const int32_t* proposal, const int32_t* verifier, int B, int L,
                   int32_t* accept_len, int32_t* committed, int32_t* n_committed, hipStream_t s);

// ---- corrector training loss (forward) ---------------------------------------
void launch_corrector_loss(const uint16_t* ver_hidden, const uint16_t* lm_head, const int32_t* cand_id,
                           const float* cand_logit, const float* refined, const int32_t* accept_len,
                           int B, int L, int K, int d, int V, float beta, float* loss_pos, float* ce,
                           float* kl, float* loss_mean, hipStream_t s);

// ---- acceptance profile -------------------------------------------------------
size_t accept_profile_workspace_bytes(int n_blocks, int M);
void launch_accept_profile(const int32_t* accept_len, int n_blocks, int M, double eps, double* a,
                           double* w_raw, double* w, double* tpf_fpt, void* ws, hipStream_t s);

}  // namespace brisk
