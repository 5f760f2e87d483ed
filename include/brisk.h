/*
 * brisk.h - C ABI of the BRISK-DLM decoding hot path on MI355X (gfx950).
 *
 * One decoding step of the paper's prefix-conditioned proposal selection
 * (Section 3.3, Algorithm 1(b)) in three calls:
 *
 *   brisk_propose_block  LM-head projection of every masked position's hidden
 *                        state and its ordered top-K candidate set;
 *   brisk_rerank         the corrector that re-scores those candidates left to
 *                        right, conditioned on the tokens already selected;
 *   brisk_verify_accept  greedy verification: accepted-prefix length and the
 *                        correction token of each block.
 *
 * brisk_rerank_verify makes the last two in one call; brisk_rerank_hoist and
 * brisk_rerank_finish split the rerank at the candidates, so that its first
 * part can overlap the LM-head pass.
 *
 * Conventions shared by every entry point
 *   - Every pointer argument is a DEVICE pointer owned by the caller, except
 *     the brisk_corrector struct itself (host memory, read during the call)
 *     and the size out-parameters.  The library allocates nothing and is
 *     reentrant; calls on different streams are safe when their workspaces
 *     and outputs differ.  Its only global state is the fixed scratch of
 *     brisk_propose_block_noalloc (one array per GPU, and its address).
 *   - bf16 tensors are passed as uint16_t bit patterns; all matrices are
 *     row-major and densely packed (row stride = row length).
 *   - Rows of a block are numbered r = b * L + (i - 1) for sequence b and
 *     in-block position i = 1..L.
 *   - `stream` is a hipStream_t (NULL = the default stream).  Work is queued
 *     on it asynchronously; nothing synchronises.
 *   - Every call returns a brisk_status.  Arguments are validated on the host
 *     before any HIP call: on an error return nothing has been launched and no
 *     output has been touched.  BRISK_ERR_HIP reports a failed launch.
 *   - Token ids read from device memory (candidate ids, anchor tokens) are
 *     clamped into [0, V) before they address a table, so a bad id cannot make
 *     a kernel read out of bounds; the results for such a row are unspecified.
 *   - Pointers must be 16-byte aligned and d a multiple of 8, otherwise
 *     BRISK_ERR_UNSUPPORTED.
 */
#ifndef BRISK_H_
#define BRISK_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  BRISK_OK = 0,
  BRISK_ERR_NULL = -1,        /* a required pointer is NULL                   */
  BRISK_ERR_SHAPE = -2,       /* a size is out of range or inconsistent        */
  BRISK_ERR_UNSUPPORTED = -3, /* alignment / divisibility the kernels need     */
  BRISK_ERR_WORKSPACE = -4,   /* workspace missing or smaller than required    */
  BRISK_ERR_HIP = -5,         /* a HIP launch failed                           */
  BRISK_ERR_SCRATCH = -6      /* the shape needs more than the fixed scratch  */
} brisk_status;

/* Static, NUL-terminated description of a status code. */
const char* brisk_status_str(int status);

/* Library ABI version (bumped on any signature or struct change). */
int brisk_abi_version(void);

/*
 * Corrector parameters psi (Section 3.3 Eq. inference_head_state and
 * Eq. candidate_residual; Appendix "Candidate-Refinement Head Details",
 * Eq. head_residual_logits and the head configuration table).  All tensor
 * pointers are device bf16 bit patterns, row-major:
 *
 *   u_0      = tanh(A_h h_c + A_e E(x_0))
 *   x_hat_i  = [P_h m_i ; P_e E(x_{i-1}) ; pos_emb[i-1] ; P_phi phi_i]
 *   z        = sigmoid(W_z x_hat_i),  u_i = (1 - z) * u_{i-1} + z * (W_h x_hat_i)
 *   gamma_i  = sigmoid(alpha) * sigmoid(w_g . [u_i ; phi_i] + b_g)
 *   l~_{i,k} = l_{i,k} + gamma_i * <W_s u_i, W_c E_out(v_{i,k})>
 *
 * with phi_i = [top1-top2, top1-top4, 1[x_{i-1} = top1], 1[x_{i-1} in top4],
 * top1 - l_i(x_{i-1})] from the position's ordered candidates and E_out the
 * LM head.  Dimension limits: d_state in [1, 512], d_hproj, d_tproj, rank in
 * [1, 256], d_pos, d_feat in [1, 64], max_L >= 1.
 */
typedef struct brisk_corrector {
  int32_t d_state, d_hproj, d_tproj, d_pos, d_feat, rank, max_L;
  const uint16_t* A_h;      /* [d_state, d]                               */
  const uint16_t* A_e;      /* [d_state, d]                               */
  const uint16_t* P_h;      /* [d_hproj, d]                               */
  const uint16_t* P_e;      /* [d_tproj, d]                               */
  const uint16_t* pos_emb;  /* [max_L, d_pos]                             */
  const uint16_t* P_phi;    /* [d_feat, 5]                                */
  const uint16_t* W_z;      /* [d_state, d_in], d_in = d_hproj+d_tproj+d_pos+d_feat */
  const uint16_t* W_h;      /* [d_state, d_in]                            */
  const uint16_t* W_s;      /* [rank, d_state]                            */
  const uint16_t* W_c;      /* [rank, d]                                  */
  const uint16_t* w_g;      /* [d_state + 5]                              */
  float alpha;              /* gate scale logit (host value)               */
  float b_g;                /* gate bias (host value)                      */
  /* Optional per-token tables from brisk_corrector_prepare (NULL: none).
   * When set, the rerank calls read the lifts of candidate and anchor tokens
   * from them instead of projecting their embedding rows; tables_V must then
   * equal the call's V, and the tables must have been prepared from these
   * parameters and the same lm_head and tok_embed (not checked). */
  const float* tables;      /* [3][tables_V][max(256, d_state)] fp32       */
  int32_t tables_V;
} brisk_corrector;

/*
 * Per-token tables of the corrector (Section 3.3 Eq. inference_head_state and
 * Eq. candidate_residual; Appendix Eq. head_residual_logits).  Every map the
 * corrector applies to a token's embedding rows is linear and fixed once the
 * model is loaded: the token projection reaches the state update as
 * TZ(v) = W_z[:, t] P_e E(v) and TH(v) = W_h[:, t] P_e E(v), and the residual
 * re-associates to <u_i, EH(v)> with EH(v) = W_s^T W_c E_out(v) (t = the
 * d_tproj columns of W_z and W_h that read P_e E).  brisk_corrector_prepare
 * computes the three for every token (bf16 inputs, fp32 accumulation) into
 * tables [EH; TZ; TH], each [V][max(256, d_state)] fp32 with rows zero-padded
 * past d_state.  Preparing once per model replaces the per-step gathers of
 * whole E and E_out rows by gathers of table rows; the decoding results are
 * those of the per-step projections up to fp32 rounding.
 *
 *   c          corrector parameters (its tables field is ignored here)
 *   lm_head    [V, d] bf16  E_out;   tok_embed [V, d] bf16  E
 *   tables     out, table_bytes >= *table_bytes of brisk_corrector_tables_size
 *   ws         scratch of at least *ws_bytes bytes (V * (d_tproj + rank) fp32)
 *
 * Limits as brisk_rerank's for the corrector; 1 <= V <= 2^24, 8 <= d <= 65536,
 * d % 8 == 0, 16-byte aligned pointers.
 */
int brisk_corrector_tables_size(const brisk_corrector* c, int32_t V, size_t* table_bytes, size_t* ws_bytes);
int brisk_corrector_prepare(const brisk_corrector* c, const uint16_t* lm_head, const uint16_t* tok_embed,
                            int32_t V, int32_t d, float* tables, size_t table_bytes, void* ws,
                            size_t ws_bytes, void* stream);

/*
 * Workspace bytes brisk_propose_block needs for this shape (written to *bytes).
 * Returns BRISK_ERR_SHAPE / BRISK_ERR_NULL on bad arguments.
 */
int brisk_propose_workspace_size(int32_t rows, int32_t d, int32_t V, int32_t K, size_t* bytes);

/*
 * Candidate construction C_i = TopK(q_i, K) (Section 3.3; Appendix head
 * details; Algorithm 1(b) first step and loop head).  Computes the proposal
 * logits l[r, v] = sum_k hidden[r, k] * lm_head[v, k] (bf16 inputs, fp32
 * accumulation; the [rows, V] logits never reach memory) and returns the K
 * largest per row, ordered by logit descending and, among equal logits, by
 * token id ascending.  Top-K of the softmax q equals top-K of the logits.
 *
 *   hidden      [rows, d]  bf16   masked-position hidden states m_i
 *   lm_head     [V, d]     bf16   frozen LM head (output vocabulary rows)
 *   cand_logit  [rows, K]  fp32   out: candidate logits, descending
 *   cand_id     [rows, K]  int32  out: candidate token ids
 *   ws          device scratch of at least brisk_propose_workspace_size bytes
 *
 * Limits: 1 <= rows <= 2^20, 8 <= d <= 65536, 1 <= K <= 64, K <= V; V*d*2 and
 * rows*d*2 below 2^32 bytes (BRISK_ERR_UNSUPPORTED otherwise).
 */
int brisk_propose_block(const uint16_t* hidden, const uint16_t* lm_head,
                        int32_t rows, int32_t d, int32_t V, int32_t K,
                        float* cand_logit, int32_t* cand_id,
                        void* ws, size_t ws_bytes, void* stream);

/*
 * brisk_propose_block without a workspace, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc).  Same arguments, results, limits and errors as
 * brisk_propose_block, minus ws and ws_bytes: the key lists live in a fixed
 * array of BRISK_NOALLOC_SCRATCH_BYTES (16 MiB) that the library holds on
 * each GPU it runs on until the process ends.  A shape whose
 * brisk_propose_workspace_size exceeds that returns BRISK_ERR_SCRATCH (the
 * five decoding workloads need 0.5-8 MiB).  The call allocates nothing; its
 * first call on a device looks up that device's copy of the array (with the
 * stream's device made current for the lookup), and BRISK_ERR_HIP reports a
 * failed lookup.  Every call on one GPU uses the same array: calls that
 * overlap in time on one GPU (on different streams, or from different host
 * threads) race and their results are undefined; serialise them.
 */
#define BRISK_NOALLOC_SCRATCH_BYTES ((size_t)16 << 20)
int brisk_propose_block_noalloc(const uint16_t* hidden, const uint16_t* lm_head,
                                int32_t rows, int32_t d, int32_t V, int32_t K,
                                float* cand_logit, int32_t* cand_id, void* stream);

/*
 * The two launches of brisk_propose_block, one call each (same section of the
 * paper, same arguments, limits and workspace).  brisk_propose_lmhead is the
 * LM-head pass: it leaves in ws, for every row and vocabulary share, the
 * ordered keys of that share's K largest logits.  brisk_propose_merge reduces
 * those keys to the candidates.  brisk_propose_block is exactly the two in
 * order on one stream; calling them separately lets a caller time or
 * schedule each launch on its own.  A merge reads the workspace of the pass
 * before it on the same stream, which must have used the same rows, V and K
 * (the layout depends on them); it does not check that.
 */
int brisk_propose_lmhead(const uint16_t* hidden, const uint16_t* lm_head, int32_t rows, int32_t d,
                         int32_t V, int32_t K, void* ws, size_t ws_bytes, void* stream);
int brisk_propose_merge(int32_t rows, int32_t V, int32_t K, float* cand_logit, int32_t* cand_id,
                        const void* ws, size_t ws_bytes, void* stream);

/* Workspace bytes brisk_rerank needs (written to *bytes). */
int brisk_rerank_workspace_size(const brisk_corrector* c, int32_t B, int32_t L, int32_t K,
                                size_t* bytes);

/*
 * Prefix-conditioned rerank of the candidates (Section 3.3; Appendix head
 * details; Algorithm 1(b) loop): steps the corrector over i = 1..L for every
 * sequence, feeding the token selected at i-1 (x_0 at i = 1) into step i, and
 * selects x_i = the candidate with the largest refined logit (the smallest
 * candidate index on ties).
 *
 *   c           host struct of device parameter pointers (see above)
 *   hidden      [B*L, d] bf16   m_i
 *   ctx_hidden  [B, d]   bf16   h_c
 *   anchor_tok  [B]      int32  x_0, the token preceding each block
 *   lm_head     [V, d]   bf16   E_out (the same matrix brisk_propose_block used)
 *   tok_embed   [V, d]   bf16   E, the input token embedding
 *   cand_logit, cand_id [B*L, K] the candidate sets from brisk_propose_block
 *   selected    [B, L]   int32  out: x_{1..L}
 *   refined     [B*L, K] fp32   out, nullable: refined logits l~
 *   gamma       [B*L]    fp32   out, nullable: gate gamma_i
 *   resid       [B*L, K] fp32   out, nullable: residual <W_s u_i, W_c E_out(v)>
 *
 * Limits: 4 <= K <= 64 (the features read the top-4), 1 <= L <= max_L,
 * B*L <= 2^20, and one sequence's step blocks L*(2+3K)*max(256, d_state)*4
 * below 2^31 bytes (each step vector is padded to at least 256 floats);
 * beyond that the call returns BRISK_ERR_UNSUPPORTED.
 */
int brisk_rerank(const brisk_corrector* c, const uint16_t* hidden, const uint16_t* ctx_hidden,
                 const int32_t* anchor_tok, const uint16_t* lm_head, const uint16_t* tok_embed,
                 const float* cand_logit, const int32_t* cand_id,
                 int32_t B, int32_t L, int32_t K, int32_t d, int32_t V,
                 int32_t* selected, float* refined, float* gamma, float* resid,
                 void* ws, size_t ws_bytes, void* stream);

/*
 * Greedy verification (Section 2.2 accepted prefix; Section 3.3 speculative
 * acceptance, temperature-zero case; Algorithm 1(b) verify and commit):
 * accept_len[b] = number of leading positions i with proposal[b, i] ==
 * verifier[b, i], in [0, L]; correction[b] = verifier[b, accept_len[b]] when
 * accept_len[b] < L, else -1.
 *
 *   proposal    [B, L] int32   proposed tokens x_{1..L}
 *   verifier    [B, L] int32   the verifier's argmax tokens
 *   accept_len  [B]    int32   out
 *   correction  [B]    int32   out, nullable
 */
int brisk_verify_accept(const int32_t* proposal, const int32_t* verifier, int32_t B, int32_t L,
                        int32_t* accept_len, int32_t* correction, void* stream);

/*
 * brisk_rerank followed by brisk_verify_accept on its selections, in one call
 * (Algorithm 1(b): select, then verify).  Same arguments as brisk_rerank plus
 *
 *   verifier    [B, L] int32  the verifier's token at every position
 *   accept_len  [B] int32 out, correction [B] int32 out (nullable), as in
 *               brisk_verify_accept
 *
 * When the single-wavefront scan runs (d_state <= 256, K <= 16) the scan
 * itself compares each selection with the verifier's token, so no separate
 * launch follows; otherwise the verification kernel runs after the scan.
 * Results equal the two calls made one after the other.
 */
int brisk_rerank_verify(const brisk_corrector* c, const uint16_t* hidden, const uint16_t* ctx_hidden,
                        const int32_t* anchor_tok, const uint16_t* lm_head, const uint16_t* tok_embed,
                        const float* cand_logit, const int32_t* cand_id, const int32_t* verifier,
                        int32_t B, int32_t L, int32_t K, int32_t d, int32_t V, int32_t* selected,
                        float* refined, float* gamma, float* resid, int32_t* accept_len,
                        int32_t* correction, void* ws, size_t ws_bytes, void* stream);

/*
 * brisk_rerank (or brisk_rerank_verify) in two parts, so that the first can
 * run while the LM-head pass that makes the candidates streams (same section
 * of the paper).  brisk_rerank_hoist queues the work that does not read the
 * candidates: the projections P_h m_i, A_h h_c and A_e E(x_0), the sums of
 * their split reductions, and their lifts into the step vectors together
 * with the position and feature terms.  brisk_rerank_finish queues the rest
 * on a workspace that a brisk_rerank_hoist call filled and nothing has
 * written since: with verifier NULL it completes brisk_rerank, otherwise
 * brisk_rerank_verify (then accept_len is required; correction is nullable).
 *
 * Both calls take brisk_rerank's arguments (brisk_rerank_hoist only those it
 * reads) with the same c, hidden, ctx_hidden, anchor_tok, tok_embed, B, L,
 * K, d, V and workspace, and the same limits and errors; the library does
 * not check that the two calls agree.  The caller orders them: on one
 * stream, or the finishing call's stream waits on an event recorded after
 * the hoist.  The results are bitwise those of the single call.
 */
int brisk_rerank_hoist(const brisk_corrector* c, const uint16_t* hidden, const uint16_t* ctx_hidden,
                       const int32_t* anchor_tok, const uint16_t* tok_embed, int32_t B, int32_t L,
                       int32_t K, int32_t d, int32_t V, void* ws, size_t ws_bytes, void* stream);
int brisk_rerank_finish(const brisk_corrector* c, const uint16_t* hidden, const uint16_t* ctx_hidden,
                        const int32_t* anchor_tok, const uint16_t* lm_head, const uint16_t* tok_embed,
                        const float* cand_logit, const int32_t* cand_id, const int32_t* verifier,
                        int32_t B, int32_t L, int32_t K, int32_t d, int32_t V, int32_t* selected,
                        float* refined, float* gamma, float* resid, int32_t* accept_len,
                        int32_t* correction, void* ws, size_t ws_bytes, void* stream);

/* Workspace bytes brisk_propose_verify needs (written to *bytes). */
int brisk_propose_verify_workspace_size(int32_t rows_prop, int32_t rows_ver, int32_t d, int32_t V,
                                        int32_t K, size_t* bytes);

/*
 * One LM-head pass for both kinds of rows a self-verifying decoding step
 * produces (Section 2.1 introspective strided decoding, where proposal and
 * causal verification come from the same model evaluation; Section 3.3;
 * Algorithm 1(b) first step and verify): the proposal rows of the next block
 * get their ordered top-K candidates, exactly as brisk_propose_block, and the
 * verifier rows of the block under verification get their argmax token (the
 * largest logit, the lower id on ties), without a second pass over lm_head.
 *
 *   hidden      [rows_prop + rows_ver, d] bf16: proposal rows first, then
 *               verifier rows
 *   lm_head     [V, d] bf16
 *   cand_logit, cand_id  [rows_prop, K] out (may be NULL when rows_prop == 0)
 *   ver_token   [rows_ver] int32 out (may be NULL when rows_ver == 0)
 *   ws          device scratch of brisk_propose_verify_workspace_size bytes
 *
 * Limits as brisk_propose_block with rows = rows_prop + rows_ver >= 1.
 */
int brisk_propose_verify(const uint16_t* hidden, const uint16_t* lm_head, int32_t rows_prop,
                         int32_t rows_ver, int32_t d, int32_t V, int32_t K, float* cand_logit,
                         int32_t* cand_id, int32_t* ver_token, void* ws, size_t ws_bytes,
                         void* stream);

/*
 * Greedy verification and commit (Algorithm 1(b): verify, then commit the
 * accepted prefix and the correction; Section 2.2 accepted prefix).  For
 * block b with a = accept length (as brisk_verify_accept):
 *   committed[b, 0..a-1] = proposal[b, 0..a-1];
 *   committed[b, a]      = verifier[b, a]        when a < L;
 *   the rest of the L + 1 slots = -1;  n_committed[b] = a + (a < L).
 *
 *   proposal, verifier  [B, L] int32
 *   accept_len          [B] int32 out, nullable
 *   committed           [B, L + 1] int32 out
 *   n_committed         [B] int32 out
 */
int brisk_verify_commit(const int32_t* proposal, const int32_t* verifier, int32_t B, int32_t L,
                        int32_t* accept_len, int32_t* committed, int32_t* n_committed,
                        void* stream);

/* Workspace bytes brisk_spec_verify needs (written to *bytes). */
int brisk_spec_verify_workspace_size(int32_t B, int32_t L, int32_t V, int32_t K, size_t* bytes);

/*
 * Stochastic speculative verification (Section 3.3; Algorithm 1(b) verify
 * and commit).  Position i of block b (row r = b * L + i) accepts its
 * proposal x_r with probability min{1, p_r(x_r) / pi_r(x_r)}, where p_r is
 * the verifier's softmax at temperature T over the whole vocabulary (logits
 * <lm_head[v], ver_hidden[r]>, one fused LM-head pass with an online
 * log-sum-exp) and pi_r the proposal law over the position's candidates.
 * Each row also draws y_r from the normalised positive part [p_r - pi_r]_+,
 * which keeps the committed token distributed as p_r; the block stops at its
 * first rejection a and commits y at position a.
 *
 *   ver_hidden  [B*L, d] bf16    verifier hidden states
 *   lm_head     [V, d]   bf16
 *   proposal    [B, L]   int32   x
 *   cand_id     [B*L, K] int32   distinct candidate ids of each position
 *   cand_prob   [B*L, K] fp32    pi over those ids (tokens outside have pi = 0);
 *               nullable: NULL means the greedy proposer, pi = point mass at
 *               x (when x is among the candidates)
 *   u_accept    [B*L]    fp32    uniforms in [0, 1) for the accept tests
 *   seed        key of the Philox4x32-10 generator of the residual draws
 *               (Gumbel variate of token v at row r from word v mod 4 of
 *               counter (v / 4, r, 0, 0))
 *   accept_len  [B] int32 out;  correction [B] int32 out, nullable (-1 when
 *               the block is fully accepted)
 *   row_accept, row_resample  [B*L] int32 out, nullable: every position's
 *               accept decision (1/0) and residual draw
 *   ws          device scratch of brisk_spec_verify_workspace_size bytes
 *
 * Limits: 1 <= K <= 64, K < V, temperature > 0, B*L <= 2^20, and the LM-head
 * limits of brisk_propose_block.
 */
int brisk_spec_verify(const uint16_t* ver_hidden, const uint16_t* lm_head, const int32_t* proposal,
                      const int32_t* cand_id, const float* cand_prob, const float* u_accept,
                      uint64_t seed, float temperature, int32_t B, int32_t L, int32_t K, int32_t d,
                      int32_t V, int32_t* accept_len, int32_t* correction, int32_t* row_accept,
                      int32_t* row_resample, void* ws, size_t ws_bytes, void* stream);

/*
 * Corrector training loss, forward (Appendix "Candidate-Refinement Head
 * Details", Eq. head_training_loss).  For position j of block b (row
 * r = b * L + j) with candidates v_{r,k}:
 *   p_S = softmax_k <lm_head[v_{r,k}], ver_hidden[r]>   (verifier, restricted)
 *   q_S = softmax_k cand_logit[r, k]                     (base proposal, restricted)
 *   r   = softmax_k refined[r, k]                        (corrector)
 *   loss_pos[r] = CE(p_S, r) + beta * KL(q_S || r)  on reached positions
 *                 (j <= accept_len[b]: the accepted prefix and the first
 *                 rejection), 0 elsewhere
 *   loss_mean   = {mean of loss_pos over reached positions, their count}
 *
 *   ver_hidden  [B*L, d] bf16   the verifier's hidden states
 *   lm_head     [V, d]   bf16
 *   cand_id, cand_logit, refined  [B*L, K] (from brisk_propose_block and
 *               brisk_rerank)
 *   accept_len  [B] int32      (from brisk_verify_accept)
 *   loss_pos    [B*L] fp32 out;  ce, kl [B*L] fp32 out, nullable
 *   loss_mean   [2]   fp32 out
 *
 * Limits: 1 <= K <= 64, d % 8 == 0 with 16-byte aligned bf16 pointers, B*L
 * <= 2^20.  Deterministic (fixed-order sums).
 */
int brisk_corrector_loss(const uint16_t* ver_hidden, const uint16_t* lm_head, const int32_t* cand_id,
                         const float* cand_logit, const float* refined, const int32_t* accept_len,
                         int32_t B, int32_t L, int32_t K, int32_t d, int32_t V, float beta,
                         float* loss_pos, float* ce, float* kl, float* loss_mean, void* stream);

/* Workspace bytes brisk_accept_profile needs (written to *bytes). */
int brisk_accept_profile_workspace_size(int32_t n_blocks, int32_t M, size_t* bytes);

/*
 * Acceptance profile and efficiency statistics of verified blocks (Section
 * 3.2 Eq. nonuniform_tpf and Eq. brisk_weighting; Appendix "Brisk Backbone",
 * Eq. idlm_tpf_instantiation and the rejection-rate estimate of a_i).  From
 * the accepted-prefix lengths of n_blocks blocks of M proposal positions
 * (block b reaches positions 1..L_b + 1 and is rejected at L_b + 1 when
 * L_b < M):
 *   a[i]      = 1 - rejected_i / reached_i   (1 for a position no block reaches)
 *   w_raw[i]  = -dFPT/dz_i, z_i = log(a_i / (1 - a_i)), FPT = 1 / TPF with the
 *               ISD instantiation TPF = (2 + sum_{k=1}^{M-1} A_k) / (2 - A_M),
 *               A_k = prod_{j<=k} a_j
 *   w[i]      = M w_raw[i] / (sum_j w_raw[j] + eps)
 *   tpf_fpt   = {TPF, FPT}
 *
 *   accept_len  [n_blocks] int32   accepted-prefix lengths (e.g. the output of
 *                                  brisk_verify_accept); values outside [0, M]
 *                                  are clamped into it; may be NULL when
 *                                  n_blocks == 0
 *   a, w_raw, w [M] fp64 out;  tpf_fpt [2] fp64 out
 *   ws          device scratch of brisk_accept_profile_workspace_size bytes
 *
 * Limits: 1 <= M <= 1024, 0 <= n_blocks <= 2^30.  Deterministic: the counts
 * are integers and every floating-point sum runs in a fixed order.
 */
int brisk_accept_profile(const int32_t* accept_len, int32_t n_blocks, int32_t M, double eps,
                         double* a, double* w_raw, double* w, double* tpf_fpt,
                         void* ws, size_t ws_bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* BRISK_H_ */
