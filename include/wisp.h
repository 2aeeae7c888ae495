/*
 * wisp.h -- C ABI of the MI355X (gfx950) batched speculative-verification step.
 *
 * The step is the server-side verification of WISP (arXiv 2601.11652): Sec. 4.5
 * ("batched one-step verification") forwards each request's drafted block on top of
 * its cached prefix KV in one pass, then applies the speculative-sampling rule of
 * Sec. 2.4 (Eq. (1) acceptance u <= min(1, p/q), Eq. (2) first rejection R and
 * accepted length L = R - 1, Eq. (3) the extra token), returning (L, extra token)
 * per request.  At a rejection the extra token is drawn from norm(max(0, p - q)) --
 * the residual that makes the rule lossless (Leviathan et al., cited in Sec. 4.5);
 * after a fully accepted block it is drawn from p.
 *
 * Conventions for every entry point:
 *   - "DEVICE" pointers are HIP device memory owned by the caller; "HOST" pointers
 *     are ordinary host memory owned by the caller and read during the call only.
 *   - All GPU work is enqueued on `stream` (a hipStream_t passed as void*; NULL is
 *     the default stream).  Calls return after enqueueing; outputs are valid once
 *     the stream is synchronised.  Nothing here allocates device memory except
 *     where stated; scratch comes from the caller's workspace.
 *   - Non-zero return values are errors; wisp_last_error() returns a thread-local
 *     message for the last failing call.  No C++ exception crosses this boundary.
 *   - Calls that share a workspace must not overlap on the GPU.
 */
#ifndef WISP_H
#define WISP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  WISP_OK = 0,
  WISP_E_INVALID = -1,      /* bad descriptor, NULL pointer, gamma > 16, ctx_len < 0, T < 0   */
  WISP_E_CAPACITY = -2,     /* page table too short for ctx_len + gamma + 1 tokens           */
  WISP_E_WORKSPACE = -3,    /* workspace smaller than wisp_workspace_size()                  */
  WISP_E_UNSUPPORTED = -4,  /* shape outside what the kernels implement                      */
  WISP_E_HIP = -5,          /* HIP runtime error                                             */
  WISP_E_DEVICE_INPUT = -6, /* a device-side input check failed (token id, block id)         */
  WISP_E_HOST_MEMORY = -7   /* host memory exhausted while planning or bookkeeping           */
} wisp_status;

typedef enum { WISP_F32 = 0, WISP_BF16 = 1 } wisp_dtype;

#define WISP_PAGE 16        /* tokens per KV page                                            */
#define WISP_GAMMA_MAX 16   /* most draft tokens per request                                 */
#define WISP_PREFILL_MAX 32768 /* most uncached prompt tokens per request and call (prefill_len) */
#define WISP_ROWS_MAX 262144  /* most rows per model call (wisp_verify, wisp_attention): sum of
                                 prefill_len + gamma + 1; WISP_E_UNSUPPORTED beyond.  The
                                 acceptance alone (wisp_accept) takes up to 2^29 rows.    */

/*
 * Decoder-only transformer (RMSNorm, rotary embedding with rotate-half pairing,
 * grouped-query attention, SwiGLU MLP, untied LM head) -- the target model of the
 * verification engine (Sec. 4.5).  The paper names its target models (Qwen3,
 * Llama) but not their internals; this layout follows the Llama-3 family.
 *
 * All weight pointers are DEVICE pointers of `dtype`.  The per-layer arrays are
 * HOST arrays of n_layers DEVICE pointers.
 *   embed       [vocab][d_model]                 natural row-major
 *   final_norm, attn_norm[l], mlp_norm[l]  [d_model]
 *   w_qkv[l]    rows (n_q + 2 n_kv) * head_dim  (W_q rows, then W_k, then W_v), K = d_model
 *   w_o[l]      rows d_model,   K = n_q * head_dim
 *   w_gate_up[l] rows 2 * d_ff, K = d_model: W_gate and W_up packed together by
 *               wisp_pack_gate_up (for WISP_BF16 their 32-row blocks interleave, so one
 *               output tile holds both halves of each SwiGLU pair; WISP_F32: W_gate rows,
 *               then W_up)
 *   w_down[l]   rows d_model,   K = d_ff
 *   lm_head     rows vocab,     K = d_model
 * Shapes: d_model and d_ff multiples of 32, d_model <= 8192; head_dim a multiple of 32 up
 * to 256 (64 or 128 for WISP_BF16), n_q_heads a multiple of n_kv_heads; for WISP_BF16 also vocab a
 * multiple of 32 and at most 64 query heads per kv head.  Others: WISP_E_UNSUPPORTED.
 * Linear weights ("rows x K", nn.Linear's [out][in]) must be stored in the packed
 * form made by wisp_pack_linear() (wisp_pack_gate_up() for w_gate_up): for WISP_BF16 an
 * MFMA-fragment order, for WISP_F32 plain row-major.
 */
typedef struct {
  int32_t n_layers, d_model, n_q_heads, n_kv_heads, head_dim, d_ff, vocab;
  float rms_eps;      /* RMSNorm epsilon (1e-5 for the Llama shapes)                       */
  float rope_base;    /* rotary base theta                                                 */
  int32_t dtype;      /* wisp_dtype of weights, KV pages and GEMM-input activations        */
  const void *embed, *final_norm, *lm_head;
  const void *const *attn_norm, *const *w_qkv, *const *w_o;
  const void *const *mlp_norm, *const *w_gate_up, *const *w_down;
} wisp_model;

/*
 * Paged KV cache (PageAttention-style fixed-size blocks plus a per-request block
 * table, Sec. 4.5).  Two DEVICE pools of `dtype`, each
 *   [n_layers][n_blocks][n_kv_heads][page of 16 * head_dim elements].
 * Inside one page (one block, one kv head) element (slot s, dim e) sits at
 *   K:  (((e / 32) * 2 + (s / 4) % 2) * 4 + (e % 32) / 8) * 64 + ((s / 8) * 4 + s % 4) * 8 + e % 8
 *   V:  ((e / 16) * 2 + s / 8) * 128 + (e % 16) * 8 + s % 8
 * (operand order of gfx950's 16x16x32 matrix instructions: a pair of pages streams as
 * contiguous 512-byte half-wave loads, and every lane's K or V operand is one 16-byte
 * load from one page).  head_dim must be a multiple of 32.
 * Token t of request i lives in block kv_page_table[i][t / 16], slot t % 16.
 */
typedef struct {
  void *k_pool;
  void *v_pool;
  int32_t n_blocks;
  int32_t page_size;  /* must be WISP_PAGE                                                 */
} wisp_kv;

/*
 * One verification batch (a micro-batch chosen by the scheduler, Sec. 4.3).
 * Request i brings gamma[i] draft tokens on top of ctx_len[i] cached tokens; the
 * step forwards gamma[i] + 1 rows [root, y_1..y_gamma] at positions
 * ctx_len[i] .. ctx_len[i] + gamma[i], where root is the last committed token
 * (the previous round's extra token), whose KV is not cached yet.  Row j's logits
 * score draft y_{j+1}; row gamma[i] is the bonus position.
 *
 * First-time (cold-start) verification and chunked prefill (Sec. 4.4's two verification
 * types): prefill_len[i] > 0 adds that many uncached prompt tokens in front of the root,
 * so the request forwards prefill_len[i] + gamma[i] + 1 rows [p_0 .. p_{P-1}, root,
 * y_1 .. y_gamma] at positions ctx_len[i] ..; root is then the prompt's last token.  Their
 * K/V are appended and they take part in the causal attention, but only the gamma[i] + 1
 * verification rows produce logits and enter the acceptance.  A cold start has
 * ctx_len[i] = 0; a later chunk of a long prompt has the earlier chunks cached.
 */
typedef struct {
  int32_t B;
  const int32_t *ctx_len;        /* HOST [B]  tokens already cached, >= 0                   */
  const int32_t *gamma;          /* HOST [B]  0..WISP_GAMMA_MAX; 0 = ordinary decoding      */
  const uint32_t *req_id;        /* HOST [B]  keys the request's random stream; NULL = i    */
  const int32_t *kv_page_table;  /* DEVICE [B][pt_stride] block ids                         */
  int32_t pt_stride;             /* pages per request in the table                         */
  float temperature;             /* target temperature: > 0 sampled, 0 greedy              */
  const int32_t *prefill_len;    /* HOST [B]  0..WISP_PREFILL_MAX uncached prompt tokens
                                    before the root; NULL = none                            */
} wisp_batch_desc;

/* Bytes of DEVICE workspace wisp_verify needs for this model and batch (0 on error), and
 * the extra bytes it needs when the caller passes no target_logits buffer. */
size_t wisp_workspace_size(const wisp_model *model, const wisp_batch_desc *desc);
size_t wisp_logits_workspace_size(const wisp_model *model, const wisp_batch_desc *desc);

/*
 * Pack one linear weight (natural [rows][cols] row-major, DEVICE `src`) into the
 * layout the GEMMs read (DEVICE `dst`, same byte size; must not alias src).
 * WISP_BF16: rows % 32 == 0 and cols % 16 == 0; the packed matrix is a sequence of
 * 32 x 16 fragments, fragment (rb, kb) at ((rb * cols/16 + kb) * 512) elements,
 * lane l's 8 elements at l * 8 holding row rb*32 + l%32, columns kb*16 + (l/32)*8 + 0..7.
 * Row blocks are independent, so several matrices stacked by rows (W_q|W_k|W_v)
 * are packed by calling this once per matrix at dst + (row offset * cols).
 * WISP_F32: a plain copy.
 */
wisp_status wisp_pack_linear(void *dst, const void *src, int32_t rows, int32_t cols, int32_t dtype,
                             void *stream);

/*
 * Pack the MLP's gate and up weights (natural [d_ff][d_model] row-major each, DEVICE) into
 * w_gate_up (DEVICE, 2 * d_ff * d_model elements; must not alias the sources).
 * WISP_BF16: d_ff % 32 == 0 and d_model % 16 == 0; the fragment order of wisp_pack_linear
 * over 2 * d_ff rows whose 32-row blocks interleave, block 2b holding W_gate rows
 * 32b .. 32b + 31 and block 2b + 1 the W_up rows of the same b.  An output tile of the
 * gate/up projection then holds gate and up of the same columns, and the step applies
 * SwiGLU (silu(gate) * up, Sec. 4.5's target model) in that projection's epilogue.
 * WISP_F32: W_gate rows, then W_up rows (plain copies).
 */
wisp_status wisp_pack_gate_up(void *dst, const void *w_gate, const void *w_up, int32_t d_ff, int32_t d_model,
                              int32_t dtype, void *stream);

/*
 * The verification step (Sec. 4.5): forward + acceptance, returns L and the extra token.
 *   tokens        DEVICE int32 [sum(prefill_len+gamma+1)]: per request the prompt tokens
 *                 (prefill_len of them), root, y_1..y_gamma; M below = sum(gamma+1)
 *   draft_probs   DEVICE fp32 [sum gamma][vocab]: q_j rows, request-major (finite, >= 0)
 *   rng_seed      keys every random draw (Philox4x32-10, Salmon et al. SC'11): the
 *                 acceptance draw of draft j uses counter (0, j, req_id, 1), word 0; the
 *                 race over token k on logits row r uses counter (k/4, r, req_id, 2), word
 *                 k%4; key = (lo32, hi32) of rng_seed; a word w maps to the uniform
 *                 (2 * (w >> 9) + 1) * 2^-24 in (0, 1).  Vary the seed between rounds.
 *   accept_len    DEVICE int32 [B]: L_i = R_i - 1 (Eq. (2))
 *   out_tokens    DEVICE int32 [M]: request i's slots hold y_1..y_L, the extra token, then -1
 *   target_logits DEVICE fp32 [M][vocab]: the target's logits of every verification row
 *                 (root .. y_gamma of each request; prompt rows produce none), or NULL: the
 *                 logits then live in the workspace, which must hold
 *                 wisp_workspace_size + wisp_logits_workspace_size bytes
 *   workspace     DEVICE scratch of >= wisp_workspace_size() bytes; its first 256 bytes
 *                 hold the fault record and must be zero before the first use (wisp_check)
 * KV: K/V of all prefill_len+gamma+1 new positions are written in place (rejected
 * drafts included); the valid prefix afterwards is ctx_len + prefill_len + 1 + L and
 * later calls overwrite the stale slots (rollback by length).  Repeating a call with the same inputs gives
 * the same outputs.  Extra tokens are drawn by an exponential race (Gumbel-max):
 * argmax_k [score_k - ln(-ln u_k)], ties to the smallest k, score = ln(residual) after
 * a rejection (or z = logits/T when the residual is empty), z after full acceptance.
 * Device-side input faults (token id outside [0, vocab), block id outside
 * [0, n_blocks)) are recorded in the workspace (sticky across calls) and reported by
 * wisp_check().
 * Batches of more than WISP_ROWS_MAX rows, or whose contexts would need more than 2^22
 * split-KV work items (about 2^22 x 1024 tokens summed over requests, kv heads and
 * 48-row groups), return WISP_E_UNSUPPORTED; the workspace sizes are then 0.
 */
wisp_status wisp_verify(const wisp_model *model, const wisp_kv *kv, const wisp_batch_desc *desc,
                        const int32_t *tokens, const float *draft_probs, uint64_t rng_seed,
                        int32_t *accept_len, int32_t *out_tokens, float *target_logits,
                        void *workspace, size_t workspace_bytes, void *stream);

/*
 * wisp_verify for callers that cannot allocate: code under HIP graph capture, serving loops
 * and harnesses that forbid hipMalloc.  It takes no workspace: the step's scratch is a
 * static array of WISP_NOALLOC_SCRATCH_BYTES that every GPU the library runs on holds
 * until the process ends, and the batch descriptor reaches the device as kernel arguments
 * (no pinned staging).  It calls no hipMalloc, hipFree or other allocating HIP routine (its
 * host-side planning uses ordinary heap memory).  Same inputs, outputs, kernels and results
 * as wisp_verify, plus:
 *   fault   DEVICE int32 [1] or NULL: device-side input faults are OR-ed into it (1: a token
 *           id outside [0, vocab), 2: a block id outside [0, n_blocks)); the caller zeroes it
 *           and reads it after synchronising.  With NULL, faults go unreported.
 * A batch whose scratch (wisp_workspace_size, plus wisp_logits_workspace_size when
 * target_logits is NULL) exceeds WISP_NOALLOC_SCRATCH_BYTES returns WISP_E_WORKSPACE before
 * any GPU work.  Every call on one GPU shares that GPU's array: calls that overlap on it
 * (other streams, other threads) race and must be serialised by the caller.
 */
#define WISP_NOALLOC_SCRATCH_BYTES (128u << 20)
wisp_status wisp_verify_noalloc(const wisp_model *model, const wisp_kv *kv, const wisp_batch_desc *desc,
                                const int32_t *tokens, const float *draft_probs, uint64_t rng_seed,
                                int32_t *accept_len, int32_t *out_tokens, float *target_logits, int32_t *fault,
                                void *stream);

/*
 * The acceptance stage alone (Sec. 2.4, Eq. (1)-(3) with the residual), on given
 * logits: the same kernels and random streams as wisp_verify's last stage.
 * Uses desc->B, gamma, req_id, temperature only.  logits DEVICE fp32 [M][vocab].
 */
size_t wisp_accept_workspace_size(const wisp_batch_desc *desc, int32_t vocab);
wisp_status wisp_accept(const wisp_batch_desc *desc, int32_t vocab, const float *logits,
                        const int32_t *tokens, const float *draft_probs, uint64_t rng_seed,
                        int32_t *accept_len, int32_t *out_tokens, void *workspace,
                        size_t workspace_bytes, void *stream);

/*
 * The attention of the step on its own, for one layer's pools (the causal attention
 * of the new rows over each request's paged KV inside Sec. 4.5's forward):
 *   q   DEVICE [M][n_q_heads][head_dim] of model->dtype (already rotated)
 *   out DEVICE [M][n_q_heads][head_dim] of model->dtype
 * kv->k_pool / v_pool point at that layer's [n_blocks] pages.  Row j of request i sees
 * keys 0 .. ctx_len[i] + j.  Workspace: wisp_workspace_size() of the same batch.
 */
wisp_status wisp_attention(const wisp_model *model, const wisp_kv *kv, const wisp_batch_desc *desc,
                           const void *q, void *out, void *workspace, size_t workspace_bytes,
                           void *stream);

/* Uniform draws of the step's random stream: out[k] = draw (seed, req_id, tag, row, k),
 * k < n (DEVICE fp32).  tag 1 = acceptance, 2 = race. */
wisp_status wisp_uniform(uint64_t rng_seed, uint32_t req_id, uint32_t tag, uint32_t row, uint32_t n,
                         float *out, void *stream);

/* Synchronise `stream`, then report (and clear) the device-side input faults recorded in
 * `workspace` since it was last cleared.  The record (the workspace's first 256 bytes) is
 * sticky: wisp_verify, wisp_accept and wisp_attention only add to it, so faults of several
 * calls on one workspace are all reported by the next wisp_check.  A new workspace's first
 * 256 bytes must be zero before its first use (hipMemset after allocation). */
wisp_status wisp_check(void *workspace, void *stream);

/*
 * Opt-in timing of wisp_verify's kernels by kernel (instrumentation for benchmarks; off by
 * default, process-wide, not thread-safe).  While enabled, each launch of a class gets a
 * pair of HIP events on the caller's stream that the runtime stamps with the dispatch's own
 * begin and end, and the class accumulates the measured milliseconds, the launch count and
 * the algorithmic bytes / flops of its launches:
 *   GEMM classes: the weights, 2 (bf16) or 4 (fp32) bytes x N*K, read once per step;
 *   ATTN: K and V bytes of every token each kv head reads (ctx_len + gamma + 1 per request);
 *   SAMPLER: two passes over the fp32 logits plus one row per request;
 *   ATTN_COMBINE, ROWS: none (overhead kernels).
 * wisp_profile_read synchronises on the recorded events.  The profiling state is one per
 * process: enable, read and reset it from one thread, while no other thread calls the
 * library.
 */
#define WISP_PROF_GEMM_RING1 0   /* gemm_ring_kernel, one 32-column fragment per wave (4 or 8 waves) */
#define WISP_PROF_GEMM_RING2 1   /* gemm_ring_kernel, two 32-column fragments per wave  */
#define WISP_PROF_GEMM_TILED 2   /* the fp32 GEMM                                        */
#define WISP_PROF_ATTN 3         /* attn_bf16_kernel / attn_f32_kernel                   */
#define WISP_PROF_ATTN_COMBINE 4 /* attn_combine_kernel                                  */
#define WISP_PROF_ROWS 5         /* embedding, norms, RoPE + KV append, SwiGLU           */
#define WISP_PROF_SAMPLER 6      /* acceptance kernels                                    */
#define WISP_PROF_GEMM_TILE 7    /* gemm_tile_kernel, LDS-staged output tiles (>= 161 rows) */
#define WISP_PROF_KINDS 8
wisp_status wisp_profile_enable(int on);
wisp_status wisp_profile_read(int kind, double *ms, int64_t *launches, double *bytes, double *flops);
wisp_status wisp_profile_reset(void);

/*
 * Launch plan of one bf16 projection of the step (host only; introspection for tests and
 * benchmarks): M rows, N output columns, K inputs.  out[0] = kernel variant (1: 32-column
 * weight ring, 2: 64-column weight ring, 3: 32-column weight ring with two waves per SIMD,
 * 4: LDS-staged output tiles, from 161 rows), out[1] = row blocks (row tiles),
 * out[2] = 32-row fragments per row block, out[3] = K ranges whose fp32 partial sums are
 * added in fixed order.  WISP_E_INVALID for M, N or K < 1, or N and
 * K not multiples of 32 and 16.
 */
wisp_status wisp_gemm_plan(int32_t M, int32_t N, int32_t K, int32_t out[4]);

/*
 * Verification batch scheduling (Sec. 4.3, Alg. 1), host code.
 *
 * Batch-time estimator of Sec. 4.4 (seconds):
 *   T(B) = a * N_linear + b_compute * N_interactions + b_read * N_cached + c,
 *   N_linear = sum L_new, N_interactions = sum (L_cached + L_new) * L_new,
 *   N_cached = sum L_cached over the requests of B.
 * A pending request carries its deadline d_i = a_i + tau_c(i) (Sec. 4.3, with the
 * server budget tau of the class), its expected verified tokens g_i = alpha_i * N_d,i
 * (the verified-token estimate of Sec. 3), its memory footprint m_i and its L_cached,
 * L_new.  Its verification cost is v_i = T({i}), its utility U_i = g_i / v_i and its
 * latest start time LST_i = d_i - v_i - guard (Sec. 4.3).
 *
 * wisp_schedule picks the batch dispatched at time t_now from the n pending requests:
 *   WISP_SCHED_SLO  Alg. 1: requests with t_now >= LST_i ("critical") in increasing d_i,
 *                   then the others in decreasing U_i (ties: lower index first), each
 *                   admitted while the batch stays feasible (sum m <= mem_budget and
 *                   t_now + T(batch) <= min d over the batch); the first infeasible
 *                   admission ends the batch, and a critical one also skips the others.
 *                   A request with t_now + v_i > d_i has lost its deadline already: it
 *                   keeps its place in deadline order and counts against memory, but its
 *                   d_i is left out of the min (as printed, it would end every batch
 *                   before any admission and the queue would stall).  A request whose
 *                   m_i alone exceeds mem_budget is never admitted: the caller turns it
 *                   away.
 *   WISP_SCHED_FCFS requests in increasing arrival time (ties: lower index first) while
 *                   sum m <= mem_budget (the scheduler disabled: no deadline test).
 *   WISP_SCHED_SLO_LIVE  as WISP_SCHED_SLO, except that a request whose deadline is lost
 *                   already is not critical: it joins the utility fill (an ablation of
 *                   the reading above, for comparison).
 * batch receives the chosen request indices in admission order (capacity n), batch_len
 * their count (0 when nothing fits).  Errors: WISP_E_INVALID for NULL pointers, n < 0, an
 * unknown policy or a request with l_new < 1 or ctx_len < 0.
 */
typedef struct {
  double a, b_compute, b_read, c;
} wisp_latency_model;

typedef struct {
  double arrival;   /* a_i, seconds                                                           */
  double deadline;  /* d_i, seconds (same clock)                                              */
  double g_hat;     /* expected verified tokens                                               */
  double m_hat;     /* memory footprint, in the unit of mem_budget                            */
  int32_t ctx_len;  /* L_cached                                                               */
  int32_t l_new;    /* L_new (prompt rows + root + drafts)                                    */
} wisp_sched_request;

#define WISP_SCHED_SLO 0
#define WISP_SCHED_FCFS 1
#define WISP_SCHED_SLO_LIVE 2
wisp_status wisp_schedule(int32_t policy, const wisp_sched_request *requests, int32_t n, double t_now,
                          double mem_budget, double guard, const wisp_latency_model *model,
                          int32_t *batch, int32_t *batch_len);

/*
 * KV page-pool manager for multi-round sessions (Sec. 4.5: each round forwards only the
 * newly drafted block and updates the session's KV in place, the committed prefix staying
 * cached across rounds), host code.  It hands out the page ids that the page tables of
 * wisp_batch_desc hold; the pool memory itself (wisp_kv) belongs to the caller.  Not
 * thread-safe: one manager per thread, or external locking.
 *
 * Sessions are caller-chosen int64 ids.  Pages are given out lowest id first.
 *   wisp_kvm_lookup   cached[i] = tokens whose KV is held for sid[i]; 0 for a session the
 *                     manager does not hold (new, released or evicted), whose owner must
 *                     then send its whole sequence as prefill (ctx_len = 0).
 *   wisp_kvm_reserve  makes each sid[i] (created if new) hold pages for n_tokens[i]
 *                     positions, n_tokens[i] >= its cached tokens (a round reserves
 *                     ctx_len + prefill_len + gamma + 1), and writes its page ids to
 *                     page_table[i * pt_stride ..], -1 past its last page.  When the free
 *                     pages do not suffice, sessions outside the call are evicted least
 *                     recently used first (ties: smaller id).  On WISP_E_CAPACITY (the
 *                     pool cannot hold the call even after evicting every other session,
 *                     or a row of pt_stride is too short) nothing changes.  *n_evicted
 *                     (may be NULL) = sessions this call evicted.
 *   wisp_kvm_commit   rollback by length: sid[i] keeps the KV of its first cached[i]
 *                     tokens (at most the positions reserved); whole pages past them
 *                     return to the pool.  A round commits ctx_len + prefill_len + L + 1
 *                     (prompt rows, root and accepted drafts; the extra token is the next
 *                     round's root).  Commit a round before reserving the next batch: a
 *                     session evicted in between cannot be committed (WISP_E_INVALID).
 *   wisp_kvm_release  forgets the sessions and frees their pages (unknown ids ignored).
 * reserve and commit mark their sessions as used (one clock tick per call).  Errors:
 * WISP_E_INVALID for NULL pointers, n < 0, a session twice in one call, n_tokens below
 * the cached tokens, or a commit outside the reserved pages; WISP_E_HOST_MEMORY when the
 * manager's host bookkeeping cannot grow (the manager is then only fit for destroy).
 */
typedef struct wisp_kv_manager wisp_kv_manager;

typedef struct {
  int32_t n_pages, free_pages, sessions;       /* pool size, free pages, resident sessions  */
  int64_t evictions, pages_evicted;            /* sessions evicted, their pages              */
  int64_t pages_allocated, pages_freed;        /* by reserve; by commit and release          */
  int64_t lookup_hits, lookup_misses;          /* lookups that found cached tokens, or none  */
} wisp_kvm_stats;

wisp_status wisp_kvm_create(int32_t n_pages, int32_t page_size, wisp_kv_manager **out);
void wisp_kvm_destroy(wisp_kv_manager *m);
wisp_status wisp_kvm_lookup(wisp_kv_manager *m, const int64_t *sid, int32_t n, int32_t *cached);
wisp_status wisp_kvm_reserve(wisp_kv_manager *m, const int64_t *sid, const int32_t *n_tokens, int32_t n,
                             int32_t *page_table, int32_t pt_stride, int32_t *n_evicted);
wisp_status wisp_kvm_commit(wisp_kv_manager *m, const int64_t *sid, const int32_t *cached, int32_t n);
wisp_status wisp_kvm_release(wisp_kv_manager *m, const int64_t *sid, int32_t n);
wisp_status wisp_kvm_get_stats(const wisp_kv_manager *m, wisp_kvm_stats *out);

/*
 * Draft-side rejection predictor (Sec. 3.3, Sec. 4.1, App. B): statistics of the draft
 * model's next-token distribution, and the MLP (hidden widths 512, 128, 64) that turns
 * them into the probability that the drafted token is accepted; the drafting controller
 * stops drafting at the first predicted rejection.
 *
 * wisp_draft_stats: for each of `rows` rows of DEVICE fp32 logits (row r at logits + r*ld,
 *   `vocab` finite entries, ld >= vocab), with z = logits / temperature and p = softmax(z),
 *   writes DEVICE fp32 stats[r][4] = (confidence max_k p_k, entropy -sum p ln p (nats),
 *   top-2 margin p_(1) - p_(2) (0 when the maximum repeats, p_(1) when vocab = 1),
 *   dispersion: the population standard deviation of z).  stats and workspace (DEVICE,
 *   wisp_draft_stats_workspace_size bytes: per-chunk partial sums) must be 16-byte aligned.
 * wisp_reject_predict: for each of `rows` feature rows (DEVICE fp32 [rows][n_in]), with
 *   x = (f - mean) * inv_std, writes DEVICE fp32 p_accept[r] =
 *   sigmoid(w4 . relu(W3 relu(W2 relu(W1 x + b1) + b2) + b3) + b4).  The features are the
 *   four statistics above, optionally followed by caller-chosen ones (the draft position,
 *   say); all weights are DEVICE fp32, row-major [out][in], w2 16-byte and w3 8-byte
 *   aligned.  At most 65535 rows per wisp_draft_stats call (WISP_E_UNSUPPORTED beyond).
 * Errors: WISP_E_INVALID for NULL pointers, rows < 0, vocab < 1, ld < vocab,
 * temperature <= 0 or n_in outside 1..8; WISP_E_WORKSPACE for a short workspace.  Both only
 * enqueue work on `stream`.
 */
typedef struct {
  int32_t n_in;                  /* features per row, 1..8                                 */
  const float *mean, *inv_std;   /* DEVICE [n_in] input standardisation                    */
  const float *w1, *b1;          /* DEVICE [512][n_in], [512]                              */
  const float *w2, *b2;          /* DEVICE [128][512], [128]                               */
  const float *w3, *b3;          /* DEVICE [64][128], [64]                                 */
  const float *w4;               /* DEVICE [64]                                            */
  float b4;
} wisp_reject_mlp;

size_t wisp_draft_stats_workspace_size(int32_t rows, int32_t vocab);
wisp_status wisp_draft_stats(const float *logits, int32_t rows, int32_t vocab, int64_t ld, float temperature,
                             float *stats, void *workspace, size_t workspace_bytes, void *stream);
wisp_status wisp_reject_predict(const wisp_reject_mlp *mlp, const float *features, int32_t rows, float *p_accept,
                                void *stream);

/* Message of the last failing call on this thread ("" if none). */
const char *wisp_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* WISP_H */
