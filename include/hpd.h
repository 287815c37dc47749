/*
 * hpd.h -- C ABI of the MI355X (gfx950) branch-parallel decode step.
 *
 * Method: "HPD-Parsing: Hierarchical Parallel Document Parsing"
 * (arXiv 2607.18839).  In one decode step the main layout branch of a page and
 * every content branch forked from it each bring k new (draft-verify) query
 * tokens.  Every branch attends over the page's shared visual + structural
 * prefix KV and over its own private (incremental) KV only, never over other
 * branches' text (section "Layout-Coordinated Parallel Decoding", paragraph
 * "Dynamic Branch Forking and Efficient Context Isolation").  The k drafts of a
 * branch are verified together in one forward, so they are causal among
 * themselves (section "Integration with P-MTP", last paragraph; Algorithm 1,
 * the parallel draft over the active pool).  The decoder is a GQA / RMSNorm /
 * SwiGLU stack (section "Overview", paragraph "LLM Decoder").
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Pure C.  No exception crosses the boundary; every call returns an
 *    hpd_status and never aborts.  hpd_last_error_message() gives a
 *    thread-local description of the last non-OK status of the calling thread.
 *  - "Host" pointers are ordinary CPU memory, read only during the call.
 *    "Device" pointers are GPU memory owned by the caller; the library never
 *    allocates or frees device memory and never synchronises a stream.
 *  - Streams are passed as `void *stream`, a hipStream_t (NULL = the null
 *    stream).  Work is enqueued in stream order and runs asynchronously.
 *  - Validation happens before any launch: a validation error writes nothing.
 *    A HIP launch error returns HPD_ERR_HIP; outputs are then undefined.
 *  - Tensors are row-major and contiguous:
 *        q          [T][Hq][D]              token t = j-th new token of branch b
 *                                            at t = q_row[b] + j
 *        shared_k/v [shared rows][Hkv][D]   page p's prefix at rows
 *                                            prefix_row[p] .. + P_p - 1
 *        priv_k/v   [private rows][Hkv][D]  branch b's rows at priv_row[b] ..
 *                                            + L_b + k_b - 1: its L_b past
 *                                            tokens, then its k_b new tokens
 *        out        [T][Hq][D]              out_dtype
 *        lse        [T][Hq] float           natural-log log-sum-exp of the
 *                                            scaled scores (nullable)
 *    Query head h uses KV head h / (Hq / Hkv) (contiguous GQA groups).
 *  - Visibility: new token j of branch b on page p sees shared rows
 *    0 .. F_b - 1 of page p (F_b = P_p unless fork_len is given) and private
 *    rows 0 .. L_b + j of branch b (bottom-right causal among the drafts).
 */
#ifndef HPD_H
#define HPD_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define HPD_MAX_K 16        /* new tokens per branch per step (draft window) */
#define HPD_HEAD_DIM 64     /* the only supported head dimension */
#define HPD_MAX_Q_HEADS 64
#define HPD_MAX_GROUP 32    /* Hq / Hkv */

typedef enum {
  HPD_OK = 0,
  HPD_ERR_INVALID_ARGUMENT = 1,
  HPD_ERR_UNSUPPORTED = 2,
  HPD_ERR_WORKSPACE_TOO_SMALL = 3,
  HPD_ERR_HIP = 4,
  HPD_ERR_HOST_ALLOC = 5,
  HPD_ERR_OUT_OF_BLOCKS = 6
} hpd_status;

typedef enum { HPD_F32 = 0, HPD_BF16 = 1 } hpd_dtype;

/* One attention layer's shape. */
typedef struct {
  int32_t num_q_heads;   /* Hq, 1..HPD_MAX_Q_HEADS, Hq % Hkv == 0            */
  int32_t num_kv_heads;  /* Hkv >= 1, Hq / Hkv <= HPD_MAX_GROUP               */
  int32_t head_dim;      /* D; must be HPD_HEAD_DIM, else HPD_ERR_UNSUPPORTED */
  float softmax_scale;   /* <= 0 selects 1 / sqrt(D)                          */
  int32_t dtype;         /* hpd_dtype of q, shared_k/v, priv_k/v              */
  int32_t out_dtype;     /* hpd_dtype of out                                  */
} hpd_attn_desc;

/* Paged K/V (the paged-KV memory model of the inference workflow: section
 * "Inference Workflow", Algorithm 1, where a forked branch shares its page's
 * prefix by reference and keeps only its own incremental KV).  K and V rows
 * live in blocks of block_rows rows of a pool: shared_k/v and priv_k/v are
 * then the pool bases ([num_blocks * block_rows][Hkv][D]; the same pool may
 * be passed for both).  Row i of page p's prefix is pool row
 * blocks[page_block0[p] + i / block_rows] * block_rows + i % block_rows, and
 * row i of branch b's private rows (its L_b past rows, then its k_b new rows)
 * likewise from branch_block0[b].  Page p uses ceil(P_p / block_rows) entries
 * of `blocks`, branch b ceil((L_b + k_b) / block_rows).  HOST arrays, read
 * only inside hpd_plan_create.  hpd_kv_pool below manages such blocks. */
typedef struct {
  int32_t block_rows;            /* rows per block, a positive multiple of 64  */
  int32_t num_blocks;            /* blocks in the pool(s); ids 0..num_blocks-1 */
  int32_t num_entries;           /* length of `blocks`                         */
  const int32_t *blocks;         /* [num_entries] block ids                    */
  const int32_t *page_block0;    /* [num_pages] first entry of page p          */
  const int32_t *branch_block0;  /* [num_branches] first entry of branch b     */
} hpd_paged_kv;

/* A ragged batch of pages and branches.  HOST arrays, read only inside
 * hpd_plan_create.  Branches are grouped by page (branch_page non-decreasing);
 * within a page the layout branch conventionally comes first. */
typedef struct {
  int32_t num_pages;          /* >= 1                                          */
  const int32_t *prefix_len;  /* [num_pages] P_p >= 0                          */
  const int64_t *prefix_row;  /* [num_pages] first shared row of page p;
                                 NULL = packed (exclusive prefix sum of P_p)   */
  int32_t num_branches;       /* >= 1                                          */
  const int32_t *branch_page; /* [nb] page of branch b, non-decreasing         */
  const int32_t *num_new;     /* [nb] k_b in 1..HPD_MAX_K                      */
  const int32_t *past_len;    /* [nb] L_b >= 0 (excludes the k_b new tokens)   */
  const int64_t *priv_row;    /* [nb] first private row of branch b;
                                 NULL = packed (exclusive sum of L_b + k_b)    */
  const int32_t *fork_len;    /* [nb] visible prefix F_b in 0..P_p; NULL = P_p */
  const hpd_paged_kv *paged;  /* NULL = contiguous rows (prefix_row, priv_row);
                                 else paged K/V, prefix_row and priv_row NULL  */
} hpd_batch_desc;

/* Opaque, immutable execution plan: the canonical ragged bookkeeping (row
 * offsets, visible-key counts) plus the work lists of the three attention
 * kernels and the layout of their scratch partials.  Host memory. */
typedef struct hpd_plan hpd_plan;

/* Integer bookkeeping of a plan, for inspection and bit-exact tests.  The
 * arrays point into the plan and live as long as it does. */
typedef struct {
  int32_t num_tokens;             /* T = sum k_b                               */
  int32_t num_pages, num_branches;
  const int32_t *q_row;           /* [nb] first token of branch b              */
  const int64_t *priv_row;        /* [nb] first private row of branch b        */
  const int64_t *prefix_row;      /* [num_pages] first shared row of page p    */
  const int32_t *page_q_row;      /* [num_pages] first token of page p         */
  const int32_t *page_T;          /* [num_pages] tokens of page p              */
  const int32_t *visible;         /* [T] keys seen by token t: F_b + L_b + j + 1 */
  int64_t shared_rows;            /* rows shared_k/v must hold (max end row;
                                     paged: the pool, num_blocks * block_rows) */
  int64_t priv_rows;              /* rows priv_k/v must hold (likewise)        */
  int32_t num_shared_items;       /* work items of the shared-prefix kernel    */
  int32_t num_private_items;      /* work items of the private kernel          */
  const int32_t *shared_items;    /* [num_shared_items][12] fields: csrc/plan.h  */
  const int32_t *private_items;   /* [num_private_items][12] fields: csrc/plan.h */
  const int32_t *token_slots;     /* [T][2] first partial slot, slot count     */
  int64_t num_partial_slots;      /* partial (O, lse) rows = slots * Hq        */
  const int32_t *pos_token;       /* [T][2] (token, visible prefix F_b) held by
                                     stacked position i of the shared-prefix
                                     items: a page's positions are page_q_row[p]
                                     .. + page_T[p] - 1, and its stacked row r
                                     (per kv head) is query head g * G + r % G
                                     of position page_q_row[p] + r / G.  Without
                                     fork offsets position i holds token i; with
                                     them a page's tokens are ordered by
                                     descending F_b (ties: token order)        */
} hpd_plan_info;

/* Build a plan: validates the descriptors (see each field above), computes
 * the bookkeeping and the work lists.  On success *out owns a new plan that
 * the caller releases with hpd_plan_destroy. */
hpd_status hpd_plan_create(const hpd_attn_desc *attn, const hpd_batch_desc *batch,
                           hpd_plan **out);
void hpd_plan_destroy(hpd_plan *plan);

/* Bytes of device workspace a step with this plan needs (work lists + the
 * fp32 partials of the split softmax).  The workspace is caller-owned, at
 * least 256-byte aligned, and must not be shared by steps that overlap. */
size_t hpd_plan_workspace_bytes(const hpd_plan *plan);

hpd_status hpd_plan_query(const hpd_plan *plan, hpd_plan_info *out);

/* Copy the plan's work lists into the device workspace (asynchronous on
 * `stream`).  Must precede the first step that uses this (plan, workspace)
 * pair; the tables stay valid until the caller overwrites the workspace. */
hpd_status hpd_plan_upload(const hpd_plan *plan, void *workspace, size_t workspace_bytes,
                           void *stream);

/* One attention layer of the branch-parallel decode step.
 *
 * Computes, for every new token of every branch and every query head, softmax
 * attention over the branch's visible keys (see the conventions above) as
 * three kernels: (1) the shared-prefix kernel stacks the query rows of all
 * branches of a page that share a KV head into MFMA tiles, so each prefix K/V
 * tile is read once per page and KV head; (2) the private kernel attends each
 * branch's ragged private rows with the bottom-right causal mask; (3) the
 * log-sum-exp merge combines all partial softmaxes into out and lse.
 *
 * q, shared_k, shared_v, priv_k, priv_v: device, attn->dtype, layouts above.
 *   shared_k/v may be NULL only if every P_p is 0.
 * out: device [T][Hq][D] in attn->out_dtype.  lse: device [T][Hq] or NULL.
 * workspace: device, >= hpd_plan_workspace_bytes, uploaded with
 *   hpd_plan_upload.  The step reads only the rows the plan names. */
hpd_status hpd_branch_attn_step(const hpd_plan *plan, const void *q, const void *shared_k,
                                const void *shared_v, const void *priv_k, const void *priv_v,
                                void *out, float *lse, void *workspace, size_t workspace_bytes,
                                void *stream);

/* hpd_branch_attn_step for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): no workspace argument and no allocation.  The step's scratch
 * (the plan's tables, then the partial softmax results) lives in a static
 * array of HPD_NOALLOC_SCRATCH_BYTES inside the library, one per GPU, held
 * until the process ends; each call copies the plan's tables into it
 * (stream-ordered, from the plan's host memory) and runs the same kernels
 * as hpd_branch_attn_step, so the results are bit-identical to it.  No
 * hpd_plan_upload is needed.
 * Plans whose hpd_plan_workspace_bytes exceed HPD_NOALLOC_SCRATCH_BYTES
 * return HPD_ERR_WORKSPACE_TOO_SMALL before anything is enqueued.
 * All calls on one GPU share its array and the array keeps the last call's
 * contents: calls that may overlap on one GPU (different streams, or
 * different host threads without ordering) race; serialise them on one
 * stream.  Other arguments and errors as hpd_branch_attn_step. */
#define HPD_NOALLOC_SCRATCH_BYTES (32u << 20)
hpd_status hpd_branch_attn_step_noalloc(const hpd_plan *plan, const void *q, const void *shared_k,
                                        const void *shared_v, const void *priv_k, const void *priv_v,
                                        void *out, float *lse, void *stream);

/* The synthetic decoder stack (pre-norm GQA transformer with RMSNorm and a
 * SwiGLU MLP, section "Overview", paragraph "LLM Decoder").  Weights are bf16
 * device arrays in torch Linear layout W[out][in]; each field points to a
 * HOST array of num_layers device pointers, each 16-byte aligned. */
typedef struct {
  int32_t num_layers;           /* >= 1                                        */
  int32_t hidden;               /* positive multiple of 128                    */
  int32_t intermediate;         /* positive multiple of 128                    */
  float rms_eps;                /* RMSNorm epsilon, 0..1                       */
  const void *const *w_qkv;     /* [L] -> [(Hq + 2 Hkv) D][hidden]: q rows, then k, then v */
  const void *const *w_o;       /* [L] -> [hidden][Hq D]                       */
  const void *const *w_gate;    /* [L] -> [intermediate][hidden]               */
  const void *const *w_up;      /* [L] -> [intermediate][hidden]               */
  const void *const *w_down;    /* [L] -> [hidden][intermediate]               */
  const void *const *g_attn_norm; /* [L] -> [hidden] bf16 RMSNorm gain; NULL = ones */
  const void *const *g_mlp_norm;  /* [L] -> [hidden] bf16 RMSNorm gain; NULL = ones */
  int32_t weight_format;        /* hpd_weight_format; 0 = HPD_WEIGHTS_TORCH      */
  /* Qwen3-style attention inputs (optional; NULL / 0 = off, the plain stack
   * above).  The "Overview" section names Qwen3-0.6B as the decoder's base;
   * its attention normalises each head's q and k and rotates them by
   * position.  q_norm, k_norm: [L] -> [64] bf16 gains of an RMSNorm (epsilon
   * rms_eps) over each head's 64 q (k) values after the projection.
   * rope_theta > 0: rotary position embedding after the norm, dims i and
   * i + 32 of a head rotated by the angle pos * rope_theta^(-i / 32)
   * (x_i, x_{i+32}) -> (x_i cos - x_{i+32} sin, x_{i+32} cos + x_i sin), pos
   * = F_b + L_b + j, the token's position in its branch's sequence.  The
   * shared and past K rows are taken as already normalised and rotated. */
  const void *const *q_norm;
  const void *const *k_norm;
  float rope_theta;
} hpd_model_desc;

/* Layout of the projection weights of an hpd_model_desc.
 * HPD_WEIGHTS_TORCH: the layouts above (torch Linear, W[out][in], bf16).
 * HPD_WEIGHTS_PACKED: every projection packed once: w_qkv and w_o with
 *   hpd_pack_weight, w_down with hpd_pack_weight_f16, and the gate/up pair
 *   with hpd_pack_gate_up (w_gate points to it; w_up is ignored and may be
 *   NULL).  The decode step then reads each weight tile with whole
 *   contiguous 1 KB loads per wave, and the MLP weights already in the fp16
 *   its MLP projections compute in (the same values the torch layout is
 *   converted to on the fly, so both formats give identical results). */
typedef enum { HPD_WEIGHTS_TORCH = 0, HPD_WEIGHTS_PACKED = 1 } hpd_weight_format;

/* Packed layout of a bf16 matrix W[rows][cols] (rows % 32 == 0, cols % 64
 * == 0): tiles of 32 rows x 64 columns, 4096 bytes each, ordered by row tile
 * then column tile; inside a tile, 16-byte piece (j, l) for j = 0..3 and
 * l = 0..63 sits at byte 1024 j + 16 l and holds row 32 r + l % 32, columns
 * 64 c + 32 (l / 32) + 8 j .. + 7 of tile (r, c).  The packed matrix has the
 * same size as W: hpd_packed_weight_bytes(rows, cols) = rows * cols * 2.
 * w: device [rows][cols] bf16; out: device buffer of that size (not
 * overlapping w), 16-byte aligned.  Stream-ordered; HPD_ERR_INVALID_ARGUMENT
 * for NULL pointers or bad sizes, HPD_ERR_HIP if the launch fails. */
size_t hpd_packed_weight_bytes(int32_t rows, int32_t cols);
hpd_status hpd_pack_weight(const void *w, int32_t rows, int32_t cols, void *out, void *stream);

/* As hpd_pack_weight, with every element converted from bf16 to fp16
 * (round to nearest even; fp16 subnormals below 2^-14, 0 below 2^-25; the
 * bf16 inputs of a decoder stay far inside the fp16 range). */
hpd_status hpd_pack_weight_f16(const void *w, int32_t rows, int32_t cols, void *out, void *stream);

/* Packed gate/up pair of a SwiGLU MLP: w_gate, w_up are device
 * [intermediate][hidden] bf16 (intermediate % 16 == 0, hidden % 64 == 0);
 * out (hpd_packed_weight_bytes(2 intermediate, hidden) bytes) holds the
 * packed [2 intermediate][hidden] fp16 matrix (converted as in
 * hpd_pack_weight_f16) whose row tile r is gate rows 16 r .. 16 r + 15
 * followed by up rows 16 r .. 16 r + 15 (so a row tile computes 16 gate
 * and their 16 up outputs together). */
hpd_status hpd_pack_gate_up(const void *w_gate, const void *w_up, int32_t intermediate, int32_t hidden,
                            void *out, void *stream);

/* Bytes of device workspace hpd_decode_step needs on top of
 * hpd_plan_workspace_bytes (activations of the T tokens and per-token
 * sums of squares for the folded RMSNorm). */
size_t hpd_decode_workspace_bytes(const hpd_model_desc *model, const hpd_plan *plan);

/* One full decode step of the decoder stack for every new token of every
 * branch.  For each layer l: x = RMSNorm(h); [q|k|v] = x W_qkv^T; k and v are
 * rounded to bf16 and written into private rows priv_row[b] + L_b + j of
 * priv_k[l] / priv_v[l] (no other row is written); a = attention as in
 * hpd_branch_attn_step; h += a W_o^T; x = RMSNorm(h);
 * h += (silu(x W_gate^T) * (x W_up^T)) W_down^T.
 * hidden_in, hidden_out: device float [T][hidden], 16-byte aligned; the
 *   step copies hidden_in to hidden_out first and then updates hidden_out
 *   in place (they may be the same buffer).
 * shared_k/v, priv_k/v: HOST arrays of num_layers device pointers (bf16,
 *   16-byte aligned) in the layouts of hpd_branch_attn_step.
 * The plan's dtype and out_dtype must be HPD_BF16 and Hq * 64 a multiple of
 * 128 (else HPD_ERR_UNSUPPORTED).
 * workspace: >= hpd_plan_workspace_bytes + hpd_decode_workspace_bytes,
 *   256-byte aligned, uploaded with hpd_plan_upload.
 * Numerics: weights bf16; q, k, v, the attention output and the attention
 * input norm enter their products as bf16; the MLP projections run in fp16
 * (the bf16 weights convert exactly, the MLP input norm and the SwiGLU
 * product are rounded to fp16); all accumulation and the residual stream in
 * fp32.
 * fp16 range: the MLP input is written as h * gamma_mlp * s_t, with s_t the
 * power of two at or below the token's attention-norm factor
 * 1 / RMS(h before the attention); the gate/up projection divides by s_t
 * (both exact).  Since |h_i| <= sqrt(hidden) * RMS(h), an element stays
 * below fp16's 65504 while |gamma_mlp_i| * RMS(h after the attention) /
 * RMS(h before) < 65504 / (2 sqrt(hidden)) (1023 at hidden 1024), whatever
 * the scale of h.  The SwiGLU product silu(x W_gate^T) * (x W_up^T) of the
 * normalised input must itself stay below 65504 in magnitude.  Past either
 * bound the step's outputs become inf or NaN (no error is returned). */
hpd_status hpd_decode_step(const hpd_model_desc *model, const hpd_plan *plan,
                           const float *hidden_in, float *hidden_out,
                           const void *const *shared_k, const void *const *shared_v,
                           void *const *priv_k, void *const *priv_v,
                           void *workspace, size_t workspace_bytes, void *stream);

/* ---- P-MTP verification and drafting (section "Integration with P-MTP";
 * Algorithm 1, speculative decoding and verification).  After a decode step
 * the k_b hidden states of branch b are projected through the LM head: the
 * token fed at position j (tokens_in: position 0 is the branch's last
 * accepted token, positions 1.. its drafts) is verified against the argmax at
 * position j - 1, and the branch accepts its longest verified prefix of
 * drafts, n_acc.  The argmax y* at the first unverified position is the
 * step's bonus token and the first token of the next step's window; the
 * small residual MLP then drafts the rest of the window from that
 * position's hidden state: f <- f + SwiGLU(RMSNorm([f ; embed(token)]))
 * W_down^T, next token = argmax of the LM head on RMSNorm(f), as often as
 * the branch's window needs.
 *
 *  vocab            V, a positive multiple of 128
 *  draft_inner      I_d, inner width of the draft MLP, a multiple of 128
 *  lm_head          [V][hidden] bf16, packed with hpd_pack_weight (shared by
 *                   verification and drafting)
 *  g_final          [hidden] bf16 gain of the RMSNorm before the LM head;
 *                   NULL = ones
 *  embed            [V][hidden] bf16 token embedding, row-major
 *  w_draft_gate_up  gate/up of the draft MLP, [I_d][2 hidden] each, packed
 *                   with hpd_pack_gate_up
 *  w_draft_down     [hidden][I_d], packed with hpd_pack_weight_f16
 *  window           tokens of the next window of every branch (the bonus
 *                   token and window - 1 drafts), 0..HPD_MAX_K; 0 = the
 *                   plan's largest k_b.  A branch that fed fewer tokens this
 *                   step (one just started) still gets a full window.
 *
 * Argmax ties go to the smallest token id.  The LM head runs on the bf16
 * rounding of x = h * g_final; the positive per-token RMSNorm factor does not
 * change the argmax and is not applied.  All pointers 16-byte aligned. */
typedef struct {
  int32_t vocab;
  int32_t draft_inner;
  const void *lm_head;
  const void *g_final;
  const void *embed;
  const void *w_draft_gate_up;
  const void *w_draft_down;
  int32_t window;
} hpd_pmtp_desc;

/* The input of a decode step from the tokens it feeds: out[t][:] = the
 * embedding row of tokens[t] as fp32.  embed [vocab][hidden] bf16 (8-byte
 * aligned), tokens device int32 [T], out device float [T][hidden] (16-byte
 * aligned); hidden a positive multiple of 4.  An id outside 0..vocab-1
 * gives a zero row. */
hpd_status hpd_embed_tokens(const void *embed, int32_t vocab, int32_t hidden, const int32_t *tokens, int32_t T,
                            float *out, void *stream);

/* Bytes of device workspace hpd_verify_draft_step needs on top of
 * hpd_plan_workspace_bytes. */
size_t hpd_pmtp_workspace_bytes(const hpd_model_desc *model, const hpd_pmtp_desc *pmtp, const hpd_plan *plan);

/* One verification + drafting pass for every branch of the plan.
 * hidden      device float [T][hidden]: the decode step's output
 * tokens_in   device int32 [T]: the token fed at each position, ids < V
 * verified    device int32 [T]: argmax token at each position (written)
 * n_acc       device int32 [num_branches]: accepted drafts, 0..k_b - 1
 * draft_out   device int32 [num_branches][HPD_MAX_K]: the next window of
 *             branch b in entries 0..W - 1 (entry 0 the bonus token; W =
 *             pmtp->window, or the largest k_b if it is 0); later entries
 *             unspecified
 * workspace   >= hpd_plan_workspace_bytes + hpd_pmtp_workspace_bytes,
 *             256-byte aligned, uploaded with hpd_plan_upload (it may be the
 *             decode step's workspace if it is large enough for both).
 * The plan must be HPD_BF16 and the model's hidden a multiple of 256. */
hpd_status hpd_verify_draft_step(const hpd_model_desc *model, const hpd_pmtp_desc *pmtp, const hpd_plan *plan,
                                 const float *hidden, const int32_t *tokens_in, int32_t *verified,
                                 int32_t *n_acc, int32_t *draft_out, void *workspace, size_t workspace_bytes,
                                 void *stream);

/* ---- Benchmark support: per-kernel timing with HIP events.
 * When enabled, every kernel a step enqueues is launched with a pair of HIP
 * events bound to its own dispatch (hipExtLaunchKernel), so each pair spans
 * the kernel's execution, as a kernel trace reports it.  hpd_kernel_times_read
 * waits for the pairs and returns, per kernel kind, the number of launches and
 * the sum of their durations since the previous read.  The event pool
 * (max_launches pairs) is created by hpd_kernel_timing(1, n), outside any
 * timed region; launches beyond it are counted in `dropped`.  Timing is for
 * eager launches: do not enable it while capturing a graph.  keep_pairs = 1
 * keeps the pairs assigned after the read (re-read after re-running the same
 * launches); keep_pairs = 0 releases them. */
#define HPD_NUM_KERNEL_KINDS 14
typedef struct {
  int64_t count[HPD_NUM_KERNEL_KINDS];
  double total_ms[HPD_NUM_KERNEL_KINDS];
  int64_t dropped;
} hpd_kernel_times;
hpd_status hpd_kernel_timing(int enable, int max_launches);
hpd_status hpd_kernel_times_read(hpd_kernel_times *out, int keep_pairs);
/* Kind k: 0 shared_prefix, 1 private, 2 merge, 3 gemm_qkv, 4 gemm_o,
 * 5 gemm_gate_up, 6 gemm_down, 7 norm_input, 8 lm_head, 9 verify,
 * 10 draft_mlp (the draft MLP's two projections and its input),
 * 11 draft_token, 12 embed, 13 qk_norm_rope.  With bf16 inputs kind 0 is
 * one launch that runs the shared-prefix and the private work items (kind 1
 * is then never launched) unless phase isolation is on. */
const char *hpd_kernel_kind_name(int kind);

/* Phase isolation (benchmark support, process-wide, default off).  When on,
 * the bf16 attention enqueues its private work items as a launch of their
 * own (kind 1) after the shared-prefix launch (kind 0) instead of running
 * both in one launch, so each phase can be timed and profiled on its own.
 * Results are bit-identical either way.  Not to be changed while a step is
 * being enqueued or captured. */
hpd_status hpd_attn_phase_isolation(int enable);

/* Host manager of paged K/V blocks (section "Inference Workflow",
 * Algorithm 1: KV owned per request, a forked branch sharing its page's
 * prefix by reference, rejected drafts rolled back).  A pool hands out block
 * ids 0..num_blocks-1 of block_rows rows each; the device K/V pools
 * themselves are the caller's.  A sequence is either a root (a page's
 * prefix) or a branch forked from a root: the branch sees the root's first
 * fork_len rows without copying them (the root's blocks stay allocated while
 * any branch forked from it lives) and owns its private rows.  Host memory
 * only; a pool is not thread-safe.  Freed blocks are reused last-freed
 * first.
 *
 *  hpd_kv_seq_new       parent = -1: new root; else a branch of root
 *                       `parent` (a live root, not a branch) seeing its first
 *                       fork_len (0..parent length) rows.  New sequences are
 *                       empty.
 *  hpd_kv_seq_reserve   grows a sequence to new_len rows (append), taking
 *                       blocks from the pool; HPD_ERR_OUT_OF_BLOCKS, with
 *                       nothing changed, when the pool has too few.
 *  hpd_kv_seq_truncate  shrinks to new_len rows (rollback of rejected
 *                       drafts), returning whole blocks past it; a root
 *                       cannot shrink below a live branch's fork_len.
 *  hpd_kv_seq_release   ends a sequence: a branch returns its blocks; a root
 *                       returns the blocks past every live branch's fork_len
 *                       at once and the rest as the branches that see them
 *                       are released (per-block reference counting).
 *  hpd_kv_seq_info      length, block count, parent (-1 for a root) and
 *                       fork_len of a live sequence.
 *  hpd_kv_seq_blocks    copies its block ids (capacity entries at most).
 *  hpd_kv_batch_tables  fills hpd_paged_kv tables for a batch: the block ids
 *                       of each page's root (live, or released with live
 *                       branches), then of each (live) branch,
 *                       concatenated into blocks_out (capacity entries),
 *                       with page_block0_out / branch_block0_out; *entries is
 *                       the length needed (HPD_ERR_INVALID_ARGUMENT if above
 *                       capacity). */
typedef struct hpd_kv_pool hpd_kv_pool;
hpd_status hpd_kv_pool_create(int32_t num_blocks, int32_t block_rows, hpd_kv_pool **out);
void hpd_kv_pool_destroy(hpd_kv_pool *pool);
int32_t hpd_kv_pool_free_blocks(const hpd_kv_pool *pool);
hpd_status hpd_kv_seq_new(hpd_kv_pool *pool, int32_t parent, int32_t fork_len, int32_t *seq);
hpd_status hpd_kv_seq_reserve(hpd_kv_pool *pool, int32_t seq, int32_t new_len);
hpd_status hpd_kv_seq_truncate(hpd_kv_pool *pool, int32_t seq, int32_t new_len);
hpd_status hpd_kv_seq_release(hpd_kv_pool *pool, int32_t seq);
hpd_status hpd_kv_seq_info(const hpd_kv_pool *pool, int32_t seq, int32_t *len, int32_t *num_blocks,
                           int32_t *parent, int32_t *fork_len);
hpd_status hpd_kv_seq_blocks(const hpd_kv_pool *pool, int32_t seq, int32_t *blocks_out, int32_t capacity);
hpd_status hpd_kv_batch_tables(const hpd_kv_pool *pool, int32_t num_pages, const int32_t *page_seq,
                               int32_t num_branches, const int32_t *branch_seq, int32_t *blocks_out,
                               int32_t capacity, int32_t *page_block0_out, int32_t *branch_block0_out,
                               int32_t *entries);

/* ---- Host scheduler (section "Inference Workflow", Algorithm 1: FCFS
 * scheduling with hierarchical parallel decoding).
 *
 * Requests.  A parent is a page: its layout branch decodes after a prefill of
 * prompt_len rows (visual tokens and prompt, computed by the caller) that
 * also gave its first token.  When a parent emits fork_token the scheduler
 * spawns a child (a content branch) that sees the parent's rows before that
 * token by reference and starts from child_token.  Request ids count up from
 * 0 in order of submission or spawn and are also the arrival order.
 *
 * One engine iteration:
 *  hpd_sched_schedule  sorts the waiting queue when forks dirtied it
 *                      (children before parents; children by their parent's
 *                      arrival, then by more live siblings first, then by
 *                      their own arrival; parents by arrival), makes room in
 *                      the K/V pool for every active request's next step
 *                      (len + k rows), preempting the youngest active
 *                      request while that fails (its unshared blocks are
 *                      freed, its rows recomputed when it resumes, and it
 *                      goes to the front of the queue), then admits from the
 *                      queue's front: parents only while the pool's used
 *                      blocks are <= kv_threshold * num_blocks and fewer than
 *                      max_active requests are active; children regardless;
 *                      a request whose K/V does not fit stops admission.
 *                      It returns the step's batch.
 *  (the caller)        computes the prefill rows the batch asks for, runs
 *                      hpd_decode_step on the batch's plan (paged, with the
 *                      batch's tables) and hpd_verify_draft_step with
 *                      window = config window.
 *  hpd_sched_commit    takes the verification results: each request keeps
 *                      the rows of the tokens it fed up to its accepted
 *                      drafts (len += n_acc + 1; the rest is rolled back),
 *                      records its emitted tokens y*_0 .. y*_{n_acc} (eos ends
 *                      it and is not recorded; so does reaching max_new
 *                      recorded tokens), spawns a child per fork_token a
 *                      parent emits, takes draft_out as its next window, and
 *                      releases finished requests.  A page is output once
 *                      its parent and every child of it have finished: the
 *                      parent's tokens with each child's tokens right after
 *                      the fork token that spawned the child.
 *
 * K/V.  The scheduler owns an hpd_kv_pool of num_blocks blocks of block_rows
 * rows; the device K/V pools are the caller's (shared_k/v and priv_k/v of
 * the step are the same pool tensors).  A page's rows (prompt + the
 * parent's accepted tokens) form a root sequence; the parent branch reads
 * them as its own rows (fork_len 0, past_len = its length) and writes its new
 * rows after them; a child reads the page's first fork_len rows as the
 * shared prefix and owns its rows.  Host memory only; not thread-safe. */
typedef struct {
  int32_t num_blocks;      /* K/V pool blocks (> 0)                          */
  int32_t block_rows;      /* rows per block, a positive multiple of 64      */
  double kv_threshold;     /* tau in [0, 1]                                   */
  int32_t window;          /* K: tokens fed per step after the first, 1..HPD_MAX_K */
  int32_t max_active;      /* N_max >= 1                                     */
  int32_t fork_token, child_token, eos_token;
} hpd_sched_config;

/* The batch of one step.  Arrays are owned by the scheduler and valid until
 * its next call.  num_branches = 0: nothing to run (commit with NULLs). */
typedef struct {
  int32_t num_pages, num_branches, num_tokens;
  const int32_t *prefix_len;    /* [num_pages] P_p: the largest fork_len of
                                   the page's children in the batch        */
  const int32_t *branch_page;   /* [nb] pages in order of their parent's
                                   arrival; a page's parent first, then its
                                   children by arrival                     */
  const int32_t *num_new;       /* [nb] tokens fed                          */
  const int32_t *past_len;      /* [nb] rows before them                    */
  const int32_t *fork_len;      /* [nb] parent 0, child its fork point       */
  hpd_paged_kv paged;           /* the batch's block tables                 */
  const int32_t *request;       /* [nb] request id                          */
  const int32_t *tokens_in;     /* [num_tokens] tokens fed                  */
  const int32_t *prefill_from;  /* [nb] rows prefill_from..prefill_to - 1 of
                                   the branch's own rows (a parent: the
                                   page's) must be computed before the step;
                                   equal when none                          */
  const int32_t *prefill_to;    /* [nb]                                     */
  int32_t num_preempted;        /* requests preempted by this schedule      */
  const int32_t *preempted;
  int32_t num_admitted;         /* requests admitted by it, in order        */
  const int32_t *admitted;
} hpd_sched_batch;

typedef struct hpd_sched hpd_sched;
hpd_status hpd_sched_create(const hpd_sched_config *config, hpd_sched **out);
void hpd_sched_destroy(hpd_sched *sched);
/* A new page: prompt_len >= 1 prefill rows, its first token, at most
 * max_new >= 1 recorded tokens per request (its children too). */
hpd_status hpd_sched_submit(hpd_sched *sched, int32_t prompt_len, int32_t first_token, int32_t max_new,
                            int32_t *request);
hpd_status hpd_sched_schedule(hpd_sched *sched, hpd_sched_batch *out);
/* verified [num_tokens], n_acc [num_branches] (0..num_new - 1), draft_out
 * [num_branches][HPD_MAX_K] (entries 0..window - 1 read): HOST copies of
 * hpd_verify_draft_step's outputs for the last scheduled batch.  Validated
 * before anything changes. */
hpd_status hpd_sched_commit(hpd_sched *sched, const int32_t *verified, const int32_t *n_acc,
                            const int32_t *draft_out);
/* The oldest finished page not yet taken: *page = its parent's id (-1 if
 * none) and *len its tokens; they are copied and the page is dropped when
 * capacity >= *len (tokens may be NULL with capacity 0 to ask the length). */
hpd_status hpd_sched_next_output(hpd_sched *sched, int32_t *page, int32_t *tokens, int32_t capacity,
                                 int32_t *len);
/* Waiting and active requests, free pool blocks. */
hpd_status hpd_sched_counts(const hpd_sched *sched, int32_t *waiting, int32_t *active, int32_t *free_blocks);
/* state: 0 waiting, 1 active, 2 finished; len: rows of its own sequence;
 * kept: of them, rows whose K/V is held; recorded: tokens recorded. */
hpd_status hpd_sched_request(const hpd_sched *sched, int32_t request, int32_t *state, int32_t *len,
                             int32_t *kept, int32_t *recorded);

const char *hpd_status_string(hpd_status status);
const char *hpd_last_error_message(void);

#ifdef __cplusplus
}
#endif

#endif /* HPD_H */
