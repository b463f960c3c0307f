/*
 * dopr.h -- C ABI of the DoPR online-scoring hot path on MI355X (gfx950).
 *
 * DoPR (Reusable Compressed Document Prefixes for Efficient LLM Reranking)
 * scores a (query, document) pair by running only the query tokens and one
 * scoring token through the reranker, while every layer's attention also sees
 * the document's compressed prefix key/value states, computed offline and
 * injected as a pre-filled cache (Sec. 3.1, Eq. 3; Sec. 3.3; Sec. 3.4).  This
 * library implements one decoder layer's share of that online step:
 *
 *   dopr_store_*       the HBM-resident prefix store of per-document K/V
 *                      states (Sec. 3.3: query-independent, reused across
 *                      queries; bf16 per Table 7).
 *   dopr_prefix_attn   batched GQA attention in which each pair's online
 *                      tokens attend to [that document's prefix ; their own
 *                      causal keys] (Sec. 3.4; the query/score tokens see the
 *                      document only through its prefix states, Sec. 3.2.2).
 *   dopr_score_logits  the relevance score read off the score token's state
 *                      (Sec. 3.2.3, Eq. for s(q,d)), as a yes/no logit pair.
 *   dopr_prefix_attn_score
 *                      the last layer's share: only the score token's rows,
 *                      with the score head fused into the attention epilogue.
 *   dopr_decoder_layer the whole decoder layer around that attention.
 *   dopr_salience      offline: which document positions become prefix
 *                      slots (Sec. 3.2.1 salience, top-K selection).
 *
 * Conventions shared by every call
 *   - All device buffers are allocated by the caller and passed as raw device
 *     pointers; the library never calls hipMalloc/hipFree.  Buffers must stay
 *     alive until the stream has passed the call.  (The one exception is
 *     dopr_prefix_attn_noalloc, whose plan lives in a fixed scratch array
 *     that the library's code object holds on each device.)
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *     Every call is asynchronous on that stream unless stated otherwise.
 *   - bf16 means IEEE bfloat16 bit patterns (uint16); fp32 means IEEE float.
 *   - head_dim D is 128 (Qwen3, Llama 3) or 64 (Llama 3.2 1B, the model of
 *     the cross-family check in the Appendix); the decoder layer and the
 *     salience selection take D = 128 only.  n_q_heads must be a multiple
 *     of n_kv_heads; q head h reads kv head h / (n_q_heads / n_kv_heads).
 *   - Every call returns a dopr_status_t.  Host-checkable argument errors are
 *     returned before anything is launched.  Errors found on the device (a
 *     doc id that is out of range or not resident, malformed cu_seqlens) are
 *     deferred: the affected outputs are written as zeros, nothing is read
 *     out of bounds, and dopr_check_status() reports the error.
 *   - No C++ exception crosses this ABI and the library never aborts.
 *   - Calls that share a store and overlap on different streams may race on
 *     the store's deferred status word only (never on data).
 */
#ifndef DOPR_H
#define DOPR_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  DOPR_OK = 0,
  DOPR_ERR_INVALID_ARG = -1, /* null pointer, bad size, bad shape          */
  DOPR_ERR_UNSUPPORTED = -2, /* valid but not implemented (e.g. D = 96)    */
  DOPR_ERR_DOC_RANGE = -3,   /* doc id outside [0,n_docs) or not resident  */
  DOPR_ERR_WORKSPACE = -4,   /* workspace or pool smaller than required    */
  DOPR_ERR_HIP = -5,         /* a HIP runtime call failed                  */
  DOPR_ERR_SEQLEN = -6       /* cu_seqlens not monotone, T_p < 1,
                                T_p > max_tokens or cu[P] != total_tokens  */
} dopr_status_t;

/* Opaque store handle.  The library owns only this small host struct; the
 * store's index and payload live in the caller's device pool. */
typedef struct dopr_store *dopr_store_t;

/* ------------------------------------------------------------------------ */
/* Prefix store (Sec. 3.1 Eq. 3 and Sec. 3.3: per document d, the multi-layer
 * K/V states C~_d of its K_infer selected prefix slots, stored offline).      */

typedef struct {
  int32_t n_layers;       /* decoder layers held per document (>= 1)        */
  int32_t n_kv_heads;     /* Hkv (>= 1)                                     */
  int32_t head_dim;       /* D; 128 or 64 (UNSUPPORTED otherwise)           */
  int64_t n_docs;         /* size of the doc-id space [0, n_docs)           */
  const int32_t *doc_len; /* HOST [n_docs]: prefix slots L_d of doc d.
                             0 is allowed (no prefix); -1 = not resident
                             (pairs naming it fail with DOC_RANGE).         */
} dopr_store_desc_t;

/* Sizes of a store.  *pool_bytes (required) is what dopr_store_create needs
 * in the caller's pool: a small header, the index (12 B per doc id) and the
 * payload in the library's internal layout (V rows padded to 8 slots).
 * *payload_bytes (optional, may be NULL) is the canonical K/V size
 * sum_d L_d * n_layers * Hkv * D * 2 (K and V) * 2 bytes, the document-side
 * memory the paper reports per pair (Tables 3 and 9).  Pure host arithmetic. */
dopr_status_t dopr_store_bytes(const dopr_store_desc_t *desc,
                               size_t *pool_bytes, size_t *payload_bytes);

/* Lay out a store in `pool` (device, >= pool_bytes, 256-byte aligned) and
 * write its index (stream-ordered copy from host).  The payload is left
 * uninitialised until dopr_store_put fills it.  *out receives a handle that
 * must be released with dopr_store_destroy (which does not free the pool). */
dopr_status_t dopr_store_create(const dopr_store_desc_t *desc, void *pool,
                                size_t pool_bytes, void *stream,
                                dopr_store_t *out);

/* Copy the prefix K/V states of `n` documents for one layer into the store.
 *   doc_ids      dev int32 [n]   documents to fill (resident ones)
 *   src_cu_slots dev int64 [n+1] slot ranges of each document in k_src/v_src;
 *                must satisfy src_cu_slots[i+1]-src_cu_slots[i] == L_d
 *   k_src, v_src dev bf16 [src_cu_slots[n], Hkv, D] (canonical layout: the
 *                final keys/values of each prefix slot, already normed and
 *                rotated at positions 0..L_d-1 as in any pre-filled cache)
 * A doc id that is out of range, not resident, or whose slot count differs
 * from L_d is skipped and reported by dopr_check_status as DOC_RANGE.      */
dopr_status_t dopr_store_put(dopr_store_t st, int32_t layer, int64_t n,
                             const int32_t *doc_ids,
                             const int64_t *src_cu_slots, const void *k_src,
                             const void *v_src, void *stream);

dopr_status_t dopr_store_destroy(dopr_store_t st);

/* Carry documents over from one store to another (store maintenance: the
 * prefix states are built once per document offline and kept for reuse,
 * Sec. 3.3-3.4, so a collection that grows or shrinks is served by a new
 * store holding the kept documents).  For every document id resident in
 * both stores with the same slot count, dst receives src's states for all
 * layers and kv heads (and their key-norm bounds); ids resident only in dst
 * keep their contents (fill them with dopr_store_put), ids resident only in
 * src are dropped.  So a store with more resident ids appends documents,
 * and one with fewer repacks the kept ones densely.  Both stores must have
 * the same n_docs (id space), n_layers and n_kv_heads and distinct,
 * non-overlapping pools (INVALID_ARG otherwise).  A document resident in
 * both with different slot counts is skipped and reported as a deferred
 * DOC_RANGE on dst.  Asynchronous on `stream`.                             */
dopr_status_t dopr_store_copy_docs(dopr_store_t dst, dopr_store_t src,
                                   void *stream);

/* ------------------------------------------------------------------------ */
/* Online prefix attention (Sec. 3.4): for every pair p with document
 * d = doc_ids[p] and online tokens j = 0..T_p-1 (query tokens, then the
 * score token last), q head h, kv head g = h / n_rep:
 *   q^ = RoPE_{L_d + j}(RMSNorm(q[j,h]) * q_norm_w)
 *   k^ = RoPE_{L_d + j}(RMSNorm(k[j,g]) * k_norm_w)        (own keys)
 *   keys   = [ K_d[g, 0..L_d-1] ; k^[0..j, g] ]
 *   values = [ V_d[g, 0..L_d-1] ;  v[0..j, g] ]
 *   out[j,h] = softmax(softmax_scale * q^ . keys) . values
 * RoPE is the rotate-half form: the pair (x_i, x_{i+D/2}) turns by
 * position * omega_i with omega_i = rope_theta^(-2i/D), or rope_inv_freq[i]
 * when given.  RMSNorm is per head over D with epsilon rms_eps; with both
 * norm gains NULL there is no RMSNorm (q^ = RoPE(q), k^ = RoPE(k), as in
 * attention families without QK-norm such as Llama).  Online positions
 * continue after the prefix.                                               */
typedef struct {
  int32_t n_pairs;          /* P >= 0                                       */
  int32_t n_q_heads;        /* Hq, multiple of the store's Hkv              */
  int32_t max_tokens;       /* upper bound on every T_p (>= 1)              */
  int32_t kernel_variant;   /* 0 = automatic: 8, or 6 when every prefix is
                               at most 96 slots at D = 128; 1, 2, 3, 6, 8
                               select a
                               kernel (identical results; for tuning
                               sweeps): 1 = 4 waves x 64 rows, 2 = 8 waves
                               x 32 rows, 3 = 4 waves x 32 rows (each one
                               block per CU, 256 prefix slots resident;
                               512 at D = 64), 6 = 4 waves x 32 rows, two
                               blocks per CU, 96 slots resident (256 at
                               D = 64); 8 = the pass kernel: an 8-wave
                               block (one per CU at D = 128, two at D = 64)
                               takes a (work item, kv head) unit, keeps a
                               prefix of up to 256 slots in LDS for all its
                               passes of 256 rows, and reads the own keys
                               from a k^ buffer in the workspace (2 Hkv D
                               bytes per online token) filled by a
                               separate normalise-and-rotate kernel;
                               4 = exact running-max softmax for every row
                               (slower; the reference for the fast path);
                               5 = self-check: the fast pass queues every
                               work unit for the exact pass (tests only)   */
  int64_t total_tokens;     /* Ntok = cu_seqlens[P]                         */
  const int32_t *doc_ids;   /* dev int32 [P]                                */
  const int32_t *cu_seqlens;/* dev int32 [P+1], cu[0] = 0, T_p >= 1         */
  const void *q;            /* dev bf16 [Ntok, Hq, D]   raw (pre-norm)      */
  const void *k;            /* dev bf16 [Ntok, Hkv, D]  raw (pre-norm)      */
  const void *v;            /* dev bf16 [Ntok, Hkv, D]                      */
  const void *q_norm_w;     /* dev bf16 [D], or NULL with k_norm_w NULL:
                               no per-head RMSNorm                          */
  const void *k_norm_w;     /* dev bf16 [D], or NULL (see q_norm_w)         */
  float rms_eps;            /* e.g. 1e-6                                    */
  float rope_theta;         /* e.g. 1e6                                     */
  float softmax_scale;      /* e.g. 1/sqrt(D); finite and > 0               */
  void *out;                /* dev bf16 [Ntok, Hq, D]                       */
  float *lse;               /* dev fp32 [Ntok, Hq] natural-log sum-exp of
                               the scaled logits, or NULL                   */
  void *workspace;          /* dev scratch, >= dopr_prefix_attn_workspace() */
  size_t workspace_bytes;
  void *timing_begin;       /* optional hipEvent_t recorded on the stream
                               right before the attention kernel, or NULL  */
  void *timing_end;         /* optional hipEvent_t recorded right after it,
                               or NULL (profiling of the dominant kernel)   */
  const float *rope_inv_freq; /* dev fp32 [D/2] rotation frequencies
                               omega_i (e.g. a family's rescaled ones), or
                               NULL for rope_theta^(-2i/D); 4-byte aligned */
  int32_t rows_per_item;    /* 0 = automatic.  Else the size, in stacked
                               rows (token x q head of one kv head), of the
                               work items a document's rows are cut into:
                               a multiple of 32 in [64, 2^20].  Outputs do
                               not depend on it (a tuning and test knob).
                               Full-row calls only: must be 0 for
                               dopr_prefix_attn_score (INVALID_ARG).        */
  int32_t queue_order;      /* order in which each of the 8 work queues
                               (one per XCD) hands out its (item, kv head)
                               units.  0 = automatic: longest-first while
                               the CUs average at most 128 units each,
                               else natural; 1 = natural (item order);
                               2 = longest-first (costliest document group
                               first, item order within a cost class) up to
                               32768 units, natural beyond.  Outputs do not
                               depend on it (a tuning and test knob); other
                               values are INVALID_ARG.                      */
} dopr_attn_args_t;

/* Workspace bytes needed by dopr_prefix_attn for these arguments (host). */
dopr_status_t dopr_prefix_attn_workspace(dopr_store_t st,
                                         const dopr_attn_args_t *args,
                                         size_t *bytes);

/* Run the online attention of one layer for a batch of pairs.  Pairs that
 * share a document are grouped on the device so that the document's prefix
 * is read from HBM once per group and reused from LDS.  Pairs with a bad doc
 * id get zero outputs (lse = -inf) and a deferred DOC_RANGE status.        */
dopr_status_t dopr_prefix_attn(dopr_store_t st, int32_t layer,
                               const dopr_attn_args_t *args, void *stream);

/* dopr_prefix_attn for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc).  Same arguments, results and errors as dopr_prefix_attn,
 * except:
 *   - args->workspace must be NULL and args->workspace_bytes 0: the plan is
 *     laid out in a scratch array that the library holds, one copy per
 *     device, from the first use on that device until the process ends;
 *   - the scratch holds at most 64 MiB (DOPR_NOALLOC_SCRATCH_BYTES).  A call
 *     whose plan needs more returns DOPR_ERR_WORKSPACE and launches nothing;
 *     dopr_prefix_attn_workspace gives the size, except that here the
 *     automatic choice (kernel_variant 0) and the self-check variant 5 never
 *     take the pass kernel (8), whose plan grows with every token; variant 8
 *     is run only when asked for and its plan fits;
 *   - the call allocates nothing: no hipMalloc, hipFree or allocating
 *     library routine.
 * Every call on one device shares that device's scratch: calls that overlap
 * on one device (other streams, other threads) race and must be ordered by
 * the caller.  The plan's kernels clear what must start at zero.  Outputs
 * are bitwise identical to dopr_prefix_attn's for the same inputs.        */
#define DOPR_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
dopr_status_t dopr_prefix_attn_noalloc(dopr_store_t st, int32_t layer,
                                       const dopr_attn_args_t *args,
                                       void *stream);

/* ------------------------------------------------------------------------ */
/* Score head (Sec. 3.2.3): s(q,d) from the score token's hidden state h.
 * Read as RMSNorm followed by a two-row linear head (yes, no):
 *   h^ = RMSNorm(h) * norm_w;  l_yes = w_yes . h^;  l_no = w_no . h^;
 *   s  = l_yes - l_no   (log-odds of "relevant"; what RankNet consumes).   */
typedef struct {
  int32_t n_pairs;           /* P >= 0                                      */
  int32_t width;             /* W, multiple of 8, >= 8                      */
  const void *h;             /* dev bf16; row r starts at h + r*h_row_stride */
  int64_t h_row_stride;      /* elements between rows, >= width, mult. of 8 */
  const int32_t *row_index;  /* dev int32 [P]: h row of pair p, or NULL    */
  const int32_t *cu_seqlens; /* dev int32 [P+1]: used when row_index is
                                NULL: row = cu_seqlens[p+1]-1 (the score
                                token is each pair's last online token).
                                Both NULL: row = p.                         */
  const void *norm_w;        /* dev bf16 [W]                                */
  const void *w_head;        /* dev bf16 [2, W]: row 0 = yes, row 1 = no    */
  float rms_eps;
  float *logits;             /* dev fp32 [P, 2] (l_yes, l_no), or NULL      */
  float *score;              /* dev fp32 [P]                                */
} dopr_score_args_t;

dopr_status_t dopr_score_logits(const dopr_score_args_t *args, void *stream);

/* ------------------------------------------------------------------------ */
/* Last-layer scoring (Sec. 3.2.3 with Sec. 3.4).  The score head reads only
 * the score token's hidden state, so in the last layer only the final row
 * j = T_p - 1 of every pair needs an attention output.  This call computes
 * exactly the rows dopr_prefix_attn computes for those tokens (same keys:
 * all L_d prefix slots and all T_p own keys, so every own key and value is
 * still read and every own key is normed and rotated), and feeds them to
 * the score head of dopr_score_logits with width W = n_q_heads * D:
 *   h = out[p] viewed as [W] (bf16-rounded attention output),
 *   h^ = RMSNorm(h) * norm_w;  l_yes = w_yes . h^;  l_no = w_no . h^;
 *   s = l_yes - l_no.
 * The head is fused into the attention epilogue: each (pair, q head) row
 * contributes its partial sums of h^2, norm_w*w_yes*h and norm_w*w_no*h;
 * a small kernel adds the n_q_heads partials of a pair in head order.
 * Arguments are those of dopr_prefix_attn with two differences:
 *   out  dev bf16 [P, Hq, D]: the score rows, or NULL (not written);
 *   lse  dev fp32 [P, Hq], or NULL;
 * and the workspace comes from dopr_prefix_attn_score_workspace.
 * kernel_variant 0 (automatic) runs one wave per work unit of at most 32
 * score rows while every resident prefix is at most 512 slots (one 4-wave
 * block per 4 units, no block barrier), else shape 6; 1 and 3 select
 * shape 6 here (2 and 6 as above; identical results in every case).  A
 * pair with a bad doc id gets zero rows, lse -inf, logits and score 0, and
 * a deferred DOC_RANGE status.  All buffers are caller-owned.              */
typedef struct {
  const void *norm_w;       /* dev bf16 [W], W = n_q_heads * D              */
  const void *w_head;       /* dev bf16 [2, W]: row 0 = yes, row 1 = no    */
  float rms_eps;            /* >= 0, finite                                 */
  float *logits;            /* dev fp32 [P, 2] (l_yes, l_no), or NULL      */
  float *score;             /* dev fp32 [P]                                 */
} dopr_score_head_t;

dopr_status_t dopr_prefix_attn_score_workspace(dopr_store_t st,
                                               const dopr_attn_args_t *args,
                                               size_t *bytes);

dopr_status_t dopr_prefix_attn_score(dopr_store_t st, int32_t layer,
                                     const dopr_attn_args_t *args,
                                     const dopr_score_head_t *head,
                                     void *stream);

/* ------------------------------------------------------------------------ */
/* One decoder layer of the online pass (Sec. 3.4: only [q; t_score] runs
 * through the reranker, every layer's attention also seeing the stored
 * prefix states).  The layer is the Qwen3 decoder layer, in the stored-weight
 * convention y = x W^T with W [out, in]:
 *   h  = RMSNorm(x) * attn_norm_w
 *   q, k, v = h w_q^T, h w_k^T, h w_v^T          (then as dopr_prefix_attn)
 *   x2 = x + attention(q, k, v) w_o^T
 *   h2 = RMSNorm(x2) * mlp_norm_w
 *   y  = x2 + (SiLU(h2 w_gate^T) * (h2 w_up^T)) w_down^T
 * RMSNorm is over the hidden width with epsilon rms_eps of the batch args.
 * Projections accumulate in fp32 and every activation between steps is
 * stored as bf16.  The batch is described by a dopr_attn_args_t whose q, k,
 * v and out must be NULL (the layer forms them in its workspace); lse may be
 * given ([Ntok, Hq]); workspace and workspace_bytes come from
 * dopr_decoder_layer_workspace.  x and y may be the same buffer.           */
typedef struct {
  int32_t hidden;            /* W, multiple of 8                            */
  int32_t intermediate;      /* I, multiple of 8                            */
  const void *attn_norm_w;   /* dev bf16 [W]                                */
  const void *w_q;           /* dev bf16 [Hq*D, W]                          */
  const void *w_k;           /* dev bf16 [Hkv*D, W]                         */
  const void *w_v;           /* dev bf16 [Hkv*D, W]                         */
  const void *w_o;           /* dev bf16 [W, Hq*D]                          */
  const void *mlp_norm_w;    /* dev bf16 [W]                                */
  const void *w_gate;        /* dev bf16 [I, W]                             */
  const void *w_up;          /* dev bf16 [I, W]                             */
  const void *w_down;        /* dev bf16 [W, I]                             */
  const void *x;             /* dev bf16 [Ntok, W] entering the layer       */
  void *y;                   /* dev bf16 [Ntok, W] leaving it               */
} dopr_layer_args_t;

dopr_status_t dopr_decoder_layer_workspace(dopr_store_t st,
                                           const dopr_attn_args_t *batch,
                                           const dopr_layer_args_t *lw,
                                           size_t *bytes);

dopr_status_t dopr_decoder_layer(dopr_store_t st, int32_t layer,
                                 const dopr_attn_args_t *batch,
                                 const dopr_layer_args_t *lw, void *stream);

/* ------------------------------------------------------------------------ */
/* ------------------------------------------------------------------------ */
/* Offline salience selection (Sec. 3.2.1, applied offline in Sec. 3.3): for
 * each document, independently encoded at positions 0..n_d-1, with the final
 * layer's queries q^ and keys k^ as they enter the attention product (after
 * any norm and rotary embedding), q head h reading kv head h / n_rep:
 *   A_h[j, i] = softmax over i <= j of softmax_scale * q^_h[j] . k^_g[i]
 *   Abar      = mean of A_h over the Hq query heads (row j attends,
 *               column i is attended; zero above the diagonal)
 *   u_i       = mean of the m = min(p, n_d - i) largest Abar[j, i] over the
 *               visible rows j >= i (the paper's |T_p| = min(p, n - i + 1)
 *               with 1-based i)
 *   selected  = the K_d positions with the largest u, ties to the lower
 *               position, written in ascending position order.
 * The GPU computes logits in fp32 from the bf16 operands, probabilities
 * with exp2 against each row's log-sum-exp, Abar and u in fp32.           */
#define DOPR_SALIENCE_MAX_LEN 4096
#define DOPR_SALIENCE_MAX_P 64

typedef struct {
  int32_t n_docs;            /* documents in the batch (>= 0)              */
  int32_t max_doclen;        /* M: bound on every n_d, 1..4096             */
  int32_t n_q_heads;         /* Hq, multiple of n_kv_heads                 */
  int32_t n_kv_heads;        /* Hkv >= 1                                   */
  int32_t top_p;             /* p, 1..64                                   */
  float softmax_scale;       /* e.g. 1/sqrt(D); finite and > 0             */
  int64_t total_tokens;      /* Ntok = cu_doclens[n_docs]                  */
  int64_t total_select;      /* cu_select[n_docs] (ignored if selected is
                                NULL)                                      */
  const int32_t *cu_doclens; /* dev int32 [n_docs+1]: document d owns token
                                rows cu[d] .. cu[d+1]-1, 1 <= n_d <= M    */
  const int32_t *cu_select;  /* dev int32 [n_docs+1]: K_d = cs[d+1]-cs[d],
                                0 <= K_d <= n_d; or NULL with selected    */
  const void *q;             /* dev bf16 [Ntok, Hq, D]                     */
  const void *k;             /* dev bf16 [Ntok, Hkv, D]                    */
  float *u;                  /* dev fp32 [Ntok]: salience of every token
                                (output of dopr_salience, input of
                                dopr_select_top_k)                         */
  int32_t *selected;         /* dev int32 [total_select]: doc d's chosen
                                positions (0-based within the document) at
                                cs[d] .., ascending; or NULL (u only)     */
  float *attn_mean;          /* optional dev fp32 [n_docs, M, M]: Abar of
                                doc d at d*M*M + j*M + i; only i <= j < n_d
                                is written.  NULL: kept in the workspace  */
  int32_t *status;           /* optional dev int32, zeroed by the caller:
                                receives DOPR_ERR_SEQLEN when cu_doclens or
                                cu_select is malformed (the affected
                                documents are skipped), else untouched    */
  void *workspace;           /* dev scratch >= dopr_salience_workspace()   */
  size_t workspace_bytes;
} dopr_salience_args_t;

/* Workspace bytes for these arguments (host): the row log-sum-exp of every
 * (token, q head), eight partial maxima of the key norms of every
 * (document, kv head) and,
 * unless attn_mean is given, Abar for as many documents at a time as fit
 * in 1 GiB (at least one).  dopr_salience accepts any workspace that holds
 * the row statistics and key norms plus one document's Abar (4 M^2 bytes)
 * and processes as many documents per pass as fit. */
dopr_status_t dopr_salience_workspace(const dopr_salience_args_t *args,
                                      size_t *bytes);

/* Salience u of every token and, if selected is not NULL, the top-K_d
 * positions of every document.  Asynchronous on `stream`. */
dopr_status_t dopr_salience(const dopr_salience_args_t *args, void *stream);

/* The selection step alone, on u given by the caller: uses n_docs,
 * max_doclen, total_tokens, total_select, cu_doclens, cu_select, u,
 * selected and status; values order as IEEE-754 totalOrder (-0 < +0),
 * ties to the lower position.  No workspace. */
dopr_status_t dopr_select_top_k(const dopr_salience_args_t *args,
                                void *stream);

/* ------------------------------------------------------------------------ */
/* Exports used by the bit-exact tests of the integer steps.               */

/* Doc-id grouping (Sec. 3.4 with Sec. 4.5.2: the pairs that retrieve the
 * same document share its stored prefix, so they are batched by document)
 * in canonical form: valid pairs (doc id in range and
 * resident) sorted by (doc id, pair index).  group_doc[G] ascending doc ids,
 * group_ptr[G+1] offsets into pair_order[], pair_order[n_valid] pair indices.
 * Capacities: group_doc and pair_order >= n_pairs, group_ptr >= n_pairs+1.
 * `workspace` must hold dopr_prefix_attn_workspace() bytes for the same
 * pairs.  Synchronises `stream` to return *n_groups and *n_valid on the host. */
dopr_status_t dopr_group_pairs(dopr_store_t st, int32_t n_pairs,
                               const int32_t *doc_ids, void *workspace,
                               size_t workspace_bytes, int32_t *n_groups,
                               int32_t *n_valid, int32_t *group_doc,
                               int32_t *group_ptr, int32_t *pair_order,
                               void *stream);

/* Gather the prefix K/V states of doc_ids[i] for one layer out of the store
 * (Sec. 3.4: a candidate's stored prefix states are fetched by its id)
 * into canonical layout: k_out/v_out dev bf16 [out_cu_slots[n], Hkv, D],
 * pair i's slots at rows out_cu_slots[i] .. out_cu_slots[i+1]-1.  A bad doc
 * id, or a slot range that differs from L_d, leaves its rows untouched and
 * raises a deferred DOC_RANGE.                                             */
dopr_status_t dopr_gather_prefix(dopr_store_t st, int32_t layer, int32_t n,
                                 const int32_t *doc_ids,
                                 const int64_t *out_cu_slots, void *k_out,
                                 void *v_out, void *stream);

/* ------------------------------------------------------------------------ */
/* Status (library plumbing; no passage of the paper defines it).          */

/* Synchronise `stream`, then return (and clear) the first deferred device
 * error raised by calls on this store since the last check, else DOPR_OK.  */
dopr_status_t dopr_check_status(dopr_store_t st, void *stream);

/* Human-readable name of a status code (static string). */
const char *dopr_status_str(dopr_status_t s);

/* Thread-local text describing the last non-OK status returned on this
 * thread ("" if none). */
const char *dopr_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* DOPR_H */
