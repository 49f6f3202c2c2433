/*
 * focus.h -- C interface of the FOCUS hot path for AMD MI355X (CDNA4, gfx950).
 *
 * FOCUS (arXiv 2511.14694) inserts one summary token after every k bases of a
 * DNA sequence, processes the sequence in base-domain windows, and keeps only
 * the summary tokens' key/value rows across windows.  This library implements
 * the per-layer hot path of that scheme:
 *
 *   focus_layout_plan / focus_layout   summary-token layout and index metadata
 *   focus_compact_kv                   append summary K/V rows to the cache
 *   focus_window_attn                  window attention over [cache ; window]
 *   focus_decode_step                  one-token decode over [cache ; window]
 *
 * Conventions shared by every call
 * --------------------------------
 * Memory.  Pointers marked [device] are HIP device pointers owned by the
 *   caller; [host] pointers are ordinary host memory.  The library never
 *   allocates, frees or keeps a pointer after a call returns.  Tensors are
 *   row-major with head_dim contiguous and 16-byte aligned base pointers:
 *     token tensors   [rows, heads, head_dim]       ("THD")
 *     caches          [batch, capacity, kv_heads, head_dim]
 * Types.  FOCUS_BF16 tensors hold bfloat16, FOCUS_F32 tensors float32; one
 *   call uses one dtype for q, k, v, caches and o.  Scores, softmax and
 *   accumulation are float32; o is rounded to the tensor dtype (nearest-even);
 *   lse is float32 natural-log.
 * Execution.  Every device-side call only enqueues kernels on `stream` (a
 *   hipStream_t passed as void*; NULL = the null stream) and never
 *   synchronises.  Calls are re-entrant; the library holds no state.
 * Errors.  Every call returns a focus_status.  Problems visible on the host
 *   (NULL or misaligned pointers, inconsistent sizes, unsupported shapes, a
 *   short workspace) are reported before anything is enqueued, so nothing is
 *   written.  Problems only the device can see (a row index outside a buffer, a
 *   cache at capacity, layout totals that differ from the plan) skip the
 *   affected rows and OR a FOCUS_ERR_* bit into the optional [device] `err`
 *   word; no kernel ever writes outside the buffers described to it.
 * Indexing (0-based).  Windows, augmented tokens and summaries of all
 *   sequences of a batch are numbered globally, sequence after sequence
 *   ("global window / token / summary index"); bases of all sequences are
 *   concatenated ("global base index"); a cache row is counted inside its own
 *   sequence.
 */
#ifndef FOCUS_H
#define FOCUS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define FOCUS_ABI_VERSION 3

typedef int32_t focus_status;
enum {
  FOCUS_OK = 0,
  FOCUS_E_NULL = 1,        /* a required pointer is NULL                        */
  FOCUS_E_ARG = 2,         /* a value out of range, or a misaligned pointer     */
  FOCUS_E_SHAPE = 3,       /* sizes inconsistent with each other                */
  FOCUS_E_DTYPE = 4,       /* unknown dtype                                     */
  FOCUS_E_UNSUPPORTED = 5, /* well-formed request this build does not implement */
  FOCUS_E_WORKSPACE = 6,   /* workspace missing or too small                    */
  FOCUS_E_CAPACITY = 7,    /* a cache is too small for the planned rows         */
  FOCUS_E_HIP = 8          /* the HIP runtime refused a launch                  */
};

typedef enum { FOCUS_BF16 = 0, FOCUS_F32 = 1 } focus_dtype;

/* Visibility rule of focus_window_attn.
 * FOCUS_MASK_CT: the set C(t) of Appendix A.1 ("Objective and visibility"):
 *   a token sees every earlier-or-equal token of its own window and every
 *   retained summary of the earlier windows of its sequence.
 * FOCUS_MASK_KMER_LOCAL: the stricter rule of Section 3.2 ("Visibility and
 *   summarization rule"): a token sees the earlier-or-equal tokens of its own
 *   k-mer (a summary closes its k-mer), the earlier summaries of its own window
 *   and the boundary summary carried over from the previous window, which is
 *   the last retained cache row C_w - 1.  Nothing else of earlier windows is
 *   visible.  A window with k = 0 is one k-mer (causal inside the window). */
typedef enum { FOCUS_MASK_CT = 0, FOCUS_MASK_KMER_LOCAL = 1 } focus_mask;

/* tok_kind values */
enum { FOCUS_TOK_BASE = 0, FOCUS_TOK_SUMMARY = 1 };
/* focus_decode_desc.kind bits */
enum { FOCUS_STEP_SUMMARY = 1, FOCUS_STEP_WINDOW_END = 2 };
/* bits of the device error word */
enum { FOCUS_ERR_CAPACITY = 1, FOCUS_ERR_BOUNDS = 2, FOCUS_ERR_PLAN = 4 };

typedef void* focus_stream_t;   /* a hipStream_t */

int32_t focus_abi_version(void);
const char* focus_status_str(focus_status s);
/* sizeof of the descriptor structs below, in declaration order
 * (0 totals, 1 layout, 2 compact, 3 attn, 4 decode, 5 fidelity, 6 gemm,
 * 7 adapter, 8 adapter layer, 9 qkv projection, 10 decode schedule); -1
 * otherwise.
 * Lets a binding check its mirror of the structs. */
int64_t focus_struct_size(int32_t which);

/* ------------------------------------------------------------------------ */
/* Layout                                                                    */
/* ------------------------------------------------------------------------ */

/* Totals of a layout, computed on the host by focus_layout_plan. */
typedef struct {
  int64_t n_windows;            /* sum_b ceil(L_b / W)                       */
  int64_t n_tokens;             /* augmented tokens: bases + summaries       */
  int64_t n_summaries;          /* sum_w B_w                                 */
  int64_t max_window_tokens;    /* max_w T_w, T_w = n_w + B_w                */
  int64_t max_window_summaries; /* max_w B_w                                 */
  int64_t max_cache_per_seq;    /* max_b sum_{w in b} B_w (cache rows needed) */
  int64_t max_window_cache;     /* max_w C_w (cache rows a window attends to) */
} focus_layout_totals;

/* Summary-token layout totals (Appendix A: windows I_w = [(w-1)W+1, wW] clipped
 * to [1, L], ceil(L/W) per sequence, B_w = ceil(|I_w| / k_w) summaries each;
 * Section 3.2: one summary after every k bases, a trailing partial k-mer
 * included).
 *   batch      number of sequences, >= 0
 *   seq_nt     [host] [batch] bases per sequence, each >= 0
 *   window_nt  W, bases per window, >= 1
 *   kmer       [host] [n_windows] cadence k_w per global window, or NULL to
 *              use kmer_uniform for all; k_w = 0 means no summary tokens
 *   out        [host] receives the totals
 * O(number of windows) host work.  Errors: E_NULL, E_ARG. */
focus_status focus_layout_plan(int32_t batch, const int64_t* seq_nt, int32_t window_nt,
                               const int32_t* kmer, int32_t kmer_uniform,
                               focus_layout_totals* out);

/* Everything focus_layout reads and writes.  All arrays [device].
 * Per window w (global index): the window belongs to sequence win_seq[w], holds
 * n_w = win_nt[w] bases and B_w = win_nsum[w] summaries, T_w = win_ntok[w]
 * augmented tokens starting at global token win_tok_off[w] and global base
 * win_base_off[w]; its first summary is global summary win_sum_off[w]; it sees
 * cache rows [0, C_w) with C_w = win_cache_off[w].
 * Per token t (global index), in window order [k-mer bases, summary, ...]:
 * tok_kind[t] (FOCUS_TOK_*), tok_pos[t] = position in its sequence's augmented
 * stream, tok_win[t] = window, tok_base[t] = global base index or -1 for a
 * summary, tok_kmer[t] = cache row of the summary closing its k-mer (-1 when
 * k_w = 0), token_ids[t] = bases[tok_base[t]] or summary_token_id, and, if
 * asked for, tok_next_base[t] = the global base index of pi(t), the first real
 * base after t in its sequence (the training target of every position,
 * Appendix A.1 eq. loss), or -1 past the sequence's last base.
 * Per summary s: sum_tok[s] = its global token index.
 * cu_*[b] = first global window / token / summary of sequence b; cu_*[batch] =
 * the total. */
typedef struct {
  focus_layout_totals totals;   /* from focus_layout_plan on the same inputs */
  int32_t batch;
  int32_t window_nt;
  int32_t kmer_uniform;         /* cadence when kmer == NULL                 */
  int32_t summary_token_id;     /* token id written at summary positions    */
  const int64_t* seq_nt;        /* [batch]                                   */
  const int32_t* kmer;          /* [n_windows] or NULL                       */
  const uint8_t* bases;         /* [sum seq_nt] base bytes, or NULL           */
  int64_t* cu_windows;          /* [batch + 1]                               */
  int64_t* cu_tokens;           /* [batch + 1]                               */
  int64_t* cu_summaries;        /* [batch + 1]                               */
  int32_t* win_seq;             /* [n_windows]                               */
  int32_t* win_nt;
  int32_t* win_nsum;
  int32_t* win_ntok;
  int32_t* win_cache_off;
  int64_t* win_tok_off;
  int64_t* win_sum_off;
  int64_t* win_base_off;
  int32_t* tok_pos;             /* [n_tokens]                                */
  int32_t* tok_kmer;
  int32_t* tok_win;
  uint8_t* tok_kind;
  int64_t* tok_base;
  int64_t* sum_tok;             /* [n_summaries]                             */
  int32_t* token_ids;           /* [n_tokens], written only if bases != NULL */
  int64_t* tok_next_base;       /* [n_tokens] or NULL: pi(t), see above      */
  int32_t* err;                 /* optional error word                       */
} focus_layout_desc;

/* Fill every layout array (definitions above).  The result is bit-exact: it is
 * pure integer work.  Device check: if the totals the device finds differ from
 * d->totals, FOCUS_ERR_PLAN is raised and nothing beyond the planned sizes is
 * written.  Errors: E_NULL, E_ARG, E_SHAPE, E_HIP. */
focus_status focus_layout(const focus_layout_desc* d, focus_stream_t stream);

/* ------------------------------------------------------------------------ */
/* Compaction                                                                */
/* ------------------------------------------------------------------------ */

/* Retained-KV compaction (Appendix A "KV compression and budget", A.2): after
 * window w, the K/V rows of its B_w summary tokens are appended to its
 * sequence's cache, at rows [C_w, C_w + B_w); ordinary rows are not copied.
 * The shared boundary summary is the last row window w writes and is stored
 * once.  The copy is bit-exact. */
typedef struct {
  focus_layout_totals totals;   /* of the layout the arrays below belong to  */
  int32_t dtype;                /* focus_dtype of k, v, cache_k, cache_v     */
  int32_t n_kv_heads;
  int32_t head_dim;             /* 64 or 128                                 */
  int32_t batch;
  int64_t n_win;                /* entries of win_ids (ignored if NULL)      */
  const int32_t* win_ids;       /* [device] global windows to compact, or
                                   NULL for every window of the layout       */
  const int32_t* win_seq;       /* [device] layout arrays                    */
  const int32_t* win_nsum;
  const int32_t* win_cache_off;
  const int64_t* win_sum_off;
  const int64_t* sum_tok;
  const void* k;                /* [kv_rows, n_kv_heads, head_dim]: row r is  */
  const void* v;                /*   global token kv_tok_base + r             */
  int64_t kv_tok_base;
  int64_t kv_rows;
  void* cache_k;                /* [batch, cache_cap, n_kv_heads, head_dim]  */
  void* cache_v;
  int64_t cache_cap;
  int32_t* cache_len;           /* [device][batch] or NULL: raised (never
                                   lowered) to C_w + B_w of each listed window */
  int32_t* err;                 /* optional error word                       */
} focus_compact_desc;

/* Errors: E_NULL, E_ARG, E_DTYPE, E_SHAPE, E_UNSUPPORTED, E_CAPACITY (the
 * plan's max_cache_per_seq exceeds cache_cap), E_HIP.  A summary row outside
 * [0, kv_rows) or a cache row >= cache_cap is skipped on the device with
 * FOCUS_ERR_BOUNDS / FOCUS_ERR_CAPACITY. */
focus_status focus_compact_kv(const focus_compact_desc* d, focus_stream_t stream);

/* ------------------------------------------------------------------------ */
/* Window attention (prefill)                                                */
/* ------------------------------------------------------------------------ */

/* For every listed window w of sequence b, every head h and every window query
 * row i in [0, T_w) (global token t = win_tok_off[w] + i):
 *     keys     = [cache_k[b, 0:C_w, g] ; k[window rows, g]],  g = h / (H / H_kv)
 *     visible  = every cache row, and window rows u <= i      (FOCUS_MASK_CT)
 *              = cache row C_w - 1, and window rows u <= i that are summaries
 *                or lie in row i's k-mer                   (FOCUS_MASK_KMER_LOCAL)
 *     o[t, h]  = softmax(scale * q[t, h] . keys^T over visible) . values
 *     lse[t,h] = log sum_visible exp(scale * q[t, h] . key)
 * (Appendix A eq. focus-attn with the visibility set C(t) of A.1.)  The cache
 * rows [0, C_w) must hold the summaries of the earlier windows, as
 * focus_compact_kv leaves them; windows may be listed in any order and mixed
 * across sequences (the masked-parallel form of A.1), or one at a time
 * (streaming, A.2).  Windows listed first are started first: list the ones
 * with the largest C_w + T_w first.
 *   softmax_scale <= 0 selects 1/sqrt(head_dim).
 *   Supported: head_dim 64 or 128, bf16 or f32, n_heads a multiple of n_kv_heads.
 * FOCUS_MASK_KMER_LOCAL reads the window's own summaries from its window rows
 * (k-mer j of a window with cadence k spans window rows [j (k+1), j (k+1) + k],
 * its summary last, as focus_layout places them) and needs each window's k:
 * win_kmer (the per-window array given to focus_layout) or kmer_uniform.
 */
typedef struct {
  focus_layout_totals totals;
  int32_t dtype;
  int32_t n_heads;
  int32_t n_kv_heads;
  int32_t head_dim;
  float softmax_scale;
  int32_t mask;                 /* focus_mask                                */
  int32_t batch;
  int32_t kmer_uniform;         /* k of every window if win_kmer is NULL
                                   (FOCUS_MASK_KMER_LOCAL only; >= 0)        */
  int64_t n_win;                /* entries of win_ids (ignored if NULL)      */
  const int32_t* win_ids;       /* [device] or NULL = all windows, in the
                                   order last window first                   */
  const int32_t* win_seq;       /* [device] layout arrays                    */
  const int32_t* win_ntok;
  const int32_t* win_cache_off;
  const int64_t* win_tok_off;
  const int32_t* win_kmer;      /* [device][n_windows] k per window, or NULL
                                   (FOCUS_MASK_KMER_LOCAL only)              */
  const void* q;                /* [qkv_rows, n_heads, head_dim]             */
  const void* k;                /* [qkv_rows, n_kv_heads, head_dim]          */
  const void* v;                /*   row r = global token qkv_tok_base + r   */
  int64_t qkv_tok_base;
  int64_t qkv_rows;
  const void* cache_k;          /* [batch, cache_cap, n_kv_heads, head_dim]  */
  const void* cache_v;
  int64_t cache_cap;
  void* o;                      /* [qkv_rows, n_heads, head_dim], dtype      */
  float* lse;                   /* [qkv_rows, n_heads] float32, or NULL      */
  void* workspace;              /* optional key-split scratch (see below)    */
  size_t workspace_bytes;
  int32_t* err;
} focus_attn_desc;

/* Workspace bytes that let focus_window_attn split keys for this descriptor
 * on the current device (0 when it would not split).  A bf16 C(t) launch whose
 * (window, head, query tile) items are too few to occupy every compute unit
 * (one window per call) splits each item's key tiles over n workgroups, which
 * write unnormalised float32 partials to the workspace, merged by a second
 * kernel through their log-sum-exp (results differ from the unsplit ones by
 * float32 rounding only).  The workspace is optional: with d->workspace NULL,
 * not 16-byte aligned or smaller than this, the launch runs unsplit.  It is
 * scratch for the duration of the call; calls that share one on overlapping
 * streams race. */
size_t focus_window_attn_workspace(const focus_attn_desc* d);
/* Errors: E_NULL, E_ARG, E_DTYPE, E_SHAPE, E_UNSUPPORTED, E_CAPACITY (plan's
 * max_window_cache > cache_cap), E_HIP.  A window whose rows fall outside the
 * buffers is skipped with FOCUS_ERR_BOUNDS. */
focus_status focus_window_attn(const focus_attn_desc* d, focus_stream_t stream);

/* ------------------------------------------------------------------------ */
/* Decode                                                                    */
/* ------------------------------------------------------------------------ */

/* One autoregressive step for every sequence b of a batch (Appendix A.2,
 * streaming inference with the retained summary cache):
 *   1. append (k_new[b], v_new[b]) to the cache at row cache_len[b] if
 *      kind[b] & FOCUS_STEP_SUMMARY, else to the window buffer at row
 *      win_len[b]; bump that length;
 *   2. o[b, h] = softmax(scale * q[b, h] . [cache[0:cache_len] ;
 *      win[0:win_len]]^T) . values, every row visible; lse likewise;
 *   3. if kind[b] & FOCUS_STEP_WINDOW_END, set win_len[b] = 0 afterwards.
 * focus_decode_next_kind derives kind on the device from each sequence's
 * position in the layout (a summary every k bases, the last summary of a
 * window ends it).  Keys are split into chunks of split_keys rows
 * processed in parallel and merged by log-sum-exp; results do not depend on
 * the split beyond float32 rounding, and are deterministic for a fixed split.
 * All state lives in device memory, so steps can be enqueued back to back
 * without host synchronisation.
 */
typedef struct {
  int32_t dtype;
  int32_t batch;
  int32_t n_heads;
  int32_t n_kv_heads;
  int32_t head_dim;             /* 64 or 128                                 */
  float softmax_scale;          /* <= 0: 1/sqrt(head_dim)                    */
  int32_t split_keys;           /* keys per split, multiple of 16; 0 = auto:
                                   batch x capacity spread over about 7/8 of
                                   the current device's compute units        */
  int32_t reserved;
  const void* q;                /* [batch, n_heads, head_dim]                */
  const void* k_new;            /* [batch, n_kv_heads, head_dim]             */
  const void* v_new;
  const uint8_t* kind;          /* [device][batch] FOCUS_STEP_* bits         */
  void* cache_k;                /* [batch, cache_cap, n_kv_heads, head_dim]  */
  void* cache_v;
  int64_t cache_cap;
  int32_t* cache_len;           /* [device][batch] in/out                    */
  void* win_k;                  /* [batch, win_cap, n_kv_heads, head_dim]    */
  void* win_v;
  int64_t win_cap;
  int32_t* win_len;             /* [device][batch] in/out                    */
  void* o;                      /* [batch, n_heads, head_dim]                */
  float* lse;                   /* [batch, n_heads] or NULL                  */
  void* workspace;
  size_t workspace_bytes;
  int32_t* err;
} focus_decode_desc;

/* Workspace bytes for the split partials of this descriptor. */
size_t focus_decode_workspace(const focus_decode_desc* d);
/* Errors: E_NULL, E_ARG, E_DTYPE, E_SHAPE, E_UNSUPPORTED, E_WORKSPACE, E_HIP.
 * An append into a full cache or window buffer is skipped with
 * FOCUS_ERR_CAPACITY (the step still attends over what is there). */
focus_status focus_decode_step(const focus_decode_desc* d, focus_stream_t stream);

/* Decode schedule: where each sequence of a decode batch stands in the
 * summary layout, followed token by token (the insertion rule of Section 3.2
 * and Appendix A: a summary after every k_w bases of window w, a trailing
 * partial k-mer closed by one at the window's end; Appendix A.2 streaming).
 * The next token of sequence b is a summary when its window's cadence k > 0
 * and either the open k-mer holds k bases or the window holds W bases with a
 * k-mer open; it ends the window when it is that window's last summary (or,
 * for k = 0, its W-th base).  All arrays [device][batch] unless noted. */
typedef struct {
  int32_t batch;
  int32_t window_nt;            /* W, bases per window, >= 1                 */
  int32_t kmer_uniform;         /* cadence of every window when kmer == NULL */
  int32_t kmer_stride;          /* cadences per sequence in kmer (>= 1)      */
  const int32_t* kmer;          /* [batch][kmer_stride] or NULL: cadence of
                                   window j of sequence b at
                                   kmer[b * kmer_stride + min(j, stride - 1)] */
  int32_t* win_index;           /* in/out: the sequence's current window j   */
  int32_t* bases_in_window;     /* in/out: bases of window j so far          */
  int32_t* bases_in_kmer;       /* in/out: bases of its open k-mer           */
  uint8_t* kind;                /* out, focus_decode_next_kind: FOCUS_STEP_*
                                   bits of the next token (the kind argument
                                   of focus_decode_step)                     */
  const int32_t* tokens;        /* in, focus_decode_sched_start: tokens of
                                   window j already in the cache / window    */
  int32_t* summaries;           /* out, focus_decode_sched_start (or NULL):
                                   how many of those tokens are summaries    */
  int32_t* err;                 /* optional error word                       */
} focus_decode_sched;

/* Set bases_in_window / bases_in_kmer of every sequence by walking tokens[b]
 * tokens from the start of its window win_index[b] with the rule above (a
 * walk that closes the window moves on to the next one); summaries[b] gets
 * the number of summary tokens walked.  Use it to start decoding part-way
 * into a window.  A negative cadence raises FOCUS_ERR_BOUNDS and counts as 0.
 * Errors: E_NULL, E_ARG, E_HIP. */
focus_status focus_decode_sched_start(const focus_decode_sched* s, focus_stream_t stream);

/* Derive the kind of every sequence's next token into s->kind and advance
 * the counters past it (a window end moves to the next window).  Enqueue it
 * before each focus_decode_step that takes s->kind.  Errors: E_NULL, E_ARG,
 * E_HIP. */
focus_status focus_decode_next_kind(const focus_decode_sched* s, focus_stream_t stream);

/* Bytes of device scratch behind focus_decode_step_noalloc (16 MiB per GPU).
 * With the automatic split on a 256-CU device and 32 heads x 128, the split
 * partials (what focus_decode_workspace reports) take under 12 MiB for
 * batches up to 700 at any cache length; explicit small split_keys values
 * can need more. */
#define FOCUS_DECODE_SCRATCH_BYTES (16u << 20)

/* focus_decode_step for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): the same step, with the split partials kept in a scratch array
 * of FOCUS_DECODE_SCRATCH_BYTES that the library holds on each GPU it runs on
 * until the process ends.  d->workspace and d->workspace_bytes are ignored;
 * every other argument means what it means for focus_decode_step.  The call
 * allocates nothing (no hipMalloc / hipFree); its first call on a device
 * looks the array's device address up once.  Every call on one GPU shares
 * that GPU's array: calls that overlap on one GPU (other streams, other host
 * threads) race and must be serialised by the caller.
 * Errors: those of focus_decode_step; E_WORKSPACE when the step's partials
 * (focus_decode_workspace(d)) exceed FOCUS_DECODE_SCRATCH_BYTES; E_HIP when
 * the array's address cannot be obtained. */
focus_status focus_decode_step_noalloc(const focus_decode_desc* d, focus_stream_t stream);

/* ------------------------------------------------------------------------ */
/* Fidelity metrics                                                          */
/* ------------------------------------------------------------------------ */

/* Per-position distances between the base model's next-base distribution p_t
 * and the FOCUS model's q_t over `vocab` categories (Appendix "Metrics"):
 *   out[t, 0] = L1          sum_i |p_i - q_i|
 *   out[t, 1] = L2          (sum_i (p_i - q_i)^2)^(1/2)
 *   out[t, 2] = Hellinger   || sqrt p - sqrt q ||_2 / sqrt 2
 *   out[t, 3] = JS          (KL(p || m) + KL(q || m)) / 2,  m = (p + q) / 2
 *   out[t, 4] = KL          KL(p || q) = sum_i p_i ln(p_i / q_i)   (nats)
 * Both distributions are clipped from below at 1e-12 and renormalised before
 * every metric.  With FOCUS_FID_LOGITS the inputs are logits and the softmax
 * is taken first; with FOCUS_FID_PROBS they are probabilities.  Arithmetic is
 * float32.  If seq_mean is given, seq_mean[b, m] is the mean of out[t, m] over
 * t in [cu_pos[b], cu_pos[b+1]) (0 for an empty sequence), the sequence-level
 * score of the appendix; it needs out (unless n_pos is 0).
 */
enum { FOCUS_FID_LOGITS = 0, FOCUS_FID_PROBS = 1 };
enum { FOCUS_FID_L1 = 0, FOCUS_FID_L2 = 1, FOCUS_FID_HELLINGER = 2, FOCUS_FID_JS = 3, FOCUS_FID_KL = 4,
       FOCUS_FID_N = 5 };

typedef struct {
  int32_t dtype;                /* of p and q: FOCUS_BF16 or FOCUS_F32       */
  int32_t input_kind;           /* FOCUS_FID_LOGITS or FOCUS_FID_PROBS       */
  int64_t n_pos;                /* positions (rows of p and q)               */
  int32_t vocab;                /* categories per row, 1 .. 1024             */
  int32_t n_seq;                /* sequences of seq_mean (0: none)           */
  const void* p;                /* [device][n_pos, vocab] row-major           */
  const void* q;                /* [device][n_pos, vocab]                     */
  float* out;                   /* [device][n_pos, FOCUS_FID_N]               */
  const int64_t* cu_pos;        /* [device][n_seq + 1] row offsets, or NULL  */
  float* seq_mean;              /* [device][n_seq, FOCUS_FID_N], or NULL      */
  int32_t* err;                 /* optional error word                       */
} focus_fidelity_desc;

/* Errors: E_NULL, E_ARG (vocab, n_pos, input_kind, alignment: p and q aligned
 * to their element size, out and seq_mean to 4 bytes; seq_mean without out or
 * cu_pos), E_DTYPE, E_UNSUPPORTED (vocab > 1024), E_HIP.  Sequences whose
 * offsets fall outside [0, n_pos] get FOCUS_ERR_BOUNDS and a zero mean. */
focus_status focus_fidelity(const focus_fidelity_desc* d, focus_stream_t stream);

/* ------------------------------------------------------------------------ */
/* FOCUS adapter attention                                                   */
/* ------------------------------------------------------------------------ */

/* The summary tokens' attention of the FOCUS adapter (Appendix A eq.
 * focus-attn): for every listed window w of sequence b, every head h and every
 * summary s of w (global summary index, token t = sum_tok[s], window row
 * i = t - win_tok_off[w]):
 *     keys     = [cache_k[b, 0:C_w, g] ; k[window rows, g]],  g = h / (H / H_kv)
 *     visible  = as focus_window_attn's row i under `mask` (C(t): the paper's
 *                visible set of the adapter; k-mer-local: Sec. 3.2's own k-mer
 *                plus earlier summaries of the window plus the carried boundary)
 *     o_sum[s - sum_base, h]   = softmax(scale * q_sum[s - sum_base, h] . keys^T) . values
 *     lse_sum[s - sum_base, h] = log sum_visible exp(...)
 * k / v hold the adapter's key / value projections of the window tokens (row
 * r = token kv_tok_base + r); cache_k / cache_v those of the earlier windows'
 * summaries, as focus_compact_kv leaves them.  Only the summary queries are
 * computed (B_w per window instead of T_w).  bf16 only.
 * Errors: as focus_window_attn; E_UNSUPPORTED for f32.  A window whose rows or
 * summaries fall outside the buffers is skipped with FOCUS_ERR_BOUNDS. */
typedef struct {
  focus_layout_totals totals;
  int32_t dtype;                /* FOCUS_BF16                                */
  int32_t n_heads;
  int32_t n_kv_heads;
  int32_t head_dim;             /* 64 or 128                                 */
  float softmax_scale;          /* <= 0: 1/sqrt(head_dim)                    */
  int32_t mask;                 /* focus_mask                                */
  int32_t batch;
  int32_t kmer_uniform;         /* as in focus_attn_desc                     */
  int64_t n_win;
  const int32_t* win_ids;       /* [device] or NULL = all windows            */
  const int32_t* win_seq;       /* [device] layout arrays                    */
  const int32_t* win_ntok;
  const int32_t* win_cache_off;
  const int64_t* win_tok_off;
  const int32_t* win_kmer;      /* as in focus_attn_desc                     */
  const int32_t* win_nsum;
  const int64_t* win_sum_off;
  const int64_t* sum_tok;
  const void* q_sum;            /* [sum_rows, n_heads, head_dim]             */
  int64_t sum_base;             /* global summary index of row 0             */
  int64_t sum_rows;
  const void* k;                /* [kv_rows, n_kv_heads, head_dim]           */
  const void* v;
  int64_t kv_tok_base;
  int64_t kv_rows;
  const void* cache_k;          /* [batch, cache_cap, n_kv_heads, head_dim]  */
  const void* cache_v;
  int64_t cache_cap;
  void* o_sum;                  /* [sum_rows, n_heads, head_dim]             */
  float* lse_sum;               /* [sum_rows, n_heads] or NULL               */
  int32_t* err;
} focus_adapter_desc;

focus_status focus_adapter_attn(const focus_adapter_desc* d, focus_stream_t stream);

/* The whole adapter update of the summary tokens at one layer (eq. focus-attn
 * with the output projection), over every window of the layout:
 *     K = hidden W_K, V = hidden W_V               (every token; focus_gemm)
 *     cache = K, V rows of the summary tokens      (focus_compact_kv)
 *     Q = hidden[sum_tok] W_Q                      (summary tokens only)
 *     A = focus_adapter_attn(Q, K, V, cache, mask)
 *     out = A W_O                                  ([n_summaries, d_model])
 * hidden [n_tokens, d_model] (global token order); w_q [d_model, H D]; w_k, w_v
 * [d_model, H_kv D]; w_o [H D, d_model]; all bf16, row-major.  Intermediates
 * live in the caller's workspace (size from focus_adapter_layer_workspace).
 * Requirements: d_model a multiple of 128 and of 64; H D and H_kv D multiples of
 * 128.  Errors: as the calls above. */
typedef struct {
  focus_layout_totals totals;
  int32_t dtype;                /* FOCUS_BF16                                */
  int32_t n_heads;
  int32_t n_kv_heads;
  int32_t head_dim;             /* 64 or 128                                 */
  int32_t d_model;
  float softmax_scale;          /* <= 0: 1/sqrt(head_dim)                    */
  int32_t mask;                 /* focus_mask                                */
  int32_t batch;
  int32_t kmer_uniform;
  int32_t reserved;
  const int32_t* win_seq;       /* [device] layout arrays                    */
  const int32_t* win_ntok;
  const int32_t* win_cache_off;
  const int64_t* win_tok_off;
  const int32_t* win_kmer;
  const int32_t* win_nsum;
  const int64_t* win_sum_off;
  const int64_t* sum_tok;
  const void* hidden;           /* [n_tokens, d_model]                       */
  const void* w_q;
  const void* w_k;
  const void* w_v;
  const void* w_o;
  void* out;                    /* [n_summaries, d_model]                    */
  void* workspace;
  size_t workspace_bytes;
  int32_t* err;
} focus_adapter_layer_desc;

size_t focus_adapter_layer_workspace(const focus_adapter_layer_desc* d);
focus_status focus_adapter_layer(const focus_adapter_layer_desc* d, focus_stream_t stream);

/* ------------------------------------------------------------------------ */
/* Projections                                                               */
/* ------------------------------------------------------------------------ */

/* bf16 matrix product with float32 accumulation, for the projections around
 * the attention (the FOCUS adapter's W_Q, W_K, W_V, W_O of Appendix A eq.
 * focus-attn, and the layer's Q/K/V projection):
 *     C[i, n] = alpha * sum_k A[r(i), k] * B[k, n],  0 <= i < m, 0 <= n < n,
 *     r(i) = a_rows ? a_rows[i] : i
 * A, B, C row-major with leading dimensions lda, ldb, ldc (elements).  a_rows
 * (device, int64) gathers rows of A, e.g. the hidden states of the summary
 * tokens (sum_tok of focus_layout).  C is bf16 (round to nearest even) or f32.
 * Requirements: k a multiple of 64, n a multiple of 128, lda and ldb multiples
 * of 8, A and B 16-byte aligned.  Errors: E_NULL, E_ARG, E_DTYPE,
 * E_UNSUPPORTED (k or n not a multiple of the tile), E_SHAPE, E_HIP.  A gathered
 * row outside [0, a_nrows) reads row 0 instead and sets FOCUS_ERR_BOUNDS. */
typedef struct {
  int64_t m, n, k;
  const void* a;                /* [device] bf16, rows of lda elements       */
  int64_t lda;
  const int64_t* a_rows;        /* [device][m] row of A for each row of C, or NULL */
  int64_t a_nrows;              /* rows of A (a_rows entries must be below)  */
  const void* b;                /* [device] bf16 [k, ldb]                    */
  int64_t ldb;
  void* c;                      /* [device] [m, ldc] of c_dtype              */
  int64_t ldc;
  int32_t c_dtype;              /* FOCUS_BF16 or FOCUS_F32                   */
  float alpha;
  int32_t* err;                 /* optional error word                       */
} focus_gemm_desc;

focus_status focus_gemm(const focus_gemm_desc* d, focus_stream_t stream);

/* The layer's Q/K/V projection with FOCUS-aware rotary positions and the
 * compaction fused into its store (the step before the hot path; App. A: the
 * compression is effected by which K/V rows are retained):
 *     [Q | K | V] = hidden W_qkv          (rows = tokens tok_base .. +n_rows)
 *     Q, K rotated by RoPE at tok_pos[t], the token's index in its sequence's
 *     augmented stream (summary tokens hold real positions, Sec. 3.2 / App. A):
 *     pairs (2i, 2i+1) of each head turn by tok_pos * theta^(-2i/D)
 *     K, V rows of summary tokens are also written to cache row tok_kmer[t]
 *     of sequence win_seq[tok_win[t]], and cache_len raised past it.
 * w_qkv [d_model, (H + 2 H_kv) D] holds the Q heads, then the K heads, then the
 * V heads; q [n_rows, H, D], k / v [n_rows, H_kv, D]; all bf16 (float32
 * accumulation and rotation, then rounding).  rope_theta <= 0 skips the
 * rotation.  cache_k NULL skips the cache write.  Requirements: (H + 2 H_kv) D
 * a multiple of 128, d_model a multiple of 64, hidden and w_qkv 16-byte
 * aligned, q, k, v and the caches 4-byte aligned.  Errors: E_NULL, E_ARG, E_DTYPE,
 * E_SHAPE, E_UNSUPPORTED (f32, tile multiples), E_CAPACITY (whole layout and
 * cache_cap < max_cache_per_seq), E_HIP; a cache row outside the cache is
 * skipped with FOCUS_ERR_CAPACITY. */
typedef struct {
  focus_layout_totals totals;
  int32_t dtype;                /* FOCUS_BF16                                */
  int32_t n_heads;
  int32_t n_kv_heads;
  int32_t head_dim;             /* 64 or 128                                 */
  int32_t d_model;
  int32_t batch;
  float rope_theta;             /* RoPE base, > 1; <= 0: no rotation         */
  int32_t reserved;
  const int32_t* tok_pos;       /* [device] layout arrays                    */
  const uint8_t* tok_kind;
  const int32_t* tok_kmer;
  const int32_t* tok_win;
  const int32_t* win_seq;
  int64_t tok_base;             /* global token of hidden row 0              */
  int64_t n_rows;
  const void* hidden;           /* [n_rows, d_model]                         */
  const void* w_qkv;            /* [d_model, (H + 2 H_kv) D]                 */
  void* q;                      /* [n_rows, H, D]                            */
  void* k;                      /* [n_rows, H_kv, D]                         */
  void* v;
  void* cache_k;                /* [batch, cache_cap, H_kv, D] or NULL       */
  void* cache_v;
  int64_t cache_cap;
  int32_t* cache_len;           /* [device][batch] or NULL                   */
  int32_t* err;
} focus_qkv_desc;

focus_status focus_qkv_project(const focus_qkv_desc* d, focus_stream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* FOCUS_H */
