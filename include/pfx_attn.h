/*
 * pfx_attn.h -- shared-prefix paged attention for AMD MI355X (gfx950).
 *
 * The C interface of libpfxattn.so.  It follows the problem statement of
 * TOPAS ("Workflow-Aware Prefix-State Scheduling for Multi-Agent LLM
 * Serving"):
 *   - requests of one agent share that agent's static prefix, whose KV lives
 *     once in the GPU pool and is reused by all of them; each request then
 *     appends its own dynamic content (Sec. 1, the radix-tree prefix cache;
 *     Sec. 3, "Workflow and objective": prefix length l_a per agent);
 *   - a request may run only while its agent's prefix is resident, and the
 *     resident prefixes plus the requests' own KV must fit the KV budget,
 *     with each prefix counted once (Sec. 3, Eq. (2));
 *   - prefix KV moves between host and GPU memory as agents enter and leave
 *     the resident set (Sec. 4.2, Eq. (8) and the paragraph before it).
 * The attention these calls compute is the textbook causal softmax attention
 * over [agent prefix ; request suffix] (the paper states no numerics of its
 * own); how the work is split and recombined does not change the result
 * beyond floating-point rounding.
 *
 * Conventions shared by every call
 *   - Every call returns an int status: PFX_OK or one of the negative codes
 *     below.  No call aborts or throws; pfx_last_error() returns a
 *     thread-local message describing the last failure on this thread.
 *   - Arguments are validated before anything is launched: a call that fails
 *     validation launches nothing and writes nothing.
 *   - Device work is asynchronous on the HIP stream passed in (a hipStream_t
 *     cast to void*; NULL is the default stream).  Errors raised later by the
 *     device surface through pfx_sync_check().
 *   - All buffers are borrowed from the caller: the library never frees them
 *     and never allocates device memory.  A buffer must stay valid until the
 *     stream work that uses it has finished.  The one piece of device memory
 *     the library holds itself is the static array behind
 *     pfx_attention_noalloc (PFX_NOALLOC_MAX_WORKSPACE bytes per GPU).
 *   - bf16 means IEEE binary32 truncated to its upper 16 bits (bfloat16).
 *   - Page size is fixed at 16 tokens; head_dim must be 64 or 128; the query
 *     group G = num_q_heads / num_kv_heads must be 1, 2, 4, 8 or 16; query
 *     head h reads KV head h / G (consecutive query heads share a KV head).
 */
#ifndef PFX_ATTN_H
#define PFX_ATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define PFX_VERSION 20200 /* 2.2.0 */

#define PFX_OK 0
#define PFX_EINVAL (-1)       /* malformed argument (null pointer, bad CSR, overlapping pages, ...) */
#define PFX_ERANGE (-2)       /* a page id or a length is out of range */
#define PFX_ENOMEM (-3)       /* KV budget of Sec. 3, Eq. (2) exceeded; workspace too small */
#define PFX_EUNSUPPORTED (-4) /* head_dim, page size or query group not supported */
#define PFX_EHIP (-5)         /* the HIP runtime reported an error */

#define PFX_PAGE_SIZE 16

#define PFX_MODE_EXTEND 1 /* any number of query rows per request */
#define PFX_MODE_DECODE 2 /* at most one query row per request */
#define PFX_MODE_MIXED 3  /* both kinds in one batch */

/* Library version (PFX_VERSION of the build). */
int pfx_version(void);

/* Message for the last non-OK status returned on the calling thread
 * ("" if none).  The string stays valid until the next failing call on the
 * same thread. */
const char* pfx_last_error(void);

/*
 * KV page pool (Sec. 1: paged KV cache; Sec. 3: the resident prefix set and
 * the running requests share one KV budget).
 *
 * k_pages and v_pages each point to bf16 [num_pages][num_kv_heads][16][head_dim]:
 * inside a page the layout is head-major, so one (page, KV head) is a
 * contiguous 16 * head_dim * 2 byte block.  Page p of K starts at byte
 * p * num_kv_heads * 16 * head_dim * 2.  The memory is caller-owned device
 * memory, or host memory from hipHostMalloc (which the GPU can read and
 * write) when the descriptor names a host page store for pfx_page_copy.
 */
typedef struct pfx_pool {
  int32_t num_pages;
  int32_t page_size; /* must be PFX_PAGE_SIZE */
  int32_t num_kv_heads;
  int32_t head_dim; /* 64 or 128 */
  void* k_pages;
  void* v_pages;
} pfx_pool;

/*
 * Prefix table: agent a's static prefix (Sec. 3, length l_a) occupies the
 * ordered pages page_ids[page_indptr[a] .. page_indptr[a+1]) -- the pages of
 * its radix-tree path (Sec. 1) -- and has prefix_len[a] tokens.  Token j of
 * the prefix is slot j % 16 of page page_ids[page_indptr[a] + j / 16].  The
 * page count must equal ceil(prefix_len[a] / 16).  Host arrays.
 */
typedef struct pfx_prefix_table {
  int32_t num_agents;
  const int32_t* page_indptr; /* [num_agents + 1], page_indptr[0] == 0 */
  const int32_t* page_ids;    /* [page_indptr[num_agents]] */
  const int32_t* prefix_len;  /* [num_agents] */
} pfx_prefix_table;

/*
 * A batch of admitted requests (Sec. 3: the running set Q', each request
 * tied to its agent a(r), whose prefix must be resident).
 *   agent[r]           agent id, or -1 for a request with no shared prefix;
 *   suffix pages       suffix_page_ids[suffix_indptr[r] .. suffix_indptr[r+1]),
 *                      exactly ceil(suffix_len[r] / 16) pages; token j of the
 *                      suffix is slot j % 16 of the (j / 16)-th page;
 *   suffix_len[r]      L_r, the request's own KV tokens *including* the n_r
 *                      tokens of this step;
 *   q_indptr           request r owns query rows q_indptr[r] .. q_indptr[r+1]
 *                      (n_r of them, 0 <= n_r <= L_r); row i of the request
 *                      is the token at suffix position L_r - n_r + i.
 * A prefix page may never double as a suffix page, no page may appear twice,
 * and a suffix starts on its own page.  Host arrays.
 */
typedef struct pfx_batch {
  int32_t num_reqs;
  const int32_t* agent;           /* [num_reqs] */
  const int32_t* suffix_indptr;   /* [num_reqs + 1], suffix_indptr[0] == 0 */
  const int32_t* suffix_page_ids; /* [suffix_indptr[num_reqs]] */
  const int32_t* suffix_len;      /* [num_reqs] */
  const int32_t* q_indptr;        /* [num_reqs + 1], q_indptr[0] == 0 */
} pfx_batch;

/* ---------------------------------------------------------------------
 * Page allocator (host side, deterministic).  Sec. 3, Eq. (2): the pool's
 * pages are the token-equivalent KV budget B_t.  Pages are handed out LIFO
 * from a free list that starts as 0, 1, ..., num_pages - 1 (0 first).
 * pfx_alloc_pages writes n ids to out_ids, or returns PFX_ENOMEM and hands
 * out nothing when fewer than n pages are free.  pfx_free_pages returns
 * PFX_EINVAL (and frees nothing) if an id is out of range or not allocated.
 * --------------------------------------------------------------------- */
typedef struct pfx_alloc pfx_alloc;
int pfx_alloc_create(int32_t num_pages, pfx_alloc** out);
int pfx_alloc_pages(pfx_alloc* alloc, int32_t n, int32_t* out_ids);
int pfx_free_pages(pfx_alloc* alloc, const int32_t* ids, int32_t n);
int pfx_alloc_num_free(const pfx_alloc* alloc, int32_t* out);
void pfx_alloc_destroy(pfx_alloc* alloc);

/* ---------------------------------------------------------------------
 * Plan: the device work list for one batch.
 *
 * pfx_plan_create validates the pool shape, the prefix table and the batch
 * (all host arrays; copied, so they may be freed afterwards), groups the
 * decode requests by agent (each prefix read once for all of an agent's
 * decode rows and a KV head), cuts the decode items into pieces of at most
 * piece_steps 32-key steps, and builds the extend blocks.  It
 * checks the budget of Sec. 3, Eq. (2) in pages:
 *     sum over distinct agents referenced of ceil(l_a / 16)
 *   + sum over requests of ceil(L_r / 16)   <=  num_pages,
 * returning PFX_ENOMEM otherwise; then PFX_ERANGE for ids or lengths out of
 * range and PFX_EINVAL for overlapping ownership or malformed arrays.
 * mode: PFX_MODE_DECODE rejects n_r > 1 (PFX_EINVAL).  opts may be NULL.
 * num_q_heads: Hq (a multiple of num_kv_heads).  The plan is host memory
 * owned by the library until pfx_plan_destroy.
 * --------------------------------------------------------------------- */
typedef struct pfx_plan pfx_plan;

typedef struct pfx_plan_opts {
  /* Workgroups of the decode launch (0 = automatic: one per decode piece,
   * handed out by the dispatcher; a smaller count makes them persistent,
   * each running several pieces through its LDS ring; never more than there
   * are pieces).  The work division does not depend on it, only its
   * timing. */
  int32_t decode_workers;
  /* Longest decode piece, in 32-key steps (0 = automatic: 16, or 64 when
   * the decode items hold at least 32768 steps; at most 64).  Shorter pieces
   * balance the workgroups better but give each decode row more partial
   * results to merge. */
  int32_t piece_steps;
  /* Engine of the decode pieces: PFX_DECODE_MFMA (0, the default: matrix
   * cores, and wide prefix blocks for agents with more than 64 decode
   * columns per KV head) or PFX_DECODE_VALU (two-wide bf16 dot products on
   * the vector ALU, no wide blocks).  Same results within rounding; the
   * vector-ALU engine is slower and is kept to compare the two on hardware
   * counters.  Extend blocks always run on the matrix cores. */
  int32_t decode_engine;
  int32_t reserved[5]; /* must be zero */
} pfx_plan_opts;

#define PFX_DECODE_MFMA 0
#define PFX_DECODE_VALU 1

typedef struct pfx_plan_stats {
  int32_t num_requests;
  int32_t num_tokens;        /* sum of n_r: query rows of the batch */
  int32_t num_items;           /* prefix + suffix + extend items */
  int32_t num_prefix_items;    /* grouped decode: (agent, block of <= 64 decode columns, KV head) over the prefix */
  int32_t num_suffix_items;    /* decode: (request, KV head) over the request's own suffix */
  int32_t num_extend_items;    /* extend blocks: (<= 128 columns of one request, KV head), one workgroup each */
  int32_t num_partial_rows;    /* partial result rows (one query head each) kept in the workspace */
  int32_t pages_needed;        /* left-hand side of the Eq. (2) check, in pages */
  int32_t num_decode_steps;    /* 32-key steps of all decode items */
  int32_t num_decode_pieces;   /* runs of at most piece_steps steps of one decode item */
  int32_t num_wide_blocks;     /* prefix pieces of agents with more than 64 decode columns per KV head,
                                  run 128 columns at a time (counted apart from num_decode_pieces) */
  int32_t reserved;
  int64_t workspace_bytes;
} pfx_plan_stats;

int pfx_plan_create(const pfx_pool* pool, const pfx_prefix_table* prefixes, const pfx_batch* batch,
                    int32_t num_q_heads, int32_t mode, const pfx_plan_opts* opts, pfx_plan** out);

/* Bytes of device workspace the plan needs (work lists, partial states). */
int pfx_plan_workspace_bytes(const pfx_plan* plan, size_t* bytes);

/* Counts describing the plan (host only). */
int pfx_plan_get_stats(const pfx_plan* plan, pfx_plan_stats* out);

/* Copy one of the plan's host arrays out, for inspection and tests:
 * which = 0: extend blocks, then wide prefix blocks, 32 int32 each;
 * 1: their row-token list; 8: the partial row base of each of those rows
 * (-1 for extend rows); 2: page list; 3: decode pieces, 272 int32 each
 * (header, row tokens, output rows, page blocks of the steps); 6: tokens
 * whose rows are merged; 7: their (base, count) of partial slots per KV
 * head.
 * Writes min(cap, size) values and sets *count to the full size. */
int pfx_plan_export(const pfx_plan* plan, int32_t which, int32_t* out, int64_t cap, int64_t* count);

/* Copy the plan into a caller-owned device workspace of at least
 * pfx_plan_workspace_bytes bytes (PFX_ENOMEM if smaller) and clear its
 * counters, asynchronously on the stream.  The plan remembers the workspace;
 * pfx_append_kv and pfx_attention use it until the next upload.  The
 * workspace (256-byte aligned) must not be shared by calls that may overlap. */
int pfx_plan_upload(pfx_plan* plan, void* dev_workspace, size_t bytes, void* hip_stream);

void pfx_plan_destroy(pfx_plan* plan);

/* ---------------------------------------------------------------------
 * KV append (each request appends its own dynamic content, Sec. 1).
 * k_new, v_new: device bf16 [num_tokens][num_kv_heads][head_dim], rows in
 * request order (q_indptr).  Row i of request r is written to suffix
 * position L_r - n_r + i of the pool (K and V).  Only those slots are
 * written; prefix pages never are.  Bit-exact copy.  The pool must have the
 * shape the plan was created for; the plan must be uploaded.
 * --------------------------------------------------------------------- */
int pfx_append_kv(const pfx_pool* pool, const pfx_plan* plan, const void* k_new, const void* v_new,
                  void* hip_stream);

/* ---------------------------------------------------------------------
 * Attention for every query row of the planned batch.
 * q: device bf16 [num_tokens][num_q_heads][head_dim] (rows by q_indptr);
 * o: device bf16, same shape, written (round to nearest even);
 * lse: device fp32 [num_tokens][num_q_heads], natural-log log-sum-exp of
 *      the row's scaled scores (may be NULL).
 * Row i of request r at position t = l_a + L_r - n_r + i attends to the
 * whole prefix of its agent and to suffix tokens 0 .. L_r - n_r + i:
 *     O = sum_j softmax_j(sm_scale * q . k_j) v_j,
 * accumulated in fp32 from bf16 inputs.  sm_scale <= 0 selects
 * 1/sqrt(head_dim).  Prefix KV is read once per agent group and KV head;
 * the states of a decode row's pieces are combined with the log-sum-exp
 * merge (as pfx_merge_states), in a second launch on the same stream.
 * Results are deterministic: the same plan shape and inputs give
 * bit-identical outputs, wherever the pages sit.  Calls that share a plan
 * workspace must not overlap.
 * --------------------------------------------------------------------- */
int pfx_attention(const pfx_pool* pool, const pfx_plan* plan, const void* q, void* o, float* lse,
                  float sm_scale, void* hip_stream);

/* ---------------------------------------------------------------------
 * One step: the KV append of the step's new tokens (as pfx_append_kv)
 * followed by attention for every query row (as pfx_attention), with the
 * same results bit for bit, in the fewest launches.  When the plan has no
 * extend blocks, the decode launch appends as it goes: a decode request's
 * new tokens are read straight from k_new / v_new into the step that
 * attends them and written into their pool slots by the same workgroup (no
 * other work of the launch reads those slots).  Extend blocks read one
 * another's new tokens, so with extend blocks the append runs first as its
 * own launch.  Arguments as pfx_append_kv and pfx_attention; k_new and
 * v_new may be NULL only when the plan has no query rows.
 * --------------------------------------------------------------------- */
int pfx_step(const pfx_pool* pool, const pfx_plan* plan, const void* k_new, const void* v_new, const void* q,
             void* o, float* lse, float sm_scale, void* hip_stream);

/* ---------------------------------------------------------------------
 * Log-sum-exp merge of attention results computed over disjoint key ranges
 * (the same arithmetic pfx_attention applies to its decode pieces):
 *     lse = ln sum_k exp(lse_k),   O = sum_k exp(lse_k - lse) O_k.
 * o_parts: device fp32 [num_parts][rows][head_dim] (each O_k normalised
 * over its own keys); lse_parts: device fp32 [num_parts][rows];
 * o: device bf16 [rows][head_dim]; lse: device fp32 [rows] (may be NULL).
 * head_dim 64 or 128; 1 <= num_parts <= 4096.
 * --------------------------------------------------------------------- */
int pfx_merge_states(const float* o_parts, const float* lse_parts, int32_t num_parts, int32_t rows,
                     int32_t head_dim, void* o, float* lse, void* hip_stream);

/* ---------------------------------------------------------------------
 * Page copy: prefix movement between a host page store and the GPU pool
 * (Sec. 4.2, Eq. (8): an agent entering the resident set has its prefix
 * brought in, one leaving has it written out).  For i < n:
 *     dst page dst_pages[i]  <-  src page src_pages[i]   (K and V, all heads),
 * a bit-exact copy.  dst and src are pool descriptors with the same
 * num_kv_heads and head_dim; either may describe device memory or pinned
 * host memory (hipHostMalloc), so the same call loads (host -> GPU) and
 * evicts (GPU -> host).  src_pages and dst_pages are host arrays, checked
 * against the two page counts (PFX_ERANGE) and for repeated destinations
 * (PFX_EINVAL) before anything runs; they are staged in the caller's device
 * workspace (at least pfx_page_copy_workspace_bytes(n) bytes).  A page
 * array that is neither device memory nor pinned host memory is rejected
 * (PFX_EINVAL) before anything runs.
 * --------------------------------------------------------------------- */
size_t pfx_page_copy_workspace_bytes(int32_t n);
int pfx_page_copy(const pfx_pool* dst, const pfx_pool* src, const int32_t* dst_pages,
                  const int32_t* src_pages, int32_t n, void* dev_workspace, size_t workspace_bytes,
                  void* hip_stream);

/* ---------------------------------------------------------------------
 * Allocation-free attention step, for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc).  Same results as pfx_append_kv (when k_new and v_new
 * are given) followed by pfx_attention on the same plan, bit for bit; the
 * plan need not be uploaded and no caller workspace is used.  Instead the
 * plan's tables (copied from its host image on the stream at every call)
 * and the decode pieces' partial states live in a static device array of
 * PFX_NOALLOC_MAX_WORKSPACE bytes, which each GPU the library runs on holds
 * until the process ends.  The call allocates nothing: no hipMalloc, no
 * hipFree.
 *   k_new, v_new  as pfx_append_kv, or both NULL to skip the append;
 *   q, o, lse, sm_scale  as pfx_attention.
 * Errors: PFX_ENOMEM, before anything runs, when the plan's workspace
 * (pfx_plan_workspace_bytes) exceeds PFX_NOALLOC_MAX_WORKSPACE; PFX_EINVAL
 * when only one of k_new, v_new is NULL; otherwise as pfx_append_kv and
 * pfx_attention.
 * All calls on one GPU share that GPU's array and leave their contents in
 * it: calls that may overlap on one GPU (several streams or threads) race,
 * and the caller must serialise them.
 * --------------------------------------------------------------------- */
#define PFX_NOALLOC_MAX_WORKSPACE ((size_t)128 << 20) /* 128 MiB per GPU */
int pfx_attention_noalloc(const pfx_pool* pool, const pfx_plan* plan, const void* k_new, const void* v_new,
                          const void* q, void* o, float* lse, float sm_scale, void* hip_stream);

/* Wait for the stream and report any device-side error as PFX_EHIP. */
int pfx_sync_check(void* hip_stream);

#ifdef __cplusplus
}
#endif

#endif /* PFX_ATTN_H */
