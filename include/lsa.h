/*
 * lsa.h - C interface of the LongCat Sparse Attention (LSA) hot path on AMD Instinct MI355X
 * (gfx950).
 *
 * The operations follow "LongCat Sparse Attention: Taming the Lightning via Streaming-aware
 * Hierarchical Cross-Layer Indexing" (arXiv 2608.01662):
 *   - lightning-indexer score and top-K (Sec. 2.2, Eq. 1-2),
 *   - streaming-aware budget split into sink, sliding window and sparse part (Sec. 3.1, Eq. 6-7),
 *   - hierarchical coarse-to-fine selection (Sec. 3.3, Eq. 9-12),
 *   - sparse attention over the selected MLA latent rows (Sec. 2.2, Eq. 3),
 *   - cross-layer indexing (Sec. 3.2): one index list is passed unchanged to the attention of
 *     every layer in a group; there is no separate call for it.
 *
 * Conventions shared by every call
 *   - Tensor pointers are DEVICE pointers owned by the caller, row-major and contiguous, each
 *     aligned to 16 bytes. No call allocates device memory, frees anything, or synchronises the
 *     host: work is enqueued on `stream` (a hipStream_t; NULL = the default stream) and the
 *     caller orders it like any other kernel launch.
 *   - Positions are 0-based token positions (the paper counts from 1). The query at absolute
 *     position t may see positions 0..t. Sink = [0, k_sink), window = [t-k_swa+1, t], eligible
 *     range E_t = [k_sink, t-k_swa].
 *   - Every call checks its arguments on the host before any HIP call. On error it returns a
 *     non-zero lsa_status, launches nothing, and lsa_last_error() names the argument. Errors
 *     reported by the HIP runtime at launch time come back as LSA_ERR_HIP with the HIP message.
 *   - Device-side contents (positions in idx, page-table entries, context lengths) cannot be
 *     checked on the host. The kernels bound-check them instead: an out-of-range position or
 *     page is skipped (it selects or attends to nothing) and never dereferenced.
 *   - bf16 = bfloat16, fp8 = OCP e4m3fn (the gfx950 native format), both stored as raw bits.
 */
#ifndef LSA_H
#define LSA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum lsa_status {
  LSA_OK = 0,
  LSA_ERR_INVALID_ARG = 1, /* null / misaligned pointer, negative size, inconsistent sizes   */
  LSA_ERR_UNSUPPORTED = 2, /* valid request outside what the kernels implement               */
  LSA_ERR_WORKSPACE = 3,   /* workspace missing or smaller than the *_workspace_size value   */
  LSA_ERR_HIP = 4          /* the HIP runtime reported an error                             */
} lsa_status;

typedef enum lsa_key_dtype {
  LSA_KEY_BF16 = 0,        /* indexer keys in bf16                                           */
  LSA_KEY_FP8_E4M3FN = 1   /* indexer keys in fp8 with one fp32 scale per token (k = s * k8) */
} lsa_key_dtype;

/* Block summary of the coarse stage (Stage 1 of Sec. 3.3). */
typedef enum lsa_pooling {
  LSA_POOL_MEAN = 0,       /* one mean key per sub-block; block score q . k_mean (Eq. 9)        */
  LSA_POOL_MINMAX = 1      /* per-dimension extrema per sub-block; block score of Eq. 13          */
} lsa_pooling;
/* Hyper-parameters of one LSA indexer (Sec. 3.1 and Sec. 3.3). */
typedef struct lsa_index_params {
  int32_t n_heads;     /* H^I, indexer heads sharing one key (Eq. 1). 1..32                     */
  int32_t head_dim;    /* d_I, 64 or 128                                                         */
  int32_t key_dtype;   /* lsa_key_dtype                                                          */
  int32_t page;        /* P, page size of the coarse stage; multiple of 32, <= 256               */
  int32_t sub_block;   /* B, tokens per mean key (Eq. 9); divides P, P/B <= 32, power of two    */
  int32_t keep_pages;  /* M, pages recalled per query (Eq. 10). <= 0: flat selection over the
                          whole eligible range (Eq. 7), no coarse stage                           */
  int32_t k_sparse;    /* K_sparse, tokens chosen by the fine stage (Eq. 7 / Eq. 12)             */
  int32_t k_sink;      /* K_sink (Eq. 6)                                                          */
  int32_t k_swa;       /* K_swa (Eq. 6); must be >= P when keep_pages > 0, so that every scored
                          page lies entirely at or before the query                              */
  int32_t run_align;   /* C: runs are cut at every multiple of C (>= 1)                           */
  int32_t pooling;     /* lsa_pooling of the coarse stage (hierarchical mode only)               */
  int32_t hi_min_kv;   /* adaptive dispatch between hierarchical and flat indexing (Sec. 3.3: the
                          hierarchy pays off only beyond a crossover length): with keep_pages > 0,
                          a call whose cache covers at most hi_min_kv tokens (prefill: n_kv;
                          decode: max_pages * kv_page_size) runs flat, and its pages_out rows are
                          all -1. 0: always hierarchical when keep_pages > 0                      */
} lsa_index_params;

/* A run of consecutive selected positions [start, start+len) inside one C-aligned chunk. */
typedef struct lsa_run {
  int32_t start;
  int32_t len;
} lsa_run;

/* K_cap = k_sink + k_swa + k_sparse: the index budget K of Sec. 3.1, split by Eq. (6) into sink,
 * sliding window and sparse part; the row length of idx and runs. 0 for a NULL p. */
int32_t lsa_index_k_cap(const lsa_index_params* p);

/*
 * Workspace bytes for lsa_index_prefill (n_rows = n_q, max_kv = n_kv) or lsa_index_decode
 * (n_rows = batch, max_kv = max_pages * kv_page_size). Returns 0 when the parameters are invalid.
 */
size_t lsa_index_workspace_size(const lsa_index_params* p, int64_t n_rows, int64_t max_kv);

/*
 * Mean-key cache of Stage 1 (Sec. 3.3): block_keys[n] = per-dimension mean of the dequantised
 * keys s_i * k_i of tokens [n*B, n*B+B), accumulated in fp32 and rounded once to bf16.
 *   k          [n_tok, d_I] bf16 or fp8 codes (p->key_dtype)
 *   k_scale    [n_tok] fp32 per-token scale (fp8 keys), must be NULL for bf16 keys
 *   block_keys [n_tok / B, d_I] bf16 output; a trailing partial sub-block is not written.
 * For a paged cache pass the page pool as n_tok = n_pages * page_size tokens; page_size must be
 * a multiple of B so that no sub-block straddles two pages.
 */
lsa_status lsa_block_means(const lsa_index_params* p, int64_t n_tok, const void* k,
                           const float* k_scale, void* block_keys, void* stream);
/*
 * Min-max block cache (Eq. 13, the pooling ablation of hierarchical indexing): for sub-block n,
 * block_keys[n] = [k_max | k_min], the per-dimension maximum and minimum of the dequantised keys
 * s_i * k_i of tokens [n*B, n*B+B). Each extremum is taken exactly (products in fp64) and rounded
 * once to bf16, nearest-even. Arguments as lsa_block_means, except
 *   block_keys [n_tok / B, 2 * d_I] bf16 output.
 */
lsa_status lsa_block_minmax(const lsa_index_params* p, int64_t n_tok, const void* k,
                            const float* k_scale, void* block_keys, void* stream);
/*
 * Maintenance of the Stage-1 block cache of Sec. 3.3 (mean keys of Eq. 9, or the extrema of
 * Eq. 13), which the paper computes once and keeps current as the sequence grows (the block-mean
 * maintenance it names among the hierarchy's costs).
 * Keeps a block cache current while tokens are appended (decode): recomputes, from the keys in
 * the cache, the summary of every sub-block that contains one of the n_rows token rows in `rows`
 * (mean keys as lsa_block_means, or [k_max | k_min] as lsa_block_minmax, by p->pooling). The
 * result is bit-identical to recomputing the whole cache.
 *   rows       [n_rows] int64 device array of token rows (physical rows of a paged pool); rows
 *              outside [0, n_tok) or in the incomplete trailing sub-block are skipped. A row may
 *              repeat; every copy writes the same value.
 *   n_tok, k, k_scale, block_keys as in lsa_block_means / lsa_block_minmax.
 */
lsa_status lsa_block_keys_update(const lsa_index_params* p, int64_t n_rows, const int64_t* rows,
                                 int64_t n_tok, const void* k, const float* k_scale,
                                 void* block_keys, void* stream);

/*
 * Indexer for prefill (Eq. 6-7, 9-12): query rows i = 0..n_q-1 at positions t = q_start + i of
 * one sequence whose first n_kv tokens are cached (requires q_start + n_q <= n_kv, n_kv < 2^31
 * and n_q < 2^28; longer prefills are issued in chunks through q_start).
 *   q          [n_q, H^I, d_I] bf16 indexer queries
 *   w          [n_q, H^I] fp32 head weights (any sign)
 *   k, k_scale [n_kv, d_I] keys (+ [n_kv] fp32 scales for fp8, NULL for bf16). Scales must be
 *              finite and >= 0: a token's scale multiplies its score after the ReLU and the head
 *              sum, which equals Eq. (1) on the dequantised key s*k only for s >= 0 (the
 *              per-token quantiser's max|k|/448 always is)
 *   block_keys [n_kv / B, d_I] bf16 from lsa_block_means, or [n_kv / B, 2 d_I] from
 *              lsa_block_minmax when p->pooling is LSA_POOL_MINMAX (ignored in flat mode, may be
 *              NULL)
 * Outputs (row i of each):
 *   idx        [n_q, K_cap] int32: S_t in ascending order = sink, then the K_sparse positions of
 *              largest score (ties to the smaller position), then the window; -1 after count[i]
 *   count      [n_q] int32: |S_t| = min(t+1, k_sink + k_swa + min(k_sparse, |candidates|))
 *   runs       [n_q, K_cap] lsa_run or NULL: idx re-encoded as maximal runs of consecutive
 *              positions, cut at multiples of run_align; entries past run_count[i] are not written
 *              (they keep whatever the buffer held); 8-byte aligned
 *   run_count  [n_q] int32, required iff runs != NULL
 *   pages_out  [n_q, M] int32 or NULL (hierarchical mode only): the recalled pages P_t (Eq. 10)
 *              in ascending order, -1 padded
 *   workspace  >= lsa_index_workspace_size(p, n_q, n_kv) bytes, 256-byte aligned
 * The same idx/count/runs feed the attention of every layer of a cross-layer group (Sec. 3.2).
 */
lsa_status lsa_index_prefill(const lsa_index_params* p, int64_t q_start, int64_t n_q, int64_t n_kv,
                             const void* q, const float* w, const void* k, const float* k_scale,
                             const void* block_keys, int32_t* idx, int32_t* count, lsa_run* runs,
                             int32_t* run_count, int32_t* pages_out, void* workspace,
                             size_t ws_bytes, void* stream);

/*
 * Indexer for decode (the decode setting of Table 1): Eq. (6)-(7) and, in hierarchical mode,
 * Eq. (9)-(12) for one query per sequence b at position t_b = ctx_len[b] - 1 (the new token
 * is already in the cache). Keys live in pages of kv_page_size tokens: logical position s of
 * sequence b is row s % kv_page_size of physical page page_table[b * max_pages + s / kv_page_size].
 * Hierarchical mode needs page == kv_page_size (one coarse page = one cache page).
 *   ctx_len     [batch] int32 device array, 1 <= ctx_len <= max_pages * kv_page_size
 *   page_table  [batch, max_pages] int32 device array of physical pages in [0, n_phys)
 *   k, k_scale  [n_phys * kv_page_size, d_I] keys (+ scales) of the page pool
 *   block_keys  [n_phys * kv_page_size / B, d_I] bf16 mean keys of the page pool
 *               ([.., 2 d_I] extrema with LSA_POOL_MINMAX)
 * Outputs as in lsa_index_prefill with n_q = batch. Rows whose ctx_len is out of range get
 * count = 0. A page whose page-table entry lies outside [0, n_phys) is scored 0 and gives no token
 * to the sparse part (its keys are never read); the row's sink and window positions are listed
 * whatever the table holds (lsa_sparse_attn skips the positions it cannot map).
 */
lsa_status lsa_index_decode(const lsa_index_params* p, int32_t batch, const int32_t* ctx_len,
                            const int32_t* page_table, int32_t max_pages, int32_t kv_page_size,
                            int64_t n_phys, const void* q, const float* w, const void* k,
                            const float* k_scale, const void* block_keys, int32_t* idx,
                            int32_t* count, lsa_run* runs, int32_t* run_count, int32_t* pages_out,
                            void* workspace, size_t ws_bytes, void* stream);

/*
 * lsa_index_decode without a workspace, for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid allocation). The indexer's
 * scratch (page-score keys, recalled pages and fine-score keys of a pass of rows) lives in a fixed
 * device array of LSA_STATIC_SCRATCH_BYTES inside the library, one per device, held until the
 * process ends; rows are processed in as many passes as that array requires. The call allocates
 * and frees nothing. Arguments and outputs as lsa_index_decode without workspace / ws_bytes;
 * the outputs are bit-identical to lsa_index_decode's.
 * Returns LSA_ERR_WORKSPACE (before any HIP call) when one query row needs more than the array
 * holds: 4 * (M * P + number of pages + M) bytes + 768 in hierarchical mode, 4 * (pages * P) + 768
 * flat, with pages = ceil(max_pages * kv_page_size / P).
 * Every call on one device shares that device's array: calls that overlap in time on one device
 * (several host threads, or several streams) race and must be serialised by the caller.
 */
#define LSA_STATIC_SCRATCH_BYTES ((size_t)32 << 20)
lsa_status lsa_index_decode_static(const lsa_index_params* p, int32_t batch, const int32_t* ctx_len,
                                   const int32_t* page_table, int32_t max_pages, int32_t kv_page_size,
                                   int64_t n_phys, const void* q, const float* w, const void* k,
                                   const float* k_scale, const void* block_keys, int32_t* idx, int32_t* count,
                                   lsa_run* runs, int32_t* run_count, int32_t* pages_out, void* stream);

/* Sparse attention shapes. Supported: MQA {n_heads 16, d_qk 128, d_v 128, latent 0} and
 * MLA absorbed {n_heads 64, d_qk 576, d_v 512, latent 1}. */
typedef struct lsa_attn_params {
  int32_t n_heads; /* query heads sharing one key/value head                                   */
  int32_t d_qk;    /* query/key width                                                          */
  int32_t d_v;     /* value width                                                              */
  int32_t latent;  /* 1: MLA latent cache, V = first d_v columns of the same row (Eq. 3)       */
  float sm_scale;  /* softmax scale applied to q . k                                           */
} lsa_attn_params;

/* Workspace bytes for lsa_sparse_attn (non-zero only for split calls and paged MQA calls). */
size_t lsa_sparse_attn_workspace_size(const lsa_attn_params* p, int64_t n_rows, int32_t k_cap,
                                      int32_t paged);

/*
 * Sparse attention, Eq. (3): for each row r and head h,
 *   o[r,h] = sum_{s in S_r} softmax_s(sm_scale * q[r,h] . k_s) v_s,
 *   lse[r,h] = log sum_{s in S_r} exp(sm_scale * q[r,h] . k_s)   (natural log),
 * with S_r = idx[r, 0..count[r]) (any order; entries outside [0, n_kv_rows) are skipped). A row
 * with an empty set gets o = 0 and lse = -inf.
 *   q          [n_rows, n_heads, d_qk] bf16
 *   kv         latent: [n_kv_rows, d_qk] bf16 (V = kv[:, :d_v]); otherwise K [n_kv_rows, d_qk]
 *   v          NULL when latent, else V [n_kv_rows, d_v] bf16
 *   idx, count [n_rows, k_cap] int32 / [n_rows] int32, e.g. straight from the indexer
 *   page_table NULL for a contiguous cache. Otherwise the cache is paged: position s of row r
 *              (sequence r / rows_per_seq) is row s % kv_page_size of physical page
 *              page_table[(r / rows_per_seq) * max_pages + s / kv_page_size], and
 *              n_kv_rows = n_phys * kv_page_size.
 *   out        [n_rows, n_heads, d_v] bf16; lse [n_rows, n_heads] fp32 or NULL
 *   workspace  >= lsa_sparse_attn_workspace_size(p, n_rows, k_cap, page_table != NULL)
 * Cross-layer indexing: call once per layer with that layer's q and kv and the same idx/count.
 */
lsa_status lsa_sparse_attn(const lsa_attn_params* p, int64_t n_rows, const void* q, const void* kv,
                           const void* v, int64_t n_kv_rows, const int32_t* idx,
                           const int32_t* count, int32_t k_cap, const int32_t* page_table,
                           int32_t max_pages, int32_t kv_page_size, int32_t rows_per_seq,
                           void* out, float* lse, void* workspace, size_t ws_bytes, void* stream);

/*
 * Sparse attention, Eq. (3), over the run encoding of the index lists instead of idx/count: row
 * r attends to the concatenation of runs[r, 0..run_count[r]), run j covering positions
 * [start, start + len) (the runs output of lsa_index_prefill / lsa_index_decode). The result equals
 * lsa_sparse_attn over the same list, bit for bit. With a contiguous MLA latent cache the kernel
 * expands the runs itself while staging a row's list; otherwise (MQA, paged cache) the runs are
 * first expanded into a position list at the head of the workspace.
 *   runs       [n_rows, k_cap] lsa_run, 8-byte aligned; run_count [n_rows] int32, clamped to
 *              [0, k_cap]
 *   k_cap      row stride of runs and the list capacity: entries past k_cap are not attended;
 *              negative lengths count as 0; entries outside [0, n_kv_rows) are skipped
 *   workspace  >= lsa_sparse_attn_runs_workspace_size(p, n_rows, k_cap, page_table != NULL)
 * Other arguments (v, page_table, max_pages, kv_page_size, rows_per_seq) as lsa_sparse_attn.
 */
size_t lsa_sparse_attn_runs_workspace_size(const lsa_attn_params* p, int64_t n_rows, int32_t k_cap,
                                           int32_t paged);
lsa_status lsa_sparse_attn_runs(const lsa_attn_params* p, int64_t n_rows, const void* q,
                                const void* kv, const void* v, int64_t n_kv_rows, const lsa_run* runs,
                                const int32_t* run_count, int32_t k_cap, const int32_t* page_table,
                                int32_t max_pages, int32_t kv_page_size, int32_t rows_per_seq,
                                void* out, float* lse, void* workspace, size_t ws_bytes, void* stream);

/*
 * Split sparse attention of prefill (Sec. 4.1.1, the hybrid operator): the same result as
 * lsa_sparse_attn over S_t, computed as two partial attentions merged by online-softmax
 * (log-sum-exp) rescaling: the listed part of S_t without its sliding window (sink and sparse
 * positions: the first count[r] - min(k_swa, t+1) entries of the ascending list), and the window
 * [t - k_swa + 1, t] read as contiguous cache rows. The two run on two streams (the caller's and a
 * library-owned non-blocking one, default priority, joined by events before the merge), in passes
 * of 16384 rows. MLA latent cache only, contiguous cache only.
 *   q_start    position t of row 0 (row r is the query at t = q_start + r); q_start + n_rows <=
 *              n_kv_rows
 *   k_swa      the indexer's window size: idx must end with the whole window of each row, as
 *              lsa_index_prefill writes it (rows shorter than the window hold [0, t])
 *   workspace  >= lsa_hfa_attn_workspace_size(p, n_rows) bytes, 256-byte aligned (the partials)
 * Other arguments as lsa_sparse_attn. Calls on one device share the side stream and its two
 * events; the library enqueues one call's whole sequence under a lock, so concurrent calls from
 * several host threads are correct (their work on the side stream runs one call after the other).
 */
size_t lsa_hfa_attn_workspace_size(const lsa_attn_params* p, int64_t n_rows);
lsa_status lsa_hfa_attn(const lsa_attn_params* p, int64_t n_rows, const void* q, const void* kv, int64_t n_kv_rows,
                        const int32_t* idx, const int32_t* count, int32_t k_cap, int64_t q_start, int32_t k_swa,
                        void* out, float* lse, void* workspace, size_t ws_bytes, void* stream);
/* Human-readable name of a status code (static string). */
const char* lsa_status_string(int32_t status);

/* Message of the last failing call on this thread ("" if none). Valid until the next call. */
const char* lsa_last_error(void);

/* Library version, e.g. "lsa-mi355x 0.1". */
const char* lsa_version(void);

#ifdef __cplusplus
}
#endif

#endif /* LSA_H */
