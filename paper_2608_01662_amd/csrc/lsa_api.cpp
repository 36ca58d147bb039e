// C-ABI front end of the LSA library: argument checks (host only, before any HIP call),
// workspace layout, kernel selection and error reporting. See include/lsa.h.
#include "../../include/lsa.h"

#include <hip/hip_runtime.h>

#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>

#include "launch.hpp"

namespace {

thread_local char g_err[512] = "";
constexpr size_t kMaxLds = 160 * 1024;        // gfx950 LDS per workgroup
constexpr size_t kSelectStaticLds = 8 * 1024;  // static LDS of the page selection (upper bound)

lsa_status fail(lsa_status st, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return st;
}

lsa_status hip_fail(hipError_t e, const char* where) {
  return fail(LSA_ERR_HIP, "%s: %s", where, hipGetErrorString(e));
}

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }
bool pow2(int64_t x) { return x > 0 && (x & (x - 1)) == 0; }
size_t round_up(size_t x, size_t a) { return (x + a - 1) / a * a; }
int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

#define LSA_REQUIRE(cond, st, ...) \
  do {                             \
    if (!(cond)) return fail(st, __VA_ARGS__); \
  } while (0)

lsa_status check_index_params(const lsa_index_params* p) {
  LSA_REQUIRE(p != nullptr, LSA_ERR_INVALID_ARG, "params is NULL");
  LSA_REQUIRE(p->n_heads >= 1 && p->n_heads <= 32, LSA_ERR_UNSUPPORTED, "n_heads=%d not in [1, 32]", p->n_heads);
  LSA_REQUIRE(p->head_dim == 64 || p->head_dim == 128, LSA_ERR_UNSUPPORTED, "head_dim=%d not 64 or 128", p->head_dim);
  LSA_REQUIRE(p->key_dtype == LSA_KEY_BF16 || p->key_dtype == LSA_KEY_FP8_E4M3FN, LSA_ERR_INVALID_ARG,
              "key_dtype=%d unknown", p->key_dtype);
  LSA_REQUIRE(p->page >= 32 && p->page <= 256 && p->page % 32 == 0, LSA_ERR_UNSUPPORTED,
              "page=%d must be a multiple of 32 in [32, 256]", p->page);
  LSA_REQUIRE(p->sub_block >= 1 && pow2(p->sub_block) && p->page % p->sub_block == 0 && p->page / p->sub_block <= 32,
              LSA_ERR_UNSUPPORTED, "sub_block=%d must be a power of two dividing page=%d with page/sub_block <= 32",
              p->sub_block, p->page);
  LSA_REQUIRE(p->k_sparse >= 1, LSA_ERR_INVALID_ARG, "k_sparse=%d must be >= 1", p->k_sparse);
  LSA_REQUIRE(p->k_sink >= 0 && p->k_swa >= 0, LSA_ERR_INVALID_ARG, "k_sink=%d / k_swa=%d must be >= 0", p->k_sink,
              p->k_swa);
  LSA_REQUIRE(p->run_align >= 1, LSA_ERR_INVALID_ARG, "run_align=%d must be >= 1", p->run_align);
  LSA_REQUIRE((int64_t)p->k_sink + p->k_swa + p->k_sparse < (1LL << 30), LSA_ERR_INVALID_ARG, "k_cap too large");
  LSA_REQUIRE(p->pooling == LSA_POOL_MEAN || p->pooling == LSA_POOL_MINMAX, LSA_ERR_INVALID_ARG, "pooling=%d unknown",
              p->pooling);
  LSA_REQUIRE(p->hi_min_kv >= 0, LSA_ERR_INVALID_ARG, "hi_min_kv=%d < 0", p->hi_min_kv);
  if (p->keep_pages > 0)
    LSA_REQUIRE(p->k_swa >= p->page, LSA_ERR_UNSUPPORTED,
                "hierarchical mode needs k_swa=%d >= page=%d (scored pages must not reach past the query)", p->k_swa,
                p->page);
  return LSA_OK;
}

// Adaptive dispatch: a hierarchical indexer whose call covers at most hi_min_kv cached tokens runs
// flat (Eq. 7 over the whole eligible range), where scoring every candidate costs less than the
// coarse stage plus the recalled pages.
lsa_index_params effective_params(const lsa_index_params* p, int64_t max_kv) {
  lsa_index_params e = *p;
  if (e.keep_pages > 0 && max_kv <= (int64_t)e.hi_min_kv) e.keep_pages = 0;
  return e;
}

// Rows of fine-score slots and page-score entries for a given key range. Rows are processed in
// passes of rows_per_pass so that the workspace stays within kPassBytes however long the rows are
// (flat mode over a long cache holds one score per cached token per row).
constexpr size_t kPassBytes = size_t(8) << 30;

struct IndexPlan {
  int64_t n_pages;        // pages in [0, max_kv)
  int64_t slots;          // fine-score slots per row
  int64_t rows_per_pass;  // query rows per pass over the workspace
  size_t off_page_keys, off_pages, off_fine, total;
};

// Workspace bytes one query row needs (page-score keys, recalled pages, fine-score keys).
size_t index_row_bytes(const lsa_index_params* p, int64_t max_kv) {
  const int64_t n_pages = cdiv(max_kv, p->page);
  const bool hi = p->keep_pages > 0;
  const int64_t slots = (hi ? (int64_t)p->keep_pages : n_pages) * p->page;
  return (size_t)slots * 4 + (hi ? (size_t)(n_pages + p->keep_pages) * 4 : 0);
}

// budget == 0: passes of about kPassBytes in multiples of 8 rows (the caller's workspace is sized
// from this plan); otherwise the plan fits within `budget` bytes (a fixed scratch array), in as
// many rows per pass as fit, at least one (the caller checks that one row fits).
IndexPlan plan_index(const lsa_index_params* p, int64_t n_rows, int64_t max_kv, size_t budget = 0) {
  IndexPlan pl{};
  pl.n_pages = cdiv(max_kv, p->page);
  const bool hi = p->keep_pages > 0;
  pl.slots = (hi ? (int64_t)p->keep_pages : pl.n_pages) * p->page;
  const size_t per_row = index_row_bytes(p, max_kv);
  int64_t rpp;
  if (budget == 0) {
    rpp = (int64_t)(kPassBytes / (per_row > 0 ? per_row : 1));
    rpp = rpp < 8 ? 8 : rpp / 8 * 8;
  } else {  // three areas, each rounded up to 256 bytes
    rpp = budget > 768 ? (int64_t)((budget - 768) / (per_row > 0 ? per_row : 1)) : 0;
    rpp = rpp < 1 ? 1 : rpp;
  }
  pl.rows_per_pass = n_rows < rpp ? n_rows : rpp;
  const size_t r = (size_t)pl.rows_per_pass;
  size_t off = 0;
  pl.off_page_keys = off;
  if (hi) off += round_up(r * pl.n_pages * 4, 256);
  pl.off_pages = off;
  if (hi) off += round_up(r * p->keep_pages * 4, 256);
  pl.off_fine = off;
  off += round_up(r * pl.slots * 4, 256);
  pl.total = off;
  return pl;
}

// paged: decode (the page selection also stages the page-table entries of the eligible pages)
lsa_status check_lds(const lsa_index_params* p, const IndexPlan& pl, bool paged) {
  const int k_cap = p->k_sink + p->k_swa + p->k_sparse;
  const size_t ts = lsa::token_select_lds_bytes(pl.slots, k_cap, p->keep_pages);
  LSA_REQUIRE(ts + lsa::token_select_static_lds(pl.slots) <= kMaxLds, LSA_ERR_UNSUPPORTED,
              "the selection of %lld candidate slots with k_cap=%d does not fit the LDS of one workgroup; "
              "lower k_sparse + k_sink + k_swa or keep_pages",
              (long long)pl.slots, k_cap);
  if (p->keep_pages > 0)
    LSA_REQUIRE(lsa::page_select_lds_bytes(pl.n_pages, paged) + kSelectStaticLds <= kMaxLds, LSA_ERR_UNSUPPORTED,
                "%lld pages per row exceed the LDS of the page selection", (long long)pl.n_pages);
  return LSA_OK;
}

lsa::IndexGeom make_geom(const lsa_index_params* p) {
  lsa::IndexGeom g{};
  g.H = p->n_heads;
  g.D = p->head_dim;
  g.fp8 = p->key_dtype == LSA_KEY_FP8_E4M3FN;
  g.P = p->page;
  g.B = p->sub_block;
  g.M = p->keep_pages > 0 ? p->keep_pages : 0;
  g.minmax = p->pooling == LSA_POOL_MINMAX;
  g.k_sparse = p->k_sparse;
  g.k_sink = p->k_sink;
  g.k_swa = p->k_swa;
  g.C = p->run_align;
  return g;
}

lsa_status run_index(const lsa_index_params* p, const lsa::IndexGeom& g, int64_t n_rows, int64_t max_kv,
                     const void* q, const float* w, const void* k, const float* k_scale, const void* block_keys,
                     int32_t* idx, int32_t* count, lsa_run* runs, int32_t* run_count, int32_t* pages_out,
                     void* workspace, hipStream_t st, size_t budget = 0) {
  const IndexPlan pl = plan_index(p, n_rows, max_kv, budget);
  uint8_t* ws = static_cast<uint8_t*>(workspace);
  uint32_t* page_keys = reinterpret_cast<uint32_t*>(ws + pl.off_page_keys);
  uint32_t* fine = reinterpret_cast<uint32_t*>(ws + pl.off_fine);
  hipError_t e = lsa::prepare_index_kernels();
  if (e != hipSuccess) return hip_fail(e, "prepare");
  const int k_cap = p->k_sink + p->k_swa + p->k_sparse;
  // eligible pages of the last row bound every row's work
  const int64_t max_elig = pl.n_pages;
  const int64_t max_sel = g.M > 0 ? (max_elig < g.M ? max_elig : g.M) : max_elig;
  for (int64_t r0 = 0; r0 < n_rows; r0 += pl.rows_per_pass) {
    const int64_t nr = n_rows - r0 < pl.rows_per_pass ? n_rows - r0 : pl.rows_per_pass;
    // this pass's rows: shift the row-indexed inputs and outputs (prefill: positions; decode:
    // context lengths and page-table rows)
    lsa::IndexGeom gp = g;
    if (g.ctx_len) {
      gp.ctx_len = g.ctx_len + r0;
      gp.page_table = g.page_table + r0 * g.max_pages;
    } else {
      gp.q_start = g.q_start + r0;
    }
    const auto* q16 = static_cast<const uint16_t*>(q) + r0 * g.H * g.D;
    const float* wp = w + r0 * g.H;
    int32_t* pages = pages_out ? pages_out + r0 * g.M : reinterpret_cast<int32_t*>(ws + pl.off_pages);
    int32_t* phys = (g.ctx_len && g.M > 0) ? reinterpret_cast<int32_t*>(page_keys) : nullptr;
    if (g.M > 0) {
      const int64_t max_tiles = cdiv(max_elig * (g.P / g.B), 32);
      e = lsa::launch_coarse(gp, nr, q16, wp, static_cast<const uint16_t*>(block_keys), page_keys, pl.n_pages,
                             max_tiles, st);
      if (e != hipSuccess) return hip_fail(e, "coarse page scoring");
      // decode: the physical pages of the recalled ones go to the row's page-key area, which the
      // page selection has read by then
      e = lsa::launch_page_select(gp, nr, page_keys, pl.n_pages, pages, phys, max_elig, st);
      if (e != hipSuccess) return hip_fail(e, "page selection");
    }
    e = lsa::launch_fine(gp, nr, q16, wp, k, k_scale, pages, phys, pl.n_pages, fine, pl.slots, max_sel, st);
    if (e != hipSuccess) return hip_fail(e, "fine token scoring");
    e = lsa::launch_token_select(gp, nr, fine, pl.slots, g.M > 0 ? pages : nullptr, idx + r0 * k_cap, count + r0,
                                 runs ? reinterpret_cast<int32_t*>(runs + r0 * k_cap) : nullptr,
                                 run_count ? run_count + r0 : nullptr, pl.slots, st);
    if (e != hipSuccess) return hip_fail(e, "token selection");
  }
  return LSA_OK;
}

// ---------------------------------------------------------------- attention planning
struct AttnPlan {
  int n_split, split_len;
  size_t off_rows, off_po, off_ml, total;
};

// Workgroups a split attention call aims for: one per CU (the MLA kernel's LDS admits one per CU).
// Every split re-loads its row's 73 KB of Q and writes 128 KB of fp32 partials, so more, shorter
// splits cost more than they add in parallelism (64-sequence decode: 0.067 ms per layer at 256
// workgroups, 0.166 ms at 2048).
constexpr int64_t kSplitTarget = 256;

AttnPlan plan_attn(const lsa_attn_params* p, int64_t n_rows, int32_t k_cap, int32_t paged) {
  AttnPlan pl{};
  pl.n_split = 1;
  pl.split_len = k_cap;
  const bool mla = p->latent != 0;
  if (mla && n_rows > 0 && n_rows < kSplitTarget) {
    // too few rows to fill 256 CUs: split every row's list into 32-token-aligned pieces
    int64_t want = cdiv(kSplitTarget, n_rows);
    int64_t max_split = cdiv(k_cap, 32);
    int64_t ns = want < max_split ? want : max_split;
    if (ns > 1) {
      int64_t len = round_up((size_t)cdiv(k_cap, ns), 32);
      pl.split_len = (int)len;
      pl.n_split = (int)cdiv(k_cap, len);
    }
  }
  size_t off = 0;
  pl.off_rows = off;  // translated cache rows (paged MQA; the MLA kernel translates as it stages)
  if (paged && !mla) off += round_up((size_t)n_rows * k_cap * 4, 256);
  pl.off_po = off;
  if (pl.n_split > 1) off += round_up((size_t)n_rows * pl.n_split * p->n_heads * p->d_v * 2, 256);
  pl.off_ml = off;
  if (pl.n_split > 1) off += round_up((size_t)n_rows * pl.n_split * p->n_heads * 2 * 4, 256);
  pl.total = off;
  return pl;
}

lsa_status check_attn_params(const lsa_attn_params* p) {
  LSA_REQUIRE(p != nullptr, LSA_ERR_INVALID_ARG, "params is NULL");
  const bool mla = p->n_heads == 64 && p->d_qk == 576 && p->d_v == 512 && p->latent == 1;
  const bool mqa = p->n_heads == 16 && p->d_qk == 128 && p->d_v == 128 && p->latent == 0;
  LSA_REQUIRE(mla || mqa, LSA_ERR_UNSUPPORTED,
              "attention shape (n_heads=%d, d_qk=%d, d_v=%d, latent=%d) not supported; use (64,576,512,1) or "
              "(16,128,128,0)",
              p->n_heads, p->d_qk, p->d_v, p->latent);
  LSA_REQUIRE(p->sm_scale > 0.f && p->sm_scale < 1e30f, LSA_ERR_INVALID_ARG, "sm_scale must be positive and finite");
  return LSA_OK;
}

}  // namespace

namespace lsa {
hipError_t prepare_index_kernels();
}

extern "C" {

int32_t lsa_index_k_cap(const lsa_index_params* p) {
  if (!p) return 0;
  return p->k_sink + p->k_swa + p->k_sparse;
}

size_t lsa_index_workspace_size(const lsa_index_params* p, int64_t n_rows, int64_t max_kv) {
  if (check_index_params(p) != LSA_OK || n_rows < 0 || max_kv < 0) return 0;
  const lsa_index_params e = effective_params(p, max_kv);
  return plan_index(&e, n_rows, max_kv).total;
}

static lsa_status run_block_cache(const lsa_index_params* p, bool minmax, int64_t n_items, const int64_t* rows,
                                  int64_t n_tok, const void* k, const float* k_scale, void* block_keys, void* stream,
                                  const char* what) {
  g_err[0] = 0;
  lsa_status s = check_index_params(p);
  if (s != LSA_OK) return s;
  const bool fp8 = p->key_dtype == LSA_KEY_FP8_E4M3FN;
  LSA_REQUIRE(n_tok >= 0 && n_items >= 0, LSA_ERR_INVALID_ARG, "n_tok=%lld / n_rows=%lld < 0", (long long)n_tok,
              (long long)n_items);
  if (n_items == 0 || n_tok / p->sub_block == 0) return LSA_OK;  // nothing to read or write
  LSA_REQUIRE(k && block_keys, LSA_ERR_INVALID_ARG, "k / block_keys is NULL");
  LSA_REQUIRE(fp8 == (k_scale != nullptr), LSA_ERR_INVALID_ARG, "k_scale must be given exactly for fp8 keys");
  LSA_REQUIRE(aligned(k, 16) && aligned(block_keys, 16) && aligned(k_scale, 4) && aligned(rows, 8),
              LSA_ERR_INVALID_ARG, "k/block_keys must be 16-byte aligned, k_scale 4-byte, rows 8-byte aligned");
  hipError_t e = lsa::launch_block_keys(n_items, rows, n_tok, p->head_dim, p->sub_block, fp8, minmax, k, k_scale,
                                        static_cast<uint16_t*>(block_keys), static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, what);
  return LSA_OK;
}

lsa_status lsa_block_means(const lsa_index_params* p, int64_t n_tok, const void* k, const float* k_scale,
                           void* block_keys, void* stream) {
  if (p == nullptr) return fail(LSA_ERR_INVALID_ARG, "params is NULL");
  const int64_t n_sub = n_tok / (p->sub_block > 0 ? p->sub_block : 1);
  return run_block_cache(p, false, n_sub, nullptr, n_tok, k, k_scale, block_keys, stream, "block means");
}

lsa_status lsa_block_minmax(const lsa_index_params* p, int64_t n_tok, const void* k, const float* k_scale,
                            void* block_keys, void* stream) {
  if (p == nullptr) return fail(LSA_ERR_INVALID_ARG, "params is NULL");
  const int64_t n_sub = n_tok / (p->sub_block > 0 ? p->sub_block : 1);
  return run_block_cache(p, true, n_sub, nullptr, n_tok, k, k_scale, block_keys, stream, "block min-max");
}

lsa_status lsa_block_keys_update(const lsa_index_params* p, int64_t n_rows, const int64_t* rows, int64_t n_tok,
                                 const void* k, const float* k_scale, void* block_keys, void* stream) {
  if (p == nullptr) return fail(LSA_ERR_INVALID_ARG, "params is NULL");
  if (n_rows > 0 && rows == nullptr) return fail(LSA_ERR_INVALID_ARG, "rows is NULL");
  return run_block_cache(p, p->pooling == LSA_POOL_MINMAX, n_rows, rows, n_tok, k, k_scale, block_keys, stream,
                         "block cache update");
}

// A hierarchical call that the dispatch ran flat recalls no pages: its pages_out rows are all -1.
static lsa_status clear_pages_if_flat(const lsa_index_params* p, const lsa_index_params* e, int32_t* pages_out,
                                      int64_t n_rows, hipStream_t st) {
  if (pages_out == nullptr || e->keep_pages > 0 || n_rows == 0) return LSA_OK;
  hipError_t err = lsa::launch_fill_i32(pages_out, n_rows * p->keep_pages, -1, st);
  return err == hipSuccess ? LSA_OK : hip_fail(err, "clear pages_out");
}

static lsa_status check_index_io(const lsa_index_params* p, const void* q, const float* w, const void* k,
                                 const float* k_scale, const void* block_keys, int64_t n_sub, int32_t* idx,
                                 int32_t* count, lsa_run* runs, int32_t* run_count, void* workspace,
                                 size_t ws_bytes, size_t need) {
  const bool fp8 = p->key_dtype == LSA_KEY_FP8_E4M3FN;
  LSA_REQUIRE(q && w && k && idx && count, LSA_ERR_INVALID_ARG, "q, w, k, idx and count must be non-NULL");
  LSA_REQUIRE(fp8 == (k_scale != nullptr), LSA_ERR_INVALID_ARG, "k_scale must be given exactly for fp8 keys");
  LSA_REQUIRE(p->keep_pages <= 0 || n_sub == 0 || block_keys != nullptr, LSA_ERR_INVALID_ARG,
              "block_keys is NULL but keep_pages > 0 (hierarchical mode)");
  LSA_REQUIRE((runs == nullptr) == (run_count == nullptr), LSA_ERR_INVALID_ARG,
              "runs and run_count must be both NULL or both non-NULL");
  LSA_REQUIRE(aligned(q, 16) && aligned(k, 16) && aligned(block_keys, 16), LSA_ERR_INVALID_ARG,
              "q, k and block_keys must be 16-byte aligned");
  LSA_REQUIRE(aligned(w, 4) && aligned(k_scale, 4) && aligned(idx, 4) && aligned(count, 4) && aligned(run_count, 4),
              LSA_ERR_INVALID_ARG, "w, k_scale, idx, count, run_count must be 4-byte aligned");
  LSA_REQUIRE(aligned(runs, 8), LSA_ERR_INVALID_ARG, "runs must be 8-byte aligned");
  LSA_REQUIRE(need == 0 || (workspace != nullptr && aligned(workspace, 256)), LSA_ERR_WORKSPACE,
              "workspace must be non-NULL and 256-byte aligned");
  LSA_REQUIRE(ws_bytes >= need, LSA_ERR_WORKSPACE, "workspace of %zu bytes < %zu needed", ws_bytes, need);
  return LSA_OK;
}

lsa_status lsa_index_prefill(const lsa_index_params* p, int64_t q_start, int64_t n_q, int64_t n_kv, const void* q,
                             const float* w, const void* k, const float* k_scale, const void* block_keys, int32_t* idx,
                             int32_t* count, lsa_run* runs, int32_t* run_count, int32_t* pages_out, void* workspace,
                             size_t ws_bytes, void* stream) {
  g_err[0] = 0;
  lsa_status s = check_index_params(p);
  if (s != LSA_OK) return s;
  LSA_REQUIRE(q_start >= 0 && n_q >= 0 && n_kv >= 0, LSA_ERR_INVALID_ARG, "negative q_start / n_q / n_kv");
  LSA_REQUIRE(q_start <= n_kv && n_q <= n_kv - q_start, LSA_ERR_INVALID_ARG,
              "rows [q_start, q_start + n_q) = [%lld, +%lld) exceed n_kv = %lld", (long long)q_start, (long long)n_q,
              (long long)n_kv);
  LSA_REQUIRE(n_kv < (1LL << 31), LSA_ERR_UNSUPPORTED, "n_kv must be < 2^31 (int32 positions)");
  LSA_REQUIRE(n_q < (1LL << 28), LSA_ERR_UNSUPPORTED, "n_q must be < 2^28 per call (chunk longer prefills)");
  LSA_REQUIRE(pages_out == nullptr || p->keep_pages > 0, LSA_ERR_INVALID_ARG, "pages_out needs keep_pages > 0");
  LSA_REQUIRE(aligned(pages_out, 4), LSA_ERR_INVALID_ARG, "pages_out must be 4-byte aligned");
  const lsa_index_params e = effective_params(p, n_kv);
  const IndexPlan pl = plan_index(&e, n_q, n_kv);
  s = check_lds(&e, pl, false);
  if (s != LSA_OK) return s;
  if (n_q == 0) return LSA_OK;  // nothing to read or write
  s = check_index_io(&e, q, w, k, k_scale, block_keys, n_kv / p->sub_block, idx, count, runs, run_count, workspace,
                     ws_bytes, pl.total);
  if (s != LSA_OK) return s;
  s = clear_pages_if_flat(p, &e, pages_out, n_q, static_cast<hipStream_t>(stream));
  if (s != LSA_OK) return s;
  lsa::IndexGeom g = make_geom(&e);
  g.q_start = q_start;
  g.n_kv = n_kv;
  g.n_sub = n_kv / p->sub_block;
  return run_index(&e, g, n_q, n_kv, q, w, k, k_scale, block_keys, idx, count, runs, run_count,
                   e.keep_pages > 0 ? pages_out : nullptr, workspace, static_cast<hipStream_t>(stream));
}

// Checks and geometry shared by the two decode entry points. `budget` = 0: the caller's workspace
// (ws_bytes must cover the plan); otherwise the fixed scratch array of that many bytes.
static lsa_status decode_setup(const lsa_index_params* p, int32_t batch, const int32_t* ctx_len,
                               const int32_t* page_table, int32_t max_pages, int32_t kv_page_size, int64_t n_phys,
                               const void* q, const float* w, const void* k, const float* k_scale,
                               const void* block_keys, int32_t* idx, int32_t* count, lsa_run* runs,
                               int32_t* run_count, int32_t* pages_out, void* workspace, size_t ws_bytes, size_t budget,
                               lsa_index_params* e_out, lsa::IndexGeom* g_out) {
  lsa_status s = check_index_params(p);
  if (s != LSA_OK) return s;
  LSA_REQUIRE(batch >= 0, LSA_ERR_INVALID_ARG, "batch=%d < 0", batch);
  LSA_REQUIRE(max_pages >= 1 && kv_page_size >= 1 && n_phys >= 1, LSA_ERR_INVALID_ARG,
              "max_pages, kv_page_size and n_phys must be >= 1");
  LSA_REQUIRE(kv_page_size == p->page, LSA_ERR_UNSUPPORTED,
              "paged indexing needs page (%d) == kv_page_size (%d)", p->page, kv_page_size);
  LSA_REQUIRE((int64_t)max_pages * kv_page_size < (1LL << 31) && n_phys * kv_page_size < (1LL << 31),
              LSA_ERR_UNSUPPORTED, "positions and cache rows must fit in int32");
  LSA_REQUIRE(ctx_len && page_table, LSA_ERR_INVALID_ARG, "ctx_len / page_table is NULL");
  LSA_REQUIRE(aligned(ctx_len, 4) && aligned(page_table, 4) && aligned(pages_out, 4), LSA_ERR_INVALID_ARG,
              "ctx_len, page_table, pages_out must be 4-byte aligned");
  LSA_REQUIRE(pages_out == nullptr || p->keep_pages > 0, LSA_ERR_INVALID_ARG, "pages_out needs keep_pages > 0");
  const int64_t max_kv = (int64_t)max_pages * kv_page_size;
  const lsa_index_params e = effective_params(p, max_kv);
  const IndexPlan pl = plan_index(&e, batch, max_kv, budget);
  s = check_lds(&e, pl, true);
  if (s != LSA_OK) return s;
  if (budget != 0) {
    const size_t row = index_row_bytes(&e, max_kv);
    LSA_REQUIRE(row + 768 <= budget, LSA_ERR_WORKSPACE,
                "one query row of this call needs %zu bytes of indexer workspace; the fixed scratch array holds "
                "%zu (lower max_pages or keep_pages, or use lsa_index_decode with a workspace)",
                row + 768, budget);
  }
  if (batch == 0) return LSA_OK;  // nothing to read or write
  // (with the fixed scratch array there is no caller workspace to check)
  s = check_index_io(&e, q, w, k, k_scale, block_keys, n_phys * kv_page_size / p->sub_block, idx, count, runs,
                     run_count, workspace, ws_bytes, budget != 0 ? 0 : pl.total);
  if (s != LSA_OK) return s;
  lsa::IndexGeom g = make_geom(&e);
  g.ctx_len = ctx_len;
  g.page_table = page_table;
  g.max_pages = max_pages;
  g.kv_page = kv_page_size;
  g.n_phys = n_phys;
  g.n_kv = n_phys * kv_page_size;
  g.n_sub = g.n_kv / p->sub_block;
  *e_out = e;
  *g_out = g;
  return LSA_OK;
}

lsa_status lsa_index_decode(const lsa_index_params* p, int32_t batch, const int32_t* ctx_len,
                            const int32_t* page_table, int32_t max_pages, int32_t kv_page_size, int64_t n_phys,
                            const void* q, const float* w, const void* k, const float* k_scale, const void* block_keys,
                            int32_t* idx, int32_t* count, lsa_run* runs, int32_t* run_count, int32_t* pages_out,
                            void* workspace, size_t ws_bytes, void* stream) {
  g_err[0] = 0;
  lsa_index_params e{};
  lsa::IndexGeom g{};
  lsa_status s = decode_setup(p, batch, ctx_len, page_table, max_pages, kv_page_size, n_phys, q, w, k, k_scale,
                              block_keys, idx, count, runs, run_count, pages_out, workspace, ws_bytes, 0, &e, &g);
  if (s != LSA_OK || batch == 0) return s;
  hipStream_t st = static_cast<hipStream_t>(stream);
  s = clear_pages_if_flat(p, &e, pages_out, batch, st);
  if (s != LSA_OK) return s;
  return run_index(&e, g, batch, (int64_t)max_pages * kv_page_size, q, w, k, k_scale, block_keys, idx, count, runs,
                   run_count, e.keep_pages > 0 ? pages_out : nullptr, workspace, st);
}

}  // extern "C"

// ---------------------------------------------------------------- decode indexer without allocation
// Scratch of lsa_index_decode_static: the indexer workspace (page-score keys, recalled pages,
// fine-score keys) of one row pass lives in this fixed device array instead of a caller-owned
// workspace. Each device holds its own copy until the process ends. Host code must not use the
// array's name as an address: its device address is looked up once per device (first call there)
// and only that pointer is passed to kernels. Nothing in it needs to start at zero: every entry a
// kernel uses is written earlier in the same call (the paged fine kernel requests the page slots
// of its chunk before it knows how many of them the row has, and ignores the others), and it
// keeps the last call's contents.
static __device__ __align__(256) uint8_t scratch[LSA_STATIC_SCRATCH_BYTES];

namespace {
std::mutex g_scratch_mu;
void* g_scratch_ptr[64] = {};

// Device address of `scratch` on the current device (looked up on the first call there).
hipError_t static_scratch(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (ptr == nullptr) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}
}  // namespace

extern "C" {

lsa_status lsa_index_decode_static(const lsa_index_params* p, int32_t batch, const int32_t* ctx_len,
                                   const int32_t* page_table, int32_t max_pages, int32_t kv_page_size,
                                   int64_t n_phys, const void* q, const float* w, const void* k,
                                   const float* k_scale, const void* block_keys, int32_t* idx, int32_t* count,
                                   lsa_run* runs, int32_t* run_count, int32_t* pages_out, void* stream) {
  g_err[0] = 0;
  lsa_index_params e{};
  lsa::IndexGeom g{};
  lsa_status s = decode_setup(p, batch, ctx_len, page_table, max_pages, kv_page_size, n_phys, q, w, k, k_scale,
                              block_keys, idx, count, runs, run_count, pages_out, nullptr, 0,
                              LSA_STATIC_SCRATCH_BYTES, &e, &g);
  if (s != LSA_OK || batch == 0) return s;
  void* ws = nullptr;
  hipError_t err = static_scratch(&ws);
  if (err != hipSuccess) return hip_fail(err, "static scratch address");
  hipStream_t st = static_cast<hipStream_t>(stream);
  s = clear_pages_if_flat(p, &e, pages_out, batch, st);
  if (s != LSA_OK) return s;
  return run_index(&e, g, batch, (int64_t)max_pages * kv_page_size, q, w, k, k_scale, block_keys, idx, count, runs,
                   run_count, e.keep_pages > 0 ? pages_out : nullptr, ws, st, LSA_STATIC_SCRATCH_BYTES);
}

size_t lsa_sparse_attn_workspace_size(const lsa_attn_params* p, int64_t n_rows, int32_t k_cap, int32_t paged) {
  if (check_attn_params(p) != LSA_OK || n_rows < 0 || k_cap < 1) return 0;
  return plan_attn(p, n_rows, k_cap, paged).total;
}

lsa_status lsa_sparse_attn(const lsa_attn_params* p, int64_t n_rows, const void* q, const void* kv, const void* v,
                           int64_t n_kv_rows, const int32_t* idx, const int32_t* count, int32_t k_cap,
                           const int32_t* page_table, int32_t max_pages, int32_t kv_page_size, int32_t rows_per_seq,
                           void* out, float* lse, void* workspace, size_t ws_bytes, void* stream) {
  g_err[0] = 0;
  lsa_status s = check_attn_params(p);
  if (s != LSA_OK) return s;
  const bool mla = p->latent != 0;
  LSA_REQUIRE(n_rows >= 0 && k_cap >= 1, LSA_ERR_INVALID_ARG, "n_rows < 0 or k_cap < 1");
  LSA_REQUIRE(n_rows < (1LL << 31), LSA_ERR_UNSUPPORTED, "n_rows must be < 2^31");
  if (n_rows == 0) return LSA_OK;  // nothing to read or write
  LSA_REQUIRE(n_kv_rows >= 1 && n_kv_rows < (1LL << 31), LSA_ERR_INVALID_ARG, "n_kv_rows=%lld not in [1, 2^31)",
              (long long)n_kv_rows);
  LSA_REQUIRE(q && kv && idx && count && out, LSA_ERR_INVALID_ARG, "q, kv, idx, count and out must be non-NULL");
  LSA_REQUIRE(mla == (v == nullptr), LSA_ERR_INVALID_ARG, mla ? "v must be NULL for a latent cache" : "v is NULL");
  LSA_REQUIRE(aligned(q, 16) && aligned(kv, 16) && aligned(v, 16) && aligned(out, 16), LSA_ERR_INVALID_ARG,
              "q, kv, v and out must be 16-byte aligned");
  LSA_REQUIRE(aligned(idx, 4) && aligned(count, 4) && aligned(lse, 4) && aligned(page_table, 4), LSA_ERR_INVALID_ARG,
              "idx, count, lse and page_table must be 4-byte aligned");
  const bool paged = page_table != nullptr;
  if (paged)
    LSA_REQUIRE(max_pages >= 1 && kv_page_size >= 1 && rows_per_seq >= 1, LSA_ERR_INVALID_ARG,
                "paged cache needs max_pages, kv_page_size and rows_per_seq >= 1");
  const AttnPlan pl = plan_attn(p, n_rows, k_cap, paged);
  LSA_REQUIRE(pl.total == 0 || (workspace != nullptr && aligned(workspace, 256)), LSA_ERR_WORKSPACE,
              "workspace must be non-NULL and 256-byte aligned");
  LSA_REQUIRE(ws_bytes >= pl.total, LSA_ERR_WORKSPACE, "workspace of %zu bytes < %zu needed", ws_bytes, pl.total);
  if (n_rows == 0) return LSA_OK;

  hipStream_t st = static_cast<hipStream_t>(stream);
  uint8_t* ws = static_cast<uint8_t*>(workspace);
  lsa::AttnGeom a{};
  a.q = static_cast<const uint16_t*>(q);
  a.kv = static_cast<const uint16_t*>(kv);
  a.v = static_cast<const uint16_t*>(v);
  a.n_kv_rows = n_kv_rows;
  a.rows = idx;
  a.count = count;
  a.k_cap = k_cap;
  a.out = static_cast<uint16_t*>(out);
  a.lse = lse;
  a.n_rows = n_rows;
  a.n_split = pl.n_split;
  a.split_len = pl.split_len;
  a.scale_log2 = p->sm_scale * 1.4426950408889634f;
  a.part = -1;  // the whole index list
  if (paged && mla) {  // the MLA kernel translates positions while it stages each list
    a.page_table = page_table;
    a.max_pages = max_pages;
    a.kv_page = kv_page_size;
    a.rows_per_seq = rows_per_seq;
  } else if (paged) {
    int32_t* rows = reinterpret_cast<int32_t*>(ws + pl.off_rows);
    hipError_t e = lsa::launch_translate_rows(idx, count, n_rows, k_cap, page_table, max_pages, kv_page_size,
                                              rows_per_seq, n_kv_rows, rows, st);
    if (e != hipSuccess) return hip_fail(e, "page-table translation");
    a.rows = rows;
  }
  if (pl.n_split > 1) {
    a.part_o = reinterpret_cast<uint16_t*>(ws + pl.off_po);
    a.part_ml = reinterpret_cast<float*>(ws + pl.off_ml);
  }
  hipError_t e = mla ? lsa::launch_mla_attn(a, st) : lsa::launch_mqa_attn(a, st);
  if (e != hipSuccess) return hip_fail(e, "sparse attention");
  return LSA_OK;
}

// The run form reads the runs inside the attention kernel for the contiguous MLA cache; any other
// layout (MQA, paged cache) first expands them into a position list at the head of the workspace
// and then runs the list form on it.
static bool runs_fused(const lsa_attn_params* p, bool paged) { return p->latent != 0 && !paged; }

static size_t runs_list_bytes(int64_t n_rows, int32_t k_cap) {
  return round_up((size_t)n_rows * k_cap * 4, 256) + round_up((size_t)n_rows * 4, 256);
}

size_t lsa_sparse_attn_runs_workspace_size(const lsa_attn_params* p, int64_t n_rows, int32_t k_cap, int32_t paged) {
  if (check_attn_params(p) != LSA_OK || n_rows < 0 || k_cap < 1) return 0;
  const size_t attn = plan_attn(p, n_rows, k_cap, paged).total;
  return runs_fused(p, paged != 0) ? attn : runs_list_bytes(n_rows, k_cap) + attn;
}

lsa_status lsa_sparse_attn_runs(const lsa_attn_params* p, int64_t n_rows, const void* q, const void* kv, const void* v,
                                int64_t n_kv_rows, const lsa_run* runs, const int32_t* run_count, int32_t k_cap,
                                const int32_t* page_table, int32_t max_pages, int32_t kv_page_size,
                                int32_t rows_per_seq, void* out, float* lse, void* workspace, size_t ws_bytes,
                                void* stream) {
  g_err[0] = 0;
  lsa_status s = check_attn_params(p);
  if (s != LSA_OK) return s;
  const bool mla = p->latent != 0, paged = page_table != nullptr;
  LSA_REQUIRE(n_rows >= 0 && k_cap >= 1, LSA_ERR_INVALID_ARG, "n_rows < 0 or k_cap < 1");
  LSA_REQUIRE(n_rows < (1LL << 31) && k_cap < (1 << 30), LSA_ERR_UNSUPPORTED, "n_rows must be < 2^31, k_cap < 2^30");
  if (n_rows == 0) return LSA_OK;  // nothing to read or write
  LSA_REQUIRE(n_kv_rows >= 1 && n_kv_rows < (1LL << 31), LSA_ERR_INVALID_ARG, "n_kv_rows=%lld not in [1, 2^31)",
              (long long)n_kv_rows);
  LSA_REQUIRE(q && kv && runs && run_count && out, LSA_ERR_INVALID_ARG,
              "q, kv, runs, run_count and out must be non-NULL");
  LSA_REQUIRE(mla == (v == nullptr), LSA_ERR_INVALID_ARG, mla ? "v must be NULL for a latent cache" : "v is NULL");
  LSA_REQUIRE(aligned(q, 16) && aligned(kv, 16) && aligned(v, 16) && aligned(out, 16), LSA_ERR_INVALID_ARG,
              "q, kv, v and out must be 16-byte aligned");
  LSA_REQUIRE(aligned(runs, 8) && aligned(run_count, 4) && aligned(lse, 4) && aligned(page_table, 4),
              LSA_ERR_INVALID_ARG, "runs must be 8-byte aligned, run_count, lse and page_table 4-byte aligned");
  if (paged)
    LSA_REQUIRE(max_pages >= 1 && kv_page_size >= 1 && rows_per_seq >= 1, LSA_ERR_INVALID_ARG,
                "paged cache needs max_pages, kv_page_size and rows_per_seq >= 1");
  const size_t need = lsa_sparse_attn_runs_workspace_size(p, n_rows, k_cap, paged);
  LSA_REQUIRE(need == 0 || (workspace != nullptr && aligned(workspace, 256)), LSA_ERR_WORKSPACE,
              "workspace must be non-NULL and 256-byte aligned");
  LSA_REQUIRE(ws_bytes >= need, LSA_ERR_WORKSPACE, "workspace of %zu bytes < %zu needed", ws_bytes, need);
  hipStream_t st = static_cast<hipStream_t>(stream);
  uint8_t* ws = static_cast<uint8_t*>(workspace);

  if (!runs_fused(p, paged)) {
    int32_t* idx = reinterpret_cast<int32_t*>(ws);
    int32_t* count = reinterpret_cast<int32_t*>(ws + round_up((size_t)n_rows * k_cap * 4, 256));
    const hipError_t e = lsa::launch_expand_runs(reinterpret_cast<const int32_t*>(runs), run_count, n_rows, k_cap,
                                                 idx, count, st);
    if (e != hipSuccess) return hip_fail(e, "run expansion");
    const size_t head = runs_list_bytes(n_rows, k_cap);
    return lsa_sparse_attn(p, n_rows, q, kv, v, n_kv_rows, idx, count, k_cap, page_table, max_pages, kv_page_size,
                           rows_per_seq, out, lse, ws + head, ws_bytes - head, stream);
  }
  const AttnPlan pl = plan_attn(p, n_rows, k_cap, 0);
  lsa::AttnGeom a{};
  a.q = static_cast<const uint16_t*>(q);
  a.kv = static_cast<const uint16_t*>(kv);
  a.n_kv_rows = n_kv_rows;
  a.runs = reinterpret_cast<const int32_t*>(runs);
  a.run_count = run_count;
  a.k_cap = k_cap;
  a.out = static_cast<uint16_t*>(out);
  a.lse = lse;
  a.n_rows = n_rows;
  a.n_split = pl.n_split;
  a.split_len = pl.split_len;
  a.scale_log2 = p->sm_scale * 1.4426950408889634f;
  a.part = -1;
  if (pl.n_split > 1) {
    a.part_o = reinterpret_cast<uint16_t*>(ws + pl.off_po);
    a.part_ml = reinterpret_cast<float*>(ws + pl.off_ml);
  }
  const hipError_t e = lsa::launch_mla_attn(a, st);
  if (e != hipSuccess) return hip_fail(e, "sparse attention (run form)");
  return LSA_OK;
}

// ---------------------------------------------------------------- split attention (HFA)
// Rows per pass of lsa_hfa_attn: the two partials of a row (bf16 values, fp32 maximum and sum per
// head) take 2 * 64 * (512 * 2 + 2 * 4) bytes.
constexpr int64_t kHfaRowsPerPass = 16384;

static int64_t hfa_rows_per_pass(int64_t n_rows) { return n_rows < kHfaRowsPerPass ? n_rows : kHfaRowsPerPass; }

size_t lsa_hfa_attn_workspace_size(const lsa_attn_params* p, int64_t n_rows) {
  if (check_attn_params(p) != LSA_OK || n_rows < 0 || p->latent == 0) return 0;
  const size_t r = (size_t)hfa_rows_per_pass(n_rows);
  return round_up(r * 2 * 64 * 512 * 2, 256) + round_up(r * 2 * 64 * 2 * 4, 256);
}

namespace {
// The second stream of the split attention and the two events that fork and join it, one set
// per device, created on first use (default priority, non-blocking).
struct HfaStreams {
  hipStream_t side = nullptr;
  hipEvent_t fork = nullptr, join = nullptr;
};
std::mutex g_hfa_mu;       // creation of the per-device streams and events
std::mutex g_hfa_call_mu;  // one call's enqueue sequence at a time
HfaStreams g_hfa[64];

hipError_t hfa_streams(HfaStreams** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lk(g_hfa_mu);
  HfaStreams& h = g_hfa[dev];
  if (h.side == nullptr) {  // all three objects, or none (a failed call leaves nothing half-made)
    HfaStreams n;
    if ((e = hipStreamCreateWithFlags(&n.side, hipStreamNonBlocking)) == hipSuccess &&
        (e = hipEventCreateWithFlags(&n.fork, hipEventDisableTiming)) == hipSuccess &&
        (e = hipEventCreateWithFlags(&n.join, hipEventDisableTiming)) == hipSuccess) {
      h = n;
    } else {
      if (n.fork) (void)hipEventDestroy(n.fork);
      if (n.side) (void)hipStreamDestroy(n.side);
      return e;
    }
  }
  *out = &h;
  return hipSuccess;
}
}  // namespace

lsa_status lsa_hfa_attn(const lsa_attn_params* p, int64_t n_rows, const void* q, const void* kv, int64_t n_kv_rows,
                        const int32_t* idx, const int32_t* count, int32_t k_cap, int64_t q_start, int32_t k_swa,
                        void* out, float* lse, void* workspace, size_t ws_bytes, void* stream) {
  g_err[0] = 0;
  lsa_status s = check_attn_params(p);
  if (s != LSA_OK) return s;
  LSA_REQUIRE(p->latent != 0, LSA_ERR_UNSUPPORTED, "the split attention is implemented for the MLA latent cache");
  LSA_REQUIRE(n_rows >= 0 && k_cap >= 1 && q_start >= 0 && k_swa >= 0, LSA_ERR_INVALID_ARG,
              "n_rows, q_start, k_swa must be >= 0 and k_cap >= 1");
  LSA_REQUIRE(n_rows < (1LL << 31), LSA_ERR_UNSUPPORTED, "n_rows must be < 2^31");
  if (n_rows == 0) return LSA_OK;  // nothing to read or write
  LSA_REQUIRE(n_kv_rows >= 1 && n_kv_rows < (1LL << 31), LSA_ERR_INVALID_ARG, "n_kv_rows=%lld not in [1, 2^31)",
              (long long)n_kv_rows);
  LSA_REQUIRE(q_start <= n_kv_rows && n_rows <= n_kv_rows - q_start, LSA_ERR_INVALID_ARG,
              "rows [q_start, q_start + n_rows) = [%lld, +%lld) exceed n_kv_rows = %lld (the window reads the "
              "cache up to the query)",
              (long long)q_start, (long long)n_rows, (long long)n_kv_rows);
  LSA_REQUIRE(q && kv && idx && count && out, LSA_ERR_INVALID_ARG, "q, kv, idx, count and out must be non-NULL");
  LSA_REQUIRE(aligned(q, 16) && aligned(kv, 16) && aligned(out, 16), LSA_ERR_INVALID_ARG,
              "q, kv and out must be 16-byte aligned");
  LSA_REQUIRE(aligned(idx, 4) && aligned(count, 4) && aligned(lse, 4), LSA_ERR_INVALID_ARG,
              "idx, count and lse must be 4-byte aligned");
  const size_t need = lsa_hfa_attn_workspace_size(p, n_rows);
  LSA_REQUIRE(workspace != nullptr && aligned(workspace, 256), LSA_ERR_WORKSPACE,
              "workspace must be non-NULL and 256-byte aligned");
  LSA_REQUIRE(ws_bytes >= need, LSA_ERR_WORKSPACE, "workspace of %zu bytes < %zu needed", ws_bytes, need);

  hipStream_t st = static_cast<hipStream_t>(stream);
  HfaStreams* hs = nullptr;
  hipError_t e = hfa_streams(&hs);
  if (e != hipSuccess) return hip_fail(e, "split attention streams");
  // the side stream and the fork/join events are shared by every call on this device: enqueue a
  // whole call's record / wait / launch sequence under the lock, so that the side stream never
  // interleaves the parts of two calls and each part waits on its own call's fork
  std::lock_guard<std::mutex> call_lock(g_hfa_call_mu);
  const int64_t rpp = hfa_rows_per_pass(n_rows);
  uint8_t* ws = static_cast<uint8_t*>(workspace);
  uint16_t* part_o = reinterpret_cast<uint16_t*>(ws);
  float* part_ml = reinterpret_cast<float*>(ws + round_up((size_t)rpp * 2 * 64 * 512 * 2, 256));
  for (int64_t r0 = 0; r0 < n_rows; r0 += rpp) {
    const int64_t nr = n_rows - r0 < rpp ? n_rows - r0 : rpp;
    lsa::AttnGeom a{};
    a.q = static_cast<const uint16_t*>(q) + r0 * 64 * 576;
    a.kv = static_cast<const uint16_t*>(kv);
    a.n_kv_rows = n_kv_rows;
    a.rows = idx + r0 * k_cap;
    a.count = count + r0;
    a.k_cap = k_cap;
    a.out = static_cast<uint16_t*>(out) + r0 * 64 * 512;
    a.lse = lse ? lse + r0 * 64 : nullptr;
    a.part_o = part_o;
    a.part_ml = part_ml;
    a.n_rows = nr;
    a.n_split = 2;
    a.split_len = k_cap;
    a.scale_log2 = p->sm_scale * 1.4426950408889634f;
    a.k_swa = k_swa;
    a.q_pos0 = q_start + r0;
    // the listed non-window part on the caller's stream, the window on the side stream, then the
    // log-sum-exp merge once both partials exist (each pass reuses the partial buffers, which the
    // stream order of the merge and the next pass's first kernel protects)
    if ((e = hipEventRecord(hs->fork, st)) != hipSuccess) return hip_fail(e, "split attention fork");
    if ((e = hipStreamWaitEvent(hs->side, hs->fork, 0)) != hipSuccess) return hip_fail(e, "split attention fork");
    a.part = 0;
    if ((e = lsa::launch_mla_attn_part(a, st)) != hipSuccess) return hip_fail(e, "split attention (listed part)");
    a.part = 1;
    if ((e = lsa::launch_mla_attn_window(a, hs->side)) != hipSuccess) return hip_fail(e, "split attention (window)");
    if ((e = hipEventRecord(hs->join, hs->side)) != hipSuccess) return hip_fail(e, "split attention join");
    if ((e = hipStreamWaitEvent(st, hs->join, 0)) != hipSuccess) return hip_fail(e, "split attention join");
    if ((e = lsa::launch_attn_combine(a, 64, 512, st)) != hipSuccess) return hip_fail(e, "split attention merge");
  }
  return LSA_OK;
}

const char* lsa_status_string(int32_t status) {
  switch (status) {
    case LSA_OK: return "LSA_OK";
    case LSA_ERR_INVALID_ARG: return "LSA_ERR_INVALID_ARG";
    case LSA_ERR_UNSUPPORTED: return "LSA_ERR_UNSUPPORTED";
    case LSA_ERR_WORKSPACE: return "LSA_ERR_WORKSPACE";
    case LSA_ERR_HIP: return "LSA_ERR_HIP";
    default: return "LSA_ERR_UNKNOWN";
  }
}

const char* lsa_last_error(void) { return g_err; }

const char* lsa_version(void) { return "lsa-mi355x 0.1"; }

}  // extern "C"
