// Internal interface between the C-ABI front end (lsa_api.cpp) and the HIP kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stddef.h>

namespace lsa {

// Everything the indexer kernels need to know about one call, passed by value.
struct IndexGeom {
  int H, D, fp8;                 // indexer heads, head dim, fp8 keys
  int P, B, M;                   // page, sub-block, kept pages (M <= 0: flat)
  int minmax;                    // coarse stage: min-max pooling (block keys [k_max | k_min])
  int k_sparse, k_sink, k_swa, C;
  int64_t q_start;               // prefill: position of row 0
  int64_t n_kv;                  // prefill: cached tokens
  int64_t n_sub;                 // mean keys available
  const int32_t* ctx_len;        // decode: [rows] (nullptr for prefill)
  const int32_t* page_table;     // decode: [rows, max_pages]
  int max_pages, kv_page;
  int64_t n_phys;
};

// Block cache of the coarse stage: mean keys [n_sub, D] or min-max extrema [n_sub, 2D]. rows == nullptr:
// every sub-block 0..n_items-1; otherwise the sub-blocks holding token rows[0..n_items).
hipError_t launch_block_keys(int64_t n_items, const int64_t* rows, int64_t n_tok, int D, int B, bool fp8, bool minmax,
                             const void* k, const float* ks, uint16_t* out, hipStream_t st);
hipError_t launch_coarse(const IndexGeom& g, int64_t n_rows, const uint16_t* q, const float* w, const uint16_t* kmean,
                         uint32_t* page_keys, int64_t ld, int64_t max_tiles, hipStream_t st);
// Page selection; with phys != nullptr (paged decode) it also writes each recalled page's physical
// page to phys[row * ld + k], which may alias page_keys (the row's keys are read first).
hipError_t launch_page_select(const IndexGeom& g, int64_t n_rows, const uint32_t* page_keys, int64_t ld,
                              int32_t* pages, int32_t* phys, int64_t max_elig, hipStream_t st);
// Dynamic LDS bytes of the page selection over rows of up to max_elig eligible pages.
inline size_t page_select_lds_bytes(int64_t max_elig, bool with_phys) {
  return (size_t)(max_elig > 0 ? max_elig : 1) * (with_phys ? 8 : 4);
}
// Fine scoring; paged decode reads the recalled pages' physical pages from phys (row stride ldp)
// as the page selection wrote them (nullptr in flat mode: looked up in the page table).
hipError_t launch_fine(const IndexGeom& g, int64_t n_rows, const uint16_t* q, const float* w, const void* k,
                       const float* ks, const int32_t* pages, const int32_t* phys, int64_t ldp, uint32_t* fine_keys,
                       int64_t ldf, int64_t max_sel, hipStream_t st);
// Dynamic LDS bytes of the token selection; rows of up to kSelectRegMax candidates keep their keys
// in registers (20 KB of static LDS), larger ones stage them in LDS (4 KB of static LDS).
constexpr int64_t kSelectRegMax = 512 * 64;
// Calls with at most this many rows (decode batches) select tokens (rows of <= 8192 candidates) and
// pages with 1024 threads per row instead of 512 and 256: with few rows the GPU is mostly idle and
// per-row latency counts.
constexpr int64_t kSelectFewRows = 1024;
size_t token_select_lds_bytes(int64_t slots_cap, int k_cap, int M);
inline size_t token_select_static_lds(int64_t slots_cap) { return slots_cap <= kSelectRegMax ? 20 * 1024 : 4 * 1024; }
hipError_t launch_token_select(const IndexGeom& g, int64_t n_rows, const uint32_t* fine_keys, int64_t ldf,
                               const int32_t* pages, int32_t* idx, int32_t* count, int32_t* runs, int32_t* run_count,
                               int64_t slots_cap, hipStream_t st);
hipError_t prepare_index_kernels();
// p[0..n) = v (a kernel, so that the call also records correctly inside a captured graph).
hipError_t launch_fill_i32(int32_t* p, int64_t n, int32_t v, hipStream_t st);
// Run encoding -> position list: idx[r, 0..count[r]) from runs[r, 0..run_count[r]) (int32 pairs).
hipError_t launch_expand_runs(const int32_t* runs, const int32_t* run_count, int64_t n_rows, int k_cap, int32_t* idx,
                              int32_t* count, hipStream_t st);

// Sparse attention over gathered rows.
struct AttnGeom {
  const uint16_t* q;       // [n_rows, H, d_qk]
  const uint16_t* kv;      // latent [n_kv_rows, d_qk] or K
  const uint16_t* v;       // V [n_kv_rows, d_v] or nullptr
  int64_t n_kv_rows;
  const int32_t* rows;     // [n_rows, k_cap] cache rows to attend (positions, or translated rows)
  const int32_t* count;    // [n_rows]
  int k_cap;
  uint16_t* out;           // [n_rows, H, d_v]
  float* lse;              // [n_rows, H] or nullptr
  uint16_t* part_o;        // split partials, each normalised by its own sum, bf16 [n_rows, n_split, H, d_v]
  float* part_ml;          // [n_rows, n_split, H, 2]
  int64_t n_rows;
  int n_split, split_len;  // slots per split (multiple of the tile)
  float scale_log2;        // sm_scale * log2(e)
  // Split by kind of position (Sec. 4.1.1): part -1 = the whole list; 0 = the list without its
  // window entries (the sliding window is the list's last min(k_swa, t + 1) entries); 1 = the
  // window [t - k_swa + 1, t] as contiguous cache rows. Parts write split `part` of n_split = 2.
  int part;
  int k_swa;
  int64_t q_pos0;          // position t of row 0
  // Run form of the lists (MLA only; nullptr = use rows/count): row r's list is the concatenation
  // of the runs (start, length) runs[r, 0..run_count[r]), int32 pairs with row stride k_cap.
  const int32_t* runs;
  const int32_t* run_count;
  // Paged cache (MLA list form; nullptr = rows are cache rows): rows holds positions, and position
  // s of query row r is cache row page_table[(r / rows_per_seq) * max_pages + s / kv_page] *
  // kv_page + s % kv_page, translated while the list is staged.
  const int32_t* page_table;
  int max_pages, kv_page, rows_per_seq;
};

hipError_t launch_mla_attn(const AttnGeom& a, hipStream_t st);
hipError_t launch_mqa_attn(const AttnGeom& a, hipStream_t st);
hipError_t launch_attn_combine(const AttnGeom& a, int H, int d_v, hipStream_t st);
// One part (a.part = 0 or 1) of the split attention into the partials a.part_o / a.part_ml.
hipError_t launch_mla_attn_part(const AttnGeom& a, hipStream_t st);
// The window part (a.part = 1) as the query-tiled kernel: two consecutive rows per workgroup
// share each contiguous window tile.
hipError_t launch_mla_attn_window(const AttnGeom& a, hipStream_t st);
hipError_t launch_translate_rows(const int32_t* idx, const int32_t* count, int64_t n_rows, int k_cap,
                                 const int32_t* page_table, int max_pages, int kv_page, int rows_per_seq,
                                 int64_t n_kv_rows, int32_t* out_rows, hipStream_t st);

}  // namespace lsa
